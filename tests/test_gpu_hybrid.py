"""The hybrids' attention layers in the library: the linear maps
(hcmix_linear_forward / _backward) against their plain definitions, and a
whole hybrid step (sparse stacks, projections, attention cores, all weight
gradients; paper_2609_18145_amd.hybrid) against the composed oracle
(oracle/hybrid.py), through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
from oracle import hybrid as hybrid_oracle
from paper_2609_18145_amd import hcmix, inputs
from paper_2609_18145_amd.hybrid import HybridStack
from tests.util import TOL, fro_rel_err, row_rel_err, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hcmix.load()


def log(msg):
    print(msg, flush=True)


def bf(rng, shape, scale=1.0):
    return inputs.round_bf16((rng.standard_normal(shape) * scale).astype(np.float32))


# (rows, in, out): the hybrid's QKV and output projections at full size, and
# ragged row counts, narrow and non-square maps
LINEAR = [(16384, 512, 1536), (16384, 512, 512), (62, 128, 192), (1000, 64, 64),
          (2 * 128, 192, 128)]


@pytest.mark.parametrize("rows,n_in,n_out", LINEAR)
def test_linear_map_against_its_definition(rows, n_in, n_out):
    log(f"case: linear rows={rows} in={n_in} out={n_out}")
    rng = np.random.default_rng(rows + n_in)
    x, w, dy = bf(rng, (rows, n_in)), bf(rng, (n_out, n_in), n_in ** -0.5), bf(rng, (rows, n_out))
    tx, tw, tdy = to_dev(x, "bf16"), to_dev(w, "bf16"), to_dev(dy, "bf16")
    y = hcmix.linear_forward(tx, tw)
    dx, dw = hcmix.linear_backward(tx, tw, tdy)
    dx2, dw2 = hcmix.linear_backward(tx, tw, tdy)
    acc = torch.ones_like(dw)
    hcmix.linear_backward(tx, tw, tdy, dw=acc, with_dx=False, accumulate=True)
    torch.cuda.synchronize()
    ry = hybrid_oracle.linear_forward(x, w)
    rdx, rdw = hybrid_oracle.linear_backward(x, w, dy)
    assert row_rel_err(to_host(y), ry) <= 1e-2
    assert row_rel_err(to_host(dx), rdx) <= 1e-2
    assert fro_rel_err(to_host(dw), rdw) <= 1e-4
    assert torch.equal(dx, dx2) and torch.equal(dw, dw2)
    assert torch.equal(acc, dw + 1.0)


def make_hybrid(batch, n, width, heads, schedule, seed):
    """The stack's inputs and weights, and per attention layer a QKV projection
    drawn at a quarter of N(0, 1/width)'s scale, so that the attention scores
    stay of order one, as a normalised model keeps them.  With the full scale
    the unnormalised activations give rows of scores up to about 40, whose
    softmax backward cancels so strongly that bf16 arithmetic itself (the
    products of this segment emulated in bf16 on the CPU) is 20% off fp64 in
    dX: that would test the conditioning, not the kernels."""
    ns = sum(1 for e in schedule if e != "attn")
    na = sum(1 for e in schedule if e == "attn")
    s = inputs.make_stack(batch, n, width, ns, True, "bf16", seed=seed)
    rng = np.random.default_rng(seed + 100)
    attn = [(bf(rng, (3 * width, width), 0.25 * width ** -0.5),
             bf(rng, (width, width), width ** -0.5)) for _ in range(na)]
    return s, attn


HYBRIDS = [
    (2, 128, 128, 2, [0, 1, "attn", 2, 3, 4, "attn", 5, 6]),
    (2, 64, 192, 3, [oracle.NEAR, 5, "attn", oracle.NEAR, 3, oracle.NEAR, "attn", 1]),
    (4, 256, 512, 8, [0, 1, 2, "attn", 3, 4, 5, 6, 7, "attn", 0, 1, 2, 3, 4, 5, 6, 7]),
]


@pytest.mark.parametrize("batch,n,width,heads,schedule", HYBRIDS)
def test_hybrid_step_against_composed_oracle(batch, n, width, heads, schedule):
    """Segment by segment, each fed the library's own input (its forward input,
    or its output gradient for the backward), as the per-layer checks of the
    stacks: the sharp softmax rows of unnormalised activations make the
    end-to-end comparison ill-conditioned (bf16 storage of the activations
    alone moves the output of the first case by about 5% against fp64; that
    figure is printed beside the end-to-end error), while every segment and
    every weight gradient must stay within the bf16 bound.  The segments
    chain through the library's outputs, so the checks cover the whole step."""
    log(f"case: hybrid step B={batch} n={n} w={width} heads={heads} schedule={schedule}")
    s, attn = make_hybrid(batch, n, width, heads, schedule, seed=batch + n)
    h = HybridStack(schedule, [to_dev(a, "bf16") for a in s.w_self],
                    [to_dev(a, "bf16") for a in s.w_off],
                    [(to_dev(a, "bf16"), to_dev(b, "bf16")) for a, b in attn], heads)
    K = len(h.segments)
    xs = [to_dev(s.x, "bf16")]
    h._saved = []
    for k in range(K):
        xs.append(h.forward_segment(k, xs[-1]))
    gs = [None] * K + [to_dev(s.dy, "bf16")]
    h._dw_in, h.dw_attn = [], [None] * len(attn)
    for k in reversed(range(K)):
        gs[k] = h.backward_segment(k, gs[k + 1])
    h.sparse_weight_gradients()
    torch.cuda.synchronize()
    worst = {"y": 0.0, "dx": 0.0, "dW": 0.0}
    for k, (kind, arg) in enumerate(h.segments):
        xin, gout = to_host(xs[k]), to_host(gs[k + 1])
        if kind == "sparse":
            idx = [j for j, _ in arg]
            codes = [c for _, c in arg]
            rws, rwo = [s.w_self[j] for j in idx], [s.w_off[j] for j in idx]
            rxs = oracle.stack_forward(xin, rws, rwo, codes, True)
            rdx, dws, dwo = oracle.stack_backward(rxs, rws, rwo, codes, gout, True)
            # within a run the oracle goes through all its layers from the
            # run's input, as the whole-stack tests do
            got = [(h.dw_self[j], h.dw_off[j]) for j in idx]
            ref = list(zip(dws, dwo))
        else:
            ry, sv = hybrid_oracle.forward(xin, ["attn"], [], [], [attn[arg]], heads)
            rdx, _, _, ra = hybrid_oracle.backward(sv, gout, ["attn"], [], [], [attn[arg]], heads)
            rxs = [None, ry]
            got, ref = [h.dw_attn[arg]], [ra[0]]
        e_y = row_rel_err(to_host(xs[k + 1]), rxs[-1])
        e_dx = row_rel_err(to_host(gs[k]), rdx)
        e_w = max(fro_rel_err(to_host(g), r) for pair, rpair in zip(got, ref)
                  for g, r in zip(pair, rpair))
        log(f"  segment {k} {kind}: y {e_y:.2e}  dx {e_dx:.2e}  dW {e_w:.2e}")
        worst = {"y": max(worst["y"], e_y), "dx": max(worst["dx"], e_dx),
                 "dW": max(worst["dW"], e_w)}
    ry, _ = hybrid_oracle.forward(s.x, schedule, s.w_self, s.w_off, attn, heads)
    log(f"  end to end: y {row_rel_err(to_host(xs[-1]), ry):.2e} (fp64 oracle, for reference)")
    assert max(worst.values()) <= TOL["bf16"], worst
