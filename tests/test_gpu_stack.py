"""Whole-stack parity of the HIP path against the CPU oracle, at the
workloads' real shapes (through the C ABI via the Python binding)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_18145_amd import hcmix, inputs
from tests.util import TOL, fro_rel_err, row_rel_err, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hcmix.load()


def log(msg):
    print(msg, flush=True)


def run_gpu_stack(s, with_backward=True):
    dt = s.dtype
    x = to_dev(s.x, dt)
    ws = [to_dev(w, dt) for w in s.w_self]
    wo = [to_dev(w, dt) for w in s.w_off]
    xs = hcmix.stack_forward(x, ws, wo, s.layers, s.causal)
    out = {"y": xs[-1]}
    if with_backward:
        dx, dws, dwo = hcmix.stack_backward(xs, ws, wo, s.layers, to_dev(s.dy, dt), s.causal)
        out.update(dx=dx, dws=dws, dwo=dwo)
    torch.cuda.synchronize()
    return {k: ([to_host(t) for t in v] if isinstance(v, list) else to_host(v))
            for k, v in out.items()}


def check_stack(s, got, windows=None, with_dw=True, tol=None):
    tol = TOL[s.dtype] if tol is None else tol
    sel = slice(None) if windows is None else windows
    x = s.x[sel]
    xs = oracle.stack_forward(x, s.w_self, s.w_off, s.layers, s.causal)
    e_y = row_rel_err(got["y"][sel], xs[-1])
    log(f"  y row err {e_y:.3e}")
    assert e_y <= tol
    if "dx" in got:
        dx, dws, dwo = oracle.stack_backward(xs, s.w_self, s.w_off, s.layers, s.dy[sel], s.causal)
        e_dx = row_rel_err(got["dx"][sel], dx)
        log(f"  dx row err {e_dx:.3e}")
        assert e_dx <= tol
        if with_dw:
            e_w = max(max(fro_rel_err(g, r) for g, r in zip(got["dws"], dws)),
                      max(fro_rel_err(g, r) for g, r in zip(got["dwo"], dwo)))
            log(f"  dW fro err {e_w:.3e}")
            assert e_w <= tol


@pytest.mark.parametrize("schedule", ["rot", "fixed"])
def test_tiny_stack_fp32(schedule):
    """n=16, width 32, batch 2, 4 layers in fp32: the rotated stack (d = 0..3)
    and the un-rotated control that repeats d = 0."""
    layers = oracle.schedule_rot(4) if schedule == "rot" else oracle.schedule_fixed(4)
    s = inputs.make_preset("tiny", layers=layers)
    log(f"tiny fp32 {schedule}")
    check_stack(s, run_gpu_stack(s))


def test_tiny_impulse_reaches_everyone_only_when_rotated():
    """Impulse at one position: after log2 n rotated layers every position of
    its window is nonzero; under the fixed control only the pair {j, j^1}."""
    n, width = 16, 32
    for j in [0, 5, 15]:
        x = np.zeros((1, n, width), dtype=np.float32)
        x[0, j] = 1.0
        one = np.eye(width, dtype=np.float32)
        tx = to_dev(x, "f32")
        te = to_dev(one, "f32")
        for layers, expect_all in ((oracle.schedule_rot(4), True), (oracle.schedule_fixed(4), False)):
            xs = hcmix.stack_forward(tx, [te] * 4, [te] * 4, layers, False)
            y = to_host(xs[-1])[0]
            reached = set(np.flatnonzero(np.abs(y).sum(axis=1)))
            assert reached == (set(range(n)) if expect_all else {j, j ^ 1})


@pytest.mark.parametrize("schedule", ["rot", "fixed"])
def test_reach_stack_bf16_full_size(schedule):
    """n=256, width 64, batch 64, 8 bidirectional layers, bf16: whole stack,
    forward and backward, every output compared."""
    layers = oracle.schedule_rot(8) if schedule == "rot" else oracle.schedule_fixed(8)
    s = inputs.make_preset("reach", layers=layers)
    log(f"reach bf16 {schedule}")
    check_stack(s, run_gpu_stack(s))


def test_lm256_stack_bf16_sampled_windows():
    """n=256, width 512, batch 64, 16 causal layers, bf16, in the launch
    configuration of the benchmark; the oracle recomputes three of the 64
    windows (windows are independent, so this is their exact reference)."""
    s = inputs.make_preset("lm256")
    log("lm256 bf16 full batch")
    got = run_gpu_stack(s)
    check_stack(s, got, windows=[0, 31, 63], with_dw=False)


def test_lm256_stack_bf16_weight_gradients():
    """Same stack at batch 4 so the oracle can form every weight gradient."""
    s = inputs.make_preset("lm256", batch=4)
    log("lm256 bf16 batch 4")
    check_stack(s, run_gpu_stack(s))


def test_lm256_layer_full_size_with_weight_gradients():
    """One layer at the benchmark's full shape and launch configuration
    (64 windows of 256 x 512): every output, including both weight gradients,
    against the oracle."""
    s = inputs.make_preset("lm256", num_layers=1)
    x, ws, wo, dy = (to_dev(a, "bf16") for a in (s.x, s.w_self[0], s.w_off[0], s.dy))
    for layer in (7, 0):
        log(f"lm256 full-size layer {layer}")
        y = hcmix.forward(x, ws, wo, layer, True)
        dx, dws, dwo = hcmix.backward(x, ws, wo, dy, layer, True)
        torch.cuda.synchronize()
        ry = oracle.forward(s.x, s.w_self[0], s.w_off[0], layer, True)
        rdx, rws, rwo = oracle.backward(s.x, s.w_self[0], s.w_off[0], s.dy, layer, True)
        assert row_rel_err(to_host(y), ry) <= TOL["bf16"]
        assert row_rel_err(to_host(dx), rdx) <= TOL["bf16"]
        assert fro_rel_err(to_host(dws), rws) <= 1e-4
        assert fro_rel_err(to_host(dwo), rwo) <= 1e-4


def test_long4096_layers_bf16_sampled():
    """n=4096, width 1024 (strides up to 2048 rows): the layers with the
    largest and smallest strides at full shape (batch 8), outputs of window 0
    against the oracle; weight gradients from a one-window call."""
    s = inputs.make_preset("long4096", num_layers=1)
    x = to_dev(s.x, "bf16")
    dy = to_dev(s.dy, "bf16")
    ws = to_dev(s.w_self[0], "bf16")
    wo = to_dev(s.w_off[0], "bf16")
    for layer in (11, 0):
        log(f"long4096 layer {layer}")
        y = hcmix.forward(x, ws, wo, layer, True)
        dx, _, _ = hcmix.backward(x, ws, wo, dy, layer, True)
        _, dws1, dwo1 = hcmix.backward(x[:1].contiguous(), ws, wo, dy[:1].contiguous(), layer, True)
        torch.cuda.synchronize()
        ry = oracle.forward(s.x[:1], s.w_self[0], s.w_off[0], layer, True)
        rdx, rws, rwo = oracle.backward(s.x[:1], s.w_self[0], s.w_off[0], s.dy[:1], layer, True)
        assert row_rel_err(to_host(y)[:1], ry) <= TOL["bf16"]
        assert row_rel_err(to_host(dx)[:1], rdx) <= TOL["bf16"]
        assert fro_rel_err(to_host(dws1), rws) <= 1e-4
        assert fro_rel_err(to_host(dwo1), rwo) <= 1e-4


def test_autograd_stack_matches_oracle():
    s = inputs.make_preset("reach", batch=4, num_layers=8)
    dt = torch.bfloat16
    x = to_dev(s.x, "bf16").requires_grad_(True)
    ws = [to_dev(w, "bf16").requires_grad_(True) for w in s.w_self]
    wo = [to_dev(w, "bf16").requires_grad_(True) for w in s.w_off]
    y = hcmix.Stack.apply(x, s.layers, s.causal, *ws, *wo)
    y.backward(to_dev(s.dy, "bf16"))
    torch.cuda.synchronize()
    xs = oracle.stack_forward(s.x, s.w_self, s.w_off, s.layers, s.causal)
    dx, dws, dwo = oracle.stack_backward(xs, s.w_self, s.w_off, s.layers, s.dy, s.causal)
    assert y.dtype == dt
    assert row_rel_err(to_host(y), xs[-1]) <= TOL["bf16"]
    assert row_rel_err(to_host(x.grad), dx) <= TOL["bf16"]
    for g, r in zip(ws, dws):
        assert fro_rel_err(to_host(g.grad), r) <= TOL["bf16"]
    for g, r in zip(wo, dwo):
        assert fro_rel_err(to_host(g.grad), r) <= TOL["bf16"]


def test_layer_by_layer_backward_matches_oracle_and_replays_in_a_graph():
    """bf16 stack backward on the layer-by-layer path (width 128: not the fused
    path): against the oracle, then captured as a graph from a side stream and
    replayed three times with eager work and synchronisation in between, every
    replay bitwise equal to the eager call."""
    s = inputs.make_stack(batch=4, n=256, width=128, num_layers=5, causal=True, dtype="bf16",
                          seed=11)
    log("case: layer-by-layer bf16 backward, B=4 n=256 w=128 L=5 causal, seed 11")
    dt = s.dtype
    x = to_dev(s.x, dt)
    ws = [to_dev(w, dt) for w in s.w_self]
    wo = [to_dev(w, dt) for w in s.w_off]
    dy = to_dev(s.dy, dt)
    xs = hcmix.stack_forward(x, ws, wo, s.layers, s.causal)
    wsp = hcmix.alloc_stack_workspace(4, 256, 128, 5, torch.bfloat16, x.device)
    dx, dws, dwo = hcmix.stack_backward(xs, ws, wo, s.layers, dy, s.causal, workspace=wsp)
    torch.cuda.synchronize()
    check_stack(s, {"y": to_host(xs[-1]), "dx": to_host(dx), "dws": [to_host(t) for t in dws],
                    "dwo": [to_host(t) for t in dwo]})
    ref = [dx.clone()] + [t.clone() for t in dws + dwo]

    g_dx = torch.empty_like(dx)
    g_dws = [torch.empty_like(t) for t in dws]
    g_dwo = [torch.empty_like(t) for t in dwo]
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        hcmix.stack_backward(xs, ws, wo, s.layers, dy, s.causal, dx=g_dx, dws=g_dws, dwo=g_dwo,
                             workspace=wsp)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=side):
            hcmix.stack_backward(xs, ws, wo, s.layers, dy, s.causal, dx=g_dx, dws=g_dws,
                                 dwo=g_dwo, workspace=wsp)
    for rep in range(3):
        for t in [g_dx, *g_dws, *g_dwo]:
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = [g_dx] + g_dws + g_dwo
        for a, b in zip(got, ref):
            assert torch.equal(a, b), f"replay {rep} differs from the eager call"
        log(f"  replay {rep} bitwise equal")


@pytest.mark.parametrize("causal", [False, True])
def test_layer_by_layer_backward_ragged_rows(causal):
    """bf16 stack backward on the layer-by-layer path (width 256, 6 rotated
    layers) with 3 windows of 64 positions: 96 row pairs, one partial 128-pair
    tile, in both modes; every output and weight gradient against the oracle."""
    s = inputs.make_stack(batch=3, n=64, width=256, num_layers=6, causal=causal, dtype="bf16",
                          seed=12)
    log(f"case: layer-by-layer bf16 backward, B=3 n=64 w=256 L=6 causal={causal}, seed 12")
    check_stack(s, run_gpu_stack(s))


def test_deferred_backward_longer_than_one_chunk():
    """bf16 stack of 66 rotated causal layers (width 128): the deferred path
    keeps a ring of 65 gradients and forms the weight gradients in two
    launches (64 + 2 layers); every output against the oracle.  The bf16
    storage of each layer's output is a rounding step, and over a stack these
    compound like a random walk (about sqrt(L) 2^-9 per row), so the bound of
    the 2e-2 workloads (at most 24 layers) is scaled by sqrt(L / 24) here."""
    L = 66
    s = inputs.make_stack(batch=1, n=64, width=128, num_layers=L, causal=True, dtype="bf16",
                          seed=13)
    log(f"case: deferred backward, B=1 n=64 w=128 L={L} causal, seed 13")
    check_stack(s, run_gpu_stack(s), tol=TOL["bf16"] * (L / 24) ** 0.5)


def test_deferred_backward_bidirectional_short_stack():
    """Bidirectional deferred path on a two-layer stack (row ranges and the
    fixed-order sum of the weight-gradient launch), against the oracle."""
    s = inputs.make_stack(batch=8, n=256, width=256, num_layers=2, causal=False, dtype="bf16",
                          seed=14)
    log("case: deferred backward, B=8 n=256 w=256 L=2 bidirectional, seed 14")
    check_stack(s, run_gpu_stack(s))
