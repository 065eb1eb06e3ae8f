"""Decode step (hcmix_decode_step): positions of a window decoded one at a
time must give the causal stack's output at that position, as the oracle's
full-window forward computes it."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_18145_amd import hcmix, inputs
from tests.util import TOL, row_rel_err, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hcmix.load()


def log(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("batch,n,width,dtype,schedule", [
    (3, 16, 64, "bf16", "rot"), (40, 16, 128, "bf16", "mixa"), (2, 64, 64, "bf16", "rot"),
    (5, 8, 32, "f32", "rot"), (2, 16, 24, "f32", "mixa"), (33, 32, 512, "bf16", "mixa"),
    (17, 16, 1024, "bf16", "rot"), (3, 16, 192, "bf16", "mixa"),   # two rounds; a partial one
])
def test_decode_every_position_matches_the_stack(batch, n, width, dtype, schedule):
    layers = (list(range(2 * oracle.log2n(n))) if schedule == "rot"
              else oracle.schedule_mixa(n))
    L = len(layers)
    log(f"decode {batch}x{n}x{width} {dtype} {schedule} L={L}")
    s = inputs.make_stack(batch=batch, n=n, width=width, num_layers=L, causal=True, dtype=dtype,
                          seed=41, layers=layers, with_dy=False)
    want = oracle.stack_forward(s.x, s.w_self, s.w_off, layers, True)[-1]
    x = to_dev(s.x, dtype)
    ws = [to_dev(w, dtype) for w in s.w_self]
    wo = [to_dev(w, dtype) for w in s.w_off]
    cache = hcmix.alloc_decode_cache(batch, n, width, layers, x.dtype, x.device)
    cache.fill_(0xFF)                      # never-written contents must never be read
    got = np.zeros_like(want)
    for pos in range(n):
        y = hcmix.decode_step(x[:, pos].contiguous(), ws, wo, layers, n, pos, cache)
        got[:, pos] = to_host(y)
    torch.cuda.synchronize()
    err = row_rel_err(got, want)
    log(f"  row err {err:.2e}")
    assert err <= TOL[dtype]


def test_decode_restarts_at_position_zero():
    """A second window decoded into the same cache starts over at pos 0."""
    batch, n, width = 4, 16, 64
    layers = oracle.schedule_mixa(n)
    L = len(layers)
    s1 = inputs.make_stack(batch=batch, n=n, width=width, num_layers=L, causal=True, dtype="bf16",
                           seed=42, layers=layers, with_dy=False)
    s2 = inputs.make_stack(batch=batch, n=n, width=width, num_layers=L, causal=True, dtype="bf16",
                           seed=43, layers=layers, with_dy=False)
    ws = [to_dev(w, "bf16") for w in s1.w_self]
    wo = [to_dev(w, "bf16") for w in s1.w_off]
    cache = hcmix.alloc_decode_cache(batch, n, width, layers, torch.bfloat16, "cuda")
    for s in (s1, s2):
        x = to_dev(s.x, "bf16")
        got = np.stack([to_host(hcmix.decode_step(x[:, p].contiguous(), ws, wo, layers, n, p, cache))
                        for p in range(n)], axis=1)
        want = oracle.stack_forward(s.x, s1.w_self, s1.w_off, layers, True)[-1]
        assert row_rel_err(got, want) <= TOL["bf16"]


def test_decode_lm256_shape_sampled_windows():
    """The benchmark's decode configuration: 64 windows of 256 positions,
    width 512, 16 rotated causal layers, every position decoded in turn into
    one cache; the oracle's full-window forward of three of the windows is
    their exact reference (windows are independent)."""
    s = inputs.make_preset("lm256", with_dy=False)
    B, n = s.x.shape[0], s.x.shape[1]
    log(f"decode lm256 shape B={B} n={n} w={s.x.shape[2]} L={len(s.layers)}")
    x = to_dev(s.x, "bf16")
    ws = [to_dev(w, "bf16") for w in s.w_self]
    wo = [to_dev(w, "bf16") for w in s.w_off]
    cache = hcmix.alloc_decode_cache(B, n, x.shape[2], s.layers, x.dtype, x.device)
    cols = [x[:, p].contiguous() for p in range(n)]
    ys = [hcmix.decode_step(cols[p], ws, wo, s.layers, n, p, cache) for p in range(n)]
    got = to_host(torch.stack(ys, dim=1))
    windows = [0, 31, 63]
    want = oracle.stack_forward(s.x[windows], s.w_self, s.w_off, s.layers, True)[-1]
    err = row_rel_err(got[windows], want)
    log(f"  row err {err:.2e}")
    assert err <= TOL["bf16"]
    assert np.isfinite(got).all()
