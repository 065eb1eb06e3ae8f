"""Channel-shared mixing stack (hcmix_shared_stack_forward / _backward)
against the CPU oracle oracle/shared_mix.py, through the C ABI: a bit-exact
partner probe for every stride, whole stacks (rotated, fixed, mixa, local) in
bf16 and fp32 with ragged channel slices, the workload's full shape (64
windows of 256 positions x 512 channels, 16 layers) with every output and
table gradient, accumulation and bitwise repeatability."""
import numpy as np
import pytest
import torch

import oracle
from oracle import shared_mix
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


def ftab(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def probe_codes(rows, width):
    x = np.zeros((rows, width), dtype=np.float32)
    for c in range(min(width, 15)):
        x[:, c] = (np.arange(rows) >> c) & 1
    return x


@pytest.mark.parametrize("n,width,dtype", [(2, 64, "bf16"), (16, 64, "bf16"), (256, 128, "bf16"),
                                           (64, 32, "f32"), (256, 96, "f32")])
@pytest.mark.parametrize("causal", [False, True])
def test_partner_probe_bit_exact(n, width, dtype, causal):
    """T[i][p(i)] = 1, T[i][i] = 0: every output row is its partner's code, or
    zero where the link is masked; dX sends each code back to the sender."""
    batch = 3
    log(f"case: shared probe B={batch} n={n} w={width} {dtype} causal={causal}")
    rows = batch * n
    codes = probe_codes(rows, width)
    x = to_dev(codes.reshape(batch, n, width), dtype)
    b = oracle.log2n(n)
    codes_list = list(range(b)) + ([oracle.NEAR] if causal else [])
    for layer in codes_list:
        t = np.zeros((n, n), dtype=np.float32)
        want = np.zeros_like(codes)
        want_dx = np.zeros_like(codes)
        for i in range(n):
            p = oracle.partner(i, layer, n)
            if oracle.receives(i, layer, n, causal):
                t[i, p] = 1.0
                for w in range(batch):
                    want[w * n + i] = codes[w * n + p]
                    want_dx[w * n + p] = codes[w * n + i]
        xs = hcmix.shared_stack_forward(x, [ftab(t)], [layer], causal)
        dx, dts = hcmix.shared_stack_backward(xs[:1], [ftab(t)], [layer], x, causal)
        torch.cuda.synchronize()
        assert np.array_equal(to_host(xs[1]).reshape(rows, width), want), f"layer {layer}"
        assert np.array_equal(to_host(dx).reshape(rows, width), want_dx), f"dX layer {layer}"


def run_and_check(s, tol=None, tol_dt=None):
    dt = s.dtype
    x = to_dev(s.x, dt)
    tabs = [ftab(t) for t in s.tables]
    xs = hcmix.shared_stack_forward(x, tabs, s.layers, s.causal)
    dx, dts = hcmix.shared_stack_backward(xs[:-1], tabs, s.layers, to_dev(s.dy, dt), s.causal)
    torch.cuda.synchronize()
    ref = shared_mix.stack_forward(s.x, s.tables, s.layers, s.causal)
    rdx, rdts = shared_mix.stack_backward(ref, s.tables, s.layers, s.dy, s.causal)
    tol = TOL[dt] if tol is None else tol
    tol_dt = tol if tol_dt is None else tol_dt
    e_y = row_rel_err(to_host(xs[-1]), ref[-1])
    e_dx = row_rel_err(to_host(dx), rdx)
    e_dt = max(fro_rel_err(to_host(g), r) for g, r in zip(dts, rdts))
    log(f"  y {e_y:.2e}  dx {e_dx:.2e}  dT {e_dt:.2e}")
    assert e_y <= tol and e_dx <= tol and e_dt <= tol_dt
    # off the links the table gradient is exactly zero
    for g, r in zip(dts, rdts):
        assert np.all(to_host(g)[r == 0] == 0)
    return x, tabs, xs, dx, dts


CASES = [
    (3, 16, 64, "rot", True, "bf16"), (2, 256, 128, "rot", True, "bf16"),
    (4, 64, 192, "fixed", True, "bf16"), (2, 64, 64, "mixa", True, "bf16"),
    (3, 32, 128, "rot", False, "bf16"), (2, 2, 64, "rot", True, "bf16"),
    (2, 16, 32, "rot", False, "f32"), (3, 128, 96, "mixa", True, "f32"),
    (1, 256, 64, "local", True, "bf16"),
]


@pytest.mark.parametrize("batch,n,width,schedule,causal,dtype", CASES)
def test_stack_against_oracle(batch, n, width, schedule, causal, dtype):
    L = {"rot": 2 * oracle.log2n(n), "fixed": 6, "local": 5}.get(schedule, 0)
    layers = {"rot": oracle.schedule_rot(L), "fixed": oracle.schedule_fixed(L, 1 % oracle.log2n(n)),
              "local": oracle.schedule_local(L)}.get(schedule) or oracle.schedule_mixa(n)
    log(f"case: shared stack B={batch} n={n} w={width} {schedule} L={len(layers)} "
        f"causal={causal} {dtype}")
    s = inputs.make_shared_stack(batch, n, width, len(layers), causal, dtype, seed=n + width,
                                 layers=layers)
    run_and_check(s)


def test_workload_shape_every_output_repeat_and_accumulate():
    """64 windows x 256 positions x 512 channels, 16 rotated causal layers (the
    bench's launch configuration): every output and table gradient against the
    oracle; a second backward is bitwise equal; accumulate adds."""
    s = inputs.make_shared_stack(64, 256, 512, 16, True, "bf16", kind="zipf_bytes", seed=0)
    log("case: shared stack workload shape B=64 n=256 w=512 L=16 causal bf16")
    x, tabs, xs, dx, dts = run_and_check(s)
    dy = to_dev(s.dy, "bf16")
    dx2, dts2 = hcmix.shared_stack_backward(xs[:-1], tabs, s.layers, dy, True)
    acc = [torch.ones_like(g) for g in dts]
    hcmix.shared_stack_backward(xs[:-1], tabs, s.layers, dy, True, dtables=acc, accumulate=True)
    torch.cuda.synchronize()
    assert torch.equal(dx, dx2)
    for a, b, c in zip(dts, dts2, acc):
        assert torch.equal(a, b)
        assert torch.equal(c, a + 1.0)
