"""The HIP field coupling (Section 3.4's dynamics variant) against the field
oracle (oracle/field.py), through the C ABI.

Inputs: fp32 coordinates and exact bf16 x and dy, the same numbers on both
sides.  Tolerances: y and dx (bf16 outputs of bf16 products whose couplings
are rounded to bf16, fp32 accumulation) by the row-relative bound of the bf16
path, 2e-2; the fp32 statistics and the coordinate gradient by what the
split-bf16 Gram product leaves (about 2^-17 of the squared norms of the
centred coordinates, amplified by the logits' size): row means 1e-4
relative, ln Z 2e-4 absolute, partners 1e-3 relative, dp 2e-3 as a Frobenius
ratio per window."""
import numpy as np
import pytest
import torch

from oracle import field
from paper_2609_18145_amd import hcmix, inputs
from tests.util import row_rel_err, to_dev, to_host

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hcmix.load()


def run(inp, want_partners=True):
    """Forward, then the backward twice: on the forward's workspace taking its
    coordinate tables (reuse_table), and on a fresh workspace building them;
    the two must agree bitwise."""
    p = torch.from_numpy(inp.p).cuda()
    x = to_dev(inp.x, "bf16")
    dy = to_dev(inp.dy, "bf16")
    batch, n, c = inp.p.shape
    ws = torch.empty(hcmix.field_workspace_bytes(batch, n, c), dtype=torch.uint8, device="cuda")
    y, m, lse, part = hcmix.field_forward(p, x, inp.tau, inp.scaled, partners=want_partners,
                                          workspace=ws)
    dp, dx = hcmix.field_backward(p, x, m, lse, dy, inp.tau, inp.scaled, workspace=ws,
                                  reuse_table=True)
    dp2, dx2 = hcmix.field_backward(p, x, m, lse, dy, inp.tau, inp.scaled)
    torch.cuda.synchronize()
    assert torch.equal(dp, dp2) and torch.equal(dx, dx2), "tables from the forward differ"
    return dict(y=to_host(y), m=to_host(m), lse=to_host(lse),
                part=to_host(part) if part is not None else None, dp=to_host(dp), dx=to_host(dx))


def reference(inp):
    y, _, eff = field.forward(inp.p, inp.x, inp.tau, inp.scaled)
    m, lse = field.row_stats(inp.p, inp.tau, inp.scaled)
    dp, dx = field.backward(inp.p, inp.x, inp.dy, inp.tau, inp.scaled)
    return dict(y=y, m=m, lse=lse, part=eff, dp=dp, dx=dx)


def dp_err(got, ref):
    worst = 0.0
    for b in range(ref.shape[0]):
        den = max(np.linalg.norm(ref[b]), 1e-30)
        worst = max(worst, np.linalg.norm(got[b] - ref[b]) / den)
    return worst


def check(got, ref, tag):
    ey, edx = row_rel_err(got["y"], ref["y"]), row_rel_err(got["dx"], ref["dx"])
    em = float(np.max(np.abs(got["m"] - ref["m"]) / np.maximum(np.abs(ref["m"]), 1e-30)))
    el = float(np.max(np.abs(got["lse"] - ref["lse"])))
    edp = dp_err(got["dp"], ref["dp"])
    msg = f"{tag}: y {ey:.2e} dx {edx:.2e} m {em:.2e} lse {el:.2e} dp {edp:.2e}"
    print(msg, flush=True)
    assert ey < TOL and edx < TOL, msg
    assert em < 1e-4 and el < 2e-4, msg
    assert edp < 2e-3, msg
    if got["part"] is not None:
        ep = float(np.max(np.abs(got["part"] - ref["part"]) / ref["part"]))
        assert ep < 1e-3, f"{msg} partners {ep:.2e}"


# (batch, n, width, coord_dim, tau, scaled, mean squared distance): every tile
# count, ragged windows, one and several 32-wide coordinate tiles, both forms,
# the saturated regime of Section 7 (unscaled, d^2 about 100, tau 1), an
# unscaled kernel with spread-out partners, and full 8-tile windows with the
# widest coordinates (64, and 61 padded to 64) and widths that are not a
# multiple of 128
CASES = [
    (2, 256, 128, 32, 1.0, True, 100.0),
    (2, 256, 64, 32, 1.0, False, 100.0),
    (3, 45, 64, 3, 0.7, True, 100.0),
    (2, 100, 128, 50, 1.3, True, 100.0),
    (1, 1, 64, 5, 1.0, True, 100.0),
    (2, 32, 64, 64, 0.5, True, 10.0),
    (2, 33, 192, 16, 2.0, False, 4.0),
    (1, 200, 512, 1, 1.0, True, 1.0),
    (2, 160, 64, 17, 1.0, True, 30.0),
    (2, 128, 128, 8, 1.0, False, 2.0),
    (1, 224, 256, 40, 0.25, False, 0.5),
    (2, 96, 64, 2, 3.0, True, 1e4),
    (2, 256, 192, 64, 1.0, True, 100.0),
    (1, 250, 128, 61, 0.8, False, 30.0),
]


@pytest.mark.parametrize("batch,n,width,c,tau,scaled,msd", CASES)
def test_field_matches_oracle(batch, n, width, c, tau, scaled, msd):
    print(f"case: field B={batch} n={n} width={width} c={c} tau={tau} scaled={scaled} "
          f"msd={msd}", flush=True)
    inp = inputs.make_field(batch, n, width, coord_dim=c, tau=tau, scaled=scaled,
                            mean_sq_dist=msd, seed=n + c)
    check(run(inp), reference(inp), f"n={n} c={c}")


def test_field_full_workload():
    """64 windows of 256 positions, width 512, 32 coordinates (Section 7's
    window), byte-token inputs: every window against the oracle."""
    print("case: field full workload B=64 n=256 width=512 c=32", flush=True)
    inp = inputs.make_field(64, 256, 512, coord_dim=32, kind="zipf_bytes", seed=11)
    check(run(inp), reference(inp), "full")


def test_equal_coordinates_give_prefix_means():
    print("case: field equal coordinates", flush=True)
    inp = inputs.make_field(2, 70, 64, coord_dim=4, seed=5)
    inp.p[:] = np.float32(3.25)
    got = run(inp)
    n = 70
    cum = np.cumsum(inp.x.astype(np.float64), axis=1) / np.arange(1, n + 1)[None, :, None]
    assert row_rel_err(got["y"], cum) < TOL
    assert np.all(got["m"] == 0)
    assert np.allclose(got["part"], np.arange(1, n + 1)[None, :], rtol=1e-5)
    assert np.all(got["dp"] == 0)


def test_offset_cluster_is_resolved():
    """Coordinates far from the origin with a small spread: distances are
    taken relative to the window's first position, so the couplings match."""
    print("case: field offset cluster", flush=True)
    inp = inputs.make_field(2, 128, 64, coord_dim=8, mean_sq_dist=2.0, seed=6)
    inp.p += np.float32(1000.0)
    for scaled in (True, False):
        inp.scaled = scaled
        check(run(inp), reference(inp), f"offset scaled={scaled}")


def test_deterministic_and_partners_optional():
    print("case: field determinism", flush=True)
    inp = inputs.make_field(2, 150, 128, coord_dim=24, seed=7)
    a, b = run(inp), run(inp, want_partners=False)
    for k in ("y", "m", "lse", "dp", "dx"):
        assert np.array_equal(a[k], b[k]), k
    assert b["part"] is None
