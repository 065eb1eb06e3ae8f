"""hcmix_backward_no_alloc (the backward for callers that cannot allocate:
split-K partials in the library's own scratch array) against hcmix_backward
with a caller workspace, through the C ABI: bitwise equal, since both run the
same kernels in the same order.  Two calls in a row on one GPU, the second
with a smaller input, so that the second reuses the scratch the first left
behind; plus accumulation, the largest width the scratch holds, and the
refusal of a shape that needs more scratch than it has."""
import numpy as np
import pytest
import torch

from paper_2609_18145_amd import hcmix, inputs
from tests.util import to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hcmix.load()


def log(msg):
    print(msg, flush=True)


def both(batch, n, width, layer, causal, dtype, seed, accumulate=False):
    x, ws, wo, dy = (to_dev(a, dtype) for a in inputs.make_layer(batch, n, width, dtype, seed))
    dev = x.device
    outs = []
    for fn in ("workspace", "no_alloc"):
        dx = torch.full_like(x, float("nan"))
        g = torch.Generator(device="cpu").manual_seed(seed)
        init = torch.randn((2, width, width), generator=g).to(dev)
        dws, dwo = init[0].clone(), init[1].clone()
        if fn == "workspace":
            hcmix.backward(x, ws, wo, dy, layer, causal, dx=dx, dw_self=dws, dw_off=dwo,
                           accumulate=accumulate)
        else:
            hcmix.backward_no_alloc(x, ws, wo, dy, layer, causal, dx, dws, dwo,
                                    accumulate=accumulate)
        outs.append((dx, dws, dwo))
    torch.cuda.synchronize()
    for a, b in zip(*outs):
        assert torch.equal(a, b)
    assert not torch.isnan(outs[1][0].float()).any()


def test_two_calls_in_a_row_second_smaller():
    log("case: no-alloc backward, B=64 n=256 w=512 layer 7 causal bf16, then B=3 n=64 w=256 "
        "layer 2 bidir")
    both(64, 256, 512, 7, True, "bf16", seed=1)
    both(3, 64, 256, 2, False, "bf16", seed=2)


def test_accumulate_local_layer_and_fp32():
    log("case: no-alloc backward, accumulate; local layer; fp32")
    both(4, 256, 128, 3, True, "bf16", seed=3, accumulate=True)
    both(2, 128, 192, hcmix.LAYER_NEAR, True, "bf16", seed=4)
    both(2, 16, 32, 1, False, "f32", seed=5)


def test_largest_width_and_refusal_beyond_the_scratch():
    log("case: no-alloc backward at width 2048 (the largest the scratch holds)")
    both(1, 64, 2048, 5, True, "bf16", seed=6)
    log("case: width 2112 needs more scratch than the library holds: refused")
    w = 2112
    x = torch.zeros((1, 64, w), dtype=torch.bfloat16, device="cuda")
    m = torch.zeros((w, w), dtype=torch.bfloat16, device="cuda")
    g = torch.zeros((w, w), dtype=torch.float32, device="cuda")
    with pytest.raises(hcmix.HcmixError) as e:
        hcmix.backward_no_alloc(x, m, m, x, 0, True, torch.empty_like(x), g, g.clone())
    assert e.value.status == hcmix.HCMIX_ERR_UNSUPPORTED
