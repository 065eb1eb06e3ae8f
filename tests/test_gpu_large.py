"""Maximum sizes: activations of more than 2^31 elements (16386 windows of 256
positions at width 512, 4.3 GB per bf16 tensor; for the attention core 8193
windows of Q, K and V for 8 heads; for the language model's ends 2^22 + 256
rows), so that every element offset past 2^31 goes through the kernels'
64-bit address arithmetic.

Forward and dX are compared with the oracle on whole windows (the first, a
middle one, the two on either side of element 2^31 and the last), each run
through the oracle on its own.  The weight gradients, sums over all 4.2
million rows, are checked by a property that holds at any size: they are
additive over windows (rows), so the library's gradient of the whole batch
must equal the sum of its gradients of two halves whose offsets all fit in
31 bits (and the halves' path is the one the oracle tests check at smaller
sizes).  The same holds for the channel-shared table gradients, the bias,
head and embedding gradients.  Inputs are seeded draws made on the device."""
import numpy as np
import pytest
import torch

import oracle
from oracle import attention, lm_head, shared_mix
from paper_2609_18145_amd import hcmix
from tests.util import TOL, fro_rel_err, row_rel_err, to_host

pytestmark = pytest.mark.gpu

B, N, W = 16386, 256, 512          # B * N * W = 2^31 + 2^18 elements
HALF = 8193                        # each half below 2^31 elements
WINDOWS = (0, 8191, 16383, 16384, 16385)   # window 16384 starts at element 2^31


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hcmix.load()


def log(msg):
    print(msg, flush=True)


def draw(shape, seed, scale=1.0):
    g = torch.Generator(device="cuda").manual_seed(seed)
    t = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    step = 1 << 28
    flat = t.view(-1)
    for i in range(0, flat.numel(), step):
        m = min(step, flat.numel() - i)
        flat[i:i + m] = (torch.randn(m, generator=g, device="cuda") * scale).to(torch.bfloat16)
    return t


def host_window(t, w):
    return to_host(t[w:w + 1])


def test_single_layer_beyond_2_31_elements():
    assert B * N * W > 2 ** 31 and HALF * N * W < 2 ** 31
    layer, causal = 7, True          # stride 128: partners across the tile halves
    log(f"case: single layer B={B} n={N} w={W} layer={layer} causal ({B * N * W} elements)")
    x = draw((B, N, W), 1)
    dy = draw((B, N, W), 2)
    ws = draw((W, W), 3, W ** -0.5)
    wo = draw((W, W), 4, W ** -0.5)
    y = hcmix.forward(x, ws, wo, layer, causal)
    dx, dws, dwo = hcmix.backward(x, ws, wo, dy, layer, causal)
    torch.cuda.synchronize()
    hws, hwo = to_host(ws), to_host(wo)
    for w in WINDOWS:
        xw, dyw = host_window(x, w), host_window(dy, w)
        ref = oracle.stack_forward(xw, [hws], [hwo], [layer], causal)
        rdx, _, _ = oracle.stack_backward(ref, [hws], [hwo], [layer], dyw, causal)
        e_y = row_rel_err(host_window(y, w), ref[-1])
        e_dx = row_rel_err(host_window(dx, w), rdx)
        log(f"  window {w}: y {e_y:.2e} dx {e_dx:.2e}")
        assert e_y <= TOL["bf16"] and e_dx <= TOL["bf16"]
    del y, dx
    # additivity of the weight gradients over windows
    _, s1, o1 = hcmix.backward(x[:HALF], ws, wo, dy[:HALF], layer, causal)
    _, s2, o2 = hcmix.backward(x[HALF:], ws, wo, dy[HALF:], layer, causal)
    torch.cuda.synchronize()
    e_s = fro_rel_err(to_host(dws), to_host(s1) + to_host(s2))
    e_o = fro_rel_err(to_host(dwo), to_host(o1) + to_host(o2))
    log(f"  dW additivity: self {e_s:.2e} off {e_o:.2e}")
    assert e_s <= 1e-5 and e_o <= 1e-5


def test_stack_beyond_2_31_elements():
    """Two causal layers through hcmix_stack_forward / _backward (the deferred
    path: dX chain, then one weight-gradient launch for both layers)."""
    layers, causal = [7, 0], True
    log(f"case: stack B={B} n={N} w={W} layers={layers} causal")
    x = draw((B, N, W), 11)
    dy = draw((B, N, W), 12)
    ws = [draw((W, W), 13 + i, W ** -0.5) for i in range(2)]
    wo = [draw((W, W), 15 + i, W ** -0.5) for i in range(2)]
    xs = hcmix.stack_forward(x, ws, wo, layers, causal)
    dx, dws, dwo = hcmix.stack_backward(xs, ws, wo, layers, dy, causal)
    torch.cuda.synchronize()
    hws, hwo = [to_host(w) for w in ws], [to_host(w) for w in wo]
    for w in WINDOWS:
        xw, dyw = host_window(x, w), host_window(dy, w)
        ref = oracle.stack_forward(xw, hws, hwo, layers, causal)
        rdx, _, _ = oracle.stack_backward(ref, hws, hwo, layers, dyw, causal)
        e_y = row_rel_err(host_window(xs[-1], w), ref[-1])
        e_dx = row_rel_err(host_window(dx, w), rdx)
        log(f"  window {w}: y {e_y:.2e} dx {e_dx:.2e}")
        assert e_y <= TOL["bf16"] and e_dx <= TOL["bf16"]
    del dx
    parts = []
    for sl in (slice(0, HALF), slice(HALF, B)):
        xh = [t[sl] for t in xs]
        _, a, b = hcmix.stack_backward(xh, ws, wo, layers, dy[sl], causal)
        parts.append((a, b))
    torch.cuda.synchronize()
    for l in range(2):
        e_s = fro_rel_err(to_host(dws[l]), to_host(parts[0][0][l]) + to_host(parts[1][0][l]))
        e_o = fro_rel_err(to_host(dwo[l]), to_host(parts[0][1][l]) + to_host(parts[1][1][l]))
        log(f"  layer {l} dW additivity: self {e_s:.2e} off {e_o:.2e}")
        assert e_s <= 1e-5 and e_o <= 1e-5


def test_shared_stack_beyond_2_31_elements():
    layers, causal = [7, 3], True
    log(f"case: channel-shared stack B={B} n={N} w={W} layers={layers} causal")
    x = draw((B, N, W), 21)
    dy = draw((B, N, W), 22)
    g = torch.Generator(device="cuda").manual_seed(23)
    tabs = [torch.randn(N, N, generator=g, device="cuda") * 0.5 ** 0.5 for _ in layers]
    xs = hcmix.shared_stack_forward(x, tabs, layers, causal)
    dx, dts = hcmix.shared_stack_backward(xs[:-1], tabs, layers, dy, causal)
    torch.cuda.synchronize()
    htabs = [t.double().cpu().numpy() for t in tabs]
    for w in WINDOWS:
        xw, dyw = host_window(x, w), host_window(dy, w)
        ref = shared_mix.stack_forward(xw, htabs, layers, causal)
        rdx, _ = shared_mix.stack_backward(ref, htabs, layers, dyw, causal)
        e_y = row_rel_err(host_window(xs[-1], w), ref[-1])
        e_dx = row_rel_err(host_window(dx, w), rdx)
        log(f"  window {w}: y {e_y:.2e} dx {e_dx:.2e}")
        assert e_y <= TOL["bf16"] and e_dx <= TOL["bf16"]
    del dx
    parts = []
    for sl in (slice(0, HALF), slice(HALF, B)):
        _, d = hcmix.shared_stack_backward([t[sl] for t in xs[:-1]], tabs, layers, dy[sl], causal)
        parts.append(d)
    torch.cuda.synchronize()
    for l in range(len(layers)):
        e = fro_rel_err(to_host(dts[l]), to_host(parts[0][l]) + to_host(parts[1][l]))
        log(f"  layer {l} dT additivity {e:.2e}")
        assert e <= 1e-5


def test_attention_beyond_2_31_elements():
    BA, H, HD = 8193, 8, 64        # qkv: 8193 * 256 * 3 * 8 * 64 > 2^31 elements
    per = N * 3 * H * HD
    wins = (0, (2 ** 31) // per, (2 ** 31) // per + 1, BA - 1)   # the second straddles 2^31
    log(f"case: attention B={BA} n={N} heads={H} ({BA * per} qkv elements)")
    qkv = draw((BA, N, 3, H, HD), 31)
    dout = draw((BA, N, H, HD), 32)
    out, lse = hcmix.attention_forward(qkv)
    dqkv = hcmix.attention_backward(qkv, out, lse, dout)
    torch.cuda.synchronize()
    for w in wins:
        q = to_host(qkv[w:w + 1])
        ro, rl = attention.forward(q)
        rd = attention.backward(q, to_host(dout[w:w + 1]))
        e_o = row_rel_err(to_host(out[w:w + 1]), ro)
        e_l = float(np.abs(to_host(lse[w:w + 1]) - rl).max())
        e_d = fro_rel_err(to_host(dqkv[w:w + 1]), rd)
        log(f"  window {w}: out {e_o:.2e} lse {e_l:.1e} dqkv {e_d:.2e}")
        assert e_o <= TOL["bf16"] and e_l <= 1e-4 and e_d <= TOL["bf16"]


def test_language_model_ends_beyond_2_31_elements():
    rows, V = 2 ** 22 + 256, 256    # x: rows * 512 > 2^31 elements
    half = rows // 2
    samples = (slice(0, 64), slice(2 ** 22 - 32, 2 ** 22 + 32), slice(rows - 64, rows))
    log(f"case: embedding, head and cross-entropy, rows={rows} width={W} vocab={V}")
    g = torch.Generator(device="cuda").manual_seed(41)
    tokens = torch.randint(0, V, (rows,), generator=g, device="cuda", dtype=torch.int32)
    targets = torch.randint(0, V, (rows,), generator=g, device="cuda", dtype=torch.int32)
    table = draw((V, W), 42)
    w = draw((V, W), 43, W ** -0.5)
    bias = torch.randn(V, generator=g, device="cuda")
    scale = 1.0 / rows
    x = hcmix.embedding_forward(table, tokens)
    loss, dl, db = hcmix.head_cross_entropy(x, w, bias, targets, scale, with_dbias=True)
    gx, dw = hcmix.head_backward(x, w, dl)
    dtab = hcmix.embedding_backward(tokens, gx, V)
    torch.cuda.synchronize()
    ht, hw, hb = to_host(table), to_host(w), bias.double().cpu().numpy()
    for sl in samples:
        tk, tg = tokens[sl].cpu().numpy(), targets[sl].cpu().numpy()
        rx = lm_head.embedding_forward(ht, tk)
        assert np.array_equal(to_host(x[sl]), rx)              # a gather: exact
        rloss, rdl = lm_head.head_cross_entropy(rx, hw, hb, tg, scale)
        e_l = float(np.abs(to_host(loss[sl]) - rloss).max() / np.abs(rloss).max())
        e_d = row_rel_err(to_host(dl[sl]), rdl)
        rgx, _ = lm_head.head_backward(rx, hw, rdl)
        e_g = row_rel_err(to_host(gx[sl]), rgx)
        log(f"  rows {sl.start}..{sl.stop}: loss {e_l:.1e} dlogits {e_d:.2e} gx {e_g:.2e}")
        assert e_l <= 1e-3 and e_d <= TOL["bf16"] and e_g <= TOL["bf16"]
    # the row sums (bias, head and embedding gradients) are additive over rows
    sums = []
    for sl in (slice(0, half), slice(half, rows)):
        _, _, b_h = hcmix.head_cross_entropy(x[sl], w, bias, targets[sl], scale, with_dbias=True)
        _, w_h = hcmix.head_backward(x[sl], w, dl[sl], with_gx=False)
        t_h = hcmix.embedding_backward(tokens[sl], gx[sl], V)
        sums.append((b_h, w_h, t_h))
    torch.cuda.synchronize()
    for name, full, a, b in (("dbias", db, sums[0][0], sums[1][0]),
                             ("head dW", dw, sums[0][1], sums[1][1]),
                             ("dtable", dtab, sums[0][2], sums[1][2])):
        e = fro_rel_err(to_host(full), to_host(a) + to_host(b))
        log(f"  {name} additivity {e:.2e}")
        assert e <= 1e-5
