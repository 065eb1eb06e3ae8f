"""The Python binding checks every operand (shape, dtype, contiguity, device)
before the library is called: the C ABI derives every buffer extent from the
sizes alone, so a short or mistyped tensor would otherwise be read or written
out of bounds on the GPU.  These run on the CPU: shapes and dtypes are
checked before the device, and a well-formed call on CPU tensors is refused
for not being on a GPU -- in every case before anything reaches the library."""
import pytest
import torch

from paper_2609_18145_amd import hcmix

bf, f32, i32 = torch.bfloat16, torch.float32, torch.int32


def z(*shape, dtype=bf):
    return torch.zeros(shape, dtype=dtype)


@pytest.fixture(autouse=True)
def _library_untouched(monkeypatch):
    """Any call that got past the checks would load the library: make that fail
    loudly instead, so a test can only pass by raising ValueError first."""
    def boom():
        raise AssertionError("the library was reached")
    monkeypatch.setattr(hcmix, "load", boom)


def refused(fn, *args, match=None, **kw):
    with pytest.raises(ValueError, match=match):
        fn(*args, **kw)


B, N, W = 2, 16, 64


def test_forward_checks():
    x, w = z(B, N, W), z(W, W)
    refused(hcmix.forward, x, z(W, W - 1), w, 0, True, match="w_self/w_off")
    refused(hcmix.forward, x, w, z(W, W, dtype=f32), 0, True, match="dtype")
    refused(hcmix.forward, x, w, w, 0, True, out=z(B, N, W - 8), match="out")
    refused(hcmix.forward, x, w, w, 0, True, out=z(B, N, W, dtype=f32), match="out")
    refused(hcmix.forward, z(B, N, W).transpose(1, 2).contiguous().transpose(1, 2), w, w, 0, True,
            match="contiguous")
    refused(hcmix.forward, z(B * N, W), w, w, 0, True, match="batch, n, width")
    refused(hcmix.forward, z(B, N, W, dtype=torch.float16), w, w, 0, True, match="dtype")
    refused(hcmix.forward, x, w, w, 0, True, match="GPU")      # well formed, but on the CPU


def test_backward_checks():
    x, w = z(B, N, W), z(W, W)
    refused(hcmix.backward, x, w, w, z(B, N - 1, W), 0, True, match="dy")
    refused(hcmix.backward, x, w, w, x, 0, True, dx=z(B, N, W, dtype=f32), match="dx")
    # caller-supplied weight gradients must be fp32 [width, width]
    refused(hcmix.backward, x, w, w, x, 0, True, dw_self=z(W, W), match="dw_self")
    refused(hcmix.backward, x, w, w, x, 0, True, dw_off=z(W, W // 2, dtype=f32), match="dw_off")
    refused(hcmix.backward, x, w, w, x, 0, True, match="GPU")


def test_stack_checks():
    L = 3
    x, w = z(B, N, W), z(W, W)
    ws = [w] * L
    refused(hcmix.stack_forward, x, ws[:2], ws, [0, 1, 2], True, match="w_selfs")
    refused(hcmix.stack_forward, x, ws, ws, [0, 1, 2], True, outs=[x, x], match="outs")
    refused(hcmix.stack_forward, x, ws, [w, w, z(W, W + 64)], [0, 1, 2], True, match="w_offs")
    refused(hcmix.stack_forward, x, ws, ws, [0, 1, 2], True, match="GPU")
    xs = [x] * L
    refused(hcmix.stack_backward, xs[:2], ws, ws, [0, 1, 2], x, True, match="xs")
    refused(hcmix.stack_backward, xs, ws, ws, [0, 1, 2], z(B, N, W, dtype=f32), True, match="dy")
    refused(hcmix.stack_backward, xs, ws, ws, [0, 1, 2], x, True, dws=[z(W, W)] * L, match="dws")
    refused(hcmix.stack_backward, xs, ws, ws, [0, 1, 2], x, True,
            dwo=[z(W, W, dtype=f32)] * 2, match="dwo")
    refused(hcmix.stack_backward, xs, ws, ws, [0, 1, 2], x, True, match="GPU")
    refused(hcmix.stack_backward_data, ws, ws, [0, 1, 2], x, True, grads=[x], match="grads")
    refused(hcmix.stack_backward_data, ws, ws, [0, 1, 2], x, True, dx=z(B, N, 2 * W), match="dx")
    refused(hcmix.stack_backward_data, ws, ws, [0, 1, 2], x, True, match="GPU")
    refused(hcmix.stack_weight_gradients, xs, [x, x, z(B, N, W + 64)], [0, 1, 2], True,
            match="dys")
    refused(hcmix.stack_weight_gradients, xs, xs, [0, 1, 2], True, dws=[z(W, W)] * L,
            match="dws")
    refused(hcmix.stack_weight_gradients, xs, xs, [0, 1, 2], True, match="GPU")


def test_attention_checks():
    H = 2
    qkv = z(B, N, 3, H, 64)
    refused(hcmix.attention_forward, z(B, N, 2, H, 64), match="qkv")
    refused(hcmix.attention_forward, z(B, N, 3, H, 64, dtype=f32), match="qkv")
    refused(hcmix.attention_forward, qkv, out=z(B, N, H, 32), match="out")
    refused(hcmix.attention_forward, qkv, lse=z(B, H, N), match="lse")          # bf16 lse
    refused(hcmix.attention_forward, qkv, match="GPU")
    out, lse, dout = z(B, N, H, 64), z(B, H, N, dtype=f32), z(B, N, H, 64)
    refused(hcmix.attention_backward, qkv, out, z(B, H, N - 1, dtype=f32), dout, match="lse")
    refused(hcmix.attention_backward, qkv, out, lse, z(B, N, H + 1, 64), match="dout")
    refused(hcmix.attention_backward, qkv, out, lse, dout, dqkv=z(B, N, 3, H, 32), match="dqkv")
    refused(hcmix.attention_backward, qkv, out, lse, dout, match="GPU")


def test_language_model_end_checks():
    V, rows = 32, B * N
    table, tokens = z(V, W), z(rows, dtype=i32)
    refused(hcmix.embedding_forward, table, z(rows, dtype=torch.int64), match="tokens")
    refused(hcmix.embedding_forward, table, tokens, out=z(rows - 1, W), match="out")
    refused(hcmix.embedding_forward, z(V, W, dtype=f32), tokens, match="table")
    refused(hcmix.embedding_forward, table, tokens, match="GPU")
    dx = z(rows, W)
    refused(hcmix.embedding_backward, tokens, z(rows + 1, W), V, match="dx")
    refused(hcmix.embedding_backward, tokens, dx, V, dtable=z(V, W), match="dtable")   # bf16
    refused(hcmix.embedding_backward, tokens, dx, V, dtable=z(V + 1, W, dtype=f32),
            match="dtable")
    refused(hcmix.embedding_backward, tokens, dx, V, match="GPU")
    x, w, bias, targets = z(rows, W), z(V, W), z(V, dtype=f32), z(rows, dtype=i32)
    ce = hcmix.head_cross_entropy
    refused(ce, z(rows - 1, W), w, bias, targets, 1.0, match="x")
    refused(ce, x, w, z(V), targets, 1.0, match="bias")
    refused(ce, x, w, bias, targets, 1.0, dlogits=z(rows, V, dtype=f32), match="dlogits")
    refused(ce, x, w, bias, targets, 1.0, loss=z(rows), match="loss")
    refused(ce, x, w, bias, targets, 1.0, dbias=z(V), match="dbias")
    refused(ce, x, w, bias, targets, 1.0, match="GPU")
    dl = z(rows, V)
    hb = hcmix.head_backward
    refused(hb, x, w, dl.to(f32), match="dlogits")
    refused(hb, z(rows, W + 64), w, dl, match="x")
    refused(hb, None, w, dl, match="x")                       # x is needed for dw
    refused(hb, x, w, dl, gx=z(rows, W, dtype=f32), match="gx")
    refused(hb, x, w, dl, dw=z(V, W), match="dw")             # dw must be fp32
    refused(hb, x, w, dl, with_gx=False, with_dw=False, match="neither")
    refused(hb, x, w, dl, match="GPU")
    refused(hb, None, w, dl, with_dw=False, match="GPU")      # gx alone needs no x


def test_decode_checks():
    L = 2
    x, w = z(B, W), z(W, W)
    cache = z(1024, dtype=torch.uint8)
    refused(hcmix.decode_step, z(B, 1, W), [w] * L, [w] * L, [0, 1], N, 0, cache, match="x")
    refused(hcmix.decode_step, x, [w], [w] * L, [0, 1], N, 0, cache, match="w_selfs")
    refused(hcmix.decode_step, x, [w] * L, [w] * L, [0, 1], N, 0, cache, out=z(B, W + 64),
            match="out")
    refused(hcmix.decode_step, x, [w] * L, [w] * L, [0, 1], N, 0, cache, match="GPU")


def test_shared_stack_checks():
    L, n = 2, N
    x = z(B, n, W)
    t = z(n, n, dtype=f32)
    refused(hcmix.shared_stack_forward, x, [t], [0, 1], True, match="tables")
    refused(hcmix.shared_stack_forward, x, [t, z(n, n)], [0, 1], True, match="tables")   # bf16
    refused(hcmix.shared_stack_forward, x, [t, z(n, n + 1, dtype=f32)], [0, 1], True,
            match="tables")
    refused(hcmix.shared_stack_forward, x, [t, t], [0, 1], True, outs=[x], match="outs")
    refused(hcmix.shared_stack_forward, x, [t, t], [0, 1], True, match="GPU")
    refused(hcmix.shared_stack_backward, [x, x], [t, t], [0, 1], z(B, n, W + 64), True,
            match="dy")
    refused(hcmix.shared_stack_backward, [x, x], [t, t], [0, 1], x, True,
            dtables=[t, z(n, n)], match="dtables")
    refused(hcmix.shared_stack_backward, [x, x], [t, t], [0, 1], x, True, match="GPU")


def test_workspace_must_be_gpu_memory():
    """A caller's workspace or cache reaches kernels as a raw pointer, so one in
    host memory is refused before the library is called."""
    with pytest.raises(ValueError, match="GPU memory"):
        hcmix._bytes(torch.zeros(64, dtype=torch.uint8))
    with pytest.raises(ValueError, match="contiguous"):
        hcmix._bytes(torch.zeros(8, 8, dtype=torch.uint8).t())
    assert hcmix._bytes(None) == 0
