"""Python binding of libhcmix.so (ctypes; argument marshalling only).

Every step of the layer runs in the HIP library; PyTorch supplies device
memory and the current stream.  If the library is not built this module
raises on first use: there is no CPU or PyTorch fallback.

    y = forward(x, w_self, w_off, layer, causal)
    dx, dws, dwo = backward(x, w_self, w_off, dy, layer, causal)
    y = Stack.apply(x, layers, causal, *w_selfs, *w_offs)   # autograd over L layers
    y, m, lse, partners = field_forward(p, x, tau, scaled, workspace=ws)
    dp, dx = field_backward(p, x, m, lse, dy, tau, scaled, workspace=ws, reuse_table=True)
"""
from __future__ import annotations

import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhcmix.so")

HCMIX_OK, HCMIX_ERR_INVALID_VALUE, HCMIX_ERR_UNSUPPORTED, HCMIX_ERR_HIP = 0, 1, 2, 3
HCMIX_F32, HCMIX_BF16 = 0, 1
HCMIX_BIDIR, HCMIX_CAUSAL = 0, 1
# layer code of the local layer (Eq. (1) with jump 1; causal only); codes >= 0
# are hypercube layers
LAYER_NEAR = -1

# every symbol declared in include/hcmix.h
EXPORTS = ("hcmix_status_string", "hcmix_last_hip_error", "hcmix_dim", "hcmix_forward",
           "hcmix_backward_workspace_bytes", "hcmix_backward", "hcmix_stack_forward",
           "hcmix_stack_backward_workspace_bytes", "hcmix_stack_backward",
           "hcmix_stack_weight_gradients_workspace_bytes", "hcmix_stack_weight_gradients",
           "hcmix_stack_backward_data_workspace_bytes", "hcmix_stack_backward_data",
           "hcmix_decode_cache_bytes", "hcmix_decode_step", "hcmix_attention_forward",
           "hcmix_attention_backward", "hcmix_embedding_forward",
           "hcmix_embedding_backward_workspace_bytes", "hcmix_embedding_backward",
           "hcmix_head_cross_entropy_workspace_bytes", "hcmix_head_cross_entropy",
           "hcmix_head_backward_workspace_bytes", "hcmix_head_backward",
           "hcmix_backward_no_alloc", "hcmix_shared_stack_forward",
           "hcmix_shared_stack_backward_workspace_bytes", "hcmix_shared_stack_backward",
           "hcmix_linear_forward", "hcmix_linear_backward_workspace_bytes",
           "hcmix_linear_backward", "hcmix_field_forward", "hcmix_field_workspace_bytes",
           "hcmix_field_backward")

_lib = None


class HcmixError(RuntimeError):
    def __init__(self, status: int, what: str):
        lib = load()
        msg = lib.hcmix_status_string(status).decode()
        if status == HCMIX_ERR_HIP:
            msg += ": " + lib.hcmix_last_hip_error().decode()
        super().__init__(f"{what}: {msg}")
        self.status = status


def load():
    """Load libhcmix.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_18145_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        i64, i32, vp, sz = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t
        fp = ctypes.POINTER(ctypes.c_float)
        lib.hcmix_status_string.argtypes, lib.hcmix_status_string.restype = [i32], ctypes.c_char_p
        lib.hcmix_last_hip_error.argtypes, lib.hcmix_last_hip_error.restype = [], ctypes.c_char_p
        lib.hcmix_dim.argtypes, lib.hcmix_dim.restype = [i32, i64], i32
        lib.hcmix_forward.argtypes = [i64, i64, i64, i32, i32, i32, vp, vp, vp, vp, vp]
        lib.hcmix_forward.restype = i32
        lib.hcmix_backward_workspace_bytes.argtypes = [i64, i64, i64, i32]
        lib.hcmix_backward_workspace_bytes.restype = sz
        lib.hcmix_backward.argtypes = [i64, i64, i64, i32, i32, i32, vp, vp, vp, vp, vp, fp, fp,
                                       i32, vp, sz, vp]
        lib.hcmix_backward.restype = i32
        lib.hcmix_backward_no_alloc.argtypes = [i64, i64, i64, i32, i32, i32, vp, vp, vp, vp, vp,
                                                fp, fp, i32, vp]
        lib.hcmix_backward_no_alloc.restype = i32
        pp = ctypes.POINTER(ctypes.c_void_p)
        ip = ctypes.POINTER(ctypes.c_int32)
        lib.hcmix_stack_forward.argtypes = [i64, i64, i64, i32, ip, i32, i32, vp, pp, pp, pp, vp]
        lib.hcmix_stack_forward.restype = i32
        lib.hcmix_stack_backward_workspace_bytes.argtypes = [i64, i64, i64, i32, i32]
        lib.hcmix_stack_backward_workspace_bytes.restype = sz
        lib.hcmix_stack_backward.argtypes = [i64, i64, i64, i32, ip, i32, i32, pp, pp, pp, vp, vp,
                                             pp, pp, i32, vp, sz, vp]
        lib.hcmix_stack_backward.restype = i32
        lib.hcmix_stack_weight_gradients_workspace_bytes.argtypes = [i64, i64, i64, i32, i32]
        lib.hcmix_stack_weight_gradients_workspace_bytes.restype = sz
        lib.hcmix_stack_weight_gradients.argtypes = [i64, i64, i64, i32, ip, i32, i32, pp, pp, pp,
                                                     pp, i32, vp, sz, vp]
        lib.hcmix_stack_weight_gradients.restype = i32
        lib.hcmix_stack_backward_data_workspace_bytes.argtypes = [i64, i32, i32]
        lib.hcmix_stack_backward_data_workspace_bytes.restype = sz
        lib.hcmix_stack_backward_data.argtypes = [i64, i64, i64, i32, ip, i32, i32, pp, pp, vp, pp,
                                                  vp, vp, sz, vp]
        lib.hcmix_stack_backward_data.restype = i32
        lib.hcmix_attention_forward.argtypes = [i64, i64, i32, i32, vp, vp, fp, vp]
        lib.hcmix_attention_forward.restype = i32
        lib.hcmix_attention_backward.argtypes = [i64, i64, i32, i32, vp, vp, fp, vp, vp, vp]
        lib.hcmix_attention_backward.restype = i32
        lib.hcmix_field_forward.argtypes = [i64, i64, i64, i32, ctypes.c_float, i32, fp, vp, vp,
                                            fp, fp, fp, vp, sz, vp]
        lib.hcmix_field_forward.restype = i32
        lib.hcmix_field_workspace_bytes.argtypes = [i64, i64, i32]
        lib.hcmix_field_workspace_bytes.restype = sz
        lib.hcmix_field_backward.argtypes = [i64, i64, i64, i32, ctypes.c_float, i32, fp, vp, fp,
                                             fp, vp, fp, vp, i32, vp, sz, vp]
        lib.hcmix_field_backward.restype = i32
        lib.hcmix_embedding_forward.argtypes = [i64, i64, i32, vp, vp, vp, vp]
        lib.hcmix_embedding_forward.restype = i32
        lib.hcmix_embedding_backward_workspace_bytes.argtypes = [i64, i64, i32]
        lib.hcmix_embedding_backward_workspace_bytes.restype = sz
        lib.hcmix_embedding_backward.argtypes = [i64, i64, i32, vp, vp, fp, i32, vp, sz, vp]
        lib.hcmix_embedding_backward.restype = i32
        lib.hcmix_head_cross_entropy_workspace_bytes.argtypes = [i64, i32]
        lib.hcmix_head_cross_entropy_workspace_bytes.restype = sz
        lib.hcmix_head_cross_entropy.argtypes = [i64, i64, i32, vp, vp, fp, vp, ctypes.c_float,
                                                 fp, vp, fp, vp, sz, vp]
        lib.hcmix_head_cross_entropy.restype = i32
        lib.hcmix_head_backward_workspace_bytes.argtypes = [i64, i64, i32]
        lib.hcmix_head_backward_workspace_bytes.restype = sz
        lib.hcmix_head_backward.argtypes = [i64, i64, i32, vp, vp, vp, vp, fp, i32, vp, sz, vp]
        lib.hcmix_head_backward.restype = i32
        lib.hcmix_decode_cache_bytes.argtypes = [i64, i64, i64, i32, ip, i32]
        lib.hcmix_decode_cache_bytes.restype = sz
        lib.hcmix_decode_step.argtypes = [i64, i64, i64, i32, ip, i32, i64, vp, pp, pp, vp, sz, vp,
                                          vp]
        lib.hcmix_decode_step.restype = i32
        lib.hcmix_shared_stack_forward.argtypes = [i64, i64, i64, i32, ip, i32, i32, vp, pp, pp,
                                                   vp]
        lib.hcmix_shared_stack_forward.restype = i32
        lib.hcmix_shared_stack_backward_workspace_bytes.argtypes = [i64, i64, i64, i32, i32]
        lib.hcmix_shared_stack_backward_workspace_bytes.restype = sz
        lib.hcmix_shared_stack_backward.argtypes = [i64, i64, i64, i32, ip, i32, i32, pp, pp, vp,
                                                    vp, pp, i32, vp, sz, vp]
        lib.hcmix_shared_stack_backward.restype = i32
        lib.hcmix_linear_forward.argtypes = [i64, i64, i64, vp, vp, vp, vp]
        lib.hcmix_linear_forward.restype = i32
        lib.hcmix_linear_backward_workspace_bytes.argtypes = [i64, i64, i64]
        lib.hcmix_linear_backward_workspace_bytes.restype = sz
        lib.hcmix_linear_backward.argtypes = [i64, i64, i64, vp, vp, vp, vp, fp, i32, vp, sz, vp]
        lib.hcmix_linear_backward.restype = i32
        _lib = lib
    return _lib


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return HCMIX_BF16
    if t.dtype == torch.float32:
        return HCMIX_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _fptr(t):
    return ctypes.cast(ctypes.c_void_p(t.data_ptr()), ctypes.POINTER(ctypes.c_float))


def _need(t, name, shape, dtype, device=None):
    """Validate one operand before anything reaches the library: a tensor of
    exactly `shape` (None entries match any extent), of `dtype`, contiguous,
    and (once the device is known) on `device`.  Raises ValueError."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name}: expected a tensor, got {type(t).__name__}")
    if shape is not None:
        got = tuple(t.shape)
        if len(got) != len(shape) or any(e is not None and g != e for g, e in zip(got, shape)):
            raise ValueError(f"{name}: shape {got}, expected {tuple(shape)}")
    if t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if device is not None and t.device != device:
        raise ValueError(f"{name}: on {t.device}, expected {device}")


def _gpu(dev):
    """Every operand shares `dev` (checked per operand); it must be a GPU.
    Checked after the shapes and dtypes, before the library is touched."""
    if dev.type != "cuda":
        raise ValueError(f"hcmix works on GPU tensors only (got {dev})")


def _act_dtype(x, name="x"):
    if x.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError(f"{name}: dtype {x.dtype}, expected bfloat16 or float32")
    return x.dtype


def _bytes(t):
    """Byte extent of a workspace or cache tensor (any dtype, contiguous, in GPU
    memory: the library hands it to kernels as it is)."""
    if t is None:
        return 0
    if not isinstance(t, torch.Tensor) or not t.is_contiguous():
        raise ValueError("workspace/cache: expected a contiguous tensor")
    if t.device.type != "cuda":
        raise ValueError(f"workspace/cache: on {t.device}, expected GPU memory")
    return t.numel() * t.element_size()


def _stream(x):
    return ctypes.c_void_p(torch.cuda.current_stream(x.device).cuda_stream)


def dim(layer: int, n: int) -> int:
    return load().hcmix_dim(layer, n)


def _act_shape(x, name="x"):
    """[batch, n, width] of an activation tensor (checked to be 3-D)."""
    if not isinstance(x, torch.Tensor) or x.dim() != 3:
        raise ValueError(f"{name}: expected a [batch, n, width] tensor")
    return tuple(x.shape)


def _weights(ws, name, width, dtype, dev, count=None):
    if count is not None and len(ws) != count:
        raise ValueError(f"{name}: {len(ws)} matrices, expected {count}")
    for k, w in enumerate(ws):
        _need(w, f"{name}[{k}]", (width, width), dtype, dev)


def forward(x: torch.Tensor, w_self: torch.Tensor, w_off: torch.Tensor, layer: int,
            causal: bool, out: torch.Tensor | None = None) -> torch.Tensor:
    """y = W_self x_i + m(i) W_off x_(i xor 2^d) over x of shape [batch, n, width]."""
    batch, n, width = _act_shape(x)
    dt = _act_dtype(x)
    _need(x, "x", None, dt)
    dev = x.device
    _weights([w_self, w_off], "w_self/w_off", width, dt, dev)
    if out is None:
        out = torch.empty_like(x)
    _need(out, "out", (batch, n, width), dt, dev)
    _gpu(dev)
    rc = load().hcmix_forward(batch, n, width, layer, int(bool(causal)), _dtype_code(x),
                              _ptr(x), _ptr(w_self), _ptr(w_off), _ptr(out), _stream(x))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_forward")
    return out


def workspace_bytes(batch: int, n: int, width: int, dtype: torch.dtype) -> int:
    code = HCMIX_BF16 if dtype == torch.bfloat16 else HCMIX_F32
    return load().hcmix_backward_workspace_bytes(batch, n, width, code)


def alloc_workspace(batch, n, width, dtype, device) -> torch.Tensor | None:
    nbytes = workspace_bytes(batch, n, width, dtype)
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def _grad_out(t, name, width, dev, shape=None):
    """A caller-supplied fp32 weight-gradient buffer ([width, width] unless given)."""
    _need(t, name, shape or (width, width), torch.float32, dev)


def backward(x, w_self, w_off, dy, layer: int, causal: bool, dx=None, dw_self=None,
             dw_off=None, accumulate: bool = False, workspace=None):
    """Adjoint of ``forward``: returns (dx, dw_self, dw_off); dw_* are fp32."""
    batch, n, width = _act_shape(x)
    dt = _act_dtype(x)
    _need(x, "x", None, dt)
    dev = x.device
    _weights([w_self, w_off], "w_self/w_off", width, dt, dev)
    _need(dy, "dy", (batch, n, width), dt, dev)
    if dx is None:
        dx = torch.empty_like(x)
    _need(dx, "dx", (batch, n, width), dt, dev)
    if dw_self is None:
        dw_self = torch.empty((width, width), dtype=torch.float32, device=dev)
    if dw_off is None:
        dw_off = torch.empty((width, width), dtype=torch.float32, device=dev)
    _grad_out(dw_self, "dw_self", width, dev)
    _grad_out(dw_off, "dw_off", width, dev)
    _gpu(dev)
    if workspace is None:
        workspace = alloc_workspace(batch, n, width, x.dtype, dev)
    rc = load().hcmix_backward(batch, n, width, layer, int(bool(causal)), _dtype_code(x),
                               _ptr(x), _ptr(w_self), _ptr(w_off), _ptr(dy), _ptr(dx),
                               _fptr(dw_self), _fptr(dw_off), int(bool(accumulate)),
                               _ptr(workspace), _bytes(workspace), _stream(x))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_backward")
    return dx, dw_self, dw_off


def backward_no_alloc(x, w_self, w_off, dy, layer: int, causal: bool, dx, dw_self, dw_off,
                      accumulate: bool = False):
    """``backward`` for callers that cannot allocate: every output is the
    caller's, and the split-K partials live in the library's own scratch array
    (hcmix_backward_no_alloc); calls that overlap on one GPU race."""
    batch, n, width = _act_shape(x)
    dt = _act_dtype(x)
    _need(x, "x", None, dt)
    dev = x.device
    _weights([w_self, w_off], "w_self/w_off", width, dt, dev)
    _need(dy, "dy", (batch, n, width), dt, dev)
    _need(dx, "dx", (batch, n, width), dt, dev)
    _grad_out(dw_self, "dw_self", width, dev)
    _grad_out(dw_off, "dw_off", width, dev)
    _gpu(dev)
    rc = load().hcmix_backward_no_alloc(batch, n, width, layer, int(bool(causal)),
                                        _dtype_code(x), _ptr(x), _ptr(w_self), _ptr(w_off),
                                        _ptr(dy), _ptr(dx), _fptr(dw_self), _fptr(dw_off),
                                        int(bool(accumulate)), _stream(x))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_backward_no_alloc")
    return dx, dw_self, dw_off


def _ptrs(ts):
    return (ctypes.c_void_p * len(ts))(*[t.data_ptr() for t in ts])


def _layers(layers):
    return (ctypes.c_int32 * len(layers))(*[int(v) for v in layers])


def _acts(ts, name, shape, dt, dev, count):
    if len(ts) < count:
        raise ValueError(f"{name}: {len(ts)} tensors, expected {count}")
    for k in range(count):
        _need(ts[k], f"{name}[{k}]", shape, dt, dev)


def stack_forward(x, w_selfs, w_offs, layers, causal, outs=None):
    """Run the layers in order in one library call; returns [x_0, x_1, ..., x_L]."""
    L = len(layers)
    shape = _act_shape(x)
    batch, n, width = shape
    dt = _act_dtype(x)
    _need(x, "x", None, dt)
    dev = x.device
    _weights(w_selfs, "w_selfs", width, dt, dev, L)
    _weights(w_offs, "w_offs", width, dt, dev, L)
    if outs is None:
        outs = [torch.empty_like(x) for _ in range(L)]
    _acts(outs, "outs", shape, dt, dev, L)
    _gpu(dev)
    rc = load().hcmix_stack_forward(batch, n, width, L, _layers(layers), int(bool(causal)),
                                    _dtype_code(x), _ptr(x), _ptrs(w_selfs), _ptrs(w_offs),
                                    _ptrs(outs[:L]), _stream(x))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_stack_forward")
    return [x, *outs[:L]]


def stack_workspace_bytes(batch, n, width, num_layers, dtype) -> int:
    code = HCMIX_BF16 if dtype == torch.bfloat16 else HCMIX_F32
    return load().hcmix_stack_backward_workspace_bytes(batch, n, width, num_layers, code)


def alloc_stack_workspace(batch, n, width, num_layers, dtype, device):
    nbytes = stack_workspace_bytes(batch, n, width, num_layers, dtype)
    return None if nbytes == 0 else torch.empty(nbytes, dtype=torch.uint8, device=device)


def stack_backward(xs, w_selfs, w_offs, layers, dy, causal, dx=None, dws=None, dwo=None,
                   accumulate=False, workspace=None):
    """Backward through the stack in one library call, using the saved layer
    inputs xs[0..L-1]; returns (dx_0, [dW_self], [dW_off])."""
    L = len(layers)
    x0 = xs[0]
    shape = _act_shape(x0, "xs[0]")
    batch, n, width = shape
    dt = _act_dtype(x0, "xs[0]")
    dev = x0.device
    _acts(xs, "xs", shape, dt, dev, L)
    _weights(w_selfs, "w_selfs", width, dt, dev, L)
    _weights(w_offs, "w_offs", width, dt, dev, L)
    _need(dy, "dy", shape, dt, dev)
    if dx is None:
        dx = torch.empty_like(x0)
    _need(dx, "dx", shape, dt, dev)
    if dws is None:
        dws = [torch.empty((width, width), dtype=torch.float32, device=dev) for _ in range(L)]
    if dwo is None:
        dwo = [torch.empty((width, width), dtype=torch.float32, device=dev) for _ in range(L)]
    _acts(dws, "dws", (width, width), torch.float32, dev, L)
    _acts(dwo, "dwo", (width, width), torch.float32, dev, L)
    _gpu(dev)
    if workspace is None:
        workspace = alloc_stack_workspace(batch, n, width, L, x0.dtype, dev)
    rc = load().hcmix_stack_backward(batch, n, width, L, _layers(layers), int(bool(causal)),
                                     _dtype_code(x0), _ptrs(xs[:L]), _ptrs(w_selfs), _ptrs(w_offs),
                                     _ptr(dy), _ptr(dx), _ptrs(dws[:L]), _ptrs(dwo[:L]),
                                     int(bool(accumulate)), _ptr(workspace), _bytes(workspace),
                                     _stream(x0))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_stack_backward")
    return dx, dws, dwo


def stack_backward_data(w_selfs, w_offs, layers, dy, causal, dx=None, grads=None,
                        workspace=None):
    """The dX chain of the stack alone (no weight gradients); returns
    (dx_0, [g_1, ..., g_{L-1}]) with g_l the gradient of layer l's input, so
    that layer l's output gradient is grads[l] (dy for the last layer)."""
    L = len(layers)
    shape = _act_shape(dy, "dy")
    batch, n, width = shape
    dt = _act_dtype(dy, "dy")
    _need(dy, "dy", None, dt)
    dev = dy.device
    _weights(w_selfs, "w_selfs", width, dt, dev, L)
    _weights(w_offs, "w_offs", width, dt, dev, L)
    if dx is None:
        dx = torch.empty_like(dy)
    if grads is None:
        grads = [torch.empty_like(dy) for _ in range(L - 1)]
    _need(dx, "dx", shape, dt, dev)
    _acts(grads, "grads", shape, dt, dev, L - 1)
    _gpu(dev)
    nbytes = load().hcmix_stack_backward_data_workspace_bytes(width, L, _dtype_code(dy))
    if workspace is None and nbytes:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    gp = _ptrs(grads[:L - 1]) if L > 1 else None
    rc = load().hcmix_stack_backward_data(batch, n, width, L, _layers(layers), int(bool(causal)),
                                          _dtype_code(dy), _ptrs(w_selfs), _ptrs(w_offs), _ptr(dy),
                                          gp, _ptr(dx), _ptr(workspace), _bytes(workspace),
                                          _stream(dy))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_stack_backward_data")
    return dx, grads


def weight_gradients_workspace_bytes(batch, n, width, num_layers, dtype) -> int:
    code = HCMIX_BF16 if dtype == torch.bfloat16 else HCMIX_F32
    return load().hcmix_stack_weight_gradients_workspace_bytes(batch, n, width, num_layers, code)


def stack_weight_gradients(xs, dys, layers, causal, dws=None, dwo=None, accumulate=False,
                           workspace=None):
    """Weight gradients of every layer from its input xs[l] and the gradient of
    its output dys[l], in one library call; returns ([dW_self], [dW_off])."""
    L = len(layers)
    x0 = xs[0]
    shape = _act_shape(x0, "xs[0]")
    batch, n, width = shape
    dt = _act_dtype(x0, "xs[0]")
    dev = x0.device
    _acts(xs, "xs", shape, dt, dev, L)
    _acts(dys, "dys", shape, dt, dev, L)
    if dws is None:
        dws = [torch.empty((width, width), dtype=torch.float32, device=dev) for _ in range(L)]
    if dwo is None:
        dwo = [torch.empty((width, width), dtype=torch.float32, device=dev) for _ in range(L)]
    _acts(dws, "dws", (width, width), torch.float32, dev, L)
    _acts(dwo, "dwo", (width, width), torch.float32, dev, L)
    _gpu(dev)
    if workspace is None:
        nbytes = weight_gradients_workspace_bytes(batch, n, width, L, x0.dtype)
        workspace = (torch.empty(nbytes, dtype=torch.uint8, device=dev) if nbytes
                     else None)
    rc = load().hcmix_stack_weight_gradients(batch, n, width, L, _layers(layers),
                                             int(bool(causal)), _dtype_code(x0), _ptrs(xs[:L]),
                                             _ptrs(dys[:L]), _ptrs(dws[:L]), _ptrs(dwo[:L]),
                                             int(bool(accumulate)), _ptr(workspace),
                                             _bytes(workspace), _stream(x0))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_stack_weight_gradients")
    return dws, dwo


def _qkv_shape(qkv):
    if not isinstance(qkv, torch.Tensor) or qkv.dim() != 5 or qkv.shape[2] != 3:
        raise ValueError("qkv: expected a [batch, n, 3, heads, head_dim] tensor")
    batch, n, _, heads, hd = qkv.shape
    return batch, n, heads, hd


def attention_forward(qkv, out=None, lse=None):
    """Causal multi-head attention core: qkv [batch, n, 3, heads, 64] bf16 ->
    (out [batch, n, heads, 64] bf16, lse [batch, heads, n] fp32)."""
    batch, n, heads, hd = _qkv_shape(qkv)
    _need(qkv, "qkv", None, torch.bfloat16)
    dev = qkv.device
    if out is None:
        out = torch.empty((batch, n, heads, hd), dtype=qkv.dtype, device=dev)
    if lse is None:
        lse = torch.empty((batch, heads, n), dtype=torch.float32, device=dev)
    _need(out, "out", (batch, n, heads, hd), torch.bfloat16, dev)
    _need(lse, "lse", (batch, heads, n), torch.float32, dev)
    _gpu(dev)
    rc = load().hcmix_attention_forward(batch, n, heads, hd, _ptr(qkv), _ptr(out), _fptr(lse),
                                        _stream(qkv))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_attention_forward")
    return out, lse


def attention_backward(qkv, out, lse, dout, dqkv=None):
    """Gradient of qkv ([batch, n, 3, heads, 64]) given dout = dL/dout."""
    batch, n, heads, hd = _qkv_shape(qkv)
    _need(qkv, "qkv", None, torch.bfloat16)
    dev = qkv.device
    _need(out, "out", (batch, n, heads, hd), torch.bfloat16, dev)
    _need(lse, "lse", (batch, heads, n), torch.float32, dev)
    _need(dout, "dout", (batch, n, heads, hd), torch.bfloat16, dev)
    if dqkv is None:
        dqkv = torch.empty_like(qkv)
    _need(dqkv, "dqkv", tuple(qkv.shape), torch.bfloat16, dev)
    _gpu(dev)
    rc = load().hcmix_attention_backward(batch, n, heads, hd, _ptr(qkv), _ptr(out), _fptr(lse),
                                         _ptr(dout), _ptr(dqkv), _stream(qkv))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_attention_backward")
    return dqkv


def _field_shapes(p, x):
    if not isinstance(p, torch.Tensor) or p.dim() != 3:
        raise ValueError("p: expected a [batch, n, coord_dim] tensor")
    batch, n, width = _act_shape(x)
    if tuple(p.shape[:2]) != (batch, n):
        raise ValueError(f"p: shape {tuple(p.shape)} does not match x {tuple(x.shape)}")
    _need(p, "p", None, torch.float32)
    _need(x, "x", None, torch.bfloat16, p.device)
    return batch, n, width, p.shape[2]


def field_workspace_bytes(batch: int, n: int, coord_dim: int) -> int:
    return load().hcmix_field_workspace_bytes(batch, n, coord_dim)


def _field_workspace(workspace, batch, n, c, dev):
    if workspace is None:
        need = field_workspace_bytes(batch, n, c)
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    return workspace


def field_forward(p, x, tau=1.0, scaled=True, partners=False, y=None, row_mean=None, lse=None,
                  workspace=None):
    """Field coupling (Section 3.4): p [batch, n, c] fp32 coordinates, x
    [batch, n, width] bf16 -> (y bf16, row_mean fp32 [batch, n], lse fp32
    [batch, n], partners fp32 [batch, n] or None)."""
    batch, n, width, c = _field_shapes(p, x)
    dev = x.device
    if y is None:
        y = torch.empty_like(x)
    if row_mean is None:
        row_mean = torch.empty((batch, n), dtype=torch.float32, device=dev)
    if lse is None:
        lse = torch.empty((batch, n), dtype=torch.float32, device=dev)
    part = torch.empty((batch, n), dtype=torch.float32, device=dev) if partners else None
    _need(y, "y", (batch, n, width), torch.bfloat16, dev)
    _need(row_mean, "row_mean", (batch, n), torch.float32, dev)
    _need(lse, "lse", (batch, n), torch.float32, dev)
    _gpu(dev)
    workspace = _field_workspace(workspace, batch, n, c, dev)
    rc = load().hcmix_field_forward(batch, n, width, c, float(tau), int(bool(scaled)), _fptr(p),
                                    _ptr(x), _ptr(y), _fptr(row_mean), _fptr(lse),
                                    _fptr(part) if part is not None else None, _ptr(workspace),
                                    _bytes(workspace), _stream(x))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_field_forward")
    return y, row_mean, lse, part


def field_backward(p, x, row_mean, lse, dy, tau=1.0, scaled=True, dp=None, dx=None,
                   workspace=None, reuse_table=False):
    """(dp fp32 [batch, n, c], dx bf16 [batch, n, width]) given dy = dL/dy and
    the forward's row_mean and lse.  reuse_table: `workspace` is the one the
    forward of these same coordinates used, untouched since, and its
    coordinate tables are taken as they are."""
    batch, n, width, c = _field_shapes(p, x)
    if reuse_table and workspace is None:
        raise ValueError("reuse_table needs the workspace the forward wrote its tables to")
    dev = x.device
    _need(row_mean, "row_mean", (batch, n), torch.float32, dev)
    _need(lse, "lse", (batch, n), torch.float32, dev)
    _need(dy, "dy", (batch, n, width), torch.bfloat16, dev)
    if dp is None:
        dp = torch.empty_like(p)
    if dx is None:
        dx = torch.empty_like(x)
    _need(dp, "dp", tuple(p.shape), torch.float32, dev)
    _need(dx, "dx", (batch, n, width), torch.bfloat16, dev)
    _gpu(dev)
    workspace = _field_workspace(workspace, batch, n, c, dev)
    rc = load().hcmix_field_backward(batch, n, width, c, float(tau), int(bool(scaled)), _fptr(p),
                                     _ptr(x), _fptr(row_mean), _fptr(lse), _ptr(dy), _fptr(dp),
                                     _ptr(dx), int(bool(reuse_table)), _ptr(workspace),
                                     _bytes(workspace), _stream(x))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_field_backward")
    return dp, dx


def _rows_of(t, name, width, dtype, dev):
    """A [..., width] tensor of `dtype`; returns its number of rows."""
    if not isinstance(t, torch.Tensor) or t.dim() < 1 or t.shape[-1] != width:
        raise ValueError(f"{name}: expected a [..., {width}] tensor")
    _need(t, name, None, dtype, dev)
    return t.numel() // width


def embedding_forward(table, tokens, out=None):
    """x[r] = table[tokens[r]]: table [vocab, width] bf16, tokens int32 (any shape)."""
    if not isinstance(table, torch.Tensor) or table.dim() != 2:
        raise ValueError("table: expected a [vocab, width] tensor")
    vocab, width = table.shape
    _need(table, "table", None, torch.bfloat16)
    dev = table.device
    _need(tokens, "tokens", None, torch.int32, dev)
    rows = tokens.numel()
    if out is None:
        out = torch.empty((*tokens.shape, width), dtype=table.dtype, device=dev)
    if _rows_of(out, "out", width, torch.bfloat16, dev) != rows:
        raise ValueError(f"out: {out.numel() // width} rows, expected {rows}")
    _gpu(dev)
    rc = load().hcmix_embedding_forward(rows, width, vocab, _ptr(table), _ptr(tokens), _ptr(out),
                                        _stream(table))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_embedding_forward")
    return out


def embedding_backward(tokens, dx, vocab, dtable=None, accumulate=False, workspace=None):
    """dtable[v] (+)= sum of dx rows whose token is v (fp32 [vocab, width])."""
    if not isinstance(dx, torch.Tensor) or dx.dim() < 1:
        raise ValueError("dx: expected a [..., width] tensor")
    width = dx.shape[-1]
    _need(dx, "dx", None, torch.bfloat16)
    dev = dx.device
    _need(tokens, "tokens", None, torch.int32, dev)
    rows = tokens.numel()
    if _rows_of(dx, "dx", width, torch.bfloat16, dev) != rows:
        raise ValueError(f"dx: {dx.numel() // width} rows, expected {rows} (one per token)")
    if dtable is None:
        dtable = torch.empty((vocab, width), dtype=torch.float32, device=dev)
    _need(dtable, "dtable", (vocab, width), torch.float32, dev)
    _gpu(dev)
    nbytes = load().hcmix_embedding_backward_workspace_bytes(rows, width, vocab)
    if workspace is None:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    rc = load().hcmix_embedding_backward(rows, width, vocab, _ptr(tokens), _ptr(dx), _fptr(dtable),
                                         int(bool(accumulate)), _ptr(workspace),
                                         _bytes(workspace), _stream(dx))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_embedding_backward")
    return dtable


def head_cross_entropy(x, w, bias, targets, scale, loss=None, dlogits=None, dbias=None,
                       with_dbias=False, workspace=None):
    """Per-row loss (fp32 [rows]) and scale * (softmax - onehot) (bf16 [rows, vocab]);
    with with_dbias (or a dbias buffer), also the bias gradient (fp32 [vocab]):
    returns (loss, dlogits) or (loss, dlogits, dbias)."""
    if not isinstance(w, torch.Tensor) or w.dim() != 2:
        raise ValueError("w: expected a [vocab, width] tensor")
    vocab, width = w.shape
    _need(w, "w", None, torch.bfloat16)
    dev = w.device
    _need(targets, "targets", None, torch.int32, dev)
    rows = targets.numel()
    _need(x, "x", (rows, width), torch.bfloat16, dev)
    _need(bias, "bias", (vocab,), torch.float32, dev)
    if loss is None:
        loss = torch.empty(rows, dtype=torch.float32, device=dev)
    if dlogits is None:
        dlogits = torch.empty((rows, vocab), dtype=x.dtype, device=dev)
    _need(loss, "loss", (rows,), torch.float32, dev)
    _need(dlogits, "dlogits", (rows, vocab), torch.bfloat16, dev)
    want_db = with_dbias or dbias is not None
    if want_db:
        if dbias is None:
            dbias = torch.empty(vocab, dtype=torch.float32, device=dev)
        _need(dbias, "dbias", (vocab,), torch.float32, dev)
    _gpu(dev)
    if want_db and workspace is None:
        workspace = torch.empty(load().hcmix_head_cross_entropy_workspace_bytes(rows, vocab),
                                dtype=torch.uint8, device=dev)
    rc = load().hcmix_head_cross_entropy(rows, width, vocab, _ptr(x), _ptr(w), _fptr(bias),
                                         _ptr(targets), float(scale), _fptr(loss), _ptr(dlogits),
                                         _fptr(dbias) if want_db else None,
                                         _ptr(workspace) if want_db else None,
                                         _bytes(workspace) if want_db else 0, _stream(x))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_head_cross_entropy")
    return (loss, dlogits, dbias) if want_db else (loss, dlogits)


def head_backward(x, w, dlogits, gx=None, dw=None, with_gx=True, with_dw=True,
                  accumulate=False, workspace=None):
    """The head's input gradient dlogits W (bf16 [rows, width]) and weight
    gradient dlogits^T x (fp32 [vocab, width], added to dw with accumulate):
    returns (gx, dw), None for one not asked for.  x is only read for dw (it
    may be None without it)."""
    if not isinstance(w, torch.Tensor) or w.dim() != 2:
        raise ValueError("w: expected a [vocab, width] tensor")
    vocab, width = w.shape
    _need(w, "w", None, torch.bfloat16)
    dev = w.device
    if not isinstance(dlogits, torch.Tensor) or dlogits.dim() != 2:
        raise ValueError("dlogits: expected a [rows, vocab] tensor")
    rows = dlogits.shape[0]
    _need(dlogits, "dlogits", (rows, vocab), torch.bfloat16, dev)
    want_gx = with_gx or gx is not None
    want_dw = with_dw or dw is not None
    if not want_gx and not want_dw:
        raise ValueError("head_backward: neither gx nor dw asked for")
    if want_dw:
        _need(x, "x", (rows, width), torch.bfloat16, dev)
    if want_gx:
        if gx is None:
            gx = torch.empty((rows, width), dtype=dlogits.dtype, device=dev)
        _need(gx, "gx", (rows, width), torch.bfloat16, dev)
    if want_dw:
        if dw is None:
            dw = torch.empty((vocab, width), dtype=torch.float32, device=dev)
        _need(dw, "dw", (vocab, width), torch.float32, dev)
    _gpu(dev)
    if want_dw and workspace is None:
        workspace = torch.empty(load().hcmix_head_backward_workspace_bytes(rows, width, vocab),
                                dtype=torch.uint8, device=dev)
    rc = load().hcmix_head_backward(rows, width, vocab, _ptr(x) if want_dw else None, _ptr(w),
                                    _ptr(dlogits), _ptr(gx) if want_gx else None,
                                    _fptr(dw) if want_dw else None, int(bool(accumulate)),
                                    _ptr(workspace) if want_dw else None,
                                    _bytes(workspace) if want_dw else 0, _stream(dlogits))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_head_backward")
    return (gx if want_gx else None), (dw if want_dw else None)


def _tables(ts, name, n, dev, count):
    if len(ts) < count:
        raise ValueError(f"{name}: {len(ts)} tables, expected {count}")
    for k in range(count):
        _need(ts[k], f"{name}[{k}]", (n, n), torch.float32, dev)


def shared_stack_forward(x, tables, layers, causal, outs=None):
    """Channel-shared stack: y_i = T[i][i] x_i + m(i) T[i][p(i)] x_p(i) per
    layer, tables fp32 [n, n]; returns [x_0, x_1, ..., x_L]."""
    L = len(layers)
    shape = _act_shape(x)
    batch, n, width = shape
    dt = _act_dtype(x)
    _need(x, "x", None, dt)
    dev = x.device
    _tables(tables, "tables", n, dev, L)
    if outs is None:
        outs = [torch.empty_like(x) for _ in range(L)]
    _acts(outs, "outs", shape, dt, dev, L)
    _gpu(dev)
    rc = load().hcmix_shared_stack_forward(batch, n, width, L, _layers(layers), int(bool(causal)),
                                           _dtype_code(x), _ptr(x), _ptrs(tables[:L]),
                                           _ptrs(outs[:L]), _stream(x))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_shared_stack_forward")
    return [x, *outs[:L]]


def shared_stack_backward(xs, tables, layers, dy, causal, dx=None, dtables=None,
                          accumulate=False, workspace=None):
    """Backward of ``shared_stack_forward`` from the saved inputs xs[0..L-1]:
    returns (dx, [dT_l]) with dT_l fp32 [n, n] (zero off the layer's links)."""
    L = len(layers)
    x0 = xs[0]
    shape = _act_shape(x0, "xs[0]")
    batch, n, width = shape
    dt = _act_dtype(x0, "xs[0]")
    dev = x0.device
    _acts(xs, "xs", shape, dt, dev, L)
    _tables(tables, "tables", n, dev, L)
    _need(dy, "dy", shape, dt, dev)
    if dx is None:
        dx = torch.empty_like(x0)
    _need(dx, "dx", shape, dt, dev)
    if dtables is None:
        dtables = [torch.empty((n, n), dtype=torch.float32, device=dev) for _ in range(L)]
    _tables(dtables, "dtables", n, dev, L)
    _gpu(dev)
    if workspace is None:
        nbytes = load().hcmix_shared_stack_backward_workspace_bytes(batch, n, width, L,
                                                                    _dtype_code(x0))
        workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    rc = load().hcmix_shared_stack_backward(batch, n, width, L, _layers(layers),
                                            int(bool(causal)), _dtype_code(x0), _ptrs(xs[:L]),
                                            _ptrs(tables[:L]), _ptr(dy), _ptr(dx),
                                            _ptrs(dtables[:L]), int(bool(accumulate)),
                                            _ptr(workspace), _bytes(workspace), _stream(x0))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_shared_stack_backward")
    return dx, dtables


def linear_forward(x, w, out=None):
    """y = x W^T: x [rows, in] bf16, W [out, in] bf16 -> y [rows, out] bf16."""
    if not isinstance(w, torch.Tensor) or w.dim() != 2:
        raise ValueError("w: expected an [out, in] tensor")
    n_out, n_in = w.shape
    _need(w, "w", None, torch.bfloat16)
    dev = w.device
    _need(x, "x", (None, n_in), torch.bfloat16, dev)
    rows = x.shape[0]
    if out is None:
        out = torch.empty((rows, n_out), dtype=torch.bfloat16, device=dev)
    _need(out, "out", (rows, n_out), torch.bfloat16, dev)
    _gpu(dev)
    rc = load().hcmix_linear_forward(rows, n_in, n_out, _ptr(x), _ptr(w), _ptr(out), _stream(w))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_linear_forward")
    return out


def linear_backward(x, w, dy, dx=None, dw=None, with_dx=True, with_dw=True, accumulate=False,
                    workspace=None):
    """dx = dy W (bf16 [rows, in]) and dW (+)= dy^T x (fp32 [out, in]); returns
    (dx, dw), None for one not asked for.  x is read only for dW."""
    if not isinstance(w, torch.Tensor) or w.dim() != 2:
        raise ValueError("w: expected an [out, in] tensor")
    n_out, n_in = w.shape
    _need(w, "w", None, torch.bfloat16)
    dev = w.device
    _need(dy, "dy", (None, n_out), torch.bfloat16, dev)
    rows = dy.shape[0]
    want_dx = with_dx or dx is not None
    want_dw = with_dw or dw is not None
    if not want_dx and not want_dw:
        raise ValueError("linear_backward: neither dx nor dw asked for")
    if want_dw:
        _need(x, "x", (rows, n_in), torch.bfloat16, dev)
    if want_dx:
        if dx is None:
            dx = torch.empty((rows, n_in), dtype=torch.bfloat16, device=dev)
        _need(dx, "dx", (rows, n_in), torch.bfloat16, dev)
    if want_dw:
        if dw is None:
            dw = torch.empty((n_out, n_in), dtype=torch.float32, device=dev)
        _need(dw, "dw", (n_out, n_in), torch.float32, dev)
    _gpu(dev)
    if want_dw and workspace is None:
        workspace = torch.empty(load().hcmix_linear_backward_workspace_bytes(rows, n_in, n_out),
                                dtype=torch.uint8, device=dev)
    rc = load().hcmix_linear_backward(rows, n_in, n_out, _ptr(x) if want_dw else None, _ptr(w),
                                      _ptr(dy), _ptr(dx) if want_dx else None,
                                      _fptr(dw) if want_dw else None, int(bool(accumulate)),
                                      _ptr(workspace) if want_dw else None,
                                      _bytes(workspace) if want_dw else 0, _stream(w))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_linear_backward")
    return (dx if want_dx else None), (dw if want_dw else None)


class Attention(torch.autograd.Function):
    """The attention core as an autograd function over qkv."""

    @staticmethod
    def forward(ctx, qkv):
        out, lse = attention_forward(qkv.contiguous())
        ctx.save_for_backward(qkv, out, lse)
        return out

    @staticmethod
    def backward(ctx, gout):
        qkv, out, lse = ctx.saved_tensors
        return attention_backward(qkv, out, lse, gout.contiguous())


def decode_cache_bytes(batch, n, width, layers, dtype) -> int:
    code = HCMIX_BF16 if dtype == torch.bfloat16 else HCMIX_F32
    return load().hcmix_decode_cache_bytes(batch, n, width, len(layers), _layers(layers), code)


def alloc_decode_cache(batch, n, width, layers, dtype, device):
    """Device memory for hcmix_decode_step with this schedule: per layer a ring
    of the inputs later positions take as partners (2^d slots for dimension d,
    two for the local layer) and two pass-on buffers (no initialisation)."""
    return torch.empty(decode_cache_bytes(batch, n, width, layers, dtype), dtype=torch.uint8,
                       device=device)


def decode_step(x, w_selfs, w_offs, layers, n, pos, cache, out=None):
    """Position ``pos`` of every window through the causal stack: x and the
    result are [batch, width]; positions of a window must come in order."""
    L = len(layers)
    if not isinstance(x, torch.Tensor) or x.dim() != 2:
        raise ValueError("x: expected a [batch, width] tensor")
    batch, width = x.shape
    dt = _act_dtype(x)
    _need(x, "x", None, dt)
    dev = x.device
    _weights(w_selfs, "w_selfs", width, dt, dev, L)
    _weights(w_offs, "w_offs", width, dt, dev, L)
    if out is None:
        out = torch.empty_like(x)
    _need(out, "out", (batch, width), dt, dev)
    if not isinstance(cache, torch.Tensor) or cache.device != dev:
        raise ValueError(f"cache: expected a tensor on {dev}")
    _gpu(dev)
    rc = load().hcmix_decode_step(batch, n, width, L, _layers(layers), _dtype_code(x), pos,
                                  _ptr(x), _ptrs(w_selfs), _ptrs(w_offs), _ptr(cache),
                                  _bytes(cache), _ptr(out), _stream(x))
    if rc != HCMIX_OK:
        raise HcmixError(rc, "hcmix_decode_step")
    return out


class Stack(torch.autograd.Function):
    """Autograd over a stack of mixing layers.

    Stack.apply(x, layers, causal, *w_selfs, *w_offs) -> x_L"""

    @staticmethod
    def forward(ctx, x, layers, causal, *weights):
        L = len(layers)
        w_selfs, w_offs = weights[:L], weights[L:]
        xs = stack_forward(x.contiguous(), w_selfs, w_offs, layers, causal)
        ctx.layers, ctx.causal = list(layers), causal
        ctx.save_for_backward(*xs[:-1], *weights)
        return xs[-1]

    @staticmethod
    def backward(ctx, gy):
        L = len(ctx.layers)
        saved = ctx.saved_tensors
        xs, w_selfs, w_offs = saved[:L], saved[L:2 * L], saved[2 * L:]
        dx, dws, dwo = stack_backward(list(xs), w_selfs, w_offs, ctx.layers, gy.contiguous(),
                                      ctx.causal)
        grads_w = [g.to(w.dtype) for g, w in zip(dws + dwo, list(w_selfs) + list(w_offs))]
        return (dx, None, None, *grads_w)
