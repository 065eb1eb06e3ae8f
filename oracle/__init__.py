"""hcmix CPU oracle -- TEST INFRASTRUCTURE ONLY.

Plain, slow, double-precision implementation of the rotating-hypercube mixing
layer (paper Section 3.1 and Eq. (1)), used to check the GPU library.  Only the
tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may
import it.  It shares no code with ``paper_2609_18145_amd`` and imports nothing
from it.

The per-layer arithmetic lives in ``hcmix_oracle.c`` (plain loops, fp64
accumulation, OpenMP over rows); this module only marshals numpy arrays,
chains layers into a stack, and spells out the layer schedules of Section 3.3.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

# Layer code of the local layer (Eq. (1) with jump k = 1, partner i - 1); layer
# codes >= 0 are hypercube layers.
NEAR = -1

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hcmix_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (plain -O2, OpenMP); returns the .so path."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11",
                               _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        i64, i32, dp = ctypes.c_int64, ctypes.c_int32, ctypes.POINTER(ctypes.c_double)
        lib.oracle_log2n.argtypes, lib.oracle_log2n.restype = [i64], i32
        lib.oracle_dim.argtypes, lib.oracle_dim.restype = [i32, i64], i32
        lib.oracle_partner.argtypes, lib.oracle_partner.restype = [i64, i32, i64], i64
        lib.oracle_receives.argtypes, lib.oracle_receives.restype = [i64, i32, i64, i32], i32
        lib.oracle_valid_layer.argtypes, lib.oracle_valid_layer.restype = [i32, i64, i32], i32
        lib.oracle_num_threads.argtypes, lib.oracle_num_threads.restype = [], i32
        lib.oracle_set_num_threads.argtypes, lib.oracle_set_num_threads.restype = [i32], None
        lib.oracle_forward.argtypes = [i64, i64, i64, i32, i32, dp, dp, dp, dp]
        lib.oracle_forward.restype = i32
        lib.oracle_backward.argtypes = [i64, i64, i64, i32, i32, dp, dp, dp, dp, dp, dp, dp]
        lib.oracle_backward.restype = i32
        _lib = lib
    return _lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def log2n(n: int) -> int:
    return _load().oracle_log2n(n)


def dim(layer: int, n: int) -> int:
    """Hypercube dimension of layer ``layer``: layer mod log2 n (Section 3.1)."""
    return _load().oracle_dim(layer, n)


def partner(i: int, layer: int, n: int) -> int:
    """Partner of position i at layer ``layer``: i XOR 2^(layer mod b) (Section 3.1),
    or i - 1 for the local layer (NEAR; -1 at position 0)."""
    return _load().oracle_partner(i, layer, n)


def receives(i: int, layer: int, n: int, causal: bool) -> int:
    """1 if position i takes its partner's vector (causal: partner is earlier)."""
    return _load().oracle_receives(i, layer, n, int(bool(causal)))


def num_threads() -> int:
    return _load().oracle_num_threads()


def set_num_threads(k: int) -> None:
    """Threads the C loops use from now on (for timing; results do not change)."""
    _load().oracle_set_num_threads(int(k))


def forward(x, w_self, w_off, layer: int, causal: bool) -> np.ndarray:
    """One layer of Eq. (1) on x of shape [batch, n, width]; returns fp64."""
    x = _f64(x)
    ws, wo = _f64(w_self), _f64(w_off)
    batch, n, width = x.shape
    assert ws.shape == (width, width) and wo.shape == (width, width)
    y = np.empty_like(x)
    rc = _load().oracle_forward(batch, n, width, layer, int(bool(causal)),
                                _ptr(x), _ptr(ws), _ptr(wo), _ptr(y))
    if rc != 0:
        raise ValueError("oracle_forward rejected its arguments")
    return y


def backward(x, w_self, w_off, dy, layer: int, causal: bool):
    """Adjoint of ``forward``: returns (dx, dw_self, dw_off) in fp64."""
    x, dy = _f64(x), _f64(dy)
    ws, wo = _f64(w_self), _f64(w_off)
    batch, n, width = x.shape
    assert dy.shape == x.shape
    dx = np.empty_like(x)
    dws = np.empty((width, width))
    dwo = np.empty((width, width))
    rc = _load().oracle_backward(batch, n, width, layer, int(bool(causal)),
                                 _ptr(x), _ptr(ws), _ptr(wo), _ptr(dy),
                                 _ptr(dx), _ptr(dws), _ptr(dwo))
    if rc != 0:
        raise ValueError("oracle_backward rejected its arguments")
    return dx, dws, dwo


def stack_forward(x, w_selfs, w_offs, layers, causal: bool):
    """Apply the layers in order; returns [x_0, x_1, ..., x_L] (all fp64)."""
    xs = [_f64(x)]
    for ws, wo, layer in zip(w_selfs, w_offs, layers):
        xs.append(forward(xs[-1], ws, wo, layer, causal))
    return xs


def stack_backward(xs, w_selfs, w_offs, layers, dy, causal: bool):
    """Backward through the stack in reverse order, using the saved inputs xs[l].

    Returns (dx_0, [dw_self_l], [dw_off_l])."""
    g = _f64(dy)
    L = len(layers)
    dws = [None] * L
    dwo = [None] * L
    for l in reversed(range(L)):
        g, dws[l], dwo[l] = backward(xs[l], w_selfs[l], w_offs[l], g, layers[l], causal)
    return g, dws, dwo


# --- Layer schedules (Section 3.3, Section 4) ---------------------------------
# A schedule is the list of layer indices handed to the layer; the layer itself
# uses index mod log2 n.  Passing a dimension d < log2 n directly selects it.

def schedule_rot(num_layers: int) -> list[int]:
    """rot: hypercube dimension l mod b at layer l."""
    return list(range(num_layers))


def schedule_fixed(num_layers: int, d: int = 0) -> list[int]:
    """fixed: the same dimension at every layer (the un-rotated control)."""
    return [d] * num_layers


def schedule_gray(num_layers: int) -> list[int]:
    """Gray-code order: step t = 1, 2, ... flips the bit that a binary reflected
    Gray code flips there, i.e. the lowest set bit of t."""
    out = []
    for t in range(1, num_layers + 1):
        d = 0
        while not (t >> d) & 1:
            d += 1
        out.append(d)
    return out


def schedule_local(num_layers: int) -> list[int]:
    """local: the jump k = 1 layer (NEAR) at every layer (Section 3.3)."""
    return [NEAR] * num_layers


def schedule_mixa(n: int) -> list[int]:
    """mixa: local layers alternating with causal hypercube jumps that visit each
    scale once, longest first (Section 3.3: 32, 16, 8, 4, 2, 1 for n = 64).  A
    jump of length 2^d is the hypercube layer of dimension d."""
    b = log2n(n)
    out = []
    for d in range(b - 1, -1, -1):
        out += [NEAR, d]
    return out


def schedule_from_names(names) -> list:
    """Layer codes of a schedule written as layer names (Appendix A): "near",
    "jumpK" (K a power of two: the hypercube layer of dimension log2 K) and
    "attn" (an attention layer, which this oracle does not compute: None)."""
    out = []
    for name in names:
        if name == "near":
            out.append(NEAR)
        elif name == "attn":
            out.append(None)
        elif name.startswith("jump"):
            k = int(name[len("jump"):])
            d = k.bit_length() - 1
            assert k == 1 << d, name
            out.append(d)
        else:
            raise ValueError(f"unknown layer name {name!r}")
    return out
