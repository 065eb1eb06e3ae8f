"""The C ABI without a GPU: the library loads, exports every declared symbol,
and rejects bad arguments before touching the device."""
import ctypes
import os
import re

import pytest

import oracle
from paper_2609_18145_amd import hcmix

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "hcmix.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hcmix_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = hcmix.load()
    names = declared_functions()
    assert set(names) == set(hcmix.EXPORTS)
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings():
    lib = hcmix.load()
    assert lib.hcmix_status_string(0) == b"HCMIX_OK"
    assert lib.hcmix_status_string(1) == b"HCMIX_ERR_INVALID_VALUE"
    assert lib.hcmix_status_string(2) == b"HCMIX_ERR_UNSUPPORTED"
    assert lib.hcmix_status_string(3) == b"HCMIX_ERR_HIP"
    assert lib.hcmix_status_string(99) == b"HCMIX_ERR_UNKNOWN_STATUS"


def test_dim_matches_oracle_schedule():
    for b in range(1, 13):
        n = 1 << b
        for layer in range(3 * b):
            assert hcmix.dim(layer, n) == oracle.dim(layer, n)
    for n in [0, 1, 3, 6, 100]:
        assert hcmix.dim(0, n) == -1
    assert hcmix.dim(-1, 8) == -1


# fake, never-dereferenced device addresses: validation must reject before any launch
P = [ctypes.c_void_p(0x100000 * (k + 1)) for k in range(8)]
FP = [ctypes.cast(p, ctypes.POINTER(ctypes.c_float)) for p in P]


def fwd(batch=2, n=16, width=64, layer=0, mode=0, dtype=1, x=P[0], ws=P[1], wo=P[2], y=P[3]):
    return hcmix.load().hcmix_forward(batch, n, width, layer, mode, dtype, x, ws, wo, y, None)


def bwd(batch=2, n=16, width=64, layer=0, mode=0, dtype=1, x=P[0], ws=P[1], wo=P[2], dy=P[3],
        dx=P[4], dws=FP[5], dwo=FP[6], acc=0, workspace=P[7], wsb=None):
    lib = hcmix.load()
    if wsb is None:
        wsb = lib.hcmix_backward_workspace_bytes(batch, n, width, dtype)
    return lib.hcmix_backward(batch, n, width, layer, mode, dtype, x, ws, wo, dy, dx, dws, dwo,
                              acc, workspace, wsb, None)


INVALID = hcmix.HCMIX_ERR_INVALID_VALUE
UNSUPPORTED = hcmix.HCMIX_ERR_UNSUPPORTED


@pytest.mark.parametrize("kw,code", [
    (dict(n=0), INVALID), (dict(n=1), INVALID), (dict(n=12), INVALID),
    (dict(batch=0), INVALID), (dict(batch=-3), INVALID), (dict(width=0), INVALID),
    (dict(layer=-1), INVALID), (dict(mode=2), INVALID), (dict(dtype=7), INVALID),
    (dict(layer=-1, mode=0), INVALID),                # the local layer is causal only
    (dict(layer=-2, mode=1), INVALID), (dict(layer=-1, mode=1, n=12), INVALID),
    (dict(layer=-1, mode=1, width=96), UNSUPPORTED),  # a valid local layer, unsupported width
    (dict(x=None), INVALID), (dict(ws=None), INVALID), (dict(wo=None), INVALID),
    (dict(y=None), INVALID), (dict(y=P[0]), INVALID),                      # y aliases x
    (dict(batch=1 << 40), INVALID),                                       # too many rows
    (dict(width=96), UNSUPPORTED), (dict(width=8), UNSUPPORTED),          # bf16 needs 64 | width
    (dict(x=ctypes.c_void_p(0x100008)), UNSUPPORTED),                     # bf16 needs 16-byte alignment
    (dict(dtype=0, x=ctypes.c_void_p(0x100002)), UNSUPPORTED),            # fp32 needs 4-byte alignment
])
def test_forward_rejects_bad_arguments(kw, code):
    assert fwd(**kw) == code


def test_forward_aliasing_checks_whole_extent():
    # x spans 2*16*64 bf16 = 4096 bytes; a y starting inside that extent is rejected
    assert fwd(x=ctypes.c_void_p(0x200000), y=ctypes.c_void_p(0x200000 + 4080)) == INVALID
    # y overlapping a weight matrix (64*64 bf16 = 8192 bytes) is rejected too
    assert fwd(ws=ctypes.c_void_p(0x300000), y=ctypes.c_void_p(0x300000 - 2048)) == INVALID


@pytest.mark.parametrize("kw,code", [
    (dict(n=3), INVALID), (dict(layer=-2), INVALID), (dict(dy=None), INVALID),
    (dict(layer=-1, mode=0), INVALID), (dict(layer=-1, mode=1, dx=P[3]), INVALID),
    (dict(dx=None), INVALID), (dict(dws=None), INVALID), (dict(dwo=None), INVALID),
    (dict(dx=P[3]), INVALID),                         # dx aliases dy
    (dict(dws=FP[6]), INVALID),                       # dw_self aliases dw_off
    (dict(workspace=None), INVALID), (dict(wsb=16), INVALID),
    (dict(workspace=P[0]), INVALID),                  # workspace aliases x
    (dict(width=32), UNSUPPORTED),
    (dict(workspace=ctypes.c_void_p(0x800010)), UNSUPPORTED),   # workspace not 256-aligned
])
def test_backward_rejects_bad_arguments(kw, code):
    assert bwd(**kw) == code


def test_workspace_query():
    lib = hcmix.load()
    assert lib.hcmix_backward_workspace_bytes(2, 16, 64, hcmix.HCMIX_F32) == 0
    nb = lib.hcmix_backward_workspace_bytes(64, 256, 512, hcmix.HCMIX_BF16)
    assert nb > 2 * 512 * 512 * 2 and nb % 256 == 0
    assert lib.hcmix_backward_workspace_bytes(2, 12, 64, hcmix.HCMIX_BF16) == 0   # invalid n
    assert lib.hcmix_backward_workspace_bytes(2, 16, 96, hcmix.HCMIX_BF16) == 0   # unsupported


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(hcmix, "_lib", None)
    monkeypatch.setattr(hcmix, "LIB_PATH", str(tmp_path / "libhcmix.so"))
    with pytest.raises(RuntimeError, match="missing"):
        hcmix.load()


LP = (ctypes.c_int32 * 4)(0, 1, 2, 3)
PP = lambda *ps: (ctypes.c_void_p * len(ps))(*[p.value for p in ps])  # noqa: E731


def sfwd(batch=2, n=16, width=64, L=4, layers=LP, mode=0, dtype=1, x=P[0], ws=None, wo=None, xs=None):
    ws = ws if ws is not None else PP(P[1], P[1], P[1], P[1])
    wo = wo if wo is not None else PP(P[2], P[2], P[2], P[2])
    xs = xs if xs is not None else PP(P[3], P[4], P[5], P[6])
    return hcmix.load().hcmix_stack_forward(batch, n, width, L, layers, mode, dtype, x, ws, wo, xs, None)


@pytest.mark.parametrize("kw,code", [
    (dict(L=0), INVALID), (dict(n=12), INVALID), (dict(layers=(ctypes.c_int32 * 4)(0, -1, 2, 3)), INVALID),
    (dict(x=None), INVALID), (dict(xs=PP(P[3], P[3], P[5], P[6])), INVALID),   # two outputs alias
    (dict(xs=PP(P[0], P[4], P[5], P[6])), INVALID),                            # output aliases x
    (dict(xs=PP(P[3], P[4], P[1], P[6])), INVALID),                            # output aliases a weight
    (dict(width=96), UNSUPPORTED),
])
def test_stack_forward_rejects_bad_arguments(kw, code):
    assert sfwd(**kw) == code


def test_stack_workspace_query():
    lib = hcmix.load()
    fused = lib.hcmix_stack_backward_workspace_bytes(64, 256, 64, 8, hcmix.HCMIX_BF16)
    assert fused == 64 * 8 * 2 * 64 * 64 * 4          # per-window partial weight gradients
    wide = lib.hcmix_stack_backward_workspace_bytes(64, 256, 512, 16, hcmix.HCMIX_BF16)
    layer = lib.hcmix_backward_workspace_bytes(64, 256, 512, hcmix.HCMIX_BF16)
    # two gradient buffers, two layers' split-K partials (one layer's are summed
    # inside the next layer's launch), transposed weights of every layer
    assert wide == 2 * 64 * 256 * 512 * 2 + 2 * layer + 2 * 16 * 512 * 512 * 2
    # a width that is not a multiple of 128: one layer's partials
    w192 = lib.hcmix_stack_backward_workspace_bytes(64, 256, 192, 4, hcmix.HCMIX_BF16)
    layer192 = lib.hcmix_backward_workspace_bytes(64, 256, 192, hcmix.HCMIX_BF16)
    assert w192 == 2 * 64 * 256 * 192 * 2 + layer192 + 2 * 4 * 192 * 192 * 2
    assert lib.hcmix_stack_backward_workspace_bytes(64, 256, 512, 1, hcmix.HCMIX_BF16) == layer
    assert lib.hcmix_stack_backward_workspace_bytes(64, 256, 64, 0, hcmix.HCMIX_BF16) == 0
    assert lib.hcmix_stack_backward_workspace_bytes(2, 16, 32, 1, hcmix.HCMIX_F32) == 0


def dec(batch=2, n=16, width=64, L=4, layers=LP, dtype=1, pos=0, x=P[0], ws=None, wo=None,
        cache=P[3], cb=None, y=P[4]):
    lib = hcmix.load()
    ws = ws if ws is not None else PP(P[1], P[1], P[1], P[1])
    wo = wo if wo is not None else PP(P[2], P[2], P[2], P[2])
    if cb is None:
        cb = lib.hcmix_decode_cache_bytes(batch, n, width, L, dtype)
    return lib.hcmix_decode_step(batch, n, width, L, layers, dtype, pos, x, ws, wo, cache, cb, y,
                                 None)


@pytest.mark.parametrize("kw,code", [
    (dict(pos=-1), INVALID), (dict(pos=16), INVALID), (dict(L=0), INVALID), (dict(n=12), INVALID),
    (dict(layers=(ctypes.c_int32 * 4)(0, -2, 2, 3)), INVALID),
    (dict(cb=16), INVALID), (dict(cache=None), INVALID), (dict(x=None), INVALID),
    (dict(y=P[0]), INVALID),                          # y aliases x
    (dict(y=P[3]), INVALID),                          # y aliases the cache
    (dict(cache=P[1]), INVALID),                      # cache aliases a weight
    (dict(cache=ctypes.c_void_p(0x400010)), UNSUPPORTED),   # cache not 256-aligned
    (dict(width=96), UNSUPPORTED),
])
def test_decode_rejects_bad_arguments(kw, code):
    assert dec(**kw) == code


def test_decode_cache_query():
    lib = hcmix.load()
    assert lib.hcmix_decode_cache_bytes(2, 16, 64, 4, hcmix.HCMIX_BF16) == 4 * 2 * 16 * 64 * 2
    assert lib.hcmix_decode_cache_bytes(64, 256, 512, 16, hcmix.HCMIX_BF16) == 16 * 64 * 256 * 512 * 2
    assert lib.hcmix_decode_cache_bytes(2, 12, 64, 4, hcmix.HCMIX_BF16) == 0
    assert lib.hcmix_decode_cache_bytes(2, 16, 64, 0, hcmix.HCMIX_BF16) == 0
