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
    (dict(width=1 << 17), INVALID),
    (dict(layer=-1), INVALID), (dict(mode=2), INVALID), (dict(dtype=7), INVALID),
    (dict(layer=-1, mode=0), INVALID),                # the local layer is causal only
    (dict(layer=-2, mode=1), INVALID), (dict(layer=-1, mode=1, n=12), INVALID),
    (dict(layer=-1, mode=1, width=100), UNSUPPORTED),  # a valid local layer, unsupported width
    (dict(x=None), INVALID), (dict(ws=None), INVALID), (dict(wo=None), INVALID),
    (dict(y=None), INVALID), (dict(y=P[0]), INVALID),                      # y aliases x
    (dict(batch=1 << 40), INVALID),                                       # too many rows
    (dict(width=100), UNSUPPORTED), (dict(width=4), UNSUPPORTED),         # bf16 needs 8 | width
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
    (dict(width=36), UNSUPPORTED),                    # bf16 needs 8 | width
    (dict(workspace=ctypes.c_void_p(0x800010)), UNSUPPORTED),   # workspace not 256-aligned
])
def test_backward_rejects_bad_arguments(kw, code):
    assert bwd(**kw) == code


def bwd_no_alloc(batch=2, n=16, width=64, layer=0, mode=0, dtype=1, x=P[0], ws=P[1], wo=P[2],
                 dy=P[3], dx=P[4], dws=FP[5], dwo=FP[6], acc=0):
    return hcmix.load().hcmix_backward_no_alloc(batch, n, width, layer, mode, dtype, x, ws, wo, dy,
                                                dx, dws, dwo, acc, None)


@pytest.mark.parametrize("kw,code", [
    (dict(n=3), INVALID), (dict(batch=0), INVALID), (dict(dy=None), INVALID),
    (dict(dx=P[3]), INVALID), (dict(dws=FP[6]), INVALID), (dict(dx=P[0]), INVALID),
    (dict(width=36), UNSUPPORTED),                    # bf16 needs 8 | width
    (dict(width=2112, n=64, batch=1), UNSUPPORTED),   # needs more than the 32 MiB scratch
])
def test_backward_no_alloc_rejects_bad_arguments(kw, code):
    assert bwd_no_alloc(**kw) == code


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
    (dict(width=100), UNSUPPORTED),
])
def test_stack_forward_rejects_bad_arguments(kw, code):
    assert sfwd(**kw) == code


def swg(batch=2, n=16, width=128, L=4, layers=LP, mode=0, dtype=1, xs=None, dys=None, dws=None,
        dwo=None, wsp=P[7], wsb=1 << 20):
    xs = xs if xs is not None else PP(P[0], P[0], P[0], P[0])
    dys = dys if dys is not None else PP(P[1], P[1], P[1], P[1])
    dws = dws if dws is not None else PP(*[ctypes.c_void_p(P[2].value + k * 0x10000) for k in range(4)])
    dwo = dwo if dwo is not None else PP(*[ctypes.c_void_p(P[3].value + k * 0x10000) for k in range(4)])
    return hcmix.load().hcmix_stack_weight_gradients(batch, n, width, L, layers, mode, dtype, xs,
                                                     dys, dws, dwo, 0, wsp, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(L=0), INVALID), (dict(n=12), INVALID),
    (dict(layers=(ctypes.c_int32 * 4)(0, -1, 2, 3)), INVALID),     # local layer needs causal mode
    (dict(xs=ctypes.POINTER(ctypes.c_void_p)()), INVALID),        # null array
    (dict(dys=(ctypes.c_void_p * 4)(P[1].value, P[1].value, None, P[1].value)), INVALID),
    (dict(dws=PP(P[2], P[2], P[4], P[5])), INVALID),                # two gradients alias
    (dict(dws=PP(P[0], P[2], P[4], P[5])), INVALID),                # a gradient aliases an input
    (dict(dws=PP(ctypes.c_void_p(P[2].value + 4), P[4], P[5], P[6])), UNSUPPORTED),   # misaligned
    (dict(width=100), UNSUPPORTED),
])
def test_weight_gradients_reject_bad_arguments(kw, code):
    assert swg(**kw) == code


def test_weight_gradients_check_the_workspace():
    # 64 windows of 256 x 512, 2 layers: 32 MiB of row-range partials
    V = lambda a: ctypes.c_void_p(a)  # noqa: E731
    need = hcmix.load().hcmix_stack_weight_gradients_workspace_bytes(64, 256, 512, 2, 1)
    assert need == 2 * 8 * 2 * 512 * 512 * 4
    kw = dict(batch=64, n=256, width=512, L=2, layers=(ctypes.c_int32 * 2)(3, 4),
              xs=PP(V(0x10000000), V(0x12000000)), dys=PP(V(0x20000000), V(0x22000000)),
              dws=PP(V(0x30000000), V(0x30400000)), dwo=PP(V(0x31000000), V(0x31400000)),
              wsp=V(0x40000000), wsb=need)
    assert swg(**{**kw, "wsb": need - 1}) == INVALID                          # short workspace
    assert swg(**{**kw, "dwo": PP(V(0x40000000 + 4096), V(0x31400000))}) == INVALID   # aliases it
    assert swg(**{**kw, "wsp": V(0x40000010)}) == UNSUPPORTED                 # not 256-aligned


def test_weight_gradients_workspace_query():
    lib = hcmix.load()
    q = lib.hcmix_stack_weight_gradients_workspace_bytes
    # 16 layers x 16 tiles of 128 x 128 fill the chip: every block covers all rows, no partials
    assert q(64, 256, 512, 16, hcmix.HCMIX_BF16) == 0
    # 2 layers: 8 row ranges per layer, their partials
    assert q(64, 256, 512, 2, hcmix.HCMIX_BF16) == 2 * 8 * 2 * 512 * 512 * 4
    # width not a multiple of 128, and fp32: the per-layer kernels of hcmix_backward
    assert q(64, 256, 192, 4, hcmix.HCMIX_BF16) == lib.hcmix_backward_workspace_bytes(
        64, 256, 192, hcmix.HCMIX_BF16)
    assert q(2, 16, 32, 4, hcmix.HCMIX_F32) == 0
    assert q(64, 256, 512, 0, hcmix.HCMIX_BF16) == 0


def att(batch=2, n=64, heads=2, hd=64, qkv=P[0], out=P[1], lse=P[2]):
    fp = ctypes.cast(lse, ctypes.POINTER(ctypes.c_float)) if lse is not None else None
    return hcmix.load().hcmix_attention_forward(batch, n, heads, hd, qkv, out, fp, None)


def attb(batch=2, n=64, heads=2, hd=64, qkv=P[0], out=P[1], lse=P[2], dout=P[3], dqkv=P[4]):
    fp = ctypes.cast(lse, ctypes.POINTER(ctypes.c_float)) if lse is not None else None
    return hcmix.load().hcmix_attention_backward(batch, n, heads, hd, qkv, out, fp, dout, dqkv,
                                                 None)


@pytest.mark.parametrize("kw,code", [
    (dict(batch=0), INVALID), (dict(n=0), INVALID), (dict(heads=0), INVALID),
    (dict(qkv=None), INVALID), (dict(out=None), INVALID), (dict(lse=None), INVALID),
    (dict(out=P[0]), INVALID),                                   # out aliases qkv
    (dict(lse=ctypes.c_void_p(P[1].value + 64)), INVALID),       # lse inside out
    (dict(hd=32), UNSUPPORTED), (dict(n=48), UNSUPPORTED), (dict(n=288), UNSUPPORTED),
    (dict(out=ctypes.c_void_p(P[1].value + 8)), UNSUPPORTED),    # misaligned
])
def test_attention_forward_rejects_bad_arguments(kw, code):
    assert att(**kw) == code


@pytest.mark.parametrize("kw,code", [
    (dict(dout=None), INVALID), (dict(dqkv=None), INVALID),
    (dict(dqkv=P[3]), INVALID),                                  # dqkv aliases dout
    (dict(dqkv=ctypes.c_void_p(P[2].value - 4096)), INVALID),    # dqkv covers lse
    (dict(hd=128), UNSUPPORTED), (dict(n=40), UNSUPPORTED),
    (dict(lse=ctypes.c_void_p(P[2].value + 2)), UNSUPPORTED),
])
def test_attention_backward_rejects_bad_arguments(kw, code):
    assert attb(**kw) == code


def test_lm_entry_points_reject_bad_arguments():
    lib = hcmix.load()
    fp = lambda p: ctypes.cast(p, ctypes.POINTER(ctypes.c_float))  # noqa: E731
    ef = lib.hcmix_embedding_forward
    assert ef(0, 64, 16, P[0], P[1], P[2], None) == INVALID
    assert ef(10, 64, 16, None, P[1], P[2], None) == INVALID
    assert ef(10, 64, 16, P[0], P[1], P[0], None) == INVALID          # x aliases the table
    assert ef(10, 96, 16, P[0], P[1], P[2], None) == UNSUPPORTED      # width % 64
    assert ef(10, 64, 16, P[0], P[1], ctypes.c_void_p(P[2].value + 4), None) == UNSUPPORTED
    need = lib.hcmix_embedding_backward_workspace_bytes(1000, 64, 16)
    assert need == 32 * 16 * 64 * 4        # 32 row chunks of partial sums
    assert lib.hcmix_embedding_backward_workspace_bytes(200000, 64, 16) == 49 * 16 * 64 * 4
    eb = lib.hcmix_embedding_backward
    assert eb(1000, 64, 16, P[0], P[1], fp(P[2]), 0, P[3], need - 1, None) == INVALID
    assert eb(1000, 64, 16, P[0], P[1], fp(P[1]), 0, P[3], need, None) == INVALID   # dtable = dx
    assert eb(1000, 64, 16, P[0], P[1], fp(P[2]), 0, ctypes.c_void_p(P[3].value + 16), need,
              None) == UNSUPPORTED
    hc = lib.hcmix_head_cross_entropy
    nodb = [None, None, 0, None]                                      # no bias gradient
    args = [P[0], P[1], fp(P[2]), P[3], ctypes.c_float(0.5), fp(P[4]), P[5], *nodb]
    assert hc(100, 64, 0, *args) == INVALID
    assert hc(100, 64, 48, *args) == UNSUPPORTED                      # vocab % 32
    assert hc(100, 64, 288, *args) == UNSUPPORTED                     # vocab > 256
    assert hc(100, 64, 256, P[0], P[1], fp(P[2]), P[3], ctypes.c_float(0.5), fp(P[4]), P[4],
              *nodb) == INVALID                                       # dlogits over the loss
    assert hc(100, 64, 256, P[0], P[1], fp(ctypes.c_void_p(P[2].value + 4)), P[3],
              ctypes.c_float(0.5), fp(P[4]), P[5], *nodb) == UNSUPPORTED   # bias alignment
    # the bias gradient: per-block column sums of 64 rows each
    q = lib.hcmix_head_cross_entropy_workspace_bytes
    assert q(16384, 256) == 256 * 256 * 4
    assert q(100, 96) == 768                                          # 2 blocks x 96 x 4 bytes
    assert q(100, 48) == 0 and q(0, 256) == 0
    dneed = q(100, 256)
    base = [P[0], P[1], fp(P[2]), P[3], ctypes.c_float(0.5), fp(P[4]), P[5]]
    assert hc(100, 64, 256, *base, fp(P[6]), None, dneed, None) == INVALID       # no workspace
    assert hc(100, 64, 256, *base, fp(P[6]), P[7], dneed - 1, None) == INVALID   # short
    assert hc(100, 64, 256, *base, fp(P[1]), P[7], dneed, None) == INVALID       # dbias over w
    assert hc(100, 64, 256, *base, fp(P[6]), P[5], dneed, None) == INVALID       # over dlogits
    assert hc(100, 64, 256, *base, fp(P[6]), ctypes.c_void_p(P[7].value + 16), dneed,
              None) == UNSUPPORTED                                    # workspace alignment



def test_head_backward_rejects_before_launch():
    lib = hcmix.load()
    fp = lambda p: ctypes.cast(p, ctypes.POINTER(ctypes.c_float))  # noqa: E731
    q = lib.hcmix_head_backward_workspace_bytes
    assert q(16384, 512, 256) == 32 * 256 * 512 * 4     # 32 row ranges of 512 rows
    assert q(100, 64, 32) == 2 * 32 * 64 * 4            # 2 ranges of 64 rows
    assert q(100, 64, 48) == 0 and q(0, 64, 32) == 0 and q(100, 96, 32) == 0
    hb = lib.hcmix_head_backward
    need = q(100, 64, 256)
    ok = [P[0], P[1], P[2], P[3], fp(P[4]), 0, P[5], need, None]
    assert hb(0, 64, 256, *ok) == INVALID
    assert hb(100, 64, 256, None, *ok[1:]) == INVALID                         # no x for dw
    assert hb(100, 64, 256, P[0], None, *ok[2:]) == INVALID                   # no w
    assert hb(100, 64, 256, P[0], P[1], P[2], None, None, 0, P[5], need, None) == INVALID
    assert hb(100, 64, 48, *ok) == UNSUPPORTED                                # vocab % 32
    assert hb(100, 96, 256, *ok) == UNSUPPORTED                               # width % 64
    assert hb(100, 64, 256, P[0], P[1], P[2], P[3], fp(P[4]), 0, None, need, None) == INVALID
    assert hb(100, 64, 256, P[0], P[1], P[2], P[3], fp(P[4]), 0, P[5], need - 1, None) == INVALID
    assert hb(100, 64, 256, P[0], P[1], P[2], P[0], fp(P[4]), 0, P[5], need, None) == INVALID
    assert hb(100, 64, 256, P[0], P[1], P[2], P[3], fp(P[2]), 0, P[5], need, None) == INVALID
    assert hb(100, 64, 256, P[0], P[1], P[2], ctypes.c_void_p(P[3].value + 8), fp(P[4]), 0,
              P[5], need, None) == UNSUPPORTED                                # gx alignment
    assert hb(100, 64, 256, P[0], P[1], P[2], P[3], fp(P[4]), 0,
              ctypes.c_void_p(P[5].value + 16), need, None) == UNSUPPORTED    # workspace

def test_stack_workspace_query():
    lib = hcmix.load()
    fused = lib.hcmix_stack_backward_workspace_bytes(64, 256, 64, 8, hcmix.HCMIX_BF16)
    assert fused == 64 * 8 * 2 * 64 * 64 * 4          # per-window partial weight gradients
    wide = lib.hcmix_stack_backward_workspace_bytes(64, 256, 512, 16, hcmix.HCMIX_BF16)
    layer = lib.hcmix_backward_workspace_bytes(64, 256, 512, hcmix.HCMIX_BF16)
    act = 64 * 256 * 512 * 2
    # deferred weight gradients: the 15 intermediate gradients and the transposed
    # weights of every layer; 16 layers x 16 tiles fill the chip, so no partials
    assert wide == 15 * act + 2 * 16 * 512 * 512 * 2
    # two layers: 32 tiles, so 8 row ranges per layer and their partials
    two = lib.hcmix_stack_backward_workspace_bytes(64, 256, 512, 2, hcmix.HCMIX_BF16)
    assert two == act + 2 * 2 * 512 * 512 * 2 + 2 * 8 * 2 * 512 * 512 * 4
    # longer than one chunk of 64 layers: a ring of 65 gradients
    long = lib.hcmix_stack_backward_workspace_bytes(4, 256, 512, 100, hcmix.HCMIX_BF16)
    act4 = 4 * 256 * 512 * 2
    assert long == 65 * act4 + 2 * 100 * 512 * 512 * 2
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
        cb = lib.hcmix_decode_cache_bytes(batch, n, width, L, layers, dtype)
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
    (dict(width=100), UNSUPPORTED),
])
def test_decode_rejects_bad_arguments(kw, code):
    assert dec(**kw) == code


def test_decode_cache_query():
    """Two pass-on buffers plus, per layer, 2^d ring slots (dimension d) or two
    (the local layer), each [batch][width]: bounded by the schedule, not by
    the window."""
    lib = hcmix.load()
    q = lib.hcmix_decode_cache_bytes
    lay = lambda *c: (ctypes.c_int32 * len(c))(*c)   # noqa: E731
    # rotated n = 16: dimensions 0, 1, 2, 3 -> 1 + 2 + 4 + 8 slots
    assert q(2, 16, 64, 4, lay(0, 1, 2, 3), hcmix.HCMIX_BF16) == (2 + 15) * 2 * 64 * 2
    # the window-256 rotated stack: dimensions 0..7 twice, 510 ring slots + 2
    rot = lay(*range(16))
    assert q(64, 256, 512, 16, rot, hcmix.HCMIX_BF16) == 512 * 64 * 512 * 2
    assert q(64, 256, 512, 16, rot, hcmix.HCMIX_BF16) <= 40 << 20
    # the local layer: two slots
    assert q(4, 64, 128, 2, lay(-1, -1), hcmix.HCMIX_BF16) == (2 + 4) * 4 * 128 * 2
    assert q(2, 12, 64, 4, LP, hcmix.HCMIX_BF16) == 0
    assert q(2, 16, 64, 0, LP, hcmix.HCMIX_BF16) == 0
    assert q(2, 16, 64, 4, None, hcmix.HCMIX_BF16) == 0


def sbd(batch=2, n=16, width=128, L=4, layers=LP, mode=1, dtype=1, ws=None, wo=None, dy=P[0],
        grads=None, dx=P[4], wsp=P[7], wsb=1 << 20):
    ws = ws if ws is not None else PP(P[1], P[1], P[1], P[1])
    wo = wo if wo is not None else PP(P[2], P[2], P[2], P[2])
    grads = grads if grads is not None else PP(P[3], P[5], P[6])
    return hcmix.load().hcmix_stack_backward_data(batch, n, width, L, layers, mode, dtype, ws, wo,
                                                  dy, grads, dx, wsp, wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(L=0), INVALID), (dict(n=12), INVALID), (dict(dy=None), INVALID), (dict(dx=None), INVALID),
    (dict(grads=ctypes.POINTER(ctypes.c_void_p)()), INVALID),       # null array, L > 1
    (dict(grads=(ctypes.c_void_p * 3)(P[3].value, None, P[6].value)), INVALID),
    (dict(grads=PP(P[0], P[5], P[6])), INVALID),                    # a gradient aliases dy
    (dict(grads=PP(P[3], P[3], P[6])), INVALID),                    # two gradients alias
    (dict(grads=PP(P[3], P[5], P[2])), INVALID),                    # a gradient aliases a weight
    (dict(dx=P[1]), INVALID),                                       # dx aliases a weight
    (dict(dx=P[5]), INVALID),                                       # dx aliases a gradient
    (dict(grads=PP(P[7], P[5], P[6])), INVALID),                    # a gradient in the workspace
    (dict(wsb=2 * 4 * 128 * 128 * 2 - 1), INVALID),                 # short workspace
    (dict(wsp=None), INVALID),
    (dict(wsp=ctypes.c_void_p(P[7].value + 16)), UNSUPPORTED),      # not 256-aligned
    (dict(dy=ctypes.c_void_p(P[0].value + 2)), UNSUPPORTED),        # misaligned bf16 operand
    (dict(width=100), UNSUPPORTED),
    (dict(layers=(ctypes.c_int32 * 4)(0, -1, 2, 3), mode=0), INVALID),   # local layer, bidir
])
def test_stack_backward_data_rejects_bad_arguments(kw, code):
    assert sbd(**kw) == code


def test_stack_backward_data_workspace_query():
    q = hcmix.load().hcmix_stack_backward_data_workspace_bytes
    assert q(128, 4, hcmix.HCMIX_BF16) == 2 * 4 * 128 * 128 * 2     # transposed weights
    assert q(512, 16, hcmix.HCMIX_BF16) == 2 * 16 * 512 * 512 * 2
    assert q(128, 1, hcmix.HCMIX_BF16) == 0                         # one layer reads W transposed
    assert q(32, 4, hcmix.HCMIX_F32) == 0
    assert q(128, 0, hcmix.HCMIX_BF16) == 0
    assert q(128, 4, 7) == 0


def shared_fwd(batch=2, n=16, width=64, L=2, layers=(0, 1), mode=1, dtype=1, x=P[0],
               tables=(FP[1], FP[2]), xs=(P[3], P[4])):
    lib = hcmix.load()
    lay = (ctypes.c_int32 * len(layers))(*layers)
    tp = (ctypes.c_void_p * len(tables))(*[ctypes.cast(t, ctypes.c_void_p) if t is not None
                                           else None for t in tables])
    op = (ctypes.c_void_p * len(xs))(*[p.value if p is not None else None for p in xs])
    return lib.hcmix_shared_stack_forward(batch, n, width, L, lay, mode, dtype, x, tp, op, None)


@pytest.mark.parametrize("kw,code", [
    (dict(n=12), INVALID), (dict(batch=0), INVALID), (dict(L=0), INVALID),
    (dict(x=None), INVALID), (dict(tables=(FP[1], None)), INVALID),
    (dict(xs=(P[3], P[0])), INVALID),                 # an output aliases x
    (dict(xs=(P[3], P[3])), INVALID),                 # two outputs alias
    (dict(layers=(-1, 0), mode=0), INVALID),          # the local layer is causal only
    (dict(n=512), UNSUPPORTED),                       # windows above 256
    (dict(width=96), UNSUPPORTED),                    # bf16 slices of 64 channels
    (dict(dtype=0, width=48), UNSUPPORTED),           # fp32 slices of 32 channels
    (dict(x=ctypes.c_void_p(0x100008)), UNSUPPORTED),
])
def test_shared_forward_rejects_bad_arguments(kw, code):
    assert shared_fwd(**kw) == code


def test_shared_backward_workspace_and_rejections():
    lib = hcmix.load()
    nb = lib.hcmix_shared_stack_backward_workspace_bytes(64, 256, 512, 16, 1)
    # one fp32 pair per (layer, block, position): 16 layers x (64 windows x 8 slices) x 256 x 2
    assert nb == 16 * 64 * 8 * 256 * 2 * 4
    assert lib.hcmix_shared_stack_backward_workspace_bytes(64, 512, 512, 16, 1) == 0
    assert lib.hcmix_shared_stack_backward_workspace_bytes(64, 256, 96, 16, 1) == 0
    lay = (ctypes.c_int32 * 2)(0, 1)
    vp = lambda *ps: (ctypes.c_void_p * len(ps))(*[p.value for p in ps])   # noqa: E731
    nb = lib.hcmix_shared_stack_backward_workspace_bytes(2, 16, 64, 2, 1)
    ws = ctypes.c_void_p(0x4000000)
    call = lambda **k: lib.hcmix_shared_stack_backward(   # noqa: E731
        2, 16, 64, 2, lay, 1, 1, k.get("xs", vp(P[0], P[1])), vp(P[2], P[3]),
        k.get("dy", P[4]), k.get("dx", P[5]), k.get("dts", vp(P[6], P[7])), 0,
        k.get("ws", ws), k.get("wsb", nb), None)
    assert call(dx=P[4]) == INVALID                   # dx aliases dy
    assert call(dts=vp(P[6], P[6])) == INVALID        # two table gradients alias
    assert call(dts=vp(P[6], P[2])) == INVALID        # a table gradient aliases a table
    assert call(wsb=nb - 4) == INVALID
    assert call(ws=ctypes.c_void_p(0x4000010)) == UNSUPPORTED


def field_fwd(batch=2, n=40, width=64, c=3, tau=1.0, scaled=1, p=FP[0], x=P[1], y=P[2],
              mean=FP[3], lse=FP[4], part=FP[5], ws=ctypes.c_void_p(0x4000000), wsb=None):
    lib = hcmix.load()
    if wsb is None:
        wsb = lib.hcmix_field_workspace_bytes(batch, n, c)
    return lib.hcmix_field_forward(batch, n, width, c, tau, scaled, p, x, y, mean, lse, part, ws,
                                   wsb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(batch=0), INVALID), (dict(n=0), INVALID), (dict(width=0), INVALID),
    (dict(c=0), INVALID), (dict(tau=0.0), INVALID), (dict(tau=-1.0), INVALID),
    (dict(tau=float("nan")), INVALID), (dict(tau=float("inf")), INVALID),
    (dict(tau=2.0 ** -30), INVALID), (dict(scaled=2), INVALID),
    (dict(p=None), INVALID), (dict(x=None), INVALID), (dict(y=None), INVALID),
    (dict(mean=None), INVALID), (dict(lse=None), INVALID),
    (dict(y=P[1]), INVALID),                                            # y aliases x
    (dict(lse=FP[3]), INVALID),                                         # two outputs alias
    (dict(part=ctypes.cast(ctypes.c_void_p(P[2].value + 256), ctypes.POINTER(ctypes.c_float))),
     INVALID),                                                          # partners inside y
    (dict(n=257), UNSUPPORTED), (dict(c=65), UNSUPPORTED), (dict(width=96), UNSUPPORTED),
    (dict(x=ctypes.c_void_p(P[1].value + 8)), UNSUPPORTED),             # bf16 misaligned
    (dict(p=ctypes.cast(ctypes.c_void_p(P[0].value + 2), ctypes.POINTER(ctypes.c_float))),
     UNSUPPORTED),
    (dict(ws=None), INVALID), (dict(wsb=64), INVALID),                  # no or short workspace
    (dict(ws=P[2]), INVALID),                                           # workspace aliases y
    (dict(ws=ctypes.c_void_p(0x4000010)), UNSUPPORTED),                 # workspace alignment
])
def test_field_forward_rejects_bad_arguments(kw, code):
    assert field_fwd(**kw) == code


def test_field_backward_workspace_and_rejections():
    lib = hcmix.load()
    q = lib.hcmix_field_workspace_bytes
    # per window: the coordinate table (rows of 2 c' + 8 bf16 and the norms,
    # rounded up to 256 bytes), then the N x N fp32 squared-distance gradient
    # and the N x N bf16 couplings
    table = lambda np_, cp: -(-(np_ * (2 * cp + 8) * 2 + np_ * 4) // 256) * 256  # noqa: E731
    assert q(64, 256, 32) == 64 * (table(256, 32) + 256 * 256 * 6)
    assert q(2, 40, 3) == 2 * (table(64, 16) + 64 * 64 * 6)      # n rounded up to a multiple of 32
    assert q(1, 1, 64) == table(32, 64) + 32 * 32 * 6
    assert q(0, 16, 4) == 0 and q(2, 257, 4) == 0 and q(2, 0, 4) == 0
    assert q(2, 16, 0) == 0 and q(2, 16, 65) == 0
    need = q(2, 40, 3)
    ws = ctypes.c_void_p(0x4000000)
    call = lambda **k: lib.hcmix_field_backward(   # noqa: E731
        2, k.get("n", 40), 64, k.get("c", 3), k.get("tau", 1.0), 1, FP[0], P[1], FP[2], FP[3],
        k.get("dy", P[4]), k.get("dp", FP[5]), k.get("dx", P[6]), k.get("reuse", 0),
        k.get("ws", ws), k.get("wsb", need), None)
    assert call(wsb=need - 4) == INVALID
    assert call(ws=None) == INVALID
    assert call(dx=P[4]) == INVALID                                     # dx aliases dy
    assert call(dp=FP[0]) == INVALID                                    # dp aliases p
    assert call(ws=P[6]) == INVALID                                     # workspace aliases dx
    assert call(dy=None) == INVALID
    assert call(tau=0.0) == INVALID
    assert call(n=300) == UNSUPPORTED
    assert call(c=100) == UNSUPPORTED
    assert call(ws=ctypes.c_void_p(0x4000010)) == UNSUPPORTED          # workspace alignment
    assert call(reuse=2) == INVALID and call(reuse=-1) == INVALID       # reuse_table is 0 or 1
