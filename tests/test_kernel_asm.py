"""Static check of the gfx950 assembly of every HIP source: no MFMA may run
under a changed lane mask (EXEC) unless a branch skips the all-inactive case.

An MFMA writes its whole result whatever EXEC holds, so a guard such as
`if (k < ksteps) acc = mfma(...)` must be a wave-uniform branch.  When the
compiler cannot prove the condition uniform it lowers the guard to a lane mask
and may leave out the branch for a short block; the MFMA then runs with every
lane masked and accumulates whatever its operand registers hold.  The decode
kernel once did exactly that and produced NaN at widths >= 256.

The scan is heuristic by design: inside a region that starts at a lane-mask
change (`s_and_saveexec_b64`, `s_and_b64 exec, ...`) and ends at the restore
(`s_or_b64 exec, exec, ...`), an MFMA must be preceded by an `s_cbranch_execz`
or `s_cbranch_execnz` in that region.

A second scan covers the write-through 16-byte store (an asm statement, so
the compiler inserts no wait states for it): its data registers must not come
straight from an MFMA result or a transcendental VALU op, and the statement's
own `s_nop` must follow it, before its data registers may be rewritten."""
import concurrent.futures as cf
import os
import re
import shutil
import subprocess

import pytest

from paper_2609_18145_amd import build as pkg_build

MASK_SET = re.compile(r"s_(and|andn2|or|xor|mov)_saveexec_b64|s_(and|andn2|mov|xor)_b64 exec,")
MASK_RESTORE = re.compile(r"s_or_b64 exec, exec|s_mov_b64 exec, -1")


def unguarded_mfmas(asm: str) -> dict:
    """kernel symbol -> number of MFMAs under a lane mask with no exec branch."""
    found, kernel, masked, guarded = {}, None, False, False
    for raw in asm.splitlines():
        line = raw.strip()
        m = re.match(r"^(_Z\S+):", line)
        if m:
            kernel, masked, guarded = m.group(1), False, False
            continue
        if not line or line.startswith(";"):
            continue
        if MASK_SET.match(line):
            masked, guarded = True, False
        elif MASK_RESTORE.match(line):
            masked = False
        elif line.startswith(("s_cbranch_execz", "s_cbranch_execnz")):
            guarded = True
        elif "v_mfma" in line and masked and not guarded:
            found[kernel] = found.get(kernel, 0) + 1
    return found


WT_STORE = re.compile(r"global_store_dwordx4 (\S+), (v\[\d+:\d+\]|v\d+), off sc1$")
REG = re.compile(r"([va])\[(\d+):(\d+)\]|([va])(\d+)\b")
TRANS = ("v_exp", "v_log", "v_rcp", "v_rsq", "v_sqrt", "v_sin", "v_cos")


def _regs(operand: str) -> set:
    m = REG.fullmatch(operand.strip())
    if not m:
        return set()
    if m.group(1):
        return {(m.group(1), r) for r in range(int(m.group(2)), int(m.group(3)) + 1)}
    return {(m.group(4), int(m.group(5)))}


def _vector_dest(line: str) -> set:
    """Vector registers an instruction writes (its first operand), for the
    instructions that have one: VALU and MFMA ops and vector/LDS loads."""
    op, _, rest = line.partition(" ")
    writes = op.startswith("v_") or op.startswith(("ds_read", "global_load", "buffer_load",
                                                   "flat_load", "scratch_load"))
    if not writes or not rest:
        return set()
    return _regs(rest.split(",")[0])


def wt_store_hazards(asm: str) -> list:
    """(kernel, store line, reason) for every write-through 16-byte store
    whose data registers were last written by an MFMA or a transcendental op
    (scanning back in program order within the kernel), or that is not
    followed by an s_nop."""
    found, kernel, body = [], None, []
    for raw in asm.splitlines():
        line = raw.strip()
        m = re.match(r"^(_Z\S+):", line)
        if m:
            kernel, body = m.group(1), []
            continue
        if not line or line.startswith((";", ".")) or line.endswith(":"):
            continue
        body.append(line)
        w = WT_STORE.match(line)
        if not w:
            continue
        data = _regs(w.group(2))
        for prev in reversed(body[:-1]):
            hit = _vector_dest(prev) & data
            if hit:
                if "v_mfma" in prev:
                    found.append((kernel, line, f"data written by an MFMA: {prev}"))
                elif prev.startswith(TRANS):
                    found.append((kernel, line, f"data written by a transcendental op: {prev}"))
                break
    # the wait states after each store: the next instruction is the s_nop
    lines = [l.strip() for l in asm.splitlines()
             if l.strip() and not l.strip().startswith(";")]
    for i, line in enumerate(lines):
        if WT_STORE.match(line) and (i + 1 >= len(lines) or not lines[i + 1].startswith("s_nop")):
            found.append(("?", line, "no s_nop after the store"))
    return found


def test_wt_store_scanner_flags_mfma_fed_data():
    bad = """_Zkernel:
\tv_mfma_f32_32x32x16_bf16 v[4:19], v[40:43], v[28:31], v[4:19]
\tv_add_u32_e32 v30, 1, v30
\tglobal_store_dwordx4 v[0:1], v[8:11], off sc1
\ts_nop 1
"""
    good = """_Zkernel:
\tv_mfma_f32_32x32x16_bf16 v[4:19], v[40:43], v[28:31], v[4:19]
\tds_read_b128 v[8:11], v2
\ts_waitcnt lgkmcnt(0)
\tglobal_store_dwordx4 v[0:1], v[8:11], off sc1
\ts_nop 1
"""
    no_nop = """_Zkernel:
\tds_read_b128 v[8:11], v2
\tglobal_store_dwordx4 v[0:1], v[8:11], off sc1
\tv_mov_b32_e32 v8, 0
"""
    assert len(wt_store_hazards(bad)) == 1
    assert wt_store_hazards(good) == []
    assert [r for _, _, r in wt_store_hazards(no_nop)] == ["no s_nop after the store"]


def test_scanner_flags_a_masked_mfma_and_passes_a_guarded_one():
    bad = """_Zkernel:
\ts_and_saveexec_b64 s[2:3], vcc
\tv_mfma_f32_32x32x16_bf16 v[4:19], v[40:43], v[28:31], v[4:19]
\ts_or_b64 exec, exec, s[2:3]
"""
    good = """_Zkernel:
\ts_and_saveexec_b64 s[2:3], vcc
\ts_cbranch_execz .LBB0_2
\tv_mfma_f32_32x32x16_bf16 v[4:19], v[40:43], v[28:31], v[4:19]
.LBB0_2:
\ts_or_b64 exec, exec, s[2:3]
\tv_mfma_f32_32x32x16_bf16 v[4:19], v[40:43], v[28:31], v[4:19]
"""
    assert unguarded_mfmas(bad) == {"_Zkernel": 1}
    assert unguarded_mfmas(good) == {}


def _device_asm(src: str, out_dir: str) -> str:
    out = os.path.join(out_dir, os.path.basename(src) + ".s")
    cmd = [pkg_build.HIPCC, *[f for f in pkg_build.FLAGS if f != "-fPIC"], "--cuda-device-only",
           "-S", src, "-o", out]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc -S failed for {src}:\n{res.stderr}")
    with open(out) as f:
        return f.read()


@pytest.mark.skipif(not os.path.exists(pkg_build.HIPCC) and shutil.which("hipcc") is None,
                    reason="hipcc not available")
def test_no_mfma_runs_under_a_lane_mask(tmp_path):
    srcs = pkg_build.sources()
    assert srcs
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        asms = list(ex.map(lambda s: _device_asm(s, str(tmp_path)), srcs))
    assert sum(a.count("v_mfma") for a in asms) > 100      # the scan is not vacuous
    bad = {}
    for src, asm in zip(srcs, asms):
        for k, v in unguarded_mfmas(asm).items():
            bad[f"{os.path.basename(src)}: {k}"] = v
    assert not bad, f"MFMAs under a lane mask without an exec branch: {bad}"


@pytest.mark.skipif(not os.path.exists(pkg_build.HIPCC) and shutil.which("hipcc") is None,
                    reason="hipcc not available")
def test_write_through_stores_never_take_mfma_results(tmp_path):
    srcs = pkg_build.sources()
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        asms = list(ex.map(lambda s: _device_asm(s, str(tmp_path)), srcs))
    stores = sum(len(re.findall(r"global_store_dwordx4 .*, off sc1", a)) for a in asms)
    assert stores > 50                                    # the scan is not vacuous
    bad = [(os.path.basename(src), k, line, why) for src, asm in zip(srcs, asms)
           for k, line, why in wt_store_hazards(asm)]
    assert not bad, f"write-through stores with unsafe data: {bad[:5]}"
