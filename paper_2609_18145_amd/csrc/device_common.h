// Device helpers shared by the bf16 kernels: MFMA wrapper, LDS DMA, waits,
// scheduling hints, LDS swizzles and transposed LDS fragment reads.
#pragma once

#include "hcmix_internal.h"

namespace hcmix {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// Block index -> tile index, keeping consecutive tiles (the column tiles of
// one row tile, the tiles of one window) on one XCD: blocks are dealt to the
// 8 XCDs round-robin.
__device__ __forceinline__ int xcd_tile(int bid, int total) {
  if (total % 8 != 0) return bid;
  return (bid % 8) * (total / 8) + bid / 8;
}

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// 16 x 16 x 32: lane l holds row (A) or column (B) l % 16, K elements
// 8 (l / 16) .. 8 (l / 16) + 7; the result's lane l holds column l % 16, rows
// 4 (l / 16) .. 4 (l / 16) + 3.
__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// 16 bytes global -> LDS; `lds` is the wave-uniform base, lane i lands at +16*i.
__device__ __forceinline__ void dma16(const bf16* src, bf16* lds) {
  __builtin_amdgcn_global_load_lds(src, lds, 16, 0, 0);
}

// Pointers read from memory (rather than taken from kernel arguments) are
// generic, and a generic store becomes a FLAT instruction, which also counts
// on lgkmcnt and so serialises with the LDS reads that feed it; stores through
// this type stay global.
typedef __attribute__((address_space(1))) u32x4 global_u32x4;

// Stores that write through L2 to memory at device scope (the sc1 policy
// bit).  A kernel's completion has to write the dirty L2 lines its ordinary
// stores left behind back to memory before a dependent kernel may start;
// lines written through are clean, so the tail of an output-heavy kernel is
// shorter (about a microsecond per 16 MiB of output, measured).  Values and
// ordering are those of an ordinary global store.
//
// store_wt16 is an asm statement, which the compiler does not know to be a
// store: it inserts neither the wait states that must separate a store of
// more than 8 bytes from a VALU write of its data registers (2 on
// gfx94x/gfx950; the s_nop supplies them) nor those an MFMA result needs
// before a memory instruction reads it.  So its data must come from LDS or
// from VALU work, never straight from MFMA accumulators.  store_wt4 is a
// relaxed device-scope atomic store, which compiles to the same sc1 store
// with every hazard known to the compiler.
__device__ __forceinline__ void store_wt16(void* dst, const u32x4& v) {
  asm volatile("global_store_dwordx4 %0, %1, off sc1\n\ts_nop 1" ::"v"(dst), "v"(v) : "memory");
}
__device__ __forceinline__ void store_wt4(float* dst, float v) {
  __hip_atomic_store(dst, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Wait until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

// Wait for all but the `ahead` most recently issued pipeline stages (DPS DMA
// instructions each) of this wave; ahead < NA.
template <int NA, int DPS>
__device__ __forceinline__ void wait_stages(int ahead) {
  if constexpr (NA > 0) {
    if (ahead >= NA - 1) { wait_vmcnt<(NA - 1) * DPS>(); return; }
    wait_stages<NA - 1, DPS>(ahead);
  }
}

// Scheduling hint for one MFMA sub-step: alternate its NMFMA matrix
// instructions with the NDS LDS reads that fetch the next sub-step's
// fragments, spreading the reads evenly, so LDS latency hides under MFMAs.
template <int NMFMA, int NDS>
__device__ __forceinline__ void interleave_mfma_ds() {
#pragma unroll
  for (int i = 0; i < NMFMA; i++) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);            // one MFMA
    const int nds = (NDS * (i + 1)) / NMFMA - (NDS * i) / NMFMA;
    if (nds == 1) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one DS read
    if (nds == 2) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    if (nds == 3) __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
  }
}

// Same, with the DS reads front-loaded: with NDS <= NMFMA one read follows
// each of the first NDS MFMAs, so the last read is issued several MFMAs before
// the region ends and the next region's first MFMA does not wait for it
// (with more reads than MFMAs, the extra ones go to the first MFMAs).  Use
// inside a region fenced with __builtin_amdgcn_sched_barrier(0) on both sides.
template <int NMFMA, int NDS>
__device__ __forceinline__ void interleave_front() {
  static_assert(NDS <= 3 * NMFMA, "");
#pragma unroll
  for (int i = 0; i < NMFMA; i++) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    const int nds = NDS / NMFMA + (i < NDS % NMFMA ? 1 : 0);
    if (nds == 1) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    if (nds == 2) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    if (nds == 3) __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
  }
}

// LDS has 64 banks of 4 bytes: a 128-bit access is conflict-free when each
// group of 16 lanes covers 256 distinct bytes (mod 256), a 64-bit access when
// each group of 32 lanes does.
//
// k-contiguous tile [rows][BK] (2*BK-byte rows, BK = 32 or 64): 16-byte piece
// `ch` of row m sits at piece ch ^ ((m / (128/BK)) % (BK/8)), so 16 consecutive
// rows reading the same piece land in 16 distinct 16-byte slots.  Elements.
template <int BK>
__device__ __forceinline__ int swz(int m, int ch) {
  static_assert(BK == 32 || BK == 64, "");
  constexpr int RPQ = 128 / BK;   // rows sharing one 256-byte bank window
  return m * BK + ((ch ^ ((m / RPQ) & (BK / 8 - 1))) << 3);
}

// Row-major tile read transposed, RB bytes per row (256 or 128): 64-byte
// segment `seg` of row `row` is stored at segment seg ^ f(row), so the 4 rows
// x 64 bytes that 32 lanes of a tr read touch fall in distinct bank quarters.
template <int RB>
__device__ __forceinline__ int trswz(int row, int seg) {
  static_assert(RB == 256 || RB == 128, "row of 64 or 128 bf16");
  return RB == 256 ? (seg ^ (row & 3)) : (seg ^ ((row >> 1) & 1));
}

// Transposed 32x32x16 operand fragment from a row-major tile T[k][col] with
// RB-byte rows: lane l gets T[k0 + 8*(l/32) + t][c0 + l%32], t = 0..7, the same
// k order as a ds_read_b128 fragment of a k-contiguous tile.  c0 % 32 == 0.
template <int RB>
__device__ __forceinline__ bf16x8 tr_frag(const bf16* tile, int k0, int c0, int lane) {
  const int g = lane >> 4, j = lane & 15;
  const int row = k0 + 8 * (g >> 1) + (j >> 2);
  const int seg = c0 >> 5;                                   // 32 columns = 64 bytes
  const int in = 16 * (g & 1) + 4 * (j & 3);                 // column within the segment
  const bf16* p = tile + row * (RB / 2) + trswz<RB>(row, seg) * 32 + in;
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)p);
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p + 4 * (RB / 2)));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Source element offset (row, column) for lane i of DMA block b of a tr tile.
template <int RB>
__device__ __forceinline__ void tr_dma_coord(int b, int i, int* row, int* col) {
  const int o = b * 1024 + 16 * i;          // byte offset in the tile
  const int r = o / RB, ob = o % RB;
  const int seg = trswz<RB>(r, ob >> 6);    // the swizzle is an involution
  *row = r;
  *col = seg * 32 + ((ob & 63) >> 1);
}

}  // namespace hcmix
