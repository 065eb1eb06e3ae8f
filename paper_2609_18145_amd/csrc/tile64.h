// Tiles of 64 bf16 columns in LDS and the 32 x 32 x 16 MFMA fragments read
// from them, shared by the kernels whose second product takes a score tile
// straight from registers (attention and the field coupling).
#pragma once

#include "hcmix_internal.h"
#include "device_common.h"

namespace hcmix {

constexpr int HD = 64;          // columns of a tile

// LDS tile [rows][64] bf16: 16-byte piece p of row r at piece p ^ sw(r), with
// sw a 3-bit rotation of (r / 2) % 8.  16 consecutive rows reading one piece
// (128-bit fragment reads) cover 256 distinct bytes, and 4 rows aligned to 4
// x 64 bytes (a 32-lane transposed read) do as well: rows r and r + 2 differ
// in bit 2 of sw, so they use different 64-byte halves of the 128-byte row.
__device__ __forceinline__ int att_sw(int r) {
  const int u = (r >> 1) & 7;
  return ((u << 2) | (u >> 1)) & 7;
}
__device__ __forceinline__ int att_off(int r, int col) {
  return r * HD + ((((col >> 3) ^ att_sw(r))) << 3) + (col & 7);
}

// 32 x 16 fragment of a [rows][64] tile as an MFMA operand with the row
// index as the fragment row and 8 contiguous columns per lane: lane l gets
// row r0 + l % 32, columns c0 + 8 (l / 32) .. + 8.
__device__ __forceinline__ bf16x8 att_frag(const bf16* t, int r0, int c0, int lane) {
  return *(const bf16x8*)(t + att_off(r0 + (lane & 31), c0 + 8 * (lane >> 5)));
}

// Transposed fragment for the second product: lane l gets column c0 + l % 32
// of rows {k0 + 4h + 0..3} then {k0 + 8 + 4h + 0..3}, h = l / 32 (the key
// order of a score tile's registers 8m .. 8m + 7 when k0 = 32 kt + 16 m).
__device__ __forceinline__ bf16x8 att_trfrag(const bf16* t, int k0, int c0, int lane) {
  const int g = lane >> 4, j = lane & 15;
  const int row = k0 + 4 * (g >> 1) + (j >> 2);
  const int col = c0 + 16 * (g & 1) + 4 * (j & 3);
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(t + att_off(row, col)));
  const bf16x4 hi =
      __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(t + att_off(row + 8, col)));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Registers 8m .. 8m + 7 of a score tile as a bf16 MFMA operand.
__device__ __forceinline__ bf16x8 att_pack(const f32x16& s, int m) {
  bf16x8 v;
#pragma unroll
  for (int e = 0; e < 8; e++) v[e] = to_bf16(s[8 * m + e]);
  return v;
}

// The query tiles (of 32 positions) of wave w: w and 7 - w, so that every wave
// has the same causal work (w + 1 and 8 - w key tiles) at n = 256.
__device__ __forceinline__ int att_tile(int wave, int which) { return which ? 7 - wave : wave; }

// Causal mask of a diagonal score tile: register e of lane l holds key
// 8 (e / 4) + 4 (l / 32) + e % 4 for query l % 32.
__device__ __forceinline__ bool att_masked(int e, int lane) {
  return 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3) > (lane & 31);
}

}  // namespace hcmix
