// Field coupling of the dynamics variant (Section 3.4): every position i of a
// window carries a coordinate p_i (c <= 64 components, fp32), and the causal
// coupling of row i is the row-normalised Gaussian of squared distances,
//   D[i][j] = |p_i - p_j|^2,  m_i = mean of D[i][j] over j <= i,
//   a[i][j] = -D[i][j] / (tau m_i)   (scaled form, "field"; 0 when m_i = 0)
//           = -D[i][j] / tau         (unscaled form),
//   C[i][j] = exp(a[i][j]) / Z_i over j <= i,  y_i = sum_j C[i][j] x_j,
// with the effective number of partners exp(-sum_j C ln C) of Section 7 as a
// by-product.  x, y bf16 [batch][n][width], width % 64 == 0, n <= 256.
//
// Distances go through the Gram matrix on the bf16 matrix cores:
//   D[i][j] = N_i + N_j - 2 p'_i . p'_j,  p' = p - p_0 (D is translation
// invariant; centring on the window's first position keeps the norms near the
// distances' scale, and makes D exactly 0 when all coordinates are equal),
// each centred component split into bf16 hi + lo (exact in fp32, 2^-17
// relative) and the dot product taken as hi.hi + lo.hi + hi.lo (three MFMAs
// per 16 components, fp32 accumulation; the dropped lo.lo term is below
// 2^-17 of the norms).  The diagonal is set to exactly 0 (its rounding would
// otherwise reach the unscaled logits undivided).  Every logit is <= 0 up to
// that rounding and the diagonal's is 0, so each row's maximum is known: the
// exponentials need no running maximum and Z_i lies in [1, i + 1].
//
// Kernels (one window's coordinates and one 64-column slab per block, the
// whole causal row of a 32-query tile in registers as in the attention core):
//   field_fwd_kernel        y slab, and (slab 0) m_i, ln Z_i, partners;
//   field_bwd_rows_kernel   per query tile: dP[i][j] = dy_i . x_j over the full
//                           width, Delta_i = sum_j C dP (= dy_i . y_i),
//                           da = C (dP - Delta), and the gradient of the
//                           squared distances dD (written, fp32, [key][query]);
//   field_bwd_dx_kernel     dx slab = C^T dy (keys in lanes);
//   field_bwd_coord_kernel  dp_i = 2 sum_j E[i][j] (p_i - p_j), E = dD + dD^T,
//                           on the fp32 matrix cores.
#include "hcmix_internal.h"
#include "device_common.h"
#include "tile64.h"

namespace hcmix {

namespace {

constexpr int FT = 512;                       // threads per block, 8 waves (coordinate kernel: 256)
constexpr int FTC = 256;
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Coordinate table in LDS: row r = [hi (cp) | lo (cp) | 8 pad] bf16 of the
// centred coordinate p_r - p_0 (cp = c rounded up to 16, zero padded).  The
// row stride 2 cp + 8 elements is an odd multiple of 16 bytes, so 16
// consecutive rows read at one column fall in 16 distinct 16-byte bank slots.
__device__ __forceinline__ int ct_stride(int cp) { return 2 * cp + 8; }

__device__ __forceinline__ bf16x8 ct_frag(const bf16* t, int rs, int r0, int c0, int lane) {
  return *(const bf16x8*)(t + (r0 + (lane & 31)) * rs + c0 + 8 * (lane >> 5));
}
// The 8 components of row r that lane half h contributes to a 16-wide k step.
__device__ __forceinline__ bf16x8 ct_row(const bf16* t, int rs, int r, int c0, int half) {
  return *(const bf16x8*)(t + r * rs + c0 + 8 * half);
}

// Copy a window's coordinates (pw: rows x c fp32, contiguous) into LDS rows
// `stride` bytes apart: consecutive threads take consecutive elements (every
// load coalesced, all of a thread's loads issued before its first LDS write);
// the element -> (row, column) walk advances by a precomputed step, with no
// division per element.
template <int THREADS, int PER>
__device__ __forceinline__ void stage_coords(const float* __restrict__ pw, int rows, int c,
                                             unsigned char* dst, int stride) {
  const int total = rows * c;
  float v[PER];
#pragma unroll
  for (int u = 0; u < PER; u++) {   // unconditional loads (clamped): no branch waits per load
    const int e = min(threadIdx.x + THREADS * u, total - 1);
    v[u] = pw[e];
  }
  int r = threadIdx.x / c, k = threadIdx.x % c;
  const int dr = THREADS / c, dk = THREADS % c;
#pragma unroll
  for (int u = 0; u < PER; u++) {
    if (threadIdx.x + THREADS * u < total) *(float*)(dst + r * stride + 4 * k) = v[u];
    k += dk;
    r += dr;
    if (k >= c) {
      k -= c;
      r += 1;
    }
  }
}

// The table rows [0, rows) (rows <= the block's threads) and their squared
// norms N_r (of hi + lo, fp32), from the window's coordinates pw [n][c]:
// the raw rows are staged into the table's own space, each thread reads its
// row and row 0, and after a barrier overwrites its row with the split centred
// values.  Ends with a barrier.
__device__ __forceinline__ void build_coords(const float* __restrict__ pw, int n, int c, int cp,
                                             int rows, bf16* sT, float* sN) {
  const int rsb = ct_stride(cp) * 2;                 // bytes per table row
  unsigned char* base = (unsigned char*)sT;
  stage_coords<FT, 32>(pw, rows < n ? rows : n, c, base, rsb);
  __syncthreads();
  const int r = threadIdx.x;
  const bool live = r < n && r < rows;
  const int rr = live ? r : 0;
  float v[64];
#pragma unroll
  for (int k = 0; k < 64; k++) {
    float t = 0.f;
    if (k < c) t = *(const float*)(base + rr * rsb + 4 * k) - *(const float*)(base + 4 * k);
    v[k] = live ? t : 0.f;
  }
  __syncthreads();
  if (r < rows) {
    bf16* row = sT + r * ct_stride(cp);
    float nn = 0.f;
#pragma unroll
    for (int k = 0; k < 64; k += 2) {
      const bf16 ha = to_bf16(v[k]), hb = to_bf16(v[k + 1]);
      const bf16 la = to_bf16(v[k] - (float)ha), lb = to_bf16(v[k + 1] - (float)hb);
      if (k < cp) {
        *(bf16x2*)(row + k) = bf16x2{ha, hb};
        *(bf16x2*)(row + cp + k) = bf16x2{la, lb};
      }
      const float ta = (float)ha + (float)la, tb = (float)hb + (float)lb;
      nn = fmaf(ta, ta, nn);
      nn = fmaf(tb, tb, nn);
    }
    *(u32x4*)(row + 2 * cp) = u32x4{0u, 0u, 0u, 0u};
    sN[r] = nn;
  }
  __syncthreads();
}

// Rows [0, NT * 32) of one slab of SW columns (SW / 64 tiles of 64 columns;
// src: row 0's first column, rows `stride` apart) into swizzled LDS tiles
// NT * 32 * 64 elements apart; rows >= n are zero.  Every load is in flight
// before the first LDS write.
template <int NT, int SW>
__device__ __forceinline__ void load_slab(const bf16* __restrict__ src, size_t stride, int n,
                                          bf16* tile) {
  constexpr int NP = NT * 32, TP = NP * 8, PIECES = TP * (SW / 64), PER = (PIECES + FT - 1) / FT;
  u32x4 v[PER];
#pragma unroll
  for (int j = 0; j < PER; j++) {   // unconditional loads (clamped), zeroed after
    const int pi = min(threadIdx.x + FT * j, PIECES - 1), tl = pi / TP, r = (pi % TP) >> 3,
              pc = pi & 7;
    v[j] = *(const u32x4*)(src + (size_t)min(r, n - 1) * stride + 64 * tl + 8 * pc);
    if (r >= n) v[j] = u32x4{0u, 0u, 0u, 0u};
  }
#pragma unroll
  for (int j = 0; j < PER; j++) {
    const int pi = threadIdx.x + FT * j, tl = pi / TP, r = (pi % TP) >> 3, pc = pi & 7;
    if (pi < PIECES) *(u32x4*)(tile + tl * NP * 64 + att_off(r, 8 * pc)) = v[j];
  }
}

// s_waitcnt vmcnt(n) for a wave-uniform runtime n <= 15.
__device__ __forceinline__ void wait_vmcnt_upto(int n) {
  switch (n) {
    case 0: wait_vmcnt<0>(); break;
    case 1: wait_vmcnt<1>(); break;
    case 2: wait_vmcnt<2>(); break;
    case 3: wait_vmcnt<3>(); break;
    case 4: wait_vmcnt<4>(); break;
    case 5: wait_vmcnt<5>(); break;
    case 6: wait_vmcnt<6>(); break;
    case 7: wait_vmcnt<7>(); break;
    case 8: wait_vmcnt<8>(); break;
    case 9: wait_vmcnt<9>(); break;
    case 10: wait_vmcnt<10>(); break;
    default: wait_vmcnt<0>(); break;
  }
}

// The 32-row tile a wave of an 8-wave block works on: waves w and w + 4 share
// a SIMD and take tiles w and 7 - w, whose causal work (w + 1 and 8 - w tiles
// of the other side) sums to the same 9 for every SIMD at 8 tiles.
__device__ __forceinline__ int wave_tile(int wave) { return wave < 4 ? wave : 11 - wave; }

// Gram tile G^T[key][query] for keys kt*32.. (A operand, table rows) and the
// lane's query q (B operand): hi.hi + lo.hi + hi.lo, in that order.
__device__ __forceinline__ f32x16 gram_keys(const bf16* sT, int rs, int cp, int kt, int q,
                                            int lane) {
  const int half = lane >> 5;
  f32x16 acc = {};
  for (int k0 = 0; k0 < cp; k0 += 16) {
    const bf16x8 khi = ct_frag(sT, rs, kt * 32, k0, lane);
    const bf16x8 klo = ct_frag(sT, rs, kt * 32, cp + k0, lane);
    const bf16x8 qhi = ct_row(sT, rs, q, k0, half);
    const bf16x8 qlo = ct_row(sT, rs, q, cp + k0, half);
    acc = mfma32(khi, qhi, acc);
    acc = mfma32(klo, qhi, acc);
    acc = mfma32(khi, qlo, acc);
  }
  return acc;
}

// Same products with queries qt*32.. as the A operand and the lane's key j as
// the B operand (G[query][key]), in the same order of terms.
__device__ __forceinline__ f32x16 gram_queries(const bf16* sT, int rs, int cp, int qt, int j,
                                               int lane) {
  const int half = lane >> 5;
  f32x16 acc = {};
  for (int k0 = 0; k0 < cp; k0 += 16) {
    const bf16x8 qhi = ct_frag(sT, rs, qt * 32, k0, lane);
    const bf16x8 qlo = ct_frag(sT, rs, qt * 32, cp + k0, lane);
    const bf16x8 khi = ct_row(sT, rs, j, k0, half);
    const bf16x8 klo = ct_row(sT, rs, j, cp + k0, half);
    acc = mfma32(qhi, khi, acc);
    acc = mfma32(qhi, klo, acc);
    acc = mfma32(qlo, khi, acc);
  }
  return acc;
}

// Scale of the logits of a row with mean squared distance m: a = -D * scale.
// A positive mean below 2^-100 is taken as 2^-100 (such coordinates are not
// resolved by fp32 squared distances anyway), which keeps the scale finite for
// tau >= 2^-24.
__device__ __forceinline__ float clamped_mean(float m) { return fmaxf(m, 0x1p-100f); }
__device__ __forceinline__ float logit_scale(float m, float inv_tau, int scaled) {
  if (!scaled) return inv_tau;
  return m > 0.f ? inv_tau / clamped_mean(m) : 0.f;
}

// Dynamic LDS layouts (bytes).
constexpr int table_bytes(int NT, int cp) { return NT * 32 * (2 * cp + 8) * 2; }
constexpr int fwd_lds_bytes(int NT, int SW, int cp) {
  return NT * 32 * SW * 2 + NT * 32 * 4 + table_bytes(NT, cp);
}
constexpr int dx_lds_bytes(int NT, int SW, int cp) {
  return NT * 32 * SW * 2 + 3 * NT * 32 * 4 + table_bytes(NT, cp);
}
// rows kernel: NS stages of [x rows (NT * 32)][64] + [dy rows (32)][64] bf16
constexpr int rows_stage_elems(int NT) { return (NT * 32 + 32) * 64; }
constexpr int rows_lds_bytes(int NT, int NS, int cp) {
  return NS * rows_stage_elems(NT) * 2 + NT * 32 * 4 + 2 * 8 * 32 * 4 + table_bytes(NT, cp);
}
constexpr int rows_stages(int NT, int cp) {
  return rows_lds_bytes(NT, 3, cp) <= 160 * 1024 ? 3 : 2;
}
// coordinate kernel: E tile [32][NP + 1] fp32, coordinates [NP][ck + 1] fp32,
// row-sum parts [8][32], and the per-wave partial products [4][32][ck + 1]
// (in the E tile's space where they fit, else after the rest)
constexpr bool coord_part_in_e(int NT, int ck) { return 4 * 32 * (ck + 1) <= 32 * (NT * 32 + 1); }
constexpr int coord_lds_bytes(int NT, int ck) {
  return 32 * (NT * 32 + 1) * 4 + NT * 32 * (ck + 1) * 4 + 8 * 32 * 4 +
         (coord_part_in_e(NT, ck) ? 0 : 4 * 32 * (ck + 1) * 4);
}

// ---------------------------------------------------------------------------
// Forward.  Block = (window b, slab s of SW columns), 8 waves, wave w on query
// tile wave_tile(w); grid = batch * slabs, dealt so that the slabs of one
// window share an XCD (its coordinates are read from HBM once).  Per
// coupling: D = N_key + N_q - 2 G (one add, one FMA), the row sum, then the
// logit D * k2 and its exponential, its sum and (PARTNERS) the entropy term;
// the causal mask only on the diagonal tile.
// ---------------------------------------------------------------------------
template <int NT, int SW, bool PARTNERS>
__global__ __launch_bounds__(FT) void field_fwd_kernel(
    const float* __restrict__ p, const bf16* __restrict__ x, bf16* __restrict__ y,
    float* __restrict__ row_mean, float* __restrict__ lse, float* __restrict__ partners, int n,
    int c, int cp, int width, int slabs, float inv_tau, int scaled) {
  constexpr int NP = NT * 32, DT = SW / 32;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  bf16* sX = (bf16*)smem;
  float* sN = (float*)(smem + NP * SW * 2);
  bf16* sT = (bf16*)(smem + NP * SW * 2 + NP * 4);
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int b = lin / slabs, s = lin % slabs;
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int rs = ct_stride(cp);
  load_slab<NT, SW>(x + (size_t)b * n * width + (size_t)s * SW, width, n, sX);
  build_coords(p + (size_t)b * n * c, n, c, cp, NP, sT, sN);
  const int qt = wave_tile(wave);
  if (qt >= NT) return;
  const int q = qt * 32 + (lane & 31);
  const float nq = sN[q];
  f32x16 sc[NT];
  float dsum = 0.f;
#pragma unroll
  for (int kt = 0; kt < NT; kt++) {
    if (kt > qt) continue;
    f32x16 acc = gram_keys(sT, rs, cp, kt, q, lane);
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const f32x4 n4 = *(const f32x4*)(sN + kt * 32 + 8 * g + 4 * half);
#pragma unroll
      for (int r = 0; r < 4; r++) {
        const int e = 4 * g + r;
        float d = fmaf(acc[e], -2.f, n4[r] + nq);
        if (kt == qt && 8 * g + 4 * half + r >= (lane & 31)) d = 0.f;  // q itself, keys after q
        acc[e] = d;
        dsum += d;
      }
    }
    sc[kt] = acc;
  }
  dsum += __shfl_xor(dsum, 32);
  const float m = dsum / (float)(q + 1);
  const float k2 = -logit_scale(m, inv_tau, scaled) * LOG2E;
  float z = 0.f, za = 0.f;                  // sum of exp, sum of exp * logit (log2 units)
#pragma unroll
  for (int kt = 0; kt < NT; kt++) {
    if (kt > qt) continue;
#pragma unroll
    for (int e = 0; e < 16; e++) {
      const float a = sc[kt][e] * k2;
      float pe = __builtin_amdgcn_exp2f(a);
      if (kt == qt && att_masked(e, lane)) pe = 0.f;
      sc[kt][e] = pe;
      z += pe;
      if constexpr (PARTNERS) za += pe * a;
    }
  }
  z += __shfl_xor(z, 32);
  if constexpr (PARTNERS) za += __shfl_xor(za, 32);
  f32x16 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; dt++) o[dt] = f32x16{};
#pragma unroll
  for (int kt = 0; kt < NT; kt++) {
    if (kt > qt) continue;
#pragma unroll
    for (int mm = 0; mm < 2; mm++) {
      const bf16x8 pf = att_pack(sc[kt], mm);
#pragma unroll
      for (int dt = 0; dt < DT; dt++)
        o[dt] = mfma32(att_trfrag(sX + (dt / 2) * NP * 64, kt * 32 + 16 * mm, 32 * (dt % 2), lane),
                       pf, o[dt]);
    }
  }
  if (q >= n) return;
  // O^T register e of lane l: query q, column 32 dt + 8 (e / 4) + 4 half + e % 4
  const float inv = 1.f / z;
  bf16* yrow = y + ((size_t)b * n + q) * width + (size_t)s * SW;
#pragma unroll
  for (int dt = 0; dt < DT; dt++)
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const bf16x4 v = {to_bf16(o[dt][4 * g] * inv), to_bf16(o[dt][4 * g + 1] * inv),
                        to_bf16(o[dt][4 * g + 2] * inv), to_bf16(o[dt][4 * g + 3] * inv)};
      *(bf16x4*)(yrow + 32 * dt + 8 * g + 4 * half) = v;
    }
  if (s == 0 && half == 0) {
    const float l2z = __builtin_amdgcn_logf(z);         // log2 Z
    const size_t at = (size_t)b * n + q;
    row_mean[at] = m;
    lse[at] = l2z * LN2;
    if constexpr (PARTNERS) partners[at] = __builtin_amdgcn_exp2f(l2z - za * inv);
  }
}

// ---------------------------------------------------------------------------
// Backward, rows.  Block = (window b, query tile qt), the heaviest tiles of a
// window first; 8 waves, wave w owning key tile w (w <= qt).
// dP^T[key][q] = x_key . dy_q sums over the width in 64-column steps: each
// step's x rows [0, 32 (qt + 1)) and the tile's 32 dy rows go global -> LDS by
// DMA (coalesced, 8 rows of 128 bytes per instruction, swizzled as the 64-
// column tiles), NS stages in flight, the instructions of a step dealt over
// the 8 waves.  The couplings, their squared distances and the row sums come
// from the coordinate table first; the per-row sums Delta and sum(da D) across
// the waves go through LDS.
// ---------------------------------------------------------------------------
template <int NT, int NS>
__global__ __launch_bounds__(FT) void field_bwd_rows_kernel(
    const float* __restrict__ p, const bf16* __restrict__ x, const bf16* __restrict__ dy,
    const float* __restrict__ row_mean, const float* __restrict__ lse, float* __restrict__ ddt,
    int n, int c, int cp, int width, float inv_tau, int scaled) {
  constexpr int NP = NT * 32, STAGE = rows_stage_elems(NT);
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  bf16* sStage = (bf16*)smem;
  float* sN = (float*)(smem + NS * STAGE * 2);
  float* sRed = sN + NP;                              // [2][8 waves][32]
  bf16* sT = (bf16*)(sRed + 2 * 8 * 32);
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int b = lin / NT, qt = NT - 1 - lin % NT;
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int rs = ct_stride(cp);
  const int q = qt * 32 + (lane & 31);
  const bool qvalid = q < n;
  const bool own = wave <= qt;                        // this wave's key tile kt = wave
  const int steps = width / 64;
  // DMA plan of one step: instructions u < XI are x rows 8u .. 8u + 7, the
  // next 4 the tile's dy rows; wave w issues u = w, w + 8, ...  Rows past the
  // window read its last row (finite values that only reach couplings the
  // causal mask removes, or rows whose results are not used).
  const int XI = (qt + 1) * 4, TI = XI + 4;
  const int cnt = wave < TI ? (TI - 1 - wave) / 8 + 1 : 0;
  const bf16* xw = x + (size_t)b * n * width;
  const bf16* dyw = dy + (size_t)b * n * width;
  auto dma = [&](int st, int slot) {
    bf16* dst = sStage + slot * STAGE;
#pragma unroll
    for (int v = 0; v < 5; v++) {
      if (v < cnt) {
        const int u = wave + 8 * v;
        const int lr = 8 * u + (lane >> 3);               // row in the stage (x rows, then dy)
        const int tr = u < XI ? lr : qt * 32 + (lr - 8 * XI);   // row in the window
        const int gr = tr < n ? tr : n - 1;
        const int tile_row = u < XI ? lr : lr - 8 * XI;
        const int piece = (lane & 7) ^ att_sw(tile_row);
        const bf16* src = (u < XI ? xw : dyw) + (size_t)gr * width + st * 64 + 8 * piece;
        bf16* d0 = u < XI ? dst + u * 512 : dst + NP * 64 + (u - XI) * 512;
        dma16(src, d0);
      }
    }
  };
#pragma unroll
  for (int st = 0; st < NS - 1; st++)
    if (st < steps) dma(st, st);
  const float m_ld = row_mean[(size_t)b * n + min(q, n - 1)];
  const float l_ld = lse[(size_t)b * n + min(q, n - 1)];
  build_coords(p + (size_t)b * n * c, n, c, cp, (qt + 1) * 32, sT, sN);
  const float m = qvalid ? m_ld : 0.f;
  const float l2 = qvalid ? l_ld * LOG2E : 0.f;
  const float scale = qvalid ? logit_scale(m, inv_tau, scaled) : 0.f;
  const float k2 = -scale * LOG2E;
  const float nq = sN[q];
  f32x16 dd = {}, cc = {}, g = {};
  if (own) {
    f32x16 acc = gram_keys(sT, rs, cp, wave, q, lane);
#pragma unroll
    for (int gq = 0; gq < 4; gq++) {
      const f32x4 n4 = *(const f32x4*)(sN + wave * 32 + 8 * gq + 4 * half);
#pragma unroll
      for (int r = 0; r < 4; r++) {
        const int e = 4 * gq + r;
        const int lk = 8 * gq + 4 * half + r, lq = lane & 31;   // within the tiles
        const bool diag = wave == qt;
        float d = fmaf(acc[e], -2.f, n4[r] + nq);
        if (diag && lk >= lq) d = 0.f;                 // q itself, keys after q
        dd[e] = d;
        cc[e] = diag && lk > lq ? 0.f : __builtin_amdgcn_exp2f(d * k2 - l2);
      }
    }
  }
  for (int st = 0; st < steps; st++) {
    // this wave's DMA of step st has landed (those of the next NS - 2 steps may
    // still be in flight); after the barrier every wave's has, and every wave
    // is done with step st - 1, whose slot the next DMA overwrites
    const int later = min(NS - 2, steps - 1 - st);
    wait_vmcnt_upto(cnt * later);
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (st + NS - 1 < steps) dma(st + NS - 1, (st + NS - 1) % NS);
    if (own) {
      const bf16* cur = sStage + (st % NS) * STAGE;
#pragma unroll
      for (int ks = 0; ks < 4; ks++)
        g = mfma32(att_frag(cur, wave * 32, 16 * ks, lane),
                   att_frag(cur + NP * 64, 0, 16 * ks, lane), g);
    }
  }
  // Delta_q = sum_j C dP (in-lane, the lane ^ 32 exchange, then the 8 waves)
  float del = 0.f;
#pragma unroll
  for (int e = 0; e < 16; e++) del += cc[e] * g[e];
  del += __shfl_xor(del, 32);
  if (half == 0) sRed[wave * 32 + lane] = del;
  __syncthreads();
  del = 0.f;
#pragma unroll
  for (int w = 0; w < 8; w++) del += sRed[w * 32 + (lane & 31)];
  float tdm = 0.f;
#pragma unroll
  for (int e = 0; e < 16; e++) {
    const float da = cc[e] * (g[e] - del);
    g[e] = da;
    tdm += da * dd[e];
  }
  tdm += __shfl_xor(tdm, 32);
  if (half == 0) sRed[256 + wave * 32 + lane] = tdm;
  __syncthreads();
  if (!own) return;
  tdm = 0.f;
#pragma unroll
  for (int w = 0; w < 8; w++) tdm += sRed[256 + w * 32 + (lane & 31)];
  // dD = -scale da + [scaled, m > 0] (scale / m) (sum_j da D) / (q + 1)
  const float coef =
      (scaled && m > 0.f) ? scale * tdm / clamped_mean(m) / (float)(q + 1) : 0.f;
  float* dw = ddt + (size_t)b * NP * NP;
#pragma unroll
  for (int e = 0; e < 16; e++) {
    const int kk = wave * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
    dw[(size_t)kk * NP + q] = kk > q ? 0.f : -scale * g[e] + coef;
  }
}

// ---------------------------------------------------------------------------
// Backward, dx.  Block = (window b, slab s of SW columns), 8 waves, wave w on
// key tile wave_tile(w), a lane one key j; C[q][j] is recomputed from the
// forward's m and ln Z (one add, two FMAs and the exponential per coupling,
// the mask only on the diagonal tile), and dx^T[col][j] += dy^T[col][q]
// C[q][j] as in the attention core's dV.
// ---------------------------------------------------------------------------
template <int NT, int SW>
__global__ __launch_bounds__(FT) void field_bwd_dx_kernel(
    const float* __restrict__ p, const float* __restrict__ row_mean, const float* __restrict__ lse,
    const bf16* __restrict__ dy, bf16* __restrict__ dx, int n, int c, int cp, int width,
    int slabs, float inv_tau, int scaled) {
  constexpr int NP = NT * 32, DT = SW / 32;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  bf16* sDY = (bf16*)smem;
  float* sN = (float*)(smem + NP * SW * 2);
  float* sK2 = sN + NP;                       // -scale_q log2 e
  float* sL2 = sK2 + NP;                      // -ln Z_q log2 e
  bf16* sT = (bf16*)(sL2 + NP);
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int b = lin / slabs, s = lin % slabs;
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int rs = ct_stride(cp);
  if (threadIdx.x < NP) {
    const int q = threadIdx.x;
    const bool v = q < n;
    const float m = row_mean[(size_t)b * n + min(q, n - 1)];
    const float l = lse[(size_t)b * n + min(q, n - 1)];
    sK2[q] = v ? -logit_scale(m, inv_tau, scaled) * LOG2E : 0.f;
    sL2[q] = v ? -l * LOG2E : 0.f;
  }
  load_slab<NT, SW>(dy + (size_t)b * n * width + (size_t)s * SW, width, n, sDY);
  build_coords(p + (size_t)b * n * c, n, c, cp, NP, sT, sN);
  const int kt = wave_tile(wave);
  if (kt >= NT) return;
  const int j = kt * 32 + (lane & 31);
  const float nj = sN[j];
  f32x16 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; dt++) o[dt] = f32x16{};
#pragma unroll
  for (int qt = 0; qt < NT; qt++) {
    if (qt < kt) continue;
    f32x16 acc = gram_queries(sT, rs, cp, qt, j, lane);
    // register e: query qt*32 + 8 (e/4) + 4 half + e%4, key j
#pragma unroll
    for (int gq = 0; gq < 4; gq++) {
      const int q0 = qt * 32 + 8 * gq + 4 * half;
      const f32x4 n4 = *(const f32x4*)(sN + q0);
      const f32x4 k4 = *(const f32x4*)(sK2 + q0);
      const f32x4 l4 = *(const f32x4*)(sL2 + q0);
#pragma unroll
      for (int r = 0; r < 4; r++) {
        const int e = 4 * gq + r;
        const int lq = 8 * gq + 4 * half + r, lj = lane & 31;   // within the tiles
        float d = fmaf(acc[e], -2.f, n4[r] + nj);
        if (qt == kt && lq == lj) d = 0.f;                     // the diagonal
        float ce = __builtin_amdgcn_exp2f(fmaf(d, k4[r], l4[r]));
        if (qt == kt && lq < lj) ce = 0.f;                     // query before j
        acc[e] = ce;
      }
    }
#pragma unroll
    for (int mm = 0; mm < 2; mm++) {
      const bf16x8 pf = att_pack(acc, mm);
#pragma unroll
      for (int dt = 0; dt < DT; dt++)
        o[dt] = mfma32(att_trfrag(sDY + (dt / 2) * NP * 64, qt * 32 + 16 * mm, 32 * (dt % 2), lane),
                       pf, o[dt]);
    }
  }
  if (j >= n) return;
  bf16* xrow = dx + ((size_t)b * n + j) * width + (size_t)s * SW;
#pragma unroll
  for (int dt = 0; dt < DT; dt++)
#pragma unroll
    for (int gq = 0; gq < 4; gq++) {
      const bf16x4 v = {to_bf16(o[dt][4 * gq]), to_bf16(o[dt][4 * gq + 1]),
                        to_bf16(o[dt][4 * gq + 2]), to_bf16(o[dt][4 * gq + 3])};
      *(bf16x4*)(xrow + 32 * dt + 8 * gq + 4 * half) = v;
    }
}

// ---------------------------------------------------------------------------
// Backward, coordinates.  Block = (window b, row tile t), 4 waves: E[i][j] for
// the tile's 32 rows i and every j (dD[i][j] = ddt[j][i] for j < i, dD[j][i] =
// ddt[i][j] for j > i; 0 at j = i and outside the window) into LDS; then
//   dp_i = 2 (sum_j E[i][j]) p'_i - 2 sum_j E[i][j] p'_j,  p' = p - p_0,
// the second sum on the fp32 matrix cores (32 x 32 x 2: A = p'^T, B = E^T),
// wave w taking a quarter of the j range; partial products meet in LDS.
// ---------------------------------------------------------------------------
template <int NT, int CK>
__global__ __launch_bounds__(FTC) void field_bwd_coord_kernel(const float* __restrict__ p,
                                                             const float* __restrict__ ddt,
                                                             float* __restrict__ dp, int n,
                                                             int c) {
  constexpr int NP = NT * 32, ES = NP + 1, CKP = CK + 1;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  float* sE = (float*)smem;                          // [32][ES]
  float* sP = sE + 32 * ES;                          // [NP][CKP]
  float* sRowPart = sP + NP * CKP;                   // [8][32]
  float* sPart = coord_part_in_e(NT, CK) ? sE : sRowPart + 8 * 32;   // [4][32][CKP]
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int b = lin / NT, t = lin % NT;
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const float* pw = p + (size_t)b * n * c;
  const float* dw = ddt + (size_t)b * NP * NP;
  // E: element u of this thread is e = tid + 256 u of the 32 * NP entries,
  // first those with j < (t + 1) * 32 (j = e / 32, consecutive i along ddt
  // rows j, or ddt[i][j] for j > i), then the rest (i = e' / rest, j
  // contiguous along ddt rows i).  All loads before the first LDS write; every
  // address lies in the window's NP x NP workspace, and the entries that are
  // not part of E (j = i, outside the window) are replaced by 0.
  constexpr int PER = NT * 4;
  const int split = (t + 1) * 32 * 32, rest = NP - (t + 1) * 32;
  float ev[PER];
#pragma unroll
  for (int u = 0; u < PER; u++) {
    const int e = threadIdx.x + FTC * u;
    int ii, j;
    if (e < split) {
      j = e >> 5;
      ii = e & 31;
    } else {
      ii = (e - split) / rest;
      j = (t + 1) * 32 + (e - split) % rest;
    }
    const int i = t * 32 + ii;
    const float v = dw[j < i ? (size_t)j * NP + i : (size_t)i * NP + j];
    ev[u] = (i < n && j < n && j != i) ? v : 0.f;
  }
  // coordinates: rows past the window zero (their E entries are 0, so they
  // must be finite); columns past c are left as they are (they only reach
  // output rows that are not used)
  for (int idx = threadIdx.x; idx < (NP - n) * CKP; idx += FTC) sP[n * CKP + idx] = 0.f;
  stage_coords<FTC, 64>(pw, n, c, (unsigned char*)sP, CKP * 4);
#pragma unroll
  for (int u = 0; u < PER; u++) {
    const int e = threadIdx.x + FTC * u;
    int ii, j;
    if (e < split) {
      j = e >> 5;
      ii = e & 31;
    } else {
      ii = (e - split) / rest;
      j = (t + 1) * 32 + (e - split) % rest;
    }
    sE[ii * ES + j] = ev[u];
  }
  __syncthreads();
  {
    // row sums: lane group of 32 = the 32 rows at one j, 8 groups over j
    const int ii = threadIdx.x & 31, part = threadIdx.x >> 5;
    float rsum = 0.f;
    for (int j = part; j < NP; j += 8) rsum += sE[ii * ES + j];
    sRowPart[part * 32 + ii] = rsum;
  }
  constexpr int JW = NP / 4;                         // j range of one wave
  f32x16 acc[CK / 32];
#pragma unroll
  for (int kc = 0; kc < CK / 32; kc++) acc[kc] = f32x16{};
  float p0[CK / 32];                                 // p_0 at this lane's coordinates
#pragma unroll
  for (int kc = 0; kc < CK / 32; kc++) p0[kc] = sP[kc * 32 + (lane & 31)];
  for (int js = 0; js < JW; js += 2) {
    const int j = wave * JW + js + half;
    const float bv = sE[(lane & 31) * ES + j];       // B[k = half][col i] = E[i][j]
#pragma unroll
    for (int kc = 0; kc < CK / 32; kc++) {
      // A[row k][half] = p'_j[k] = p_j[k] - p_0[k]
      const float av = sP[j * CKP + kc * 32 + (lane & 31)] - p0[kc];
      acc[kc] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc[kc], 0, 0, 0);
    }
  }
  __syncthreads();                                   // sE may be reused for the partials
  // register e: coordinate k = kc*32 + 8 (e/4) + 4 half + e%4, row i = lane % 32
#pragma unroll
  for (int kc = 0; kc < CK / 32; kc++)
#pragma unroll
    for (int e = 0; e < 16; e++) {
      const int k = kc * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
      sPart[(wave * 32 + (lane & 31)) * CKP + k] = acc[kc][e];
    }
  __syncthreads();
  for (int idx = threadIdx.x; idx < 32 * c; idx += FTC) {
    const int ii = idx / c, k = idx % c, i = t * 32 + ii;
    if (i >= n) continue;
    float rsum = 0.f;
#pragma unroll
    for (int part = 0; part < 8; part++) rsum += sRowPart[part * 32 + ii];
    const float ep = sPart[(0 * 32 + ii) * CKP + k] + sPart[(1 * 32 + ii) * CKP + k] +
                     sPart[(2 * 32 + ii) * CKP + k] + sPart[(3 * 32 + ii) * CKP + k];
    dp[((size_t)b * n + i) * c + k] = 2.f * (rsum * (sP[i * CKP + k] - sP[k]) - ep);
  }
}

template <int NT, int SW, bool PARTNERS>
hipError_t field_fwd_launch(const float* p, const bf16* x, bf16* y, float* row_mean, float* lse,
                            float* partners, int batch, int n, int c, int cp, int width,
                            float inv_tau, int scaled, hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  hipError_t e = lds_limit_once(done, (const void*)field_fwd_kernel<NT, SW, PARTNERS>,
                                fwd_lds_bytes(NT, SW, 64));
  if (e != hipSuccess) return e;
  const int slabs = width / SW;
  field_fwd_kernel<NT, SW, PARTNERS><<<batch * slabs, FT, fwd_lds_bytes(NT, SW, cp), st>>>(
      p, x, y, row_mean, lse, partners, n, c, cp, width, slabs, inv_tau, scaled);
  return hipGetLastError();
}

template <int NT>
hipError_t field_fwd_pick(const float* p, const bf16* x, bf16* y, float* row_mean, float* lse,
                          float* partners, int batch, int n, int c, int cp, int width,
                          float inv_tau, int scaled, hipStream_t st) {
  const bool wide = width % 128 == 0;
  if (partners)
    return wide ? field_fwd_launch<NT, 128, true>(p, x, y, row_mean, lse, partners, batch, n, c,
                                                  cp, width, inv_tau, scaled, st)
                : field_fwd_launch<NT, 64, true>(p, x, y, row_mean, lse, partners, batch, n, c,
                                                 cp, width, inv_tau, scaled, st);
  return wide ? field_fwd_launch<NT, 128, false>(p, x, y, row_mean, lse, partners, batch, n, c,
                                                 cp, width, inv_tau, scaled, st)
              : field_fwd_launch<NT, 64, false>(p, x, y, row_mean, lse, partners, batch, n, c, cp,
                                                width, inv_tau, scaled, st);
}

template <int NT, int SW>
hipError_t field_dx_launch(const float* p, const float* row_mean, const float* lse,
                           const bf16* dy, bf16* dx, int batch, int n, int c, int cp, int width,
                           float inv_tau, int scaled, hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  hipError_t e = lds_limit_once(done, (const void*)field_bwd_dx_kernel<NT, SW>,
                                dx_lds_bytes(NT, SW, 64));
  if (e != hipSuccess) return e;
  const int slabs = width / SW;
  field_bwd_dx_kernel<NT, SW><<<batch * slabs, FT, dx_lds_bytes(NT, SW, cp), st>>>(
      p, row_mean, lse, dy, dx, n, c, cp, width, slabs, inv_tau, scaled);
  return hipGetLastError();
}

template <int NT, int NS>
hipError_t field_rows_launch(const float* p, const bf16* x, const float* row_mean,
                             const float* lse, const bf16* dy, float* ddt, int batch, int n,
                             int c, int cp, int width, float inv_tau, int scaled, hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  hipError_t e = lds_limit_once(done, (const void*)field_bwd_rows_kernel<NT, NS>, 160 * 1024);
  if (e != hipSuccess) return e;
  field_bwd_rows_kernel<NT, NS><<<batch * NT, FT, rows_lds_bytes(NT, NS, cp), st>>>(
      p, x, dy, row_mean, lse, ddt, n, c, cp, width, inv_tau, scaled);
  return hipGetLastError();
}

template <int NT, int CK>
hipError_t field_coord_launch(const float* p, const float* ddt, float* dp, int batch, int n,
                              int c, hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  hipError_t e = lds_limit_once(done, (const void*)field_bwd_coord_kernel<NT, CK>,
                                coord_lds_bytes(NT, CK));
  if (e != hipSuccess) return e;
  field_bwd_coord_kernel<NT, CK><<<batch * NT, FTC, coord_lds_bytes(NT, CK), st>>>(p, ddt, dp, n,
                                                                                  c);
  return hipGetLastError();
}

template <int NT>
hipError_t field_bwd_launch(const float* p, const bf16* x, const float* row_mean,
                            const float* lse, const bf16* dy, float* dp, bf16* dx, float* ddt,
                            int batch, int n, int c, int cp, int width, float inv_tau, int scaled,
                            hipStream_t st) {
  hipError_t e = rows_stages(NT, cp) == 3
                     ? field_rows_launch<NT, 3>(p, x, row_mean, lse, dy, ddt, batch, n, c, cp,
                                                width, inv_tau, scaled, st)
                     : field_rows_launch<NT, 2>(p, x, row_mean, lse, dy, ddt, batch, n, c, cp,
                                                width, inv_tau, scaled, st);
  if (e != hipSuccess) return e;
  e = width % 128 == 0 ? field_dx_launch<NT, 128>(p, row_mean, lse, dy, dx, batch, n, c, cp,
                                                   width, inv_tau, scaled, st)
                       : field_dx_launch<NT, 64>(p, row_mean, lse, dy, dx, batch, n, c, cp, width,
                                                 inv_tau, scaled, st);
  if (e != hipSuccess) return e;
  return c <= 32 ? field_coord_launch<NT, 32>(p, ddt, dp, batch, n, c, st)
                 : field_coord_launch<NT, 64>(p, ddt, dp, batch, n, c, st);
}

}  // namespace

#define HCMIX_FIELD_CASES(F, ...)            \
  switch ((n + 31) / 32) {                   \
    case 1: return F<1>(__VA_ARGS__);        \
    case 2: return F<2>(__VA_ARGS__);        \
    case 3: return F<3>(__VA_ARGS__);        \
    case 4: return F<4>(__VA_ARGS__);        \
    case 5: return F<5>(__VA_ARGS__);        \
    case 6: return F<6>(__VA_ARGS__);        \
    case 7: return F<7>(__VA_ARGS__);        \
    case 8: return F<8>(__VA_ARGS__);        \
    default: return hipErrorInvalidValue;    \
  }

hipError_t launch_field_fwd(const float* p, const bf16* x, bf16* y, float* row_mean, float* lse,
                            float* partners, int batch, int n, int c, int width, float inv_tau,
                            int scaled, hipStream_t st) {
  const int cp = (c + 15) / 16 * 16;
  HCMIX_FIELD_CASES(field_fwd_pick, p, x, y, row_mean, lse, partners, batch, n, c, cp, width,
                    inv_tau, scaled, st)
}

hipError_t launch_field_bwd(const float* p, const bf16* x, const float* row_mean,
                            const float* lse, const bf16* dy, float* dp, bf16* dx, float* ddt,
                            int batch, int n, int c, int width, float inv_tau, int scaled,
                            hipStream_t st) {
  const int cp = (c + 15) / 16 * 16;
  HCMIX_FIELD_CASES(field_bwd_launch, p, x, row_mean, lse, dy, dp, dx, ddt, batch, n, c, cp,
                    width, inv_tau, scaled, st)
}
#undef HCMIX_FIELD_CASES

}  // namespace hcmix
