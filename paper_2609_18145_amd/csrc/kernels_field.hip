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
// 2^-17 of the norms).  The diagonal is set to exactly 0 and negative values
// (rounding) to 0.  Every logit is <= 0 and the diagonal's is 0, so each
// row's maximum is known: the exponentials need no running maximum and Z_i
// lies in [1, i + 1].
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

constexpr int FT = 256;                       // threads per block (4 waves)
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

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

// Rows [0, rows) of the table and their squared norms N_r (of hi + lo, fp32),
// from the window's coordinates pw [n][c].  Rows >= n are zero.
__device__ __forceinline__ void build_coords(const float* __restrict__ pw, int n, int c, int cp,
                                             int rows, bf16* sT, float* sN) {
  const int rs = ct_stride(cp);
  for (int r = threadIdx.x; r < rows; r += FT) {
    float nn = 0.f;
    bf16* row = sT + r * rs;
    for (int k = 0; k < cp; k++) {
      float v = 0.f;
      if (r < n && k < c) v = pw[(size_t)r * c + k] - pw[k];
      const bf16 hi = to_bf16(v);
      const bf16 lo = to_bf16(v - (float)hi);
      row[k] = hi;
      row[cp + k] = lo;
      const float t = (float)hi + (float)lo;
      nn = fmaf(t, t, nn);
    }
#pragma unroll
    for (int k = 0; k < 8; k++) row[2 * cp + k] = to_bf16(0.f);
    sN[r] = nn;
  }
}

// Rows [0, NT * 32) of one 64-column slab (src: row 0, rows `stride` apart)
// into a swizzled LDS tile; rows >= n are zero.  Every load is in flight
// before the first LDS write.
template <int NT>
__device__ __forceinline__ void load_slab(const bf16* __restrict__ src, size_t stride, int n,
                                          bf16* tile) {
  constexpr int PER = NT;                     // NT * 32 rows * 8 pieces / FT
  u32x4 v[PER];
#pragma unroll
  for (int j = 0; j < PER; j++) {
    const int pi = threadIdx.x + FT * j, r = pi >> 3, pc = pi & 7;
    v[j] = u32x4{0u, 0u, 0u, 0u};
    if (r < n) v[j] = *(const u32x4*)(src + (size_t)r * stride + 8 * pc);
  }
#pragma unroll
  for (int j = 0; j < PER; j++) {
    const int pi = threadIdx.x + FT * j, r = pi >> 3, pc = pi & 7;
    *(u32x4*)(tile + att_off(r, 8 * pc)) = v[j];
  }
}

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
constexpr int fwd_lds_bytes(int NT, int cp) {
  return NT * 32 * HD * 2 + NT * 32 * 4 + NT * 32 * (2 * cp + 8) * 2;
}
constexpr int rows_lds_bytes(int NT, int cp) {
  return NT * 32 * 4 + 2 * 4 * 32 * 4 + NT * 32 * (2 * cp + 8) * 2;
}
constexpr int dx_lds_bytes(int NT, int cp) {
  return NT * 32 * HD * 2 + 3 * NT * 32 * 4 + NT * 32 * (2 * cp + 8) * 2;
}
// coordinate kernel: E tile [32][NP + 1] fp32, centred coordinates [NP][ck]
// fp32 (ck = 32 or 64), row sums [32]; the per-wave partial products
// [4][ck][32] reuse the E tile's space where it is large enough, else follow.
constexpr bool coord_part_in_e(int NT, int ck) { return 4 * ck * 32 <= 32 * (NT * 32 + 1); }
constexpr int coord_lds_bytes(int NT, int ck) {
  return 32 * (NT * 32 + 1) * 4 + NT * 32 * ck * 4 + 32 * 4 +
         (coord_part_in_e(NT, ck) ? 0 : 4 * ck * 32 * 4);
}

// ---------------------------------------------------------------------------
// Forward.  Block = (window b, slab s); grid = batch * slabs, dealt so that the
// slabs of one window share an XCD (its coordinates are read once).
// ---------------------------------------------------------------------------
template <int NT>
__global__ __launch_bounds__(FT, 1) void field_fwd_kernel(
    const float* __restrict__ p, const bf16* __restrict__ x, bf16* __restrict__ y,
    float* __restrict__ row_mean, float* __restrict__ lse, float* __restrict__ partners, int n,
    int c, int cp, int width, int slabs, float inv_tau, int scaled) {
  constexpr int NP = NT * 32;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  bf16* sX = (bf16*)smem;
  float* sN = (float*)(smem + NP * HD * 2);
  bf16* sT = (bf16*)(smem + NP * HD * 2 + NP * 4);
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int b = lin / slabs, s = lin % slabs;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
  const int rs = ct_stride(cp);
  load_slab<NT>(x + (size_t)b * n * width + (size_t)s * HD, width, n, sX);
  build_coords(p + (size_t)b * n * c, n, c, cp, NP, sT, sN);
  __syncthreads();
#pragma unroll
  for (int which = 0; which < 2; which++) {
    const int qt = att_tile(wave, which);
    if (qt >= NT) continue;
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
          const int e = 4 * g + r, key = kt * 32 + 8 * g + 4 * half + r;
          float d = fmaxf(n4[r] + nq - 2.f * acc[e], 0.f);
          if (key >= q) d = 0.f;            // the diagonal, and keys after q (masked below)
          acc[e] = d;
          dsum += d;
        }
      }
      sc[kt] = acc;
    }
    dsum += __shfl_xor(dsum, 32);
    const float m = dsum / (float)(q + 1);
    const float k2 = -logit_scale(m, inv_tau, scaled) * LOG2E;
    float z = 0.f, za = 0.f;                // sum of exp, sum of exp * logit (log2 units)
#pragma unroll
    for (int kt = 0; kt < NT; kt++) {
      if (kt > qt) continue;
#pragma unroll
      for (int e = 0; e < 16; e++) {
        const float a = sc[kt][e] * k2;
        const float pe = (kt == qt && att_masked(e, lane)) ? 0.f : __builtin_amdgcn_exp2f(a);
        sc[kt][e] = pe;
        z += pe;
        za += pe * a;
      }
    }
    z += __shfl_xor(z, 32);
    za += __shfl_xor(za, 32);
    f32x16 o[2] = {};
#pragma unroll
    for (int kt = 0; kt < NT; kt++) {
      if (kt > qt) continue;
#pragma unroll
      for (int mm = 0; mm < 2; mm++) {
        const bf16x8 pf = att_pack(sc[kt], mm);
#pragma unroll
        for (int dt = 0; dt < 2; dt++)
          o[dt] = mfma32(att_trfrag(sX, kt * 32 + 16 * mm, 32 * dt, lane), pf, o[dt]);
      }
    }
    if (q >= n) continue;
    // O^T register e of lane l: query q, column 32 dt + 8 (e / 4) + 4 half + e % 4
    const float inv = 1.f / z;
    bf16* yrow = y + ((size_t)b * n + q) * width + (size_t)s * HD;
#pragma unroll
    for (int dt = 0; dt < 2; dt++)
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const bf16x4 v = {to_bf16(o[dt][4 * g] * inv), to_bf16(o[dt][4 * g + 1] * inv),
                          to_bf16(o[dt][4 * g + 2] * inv), to_bf16(o[dt][4 * g + 3] * inv)};
        *(bf16x4*)(yrow + 32 * dt + 8 * g + 4 * half) = v;
      }
    if (s == 0 && half == 0) {
      const float l2z = __builtin_amdgcn_logf(z);       // log2 Z
      const size_t at = (size_t)b * n + q;
      row_mean[at] = m;
      lse[at] = l2z * LN2;
      if (partners) partners[at] = __builtin_amdgcn_exp2f(l2z - za * inv);
    }
  }
}

// ---------------------------------------------------------------------------
// Backward, rows.  Block = (window b, query tile qt), the heaviest tiles of a
// window first; wave w owns key tiles w and w + 4.  dP^T[key][query] sums
// x_key . dy_q over the width in 64-column steps, both operands read straight
// from global memory (one 64-byte piece per lane and row: within a step,
// lane half h takes columns 32 h .. 32 h + 31, in the same order for both
// operands, so the contraction covers each column once), the next step's
// pieces loaded while the current one is multiplied.  Row sums across the
// waves go through LDS.
// ---------------------------------------------------------------------------
template <int NT>
__global__ __launch_bounds__(FT, 1) void field_bwd_rows_kernel(
    const float* __restrict__ p, const bf16* __restrict__ x, const bf16* __restrict__ dy,
    const float* __restrict__ row_mean, const float* __restrict__ lse, float* __restrict__ ddt,
    int n, int c, int cp, int width, float inv_tau, int scaled) {
  constexpr int NP = NT * 32;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  float* sN = (float*)smem;
  float* sRed = (float*)(smem + NP * 4);              // [2][4 waves][32]
  bf16* sT = (bf16*)(smem + NP * 4 + 2 * 4 * 32 * 4);
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int b = lin / NT, qt = NT - 1 - lin % NT;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
  const int rs = ct_stride(cp);
  build_coords(p + (size_t)b * n * c, n, c, cp, (qt + 1) * 32, sT, sN);
  __syncthreads();
  const int q = qt * 32 + (lane & 31);
  const bool qvalid = q < n;
  const float m = qvalid ? row_mean[(size_t)b * n + q] : 0.f;
  const float l2 = qvalid ? lse[(size_t)b * n + q] * LOG2E : 0.f;
  const float scale = qvalid ? logit_scale(m, inv_tau, scaled) : 0.f;
  const float k2 = -scale * LOG2E;
  const float nq = sN[q];
  f32x16 dd[2], cc[2], g[2];
#pragma unroll
  for (int t = 0; t < 2; t++) {
    dd[t] = f32x16{};
    cc[t] = f32x16{};
    g[t] = f32x16{};
    const int kt = wave + 4 * t;
    if (kt > qt) continue;
    f32x16 acc = gram_keys(sT, rs, cp, kt, q, lane);
#pragma unroll
    for (int gq = 0; gq < 4; gq++) {
      const f32x4 n4 = *(const f32x4*)(sN + kt * 32 + 8 * gq + 4 * half);
#pragma unroll
      for (int r = 0; r < 4; r++) {
        const int e = 4 * gq + r, key = kt * 32 + 8 * gq + 4 * half + r;
        float d = fmaxf(n4[r] + nq - 2.f * acc[e], 0.f);
        if (key >= q) d = 0.f;
        dd[t][e] = d;
        cc[t][e] = key > q ? 0.f : __builtin_amdgcn_exp2f(d * k2 - l2);
      }
    }
  }
  // dP^T over the width
  const bf16* xw = x + (size_t)b * n * width;
  const bf16* dyq = dy + ((size_t)b * n + q) * width;
  const bf16x8 zero8 = {};
  bf16x8 ca[2][4], cb[4], na[2][4], nb[4];
#pragma unroll
  for (int ks = 0; ks < 4; ks++) {
    cb[ks] = qvalid ? *(const bf16x8*)(dyq + 32 * half + 8 * ks) : zero8;
#pragma unroll
    for (int t = 0; t < 2; t++) {
      const int key = (wave + 4 * t) * 32 + (lane & 31);
      const bool ok = wave + 4 * t <= qt && key < n;
      ca[t][ks] = ok ? *(const bf16x8*)(xw + (size_t)key * width + 32 * half + 8 * ks) : zero8;
    }
  }
  for (int w0 = 0; w0 < width; w0 += 64) {
    const int w1 = w0 + 64;
    if (w1 < width) {
#pragma unroll
      for (int ks = 0; ks < 4; ks++) {
        nb[ks] = qvalid ? *(const bf16x8*)(dyq + w1 + 32 * half + 8 * ks) : zero8;
#pragma unroll
        for (int t = 0; t < 2; t++) {
          const int key = (wave + 4 * t) * 32 + (lane & 31);
          const bool ok = wave + 4 * t <= qt && key < n;
          na[t][ks] =
              ok ? *(const bf16x8*)(xw + (size_t)key * width + w1 + 32 * half + 8 * ks) : zero8;
        }
      }
    }
#pragma unroll
    for (int t = 0; t < 2; t++) {
      if (wave + 4 * t > qt) continue;
#pragma unroll
      for (int ks = 0; ks < 4; ks++) g[t] = mfma32(ca[t][ks], cb[ks], g[t]);
    }
#pragma unroll
    for (int ks = 0; ks < 4; ks++) {
      cb[ks] = nb[ks];
#pragma unroll
      for (int t = 0; t < 2; t++) ca[t][ks] = na[t][ks];
    }
  }
  // Delta_q = sum_j C dP (in-lane, the lane ^ 32 exchange, then the 4 waves)
  float del = 0.f;
#pragma unroll
  for (int t = 0; t < 2; t++)
#pragma unroll
    for (int e = 0; e < 16; e++) del += cc[t][e] * g[t][e];
  del += __shfl_xor(del, 32);
  if (half == 0) sRed[wave * 32 + lane] = del;
  __syncthreads();
  del = sRed[lane & 31] + sRed[32 + (lane & 31)] + sRed[64 + (lane & 31)] +
        sRed[96 + (lane & 31)];
  float tdm = 0.f;
#pragma unroll
  for (int t = 0; t < 2; t++)
#pragma unroll
    for (int e = 0; e < 16; e++) {
      const float da = cc[t][e] * (g[t][e] - del);
      g[t][e] = da;
      tdm += da * dd[t][e];
    }
  tdm += __shfl_xor(tdm, 32);
  if (half == 0) sRed[128 + wave * 32 + lane] = tdm;
  __syncthreads();
  tdm = sRed[128 + (lane & 31)] + sRed[160 + (lane & 31)] + sRed[192 + (lane & 31)] +
        sRed[224 + (lane & 31)];
  // dD = -scale da + [scaled, m > 0] (scale / m) (sum_j da D) / (q + 1)
  const float coef =
      (scaled && m > 0.f) ? scale * tdm / clamped_mean(m) / (float)(q + 1) : 0.f;
  float* dw = ddt + (size_t)b * NP * NP;
#pragma unroll
  for (int t = 0; t < 2; t++) {
    const int kt = wave + 4 * t;
    if (kt > qt) continue;
#pragma unroll
    for (int e = 0; e < 16; e++) {
      const int key = kt * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
      dw[(size_t)key * NP + q] = key > q ? 0.f : -scale * g[t][e] + coef;
    }
  }
}

// ---------------------------------------------------------------------------
// Backward, dx.  Block = (window b, slab s); wave w owns key tiles w and
// 7 - w, a lane one key j; C[q][j] is recomputed from the forward's m and
// ln Z, and dx^T[col][j] += dy^T[col][q] C[q][j] as in the attention core's
// dV.
// ---------------------------------------------------------------------------
template <int NT>
__global__ __launch_bounds__(FT, 1) void field_bwd_dx_kernel(
    const float* __restrict__ p, const float* __restrict__ row_mean, const float* __restrict__ lse,
    const bf16* __restrict__ dy, bf16* __restrict__ dx, int n, int c, int cp, int width,
    int slabs, float inv_tau, int scaled) {
  constexpr int NP = NT * 32;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  bf16* sDY = (bf16*)smem;
  float* sN = (float*)(smem + NP * HD * 2);
  float* sK2 = sN + NP;                       // -scale_q log2 e
  float* sL2 = sK2 + NP;                      // ln Z_q log2 e
  bf16* sT = (bf16*)(sL2 + NP);
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int b = lin / slabs, s = lin % slabs;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
  const int rs = ct_stride(cp);
  load_slab<NT>(dy + (size_t)b * n * width + (size_t)s * HD, width, n, sDY);
  build_coords(p + (size_t)b * n * c, n, c, cp, NP, sT, sN);
  for (int q = threadIdx.x; q < NP; q += FT) {
    const bool v = q < n;
    const float m = v ? row_mean[(size_t)b * n + q] : 0.f;
    sK2[q] = v ? -logit_scale(m, inv_tau, scaled) * LOG2E : 0.f;
    sL2[q] = v ? lse[(size_t)b * n + q] * LOG2E : 0.f;
  }
  __syncthreads();
#pragma unroll
  for (int which = 0; which < 2; which++) {
    const int kt = att_tile(wave, which);
    if (kt >= NT) continue;
    const int j = kt * 32 + (lane & 31);
    const float nj = sN[j];
    f32x16 o[2] = {};
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
          const int e = 4 * gq + r, qq = q0 + r;
          float d = fmaxf(n4[r] + nj - 2.f * acc[e], 0.f);
          if (qq == j) d = 0.f;
          acc[e] = qq < j ? 0.f : __builtin_amdgcn_exp2f(d * k4[r] - l4[r]);
        }
      }
#pragma unroll
      for (int mm = 0; mm < 2; mm++) {
        const bf16x8 pf = att_pack(acc, mm);
#pragma unroll
        for (int dt = 0; dt < 2; dt++)
          o[dt] = mfma32(att_trfrag(sDY, qt * 32 + 16 * mm, 32 * dt, lane), pf, o[dt]);
      }
    }
    if (j >= n) continue;
    bf16* xrow = dx + ((size_t)b * n + j) * width + (size_t)s * HD;
#pragma unroll
    for (int dt = 0; dt < 2; dt++)
#pragma unroll
      for (int gq = 0; gq < 4; gq++) {
        const bf16x4 v = {to_bf16(o[dt][4 * gq]), to_bf16(o[dt][4 * gq + 1]),
                          to_bf16(o[dt][4 * gq + 2]), to_bf16(o[dt][4 * gq + 3])};
        *(bf16x4*)(xrow + 32 * dt + 8 * gq + 4 * half) = v;
      }
  }
}

// ---------------------------------------------------------------------------
// Backward, coordinates.  Block = (window b, row tile t): E[i][j] for the
// tile's 32 rows i and every j (dD[i][j] = ddt[j][i] for j < i, dD[j][i] =
// ddt[i][j] for j > i; 0 at j = i and outside the window) into LDS; then
//   dp_i = 2 (sum_j E[i][j]) p'_i - 2 sum_j E[i][j] p'_j,
// the second sum on the fp32 matrix cores (32 x 32 x 2: A = p'^T, B = E^T),
// wave w taking a quarter of the j range; partial products meet in LDS.
// ---------------------------------------------------------------------------
template <int NT, int CK>
__global__ __launch_bounds__(FT, 1) void field_bwd_coord_kernel(const float* __restrict__ p,
                                                                const float* __restrict__ ddt,
                                                                float* __restrict__ dp, int n,
                                                                int c) {
  constexpr int NP = NT * 32, ES = NP + 1;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  float* sE = (float*)smem;                          // [32][ES]
  float* sP = sE + 32 * ES;                          // [NP][CK]
  float* sRow = sP + NP * CK;                        // [32]
  float* sPart = coord_part_in_e(NT, CK) ? sE : sRow + 32;   // [4][CK][32]
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int b = lin / NT, t = lin % NT;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
  const float* pw = p + (size_t)b * n * c;
  const float* dw = ddt + (size_t)b * NP * NP;
  for (int idx = threadIdx.x; idx < NP * CK; idx += FT) {
    const int r = idx / CK, k = idx % CK;
    sP[idx] = (r < n && k < c) ? pw[(size_t)r * c + k] - pw[k] : 0.f;
  }
  // j < (t + 1) * 32: reads along ddt rows j (32 consecutive i), or ddt[i][j] for j > i
  for (int idx = threadIdx.x; idx < (t + 1) * 32 * 32; idx += FT) {
    const int j = idx >> 5, ii = idx & 31, i = t * 32 + ii;
    float v = 0.f;
    if (i < n && j < n && j != i) v = j < i ? dw[(size_t)j * NP + i] : dw[(size_t)i * NP + j];
    sE[ii * ES + j] = v;
  }
  // j >= (t + 1) * 32: E[i][j] = ddt[i][j], contiguous in j
  const int rest = NP - (t + 1) * 32;
  for (int idx = threadIdx.x; idx < 32 * rest; idx += FT) {
    const int ii = idx / rest, j = (t + 1) * 32 + idx % rest, i = t * 32 + ii;
    sE[ii * ES + j] = (i < n && j < n) ? dw[(size_t)i * NP + j] : 0.f;
  }
  __syncthreads();
  {
    const int ii = threadIdx.x >> 3, part = threadIdx.x & 7;
    float rsum = 0.f;
    for (int j = part; j < NP; j += 8) rsum += sE[ii * ES + j];
    rsum += __shfl_xor(rsum, 1);
    rsum += __shfl_xor(rsum, 2);
    rsum += __shfl_xor(rsum, 4);
    if (part == 0) sRow[ii] = rsum;
  }
  constexpr int JW = NP / 4;                         // j range of one wave
  f32x16 acc[CK / 32];
#pragma unroll
  for (int kc = 0; kc < CK / 32; kc++) acc[kc] = f32x16{};
  for (int js = 0; js < JW; js += 2) {
    const int j = wave * JW + js + half;
    const float bv = sE[(lane & 31) * ES + j];       // B[k = half][col i] = E[i][j]
#pragma unroll
    for (int kc = 0; kc < CK / 32; kc++) {
      const float av = sP[j * CK + kc * 32 + (lane & 31)];   // A[row k][half] = p'_j[k]
      acc[kc] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc[kc], 0, 0, 0);
    }
  }
  __syncthreads();                                   // sE is reused for the partials
  // register e: coordinate k = kc*32 + 8 (e/4) + 4 half + e%4, row i = lane % 32
#pragma unroll
  for (int kc = 0; kc < CK / 32; kc++)
#pragma unroll
    for (int e = 0; e < 16; e++) {
      const int k = kc * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
      sPart[(wave * CK + k) * 32 + (lane & 31)] = acc[kc][e];
    }
  __syncthreads();
  for (int idx = threadIdx.x; idx < 32 * c; idx += FT) {
    const int ii = idx / c, k = idx % c, i = t * 32 + ii;
    if (i >= n) continue;
    const float ep = sPart[(0 * CK + k) * 32 + ii] + sPart[(1 * CK + k) * 32 + ii] +
                     sPart[(2 * CK + k) * 32 + ii] + sPart[(3 * CK + k) * 32 + ii];
    dp[((size_t)b * n + i) * c + k] = 2.f * (sRow[ii] * sP[i * CK + k] - ep);
  }
}

template <int NT>
hipError_t field_fwd_launch(const float* p, const bf16* x, bf16* y, float* row_mean, float* lse,
                            float* partners, int batch, int n, int c, int cp, int width,
                            float inv_tau, int scaled, hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  const int bytes = fwd_lds_bytes(NT, cp);
  hipError_t e = lds_limit_once(done, (const void*)field_fwd_kernel<NT>, fwd_lds_bytes(NT, 64));
  if (e != hipSuccess) return e;
  const int slabs = width / HD;
  field_fwd_kernel<NT><<<batch * slabs, FT, bytes, st>>>(p, x, y, row_mean, lse, partners, n, c,
                                                          cp, width, slabs, inv_tau, scaled);
  return hipGetLastError();
}

template <int NT>
hipError_t field_bwd_launch(const float* p, const bf16* x, const float* row_mean,
                            const float* lse, const bf16* dy, float* dp, bf16* dx, float* ddt,
                            int batch, int n, int c, int cp, int width, float inv_tau, int scaled,
                            hipStream_t st) {
  static std::atomic<unsigned long long> done_rows{0}, done_dx{0}, done_c32{0}, done_c64{0};
  hipError_t e = lds_limit_once(done_rows, (const void*)field_bwd_rows_kernel<NT>,
                                rows_lds_bytes(NT, 64));
  if (e == hipSuccess)
    e = lds_limit_once(done_dx, (const void*)field_bwd_dx_kernel<NT>, dx_lds_bytes(NT, 64));
  if (e == hipSuccess)
    e = c <= 32 ? lds_limit_once(done_c32, (const void*)field_bwd_coord_kernel<NT, 32>,
                                 coord_lds_bytes(NT, 32))
                : lds_limit_once(done_c64, (const void*)field_bwd_coord_kernel<NT, 64>,
                                 coord_lds_bytes(NT, 64));
  if (e != hipSuccess) return e;
  field_bwd_rows_kernel<NT><<<batch * NT, FT, rows_lds_bytes(NT, cp), st>>>(
      p, x, dy, row_mean, lse, ddt, n, c, cp, width, inv_tau, scaled);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int slabs = width / HD;
  field_bwd_dx_kernel<NT><<<batch * slabs, FT, dx_lds_bytes(NT, cp), st>>>(
      p, row_mean, lse, dy, dx, n, c, cp, width, slabs, inv_tau, scaled);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (c <= 32)
    field_bwd_coord_kernel<NT, 32><<<batch * NT, FT, coord_lds_bytes(NT, 32), st>>>(p, ddt, dp, n,
                                                                                    c);
  else
    field_bwd_coord_kernel<NT, 64><<<batch * NT, FT, coord_lds_bytes(NT, 64), st>>>(p, ddt, dp, n,
                                                                                    c);
  return hipGetLastError();
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
  HCMIX_FIELD_CASES(field_fwd_launch, p, x, y, row_mean, lse, partners, batch, n, c, cp, width,
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
