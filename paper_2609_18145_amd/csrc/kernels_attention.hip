// Causal multi-head softmax attention for the hybrid schedules' attention
// layers (bf16 in, fp32 accumulation), windows of at most 256 positions, head
// dimension 64.  One block per (window, head): two of the window's tiles sit in
// LDS (keys and values; for the backward's two kernels queries and output
// gradients, or keys and values), the whole causal row of scores fits in
// registers and the softmax is exact (no running rescale).
//
// Layouts: qkv [batch][n][3][heads][64] (Q, K, V of every position), out and
// dout [batch][n][heads][64], lse [batch][heads][n] fp32.
//
// Scores are computed transposed, S^T = K Q^T, so that a lane owns one query
// (column) and 16 of its keys per 32 x 32 tile: row statistics are in-lane
// sums plus one exchange with lane ^ 32.  The second product (P V, or its
// gradients) takes P straight from those registers as the MFMA B operand: the
// contraction over keys may visit the keys in any order as long as both
// operands agree, so a lane's 8 keys {16m + 4h + r, 16m + 8 + 4h + r} (h =
// lane / 32, r < 4) are its own score registers 8m .. 8m + 7, and the A
// operand (V^T, or Q^T, K^T, dO^T) is read from LDS transposed in that order.
#include "hcmix_internal.h"
#include "device_common.h"
#include "tile64.h"

namespace hcmix {

namespace {

constexpr int ATT_THREADS = 256;
constexpr float LOG2E = 1.4426950408889634f;

// Copy rows [0, NT * 32) of one head's 64 columns of two arrays (src: the
// first row's, row_stride elements apart: 3 * heads * 64 in qkv, heads * 64
// in out and dout) into two swizzled LDS tiles, every load in flight before
// the first LDS write (one memory latency for both tiles).
template <int NT>
__device__ __forceinline__ void att_load_tiles(const bf16* __restrict__ src_a, size_t stride_a,
                                               bf16* tile_a, const bf16* __restrict__ src_b,
                                               size_t stride_b, bf16* tile_b) {
  constexpr int PER = NT * 32 * 8 / ATT_THREADS;   // 16-byte pieces per thread and tile
  static_assert(PER * ATT_THREADS == NT * 32 * 8, "");
  u32x4 va[PER], vb[PER];
#pragma unroll
  for (int j = 0; j < PER; j++) {
    const int pi = threadIdx.x + ATT_THREADS * j, r = pi >> 3, p = pi & 7;
    va[j] = *(const u32x4*)(src_a + (size_t)r * stride_a + 8 * p);
    vb[j] = *(const u32x4*)(src_b + (size_t)r * stride_b + 8 * p);
  }
#pragma unroll
  for (int j = 0; j < PER; j++) {
    const int pi = threadIdx.x + ATT_THREADS * j, r = pi >> 3, p = pi & 7;
    *(u32x4*)(tile_a + att_off(r, 8 * p)) = va[j];
    *(u32x4*)(tile_b + att_off(r, 8 * p)) = vb[j];
  }
}

// ---------------------------------------------------------------------------
// Forward: O = softmax(s Q K^T, causal) V and lse, s = 1/8.
// ---------------------------------------------------------------------------
template <int NT>
__global__ __launch_bounds__(ATT_THREADS, 2) void attn_fwd_kernel(
    const bf16* __restrict__ qkv, bf16* __restrict__ out, float* __restrict__ lse, int heads) {
  constexpr int n = NT * 32;
  __shared__ __attribute__((aligned(1024))) bf16 sK[n * HD], sV[n * HD];
  const int bh = blockIdx.x, b = bh / heads, h = bh % heads;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
  const size_t rs = (size_t)3 * heads * HD;                 // qkv row stride
  const bf16* base = qkv + (size_t)b * n * rs + (size_t)h * HD;
  att_load_tiles<NT>(base + (size_t)heads * HD, rs, sK, base + (size_t)2 * heads * HD, rs, sV);
  __syncthreads();
  const float sc = 0.125f * LOG2E;     // scores in log2 units
#pragma unroll
  for (int which = 0; which < 2; which++) {
    const int qt = att_tile(wave, which);
    if (qt >= NT) continue;
    const int q = qt * 32 + (lane & 31);
    bf16x8 qf[4];                      // Q^T fragments: this lane's query, 8 dims per k16 step
#pragma unroll
    for (int ks = 0; ks < 4; ks++)
      qf[ks] = *(const bf16x8*)(base + (size_t)q * rs + 16 * ks + 8 * half);
    f32x16 s[NT];
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < NT; kt++) {
      if (kt > qt) continue;
      f32x16 acc = {};
#pragma unroll
      for (int ks = 0; ks < 4; ks++) acc = mfma32(att_frag(sK, kt * 32, 16 * ks, lane), qf[ks], acc);
#pragma unroll
      for (int e = 0; e < 16; e++) {
        float v = acc[e] * sc;
        if (kt == qt && att_masked(e, lane)) v = -INFINITY;
        acc[e] = v;
        mx = fmaxf(mx, v);
      }
      s[kt] = acc;
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    float sum = 0.f;
#pragma unroll
    for (int kt = 0; kt < NT; kt++) {
      if (kt > qt) continue;
#pragma unroll
      for (int e = 0; e < 16; e++) {
        const float p = __builtin_amdgcn_exp2f(s[kt][e] - mx);
        s[kt][e] = p;
        sum += p;
      }
    }
    sum += __shfl_xor(sum, 32);
    f32x16 o[2] = {};
#pragma unroll
    for (int kt = 0; kt < NT; kt++) {
      if (kt > qt) continue;
#pragma unroll
      for (int m = 0; m < 2; m++) {
        const bf16x8 pf = att_pack(s[kt], m);
#pragma unroll
        for (int dt = 0; dt < 2; dt++)
          o[dt] = mfma32(att_trfrag(sV, kt * 32 + 16 * m, 32 * dt, lane), pf, o[dt]);
      }
    }
    // O^T register e of lane l: query q, dimension 32 dt + 8 (e / 4) + 4 half + e % 4
    const float inv = 1.f / sum;
    bf16* orow = out + (((size_t)b * n + q) * heads + h) * HD;
#pragma unroll
    for (int dt = 0; dt < 2; dt++)
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const bf16x4 v = {to_bf16(o[dt][4 * g] * inv), to_bf16(o[dt][4 * g + 1] * inv),
                          to_bf16(o[dt][4 * g + 2] * inv), to_bf16(o[dt][4 * g + 3] * inv)};
        *(bf16x4*)(orow + 32 * dt + 8 * g + 4 * half) = v;
      }
    if (half == 0) lse[(size_t)bh * n + q] = (mx + __builtin_amdgcn_logf(sum)) * 0.6931471805599453f;
  }
}

// ---------------------------------------------------------------------------
// Backward.  With P = exp(s S - lse) and D = rowsum(dO * O):
//   dV = P^T dO,  dS = P (dO V^T - D),  dK = s dS^T Q,  dQ = s dS K.
// Two kernels, each with two of the window's four tiles in LDS (64 KB, two
// blocks per CU), writing disjoint parts of dqkv:
//   attn_bwd_kv_kernel: waves own key tiles; S and dP with lanes = keys,
//     accumulating dK^T and dV^T (Q and dO in LDS, read both ways);
//   attn_bwd_q_kernel: waves own query tiles; S^T and dP^T with lanes =
//     queries, accumulating dQ^T (K and V in LDS).
// P, S and dP are recomputed rather than stored; no atomics, deterministic.
// ---------------------------------------------------------------------------

// lse in log2 units and D = rowsum(dO * O) of the window's rows into LDS.
__device__ __forceinline__ void att_row_stats(const bf16* __restrict__ obase,
                                              const bf16* __restrict__ dobase, size_t os,
                                              const float* __restrict__ lse_row, int n, float* sL,
                                              float* sD) {
  for (int i = threadIdx.x; i < n; i += ATT_THREADS) {
    float d = 0.f;
#pragma unroll
    for (int p = 0; p < 8; p++) {
      const bf16x8 a = *(const bf16x8*)(obase + (size_t)i * os + 8 * p);
      const bf16x8 g = *(const bf16x8*)(dobase + (size_t)i * os + 8 * p);
#pragma unroll
      for (int e = 0; e < 8; e++) d += (float)a[e] * (float)g[e];
    }
    sD[i] = d;
    sL[i] = lse_row[i] * LOG2E;
  }
}

template <int NT>
__global__ __launch_bounds__(ATT_THREADS, 2) void attn_bwd_kv_kernel(
    const bf16* __restrict__ qkv, const bf16* __restrict__ out, const float* __restrict__ lse,
    const bf16* __restrict__ dout, bf16* __restrict__ dqkv, int heads) {
  constexpr int n = NT * 32;
  __shared__ __attribute__((aligned(1024))) bf16 sQ[n * HD], sO[n * HD];   // sO: dO
  __shared__ __attribute__((aligned(16))) float sL[n], sD[n];
  const int bh = blockIdx.x, b = bh / heads, h = bh % heads;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
  const size_t rs = (size_t)3 * heads * HD, os = (size_t)heads * HD;
  const bf16* base = qkv + (size_t)b * n * rs + (size_t)h * HD;
  const bf16* dobase = dout + (size_t)b * n * os + (size_t)h * HD;
  bf16* gbase = dqkv + (size_t)b * n * rs + (size_t)h * HD;
  att_load_tiles<NT>(base, rs, sQ, dobase, os, sO);
  att_row_stats(out + (size_t)b * n * os + (size_t)h * HD, dobase, os, lse + (size_t)bh * n, n,
                sL, sD);
  __syncthreads();
  const float sc = 0.125f * LOG2E;
#pragma unroll
  for (int which = 0; which < 2; which++) {
    const int kt = att_tile(wave, which);
    if (kt >= NT) continue;
    // K and V rows of this lane's key as B operands, straight from global memory
    const int key = kt * 32 + (lane & 31);
    bf16x8 kf[4], vf[4];
#pragma unroll
    for (int ks = 0; ks < 4; ks++) {
      kf[ks] = *(const bf16x8*)(base + (size_t)key * rs + os + 16 * ks + 8 * half);
      vf[ks] = *(const bf16x8*)(base + (size_t)key * rs + 2 * os + 16 * ks + 8 * half);
    }
    f32x16 dk[2] = {}, dv[2] = {};
#pragma unroll
    for (int qt = 0; qt < NT; qt++) {
      if (qt < kt) continue;
      f32x16 sacc = {}, pacc = {};
#pragma unroll
      for (int ks = 0; ks < 4; ks++) {
        sacc = mfma32(att_frag(sQ, qt * 32, 16 * ks, lane), kf[ks], sacc);
        pacc = mfma32(att_frag(sO, qt * 32, 16 * ks, lane), vf[ks], pacc);
      }
      // register e: query qt*32 + 8 (e/4) + 4 half + e%4, key kt*32 + lane%32
      f32x16 p, ds;
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const int q0 = qt * 32 + 8 * g + 4 * half;
        const f32x4 l4 = *(const f32x4*)(sL + q0);
        const f32x4 d4 = *(const f32x4*)(sD + q0);
#pragma unroll
        for (int r = 0; r < 4; r++) {
          const int e = 4 * g + r;
          const bool masked = qt == kt && (lane & 31) > 8 * g + 4 * half + r;
          const float pe = masked ? 0.f : __builtin_amdgcn_exp2f(sacc[e] * sc - l4[r]);
          p[e] = pe;
          ds[e] = pe * (pacc[e] - d4[r]);
        }
      }
#pragma unroll
      for (int m = 0; m < 2; m++) {
        const bf16x8 pf = att_pack(p, m), sf = att_pack(ds, m);
#pragma unroll
        for (int dt = 0; dt < 2; dt++) {
          dv[dt] = mfma32(att_trfrag(sO, qt * 32 + 16 * m, 32 * dt, lane), pf, dv[dt]);
          dk[dt] = mfma32(att_trfrag(sQ, qt * 32 + 16 * m, 32 * dt, lane), sf, dk[dt]);
        }
      }
    }
    // dK^T / dV^T register e of lane l: key kt*32 + l%32, dim 32 dt + 8 (e/4) + 4 half + e%4
    bf16* krow = gbase + (size_t)key * rs + os;
    bf16* vrow = gbase + (size_t)key * rs + 2 * os;
#pragma unroll
    for (int dt = 0; dt < 2; dt++)
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const int c = 32 * dt + 8 * g + 4 * half;
        const bf16x4 kv = {to_bf16(dk[dt][4 * g] * 0.125f), to_bf16(dk[dt][4 * g + 1] * 0.125f),
                           to_bf16(dk[dt][4 * g + 2] * 0.125f), to_bf16(dk[dt][4 * g + 3] * 0.125f)};
        const bf16x4 vv = {to_bf16(dv[dt][4 * g]), to_bf16(dv[dt][4 * g + 1]),
                           to_bf16(dv[dt][4 * g + 2]), to_bf16(dv[dt][4 * g + 3])};
        *(bf16x4*)(krow + c) = kv;
        *(bf16x4*)(vrow + c) = vv;
      }
  }
}

template <int NT>
__global__ __launch_bounds__(ATT_THREADS, 2) void attn_bwd_q_kernel(
    const bf16* __restrict__ qkv, const bf16* __restrict__ out, const float* __restrict__ lse,
    const bf16* __restrict__ dout, bf16* __restrict__ dqkv, int heads) {
  constexpr int n = NT * 32;
  __shared__ __attribute__((aligned(1024))) bf16 sK[n * HD], sV[n * HD];
  __shared__ __attribute__((aligned(16))) float sL[n], sD[n];
  const int bh = blockIdx.x, b = bh / heads, h = bh % heads;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
  const size_t rs = (size_t)3 * heads * HD, os = (size_t)heads * HD;
  const bf16* base = qkv + (size_t)b * n * rs + (size_t)h * HD;
  const bf16* dobase = dout + (size_t)b * n * os + (size_t)h * HD;
  bf16* gbase = dqkv + (size_t)b * n * rs + (size_t)h * HD;
  att_load_tiles<NT>(base + os, rs, sK, base + 2 * os, rs, sV);
  att_row_stats(out + (size_t)b * n * os + (size_t)h * HD, dobase, os, lse + (size_t)bh * n, n,
                sL, sD);
  __syncthreads();
  const float sc = 0.125f * LOG2E;
#pragma unroll
  for (int which = 0; which < 2; which++) {
    const int qt = att_tile(wave, which);
    if (qt >= NT) continue;
    const int q = qt * 32 + (lane & 31);
    bf16x8 qf[4], of[4];            // this lane's query and output-gradient rows, from global
#pragma unroll
    for (int ks = 0; ks < 4; ks++) {
      qf[ks] = *(const bf16x8*)(base + (size_t)q * rs + 16 * ks + 8 * half);
      of[ks] = *(const bf16x8*)(dobase + (size_t)q * os + 16 * ks + 8 * half);
    }
    const float lq = sL[q], dq = sD[q];
    f32x16 gq[2] = {};
#pragma unroll
    for (int kt = 0; kt < NT; kt++) {
      if (kt > qt) continue;
      f32x16 sacc = {}, pacc = {};
#pragma unroll
      for (int ks = 0; ks < 4; ks++) {
        sacc = mfma32(att_frag(sK, kt * 32, 16 * ks, lane), qf[ks], sacc);
        pacc = mfma32(att_frag(sV, kt * 32, 16 * ks, lane), of[ks], pacc);
      }
      f32x16 ds;
#pragma unroll
      for (int e = 0; e < 16; e++) {
        const bool masked = kt == qt && att_masked(e, lane);
        const float pe = masked ? 0.f : __builtin_amdgcn_exp2f(sacc[e] * sc - lq);
        ds[e] = pe * (pacc[e] - dq);
      }
#pragma unroll
      for (int m = 0; m < 2; m++) {
        const bf16x8 sf = att_pack(ds, m);
#pragma unroll
        for (int dt = 0; dt < 2; dt++)
          gq[dt] = mfma32(att_trfrag(sK, kt * 32 + 16 * m, 32 * dt, lane), sf, gq[dt]);
      }
    }
    bf16* qrow = gbase + (size_t)q * rs;
#pragma unroll
    for (int dt = 0; dt < 2; dt++)
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const bf16x4 v = {to_bf16(gq[dt][4 * g] * 0.125f), to_bf16(gq[dt][4 * g + 1] * 0.125f),
                          to_bf16(gq[dt][4 * g + 2] * 0.125f), to_bf16(gq[dt][4 * g + 3] * 0.125f)};
        *(bf16x4*)(qrow + 32 * dt + 8 * g + 4 * half) = v;
      }
  }
}

template <int NT>
hipError_t attn_fwd_launch(const bf16* qkv, bf16* out, float* lse, int batch, int heads,
                           hipStream_t st) {
  attn_fwd_kernel<NT><<<batch * heads, ATT_THREADS, 0, st>>>(qkv, out, lse, heads);
  return hipGetLastError();
}

template <int NT>
hipError_t attn_bwd_launch(const bf16* qkv, const bf16* out, const float* lse, const bf16* dout,
                           bf16* dqkv, int batch, int heads, hipStream_t st) {
  attn_bwd_kv_kernel<NT><<<batch * heads, ATT_THREADS, 0, st>>>(qkv, out, lse, dout, dqkv, heads);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  attn_bwd_q_kernel<NT><<<batch * heads, ATT_THREADS, 0, st>>>(qkv, out, lse, dout, dqkv, heads);
  return hipGetLastError();
}

}  // namespace

#define HCMIX_ATT_CASES(F, ...)              \
  switch (n / 32) {                          \
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

hipError_t launch_attention_fwd_bf16(const bf16* qkv, bf16* out, float* lse, int batch, int n,
                                     int heads, hipStream_t st) {
  HCMIX_ATT_CASES(attn_fwd_launch, qkv, out, lse, batch, heads, st)
}

hipError_t launch_attention_bwd_bf16(const bf16* qkv, const bf16* out, const float* lse,
                                     const bf16* dout, bf16* dqkv, int batch, int n, int heads,
                                     hipStream_t st) {
  HCMIX_ATT_CASES(attn_bwd_launch, qkv, out, lse, dout, dqkv, batch, heads, st)
}
#undef HCMIX_ATT_CASES

}  // namespace hcmix
