// FMA path of the mixing layer: LDS-tiled kernels with no matrix
// instructions, every product and sum an IEEE fp32 operation.  Used for fp32
// inputs of any width, and for bf16 inputs whose width is a multiple of 8 but
// not of 64 (the MFMA tiles of kernels_bf16.hip need 64): bf16 operands are
// widened to fp32 exactly, and each bf16 output is rounded once (RNE), as on
// the MFMA path.
#include "hcmix_internal.h"

namespace hcmix {

namespace {

__device__ __forceinline__ float widen(float v) { return v; }
__device__ __forceinline__ float widen(bf16 v) { return (float)v; }
template <typename E> __device__ __forceinline__ E narrow(float v);
template <> __device__ __forceinline__ float narrow<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 narrow<bf16>(float v) { return to_bf16(v); }

constexpr int T = 64;    // output tile edge
constexpr int KC = 16;   // contraction chunk
constexpr int NT = 256;  // threads per block: 16 x 16, 4 x 4 outputs each

// out[r][j] = sum_k A[r][k] W1(j,k) + m(r) sum_k A[p(r)][k] W2(j,k)
// Hypercube layer (d >= 0): p(r) = r ^ 2^d, m(r) = partner_upper / partner_lower
// by bit d of r.  Local layer (d < 0): p(r) = r + shift with shift = -1
// (forward; m = 0 at a window's first row) or +1 (dX; m = 0 at its last row).
template <typename E, bool TRANSPOSE_W>
__global__ __launch_bounds__(NT) void mix_fma_kernel(
    const E* __restrict__ A, const E* __restrict__ W1, const E* __restrict__ W2,
    E* __restrict__ out, int rows, int width, int d, int partner_lower, int partner_upper,
    int n, int shift) {
  __shared__ float sA[KC][T + 1];
  __shared__ float sP[KC][T + 1];
  __shared__ float sW1[KC][T + 1];
  __shared__ float sW2[KC][T + 1];
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;
  const int r0 = blockIdx.x * T, j0 = blockIdx.y * T;
  const int s = d >= 0 ? 1 << d : 0;
  float acc[4][4] = {};

  for (int k0 = 0; k0 < width; k0 += KC) {
    for (int e = 0; e < (T * KC) / NT; e++) {
      const int idx = tid + NT * e;
      // activations: 16 consecutive k of one row per 16 threads
      {
        const int m = idx / KC, kk = idx % KC;
        const int r = r0 + m, k = k0 + kk;
        float a = 0.f, p = 0.f;
        if (r < rows && k < width) {
          a = widen(A[(size_t)r * width + k]);
          int take, pr;
          if (d >= 0) {
            take = ((r >> d) & 1) ? partner_upper : partner_lower;
            pr = r ^ s;
          } else {
            const int pos = r & (n - 1);
            take = shift < 0 ? pos != 0 : pos != n - 1;
            pr = r + shift;
          }
          if (take) p = widen(A[(size_t)pr * width + k]);
        }
        sA[kk][m] = a;
        sP[kk][m] = p;
      }
      // weights
      {
        int j, kk;
        if (TRANSPOSE_W) { kk = idx / T; j = idx % T; }   // contiguous along j
        else { j = idx / KC; kk = idx % KC; }             // contiguous along k
        const int jj = j0 + j, k = k0 + kk;
        float w1 = 0.f, w2 = 0.f;
        if (jj < width && k < width) {
          const size_t off = TRANSPOSE_W ? (size_t)k * width + jj : (size_t)jj * width + k;
          w1 = widen(W1[off]);
          w2 = widen(W2[off]);
        }
        sW1[kk][j] = w1;
        sW2[kk][j] = w2;
      }
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < KC; kk++) {
      float a[4], p[4], b1[4], b2[4];
#pragma unroll
      for (int i = 0; i < 4; i++) {
        a[i] = sA[kk][ty * 4 + i];
        p[i] = sP[kk][ty * 4 + i];
        b1[i] = sW1[kk][tx * 4 + i];
        b2[i] = sW2[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) acc[i][j] = fmaf(p[i], b2[j], fmaf(a[i], b1[j], acc[i][j]));
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int r = r0 + ty * 4 + i;
    if (r >= rows) continue;
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int jj = j0 + tx * 4 + j;
      if (jj < width) out[(size_t)r * width + jj] = narrow<E>(acc[i][j]);
    }
  }
}

// dws[o][c] (+)= sum_r dY[r][o] X[r][c];  dwo[o][c] (+)= sum_r m(r) dY[r][o] X[p(r)][c]
// with p(r) = r ^ 2^d (hypercube layer) or r - 1 (local layer, d < 0; m = 0 at
// a window's first row).  One block per 64 x 64 output tile walks every row in
// a fixed order.
template <typename E>
__global__ __launch_bounds__(NT) void dw_fma_kernel(
    const E* __restrict__ X, const E* __restrict__ dY, float* __restrict__ dws,
    float* __restrict__ dwo, int rows, int width, int d, int n, int bidir, int accumulate) {
  __shared__ float sG[KC][T + 1];
  __shared__ float sX[KC][T + 1];
  __shared__ float sXP[KC][T + 1];
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;
  const int o0 = blockIdx.y * T, c0 = blockIdx.x * T;
  const int s = d >= 0 ? 1 << d : 0;
  float accS[4][4] = {}, accO[4][4] = {};

  for (int rb = 0; rb < rows; rb += KC) {
    for (int e = 0; e < (T * KC) / NT; e++) {
      const int idx = tid + NT * e;
      const int kk = idx / T, j = idx % T;  // row kk of the chunk, column j of the tile
      const int r = rb + kk;
      float g = 0.f, xv = 0.f, xp = 0.f;
      if (r < rows) {
        if (o0 + j < width) g = widen(dY[(size_t)r * width + o0 + j]);
        if (c0 + j < width) {
          xv = widen(X[(size_t)r * width + c0 + j]);
          if (d < 0) {
            if (r & (n - 1)) xp = widen(X[(size_t)(r - 1) * width + c0 + j]);
          } else if (bidir || ((r >> d) & 1)) {
            xp = widen(X[(size_t)(r ^ s) * width + c0 + j]);
          }
        }
      }
      sG[kk][j] = g;
      sX[kk][j] = xv;
      sXP[kk][j] = xp;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < KC; kk++) {
      float g[4], xv[4], xp[4];
#pragma unroll
      for (int i = 0; i < 4; i++) {
        g[i] = sG[kk][ty * 4 + i];
        xv[i] = sX[kk][tx * 4 + i];
        xp[i] = sXP[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) {
          accS[i][j] = fmaf(g[i], xv[j], accS[i][j]);
          accO[i][j] = fmaf(g[i], xp[j], accO[i][j]);
        }
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int o = o0 + ty * 4 + i;
    if (o >= width) continue;
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int c = c0 + tx * 4 + j;
      if (c >= width) continue;
      const size_t off = (size_t)o * width + c;
      dws[off] = accumulate ? dws[off] + accS[i][j] : accS[i][j];
      dwo[off] = accumulate ? dwo[off] + accO[i][j] : accO[i][j];
    }
  }
}

}  // namespace

template <typename E>
hipError_t mix_fma_launch(const void* A, const void* W1, const void* W2, void* out, int rows,
                          int width, int d, int partner_lower, int partner_upper, int n, int shift,
                          bool transpose_w, hipStream_t st) {
  dim3 grid((rows + T - 1) / T, (width + T - 1) / T);
  const E *a = (const E*)A, *w1 = (const E*)W1, *w2 = (const E*)W2;
  if (transpose_w)
    mix_fma_kernel<E, true><<<grid, NT, 0, st>>>(a, w1, w2, (E*)out, rows, width, d,
                                                 partner_lower, partner_upper, n, shift);
  else
    mix_fma_kernel<E, false><<<grid, NT, 0, st>>>(a, w1, w2, (E*)out, rows, width, d,
                                                  partner_lower, partner_upper, n, shift);
  return hipGetLastError();
}

hipError_t launch_mix_fma(const void* A, const void* W1, const void* W2, void* out, int rows,
                          int width, int d, int partner_lower, int partner_upper, int n,
                          int shift, bool transpose_w, bool bf16_data, hipStream_t st) {
  return bf16_data ? mix_fma_launch<bf16>(A, W1, W2, out, rows, width, d, partner_lower,
                                          partner_upper, n, shift, transpose_w, st)
                   : mix_fma_launch<float>(A, W1, W2, out, rows, width, d, partner_lower,
                                           partner_upper, n, shift, transpose_w, st);
}

hipError_t launch_dw_fma(const void* X, const void* dY, float* dws, float* dwo, int rows,
                         int width, int d, int n, int bidir, int accumulate, bool bf16_data,
                         hipStream_t st) {
  dim3 grid((width + T - 1) / T, (width + T - 1) / T);
  if (bf16_data)
    dw_fma_kernel<bf16><<<grid, NT, 0, st>>>((const bf16*)X, (const bf16*)dY, dws, dwo, rows,
                                             width, d, n, bidir, accumulate);
  else
    dw_fma_kernel<float><<<grid, NT, 0, st>>>((const float*)X, (const float*)dY, dws, dwo, rows,
                                              width, d, n, bidir, accumulate);
  return hipGetLastError();
}

}  // namespace hcmix
