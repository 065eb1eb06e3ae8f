// bf16 path of the mixing layer on gfx950 matrix cores
// (v_mfma_f32_32x32x16_bf16: bf16 operands, fp32 accumulation).
//
// Every layer pairs each "lower" row (bit d clear) with its partner "upper"
// row (bit d set).  A block owns BMP lower rows and their BMP partners: the
// block's row set is closed under XOR 2^d for every stride 1 .. n/2, so the
// partner of LDS row m is LDS row m +- BMP and the XOR gather is just a
// different LDS base address; no permuted copy of the activations is ever
// written.  Each 16-byte global load is a whole 16-byte piece of one row, so
// every stride is fetched at full line efficiency.
#include "hcmix_internal.h"

namespace hcmix {

namespace {

constexpr int BK = 64;       // contraction slice held in LDS (128 bytes per row)
constexpr int CH = BK / 8;   // 16-byte pieces per row of a slice

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// LDS offset (in elements) of 16-byte piece `ch` of tile row `m`; the piece
// index is XOR-swizzled with the row so that 8 consecutive rows read at the
// same piece hit 8 different bank groups.
__device__ __forceinline__ int swz(int m, int ch) { return m * BK + ((ch ^ (m & 7)) << 3); }

// ---------------------------------------------------------------------------
// Mix GEMM.  For the block's lower rows L and upper rows U:
//   out_L = A_L B1^T + [partner_lower] A_U B2^T
//   out_U = A_U B1^T + [partner_upper] A_L B2^T
// Forward: A = x, B1 = W_self, B2 = W_off, partner_upper = 1, partner_lower = bidir.
// dX:      A = dy, B1 = W_self^T, B2 = W_off^T, partner_lower = 1, partner_upper = bidir.
// ---------------------------------------------------------------------------
template <int BMP, int BN, int WAVES_M, int WAVES_N>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) void mix_bf16_kernel(
    const bf16* __restrict__ A, const bf16* __restrict__ B1, const bf16* __restrict__ B2,
    bf16* __restrict__ out, int pairs, int width, int d, int partner_lower, int partner_upper) {
  constexpr int NT = 64 * WAVES_M * WAVES_N;
  constexpr int BM = 2 * BMP;
  constexpr int TMP = BMP / (32 * WAVES_M);  // 32-row pair blocks per wave
  constexpr int TN = BN / (32 * WAVES_N);    // 32-column blocks per wave
  constexpr int A_IT = BM * CH / NT;
  constexpr int B_IT = BN * CH / NT;
  static_assert(TMP >= 1 && TN >= 1, "tile too small for the wave grid");
  static_assert(A_IT * NT == BM * CH && B_IT * NT == BN * CH, "loads must tile evenly");

  __shared__ __attribute__((aligned(16))) bf16 sA[BM * BK];
  __shared__ __attribute__((aligned(16))) bf16 sB1[BN * BK];
  __shared__ __attribute__((aligned(16))) bf16 sB2[BN * BK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const int s = 1 << d;
  const int q0 = blockIdx.x * BMP;
  const int n0 = blockIdx.y * BN;

  // Source pointers and LDS slots of this thread's 16-byte pieces.
  const bf16* a_src[A_IT];
  int a_dst[A_IT];
#pragma unroll
  for (int j = 0; j < A_IT; j++) {
    const int idx = tid + NT * j;
    const int m = idx / CH, ch = idx % CH;
    int q = q0 + (m % BMP);
    if (q >= pairs) q = pairs - 1;  // ragged last block: load a valid row, never store it
    const int r = lower_row(q, d) + (m >= BMP ? s : 0);
    a_src[j] = A + (size_t)r * width + ch * 8;
    a_dst[j] = swz(m, ch);
  }
  const bf16* b1_src[B_IT];
  const bf16* b2_src[B_IT];
  int b_dst[B_IT];
#pragma unroll
  for (int j = 0; j < B_IT; j++) {
    const int idx = tid + NT * j;
    const int nr = idx / CH, ch = idx % CH;
    b1_src[j] = B1 + (size_t)(n0 + nr) * width + ch * 8;
    b2_src[j] = B2 + (size_t)(n0 + nr) * width + ch * 8;
    b_dst[j] = swz(nr, ch);
  }

  f32x16 accL[TMP][TN], accU[TMP][TN];
#pragma unroll
  for (int p = 0; p < TMP; p++)
#pragma unroll
    for (int t = 0; t < TN; t++)
#pragma unroll
      for (int e = 0; e < 16; e++) { accL[p][t][e] = 0.f; accU[p][t][e] = 0.f; }

  for (int k0 = 0; k0 < width; k0 += BK) {
    uint4 ra[A_IT], rb1[B_IT], rb2[B_IT];
#pragma unroll
    for (int j = 0; j < A_IT; j++) ra[j] = *(const uint4*)(a_src[j] + k0);
#pragma unroll
    for (int j = 0; j < B_IT; j++) {
      rb1[j] = *(const uint4*)(b1_src[j] + k0);
      rb2[j] = *(const uint4*)(b2_src[j] + k0);
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < A_IT; j++) *(uint4*)(sA + a_dst[j]) = ra[j];
#pragma unroll
    for (int j = 0; j < B_IT; j++) {
      *(uint4*)(sB1 + b_dst[j]) = rb1[j];
      *(uint4*)(sB2 + b_dst[j]) = rb2[j];
    }
    __syncthreads();

#pragma unroll
    for (int kk = 0; kk < BK / 16; kk++) {
      const int ch = kk * 2 + (lane >> 5);
      bf16x8 aL[TMP], aU[TMP], b1[TN], b2[TN];
#pragma unroll
      for (int p = 0; p < TMP; p++) {
        const int m = (wm * TMP + p) * 32 + (lane & 31);
        aL[p] = *(const bf16x8*)(sA + swz(m, ch));
        aU[p] = *(const bf16x8*)(sA + swz(m + BMP, ch));
      }
#pragma unroll
      for (int t = 0; t < TN; t++) {
        const int nr = (wn * TN + t) * 32 + (lane & 31);
        b1[t] = *(const bf16x8*)(sB1 + swz(nr, ch));
        b2[t] = *(const bf16x8*)(sB2 + swz(nr, ch));
      }
#pragma unroll
      for (int p = 0; p < TMP; p++)
#pragma unroll
        for (int t = 0; t < TN; t++) {
          accL[p][t] = mfma32(aL[p], b1[t], accL[p][t]);
          accU[p][t] = mfma32(aU[p], b1[t], accU[p][t]);
          if (partner_upper) accU[p][t] = mfma32(aL[p], b2[t], accU[p][t]);
          if (partner_lower) accL[p][t] = mfma32(aU[p], b2[t], accL[p][t]);
        }
    }
  }

  // Epilogue: accumulator element e of lane l is C[8*(e/4) + 4*(l/32) + e%4][l%32].
#pragma unroll
  for (int p = 0; p < TMP; p++) {
#pragma unroll
    for (int e = 0; e < 16; e++) {
      const int i = 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
      const int q = q0 + (wm * TMP + p) * 32 + i;
      if (q >= pairs) continue;
      const int rL = lower_row(q, d), rU = rL + s;
#pragma unroll
      for (int t = 0; t < TN; t++) {
        const int col = n0 + (wn * TN + t) * 32 + (lane & 31);
        out[(size_t)rL * width + col] = to_bf16(accL[p][t][e]);
        out[(size_t)rU * width + col] = to_bf16(accU[p][t][e]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Transpose of two width x width bf16 matrices (for the dX contraction).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void transpose2_kernel(const bf16* __restrict__ W1,
                                                         const bf16* __restrict__ W2,
                                                         bf16* __restrict__ W1T,
                                                         bf16* __restrict__ W2T, int width) {
  __shared__ bf16 tile[32][33];
  const bf16* src = blockIdx.z ? W2 : W1;
  bf16* dst = blockIdx.z ? W2T : W1T;
  const int c0 = blockIdx.x * 32, o0 = blockIdx.y * 32;
  const int tx = threadIdx.x % 32, ty = threadIdx.x / 32;  // 32 x 8
  for (int i = ty; i < 32; i += 8) tile[i][tx] = src[(size_t)(o0 + i) * width + c0 + tx];
  __syncthreads();
  for (int i = ty; i < 32; i += 8) dst[(size_t)(c0 + i) * width + o0 + tx] = tile[tx][i];
}

// ---------------------------------------------------------------------------
// Weight gradients, split over rows.  Block (x, y, z) computes the BO x BC
// tile (o0 = y*BO, c0 = x*BC) of dW_self and dW_off over the pairs of split z:
//   dW_self += dY_L^T X_L + dY_U^T X_U
//   dW_off  += dY_U^T X_L            (+ dY_L^T X_U when bidirectional)
// K-step = KP pairs = 2*KP rows, staged transposed in LDS ([column][row slot],
// slots 0..KP-1 lower rows, KP..2KP-1 their partners) so both MFMA operands
// are read as 16 contiguous bytes along the row (contraction) index.
// ---------------------------------------------------------------------------
constexpr int KP = 32;
constexpr int SLOTS = 2 * KP;
constexpr int LDT = SLOTS + 8;  // padded LDS row, elements (144 bytes)

template <int BO, int BC, int WAVES_O, int WAVES_C>
__global__ __launch_bounds__(64 * WAVES_O * WAVES_C) void dw_bf16_kernel(
    const bf16* __restrict__ X, const bf16* __restrict__ dY, float* __restrict__ partial,
    int pairs, int width, int d, int bidir, int pairs_per_split) {
  constexpr int NT = 64 * WAVES_O * WAVES_C;
  constexpr int TO = BO / (32 * WAVES_O);
  constexpr int TC = BC / (32 * WAVES_C);
  constexpr int G_IT = SLOTS * (BO / 8) / NT;
  constexpr int X_IT = SLOTS * (BC / 8) / NT;
  static_assert(G_IT * NT == SLOTS * (BO / 8) && X_IT * NT == SLOTS * (BC / 8), "");
  __shared__ __attribute__((aligned(16))) bf16 sG[BO * LDT];
  __shared__ __attribute__((aligned(16))) bf16 sX[BC * LDT];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wo = wave % WAVES_O, wc = wave / WAVES_O;
  const int c0 = blockIdx.x * BC, o0 = blockIdx.y * BO;
  const int s = 1 << d;
  const int pbeg = blockIdx.z * pairs_per_split;
  const int pend = min(pairs, pbeg + pairs_per_split);

  f32x16 accS[TO][TC], accO[TO][TC];
#pragma unroll
  for (int a = 0; a < TO; a++)
#pragma unroll
    for (int b = 0; b < TC; b++)
#pragma unroll
      for (int e = 0; e < 16; e++) { accS[a][b][e] = 0.f; accO[a][b][e] = 0.f; }

  for (int p0 = pbeg; p0 < pend; p0 += KP) {
    uint4 rg[G_IT], rx[X_IT];
#pragma unroll
    for (int j = 0; j < G_IT; j++) {
      const int idx = tid + NT * j;
      const int slot = idx / (BO / 8), ch = idx % (BO / 8);
      const int q = p0 + (slot % KP);
      uint4 v = make_uint4(0, 0, 0, 0);
      if (q < pend) {
        const int r = lower_row(q, d) + (slot >= KP ? s : 0);
        v = *(const uint4*)(dY + (size_t)r * width + o0 + ch * 8);
      }
      rg[j] = v;
    }
#pragma unroll
    for (int j = 0; j < X_IT; j++) {
      const int idx = tid + NT * j;
      const int slot = idx / (BC / 8), ch = idx % (BC / 8);
      const int q = p0 + (slot % KP);
      uint4 v = make_uint4(0, 0, 0, 0);
      if (q < pend) {
        const int r = lower_row(q, d) + (slot >= KP ? s : 0);
        v = *(const uint4*)(X + (size_t)r * width + c0 + ch * 8);
      }
      rx[j] = v;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < G_IT; j++) {
      const int idx = tid + NT * j;
      const int slot = idx / (BO / 8), ch = idx % (BO / 8);
      const bf16* v = (const bf16*)&rg[j];
#pragma unroll
      for (int e = 0; e < 8; e++) sG[(ch * 8 + e) * LDT + slot] = v[e];
    }
#pragma unroll
    for (int j = 0; j < X_IT; j++) {
      const int idx = tid + NT * j;
      const int slot = idx / (BC / 8), ch = idx % (BC / 8);
      const bf16* v = (const bf16*)&rx[j];
#pragma unroll
      for (int e = 0; e < 8; e++) sX[(ch * 8 + e) * LDT + slot] = v[e];
    }
    __syncthreads();

    const int half = 8 * (lane >> 5);
    // dW_self: all 64 slots
#pragma unroll
    for (int kk = 0; kk < SLOTS / 16; kk++) {
      bf16x8 ga[TO], xb[TC];
#pragma unroll
      for (int a = 0; a < TO; a++)
        ga[a] = *(const bf16x8*)(sG + ((wo * TO + a) * 32 + (lane & 31)) * LDT + kk * 16 + half);
#pragma unroll
      for (int b = 0; b < TC; b++)
        xb[b] = *(const bf16x8*)(sX + ((wc * TC + b) * 32 + (lane & 31)) * LDT + kk * 16 + half);
#pragma unroll
      for (int a = 0; a < TO; a++)
#pragma unroll
        for (int b = 0; b < TC; b++) accS[a][b] = mfma32(ga[a], xb[b], accS[a][b]);
    }
    // dW_off: receiver gradient slots x sender activation slots
#pragma unroll
    for (int kk = 0; kk < KP / 16; kk++) {
      bf16x8 gU[TO], xL[TC], gL[TO], xU[TC];
#pragma unroll
      for (int a = 0; a < TO; a++) {
        const int row = ((wo * TO + a) * 32 + (lane & 31)) * LDT + kk * 16 + half;
        gU[a] = *(const bf16x8*)(sG + row + KP);
        gL[a] = *(const bf16x8*)(sG + row);
      }
#pragma unroll
      for (int b = 0; b < TC; b++) {
        const int row = ((wc * TC + b) * 32 + (lane & 31)) * LDT + kk * 16 + half;
        xL[b] = *(const bf16x8*)(sX + row);
        xU[b] = *(const bf16x8*)(sX + row + KP);
      }
#pragma unroll
      for (int a = 0; a < TO; a++)
#pragma unroll
        for (int b = 0; b < TC; b++) {
          accO[a][b] = mfma32(gU[a], xL[b], accO[a][b]);
          if (bidir) accO[a][b] = mfma32(gL[a], xU[b], accO[a][b]);
        }
    }
  }

  const size_t ww = (size_t)width * width;
  float* outS = partial + (size_t)blockIdx.z * 2 * ww;
  float* outO = outS + ww;
#pragma unroll
  for (int a = 0; a < TO; a++)
#pragma unroll
    for (int b = 0; b < TC; b++)
#pragma unroll
      for (int e = 0; e < 16; e++) {
        const int o = o0 + (wo * TO + a) * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        const int c = c0 + (wc * TC + b) * 32 + (lane & 31);
        outS[(size_t)o * width + c] = accS[a][b][e];
        outO[(size_t)o * width + c] = accO[a][b][e];
      }
}

// dW (+)= sum over splits, in split order.
__global__ __launch_bounds__(256) void dw_reduce_kernel(const float* __restrict__ partial,
                                                        float* __restrict__ dws,
                                                        float* __restrict__ dwo, int splits,
                                                        size_t ww, int accumulate) {
  const size_t n4 = ww / 4;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < 2 * n4;
       i += (size_t)gridDim.x * blockDim.x) {
    const int m = i >= n4;
    const size_t j = i - m * n4;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int sp = 0; sp < splits; sp++) {
      const float4 v = ((const float4*)(partial + ((size_t)sp * 2 + m) * ww))[j];
      acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
    }
    float4* dst = (float4*)(m ? dwo : dws) + j;
    if (accumulate) {
      const float4 o = *dst;
      acc.x += o.x; acc.y += o.y; acc.z += o.z; acc.w += o.w;
    }
    *dst = acc;
  }
}

constexpr int DW_BO = 128, DW_BC = 128;

}  // namespace

hipError_t launch_mix_bf16(const bf16* A, const bf16* B1, const bf16* B2, bf16* out, int rows,
                           int width, int d, int partner_lower, int partner_upper,
                           hipStream_t st) {
  const int pairs = rows / 2;
  if (width % 128 == 0) {
    constexpr int BMP = 64, BN = 128;
    dim3 grid((pairs + BMP - 1) / BMP, width / BN);
    mix_bf16_kernel<BMP, BN, 2, 2><<<grid, 256, 0, st>>>(A, B1, B2, out, pairs, width, d,
                                                         partner_lower, partner_upper);
  } else {
    constexpr int BMP = 64, BN = 64;
    dim3 grid((pairs + BMP - 1) / BMP, width / BN);
    mix_bf16_kernel<BMP, BN, 2, 2><<<grid, 256, 0, st>>>(A, B1, B2, out, pairs, width, d,
                                                         partner_lower, partner_upper);
  }
  return hipGetLastError();
}

hipError_t launch_transpose2_bf16(const bf16* W1, const bf16* W2, bf16* W1T, bf16* W2T,
                                  int width, hipStream_t st) {
  dim3 grid(width / 32, width / 32, 2);
  transpose2_kernel<<<grid, 256, 0, st>>>(W1, W2, W1T, W2T, width);
  return hipGetLastError();
}

// Split-K plan: enough blocks to fill the chip (about 512), each split a whole
// number of K-steps.  Returns the split count; *pps gets pairs per split.
static int dw_plan(int rows, int width, int* pps) {
  const int pairs = rows / 2;
  const int bo = width % DW_BO == 0 ? DW_BO : 64;
  const int tiles = (width / bo) * (width / bo);
  const int ksteps = (pairs + KP - 1) / KP;
  int splits = (512 + tiles - 1) / tiles;
  if (splits > ksteps) splits = ksteps;
  if (splits < 1) splits = 1;
  *pps = ((ksteps + splits - 1) / splits) * KP;
  return (pairs + *pps - 1) / *pps;
}

int dw_bf16_splits(int rows, int width) {
  int pps;
  return dw_plan(rows, width, &pps);
}

hipError_t launch_dw_bf16(const bf16* X, const bf16* dY, float* partial, float* dws, float* dwo,
                          int rows, int width, int d, int bidir, int accumulate,
                          hipStream_t st) {
  const int pairs = rows / 2;
  int pps;
  const int splits = dw_plan(rows, width, &pps);
  if (width % DW_BO == 0) {
    dim3 grid(width / DW_BC, width / DW_BO, splits);
    dw_bf16_kernel<DW_BO, DW_BC, 2, 2><<<grid, 256, 0, st>>>(X, dY, partial, pairs, width, d,
                                                             bidir, pps);
  } else {
    dim3 grid(width / 64, width / 64, splits);
    dw_bf16_kernel<64, 64, 2, 2><<<grid, 256, 0, st>>>(X, dY, partial, pairs, width, d, bidir,
                                                       pps);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t ww = (size_t)width * width;
  int blocks = (int)((2 * ww / 4 + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  dw_reduce_kernel<<<blocks, 256, 0, st>>>(partial, dws, dwo, splits, ww, accumulate);
  return hipGetLastError();
}

}  // namespace hcmix
