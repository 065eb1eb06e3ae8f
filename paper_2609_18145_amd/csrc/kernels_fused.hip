// Fused small-width stack (bf16, width 64, n in {64, 128, 256}): every window
// of n positions x 64 features stays in LDS through all layers, so the whole
// forward stack is one launch and the whole backward stack one launch plus a
// fixed-order reduction of the per-window weight gradients.  One block per
// window, n/64 waves, each wave owning 32 row pairs of the current layer.
//
// Activation buffers use the k-contiguous swizzle (rows of 128 bytes, 16-byte
// piece ch stored at ch ^ ((row >> 1) & 7)); weight buffers read transposed
// (backward) use the 64-byte segment swizzle of tr_frag.  Fragments whose
// contraction index runs over rows are gathered with ds_read_b64_tr_b16 whose
// per-lane row addresses apply the XOR pairing directly.
#include "device_common.h"
#include "hcmix_internal.h"

namespace hcmix {

namespace {

constexpr int FW = 64;        // width of the fused path
constexpr int FRB = 2 * FW;   // bytes per activation / weight row
constexpr int WW = FW * FW;   // elements per weight matrix

__device__ __forceinline__ int act_off(int row, int col) {
  return swz<FW>(row, col >> 3) + (col & 7);
}

// Transposed 32x32x16 fragment over an activation buffer: lane l receives
// buf[row(k0 + 8*(l/32) + t)][c0 + l%32] for t = 0..7, where row(kappa) maps
// the contraction index to a buffer row (identity, or a pair member).
template <typename RowFn>
__device__ __forceinline__ bf16x8 tr_act(const bf16* buf, int k0, int c0, int lane, RowFn row) {
  const int g = lane >> 4, j = lane & 15;
  const int kap = k0 + 8 * (g >> 1) + (j >> 2);
  const int col = c0 + 16 * (g & 1) + 4 * (j & 3);
  const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(buf + act_off(row(kap), col)));
  const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(buf + act_off(row(kap + 4), col)));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Rounds a wave's two 32-row output blocks to bf16 into an activation buffer.
// The accumulators hold the transposed products (weight fragment as the MFMA
// "A" operand), so element e of lane l belongs to row rL / rU (the lane's pair)
// and column 32 t + 8 (e/4) + 4 (l/32) + e%4: four runs of four columns.
__device__ __forceinline__ void store_rows(bf16* buf, const f32x16 (&accL)[2],
                                           const f32x16 (&accU)[2], int rL, int rU, int lane) {
#pragma unroll
  for (int t = 0; t < 2; t++)
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const int col = 32 * t + 8 * g + 4 * (lane >> 5);
      const bf16x4 vl = {to_bf16(accL[t][4 * g]), to_bf16(accL[t][4 * g + 1]),
                         to_bf16(accL[t][4 * g + 2]), to_bf16(accL[t][4 * g + 3])};
      const bf16x4 vu = {to_bf16(accU[t][4 * g]), to_bf16(accU[t][4 * g + 1]),
                         to_bf16(accU[t][4 * g + 2]), to_bf16(accU[t][4 * g + 3])};
      *(bf16x4*)(buf + act_off(rL, col)) = vl;
      *(bf16x4*)(buf + act_off(rU, col)) = vu;
    }
}

// Window rows (n rows of 128 bytes) global -> LDS in the activation swizzle.
__device__ __forceinline__ void dma_act(const bf16* src, bf16* dst, int n, int wave, int nw, int lane) {
  for (int b = wave; b < n / 8; b += nw) {
    const int o = b * 1024 + 16 * lane;
    const int row = o / FRB;
    const int ch = ((o % FRB) / 16) ^ ((row >> 1) & 7);
    dma16(src + (size_t)row * FW + ch * 8, dst + b * 512);
  }
}

// One weight matrix global -> LDS, k-contiguous rows (forward B operand).
__device__ __forceinline__ void dma_w_rows(const bf16* src, bf16* dst, int wave, int nw, int lane) {
  for (int b = wave; b < WW * 2 / 1024; b += nw) {
    const int o = b * 1024 + 16 * lane;
    const int row = o / FRB;
    const int ch = ((o % FRB) / 16) ^ ((row >> 1) & 7);
    dma16(src + (size_t)row * FW + ch * 8, dst + b * 512);
  }
}

// One weight matrix global -> LDS for transposed reads (backward B operand).
__device__ __forceinline__ void dma_w_tr(const bf16* src, bf16* dst, int wave, int nw, int lane) {
  for (int b = wave; b < WW * 2 / 1024; b += nw) {
    int row, col;
    tr_dma_coord<FRB>(b, lane, &row, &col);
    dma16(src + (size_t)row * FW + col, dst + b * 512);
  }
}

// ---------------------------------------------------------------------------
// Forward: x_{l+1} = layer_l(x_l) for l = 0..L-1, each x_{l+1} also stored.
// ---------------------------------------------------------------------------
template <bool BIDIR>
__global__ __launch_bounds__(256) void fused_fwd_kernel(FusedFwdArgs a) {
  extern __shared__ __attribute__((aligned(1024))) bf16 smem[];
  const int n = a.n, nw = n / 64, nthreads = 64 * nw;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const size_t win = (size_t)blockIdx.x * n * FW;
  bf16* X = smem;
  bf16* Y = X + n * FW;
  bf16* Wb = Y + n * FW;  // two sets of [W_self | W_off]

  dma_act(a.x0 + win, X, n, wave, nw, lane);
  dma_w_rows(a.ws[0], Wb, wave, nw, lane);
  dma_w_rows(a.wo[0], Wb + WW, wave, nw, lane);
  wait_dma();
  __syncthreads();

  for (int l = 0; l < a.num_layers; l++) {
    const int d = a.dim[l], s = 1 << d;
    const bf16* Ws = Wb + (l & 1) * 2 * WW;
    const bf16* Wo = Ws + WW;
    if (l + 1 < a.num_layers) {
      bf16* Wn = Wb + ((l + 1) & 1) * 2 * WW;
      dma_w_rows(a.ws[l + 1], Wn, wave, nw, lane);
      dma_w_rows(a.wo[l + 1], Wn + WW, wave, nw, lane);
    }
    f32x16 accL[2], accU[2];
#pragma unroll
    for (int t = 0; t < 2; t++)
#pragma unroll
      for (int e = 0; e < 16; e++) { accL[t][e] = 0.f; accU[t][e] = 0.f; }
    const int rL = lower_row(32 * wave + (lane & 31), d), rU = rL + s;
#pragma unroll
    for (int kk = 0; kk < FW / 16; kk++) {
      const int ch = kk * 2 + (lane >> 5);
      const bf16x8 aL = *(const bf16x8*)(X + swz<FW>(rL, ch));
      const bf16x8 aU = *(const bf16x8*)(X + swz<FW>(rU, ch));
      bf16x8 b1[2], b2[2];
#pragma unroll
      for (int t = 0; t < 2; t++) {
        const int nr = 32 * t + (lane & 31);
        b1[t] = *(const bf16x8*)(Ws + swz<FW>(nr, ch));
        b2[t] = *(const bf16x8*)(Wo + swz<FW>(nr, ch));
      }
      // self terms first, partner terms after: no MFMA waits on the one before it
#pragma unroll
      for (int t = 0; t < 2; t++) {
        accL[t] = mfma32(b1[t], aL, accL[t]);
        accU[t] = mfma32(b1[t], aU, accU[t]);
      }
#pragma unroll
      for (int t = 0; t < 2; t++) {
        accU[t] = mfma32(b2[t], aL, accU[t]);
        if (BIDIR) accL[t] = mfma32(b2[t], aU, accL[t]);
      }
    }
    store_rows(Y, accL, accU, rL, rU, lane);
    wait_dma();
    __syncthreads();  // Y complete, next weights landed, X and this layer's weights free
    bf16* dst = a.xs[l] + win;
    for (int p = tid; p < n * FW / 8; p += nthreads) {
      const int row = p / (FW / 8), ch = p % (FW / 8);
      *(u32x4*)(dst + (size_t)row * FW + ch * 8) = *(const u32x4*)(Y + swz<FW>(row, ch));
    }
    bf16* t = X;
    X = Y;
    Y = t;
  }
}

// ---------------------------------------------------------------------------
// Backward: walks the layers in reverse with the gradient resident in LDS.
// Per layer: per-window weight-gradient blocks to `partial`, then dX.
// ---------------------------------------------------------------------------
template <bool BIDIR>
__global__ __launch_bounds__(256) void fused_bwd_kernel(FusedBwdArgs a) {
  extern __shared__ __attribute__((aligned(1024))) bf16 smem[];
  const int n = a.n, nw = n / 64, nthreads = 64 * nw;
  const int L = a.num_layers;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const size_t win = (size_t)blockIdx.x * n * FW;
  bf16* G = smem;          // gradient of the current layer's output
  bf16* Gn = G + n * FW;   // gradient of its input (being built)
  bf16* Xb = Gn + n * FW;  // the current layer's input
  bf16* Wb = Xb + n * FW;  // two sets of [W_self | W_off], transposed-read layout

  dma_act(a.dy + win, G, n, wave, nw, lane);
  dma_act(a.xs[L - 1] + win, Xb, n, wave, nw, lane);
  dma_w_tr(a.ws[L - 1], Wb + ((L - 1) & 1) * 2 * WW, wave, nw, lane);
  dma_w_tr(a.wo[L - 1], Wb + ((L - 1) & 1) * 2 * WW + WW, wave, nw, lane);
  wait_dma();
  __syncthreads();

  for (int l = L - 1; l >= 0; l--) {
    const int d = a.dim[l], s = 1 << d;
    const bf16* Ws = Wb + (l & 1) * 2 * WW;
    const bf16* Wo = Ws + WW;
    if (l > 0) {
      bf16* Wn = Wb + ((l - 1) & 1) * 2 * WW;
      dma_w_tr(a.ws[l - 1], Wn, wave, nw, lane);
      dma_w_tr(a.wo[l - 1], Wn + WW, wave, nw, lane);
    }
    auto same = [](int k) { return k; };
    auto lowr = [d](int k) { return lower_row(k, d); };
    auto uppr = [d, s](int k) { return lower_row(k, d) + s; };

    // 1. weight-gradient blocks: 0..3 of dW_self, 4..7 of dW_off (32 x 32 each)
    float* part = a.partial + ((size_t)blockIdx.x * L + l) * 2 * WW;
    for (int blk = wave; blk < 8; blk += nw) {
      const int is_off = blk >> 2, ob = ((blk >> 1) & 1) * 32, cb = (blk & 1) * 32;
      f32x16 acc;
#pragma unroll
      for (int e = 0; e < 16; e++) acc[e] = 0.f;
      if (!is_off) {
        for (int k0 = 0; k0 < n; k0 += 16)
          acc = mfma32(tr_act(G, k0, ob, lane, same), tr_act(Xb, k0, cb, lane, same), acc);
      } else {
        // receivers' gradients against their senders' inputs, over the n/2 pairs
        for (int k0 = 0; k0 < n / 2; k0 += 16) {
          acc = mfma32(tr_act(G, k0, ob, lane, uppr), tr_act(Xb, k0, cb, lane, lowr), acc);
          if (BIDIR) acc = mfma32(tr_act(G, k0, ob, lane, lowr), tr_act(Xb, k0, cb, lane, uppr), acc);
        }
      }
      float* dst = part + is_off * WW;
#pragma unroll
      for (int e = 0; e < 16; e++) {
        const int o = ob + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        dst[o * FW + cb + (lane & 31)] = acc[e];
      }
    }
    __syncthreads();  // Xb free
    if (l > 0) dma_act(a.xs[l - 1] + win, Xb, n, wave, nw, lane);

    // 2. dX: lower rows always take their partner's gradient through W_off^T
    //    (causal: the lower row is the sender), upper rows only when bidirectional.
    f32x16 accL[2], accU[2];
#pragma unroll
    for (int t = 0; t < 2; t++)
#pragma unroll
      for (int e = 0; e < 16; e++) { accL[t][e] = 0.f; accU[t][e] = 0.f; }
    const int rL = lower_row(32 * wave + (lane & 31), d), rU = rL + s;
#pragma unroll
    for (int kk = 0; kk < FW / 16; kk++) {
      const int ch = kk * 2 + (lane >> 5);
      const bf16x8 gL = *(const bf16x8*)(G + swz<FW>(rL, ch));
      const bf16x8 gU = *(const bf16x8*)(G + swz<FW>(rU, ch));
      bf16x8 b1[2], b2[2];
#pragma unroll
      for (int t = 0; t < 2; t++) {
        b1[t] = tr_frag<FRB>(Ws, kk * 16, 32 * t, lane);
        b2[t] = tr_frag<FRB>(Wo, kk * 16, 32 * t, lane);
      }
#pragma unroll
      for (int t = 0; t < 2; t++) {
        accL[t] = mfma32(b1[t], gL, accL[t]);
        accU[t] = mfma32(b1[t], gU, accU[t]);
      }
#pragma unroll
      for (int t = 0; t < 2; t++) {
        accL[t] = mfma32(b2[t], gU, accL[t]);
        if (BIDIR) accU[t] = mfma32(b2[t], gL, accU[t]);
      }
    }
    store_rows(Gn, accL, accU, rL, rU, lane);
    wait_dma();
    __syncthreads();  // Gn complete; next input and weights landed
    bf16* t = G;
    G = Gn;
    Gn = t;
  }
  bf16* dst = a.dx + win;
  for (int p = tid; p < n * FW / 8; p += nthreads) {
    const int row = p / (FW / 8), ch = p % (FW / 8);
    *(u32x4*)(dst + (size_t)row * FW + ch * 8) = *(const u32x4*)(G + swz<FW>(row, ch));
  }
}

// dW_self[l] / dW_off[l] (+)= sum over windows of the partials.  Each block
// handles 64 float4 outputs; its 4 thread groups sum consecutive quarters of
// the windows in window order, and the quarters are then added in order, so
// the result is the same on every run.
constexpr int RED_OUT = 64;   // float4 outputs per block
__global__ __launch_bounds__(256) void fused_dw_reduce_kernel(FusedReduceArgs a) {
  __shared__ f32x4 part[4][RED_OUT];
  const int per = WW / 4;                           // float4 per matrix
  const int idx = blockIdx.x * RED_OUT + (threadIdx.x % RED_OUT);
  const int quarter = threadIdx.x / RED_OUT;
  const int l = idx / (2 * per), m = (idx / per) % 2, j = idx % per;
  const int q_len = (a.batch + 3) / 4;
  const int b0 = quarter * q_len, b1 = min(a.batch, b0 + q_len);
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int b = b0; b < b1; b++)
    acc += ((const f32x4*)(a.partial + (((size_t)b * a.num_layers + l) * 2 + m) * WW))[j];
  part[quarter][threadIdx.x % RED_OUT] = acc;
  __syncthreads();
  if (quarter == 0) {
    const int o = threadIdx.x;
    f32x4 sum = part[0][o];
    sum += part[1][o];
    sum += part[2][o];
    sum += part[3][o];
    f32x4* dst = (f32x4*)(m ? a.dwo[l] : a.dws[l]) + j;
    if (a.accumulate) sum += *dst;
    *dst = sum;
  }
}

size_t fwd_lds_bytes(int n) { return ((size_t)2 * n * FW + 4 * WW) * sizeof(bf16); }
size_t bwd_lds_bytes(int n) { return ((size_t)3 * n * FW + 4 * WW) * sizeof(bf16); }

}  // namespace

bool fused_stack_eligible(int64_t n, int64_t width, int32_t num_layers) {
  return width == FW && (n == 64 || n == 128 || n == 256) && num_layers >= 1 &&
         num_layers <= kFusedMaxLayers;
}

size_t fused_partial_bytes(int64_t batch, int32_t num_layers) {
  return (size_t)batch * num_layers * 2 * WW * sizeof(float);
}

hipError_t launch_fused_forward(const FusedFwdArgs& a, int batch, bool bidir, hipStream_t st) {
  const size_t lds = fwd_lds_bytes(a.n);
  const int threads = 64 * (a.n / 64);
  if (bidir) {
    static const hipError_t attr = hipFuncSetAttribute(
        (const void*)fused_fwd_kernel<true>, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (attr != hipSuccess) return attr;
    fused_fwd_kernel<true><<<batch, threads, lds, st>>>(a);
  } else {
    static const hipError_t attr = hipFuncSetAttribute(
        (const void*)fused_fwd_kernel<false>, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (attr != hipSuccess) return attr;
    fused_fwd_kernel<false><<<batch, threads, lds, st>>>(a);
  }
  return hipGetLastError();
}

hipError_t launch_fused_backward(const FusedBwdArgs& a, const FusedReduceArgs& r, int batch,
                                 bool bidir, hipStream_t st) {
  const size_t lds = bwd_lds_bytes(a.n);
  const int threads = 64 * (a.n / 64);
  if (bidir) {
    static const hipError_t attr = hipFuncSetAttribute(
        (const void*)fused_bwd_kernel<true>, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (attr != hipSuccess) return attr;
    fused_bwd_kernel<true><<<batch, threads, lds, st>>>(a);
  } else {
    static const hipError_t attr = hipFuncSetAttribute(
        (const void*)fused_bwd_kernel<false>, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (attr != hipSuccess) return attr;
    fused_bwd_kernel<false><<<batch, threads, lds, st>>>(a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int blocks = r.num_layers * 2 * (WW / 4) / RED_OUT;   // exact: WW/4 = 1024
  fused_dw_reduce_kernel<<<blocks, 256, 0, st>>>(r);
  return hipGetLastError();
}

}  // namespace hcmix
