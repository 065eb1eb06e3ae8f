// Fused small-width stack (bf16, width 64, n in {64, 128, 256}): every window
// of n positions x 64 features stays in LDS through all layers, so the whole
// forward stack is one launch and the whole backward stack one launch plus a
// fixed-order reduction of the per-window weight gradients.  One block per
// window, n/64 waves, each wave owning 32 row pairs of the current layer.
//
// Activation buffers use the k-contiguous swizzle (rows of 128 bytes, 16-byte
// piece ch stored at ch ^ ((row >> 1) & 7)); weight buffers read transposed
// (backward) use the 64-byte segment swizzle of tr_frag.  Fragments whose
// contraction index runs over row pairs are gathered with ds_read_b64_tr_b16.
//
// In the forward kernel the per-layer arguments (dimension, weight and
// activation pointers) are copied into LDS once at kernel start, so a layer
// never waits on a scalar load of the kernel-argument block.
#include <type_traits>

#include "device_common.h"
#include "hcmix_internal.h"

namespace hcmix {

namespace {

constexpr int FW = 64;        // width of the fused path
constexpr int FRB = 2 * FW;   // bytes per activation / weight row
constexpr int WW = FW * FW;   // elements per weight matrix

struct LayerArg {
  const bf16* ws;
  const bf16* wo;
  bf16* xs;
  int d, pad;
};
constexpr int ARG_BYTES = kFusedMaxLayers * (int)sizeof(LayerArg);

__device__ __forceinline__ int act_off(int row, int col) {
  return swz<FW>(row, col >> 3) + (col & 7);
}

// ---- transposed pair fragments ------------------------------------------
// A 16-pair step k0 .. k0+15 (k0 % 16 == 0) of dimension d covers the lower
// rows base + off(delta), delta = 0..15, with
//   d < 4:  base = 2 k0,               off(delta) = lower_row(delta, d)
//   d >= 4: base = lower_row(k0, d),   off(delta) = delta
// and base a multiple of 16, so act_off(base + r, c) = base * FW + act_off(r, c)
// (the swizzle only sees row bits 1..3).  Each lane's two reads of a
// fragment (contraction rows 8 (l/32) + (l%16)/4 and +4, column c0 + 16 ((l/16)%2)
// + 4 (l%4)) therefore sit at a per-layer lane constant plus a per-step base.
struct PairOffs {
  int lo_l, hi_l, lo_u, hi_u;   // element offsets: lower / upper pair member
};

__device__ __forceinline__ PairOffs pair_offs(int c0, int lane, int d) {
  const int g = lane >> 4, j = lane & 15;
  const int dl = 8 * (g >> 1) + (j >> 2);
  const int col = c0 + 16 * (g & 1) + 4 * (j & 3);
  const int s = 1 << d;
  const int rl = d < 4 ? lower_row(dl, d) : dl;
  const int rh = d < 4 ? lower_row(dl + 4, d) : dl + 4;
  return {act_off(rl, col), act_off(rh, col), act_off(rl + s, col), act_off(rh + s, col)};
}

__device__ __forceinline__ int step_base(int k0, int d) {
  return d < 4 ? 2 * k0 : lower_row(k0, d);
}

// Lane l receives buf[row(k0 + 8 (l/32) + t)][c0 + l%32], t = 0..7 (the MFMA
// operand layout with the contraction over pairs).
__device__ __forceinline__ bf16x8 tr_pair(const bf16* step, int lo, int hi) {
  const bf16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(step + lo));
  const bf16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(step + hi));
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// ---- staging -------------------------------------------------------------
// Window rows (N rows of 128 bytes) global -> LDS in the activation swizzle.
template <int N, int NW>
__device__ __forceinline__ void dma_act(const bf16* src, bf16* dst, int wave, int lane) {
  static_assert((N / 8) % NW == 0, "");
#pragma unroll
  for (int i = 0; i < N / 8 / NW; i++) {
    const int b = wave + i * NW;
    const int o = b * 1024 + 16 * lane;
    const int row = o / FRB;
    const int ch = ((o % FRB) / 16) ^ ((row >> 1) & 7);
    dma16(src + (size_t)row * FW + ch * 8, dst + b * 512);
  }
}

// One weight matrix global -> LDS, k-contiguous rows (forward B operand).
template <int NW>
__device__ __forceinline__ void dma_w_rows(const bf16* src, bf16* dst, int wave, int lane) {
  static_assert(8 % NW == 0, "");
#pragma unroll
  for (int i = 0; i < 8 / NW; i++) {
    const int b = wave + i * NW;
    const int o = b * 1024 + 16 * lane;
    const int row = o / FRB;
    const int ch = ((o % FRB) / 16) ^ ((row >> 1) & 7);
    dma16(src + (size_t)row * FW + ch * 8, dst + b * 512);
  }
}

// One weight matrix global -> LDS for transposed reads (backward B operand).
template <int NW>
__device__ __forceinline__ void dma_w_tr(const bf16* src, bf16* dst, int wave, int lane) {
#pragma unroll
  for (int i = 0; i < 8 / NW; i++) {
    const int b = wave + i * NW;
    int row, col;
    tr_dma_coord<FRB>(b, lane, &row, &col);
    dma16(src + (size_t)row * FW + col, dst + b * 512);
  }
}

// Rounds column block t (32 columns) of a wave's output rows to bf16 into an
// activation buffer (transposed accumulators: lane l holds row rL / rU and
// columns 32 t + 8 (e/4) + 4 (l/32) + e%4).
__device__ __forceinline__ void store_block(bf16* buf, const f32x16& accL, const f32x16& accU,
                                            int rL, int rU, int t, int lane) {
#pragma unroll
  for (int g = 0; g < 4; g++) {
    const int col = 32 * t + 8 * g + 4 * (lane >> 5);
    const bf16x4 vl = {to_bf16(accL[4 * g]), to_bf16(accL[4 * g + 1]), to_bf16(accL[4 * g + 2]),
                       to_bf16(accL[4 * g + 3])};
    const bf16x4 vu = {to_bf16(accU[4 * g]), to_bf16(accU[4 * g + 1]), to_bf16(accU[4 * g + 2]),
                       to_bf16(accU[4 * g + 3])};
    *(bf16x4*)(buf + act_off(rL, col)) = vl;
    *(bf16x4*)(buf + act_off(rU, col)) = vu;
  }
}

// 16-byte pieces p0, p0 + stride, ... (K of them) of a window's activation
// buffer -> their row-major places in global memory; all LDS reads first.
// WT writes through L2 (store_wt16), which pays for copies that overlap later
// compute; a copy that ends the kernel is faster with ordinary stores.
template <int K, bool WT>
__device__ __forceinline__ void copy_out(const bf16* buf, bf16* dst, int p0, int stride) {
  u32x4 v[K];
#pragma unroll
  for (int i = 0; i < K; i++) {
    const int p = p0 + i * stride;
    v[i] = *(const u32x4*)(buf + swz<FW>(p / (FW / 8), p % (FW / 8)));
  }
#pragma unroll
  for (int i = 0; i < K; i++) {
    const int p = p0 + i * stride;
    bf16* q = dst + (size_t)(p / (FW / 8)) * FW + (p % (FW / 8)) * 8;
    if (WT)
      store_wt16(q, v[i]);
    else
      *(global_u32x4*)q = v[i];
  }
}

template <int N> constexpr size_t fwd_lds() { return (size_t)(2 * N * FW + 4 * WW) * 2 + ARG_BYTES; }
template <int N> constexpr size_t bwd_lds() { return (size_t)(4 * N * FW + 4 * WW) * 2; }

// ---------------------------------------------------------------------------
// Forward: x_{l+1} = layer_l(x_l) for l = 0..L-1, each x_{l+1} also stored.
//
// 3 n / 64 waves in two roles:
//  * 2 n / 64 compute waves (two per SIMD at n = 256): wave w multiplies the
//    32 row pairs of block w / 2 into the 32 output columns of half w % 2 and
//    fetches its share of the next layer's weights;
//  * n / 64 store waves copy x_l (the layer's input, in LDS during layer l)
//    to global memory.  A CU writes to memory at roughly half the rate it
//    reads, so the stores take about as long as the layer's MFMAs; in waves
//    of their own they never hold up an MFMA, and no wave waits for them to
//    complete (the LDS reads that feed them finish before the layer ends).
// ---------------------------------------------------------------------------
template <int N, bool BIDIR>
__global__ __launch_bounds__(3 * N) void fused_fwd_kernel(FusedFwdArgs a) {
  constexpr int CT = 2 * N, CW = CT / 64;   // compute threads / waves
  constexpr int SPT = N * FW / 8 / N;       // 16-byte pieces per store thread (8)
  constexpr int CPT = N * FW / 8 / CT;      // pieces per compute thread (4)
  extern __shared__ __attribute__((aligned(1024))) bf16 smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool compute = wave < CW;
  const int pb = wave >> 1, half = wave & 1;
  const int L = a.num_layers;
  const size_t win = (size_t)blockIdx.x * N * FW;
  bf16* X = smem;
  bf16* Y = X + N * FW;
  bf16* Wb = Y + N * FW;  // two sets of [W_self | W_off]
  LayerArg* tab = (LayerArg*)(Wb + 4 * WW);

  if (tid < L) tab[tid] = LayerArg{a.ws[tid], a.wo[tid], a.xs[tid], a.dim[tid], 0};
  if (compute) {
    dma_act<N, CW>(a.x0 + win, X, wave, lane);
    dma_w_rows<CW>(a.ws[0], Wb, wave, lane);
    dma_w_rows<CW>(a.wo[0], Wb + WW, wave, lane);
    wait_dma();
  }
  __syncthreads();

  for (int l = 0; l < L; l++) {
    if (compute) {
      const int d = tab[l].d, s = 1 << d;
      const bf16* Ws = Wb + (l & 1) * 2 * WW;
      const bf16* Wo = Ws + WW;
      if (l + 1 < L) {
        bf16* Wn = Wb + ((l + 1) & 1) * 2 * WW;
        dma_w_rows<CW>(tab[l + 1].ws, Wn, wave, lane);
        dma_w_rows<CW>(tab[l + 1].wo, Wn + WW, wave, lane);
      }
      const int rL = lower_row(32 * pb + (lane & 31), d), rU = rL + s;
      const int nr = 32 * half + (lane & 31);
      bf16x8 aL[4], aU[4], b1[4], b2[4];
#pragma unroll
      for (int kk = 0; kk < 4; kk++) {
        const int ch = kk * 2 + (lane >> 5);
        aL[kk] = *(const bf16x8*)(X + swz<FW>(rL, ch));
        aU[kk] = *(const bf16x8*)(X + swz<FW>(rU, ch));
        b1[kk] = *(const bf16x8*)(Ws + swz<FW>(nr, ch));
        b2[kk] = *(const bf16x8*)(Wo + swz<FW>(nr, ch));
      }
      f32x16 accL, accU;
#pragma unroll
      for (int e = 0; e < 16; e++) { accL[e] = 0.f; accU[e] = 0.f; }
#pragma unroll
      for (int kk = 0; kk < 4; kk++) {
        accL = mfma32(b1[kk], aL[kk], accL);
        accU = mfma32(b1[kk], aU[kk], accU);
        accU = mfma32(b2[kk], aL[kk], accU);
        if (BIDIR) accL = mfma32(b2[kk], aU[kk], accL);
      }
      store_block(Y, accL, accU, rL, rU, half, lane);
      wait_dma();  // this wave's share of the next weights
    } else if (l > 0) {
      bf16* dst = tab[l - 1].xs + win;
      copy_out<SPT, true>(X, dst, tid - CT, N);
    }
    __syncthreads();  // Y complete, next weights landed, X and this layer's weights free
    bf16* t = X;
    X = Y;
    Y = t;
  }
  if (compute) {
    bf16* dst = tab[L - 1].xs + win;
    copy_out<CPT, false>(X, dst, tid, CT);
  }
}

// ---------------------------------------------------------------------------
// Backward: walks the layers in reverse with the gradient resident in LDS.
//
// A window's backward may be shared by `split` blocks (small batches, so that
// the grid fills the chip): every block runs the dX chain from the top layer
// down, which needs only dY and the weights, and forms the weight gradients
// of its own layers lo .. hi only, so it reads only those layers' inputs;
// block 0 owns the lowest layers and also writes dx.  Each (window, layer)
// partial is still written by exactly one block, and every value is formed
// by the same sequence of operations whatever the split, so the results do
// not depend on it (bitwise).
//
// Per layer, 2 n / 64 waves in two roles that run side by side (one wave of
// each role per SIMD at n = 256); they share only the gradient G, which both
// read:
//  * weight-gradient waves: block c (0..3) is the 32 x 32 piece (outputs ob,
//    inputs cb) of both dW_self and dW_off; one pass over the row pairs reads
//    the fragments dY_L, dY_U (outputs) and X_L, X_U (inputs) and feeds
//      dW_self += dY_L^T X_L + dY_U^T X_U,  dW_off += dY_U^T X_L (+ dY_L^T X_U bidir),
//    then stores the window's partial;
//  * dX waves: 32 row pairs each, in two 32-column halves (the second half's
//    MFMAs carry the first half's rounding and LDS writes).
// A layer above the block's own takes the dX alone, and then every wave
// takes one 32-column half of 32 row pairs; the block's lowest layer (blocks
// other than 0) takes the weight gradients alone.  The first two layer inputs
// the block needs are fetched at the start, the others one layer ahead
// (double-buffered), the weights one layer ahead.  The per-layer arguments
// are read from the kernel-argument block (the four activation buffers and
// two weight sets fill the 160 KB of LDS at n = 256).
// ---------------------------------------------------------------------------
template <int N, bool BIDIR>
__global__ __launch_bounds__(2 * N) void fused_bwd_kernel(FusedBwdArgs a) {
  constexpr int NT = 2 * N, NW = NT / 64, HW = NW / 2;
  constexpr int PCS = N * FW / 8 / NT;
  extern __shared__ __attribute__((aligned(1024))) bf16 smem[];
  const int L = a.num_layers;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int part = (int)(blockIdx.x % (unsigned)a.split);
  const size_t win = (size_t)(blockIdx.x / (unsigned)a.split) * N * FW;
  const int lo = a.lo[part], hi = a.hi[part];
  const int last = part == 0 ? 0 : lo;   // the lowest layer this block visits
  bf16* G = smem;            // gradient of the current layer's output
  bf16* Gn = G + N * FW;     // gradient of its input (being built)
  bf16* Xs = Gn + N * FW;    // two layer-input buffers: x_l in buffer l % 2
  bf16* Wb = Xs + 2 * N * FW;  // two sets of [W_self | W_off], transposed-read layout

  dma_act<N, NW>(a.dy + win, G, wave, lane);
  dma_w_tr<NW>(a.ws[L - 1], Wb + ((L - 1) & 1) * 2 * WW, wave, lane);
  dma_w_tr<NW>(a.wo[L - 1], Wb + ((L - 1) & 1) * 2 * WW + WW, wave, lane);
  dma_act<N, NW>(a.xs[hi] + win, Xs + (hi & 1) * N * FW, wave, lane);
  const bool two = hi - 1 >= lo;
  if (two) dma_act<N, NW>(a.xs[hi - 1] + win, Xs + ((hi - 1) & 1) * N * FW, wave, lane);
  // the top layer needs dY, its weights and (if it is the block's own) its
  // input; the other inputs may still be in flight (loads complete in issue
  // order, XI per activation buffer and wave) until the layer's closing wait
  constexpr int XI = N / 8 / NW;
  const int pending = (two ? 2 : 1) - (hi == L - 1 ? 1 : 0);
  if (pending == 2)
    wait_vmcnt<2 * XI>();
  else if (pending == 1)
    wait_vmcnt<XI>();
  else
    wait_dma();
  __syncthreads();

  for (int l = L - 1; l >= last; l--) {
    const int d = a.dim[l], s = 1 << d;
    const bool do_dw = l >= lo && l <= hi;
    const bool do_dx = l > lo || part == 0;
    const bf16* Ws = Wb + (l & 1) * 2 * WW;
    const bf16* Wo = Ws + WW;
    const bf16* Xb = Xs + (l & 1) * N * FW;
    if (l > last) {
      if (l - 1 > lo || part == 0) {
        bf16* Wn = Wb + ((l - 1) & 1) * 2 * WW;
        dma_w_tr<NW>(a.ws[l - 1], Wn, wave, lane);
        dma_w_tr<NW>(a.wo[l - 1], Wn + WW, wave, lane);
      }
      if (l < hi && l - 1 >= lo)
        dma_act<N, NW>(a.xs[l - 1] + win, Xs + ((l - 1) & 1) * N * FW, wave, lane);
    }
    if (do_dw && wave < HW) {
      // weight-gradient partials of this window
      float* prt = a.partial + ((size_t)(blockIdx.x / (unsigned)a.split) * L + l) * 2 * WW;
#pragma unroll
      for (int c = wave; c < 4; c += HW) {
        const int ob = (c >> 1) * 32, cb = (c & 1) * 32;
        const PairOffs pg = pair_offs(ob, lane, d), px = pair_offs(cb, lane, d);
        f32x16 accS, accO;
#pragma unroll
        for (int e = 0; e < 16; e++) { accS[e] = 0.f; accO[e] = 0.f; }
        // fragments of the 16-pair step at k0: dY_L, dY_U, X_L, X_U
        auto frags = [&](bf16x8 (&f)[4], int k0) {
          const int base = step_base(k0, d) * FW;
          f[0] = tr_pair(G + base, pg.lo_l, pg.hi_l);
          f[1] = tr_pair(G + base, pg.lo_u, pg.hi_u);
          f[2] = tr_pair(Xb + base, px.lo_l, px.hi_l);
          f[3] = tr_pair(Xb + base, px.lo_u, px.hi_u);
        };
        auto mma = [&](const bf16x8 (&f)[4]) {
          accS = mfma32(f[2], f[0], accS);
          accO = mfma32(f[2], f[1], accO);
          accS = mfma32(f[3], f[1], accS);
          if (BIDIR) accO = mfma32(f[3], f[0], accO);
        };
        // each step's reads are issued under the previous step's MFMAs
        bf16x8 fr[2][4];
        frags(fr[0], 0);
#pragma unroll
        for (int k = 0; k < N / 32; k++) {
          if (k + 1 < N / 32) frags(fr[(k + 1) & 1], 16 * (k + 1));
          mma(fr[k & 1]);
        }
        // transposed accumulators: lane l holds output ob + l%32 and inputs
        // cb + 8 g + 4 (l/32) + 0..3.  Ordinary stores: the data comes
        // straight from MFMA accumulators, and the split into 8-byte
        // write-through stores left half-written sectors that doubled the
        // HBM writes.
        float* rowS = prt + (size_t)(ob + (lane & 31)) * FW + cb + 4 * (lane >> 5);
#pragma unroll
        for (int g = 0; g < 4; g++) {
          *(f32x4*)(rowS + 8 * g) = f32x4{accS[4 * g], accS[4 * g + 1], accS[4 * g + 2], accS[4 * g + 3]};
          *(f32x4*)(rowS + WW + 8 * g) = f32x4{accO[4 * g], accO[4 * g + 1], accO[4 * g + 2], accO[4 * g + 3]};
        }
      }
    } else if (do_dx && wave >= HW && do_dw) {
      // dX beside the weight gradients: lower rows always take their
      // partner's gradient through W_off^T (causal: the lower row is the
      // sender), upper rows only when bidirectional.
      const int rL = lower_row(32 * (wave - HW) + (lane & 31), d), rU = rL + s;
      bf16x8 gL[4], gU[4], b1[2][4], b2[2][4];
#pragma unroll
      for (int kk = 0; kk < 4; kk++) {
        const int ch = kk * 2 + (lane >> 5);
        gL[kk] = *(const bf16x8*)(G + swz<FW>(rL, ch));
        gU[kk] = *(const bf16x8*)(G + swz<FW>(rU, ch));
        b1[0][kk] = tr_frag<FRB>(Ws, kk * 16, 0, lane);
        b2[0][kk] = tr_frag<FRB>(Wo, kk * 16, 0, lane);
      }
      f32x16 accL[2], accU[2];
#pragma unroll
      for (int t = 0; t < 2; t++)
#pragma unroll
        for (int e = 0; e < 16; e++) { accL[t][e] = 0.f; accU[t][e] = 0.f; }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kk = 0; kk < 4; kk++) {
        b1[1][kk] = tr_frag<FRB>(Ws, kk * 16, 32, lane);
        b2[1][kk] = tr_frag<FRB>(Wo, kk * 16, 32, lane);
        accL[0] = mfma32(b1[0][kk], gL[kk], accL[0]);
        accU[0] = mfma32(b1[0][kk], gU[kk], accU[0]);
        accL[0] = mfma32(b2[0][kk], gU[kk], accL[0]);
        if (BIDIR) accU[0] = mfma32(b2[0][kk], gL[kk], accU[0]);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kk = 0; kk < 4; kk++) {
        accL[1] = mfma32(b1[1][kk], gL[kk], accL[1]);
        accU[1] = mfma32(b1[1][kk], gU[kk], accU[1]);
        accL[1] = mfma32(b2[1][kk], gU[kk], accL[1]);
        if (BIDIR) accU[1] = mfma32(b2[1][kk], gL[kk], accU[1]);
      }
      store_block(Gn, accL[0], accU[0], rL, rU, 0, lane);
      __builtin_amdgcn_sched_barrier(0);
      store_block(Gn, accL[1], accU[1], rL, rU, 1, lane);
    } else if (do_dx && !do_dw) {
      // dX alone: every wave takes one 32-column half of 32 row pairs, with
      // the same operations per output as above.
      const int t = wave / HW;
      const int rL = lower_row(32 * (wave % HW) + (lane & 31), d), rU = rL + s;
      bf16x8 gL[4], gU[4], b1[4], b2[4];
#pragma unroll
      for (int kk = 0; kk < 4; kk++) {
        const int ch = kk * 2 + (lane >> 5);
        gL[kk] = *(const bf16x8*)(G + swz<FW>(rL, ch));
        gU[kk] = *(const bf16x8*)(G + swz<FW>(rU, ch));
        b1[kk] = tr_frag<FRB>(Ws, kk * 16, 32 * t, lane);
        b2[kk] = tr_frag<FRB>(Wo, kk * 16, 32 * t, lane);
      }
      f32x16 accL, accU;
#pragma unroll
      for (int e = 0; e < 16; e++) { accL[e] = 0.f; accU[e] = 0.f; }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kk = 0; kk < 4; kk++) {
        accL = mfma32(b1[kk], gL[kk], accL);
        accU = mfma32(b1[kk], gU[kk], accU);
        accL = mfma32(b2[kk], gU[kk], accL);
        if (BIDIR) accU = mfma32(b2[kk], gL[kk], accU);
      }
      store_block(Gn, accL, accU, rL, rU, t, lane);
    }
    wait_dma();
    __syncthreads();  // Gn complete, partial stored; next input and weights landed
    bf16* tmp = G;
    G = Gn;
    Gn = tmp;
  }
  if (part == 0) copy_out<PCS, false>(G, a.dx + win, tid, NT);
}

// dW_self[l] / dW_off[l] (+)= sum over windows of the partials.  Each block
// handles 64 float4 outputs with 1024 threads: its 16 thread groups sum
// consecutive sixteenths of the windows in window order (every wave reads
// 1 KB contiguous per window), and the 16 group sums are then added in
// order, so the result is the same on every run.
constexpr int RED_OUT = 64;    // float4 outputs per block
constexpr int RED_GROUPS = 16;
__global__ __launch_bounds__(RED_OUT * RED_GROUPS) void fused_dw_reduce_kernel(FusedReduceArgs a) {
  __shared__ f32x4 part[RED_GROUPS][RED_OUT];
  const int per = WW / 4;                           // float4 per matrix
  const int o = threadIdx.x % RED_OUT, grp = threadIdx.x / RED_OUT;
  const int idx = blockIdx.x * RED_OUT + o;
  const int l = idx / (2 * per), m = (idx / per) % 2, j = idx % per;
  const int q_len = (a.batch + RED_GROUPS - 1) / RED_GROUPS;
  const int b0 = grp * q_len, b1 = min(a.batch, b0 + q_len);
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int b = b0; b < b1; b++)
    acc += ((const f32x4*)(a.partial + (((size_t)b * a.num_layers + l) * 2 + m) * WW))[j];
  part[grp][o] = acc;
  __syncthreads();
  if (grp == 0) {
    f32x4 sum = part[0][o];
#pragma unroll
    for (int g = 1; g < RED_GROUPS; g++) sum += part[g][o];
    f32x4* dst = (f32x4*)(m ? a.dwo[l] : a.dws[l]) + j;
    if (a.accumulate) sum += *dst;
    store_wt16(dst, __builtin_bit_cast(u32x4, sum));
  }
}


template <int N, bool BIDIR>
hipError_t fwd_launch(const FusedFwdArgs& a, int batch, hipStream_t st) {
  static std::atomic<unsigned long long> lds_set{0};
  const hipError_t attr =
      lds_limit_once(lds_set, (const void*)fused_fwd_kernel<N, BIDIR>, (int)fwd_lds<N>());
  if (attr != hipSuccess) return attr;
  fused_fwd_kernel<N, BIDIR><<<batch, 3 * N, fwd_lds<N>(), st>>>(a);
  return hipGetLastError();
}

template <int N, bool BIDIR>
hipError_t bwd_launch(const FusedBwdArgs& a, int batch, hipStream_t st) {
  static std::atomic<unsigned long long> lds_set{0};
  const hipError_t attr =
      lds_limit_once(lds_set, (const void*)fused_bwd_kernel<N, BIDIR>, (int)bwd_lds<N>());
  if (attr != hipSuccess) return attr;
  fused_bwd_kernel<N, BIDIR><<<batch * a.split, 2 * N, bwd_lds<N>(), st>>>(a);
  return hipGetLastError();
}

template <bool BIDIR>
hipError_t fwd_dispatch(const FusedFwdArgs& a, int batch, hipStream_t st) {
  switch (a.n) {
    case 64: return fwd_launch<64, BIDIR>(a, batch, st);
    case 128: return fwd_launch<128, BIDIR>(a, batch, st);
    case 256: return fwd_launch<256, BIDIR>(a, batch, st);
    default: return hipErrorInvalidValue;
  }
}

template <bool BIDIR>
hipError_t bwd_dispatch(const FusedBwdArgs& a, int batch, hipStream_t st) {
  switch (a.n) {
    case 64: return bwd_launch<64, BIDIR>(a, batch, st);
    case 128: return bwd_launch<128, BIDIR>(a, batch, st);
    case 256: return bwd_launch<256, BIDIR>(a, batch, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

bool fused_stack_eligible(int64_t n, int64_t width, int32_t num_layers) {
  return width == FW && (n == 64 || n == 128 || n == 256) && num_layers >= 1 &&
         num_layers <= kFusedMaxLayers;
}

size_t fused_partial_bytes(int64_t batch, int32_t num_layers) {
  return (size_t)batch * num_layers * 2 * WW * sizeof(float);
}

hipError_t launch_fused_forward(const FusedFwdArgs& a, int batch, bool bidir, hipStream_t st) {
  return bidir ? fwd_dispatch<true>(a, batch, st) : fwd_dispatch<false>(a, batch, st);
}

// Compute units of the current device (cached per device).
static int device_cus() {
  static int cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int c = 0;
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        c <= 0)
      c = 256;
    cached[dev] = c;
  }
  return cached[dev];
}

// Relative time of a block of a split backward, from per-layer timings at
// n = 256 (in units of about 0.5 us): a layer that runs the dX alone 3, one
// with both roles 6, the lowest layer of a block other than 0 (weight
// gradients alone) 4, and every own layer after the first two one more (its
// input is fetched one layer ahead rather than at the start).
static int split_cost(int L, int lo, int hi, bool first) {
  const int own = hi - lo + 1;
  const int late = own > 2 ? own - 2 : 0;
  if (first) return 3 * (L - 1 - hi) + 6 * own + late;
  return 3 * (L - 1 - hi) + 6 * (own - 1) + 4 + late;
}

void fused_backward_split(int batch, int num_layers, int cus, int* split, int* lo, int* hi) {
  const int L = num_layers;
  int S = batch > 0 ? cus / batch : 1;
  S = S < 1 ? 1 : S;
  S = S > kFusedMaxSplit ? kFusedMaxSplit : S;
  S = S > L ? L : S;
  *split = S;
  if (S == 1) {
    lo[0] = 0;
    hi[0] = L - 1;
    return;
  }
  // smallest bound T on every block's cost that a top-down greedy partition
  // meets: each block from the top takes the longest range within T
  for (int T = 1;; T++) {
    int top = L - 1;
    bool ok = true;
    for (int j = S - 1; j >= 1 && ok; j--) {
      int best = -1;
      for (int c = j; c <= top; c++)
        if (split_cost(L, c, top, false) <= T) {
          best = c;
          break;
        }
      if (best < 0) {
        ok = false;
      } else {
        lo[j] = best;
        hi[j] = top;
        top = best - 1;
      }
    }
    if (ok && split_cost(L, 0, top, true) <= T) {
      lo[0] = 0;
      hi[0] = top;
      return;
    }
  }
}

hipError_t launch_fused_backward(const FusedBwdArgs& a0, const FusedReduceArgs& r, int batch,
                                 bool bidir, hipStream_t st) {
  FusedBwdArgs a = a0;
  fused_backward_split(batch, a.num_layers, device_cus(), &a.split, a.lo, a.hi);
  hipError_t e = bidir ? bwd_dispatch<true>(a, batch, st) : bwd_dispatch<false>(a, batch, st);
  if (e != hipSuccess) return e;
  const int blocks = r.num_layers * 2 * (WW / 4) / RED_OUT;   // exact: WW/4 = 1024
  fused_dw_reduce_kernel<<<blocks, RED_OUT * RED_GROUPS, 0, st>>>(r);
  return hipGetLastError();
}

}  // namespace hcmix
