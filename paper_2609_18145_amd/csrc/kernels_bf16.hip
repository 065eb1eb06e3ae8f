// bf16 path of the mixing layer on gfx950 matrix cores
// (v_mfma_f32_32x32x16_bf16: bf16 operands, fp32 accumulation).
//
// Every layer pairs each "lower" row (bit d clear) with its partner "upper"
// row (bit d set).  A block owns BMP lower rows and their BMP partners: the
// block's row set is closed under XOR 2^d for every stride 1 .. n/2, so the
// partner of LDS row m is LDS row m +- BMP and the XOR gather is just a
// different LDS base address; no permuted copy of the activations is ever
// written.  Each 16-byte load is a whole 16-byte piece of one row, so every
// stride is fetched at full line efficiency.
//
// Tiles move global -> LDS with global_load_lds_dwordx4 (lane i of a wave
// writes 16 bytes at LDS base + 16*i), so the swizzled LDS layouts below are
// produced by choosing each lane's source address.
//
// Operands whose contraction index is not the contiguous one (the weights in
// the dX product, both operands of the weight gradients) stay in their
// natural row-major layout in LDS and are read transposed with
// ds_read_b64_tr_b16: within each group of 16 lanes, source lane j points at
// row (base + j/4), column (c0 + 4*(j%4)); lane i then receives column c0 + i
// of those 4 rows.
#include "hcmix_internal.h"
#include "device_common.h"

namespace hcmix {

namespace {

// ---------------------------------------------------------------------------
// Mix GEMM.  For the block's lower rows L and upper rows U:
//   out_L = A_L B1^T + [PL] A_U B2^T
//   out_U = A_U B1^T + [PU] A_L B2^T
// B(n, k) is B[n*width + k] (k contiguous), or B[k*width + n] when TRANS_B.
// Forward: A = x, B1 = W_self, B2 = W_off, PU = 1, PL = bidir.
// dX:      A = dy, B = W read transposed, PL = 1, PU = bidir.
// ---------------------------------------------------------------------------
template <int BMP, int BN, int WM, int WN, int BK, int NS>
struct MixCfg {
  static constexpr int NT = 64 * WM * WN;
  static constexpr int NW = WM * WN;
  static constexpr int BM = 2 * BMP;
  static constexpr int TMP = BMP / (32 * WM);   // 32-row pair blocks per wave
  static constexpr int TN = BN / (32 * WN);     // 32-column blocks per wave
  static constexpr int A_ELEMS = BM * BK;
  static constexpr int B_ELEMS = BN * BK;       // same size in both layouts
  static constexpr int STAGE = A_ELEMS + 2 * B_ELEMS;
  static constexpr int LDO = BN + 8;            // row stride of the output staging tile
  static constexpr int LDS_ELEMS = (NS * STAGE > BM * LDO) ? NS * STAGE : BM * LDO;
  static constexpr int A_DMA = A_ELEMS * 2 / 1024 / NW;   // 1 KB DMA blocks per wave
  static constexpr int B_DMA = B_ELEMS * 2 / 1024 / NW;
  static constexpr int O_IT = BM * (BN / 8) / NT;
  static_assert(TMP >= 1 && TN >= 1, "tile too small for the wave grid");
  static_assert(A_DMA * NW * 1024 == A_ELEMS * 2 && B_DMA * NW * 1024 == B_ELEMS * 2, "");
  static constexpr int DPS = A_DMA + 2 * B_DMA;  // DMA instructions per wave per stage
  static_assert(O_IT * NT == BM * (BN / 8), "stores must tile evenly");
  static_assert(NS >= 2 && (NS - 2) * DPS <= 63, "vmcnt range");
};

// One block's work: `block` indexes the (row tile, column tile) grid, dealt
// to XCDs; `smem` is the block's dynamic LDS (MixCfg::LDS_ELEMS elements).
//
// The same block with no partner terms (PL = PU = false) is a plain product
// out = A B1^T (or A B1 with TRANS_B) over any row count: the linear maps of
// the hybrids' attention layers.  K is the contraction length and A's row
// stride, N the output columns, ldb the row stride of B (k-contiguous B: its
// rows are n; TRANS_B: its rows are k), ldo the output's row stride; the
// mixing layer has K = N = ldb = ldo = width.
template <int BMP, int BN, int WM, int WN, int BK, int NS, bool PL, bool PU, bool TRANS_B>
__device__ __forceinline__ void mix_bf16_block(
    const bf16* __restrict__ A, const bf16* __restrict__ B1, const bf16* __restrict__ B2,
    bf16* __restrict__ out, int pairs, int K, int N, int ldb, int ldo, int d, int block,
    bf16* smem) {
  using C = MixCfg<BMP, BN, WM, WN, BK, NS>;
  constexpr int RB = BN * 2;   // bytes per row of a transposed B tile
  constexpr bool HAS_B2 = PL || PU;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WM, wn = wave / WM;
  const int s = 1 << d;
  const int tiles_n = N / BN;
  const int tiles_m = (pairs + BMP - 1) / BMP;
  const int tile = xcd_tile(block, tiles_m * tiles_n);
  const int q0 = (tile / tiles_n) * BMP;
  const int n0 = (tile % tiles_n) * BN;

  // DMA sources (element offsets at k-slice 0) of this lane for each 1 KB block.
  const bf16* a_src[C::A_DMA];
#pragma unroll
  for (int j = 0; j < C::A_DMA; j++) {
    const int b = j * C::NW + wave;
    const int o = b * 1024 + 16 * lane;               // byte offset in the tile
    const int m = o / (2 * BK);                       // tile row
    const int ch = (swz<BK>(m, (o % (2 * BK)) / 16) - m * BK) / 8;   // swizzle is an involution
    int q = q0 + (m % BMP);
    if (q >= pairs) q = pairs - 1;  // ragged last block: load a valid row, never store it
    const int r = lower_row(q, d) + (m >= BMP ? s : 0);
    a_src[j] = A + (size_t)r * K + ch * 8;
  }
  size_t b_src[C::B_DMA];
#pragma unroll
  for (int j = 0; j < C::B_DMA; j++) {
    const int b = j * C::NW + wave;
    if constexpr (TRANS_B) {  // tile rows are k, columns n
      int kr, col;
      tr_dma_coord<RB>(b, lane, &kr, &col);
      b_src[j] = (size_t)kr * ldb + n0 + col;
    } else {                  // tile rows are n, columns k
      const int o = b * 1024 + 16 * lane;
      const int nr = o / (2 * BK);
      const int ch = (swz<BK>(nr, (o % (2 * BK)) / 16) - nr * BK) / 8;
      b_src[j] = (size_t)(n0 + nr) * ldb + ch * 8;
    }
  }
  const size_t b_step = TRANS_B ? (size_t)BK * ldb : BK;

  auto issue = [&](int kt, int stage) {
    bf16* sA = smem + stage * C::STAGE;
    bf16* sB1 = sA + C::A_ELEMS;
    bf16* sB2 = sB1 + C::B_ELEMS;
#pragma unroll
    for (int j = 0; j < C::A_DMA; j++) dma16(a_src[j] + kt * BK, sA + (j * C::NW + wave) * 512);
#pragma unroll
    for (int j = 0; j < C::B_DMA; j++) {
      dma16(B1 + b_src[j] + kt * b_step, sB1 + (j * C::NW + wave) * 512);
      if constexpr (HAS_B2) dma16(B2 + b_src[j] + kt * b_step, sB2 + (j * C::NW + wave) * 512);
    }
  };

  f32x16 accL[C::TMP][C::TN], accU[C::TMP][C::TN];
#pragma unroll
  for (int p = 0; p < C::TMP; p++)
#pragma unroll
    for (int t = 0; t < C::TN; t++)
#pragma unroll
      for (int e = 0; e < 16; e++) { accL[p][t][e] = 0.f; accU[p][t][e] = 0.f; }

  struct Frags { bf16x8 aL[C::TMP], aU[C::TMP], b1[C::TN], b2[C::TN]; };
  auto load_frags = [&](Frags& f, const bf16* sA, int kk) {
    const bf16* sB1 = sA + C::A_ELEMS;
    const bf16* sB2 = sB1 + C::B_ELEMS;
    const int ch = kk * 2 + (lane >> 5);
#pragma unroll
    for (int p = 0; p < C::TMP; p++) {
      const int m = (wm * C::TMP + p) * 32 + (lane & 31);
      f.aL[p] = *(const bf16x8*)(sA + swz<BK>(m, ch));
      f.aU[p] = *(const bf16x8*)(sA + swz<BK>(m + BMP, ch));
    }
#pragma unroll
    for (int t = 0; t < C::TN; t++) {
      const int nb = (wn * C::TN + t) * 32;
      if constexpr (TRANS_B) {
        f.b1[t] = tr_frag<RB>(sB1, kk * 16, nb, lane);
        if constexpr (HAS_B2) f.b2[t] = tr_frag<RB>(sB2, kk * 16, nb, lane);
      } else {
        f.b1[t] = *(const bf16x8*)(sB1 + swz<BK>(nb + (lane & 31), ch));
        if constexpr (HAS_B2) f.b2[t] = *(const bf16x8*)(sB2 + swz<BK>(nb + (lane & 31), ch));
      }
    }
  };
  // The accumulators hold the transposed product (weights as the MFMA "A"
  // operand, activation rows as "B"), so each lane owns one output row and 16
  // of its columns: the epilogue writes 8-byte runs instead of single values.
  auto mma = [&](const Frags& f) {
    // self terms first, partner terms after, so no MFMA waits on the one before it
#pragma unroll
    for (int p = 0; p < C::TMP; p++)
#pragma unroll
      for (int t = 0; t < C::TN; t++) {
        accL[p][t] = mfma32(f.b1[t], f.aL[p], accL[p][t]);
        accU[p][t] = mfma32(f.b1[t], f.aU[p], accU[p][t]);
      }
#pragma unroll
    for (int p = 0; p < C::TMP; p++)
#pragma unroll
      for (int t = 0; t < C::TN; t++) {
        if (PU) accU[p][t] = mfma32(f.b2[t], f.aL[p], accU[p][t]);
        if (PL) accL[p][t] = mfma32(f.b2[t], f.aU[p], accL[p][t]);
      }
  };

  constexpr int KK = BK / 16;
  constexpr int NMFMA = C::TMP * C::TN * (2 + (PL ? 1 : 0) + (PU ? 1 : 0));
  constexpr int NDS = 2 * C::TMP + (HAS_B2 ? 2 : 1) * C::TN * (TRANS_B ? 2 : 1);
  const int nk = K / BK;
  // NS-stage ring: stage kt lives in buffer kt % NS; while stage kt is being
  // multiplied, stages kt+1 .. kt+NS-1 are in flight.
#pragma unroll
  for (int st = 0; st < NS - 1; st++)
    if (st < nk) issue(st, st);
  Frags f[2];
  for (int kt = 0; kt < nk; kt++) {
    wait_stages<NS - 1, C::DPS>(min(nk, kt + NS - 1) - (kt + 1));
    __syncthreads();  // stage kt visible to all waves; buffer (kt-1) % NS free
    if (kt + NS - 1 < nk) issue(kt + NS - 1, (kt + NS - 1) % NS);
    const bf16* sA = smem + (kt % NS) * C::STAGE;
    load_frags(f[0], sA, 0);
#pragma unroll
    for (int kk = 0; kk < KK; kk++) {
      // one fenced region per kk: this kk's MFMAs with the next kk's reads
      if (kk + 1 < KK) {
        load_frags(f[(kk + 1) & 1], sA, kk + 1);
        mma(f[kk & 1]);
        interleave_front<NMFMA, NDS>();
      } else {
        mma(f[kk & 1]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  __syncthreads();  // every wave done with the stage buffers

  // Epilogue: round to bf16 into an LDS tile [BM][LDO], then 16-byte row stores.
  // Accumulator element e of lane l holds output row (lane's row l%32) and
  // column 8*(e/4) + 4*(l/32) + e%4 of its 32 x 32 block.
  bf16* sO = smem;
#pragma unroll
  for (int p = 0; p < C::TMP; p++)
#pragma unroll
    for (int t = 0; t < C::TN; t++) {
      const int m = (wm * C::TMP + p) * 32 + (lane & 31);
      const int col = (wn * C::TN + t) * 32 + 4 * (lane >> 5);
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const bf16x4 vl = {to_bf16(accL[p][t][4 * g]), to_bf16(accL[p][t][4 * g + 1]),
                           to_bf16(accL[p][t][4 * g + 2]), to_bf16(accL[p][t][4 * g + 3])};
        const bf16x4 vu = {to_bf16(accU[p][t][4 * g]), to_bf16(accU[p][t][4 * g + 1]),
                           to_bf16(accU[p][t][4 * g + 2]), to_bf16(accU[p][t][4 * g + 3])};
        *(bf16x4*)(sO + m * C::LDO + col + 8 * g) = vl;
        *(bf16x4*)(sO + (m + BMP) * C::LDO + col + 8 * g) = vu;
      }
    }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < C::O_IT; j++) {
    const int idx = tid + C::NT * j;
    const int m = idx / (BN / 8), ch = idx % (BN / 8);
    const int q = q0 + (m % BMP);
    if (q >= pairs) continue;
    const int r = lower_row(q, d) + (m >= BMP ? s : 0);
    store_wt16(out + (size_t)r * ldo + n0 + ch * 8, *(const u32x4*)(sO + m * C::LDO + ch * 8));
  }
}

template <int BMP, int BN, int WM, int WN, int BK, int NS, bool PL, bool PU, bool TRANS_B>
__global__ __launch_bounds__(64 * WM * WN) void mix_bf16_kernel(
    const bf16* __restrict__ A, const bf16* __restrict__ B1, const bf16* __restrict__ B2,
    bf16* __restrict__ out, int pairs, int K, int N, int ldb, int ldo, int d) {
  extern __shared__ __attribute__((aligned(1024))) bf16 smem[];
  mix_bf16_block<BMP, BN, WM, WN, BK, NS, PL, PU, TRANS_B>(A, B1, B2, out, pairs, K, N, ldb, ldo,
                                                           d, blockIdx.x, smem);
}

// ---------------------------------------------------------------------------
// Shift GEMM: the local layer (Eq. (1) with jump 1).  For the block's BM
// consecutive rows r:
//   out_r = A_r B1^T + m(r) A_(r+DELTA) B2^T
// DELTA = -1: forward, the previous row, m(r) = 0 at a window's first row.
// DELTA = +1: dX, the next row, m(r) = 0 at a window's last row.
// The A tile is the block's rows plus HALO rows on the partner's side, so the
// partner of LDS row m is LDS row m + DELTA; a lane whose output row is masked
// zeroes its partner fragment, and both products go to one accumulator tile.
// ---------------------------------------------------------------------------
template <int BM, int BN, int WM, int WN, int BK>
struct ShiftCfg {
  static constexpr int NS = 2;                   // pipeline stages
  static constexpr int NT = 64 * WM * WN;
  static constexpr int NW = WM * WN;
  static constexpr int HALO = 8;                 // one 1 KB DMA block of rows at BK = 64
  static constexpr int AR = BM + HALO;           // staged A rows
  static constexpr int TM = BM / (32 * WM);      // 32-row blocks per wave
  static constexpr int TN = BN / (32 * WN);      // 32-column blocks per wave
  static constexpr int A_ELEMS = AR * BK;
  static constexpr int B_ELEMS = BN * BK;
  static constexpr int STAGE = A_ELEMS + 2 * B_ELEMS;
  static constexpr int LDO = BN + 8;
  static constexpr int LDS_ELEMS = (NS * STAGE > BM * LDO) ? NS * STAGE : BM * LDO;
  static constexpr int A_BLOCKS = A_ELEMS * 2 / 1024;
  static constexpr int A_DMA = (A_BLOCKS + NW - 1) / NW;   // per wave; the last may idle
  static constexpr int B_DMA = B_ELEMS * 2 / 1024 / NW;
  static constexpr int O_IT = BM * (BN / 8) / NT;
  static_assert(A_BLOCKS * 1024 == A_ELEMS * 2 && B_DMA * NW * 1024 == B_ELEMS * 2, "");
  static_assert(TM >= 1 && TN >= 1 && O_IT * NT == BM * (BN / 8), "");
};

template <int BM, int BN, int WM, int WN, int BK, int DELTA, bool TRANS_B>
__global__ __launch_bounds__(64 * WM * WN) void shift_bf16_kernel(
    const bf16* __restrict__ A, const bf16* __restrict__ B1, const bf16* __restrict__ B2,
    bf16* __restrict__ out, int rows, int width, int n) {
  using C = ShiftCfg<BM, BN, WM, WN, BK>;
  static_assert(DELTA == -1 || DELTA == 1, "");
  constexpr int RB = BN * 2;
  constexpr int OFF0 = DELTA < 0 ? C::HALO : 0;   // LDS row of the block's first row
  extern __shared__ __attribute__((aligned(1024))) bf16 smem[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WM, wn = wave / WM;
  const int tiles_n = width / BN;
  const int tiles_m = (rows + BM - 1) / BM;
  const int tile = xcd_tile(blockIdx.x, tiles_m * tiles_n);
  const int r0 = (tile / tiles_n) * BM;
  const int n0 = (tile % tiles_n) * BN;

  // DMA sources of this lane at k-slice 0; rows outside the tensor read a
  // valid row whose products are masked or never stored.
  const bf16* a_src[C::A_DMA];
#pragma unroll
  for (int j = 0; j < C::A_DMA; j++) {
    const int b = min(j * C::NW + wave, C::A_BLOCKS - 1);
    const int o = b * 1024 + 16 * lane;
    const int m = o / (2 * BK);
    const int ch = (swz<BK>(m, (o % (2 * BK)) / 16) - m * BK) / 8;
    const int r = min(max(r0 - OFF0 + m, 0), rows - 1);
    a_src[j] = A + (size_t)r * width + ch * 8;
  }
  size_t b_src[C::B_DMA];
#pragma unroll
  for (int j = 0; j < C::B_DMA; j++) {
    const int b = j * C::NW + wave;
    if constexpr (TRANS_B) {
      int kr, col;
      tr_dma_coord<RB>(b, lane, &kr, &col);
      b_src[j] = (size_t)kr * width + n0 + col;
    } else {
      const int o = b * 1024 + 16 * lane;
      const int nr = o / (2 * BK);
      const int ch = (swz<BK>(nr, (o % (2 * BK)) / 16) - nr * BK) / 8;
      b_src[j] = (size_t)(n0 + nr) * width + ch * 8;
    }
  }
  const size_t b_step = TRANS_B ? (size_t)BK * width : BK;
  auto issue = [&](int kt, int stage) {
    bf16* sA = smem + stage * C::STAGE;
    bf16* sB1 = sA + C::A_ELEMS;
    bf16* sB2 = sB1 + C::B_ELEMS;
#pragma unroll
    for (int j = 0; j < C::A_DMA; j++)
      if (j * C::NW + wave < C::A_BLOCKS)   // wave-uniform
        dma16(a_src[j] + kt * BK, sA + (j * C::NW + wave) * 512);
#pragma unroll
    for (int j = 0; j < C::B_DMA; j++) {
      dma16(B1 + b_src[j] + kt * b_step, sB1 + (j * C::NW + wave) * 512);
      dma16(B2 + b_src[j] + kt * b_step, sB2 + (j * C::NW + wave) * 512);
    }
  };

  // partner mask of this lane's output row in each 32-row block
  bool keep[C::TM];
#pragma unroll
  for (int t = 0; t < C::TM; t++) {
    const int pos = (r0 + (wm * C::TM + t) * 32 + (lane & 31)) & (n - 1);
    keep[t] = DELTA < 0 ? pos != 0 : pos != n - 1;
  }

  f32x16 acc[C::TM][C::TN];
#pragma unroll
  for (int t = 0; t < C::TM; t++)
#pragma unroll
    for (int u = 0; u < C::TN; u++)
#pragma unroll
      for (int e = 0; e < 16; e++) acc[t][u][e] = 0.f;

  struct Frags { bf16x8 as[C::TM], ap[C::TM], b1[C::TN], b2[C::TN]; };
  auto load_frags = [&](Frags& f, const bf16* sA, int kk) {
    const bf16* sB1 = sA + C::A_ELEMS;
    const bf16* sB2 = sB1 + C::B_ELEMS;
    const int ch = kk * 2 + (lane >> 5);
#pragma unroll
    for (int t = 0; t < C::TM; t++) {
      const int m = OFF0 + (wm * C::TM + t) * 32 + (lane & 31);
      f.as[t] = *(const bf16x8*)(sA + swz<BK>(m, ch));
      f.ap[t] = *(const bf16x8*)(sA + swz<BK>(m + DELTA, ch));
    }
#pragma unroll
    for (int u = 0; u < C::TN; u++) {
      const int nb = (wn * C::TN + u) * 32;
      if constexpr (TRANS_B) {
        f.b1[u] = tr_frag<RB>(sB1, kk * 16, nb, lane);
        f.b2[u] = tr_frag<RB>(sB2, kk * 16, nb, lane);
      } else {
        f.b1[u] = *(const bf16x8*)(sB1 + swz<BK>(nb + (lane & 31), ch));
        f.b2[u] = *(const bf16x8*)(sB2 + swz<BK>(nb + (lane & 31), ch));
      }
    }
  };
  // transposed products (weights as the MFMA A operand): lane l owns output
  // row l % 32 of each block and 16 of its columns
  auto mma = [&](const Frags& f) {
    const bf16x8 zero = {};
#pragma unroll
    for (int t = 0; t < C::TM; t++)
#pragma unroll
      for (int u = 0; u < C::TN; u++) acc[t][u] = mfma32(f.b1[u], f.as[t], acc[t][u]);
#pragma unroll
    for (int t = 0; t < C::TM; t++) {
      const bf16x8 ap = keep[t] ? f.ap[t] : zero;
#pragma unroll
      for (int u = 0; u < C::TN; u++) acc[t][u] = mfma32(f.b2[u], ap, acc[t][u]);
    }
  };

  constexpr int KK = BK / 16;
  constexpr int NMFMA = 2 * C::TM * C::TN;
  constexpr int NDS = 2 * C::TM + 2 * C::TN * (TRANS_B ? 2 : 1);
  const int nk = width / BK;
  issue(0, 0);
  Frags f[2];
  for (int kt = 0; kt < nk; kt++) {
    wait_dma();
    __syncthreads();  // stage kt visible to all waves; buffer (kt-1) % 2 free
    if (kt + 1 < nk) issue(kt + 1, (kt + 1) & 1);
    const bf16* sA = smem + (kt & 1) * C::STAGE;
    load_frags(f[0], sA, 0);
#pragma unroll
    for (int kk = 0; kk < KK; kk++) {
      if (kk + 1 < KK) {
        load_frags(f[(kk + 1) & 1], sA, kk + 1);
        mma(f[kk & 1]);
        interleave_front<NMFMA, NDS>();
      } else {
        mma(f[kk & 1]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  __syncthreads();  // every wave done with the stage buffers

  bf16* sO = smem;
#pragma unroll
  for (int t = 0; t < C::TM; t++)
#pragma unroll
    for (int u = 0; u < C::TN; u++) {
      const int m = (wm * C::TM + t) * 32 + (lane & 31);
      const int col = (wn * C::TN + u) * 32 + 4 * (lane >> 5);
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const bf16x4 v = {to_bf16(acc[t][u][4 * g]), to_bf16(acc[t][u][4 * g + 1]),
                          to_bf16(acc[t][u][4 * g + 2]), to_bf16(acc[t][u][4 * g + 3])};
        *(bf16x4*)(sO + m * C::LDO + col + 8 * g) = v;
      }
    }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < C::O_IT; j++) {
    const int idx = tid + C::NT * j;
    const int m = idx / (BN / 8), ch = idx % (BN / 8);
    if (r0 + m >= rows) continue;
    store_wt16(out + (size_t)(r0 + m) * width + n0 + ch * 8, *(const u32x4*)(sO + m * C::LDO + ch * 8));
  }
}

// ---------------------------------------------------------------------------
// Weight gradients, split over rows.  Block (tile, slot) computes the BO x BC
// tile of dW_self and dW_off over the row pairs of its slot:
//   dW_self += dY_L^T X_L + dY_U^T X_U
//   dW_off  += dY_U^T X_L            (+ dY_L^T X_U when bidirectional)
// A K-step stages KP pairs = 2*KP rows of dY and X in LDS in their natural
// layout (slots 0..KP-1 the lower rows, KP..2KP-1 their partners); both MFMA
// operands are read transposed, the row (slot) index being the contraction.
// The local layer (LINK_NEAR) uses the same machinery with pairs (r - 1, r):
//   dW_self += dY_U^T X_U,  dW_off += dY_U^T X_L.
//
// A block is two groups of WO x WC waves (two waves per SIMD): the groups walk
// the two halves of the block's row range side by side, each with its own
// two-stage pipeline, and at the end group 1 hands its accumulators to group 0
// through LDS; group 0 adds them (always in that order) and stores the block's
// partial.  One partial per block halves the partial traffic of one block per
// half range, with the same number of waves in flight.
// ---------------------------------------------------------------------------
constexpr int KP = 32;
constexpr int SLOTS = 2 * KP;

// Link of a weight-gradient launch.  Hypercube layers: K runs over row pairs
// (lower row, upper row = lower + 2^d).  Local layer: K runs over rows r, the
// "lower" slot holding row r - 1 (zero at a window's first row) and the "upper"
// slot row r; only the upper slots' dY is used.
constexpr int LINK_CAUSAL = 0, LINK_BIDIR = 1, LINK_NEAR = 2;

// 16 zero bytes in global memory: the DMA source of masked slots.
__device__ __attribute__((aligned(16))) bf16 g_zero16[8];

template <int BO, int BC, int WO, int WC>
struct DwCfg {
  static constexpr int NG = 2;                  // row-range groups per block
  static constexpr int NW = WO * WC;            // waves per group
  static constexpr int NT = 64 * NW * NG;
  static constexpr int TO = BO / (32 * WO);
  static constexpr int TC = BC / (32 * WC);
  static constexpr int G_ELEMS = SLOTS * BO;
  static constexpr int X_ELEMS = SLOTS * BC;
  static constexpr int STAGE = G_ELEMS + X_ELEMS;
  static constexpr int G_DMA = G_ELEMS * 2 / 1024 / NW;
  static constexpr int X_DMA = X_ELEMS * 2 / 1024 / NW;
  static_assert(G_DMA * NW * 1024 == G_ELEMS * 2 && X_DMA * NW * 1024 == X_ELEMS * 2, "");
  static constexpr int ACC = 2 * TO * TC * 16;  // accumulator floats per lane
  static constexpr size_t LDS = (size_t)NG * 2 * STAGE * 2;   // bytes: two stages per group
  static_assert((size_t)NW * ACC * 64 * 4 <= LDS, "hand-over fits in the stage buffers");
};

// One block's work: the BO x BC tile `tile` over the pairs of range `split`
// (two groups of pairs_per_group each), written to out_s / out_o (row stride
// width; added to what they hold when `accumulate`).  `smem_all` is the
// block's dynamic LDS (DwCfg::LDS bytes).
template <int BO, int BC, int WO, int WC, int LINK>
__device__ __forceinline__ void dw_bf16_block(
    const bf16* __restrict__ X, const bf16* __restrict__ dY, float* __restrict__ out_s,
    float* __restrict__ out_o, int accumulate, int pairs, int width, int d, int n,
    int pairs_per_group, int tile, int split, bf16* smem_all) {
  constexpr bool BIDIR = LINK == LINK_BIDIR, NEAR = LINK == LINK_NEAR;
  using C = DwCfg<BO, BC, WO, WC>;
  constexpr int RBG = BO * 2, RBX = BC * 2;

  const int tid = threadIdx.x, lane = tid & 63;
  const int group = (tid >> 6) / C::NW, wave = (tid >> 6) % C::NW;
  bf16* smem = smem_all + group * 2 * C::STAGE;
  const int wo = wave % WO, wc = wave / WO;
  const int tiles_c = width / BC;
  const int o0 = (tile / tiles_c) * BO, c0 = (tile % tiles_c) * BC;
  const int s = NEAR ? 0 : 1 << d;
  const int pbeg = (2 * split + group) * pairs_per_group;
  const int pend = min(pairs, pbeg + pairs_per_group);   // may be <= pbeg: all zero-filled

  // Per-lane (slot, column) of each DMA block.
  int g_slot[C::G_DMA], g_col[C::G_DMA], x_slot[C::X_DMA], x_col[C::X_DMA];
#pragma unroll
  for (int j = 0; j < C::G_DMA; j++) tr_dma_coord<RBG>(j * C::NW + wave, lane, &g_slot[j], &g_col[j]);
#pragma unroll
  for (int j = 0; j < C::X_DMA; j++) tr_dma_coord<RBX>(j * C::NW + wave, lane, &x_slot[j], &x_col[j]);

  auto row_of = [&](int p0, int slot) {
    if constexpr (NEAR) return p0 + (slot % KP) - (slot < KP ? 1 : 0);
    return lower_row(p0 + (slot % KP), d) + (slot >= KP ? s : 0);
  };
  // Local layer: a lower slot is zero when its row r = p0 + slot starts a
  // window (no predecessor); dY's lower slots are never read.
  auto x_zero = [&](int p0, int slot) {
    return NEAR && slot < KP && ((p0 + slot) & (n - 1)) == 0;
  };
  auto g_zero = [&](int slot) { return NEAR && slot < KP; };
  // Whole K-step: every slot valid, straight DMA.
  auto issue = [&](int p0, int stage) {
    bf16* sG = smem + stage * C::STAGE;
    bf16* sX = sG + C::G_ELEMS;
#pragma unroll
    for (int j = 0; j < C::G_DMA; j++)
      dma16(g_zero(g_slot[j]) ? g_zero16 : dY + (size_t)row_of(p0, g_slot[j]) * width + o0 + g_col[j],
            sG + (j * C::NW + wave) * 512);
#pragma unroll
    for (int j = 0; j < C::X_DMA; j++)
      dma16(x_zero(p0, x_slot[j]) ? g_zero16 : X + (size_t)row_of(p0, x_slot[j]) * width + c0 + x_col[j],
            sX + (j * C::NW + wave) * 512);
  };
  // Ragged last K-step: slots past the end of the split are zero-filled.
  auto fill_tail = [&](int p0, int stage) {
    bf16* sG = smem + stage * C::STAGE;
    bf16* sX = sG + C::G_ELEMS;
#pragma unroll
    for (int j = 0; j < C::G_DMA; j++) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (p0 + (g_slot[j] % KP) < pend && !g_zero(g_slot[j]))
        v = *(const u32x4*)(dY + (size_t)row_of(p0, g_slot[j]) * width + o0 + g_col[j]);
      *(u32x4*)(sG + (j * C::NW + wave) * 512 + lane * 8) = v;
    }
#pragma unroll
    for (int j = 0; j < C::X_DMA; j++) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (p0 + (x_slot[j] % KP) < pend && !x_zero(p0, x_slot[j]))
        v = *(const u32x4*)(X + (size_t)row_of(p0, x_slot[j]) * width + c0 + x_col[j]);
      *(u32x4*)(sX + (j * C::NW + wave) * 512 + lane * 8) = v;
    }
  };
  auto stage_in = [&](int p0, int stage) {
    if (p0 + KP <= pend) issue(p0, stage);
    else fill_tail(p0, stage);
  };

  f32x16 accS[C::TO][C::TC], accO[C::TO][C::TC];
#pragma unroll
  for (int a = 0; a < C::TO; a++)
#pragma unroll
    for (int b = 0; b < C::TC; b++)
#pragma unroll
      for (int e = 0; e < 16; e++) { accS[a][b][e] = 0.f; accO[a][b][e] = 0.f; }

  struct Frags { bf16x8 gL[C::TO], gU[C::TO], xL[C::TC], xU[C::TC]; };
  auto load_frags = [&](Frags& f, const bf16* sG, int kk) {
    const bf16* sX = sG + C::G_ELEMS;
#pragma unroll
    for (int a = 0; a < C::TO; a++) {
      const int ob = (wo * C::TO + a) * 32;
      if constexpr (!NEAR) f.gL[a] = tr_frag<RBG>(sG, kk * 16, ob, lane);
      f.gU[a] = tr_frag<RBG>(sG, KP + kk * 16, ob, lane);
    }
#pragma unroll
    for (int b = 0; b < C::TC; b++) {
      const int cb = (wc * C::TC + b) * 32;
      f.xL[b] = tr_frag<RBX>(sX, kk * 16, cb, lane);
      f.xU[b] = tr_frag<RBX>(sX, KP + kk * 16, cb, lane);
    }
  };
  auto mma = [&](const Frags& f) {
    if constexpr (NEAR) {
#pragma unroll
      for (int a = 0; a < C::TO; a++)
#pragma unroll
        for (int b = 0; b < C::TC; b++) {
          accS[a][b] = mfma32(f.gU[a], f.xU[b], accS[a][b]);
          accO[a][b] = mfma32(f.gU[a], f.xL[b], accO[a][b]);
        }
      return;
    }
#pragma unroll
    for (int a = 0; a < C::TO; a++)
#pragma unroll
      for (int b = 0; b < C::TC; b++) {
        accS[a][b] = mfma32(f.gL[a], f.xL[b], accS[a][b]);
        accO[a][b] = mfma32(f.gU[a], f.xL[b], accO[a][b]);
      }
#pragma unroll
    for (int a = 0; a < C::TO; a++)
#pragma unroll
      for (int b = 0; b < C::TC; b++) {
        accS[a][b] = mfma32(f.gU[a], f.xU[b], accS[a][b]);
        if (BIDIR) accO[a][b] = mfma32(f.gL[a], f.xU[b], accO[a][b]);
      }
  };

  constexpr int NMFMA = C::TO * C::TC * (NEAR ? 2 : 3 + (BIDIR ? 1 : 0));
  constexpr int NDS = 2 * ((NEAR ? 1 : 2) * C::TO + 2 * C::TC);   // two tr reads per fragment
  // the same step count in both groups (their barriers are shared); steps past
  // a group's range are zero-filled
  const int nsteps = pairs_per_group / KP;
  if (nsteps > 0) stage_in(pbeg, 0);
  wait_dma();
  __syncthreads();
  Frags f0, f1;
  if (nsteps > 0) load_frags(f0, smem, 0);
  for (int it = 0; it < nsteps; it++) {
    const bf16* sG = smem + (it & 1) * C::STAGE;
    if (it + 1 < nsteps) stage_in(pbeg + (it + 1) * KP, (it + 1) & 1);
    load_frags(f1, sG, 1);
    mma(f0);
    interleave_mfma_ds<NMFMA, NDS>();
    mma(f1);
    wait_dma();
    __syncthreads();
    if (it + 1 < nsteps) load_frags(f0, smem + ((it + 1) & 1) * C::STAGE, 0);
  }

  // group 1 -> LDS -> group 0, which adds in a fixed order and stores
  float* hand = (float*)smem_all + (size_t)wave * C::ACC * 64;
  if (group == 1) {
    int i = 0;
#pragma unroll
    for (int a = 0; a < C::TO; a++)
#pragma unroll
      for (int b = 0; b < C::TC; b++)
#pragma unroll
        for (int e = 0; e < 16; e++) {
          hand[(i++) * 64 + lane] = accS[a][b][e];
          hand[(i++) * 64 + lane] = accO[a][b][e];
        }
  }
  __syncthreads();
  if (group == 1) return;
  {
    int i = 0;
#pragma unroll
    for (int a = 0; a < C::TO; a++)
#pragma unroll
      for (int b = 0; b < C::TC; b++)
#pragma unroll
        for (int e = 0; e < 16; e++) {
          accS[a][b][e] += hand[(i++) * 64 + lane];
          accO[a][b][e] += hand[(i++) * 64 + lane];
        }
  }

#pragma unroll
  for (int a = 0; a < C::TO; a++)
#pragma unroll
    for (int b = 0; b < C::TC; b++)
#pragma unroll
      for (int e = 0; e < 16; e++) {
        const int o = o0 + (wo * C::TO + a) * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        const int c = c0 + (wc * C::TC + b) * 32 + (lane & 31);
        float* ps = out_s + (size_t)o * width + c;
        float* po = out_o + (size_t)o * width + c;
        store_wt4(ps, accumulate ? *ps + accS[a][b][e] : accS[a][b][e]);
        store_wt4(po, accumulate ? *po + accO[a][b][e] : accO[a][b][e]);
      }
}

// Split-K launch: block -> (split, tile), split-major through the XCD deal, so
// every tile of one split (they all read the same rows of X and dY) runs on
// one XCD and shares its L2.  Split `sp` writes partial[sp] = [2][width][width].
template <int BO, int BC, int WO, int WC, int LINK>
__global__ __launch_bounds__(128 * WO * WC) void dw_bf16_kernel(
    const bf16* __restrict__ X, const bf16* __restrict__ dY, float* __restrict__ partial,
    int pairs, int width, int d, int n, int pairs_per_group) {
  extern __shared__ __attribute__((aligned(1024))) bf16 smem_all[];
  const int tiles = (width / BO) * (width / BC);
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const size_t ww = (size_t)width * width;
  float* out = partial + (size_t)(lin / tiles) * 2 * ww;
  dw_bf16_block<BO, BC, WO, WC, LINK>(X, dY, out, out + ww, 0, pairs, width, d, n,
                                      pairs_per_group, lin % tiles, lin / tiles, smem_all);
}

// Weight gradients of every layer of a stack in one launch: block ->
// (layer, split, tile), in that order through the XCD deal, so the tiles of
// one layer and split (which read the same rows) share an L2.  With one split
// each block owns its tiles over all row pairs and writes the layer's dW_self
// and dW_off directly; otherwise split sp of layer l writes the partial
// [l][sp][2][width][width] for dw_batch_reduce_kernel.
template <int BO, int BC, int WO, int WC>
__global__ __launch_bounds__(128 * WO * WC) void dw_batch_kernel(DwBatchArgs a) {
  extern __shared__ __attribute__((aligned(1024))) bf16 smem_all[];
  const int tiles = (a.width / BO) * (a.width / BC);
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int layer = lin / (a.splits * tiles);
  const int split = (lin / tiles) % a.splits;
  const int tile = lin % tiles;
  const int d = a.dim[layer];
  const int units = d < 0 ? a.rows : a.rows / 2;   // rows (local layer) or row pairs
  const int ppg = ((units + KP - 1) / KP + 2 * a.splits - 1) / (2 * a.splits) * KP;
  const size_t ww = (size_t)a.width * a.width;
  float *out_s, *out_o;
  int acc = a.accumulate;
  if (a.splits == 1) {
    out_s = a.dws[layer];
    out_o = a.dwo[layer];
  } else {
    out_s = a.partial + ((size_t)layer * a.splits + split) * 2 * ww;
    out_o = out_s + ww;
    acc = 0;
  }
  if (d < 0)
    dw_bf16_block<BO, BC, WO, WC, LINK_NEAR>(a.x[layer], a.dy[layer], out_s, out_o, acc, units,
                                             a.width, d, a.n, ppg, tile, split, smem_all);
  else if (a.bidir)
    dw_bf16_block<BO, BC, WO, WC, LINK_BIDIR>(a.x[layer], a.dy[layer], out_s, out_o, acc, units,
                                              a.width, d, a.n, ppg, tile, split, smem_all);
  else
    dw_bf16_block<BO, BC, WO, WC, LINK_CAUSAL>(a.x[layer], a.dy[layer], out_s, out_o, acc, units,
                                               a.width, d, a.n, ppg, tile, split, smem_all);
}

// dW[l] (+)= sum over splits of partial[l][sp], in split order: block (l, j)
// strides over the float4 outputs of layer l's two matrices.
__global__ __launch_bounds__(256) void dw_batch_reduce_kernel(DwBatchArgs a, int blocks_per_layer) {
  const int l = blockIdx.x / blocks_per_layer, j0 = blockIdx.x % blocks_per_layer;
  const size_t ww = (size_t)a.width * a.width, n4 = ww / 4;
  const float* part = a.partial + (size_t)l * a.splits * 2 * ww;
  for (size_t i = j0 * (size_t)256 + threadIdx.x; i < 2 * n4; i += (size_t)blocks_per_layer * 256) {
    const int m = i >= n4;
    const size_t j = i - m * n4;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < a.splits; sp++) acc += ((const f32x4*)(part + ((size_t)sp * 2 + m) * ww))[j];
    f32x4* dst = (f32x4*)(m ? a.dwo[l] : a.dws[l]) + j;
    if (a.accumulate) acc += *dst;
    store_wt16(dst, __builtin_bit_cast(u32x4, acc));
  }
}

// dW (+)= sum over splits, in split order; `block` of `nblocks`, `nthreads`
// threads each, striding over the float4 outputs of both matrices.
__device__ __forceinline__ void dw_reduce_block(const float* __restrict__ partial,
                                                float* __restrict__ dws, float* __restrict__ dwo,
                                                int splits, size_t ww, int accumulate, int block,
                                                int nblocks, int nthreads) {
  const size_t n4 = ww / 4;
  for (size_t i = block * (size_t)nthreads + threadIdx.x; i < 2 * n4;
       i += (size_t)nblocks * nthreads) {
    const int m = i >= n4;
    const size_t j = i - m * n4;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < splits; sp++)
      acc += ((const f32x4*)(partial + ((size_t)sp * 2 + m) * ww))[j];
    f32x4* dst = (f32x4*)(m ? dwo : dws) + j;
    if (accumulate) acc += *dst;
    store_wt16(dst, __builtin_bit_cast(u32x4, acc));
  }
}

__global__ __launch_bounds__(256) void dw_reduce_kernel(const float* __restrict__ partial,
                                                        float* __restrict__ dws,
                                                        float* __restrict__ dwo, int splits,
                                                        size_t ww, int accumulate) {
  dw_reduce_block(partial, dws, dwo, splits, ww, accumulate, blockIdx.x, gridDim.x, blockDim.x);
}

// ---- launch configurations ----
constexpr int MIX_BMP = 128;          // 256 rows per block
constexpr int MIX_BK = 64;            // contraction slice per pipeline stage
constexpr int MIX_NS = 2;             // pipeline stages in LDS
constexpr int DW_BO = 128, DW_BC = 128;
constexpr int DW_TARGET_BLOCKS = 256;  // split-K blocks aimed for (8 waves each)
template <int BMP, int BN, int WM, int WN, int BK, int NS, bool TRANS_B>
hipError_t mix_launch(const bf16* A, const bf16* B1, const bf16* B2, bf16* out, int pairs,
                      int width, int d, int partner_lower, int partner_upper, hipStream_t st) {
  using C = MixCfg<BMP, BN, WM, WN, BK, NS>;
  const int blocks = ((pairs + BMP - 1) / BMP) * (width / BN);
  const size_t lds = (size_t)C::LDS_ELEMS * sizeof(bf16);
#define HCMIX_MIX(PL, PU)                                                                   \
  {                                                                                         \
    auto k = mix_bf16_kernel<BMP, BN, WM, WN, BK, NS, PL, PU, TRANS_B>;                     \
    static std::atomic<unsigned long long> lds_set{0};                                      \
    const hipError_t attr = lds_limit_once(lds_set, (const void*)k, (int)lds);             \
    if (attr != hipSuccess) return attr;                                                    \
    k<<<blocks, C::NT, lds, st>>>(A, B1, B2, out, pairs, width, width, width, width, d);     \
  }
  if (partner_lower && partner_upper) HCMIX_MIX(true, true)
  else if (partner_upper) HCMIX_MIX(false, true)
  else HCMIX_MIX(true, false)
#undef HCMIX_MIX
  return hipGetLastError();
}

// The plain product instance (no partner terms): out [rows][N] (row stride
// ldo) = A [rows][K] B^T with B [N][ldb] k-contiguous, or A B with B [K][ldb]
// (TRANS_B).  Rows in consecutive pairs (dimension 0).
template <int BN, int WM, int WN, bool TRANS_B>
hipError_t gemm_launch(const bf16* A, const bf16* B, bf16* out, int rows, int K, int N, int ldb,
                       int ldo, hipStream_t st) {
  using C = MixCfg<MIX_BMP, BN, WM, WN, MIX_BK, MIX_NS>;
  const int pairs = rows / 2;
  const int blocks = ((pairs + MIX_BMP - 1) / MIX_BMP) * (N / BN);
  const size_t lds = (size_t)C::LDS_ELEMS * sizeof(bf16);
  auto k = mix_bf16_kernel<MIX_BMP, BN, WM, WN, MIX_BK, MIX_NS, false, false, TRANS_B>;
  static std::atomic<unsigned long long> lds_set{0};
  const hipError_t attr = lds_limit_once(lds_set, (const void*)k, (int)lds);
  if (attr != hipSuccess) return attr;
  k<<<blocks, C::NT, lds, st>>>(A, B, B, out, pairs, K, N, ldb, ldo, 0);
  return hipGetLastError();
}

template <int BN, int WM, int WN, int DELTA, bool TRANS_B>
hipError_t shift_launch(const bf16* A, const bf16* B1, const bf16* B2, bf16* out, int rows,
                        int width, int n, hipStream_t st) {
  constexpr int BM = 256;
  using C = ShiftCfg<BM, BN, WM, WN, MIX_BK>;
  const int blocks = ((rows + BM - 1) / BM) * (width / BN);
  const size_t lds = (size_t)C::LDS_ELEMS * sizeof(bf16);
  auto k = shift_bf16_kernel<BM, BN, WM, WN, MIX_BK, DELTA, TRANS_B>;
  static std::atomic<unsigned long long> lds_set{0};
  const hipError_t attr = lds_limit_once(lds_set, (const void*)k, (int)lds);
  if (attr != hipSuccess) return attr;
  k<<<blocks, C::NT, lds, st>>>(A, B1, B2, out, rows, width, n);
  return hipGetLastError();
}

template <int DELTA, bool TRANS_B>
hipError_t shift_dispatch(const bf16* A, const bf16* B1, const bf16* B2, bf16* out, int rows,
                          int width, int n, hipStream_t st) {
  if (width % 128 == 0)
    return shift_launch<128, 2, 2, DELTA, TRANS_B>(A, B1, B2, out, rows, width, n, st);
  return shift_launch<64, 4, 1, DELTA, TRANS_B>(A, B1, B2, out, rows, width, n, st);
}

template <bool TRANS_B>
hipError_t mix_dispatch(const bf16* A, const bf16* B1, const bf16* B2, bf16* out, int rows,
                        int width, int d, int partner_lower, int partner_upper, hipStream_t st) {
  const int pairs = rows / 2;
  // Wide layers (1024 and up): 256-column tiles, 96 flop -> 131 flop per byte
  // moved into the CU, in 32-wide K-steps with three stages (the LDS holds
  // 3 x 48 KB).  Measured at 32768 x 1024: 126-130 -> 119-124 us per forward
  // launch.  Weights read transposed keep the 128-column tile.
  if constexpr (!TRANS_B) {
    if (width % 256 == 0 && width >= 1024)
      return mix_launch<MIX_BMP, 256, 2, 4, 32, 3, TRANS_B>(A, B1, B2, out, pairs, width, d,
                                                            partner_lower, partner_upper, st);
  }
  // Two waves per SIMD (8 per block, each 64 pairs x 32 columns): one wave's
  // LDS reads and barrier waits hide under the other's MFMAs.  Measured at
  // 16384 x 512: dX 18.1 -> 16.8 us, forward unchanged within noise.
  if (width % 128 == 0)
    return mix_launch<MIX_BMP, 128, 2, 4, MIX_BK, MIX_NS, TRANS_B>(
        A, B1, B2, out, pairs, width, d, partner_lower, partner_upper, st);
  return mix_launch<MIX_BMP, 64, 4, 1, MIX_BK, MIX_NS, TRANS_B>(
      A, B1, B2, out, pairs, width, d, partner_lower, partner_upper, st);
}

// Batched bf16 transpose: dst[m] = src[m]^T for up to kTransposeBatch square
// width x width matrices, one 64 x 64 tile per block through a padded LDS tile.
__global__ __launch_bounds__(256) void transpose_bf16_kernel(TransposeArgs a) {
  __shared__ bf16 t[64][64 + 8];
  const int tiles = a.width / 64;
  const int tr = blockIdx.x / tiles, tc = blockIdx.x % tiles;
  const bf16* src = a.src[blockIdx.y];
  bf16* dst = a.dst[blockIdx.y];
#pragma unroll
  for (int i = threadIdx.x; i < 512; i += 256) {
    const int r = i / 8, c = (i % 8) * 8;
    const bf16x8 v = *(const bf16x8*)(src + (size_t)(tr * 64 + r) * a.width + tc * 64 + c);
#pragma unroll
    for (int j = 0; j < 8; j++) t[r][c + j] = v[j];
  }
  __syncthreads();
#pragma unroll
  for (int i = threadIdx.x; i < 512; i += 256) {
    const int r = i / 8, c = (i % 8) * 8;
    bf16x8 v;
#pragma unroll
    for (int j = 0; j < 8; j++) v[j] = t[c + j][r];
    store_wt16(dst + (size_t)(tc * 64 + r) * a.width + tr * 64 + c, __builtin_bit_cast(u32x4, v));
  }
}

// Split-K plan: about one block per CU, each block's row range two groups of
// whole K-steps.  Returns the number of partial slots (blocks per tile);
// *ppg gets the pairs per group.
int dw_plan(int pairs, int width, int* ppg, int target_blocks = DW_TARGET_BLOCKS) {
  const int bo = width % DW_BO == 0 ? DW_BO : 64;
  const int tiles = (width / bo) * (width / bo);
  const int ksteps = (pairs + KP - 1) / KP;
  int slots = (target_blocks + tiles - 1) / tiles;
  if (slots > (ksteps + 1) / 2) slots = (ksteps + 1) / 2;
  if (slots < 1) slots = 1;
  *ppg = ((ksteps + 2 * slots - 1) / (2 * slots)) * KP;
  return (pairs + 2 * *ppg - 1) / (2 * *ppg);
}

template <int BO, int BC, int WO, int WC>
hipError_t dw_launch(const bf16* X, const bf16* dY, float* partial, int pairs, int width, int d,
                     int n, int link, int splits, int pps, hipStream_t st) {
  using C = DwCfg<BO, BC, WO, WC>;
  const int blocks = (width / BO) * (width / BC) * splits;
  const size_t lds = C::LDS;
#define HCMIX_DW(LINK)                                                                      \
  {                                                                                         \
    auto k = dw_bf16_kernel<BO, BC, WO, WC, LINK>;                                          \
    static std::atomic<unsigned long long> lds_set{0};                                      \
    const hipError_t attr = lds_limit_once(lds_set, (const void*)k, (int)lds);             \
    if (attr != hipSuccess) return attr;                                                    \
    k<<<blocks, C::NT, lds, st>>>(X, dY, partial, pairs, width, d, n, pps);                 \
  }
  if (link == LINK_NEAR) HCMIX_DW(LINK_NEAR)
  else if (link == LINK_BIDIR) HCMIX_DW(LINK_BIDIR)
  else HCMIX_DW(LINK_CAUSAL)
#undef HCMIX_DW
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16(const bf16* A, const bf16* B, bf16* out, int rows, int K, int N,
                            int ldb, int ldo, bool transpose_b, hipStream_t st) {
  if (N % 128 == 0)
    return transpose_b ? gemm_launch<128, 2, 4, true>(A, B, out, rows, K, N, ldb, ldo, st)
                       : gemm_launch<128, 2, 4, false>(A, B, out, rows, K, N, ldb, ldo, st);
  return transpose_b ? gemm_launch<64, 4, 1, true>(A, B, out, rows, K, N, ldb, ldo, st)
                     : gemm_launch<64, 4, 1, false>(A, B, out, rows, K, N, ldb, ldo, st);
}

hipError_t launch_mix_bf16(const bf16* A, const bf16* B1, const bf16* B2, bf16* out, int rows,
                           int width, int d, int partner_lower, int partner_upper,
                           bool transpose_b, hipStream_t st) {
  if (transpose_b)
    return mix_dispatch<true>(A, B1, B2, out, rows, width, d, partner_lower, partner_upper, st);
  return mix_dispatch<false>(A, B1, B2, out, rows, width, d, partner_lower, partner_upper, st);
}

hipError_t launch_transpose_bf16(const TransposeArgs& a, int count, hipStream_t st) {
  const int tiles = a.width / 64;
  transpose_bf16_kernel<<<dim3(tiles * tiles, count), 256, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_shift_bf16(const bf16* A, const bf16* B1, const bf16* B2, bf16* out, int rows,
                             int width, int n, int delta, bool transpose_b, hipStream_t st) {
  if (delta < 0)
    return transpose_b ? shift_dispatch<-1, true>(A, B1, B2, out, rows, width, n, st)
                       : shift_dispatch<-1, false>(A, B1, B2, out, rows, width, n, st);
  return transpose_b ? shift_dispatch<1, true>(A, B1, B2, out, rows, width, n, st)
                     : shift_dispatch<1, false>(A, B1, B2, out, rows, width, n, st);
}

hipError_t launch_dw_reduce(const DwReduce& r, int width, hipStream_t st) {
  const size_t ww = (size_t)width * width;
  int blocks = (int)((2 * ww / 4 + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  dw_reduce_kernel<<<blocks, 256, 0, st>>>(r.partial, r.dws, r.dwo, r.splits, ww, r.accumulate);
  return hipGetLastError();
}

int dw_bf16_splits(int rows, int width) {
  // the partial slots of either kind of layer (pairs for hypercube layers,
  // rows for the local layer), so one workspace size serves both
  int ppg;
  const int a = dw_plan(rows / 2, width, &ppg);
  const int b = dw_plan(rows, width, &ppg);
  return a > b ? a : b;
}

hipError_t launch_dw_bf16(const bf16* X, const bf16* dY, float* partial, float* dws, float* dwo,
                          int rows, int width, int d, int n, int bidir, int accumulate,
                          hipStream_t st) {
  const bool near = d < 0;
  const int units = near ? rows : rows / 2;
  const int link = near ? LINK_NEAR : bidir ? LINK_BIDIR : LINK_CAUSAL;
  int ppg;
  const int splits = dw_plan(units, width, &ppg);
  hipError_t e;
  if (width % DW_BO == 0)
    e = dw_launch<DW_BO, DW_BC, 2, 2>(X, dY, partial, units, width, d, n, link, splits, ppg, st);
  else
    e = dw_launch<64, 64, 2, 2>(X, dY, partial, units, width, d, n, link, splits, ppg, st);
  if (e != hipSuccess) return e;
  return launch_dw_reduce(DwReduce{partial, dws, dwo, splits, accumulate}, width, st);
}

int dw_batch_splits(int rows, int width, int num_layers) {
  const int tiles = (width / DW_BO) * (width / DW_BC);
  const int per_split = num_layers * tiles;
  int splits = (DW_TARGET_BLOCKS + per_split - 1) / per_split;
  // at least two K-steps per group: rows / 2 pairs over 2 * splits groups
  const int max_splits = (rows / 2) / (4 * KP);
  if (splits > max_splits) splits = max_splits;
  return splits < 1 ? 1 : splits;
}

hipError_t launch_dw_batch_bf16(const DwBatchArgs& a, hipStream_t st) {
  using C = DwCfg<DW_BO, DW_BC, 2, 2>;
  const int tiles = (a.width / DW_BO) * (a.width / DW_BC);
  const int blocks = a.num_layers * a.splits * tiles;
  auto k = dw_batch_kernel<DW_BO, DW_BC, 2, 2>;
  static std::atomic<unsigned long long> lds_set{0};
  const hipError_t attr = lds_limit_once(lds_set, (const void*)k, (int)C::LDS);
  if (attr != hipSuccess) return attr;
  k<<<blocks, C::NT, C::LDS, st>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  int per_layer = (int)((2 * (size_t)a.width * a.width / 4 + 255) / 256);
  if (per_layer * a.num_layers > 2048) per_layer = (2048 + a.num_layers - 1) / a.num_layers;
  dw_batch_reduce_kernel<<<per_layer * a.num_layers, 256, 0, st>>>(a, per_layer);
  return hipGetLastError();
}

}  // namespace hcmix
