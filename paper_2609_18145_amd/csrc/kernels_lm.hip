// Token embedding, output head and cross-entropy of the language-model
// workloads (bf16 activations and weights, fp32 accumulation).
//
//   embedding:  x[r] = table[tokens[r]];  dtable[v] = sum over r with tokens[r] == v of dx[r]
//   head + CE:  logits[r] = W x[r] + bias, loss[r] = lse(logits[r]) - logits[r][target[r]],
//               dlogits[r] = scale (softmax(logits[r]) - onehot(target[r]))
//
// The head computes logits^T = W x^T so that a lane owns one row and 16 of its
// vocabulary entries per 32 x 32 tile: the row's whole softmax is in-lane plus
// one exchange with lane ^ 32.
#include "hcmix_internal.h"
#include "device_common.h"

namespace hcmix {

namespace {

constexpr int LM_THREADS = 256;

// ---------------------------------------------------------------------------
// Embedding forward: one thread per 16-byte piece of an output row; a token
// outside [0, vocab) gives a zero row.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(LM_THREADS) void embed_fwd_kernel(
    const bf16* __restrict__ table, const int* __restrict__ tokens, bf16* __restrict__ x,
    int rows, int width, int vocab) {
  const int pieces = width / 8;
  const size_t i = (size_t)blockIdx.x * LM_THREADS + threadIdx.x;
  if (i >= (size_t)rows * pieces) return;
  const int r = (int)(i / pieces), p = (int)(i % pieces);
  const int t = tokens[r];
  u32x4 v = {0u, 0u, 0u, 0u};
  if (t >= 0 && t < vocab) v = *(const u32x4*)(table + (size_t)t * width + 8 * p);
  *(u32x4*)(x + (size_t)r * width + 8 * p) = v;
}

// ---------------------------------------------------------------------------
// Embedding backward, fixed summation order.  Block (v, c) sums, for vocabulary
// entry v, the rows of chunk c (emb_chunks(rows) chunks of consecutive rows,
// at most EMB_MAX_CHUNK each) whose token is v.  Each of the four waves lists
// the matching rows of its quarter of the chunk, in row order, with all its
// token loads in flight at once; the four lists read back to back are the
// chunk's matches in row order.  Wave k then adds matches k, k + 4, ... in
// that order (8 columns per lane, 64 lanes: 512 columns per pass), and the
// four wave sums are added in wave order into partial[c][v].
// A second kernel adds the chunks in chunk order.
// ---------------------------------------------------------------------------
constexpr int EMB_MIN_CHUNKS = 32;    // spreads a frequent token's rows over blocks
constexpr int EMB_MAX_CHUNK = 4096;   // rows per chunk held in LDS as a match list
constexpr int EMB_SCAN_LOADS = 4;     // token loads in flight per lane while listing
int emb_chunks(int rows) {
  const int c = (rows + EMB_MAX_CHUNK - 1) / EMB_MAX_CHUNK;
  return c > EMB_MIN_CHUNKS ? c : EMB_MIN_CHUNKS;
}

__global__ __launch_bounds__(LM_THREADS) void embed_bwd_partial_kernel(
    const int* __restrict__ tokens, const bf16* __restrict__ dx, float* __restrict__ partial,
    int rows, int width, int vocab, int chunk) {
  __shared__ int list[EMB_MAX_CHUNK];
  __shared__ int count[4];
  __shared__ float red[4][512];
  const int v = blockIdx.x % vocab, c = blockIdx.x / vocab;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = c * chunk, r1 = min(rows, r0 + chunk);
  // wave w lists rows [q0, q1) into list[w * span ...]
  const int span = (chunk + 3) / 4;
  const int q0 = min(r1, r0 + wave * span), q1 = min(r1, q0 + span);
  {
    int* wl = list + wave * span;
    int n = 0;
    for (int base = q0; base < q1; base += 64 * EMB_SCAN_LOADS) {
      int tk[EMB_SCAN_LOADS];
#pragma unroll
      for (int u = 0; u < EMB_SCAN_LOADS; u++) {
        const int r = base + 64 * u + lane;
        tk[u] = r < q1 ? tokens[r] : -1;
      }
#pragma unroll
      for (int u = 0; u < EMB_SCAN_LOADS; u++) {
        const bool hit = tk[u] == v;       // v >= 0, so rows past q1 never hit
        const unsigned long long m = __ballot(hit);
        if (hit) wl[n + __popcll(m & ((1ull << lane) - 1))] = base + 64 * u + lane;
        n += __popcll(m);
      }
    }
    if (lane == 0) count[wave] = n;
  }
  __syncthreads();
  const int o1 = count[0], o2 = o1 + count[1], o3 = o2 + count[2], n = o3 + count[3];
  // match k of the chunk, in row order
  auto match = [&](int k) {
    const int w = (k >= o1) + (k >= o2) + (k >= o3);
    const int o = w == 0 ? 0 : w == 1 ? o1 : w == 2 ? o2 : o3;
    return list[w * span + k - o];
  };
  float* out = partial + ((size_t)c * vocab + v) * width;
  for (int c0 = 0; c0 < width; c0 += 512) {
    const int col = c0 + 8 * lane;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (col < width) {
      // eight rows in flight per step (a frequent token has hundreds per chunk),
      // added in row order
      int k = wave;
      for (; k + 28 < n; k += 32) {
        bf16x8 g[8];
#pragma unroll
        for (int u = 0; u < 8; u++) g[u] = *(const bf16x8*)(dx + (size_t)match(k + 4 * u) * width + col);
#pragma unroll
        for (int u = 0; u < 8; u++)
#pragma unroll
          for (int e = 0; e < 8; e++) acc[e] += (float)g[u][e];
      }
      for (; k < n; k += 4) {
        const bf16x8 g = *(const bf16x8*)(dx + (size_t)match(k) * width + col);
#pragma unroll
        for (int e = 0; e < 8; e++) acc[e] += (float)g[e];
      }
    }
#pragma unroll
    for (int e = 0; e < 8; e++) red[wave][8 * lane + e] = acc[e];
    __syncthreads();
    for (int j = threadIdx.x; j < 512 && c0 + j < width; j += LM_THREADS)
      out[c0 + j] = ((red[0][j] + red[1][j]) + red[2][j]) + red[3][j];
    __syncthreads();
  }
}

// Four consecutive entries per thread (elems is a multiple of 4: width % 64 ==
// 0), eight chunks' loads in flight; each entry still adds the chunks in
// order.  dtable is only 4-byte aligned, so it is written entry by entry.
__global__ __launch_bounds__(LM_THREADS) void embed_bwd_reduce_kernel(
    const float* __restrict__ partial, float* __restrict__ dtable, size_t elems, int chunks,
    int accumulate) {
  const size_t i4 = (size_t)blockIdx.x * LM_THREADS + threadIdx.x;
  if (i4 * 4 >= elems) return;
  const f32x4* p = (const f32x4*)partial + i4;
  const size_t cs = elems / 4;
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
  int c = 0;
  for (; c + 8 <= chunks; c += 8) {
    f32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; u++) v[u] = p[(size_t)(c + u) * cs];
#pragma unroll
    for (int u = 0; u < 8; u++) s += v[u];
  }
  for (; c < chunks; c++) s += p[(size_t)c * cs];
  float* d = dtable + i4 * 4;
#pragma unroll
  for (int e = 0; e < 4; e++) d[e] = accumulate ? d[e] + s[e] : s[e];
}

// ---------------------------------------------------------------------------
// Head + cross-entropy.  Block: 64 rows, four waves; wave (g, h) = (wave % 2,
// wave / 2) computes logits^T for rows 32 g .. 32 g + 31 of the block and the
// vocabulary tiles of half h (tiles 0 .. TA-1 or TA .. NT-1, TA = ceil(NT/2)).
// The weights and the block's x rows pass through LDS in 64-column slices,
// three stages filled by LDS DMA two slices ahead, each block starting at its
// own slice.  Register e of tile t holds entry 32 t + 8 (e / 4) + 4 (lane / 32)
// + e % 4 of row lane % 32, so a row's softmax is in-lane, one exchange with
// lane ^ 32 and one exchange with the other half's wave through LDS.
// With `dbp` the block also writes the column sums of its rows' dlogits (fp32,
// rows in order) to dbp[block][V], which head_db_reduce_kernel adds up.
// ---------------------------------------------------------------------------
constexpr int HEAD_ROWS = 64;

template <int NT>
struct HeadCfg {
  static constexpr int V = NT * 32;
  static constexpr int TA = (NT + 1) / 2;         // tiles of the first half
  static constexpr int SLICE = V * 64;            // bf16 elements per weight slice
  static constexpr int XSLICE = HEAD_ROWS * 64;   // bf16 elements per x slice
  static constexpr int STAGE = SLICE + XSLICE;
  static constexpr int DMA = V / 32 + 2;          // 1 KB DMA blocks per wave per stage
  static constexpr int DB_LD = V + 4;             // fp32 row stride of the dlogits staging
  static constexpr size_t LDS = (size_t)3 * STAGE * sizeof(bf16);
  static_assert((size_t)HEAD_ROWS * DB_LD * sizeof(float) <= LDS, "dlogits staging fits");
};

template <int NT>
__global__ __launch_bounds__(LM_THREADS) void head_ce_kernel(
    const bf16* __restrict__ x, const bf16* __restrict__ w, const float* __restrict__ bias,
    const int* __restrict__ targets, float scale, float* __restrict__ loss,
    bf16* __restrict__ dlogits, float* __restrict__ dbp, int rows, int width) {
  using C = HeadCfg<NT>;
  constexpr int V = C::V, TA = C::TA;
  extern __shared__ __attribute__((aligned(1024))) bf16 smem[];
  __shared__ float xmax[2][HEAD_ROWS], xsum[2][HEAD_ROWS], xtl[2][HEAD_ROWS];
  __shared__ __attribute__((aligned(16))) float sbias[V];
  const int lane = threadIdx.x & 63;
  // wave-uniform as far as the compiler knows: every MFMA guard below is a
  // scalar branch
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = wave & 1, hv = wave >> 1, half = lane >> 5;
  const int t0 = hv ? TA : 0, nt = hv ? NT - TA : TA;
  const int lrow = g * 32 + (lane & 31);               // row within the block
  int r = blockIdx.x * HEAD_ROWS + lrow;
  const bool live = r < rows;
  if (!live) r = rows - 1;                              // load a valid row, store nothing
  const int slices = width / 64;
  // the row's target and the bias, fetched before the main loop (the bias
  // goes to LDS after it)
  static_assert(V <= LM_THREADS, "one bias entry per thread");
  const int tgt = targets[r];
  const float bias_v = threadIdx.x < V ? bias[threadIdx.x] : 0.f;
  // the blocks walk the weight slices from different starting points (the
  // contraction's order is free), so that they do not all stream the same
  // weight lines out of L2 at once
  const int rot = blockIdx.x % slices;
  auto col0 = [&](int sl) {                 // logical slice -> first column
    const int p = min(sl, slices - 1) + rot;
    return (p >= slices ? p - slices : p) * 64;
  };

  // weight slice sl (clamped: issues past the last slice repeat it into a
  // stage nobody reads again) -> stage
  // stage = the weight slice [V][64] and the block's x slice [64 rows][64],
  // both swizzled (16-byte piece p of row m at p ^ ((m / 2) % 8))
  const int row0 = blockIdx.x * HEAD_ROWS;
  auto dma = [&](int sl, int stage) {
    const int k0 = col0(sl);
    bf16* dst = smem + stage * C::STAGE;
#pragma unroll
    for (int j = 0; j < V / 32; j++) {
      const int blk = j * 4 + wave, row = blk * 8 + (lane >> 3);
      const int piece = (lane & 7) ^ ((row >> 1) & 7);
      dma16(w + (size_t)row * width + k0 + 8 * piece, dst + blk * 512);
    }
#pragma unroll
    for (int j = 0; j < 2; j++) {
      const int blk = j * 4 + wave, row = blk * 8 + (lane >> 3);
      const int piece = (lane & 7) ^ ((row >> 1) & 7);
      const int xr = min(row0 + row, rows - 1);       // rows past the end: a valid row
      dma16(x + (size_t)xr * width + k0 + 8 * piece, dst + C::SLICE + blk * 512);
    }
  };
  f32x16 acc[TA];
#pragma unroll
  for (int t = 0; t < TA; t++) acc[t] = f32x16{};
  dma(0, 0);
  dma(1, 1);
  for (int sl = 0; sl < slices; sl++) {
    // stage sl landed (only stage sl + 1's DMA may be outstanding), and every
    // wave is done with stage sl - 1, which the next DMA overwrites
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(C::DMA) : "memory");
    dma(sl + 2, (sl + 2) % 3);
    const bf16* cur = smem + (sl % 3) * C::STAGE;
    const bf16* xs = cur + C::SLICE;
#pragma unroll
    for (int kk = 0; kk < 4; kk++) {
      const bf16x8 xf = *(const bf16x8*)(xs + swz<64>(lrow, 2 * kk + half));
#pragma unroll
      for (int t = 0; t < TA; t++)
        if (t < nt)
          acc[t] = mfma32(*(const bf16x8*)(cur + swz<64>(32 * (t0 + t) + (lane & 31), 2 * kk + half)),
                          xf, acc[t]);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  if (threadIdx.x < V) sbias[threadIdx.x] = bias_v;
  __syncthreads();

  // softmax over the row: in-lane, lane ^ 32, then the other half's wave
  float mx = -INFINITY, tl = 0.f;
#pragma unroll
  for (int t = 0; t < TA; t++) {
    if (t >= nt) continue;
#pragma unroll
    for (int q = 0; q < 4; q++) {
      const int v0 = 32 * (t0 + t) + 8 * q + 4 * half;
      const f32x4 b4 = *(const f32x4*)(sbias + v0);
#pragma unroll
      for (int j = 0; j < 4; j++) {
        const float l = acc[t][4 * q + j] + b4[j];
        acc[t][4 * q + j] = l;
        mx = fmaxf(mx, l);
        if (v0 + j == tgt) tl = l;
      }
    }
  }
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  tl += __shfl_xor(tl, 32);
  if (half == 0) {
    xmax[hv][lrow] = mx;
    xtl[hv][lrow] = tl;
  }
  __syncthreads();
  mx = fmaxf(xmax[0][lrow], xmax[1][lrow]);
  tl = xtl[0][lrow] + xtl[1][lrow];
  const float LOG2E = 1.4426950408889634f;
  float sum = 0.f;
#pragma unroll
  for (int t = 0; t < TA; t++) {
    if (t >= nt) continue;
#pragma unroll
    for (int e = 0; e < 16; e++) {
      const float p = __builtin_amdgcn_exp2f((acc[t][e] - mx) * LOG2E);
      acc[t][e] = p;
      sum += p;
    }
  }
  sum += __shfl_xor(sum, 32);
  if (half == 0) xsum[hv][lrow] = sum;
  __syncthreads();
  sum = xsum[0][lrow] + xsum[1][lrow];
  const float inv = 1.f / sum;
  if (live && hv == 0 && half == 0)
    loss[r] = mx + __builtin_amdgcn_logf(sum) * 0.6931471805599453f - tl;
  // the block's fp32 dlogits go through LDS: written back as bf16 in whole
  // 16-byte pieces of rows, and summed per column for the bias gradient
  float* dbs = (float*)smem;                            // [HEAD_ROWS][DB_LD] fp32
#pragma unroll
  for (int t = 0; t < TA; t++) {
    if (t >= nt) continue;
#pragma unroll
    for (int q = 0; q < 4; q++) {
      const int v0 = 32 * (t0 + t) + 8 * q + 4 * half;
      f32x4 d;
#pragma unroll
      for (int j = 0; j < 4; j++)
        d[j] = live ? scale * (acc[t][4 * q + j] * inv - (v0 + j == tgt ? 1.f : 0.f)) : 0.f;
      *(f32x4*)(dbs + lrow * C::DB_LD + v0) = d;
    }
  }
  __syncthreads();
  for (int pi = threadIdx.x; pi < HEAD_ROWS * (V / 8); pi += LM_THREADS) {
    const int lr = pi / (V / 8), c8 = (pi % (V / 8)) * 8;
    if (row0 + lr >= rows) continue;
    const f32x4 a = *(const f32x4*)(dbs + lr * C::DB_LD + c8);
    const f32x4 b = *(const f32x4*)(dbs + lr * C::DB_LD + c8 + 4);
    const bf16x8 o = {to_bf16(a[0]), to_bf16(a[1]), to_bf16(a[2]), to_bf16(a[3]),
                      to_bf16(b[0]), to_bf16(b[1]), to_bf16(b[2]), to_bf16(b[3])};
    *(bf16x8*)(dlogits + (size_t)(row0 + lr) * V + c8) = o;
  }
  if (!dbp) return;
  for (int v = threadIdx.x; v < V; v += LM_THREADS) {
    float s = 0.f;
    for (int k = 0; k < HEAD_ROWS; k++) s += dbs[k * C::DB_LD + v];
    dbp[(size_t)blockIdx.x * V + v] = s;
  }
}

// dbias[v] = sum over blocks b of dbp[b][v]: one wave per entry, lane j adding
// blocks j, j + 64, ... in order, then a fixed butterfly over the lanes.
__global__ __launch_bounds__(64) void head_db_reduce_kernel(const float* __restrict__ dbp,
                                                             float* __restrict__ dbias, int blocks,
                                                             int vocab) {
  const int v = blockIdx.x, lane = threadIdx.x;
  float s = 0.f;
  for (int b = lane; b < blocks; b += 64) s += dbp[(size_t)b * vocab + v];
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) s += __shfl_xor(s, m);
  if (lane == 0) dbias[v] = s;
}

template <int NT>
hipError_t head_launch(const bf16* x, const bf16* w, const float* bias, const int* targets,
                       float scale, float* loss, bf16* dlogits, float* dbias, float* dbp,
                       int rows, int width, hipStream_t st) {
  using C = HeadCfg<NT>;
  const int blocks = (rows + HEAD_ROWS - 1) / HEAD_ROWS;
  auto k = head_ce_kernel<NT>;
  static std::atomic<unsigned long long> lds_set{0};
  hipError_t e = lds_limit_once(lds_set, (const void*)k, (int)C::LDS);
  if (e != hipSuccess) return e;
  k<<<blocks, LM_THREADS, C::LDS, st>>>(x, w, bias, targets, scale, loss, dlogits,
                                         dbias ? dbp : nullptr, rows, width);
  e = hipGetLastError();
  if (e != hipSuccess || !dbias) return e;
  head_db_reduce_kernel<<<C::V, 64, 0, st>>>(dbp, dbias, blocks, C::V);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Head backward: the output head's weight and input gradients from dlogits,
// the two products the chain rule gives for logits = W x + bias:
//   dW[v][k] = sum over rows r of dl[r][v] x[r][k]   (fp32)
//   gx[r][k] = sum over v of dl[r][v] W[v][k]        (bf16)
// Both kernels: 128 x 128 output tiles, four waves of 64 x 64 (2 x 2 MFMA
// tiles of 32 x 32), 64-wide contraction steps staged in two LDS buffers; each
// thread loads the next step's pieces into registers before the MFMAs of the
// current one.  Pieces outside the rows, the vocabulary or the width are zero.
// ---------------------------------------------------------------------------
constexpr int HB_TILE = 128;
constexpr int HB_KS = 64;
constexpr int HB_TARGET_BLOCKS = 256;

// Rows per split of the weight gradient (a multiple of HB_KS) and the number
// of splits, so that about HB_TARGET_BLOCKS blocks work.
void head_dw_split(int rows, int width, int vocab, int* range, int* splits) {
  const int tiles = ((vocab + HB_TILE - 1) / HB_TILE) * ((width + HB_TILE - 1) / HB_TILE);
  int s = (HB_TARGET_BLOCKS + tiles - 1) / tiles;
  const int steps = (rows + HB_KS - 1) / HB_KS;
  if (s > steps) s = steps;
  if (s < 1) s = 1;
  const int per = (steps + s - 1) / s;                 // steps per split
  *range = per * HB_KS;
  *splits = (rows + *range - 1) / *range;
}

// LDS element offset of column `col` (a multiple of 8) of row `row` in a
// [rows][128] tile read with tr_frag<256>.
__device__ __forceinline__ int hb_tr_off(int row, int col) {
  return row * HB_TILE + trswz<256>(row, col >> 5) * 32 + (col & 31);
}

// Weight-gradient partials: block (vocabulary tile, width tile, split s) sums
// rows [s * range, (s + 1) * range) into part[s][v][k].  Both operands are
// row-major over the contraction (the rows), staged as [64 rows][128 columns]
// tiles and read transposed.
__global__ __launch_bounds__(256) void head_dw_kernel(const bf16* __restrict__ dl,
                                                      const bf16* __restrict__ x,
                                                      float* __restrict__ part, int rows,
                                                      int width, int vocab, int range) {
  __shared__ __attribute__((aligned(16))) bf16 ta[2][HB_KS * HB_TILE];
  __shared__ __attribute__((aligned(16))) bf16 tb[2][HB_KS * HB_TILE];
  const int tk_n = (width + HB_TILE - 1) / HB_TILE, tv_n = (vocab + HB_TILE - 1) / HB_TILE;
  int b = blockIdx.x;
  const int tk = b % tk_n;
  b /= tk_n;
  const int tv = b % tv_n, sp = b / tv_n;
  const int v0 = tv * HB_TILE, k0 = tk * HB_TILE;
  const int r0 = sp * range, r1 = min(rows, r0 + range);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;
  const int nsteps = r1 > r0 ? (r1 - r0 + HB_KS - 1) / HB_KS : 0;
  u32x4 ga[4], gb[4];
  auto load = [&](int t) {
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int p = tid + 256 * j, row = p >> 4, col = 8 * (p & 15);
      const int r = r0 + t * HB_KS + row;
      const bool rok = r < r1;
      ga[j] = rok && v0 + col < vocab ? *(const u32x4*)(dl + (size_t)r * vocab + v0 + col)
                                      : u32x4{0u, 0u, 0u, 0u};
      gb[j] = rok && k0 + col < width ? *(const u32x4*)(x + (size_t)r * width + k0 + col)
                                      : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int p = tid + 256 * j, row = p >> 4, col = 8 * (p & 15);
      *(u32x4*)(ta[buf] + hb_tr_off(row, col)) = ga[j];
      *(u32x4*)(tb[buf] + hb_tr_off(row, col)) = gb[j];
    }
  };
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; i++)
#pragma unroll
    for (int j = 0; j < 2; j++)
#pragma unroll
      for (int e = 0; e < 16; e++) acc[i][j][e] = 0.f;
  if (nsteps > 0) {
    load(0);
    stash(0);
  }
  __syncthreads();
  for (int t = 0; t < nsteps; t++) {
    const int buf = t & 1;
    if (t + 1 < nsteps) load(t + 1);
#pragma unroll
    for (int kk = 0; kk < HB_KS; kk += 16) {
      bf16x8 a[2], bb[2];
#pragma unroll
      for (int i = 0; i < 2; i++) a[i] = tr_frag<256>(ta[buf], kk, 64 * wm + 32 * i, lane);
#pragma unroll
      for (int j = 0; j < 2; j++) bb[j] = tr_frag<256>(tb[buf], kk, 64 * wn + 32 * j, lane);
#pragma unroll
      for (int i = 0; i < 2; i++)
#pragma unroll
        for (int j = 0; j < 2; j++) acc[i][j] = mfma32(a[i], bb[j], acc[i][j]);
    }
    if (t + 1 < nsteps) stash(buf ^ 1);
    __syncthreads();
  }
  // C[m = v][n = k]: lane l holds column k = .. + l % 32 and rows
  // v = .. + 8 (e / 4) + 4 (l / 32) + e % 4
  float* out = part + (size_t)sp * vocab * width;
#pragma unroll
  for (int i = 0; i < 2; i++)
#pragma unroll
    for (int j = 0; j < 2; j++) {
      const int k = k0 + 64 * wn + 32 * j + (lane & 31);
      if (k >= width) continue;
#pragma unroll
      for (int e = 0; e < 16; e++) {
        const int v = v0 + 64 * wm + 32 * i + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (v < vocab) out[(size_t)v * width + k] = acc[i][j][e];
      }
    }
}

// Input gradient: block (row tile, width tile) computes the transposed tile
// gx^T = W^T dl^T, so that a lane owns one row and four runs of four columns.
// W is row-major over the contraction (the vocabulary): [64 v][128 k] tiles
// read transposed; dl rows are contraction-contiguous: [128 r][64 v] tiles.
__global__ __launch_bounds__(256) void head_gx_kernel(const bf16* __restrict__ dl,
                                                      const bf16* __restrict__ w,
                                                      bf16* __restrict__ gx, int rows, int width,
                                                      int vocab) {
  __shared__ __attribute__((aligned(16))) bf16 tw[2][HB_KS * HB_TILE];
  __shared__ __attribute__((aligned(16))) bf16 td[2][HB_TILE * HB_KS];
  const int tk_n = (width + HB_TILE - 1) / HB_TILE;
  const int tk = blockIdx.x % tk_n, tr = blockIdx.x / tk_n;
  const int k0 = tk * HB_TILE, rb = tr * HB_TILE;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;      // columns 64 wm.., rows 64 wn..
  const int nsteps = (vocab + HB_KS - 1) / HB_KS;
  u32x4 gw[4], gd[4];
  auto load = [&](int t) {
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int p = tid + 256 * j;
      const int v = t * HB_KS + (p >> 4), col = 8 * (p & 15);
      gw[j] = v < vocab && k0 + col < width ? *(const u32x4*)(w + (size_t)v * width + k0 + col)
                                            : u32x4{0u, 0u, 0u, 0u};
      const int r = rb + (p >> 3), vc = t * HB_KS + 8 * (p & 7);
      gd[j] = r < rows && vc < vocab ? *(const u32x4*)(dl + (size_t)r * vocab + vc)
                                     : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int p = tid + 256 * j;
      *(u32x4*)(tw[buf] + hb_tr_off(p >> 4, 8 * (p & 15))) = gw[j];
      *(u32x4*)(td[buf] + swz<64>(p >> 3, p & 7)) = gd[j];
    }
  };
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; i++)
#pragma unroll
    for (int j = 0; j < 2; j++)
#pragma unroll
      for (int e = 0; e < 16; e++) acc[i][j][e] = 0.f;
  load(0);
  stash(0);
  __syncthreads();
  for (int t = 0; t < nsteps; t++) {
    const int buf = t & 1;
    if (t + 1 < nsteps) load(t + 1);
#pragma unroll
    for (int kk = 0; kk < HB_KS; kk += 16) {
      bf16x8 a[2], bb[2];
#pragma unroll
      for (int i = 0; i < 2; i++) a[i] = tr_frag<256>(tw[buf], kk, 64 * wm + 32 * i, lane);
#pragma unroll
      for (int j = 0; j < 2; j++)
        bb[j] = *(const bf16x8*)(td[buf] + swz<64>(64 * wn + 32 * j + (lane & 31),
                                                   (kk >> 3) + (lane >> 5)));
#pragma unroll
      for (int i = 0; i < 2; i++)
#pragma unroll
        for (int j = 0; j < 2; j++) acc[i][j] = mfma32(a[i], bb[j], acc[i][j]);
    }
    if (t + 1 < nsteps) stash(buf ^ 1);
    __syncthreads();
  }
  // C[m = k][n = r]: lane l holds row r = .. + l % 32 and columns
  // k = .. + 8 g + 4 (l / 32) + 0..3 for g = 0..3
#pragma unroll
  for (int i = 0; i < 2; i++)
#pragma unroll
    for (int j = 0; j < 2; j++) {
      const int r = rb + 64 * wn + 32 * j + (lane & 31);
      if (r >= rows) continue;
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const int k = k0 + 64 * wm + 32 * i + 8 * g + 4 * (lane >> 5);
        if (k >= width) continue;
        const bf16x4 v = {to_bf16(acc[i][j][4 * g]), to_bf16(acc[i][j][4 * g + 1]),
                          to_bf16(acc[i][j][4 * g + 2]), to_bf16(acc[i][j][4 * g + 3])};
        *(bf16x4*)(gx + (size_t)r * width + k) = v;
      }
    }
}

}  // namespace

size_t embedding_workspace_bytes(int rows, int width, int vocab) {
  return (size_t)emb_chunks(rows) * vocab * width * sizeof(float);
}

hipError_t launch_embedding_fwd(const bf16* table, const int* tokens, bf16* x, int rows,
                                int width, int vocab, hipStream_t st) {
  const size_t work = (size_t)rows * (width / 8);
  embed_fwd_kernel<<<(unsigned)((work + LM_THREADS - 1) / LM_THREADS), LM_THREADS, 0, st>>>(
      table, tokens, x, rows, width, vocab);
  return hipGetLastError();
}

hipError_t launch_embedding_bwd(const int* tokens, const bf16* dx, float* dtable, int accumulate,
                                float* workspace, int rows, int width, int vocab,
                                hipStream_t st) {
  const int chunks = emb_chunks(rows);
  const int chunk = (rows + chunks - 1) / chunks;
  embed_bwd_partial_kernel<<<chunks * vocab, LM_THREADS, 0, st>>>(tokens, dx, workspace, rows,
                                                                  width, vocab, chunk);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t elems = (size_t)vocab * width;
  embed_bwd_reduce_kernel<<<(unsigned)((elems / 4 + LM_THREADS - 1) / LM_THREADS), LM_THREADS,
                            0, st>>>(workspace, dtable, elems, chunks, accumulate);
  return hipGetLastError();
}

size_t head_workspace_bytes(int rows, int vocab) {
  return (size_t)((rows + HEAD_ROWS - 1) / HEAD_ROWS) * vocab * sizeof(float);
}

size_t head_backward_workspace_bytes(int rows, int width, int vocab) {
  int range, splits;
  head_dw_split(rows, width, vocab, &range, &splits);
  return (size_t)splits * vocab * width * sizeof(float);
}

hipError_t launch_head_backward(const bf16* x, const bf16* w, const bf16* dl, bf16* gx, float* dw,
                                int accumulate, float* workspace, int rows, int width, int vocab,
                                hipStream_t st) {
  const int tk_n = (width + HB_TILE - 1) / HB_TILE;
  if (gx) {
    const int tr_n = (rows + HB_TILE - 1) / HB_TILE;
    head_gx_kernel<<<tr_n * tk_n, 256, 0, st>>>(dl, w, gx, rows, width, vocab);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (!dw) return hipSuccess;
  int range, splits;
  head_dw_split(rows, width, vocab, &range, &splits);
  const int tv_n = (vocab + HB_TILE - 1) / HB_TILE;
  head_dw_kernel<<<tk_n * tv_n * splits, 256, 0, st>>>(dl, x, workspace, rows, width, vocab, range);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t elems = (size_t)vocab * width;
  embed_bwd_reduce_kernel<<<(unsigned)((elems / 4 + LM_THREADS - 1) / LM_THREADS), LM_THREADS,
                            0, st>>>(workspace, dw, elems, splits, accumulate);
  return hipGetLastError();
}

hipError_t launch_head_ce(const bf16* x, const bf16* w, const float* bias, const int* targets,
                          float scale, float* loss, bf16* dlogits, float* dbias, float* workspace,
                          int rows, int width, int vocab, hipStream_t st) {
#define HCMIX_HEAD_CASE(NT)                                                                    \
  case NT:                                                                                     \
    return head_launch<NT>(x, w, bias, targets, scale, loss, dlogits, dbias, workspace, rows, \
                           width, st);
  switch (vocab / 32) {
    HCMIX_HEAD_CASE(1)
    HCMIX_HEAD_CASE(2)
    HCMIX_HEAD_CASE(3)
    HCMIX_HEAD_CASE(4)
    HCMIX_HEAD_CASE(5)
    HCMIX_HEAD_CASE(6)
    HCMIX_HEAD_CASE(7)
    HCMIX_HEAD_CASE(8)
    default: return hipErrorInvalidValue;
  }
#undef HCMIX_HEAD_CASE
}

}  // namespace hcmix
