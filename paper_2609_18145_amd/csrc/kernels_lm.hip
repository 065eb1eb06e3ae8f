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
// at most EMB_MAX_CHUNK each) whose token is v: wave 0 lists the matching rows
// in row order, then wave k adds matches k, k + 4, ... in that order (8 columns
// per lane, 64 lanes: 512 columns per pass), and the four wave sums are added
// in wave order into partial[c][v].
// A second kernel adds the chunks in chunk order.
// ---------------------------------------------------------------------------
constexpr int EMB_MIN_CHUNKS = 32;    // spreads a frequent token's rows over blocks
constexpr int EMB_MAX_CHUNK = 4096;   // rows per chunk held in LDS as a match list
int emb_chunks(int rows) {
  const int c = (rows + EMB_MAX_CHUNK - 1) / EMB_MAX_CHUNK;
  return c > EMB_MIN_CHUNKS ? c : EMB_MIN_CHUNKS;
}

__global__ __launch_bounds__(LM_THREADS) void embed_bwd_partial_kernel(
    const int* __restrict__ tokens, const bf16* __restrict__ dx, float* __restrict__ partial,
    int rows, int width, int vocab, int chunk) {
  __shared__ int list[EMB_MAX_CHUNK];
  __shared__ int count;
  __shared__ float red[4][512];
  const int v = blockIdx.x % vocab, c = blockIdx.x / vocab;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = c * chunk, r1 = min(rows, r0 + chunk);
  if (wave == 0) {
    int n = 0;
    for (int base = r0; base < r1; base += 64) {
      const int r = base + lane;
      const bool hit = r < r1 && tokens[r] == v;
      const unsigned long long m = __ballot(hit);
      if (hit) list[n + __popcll(m & ((1ull << lane) - 1))] = r;
      n += __popcll(m);
    }
    if (lane == 0) count = n;
  }
  __syncthreads();
  const int n = count;
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
        for (int u = 0; u < 8; u++) g[u] = *(const bf16x8*)(dx + (size_t)list[k + 4 * u] * width + col);
#pragma unroll
        for (int u = 0; u < 8; u++)
#pragma unroll
          for (int e = 0; e < 8; e++) acc[e] += (float)g[u][e];
      }
      for (; k < n; k += 4) {
        const bf16x8 g = *(const bf16x8*)(dx + (size_t)list[k] * width + col);
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

__global__ __launch_bounds__(LM_THREADS) void embed_bwd_reduce_kernel(
    const float* __restrict__ partial, float* __restrict__ dtable, size_t elems, int chunks,
    int accumulate) {
  const size_t i = (size_t)blockIdx.x * LM_THREADS + threadIdx.x;
  if (i >= elems) return;
  float s = 0.f;
  for (int c = 0; c < chunks; c++) s += partial[(size_t)c * elems + i];
  dtable[i] = accumulate ? dtable[i] + s : s;
}

// ---------------------------------------------------------------------------
// Head + cross-entropy.  Block: 4 waves x 32 rows.  Wave: logits^T for its 32
// rows and all NT * 32 vocabulary entries; the weights pass through LDS in
// 64-column slices shared by the four waves (two buffers), the wave's rows
// come straight from global memory.  Register e of tile t holds entry
// 32 t + 8 (e / 4) + 4 (lane / 32) + e % 4 of row lane % 32.
// ---------------------------------------------------------------------------
template <int NT>
__global__ __launch_bounds__(LM_THREADS) void head_ce_kernel(
    const bf16* __restrict__ x, const bf16* __restrict__ w, const float* __restrict__ bias,
    const int* __restrict__ targets, float scale, float* __restrict__ loss,
    bf16* __restrict__ dlogits, int rows, int width) {
  constexpr int V = NT * 32;
  constexpr int PIECES = V * 8 / LM_THREADS;        // 16-byte pieces of a slice per thread
  __shared__ __attribute__((aligned(1024))) bf16 sw[2][V * 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5;
  int r = (blockIdx.x * 4 + wave) * 32 + (lane & 31);
  const bool live = r < rows;
  if (!live) r = rows - 1;                     // load a valid row, store nothing
  const bf16* xr = x + (size_t)r * width + 8 * half;
  u32x4 wreg[PIECES];
  auto fetch = [&](int k0) {
#pragma unroll
    for (int j = 0; j < PIECES; j++) {
      const int pi = threadIdx.x + LM_THREADS * j, row = pi >> 3, p = pi & 7;
      wreg[j] = *(const u32x4*)(w + (size_t)row * width + k0 + 8 * p);
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int j = 0; j < PIECES; j++) {
      const int pi = threadIdx.x + LM_THREADS * j, row = pi >> 3, p = pi & 7;
      *(u32x4*)(sw[buf] + swz<64>(row, p)) = wreg[j];
    }
  };
  f32x16 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; t++) acc[t] = f32x16{};
  const int slices = width / 64;
  fetch(0);
  stash(0);
  __syncthreads();
  for (int sl = 0; sl < slices; sl++) {
    const int k0 = sl * 64;
    bf16x8 b[4];
#pragma unroll
    for (int kk = 0; kk < 4; kk++) b[kk] = *(const bf16x8*)(xr + k0 + 16 * kk);
    if (sl + 1 < slices) fetch(k0 + 64);
    const bf16* cur = sw[sl & 1];
#pragma unroll
    for (int kk = 0; kk < 4; kk++)
#pragma unroll
      for (int t = 0; t < NT; t++)
        acc[t] = mfma32(*(const bf16x8*)(cur + swz<64>(32 * t + (lane & 31), 2 * kk + half)),
                        b[kk], acc[t]);
    if (sl + 1 < slices) stash((sl + 1) & 1);
    __syncthreads();
  }
  const int tgt = targets[r];
  float mx = -INFINITY, tl = 0.f;
#pragma unroll
  for (int t = 0; t < NT; t++)
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const int v0 = 32 * t + 8 * g + 4 * half;
      const f32x4 b4 = *(const f32x4*)(bias + v0);
#pragma unroll
      for (int j = 0; j < 4; j++) {
        const float l = acc[t][4 * g + j] + b4[j];
        acc[t][4 * g + j] = l;
        mx = fmaxf(mx, l);
        if (v0 + j == tgt) tl = l;
      }
    }
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  tl += __shfl_xor(tl, 32);
  const float LOG2E = 1.4426950408889634f;
  float sum = 0.f;
#pragma unroll
  for (int t = 0; t < NT; t++)
#pragma unroll
    for (int e = 0; e < 16; e++) {
      const float p = __builtin_amdgcn_exp2f((acc[t][e] - mx) * LOG2E);
      acc[t][e] = p;
      sum += p;
    }
  sum += __shfl_xor(sum, 32);
  const float inv = 1.f / sum;
  if (!live) return;
  if (half == 0) loss[r] = mx + __builtin_amdgcn_logf(sum) * 0.6931471805599453f - tl;
  bf16* dr = dlogits + (size_t)r * V;
#pragma unroll
  for (int t = 0; t < NT; t++)
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const int v0 = 32 * t + 8 * g + 4 * half;
      bf16x4 o;
#pragma unroll
      for (int j = 0; j < 4; j++)
        o[j] = to_bf16(scale * (acc[t][4 * g + j] * inv - (v0 + j == tgt ? 1.f : 0.f)));
      *(bf16x4*)(dr + v0) = o;
    }
}

template <int NT>
hipError_t head_launch(const bf16* x, const bf16* w, const float* bias, const int* targets,
                       float scale, float* loss, bf16* dlogits, int rows, int width,
                       hipStream_t st) {
  const int blocks = (rows + 127) / 128;
  head_ce_kernel<NT><<<blocks, LM_THREADS, 0, st>>>(x, w, bias, targets, scale, loss, dlogits,
                                                    rows, width);
  return hipGetLastError();
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
  embed_bwd_reduce_kernel<<<(unsigned)((elems + LM_THREADS - 1) / LM_THREADS), LM_THREADS, 0,
                            st>>>(workspace, dtable, elems, chunks, accumulate);
  return hipGetLastError();
}

hipError_t launch_head_ce(const bf16* x, const bf16* w, const float* bias, const int* targets,
                          float scale, float* loss, bf16* dlogits, int rows, int width, int vocab,
                          hipStream_t st) {
  switch (vocab / 32) {
    case 1: return head_launch<1>(x, w, bias, targets, scale, loss, dlogits, rows, width, st);
    case 2: return head_launch<2>(x, w, bias, targets, scale, loss, dlogits, rows, width, st);
    case 3: return head_launch<3>(x, w, bias, targets, scale, loss, dlogits, rows, width, st);
    case 4: return head_launch<4>(x, w, bias, targets, scale, loss, dlogits, rows, width, st);
    case 5: return head_launch<5>(x, w, bias, targets, scale, loss, dlogits, rows, width, st);
    case 6: return head_launch<6>(x, w, bias, targets, scale, loss, dlogits, rows, width, st);
    case 7: return head_launch<7>(x, w, bias, targets, scale, loss, dlogits, rows, width, st);
    case 8: return head_launch<8>(x, w, bias, targets, scale, loss, dlogits, rows, width, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hcmix
