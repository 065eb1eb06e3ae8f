// Channel-shared mixing stack: Eq. (1) with both maps reduced to per-position
// scalars shared by every channel, taken from an n x n table per layer:
//   y[t][i][c] = A_l[i] x[t][i][c] + B_l[i] x[t][p(i)][c],
//   A_l[i] = T_l[i][i],  B_l[i] = m(i) T_l[i][p(i)].
// Every channel is independent, so a block owns one window and one slice of
// channels (8 pieces of 16 bytes in memory: 64 bf16 or 32 fp32 channels) and
// keeps that tile in LDS, in fp32, through every layer of the stack: the
// forward reads x_0 once and writes each layer's output once (rounded to the
// storage type; the chain itself goes on in fp32), and the backward reads dy
// once and each saved input once, and writes dx once.  The work is a handful
// of FMAs per element, so HBM bandwidth bounds it.
//
// Thread mapping (256 threads): thread tid owns memory piece k = tid % 8 of
// the positions tid / 8 + 32 j.  A wave covers 8 consecutive positions, and
// its global accesses are 128 contiguous bytes per position.  In LDS a row
// holds the slice in fp32 (256 bytes for bf16 slices, two 16-byte LDS pieces
// per thread, the pair swapped on odd rows; 128 bytes for fp32 slices): each
// 16-lane group of a read then covers two rows in distinct banks, for its
// own rows and for the partner rows alike (a stride of 8 or more maps 8
// consecutive rows onto 8 consecutive rows; a smaller stride or the local
// layer keeps neighbouring rows of opposite parity).
#include "device_common.h"
#include "hcmix_internal.h"

namespace hcmix {

namespace {

constexpr int SH_THREADS = 256;
constexpr int SH_PIECES = 8;   // 16-byte pieces of a row that one block owns

// 16 bytes of E as floats.
template <typename E>
struct Piece {
  static constexpr int V = 16 / (int)sizeof(E);
  float v[V];
};

template <typename E>
__device__ __forceinline__ Piece<E> unpack(const u32x4& u) {
  Piece<E> p;
  if constexpr (sizeof(E) == 2) {
#pragma unroll
    for (int q = 0; q < 4; q++) {
      p.v[2 * q] = __uint_as_float(u[q] << 16);
      p.v[2 * q + 1] = __uint_as_float(u[q] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int q = 0; q < 4; q++) p.v[q] = __uint_as_float(u[q]);
  }
  return p;
}

template <typename E>
__device__ __forceinline__ u32x4 pack(const Piece<E>& p) {
  u32x4 u;
  if constexpr (sizeof(E) == 2) {
#pragma unroll
    for (int q = 0; q < 4; q++) {
      const bf16 lo = to_bf16(p.v[2 * q]), hi = to_bf16(p.v[2 * q + 1]);
      u[q] = (unsigned)__builtin_bit_cast(unsigned short, lo) |
             ((unsigned)__builtin_bit_cast(unsigned short, hi) << 16);
    }
  } else {
#pragma unroll
    for (int q = 0; q < 4; q++) u[q] = __float_as_uint(p.v[q]);
  }
  return u;
}

// Partner of position i and whether i takes it (forward), for dimension d
// (d < 0: the local layer, partner i - 1).  The partner is always a valid row
// (i itself where there is none), so reads stay in the tile.
__device__ __forceinline__ int fwd_partner(int i, int d, int bidir, bool* takes) {
  if (d < 0) {
    *takes = i >= 1;
    return i >= 1 ? i - 1 : i;
  }
  *takes = bidir || ((i >> d) & 1);
  return i ^ (1 << d);
}

// The position that i sends to (whose output takes i's value), if any.
__device__ __forceinline__ int receiver(int i, int d, int n, int bidir, bool* sends) {
  if (d < 0) {
    *sends = i + 1 < n;
    return i + 1 < n ? i + 1 : i;
  }
  *sends = bidir || !((i >> d) & 1);
  return i ^ (1 << d);
}

// Sum over the 8 lanes of an aligned group (the 8 pieces of one position):
// within quads by swapping neighbours and pairs, then across the two quads of
// the group by mirroring it, all in DPP lane moves; every lane ends with the
// same value, (q0 + q1) with q the two quad sums, added in a fixed order.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}

__device__ __forceinline__ float sum8(float v) {
  v += dpp_move<0xb1>(v);          // quad_perm [1,0,3,2]
  v += dpp_move<0x4e>(v);          // quad_perm [2,3,0,1]
  return v + dpp_move<0x141>(v);   // row_half_mirror: lane l of 8 <- lane 7 - l
}

// (A_l[i], B_l[i]) of every position of layer l into coef[0 .. n).
__device__ __forceinline__ void load_coef(const float* __restrict__ tab, int d, int n, int bidir,
                                          float2* coef) {
  for (int i = threadIdx.x; i < n; i += SH_THREADS) {
    bool takes;
    const int p = fwd_partner(i, d, bidir, &takes);
    const float a = tab[(size_t)i * n + i];
    const float b = takes ? tab[(size_t)i * n + p] : 0.f;
    coef[i] = make_float2(a, b);
  }
}

// Per-thread view of a slice: V channels per memory piece, LP 16-byte LDS
// pieces (fp32) per memory piece, 8 * LP LDS pieces per row.
template <typename E>
struct Slice {
  static constexpr int V = Piece<E>::V;
  static constexpr int LP = V / 4;
  static constexpr int ROW = SH_PIECES * LP;
  // LDS piece h (< LP) of memory piece k of row i
  __device__ static int at(int i, int k, int h) {
    return i * ROW + ((k * LP + h) ^ (LP == 2 ? (i & 1) : 0));
  }
};

template <typename E>
__device__ __forceinline__ void lds_put(f32x4* tile, int i, int k, const Piece<E>& p) {
  using S = Slice<E>;
#pragma unroll
  for (int h = 0; h < S::LP; h++)
    tile[S::at(i, k, h)] = f32x4{p.v[4 * h], p.v[4 * h + 1], p.v[4 * h + 2], p.v[4 * h + 3]};
}

template <typename E>
__device__ __forceinline__ Piece<E> lds_get(const f32x4* tile, int i, int k) {
  using S = Slice<E>;
  Piece<E> p;
#pragma unroll
  for (int h = 0; h < S::LP; h++) {
    const f32x4 q = tile[S::at(i, k, h)];
    p.v[4 * h] = q[0];
    p.v[4 * h + 1] = q[1];
    p.v[4 * h + 2] = q[2];
    p.v[4 * h + 3] = q[3];
  }
  return p;
}

constexpr int SH_MAX_J = kSharedMaxN / (SH_THREADS / SH_PIECES);   // positions per thread

template <typename E>
__global__ __launch_bounds__(SH_THREADS) void shared_fwd_kernel(SharedFwdArgs a) {
  using S = Slice<E>;
  constexpr int V = S::V;
  const int n = a.n, width = a.width;
  const int chunks = width / (SH_PIECES * V);
  const int t = blockIdx.x / chunks;
  const int c0 = (blockIdx.x % chunks) * SH_PIECES * V;
  extern __shared__ __align__(16) unsigned char smem[];
  f32x4* tile = (f32x4*)smem;
  float2* coef = (float2*)(tile + n * S::ROW);   // [2][n]
  const int k = threadIdx.x % SH_PIECES;
  const int i0 = threadIdx.x / SH_PIECES;
  const int nj = n > i0 ? (n - i0 + 31) / 32 : 0;
  const size_t row0 = (size_t)t * n;
  const E* x0 = (const E*)a.x0;

  for (int j = 0; j < nj; j++) {
    const int i = i0 + 32 * j;
    lds_put<E>(tile, i, k, unpack<E>(*(const u32x4*)(x0 + (row0 + i) * width + c0 + k * V)));
  }
  load_coef(a.tab[0], a.dim[0], n, a.bidir, coef);
  __syncthreads();

  for (int l = 0; l < a.num_layers; l++) {
    const float2* cf = coef + (l & 1) * n;
    // the next layer's coefficients go to the other half, last read a layer ago
    if (l + 1 < a.num_layers)
      load_coef(a.tab[l + 1], a.dim[l + 1], n, a.bidir, coef + ((l + 1) & 1) * n);
    const int d = a.dim[l];
    E* out = (E*)a.xs[l];
    Piece<E> y[SH_MAX_J];
#pragma unroll
    for (int j = 0; j < SH_MAX_J; j++) {
      if (j < nj) {
        const int i = i0 + 32 * j;
        bool takes;
        const int p = fwd_partner(i, d, a.bidir, &takes);
        const float2 ab = cf[i];
        const Piece<E> xs = lds_get<E>(tile, i, k);
        const Piece<E> xp = lds_get<E>(tile, p, k);
#pragma unroll
        for (int v = 0; v < V; v++)
          y[j].v[v] = takes ? fmaf(ab.y, xp.v[v], ab.x * xs.v[v]) : ab.x * xs.v[v];
        *(global_u32x4*)(out + (row0 + i) * width + c0 + k * V) = pack<E>(y[j]);
      }
    }
    __syncthreads();    // every read of this layer's input is done
#pragma unroll
    for (int j = 0; j < SH_MAX_J; j++)
      if (j < nj) lds_put<E>(tile, i0 + 32 * j, k, y[j]);
    __syncthreads();
  }
}

template <typename E>
__global__ __launch_bounds__(SH_THREADS) void shared_bwd_kernel(SharedBwdArgs a) {
  using S = Slice<E>;
  constexpr int V = S::V;
  const int n = a.n, width = a.width;
  const int chunks = width / (SH_PIECES * V);
  const int t = blockIdx.x / chunks;
  const int c0 = (blockIdx.x % chunks) * SH_PIECES * V;
  extern __shared__ __align__(16) unsigned char smem[];
  f32x4* tile = (f32x4*)smem;
  float2* coef = (float2*)(tile + n * S::ROW);
  const int k = threadIdx.x % SH_PIECES;
  const int i0 = threadIdx.x / SH_PIECES;
  const int nj = n > i0 ? (n - i0 + 31) / 32 : 0;
  const size_t row0 = (size_t)t * n;
  const int L = a.num_layers;
  const E* dy = (const E*)a.dy;

  for (int j = 0; j < nj; j++) {
    const int i = i0 + 32 * j;
    lds_put<E>(tile, i, k, unpack<E>(*(const u32x4*)(dy + (row0 + i) * width + c0 + k * V)));
  }
  load_coef(a.tab[L - 1], a.dim[L - 1], n, a.bidir, coef + ((L - 1) & 1) * n);
  __syncthreads();

  // x_l rows of the layer to come, loaded one layer ahead so that their
  // latency passes under the barriers and LDS work of the layer before
  // (issued inside the layer, they would cost one memory latency per
  // position and layer).  Only the thread's own rows: the partner term of
  // dT, sum over c of g[r][c] x[i][c] for the receiver r of i, is formed by
  // i's thread, which holds x[i] and reads g[r] for dX anyway.
  u32x4 xo[SH_MAX_J];
  auto fetch_x = [&](int l) {
    const E* x = (const E*)a.xs[l];
#pragma unroll
    for (int j = 0; j < SH_MAX_J; j++)
      if (j < nj) xo[j] = *(const u32x4*)(x + (row0 + i0 + 32 * j) * width + c0 + k * V);
  };
  fetch_x(L - 1);

  for (int l = L - 1; l >= 0; l--) {
    // the tile holds g, the gradient of layer l's output
    const float2* cf = coef + (l & 1) * n;
    if (l > 0) load_coef(a.tab[l - 1], a.dim[l - 1], n, a.bidir, coef + ((l - 1) & 1) * n);
    const int d = a.dim[l];
    float* part = a.partial + ((size_t)l * gridDim.x + blockIdx.x) * n * 2;
    Piece<E> g[SH_MAX_J];
#pragma unroll
    for (int j = 0; j < SH_MAX_J; j++) {
      if (j < nj) {
        const int i = i0 + 32 * j;
        bool takes, sends;
        fwd_partner(i, d, a.bidir, &takes);
        const int r = receiver(i, d, n, a.bidir, &sends);
        // i sends to r exactly when r takes i: every partner slot of the
        // layer is written once, by the sender or (no sender) as zero
        const float ai = cf[i].x;
        const float cr = sends ? cf[r].y : 0.f;
        const Piece<E> gi = lds_get<E>(tile, i, k);
        const Piece<E> gr = lds_get<E>(tile, r, k);
        const Piece<E> xi = unpack<E>(xo[j]);
        float sd = 0.f, so = 0.f;
#pragma unroll
        for (int v = 0; v < V; v++) {
          g[j].v[v] = sends ? fmaf(cr, gr.v[v], ai * gi.v[v]) : ai * gi.v[v];
          sd = fmaf(gi.v[v], xi.v[v], sd);
          so = fmaf(gr.v[v], xi.v[v], so);
        }
        if (l == 0)
          *(global_u32x4*)((E*)a.dx + (row0 + i) * width + c0 + k * V) = pack<E>(g[j]);
        // the 8 pieces of position i sit in an aligned group of 8 lanes:
        // fixed-order sum, then the piece-0 lane writes the sums: the
        // diagonal one of i, and the partner one of i's receiver (or, when
        // nobody sends to i, a zero for i's own partner slot)
        sd = sum8(sd);
        so = sum8(so);
        if (k == 0) {
          part[2 * i] = sd;
          if (sends) part[2 * r + 1] = so;
          if (!takes) part[2 * i + 1] = 0.f;
        }
      }
    }
    if (l > 0) fetch_x(l - 1);
    __syncthreads();    // every read of g is done
    if (l > 0) {
#pragma unroll
      for (int j = 0; j < SH_MAX_J; j++)
        if (j < nj) lds_put<E>(tile, i0 + 32 * j, k, g[j]);
    }
    __syncthreads();
  }
}

// dT_l: the two sums of every position over all blocks (window x channel
// slice), then the table gradient's rows (zero off the layer's links unless
// accumulating).  Block = (layer, 16 positions: 128 contiguous bytes of
// every block's partials), 512 threads = 32 sums (16 positions x 2) x 16
// block classes: thread (q, v) adds the blocks b = q, q + 16, ... in order,
// and the 16 class sums are added in a fixed tree.
constexpr int SH_RED_ROWS = 16;
constexpr int SH_RED_CLASSES = 16;
constexpr int SH_RED_THREADS = 2 * SH_RED_ROWS * SH_RED_CLASSES;

__global__ __launch_bounds__(SH_RED_THREADS) void shared_dt_reduce_kernel(SharedReduceArgs a) {
  const int n = a.n;
  const int rows = n < SH_RED_ROWS ? n : SH_RED_ROWS;
  const int groups = n / rows;
  const int l = blockIdx.x / groups;
  const int i_base = (blockIdx.x % groups) * rows;
  const int v = threadIdx.x % (2 * SH_RED_ROWS);    // (position, which sum)
  const int q = threadIdx.x / (2 * SH_RED_ROWS);    // block class
  __shared__ float cls[SH_RED_CLASSES][2 * SH_RED_ROWS];
  __shared__ float sums[2 * SH_RED_ROWS];
  float acc = 0.f;
  if (v < 2 * rows) {
    // eight loads in flight, added in block order
    const float* src = a.partial + (size_t)l * a.blocks * n * 2 + 2 * i_base + v;
    for (int b0 = q; b0 < a.blocks; b0 += 8 * SH_RED_CLASSES) {
      float t[8];
#pragma unroll
      for (int u = 0; u < 8; u++) {
        const int b = b0 + u * SH_RED_CLASSES;
        t[u] = b < a.blocks ? src[(size_t)b * n * 2] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 8; u++) acc += t[u];
    }
  }
  cls[q][v] = acc;
  __syncthreads();
  if (threadIdx.x < 2 * SH_RED_ROWS) {
    float t[SH_RED_CLASSES];
#pragma unroll
    for (int c = 0; c < SH_RED_CLASSES; c++) t[c] = cls[c][threadIdx.x];
#pragma unroll
    for (int h = SH_RED_CLASSES / 2; h >= 1; h /= 2)
#pragma unroll
      for (int c = 0; c < h; c++) t[c] += t[c + h];
    sums[threadIdx.x] = t[0];
  }
  __syncthreads();
  float* dt = a.dt[l];
  const int d = a.dim[l];
  for (int e = threadIdx.x; e < rows * n; e += SH_RED_THREADS) {
    const int row = i_base + e / n, j = e % n;
    bool takes;
    const int p = fwd_partner(row, d, a.bidir, &takes);
    const bool diag = j == row, off = takes && j == p;
    const float val = diag ? sums[2 * (row - i_base)] : off ? sums[2 * (row - i_base) + 1] : 0.f;
    float* o = dt + (size_t)row * n + j;
    if (a.accumulate) {
      if (diag || off) *o += val;
    } else {
      *o = val;
    }
  }
}

}  // namespace

bool shared_stack_eligible(int64_t n, int64_t width, int32_t num_layers, int32_t elem_bytes) {
  const int64_t c = SH_PIECES * (16 / elem_bytes);
  return n >= 2 && n <= kSharedMaxN && (n & (n - 1)) == 0 && width % c == 0 && num_layers >= 1 &&
         num_layers <= kSharedMaxLayers;
}

// The fp32 tile (4 bytes per channel) and two layers' coefficients.
static size_t shared_lds_bytes(int n, int elem_bytes) {
  return (size_t)n * SH_PIECES * (16 / elem_bytes) * 4 + (size_t)2 * n * sizeof(float2);
}

static int shared_blocks(int batch, int width, int elem_bytes) {
  return batch * (width / (SH_PIECES * (16 / elem_bytes)));
}

size_t shared_partial_bytes(int64_t batch, int64_t n, int64_t width, int32_t num_layers,
                            int32_t elem_bytes) {
  return (size_t)num_layers * shared_blocks((int)batch, (int)width, elem_bytes) * n * 2 *
         sizeof(float);
}

hipError_t launch_shared_forward(const SharedFwdArgs& a, int batch, int elem_bytes, hipStream_t st) {
  const int blocks = shared_blocks(batch, a.width, elem_bytes);
  const size_t lds = shared_lds_bytes(a.n, elem_bytes);
  if (elem_bytes == 2) {
    static std::atomic<unsigned long long> lds_set{0};
    const hipError_t attr =
        lds_limit_once(lds_set, (const void*)shared_fwd_kernel<bf16>, (int)shared_lds_bytes(kSharedMaxN, 2));
    if (attr != hipSuccess) return attr;
    shared_fwd_kernel<bf16><<<blocks, SH_THREADS, lds, st>>>(a);
  } else {
    static std::atomic<unsigned long long> lds_set{0};
    const hipError_t attr =
        lds_limit_once(lds_set, (const void*)shared_fwd_kernel<float>, (int)shared_lds_bytes(kSharedMaxN, 2));
    if (attr != hipSuccess) return attr;
    shared_fwd_kernel<float><<<blocks, SH_THREADS, lds, st>>>(a);
  }
  return hipGetLastError();
}

hipError_t launch_shared_backward(const SharedBwdArgs& a, const SharedReduceArgs& r, int batch,
                                  int elem_bytes, hipStream_t st) {
  const int blocks = shared_blocks(batch, a.width, elem_bytes);
  const size_t lds = shared_lds_bytes(a.n, elem_bytes);
  if (elem_bytes == 2) {
    static std::atomic<unsigned long long> lds_set{0};
    const hipError_t attr =
        lds_limit_once(lds_set, (const void*)shared_bwd_kernel<bf16>, (int)shared_lds_bytes(kSharedMaxN, 2));
    if (attr != hipSuccess) return attr;
    shared_bwd_kernel<bf16><<<blocks, SH_THREADS, lds, st>>>(a);
  } else {
    static std::atomic<unsigned long long> lds_set{0};
    const hipError_t attr =
        lds_limit_once(lds_set, (const void*)shared_bwd_kernel<float>, (int)shared_lds_bytes(kSharedMaxN, 2));
    if (attr != hipSuccess) return attr;
    shared_bwd_kernel<float><<<blocks, SH_THREADS, lds, st>>>(a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  SharedReduceArgs rr = r;
  rr.blocks = blocks;
  const int groups = a.n / (a.n < SH_RED_ROWS ? a.n : SH_RED_ROWS);
  shared_dt_reduce_kernel<<<a.num_layers * groups, SH_RED_THREADS, 0, st>>>(rr);
  return hipGetLastError();
}

}  // namespace hcmix
