// Internal declarations shared by the hcmix HIP sources (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <atomic>

namespace hcmix {

// Raises kernel `fn`'s dynamic LDS limit to `bytes` on the current device,
// once per device and call site: `done` is the call site's record of the
// devices already set (bit = device index; devices past 63 are set on every
// call).  The attribute is per device, so a process that drives several GPUs
// needs it on each.
inline hipError_t lds_limit_once(std::atomic<unsigned long long>& done, const void* fn,
                                 int bytes) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const unsigned long long bit = (dev >= 0 && dev < 64) ? 1ull << dev : 0ull;
  if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
  e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_release);
  return e;
}

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Row bookkeeping for one layer along hypercube dimension d (stride s = 2^d).
// A flattened row r = t*n + i (window t, position i) keeps bit d of i as bit d
// of r because n is a power of two above s, so r XOR s is the partner in the
// same window.  The rows with bit d clear ("lower" rows: the earlier endpoint
// of each link) are enumerated by q = 0 .. rows/2-1 by inserting a zero bit at
// position d; the partner "upper" row is lower_row(q) + s.
__device__ __forceinline__ int lower_row(int q, int d) {
  const int lo = q & ((1 << d) - 1);
  return ((q >> d) << (d + 1)) | lo;
}

// fp32 -> bf16, round to nearest even (the gfx950 conversion instruction).
__device__ __forceinline__ bf16 to_bf16(float v) { return (bf16)v; }

// ---- launchers (each returns hipGetLastError() of its launch) ----

// FMA path (fp32 arithmetic; data fp32, or bf16 when bf16_data, widened
// exactly and each output rounded once):
// out[r][j] = sum_k A[r][k] B1(j,k) + m(r) sum_k A[p(r)][k] B2(j,k).
// B(j,k) = W[j*width+k] when !transpose_w, W[k*width+j] when transpose_w.
// d >= 0: p(r) = r ^ 2^d, m(r) = partner_lower for rows with bit d clear,
// partner_upper otherwise.  d < 0 (local layer): p(r) = r + shift over windows
// of n rows, shift = -1 (m = 0 at a window's first row) or +1 (at its last).
// The weight gradients (fp32 out) of a local layer (d < 0) pair row r with
// r - 1.
hipError_t launch_mix_fma(const void* A, const void* W1, const void* W2, void* out, int rows,
                          int width, int d, int partner_lower, int partner_upper, int n,
                          int shift, bool transpose_w, bool bf16_data, hipStream_t st);

hipError_t launch_dw_fma(const void* X, const void* dY, float* dws, float* dwo, int rows,
                         int width, int d, int n, int bidir, int accumulate, bool bf16_data,
                         hipStream_t st);

// bf16 MFMA: same contraction as launch_mix_fma.  B(j,k) = B[j*width+k] when
// !transpose_b, B[k*width+j] when transpose_b (read transposed from LDS).
// width % 64 == 0.
hipError_t launch_mix_bf16(const bf16* A, const bf16* B1, const bf16* B2, bf16* out,
                           int rows, int width, int d, int partner_lower, int partner_upper,
                           bool transpose_b, hipStream_t st);

// Plain bf16 product with the mix kernel's pipeline: out [rows][N] (row stride
// ldo) = A [rows][K] B^T, B [N][ldb] (k contiguous), or = A B with B [K][ldb]
// when transpose_b.  rows even, K % 64 == 0, N % 64 == 0; fp32 accumulation,
// bf16 output.
hipError_t launch_gemm_bf16(const bf16* A, const bf16* B, bf16* out, int rows, int K, int N,
                            int ldb, int ldo, bool transpose_b, hipStream_t st);

// Split-K weight gradients into `partial` ([splits][2][width][width] fp32),
// then a fixed-order reduction into dws / dwo.
// Local layer (jump 1), bf16: out_r = A_r B1^T + m(r) A_(r+delta) B2^T over
// windows of n rows; delta = -1 (forward: m = 0 at a window's first row) or +1
// (dX: m = 0 at a window's last row).  transpose_b as launch_mix_bf16.
hipError_t launch_shift_bf16(const bf16* A, const bf16* B1, const bf16* B2, bf16* out, int rows,
                             int width, int n, int delta, bool transpose_b, hipStream_t st);
int dw_bf16_splits(int rows, int width);
// dst[m] = src[m]^T for `count` (<= kTransposeBatch) bf16 matrices of
// width x width, width a multiple of 64.
constexpr int kTransposeBatch = 64;
struct TransposeArgs {
  const bf16* src[kTransposeBatch];
  bf16* dst[kTransposeBatch];
  int width;
};
hipError_t launch_transpose_bf16(const TransposeArgs& a, int count, hipStream_t st);

hipError_t launch_dw_bf16(const bf16* X, const bf16* dY, float* partial, float* dws, float* dwo,
                          int rows, int width, int d, int n, int bidir, int accumulate,
                          hipStream_t st);

// A weight-gradient reduction whose split partials are complete:
// dW_self/dW_off (+)= the sum of `splits` partial slots (each 2 x width^2
// floats: the dW_self part, then the dW_off part), in slot order.
struct DwReduce {
  const float* partial;   // null: nothing to reduce
  float* dws;
  float* dwo;
  int splits;
  int accumulate;
};
hipError_t launch_dw_reduce(const DwReduce& r, int width, hipStream_t st);

// Weight gradients of a whole stack (up to kBatchMaxLayers layers) in one
// launch (bf16, width % 128 == 0), plus a fixed-order reduction when the
// layers are split over row ranges.
constexpr int kBatchMaxLayers = 64;
struct DwBatchArgs {
  const bf16* x[kBatchMaxLayers];    // input of each layer
  const bf16* dy[kBatchMaxLayers];   // gradient of each layer's output
  float* dws[kBatchMaxLayers];
  float* dwo[kBatchMaxLayers];
  int dim[kBatchMaxLayers];          // hypercube dimension, or -1 for the local layer
  float* partial;                    // [L][splits][2][width][width] when splits > 1
  int rows, width, n, num_layers, splits, bidir, accumulate;
};
// Splits per layer for num_layers layers of this shape (1: no partials).
int dw_batch_splits(int rows, int width, int num_layers);
hipError_t launch_dw_batch_bf16(const DwBatchArgs& a, hipStream_t st);

// ---- fused small-width stack (width 64, n in {64, 128, 256}) ----

constexpr int kFusedMaxLayers = 64;

struct FusedFwdArgs {
  const bf16* x0;
  const bf16* ws[kFusedMaxLayers];
  const bf16* wo[kFusedMaxLayers];
  bf16* xs[kFusedMaxLayers];       // x_1 .. x_L
  int dim[kFusedMaxLayers];        // hypercube dimension of each layer
  int n, num_layers;
};

constexpr int kFusedMaxSplit = 4;    // blocks sharing one window's backward

struct FusedBwdArgs {
  const bf16* xs[kFusedMaxLayers];  // input of each layer, x_0 .. x_{L-1}
  const bf16* ws[kFusedMaxLayers];
  const bf16* wo[kFusedMaxLayers];
  int dim[kFusedMaxLayers];
  const bf16* dy;                   // gradient of x_L
  bf16* dx;                         // gradient of x_0
  float* partial;                   // [batch][L][2][64][64] per-window weight gradients
  int n, num_layers;
  // Set by launch_fused_backward: `split` blocks per window; block j of a
  // window forms the weight gradients of layers lo[j] .. hi[j] (a partition
  // of 0 .. L-1, block 0 lowest) and block 0 also writes dx.
  int split;
  int lo[kFusedMaxSplit], hi[kFusedMaxSplit];
};

struct FusedReduceArgs {
  const float* partial;
  float* dws[kFusedMaxLayers];
  float* dwo[kFusedMaxLayers];
  int batch, num_layers, accumulate;
};

bool fused_stack_eligible(int64_t n, int64_t width, int32_t num_layers);
size_t fused_partial_bytes(int64_t batch, int32_t num_layers);
hipError_t launch_fused_forward(const FusedFwdArgs& a, int batch, bool bidir, hipStream_t st);
// Blocks per window of the fused backward and their layer ranges (see
// FusedBwdArgs), for `cus` compute units: up to kFusedMaxSplit when the
// batch alone would leave compute units idle.
void fused_backward_split(int batch, int num_layers, int cus, int* split, int* lo, int* hi);

hipError_t launch_fused_backward(const FusedBwdArgs& a, const FusedReduceArgs& r, int batch,
                                 bool bidir, hipStream_t st);

// ---- channel-shared mixing stack (per-position scalars from n x n tables) ----
// y[t][i][c] = T[i][i] x[t][i][c] + m(i) T[i][p(i)] x[t][p(i)][c]; tables fp32
// [n][n]; activations bf16 or fp32; n a power of two up to kSharedMaxN; width a
// multiple of 64 (bf16) or 32 (fp32).  One block per window and slice of
// channels, the tile resident in LDS through every layer.

constexpr int kSharedMaxLayers = 64;
constexpr int kSharedMaxN = 256;

struct SharedFwdArgs {
  const void* x0;
  void* xs[kSharedMaxLayers];          // x_1 .. x_L
  const float* tab[kSharedMaxLayers];
  int dim[kSharedMaxLayers];           // hypercube dimension, or -1 for the local layer
  int n, width, num_layers, bidir;
};

struct SharedBwdArgs {
  const void* xs[kSharedMaxLayers];    // inputs x_0 .. x_{L-1}
  const float* tab[kSharedMaxLayers];
  int dim[kSharedMaxLayers];
  const void* dy;
  void* dx;
  float* partial;                      // [L][blocks][n][2] per-block sums of the table gradient
  int n, width, num_layers, bidir;
};

struct SharedReduceArgs {
  const float* partial;
  float* dt[kSharedMaxLayers];         // fp32 [n][n] table gradients
  int dim[kSharedMaxLayers];
  int n, blocks, num_layers, bidir, accumulate;
};

bool shared_stack_eligible(int64_t n, int64_t width, int32_t num_layers, int32_t elem_bytes);
size_t shared_partial_bytes(int64_t batch, int64_t n, int64_t width, int32_t num_layers,
                            int32_t elem_bytes);
hipError_t launch_shared_forward(const SharedFwdArgs& a, int batch, int elem_bytes, hipStream_t st);
hipError_t launch_shared_backward(const SharedBwdArgs& a, const SharedReduceArgs& r, int batch,
                                  int elem_bytes, hipStream_t st);

// ---- decode step (one position of every window through one layer) ----
// x_in / x_partner / record / out are row bases of window 0; window b is at
// + b * stride elements.  x_partner null: the position takes no partner.
// record (may be null): where the layer's input is written for later positions.
// Causal multi-head attention, bf16, head dimension 64, n a multiple of 32
// up to 256: qkv [batch][n][3][heads][64], out / dout [batch][n][heads][64],
// lse [batch][heads][n] fp32.
hipError_t launch_attention_fwd_bf16(const bf16* qkv, bf16* out, float* lse, int batch, int n,
                                     int heads, hipStream_t st);
hipError_t launch_attention_bwd_bf16(const bf16* qkv, const bf16* out, const float* lse,
                                     const bf16* dout, bf16* dqkv, int batch, int n, int heads,
                                     hipStream_t st);

// Field coupling (coordinates p fp32 [batch][n][c], c <= 64; x, y, dy, dx
// bf16 [batch][n][width], width % 64 == 0; n <= 256): row statistics
// row_mean and lse fp32 [batch][n], partners fp32 [batch][n] or null.
// workspace: field_workspace_bytes(batch, n, c) bytes, 256-byte aligned (each
// window's coordinate table, written by the forward, then for the backward the
// gradient of the squared distances, fp32 [batch][NP][NP] with NP = n rounded
// up to 32, and the couplings, bf16 [batch][NP][NP]).  reuse_table: the
// backward takes the tables the forward wrote to this workspace for the same
// p instead of building them again.
size_t field_workspace_bytes(int batch, int n, int c);
hipError_t launch_field_fwd(const float* p, const bf16* x, bf16* y, float* row_mean, float* lse,
                            float* partners, void* workspace, int batch, int n, int c, int width,
                            float inv_tau, int scaled, hipStream_t st);
hipError_t launch_field_bwd(const float* p, const bf16* x, const float* row_mean,
                            const float* lse, const bf16* dy, float* dp, bf16* dx, void* workspace,
                            int reuse_table, int batch, int n, int c, int width, float inv_tau,
                            int scaled, hipStream_t st);

// Language-model harness kernels (bf16, width % 64 == 0): embedding gather and
// its fixed-order scatter sum (workspace embedding_workspace_bytes), fused
// output head + cross-entropy (vocab a multiple of 32 up to 256).
size_t embedding_workspace_bytes(int rows, int width, int vocab);
hipError_t launch_embedding_fwd(const bf16* table, const int* tokens, bf16* x, int rows,
                                int width, int vocab, hipStream_t st);
hipError_t launch_embedding_bwd(const int* tokens, const bf16* dx, float* dtable, int accumulate,
                                float* workspace, int rows, int width, int vocab, hipStream_t st);
// Head: with dbias, also the bias gradient (column sums of dlogits) through
// head_workspace_bytes of per-block sums.
size_t head_workspace_bytes(int rows, int vocab);
hipError_t launch_head_ce(const bf16* x, const bf16* w, const float* bias, const int* targets,
                          float scale, float* loss, bf16* dlogits, float* dbias, float* workspace,
                          int rows, int width, int vocab, hipStream_t st);
// Head backward: gx = dl W (bf16, optional) and dW (+)= dl^T x (fp32, optional)
// through head_backward_workspace_bytes of row-range partials summed in order;
// vocab a multiple of 32.
size_t head_backward_workspace_bytes(int rows, int width, int vocab);
hipError_t launch_head_backward(const bf16* x, const bf16* w, const bf16* dl, bf16* gx, float* dw,
                                int accumulate, float* workspace, int rows, int width, int vocab,
                                hipStream_t st);

struct DecodeLayerArgs {
  const bf16* x_in;
  const bf16* x_partner;
  const bf16* w_self;
  const bf16* w_off;
  bf16* out;
  bf16* record;
  int64_t in_stride, partner_stride, out_stride, rec_stride;
  int batch, width;
};
struct DecodeLayerArgsF32 {
  const float* x_in;
  const float* x_partner;
  const float* w_self;
  const float* w_off;
  float* out;
  float* record;
  int64_t in_stride, partner_stride, out_stride, rec_stride;
  int batch, width;
};
hipError_t launch_decode_bf16(const DecodeLayerArgs& a, hipStream_t st);   // width % 64 == 0
hipError_t launch_decode_f32(const DecodeLayerArgsF32& a, hipStream_t st);
// bf16 widths that are not a multiple of 64: plain fp32 FMAs, one rounding
hipError_t launch_decode_bf16_fma(const DecodeLayerArgs& a, hipStream_t st);

}  // namespace hcmix
