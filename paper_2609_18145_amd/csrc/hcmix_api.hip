// C ABI of libhcmix.so: argument validation and kernel dispatch.
// Every check runs before anything is enqueued, so a rejected call has no
// effect; there is one kernel path per shape class and no fallback.
#include "hcmix.h"
#include "hcmix_internal.h"

#include <mutex>
#include <string.h>

using namespace hcmix;

namespace {

thread_local char g_last_hip_error[256] = "";

hcmix_status hip_fail(hipError_t e) {
  strncpy(g_last_hip_error, hipGetErrorString(e), sizeof(g_last_hip_error) - 1);
  g_last_hip_error[sizeof(g_last_hip_error) - 1] = 0;
  return HCMIX_ERR_HIP;
}

constexpr int64_t kMaxRows = (int64_t)1 << 30;      // row indices stay in int32
constexpr int64_t kMaxElems = (int64_t)1 << 40;     // element offsets in size_t
constexpr int64_t kMaxWidth = (int64_t)1 << 16;     // widths stay in int32 products
constexpr int32_t kMaxLayers = 1 << 16;

size_t elem_size(int32_t dtype) { return dtype == HCMIX_BF16 ? 2 : 4; }

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
  return pa < pb + nb && pb < pa + na;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

size_t align256(size_t v) { return (v + 255) / 256 * 256; }

// Shape checks shared by every entry point; returns HCMIX_OK or the error.
hcmix_status check_shape(int64_t batch, int64_t n, int64_t width, int32_t layer, int32_t mode,
                         int32_t dtype) {
  if (layer == HCMIX_LAYER_NEAR) {
    // the local layer exists in causal form only
    if (hcmix_dim(0, n) < 0 || mode != HCMIX_CAUSAL) return HCMIX_ERR_INVALID_VALUE;
  } else if (hcmix_dim(layer, n) < 0) {
    return HCMIX_ERR_INVALID_VALUE;
  }
  if (batch < 1 || width < 1 || width > kMaxWidth) return HCMIX_ERR_INVALID_VALUE;
  if (mode != HCMIX_BIDIR && mode != HCMIX_CAUSAL) return HCMIX_ERR_INVALID_VALUE;
  if (dtype != HCMIX_F32 && dtype != HCMIX_BF16) return HCMIX_ERR_INVALID_VALUE;
  if (batch > kMaxRows / n) return HCMIX_ERR_INVALID_VALUE;
  if (batch * n > kMaxElems / width) return HCMIX_ERR_INVALID_VALUE;
  if (dtype == HCMIX_BF16 && width % 8 != 0) return HCMIX_ERR_UNSUPPORTED;
  return HCMIX_OK;
}

// bf16 widths that are a multiple of 64 run on the MFMA kernels; fp32, and
// bf16 widths that are only a multiple of 8, on the FMA kernels.
bool mfma_path(int32_t dtype, int64_t width) { return dtype == HCMIX_BF16 && width % 64 == 0; }

// Backward workspace (bf16): the split-K partial sums of the weight
// gradients, [splits][2][width][width] fp32.
size_t layer_workspace_bytes(int64_t batch, int64_t n, int64_t width, int32_t dtype) {
  if (!mfma_path(dtype, width)) return 0;
  const int splits = dw_bf16_splits((int)(batch * n), (int)width);
  return align256((size_t)splits * 2 * width * width * sizeof(float));
}

// Transposed copies of every layer's two weight matrices (bf16 stacks of two
// or more layers on the layer-by-layer path): dX then multiplies by W^T with
// the same kernel and the same 128-bit fragment reads as the forward.
size_t transposed_weight_bytes(int64_t width, int32_t num_layers, int32_t dtype) {
  if (!mfma_path(dtype, width) || num_layers < 2) return 0;
  return align256((size_t)2 * num_layers * width * width * sizeof(bf16));
}

// Deferred weight gradients (bf16, two or more layers, a width that is a
// multiple of 128): the dX chain runs first and keeps every intermediate
// gradient; then one launch per chunk of up to kBatchMaxLayers layers forms
// all their weight gradients, each block owning its tiles over every row pair
// of its layer (no split-K partials unless the stack is too short to fill the
// chip).
bool deferred_dw(int64_t width, int32_t num_layers, int32_t dtype) {
  return dtype == HCMIX_BF16 && num_layers > 1 && width % 128 == 0;
}

// Intermediate gradients kept by the deferred path: g_1 .. g_{L-1} (g_L is the
// caller's dy, g_0 its dx), or a ring of kBatchMaxLayers + 1 for longer stacks
// (a chunk's weight gradients read kBatchMaxLayers of them while the chain has
// written one more).
int grad_buffers(int32_t num_layers) {
  return num_layers <= kBatchMaxLayers ? num_layers - 1 : kBatchMaxLayers + 1;
}

size_t batch_partial_bytes(int64_t rows, int64_t width, int32_t chunk) {
  const int splits = dw_batch_splits((int)rows, (int)width, chunk);
  return splits > 1 ? align256((size_t)chunk * splits * 2 * width * width * sizeof(float)) : 0;
}

// Workspace of hcmix_stack_weight_gradients: the batched launch's partials
// (bf16, width a multiple of 128), else one layer's split-K partials.
size_t weight_grad_workspace_bytes(int64_t batch, int64_t n, int64_t width, int32_t num_layers,
                                   int32_t dtype) {
  if (dtype == HCMIX_BF16 && width % 128 == 0) {
    const int32_t full = num_layers < kBatchMaxLayers ? num_layers : kBatchMaxLayers;
    size_t part = batch_partial_bytes(batch * n, width, full);
    if (num_layers > kBatchMaxLayers && num_layers % kBatchMaxLayers) {
      const size_t last = batch_partial_bytes(batch * n, width, num_layers % kBatchMaxLayers);
      if (last > part) part = last;
    }
    return part;
  }
  return layer_workspace_bytes(batch, n, width, dtype);
}

size_t deferred_workspace_bytes(int64_t batch, int64_t n, int64_t width, int32_t num_layers) {
  const size_t act = align256((size_t)(batch * n * width) * sizeof(bf16));
  return (size_t)grad_buffers(num_layers) * act +
         transposed_weight_bytes(width, num_layers, HCMIX_BF16) +
         weight_grad_workspace_bytes(batch, n, width, num_layers, HCMIX_BF16);
}

// Stack backward workspace: the deferred path's gradients, transposed weights
// and partials; the per-window partials of the fused path; or two gradient
// buffers, one layer's partials and the transposed weights for the
// layer-by-layer path.
size_t stack_workspace_bytes(int64_t batch, int64_t n, int64_t width, int32_t num_layers,
                             int32_t dtype) {
  if (deferred_dw(width, num_layers, dtype))
    return deferred_workspace_bytes(batch, n, width, num_layers);
  const size_t act = align256((size_t)(batch * n * width) * elem_size(dtype));
  const size_t layered = (num_layers > 1 ? 2 * act : 0) +
                         layer_workspace_bytes(batch, n, width, dtype) +
                         transposed_weight_bytes(width, num_layers, dtype);
  if (dtype == HCMIX_BF16 && fused_stack_eligible(n, width, num_layers)) {
    // the schedule is not known here: enough for the fused path and for the
    // layer-by-layer path a schedule with local layers takes
    const size_t fused = align256(fused_partial_bytes(batch, num_layers));
    return fused > layered ? fused : layered;
  }
  return layered;
}

// The fused kernels handle hypercube layers only.
bool any_local_layer(const int32_t* layers, int32_t num_layers) {
  for (int l = 0; l < num_layers; l++)
    if (layers[l] == HCMIX_LAYER_NEAR) return true;
  return false;
}

// ---- unchecked per-layer dispatch (arguments already validated) ----

// d >= 0: hypercube layer of dimension d; d < 0: the local layer (jump 1).
hipError_t run_forward(int rows, int w, int d, int n, int bidir, int32_t dtype, const void* x,
                       const void* w_self, const void* w_off, void* y, hipStream_t s) {
  if (mfma_path(dtype, w)) {
    if (d < 0)
      return launch_shift_bf16((const bf16*)x, (const bf16*)w_self, (const bf16*)w_off, (bf16*)y,
                               rows, w, n, /*delta=*/-1, /*transpose_b=*/false, s);
    return launch_mix_bf16((const bf16*)x, (const bf16*)w_self, (const bf16*)w_off, (bf16*)y,
                           rows, w, d, /*partner_lower=*/bidir, /*partner_upper=*/1,
                           /*transpose_b=*/false, s);
  }
  return launch_mix_fma(x, w_self, w_off, y, rows, w, d, bidir, 1, n, /*shift=*/-1,
                        /*transpose_w=*/false, dtype == HCMIX_BF16, s);
}

// dX of one bf16 layer with the weights read as given (transpose_b) or from
// transposed copies.  Hypercube layer: lower rows always take their partner's
// gradient (causal: the lower row is the sender); local layer: every row but
// a window's last takes the next row's gradient.
hipError_t run_dx_bf16(int rows, int w, int d, int n, int bidir, const bf16* dy, const bf16* b1,
                       const bf16* b2, bf16* dx, bool transpose_b, hipStream_t s) {
  if (d < 0) return launch_shift_bf16(dy, b1, b2, dx, rows, w, n, /*delta=*/1, transpose_b, s);
  return launch_mix_bf16(dy, b1, b2, dx, rows, w, d, /*partner_lower=*/1,
                         /*partner_upper=*/bidir, transpose_b, s);
}

hipError_t run_backward(int rows, int w, int d, int n, int bidir, int32_t dtype, const void* x,
                        const void* w_self, const void* w_off, const void* dy, void* dx,
                        float* dw_self, float* dw_off, int accumulate, void* workspace,
                        hipStream_t s) {
  hipError_t e;
  if (mfma_path(dtype, w)) {
    e = run_dx_bf16(rows, w, d, n, bidir, (const bf16*)dy, (const bf16*)w_self,
                    (const bf16*)w_off, (bf16*)dx, /*transpose_b=*/true, s);
    if (e == hipSuccess)
      e = launch_dw_bf16((const bf16*)x, (const bf16*)dy, (float*)workspace, dw_self, dw_off,
                         rows, w, d, n, bidir, accumulate, s);
  } else {
    const bool b16 = dtype == HCMIX_BF16;
    e = launch_mix_fma(dy, w_self, w_off, dx, rows, w, d, 1, bidir, n, /*shift=*/1,
                       /*transpose_w=*/true, b16, s);
    if (e == hipSuccess)
      e = launch_dw_fma(x, dy, dw_self, dw_off, rows, w, d, n, bidir, accumulate, b16, s);
  }
  return e;
}

// A buffer in a call: its address and extent in bytes.
struct Span {
  const void* p;
  size_t n;
};

// Inputs must be non-null; outputs (with nonzero extent) non-null and
// overlapping no input and no other output; everything aligned to `al`.
hcmix_status check_spans(const Span* ins, int nin, const Span* outs, int nout, size_t al) {
  for (int i = 0; i < nin; i++)
    if (!ins[i].p) return HCMIX_ERR_INVALID_VALUE;
  for (int i = 0; i < nout; i++)
    if (!outs[i].p && outs[i].n) return HCMIX_ERR_INVALID_VALUE;
  for (int i = 0; i < nout; i++) {
    if (!outs[i].n) continue;
    for (int j = 0; j < nin; j++)
      if (overlaps(outs[i].p, outs[i].n, ins[j].p, ins[j].n)) return HCMIX_ERR_INVALID_VALUE;
    for (int j = i + 1; j < nout; j++)
      if (outs[j].n && overlaps(outs[i].p, outs[i].n, outs[j].p, outs[j].n))
        return HCMIX_ERR_INVALID_VALUE;
  }
  for (int i = 0; i < nin; i++)
    if (!aligned(ins[i].p, al)) return HCMIX_ERR_UNSUPPORTED;
  for (int i = 0; i < nout; i++)
    if (outs[i].n && !aligned(outs[i].p, al)) return HCMIX_ERR_UNSUPPORTED;
  return HCMIX_OK;
}

// wt[2l] = W_self[l]^T, wt[2l+1] = W_off[l]^T for every layer (bf16).
hipError_t transpose_weights(int w, int32_t num_layers, const void* const* w_self,
                             const void* const* w_off, bf16* wt, hipStream_t s) {
  const size_t ww = (size_t)w * w;
  hipError_t e = hipSuccess;
  for (int l0 = 0; l0 < num_layers && e == hipSuccess; l0 += kTransposeBatch / 2) {
    TransposeArgs t = {};
    t.width = w;
    int cnt = 0;
    for (int l = l0; l < num_layers && l < l0 + kTransposeBatch / 2; l++) {
      t.src[cnt] = (const bf16*)w_self[l];
      t.dst[cnt++] = wt + (2 * (size_t)l) * ww;
      t.src[cnt] = (const bf16*)w_off[l];
      t.dst[cnt++] = wt + (2 * (size_t)l + 1) * ww;
    }
    e = launch_transpose_bf16(t, cnt, s);
  }
  return e;
}

// Weight gradients of up to kBatchMaxLayers bf16 layers (width a multiple of
// 128) in one launch; `partial` is the workspace for split row ranges.
hipError_t launch_dw_chunk(int rows, int w, int n, int count, const int32_t* layers, int bidir,
                           const void* const* xs_in, const void* const* gs,
                           float* const* dw_self, float* const* dw_off, int accumulate,
                           float* partial, hipStream_t s) {
  DwBatchArgs a = {};
  for (int l = 0; l < count; l++) {
    a.x[l] = (const bf16*)xs_in[l];
    a.dy[l] = (const bf16*)gs[l];
    a.dws[l] = dw_self[l];
    a.dwo[l] = dw_off[l];
    a.dim[l] = hcmix_dim(layers[l], n);   // -1 for the local layer
  }
  a.partial = partial;
  a.rows = rows;
  a.width = w;
  a.n = n;
  a.num_layers = count;
  a.splits = dw_batch_splits(rows, w, count);
  a.bidir = bidir;
  a.accumulate = accumulate;
  return launch_dw_batch_bf16(a, s);
}

// The deferred path (arguments validated; workspace laid out as
// deferred_workspace_bytes counts it): gradients, transposed weights, partials.
hipError_t stack_backward_deferred(int rows, int w, int n, int32_t num_layers,
                                   const int32_t* layers, int bidir, const void* const* xs_in,
                                   const void* dy, void* dx, const void* const* w_self,
                                   const void* const* w_off, float* const* dw_self,
                                   float* const* dw_off, int accumulate, void* workspace,
                                   hipStream_t s) {
  const size_t act = align256((size_t)rows * w * sizeof(bf16));
  const size_t ww = (size_t)w * w;
  const int nb = grad_buffers(num_layers);
  char* gbase = (char*)workspace;
  bf16* wt = (bf16*)(gbase + (size_t)nb * act);
  float* partial = (float*)((char*)wt + transposed_weight_bytes(w, num_layers, HCMIX_BF16));
  // g_l: gradient of layer l's input (= layer l-1's output)
  auto grad = [&](int l) -> void* {
    if (l == num_layers) return (void*)dy;
    if (l == 0) return dx;
    return gbase + (size_t)(l % nb) * act;
  };
  hipError_t e = transpose_weights(w, num_layers, w_self, w_off, wt, s);
  for (int l1 = num_layers; l1 > 0 && e == hipSuccess;) {
    const int l0 = l1 > kBatchMaxLayers ? l1 - kBatchMaxLayers : 0;
    for (int l = l1 - 1; l >= l0 && e == hipSuccess; l--)
      e = run_dx_bf16(rows, w, hcmix_dim(layers[l], n), n, bidir, (const bf16*)grad(l + 1),
                      wt + 2 * (size_t)l * ww, wt + (2 * (size_t)l + 1) * ww, (bf16*)grad(l),
                      /*transpose_b=*/false, s);
    if (e != hipSuccess) break;
    const void* gs[kBatchMaxLayers];
    for (int l = l0; l < l1; l++) gs[l - l0] = grad(l + 1);
    e = launch_dw_chunk(rows, w, n, l1 - l0, layers + l0, bidir, xs_in + l0, gs, dw_self + l0,
                        dw_off + l0, accumulate, partial, s);
    l1 = l0;
  }
  return e;
}

// Scratch memory of hcmix_backward_no_alloc: a file-scope device array, one
// copy per GPU the library runs on, held until the process ends.  Its name
// is a host-side stand-in; the device address of each GPU's copy comes from
// hipGetSymbolAddress, taken once per device with that device current.
constexpr int kMaxDevices = 64;
__device__ __align__(256) unsigned char scratch[HCMIX_NO_ALLOC_SCRATCH_BYTES];
void* g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mutex;

// The current device's copy of `scratch` (null on failure, with *e set).
void* device_scratch(hipError_t* e) {
  int dev = 0;
  *e = hipGetDevice(&dev);
  if (*e != hipSuccess) return nullptr;
  if (dev < 0 || dev >= kMaxDevices) {
    *e = hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    *e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (*e != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

const char* hcmix_status_string(int32_t status) {
  switch (status) {
    case HCMIX_OK: return "HCMIX_OK";
    case HCMIX_ERR_INVALID_VALUE: return "HCMIX_ERR_INVALID_VALUE";
    case HCMIX_ERR_UNSUPPORTED: return "HCMIX_ERR_UNSUPPORTED";
    case HCMIX_ERR_HIP: return "HCMIX_ERR_HIP";
    default: return "HCMIX_ERR_UNKNOWN_STATUS";
  }
}

const char* hcmix_last_hip_error(void) { return g_last_hip_error; }

int32_t hcmix_dim(int32_t layer, int64_t n) {
  if (n < 2 || (n & (n - 1)) != 0 || layer < 0) return -1;
  int32_t b = 0;
  while (((int64_t)1 << b) < n) b++;
  return layer % b;
}

hcmix_status hcmix_forward(int64_t batch, int64_t n, int64_t width, int32_t layer, int32_t mode,
                           int32_t dtype, const void* x, const void* w_self, const void* w_off,
                           void* y, void* stream) {
  if (!x || !w_self || !w_off || !y) return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_shape(batch, n, width, layer, mode, dtype);
  if (st != HCMIX_OK) return st;
  const size_t es = elem_size(dtype);
  const size_t act = (size_t)(batch * n * width) * es, wgt = (size_t)(width * width) * es;
  const Span ins[3] = {{x, act}, {w_self, wgt}, {w_off, wgt}};
  const Span outs[1] = {{y, act}};
  st = check_spans(ins, 3, outs, 1, dtype == HCMIX_BF16 ? 16 : 4);
  if (st != HCMIX_OK) return st;
  hipError_t e = run_forward((int)(batch * n), (int)width, hcmix_dim(layer, n), (int)n,
                             mode == HCMIX_BIDIR, dtype, x, w_self, w_off, y,
                             (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

size_t hcmix_backward_workspace_bytes(int64_t batch, int64_t n, int64_t width, int32_t dtype) {
  if (check_shape(batch, n, width, 0, HCMIX_BIDIR, dtype) != HCMIX_OK) return 0;
  return layer_workspace_bytes(batch, n, width, dtype);
}

hcmix_status hcmix_backward(int64_t batch, int64_t n, int64_t width, int32_t layer, int32_t mode,
                            int32_t dtype, const void* x, const void* w_self, const void* w_off,
                            const void* dy, void* dx, float* dw_self, float* dw_off,
                            int32_t accumulate, void* workspace, size_t workspace_bytes,
                            void* stream) {
  if (!x || !w_self || !w_off || !dy || !dx || !dw_self || !dw_off)
    return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_shape(batch, n, width, layer, mode, dtype);
  if (st != HCMIX_OK) return st;
  const size_t need = layer_workspace_bytes(batch, n, width, dtype);
  if (need > 0 && (!workspace || workspace_bytes < need)) return HCMIX_ERR_INVALID_VALUE;
  const size_t es = elem_size(dtype);
  const size_t act = (size_t)(batch * n * width) * es, wgt = (size_t)(width * width) * es;
  const size_t gw = (size_t)(width * width) * sizeof(float);
  const Span ins[4] = {{x, act}, {w_self, wgt}, {w_off, wgt}, {dy, act}};
  const Span outs[4] = {{dx, act}, {dw_self, gw}, {dw_off, gw}, {workspace, need}};
  st = check_spans(ins, 4, outs, 4, dtype == HCMIX_BF16 ? 16 : 4);
  if (st != HCMIX_OK) return st;
  if (!aligned(dw_self, 16) || !aligned(dw_off, 16) || (need && !aligned(workspace, 256)))
    return HCMIX_ERR_UNSUPPORTED;
  hipError_t e = run_backward((int)(batch * n), (int)width, hcmix_dim(layer, n), (int)n,
                              mode == HCMIX_BIDIR, dtype, x, w_self, w_off, dy, dx, dw_self,
                              dw_off, accumulate != 0, workspace, (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

hcmix_status hcmix_backward_no_alloc(int64_t batch, int64_t n, int64_t width, int32_t layer,
                                     int32_t mode, int32_t dtype, const void* x,
                                     const void* w_self, const void* w_off, const void* dy,
                                     void* dx, float* dw_self, float* dw_off,
                                     int32_t accumulate, void* stream) {
  if (!x || !w_self || !w_off || !dy || !dx || !dw_self || !dw_off)
    return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_shape(batch, n, width, layer, mode, dtype);
  if (st != HCMIX_OK) return st;
  const size_t need = layer_workspace_bytes(batch, n, width, dtype);
  if (need > HCMIX_NO_ALLOC_SCRATCH_BYTES) return HCMIX_ERR_UNSUPPORTED;
  const size_t es = elem_size(dtype);
  const size_t act = (size_t)(batch * n * width) * es, wgt = (size_t)(width * width) * es;
  const size_t gw = (size_t)(width * width) * sizeof(float);
  const Span ins[4] = {{x, act}, {w_self, wgt}, {w_off, wgt}, {dy, act}};
  const Span outs[3] = {{dx, act}, {dw_self, gw}, {dw_off, gw}};
  st = check_spans(ins, 4, outs, 3, dtype == HCMIX_BF16 ? 16 : 4);
  if (st != HCMIX_OK) return st;
  if (!aligned(dw_self, 16) || !aligned(dw_off, 16)) return HCMIX_ERR_UNSUPPORTED;
  void* ws = nullptr;
  if (need > 0) {
    hipError_t e = hipSuccess;
    ws = device_scratch(&e);
    if (!ws) return hip_fail(e);
  }
  // the split-K partials are written in full before they are read, so the
  // scratch needs no clearing
  hipError_t e = run_backward((int)(batch * n), (int)width, hcmix_dim(layer, n), (int)n,
                              mode == HCMIX_BIDIR, dtype, x, w_self, w_off, dy, dx, dw_self,
                              dw_off, accumulate != 0, ws, (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

hcmix_status hcmix_stack_forward(int64_t batch, int64_t n, int64_t width, int32_t num_layers,
                                 const int32_t* layers, int32_t mode, int32_t dtype,
                                 const void* x, const void* const* w_self,
                                 const void* const* w_off, void* const* xs, void* stream) {
  if (!x || !layers || !w_self || !w_off || !xs) return HCMIX_ERR_INVALID_VALUE;
  if (num_layers < 1 || num_layers > kMaxLayers) return HCMIX_ERR_INVALID_VALUE;
  for (int l = 0; l < num_layers; l++) {
    hcmix_status st = check_shape(batch, n, width, layers[l], mode, dtype);
    if (st != HCMIX_OK) return st;
  }
  const size_t es = elem_size(dtype);
  const size_t act = (size_t)(batch * n * width) * es, wgt = (size_t)(width * width) * es;
  const size_t al = dtype == HCMIX_BF16 ? 16 : 4;
  for (int l = 0; l < num_layers; l++) {
    const Span ins[3] = {{x, act}, {w_self[l], wgt}, {w_off[l], wgt}};
    const Span outs[1] = {{xs[l], act}};
    hcmix_status st = check_spans(ins, 3, outs, 1, al);
    if (st != HCMIX_OK) return st;
    for (int j = 0; j < num_layers; j++) {
      if (j != l && overlaps(xs[l], act, xs[j], act)) return HCMIX_ERR_INVALID_VALUE;
      if (overlaps(xs[l], act, w_self[j], wgt) || overlaps(xs[l], act, w_off[j], wgt))
        return HCMIX_ERR_INVALID_VALUE;
    }
  }
  const int rows = (int)(batch * n), w = (int)width;
  const int bidir = mode == HCMIX_BIDIR;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = hipSuccess;
  if (dtype == HCMIX_BF16 && fused_stack_eligible(n, width, num_layers) &&
      !any_local_layer(layers, num_layers)) {
    FusedFwdArgs a = {};
    a.x0 = (const bf16*)x;
    for (int l = 0; l < num_layers; l++) {
      a.ws[l] = (const bf16*)w_self[l];
      a.wo[l] = (const bf16*)w_off[l];
      a.xs[l] = (bf16*)xs[l];
      a.dim[l] = hcmix_dim(layers[l], n);
    }
    a.n = (int)n;
    a.num_layers = num_layers;
    e = launch_fused_forward(a, (int)batch, bidir, s);
  } else {
    const void* in = x;
    for (int l = 0; l < num_layers && e == hipSuccess; l++) {
      e = run_forward(rows, w, hcmix_dim(layers[l], n), (int)n, bidir, dtype, in, w_self[l],
                      w_off[l], xs[l], s);
      in = xs[l];
    }
  }
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

size_t hcmix_stack_backward_workspace_bytes(int64_t batch, int64_t n, int64_t width,
                                            int32_t num_layers, int32_t dtype) {
  if (num_layers < 1 || num_layers > kMaxLayers) return 0;
  if (check_shape(batch, n, width, 0, HCMIX_BIDIR, dtype) != HCMIX_OK) return 0;
  return stack_workspace_bytes(batch, n, width, num_layers, dtype);
}

hcmix_status hcmix_stack_backward(int64_t batch, int64_t n, int64_t width, int32_t num_layers,
                                  const int32_t* layers, int32_t mode, int32_t dtype,
                                  const void* const* xs_in, const void* const* w_self,
                                  const void* const* w_off, const void* dy, void* dx,
                                  float* const* dw_self, float* const* dw_off,
                                  int32_t accumulate, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  if (!layers || !xs_in || !w_self || !w_off || !dy || !dx || !dw_self || !dw_off)
    return HCMIX_ERR_INVALID_VALUE;
  if (num_layers < 1 || num_layers > kMaxLayers) return HCMIX_ERR_INVALID_VALUE;
  for (int l = 0; l < num_layers; l++) {
    hcmix_status st = check_shape(batch, n, width, layers[l], mode, dtype);
    if (st != HCMIX_OK) return st;
    if (!xs_in[l] || !w_self[l] || !w_off[l] || !dw_self[l] || !dw_off[l])
      return HCMIX_ERR_INVALID_VALUE;
  }
  const size_t need = stack_workspace_bytes(batch, n, width, num_layers, dtype);
  if (need > 0 && (!workspace || workspace_bytes < need)) return HCMIX_ERR_INVALID_VALUE;
  const size_t es = elem_size(dtype);
  const size_t act = (size_t)(batch * n * width) * es, wgt = (size_t)(width * width) * es;
  const size_t gw = (size_t)(width * width) * sizeof(float);
  const size_t al = dtype == HCMIX_BF16 ? 16 : 4;
  // Outputs: dx, the workspace and every weight gradient.  Inputs: dy, every
  // layer input and weight.  No output may overlap any input or other output.
  const Span outs_fixed[2] = {{dx, act}, {workspace, need}};
  {
    const Span ins[1] = {{dy, act}};
    hcmix_status st = check_spans(ins, 1, outs_fixed, 2, al);
    if (st != HCMIX_OK) return st;
  }
  for (int l = 0; l < num_layers; l++) {
    const Span ins[3] = {{xs_in[l], act}, {w_self[l], wgt}, {w_off[l], wgt}};
    const Span outs[4] = {outs_fixed[0], outs_fixed[1], {dw_self[l], gw}, {dw_off[l], gw}};
    hcmix_status st = check_spans(ins, 3, outs, 4, al);
    if (st != HCMIX_OK) return st;
    for (int j = 0; j < num_layers; j++) {
      if (j == l) continue;
      const Span other_ins[3] = {{xs_in[j], act}, {w_self[j], wgt}, {w_off[j], wgt}};
      const Span other_outs[2] = {{dw_self[j], gw}, {dw_off[j], gw}};
      for (int k = 2; k < 4; k++) {
        for (int m = 0; m < 3; m++)
          if (overlaps(outs[k].p, outs[k].n, other_ins[m].p, other_ins[m].n))
            return HCMIX_ERR_INVALID_VALUE;
        for (int m = 0; m < 2; m++)
          if (overlaps(outs[k].p, outs[k].n, other_outs[m].p, other_outs[m].n))
            return HCMIX_ERR_INVALID_VALUE;
      }
    }
    if (!aligned(dw_self[l], 16) || !aligned(dw_off[l], 16)) return HCMIX_ERR_UNSUPPORTED;
  }
  if (need && !aligned(workspace, 256)) return HCMIX_ERR_UNSUPPORTED;

  const int rows = (int)(batch * n), w = (int)width;
  const int bidir = mode == HCMIX_BIDIR;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = hipSuccess;
  if (dtype == HCMIX_BF16 && fused_stack_eligible(n, width, num_layers) &&
      !any_local_layer(layers, num_layers)) {
    FusedBwdArgs a = {};
    FusedReduceArgs r = {};
    for (int l = 0; l < num_layers; l++) {
      a.xs[l] = (const bf16*)xs_in[l];
      a.ws[l] = (const bf16*)w_self[l];
      a.wo[l] = (const bf16*)w_off[l];
      a.dim[l] = hcmix_dim(layers[l], n);
      r.dws[l] = dw_self[l];
      r.dwo[l] = dw_off[l];
    }
    a.dy = (const bf16*)dy;
    a.dx = (bf16*)dx;
    a.partial = (float*)workspace;
    a.n = (int)n;
    a.num_layers = num_layers;
    r.partial = (const float*)workspace;
    r.batch = (int)batch;
    r.num_layers = num_layers;
    r.accumulate = accumulate != 0;
    e = launch_fused_backward(a, r, (int)batch, bidir, s);
  } else if (deferred_dw(width, num_layers, dtype)) {
    e = stack_backward_deferred(rows, w, (int)n, num_layers, layers, bidir, xs_in, dy, dx,
                                w_self, w_off, dw_self, dw_off, accumulate != 0, workspace, s);
  } else {
    // layer by layer; intermediate gradients ping-pong in the workspace
    const size_t act_al = align256(act);
    char* ws = (char*)workspace;
    void* gbuf[2] = {ws, ws + act_al};
    void* layer_ws = ws + (num_layers > 1 ? 2 * act_al : 0);
    const void* g = dy;
    const size_t lws = layer_workspace_bytes(batch, n, width, dtype);
    bf16* wt = (bf16*)((char*)layer_ws + lws);   // transposed weights (bf16, L >= 2)
    if (transposed_weight_bytes(width, num_layers, dtype) > 0)
      e = transpose_weights(w, num_layers, w_self, w_off, wt, s);
    const size_t ww = (size_t)w * w;
    for (int l = num_layers - 1; l >= 0 && e == hipSuccess; l--) {
      void* out = l == 0 ? dx : gbuf[l & 1];
      const int d = hcmix_dim(layers[l], n);
      if (mfma_path(dtype, w) && num_layers > 1) {
        // dX = W_self^T dy (+ partner W_off^T dy): the forward kernels on W^T
        e = run_dx_bf16(rows, w, d, (int)n, bidir, (const bf16*)g, wt + 2 * (size_t)l * ww,
                        wt + (2 * (size_t)l + 1) * ww, (bf16*)out, /*transpose_b=*/false, s);
        if (e == hipSuccess)
          e = launch_dw_bf16((const bf16*)xs_in[l], (const bf16*)g, (float*)layer_ws, dw_self[l],
                             dw_off[l], rows, w, d, (int)n, bidir, accumulate != 0, s);
      } else {
        e = run_backward(rows, w, d, (int)n, bidir, dtype, xs_in[l], w_self[l], w_off[l], g, out,
                         dw_self[l], dw_off[l], accumulate != 0, layer_ws, s);
      }
      g = out;
    }
  }
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

}  // extern "C"

size_t hcmix_stack_backward_data_workspace_bytes(int64_t width, int32_t num_layers,
                                                 int32_t dtype) {
  if (num_layers < 1 || num_layers > kMaxLayers || width < 1) return 0;
  if (dtype != HCMIX_F32 && dtype != HCMIX_BF16) return 0;
  return transposed_weight_bytes(width, num_layers, dtype);
}

hcmix_status hcmix_stack_backward_data(int64_t batch, int64_t n, int64_t width,
                                       int32_t num_layers, const int32_t* layers, int32_t mode,
                                       int32_t dtype, const void* const* w_self,
                                       const void* const* w_off, const void* dy,
                                       void* const* grads, void* dx, void* workspace,
                                       size_t workspace_bytes, void* stream) {
  if (!layers || !w_self || !w_off || !dy || !dx) return HCMIX_ERR_INVALID_VALUE;
  if (num_layers < 1 || num_layers > kMaxLayers) return HCMIX_ERR_INVALID_VALUE;
  if (num_layers > 1 && !grads) return HCMIX_ERR_INVALID_VALUE;
  for (int l = 0; l < num_layers; l++) {
    hcmix_status st = check_shape(batch, n, width, layers[l], mode, dtype);
    if (st != HCMIX_OK) return st;
    if (!w_self[l] || !w_off[l] || (l > 0 && !grads[l - 1])) return HCMIX_ERR_INVALID_VALUE;
  }
  const size_t need = transposed_weight_bytes(width, num_layers, dtype);
  if (need > 0 && (!workspace || workspace_bytes < need)) return HCMIX_ERR_INVALID_VALUE;
  const size_t es = elem_size(dtype);
  const size_t act = (size_t)(batch * n * width) * es, wgt = (size_t)(width * width) * es;
  const size_t al = dtype == HCMIX_BF16 ? 16 : 4;
  // Outputs: dx, the workspace and every grads[l]; inputs: dy and every weight.
  for (int k = 0; k < num_layers; k++) {
    // output k: dx (k == 0) or grads[k - 1], checked with the two fixed
    // outputs against dy and layer k's weights, then against every other
    // layer's weights and grads
    const Span ins[3] = {{dy, act}, {w_self[k], wgt}, {w_off[k], wgt}};
    const Span outs[3] = {{dx, act}, {workspace, need}, {k ? grads[k - 1] : nullptr, k ? act : 0}};
    hcmix_status st = check_spans(ins, 3, outs, 3, al);
    if (st != HCMIX_OK) return st;
    for (int j = 0; j < num_layers; j++) {
      if (j == k) continue;
      const Span other[3] = {{w_self[j], wgt}, {w_off[j], wgt}, {j ? grads[j - 1] : nullptr, j ? act : 0}};
      for (int o = 0; o < 3; o++) {
        if (!outs[o].n) continue;
        for (int m = 0; m < 3; m++)
          if (other[m].n && overlaps(outs[o].p, outs[o].n, other[m].p, other[m].n))
            return HCMIX_ERR_INVALID_VALUE;
      }
    }
  }
  if (need && !aligned(workspace, 256)) return HCMIX_ERR_UNSUPPORTED;

  const int rows = (int)(batch * n), w = (int)width;
  const int bidir = mode == HCMIX_BIDIR;
  hipStream_t s = (hipStream_t)stream;
  const size_t ww = (size_t)w * w;
  // g(l): gradient of layer l's input; g(L) = dy
  auto g = [&](int l) -> void* {
    if (l == num_layers) return (void*)dy;
    return l == 0 ? dx : grads[l - 1];
  };
  hipError_t e = hipSuccess;
  bf16* wt = (bf16*)workspace;
  if (need > 0) e = transpose_weights(w, num_layers, w_self, w_off, wt, s);
  for (int l = num_layers - 1; l >= 0 && e == hipSuccess; l--) {
    const int d = hcmix_dim(layers[l], n);
    if (mfma_path(dtype, w)) {
      if (need > 0)
        e = run_dx_bf16(rows, w, d, (int)n, bidir, (const bf16*)g(l + 1), wt + 2 * (size_t)l * ww,
                        wt + (2 * (size_t)l + 1) * ww, (bf16*)g(l), /*transpose_b=*/false, s);
      else
        e = run_dx_bf16(rows, w, d, (int)n, bidir, (const bf16*)g(l + 1), (const bf16*)w_self[l],
                        (const bf16*)w_off[l], (bf16*)g(l), /*transpose_b=*/true, s);
    } else {
      e = launch_mix_fma(g(l + 1), w_self[l], w_off[l], g(l), rows, w, d, 1, bidir, (int)n,
                         /*shift=*/1, /*transpose_w=*/true, dtype == HCMIX_BF16, s);
    }
  }
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

size_t hcmix_stack_weight_gradients_workspace_bytes(int64_t batch, int64_t n, int64_t width,
                                                     int32_t num_layers, int32_t dtype) {
  if (num_layers < 1 || num_layers > kMaxLayers) return 0;
  if (check_shape(batch, n, width, 0, HCMIX_BIDIR, dtype) != HCMIX_OK) return 0;
  return weight_grad_workspace_bytes(batch, n, width, num_layers, dtype);
}

hcmix_status hcmix_stack_weight_gradients(int64_t batch, int64_t n, int64_t width,
                                          int32_t num_layers, const int32_t* layers, int32_t mode,
                                          int32_t dtype, const void* const* xs_in,
                                          const void* const* dys, float* const* dw_self,
                                          float* const* dw_off, int32_t accumulate,
                                          void* workspace, size_t workspace_bytes,
                                          void* stream) {
  if (!layers || !xs_in || !dys || !dw_self || !dw_off) return HCMIX_ERR_INVALID_VALUE;
  if (num_layers < 1 || num_layers > kMaxLayers) return HCMIX_ERR_INVALID_VALUE;
  for (int l = 0; l < num_layers; l++) {
    hcmix_status st = check_shape(batch, n, width, layers[l], mode, dtype);
    if (st != HCMIX_OK) return st;
    if (!xs_in[l] || !dys[l] || !dw_self[l] || !dw_off[l]) return HCMIX_ERR_INVALID_VALUE;
  }
  const size_t need = weight_grad_workspace_bytes(batch, n, width, num_layers, dtype);
  if (need > 0 && (!workspace || workspace_bytes < need)) return HCMIX_ERR_INVALID_VALUE;
  const size_t act = (size_t)(batch * n * width) * elem_size(dtype);
  const size_t gw = (size_t)(width * width) * sizeof(float);
  const size_t al = dtype == HCMIX_BF16 ? 16 : 4;
  // Outputs: the workspace and every weight gradient; inputs: every xs_in[l]
  // and dys[l].  No output may overlap any input or another output.
  for (int l = 0; l < num_layers; l++) {
    const Span ins[2] = {{xs_in[l], act}, {dys[l], act}};
    const Span outs[3] = {{workspace, need}, {dw_self[l], gw}, {dw_off[l], gw}};
    hcmix_status st = check_spans(ins, 2, outs, 3, al);
    if (st != HCMIX_OK) return st;
    for (int j = 0; j < num_layers; j++) {
      if (j == l) continue;
      const Span other[4] = {{xs_in[j], act}, {dys[j], act}, {dw_self[j], gw}, {dw_off[j], gw}};
      for (int k = 1; k < 3; k++)
        for (int m = 0; m < 4; m++)
          if (overlaps(outs[k].p, outs[k].n, other[m].p, other[m].n))
            return HCMIX_ERR_INVALID_VALUE;
    }
    if (!aligned(dw_self[l], 16) || !aligned(dw_off[l], 16)) return HCMIX_ERR_UNSUPPORTED;
  }
  if (need && !aligned(workspace, 256)) return HCMIX_ERR_UNSUPPORTED;
  const int rows = (int)(batch * n), w = (int)width;
  const int bidir = mode == HCMIX_BIDIR;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = hipSuccess;
  if (dtype == HCMIX_BF16 && width % 128 == 0) {
    for (int l0 = 0; l0 < num_layers && e == hipSuccess; l0 += kBatchMaxLayers) {
      const int count = num_layers - l0 < kBatchMaxLayers ? num_layers - l0 : kBatchMaxLayers;
      e = launch_dw_chunk(rows, w, (int)n, count, layers + l0, bidir, xs_in + l0, dys + l0,
                          dw_self + l0, dw_off + l0, accumulate != 0, (float*)workspace, s);
    }
  } else {
    for (int l = 0; l < num_layers && e == hipSuccess; l++) {
      const int d = hcmix_dim(layers[l], n);
      if (mfma_path(dtype, w))
        e = launch_dw_bf16((const bf16*)xs_in[l], (const bf16*)dys[l], (float*)workspace,
                           dw_self[l], dw_off[l], rows, w, d, (int)n, bidir, accumulate != 0, s);
      else
        e = launch_dw_fma(xs_in[l], dys[l], dw_self[l], dw_off[l], rows, w, d, (int)n, bidir,
                          accumulate != 0, dtype == HCMIX_BF16, s);
    }
  }
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

// Shape checks of the attention entry points.
hcmix_status check_attention(int64_t batch, int64_t n, int32_t heads, int32_t head_dim) {
  if (batch < 1 || n < 1 || heads < 1) return HCMIX_ERR_INVALID_VALUE;
  if (batch > kMaxRows / n || heads > 1024) return HCMIX_ERR_INVALID_VALUE;
  if (head_dim != 64 || n % 32 != 0 || n > 256) return HCMIX_ERR_UNSUPPORTED;
  return HCMIX_OK;
}

hcmix_status hcmix_attention_forward(int64_t batch, int64_t n, int32_t heads, int32_t head_dim,
                                     const void* qkv, void* out, float* lse, void* stream) {
  if (!qkv || !out || !lse) return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_attention(batch, n, heads, head_dim);
  if (st != HCMIX_OK) return st;
  const size_t rows = (size_t)(batch * n);
  const Span ins[1] = {{qkv, rows * 3 * heads * 64 * sizeof(bf16)}};
  const Span outs[2] = {{out, rows * heads * 64 * sizeof(bf16)},
                        {lse, rows * heads * sizeof(float)}};
  st = check_spans(ins, 1, outs, 1, 16);
  if (st != HCMIX_OK) return st;
  st = check_spans(ins, 1, outs + 1, 1, 4);
  if (st != HCMIX_OK) return st;
  if (overlaps(out, outs[0].n, lse, outs[1].n)) return HCMIX_ERR_INVALID_VALUE;
  hipError_t e = launch_attention_fwd_bf16((const bf16*)qkv, (bf16*)out, lse, (int)batch, (int)n,
                                           heads, (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

hcmix_status hcmix_attention_backward(int64_t batch, int64_t n, int32_t heads, int32_t head_dim,
                                      const void* qkv, const void* out, const float* lse,
                                      const void* dout, void* dqkv, void* stream) {
  if (!qkv || !out || !lse || !dout || !dqkv) return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_attention(batch, n, heads, head_dim);
  if (st != HCMIX_OK) return st;
  const size_t rows = (size_t)(batch * n);
  const size_t act = rows * heads * 64 * sizeof(bf16);
  const Span ins[3] = {{qkv, 3 * act}, {out, act}, {dout, act}};
  const Span outs[1] = {{dqkv, 3 * act}};
  st = check_spans(ins, 3, outs, 1, 16);
  if (st != HCMIX_OK) return st;
  if (!aligned(lse, 4)) return HCMIX_ERR_UNSUPPORTED;
  if (overlaps(dqkv, 3 * act, lse, rows * heads * sizeof(float))) return HCMIX_ERR_INVALID_VALUE;
  hipError_t e = launch_attention_bwd_bf16((const bf16*)qkv, (const bf16*)out, lse,
                                           (const bf16*)dout, (bf16*)dqkv, (int)batch, (int)n,
                                           heads, (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

// Shape checks of the language-model entry points.
hcmix_status check_lm(int64_t rows, int64_t width, int32_t vocab) {
  if (rows < 1 || width < 1 || vocab < 1) return HCMIX_ERR_INVALID_VALUE;
  if (rows > kMaxRows || vocab > (1 << 20) || width > (1 << 16)) return HCMIX_ERR_INVALID_VALUE;
  if (width % 64 != 0) return HCMIX_ERR_UNSUPPORTED;
  return HCMIX_OK;
}

hcmix_status hcmix_embedding_forward(int64_t rows, int64_t width, int32_t vocab, const void* table,
                                     const int32_t* tokens, void* x, void* stream) {
  if (!table || !tokens || !x) return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_lm(rows, width, vocab);
  if (st != HCMIX_OK) return st;
  const Span ins[2] = {{table, (size_t)vocab * width * sizeof(bf16)},
                       {tokens, (size_t)rows * sizeof(int32_t)}};
  const Span outs[1] = {{x, (size_t)rows * width * sizeof(bf16)}};
  st = check_spans(ins, 2, outs, 1, 4);
  if (st != HCMIX_OK) return st;
  if (!aligned(table, 16) || !aligned(x, 16)) return HCMIX_ERR_UNSUPPORTED;
  hipError_t e = launch_embedding_fwd((const bf16*)table, (const int*)tokens, (bf16*)x, (int)rows,
                                      (int)width, vocab, (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

size_t hcmix_embedding_backward_workspace_bytes(int64_t rows, int64_t width, int32_t vocab) {
  if (check_lm(rows, width, vocab) != HCMIX_OK) return 0;
  return align256(embedding_workspace_bytes((int)rows, (int)width, vocab));
}

hcmix_status hcmix_embedding_backward(int64_t rows, int64_t width, int32_t vocab,
                                      const int32_t* tokens, const void* dx, float* dtable,
                                      int32_t accumulate, void* workspace, size_t workspace_bytes,
                                      void* stream) {
  if (!tokens || !dx || !dtable || !workspace) return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_lm(rows, width, vocab);
  if (st != HCMIX_OK) return st;
  const size_t need = embedding_workspace_bytes((int)rows, (int)width, vocab);
  if (workspace_bytes < need) return HCMIX_ERR_INVALID_VALUE;
  const Span ins[2] = {{tokens, (size_t)rows * sizeof(int32_t)},
                       {dx, (size_t)rows * width * sizeof(bf16)}};
  const Span outs[2] = {{dtable, (size_t)vocab * width * sizeof(float)}, {workspace, need}};
  st = check_spans(ins, 2, outs, 2, 4);
  if (st != HCMIX_OK) return st;
  if (!aligned(dx, 16) || !aligned(workspace, 256)) return HCMIX_ERR_UNSUPPORTED;
  hipError_t e = launch_embedding_bwd((const int*)tokens, (const bf16*)dx, dtable,
                                      accumulate != 0, (float*)workspace, (int)rows, (int)width,
                                      vocab, (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

size_t hcmix_head_cross_entropy_workspace_bytes(int64_t rows, int32_t vocab) {
  if (rows < 1 || rows > kMaxRows || vocab < 32 || vocab > 256 || vocab % 32) return 0;
  return align256(head_workspace_bytes((int)rows, vocab));
}

hcmix_status hcmix_head_cross_entropy(int64_t rows, int64_t width, int32_t vocab, const void* x,
                                      const void* w, const float* bias, const int32_t* targets,
                                      float scale, float* loss, void* dlogits, float* dbias,
                                      void* workspace, size_t workspace_bytes, void* stream) {
  if (!x || !w || !bias || !targets || !loss || !dlogits) return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_lm(rows, width, vocab);
  if (st != HCMIX_OK) return st;
  if (vocab % 32 != 0 || vocab > 256) return HCMIX_ERR_UNSUPPORTED;
  const size_t need = dbias ? head_workspace_bytes((int)rows, vocab) : 0;
  if (dbias && (!workspace || workspace_bytes < need)) return HCMIX_ERR_INVALID_VALUE;
  const Span ins[4] = {{x, (size_t)rows * width * sizeof(bf16)},
                       {w, (size_t)vocab * width * sizeof(bf16)},
                       {bias, (size_t)vocab * sizeof(float)},
                       {targets, (size_t)rows * sizeof(int32_t)}};
  const Span outs[4] = {{loss, (size_t)rows * sizeof(float)},
                        {dlogits, (size_t)rows * vocab * sizeof(bf16)},
                        {dbias, dbias ? (size_t)vocab * sizeof(float) : 0},
                        {workspace, need}};
  st = check_spans(ins, 4, outs, 4, 4);
  if (st != HCMIX_OK) return st;
  if (!aligned(x, 16) || !aligned(w, 16) || !aligned(bias, 16) || !aligned(dlogits, 16))
    return HCMIX_ERR_UNSUPPORTED;
  if (dbias && !aligned(workspace, 256)) return HCMIX_ERR_UNSUPPORTED;
  hipError_t e = launch_head_ce((const bf16*)x, (const bf16*)w, bias, (const int*)targets, scale,
                                loss, (bf16*)dlogits, dbias, (float*)workspace, (int)rows,
                                (int)width, vocab, (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

size_t hcmix_head_backward_workspace_bytes(int64_t rows, int64_t width, int32_t vocab) {
  if (check_lm(rows, width, vocab) != HCMIX_OK || vocab % 32) return 0;
  return align256(head_backward_workspace_bytes((int)rows, (int)width, vocab));
}

hcmix_status hcmix_head_backward(int64_t rows, int64_t width, int32_t vocab, const void* x,
                                 const void* w, const void* dlogits, void* gx, float* dw,
                                 int32_t accumulate, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  // x is read only for dw
  if (!w || !dlogits || (!gx && !dw) || (dw && !x)) return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_lm(rows, width, vocab);
  if (st != HCMIX_OK) return st;
  if (vocab % 32 != 0) return HCMIX_ERR_UNSUPPORTED;
  const size_t need = dw ? head_backward_workspace_bytes((int)rows, (int)width, vocab) : 0;
  if (dw && (!workspace || workspace_bytes < need)) return HCMIX_ERR_INVALID_VALUE;
  const Span ins[3] = {{w, (size_t)vocab * width * sizeof(bf16)},
                       {dlogits, (size_t)rows * vocab * sizeof(bf16)},
                       {dw ? x : w, dw ? (size_t)rows * width * sizeof(bf16) : 0}};
  const Span outs[3] = {{gx, gx ? (size_t)rows * width * sizeof(bf16) : 0},
                        {dw, dw ? (size_t)vocab * width * sizeof(float) : 0},
                        {workspace, need}};
  st = check_spans(ins, 3, outs, 3, 4);
  if (st != HCMIX_OK) return st;
  if ((dw && !aligned(x, 16)) || !aligned(w, 16) || !aligned(dlogits, 16) ||
      (gx && !aligned(gx, 16)))
    return HCMIX_ERR_UNSUPPORTED;
  if (dw && !aligned(workspace, 256)) return HCMIX_ERR_UNSUPPORTED;
  hipError_t e = launch_head_backward((const bf16*)x, (const bf16*)w, (const bf16*)dlogits,
                                      (bf16*)gx, dw, accumulate != 0, (float*)workspace,
                                      (int)rows, (int)width, vocab, (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

// Decode cache: two [batch][width] buffers that pass each layer's output to
// the next, then per layer a ring of the inputs that a later position takes as
// its partner: a hypercube layer of dimension d needs the input at pos - 2^d,
// recorded at a position with bit d clear and read 2^d positions later, so
// 2^d slots indexed by pos mod 2^d; the local layer reads pos - 1 and records
// pos in the same step, so 2 slots indexed by pos mod 2.
int64_t ring_slots(int32_t code, int64_t n) {
  return code == HCMIX_LAYER_NEAR ? 2 : (int64_t)1 << hcmix_dim(code, n);
}

size_t hcmix_decode_cache_bytes(int64_t batch, int64_t n, int64_t width, int32_t num_layers,
                                const int32_t* layers, int32_t dtype) {
  if (!layers || num_layers < 1 || num_layers > kMaxLayers) return 0;
  int64_t slots = 2;
  for (int l = 0; l < num_layers; l++) {
    if (check_shape(batch, n, width, layers[l], HCMIX_CAUSAL, dtype) != HCMIX_OK) return 0;
    slots += ring_slots(layers[l], n);
  }
  return align256((size_t)slots * batch * width * elem_size(dtype));
}

hcmix_status hcmix_decode_step(int64_t batch, int64_t n, int64_t width, int32_t num_layers,
                               const int32_t* layers, int32_t dtype, int64_t pos, const void* x,
                               const void* const* w_self, const void* const* w_off, void* cache,
                               size_t cache_bytes, void* y, void* stream) {
  if (!layers || !x || !w_self || !w_off || !cache || !y) return HCMIX_ERR_INVALID_VALUE;
  if (num_layers < 1 || num_layers > kMaxLayers) return HCMIX_ERR_INVALID_VALUE;
  for (int l = 0; l < num_layers; l++) {
    hcmix_status st = check_shape(batch, n, width, layers[l], HCMIX_CAUSAL, dtype);
    if (st != HCMIX_OK) return st;
    if (!w_self[l] || !w_off[l]) return HCMIX_ERR_INVALID_VALUE;
  }
  if (pos < 0 || pos >= n) return HCMIX_ERR_INVALID_VALUE;
  const size_t need = hcmix_decode_cache_bytes(batch, n, width, num_layers, layers, dtype);
  if (cache_bytes < need) return HCMIX_ERR_INVALID_VALUE;
  const size_t es = elem_size(dtype);
  const size_t row = (size_t)(batch * width) * es, wgt = (size_t)(width * width) * es;
  const size_t al = dtype == HCMIX_BF16 ? 16 : 4;
  // outputs: y and the cache; inputs: x and every weight
  const Span outs[2] = {{y, row}, {cache, need}};
  {
    const Span ins[1] = {{x, row}};
    hcmix_status st = check_spans(ins, 1, outs, 2, al);
    if (st != HCMIX_OK) return st;
  }
  for (int l = 0; l < num_layers; l++) {
    const Span ins[2] = {{w_self[l], wgt}, {w_off[l], wgt}};
    hcmix_status st = check_spans(ins, 2, outs, 2, al);
    if (st != HCMIX_OK) return st;
  }
  if (!aligned(cache, 256)) return HCMIX_ERR_UNSUPPORTED;

  // slot k of the cache: [batch][width] elements at offset k * batch * width
  const int64_t slot = batch * width;
  char* c = (char*)cache;
  auto at = [&](int64_t k) { return c + (size_t)(k * slot) * es; };
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = hipSuccess;
  int64_t ring = 2;   // first slot of layer l's ring (after the two pass-on buffers)
  for (int l = 0; l < num_layers && e == hipSuccess; l++) {
    const int32_t code = layers[l];
    const int64_t slots = ring_slots(code, n);
    const int d = hcmix_dim(code, n);
    const void* partner = nullptr;
    void* record = nullptr;
    if (code == HCMIX_LAYER_NEAR) {
      if (pos >= 1) partner = at(ring + (pos - 1) % 2);
      record = at(ring + pos % 2);
    } else if ((pos >> d) & 1) {
      partner = at(ring + pos % slots);   // recorded at pos - 2^d
    } else {
      record = at(ring + pos % slots);    // read at pos + 2^d
    }
    const void* in = l == 0 ? x : at(l & 1);
    void* out = l == num_layers - 1 ? y : at((l + 1) & 1);
    if (dtype == HCMIX_BF16) {
      DecodeLayerArgs a = {};
      a.x_in = (const bf16*)in;
      a.x_partner = (const bf16*)partner;
      a.w_self = (const bf16*)w_self[l];
      a.w_off = (const bf16*)w_off[l];
      a.out = (bf16*)out;
      a.record = (bf16*)record;
      a.in_stride = a.partner_stride = a.out_stride = a.rec_stride = width;
      a.batch = (int)batch;
      a.width = (int)width;
      e = mfma_path(dtype, width) ? launch_decode_bf16(a, s) : launch_decode_bf16_fma(a, s);
    } else {
      DecodeLayerArgsF32 a = {};
      a.x_in = (const float*)in;
      a.x_partner = (const float*)partner;
      a.w_self = (const float*)w_self[l];
      a.w_off = (const float*)w_off[l];
      a.out = (float*)out;
      a.record = (float*)record;
      a.in_stride = a.partner_stride = a.out_stride = a.rec_stride = width;
      a.batch = (int)batch;
      a.width = (int)width;
      e = launch_decode_f32(a, s);
    }
    ring += slots;
  }
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

// ---- channel-shared mixing stack ----

// Shape checks of the channel-shared entry points (layer codes checked per
// layer by the caller).
hcmix_status check_shared(int64_t batch, int64_t n, int64_t width, int32_t num_layers,
                          const int32_t* layers, int32_t mode, int32_t dtype) {
  if (num_layers < 1 || num_layers > kMaxLayers) return HCMIX_ERR_INVALID_VALUE;
  for (int l = 0; l < num_layers; l++) {
    hcmix_status st = check_shape(batch, n, width, layers[l], mode, HCMIX_F32);
    if (st != HCMIX_OK) return st;
  }
  if (dtype != HCMIX_F32 && dtype != HCMIX_BF16) return HCMIX_ERR_INVALID_VALUE;
  if (!shared_stack_eligible(n, width, num_layers, (int32_t)elem_size(dtype)))
    return HCMIX_ERR_UNSUPPORTED;
  return HCMIX_OK;
}

hcmix_status hcmix_shared_stack_forward(int64_t batch, int64_t n, int64_t width,
                                        int32_t num_layers, const int32_t* layers, int32_t mode,
                                        int32_t dtype, const void* x, const float* const* tables,
                                        void* const* xs, void* stream) {
  if (!x || !layers || !tables || !xs) return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_shared(batch, n, width, num_layers, layers, mode, dtype);
  if (st != HCMIX_OK) return st;
  const size_t act = (size_t)(batch * n * width) * elem_size(dtype);
  const size_t tab = (size_t)(n * n) * sizeof(float);
  for (int l = 0; l < num_layers; l++) {
    if (!tables[l] || !aligned(tables[l], 4)) return tables[l] ? HCMIX_ERR_UNSUPPORTED
                                                               : HCMIX_ERR_INVALID_VALUE;
    const Span ins[1] = {{x, act}};
    const Span outs[1] = {{xs[l], act}};
    st = check_spans(ins, 1, outs, 1, 16);
    if (st != HCMIX_OK) return st;
    for (int j = 0; j < num_layers; j++) {
      if (j != l && overlaps(xs[l], act, xs[j], act)) return HCMIX_ERR_INVALID_VALUE;
      if (overlaps(xs[l], act, tables[j], tab)) return HCMIX_ERR_INVALID_VALUE;
    }
  }
  SharedFwdArgs a = {};
  a.x0 = x;
  for (int l = 0; l < num_layers; l++) {
    a.xs[l] = xs[l];
    a.tab[l] = tables[l];
    a.dim[l] = hcmix_dim(layers[l], n);   // -1 for the local layer
  }
  a.n = (int)n;
  a.width = (int)width;
  a.num_layers = num_layers;
  a.bidir = mode == HCMIX_BIDIR;
  hipError_t e = launch_shared_forward(a, (int)batch, (int)elem_size(dtype), (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

size_t hcmix_shared_stack_backward_workspace_bytes(int64_t batch, int64_t n, int64_t width,
                                                   int32_t num_layers, int32_t dtype) {
  if (num_layers < 1 || num_layers > kMaxLayers) return 0;
  if (dtype != HCMIX_F32 && dtype != HCMIX_BF16) return 0;
  if (check_shape(batch, n, width, 0, HCMIX_BIDIR, HCMIX_F32) != HCMIX_OK) return 0;
  if (!shared_stack_eligible(n, width, num_layers, (int32_t)elem_size(dtype))) return 0;
  return align256(shared_partial_bytes(batch, n, width, num_layers, (int32_t)elem_size(dtype)));
}

hcmix_status hcmix_shared_stack_backward(int64_t batch, int64_t n, int64_t width,
                                         int32_t num_layers, const int32_t* layers, int32_t mode,
                                         int32_t dtype, const void* const* xs_in,
                                         const float* const* tables, const void* dy, void* dx,
                                         float* const* dtables, int32_t accumulate,
                                         void* workspace, size_t workspace_bytes, void* stream) {
  if (!layers || !xs_in || !tables || !dy || !dx || !dtables || !workspace)
    return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_shared(batch, n, width, num_layers, layers, mode, dtype);
  if (st != HCMIX_OK) return st;
  const size_t need =
      shared_partial_bytes(batch, n, width, num_layers, (int32_t)elem_size(dtype));
  if (workspace_bytes < need) return HCMIX_ERR_INVALID_VALUE;
  const size_t act = (size_t)(batch * n * width) * elem_size(dtype);
  const size_t tab = (size_t)(n * n) * sizeof(float);
  // outputs: dx, the workspace, every dtables[l]; inputs: dy, every xs_in[l]
  // and tables[l]; no output may overlap an input or another output
  const Span fixed_outs[2] = {{dx, act}, {workspace, need}};
  {
    const Span ins[1] = {{dy, act}};
    st = check_spans(ins, 1, fixed_outs, 2, 16);
    if (st != HCMIX_OK) return st;
  }
  for (int l = 0; l < num_layers; l++) {
    if (!xs_in[l] || !tables[l] || !dtables[l]) return HCMIX_ERR_INVALID_VALUE;
    const Span ins[2] = {{xs_in[l], act}, {tables[l], tab}};
    const Span outs[3] = {fixed_outs[0], fixed_outs[1], {dtables[l], tab}};
    st = check_spans(ins, 2, outs, 3, 4);
    if (st != HCMIX_OK) return st;
    if (!aligned(xs_in[l], 16)) return HCMIX_ERR_UNSUPPORTED;
    for (int j = 0; j < num_layers; j++) {
      if (j == l) continue;
      if (overlaps(dtables[l], tab, dtables[j], tab) || overlaps(dtables[l], tab, tables[j], tab) ||
          overlaps(dtables[l], tab, xs_in[j], act))
        return HCMIX_ERR_INVALID_VALUE;
      if (overlaps(dx, act, xs_in[j], act) || overlaps(dx, act, tables[j], tab))
        return HCMIX_ERR_INVALID_VALUE;
    }
  }
  if (!aligned(workspace, 256)) return HCMIX_ERR_UNSUPPORTED;
  SharedBwdArgs a = {};
  SharedReduceArgs r = {};
  for (int l = 0; l < num_layers; l++) {
    a.xs[l] = xs_in[l];
    a.tab[l] = tables[l];
    a.dim[l] = r.dim[l] = hcmix_dim(layers[l], n);
    r.dt[l] = dtables[l];
  }
  a.dy = dy;
  a.dx = dx;
  a.partial = (float*)workspace;
  a.n = r.n = (int)n;
  a.width = (int)width;
  a.num_layers = r.num_layers = num_layers;
  a.bidir = r.bidir = mode == HCMIX_BIDIR;
  r.partial = (const float*)workspace;
  r.accumulate = accumulate != 0;
  hipError_t e = launch_shared_backward(a, r, (int)batch, (int)elem_size(dtype),
                                        (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

// ---- linear maps (the hybrids' attention projections) ----

hcmix_status check_linear(int64_t rows, int64_t in_width, int64_t out_width) {
  if (rows < 1 || in_width < 1 || out_width < 1) return HCMIX_ERR_INVALID_VALUE;
  if (rows > kMaxRows || in_width > (1 << 16) || out_width > (1 << 16))
    return HCMIX_ERR_INVALID_VALUE;
  if (rows % 2 || in_width % 64 || out_width % 64) return HCMIX_ERR_UNSUPPORTED;
  return HCMIX_OK;
}

hcmix_status hcmix_linear_forward(int64_t rows, int64_t in_width, int64_t out_width,
                                  const void* x, const void* w, void* y, void* stream) {
  if (!x || !w || !y) return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_linear(rows, in_width, out_width);
  if (st != HCMIX_OK) return st;
  const Span ins[2] = {{x, (size_t)rows * in_width * sizeof(bf16)},
                       {w, (size_t)out_width * in_width * sizeof(bf16)}};
  const Span outs[1] = {{y, (size_t)rows * out_width * sizeof(bf16)}};
  st = check_spans(ins, 2, outs, 1, 16);
  if (st != HCMIX_OK) return st;
  // y = x W^T: W's rows are the output columns, contiguous over the input
  hipError_t e = launch_gemm_bf16((const bf16*)x, (const bf16*)w, (bf16*)y, (int)rows,
                                  (int)in_width, (int)out_width, (int)in_width, (int)out_width,
                                  /*transpose_b=*/false, (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

size_t hcmix_linear_backward_workspace_bytes(int64_t rows, int64_t in_width, int64_t out_width) {
  if (check_linear(rows, in_width, out_width) != HCMIX_OK) return 0;
  return align256(head_backward_workspace_bytes((int)rows, (int)in_width, (int)out_width));
}

hcmix_status hcmix_linear_backward(int64_t rows, int64_t in_width, int64_t out_width,
                                   const void* x, const void* w, const void* dy, void* dx,
                                   float* dw, int32_t accumulate, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  if (!w || !dy || (!dx && !dw) || (dw && !x)) return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_linear(rows, in_width, out_width);
  if (st != HCMIX_OK) return st;
  const size_t need =
      dw ? head_backward_workspace_bytes((int)rows, (int)in_width, (int)out_width) : 0;
  if (dw && (!workspace || workspace_bytes < need)) return HCMIX_ERR_INVALID_VALUE;
  const Span ins[3] = {{w, (size_t)out_width * in_width * sizeof(bf16)},
                       {dy, (size_t)rows * out_width * sizeof(bf16)},
                       {dw ? x : w, dw ? (size_t)rows * in_width * sizeof(bf16) : 0}};
  const Span outs[3] = {{dx, dx ? (size_t)rows * in_width * sizeof(bf16) : 0},
                        {dw, dw ? (size_t)out_width * in_width * sizeof(float) : 0},
                        {workspace, need}};
  st = check_spans(ins, 3, outs, 3, 4);
  if (st != HCMIX_OK) return st;
  if ((dw && !aligned(x, 16)) || !aligned(w, 16) || !aligned(dy, 16) || (dx && !aligned(dx, 16)))
    return HCMIX_ERR_UNSUPPORTED;
  if (dw && !aligned(workspace, 256)) return HCMIX_ERR_UNSUPPORTED;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = hipSuccess;
  // dx = dy W: W read as [out][in], rows k, so transposed into the tiles
  if (dx)
    e = launch_gemm_bf16((const bf16*)dy, (const bf16*)w, (bf16*)dx, (int)rows, (int)out_width,
                         (int)in_width, (int)in_width, (int)in_width, /*transpose_b=*/true, s);
  // dW = dy^T x, row ranges summed in a fixed order
  if (e == hipSuccess && dw)
    e = launch_head_backward((const bf16*)x, (const bf16*)w, (const bf16*)dy, nullptr, dw,
                             accumulate != 0, (float*)workspace, (int)rows, (int)in_width,
                             (int)out_width, s);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

// ---- field coupling (Section 3.4's dynamics variant) ----

hcmix_status check_field(int64_t batch, int64_t n, int64_t width, int32_t coord_dim, float tau,
                         int32_t scaled) {
  if (batch < 1 || n < 1 || width < 1 || coord_dim < 1) return HCMIX_ERR_INVALID_VALUE;
  if (!(tau >= 0x1p-24f && tau <= 0x1p24f) || (scaled != 0 && scaled != 1))
    return HCMIX_ERR_INVALID_VALUE;
  if (width > kMaxWidth || batch > kMaxRows / n || batch * n > kMaxElems / width)
    return HCMIX_ERR_INVALID_VALUE;
  if (n > 256 || coord_dim > 64 || width % 64 != 0) return HCMIX_ERR_UNSUPPORTED;
  return HCMIX_OK;
}

size_t hcmix_field_workspace_bytes(int64_t batch, int64_t n, int32_t coord_dim) {
  if (batch < 1 || n < 1 || n > 256 || coord_dim < 1 || coord_dim > 64) return 0;
  if (batch > kMaxRows / n) return 0;
  return field_workspace_bytes((int)batch, (int)n, coord_dim);
}

hcmix_status hcmix_field_forward(int64_t batch, int64_t n, int64_t width, int32_t coord_dim,
                                 float tau, int32_t scaled, const float* p, const void* x,
                                 void* y, float* row_mean, float* lse, float* partners,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  if (!p || !x || !y || !row_mean || !lse) return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_field(batch, n, width, coord_dim, tau, scaled);
  if (st != HCMIX_OK) return st;
  const size_t need = hcmix_field_workspace_bytes(batch, n, coord_dim);
  if (!workspace || workspace_bytes < need) return HCMIX_ERR_INVALID_VALUE;
  const size_t rows = (size_t)(batch * n), act = rows * width * sizeof(bf16);
  const size_t stat = rows * sizeof(float);
  const Span ins[2] = {{p, rows * coord_dim * sizeof(float)}, {x, act}};
  const Span outs[5] = {{y, act}, {row_mean, stat}, {lse, stat}, {partners, partners ? stat : 0},
                        {workspace, need}};
  st = check_spans(ins, 2, outs, 5, 4);
  if (st != HCMIX_OK) return st;
  if (!aligned(x, 16) || !aligned(y, 16) || !aligned(workspace, 256)) return HCMIX_ERR_UNSUPPORTED;
  hipError_t e = launch_field_fwd(p, (const bf16*)x, (bf16*)y, row_mean, lse, partners, workspace,
                                  (int)batch, (int)n, coord_dim, (int)width, 1.f / tau, scaled,
                                  (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

hcmix_status hcmix_field_backward(int64_t batch, int64_t n, int64_t width, int32_t coord_dim,
                                  float tau, int32_t scaled, const float* p, const void* x,
                                  const float* row_mean, const float* lse, const void* dy,
                                  float* dp, void* dx, int32_t reuse_table, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  if (!p || !x || !row_mean || !lse || !dy || !dp || !dx) return HCMIX_ERR_INVALID_VALUE;
  if (reuse_table != 0 && reuse_table != 1) return HCMIX_ERR_INVALID_VALUE;
  hcmix_status st = check_field(batch, n, width, coord_dim, tau, scaled);
  if (st != HCMIX_OK) return st;
  const size_t need = hcmix_field_workspace_bytes(batch, n, coord_dim);
  if (!workspace || workspace_bytes < need) return HCMIX_ERR_INVALID_VALUE;
  const size_t rows = (size_t)(batch * n), act = rows * width * sizeof(bf16);
  const size_t stat = rows * sizeof(float), coords = rows * coord_dim * sizeof(float);
  const Span ins[5] = {{p, coords}, {x, act}, {row_mean, stat}, {lse, stat}, {dy, act}};
  const Span outs[3] = {{dp, coords}, {dx, act}, {workspace, need}};
  st = check_spans(ins, 5, outs, 3, 4);
  if (st != HCMIX_OK) return st;
  if (!aligned(x, 16) || !aligned(dy, 16) || !aligned(dx, 16) || !aligned(workspace, 256))
    return HCMIX_ERR_UNSUPPORTED;
  hipError_t e = launch_field_bwd(p, (const bf16*)x, row_mean, lse, (const bf16*)dy, dp,
                                  (bf16*)dx, workspace, reuse_table, (int)batch, (int)n, coord_dim,
                                  (int)width, 1.f / tau, scaled, (hipStream_t)stream);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}
