// C ABI of libhcmix.so: argument validation and kernel dispatch.
// Every check runs before anything is enqueued, so a rejected call has no
// effect; there is one kernel path per dtype and no fallback.
#include "hcmix.h"
#include "hcmix_internal.h"

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

size_t elem_size(int32_t dtype) { return dtype == HCMIX_BF16 ? 2 : 4; }

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b;
  return pa < pb + nb && pb < pa + na;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Shape checks shared by forward and backward; returns HCMIX_OK or the error.
hcmix_status check_shape(int64_t batch, int64_t n, int64_t width, int32_t layer, int32_t mode,
                         int32_t dtype) {
  if (hcmix_dim(layer, n) < 0) return HCMIX_ERR_INVALID_VALUE;
  if (batch < 1 || width < 1) return HCMIX_ERR_INVALID_VALUE;
  if (mode != HCMIX_BIDIR && mode != HCMIX_CAUSAL) return HCMIX_ERR_INVALID_VALUE;
  if (dtype != HCMIX_F32 && dtype != HCMIX_BF16) return HCMIX_ERR_INVALID_VALUE;
  if (batch > kMaxRows / n) return HCMIX_ERR_INVALID_VALUE;
  if (batch * n > kMaxElems / width) return HCMIX_ERR_INVALID_VALUE;
  if (dtype == HCMIX_BF16 && width % 64 != 0) return HCMIX_ERR_UNSUPPORTED;
  return HCMIX_OK;
}

// Backward workspace (bf16): the split-K partial sums of the weight gradients,
// [splits][2][width][width] fp32.
size_t align256(size_t v) { return (v + 255) / 256 * 256; }

size_t workspace_bytes_checked(int64_t batch, int64_t n, int64_t width, int32_t dtype) {
  if (dtype != HCMIX_BF16) return 0;
  const int splits = dw_bf16_splits((int)(batch * n), (int)width);
  return align256((size_t)splits * 2 * width * width * sizeof(float));
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
  if (overlaps(y, act, x, act) || overlaps(y, act, w_self, wgt) || overlaps(y, act, w_off, wgt))
    return HCMIX_ERR_INVALID_VALUE;
  const size_t al = dtype == HCMIX_BF16 ? 16 : 4;
  if (!aligned(x, al) || !aligned(w_self, al) || !aligned(w_off, al) || !aligned(y, al))
    return HCMIX_ERR_UNSUPPORTED;

  const int d = hcmix_dim(layer, n);
  const int rows = (int)(batch * n), w = (int)width;
  const int bidir = mode == HCMIX_BIDIR;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e;
  if (dtype == HCMIX_BF16)
    e = launch_mix_bf16((const bf16*)x, (const bf16*)w_self, (const bf16*)w_off, (bf16*)y, rows,
                        w, d, /*partner_lower=*/bidir, /*partner_upper=*/1,
                        /*transpose_b=*/false, s);
  else
    e = launch_mix_f32((const float*)x, (const float*)w_self, (const float*)w_off, (float*)y,
                       rows, w, d, bidir, 1, /*transpose_w=*/false, s);
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

size_t hcmix_backward_workspace_bytes(int64_t batch, int64_t n, int64_t width, int32_t dtype) {
  if (check_shape(batch, n, width, 0, HCMIX_BIDIR, dtype) != HCMIX_OK) return 0;
  return workspace_bytes_checked(batch, n, width, dtype);
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
  const size_t need = workspace_bytes_checked(batch, n, width, dtype);
  if (need > 0 && (!workspace || workspace_bytes < need)) return HCMIX_ERR_INVALID_VALUE;
  const size_t es = elem_size(dtype);
  const size_t act = (size_t)(batch * n * width) * es, wgt = (size_t)(width * width) * es;
  const size_t gw = (size_t)(width * width) * sizeof(float);
  // outputs must not overlap each other or any input
  const void* outs[4] = {dx, dw_self, dw_off, workspace};
  const size_t out_n[4] = {act, gw, gw, need};
  const void* ins[4] = {x, w_self, w_off, dy};
  const size_t in_n[4] = {act, wgt, wgt, act};
  for (int i = 0; i < 4; i++) {
    if (out_n[i] == 0) continue;
    for (int j = 0; j < 4; j++)
      if (overlaps(outs[i], out_n[i], ins[j], in_n[j])) return HCMIX_ERR_INVALID_VALUE;
    for (int j = i + 1; j < 4; j++)
      if (out_n[j] && overlaps(outs[i], out_n[i], outs[j], out_n[j]))
        return HCMIX_ERR_INVALID_VALUE;
  }
  const size_t al = dtype == HCMIX_BF16 ? 16 : 4;
  if (!aligned(x, al) || !aligned(w_self, al) || !aligned(w_off, al) || !aligned(dy, al) ||
      !aligned(dx, al) || !aligned(dw_self, 16) || !aligned(dw_off, 16))
    return HCMIX_ERR_UNSUPPORTED;
  if (need > 0 && !aligned(workspace, 256)) return HCMIX_ERR_UNSUPPORTED;

  const int d = hcmix_dim(layer, n);
  const int rows = (int)(batch * n), w = (int)width;
  const int bidir = mode == HCMIX_BIDIR;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e;
  if (dtype == HCMIX_BF16) {
    float* partial = (float*)workspace;
    e = launch_mix_bf16((const bf16*)dy, (const bf16*)w_self, (const bf16*)w_off, (bf16*)dx,
                        rows, w, d, /*partner_lower=*/1, /*partner_upper=*/bidir,
                        /*transpose_b=*/true, s);
    if (e == hipSuccess)
      e = launch_dw_bf16((const bf16*)x, (const bf16*)dy, partial, dw_self, dw_off, rows, w, d,
                         bidir, accumulate != 0, s);
  } else {
    e = launch_mix_f32((const float*)dy, (const float*)w_self, (const float*)w_off, (float*)dx,
                       rows, w, d, 1, bidir, /*transpose_w=*/true, s);
    if (e == hipSuccess)
      e = launch_dw_f32((const float*)x, (const float*)dy, dw_self, dw_off, rows, w, d, bidir,
                        accumulate != 0, s);
  }
  return e == hipSuccess ? HCMIX_OK : hip_fail(e);
}

}  // extern "C"
