// Decode step: one new position `pos` of every window through every layer.
// All windows are at the same position, so each layer is one small dense
// product over the batch:
//   y[b] = W_self x[b] + m(pos) W_off x_partner[b]
// with the partner's layer input read from the cache.  The kernel of layer l
// reads its input at `pos` (from the caller's x or the buffer the previous
// layer wrote), the partner's from that layer's ring of earlier inputs, may
// record its own input into the ring for a later position, and writes its
// output to the other pass-on buffer (or to y after the last layer); the
// buffers a launch writes are never ones it reads.
#include "device_common.h"
#include "hcmix_internal.h"

namespace hcmix {

namespace {

// bf16: one block per 16 output columns x 16 windows (128 blocks at width 512
// and 64 windows), 16x16x32 MFMAs with the weights as the A operand, so the
// result is C[o][b].  The 4 waves split the contraction in 32-wide steps
// (wave w takes steps w, w + 4, ...); each wave loads the self and partner
// operands of CH steps before any of their MFMAs, so at width 512 every load of
// the block is in flight at once and a layer costs one memory latency.  The
// wave partials are summed through LDS in wave order.  Against 32 x 32 blocks
// of 8 waves (32 blocks at that shape) this spreads the loads over four times
// as many CUs: 6.3 -> 4.1 us per layer launch in a graph, with partners.
constexpr int DEC_WAVES = 4;
template <int CH>
__global__ __launch_bounds__(64 * DEC_WAVES) void decode_bf16_kernel(DecodeLayerArgs a) {
  __shared__ f32x4 part[DEC_WAVES][64];
  // `wave` and `has_partner` are wave-uniform and must be known so: an MFMA
  // under a lane mask (EXEC) still writes its whole result, so every MFMA
  // guard below has to be a scalar branch.
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool has_partner = a.x_partner != nullptr;
  const int o0 = blockIdx.x * 16, b0 = blockIdx.y * 16;
  const int w = a.width;
  const int b = min(b0 + (lane & 15), a.batch - 1);      // clamped; stores are masked
  const int q = lane >> 4;                               // K piece 8q .. 8q + 7 of a step
  const bf16* xin = a.x_in + (size_t)b * a.in_stride;
  const bf16* xp = has_partner ? a.x_partner + (size_t)b * a.partner_stride : a.x_in;
  const bf16* ws = a.w_self + (size_t)(o0 + (lane & 15)) * w;
  const bf16* wo = a.w_off + (size_t)(o0 + (lane & 15)) * w;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  const int ksteps = w / 32;
  for (int kb = wave; kb < ksteps; kb += DEC_WAVES * CH) {
    bf16x8 sw[CH], sx[CH], pw[CH], px[CH];
#pragma unroll
    for (int j = 0; j < CH; j++) {
      const int k = kb + DEC_WAVES * j;
      const int k0 = (k < ksteps ? k : 0) * 32 + 8 * q;   // clamped; the MFMA is skipped
      sw[j] = *(const bf16x8*)(ws + k0);
      sx[j] = *(const bf16x8*)(xin + k0);
      if (has_partner) {
        pw[j] = *(const bf16x8*)(wo + k0);
        px[j] = *(const bf16x8*)(xp + k0);
      }
    }
#pragma unroll
    for (int j = 0; j < CH; j++) {
      if (kb + DEC_WAVES * j >= ksteps) continue;
      acc = mfma16(sw[j], sx[j], acc);
      if (has_partner) acc = mfma16(pw[j], px[j], acc);
    }
  }
  part[wave][lane] = acc;
  // the layer records its input for a later position: this block's 16 columns
  if (a.record && wave == 0 && b0 + (lane & 15) < a.batch) {
    const int c = o0 + 4 * q;
    *(bf16x4*)(a.record + (size_t)b * a.rec_stride + c) = *(const bf16x4*)(xin + c);
  }
  __syncthreads();
  if (wave != 0) return;
  f32x4 s = part[0][lane];
#pragma unroll
  for (int v = 1; v < DEC_WAVES; v++) s += part[v][lane];
  if (b0 + (lane & 15) >= a.batch) return;
  // C[o][b]: lane l holds window b0 + l%16 and outputs o0 + 4 (l/16) + 0..3
  const bf16x4 v = {to_bf16(s[0]), to_bf16(s[1]), to_bf16(s[2]), to_bf16(s[3])};
  *(bf16x4*)(a.out + (size_t)b * a.out_stride + o0 + 4 * q) = v;
}

// fp32 arithmetic, one thread per output (window b, column o), plain FMAs:
// fp32 data, or bf16 widths that are not a multiple of 64 (operands widened
// exactly, the output rounded once).
__device__ __forceinline__ float dec_widen(float v) { return v; }
__device__ __forceinline__ float dec_widen(bf16 v) { return (float)v; }
__device__ __forceinline__ void dec_store(float* p, float v) { *p = v; }
__device__ __forceinline__ void dec_store(bf16* p, float v) { *p = to_bf16(v); }

template <typename Args>
__global__ __launch_bounds__(256) void decode_fma_kernel(Args a) {
  const int o = blockIdx.x * 64 + (threadIdx.x & 63);
  const int b = blockIdx.y * 4 + (threadIdx.x >> 6);
  if (o >= a.width || b >= a.batch) return;
  const auto* xin = a.x_in + (size_t)b * a.in_stride;
  float acc = 0.f;
  for (int c = 0; c < a.width; c++)
    acc = fmaf(dec_widen(a.w_self[(size_t)o * a.width + c]), dec_widen(xin[c]), acc);
  if (a.x_partner) {
    const auto* xp = a.x_partner + (size_t)b * a.partner_stride;
    for (int c = 0; c < a.width; c++)
      acc = fmaf(dec_widen(a.w_off[(size_t)o * a.width + c]), dec_widen(xp[c]), acc);
  }
  if (a.record) a.record[(size_t)b * a.rec_stride + o] = xin[o];
  dec_store(a.out + (size_t)b * a.out_stride + o, acc);
}

}  // namespace

hipError_t launch_decode_bf16(const DecodeLayerArgs& a, hipStream_t st) {
  // CH: steps per wave per round, as many as cover the width (no clamped
  // duplicate loads) up to 4 (the whole of width 512 in one round)
  const dim3 grid(a.width / 16, (a.batch + 15) / 16);
  const int ksteps = a.width / 32;
  if (ksteps <= DEC_WAVES) decode_bf16_kernel<1><<<grid, 64 * DEC_WAVES, 0, st>>>(a);
  else if (ksteps <= 2 * DEC_WAVES) decode_bf16_kernel<2><<<grid, 64 * DEC_WAVES, 0, st>>>(a);
  else decode_bf16_kernel<4><<<grid, 64 * DEC_WAVES, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_decode_f32(const DecodeLayerArgsF32& a, hipStream_t st) {
  decode_fma_kernel<<<dim3((a.width + 63) / 64, (a.batch + 3) / 4), 256, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_decode_bf16_fma(const DecodeLayerArgs& a, hipStream_t st) {
  decode_fma_kernel<<<dim3((a.width + 63) / 64, (a.batch + 3) / 4), 256, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace hcmix
