/*
 * hcmix -- rotating-hypercube mixing layers on AMD Instinct MI355X (gfx950).
 *
 * C ABI of libhcmix.so.  Plain pointers and sizes only; no HIP or framework
 * types appear here (a stream is passed as `void*` holding a hipStream_t,
 * NULL meaning the default stream).
 *
 * The operation (paper "Reaching Every Position Without Searching"):
 *   Section 3.1 -- a window of n = 2^b positions is a b-dimensional hypercube;
 *   at layer l position i is linked to its partner i XOR 2^(l mod b).  In the
 *   causal form only the earlier endpoint of each link is kept: position i
 *   takes its partner's vector only when bit (l mod b) of i is set.
 *   Section 3.2, Eq. (1) -- y_i = W_self x_i + W_off x_partner(i): two linear
 *   maps and a shift, with no bias, residual or nonlinearity.
 *
 * Layouts (all row-major, contiguous, no padding):
 *   x, y, dx, dy   [batch][n][width] in `dtype` (bf16 or fp32).  Windows are
 *                  independent; position i of window t is row t*n + i.
 *   w_self, w_off  [width_out][width_in] in `dtype`, so y = W x reads
 *                  y[o] = sum_c W[o][c] x[c].
 *   dw_self, dw_off  [width_out][width_in] fp32.
 *
 * Ownership and ordering: the caller owns every buffer (device memory) and
 * keeps it alive until the enqueued work finishes.  The library allocates and
 * frees nothing, keeps no state between calls (two exceptions, stated where
 * they apply: hcmix_backward_no_alloc's scratch array, and the coordinate
 * tables the field forward leaves in the caller's workspace), never
 * synchronises, and enqueues all work on `stream` in call order.  Calls on
 * different streams that share an output buffer race.
 *
 * Errors: arguments are validated before anything is enqueued; a rejected
 * call has no effect.  HCMIX_ERR_INVALID_VALUE: null pointer, batch < 1, n not
 * a power of two >= 2, width < 1 or above 65536, layer < 0, unknown mode or
 * dtype, an output that overlaps an input, workspace smaller than the query,
 * more than 2^30 rows (batch * n) or 2^40 elements.  HCMIX_ERR_UNSUPPORTED: a
 * shape or alignment the library has no kernel for (bf16 needs width a
 * multiple of 8 and 16-byte aligned pointers; fp32 needs 4-byte aligned
 * pointers).  HCMIX_ERR_HIP: a HIP call or kernel launch failed; the message
 * is available from hcmix_last_hip_error().
 *
 * Kernels of the mixing layer: bf16 widths that are a multiple of 64 run on
 * matrix-core (MFMA) kernels; fp32 and the other bf16 widths (multiples of 8)
 * run on fp32 FMA kernels.  Both accumulate in fp32 and round each bf16
 * output once, so they agree up to the order of summation.
 */
#ifndef HCMIX_H
#define HCMIX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HCMIX_OK = 0,
  HCMIX_ERR_INVALID_VALUE = 1,
  HCMIX_ERR_UNSUPPORTED = 2,
  HCMIX_ERR_HIP = 3
} hcmix_status;

typedef enum { HCMIX_F32 = 0, HCMIX_BF16 = 1 } hcmix_dtype;

/* HCMIX_BIDIR: every position takes its partner (Section 3.1, 2n links per
 * layer counting self).  HCMIX_CAUSAL: only the later endpoint of a link
 * receives, i.e. position i receives when bit d of i is 1 (n + n/2 links). */
typedef enum { HCMIX_BIDIR = 0, HCMIX_CAUSAL = 1 } hcmix_mode;

/* Layer code of the local layer: Eq. (1) with jump k = 1, the schedules'
 * "near" layer (Section 3.3, Appendix A):
 *   y[t][i] = W_self x[t][i] + W_off x[t][i-1]   (i >= 1; position 0 of a
 *                                                  window takes no partner)
 * It exists in causal form only (mode must be HCMIX_CAUSAL).  Wherever a
 * layer index is taken (`layer`, `layers[l]`), this value selects it; values
 * >= 0 select the hypercube layer of dimension hcmix_dim(value, n). */
enum { HCMIX_LAYER_NEAR = -1 };

/* Human-readable name of a status code (static storage). */
const char* hcmix_status_string(int32_t status);

/* Text of the last HIP error seen by this thread ("" if none). */
const char* hcmix_last_hip_error(void);

/* Hypercube dimension used at layer `layer` for windows of n positions
 * (Section 3.1): layer mod log2(n).  Returns -1 if n is not a power of two
 * >= 2 or layer < 0.  A fixed (un-rotated) schedule simply passes the same
 * layer index every time; any dimension d < log2(n) is selected by layer = d. */
int32_t hcmix_dim(int32_t layer, int64_t n);

/* Forward of one layer, Eq. (1):
 *   y[t][i] = W_self x[t][i] + m(i) W_off x[t][i XOR 2^d],   d = hcmix_dim(layer, n)
 * with m(i) = 1 (HCMIX_BIDIR) or bit d of i (HCMIX_CAUSAL); for
 * layer == HCMIX_LAYER_NEAR the partner is i - 1 and m(i) = (i >= 1).
 * bf16: inputs bf16, products accumulated in fp32, y rounded to bf16 (nearest
 * even).  fp32: fp32 throughout, no reduced-precision matrix instructions.
 * y must not overlap x. */
hcmix_status hcmix_forward(int64_t batch, int64_t n, int64_t width, int32_t layer,
                           int32_t mode, int32_t dtype, const void* x,
                           const void* w_self, const void* w_off, void* y,
                           void* stream);

/* Bytes of device workspace hcmix_backward needs for this shape (0 if none),
 * or 0 for invalid arguments. The workspace must be 256-byte aligned. */
size_t hcmix_backward_workspace_bytes(int64_t batch, int64_t n, int64_t width,
                                      int32_t dtype);

/* Backward of one layer: the adjoint of hcmix_forward.  Given dy = dL/dy,
 *   dx[t][j]  = W_self^T dy[t][j] + m'(j) W_off^T dy[t][j XOR 2^d]
 *               with m'(j) = 1 (bidir) or 1 - bit d of j (causal: j is the
 *               earlier endpoint of the link it sends on); for the local layer
 *               dy[t][j+1] with m'(j) = (j <= n - 2)
 *   dw_self   = sum over (t, i) of dy[t][i] x[t][i]^T
 *   dw_off    = sum over (t, i) of m(i) dy[t][i] x[t][partner(i)]^T
 * dx is in `dtype` (bf16: fp32 accumulation, rounded once); dw_* are fp32,
 * overwritten when accumulate == 0 and added to when accumulate != 0.
 * dx, dw_self, dw_off and workspace must not overlap each other or any input.
 * The weight-gradient reduction over rows runs in a fixed order, so repeated
 * calls give bitwise-identical results. */
hcmix_status hcmix_backward(int64_t batch, int64_t n, int64_t width, int32_t layer,
                            int32_t mode, int32_t dtype, const void* x,
                            const void* w_self, const void* w_off, const void* dy,
                            void* dx, float* dw_self, float* dw_off,
                            int32_t accumulate, void* workspace,
                            size_t workspace_bytes, void* stream);

/* hcmix_backward for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same computation and kernels, hence bitwise the same results, with the
 * split-K partial sums kept in a scratch array inside the library instead of a
 * caller workspace.  The array is HCMIX_NO_ALLOC_SCRATCH_BYTES of device
 * memory per GPU, held from the first call on that GPU until the process
 * ends; the call allocates and frees nothing.  Shapes whose partials need
 * more than that (bf16 widths above 2048) return HCMIX_ERR_UNSUPPORTED; fp32
 * calls use no scratch.  Every call on one GPU shares that GPU's array, so
 * calls that overlap in time on one GPU (other streams, other threads) race
 * and give wrong weight gradients; serialise them.  The array's contents are
 * overwritten by every call before they are read.  Other arguments and
 * errors as for hcmix_backward. */
#define HCMIX_NO_ALLOC_SCRATCH_BYTES ((size_t)32 << 20)

hcmix_status hcmix_backward_no_alloc(int64_t batch, int64_t n, int64_t width, int32_t layer,
                                     int32_t mode, int32_t dtype, const void* x,
                                     const void* w_self, const void* w_off, const void* dy,
                                     void* dx, float* dw_self, float* dw_off,
                                     int32_t accumulate, void* stream);

/* ---- Whole stacks (Section 3.3: a schedule is a list of layer indices) ----
 *
 * layers:        host array of num_layers layer indices (layer l uses
 *                dimension hcmix_dim(layers[l], n)); the rotated schedule is
 *                0, 1, 2, ..., the fixed control repeats one index.
 * w_self, w_off: host arrays of num_layers device pointers, one pair per layer.
 *
 * layers[l] may also be HCMIX_LAYER_NEAR (causal mode), so the local, mixa
 * and hybrid schedules of Section 3.3 are lists such as
 * {NEAR, 5, NEAR, 4, ..., NEAR, 0} (jump 2^d = hypercube layer d).
 *
 * For bf16, width 64 and n in {64, 128, 256} (a window of at most 32 KB) a
 * stack of hypercube layers runs in one kernel with every window resident in
 * LDS (one block per window); otherwise (or with local layers) the layers run
 * one launch each, with results identical to calling hcmix_forward /
 * hcmix_backward layer by layer up to the order of floating-point summation.
 * num_layers may be at most 64 for the fused kernels; longer stacks run layer
 * by layer.
 */

/* Forward through the stack: xs is a host array of num_layers device
 * pointers receiving x_1 .. x_L, where x_0 = x and x_{l+1} is layer l
 * applied to x_l.  Every xs[l] must be distinct from each other and from
 * the inputs. */
hcmix_status hcmix_stack_forward(int64_t batch, int64_t n, int64_t width, int32_t num_layers,
                                 const int32_t* layers, int32_t mode, int32_t dtype,
                                 const void* x, const void* const* w_self,
                                 const void* const* w_off, void* const* xs, void* stream);

/* Bytes of device workspace hcmix_stack_backward needs (0 for invalid
 * arguments).  256-byte aligned.
 *  - bf16, two or more layers, width a multiple of 128 (deferred weight
 *    gradients): the gradient of every intermediate activation (L - 1 of
 *    [batch][n][width], or a ring of 65 for stacks longer than 64 layers), a
 *    transposed copy of every weight matrix, and the row-range partials of the
 *    weight-gradient launch when the stack is too short to fill the chip
 *    (hcmix_stack_weight_gradients_workspace_bytes).
 *  - fused path: the per-window weight-gradient partials;
 *  - otherwise, layer by layer: two gradient buffers, the split-K partials of
 *    one layer and (bf16, two or more layers) the transposed weights. */
size_t hcmix_stack_backward_workspace_bytes(int64_t batch, int64_t n, int64_t width,
                                            int32_t num_layers, int32_t dtype);

/* Backward through the stack: xs_in is a host array of the num_layers layer
 * inputs x_0 .. x_{L-1} (device pointers), dy the gradient of x_L.  Writes dx
 * (gradient of x_0, in dtype) and, for every layer, dw_self[l] and dw_off[l]
 * (host arrays of device pointers to fp32 [width][width]), overwritten when
 * accumulate == 0, added to otherwise.  Weight gradients are summed in a
 * fixed order (bitwise-repeatable).  On the deferred path (bf16, two or more
 * layers, width a multiple of 128) the dX chain runs first, keeping every
 * intermediate gradient in the workspace, and then
 * hcmix_stack_weight_gradients forms all weight gradients at once. */
hcmix_status hcmix_stack_backward(int64_t batch, int64_t n, int64_t width, int32_t num_layers,
                                  const int32_t* layers, int32_t mode, int32_t dtype,
                                  const void* const* xs_in, const void* const* w_self,
                                  const void* const* w_off, const void* dy, void* dx,
                                  float* const* dw_self, float* const* dw_off,
                                  int32_t accumulate, void* workspace, size_t workspace_bytes,
                                  void* stream);

/* Weight gradients of every layer of a stack from the layers' inputs and the
 * gradients of their outputs (the weight-gradient half of the backward, e.g.
 * for schedules that defer it):
 *   dw_self[l] (+)= sum over (t, i) of dys[l][t][i] xs_in[l][t][i]^T
 *   dw_off[l]  (+)= sum over (t, i) of m(i) dys[l][t][i] xs_in[l][t][partner(i)]^T
 * with partner and m as in hcmix_backward for layer code layers[l].  xs_in and
 * dys: host arrays of num_layers device pointers to [batch][n][width] in dtype;
 * dw_self, dw_off: host arrays of device pointers to fp32 [width][width],
 * overwritten when accumulate == 0, added to otherwise; no output may overlap
 * any input or another output.  bf16 with width a multiple of 128: one launch
 * per 64 layers whose blocks each own a 128 x 128 tile of both matrices over
 * every row (or, when layers x tiles cannot fill the chip, over a row range,
 * plus a fixed-order sum of the ranges); other shapes: the per-layer kernels
 * of hcmix_backward.  Bitwise-repeatable.  The workspace (256-byte aligned,
 * hcmix_stack_weight_gradients_workspace_bytes, possibly 0) holds those
 * partial sums. */
size_t hcmix_stack_weight_gradients_workspace_bytes(int64_t batch, int64_t n, int64_t width,
                                                     int32_t num_layers, int32_t dtype);

hcmix_status hcmix_stack_weight_gradients(int64_t batch, int64_t n, int64_t width,
                                          int32_t num_layers, const int32_t* layers, int32_t mode,
                                          int32_t dtype, const void* const* xs_in,
                                          const void* const* dys, float* const* dw_self,
                                          float* const* dw_off, int32_t accumulate,
                                          void* workspace, size_t workspace_bytes,
                                          void* stream);

/* The data half of the stack backward: the dX chain alone (the adjoint of
 * Eq. (1) layer after layer, from the top), keeping every intermediate
 * gradient in caller memory, so that a model whose sparse stacks alternate
 * with other layers can form the weight gradients of all its sparse layers
 * afterwards in one hcmix_stack_weight_gradients call.  dy: the gradient of
 * the stack's output x_L; grads: host array of num_layers - 1 device pointers
 * (ignored, may be NULL, when num_layers == 1), grads[l - 1] receiving g_l,
 * the gradient of layer l's input, for l = 1 .. L-1; dx receives g_0.  Layer
 * l's output gradient is then grads[l] (or dy for the last layer), which is
 * what hcmix_stack_weight_gradients takes as dys[l].  The dX products are the
 * ones hcmix_stack_backward runs, so dx and the grads equal its intermediate
 * gradients bitwise on the layer-by-layer and deferred paths.  Layouts,
 * layer codes, modes and alignment as for hcmix_stack_backward; no output
 * (dx, grads, workspace) may overlap an input (dy, weights) or another
 * output.  Workspace (256-byte aligned, possibly 0 bytes): bf16 stacks of two
 * or more layers keep a transposed copy of every weight matrix there. */
size_t hcmix_stack_backward_data_workspace_bytes(int64_t width, int32_t num_layers,
                                                 int32_t dtype);

hcmix_status hcmix_stack_backward_data(int64_t batch, int64_t n, int64_t width,
                                       int32_t num_layers, const int32_t* layers, int32_t mode,
                                       int32_t dtype, const void* const* w_self,
                                       const void* const* w_off, const void* dy,
                                       void* const* grads, void* dx, void* workspace,
                                       size_t workspace_bytes, void* stream);

/* Output head backward: the gradients that the chain rule gives for
 * logits = W x + bias from dlogits (the products named above):
 *   gx[r][k] = sum over v of dlogits[r][v] W[v][k]              (bf16, [rows][width]),
 *   dw[v][k] (+)= sum over rows r of dlogits[r][v] x[r][k]      (fp32, [vocab][width]).
 * Either output may be NULL (not both); x is read only for dw and may be NULL
 * without it (gx alone is then a plain product of two bf16 matrices, which
 * also serves a linear map's forward on the transposed weights).  dw is summed in a fixed order
 * (row-range partials, then the ranges in order: bitwise-repeatable) through a
 * workspace of hcmix_head_backward_workspace_bytes (256-byte aligned; unused,
 * may be NULL, without dw); accumulate != 0 adds to dw instead of overwriting.
 * vocab a multiple of 32, width a multiple of 64; x, w, dlogits and gx 16-byte
 * aligned, dw 4-byte aligned.  Errors as for the entry points above. */
size_t hcmix_head_backward_workspace_bytes(int64_t rows, int64_t width, int32_t vocab);

hcmix_status hcmix_head_backward(int64_t rows, int64_t width, int32_t vocab, const void* x,
                                 const void* w, const void* dlogits, void* gx, float* dw,
                                 int32_t accumulate, void* workspace, size_t workspace_bytes,
                                 void* stream);

/* ---- Decode: one new position of every window through the whole stack ----
 *
 * The causal stack evaluated incrementally (the one-position-at-a-time path
 * of the paper's deployment paragraph, Section 8): at position `pos` layer l
 * needs its own input there and, when the position receives, its input at the
 * partner position (pos - 2^d for a hypercube layer whose bit d of pos is set,
 * pos - 1 for the local layer), which an earlier step recorded in the cache.
 *
 * Cache: caller-owned device memory of hcmix_decode_cache_bytes() bytes,
 * 256-byte aligned, sized by the schedule as the deployment paragraph bounds
 * it: a hypercube layer of dimension d keeps the inputs of the last 2^d
 * positions (a ring of 2^d [batch][width] slots: a position with bit d clear
 * records its input, the position 2^d later reads it), the local layer the
 * last two, plus two [batch][width] buffers that pass each layer's output to
 * the next.  So it never grows with the position, and for the window-256
 * rotated stack (dimensions 0..7 twice) it holds 512 slots instead of 16 x
 * 256.  Positions of a window must be decoded in order 0, 1, 2, ... (a step
 * reads what earlier steps recorded); starting a new window is starting
 * again at pos = 0.  Only slots that earlier steps of the window wrote are
 * ever read, so the cache needs no initialisation.
 *
 * x: [batch][width], the stack's input at `pos` for every window; y:
 * [batch][width], the stack's output there.  layers: host array of layer codes
 * as for the stacks (hypercube layers or HCMIX_LAYER_NEAR); the stack is
 * causal.  bf16: width a multiple of 8, 16-byte aligned pointers; fp32: 4-byte
 * aligned.  Results equal those of hcmix_stack_forward over the window at
 * position pos, up to the order of floating-point summation.
 * HCMIX_ERR_INVALID_VALUE also for pos outside [0, n), a short cache, or y or
 * the cache overlapping an input. */
size_t hcmix_decode_cache_bytes(int64_t batch, int64_t n, int64_t width, int32_t num_layers,
                                const int32_t* layers, int32_t dtype);

hcmix_status hcmix_decode_step(int64_t batch, int64_t n, int64_t width, int32_t num_layers,
                               const int32_t* layers, int32_t dtype, int64_t pos, const void* x,
                               const void* const* w_self, const void* const* w_off, void* cache,
                               size_t cache_bytes, void* y, void* stream);

/* ---- Channel-shared mixing: the two maps as per-position scalars ----
 *
 * The sparse layer of Eq. (1) with both linear maps reduced to scalars per
 * position, shared by every channel and taken from an n x n table T_l per
 * layer (the paper's parameter totals, Section 5's cost tables, count n^2
 * mixing parameters per layer, and its dense schedule uses the whole table):
 *   y[t][i][c] = T_l[i][i] x[t][i][c] + m(i) T_l[i][p(i)] x[t][p(i)][c]
 * with partner p and mask m exactly as for hcmix_forward (hypercube layer of
 * dimension hcmix_dim(layer, n), or HCMIX_LAYER_NEAR in causal mode).  Entries
 * of T_l off the layer's links are never read.
 *
 * tables: host array of num_layers device pointers to fp32 [n][n] tables
 * (row = receiving position).  x, xs[l], dy, dx: [batch][n][width] in dtype
 * (bf16: fp32 arithmetic, every layer's output rounded once to bf16).  The
 * whole stack runs in one launch per direction, each window's slice of
 * channels staying on chip through every layer.  Shapes: n a power of two
 * from 2 to 256, width a multiple of 64 (bf16) or 32 (fp32), at most 64
 * layers (HCMIX_ERR_UNSUPPORTED otherwise); activations 16-byte aligned,
 * tables 4-byte aligned.  Other errors as for the stacks above. */
hcmix_status hcmix_shared_stack_forward(int64_t batch, int64_t n, int64_t width,
                                        int32_t num_layers, const int32_t* layers, int32_t mode,
                                        int32_t dtype, const void* x, const float* const* tables,
                                        void* const* xs, void* stream);

/* Backward: dx (gradient of x_0, in dtype) and the table gradients
 *   dT_l[i][i]    = sum over (t, c) of g[t][i][c] x_l[t][i][c]
 *   dT_l[i][p(i)] = m(i) sum over (t, c) of g[t][i][c] x_l[t][p(i)][c]
 * (g the gradient of layer l's output), every other entry 0; dtables[l] fp32
 * [n][n], overwritten (accumulate == 0) or added to on the link entries only.
 * xs_in: the layer inputs x_0 .. x_{L-1} as hcmix_shared_stack_forward wrote
 * them.  Sums run in a fixed order (bitwise-repeatable) through a workspace of
 * hcmix_shared_stack_backward_workspace_bytes (256-byte aligned) holding
 * per-block partial sums. */
size_t hcmix_shared_stack_backward_workspace_bytes(int64_t batch, int64_t n, int64_t width,
                                                   int32_t num_layers, int32_t dtype);

hcmix_status hcmix_shared_stack_backward(int64_t batch, int64_t n, int64_t width,
                                         int32_t num_layers, const int32_t* layers, int32_t mode,
                                         int32_t dtype, const void* const* xs_in,
                                         const float* const* tables, const void* dy, void* dx,
                                         float* const* dtables, int32_t accumulate,
                                         void* workspace, size_t workspace_bytes, void* stream);

/* ---- Causal multi-head softmax attention (the hybrids' attention layers) ----
 *
 * The hybrid schedules (Section 3.3; the window-256 hybrid of Appendix A keeps
 * two attention layers among sixteen) replace some sparse layers with standard
 * multi-head attention.  These entry points are its core, per window and head:
 *   S = Q K^T / sqrt(64), S[i][j] = -inf for j > i (a position sees itself and
 *   the past), P = row softmax of S, out = P V,
 * for windows of n positions (n a multiple of 32, at most 256), head dimension
 * 64, bf16 in and out with fp32 accumulation.  The projections around it are
 * plain GEMMs and stay with the caller.
 *   qkv:  [batch][n][3][heads][64] bf16, Q, K, V of every position (the
 *         [batch, n, 3 * heads * 64] output of a QKV projection).
 *   out:  [batch][n][heads][64] bf16.
 *   lse:  fp32 [batch][heads][n], the natural log of each query row's softmax
 *         denominator, log sum_j exp(S[i][j]); written by the forward, read by
 *         the backward.
 * HCMIX_ERR_INVALID_VALUE: null pointers, batch, heads or n < 1, an output
 * overlapping an input or another output.  HCMIX_ERR_UNSUPPORTED: head_dim !=
 * 64, n not a multiple of 32 or above 256, bf16 pointers not 16-byte aligned,
 * lse not 4-byte aligned. */
hcmix_status hcmix_attention_forward(int64_t batch, int64_t n, int32_t heads, int32_t head_dim,
                                     const void* qkv, void* out, float* lse, void* stream);

/* Backward: dqkv [batch][n][3][heads][64] bf16, the gradients of Q, K and V,
 * from qkv, the forward's out and lse, and dout = dL/dout:
 *   dV = P^T dout, dS = P * (dout V^T - rowsum(dout * out)),
 *   dQ = dS K / 8, dK = dS^T Q / 8. */
hcmix_status hcmix_attention_backward(int64_t batch, int64_t n, int32_t heads, int32_t head_dim,
                                      const void* qkv, const void* out, const float* lse,
                                      const void* dout, void* dqkv, void* stream);

/* ---- Field coupling (Section 3.4's dynamics variant; Section 7) ----
 *
 * Every position i of a window carries a coordinate p_i with coord_dim
 * components; positions are coupled by a Gaussian of their squared distance,
 * and the scaled form ("field") divides each squared distance by its causal
 * row mean first.  Reading taken here (the paper states the coupling in words;
 * the force that moves the coordinates and the number of repetitions T belong
 * to the model and stay with the caller, who passes the coordinates of each
 * application):
 *   D[i][j] = |p_i - p_j|^2,  m_i = (1 / (i + 1)) sum_{j <= i} D[i][j],
 *   a[i][j] = -D[i][j] / (tau m_i)   (scaled = 1; all 0 when m_i = 0)
 *           = -D[i][j] / tau         (scaled = 0),
 *   C[i][j] = exp(a[i][j]) / Z_i,  Z_i = sum_{j <= i} exp(a[i][j]),  C = 0 for j > i,
 *   y_i = sum_{j <= i} C[i][j] x_j,
 *   partners_i = exp(-sum_j C[i][j] ln C[i][j])  (Section 7's effective number
 *   of partners).
 * Layouts: p [batch][n][coord_dim] fp32; x, y, dy, dx [batch][n][width] bf16;
 * row_mean, lse, partners [batch][n] fp32 (lse = ln Z_i); dp like p.
 * Precision: distances from a split-bf16 Gram product with fp32 accumulation
 * (about 2^-17 of the squared norms of p_i - p_0), couplings and statistics in
 * fp32, the two products with x and dy on bf16 matrix cores (couplings rounded
 * to bf16, fp32 accumulation), outputs rounded once.  In the scaled form a
 * positive row mean below 2^-100 is taken as 2^-100.
 * workspace: hcmix_field_workspace_bytes(batch, n, coord_dim) bytes of device
 * memory, 256-byte aligned, owned by the caller.  The forward leaves each
 * window's coordinate table (the split centred coordinates and their norms)
 * in it, which the backward can take instead of building it again
 * (reuse_table); the backward also keeps the couplings and the gradient of
 * the squared distances there during the call.  Calls that share a workspace must not
 * overlap.
 * HCMIX_ERR_INVALID_VALUE: null pointers (partners may be null), batch, n,
 * width or coord_dim < 1, tau outside [2^-24, 2^24] or not finite, scaled not 0
 * or 1, an output overlapping an input or another output, a workspace smaller
 * than the query, sizes past the limits above.
 * HCMIX_ERR_UNSUPPORTED: n above 256, coord_dim above 64, width not a
 * multiple of 64, bf16 pointers not 16-byte aligned, fp32 pointers not 4-byte
 * aligned, a workspace not 256-byte aligned. */
hcmix_status hcmix_field_forward(int64_t batch, int64_t n, int64_t width, int32_t coord_dim,
                                 float tau, int32_t scaled, const float* p, const void* x,
                                 void* y, float* row_mean, float* lse, float* partners,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of device workspace the field calls need: for each window its
 * coordinate table (N (4 c' + 20) bytes rounded up to 256, c' = coord_dim
 * rounded up to 16), plus N * N * 6 with N = n rounded up to a multiple of 32
 * (the gradient of the window's squared distances in fp32 and its couplings in
 * bf16, used by the backward); 0 for arguments outside the supported range. */
size_t hcmix_field_workspace_bytes(int64_t batch, int64_t n, int32_t coord_dim);

/* Backward: dp = dL/dp and dx = dL/dx (both overwritten) from p, x, the
 * forward's row_mean and lse (same coordinates, tau and scaled), and dy:
 *   dx_j = sum_{i >= j} C[i][j] dy_i,
 *   da[i][j] = C[i][j] (dy_i . x_j - dy_i . y_i),
 *   dD[i][j] = -da[i][j] / (tau m_i) + (sum_k da[i][k] D[i][k]) / (tau m_i^2 (i + 1))
 *              (scaled; -da[i][j] / tau unscaled; 0 for rows with m_i = 0),
 *   dp_i = 2 sum_{j <= i} dD[i][j] (p_i - p_j) + 2 sum_{k >= i} dD[k][i] (p_i - p_k).
 * dy_i . y_i is taken as sum_j C[i][j] (dy_i . x_j), so y is not read.
 * reuse_table = 1: the workspace still holds the tables hcmix_field_forward
 * wrote for these same p, batch, n and coord_dim (no call has used the
 * workspace since), and the backward reads them instead of building them
 * (one launch fewer; the results are bitwise those of reuse_table = 0).  The
 * library cannot check this; tables of other coordinates give wrong dp and
 * dx, never an access outside the buffers.  reuse_table = 0 builds them from
 * p.  Other values: HCMIX_ERR_INVALID_VALUE. */
hcmix_status hcmix_field_backward(int64_t batch, int64_t n, int64_t width, int32_t coord_dim,
                                  float tau, int32_t scaled, const float* p, const void* x,
                                  const float* row_mean, const float* lse, const void* dy,
                                  float* dp, void* dx, int32_t reuse_table, void* workspace,
                                  size_t workspace_bytes, void* stream);

/* ---- Linear maps: the attention layers' projections in the hybrids ----
 *
 * The hybrid schedules' attention layers (Section 3.3) project each position
 * to queries, keys and values and back: plain linear maps y = x W^T around the
 * attention core above.  bf16 in and out, fp32 accumulation.
 *   x [rows][in_width], W [out_width][in_width], y [rows][out_width].
 * rows even; in_width and out_width multiples of 64 (HCMIX_ERR_UNSUPPORTED
 * otherwise); bf16 pointers 16-byte aligned.  Errors as above. */
hcmix_status hcmix_linear_forward(int64_t rows, int64_t in_width, int64_t out_width,
                                  const void* x, const void* w, void* y, void* stream);

/* Backward of the linear map: dx = dy W (bf16 [rows][in_width]) and
 * dw (+)= dy^T x (fp32 [out_width][in_width], row ranges summed in a fixed
 * order through a workspace of hcmix_linear_backward_workspace_bytes, 256-byte
 * aligned; bitwise-repeatable).  Either output may be NULL (not both); x is
 * read only for dw.  accumulate != 0 adds to dw. */
size_t hcmix_linear_backward_workspace_bytes(int64_t rows, int64_t in_width, int64_t out_width);

hcmix_status hcmix_linear_backward(int64_t rows, int64_t in_width, int64_t out_width,
                                   const void* x, const void* w, const void* dy, void* dx,
                                   float* dw, int32_t accumulate, void* workspace,
                                   size_t workspace_bytes, void* stream);

/* ---- Token embedding, output head and cross-entropy (language-model workloads) ----
 *
 * Section 5 trains character-level language models and reports bits per
 * character, the mean next-symbol cross-entropy.  These entry points are the
 * model's input and output ends around the sparse stack:
 *   x[r] = table[tokens[r]],        dtable[v] (+)= sum of dx[r] over tokens[r] == v,
 *   logits[r] = W x[r] + bias,      loss[r] = log sum_v exp(logits[r][v]) - logits[r][targets[r]],
 *   dlogits[r] = scale (softmax(logits[r]) - onehot(targets[r]))   (scale = 1/rows: mean loss).
 * rows = batch * n positions; table and W are [vocab][width] bf16, x and dx
 * [rows][width] bf16, tokens and targets int32 [rows], bias, loss and dtable
 * fp32, dlogits [rows][vocab] bf16 (the gradients of W and x then are plain
 * products with it, dlogits^T x and dlogits W, which hcmix_head_backward
 * computes; the bias gradient, its column sums, comes with dlogits).
 * bf16 only; width a multiple of 64; head: vocab a multiple of 32 up to 256.
 * A token outside [0, vocab) embeds as a zero row and is skipped by the
 * backward; a target outside it contributes log sum exp alone.  The embedding
 * backward sums in a fixed order (bitwise-repeatable) through a workspace of
 * hcmix_embedding_backward_workspace_bytes (256-byte aligned).
 * HCMIX_ERR_INVALID_VALUE: null pointers, rows, width or vocab < 1, an output
 * overlapping an input or another output, a short workspace.
 * HCMIX_ERR_UNSUPPORTED: other shapes, bf16 pointers not 16-byte aligned, fp32
 * and int32 pointers not 16-byte (bias) or 4-byte aligned. */
hcmix_status hcmix_embedding_forward(int64_t rows, int64_t width, int32_t vocab, const void* table,
                                     const int32_t* tokens, void* x, void* stream);

size_t hcmix_embedding_backward_workspace_bytes(int64_t rows, int64_t width, int32_t vocab);

hcmix_status hcmix_embedding_backward(int64_t rows, int64_t width, int32_t vocab,
                                      const int32_t* tokens, const void* dx, float* dtable,
                                      int32_t accumulate, void* workspace, size_t workspace_bytes,
                                      void* stream);

/* Output head and cross-entropy: loss and dlogits as above and, when dbias is
 * not NULL, the bias gradient dbias[v] = sum over rows of dlogits[r][v]
 * (overwritten; summed from the unrounded fp32 values in a fixed order,
 * bitwise-repeatable) through a workspace of
 * hcmix_head_cross_entropy_workspace_bytes (256-byte aligned; unused, may be
 * NULL, without dbias). */
size_t hcmix_head_cross_entropy_workspace_bytes(int64_t rows, int32_t vocab);

hcmix_status hcmix_head_cross_entropy(int64_t rows, int64_t width, int32_t vocab, const void* x,
                                      const void* w, const float* bias, const int32_t* targets,
                                      float scale, float* loss, void* dlogits, float* dbias,
                                      void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* HCMIX_H */
