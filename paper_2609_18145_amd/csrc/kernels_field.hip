// Field coupling of the dynamics variant (Section 3.4): every position i of a
// window carries a coordinate p_i (c <= 64 components, fp32), and the causal
// coupling of row i is the row-normalised Gaussian of squared distances,
//   D[i][j] = |p_i - p_j|^2,  m_i = mean of D[i][j] over j <= i,
//   a[i][j] = -D[i][j] / (tau m_i)   (scaled form, "field"; 0 when m_i = 0)
//           = -D[i][j] / tau         (unscaled form),
//   C[i][j] = exp(a[i][j]) / Z_i over j <= i,  y_i = sum_j C[i][j] x_j,
// with the effective number of partners exp(-sum_j C ln C) of Section 7 as a
// by-product.  x, y bf16 [batch][n][width], width % 64 == 0, n <= 256.
//
// Distances go through the Gram matrix on the bf16 matrix cores:
//   D[i][j] = N_i + N_j - 2 p'_i . p'_j,  p' = p - p_0 (D is translation
// invariant; centring on the window's first position keeps the norms near the
// distances' scale, and makes D exactly 0 when all coordinates are equal),
// each centred component split into bf16 hi + lo (exact in fp32, 2^-17
// relative) and the dot product taken as hi.hi + lo.hi + hi.lo (three MFMAs
// per 16 components, fp32 accumulation; the dropped lo.lo term is below
// 2^-17 of the norms).  The diagonal is set to exactly 0 (its rounding would
// otherwise reach the unscaled logits undivided).  Every logit is <= 0 up to
// that rounding and the diagonal's is 0, so each row's maximum is known: the
// exponentials need no running maximum and Z_i lies in [1, i + 1].
//
// Kernels (one window's coordinates and one 64-column slab per block, the
// whole causal row of a 32-query tile in registers as in the attention core):
//   field_fwd_kernel        y slab, and (slab 0) m_i, ln Z_i, partners;
//   field_bwd_rows_kernel   per query tile: the couplings C (written, bf16,
//                           transposed, for the dx kernel), dP[i][j] = dy_i .
//                           x_j over the full width, Delta_i = sum_j C dP (=
//                           dy_i . y_i), da = C (dP - Delta), and the gradient
//                           of the squared distances dD (written, fp32,
//                           [key][query]);
//   field_bwd_dx_kernel     dx slab = C^T dy (keys in lanes, C as written);
//   field_bwd_coord_kernel  dp_i = 2 sum_j E[i][j] (p_i - p_j), E = dD + dD^T,
//                           on the fp32 matrix cores.
#include "hcmix_internal.h"
#include "device_common.h"
#include "tile64.h"

namespace hcmix {

namespace {

constexpr int FT = 512;                       // threads per block, 8 waves
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Coordinate table in LDS: row r = [hi (cp) | lo (cp) | 8 pad] bf16 of the
// centred coordinate p_r - p_0 (cp = c rounded up to 16, zero padded).  The
// row stride 2 cp + 8 elements is an odd multiple of 16 bytes, so 16
// consecutive rows read at one column fall in 16 distinct 16-byte bank slots.
__device__ __forceinline__ int ct_stride(int cp) { return 2 * cp + 8; }

__device__ __forceinline__ bf16x8 ct_frag(const bf16* t, int rs, int r0, int c0, int lane) {
  return *(const bf16x8*)(t + (r0 + (lane & 31)) * rs + c0 + 8 * (lane >> 5));
}
// The 8 components of row r that lane half h contributes to a 16-wide k step.
__device__ __forceinline__ bf16x8 ct_row(const bf16* t, int rs, int r, int c0, int half) {
  return *(const bf16x8*)(t + r * rs + c0 + 8 * half);
}

// Copy a window's coordinates (pw: rows x c fp32, contiguous) into LDS rows
// `stride` bytes apart: consecutive threads take consecutive elements (every
// load coalesced, all of a thread's loads issued before its first LDS write);
// the element -> (row, column) walk advances by a precomputed step, with no
// division per element.
struct NoIssue {
  __device__ __forceinline__ void operator()() const {}
};
// `then` runs after the loads are issued and before their values are used
// (loads it issues queue behind them).  vec: pw is 16-byte aligned and c a
// multiple of 4, so 16-byte loads never straddle a row (a wave-wide memory
// instruction costs about the same whatever its width, so wide loads move
// four times the bytes per instruction).
template <int THREADS, class Then = NoIssue>
__device__ __forceinline__ void stage_coords(const float* __restrict__ pw, int rows, int c,
                                             unsigned char* dst, int stride, bool vec,
                                             Then then = {}) {
  const int total = rows * c;
  if (vec) {
    constexpr int PER = 256 * 64 / 4 / THREADS;     // float4 per thread at 256 rows x 64
    const int total4 = total >> 2;
    f32x4 v[PER];
#pragma unroll
    for (int u = 0; u < PER; u++)
      v[u] = ((const f32x4*)pw)[min((int)threadIdx.x + THREADS * u, total4 - 1)];
    then();
    int r = (4 * threadIdx.x) / c, k = (4 * threadIdx.x) % c;
    const int dr = (4 * THREADS) / c, dk = (4 * THREADS) % c;
#pragma unroll
    for (int u = 0; u < PER; u++) {
      if ((int)threadIdx.x + THREADS * u < total4) {
        float* d = (float*)(dst + r * stride) + k;
        d[0] = v[u][0];
        d[1] = v[u][1];
        d[2] = v[u][2];
        d[3] = v[u][3];
      }
      k += dk;
      r += dr;
      if (k >= c) {
        k -= c;
        r += 1;
      }
    }
  } else {
    constexpr int PER = 256 * 64 / THREADS;
    float v[PER];
#pragma unroll
    for (int u = 0; u < PER; u++)   // unconditional loads (clamped): no branch waits per load
      v[u] = pw[min((int)threadIdx.x + THREADS * u, total - 1)];
    then();
    int r = threadIdx.x / c, k = threadIdx.x % c;
    const int dr = THREADS / c, dk = THREADS % c;
#pragma unroll
    for (int u = 0; u < PER; u++) {
      if ((int)threadIdx.x + THREADS * u < total) *(float*)(dst + r * stride + 4 * k) = v[u];
      k += dk;
      r += dr;
      if (k >= c) {
        k -= c;
        r += 1;
      }
    }
  }
}

// The coordinate table rows [0, rows) (rows <= 256) and their squared norms
// N_r (of hi + lo, fp32), from the window's coordinates pw [n][c]; with TILES
// also what a row's mean needs from the tiles before it:
//   sTS[t][k] = sum over rows j < 32 t (of the window) of the centred p_j[k]
//   (fp32, t = 0 .. NT; each tile's column sum by one thread, then a running
//   sum over the tiles), and sPN[t] = sum of N_j over tile t.  Then, for
//   query q in tile t,
//   sum_{j < 32 t} D[q][j] = 32 t N_q + sum_{t' < t} sPN[t'] - 2 p'_q . sTS[t].
// The raw rows are staged in the table's own space with a stride of c + 1
// words (consecutive rows in distinct banks; (c + 1) * 4 <= (2 cp + 8) * 2
// bytes, so they fit); each table row is then split by two threads (cp / 2
// columns each: thread tid takes row tid % 256, half tid / 256), every LDS
// read of a phase issued before its values are used.  Rows at or past n are
// zero, N_r = 0.  `then` is passed on to stage_coords.  Three barriers; ends
// with one.  sNh: [2][NT * 32] scratch for the half-row norms.
template <int NT, bool TILES, class Then>
__device__ __forceinline__ void build_table(const float* __restrict__ pw, int n, int c, int cp,
                                            int rows, bf16* sT, float* sN, float* sNh,
                                            float* sTS, float* sPN, bool vec, Then then) {
  constexpr int NP = NT * 32;
  const int rws = (c + 1) * 4;                       // raw staging row stride (bytes)
  unsigned char* base = (unsigned char*)sT;
  stage_coords<FT>(pw, rows < n ? rows : n, c, base, rws, vec, then);
  __syncthreads();
  const int r = threadIdx.x & 255, h = threadIdx.x >> 8;
  const int hc = cp >> 1, k0 = h * hc;               // this thread's columns [k0, k0 + hc)
  const bool live = r < n && r < rows;
  const int rr = live ? r : 0;
  float v[32];
  {
    float raw[32], p0[32];
#pragma unroll
    for (int k = 0; k < 32; k++) {
      const int kk = min(k0 + k, c - 1);
      raw[k] = *(const float*)(base + rr * rws + 4 * kk);
      p0[k] = *(const float*)(base + 4 * kk);
    }
#pragma unroll
    for (int k = 0; k < 32; k++) v[k] = (live && k < hc && k0 + k < c) ? raw[k] - p0[k] : 0.f;
  }
  if constexpr (TILES) {
    // tile t's column k: thread (t, k) = (tid / 64, tid % 64); 8 tiles x 64 columns
    const int t = threadIdx.x >> 6, k = threadIdx.x & 63;
    if (t < NT) {
      const int kk = min(k, c - 1);
      const float p0k = *(const float*)(base + 4 * kk);
      float col[32];
#pragma unroll
      for (int j = 0; j < 32; j++)
        col[j] = *(const float*)(base + min(32 * t + j, n - 1) * rws + 4 * kk);
      float part[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < 32; j++) part[j & 3] += (32 * t + j < n) ? col[j] - p0k : 0.f;
      sTS[(t + 1) * 64 + k] = k < c ? (part[0] + part[1]) + (part[2] + part[3]) : 0.f;
    }
  }
  __syncthreads();
  float nn = 0.f;
  if (r < rows) {
    bf16* row = sT + r * ct_stride(cp) + k0;
#pragma unroll
    for (int k = 0; k < 32; k += 2) {
      const bf16x2 hi2 = {to_bf16(v[k]), to_bf16(v[k + 1])};
      const float ha = (float)hi2[0], hb = (float)hi2[1];
      const bf16x2 lo2 = {to_bf16(v[k] - ha), to_bf16(v[k + 1] - hb)};
      if (k < hc) {
        *(bf16x2*)(row + k) = hi2;
        *(bf16x2*)(row + cp + k) = lo2;
      }
      const float ta = ha + (float)lo2[0], tb = hb + (float)lo2[1];
      nn = fmaf(ta, ta, nn);
      nn = fmaf(tb, tb, nn);
    }
    if (h == 0) *(u32x4*)(sT + r * ct_stride(cp) + 2 * cp) = u32x4{0u, 0u, 0u, 0u};
  }
  if (r < rows) sNh[h * NP + r] = nn;
  if constexpr (TILES) {
    if (threadIdx.x < 64) {
      float acc = 0.f;
      sTS[threadIdx.x] = 0.f;
#pragma unroll
      for (int t = 0; t < NT; t++) {
        acc += sTS[(t + 1) * 64 + threadIdx.x];
        sTS[(t + 1) * 64 + threadIdx.x] = acc;
      }
    }
  }
  __syncthreads();
  // N_r from the two halves; tile sums of N (rows 32 t .. 32 t + 31 are one
  // half of a wave)
  if (threadIdx.x < rows) {
    float nr = sNh[threadIdx.x] + sNh[NP + threadIdx.x];
    sN[threadIdx.x] = nr;
    if constexpr (TILES) {
#pragma unroll
      for (int o = 16; o >= 1; o >>= 1) nr += __shfl_xor(nr, o);
      if ((threadIdx.x & 31) == 0) sPN[threadIdx.x >> 5] = nr;
    }
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// A window's coordinate table as kept in the caller's workspace for the
// backward (written by the forward, or by field_prep_kernel when the backward
// is asked to build it), windows tab_stride bytes apart (a multiple of 256):
//   rows [NP][2 cp + 8] bf16: the table rows as in LDS (hi | lo | 8 zeros),
//   nrm  [NP] fp32: N_r.
// Both writers run build_table over all NP rows, so the stored bytes do not
// depend on which of them wrote them.
// ---------------------------------------------------------------------------
__host__ __device__ constexpr size_t tab_nrm(int NT, int cp) { return (size_t)NT * 32 * (2 * cp + 8) * 2; }
__host__ __device__ constexpr size_t tab_stride(int NT, int cp) {
  return (tab_nrm(NT, cp) + (size_t)NT * 32 * 4 + 255) / 256 * 256;
}

// Block `part` of `parts` blocks copies its share of the LDS table (rows and
// norms, NP rows) to the window's place tw in the workspace, 16 bytes per
// store.  No wait: nothing in the block reads it back.
template <int NT>
__device__ __forceinline__ void store_table(const bf16* sT, const float* sN,
                                            unsigned char* __restrict__ tw, int cp, int part,
                                            int parts) {
  constexpr int NP = NT * 32;
  const int rowp = NP * (2 * cp + 8) * 2 / 16, pieces = rowp + NP * 4 / 16;
  const int per = (pieces + parts - 1) / parts;
  const int lo = part * per, hi = min(pieces, lo + per);
  for (int i = lo + (int)threadIdx.x; i < hi; i += FT) {
    const u32x4 v = i < rowp ? ((const u32x4*)sT)[i] : ((const u32x4*)sN)[i - rowp];
    ((u32x4*)tw)[i] = v;
  }
}

// Block = window b, FT threads: the table built in LDS as the forward builds
// it, then copied to the workspace.
template <int NT>
__global__ __launch_bounds__(FT) void field_prep_kernel(const float* __restrict__ p,
                                                       unsigned char* __restrict__ tab, int n,
                                                       int c, int cp, int vec) {
  constexpr int NP = NT * 32;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  float* sN = (float*)smem;
  float* sNh = sN + NP;                       // [2][NP]
  bf16* sT = (bf16*)(sNh + 2 * NP);
  const int b = blockIdx.x;
  build_table<NT, false>(p + (size_t)b * n * c, n, c, cp, NP, sT, sN, sNh, nullptr, nullptr, vec,
                         NoIssue{});
  store_table<NT>(sT, sN, tab + (size_t)b * tab_stride(NT, cp), cp, 0, 1);
}

// Rows [0, rows) of window b's stored table and their norms, into LDS.  Every
// load is issued before the first LDS write; `then` runs after the loads are
// issued.  Ends with a barrier.
template <int NT, class Then>
__device__ __forceinline__ void load_table(const unsigned char* __restrict__ tw, int cp, int rows,
                                           bf16* sT, float* sN, Then then) {
  constexpr int MAXP = (NT * 32 * 136 * 2 / 16 + FT - 1) / FT;   // 16-byte pieces per thread
  const int pieces = rows * (2 * cp + 8) * 2 / 16;
  u32x4 v[MAXP];
#pragma unroll
  for (int u = 0; u < MAXP; u++)
    v[u] = ((const u32x4*)tw)[min((int)threadIdx.x + FT * u, pieces - 1)];
  const float* nrm = (const float*)(tw + tab_nrm(NT, cp));
  const float nv = nrm[min((int)threadIdx.x, rows - 1)];
  then();
#pragma unroll
  for (int u = 0; u < MAXP; u++)
    if ((int)threadIdx.x + FT * u < pieces) ((u32x4*)sT)[threadIdx.x + FT * u] = v[u];
  if ((int)threadIdx.x < rows) sN[threadIdx.x] = nv;
  __syncthreads();
}

// One slab of SW columns (SW / 64 tiles of 64 columns; src: row 0's first
// column, rows `stride` apart), rows [0, NT * 32), in two steps: issue every
// load into registers (unconditional, rows clamped into the window), and later
// write them to swizzled LDS tiles NT * 32 * 64 elements apart, rows >= n as
// zero.  The loads can then overlap other work; vector-memory waits are in
// issue order, so loads issued before them do not delay later ones' use.
template <int NT, int SW>
struct Slab {
  static constexpr int NP = NT * 32, TP = NP * 8, PIECES = TP * (SW / 64),
                       PER = (PIECES + FT - 1) / FT;
  u32x4 v[PER];
  __device__ __forceinline__ void issue(const bf16* __restrict__ src, size_t stride, int n) {
#pragma unroll
    for (int j = 0; j < PER; j++) {
      const int pi = min((int)threadIdx.x + FT * j, PIECES - 1), tl = pi / TP,
                r = (pi % TP) >> 3, pc = pi & 7;
      v[j] = *(const u32x4*)(src + (size_t)min(r, n - 1) * stride + 64 * tl + 8 * pc);
    }
  }
  __device__ __forceinline__ void store(bf16* tile, int n) {
#pragma unroll
    for (int j = 0; j < PER; j++) {
      const int pi = threadIdx.x + FT * j, tl = pi / TP, r = (pi % TP) >> 3, pc = pi & 7;
      if (pi < PIECES)
        *(u32x4*)(tile + tl * NP * 64 + att_off(r, 8 * pc)) =
            r < n ? v[j] : u32x4{0u, 0u, 0u, 0u};
    }
  }
};

// s_waitcnt vmcnt(n) for a wave-uniform runtime n <= 15.
__device__ __forceinline__ void wait_vmcnt_upto(int n) {
  switch (n) {
    case 0: wait_vmcnt<0>(); break;
    case 1: wait_vmcnt<1>(); break;
    case 2: wait_vmcnt<2>(); break;
    case 3: wait_vmcnt<3>(); break;
    case 4: wait_vmcnt<4>(); break;
    case 5: wait_vmcnt<5>(); break;
    case 6: wait_vmcnt<6>(); break;
    case 7: wait_vmcnt<7>(); break;
    case 8: wait_vmcnt<8>(); break;
    case 9: wait_vmcnt<9>(); break;
    case 10: wait_vmcnt<10>(); break;
    default: wait_vmcnt<0>(); break;
  }
}

// The 32-row tile a wave of an 8-wave block works on: waves w and w + 4 share
// a SIMD and take tiles w and 7 - w, whose causal work (w + 1 and 8 - w tiles
// of the other side) sums to the same 9 for every SIMD at 8 tiles.
__device__ __forceinline__ int wave_tile(int wave) { return wave < 4 ? wave : 11 - wave; }

// The lane's own row of the table as B-operand fragments: hi and lo halves,
// the 8 components of each 16-wide k step that lane half h contributes.
struct RowFrags {
  bf16x8 hi[4], lo[4];
};
__device__ __forceinline__ void row_frags(const bf16* sT, int rs, int cp, int r, int half,
                                          RowFrags& f) {
#pragma unroll
  for (int ks = 0; ks < 4; ks++) {
    f.hi[ks] = bf16x8{};
    f.lo[ks] = bf16x8{};
    if (16 * ks < cp) {
      f.hi[ks] = ct_row(sT, rs, r, 16 * ks, half);
      f.lo[ks] = ct_row(sT, rs, r, cp + 16 * ks, half);
    }
  }
}

// Gram tile of table rows t0 .. t0 + 31 (A operand) against the lane's row
// fragments f (B operand): hi.hi, then key-lo . query-hi, then key-hi .
// query-lo, so that both orientations (A_IS_KEY: the tile holds keys, f the
// query; else the tile holds queries, f the key) add the same products in the
// same order.
template <bool A_IS_KEY>
__device__ __forceinline__ f32x16 gram_tile(const bf16* sT, int rs, int cp, int t0,
                                            const RowFrags& f, int lane) {
  f32x16 acc = {};
#pragma unroll
  for (int ks = 0; ks < 4; ks++) {
    if (16 * ks < cp) {
      const bf16x8 ahi = ct_frag(sT, rs, t0, 16 * ks, lane);
      const bf16x8 alo = ct_frag(sT, rs, t0, cp + 16 * ks, lane);
      acc = mfma32(ahi, f.hi[ks], acc);
      if constexpr (A_IS_KEY) {
        acc = mfma32(alo, f.hi[ks], acc);
        acc = mfma32(ahi, f.lo[ks], acc);
      } else {
        acc = mfma32(ahi, f.lo[ks], acc);
        acc = mfma32(alo, f.hi[ks], acc);
      }
    }
  }
  return acc;
}

// Gram tile G^T[key][query] for keys kt*32.. (A operand, table rows) and the
// lane's query q (B operand): hi.hi + lo.hi + hi.lo, in that order.
__device__ __forceinline__ f32x16 gram_keys(const bf16* sT, int rs, int cp, int kt, int q,
                                            int lane) {
  RowFrags f;
  row_frags(sT, rs, cp, q, lane >> 5, f);
  return gram_tile<true>(sT, rs, cp, kt * 32, f, lane);
}

// Scale of the logits of a row with mean squared distance m: a = -D * scale.
// A positive mean below 2^-100 is taken as 2^-100 (such coordinates are not
// resolved by fp32 squared distances anyway), which keeps the scale finite for
// tau >= 2^-24.
__device__ __forceinline__ float clamped_mean(float m) { return fmaxf(m, 0x1p-100f); }
__device__ __forceinline__ float logit_scale(float m, float inv_tau, int scaled) {
  if (!scaled) return inv_tau;
  return m > 0.f ? inv_tau / clamped_mean(m) : 0.f;
}

// Dynamic LDS layouts (bytes).
constexpr int cmax(int a, int b) { return a > b ? a : b; }
constexpr int table_bytes(int NT, int cp) { return NT * 32 * (2 * cp + 8) * 2; }
// (the forward's last phase reuses the space for (NT + 1) / 2 partial
// readouts of (SW / 32 * 16 + 2) x 64 floats)
constexpr int fwd_lds_bytes(int NT, int SW, int cp) {
  return cmax(NT * 32 * SW * 2 + NT * 32 * 4 + (NT + 1) * 64 * 4 + 16 * 4 + 2 * NT * 32 * 4 +
                  table_bytes(NT, cp),
              (NT + 1) / 2 * (SW / 32 * 16 + 2) * 64 * 4);
}
constexpr int prep_lds_bytes(int NT, int cp) { return 3 * NT * 32 * 4 + table_bytes(NT, cp); }
constexpr int dx_lds_bytes(int NT, int SW) { return NT * 32 * SW * 2; }

// Transposed coupling tiles as the rows kernel writes them and the dx kernel
// reads them: per window NT x NT tiles of 32 x 32 bf16 (tile (kt, qt) at kt *
// NT + qt; only qt >= kt written), row = key, and within a row the 32
// queries in the order of a key lane's score registers: query 8 g + 4 h + r
// (g, r < 4, h < 2) at 16 h + 4 g + r.  A lane of half h then finds its 16
// couplings of a tile in 32 contiguous bytes.
__device__ __forceinline__ int ct_pos(int lq) { return 16 * ((lq >> 2) & 1) + 4 * (lq >> 3) + (lq & 3); }
// rows kernel: NS stages of [x rows (NT * 32)][64] + [dy rows (32)][64] bf16,
// the coordinate table in the same space before the stages are used, then
// the norms and the per-wave row sums.  At NS = 2 a block needs at most 77
// KB, so two blocks share a CU.
constexpr int rows_stage_elems(int NT) { return (NT * 32 + 32) * 64; }
constexpr int rows_lds_bytes(int NT, int NS, int cp) {
  return cmax(NS * rows_stage_elems(NT) * 2, table_bytes(NT, cp)) + NT * 32 * 4 + 2 * 8 * 32 * 4;
}
constexpr int ROWS_NS = 2;
// coordinate kernel: E tile [32][NP + 1] fp32, coordinates [NP][ck + 1] fp32,
// row-sum parts [16][32], and the per-wave partial products [4][32][ck + 1]
// (in the E tile's space where they fit, else after the rest)
constexpr bool coord_part_in_e(int NT, int ck) { return 4 * 32 * (ck + 1) <= 32 * (NT * 32 + 1); }
constexpr int coord_lds_bytes(int NT, int ck) {
  return 32 * (NT * 32 + 1) * 4 + NT * 32 * (ck + 1) * 4 + 16 * 32 * 4 +
         (coord_part_in_e(NT, ck) ? 0 : 4 * 32 * (ck + 1) * 4);
}

// ---------------------------------------------------------------------------
// Forward.  Block = (window b, slab s of SW columns), 8 waves; grid = batch *
// slabs, dealt so that the slabs of one window share an XCD (its coordinates
// are read from HBM once).
//
// Work plan: the query tiles pair up as (i, NT - 1 - i), i < ceil(NT / 2),
// and the two waves of SIMD i (waves i and i + 4) share pair i's causal work
// (NT + 1 key tiles) evenly: wave i takes query tile i whole (when it differs
// from the other) and key tiles [0, sA) of query tile qb = NT - 1 - i; wave
// i + 4 takes key tiles [sA, qb] of qb, the diagonal first.  The two partial
// readouts of qb (numerator and sums) meet in LDS at the end.
//
// A row's mean is known before any exponential: the earlier tiles' part from
// the tile sums (build_table), the diagonal tile's from its Gram tile (wave i
// recomputes qb's for its share).  Then per key tile: D = N_key + N_q - 2 G
// (one add, one FMA), the exponential of D k2, its sum (and, PARTNERS, the
// entropy term), and the tile's product with the x slab; the query's table
// fragments stay in registers.
// ---------------------------------------------------------------------------
template <int NT, int SW, bool PARTNERS>
__global__ __launch_bounds__(FT) void field_fwd_kernel(
    const float* __restrict__ p, unsigned char* __restrict__ tab, const bf16* __restrict__ x,
    bf16* __restrict__ y, float* __restrict__ row_mean, float* __restrict__ lse,
    float* __restrict__ partners, int n, int c, int cp, int width, int slabs, float inv_tau,
    int scaled, int vec) {
  constexpr int NP = NT * 32, DT = SW / 32;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  bf16* sX = (bf16*)smem;
  float* sN = (float*)(smem + NP * SW * 2);
  float* sTS = sN + NP;                       // [NT + 1][64]
  float* sPN = sTS + (NT + 1) * 64;           // [16]
  float* sNh = sPN + 16;                      // [2][NP]
  bf16* sT = (bf16*)(sNh + 2 * NP);
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int b = lin / slabs, s = lin % slabs;
  const int lane = threadIdx.x & 63, half = lane >> 5, lq = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int rs = ct_stride(cp);
  Slab<NT, SW> slab;
  build_table<NT, true>(p + (size_t)b * n * c, n, c, cp, NP, sT, sN, sNh, sTS, sPN, vec,
                        [&] { slab.issue(x + (size_t)b * n * width + (size_t)s * SW, width, n); });
  // the window's slab blocks share the copy of its table for the backward
  store_table<NT>(sT, sN, tab + (size_t)b * tab_stride(NT, cp), cp, s, slabs);
  // the plan of this wave
  const int pi = wave & 3;
  const bool roleA = wave < 4, active = pi < (NT + 1) / 2;
  const int qa = pi, qb = NT - 1 - pi;
  const int sA = qa < qb ? (qb - qa) / 2 : (qb + 1) / 2;
  const bool own = roleA && active && qa < qb;          // wave A's whole tile
  f32x16 o[DT];
  float z = 0.f, za = 0.f;
  auto reset = [&] {
#pragma unroll
    for (int dt = 0; dt < DT; dt++) o[dt] = f32x16{};
    z = 0.f;
    za = 0.f;
  };
  // sum of D over the keys of the tiles before Q
  auto row_off = [&](const RowFrags& fr, int Q, float nqv) {
    float dotp = 0.f;
#pragma unroll
    for (int ks = 0; ks < 4; ks++) {
      if (16 * ks < cp) {
        const float* ts = sTS + Q * 64 + 16 * ks + 8 * half;
        const f32x4 t0 = *(const f32x4*)ts, t1 = *(const f32x4*)(ts + 4);
#pragma unroll
        for (int e = 0; e < 8; e++)
          dotp = fmaf((float)fr.hi[ks][e] + (float)fr.lo[ks][e], e < 4 ? t0[e] : t1[e - 4], dotp);
      }
    }
    dotp += __shfl_xor(dotp, 32);
    float pn = 0.f;
    for (int t = 0; t < Q; t++) pn += sPN[t];
    return (float)(32 * Q) * nqv + pn - 2.f * dotp;
  };
  // the diagonal tile of Q: D (q itself and keys after q set to 0) and its row sum
  auto diag = [&](const RowFrags& fr, int Q, float nqv, f32x16& d) {
    d = gram_tile<true>(sT, rs, cp, Q * 32, fr, lane);
    float dsum = 0.f;
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const f32x4 n4 = *(const f32x4*)(sN + Q * 32 + 8 * g + 4 * half);
#pragma unroll
      for (int r = 0; r < 4; r++) {
        const int e = 4 * g + r;
        float dv = fmaf(d[e], -2.f, n4[r] + nqv);
        if (8 * g + 4 * half + r >= lq) dv = 0.f;
        d[e] = dv;
        dsum += dv;
      }
    }
    return dsum + __shfl_xor(dsum, 32);
  };
  auto readout = [&](f32x16& pe, int kt) {
#pragma unroll
    for (int mm = 0; mm < 2; mm++) {
      const bf16x8 pf = att_pack(pe, mm);
#pragma unroll
      for (int dt = 0; dt < DT; dt++)
        o[dt] = mfma32(att_trfrag(sX + (dt / 2) * NP * 64, kt * 32 + 16 * mm, 32 * (dt % 2), lane),
                       pf, o[dt]);
    }
  };
  // exponentials of a tile of D (diagonal: masked), their sums
  auto expo = [&](f32x16& d, float k2, bool is_diag) {
#pragma unroll
    for (int e = 0; e < 16; e++) {
      const float a = d[e] * k2;
      float pe = __builtin_amdgcn_exp2f(a);
      if (is_diag && att_masked(e, lane)) pe = 0.f;
      d[e] = pe;
      z += pe;
      if constexpr (PARTNERS) za += pe * a;
    }
  };
  // one off-diagonal key tile of query tile Q
  auto tile = [&](const RowFrags& fr, int kt, float nqv, float k2) {
    f32x16 acc = gram_tile<true>(sT, rs, cp, kt * 32, fr, lane);
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const f32x4 n4 = *(const f32x4*)(sN + kt * 32 + 8 * g + 4 * half);
#pragma unroll
      for (int r = 0; r < 4; r++) acc[4 * g + r] = fmaf(acc[4 * g + r], -2.f, n4[r] + nqv);
    }
    expo(acc, k2, false);
    readout(acc, kt);
  };
  auto finish = [&](int Q, float m) {
    const int q = Q * 32 + lq;
    if (q >= n) return;
    // O^T register e of lane l: query q, column 32 dt + 8 (e / 4) + 4 half + e % 4
    const float inv = 1.f / z;
    bf16* yrow = y + ((size_t)b * n + q) * width + (size_t)s * SW;
#pragma unroll
    for (int dt = 0; dt < DT; dt++)
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const bf16x4 v = {to_bf16(o[dt][4 * g] * inv), to_bf16(o[dt][4 * g + 1] * inv),
                          to_bf16(o[dt][4 * g + 2] * inv), to_bf16(o[dt][4 * g + 3] * inv)};
        *(bf16x4*)(yrow + 32 * dt + 8 * g + 4 * half) = v;
      }
    if (s == 0 && half == 0) {
      const float l2z = __builtin_amdgcn_logf(z);       // log2 Z
      const size_t at = (size_t)b * n + q;
      row_mean[at] = m;
      lse[at] = l2z * LN2;
      if constexpr (PARTNERS) partners[at] = __builtin_amdgcn_exp2f(l2z - za * inv);
    }
  };

  // before the slab barrier: every wave's diagonal tile (wave A: its own
  // tile's, and qb's row sum for the mean of its share)
  RowFrags fa, fb;
  float nqa = 0.f, nqb = 0.f, ma = 0.f, mb = 0.f, k2a = 0.f, k2b = 0.f;
  f32x16 dA = {}, dB = {};
  if (active) {
    row_frags(sT, rs, cp, qb * 32 + lq, half, fb);
    nqb = sN[qb * 32 + lq];
    const float dsb = diag(fb, qb, nqb, dB);
    mb = (row_off(fb, qb, nqb) + dsb) / (float)(qb * 32 + lq + 1);
    k2b = -logit_scale(mb, inv_tau, scaled) * LOG2E;
    if (own) {
      row_frags(sT, rs, cp, qa * 32 + lq, half, fa);
      nqa = sN[qa * 32 + lq];
      const float dsa = diag(fa, qa, nqa, dA);
      ma = (row_off(fa, qa, nqa) + dsa) / (float)(qa * 32 + lq + 1);
      k2a = -logit_scale(ma, inv_tau, scaled) * LOG2E;
    }
  }
  slab.store(sX, n);
  __syncthreads();
  if (own) {                                  // wave A: query tile qa whole
    reset();
    expo(dA, k2a, true);
    readout(dA, qa);
    for (int kt = qa - 1; kt >= 0; kt--) tile(fa, kt, nqa, k2a);
    z += __shfl_xor(z, 32);
    if constexpr (PARTNERS) za += __shfl_xor(za, 32);
    finish(qa, ma);
  }
  reset();
  if (active) {
    if (roleA) {                              // wave A: key tiles [0, sA) of qb
      for (int kt = 0; kt < sA; kt++) tile(fb, kt, nqb, k2b);
    } else {                                  // wave B: key tiles [sA, qb] of qb
      expo(dB, k2b, true);
      readout(dB, qb);
      for (int kt = qb - 1; kt >= sA; kt--) tile(fb, kt, nqb, k2b);
    }
  }
  // wave A's partial readout of qb joins wave B's through LDS (the slab and
  // the table are no longer read)
  __syncthreads();
  float* part = (float*)smem + pi * (DT * 16 + 2) * 64;
  if (active && roleA) {
#pragma unroll
    for (int dt = 0; dt < DT; dt++)
#pragma unroll
      for (int e = 0; e < 16; e++) part[(dt * 16 + e) * 64 + lane] = o[dt][e];
    part[DT * 16 * 64 + lane] = z;
    part[(DT * 16 + 1) * 64 + lane] = za;
  }
  __syncthreads();
  if (active && !roleA) {
#pragma unroll
    for (int dt = 0; dt < DT; dt++)
#pragma unroll
      for (int e = 0; e < 16; e++) o[dt][e] += part[(dt * 16 + e) * 64 + lane];
    z += part[DT * 16 * 64 + lane];
    za += part[(DT * 16 + 1) * 64 + lane];
    z += __shfl_xor(z, 32);
    if constexpr (PARTNERS) za += __shfl_xor(za, 32);
    finish(qb, mb);
  }
}

// ---------------------------------------------------------------------------
// Backward, rows.  Block = (window b, query tile qt), the heaviest tiles of a
// window first; 8 waves, wave w owning key tile w (w <= qt).  Two blocks share
// a CU (the grid's second half, the light tiles, beside the first), so one
// block's set-up and reductions overlap the other's streaming.
// The couplings, their squared distances and the row sums come first, from
// the coordinate table (loaded into the stage space).  Then dP^T[key][q] =
// x_key . dy_q sums over the width in 64-column steps: each step's x rows
// [0, 32 (qt + 1)) and the tile's 32 dy rows go global -> LDS by DMA
// (coalesced, 8 rows of 128 bytes per instruction, swizzled as the 64-column
// tiles), NS stages in flight, the instructions of a step dealt over the 8
// waves.  The per-row sums Delta and sum(da D) across the waves go through
// LDS.
// ---------------------------------------------------------------------------
template <int NT, int NS>
__global__ __launch_bounds__(FT) void field_bwd_rows_kernel(
    const unsigned char* __restrict__ tab, const bf16* __restrict__ x, const bf16* __restrict__ dy,
    const float* __restrict__ row_mean, const float* __restrict__ lse, float* __restrict__ ddt,
    bf16* __restrict__ ct, int n, int cp, int width, float inv_tau, int scaled) {
  constexpr int NP = NT * 32, STAGE = rows_stage_elems(NT);
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  bf16* sStage = (bf16*)smem;
  bf16* sT = sStage;                                  // the table, until the first DMA
  float* sN = (float*)(smem + cmax(NS * STAGE * 2, table_bytes(NT, cp)));
  float* sRed = sN + NP;                              // [2][8 waves][32]
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int b = lin / NT, qt = NT - 1 - lin % NT;
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int rs = ct_stride(cp);
  const int q = qt * 32 + (lane & 31);
  const bool qvalid = q < n;
  const bool own = wave <= qt;                        // this wave's key tile kt = wave
  const int steps = width / 64;
  // DMA plan of one step: instructions u < XI are x rows 8u .. 8u + 7, the
  // next 4 the tile's dy rows; wave w issues u = w, w + 8, ...  Rows past the
  // window read its last row (finite values that only reach couplings the
  // causal mask removes, or rows whose results are not used).
  const int XI = (qt + 1) * 4, TI = XI + 4;
  const int cnt = wave < TI ? (TI - 1 - wave) / 8 + 1 : 0;
  const bf16* xw = x + (size_t)b * n * width;
  const bf16* dyw = dy + (size_t)b * n * width;
  auto dma = [&](int st, int slot) {
    bf16* dst = sStage + slot * STAGE;
#pragma unroll
    for (int v = 0; v < 5; v++) {
      if (v < cnt) {
        const int u = wave + 8 * v;
        const int lr = 8 * u + (lane >> 3);               // row in the stage (x rows, then dy)
        const int tr = u < XI ? lr : qt * 32 + (lr - 8 * XI);   // row in the window
        const int gr = tr < n ? tr : n - 1;
        const int tile_row = u < XI ? lr : lr - 8 * XI;
        const int piece = (lane & 7) ^ att_sw(tile_row);
        const bf16* src = (u < XI ? xw : dyw) + (size_t)gr * width + st * 64 + 8 * piece;
        bf16* d0 = u < XI ? dst + u * 512 : dst + NP * 64 + (u - XI) * 512;
        dma16(src, d0);
      }
    }
  };
  const float m_ld = row_mean[(size_t)b * n + min(q, n - 1)];
  const float l_ld = lse[(size_t)b * n + min(q, n - 1)];
  load_table<NT>(tab + (size_t)b * tab_stride(NT, cp), cp, (qt + 1) * 32, sT, sN, NoIssue{});
  const float m = qvalid ? m_ld : 0.f;
  const float l2 = qvalid ? l_ld * LOG2E : 0.f;
  const float scale = qvalid ? logit_scale(m, inv_tau, scaled) : 0.f;
  const float k2 = -scale * LOG2E;
  const float nq = sN[q];
  f32x16 dd = {}, cc = {}, g = {};
  if (own) {
    f32x16 acc = gram_keys(sT, rs, cp, wave, q, lane);
#pragma unroll
    for (int gq = 0; gq < 4; gq++) {
      const f32x4 n4 = *(const f32x4*)(sN + wave * 32 + 8 * gq + 4 * half);
#pragma unroll
      for (int r = 0; r < 4; r++) {
        const int e = 4 * gq + r;
        const int lk = 8 * gq + 4 * half + r, lq = lane & 31;   // within the tiles
        const bool diag = wave == qt;
        float d = fmaf(acc[e], -2.f, n4[r] + nq);
        if (diag && lk >= lq) d = 0.f;                 // q itself, keys after q
        dd[e] = d;
        cc[e] = diag && lk > lq ? 0.f : __builtin_amdgcn_exp2f(d * k2 - l2);
      }
    }
    // C^T tile (key tile = wave, query tile qt) for the dx kernel
    bf16* cw = ct + ((size_t)b * NT * NT + wave * NT + qt) * 1024 + ct_pos(lane & 31);
#pragma unroll
    for (int e = 0; e < 16; e++) cw[(8 * (e >> 2) + 4 * half + (e & 3)) * 32] = to_bf16(cc[e]);
  }
  __syncthreads();                                    // the table's space becomes the stages
#pragma unroll
  for (int st = 0; st < NS - 1; st++)
    if (st < steps) dma(st, st);
  for (int st = 0; st < steps; st++) {
    // this wave's DMA of step st has landed (those of the next NS - 2 steps may
    // still be in flight); after the barrier every wave's has, and every wave
    // is done with step st - 1, whose slot the next DMA overwrites
    const int later = min(NS - 2, steps - 1 - st);
    wait_vmcnt_upto(cnt * later);
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (st + NS - 1 < steps) dma(st + NS - 1, (st + NS - 1) % NS);
    if (own) {
      const bf16* cur = sStage + (st % NS) * STAGE;
#pragma unroll
      for (int ks = 0; ks < 4; ks++)
        g = mfma32(att_frag(cur, wave * 32, 16 * ks, lane),
                   att_frag(cur + NP * 64, 0, 16 * ks, lane), g);
    }
  }
  // Delta_q = sum_j C dP (in-lane, the lane ^ 32 exchange, then the 8 waves)
  float del = 0.f;
#pragma unroll
  for (int e = 0; e < 16; e++) del += cc[e] * g[e];
  del += __shfl_xor(del, 32);
  if (half == 0) sRed[wave * 32 + lane] = del;
  __syncthreads();
  del = 0.f;
#pragma unroll
  for (int w = 0; w < 8; w++) del += sRed[w * 32 + (lane & 31)];
  float tdm = 0.f;
#pragma unroll
  for (int e = 0; e < 16; e++) {
    const float da = cc[e] * (g[e] - del);
    g[e] = da;
    tdm += da * dd[e];
  }
  tdm += __shfl_xor(tdm, 32);
  if (half == 0) sRed[256 + wave * 32 + lane] = tdm;
  __syncthreads();
  if (!own) return;
  tdm = 0.f;
#pragma unroll
  for (int w = 0; w < 8; w++) tdm += sRed[256 + w * 32 + (lane & 31)];
  // dD = -scale da + [scaled, m > 0] (scale / m) (sum_j da D) / (q + 1)
  const float coef =
      (scaled && m > 0.f) ? scale * tdm / clamped_mean(m) / (float)(q + 1) : 0.f;
  float* dw = ddt + (size_t)b * NP * NP;
#pragma unroll
  for (int e = 0; e < 16; e++) {
    const int kk = wave * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
    dw[(size_t)kk * NP + q] = kk > q ? 0.f : -scale * g[e] + coef;
  }
}

// ---------------------------------------------------------------------------
// Backward, dx.  Block = (window b, slab s of SW columns), 8 waves, wave w on
// key tile wave_tile(w), a lane one key j; the couplings come as the rows
// kernel wrote them (bf16, the lane's 16 queries of a tile in one 32-byte
// load, PF tiles in flight), and dx^T[col][j] += dy^T[col][q] C[q][j] as in
// the attention core's dV, dy^T read transposed from the LDS slab.
// ---------------------------------------------------------------------------
template <int NT, int SW>
__global__ __launch_bounds__(FT) void field_bwd_dx_kernel(const bf16* __restrict__ ct,
                                                         const bf16* __restrict__ dy,
                                                         bf16* __restrict__ dx, int n, int width,
                                                         int slabs) {
  constexpr int NP = NT * 32, DT = SW / 32, PF = NT < 3 ? NT : 3;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  bf16* sDY = (bf16*)smem;
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int b = lin / slabs, s = lin % slabs;
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int kt = wave_tile(wave);
  Slab<NT, SW> slab;
  slab.issue(dy + (size_t)b * n * width + (size_t)s * SW, width, n);
  // tile (kt, kt + u) for u < NT - kt; past that (and for waves without a key
  // tile) the loads are clamped to tile (min(kt, NT - 1), NT - 1), in bounds
  const bf16* cw = ct + ((size_t)b * NT * NT + (size_t)min(kt, NT - 1) * NT) * 1024 +
                   (lane & 31) * 32 + 16 * half;
  bf16x8 cf[PF][2];
  auto fetch = [&](int u, bf16x8* dst) {
    const bf16* src = cw + (size_t)min(kt + u, NT - 1) * 1024;
    dst[0] = *(const bf16x8*)src;
    dst[1] = *(const bf16x8*)(src + 8);
  };
#pragma unroll
  for (int u = 0; u < PF; u++) fetch(u, cf[u]);
  slab.store(sDY, n);
  __syncthreads();
  if (kt >= NT) return;
  f32x16 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; dt++) o[dt] = f32x16{};
#pragma unroll
  for (int u = 0; u < NT; u++) {
    if (u < NT - kt) {
      const int qt = kt + u;
      bf16x8 cur[2] = {cf[u % PF][0], cf[u % PF][1]};
      if (u + PF < NT) fetch(u + PF, cf[u % PF]);
#pragma unroll
      for (int mm = 0; mm < 2; mm++)
#pragma unroll
        for (int dt = 0; dt < DT; dt++)
          o[dt] = mfma32(att_trfrag(sDY + (dt / 2) * NP * 64, qt * 32 + 16 * mm, 32 * (dt % 2), lane),
                         cur[mm], o[dt]);
    }
  }
  const int j = kt * 32 + (lane & 31);
  if (j >= n) return;
  bf16* xrow = dx + ((size_t)b * n + j) * width + (size_t)s * SW;
#pragma unroll
  for (int dt = 0; dt < DT; dt++)
#pragma unroll
    for (int gq = 0; gq < 4; gq++) {
      const bf16x4 v = {to_bf16(o[dt][4 * gq]), to_bf16(o[dt][4 * gq + 1]),
                        to_bf16(o[dt][4 * gq + 2]), to_bf16(o[dt][4 * gq + 3])};
      *(bf16x4*)(xrow + 32 * dt + 8 * gq + 4 * half) = v;
    }
}

// ---------------------------------------------------------------------------
// Backward, coordinates.  Block = (window b, row tile t), 8 waves: E[i][j] for
// the tile's 32 rows i and every j (dD[i][j] = ddt[j][i] for j < i, dD[j][i] =
// ddt[i][j] for j > i; 0 at j = i and outside the window) into LDS; then
//   dp_i = 2 (sum_j E[i][j]) p'_i - 2 sum_j E[i][j] p'_j,  p' = p - p_0,
// the second sum on the fp32 matrix cores (32 x 32 x 2: A = p'^T, B = E^T),
// waves 0-3 taking a quarter of the j range each; partial products meet in
// LDS.
// ---------------------------------------------------------------------------
template <int NT, int CK>
__global__ __launch_bounds__(FT) void field_bwd_coord_kernel(const float* __restrict__ p,
                                                            const float* __restrict__ ddt,
                                                            float* __restrict__ dp, int n,
                                                            int c, int vec) {
  constexpr int NP = NT * 32, ES = NP + 1, CKP = CK + 1;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  float* sE = (float*)smem;                          // [32][ES]
  float* sP = sE + 32 * ES;                          // [NP][CKP]
  float* sRowPart = sP + NP * CKP;                   // [16][32]
  float* sPart = coord_part_in_e(NT, CK) ? sE : sRowPart + 16 * 32;   // [4][32][CKP]
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int b = lin / NT, t = lin % NT;
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const float* pw = p + (size_t)b * n * c;
  const float* dw = ddt + (size_t)b * NP * NP;
  // E in three parts, 16-byte loads where the rows are contiguous, every load
  // unconditional (indices inside the window's NP x NP workspace) and the
  // entries outside E (j = i, outside the window) replaced by 0 afterwards:
  //   j < 32 t: ddt[j][32 t .. 32 t + 31] (i consecutive): 8 float4 per j,
  //     group g = tid + 512 u, j = g / 8;
  //   the diagonal tile: ddt[j][i] for j < i, ddt[i][j] for j > i, scalar;
  //   j >= 32 (t + 1): ddt[i][j] (j consecutive): wave w takes rows
  //     ii = 4 w .. 4 w + 3, lane l the float4 at j = 32 (t + 1) + 4 l.
  constexpr int PA = (NT + 1) / 2;
  const int na = (t * 32 * 8 + FT - 1) / FT, j0 = (t + 1) * 32;
  f32x4 ea[PA], eb[4];
  float ed[2];
#pragma unroll
  for (int u = 0; u < PA; u++) {
    const int g = min((int)threadIdx.x + FT * u, max(t * 32 * 8 - 1, 0));
    ea[u] = *(const f32x4*)(dw + (size_t)(g >> 3) * NP + 32 * t + 4 * (g & 7));
  }
#pragma unroll
  for (int u = 0; u < 2; u++) {
    const int e = threadIdx.x + FT * u, jj = e >> 5, ii = e & 31;
    const int i = 32 * t + ii, j = 32 * t + jj;
    ed[u] = dw[jj < ii ? (size_t)j * NP + i : (size_t)i * NP + j];
  }
#pragma unroll
  for (int u = 0; u < 4; u++) {
    const int ii = 4 * wave + u, j = min(j0 + 4 * lane, NP - 4);
    eb[u] = *(const f32x4*)(dw + (size_t)(32 * t + ii) * NP + j);
  }
  // coordinates: rows past the window zero (their E entries are 0, so they
  // must be finite); columns past c are left as they are (they only reach
  // output rows that are not used)
  for (int idx = threadIdx.x; idx < (NP - n) * CKP; idx += FT) sP[n * CKP + idx] = 0.f;
  stage_coords<FT>(pw, n, c, (unsigned char*)sP, CKP * 4, vec);
#pragma unroll
  for (int u = 0; u < PA; u++) {
    if (u < na && (int)threadIdx.x + FT * u < t * 32 * 8) {
      const int g = threadIdx.x + FT * u, j = g >> 3;
#pragma unroll
      for (int e = 0; e < 4; e++) {
        const int ii = 4 * (g & 7) + e, i = 32 * t + ii;
        sE[ii * ES + j] = (i < n && j < n) ? ea[u][e] : 0.f;
      }
    }
  }
#pragma unroll
  for (int u = 0; u < 2; u++) {
    const int e = threadIdx.x + FT * u, jj = e >> 5, ii = e & 31;
    const int i = 32 * t + ii, j = 32 * t + jj;
    sE[ii * ES + j] = (i < n && j < n && jj != ii) ? ed[u] : 0.f;
  }
#pragma unroll
  for (int u = 0; u < 4; u++) {
    const int ii = 4 * wave + u, i = 32 * t + ii, j = j0 + 4 * lane;
    if (j < NP) {
#pragma unroll
      for (int e = 0; e < 4; e++) sE[ii * ES + j + e] = (i < n && j + e < n) ? eb[u][e] : 0.f;
    }
  }
  __syncthreads();
  {
    // row sums: lane group of 32 = the 32 rows at one j, 16 groups over j
    const int ii = threadIdx.x & 31, part = threadIdx.x >> 5;
    float rsum = 0.f;
    for (int j = part; j < NP; j += 16) rsum += sE[ii * ES + j];
    sRowPart[part * 32 + ii] = rsum;
  }
  constexpr int JW = NP / 4;                         // j range of one of waves 0-3
  f32x16 acc[CK / 32];
#pragma unroll
  for (int kc = 0; kc < CK / 32; kc++) acc[kc] = f32x16{};
  if (wave < 4) {
    float p0[CK / 32];                               // p_0 at this lane's coordinates
#pragma unroll
    for (int kc = 0; kc < CK / 32; kc++) p0[kc] = sP[kc * 32 + (lane & 31)];
    for (int js = 0; js < JW; js += 2) {
      const int j = wave * JW + js + half;
      const float bv = sE[(lane & 31) * ES + j];     // B[k = half][col i] = E[i][j]
#pragma unroll
      for (int kc = 0; kc < CK / 32; kc++) {
        // A[row k][half] = p'_j[k] = p_j[k] - p_0[k]
        const float av = sP[j * CKP + kc * 32 + (lane & 31)] - p0[kc];
        acc[kc] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc[kc], 0, 0, 0);
      }
    }
  }
  __syncthreads();                                   // sE may be reused for the partials
  // register e: coordinate k = kc*32 + 8 (e/4) + 4 half + e%4, row i = lane % 32
  if (wave < 4) {
#pragma unroll
    for (int kc = 0; kc < CK / 32; kc++)
#pragma unroll
      for (int e = 0; e < 16; e++) {
        const int k = kc * 32 + 8 * (e >> 2) + 4 * half + (e & 3);
        sPart[(wave * 32 + (lane & 31)) * CKP + k] = acc[kc][e];
      }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < 32 * c; idx += FT) {
    const int ii = idx / c, k = idx % c, i = t * 32 + ii;
    if (i >= n) continue;
    float rsum = 0.f;
#pragma unroll
    for (int part = 0; part < 16; part++) rsum += sRowPart[part * 32 + ii];
    const float ep = sPart[(0 * 32 + ii) * CKP + k] + sPart[(1 * 32 + ii) * CKP + k] +
                     sPart[(2 * 32 + ii) * CKP + k] + sPart[(3 * 32 + ii) * CKP + k];
    dp[((size_t)b * n + i) * c + k] = 2.f * (rsum * (sP[i * CKP + k] - sP[k]) - ep);
  }
}

// Whether the coordinates take the 16-byte load path: p 16-byte aligned and
// c a multiple of 4 (then every window's rows start 16-byte aligned too).
inline int coords_vec(const float* p, int c) {
  return ((uintptr_t)p % 16 == 0 && c % 4 == 0) ? 1 : 0;
}

template <int NT>
hipError_t field_prep_launch(const float* p, unsigned char* tab, int batch, int n, int c, int cp,
                             hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  hipError_t e = lds_limit_once(done, (const void*)field_prep_kernel<NT>, prep_lds_bytes(NT, 64));
  if (e != hipSuccess) return e;
  field_prep_kernel<NT><<<batch, FT, prep_lds_bytes(NT, cp), st>>>(p, tab, n, c, cp,
                                                                   coords_vec(p, c));
  return hipGetLastError();
}

template <int NT, int SW, bool PARTNERS>
hipError_t field_fwd_launch(const float* p, unsigned char* tab, const bf16* x, bf16* y,
                            float* row_mean, float* lse, float* partners, int batch, int n, int c,
                            int cp, int width, float inv_tau, int scaled, hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  hipError_t e = lds_limit_once(done, (const void*)field_fwd_kernel<NT, SW, PARTNERS>,
                                fwd_lds_bytes(NT, SW, 64));
  if (e != hipSuccess) return e;
  const int slabs = width / SW;
  field_fwd_kernel<NT, SW, PARTNERS><<<batch * slabs, FT, fwd_lds_bytes(NT, SW, cp), st>>>(
      p, tab, x, y, row_mean, lse, partners, n, c, cp, width, slabs, inv_tau, scaled,
      coords_vec(p, c));
  return hipGetLastError();
}

template <int NT>
hipError_t field_fwd_pick(const float* p, const bf16* x, bf16* y, float* row_mean, float* lse,
                          float* partners, unsigned char* tab, int batch, int n, int c, int cp,
                          int width, float inv_tau, int scaled, hipStream_t st) {
  const bool wide = width % 128 == 0;
  if (partners)
    return wide ? field_fwd_launch<NT, 128, true>(p, tab, x, y, row_mean, lse, partners, batch,
                                                  n, c, cp, width, inv_tau, scaled, st)
                : field_fwd_launch<NT, 64, true>(p, tab, x, y, row_mean, lse, partners, batch, n,
                                                 c, cp, width, inv_tau, scaled, st);
  return wide ? field_fwd_launch<NT, 128, false>(p, tab, x, y, row_mean, lse, partners, batch, n,
                                                 c, cp, width, inv_tau, scaled, st)
              : field_fwd_launch<NT, 64, false>(p, tab, x, y, row_mean, lse, partners, batch, n,
                                                c, cp, width, inv_tau, scaled, st);
}

template <int NT, int SW>
hipError_t field_dx_launch(const bf16* ct, const bf16* dy, bf16* dx, int batch, int n, int width,
                           hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  hipError_t e = lds_limit_once(done, (const void*)field_bwd_dx_kernel<NT, SW>,
                                dx_lds_bytes(NT, SW));
  if (e != hipSuccess) return e;
  const int slabs = width / SW;
  field_bwd_dx_kernel<NT, SW><<<batch * slabs, FT, dx_lds_bytes(NT, SW), st>>>(ct, dy, dx, n,
                                                                               width, slabs);
  return hipGetLastError();
}

template <int NT, int NS>
hipError_t field_rows_launch(const unsigned char* tab, const bf16* x, const float* row_mean,
                             const float* lse, const bf16* dy, float* ddt, bf16* ct, int batch, int n,
                             int cp, int width, float inv_tau, int scaled, hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  hipError_t e = lds_limit_once(done, (const void*)field_bwd_rows_kernel<NT, NS>,
                                rows_lds_bytes(NT, NS, 64));
  if (e != hipSuccess) return e;
  field_bwd_rows_kernel<NT, NS><<<batch * NT, FT, rows_lds_bytes(NT, NS, cp), st>>>(
      tab, x, dy, row_mean, lse, ddt, ct, n, cp, width, inv_tau, scaled);
  return hipGetLastError();
}

template <int NT, int CK>
hipError_t field_coord_launch(const float* p, const float* ddt, float* dp, int batch, int n,
                              int c, hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  hipError_t e = lds_limit_once(done, (const void*)field_bwd_coord_kernel<NT, CK>,
                                coord_lds_bytes(NT, CK));
  if (e != hipSuccess) return e;
  field_bwd_coord_kernel<NT, CK><<<batch * NT, FT, coord_lds_bytes(NT, CK), st>>>(
      p, ddt, dp, n, c, coords_vec(p, c));
  return hipGetLastError();
}

template <int NT>
hipError_t field_bwd_launch(const float* p, const bf16* x, const float* row_mean,
                            const float* lse, const bf16* dy, float* dp, bf16* dx,
                            unsigned char* ws, int reuse_table, int batch, int n, int c, int cp,
                            int width, float inv_tau, int scaled, hipStream_t st) {
  unsigned char* tab = ws;
  float* ddt = (float*)(ws + (size_t)batch * tab_stride(NT, cp));
  bf16* ct = (bf16*)(ddt + (size_t)batch * NT * 32 * NT * 32);
  hipError_t e = hipSuccess;
  if (!reuse_table) {
    e = field_prep_launch<NT>(p, tab, batch, n, c, cp, st);
    if (e != hipSuccess) return e;
  }
  e = field_rows_launch<NT, ROWS_NS>(tab, x, row_mean, lse, dy, ddt, ct, batch, n, cp, width,
                                     inv_tau, scaled, st);
  if (e != hipSuccess) return e;
  e = width % 128 == 0 ? field_dx_launch<NT, 128>(ct, dy, dx, batch, n, width, st)
                       : field_dx_launch<NT, 64>(ct, dy, dx, batch, n, width, st);
  if (e != hipSuccess) return e;
  return c <= 32 ? field_coord_launch<NT, 32>(p, ddt, dp, batch, n, c, st)
                 : field_coord_launch<NT, 64>(p, ddt, dp, batch, n, c, st);
}

template <int NT>
size_t field_ws_bytes(int batch, int cp) {
  return (size_t)batch * (tab_stride(NT, cp) + (size_t)NT * 32 * NT * 32 * 6);
}

}  // namespace

#define HCMIX_FIELD_CASES(F, ...)            \
  switch ((n + 31) / 32) {                   \
    case 1: return F<1>(__VA_ARGS__);        \
    case 2: return F<2>(__VA_ARGS__);        \
    case 3: return F<3>(__VA_ARGS__);        \
    case 4: return F<4>(__VA_ARGS__);        \
    case 5: return F<5>(__VA_ARGS__);        \
    case 6: return F<6>(__VA_ARGS__);        \
    case 7: return F<7>(__VA_ARGS__);        \
    case 8: return F<8>(__VA_ARGS__);        \
    default: return hipErrorInvalidValue;    \
  }

size_t field_workspace_bytes(int batch, int n, int c) {
  const int cp = (c + 15) / 16 * 16;
  switch ((n + 31) / 32) {
    case 1: return field_ws_bytes<1>(batch, cp);
    case 2: return field_ws_bytes<2>(batch, cp);
    case 3: return field_ws_bytes<3>(batch, cp);
    case 4: return field_ws_bytes<4>(batch, cp);
    case 5: return field_ws_bytes<5>(batch, cp);
    case 6: return field_ws_bytes<6>(batch, cp);
    case 7: return field_ws_bytes<7>(batch, cp);
    case 8: return field_ws_bytes<8>(batch, cp);
    default: return 0;
  }
}

hipError_t launch_field_fwd(const float* p, const bf16* x, bf16* y, float* row_mean, float* lse,
                            float* partners, void* workspace, int batch, int n, int c, int width,
                            float inv_tau, int scaled, hipStream_t st) {
  const int cp = (c + 15) / 16 * 16;
  HCMIX_FIELD_CASES(field_fwd_pick, p, x, y, row_mean, lse, partners, (unsigned char*)workspace,
                    batch, n, c, cp, width, inv_tau, scaled, st)
}

hipError_t launch_field_bwd(const float* p, const bf16* x, const float* row_mean,
                            const float* lse, const bf16* dy, float* dp, bf16* dx, void* workspace,
                            int reuse_table, int batch, int n, int c, int width, float inv_tau,
                            int scaled, hipStream_t st) {
  const int cp = (c + 15) / 16 * 16;
  HCMIX_FIELD_CASES(field_bwd_launch, p, x, row_mean, lse, dy, dp, dx, (unsigned char*)workspace,
                    reuse_table, batch, n, c, cp, width, inv_tau, scaled, st)
}
#undef HCMIX_FIELD_CASES

}  // namespace hcmix
