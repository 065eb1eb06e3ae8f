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
// Kernels (a 32-query or 32-key tile of one window per wave, its scores in
// registers as in the attention core):
//   field_couple_kernel     per query tile: m_i, ln Z_i, partners, and the
//                           couplings C (written, bf16, in the readout's
//                           operand order); the window's table for the
//                           backward;
//   field_readout_kernel    y slab = C x (queries in lanes, C as written);
//   field_prep_kernel       the window's table, when the backward builds it;
//   field_bwd_rows_kernel   per query tile: the couplings C (written, bf16,
//                           transposed, for the dx kernel), dP[i][j] = dy_i .
//                           x_j over the full width, Delta_i = sum_j C dP (=
//                           dy_i . y_i), da = C (dP - Delta), and the gradient
//                           of the squared distances dD (written, fp32,
//                           [key][query]);
//   field_bwd_tail_kernel   one launch, two block roles: dx slab = C^T dy
//                           (keys in lanes, C as written), and
//                           dp_i = 2 sum_j E[i][j] (p_i - p_j), E = dD + dD^T,
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
// division per element.  vec: pw is 16-byte aligned and c a multiple of 4, so
// 16-byte loads never straddle a row (a wave-wide memory instruction costs
// about the same whatever its width, so wide loads move four times the bytes
// per instruction).
template <int THREADS>
__device__ __forceinline__ void stage_coords(const float* __restrict__ pw, int rows, int c,
                                             unsigned char* dst, int stride, bool vec) {
  const int total = rows * c;
  if (vec) {
    constexpr int PER = 256 * 64 / 4 / THREADS;     // float4 per thread at 256 rows x 64
    const int total4 = total >> 2;
    f32x4 v[PER];
#pragma unroll
    for (int u = 0; u < PER; u++)
      v[u] = ((const f32x4*)pw)[min((int)threadIdx.x + THREADS * u, total4 - 1)];
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

constexpr int cmax(int a, int b) { return a > b ? a : b; }
// bytes of a window's table rows (NT * 32 rows of 2 cp + 8 bf16)
constexpr int table_bytes(int NT, int cp) { return NT * 32 * (2 * cp + 8) * 2; }

// The coordinate table rows [0, rows) (rows <= 256) and their squared norms
// N_r (of hi + lo, fp32), from the window's coordinates pw [n][c].  Work is
// dealt in pieces of 4 columns, consecutive threads on consecutive pieces of
// a row (so a wave's 16-byte loads, with vec, cover contiguous memory; every
// load unconditional, indices clamped into the window): a piece is centred on
// the window's first row, split into hi + lo, written to its row, and the sum
// of the squares of hi + lo over its 4 columns goes to sNp[piece][row]; after
// a barrier each row adds its pieces in column order.  Rows at or past n are
// zero, N_r = 0.  sNp: (cp / 4) x NT * 32 floats.  Two barriers; ends with one.
template <int NT>
__device__ __forceinline__ void build_table(const float* __restrict__ pw, int n, int c, int cp,
                                            int rows, bf16* sT, float* sN, float* sNp, bool vec) {
  constexpr int NP = NT * 32, MAXI = (NP * 16 + FT - 1) / FT;
  const int cp4 = cp >> 2, pieces = rows * cp4, rs = ct_stride(cp);
  const float inv4 = 1.f / (float)cp4;             // (idx + 0.5) * inv4 never rounds across an integer
  f32x4 raw[MAXI], p0[MAXI];
#pragma unroll
  for (int u = 0; u < MAXI; u++) {
    const int idx = min((int)threadIdx.x + FT * u, pieces - 1);
    const int r = (int)(((float)idx + 0.5f) * inv4), j = idx - r * cp4;
    const float* prow = pw + (size_t)min(r, n - 1) * c;
    if (vec) {
      const int kk = min(4 * j, c - 4);
      raw[u] = *(const f32x4*)(prow + kk);
      p0[u] = *(const f32x4*)(pw + kk);
    } else {
#pragma unroll
      for (int e = 0; e < 4; e++) {
        const int kk = min(4 * j + e, c - 1);
        raw[u][e] = prow[kk];
        p0[u][e] = pw[kk];
      }
    }
  }
#pragma unroll
  for (int u = 0; u < MAXI; u++) {
    const int idx = threadIdx.x + FT * u;
    if (idx < pieces) {
      const int r = (int)(((float)idx + 0.5f) * inv4), j = idx - r * cp4;
      float nn = 0.f;
      bf16x4 hi, lo;
#pragma unroll
      for (int e = 0; e < 4; e++) {
        const float v = (r < n && 4 * j + e < c) ? raw[u][e] - p0[u][e] : 0.f;
        hi[e] = to_bf16(v);
        const float hv = (float)hi[e];
        lo[e] = to_bf16(v - hv);
        const float t = hv + (float)lo[e];
        nn = fmaf(t, t, nn);
      }
      *(bf16x4*)(sT + r * rs + 4 * j) = hi;
      *(bf16x4*)(sT + r * rs + cp + 4 * j) = lo;
      if (j == 0) *(u32x4*)(sT + r * rs + 2 * cp) = u32x4{0u, 0u, 0u, 0u};
      sNp[j * NP + r] = nn;
    }
  }
  __syncthreads();
  if ((int)threadIdx.x < rows) {
    float nr = 0.f;
    for (int j = 0; j < cp4; j++) nr += sNp[j * NP + threadIdx.x];
    sN[threadIdx.x] = nr;
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
  bf16* sT = (bf16*)smem;
  float* sN = (float*)(smem + table_bytes(NT, cp));
  float* sNp = sN + NP;                       // [cp / 4][NP]
  const int b = blockIdx.x;
  build_table<NT>(p + (size_t)b * n * c, n, c, cp, NP, sT, sN, sNp, vec);
  store_table<NT>(sT, sN, tab + (size_t)b * tab_stride(NT, cp), cp, 0, 1);
}

// Rows [0, rows) of window b's stored table and their norms, into LDS.  Every
// load is issued before the first LDS write.  Ends with a barrier.
template <int NT>
__device__ __forceinline__ void load_table(const unsigned char* __restrict__ tw, int cp, int rows,
                                           bf16* sT, float* sN) {
  constexpr int MAXP = (NT * 32 * 136 * 2 / 16 + FT - 1) / FT;   // 16-byte pieces per thread
  const int pieces = rows * (2 * cp + 8) * 2 / 16;
  u32x4 v[MAXP];
#pragma unroll
  for (int u = 0; u < MAXP; u++)
    v[u] = ((const u32x4*)tw)[min((int)threadIdx.x + FT * u, pieces - 1)];
  const float* nrm = (const float*)(tw + tab_nrm(NT, cp));
  const float nv = nrm[min((int)threadIdx.x, rows - 1)];
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

// s_waitcnt vmcnt(n) for a wave-uniform runtime n (n > 10 waits for all).
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

// Block bid of total -> (window b, query tile qt) for the kernels with one
// block per query tile, two of them per CU.  Blocks go to the 8 XCDs round
// robin (xcd_tile keeps a window's tiles on one XCD) and, within an XCD, to
// its CUs in order, so the first and the second half of an XCD's blocks meet
// on the same CUs.  The first half takes its windows' tiles heaviest first,
// the second half lightest first: each CU then pairs tile t with tile NT - 1 -
// t (NT + 1 key tiles of causal work) instead of holding two copies of one.
// When an XCD's half is not a whole number of windows, all go heaviest first.
__device__ __forceinline__ void query_tile_of(int bid, int total, int NT, int* b, int* qt) {
  const int lin = xcd_tile(bid, total);
  const int t = lin % NT, group = total / 8;
  *b = lin / NT;
  const bool paired = total % (16 * NT) == 0 && lin % group >= group / 2;
  *qt = paired ? t : NT - 1 - t;
}

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

// Gram tile G^T[key][query] for keys kt*32 .. kt*32 + 31 (A operand, table
// rows) and the lane's query q (B operand, its own row's fragments):
// hi.hi, then key-lo . query-hi, then key-hi . query-lo.  The forward's
// couplings and the backward's rows kernel both take D from here, so they
// agree bitwise.
__device__ __forceinline__ f32x16 gram_keys(const bf16* sT, int rs, int cp, int kt, int q,
                                            int lane) {
  RowFrags f;
  row_frags(sT, rs, cp, q, lane >> 5, f);
  f32x16 acc = {};
#pragma unroll
  for (int ks = 0; ks < 4; ks++) {
    if (16 * ks < cp) {
      const bf16x8 ahi = ct_frag(sT, rs, kt * 32, 16 * ks, lane);
      const bf16x8 alo = ct_frag(sT, rs, kt * 32, cp + 16 * ks, lane);
      acc = mfma32(ahi, f.hi[ks], acc);
      acc = mfma32(alo, f.hi[ks], acc);
      acc = mfma32(ahi, f.lo[ks], acc);
    }
  }
  return acc;
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
constexpr int prep_lds_bytes(int NT, int cp) { return table_bytes(NT, cp) + (1 + cp / 4) * NT * 32 * 4; }
constexpr int dx_lds_bytes(int NT, int SW) { return NT * 32 * SW * 2; }

// Transposed coupling tiles as the rows kernel writes them and the dx kernel
// reads them: per window NT x NT tiles of 32 x 32 bf16 (tile (kt, qt) at kt *
// NT + qt; only qt >= kt written), row = key, and within a row the 32
// queries in the order of a key lane's score registers: query 8 g + 4 h + r
// (g, r < 4, h < 2) at 16 h + 4 g + r.  A lane of half h then finds its 16
// couplings of a tile in 32 contiguous bytes.
__device__ __forceinline__ int ct_pos(int lq) { return 16 * ((lq >> 2) & 1) + 4 * (lq >> 3) + (lq & 3); }
// rows kernel: NS stages of [x rows (NT * 32)][SC] + [dy rows (32)][SC] bf16,
// the coordinate table in the same space before the stages are used, then
// the norms and the per-wave row sums.  NS * SC = 128 keeps a block within 77
// KB, so two blocks share a CU.  Two stages of 64 columns (one step in flight)
// ran 17.7 us at 64 windows x 256 x 512; four of 32 columns (three in flight,
// twice the steps and barriers) 20.0 us.
constexpr int rows_stage_elems(int NT, int SC) { return (NT * 32 + 32) * SC; }
constexpr int rows_lds_bytes(int NT, int NS, int SC, int cp) {
  return cmax(NS * rows_stage_elems(NT, SC) * 2, table_bytes(NT, cp)) + NT * 32 * 4 +
         2 * 8 * 32 * 4;
}
constexpr int ROWS_NS = 2, ROWS_SC = 64;

// 32 x 16 operand fragment of a [rows][SC] stage tile (lane l: row r0 + l % 32,
// columns c0 + 8 (l / 32) .. + 8): SC = 64 in the attention tiles' layout, SC
// = 32 in the 32-wide k-contiguous swizzle.
template <int SC>
__device__ __forceinline__ bf16x8 stage_frag(const bf16* t, int r0, int c0, int lane) {
  if constexpr (SC == 64) {
    return att_frag(t, r0, c0, lane);
  } else {
    return *(const bf16x8*)(t + swz<32>(r0 + (lane & 31), (c0 >> 3) + (lane >> 5)));
  }
}
// coordinate kernel: E tile [32][NP + 1] fp32, coordinates [NP][ck + 1] fp32,
// row-sum parts [16][32], and the per-wave partial products [4][32][ck + 1]
// (in the E tile's space where they fit, else after the rest)
constexpr bool coord_part_in_e(int NT, int ck) { return 4 * 32 * (ck + 1) <= 32 * (NT * 32 + 1); }
constexpr int coord_lds_bytes(int NT, int ck) {
  return 32 * (NT * 32 + 1) * 4 + NT * 32 * (ck + 1) * 4 + 16 * 32 * 4 +
         (coord_part_in_e(NT, ck) ? 0 : 4 * 32 * (ck + 1) * 4);
}

// ---------------------------------------------------------------------------
// Forward, couplings.  Block = (window b, query tile qt) (query_tile_of), 8
// waves; grid = batch * NT.
//   1. The table rows [0, 32 (qt + 1)) are built in LDS; the block of the
//      last tile, which has every row, leaves the table in the workspace for
//      the backward.
//   2. Wave w <= qt takes key tile w: D for the tile's 32 queries (lanes) and
//      32 keys (registers) from the Gram tile; the row sums of D meet in LDS
//      (in wave order), giving each query's mean and logit scale; then the
//      weights exp2(D k2) (<= 1; keys after the query 0), whose sums (and the
//      entropy term) meet in LDS the same way.
//   3. The couplings C = weight / Z, as the bf16 MFMA operand fragments of the
//      readout (lane = query, the 8 keys of a k step in score-register
//      order), go to the workspace: tile (qt, kt) at qt * NT + kt, [2][64
//      lanes][8].  Each coupling is computed once.
// ---------------------------------------------------------------------------
constexpr int couple_lds_bytes(int NT, int cp) {
  return table_bytes(NT, cp) + NT * 32 * 4 + cmax(cp / 4 * NT * 32 * 4, 3 * 8 * 32 * 4);
}

template <int NT, bool PARTNERS>
__global__ __launch_bounds__(FT) void field_couple_kernel(
    const float* __restrict__ p, unsigned char* __restrict__ tab, bf16x8* __restrict__ cq,
    float* __restrict__ row_mean, float* __restrict__ lse, float* __restrict__ partners, int n,
    int c, int cp, float inv_tau, int scaled, int vec) {
  constexpr int NP = NT * 32;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  bf16* sT = (bf16*)smem;
  float* sN = (float*)(smem + table_bytes(NT, cp));
  float* sNp = sN + NP;                               // [cp / 4][NP] while the table is built,
  float* sRed = sNp;                                  // then [3][8 waves][32]: D, Z, entropy sums
  int b, qt;
  query_tile_of(blockIdx.x, gridDim.x, NT, &b, &qt);
  const int lane = threadIdx.x & 63, half = lane >> 5, lq = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int rs = ct_stride(cp);
  const int q = qt * 32 + lq;
  const bool qvalid = q < n;
  build_table<NT>(p + (size_t)b * n * c, n, c, cp, (qt + 1) * 32, sT, sN, sNp, vec);
  if (qt == NT - 1) store_table<NT>(sT, sN, tab + (size_t)b * tab_stride(NT, cp), cp, 0, 1);
  const bool own = wave <= qt;                        // this wave's key tile kt = wave
  const bool diag = wave == qt;
  const float nq = sN[q];
  f32x16 d = {};
  if (own) {
    const f32x16 acc = gram_keys(sT, rs, cp, wave, q, lane);
    float ds = 0.f;
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const f32x4 n4 = *(const f32x4*)(sN + wave * 32 + 8 * g + 4 * half);
#pragma unroll
      for (int r = 0; r < 4; r++) {
        const int e = 4 * g + r;
        float dv = fmaf(acc[e], -2.f, n4[r] + nq);
        if (diag && 8 * g + 4 * half + r >= lq) dv = 0.f;   // q itself, keys after q
        d[e] = dv;
        ds += dv;
      }
    }
    ds += __shfl_xor(ds, 32);
    if (half == 0) sRed[wave * 32 + lq] = ds;
  }
  __syncthreads();
  float dsum = 0.f;
  for (int w = 0; w <= qt; w++) dsum += sRed[w * 32 + lq];
  const float m = qvalid ? dsum / (float)(q + 1) : 0.f;
  const float k2 = qvalid ? -logit_scale(m, inv_tau, scaled) * LOG2E : 0.f;
  if (own) {
    float z = 0.f, za = 0.f;
#pragma unroll
    for (int e = 0; e < 16; e++) {
      const float a = d[e] * k2;
      float pe = __builtin_amdgcn_exp2f(a);
      if (diag && att_masked(e, lane)) pe = 0.f;
      d[e] = pe;
      z += pe;
      if constexpr (PARTNERS) za += pe * a;
    }
    z += __shfl_xor(z, 32);
    if constexpr (PARTNERS) za += __shfl_xor(za, 32);
    if (half == 0) {
      sRed[256 + wave * 32 + lq] = z;
      if constexpr (PARTNERS) sRed[512 + wave * 32 + lq] = za;
    }
  }
  __syncthreads();
  float z = 0.f, za = 0.f;
  for (int w = 0; w <= qt; w++) {
    z += sRed[256 + w * 32 + lq];
    if constexpr (PARTNERS) za += sRed[512 + w * 32 + lq];
  }
  const float inv = 1.f / z;
  if (wave == 0 && half == 0 && qvalid) {
    const float l2z = __builtin_amdgcn_logf(z);       // log2 Z
    const size_t at = (size_t)b * n + q;
    row_mean[at] = m;
    lse[at] = l2z * LN2;
    if constexpr (PARTNERS) partners[at] = __builtin_amdgcn_exp2f(l2z - za * inv);
  }
  if (own) {
#pragma unroll
    for (int e = 0; e < 16; e++) d[e] *= inv;
    bf16x8* dst = cq + ((size_t)(b * NT + qt) * NT + wave) * 128 + lane;
    dst[0] = att_pack(d, 0);
    dst[64] = att_pack(d, 1);
  }
}

// ---------------------------------------------------------------------------
// Forward, readout.  Block = (window b, slab s of SW columns), 8 waves, wave w
// on query tile wave_tile(w) (lane = query); y^T[col][q] = sum over key tiles
// kt <= qt of x^T[col][k] C[q][k], with C as the couplings kernel wrote it
// (PF tiles in flight) and x^T read transposed from the LDS slab.
// ---------------------------------------------------------------------------
template <int NT, int SW>
__global__ __launch_bounds__(FT) void field_readout_kernel(const bf16x8* __restrict__ cq,
                                                          const bf16* __restrict__ x,
                                                          bf16* __restrict__ y, int n, int width,
                                                          int slabs) {
  constexpr int NP = NT * 32, DT = SW / 32, PF = NT < 3 ? NT : 3;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  bf16* sX = (bf16*)smem;
  const int lin = xcd_tile(blockIdx.x, gridDim.x);
  const int b = lin / slabs, s = lin % slabs;
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int qt = wave_tile(wave);
  Slab<NT, SW> slab;
  slab.issue(x + (size_t)b * n * width + (size_t)s * SW, width, n);
  // tile (qt, u) for u <= qt; past that (and for waves without a query tile)
  // the loads are clamped to a tile of the window, in bounds
  const bf16x8* cw = cq + ((size_t)b * NT + min(qt, NT - 1)) * NT * 128 + lane;
  bf16x8 cf[PF][2];
  auto fetch = [&](int u, bf16x8* dst) {
    const bf16x8* src = cw + (size_t)min(u, NT - 1) * 128;
    dst[0] = src[0];
    dst[1] = src[64];
  };
#pragma unroll
  for (int u = 0; u < PF; u++) fetch(u, cf[u]);
  slab.store(sX, n);
  __syncthreads();
  if (qt >= NT) return;
  f32x16 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; dt++) o[dt] = f32x16{};
#pragma unroll
  for (int u = 0; u < NT; u++) {
    if (u <= qt) {
      bf16x8 cur[2] = {cf[u % PF][0], cf[u % PF][1]};
      if (u + PF < NT) fetch(u + PF, cf[u % PF]);
#pragma unroll
      for (int mm = 0; mm < 2; mm++)
#pragma unroll
        for (int dt = 0; dt < DT; dt++)
          o[dt] = mfma32(att_trfrag(sX + (dt / 2) * NP * 64, u * 32 + 16 * mm, 32 * (dt % 2), lane),
                         cur[mm], o[dt]);
    }
  }
  const int q = qt * 32 + (lane & 31);
  if (q >= n) return;
  // register e of o[dt]: column 32 dt + 8 (e / 4) + 4 half + e % 4
  bf16* yrow = y + ((size_t)b * n + q) * width + (size_t)s * SW;
#pragma unroll
  for (int dt = 0; dt < DT; dt++)
#pragma unroll
    for (int g = 0; g < 4; g++) {
      const bf16x4 v = {to_bf16(o[dt][4 * g]), to_bf16(o[dt][4 * g + 1]), to_bf16(o[dt][4 * g + 2]),
                        to_bf16(o[dt][4 * g + 3])};
      *(bf16x4*)(yrow + 32 * dt + 8 * g + 4 * half) = v;
    }
}

// ---------------------------------------------------------------------------
// Backward, rows.  Block = (window b, query tile qt) (query_tile_of); 8 waves,
// wave w owning key tile w (w <= qt).  Two blocks share a CU, a heavy tile
// beside a light one, so one block's set-up and reductions overlap the
// other's streaming.
// The couplings, their squared distances and the row sums come first, from
// the coordinate table (loaded into the stage space).  Then dP^T[key][q] =
// x_key . dy_q sums over the width in SC-column steps: each step's x rows
// [0, 32 (qt + 1)) and the tile's 32 dy rows go global -> LDS by DMA
// (coalesced, 1 KB of whole rows per instruction, swizzled as stage_frag
// reads them), NS - 1 steps in flight, the instructions of a step dealt over
// the 8 waves.  The per-row sums Delta and sum(da D) across the waves go through
// LDS.
// ---------------------------------------------------------------------------
template <int NT, int NS, int SC>
__global__ __launch_bounds__(FT) void field_bwd_rows_kernel(
    const unsigned char* __restrict__ tab, const bf16* __restrict__ x, const bf16* __restrict__ dy,
    const float* __restrict__ row_mean, const float* __restrict__ lse, float* __restrict__ ddt,
    bf16* __restrict__ ct, int n, int cp, int width, float inv_tau, int scaled) {
  constexpr int NP = NT * 32, STAGE = rows_stage_elems(NT, SC);
  constexpr int RPI = 512 / SC, LPR = SC / 8;         // rows per DMA instruction, lanes per row
  constexpr int VMAX = ((NP + 32) / RPI + 7) / 8;     // DMA instructions per wave and step
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  bf16* sStage = (bf16*)smem;
  bf16* sT = sStage;                                  // the table, until the first DMA
  float* sN = (float*)(smem + cmax(NS * STAGE * 2, table_bytes(NT, cp)));
  float* sRed = sN + NP;                              // [2][8 waves][32]
  int b, qt;
  query_tile_of(blockIdx.x, gridDim.x, NT, &b, &qt);
  const int lane = threadIdx.x & 63, half = lane >> 5;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int rs = ct_stride(cp);
  const int q = qt * 32 + (lane & 31);
  const bool qvalid = q < n;
  const bool own = wave <= qt;                        // this wave's key tile kt = wave
  const int steps = width / SC;
  // DMA plan of one step: instructions u < XI are x rows RPI u .. RPI u +
  // RPI - 1, the next 32 / RPI the tile's dy rows; wave w issues u = w, w + 8,
  // ...  Rows past the window read its last row (finite values that only reach
  // couplings the causal mask removes, or rows whose results are not used).
  const int XI = (qt + 1) * 32 / RPI, TI = XI + 32 / RPI;
  const int cnt = wave < TI ? (TI - 1 - wave) / 8 + 1 : 0;
  const bf16* xw = x + (size_t)b * n * width;
  const bf16* dyw = dy + (size_t)b * n * width;
  auto dma = [&](int st, int slot) {
    bf16* dst = sStage + slot * STAGE;
#pragma unroll
    for (int v = 0; v < VMAX; v++) {
      if (v < cnt) {
        const int u = wave + 8 * v;
        const int lr = RPI * u + lane / LPR;              // row in the stage (x rows, then dy)
        const int tr = u < XI ? lr : qt * 32 + (lr - RPI * XI);   // row in the window
        const int gr = tr < n ? tr : n - 1;
        const int tile_row = u < XI ? lr : lr - RPI * XI;
        const int lp = lane % LPR;
        const int piece = SC == 64 ? lp ^ att_sw(tile_row) : lp ^ ((tile_row >> 2) & 3);
        const bf16* src = (u < XI ? xw : dyw) + (size_t)gr * width + st * SC + 8 * piece;
        bf16* d0 = u < XI ? dst + u * 512 : dst + NP * SC + (u - XI) * 512;
        dma16(src, d0);
      }
    }
  };
  const float m_ld = row_mean[(size_t)b * n + min(q, n - 1)];
  const float l_ld = lse[(size_t)b * n + min(q, n - 1)];
  load_table<NT>(tab + (size_t)b * tab_stride(NT, cp), cp, (qt + 1) * 32, sT, sN);
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
      for (int ks = 0; ks < SC / 16; ks++)
        g = mfma32(stage_frag<SC>(cur, wave * 32, 16 * ks, lane),
                   stage_frag<SC>(cur + NP * SC, 0, 16 * ks, lane), g);
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
// Backward, dx.  Block bid of nblk = (window b, slab s of SW columns), 8 waves, wave w on
// key tile wave_tile(w), a lane one key j; the couplings come as the rows
// kernel wrote them (bf16, the lane's 16 queries of a tile in one 32-byte
// load, PF tiles in flight), and dx^T[col][j] += dy^T[col][q] C[q][j] as in
// the attention core's dV, dy^T read transposed from the LDS slab.
// ---------------------------------------------------------------------------
template <int NT, int SW>
__device__ __forceinline__ void dx_block(int bid, int nblk, const bf16* __restrict__ ct,
                                         const bf16* __restrict__ dy, bf16* __restrict__ dx, int n,
                                         int width, int slabs) {
  constexpr int NP = NT * 32, DT = SW / 32, PF = NT < 3 ? NT : 3;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  bf16* sDY = (bf16*)smem;
  const int lin = xcd_tile(bid, nblk);
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
// Backward, coordinates.  Block bid of nblk = (window b, row tile t), 8 waves: E[i][j] for
// the tile's 32 rows i and every j (dD[i][j] = ddt[j][i] for j < i, dD[j][i] =
// ddt[i][j] for j > i; 0 at j = i and outside the window) into LDS; then
//   dp_i = 2 (sum_j E[i][j]) p'_i - 2 sum_j E[i][j] p'_j,  p' = p - p_0,
// the second sum on the fp32 matrix cores (32 x 32 x 2: A = p'^T, B = E^T),
// waves 0-3 taking a quarter of the j range each; partial products meet in
// LDS.
// ---------------------------------------------------------------------------
template <int NT, int CK>
__device__ __forceinline__ void coord_block(int bid, int nblk, const float* __restrict__ p,
                                            const float* __restrict__ ddt, float* __restrict__ dp,
                                            int n, int c, int vec) {
  constexpr int NP = NT * 32, ES = NP + 1, CKP = CK + 1;
  extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
  float* sE = (float*)smem;                          // [32][ES]
  float* sP = sE + 32 * ES;                          // [NP][CKP]
  float* sRowPart = sP + NP * CKP;                   // [16][32]
  float* sPart = coord_part_in_e(NT, CK) ? sE : sRowPart + 16 * 32;   // [4][32][CKP]
  const int lin = xcd_tile(bid, nblk);
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

// ---------------------------------------------------------------------------
// Backward, dx and coordinates in one launch: blocks [0, dx_blocks) are dx
// blocks, the rest coordinate blocks.  Both read only what the rows kernel
// wrote, so the coordinate blocks' latency-bound work overlaps the dx
// blocks' memory traffic, and one kernel boundary goes.
// ---------------------------------------------------------------------------
template <int NT, int SW, int CK>
__global__ __launch_bounds__(FT) void field_bwd_tail_kernel(
    const bf16* __restrict__ ct, const bf16* __restrict__ dy, bf16* __restrict__ dx, int width,
    int slabs, const float* __restrict__ p, const float* __restrict__ ddt, float* __restrict__ dp,
    int n, int c, int vec, int dx_blocks) {
  const int coord_blocks = gridDim.x - dx_blocks;
  if ((int)blockIdx.x < coord_blocks)
    coord_block<NT, CK>(blockIdx.x, coord_blocks, p, ddt, dp, n, c, vec);
  else
    dx_block<NT, SW>(blockIdx.x - coord_blocks, dx_blocks, ct, dy, dx, n, width, slabs);
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

template <int NT, bool PARTNERS>
hipError_t field_couple_launch(const float* p, unsigned char* tab, bf16x8* cq, float* row_mean,
                               float* lse, float* partners, int batch, int n, int c, int cp,
                               float inv_tau, int scaled, hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  hipError_t e = lds_limit_once(done, (const void*)field_couple_kernel<NT, PARTNERS>,
                                couple_lds_bytes(NT, 64));
  if (e != hipSuccess) return e;
  field_couple_kernel<NT, PARTNERS><<<batch * NT, FT, couple_lds_bytes(NT, cp), st>>>(
      p, tab, cq, row_mean, lse, partners, n, c, cp, inv_tau, scaled, coords_vec(p, c));
  return hipGetLastError();
}

template <int NT, int SW>
hipError_t field_readout_launch(const bf16x8* cq, const bf16* x, bf16* y, int batch, int n,
                                int width, hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  hipError_t e = lds_limit_once(done, (const void*)field_readout_kernel<NT, SW>,
                                dx_lds_bytes(NT, SW));
  if (e != hipSuccess) return e;
  const int slabs = width / SW;
  field_readout_kernel<NT, SW><<<batch * slabs, FT, dx_lds_bytes(NT, SW), st>>>(cq, x, y, n,
                                                                                width, slabs);
  return hipGetLastError();
}

// Workspace: the tables, then the squared-distance gradient (backward), then
// the couplings: the forward's [batch][NT][NT] fragment tiles, later the
// backward's transposed tiles (each call's use ends with the call).
template <int NT>
unsigned char* field_coupling_space(unsigned char* ws, int batch, int cp) {
  return ws + (size_t)batch * tab_stride(NT, cp) + (size_t)batch * NT * 32 * NT * 32 * 4;
}

template <int NT>
hipError_t field_fwd_pick(const float* p, const bf16* x, bf16* y, float* row_mean, float* lse,
                          float* partners, unsigned char* ws, int batch, int n, int c, int cp,
                          int width, float inv_tau, int scaled, hipStream_t st) {
  bf16x8* cq = (bf16x8*)field_coupling_space<NT>(ws, batch, cp);
  hipError_t e = partners ? field_couple_launch<NT, true>(p, ws, cq, row_mean, lse, partners, batch,
                                                          n, c, cp, inv_tau, scaled, st)
                          : field_couple_launch<NT, false>(p, ws, cq, row_mean, lse, partners,
                                                           batch, n, c, cp, inv_tau, scaled, st);
  if (e != hipSuccess) return e;
  return width % 128 == 0 ? field_readout_launch<NT, 128>(cq, x, y, batch, n, width, st)
                          : field_readout_launch<NT, 64>(cq, x, y, batch, n, width, st);
}

template <int NT, int NS, int SC>
hipError_t field_rows_launch(const unsigned char* tab, const bf16* x, const float* row_mean,
                             const float* lse, const bf16* dy, float* ddt, bf16* ct, int batch, int n,
                             int cp, int width, float inv_tau, int scaled, hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  hipError_t e = lds_limit_once(done, (const void*)field_bwd_rows_kernel<NT, NS, SC>,
                                rows_lds_bytes(NT, NS, SC, 64));
  if (e != hipSuccess) return e;
  field_bwd_rows_kernel<NT, NS, SC><<<batch * NT, FT, rows_lds_bytes(NT, NS, SC, cp), st>>>(
      tab, x, dy, row_mean, lse, ddt, ct, n, cp, width, inv_tau, scaled);
  return hipGetLastError();
}

template <int NT, int SW, int CK>
hipError_t field_tail_launch(const bf16* ct, const bf16* dy, bf16* dx, const float* p,
                             const float* ddt, float* dp, int batch, int n, int c, int width,
                             hipStream_t st) {
  static std::atomic<unsigned long long> done{0};
  constexpr int lds = cmax(dx_lds_bytes(NT, SW), coord_lds_bytes(NT, CK));
  hipError_t e = lds_limit_once(done, (const void*)field_bwd_tail_kernel<NT, SW, CK>, lds);
  if (e != hipSuccess) return e;
  const int slabs = width / SW, dxb = batch * slabs;
  field_bwd_tail_kernel<NT, SW, CK><<<dxb + batch * NT, FT, lds, st>>>(
      ct, dy, dx, width, slabs, p, ddt, dp, n, c, coords_vec(p, c), dxb);
  return hipGetLastError();
}

template <int NT, int SW>
hipError_t field_tail_pick(const bf16* ct, const bf16* dy, bf16* dx, const float* p,
                           const float* ddt, float* dp, int batch, int n, int c, int width,
                           hipStream_t st) {
  return c <= 32 ? field_tail_launch<NT, SW, 32>(ct, dy, dx, p, ddt, dp, batch, n, c, width, st)
                 : field_tail_launch<NT, SW, 64>(ct, dy, dx, p, ddt, dp, batch, n, c, width, st);
}

template <int NT>
hipError_t field_bwd_launch(const float* p, const bf16* x, const float* row_mean,
                            const float* lse, const bf16* dy, float* dp, bf16* dx,
                            unsigned char* ws, int reuse_table, int batch, int n, int c, int cp,
                            int width, float inv_tau, int scaled, hipStream_t st) {
  unsigned char* tab = ws;
  float* ddt = (float*)(ws + (size_t)batch * tab_stride(NT, cp));
  bf16* ct = (bf16*)field_coupling_space<NT>(ws, batch, cp);
  hipError_t e = hipSuccess;
  if (!reuse_table) {
    e = field_prep_launch<NT>(p, tab, batch, n, c, cp, st);
    if (e != hipSuccess) return e;
  }
  e = field_rows_launch<NT, ROWS_NS, ROWS_SC>(tab, x, row_mean, lse, dy, ddt, ct, batch, n, cp,
                                              width, inv_tau, scaled, st);
  if (e != hipSuccess) return e;
  return width % 128 == 0 ? field_tail_pick<NT, 128>(ct, dy, dx, p, ddt, dp, batch, n, c, width, st)
                          : field_tail_pick<NT, 64>(ct, dy, dx, p, ddt, dp, batch, n, c, width, st);
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
