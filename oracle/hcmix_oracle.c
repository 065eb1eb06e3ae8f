/*
 * hcmix CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, deliberately obvious implementation of the rotating-hypercube
 * mixing layer, used to check the GPU library and nothing else.  Only the test
 * suite, the smoke check and the benchmark's CPU-baseline leg may load it; the
 * product path never does.  It shares no code, header or constant with the GPU
 * library.
 *
 * Everything is computed in double precision with plain loops: no BLAS, no
 * blocking, no reordering beyond what the definitions below state.  Inputs are
 * doubles (bf16 or fp32 values widen to double exactly), results are doubles.
 *
 * Definitions followed (paper: "Reaching Every Position Without Searching"):
 *  - Section 3.1: n = 2^b positions indexed by b-bit integers; at layer l
 *    position i is linked to i XOR 2^(l mod b).  For causal modelling only the
 *    earlier of the two endpoints is kept, i.e. position i takes the vector of
 *    its partner only when the partner comes before it.
 *  - Section 3.2, Eq. (1): y_i = W_self x_i + W_off x_partner(i); two linear
 *    maps and a shift, nothing else (no bias, residual or activation).
 *  - Section 3.2, Eq. (1) with jump k = 1 is the local ("near") layer of the
 *    schedules of Section 3.3 and Appendix A: y_i = W_self x_i + W_off x_(i-1),
 *    position 0 of a window having no predecessor.  It is causal by
 *    construction and exists in causal mode only.  Layer code ORACLE_NEAR.
 *  - The backward pass is the adjoint of Eq. (1); the paper trains every model
 *    but prints no gradient, so it is written here from the chain rule: for
 *    every link (receiver i <- sender p) the gradient flows back from i to p.
 *
 * Layouts: x, y, dx, dy are [batch][n][width] row-major; w_self, w_off,
 * dw_self, dw_off are [width_out][width_in] row-major, so y = W x means
 * y[o] = sum_c W[o][c] * x[c].
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Layer code of the local layer (jump k = 1); layer codes >= 0 are hypercube
 * layers with dimension code mod b. */
#define ORACLE_NEAR (-1)

/* b = log2 n for n a power of two >= 2, else -1. */
int32_t oracle_log2n(int64_t n) {
    if (n < 2) return -1;
    int32_t b = 0;
    int64_t v = 1;
    while (v < n) { v *= 2; b++; }
    return v == n ? b : -1;
}

/* Hypercube dimension used at layer l: l mod b (Section 3.1). */
int32_t oracle_dim(int32_t layer, int64_t n) {
    int32_t b = oracle_log2n(n);
    if (b < 0 || layer < 0) return -1;
    return layer % b;
}

/* 1 if `layer` is a layer code this oracle knows for windows of n (and the
 * mode allows it): a hypercube layer, or the local layer in causal mode. */
int32_t oracle_valid_layer(int32_t layer, int64_t n, int32_t causal) {
    if (oracle_log2n(n) < 0) return 0;
    if (layer == ORACLE_NEAR) return causal ? 1 : 0;
    return layer >= 0;
}

/* Partner of position i at layer l: i XOR 2^(l mod b) (Section 3.1); for the
 * local layer the previous position i - 1, or -1 at position 0 (no partner). */
int64_t oracle_partner(int64_t i, int32_t layer, int64_t n) {
    if (i < 0 || i >= n || oracle_log2n(n) < 0) return -1;
    if (layer == ORACLE_NEAR) return i - 1;
    int32_t d = oracle_dim(layer, n);
    if (d < 0) return -1;
    return i ^ ((int64_t)1 << d);
}

/* 1 when position i takes its partner's vector at layer l.  Bidirectional:
 * always.  Causal: only the earlier endpoint of a link is kept (Section 3.1),
 * so i receives exactly when its partner precedes it (for the local layer:
 * whenever it has a predecessor).  -1 for an invalid layer, position or mode. */
int32_t oracle_receives(int64_t i, int32_t layer, int64_t n, int32_t causal) {
    if (i < 0 || i >= n || !oracle_valid_layer(layer, n, causal)) return -1;
    int64_t p = oracle_partner(i, layer, n);
    if (layer == ORACLE_NEAR) return p >= 0 ? 1 : 0;
    if (!causal) return 1;
    return p < i ? 1 : 0;
}

int32_t oracle_num_threads(void) {
#ifdef _OPENMP
    return (int32_t)omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads the loops below use from now on (timing only; results do not
 * depend on it, every element being summed in a fixed order). */
void oracle_set_num_threads(int32_t k) {
#ifdef _OPENMP
    if (k >= 1) omp_set_num_threads(k);
#else
    (void)k;
#endif
}

/* Forward of one layer, Eq. (1):
 *   y[bt][i][o] = sum_c w_self[o][c] x[bt][i][c]
 *               + receives(i) * sum_c w_off[o][c] x[bt][partner(i)][c]. */
int32_t oracle_forward(int64_t batch, int64_t n, int64_t width, int32_t layer,
                       int32_t causal, const double* x, const double* w_self,
                       const double* w_off, double* y) {
    if (!oracle_valid_layer(layer, n, causal) || batch < 1 || width < 1) return -1;
    int64_t rows = batch * n;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; r++) {
        int64_t bt = r / n, i = r % n;
        int32_t take = oracle_receives(i, layer, n, causal);
        const double* xi = x + (bt * n + i) * width;
        double* yi = y + (bt * n + i) * width;
        for (int64_t o = 0; o < width; o++) {
            double acc = 0.0;
            for (int64_t c = 0; c < width; c++) acc += w_self[o * width + c] * xi[c];
            if (take) {
                const double* xp = x + (bt * n + oracle_partner(i, layer, n)) * width;
                for (int64_t c = 0; c < width; c++) acc += w_off[o * width + c] * xp[c];
            }
            yi[o] = acc;
        }
    }
    return 0;
}

/* Backward of one layer: the adjoint of oracle_forward.  Given dy = dL/dy,
 *   dx[bt][j][c]   = sum_o w_self[o][c] dy[bt][j][o]
 *                  + sum over links (i <- j) of sum_o w_off[o][c] dy[bt][i][o]
 *   dw_self[o][c]  = sum_{bt,i} dy[bt][i][o] x[bt][i][c]
 *   dw_off[o][c]   = sum_{bt,i} receives(i) dy[bt][i][o] x[bt][partner(i)][c]
 * dx is written in scatter form (each receiver pushes its gradient back to its
 * sender), the literal transpose of the forward's gather. */
int32_t oracle_backward(int64_t batch, int64_t n, int64_t width, int32_t layer,
                        int32_t causal, const double* x, const double* w_self,
                        const double* w_off, const double* dy, double* dx,
                        double* dw_self, double* dw_off) {
    if (!oracle_valid_layer(layer, n, causal) || batch < 1 || width < 1) return -1;
    int64_t rows = batch * n;

    /* dx: windows are independent, and so is every column c of dx; a thread
     * owns one window and one range of columns (the work items are spread over
     * both so that a single long window still uses every core).  Each element
     * is summed in the same order whatever the split: receivers i ascending,
     * then o ascending. */
    const int64_t cchunk = 64;
    const int64_t nchunks = (width + cchunk - 1) / cchunk;
#pragma omp parallel for schedule(static)
    for (int64_t item = 0; item < batch * nchunks; item++) {
        const int64_t bt = item / nchunks;
        const int64_t c0 = (item % nchunks) * cchunk;
        const int64_t c1 = c0 + cchunk < width ? c0 + cchunk : width;
        for (int64_t i = 0; i < n; i++)
            for (int64_t c = c0; c < c1; c++) dx[(bt * n + i) * width + c] = 0.0;
        for (int64_t i = 0; i < n; i++) {
            const double* gi = dy + (bt * n + i) * width;
            double* dxi = dx + (bt * n + i) * width;
            for (int64_t o = 0; o < width; o++)
                for (int64_t c = c0; c < c1; c++) dxi[c] += w_self[o * width + c] * gi[o];
            if (oracle_receives(i, layer, n, causal)) {
                int64_t p = oracle_partner(i, layer, n);
                double* dxp = dx + (bt * n + p) * width;
                for (int64_t o = 0; o < width; o++)
                    for (int64_t c = c0; c < c1; c++) dxp[c] += w_off[o * width + c] * gi[o];
            }
        }
    }

    /* weight gradients: each output row o is owned by one thread. */
#pragma omp parallel for schedule(static)
    for (int64_t o = 0; o < width; o++) {
        double* gs = dw_self + o * width;
        double* go = dw_off + o * width;
        for (int64_t c = 0; c < width; c++) { gs[c] = 0.0; go[c] = 0.0; }
        for (int64_t r = 0; r < rows; r++) {
            int64_t bt = r / n, i = r % n;
            double g = dy[r * width + o];
            const double* xi = x + r * width;
            for (int64_t c = 0; c < width; c++) gs[c] += g * xi[c];
            if (oracle_receives(i, layer, n, causal)) {
                const double* xp = x + (bt * n + oracle_partner(i, layer, n)) * width;
                for (int64_t c = 0; c < width; c++) go[c] += g * xp[c];
            }
        }
    }
    return 0;
}
