/*
 * CPU oracle for the CoSpec verify-and-arbitrate step.
 *
 * TEST INFRASTRUCTURE ONLY.  The test suite, the package smoke check and the
 * benchmark's CPU-baseline leg are the only code allowed to load this library.
 * It shares no code, header, table or helper with the GPU path, and it is never
 * a fallback for it.
 *
 * Everything is computed in double precision with plain sequential loops that
 * follow the definitions they cite ("Beyond the Target: From Imitation to
 * Collaboration in Speculative Decoding", Section 3).  bf16 inputs are widened
 * exactly (bf16 -> fp32 by placing the 16 stored bits in the high half, fp32 ->
 * fp64 exactly).  Nothing here is blocked, fused or reordered.
 *
 * The scans (Eq. cospec_length, the tree reading) and the policy threshold live
 * in the Python half of the oracle (oracle/__init__.py); this file holds the two
 * loops that touch every logit or every weight.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

enum { ORACLE_F32 = 0, ORACLE_BF16 = 1 };

/* Element i of an array of fp32 values or of raw bf16 bit patterns, as a double. */
static double oracle_elem(const void *base, int dtype, int64_t i)
{
    if (dtype == ORACLE_F32)
        return (double)((const float *)base)[i];
    uint32_t bits = (uint32_t)((const uint16_t *)base)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/*
 * Statistics of `nrows` logit rows (row r starts at element r*ld) over the
 * whole vocabulary [0, V):
 *   max      m = max_v x[v]
 *   argmax   the first v with x[v] = m.  With greedy decoding (Appendix C.3)
 *            the target's verification token is the argmax of its row
 *            (Section 3.1); ties go to the lowest index.
 *   lse      log sum_v exp(x[v])  (the log-softmax normaliser), computed as
 *            m + log sum_v exp(x[v] - m)
 *   entropy  H = -sum_v p[v] log p[v] in nats, with p = softmax(x) and
 *            log p[v] = x[v] - lse.
 * Returns 0, or -(r+1) when row r holds a non-finite entry (finite logits
 * are a precondition).
 */
int64_t oracle_row_stats(const void *rows, int dtype, int64_t ld, int64_t nrows, int64_t V,
                         double *out_max, int64_t *out_arg, double *out_lse, double *out_ent)
{
    size_t esz = dtype == ORACLE_F32 ? 4 : 2;
    for (int64_t r = 0; r < nrows; ++r) {
        const void *row = (const char *)rows + (size_t)r * (size_t)ld * esz;
        double m = -INFINITY;
        int64_t arg = -1;
        for (int64_t v = 0; v < V; ++v) {
            double x = oracle_elem(row, dtype, v);
            if (!isfinite(x))
                return -(r + 1);
            if (x > m) {            /* strict: the first occurrence of the max wins */
                m = x;
                arg = v;
            }
        }
        double s = 0.0;
        for (int64_t v = 0; v < V; ++v)
            s += exp(oracle_elem(row, dtype, v) - m);
        double lse = m + log(s);
        double h = 0.0;
        for (int64_t v = 0; v < V; ++v) {
            double logp = oracle_elem(row, dtype, v) - lse;
            h -= exp(logp) * logp;
        }
        out_max[r] = m;
        out_arg[r] = arg;
        out_lse[r] = lse;
        out_ent[r] = h;
    }
    return 0;
}

/*
 * Arbitration head g_phi applied to selected hidden rows (Section 3.3:
 * z_i = g_phi(h_{l_c+1+i})).  The paper gives g_phi no explicit form beyond a small
 * head with one logit; it is read here as a two-layer MLP with a ReLU:
 *     u = W1 h + b1   (W1: [hdim][d] row-major, b1: [hdim] or absent = 0)
 *     z = w2 . max(u, 0) + b2
 * Row k of the output uses hidden row rows[k] (which starts at element
 * rows[k]*ld_h).  hidden, W1, b1 and w2 share `dtype`.
 */
void oracle_head(const void *hidden, int dtype, int64_t ld_h, const int64_t *rows, int64_t nsel,
                 const void *w1, const void *b1, const void *w2, double b2, int64_t d,
                 int64_t hdim, double *out_z)
{
    size_t esz = dtype == ORACLE_F32 ? 4 : 2;
    for (int64_t k = 0; k < nsel; ++k) {
        const void *hrow = (const char *)hidden + (size_t)rows[k] * (size_t)ld_h * esz;
        double z = b2;
        for (int64_t j = 0; j < hdim; ++j) {
            double u = b1 ? oracle_elem(b1, dtype, j) : 0.0;
            for (int64_t c = 0; c < d; ++c)
                u += oracle_elem(w1, dtype, j * d + c) * oracle_elem(hrow, dtype, c);
            double r = u > 0.0 ? u : 0.0;
            z += oracle_elem(w2, dtype, j) * r;
        }
        out_z[k] = z;
    }
}

/*
 * Probabilities p[v] = exp(x[v] - lse) of one row, lse from oracle_row_stats.
 * Returns 0, or -1 for a non-finite entry.
 */
static int oracle_softmax_row(const void *row, int dtype, int64_t V, double *p)
{
    double m, lse, h;
    int64_t arg;
    if (oracle_row_stats(row, dtype, V, 1, V, &m, &arg, &lse, &h))
        return -1;
    for (int64_t v = 0; v < V; ++v)
        p[v] = exp(oracle_elem(row, dtype, v) - lse);
    return 0;
}

/*
 * Sampling at temperature 1 (Section 3.1, stochastic decoding; Appendix C.3: at
 * T = 1 the target's verification candidate is a sample from its next-token
 * distribution).  The sample is taken by inversion: given a uniform u in [0, 1)
 * for row r, the candidate is the smallest v whose cumulative probability
 * P(v) = p[0] + ... + p[v] (in index order, p = softmax(x)) exceeds u.  When
 * rounding leaves P(V-1) <= u, the candidate is the last v with p[v] > 0.
 * Writes the candidate and P(v-1), P(v) around it.  `work` holds V doubles.
 * Returns 0, or -(r+1) when row r holds a non-finite entry.
 */
int64_t oracle_sample_rows(const void *rows, int dtype, int64_t ld, int64_t nrows, int64_t V,
                           const double *u, double *work, int64_t *out_idx, double *out_lo,
                           double *out_hi)
{
    size_t esz = dtype == ORACLE_F32 ? 4 : 2;
    for (int64_t r = 0; r < nrows; ++r) {
        const void *row = (const char *)rows + (size_t)r * (size_t)ld * esz;
        if (oracle_softmax_row(row, dtype, V, work))
            return -(r + 1);
        double before = 0.0, at = 0.0;
        int64_t pick = -1, last = 0;
        for (int64_t v = 0; v < V; ++v) {
            at = before + work[v];
            if (work[v] > 0.0)
                last = v;
            if (at > u[r]) {
                pick = v;
                break;
            }
            before = at;
        }
        if (pick < 0) {            /* u at or above the rounded total */
            pick = last;
            before = 0.0;
            for (int64_t v = 0; v < pick; ++v)
                before += work[v];
            at = before + work[pick];
        }
        out_idx[r] = pick;
        out_lo[r] = before;
        out_hi[r] = at;
    }
    return 0;
}

/*
 * Cumulative probabilities P(idx[r]-1) and P(idx[r]) of row r (the interval of
 * u values that inversion maps to idx[r]), for checking a candidate another
 * implementation chose.  Returns 0, -(r+1) for a non-finite entry in row r, or
 * -(nrows+1) for an index outside [0, V).
 */
int64_t oracle_cdf_at(const void *rows, int dtype, int64_t ld, int64_t nrows, int64_t V,
                      const int64_t *idx, double *work, double *out_lo, double *out_hi)
{
    size_t esz = dtype == ORACLE_F32 ? 4 : 2;
    for (int64_t r = 0; r < nrows; ++r) {
        const void *row = (const char *)rows + (size_t)r * (size_t)ld * esz;
        if (idx[r] < 0 || idx[r] >= V)
            return -(nrows + 1);
        if (oracle_softmax_row(row, dtype, V, work))
            return -(r + 1);
        double before = 0.0;
        for (int64_t v = 0; v < idx[r]; ++v)
            before += work[v];
        out_lo[r] = before;
        out_hi[r] = before + work[idx[r]];
    }
    return 0;
}

/*
 * Resampling step of standard speculative sampling (the distribution-preserving
 * baseline the paper runs at T = 1, Section 3.1 (stochastic decoding) and Appendix C.3).  With p = the
 * softmax of a target row and q = the softmax of the draft row at the same
 * position, the residual distribution is max(0, p - q) / Z, Z = sum_v max(0,
 * p[v] - q[v]); with no draft row (drf == NULL) the distribution is p itself
 * (the bonus token after K accepted draft tokens).  For row r:
 *   query == NULL: inversion of u[r]: the smallest v whose cumulative weight
 *                  exceeds u[r] * Z (the last v of positive weight if rounding
 *                  leaves none); writes it to out_idx[r];
 *   query != NULL: the candidate is query[r].
 * out_lo[r], out_hi[r] = the normalised cumulative weight before and at the
 * candidate.  `work` holds 2 V doubles.  Returns 0, -(r+1) for a non-finite
 * entry in row r, or -(nrows+1) for a query outside [0, V).
 */
int64_t oracle_residual_sample(const void *tgt, const void *drf, int dtype, int64_t ld, int64_t nrows,
                               int64_t V, const double *u, const int64_t *query, double *work,
                               int64_t *out_idx, double *out_lo, double *out_hi)
{
    size_t esz = dtype == ORACLE_F32 ? 4 : 2;
    double *p = work, *q = work + V;
    for (int64_t r = 0; r < nrows; ++r) {
        const void *trow = (const char *)tgt + (size_t)r * (size_t)ld * esz;
        if (oracle_softmax_row(trow, dtype, V, p))
            return -(r + 1);
        if (drf) {
            const void *drow = (const char *)drf + (size_t)r * (size_t)ld * esz;
            if (oracle_softmax_row(drow, dtype, V, q))
                return -(r + 1);
            for (int64_t v = 0; v < V; ++v)
                p[v] = p[v] > q[v] ? p[v] - q[v] : 0.0;
        }
        double z = 0.0;
        for (int64_t v = 0; v < V; ++v)
            z += p[v];
        int64_t pick;
        if (query) {
            if (query[r] < 0 || query[r] >= V)
                return -(nrows + 1);
            pick = query[r];
        } else {
            double target = u[r] * z, cum = 0.0;
            int64_t last = 0;
            pick = -1;
            for (int64_t v = 0; v < V; ++v) {
                if (p[v] > 0.0)
                    last = v;
                cum += p[v];
                if (p[v] > 0.0 && cum > target) {
                    pick = v;
                    break;
                }
            }
            if (pick < 0)
                pick = last;
            out_idx[r] = pick;
        }
        double before = 0.0;
        for (int64_t v = 0; v < pick; ++v)
            before += p[v];
        out_lo[r] = before / z;
        out_hi[r] = (before + p[pick]) / z;
    }
    return 0;
}
