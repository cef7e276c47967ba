/*
 * Reference oracle for the quantized gated-Delta decode step.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
 * cpu_baseline leg of bench.py may load or call this library.  It shares no
 * code, header, table or helper with the HIP path: the pool layout below is
 * re-derived here from its written definition in include/stepq.h.
 *
 * Everything is plain loops in double precision, in the order the paper
 * states the computation.  OpenMP is used only across independent tiles.
 *
 * Notation (paper, Section 2): a tile is one (request, value head) state
 * S in R^{d_k x d_v}; key rows i, value columns j.  Row i holds a b_i-bit
 * signed integer code per entry with q_b = 2^(b-1) - 1 (Eq. 3).  The
 * dual-axis representation (Section 4.3) reconstructs
 *     S^_ij = r_i * c_j * z_ij
 * from the level z_ij of the stored integer q_ij, in one of two level
 * normalisations (argument levels):
 *   0 (N1): z = q / q_b, so |S^_ij| <= r_i c_j at every width (the reading
 *           that makes "r_i c_j >= |S_ij|" the no-clip condition of a
 *           symmetric absmax fit);
 *   1 (N2): z = 2^(8-b) q, the fixed normalisation of the paper's KDA
 *           codebook (Appendix C.1), whose largest level is 2^(8-b) q_b.
 *
 * FP16 pivot rows (Section 3.2, Table C1): a row of width 16 holds its
 * values as IEEE binary16 (pv, bit patterns, [dk][dv] per tile, only pivot
 * rows used) instead of codes and scales.  The update treats them like any
 * other row; their new values are X rounded to binary16 (nearest, ties to
 * even), and they take no part in the scale fits (Appendix C.1 fits the
 * non-pivot integer rows).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>
#include <stdlib.h>

static double qb_of(int b) { return (double)((1 << (b - 1)) - 1); }

/* q = z * inv_nu(b): N1 q_b, N2 2^(b-8) (exact).  top_of(b): the largest
 * level q_b / inv_nu(b), 1 under N1. */
static double inv_nu(int b, int levels) { return levels ? ldexp(1.0, b - 8) : qb_of(b); }
static double top_of(int b, int levels) { return levels ? qb_of(b) * ldexp(1.0, 8 - b) : 1.0; }

/* IEEE 754 binary16, from its definition: 1 sign bit, 5 exponent bits (bias
 * 15), 10 fraction bits; exponent 0 holds subnormals k 2^-24. */
static double h2d(uint16_t h)
{
    int sgn = (h >> 15) & 1, e = (h >> 10) & 31, f = h & 1023;
    double v;
    if (e == 0) v = ldexp((double)f, -24);
    else if (e == 31) v = f ? NAN : INFINITY;
    else v = ldexp((double)(1024 + f), e - 25);
    return sgn ? -v : v;
}

/* Round to the nearest binary16, ties to even; beyond the largest finite
 * value (65504) by half an ulp or more, to infinity. */
static uint16_t d2h(double x)
{
    uint16_t sgn = signbit(x) ? 0x8000u : 0u;
    double a = fabs(x);
    if (isnan(a)) return (uint16_t)(sgn | 0x7e00u);
    if (a >= 65520.0) return (uint16_t)(sgn | 0x7c00u);
    if (a < ldexp(1.0, -14)) {                    /* subnormal range: k 2^-24, k <= 1024 */
        double k = nearbyint(ldexp(a, 24));
        return (uint16_t)(sgn | (uint16_t)k);      /* k = 1024 is the smallest normal */
    }
    int e;
    frexp(a, &e);                                 /* a = m 2^e, m in [0.5, 1) */
    double m = nearbyint(ldexp(a, 11 - e));       /* 11 significant bits, in [1024, 2048] */
    if (m == 2048.0) {
        m = 1024.0;
        ++e;
    }
    int ef = e - 1 + 15;
    if (ef >= 31) return (uint16_t)(sgn | 0x7c00u);
    return (uint16_t)(sgn | (uint16_t)(ef << 10) | (uint16_t)((int)m - 1024));
}

void orc_half_to_double(size_t n, const uint16_t *h, double *out)
{
    for (size_t i = 0; i < n; ++i) out[i] = h2d(h[i]);
}

void orc_double_to_half(size_t n, const double *x, uint16_t *out)
{
    for (size_t i = 0; i < n; ++i) out[i] = d2h(x[i]);
}

/* Reconstruction of one tile (Section 4.3, and the stored binary16 values of
 * pivot rows). */
static void reconstruct_tile(int dk, int dv, const int8_t *ci, const uint16_t *pv, const float *rt,
                             const float *ct, const uint8_t *bt, double *Sh, int levels)
{
    for (int i = 0; i < dk; ++i) {
        if (bt[i] == 16) {
            for (int j = 0; j < dv; ++j) Sh[(size_t)i * dv + j] = h2d(pv[(size_t)i * dv + j]);
            continue;
        }
        double iv = inv_nu(bt[i], levels);
        for (int j = 0; j < dv; ++j)
            Sh[(size_t)i * dv + j] = (double)rt[i] * (double)ct[j] * (double)ci[(size_t)i * dv + j] / iv;
    }
}

/* Pivot rows of an updated tile: X rounded to binary16, codes 0; y (if
 * given) receives X itself for those rows. */
static void store_pivots(int dk, int dv, const uint8_t *bt, const double *X, uint16_t *pv_out,
                         int8_t *codes_out, double *y)
{
    for (int i = 0; i < dk; ++i) {
        if (bt[i] != 16) continue;
        for (int j = 0; j < dv; ++j) {
            size_t e = (size_t)i * dv + j;
            if (pv_out) pv_out[e] = d2h(X[e]);
            codes_out[e] = 0;
            if (y) y[e] = X[e];
        }
    }
}

/* ------------------------------------------------------------------------
 * Scale fit used by the setup step (Section 4.3, "Row factors"; the column
 * factor in its absmax form).
 *   m_i = (1/d_v) sum_j |S_ij|
 *   r_i = m_i^{1/2} w_i^{-1/2}
 *   c_j = max_i |S_ij| / (r_i top_i)    (so that r_i c_j top_i >= |S_ij|; top = 1 under N1)
 * A positive floor of 2^-60 keeps both factors strictly positive
 * (Appendix C.1 asks for a positive numerical floor).  The results are
 * rounded once to fp32, the storage precision of the scales.
 * w == NULL means w_i = 1.  bits (optional under N1, [n_tiles][dk]): rows of
 * width 16 (pivots) are left out of the column factor.
 */
void orc_fit_absmax(int n_tiles, int dk, int dv, const float *S, const double *w, const uint8_t *bits,
                    float *r_out, float *c_out, int levels)
{
    const double floor_ = ldexp(1.0, -60);
    #pragma omp parallel for schedule(static)
    for (int t = 0; t < n_tiles; ++t) {
        const float *St = S + (size_t)t * dk * dv;
        double *r = (double *)malloc(sizeof(double) * dk);
        for (int i = 0; i < dk; ++i) {
            double m = 0.0;
            for (int j = 0; j < dv; ++j) m += fabs((double)St[(size_t)i * dv + j]);
            m /= (double)dv;
            double wi = w ? w[(size_t)t * dk + i] : 1.0;
            double ri = sqrt(m / wi);
            if (ri < floor_) ri = floor_;
            r_out[(size_t)t * dk + i] = (float)ri;
            r[i] = (double)r_out[(size_t)t * dk + i];   /* the column fit sees the stored r */
        }
        for (int j = 0; j < dv; ++j) {
            double cj = 0.0;
            for (int i = 0; i < dk; ++i) {
                if (bits && bits[(size_t)t * dk + i] == 16) continue;     /* pivots keep their own values */
                double a = fabs((double)St[(size_t)i * dv + j]) / r[i];
                if (levels) a /= top_of(bits[(size_t)t * dk + i], levels);
                if (a > cj) cj = a;
            }
            if (cj < floor_) cj = floor_;
            /* stored rounded upward so that r_i c_j >= |S_ij| survives the
               rounding to fp32 */
            float cf = (float)cj;
            if ((double)cf < cj) cf = nextafterf(cf, INFINITY);
            c_out[(size_t)t * dv + j] = cf;
        }
        free(r);
    }
}

/* ------------------------------------------------------------------------
 * Quantizer (Eq. 3, applied to the dual-axis representation of Section 4.3):
 *   q_ij = clip(round(X_ij * inv_nu / (r_i c_j)), -q_b, q_b)     (inv_nu = q_b under N1)
 * round = nearest, ties to even (nearbyint under the default rounding mode).
 * bits: [n_tiles][dk].  y (optional) receives the unrounded X inv_nu/(r c).
 * Pivot rows (width 16): pv receives X in binary16, codes 0.
 */
void orc_quantize(int n_tiles, int dk, int dv, const double *X, const float *r, const float *c,
                  const uint8_t *bits, int8_t *codes, double *y, uint16_t *pv, int levels)
{
    #pragma omp parallel for schedule(static)
    for (int t = 0; t < n_tiles; ++t) {
        size_t nel = (size_t)dk * dv;
        store_pivots(dk, dv, bits + (size_t)t * dk, X + t * nel, pv ? pv + t * nel : NULL, codes + t * nel,
                     y ? y + t * nel : NULL);
        for (int i = 0; i < dk; ++i) {
            if (bits[(size_t)t * dk + i] == 16) continue;
            double qb = qb_of(bits[(size_t)t * dk + i]);
            double iv = inv_nu(bits[(size_t)t * dk + i], levels);
            double ri = (double)r[(size_t)t * dk + i];
            for (int j = 0; j < dv; ++j) {
                size_t e = ((size_t)t * dk + i) * dv + j;
                double s = X[e] * iv / (ri * (double)c[(size_t)t * dv + j]);
                if (y) y[e] = s;
                double n = nearbyint(s);
                if (n > qb) n = qb;
                if (n < -qb) n = -qb;
                codes[e] = (int8_t)n;
            }
        }
    }
}

/* Reconstruction (Section 4.3): S^_ij = r_i c_j q_ij / inv_nu(b_i); pivot
 * rows from their binary16 values. */
void orc_dequant(int n_tiles, int dk, int dv, const int8_t *codes, const float *r, const float *c,
                 const uint8_t *bits, const uint16_t *pv, double *S, int levels)
{
    #pragma omp parallel for schedule(static)
    for (int t = 0; t < n_tiles; ++t) {
        size_t nel = (size_t)dk * dv;
        reconstruct_tile(dk, dv, codes + t * nel, pv ? pv + t * nel : NULL, r + (size_t)t * dk,
                         c + (size_t)t * dv, bits + (size_t)t * dk, S + t * nel, levels);
    }
}

/* ------------------------------------------------------------------------
 * Gated Delta update on a real-valued state (Eq. 1, first form) with a
 * diagonal retention gate D = diag(d) -- the KDA form; GDN is d_i = alpha
 * for every i -- and the readout of Eq. 4 taken from X before any
 * requantization:
 *   R = D S                           retained state
 *   e_j = v_j - sum_i k_i R_ij        residual of the retrieval k^T R
 *   X_ij = R_ij + beta k_i e_j
 *   o_j = sum_i X_ij q_i              (X^T q)
 */
static void update_tile(int dk, int dv, const double *S, const double *q, const double *k,
                        const double *v, const double *d, double beta, double *X, double *o)
{
    for (int i = 0; i < dk; ++i)
        for (int j = 0; j < dv; ++j) X[(size_t)i * dv + j] = d[i] * S[(size_t)i * dv + j];
    for (int j = 0; j < dv; ++j) {
        double kr = 0.0;
        for (int i = 0; i < dk; ++i) kr += k[i] * X[(size_t)i * dv + j];
        double e = v[j] - kr;
        for (int i = 0; i < dk; ++i) X[(size_t)i * dv + j] += beta * k[i] * e;
    }
    for (int j = 0; j < dv; ++j) {
        double acc = 0.0;
        for (int i = 0; i < dk; ++i) acc += X[(size_t)i * dv + j] * q[i];
        o[j] = acc;
    }
}

/* gates: alpha [n] (scalar gate per tile) when per_row == 0, or d [n][dk] */
static const double *gate_of(const double *alpha, int per_row, int t, int dk, double *buf)
{
    if (per_row) return alpha + (size_t)t * dk;
    for (int i = 0; i < dk; ++i) buf[i] = alpha[t];
    return buf;
}

void orc_update_fp(int n_tiles, int dk, int dv, const double *S, const double *q, const double *k,
                   const double *v, const double *alpha, int per_row, const double *beta, double *X,
                   double *o)
{
    #pragma omp parallel for schedule(static)
    for (int t = 0; t < n_tiles; ++t) {
        double *buf = (double *)malloc(sizeof(double) * dk);
        update_tile(dk, dv, S + (size_t)t * dk * dv, q + (size_t)t * dk, k + (size_t)t * dk,
                    v + (size_t)t * dv, gate_of(alpha, per_row, t, dk, buf), beta[t],
                    X + (size_t)t * dk * dv, o + (size_t)t * dv);
        free(buf);
    }
}

/* ------------------------------------------------------------------------
 * One decode step on a quantized tile (Appendix C, Table C2, with frozen
 * scales):  reconstruct S^ (step 1), X = D S^ + beta k (v - k^T D S^)
 * (step 2; D = alpha I or diag(d)), emit o = X^T q before requantization
 * (step 3), requantize X on the same r, c and per-row widths (Eq. 3) as the
 * new codes.
 * y (optional) receives X inv_nu/(r c) before rounding (X itself on pivot
 * rows).  pv_in / pv_out: binary16 values of pivot rows (NULL without pivots).
 */
void orc_decode_step(int n_tiles, int dk, int dv, const int8_t *codes_in, const float *r,
                     const float *c, const uint8_t *bits, const double *q, const double *k,
                     const double *v, const double *alpha, int per_row, const double *beta,
                     int8_t *codes_out, double *o, double *y, const uint16_t *pv_in, uint16_t *pv_out,
                     int levels)
{
    #pragma omp parallel for schedule(dynamic, 4)
    for (int t = 0; t < n_tiles; ++t) {
        size_t nel = (size_t)dk * dv;
        double *Sh = (double *)malloc(sizeof(double) * nel);
        double *X = (double *)malloc(sizeof(double) * nel);
        double *gbuf = (double *)malloc(sizeof(double) * dk);
        const int8_t *ci = codes_in + (size_t)t * nel;
        const float *rt = r + (size_t)t * dk, *ct = c + (size_t)t * dv;
        const uint8_t *bt = bits + (size_t)t * dk;
        reconstruct_tile(dk, dv, ci, pv_in ? pv_in + (size_t)t * nel : NULL, rt, ct, bt, Sh, levels);
        update_tile(dk, dv, Sh, q + (size_t)t * dk, k + (size_t)t * dk, v + (size_t)t * dv,
                    gate_of(alpha, per_row, t, dk, gbuf), beta[t], X, o + (size_t)t * dv);
        store_pivots(dk, dv, bt, X, pv_out ? pv_out + (size_t)t * nel : NULL, codes_out + (size_t)t * nel,
                     y ? y + (size_t)t * nel : NULL);
        for (int i = 0; i < dk; ++i) {
            if (bt[i] == 16) continue;
            double qb = qb_of(bt[i]), iv = inv_nu(bt[i], levels);
            for (int j = 0; j < dv; ++j) {
                double s = X[(size_t)i * dv + j] * iv / ((double)rt[i] * (double)ct[j]);
                if (y) y[(size_t)t * nel + (size_t)i * dv + j] = s;
                double n = nearbyint(s);
                if (n > qb) n = qb;
                if (n < -qb) n = -qb;
                codes_out[(size_t)t * nel + (size_t)i * dv + j] = (int8_t)n;
            }
        }
        free(Sh);
        free(X);
        free(gbuf);
    }
}

/* ------------------------------------------------------------------------
 * One decode step with the online Key-Row-Aware Dual-Axis refit (Appendix
 * C, Table C2 steps 1-6; Section 4.3 "Row factors" and "Column factors";
 * the fixed-code column update of Appendix C.1).  Steps 1-3 are those of
 * orc_decode_step (X and o).  Then, per tile, with row-impact factors w
 * (w == NULL: w_i = 1):
 *   row factors   m_i = (1/d_v) sum_j |X_ij|,  r'_i = (m_i / w_i)^{1/2}
 *   column start  c0_j = max_i |X_ij| / (r'_i top_i)   (absmax: no fixed code clips)
 *   fixed codes   z_ij = clip(round(X_ij inv_nu / (r'_i c0_j)), -q_b, q_b) / inv_nu   (the levels)
 *   column fit    c'_j = sum_i w_i^2 v_ij X_ij / sum_i w_i^2 v_ij^2,  v_ij = r'_i z_ij
 *                 (minimiser of sum_i w_i^2 (X_ij - r'_i c z_ij)^2 over c)
 *                 a zero denominator keeps the previous scale c_j
 *   requantize    q'_ij = clip(round(X_ij inv_nu / (r'_i c'_j)), -q_b, q_b)
 * (inv_nu = q_b and top = 1 under N1.)
 * r', c0 and c' are floored at 2^-60.  r' and c' are the stored scales:
 * each is rounded to fp32 when it is formed, and what follows it uses the
 * rounded value.
 * Optional outputs: y (X inv_nu / (r' c') before rounding), y0 (X inv_nu /
 * (r' c0) before rounding), X.  Pivot rows (width 16) are updated in binary16
 * (pv_in / pv_out), keep their stored r, and are left out of both fits.
 *
 * c_lo, c_hi (optional, for comparing with lower-precision implementations):
 * bounds on the column factor over every other rounding of the fixed codes
 * whose y0 lies within tie_window of a rounding boundary (a rounding that
 * arithmetic of lower precision may legitimately take).  Each such code
 * moves the two sums by a known amount; the bounds combine the extremes,
 * num_lo / den_hi and num_hi / den_lo, so they enclose every combination.
 * When a combination can empty the denominator the previous scale is in the
 * range and c_hi is +inf.
 */
void orc_decode_step_refit(int n_tiles, int dk, int dv, const int8_t *codes_in, const float *r,
                           const float *c, const uint8_t *bits, const double *w, const double *q,
                           const double *k, const double *v, const double *alpha, int per_row,
                           const double *beta, int8_t *codes_out, float *r_out, float *c_out, double *o,
                           double *y, double *y0, double *X_out, double tie_window, double *c_lo,
                           double *c_hi, const uint16_t *pv_in, uint16_t *pv_out, int levels)
{
    const double floor_ = ldexp(1.0, -60);
    #pragma omp parallel for schedule(dynamic, 4)
    for (int t = 0; t < n_tiles; ++t) {
        size_t nel = (size_t)dk * dv;
        double *Sh = (double *)malloc(sizeof(double) * nel);
        double *X = (double *)malloc(sizeof(double) * nel);
        double *gbuf = (double *)malloc(sizeof(double) * dk);
        double *rn = (double *)malloc(sizeof(double) * dk);
        double *zt = (double *)malloc(sizeof(double) * nel);
        const int8_t *ci = codes_in + (size_t)t * nel;
        const float *rt = r + (size_t)t * dk, *ct = c + (size_t)t * dv;
        const uint8_t *bt = bits + (size_t)t * dk;
        reconstruct_tile(dk, dv, ci, pv_in ? pv_in + (size_t)t * nel : NULL, rt, ct, bt, Sh, levels);
        update_tile(dk, dv, Sh, q + (size_t)t * dk, k + (size_t)t * dk, v + (size_t)t * dv,
                    gate_of(alpha, per_row, t, dk, gbuf), beta[t], X, o + (size_t)t * dv);
        if (X_out) memcpy(X_out + (size_t)t * nel, X, sizeof(double) * nel);
        store_pivots(dk, dv, bt, X, pv_out ? pv_out + (size_t)t * nel : NULL, codes_out + (size_t)t * nel,
                     y ? y + (size_t)t * nel : NULL);

        /* row factors (a pivot row keeps its stored, unused, factor) */
        for (int i = 0; i < dk; ++i) {
            if (bt[i] == 16) {
                r_out[(size_t)t * dk + i] = rt[i];
                rn[i] = (double)rt[i];
                continue;
            }
            double m = 0.0;
            for (int j = 0; j < dv; ++j) m += fabs(X[(size_t)i * dv + j]);
            m /= (double)dv;
            double wi = w ? w[(size_t)t * dk + i] : 1.0;
            double ri = sqrt(m / wi);
            if (ri < floor_) ri = floor_;
            r_out[(size_t)t * dk + i] = (float)ri;
            rn[i] = (double)r_out[(size_t)t * dk + i];
        }
        for (int j = 0; j < dv; ++j) {
            /* absmax start of the column factor, then the fixed codes */
            double c0 = 0.0;
            for (int i = 0; i < dk; ++i) {
                if (bt[i] == 16) continue;
                double a = fabs(X[(size_t)i * dv + j]) / rn[i];
                if (levels) a /= top_of(bt[i], levels);
                if (a > c0) c0 = a;
            }
            if (c0 < floor_) c0 = floor_;
            for (int i = 0; i < dk; ++i) {
                if (bt[i] == 16) {
                    zt[(size_t)i * dv + j] = 0.0;            /* no part in the column fit */
                    if (y0) y0[(size_t)t * nel + (size_t)i * dv + j] = 0.0;
                    continue;
                }
                double qb = qb_of(bt[i]), iv = inv_nu(bt[i], levels);
                double s = X[(size_t)i * dv + j] * iv / (rn[i] * c0);
                if (y0) y0[(size_t)t * nel + (size_t)i * dv + j] = s;
                double n = nearbyint(s);
                if (n > qb) n = qb;
                if (n < -qb) n = -qb;
                zt[(size_t)i * dv + j] = n / iv;
            }
            /* weighted least squares in c with the codes held fixed */
            double num = 0.0, den = 0.0;
            for (int i = 0; i < dk; ++i) {
                double wi = w ? w[(size_t)t * dk + i] : 1.0;
                double vij = rn[i] * zt[(size_t)i * dv + j];
                num += wi * wi * vij * X[(size_t)i * dv + j];
                den += wi * wi * vij * vij;
            }
            double cj;
            if (den > 0.0) {
                cj = num / den;
                if (cj < floor_) cj = floor_;
            } else {
                cj = (double)ct[j];
            }
            c_out[(size_t)t * dv + j] = (float)cj;
            if (c_lo && c_hi) {
                double nlo = num, nhi = num, dlo = den, dhi = den;
                for (int i = 0; i < dk; ++i) {
                    if (bt[i] == 16) continue;
                    double qb = qb_of(bt[i]), iv = inv_nu(bt[i], levels);
                    double s = y0[(size_t)t * nel + (size_t)i * dv + j];
                    double a = fabs(s);
                    if (fabs(a - floor(a) - 0.5) > tie_window) continue;
                    double z = zt[(size_t)i * dv + j] * iv;
                    double alt = (z > s) ? z - 1.0 : z + 1.0;     /* the other neighbour of s */
                    if (alt > qb || alt < -qb) continue;
                    double wi = w ? w[(size_t)t * dk + i] : 1.0;
                    double v0 = rn[i] * z / iv, v1 = rn[i] * alt / iv;
                    double dn = wi * wi * (v1 - v0) * X[(size_t)i * dv + j];
                    double dd = wi * wi * (v1 * v1 - v0 * v0);
                    if (dn < 0) nlo += dn; else nhi += dn;
                    if (dd < 0) dlo += dd; else dhi += dd;
                }
                double lo, hi;
                if (dlo > 0.0) {
                    lo = nlo / dhi;
                    hi = nhi / dlo;
                    if (lo < floor_) lo = floor_;
                    if (hi < floor_) hi = floor_;
                    if (den <= 0.0) {          /* this column kept its scale */
                        if ((double)ct[j] < lo) lo = (double)ct[j];
                        if ((double)ct[j] > hi) hi = (double)ct[j];
                    }
                } else {
                    lo = (dhi > 0.0) ? nlo / dhi : (double)ct[j];
                    if (lo < floor_) lo = floor_;
                    if ((double)ct[j] < lo) lo = (double)ct[j];
                    hi = INFINITY;
                }
                c_lo[(size_t)t * dv + j] = lo;
                c_hi[(size_t)t * dv + j] = hi;
            }
        }
        /* requantize against the stored scales */
        for (int i = 0; i < dk; ++i) {
            if (bt[i] == 16) continue;
            double qb = qb_of(bt[i]), iv = inv_nu(bt[i], levels);
            for (int j = 0; j < dv; ++j) {
                double s = X[(size_t)i * dv + j] * iv / (rn[i] * (double)c_out[(size_t)t * dv + j]);
                if (y) y[(size_t)t * nel + (size_t)i * dv + j] = s;
                double n = nearbyint(s);
                if (n > qb) n = qb;
                if (n < -qb) n = -qb;
                codes_out[(size_t)t * nel + (size_t)i * dv + j] = (int8_t)n;
            }
        }
        free(Sh);
        free(X);
        free(gbuf);
        free(rn);
        free(zt);
    }
}

/* ------------------------------------------------------------------------
 * The Key-Row-Aware Dual-Axis fit of a given state X (Section 4.3,
 * Appendix C.1) -- the spatial codec used for calibration distortions
 * (Appendix A.3): per tile
 *   r_i = (m_i / w_i)^{1/2}, m_i = mean_j |X_ij|          (floor, stored fp32)
 *   c0_j = max_i |X_ij| / r_i                              (floor)
 *   z_ij = clip(round(X_ij q_b / (r_i c0_j))) / q_b
 *   c_j = sum_i w_i^2 v_ij X_ij / sum_i w_i^2 v_ij^2, v = r z   (floor, stored
 *         fp32; a zero denominator keeps c0_j, there being no earlier scale)
 *   codes = clip(round(X q_b / (r c)))                     (stored scales)
 * Pivot rows (16) take no part and get X rounded to binary16 (pv_out).
 */
void orc_fit_dual_axis(int n_tiles, int dk, int dv, const double *Xall, const uint8_t *bits, const double *w,
                       float *r_out, float *c_out, int8_t *codes_out, uint16_t *pv_out)
{
    const double floor_ = ldexp(1.0, -60);
    #pragma omp parallel for schedule(dynamic, 4)
    for (int t = 0; t < n_tiles; ++t) {
        size_t nel = (size_t)dk * dv;
        const double *X = Xall + (size_t)t * nel;
        const uint8_t *bt = bits + (size_t)t * dk;
        double *rn = (double *)malloc(sizeof(double) * dk);
        double *zt = (double *)malloc(sizeof(double) * nel);
        store_pivots(dk, dv, bt, X, pv_out ? pv_out + (size_t)t * nel : NULL, codes_out + (size_t)t * nel, NULL);
        for (int i = 0; i < dk; ++i) {
            rn[i] = 1.0;
            if (bt[i] == 16) {
                r_out[(size_t)t * dk + i] = 1.0f;
                continue;
            }
            double m = 0.0;
            for (int j = 0; j < dv; ++j) m += fabs(X[(size_t)i * dv + j]);
            m /= (double)dv;
            double wi = w ? w[(size_t)t * dk + i] : 1.0;
            double ri = sqrt(m / wi);
            if (ri < floor_) ri = floor_;
            r_out[(size_t)t * dk + i] = (float)ri;
            rn[i] = (double)r_out[(size_t)t * dk + i];
        }
        for (int j = 0; j < dv; ++j) {
            double c0 = 0.0;
            for (int i = 0; i < dk; ++i) {
                if (bt[i] == 16) continue;
                double a = fabs(X[(size_t)i * dv + j]) / rn[i];
                if (a > c0) c0 = a;
            }
            if (c0 < floor_) c0 = floor_;
            double num = 0.0, den = 0.0;
            for (int i = 0; i < dk; ++i) {
                if (bt[i] == 16) continue;
                double qb = qb_of(bt[i]);
                double n = nearbyint(X[(size_t)i * dv + j] * qb / (rn[i] * c0));
                if (n > qb) n = qb;
                if (n < -qb) n = -qb;
                double wi = w ? w[(size_t)t * dk + i] : 1.0;
                double vij = rn[i] * n / qb;
                num += wi * wi * vij * X[(size_t)i * dv + j];
                den += wi * wi * vij * vij;
            }
            double cj = den > 0.0 ? num / den : c0;
            if (cj < floor_) cj = floor_;
            c_out[(size_t)t * dv + j] = (float)cj;
        }
        for (int i = 0; i < dk; ++i) {
            if (bt[i] == 16) continue;
            double qb = qb_of(bt[i]);
            for (int j = 0; j < dv; ++j) {
                double s = X[(size_t)i * dv + j] * qb / (rn[i] * (double)c_out[(size_t)t * dv + j]);
                double n = nearbyint(s);
                if (n > qb) n = qb;
                if (n < -qb) n = -qb;
                codes_out[(size_t)t * nel + (size_t)i * dv + j] = (int8_t)n;
            }
        }
        free(rn);
        free(zt);
    }
}

/* ------------------------------------------------------------------------
 * One decode step of the single-axis baseline the paper compares against
 * (Section 5.1: symmetric row-wise absmax INT-b), on the same quantized
 * tile: steps 1-3 of orc_decode_step, then per key row
 *   r'_i = max_j |X_ij| / top_i  (floor 2^-60, stored fp32),   c'_j = 1,
 *   q'_ij = clip(round(X_ij inv_nu / r'_i), -q_b, q_b)    with the stored r',
 * so each row's largest entry lands on the top level (inv_nu = q_b and
 * top = 1 under N1).  y (optional) receives X inv_nu / r' before rounding.  Pivot rows as in
 * orc_decode_step_refit.
 */
void orc_decode_step_rowmax(int n_tiles, int dk, int dv, const int8_t *codes_in, const float *r,
                            const float *c, const uint8_t *bits, const double *q, const double *k,
                            const double *v, const double *alpha, int per_row, const double *beta,
                            int8_t *codes_out, float *r_out, float *c_out, double *o, double *y,
                            const uint16_t *pv_in, uint16_t *pv_out, int levels)
{
    const double floor_ = ldexp(1.0, -60);
    #pragma omp parallel for schedule(dynamic, 4)
    for (int t = 0; t < n_tiles; ++t) {
        size_t nel = (size_t)dk * dv;
        double *Sh = (double *)malloc(sizeof(double) * nel);
        double *X = (double *)malloc(sizeof(double) * nel);
        double *gbuf = (double *)malloc(sizeof(double) * dk);
        const int8_t *ci = codes_in + (size_t)t * nel;
        const float *rt = r + (size_t)t * dk, *ct = c + (size_t)t * dv;
        const uint8_t *bt = bits + (size_t)t * dk;
        reconstruct_tile(dk, dv, ci, pv_in ? pv_in + (size_t)t * nel : NULL, rt, ct, bt, Sh, levels);
        update_tile(dk, dv, Sh, q + (size_t)t * dk, k + (size_t)t * dk, v + (size_t)t * dv,
                    gate_of(alpha, per_row, t, dk, gbuf), beta[t], X, o + (size_t)t * dv);
        for (int j = 0; j < dv; ++j) c_out[(size_t)t * dv + j] = 1.0f;
        store_pivots(dk, dv, bt, X, pv_out ? pv_out + (size_t)t * nel : NULL, codes_out + (size_t)t * nel,
                     y ? y + (size_t)t * nel : NULL);
        for (int i = 0; i < dk; ++i) {
            if (bt[i] == 16) {
                r_out[(size_t)t * dk + i] = rt[i];
                continue;
            }
            double m = 0.0;
            for (int j = 0; j < dv; ++j) {
                double a = fabs(X[(size_t)i * dv + j]);
                if (a > m) m = a;
            }
            if (levels) m /= top_of(bt[i], levels);
            if (m < floor_) m = floor_;
            r_out[(size_t)t * dk + i] = (float)m;
            double ri = (double)r_out[(size_t)t * dk + i];
            double qb = qb_of(bt[i]), iv = inv_nu(bt[i], levels);
            for (int j = 0; j < dv; ++j) {
                double s = X[(size_t)i * dv + j] * iv / ri;
                if (y) y[(size_t)t * nel + (size_t)i * dv + j] = s;
                double n = nearbyint(s);
                if (n > qb) n = qb;
                if (n < -qb) n = -qb;
                codes_out[(size_t)t * nel + (size_t)i * dv + j] = (int8_t)n;
            }
        }
        free(Sh);
        free(X);
        free(gbuf);
    }
}

/* ------------------------------------------------------------------------
 * Pool layout, re-derived from its definition in include/stepq.h:
 *  - physical key-row order: the pivot (16) rows, then the 8-bit rows, the
 *    4-bit rows and the 2-bit rows, each class in increasing logical index;
 *  - row groups of 8/b physical integer rows of one width (1, 2 or 4 rows);
 *    a last partial group of a width is completed with empty slots;
 *  - each group is d_v bytes; byte j holds column j, slot s of the group at
 *    bits [s*b, s*b+b) as b-bit two's complement, empty slots zero;
 *  - codes region padded with zeros to a multiple of 128 bytes; then the
 *    pivot rows, d_v binary16 values each (little-endian), in physical
 *    order; then r (d_k fp32, physical row order) and c (d_v fp32), the
 *    whole tile record padded with zeros to a multiple of 128 bytes.
 */
static size_t round128(size_t x) { return (x + 127) & ~(size_t)127; }

static void class_counts(int dk, const uint8_t *bits, int *n16, int *n8, int *n4, int *n2)
{
    *n16 = *n8 = *n4 = *n2 = 0;
    for (int i = 0; i < dk; ++i) {
        if (bits[i] == 16) ++*n16;
        else if (bits[i] == 8) ++*n8;
        else if (bits[i] == 4) ++*n4;
        else if (bits[i] == 2) ++*n2;
    }
}

/* Row groups of each width class.  Tight (one per 8-bit row, per two 4-bit
 * rows, per four 2-bit rows), except at d_k = d_v = 128 (whole-FP16 heads
 * aside): integer rows that fit one of the uniform mixes, in word-steps of
 * 8 groups {8-bit, 4-bit, 2-bit} and taken in this order, get exactly that
 * mix's group counts, the classes padded with empty groups. */
static const int uniform_mix[5][3] = {{8, 4, 0}, {4, 2, 2}, {16, 0, 0}, {0, 8, 0}, {0, 0, 4}};

static void class_groups(int dk, int dv, const uint8_t *bits, int *g8, int *g4, int *g2)
{
    int n16, n8, n4, n2;
    class_counts(dk, bits, &n16, &n8, &n4, &n2);
    *g8 = n8;
    *g4 = (n4 + 1) / 2;
    *g2 = (n2 + 3) / 4;
    if (dk != 128 || dv != 128 || n16 == dk) return;
    for (int L = 0; L < 5; ++L) {
        const int *m = uniform_mix[L];
        if (8 * m[0] >= n8 && 16 * m[1] >= n4 && 32 * m[2] >= n2) {
            *g8 = 8 * m[0];
            *g4 = 8 * m[1];
            *g2 = 8 * m[2];
            return;
        }
    }
}

static size_t codes_region(int dk, int dv, const uint8_t *bits)
{
    int g8, g4, g2;
    class_groups(dk, dv, bits, &g8, &g4, &g2);
    return round128((size_t)(g8 + g4 + g2) * (size_t)dv);
}

static size_t pivot_region(int dk, int dv, const uint8_t *bits)
{
    int n16, n8, n4, n2;
    class_counts(dk, bits, &n16, &n8, &n4, &n2);
    return round128((size_t)n16 * 2u * (size_t)dv);
}

size_t orc_tile_bytes(int dk, int dv, const uint8_t *bits)
{
    return round128(codes_region(dk, dv, bits) + pivot_region(dk, dv, bits) + 4u * (size_t)dk + 4u * (size_t)dv);
}

/* logical row of each physical row, and the (group, slot) position of each
 * logical integer row inside the codes region (pivot rows: their index
 * among the pivot rows in group, slot -1) */
static void row_positions(int dk, int dv, const uint8_t *bits, int *phys_to_log, int *group, int *slot)
{
    int n16, n8, n4, n2, c8, c4, c2;
    class_counts(dk, bits, &n16, &n8, &n4, &n2);
    class_groups(dk, dv, bits, &c8, &c4, &c2);
    int p = 0;
    static const int order[4] = {16, 8, 4, 2};
    for (int cl = 0; cl < 4; ++cl)
        for (int i = 0; i < dk; ++i)
            if (bits[i] == order[cl]) phys_to_log[p++] = i;
    int g4 = c8, g2 = c8 + c4;                     /* first 4-bit and 2-bit groups */
    (void)c2;
    for (int pp = 0; pp < dk; ++pp) {
        int i = phys_to_log[pp];
        int q = pp - n16;                          /* index among the integer rows */
        if (pp < n16) { group[i] = pp; slot[i] = -1; }
        else if (q < n8) { group[i] = q; slot[i] = 0; }
        else if (q < n8 + n4) { int k = q - n8; group[i] = g4 + k / 2; slot[i] = k % 2; }
        else { int k = q - n8 - n4; group[i] = g2 + k / 4; slot[i] = k % 4; }
    }
}

/* codes: [dk][dv] logical order; pv: [dk][dv] binary16 (pivot rows only;
 * NULL if there are none); r: [dk] logical order; c: [dv] */
void orc_pack_tile(int dk, int dv, const uint8_t *bits, const int8_t *codes, const uint16_t *pv,
                   const float *r, const float *c, uint8_t *rec)
{
    size_t creg = codes_region(dk, dv, bits);
    size_t preg = pivot_region(dk, dv, bits);
    size_t tb = orc_tile_bytes(dk, dv, bits);
    memset(rec, 0, tb);
    int *p2l = (int *)malloc(sizeof(int) * dk * 3);
    int *grp = p2l + dk, *slt = p2l + 2 * dk;
    row_positions(dk, dv, bits, p2l, grp, slt);
    for (int i = 0; i < dk; ++i) {
        int b = bits[i];
        if (b == 16) {
            uint8_t *row = rec + creg + (size_t)grp[i] * 2u * dv;
            for (int j = 0; j < dv; ++j) {
                uint16_t h = pv[(size_t)i * dv + j];
                row[2 * j] = (uint8_t)(h & 0xff);
                row[2 * j + 1] = (uint8_t)(h >> 8);
            }
            continue;
        }
        unsigned mask = (1u << b) - 1u;
        for (int j = 0; j < dv; ++j) {
            unsigned field = ((unsigned)(int)codes[(size_t)i * dv + j]) & mask;
            rec[(size_t)grp[i] * dv + j] |= (uint8_t)(field << (slt[i] * b));
        }
    }
    float *rr = (float *)(rec + creg + preg);
    float *cc = rr + dk;
    for (int p = 0; p < dk; ++p) rr[p] = r[p2l[p]];
    for (int j = 0; j < dv; ++j) cc[j] = c[j];
    free(p2l);
}

void orc_unpack_tile(int dk, int dv, const uint8_t *bits, const uint8_t *rec, int8_t *codes, uint16_t *pv,
                     float *r, float *c)
{
    size_t creg = codes_region(dk, dv, bits);
    size_t preg = pivot_region(dk, dv, bits);
    int *p2l = (int *)malloc(sizeof(int) * dk * 3);
    int *grp = p2l + dk, *slt = p2l + 2 * dk;
    row_positions(dk, dv, bits, p2l, grp, slt);
    for (int i = 0; i < dk; ++i) {
        int b = bits[i];
        if (b == 16) {
            const uint8_t *row = rec + creg + (size_t)grp[i] * 2u * dv;
            for (int j = 0; j < dv; ++j) {
                codes[(size_t)i * dv + j] = 0;
                if (pv) pv[(size_t)i * dv + j] = (uint16_t)(row[2 * j] | (row[2 * j + 1] << 8));
            }
            continue;
        }
        for (int j = 0; j < dv; ++j) {
            unsigned byte = rec[(size_t)grp[i] * dv + j];
            int field = (int)((byte >> (slt[i] * b)) & ((1u << b) - 1u));
            if (field >= (1 << (b - 1))) field -= (1 << b);    /* two's complement */
            codes[(size_t)i * dv + j] = (int8_t)field;
        }
    }
    const float *rr = (const float *)(rec + creg + preg);
    const float *cc = rr + dk;
    for (int p = 0; p < dk; ++p) r[p2l[p]] = rr[p];
    for (int j = 0; j < dv; ++j) c[j] = cc[j];
    free(p2l);
}

/* Whole-pool image: n_slots records, each the head tiles in order.
 * bits: [Hv][dk]; codes: [n_slots][Hv][dk][dv]; r: [n_slots][Hv][dk];
 * c: [n_slots][Hv][dv]. */
size_t orc_slot_bytes(int Hv, int dk, int dv, const uint8_t *bits)
{
    size_t s = 0;
    for (int h = 0; h < Hv; ++h) s += orc_tile_bytes(dk, dv, bits + (size_t)h * dk);
    return s;
}

void orc_pack_pool(int n_slots, int Hv, int dk, int dv, const uint8_t *bits, const int8_t *codes,
                   const uint16_t *pv, const float *r, const float *c, uint8_t *pool)
{
    size_t sb = orc_slot_bytes(Hv, dk, dv, bits);
    #pragma omp parallel for schedule(static)
    for (int s = 0; s < n_slots; ++s) {
        size_t off = (size_t)s * sb;
        for (int h = 0; h < Hv; ++h) {
            size_t t = (size_t)s * Hv + h;
            orc_pack_tile(dk, dv, bits + (size_t)h * dk, codes + t * dk * dv, pv ? pv + t * dk * dv : NULL,
                          r + t * dk, c + t * dv, pool + off);
            off += orc_tile_bytes(dk, dv, bits + (size_t)h * dk);
        }
    }
}

void orc_unpack_pool(int n_slots, int Hv, int dk, int dv, const uint8_t *bits, const uint8_t *pool,
                     int8_t *codes, uint16_t *pv, float *r, float *c)
{
    size_t sb = orc_slot_bytes(Hv, dk, dv, bits);
    #pragma omp parallel for schedule(static)
    for (int s = 0; s < n_slots; ++s) {
        size_t off = (size_t)s * sb;
        for (int h = 0; h < Hv; ++h) {
            size_t t = (size_t)s * Hv + h;
            orc_unpack_tile(dk, dv, bits + (size_t)h * dk, pool + off, codes + t * dk * dv,
                            pv ? pv + t * dk * dv : NULL, r + t * dk, c + t * dv);
            off += orc_tile_bytes(dk, dv, bits + (size_t)h * dk);
        }
    }
}

int orc_max_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of the tile loops from now on (n >= 1); for timing only. */
void orc_set_threads(int n)
{
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
