/*
 * oracle.c -- plain, slow, fp64 CPU reference for causal RoPE attention with
 * per-RoPE-wavelength distance windows (ATFlash, arXiv 2608.02947).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The GPU product path
 * never calls it, and it shares no code, header, table or helper with that
 * path.
 *
 * What it computes, with the paper's notation:
 *   - theta_r = B^(-2r/d) for pair r = 0..d/2-1, or a caller-supplied effective
 *     theta'_r (Sec. 3.1; Sec. 3.2 last paragraph for rope scaling).
 *   - wavelength lambda_r = 2*pi / theta_r (Sec. 3.1, eq:lambda).
 *   - window w_r = min(k * lambda_r, N) (Sec. 3.2, eq:window), or a member of
 *     the window family w_r = min(max(k_r lambda_r^gamma + a(r+1)/(d/2), beta), W)
 *     (App. A, eq:family).
 *   - the rotated score split into pair terms (Sec. 3.1, eq:pair): pair r of a
 *     rotate-half vector is dims (r, r + d/2), and its term is
 *     q[r]k[r] + q[r+d/2]k[r+d/2].  At cell (n, m), z = n - m, a pair term is
 *     kept only when z <= w_r (Sec. 3.2); the kept terms are summed and scaled
 *     by 1/sqrt(d) (or a caller scale).  An empty sum is 0: tokens are never
 *     dropped, only terms.
 *   - optionally the rounded slice of Sec. 3.3: at each distance the kept
 *     low-frequency slice is rounded up to a whole number of MMA K-steps.
 *   - causal softmax over keys m <= n and the weighted sum of V rows, done as a
 *     plain two-pass softmax (max, then sum of exponentials); LSE = m + ln(l).
 *   - the retained-term count of Sec. 4: the number of kept (cell, pair)
 *     terms, and the number of causal cells.
 *
 * Everything is evaluated in fp64.  bf16 inputs are widened exactly.
 * No tiling, no online recurrence, no slicing: one row at a time, one key at a
 * time, one pair at a time.  OpenMP only splits independent rows.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* element types of the input arrays */
enum { ORACLE_F64 = 0, ORACLE_BF16 = 1 };

static double bf16_bits_to_double(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16; /* bf16 is the top half of an fp32 */
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static double load_elem(const void *base, int64_t idx, int dtype)
{
    if (dtype == ORACLE_BF16)
        return bf16_bits_to_double(((const uint16_t *)base)[idx]);
    return ((const double *)base)[idx];
}

/*
 * Window widths w_r = min(k * lambda_r, n_ctx), lambda_r = 2*pi/theta_r
 * (eq:window, eq:lambda).  theta == NULL means theta_r = base^(-2r/d).
 * k may be +INFINITY (window off).  theta_r == 0 gives an infinite wavelength
 * (a position-free pair, App. A), so w_r = n_ctx.
 * Returns 0, or -1 on bad arguments.
 */
int oracle_window_widths(int64_t d, double base, double k, const double *theta,
                         double n_ctx, double *w_out)
{
    if (d <= 0 || d % 2 != 0 || !(k > 0) || w_out == NULL)
        return -1;
    const double two_pi = 2.0 * 3.14159265358979323846;
    for (int64_t r = 0; r < d / 2; ++r) {
        double th = theta ? theta[r] : pow(base, -2.0 * (double)r / (double)d);
        if (!(th >= 0.0))
            return -1;
        double lambda = two_pi / th; /* +inf when th == 0 */
        double kl = k * lambda;
        w_out[r] = kl < n_ctx ? kl : n_ctx;
    }
    return 0;
}

/*
 * Window family (App. A, eq:family): for each pair r,
 *   w_r = min( max( k_r * lambda_r^gamma + a * (r + 1) / (d/2), beta ), cap )
 * with the retention profile k_r = k_prof[r], the wavelength exponent gamma, the
 * additive term a (linear in r, no wavelength in it), the floor beta and the
 * ceiling cap (the W of eq:family; +INFINITY for none).  The default window is
 * k_r = k, gamma = 1, a = 0, beta = 0, cap = N.
 * A position-free pair (theta_r == 0) has no wavelength: App. A treats it as
 * the theta -> 0 limit that is never pruned, a knob apart from the family, so
 * its width is +INFINITY whatever the other parameters are.
 * Returns 0, or -1 on bad arguments or when a width is NaN.
 */
int oracle_family_widths(int64_t d, double base, const double *theta, const double *k_prof,
                         double gamma, double a, double beta, double cap, double *w_out)
{
    if (d <= 0 || d % 2 != 0 || k_prof == NULL || w_out == NULL)
        return -1;
    const double two_pi = 2.0 * 3.14159265358979323846;
    const double half = (double)(d / 2);
    for (int64_t r = 0; r < d / 2; ++r) {
        double th = theta ? theta[r] : pow(base, -2.0 * (double)r / (double)d);
        if (!(th >= 0.0))
            return -1;
        if (th == 0.0) {
            w_out[r] = INFINITY;
            continue;
        }
        double lambda = two_pi / th;
        double w = k_prof[r] * pow(lambda, gamma) + a * (double)(r + 1) / half;
        if (w < beta)
            w = beta;
        if (w > cap)
            w = cap;
        if (isnan(w))
            return -1;
        w_out[r] = w;
    }
    return 0;
}

/*
 * Pairs kept at distance z.  atom == 0: the window itself, pair r is kept iff
 * z <= w_r (Sec. 3.2).  atom > 0: the rounded slice of Sec. 3.3: the pairs the
 * window keeps form a slice on the low-frequency side (the largest r); its length
 * n = #{r : z <= w_r} is rounded up to a whole number of K-steps of `atom` pairs,
 * n' = min(h, atom * ceil(n / atom)), and the kept pairs are r >= h - n'.
 * keep[r] receives 1 for a kept pair; returns the number kept.
 */
static int64_t kept_set(double z, const double *w, int64_t h, int64_t atom, unsigned char *keep)
{
    int64_t n = 0;
    for (int64_t r = 0; r < h; ++r)
        n += z <= w[r];
    if (atom <= 0) {
        for (int64_t r = 0; r < h; ++r)
            keep[r] = z <= w[r];
        return n;
    }
    int64_t nr = atom * ((n + atom - 1) / atom);
    if (nr > h)
        nr = h;
    for (int64_t r = 0; r < h; ++r)
        keep[r] = r >= h - nr;
    return nr;
}

/* The rounded slice is defined for a window whose kept pairs are a suffix in r:
 * widths non-decreasing in r. */
static int widths_monotone(const double *w, int64_t h)
{
    for (int64_t r = 1; r < h; ++r)
        if (!(w[r] >= w[r - 1]))
            return 0;
    return 1;
}

/*
 * Windowed score of one cell: (1/sqrt(d) or scale) * sum over kept pairs of
 * q[r]k[r] + q[r+h]k[r+h] (eq:pair with the keep rule of Sec. 3.2, or the
 * rounded slice of Sec. 3.3 when atom > 0).
 * qd holds the query row in fp64; krow points at the key row.
 * *kept receives the number of kept pairs.
 */
static double cell_score(const double *qd, const void *k, int64_t krow_off, int kdt,
                         int64_t d, double z, const double *w, int64_t atom, double scale,
                         int64_t *kept)
{
    const int64_t h = d / 2;
    unsigned char keep[512];
    *kept = kept_set(z, w, h, atom, keep);
    double x = 0.0;
    for (int64_t r = 0; r < h; ++r) {
        if (keep[r]) {
            x += qd[r] * load_elem(k, krow_off + r, kdt)
               + qd[r + h] * load_elem(k, krow_off + r + h, kdt);
        }
    }
    return x * scale;
}

/*
 * Scores of one (batch, query head) slice: s[i][j] for i < n_q, j < n_k.
 * Cells with key position j > query position q_pos0 + i get -INFINITY.
 * Layouts: q [B][n_q][h_q][d], k [B][n_k][h_kv][d]; s_out [n_q][n_k].
 * The key head of query head hq is hq / (h_q / h_kv).
 */
int oracle_scores(const void *q, const void *k, int dtype,
                  int64_t batch, int64_t n_q, int64_t n_k, int64_t q_pos0,
                  int64_t h_q, int64_t h_kv, int64_t d,
                  const double *w, int64_t atom, double scale, int64_t b, int64_t hq,
                  double *s_out)
{
    if (d <= 0 || d % 2 || h_kv <= 0 || h_q % h_kv || b < 0 || b >= batch ||
        hq < 0 || hq >= h_q || d > 1024 || (atom > 0 && !widths_monotone(w, d / 2)))
        return -1;
    const int64_t g = hq / (h_q / h_kv);
    double qd[1024];
    for (int64_t i = 0; i < n_q; ++i) {
        const int64_t qoff = ((b * n_q + i) * h_q + hq) * d;
        for (int64_t x = 0; x < d; ++x)
            qd[x] = load_elem(q, qoff + x, dtype);
        const int64_t p = q_pos0 + i;
        for (int64_t j = 0; j < n_k; ++j) {
            if (j > p) {
                s_out[i * n_k + j] = -INFINITY;
                continue;
            }
            int64_t kept;
            const int64_t koff = ((b * n_k + j) * h_kv + g) * d;
            s_out[i * n_k + j] = cell_score(qd, k, koff, dtype, d, (double)(p - j),
                                            w, atom, scale, &kept);
        }
    }
    return 0;
}

/*
 * Windowed causal attention for a list of query rows (atom: see kept_set).
 *   rows: n_rows triples (b, hq, i); row i sits at position q_pos0 + i and
 *         attends keys j = 0 .. min(q_pos0 + i, n_k - 1).
 *   o_out [n_rows][d], lse_out [n_rows], terms_out [n_rows] (may be NULL).
 * Returns 0, or -1 on bad arguments (including a row with no key).
 */
int oracle_attend(const void *q, const void *k, const void *v, int dtype,
                  int64_t batch, int64_t n_q, int64_t n_k, int64_t q_pos0,
                  int64_t h_q, int64_t h_kv, int64_t d,
                  const double *w, int64_t atom, double scale,
                  int64_t n_rows, const int64_t *rows,
                  double *o_out, double *lse_out, uint64_t *terms_out,
                  int n_threads)
{
    if (d <= 0 || d % 2 || d > 1024 || h_kv <= 0 || h_q % h_kv || n_k <= 0 ||
        q_pos0 < 0 || rows == NULL || o_out == NULL || lse_out == NULL ||
        (atom > 0 && !widths_monotone(w, d / 2)))
        return -1;
    for (int64_t t = 0; t < n_rows; ++t) {
        const int64_t b = rows[3 * t], hq = rows[3 * t + 1], i = rows[3 * t + 2];
        if (b < 0 || b >= batch || hq < 0 || hq >= h_q || i < 0 || i >= n_q)
            return -1;
    }
    const int64_t group = h_q / h_kv;
    int bad = 0;
#ifdef _OPENMP
    if (n_threads > 0)
        omp_set_num_threads(n_threads);
#else
    (void)n_threads;
#endif
#pragma omp parallel reduction(| : bad)
    {
        double *s = (double *)malloc(sizeof(double) * (size_t)n_k);
        double qd[1024];
        if (s == NULL)
            bad = 1;
#pragma omp for schedule(dynamic, 1)
        for (int64_t t = 0; t < n_rows; ++t) {
            if (s == NULL)
                continue;
            const int64_t b = rows[3 * t], hq = rows[3 * t + 1], i = rows[3 * t + 2];
            const int64_t g = hq / group;
            const int64_t p = q_pos0 + i;
            const int64_t last = p < n_k - 1 ? p : n_k - 1; /* causal: keys j <= p */
            const int64_t qoff = ((b * n_q + i) * h_q + hq) * d;
            for (int64_t x = 0; x < d; ++x)
                qd[x] = load_elem(q, qoff + x, dtype);

            /* pass 1: windowed scores and their maximum */
            double m = -INFINITY;
            uint64_t kept_total = 0;
            for (int64_t j = 0; j <= last; ++j) {
                int64_t kept;
                const int64_t koff = ((b * n_k + j) * h_kv + g) * d;
                s[j] = cell_score(qd, k, koff, dtype, d, (double)(p - j), w, atom, scale,
                                  &kept);
                kept_total += (uint64_t)kept;
                if (s[j] > m)
                    m = s[j];
            }
            /* pass 2: normaliser and weighted sum of V rows */
            double l = 0.0;
            double *o = o_out + t * d;
            for (int64_t x = 0; x < d; ++x)
                o[x] = 0.0;
            for (int64_t j = 0; j <= last; ++j) {
                const double e = exp(s[j] - m);
                l += e;
                const int64_t voff = ((b * n_k + j) * h_kv + g) * d;
                for (int64_t x = 0; x < d; ++x)
                    o[x] += e * load_elem(v, voff + x, dtype);
            }
            for (int64_t x = 0; x < d; ++x)
                o[x] /= l;
            lse_out[t] = m + log(l);
            if (terms_out)
                terms_out[t] = kept_total;
        }
        free(s);
    }
    return bad ? -1 : 0;
}

/*
 * Retained-term count of Sec. 4 for one (batch, query head): rows at positions
 * q_pos0 .. q_pos0 + n_q - 1, keys 0 .. n_k - 1, causal (key <= query).
 * For each row p and pair r the kept keys are those j in [0, min(p, n_k - 1)]
 * with p - j <= w_r, i.e. j >= p - floor(w_r); their number is the length of
 * that integer interval.  *causal_out is the number of causal cells.
 */
int oracle_count_terms(const double *w, int64_t n_pairs, int64_t n_q, int64_t q_pos0,
                       int64_t n_k, uint64_t *retained_out, uint64_t *causal_out);

/*
 * The same count with the keep rule of kept_set (atom > 0: the rounded slice of
 * Sec. 3.3), summed by distance: the cells at distance z are the rows p in
 * [max(q_pos0, z), min(q_pos0 + n_q - 1, z + n_k - 1)] (key j = p - z must lie in
 * [0, n_k - 1]), and each keeps kept_set(z) pairs.
 */
int oracle_count_terms_by_distance(const double *w, int64_t n_pairs, int64_t atom,
                                   int64_t n_q, int64_t q_pos0, int64_t n_k,
                                   uint64_t *retained_out, uint64_t *causal_out)
{
    if (n_pairs <= 0 || n_pairs > 512 || n_q < 0 || q_pos0 < 0 || n_k < 0 ||
        retained_out == NULL || causal_out == NULL ||
        (atom > 0 && !widths_monotone(w, n_pairs)))
        return -1;
    const int64_t p0 = q_pos0, p1 = q_pos0 + n_q - 1;
    uint64_t retained = 0, causal = 0;
#pragma omp parallel for reduction(+ : retained, causal) schedule(static)
    for (int64_t z = 0; z <= p1; ++z) {
        const int64_t lo = p0 > z ? p0 : z;
        const int64_t hi = p1 < z + n_k - 1 ? p1 : z + n_k - 1;
        if (hi < lo)
            continue;
        unsigned char keep[512];
        const int64_t kept = kept_set((double)z, w, n_pairs, atom, keep);
        causal += (uint64_t)(hi - lo + 1);
        retained += (uint64_t)(hi - lo + 1) * (uint64_t)kept;
    }
    *retained_out = retained;
    *causal_out = causal;
    return 0;
}

int oracle_count_terms(const double *w, int64_t n_pairs, int64_t n_q, int64_t q_pos0,
                       int64_t n_k, uint64_t *retained_out, uint64_t *causal_out)
{
    if (n_pairs <= 0 || n_q < 0 || q_pos0 < 0 || n_k < 0 || retained_out == NULL ||
        causal_out == NULL)
        return -1;
    uint64_t retained = 0, causal = 0;
#pragma omp parallel for reduction(+ : retained, causal) schedule(static)
    for (int64_t i = 0; i < n_q; ++i) {
        const int64_t p = q_pos0 + i;
        const int64_t last = p < n_k - 1 ? p : n_k - 1;
        if (last < 0)
            continue;
        causal += (uint64_t)(last + 1);
        for (int64_t r = 0; r < n_pairs; ++r) {
            const double lo = (double)p - floor(w[r]);
            if (!(lo <= (double)last))
                continue; /* no key is close enough (also w_r < 0) */
            const int64_t first = lo <= 0.0 ? 0 : (int64_t)lo;
            retained += (uint64_t)(last - first + 1);
        }
    }
    *retained_out = retained;
    *causal_out = causal;
    return 0;
}
