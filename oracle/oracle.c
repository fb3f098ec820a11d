/*
 * Reference oracle for fork-aware decode attention -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg load this
 * library.  It shares no code, header or table with the HIP library: it is a
 * plain, slow, obviously correct fp64 implementation of what the GPU path
 * computes, so that the GPU path can be compared against it.
 *
 * What is computed (paper, Sec. 3.3 Forking via Trajectory Continuation): at the
 * fork instant each branch receives the same snapshot -- the history H_t and the
 * thought R_t -- followed by its own continuation, and the key/value cache of the
 * shared part is reused by all decoding streams (Sec. 3.2: main thread plus four
 * branches decoding concurrently).  Reuse is an optimisation only, so the result
 * for branch b is ordinary attention of b's query over the concatenation
 * [shared prefix ; b's own suffix].  The paper never writes the attention formula;
 * the standard scaled dot-product softmax attention is used, with no bias, mask,
 * window or soft-cap:
 *
 *   g      = h / G                       (grouped query heads, G = Hq / Hkv)
 *   s_j    = scale * sum_c q[b][h][c] * K_b[j][c]
 *   m      = max_j s_j ;  l = sum_j exp(s_j - m)
 *   o[c]   = sum_j exp(s_j - m) * V_b[j][c] / l ;   lse = m + ln l
 *
 * An empty context gives o = 0 and lse = -inf.  Inputs are bf16 bit patterns,
 * widened exactly to fp64; all arithmetic is fp64, two passes over the keys.
 *
 * Paged storage: position p of sequence i lives in pool page
 * page_table[i][p / P] at slot p % P when p is a prefix position; suffix position
 * u starts on a fresh page, at page index ceil(Lp / P) + u / P, slot u % P.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double widen(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Attention of one query row over an ordered list of key/value rows. */
static void attend_row(const uint16_t *q, int d, double scale, long n, const uint16_t *const *krow,
                       const uint16_t *const *vrow, double *s, double *o, double *lse)
{
    for (int c = 0; c < d; ++c) o[c] = 0.0;
    if (n == 0) {
        *lse = -INFINITY;
        return;
    }
    double m = -INFINITY;
    for (long j = 0; j < n; ++j) {
        double acc = 0.0;
        for (int c = 0; c < d; ++c) acc += widen(q[c]) * widen(krow[j][c]);
        s[j] = scale * acc;
        if (s[j] > m) m = s[j];
    }
    double l = 0.0;
    for (long j = 0; j < n; ++j) {
        double p = exp(s[j] - m);
        l += p;
        for (int c = 0; c < d; ++c) o[c] += p * widen(vrow[j][c]);
    }
    for (int c = 0; c < d; ++c) o[c] /= l;
    *lse = m + log(l);
}

/*
 * Contiguous layout.
 *   q         [N][Hq][d]        prefix_k/v [Hkv][Lp][d]
 *   suffix_k/v [N][Hkv][cap][d] suffix_len [N]
 * Only prefix positions [p_lo, p_hi) and suffix positions [s_lo, min(s_hi, len_b))
 * are included, so the same routine gives the full result (0, Lp, 0, cap) and the
 * attention restricted to one chunk of keys.
 * rows: optional list of n_rows row ids (b * Hq + h); NULL computes all N*Hq rows.
 * out [N][Hq][d] and out_lse [N][Hq] are written only at the computed rows.
 */
int oracle_decode_contig(int N, int Hq, int Hkv, int d, double scale, const uint16_t *q, int Lp,
                         const uint16_t *prefix_k, const uint16_t *prefix_v, int cap,
                         const uint16_t *suffix_k, const uint16_t *suffix_v, const int32_t *suffix_len,
                         int p_lo, int p_hi, int s_lo, int s_hi, const int32_t *rows, int n_rows,
                         double *out, double *out_lse)
{
    if (N < 0 || Hq <= 0 || Hkv <= 0 || d <= 0 || Hq % Hkv != 0) return -1;
    if (p_lo < 0) p_lo = 0;
    if (p_hi > Lp) p_hi = Lp;
    if (p_hi < p_lo) p_hi = p_lo;
    if (s_lo < 0) s_lo = 0;
    const int G = Hq / Hkv;
    const int total = rows ? n_rows : N * Hq;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int t = 0; t < total; ++t) {
        const int row = rows ? rows[t] : t;
        const int b = row / Hq, h = row % Hq, g = h / G;
        const int len = suffix_len[b];
        if (len < 0 || len > cap) {  /* a suffix holds 0..cap tokens: anything else is not an input */
            bad |= 2;
            continue;
        }
        int shi = s_hi < len ? s_hi : len;
        int nsuf = shi > s_lo ? shi - s_lo : 0;
        long n = (long)(p_hi - p_lo) + nsuf;
        const uint16_t **kr = malloc(sizeof(*kr) * (size_t)(n ? n : 1));
        const uint16_t **vr = malloc(sizeof(*vr) * (size_t)(n ? n : 1));
        double *s = malloc(sizeof(double) * (size_t)(n ? n : 1));
        if (!kr || !vr || !s) {
            bad = 1;
        } else {
            long j = 0;
            for (int p = p_lo; p < p_hi; ++p, ++j) {
                kr[j] = prefix_k + ((size_t)g * Lp + p) * d;
                vr[j] = prefix_v + ((size_t)g * Lp + p) * d;
            }
            for (int u = s_lo; u < shi; ++u, ++j) {
                kr[j] = suffix_k + (((size_t)b * Hkv + g) * cap + u) * d;
                vr[j] = suffix_v + (((size_t)b * Hkv + g) * cap + u) * d;
            }
            attend_row(q + ((size_t)b * Hq + h) * d, d, scale, n, kr, vr, s, out + (size_t)row * d,
                       out_lse + row);
        }
        free(kr);
        free(vr);
        free(s);
    }
    return (bad & 2) ? -3 : bad ? -2 : 0;
}

/* Pool address of logical position p of sequence `seq` (prefix length Lp). */
static const uint16_t *paged_row(const uint16_t *pool, long n_pages, const int32_t *page_table, int max_pages,
                                 int seq, int Lp, int P, int Hkv, int d, int g, long p)
{
    long page_idx, slot;
    if (p < Lp) {
        page_idx = p / P;
        slot = p % P;
    } else {
        long u = p - Lp;
        page_idx = (Lp + P - 1) / P + u / P;
        slot = u % P;
    }
    if (page_idx >= max_pages) return NULL;
    int32_t page = page_table[(size_t)seq * max_pages + page_idx];
    if (page < 0 || page >= n_pages) return NULL;
    return pool + (((size_t)page * Hkv + g) * P + slot) * d;
}

/*
 * Paged layout.
 *   q [S][Hq][d]; k_pool/v_pool [n_pages][Hkv][P][d]; page_table [S][max_pages]
 *   seq_prefix_len [S]; suffix_len [S]
 * rows: optional list of row ids (i * Hq + h).  Returns -3 on a missing page.
 */
int oracle_decode_paged(int S, int Hq, int Hkv, int d, double scale, const uint16_t *q, int P,
                        const uint16_t *k_pool, const uint16_t *v_pool, long n_pages, const int32_t *page_table,
                        int max_pages, const int32_t *seq_prefix_len, const int32_t *suffix_len,
                        const int32_t *rows, int n_rows, double *out, double *out_lse)
{
    if (S < 0 || Hq <= 0 || Hkv <= 0 || d <= 0 || P <= 0 || Hq % Hkv != 0) return -1;
    const int G = Hq / Hkv;
    const int total = rows ? n_rows : S * Hq;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int t = 0; t < total; ++t) {
        const int row = rows ? rows[t] : t;
        const int i = row / Hq, h = row % Hq, g = h / G;
        const int Lp = seq_prefix_len[i];
        if (suffix_len[i] < 0 || Lp < 0) {  /* not an input: lengths are counts */
            bad |= 4;
            continue;
        }
        long n = (long)Lp + suffix_len[i];
        const uint16_t **kr = malloc(sizeof(*kr) * (size_t)(n ? n : 1));
        const uint16_t **vr = malloc(sizeof(*vr) * (size_t)(n ? n : 1));
        double *s = malloc(sizeof(double) * (size_t)(n ? n : 1));
        if (!kr || !vr || !s) {
            bad |= 2;
        } else {
            int ok = 1;
            for (long p = 0; p < n; ++p) {
                kr[p] = paged_row(k_pool, n_pages, page_table, max_pages, i, Lp, P, Hkv, d, g, p);
                vr[p] = paged_row(v_pool, n_pages, page_table, max_pages, i, Lp, P, Hkv, d, g, p);
                if (!kr[p] || !vr[p]) ok = 0;
            }
            if (ok)
                attend_row(q + ((size_t)i * Hq + h) * d, d, scale, n, kr, vr, s, out + (size_t)row * d,
                           out_lse + row);
            else
                bad |= 4;
        }
        free(kr);
        free(vr);
        free(s);
    }
    return bad ? (bad & 4 ? -3 : -2) : 0;
}

/*
 * Copy the K and V rows of one paged sequence, in logical order, into contiguous
 * [Hkv][L][d] arrays, L = prefix + suffix length.  Pure data movement.
 */
int oracle_gather_paged(int Hkv, int d, int P, const uint16_t *k_pool, const uint16_t *v_pool, long n_pages,
                        const int32_t *page_table, int max_pages, int seq, int Lp, int Ls, uint16_t *k_out,
                        uint16_t *v_out)
{
    if (Lp < 0 || Ls < 0) return -1;
    long L = (long)Lp + Ls;
    for (int g = 0; g < Hkv; ++g)
        for (long p = 0; p < L; ++p) {
            const uint16_t *kr = paged_row(k_pool, n_pages, page_table, max_pages, seq, Lp, P, Hkv, d, g, p);
            const uint16_t *vr = paged_row(v_pool, n_pages, page_table, max_pages, seq, Lp, P, Hkv, d, g, p);
            if (!kr || !vr) return -3;
            memcpy(k_out + ((size_t)g * L + p) * d, kr, sizeof(uint16_t) * (size_t)d);
            memcpy(v_out + ((size_t)g * L + p) * d, vr, sizeof(uint16_t) * (size_t)d);
        }
    return 0;
}

/*
 * Combine attention results computed over disjoint key sets into the result over
 * their union.  With part p holding normalised output o_p and log-sum-exp lse_p,
 * softmax over the union weights part p by exp(lse_p) / sum_q exp(lse_q):
 *   o = sum_p exp(lse_p - M) o_p / sum_p exp(lse_p - M),  lse = M + ln sum_p exp(lse_p - M)
 * with M = max_p lse_p (any M gives the same value; the max keeps exp in range).
 * Parts with lse = -inf carry no keys and get weight 0; if every part is empty the
 * result is o = 0, lse = -inf.
 *   o_parts [rows][n_parts][d], lse_parts [rows][n_parts], out [rows][d], out_lse [rows]
 */
int oracle_lse_merge(int rows, int n_parts, int d, const double *o_parts, const double *lse_parts, double *out,
                     double *out_lse)
{
    if (rows < 0 || n_parts < 0 || d <= 0) return -1;
#pragma omp parallel for schedule(static)
    for (int r = 0; r < rows; ++r) {
        const double *lp = lse_parts + (size_t)r * n_parts;
        double M = -INFINITY;
        for (int p = 0; p < n_parts; ++p)
            if (lp[p] > M) M = lp[p];
        double *o = out + (size_t)r * d;
        for (int c = 0; c < d; ++c) o[c] = 0.0;
        if (M == -INFINITY) {
            out_lse[r] = -INFINITY;
            continue;
        }
        double wsum = 0.0;
        for (int p = 0; p < n_parts; ++p) {
            if (lp[p] == -INFINITY) continue;
            double w = exp(lp[p] - M);
            wsum += w;
            const double *op = o_parts + ((size_t)r * n_parts + p) * d;
            for (int c = 0; c < d; ++c) o[c] += w * op[c];
        }
        for (int c = 0; c < d; ++c) o[c] /= wsum;
        out_lse[r] = M + log(wsum);
    }
    return 0;
}

/* Sets the threads of the following parallel regions (n >= 1); used to time the oracle on one
 * core and on all of them. */
void oracle_set_threads(int n)
{
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    omp_set_num_threads(n > 0 ? n : 1);
#else
    (void)n;
#endif
}

/* Threads an OpenMP parallel region uses (reported next to oracle timings). */
int oracle_threads(void)
{
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}
