/*
 * EVA attention oracle: plain, slow, obviously correct CPU reference in fp64.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file.  Only the tests, the smoke check and the benchmark's CPU
 * baseline leg use it.  It shares no code, header, table or helper with the
 * HIP library.
 *
 * What it computes (FlashEVA, section "FlashEVA", the reformulation of EVA as
 * softmax attention over an augmented key/value set; with the local set E and
 * the disjoint chunk partition P_c of section "EVA Attention", eq. (eva) and
 * eq. (eva_normalization)):
 *
 *   Summaries, one per complete chunk c of C tokens, positions [cC, cC+C):
 *     khat_c = (1/C) * sum_j k_j                     (mean key)
 *     a_j    = khat_c . k_j / sqrt(d)
 *     vhat_c = sum_j softmax_j(a) * v_j             (query-independent value,
 *                                                    the S=1 property)
 *   Attention row n (causal):
 *     window   E(n) = [max(0, n-W+1), n]              (W tokens, self included)
 *     summaries c < s(n), s(n) = floor(max(0, n-W+1) / C)
 *                                   (only chunks lying fully before the window)
 *     logits   q_n.k_m / sqrt(d)          for m in E(n)
 *              q_n.khat_c / sqrt(d) + ln C for c < s(n)
 *     o_n = sum_i exp(l_i - max l) val_i / sum_i exp(l_i - max l)
 *
 * Everything is the plain definition: no tiling, no online softmax, no
 * reordering.  Inputs are fp64 copies of whatever the caller rounded them to.
 * The paper is silent on several details (window extent, chunk alignment,
 * tokens between the last summarized chunk and the window, the summary key
 * form, the logit offset, 1/sqrt(d) scaling, GQA head mapping); the readings
 * taken here are the ones listed in the design notes and are pinned by the
 * CPU tests (closed forms, reductions to exact softmax attention,
 * invariants).
 *
 * Layouts: row-major, contiguous.
 *   single sequence: K, V [L][d]; Ksum, Vsum [floor(L/C)][d]
 *   batched:         Q, O [B][H][L][d]; K, V [B][Hkv][L][d]
 *   GQA: query head h reads key/value head h / (H/Hkv).
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>

/* Number of chunk summaries visible to the query at position n. */
long eva_ref_visible_summaries(long n, long W, long C)
{
    long window_start = n - W + 1;
    if (window_start <= 0) return 0;
    return window_start / C;
}

/* Summaries of one sequence: for each complete chunk, the mean key and the
 * softmax(mean-key . key / sqrt(d))-weighted value. */
void eva_ref_summaries(const double* K, const double* V, long L, int d, long C,
                       double* Ksum, double* Vsum)
{
    long n_chunks = L / C;
    double inv_sqrt_d = 1.0 / sqrt((double)d);
    double* a = (double*)malloc((size_t)C * sizeof(double));
    for (long c = 0; c < n_chunks; ++c) {
        const double* Kc = K + (size_t)c * C * d;
        const double* Vc = V + (size_t)c * C * d;
        double* kh = Ksum + (size_t)c * d;
        double* vh = Vsum + (size_t)c * d;

        /* mean key */
        for (int e = 0; e < d; ++e) {
            double s = 0.0;
            for (long j = 0; j < C; ++j) s += Kc[(size_t)j * d + e];
            kh[e] = s / (double)C;
        }
        /* scores of each chunk key against the mean key */
        double amax = -INFINITY;
        for (long j = 0; j < C; ++j) {
            double s = 0.0;
            for (int e = 0; e < d; ++e) s += kh[e] * Kc[(size_t)j * d + e];
            a[j] = s * inv_sqrt_d;
            if (a[j] > amax) amax = a[j];
        }
        /* softmax-weighted value */
        double den = 0.0;
        for (long j = 0; j < C; ++j) den += exp(a[j] - amax);
        for (int e = 0; e < d; ++e) {
            double num = 0.0;
            for (long j = 0; j < C; ++j) num += exp(a[j] - amax) * Vc[(size_t)j * d + e];
            vh[e] = num / den;
        }
    }
    free(a);
}

/* Stochastic random-feature summaries (section "EVA Attention": with one
 * sample omega per chunk the chunk's value is the ratio of the sums of
 * g_m and h_m, in which every query-dependent factor is common to all terms
 * and cancels, leaving
 *     vhat_c = sum_j xi(k_j, omega) v_j / sum_j xi(k_j, omega),
 *     xi(x, omega) = exp(omega . x - |x|^2 / 2)
 * (section "Random Feature Attention"); the sample comes from the clipped,
 * downscaled proposal of the ablation "Impact of random feature sampling
 * distribution": omega = mu_c + lambda * clip(eps, -1, 1), eps ~ N(0, I)
 * given by the caller, mu_c the chunk's mean key).  The feature map acts on
 * the scaled keys x = k / d^(1/4), the scaling under which exp(q.k/sqrt(d))
 * is exp(q'.k'), so mu_c is the mean of the scaled keys.  The summary key is
 * the unscaled mean key, as for the deterministic summaries.
 * eps: [floor(L/C)][d], one draw per chunk. */
void eva_ref_summaries_rf(const double* K, const double* V, const double* eps, long L, int d, long C,
                          double lambda, double* Ksum, double* Vsum)
{
    long n_chunks = L / C;
    double inv_root4_d = 1.0 / sqrt(sqrt((double)d));
    double* a = (double*)malloc((size_t)C * sizeof(double));
    double* x = (double*)malloc((size_t)d * sizeof(double));
    double* omega = (double*)malloc((size_t)d * sizeof(double));
    for (long c = 0; c < n_chunks; ++c) {
        const double* Kc = K + (size_t)c * C * d;
        const double* Vc = V + (size_t)c * C * d;
        const double* ec = eps + (size_t)c * d;
        double* kh = Ksum + (size_t)c * d;
        double* vh = Vsum + (size_t)c * d;

        /* mean key, and the sample: mean scaled key + lambda * clip(eps) */
        for (int e = 0; e < d; ++e) {
            double s = 0.0;
            for (long j = 0; j < C; ++j) s += Kc[(size_t)j * d + e];
            kh[e] = s / (double)C;
            double clipped = ec[e] < -1.0 ? -1.0 : (ec[e] > 1.0 ? 1.0 : ec[e]);
            omega[e] = kh[e] * inv_root4_d + lambda * clipped;
        }
        /* log xi(x_j, omega) for the scaled keys x_j */
        double amax = -INFINITY;
        for (long j = 0; j < C; ++j) {
            double dot = 0.0, norm2 = 0.0;
            for (int e = 0; e < d; ++e) {
                x[e] = Kc[(size_t)j * d + e] * inv_root4_d;
                dot += omega[e] * x[e];
                norm2 += x[e] * x[e];
            }
            a[j] = dot - 0.5 * norm2;
            if (a[j] > amax) amax = a[j];
        }
        /* ratio of xi-weighted sums (the common factor exp(amax) cancels) */
        double den = 0.0;
        for (long j = 0; j < C; ++j) den += exp(a[j] - amax);
        for (int e = 0; e < d; ++e) {
            double num = 0.0;
            for (long j = 0; j < C; ++j) num += exp(a[j] - amax) * Vc[(size_t)j * d + e];
            vh[e] = num / den;
        }
    }
    free(a);
    free(x);
    free(omega);
}

/* Counter-based normal draws for the stochastic summaries (test
 * infrastructure for the paper's single-sample estimator: the draw of chunk
 * c of sequence-head s must be reproducible wherever the chunk's summary is
 * built, at prefill or when decode completes the chunk).
 *
 * Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
 * easy as 1, 2, 3", SC 2011): a 128-bit counter and a 64-bit key; each of ten
 * rounds multiplies counter words 0 and 2 by 0xD2511F53 and 0xCD9E8D57 into
 * 64-bit products (hi, lo) and produces
 *     (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0)),
 * the key advancing by (0x9E3779B9, 0xBB67AE85) between rounds. */
void eva_ref_philox4x32_10(const unsigned* ctr, const unsigned* key, unsigned* out)
{
    unsigned c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
    unsigned k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        unsigned long long p0 = (unsigned long long)0xD2511F53u * c[0];
        unsigned long long p1 = (unsigned long long)0xCD9E8D57u * c[2];
        unsigned hi0 = (unsigned)(p0 >> 32), lo0 = (unsigned)p0;
        unsigned hi1 = (unsigned)(p1 >> 32), lo1 = (unsigned)p1;
        unsigned n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0;
        c[1] = lo1;
        c[2] = n2;
        c[3] = lo0;
    }
    for (int i = 0; i < 4; ++i) out[i] = c[i];
}

/* eps[s][c][f] for s < n_seq, c < n_chunks, f < d (d a multiple of 4):
 * standard normal draws.  Features 4i .. 4i+3 of (s, c) come from one Philox
 * block, counter (i, c, s, 0), key (seed low word, seed high word); the
 * Box-Muller transform (G. E. P. Box and M. E. Muller, 1958) turns each pair of
 * its words (x, y) into two normals: with u = (x >> 8) + 1/2 and
 * v = (y >> 8) + 1/2 scaled by 2^-24 (24-bit uniforms on (0, 1)),
 * sqrt(-2 ln u) cos(2 pi v) and sqrt(-2 ln u) sin(2 pi v). */
void eva_ref_rf_noise(double* eps, long n_seq, long n_chunks, int d, unsigned long long seed)
{
    const unsigned key[2] = {(unsigned)seed, (unsigned)(seed >> 32)};
    const double two_pi = 6.283185307179586476925286766559;
    for (long s = 0; s < n_seq; ++s)
        for (long c = 0; c < n_chunks; ++c)
            for (int i = 0; i < d / 4; ++i) {
                const unsigned ctr[4] = {(unsigned)i, (unsigned)c, (unsigned)s, 0u};
                unsigned x[4];
                eva_ref_philox4x32_10(ctr, key, x);
                double* e = eps + ((size_t)s * n_chunks + c) * d + 4 * i;
                for (int h = 0; h < 2; ++h) {
                    double u = ((double)(x[2 * h] >> 8) + 0.5) / 16777216.0;
                    double v = ((double)(x[2 * h + 1] >> 8) + 0.5) / 16777216.0;
                    double r = sqrt(-2.0 * log(u));
                    e[2 * h] = r * cos(two_pi * v);
                    e[2 * h + 1] = r * sin(two_pi * v);
                }
            }
}

/* One attention row: query q at position n against the exact keys of its
 * window and the visible chunk summaries. */
void eva_ref_attend_row(const double* q, const double* K, const double* V,
                        const double* Ksum, const double* Vsum,
                        long n, int d, long W, long C, double* o)
{
    double inv_sqrt_d = 1.0 / sqrt((double)d);
    long lo = n - W + 1;
    if (lo < 0) lo = 0;
    long n_win = n - lo + 1;
    long n_sum = eva_ref_visible_summaries(n, W, C);
    long count = n_win + n_sum;

    double* logit = (double*)malloc((size_t)count * sizeof(double));
    const double** val = (const double**)malloc((size_t)count * sizeof(double*));
    long i = 0;
    for (long m = lo; m <= n; ++m, ++i) {
        double s = 0.0;
        for (int e = 0; e < d; ++e) s += q[e] * K[(size_t)m * d + e];
        logit[i] = s * inv_sqrt_d;
        val[i] = V + (size_t)m * d;
    }
    for (long c = 0; c < n_sum; ++c, ++i) {
        double s = 0.0;
        for (int e = 0; e < d; ++e) s += q[e] * Ksum[(size_t)c * d + e];
        logit[i] = s * inv_sqrt_d + log((double)C);
        val[i] = Vsum + (size_t)c * d;
    }

    double lmax = -INFINITY;
    for (i = 0; i < count; ++i)
        if (logit[i] > lmax) lmax = logit[i];
    double den = 0.0;
    for (i = 0; i < count; ++i) den += exp(logit[i] - lmax);
    for (int e = 0; e < d; ++e) {
        double num = 0.0;
        for (i = 0; i < count; ++i) num += exp(logit[i] - lmax) * val[i][e];
        o[e] = num / den;
    }
    free(logit);
    free(val);
}

/* Selected rows of one sequence: rows[r] is a position, Qrows[r] its query. */
/* Window variants (the ablation "EVA Local Window Attention Variants": the
 * original EVA's blocked local windows besides the sliding window of section
 * "FlashEVA"; the non-causal form of section "FlashEVA"; and a sliding window
 * extended down to its chunk boundary).  Row n of a sequence of L tokens
 * attends the exact keys m in [lo, hi] and the summaries of the complete
 * chunks c < n_chunks = floor(L / C) listed below:
 *   0 sliding        lo = max(0, n-W+1), hi = n;  chunks ending at or before lo
 *   1 chunk-aligned  s = floor(max(0, n-W+1) / C), lo = s*C, hi = n;  c < s
 *                    (no token between the summaries and the window)
 *   2 blocked        lo = floor(n/W)*W, hi = n;  chunks ending at or before lo
 *   3 non-causal     lo = floor(n/W)*W, hi = min(L, lo+W) - 1;  chunks ending
 *                    at or before lo and chunks starting after hi
 * Summary logits carry + ln C as in eva_ref_attend_row. */
void eva_ref_attend_row_variant(const double* q, const double* K, const double* V,
                                const double* Ksum, const double* Vsum,
                                long n, long L, int d, long W, long C, int variant, double* o)
{
    double inv_sqrt_d = 1.0 / sqrt((double)d);
    long n_chunks = L / C;
    long lo, hi;
    if (variant == 0) {
        lo = n - W + 1 < 0 ? 0 : n - W + 1;
        hi = n;
    } else if (variant == 1) {
        long start = n - W + 1 < 0 ? 0 : n - W + 1;
        lo = (start / C) * C;
        hi = n;
    } else if (variant == 2) {
        lo = (n / W) * W;
        hi = n;
    } else {
        lo = (n / W) * W;
        hi = lo + W - 1 < L - 1 ? lo + W - 1 : L - 1;
    }
    /* chunk c is summarized iff it lies wholly before lo, or (non-causal)
     * wholly after hi */
    char* take = (char*)calloc((size_t)(n_chunks > 0 ? n_chunks : 1), 1);
    long n_take = 0;
    for (long c = 0; c < n_chunks; ++c) {
        int before = (c + 1) * C <= lo;
        int after = variant == 3 && c * C > hi;
        take[c] = (char)(before || after);
        n_take += take[c];
    }
    long count = (hi - lo + 1) + n_take;
    double* logit = (double*)malloc((size_t)count * sizeof(double));
    const double** val = (const double**)malloc((size_t)count * sizeof(double*));
    long i = 0;
    for (long m = lo; m <= hi; ++m, ++i) {
        double s = 0.0;
        for (int e = 0; e < d; ++e) s += q[e] * K[(size_t)m * d + e];
        logit[i] = s * inv_sqrt_d;
        val[i] = V + (size_t)m * d;
    }
    for (long c = 0; c < n_chunks; ++c) {
        if (!take[c]) continue;
        double s = 0.0;
        for (int e = 0; e < d; ++e) s += q[e] * Ksum[(size_t)c * d + e];
        logit[i] = s * inv_sqrt_d + log((double)C);
        val[i] = Vsum + (size_t)c * d;
        ++i;
    }
    double lmax = -INFINITY;
    for (i = 0; i < count; ++i)
        if (logit[i] > lmax) lmax = logit[i];
    double den = 0.0;
    for (i = 0; i < count; ++i) den += exp(logit[i] - lmax);
    for (int e = 0; e < d; ++e) {
        double num = 0.0;
        for (i = 0; i < count; ++i) num += exp(logit[i] - lmax) * val[i][e];
        o[e] = num / den;
    }
    free(take);
    free(logit);
    free(val);
}

void eva_ref_attend_rows_variant(const double* Qrows, const long* rows, long n_rows,
                                 const double* K, const double* V,
                                 const double* Ksum, const double* Vsum,
                                 long L, int d, long W, long C, int variant, double* Orows)
{
    #pragma omp parallel for schedule(dynamic, 1)
    for (long r = 0; r < n_rows; ++r)
        eva_ref_attend_row_variant(Qrows + (size_t)r * d, K, V, Ksum, Vsum, rows[r], L, d, W, C, variant,
                                   Orows + (size_t)r * d);
}

void eva_ref_attend_rows(const double* Qrows, const long* rows, long n_rows,
                         const double* K, const double* V,
                         const double* Ksum, const double* Vsum,
                         int d, long W, long C, double* Orows)
{
    #pragma omp parallel for schedule(dynamic, 1)
    for (long r = 0; r < n_rows; ++r)
        eva_ref_attend_row(Qrows + (size_t)r * d, K, V, Ksum, Vsum, rows[r], d, W, C,
                           Orows + (size_t)r * d);
}

/* Whole prefill: summaries of every (b, kv head), then every row of every
 * query head.  Ksum/Vsum receive [B][Hkv][floor(L/C)][d]. */
/* Whole prefill with a window variant (see eva_ref_attend_row_variant). */
void eva_ref_prefill_variant(const double* Q, const double* K, const double* V, double* O,
                             int B, int H, int Hkv, long L, int d, long W, long C, int variant,
                             double* Ksum, double* Vsum)
{
    int G = H / Hkv;
    long n_chunks = L / C;
    size_t seq = (size_t)L * d;
    size_t sseq = (size_t)n_chunks * d;

    #pragma omp parallel for schedule(dynamic, 1)
    for (long bg = 0; bg < (long)B * Hkv; ++bg)
        eva_ref_summaries(K + bg * seq, V + bg * seq, L, d, C, Ksum + bg * sseq, Vsum + bg * sseq);

    #pragma omp parallel for collapse(2) schedule(dynamic, 16)
    for (long bh = 0; bh < (long)B * H; ++bh) {
        for (long n = 0; n < L; ++n) {
            long b = bh / H, h = bh % H;
            long bg = b * Hkv + h / G;
            eva_ref_attend_row_variant(Q + bh * seq + (size_t)n * d, K + bg * seq, V + bg * seq,
                                       Ksum + bg * sseq, Vsum + bg * sseq, n, L, d, W, C, variant,
                                       O + bh * seq + (size_t)n * d);
        }
    }
}

void eva_ref_prefill(const double* Q, const double* K, const double* V, double* O,
                     int B, int H, int Hkv, long L, int d, long W, long C,
                     double* Ksum, double* Vsum)
{
    int G = H / Hkv;
    long n_chunks = L / C;
    size_t seq = (size_t)L * d;
    size_t sseq = (size_t)n_chunks * d;

    #pragma omp parallel for schedule(dynamic, 1)
    for (long bg = 0; bg < (long)B * Hkv; ++bg)
        eva_ref_summaries(K + bg * seq, V + bg * seq, L, d, C, Ksum + bg * sseq, Vsum + bg * sseq);

    #pragma omp parallel for collapse(2) schedule(dynamic, 16)
    for (long bh = 0; bh < (long)B * H; ++bh) {
        for (long n = 0; n < L; ++n) {
            long b = bh / H, h = bh % H;
            long bg = b * Hkv + h / G;
            eva_ref_attend_row(Q + bh * seq + (size_t)n * d, K + bg * seq, V + bg * seq,
                               Ksum + bg * sseq, Vsum + bg * sseq, n, d, W, C,
                               O + bh * seq + (size_t)n * d);
        }
    }
}

/* The items row n attends under a window variant (see
 * eva_ref_attend_row_variant): exact keys [*lo, *hi], then the summaries
 * listed in sum_idx (ascending); returns how many summaries. */
static long variant_row_items(long n, long L, long W, long C, int variant, long* lo, long* hi, long* sum_idx)
{
    long n_chunks = L / C;
    if (variant == 0) {
        *lo = n - W + 1 < 0 ? 0 : n - W + 1;
        *hi = n;
    } else if (variant == 1) {
        long start = n - W + 1 < 0 ? 0 : n - W + 1;
        *lo = (start / C) * C;
        *hi = n;
    } else if (variant == 2) {
        *lo = (n / W) * W;
        *hi = n;
    } else {
        *lo = (n / W) * W;
        *hi = *lo + W - 1 < L - 1 ? *lo + W - 1 : L - 1;
    }
    long ns = 0;
    for (long c = 0; c < n_chunks; ++c)
        if ((c + 1) * C <= *lo || (variant == 3 && c * C > *hi)) sum_idx[ns++] = c;
    return ns;
}

/* Threads the OpenMP runtime will use (1 when built without OpenMP). */
/* Backward pass of the EVA prefill for one kv group: G query heads sharing
 * K, V.  Given dO (the gradient of a loss with respect to O), returns dQ,
 * dK, dV of that loss, through the window keys and values, the summary keys
 * and values, and the summaries' own dependence on K and V (the mean key and
 * the softmax(mean . k / sqrt(d))-weighted value).
 *   Q, dO, dQ: [G][L][d];  K, V, dK, dV: [L][d]  (dK, dV are overwritten).
 * Plain chain rule, row by row: with p the row's softmax over its items
 * (keys key_i, values val_i), o = sum_i p_i val_i and D = dO . o,
 *   dlogit_i = p_i (dO . val_i - D),  dq = sum_i dlogit_i key_i / sqrt(d),
 *   dkey_i += dlogit_i q / sqrt(d),   dval_i += p_i dO;
 * then for each chunk (a_j = khat . k_j / sqrt(d), b = softmax(a)):
 *   dv_j += b_j dvhat,  da_j = b_j (dvhat . v_j - dvhat . vhat),
 *   dkhat = dkey_c + sum_j da_j k_j / sqrt(d),
 *   dk_j += da_j khat / sqrt(d) + dkhat / C.
 * The + ln C logit offset is a constant. */
void eva_ref_backward_group_variant(const double* Q, const double* K, const double* V, const double* dO,
                                    int G, long L, int d, long W, long C, int variant,
                                    double* dQ, double* dK, double* dV)
{
    double inv_sqrt_d = 1.0 / sqrt((double)d);
    long n_chunks = L / C;
    size_t nc1 = (size_t)(n_chunks > 0 ? n_chunks : 1);
    double* Ks = (double*)calloc(nc1 * d, sizeof(double));
    double* Vs = (double*)calloc(nc1 * d, sizeof(double));
    double* dKs = (double*)calloc(nc1 * d, sizeof(double));
    double* dVs = (double*)calloc(nc1 * d, sizeof(double));
    eva_ref_summaries(K, V, L, d, C, Ks, Vs);
    memset(dK, 0, (size_t)L * d * sizeof(double));
    memset(dV, 0, (size_t)L * d * sizeof(double));

    long* sidx = (long*)malloc(nc1 * sizeof(long));
    double* logit = (double*)malloc((size_t)(L + nc1) * sizeof(double));
    double* p = (double*)malloc((size_t)(L + nc1) * sizeof(double));
    double* o = (double*)malloc((size_t)d * sizeof(double));
    for (int h = 0; h < G; ++h) {
        for (long n = 0; n < L; ++n) {
            const double* q = Q + ((size_t)h * L + n) * d;
            const double* g = dO + ((size_t)h * L + n) * d;
            double* dq = dQ + ((size_t)h * L + n) * d;
            long lo, hi;
            long n_sum = variant_row_items(n, L, W, C, variant, &lo, &hi, sidx);
            long n_win = hi - lo + 1;
            long count = n_win + n_sum;
            /* forward of the row: items 0..n_win-1 are keys lo..n, then summaries */
            double lmax = -INFINITY;
            for (long i = 0; i < count; ++i) {
                const double* key = i < n_win ? K + (size_t)(lo + i) * d : Ks + (size_t)sidx[i - n_win] * d;
                double s = 0.0;
                for (int e = 0; e < d; ++e) s += q[e] * key[e];
                logit[i] = s * inv_sqrt_d + (i < n_win ? 0.0 : log((double)C));
                if (logit[i] > lmax) lmax = logit[i];
            }
            double den = 0.0;
            for (long i = 0; i < count; ++i) {
                p[i] = exp(logit[i] - lmax);
                den += p[i];
            }
            for (long i = 0; i < count; ++i) p[i] /= den;
            for (int e = 0; e < d; ++e) {
                double acc = 0.0;
                for (long i = 0; i < count; ++i) {
                    const double* val = i < n_win ? V + (size_t)(lo + i) * d : Vs + (size_t)sidx[i - n_win] * d;
                    acc += p[i] * val[e];
                }
                o[e] = acc;
            }
            double D = 0.0;
            for (int e = 0; e < d; ++e) D += g[e] * o[e];
            /* backward of the row */
            for (int e = 0; e < d; ++e) dq[e] = 0.0;
            for (long i = 0; i < count; ++i) {
                const int win = i < n_win;
                const double* key = win ? K + (size_t)(lo + i) * d : Ks + (size_t)sidx[i - n_win] * d;
                const double* val = win ? V + (size_t)(lo + i) * d : Vs + (size_t)sidx[i - n_win] * d;
                double* dkey = win ? dK + (size_t)(lo + i) * d : dKs + (size_t)sidx[i - n_win] * d;
                double* dval = win ? dV + (size_t)(lo + i) * d : dVs + (size_t)sidx[i - n_win] * d;
                double gv = 0.0;
                for (int e = 0; e < d; ++e) gv += g[e] * val[e];
                const double dl = p[i] * (gv - D);
                for (int e = 0; e < d; ++e) {
                    dq[e] += dl * key[e] * inv_sqrt_d;
                    dkey[e] += dl * q[e] * inv_sqrt_d;
                    dval[e] += p[i] * g[e];
                }
            }
        }
    }
    /* through the summaries */
    double* a = (double*)malloc((size_t)C * sizeof(double));
    double* b = (double*)malloc((size_t)C * sizeof(double));
    double* dkh = (double*)malloc((size_t)d * sizeof(double));
    for (long c = 0; c < n_chunks; ++c) {
        const double* Kc = K + (size_t)c * C * d;
        const double* Vc = V + (size_t)c * C * d;
        const double* kh = Ks + (size_t)c * d;
        const double* vh = Vs + (size_t)c * d;
        const double* gk = dKs + (size_t)c * d;
        const double* gvh = dVs + (size_t)c * d;
        double amax = -INFINITY;
        for (long j = 0; j < C; ++j) {
            double s = 0.0;
            for (int e = 0; e < d; ++e) s += kh[e] * Kc[(size_t)j * d + e];
            a[j] = s * inv_sqrt_d;
            if (a[j] > amax) amax = a[j];
        }
        double den = 0.0;
        for (long j = 0; j < C; ++j) {
            b[j] = exp(a[j] - amax);
            den += b[j];
        }
        for (long j = 0; j < C; ++j) b[j] /= den;
        double gvh_vh = 0.0;
        for (int e = 0; e < d; ++e) gvh_vh += gvh[e] * vh[e];
        for (int e = 0; e < d; ++e) dkh[e] = gk[e];
        for (long j = 0; j < C; ++j) {
            double gv = 0.0;
            for (int e = 0; e < d; ++e) gv += gvh[e] * Vc[(size_t)j * d + e];
            const double da = b[j] * (gv - gvh_vh);
            for (int e = 0; e < d; ++e) {
                dV[((size_t)c * C + j) * d + e] += b[j] * gvh[e];
                dkh[e] += da * Kc[(size_t)j * d + e] * inv_sqrt_d;
                dK[((size_t)c * C + j) * d + e] += da * kh[e] * inv_sqrt_d;
            }
        }
        for (long j = 0; j < C; ++j)
            for (int e = 0; e < d; ++e) dK[((size_t)c * C + j) * d + e] += dkh[e] / (double)C;
    }
    free(a);
    free(b);
    free(dkh);
    free(sidx);
    free(logit);
    free(p);
    free(o);
    free(Ks);
    free(Vs);
    free(dKs);
    free(dVs);
}

/* The sliding window (variant 0). */
void eva_ref_backward_group(const double* Q, const double* K, const double* V, const double* dO,
                            int G, long L, int d, long W, long C,
                            double* dQ, double* dK, double* dV)
{
    eva_ref_backward_group_variant(Q, K, V, dO, G, L, d, W, C, 0, dQ, dK, dV);
}

/* Term magnitudes of eva_ref_backward_group, for rounding-error bounds (test
 * infrastructure: not part of the method).  Each gradient entry is a sum of
 * terms; this returns, per entry, the sum of the terms' absolute values,
 * carried through the same steps: a term that is itself a sum (the summary
 * gradients dkhat, dvhat and the chunk-logit gradients da_j) contributes the
 * magnitude of its own terms.  A floating-point evaluation that rounds each
 * term to relative precision u is then off by at most about u times this
 * magnitude, however much the terms cancel.  Same arguments and layouts as
 * eva_ref_backward_group; Tq, Tk, Tv take the places of dQ, dK, dV. */
void eva_ref_backward_terms_variant(const double* Q, const double* K, const double* V, const double* dO,
                                    int G, long L, int d, long W, long C, int variant,
                                    double* Tq, double* Tk, double* Tv)
{
    double inv_sqrt_d = 1.0 / sqrt((double)d);
    long n_chunks = L / C;
    size_t nc1 = (size_t)(n_chunks > 0 ? n_chunks : 1);
    double* Ks = (double*)calloc(nc1 * d, sizeof(double));
    double* Vs = (double*)calloc(nc1 * d, sizeof(double));
    double* Tks = (double*)calloc(nc1 * d, sizeof(double));
    double* Tvs = (double*)calloc(nc1 * d, sizeof(double));
    eva_ref_summaries(K, V, L, d, C, Ks, Vs);
    memset(Tk, 0, (size_t)L * d * sizeof(double));
    memset(Tv, 0, (size_t)L * d * sizeof(double));

    long* sidx = (long*)malloc(nc1 * sizeof(long));
    double* logit = (double*)malloc((size_t)(L + nc1) * sizeof(double));
    double* p = (double*)malloc((size_t)(L + nc1) * sizeof(double));
    double* o = (double*)malloc((size_t)d * sizeof(double));
    for (int h = 0; h < G; ++h) {
        for (long n = 0; n < L; ++n) {
            const double* q = Q + ((size_t)h * L + n) * d;
            const double* g = dO + ((size_t)h * L + n) * d;
            double* tq = Tq + ((size_t)h * L + n) * d;
            long lo, hi;
            long n_sum = variant_row_items(n, L, W, C, variant, &lo, &hi, sidx);
            long n_win = hi - lo + 1;
            long count = n_win + n_sum;
            double lmax = -INFINITY;
            for (long i = 0; i < count; ++i) {
                const double* key = i < n_win ? K + (size_t)(lo + i) * d : Ks + (size_t)sidx[i - n_win] * d;
                double s = 0.0;
                for (int e = 0; e < d; ++e) s += q[e] * key[e];
                logit[i] = s * inv_sqrt_d + (i < n_win ? 0.0 : log((double)C));
                if (logit[i] > lmax) lmax = logit[i];
            }
            double den = 0.0;
            for (long i = 0; i < count; ++i) {
                p[i] = exp(logit[i] - lmax);
                den += p[i];
            }
            for (long i = 0; i < count; ++i) p[i] /= den;
            for (int e = 0; e < d; ++e) {
                double acc = 0.0;
                for (long i = 0; i < count; ++i) {
                    const double* val = i < n_win ? V + (size_t)(lo + i) * d : Vs + (size_t)sidx[i - n_win] * d;
                    acc += p[i] * val[e];
                }
                o[e] = acc;
            }
            double Dabs = 0.0;
            for (int e = 0; e < d; ++e) Dabs += fabs(g[e] * o[e]);
            for (int e = 0; e < d; ++e) tq[e] = 0.0;
            for (long i = 0; i < count; ++i) {
                const int win = i < n_win;
                const double* key = win ? K + (size_t)(lo + i) * d : Ks + (size_t)sidx[i - n_win] * d;
                const double* val = win ? V + (size_t)(lo + i) * d : Vs + (size_t)sidx[i - n_win] * d;
                double* tkey = win ? Tk + (size_t)(lo + i) * d : Tks + (size_t)sidx[i - n_win] * d;
                double* tval = win ? Tv + (size_t)(lo + i) * d : Tvs + (size_t)sidx[i - n_win] * d;
                double gva = 0.0;
                for (int e = 0; e < d; ++e) gva += fabs(g[e] * val[e]);
                /* the logit gradient p_i (dO.v_i - D), D = dO.o, is a sum of
                 * the terms of both dot products */
                const double dl = p[i] * (gva + Dabs);
                for (int e = 0; e < d; ++e) {
                    tq[e] += dl * fabs(key[e]) * inv_sqrt_d;
                    tkey[e] += dl * fabs(q[e]) * inv_sqrt_d;
                    tval[e] += p[i] * fabs(g[e]);
                }
            }
        }
    }
    /* through the summaries, magnitudes of dvhat (Tvs) and dkhat's direct
     * part (Tks) standing for those sums */
    double* a = (double*)malloc((size_t)C * sizeof(double));
    double* b = (double*)malloc((size_t)C * sizeof(double));
    double* tkh = (double*)malloc((size_t)d * sizeof(double));
    for (long c = 0; c < n_chunks; ++c) {
        const double* Kc = K + (size_t)c * C * d;
        const double* Vc = V + (size_t)c * C * d;
        const double* kh = Ks + (size_t)c * d;
        const double* vh = Vs + (size_t)c * d;
        const double* tgk = Tks + (size_t)c * d;
        const double* tgv = Tvs + (size_t)c * d;
        double amax = -INFINITY;
        for (long j = 0; j < C; ++j) {
            double s = 0.0;
            for (int e = 0; e < d; ++e) s += kh[e] * Kc[(size_t)j * d + e];
            a[j] = s * inv_sqrt_d;
            if (a[j] > amax) amax = a[j];
        }
        double den = 0.0;
        for (long j = 0; j < C; ++j) {
            b[j] = exp(a[j] - amax);
            den += b[j];
        }
        for (long j = 0; j < C; ++j) b[j] /= den;
        double tgv_vh = 0.0;
        for (int e = 0; e < d; ++e) tgv_vh += tgv[e] * fabs(vh[e]);
        for (int e = 0; e < d; ++e) tkh[e] = tgk[e];
        for (long j = 0; j < C; ++j) {
            double tgv_v = 0.0;
            for (int e = 0; e < d; ++e) tgv_v += tgv[e] * fabs(Vc[(size_t)j * d + e]);
            const double tda = b[j] * (tgv_v + tgv_vh);
            for (int e = 0; e < d; ++e) {
                Tv[((size_t)c * C + j) * d + e] += b[j] * tgv[e];
                tkh[e] += tda * fabs(Kc[(size_t)j * d + e]) * inv_sqrt_d;
                Tk[((size_t)c * C + j) * d + e] += tda * fabs(kh[e]) * inv_sqrt_d;
            }
        }
        for (long j = 0; j < C; ++j)
            for (int e = 0; e < d; ++e) Tk[((size_t)c * C + j) * d + e] += tkh[e] / (double)C;
    }
    free(a);
    free(b);
    free(tkh);
    free(sidx);
    free(logit);
    free(p);
    free(o);
    free(Ks);
    free(Vs);
    free(Tks);
    free(Tvs);
}

/* The sliding window (variant 0). */
void eva_ref_backward_terms(const double* Q, const double* K, const double* V, const double* dO,
                            int G, long L, int d, long W, long C,
                            double* Tq, double* Tk, double* Tv)
{
    eva_ref_backward_terms_variant(Q, K, V, dO, G, L, d, W, C, 0, Tq, Tk, Tv);
}

int eva_ref_num_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads the parallel loops use from now on (timing of a single-thread
 * slice); n < 1 is ignored. */
void eva_ref_set_num_threads(int n)
{
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
