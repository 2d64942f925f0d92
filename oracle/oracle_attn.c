/*
 * Oracle for exact softmax attention -- TEST INFRASTRUCTURE ONLY.
 *
 * Only tests, the package smoke check and the CPU-baseline leg of the
 * benchmark may load this library.  The product path (the HIP library) never
 * links, imports or calls it, and this file includes nothing from the product.
 *
 * What it computes (plain definition, fp64, straight loops, no blocking):
 *   The paper evaluates Flash Attention and Flash Decode (Evaluation,
 *   Experimental Setup): scores from a product of queries and keys, a
 *   softmax over the allowed keys, then a weighted sum of value rows; Flash
 *   Decode is the same with one query per head, bound by reading the cached
 *   keys and values.  The paper never writes the formula; the textbook one is
 *       s_ij = scale * sum_c q[i][c] k[j][c]        (matrix multiplication)
 *       P_ij = exp(s_ij) / sum_{j' in A_i} exp(s_ij') (softmax over allowed keys)
 *       o[i][c] = sum_{j in A_i} P_ij v[j][c]        (value aggregation)
 *   with A_i = all keys (non-causal) or {j : j <= i + Skv - Sq} (causal,
 *   bottom-right aligned -- a reading: the paper evaluates non-causal only).
 *   The max is subtracted before exp; that changes rounding only, not the
 *   exact value.
 *
 *   Variants (beyond the paper's evaluation):
 *   grouped-query heads -- query head h of Hq reads key/value head
 *   h / (Hq / Hkv) of Hkv -- and the log-sum-exp of each row's scores,
 *       lse_i = log sum_{j in A_i} exp(s_ij)  (natural log),
 *   so that P_ij = exp(s_ij - lse_i).
 *
 *   oracle_decode_split follows the paper's decomposition of Flash Decode in
 *   the latency-modelling section (HEG paragraph): a local softmax loop over
 *   each chunk of the sequence axis, then gathering the partial results, a
 *   global softmax over them, and the final output.
 *
 * Inputs are bf16 bit patterns (uint16) widened exactly to fp64 (bits << 16
 * is the fp32 value; fp32 -> fp64 is exact).  Layout: contiguous
 * [B][H][S][d] for q/k/v/o (decode: q and o are [B][H][d]).
 *
 * Parity status: every function here is pinned by tests under tests/
 * (closed forms, invariants, library routines, hand-derived fixtures).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double widen_bf16(uint16_t bits) {
    uint32_t u = ((uint32_t)bits) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Largest allowed key index (inclusive) for query row i, or Skv-1. */
static int64_t last_key(int64_t i, int64_t Sq, int64_t Skv, int causal) {
    if (!causal) return Skv - 1;
    int64_t lim = i + (Skv - Sq);
    return lim < Skv - 1 ? lim : Skv - 1;
}

/*
 * One output row: o_row[c] = sum_j softmax_j(s) v[j][c] over keys
 * j in [0, jmax].  Optionally also writes the probabilities P_ij to p_row
 * (length Skv, zero for keys outside the allowed set).
 */
static void attend_row(const uint16_t* qrow, const uint16_t* kslab,
                       const uint16_t* vslab, int64_t jmax, int64_t Skv,
                       int64_t d, double scale, double* s, double* acc,
                       double* o_row, double* p_row, double* lse) {
    /* matrix multiplication: scores of the allowed keys */
    double m = -INFINITY;
    for (int64_t j = 0; j <= jmax; ++j) {
        double dot = 0.0;
        for (int64_t c = 0; c < d; ++c)
            dot += widen_bf16(qrow[c]) * widen_bf16(kslab[j * d + c]);
        s[j] = scale * dot;
        if (s[j] > m) m = s[j];
    }
    /* softmax: exponentials and their sum */
    double l = 0.0;
    for (int64_t j = 0; j <= jmax; ++j) {
        s[j] = exp(s[j] - m);
        l += s[j];
    }
    /* value aggregation */
    for (int64_t c = 0; c < d; ++c) acc[c] = 0.0;
    for (int64_t j = 0; j <= jmax; ++j) {
        double w = s[j];
        for (int64_t c = 0; c < d; ++c) acc[c] += w * widen_bf16(vslab[j * d + c]);
    }
    for (int64_t c = 0; c < d; ++c) o_row[c] = acc[c] / l;
    /* log-sum-exp: the stabiliser plus the log of the sum */
    if (lse) *lse = m + log(l);
    if (p_row) {
        for (int64_t j = 0; j < Skv; ++j) p_row[j] = (j <= jmax) ? s[j] / l : 0.0;
    }
}

static int check_dims(int B, int H, int Sq, int Skv, int d, int causal) {
    if (B <= 0 || H <= 0 || Sq <= 0 || Skv <= 0 || d <= 0) return -1;
    if (causal && Sq > Skv) return -2; /* rows with no allowed key */
    return 0;
}

/* Query head h of Hq reads key/value head h / (Hq / Hkv). */
static int check_heads(int Hq, int Hkv) {
    if (Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0) return -1;
    return 0;
}

static int attend_all(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                      double* o, double* p, double* lse, int B, int Hq, int Hkv, int Sq,
                      int Skv, int d, float scale, int causal) {
    int rc = check_dims(B, Hq, Sq, Skv, d, causal);
    if (!rc) rc = check_heads(Hq, Hkv);
    if (rc) return rc;
    const int64_t rows = (int64_t)B * Hq * Sq;
    const int64_t group = Hq / Hkv;
    const double sc = (double)scale;
    int failed = 0;
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)Skv);
        double* acc = (double*)malloc(sizeof(double) * (size_t)d);
        if (!s || !acc) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(dynamic, 4)
        for (int64_t r = 0; r < rows; ++r) {
            if (!s || !acc) continue;
            const int64_t bh = r / Sq, i = r % Sq;
            const int64_t b = bh / Hq, h = bh % Hq;
            const int64_t kvh = b * Hkv + h / group; /* shared key/value head */
            const uint16_t* qrow = q + r * d;
            const uint16_t* kslab = k + kvh * (int64_t)Skv * d;
            const uint16_t* vslab = v + kvh * (int64_t)Skv * d;
            attend_row(qrow, kslab, vslab, last_key(i, Sq, Skv, causal), Skv, d, sc,
                       s, acc, o + r * d, p ? p + r * (int64_t)Skv : NULL,
                       lse ? lse + r : NULL);
        }
        free(s);
        free(acc);
    }
    return failed ? -4 : 0;
}

/* o: fp64 [B][H][Sq][d].  Returns 0, -1 (bad dims), -2 (causal, Sq > Skv). */
int oracle_attn(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                double* o, int B, int H, int Sq, int Skv, int d, float scale,
                int causal) {
    return attend_all(q, k, v, o, NULL, NULL, B, H, H, Sq, Skv, d, scale, causal);
}

/* As oracle_attn, and also the probabilities p: fp64 [B][H][Sq][Skv]. */
int oracle_attn_probs(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                      double* o, double* p, int B, int H, int Sq, int Skv,
                      int d, float scale, int causal) {
    return attend_all(q, k, v, o, p, NULL, B, H, H, Sq, Skv, d, scale, causal);
}

/*
 * Grouped-query heads and the log-sum-exp: q, o [B][Hq][Sq][d]; k, v
 * [B][Hkv][Skv][d] with Hkv dividing Hq; lse (may be NULL) [B][Hq][Sq].
 * Returns 0, -1 (bad dims or heads), -2 (causal, Sq > Skv).
 */
int oracle_attn_gqa(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                    double* o, double* lse, int B, int Hq, int Hkv, int Sq, int Skv,
                    int d, float scale, int causal) {
    return attend_all(q, k, v, o, NULL, lse, B, Hq, Hkv, Sq, Skv, d, scale, causal);
}

/*
 * Output rows for a subset of query rows only (for sampled checks at full
 * size).  rows[r] is a flat row index into [B][H][Sq]; o is [nrows][d].
 */
int oracle_attn_rows(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                     double* o, const int64_t* rows, int64_t nrows, int B, int H,
                     int Sq, int Skv, int d, float scale, int causal) {
    int rc = check_dims(B, H, Sq, Skv, d, causal);
    if (rc) return rc;
    const int64_t total = (int64_t)B * H * Sq;
    for (int64_t n = 0; n < nrows; ++n)
        if (rows[n] < 0 || rows[n] >= total) return -1;
    const double sc = (double)scale;
    int failed = 0;
#pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)Skv);
        double* acc = (double*)malloc(sizeof(double) * (size_t)d);
        if (!s || !acc) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(dynamic, 1)
        for (int64_t n = 0; n < nrows; ++n) {
            if (!s || !acc) continue;
            const int64_t r = rows[n], bh = r / Sq, i = r % Sq;
            attend_row(q + r * d, k + bh * (int64_t)Skv * d, v + bh * (int64_t)Skv * d,
                       last_key(i, Sq, Skv, causal), Skv, d, sc, s, acc, o + n * d, NULL,
                       NULL);
        }
        free(s);
        free(acc);
    }
    return failed ? -4 : 0;
}

/*
 * Flash-Decode by the paper's decomposition (one query per (b, h)):
 *   chunk = ceil(Skv / n_splits); split t covers keys [t*chunk, (t+1)*chunk)
 *   clipped to Skv (empty splits are skipped).
 *   local softmax loop:  m_t = max s_j,  l_t = sum exp(s_j - m_t),
 *                        u_t[c] = sum exp(s_j - m_t) v[j][c]
 *   gather + global softmax:  M = max_t m_t,  w_t = exp(m_t - M)
 *   final:  o[c] = sum_t w_t u_t[c] / sum_t w_t l_t
 * q, o: [B][H][d]; k, v: [B][H][Skv][d].  The partials are optionally
 * returned: part_m/part_l [B][H][n_splits], part_u [B][H][n_splits][d]
 * (splits beyond the effective count are left untouched).
 */
int oracle_decode_split(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                        double* o, int B, int H, int Skv, int d, float scale,
                        int n_splits, double* part_m, double* part_l,
                        double* part_u) {
    int rc = check_dims(B, H, 1, Skv, d, 0);
    if (rc) return rc;
    if (n_splits <= 0) return -1;
    const int64_t stride = n_splits; /* row length of the partial arrays */
    if (n_splits > Skv) n_splits = Skv;
    const int64_t chunk = ((int64_t)Skv + n_splits - 1) / n_splits;
    const int64_t eff = ((int64_t)Skv + chunk - 1) / chunk;
    const int64_t BH = (int64_t)B * H;
    const double sc = (double)scale;
    int failed = 0;
#pragma omp parallel
    {
        double* m = (double*)malloc(sizeof(double) * (size_t)eff);
        double* l = (double*)malloc(sizeof(double) * (size_t)eff);
        double* u = (double*)malloc(sizeof(double) * (size_t)(eff * d));
        double* s = (double*)malloc(sizeof(double) * (size_t)chunk);
        if (!m || !l || !u || !s) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(dynamic, 1)
        for (int64_t bh = 0; bh < BH; ++bh) {
            if (!m || !l || !u || !s) continue;
            const uint16_t* qrow = q + bh * d;
            const uint16_t* kslab = k + bh * (int64_t)Skv * d;
            const uint16_t* vslab = v + bh * (int64_t)Skv * d;
            /* local softmax loop per split */
            for (int64_t t = 0; t < eff; ++t) {
                const int64_t j0 = t * chunk;
                const int64_t j1 = (j0 + chunk < Skv) ? j0 + chunk : Skv;
                double mt = -INFINITY;
                for (int64_t j = j0; j < j1; ++j) {
                    double dot = 0.0;
                    for (int64_t c = 0; c < d; ++c)
                        dot += widen_bf16(qrow[c]) * widen_bf16(kslab[j * d + c]);
                    s[j - j0] = sc * dot;
                    if (s[j - j0] > mt) mt = s[j - j0];
                }
                double lt = 0.0;
                double* ut = u + t * d;
                for (int64_t c = 0; c < d; ++c) ut[c] = 0.0;
                for (int64_t j = j0; j < j1; ++j) {
                    double e = exp(s[j - j0] - mt);
                    lt += e;
                    for (int64_t c = 0; c < d; ++c) ut[c] += e * widen_bf16(vslab[j * d + c]);
                }
                m[t] = mt;
                l[t] = lt;
                if (part_m) part_m[bh * stride + t] = mt;
                if (part_l) part_l[bh * stride + t] = lt;
                if (part_u)
                    for (int64_t c = 0; c < d; ++c) part_u[(bh * stride + t) * d + c] = ut[c];
            }
            /* gather partials and take the global softmax over them */
            double M = -INFINITY;
            for (int64_t t = 0; t < eff; ++t)
                if (m[t] > M) M = m[t];
            double L = 0.0;
            for (int64_t t = 0; t < eff; ++t) L += exp(m[t] - M) * l[t];
            /* final output */
            for (int64_t c = 0; c < d; ++c) {
                double num = 0.0;
                for (int64_t t = 0; t < eff; ++t) num += exp(m[t] - M) * u[t * d + c];
                o[bh * d + c] = num / L;
            }
        }
        free(m);
        free(l);
        free(u);
        free(s);
    }
    return failed ? -4 : 0;
}

/*
 * Matrix multiplication, the paper's third workload (Evaluation, GEMM
 * paragraph), as its plain definition in fp64
 * over bf16 inputs:
 *     c[m][n] = sum_{k < K} a[m][k] * b(k, n)
 * a: [M][K]; b: [K][N] with b(k, n) = b[k][n] (b_nk = 0), or [N][K] with
 * b(k, n) = b[n][k] (b_nk = 1).  rows: NULL for every output row (c is
 * [M][N]), else nrows row indices (c is [nrows][N]).  absc, if not NULL,
 * receives sum_k |a[m][k] * b(k, n)| in the same layout (the scale of the
 * rounding error of any summation order).  Products of two widened bf16
 * values are exact in fp64; only the sum rounds.
 */
int oracle_gemm(const uint16_t* a, const uint16_t* b, double* c, double* absc, int M, int N,
                int K, int b_nk, const int64_t* rows, int64_t nrows) {
    if (M <= 0 || N <= 0 || K <= 0 || (b_nk != 0 && b_nk != 1)) return -1;
    const int64_t n_out = rows ? nrows : (int64_t)M;
    if (rows)
        for (int64_t i = 0; i < nrows; ++i)
            if (rows[i] < 0 || rows[i] >= M) return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < n_out; ++i) {
        const int64_t m = rows ? rows[i] : i;
        const uint16_t* arow = a + m * (int64_t)K;
        for (int n = 0; n < N; ++n) {
            double sum = 0.0, mag = 0.0;
            for (int k = 0; k < K; ++k) {
                const uint16_t bk = b_nk ? b[(int64_t)n * K + k] : b[(int64_t)k * N + n];
                const double p = widen_bf16(arow[k]) * widen_bf16(bk);
                sum += p;
                mag += fabs(p);
            }
            c[i * N + n] = sum;
            if (absc) absc[i * N + n] = mag;
        }
    }
    return 0;
}
