/*
 * kvr_oracle.c -- plain, slow CPU oracle for the KV-Rescue candidate-decode
 * hot path (arxiv 2608.15797).
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may link, load or call
 * this file; only the tests, the smoke check and the benchmark's CPU-baseline
 * leg do. It shares no code, header or constant with the HIP library.
 *
 * Everything is computed in double precision from the exact stored input
 * values (bf16 inputs are widened bit-exactly). Loops are written in the most
 * direct order; the only parallelism is an OpenMP loop over independent
 * (sequence, layer, kv-head) units, which does not change any result.
 *
 * Layouts (row-major, innermost last):
 *   cache K,V   [S][L][Hkv][cap][D]        pos [S][L][Hkv][cap] (int32)
 *   prefix K,V  [P][L][Hkv][plen][D]       sequence s uses prefix s / (S/P)
 *   q           [S][L][Hq][D]
 *   out         [S][L][Hq][D]  (double)
 *   psum        [S][L][Hkv][cap] (double)
 * Query head qh reads KV head qh / G with G = Hq / Hkv (grouped-query
 * attention: consecutive query heads share one KV head).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_F32 0
#define ORC_BF16 1

/* Exact value of element i of a float32 or bfloat16 array. A bfloat16 is the
 * top 16 bits of a float32, so widening is a 16-bit left shift. */
static double elem(const void *base, int dtype, size_t i) {
    if (dtype == ORC_F32) return (double)((const float *)base)[i];
    uint32_t u = (uint32_t)((const uint16_t *)base)[i] << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static size_t esize(int dtype) { return dtype == ORC_F32 ? 4 : 2; }

/*
 * Attention of one query row over a list of keys/values, Eq. (1) third line:
 * a = Attn(q, C) = sum_j p_j v_j with p = softmax_j(scale * <q, k_j>).
 * Keys come from up to two segments (a shared prefix, then the sequence's own
 * cache). p_out receives the probabilities of the second segment's n2 keys.
 */
static void attend_row(const void *q, size_t q_off, int dtype, int D, double scale,
                       const void *K1, const void *V1, size_t off1, int n1,
                       const void *K2, const void *V2, size_t off2, int n2,
                       double *o, double *p_out) {
    int n = n1 + n2;
    double *x = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    for (int j = 0; j < n; j++) {
        const void *Kb = j < n1 ? K1 : K2;
        size_t base = j < n1 ? off1 + (size_t)j * D : off2 + (size_t)(j - n1) * D;
        double dot = 0.0;
        for (int d = 0; d < D; d++) dot += elem(q, dtype, q_off + d) * elem(Kb, dtype, base + d);
        x[j] = scale * dot;
    }
    double m = -INFINITY;
    for (int j = 0; j < n; j++) if (x[j] > m) m = x[j];
    double Z = 0.0;
    for (int j = 0; j < n; j++) Z += exp(x[j] - m);
    for (int d = 0; d < D; d++) o[d] = 0.0;
    for (int j = 0; j < n; j++) {
        double p = exp(x[j] - m) / Z;
        const void *Vb = j < n1 ? V1 : V2;
        size_t base = j < n1 ? off1 + (size_t)j * D : off2 + (size_t)(j - n1) * D;
        for (int d = 0; d < D; d++) o[d] += p * elem(Vb, dtype, base + d);
        if (j >= n1 && p_out) p_out[j - n1] = p;
    }
    free(x);
}

/*
 * Decode attention for a batch of candidate sequences (Eq. (1): attention of
 * the current query over the kept cache; Eq. (3): the N candidates of a step
 * decode together). n[s] is the number of live cache entries of sequence s,
 * including the token just appended. With a prefix (P > 0) each query also
 * attends over plen shared prefix entries before its own cache entries.
 * psum (optional) receives, per KV head, the sum over its G query heads of the
 * probability each cache entry received: the per-step attention mass that the
 * accumulated-attention importance score of Section 2.1 adds up.
 */
int orc_decode_attn(const void *K, const void *V, int dtype, int S, int L, int Hkv,
                    int cap, int D, const void *PK, const void *PV, int P, int plen,
                    const int32_t *n, const void *q, int Hq, double scale,
                    double *out, double *psum) {
    if (Hkv <= 0 || Hq % Hkv != 0 || (P > 0 && S % P != 0)) return -1;
    int G = Hq / Hkv;
    long units = (long)S * L * Hkv;
#pragma omp parallel for schedule(dynamic)
    for (long u = 0; u < units; u++) {
        int s = (int)(u / ((long)L * Hkv));
        int l = (int)((u / Hkv) % L);
        int h = (int)(u % Hkv);
        int ns = n[s];
        size_t coff = (((size_t)s * L + l) * Hkv + h) * (size_t)cap * D;
        size_t poff = 0;
        int n1 = 0;
        if (P > 0) {
            int p = s / (S / P);
            poff = (((size_t)p * L + l) * Hkv + h) * (size_t)plen * D;
            n1 = plen;
        }
        double *ps = psum ? psum + (((size_t)s * L + l) * Hkv + h) * (size_t)cap : NULL;
        double *prow = (double *)malloc(sizeof(double) * (size_t)(ns > 0 ? ns : 1));
        if (ps) for (int j = 0; j < cap; j++) ps[j] = 0.0;
        for (int g = 0; g < G; g++) {
            int qh = h * G + g;
            size_t qoff = (((size_t)s * L + l) * Hq + qh) * (size_t)D;
            double *o = out + qoff;
            attend_row(q, qoff, dtype, D, scale, PK, PV, poff, n1, K, V, coff, ns, o, prow);
            if (ps) for (int j = 0; j < ns; j++) ps[j] += prow[j];
        }
        free(prow);
    }
    return 0;
}

/*
 * Window re-computation of the importance score: queries q_win[S][L][Hq][nq][D]
 * are the last nq tokens of each sequence; window row r sees the first
 * n[s] - (nq-1-r) cache entries (causal). For every cache entry the score is
 * the attention mass it received, summed over the window rows and over the G
 * query heads of its KV head (accumulated attention, Section 2.1). scores is
 * [S][L][Hkv][cap]; entries at or beyond n[s] are set to 0.
 */
int orc_window_scores(const void *K, const void *V, int dtype, int S, int L, int Hkv,
                      int cap, int D, const int32_t *n, const void *q_win, int Hq, int nq,
                      double scale, double *scores) {
    if (Hkv <= 0 || Hq % Hkv != 0) return -1;
    int G = Hq / Hkv;
    long units = (long)S * L * Hkv;
#pragma omp parallel for schedule(dynamic)
    for (long u = 0; u < units; u++) {
        int s = (int)(u / ((long)L * Hkv));
        int l = (int)((u / Hkv) % L);
        int h = (int)(u % Hkv);
        size_t coff = (((size_t)s * L + l) * Hkv + h) * (size_t)cap * D;
        double *sc = scores + (((size_t)s * L + l) * Hkv + h) * (size_t)cap;
        for (int j = 0; j < cap; j++) sc[j] = 0.0;
        double *o = (double *)malloc(sizeof(double) * (size_t)D);
        double *prow = (double *)malloc(sizeof(double) * (size_t)(n[s] > 0 ? n[s] : 1));
        for (int r = 0; r < nq; r++) {
            int nr = n[s] - (nq - 1 - r);
            if (nr <= 0) continue;
            for (int g = 0; g < G; g++) {
                int qh = h * G + g;
                size_t qoff = ((((size_t)s * L + l) * Hq + qh) * (size_t)nq + r) * (size_t)D;
                attend_row(q_win, qoff, dtype, D, scale, NULL, NULL, 0, 0, K, V, coff, nr, o, prow);
                for (int j = 0; j < nr; j++) sc[j] += prow[j];
            }
        }
        free(o);
        free(prow);
    }
    return 0;
}

/*
 * TopB of Eq. (1) with a protected recent window: of the n live entries the W
 * newest are always kept; among the other n-W the B-W with the largest score
 * are kept, ties going to the lower slot. kept[0..B) receives the kept slot
 * ids in ascending order (so the window's slots n-W..n-1 come last).
 * Selection is done the plain way: B-W rounds, each taking the best slot not
 * yet taken.
 */
int orc_select_topb(const double *score, int n, int B, int W, int32_t *kept) {
    if (W < 0 || W > B || n < B || B <= 0) return -1;
    int ncand = n - W, take = B - W;
    char *taken = (char *)calloc((size_t)(ncand > 0 ? ncand : 1), 1);
    int cnt = 0;
    for (int k = 0; k < take; k++) {
        int best = -1;
        for (int j = 0; j < ncand; j++) {
            if (taken[j]) continue;
            if (best < 0 || score[j] > score[best]) best = j;
        }
        taken[best] = 1;
    }
    for (int j = 0; j < ncand; j++) if (taken[j]) kept[cnt++] = j;
    for (int j = ncand; j < n; j++) kept[cnt++] = j;
    free(taken);
    return cnt == B ? 0 : -2;
}

/*
 * The evicted cache C_t^B of Eq. (1): rows kept[0..B) of one head's K, V and
 * pos, moved to slots 0..B-1 in order. kept must be strictly ascending, so
 * kept[i] >= i and copying in increasing i never overwrites a row still to
 * be read.
 */
int orc_compact_head(void *K, void *V, int32_t *pos, int dtype, int D,
                     const int32_t *kept, int B) {
    size_t row = esize(dtype) * (size_t)D;
    for (int i = 0; i < B; i++) {
        int src = kept[i];
        if (i > 0 && src <= kept[i - 1]) return -1;
        if (src == i) continue;
        memmove((char *)K + (size_t)i * row, (char *)K + (size_t)src * row, row);
        memmove((char *)V + (size_t)i * row, (char *)V + (size_t)src * row, row);
        if (pos) pos[i] = pos[src];
    }
    return 0;
}

/*
 * Token entropy H_e of Eq. (4): H = -sum_v p(v) log p(v) with
 * p = softmax(inv_temp * logits). Entries with p(v) = 0 contribute 0.
 * logits is [R][ld] (float32 or bfloat16), only the first V columns are used.
 */
int orc_entropy(const void *logits, int dtype, int R, int V, long ld, double inv_temp,
                double *H) {
    if (V <= 0 || ld < V) return -1;
#pragma omp parallel for schedule(dynamic)
    for (int r = 0; r < R; r++) {
        size_t base = (size_t)r * (size_t)ld;
        double m = -INFINITY;
        for (int v = 0; v < V; v++) {
            double y = inv_temp * elem(logits, dtype, base + v);
            if (y > m) m = y;
        }
        double Z = 0.0;
        for (int v = 0; v < V; v++) Z += exp(inv_temp * elem(logits, dtype, base + v) - m);
        double h = 0.0;
        for (int v = 0; v < V; v++) {
            double p = exp(inv_temp * elem(logits, dtype, base + v) - m) / Z;
            if (p > 0.0) h -= p * log(p);
        }
        H[r] = h;
    }
    return 0;
}

/*
 * One position of the online entropy detector (Eq. (4) moving average and the
 * implementation-details constants): push H[r] into row r's history of the
 * last `window` entropies; once the candidate has produced at least `guard`
 * tokens, it is flagged when the mean of that history exceeds tau. The flag is
 * sticky: a candidate is degenerate once any position fired (deg(s) is the OR
 * over positions). hist is [R][window] in push order modulo window.
 */
int orc_detector_step(const double *H, int R, double *hist, int32_t *cnt, uint8_t *flag,
                      int window, int guard, double tau) {
    if (window <= 0) return -1;
    for (int r = 0; r < R; r++) {
        hist[(size_t)r * window + (cnt[r] % window)] = H[r];
        cnt[r] += 1;
        if (cnt[r] >= guard) {
            int k = cnt[r] < window ? cnt[r] : window;
            double sum = 0.0;
            for (int i = 0; i < k; i++) sum += hist[(size_t)r * window + i];
            if (sum / k > tau) flag[r] = 1;
        }
    }
    return 0;
}
