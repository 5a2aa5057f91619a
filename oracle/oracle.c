/*
 * oracle.c -- plain, slow CPU reference for the SparseSpec-L decode hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  The product path never
 * calls it, and it shares no code with the HIP library.
 *
 * Everything is computed in double precision straight from the definitions in
 * "A Sparse Glimpse of the Whole: Train-Free Self-Speculative Decoding":
 *
 *   verify   Sec. 3.1 (full verification as one dense attention pass that
 *            materializes the attention weights) and Sec. 3.2 Eq. 3 (per-head
 *            importance = attention mass received from the last W queries);
 *   select   Sec. 3.2 Eq. 4 (sink + top-K_mid of the remaining span + recent);
 *   draft    Sec. 3.2 Eq. 5 (attention over the gathered K/V rows), and one
 *            step of a draft round (Sec. 3.1) over that view with its recent
 *            window slid to the newest drafted token;
 *   control  Sec. 3.3 Eq. 6 (entropy EMAs), Eq. 7 (soft acceptance
 *            probability), Eq. 8 (speculation length maximizing expected
 *            tokens per unit cost).
 *
 * Readings of points the paper leaves open (all documented with the tests):
 *   - scores are kept per KV head and summed over the query heads sharing it;
 *   - the window is the last min(W, q) rows of the verify block, rejected
 *     drafts included;
 *   - the verify block is causal, bottom-right aligned: row j of q rows sees
 *     keys 0 .. T-q+j;
 *   - positions are 0-based; sink = [0, min(K_sink,T)), recent =
 *     [max(T-K_recent, sink end), T), the middle span is what lies between;
 *   - top-K ties go to the lower position; output is sorted ascending.
 *
 * Inputs are bf16 bit patterns (uint16) widened exactly to double.
 * Layouts:
 *   q       [batch][max_q][Hq][d]      verify queries
 *   k, v    [batch][Hkv][max_ctx][d]   dense cache, head-major
 *   out     [batch][max_q][Hq][d]      double
 *   scores  [batch][Hkv][max_ctx]      double
 *   idx     [batch][Hkv][budget]       int32
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double widen_bf16(uint16_t h)
{
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/*
 * Verification attention with importance-score emission.
 *
 * For sequence b with T = ctx_len[b] cached tokens (the q = q_len[b] verify
 * tokens included), verify row j (0 <= j < q) sits at position p = T - q + j.
 * For query head h and its KV head c = h / (Hq/Hkv):
 *     x_i = sm_scale * <q[b,j,h], k[b,c,i]>          for 0 <= i <= p
 *     P_i = exp(x_i - max x) / sum_t exp(x_t - max x)
 *     out[b,j,h] = sum_i P_i v[b,c,i]
 *     scores[b,c,i] += P_i   when j is among the last min(W, q) rows.
 * Entries of scores beyond T are left untouched; entries below T start at 0.
 *
 * units: optional list of (b * Hkv + c) to compute (NULL: all); lets tests
 * evaluate a sample of a large workload.  Returns 0, or -1 on bad arguments.
 */
int oracle_verify(int batch, int n_q_heads, int n_kv_heads, int head_dim,
                  int max_ctx, int max_q,
                  const int32_t *ctx_len, const int32_t *q_len,
                  const uint16_t *q, const uint16_t *k, const uint16_t *v,
                  double sm_scale, int window,
                  const int32_t *units, int n_units,
                  double *out, double *scores)
{
    if (batch < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads != 0 || head_dim < 1 ||
        window < 1)
        return -1;
    for (int b = 0; b < batch; ++b)
        if (q_len[b] < 1 || q_len[b] > max_q || ctx_len[b] < q_len[b] || ctx_len[b] > max_ctx)
            return -1;
    const int g = n_q_heads / n_kv_heads;
    const int d = head_dim;
    const int total = units ? n_units : batch * n_kv_heads;

#pragma omp parallel for schedule(dynamic, 1)
    for (int u = 0; u < total; ++u) {
        const int unit = units ? units[u] : u;
        const int b = unit / n_kv_heads;
        const int c = unit % n_kv_heads;
        const int T = ctx_len[b];
        const int nq = q_len[b];
        const int w = window < nq ? window : nq;
        double *S = scores + ((size_t)b * n_kv_heads + c) * max_ctx;
        const uint16_t *kc = k + ((size_t)b * n_kv_heads + c) * max_ctx * d;
        const uint16_t *vc = v + ((size_t)b * n_kv_heads + c) * max_ctx * d;
        double *x = (double *)malloc(sizeof(double) * (size_t)T);
        double *qrow = (double *)malloc(sizeof(double) * (size_t)d);
        for (int i = 0; i < T; ++i) S[i] = 0.0;

        for (int j = 0; j < nq; ++j) {
            const int p = T - nq + j;               /* last visible key */
            const int in_window = (j >= nq - w);
            for (int hh = 0; hh < g; ++hh) {
                const int h = c * g + hh;
                const uint16_t *qs = q + (((size_t)b * max_q + j) * n_q_heads + h) * d;
                for (int e = 0; e < d; ++e) qrow[e] = widen_bf16(qs[e]);

                double m = -INFINITY;
                for (int i = 0; i <= p; ++i) {
                    double dot = 0.0;
                    for (int e = 0; e < d; ++e) dot += qrow[e] * widen_bf16(kc[(size_t)i * d + e]);
                    x[i] = sm_scale * dot;
                    if (x[i] > m) m = x[i];
                }
                double L = 0.0;
                for (int i = 0; i <= p; ++i) {
                    x[i] = exp(x[i] - m);
                    L += x[i];
                }
                double *o = out + (((size_t)b * max_q + j) * n_q_heads + h) * d;
                for (int e = 0; e < d; ++e) o[e] = 0.0;
                for (int i = 0; i <= p; ++i) {
                    const double P = x[i] / L;
                    for (int e = 0; e < d; ++e) o[e] += P * widen_bf16(vc[(size_t)i * d + e]);
                    if (in_window) S[i] += P;
                }
            }
        }
        free(x);
        free(qrow);
    }
    return 0;
}

/* Candidate for the top-K ranking: higher score first, lower position on ties. */
typedef struct { double s; int32_t i; } cand_t;

static int cand_cmp(const void *pa, const void *pb)
{
    const cand_t *a = (const cand_t *)pa, *b = (const cand_t *)pb;
    if (a->s > b->s) return -1;
    if (a->s < b->s) return 1;
    return (a->i > b->i) - (a->i < b->i);
}

/* Number of indices Eq. 4 yields for T positions (same for every head). */
int oracle_index_count(int T, int k_sink, int k_recent, int budget)
{
    const int k_mid = budget - k_sink - k_recent;
    const int s_end = k_sink < T ? k_sink : T;
    const int r_start = (T - k_recent) > s_end ? (T - k_recent) : s_end;
    const int n_mid = r_start - s_end;
    return s_end + (k_mid < n_mid ? k_mid : n_mid) + (T - r_start);
}

/*
 * Recallable index construction (Eq. 4).  For each (b, c) with T = ctx_len[b]:
 *   sink    = [0, min(K_sink, T))
 *   recent  = [max(T - K_recent, end of sink), T)
 *   mid     = the positions in between
 *   TopK    = the min(K_mid, |mid|) mid positions of highest score,
 *             K_mid = budget - K_sink - K_recent
 * idx[b,c,:] = sink U TopK U recent in ascending order; n_idx[b] = its size.
 * Slots of idx past n_idx[b] are not written.  Returns 0 or -1.
 */
int oracle_select(int batch, int n_kv_heads, int max_ctx, const int32_t *ctx_len,
                  const double *scores, int k_sink, int k_recent, int budget,
                  int32_t *idx, int32_t *n_idx)
{
    if (batch < 1 || n_kv_heads < 1 || k_sink < 0 || k_recent < 0 || budget < 1 ||
        k_sink + k_recent > budget)
        return -1;
    for (int b = 0; b < batch; ++b)
        if (ctx_len[b] < 1 || ctx_len[b] > max_ctx) return -1;
    const int k_mid = budget - k_sink - k_recent;

#pragma omp parallel for schedule(dynamic, 1)
    for (int u = 0; u < batch * n_kv_heads; ++u) {
        const int b = u / n_kv_heads, c = u % n_kv_heads;
        const int T = ctx_len[b];
        const double *S = scores + ((size_t)b * n_kv_heads + c) * max_ctx;
        const int s_end = k_sink < T ? k_sink : T;
        const int r_start = (T - k_recent) > s_end ? (T - k_recent) : s_end;
        const int n_mid = r_start - s_end;
        const int take = k_mid < n_mid ? k_mid : n_mid;

        char *keep = (char *)calloc((size_t)T, 1);
        cand_t *cands = (cand_t *)malloc(sizeof(cand_t) * (size_t)(n_mid > 0 ? n_mid : 1));
        for (int t = 0; t < n_mid; ++t) {
            cands[t].s = S[s_end + t];
            cands[t].i = s_end + t;
        }
        qsort(cands, (size_t)n_mid, sizeof(cand_t), cand_cmp);
        for (int t = 0; t < take; ++t) keep[cands[t].i] = 1;
        for (int i = 0; i < s_end; ++i) keep[i] = 1;
        for (int i = r_start; i < T; ++i) keep[i] = 1;

        int32_t *out = idx + ((size_t)b * n_kv_heads + c) * budget;
        int n = 0;
        for (int i = 0; i < T; ++i)
            if (keep[i]) out[n++] = i;
        if (c == 0) n_idx[b] = n;
        free(keep);
        free(cands);
    }
    return 0;
}

/*
 * Draft attention over the gathered rows (Eq. 5): for sequence b, query head
 * h, KV head c = h / g, with the n = n_idx[b] indices I = idx[b,c,0..n):
 *     x_t = sm_scale * <q_draft[b,h], k[b,c,I_t]>,  P = softmax(x),
 *     out[b,h] = sum_t P_t v[b,c,I_t].
 * Layouts: q_draft / out [batch][Hq][d].  Returns 0 or -1.
 */
int oracle_draft(int batch, int n_q_heads, int n_kv_heads, int head_dim, int max_ctx,
                 int budget, const int32_t *n_idx, const uint16_t *q_draft,
                 const uint16_t *k, const uint16_t *v, const int32_t *idx,
                 double sm_scale, double *out)
{
    if (batch < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads != 0 || head_dim < 1)
        return -1;
    for (int b = 0; b < batch; ++b)
        if (n_idx[b] < 1 || n_idx[b] > budget) return -1;
    const int g = n_q_heads / n_kv_heads;
    const int d = head_dim;

#pragma omp parallel for schedule(dynamic, 1)
    for (int bh = 0; bh < batch * n_q_heads; ++bh) {
        const int b = bh / n_q_heads, h = bh % n_q_heads, c = h / g;
        const int n = n_idx[b];
        const int32_t *I = idx + ((size_t)b * n_kv_heads + c) * budget;
        const uint16_t *kc = k + ((size_t)b * n_kv_heads + c) * max_ctx * d;
        const uint16_t *vc = v + ((size_t)b * n_kv_heads + c) * max_ctx * d;
        const uint16_t *qs = q_draft + ((size_t)b * n_q_heads + h) * d;
        double *x = (double *)malloc(sizeof(double) * (size_t)n);
        double m = -INFINITY;
        for (int t = 0; t < n; ++t) {
            double dot = 0.0;
            for (int e = 0; e < d; ++e)
                dot += widen_bf16(qs[e]) * widen_bf16(kc[(size_t)I[t] * d + e]);
            x[t] = sm_scale * dot;
            if (x[t] > m) m = x[t];
        }
        double L = 0.0;
        for (int t = 0; t < n; ++t) {
            x[t] = exp(x[t] - m);
            L += x[t];
        }
        double *o = out + ((size_t)b * n_q_heads + h) * d;
        for (int e = 0; e < d; ++e) o[e] = 0.0;
        for (int t = 0; t < n; ++t) {
            const double P = x[t] / L;
            for (int e = 0; e < d; ++e) o[e] += P * widen_bf16(vc[(size_t)I[t] * d + e]);
        }
        free(x);
    }
    return 0;
}

/*
 * One step of a draft round.  Sec. 3.1: the target model drafts k tokens one
 * after another over the sparse view of Sec. 3.2 (Eq. 5).  The index set
 * I = idx[b,c,0..n), n = oracle_index_count(T, ...), was built by Eq. 4 at
 * T = base_len[b].  After i tokens have been drafted (cur = cur_len[b] = T + i,
 * their K/V rows already in the cache) the step attends over
 *     F = the entries of I below r_T = max(T - K_recent, min(K_sink, T)),
 *         i.e. the sink and TopK parts, fixed for the whole round;
 *     W = [max(r_T, cur - K_recent), cur), the recent window slid forward so
 *         that it ends at the newest token.
 * (Reading: the paper keeps the most recent tokens in the draft view but does
 * not say how that window moves while a round drafts; here it slides and the
 * budget stays n.)  Requires T <= cur <= T + K_recent, so that every drafted
 * token lies in W, and cur <= max_ctx.  With x_t = sm_scale <q[b,h], k[b,c,t]>
 * over t in F u W:  out[b,h] = sum_t softmax(x)_t v[b,c,t].
 * Layouts as oracle_draft.  Returns 0 or -1.
 */
static int draft_step_sets(int per_head, int batch, int n_q_heads, int n_kv_heads, int head_dim,
                           int max_ctx, int budget, int k_sink, int k_recent,
                           const int32_t *base_len, const int32_t *cur_len,
                           const uint16_t *q_draft, const uint16_t *k, const uint16_t *v,
                           const int32_t *idx, double sm_scale, double *out)
{
    if (batch < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads != 0 || head_dim < 1)
        return -1;
    if (budget < 1 || k_sink < 0 || k_recent < 0 || k_sink + k_recent > budget) return -1;
    for (int b = 0; b < batch; ++b) {
        const int T = base_len[b], cur = cur_len[b];
        if (T < 1 || cur < T || cur - T > k_recent || cur > max_ctx) return -1;
    }
    const int g = n_q_heads / n_kv_heads;
    const int d = head_dim;

#pragma omp parallel for schedule(dynamic, 1)
    for (int bh = 0; bh < batch * n_q_heads; ++bh) {
        const int b = bh / n_q_heads, h = bh % n_q_heads, c = h / g;
        const int T = base_len[b], cur = cur_len[b];
        const int n = oracle_index_count(T, k_sink, k_recent, budget);
        const int s_end = k_sink < T ? k_sink : T;
        const int r_T = (T - k_recent) > s_end ? (T - k_recent) : s_end;
        const int w0 = (cur - k_recent) > r_T ? (cur - k_recent) : r_T;
        /* the index set of head h: its own (per_head), else its KV head's */
        const int32_t *I = per_head ? idx + ((size_t)b * n_q_heads + h) * budget
                                    : idx + ((size_t)b * n_kv_heads + c) * budget;
        /* the step's positions: F, then W */
        int *S = (int *)malloc(sizeof(int) * (size_t)(n + k_recent + 1));
        int m_S = 0;
        for (int t = 0; t < n; ++t)
            if (I[t] < r_T) S[m_S++] = I[t];
        for (int t = w0; t < cur; ++t) S[m_S++] = t;
        const uint16_t *kc = k + ((size_t)b * n_kv_heads + c) * max_ctx * d;
        const uint16_t *vc = v + ((size_t)b * n_kv_heads + c) * max_ctx * d;
        const uint16_t *qs = q_draft + ((size_t)b * n_q_heads + h) * d;
        double *x = (double *)malloc(sizeof(double) * (size_t)(m_S > 0 ? m_S : 1));
        double m = -INFINITY;
        for (int t = 0; t < m_S; ++t) {
            double dot = 0.0;
            for (int e = 0; e < d; ++e)
                dot += widen_bf16(qs[e]) * widen_bf16(kc[(size_t)S[t] * d + e]);
            x[t] = sm_scale * dot;
            if (x[t] > m) m = x[t];
        }
        double L = 0.0;
        for (int t = 0; t < m_S; ++t) {
            x[t] = exp(x[t] - m);
            L += x[t];
        }
        double *o = out + ((size_t)b * n_q_heads + h) * d;
        for (int e = 0; e < d; ++e) o[e] = 0.0;
        for (int t = 0; t < m_S; ++t) {
            const double P = x[t] / L;
            for (int e = 0; e < d; ++e) o[e] += P * widen_bf16(vc[(size_t)S[t] * d + e]);
        }
        free(x);
        free(S);
    }
    return 0;
}

int oracle_draft_step(int batch, int n_q_heads, int n_kv_heads, int head_dim, int max_ctx,
                      int budget, int k_sink, int k_recent, const int32_t *base_len,
                      const int32_t *cur_len, const uint16_t *q_draft, const uint16_t *k,
                      const uint16_t *v, const int32_t *idx, double sm_scale, double *out)
{
    return draft_step_sets(0, batch, n_q_heads, n_kv_heads, head_dim, max_ctx, budget, k_sink,
                           k_recent, base_len, cur_len, q_draft, k, v, idx, sm_scale, out);
}

/*
 * The same step with one index set per query head (Sec. 3.2 keeps importance
 * for every attention head): idx is [batch][Hq][budget], the set of head h
 * built at base_len by select over that head's scores; head h attends over the
 * fixed part of its own set and the shared slid window, with the rows of its
 * KV head h / (Hq/Hkv).
 */
int oracle_draft_step_heads(int batch, int n_q_heads, int n_kv_heads, int head_dim, int max_ctx,
                            int budget, int k_sink, int k_recent, const int32_t *base_len,
                            const int32_t *cur_len, const uint16_t *q_draft, const uint16_t *k,
                            const uint16_t *v, const int32_t *idx, double sm_scale, double *out)
{
    return draft_step_sets(1, batch, n_q_heads, n_kv_heads, head_dim, max_ctx, budget, k_sink,
                           k_recent, base_len, cur_len, q_draft, k, v, idx, sm_scale, out);
}

/* ---------------------------------------------------------------------------
 * Adaptive speculation length (Sec. 3.3).
 * ------------------------------------------------------------------------- */

/* Eq. 6: one exponential-moving-average step of a class-mean entropy. */
double oracle_ema(double prev, double observed, double beta)
{
    return beta * prev + (1.0 - beta) * observed;
}

/*
 * Eq. 6 applied to one verification (readings of Sec. 3.3, which labels every
 * drafted token accepted or rejected and tracks one mean entropy per label):
 * H[0 .. n_drafted) are the draft entropies in drafting order and the first
 * n_accepted of them were accepted.  The accepted label observes the mean of
 * H[0 .. n_accepted), the rejected label the mean of H[n_accepted ..
 * n_drafted).  A label's first observation sets its mean; later ones move it
 * by one EMA step with coefficient beta.  A label with no tokens in this
 * verification keeps its state.
 * state[0 .. 4) = {h_acc, h_rej, seen_acc, seen_rej}, updated in place.
 * Returns 0, or -1 on bad counts.
 */
int oracle_ctrl_observe(double *state, const double *H, int n_drafted, int n_accepted,
                        double beta)
{
    if (n_drafted < 0 || n_accepted < 0 || n_accepted > n_drafted) return -1;
    for (int cls = 0; cls < 2; ++cls) {
        const int lo = cls == 0 ? 0 : n_accepted;
        const int hi = cls == 0 ? n_accepted : n_drafted;
        if (hi == lo) continue;                 /* no token carries this label */
        double sum = 0.0;
        for (int i = lo; i < hi; ++i) sum += H[i];
        const double mean = sum / (double)(hi - lo);
        if (state[2 + cls] != 0.0)
            state[cls] = oracle_ema(state[cls], mean, beta);
        else
            state[cls] = mean;
        state[2 + cls] = 1.0;
    }
    return 0;
}

/* Eq. 7, as printed: softmax over the negative L1 distances to the centers. */
double oracle_accept_prob(double H, double h_acc, double h_rej)
{
    const double ea = exp(-fabs(H - h_acc));
    const double er = exp(-fabs(H - h_rej));
    return ea / (ea + er);
}

/* Expected number of accepted drafts among the first k: sum_m prod_{i<=m} p_i. */
double oracle_expected_accepted(const double *p, int k)
{
    double sum = 0.0;
    for (int m = 1; m <= k; ++m) {
        double prod = 1.0;
        for (int i = 0; i < m; ++i) prod *= p[i];
        sum += prod;
    }
    return sum;
}

/* The Eq. 8 objective: expected tokens per step over the step's cost. */
double oracle_step_efficiency(const double *p, int k, double c_draft, double c_verify)
{
    return (1.0 + oracle_expected_accepted(p, k)) / ((double)k * c_draft + c_verify);
}

/*
 * Eq. 8: k* = argmax over candidates k (with k <= n, so that p_1..p_k are
 * known) of the objective.  Equal objectives resolve to the smaller k.
 * Returns -1 if no candidate qualifies.
 */
int oracle_choose_k(const double *p, int n, const int32_t *cands, int n_cands,
                    double c_draft, double c_verify)
{
    int best = -1;
    double best_val = 0.0;
    for (int t = 0; t < n_cands; ++t) {
        const int k = cands[t];
        if (k < 0 || k > n) continue;
        const double val = oracle_step_efficiency(p, k, c_draft, c_verify);
        if (best < 0 || val > best_val || (val == best_val && k < best)) {
            best = k;
            best_val = val;
        }
    }
    return best;
}

/* ---------------------------------------------------------------------------
 * Around the path: the statistics of token logits that the controller and the
 * verification stage consume.
 * ------------------------------------------------------------------------- */

/*
 * Per-row token statistics (Sec. 3.3: H_i is the entropy of the drafter's
 * output distribution for draft token i; Sec. 2.1: verification keeps the
 * drafted tokens the target model agrees with).  Row r of logits
 * [n_rows][row_stride], its first vocab entries, as bf16 bit patterns
 * (logits_bf16) or fp32 values (logits_f32; exactly one of the two given):
 *     p = softmax(x),  entropy[r] = -sum_i p_i ln p_i  (nats),
 *     argmax[r] = the lowest index of the largest logit.
 * Either output may be NULL.  Returns 0 or -1.
 */
int oracle_row_stats(int n_rows, int vocab, int row_stride, const uint16_t *logits_bf16,
                     const float *logits_f32, double *entropy, int32_t *argmax)
{
    if (n_rows < 1 || vocab < 1 || row_stride < vocab) return -1;
    if ((logits_bf16 == NULL) == (logits_f32 == NULL)) return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int r = 0; r < n_rows; ++r) {
        double *x = (double *)malloc(sizeof(double) * (size_t)vocab);
        for (int i = 0; i < vocab; ++i)
            x[i] = logits_bf16 ? widen_bf16(logits_bf16[(size_t)r * row_stride + i])
                               : (double)logits_f32[(size_t)r * row_stride + i];
        int a = 0;
        for (int i = 1; i < vocab; ++i)
            if (x[i] > x[a]) a = i;
        const double m = x[a];
        double Z = 0.0;
        for (int i = 0; i < vocab; ++i) Z += exp(x[i] - m);
        double H = 0.0;
        for (int i = 0; i < vocab; ++i) {
            const double lp = x[i] - m - log(Z);      /* ln p_i */
            H -= exp(lp) * lp;
        }
        if (entropy) entropy[r] = H;
        if (argmax) argmax[r] = a;
        free(x);
    }
    return 0;
}

/*
 * Greedy verification (Sec. 2.1's verification stage with the greedy
 * criterion; the paper does not spell out its acceptance rule).  Sequence b
 * drafted k = k_len[b] tokens draft[b][0..k); its verify pass produced the
 * k + 1 logit rows logits[b][0..k] (row j predicts the token after drafted
 * token j - 1; layout [batch][max_k + 1][row_stride]).  With t_j = the argmax
 * of row j (lowest index on ties):
 *     n_accepted[b] = the largest m <= k with draft[b][j] == t_j for all j < m,
 *     next_token[b] = t_m, the corrected (or, if m == k, the bonus) token.
 * Returns 0 or -1.
 */
int oracle_greedy_accept(int batch, int max_k, int vocab, int row_stride, const int32_t *k_len,
                         const uint16_t *logits_bf16, const float *logits_f32,
                         const int32_t *draft, int32_t *n_accepted, int32_t *next_token)
{
    if (batch < 1 || max_k < 0 || vocab < 1 || row_stride < vocab) return -1;
    if ((logits_bf16 == NULL) == (logits_f32 == NULL)) return -1;
    for (int b = 0; b < batch; ++b)
        if (k_len[b] < 0 || k_len[b] > max_k) return -1;
    const int rows = batch * (max_k + 1);
    int32_t *t = (int32_t *)malloc(sizeof(int32_t) * (size_t)rows);
    const int rc = oracle_row_stats(rows, vocab, row_stride, logits_bf16, logits_f32, NULL, t);
    if (rc == 0) {
        for (int b = 0; b < batch; ++b) {
            const int32_t *tb = t + (size_t)b * (max_k + 1);
            const int32_t *db = draft + (size_t)b * max_k;
            int m = 0;
            while (m < k_len[b] && db[m] == tb[m]) ++m;
            n_accepted[b] = m;
            next_token[b] = tb[m];
        }
    }
    free(t);
    return rc;
}

/* One logit row at temperature tau as a distribution: its largest scaled
 * logit m and normalizer Z = sum_i exp(x_i / tau - m). */
static void row_dist(const float *x, int vocab, double tau, double *m, double *Z)
{
    double mx = -INFINITY;
    for (int i = 0; i < vocab; ++i) {
        const double y = (double)x[i] / tau;
        if (y > mx) mx = y;
    }
    double z = 0.0;
    for (int i = 0; i < vocab; ++i) z += exp((double)x[i] / tau - mx);
    *m = mx;
    *Z = z;
}

static double row_prob(const float *x, int i, double tau, double m, double Z)
{
    return exp((double)x[i] / tau - m) / Z;
}

/* The smallest index whose cumulative mass (in index order) exceeds
 * u * total; the last index with mass when rounding leaves none. */
static int draw_by_inversion(const double *w, int vocab, double u)
{
    double total = 0.0;
    for (int i = 0; i < vocab; ++i) total += w[i];
    const double target = u * total;
    double run = 0.0;
    int last = 0;
    for (int i = 0; i < vocab; ++i) {
        if (w[i] > 0.0) last = i;
        run += w[i];
        if (run > target) return i;
    }
    return last;
}

/*
 * Speculative sampling, the verification rule that keeps the target model's
 * output distribution (Sec. 1 and Sec. 2.1 rely on it; the paper does not
 * print it).  Sequence b drafted k = k_len[b] tokens x_j = draft[b][j] from
 * the drafter's logit rows dlogits[b][j] (layout [batch][max_k][row_stride]);
 * its verify pass gave the target rows tlogits[b][0..k] (layout
 * [batch][max_k + 1][row_stride]; row j scores the token after drafted token
 * j - 1).  At temperature tau > 0 let p_j = softmax(tlogits[b][j] / tau) and
 * q_j = softmax(dlogits[b][j] / tau).  With the caller's uniforms
 * u_acc[b][j] ([batch][max_k]) and u_smp[b] in [0, 1):
 *   drafted token j passes when u_acc[b][j] * q_j(x_j) < p_j(x_j), i.e. with
 *   probability min(1, p_j(x_j) / q_j(x_j));
 *   n_accepted[b] = m, the number that pass before the first that does not;
 *   next_token[b] is drawn by inversion with u_smp[b] from
 *   r(x) = max(0, p_m(x) - q_m(x)) when m < k (from p_m if r has no mass),
 *   or from p_k when every drafted token passed.
 * Returns 0 or -1.
 */
int oracle_spec_accept(int batch, int max_k, int vocab, int row_stride, const int32_t *k_len,
                       const float *tlogits, const float *dlogits, double tau,
                       const int32_t *draft, const double *u_acc, const double *u_smp,
                       int32_t *n_accepted, int32_t *next_token)
{
    if (batch < 1 || max_k < 0 || vocab < 1 || row_stride < vocab || !(tau > 0.0)) return -1;
    for (int b = 0; b < batch; ++b)
        if (k_len[b] < 0 || k_len[b] > max_k) return -1;
    double *w = (double *)malloc(sizeof(double) * (size_t)vocab);
    for (int b = 0; b < batch; ++b) {
        const int k = k_len[b];
        int m = 0;
        for (; m < k; ++m) {
            const float *t = tlogits + ((size_t)b * (max_k + 1) + m) * row_stride;
            const float *d = dlogits + ((size_t)b * max_k + m) * row_stride;
            const int x = draft[(size_t)b * max_k + m];
            double mt, zt, md, zd;
            row_dist(t, vocab, tau, &mt, &zt);
            row_dist(d, vocab, tau, &md, &zd);
            const double p = row_prob(t, x, tau, mt, zt);
            const double q = row_prob(d, x, tau, md, zd);
            if (!(u_acc[(size_t)b * max_k + m] * q < p)) break;
        }
        const float *t = tlogits + ((size_t)b * (max_k + 1) + m) * row_stride;
        double mt, zt;
        row_dist(t, vocab, tau, &mt, &zt);
        double mass = 0.0;
        if (m < k) {   /* the residual of the first rejected position */
            const float *d = dlogits + ((size_t)b * max_k + m) * row_stride;
            double md, zd;
            row_dist(d, vocab, tau, &md, &zd);
            for (int i = 0; i < vocab; ++i) {
                const double r = row_prob(t, i, tau, mt, zt) - row_prob(d, i, tau, md, zd);
                w[i] = r > 0.0 ? r : 0.0;
                mass += w[i];
            }
        }
        if (!(mass > 0.0))
            for (int i = 0; i < vocab; ++i) w[i] = row_prob(t, i, tau, mt, zt);
        n_accepted[b] = m;
        next_token[b] = draw_by_inversion(w, vocab, u_smp[b]);
    }
    free(w);
    return 0;
}

/* ---------------------------------------------------------------------------
 * Per-query-head variant of Eq. 3 / Eq. 5 (Sec. 3.2 states importance "for
 * every layer and attention head"; the main path keeps it per KV head).
 * ------------------------------------------------------------------------- */

/*
 * Eq. 3 per query head: scores[b,h,i] = sum over the last min(W, q) verify
 * rows j of P_{j,h,i}, the softmax probability of row j, head h on key i
 * (causal as in oracle_verify).  Layout [batch][Hq][max_ctx]; entries past T
 * are left untouched, entries below T start at 0.  Returns 0 or -1.
 */
int oracle_head_scores(int batch, int n_q_heads, int n_kv_heads, int head_dim, int max_ctx,
                       int max_q, const int32_t *ctx_len, const int32_t *q_len,
                       const uint16_t *q, const uint16_t *k, double sm_scale, int window,
                       double *scores)
{
    if (batch < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads != 0 || head_dim < 1 ||
        window < 1)
        return -1;
    for (int b = 0; b < batch; ++b)
        if (q_len[b] < 1 || q_len[b] > max_q || ctx_len[b] < q_len[b] || ctx_len[b] > max_ctx)
            return -1;
    const int g = n_q_heads / n_kv_heads;
    const int d = head_dim;
#pragma omp parallel for schedule(dynamic, 1)
    for (int bh = 0; bh < batch * n_q_heads; ++bh) {
        const int b = bh / n_q_heads, h = bh % n_q_heads, c = h / g;
        const int T = ctx_len[b], nq = q_len[b];
        const int w = window < nq ? window : nq;
        double *S = scores + ((size_t)b * n_q_heads + h) * max_ctx;
        const uint16_t *kc = k + ((size_t)b * n_kv_heads + c) * max_ctx * d;
        double *x = (double *)malloc(sizeof(double) * (size_t)T);
        for (int i = 0; i < T; ++i) S[i] = 0.0;
        for (int j = nq - w; j < nq; ++j) {
            const int p = T - nq + j;
            const uint16_t *qs = q + (((size_t)b * max_q + j) * n_q_heads + h) * d;
            double m = -INFINITY;
            for (int i = 0; i <= p; ++i) {
                double dot = 0.0;
                for (int e = 0; e < d; ++e)
                    dot += widen_bf16(qs[e]) * widen_bf16(kc[(size_t)i * d + e]);
                x[i] = sm_scale * dot;
                if (x[i] > m) m = x[i];
            }
            double L = 0.0;
            for (int i = 0; i <= p; ++i) {
                x[i] = exp(x[i] - m);
                L += x[i];
            }
            for (int i = 0; i <= p; ++i) S[i] += x[i] / L;
        }
        free(x);
    }
    return 0;
}

/*
 * Eq. 5 with one index set per query head: head h of sequence b attends over
 * the n = n_idx[b] rows I = idx[b,h,0..n) of its KV head c = h / g.
 * Layouts: idx [batch][Hq][budget], q_draft / out [batch][Hq][d].
 * Returns 0 or -1.
 */
int oracle_draft_heads(int batch, int n_q_heads, int n_kv_heads, int head_dim, int max_ctx,
                       int budget, const int32_t *n_idx, const uint16_t *q_draft,
                       const uint16_t *k, const uint16_t *v, const int32_t *idx,
                       double sm_scale, double *out)
{
    if (batch < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads != 0 || head_dim < 1)
        return -1;
    for (int b = 0; b < batch; ++b)
        if (n_idx[b] < 1 || n_idx[b] > budget) return -1;
    const int g = n_q_heads / n_kv_heads;
    const int d = head_dim;
#pragma omp parallel for schedule(dynamic, 1)
    for (int bh = 0; bh < batch * n_q_heads; ++bh) {
        const int b = bh / n_q_heads, h = bh % n_q_heads, c = h / g;
        const int n = n_idx[b];
        const int32_t *I = idx + ((size_t)b * n_q_heads + h) * budget;
        const uint16_t *kc = k + ((size_t)b * n_kv_heads + c) * max_ctx * d;
        const uint16_t *vc = v + ((size_t)b * n_kv_heads + c) * max_ctx * d;
        const uint16_t *qs = q_draft + ((size_t)b * n_q_heads + h) * d;
        double *x = (double *)malloc(sizeof(double) * (size_t)n);
        double m = -INFINITY;
        for (int t = 0; t < n; ++t) {
            double dot = 0.0;
            for (int e = 0; e < d; ++e)
                dot += widen_bf16(qs[e]) * widen_bf16(kc[(size_t)I[t] * d + e]);
            x[t] = sm_scale * dot;
            if (x[t] > m) m = x[t];
        }
        double L = 0.0;
        for (int t = 0; t < n; ++t) {
            x[t] = exp(x[t] - m);
            L += x[t];
        }
        double *o = out + ((size_t)b * n_q_heads + h) * d;
        for (int e = 0; e < d; ++e) o[e] = 0.0;
        for (int t = 0; t < n; ++t) {
            const double P = x[t] / L;
            for (int e = 0; e < d; ++e) o[e] += P * widen_bf16(vc[(size_t)I[t] * d + e]);
        }
        free(x);
    }
    return 0;
}
