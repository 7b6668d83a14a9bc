/*
 * Plain fp64 CPU oracle for DSpark's batched verification step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path links, loads or
 * calls this file: only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header, table or constant with
 * the GPU library.
 *
 * It is deliberately slow and literal:
 *   - scheduling follows the hardware-aware prefix scheduler (Algorithm 1 of
 *     the section on confidence-scheduled verification) step by step, and its
 *     asynchronous form (the section on the scheduler in practice): a
 *     capacity from the no-break search on earlier confidences, then top-K
 *     admission of the current candidates;
 *   - attention is the textbook masked softmax attention, written out;
 *   - acceptance is the left-to-right speculative acceptance rule of the
 *     background section on speculative decoding, with the conventions listed
 *     at each function;
 *   - the Markov-head and RNN-head draft blocks follow the left-to-right
 *     factorisation of the semi-autoregressive stage, one position at a time.
 * All arithmetic is fp64; bf16 inputs are widened exactly.  OpenMP only runs
 * independent rows side by side; no row's arithmetic is reordered.
 *
 * Parity pins: every function here is pinned by tests against values printed
 * in the paper's appendix counterexample, closed forms, library routines and
 * brute force on tiny inputs.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_EINVAL 1

/* ----------------------------------------------------------------- helpers */

static double bf16_to_f64(uint16_t b) {
    uint32_t u = ((uint32_t)b) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* dtype 0 = fp32, 1 = bf16 (uint16 bit patterns) */
static double elem(const void* base, int64_t i, int dtype) {
    if (dtype == 0) return (double)((const float*)base)[i];
    return bf16_to_f64(((const uint16_t*)base)[i]);
}

/* Confidence as used in the survival product.  The paper takes c in (0,1);
   a value that is not > 0 (zero, negative, NaN) ends the request's candidate
   list, a value above 1 is read as 1. */
static double conf_value(float c) {
    if (!(c > 0.0f)) return 0.0;
    if (c > 1.0f) return 1.0;
    return (double)c;
}

/* ------------------------------------------------------- prefix survival */

/* Prefix survival probabilities a[r, j-1] = prod_{i<=j} c[r, i]
   (Algorithm 1, first loop; "Hardware-Aware Prefix Scheduler" section).
   Sequential fp64 multiplication in increasing j. */
int oracle_survival(const float* conf, int R, int K, double* a) {
    if (!conf || !a || R < 0 || K < 0) return ORACLE_EINVAL;
    for (int r = 0; r < R; ++r) {
        double p = 1.0;
        for (int j = 0; j < K; ++j) {
            double c = conf_value(conf[(int64_t)r * K + j]);
            p = p * c;
            a[(int64_t)r * K + j] = p;
        }
    }
    return ORACLE_OK;
}

/* -------------------------------------------------- Algorithm 1 scheduler */

typedef struct {
    double a;
    int32_t r;
    int32_t j; /* 1-based draft position */
} cand_t;

/* Descending survival; ties by request, then position, ascending. */
static int cand_order(const void* x, const void* y) {
    const cand_t* p = (const cand_t*)x;
    const cand_t* q = (const cand_t*)y;
    if (p->a > q->a) return -1;
    if (p->a < q->a) return 1;
    if (p->r != q->r) return p->r < q->r ? -1 : 1;
    if (p->j != q->j) return p->j < q->j ? -1 : 1;
    return 0;
}

/*
 * Algorithm 1 ("Hardware-Aware Prefix Scheduler").
 *   conf [R, K] fp32, sps [sps_len] fp64 with sps[B] = steps/s at B verify
 *   tokens (B = sum_r (1 + l_r)); sps_len must exceed R*(K+1).
 *   mode 0: causal greedy with early stop (the algorithm as printed);
 *   mode 1: no break -- the same greedy path, keeping the best prefix of it
 *           (the production variant of the "scheduler in practice" section).
 * Outputs: len[R] = l*_r; *theta_best; *n_admitted = number of admitted
 * candidates; *min_margin = min over the throughput comparisons made of
 * |Theta - Theta_best| / Theta_best (how far the decisions are from a tie).
 * theta_trace (nullable, room for R*K+1 values) receives Theta_0, Theta_1, ...
 * for every step evaluated, and *n_trace their count.
 */
int oracle_schedule(const float* conf, int R, int K, const double* sps, int64_t sps_len,
                    int mode, int32_t* len, double* theta_best_out, int32_t* n_admitted_out,
                    double* min_margin_out, double* theta_trace, int64_t* n_trace) {
    if (!conf || !sps || !len || R <= 0 || K < 0) return ORACLE_EINVAL;
    if (mode != 0 && mode != 1) return ORACLE_EINVAL;
    if (sps_len <= (int64_t)R * (K + 1)) return ORACLE_EINVAL;

    double* a = (double*)malloc(sizeof(double) * ((size_t)R * K + 1));
    cand_t* E = (cand_t*)malloc(sizeof(cand_t) * ((size_t)R * K + 1));
    int32_t* l = (int32_t*)calloc((size_t)R, sizeof(int32_t));
    if (!a || !E || !l) { free(a); free(E); free(l); return ORACLE_EINVAL; }

    /* survival probabilities */
    oracle_survival(conf, R, K, a);

    /* candidate space {(r, j) : a_{r,j} > 0}, sorted descending by a */
    int64_t n = 0;
    for (int r = 0; r < R; ++r)
        for (int j = 1; j <= K; ++j) {
            double v = a[(int64_t)r * K + (j - 1)];
            if (v > 0.0) { E[n].a = v; E[n].r = r; E[n].j = j; ++n; }
        }
    qsort(E, (size_t)n, sizeof(cand_t), cand_order);

    /* initial state */
    for (int r = 0; r < R; ++r) { l[r] = 0; len[r] = 0; }
    int64_t B = R;
    double tau = (double)R;
    double theta_best = (double)R * sps[R];
    double min_margin = INFINITY;
    int32_t admitted = 0;
    int64_t nt = 0;
    if (theta_trace) theta_trace[nt] = theta_best;
    ++nt;

    for (int64_t i = 0; i < n; ++i) {
        l[E[i].r] = E[i].j;
        B = B + 1;
        tau = tau + E[i].a;
        double theta = tau * sps[B];
        if (theta_trace) theta_trace[nt] = theta;
        ++nt;
        double m = fabs(theta - theta_best) / theta_best;
        if (m < min_margin) min_margin = m;
        if (theta > theta_best) {
            theta_best = theta;
            for (int r = 0; r < R; ++r) len[r] = l[r]; /* snapshot l* <- l */
            admitted = (int32_t)(i + 1);
        } else if (mode == 0) {
            break;
        }
    }
    if (theta_best_out) *theta_best_out = theta_best;
    if (n_admitted_out) *n_admitted_out = admitted;
    if (min_margin_out) *min_margin_out = min_margin;
    if (n_trace) *n_trace = nt;
    free(a); free(E); free(l);
    return ORACLE_OK;
}

/*
 * Capacity of the asynchronous scheduler (section "Hardware-Aware Prefix
 * Scheduler in Practice").  The search without the early stop (mode 1 above)
 * runs on the confidences of an earlier step; the number of draft tokens it
 * admits is the truncation length of a later step's top-K admission.
 *   conf_prev [R, K] fp32, sps as for oracle_schedule.
 * Outputs *capacity; *min_margin (nullable) as for oracle_schedule.
 */
int oracle_schedule_capacity(const float* conf_prev, int R, int K, const double* sps,
                             int64_t sps_len, int32_t* capacity, double* min_margin_out) {
    if (!capacity) return ORACLE_EINVAL;
    int32_t* len = (int32_t*)malloc(sizeof(int32_t) * (size_t)(R > 0 ? R : 1));
    if (!len) return ORACLE_EINVAL;
    int32_t n_adm = 0;
    int rc = oracle_schedule(conf_prev, R, K, sps, sps_len, 1, len, NULL, &n_adm,
                             min_margin_out, NULL, NULL);
    free(len);
    if (rc != ORACLE_OK) return rc;
    *capacity = n_adm;
    return ORACLE_OK;
}

/*
 * Dynamic top-K admission of the same section.  The current candidates
 * {(r, j) : a_{r,j} > 0}, with a the survival products of the CURRENT
 * confidences, are ranked exactly as in Algorithm 1 (descending a, ties by
 * request then position) and admitted in that order, each admission setting
 * l_r = j, until `capacity` of them are in (all of them if there are fewer;
 * a negative capacity admits none).  No throughput is evaluated here: the
 * capacity carries the whole trade-off, decided on earlier information.
 * Outputs len[R] and *n_admitted (nullable).
 */
int oracle_schedule_topk(const float* conf, int R, int K, int64_t capacity, int32_t* len,
                         int32_t* n_admitted_out) {
    if (!conf || !len || R <= 0 || K < 0) return ORACLE_EINVAL;
    double* a = (double*)malloc(sizeof(double) * ((size_t)R * K + 1));
    cand_t* E = (cand_t*)malloc(sizeof(cand_t) * ((size_t)R * K + 1));
    if (!a || !E) { free(a); free(E); return ORACLE_EINVAL; }
    oracle_survival(conf, R, K, a);
    int64_t n = 0;
    for (int r = 0; r < R; ++r)
        for (int j = 1; j <= K; ++j) {
            double v = a[(int64_t)r * K + (j - 1)];
            if (v > 0.0) { E[n].a = v; E[n].r = r; E[n].j = j; ++n; }
        }
    qsort(E, (size_t)n, sizeof(cand_t), cand_order);
    int64_t take = capacity < 0 ? 0 : (capacity < n ? capacity : n);
    for (int r = 0; r < R; ++r) len[r] = 0;
    for (int64_t i = 0; i < take; ++i) len[E[i].r] = E[i].j;
    if (n_admitted_out) *n_admitted_out = (int32_t)take;
    free(a); free(E);
    return ORACLE_OK;
}

/* -------------------------------------------------------- verify attention */

/*
 * Ragged causal verify attention over a paged KV cache.
 *   Request r owns q_len_r = cu_q[r+1] - cu_q[r] consecutive query tokens of
 *   q [total_q, Hq, Dqk]; its context holds kv_len_r tokens, the last q_len_r
 *   of which are the verify tokens themselves, so query t (0-based) sees keys
 *   0 .. kv_len_r - q_len_r + t.  Key token j lives in page
 *   block_table[r, j / page_size], slot j % page_size; element (page, head,
 *   slot, d) is at page*s[0] + head*s[1] + slot*s[2] + d.  Query head h reads
 *   KV head h / (Hq / Hkv).
 *   o = sum_j softmax_j(scale * <q, k_j>) v_j ;  lse = log sum_j exp(scale <q,k_j>).
 * If rows != NULL only the n_rows listed (token, head) pairs are computed and
 * written, packed in list order; otherwise all total_q * Hq rows are written
 * in [token, head] order.  out: fp64 [.., Dv], lse: fp64 [..] (nullable).
 */
int oracle_verify_attn(const void* q, const void* k_cache, const void* v_cache,
                       const int64_t* ks, const int64_t* vs, const int32_t* block_table,
                       int max_pages, const int32_t* kv_len, const int32_t* cu_q, int R,
                       int Hq, int Hkv, int Dqk, int Dv, int page_size, double scale,
                       int dtype, const int32_t* rows, int64_t n_rows, double* out,
                       double* lse) {
    if (!q || !k_cache || !v_cache || !ks || !vs || !block_table || !kv_len || !cu_q || !out)
        return ORACLE_EINVAL;
    if (R <= 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv || Dqk <= 0 || Dv <= 0 || page_size <= 0)
        return ORACLE_EINVAL;
    for (int r = 0; r < R; ++r) {
        int ql = cu_q[r + 1] - cu_q[r];
        if (ql < 0 || kv_len[r] < ql || kv_len[r] > (int64_t)max_pages * page_size)
            return ORACLE_EINVAL;
    }
    const int64_t total_q = cu_q[R];
    const int64_t count = rows ? n_rows : total_q * Hq;
    const int group = Hq / Hkv;

    /* token -> request */
    int32_t* req_of = (int32_t*)malloc(sizeof(int32_t) * (size_t)(total_q + 1));
    if (!req_of) return ORACLE_EINVAL;
    for (int r = 0; r < R; ++r)
        for (int t = cu_q[r]; t < cu_q[r + 1]; ++t) req_of[t] = r;
    if (rows)
        for (int64_t i = 0; i < count; ++i)
            if (rows[2 * i] < 0 || rows[2 * i] >= total_q || rows[2 * i + 1] < 0 ||
                rows[2 * i + 1] >= Hq) { free(req_of); return ORACLE_EINVAL; }

    int bad = 0;
#pragma omp parallel for schedule(dynamic, 4) reduction(| : bad)
    for (int64_t i = 0; i < count; ++i) {
        int64_t tok = rows ? rows[2 * i] : i / Hq;
        int h = rows ? rows[2 * i + 1] : (int)(i % Hq);
        int r = req_of[tok];
        int ql = cu_q[r + 1] - cu_q[r];
        int t = (int)(tok - cu_q[r]);
        int64_t visible = (int64_t)kv_len[r] - ql + t + 1;
        int g = h / group;
        double* s = (double*)malloc(sizeof(double) * (size_t)(visible > 0 ? visible : 1));
        if (!s) { bad = 1; continue; }
        const int64_t qoff = (tok * Hq + h) * (int64_t)Dqk;
        for (int64_t j = 0; j < visible; ++j) {
            int64_t page = block_table[(int64_t)r * max_pages + j / page_size];
            int64_t base = page * ks[0] + g * ks[1] + (j % page_size) * ks[2];
            double dot = 0.0;
            for (int d = 0; d < Dqk; ++d)
                dot += elem(q, qoff + d, dtype) * elem(k_cache, base + d, dtype);
            s[j] = scale * dot;
        }
        double m = -INFINITY;
        for (int64_t j = 0; j < visible; ++j) if (s[j] > m) m = s[j];
        double den = 0.0;
        for (int64_t j = 0; j < visible; ++j) { s[j] = exp(s[j] - m); den += s[j]; }
        double* o = out + i * (int64_t)Dv;
        for (int d = 0; d < Dv; ++d) o[d] = 0.0;
        for (int64_t j = 0; j < visible; ++j) {
            int64_t page = block_table[(int64_t)r * max_pages + j / page_size];
            int64_t base = page * vs[0] + g * vs[1] + (j % page_size) * vs[2];
            double w = s[j] / den;
            for (int d = 0; d < Dv; ++d) o[d] += w * elem(v_cache, base + d, dtype);
        }
        if (lse) lse[i] = m + log(den);
        free(s);
    }
    free(req_of);
    return bad ? ORACLE_EINVAL : ORACLE_OK;
}

/* ------------------------------------------------------------- acceptance */

/* Target distribution p = softmax(inv_temp * z) of one logit row, fp64. */
static void target_dist(const void* row, int dtype, int V, double inv_temp, double* p) {
    double m = -INFINITY;
    for (int v = 0; v < V; ++v) {
        p[v] = inv_temp * elem(row, v, dtype);
        if (p[v] > m) m = p[v];
    }
    double S = 0.0;
    for (int v = 0; v < V; ++v) { p[v] = exp(p[v] - m); S += p[v]; }
    for (int v = 0; v < V; ++v) p[v] = p[v] / S;
}

/* Index of the largest raw logit; the lowest index among equals. */
static int argmax_row(const void* row, int dtype, int V) {
    int best = 0;
    double bv = elem(row, 0, dtype);
    for (int v = 1; v < V; ++v) {
        double x = elem(row, v, dtype);
        if (x > bv) { bv = x; best = v; }
    }
    return best;
}

/* Inverse-CDF draw from unnormalised non-negative masses with one uniform:
   the smallest v (ascending vocabulary order) whose running mass exceeds
   u * total.  *margin = distance of u*total from the chosen bucket's edges,
   in units of the total mass. */
static int inverse_cdf(const double* mass, int V, double u, double* margin) {
    double total = 0.0;
    for (int v = 0; v < V; ++v) total += mass[v];
    double thr = u * total;
    double cum = 0.0;
    int last_pos = 0;
    for (int v = 0; v < V; ++v) {
        double prev = cum;
        cum += mass[v];
        if (mass[v] > 0.0) last_pos = v;
        if (cum > thr) {
            double m1 = (thr - prev) / total, m2 = (cum - thr) / total;
            *margin = m1 < m2 ? m1 : m2;
            return v;
        }
    }
    *margin = 0.0;
    return last_pos;
}

/*
 * Speculative acceptance for every request.
 *   Rows: logits row cu_q[r] + t (row stride ld elements) is the target's
 *   distribution for the token after verify slot t; slot t < l_r tests draft
 *   token draft_tok[r, t] (the paper's x_{t+1}), slot l_r supplies the bonus
 *   token.  l_r = q_len_r - 1 must not exceed K.
 *   Greedy (draft_p == NULL and u == NULL): x_{t+1} is accepted iff it equals
 *     the argmax of the raw logits (lowest index on ties); the emitted token is
 *     the argmax of the first rejected row, or of row l_r if all are accepted.
 *   Stochastic: p_t = softmax(inv_temp * z_t); x_{t+1} is accepted iff
 *     u[r, t] < p_t(x) / p_d(x) (p_d(x) = 0 accepts), i.e. with probability
 *     min(1, p_t/p_d); left to right, the first rejection at t* ends the
 *     request and the corrected token is drawn from max(0, p_t - p_d) (p_t if
 *     that has no mass); with no rejection the bonus token is drawn from
 *     p_{l_r}.  Draws use the inverse CDF at u[r, K].
 * Outputs accepted_len[R], next_tok[R]; margin[R] (nullable) = the smallest
 * distance of any stochastic decision taken from its tie (|u - min(1,ratio)|
 * for tests, CDF units for the draw), +inf for greedy requests.
 * accept_rate (nullable, [total_q]) = sum_v min(p_t(v), p_d(v)) for every
 * row t < l_r that carries a draft, whether or not an earlier draft was
 * rejected (the analytic per-step acceptance rate of the confidence-head
 * section: one minus the total variation distance); -1 for bonus rows and in
 * greedy mode.
 */
int oracle_accept(const int32_t* draft_tok, const float* draft_p, const void* logits,
                  int logit_dtype, int64_t ld, const float* u, const int32_t* cu_q, int R,
                  int K, int V, double inv_temp, int32_t* accepted_len, int32_t* next_tok,
                  double* margin, double* accept_rate) {
    if (!draft_tok || !logits || !cu_q || !accepted_len || !next_tok) return ORACLE_EINVAL;
    if (R <= 0 || K < 0 || V <= 0 || ld < V || !(inv_temp > 0.0)) return ORACLE_EINVAL;
    const int greedy = (draft_p == NULL && u == NULL);
    if (!greedy && (draft_p == NULL || u == NULL)) return ORACLE_EINVAL;
    const size_t esz = logit_dtype == 0 ? 4 : 2;
    for (int r = 0; r < R; ++r) {
        int ql = cu_q[r + 1] - cu_q[r];
        if (ql < 1 || ql > K + 1) return ORACLE_EINVAL;
        for (int t = 0; t < ql - 1; ++t) {
            int32_t x = draft_tok[(int64_t)r * K + t];
            if (x < 0 || x >= V) return ORACLE_EINVAL;
        }
    }
    if (accept_rate)
        for (int64_t i = 0; i < cu_q[R]; ++i) accept_rate[i] = -1.0;

    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int r = 0; r < R; ++r) {
        const int l = cu_q[r + 1] - cu_q[r] - 1;
        const char* base = (const char*)logits;
        double mg = INFINITY;
        int acc = l, tok = -1;
        if (greedy) {
            for (int t = 0; t < l; ++t) {
                const void* row = base + (size_t)(cu_q[r] + t) * (size_t)ld * esz;
                int am = argmax_row(row, logit_dtype, V);
                if (draft_tok[(int64_t)r * K + t] != am) { acc = t; tok = am; break; }
            }
            if (tok < 0)
                tok = argmax_row(base + (size_t)(cu_q[r] + l) * (size_t)ld * esz, logit_dtype, V);
        } else {
            double* p = (double*)malloc(sizeof(double) * (size_t)V);
            double* m = (double*)malloc(sizeof(double) * (size_t)V);
            if (!p || !m) { free(p); free(m); bad = 1; continue; }
            if (accept_rate)
                for (int t = 0; t < l; ++t) {
                    const void* row = base + (size_t)(cu_q[r] + t) * (size_t)ld * esz;
                    const float* pd = draft_p + ((int64_t)r * K + t) * (int64_t)V;
                    target_dist(row, logit_dtype, V, inv_temp, p);
                    double ar = 0.0;
                    for (int v = 0; v < V; ++v) ar += p[v] < (double)pd[v] ? p[v] : (double)pd[v];
                    accept_rate[cu_q[r] + t] = ar;
                }
            for (int t = 0; t < l; ++t) {
                const void* row = base + (size_t)(cu_q[r] + t) * (size_t)ld * esz;
                const float* pd = draft_p + ((int64_t)r * K + t) * (int64_t)V;
                target_dist(row, logit_dtype, V, inv_temp, p);
                int32_t x = draft_tok[(int64_t)r * K + t];
                double pdx = (double)pd[x];
                double ratio = pdx > 0.0 ? p[x] / pdx : INFINITY;
                double uu = (double)u[(int64_t)r * (K + 1) + t];
                double d = fabs(uu - (ratio < 1.0 ? ratio : 1.0));
                if (d < mg) mg = d;
                if (!(uu < ratio)) {
                    acc = t;
                    double tot = 0.0;
                    for (int v = 0; v < V; ++v) {
                        double e = p[v] - (double)pd[v];
                        m[v] = e > 0.0 ? e : 0.0;
                        tot += m[v];
                    }
                    if (!(tot > 0.0)) memcpy(m, p, sizeof(double) * (size_t)V);
                    double cm;
                    tok = inverse_cdf(m, V, (double)u[(int64_t)r * (K + 1) + K], &cm);
                    if (cm < mg) mg = cm;
                    break;
                }
            }
            if (tok < 0) {
                const void* row = base + (size_t)(cu_q[r] + l) * (size_t)ld * esz;
                target_dist(row, logit_dtype, V, inv_temp, p);
                double cm;
                tok = inverse_cdf(p, V, (double)u[(int64_t)r * (K + 1) + K], &cm);
                if (cm < mg) mg = cm;
            }
            free(p); free(m);
        }
        accepted_len[r] = acc;
        next_tok[r] = tok;
        if (margin) margin[r] = mg;
    }
    return bad ? ORACLE_EINVAL : ORACLE_OK;
}

/* ------------------------------------------------ Markov-head draft block */

/*
 * The sequential stage of semi-autoregressive drafting with the Markov head
 * (section on semi-autoregressive generation: the block distribution factors
 * left to right, eq. sequential-factorization, and the Markov head's
 * transition bias is the low-rank product of eq. markov), plus the confidence
 * head of the confidence-scheduled verification section (eq. confidence) with
 * the per-position temperatures of its post-hoc calibration.
 *
 * For every request r, with x_0 = anchor[r] and k = 1 .. K:
 *   e_k      = W1[x_{k-1}]                       (embedding row, rank dims)
 *   B_k(v)   = sum_j e_k[j] * W2[j, v]           (transition bias)
 *   p_k      = softmax(inv_temp * (U_k + B_k))   (U_k = base logits of position k)
 *   x_k      = inverse CDF of p_k at u[r, k-1]   (smallest v, ascending, whose
 *                                                running mass exceeds u * total)
 *   c_k      = sigmoid((w_h . h_k + w_e . e_k) / T_k)   (w = [w_h; w_e])
 * Storage: U row (r, k) starts at element (r * K + k - 1) * ld (fp32 or bf16);
 * W1 [V, rank] and the projection W2t [V, rank] (row v holds W2[:, v]) in
 * bf16; hidden [R, K, d] bf16 (nullable when d = 0); w_conf [d + rank] fp32;
 * sts_temp [K] fp32 (nullable: all 1); u [R, K] fp32.
 * Outputs: draft_tok [R, K] = x_k, draft_p [R, K, V] = p_k (nullable),
 * conf [R, K] = c_k, margin [R, K] (nullable) = the distance of each draw from
 * its bucket's edges, in units of the total mass.
 */
int oracle_markov_draft(const int32_t* anchor, const void* U, int u_dtype, int64_t ld,
                        const uint16_t* W1, const uint16_t* W2t, int rank,
                        const uint16_t* hidden, const float* w_conf, int d,
                        const float* sts_temp, const float* u, double inv_temp, int R, int K,
                        int V, int32_t* draft_tok, double* draft_p, double* conf,
                        double* margin) {
    if (!anchor || !U || !W1 || !W2t || !w_conf || !u || !draft_tok || !conf) return ORACLE_EINVAL;
    if (R < 0 || K < 1 || V < 1 || rank < 1 || d < 0 || ld < V || (d > 0 && !hidden))
        return ORACLE_EINVAL;
    for (int r = 0; r < R; ++r)
        if (anchor[r] < 0 || anchor[r] >= V) return ORACLE_EINVAL;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(|| : bad)
    for (int r = 0; r < R; ++r) {
        double* z = (double*)malloc(sizeof(double) * (size_t)V);
        double* e = (double*)malloc(sizeof(double) * (size_t)rank);
        if (!z || !e) { bad = 1; free(z); free(e); continue; }
        int prev = anchor[r];
        for (int k = 1; k <= K; ++k) {
            const int64_t row = (int64_t)r * K + (k - 1);
            /* embedding of the preceding token */
            for (int j = 0; j < rank; ++j) e[j] = bf16_to_f64(W1[(int64_t)prev * rank + j]);
            /* z = inv_temp * (U_k + B_k), then the softmax */
            double m = -INFINITY;
            for (int v = 0; v < V; ++v) {
                double b = 0.0;
                for (int j = 0; j < rank; ++j) b += e[j] * bf16_to_f64(W2t[(int64_t)v * rank + j]);
                z[v] = inv_temp * (elem(U, row * ld + v, u_dtype) + b);
                if (z[v] > m) m = z[v];
            }
            double S = 0.0;
            for (int v = 0; v < V; ++v) { z[v] = exp(z[v] - m); S += z[v]; }
            for (int v = 0; v < V; ++v) z[v] = z[v] / S;
            if (draft_p)
                memcpy(draft_p + row * (int64_t)V, z, sizeof(double) * (size_t)V);
            /* draw x_k */
            double mg;
            const int x = inverse_cdf(z, V, (double)u[row], &mg);
            if (margin) margin[row] = mg;
            draft_tok[row] = x;
            /* confidence of position k: the backbone state and the embedding of x_{k-1} */
            double sacc = 0.0;
            for (int i = 0; i < d; ++i) sacc += (double)w_conf[i] * bf16_to_f64(hidden[row * d + i]);
            for (int j = 0; j < rank; ++j) sacc += (double)w_conf[d + j] * e[j];
            const double T = sts_temp ? (double)sts_temp[k - 1] : 1.0;
            conf[row] = 1.0 / (1.0 + exp(-sacc / T));
            prev = x;
        }
        free(z);
        free(e);
    }
    return bad ? ORACLE_EINVAL : ORACLE_OK;
}

/* --------------------------------------------------- RNN-head draft block */

static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

/*
 * The sequential stage with the RNN head (section on semi-autoregressive
 * generation, the RNN-head item, eq. rnn): the same left-to-right
 * factorisation as the Markov head, with the transition bias read from a
 * recurrent state that sees the whole prefix of the block.
 *
 * For every request r, with x_0 = anchor[r], s_0 = 0 and k = 1 .. K:
 *   e_k    = W1[x_{k-1}]
 *   z_k    = [s_{k-1}; e_k; h_k]                     (2 rank + d values)
 *   a_k    = W z_k, W = [W_g; W_c; W_o]              (3 rank values)
 *   s_k    = sigmoid(a_g) * s_{k-1} + (1 - sigmoid(a_g)) * tanh(a_c)
 *   B_k(v) = sum_j W2[j, v] * tanh(a_o)[j]
 *   p_k    = softmax(inv_temp * (U_k + B_k)),   x_k = inverse CDF at u[r, k-1]
 *   c_k    = sigmoid((w_h . h_k + w_e . e_k) / T_k)  (eq. confidence)
 * Storage as oracle_markov_draft, plus Wrnn [3 rank, 2 rank + d] bf16
 * row-major: rows 0 .. rank-1 the gate, then the candidate, then the output
 * component; columns in the order of z_k.  The equation has no bias terms.
 */
int oracle_rnn_draft(const int32_t* anchor, const void* U, int u_dtype, int64_t ld,
                     const uint16_t* W1, const uint16_t* W2t, const uint16_t* Wrnn, int rank,
                     const uint16_t* hidden, const float* w_conf, int d,
                     const float* sts_temp, const float* u, double inv_temp, int R, int K,
                     int V, int32_t* draft_tok, double* draft_p, double* conf,
                     double* margin) {
    if (!anchor || !U || !W1 || !W2t || !Wrnn || !w_conf || !u || !draft_tok || !conf)
        return ORACLE_EINVAL;
    if (R < 0 || K < 1 || V < 1 || rank < 1 || d < 0 || ld < V || (d > 0 && !hidden))
        return ORACLE_EINVAL;
    for (int r = 0; r < R; ++r)
        if (anchor[r] < 0 || anchor[r] >= V) return ORACLE_EINVAL;
    const int nz = 2 * rank + d;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(|| : bad)
    for (int r = 0; r < R; ++r) {
        double* zl = (double*)malloc(sizeof(double) * (size_t)V);
        double* zin = (double*)malloc(sizeof(double) * (size_t)nz);
        double* act = (double*)malloc(sizeof(double) * (size_t)(3 * rank));
        double* st = (double*)calloc((size_t)rank, sizeof(double));
        double* o = (double*)malloc(sizeof(double) * (size_t)rank);
        if (!zl || !zin || !act || !st || !o) {
            bad = 1;
            free(zl); free(zin); free(act); free(st); free(o);
            continue;
        }
        int prev = anchor[r];
        for (int k = 1; k <= K; ++k) {
            const int64_t row = (int64_t)r * K + (k - 1);
            /* z_k = [s_{k-1}; W1[x_{k-1}]; h_k] */
            for (int j = 0; j < rank; ++j) zin[j] = st[j];
            for (int j = 0; j < rank; ++j) zin[rank + j] = bf16_to_f64(W1[(int64_t)prev * rank + j]);
            for (int i = 0; i < d; ++i) zin[2 * rank + i] = bf16_to_f64(hidden[row * d + i]);
            /* the single projection, split into gate, candidate and output */
            for (int i = 0; i < 3 * rank; ++i) {
                double acc = 0.0;
                for (int j = 0; j < nz; ++j) acc += bf16_to_f64(Wrnn[(int64_t)i * nz + j]) * zin[j];
                act[i] = acc;
            }
            /* gated state update (uses s_{k-1} through zin only) and the head's output */
            for (int j = 0; j < rank; ++j) {
                const double g = sigmoid(act[j]);
                st[j] = g * st[j] + (1.0 - g) * tanh(act[rank + j]);
                o[j] = tanh(act[2 * rank + j]);
            }
            /* B_k = W2^T o, then the softmax of inv_temp * (U_k + B_k) */
            double m = -INFINITY;
            for (int v = 0; v < V; ++v) {
                double b = 0.0;
                for (int j = 0; j < rank; ++j) b += bf16_to_f64(W2t[(int64_t)v * rank + j]) * o[j];
                zl[v] = inv_temp * (elem(U, row * ld + v, u_dtype) + b);
                if (zl[v] > m) m = zl[v];
            }
            double S = 0.0;
            for (int v = 0; v < V; ++v) { zl[v] = exp(zl[v] - m); S += zl[v]; }
            for (int v = 0; v < V; ++v) zl[v] = zl[v] / S;
            if (draft_p) memcpy(draft_p + row * (int64_t)V, zl, sizeof(double) * (size_t)V);
            double mg;
            const int x = inverse_cdf(zl, V, (double)u[row], &mg);
            if (margin) margin[row] = mg;
            draft_tok[row] = x;
            /* confidence: the backbone state and the embedding of x_{k-1} */
            double sacc = 0.0;
            for (int i = 0; i < d; ++i) sacc += (double)w_conf[i] * zin[2 * rank + i];
            for (int j = 0; j < rank; ++j) sacc += (double)w_conf[d + j] * zin[rank + j];
            const double T = sts_temp ? (double)sts_temp[k - 1] : 1.0;
            conf[row] = sigmoid(sacc / T);
            prev = x;
        }
        free(zl); free(zin); free(act); free(st); free(o);
    }
    return bad ? ORACLE_EINVAL : ORACLE_OK;
}

/* Sets how many OpenMP threads later parallel regions of the oracle use. */
void oracle_set_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Reports how many OpenMP threads a parallel region of the oracle uses. */
int oracle_threads(void) {
    int n = 1;
#ifdef _OPENMP
#pragma omp parallel
    {
#pragma omp single
        n = omp_get_num_threads();
    }
#endif
    return n;
}
