/*
 * fp64 CPU oracle for the rollout hot path.  TEST INFRASTRUCTURE ONLY: the
 * tests, the smoke check and the bench's CPU-baseline leg call it; the GPU
 * library never does, and this file shares no code, header or table with it.
 *
 * It computes the plain definitions, in double precision, with two-pass
 * (max first, then sum) softmax and no blocking, splitting or online merge:
 *
 *  1. Decode attention for a group of candidates (Sec. 2.2.1, Problem Setup:
 *     every input x gets g candidates y_1..y_g).  Candidate s = p*G + g sees
 *     the KV of its prompt p followed by its own generated KV (the prompt is
 *     shared by the group; refinement turns lengthen it, Sec. 3, Structured
 *     Feedback and Iterative Refinement).  For query head h the key/value
 *     head is h / (Hq/Hkv).  With x_j = scale * <q, k_j>, m = max_j x_j,
 *     w_j = exp(x_j - m) / sum_i exp(x_i - m):
 *         out = sum_j w_j v_j,   lse = m + ln sum_j exp(x_j - m).
 *     An empty context gives out = 0 and lse = -inf.
 *
 *  2. Token log-probability of the sampled token under the policy, the
 *     quantity whose ratio between the new and old policy drives the GRPO
 *     objective (Sec. 3, Eq. grpo-loss), taken over the full vocabulary:
 *         z_v = inv_T * <hidden_r, W_v>,  lse = M + ln sum_v exp(z_v - M),
 *         logprob = z_t - lse  for target t in [0, V);
 *     target -1 marks a masked position (the masked log-prob window of
 *     Sec. 3, Multi-turn RL Training) and gives logprob 0; any other
 *     target outside [0, V) gives NaN.  lse is computed in every case.
 *
 *  3. Group-relative advantages (Sec. 3, the definition under Eq.
 *     grpo-loss): for each prompt's group of G candidates with rewards r_i,
 *         A_i = (r_i - mean(r)) / std(r),
 *     std taken as the sample standard deviation (divisor G-1); a group whose
 *     rewards are all equal (or G = 1) carries no signal and gets A_i = 0.
 *
 *  4. The clipped GRPO surrogate with beta * D_KL = 0 (Sec. 3, Eq.
 *     grpo-loss), as a loss to minimise over a batch of P prompts:
 *         rho = exp(logp_new - logp_old),
 *         L = -(1/(P G)) sum_i (1/|o_i|) sum_t min(rho A_i, clip(rho, 1-eps, 1+eps) A_i),
 *     |o_i| = the number of token rows of candidate i; rows of no candidate
 *     (seq = -1) do not count.  dL/dlogp_new of a row is
 *     -(1/(P G |o_i|)) rho A_i when the ratio term is the minimum (ties
 *     included) and 0 when the clipped term is (clipping then holds the
 *     ratio at a bound, so the term does not depend on logp_new).
 *
 *  5. The backward of the token log-probability with respect to the hidden
 *     rows, given dL/dlogprob = g_r per row (the lm-head itself is frozen
 *     under the paper's QLoRA fine-tuning, Sec. 3, Multi-turn RL Training):
 *     with p_v = softmax_v(z),
 *         dL/dhidden_r = g_r * inv_T * (W_t - sum_v p_v W_v);
 *     a masked row (target -1) gets 0 and an invalid target NaN.
 *
 *  6. Nucleus (top-p) sampling of the next token of each row (Sec. 3,
 *     Multi-turn RL Training: each turn draws its candidates by nucleus
 *     sampling at a temperature).  With y_v = inv_T_r * <hidden_r, W_v> and
 *     p_v = softmax_v(y):
 *       - the tokens are ranked by p_v, largest first, equal p_v by the
 *         smaller id first;
 *       - the nucleus N is the shortest prefix of that ranking whose total
 *         probability reaches top_p;
 *       - given u_r in [0, 1), the sampled token is the smallest id t in N
 *         with sum_{v in N, v <= t} p_v > u_r * sum_{v in N} p_v, i.e. the
 *         inverse CDF of the renormalised nucleus taken in id order.
 *     Also returned: the sampled token's log-prob under the full tempered
 *     softmax (y_t - lse), and three margins that let tests tell robust rows
 *     from knife-edge ones: the distance of u * sum_N p from the ends of the
 *     token's interval (as a fraction of the nucleus mass); how close the
 *     nucleus is to changing (top_p against the mass before and at its last
 *     member, and the probability gap to the next ranked token); and the
 *     mass such a change could move (last member plus next token, over the
 *     nucleus mass; infinite when the sample is one of them).
 *
 *  7. Extend (prefill) attention of a refinement turn (Sec. 3, Structured
 *     Feedback and Iterative Refinement: each turn appends feedback and a
 *     summary to the candidate's context, and the policy reads the whole
 *     context before it generates).  Candidate s = p*G + g has the context
 *     prefix(p) followed by suffix(s), Lp + Ls tokens, whose last n_s <= Ls
 *     suffix tokens are new.  New token i (0 <= i < n_s) is at position
 *     c_i = Lp + Ls - n_s + i of that sequence and attends causally: to
 *     positions 0..c_i, itself included.  With that visible set in place of
 *     the whole context, out and lse are those of definition 1.  Its query
 *     and output rows are q_start[s] + i of a packed [rows, Hq, D] array.
 *     With n_s = 1 this is definition 1 exactly.
 *
 * Inputs are raw bf16 bit patterns (uint16).  Each is widened exactly:
 * bits << 16 is the float32 pattern, and float32 -> double is exact.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static double bf16_to_f64(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

int oracle_abi_version(void) { return 4; }

/* Returns 0 on success, 1 if a scratch allocation failed. */
int oracle_decode_attn(int32_t P, int32_t G, int32_t Hq, int32_t Hkv, int32_t D,
                       float scale,
                       const int64_t *prefix_start, const int32_t *prefix_len,
                       const int64_t *suffix_start, const int32_t *suffix_len,
                       const uint16_t *q,
                       const uint16_t *k_prefix, const uint16_t *v_prefix,
                       const uint16_t *k_suffix, const uint16_t *v_suffix,
                       double *out, double *lse)
{
    const int64_t S = (int64_t)P * G;
    const int32_t r = Hq / Hkv;
    const double sigma = (double)scale;
    int failed = 0;

#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t s = 0; s < S; ++s) {
        for (int32_t h = 0; h < Hq; ++h) {
            const int64_t p = s / G;
            const int32_t kh = h / r;
            const int64_t Lp = prefix_len[p];
            const int64_t Ls = suffix_len[s];
            const int64_t T = Lp + Ls;
            double *o = out + (s * Hq + h) * (int64_t)D;
            const uint16_t *qv = q + (s * Hq + h) * (int64_t)D;

            if (T == 0) {
                for (int32_t d = 0; d < D; ++d) o[d] = 0.0;
                lse[s * Hq + h] = -INFINITY;
                continue;
            }
            double *x = (double *)malloc((size_t)T * sizeof(double));
            if (!x) {
#pragma omp atomic write
                failed = 1;
                continue;
            }
            /* pass 1: scores over the concatenated context prefix ++ suffix */
            for (int64_t j = 0; j < T; ++j) {
                const uint16_t *kr = (j < Lp)
                    ? k_prefix + ((prefix_start[p] + j) * Hkv + kh) * (int64_t)D
                    : k_suffix + ((suffix_start[s] + (j - Lp)) * Hkv + kh) * (int64_t)D;
                double dot = 0.0;
                for (int32_t d = 0; d < D; ++d) dot += bf16_to_f64(qv[d]) * bf16_to_f64(kr[d]);
                x[j] = sigma * dot;
            }
            double m = x[0];
            for (int64_t j = 1; j < T; ++j) if (x[j] > m) m = x[j];
            double Z = 0.0;
            for (int64_t j = 0; j < T; ++j) Z += exp(x[j] - m);
            /* pass 2: softmax-weighted sum of the values */
            for (int32_t d = 0; d < D; ++d) o[d] = 0.0;
            for (int64_t j = 0; j < T; ++j) {
                const uint16_t *vr = (j < Lp)
                    ? v_prefix + ((prefix_start[p] + j) * Hkv + kh) * (int64_t)D
                    : v_suffix + ((suffix_start[s] + (j - Lp)) * Hkv + kh) * (int64_t)D;
                const double w = exp(x[j] - m) / Z;
                for (int32_t d = 0; d < D; ++d) o[d] += w * bf16_to_f64(vr[d]);
            }
            lse[s * Hq + h] = m + log(Z);
            free(x);
        }
    }
    return failed;
}

/* Returns 0 on success, 1 if a scratch allocation failed. */
/* The V logits z_v = inv_T * <h, W_v> of one row whose hidden vector is
 * given in double, and their log-sum-exp (max first, then the sum). */
static double row_logits(int32_t H, int32_t V, const double *h, const uint16_t *w_lm,
                         double inv_T, double *z)
{
    for (int32_t v = 0; v < V; ++v) {
        const uint16_t *wr = w_lm + (int64_t)v * H;
        double dot = 0.0;
        for (int32_t k = 0; k < H; ++k) dot += h[k] * bf16_to_f64(wr[k]);
        z[v] = inv_T * dot;
    }
    double M = z[0];
    for (int32_t v = 1; v < V; ++v) if (z[v] > M) M = z[v];
    double sum = 0.0;
    for (int32_t v = 0; v < V; ++v) sum += exp(z[v] - M);
    return M + log(sum);
}

static double target_logprob(int32_t V, int32_t t, const double *z, double l)
{
    if (t == -1) return 0.0;
    if (t >= 0 && t < V) return z[t] - l;
    return NAN;
}

/* Token log-prob with the hidden rows given in double (finite-difference
 * checks of the backward perturb them). */
int oracle_token_logprob_f64(int64_t R, int32_t H, int32_t V,
                             const double *hidden, const uint16_t *w_lm,
                             const int32_t *target, float inv_temperature,
                             double *logprob, double *lse)
{
    const double inv_T = (double)inv_temperature;
    int failed = 0;

#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < R; ++r) {
        double *z = (double *)malloc((size_t)V * sizeof(double));
        if (!z) {
#pragma omp atomic write
            failed = 1;
            continue;
        }
        const double l = row_logits(H, V, hidden + r * (int64_t)H, w_lm, inv_T, z);
        lse[r] = l;
        logprob[r] = target_logprob(V, target[r], z, l);
        free(z);
    }
    return failed;
}

int oracle_token_logprob(int64_t R, int32_t H, int32_t V,
                         const uint16_t *hidden, const uint16_t *w_lm,
                         const int32_t *target, float inv_temperature,
                         double *logprob, double *lse)
{
    const double inv_T = (double)inv_temperature;
    int failed = 0;

#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < R; ++r) {
        double *z = (double *)malloc((size_t)V * sizeof(double));
        double *h = (double *)malloc((size_t)H * sizeof(double));
        if (!z || !h) {
#pragma omp atomic write
            failed = 1;
            free(z);
            free(h);
            continue;
        }
        const uint16_t *hr = hidden + r * (int64_t)H;
        for (int32_t k = 0; k < H; ++k) h[k] = bf16_to_f64(hr[k]);
        const double l = row_logits(H, V, h, w_lm, inv_T, z);
        lse[r] = l;
        logprob[r] = target_logprob(V, target[r], z, l);
        free(z);
        free(h);
    }
    return failed;
}

int oracle_grpo_advantage(int64_t P, int32_t G, const double *reward, double *adv)
{
    for (int64_t p = 0; p < P; ++p) {
        const double *r = reward + p * G;
        double *a = adv + p * G;
        double mean = 0.0;
        for (int32_t i = 0; i < G; ++i) mean += r[i];
        mean /= G;
        double ss = 0.0;
        for (int32_t i = 0; i < G; ++i) ss += (r[i] - mean) * (r[i] - mean);
        const double sd = G > 1 ? sqrt(ss / (G - 1)) : 0.0;
        for (int32_t i = 0; i < G; ++i) a[i] = sd > 0.0 ? (r[i] - mean) / sd : 0.0;
    }
    return 0;
}

int oracle_grpo_surrogate(int64_t R, int64_t P, int32_t G,
                          const double *logp_new, const double *logp_old,
                          const int32_t *seq, const double *adv, double eps,
                          double *loss, double *grad)
{
    const int64_t S = P * G;
    int64_t *count = (int64_t *)calloc((size_t)(S > 0 ? S : 1), sizeof(int64_t));
    if (!count) return 1;
    for (int64_t r = 0; r < R; ++r)
        if (seq[r] >= 0 && seq[r] < S) count[seq[r]] += 1;
    double total = 0.0;
    for (int64_t r = 0; r < R; ++r) {
        const int32_t i = seq[r];
        grad[r] = 0.0;
        if (i < 0 || i >= S) continue;
        const double rho = exp(logp_new[r] - logp_old[r]);
        const double clipped = rho < 1.0 - eps ? 1.0 - eps : (rho > 1.0 + eps ? 1.0 + eps : rho);
        const double u = rho * adv[i], c = clipped * adv[i];
        const double w = 1.0 / ((double)P * G * (double)count[i]);
        total += (u <= c ? u : c) * w;
        grad[r] = u <= c ? -w * rho * adv[i] : 0.0;
    }
    *loss = -total;
    free(count);
    return 0;
}

int oracle_token_logprob_backward(int64_t R, int32_t H, int32_t V,
                                  const uint16_t *hidden, const uint16_t *w_lm,
                                  const int32_t *target, float inv_temperature,
                                  const double *grad_logprob, double *grad_hidden)
{
    const double inv_T = (double)inv_temperature;
    int failed = 0;

#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < R; ++r) {
        double *dh = grad_hidden + r * (int64_t)H;
        const int32_t t = target[r];
        if (t == -1) {
            for (int32_t k = 0; k < H; ++k) dh[k] = 0.0;
            continue;
        }
        if (t < 0 || t >= V) {
            for (int32_t k = 0; k < H; ++k) dh[k] = NAN;
            continue;
        }
        double *z = (double *)malloc((size_t)V * sizeof(double));
        double *h = (double *)malloc((size_t)H * sizeof(double));
        if (!z || !h) {
#pragma omp atomic write
            failed = 1;
            free(z);
            free(h);
            continue;
        }
        const uint16_t *hr = hidden + r * (int64_t)H;
        for (int32_t k = 0; k < H; ++k) h[k] = bf16_to_f64(hr[k]);
        const double l = row_logits(H, V, h, w_lm, inv_T, z);
        /* expected weight row under the softmax, then the target row */
        for (int32_t k = 0; k < H; ++k) dh[k] = 0.0;
        for (int32_t v = 0; v < V; ++v) {
            const double pv = exp(z[v] - l);
            const uint16_t *wr = w_lm + (int64_t)v * H;
            for (int32_t k = 0; k < H; ++k) dh[k] -= pv * bf16_to_f64(wr[k]);
        }
        const uint16_t *wt = w_lm + (int64_t)t * H;
        const double scale = grad_logprob[r] * inv_T;
        for (int32_t k = 0; k < H; ++k) dh[k] = scale * (bf16_to_f64(wt[k]) + dh[k]);
        free(z);
        free(h);
    }
    return failed;
}

/* ---- 6. nucleus sampling --------------------------------------------- */

typedef struct {
    double y;
    int32_t v;
} ranked_token;

/* Larger logit first (same order as p), equal logits by the smaller id. */
static int rank_cmp(const void *a, const void *b)
{
    const ranked_token *x = (const ranked_token *)a, *y = (const ranked_token *)b;
    if (x->y > y->y) return -1;
    if (x->y < y->y) return 1;
    return (x->v > y->v) - (x->v < y->v);
}

/* The nucleus of one row: logits y (and their lse), the ranking rk, the
 * member flags in_n, and, through the out-pointers, the mass before and at
 * the last member and the member count. */
static double row_nucleus(int32_t H, int32_t V, const uint16_t *hr, const uint16_t *w_lm, double inv_T,
                          double top_p, double *h, double *y, ranked_token *rk, unsigned char *in_n,
                          double *before_out, double *cum_out, int32_t *n_out)
{
    for (int32_t k = 0; k < H; ++k) h[k] = bf16_to_f64(hr[k]);
    const double lse = row_logits(H, V, h, w_lm, inv_T, y);
    for (int32_t v = 0; v < V; ++v) {
        rk[v].y = y[v];
        rk[v].v = v;
        in_n[v] = 0;
    }
    qsort(rk, (size_t)V, sizeof(ranked_token), rank_cmp);
    double before = 0.0, cum = 0.0;
    int32_t n = 0;
    while (n < V) {
        before = cum;
        cum += exp(rk[n].y - lse);
        in_n[rk[n].v] = 1;
        ++n;
        if (cum >= top_p) break;
    }
    *before_out = before;
    *cum_out = cum;
    *n_out = n;
    return lse;
}

int oracle_sample_top_p(int64_t R, int32_t H, int32_t V,
                        const uint16_t *hidden, const uint16_t *w_lm,
                        const float *inv_temperature, double top_p,
                        const double *uniform, int32_t *token,
                        double *logprob, double *margin)
{
    int failed = 0;

#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < R; ++r) {
        double *y = (double *)malloc((size_t)V * sizeof(double));
        double *h = (double *)malloc((size_t)H * sizeof(double));
        ranked_token *rk = (ranked_token *)malloc((size_t)V * sizeof(ranked_token));
        unsigned char *in_n = (unsigned char *)malloc((size_t)V);
        if (!y || !h || !rk || !in_n) {
#pragma omp atomic write
            failed = 1;
            free(y);
            free(h);
            free(rk);
            free(in_n);
            continue;
        }
        double before, cum;
        int32_t n;
        const double lse = row_nucleus(H, V, hidden + r * (int64_t)H, w_lm, (double)inv_temperature[r], top_p,
                                       h, y, rk, in_n, &before, &cum, &n);
        /* how close the nucleus is to changing (top_p < 1 only: with
           top_p = 1 every token is in): the mass just before and at the last
           member, and the gap between the last member and the next token */
        double nm = INFINITY;
        if (top_p < 1.0) {
            nm = fmin(top_p - before, cum - top_p);
            if (n < V) nm = fmin(nm, exp(rk[n - 1].y - lse) - exp(rk[n].y - lse));
        }
        /* what such a change could move: the last member and the next token */
        const int32_t last = rk[n - 1].v, next = n < V ? rk[n].v : -1;
        double bmass = exp(rk[n - 1].y - lse) + (n < V ? exp(rk[n].y - lse) : 0.0);

        /* inverse CDF of the renormalised nucleus, in id order */
        double zn = 0.0;
        for (int32_t v = 0; v < V; ++v)
            if (in_n[v]) zn += exp(y[v] - lse);
        const double target = uniform[r] * zn;
        double acc = 0.0, prev = 0.0;
        int32_t t = -1;
        for (int32_t v = 0; v < V; ++v) {
            if (!in_n[v]) continue;
            prev = acc;
            acc += exp(y[v] - lse);
            t = v;
            if (acc > target) break;
        }
        token[r] = t;
        logprob[r] = y[t] - lse;
        margin[3 * r] = fmin(acc - target, target - prev) / zn;
        margin[3 * r + 1] = nm;
        margin[3 * r + 2] = (t == last || t == next) ? INFINITY : bmass / zn;
        free(y);
        free(h);
        free(rk);
        free(in_n);
    }
    return failed;
}

/* For a given token per row: the range [lo, hi) of u that samples it (its
 * share of the renormalised nucleus, in id order), or lo = hi = -1 if the
 * token is outside the nucleus or not a valid id. */
int oracle_top_p_interval(int64_t R, int32_t H, int32_t V,
                          const uint16_t *hidden, const uint16_t *w_lm,
                          const float *inv_temperature, double top_p,
                          const int32_t *token, double *lo, double *hi)
{
    int failed = 0;

#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < R; ++r) {
        double *y = (double *)malloc((size_t)V * sizeof(double));
        double *h = (double *)malloc((size_t)H * sizeof(double));
        ranked_token *rk = (ranked_token *)malloc((size_t)V * sizeof(ranked_token));
        unsigned char *in_n = (unsigned char *)malloc((size_t)V);
        if (!y || !h || !rk || !in_n) {
#pragma omp atomic write
            failed = 1;
            free(y);
            free(h);
            free(rk);
            free(in_n);
            continue;
        }
        double before, cum;
        int32_t n;
        const double lse = row_nucleus(H, V, hidden + r * (int64_t)H, w_lm, (double)inv_temperature[r], top_p,
                                       h, y, rk, in_n, &before, &cum, &n);
        const int32_t t = token[r];
        lo[r] = -1.0;
        hi[r] = -1.0;
        if (t >= 0 && t < V && in_n[t]) {
            double zn = 0.0, below = 0.0;
            for (int32_t v = 0; v < V; ++v) {
                if (!in_n[v]) continue;
                const double pv = exp(y[v] - lse);
                if (v < t) below += pv;
                zn += pv;
            }
            lo[r] = below / zn;
            hi[r] = (below + exp(y[t] - lse)) / zn;
        }
        free(y);
        free(h);
        free(rk);
        free(in_n);
    }
    return failed;
}

/* Definition 7.  Returns 0 on success, 1 if a scratch allocation failed, 2
 * if some n_s exceeds Ls. */
int oracle_extend_attn(int32_t P, int32_t G, int32_t Hq, int32_t Hkv, int32_t D,
                       float scale,
                       const int64_t *prefix_start, const int32_t *prefix_len,
                       const int64_t *suffix_start, const int32_t *suffix_len,
                       const int32_t *new_len, const int64_t *q_start,
                       const uint16_t *q,
                       const uint16_t *k_prefix, const uint16_t *v_prefix,
                       const uint16_t *k_suffix, const uint16_t *v_suffix,
                       double *out, double *lse)
{
    const int64_t n_cand = (int64_t)P * G;
    const int32_t heads_per_kv = Hq / Hkv;
    int failed = 0;

    for (int64_t c = 0; c < n_cand; ++c)
        if (new_len[c] < 0 || new_len[c] > suffix_len[c]) return 2;

#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t c = 0; c < n_cand; ++c) {
        for (int32_t head = 0; head < Hq; ++head) {
            const int64_t prompt = c / G;
            const int32_t kv_head = head / heads_per_kv;
            const int64_t n_pre = prefix_len[prompt];
            const int64_t n_suf = suffix_len[c];
            const int64_t n_new = new_len[c];
            double *score = (double *)malloc((size_t)(n_pre + n_suf + 1) * sizeof(double));
            if (!score) {
#pragma omp atomic write
                failed = 1;
                continue;
            }
            for (int64_t i = 0; i < n_new; ++i) {
                const int64_t qrow = q_start[c] + i;
                const uint16_t *qi = q + (qrow * Hq + head) * (int64_t)D;
                double *oi = out + (qrow * Hq + head) * (int64_t)D;
                /* new token i sits at position n_pre + n_suf - n_new + i of
                 * prefix ++ suffix and sees positions 0 .. itself */
                const int64_t visible = n_pre + (n_suf - n_new + i) + 1;
                for (int64_t j = 0; j < visible; ++j) {
                    const uint16_t *kj = (j < n_pre)
                        ? k_prefix + ((prefix_start[prompt] + j) * Hkv + kv_head) * (int64_t)D
                        : k_suffix + ((suffix_start[c] + (j - n_pre)) * Hkv + kv_head) * (int64_t)D;
                    double qk = 0.0;
                    for (int32_t d = 0; d < D; ++d) qk += bf16_to_f64(qi[d]) * bf16_to_f64(kj[d]);
                    score[j] = (double)scale * qk;
                }
                double mx = score[0];
                for (int64_t j = 1; j < visible; ++j) if (score[j] > mx) mx = score[j];
                double zsum = 0.0;
                for (int64_t j = 0; j < visible; ++j) zsum += exp(score[j] - mx);
                for (int32_t d = 0; d < D; ++d) oi[d] = 0.0;
                for (int64_t j = 0; j < visible; ++j) {
                    const uint16_t *vj = (j < n_pre)
                        ? v_prefix + ((prefix_start[prompt] + j) * Hkv + kv_head) * (int64_t)D
                        : v_suffix + ((suffix_start[c] + (j - n_pre)) * Hkv + kv_head) * (int64_t)D;
                    const double wj = exp(score[j] - mx) / zsum;
                    for (int32_t d = 0; d < D; ++d) oi[d] += wj * bf16_to_f64(vj[d]);
                }
                lse[qrow * Hq + head] = mx + log(zsum);
            }
            free(score);
        }
    }
    return failed;
}
