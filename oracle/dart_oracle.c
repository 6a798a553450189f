/* DART policy-update oracle: a plain, slow, float64 CPU implementation.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may link, load or call
 * this file; it exists so that the HIP kernels can be checked against an
 * independent, obviously correct reading of the paper. It shares no source,
 * header, helper or table with the HIP path.
 *
 * Paper: "Efficient Multi-turn RL for GUI Agents via Decoupled Training and
 * Adaptive Data Curation" (DART), arXiv 2509.23866.
 *
 * Every quantity is computed from its plain definition, in the order the paper
 * states it, with two-pass formulas (max, then sums) and no fusion:
 *   token entropy and log-prob ........ Sec. 4.3 (definition of H_{t,i} and p)
 *                                        and Eq. (1) (the ratio's numerator)
 *   step entropy (mean over tokens) .... Sec. 4.3 (definition of H_t)
 *   high-entropy step mask ............. Sec. 4.3 (the highest-entropy 80% of steps) and the
 *                                        indicator of Eq. (2)
 *   TIS weight ......................... Sec. 4.4 (truncated ratio of the
 *                                        trainer's to the rollout policy, cap C)
 *   clipped surrogate .................. Eq. (1) and Eq. (2)
 *   gradient w.r.t. the logits ......... chain rule through log pi_theta in Eq. (2)
 * Where the paper is silent, the reading taken is stated at its point of use
 * below.
 *
 * Inputs are the exact float32 / bfloat16 values the GPU sees, widened to
 * double. Build: gcc -O2 -fopenmp (no -ffast-math: IEEE semantics are kept). */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Compensated (Neumaier) summation. The normaliser of a near-one-hot row adds
 * ~1.5e5 terms of 1e-13 onto 1.0; a plain double sum would lose ~1e-3 of their
 * total, which is exactly 1 - p_target. With compensation the error of a sum
 * stays a few ulps whatever its length. */
typedef struct { double sum, comp; } ksum_t;

static inline void ksum_add(ksum_t* k, double x) {
    const double t = k->sum + x;
    if (fabs(k->sum) >= fabs(x))
        k->comp += (k->sum - t) + x;
    else
        k->comp += (x - t) + k->sum;
    k->sum = t;
}

static inline double ksum_value(const ksum_t* k) { return k->sum + k->comp; }

/* Logit element (t, v) widened exactly to double. dtype 0 = float32,
 * dtype 1 = bfloat16 stored as its 16-bit pattern, dtype 2 = float64 (logits
 * the oracle formed itself, e.g. from an LM head in double). */
static double logit_at(const void* z, int dtype, int64_t ld, int64_t t, int64_t v) {
    if (dtype == 0) return (double)((const float*)z)[t * ld + v];
    if (dtype == 2) return ((const double*)z)[t * ld + v];
    uint32_t bits = (uint32_t)((const uint16_t*)z)[t * ld + v] << 16;
    float f;
    memcpy(&f, &bits, 4);
    return (double)f;
}

/* Sec. 4.3: p_v = softmax(z)_v, H = -sum_v p_v log p_v (nats: the natural log),
 * and log pi(y) = z_y - log sum_v exp(z_v) for the target id y (Eq. 1 numerator).
 * The logits are first multiplied by inv_temp (an inverse sampling temperature;
 * 1 in the paper, App. A.4). Per row: (1) the maximum m; (2) e_v = exp(z_v - m)
 * and their sum s, so that lse = m + log s; (3) p_v = e_v / s and
 * log p_v = (z_v - m) - log s, summed into the entropy from its definition. A term with
 * p_v == 0 contributes 0 (a reading: -inf logits allowed, 0 log 0 := 0). */
void oracle_token_stats_ex(const void* z, int dtype, int64_t nrows, int64_t V, int64_t ld,
                           const int32_t* target, double inv_temp, double* logp, double* H,
                           double* lse, int nthreads) {
    if (nthreads < 1) nthreads = 1;
#pragma omp parallel num_threads(nthreads)
    {
        double* e = (double*)malloc((size_t)V * sizeof(double));
#pragma omp for schedule(dynamic, 1)
        for (int64_t t = 0; t < nrows; ++t) {
            double m = -INFINITY;
            for (int64_t v = 0; v < V; ++v) {
                double x = inv_temp * logit_at(z, dtype, ld, t, v);
                if (x > m) m = x;
            }
            ksum_t s = {0.0, 0.0};
            for (int64_t v = 0; v < V; ++v) {
                e[v] = exp(inv_temp * logit_at(z, dtype, ld, t, v) - m);
                ksum_add(&s, e[v]);
            }
            const double sum = ksum_value(&s);
            /* log s without rounding s: the largest term is exp(0) = 1, so
             * s - 1 = (sum - 1) + compensation is exact to the compensation's
             * accuracy and log s = log1p(s - 1) keeps full relative accuracy
             * even when s - 1 ~ 1e-11 (a near-one-hot row) */
            const double log_s = log1p((s.sum - 1.0) + s.comp);
            ksum_t h = {0.0, 0.0};
            for (int64_t v = 0; v < V; ++v) {
                const double p = e[v] / sum;
                const double log_p = (inv_temp * logit_at(z, dtype, ld, t, v) - m) - log_s;
                if (p > 0.0) ksum_add(&h, -p * log_p);
            }
            lse[t] = m + log_s;
            H[t] = ksum_value(&h);
            logp[t] = (inv_temp * logit_at(z, dtype, ld, t, target[t]) - m) - log_s;
        }
        free(e);
    }
}

void oracle_token_stats(const void* z, int dtype, int64_t nrows, int64_t V, int64_t ld,
                        const int32_t* target, double* logp, double* H, double* lse,
                        int nthreads) {
    oracle_token_stats_ex(z, dtype, nrows, V, ld, target, 1.0, logp, H, lse, nthreads);
}

/* Sec. 4.3: the step entropy is the mean of the token entropies over the
 * step's tokens (thought and action concatenated); step s = tokens
 * [off[s], off[s+1]). The mean is taken in double; the selection below decides
 * on it rounded to float32 (a reading: the decision is taken in the kernel's
 * precision). */
void oracle_step_entropy(const double* H, const int32_t* off, int64_t S, double* Hs,
                         float* Hs32) {
    for (int64_t s = 0; s < S; ++s) {
        ksum_t sum = {0.0, 0.0};
        for (int64_t t = off[s]; t < off[s + 1]; ++t) ksum_add(&sum, H[t]);
        Hs[s] = ksum_value(&sum) / (double)(off[s + 1] - off[s]);
        Hs32[s] = (float)Hs[s];
    }
}

/* Reading: number of kept steps k = ceil(rho * S), computed in double with a
 * 1e-6 guard against representation error of rho (0.8 * 240 must give 192),
 * clamped to [0, S]. */
int64_t oracle_kept_steps(int64_t S, double rho) {
    double k = ceil(rho * (double)S - 1e-6);
    if (k < 0.0) k = 0.0;
    if (k > (double)S) k = (double)S;
    return (int64_t)k;
}

/* Sec. 4.3 / Eq. (2): keep the k highest-entropy steps of the group. Reading: the
 * rank of step s counts the steps that beat it, a step with equal entropy and
 * a lower index beating it; s is kept iff its rank is below k. O(S^2), no
 * sorting. Returns k. */
int64_t oracle_step_mask(const float* Hs32, int64_t S, double rho, uint8_t* mask) {
    const int64_t k = oracle_kept_steps(S, rho);
    for (int64_t s = 0; s < S; ++s) {
        int64_t rank = 0;
        for (int64_t o = 0; o < S; ++o) {
            if (Hs32[o] > Hs32[s] || (Hs32[o] == Hs32[s] && o < s)) ++rank;
        }
        mask[s] = rank < k ? 1 : 0;
    }
    return k;
}

/* KL estimators of D_KL(pi_theta || pi_ref) from the sampled token, with
 * delta = log pi_ref - log pi_theta (the paper leaves the estimator unstated;
 * k3 is the one GRPO uses): k1 = -delta, k2 = delta^2 / 2,
 * k3 = exp(delta) - delta - 1, and their derivatives w.r.t. log pi_theta. */
enum { KL_NONE = 0, KL_K1 = 1, KL_K2 = 2, KL_K3 = 3 };
enum { AGG_TOKEN_MEAN = 0, AGG_TOKEN_MEAN_ALL = 1, AGG_STEP_MEAN = 2 };
enum { RATIO_TOKEN = 0, RATIO_STEP_GEOMEAN = 1, RATIO_STEP_PRODUCT = 2 };

static double kl_value(int kl, double delta) {
    if (kl == KL_K1) return -delta;
    if (kl == KL_K2) return 0.5 * delta * delta;
    if (kl == KL_K3) return exp(delta) - delta - 1.0;
    return 0.0;
}

static double kl_dlogp(int kl, double delta) {
    if (kl == KL_K1) return 1.0;
    if (kl == KL_K2) return -delta;
    if (kl == KL_K3) return 1.0 - exp(delta);
    return 0.0;
}

/* Eq. (2), per token t of step s(t), as the loss L = -J (a reading):
 *   r  = pi_theta / pi_old            = exp(logp - lp_old)             (Eq. 1)
 *   w  = min(pi_old / pi_rollout, C)  = min(exp(lp_old - lp_roll), C)  (Sec. 4.4)
 *   u  = r A,  c = clip(r, 1 - eps_low, 1 + eps_high) A,  o = min(u, c)
 *   l_t = -M_s om_t (w o - beta kl_t)
 *   L  = sum_t l_t
 * om_t is the aggregation weight: 1/N with N the tokens of kept steps (the
 * default reading), 1/T over all tokens, or 1/(K |s|) for the mean over the K kept
 * steps of each step's token mean. With a step-level ratio (Eq. 1 written for
 * the whole action) r, w and A are taken per step: log r_s and log w_s are the
 * sum (product ratio) or mean (geometric-mean ratio) of the token log-ratios, A_s
 * the mean advantage of the step, and every token of the step carries the
 * step's w_s o_s.
 *   g_t = dL/dlogp_t = -M (om_t w d o/dlogp_t - om_t beta dkl_t/dlogp_t), where
 * d o / d logp_t = r A when u <= c (the unclipped branch is the minimum) and 0
 * when u > c (the clipped branch is a constant, a reading); in step mode the step
 * term differentiates through log r_s, whose derivative w.r.t. logp_t is 1
 * (product) or 1/|s| (geometric mean), and the step's weights sum to
 * Om_s = sum_{t in s} om_t. w, M, N, K are constants (a reading). The KL term sits
 * inside the indicator and outside the TIS weight, as in Eq. (2).
 * boundary[t] = 1 marks tokens whose gate may legitimately differ between
 * precisions: A != 0 and the ratio within 1e-4 (relative) of a clip bound.
 * stats[6]: clip fraction, mean TIS
 * weight, fraction of weights at the cap, N, mean KL, K (over kept tokens /
 * steps; zeros when nothing is kept). Returns L. */
double oracle_tis_loss_ex(int64_t T, const double* logp, const float* lp_old,
                          const float* lp_roll, const float* lp_ref, const float* adv,
                          const int32_t* off, int64_t S, const uint8_t* mask, double eps_low,
                          double eps_high, double C, int kl, double beta, int agg, int ratio,
                          double* g, double* ell, uint8_t* boundary, double* stats) {
    int64_t N = 0, K = 0;
    for (int64_t s = 0; s < S; ++s)
        if (mask[s]) {
            N += off[s + 1] - off[s];
            K += 1;
        }
    ksum_t L = {0.0, 0.0};
    double n_clip = 0.0, sum_w = 0.0, n_cap = 0.0, sum_kl = 0.0;
    for (int64_t s = 0; s < S; ++s) {
        const int64_t len = off[s + 1] - off[s];
        const double M = mask[s] ? 1.0 : 0.0;
        double om = 0.0;
        if (agg == AGG_TOKEN_MEAN) om = N > 0 ? 1.0 / (double)N : 0.0;
        if (agg == AGG_TOKEN_MEAN_ALL) om = 1.0 / (double)T;
        if (agg == AGG_STEP_MEAN) om = K > 0 ? 1.0 / ((double)K * (double)len) : 0.0;
        /* step-level ratio, TIS weight and advantage */
        double r_s = 0.0, w_s = 0.0, A_s = 0.0, ratio_tis_s = 0.0;
        if (ratio != RATIO_TOKEN) {
            double lr = 0.0, lw = 0.0, sa = 0.0;
            for (int64_t t = off[s]; t < off[s + 1]; ++t) {
                lr += logp[t] - (double)lp_old[t];
                lw += (double)lp_old[t] - (double)lp_roll[t];
                sa += (double)adv[t];
            }
            if (ratio == RATIO_STEP_GEOMEAN) {
                lr /= (double)len;
                lw /= (double)len;
            }
            r_s = exp(lr);
            ratio_tis_s = exp(lw);
            w_s = ratio_tis_s < C ? ratio_tis_s : C;
            A_s = sa / (double)len;
        }
        for (int64_t t = off[s]; t < off[s + 1]; ++t) {
            double r, w, A, ratio_tis, dlog = 1.0, om_obj = om;
            if (ratio == RATIO_TOKEN) {
                A = (double)adv[t];
                r = exp(logp[t] - (double)lp_old[t]);
                ratio_tis = exp((double)lp_old[t] - (double)lp_roll[t]);
                w = ratio_tis < C ? ratio_tis : C;
            } else {
                A = A_s;
                r = r_s;
                ratio_tis = ratio_tis_s;
                w = w_s;
                om_obj = om * (double)len; /* Om_s: the step term's weight */
                dlog = ratio == RATIO_STEP_GEOMEAN ? 1.0 / (double)len : 1.0;
            }
            double rc = r;
            if (rc < 1.0 - eps_low) rc = 1.0 - eps_low;
            if (rc > 1.0 + eps_high) rc = 1.0 + eps_high;
            const double u = r * A;
            const double c = rc * A;
            const double o = u < c ? u : c;
            double klv = 0.0, kld = 0.0;
            if (kl != KL_NONE) {
                const double delta = (double)lp_ref[t] - logp[t];
                klv = kl_value(kl, delta);
                kld = kl_dlogp(kl, delta);
            }
            const double lt = -M * om * (w * o - beta * klv);
            const double d_obj = u <= c ? r * A * dlog : 0.0;
            const double gt = -M * (om_obj * w * d_obj - om * beta * kld);
            if (ell) ell[t] = lt;
            if (g) g[t] = gt;
            /* The gate u <= c can flip between precisions only when the ratio sits
             * at a clip bound (inside the range clip(r) = r and u == c exactly) */
            if (boundary)
                boundary[t] = A != 0.0 && (fabs(r - (1.0 - eps_low)) <= 1e-4 * (1.0 - eps_low) ||
                                           fabs(r - (1.0 + eps_high)) <= 1e-4 * (1.0 + eps_high))
                                  ? 1
                                  : 0;
            ksum_add(&L, lt);
            if (mask[s]) {
                n_clip += u > c ? 1.0 : 0.0;
                sum_w += w;
                n_cap += ratio_tis >= C ? 1.0 : 0.0;
                sum_kl += klv;
            }
        }
    }
    if (stats) {
        stats[0] = N > 0 ? n_clip / (double)N : 0.0;
        stats[1] = N > 0 ? sum_w / (double)N : 0.0;
        stats[2] = N > 0 ? n_cap / (double)N : 0.0;
        stats[3] = (double)N;
        stats[4] = N > 0 ? sum_kl / (double)N : 0.0;
        stats[5] = (double)K;
    }
    return ksum_value(&L);
}

/* The paper's default configuration: Eq. (2) without the KL term,
 * per-token ratios, token mean over kept tokens (readings); stats[4]. */
double oracle_tis_loss(int64_t T, const double* logp, const float* lp_old, const float* lp_roll,
                       const float* adv, const int32_t* off, int64_t S, const uint8_t* mask,
                       double eps_low, double eps_high, double C, double* g, double* ell,
                       uint8_t* boundary, double* stats) {
    double st[6];
    const double L = oracle_tis_loss_ex(T, logp, lp_old, lp_roll, NULL, adv, off, S, mask,
                                        eps_low, eps_high, C, KL_NONE, 0.0, AGG_TOKEN_MEAN,
                                        RATIO_TOKEN, g, ell, boundary, st);
    if (stats)
        for (int i = 0; i < 4; ++i) stats[i] = st[i];
    return L;
}

/* Gradient of L w.r.t. the logits: dL/dz_{t,v} = g_t * d logp_t / d z_{t,v}
 * = inv_temp * g_t * (delta_{v, y_t} - p_{t,v}), with p = exp(inv_temp z - lse)
 * (softmax derivative, and the chain rule through z -> inv_temp z). Rows are the
 * same rows as z (nrows of them); out is [nrows, V] double. */
void oracle_dlogits_ex(const void* z, int dtype, int64_t nrows, int64_t V, int64_t ld,
                       const int32_t* target, const double* lse, const double* logp,
                       const double* g, double inv_temp, double* out, int nthreads) {
    if (nthreads < 1) nthreads = 1;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
    for (int64_t t = 0; t < nrows; ++t) {
        for (int64_t v = 0; v < V; ++v) {
            const double p = exp(inv_temp * logit_at(z, dtype, ld, t, v) - lse[t]);
            const double delta = v == target[t] ? 1.0 : 0.0;
            out[t * V + v] = inv_temp * g[t] * (delta - p);
        }
        /* at the target 1 - p_y = -expm1(log p_y): exact where p_y -> 1, where
         * 1 - exp(z_y - lse) would keep only the digits lse has below its
         * integer part */
        const int64_t y = target[t];
        out[t * V + y] = inv_temp * g[t] * -expm1(logp[t]);
    }
}

void oracle_dlogits(const void* z, int dtype, int64_t nrows, int64_t V, int64_t ld,
                    const int32_t* target, const double* lse, const double* logp, const double* g,
                    double* out, int nthreads) {
    oracle_dlogits_ex(z, dtype, nrows, V, ld, target, lse, logp, g, 1.0, out, nthreads);
}

/* Sec. 3.3, step-wise GRPO advantage. The step group D of a task holds every
 * step of its N trajectories, each step carrying its trajectory's reward R_i.
 * Over D: Rbar = (1/|D|) sum R, sigma^2 = (1/|D|) sum (R - Rbar)^2 (population
 * variance, as written), and every step (i, j) gets A = (R_i - Rbar) / sigma;
 * every token of the step carries it. A guard: sigma == 0 (all rewards
 * equal; the data manager excludes such groups) gives A = 0.
 * Layout: trajectories [grp_off[g], grp_off[g+1]) form group g; steps
 * [traj_off[i], traj_off[i+1]) form trajectory i; tokens [off[s], off[s+1])
 * form step s. adv is [T]; group_mean / group_std are [G] (or NULL). */
void oracle_grpo_advantage(const float* reward, const int32_t* traj_off, int64_t n_traj,
                           const int32_t* grp_off, int64_t G, const int32_t* off, double* adv,
                           double* group_mean, double* group_std) {
    (void)n_traj;
    for (int64_t g = 0; g < G; ++g) {
        /* walk the steps of the group: D as a list of rewards */
        ksum_t sum = {0.0, 0.0};
        int64_t count = 0;
        for (int64_t i = grp_off[g]; i < grp_off[g + 1]; ++i)
            for (int64_t s = traj_off[i]; s < traj_off[i + 1]; ++s) {
                ksum_add(&sum, (double)reward[i]);
                ++count;
            }
        const double mean = count > 0 ? ksum_value(&sum) / (double)count : 0.0;
        ksum_t sq = {0.0, 0.0};
        for (int64_t i = grp_off[g]; i < grp_off[g + 1]; ++i)
            for (int64_t s = traj_off[i]; s < traj_off[i + 1]; ++s) {
                const double d = (double)reward[i] - mean;
                ksum_add(&sq, d * d);
            }
        const double sd = count > 0 ? sqrt(ksum_value(&sq) / (double)count) : 0.0;
        if (group_mean) group_mean[g] = mean;
        if (group_std) group_std[g] = sd;
        for (int64_t i = grp_off[g]; i < grp_off[g + 1]; ++i) {
            const double a = sd > 0.0 ? ((double)reward[i] - mean) / sd : 0.0;
            for (int64_t s = traj_off[i]; s < traj_off[i + 1]; ++s)
                for (int64_t t = off[s]; t < off[s + 1]; ++t) adv[t] = a;
        }
    }
}
