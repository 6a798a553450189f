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
 *   high-entropy step mask ............. Sec. 4.3 ("top 80%" of steps) and the
 *                                        indicator of Eq. (2)
 *   TIS weight ......................... Sec. 4.4 (truncated ratio of the
 *                                        trainer's to the rollout policy, cap C)
 *   clipped surrogate .................. Eq. (1) and Eq. (2)
 *   gradient w.r.t. the logits ......... chain rule through log pi_theta in Eq. (2)
 * Readings where the paper is silent are listed in the design doc (R1..R12) and are
 * named at the point of use below.
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
 * dtype 1 = bfloat16 stored as its 16-bit pattern. */
static double logit_at(const void* z, int dtype, int64_t ld, int64_t t, int64_t v) {
    if (dtype == 0) return (double)((const float*)z)[t * ld + v];
    uint32_t bits = (uint32_t)((const uint16_t*)z)[t * ld + v] << 16;
    float f;
    memcpy(&f, &bits, 4);
    return (double)f;
}

/* Sec. 4.3: p_v = softmax(z)_v, H = -sum_v p_v log p_v (nats, R10: natural log),
 * and log pi(y) = z_y - log sum_v exp(z_v) for the target id y (Eq. 1 numerator).
 * Per row: (1) the maximum m; (2) e_v = exp(z_v - m) and their sum s, so that
 * lse = m + log s; (3) p_v = e_v / s and log p_v = z_v - lse, summed into the
 * entropy from its definition. A term with p_v == 0 contributes 0 (R9: -inf
 * logits allowed, 0 log 0 := 0). */
void oracle_token_stats(const void* z, int dtype, int64_t nrows, int64_t V, int64_t ld,
                        const int32_t* target, double* logp, double* H, double* lse,
                        int nthreads) {
    if (nthreads < 1) nthreads = 1;
#pragma omp parallel num_threads(nthreads)
    {
        double* e = (double*)malloc((size_t)V * sizeof(double));
#pragma omp for schedule(dynamic, 1)
        for (int64_t t = 0; t < nrows; ++t) {
            double m = -INFINITY;
            for (int64_t v = 0; v < V; ++v) {
                double x = logit_at(z, dtype, ld, t, v);
                if (x > m) m = x;
            }
            ksum_t s = {0.0, 0.0};
            for (int64_t v = 0; v < V; ++v) {
                e[v] = exp(logit_at(z, dtype, ld, t, v) - m);
                ksum_add(&s, e[v]);
            }
            const double sum = ksum_value(&s);
            const double log_norm = m + log(sum);
            ksum_t h = {0.0, 0.0};
            for (int64_t v = 0; v < V; ++v) {
                const double p = e[v] / sum;
                const double log_p = logit_at(z, dtype, ld, t, v) - log_norm;
                if (p > 0.0) ksum_add(&h, -p * log_p);
            }
            lse[t] = log_norm;
            H[t] = ksum_value(&h);
            logp[t] = logit_at(z, dtype, ld, t, target[t]) - log_norm;
        }
        free(e);
    }
}

/* Sec. 4.3: the step entropy is the mean of the token entropies over the
 * step's tokens (thought and action concatenated); step s = tokens
 * [off[s], off[s+1]). The mean is taken in double; the selection below decides
 * on it rounded to float32 (R4: the decision is taken in the kernel's
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

/* R3: number of kept steps k = ceil(rho * S), computed in double with a
 * 1e-6 guard against representation error of rho (0.8 * 240 must give 192),
 * clamped to [0, S]. */
int64_t oracle_kept_steps(int64_t S, double rho) {
    double k = ceil(rho * (double)S - 1e-6);
    if (k < 0.0) k = 0.0;
    if (k > (double)S) k = (double)S;
    return (int64_t)k;
}

/* Sec. 4.3 / Eq. (2): keep the k highest-entropy steps of the group. R3: the
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

/* Eq. (2) without the KL term (R7), per token t of step s(t):
 *   r  = pi_theta / pi_old            = exp(logp - lp_old)             (Eq. 1)
 *   w  = min(pi_old / pi_rollout, C)  = min(exp(lp_old - lp_roll), C)  (Sec. 4.4)
 *   u  = r A,  c = clip(r, 1 - eps_low, 1 + eps_high) A,  o = min(u, c)
 *   l_t = -M_s w o / N,   N = number of tokens in kept steps (R1: token mean)
 *   L  = sum_t l_t        (the loss is the negated objective)
 *   g_t = dL/dlogp_t = -(M_s w / N) * d o / d logp_t, and d o / d logp_t = r A
 *         when u <= c (the unclipped branch is the minimum), 0 when u > c (the
 *         clipped branch is a constant) (R6; w, M and N are constants, R5).
 * Per-token ratios, weights and clips (R2). If N == 0, L = 0 and g = 0 (R8).
 * boundary[t] = 1 marks tokens with |u - c| <= 1e-6 max(1, |A|), where the gate
 * of g may legitimately differ between precisions. stats: clip fraction, mean
 * TIS weight, fraction of weights at the cap, N (all over kept tokens; zeros
 * if N == 0). Returns L. */
double oracle_tis_loss(int64_t T, const double* logp, const float* lp_old, const float* lp_roll,
                       const float* adv, const int32_t* off, int64_t S, const uint8_t* mask,
                       double eps_low, double eps_high, double C, double* g, double* ell,
                       uint8_t* boundary, double* stats) {
    int64_t N = 0;
    for (int64_t s = 0; s < S; ++s)
        if (mask[s]) N += off[s + 1] - off[s];
    ksum_t L = {0.0, 0.0};
    double n_clip = 0.0, sum_w = 0.0, n_cap = 0.0;
    for (int64_t s = 0; s < S; ++s) {
        for (int64_t t = off[s]; t < off[s + 1]; ++t) {
            const double M = mask[s] ? 1.0 : 0.0;
            const double A = (double)adv[t];
            const double r = exp(logp[t] - (double)lp_old[t]);
            const double ratio_tis = exp((double)lp_old[t] - (double)lp_roll[t]);
            const double w = ratio_tis < C ? ratio_tis : C;
            double rc = r;
            if (rc < 1.0 - eps_low) rc = 1.0 - eps_low;
            if (rc > 1.0 + eps_high) rc = 1.0 + eps_high;
            const double u = r * A;
            const double c = rc * A;
            const double o = u < c ? u : c;
            double lt = 0.0, gt = 0.0;
            if (N > 0) {
                lt = -M * w * o / (double)N;
                gt = u <= c ? -M * w * A * r / (double)N : 0.0;
            }
            if (ell) ell[t] = lt;
            if (g) g[t] = gt;
            if (boundary) boundary[t] = fabs(u - c) <= 1e-6 * fmax(1.0, fabs(A)) ? 1 : 0;
            ksum_add(&L, lt);
            if (mask[s]) {
                n_clip += u > c ? 1.0 : 0.0;
                sum_w += w;
                n_cap += ratio_tis >= C ? 1.0 : 0.0;
            }
        }
    }
    if (stats) {
        stats[0] = N > 0 ? n_clip / (double)N : 0.0;
        stats[1] = N > 0 ? sum_w / (double)N : 0.0;
        stats[2] = N > 0 ? n_cap / (double)N : 0.0;
        stats[3] = (double)N;
    }
    return ksum_value(&L);
}

/* Gradient of L w.r.t. the logits: dL/dz_{t,v} = g_t * d logp_t / d z_{t,v}
 * = g_t * (delta_{v, y_t} - p_{t,v}), with p = exp(z - lse) (softmax
 * derivative). Rows are the same rows as z (nrows of them); out is
 * [nrows, V] double. */
void oracle_dlogits(const void* z, int dtype, int64_t nrows, int64_t V, int64_t ld,
                    const int32_t* target, const double* lse, const double* g, double* out,
                    int nthreads) {
    if (nthreads < 1) nthreads = 1;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
    for (int64_t t = 0; t < nrows; ++t) {
        for (int64_t v = 0; v < V; ++v) {
            const double p = exp(logit_at(z, dtype, ld, t, v) - lse[t]);
            const double delta = v == target[t] ? 1.0 : 0.0;
            out[t * V + v] = g[t] * (delta - p);
        }
    }
}
