/*
 * PrunePath sparse-FFN forward -- CPU oracle in fp64.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark use it.  It shares no code, header, table or helper with the
 * HIP library: the two meet only at the seeded bf16 input arrays.
 *
 * Every quantity is computed in double precision from the exact values of the
 * same bf16 bit patterns the GPU path consumes.  The code follows the paper's
 * equations in their own order and notation (Sec. 2.1 and Sec. 3.1):
 *
 *   g = W_r^T x                         Eq. (routing_logits)
 *   p = softmax(g)                      Eq. (softmax_prob)
 *   pi = descending order of p          Sec. 3.1, text after Eq. (softmax_prob)
 *   C_i = sum_{r<=i} p_{pi_r}
 *   A_tau(x) from C and tau             Eq. (tau_thresh_activate), nucleus reading
 *   y = sum_{e in A} [sigmoid(g_e)] FFN_e(x)   Eqs. (moefication_decomp), (moe_output)
 *   FFN_e(x) = (phi(x Wg^(e)) . x Wu^(e)) Wd^(e), phi = SiLU   Eq. (ffn)
 *   non-gated variant (GPT-2 MLP): GELU(x W_fc^(e) + b_fc^(e)) W_proj^(e),
 *   plus b_proj once per token                                  Sec. 2.1
 *
 * Readings of points the paper leaves open (each is listed in the design notes):
 *  - Selection rule.  Default (nucleus): the smallest prefix of pi whose mass
 *    reaches tau; tau >= 1 keeps all E experts (exact-arithmetic result: every
 *    softmax probability is positive).  Flag PPO_SELECT_STRICT: the rule as
 *    printed, {pi_1} U {pi_i : C_i < tau}, with C_E = 1 by definition.
 *    Comparison rules on the same router: PPO_SELECT_TOPK keeps pi_1..pi_k,
 *    k = tau rounded to nearest and clamped to [1, E] (the forced top-k of the
 *    reconstruction analysis); PPO_SELECT_LTE keeps {e : sigmoid(g_e) > tau},
 *    Eq. (lte_hard_set), possibly empty, listed in pi order.
 *  - Ties in the ordering: the lower expert index comes first.  The order is
 *    taken on g, which is equivalent to ordering p (softmax is monotone).
 *  - Aggregation.  Default: plain sum (Eq. moefication_decomp, whose all-expert
 *    case is the dense FFN).  Flag PPO_AGG_SIGMOID: Eq. (moe_output).
 *  - Router extras for the skewed workload: g = (W_r x + b) * inv_temp_t.
 *  - Layouts follow the API: W_r [E,d], W_gate/W_up [d_ff,d], W_down [d,d_ff]
 *    (the paper's matrices transposed).  Expert e owns neurons
 *    perm[e*de .. e*de+de-1] (identity when perm is NULL), de = d_ff / E.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define PPO_SELECT_STRICT 1u
#define PPO_AGG_SIGMOID 2u
#define PPO_SELECT_TOPK 4u
#define PPO_SELECT_LTE 8u

/* Exact value of a bf16 bit pattern: its bits are the top half of an IEEE
 * binary32 number. */
static double bf16_value(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

int ppo_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads of the following parallel regions (n >= 1); used to time the
 * oracle single-threaded next to its all-core run. */
void ppo_set_num_threads(int n) {
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Eq. (routing_logits), one token: g_e = sum_j W_r[e,j] x_j, then the optional
 * per-expert bias and per-token inverse temperature of the skewed workload. */
static void logits_one(int64_t d, int64_t E, const uint16_t *x, const uint16_t *Wr,
                       const float *bias, double inv_temp, double *g) {
    for (int64_t e = 0; e < E; ++e) {
        double s = 0.0;
        const uint16_t *w = Wr + e * d;
        for (int64_t j = 0; j < d; ++j) s += bf16_value(w[j]) * bf16_value(x[j]);
        if (bias) s += (double)bias[e];
        g[e] = s * inv_temp;
    }
}

/* Eq. (softmax_prob).  Subtracting max g leaves the value unchanged. */
void ppo_softmax(int64_t E, const double *g, double *p) {
    double m = g[0];
    for (int64_t e = 1; e < E; ++e)
        if (g[e] > m) m = g[e];
    double z = 0.0;
    for (int64_t e = 0; e < E; ++e) {
        p[e] = exp(g[e] - m);
        z += p[e];
    }
    for (int64_t e = 0; e < E; ++e) p[e] /= z;
}

/* pi: experts in descending order of probability (equivalently of logit);
 * equal logits keep ascending expert index.  Insertion sort, E <= a few
 * hundred. */
void ppo_order(int64_t E, const double *g, int32_t *pi) {
    for (int64_t i = 0; i < E; ++i) {
        int32_t e = (int32_t)i;
        int64_t j = i;
        while (j > 0 && g[pi[j - 1]] < g[e]) {
            pi[j] = pi[j - 1];
            --j;
        }
        pi[j] = e;
    }
}

/* Eq. (tau_thresh_activate): given p already in the order pi, form the
 * cumulative masses C_1..C_E (written to C) and return the number k of
 * selected experts; the selection is always the prefix pi_1..pi_k.
 *
 *  nucleus (default): k = min{i : C_i >= tau}; all E when tau >= 1.
 *  strict:            k = max(1, #{i : C_i < tau}) with C_E taken as exactly 1.
 */
int64_t ppo_cut(int64_t E, const double *p_sorted, double tau, unsigned flags, double *C) {
    double c = 0.0;
    for (int64_t i = 0; i < E; ++i) {
        c += p_sorted[i];
        C[i] = c;
    }
    if (flags & PPO_SELECT_STRICT) {
        int64_t m = 0;
        for (int64_t i = 0; i < E - 1; ++i)
            if (C[i] < tau) ++m;
        if (1.0 < tau) ++m; /* C_E = 1 */
        return m < 1 ? 1 : m;
    }
    if (tau >= 1.0) return E;
    for (int64_t i = 0; i < E; ++i)
        if (C[i] >= tau) return i + 1;
    return E;
}

/* Routing for T tokens.  Outputs per token t (row-major [T,E]):
 *   idx[t, 0..k-1] = pi_1..pi_k (rest -1), count[t] = k,
 *   g[t, e] logits, cum[t, i] = C_{i+1} in the order pi.
 * Returns 0, or -1 on bad arguments. */
int ppo_route(int64_t T, int64_t d, int64_t E, const uint16_t *x, const uint16_t *Wr,
              const float *bias, const float *inv_temp, double tau, unsigned flags,
              int32_t *idx, int32_t *count, double *g, double *cum) {
    if (T < 0 || d < 1 || E < 1 || !x || !Wr || !idx || !count || !g || !cum) return -1;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int64_t t = 0; t < T; ++t) {
        double *gt = g + t * E;
        double *p = (double *)malloc(sizeof(double) * (size_t)E * 2);
        int32_t *pi = (int32_t *)malloc(sizeof(int32_t) * (size_t)E);
        if (!p || !pi) {
            bad = 1;
            free(p);
            free(pi);
            continue;
        }
        double *ps = p + E;
        logits_one(d, E, x + t * d, Wr, bias, inv_temp ? (double)inv_temp[t] : 1.0, gt);
        ppo_softmax(E, gt, p);
        ppo_order(E, gt, pi);
        for (int64_t i = 0; i < E; ++i) ps[i] = p[pi[i]];
        int64_t k = ppo_cut(E, ps, tau, flags, cum + t * E);
        if (flags & PPO_SELECT_TOPK) {
            double r = floor(tau + 0.5);
            k = r < 1.0 ? 1 : (r > (double)E ? E : (int64_t)r);
        } else if (flags & PPO_SELECT_LTE) {
            /* Eq. (lte_hard_set): independent sigmoid scores against delta = tau;
             * the kept experts are the ones ranked first, since sigmoid is
             * increasing */
            k = 0;
            for (int64_t e = 0; e < E; ++e)
                if (1.0 / (1.0 + exp(-gt[e])) > tau) ++k;
        }
        count[t] = (int32_t)k;
        for (int64_t i = 0; i < E; ++i) idx[t * E + i] = i < k ? pi[i] : -1;
        free(p);
        free(pi);
    }
    return bad ? -1 : 0;
}

/* Expert outputs summed over a given selection, Eqs. (moefication_decomp) and
 * (moe_output), with FFN_e from Eq. (ffn) restricted to expert e's neurons:
 *   a_n = Wg[n,:] . x,  b_n = Wu[n,:] . x,  h_n = SiLU(a_n) b_n [* sigmoid(g_e)]
 *   y_i = sum over selected neurons n of Wd[i, n] h_n.
 * idx/count use the layout written by ppo_route (any order of experts is
 * accepted).  g is needed only with PPO_AGG_SIGMOID.  y is [T,d], overwritten.
 * Returns 0, or -1 on bad arguments. */
int ppo_ffn(int64_t T, int64_t d, int64_t d_ff, int64_t E, const uint16_t *x,
            const uint16_t *Wg, const uint16_t *Wu, const uint16_t *Wd, const int32_t *perm,
            const int32_t *idx, const int32_t *count, const double *g, unsigned flags,
            double *y) {
    if (T < 0 || d < 1 || E < 1 || d_ff % E != 0 || !x || !Wg || !Wu || !Wd || !idx || !count ||
        !y)
        return -1;
    if ((flags & PPO_AGG_SIGMOID) && !g) return -1;
    const int64_t de = d_ff / E;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int64_t t = 0; t < T; ++t) {
        const uint16_t *xt = x + t * d;
        double *yt = y + t * d;
        int64_t k = count[t];
        int32_t *nsel = (int32_t *)malloc(sizeof(int32_t) * (size_t)(k * de + 1));
        double *h = (double *)malloc(sizeof(double) * (size_t)(k * de + 1));
        double *xv = (double *)malloc(sizeof(double) * (size_t)d);
        if (!nsel || !h || !xv || k < 0 || k > E) {
            bad = 1;
            free(nsel);
            free(h);
            free(xv);
            continue;
        }
        for (int64_t j = 0; j < d; ++j) xv[j] = bf16_value(xt[j]);
        /* intermediate activations of the selected neurons */
        for (int64_t s = 0; s < k; ++s) {
            int64_t e = idx[t * E + s];
            double scale = 1.0;
            if (flags & PPO_AGG_SIGMOID) scale = 1.0 / (1.0 + exp(-g[t * E + e]));
            for (int64_t r = 0; r < de; ++r) {
                int64_t n = perm ? perm[e * de + r] : e * de + r;
                const uint16_t *wg = Wg + n * d;
                const uint16_t *wu = Wu + n * d;
                double a = 0.0, b = 0.0;
                for (int64_t j = 0; j < d; ++j) {
                    a += bf16_value(wg[j]) * xv[j];
                    b += bf16_value(wu[j]) * xv[j];
                }
                nsel[s * de + r] = (int32_t)n;
                h[s * de + r] = a / (1.0 + exp(-a)) * b * scale;
            }
        }
        /* down projection over the selected neurons */
        for (int64_t i = 0; i < d; ++i) {
            const uint16_t *wd = Wd + i * d_ff;
            double acc = 0.0;
            for (int64_t q = 0; q < k * de; ++q) acc += bf16_value(wd[nsel[q]]) * h[q];
            yt[i] = acc;
        }
        free(nsel);
        free(h);
        free(xv);
    }
    return bad ? -1 : 0;
}

/* GELU as used by GPT-2, the paper's GPT-2 Medium target (Sec. 4.2.2,
 * Sec. 4.5): the tanh form 0.5 a (1 + tanh(sqrt(2/pi) (a + 0.044715 a^3))). */
double ppo_gelu(double a) {
    const double c = sqrt(2.0 / 3.14159265358979323846);
    return 0.5 * a * (1.0 + tanh(c * (a + 0.044715 * a * a * a)));
}

void ppo_gelu_n(int64_t n, const double *a, double *out) {
    for (int64_t i = 0; i < n; ++i) out[i] = ppo_gelu(a[i]);
}

/* Non-gated MLP variant (Sec. 2.1: the decomposition holds for any FFN whose
 * intermediate neurons are separable): FFN(x) = GELU(x W_fc + b_fc) W_proj +
 * b_proj with GPT-2's layouts transposed to the API's, W_fc [d_ff, d],
 * W_proj [d, d_ff].  Neuron n's input bias b_fc[n] belongs to its expert;
 * the output bias b_proj is added once per token, whatever the selection:
 *   h_n = GELU(W_fc[n,:] . x + b_fc[n]) [* sigmoid(g_e)]
 *   y_i = b_proj[i] + sum over selected neurons n of W_proj[i, n] h_n.
 * b_fc / b_proj may be NULL (zero).  Other arguments as for ppo_ffn. */
int ppo_mlp(int64_t T, int64_t d, int64_t d_ff, int64_t E, const uint16_t *x,
            const uint16_t *Wfc, const float *bfc, const uint16_t *Wproj, const float *bproj,
            const int32_t *perm, const int32_t *idx, const int32_t *count, const double *g,
            unsigned flags, double *y) {
    if (T < 0 || d < 1 || E < 1 || d_ff % E != 0 || !x || !Wfc || !Wproj || !idx || !count || !y)
        return -1;
    if ((flags & PPO_AGG_SIGMOID) && !g) return -1;
    const int64_t de = d_ff / E;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int64_t t = 0; t < T; ++t) {
        const uint16_t *xt = x + t * d;
        double *yt = y + t * d;
        int64_t k = count[t];
        int32_t *nsel = (int32_t *)malloc(sizeof(int32_t) * (size_t)(k * de + 1));
        double *h = (double *)malloc(sizeof(double) * (size_t)(k * de + 1));
        double *xv = (double *)malloc(sizeof(double) * (size_t)d);
        if (!nsel || !h || !xv || k < 0 || k > E) {
            bad = 1;
            free(nsel);
            free(h);
            free(xv);
            continue;
        }
        for (int64_t j = 0; j < d; ++j) xv[j] = bf16_value(xt[j]);
        for (int64_t s = 0; s < k; ++s) {
            int64_t e = idx[t * E + s];
            double scale = 1.0;
            if (flags & PPO_AGG_SIGMOID) scale = 1.0 / (1.0 + exp(-g[t * E + e]));
            for (int64_t r = 0; r < de; ++r) {
                int64_t n = perm ? perm[e * de + r] : e * de + r;
                const uint16_t *w = Wfc + n * d;
                double a = bfc ? (double)bfc[n] : 0.0;
                for (int64_t j = 0; j < d; ++j) a += bf16_value(w[j]) * xv[j];
                nsel[s * de + r] = (int32_t)n;
                h[s * de + r] = ppo_gelu(a) * scale;
            }
        }
        for (int64_t i = 0; i < d; ++i) {
            const uint16_t *wp = Wproj + i * d_ff;
            double acc = bproj ? (double)bproj[i] : 0.0;
            for (int64_t q = 0; q < k * de; ++q) acc += bf16_value(wp[nsel[q]]) * h[q];
            yt[i] = acc;
        }
        free(nsel);
        free(h);
        free(xv);
    }
    return bad ? -1 : 0;
}

/* ------------------------------------------------------------------------
 * Wiring of the stacked-layer decode workload (not part of the paper's
 * method): pre-norm residual layers, x_{l+1} = x_l + FFN_l(u_l) with
 * u_l = RMSNorm(x_l), norm weight 1, carried to the next layer in bf16.
 * ------------------------------------------------------------------------ */

/* bf16 bit pattern nearest to v (ties to the even significand), rounded once
 * from the double value (no intermediate binary32 rounding).  bf16 has an
 * 8-bit significand, binary32's exponent range and its subnormals (quantum
 * 2^-133); values beyond the largest finite bf16 round to infinity. */
uint16_t ppo_bf16_round(double v) {
    uint16_t sign = (uint16_t)(signbit(v) ? 0x8000u : 0u);
    double a = fabs(v);
    if (isnan(v)) return (uint16_t)(0x7FC0u | sign);
    if (a == 0.0) return sign;
    int ex;
    (void)frexp(a, &ex); /* a = m * 2^ex, 0.5 <= m < 1 */
    int q_exp = ex - 8;  /* quantum of an 8-bit significand at this binade */
    if (q_exp < -133) q_exp = -133;
    double q = ldexp(a, -q_exp); /* exact scaling by a power of two */
    double r = nearbyint(q);     /* default rounding mode: nearest, ties to even */
    double rv = ldexp(r, q_exp);
    if (rv > 3.3895313892515355e38) return (uint16_t)(0x7F80u | sign); /* above max finite */
    float f = (float)rv; /* exact: rv has at most 8 significant bits */
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return (uint16_t)((u >> 16) | sign);
}

void ppo_bf16_round_n(int64_t n, const double *v, uint16_t *out) {
    for (int64_t i = 0; i < n; ++i) out[i] = ppo_bf16_round(v[i]);
}

/* u[t, :] = x[t, :] / sqrt(mean_j x[t, j]^2 + eps) in fp64 (unrounded), and
 * its bf16 rounding u_bits. */
int ppo_rmsnorm(int64_t T, int64_t d, const double *x, double eps, double *u, uint16_t *u_bits) {
    if (T < 0 || d < 1 || !x || !u || !u_bits || !(eps >= 0.0)) return -1;
    for (int64_t t = 0; t < T; ++t) {
        const double *xt = x + t * d;
        double ss = 0.0;
        for (int64_t j = 0; j < d; ++j) ss += xt[j] * xt[j];
        double den = sqrt(ss / (double)d + eps);
        for (int64_t j = 0; j < d; ++j) {
            u[t * d + j] = xt[j] / den;
            u_bits[t * d + j] = ppo_bf16_round(u[t * d + j]);
        }
    }
    return 0;
}

/* ------------------------------------------------------------------------
 * Routing regularisers of the training objective, forward and gradient.
 *
 *   p_ij   = softmax_j(g_i)                              Eq. (softmax_prob)
 *   L_ent  = -(1/B) sum_i sum_j p_ij log(p_ij + eps)     Eq. (entropy_loss), Sec. 3.2
 *   L_bal  = E sum_j (m_j)^2, m_j = (1/B) sum_i p_ij     Eq. (load_balance_loss), Sec. 3.2
 *   L_gate = (1/(B E)) sum_i sum_j sigmoid(g_ij)         gate-magnitude term, Sec. 4.2.3
 *   L      = eta L_ent + lambda L_bal + gamma L_gate     Eq. (train_loss) with the Sec. 4.2.3 term
 *
 * (the task loss of Eq. (train_loss) is not part of this function).
 * losses = [L_ent, L_bal, L_gate, L].  dg (optional) = dL/dg by the chain
 * rule through the full softmax Jacobian dp_ij/dg_ik = p_ij (delta_jk - p_ik).
 * Reading for p_ij = 0 (possible only with eps = 0): the term p log p is 0,
 * its limit.
 * ------------------------------------------------------------------------ */
int ppo_router_loss(int64_t B, int64_t E, const double *g, double eps, double eta, double lambda,
                    double gamma, double *losses, double *dg) {
    if (B < 1 || E < 1 || !g || !losses || !(eps >= 0.0)) return -1;
    double *p = (double *)malloc(sizeof(double) * (size_t)(B * E));
    double *m = (double *)calloc((size_t)E, sizeof(double));
    double *dldp = (double *)malloc(sizeof(double) * (size_t)E);
    if (!p || !m || !dldp) {
        free(p);
        free(m);
        free(dldp);
        return -2;
    }
    for (int64_t i = 0; i < B; ++i) ppo_softmax(E, g + i * E, p + i * E);

    double ent = 0.0, gate = 0.0;
    for (int64_t i = 0; i < B; ++i)
        for (int64_t j = 0; j < E; ++j) {
            double pij = p[i * E + j];
            if (pij > 0.0) ent += pij * log(pij + eps);
            gate += 1.0 / (1.0 + exp(-g[i * E + j]));
        }
    double l_ent = -ent / (double)B;
    for (int64_t j = 0; j < E; ++j) {
        for (int64_t i = 0; i < B; ++i) m[j] += p[i * E + j];
        m[j] /= (double)B;
    }
    double l_bal = 0.0;
    for (int64_t j = 0; j < E; ++j) l_bal += m[j] * m[j];
    l_bal *= (double)E;
    double l_gate = gate / ((double)B * (double)E);
    losses[0] = l_ent;
    losses[1] = l_bal;
    losses[2] = l_gate;
    losses[3] = eta * l_ent + lambda * l_bal + gamma * l_gate;

    if (dg) {
        for (int64_t i = 0; i < B; ++i) {
            const double *pi = p + i * E;
            /* dL/dp_ij: d/dp [p log(p + eps)] = log(p + eps) + p / (p + eps);
             * dL_bal/dp_ij = 2 E m_j / B */
            for (int64_t j = 0; j < E; ++j) {
                double de = pi[j] > 0.0 ? log(pi[j] + eps) + pi[j] / (pi[j] + eps) : 0.0;
                dldp[j] = -eta * de / (double)B + lambda * 2.0 * (double)E * m[j] / (double)B;
            }
            for (int64_t k = 0; k < E; ++k) {
                double acc = 0.0;
                for (int64_t j = 0; j < E; ++j)
                    acc += dldp[j] * pi[j] * ((j == k ? 1.0 : 0.0) - pi[k]);
                double s = 1.0 / (1.0 + exp(-g[i * E + k]));
                dg[i * E + k] = acc + gamma * s * (1.0 - s) / ((double)B * (double)E);
            }
        }
    }
    free(p);
    free(m);
    free(dldp);
    return 0;
}
