/*
 * Float64 CPU oracle of one AGS optimizer step with its gradient statistics.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * statement of what the GPU path computes, written from the paper (Tula,
 * arXiv 2603.18112).  Only the test-suite, the smoke check and the CPU
 * baseline leg of the benchmark may load it.  It shares no code, header,
 * helper or constant with the GPU library, and the GPU library never calls
 * it.
 *
 * What one step computes, in the paper's order:
 *
 *   1. Large-batch gradient = mean of the K replica gradients
 *        gbar_j = (1/K) sum_k g_kj                       (Eq. (1c), Eq. (7a))
 *   2. Per-layer statistics (one layer = one parameter tensor):
 *        W_l = sum_j w_j^2,  G_l = sum_j gbar_j^2        (norms of Eq. (5))
 *        V_l = (1/K) sum_k sum_j (g_kj - gbar_j)^2       (spread of the noise
 *                                                         term gamma, Eq. (6))
 *        S_l = sum_j g_rj^2 (small-batch gradient = replica r; r = -1 takes
 *              the mean over replicas of sum_j g_kj^2)   (UpdateGradScale,
 *                                                         Algorithm 1)
 *        rho_l = V_l / G_l
 *   3. Global squared norm G = sum_l G_l, gradient variability
 *        Delta = |G - G_prev| / G_prev                   (Eq. (5))
 *      sensitive = !(Delta < delta)                      (Algorithm 1 branch,
 *                                                         Sec. III-C)
 *      On the first step (no G_prev), G_prev <= 0 or a non-finite value,
 *      Delta = +inf, i.e. the step is treated as sensitive.
 *      Per layer, the same measure on the layer's own norm:
 *        Delta_l = |G_l - G_l,prev| / G_l,prev   (+inf under the same rules)
 *      It is always reported; with the per-layer scope (a variant of Eq. (5)
 *      for the spatial side of the mapping M of Sec. III-C) layer l's
 *      coefficient follows its own bit sensitive_l = !(Delta_l < delta)
 *      instead of the global one.
 *   4. Per-layer coefficients of the update d = a_l * gbar + b_l * w:
 *        AGS : a_l = gradscale_l if (layer scaled and not sensitive) else 1,
 *              b_l = lambda_l                 (Algorithm 1; Eq. (8b) form
 *                                              G~ = s (.) G, with the wrapped
 *                                              momentum-SGD adding decay)
 *        LARS: a_l = tau ||w|| / (||gbar|| + lambda_l ||w||) if scaled
 *              (1 when ||w|| = 0 or ||gbar|| = 0), b_l = a_l * lambda_l
 *              (LARS baseline, Sec. IV-D: learning rate scaled by
 *               ||w|| / ||grad w|| per layer)
 *        STATIC: a_l = s if (layer scaled and not sensitive) else 1,
 *              b_l = lambda_l                 (static gradient scaling U(s),
 *                                              Eq. (8a), (8b), Sec. III-C)
 *        SGD : a_l = 1, b_l = lambda_l        (vanilla large-batch baseline)
 *      lambda_l = weight_decay if the layer is decayed, else 0.
 *      Elementwise AGS (Algorithm 1 read per element): element j of a scaled
 *      layer takes a_j = gradscale_j on a non-sensitive step.
 *   5. Wrapped momentum SGD (Sec. IV-A, IV-B: SGD, momentum 0.9, weight decay;
 *      PyTorch semantics, no dampening, no Nesterov):
 *        m_j <- mu m_j + d_j ;  w_j <- w_j - eta m_j     (Eq. (7b))
 *   6. UpdateGradScale after the update when a refresh is due
 *      (refresh_every > 0 and t mod refresh_every == 0), for scaled layers:
 *        gradscale_l <- min( sqrt(S_l) / (sqrt(G_l) + eps), s_max )
 *      (1 when S_l = 0 or G_l = 0); s_max = sqrt(b_large / b_small), which
 *      is sqrt(K) when one replica's share is the small batch.  The new
 *      value is used from step t + 1 on (Algorithm 1 refreshes after the
 *      iterations that used the old one).
 *
 * Everything is float64.  Inputs are read exactly: fp32 values convert to
 * double without rounding, and a bf16 value is the upper half of an fp32.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_SCALE 1u
#define ORACLE_DECAY 2u

enum { ORACLE_SGD = 0, ORACLE_AGS = 1, ORACLE_LARS = 2, ORACLE_STATIC = 3 };

typedef struct {
    int64_t offset;
    int64_t numel;
    uint32_t flags;
    uint32_t pad_;
} oracle_layer;

typedef struct {
    int32_t n_layers;
    int32_t K;
    int32_t grad_is_bf16;
    int32_t mode;
    int32_t refresh_every;
    int32_t small_replica;
    int64_t n_flat;
    int64_t replica_stride;
    double lr, momentum, weight_decay, delta, eps, s_max, trust_coef;
    double static_scale; /* s of the static mapping U(s) */
    int32_t elementwise; /* AGS scale per element instead of per layer */
    int32_t delta_scope; /* 0: one global Delta decides; 1: Delta_l per layer */
} oracle_config;

/* Per-layer output record: W, G, V, S, rho, a, b, gradscale (after refresh),
 * Delta_l and the sensitive bit that decided the layer's coefficient.
 * With elementwise scales, a is the layer mean of the coefficients applied
 * to its elements and gradscale the layer mean of its scales. */
enum { OUT_W = 0, OUT_G, OUT_V, OUT_S, OUT_RHO, OUT_A, OUT_B, OUT_GRADSCALE, OUT_DELTA,
       OUT_SENS, OUT_N };
/* Global output record: G, G_prev (value used), Delta, sensitive, nonfinite. */
enum { GOUT_G = 0, GOUT_GPREV, GOUT_DELTA, GOUT_SENSITIVE, GOUT_NONFINITE, GOUT_N };

static double grad_at(const oracle_config *c, const void *grads, int k, int64_t j)
{
    int64_t idx = (int64_t)k * c->replica_stride + j;
    if (c->grad_is_bf16) {
        uint32_t bits = (uint32_t)((const uint16_t *)grads)[idx] << 16;
        float f;
        memcpy(&f, &bits, sizeof f);
        return (double)f;
    }
    return (double)((const float *)grads)[idx];
}

/*
 * One step.  w, m: float64 state [n_flat], updated in place when commit != 0.
 * gradscale [n_layers] (or [n_flat] with elementwise scales), *g_prev,
 * g_prev_layers [n_layers], *step: AGS state, updated when commit != 0.
 * out_layers [n_layers][OUT_N], out_global [GOUT_N].
 * Returns 0, or -1 on a bad argument, -2 when out of memory.
 */
int oracle_ags_step(const oracle_config *c, double *w, double *m, const void *grads,
                    double *gradscale, double *g_prev, double *g_prev_layers, int64_t *step,
                    int commit, const oracle_layer *layers, double *out_layers,
                    double *out_global)
{
    if (!c || !w || !m || !grads || !gradscale || !g_prev || !g_prev_layers || !step ||
        !layers || !out_layers || !out_global || c->n_layers < 1 || c->K < 1)
        return -1;
    const int L = c->n_layers, K = c->K;
    const int64_t t = *step + 1; /* the step being taken, 1-based */

    int64_t max_n = 0;
    for (int l = 0; l < L; ++l)
        if (layers[l].numel > max_n) max_n = layers[l].numel;
    double *gbar = (double *)malloc((size_t)max_n * sizeof(double));
    double *G_l = (double *)calloc((size_t)L, sizeof(double));
    double *a_l = (double *)calloc((size_t)L, sizeof(double));
    double *b_l = (double *)calloc((size_t)L, sizeof(double));
    double **gbar_keep = (double **)calloc((size_t)L, sizeof(double *));
    if (!gbar || !G_l || !a_l || !b_l || !gbar_keep) {
        free(gbar); free(G_l); free(a_l); free(b_l); free(gbar_keep);
        return -2;
    }
    int nonfinite = 0;

    /* Steps 1 and 2, layer by layer. */
    for (int l = 0; l < L; ++l) {
        const int64_t o = layers[l].offset, n = layers[l].numel;
        double *out = out_layers + (size_t)l * OUT_N;

        for (int64_t j = 0; j < n; ++j) {
            double s = 0.0;
            for (int k = 0; k < K; ++k) s += grad_at(c, grads, k, o + j);
            gbar[j] = s / K;
        }
        double W = 0.0, G = 0.0, V = 0.0, S = 0.0;
        for (int64_t j = 0; j < n; ++j) W += w[o + j] * w[o + j];
        for (int64_t j = 0; j < n; ++j) G += gbar[j] * gbar[j];
        for (int k = 0; k < K; ++k)
            for (int64_t j = 0; j < n; ++j) {
                double d = grad_at(c, grads, k, o + j) - gbar[j];
                V += d * d;
            }
        V /= K;
        if (c->small_replica >= 0) {
            for (int64_t j = 0; j < n; ++j) {
                double g = grad_at(c, grads, c->small_replica, o + j);
                S += g * g;
            }
        } else {
            for (int k = 0; k < K; ++k)
                for (int64_t j = 0; j < n; ++j) {
                    double g = grad_at(c, grads, k, o + j);
                    S += g * g;
                }
            S /= K;
        }
        double rho;
        if (G > 0.0) rho = V / G;
        else rho = (V > 0.0) ? INFINITY : 0.0;
        if (!isfinite(W) || !isfinite(G) || !isfinite(V) || !isfinite(S)) nonfinite = 1;

        out[OUT_W] = W; out[OUT_G] = G; out[OUT_V] = V; out[OUT_S] = S; out[OUT_RHO] = rho;
        G_l[l] = G;

        /* keep gbar of this layer for the update in step 5 */
        gbar_keep[l] = (double *)malloc((size_t)n * sizeof(double));
        if (!gbar_keep[l]) {
            for (int q = 0; q < l; ++q) free(gbar_keep[q]);
            free(gbar); free(G_l); free(a_l); free(b_l); free(gbar_keep);
            return -2;
        }
        memcpy(gbar_keep[l], gbar, (size_t)n * sizeof(double));
    }

    /* Step 3: global norm and gradient variability. */
    double G = 0.0;
    for (int l = 0; l < L; ++l) G += G_l[l];
    double Gp = *g_prev;
    double delta;
    if (t == 1 || !(Gp > 0.0) || !isfinite(Gp) || !isfinite(G))
        delta = INFINITY;
    else
        delta = fabs((G - Gp) / Gp);
    if (!isfinite(G)) nonfinite = 1;
    const int sensitive = !(delta < c->delta);

    /* Step 3b: per-layer variability, and the bit that decides each layer. */
    for (int l = 0; l < L; ++l) {
        const double Gpl = g_prev_layers[l];
        double dl;
        if (t == 1 || !(Gpl > 0.0) || !isfinite(Gpl) || !isfinite(G_l[l]))
            dl = INFINITY;
        else
            dl = fabs((G_l[l] - Gpl) / Gpl);
        double *out = out_layers + (size_t)l * OUT_N;
        out[OUT_DELTA] = dl;
        out[OUT_SENS] = c->delta_scope ? !(dl < c->delta) : sensitive;
    }

    /* Step 4: coefficients. */
    for (int l = 0; l < L; ++l) {
        const int scaled = (layers[l].flags & ORACLE_SCALE) != 0;
        const double lam = (layers[l].flags & ORACLE_DECAY) ? c->weight_decay : 0.0;
        double *out = out_layers + (size_t)l * OUT_N;
        double a = 1.0, b = lam;
        if (c->mode == ORACLE_AGS) {
            a = (scaled && !out[OUT_SENS]) ? gradscale[l] : 1.0;
            b = lam;
        } else if (c->mode == ORACLE_STATIC) {
            a = (scaled && !out[OUT_SENS]) ? c->static_scale : 1.0;
            b = lam;
        } else if (c->mode == ORACLE_LARS) {
            if (scaled) {
                const double wn = sqrt(out[OUT_W]), gn = sqrt(out[OUT_G]);
                a = (wn > 0.0 && gn > 0.0) ? c->trust_coef * wn / (gn + lam * wn) : 1.0;
            }
            b = a * lam;
        }
        a_l[l] = a;
        b_l[l] = b;
        out[OUT_A] = a;
        out[OUT_B] = b;
    }

    /* Elementwise AGS (Algorithm 1 read per element): element j of a scaled
     * layer takes gradscale_j on a non-sensitive step.  The layer record
     * gets the mean of the coefficients applied. */
    const int ew = c->mode == ORACLE_AGS && c->elementwise;
    if (ew) {
        for (int l = 0; l < L; ++l) {
            const int64_t o = layers[l].offset, n = layers[l].numel;
            const int scaled = (layers[l].flags & ORACLE_SCALE) != 0;
            double sum = 0.0;
            const int sens_l = out_layers[(size_t)l * OUT_N + OUT_SENS] != 0.0;
            for (int64_t j = 0; j < n; ++j) sum += (scaled && !sens_l) ? gradscale[o + j] : 1.0;
            out_layers[(size_t)l * OUT_N + OUT_A] = sum / (double)n;
        }
    }

    /* Step 5: momentum SGD on d = a gbar + b w. */
    if (commit) {
        for (int l = 0; l < L; ++l) {
            const int64_t o = layers[l].offset, n = layers[l].numel;
            const int scaled = (layers[l].flags & ORACLE_SCALE) != 0;
            for (int64_t j = 0; j < n; ++j) {
                const int sens_l = out_layers[(size_t)l * OUT_N + OUT_SENS] != 0.0;
                const double a = ew ? ((scaled && !sens_l) ? gradscale[o + j] : 1.0) : a_l[l];
                const double d = a * gbar_keep[l][j] + b_l[l] * w[o + j];
                m[o + j] = c->momentum * m[o + j] + d;
                w[o + j] = w[o + j] - c->lr * m[o + j];
            }
        }
    }

    /* Step 6: UpdateGradScale for the steps that follow. */
    const double smax = (c->s_max > 0.0) ? c->s_max : sqrt((double)K);
    const int refresh = commit && c->mode == ORACLE_AGS && c->refresh_every > 0 &&
                        (t % c->refresh_every) == 0;
    for (int l = 0; l < L; ++l) {
        double *out = out_layers + (size_t)l * OUT_N;
        if (ew) {
            /* Per element: s_j = min(|g_small,j / (gbar_j + eps)|, s_max), with
             * g_small = replica r, or the root mean square over replicas
             * (r = -1); a 0/0 ratio gives 1. */
            const int64_t o = layers[l].offset, n = layers[l].numel;
            if (refresh && (layers[l].flags & ORACLE_SCALE)) {
                for (int64_t j = 0; j < n; ++j) {
                    double gs;
                    if (c->small_replica >= 0) {
                        gs = grad_at(c, grads, c->small_replica, o + j);
                    } else {
                        double q = 0.0;
                        for (int k = 0; k < K; ++k) {
                            const double g = grad_at(c, grads, k, o + j);
                            q += g * g;
                        }
                        gs = sqrt(q / K);
                    }
                    double s = fabs(gs / (gbar_keep[l][j] + c->eps));
                    if (isnan(s)) s = 1.0;
                    if (s > smax) s = smax;
                    gradscale[o + j] = s;
                }
            }
            double sum = 0.0;
            for (int64_t j = 0; j < n; ++j) sum += gradscale[o + j];
            out[OUT_GRADSCALE] = sum / (double)n;
            continue;
        }
        if (refresh && (layers[l].flags & ORACLE_SCALE)) {
            const double S = out[OUT_S], Gl = out[OUT_G];
            double s;
            if (S > 0.0 && Gl > 0.0) {
                s = sqrt(S) / (sqrt(Gl) + c->eps);
                if (s > smax) s = smax;
            } else {
                s = 1.0;
            }
            gradscale[l] = s;
        }
        out[OUT_GRADSCALE] = gradscale[l];
    }

    out_global[GOUT_G] = G;
    out_global[GOUT_GPREV] = (t == 1) ? 0.0 : Gp;
    out_global[GOUT_DELTA] = delta;
    out_global[GOUT_SENSITIVE] = sensitive;
    out_global[GOUT_NONFINITE] = nonfinite;

    if (commit) {
        *g_prev = G;
        for (int l = 0; l < L; ++l) g_prev_layers[l] = G_l[l];
        *step = t;
    }

    for (int l = 0; l < L; ++l) free(gbar_keep[l]);
    free(gbar); free(G_l); free(a_l); free(b_l); free(gbar_keep);
    return 0;
}
