/*
 * CPU oracle for one sparse V-MoE layer, forward and backward.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the slow, plain reference that the
 * HIP path is checked against. Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load it; the product path never does.
 * It shares no code, header or constant with the HIP library.
 *
 * What it computes. The paper builds on V-MoE's sparse expert routing
 * (Sec. 1 and Sec. 2.1: tokens are routed to a few of E expert MLP blocks)
 * and adapts the pooled experts by back-propagation (Sec. 3.1, Sec. 3.2).
 * It does not spell out the layer, so the steps below follow V-MoE's
 * published definition as read for this build:
 *   z      = logits + bias + noise                    (noisy gating)
 *   p      = softmax(z)                               (exp_spec, fp32)
 *   e_1..k = top-k of z, ties to the lower expert
 *   pi     = p[e_1]                                   (batch priority)
 *   order  = tokens of each group by pi desc, index asc
 *   slots  = capacity C per (group, expert); round r = 1..k walks `order`
 *            and keeps an assignment while its expert has room
 *   xe     = dispatch of kept tokens into per-expert buffers
 *   ye     = W2 gelu(W1 xe + b1) + b2                 (exact erf GELU)
 *   y[t]   = sum over kept j of gate[t,j] * ye[row(t,j)]
 * plus the gradients of y with respect to every float input.
 *
 * Floating point. Everything after routing accumulates in double with no
 * intermediate rounding. Routing itself is defined in float32 (the priority
 * and top-k decisions are taken in the kernel's precision) and is written
 * with explicit fmaf and IEEE division so that the result is unique. Build
 * with -ffp-contract=off and without -ffast-math.
 *
 * Array conventions: row-major; float64 arrays hold values that are exactly
 * representable in the layer's dtype (bf16 or f32), widened by the caller.
 *
 * Threads. Built with OpenMP, loops over independent outputs (tokens, rows,
 * weight entries) are shared among threads; every output is still computed
 * by one thread with the sums in the order written, so results do not depend
 * on the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------ capacity */

/* Expert capacity per routing group: C = round(k * N_g * c / E), at least 1.
 * rounding 0 = half away from zero (V-MoE's buffer size), 1 = ceil. */
int orc_capacity(int n_tokens, int n_groups, int n_experts, int k, double capacity_factor,
                 int rounding) {
    double ng = (double)(n_tokens / n_groups);
    double c = (double)k * ng * capacity_factor / (double)n_experts;
    double r = rounding == 1 ? ceil(c) : floor(c + 0.5);
    if (r < 1.0) r = 1.0;
    return (int)r;
}

/* ------------------------------------------------------------ exp_spec */

/* exp(u) in float32 by Cody-Waite range reduction (Cody & Waite 1980):
 *   n = rint(u * log2(e)),  r = u - n*ln2_hi - n*ln2_lo,  |r| <= ~ln2/2
 *   exp(u) = 2^n * P(r),    P = Taylor polynomial of degree 7, Horner, fmaf
 * The high part of ln 2 has 9 significant bits, so n*ln2_hi is exact for
 * |n| <= 2^15. Results below the smallest normal are flushed to zero
 * (u < -87), overflow gives +inf (u > 88). exp_spec(0) = 1 exactly. */
float orc_exp(float u) {
    if (u < -87.0f) return 0.0f;
    if (u > 88.0f) return INFINITY;
    const float log2e = 1.44269504088896341f;
    const float ln2_hi = 0.693359375f;
    const float ln2_lo = -2.12194440e-4f;
    float t = u * log2e;
    float n = rintf(t);
    float r = fmaf(-n, ln2_hi, u);
    r = fmaf(-n, ln2_lo, r);
    /* 1/j! for j = 7..1, rounded to float */
    float p = 1.98412698e-4f;       /* 1/5040 */
    p = fmaf(p, r, 1.38888889e-3f); /* 1/720 */
    p = fmaf(p, r, 8.33333333e-3f); /* 1/120 */
    p = fmaf(p, r, 4.16666667e-2f); /* 1/24 */
    p = fmaf(p, r, 1.66666667e-1f); /* 1/6 */
    p = fmaf(p, r, 0.5f);
    p = fmaf(p, r, 1.0f);
    p = fmaf(p, r, 1.0f);
    int32_t bits;
    memcpy(&bits, &p, 4);
    bits += ((int32_t)n) << 23;
    float out;
    memcpy(&out, &bits, 4);
    return out;
}

/* ------------------------------------------------------------ router */

/* logits[t,e] = fl32( sum_{i=0..d-1} x[t,i] * w_router[g(t),e,i] ), summed in
 * double in increasing i; g(t) = t / (N/G). Every product of two bf16 or two
 * f32 values is exact in double, so this value is unique for the given order. */
void orc_router_logits(int N, int G, int d, int E, const double* x, const double* wr,
                       float* logits) {
    int ng = N / G;
#pragma omp parallel for schedule(static)
    for (int t = 0; t < N; ++t) {
        const double* w = wr + (size_t)(t / ng) * E * d;
        for (int e = 0; e < E; ++e) {
            double acc = 0.0;
            for (int i = 0; i < d; ++i) acc += x[(size_t)t * d + i] * w[(size_t)e * d + i];
            logits[(size_t)t * E + e] = (float)acc;
        }
    }
}

/* ------------------------------------------------------------ gating */

/* Noisy softmax gate and top-k for every token.
 *   z_e = (logit_e + bias_e) + noise_e          (float32, in that order)
 *   m = max_e z_e,  q_e = exp_spec(z_e - m),  s = q_0 + q_1 + ... (float32, e order)
 *   p_e = q_e / s                               (IEEE float32 division)
 *   idx[t, j] = j-th largest z, ties to the lower expert index
 *   prio[t] = p[t, idx[t, 0]]
 * bias and noise may be NULL. */
void orc_gate(int N, int E, int k, const float* logits, const float* bias, const float* noise,
              float* z_out, float* probs, int32_t* idx, float* prio) {
    float* z = (float*)malloc(sizeof(float) * E);
    float* q = (float*)malloc(sizeof(float) * E);
    char* taken = (char*)malloc(E);
    for (int t = 0; t < N; ++t) {
        for (int e = 0; e < E; ++e) {
            float v = logits[(size_t)t * E + e];
            if (bias) v = v + bias[e];
            if (noise) v = v + noise[(size_t)t * E + e];
            z[e] = v;
        }
        float m = z[0];
        for (int e = 1; e < E; ++e)
            if (z[e] > m) m = z[e];
        float s = 0.0f;
        for (int e = 0; e < E; ++e) {
            q[e] = orc_exp(z[e] - m);
            s = s + q[e];
        }
        for (int e = 0; e < E; ++e) probs[(size_t)t * E + e] = q[e] / s;
        if (z_out)
            for (int e = 0; e < E; ++e) z_out[(size_t)t * E + e] = z[e];
        memset(taken, 0, E);
        for (int j = 0; j < k; ++j) {
            int best = -1;
            for (int e = 0; e < E; ++e)
                if (!taken[e] && (best < 0 || z[e] > z[best])) best = e;
            taken[best] = 1;
            idx[(size_t)t * k + j] = best;
        }
        prio[t] = probs[(size_t)t * E + idx[(size_t)t * k]];
    }
    free(z);
    free(q);
    free(taken);
}

/* ------------------------------------------------------------ batch priority */

static const float* g_sort_prio;
static int by_priority(const void* a, const void* b) {
    int ta = *(const int32_t*)a, tb = *(const int32_t*)b;
    float pa = g_sort_prio[ta], pb = g_sort_prio[tb];
    if (pa > pb) return -1;
    if (pa < pb) return 1;
    return (ta > tb) - (ta < tb);
}

/* Batch-prioritized routing with capacity.
 * order[g*Ng + i] = i-th token of group g by (prio desc, token index asc).
 * For r = 0..k-1, walking each group's tokens in that order, assignment (t, r)
 * to expert e = idx[t, r] takes slot cnt[g, e] and is kept while cnt < C;
 * otherwise it is dropped (slot -1, gate 0). Kept gates are the probabilities
 * p[t, e] themselves (no renormalisation).
 * counts[g, e] = kept assignments; row_base[g, e] = sum_{g' < g} counts[g', e],
 * the first row of group g inside expert e's buffer. */
void orc_bpr(int N, int G, int E, int k, int C, const float* probs, const int32_t* idx,
             const float* prio, int32_t* order, int32_t* slot, float* gate, int32_t* counts,
             int32_t* row_base) {
    int ng = N / G;
    for (int t = 0; t < N; ++t) order[t] = t;
    g_sort_prio = prio;
    for (int g = 0; g < G; ++g) qsort(order + (size_t)g * ng, ng, sizeof(int32_t), by_priority);
    memset(counts, 0, sizeof(int32_t) * G * E);
    for (int g = 0; g < G; ++g) {
        for (int r = 0; r < k; ++r) {
            for (int i = 0; i < ng; ++i) {
                int t = order[(size_t)g * ng + i];
                int e = idx[(size_t)t * k + r];
                int32_t* cnt = &counts[g * E + e];
                if (*cnt < C) {
                    slot[(size_t)t * k + r] = *cnt;
                    gate[(size_t)t * k + r] = probs[(size_t)t * E + e];
                    *cnt += 1;
                } else {
                    slot[(size_t)t * k + r] = -1;
                    gate[(size_t)t * k + r] = 0.0f;
                }
            }
        }
    }
    for (int e = 0; e < E; ++e) {
        int base = 0;
        for (int g = 0; g < G; ++g) {
            row_base[g * E + e] = base;
            base += counts[g * E + e];
        }
    }
}

/* Row of assignment (t, j) in the [E, G*C, d] expert buffers, or -1 if dropped. */
static long row_of(int t, int j, int ng, int E, int k, int C, int G, const int32_t* idx,
                   const int32_t* slot, const int32_t* row_base) {
    int s = slot[(size_t)t * k + j];
    if (s < 0) return -1;
    int e = idx[(size_t)t * k + j];
    int g = t / ng;
    return (long)e * G * C + row_base[g * E + e] + s;
}

/* ------------------------------------------------------------ dispatch / combine */

/* xe[row(t,j), :] = x[t, :] for every kept assignment. Rows no assignment
 * lands on are left untouched. */
void orc_dispatch(int N, int G, int d, int E, int k, int C, const double* x, const int32_t* idx,
                  const int32_t* slot, const int32_t* row_base, double* xe) {
    int ng = N / G;
#pragma omp parallel for schedule(static)
    for (int t = 0; t < N; ++t)
        for (int j = 0; j < k; ++j) {
            long row = row_of(t, j, ng, E, k, C, G, idx, slot, row_base);
            if (row < 0) continue;
            for (int i = 0; i < d; ++i) xe[(size_t)row * d + i] = x[(size_t)t * d + i];
        }
}

/* y[t, :] = sum over kept j (in j order) of gate[t,j] * ye[row(t,j), :];
 * a token whose assignments were all dropped gets 0. */
void orc_combine_fwd(int N, int G, int d, int E, int k, int C, const double* ye,
                     const int32_t* idx, const int32_t* slot, const int32_t* row_base,
                     const float* gate, double* y) {
    int ng = N / G;
#pragma omp parallel for schedule(static)
    for (int t = 0; t < N; ++t) {
        for (int i = 0; i < d; ++i) y[(size_t)t * d + i] = 0.0;
        for (int j = 0; j < k; ++j) {
            long row = row_of(t, j, ng, E, k, C, G, idx, slot, row_base);
            if (row < 0) continue;
            double g = (double)gate[(size_t)t * k + j];
            for (int i = 0; i < d; ++i) y[(size_t)t * d + i] += g * ye[(size_t)row * d + i];
        }
    }
}

/* Backward of the combine: dye[row(t,j)] = gate[t,j] * dy[t];
 * dgate[t,j] = <dy[t], ye[row(t,j)]> for kept j, 0 for dropped j. */
void orc_combine_bwd(int N, int G, int d, int E, int k, int C, const double* dy,
                     const double* ye, const int32_t* idx, const int32_t* slot,
                     const int32_t* row_base, const float* gate, double* dye, double* dgate) {
    int ng = N / G;
#pragma omp parallel for schedule(static)
    for (int t = 0; t < N; ++t)
        for (int j = 0; j < k; ++j) {
            long row = row_of(t, j, ng, E, k, C, G, idx, slot, row_base);
            if (row < 0) {
                dgate[(size_t)t * k + j] = 0.0;
                continue;
            }
            double g = (double)gate[(size_t)t * k + j];
            double acc = 0.0;
            for (int i = 0; i < d; ++i) {
                dye[(size_t)row * d + i] = g * dy[(size_t)t * d + i];
                acc += dy[(size_t)t * d + i] * ye[(size_t)row * d + i];
            }
            dgate[(size_t)t * k + j] = acc;
        }
}

/* Backward of the dispatch: dx[t] = sum over kept j of dxe[row(t,j)] (0 if none). */
void orc_dispatch_bwd(int N, int G, int d, int E, int k, int C, const double* dxe,
                      const int32_t* idx, const int32_t* slot, const int32_t* row_base,
                      double* dx) {
    int ng = N / G;
#pragma omp parallel for schedule(static)
    for (int t = 0; t < N; ++t) {
        for (int i = 0; i < d; ++i) dx[(size_t)t * d + i] = 0.0;
        for (int j = 0; j < k; ++j) {
            long row = row_of(t, j, ng, E, k, C, G, idx, slot, row_base);
            if (row < 0) continue;
            for (int i = 0; i < d; ++i) dx[(size_t)t * d + i] += dxe[(size_t)row * d + i];
        }
    }
}

/* ------------------------------------------------------------ expert MLP */

static double gelu(double h) { return 0.5 * h * (1.0 + erf(h / sqrt(2.0))); }

/* d gelu / dh = Phi(h) + h * phi(h) */
static double gelu_grad(double h) {
    const double inv_sqrt_2pi = 0.39894228040143267794;
    return 0.5 * (1.0 + erf(h / sqrt(2.0))) + h * inv_sqrt_2pi * exp(-0.5 * h * h);
}

/* One expert's MLP over `rows` rows of its buffer:
 *   H[r, j]  = b1[j] + sum_i xe[r, i] * w1[j, i]        (w1: [f, d])
 *   A[r, j]  = gelu(H[r, j]),  G[r, j] = gelu'(H[r, j])
 *   ye[r, o] = b2[o] + sum_j A[r, j] * w2[o, j]         (w2: [d, f])
 * H, A and G may be NULL. */
void orc_ffn_fwd(int rows, int d, int f, const double* xe, const double* w1, const double* b1,
                 const double* w2, const double* b2, double* H, double* A, double* G,
                 double* ye) {
#pragma omp parallel
    {
    double* h = (double*)malloc(sizeof(double) * f);
    double* a = (double*)malloc(sizeof(double) * f);
#pragma omp for schedule(static)
    for (int r = 0; r < rows; ++r) {
        for (int j = 0; j < f; ++j) {
            double acc = b1[j];
            for (int i = 0; i < d; ++i) acc += xe[(size_t)r * d + i] * w1[(size_t)j * d + i];
            h[j] = acc;
            a[j] = gelu(acc);
            if (H) H[(size_t)r * f + j] = acc;
            if (A) A[(size_t)r * f + j] = a[j];
            if (G) G[(size_t)r * f + j] = gelu_grad(acc);
        }
        for (int o = 0; o < d; ++o) {
            double acc = b2[o];
            for (int j = 0; j < f; ++j) acc += a[j] * w2[(size_t)o * f + j];
            ye[(size_t)r * d + o] = acc;
        }
    }
    free(h);
    free(a);
    }
}

/* Per-row backward of one expert's MLP (H is recomputed from xe):
 *   dA[r, j]  = sum_o dye[r, o] * w2[o, j]
 *   dH[r, j]  = dA[r, j] * gelu'(H[r, j])
 *   dxe[r, i] = sum_j dH[r, j] * w1[j, i]
 * dH may be NULL. */
void orc_ffn_bwd_rows(int rows, int d, int f, const double* xe, const double* w1,
                      const double* b1, const double* w2, const double* dye, double* dxe,
                      double* dH) {
#pragma omp parallel
    {
    double* dh = (double*)malloc(sizeof(double) * f);
#pragma omp for schedule(static)
    for (int r = 0; r < rows; ++r) {
        for (int j = 0; j < f; ++j) {
            double h = b1[j];
            for (int i = 0; i < d; ++i) h += xe[(size_t)r * d + i] * w1[(size_t)j * d + i];
            double da = 0.0;
            for (int o = 0; o < d; ++o) da += dye[(size_t)r * d + o] * w2[(size_t)o * f + j];
            dh[j] = da * gelu_grad(h);
            if (dH) dH[(size_t)r * f + j] = dh[j];
        }
        for (int i = 0; i < d; ++i) {
            double acc = 0.0;
            for (int j = 0; j < f; ++j) acc += dh[j] * w1[(size_t)j * d + i];
            dxe[(size_t)r * d + i] = acc;
        }
    }
    free(dh);
    }
}

/* Weight gradients of one expert's MLP over its `rows` kept rows:
 *   dW2[o, j] = sum_r dye[r, o] * A[r, j]       db2[o] = sum_r dye[r, o]
 *   dW1[j, i] = sum_r dH[r, j] * xe[r, i]       db1[j] = sum_r dH[r, j]
 * A and dH are recomputed from xe as in orc_ffn_fwd / orc_ffn_bwd_rows.
 * With rows = 0 every gradient is 0. */
void orc_ffn_bwd_weights(int rows, int d, int f, const double* xe, const double* w1,
                         const double* b1, const double* w2, const double* dye, double* dw1,
                         double* db1, double* dw2, double* db2) {
    double* A = (double*)malloc(sizeof(double) * ((size_t)rows * f + 1));
    double* dH = (double*)malloc(sizeof(double) * ((size_t)rows * f + 1));
#pragma omp parallel for schedule(static)
    for (int r = 0; r < rows; ++r)
        for (int j = 0; j < f; ++j) {
            double h = b1[j];
            for (int i = 0; i < d; ++i) h += xe[(size_t)r * d + i] * w1[(size_t)j * d + i];
            double da = 0.0;
            for (int o = 0; o < d; ++o) da += dye[(size_t)r * d + o] * w2[(size_t)o * f + j];
            A[(size_t)r * f + j] = gelu(h);
            dH[(size_t)r * f + j] = da * gelu_grad(h);
        }
#pragma omp parallel for schedule(static)
    for (int o = 0; o < d; ++o) {
        double sb = 0.0;
        for (int r = 0; r < rows; ++r) sb += dye[(size_t)r * d + o];
        db2[o] = sb;
        for (int j = 0; j < f; ++j) {
            double acc = 0.0;
            for (int r = 0; r < rows; ++r) acc += dye[(size_t)r * d + o] * A[(size_t)r * f + j];
            dw2[(size_t)o * f + j] = acc;
        }
    }
#pragma omp parallel for schedule(static)
    for (int j = 0; j < f; ++j) {
        double sb = 0.0;
        for (int r = 0; r < rows; ++r) sb += dH[(size_t)r * f + j];
        db1[j] = sb;
        for (int i = 0; i < d; ++i) {
            double acc = 0.0;
            for (int r = 0; r < rows; ++r) acc += dH[(size_t)r * f + j] * xe[(size_t)r * d + i];
            dw1[(size_t)j * d + i] = acc;
        }
    }
    free(A);
    free(dH);
}

/* Selected weight-gradient entries of one expert, each by its definition:
 * which[s] = 1 -> dW1[row[s], col[s]], 2 -> dW2[row[s], col[s]],
 *            3 -> db1[row[s]],        4 -> db2[row[s]]. */
void orc_ffn_bwd_weight_entries(int rows, int d, int f, const double* xe, const double* w1,
                                const double* b1, const double* w2, const double* dye,
                                int n_samples, const int32_t* which, const int32_t* row,
                                const int32_t* col, double* out) {
#pragma omp parallel for schedule(dynamic)
    for (int s = 0; s < n_samples; ++s) {
        int w = which[s];
        /* column j of H / dH is needed by dW1, db1 (j = row) and dW2 (j = col) */
        int j = (w == 2) ? col[s] : row[s];
        double acc = 0.0;
        for (int r = 0; r < rows; ++r) {
            if (w == 4) {
                acc += dye[(size_t)r * d + row[s]];
                continue;
            }
            double h = b1[j];
            for (int i = 0; i < d; ++i) h += xe[(size_t)r * d + i] * w1[(size_t)j * d + i];
            if (w == 2) {
                acc += dye[(size_t)r * d + row[s]] * gelu(h);
                continue;
            }
            double da = 0.0;
            for (int o = 0; o < d; ++o) da += dye[(size_t)r * d + o] * w2[(size_t)o * f + j];
            double dh = da * gelu_grad(h);
            acc += (w == 1) ? dh * xe[(size_t)r * d + col[s]] : dh;
        }
        out[s] = acc;
    }
}

/* ------------------------------------------------------------ router backward */

/* Gradient through the gate into the router:
 *   dp[t, e]  = sum over kept j with idx[t,j] = e of dgate[t,j]
 *   dz[t, e]  = p[t,e] * (dp[t,e] - sum_e' p[t,e'] dp[t,e'])    (softmax Jacobian)
 *   dx[t, i] += sum_e dz[t,e] * w_router[g(t), e, i]
 *   dw_router[g, e, i] = sum_{t in g} dz[t,e] * x[t,i]          (if dwr != NULL)
 * Top-k, capacity and the priority order are piecewise constant: no gradient.
 * dz_out (may be NULL) receives dz. */
void orc_route_bwd(int N, int G, int d, int E, int k, const double* x, const double* wr,
                   const float* probs, const int32_t* idx, const int32_t* slot,
                   const double* dgate, double* dx, double* dwr, double* dz_out) {
    int ng = N / G;
    double* dz = (double*)malloc(sizeof(double) * (size_t)N * E);
#pragma omp parallel
    {
    double* dp = (double*)malloc(sizeof(double) * E);
#pragma omp for schedule(static)
    for (int t = 0; t < N; ++t) {
        for (int e = 0; e < E; ++e) dp[e] = 0.0;
        for (int j = 0; j < k; ++j)
            if (slot[(size_t)t * k + j] >= 0) dp[idx[(size_t)t * k + j]] += dgate[(size_t)t * k + j];
        double pdp = 0.0;
        for (int e = 0; e < E; ++e) pdp += (double)probs[(size_t)t * E + e] * dp[e];
        for (int e = 0; e < E; ++e)
            dz[(size_t)t * E + e] = (double)probs[(size_t)t * E + e] * (dp[e] - pdp);
    }
    free(dp);
    }
#pragma omp parallel for schedule(static)
    for (int t = 0; t < N; ++t) {
        const double* w = wr + (size_t)(t / ng) * E * d;
        for (int i = 0; i < d; ++i) {
            double acc = 0.0;
            for (int e = 0; e < E; ++e) acc += dz[(size_t)t * E + e] * w[(size_t)e * d + i];
            dx[(size_t)t * d + i] += acc;
        }
    }
    if (dwr) {
#pragma omp parallel for collapse(3) schedule(static)
        for (int g = 0; g < G; ++g)
            for (int e = 0; e < E; ++e)
                for (int i = 0; i < d; ++i) {
                    double acc = 0.0;
                    for (int t = g * ng; t < (g + 1) * ng; ++t)
                        acc += dz[(size_t)t * E + e] * x[(size_t)t * d + i];
                    dwr[((size_t)g * E + e) * d + i] = acc;
                }
    }
    if (dz_out) memcpy(dz_out, dz, sizeof(double) * (size_t)N * E);
    free(dz);
}
