// Auxiliary balance losses on the gate and their gradient with respect to the
// router logits (the balance losses that the paper cites in Sec. 1 and
// Sec. 2.3 as the alternative to capacity limits, in the published noisy
// top-k gating form):
//   importance imp[g,e]  = sum over the group's tokens of probs[t,e];
//   load       load[g,e] = sum over tokens of Phi((l'[t,e] - thr[t,e]) / sigma),
//              l' = logits + bias, thr = k-th largest noisy logit
//              z = (logits + bias) + noise among the other experts (-inf if
//              fewer than k), i.e. the chance that e stays in the top-k when
//              only its own noise is drawn again;
//   losses     CV^2 = var / mean^2 over the experts (0 for a zero sum), and
//   dlogits    = d/dlogits of sum_g w_imp CV^2(imp[g]) + w_load CV^2(load[g]).
// Two launches: per-chunk sums (one thread per token, wave-shuffle sums), then
// the per-token gradient row, each block of which first forms its group's
// losses and coefficients from the chunk sums in double (fixed order). Every pass reads the [N, E] rows once; N x E is small next to
// the layer's activations, so the launches are latency-bound.
#include <type_traits>

#include "common.h"

namespace vmoe {
namespace {

constexpr int kBalTok = 256;  // tokens per block (one per thread)

// The token's noisy logits in f32, formed as the router forms them, and the
// indices of its k + 1 largest (ties: lower index first).
template <int EMAX>
struct TokenTop {
    float clean[EMAX], z[EMAX];
    int s_km1, s_k;     // ranks k-1 and k (s_k = -1 when k = E)
    uint64_t topk;      // bit e set for the k chosen experts
};

template <int EMAX>
__device__ __forceinline__ void token_top(TokenTop<EMAX>& r, const float* __restrict__ logits,
                                          const float* __restrict__ bias,
                                          const float* __restrict__ noise, size_t t, int E,
                                          int k) {
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
        if (e < E) {
            const float l = logits[t * E + e];
            const float c = bias ? __fadd_rn(l, bias[e]) : l;
            r.clean[e] = c;
            r.z[e] = noise ? __fadd_rn(c, noise[t * E + e]) : c;
        } else {
            r.clean[e] = 0.0f;
            r.z[e] = -INFINITY;
        }
    }
    uint64_t taken = 0;
    r.s_km1 = -1;
    r.s_k = -1;
    const int ranks = k < E ? k + 1 : k;
    for (int j = 0; j < ranks; ++j) {
        int best = -1;
        float bv = 0.0f;
#pragma unroll
        for (int e = 0; e < EMAX; ++e) {
            const bool free_e = e < E && !((taken >> e) & 1ull);
            if (free_e && (best < 0 || r.z[e] > bv)) {
                best = e;
                bv = r.z[e];
            }
        }
        taken |= 1ull << best;
        if (j == k - 1) {
            r.s_km1 = best;
            r.topk = taken;
        }
        if (j == k) r.s_k = best;
    }
}

// thr[e]: rank k among the others = rank k overall (s_k) if e is in the top
// k, else rank k-1 (s_{k-1}); u = (l' - thr) / sigma.
template <int EMAX>
__device__ __forceinline__ float token_u(const TokenTop<EMAX>& r, int e, float sigma,
                                         int* thr_e) {
    const bool in_top = (r.topk >> e) & 1ull;
    const int s = in_top ? r.s_k : r.s_km1;
    *thr_e = s;
    if (s < 0) return INFINITY;
    float thr = 0.0f;
#pragma unroll
    for (int q = 0; q < EMAX; ++q)
        if (q == s) thr = r.z[q];
    return (r.clean[e] - thr) / sigma;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// partial[g][chunk][0 | 1][e] = sums of probs and of the load probability over
// the chunk's tokens.
template <int EMAX>
__global__ __launch_bounds__(kBalTok) void balance_partial_kernel(
    const float* __restrict__ logits, const float* __restrict__ bias,
    const float* __restrict__ noise, const float* __restrict__ probs, float sigma, int Ng, int E,
    int k, int nch, float* __restrict__ partial) {
    __shared__ float wsum[kBalTok / 64][2][EMAX];
    const int chunk = blockIdx.x, g = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int tl = chunk * kBalTok + tid;
    const bool live = tl < Ng;
    const size_t t = static_cast<size_t>(g) * Ng + (live ? tl : 0);
    TokenTop<EMAX> r;
    token_top<EMAX>(r, logits, bias, noise, t, E, k);
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
        if (e >= E) break;
        int s;
        const float u = token_u<EMAX>(r, e, sigma, &s);
        const float pl = live ? normcdff(u) : 0.0f;
        const float pi = live ? probs[t * E + e] : 0.0f;
        const float a = wave_sum(pi), b = wave_sum(pl);
        if (lane == 0) {
            wsum[wave][0][e] = a;
            wsum[wave][1][e] = b;
        }
    }
    __syncthreads();
    if (tid < 2 * E) {
        const int which = tid / E, e = tid % E;
        float s = 0.0f;
#pragma unroll
        for (int w = 0; w < kBalTok / 64; ++w) s += wsum[w][which][e];
        partial[((static_cast<size_t>(g) * nch + chunk) * 2 + which) * E + e] = s;
    }
}

// Per group: the chunk sums in double (chunk order), both CV^2 values and the
// gradient coefficients c[e] = w 2 / (E mu^2) (v_e - mu - var / mu) into cs
// (every block of the group forms the same values; block 0 writes the losses
// and the optional sums).
template <int EMAX>
__device__ __forceinline__ void balance_coefficients(const float* __restrict__ partial, int nch,
                                                     int E, int g, float w_imp, float w_load,
                                                     float (&cs)[2][EMAX], bool writer,
                                                     float* __restrict__ losses,
                                                     float* __restrict__ imp_out,
                                                     float* __restrict__ load_out) {
    __shared__ double v[2][EMAX];
    __shared__ double stat[2][2];  // mean, variance
    const int tid = threadIdx.x;
    if (tid < 2 * E) {
        const int which = tid / E, e = tid % E;
        const float* src = partial + (static_cast<size_t>(g) * nch * 2 + which) * E + e;
        double s = 0.0;
        int c = 0;
        for (; c + 4 <= nch; c += 4) {  // four chunk values in flight, summed in chunk order
            const float a0 = src[(c + 0) * 2 * E], a1 = src[(c + 1) * 2 * E];
            const float a2 = src[(c + 2) * 2 * E], a3 = src[(c + 3) * 2 * E];
            s += a0;
            s += a1;
            s += a2;
            s += a3;
        }
        for (; c < nch; ++c) s += src[c * 2 * E];
        v[which][e] = s;
        float* out = which == 0 ? imp_out : load_out;
        if (writer && out) out[static_cast<size_t>(g) * E + e] = static_cast<float>(s);
    }
    __syncthreads();
    if (tid < 2) {
        double sum = 0.0;
        for (int e = 0; e < E; ++e) sum += v[tid][e];
        const double mu = sum / E;
        double var = 0.0;
        for (int e = 0; e < E; ++e) var += (v[tid][e] - mu) * (v[tid][e] - mu);
        var /= E;
        stat[tid][0] = mu;
        stat[tid][1] = var;
        if (writer)
            losses[static_cast<size_t>(g) * 2 + tid] =
                static_cast<float>(sum == 0.0 ? 0.0 : var / (mu * mu));
    }
    __syncthreads();
    if (tid < 2 * E) {
        const int which = tid / E, e = tid % E;
        const double mu = stat[which][0], var = stat[which][1];
        const double w = which == 0 ? w_imp : w_load;
        const double c = mu == 0.0 ? 0.0 : w * 2.0 / (E * mu * mu) * (v[which][e] - mu - var / mu);
        cs[which][e] = static_cast<float>(c);
    }
    __syncthreads();
}

// dlogits[t,e] = p_e (ci_e - sum p ci) + cl_e phi(u_e) / sigma, minus at the
// threshold expert of every e its cl_e phi(u_e) / sigma (s_k for the chosen
// experts, s_{k-1} for the others).
template <int EMAX>
__global__ __launch_bounds__(kBalTok) void balance_grad_kernel(
    const float* __restrict__ logits, const float* __restrict__ bias,
    const float* __restrict__ noise, const float* __restrict__ probs,
    const float* __restrict__ partial, int nch, float sigma, float w_imp, float w_load, int Ng,
    int E, int k, float* __restrict__ losses, float* __restrict__ imp_out,
    float* __restrict__ load_out, float* __restrict__ dlogits) {
    __shared__ float cs[2][EMAX];
    const int g = blockIdx.y, tid = threadIdx.x;
    balance_coefficients<EMAX>(partial, nch, E, g, w_imp, w_load, cs, blockIdx.x == 0, losses,
                               imp_out, load_out);
    const int tl = blockIdx.x * kBalTok + tid;
    if (tl >= Ng) return;
    const size_t t = static_cast<size_t>(g) * Ng + tl;
    TokenTop<EMAX> r;
    token_top<EMAX>(r, logits, bias, noise, t, E, k);
    constexpr float kInvSqrt2Pi = 0.398942280401432678f;
    float p[EMAX], dl[EMAX];
    float pc = 0.0f, at_k = 0.0f, at_km1 = 0.0f;
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
        p[e] = e < E ? probs[t * E + e] : 0.0f;
        pc = e < E ? __builtin_fmaf(p[e], cs[0][e], pc) : pc;
    }
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
        if (e >= E) break;
        int s;
        const float u = token_u<EMAX>(r, e, sigma, &s);
        const float a = s < 0 ? 0.0f : cs[1][e] * (expf(-0.5f * u * u) * kInvSqrt2Pi) / sigma;
        dl[e] = p[e] * (cs[0][e] - pc) + a;
        if ((r.topk >> e) & 1ull) at_k += a;
        else at_km1 += a;
    }
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
        if (e >= E) break;
        float v = dl[e];
        if (e == r.s_k) v -= at_k;
        if (e == r.s_km1) v -= at_km1;
        dlogits[t * E + e] = v;
    }
}

unsigned balance_chunks(const Dims& D) { return cdiv(D.Ng, kBalTok); }

template <int EMAX>
void launch_balance(const Dims& D, const float* logits, const float* bias, const float* noise,
                    const float* probs, float sigma, float w_imp, float w_load, float* losses,
                    float* imp, float* load, float* dlogits, float* partial, hipStream_t st) {
    // nch = 0 (no tokens) still runs one block per group to write zero losses
    const unsigned nch = balance_chunks(D);
    if (nch > 0)
        balance_partial_kernel<EMAX><<<dim3(nch, D.G), kBalTok, 0, st>>>(
            logits, bias, noise, probs, sigma, D.Ng, D.E, D.k, nch, partial);
    balance_grad_kernel<EMAX><<<dim3(nch > 0 ? nch : 1, D.G), kBalTok, 0, st>>>(
        logits, bias, noise, probs, partial, static_cast<int>(nch), sigma, w_imp, w_load, D.Ng,
        D.E, D.k, losses, imp, load, dlogits);
}

}  // namespace

// Workspace: per-chunk sums [G, chunks, 2, E] f32.
size_t balance_workspace_bytes(const Dims& D) {
    return sizeof(float) * static_cast<size_t>(D.G) * 2 * D.E * balance_chunks(D);
}

vmoe_status balance_launch(const Dims& D, const float* logits, const float* bias,
                           const float* noise, const float* probs, float sigma, float w_imp,
                           float w_load, float* losses, float* imp, float* load, float* dlogits,
                           void* ws, hipStream_t st) {
    float* partial = static_cast<float*>(ws);
    auto go = [&](auto tag) {
        constexpr int EM = decltype(tag)::value;
        launch_balance<EM>(D, logits, bias, noise, probs, sigma, w_imp, w_load, losses, imp, load,
                           dlogits, partial, st);
    };
    if (D.E <= 8) go(std::integral_constant<int, 8>{});
    else if (D.E <= 16) go(std::integral_constant<int, 16>{});
    else if (D.E <= 32) go(std::integral_constant<int, 32>{});
    else go(std::integral_constant<int, 64>{});
    return launch_status();
}

}  // namespace vmoe
