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
// Two launches: per-chunk sums, then the gradient rows, each block of which
// first forms its group's losses and coefficients from the chunk sums in
// double (fixed order). Up to 8 experts a thread holds a whole token; beyond,
// lanes run over experts (a token's E values on consecutive lanes), so no
// thread keeps an E-wide array and every row access is contiguous. Each
// launch reads the [N, E] rows once; N x E is small next to the layer's
// activations, so both are latency-bound.
#include <type_traits>

#include "common.h"

namespace vmoe {
namespace {

constexpr int kBalWaves = 4;  // waves per block
constexpr int kBalIters = 4;  // token steps per wave (more waves in flight: 71 -> 45 us at E = 32, N = 36 928)

// Lanes over experts: a token's E values sit on EMAX consecutive lanes (EMAX
// the power of two >= E), 64 / EMAX tokens per wave step, kBalIters steps per
// wave, so a block covers CH tokens and every row access is contiguous.
template <int EMAX>
struct BalGeom {
    static constexpr int TPW = 64 / EMAX;
    static constexpr int CH = TPW * kBalWaves * kBalIters;
};

// One (token, expert) lane: the noisy logit z in f32 formed as the router
// forms it, (logits + bias) + noise; the top k + 1 of the token by a
// butterfly arg-max inside the segment (ties: lower index); u = (l - thr) /
// sigma with thr the k-th largest noisy logit among the other experts, which
// is rank k overall (s_k) for a chosen expert and rank k - 1 (s_km1)
// otherwise; u = +inf when that rank does not exist (k = E).
struct LaneTok {
    float u;
    bool in_top;
    int s_km1, s_k, thr_e;
};

// The lane's inputs of every token step, requested before any is used.
struct LaneRows {
    float l[kBalIters], n[kBalIters], p[kBalIters];
};

template <int EMAX>
__device__ __forceinline__ void lane_rows(LaneRows& x, const float* __restrict__ logits,
                                          const float* __restrict__ noise,
                                          const float* __restrict__ probs, int chunk, int Ng,
                                          int g, int E, int wave, int sub, int e) {
    using Gm = BalGeom<EMAX>;
#pragma unroll
    for (int it = 0; it < kBalIters; ++it) {
        const int tl = chunk * Gm::CH + (it * kBalWaves + wave) * Gm::TPW + sub;
        const bool live = tl < Ng && e < E;
        const size_t q = (static_cast<size_t>(g) * Ng + (live ? tl : 0)) * E + (live ? e : 0);
        x.l[it] = live ? logits[q] : 0.0f;
        x.n[it] = (live && noise) ? noise[q] : 0.0f;
        x.p[it] = live ? probs[q] : 0.0f;
    }
}

template <int EMAX>
__device__ __forceinline__ LaneTok lane_token(float l, float nz, float be, bool has_bias,
                                              bool has_noise, bool live, int e, int E, int k,
                                              float sigma) {
    float clean = 0.0f, z = -INFINITY;
    if (live) {
        clean = has_bias ? __fadd_rn(l, be) : l;
        z = has_noise ? __fadd_rn(clean, nz) : clean;
    }
    LaneTok r;
    r.s_km1 = -1;
    r.s_k = -1;
    r.in_top = false;
    bool taken = false;
    const int ranks = k < E ? k + 1 : k;
    for (int j = 0; j < ranks; ++j) {
        float bv = (taken || e >= E) ? -INFINITY : z;
        int bi = (taken || e >= E) ? (1 << 30) : e;
#pragma unroll
        for (int o = EMAX / 2; o > 0; o >>= 1) {
            const float ov = __shfl_xor(bv, o);
            const int oi = __shfl_xor(bi, o);
            if (ov > bv || (ov == bv && oi < bi)) {
                bv = ov;
                bi = oi;
            }
        }
        taken = taken || (e == bi);
        if (j == k - 1) {
            r.s_km1 = bi;
            r.in_top = taken;
        }
        if (j == k) r.s_k = bi;
    }
    const int s = r.in_top ? r.s_k : r.s_km1;
    r.thr_e = s;
    const int seg = (threadIdx.x & 63) & ~(EMAX - 1);
    const float thr = __shfl(z, seg + (s < 0 ? 0 : s));
    r.u = s < 0 ? INFINITY : (clean - thr) / sigma;
    return r;
}

// partial[g][chunk][0 | 1][e] = sums of probs and of the load probability
// over the chunk's tokens (each lane in step order, then the wave's token
// lanes, then the waves, all in a fixed order).
template <int EMAX>
__global__ __launch_bounds__(64 * kBalWaves) void balance_partial_kernel(
    const float* __restrict__ logits, const float* __restrict__ bias,
    const float* __restrict__ noise, const float* __restrict__ probs, float sigma, int Ng, int E,
    int k, float* __restrict__ partial) {
    using Gm = BalGeom<EMAX>;
    __shared__ float wsum[kBalWaves][2][EMAX];
    const int chunk = blockIdx.x, g = blockIdx.y, nch = gridDim.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int e = lane % EMAX, sub = lane / EMAX;
    LaneRows x;
    lane_rows<EMAX>(x, logits, noise, probs, chunk, Ng, g, E, wave, sub, e);
    const float be = (bias && e < E) ? bias[e] : 0.0f;
    float ap = 0.0f, al = 0.0f;
#pragma unroll
    for (int it = 0; it < kBalIters; ++it) {
        const int tl = chunk * Gm::CH + (it * kBalWaves + wave) * Gm::TPW + sub;
        const bool live = tl < Ng && e < E;
        const LaneTok r = lane_token<EMAX>(x.l[it], x.n[it], be, bias != nullptr,
                                           noise != nullptr, live, e, E, k, sigma);
        if (live) {
            ap += x.p[it];
            al += normcdff(r.u);
        }
    }
#pragma unroll
    for (int o = EMAX; o < 64; o <<= 1) {
        ap += __shfl_xor(ap, o);
        al += __shfl_xor(al, o);
    }
    if (sub == 0) {
        wsum[wave][0][e] = ap;
        wsum[wave][1][e] = al;
    }
    __syncthreads();
    if (tid < 2 * E) {
        const int which = tid / E, q = tid % E;
        float v = 0.0f;
#pragma unroll
        for (int w = 0; w < kBalWaves; ++w) v += wsum[w][which][q];
        partial[(static_cast<size_t>(g) * nch + chunk) * 2 * E + tid] = v;
    }
}

// Per group: the chunk sums in double (each of 256 / 2E threads per column
// takes every (256 / 2E)-th chunk in order, the parts then added in order),
// both CV^2 values and the gradient coefficients
// c[e] = w 2 / (E mu^2) (v_e - mu - var / mu) into cs. Every block of the
// group forms the same values; block 0 writes the losses and optional sums.
template <int EMAX>
__device__ __forceinline__ void balance_coefficients(const float* __restrict__ partial, int nch,
                                                     int E, int g, float w_imp, float w_load,
                                                     float (&cs)[2][EMAX], bool writer,
                                                     float* __restrict__ losses,
                                                     float* __restrict__ imp_out,
                                                     float* __restrict__ load_out) {
    __shared__ double part[64 * kBalWaves];
    __shared__ double v[2][EMAX];
    __shared__ double stat[2][2];  // mean, variance
    const int tid = threadIdx.x, cols = 2 * E, P = (64 * kBalWaves) / cols;
    const int c = tid % cols, q = tid / cols;
    double s = 0.0;
    if (q < P) {
        const float* src = partial + static_cast<size_t>(g) * nch * cols + c;
        int ch = q;
        for (; ch + 7 * P < nch; ch += 8 * P) {  // eight chunks in flight, added in order
            float a[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) a[u] = src[static_cast<size_t>(ch + u * P) * cols];
#pragma unroll
            for (int u = 0; u < 8; ++u) s += a[u];
        }
        for (; ch < nch; ch += P) s += src[static_cast<size_t>(ch) * cols];
    }
    part[tid] = s;
    __syncthreads();
    if (tid < cols) {
        double t = 0.0;
        for (int r = 0; r < P; ++r) t += part[r * cols + tid];
        const int which = tid / E, e = tid % E;
        v[which][e] = t;
        float* out = which == 0 ? imp_out : load_out;
        if (writer && out) out[static_cast<size_t>(g) * E + e] = static_cast<float>(t);
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
    if (tid < cols) {
        const int which = tid / E, e = tid % E;
        const double mu = stat[which][0], var = stat[which][1];
        const double w = which == 0 ? w_imp : w_load;
        const double cf = mu == 0.0 ? 0.0 : w * 2.0 / (E * mu * mu) * (v[which][e] - mu - var / mu);
        cs[which][e] = static_cast<float>(cf);
    }
    __syncthreads();
}

// dlogits[t,e] = p_e (ci_e - sum p ci) + cl_e phi(u_e) / sigma, minus at the
// threshold expert of every e its cl_e phi(u_e) / sigma (s_k collects the
// chosen experts' terms, s_km1 the others').
template <int EMAX>
__global__ __launch_bounds__(64 * kBalWaves) void balance_grad_kernel(
    const float* __restrict__ logits, const float* __restrict__ bias,
    const float* __restrict__ noise, const float* __restrict__ probs,
    const float* __restrict__ partial, int nch, float sigma, float w_imp, float w_load, int Ng,
    int E, int k, float* __restrict__ losses, float* __restrict__ imp_out,
    float* __restrict__ load_out, float* __restrict__ dlogits) {
    using Gm = BalGeom<EMAX>;
    __shared__ float cs[2][EMAX];
    const int g = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    balance_coefficients<EMAX>(partial, nch, E, g, w_imp, w_load, cs, blockIdx.x == 0, losses,
                               imp_out, load_out);
    constexpr float kInvSqrt2Pi = 0.398942280401432678f;
    const int e = lane % EMAX, sub = lane / EMAX;
    const float c0 = e < E ? cs[0][e] : 0.0f, c1 = e < E ? cs[1][e] : 0.0f;
    LaneRows x;
    lane_rows<EMAX>(x, logits, noise, probs, blockIdx.x, Ng, g, E, wave, sub, e);
    const float be = (bias && e < E) ? bias[e] : 0.0f;
#pragma unroll
    for (int it = 0; it < kBalIters; ++it) {
        const int tl = blockIdx.x * Gm::CH + (it * kBalWaves + wave) * Gm::TPW + sub;
        const bool live = tl < Ng && e < E;
        const size_t t = static_cast<size_t>(g) * Ng + (tl < Ng ? tl : 0);
        const float p = x.p[it];
        const LaneTok r = lane_token<EMAX>(x.l[it], x.n[it], be, bias != nullptr,
                                           noise != nullptr, live, e, E, k, sigma);
        const float a =
            (live && r.thr_e >= 0) ? c1 * (expf(-0.5f * r.u * r.u) * kInvSqrt2Pi) / sigma : 0.0f;
        float pc = p * c0, ak = r.in_top ? a : 0.0f, am = r.in_top ? 0.0f : a;
#pragma unroll
        for (int o = EMAX / 2; o > 0; o >>= 1) {
            pc += __shfl_xor(pc, o);
            ak += __shfl_xor(ak, o);
            am += __shfl_xor(am, o);
        }
        float dl = p * (c0 - pc) + a;
        if (e == r.s_k) dl -= ak;
        if (e == r.s_km1) dl -= am;
        if (live) dlogits[t * E + e] = dl;
    }
}

// Small expert counts (E <= 8): one thread per token, its E values in
// registers, no cross-lane selection; the same chunk-sum layout.
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

// partial[g][chunk][0 | 1][e] for the one-thread-per-token blocks.
template <int EMAX>
__global__ __launch_bounds__(kBalTok) void balance_partial_rows_kernel(
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

// dlogits[t,e] = p_e (ci_e - sum p ci) + cl_e phi(u_e) / sigma, minus at the
// threshold expert of every e its cl_e phi(u_e) / sigma (s_k for the chosen
// experts, s_{k-1} for the others).
template <int EMAX>
__global__ __launch_bounds__(kBalTok) void balance_grad_rows_kernel(
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

template <int EMAX>
unsigned balance_chunks_t(const Dims& D) {
    return cdiv(D.Ng, EMAX <= 8 ? kBalTok : BalGeom<EMAX>::CH);
}

template <int EMAX>
void launch_balance(const Dims& D, const float* logits, const float* bias, const float* noise,
                    const float* probs, float sigma, float w_imp, float w_load, float* losses,
                    float* imp, float* load, float* dlogits, float* partial, hipStream_t st) {
    // nch = 0 (no tokens) still runs one block per group to write zero losses
    const unsigned nch = balance_chunks_t<EMAX>(D);
    const dim3 grid(nch > 0 ? nch : 1, D.G);
    if constexpr (EMAX <= 8) {
        if (nch > 0)
            balance_partial_rows_kernel<EMAX><<<grid, kBalTok, 0, st>>>(
                logits, bias, noise, probs, sigma, D.Ng, D.E, D.k, nch, partial);
        balance_grad_rows_kernel<EMAX><<<grid, kBalTok, 0, st>>>(
            logits, bias, noise, probs, partial, static_cast<int>(nch), sigma, w_imp, w_load,
            D.Ng, D.E, D.k, losses, imp, load, dlogits);
    } else {
        if (nch > 0)
            balance_partial_kernel<EMAX><<<grid, 64 * kBalWaves, 0, st>>>(
                logits, bias, noise, probs, sigma, D.Ng, D.E, D.k, partial);
        balance_grad_kernel<EMAX><<<grid, 64 * kBalWaves, 0, st>>>(
            logits, bias, noise, probs, partial, static_cast<int>(nch), sigma, w_imp, w_load,
            D.Ng, D.E, D.k, losses, imp, load, dlogits);
    }
}

template <typename F>
void by_emax(int E, F f) {
    if (E <= 8) f(std::integral_constant<int, 8>{});
    else if (E <= 16) f(std::integral_constant<int, 16>{});
    else if (E <= 32) f(std::integral_constant<int, 32>{});
    else f(std::integral_constant<int, 64>{});
}

unsigned balance_chunks(const Dims& D) {
    unsigned n = 0;
    by_emax(D.E, [&](auto tag) { n = balance_chunks_t<decltype(tag)::value>(D); });
    return n;
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
    by_emax(D.E, [&](auto tag) {
        launch_balance<decltype(tag)::value>(D, logits, bias, noise, probs, sigma, w_imp, w_load,
                                             losses, imp, load, dlogits, partial, st);
    });
    return launch_status();
}

}  // namespace vmoe
