// Backward through the gate into the router on gfx950.
//
// A block owns a chunk of tokens of one group and 256 model columns. It first
// forms dz = p * (dp - <p, dp>) for its tokens in LDS (dp is non-zero only at
// the kept experts), then streams the columns: dx[t, i] += sum_e dz[t,e] W[e,i]
// and a per-chunk partial of dW_r[e, i] = sum_t dz[t,e] x[t,i]. A second
// kernel adds the partials over chunks in a fixed order (deterministic, no
// float atomics).
#include "common.h"

namespace vmoe {
namespace {

constexpr int kCols = 256;
constexpr int kMinChunk = 64;
constexpr int kMaxChunk = 256;

template <typename T> __device__ __forceinline__ float ld(const T* p, size_t i);
template <> __device__ __forceinline__ float ld<float>(const float* p, size_t i) { return p[i]; }
template <> __device__ __forceinline__ float ld<uint16_t>(const uint16_t* p, size_t i) {
    return bf16_to_f32(p[i]);
}

template <typename T, int EMAX>
__global__ __launch_bounds__(kCols) void route_bwd_kernel(
    const T* __restrict__ x, const T* __restrict__ wr, const float* __restrict__ probs,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ slot,
    const float* __restrict__ dgate, float* __restrict__ dx, float* __restrict__ partial, int Ng,
    int d, int E, int k, int tch, int nch) {
    __shared__ float dzs[kMaxChunk][EMAX + 1];
    const int c = blockIdx.x, g = blockIdx.z;
    const int t0 = c * tch;
    const int ntok = min(tch, Ng - t0);
    const size_t tok0 = static_cast<size_t>(g) * Ng + t0;

    for (int tt = threadIdx.x; tt < ntok; tt += kCols) {
        const size_t t = tok0 + tt;
        float pdp = 0.0f;
        for (int j = 0; j < k; ++j)
            if (slot[t * k + j] >= 0)
                pdp = __builtin_fmaf(probs[t * E + idx[t * k + j]], dgate[t * k + j], pdp);
        for (int e = 0; e < E; ++e) dzs[tt][e] = -probs[t * E + e] * pdp;
        for (int j = 0; j < k; ++j)
            if (slot[t * k + j] >= 0) {
                const int e = idx[t * k + j];
                dzs[tt][e] = probs[t * E + e] * (dgate[t * k + j] - pdp);
            }
    }
    __syncthreads();

    const int i = blockIdx.y * kCols + threadIdx.x;
    if (i >= d) return;
    const T* wg = wr + static_cast<size_t>(g) * E * d;
    float w[EMAX], pw[EMAX];
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
        w[e] = e < E ? ld(wg, static_cast<size_t>(e) * d + i) : 0.0f;
        pw[e] = 0.0f;
    }
    // 8 tokens per round: all 16 loads are issued before any arithmetic, so
    // each thread keeps many HBM requests in flight.
    constexpr int U = 8;
    for (int tt0 = 0; tt0 < ntok; tt0 += U) {
        float xv[U], dv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const size_t t = tok0 + min(tt0 + u, ntok - 1);
            xv[u] = ld(x, t * d + i);
            dv[u] = dx[t * d + i];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (tt0 + u >= ntok) break;
            float s = 0.0f;
#pragma unroll
            for (int e = 0; e < EMAX; ++e) {
                const float dz = dzs[tt0 + u][e < E ? e : 0];
                if (e < E) {
                    s = __builtin_fmaf(dz, w[e], s);
                    pw[e] = __builtin_fmaf(dz, xv[u], pw[e]);
                }
            }
            dx[(tok0 + tt0 + u) * d + i] = dv[u] + s;
        }
    }
    if (partial) {
        float* pg = partial + (static_cast<size_t>(g) * nch + c) * E * d;
#pragma unroll
        for (int e = 0; e < EMAX; ++e)
            if (e < E) pg[static_cast<size_t>(e) * d + i] = pw[e];
    }
}

// dW_r = sum over chunks of the partials. A block owns 32 outputs; 8 lane
// groups each add every 8th chunk (coalesced 128-byte rows), then the 8
// partial sums are added in a fixed order.
__global__ __launch_bounds__(256) void route_bwd_reduce_kernel(const float* __restrict__ partial,
                                                               float* __restrict__ dwr, int E,
                                                               int d, int nch, long long total) {
    __shared__ float part[8][33];
    const int ql = threadIdx.x & 31, r = threadIdx.x >> 5;
    const long long q = static_cast<long long>(blockIdx.x) * 32 + ql;
    const long long ed = static_cast<long long>(E) * d;
    float s = 0.0f;
    if (q < total && nch > 0) {
        const long long g = q / ed, o = q % ed;
        const float* p = partial + g * nch * ed + o;
        for (int c = r; c < nch; c += 8) s += p[c * ed];
    }
    part[r][ql] = s;
    __syncthreads();
    if (r == 0 && q < total) {
        float t = part[0][ql];
#pragma unroll
        for (int i = 1; i < 8; ++i) t += part[i][ql];
        dwr[q] = t;
    }
}

struct ChunkPlan {
    int tch, nch;
};

ChunkPlan plan(const Dims& D) {
    const int colblocks = static_cast<int>(cdiv(D.d, kCols));
    int target = 1024 / (D.G * colblocks);
    if (target < 1) target = 1;
    int tch = D.Ng > 0 ? static_cast<int>(cdiv(D.Ng, target)) : 1;
    tch = tch < kMinChunk ? kMinChunk : (tch > kMaxChunk ? kMaxChunk : tch);
    return ChunkPlan{tch, D.Ng > 0 ? static_cast<int>(cdiv(D.Ng, tch)) : 0};
}

template <typename T, int EMAX>
void launch_main(const Dims& D, const ChunkPlan& P, const void* x, const void* wr,
                 const float* probs, const int32_t* idx, const int32_t* slot, const float* dgate,
                 float* dx, float* partial, hipStream_t st) {
    dim3 grid(P.nch, cdiv(D.d, kCols), D.G);
    route_bwd_kernel<T, EMAX><<<grid, kCols, 0, st>>>(
        static_cast<const T*>(x), static_cast<const T*>(wr), probs, idx, slot, dgate, dx, partial,
        D.Ng, D.d, D.E, D.k, P.tch, P.nch);
}

template <typename T>
void launch_main_e(const Dims& D, const ChunkPlan& P, const void* x, const void* wr,
                   const float* probs, const int32_t* idx, const int32_t* slot,
                   const float* dgate, float* dx, float* partial, hipStream_t st) {
    if (D.E <= 8)
        launch_main<T, 8>(D, P, x, wr, probs, idx, slot, dgate, dx, partial, st);
    else if (D.E <= 16)
        launch_main<T, 16>(D, P, x, wr, probs, idx, slot, dgate, dx, partial, st);
    else if (D.E <= 32)
        launch_main<T, 32>(D, P, x, wr, probs, idx, slot, dgate, dx, partial, st);
    else
        launch_main<T, 64>(D, P, x, wr, probs, idx, slot, dgate, dx, partial, st);
}

}  // namespace

size_t route_bwd_workspace_bytes(const Dims& D) {
    const ChunkPlan P = plan(D);
    return sizeof(float) * static_cast<size_t>(D.G) * P.nch * D.E * D.d;
}

vmoe_status route_bwd_launch(const Dims& D, const void* x, const void* wr, const float* probs,
                             const int32_t* idx, const int32_t* slot, const float* dgate,
                             float* dx, float* dwr, void* ws, hipStream_t st) {
    const ChunkPlan P = plan(D);
    const long long total = static_cast<long long>(D.G) * D.E * D.d;
    if (D.N == 0) {
        // no tokens: the router gradient is zero (written by the reducer, nch = 0)
        if (dwr && total > 0)
            route_bwd_reduce_kernel<<<cdiv(total, 32), 256, 0, st>>>(nullptr, dwr, D.E, D.d, 0,
                                                                      total);
        return launch_status();
    }
    float* partial = dwr ? static_cast<float*>(ws) : nullptr;
    if (D.dtype == VMOE_BF16)
        launch_main_e<uint16_t>(D, P, x, wr, probs, idx, slot, dgate, dx, partial, st);
    else
        launch_main_e<float>(D, P, x, wr, probs, idx, slot, dgate, dx, partial, st);
    if (dwr)
        route_bwd_reduce_kernel<<<cdiv(total, 32), 256, 0, st>>>(partial, dwr, D.E, D.d, P.nch,
                                                                  total);
    return launch_status();
}

}  // namespace vmoe
