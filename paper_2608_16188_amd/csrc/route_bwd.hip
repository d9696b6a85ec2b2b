// Backward through the gate into the router on gfx950.
//
// A block owns a chunk of tokens of one group and a slice of model columns;
// per token it forms dz = p * (dp - <p, dp>) (dp is non-zero only at the kept
// experts), adds dz W into dx and accumulates a per-chunk partial of
// dW_r[e, i] = sum_t dz[t,e] x[t,i]. A second kernel adds the partials over
// chunks in a fixed order (deterministic, no float atomics).
#include "common.h"

namespace vmoe {
namespace {

constexpr int kMinChunk = 64;
constexpr int kMaxChunk = 256;

// VEC consecutive columns of a token row as f32 (VEC * sizeof(T) bytes, aligned).
template <int VEC>
__device__ __forceinline__ void load_cols(const uint16_t* p, float (&v)[VEC]) {
    if constexpr (VEC == 4) {
        const uint2 u = *reinterpret_cast<const uint2*>(p);
        v[0] = bf16_to_f32(u.x & 0xFFFFu); v[1] = bf16_to_f32(u.x >> 16);
        v[2] = bf16_to_f32(u.y & 0xFFFFu); v[3] = bf16_to_f32(u.y >> 16);
    } else if constexpr (VEC == 2) {
        const uint32_t u = *reinterpret_cast<const uint32_t*>(p);
        v[0] = bf16_to_f32(u & 0xFFFFu); v[1] = bf16_to_f32(u >> 16);
    } else {
        v[0] = bf16_to_f32(*p);
    }
}
template <int VEC>
__device__ __forceinline__ void load_cols(const float* p, float (&v)[VEC]) {
    if constexpr (VEC == 4) {
        const float4 u = *reinterpret_cast<const float4*>(p);
        v[0] = u.x; v[1] = u.y; v[2] = u.z; v[3] = u.w;
    } else if constexpr (VEC == 2) {
        const float2 u = *reinterpret_cast<const float2*>(p);
        v[0] = u.x; v[1] = u.y;
    } else {
        v[0] = *p;
    }
}
template <int VEC>
__device__ __forceinline__ void store_cols(float* p, const float (&v)[VEC]) {
    if constexpr (VEC == 4) *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
    else if constexpr (VEC == 2) *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
    else *p = v[0];
}

// Columns per lane: the E x VEC router weights and E x VEC gradient partials
// of a lane stay in registers.
template <int EMAX> struct ColsPerLane { static constexpr int value = EMAX <= 8 ? 4 : (EMAX <= 16 ? 2 : 1); };

// A block owns a chunk of tch tokens of one group and 64 * VEC columns. It
// first forms dz = p * (dp - <p, dp>) of its tokens in LDS (dp non-zero only at
// kept experts); wave w then takes the chunk's tokens w, w + 4, ... (a whole
// row slice per token, so dz is a broadcast read) and does
// dx[t, cols] += sum_e dz[e] W[e, cols] and acc[e][cols] += dz[e] x[t, cols].
// The four waves' accumulators are added in wave order into the chunk's
// partial of dW_r.
template <typename T, int EMAX>
__global__ __launch_bounds__(256) void route_bwd_kernel(
    const T* __restrict__ x, const T* __restrict__ wr, const float* __restrict__ probs,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ slot,
    const float* __restrict__ dgate, float* __restrict__ dx, float* __restrict__ partial, int Ng,
    int d, int E, int k, int tch, int nch) {
    constexpr int VEC = ColsPerLane<EMAX>::value;
    constexpr int COLS = 64 * VEC;
    __shared__ float red[3][EMAX][COLS];  // waves 1..3 hand their partials to wave 0
    __shared__ float dzs[kMaxChunk][EMAX + 1];
    const int c = blockIdx.x, g = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int t0 = c * tch;
    const int ntok = min(tch, Ng - t0);
    const size_t tok0 = static_cast<size_t>(g) * Ng + t0;

    // dz of the chunk's tokens, one token per thread
    for (int tt = threadIdx.x; tt < ntok; tt += 256) {
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
    const int i0 = blockIdx.y * COLS + lane * VEC;
    const bool live = i0 < d;  // d is a multiple of 8, so a lane's columns are all in or all out

    const T* wg = wr + static_cast<size_t>(g) * E * d;
    float w[EMAX][VEC], acc[EMAX][VEC];
    const int ic = live ? i0 : 0;  // idle lanes read column 0 and discard it
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
        load_cols<VEC>(wg + static_cast<size_t>(e < E ? e : E - 1) * d + ic, w[e]);
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            w[e][v] = (e < E && live) ? w[e][v] : 0.0f;
            acc[e][v] = 0.0f;
        }
    }

    // U tokens of this wave per round: their loads are all issued first
    constexpr int U = EMAX <= 16 ? 4 : (EMAX <= 32 ? 2 : 1);
    for (int r0 = wave; r0 < ntok; r0 += 4 * U) {
        float xv[U][VEC], dv[U][VEC];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int tt = min(r0 + 4 * u, ntok - 1);
            const size_t t = tok0 + tt;
            if (live) {
                load_cols<VEC>(x + t * d + i0, xv[u]);
                load_cols<VEC>(dx + t * d + i0, dv[u]);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int tt = r0 + 4 * u;
            if (tt >= ntok) break;
            const size_t t = tok0 + tt;
            float dz[EMAX];
#pragma unroll
            for (int e = 0; e < EMAX; ++e) dz[e] = e < E ? dzs[tt][e] : 0.0f;
            if (live) {
                float out[VEC];
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    float s = 0.0f;
#pragma unroll
                    for (int e = 0; e < EMAX; ++e)
                        if (e < E) s = __builtin_fmaf(dz[e], w[e][v], s);
                    out[v] = dv[u][v] + s;
                }
                store_cols<VEC>(dx + t * d + i0, out);
#pragma unroll
                for (int e = 0; e < EMAX; ++e)
#pragma unroll
                    for (int v = 0; v < VEC; ++v) acc[e][v] = __builtin_fmaf(dz[e], xv[u][v], acc[e][v]);
            }
        }
    }
    if (!partial) return;
    if (wave > 0) {
#pragma unroll
        for (int e = 0; e < EMAX; ++e)
#pragma unroll
            for (int v = 0; v < VEC; ++v) red[wave - 1][e][lane * VEC + v] = acc[e][v];
    }
    __syncthreads();
    if (wave == 0 && live) {
        float* pg = partial + (static_cast<size_t>(g) * nch + c) * E * d;
#pragma unroll
        for (int e = 0; e < EMAX; ++e) {
            if (e < E) {
                float out[VEC];
#pragma unroll
                for (int v = 0; v < VEC; ++v)
                    out[v] = ((acc[e][v] + red[0][e][lane * VEC + v]) + red[1][e][lane * VEC + v]) +
                             red[2][e][lane * VEC + v];
                store_cols<VEC>(pg + static_cast<size_t>(e) * d + i0, out);
            }
        }
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
    // about 1024 blocks over (chunks, column blocks, groups); column blocks of
    // 256 columns (E <= 16) as the common case
    const int colblocks = static_cast<int>(cdiv(D.d, 256));
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
    dim3 grid(P.nch, cdiv(D.d, 64 * ColsPerLane<EMAX>::value), D.G);
    route_bwd_kernel<T, EMAX><<<grid, 256, 0, st>>>(
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
