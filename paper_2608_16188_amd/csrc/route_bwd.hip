// Backward through the gate into the router on gfx950.
//
// dz = p * (dp - <p, dp>) (dp is non-zero only at the kept experts) is formed
// per token chunk in LDS by each kernel that needs it. One kernel adds dz W_r
// into dx (token-parallel, W_r columns in registers); one forms per-chunk
// partials of dW_r[e, i] = sum_t dz[t,e] x[t,i] (skipped for frozen routers)
// and a third adds the partials over chunks in a fixed order (deterministic,
// no float atomics).
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

// Columns per lane: a lane keeps E x VEC router weights (dx kernel) or E x VEC
// gradient partials (dW kernel) in registers.
template <int EMAX> struct ColsPerLane { static constexpr int value = EMAX <= 32 ? 4 : 2; };

// dz[t, e] = p[t,e] (dp[t,e] - <p[t], dp[t]>), dp = dgate at the kept experts
// and 0 elsewhere, written once to the workspace so the two streaming kernels
// read contiguous rows of it. One thread per (token, expert): each forms its
// token's <p, dp> itself (k assignments, in j order), so all threads wait on
// two rounds of loads at most and the rows come out coalesced.
__global__ __launch_bounds__(256) void route_bwd_dz_kernel(const float* __restrict__ probs,
                                                           const int32_t* __restrict__ idx,
                                                           const int32_t* __restrict__ slot,
                                                           const float* __restrict__ dgate,
                                                           float* __restrict__ dz, int N, int E,
                                                           int k) {
    const long long q = static_cast<long long>(blockIdx.x) * 256 + threadIdx.x;
    if (q >= static_cast<long long>(N) * E) return;
    const size_t t = static_cast<size_t>(q / E);
    const int e = static_cast<int>(q - static_cast<long long>(t) * E);
    const float* pr = probs + t * E;
    float pdp = 0.0f, dp = 0.0f;
    bool kept = false;
    for (int j = 0; j < k; ++j) {
        const size_t a = t * k + j;
        if (slot[a] >= 0) {
            const int ej = idx[a];
            const float gj = dgate[a];
            pdp = __builtin_fmaf(pr[ej], gj, pdp);
            if (ej == e) {
                kept = true;
                dp = gj;
            }
        }
    }
    // kept: p (dgate - <p, dp>); other experts: -p <p, dp>
    dz[q] = kept ? pr[e] * (dp - pdp) : -pr[e] * pdp;
}

// The dz rows of tokens [tok0, tok0 + ntok) into LDS rows of EMAX floats
// (16-byte aligned, zero past E), coalesced, one round.
template <int EMAX>
__device__ __forceinline__ void stage_dz(float (*dzs)[EMAX], const float* __restrict__ dz,
                                         size_t tok0, int ntok, int E) {
    const float* src = dz + tok0 * E;
    for (int q = threadIdx.x; q < ntok * EMAX; q += 256) {
        const int t = q / EMAX, e = q % EMAX;
        dzs[t][e] = e < E ? src[t * E + e] : 0.0f;
    }
}

// A token's dz row from LDS into registers (broadcast 16-byte reads).
template <int EMAX>
__device__ __forceinline__ void read_dz(const float (*dzs)[EMAX], int t, float (&r)[EMAX]) {
#pragma unroll
    for (int e = 0; e < EMAX; e += 4) {
        const float4 v = *reinterpret_cast<const float4*>(&dzs[t][e]);
        r[e] = v.x; r[e + 1] = v.y; r[e + 2] = v.z; r[e + 3] = v.w;
    }
}

constexpr int kDxTokens = 64;  // tokens per dx block

// dx[t, cols] += sum_e dz[t, e] W[e, cols]. A block owns kDxTokens tokens of
// one group and 64 * VEC columns; the lane's W columns stay in registers and
// wave w takes the block's tokens w, w + 4, ... (dz is a broadcast LDS read),
// U tokens' dx loads in flight at a time.
template <typename T, int EMAX>
__global__ __launch_bounds__(256) void route_bwd_dx_kernel(
    const T* __restrict__ wr, const float* __restrict__ dz, float* __restrict__ dx, int Ng, int d,
    int E) {
    constexpr int VEC = ColsPerLane<EMAX>::value;
    constexpr int U = 4;
    __shared__ __attribute__((aligned(16))) float dzs[kDxTokens][EMAX];
    const int c = blockIdx.x, g = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int t0 = c * kDxTokens;
    const int ntok = min(kDxTokens, Ng - t0);
    const size_t tok0 = static_cast<size_t>(g) * Ng + t0;
    const int i0 = blockIdx.y * 64 * VEC + lane * VEC;
    const bool live = i0 < d;  // d is a multiple of 8: a lane's columns are all in or all out
    const int ic = live ? i0 : 0;
    const T* wg = wr + static_cast<size_t>(g) * E * d;
    float w[EMAX][VEC];
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
        load_cols<VEC>(wg + static_cast<size_t>(e < E ? e : E - 1) * d + ic, w[e]);
#pragma unroll
        for (int v = 0; v < VEC; ++v) w[e][v] = (e < E && live) ? w[e][v] : 0.0f;
    }
    // this wave's tokens are wave, wave + 4, ...; round r covers U of them, and
    // the dx loads of the next round are issued before this round's arithmetic
    auto load_round = [&](int r0, float (&dv)[U][VEC]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const size_t t = tok0 + min(r0 + 4 * u, ntok - 1);
            load_cols<VEC>(dx + t * d + ic, dv[u]);
        }
    };
    float dva[U][VEC], dvb[U][VEC];
    stage_dz<EMAX>(dzs, dz, tok0, ntok, E);
    if (wave < ntok) load_round(wave, dva);
    __syncthreads();
    if (!live) return;
    auto step = [&](int r0, float (&cur)[U][VEC], float (&nxt)[U][VEC]) {
        if (r0 + 4 * U < ntok) load_round(r0 + 4 * U, nxt);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int tt = r0 + 4 * u;
            if (tt < ntok) {
                float z[EMAX];
                read_dz<EMAX>(dzs, tt, z);
                float out[VEC];
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    float s = 0.0f;
#pragma unroll
                    for (int e = 0; e < EMAX; ++e)
                        if (e < E) s = __builtin_fmaf(z[e], w[e][v], s);
                    out[v] = cur[u][v] + s;
                }
                store_cols<VEC>(dx + (tok0 + tt) * d + i0, out);
            }
        }
    };
    for (int r0 = wave; r0 < ntok; r0 += 8 * U) {
        step(r0, dva, dvb);
        if (r0 + 4 * U < ntok) step(r0 + 4 * U, dvb, dva);
    }
}

// Per-chunk partial of dW_r[e, cols] = sum_t dz[t, e] x[t, cols]. A block owns
// a chunk of tch tokens of one group and 64 * VEC columns; wave w takes the
// chunk's tokens w, w + 4, ... with E x VEC accumulators per lane, and the four
// waves' partials are added in wave order.
template <typename T, int EMAX>
__global__ __launch_bounds__(256) void route_bwd_dw_kernel(
    const T* __restrict__ x, const float* __restrict__ dz, float* __restrict__ partial, int Ng,
    int d, int E, int tch, int nch) {
    constexpr int VEC = ColsPerLane<EMAX>::value;
    constexpr int COLS = 64 * VEC;
    constexpr int U = EMAX <= 16 ? 4 : 2;
    // dz of the chunk while streaming; afterwards waves 1..3 hand their partials
    // to wave 0 through the same LDS
    constexpr int DZ_FLOATS = kMaxChunk * EMAX, RED_FLOATS = 3 * EMAX * COLS;
    __shared__ __attribute__((aligned(16))) float lds[DZ_FLOATS > RED_FLOATS ? DZ_FLOATS : RED_FLOATS];
    float (*dzs)[EMAX] = reinterpret_cast<float (*)[EMAX]>(lds);
    float (*red)[EMAX][COLS] = reinterpret_cast<float (*)[EMAX][COLS]>(lds);
    const int c = blockIdx.x, g = blockIdx.z;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int t0 = c * tch;
    const int ntok = min(tch, Ng - t0);
    const size_t tok0 = static_cast<size_t>(g) * Ng + t0;
    const int i0 = blockIdx.y * COLS + lane * VEC;
    const bool live = i0 < d;
    float acc[EMAX][VEC];
#pragma unroll
    for (int e = 0; e < EMAX; ++e)
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[e][v] = 0.0f;
    stage_dz<EMAX>(dzs, dz, tok0, ntok, E);
    __syncthreads();
    if (live) {
        for (int r0 = wave; r0 < ntok; r0 += 4 * U) {
            float xv[U][VEC];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const size_t t = tok0 + min(r0 + 4 * u, ntok - 1);
                load_cols<VEC>(x + t * d + i0, xv[u]);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int tt = r0 + 4 * u;
                if (tt < ntok) {
                    float z[EMAX];
                    read_dz<EMAX>(dzs, tt, z);
#pragma unroll
                    for (int e = 0; e < EMAX; ++e)
#pragma unroll
                        for (int v = 0; v < VEC; ++v)
                            acc[e][v] = __builtin_fmaf(z[e], xv[u][v], acc[e][v]);
                }
            }
        }
    }
    __syncthreads();  // every wave is done reading dz
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
                 float* dx, float* dz, float* partial, hipStream_t st) {
    constexpr int COLS = 64 * ColsPerLane<EMAX>::value;
    route_bwd_dz_kernel<<<cdiv(static_cast<long long>(D.N) * D.E, 256), 256, 0, st>>>(
        probs, idx, slot, dgate, dz, D.N, D.E, D.k);
    dim3 gdx(cdiv(D.Ng, kDxTokens), cdiv(D.d, COLS), D.G);
    route_bwd_dx_kernel<T, EMAX><<<gdx, 256, 0, st>>>(static_cast<const T*>(wr), dz, dx, D.Ng,
                                                       D.d, D.E);
    if (partial) {
        dim3 gdw(P.nch, cdiv(D.d, COLS), D.G);
        route_bwd_dw_kernel<T, EMAX><<<gdw, 256, 0, st>>>(static_cast<const T*>(x), dz, partial,
                                                           D.Ng, D.d, D.E, P.tch, P.nch);
    }
}

template <typename T>
void launch_main_e(const Dims& D, const ChunkPlan& P, const void* x, const void* wr,
                   const float* probs, const int32_t* idx, const int32_t* slot,
                   const float* dgate, float* dx, float* dz, float* partial, hipStream_t st) {
    if (D.E <= 8)
        launch_main<T, 8>(D, P, x, wr, probs, idx, slot, dgate, dx, dz, partial, st);
    else if (D.E <= 16)
        launch_main<T, 16>(D, P, x, wr, probs, idx, slot, dgate, dx, dz, partial, st);
    else if (D.E <= 32)
        launch_main<T, 32>(D, P, x, wr, probs, idx, slot, dgate, dx, dz, partial, st);
    else
        launch_main<T, 64>(D, P, x, wr, probs, idx, slot, dgate, dx, dz, partial, st);
}

}  // namespace

// Workspace: dz [N, E] f32, then (router gradient wanted) the per-chunk
// partials [G, chunks, E, d] f32.
size_t dz_bytes(const Dims& D) {
    return (sizeof(float) * static_cast<size_t>(D.N) * D.E + 255) & ~static_cast<size_t>(255);
}

size_t route_bwd_workspace_bytes(const Dims& D) {
    const ChunkPlan P = plan(D);
    return dz_bytes(D) + sizeof(float) * static_cast<size_t>(D.G) * P.nch * D.E * D.d;
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
    float* dz = static_cast<float*>(ws);
    float* partial = dwr ? reinterpret_cast<float*>(static_cast<char*>(ws) + dz_bytes(D)) : nullptr;
    if (D.dtype == VMOE_BF16)
        launch_main_e<uint16_t>(D, P, x, wr, probs, idx, slot, dgate, dx, dz, partial, st);
    else
        launch_main_e<float>(D, P, x, wr, probs, idx, slot, dgate, dx, dz, partial, st);
    if (dwr)
        route_bwd_reduce_kernel<<<cdiv(total, 32), 256, 0, st>>>(partial, dwr, D.E, D.d, P.nch,
                                                                  total);
    return launch_status();
}

}  // namespace vmoe
