// Dispatch, combine and their backward passes on gfx950.
//
// All four are HBM-bound gathers / scatters keyed by the routing metadata.
// One 64-lane wavefront owns one token: it reads the token's k (expert, slot)
// pairs once and streams the d-wide rows in 16-byte vectors, so every row
// access is a fully coalesced 16 B-per-lane burst. Float sums run in a fixed
// order (j ascending, then a fixed butterfly), so results are deterministic.
#include "common.h"

namespace vmoe {
namespace {

constexpr int kWavesPerBlock = 4;

// 16-byte vector of activations, viewed as f32 lanes.
template <typename T> struct Vec;
template <> struct Vec<uint16_t> {
    static constexpr int n = 8;
    static __device__ __forceinline__ void unpack(const uint4& v, float* f) {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            f[2 * i] = __uint_as_float(w[i] << 16);
            f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
        }
    }
    static __device__ __forceinline__ uint4 pack(const float* f) {
        return make_uint4(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]),
                          pack_bf16x2(f[4], f[5]), pack_bf16x2(f[6], f[7]));
    }
};
template <> struct Vec<float> {
    static constexpr int n = 4;
    static __device__ __forceinline__ void unpack(const uint4& v, float* f) {
        f[0] = __uint_as_float(v.x);
        f[1] = __uint_as_float(v.y);
        f[2] = __uint_as_float(v.z);
        f[3] = __uint_as_float(v.w);
    }
    static __device__ __forceinline__ uint4 pack(const float* f) {
        return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                          __float_as_uint(f[3]));
    }
};

struct RouteMeta {
    const int32_t* idx;
    const int32_t* slot;
    const int32_t* row_base;
    int N, Ng, E, k, C, G;
    __device__ __forceinline__ long long row(int t, int j) const {
        return assignment_row(t, j, idx, slot, row_base, k, Ng, E, C, G);
    }
};

template <typename T>
__global__ __launch_bounds__(64 * kWavesPerBlock) void dispatch_kernel(const T* __restrict__ x,
                                                                        T* __restrict__ xe,
                                                                        RouteMeta m, int d) {
    const int t = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (t >= m.N) return;
    const int nvec = d / Vec<T>::n;
    const uint4* src = reinterpret_cast<const uint4*>(x + static_cast<size_t>(t) * d);
    for (int j = 0; j < m.k; ++j) {
        const long long row = m.row(t, j);
        if (row < 0) continue;
        uint4* dst = reinterpret_cast<uint4*>(xe + static_cast<size_t>(row) * d);
        for (int v = lane; v < nvec; v += 64) dst[v] = src[v];
    }
}

template <typename T>
__global__ __launch_bounds__(64 * kWavesPerBlock) void combine_fwd_kernel(
    const T* __restrict__ ye, const float* __restrict__ gate, T* __restrict__ y, RouteMeta m,
    int d) {
    constexpr int VN = Vec<T>::n;
    const int t = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (t >= m.N) return;
    const int nvec = d / VN;
    uint4* dst = reinterpret_cast<uint4*>(y + static_cast<size_t>(t) * d);
    for (int v = lane; v < nvec; v += 64) {
        float acc[VN];
#pragma unroll
        for (int i = 0; i < VN; ++i) acc[i] = 0.0f;
        for (int j = 0; j < m.k; ++j) {
            const long long row = m.row(t, j);
            if (row < 0) continue;
            const float gj = gate[static_cast<size_t>(t) * m.k + j];
            float f[VN];
            Vec<T>::unpack(reinterpret_cast<const uint4*>(ye + static_cast<size_t>(row) * d)[v], f);
#pragma unroll
            for (int i = 0; i < VN; ++i) acc[i] = __builtin_fmaf(gj, f[i], acc[i]);
        }
        dst[v] = Vec<T>::pack(acc);
    }
}

template <typename T>
__global__ __launch_bounds__(64 * kWavesPerBlock) void combine_bwd_kernel(
    const T* __restrict__ dy, const T* __restrict__ ye, const float* __restrict__ gate,
    T* __restrict__ dye, float* __restrict__ dgate, RouteMeta m, int d) {
    constexpr int VN = Vec<T>::n;
    const int t = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (t >= m.N) return;
    const int nvec = d / VN;
    const uint4* g_dy = reinterpret_cast<const uint4*>(dy + static_cast<size_t>(t) * d);
    for (int j = 0; j < m.k; ++j) {
        const long long row = m.row(t, j);
        if (row < 0) {
            if (lane == 0) dgate[static_cast<size_t>(t) * m.k + j] = 0.0f;
            continue;
        }
        const float gj = gate[static_cast<size_t>(t) * m.k + j];
        const uint4* g_ye = reinterpret_cast<const uint4*>(ye + static_cast<size_t>(row) * d);
        uint4* g_dye = reinterpret_cast<uint4*>(dye + static_cast<size_t>(row) * d);
        float dot = 0.0f;
        for (int v = lane; v < nvec; v += 64) {
            float a[VN], b[VN], o[VN];
            Vec<T>::unpack(g_dy[v], a);
            Vec<T>::unpack(g_ye[v], b);
#pragma unroll
            for (int i = 0; i < VN; ++i) {
                dot = __builtin_fmaf(a[i], b[i], dot);
                o[i] = gj * a[i];
            }
            g_dye[v] = Vec<T>::pack(o);
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) dot += __shfl_xor(dot, o, 64);
        if (lane == 0) dgate[static_cast<size_t>(t) * m.k + j] = dot;
    }
}

template <typename T>
__global__ __launch_bounds__(64 * kWavesPerBlock) void dispatch_bwd_kernel(
    const T* __restrict__ dxe, float* __restrict__ dx, RouteMeta m, int d) {
    constexpr int VN = Vec<T>::n;
    const int t = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (t >= m.N) return;
    const int nvec = d / VN;
    float4* dst = reinterpret_cast<float4*>(dx + static_cast<size_t>(t) * d);
    for (int v = lane; v < nvec; v += 64) {
        float acc[VN];
#pragma unroll
        for (int i = 0; i < VN; ++i) acc[i] = 0.0f;
        for (int j = 0; j < m.k; ++j) {
            const long long row = m.row(t, j);
            if (row < 0) continue;
            float f[VN];
            Vec<T>::unpack(reinterpret_cast<const uint4*>(dxe + static_cast<size_t>(row) * d)[v], f);
#pragma unroll
            for (int i = 0; i < VN; ++i) acc[i] += f[i];
        }
#pragma unroll
        for (int i = 0; i < VN / 4; ++i)
            dst[v * (VN / 4) + i] = make_float4(acc[4 * i], acc[4 * i + 1], acc[4 * i + 2],
                                                acc[4 * i + 3]);
    }
}

RouteMeta meta(const Dims& D, const int32_t* idx, const int32_t* slot, const int32_t* row_base) {
    return RouteMeta{idx, slot, row_base, D.N, D.Ng, D.E, D.k, D.C, D.G};
}

}  // namespace

vmoe_status dispatch_launch(const Dims& D, const void* x, const int32_t* idx, const int32_t* slot,
                            const int32_t* row_base, void* xe, hipStream_t st) {
    if (D.N == 0) return VMOE_OK;
    const unsigned grid = cdiv(D.N, kWavesPerBlock);
    const RouteMeta m = meta(D, idx, slot, row_base);
    if (D.dtype == VMOE_BF16)
        dispatch_kernel<uint16_t><<<grid, 64 * kWavesPerBlock, 0, st>>>(
            static_cast<const uint16_t*>(x), static_cast<uint16_t*>(xe), m, D.d);
    else
        dispatch_kernel<float><<<grid, 64 * kWavesPerBlock, 0, st>>>(
            static_cast<const float*>(x), static_cast<float*>(xe), m, D.d);
    return launch_status();
}

vmoe_status combine_fwd_launch(const Dims& D, const void* ye, const int32_t* idx,
                               const int32_t* slot, const int32_t* row_base, const float* gate,
                               void* y, hipStream_t st) {
    if (D.N == 0) return VMOE_OK;
    const unsigned grid = cdiv(D.N, kWavesPerBlock);
    const RouteMeta m = meta(D, idx, slot, row_base);
    if (D.dtype == VMOE_BF16)
        combine_fwd_kernel<uint16_t><<<grid, 64 * kWavesPerBlock, 0, st>>>(
            static_cast<const uint16_t*>(ye), gate, static_cast<uint16_t*>(y), m, D.d);
    else
        combine_fwd_kernel<float><<<grid, 64 * kWavesPerBlock, 0, st>>>(
            static_cast<const float*>(ye), gate, static_cast<float*>(y), m, D.d);
    return launch_status();
}

vmoe_status combine_bwd_launch(const Dims& D, const void* dy, const void* ye, const int32_t* idx,
                               const int32_t* slot, const int32_t* row_base, const float* gate,
                               void* dye, float* dgate, hipStream_t st) {
    if (D.N == 0) return VMOE_OK;
    const unsigned grid = cdiv(D.N, kWavesPerBlock);
    const RouteMeta m = meta(D, idx, slot, row_base);
    if (D.dtype == VMOE_BF16)
        combine_bwd_kernel<uint16_t><<<grid, 64 * kWavesPerBlock, 0, st>>>(
            static_cast<const uint16_t*>(dy), static_cast<const uint16_t*>(ye), gate,
            static_cast<uint16_t*>(dye), dgate, m, D.d);
    else
        combine_bwd_kernel<float><<<grid, 64 * kWavesPerBlock, 0, st>>>(
            static_cast<const float*>(dy), static_cast<const float*>(ye), gate,
            static_cast<float*>(dye), dgate, m, D.d);
    return launch_status();
}

vmoe_status dispatch_bwd_launch(const Dims& D, const void* dxe, const int32_t* idx,
                                const int32_t* slot, const int32_t* row_base, float* dx,
                                hipStream_t st) {
    if (D.N == 0) return VMOE_OK;
    const unsigned grid = cdiv(D.N, kWavesPerBlock);
    const RouteMeta m = meta(D, idx, slot, row_base);
    if (D.dtype == VMOE_BF16)
        dispatch_bwd_kernel<uint16_t><<<grid, 64 * kWavesPerBlock, 0, st>>>(
            static_cast<const uint16_t*>(dxe), dx, m, D.d);
    else
        dispatch_bwd_kernel<float><<<grid, 64 * kWavesPerBlock, 0, st>>>(
            static_cast<const float*>(dxe), dx, m, D.d);
    return launch_status();
}

}  // namespace vmoe
