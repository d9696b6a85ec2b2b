// Dispatch, combine and their backward passes on gfx950.
//
// All four are HBM-bound gathers / scatters keyed by the routing metadata,
// moving rows in 16-byte vectors (fully coalesced). Float sums run in a fixed
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

// Flat element-wise mapping for the row moves without a reduction: item i is
// 16-byte vector v = i mod nvec of token t = i / nvec, so consecutive lanes
// touch consecutive bytes of a row and every lane is busy whatever d is. Each
// thread takes kItems items kBlock apart and issues all their loads before any
// store.
constexpr int kBlock = 256;
constexpr int kItems = 2;

template <typename T>
__global__ __launch_bounds__(kBlock) void dispatch_kernel(const T* __restrict__ x,
                                                          T* __restrict__ xe, RouteMeta m,
                                                          int nvec) {
    const long long total = static_cast<long long>(m.N) * nvec;
    const long long i0 = static_cast<long long>(blockIdx.x) * kBlock * kItems + threadIdx.x;
    const uint4* src = reinterpret_cast<const uint4*>(x);
    uint4* dst = reinterpret_cast<uint4*>(xe);
    auto item = [&](long long i) { return i < total ? src[i] : make_uint4(0u, 0u, 0u, 0u); };
    auto place = [&](long long i, const uint4 v) {
        if (i >= total) return;
        const int t = static_cast<int>(i / nvec);
        const int c = static_cast<int>(i - static_cast<long long>(t) * nvec);
        for (int j = 0; j < m.k; ++j) {
            const long long row = m.row(t, j);
            if (row >= 0) dst[row * nvec + c] = v;
        }
    };
    static_assert(kItems == 2, "two items per thread");
    const uint4 v0 = item(i0), v1 = item(i0 + kBlock);
    place(i0, v0);
    place(i0 + kBlock, v1);
}

template <typename T>
__global__ __launch_bounds__(kBlock) void combine_fwd_kernel(const T* __restrict__ ye,
                                                             const float* __restrict__ gate,
                                                             T* __restrict__ y, RouteMeta m,
                                                             int nvec) {
    constexpr int VN = Vec<T>::n;
    constexpr int KMAX = 4;  // rows gathered per pass; more assignments loop
    const long long total = static_cast<long long>(m.N) * nvec;
    const long long i0 = static_cast<long long>(blockIdx.x) * kBlock * kItems + threadIdx.x;
    const uint4* src = reinterpret_cast<const uint4*>(ye);
    uint4* dst = reinterpret_cast<uint4*>(y);
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
        const long long i = i0 + u * kBlock;
        if (i >= total) break;
        const int t = static_cast<int>(i / nvec), c = static_cast<int>(i - static_cast<long long>(t) * nvec);
        float acc[VN];
#pragma unroll
        for (int q = 0; q < VN; ++q) acc[q] = 0.0f;
        for (int j0 = 0; j0 < m.k; j0 += KMAX) {
            uint4 r[KMAX];
            float gj[KMAX];
            bool kept[KMAX];
#pragma unroll
            for (int jj = 0; jj < KMAX; ++jj) {
                const int j = j0 + jj;
                const long long row = j < m.k ? m.row(t, j) : -1;
                kept[jj] = row >= 0;
                gj[jj] = row >= 0 ? gate[static_cast<size_t>(t) * m.k + j] : 0.0f;
                r[jj] = row >= 0 ? src[row * nvec + c] : make_uint4(0u, 0u, 0u, 0u);
            }
            // j ascending over the kept assignments
#pragma unroll
            for (int jj = 0; jj < KMAX; ++jj) {
                if (!kept[jj]) continue;
                float f[VN];
                Vec<T>::unpack(r[jj], f);
#pragma unroll
                for (int q = 0; q < VN; ++q) acc[q] = __builtin_fmaf(gj[jj], f[q], acc[q]);
            }
        }
        dst[i] = Vec<T>::pack(acc);
    }
}

// One wave per token (the dot products reduce across the row): the token's dy
// vectors are loaded once, then per assignment all its ye vectors are loaded
// before the scaled copy and the dot product, which ends in a fixed butterfly.
template <typename T>
__global__ __launch_bounds__(64 * kWavesPerBlock) void combine_bwd_kernel(
    const T* __restrict__ dy, const T* __restrict__ ye, const float* __restrict__ gate,
    T* __restrict__ dye, float* __restrict__ dgate, RouteMeta m, int nvec) {
    constexpr int VN = Vec<T>::n;
    constexpr int NV = 2;  // vectors per lane per pass: rows up to 128 vectors in one pass
    const int t = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (t >= m.N) return;
    const uint4* g_dy = reinterpret_cast<const uint4*>(dy) + static_cast<size_t>(t) * nvec;
    for (int v0 = 0; v0 < nvec; v0 += 64 * NV) {
        uint4 a[NV];
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int v = v0 + lane + 64 * q;
            if (v < nvec) a[q] = g_dy[v];
        }
        for (int j = 0; j < m.k; ++j) {
            const long long row = m.row(t, j);
            if (row < 0) {
                if (lane == 0 && v0 == 0) dgate[static_cast<size_t>(t) * m.k + j] = 0.0f;
                continue;
            }
            const float gj = gate[static_cast<size_t>(t) * m.k + j];
            const uint4* g_ye = reinterpret_cast<const uint4*>(ye) + row * nvec;
            uint4* g_dye = reinterpret_cast<uint4*>(dye) + row * nvec;
            uint4 b[NV];
#pragma unroll
            for (int q = 0; q < NV; ++q) {
                const int v = v0 + lane + 64 * q;
                if (v < nvec) b[q] = g_ye[v];
            }
            float dot = 0.0f;
#pragma unroll
            for (int q = 0; q < NV; ++q) {
                const int v = v0 + lane + 64 * q;
                if (v >= nvec) break;
                float fa[VN], fb[VN], o[VN];
                Vec<T>::unpack(a[q], fa);
                Vec<T>::unpack(b[q], fb);
#pragma unroll
                for (int i = 0; i < VN; ++i) {
                    dot = __builtin_fmaf(fa[i], fb[i], dot);
                    o[i] = gj * fa[i];
                }
                g_dye[v] = Vec<T>::pack(o);
            }
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) dot += __shfl_xor(dot, o, 64);
            if (lane == 0) {
                float* dg = dgate + static_cast<size_t>(t) * m.k + j;
                *dg = v0 == 0 ? dot : *dg + dot;
            }
        }
    }
}

template <typename T>
__global__ __launch_bounds__(kBlock) void dispatch_bwd_kernel(const T* __restrict__ dxe,
                                                              float* __restrict__ dx, RouteMeta m,
                                                              int nvec) {
    constexpr int VN = Vec<T>::n;
    constexpr int KMAX = 4;
    const long long total = static_cast<long long>(m.N) * nvec;
    const long long i0 = static_cast<long long>(blockIdx.x) * kBlock * kItems + threadIdx.x;
    const uint4* src = reinterpret_cast<const uint4*>(dxe);
    float4* dst = reinterpret_cast<float4*>(dx);
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
        const long long i = i0 + u * kBlock;
        if (i >= total) break;
        const int t = static_cast<int>(i / nvec), c = static_cast<int>(i - static_cast<long long>(t) * nvec);
        float acc[VN];
#pragma unroll
        for (int q = 0; q < VN; ++q) acc[q] = 0.0f;
        for (int j0 = 0; j0 < m.k; j0 += KMAX) {
            uint4 r[KMAX];
            bool kept[KMAX];
#pragma unroll
            for (int jj = 0; jj < KMAX; ++jj) {
                const int j = j0 + jj;
                const long long row = j < m.k ? m.row(t, j) : -1;
                kept[jj] = row >= 0;
                r[jj] = row >= 0 ? src[row * nvec + c] : make_uint4(0u, 0u, 0u, 0u);
            }
            // j ascending over the kept assignments
#pragma unroll
            for (int jj = 0; jj < KMAX; ++jj) {
                if (!kept[jj]) continue;
                float f[VN];
                Vec<T>::unpack(r[jj], f);
#pragma unroll
                for (int q = 0; q < VN; ++q) acc[q] += f[q];
            }
        }
#pragma unroll
        for (int q = 0; q < VN / 4; ++q)
            dst[i * (VN / 4) + q] = make_float4(acc[4 * q], acc[4 * q + 1], acc[4 * q + 2],
                                                acc[4 * q + 3]);
    }
}

RouteMeta meta(const Dims& D, const int32_t* idx, const int32_t* slot, const int32_t* row_base) {
    return RouteMeta{idx, slot, row_base, D.N, D.Ng, D.E, D.k, D.C, D.G};
}

}  // namespace

vmoe_status dispatch_launch(const Dims& D, const void* x, const int32_t* idx, const int32_t* slot,
                            const int32_t* row_base, void* xe, hipStream_t st) {
    if (D.N == 0) return VMOE_OK;
    const RouteMeta m = meta(D, idx, slot, row_base);
    const int nvec = D.d / (D.dtype == VMOE_BF16 ? 8 : 4);
    const unsigned grid = cdiv(static_cast<long long>(D.N) * nvec, kBlock * kItems);
    if (D.dtype == VMOE_BF16)
        dispatch_kernel<uint16_t><<<grid, kBlock, 0, st>>>(
            static_cast<const uint16_t*>(x), static_cast<uint16_t*>(xe), m, nvec);
    else
        dispatch_kernel<float><<<grid, kBlock, 0, st>>>(
            static_cast<const float*>(x), static_cast<float*>(xe), m, nvec);
    return launch_status();
}

vmoe_status combine_fwd_launch(const Dims& D, const void* ye, const int32_t* idx,
                               const int32_t* slot, const int32_t* row_base, const float* gate,
                               void* y, hipStream_t st) {
    if (D.N == 0) return VMOE_OK;
    const RouteMeta m = meta(D, idx, slot, row_base);
    const int nvec = D.d / (D.dtype == VMOE_BF16 ? 8 : 4);
    const unsigned grid = cdiv(static_cast<long long>(D.N) * nvec, kBlock * kItems);
    if (D.dtype == VMOE_BF16)
        combine_fwd_kernel<uint16_t><<<grid, kBlock, 0, st>>>(
            static_cast<const uint16_t*>(ye), gate, static_cast<uint16_t*>(y), m, nvec);
    else
        combine_fwd_kernel<float><<<grid, kBlock, 0, st>>>(
            static_cast<const float*>(ye), gate, static_cast<float*>(y), m, nvec);
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
            static_cast<uint16_t*>(dye), dgate, m, D.d / 8);
    else
        combine_bwd_kernel<float><<<grid, 64 * kWavesPerBlock, 0, st>>>(
            static_cast<const float*>(dy), static_cast<const float*>(ye), gate,
            static_cast<float*>(dye), dgate, m, D.d / 4);
    return launch_status();
}

vmoe_status dispatch_bwd_launch(const Dims& D, const void* dxe, const int32_t* idx,
                                const int32_t* slot, const int32_t* row_base, float* dx,
                                hipStream_t st) {
    if (D.N == 0) return VMOE_OK;
    const RouteMeta m = meta(D, idx, slot, row_base);
    const int nvec = D.d / (D.dtype == VMOE_BF16 ? 8 : 4);
    const unsigned grid = cdiv(static_cast<long long>(D.N) * nvec, kBlock * kItems);
    if (D.dtype == VMOE_BF16)
        dispatch_bwd_kernel<uint16_t><<<grid, kBlock, 0, st>>>(
            static_cast<const uint16_t*>(dxe), dx, m, nvec);
    else
        dispatch_bwd_kernel<float><<<grid, kBlock, 0, st>>>(
            static_cast<const float*>(dxe), dx, m, nvec);
    return launch_status();
}

}  // namespace vmoe
