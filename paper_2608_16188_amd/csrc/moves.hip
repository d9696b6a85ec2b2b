// Dispatch, combine and their backward passes on gfx950.
//
// All four are HBM-bound gathers / scatters keyed by the routing metadata,
// moving rows in 16-byte vectors (fully coalesced). Float sums run in a fixed
// order (j ascending, then a fixed butterfly), so results are deterministic.
#include <type_traits>

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
};

// Rows of assignments j0 .. j0 + J - 1 of token t (-1: dropped or past k).
// The loads run in three independent rounds (slot and expert of every j,
// then the row bases, then the caller's rows), with indices clamped instead
// of branches, so the compiler issues each round at once.
template <int J>
struct Rows {
    long long r[J];
    __device__ __forceinline__ void fetch(const RouteMeta& m, int t, int j0) {
        const size_t a0 = static_cast<size_t>(t) * m.k;
        int s[J], e[J], rb[J];
#pragma unroll
        for (int jj = 0; jj < J; ++jj) {
            const int j = min(j0 + jj, m.k - 1);
            s[jj] = m.slot[a0 + j];
            e[jj] = m.idx[a0 + j];  // a valid expert for every assignment
        }
        const int g = t / m.Ng;
#pragma unroll
        for (int jj = 0; jj < J; ++jj) rb[jj] = m.row_base[g * m.E + e[jj]];
#pragma unroll
        for (int jj = 0; jj < J; ++jj)
            r[jj] = (j0 + jj < m.k && s[jj] >= 0)
                        ? static_cast<long long>(e[jj]) * m.G * m.C + rb[jj] + s[jj]
                        : -1;
    }
};

// Whether token t keeps any of its k assignments (a dropped one has slot -1).
// Under a skewed load most tokens keep none: the moves then skip their rows.
__device__ __forceinline__ bool keeps_any(const RouteMeta& m, int t) {
    const int32_t* s = m.slot + static_cast<size_t>(t) * m.k;
    bool any = false;
    for (int j = 0; j < m.k; ++j) any = any || s[j] >= 0;
    return any;
}

// The slots and experts of assignments j0 .. j0 + J - 1 of token t, clamped
// to k - 1 (all requested at once, no branch), and whether any of them with
// j < k is kept.
template <int J>
struct Assign {
    int s[J], e[J];
    __device__ __forceinline__ void fetch(const RouteMeta& m, int t, int j0) {
        const size_t a0 = static_cast<size_t>(t) * m.k;
#pragma unroll
        for (int jj = 0; jj < J; ++jj) {
            const int j = min(j0 + jj, m.k - 1);
            s[jj] = m.slot[a0 + j];
            e[jj] = m.idx[a0 + j];  // a valid expert for every assignment
        }
    }
    __device__ __forceinline__ bool any_kept(const RouteMeta& m, int j0) const {
        bool any = false;
#pragma unroll
        for (int jj = 0; jj < J; ++jj) any = any || (j0 + jj < m.k && s[jj] >= 0);
        return any;
    }
    // the row bases of the experts in t's group (requested, not yet used)
    __device__ __forceinline__ void row_bases(const RouteMeta& m, int t, int (&rb)[J]) const {
        const int g = t / m.Ng;
#pragma unroll
        for (int jj = 0; jj < J; ++jj) rb[jj] = m.row_base[g * m.E + e[jj]];
    }
    // expert-buffer rows (-1: dropped or past k)
    __device__ __forceinline__ void rows(const RouteMeta& m, int j0, const int (&rb)[J],
                                         long long (&r)[J]) const {
#pragma unroll
        for (int jj = 0; jj < J; ++jj)
            r[jj] = (j0 + jj < m.k && s[jj] >= 0)
                        ? static_cast<long long>(e[jj]) * m.G * m.C + rb[jj] + s[jj]
                        : -1;
    }
};

// Marks values as used here, so the loads that produce them stay where they
// were issued (all of a round together) instead of moving into the branches
// that consume them, where each would wait for its own round trip.
template <int J>
__device__ __forceinline__ void keep_issued(int (&v)[J]) {
#pragma unroll
    for (int i = 0; i < J; ++i) asm volatile("" : "+v"(v[i]));
}

// Flat element-wise mapping for the row moves without a reduction: item i is
// 16-byte vector v = i mod nvec of token t = i / nvec, so consecutive lanes
// touch consecutive bytes of a row and every lane is busy whatever d is. Each
// thread takes kItems items kBlock apart; every load of both items (data,
// then metadata) is issued before the first store.
constexpr int kBlock = 256;
constexpr int kItems = 2;
// J: assignments per pass (2 when k <= 2, else 4; larger k loops)

// Three rounds of straight-line loads: the slots and experts of both items'
// tokens; then their x rows (buffer loads whose offset is out of range for a
// token that keeps nothing, which read no memory) beside the row bases; then
// the stores. A thread neither of whose tokens keeps anything stops after the
// first round.
template <typename T, int kJ>
__global__ __launch_bounds__(kBlock) void dispatch_kernel(const T* __restrict__ x,
                                                          T* __restrict__ xe, RouteMeta m,
                                                          int nvec) {
    const long long total = static_cast<long long>(m.N) * nvec;
    const long long b0 = static_cast<long long>(blockIdx.x) * kBlock * kItems;
    const long long i0 = b0 + threadIdx.x;
    uint4* dst = reinterpret_cast<uint4*>(xe);
    static_assert(kItems == 2, "two items per thread");
    const long long ia = min(i0, total - 1), ib = min(i0 + kBlock, total - 1);
    const int ta = static_cast<int>(ia / nvec), tb = static_cast<int>(ib / nvec);
    const int ca = static_cast<int>(ia - static_cast<long long>(ta) * nvec);
    const int cb = static_cast<int>(ib - static_cast<long long>(tb) * nvec);
    Assign<kJ> aa, ab;
    aa.fetch(m, ta, 0);
    ab.fetch(m, tb, 0);
    bool ka, kb;
    if (m.k <= kJ) {
        ka = aa.any_kept(m, 0);
        kb = ab.any_kept(m, 0);
    } else {
        ka = keeps_any(m, ta);
        kb = keeps_any(m, tb);
    }
    if (!ka && !kb) return;
    // the block's items of x as one buffer (the row of x is read only when
    // some assignment of its token is kept)
    const long long nb = min(static_cast<long long>(kBlock) * kItems, total - b0);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(reinterpret_cast<const uint4*>(x) + b0, nb * 16);
    const uint4 va = buf_load16(rx, ka ? static_cast<uint32_t>(ia - b0) * 16u : kOutOfRange);
    const uint4 vb = buf_load16(rx, kb ? static_cast<uint32_t>(ib - b0) * 16u : kOutOfRange);
    for (int j0 = 0; j0 < m.k; j0 += kJ) {
        if (j0 > 0) {
            aa.fetch(m, ta, j0);
            ab.fetch(m, tb, j0);
        }
        int ba[kJ], bb[kJ];
        aa.row_bases(m, ta, ba);
        ab.row_bases(m, tb, bb);
        keep_issued(ba);
        keep_issued(bb);
        long long ra[kJ], rb[kJ];
        aa.rows(m, j0, ba, ra);
        ab.rows(m, j0, bb, rb);
#pragma unroll
        for (int jj = 0; jj < kJ; ++jj) {
            if (i0 < total && ra[jj] >= 0) dst[ra[jj] * nvec + ca] = va;
            if (i0 + kBlock < total && rb[jj] >= 0) dst[rb[jj] * nvec + cb] = vb;
        }
    }
}

// y[t] = sum over kept j (ascending) of gate[t, j] ye[row(t, j)], f32 sums.
// One wave per token: its routing metadata is read once per wave, and a
// token that keeps no assignment (most of them under a skewed load) writes
// its zero row right after that.
template <typename T, int kJ>
__global__ __launch_bounds__(64 * kWavesPerBlock) void combine_fwd_kernel(
    const T* __restrict__ ye, const float* __restrict__ gate, T* __restrict__ y, RouteMeta m,
    int nvec) {
    constexpr int VN = Vec<T>::n;
    constexpr int NV = 2;  // vectors per lane per pass: rows up to 128 vectors in one pass
    const int t = blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (t >= m.N) return;
    const uint4* src = reinterpret_cast<const uint4*>(ye);
    uint4* g_y = reinterpret_cast<uint4*>(y) + static_cast<size_t>(t) * nvec;
    for (int v0 = 0; v0 < nvec; v0 += 64 * NV) {
        float acc[NV][VN];
#pragma unroll
        for (int q = 0; q < NV; ++q)
#pragma unroll
            for (int i = 0; i < VN; ++i) acc[q][i] = 0.0f;
        for (int j0 = 0; j0 < m.k; j0 += kJ) {
            Rows<kJ> rows;
            rows.fetch(m, t, j0);
            float gj[kJ];
            uint4 r[kJ][NV];
#pragma unroll
            for (int jj = 0; jj < kJ; ++jj) {
                gj[jj] = gate[static_cast<size_t>(t) * m.k + min(j0 + jj, m.k - 1)];
                if (rows.r[jj] >= 0)
#pragma unroll
                    for (int q = 0; q < NV; ++q) {
                        const int v = v0 + lane + 64 * q;
                        if (v < nvec) r[jj][q] = src[rows.r[jj] * nvec + v];
                    }
            }
#pragma unroll
            for (int jj = 0; jj < kJ; ++jj) {
                if (rows.r[jj] < 0) continue;
#pragma unroll
                for (int q = 0; q < NV; ++q) {
                    float f[VN];
                    Vec<T>::unpack(r[jj][q], f);
#pragma unroll
                    for (int i = 0; i < VN; ++i) acc[q][i] = __builtin_fmaf(gj[jj], f[i], acc[q][i]);
                }
            }
        }
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int v = v0 + lane + 64 * q;
            if (v < nvec) g_y[v] = Vec<T>::pack(acc[q]);
        }
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
    const int t = blockIdx.x * kWavesPerBlock + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (t >= m.N) return;
    // a token that keeps no assignment has zero gate gradients and no dye
    // rows: its dy row is not read
    if (!keeps_any(m, t)) {
        for (int j = lane; j < m.k; j += 64) dgate[static_cast<size_t>(t) * m.k + j] = 0.0f;
        return;
    }
    const uint4* g_dy = reinterpret_cast<const uint4*>(dy) + static_cast<size_t>(t) * nvec;
    for (int v0 = 0; v0 < nvec; v0 += 64 * NV) {
        uint4 a[NV];
#pragma unroll
        for (int q = 0; q < NV; ++q) {
            const int v = v0 + lane + 64 * q;
            if (v < nvec) a[q] = g_dy[v];
        }
        for (int j = 0; j < m.k; ++j) {
            Rows<1> rj;
            rj.fetch(m, t, j);
            const long long row = rj.r[0];
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

// dx[t] = sum over kept j (ascending) of dxe[row(t, j)], f32, overwritten.
template <typename T, int kJ>
__global__ __launch_bounds__(kBlock) void dispatch_bwd_kernel(const T* __restrict__ dxe,
                                                              float* __restrict__ dx, RouteMeta m,
                                                              int nvec) {
    constexpr int VN = Vec<T>::n;
    const long long total = static_cast<long long>(m.N) * nvec;
    const long long i0 = static_cast<long long>(blockIdx.x) * kBlock * kItems + threadIdx.x;
    const uint4* src = reinterpret_cast<const uint4*>(dxe);
    float4* dst = reinterpret_cast<float4*>(dx);
    long long it[kItems];
    int tt[kItems], cc[kItems];
    float acc[kItems][VN];
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
        it[u] = min(i0 + u * kBlock, total - 1);
        tt[u] = static_cast<int>(it[u] / nvec);
        cc[u] = static_cast<int>(it[u] - static_cast<long long>(tt[u]) * nvec);
#pragma unroll
        for (int q = 0; q < VN; ++q) acc[u][q] = 0.0f;
    }
    for (int j0 = 0; j0 < m.k; j0 += kJ) {
        Rows<kJ> rows[kItems];
        uint4 r[kItems][kJ];
#pragma unroll
        for (int u = 0; u < kItems; ++u) rows[u].fetch(m, tt[u], j0);
#pragma unroll
        for (int u = 0; u < kItems; ++u)
#pragma unroll
            for (int jj = 0; jj < kJ; ++jj)
                if (rows[u].r[jj] >= 0) r[u][jj] = src[rows[u].r[jj] * nvec + cc[u]];
#pragma unroll
        for (int u = 0; u < kItems; ++u)
#pragma unroll
            for (int jj = 0; jj < kJ; ++jj) {
                if (rows[u].r[jj] < 0) continue;
                float f[VN];
                Vec<T>::unpack(r[u][jj], f);
#pragma unroll
                for (int q = 0; q < VN; ++q) acc[u][q] += f[q];
            }
    }
#pragma unroll
    for (int u = 0; u < kItems; ++u) {
        if (i0 + u * kBlock >= total) continue;
#pragma unroll
        for (int q = 0; q < VN / 4; ++q)
            dst[it[u] * (VN / 4) + q] = make_float4(acc[u][4 * q], acc[u][4 * q + 1],
                                                    acc[u][4 * q + 2], acc[u][4 * q + 3]);
    }
}

RouteMeta meta(const Dims& D, const int32_t* idx, const int32_t* slot, const int32_t* row_base) {
    return RouteMeta{idx, slot, row_base, D.N, D.Ng, D.E, D.k, D.C, D.G};
}

// The dispatch's permutation without its data: row_token[row(t, j)] = t for
// every kept assignment (rows no assignment lands on are left as they are).
// One thread per token, its assignments J at a time.
template <int J>
__global__ __launch_bounds__(kBlock) void row_token_kernel(int32_t* __restrict__ row_token,
                                                           RouteMeta m) {
    const int t = blockIdx.x * kBlock + threadIdx.x;
    if (t >= m.N) return;
    for (int j0 = 0; j0 < m.k; j0 += J) {
        Rows<J> r;
        r.fetch(m, t, j0);
#pragma unroll
        for (int jj = 0; jj < J; ++jj)
            if (r.r[jj] >= 0) row_token[r.r[jj]] = t;
    }
}

}  // namespace

vmoe_status row_token_launch(const Dims& D, const int32_t* idx, const int32_t* slot,
                             const int32_t* row_base, int32_t* row_token, hipStream_t st) {
    if (D.N == 0) return VMOE_OK;
    const RouteMeta m = meta(D, idx, slot, row_base);
    if (D.k <= 2)
        row_token_kernel<2><<<cdiv(D.N, kBlock), kBlock, 0, st>>>(row_token, m);
    else
        row_token_kernel<4><<<cdiv(D.N, kBlock), kBlock, 0, st>>>(row_token, m);
    return launch_status();
}

vmoe_status dispatch_launch(const Dims& D, const void* x, const int32_t* idx, const int32_t* slot,
                            const int32_t* row_base, void* xe, hipStream_t st) {
    if (D.N == 0) return VMOE_OK;
    const RouteMeta m = meta(D, idx, slot, row_base);
    const int nvec = D.d / (D.dtype == VMOE_BF16 ? 8 : 4);
    const unsigned grid = cdiv(static_cast<long long>(D.N) * nvec, kBlock * kItems);
    auto go = [&](auto jc) {
        constexpr int J = decltype(jc)::value;
        if (D.dtype == VMOE_BF16)
            dispatch_kernel<uint16_t, J><<<grid, kBlock, 0, st>>>(
                static_cast<const uint16_t*>(x), static_cast<uint16_t*>(xe), m, nvec);
        else
            dispatch_kernel<float, J><<<grid, kBlock, 0, st>>>(
                static_cast<const float*>(x), static_cast<float*>(xe), m, nvec);
    };
    if (D.k <= 2) go(std::integral_constant<int, 2>{});
    else go(std::integral_constant<int, 4>{});
    return launch_status();
}

vmoe_status combine_fwd_launch(const Dims& D, const void* ye, const int32_t* idx,
                               const int32_t* slot, const int32_t* row_base, const float* gate,
                               void* y, hipStream_t st) {
    if (D.N == 0) return VMOE_OK;
    const RouteMeta m = meta(D, idx, slot, row_base);
    const int nvec = D.d / (D.dtype == VMOE_BF16 ? 8 : 4);
    const unsigned grid = cdiv(D.N, kWavesPerBlock);  // one wave per token
    auto go = [&](auto jc) {
        constexpr int J = decltype(jc)::value;
        if (D.dtype == VMOE_BF16)
            combine_fwd_kernel<uint16_t, J><<<grid, 64 * kWavesPerBlock, 0, st>>>(
                static_cast<const uint16_t*>(ye), gate, static_cast<uint16_t*>(y), m, nvec);
        else
            combine_fwd_kernel<float, J><<<grid, 64 * kWavesPerBlock, 0, st>>>(
                static_cast<const float*>(ye), gate, static_cast<float*>(y), m, nvec);
    };
    if (D.k <= 2) go(std::integral_constant<int, 2>{});
    else go(std::integral_constant<int, 4>{});
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
    auto go = [&](auto jc) {
        constexpr int J = decltype(jc)::value;
        if (D.dtype == VMOE_BF16)
            dispatch_bwd_kernel<uint16_t, J><<<grid, kBlock, 0, st>>>(
                static_cast<const uint16_t*>(dxe), dx, m, nvec);
        else
            dispatch_bwd_kernel<float, J><<<grid, kBlock, 0, st>>>(
                static_cast<const float*>(dxe), dx, m, nvec);
    };
    if (D.k <= 2) go(std::integral_constant<int, 2>{});
    else go(std::integral_constant<int, 4>{});
    return launch_status();
}

}  // namespace vmoe
