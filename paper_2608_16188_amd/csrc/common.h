// Internal helpers shared by the libvmoe HIP sources (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/vmoe.h"

namespace vmoe {

// Largest expert count the routing kernels support (one 64-bit lane mask).
constexpr int kMaxExperts = 64;

// ------------------------------------------------------------ bf16 <-> f32

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest, ties to even (inputs are finite).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return static_cast<uint32_t>(f32_to_bf16(lo)) | (static_cast<uint32_t>(f32_to_bf16(hi)) << 16);
}

// Element load / store as f32 for the two activation dtypes.
template <typename T> struct Elem;
template <> struct Elem<float> {
    static __device__ __forceinline__ float load(const float* p, size_t i) { return p[i]; }
    static __device__ __forceinline__ void store(float* p, size_t i, float v) { p[i] = v; }
};
template <> struct Elem<uint16_t> {
    static __device__ __forceinline__ float load(const uint16_t* p, size_t i) {
        return bf16_to_f32(p[i]);
    }
    static __device__ __forceinline__ void store(uint16_t* p, size_t i, float v) {
        p[i] = f32_to_bf16(v);
    }
};

// ------------------------------------------------------------ shape

struct Dims {
    int N, G, Ng, d, f, E, k, C;
    int dtype;
    long long rows_per_expert() const { return static_cast<long long>(G) * C; }
};

// Host-side validation and derived sizes; returns VMOE_OK or an error.
vmoe_status make_dims(const vmoe_shape* s, Dims* out);

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

inline vmoe_status launch_status() {
    return hipGetLastError() == hipSuccess ? VMOE_OK : VMOE_ERR_HIP;
}

inline unsigned cdiv(long long a, long long b) { return static_cast<unsigned>((a + b - 1) / b); }

// Row of assignment (t, j) in the [E, G*C, width] buffers, or -1 if dropped.
__device__ __forceinline__ long long assignment_row(int t, int j, const int32_t* idx,
                                                    const int32_t* slot, const int32_t* row_base,
                                                    int k, int Ng, int E, int C, int G) {
    int s = slot[static_cast<size_t>(t) * k + j];
    if (s < 0) return -1;
    int e = idx[static_cast<size_t>(t) * k + j];
    int g = t / Ng;
    return static_cast<long long>(e) * G * C + row_base[g * E + e] + s;
}

}  // namespace vmoe
