// Internal helpers shared by the libvmoe HIP sources (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/vmoe.h"

namespace vmoe {

// Largest expert count the routing kernels support (one 64-bit lane mask).
constexpr int kMaxExperts = 64;

// Most rows per expert (G * C) whose token list the gathered weight-gradient
// GEMM keeps in LDS beside its stage ring.
constexpr int kGatherRows = 6144;
// Byte offset marking a gathered row or column outside the operand: the sum
// of a row's and a column's offset, either one this, lands at or past
// kGatherSentinel (no 32-bit wrap) and so past the end of x, whose size
// gathered calls bound by kGatherMaxBytes; the load returns zeros.
constexpr uint32_t kGatherSentinel = 0x7FFFFFF0u;
constexpr long long kGatherMaxBytes = kGatherSentinel;

// ------------------------------------------------------------ bf16 <-> f32

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two f32 -> two bf16 (round to nearest, ties to even) in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const f32x2_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    return static_cast<uint16_t>(pack_bf16x2(f, 0.0f) & 0xFFFFu);
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

// ------------------------------------------------------------ buffer loads

typedef int v4i32 __attribute__((ext_vector_type(4)));

// Raw buffer over `bytes` bytes at `base`: loads at byte offsets >= `bytes`
// return zeros in hardware, which implements tail masks without a branch.
constexpr uint32_t kOutOfRange = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, long long bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                             static_cast<int>(bytes), 0x00020000);
}

__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
    const v4i32 v = __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
}

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

}  // namespace vmoe
