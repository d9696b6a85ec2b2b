// Noisy top-k gating with capacity and batch-prioritized routing on gfx950.
//
// Pipeline (all on the caller's stream, no host synchronisation):
//   1. router        logits (bf16: matrix-core product, f32 accumulation;
//                    f32: double-accumulated in increasing i, rounded once),
//                    noisy softmax, top-k, 26-bit priority key; each block
//                    also records its keys' range
//   2. bin_hist      per 4096 tokens of a group: the group's key range (from
//                    the router blocks' ranges) -> 4096 bins spanning it,
//                    the block's bin histogram
//   3. bin_scatter   the same blocks: bin starts and the block's offset in
//                    each bin (sums of the group's histograms, scan over the
//                    bins), then its tokens into their bins (LDS cursors;
//                    order inside a bin is irrelevant, ranks are exact next)
//   4. rank          rank of each token = tokens in lower bins + tokens of its
//                    own bin that precede it by (key, index): a stable
//                    priority sort without passes; also counts, per chunk of
//                    256 order positions, the assignments to each expert
//   5. chunk_scan    one wave per (group, expert): over the rounds, the
//                    carry min(C, earlier demand) and the exclusive scan over
//                    chunks; counts; row_base
//   6. slots         per chunk: rank of each assignment among same-expert
//                    assignments (wave ballots + cross-wave prefix), slot =
//                    carry + rank, kept while slot < C
// A group of at most 8192 tokens may instead run steps 2-6 in one block
// (local_route), all in LDS.
// This file must be compiled with -ffp-contract=off: the gate's float
// arithmetic is specified operation by operation.
#include <type_traits>

#include "common.h"

namespace vmoe {
namespace {

constexpr int kKeyBits = 26;                 // priority keys fit in 26 bits for E <= 64
constexpr int kBinBits = 12;
constexpr int kNumBins = 1 << kBinBits;

// Bin of a key inside its group: (key - kmin) >> shift, with the group's
// smallest key kmin and the least shift that maps its key range onto the
// kNumBins bins (monotone in the key, so bins keep the priority order).
struct BinMap {
    uint32_t kmin;
    int shift;
    __device__ __forceinline__ int operator()(uint32_t key) const {
        return static_cast<int>((key - kmin) >> shift);
    }
};
constexpr int kSlotChunk = 256;              // order positions per slots block
constexpr int kGateTokens = 32;              // most tokens per f64 router block
constexpr int kMfmaTokens = 32;              // tokens per bf16 router block

constexpr int kHistTokens = 4096;             // tokens per bin_hist / bin_scatter block

struct RouteWs {
    uint32_t* keys;     // [N]
    uint2* kpart;       // [G][nkp] (min, max) key of each router block
    BinMap* binmap;     // [G]
    int32_t* bin_start; // [G][kNumBins + 1]
    int32_t* bhist;     // [G][nhb][kNumBins] bin counts of each hist block
    uint2* members;     // [N] (key, token) grouped by bin
    int32_t* ccount;    // [G][nch][k][E] (a chunk's counters side by side: rank's atomics)
    int32_t* cbase;     // [G][k][E][nch]
    int32_t* carry;     // [G][k][E]
    size_t bytes;
};

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// Tokens per f32 router block: one thread per (token, expert).
int f64_router_tokens(int E) { return kGateTokens < 256 / E ? kGateTokens : 256 / E; }

// Router blocks per group (each records one key range).
int router_blocks(const Dims& D) {
    if (D.dtype == VMOE_BF16) return static_cast<int>(cdiv(D.Ng, kMfmaTokens));
    return static_cast<int>(cdiv(D.Ng, f64_router_tokens(D.E)));
}

RouteWs route_ws_layout(const Dims& D, void* base) {
    char* p = static_cast<char*>(base);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char* q = p ? p + off : nullptr;
        off += align256(bytes);
        return q;
    };
    const size_t nch = cdiv(D.Ng, kSlotChunk);
    const size_t nhb = cdiv(D.Ng, kHistTokens);
    RouteWs w;
    w.keys = reinterpret_cast<uint32_t*>(take(sizeof(uint32_t) * D.N));
    w.kpart = reinterpret_cast<uint2*>(take(sizeof(uint2) * D.G * router_blocks(D)));
    w.binmap = reinterpret_cast<BinMap*>(take(sizeof(BinMap) * D.G));
    w.bin_start = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * D.G * (kNumBins + 1)));
    w.bhist = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * D.G * nhb * kNumBins));
    w.members = reinterpret_cast<uint2*>(take(sizeof(uint2) * D.N));
    w.ccount = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * D.G * nch * D.k * D.E));
    w.cbase = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * D.G * nch * D.k * D.E));
    w.carry = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * D.G * D.k * D.E));
    w.bytes = off;
    return w;
}

// exp(u) in f32: Cody-Waite reduction with a 9-bit high part of ln 2, degree-7
// Taylor polynomial by Horner with fused multiply-adds, exponent add. Below
// the smallest normal -> 0 (u < -87); u > 88 -> +inf; exp(0) = 1 exactly.
__device__ __forceinline__ float exp_spec(float u) {
    if (u < -87.0f) return 0.0f;
    if (u > 88.0f) return __builtin_inff();
    const float t = u * 1.44269504088896341f;
    const float n = __builtin_rintf(t);
    float r = __builtin_fmaf(-n, 0.693359375f, u);
    r = __builtin_fmaf(-n, -2.12194440e-4f, r);
    float p = 1.98412698e-4f;
    p = __builtin_fmaf(p, r, 1.38888889e-3f);
    p = __builtin_fmaf(p, r, 8.33333333e-3f);
    p = __builtin_fmaf(p, r, 4.16666667e-2f);
    p = __builtin_fmaf(p, r, 1.66666667e-1f);
    p = __builtin_fmaf(p, r, 0.5f);
    p = __builtin_fmaf(p, r, 1.0f);
    p = __builtin_fmaf(p, r, 1.0f);
    return __int_as_float(__float_as_int(p) + (static_cast<int>(n) << 23));
}

// Priority key: ascending key == descending priority p in (0, 1]. Values
// outside that range (never produced from finite logits) clamp to the last bin.
__device__ __forceinline__ uint32_t priority_key(float prio) {
    uint32_t bits = __float_as_uint(prio);
    uint32_t key = bits <= 0x3F800000u ? 0x3F800000u - bits : 0xFFFFFFFFu;
    return key < (1u << kKeyBits) ? key : (1u << kKeyBits) - 1u;
}

// Eight consecutive f32 activations (16-byte aligned).
__device__ __forceinline__ void load8(const float* p, float* v) {
    const float4 a = reinterpret_cast<const float4*>(p)[0];
    const float4 b = reinterpret_cast<const float4*>(p)[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

// Gate of token t from its logits in z[0..E) (LDS; overwritten by the noisy
// logits): perturb, deterministic softmax, top-k by z (ties to the lower
// expert), priority key of p[first choice].
__device__ __forceinline__ uint32_t gate_token(float* z, size_t t, const float* __restrict__ bias,
                                           const float* __restrict__ noise,
                                           float* __restrict__ probs, int32_t* __restrict__ idx,
                                           uint32_t* __restrict__ keys, int E, int k) {
    float m = 0.0f;
    for (int e = 0; e < E; ++e) {
        float v = z[e];
        if (bias) v = v + bias[e];
        if (noise) v = v + noise[t * E + e];
        z[e] = v;
        m = (e == 0 || v > m) ? v : m;
    }
    float s = 0.0f;
    for (int e = 0; e < E; ++e) s = s + exp_spec(z[e] - m);
    for (int e = 0; e < E; ++e) probs[t * E + e] = __fdiv_rn(exp_spec(z[e] - m), s);
    uint64_t taken = 0;
    int first = 0;
    for (int j = 0; j < k; ++j) {
        int best = -1;
        for (int e = 0; e < E; ++e)
            if (!((taken >> e) & 1ull) && (best < 0 || z[e] > z[best])) best = e;
        taken |= 1ull << best;
        idx[t * k + j] = best;
        if (j == 0) first = best;
    }
    const uint32_t key = priority_key(__fdiv_rn(exp_spec(z[first] - m), s));
    keys[t] = key;
    return key;
}

// Wave 0 of a router block (lanes < ntok hold its tokens' keys): the block's
// key range into kpart.
__device__ __forceinline__ void key_range(uint32_t key, int ntok, uint2* __restrict__ kpart) {
    const int lane = threadIdx.x & 63;
    uint32_t lo = lane < ntok ? key : 0xFFFFFFFFu, hi = lane < ntok ? key : 0u;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        lo = min(lo, static_cast<uint32_t>(__shfl_xor(static_cast<int>(lo), o, 64)));
        hi = max(hi, static_cast<uint32_t>(__shfl_xor(static_cast<int>(hi), o, 64)));
    }
    if (lane == 0) *kpart = make_uint2(lo, hi);
}

// The gate of a block's tokens, by the same operations in the same order as
// gate_token, split so that no lane repeats another's work: per (token,
// expert) pair the noisy logit, the exp term and the probability (lane e of a
// group of L = next power of two >= E lanes); per token (one thread) the
// maximum, the top-k scan and, once the terms are in, their sum in expert
// order. A token's row is read into EMAX >= E registers (independent reads).
template <int EMAX>
__device__ __forceinline__ void row_to_regs(const float* row, float (&r)[EMAX]) {
#pragma unroll
    for (int e = 0; e < EMAX; ++e) r[e] = row[e];  // entries past E are never used
}

// ---------------------------------------------------------------- bf16: MFMA
//
// One block = 32 tokens of one group, four waves. The router product
// x[32, d] W_r[g]^T runs on v_mfma_f32_32x32x16_bf16 (f32 accumulation), the
// d range split in four contiguous quarters, one per wave, whose partial
// products are added in wave order; A and B fragments are 16-byte loads of
// x rows and W_r rows straight from memory (both k-contiguous), eight k-steps
// in flight. Then the gate, in phases that meet at LDS-only barriers: per
// (token, expert) pair the noisy logit, per token the maximum and top-k, per
// pair the exp terms, per token their sum and the priority key, per pair the
// probabilities — each element by gate_token's operations in its order.
typedef __bf16 bf16x8_r __attribute__((ext_vector_type(8)));
typedef float f32x16_r __attribute__((ext_vector_type(16)));

// Barrier for data exchanged through LDS only: waits for this wave's LDS
// accesses (lgkmcnt(0)), not for its global stores.
__device__ __forceinline__ void lds_barrier() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

template <bool WIDE>
__global__ __launch_bounds__(256) void router_mfma_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ wr,
    const float* __restrict__ bias, const float* __restrict__ noise, float* __restrict__ logits,
    float* __restrict__ probs, int32_t* __restrict__ idx, uint32_t* __restrict__ keys,
    uint2* __restrict__ kpart, int Ng, int d, int E, int k, int logits_in) {
    // partial products, then z and the exp terms: one row per token (padded)
    constexpr int RW = WIDE ? kMaxExperts + 1 : 33;
    __shared__ __attribute__((aligned(16))) float red[4][kMfmaTokens][RW];
    const int g = blockIdx.y;
    const int t0 = blockIdx.x * kMfmaTokens;
    const int ntok = min(kMfmaTokens, Ng - t0);
    const size_t tok0 = static_cast<size_t>(g) * Ng + t0;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (!logits_in) {
        const __amdgpu_buffer_rsrc_t rx =
            make_rsrc(x + tok0 * d, static_cast<long long>(ntok) * d * 2);
        const __amdgpu_buffer_rsrc_t rw =
            make_rsrc(wr + static_cast<size_t>(g) * E * d, static_cast<long long>(E) * d * 2);
        const int ksteps = (d + 15) / 16;
        const int per = (ksteps + 3) / 4;
        const int s0 = wave * per, s1 = min(ksteps, s0 + per);
        const int m = lane & 31, kh = (lane >> 5) * 8;
        f32x16_r acc0, acc1;
#pragma unroll
        for (int r = 0; r < 16; ++r) acc0[r] = acc1[r] = 0.0f;
        // eight k-steps in flight per round. The tokens' x rows arrive as
        // coalesced 128-byte pieces (load i: row 8 i + lane / 8, elements
        // 8 (lane % 8) .. + 7 of a 64-deep group) and pass through this wave's
        // slice of `red` (free until the products are done; 16-byte chunks
        // XOR-swizzled by row so the fragment reads miss no bank) to become
        // the same fragments a direct load would give; the router rows are
        // read straight into fragments (few, and shared by every block in L2).
        const int klim = min(d, s1 * 16);
        // 16-byte vector (row r, columns kk..kk+7), zero outside the rows or
        // past this wave's k range
        auto offk = [&](int r, int rows, int kk) {
            return (r < rows && kk < klim) ? static_cast<uint32_t>(r * d + kk) * 2u : kOutOfRange;
        };
        typedef __attribute__((address_space(3))) v4i32 lds_v4;
        lds_v4* const stage = (lds_v4*)(&red[wave][0][0]);  // 32 rows x 8 chunks of 16 bytes
        static_assert(kMfmaTokens * 64 * 2 <= kMfmaTokens * RW * 4, "a row group fits the slice");
        constexpr int U = 8;
        for (int s = s0; s < s1; s += U) {
            uint4 ax[2][4], bv0[U], bv1[U];
#pragma unroll
            for (int gi = 0; gi < 2; ++gi)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    ax[gi][i] = buf_load16(rx, offk(8 * i + (lane >> 3), ntok,
                                                    (s + 4 * gi) * 16 + 8 * (lane & 7)));
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int kk = (s + u) * 16 + kh;
                bv0[u] = buf_load16(rw, offk(m, E, kk));
                if constexpr (WIDE) bv1[u] = buf_load16(rw, offk(32 + m, E, kk));
            }
            // keep every load of the round ahead of the first MFMA (the
            // scheduler would otherwise interleave them, two loads in flight)
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int gi = 0; gi < 2; ++gi) {
                // one wave's LDS accesses run in order: the previous group's
                // fragment reads are done before these writes
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int r = 8 * i + (lane >> 3);
                    stage[r * 8 + ((lane & 7) ^ (r & 7))] = __builtin_bit_cast(v4i32, ax[gi][i]);
                }
                bf16x8_r af[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int c = 2 * q + (lane >> 5);
                    af[q] = __builtin_bit_cast(bf16x8_r, stage[m * 8 + (c ^ (m & 7))]);
                }
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        __builtin_bit_cast(bf16x8_r, bv0[4 * gi + q]), af[q], acc0, 0, 0, 0);
                    if constexpr (WIDE)
                        acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            __builtin_bit_cast(bf16x8_r, bv1[4 * gi + q]), af[q], acc1, 0, 0, 0);
                }
            }
        }
        // register 4q + r of lane l: token l % 32, expert 8q + 4 (l / 32) + r (+ 32)
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int n = 8 * q + 4 * (lane >> 5) + r;
                red[wave][m][n] = acc0[4 * q + r];
                if constexpr (WIDE) red[wave][m][32 + n] = acc1[4 * q + r];
            }
    }
    __syncthreads();
    // pairs (token t, expert e): lane e of a group of L lanes, 256 / L tokens a pass
    int lsh = 0;
    while ((1 << lsh) < E) ++lsh;
    const int sub = tid & ((1 << lsh) - 1), tg = tid >> lsh, tp = 256 >> lsh;
    __shared__ float m_s[kMfmaTokens], s_s[kMfmaTokens];
    __shared__ int first_s[kMfmaTokens];
    // 1. the logit (the four waves' partials in wave order, or the input),
    //    then the noisy logit z = (logit + bias) + noise in place of wave 1's partial
    for (int t = tg; t < ntok; t += tp) {
        if (sub < E) {
            float v;
            if (logits_in) {
                v = logits[(tok0 + t) * E + sub];
            } else {
                v = ((red[0][t][sub] + red[1][t][sub]) + red[2][t][sub]) + red[3][t][sub];
                logits[(tok0 + t) * E + sub] = v;
            }
            if (bias) v = v + bias[sub];
            if (noise) v = v + noise[(tok0 + t) * E + sub];
            red[1][t][sub] = v;
        }
    }
    lds_barrier();
    // 2. per token: the maximum and the top-k choices (larger z, then lower expert)
    auto choose = [&](auto emax) {
        constexpr int EM = decltype(emax)::value;
        float z[EM];
        row_to_regs<EM>(&red[1][tid][0], z);
        float m = z[0];
#pragma unroll
        for (int e = 1; e < EM; ++e)
            if (e < E) m = z[e] > m ? z[e] : m;
        uint64_t taken = 0;
        for (int j = 0; j < k; ++j) {
            int best = -1;
            float bz = 0.0f;
#pragma unroll
            for (int e = 0; e < EM; ++e) {
                if (e < E && !((taken >> e) & 1ull) && (best < 0 || z[e] > bz)) {
                    best = e;
                    bz = z[e];
                }
            }
            taken |= 1ull << best;
            idx[(tok0 + tid) * k + j] = best;
            if (j == 0) first_s[tid] = best;
        }
        m_s[tid] = m;
    };
    if (tid < ntok) {
        if (E <= 8) choose(std::integral_constant<int, 8>{});
        else if (E <= 16) choose(std::integral_constant<int, 16>{});
        else if (E <= 32 || !WIDE) choose(std::integral_constant<int, 32>{});
        else choose(std::integral_constant<int, 64>{});
    }
    lds_barrier();
    // 3. the exp terms q = exp(z - m), in place of wave 2's partial
    for (int t = tg; t < ntok; t += tp)
        if (sub < E) red[2][t][sub] = exp_spec(red[1][t][sub] - m_s[t]);
    lds_barrier();
    // 4. per token: s = sum of the terms in expert order; the priority key
    uint32_t key = 0u;
    auto total = [&](auto emax) {
        constexpr int EM = decltype(emax)::value;
        float q[EM];
        row_to_regs<EM>(&red[2][tid][0], q);
        float sum = 0.0f;
#pragma unroll
        for (int e = 0; e < EM; ++e)
            if (e < E) sum = sum + q[e];
        s_s[tid] = sum;
        key = priority_key(__fdiv_rn(red[2][tid][first_s[tid]], sum));
        keys[tok0 + tid] = key;
    };
    if (tid < ntok) {
        if (E <= 8) total(std::integral_constant<int, 8>{});
        else if (E <= 16) total(std::integral_constant<int, 16>{});
        else if (E <= 32 || !WIDE) total(std::integral_constant<int, 32>{});
        else total(std::integral_constant<int, 64>{});
    }
    if (wave == 0) key_range(key, ntok, kpart + static_cast<size_t>(g) * gridDim.x + blockIdx.x);
    lds_barrier();
    // 5. the probabilities p = q / s (IEEE division)
    for (int t = tg; t < ntok; t += tp)
        if (sub < E) probs[(tok0 + t) * E + sub] = __fdiv_rn(red[2][t][sub], s_s[t]);
}

// ------------------------------------------------------------ f32: f64 sums
//
// f32 activations: logit (token, expert) is a sequential dot product in
// double over increasing i (each product of two f32 values is exact in
// double, so the fused multiply-add rounds once per step). One block =
// tpb = min(32, floor(256 / E)) tokens of one group; thread tid < tpb*E owns
// one (token, expert); the block's x rows and the group's router rows are
// staged through LDS 128 columns at a time (coalesced 16-byte loads, next
// slice prefetched in registers).
constexpr int kGateVecs = 32;  // 16-byte vectors per staged row and round

__global__ __launch_bounds__(256) void router_f64_kernel(
    const float* __restrict__ x, const float* __restrict__ wr, const float* __restrict__ bias,
    const float* __restrict__ noise, float* __restrict__ logits, float* __restrict__ probs,
    int32_t* __restrict__ idx, uint32_t* __restrict__ keys, uint2* __restrict__ kpart, int Ng,
    int d, int E, int k, int logits_in, int tpb) {
    constexpr int VE = 4;                          // f32 per 16-byte vector
    constexpr int VPR = kGateVecs;                 // vectors per staged row
    constexpr int GC = VPR * VE;                   // columns per round
    constexpr int LDR = GC + VE;                   // LDS row length (elements)
    constexpr int MAXROWS = kGateTokens + kMaxExperts;
    __shared__ __attribute__((aligned(16))) float stage[MAXROWS * LDR];
    __shared__ float lg_store[kGateTokens * (kMaxExperts + 1)];
    const int g = blockIdx.y;
    const int t0 = blockIdx.x * tpb;                  // within group
    const int ntok = min(tpb, Ng - t0);
    const size_t tok0 = static_cast<size_t>(g) * Ng + t0;  // global index
    const int tid = threadIdx.x;
    const int ld = E + 1;                             // LDS row of one token's logits
    if (!logits_in) {
        // staged rows: ntok token rows, then E router rows
        const int rows = ntok + E;
        const float* wg = wr + static_cast<size_t>(g) * E * d;
        constexpr int MAXV = (MAXROWS * VPR + 255) / 256;  // vectors per thread per round
        const int nvec = rows * VPR;
        uint4 pre[MAXV];
        auto fetch = [&](int c0) {
#pragma unroll
            for (int q = 0; q < MAXV; ++q) {
                const int v = tid + 256 * q;
                const int r = v / VPR, col = c0 + (v % VPR) * VE;
                pre[q] = make_uint4(0u, 0u, 0u, 0u);
                if (v < nvec && col < d) {
                    const float* src = r < ntok ? x + (tok0 + r) * d + col
                                                : wg + static_cast<size_t>(r - ntok) * d + col;
                    pre[q] = *reinterpret_cast<const uint4*>(src);
                }
            }
        };
        auto park = [&]() {
#pragma unroll
            for (int q = 0; q < MAXV; ++q) {
                const int v = tid + 256 * q;
                if (v < nvec)
                    *reinterpret_cast<uint4*>(stage + (v / VPR) * LDR + (v % VPR) * VE) = pre[q];
            }
        };
        const bool mine = tid < ntok * E;
        const int tt = tid / E, e = tid % E;
        const float* xs = stage + tt * LDR;
        const float* wsr = stage + (ntok + e) * LDR;
        double acc = 0.0;
        fetch(0);
        for (int c0 = 0; c0 < d; c0 += GC) {
            park();
            __syncthreads();
            if (c0 + GC < d) fetch(c0 + GC);
            if (mine) {
                const int n = min(GC, d - c0);  // a multiple of 8
                for (int i = 0; i < n; i += 8) {
                    float xv[8], wv[8];
                    load8(xs + i, xv);
                    load8(wsr + i, wv);
#pragma unroll
                    for (int q = 0; q < 8; ++q)
                        acc = __builtin_fma(static_cast<double>(xv[q]), static_cast<double>(wv[q]),
                                            acc);
                }
            }
            __syncthreads();
        }
        if (mine) {
            const float v = static_cast<float>(acc);
            logits[(tok0 + tt) * E + e] = v;
            lg_store[tt * ld + e] = v;
        }
    } else if (tid < ntok * E) {
        const int tt = tid / E, e = tid % E;
        lg_store[tt * ld + e] = logits[(tok0 + tt) * E + e];
    }
    __syncthreads();
    uint32_t key = 0u;
    if (tid < ntok)
        key = gate_token(lg_store + tid * ld, tok0 + tid, bias, noise, probs, idx, keys, E, k);
    if (tid < 64) key_range(key, ntok, kpart + static_cast<size_t>(g) * gridDim.x + blockIdx.x);
}

// Exclusive scan of one value per thread over a 1024-thread block.
__device__ int block_exclusive_scan_1024(int v, int* total) {
    __shared__ int wsum[16];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        int u = __shfl_up(inc, o, 64);
        if (lane >= o) inc += u;
    }
    if (lane == 63) wsum[w] = inc;
    __syncthreads();
    if (w == 0) {
        int s = lane < 16 ? wsum[lane] : 0;
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
            int u = __shfl_up(s, o, 64);
            if (lane >= o) s += u;
        }
        if (lane < 16) wsum[lane] = s;  // inclusive wave totals
    }
    __syncthreads();
    int base = w > 0 ? wsum[w - 1] : 0;
    *total = wsum[15];
    __syncthreads();
    return base + inc - v;
}

// The key range of group g from its router blocks' ranges -> the bin map
// (every block that needs it computes the same one from the same ranges).
__device__ BinMap group_binmap(const uint2* __restrict__ kpart, int nkp) {
    __shared__ uint32_t wmin[16], wmax[16];
    __shared__ BinMap map;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
    uint32_t lo = 0xFFFFFFFFu, hi = 0u;
    for (int i = threadIdx.x; i < nkp; i += blockDim.x) {
        const uint2 v = kpart[i];
        lo = min(lo, v.x);
        hi = max(hi, v.y);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        lo = min(lo, static_cast<uint32_t>(__shfl_xor(static_cast<int>(lo), o, 64)));
        hi = max(hi, static_cast<uint32_t>(__shfl_xor(static_cast<int>(hi), o, 64)));
    }
    if (lane == 0) {
        wmin[w] = lo;
        wmax[w] = hi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t a = wmin[0], z = wmax[0];
        for (int q = 1; q < nw; ++q) {
            a = min(a, wmin[q]);
            z = max(z, wmax[q]);
        }
        int sh = 0;
        while (((z - a) >> sh) >= static_cast<uint32_t>(kNumBins)) ++sh;
        map = BinMap{a, sh};
    }
    __syncthreads();
    return map;
}

constexpr int kHistPer = kHistTokens / 1024;  // tokens per thread of a hist block

// This block's kHistTokens tokens of group g (past Ng: not used).
__device__ __forceinline__ void hist_keys(const uint32_t* __restrict__ keys, int g, int Ng,
                                          uint32_t (&kv)[kHistPer]) {
    const size_t t0 = static_cast<size_t>(g) * Ng;
#pragma unroll
    for (int u = 0; u < kHistPer; ++u) {
        const int t = blockIdx.x * kHistTokens + u * 1024 + static_cast<int>(threadIdx.x);
        kv[u] = t < Ng ? keys[t0 + t] : 0u;
    }
}

// Block (j, g): the bin histogram of tokens [j kHistTokens, (j + 1) kHistTokens)
// of group g, into bhist[g][j].
__global__ __launch_bounds__(1024) void bin_hist_kernel(const uint32_t* __restrict__ keys,
                                                        const uint2* __restrict__ kpart, int nkp,
                                                        BinMap* __restrict__ binmap,
                                                        int32_t* __restrict__ bhist,
                                                        int32_t* __restrict__ ccount,
                                                        int cc_per_group, int Ng) {
    __shared__ int hist[kNumBins];
    const int g = blockIdx.y, tid = threadIdx.x;
    uint32_t kv[kHistPer];
    hist_keys(keys, g, Ng, kv);
    for (int b = tid; b < kNumBins; b += 1024) hist[b] = 0;
    const BinMap bm = group_binmap(kpart + static_cast<size_t>(g) * nkp, nkp);
    if (blockIdx.x == 0 && tid == 0) binmap[g] = bm;
#pragma unroll
    for (int u = 0; u < kHistPer; ++u)
        if (static_cast<int>(blockIdx.x) * kHistTokens + u * 1024 + tid < Ng)
            atomicAdd(&hist[bm(kv[u])], 1);
    __syncthreads();
    int32_t* out = bhist + (static_cast<size_t>(g) * gridDim.x + blockIdx.x) * kNumBins;
    for (int b = tid; b < kNumBins; b += 1024) out[b] = hist[b];
    // the group's chunk counters, which the rank step adds into, cleared
    int32_t* cg = ccount + static_cast<size_t>(g) * cc_per_group;
    for (int q = blockIdx.x * 1024 + tid; q < cc_per_group; q += gridDim.x * 1024) cg[q] = 0;
}

// Block (j, g): the tokens bin_hist counted into their bins. Bin b starts
// after the tokens of the bins below it, and this block's tokens of bin b
// after those of hist blocks j' < j (both from the hist rows of the group:
// per thread four consecutive bins, summed over the blocks, then a block scan
// over the bins); cursors in LDS from there. Block 0 stores the bin starts.
__global__ __launch_bounds__(1024) void bin_scatter_kernel(const uint32_t* __restrict__ keys,
                                                           const BinMap* __restrict__ binmap,
                                                           const int32_t* __restrict__ bhist,
                                                           int32_t* __restrict__ bin_start,
                                                           uint2* __restrict__ members, int Ng) {
    static_assert(kNumBins == 4 * 1024, "four consecutive bins per thread");
    __shared__ int cur[kNumBins];
    const int g = blockIdx.y, j = blockIdx.x, nhb = gridDim.x, tid = threadIdx.x;
    uint32_t kv[kHistPer];
    hist_keys(keys, g, Ng, kv);
    const int4* hb = reinterpret_cast<const int4*>(bhist + static_cast<size_t>(g) * nhb * kNumBins) + tid;
    int4 before = make_int4(0, 0, 0, 0), tot = make_int4(0, 0, 0, 0);
#pragma unroll 8
    for (int i = 0; i < nhb; ++i) {
        const int4 v = hb[static_cast<size_t>(i) * (kNumBins / 4)];
        if (i < j) {
            before.x += v.x;
            before.y += v.y;
            before.z += v.z;
            before.w += v.w;
        }
        tot.x += v.x;
        tot.y += v.y;
        tot.z += v.z;
        tot.w += v.w;
    }
    int total;
    const int run = block_exclusive_scan_1024(tot.x + tot.y + tot.z + tot.w, &total);
    const int s0 = run, s1 = s0 + tot.x, s2 = s1 + tot.y, s3 = s2 + tot.z;
    if (j == 0) {
        int32_t* bs = bin_start + static_cast<size_t>(g) * (kNumBins + 1);
        bs[4 * tid] = s0;
        bs[4 * tid + 1] = s1;
        bs[4 * tid + 2] = s2;
        bs[4 * tid + 3] = s3;
        if (tid == 0) bs[kNumBins] = total;
    }
    cur[4 * tid] = s0 + before.x;
    cur[4 * tid + 1] = s1 + before.y;
    cur[4 * tid + 2] = s2 + before.z;
    cur[4 * tid + 3] = s3 + before.w;
    const BinMap bm = binmap[g];
    __syncthreads();
    const size_t t0 = static_cast<size_t>(g) * Ng;
#pragma unroll
    for (int u = 0; u < kHistPer; ++u) {
        const int t = j * kHistTokens + u * 1024 + tid;
        if (t < Ng) {
            const int pos = atomicAdd(&cur[bm(kv[u])], 1);
            members[t0 + pos] = make_uint2(kv[u], static_cast<uint32_t>(t0 + t));
        }
    }
}

// Block (i, g): bin members [256 i, 256 i + 256) of group g, one per thread.
// A member's rank is its bin's start plus the members of its bin that precede
// it by (key, token). The bins of a block's members span a contiguous range
// of members, staged in LDS (up to kRankStage of them from the span's start);
// a member whose bin reaches past the stage (a bin of thousands) reads the
// rest of its bin from global memory.
constexpr int kRankStage = 4096;

__global__ __launch_bounds__(256) void rank_kernel(
    const BinMap* __restrict__ binmap, const int32_t* __restrict__ bin_start,
    const uint2* __restrict__ members, const int32_t* __restrict__ idx,
    int32_t* __restrict__ order, int32_t* __restrict__ ccount, int Ng, int E, int k, int nch) {
    __shared__ uint2 stage[kRankStage];
    __shared__ int span[2];
    const int g = blockIdx.y, tid = threadIdx.x;
    const int p = blockIdx.x * 256 + tid;
    const int last = min(256, Ng - static_cast<int>(blockIdx.x) * 256) - 1;
    const uint2* mg = members + static_cast<size_t>(g) * Ng;
    const int32_t* bs = bin_start + static_cast<size_t>(g) * (kNumBins + 1);
    const BinMap bm = binmap[g];
    const uint2 m = mg[min(p, Ng - 1)];
    const int b = bm(m.x);
    const int lo = bs[b], hi = bs[b + 1];
    if (tid == 0) span[0] = lo;
    if (tid == last) span[1] = hi;
    __syncthreads();
    const int s0 = span[0], s1 = min(span[1], s0 + kRankStage);
    for (int q = s0 + tid; q < s1; q += 256) stage[q - s0] = mg[q];
    __syncthreads();
    if (tid > last) return;
    const uint32_t key = m.x, t = m.y;
    auto precedes = [&](uint2 o) { return o.x < key || (o.x == key && o.y < t); };
    int before = 0;
    const int hs = max(lo, min(hi, s1));  // [lo, hs) staged, [hs, hi) not
    for (int q = lo; q < hs; q += 4) {
        uint2 o[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) o[u] = stage[min(q + u, hs - 1) - s0];
#pragma unroll
        for (int u = 0; u < 4; ++u) before += (q + u < hs && precedes(o[u])) ? 1 : 0;
    }
    for (int q = hs; q < hi; q += 4) {
        uint2 o[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) o[u] = mg[min(q + u, hi - 1)];
#pragma unroll
        for (int u = 0; u < 4; ++u) before += (q + u < hi && precedes(o[u])) ? 1 : 0;
    }
    const int rank = lo + before;
    order[static_cast<size_t>(g) * Ng + rank] = static_cast<int32_t>(t);
    const int c = rank / kSlotChunk;
    for (int r = 0; r < k; ++r)
        atomicAdd(&ccount[((static_cast<size_t>(g) * nch + c) * k + r) * E +
                          idx[static_cast<size_t>(t) * k + r]],
                  1);
}

// One wave per (group, expert): over the rounds in order, the carry
// min(C, demand of the earlier rounds) and the exclusive scan of the round's
// per-chunk counts (64 chunks per step, four steps' loads together); then
// counts = min(C, total demand) and, for one group, row_base = 0.
__global__ __launch_bounds__(256) void chunk_scan_kernel(
    const int32_t* __restrict__ ccount, int32_t* __restrict__ cbase, int32_t* __restrict__ carry,
    int32_t* __restrict__ counts, int32_t* __restrict__ row_base, int G, int E, int k, int C,
    int nch) {
    const int lane = threadIdx.x & 63;
    const int q = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (q >= G * E) return;
    const int g = q / E, e = q % E;
    int acc = 0;
    for (int r = 0; r < k; ++r) {
        if (lane == 0) carry[(g * k + r) * E + e] = min(C, acc);
        const size_t row = ((static_cast<size_t>(g) * k + r) * E + e) * nch;
        const int32_t* cc = ccount + static_cast<size_t>(g) * nch * k * E + r * E + e;
        int run = 0;
        for (int c0 = 0; c0 < nch; c0 += 4 * 64) {
            int v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int c = c0 + u * 64 + lane;
                v[u] = c < nch ? cc[static_cast<size_t>(c) * k * E] : 0;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int c = c0 + u * 64 + lane;
                int inc = v[u];
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    const int w = __shfl_up(inc, o, 64);
                    if (lane >= o) inc += w;
                }
                if (c < nch) cbase[row + c] = run + inc - v[u];
                run += __shfl(inc, 63, 64);
            }
        }
        acc += run;
    }
    if (lane == 0) {
        counts[g * E + e] = min(C, acc);
        if (G == 1) row_base[e] = 0;
    }
}

__global__ __launch_bounds__(kSlotChunk) void slots_kernel(
    const int32_t* __restrict__ order, const int32_t* __restrict__ idx,
    const float* __restrict__ probs, const int32_t* __restrict__ cbase,
    const int32_t* __restrict__ carry, int32_t* __restrict__ slot, float* __restrict__ gate,
    int Ng, int E, int k, int C, int nch) {
    __shared__ int wcnt[kSlotChunk / 64][kMaxExperts + 1];
    const int g = blockIdx.y, c = blockIdx.x;
    const int p = c * kSlotChunk + threadIdx.x;
    const bool active = p < Ng;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int t = active ? order[static_cast<size_t>(g) * Ng + p] : 0;
    const uint64_t lt_mask = (1ull << lane) - 1ull;
    for (int r = 0; r < k; ++r) {
        for (int q = threadIdx.x; q < (kSlotChunk / 64) * (kMaxExperts + 1); q += kSlotChunk)
            wcnt[q / (kMaxExperts + 1)][q % (kMaxExperts + 1)] = 0;
        __syncthreads();
        const int e = active ? idx[static_cast<size_t>(t) * k + r] : kMaxExperts;
        uint64_t same = __ballot(1);
#pragma unroll
        for (int bit = 0; bit < 7; ++bit) {
            const uint64_t bal = __ballot((e >> bit) & 1);
            same &= ((e >> bit) & 1) ? bal : ~bal;
        }
        const int rank_w = __popcll(same & lt_mask);
        if (rank_w == 0) wcnt[w][e] = __popcll(same);
        __syncthreads();
        if (active) {
            int rank = cbase[((static_cast<size_t>(g) * k + r) * E + e) * nch + c] + rank_w;
            for (int w2 = 0; w2 < w; ++w2) rank += wcnt[w2][e];
            const int s = carry[(g * k + r) * E + e] + rank;
            const bool kept = s < C;
            slot[static_cast<size_t>(t) * k + r] = kept ? s : -1;
            gate[static_cast<size_t>(t) * k + r] = kept ? probs[static_cast<size_t>(t) * E + e] : 0.0f;
        }
        __syncthreads();
    }
}

// ------------------------------------------ small groups: one block each
//
// A group of at most kLocalTokens tokens and kLocalAssign assignments runs
// steps 2-6 in one 1024-thread block, all in LDS: the same bin map and exact
// (key, token) rank give the order (a bin member carries the key bits below
// the bin with its token, so one LDS word decides each comparison), then the
// slots are assigned round by round over the order in tiles of 1024
// positions with the ballot ranks of slots_kernel; a round's running
// per-expert totals are its demand, which gives the next round's carry.
// Phases meet at LDS-only barriers, so the order and slot stores drain in
// the background, and the gate probabilities are fetched at the start.
constexpr int kLocalTokens = 8192;
constexpr int kLocalAssign = 16384;
constexpr int kTokBits = 13;  // token index inside a group < 2^13
static_assert(kLocalTokens <= (1 << kTokBits), "token index field");
static_assert(kKeyBits - kBinBits + kTokBits <= 32, "bin member = low key bits + token");

// NW > 0 (E <= 2 NW <= 16): slots from a block scan of per-thread expert
// counts packed two 16-bit fields to a word; NW == 0: ballot tiles.
template <int NW>
__global__ __launch_bounds__(1024) void local_route_kernel(
    const uint32_t* __restrict__ keys, const int32_t* __restrict__ idx,
    const float* __restrict__ probs, int32_t* __restrict__ order, int32_t* __restrict__ slot,
    float* __restrict__ gate, int32_t* __restrict__ counts, int32_t* __restrict__ row_base,
    int G, int Ng, int E, int k, int C) {
    constexpr int KT = kLocalTokens / 1024, KA = kLocalAssign / 1024;  // per thread
    __shared__ uint32_t key_l[kLocalTokens];
    __shared__ uint32_t memb[kLocalTokens];          // bin members: low key bits << 13 | token
    __shared__ uint16_t ord_l[kLocalTokens];         // tokens by order position
    __shared__ uint8_t idx_l[kLocalAssign];          // [Ng][k] choices
    __shared__ uint32_t kept_l[kLocalAssign / 32];   // bit t*k + r: assignment kept
    __shared__ int start[kNumBins + 1];
    __shared__ int cursor[kNumBins];                 // histogram, then fill cursors
    __shared__ int wcnt[2][16][kMaxExperts + 1];     // per-wave expert counts, two tiles
    __shared__ int running[kMaxExperts + 1];         // this round's earlier tiles
    __shared__ int carry[kMaxExperts];               // min(C, earlier rounds' demand)
    __shared__ uint32_t wtot[16][NW > 0 ? NW : 1];   // packed scan: wave totals,
    __shared__ uint32_t wpre[16][NW > 0 ? NW : 1];   // their prefixes over waves,
    __shared__ uint32_t btot[NW > 0 ? NW : 1];       // the block total,
    __shared__ uint32_t wmin[16], wmax[16];
    __shared__ BinMap map;
    const int g = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const size_t t0 = static_cast<size_t>(g) * Ng;
    const int nk = Ng * k;

    // all global loads of the group first, in flight together
    uint32_t kv[KT];
    int32_t iv[KA];
#pragma unroll
    for (int u = 0; u < KT; ++u) kv[u] = keys[t0 + min(u * 1024 + tid, Ng - 1)];
#pragma unroll
    for (int u = 0; u < KA; ++u) iv[u] = idx[t0 * k + min(u * 1024 + tid, nk - 1)];
    for (int b = tid; b < kNumBins; b += 1024) cursor[b] = 0;
    for (int q = tid; q < kLocalAssign / 32; q += 1024) kept_l[q] = 0u;
    for (int q = tid; q < 2 * 16 * (kMaxExperts + 1); q += 1024) (&wcnt[0][0][0])[q] = 0;
    if (tid <= kMaxExperts) running[tid] = 0;
    if (tid < kMaxExperts) carry[tid] = 0;
    uint32_t lo = 0xFFFFFFFFu, hi = 0u;
#pragma unroll
    for (int u = 0; u < KT; ++u) {
        const int t = u * 1024 + tid;
        if (t < Ng) {
            key_l[t] = kv[u];
            lo = min(lo, kv[u]);
            hi = max(hi, kv[u]);
        }
    }
#pragma unroll
    for (int u = 0; u < KA; ++u) {
        const int q = u * 1024 + tid;
        if (q < nk) idx_l[q] = static_cast<uint8_t>(iv[u]);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        lo = min(lo, static_cast<uint32_t>(__shfl_xor(static_cast<int>(lo), o, 64)));
        hi = max(hi, static_cast<uint32_t>(__shfl_xor(static_cast<int>(hi), o, 64)));
    }
    if (lane == 0) {
        wmin[w] = lo;
        wmax[w] = hi;
    }
    lds_barrier();
    if (tid == 0) {
        uint32_t a = wmin[0], z = wmax[0];
        for (int q = 1; q < 16; ++q) {
            a = min(a, wmin[q]);
            z = max(z, wmax[q]);
        }
        int sh = 0;
        while (((z - a) >> sh) >= static_cast<uint32_t>(kNumBins)) ++sh;
        map = BinMap{a, sh};
    }
    lds_barrier();
    const BinMap bm = map;
    const uint32_t low_mask = (1u << bm.shift) - 1u;
    for (int t = tid; t < Ng; t += 1024) atomicAdd(&cursor[bm(key_l[t])], 1);
    lds_barrier();
    {
        constexpr int per = kNumBins / 1024;
        int local[per];
        int sum = 0;
#pragma unroll
        for (int q = 0; q < per; ++q) {
            local[q] = cursor[tid * per + q];
            sum += local[q];
        }
        int total;
        int run = block_exclusive_scan_1024(sum, &total);
#pragma unroll
        for (int q = 0; q < per; ++q) {
            start[tid * per + q] = run;
            cursor[tid * per + q] = run;
            run += local[q];
        }
        if (tid == 0) start[kNumBins] = total;
    }
    lds_barrier();
    for (int t = tid; t < Ng; t += 1024) {
        const uint32_t key = key_l[t];
        const int pos = atomicAdd(&cursor[bm(key)], 1);
        memb[pos] = (((key - bm.kmin) & low_mask) << kTokBits) | static_cast<uint32_t>(t);
    }
    lds_barrier();
    {
        // this thread's tokens tid + 1024 u: keys, then bin bounds, read together
        uint32_t mine[KT];
        int lo_b[KT], hi_b[KT];
#pragma unroll
        for (int u = 0; u < KT; ++u) mine[u] = key_l[min(u * 1024 + tid, Ng - 1)];
#pragma unroll
        for (int u = 0; u < KT; ++u) {
            const int b = bm(mine[u]);
            lo_b[u] = start[b];
            hi_b[u] = start[b + 1];
            mine[u] = (((mine[u] - bm.kmin) & low_mask) << kTokBits) |
                      static_cast<uint32_t>(u * 1024 + tid);
        }
#pragma unroll
        for (int u = 0; u < KT; ++u) {
            const int t = u * 1024 + tid;
            if (t < Ng) {
                // members before this token: smaller (low key bits, token); four reads at a time
                const int pe = hi_b[u];
                int rank = lo_b[u];
                int before = 0;
                for (int p = rank; p < pe; p += 4) {
                    uint32_t m[4];
#pragma unroll
                    for (int v = 0; v < 4; ++v) m[v] = memb[min(p + v, pe - 1)];
#pragma unroll
                    for (int v = 0; v < 4; ++v) before += (p + v < pe && m[v] < mine[u]) ? 1 : 0;
                }
                rank += before;
                ord_l[rank] = static_cast<uint16_t>(t);
                order[t0 + rank] = static_cast<int32_t>(t0 + t);
            }
        }
    }
    lds_barrier();
    // the probabilities of the gates, needed at the very end (their latency
    // hides behind the slots); q / k as a multiply-high by ceil(2^32 / k),
    // exact for q k < 2^32
    const uint32_t kinv = k > 1 ? 0xFFFFFFFFu / static_cast<uint32_t>(k) + 1u : 0u;
    float pv[KA];
#pragma unroll
    for (int u = 0; u < KA; ++u) {
        const int q = min(u * 1024 + tid, nk - 1);
        const int t = k > 1 ? static_cast<int>(__umulhi(static_cast<uint32_t>(q), kinv)) : q;
        pv[u] = probs[(t0 + t) * E + idx_l[q]];
    }
    int total = 0;  // thread e < E: demand of the rounds so far
    if constexpr (NW > 0) {
        // thread tid owns order positions [tid P, tid P + P), P <= 8: its
        // per-expert counts (4-bit fields of one word) give the ranks among
        // its own positions, and an exclusive block scan of the counts
        // (16-bit fields, two experts per word) the ranks before them
        // Carries and demands never exceed N_g k <= kLocalAssign < 2^16, so
        // every thread keeps the per-expert demand of the finished rounds
        // packed like the scan, and derives the carries itself
        static_assert(kLocalAssign < (1 << 16), "16-bit demand fields");
        const int P = (Ng + 1023) / 1024;
        uint32_t done[NW];
#pragma unroll
        for (int q = 0; q < NW; ++q) done[q] = 0u;
        const uint32_t cap = static_cast<uint32_t>(min(C, 0xFFFF));
        for (int r = 0; r < k; ++r) {
            // position j's expert and its rank among this thread's earlier
            // positions, 4-bit fields of ep and rp (E <= 16, rank < 8)
            uint64_t lc = 0;
            uint32_t ep = 0u, rp = 0u;
            {
                int tt[KT];
#pragma unroll
                for (int j = 0; j < KT; ++j) tt[j] = ord_l[min(tid * P + j, Ng - 1)];
#pragma unroll
                for (int j = 0; j < KT; ++j) {
                    const int e = idx_l[tt[j] * k + r];
                    const bool act = j < P && tid * P + j < Ng;
                    rp |= static_cast<uint32_t>((lc >> (4 * e)) & 15u) << (4 * j);
                    ep |= static_cast<uint32_t>(e) << (4 * j);
                    lc += act ? (1ull << (4 * e)) : 0ull;
                }
            }
            // word q of this thread's counts: experts 2q, 2q + 1 in 16-bit fields
            auto own = [&](int q) {
                return static_cast<uint32_t>((lc >> (8 * q)) & 15u) |
                       (static_cast<uint32_t>((lc >> (8 * q + 4)) & 15u) << 16);
            };
            uint32_t inc[NW];
#pragma unroll
            for (int q = 0; q < NW; ++q) inc[q] = own(q);
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
#pragma unroll
                for (int q = 0; q < NW; ++q) {
                    const uint32_t u = static_cast<uint32_t>(__shfl_up(static_cast<int>(inc[q]), o, 64));
                    if (lane >= o) inc[q] += u;
                }
            }
            if (lane == 63) {
#pragma unroll
                for (int q = 0; q < NW; ++q) wtot[w][q] = inc[q];
            }
#pragma unroll
            for (int q = 0; q < NW; ++q) inc[q] -= own(q);  // exclusive inside the wave
            lds_barrier();
            if (tid < 16 * NW) {  // (wave, word): prefix over earlier waves
                const int w2 = tid / NW, q = tid % NW;
                uint32_t pre = 0u;
#pragma unroll
                for (int w3 = 0; w3 < 15; ++w3) pre += w3 < w2 ? wtot[w3][q] : 0u;
                wpre[w2][q] = pre;
                if (w2 == 15) btot[q] = pre + wtot[15][q];
            }
            lds_barrier();
#pragma unroll
            for (int q = 0; q < NW; ++q) inc[q] += wpre[w][q];  // exclusive over the block
#pragma unroll
            for (int j = 0; j < KT; ++j) {
                const int p = tid * P + j;
                if (j < P && p < Ng) {
                    const int e = static_cast<int>((ep >> (4 * j)) & 15u);
                    uint32_t word = inc[0], dw = done[0];
#pragma unroll
                    for (int q = 1; q < NW; ++q) {
                        word = (e >> 1) == q ? inc[q] : word;
                        dw = (e >> 1) == q ? done[q] : dw;
                    }
                    const int sh = 16 * (e & 1);
                    const int rank = static_cast<int>((word >> sh) & 0xFFFFu) +
                                     static_cast<int>((rp >> (4 * j)) & 15u);
                    const int sl = static_cast<int>(min((dw >> sh) & 0xFFFFu, cap)) + rank;
                    const int t = ord_l[p];
                    const bool kept = sl < C;
                    slot[(t0 + t) * k + r] = kept ? sl : -1;
                    if (kept) atomicOr(&kept_l[(t * k + r) >> 5], 1u << ((t * k + r) & 31));
                }
            }
#pragma unroll
            for (int q = 0; q < NW; ++q) done[q] += btot[q];
        }
        if (tid < E) {
            uint32_t word = done[0];
#pragma unroll
            for (int q = 1; q < NW; ++q) word = (tid >> 1) == q ? done[q] : word;
            total = static_cast<int>((word >> (16 * (tid & 1))) & 0xFFFFu);
        }
    } else {
    // slots: tile i counts its waves' experts into wcnt[i & 1] (cleared while
    // tile i - 1 was read), so a tile takes two barriers
    const uint64_t lt_mask = (1ull << lane) - 1ull;
    const int ntile = (Ng + 1023) / 1024;
    int it = 0;
    for (int r = 0; r < k; ++r) {
        for (int i = 0; i < ntile; ++i, ++it) {
            const int buf = it & 1;
            const int p = i * 1024 + tid;
            const bool active = p < Ng;
            const int t = active ? ord_l[p] : 0;
            const int e = active ? idx_l[t * k + r] : kMaxExperts;
            uint64_t same = __ballot(1);
#pragma unroll
            for (int bit = 0; bit < 7; ++bit) {
                const uint64_t bal = __ballot((e >> bit) & 1);
                same &= ((e >> bit) & 1) ? bal : ~bal;
            }
            const int rank_w = __popcll(same & lt_mask);
            if (rank_w == 0) wcnt[buf][w][e] = __popcll(same);
            lds_barrier();
            if (active) {
                int rank = running[e] + rank_w;
#pragma unroll
                for (int w2 = 0; w2 < 16; ++w2) rank += w2 < w ? wcnt[buf][w2][e] : 0;
                const int sl = carry[e] + rank;
                const bool kept = sl < C;
                slot[(t0 + t) * k + r] = kept ? sl : -1;
                if (kept) atomicOr(&kept_l[(t * k + r) >> 5], 1u << ((t * k + r) & 31));
            }
            for (int q = tid; q < 16 * (kMaxExperts + 1); q += 1024) (&wcnt[buf ^ 1][0][0])[q] = 0;
            lds_barrier();
            if (tid < E) {
                int sum = running[tid];
#pragma unroll
                for (int w2 = 0; w2 < 16; ++w2) sum += wcnt[buf][w2][tid];
                if (i + 1 < ntile) {
                    running[tid] = sum;
                } else {  // round done: its demand moves into the carry
                    running[tid] = 0;
                    total += sum;
                    carry[tid] = min(C, total);
                }
            }
        }
    }
    }
    if (tid < E) {
        counts[g * E + tid] = min(C, total);
        if (G == 1) row_base[tid] = 0;
    }
    lds_barrier();
#pragma unroll
    for (int u = 0; u < KA; ++u) {
        const int q = u * 1024 + tid;
        if (q < nk) gate[t0 * k + q] = ((kept_l[q >> 5] >> (q & 31)) & 1u) ? pv[u] : 0.0f;
    }
}

// row_base[g, e] = sum of counts[g', e] over g' < g: the counts of a chunk of
// groups are staged in LDS first (one load latency per chunk, not per group).
__global__ __launch_bounds__(1024) void row_base_kernel(const int32_t* __restrict__ counts,
                                                        int32_t* __restrict__ row_base, int G,
                                                        int E) {
    constexpr int kStage = 8192;
    __shared__ int cnt_l[kStage];
    const int per = kStage / E;  // groups per chunk (E <= 64)
    int base = 0;                // thread e < E
    for (int g0 = 0; g0 < G; g0 += per) {
        const int ng = min(per, G - g0);
        __syncthreads();
        for (int q = threadIdx.x; q < ng * E; q += 1024) cnt_l[q] = counts[g0 * E + q];
        __syncthreads();
        if (static_cast<int>(threadIdx.x) < E) {
            for (int g = 0; g < ng; ++g) {
                row_base[(g0 + g) * E + threadIdx.x] = base;
                base += cnt_l[g * E + threadIdx.x];
            }
        }
    }
}

}  // namespace

size_t route_workspace_bytes(const Dims& D) { return route_ws_layout(D, nullptr).bytes; }

// Steps 2-7 in one block per group (local_route) for groups that fit its LDS.
bool local_route_fits(const Dims& D) {
    return D.Ng <= kLocalTokens && static_cast<long long>(D.Ng) * D.k <= kLocalAssign;
}

vmoe_status route_launch(const Dims& D, const void* x, const void* wr, const float* bias,
                         const float* noise, int flags, float* logits, float* probs,
                         int32_t* idx, int32_t* slot, float* gate, int32_t* order, int32_t* counts,
                         int32_t* row_base, void* ws_base, hipStream_t st) {
    RouteWs ws = route_ws_layout(D, ws_base);
    const int nch = static_cast<int>(cdiv(D.Ng, kSlotChunk));
    const int nkp = router_blocks(D);
    const int logits_in = (flags & VMOE_ROUTE_LOGITS_IN) ? 1 : 0;
    if (D.N > 0) {
        if (D.dtype == VMOE_BF16) {
            dim3 grid(nkp, D.G);
            auto kern = D.E > 32 ? router_mfma_kernel<true> : router_mfma_kernel<false>;
            kern<<<grid, 256, 0, st>>>(static_cast<const uint16_t*>(x),
                                       static_cast<const uint16_t*>(wr), bias, noise, logits,
                                       probs, idx, ws.keys, ws.kpart, D.Ng, D.d, D.E, D.k,
                                       logits_in);
        } else {
            dim3 grid(nkp, D.G);
            router_f64_kernel<<<grid, 256, 0, st>>>(
                static_cast<const float*>(x), static_cast<const float*>(wr), bias, noise, logits,
                probs, idx, ws.keys, ws.kpart, D.Ng, D.d, D.E, D.k, logits_in,
                f64_router_tokens(D.E));
        }
        if (local_route_fits(D)) {
            auto kern = D.E <= 8 ? local_route_kernel<4>
                      : D.E <= 16 ? local_route_kernel<8> : local_route_kernel<0>;
            kern<<<D.G, 1024, 0, st>>>(ws.keys, idx, probs, order, slot, gate, counts, row_base,
                                       D.G, D.Ng, D.E, D.k, D.C);
            if (D.G > 1) row_base_kernel<<<1, 1024, 0, st>>>(counts, row_base, D.G, D.E);
            return launch_status();
        }
        const int nhb = static_cast<int>(cdiv(D.Ng, kHistTokens));
        bin_hist_kernel<<<dim3(nhb, D.G), 1024, 0, st>>>(ws.keys, ws.kpart, nkp, ws.binmap,
                                                          ws.bhist, ws.ccount, nch * D.k * D.E,
                                                          D.Ng);
        bin_scatter_kernel<<<dim3(nhb, D.G), 1024, 0, st>>>(ws.keys, ws.binmap, ws.bhist,
                                                             ws.bin_start, ws.members, D.Ng);
        rank_kernel<<<dim3(cdiv(D.Ng, 256), D.G), 256, 0, st>>>(
            ws.binmap, ws.bin_start, ws.members, idx, order, ws.ccount, D.Ng, D.E, D.k, nch);
    }
    chunk_scan_kernel<<<cdiv(D.G * D.E, 4), 256, 0, st>>>(ws.ccount, ws.cbase, ws.carry, counts,
                                                         row_base, D.G, D.E, D.k, D.C, nch);
    if (D.G > 1) row_base_kernel<<<1, 1024, 0, st>>>(counts, row_base, D.G, D.E);
    if (D.N > 0)
        slots_kernel<<<dim3(nch, D.G), kSlotChunk, 0, st>>>(order, idx, probs, ws.cbase, ws.carry,
                                                            slot, gate, D.Ng, D.E, D.k, D.C, nch);
    return launch_status();
}

}  // namespace vmoe
