// Noisy top-k gating with capacity and batch-prioritized routing on gfx950.
//
// Pipeline (all on the caller's stream, no host synchronisation):
//   1. router_gate   logits (double-accumulated, increasing-i order, rounded
//                    once to f32), noisy softmax, top-k, 26-bit priority key
//   2. bin_scan      per group: key range -> 4096 bins spanning it, histogram
//                    in LDS, exclusive scan -> bin starts; clears the counters
//   3. bin_scatter   tokens into their bins (atomic fill; order inside a bin
//                    is irrelevant, ranks are computed exactly next)
//   4. rank          rank of each token = tokens in lower bins + tokens of its
//                    own bin that precede it by (key, index): a stable
//                    priority sort without passes; also counts, per chunk of
//                    256 order positions, the assignments to each expert
//   5. chunk_scan    per (group, round, expert) exclusive scan over chunks;
//                    round carries min(C, earlier demand); counts; row_base
//   6. slots         per chunk: rank of each assignment among same-expert
//                    assignments (wave ballots + cross-wave prefix), slot =
//                    carry + rank, kept while slot < C
// This file must be compiled with -ffp-contract=off: the gate's float
// arithmetic is specified operation by operation.
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
constexpr int kGateTokens = 32;              // most tokens per router_gate block

struct RouteWs {
    uint32_t* keys;     // [N]
    BinMap* binmap;     // [G]
    int32_t* bin_start; // [G][kNumBins + 1]
    int32_t* fill;      // [G][kNumBins]
    int32_t* members;   // [N]
    int32_t* ccount;    // [G][nch][k][E]
    int32_t* cbase;     // [G][nch][k][E]
    int32_t* demand;    // [G][k][E]
    int32_t* carry;     // [G][k][E]
    size_t bytes;
};

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

RouteWs route_ws_layout(const Dims& D, void* base) {
    char* p = static_cast<char*>(base);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char* q = p ? p + off : nullptr;
        off += align256(bytes);
        return q;
    };
    const size_t nch = cdiv(D.Ng, kSlotChunk);
    RouteWs w;
    w.keys = reinterpret_cast<uint32_t*>(take(sizeof(uint32_t) * D.N));
    w.binmap = reinterpret_cast<BinMap*>(take(sizeof(BinMap) * D.G));
    w.bin_start = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * D.G * (kNumBins + 1)));
    w.fill = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * D.G * kNumBins));
    w.members = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * D.N));
    w.ccount = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * D.G * nch * D.k * D.E));
    w.cbase = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * D.G * nch * D.k * D.E));
    w.demand = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * D.G * D.k * D.E));
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

// Eight consecutive activations as f32 (16-byte aligned).
__device__ __forceinline__ void load8(const uint16_t* p, float* v) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        v[2 * q] = __uint_as_float(w[q] << 16);
        v[2 * q + 1] = __uint_as_float(w[q] & 0xFFFF0000u);
    }
}
__device__ __forceinline__ void load8(const float* p, float* v) {
    const float4 a = reinterpret_cast<const float4*>(p)[0];
    const float4 b = reinterpret_cast<const float4*>(p)[1];
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

// x and W_r are staged in LDS 32 vectors of 16 bytes (256 bf16 / 128 f32
// columns) per row at a time; rows are padded by one vector so the 16-byte
// reads of different rows fall in different banks.
constexpr int kGateVecs = 32;

// One block = tpb = min(32, floor(256 / E)) tokens of one group. Thread tid < tpb*E
// computes logit (token tid / E, expert tid % E) as a sequential dot product
// in double over increasing i; the block's x rows and the group's router rows
// are staged through LDS a slice of columns at a time (coalesced 16-byte loads,
// next round prefetched in registers), so the dependency chains only wait on
// LDS. The gate of each token then runs on one thread from LDS.
template <typename T>
__global__ __launch_bounds__(256) void router_gate_kernel(
    const T* __restrict__ x, const T* __restrict__ wr, const float* __restrict__ bias,
    const float* __restrict__ noise, float* __restrict__ logits, float* __restrict__ probs,
    int32_t* __restrict__ idx, uint32_t* __restrict__ keys, int Ng, int d, int E, int k,
    int logits_in, int tpb) {
    constexpr int VE = 16 / sizeof(T);             // elements per 16-byte vector
    constexpr int VPR = kGateVecs;                 // vectors per staged row
    constexpr int GC = VPR * VE;                   // columns per round
    constexpr int LDR = GC + VE;                   // LDS row length (elements)
    constexpr int MAXROWS = kGateTokens + kMaxExperts;
    __shared__ __attribute__((aligned(16))) T stage[MAXROWS * LDR];
    __shared__ float lg_store[kGateTokens * (kMaxExperts + 1)];
    __shared__ int row_bad[2][MAXROWS];
    const int g = blockIdx.y;
    const int t0 = blockIdx.x * tpb;                  // within group
    const int ntok = min(tpb, Ng - t0);
    const size_t tok0 = static_cast<size_t>(g) * Ng + t0;  // global index
    const int tid = threadIdx.x;
    const int ld = E + 1;                             // LDS row of one token's logits
    if (!logits_in) {
        // staged rows: ntok token rows, then E router rows
        const int rows = ntok + E;
        const T* wg = wr + static_cast<size_t>(g) * E * d;
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
                    const T* src = r < ntok ? x + (tok0 + r) * d + col
                                            : wg + static_cast<size_t>(r - ntok) * d + col;
                    pre[q] = *reinterpret_cast<const uint4*>(src);
                }
            }
        };
        // bf16 rows whose staged values are all zero or of magnitude in
        // [2^-63, 2^63) give products that are exact normal f32 numbers; a row
        // with any other value (subnormal, huge, inf, nan) is marked in
        // row_bad[round parity] and its dot products take the f64 path
        auto park = [&](int par) {
#pragma unroll
            for (int q = 0; q < MAXV; ++q) {
                const int v = tid + 256 * q;
                if (v < nvec) {
                    *reinterpret_cast<uint4*>(stage + (v / VPR) * LDR + (v % VPR) * VE) = pre[q];
                    if constexpr (sizeof(T) == 2) {
                        const uint32_t w4[4] = {pre[q].x, pre[q].y, pre[q].z, pre[q].w};
                        bool bad = false;
#pragma unroll
                        for (int h = 0; h < 8; ++h) {
                            const uint32_t b = (w4[h >> 1] >> (16 * (h & 1))) & 0x7FFFu;
                            const uint32_t ex = b >> 7;
                            bad |= b != 0 && (ex < 64 || ex > 189);
                        }
                        if (bad) atomicOr(&row_bad[par][v / VPR], 1);
                    }
                }
            }
        };
        const bool mine = tid < ntok * E;
        const int tt = tid / E, e = tid % E;
        const T* xs = stage + tt * LDR;
        const T* wsr = stage + (ntok + e) * LDR;
        double acc = 0.0;
        for (int r = tid; r < 2 * MAXROWS; r += 256) row_bad[r / MAXROWS][r % MAXROWS] = 0;
        __syncthreads();
        fetch(0);
        for (int c0 = 0, par = 0; c0 < d; c0 += GC, par ^= 1) {
            park(par);
            __syncthreads();
            if (c0 + GC < d) fetch(c0 + GC);
            // the other parity's flags were last read in the previous round
            for (int r = tid; r < MAXROWS; r += 256) row_bad[par ^ 1][r] = 0;
            const bool exact_f32 = mine && row_bad[par][tt] == 0 && row_bad[par][ntok + e] == 0;
            if (mine) {
                const int n = min(GC, d - c0);
                // Each product of two bf16 / f32 values is exact in double, so
                // the fused multiply-add equals add-after-multiply, in increasing i.
                // 32 columns per step; the next step's LDS reads are issued
                // before this step's multiply-add chain. Staged columns past d
                // are zeros: their products add +0 to a sum that starts at +0
                // and so can never be -0, which leaves it unchanged.
                const int nn = (n + 31) & ~31;
                float xv[2][32], wv[2][32];
                auto read32 = [&](int i, float (&xa)[32], float (&wa)[32]) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        load8(xs + i + 8 * q, xa + 8 * q);
                        load8(wsr + i + 8 * q, wa + 8 * q);
                    }
                };
                auto chain32 = [&](const float (&xa)[32], const float (&wa)[32]) {
                    if (sizeof(T) == 2 && exact_f32) {
                        // bf16 x bf16 is exact in f32 (8-bit significands), so
                        // acc + double(x * w) rounds exactly like the fused
                        // multiply-add in double; the products and widenings
                        // are off the dependency chain, which is the adds
                        double pd[32];
#pragma unroll
                        for (int q = 0; q < 32; ++q) pd[q] = static_cast<double>(xa[q] * wa[q]);
#pragma unroll
                        for (int q = 0; q < 32; ++q) acc = acc + pd[q];
                    } else {
#pragma unroll
                        for (int q = 0; q < 32; ++q)
                            acc = __builtin_fma(static_cast<double>(xa[q]),
                                                static_cast<double>(wa[q]), acc);
                    }
                };
                read32(0, xv[0], wv[0]);
                for (int i = 0; i < nn; i += 64) {
                    const bool two = i + 32 < nn;  // uniform
                    if (two) read32(i + 32, xv[1], wv[1]);
                    chain32(xv[0], wv[0]);
                    if (i + 64 < nn) read32(i + 64, xv[0], wv[0]);
                    if (two) chain32(xv[1], wv[1]);
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

    if (tid >= ntok) return;
    // Gate of token tid; its noisy logits z overwrite its row of lg_store.
    const size_t t = tok0 + tid;
    float* z = lg_store + tid * ld;
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
    keys[t] = priority_key(__fdiv_rn(exp_spec(z[first] - m), s));
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

// One block per group: key range -> bin map, bin histogram + scan; clears
// fill and chunk counters.
__global__ __launch_bounds__(1024) void bin_scan_kernel(const uint32_t* __restrict__ keys,
                                                        BinMap* __restrict__ binmap,
                                                        int32_t* __restrict__ bin_start,
                                                        int32_t* __restrict__ fill,
                                                        int32_t* __restrict__ ccount, int Ng,
                                                        int cc_per_group) {
    __shared__ int hist[kNumBins];
    __shared__ uint32_t wmin[16], wmax[16];
    __shared__ BinMap map;
    const int g = blockIdx.x;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    for (int b = threadIdx.x; b < kNumBins; b += 1024) hist[b] = 0;
    const uint32_t* kg = keys + static_cast<size_t>(g) * Ng;
    uint32_t lo = 0xFFFFFFFFu, hi = 0u;
    for (int t = threadIdx.x; t < Ng; t += 1024) {
        const uint32_t key = kg[t];
        lo = min(lo, key);
        hi = max(hi, key);
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
        for (int q = 1; q < 16; ++q) {
            a = min(a, wmin[q]);
            z = max(z, wmax[q]);
        }
        if (Ng == 0) a = z = 0u;
        int sh = 0;
        while (((z - a) >> sh) >= static_cast<uint32_t>(kNumBins)) ++sh;
        map = BinMap{a, sh};
        binmap[g] = map;
    }
    __syncthreads();
    const BinMap bm = map;
    for (int t = threadIdx.x; t < Ng; t += 1024) atomicAdd(&hist[bm(kg[t])], 1);
    __syncthreads();
    constexpr int per = kNumBins / 1024;
    int local[per];
    int sum = 0;
#pragma unroll
    for (int q = 0; q < per; ++q) {
        local[q] = hist[threadIdx.x * per + q];
        sum += local[q];
    }
    int total;
    int run = block_exclusive_scan_1024(sum, &total);
    int32_t* bs = bin_start + static_cast<size_t>(g) * (kNumBins + 1);
#pragma unroll
    for (int q = 0; q < per; ++q) {
        bs[threadIdx.x * per + q] = run;
        run += local[q];
    }
    if (threadIdx.x == 0) bs[kNumBins] = total;
    int32_t* fg = fill + static_cast<size_t>(g) * kNumBins;
    for (int b = threadIdx.x; b < kNumBins; b += 1024) fg[b] = 0;
    int32_t* cg = ccount + static_cast<size_t>(g) * cc_per_group;
    for (int q = threadIdx.x; q < cc_per_group; q += 1024) cg[q] = 0;
}

__global__ __launch_bounds__(256) void bin_scatter_kernel(const uint32_t* __restrict__ keys,
                                                          const BinMap* __restrict__ binmap,
                                                          const int32_t* __restrict__ bin_start,
                                                          int32_t* __restrict__ fill,
                                                          int32_t* __restrict__ members, int N,
                                                          int Ng) {
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= N) return;
    const int g = t / Ng;
    const int b = binmap[g](keys[t]);
    const int pos = bin_start[static_cast<size_t>(g) * (kNumBins + 1) + b] +
                    atomicAdd(&fill[static_cast<size_t>(g) * kNumBins + b], 1);
    members[static_cast<size_t>(g) * Ng + pos] = t;
}

__global__ __launch_bounds__(256) void rank_kernel(
    const uint32_t* __restrict__ keys, const BinMap* __restrict__ binmap,
    const int32_t* __restrict__ bin_start,
    const int32_t* __restrict__ members, const int32_t* __restrict__ idx,
    int32_t* __restrict__ order, int32_t* __restrict__ ccount, int N, int Ng, int E, int k,
    int nch) {
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= N) return;
    const int g = t / Ng;
    const uint32_t key = keys[t];
    const int32_t* bs = bin_start + static_cast<size_t>(g) * (kNumBins + 1);
    const int b = binmap[g](key);
    const int lo = bs[b], hi = bs[b + 1];
    const int32_t* mg = members + static_cast<size_t>(g) * Ng;
    int rank = lo;
    for (int p = lo; p < hi; ++p) {
        const int t2 = mg[p];
        const uint32_t k2 = keys[t2];
        rank += (k2 < key || (k2 == key && t2 < t)) ? 1 : 0;
    }
    order[static_cast<size_t>(g) * Ng + rank] = t;
    const int c = rank / kSlotChunk;
    int32_t* cc = ccount + (static_cast<size_t>(g) * nch + c) * k * E;
    for (int r = 0; r < k; ++r) atomicAdd(&cc[r * E + idx[static_cast<size_t>(t) * k + r]], 1);
}

// Single block: chunk offsets, round carries, counts and row bases.
__global__ __launch_bounds__(1024) void chunk_scan_kernel(
    const int32_t* __restrict__ ccount, int32_t* __restrict__ cbase, int32_t* __restrict__ demand,
    int32_t* __restrict__ carry, int32_t* __restrict__ counts, int32_t* __restrict__ row_base,
    int G, int E, int k, int C, int nch) {
    const int kE = k * E;
    const int lane = threadIdx.x & 63;
    // one wave per (group, round, expert): exclusive scan over the chunks, 64 at a time
    for (int q = threadIdx.x >> 6; q < G * kE; q += 16) {
        const int g = q / kE, re = q % kE;
        int run = 0;
        for (int c0 = 0; c0 < nch; c0 += 64) {
            const int c = c0 + lane;
            const size_t at = (static_cast<size_t>(g) * nch + c) * kE + re;
            const int v = c < nch ? ccount[at] : 0;
            int inc = v;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const int u = __shfl_up(inc, o, 64);
                if (lane >= o) inc += u;
            }
            if (c < nch) cbase[at] = run + inc - v;
            run += __shfl(inc, 63, 64);
        }
        if (lane == 0) demand[q] = run;
    }
    __syncthreads();
    for (int q = threadIdx.x; q < G * E; q += 1024) {
        const int g = q / E, e = q % E;
        int acc = 0;
        for (int r = 0; r < k; ++r) {
            carry[(g * k + r) * E + e] = min(C, acc);
            acc += demand[(g * k + r) * E + e];
        }
        counts[q] = min(C, acc);
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += 1024) {
        int base = 0;
        for (int g = 0; g < G; ++g) {
            row_base[g * E + e] = base;
            base += counts[g * E + e];
        }
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
            int rank = cbase[(static_cast<size_t>(g) * nch + c) * k * E + r * E + e] + rank_w;
            for (int w2 = 0; w2 < w; ++w2) rank += wcnt[w2][e];
            const int s = carry[(g * k + r) * E + e] + rank;
            const bool kept = s < C;
            slot[static_cast<size_t>(t) * k + r] = kept ? s : -1;
            gate[static_cast<size_t>(t) * k + r] = kept ? probs[static_cast<size_t>(t) * E + e] : 0.0f;
        }
        __syncthreads();
    }
}

}  // namespace

size_t route_workspace_bytes(const Dims& D) { return route_ws_layout(D, nullptr).bytes; }

vmoe_status route_launch(const Dims& D, const void* x, const void* wr, const float* bias,
                         const float* noise, int flags, float* logits, float* probs,
                         int32_t* idx, int32_t* slot, float* gate, int32_t* order, int32_t* counts,
                         int32_t* row_base, void* ws_base, hipStream_t st) {
    RouteWs ws = route_ws_layout(D, ws_base);
    const int nch = static_cast<int>(cdiv(D.Ng, kSlotChunk));
    const int logits_in = (flags & VMOE_ROUTE_LOGITS_IN) ? 1 : 0;
    if (D.N > 0) {
        const int tpb = min(kGateTokens, 256 / D.E);
        dim3 grid(cdiv(D.Ng, tpb), D.G);
        if (D.dtype == VMOE_BF16)
            router_gate_kernel<uint16_t><<<grid, 256, 0, st>>>(
                static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(wr), bias, noise,
                logits, probs, idx, ws.keys, D.Ng, D.d, D.E, D.k, logits_in, tpb);
        else
            router_gate_kernel<float><<<grid, 256, 0, st>>>(
                static_cast<const float*>(x), static_cast<const float*>(wr), bias, noise, logits,
                probs, idx, ws.keys, D.Ng, D.d, D.E, D.k, logits_in, tpb);
        bin_scan_kernel<<<D.G, 1024, 0, st>>>(ws.keys, ws.binmap, ws.bin_start, ws.fill,
                                               ws.ccount, D.Ng, nch * D.k * D.E);
        bin_scatter_kernel<<<cdiv(D.N, 256), 256, 0, st>>>(ws.keys, ws.binmap, ws.bin_start,
                                                            ws.fill, ws.members, D.N, D.Ng);
        rank_kernel<<<cdiv(D.N, 256), 256, 0, st>>>(ws.keys, ws.binmap, ws.bin_start, ws.members,
                                                     idx, order, ws.ccount, D.N, D.Ng, D.E, D.k,
                                                     nch);
    }
    chunk_scan_kernel<<<1, 1024, 0, st>>>(ws.ccount, ws.cbase, ws.demand, ws.carry, counts,
                                          row_base, D.G, D.E, D.k, D.C, nch);
    if (D.N > 0)
        slots_kernel<<<dim3(nch, D.G), kSlotChunk, 0, st>>>(order, idx, probs, ws.cbase, ws.carry,
                                                            slot, gate, D.Ng, D.E, D.k, D.C, nch);
    return launch_status();
}

}  // namespace vmoe
