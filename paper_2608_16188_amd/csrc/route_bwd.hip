// Backward through the gate into the router on gfx950.
//
// One streaming kernel per (token chunk, column block, group): it forms
// dz = p * (dp - <p, dp>) for the chunk's tokens in LDS (dp is non-zero only
// at the kept experts), then walks the tokens once, adding dz W_r into dx
// (W_r columns in registers) and, unless the router is frozen, accumulating
// the chunk's partial of dW_r[e, i] = sum_t dz[t,e] x[t,i] in registers. A
// second kernel adds the partials over chunks in a fixed order
// (deterministic, no float atomics).
//
// Fused with the dispatch backward, the kernel starts each dx row from the
// token's kept expert rows of dxe, summed in j order (the dispatch backward's
// sum, so the result is bit-identical to the two calls in sequence), instead
// of reading dx: two f32 passes over dx and a launch fewer.
#include <type_traits>

#include "common.h"

namespace vmoe {

// (moves.hip) dx[t] = sum over kept j of dxe[row(t, j)]
vmoe_status dispatch_bwd_launch(const Dims& D, const void* dxe, const int32_t* idx,
                                const int32_t* slot, const int32_t* row_base, float* dx,
                                hipStream_t st);

namespace {

constexpr int kMinChunk = 64;

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
// The same columns as raw bits, converted only where they are used (so a
// load can stay in flight until then).
template <typename T, int VEC> struct RawCols;
template <int VEC> struct RawCols<uint16_t, VEC> {
    uint32_t w[VEC == 4 ? 2 : 1];
    __device__ __forceinline__ void load(const uint16_t* p) {
        if constexpr (VEC == 4) {
            const uint2 u = *reinterpret_cast<const uint2*>(p);
            w[0] = u.x; w[1] = u.y;
        } else if constexpr (VEC == 2) {
            w[0] = *reinterpret_cast<const uint32_t*>(p);
        } else {
            w[0] = *p;
        }
    }
    __device__ __forceinline__ void to_f32(float (&v)[VEC]) const {
#pragma unroll
        for (int i = 0; i < VEC; ++i)
            v[i] = bf16_to_f32(static_cast<uint16_t>(i % 2 ? w[i / 2] >> 16 : w[i / 2] & 0xFFFFu));
    }
};
template <int VEC> struct RawCols<float, VEC> {
    float w[VEC];
    __device__ __forceinline__ void load(const float* p) {
        float v[VEC];
        load_cols<VEC>(p, v);
#pragma unroll
        for (int i = 0; i < VEC; ++i) w[i] = v[i];
    }
    __device__ __forceinline__ void to_f32(float (&v)[VEC]) const {
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[i] = w[i];
    }
};

template <int VEC>
__device__ __forceinline__ void store_cols(float* p, const float (&v)[VEC]) {
    if constexpr (VEC == 4) *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
    else if constexpr (VEC == 2) *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
    else *p = v[0];
}

// The value a dx row starts from. KJ == 0: dx itself (accumulating call);
// KJ > 0: the sum over the token's kept assignments j < KJ of its dxe rows, in
// j order from 0, with the rows (-1 = not kept) taken from LDS.
template <typename T, int VEC, int KJ>
struct DxIn {
    RawCols<T, VEC> r[KJ];
    int kept;
    __device__ __forceinline__ void load(const T* dxe, const int* rows, int d, int ic) {
        kept = 0;
#pragma unroll
        for (int j = 0; j < KJ; ++j) {
            const int row = rows[j];
            kept |= (row >= 0 ? 1 : 0) << j;
            if (row >= 0) r[j].load(dxe + static_cast<size_t>(row) * d + ic);
        }
    }
    __device__ __forceinline__ void to_f32(float (&v)[VEC]) const {
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[i] = 0.0f;
#pragma unroll
        for (int j = 0; j < KJ; ++j) {
            if ((kept >> j) & 1) {
                float f[VEC];
                r[j].to_f32(f);
#pragma unroll
                for (int i = 0; i < VEC; ++i) v[i] += f[i];
            }
        }
    }
};
template <typename T, int VEC>
struct DxIn<T, VEC, 0> {
    RawCols<float, VEC> r;
    __device__ __forceinline__ void load(const float* dx, const int*, int, int) { r.load(dx); }
    __device__ __forceinline__ void to_f32(float (&v)[VEC]) const { r.to_f32(v); }
};

// Most tokens per chunk: the chunk's dz and dp rows stay within 32 KB of LDS.
template <int EMAX> struct ChunkMax {
    static constexpr int value = EMAX <= 16 ? 256 : (EMAX <= 32 ? 128 : 64);
};
static_assert(ChunkMax<64>::value >= kMinChunk, "chunk bounds");

// Columns per lane: a lane keeps E x VEC router weights and E x VEC gradient
// partials in registers.
template <int EMAX> struct ColsPerLane {
    static constexpr int value = EMAX <= 8 ? 4 : (EMAX <= 16 ? 2 : 1);
};

// Barrier for LDS traffic only: this wave's LDS accesses are complete
// (lgkmcnt 0) while its global loads may stay in flight (__syncthreads would
// also wait for those). The signal fences keep the compiler from moving
// memory accesses across it.
__device__ __forceinline__ void lds_barrier() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt, expcnt not waited for
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// global loads per thread issued together when forming dz: assignments,
// probabilities
constexpr int kBatch = 4;
constexpr int kProbBatch = 16;

// A token's dz row from LDS into registers (broadcast 16-byte reads).
template <int EMAX>
__device__ __forceinline__ void read_dz(const float (*dzs)[EMAX], int t, float (&r)[EMAX]) {
#pragma unroll
    for (int e = 0; e < EMAX; e += 4) {
        const float4 v = *reinterpret_cast<const float4*>(&dzs[t][e]);
        r[e] = v.x; r[e + 1] = v.y; r[e + 2] = v.z; r[e + 3] = v.w;
    }
}

// Step 1 of a chunk: dz[t][e] = p (dp - <p, dp>) for its ntok tokens into
// dzs (row stride LD floats; columns E..EMAX-1 are zero), with dps (same
// shape) as scratch for dp (NaN where the expert was not kept) and pdp_s for
// <p, dp>; with KJ > 0 also the dxe row of each kept assignment into rows_s
// [tokens][KJ] (-1 = not kept; row_base[g] staged in rb_s). The first batch
// of inputs (assignments and probability rows, clamped indices, no
// branches) is requested before `issue()` runs the caller's first streaming
// loads, so waiting for it leaves those in flight; the barriers wait for
// LDS traffic only.
template <int EMAX, int LD, int KJ, typename Issue>
__device__ __forceinline__ void form_dz(float* dzs, float* dps, float* pdp_s, int* rows_s,
                                        int* rb_s, const float* __restrict__ probs,
                                        const int32_t* __restrict__ idx,
                                        const int32_t* __restrict__ slot,
                                        const float* __restrict__ dgate,
                                        const int32_t* __restrict__ row_base,
                                        const float* __restrict__ dz_add, size_t tok0,
                                        int ntok, int E, int k, int g, long long gc,
                                        Issue issue) {
    const int tid = threadIdx.x;
    const int na = ntok * k, np = ntok * E;
    const size_t q0 = tok0 * k, p0 = tok0 * E;
    int sl[kBatch], ex[kBatch];
    float gv[kBatch], pv[kProbBatch];
    auto fetch_assign = [&](int b0) {
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const size_t q = q0 + min(b0 + u * 256 + tid, na - 1);
            sl[u] = slot[q];
            ex[u] = idx[q];
            gv[u] = dgate[q];
        }
    };
    // the chunk's probability rows are one contiguous run of ntok * E floats
    auto fetch_probs = [&](int b0) {
#pragma unroll
        for (int u = 0; u < kProbBatch; ++u) pv[u] = probs[p0 + min(b0 + u * 256 + tid, np - 1)];
    };
    fetch_assign(0);
    fetch_probs(0);
    issue();
    for (int q = tid; q < ntok * EMAX; q += 256) dps[(q / EMAX) * LD + q % EMAX] = __builtin_nanf("");
    if constexpr (KJ > 0) {
        for (int q = tid; q < ntok * KJ; q += 256) rows_s[q] = -1;
        if (tid < E) rb_s[tid] = row_base[static_cast<size_t>(g) * E + tid];
    }
    lds_barrier();
    for (int b0 = 0; b0 < na; b0 += kBatch * 256) {
        if (b0 > 0) fetch_assign(b0);
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int q = b0 + u * 256 + tid;
            if (q < na && sl[u] >= 0) {
                dps[(q / k) * LD + ex[u]] = gv[u];
                // row(t, j) = e G C + row_base[g, e] + slot (k <= KJ)
                if constexpr (KJ > 0)
                    rows_s[(q / k) * KJ + q % k] =
                        static_cast<int>(ex[u] * gc + rb_s[ex[u]] + sl[u]);
            }
        }
    }
    for (int b0 = 0; b0 < np; b0 += kProbBatch * 256) {
        if (b0 > 0) fetch_probs(b0);
#pragma unroll
        for (int u = 0; u < kProbBatch; ++u) {
            const int q = b0 + u * 256 + tid;
            if (q < np) dzs[(q / E) * LD + q % E] = pv[u];  // columns E..EMAX set below
        }
    }
    lds_barrier();
    if (tid < ntok) {
        // <p, dp> over the kept experts, e ascending (eight entries read at a
        // time; dp is NaN at every column not kept, E..EMAX included)
        float pdp = 0.0f;
        for (int e0 = 0; e0 < E; e0 += 8) {
            float dpv[8], pv8[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int e = min(e0 + u, EMAX - 1);
                dpv[u] = dps[tid * LD + e];
                pv8[u] = dzs[tid * LD + e];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (e0 + u < E && dpv[u] == dpv[u]) pdp = __builtin_fmaf(pv8[u], dpv[u], pdp);
        }
        pdp_s[tid] = pdp;
    }
    lds_barrier();
    if (dz_add == nullptr) {
        for (int q = tid; q < ntok * EMAX; q += 256) {
            const int t = q / EMAX, e = q % EMAX;
            const float p = dzs[t * LD + e], dp = dps[t * LD + e], pdp = pdp_s[t];
            // kept: p (dgate - <p, dp>); other experts: -p <p, dp>
            dzs[t * LD + e] = e >= E ? 0.0f : (dp == dp ? p * (dp - pdp) : -p * pdp);
        }
    } else {
        // the same, plus an extra gradient with respect to the logits (four
        // of its values requested before any is used)
        for (int q0 = tid; q0 < ntok * EMAX; q0 += 4 * 256) {
            float av[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int q = q0 + u * 256, t = q / EMAX, e = q % EMAX;
                av[u] = (q < ntok * EMAX && e < E) ? dz_add[(tok0 + t) * E + e] : 0.0f;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int q = q0 + u * 256, t = q / EMAX, e = q % EMAX;
                if (q >= ntok * EMAX) break;
                const float p = dzs[t * LD + e], dp = dps[t * LD + e], pdp = pdp_s[t];
                const float v = dp == dp ? p * (dp - pdp) : -p * pdp;
                dzs[t * LD + e] = e >= E ? 0.0f : v + av[u];
            }
        }
    }
    lds_barrier();
}

// Block = a chunk of tch tokens of group g (blockIdx.x, .z) times 64 * VEC
// columns (blockIdx.y), four waves; wave w takes the chunk's tokens w, w + 4,
// ..., with the x and dx rows of U tokens in flight.
//   1. the first round's loads are issued, then dz of the chunk is formed in
//      LDS: one thread per token adds <p, dp> over its kept assignments in j
//      order and records dp, then one thread per (token, expert) writes
//      kept ? p (dp - <p, dp>) : -p <p, dp>;
//   2. per token: dx[t, cols] += sum_e dz[t,e] W[e, cols] (e ascending) and
//      acc[e, cols] += dz[t,e] x[t, cols];
//   3. (DW) the four waves' partials are added in wave order through LDS and
//      written to the chunk's slot of `partial`.
//   (KJ > 0: the chunk's dxe row indices are formed with dz in step 1 and
//   the first round's loads follow it)
template <typename T, int EMAX, bool DW, int KJ>
__global__ __launch_bounds__(256) void route_bwd_kernel(
    const T* __restrict__ x, const T* __restrict__ wr, const float* __restrict__ probs,
    const int32_t* __restrict__ idx, const int32_t* __restrict__ slot,
    const float* __restrict__ dgate, float* __restrict__ dx, float* __restrict__ partial,
    const T* __restrict__ dxe, const int32_t* __restrict__ row_base,
    const float* __restrict__ dz_add, long long gc, int Ng, int d, int E, int k, int tch,
    int nch) {
    constexpr int VEC = ColsPerLane<EMAX>::value;
    constexpr int COLS = 64 * VEC;
    constexpr int U = EMAX <= 8 ? 4 : 8;  // tokens per wave in flight
    // LDS: dz (and, while it is formed, dp) of the chunk; afterwards waves
    // 1..3 hand their partials to wave 0 through the same space
    constexpr int CH = ChunkMax<EMAX>::value;
    constexpr int DZ_FLOATS = CH * EMAX, RED_FLOATS = DW ? 3 * EMAX * COLS : 0;
    __shared__ __attribute__((aligned(16)))
    float lds[2 * DZ_FLOATS > RED_FLOATS ? 2 * DZ_FLOATS : RED_FLOATS];
    __shared__ float pdp_s[CH];
    __shared__ int rows_s[KJ > 0 ? CH : 1][KJ > 0 ? KJ : 1];  // dxe rows, -1 = not kept
    __shared__ int rb_s[KJ > 0 ? EMAX : 1];                  // row_base[g, :]
    float (*dzs)[EMAX] = reinterpret_cast<float (*)[EMAX]>(lds);
    const int c = blockIdx.x, g = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int t0 = c * tch;
    const int ntok = min(tch, Ng - t0);
    const size_t tok0 = static_cast<size_t>(g) * Ng + t0;
    const int i0 = blockIdx.y * COLS + lane * VEC;
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
    using RX = RawCols<T, VEC>;
    using RD = DxIn<T, VEC, KJ>;
    // (token indices clamp to the chunk, so a wave past its last token reloads it)
    auto load_round = [&](int r0, RX (&xv)[U], RD (&dv)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int tl = min(r0 + 4 * u, ntok - 1);
            const size_t t = tok0 + tl;
            if constexpr (DW) xv[u].load(x + t * d + ic);
            if constexpr (KJ > 0) dv[u].load(dxe, &rows_s[tl][0], d, ic);
            else dv[u].load(dx + t * d + ic, nullptr, d, ic);
        }
    };
    RX xa[U], xb[U];
    RD da[U], db[U];

    // 1. dz of the chunk; the first round of x and dx rows is issued behind
    // the first batch of routing inputs (fused: after the dxe rows are known)
    float* dps = lds + DZ_FLOATS;
    form_dz<EMAX, EMAX, KJ>(lds, dps, pdp_s, &rows_s[0][0], rb_s, probs, idx, slot, dgate,
                            row_base, dz_add, tok0, ntok, E, k, g, gc, [&] {
                                if constexpr (KJ == 0) load_round(wave, xa, da);
                            });
    if constexpr (KJ > 0) load_round(wave, xa, da);

    // 2. stream the chunk's tokens
    float acc[DW ? EMAX : 1][VEC];
#pragma unroll
    for (int e = 0; e < (DW ? EMAX : 1); ++e)
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[e][v] = 0.0f;
    auto step = [&](int r0, RX (&xc)[U], RD (&dc)[U], RX (&xn)[U], RD (&dn)[U]) {
        if (r0 + 4 * U < ntok) load_round(r0 + 4 * U, xn, dn);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int tt = r0 + 4 * u;
            if (tt < ntok) {
                float z[EMAX];
                read_dz<EMAX>(dzs, tt, z);
                float dv[VEC], out[VEC];
                dc[u].to_f32(dv);
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    float s = 0.0f;
#pragma unroll
                    for (int e = 0; e < EMAX; ++e)
                        if (e < E) s = __builtin_fmaf(z[e], w[e][v], s);
                    out[v] = dv[v] + s;
                }
                store_cols<VEC>(dx + (tok0 + tt) * d + i0, out);
                if constexpr (DW) {
                    float xv[VEC];
                    xc[u].to_f32(xv);
#pragma unroll
                    for (int e = 0; e < EMAX; ++e)
#pragma unroll
                        for (int v = 0; v < VEC; ++v)
                            acc[e][v] = __builtin_fmaf(z[e], xv[v], acc[e][v]);
                }
            }
        }
    };
    if (live) {
        for (int r0 = wave; r0 < ntok; r0 += 8 * U) {
            step(r0, xa, da, xb, db);
            if (r0 + 4 * U < ntok) step(r0 + 4 * U, xb, db, xa, da);
        }
    }

    // 3. the chunk's partial of dW_r
    if constexpr (DW) {
        float (*red)[EMAX][COLS] = reinterpret_cast<float (*)[EMAX][COLS]>(lds);
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
                        out[v] = ((acc[e][v] + red[0][e][lane * VEC + v]) +
                                  red[1][e][lane * VEC + v]) +
                                 red[2][e][lane * VEC + v];
                    store_cols<VEC>(pg + static_cast<size_t>(e) * d + i0, out);
                }
            }
        }
    }
}

// ---------------------------------------------------------------- E > 16
//
// With many experts (bf16 layers) the two products of a token chunk are small
// GEMMs, dx[t, c] += sum_e dz[t, e] W[e, c] (k = E) and
// P[e, c] = sum_t dz[t, e] x[t, c] (k = the chunk's tokens), run on the bf16
// matrix cores (v_mfma_f32_32x32x16_bf16, f32 sums). x and W are bf16 already;
// dz (f32) enters as three bf16 terms dz = hi + mid + lo (each the rounded
// remainder of the previous), which carry its 24 significant bits, so every
// product dz W or dz x is formed as three exact bf16 products summed in f32.
//
// dz is formed first, once per token, by its own kernel (rbwd_dz_kernel) into
// the workspace, so the product kernel starts streaming at once: a block takes
// kRbCols columns of one group and walks chunks of kRbTok tokens, eight waves;
// W columns (transposed to [column][expert] bf16) are staged in LDS once, the
// chunk's dz rows (f32) and x rows by waves 4-7 one chunk ahead; dx wave w
// (0-3) computes dx for tokens [32 w, 32 w + 32) over the block's columns, and
// wave 4 + w the partial P for columns [32 w, 32 w + 32) over all experts,
// summed over the block's chunks.
constexpr int kRbTok = 128, kRbCols = 128;
constexpr int kRbXLd = kRbCols + 16;  // bf16 per staged x row (rows 32 bytes apart in banks)

typedef __bf16 bf16x8_r __attribute__((ext_vector_type(8)));
typedef float f32x16_r __attribute__((ext_vector_type(16)));
typedef short s16x4_r __attribute__((ext_vector_type(4)));
typedef short s16x8_r __attribute__((ext_vector_type(8)));

// dz[t, e] = p (dp - <p, dp>) (+ dz_add) for every token, f32 [N, E]: EL lanes
// per token (EL = the power of two >= E), lane e holding expert e; <p, dp> is
// summed over the kept experts in ascending e with fused multiply-adds (the
// order the fused kernel of fewer experts uses). With rows != null also the
// expert-buffer row of each kept assignment, rows [N, k] (-1 = dropped).
// KB: assignments read per pass (2, 4 or 8: the least that holds k when k
// <= 8, so a top-2 layer issues 6 loads per lane for them rather than 24).
template <int EL, int KB>
__global__ __launch_bounds__(256) void rbwd_dz_kernel(
    const float* __restrict__ probs, const int32_t* __restrict__ idx,
    const int32_t* __restrict__ slot, const float* __restrict__ dgate,
    const float* __restrict__ dz_add, const int32_t* __restrict__ row_base,
    float* __restrict__ dz, int32_t* __restrict__ rows, long long gc, int N, int Ng, int E,
    int k) {
    constexpr int TPB = 256 / EL;
    const int sub = threadIdx.x % EL;
    const int t = blockIdx.x * TPB + static_cast<int>(threadIdx.x) / EL;
    if (t >= N) return;  // uniform per group of EL lanes (EL divides 64)
    const size_t te = static_cast<size_t>(t) * E, tk = static_cast<size_t>(t) * k;
    const int g = t / Ng;
    // every input of the token requested together: its probabilities (lane e),
    // its first KB assignments (every lane), the group's row bases (lane e)
    const float p = sub < E ? probs[te + sub] : 0.0f;
    const float add = (dz_add != nullptr && sub < E) ? dz_add[te + sub] : 0.0f;
    const int rb = (rows != nullptr && sub < E) ? row_base[static_cast<size_t>(g) * E + sub] : 0;
    int ej[KB], sj[KB];
    float gj[KB];
#pragma unroll
    for (int u = 0; u < KB; ++u) {
        const size_t q = tk + min(u, k - 1);
        ej[u] = idx[q];
        sj[u] = slot[q];
        gj[u] = dgate[q];
    }
    float dp = 0.0f;
    int kept = 0;
    for (int j0 = 0; j0 < k; j0 += KB) {
        if (j0 > 0) {
#pragma unroll
            for (int u = 0; u < KB; ++u) {
                const size_t q = tk + min(j0 + u, k - 1);
                ej[u] = idx[q];
                sj[u] = slot[q];
                gj[u] = dgate[q];
            }
        }
#pragma unroll
        for (int u = 0; u < KB; ++u) {
            if (j0 + u < k && ej[u] == sub && sj[u] >= 0) {  // top-k experts are distinct
                dp = gj[u];
                kept = 1;
            }
        }
    }
    float pdp = 0.0f;
    if (k <= KB) {
        // the kept assignments' p[e_j] dgate_j, added in ascending e_j
        float pe[KB];
#pragma unroll
        for (int u = 0; u < KB; ++u) pe[u] = __shfl(p, ej[u] & (EL - 1), EL);
        int last = -1;
        for (int r = 0; r < k; ++r) {
            int best = 1 << 30, bu = -1;
#pragma unroll
            for (int u = 0; u < KB; ++u)
                if (u < k && sj[u] >= 0 && ej[u] > last && ej[u] < best) {
                    best = ej[u];
                    bu = u;
                }
            if (bu < 0) break;
            float pv = 0.0f, gv = 0.0f;
#pragma unroll
            for (int u = 0; u < KB; ++u)
                if (u == bu) {
                    pv = pe[u];
                    gv = gj[u];
                }
            pdp = __builtin_fmaf(pv, gv, pdp);
            last = best;
        }
    } else {
        for (int e = 0; e < E; ++e) {
            const float pe = __shfl(p, e, EL), de = __shfl(dp, e, EL);
            if (__shfl(kept, e, EL)) pdp = __builtin_fmaf(pe, de, pdp);
        }
    }
    if (sub < E) {
        float v = kept ? p * (dp - pdp) : -p * pdp;
        if (dz_add != nullptr) v = v + add;
        dz[te + sub] = v;
    }
    if (rows != nullptr) {
        // lane j < k: the expert-buffer row of assignment j (k <= KB here: the
        // fused call runs for k <= 4)
        int e = 0, sl = -1;
#pragma unroll
        for (int u = 0; u < KB; ++u)
            if (u == sub) {
                e = ej[u];
                sl = sj[u];
            }
        const int rbe = __shfl(rb, e & (EL - 1), EL);
        if (sub < k)
            rows[tk + sub] = sl >= 0 ? static_cast<int>(e * gc + rbe + sl) : -1;
    }
}

// Eight f32 values as three bf16x8 terms hi + mid + lo (round to nearest even
// at each step; each remainder is exact in f32).
__device__ __forceinline__ void split3(const float (&v)[8], bf16x8_r& hi, bf16x8_r& mid,
                                       bf16x8_r& lo) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const __bf16 h = static_cast<__bf16>(v[i]);
        const float r1 = v[i] - static_cast<float>(h);
        const __bf16 m = static_cast<__bf16>(r1);
        const float r2 = r1 - static_cast<float>(m);
        hi[i] = h;
        mid[i] = m;
        lo[i] = static_cast<__bf16>(r2);
    }
}

// ds_read_b64_tr_b16: within each 16-lane group, lane j reads 4 bf16 at its
// address and lane i receives element i % 4 of lanes i/4, i/4+4, i/4+8, i/4+12.
__device__ __forceinline__ s16x4_r rb_read_tr(const uint16_t* p) {
    typedef __attribute__((address_space(3))) s16x4_r* lds_s16x4;
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4)(p));
}

template <int EMAX, bool DW, int KJ>
__global__ __launch_bounds__(512) void route_bwd_mma_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ wr,
    const float* __restrict__ dz, const int32_t* __restrict__ rows,
    const uint16_t* __restrict__ dxe, float* __restrict__ dx, float* __restrict__ partial,
    int Ng, int d, int E, int k, int nch, int has_rows) {
    constexpr int TCH = kRbTok, COLS = kRbCols, DZLD = EMAX + 1, WLD = EMAX + 8;
    constexpr int KS = EMAX / 16;  // k-steps of the dx product
    __shared__ __attribute__((aligned(16))) float dzs[TCH * DZLD];
    __shared__ __attribute__((aligned(16))) uint16_t wts[COLS * WLD];
    __shared__ __attribute__((aligned(16))) uint16_t xs[TCH * kRbXLd];
    const int g = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int c0 = blockIdx.y * COLS;
    const uint16_t* wg = wr + static_cast<size_t>(g) * E * d;
    const int m = lane & 31, kh = lane >> 5;
    // waves 0-3 form dx, waves 4-7 stage the tiles and form the router-
    // gradient partial
    const bool dx_wave = wave < 4;
    const int rw = wave & 3;
    constexpr int NJ = COLS / 32;
    constexpr int NT = 512;
    // the per-chunk dz and x tiles are loaded and staged by the 256 threads
    // of the router-gradient waves (the dx waves' registers hold their
    // products and incoming dxe rows)
    constexpr int NTT = 256;
    constexpr int DZV = TCH * EMAX / NTT;     // dz values per loading thread
    constexpr int WV = EMAX * COLS / 8 / NT;  // 16-byte W vectors per thread
    constexpr int XV = TCH * COLS / 8 / NTT;  // 16-byte x vectors per loading thread
    static_assert(DZV * NTT == TCH * EMAX && WV * NT * 8 == EMAX * COLS &&
                      XV * NTT * 8 == TCH * COLS, "tiles split evenly over the threads");
    // the block's W columns, the same for every chunk it takes: staged once
    // (transposed to [column][expert]); the first chunk's barrier publishes it
    {
        uint4 wv[WV];
#pragma unroll
        for (int u = 0; u < WV; ++u) {
            const int q = u * NT + tid, e = q / (COLS / 8), col = c0 + (q % (COLS / 8)) * 8;
            wv[u] = (e < E && col < d)
                        ? *reinterpret_cast<const uint4*>(wg + static_cast<size_t>(e) * d + col)
                        : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int u = 0; u < WV; ++u) {
            const int q = u * NT + tid, e = q / (COLS / 8), cl = (q % (COLS / 8)) * 8;
            const uint32_t hw[4] = {wv[u].x, wv[u].y, wv[u].z, wv[u].w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                wts[(cl + 2 * i) * WLD + e] = static_cast<uint16_t>(hw[i] & 0xFFFFu);
                wts[(cl + 2 * i + 1) * WLD + e] = static_cast<uint16_t>(hw[i] >> 16);
            }
        }
    }
    // The token chunks blockIdx.x, blockIdx.x + gridDim.x, ... of the group,
    // in order, software-pipelined: the next chunk's dz and x tiles (and the
    // fused call's row indices) are requested before this chunk's products,
    // the dx waves' incoming values right after this chunk's dx rows are
    // written, so a chunk's load latency hides behind the previous chunk's
    // work. Every load and store in the loops is unconditional (clamped
    // addresses with the value selected afterwards, buffer stores that drop
    // out-of-range offsets; the last chunk's prefetch repeats it), so the
    // compiler's wait counts are exact and leave the prefetched loads in
    // flight. Waves 0-3 form dx; waves 4-7 load and stage the tiles and form
    // the router-gradient partial; each role runs a loop of its own with the
    // same two LDS barriers per chunk.
    constexpr int MB = EMAX / 32;
    const int tt = tid - NTT;  // a router-gradient wave's thread: 0 .. 255
    float dzv[DZV];
    uint4 xv[XV];
    // stage 1 of chunk c (router-gradient waves): this thread's share of the
    // dz and x tiles, zero past the chunk, the experts or d (buffer loads over
    // the chunk's rows: rows past it, and offsets set out of range for
    // experts past E or columns past d, read zeros)
    auto load_tiles = [&](int c) {
        const int t0 = c * TCH;
        const int ntok = min(TCH, Ng - t0);
        const size_t tok0 = static_cast<size_t>(g) * Ng + t0;
        const __amdgpu_buffer_rsrc_t rz =
            make_rsrc(dz + tok0 * E, static_cast<long long>(ntok) * E * 4);
#pragma unroll
        for (int u = 0; u < DZV; ++u) {
            const int q = u * NTT + tt, r = q / EMAX, e = q % EMAX;
            const uint32_t off = e < E ? static_cast<uint32_t>(r * E + e) * 4u : kOutOfRange;
            dzv[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rz, off, 0, 0));
        }
        if constexpr (DW) {
            const __amdgpu_buffer_rsrc_t rx =
                make_rsrc(x + tok0 * d, static_cast<long long>(ntok) * d * 2);
#pragma unroll
            for (int u = 0; u < XV; ++u) {
                const int q = u * NTT + tt, r = q / (COLS / 8), col = c0 + (q % (COLS / 8)) * 8;
                const uint32_t off =
                    col < d ? static_cast<uint32_t>(r * d + col) * 2u : kOutOfRange;
                xv[u] = buf_load16(rx, off);
            }
        }
    };
    // stage 2: into LDS
    auto stage_tiles = [&]() {
#pragma unroll
        for (int u = 0; u < DZV; ++u) {
            const int q = u * NTT + tt;
            dzs[(q / EMAX) * DZLD + q % EMAX] = dzv[u];
        }
        if constexpr (DW) {
#pragma unroll
            for (int u = 0; u < XV; ++u) {
                const int q = u * NTT + tt, r = q / (COLS / 8), v = q % (COLS / 8);
                *reinterpret_cast<uint4*>(xs + r * kRbXLd + v * 8) = xv[u];
            }
        }
    };
    const bool any_chunk = static_cast<int>(blockIdx.x) < nch;  // uniform per block

    if (dx_wave) {
        // the dx rows of the lane: token tl of the chunk; register 4 q + r of
        // lane l holds token 32 w + l % 32, column 32 j + 8 q + 4 (l / 32) + r
        const int tl = 32 * rw + m;
        int rn[KJ > 0 ? KJ : 1];
        bool keep[KJ > 0 ? KJ : 1];
        float4 dxin[KJ == 0 ? NJ : 1][4];
        uint2 h[KJ > 0 ? KJ : 1][NJ][4];
        // (fused) the expert-buffer rows of the token's assignments, -1 dropped
        auto load_rows = [&](int c) {
            if constexpr (KJ > 0) {
                const int t0 = c * TCH;
                const int ntok = min(TCH, Ng - t0);
                const size_t tok0 = static_cast<size_t>(g) * Ng + t0;
#pragma unroll
                for (int jj = 0; jj < KJ; ++jj) {
                    const int v = rows[(tok0 + min(tl, ntok - 1)) * k + min(jj, k - 1)];
                    rn[jj] = jj < k ? v : -1;
                }
            }
        };
        // the incoming value of each dx element of chunk c: dx itself, or
        // (fused) the kept dxe rows of the row indices in rn; a dropped
        // assignment reads the first row of the expert buffers (of x when
        // they are empty) and its value is discarded
        auto load_in = [&](int c) {
            if constexpr (KJ == 0) {
                const int t0 = c * TCH;
                const int ntok = min(TCH, Ng - t0);
                const __amdgpu_buffer_rsrc_t rdx =
                    make_rsrc(dx + (static_cast<size_t>(g) * Ng + t0) * d,
                              static_cast<long long>(ntok) * d * 4);
#pragma unroll
                for (int j = 0; j < NJ; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int col = c0 + 32 * j + 8 * q + 4 * kh;
                        const uint32_t off =
                            col < d ? static_cast<uint32_t>(tl * d + col) * 4u : kOutOfRange;
                        const v4i32 v = __builtin_amdgcn_raw_buffer_load_b128(rdx, off, 0, 0);
                        dxin[j][q] = __builtin_bit_cast(float4, v);
                    }
            } else {
#pragma unroll
                for (int jj = 0; jj < KJ; ++jj) {
                    keep[jj] = rn[jj] >= 0;
                    const uint16_t* src = keep[jj] ? dxe + static_cast<size_t>(rn[jj]) * d
                                                   : (has_rows ? dxe : x);
#pragma unroll
                    for (int j = 0; j < NJ; ++j)
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const int col = min(c0 + 32 * j + 8 * q + 4 * kh, d - 4);
                            h[jj][j][q] = *reinterpret_cast<const uint2*>(src + col);
                        }
                }
            }
        };
        f32x16_r acc[NJ];
        if (any_chunk) {
            load_rows(blockIdx.x);
            load_in(blockIdx.x);
        }
        for (int c = blockIdx.x; c < nch; c += gridDim.x) {
            const int cn = min(c + static_cast<int>(gridDim.x), nch - 1);
            // the tiles of chunk c are staged; LDS only: the dx inputs stay in flight
            lds_barrier();
            load_rows(cn);
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int i = 0; i < 16; ++i) acc[j][i] = 0.0f;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                // A: dz[token m][e = 16 ks + 8 kh .. +7] as three bf16 terms
                float a8[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) a8[i] = dzs[tl * DZLD + 16 * ks + 8 * kh + i];
                bf16x8_r ahi, amid, alo;
                split3(a8, ahi, amid, alo);
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    // B: W[e][column 32 j + m], from the transposed tile
                    const bf16x8_r b = *reinterpret_cast<const bf16x8_r*>(
                        wts + (32 * j + m) * WLD + 16 * ks + 8 * kh);
                    acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, alo, acc[j], 0, 0, 0);
                    acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, amid, acc[j], 0, 0, 0);
                    acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b, ahi, acc[j], 0, 0, 0);
                }
            }
            // dx rows of the chunk: rows past the chunk and columns past d are
            // out of the store buffer's range
            const int t0 = c * TCH;
            const int ntok = min(TCH, Ng - t0);
            const __amdgpu_buffer_rsrc_t rdx =
                make_rsrc(dx + (static_cast<size_t>(g) * Ng + t0) * d,
                          static_cast<long long>(ntok) * d * 4);
#pragma unroll
            for (int j = 0; j < NJ; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float4 din;
                    if constexpr (KJ == 0) {
                        din = dxin[j][q];
                    } else {
                        float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                        for (int jj = 0; jj < KJ; ++jj) {
                            // a dropped assignment adds nothing (not even a signed zero)
                            const uint2 hv = h[jj][j][q];
                            const float h0 = bf16_to_f32(static_cast<uint16_t>(hv.x & 0xFFFFu));
                            const float h1 = bf16_to_f32(static_cast<uint16_t>(hv.x >> 16));
                            const float h2 = bf16_to_f32(static_cast<uint16_t>(hv.y & 0xFFFFu));
                            const float h3 = bf16_to_f32(static_cast<uint16_t>(hv.y >> 16));
                            v[0] = keep[jj] ? v[0] + h0 : v[0];
                            v[1] = keep[jj] ? v[1] + h1 : v[1];
                            v[2] = keep[jj] ? v[2] + h2 : v[2];
                            v[3] = keep[jj] ? v[3] + h3 : v[3];
                        }
                        din = make_float4(v[0], v[1], v[2], v[3]);
                    }
                    const int col = c0 + 32 * j + 8 * q + 4 * kh;
                    const uint32_t off =
                        col < d ? static_cast<uint32_t>(tl * d + col) * 4u : kOutOfRange;
                    const float4 o =
                        make_float4(din.x + acc[j][4 * q], din.y + acc[j][4 * q + 1],
                                    din.z + acc[j][4 * q + 2], din.w + acc[j][4 * q + 3]);
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4i32, o), rdx, off,
                                                           0, 0);
                }
            // the next chunk's incoming values, now that this chunk's are used
            load_in(cn);
            // every wave is done with this chunk's tiles before the next overwrites them
            lds_barrier();
        }
        return;
    }

    // router-gradient waves: P[e][column] += over the chunk's tokens, columns
    // [32 w, 32 w + 32): A = dz^T (expert m, tokens 16 s + 8 kh .. +7, three
    // terms), B = x (column m, the same tokens), read transposed from the x tile
    f32x16_r acc[MB];
#pragma unroll
    for (int b = 0; b < MB; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[b][i] = 0.0f;
    if (any_chunk) load_tiles(blockIdx.x);
    for (int c = blockIdx.x; c < nch; c += gridDim.x) {
        const int cn = min(c + static_cast<int>(gridDim.x), nch - 1);
        stage_tiles();
        lds_barrier();
        load_tiles(cn);
        if constexpr (DW) {
            const int ntok = min(TCH, Ng - c * TCH);
            const int gq = lane >> 4, jq = lane & 15;
            const int ntk = (ntok + 15) / 16;  // rows past the chunk are zero in both tiles
            for (int s = 0; s < ntk; ++s) {
                const int kt = 16 * s + 8 * (gq >> 1) + (jq >> 2);
                const int mn = 32 * rw + 16 * (gq & 1) + 4 * (jq & 3);
                const s16x4_r lo4 = rb_read_tr(xs + kt * kRbXLd + mn);
                const s16x4_r hi4 = rb_read_tr(xs + (kt + 4) * kRbXLd + mn);
                const bf16x8_r bx = __builtin_bit_cast(
                    bf16x8_r, __builtin_shufflevector(lo4, hi4, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
                for (int b = 0; b < MB; ++b) {
                    float a8[8];
#pragma unroll
                    for (int i = 0; i < 8; ++i)
                        a8[i] = dzs[(16 * s + 8 * kh + i) * DZLD + 32 * b + m];
                    bf16x8_r ahi, amid, alo;
                    split3(a8, ahi, amid, alo);
                    acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bx, alo, acc[b], 0, 0, 0);
                    acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bx, amid, acc[b], 0, 0, 0);
                    acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bx, ahi, acc[b], 0, 0, 0);
                }
            }
        }
        // every wave is done with this chunk's tiles before the next overwrites them
        lds_barrier();
    }

    if constexpr (DW) {
        // register 4 q + r of lane l: expert 32 b + l % 32, column
        // 32 w + 8 q + 4 (l / 32) + r
        float* pg = partial + (static_cast<size_t>(g) * gridDim.x + blockIdx.x) * E * d;
#pragma unroll
        for (int b = 0; b < MB; ++b) {
            const int e = 32 * b + m;
            if (e < E) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int col = c0 + 32 * rw + 8 * q + 4 * kh;
                    if (col < d)
                        *reinterpret_cast<float4*>(pg + static_cast<size_t>(e) * d + col) =
                            make_float4(acc[b][4 * q], acc[b][4 * q + 1], acc[b][4 * q + 2],
                                        acc[b][4 * q + 3]);
                }
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
        // chunks r, r + 8, ... added in that order, eight loads in flight
        int c = r;
        for (; c + 56 < nch; c += 64) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = p[(c + 8 * u) * ed];
#pragma unroll
            for (int u = 0; u < 8; ++u) s += v[u];
        }
        for (; c < nch; c += 8) s += p[c * ed];
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
    int npart;  // router-gradient partials per group (the reducer's count)
    int nblk;   // matrix-core kernel: blocks per (group, column block)
};

ChunkPlan plan(const Dims& D) {
    // bf16 with E > 16: the matrix-core kernel's fixed chunk; about one
    // block per CU over (column blocks, groups), each taking an even share of
    // the chunks in turn and writing one partial
    if (D.dtype == VMOE_BF16 && D.E > 16) {
        const int nch = D.Ng > 0 ? static_cast<int>(cdiv(D.Ng, kRbTok)) : 0;
        const long long per = static_cast<long long>(D.G) * cdiv(D.d, kRbCols);
        int nb = static_cast<int>(256 / per);
        nb = nb < 1 ? 1 : (nb > nch ? nch : nb);
        if (nb > 0) nb = static_cast<int>(cdiv(nch, cdiv(nch, nb)));
        return ChunkPlan{kRbTok, nch, nb, nb};
    }
    // about 1024 blocks over (chunks, column blocks, groups)
    const int cols = 64 * (D.E <= 8    ? ColsPerLane<8>::value
                           : D.E <= 16 ? ColsPerLane<16>::value
                                       : ColsPerLane<64>::value);
    const int colblocks = static_cast<int>(cdiv(D.d, cols));
    int target = 1024 / (D.G * colblocks);
    if (target < 1) target = 1;
    int tch = D.Ng > 0 ? static_cast<int>(cdiv(D.Ng, target)) : 1;
    const int tmax = D.E <= 8    ? ChunkMax<8>::value
                     : D.E <= 16 ? ChunkMax<16>::value
                     : D.E <= 32 ? ChunkMax<32>::value
                                 : ChunkMax<64>::value;
    tch = tch < kMinChunk ? kMinChunk : (tch > tmax ? tmax : tch);
    const int nch = D.Ng > 0 ? static_cast<int>(cdiv(D.Ng, tch)) : 0;
    return ChunkPlan{tch, nch, nch, nch};
}

// Inputs of one launch of the main kernel (dxe, row_base, gc: fused only).
struct BwdArgs {
    const void *x, *wr;
    const float* probs;
    const int32_t *idx, *slot;
    const float* dgate;
    float *dx, *partial;
    const void* dxe;
    const int32_t* row_base;
    const float* dz_add;  // extra gradient with respect to the logits, or null
    float* dz;            // bf16 with E > 16: dz [N, E] (workspace)
    int32_t* rows;        // bf16 with E > 16, fused: expert-buffer rows [N, k] (workspace)
};

// bf16 layers with more than 16 experts: dz (and the fused call's rows) in
// the workspace after the partials.
bool uses_dz_pass(const Dims& D) { return D.dtype == VMOE_BF16 && D.E > 16; }

template <typename T, int EMAX, int KJ>
void launch_main(const Dims& D, const ChunkPlan& P, const BwdArgs& a, hipStream_t st) {
    if constexpr (std::is_same<T, uint16_t>::value && EMAX >= 32) {
        const long long gc = static_cast<long long>(D.G) * D.C;
        constexpr int TPB = 256 / EMAX;
        auto dz_pass = [&](auto kern) {
            kern<<<cdiv(D.N, TPB), 256, 0, st>>>(a.probs, a.idx, a.slot, a.dgate, a.dz_add,
                                                 a.row_base, a.dz, KJ > 0 ? a.rows : nullptr, gc,
                                                 D.N, D.Ng, D.E, D.k);
        };
        if (D.k <= 2) dz_pass(rbwd_dz_kernel<EMAX, 2>);
        else if (D.k <= 4) dz_pass(rbwd_dz_kernel<EMAX, 4>);
        else dz_pass(rbwd_dz_kernel<EMAX, 8>);
        const dim3 grid(P.nblk, cdiv(D.d, kRbCols), D.G);
        auto go = [&](auto kern) {
            kern<<<grid, 512, 0, st>>>(static_cast<const uint16_t*>(a.x),
                                       static_cast<const uint16_t*>(a.wr), a.dz, a.rows,
                                       static_cast<const uint16_t*>(a.dxe), a.dx, a.partial,
                                       D.Ng, D.d, D.E, D.k, P.nch, gc > 0 ? 1 : 0);
        };
        if (a.partial) go(route_bwd_mma_kernel<EMAX, true, KJ>);
        else go(route_bwd_mma_kernel<EMAX, false, KJ>);
        return;
    }
    constexpr int COLS = 64 * ColsPerLane<EMAX>::value;
    const dim3 grid(P.nch, cdiv(D.d, COLS), D.G);
    const long long gc = static_cast<long long>(D.G) * D.C;
    auto go = [&](auto kern) {
        kern<<<grid, 256, 0, st>>>(static_cast<const T*>(a.x), static_cast<const T*>(a.wr),
                                   a.probs, a.idx, a.slot, a.dgate, a.dx, a.partial,
                                   static_cast<const T*>(a.dxe), a.row_base, a.dz_add, gc, D.Ng,
                                   D.d, D.E, D.k, P.tch, P.nch);
    };
    if (a.partial) go(route_bwd_kernel<T, EMAX, true, KJ>);
    else go(route_bwd_kernel<T, EMAX, false, KJ>);
}

template <typename T, int KJ>
void launch_main_e(const Dims& D, const ChunkPlan& P, const BwdArgs& a, hipStream_t st) {
    if (D.E <= 8) launch_main<T, 8, KJ>(D, P, a, st);
    else if (D.E <= 16) launch_main<T, 16, KJ>(D, P, a, st);
    else if (D.E <= 32) launch_main<T, 32, KJ>(D, P, a, st);
    else launch_main<T, 64, KJ>(D, P, a, st);
}

template <int KJ>
void launch_main_t(const Dims& D, const ChunkPlan& P, const BwdArgs& a, hipStream_t st) {
    if (D.dtype == VMOE_BF16) launch_main_e<uint16_t, KJ>(D, P, a, st);
    else launch_main_e<float, KJ>(D, P, a, st);
}

// The main kernel (fused: KJ = 2 or 4) and the reduction of the partials.
vmoe_status run_route_bwd(const Dims& D, BwdArgs a, float* dwr, void* ws, int kj,
                          hipStream_t st) {
    const ChunkPlan P = plan(D);
    const long long total = static_cast<long long>(D.G) * D.E * D.d;
    if (D.N == 0) {
        // no tokens: the router gradient is zero (written by the reducer, nch = 0)
        if (dwr && total > 0)
            route_bwd_reduce_kernel<<<cdiv(total, 32), 256, 0, st>>>(nullptr, dwr, D.E, D.d, 0,
                                                                      total);
        return launch_status();
    }
    a.partial = dwr ? static_cast<float*>(ws) : nullptr;
    if (uses_dz_pass(D)) {
        // after the partials (whose bytes are a multiple of 16: d % 8 == 0)
        char* p = static_cast<char*>(ws) + sizeof(float) * static_cast<size_t>(D.G) * P.nch * D.E * D.d;
        a.dz = reinterpret_cast<float*>(p);
        a.rows = reinterpret_cast<int32_t*>(p + sizeof(float) * static_cast<size_t>(D.N) * D.E);
    }
    if (kj == 0) launch_main_t<0>(D, P, a, st);
    else if (kj == 2) launch_main_t<2>(D, P, a, st);
    else launch_main_t<4>(D, P, a, st);
    if (dwr)
        route_bwd_reduce_kernel<<<cdiv(total, 32), 256, 0, st>>>(a.partial, dwr, D.E, D.d,
                                                                  P.npart, total);
    return launch_status();
}

}  // namespace

// Workspace: the per-chunk router-gradient partials [G, chunks, E, d] f32;
// bf16 layers with more than 16 experts also dz [N, E] f32 and rows [N, k] i32.
size_t route_bwd_workspace_bytes(const Dims& D) {
    const ChunkPlan P = plan(D);
    size_t b = sizeof(float) * static_cast<size_t>(D.G) * P.nch * D.E * D.d;
    if (uses_dz_pass(D))
        b += sizeof(float) * static_cast<size_t>(D.N) * D.E +
             sizeof(int32_t) * static_cast<size_t>(D.N) * D.k;
    return b;
}

vmoe_status route_bwd_launch(const Dims& D, const void* x, const void* wr, const float* probs,
                             const int32_t* idx, const int32_t* slot, const float* dgate,
                             const float* dz_add, float* dx, float* dwr, void* ws,
                             hipStream_t st) {
    const BwdArgs a{x, wr, probs, idx, slot, dgate, dx, nullptr, nullptr, nullptr, dz_add,
                    nullptr, nullptr};
    return run_route_bwd(D, a, dwr, ws, 0, st);
}

vmoe_status dispatch_route_bwd_launch(const Dims& D, const void* dxe, const int32_t* row_base,
                                      const void* x, const void* wr, const float* probs,
                                      const int32_t* idx, const int32_t* slot,
                                      const float* dgate, const float* dz_add, float* dx,
                                      float* dwr, void* ws, hipStream_t st) {
    // the gathered rows are indexed in int and kept in LDS for k <= 4, and a
    // lane gathers at least two columns per row (E <= 16, or the matrix-core
    // kernel of bf16 layers with more experts; f32 with E > 16 would gather
    // one column per lane, which measured slower than the separate dispatch
    // pass); otherwise the two passes run one after the other (same result)
    const long long rows = static_cast<long long>(D.E) * D.G * D.C;
    if (D.k > 4 || (D.E > 16 && D.dtype != VMOE_BF16) || rows >= (1ll << 31) || D.N == 0) {
        const vmoe_status s = dispatch_bwd_launch(D, dxe, idx, slot, row_base, dx, st);
        if (s != VMOE_OK) return s;
        return route_bwd_launch(D, x, wr, probs, idx, slot, dgate, dz_add, dx, dwr, ws, st);
    }
    const BwdArgs a{x, wr, probs, idx, slot, dgate, dx, nullptr, dxe, row_base, dz_add,
                    nullptr, nullptr};
    return run_route_bwd(D, a, dwr, ws, D.k <= 2 ? 2 : 4, st);
}

}  // namespace vmoe
