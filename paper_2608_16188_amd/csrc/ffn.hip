// Expert MLP forward and backward as grouped GEMMs on gfx950.
//
// bf16 path: one templated matrix-core kernel, C[M x N] = sum_k A(m,k) B(n,k),
// per expert (grid.z). Tiles of 128 x 128 x 64 per 256-thread block, four
// waves in 2 x 2, each wave 64 x 64 as 4 x 4 blocks of
// v_mfma_f32_16x16x32_bf16 with f32 accumulation. Both operands are staged
// in LDS k-contiguous (double buffered, one barrier per k-step); an operand
// whose k index is strided in HBM (weights read transposed in the backward,
// the row-reduced weight-gradient GEMMs) is loaded as 4 k-rows x 8 values
// per thread and transposed in registers on its way into LDS. The operand
// roles are swapped inside the MFMA so each lane ends up holding 4
// consecutive output columns of one row, which the fused epilogues (bias,
// GELU, GELU', bf16 rounding, f32 weight gradients) store directly.
//
// Each expert's row count n_e = sum_g counts[g, e] is read on the device:
// tiles past n_e exit at once (M = n_e GEMMs) or n_e bounds the k loop
// (weight-gradient GEMMs, which still write zeros for an empty expert).
//
// f32 path: a plain LDS-tiled FMA kernel with the same operand and epilogue
// description (small widths; accuracy path).
#include <type_traits>

#include "common.h"

namespace vmoe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

enum Epi { EPI_FWD1 = 0, EPI_BIAS = 1, EPI_GELU_GRAD = 2, EPI_STORE = 3, EPI_F32 = 4 };

// Operand: element (mn, k) of expert e is
//   k-major : base[e*estride + mn*ld + k]
//   mn-major: base[e*estride + k*ld + mn]
struct Operand {
    const void* base;
    long long estride;
    int ld;
};

struct GemmArgs {
    Operand a, b;
    int M, N, K;            // static sizes; M or K is replaced by n_e (see var_k)
    int var_k;              // 0: M = n_e, 1: K = n_e
    const int32_t* counts;  // [G, E]
    int G, E;
    void* out;              // primary output (EPI_FWD1: gelu(H))
    void* out2;             // EPI_FWD1: gelu'(H)
    long long out_estride;
    int ldo;
    const void* bias;       // EPI_FWD1 / EPI_BIAS
    long long bias_estride;
    const void* aux;        // EPI_GELU_GRAD: saved gelu'(H)
    float* bsum;            // EPI_F32 (bf16 path): row sums of A per expert, or null
};

__device__ __forceinline__ int expert_rows(const int32_t* counts, int G, int E, int e) {
    int n = 0;
    for (int g = 0; g < G; ++g) n += counts[g * E + e];
    return n;
}

__device__ __forceinline__ float gelu_f(float h) {
    return 0.5f * h * (1.0f + erff(h * 0.70710678118654752f));
}

__device__ __forceinline__ float gelu_grad_f(float h) {
    return 0.5f * (1.0f + erff(h * 0.70710678118654752f)) +
           h * 0.39894228040143268f * __expf(-0.5f * h * h);
}

// ------------------------------------------------------------------ bf16 MFMA

constexpr int BK = 64;          // k depth of one LDS stage
constexpr int KPAD = 8;         // k-major rows: 64 + 8 bf16 = 144 B pitch
// mn-major rows: ROWS + 32 bf16, a pitch of 16 (mod 64) dwords, so the two
// 16-lane groups of a transpose read (4 rows x 32 B each) hit disjoint banks
constexpr int MNPAD = 32;

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

// LDS elements of one operand stage: k-major [ROWS][BK + KPAD], mn-major [BK][ROWS + MNPAD].
template <int ROWS, bool KMAJOR>
__host__ __device__ constexpr int stage_elems() {
    return KMAJOR ? ROWS * (BK + KPAD) : BK * (ROWS + MNPAD);
}

typedef int v4i32 __attribute__((ext_vector_type(4)));

// Raw buffer over one expert's operand: loads at byte offsets >= `bytes` return
// zeros in hardware, which implements every tail mask without a branch.
constexpr uint32_t kOutOfRange = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, long long bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                             static_cast<int>(bytes), 0x00020000);
}

__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
    const v4i32 v = __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
}

// Global -> registers: one ROWS x BK operand stage, ROWS * 8 / NT vectors of
// 8 bf16 per thread, each row segment read by consecutive lanes (coalesced).
template <int ROWS, bool KMAJOR, int NT>
__device__ __forceinline__ void load_stage(__amdgpu_buffer_rsrc_t rs, int ld, int mn0, int mn_lim,
                                           int k0, int k_lim, uint4 (&r)[ROWS * 8 / NT]) {
    const int tid = threadIdx.x;
    if (KMAJOR) {
        const int kc = (tid & 7) * 8;
#pragma unroll
        for (int j = 0; j < ROWS * 8 / NT; ++j) {
            const int mn = mn0 + (tid >> 3) + (NT / 8) * j;
            const bool ok = (mn < mn_lim) && (k0 + kc < k_lim);
            r[j] = buf_load16(rs, ok ? static_cast<uint32_t>(mn * ld + k0 + kc) * 2u : kOutOfRange);
        }
    } else {
        constexpr int VPR = ROWS / 8;  // vectors per k row
        const int mc = mn0 + (tid % VPR) * 8;
#pragma unroll
        for (int j = 0; j < ROWS * 8 / NT; ++j) {
            const int kr = k0 + tid / VPR + (NT / VPR) * j;
            const bool ok = (kr < k_lim) && (mc < mn_lim);
            r[j] = buf_load16(rs, ok ? static_cast<uint32_t>(kr * ld + mc) * 2u : kOutOfRange);
        }
    }
}

// Registers -> LDS, same element placement as the global tile (no transpose).
template <int ROWS, bool KMAJOR, int NT>
__device__ __forceinline__ void store_stage(uint16_t* s, const uint4 (&r)[ROWS * 8 / NT]) {
    const int tid = threadIdx.x;
    if (KMAJOR) {
        const int kc = (tid & 7) * 8;
#pragma unroll
        for (int j = 0; j < ROWS * 8 / NT; ++j)
            *reinterpret_cast<uint4*>(s + ((tid >> 3) + (NT / 8) * j) * (BK + KPAD) + kc) = r[j];
    } else {
        constexpr int VPR = ROWS / 8;
        const int mc = (tid % VPR) * 8;
#pragma unroll
        for (int j = 0; j < ROWS * 8 / NT; ++j)
            *reinterpret_cast<uint4*>(s + (tid / VPR + (NT / VPR) * j) * (ROWS + MNPAD) + mc) =
                r[j];
    }
}

// ds_read_b64_tr_b16: within each 16-lane group, lane j reads 4 bf16 at its
// address and lane i receives element i % 4 of lanes i/4, i/4+4, i/4+8, i/4+12.
// With lane j pointing at row j/4, column 4*(j%4) of a 4 x 16 block, lane i
// gets column i: four consecutive k values of one mn index.
__device__ __forceinline__ s16x4 lds_read_tr(const uint16_t* p) {
    typedef __attribute__((address_space(3))) s16x4* lds_s16x4;
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4)(p));
}

// Operand fragment of v_mfma_f32_32x32x16_bf16 for 32 mn values (lane & 31)
// x 8 k values (k = 16 * kstep + 8 * (lane >> 5) + 0..7).
template <int ROWS, bool KMAJOR>
__device__ __forceinline__ bf16x8 read_frag(const uint16_t* s, int blk, int kstep, int lane) {
    if (KMAJOR) {
        return *reinterpret_cast<const bf16x8*>(s + (blk * 32 + (lane & 31)) * (BK + KPAD) +
                                                kstep * 16 + (lane >> 5) * 8);
    } else {
        // 16-lane group g covers mn [16 (g & 1), +16) and k [8 (g >> 1), +8)
        constexpr int P = ROWS + MNPAD;
        const int g = lane >> 4, j = lane & 15;
        const uint16_t* p0 = s + (kstep * 16 + 8 * (g >> 1) + (j >> 2)) * P + blk * 32 +
                             16 * (g & 1) + 4 * (j & 3);
        const s16x4 lo = lds_read_tr(p0);
        const s16x4 hi = lds_read_tr(p0 + 4 * P);
        const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        return __builtin_bit_cast(bf16x8, v);
    }
}

template <int BM_, int BN_, int WGM, int WGN, bool A_KMAJOR, bool B_KMAJOR>
struct Frags {
    static constexpr int FM = BM_ / WGM / 32, FN = BN_ / WGN / 32;  // 32 x 32 blocks per wave
    bf16x8 a[FM], b[FN];
    __device__ __forceinline__ void read(const uint16_t* As, const uint16_t* Bs, int wm, int wn,
                                         int ks, int lane) {
#pragma unroll
        for (int i = 0; i < FM; ++i) a[i] = read_frag<BM_, A_KMAJOR>(As, wm * FM + i, ks, lane);
#pragma unroll
        for (int j = 0; j < FN; ++j) b[j] = read_frag<BN_, B_KMAJOR>(Bs, wn * FN + j, ks, lane);
    }
};

// acc[i][j] += A-block i x B-block j; the operands are swapped inside the
// MFMA so that register 4q + r of lane l holds C[m = l % 32][n = 8q + 4 (l / 32) + r].
template <int FM, int FN, typename F>
__device__ __forceinline__ void mfma_block(f32x16 (&acc)[FM][FN], const F& f) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.b[j], f.a[i], acc[i][j], 0, 0, 0);
}

// GELU and its derivative from one exponential: with x = |h| / sqrt(2),
// erf(x) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) exp(-x^2), t = 1 / (1 + p x)
// (Abramowitz & Stegun 7.1.26, |error| < 1.5e-7), Phi(h) = (1 + sign(h) erf(x)) / 2,
// gelu(h) = h Phi(h) and gelu'(h) = Phi(h) + h exp(-h^2 / 2) / sqrt(2 pi).
__device__ __forceinline__ void gelu_pair(float h, float& g, float& dg) {
    const float x = fabsf(h) * 0.70710678118654752f;
    const float t = __builtin_amdgcn_rcpf(1.0f + 0.3275911f * x);
    const float ex = __expf(-x * x);
    const float poly =
        t * (0.254829592f + t * (-0.284496736f + t * (1.421413741f + t * (-1.453152027f +
                                                                           t * 1.061405429f))));
    const float erf_abs = 1.0f - poly * ex;
    const float phi_cdf = 0.5f + 0.5f * copysignf(erf_abs, h);
    g = h * phi_cdf;
    dg = phi_cdf + h * ex * 0.39894228040143268f;
}

// One BM x BN output tile of expert e per block of WGM x WGN waves, each
// (BM/WGM) x (BN/WGN) as 32 x 32 MFMA blocks. Blocks are numbered so that each
// of the 8 XCDs (blocks b = x mod 8) walks a contiguous range of tiles (n
// fastest): neighbouring tiles share operand panels in that XCD's L2.
//
// Pipeline per 64-deep k-stage kt (four 16-deep MFMA steps), one barrier:
//   issue global loads of stage kt+1 (registers)
//   steps 0..2: read fragments of step s+1      | MFMAs of step s
//   store stage kt+1 into the other LDS buffer; barrier
//   read step-0 fragments of stage kt+1         | MFMAs of step 3
// so LDS latency always hides behind a run of MFMAs on held fragments.
//
// Epilogue: each wave turns its accumulators into output values (bias,
// GELU + GELU', or GELU' product), parks them in LDS and writes every output
// row back as full 16-byte-per-lane segments (one output at a time when two
// do not fit in LDS together).
template <int BM_, int BN_, int WGM, int WGN, bool A_KMAJOR, bool B_KMAJOR, int EPI, int DIST>
__global__ __launch_bounds__(64 * WGM * WGN)
__attribute__((amdgpu_waves_per_eu(WGM * WGN == 8 || BM_ * BN_ < 256 * 128 ? 2 : 1,
                                   WGM * WGN == 8 || BM_ * BN_ < 256 * 128 ? 2 : 1)))
void gemm_bf16_kernel(GemmArgs p, int tiles_m, int tiles_n, int per_xcd, int total) {
    constexpr int NT = 64 * WGM * WGN;
    constexpr int AE = stage_elems<BM_, A_KMAJOR>();
    constexpr int BE = stage_elems<BN_, B_KMAJOR>();
    constexpr int WM = BM_ / WGM, WN = BN_ / WGN;  // wave tile
    constexpr int FM = WM / 32, FN = WN / 32;
    constexpr int KSTEPS = BK / 16;
    constexpr int VA = BM_ * 8 / NT, VB = BN_ * 8 / NT;  // staged vectors per thread
    constexpr bool F32_OUT = EPI == EPI_F32;
    constexpr int OUTS = EPI == EPI_FWD1 ? 2 : 1;
    constexpr int SMEM_ELEMS = 2 * (AE + BE);
    // Epilogue staging per wave: IPP of its FM 32-row blocks per pass, all
    // outputs of those rows when they fit, else one output per pass.
    constexpr int EP_LD = F32_OUT ? WN + 4 : WN + 4;
    constexpr int ELEM = F32_OUT ? 4 : 2;
    constexpr int EP_ROWBLK = 32 * EP_LD * ELEM;  // one 32-row block of one output
    constexpr int NW = WGM * WGN;
    constexpr int SMEM_BYTES = SMEM_ELEMS * 2;
    constexpr int EP_OUTS_AT_ONCE = OUTS * FM * EP_ROWBLK * NW <= SMEM_BYTES ? OUTS : 1;
    constexpr int IPP = EP_OUTS_AT_ONCE * FM * EP_ROWBLK * NW <= SMEM_BYTES ? FM
                        : (EP_OUTS_AT_ONCE * (FM / 2) * EP_ROWBLK * NW <= SMEM_BYTES ? FM / 2 : 1);
    constexpr int EP_TILE = IPP * EP_ROWBLK;       // bytes of one output's staged rows
    static_assert(EP_OUTS_AT_ONCE * EP_TILE * NW <= SMEM_BYTES, "epilogue staging exceeds LDS");
    static_assert(!F32_OUT || !A_KMAJOR, "row sums read an mn-major A tile");
    static_assert(NT % BM_ == 0 || !F32_OUT, "row sums give each A row NT / BM threads");
    static_assert(WM % 32 == 0 && WN % 32 == 0 && VA >= 1 && VB >= 1, "tile shape");
    __shared__ __attribute__((aligned(16))) uint16_t smem[SMEM_ELEMS];

    const int b = blockIdx.x;
    const int w = (b & 7) * per_xcd + (b >> 3);
    if (w >= total) return;
    const int tn = w % tiles_n;
    const int tm = (w / tiles_n) % tiles_m;
    const int e = w / (tiles_n * tiles_m);

    const int ne = expert_rows(p.counts, p.G, p.E, e);
    const int M = p.var_k ? p.M : ne;
    const int K = p.var_k ? ne : p.K;
    const int N = p.N;
    const int m0 = tm * BM_, n0 = tn * BN_;
    if (m0 >= M) return;

    const __amdgpu_buffer_rsrc_t ra_rs = make_rsrc(
        static_cast<const uint16_t*>(p.a.base) + e * p.a.estride, p.a.estride * 2);
    const __amdgpu_buffer_rsrc_t rb_rs = make_rsrc(
        static_cast<const uint16_t*>(p.b.base) + e * p.b.estride, p.b.estride * 2);
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    // weight-gradient GEMMs: the first n-tile also sums its A rows (bias grad);
    // thread t adds row t % BM over k slice t / BM of each stage
    const bool row_sum = F32_OUT && p.bsum != nullptr && tn == 0;
    constexpr int RS_SPLIT = F32_OUT ? NT / BM_ : 1;
    constexpr int RS_K = BK / RS_SPLIT;
    float rsum = 0.0f;

    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

    const int nk = (K + BK - 1) / BK;
    uint4 ra0[VA], rb0[VB], ra1[VA], rb1[VB];
    Frags<BM_, BN_, WGM, WGN, A_KMAJOR, B_KMAJOR> f0, f1;

    load_stage<BM_, A_KMAJOR, NT>(ra_rs, p.a.ld, m0, M, 0, K, ra0);
    load_stage<BN_, B_KMAJOR, NT>(rb_rs, p.b.ld, n0, N, 0, K, rb0);
    if constexpr (DIST == 2) {
        load_stage<BM_, A_KMAJOR, NT>(ra_rs, p.a.ld, m0, M, BK, K, ra1);
        load_stage<BN_, B_KMAJOR, NT>(rb_rs, p.b.ld, n0, N, BK, K, rb1);
    }
    store_stage<BM_, A_KMAJOR, NT>(smem, ra0);
    store_stage<BN_, B_KMAJOR, NT>(smem + AE, rb0);
    __syncthreads();
    f0.read(smem, smem + AE, wm, wn, 0, lane);

    // One k-stage. With DIST = 2 the register set PAR receives stage kt + 2
    // while the other set (stage kt + 1, loaded a stage earlier) goes to LDS.
    auto stage = [&](const int kt, auto par) {
        constexpr int PAR = decltype(par)::value;
        uint4(&la)[VA] = (DIST == 1 || PAR == 0) ? ra0 : ra1;
        uint4(&lb)[VB] = (DIST == 1 || PAR == 0) ? rb0 : rb1;
        uint4(&sa)[VA] = (DIST == 1 || PAR == 1) ? ra0 : ra1;
        uint4(&sb)[VB] = (DIST == 1 || PAR == 1) ? rb0 : rb1;
        uint16_t* As = smem + (kt & 1) * (AE + BE);
        uint16_t* An = smem + ((kt + 1) & 1) * (AE + BE);
        load_stage<BM_, A_KMAJOR, NT>(ra_rs, p.a.ld, m0, M, (kt + DIST) * BK, K, la);
        load_stage<BN_, B_KMAJOR, NT>(rb_rs, p.b.ld, n0, N, (kt + DIST) * BK, K, lb);
        if constexpr (F32_OUT) {
            if (row_sum) {
                const uint16_t* col = As + (tid / BM_) * RS_K * (BM_ + MNPAD) + tid % BM_;
#pragma unroll 8
                for (int kk = 0; kk < RS_K; ++kk) rsum += bf16_to_f32(col[kk * (BM_ + MNPAD)]);
            }
        }
#pragma unroll
        for (int s = 0; s < KSTEPS - 1; ++s) {
            if (s % 2 == 0) {
                f1.read(As, As + AE, wm, wn, s + 1, lane);
                __builtin_amdgcn_sched_barrier(0);
                mfma_block(acc, f0);
            } else {
                f0.read(As, As + AE, wm, wn, s + 1, lane);
                __builtin_amdgcn_sched_barrier(0);
                mfma_block(acc, f1);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        store_stage<BM_, A_KMAJOR, NT>(An, sa);
        store_stage<BN_, B_KMAJOR, NT>(An + AE, sb);
        __syncthreads();
        // KSTEPS is even: the last step's fragments are in f1
        f0.read(An, An + AE, wm, wn, 0, lane);
        __builtin_amdgcn_sched_barrier(0);
        mfma_block(acc, f1);
        __builtin_amdgcn_sched_barrier(0);
    };
    // Whole pairs first, without a conditional half: a skipped half would merge
    // a path with loads still in flight into the loop head, and the compiler
    // would then drain every outstanding load before the next set is issued.
    int kt = 0;
    for (; kt + 1 < nk; kt += 2) {
        stage(kt, std::integral_constant<int, 0>{});
        stage(kt + 1, std::integral_constant<int, 1>{});
    }
    if (kt < nk) stage(kt, std::integral_constant<int, 0>{});
    __syncthreads();  // every wave is done with the operand stages

    if constexpr (F32_OUT) {
        if (row_sum) {  // uniform per block
            float* part = reinterpret_cast<float*>(smem);
            part[tid] = rsum;
            __syncthreads();
            if (tid < BM_ && m0 + tid < M) {
                float t = part[tid];
#pragma unroll
                for (int q = 1; q < RS_SPLIT; ++q) t += part[tid + q * BM_];
                p.bsum[static_cast<size_t>(e) * M + m0 + tid] = t;
            }
            __syncthreads();
        }
    }

    char* ep = reinterpret_cast<char*>(smem) + wave * EP_OUTS_AT_ONCE * EP_TILE;
    constexpr int SEG = 16 / ELEM;                 // elements per 16-byte segment
    constexpr int LANES_PER_ROW = WN / SEG;
    constexpr int ROWS_PER_PASS = 64 / LANES_PER_ROW;
    static_assert(LANES_PER_ROW <= 64 && 64 % LANES_PER_ROW == 0, "epilogue row split");

#pragma unroll
    for (int i0 = 0; i0 < FM; i0 += IPP)
#pragma unroll
    for (int o0 = 0; o0 < OUTS; o0 += EP_OUTS_AT_ONCE) {
        // Stage 1: values into this wave's LDS tiles. Register 4q + r of lane l
        // holds C[m][n + r] with m = 32 i + l % 32, n = 32 j + 8 q + 4 (l / 32)
        // inside the wave tile.
#pragma unroll
        for (int ii = 0; ii < IPP; ++ii)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int i = i0 + ii;
                    const int ml = ii * 32 + (lane & 31);  // row inside the staged rows
                    const int nl = j * 32 + 8 * q + 4 * (lane >> 5);
                    const f32x16& v = acc[i][j];
                    float r[4] = {v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
                    if constexpr (F32_OUT) {
                        *reinterpret_cast<float4*>(reinterpret_cast<float*>(ep) + ml * EP_LD +
                                                   nl) = make_float4(r[0], r[1], r[2], r[3]);
                    } else {
                        const int n = n0 + wn * WN + nl;
                        const int m = m0 + wm * WM + i * 32 + (lane & 31);
                        if constexpr (EPI == EPI_FWD1 || EPI == EPI_BIAS) {
                            if (n < N) {
                                const uint2 bb = *reinterpret_cast<const uint2*>(
                                    static_cast<const uint16_t*>(p.bias) + e * p.bias_estride + n);
                                r[0] += bf16_to_f32(bb.x & 0xFFFFu);
                                r[1] += bf16_to_f32(bb.x >> 16);
                                r[2] += bf16_to_f32(bb.y & 0xFFFFu);
                                r[3] += bf16_to_f32(bb.y >> 16);
                            }
                        }
                        if constexpr (EPI == EPI_GELU_GRAD) {
                            if (n < N && m < M) {
                                const uint2 gg = *reinterpret_cast<const uint2*>(
                                    static_cast<const uint16_t*>(p.aux) + e * p.out_estride +
                                    static_cast<size_t>(m) * p.ldo + n);
                                r[0] *= bf16_to_f32(gg.x & 0xFFFFu);
                                r[1] *= bf16_to_f32(gg.x >> 16);
                                r[2] *= bf16_to_f32(gg.y & 0xFFFFu);
                                r[3] *= bf16_to_f32(gg.y >> 16);
                            }
                        }
                        uint16_t* t0 = reinterpret_cast<uint16_t*>(ep) + ml * EP_LD + nl;
                        if constexpr (EPI == EPI_FWD1) {
                            float g[4], dg[4];
#pragma unroll
                            for (int c = 0; c < 4; ++c) gelu_pair(r[c], g[c], dg[c]);
#pragma unroll
                            for (int o = 0; o < EP_OUTS_AT_ONCE; ++o) {
                                const float* src = (o0 + o == 0) ? g : dg;
                                *reinterpret_cast<uint2*>(t0 + o * (EP_TILE / 2)) =
                                    make_uint2(pack_bf16x2(src[0], src[1]),
                                               pack_bf16x2(src[2], src[3]));
                            }
                        } else {
                            *reinterpret_cast<uint2*>(t0) =
                                make_uint2(pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3]));
                        }
                    }
                }
        __syncthreads();

        // Stage 2: staged rows out in 16-byte segments.
        const int cl = (lane % LANES_PER_ROW) * SEG;
        const int n = n0 + wn * WN + cl;
#pragma unroll
        for (int o = 0; o < EP_OUTS_AT_ONCE; ++o) {
            char* dst_base = static_cast<char*>(o0 + o == 0 ? p.out : p.out2);
#pragma unroll
            for (int pass = 0; pass < IPP * 32 / ROWS_PER_PASS; ++pass) {
                const int ml = pass * ROWS_PER_PASS + lane / LANES_PER_ROW;
                const int m = m0 + wm * WM + i0 * 32 + ml;
                const uint4 v =
                    *reinterpret_cast<const uint4*>(ep + o * EP_TILE + (ml * EP_LD + cl) * ELEM);
                if (m < M && n < N)
                    *reinterpret_cast<uint4*>(
                        dst_base + (e * p.out_estride + static_cast<size_t>(m) * p.ldo + n) * ELEM) =
                        v;
            }
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------ f32 FMA path

constexpr int FT = 64, FK = 16;

template <bool KMAJOR>
__device__ __forceinline__ float f32_elem(const float* base, int ld, int mn, int k) {
    return KMAJOR ? base[static_cast<size_t>(mn) * ld + k] : base[static_cast<size_t>(k) * ld + mn];
}

template <bool A_KMAJOR, bool B_KMAJOR, int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs p) {
    __shared__ float As[FK][FT + 1];
    __shared__ float Bs[FK][FT + 1];
    const int e = blockIdx.z;
    const int ne = expert_rows(p.counts, p.G, p.E, e);
    const int M = p.var_k ? p.M : ne;
    const int K = p.var_k ? ne : p.K;
    const int N = p.N;
    const int m0 = blockIdx.y * FT, n0 = blockIdx.x * FT;
    if (m0 >= M) return;
    const float* A = static_cast<const float*>(p.a.base) + e * p.a.estride;
    const float* B = static_cast<const float*>(p.b.base) + e * p.b.estride;
    const int tm = (threadIdx.x >> 4) * 4, tn = (threadIdx.x & 15) * 4;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += FK) {
        for (int q = threadIdx.x; q < FK * FT; q += 256) {
            const int kk = q / FT, mn = q % FT;
            As[kk][mn] = (m0 + mn < M && k0 + kk < K)
                             ? f32_elem<A_KMAJOR>(A, p.a.ld, m0 + mn, k0 + kk) : 0.0f;
            Bs[kk][mn] = (n0 + mn < N && k0 + kk < K)
                             ? f32_elem<B_KMAJOR>(B, p.b.ld, n0 + mn, k0 + kk) : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < FK; ++kk)
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_fmaf(As[kk][tm + i], Bs[kk][tn + j], acc[i][j]);
        __syncthreads();
    }
    for (int i = 0; i < 4; ++i) {
        const int m = m0 + tm + i;
        if (m >= M) continue;
        for (int j = 0; j < 4; ++j) {
            const int n = n0 + tn + j;
            if (n >= N) continue;
            const size_t o = e * p.out_estride + static_cast<size_t>(m) * p.ldo + n;
            float v = acc[i][j];
            float* out = static_cast<float*>(p.out);
            if (EPI == EPI_FWD1 || EPI == EPI_BIAS)
                v += static_cast<const float*>(p.bias)[e * p.bias_estride + n];
            if (EPI == EPI_GELU_GRAD) v *= static_cast<const float*>(p.aux)[o];
            if (EPI == EPI_FWD1) {
                out[o] = gelu_f(v);
                static_cast<float*>(p.out2)[o] = gelu_grad_f(v);
            } else {
                out[o] = v;
            }
        }
    }
}

// ------------------------------------------------------------------ bias gradients

// out[e, c] = sum over the n_e rows of src[e, r, c]; 64 columns x 4 row phases
// per block, phases added in a fixed order.
template <typename T>
__global__ __launch_bounds__(256) void colsum_kernel(const T* __restrict__ src,
                                                     long long estride, int cols,
                                                     const int32_t* __restrict__ counts, int G,
                                                     int E, float* __restrict__ out) {
    __shared__ float part[4][64];
    const int e = blockIdx.y;
    const int c = blockIdx.x * 64 + (threadIdx.x & 63);
    const int ph = threadIdx.x >> 6;
    const int ne = expert_rows(counts, G, E, e);
    float s = 0.0f;
    if (c < cols) {
        const T* p = src + e * estride + c;
        for (int r = ph; r < ne; r += 4) s += Elem<T>::load(p, static_cast<size_t>(r) * cols);
    }
    part[ph][threadIdx.x & 63] = s;
    __syncthreads();
    if (ph == 0 && c < cols)
        out[static_cast<size_t>(e) * cols + c] = ((part[0][c & 63] + part[1][c & 63]) +
                                                  part[2][c & 63]) + part[3][c & 63];
}

template <int BM_, int BN_, int WGM, int WGN, bool AK, bool BK_, int EPI, int DIST = 1>
void launch_bf16(const Dims& D, const GemmArgs& a, int grid_m_rows, hipStream_t st) {
    const int tiles_m = static_cast<int>(cdiv(grid_m_rows, BM_));
    const int tiles_n = static_cast<int>(cdiv(a.N, BN_));
    const int total = D.E * tiles_m * tiles_n;
    const int per_xcd = static_cast<int>(cdiv(total, 8));
    gemm_bf16_kernel<BM_, BN_, WGM, WGN, AK, BK_, EPI, DIST><<<8 * per_xcd, 64 * WGM * WGN, 0,
                                                               st>>>(a, tiles_m, tiles_n, per_xcd,
                                                                     total);
}

template <bool AK, bool BK_, int EPI>
void launch_gemm(const Dims& D, const GemmArgs& a, int grid_m_rows, hipStream_t st) {
    if (D.dtype == VMOE_BF16) {
        // 128 x 128 tiles (4 waves, two blocks per CU) for the short-k GEMMs and
        // the weight gradients; 256 x 256 tiles of 8 waves (half the LDS traffic
        // per flop) for the long-k GEMMs with one plain bf16 output (the
        // down-projection and dxe)
        if constexpr (EPI == EPI_BIAS || EPI == EPI_STORE)
            launch_bf16<256, 256, 2, 4, AK, BK_, EPI>(D, a, grid_m_rows, st);
        else
            launch_bf16<128, 128, 2, 2, AK, BK_, EPI>(D, a, grid_m_rows, st);
    } else {
        dim3 grid(cdiv(a.N, FT), cdiv(grid_m_rows, FT), D.E);
        gemm_f32_kernel<AK, BK_, EPI><<<grid, 256, 0, st>>>(a);
    }
}

GemmArgs base_args(const Dims& D, const int32_t* counts) {
    GemmArgs a{};
    a.counts = counts;
    a.G = D.G;
    a.E = D.E;
    return a;
}

size_t esize(const Dims& D) { return D.dtype == VMOE_BF16 ? 2 : 4; }

}  // namespace

vmoe_status ffn_fwd_launch(const Dims& D, const void* xe, const int32_t* counts, const void* w1,
                           const void* b1, const void* w2, const void* b2, void* act,
                           void* act_grad, void* ye, hipStream_t st) {
    const long long rows = D.rows_per_expert();
    if (rows == 0 || D.E == 0) return VMOE_OK;
    // H = xe W1^T + b1 (never stored), A = gelu(H), A' = gelu'(H)
    GemmArgs g1 = base_args(D, counts);
    g1.a = Operand{xe, rows * D.d, D.d};
    g1.b = Operand{w1, static_cast<long long>(D.f) * D.d, D.d};
    g1.M = static_cast<int>(rows);
    g1.N = D.f;
    g1.K = D.d;
    g1.out = act;
    g1.out2 = act_grad;
    g1.out_estride = rows * D.f;
    g1.ldo = D.f;
    g1.bias = b1;
    g1.bias_estride = D.f;
    launch_gemm<true, true, EPI_FWD1>(D, g1, static_cast<int>(rows), st);
    // ye = A W2^T + b2
    GemmArgs g2 = base_args(D, counts);
    g2.a = Operand{act, rows * D.f, D.f};
    g2.b = Operand{w2, static_cast<long long>(D.d) * D.f, D.f};
    g2.M = static_cast<int>(rows);
    g2.N = D.d;
    g2.K = D.f;
    g2.out = ye;
    g2.out_estride = rows * D.d;
    g2.ldo = D.d;
    g2.bias = b2;
    g2.bias_estride = D.d;
    launch_gemm<true, true, EPI_BIAS>(D, g2, static_cast<int>(rows), st);
    return launch_status();
}

vmoe_status ffn_bwd_launch(const Dims& D, const void* xe, const int32_t* counts, const void* w1,
                           const void* w2, const void* act, const void* act_grad, const void* dye,
                           void* dh, void* dxe, float* dw1, float* db1, float* dw2, float* db2,
                           hipStream_t st) {
    const long long rows = D.rows_per_expert();
    if (D.E == 0) return VMOE_OK;
    if (rows > 0) {
        // dH = (dye W2) * A': W2 [d, f] read with k = d strided (mn-major)
        GemmArgs g = base_args(D, counts);
        g.a = Operand{dye, rows * D.d, D.d};
        g.b = Operand{w2, static_cast<long long>(D.d) * D.f, D.f};
        g.M = static_cast<int>(rows);
        g.N = D.f;
        g.K = D.d;
        g.out = dh;
        g.out_estride = rows * D.f;
        g.ldo = D.f;
        g.aux = act_grad;
        launch_gemm<true, false, EPI_GELU_GRAD>(D, g, static_cast<int>(rows), st);
        // dxe = dH W1: W1 [f, d] read with k = f strided
        GemmArgs x = base_args(D, counts);
        x.a = Operand{dh, rows * D.f, D.f};
        x.b = Operand{w1, static_cast<long long>(D.f) * D.d, D.d};
        x.M = static_cast<int>(rows);
        x.N = D.d;
        x.K = D.f;
        x.out = dxe;
        x.out_estride = rows * D.d;
        x.ldo = D.d;
        launch_gemm<true, false, EPI_STORE>(D, x, static_cast<int>(rows), st);
    }
    // dW2 [d, f] = dye^T A, reduced over the n_e rows (k = row, strided)
    GemmArgs w = base_args(D, counts);
    w.var_k = 1;
    w.a = Operand{dye, rows * D.d, D.d};
    w.b = Operand{act, rows * D.f, D.f};
    w.M = D.d;
    w.N = D.f;
    w.K = 0;
    w.out = dw2;
    w.out_estride = static_cast<long long>(D.d) * D.f;
    w.ldo = D.f;
    w.bsum = D.dtype == VMOE_BF16 ? db2 : nullptr;  // db2 = row sums of dye^T
    launch_gemm<false, false, EPI_F32>(D, w, D.d, st);
    // dW1 [f, d] = dH^T xe
    GemmArgs v = base_args(D, counts);
    v.var_k = 1;
    v.a = Operand{dh, rows * D.f, D.f};
    v.b = Operand{xe, rows * D.d, D.d};
    v.M = D.f;
    v.N = D.d;
    v.K = 0;
    v.out = dw1;
    v.out_estride = static_cast<long long>(D.f) * D.d;
    v.ldo = D.d;
    v.bsum = D.dtype == VMOE_BF16 ? db1 : nullptr;  // db1 = row sums of dH^T
    launch_gemm<false, false, EPI_F32>(D, v, D.f, st);
    // bias gradients (the bf16 path sums them inside the dW GEMMs)
    if (D.dtype == VMOE_F32) {
        colsum_kernel<float><<<dim3(cdiv(D.d, 64), D.E), 256, 0, st>>>(
            static_cast<const float*>(dye), rows * D.d, D.d, counts, D.G, D.E, db2);
        colsum_kernel<float><<<dim3(cdiv(D.f, 64), D.E), 256, 0, st>>>(
            static_cast<const float*>(dh), rows * D.f, D.f, counts, D.G, D.E, db1);
    }
    return launch_status();
}

}  // namespace vmoe
