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
#include "common.h"

namespace vmoe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

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
    void* out;              // primary output
    void* out2;             // EPI_FWD1: activation
    long long out_estride;
    int ldo;
    const void* bias;       // EPI_FWD1 / EPI_BIAS
    long long bias_estride;
    const void* aux;        // EPI_GELU_GRAD: saved pre-activation H
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
constexpr int MNPAD = 16;       // mn-major rows: ROWS + 16 bf16 (conflict-free transpose reads)

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

// LDS elements of one operand stage: k-major [ROWS][BK + KPAD], mn-major [BK][ROWS + MNPAD].
template <int ROWS, bool KMAJOR>
__host__ __device__ constexpr int stage_elems() {
    return KMAJOR ? ROWS * (BK + KPAD) : BK * (ROWS + MNPAD);
}

// A masked-off vector is still loaded, from the (always valid) operand base,
// and replaced by zeros in registers: no address ever points off the operand.
__device__ __forceinline__ uint4 masked_load(const uint16_t* __restrict__ base, size_t off,
                                             bool ok) {
    const uint4 v = *reinterpret_cast<const uint4*>(base + (ok ? off : 0));
    return ok ? v : make_uint4(0, 0, 0, 0);
}

// Global -> registers: one ROWS x BK operand stage, ROWS / 32 vectors of 8
// bf16 per thread, each row segment read by consecutive lanes (coalesced).
template <int ROWS, bool KMAJOR>
__device__ __forceinline__ void load_stage(const uint16_t* __restrict__ base, int ld, int mn0,
                                           int mn_lim, int k0, int k_lim,
                                           uint4 (&r)[ROWS / 32]) {
    const int tid = threadIdx.x;
    if (KMAJOR) {
        const int kc = (tid & 7) * 8;
#pragma unroll
        for (int j = 0; j < ROWS / 32; ++j) {
            const int mn = (tid >> 3) + 32 * j;
            r[j] = masked_load(base, static_cast<size_t>(mn0 + mn) * ld + k0 + kc,
                               (mn0 + mn < mn_lim) && (k0 + kc < k_lim));
        }
    } else {
        constexpr int VPR = ROWS / 8;  // vectors per k row
        const int mc = (tid % VPR) * 8;
#pragma unroll
        for (int j = 0; j < ROWS / 32; ++j) {
            const int kr = tid / VPR + (256 / VPR) * j;
            r[j] = masked_load(base, static_cast<size_t>(k0 + kr) * ld + mn0 + mc,
                               (k0 + kr < k_lim) && (mn0 + mc < mn_lim));
        }
    }
}

// Registers -> LDS, same element placement as the global tile (no transpose).
template <int ROWS, bool KMAJOR>
__device__ __forceinline__ void store_stage(uint16_t* s, const uint4 (&r)[ROWS / 32]) {
    const int tid = threadIdx.x;
    if (KMAJOR) {
        const int kc = (tid & 7) * 8;
#pragma unroll
        for (int j = 0; j < ROWS / 32; ++j)
            *reinterpret_cast<uint4*>(s + ((tid >> 3) + 32 * j) * (BK + KPAD) + kc) = r[j];
    } else {
        constexpr int VPR = ROWS / 8;
        const int mc = (tid % VPR) * 8;
#pragma unroll
        for (int j = 0; j < ROWS / 32; ++j)
            *reinterpret_cast<uint4*>(s + (tid / VPR + (256 / VPR) * j) * (ROWS + MNPAD) + mc) =
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

// MFMA operand fragment for 16 mn values (lane & 15) x 8 k values
// (k = kstep * 32 + 8 * (lane >> 4) + 0..7).
template <int ROWS, bool KMAJOR>
__device__ __forceinline__ bf16x8 read_frag(const uint16_t* s, int blk, int kstep, int lane) {
    if (KMAJOR) {
        return *reinterpret_cast<const bf16x8*>(s + (blk * 16 + (lane & 15)) * (BK + KPAD) +
                                                kstep * 32 + (lane >> 4) * 8);
    } else {
        constexpr int P = ROWS + MNPAD;
        const int j = lane & 15;
        const uint16_t* p0 = s + (kstep * 32 + 8 * (lane >> 4) + (j >> 2)) * P + blk * 16 +
                             4 * (j & 3);
        const s16x4 lo = lds_read_tr(p0);
        const s16x4 hi = lds_read_tr(p0 + 4 * P);
        const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        return __builtin_bit_cast(bf16x8, v);
    }
}

// One BM x BN output tile of expert e per 256-thread block; four waves in
// 2 x 2, each (BM/2) x (BN/2) as 16 x 16 MFMA blocks. Blocks are numbered so
// that each of the 8 XCDs (blocks b = x mod 8) walks a contiguous range of
// tiles (n fastest): neighbouring tiles share operand panels in that XCD's L2.
template <int BM_, int BN_, bool A_KMAJOR, bool B_KMAJOR, int EPI>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gemm_bf16_kernel(GemmArgs p, int tiles_m, int tiles_n, int per_xcd, int total) {
    constexpr int AE = stage_elems<BM_, A_KMAJOR>();
    constexpr int BE = stage_elems<BN_, B_KMAJOR>();
    constexpr int FM = BM_ / 32, FN = BN_ / 32;  // 16 x 16 blocks per wave
    static_assert(EPI != EPI_F32 || (BM_ == 256 && !A_KMAJOR), "row sums assume 256 mn-major rows");
    __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (AE + BE)];

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

    const uint16_t* A = static_cast<const uint16_t*>(p.a.base) + e * p.a.estride;
    const uint16_t* B = static_cast<const uint16_t*>(p.b.base) + e * p.b.estride;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    // weight-gradient GEMMs: the first n-tile also sums its A rows (bias grad)
    const bool row_sum = EPI == EPI_F32 && p.bsum != nullptr && tn == 0;
    float rsum = 0.0f;

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk = (K + BK - 1) / BK;
    uint4 ra[BM_ / 32], rb[BN_ / 32];
    load_stage<BM_, A_KMAJOR>(A, p.a.ld, m0, M, 0, K, ra);
    load_stage<BN_, B_KMAJOR>(B, p.b.ld, n0, N, 0, K, rb);
    store_stage<BM_, A_KMAJOR>(smem, ra);
    store_stage<BN_, B_KMAJOR>(smem + AE, rb);
    __syncthreads();

    for (int kt = 0; kt < nk; ++kt) {
        uint16_t* As = smem + (kt & 1) * (AE + BE);
        uint16_t* Bs = As + AE;
        const bool more = kt + 1 < nk;
        if (more) {
            load_stage<BM_, A_KMAJOR>(A, p.a.ld, m0, M, (kt + 1) * BK, K, ra);
            load_stage<BN_, B_KMAJOR>(B, p.b.ld, n0, N, (kt + 1) * BK, K, rb);
        }
        if (!A_KMAJOR && row_sum) {
            // thread t owns A row m0 + t (BM_ == 256): add its 64 k values
#pragma unroll 8
            for (int kk = 0; kk < BK; ++kk)
                rsum += bf16_to_f32(As[kk * (BM_ + MNPAD) + threadIdx.x]);
        }
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            bf16x8 af[FM], bfr[FN];
#pragma unroll
            for (int i = 0; i < FM; ++i) af[i] = read_frag<BM_, A_KMAJOR>(As, wm * FM + i, ks, lane);
#pragma unroll
            for (int j = 0; j < FN; ++j) bfr[j] = read_frag<BN_, B_KMAJOR>(Bs, wn * FN + j, ks, lane);
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[j], af[i], acc[i][j],
                                                                        0, 0, 0);
        }
        if (more) {
            uint16_t* An = smem + ((kt + 1) & 1) * (AE + BE);
            store_stage<BM_, A_KMAJOR>(An, ra);
            store_stage<BN_, B_KMAJOR>(An + AE, rb);
        }
        __syncthreads();
    }
    if (row_sum && m0 + static_cast<int>(threadIdx.x) < M)
        p.bsum[static_cast<size_t>(e) * M + m0 + threadIdx.x] = rsum;

    // Epilogue: lane holds C[m][n .. n+3].
#pragma unroll
    for (int i = 0; i < FM; ++i) {
        const int m = m0 + (wm * FM + i) * 16 + (lane & 15);
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
            const int n = n0 + (wn * FN + j) * 16 + (lane >> 4) * 4;
            if (n >= N) continue;
            const f32x4 v = acc[i][j];
            const size_t o = e * p.out_estride + static_cast<size_t>(m) * p.ldo + n;
            if (EPI == EPI_F32) {
                *reinterpret_cast<float4*>(static_cast<float*>(p.out) + o) =
                    make_float4(v[0], v[1], v[2], v[3]);
            } else {
                float r[4] = {v[0], v[1], v[2], v[3]};
                if (EPI == EPI_FWD1 || EPI == EPI_BIAS) {
                    const uint2 bb = *reinterpret_cast<const uint2*>(
                        static_cast<const uint16_t*>(p.bias) + e * p.bias_estride + n);
                    r[0] += bf16_to_f32(bb.x & 0xFFFFu);
                    r[1] += bf16_to_f32(bb.x >> 16);
                    r[2] += bf16_to_f32(bb.y & 0xFFFFu);
                    r[3] += bf16_to_f32(bb.y >> 16);
                }
                if (EPI == EPI_GELU_GRAD) {
                    const uint2 hh =
                        *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(p.aux) + o);
                    r[0] *= gelu_grad_f(bf16_to_f32(hh.x & 0xFFFFu));
                    r[1] *= gelu_grad_f(bf16_to_f32(hh.x >> 16));
                    r[2] *= gelu_grad_f(bf16_to_f32(hh.y & 0xFFFFu));
                    r[3] *= gelu_grad_f(bf16_to_f32(hh.y >> 16));
                }
                uint2 w2;
                w2.x = pack_bf16x2(r[0], r[1]);
                w2.y = pack_bf16x2(r[2], r[3]);
                *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.out) + o) = w2;
                if (EPI == EPI_FWD1) {
                    uint2 a;
                    a.x = pack_bf16x2(gelu_f(r[0]), gelu_f(r[1]));
                    a.y = pack_bf16x2(gelu_f(r[2]), gelu_f(r[3]));
                    *reinterpret_cast<uint2*>(static_cast<uint16_t*>(p.out2) + o) = a;
                }
            }
        }
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
            if (EPI == EPI_GELU_GRAD) v *= gelu_grad_f(static_cast<const float*>(p.aux)[o]);
            out[o] = v;
            if (EPI == EPI_FWD1) static_cast<float*>(p.out2)[o] = gelu_f(v);
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

template <int BM_, int BN_, bool AK, bool BK_, int EPI>
void launch_bf16(const Dims& D, const GemmArgs& a, int grid_m_rows, hipStream_t st) {
    const int tiles_m = static_cast<int>(cdiv(grid_m_rows, BM_));
    const int tiles_n = static_cast<int>(cdiv(a.N, BN_));
    const int total = D.E * tiles_m * tiles_n;
    const int per_xcd = static_cast<int>(cdiv(total, 8));
    gemm_bf16_kernel<BM_, BN_, AK, BK_, EPI><<<8 * per_xcd, 256, 0, st>>>(a, tiles_m, tiles_n,
                                                                         per_xcd, total);
}

template <bool AK, bool BK_, int EPI>
void launch_gemm(const Dims& D, const GemmArgs& a, int grid_m_rows, hipStream_t st) {
    if (D.dtype == VMOE_BF16) {
        if constexpr (EPI == EPI_F32) {
            launch_bf16<256, 128, AK, BK_, EPI>(D, a, grid_m_rows, st);
        } else {
            if (a.N >= 2048)
                launch_bf16<256, 256, AK, BK_, EPI>(D, a, grid_m_rows, st);
            else
                launch_bf16<256, 128, AK, BK_, EPI>(D, a, grid_m_rows, st);
        }
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
                           const void* b1, const void* w2, const void* b2, void* h, void* act,
                           void* ye, hipStream_t st) {
    const long long rows = D.rows_per_expert();
    if (rows == 0 || D.E == 0) return VMOE_OK;
    // H = xe W1^T + b1, A = gelu(H)
    GemmArgs g1 = base_args(D, counts);
    g1.a = Operand{xe, rows * D.d, D.d};
    g1.b = Operand{w1, static_cast<long long>(D.f) * D.d, D.d};
    g1.M = static_cast<int>(rows);
    g1.N = D.f;
    g1.K = D.d;
    g1.out = h;
    g1.out2 = act;
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
                           const void* w2, const void* h, const void* act, const void* dye,
                           void* dh, void* dxe, float* dw1, float* db1, float* dw2, float* db2,
                           hipStream_t st) {
    const long long rows = D.rows_per_expert();
    if (D.E == 0) return VMOE_OK;
    if (rows > 0) {
        // dH = (dye W2) * gelu'(H): W2 [d, f] read with k = d strided (mn-major)
        GemmArgs g = base_args(D, counts);
        g.a = Operand{dye, rows * D.d, D.d};
        g.b = Operand{w2, static_cast<long long>(D.d) * D.f, D.f};
        g.M = static_cast<int>(rows);
        g.N = D.f;
        g.K = D.d;
        g.out = dh;
        g.out_estride = rows * D.f;
        g.ldo = D.f;
        g.aux = h;
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
