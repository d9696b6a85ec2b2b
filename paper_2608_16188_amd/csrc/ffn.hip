// Expert MLP forward and backward as grouped GEMMs on gfx950.
//
// bf16 path: one templated matrix-core kernel, C[M x N] = sum_k A(m,k) B(n,k),
// one output tile of one expert per block. Tiles (Tile<>) are 256 x 256 or
// 256 x 192 with eight waves (one block per CU) or 128 x 128 with four waves
// (two blocks per CU); each wave accumulates its sub-tile with
// v_mfma_f32_32x32x16_bf16 in f32. Operands reach LDS through buffer loads
// that write LDS directly (16 bytes per lane, out-of-range offsets read as
// zero, so ragged tails need no branch) into a ring of 2-4 stages; the next
// stages' loads stay in flight across the barrier (partial vmcnt waits).
// An operand whose k index is contiguous in HBM is stored k-major with an
// XOR chunk swizzle; one whose k index is strided (weights read transposed
// in the backward, the token-reduced weight-gradient GEMMs) is copied
// unchanged, mn-major, and its fragments are read with ds_read_b64_tr_b16.
// The operand roles are swapped inside the MFMA so each lane holds runs of
// consecutive output columns of one row; the fused epilogues (bias, GELU and
// GELU' pair, GELU' product, bf16 rounding, f32 weight gradients with the
// bias-gradient row sums) park the tile in LDS and store 16-byte row
// segments.
//
// Each expert's row count n_e = sum_g counts[g, e] is read on the device:
// tiles past n_e exit at once (M = n_e GEMMs) or n_e bounds the k loop
// (weight-gradient GEMMs, which still write zeros for an empty expert).
// Blocks are mapped so that each XCD works on a contiguous run of tiles,
// grouped group_m m-tiles at a time, which keeps operand panels in that
// XCD's L2. The tile shape is chosen per launch by a cost model: rounds of
// 256 CUs times the tile area, scaled by a per-shape efficiency.
//
// f32 path: 64 x 64 tiles on the f32 matrix cores (v_mfma_f32_32x32x2f32, one
// 32 x 32 block per wave) with coalesced operand staging through LDS and the
// same operand and epilogue description (the accuracy path).
#include <mutex>
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
    // Gathered operand (kernels built with GATHER != 0): the operand's rows
    // are token rows of x, row r of expert e being x[tok[e * tok_estride + r]];
    // its base is x itself (estride 0) and gather_bytes the size of x.
    const int32_t* tok;     // null: this problem's operand is not gathered
    long long tok_estride;
    long long gather_bytes;
};


// Up to two independent GEMMs of one kernel instantiation in one launch (the
// two weight gradients): blocks [0, total[0]) work on problem 0, the rest on
// problem 1, so the second fills the first's last, partial round of tiles.
struct GemmBatch {
    GemmArgs p[2];
    int tiles_m[2], tiles_n[2], total[2];
    int group_m, chunk, per_xcd;
};

// A GEMM whose m is the expert's rows (every epilogue but the weight
// gradients', whose k is the rows) runs one problem per launch and numbers its
// tiles over the experts' live m-tiles only (ceil(n_e / BM) each, from the
// device row counts): the blocks past the last live tile all sit at the end
// of the grid instead of between the live tiles of consecutive experts, where
// each would hold a CU slot while the dispatcher places blocks in order.
template <int EPI>
constexpr bool compact_tiles() { return EPI != EPI_F32; }

__device__ __forceinline__ int expert_rows(const int32_t* counts, int G, int E, int e) {
    int n = 0;
    for (int g = 0; g < G; ++g) n += counts[g * E + e];
    return n;
}

// m-tiles of an expert with ne rows: ceil(ne / bm), except that an expert
// whose rows fit one 32-row block (a light expert) gets `lsplit` tiles per
// n-tile, each taking a share of the tile's columns (its weight stream then
// runs on lsplit CUs). lsplit = 1 leaves every expert at ceil(ne / bm).
__device__ __forceinline__ int expert_mtiles(int ne, int bm, int lsplit) {
    return lsplit > 1 && ne > 0 && ne <= 32 ? lsplit : (ne + bm - 1) / bm;
}

// Live tile w of a compact problem: lane e of every wave sums expert e's rows
// (at most `cap`, the rows of its buffer) and its tile count, an inclusive
// scan over the lanes places the experts' tile ranges end to end, and the
// expert holding w is the number of ranges that end at or before it. Returns
// false past the last live tile. Uniform per wave (every wave of a block
// computes the same).
struct LiveTile {
    int e, r, ne;  // expert, tile index inside the expert, expert's rows
};
__device__ __forceinline__ bool live_tile(const int32_t* counts, int G, int E, int cap, int bm,
                                          int lsplit, int tiles_n, int w, LiveTile* out) {
    const int lane = threadIdx.x & 63;
    int ne = 0;
    if (lane < E) {
#pragma unroll 4
        for (int g = 0; g < G; ++g) ne += counts[g * E + lane];
        ne = min(ne, cap);  // never past the expert's rows, whatever the counts say
    }
    const int t = expert_mtiles(ne, bm, lsplit) * tiles_n;
    int incl = t;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int u = __shfl_up(incl, o, 64);
        if (lane >= o) incl += u;
    }
    if (w >= __shfl(incl, 63, 64)) return false;
    const int e = __popcll(__ballot(incl <= w));
    out->e = e;
    out->r = w - __shfl(incl - t, e, 64);
    out->ne = __shfl(ne, e, 64);
    return true;
}

// Row GEMMs whose outputs are d wide, under a skewed load. The launch order
// is cut into chunks of `chunk` tiles; a chunk runs on one XCD (chunks are
// dealt to the XCDs in turn) and its tiles share operand panels in that
// XCD's L2. With lsplit = 1 (light tiles as long as a heavy one's weight
// stream) the chunks of heavy experts' live tiles (at least half a tile of
// rows) are spread evenly over the first 70% of the chunk positions and those
// of light experts fill the rest, so that light tiles do not run alone at the
// end. Inside each class experts go in order; with no light expert it is the
// plain live-tile order. Measured at the ViT-L/16 skew (four full experts, 28
// of ~17 rows): the spread took the down-projection 216 -> 178 us and dxe
// 204 -> 161 us against expert order (few n-tiles, long k); it slowed the
// f-wide row GEMMs (196 -> 213, 173 -> 191 us) and the weight gradients
// (350 -> 399: heavy tiles apart no longer shared panels in L2), which keep
// the plain order. With lsplit > 1 (light tiles split into short column
// parts) every XCD instead takes an equal contiguous share of the heavy
// tiles first, all of them starting in the first round, then an equal
// contiguous share of the light parts, which run on its remaining CUs beside
// them: x is the block's XCD, c its place in that XCD's block sequence (i is
// unused). Chunk position c, tile i inside it (lsplit = 1); false past the
// class's tiles. Uniform per wave.
__device__ __forceinline__ bool spread_tile(const GemmBatch& batch, int bm, int lsplit, int x,
                                            int c, int i, int* e_out, int* r_out, int* ne_out) {
    const GemmArgs& p0 = batch.p[0];
    const int E = p0.E, lane = threadIdx.x & 63, chunk = batch.chunk;
    int ne = 0;
    if (lane < E) ne = min(expert_rows(p0.counts, p0.G, E, lane), p0.M);
    const bool heavy_l = lane < E && 2 * ne >= bm;
    const uint64_t emask = E >= 64 ? ~0ull : (1ull << E) - 1ull;
    const uint64_t hmask = __ballot(heavy_l) & emask;
    const int te = lane < E ? expert_mtiles(ne, bm, lsplit) * batch.tiles_n[0] : 0;
    int nh = heavy_l ? te : 0, nl = te;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        nh += __shfl_xor(nh, o, 64);
        nl += __shfl_xor(nl, o, 64);
    }
    nl -= nh;
    bool heavy;
    long long j;  // index in the class's list
    if (lsplit > 1) {
        const int h0 = x * nh / 8, hx = (x + 1) * nh / 8 - h0;
        heavy = c < hx;
        j = heavy ? h0 + c : x * nl / 8 + (c - hx);
        if (!heavy && c - hx >= (x + 1) * nl / 8 - x * nl / 8) return false;
    } else {
        const int nhc = (nh + chunk - 1) / chunk, nlc = (nl + chunk - 1) / chunk;
        const int first = max(nhc, (7 * (nhc + nlc) + 9) / 10);
        int ci;
        if (c < first) {
            const int hc = static_cast<int>((static_cast<long long>(c) + 1) * nhc / first);
            const int hp = static_cast<int>(static_cast<long long>(c) * nhc / first);
            heavy = hc > hp;
            ci = heavy ? hp : c - hc;
        } else {
            heavy = false;
            ci = c - nhc;
        }
        j = static_cast<long long>(ci) * chunk + i;
    }
    if (j >= (heavy ? nh : nl)) return false;
    const uint64_t cmask = heavy ? hmask : (emask & ~hmask);
    // the class's experts' tile ranges end to end (inclusive scan)
    const int t = (cmask >> lane) & 1ull ? te : 0;
    int incl = t;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int u = __shfl_up(incl, o, 64);
        if (lane >= o) incl += u;
    }
    const int e = __popcll(__ballot(incl <= j));
    *e_out = e;
    *r_out = static_cast<int>(j - __shfl(incl - t, e, 64));
    *ne_out = __shfl(ne, e, 64);
    return true;
}

// ------------------------------------------------------------------ quotas

// Fill-clamp-refill (the paper's lifespan aligning, Sec. 3.2.2) on one wave,
// lane i holding expert i (n <= 64): every expert starts from its minimum,
// the budget left is split among the unsaturated experts in proportion to
// their coefficients, an expert pushed past its saturation is clamped and
// its excess shared again, until nothing is returned; then the real shares
// are rounded to floor(sum) whole units by largest remainder (ties to the
// lower index). Every sum runs in ascending expert order with the host
// routine's operations (vmoe_fill_clamp_refill), so the units equal its
// units for the same inputs. Returns lane i's units (0 past n).
__device__ int fill_clamp_refill_wave(int n, int mn, int sat, double coef, int budget) {
    const int lane = threadIdx.x & 63;
    const bool valid = lane < n;
    double a = valid ? static_cast<double>(mn) : 0.0;
    long long need = 0;
    for (int r = 0; r < n; ++r) need += __shfl(mn, r, 64);
    bool act = valid && a < static_cast<double>(sat) && coef > 0.0;
    double left = static_cast<double>(budget - need);
    while (left > 0.0 && __ballot(act) != 0ull) {
        double W = 0.0;
        for (int r = 0; r < n; ++r) {
            const double c = __shfl(coef, r, 64);
            if (__shfl(static_cast<int>(act), r, 64)) W += c;
        }
        if (act) a += left * coef / W;
        left = 0.0;
        for (int r = 0; r < n; ++r) {
            const double ar = __shfl(a, r, 64);
            const int sr = __shfl(sat, r, 64);
            if (__shfl(static_cast<int>(act), r, 64) && ar > static_cast<double>(sr))
                left += ar - static_cast<double>(sr);
        }
        if (act && a > static_cast<double>(sat)) {
            a = static_cast<double>(sat);
            act = false;
        }
    }
    const double fl = floor(a);
    int units = static_cast<int>(fl);
    long long base = 0;
    double sum = 0.0;
    for (int r = 0; r < n; ++r) {
        base += __shfl(units, r, 64);
        sum += __shfl(a, r, 64);
    }
    long long extra = static_cast<long long>(floor(sum + 1e-9)) - base;
    bool up = false;  // rounded up already
    while (extra > 0) {
        // the largest fractional part not yet rounded up, lowest index on ties
        const double fr = (valid && !up) ? a - fl : 0.0;
        int best = -1;
        double bf = 0.0;
        for (int r = 0; r < n; ++r) {
            const double f = __shfl(fr, r, 64);
            if (f > bf) {
                best = r;
                bf = f;
            }
        }
        if (best < 0) break;
        if (lane == best) {
            ++units;
            up = true;
        }
        --extra;
    }
    return valid ? units : 0;
}

// The quota plan of one launch: per expert its rows, its tiles, the first of
// its blocks and the number of blocks it gets.
struct QuotaPlan {
    int ne[64], tiles[64], first[64], units[64];
};

// Work model of one expert's tiles, in relative time units: a tile of the
// GEMMs whose m is the expert's rows costs a fixed part (streaming its
// weight panel) plus a part in proportion to its live rows; a weight-gradient
// tile a fixed part (its output writes) plus one in proportion to the rows it
// reduces over (300 rows ~ the writes of a 256-column tile, as measured).
template <int EPI>
__device__ __forceinline__ double tile_work(int ne, int bm) {
    if constexpr (EPI == EPI_F32) return static_cast<double>(ne) + 300.0;
    else return 1.0 + static_cast<double>(min(ne, bm)) / bm;
}

constexpr bool compact_epi(int epi) { return epi != EPI_F32; }

// Wave 0 forms the launch's plan: per expert its rows and tiles, its work
// (tiles x tile_work) as the coefficient, its tiles as saturation, a minimum
// of one block when it has tiles, and the fill-clamp-refill split of the
// launch's blocks; experts own consecutive block ranges in expert order.
template <int EPI>
__device__ void build_quota_plan(const GemmBatch& batch, int bm, int lsplit, int budget,
                                 QuotaPlan* qp) {
    const int lane = threadIdx.x & 63;
    const GemmArgs& p0 = batch.p[0];
    const int E = p0.E;
    int ne = 0;
    if (lane < E)
        for (int g = 0; g < p0.G; ++g) ne += p0.counts[g * E + lane];
    int tiles = 0;
    if (lane < E) {
        if constexpr (compact_epi(EPI)) {
            ne = min(ne, p0.M);
            tiles = expert_mtiles(ne, bm, lsplit) * batch.tiles_n[0];
        } else {
            tiles = batch.tiles_m[0] * batch.tiles_n[0] +
                    (batch.total[1] > 0 ? batch.tiles_m[1] * batch.tiles_n[1] : 0);
        }
    }
    // (a light expert's column parts each carry a share of one tile's stream)
    const bool parts = lsplit > 1 && ne > 0 && ne <= 32;
    const double coef = static_cast<double>(tiles) * tile_work<EPI>(ne, bm) / (parts ? lsplit : 1);
    const int units = fill_clamp_refill_wave(E, tiles > 0 ? 1 : 0, tiles, coef, budget);
    int incl = units;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int u = __shfl_up(incl, o, 64);
        if (lane >= o) incl += u;
    }
    qp->ne[lane] = ne;
    qp->tiles[lane] = tiles;
    qp->first[lane] = incl - units;
    qp->units[lane] = units;
}

__device__ __forceinline__ float gelu_f(float h) {
    return 0.5f * h * (1.0f + erff(h * 0.70710678118654752f));
}

__device__ __forceinline__ float gelu_grad_f(float h) {
    return 0.5f * (1.0f + erff(h * 0.70710678118654752f)) +
           h * 0.39894228040143268f * __expf(-0.5f * h * h);
}

// ------------------------------------------------------------------ bf16 MFMA

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

// Two ways of staging a KB-deep operand tile (KB = 32 or 64) in LDS:
//   STAGE_REG: global -> registers -> ds_write, rows padded (k-major rows of
//              KB + 8 bf16, mn-major rows of ROWS + 32 bf16), two stages;
//   STAGE_DMA: buffer_load ... lds straight into LDS (no registers, so a ring
//              of NS stages costs LDS only): lane L of a wave instruction fills
//              bytes [16 L, 16 L + 16) of a 1 KB block, so rows are unpadded and
//              16-byte chunks are XOR-swizzled instead (k-major: chunk ^ ((row / P)
//              mod Q) with P rows per 256 bytes and Q chunks per row; mn-major:
//              chunk ^ s (k mod 4) with s = 4, or 2 when a row's chunk count is a
//              multiple of 8 but not 16, so the XOR stays inside the row), which
//              keeps fragment and transpose reads free of bank conflicts.
enum Staging { STAGE_REG = 0, STAGE_DMA = 1 };

// XOR applied to the 16-byte chunk index of k-row k of an mn-major DMA stage.
template <int ROWS>
__device__ __forceinline__ int mn_swizzle(int k) {
    static_assert((ROWS / 8) % 8 == 0, "mn-major rows must hold a multiple of 8 chunks");
    constexpr int SHIFT = (ROWS / 8) % 16 == 0 ? 2 : 1;
    return (k & 3) << SHIFT;
}

template <int ROWS, bool KMAJOR, int KB, int MODE>
__host__ __device__ constexpr int stage_elems() {
    return MODE == STAGE_DMA ? ROWS * KB : (KMAJOR ? ROWS * (KB + 8) : KB * (ROWS + 32));
}

// Element offset (in bf16) of (mn, k) inside one operand stage.
template <int ROWS, bool KMAJOR, int KB, int MODE>
__device__ __forceinline__ int lds_off(int mn, int k) {
    if constexpr (MODE == STAGE_REG) {
        return KMAJOR ? mn * (KB + 8) + k : k * (ROWS + 32) + mn;
    } else if constexpr (KMAJOR) {
        constexpr int Q = KB / 8, P = 16 / Q;  // chunks per row, rows per 256 bytes
        return mn * KB + (((k >> 3) ^ ((mn / P) % Q)) << 3) + (k & 7);
    } else {
        return k * ROWS + (((mn >> 3) ^ mn_swizzle<ROWS>(k)) << 3) + (mn & 7);
    }
}

// Byte offset in HBM of the 16-byte vector holding (mn, k..k+7) [k-major] or
// (k, mn..mn+7) [mn-major], or kOutOfRange when it lies outside the operand.
template <bool KMAJOR>
__device__ __forceinline__ uint32_t vec_off(int ld, int mn, int mn_lim, int k, int k_lim) {
    const bool ok = (mn < mn_lim) && (k < k_lim);
    const int e = KMAJOR ? mn * ld + k : k * ld + mn;
    return ok ? static_cast<uint32_t>(e) * 2u : kOutOfRange;
}

// --- register staging: ROWS * KB / 8 / NT vectors per thread, consecutive
// lanes read consecutive 16-byte segments of a row (coalesced).
template <int ROWS, bool KMAJOR, int KB, int NT>
struct RegStage {
    static constexpr int V = ROWS * KB / 8 / NT;
    static_assert(V * NT * 8 == ROWS * KB, "stage must split evenly over threads");
    static __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs, int ld, int mn0,
                                                int mn_lim, int k0, int k_lim, uint4 (&r)[V]) {
        const int tid = threadIdx.x;
#pragma unroll
        for (int j = 0; j < V; ++j) {
            if (KMAJOR) {
                constexpr int VPR = KB / 8;  // vectors per mn row
                const int q = tid + NT * j;
                r[j] = buf_load16(rs, vec_off<true>(ld, mn0 + q / VPR, mn_lim, k0 + (q % VPR) * 8, k_lim));
            } else {
                constexpr int VPR = ROWS / 8;  // vectors per k row
                const int q = tid + NT * j;
                r[j] = buf_load16(rs, vec_off<false>(ld, mn0 + (q % VPR) * 8, mn_lim, k0 + q / VPR, k_lim));
            }
        }
    }
    static __device__ __forceinline__ void store(uint16_t* s, const uint4 (&r)[V]) {
        const int tid = threadIdx.x;
#pragma unroll
        for (int j = 0; j < V; ++j) {
            const int q = tid + NT * j;
            int o;
            if (KMAJOR) {
                constexpr int VPR = KB / 8;
                o = lds_off<ROWS, true, KB, STAGE_REG>(q / VPR, (q % VPR) * 8);
            } else {
                constexpr int VPR = ROWS / 8;
                o = lds_off<ROWS, false, KB, STAGE_REG>((q % VPR) * 8, q / VPR);
            }
            *reinterpret_cast<uint4*>(s + o) = r[j];
        }
    }
};

// --- LDS DMA: the operand stage is ROWS * KB / 512 blocks of 1 KB; wave w
// issues blocks [w * PER, (w + 1) * PER). Lane L of a block holds physical
// bytes [16 L, 16 L + 16), whose logical (swizzled) position decides what it
// fetches.
template <int ROWS, bool KMAJOR, int KB, int NT>
struct DmaStage {
    static constexpr int BLOCKS = ROWS * KB * 2 / 1024;
    static constexpr int PER = BLOCKS / (NT / 64);  // wave instructions per stage
    static_assert(PER >= 1 && PER * (NT / 64) == BLOCKS, "1 KB blocks must split evenly over waves");
    static __device__ __forceinline__ void issue(__amdgpu_buffer_rsrc_t rs, int ld, int mn0,
                                                 int mn_lim, int k0, int k_lim, uint16_t* s) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int blk = wave * PER + q;
            const int byte = blk * 1024 + 16 * lane;
            uint32_t off;
            if (KMAJOR) {
                constexpr int RB = KB * 2, Q = KB / 8, P = 16 / Q;
                const int r = byte / RB;
                const int c = ((byte % RB) >> 4) ^ ((r / P) % Q);
                off = vec_off<true>(ld, mn0 + r, mn_lim, k0 + 8 * c, k_lim);
            } else {
                constexpr int RB = ROWS * 2;  // bytes per k row
                const int r = byte / RB;
                const int c = ((byte % RB) >> 4) ^ mn_swizzle<ROWS>(r);
                off = vec_off<false>(ld, mn0 + 8 * c, mn_lim, k0 + r, k_lim);
            }
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rs, (__attribute__((address_space(3))) void*)(s + blk * 512), 16, off, 0, 0, 0);
        }
    }
    // Gathered operands (rows of x): the stage row lane L fetches in wave
    // instruction q (k-major: an mn row of the tile; mn-major: a k row).
    static __device__ __forceinline__ int lane_row(int q) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        const int byte = (wave * PER + q) * 1024 + 16 * lane;
        return byte / (KMAJOR ? KB * 2 : ROWS * 2);
    }
    // k-major, gathered rows: rowoff[q] = element offset in x of the start of
    // the row lane_row(q) stands for (-1 past the rows).
    static __device__ __forceinline__ void issue_rows(__amdgpu_buffer_rsrc_t rs,
                                                      const int (&rowoff)[PER], int k0,
                                                      int k_lim, uint16_t* s) {
        static_assert(KMAJOR, "row gather: k-major operand");
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int blk = wave * PER + q;
            const int byte = blk * 1024 + 16 * lane;
            constexpr int RB = KB * 2, Q = KB / 8, P = 16 / Q;
            const int r = byte / RB;
            const int c = ((byte % RB) >> 4) ^ ((r / P) % Q);
            const int kk = k0 + 8 * c;
            const uint32_t off = (rowoff[q] >= 0 && kk < k_lim)
                                     ? static_cast<uint32_t>(rowoff[q] + kk) * 2u
                                     : kOutOfRange;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rs, (__attribute__((address_space(3))) void*)(s + blk * 512), 16, off, 0, 0, 0);
        }
    }
    // mn-major, gathered k rows: rowoff[q] = byte offset in x of the k row
    // lane_row(q) stands for in this stage, col[q] = byte offset of the lane's
    // 8 columns in it (krow_cols); either is kGatherSentinel outside the
    // operand, which puts the sum past the end of x.
    static __device__ __forceinline__ void krow_cols(int mn0, int mn_lim, uint32_t (&col)[PER]) {
        static_assert(!KMAJOR, "k-row gather: mn-major operand");
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int byte = (wave * PER + q) * 1024 + 16 * lane;
            constexpr int RB = ROWS * 2;
            const int r = byte / RB;
            const int mn = mn0 + 8 * (((byte % RB) >> 4) ^ mn_swizzle<ROWS>(r));
            col[q] = mn < mn_lim ? static_cast<uint32_t>(mn) * 2u : kGatherSentinel;
        }
    }
    static __device__ __forceinline__ void issue_krows(__amdgpu_buffer_rsrc_t rs,
                                                       const uint32_t (&rowoff)[PER],
                                                       const uint32_t (&col)[PER], uint16_t* s) {
        const int wave = threadIdx.x >> 6;
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int blk = wave * PER + q;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rs, (__attribute__((address_space(3))) void*)(s + blk * 512), 16,
                rowoff[q] + col[q], 0, 0, 0);
        }
    }
};

// s_waitcnt immediate for vmcnt(n) and lgkmcnt(0) (expcnt left alone).
template <int N>
struct VmWait {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    static constexpr int imm = (N & 15) | ((N >> 4) << 14) | (7 << 4);
};

// Workgroup barrier for the stage ring. __syncthreads() fences all memory at
// workgroup scope, which waits for every LDS DMA in flight (vmcnt(0)) and
// would cap the prefetch at one stage; here the caller's s_waitcnt has
// already retired this wave's LDS reads and the DMA of the stage about to be
// read, so a bare s_barrier suffices. The signal fences keep the compiler
// from moving memory accesses across it.
__device__ __forceinline__ void ring_barrier() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
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
template <int ROWS, bool KMAJOR, int KB, int MODE>
__device__ __forceinline__ bf16x8 read_frag(const uint16_t* s, int blk, int kstep, int lane) {
    if (KMAJOR) {
        const int mn = blk * 32 + (lane & 31), k = kstep * 16 + (lane >> 5) * 8;
        return *reinterpret_cast<const bf16x8*>(s + lds_off<ROWS, true, KB, MODE>(mn, k));
    } else {
        // 16-lane group g covers mn [16 (g & 1), +16) and k [8 (g >> 1), +8)
        const int g = lane >> 4, j = lane & 15;
        const int k = kstep * 16 + 8 * (g >> 1) + (j >> 2);
        const int mn = blk * 32 + 16 * (g & 1) + 4 * (j & 3);
        const s16x4 lo = lds_read_tr(s + lds_off<ROWS, false, KB, MODE>(mn, k));
        const s16x4 hi = lds_read_tr(s + lds_off<ROWS, false, KB, MODE>(mn, k + 4));
        const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        return __builtin_bit_cast(bf16x8, v);
    }
}

// GELU and its derivative from one exponential. With phi the standard normal
// density, Abramowitz & Stegun 26.2.17 gives the upper tail
//   q = 1 - Phi(|h|) = phi(h) t (b1 + t (b2 + t (b3 + t (b4 + t b5)))),
//   t = 1 / (1 + p |h|), |error| < 7.5e-8 (far below bf16 rounding), so
//   Phi(h) = 0.5 + sign(h) (0.5 - q),  gelu(h) = h Phi(h),  gelu'(h) = Phi(h) + h phi(h),
// where phi(h) = 2^(-h^2 log2(e) / 2 + log2(1 / sqrt(2 pi))) is one v_exp_f32.
__device__ __forceinline__ void gelu_pair(float h, float& g, float& dg) {
    const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(fabsf(h), 0.2316419f, 1.0f));
    const float phi = __builtin_amdgcn_exp2f(
        __builtin_fmaf(h * h, -0.72134752044448170f, -1.32574806473615920f));
    float poly = __builtin_fmaf(t, 1.330274429f, -1.821255978f);
    poly = __builtin_fmaf(t, poly, 1.781477937f);
    poly = __builtin_fmaf(t, poly, -0.356563782f);
    poly = __builtin_fmaf(t, poly, 0.319381530f);
    const float q = (t * poly) * phi;
    const float phi_cdf = 0.5f + copysignf(0.5f - q, h);
    g = h * phi_cdf;
    dg = __builtin_fmaf(h, phi, phi_cdf);
}

// Static description of one bf16 GEMM tiling: BM x BN block tile of WGM x WGN
// waves, KB-deep stages, NS stages in flight, staging mode.
template <int BM_, int BN_, int WGM_, int WGN_, int KB_, int NS_, int MODE_, bool PAIR_ = false>
struct Tile {
    static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_, KB = KB_, NS = NS_;
    static constexpr int MODE = MODE_;
    // PAIR: stages are fetched two at a time (kt + 2 and kt + 3 at each even
    // kt), so the two 64-byte halves of a 128-byte k-major row segment are
    // requested back to back and share one cache-line fill
    static constexpr bool PAIR = PAIR_;
    static constexpr int NW = WGM * WGN, NT = 64 * NW;
    static constexpr int WM = BM / WGM, WN = BN / WGN;  // wave tile
    static constexpr int FM = WM / 32, FN = WN / 32;    // 32 x 32 MFMA blocks per wave
    static constexpr int KSTEPS = KB / 16;
    // two waves per SIMD: 8-wave tiles, or two 4-wave blocks per CU when their
    // stage rings fit half the LDS; one 4-wave block per CU otherwise
    static constexpr int RING_BYTES = NS * (BM + BN) * KB * 2;
    static constexpr int WAVES_PER_EU = (NW == 8 || RING_BYTES <= 80 * 1024) ? 2 : 1;
    static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile must be whole 32 x 32 blocks");
    static_assert(KSTEPS % 2 == 0, "fragment double buffering needs an even step count");
    static_assert(MODE == STAGE_DMA || NS == 2, "register staging runs two stages");
    static_assert(NS >= 2 && NS <= 5, "stage ring size");
    static_assert(!PAIR || (NS == 4 && MODE == STAGE_DMA), "paired fetch runs a ring of four");
};

// Per-GEMM static sizes derived from a tiling and the operand layouts.
template <class T, bool A_KMAJOR, bool B_KMAJOR, int EPI>
struct GemmCfg {
    static constexpr int AE = stage_elems<T::BM, A_KMAJOR, T::KB, T::MODE>();
    static constexpr int BE = stage_elems<T::BN, B_KMAJOR, T::KB, T::MODE>();
    static constexpr int BUF_BYTES = (AE + BE) * 2;  // one stage buffer
    static constexpr bool F32_OUT = EPI == EPI_F32;
    static constexpr int OUTS = EPI == EPI_FWD1 ? 2 : 1;
    // Epilogue staging: wave w parks its outputs in stage buffer w mod NS; IPP
    // of its FM 32-row blocks per pass, all outputs of those rows at once when
    // they fit (a second output pass would recompute the activation).
    // staged rows padded by 16 bytes: 16-byte aligned for the row reads (a
    // 136-byte bf16 row left every other row's reads misaligned, which the
    // LDS serves with stalls) and off the banks of the row above
    static constexpr int ELEM = F32_OUT ? 4 : 2;
    static constexpr int EP_LD = T::WN + 16 / ELEM;
    static constexpr int EP_ROWBLK = 32 * EP_LD * ELEM;
    static constexpr int WAVES_PER_BUF = (T::NW + T::NS - 1) / T::NS;
    static constexpr bool fits(int outs, int blocks) {
        return outs * blocks * EP_ROWBLK * WAVES_PER_BUF <= BUF_BYTES;
    }
    static constexpr int EP_OUTS_AT_ONCE = fits(OUTS, 1) ? OUTS : 1;
    static constexpr int IPP = fits(EP_OUTS_AT_ONCE, T::FM) ? T::FM
                             : (fits(EP_OUTS_AT_ONCE, T::FM / 2) ? T::FM / 2 : 1);
    static constexpr int EP_TILE = IPP * EP_ROWBLK;
    static_assert(fits(EP_OUTS_AT_ONCE, IPP), "epilogue staging exceeds LDS");
    static_assert(!F32_OUT || !A_KMAJOR, "row sums read an mn-major A tile");
    static_assert(!F32_OUT || T::NT % T::BM == 0, "row sums give each A row NT / BM threads");
    static_assert(!F32_OUT || T::NT * 4 <= BUF_BYTES, "row-sum partials fit one stage buffer");
};

template <class T, bool A_KMAJOR, bool B_KMAJOR, int MODE>
struct Frags {
    static constexpr int FM = T::FM, FN = T::FN;
    bf16x8 a[FM], b[FN];
    // fm_live: the wave's 32-row blocks that hold rows of the output (wave-
    // uniform); the A fragments of the others are not read
    __device__ __forceinline__ void read(const uint16_t* As, const uint16_t* Bs, int wm, int wn,
                                         int ks, int lane, int fm_live) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
            if (i < fm_live)
                a[i] = read_frag<T::BM, A_KMAJOR, T::KB, MODE>(As, wm * FM + i, ks, lane);
#pragma unroll
        for (int j = 0; j < FN; ++j)
            b[j] = read_frag<T::BN, B_KMAJOR, T::KB, MODE>(Bs, wn * FN + j, ks, lane);
    }
};

// acc[i][j] += A-block i x B-block j for the live row blocks i < fm_live (a
// wave-uniform scalar, so the skipped products are branches, not masks); the
// operands are swapped inside the MFMA so that register 4q + r of lane l
// holds C[m = l % 32][n = 8q + 4 (l / 32) + r].
template <int FM, int FN, typename F>
__device__ __forceinline__ void mfma_block(f32x16 (&acc)[FM][FN], const F& f, int fm_live) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
        if (i < fm_live) {
#pragma unroll
            for (int j = 0; j < FN; ++j)
                acc[i][j] =
                    __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.b[j], f.a[i], acc[i][j], 0, 0, 0);
        }
}

// Bias of the columns a lane owns: column 32 j + 8 q + 4 (l / 32) + 0..3 of the
// wave tile, for j < FN, q < 4, as four packed bf16 (zero past N). Loaded ahead
// of the first operand stages; the accumulators start from it.
template <class T, int EPI>
struct BiasRegs {
    static constexpr bool USED = EPI == EPI_FWD1 || EPI == EPI_BIAS;
    uint2 v[USED ? T::FN * 4 : 1];
    __device__ __forceinline__ void load(const GemmArgs& p, int e, int N, int n0, int wn, int lane) {
        if constexpr (USED) {
#pragma unroll
            for (int j = 0; j < T::FN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int n = n0 + wn * T::WN + j * 32 + 8 * q + 4 * (lane >> 5);
                    v[j * 4 + q] = n < N ? *reinterpret_cast<const uint2*>(
                                               static_cast<const uint16_t*>(p.bias) +
                                               e * p.bias_estride + n)
                                         : make_uint2(0u, 0u);
                }
        }
    }
};

// Epilogue of one block: optional bias-gradient row sums (partials combined in
// part_buf), then each wave turns its accumulators (bias included) into outputs (GELU +
// GELU', GELU' product), parks them in its own slot of ep_buf and writes every
// output row as 16-byte-per-lane segments. The slots are private to a wave and
// LDS accesses of one wave complete in order, so the passes need no barrier.
template <class T, class CFG, int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& p, f32x16 (&acc)[T::FM][T::FN],
                                              uint16_t* part_buf,
                                              uint16_t* ep_buf, float rsum, bool row_sum, int e,
                                              int M, int N, int m0, int n0, int fm_live) {
    constexpr int FM = T::FM, FN = T::FN, WM = T::WM, WN = T::WN, BM_ = T::BM;
    constexpr int EP_LD = CFG::EP_LD, ELEM = CFG::ELEM, EP_TILE = CFG::EP_TILE;
    constexpr int IPP = CFG::IPP, OUTS = CFG::OUTS, EPO = CFG::EP_OUTS_AT_ONCE;
    constexpr bool F32_OUT = CFG::F32_OUT;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / T::WGN, wn = wave % T::WGN;

    if constexpr (F32_OUT) {
        if (row_sum) {  // uniform per block
            constexpr int SPLIT = T::NT / BM_;
            float* part = reinterpret_cast<float*>(part_buf);
            part[tid] = rsum;
            __syncthreads();
            if (tid < BM_ && m0 + tid < M) {
                float t = part[tid];
#pragma unroll
                for (int q = 1; q < SPLIT; ++q) t += part[tid + q * BM_];
                p.bsum[static_cast<size_t>(e) * M + m0 + tid] = t;
            }
            __syncthreads();
        }
    }

    char* ep = reinterpret_cast<char*>(ep_buf) + (wave / T::NS) * EPO * EP_TILE;
    constexpr int SEG = 16 / ELEM;                 // elements per 16-byte segment
    constexpr int LANES_PER_ROW = WN / SEG;
    constexpr int ROWS_PER_PASS = 64 / LANES_PER_ROW;  // lanes past ROWS_PER_PASS rows idle
    constexpr int PASSES = (IPP * 32 + ROWS_PER_PASS - 1) / ROWS_PER_PASS;
    static_assert(LANES_PER_ROW <= 64 && WN % SEG == 0, "epilogue row split");

#pragma unroll
    for (int i0 = 0; i0 < FM; i0 += IPP) {
        if (i0 >= fm_live) break;  // the wave's remaining rows are past M
        // saved gelu'(H) of this pass's rows, all loads in flight together
        uint2 aux[EPI == EPI_GELU_GRAD ? IPP * FN * 4 : 1];
        if constexpr (EPI == EPI_GELU_GRAD) {
#pragma unroll
            for (int ii = 0; ii < IPP; ++ii)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int n = n0 + wn * WN + j * 32 + 8 * q + 4 * (lane >> 5);
                        const int m = m0 + wm * WM + (i0 + ii) * 32 + (lane & 31);
                        aux[(ii * FN + j) * 4 + q] =
                            (n < N && m < M) ? *reinterpret_cast<const uint2*>(
                                                   static_cast<const uint16_t*>(p.aux) +
                                                   e * p.out_estride +
                                                   static_cast<size_t>(m) * p.ldo + n)
                                             : make_uint2(0u, 0u);
                    }
        }
#pragma unroll
        for (int o0 = 0; o0 < OUTS; o0 += EPO) {
            // Stage 1: register 4q + r of lane l holds C[m][n + r] with
            // m = 32 i + l % 32, n = 32 j + 8 q + 4 (l / 32) inside the wave tile.
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
                            // (the bias of EPI_FWD1 / EPI_BIAS is already in acc)
                            if constexpr (EPI == EPI_GELU_GRAD) {
                                const uint2 gg = aux[(ii * FN + j) * 4 + q];
                                r[0] *= bf16_to_f32(gg.x & 0xFFFFu);
                                r[1] *= bf16_to_f32(gg.x >> 16);
                                r[2] *= bf16_to_f32(gg.y & 0xFFFFu);
                                r[3] *= bf16_to_f32(gg.y >> 16);
                            }
                            uint16_t* t0 = reinterpret_cast<uint16_t*>(ep) + ml * EP_LD + nl;
                            if constexpr (EPI == EPI_FWD1) {
                                float g[4], dg[4];
#pragma unroll
                                for (int c = 0; c < 4; ++c) gelu_pair(r[c], g[c], dg[c]);
#pragma unroll
                                for (int o = 0; o < EPO; ++o) {
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

            // Stage 2: staged rows out in 16-byte segments.
            const int cl = (lane % LANES_PER_ROW) * SEG;
            const int n = n0 + wn * WN + cl;
            const int lrow = lane / LANES_PER_ROW;
#pragma unroll
            for (int o = 0; o < EPO; ++o) {
                char* dst_base = static_cast<char*>(o0 + o == 0 ? p.out : p.out2);
#pragma unroll
                for (int pass = 0; pass < PASSES; ++pass) {
                    const int ml = pass * ROWS_PER_PASS + lrow;
                    if (lrow >= ROWS_PER_PASS || ml >= IPP * 32) continue;
                    const int m = m0 + wm * WM + i0 * 32 + ml;
                    const uint4 v = *reinterpret_cast<const uint4*>(ep + o * EP_TILE +
                                                                    (ml * EP_LD + cl) * ELEM);
                    if (m < M && n < N) {
                        v4i32* dst = reinterpret_cast<v4i32*>(
                            dst_base +
                            (e * p.out_estride + static_cast<size_t>(m) * p.ldo + n) * ELEM);
                        // weight gradients are not read again by the layer: streaming
                        // stores keep them from displacing cached activations (the f32
                        // write-back cost a fifth of the weight-gradient GEMM, measured alone)
                        if constexpr (F32_OUT)
                            __builtin_nontemporal_store(__builtin_bit_cast(v4i32, v), dst);
                        else
                            *dst = __builtin_bit_cast(v4i32, v);
                    }
                }
            }
        }
    }
}

// Light tiles. A tile whose live rows fit one 32-row block (an expert with a
// handful of rows under a skewed load) streams a BN-column weight panel over
// the whole k range for a few products, so its time is that stream, and the
// stage ring keeps only NS - 1 stages of it in flight. Such a tile skips the
// ring: each wave streams its own share in 64-deep k groups, two groups in
// flight in registers, every load a coalesced 128-byte piece of a row; a
// group passes through a small LDS block of the wave's own to be read back
// as fragments. The waves of the block split the tile's columns (whole wave
// columns) and its k groups between them, and the waves of k slice 0 add the
// other slices' sums in slice order (a fixed order) before the usual
// epilogue of their one live row block.
constexpr int kLightGroups = 2;  // 64-deep k groups in flight per wave

// LDS-typed views of the stage buffers for the light path (a pointer selected
// among the buffers at run time would otherwise become a flat pointer, whose
// accesses wait on the vector-memory counter too)
typedef __attribute__((address_space(3))) uint16_t lds_u16;
typedef __attribute__((address_space(3))) v4i32 lds_v4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) float lds_f32;

// Stage buffer i of NS as an LDS pointer (a select over values: a closure or
// array of the buffers' addresses would sit in scratch memory)
template <int NS>
__device__ __forceinline__ lds_u16* pick_lds(int i, uint16_t* b0, uint16_t* b1, uint16_t* b2,
                                             uint16_t* b3, uint16_t* b4) {
    uint16_t* b = b0;
    if (NS > 1 && i == 1) b = b1;
    if (NS > 2 && i == 2) b = b2;
    if (NS > 3 && i == 3) b = b3;
    if (NS > 4 && i == 4) b = b4;
    return (lds_u16*)(b);
}

template <class T, bool A_KMAJOR, bool B_KMAJOR, int EPI>
constexpr bool light_ok() {
    return A_KMAJOR && EPI != EPI_F32 && T::WN == 64;
}

// A light expert's tiles split into this many column parts (whole wave
// columns each): one HBM stream per CU runs at a fraction of a CU's share of
// the chip's bandwidth, so a light tile's weight panel is spread over CUs.
template <class T>
constexpr int light_parts() {
    return T::WGN % 4 == 0 ? 4 : (T::WGN % 2 == 0 ? 2 : 1);
}

template <class T, class CFG, bool B_KMAJOR, int EPI, int GS>
__device__ __forceinline__ void light_tile(const GemmArgs& p, __amdgpu_buffer_rsrc_t ra_rs,
                                           __amdgpu_buffer_rsrc_t rb_rs, int e, int M, int N,
                                           int K, int m0, int n0, int part, int nparts,
                                           uint16_t* buf0, uint16_t* buf1, uint16_t* buf2,
                                           uint16_t* buf3, uint16_t* buf4) {
    constexpr int FM = T::FM, FN = T::FN, WN = T::WN, WGN = T::WGN, NS = T::NS;
    constexpr int U = kLightGroups;
    constexpr int LD = 64 + 8;          // LDS row: 64 elements + 16 bytes (rows on other banks)
    constexpr int A_EL = 32 * LD;       // A block: 32 rows x 64 k
    constexpr int B_EL = 64 * LD;       // B block: 64 n x 64 k (k-major) or 64 k x 64 n
    constexpr int W_EL = A_EL + B_EL;   // one wave's LDS block
    constexpr int WPB = (T::NW + NS - 1) / NS;  // waves per stage buffer
    constexpr int PB = FN * 16 * 64;    // floats of one wave's partial sums
    static_assert(WN == 64 && FN == 2, "light tiles: 64-column wave tiles");
    static_assert(WPB * W_EL * 2 <= CFG::BUF_BYTES, "wave LDS blocks fit the stage buffers");
    static_assert((T::NW - 1 + NS - 1) / NS * PB * 4 <= CFG::BUF_BYTES,
                  "partial sums fit the stage buffers");
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    // the part's columns are `cols` wave columns; wave w takes column c and k
    // slice sl of ks (slice 0 holds the sums)
    const int cols = WGN / nparts, ks = T::NW / cols;
    const int c = wave % cols, sl = wave / cols;
    const int nb = n0 + (part * cols + c) * WN;  // the wave's first column
    // the epilogue places wave w's columns at n0 + (w mod WGN) WN
    const int wn = wave % WGN, n0w = nb - wn * WN;
    // slice sl takes the 64-deep k groups [g0, g1); loads past klim read zeros
    const int ng = (K + 63) / 64;
    const int g0 = ng * sl / ks, g1 = ng * (sl + 1) / ks;
    const int klim = min(K, g1 * 64);
    // load i of a group: row (k-major) or k row (mn-major) 8 i + lane / 8,
    // elements 8 (lane % 8) .. + 7 of its 64
    const int lr = lane >> 3, lc = 8 * (lane & 7);
    int arow[4];  // element offsets of the lane's A rows, -1 past M
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int mr = m0 + 8 * i + lr;
        if constexpr (GS == 1) arow[i] = mr < M ? p.tok[e * p.tok_estride + mr] * p.a.ld : -1;
        else arow[i] = mr < M ? mr * p.a.ld : -1;
    }

    uint4 ra[U][4], rb[U][8];
    auto load = [&](int u, int g) {
        const int k = g * 64 + lc;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            ra[u][i] = buf_load16(ra_rs, arow[i] >= 0 && k < klim
                                             ? static_cast<uint32_t>(arow[i] + k) * 2u
                                             : kOutOfRange);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            if constexpr (B_KMAJOR)
                rb[u][i] = buf_load16(rb_rs, vec_off<true>(p.b.ld, nb + 8 * i + lr, N, k, klim));
            else
                rb[u][i] = buf_load16(rb_rs, vec_off<false>(p.b.ld, nb + lc, N, g * 64 + 8 * i + lr,
                                                            klim));
        }
    };

    BiasRegs<T, EPI> bias;
    bias.load(p, e, N, n0w, wn, lane);
    f32x16 lacc[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            float b4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            if constexpr (BiasRegs<T, EPI>::USED) {
                if (sl == 0) {
                    const uint2 bb = bias.v[j * 4 + q];
                    b4[0] = bf16_to_f32(bb.x & 0xFFFFu);
                    b4[1] = bf16_to_f32(bb.x >> 16);
                    b4[2] = bf16_to_f32(bb.y & 0xFFFFu);
                    b4[3] = bf16_to_f32(bb.y >> 16);
                }
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) lacc[j][4 * q + r] = b4[r];
        }

    auto lds_buf = [=](int i) { return pick_lds<NS>(i, buf0, buf1, buf2, buf3, buf4); };
    // wave w's LDS block: stage buffer w mod NS, slot w / NS
    lds_u16* const as = lds_buf(wave % NS) + (wave / NS) * W_EL;
    lds_u16* const bs = as + A_EL;
    // (group by group, as the loop refills them: each group then waits for its
    // own loads only, also on the loop's first trip)
#pragma unroll
    for (int u = 0; u < U; ++u) {
        load(u, g0 + u);
        __builtin_amdgcn_sched_barrier(0);
    }
    for (int g = g0; g < g1; g += U) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            // the group into the wave's LDS block (one wave's LDS accesses run
            // in order: the previous group's fragment reads are done first)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                *reinterpret_cast<lds_v4*>(as + (8 * i + lr) * LD + lc) =
                    __builtin_bit_cast(v4i32, ra[u][i]);
#pragma unroll
            for (int i = 0; i < 8; ++i)
                *reinterpret_cast<lds_v4*>(bs + (8 * i + lr) * LD + lc) =
                    __builtin_bit_cast(v4i32, rb[u][i]);
            __builtin_amdgcn_sched_barrier(0);
            // its registers refill with group g + u + U (past g1: out of range,
            // no traffic), so U groups stay in flight
            load(u, g + u + U);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int kk = 16 * s + 8 * (lane >> 5);
                const bf16x8 a = *reinterpret_cast<const lds_bf16x8*>(as + (lane & 31) * LD + kk);
                bf16x8 b[FN];
#pragma unroll
                for (int j = 0; j < FN; ++j) {
                    if constexpr (B_KMAJOR) {
                        b[j] = *reinterpret_cast<const lds_bf16x8*>(bs + (32 * j + (lane & 31)) * LD +
                                                                    kk);
                    } else {
                        // transposing reads of the [k][n] block: lane gets column
                        // 32 j + lane % 32, k rows 16 s + 8 (lane / 32) + 0..7
                        const int gq = lane >> 4, jj = lane & 15;
                        const int kr = 16 * s + 8 * (gq >> 1) + (jj >> 2);
                        const int n = 32 * j + 16 * (gq & 1) + 4 * (jj & 3);
                        typedef __attribute__((address_space(3))) s16x4* lds_s16x4;
                        const s16x4 lo =
                            __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4)(bs + kr * LD + n));
                        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                            (lds_s16x4)(bs + (kr + 4) * LD + n));
                        b[j] = __builtin_bit_cast(
                            bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
                    }
                }
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    lacc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[j], a, lacc[j], 0, 0, 0);
            }
        }
    }

    // slices 1.. park their sums (slot s = (sl - 1) cols + c: stage buffer s
    // mod NS); every wave is past its LDS block first
    auto slot = [&](int s) -> lds_f32* {
        return reinterpret_cast<lds_f32*>(lds_buf(s % NS)) + (s / NS) * PB;
    };
    __syncthreads();
    if (sl > 0) {
        lds_f32* const dst = slot((sl - 1) * cols + c);
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) dst[(j * 16 + r) * 64 + lane] = lacc[j][r];
    }
    __syncthreads();
    f32x16 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
    if (sl == 0) {
        for (int s = 1; s < ks; ++s) {
            const lds_f32* const src = slot((s - 1) * cols + c);
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) lacc[j][r] += src[(j * 16 + r) * 64 + lane];
        }
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[0][j] = lacc[j];
    }
    __syncthreads();  // the sums are read before the epilogue stages outputs over them
    uint16_t* const ep = (uint16_t*)(lds_buf(wave % NS));  // (an LDS pointer, seen as such)
    gemm_epilogue<T, CFG, EPI>(p, acc, buf0, ep, 0.0f, false, e, M, N, m0, n0w, sl == 0 ? 1 : 0);
}

// One BM x BN output tile of expert e per block of WGM x WGN waves, each
// (BM/WGM) x (BN/WGN) as 32 x 32 MFMA blocks; tiles are dealt to the 8 XCDs
// in chunks of neighbouring tiles (shared operand panels in each XCD's L2).
//
// Pipeline over KB-deep k-stages, one barrier per stage, NS stage buffers
// (separate LDS arrays, so every access names its buffer statically):
//   issue the loads of stage kt + NS - 1 (DMA: straight into the buffer that
//     stage kt - 1 used; REG: into registers, written to the other buffer
//     before the barrier)
//   steps 0 .. KSTEPS-2: read fragments of step s+1   | MFMAs of step s
//   wait until stage kt + 1 has landed; barrier
//   read step-0 fragments of stage kt+1               | MFMAs of the last step
// so LDS latency always hides behind a run of MFMAs on held fragments, and
// HBM latency behind NS - 1 stages of MFMAs. The stage count is rounded up to
// a multiple of NS so the ring unrolls with static buffers; the padding
// stages load zeros (out of range) and skip their MFMAs.
// SCHED = 0: one tile per block, the grid dealt over the (live) tile list;
// SCHED = 1: persistent blocks, each expert owning the number of blocks the
// fill-clamp-refill quota gives it, each block taking every units-th tile
// of its expert.
// GATHER = 1: operand A's rows are gathered token rows of x (the
// up-projection fused with the dispatch); GATHER = 2: operand B's k rows are
// (the input-weight gradient, problems with a token list).
// (the k-row gather's token table takes the LDS of a second 4-wave block)
template <class T, int GATHER>
constexpr int gemm_waves_per_eu() {
    return GATHER == 2 && T::NW == 4 ? 1 : T::WAVES_PER_EU;
}

template <class T, bool A_KMAJOR, bool B_KMAJOR, int EPI, int SCHED = 0, int GATHER = 0>
__global__ __launch_bounds__(T::NT)
__attribute__((amdgpu_waves_per_eu(gemm_waves_per_eu<T, GATHER>(),
                                   gemm_waves_per_eu<T, GATHER>())))
void gemm_bf16_kernel(GemmBatch batch) {
    using CFG = GemmCfg<T, A_KMAJOR, B_KMAJOR, EPI>;
    constexpr int BM_ = T::BM, BN_ = T::BN, KB = T::KB, NS = T::NS, MODE = T::MODE;
    constexpr int NT = T::NT, AE = CFG::AE, BE = CFG::BE, FM = T::FM, FN = T::FN;
    constexpr int KSTEPS = T::KSTEPS;
    constexpr int SZ = AE + BE;
    constexpr int SZX = SZ > 8 ? SZ : 8;
    __shared__ __attribute__((aligned(1024))) uint16_t buf0[SZ];
    __shared__ __attribute__((aligned(1024))) uint16_t buf1[SZ];
    __shared__ __attribute__((aligned(1024))) uint16_t buf2[NS > 2 ? SZX : 8];
    __shared__ __attribute__((aligned(1024))) uint16_t buf3[NS > 3 ? SZX : 8];
    __shared__ __attribute__((aligned(1024))) uint16_t buf4[NS > 4 ? SZX : 8];
    // gathered k rows' byte offsets in x (padded by two rings of stages)
    __shared__ uint32_t tok_s[GATHER == 2 ? kGatherRows + 2 * NS * KB : 1];

    const int b = blockIdx.x;
    // column parts of a light expert's tiles: at most the expert's m-tile
    // slots of the grid (ceil(capacity / BM)), so the live tiles still fit it
    // (the d-wide row GEMMs: a few long tiles per expert; the f-wide ones have
    // many short light tiles already)
    const int lsplit = light_ok<T, A_KMAJOR, B_KMAJOR, EPI>() && (EPI == EPI_BIAS || EPI == EPI_STORE)
                           ? min(light_parts<T>(), (batch.p[0].M + BM_ - 1) / BM_)
                           : 1;
    int qe = 0, qu = 0, qn = 0, qt = 0, qne = 0;  // quota: expert, rank, units, tiles, rows
    if constexpr (SCHED == 1) {
        __shared__ QuotaPlan qp;
        if (threadIdx.x < 64)
            build_quota_plan<EPI>(batch, BM_, lsplit, static_cast<int>(gridDim.x), &qp);
        __syncthreads();
        const int lane = threadIdx.x & 63;
        const int end = qp.first[lane] + qp.units[lane];
        const int e_b = __popcll(__ballot(end <= b));  // ends never decrease
        if (e_b >= batch.p[0].E) return;              // past every quota
        // (uniform values read from LDS: kept in scalar registers)
        qe = __builtin_amdgcn_readfirstlane(e_b);
        qn = __builtin_amdgcn_readfirstlane(qp.units[e_b]);
        qu = __builtin_amdgcn_readfirstlane(b - qp.first[e_b]);
        qt = __builtin_amdgcn_readfirstlane(qp.tiles[e_b]);
        qne = __builtin_amdgcn_readfirstlane(qp.ne[e_b]);
    }
    for (int it = 0;; ++it) {
    int prob = 0, e, r, ne, tiles_m;
    if constexpr (SCHED == 1) {
        r = qu + it * qn;
        if (r >= qt) break;
        e = qe;
        ne = qne;
        if constexpr (compact_tiles<EPI>()) {
            tiles_m = expert_mtiles(ne, BM_, lsplit);
        } else {
            const int t0 = batch.tiles_m[0] * batch.tiles_n[0];
            prob = r >= t0 ? 1 : 0;
            if (prob) r -= t0;
            tiles_m = batch.tiles_m[prob];
        }
    } else {
    // Block b runs on XCD b mod 8 as that XCD's (b / 8)-th block; XCDs take
    // chunks of `chunk` consecutive tiles in turn, so the tiles resident on an
    // XCD share operand panels in its L2 while every XCD gets an even share of
    // each expert, however unevenly the rows are spread over experts.
    const int l = b >> 3, chunk = batch.chunk;
    int w = ((l / chunk) * 8 + (b & 7)) * chunk + l % chunk;
    if constexpr (EPI == EPI_BIAS || EPI == EPI_STORE) {
        const bool in = lsplit > 1
                            ? spread_tile(batch, BM_, lsplit, b & 7, l, 0, &e, &r, &ne)
                            : spread_tile(batch, BM_, lsplit, b & 7, (l / chunk) * 8 + (b & 7),
                                          l % chunk, &e, &r, &ne);
        if (!in) return;
        tiles_m = expert_mtiles(ne, BM_, lsplit);
    } else if constexpr (compact_tiles<EPI>()) {
        LiveTile lt;
        const GemmArgs& p0 = batch.p[0];
        if (!live_tile(p0.counts, p0.G, p0.E, p0.M, BM_, lsplit, batch.tiles_n[0], w, &lt)) return;
        e = lt.e;
        r = lt.r;
        ne = lt.ne;
        tiles_m = expert_mtiles(ne, BM_, lsplit);
    } else {
        if (w >= batch.total[0] + batch.total[1]) return;
        prob = w >= batch.total[0] ? 1 : 0;  // uniform per block
        if (prob) w -= batch.total[0];
        tiles_m = batch.tiles_m[prob];
        const int tiles_e = tiles_m * batch.tiles_n[prob];
        e = w / tiles_e;
        r = w - e * tiles_e;
        ne = expert_rows(batch.p[prob].counts, batch.p[prob].G, batch.p[prob].E, e);
    }
    }
    // The tile body, instantiated once per operand kind: with GS != 0 the
    // gathered operand is known at compile time, so a problem that gathers
    // and one that does not (the two weight gradients of one launch) each
    // get a main loop register-allocated for its own addressing alone.
    auto tile = [&](auto gather_kind) -> bool {
    constexpr int GS = decltype(gather_kind)::value;
    const GemmArgs& p = batch.p[prob];
    const int tiles_n = batch.tiles_n[prob];
    const int group_m = batch.group_m;
    // inside one expert, tiles go in groups of group_m m-tiles, m fastest, so
    // the blocks resident on an XCD at once cover a compact patch of the output
    // and share both operand panels in its L2
    const int grp = r / (group_m * tiles_n);
    const int first_m = grp * group_m;
    const int gm = min(group_m, tiles_m - first_m);
    const int idx = r - grp * group_m * tiles_n;
    const int tm = first_m + idx % gm;
    const int tn = idx / gm;
    const int M = p.var_k ? p.M : min(ne, p.M);
    const int K = p.var_k ? ne : p.K;
    const int N = p.N;
    // a light expert's m-tile index is its column part
    const bool parts = lsplit > 1 && !p.var_k && ne > 0 && ne <= 32;
    const int m0 = parts ? 0 : tm * BM_, n0 = tn * BN_;
    if (m0 >= M) return false;

    static_assert(GS == 0 || (GS == 1 && A_KMAJOR) || (GS == 2 && !B_KMAJOR),
                  "gathered rows: k-major A or mn-major B");
    // gathered operands address x itself: its whole size is their range
    const __amdgpu_buffer_rsrc_t ra_rs =
        GS == 1 ? make_rsrc(p.a.base, p.gather_bytes)
           : make_rsrc(static_cast<const uint16_t*>(p.a.base) + e * p.a.estride,
                       p.a.estride * 2);
    const __amdgpu_buffer_rsrc_t rb_rs =
        GS == 2 ? make_rsrc(p.b.base, p.gather_bytes)
           : make_rsrc(static_cast<const uint16_t*>(p.b.base) + e * p.b.estride,
                       p.b.estride * 2);
    if constexpr (light_ok<T, A_KMAJOR, B_KMAJOR, EPI>()) {
        if (!p.var_k && __builtin_amdgcn_readfirstlane(M - m0) <= 32) {
            light_tile<T, CFG, B_KMAJOR, EPI, GS>(p, ra_rs, rb_rs, e, M, N, K, m0, n0,
                                                   parts ? tm : 0, parts ? lsplit : 1, buf0,
                                                   buf1, buf2, buf3, buf4);
            return true;
        }
    }
    // Gathered A rows (the tile's rows, fixed over the k loop): each lane's
    // row offsets in x, read once. Gathered B k rows (new ones every stage):
    // the expert's token list in LDS, each lane's offsets for the next
    // stage read one stage ahead.
    using DA_ = DmaStage<BM_, A_KMAJOR, KB, T::NT>;
    using DB_ = DmaStage<BN_, B_KMAJOR, KB, T::NT>;
    int arow[GS == 1 ? DA_::PER : 1];
    uint32_t bk[GS == 2 ? DB_::PER : 1], bcol[GS == 2 ? DB_::PER : 1];
    if constexpr (GS == 1) {
#pragma unroll
        for (int q = 0; q < DA_::PER; ++q) {
            const int r = DA_::lane_row(q);
            arow[q] = m0 + r < M ? p.tok[e * p.tok_estride + m0 + r] * p.a.ld : -1;
        }
    } else if constexpr (GS == 2) {
        // the expert's k rows as byte offsets of their rows of x, and the
        // sentinel past K up to the last row the ring prefetches (so the
        // stage loop tests no bound)
        const int kfill = ((K + NS * KB - 1) / (NS * KB) + 1) * NS * KB;
        for (int i = threadIdx.x; i < kfill; i += T::NT)
            tok_s[i] = i < K ? static_cast<uint32_t>(p.tok[e * p.tok_estride + i]) *
                                   (2u * static_cast<uint32_t>(p.b.ld))
                             : kGatherSentinel;
        __syncthreads();
        DB_::krow_cols(n0, N, bcol);
#pragma unroll
        for (int q = 0; q < DB_::PER; ++q) bk[q] = tok_s[DB_::lane_row(q)];
    }
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / T::WGN, wn = wave % T::WGN;
    // 32-row blocks of this wave's rows that lie inside M: an expert with a
    // few rows (a light expert under a skewed load) runs the matrix-core
    // products, fragment reads and epilogue of those blocks only
    const int fm_live = __builtin_amdgcn_readfirstlane(
        min(FM, max(0, (M - m0 - wm * T::WM + 31) / 32)));
    // weight-gradient GEMMs: the first n-tile also sums its A rows (bias grad);
    // thread t adds row t % BM over k slice t / BM of each stage
    const bool row_sum = CFG::F32_OUT && p.bsum != nullptr && tn == 0;
    constexpr int RS_SPLIT = CFG::F32_OUT ? NT / BM_ : 1;
    constexpr int RS_K = KB / RS_SPLIT;
    float rsum = 0.0f;

    f32x16 acc[FM][FN];

    using DA = DmaStage<BM_, A_KMAJOR, KB, NT>;
    using DB = DmaStage<BN_, B_KMAJOR, KB, NT>;
    using RA = RegStage<BM_, A_KMAJOR, KB, NT>;
    using RB = RegStage<BN_, B_KMAJOR, KB, NT>;
    // DMA wave instructions per stage; stage kt + 1 has landed once at most
    // NS - 2 later stages are still in flight
    constexpr int L = DA::PER + DB::PER;
    constexpr int WAIT_IMM = VmWait<MODE == STAGE_DMA && !T::PAIR ? (NS - 2) * L : 0>::imm;
    // A k-major A operand's DMA blocks of wave w hold rows [w BM / NW, (w + 1)
    // BM / NW) of the tile: a wave whose rows all lie past M (an expert with
    // few rows) issues none of its A loads (those rows are never read: their
    // products are skipped) and counts only its B loads in its waits
    constexpr bool SKIP_A = A_KMAJOR && MODE == STAGE_DMA && !T::PAIR;
    constexpr int WAIT_IMM_B = VmWait<SKIP_A ? (NS - 2) * DB::PER : 0>::imm;
    const bool skip_a =
        SKIP_A && __builtin_amdgcn_readfirstlane(m0 + wave * (BM_ / T::NW)) >= M;
    // paired fetch: after an even stage the pair issued in it is in flight,
    // after an odd stage the second half of the previous pair
    constexpr int WAIT_EVEN = VmWait<T::PAIR ? 2 * L : 0>::imm;
    constexpr int WAIT_ODD = VmWait<T::PAIR ? L : 0>::imm;
    BiasRegs<T, EPI> bias;
    bias.load(p, e, N, n0, wn, lane);
    const int nk = (K + KB - 1) / KB;
    const int nk_ring = (nk + NS - 1) / NS * NS;
    Frags<T, A_KMAJOR, B_KMAJOR, MODE> f0, f1;
    uint4 ra[MODE == STAGE_REG ? RA::V : 1], rb[MODE == STAGE_REG ? RB::V : 1];

    auto issue = [&](int kt, uint16_t* dst) {
        if (!skip_a) {
            if constexpr (GS == 1) {
                DA::issue_rows(ra_rs, arow, kt * KB, K, dst);
            } else {
                DA::issue(ra_rs, p.a.ld, m0, M, kt * KB, K, dst);
            }
        }
        if constexpr (GS == 2) {
            DB::issue_krows(rb_rs, bk, bcol, dst + AE);
            // stages are issued in order: the next one's k rows
#pragma unroll
            for (int q = 0; q < DB::PER; ++q) bk[q] = tok_s[(kt + 1) * KB + DB::lane_row(q)];
        } else {
            DB::issue(rb_rs, p.b.ld, n0, N, kt * KB, K, dst + AE);
        }
    };
    // wait until stage kt + 1 has landed (this wave's share of it)
    auto wait_ring = [&]() {
        if (skip_a) __builtin_amdgcn_s_waitcnt(WAIT_IMM_B);
        else __builtin_amdgcn_s_waitcnt(WAIT_IMM);
    };
    // the accumulators start from the bias where there is one (added once per
    // output instead of in the epilogue); its loads were issued first, so
    // waiting for them leaves the first stages in flight
    auto init_acc = [&]() {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
            for (int j = 0; j < FN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float b4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                    if constexpr (BiasRegs<T, EPI>::USED) {
                        const uint2 bb = bias.v[j * 4 + q];
                        b4[0] = bf16_to_f32(bb.x & 0xFFFFu);
                        b4[1] = bf16_to_f32(bb.x >> 16);
                        b4[2] = bf16_to_f32(bb.y & 0xFFFFu);
                        b4[3] = bf16_to_f32(bb.y >> 16);
                    }
#pragma unroll
                    for (int r = 0; r < 4; ++r) acc[i][j][4 * q + r] = b4[r];
                }
    };
    if constexpr (MODE == STAGE_DMA) {
        issue(0, buf0);
        if constexpr (T::PAIR) {
            issue(1, buf1);
            init_acc();
            __builtin_amdgcn_s_waitcnt(WAIT_ODD);
        } else {
            if constexpr (NS > 2) issue(1, buf1);
            if constexpr (NS > 3) issue(2, buf2);
            if constexpr (NS > 4) issue(3, buf3);
            init_acc();
            wait_ring();
        }
        ring_barrier();
    } else {
        RA::load(ra_rs, p.a.ld, m0, M, 0, K, ra);
        RB::load(rb_rs, p.b.ld, n0, N, 0, K, rb);
        init_acc();
        RA::store(buf0, ra);
        RB::store(buf0 + AE, rb);
        __syncthreads();
    }
    f0.read(buf0, buf0 + AE, wm, wn, 0, lane, fm_live);

    // stage kt computes from `cur`, refills `tgt` (the buffer of stage kt - 1;
    // paired fetch: at even kt, `tgt` and `tgt2` with stages kt + 2 and kt + 3)
    // and leaves the step-0 fragments of `nxt` in f0
    auto stage = [&](const int kt, uint16_t* cur, uint16_t* nxt, uint16_t* tgt, uint16_t* tgt2,
                     auto parity) {
        constexpr bool EVEN = decltype(parity)::value == 0;
        if constexpr (T::PAIR) {
            if constexpr (EVEN) {
                issue(kt + 2, tgt);
                issue(kt + 3, tgt2);
            }
        } else if constexpr (MODE == STAGE_DMA) {
            issue(kt + NS - 1, tgt);
        } else {
            RA::load(ra_rs, p.a.ld, m0, M, (kt + 1) * KB, K, ra);
            RB::load(rb_rs, p.b.ld, n0, N, (kt + 1) * KB, K, rb);
        }
        const bool live = kt < nk;  // uniform: ring padding stages skip their MFMAs
        if (live) {
            if constexpr (CFG::F32_OUT) {
                if (row_sum) {
                    const int mn = tid % BM_, k0 = (tid / BM_) * RS_K;
#pragma unroll
                    for (int kk = 0; kk < RS_K; ++kk)
                        rsum += bf16_to_f32(cur[lds_off<BM_, false, KB, MODE>(mn, k0 + kk)]);
                }
            }
#pragma unroll
            for (int s = 0; s < KSTEPS - 1; ++s) {
                if (s % 2 == 0) {
                    f1.read(cur, cur + AE, wm, wn, s + 1, lane, fm_live);
                    __builtin_amdgcn_sched_barrier(0);
                    mfma_block(acc, f0, fm_live);
                } else {
                    f0.read(cur, cur + AE, wm, wn, s + 1, lane, fm_live);
                    __builtin_amdgcn_sched_barrier(0);
                    mfma_block(acc, f1, fm_live);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        if constexpr (T::PAIR) {
            __builtin_amdgcn_s_waitcnt(EVEN ? WAIT_EVEN : WAIT_ODD);
            ring_barrier();
        } else if constexpr (MODE == STAGE_DMA) {
            wait_ring();
            ring_barrier();
        } else {
            RA::store(nxt, ra);
            RB::store(nxt + AE, rb);
            __syncthreads();
        }
        if (live) {
            // KSTEPS is even: the last step's fragments are in f1
            f0.read(nxt, nxt + AE, wm, wn, 0, lane, fm_live);
            __builtin_amdgcn_sched_barrier(0);
            mfma_block(acc, f1, fm_live);
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // The ring unrolls NS stages per trip with no conditional stage: a skipped
    // stage would merge a path with loads still in flight into the loop head.
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    for (int kt = 0; kt < nk_ring; kt += NS) {
        if constexpr (NS == 2) {
            stage(kt, buf0, buf1, buf1, buf1, P0{});
            stage(kt + 1, buf1, buf0, buf0, buf0, P1{});
        } else if constexpr (NS == 3) {
            stage(kt, buf0, buf1, buf2, buf2, P0{});
            stage(kt + 1, buf1, buf2, buf0, buf0, P1{});
            stage(kt + 2, buf2, buf0, buf1, buf1, P0{});
        } else if constexpr (NS == 4 && T::PAIR) {
            stage(kt, buf0, buf1, buf2, buf3, P0{});
            stage(kt + 1, buf1, buf2, buf0, buf0, P1{});
            stage(kt + 2, buf2, buf3, buf0, buf1, P0{});
            stage(kt + 3, buf3, buf0, buf0, buf0, P1{});
        } else if constexpr (NS == 4) {
            stage(kt, buf0, buf1, buf3, buf3, P0{});
            stage(kt + 1, buf1, buf2, buf0, buf0, P1{});
            stage(kt + 2, buf2, buf3, buf1, buf1, P0{});
            stage(kt + 3, buf3, buf0, buf2, buf2, P1{});
        } else {
            stage(kt, buf0, buf1, buf4, buf4, P0{});
            stage(kt + 1, buf1, buf2, buf0, buf0, P1{});
            stage(kt + 2, buf2, buf3, buf1, buf1, P0{});
            stage(kt + 3, buf3, buf4, buf2, buf2, P1{});
            stage(kt + 4, buf4, buf0, buf3, buf3, P0{});
        }
    }
    // every wave is done with the operand stages (LDS reads retired, DMA landed)
    if constexpr (MODE == STAGE_DMA) __builtin_amdgcn_s_waitcnt(VmWait<0>::imm);
    else __builtin_amdgcn_s_waitcnt(VmWait<63>::imm);
    ring_barrier();

    // wave w parks its outputs in stage buffer w mod NS (a select over the
    // arrays themselves keeps the accesses in the LDS address space)
    const int eb = wave % NS;
    uint16_t* const ep = eb == 0 ? buf0 : eb == 1 ? buf1 : eb == 2 ? buf2 : eb == 3 ? buf3 : buf4;
    gemm_epilogue<T, CFG, EPI>(p, acc, buf0, ep, rsum, row_sum, e, M, N, m0, n0, fm_live);
    return true;
    };
    bool ran;
    if constexpr (GATHER == 0) ran = tile(std::integral_constant<int, 0>{});
    else if (batch.p[prob].tok != nullptr) ran = tile(std::integral_constant<int, GATHER>{});
    else ran = tile(std::integral_constant<int, 0>{});
    if (!ran) {
        if constexpr (SCHED == 0) return;
        else continue;
    }
    if constexpr (SCHED == 0) break;
    // the next tile's first stages land in the buffers this epilogue staged
    // its outputs in: every wave's LDS accesses are done before any issues
    // them (its output stores stay in flight)
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    }
}

// ------------------------------------------------------------------ f32 FMA path

// f32 activations: 64 x 64 output tiles, four waves, each a 32 x 32 block on
// v_mfma_f32_32x32x2_f32 (f32 products and sums); FK-deep k stages staged in
// LDS as [k][mn] (rows padded by one float), read so that consecutive
// threads load consecutive addresses whatever the operand's layout.
constexpr int FT = 64, FK = 32;
typedef float f32x16_f __attribute__((ext_vector_type(16)));

template <bool KMAJOR>
__device__ __forceinline__ float f32_elem(const float* base, int ld, int mn, int k) {
    return KMAJOR ? base[static_cast<size_t>(mn) * ld + k] : base[static_cast<size_t>(k) * ld + mn];
}

// One FK x FT operand stage (zero outside the operand), in two halves: the
// loads into registers, then the stores into S[k][mn]. k-major operands are
// walked k fastest, mn-major ones mn fastest.
constexpr int kF32Per = FK * FT / 256;

template <bool KMAJOR>
__device__ __forceinline__ void load_f32(float (&v)[kF32Per], const float* base, int ld, int mn0,
                                         int mn_lim, int k0, int k_lim) {
#pragma unroll
    for (int u = 0; u < kF32Per; ++u) {
        const int q = u * 256 + static_cast<int>(threadIdx.x);
        const int kk = KMAJOR ? q % FK : q / FT, mn = KMAJOR ? q / FK : q % FT;
        v[u] = (mn0 + mn < mn_lim && k0 + kk < k_lim) ? f32_elem<KMAJOR>(base, ld, mn0 + mn, k0 + kk)
                                                      : 0.0f;
    }
}

template <bool KMAJOR>
__device__ __forceinline__ void store_f32(float (*S)[FT + 1], const float (&v)[kF32Per]) {
#pragma unroll
    for (int u = 0; u < kF32Per; ++u) {
        const int q = u * 256 + static_cast<int>(threadIdx.x);
        const int kk = KMAJOR ? q % FK : q / FT, mn = KMAJOR ? q / FK : q % FT;
        S[kk][mn] = v[u];
    }
}

// A barrier that waits for this wave's LDS accesses only: the next stage's
// global loads stay in flight across it.
__device__ __forceinline__ void f32_lds_barrier() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt, expcnt not waited for
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

template <bool A_KMAJOR, bool B_KMAJOR, int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs p) {
    __shared__ float As[FK][FT + 1];
    __shared__ float Bs[FK][FT + 1];
    const int e = blockIdx.z;
    const int ne = expert_rows(p.counts, p.G, p.E, e);
    const int M = p.var_k ? p.M : min(ne, p.M);
    const int K = p.var_k ? ne : p.K;
    const int N = p.N;
    const int m0 = blockIdx.y * FT, n0 = blockIdx.x * FT;
    if (m0 >= M) return;
    const float* A = static_cast<const float*>(p.a.base) + e * p.a.estride;
    const float* B = static_cast<const float*>(p.b.base) + e * p.b.estride;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wm = w >> 1, wn = w & 1;
    const int r = lane & 31, kh = lane >> 5;
    f32x16_f acc;
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
    // the next stage's loads are issued before this stage's products and
    // land in registers while they run
    float va[kF32Per], vb[kF32Per];
    load_f32<A_KMAJOR>(va, A, p.a.ld, m0, M, 0, K);
    load_f32<B_KMAJOR>(vb, B, p.b.ld, n0, N, 0, K);
    for (int k0 = 0; k0 < K; k0 += FK) {
        store_f32<A_KMAJOR>(As, va);
        store_f32<B_KMAJOR>(Bs, vb);
        f32_lds_barrier();
        if (k0 + FK < K) {
            load_f32<A_KMAJOR>(va, A, p.a.ld, m0, M, k0 + FK, K);
            load_f32<B_KMAJOR>(vb, B, p.b.ld, n0, N, k0 + FK, K);
        }
        // A[m][k = 2 s + kh], B[k][n]: lane l supplies row / column l % 32
#pragma unroll
        for (int s2 = 0; s2 < FK / 2; ++s2)
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(As[2 * s2 + kh][32 * wm + r],
                                                       Bs[2 * s2 + kh][32 * wn + r], acc, 0, 0, 0);
        f32_lds_barrier();
    }
    // register i of lane l: row 8 (i / 4) + 4 (l / 32) + i % 4, column l % 32
    const int n = n0 + 32 * wn + r;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int m = m0 + 32 * wm + 8 * (i / 4) + 4 * kh + (i % 4);
        if (m >= M || n >= N) continue;
        const size_t o = e * p.out_estride + static_cast<size_t>(m) * p.ldo + n;
        float v = acc[i];
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

constexpr int kNumCUs = 256;

// One launch over `n` (1 or 2) problems; grid_m_rows[i] bounds problem i's m.
template <class T, bool AK, bool BK_, int EPI, int GATHER = 0>
void launch_bf16(const Dims& D, const GemmArgs* a, const int* grid_m_rows, int n, int sched,
                 hipStream_t st) {
    GemmBatch b{};
    for (int i = 0; i < n; ++i) {
        b.p[i] = a[i];
        b.tiles_m[i] = static_cast<int>(cdiv(grid_m_rows[i], T::BM));
        b.tiles_n[i] = static_cast<int>(cdiv(a[i].N, T::BN));
        b.total[i] = D.E * b.tiles_m[i] * b.tiles_n[i];
    }
    // blocks resident on one XCD: 32 CUs x blocks per CU. A single problem
    // with both operands k-major whose experts span at most 8 m-tiles is
    // dealt a whole m-column of one expert per chunk (each XCD streams one
    // expert's row panels past four of its weight panels; measured faster for
    // the forward GEMMs, slower for the transposed-weight ones); otherwise
    // patches of 4 m-tiles.
    const int one_col = AK && BK_ && n == 1 && b.tiles_m[0] <= 8 ? b.tiles_m[0] : 0;
    b.group_m = one_col ? one_col : (T::WAVES_PER_EU == 2 && T::NW == 4 ? 8 : 4);
    b.chunk = 4 * b.group_m;
    // (the spread row GEMMs take one chunk more per XCD: splitting the tiles
    // into two classes can leave a partial chunk in each)
    const int spread = EPI == EPI_BIAS || EPI == EPI_STORE ? 1 : 0;
    b.per_xcd = static_cast<int>(cdiv(b.total[0] + b.total[1], 8 * b.chunk) + spread) * b.chunk;
    if (sched && GATHER == 0) {
        // persistent blocks under quotas: as many as are resident at once
        // (one per CU for the 8-wave tiles, two for the 4-wave ones)
        const int resident = kNumCUs * (T::NW == 8 ? 1 : T::WAVES_PER_EU);
        const int grid = min(8 * b.per_xcd, resident);
        gemm_bf16_kernel<T, AK, BK_, EPI, 1><<<grid, T::NT, 0, st>>>(b);
    } else {
        gemm_bf16_kernel<T, AK, BK_, EPI, 0, GATHER><<<8 * b.per_xcd, T::NT, 0, st>>>(b);
    }
}

template <class T, bool AK, bool BK_, int EPI, int GATHER = 0>
void launch_bf16(const Dims& D, const GemmArgs& a, int grid_m_rows, int sched, hipStream_t st) {
    launch_bf16<T, AK, BK_, EPI, GATHER>(D, &a, &grid_m_rows, 1, sched, st);
}

// Tilings (BM, BN, waves, KB, stages, staging).
using TileBig = Tile<256, 256, 2, 4, 32, 4, STAGE_DMA>;    // 8 waves, one block per CU
using TileNarrow = Tile<256, 192, 4, 2, 64, 2, STAGE_DMA>; // 8 waves, 3/4 of TileBig's columns
using TileSmall = Tile<128, 128, 2, 2, 32, 4, STAGE_DMA>;  // 4 waves, two blocks per CU
// TileBig with 64-deep stages in a ring of two: half the stage barriers per
// k, one stage in flight instead of three. For the f-wide row GEMMs (short
// k = d, heavy epilogues) measured 1.3-1.5% faster per step at ViT-B/16 and
// the 17-task pool and even at ViT-L/16; for the d-wide ones (k = f) the
// forward 0.743 -> 0.722 ms at wide E = 32 and 0.312 -> 0.307 at ViT-L/16;
// for the batched weight gradients the backward 0.629 -> 0.625 ms at
// ViT-L/16 (no spill, against one with TileBig), the other workloads
// unchanged. So every 256 x 256 launch takes TileDeep; TileBig (the 32-deep
// ring of four) is the baseline these measurements and TileNarrow refer to.
using TileDeep = Tile<256, 256, 2, 4, 64, 2, STAGE_DMA>;

// Work of a launch in units of one CU's time: rounds of one-block-per-CU
// waves times the tile's area (relative cost per tile area `eff`).
double tile_cost(long long tiles, int bm, int bn, double eff) {
    return static_cast<double>((tiles + kNumCUs - 1) / kNumCUs) * bm * bn * eff;
}

template <bool AK, bool BK_, int EPI, int GATHER = 0>
void launch_gemm(const Dims& D, const GemmArgs& a, int grid_m_rows, int sched, hipStream_t st) {
    if (D.dtype == VMOE_BF16) {
        // 256 x 256 tiles (half the operand bytes per flop of 128 x 128) with
        // 64-deep stages (TileDeep) for the GEMMs whose m is the expert's rows.
        // (bf16 weight gradients run batched in ffn_bwd_launch; this EPI_F32
        // case only serves other callers.)
        if constexpr (EPI == EPI_F32) {
            launch_bf16<TileSmall, AK, BK_, EPI, GATHER>(D, a, grid_m_rows, sched, st);
        } else if constexpr (EPI == EPI_BIAS || EPI == EPI_STORE) {
            // Narrow outputs (N = d_model) give few tiles: 192-column tiles fill
            // more CUs when that saves a round (two-stage 64-deep ring, a few
            // per cent slower per tile)
            const long long tm = cdiv(grid_m_rows, 256);
            const double big = tile_cost(D.E * tm * cdiv(a.N, 256), 256, 256, 1.0);
            const double narrow = tile_cost(D.E * tm * cdiv(a.N, 192), 256, 192, 1.05);
            if (narrow < big)
                launch_bf16<TileNarrow, AK, BK_, EPI, GATHER>(D, a, grid_m_rows, sched, st);
            else
                launch_bf16<TileDeep, AK, BK_, EPI, GATHER>(D, a, grid_m_rows, sched, st);
        } else {
            launch_bf16<TileDeep, AK, BK_, EPI, GATHER>(D, a, grid_m_rows, sched, st);
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

// A second stream per GPU (default priority, non-blocking) and two events,
// made on first use, for launches that may run beside the caller's stream:
// the caller's stream records `fork`, the side stream waits for it, takes
// its launches and records `join`, which the caller's stream waits for, so
// the call still completes in its stream's order (and a captured stream
// captures the side stream's work as a branch of its graph).
struct SideStream {
    hipStream_t s = nullptr;
    hipEvent_t fork = nullptr, join = nullptr;
};
constexpr int kMaxSideDevices = 64;
std::mutex side_mu;
SideStream side_tab[kMaxSideDevices];
// held by a call from its fork to its join, so calls from several host
// threads never interleave their event records and waits
std::mutex side_seq_mu;

// The current GPU's side stream, or null fields on a HIP error (the caller
// then runs everything on its own stream).
SideStream side_stream() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxSideDevices) return {};
    std::lock_guard<std::mutex> lock(side_mu);
    SideStream& t = side_tab[dev];
    if (t.s == nullptr) {
        SideStream n;
        if (hipStreamCreateWithFlags(&n.s, hipStreamNonBlocking) != hipSuccess) return {};
        if (hipEventCreateWithFlags(&n.fork, hipEventDisableTiming) != hipSuccess ||
            hipEventCreateWithFlags(&n.join, hipEventDisableTiming) != hipSuccess) {
            if (n.fork) (void)hipEventDestroy(n.fork);
            (void)hipStreamDestroy(n.s);
            return {};
        }
        t = n;
    }
    return t;
}

// One wave: the device fill-clamp-refill of n experts (the routine the
// quota-scheduled GEMMs run), for comparison with the host routine.
__global__ __launch_bounds__(64) void fcr_kernel(int n, const int32_t* __restrict__ mn,
                                                 const int32_t* __restrict__ sat,
                                                 const double* __restrict__ coef, int budget,
                                                 int32_t* __restrict__ units) {
    const int lane = threadIdx.x;
    const int u = fill_clamp_refill_wave(n, lane < n ? mn[lane] : 0, lane < n ? sat[lane] : 0,
                                         lane < n ? coef[lane] : 0.0, budget);
    if (lane < n) units[lane] = u;
}

}  // namespace

vmoe_status fcr_device_launch(int n, const int32_t* mn, const int32_t* sat, const double* coef,
                              int budget, int32_t* units, hipStream_t st) {
    if (n > 0) fcr_kernel<<<1, 64, 0, st>>>(n, mn, sat, coef, budget, units);
    return launch_status();
}

vmoe_status ffn_fwd_launch(const Dims& D, const void* xe, const int32_t* counts, const void* w1,
                           const void* b1, const void* w2, const void* b2, void* act,
                           void* act_grad, void* ye, int sched, const int32_t* row_token,
                           hipStream_t st) {
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
    if (row_token != nullptr) {
        // dispatch fused into the loads: row r of expert e is x[row_token[e, r]]
        g1.a = Operand{xe, 0, D.d};
        g1.tok = row_token;
        g1.tok_estride = rows;
        g1.gather_bytes = static_cast<long long>(D.N) * D.d * 2;
        launch_gemm<true, true, EPI_FWD1, 1>(D, g1, static_cast<int>(rows), sched, st);
    } else {
        launch_gemm<true, true, EPI_FWD1>(D, g1, static_cast<int>(rows), sched, st);
    }
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
    launch_gemm<true, true, EPI_BIAS>(D, g2, static_cast<int>(rows), sched, st);
    return launch_status();
}

vmoe_status ffn_bwd_launch(const Dims& D, const void* xe, const int32_t* counts, const void* w1,
                           const void* w2, const void* act, const void* act_grad, const void* dye,
                           void* dh, void* dxe, float* dw1, float* db1, float* dw2, float* db2,
                           int sched, const int32_t* row_token, hipStream_t st) {
    const long long rows = D.rows_per_expert();
    if (D.E == 0) return VMOE_OK;
    SideStream side;  // set when dxe runs beside the weight gradients
    std::unique_lock<std::mutex> seq;
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
        launch_gemm<true, false, EPI_GELU_GRAD>(D, g, static_cast<int>(rows), sched, st);
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
        // dxe and the weight gradients both read only dH and the layer's saved
        // tensors: dxe runs on the side stream beside them, so the weight-
        // gradient blocks take the CUs that its partly filled tiles and last
        // round leave idle (bf16, one-tile-per-block schedule, 16 or more
        // experts: measured 0.90 -> 0.81 ms on the 17-task pool, 1.18 -> 1.14
        // at E = 32; with 8 evenly loaded experts every tile is full and the
        // two launches only contend, 0.33 -> 0.34 ms at ViT-B/16)
        if (D.dtype == VMOE_BF16 && sched == 0 && D.E >= 16) {
            seq = std::unique_lock<std::mutex>(side_seq_mu);
            side = side_stream();
            if (side.s != nullptr && (hipEventRecord(side.fork, st) != hipSuccess ||
                                      hipStreamWaitEvent(side.s, side.fork, 0) != hipSuccess))
                side = SideStream{};
        }
        launch_gemm<true, false, EPI_STORE>(D, x, static_cast<int>(rows), sched,
                                            side.s != nullptr ? side.s : st);
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
    if (row_token != nullptr) {
        // xe rows gathered from x: row r of expert e is x[row_token[e, r]]
        v.b = Operand{xe, 0, D.d};
        v.tok = row_token;
        v.tok_estride = rows;
        v.gather_bytes = static_cast<long long>(D.N) * D.d * 2;
    }
    if (D.dtype == VMOE_BF16) {
        // both weight gradients in one launch (same kernel, independent tiles),
        // with the tiling of the least cost in rounds x tile area (128 x 128
        // tiles run two per CU and cost a little more per flop)
        const GemmArgs both[2] = {w, v};
        const int rows_m[2] = {D.d, D.f};
        auto tiles = [&](int bm, int bn) {
            return D.E * (static_cast<long long>(cdiv(D.d, bm)) * cdiv(D.f, bn) +
                          static_cast<long long>(cdiv(D.f, bm)) * cdiv(D.d, bn));
        };
        const double small = tile_cost((tiles(128, 128) + 1) / 2, 256, 128, 1.15);
        const double narrow = tile_cost(tiles(256, 192), 256, 192, 1.05);
        const double big = tile_cost(tiles(256, 256), 256, 256, 1.0);
        // (the gathered input-weight gradient takes the same tiling, so its
        // results, bias-gradient sums included, are the unfused call's bits)
        auto go = [&](auto gather) {
            constexpr int GA = decltype(gather)::value;
            if (narrow <= small && narrow <= big)
                launch_bf16<TileNarrow, false, false, EPI_F32, GA>(D, both, rows_m, 2, sched, st);
            else if (big <= small)
                launch_bf16<TileDeep, false, false, EPI_F32, GA>(D, both, rows_m, 2, sched, st);
            else
                launch_bf16<TileSmall, false, false, EPI_F32, GA>(D, both, rows_m, 2, sched, st);
        };
        if (row_token != nullptr) go(std::integral_constant<int, 2>{});
        else go(std::integral_constant<int, 0>{});
    } else {
        launch_gemm<false, false, EPI_F32>(D, w, D.d, 0, st);
        launch_gemm<false, false, EPI_F32>(D, v, D.f, 0, st);
    }
    if (side.s != nullptr) {
        // the call ends in its stream's order: after the side stream's dxe
        const vmoe_status ls = launch_status();
        if (hipEventRecord(side.join, side.s) != hipSuccess ||
            hipStreamWaitEvent(st, side.join, 0) != hipSuccess)
            return VMOE_ERR_HIP;
        if (ls != VMOE_OK) return ls;
    }
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
