// Weight and bias gradients of a Dyad layer on gfx950 matrix cores.
//
// dW_c[g][j][k] = sum_m dZ[m][row_c(g, j)] * X[m][col_c(g, k)] is, for each
// component c and group g, a GEMM whose reduction runs over the M tokens:
// A = dZ^T restricted to the group's rows, B = X^T restricted to its columns.
//
// Work split.  A workgroup owns one (component, group) pair, a BJ x BK tile of
// that group's weight block and one contiguous range of tokens (a "split").
// Splits are dealt so that every workgroup of one split runs on the same XCD:
// the split's slice of dZ and X is then fetched from HBM once and served to
// all of them from that XCD's L2.  Each workgroup writes fp32 partial sums to
// the workspace; a second kernel adds the splits in a fixed order, so the
// result is bitwise reproducible.
//
// Pipeline.  Stages of 32 tokens, double-buffered in LDS with the next stage's
// loads in flight, exactly as in the grouped GEMM, so the MFMA consumes 16x32
// fragments from 64-byte swizzled LDS rows (row = weight row j or column k,
// 32 tokens per row).  Both operands are token-major in memory, so each thread
// loads 8x8 blocks (8 tokens x 8 consecutive columns, eight 16-byte loads) and
// transposes them in registers (v_perm_b32) on the way into LDS.
//
// Strided operands.  The BlockTrans component reads dZ columns j*D + g (output
// transpose) or X columns k*D + g (input transpose).  Such a side loads the
// 16-byte vectors that contain its columns -- 8/D consecutive j (or k) per
// vector for D <= 8 -- and keeps the group's residue only.
//
// Bias gradient.  Workgroups of component 1 whose column tile is the first sum
// their dZ rows over the split's tokens straight from LDS; every dZ column is
// covered by exactly one such workgroup.
#include "dyad_internal.h"
#include "mfma_common.h"

namespace dyad {
namespace {

constexpr int kThreads = 256;

struct DwArgs {
    int64_t M, n_in, n_out, bi, bo;
    const uint16_t *dZ, *X;
    float *part;          // [splits][2][D][bo][bi]
    float *part_db;       // [splits][n_out]
    int64_t tokens_per_split;
    int tiles_j, tiles_k; // tiles per (component, group)
    int splits, splits_per_xcd;
    int want_db;
};

// Column e (0..7, uniform across the workgroup) of an 8x8 bf16 block: one
// branch per value, each a compile-time shuffle.
template <int E = 0>
__device__ __forceinline__ uint4 column_uniform(const uint4 (&r)[8], int e) {
    if constexpr (E < 7) {
        if (e != E) return column_uniform<E + 1>(r, e);
    }
    return column_of(r, E);
}

// One side (A = dZ, B = X) of a workgroup's stage: which source columns it
// loads and where they land in LDS.  `rows` LDS rows (weight rows j or
// columns k of the tile), 32 tokens each.
//   plain:  source column first + row, for row in [0, rows)
//   strided (SPAN): source column (first + row) * D + g
template <int D, bool SPAN, int ROWS, int NSUB>
struct Side {
    // k values (LDS rows) per loaded 16-byte vector, and vectors per 8 tokens
    static constexpr int kPerVec = SPAN ? (D <= 8 ? 8 / D : 1) : 8;
    static constexpr int kVecCols = ROWS / kPerVec;                     // vector columns per token row
    static constexpr int kBlocks = kVecCols * (NSUB * kStageK / 8);     // 8x8 blocks per stage
    static_assert(ROWS % kPerVec == 0, "whole vectors per tile");
};

// A stage is NSUB consecutive 32-token sub-stages (one MFMA K step each), each
// stored as its own [BJ + BK][32] LDS tile.
template <int D, int BJ, int BK, int NSUB>
struct DwCfg {
    static constexpr int kWavesJ = 2, kWavesK = 2;
    static constexpr int WJ = BJ / kWavesJ, WK = BK / kWavesK;
    static constexpr int kSubJ = WJ / 16, kSubK = WK / 16;
    static constexpr int kTokens = NSUB * kStageK;                // tokens per stage
    static constexpr int kSubElems = (BJ + BK) * kStageK;         // bf16 per sub-stage tile
    static constexpr int kStageElems = NSUB * kSubElems;          // bf16 per LDS stage buffer
    static constexpr int kLds = 2 * kStageElems * 2;
    // one workgroup per CU once the accumulators pass 128 per lane
    static constexpr int kOcc = (BJ * BK / 256 > 128 || 2 * kLds > 160 * 1024) ? 1 : 2;
    static_assert(WJ % 16 == 0 && WK % 16 == 0, "whole MFMA blocks per wave");
    static_assert(kLds <= 160 * 1024, "LDS budget");
};

template <int D, int BJ, int BK, int NSUB, bool IN_T, bool OUT_T, bool C2>
__device__ __forceinline__ void dw_tile(const DwArgs &a, unsigned char *smem, int split, int g, int jt, int kt) {
    using C = DwCfg<D, BJ, BK, NSUB>;
    constexpr bool SPAN_A = C2 && OUT_T;    // dZ columns j*D + g
    constexpr bool SPAN_B = C2 && IN_T;     // X columns k*D + g
    using SA = Side<D, SPAN_A, BJ, NSUB>;
    using SB = Side<D, SPAN_B, BK, NSUB>;
    constexpr int kBlkA = SA::kBlocks, kBlk = SA::kBlocks + SB::kBlocks;
    constexpr int kIters = (kBlk + kThreads - 1) / kThreads;

    uint16_t *lds = reinterpret_cast<uint16_t *>(smem);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int j0 = jt * BJ, k0 = kt * BK;
    const int bo = (int)a.bo, bi = (int)a.bi, n_out = (int)a.n_out, n_in = (int)a.n_in;

    const int64_t t_begin = (int64_t)split * a.tokens_per_split;
    int64_t t_end = t_begin + a.tokens_per_split;
    if (t_end > a.M) t_end = a.M;
    const int stages = t_end > t_begin ? (int)((t_end - t_begin + C::kTokens - 1) / C::kTokens) : 0;

    // first source column of each side (plain: column of row 0; strided: the
    // vector holding row 0's column)
    const int colA = SPAN_A ? j0 * D + (D >= 16 ? (g & ~7) : 0) : g * bo + j0;
    const int colB = SPAN_B ? k0 * D + (D >= 16 ? (g & ~7) : 0) : g * bi + k0;
    // element of a strided vector holding row t (t < kPerVec): (t * D + g) & 7
    const int gsel = g & 7;

    // per-thread block: side, token block tb, vector column vc; byte offset of
    // its first token row within a stage
    uint32_t voff[kIters];
#pragma unroll
    for (int q = 0; q < kIters; ++q) {
        const int bid = (tid + q * kThreads) % kBlk;
        const bool sideA = bid < kBlkA;
        const int local = sideA ? bid : bid - kBlkA;
        const int vcols = sideA ? SA::kVecCols : SB::kVecCols;
        const int vc = local % vcols, tb = local / vcols;
        const int ld = sideA ? n_out : n_in;
        const bool span = sideA ? SPAN_A : SPAN_B;
        const int col = (sideA ? colA : colB) + (span ? vc * (D <= 8 ? 8 : D) : vc * 8);
        voff[q] = (uint32_t)(tb * 8) * (uint32_t)ld * 2u + (uint32_t)col * 2u;
    }

    f32x4_t acc[C::kSubJ][C::kSubK];
#pragma unroll
    for (int i = 0; i < C::kSubJ; ++i)
#pragma unroll
        for (int j = 0; j < C::kSubK; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    uint4 reg[kIters][8];

    const bool do_db = !C2 && a.want_db && kt == 0;
    // half-row hr = tid + q*256 (q < kDbIters) of a sub-stage's dZ tile: tokens 16*(hr & 1)..+16 of row hr >> 1
    constexpr int kDbIters = (2 * BJ + kThreads - 1) / kThreads;
    float dbacc[kDbIters];
#pragma unroll
    for (int q = 0; q < kDbIters; ++q) dbacc[q] = 0.f;

    // ---- global -> registers: stage s's 8x8 blocks.  The buffer is rebased at
    // the stage's first token and ends at the split's end, so tokens past it
    // read as zero.
    auto fetch = [&](int s) {
        const int64_t tok = t_begin + (int64_t)s * C::kTokens;
        const int64_t left = t_end - tok;
        const uint32_t rows = (uint32_t)(left < C::kTokens ? left : C::kTokens);
        const __amdgpu_buffer_rsrc_t rA = buffer_rsrc(a.dZ + tok * n_out, rows * (uint32_t)n_out * 2u);
        const __amdgpu_buffer_rsrc_t rB = buffer_rsrc(a.X + tok * n_in, rows * (uint32_t)n_in * 2u);
#pragma unroll
        for (int q = 0; q < kIters; ++q) {
            const int bid = tid + q * kThreads;
            if (kBlk % kThreads == 0 || bid < kBlk) {
                const bool sideA = bid < kBlkA;
                const uint32_t ld2 = (uint32_t)(sideA ? n_out : n_in) * 2u;
#pragma unroll
                for (int t = 0; t < 8; ++t) reg[q][t] = bload16(sideA ? rA : rB, voff[q] + t * ld2, 0);
            }
        }
    };

    // ---- registers -> LDS: transpose each block; a strided block keeps only
    // the group's residue
    auto stash = [&](uint16_t *buf) {
#pragma unroll
        for (int q = 0; q < kIters; ++q) {
            const int bid = tid + q * kThreads;
            if (kBlk % kThreads == 0 || bid < kBlk) {
                const bool sideA = bid < kBlkA;
                const int local = sideA ? bid : bid - kBlkA;
                const int vcols = sideA ? SA::kVecCols : SB::kVecCols;
                const int vc = local % vcols, tb = local / vcols;
                // token block tb: sub-stage tb / 4, 16-byte chunk tb % 4 of its rows
                uint16_t *dst = buf + (tb >> 2) * C::kSubElems + (sideA ? 0 : BJ * kStageK);
                const int chunk = tb & 3;
                const bool span = sideA ? SPAN_A : SPAN_B;
                if (!span) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        *reinterpret_cast<uint4 *>(dst + lds_off(vc * 8 + e, chunk)) = column_of(reg[q], e);
                } else {
                    constexpr int kpv = D <= 8 ? 8 / D : 1;
#pragma unroll
                    for (int t = 0; t < kpv; ++t)
                        *reinterpret_cast<uint4 *>(dst + lds_off(vc * kpv + t, chunk)) =
                            column_uniform(reg[q], ((t * D) & 7) + (D <= 8 ? g : gsel));
                }
            }
        }
    };

    const int wj0 = (wave / C::kWavesK) * C::WJ, wk0 = (wave % C::kWavesK) * C::WK;
    auto compute = [&](const uint16_t *stage) {
#pragma unroll
        for (int sub = 0; sub < NSUB; ++sub) {
            const uint16_t *buf = stage + sub * C::kSubElems;
            const uint16_t *bufB = buf + BJ * kStageK;
            const int lr = lane & 15, lc = lane >> 4;
            bf16x8_t af[C::kSubJ];
#pragma unroll
            for (int i = 0; i < C::kSubJ; ++i)
                af[i] = *reinterpret_cast<const bf16x8_t *>(buf + lds_off(wj0 + i * 16 + lr, lc));
#pragma unroll
            for (int j = 0; j < C::kSubK; ++j) {
                const bf16x8_t bf = *reinterpret_cast<const bf16x8_t *>(bufB + lds_off(wk0 + j * 16 + lr, lc));
#pragma unroll
                for (int i = 0; i < C::kSubJ; ++i)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf, acc[i][j], 0, 0, 0);
            }
            if (do_db) {
#pragma unroll
                for (int q = 0; q < kDbIters; ++q) {
                    const int hr = tid + q * kThreads, row = hr >> 1, h = hr & 1;
                    if (hr < 2 * BJ) {
#pragma unroll
                        for (int c = 0; c < 2; ++c) {
                            const uint4 w = *reinterpret_cast<const uint4 *>(buf + lds_off(row, 2 * h + c));
#pragma unroll
                            for (int e = 0; e < 8; ++e) dbacc[q] += unpack_bf16(word_of(w, e >> 1), e & 1);
                        }
                    }
                }
            }
        }
    };

    auto buf = [&](int s) -> uint16_t * { return lds + (s & 1) * C::kStageElems; };
    if (stages > 0) {
        fetch(0);
        stash(buf(0));
        if (stages > 1) fetch(1);
        __syncthreads();
        int s = 0;
        for (; s + 2 < stages; ++s) {
            stash(buf(s + 1));
            fetch(s + 2);
            compute(buf(s));
            __syncthreads();
        }
        if (s + 1 < stages) {
            stash(buf(s + 1));
            compute(buf(s));
            __syncthreads();
            ++s;
        }
        compute(buf(s));
    }

    // partial sums -> workspace [split][comp][g][j][k]
    const int64_t per_comp = (int64_t)(a.bo * a.bi) * (int64_t)(a.n_out / a.bo);
    float *dst = a.part + ((int64_t)split * 2 + (C2 ? 1 : 0)) * per_comp + (int64_t)g * bo * bi;
#pragma unroll
    for (int i = 0; i < C::kSubJ; ++i)
#pragma unroll
        for (int j = 0; j < C::kSubK; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int jj = j0 + wj0 + i * 16 + (lane >> 4) * 4 + v;
                const int kk = k0 + wk0 + j * 16 + (lane & 15);
                dst[(int64_t)jj * bi + kk] = acc[i][j][v];
            }
    if (do_db) {
        // the two halves of each row sit in adjacent lanes
#pragma unroll
        for (int q = 0; q < kDbIters; ++q) {
            const int hr = tid + q * kThreads;
            const float other = __shfl_xor(dbacc[q], 1);
            if (hr < 2 * BJ && (hr & 1) == 0)
                a.part_db[(int64_t)split * n_out + g * bo + j0 + (hr >> 1)] = dbacc[q] + other;
        }
    }
}

template <int D, int BJ, int BK, int NSUB, bool IN_T, bool OUT_T>
__global__ void __launch_bounds__(kThreads, (DwCfg<D, BJ, BK, NSUB>::kOcc)) dyad_dw_mfma(DwArgs a) {
    using C = DwCfg<D, BJ, BK, NSUB>;
    __shared__ __attribute__((aligned(16))) unsigned char smem[C::kLds];
    // workgroup -> (split, component, group, j tile, k tile).  With a multiple
    // of 8 splits, XCD x = w % 8 takes splits x, x + 8, ... and one split's
    // tiles are adjacent on it; otherwise splits simply follow each other.
    const int w = blockIdx.x;
    const int tiles = 2 * D * a.tiles_j * a.tiles_k;
    int split, t;
    if (a.splits % 8 == 0) {
        const int x = w & 7, i = w >> 3;
        split = x + 8 * (i / tiles);
        t = i % tiles;
    } else {
        split = w / tiles;
        t = w % tiles;
    }
    const int kt = t % a.tiles_k; t /= a.tiles_k;
    const int jt = t % a.tiles_j; t /= a.tiles_j;
    const int g = t % D, comp = t / D;
    if (split >= a.splits) return;
    if (comp == 0) dw_tile<D, BJ, BK, NSUB, IN_T, OUT_T, false>(a, smem, split, g, jt, kt);
    else dw_tile<D, BJ, BK, NSUB, IN_T, OUT_T, true>(a, smem, split, g, jt, kt);
}

// Adds the splits in order 0..S-1 and writes dW1, dW2 (and db) in bf16.
__global__ void __launch_bounds__(256) dyad_dw_reduce(const float *part, const float *part_db, int splits,
                                                      int64_t per_comp, int64_t n_out, uint16_t *dW1,
                                                      uint16_t *dW2, uint16_t *db) {
    const int64_t n4 = 2 * per_comp / 4;            // float4 groups of the two components
    const int64_t nb4 = db ? n_out / 4 : 0;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n4 + nb4;
         e += (int64_t)gridDim.x * blockDim.x) {
        const bool is_db = e >= n4;
        const int64_t idx = is_db ? (e - n4) * 4 : e * 4;
        const float *src = is_db ? part_db + idx : part + idx;
        const int64_t stride = is_db ? n_out : 2 * per_comp;
        float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int q = 0; q < splits; ++q) {
            const float4 v = *reinterpret_cast<const float4 *>(src + q * stride);
            s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
        }
        uint2 o;
        o.x = pack_bf16(s.x, s.y);
        o.y = pack_bf16(s.z, s.w);
        uint16_t *out = is_db ? db + idx : (idx < per_comp ? dW1 + idx : dW2 + (idx - per_comp));
        *reinterpret_cast<uint2 *>(out) = o;
    }
}

struct DwPlan {
    int BJ, BK, NSUB, occ, tiles_j, tiles_k, splits, splits_per_xcd;
    int64_t tokens_per_split;
};

// Tile candidates for n_dyad D, preferred first: (BJ, BK) weight tile and
// NSUB 32-token sub-stages per pipeline stage.
struct Cand { int D, BJ, BK, NSUB; };
constexpr Cand kCands[] = {
    {1, 128, 128, 1}, {1, 128, 64, 1}, {1, 64, 128, 1}, {1, 64, 64, 1},
    {2, 128, 128, 1}, {2, 128, 64, 1}, {2, 64, 128, 1}, {2, 64, 64, 1},
    {4, 128, 192, 1}, {4, 192, 128, 1}, {4, 128, 128, 1}, {4, 128, 64, 1}, {4, 64, 128, 1}, {4, 64, 64, 1},
    {8, 64, 64, 1}, {16, 64, 64, 1},
};

template <int D, int BJ, int BK, int NSUB>
constexpr int cand_occ() { return DwCfg<D, BJ, BK, NSUB>::kOcc; }

int occ_of(const Cand &c) {
#define DYAD_DW_OCC(D_, J_, K_, N_) if (c.D == D_ && c.BJ == J_ && c.BK == K_ && c.NSUB == N_) return cand_occ<D_, J_, K_, N_>();
    DYAD_DW_OCC(4, 128, 192, 1) DYAD_DW_OCC(4, 192, 128, 1)
#undef DYAD_DW_OCC
    return 2;
}

bool choose(const DwPass &p, DwPlan &pl) {
    if (p.dtype != kBF16 || p.M <= 0) return false;
    for (const Cand &c : kCands) {
        if (c.D != p.D || p.bo % c.BJ || p.bi % c.BK) continue;
        const int64_t stage_tokens = (int64_t)kStageK * c.NSUB;
        // 32-bit buffer offsets within one stage
        if (stage_tokens * (p.n_in > p.n_out ? p.n_in : p.n_out) * 2 >= ((int64_t)1 << 31)) return false;
        pl.BJ = c.BJ; pl.BK = c.BK; pl.NSUB = c.NSUB; pl.occ = occ_of(c);
        pl.tiles_j = (int)(p.bo / c.BJ);
        pl.tiles_k = (int)(p.bi / c.BK);
        // splits: a multiple of 8 (one token range per XCD and round), enough
        // workgroups to fill every CU's slots once, each split at least four
        // stages long
        const int64_t tiles = 2 * p.D * (int64_t)pl.tiles_j * pl.tiles_k;
        const int64_t slots = 256 * (int64_t)pl.occ;
        // enough tiles fill the GPU without splitting the tokens at all
        int64_t splits = tiles >= slots ? 1 : 8 * ((slots + 8 * tiles - 1) / (8 * tiles));
        const int64_t max_splits = (p.M + 4 * stage_tokens - 1) / (4 * stage_tokens);
        if (splits > max_splits) splits = max_splits;
        if (splits < 1) splits = 1;
        int64_t tps = (p.M + splits - 1) / splits;
        tps = (tps + stage_tokens - 1) / stage_tokens * stage_tokens;
        pl.tokens_per_split = tps;
        pl.splits = (int)((p.M + tps - 1) / tps);
        pl.splits_per_xcd = (pl.splits + 7) / 8;
        if (tiles * pl.splits >= ((int64_t)1 << 31)) return false;
        return true;
    }
    return false;
}

template <int D, int BJ, int BK, int NSUB, bool IN_T, bool OUT_T>
hipError_t launch_dw_cfg(const DwPass &p, const DwPlan &pl, hipStream_t s) {
    DwArgs a;
    a.M = p.M; a.n_in = p.n_in; a.n_out = p.n_out; a.bi = p.bi; a.bo = p.bo;
    a.dZ = static_cast<const uint16_t *>(p.dZ);
    a.X = static_cast<const uint16_t *>(p.X);
    a.part = static_cast<float *>(p.ws);
    a.part_db = a.part + (int64_t)pl.splits * 2 * p.D * p.bo * p.bi;
    a.tokens_per_split = pl.tokens_per_split;
    a.tiles_j = pl.tiles_j; a.tiles_k = pl.tiles_k;
    a.splits = pl.splits; a.splits_per_xcd = pl.splits_per_xcd;
    a.want_db = p.db != nullptr;
    const int64_t tiles = 2 * p.D * (int64_t)pl.tiles_j * pl.tiles_k;
    const int64_t blocks = pl.splits % 8 == 0 ? 8 * tiles * pl.splits_per_xcd : tiles * pl.splits;
    dyad_dw_mfma<D, BJ, BK, NSUB, IN_T, OUT_T><<<(unsigned)blocks, kThreads, 0, s>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t per_comp = p.D * p.bo * p.bi;
    const int64_t work = (2 * per_comp + (p.db ? p.n_out : 0)) / 4;
    int64_t grid = (work + 255) / 256;
    if (grid > 8192) grid = 8192;
    if (grid < 1) grid = 1;
    dyad_dw_reduce<<<(unsigned)grid, 256, 0, s>>>(a.part, a.part_db, pl.splits, per_comp, p.n_out,
                                                  static_cast<uint16_t *>(p.dW1),
                                                  static_cast<uint16_t *>(p.dW2),
                                                  static_cast<uint16_t *>(p.db));
    return hipGetLastError();
}

template <bool IN_T, bool OUT_T>
hipError_t launch_dw_variant(const DwPass &p, const DwPlan &pl, hipStream_t s) {
#define DYAD_DW_CASE(D_, J_, K_, N_)                                             \
    if (p.D == D_ && pl.BJ == J_ && pl.BK == K_ && pl.NSUB == N_)                \
        return launch_dw_cfg<D_, J_, K_, N_, IN_T, OUT_T>(p, pl, s);
    DYAD_DW_CASE(1, 128, 128, 1) DYAD_DW_CASE(1, 128, 64, 1) DYAD_DW_CASE(1, 64, 128, 1) DYAD_DW_CASE(1, 64, 64, 1)
    DYAD_DW_CASE(2, 128, 128, 1) DYAD_DW_CASE(2, 128, 64, 1) DYAD_DW_CASE(2, 64, 128, 1) DYAD_DW_CASE(2, 64, 64, 1)
    DYAD_DW_CASE(4, 128, 192, 1) DYAD_DW_CASE(4, 192, 128, 1) DYAD_DW_CASE(4, 128, 128, 1)
    DYAD_DW_CASE(4, 128, 64, 1) DYAD_DW_CASE(4, 64, 128, 1) DYAD_DW_CASE(4, 64, 64, 1)
    DYAD_DW_CASE(8, 64, 64, 1) DYAD_DW_CASE(16, 64, 64, 1)
#undef DYAD_DW_CASE
    return hipErrorNotSupported;
}

}  // namespace

size_t mfma_dw_workspace(const DwPass &p) {
    DwPlan pl;
    if (!choose(p, pl)) return 0;
    return (size_t)pl.splits * (size_t)(2 * p.D * p.bo * p.bi + p.n_out) * sizeof(float);
}

hipError_t launch_mfma_dw(const DwPass &p, hipStream_t s) {
    DwPlan pl;
    if (!choose(p, pl)) return hipErrorNotSupported;
    if (p.in_t && !p.out_t) return launch_dw_variant<true, false>(p, pl, s);
    if (!p.in_t && p.out_t) return launch_dw_variant<false, true>(p, pl, s);
    if (p.in_t && p.out_t) return launch_dw_variant<true, true>(p, pl, s);
    return hipErrorNotSupported;
}

}  // namespace dyad
