// Weight and bias gradients of a Dyad layer on gfx950 matrix cores.
//
// dW_c[g][j][k] = sum_m dZ[m][row_c(g, j)] * X[m][col_c(g, k)] is, for each
// component c and group g, a GEMM whose reduction runs over the tokens.
//
// Work split.  A workgroup owns one component c, a range of J weight rows and
// K weight columns, for ALL D groups at once, and one contiguous range of
// tokens (a "split").  Taking every group together means a strided operand --
// dZ columns j*D + g of an output transpose, X columns k*D + g of an input
// transpose -- is read as the contiguous span of D*J (or D*K) columns, every
// element of which belongs to one of the groups: nothing loaded is discarded.
// The unstrided side reads D block slices.  Each split writes fp32 partial sums
// to the workspace; a second kernel adds the splits in a fixed order, so the
// result is bitwise reproducible.
//
// Staging.  Both operands are token-major in memory while the MFMA wants 8
// consecutive tokens per lane, so each thread loads an 8-token x 8-column
// block (eight 16-byte loads), transposes it in registers and writes eight
// 16-byte column vectors into LDS tiles laid out [group][row][token].
//
// Bias gradient.  Workgroups of component 1 with K offset 0 also sum their dZ
// columns over the split's tokens (db partials); every dZ column is covered by
// exactly one such workgroup.
#include "dyad_device.h"
#include "dyad_internal.h"

namespace dyad {
namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

constexpr int kT = 32;               // tokens per stage (one MFMA K step)
constexpr int kRowT = kT + 8;        // LDS row pitch in bf16 (padding)
constexpr int kThreads = 256;

struct DwArgs {
    int64_t M, n_in, n_out, bi, bo;
    const uint16_t *dZ, *X;
    float *part;          // [splits][2][D][bo][bi]
    float *part_db;       // [splits][n_out]
    int64_t tokens_per_split;
    int tiles_j, tiles_k; // per component
    int splits;
    int want_db;
};

__device__ __forceinline__ uint4 ldg16(const uint16_t *p) { return *reinterpret_cast<const uint4 *>(p); }

__device__ __forceinline__ uint32_t word(const uint4 &v, int q) {
    return q == 0 ? v.x : q == 1 ? v.y : q == 2 ? v.z : v.w;
}

// Column e (0..7) of an 8x8 bf16 block given as 8 rows of 8: the 8 row values, packed.
__device__ __forceinline__ uint4 column_of(const uint4 (&r)[8], int e) {
    uint32_t o[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const uint32_t a = word(r[2 * p], e >> 1), b = word(r[2 * p + 1], e >> 1);
        o[p] = (e & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
}

// D groups; per group a J x K output tile; WJ x WK per wave; GPW groups per wave.
template <int D, int J, int K, int WJ, int WK, bool IN_T, bool OUT_T>
struct DwTile {
    static constexpr int kGPW = D >= 4 ? D / 4 : 1;              // groups per wave
    static constexpr int kWPG = D >= 4 ? 1 : 4 / D;              // waves per group
    static constexpr int kWavesK = K / WK;                       // within a group
    static constexpr int kSubJ = WJ / 16, kSubK = WK / 16;
    static constexpr int kRowsA = D * J, kRowsB = D * K;         // LDS rows
    static constexpr int kBlocksA = kRowsA / 8 * (kT / 8);       // 8x8 blocks per stage
    static constexpr int kBlocksB = kRowsB / 8 * (kT / 8);
    static constexpr int kBlocks = kBlocksA + kBlocksB;
    static constexpr int kIters = (kBlocks + kThreads - 1) / kThreads;
    static constexpr int kLds = (kRowsA + kRowsB) * kRowT * 2;
    static_assert(D >= 4 || (J / WJ) * (K / WK) == kWPG, "waves of one group tile it exactly");
    static_assert(D < 4 || (WJ == J && WK == K), "one wave holds whole group tiles");
    static_assert(kLds <= 160 * 1024, "LDS budget");
};

template <int D, int J, int K, int WJ, int WK, bool IN_T, bool OUT_T>
__global__ void __launch_bounds__(kThreads, 1) dyad_dw_mfma(DwArgs a) {
    using T = DwTile<D, J, K, WJ, WK, IN_T, OUT_T>;
    __shared__ __attribute__((aligned(16))) uint16_t lds[(T::kRowsA + T::kRowsB) * kRowT];
    uint16_t *ldsA = lds;                       // [D*J][kRowT]  dZ^T, row = g*J + j
    uint16_t *ldsB = lds + T::kRowsA * kRowT;   // [D*K][kRowT]  X^T,  row = g*K + k

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // block -> (split, component, j tile, k tile); splits of one tile are adjacent
    int b = blockIdx.x;
    const int split = b % a.splits; b /= a.splits;
    const int kt = b % a.tiles_k; b /= a.tiles_k;
    const int jt = b % a.tiles_j; b /= a.tiles_j;
    const int comp = b + 1;
    const int64_t j0 = (int64_t)jt * J, k0 = (int64_t)kt * K;
    const int64_t t_begin = (int64_t)split * a.tokens_per_split;
    int64_t t_end = t_begin + a.tokens_per_split;
    if (t_end > a.M) t_end = a.M;
    const int stages = t_end > t_begin ? (int)((t_end - t_begin + kT - 1) / kT) : 0;

    const bool spanA = comp == 2 && OUT_T;   // dZ columns j*D + g
    const bool spanB = comp == 2 && IN_T;    // X columns k*D + g
    const bool do_db = a.want_db && comp == 1 && kt == 0;

    // wave -> groups and sub-tile
    const int wg0 = D >= 4 ? wave * T::kGPW : wave / T::kWPG;
    const int wsub = D >= 4 ? 0 : wave % T::kWPG;
    const int wj0 = (wsub / T::kWavesK) * WJ, wk0 = (wsub % T::kWavesK) * WK;

    f32x4_t acc[T::kGPW][T::kSubJ][T::kSubK];
#pragma unroll
    for (int g = 0; g < T::kGPW; ++g)
#pragma unroll
        for (int i = 0; i < T::kSubJ; ++i)
#pragma unroll
            for (int j = 0; j < T::kSubK; ++j) acc[g][i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    uint4 reg[T::kIters][8];

    // block id -> (side, source column of its first element, token row block)
    // side A: rows of dZ; side B: rows of X.  8 consecutive LDS rows per block
    // in slice mode; 8 consecutive span columns in span mode.
    auto block_src = [&](int bid, bool &sideA, int64_t &col, int &tb, int &r8) {
        sideA = bid < T::kBlocksA;
        const int local = sideA ? bid : bid - T::kBlocksA;
        tb = local % (kT / 8);
        r8 = (local / (kT / 8)) * 8;             // first LDS row (slice) / span column (span)
        if (sideA) {
            if (spanA) col = j0 * D + r8;                              // span columns
            else col = (int64_t)(r8 / J) * a.bo + j0 + (r8 % J);       // group r8/J, rows
        } else {
            if (spanB) col = k0 * D + r8;
            else col = (int64_t)(r8 / K) * a.bi + k0 + (r8 % K);
        }
    };

    auto fetch = [&](int s) {
        const int64_t tok0 = t_begin + (int64_t)s * kT;
#pragma unroll
        for (int it = 0; it < T::kIters; ++it) {
            const int bid = tid + it * kThreads;
            if (bid < T::kBlocks) {
                bool sideA; int64_t col; int tb, r8;
                block_src(bid, sideA, col, tb, r8);
                const uint16_t *base = sideA ? a.dZ : a.X;
                const int64_t ld = sideA ? a.n_out : a.n_in;
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    const int64_t m = tok0 + tb * 8 + t;
                    reg[it][t] = m < t_end ? ldg16(base + m * ld + col) : make_uint4(0, 0, 0, 0);
                }
            }
        }
    };

    auto stash = [&]() {
#pragma unroll
        for (int it = 0; it < T::kIters; ++it) {
            const int bid = tid + it * kThreads;
            if (bid < T::kBlocks) {
                bool sideA; int64_t col; int tb, r8;
                block_src(bid, sideA, col, tb, r8);
                const bool span = sideA ? spanA : spanB;
                const int rows_per_group = sideA ? J : K;
                uint16_t *dst = sideA ? ldsA : ldsB;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    int row;
                    if (span) {
                        const int c = r8 + e;            // span column: group c % D, index c / D
                        row = (c % D) * rows_per_group + c / D;
                    } else {
                        row = r8 + e;
                    }
                    *reinterpret_cast<uint4 *>(dst + row * kRowT + tb * 8) = column_of(reg[it], e);
                }
            }
        }
    };

    // db: threads sum whole LDS rows of the dZ tile (comp 1: row = g*J + j, slice mode)
    constexpr int kDbRows = (T::kRowsA + kThreads - 1) / kThreads;
    float dbacc[kDbRows];
#pragma unroll
    for (int q = 0; q < kDbRows; ++q) dbacc[q] = 0.f;

    auto compute = [&]() {
        const int kq = (lane >> 4) * 8;
#pragma unroll
        for (int gg = 0; gg < T::kGPW; ++gg) {
            const int g = wg0 + gg;
            bf16x8_t bf[T::kSubK];
#pragma unroll
            for (int j = 0; j < T::kSubK; ++j)
                bf[j] = *reinterpret_cast<const bf16x8_t *>(
                    ldsB + (g * K + wk0 + j * 16 + (lane & 15)) * kRowT + kq);
#pragma unroll
            for (int i = 0; i < T::kSubJ; ++i) {
                const bf16x8_t af = *reinterpret_cast<const bf16x8_t *>(
                    ldsA + (g * J + wj0 + i * 16 + (lane & 15)) * kRowT + kq);
#pragma unroll
                for (int j = 0; j < T::kSubK; ++j)
                    acc[gg][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bf[j], acc[gg][i][j], 0, 0, 0);
            }
        }
        if (do_db) {
#pragma unroll
            for (int q = 0; q < kDbRows; ++q) {
                const int row = tid + q * kThreads;
                if (row < T::kRowsA) {
#pragma unroll
                    for (int v = 0; v < kT / 8; ++v) {
                        const uint4 w = *reinterpret_cast<const uint4 *>(ldsA + row * kRowT + v * 8);
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const uint32_t d = word(w, e);
                            dbacc[q] += bf16_to_f32((uint16_t)(d & 0xffffu)) + bf16_to_f32((uint16_t)(d >> 16));
                        }
                    }
                }
            }
        }
    };

    if (stages > 0) fetch(0);
    for (int s = 0; s < stages; ++s) {
        __syncthreads();
        stash();
        __syncthreads();
        if (s + 1 < stages) fetch(s + 1);
        compute();
    }

    // partial sums -> workspace [split][comp-1][g][j][k]
    const int64_t per_comp = (int64_t)D * a.bo * a.bi;
    float *dst = a.part + ((int64_t)split * 2 + (comp - 1)) * per_comp;
#pragma unroll
    for (int gg = 0; gg < T::kGPW; ++gg) {
        const int g = wg0 + gg;
#pragma unroll
        for (int i = 0; i < T::kSubJ; ++i)
#pragma unroll
            for (int j = 0; j < T::kSubK; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int64_t jj = j0 + wj0 + i * 16 + (lane >> 4) * 4 + v;
                    const int64_t kk = k0 + wk0 + j * 16 + (lane & 15);
                    dst[(g * a.bo + jj) * a.bi + kk] = acc[gg][i][j][v];
                }
    }
    if (do_db) {
#pragma unroll
        for (int q = 0; q < kDbRows; ++q) {
            const int row = tid + q * kThreads;
            if (row < T::kRowsA) {
                const int g = row / J, j = row % J;
                a.part_db[(int64_t)split * a.n_out + g * a.bo + j0 + j] = dbacc[q];
            }
        }
    }
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
        o.x = f32_to_bf16(s.x) | ((uint32_t)f32_to_bf16(s.y) << 16);
        o.y = f32_to_bf16(s.z) | ((uint32_t)f32_to_bf16(s.w) << 16);
        uint16_t *out = is_db ? db + idx : (idx < per_comp ? dW1 + idx : dW2 + (idx - per_comp));
        *reinterpret_cast<uint2 *>(out) = o;
    }
}

struct DwPlan {
    int J, K, tiles_j, tiles_k, splits;
    int64_t tokens_per_split;
    bool ok;
};

DwPlan plan_for(const DwPass &p, int J, int K) {
    DwPlan pl{};
    pl.J = J; pl.K = K;
    pl.tiles_j = (int)(p.bo / J);
    pl.tiles_k = (int)(p.bi / K);
    const int64_t tiles = 2 * (int64_t)pl.tiles_j * pl.tiles_k;
    // enough workgroups to cover 256 CUs about twice; each split a multiple of kT tokens
    int64_t want = (512 + tiles - 1) / tiles;
    const int64_t max_splits = (p.M + kT - 1) / kT;
    if (want > max_splits) want = max_splits;
    if (want < 1) want = 1;
    int64_t tps = (p.M + want - 1) / want;
    tps = (tps + kT - 1) / kT * kT;
    if (tps < kT) tps = kT;
    pl.tokens_per_split = tps;
    pl.splits = (int)((p.M + tps - 1) / tps);
    if (pl.splits < 1) pl.splits = 1;
    pl.ok = true;
    return pl;
}

bool choose(const DwPass &p, DwPlan &pl) {
    if (p.dtype != kBF16) return false;
    struct Cand { int D, J, K; };
    static const Cand cands[] = {
        {1, 256, 128}, {1, 128, 256}, {2, 128, 128}, {4, 128, 64}, {4, 64, 128},
        {8, 64, 64}, {16, 64, 32}, {16, 32, 64},
    };
    for (const Cand &c : cands)
        if (c.D == p.D && p.bo % c.J == 0 && p.bi % c.K == 0) {
            pl = plan_for(p, c.J, c.K);
            return true;
        }
    return false;
}

template <int D, int J, int K, int WJ, int WK, bool IN_T, bool OUT_T>
hipError_t launch_dw_cfg(const DwPass &p, const DwPlan &pl, hipStream_t s) {
    DwArgs a;
    a.M = p.M; a.n_in = p.n_in; a.n_out = p.n_out; a.bi = p.bi; a.bo = p.bo;
    a.dZ = static_cast<const uint16_t *>(p.dZ);
    a.X = static_cast<const uint16_t *>(p.X);
    a.part = static_cast<float *>(p.ws);
    a.part_db = a.part + (int64_t)pl.splits * 2 * p.D * p.bo * p.bi;
    a.tokens_per_split = pl.tokens_per_split;
    a.tiles_j = pl.tiles_j; a.tiles_k = pl.tiles_k; a.splits = pl.splits;
    a.want_db = p.db != nullptr;
    const int64_t blocks = 2 * (int64_t)pl.tiles_j * pl.tiles_k * pl.splits;
    dyad_dw_mfma<D, J, K, WJ, WK, IN_T, OUT_T><<<(unsigned)blocks, kThreads, 0, s>>>(a);
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
#define DYAD_DW_CASE(D_, J_, K_, WJ_, WK_) \
    if (p.D == D_ && pl.J == J_ && pl.K == K_) return launch_dw_cfg<D_, J_, K_, WJ_, WK_, IN_T, OUT_T>(p, pl, s);
    DYAD_DW_CASE(1, 256, 128, 128, 64)
    DYAD_DW_CASE(1, 128, 256, 64, 128)
    DYAD_DW_CASE(2, 128, 128, 64, 128)
    DYAD_DW_CASE(4, 128, 64, 128, 64)
    DYAD_DW_CASE(4, 64, 128, 64, 128)
    DYAD_DW_CASE(8, 64, 64, 64, 64)
    DYAD_DW_CASE(16, 64, 32, 64, 32)
    DYAD_DW_CASE(16, 32, 64, 32, 64)
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
