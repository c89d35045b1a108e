// The Dyad grouped GEMM on gfx950 matrix cores (bf16 in, fp32 accumulate).
//
// One workgroup computes an output tile of BM tokens x BN output features.
// Both weight components run in one K loop (the tile's accumulators take the
// BlockDiag product first, then the BlockTrans product), so neither partial
// result leaves registers and no add or concatenation is materialised.
//
// Tile columns.  The BN columns lie in one output block g1, which fixes the
// BlockDiag weight rows.  Without an output transpose the BlockTrans component
// uses the same group and rows.  With an output transpose, real column f takes
// its BlockTrans weight row from group f % D, row f / D.  The tile then keeps
// its accumulator columns in residue-major order (internal column
// q = r*(BN/D) + t holds real column r + D*t), so that every 16-column MFMA
// block reads one group r and consecutive weight rows of it; the epilogue
// undoes the order.
//
// Pipeline.  The K loop runs over stages of 32 k values (one MFMA K step),
// BlockDiag stages first.  LDS holds two stage buffers: while the waves
// multiply out of one, the next stage's operands (already in registers) are
// written into the other and the loads for the stage after that are issued,
// so global latency hides behind a stage of MFMAs and there is one barrier per
// stage.  The loop is split into phases whose stage kinds are known at compile
// time, so every path through a phase is straight-line code.  Global loads are
// buffer loads: a per-thread 32-bit offset fixed for the whole tile plus a
// per-stage scalar offset, and rows past the end of the batch fall outside the
// buffer's range and read as zero.  LDS rows are 64 bytes (32 bf16) with their
// four 16-byte chunks XOR-swizzled by row, which keeps staging writes and
// fragment reads free of bank conflicts without padding.
//
// Operand staging.  A BlockTrans stage with an input transpose needs input
// columns k*D + r: it loads the contiguous span of 32*D columns that holds
// k = kk..kk+31 for every residue r and de-interleaves it in registers
// (v_perm_b32) into one slab per residue, so the strided view is never
// materialised in HBM.  Weights read transposed (the input-gradient pass) are
// loaded as 8x8 blocks and transposed in registers.
#pragma once

#include <type_traits>

#include "dyad_device.h"
#include "dyad_internal.h"

namespace dyad {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;

constexpr int kStageK = 32;   // k per stage and per MFMA (v_mfma_f32_16x16x32_bf16)

struct GemmArgs {
    int64_t M, Kin, Nout, bk, bn, D;
    const uint16_t *in, *W1, *W2, *bias, *h_in;
    uint16_t *out, *h_out;
    int epilogue;
    int tiles_n;        // output tiles per token panel
    int tiles_total;
};

// ---- buffer loads ------------------------------------------------------------

// Word 3 of a raw buffer resource on gfx9-family parts: 32-bit data, no swizzle.
constexpr int kBufferWord3 = 0x00020000;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kBufferWord3);
}

// 16 bytes at base + voff + soff; zero when voff lies past the buffer's range.
__device__ __forceinline__ uint4 bload16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ uint4 ldg16(const uint16_t *p) { return *reinterpret_cast<const uint4 *>(p); }

// ---- register shuffles ---------------------------------------------------------

// Word w (0..3) of a 16-byte vector, w known at compile time after unrolling.
__device__ __forceinline__ uint32_t word_of(const uint4 &v, int w) {
    const uint32_t lo = (w & 1) ? v.y : v.x;
    const uint32_t hi = (w & 1) ? v.w : v.z;
    return (w & 2) ? hi : lo;
}

// v_perm_b32 selector placing the 16-bit value at byte offset b of {hi:lo} in
// the low half and the one at byte offset c in the high half.
__host__ __device__ constexpr uint32_t perm_sel(int b, int c) {
    return (uint32_t)b | ((uint32_t)(b + 1) << 8) | ((uint32_t)c << 16) | ((uint32_t)(c + 1) << 24);
}

// Residue R (compile time) of 8 consecutive k values held in D consecutive
// 16-byte vectors (input column k*D + r, residue fastest), as one 16-byte
// vector of the 8 values.  Element e of the span sits in vector e / 8, word
// (e % 8) / 2, half e % 2; each output word takes two such halves with one
// v_perm_b32.
template <int D, int R>
__device__ __forceinline__ uint4 deinterleave(const uint4 (&v)[D]) {
    uint32_t o[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const int e0 = (2 * w) * D + R, e1 = (2 * w + 1) * D + R;
        const uint32_t a = word_of(v[e0 >> 3], (e0 & 7) >> 1);   // holds e0
        const uint32_t b = word_of(v[e1 >> 3], (e1 & 7) >> 1);   // holds e1
        // bytes 0-3 of {b:a} are a, bytes 4-7 are b
        o[w] = __builtin_amdgcn_perm(b, a, perm_sel((e0 & 1) * 2, 4 + (e1 & 1) * 2));
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
}

// Residue r, a value uniform across the workgroup, of the span: one branch per
// residue, each a compile-time shuffle.
template <int D, int R = 0>
__device__ __forceinline__ uint4 deinterleave_uniform(const uint4 (&v)[D], int r) {
    if constexpr (R + 1 < D) {
        if (r != R) return deinterleave_uniform<D, R + 1>(v, r);
    }
    return deinterleave<D, R>(v);
}

// Every residue of the span into its own LDS slab (slab R at dst + R * slab).
template <int D, int R = 0>
__device__ __forceinline__ void deinterleave_all(const uint4 (&v)[D], uint16_t *dst, int slab) {
    *reinterpret_cast<uint4 *>(dst + R * slab) = deinterleave<D, R>(v);
    if constexpr (R + 1 < D) deinterleave_all<D, R + 1>(v, dst, slab);
}

// Column e (0..7) of an 8x8 block of bf16 given as 8 rows of 8: the 8 row values, packed.
__device__ __forceinline__ uint4 column_of(const uint4 (&r)[8], int e) {
    uint32_t o[4];
    const uint32_t sel = (e & 1) ? perm_sel(2, 6) : perm_sel(0, 4);
#pragma unroll
    for (int p = 0; p < 4; ++p)
        o[p] = __builtin_amdgcn_perm(word_of(r[2 * p + 1], e >> 1), word_of(r[2 * p], e >> 1), sel);
    return make_uint4(o[0], o[1], o[2], o[3]);
}

// ---- epilogue math -------------------------------------------------------------

// Two fp32 values as packed bf16, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
    const f32x2_t v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ float unpack_bf16(uint32_t w, int half) {
    return __uint_as_float(half ? (w & 0xffff0000u) : (w << 16));
}

// Standard normal CDF and density at x.  erfc(|x|/sqrt 2) uses the rational
// approximation 7.1.26 of Abramowitz & Stegun (absolute error below 1.5e-7 in
// erf), far below the bf16 rounding of the result; it shares exp(-x^2/2) with
// the density.
__device__ __forceinline__ void normal_cdf_pdf(float x, float &cdf, float &pdf) {
    const float z = fabsf(x) * 0.70710678118654752f;
    const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, z, 1.0f));
    const float poly =
        t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 1.061405429f, -1.453152027f), 1.421413741f), -0.284496736f),
                 0.254829592f);
    const float e = __builtin_amdgcn_exp2f(-z * z * 1.4426950408889634f);   // exp(-x^2 / 2)
    const float tail = 0.5f * poly * e;                                      // P(N > |x|)
    cdf = x >= 0.f ? 1.f - tail : tail;
    pdf = 0.3989422804014327f * e;
}

// ---- layout helpers --------------------------------------------------------------

// bf16 element offset of 16-byte chunk c (0..3) of LDS row `row` (rows of 32
// bf16, 64 bytes).  The chunk position is XORed with (row >> 1) & 3, which
// spreads the 16-byte fragment reads of 16 consecutive rows at one chunk over
// distinct banks (measured on gfx950: full LDS read bandwidth, where unswizzled
// 64-byte rows run at half of it).
__device__ __forceinline__ int lds_off(int row, int c) {
    return row * kStageK + ((c ^ (row >> 1)) & 3) * 8;
}

// Tile index of workgroup w, with consecutive tiles (one token panel's column
// tiles, then the next panel's) placed on one XCD: the hardware deals
// workgroups round-robin over the 8 XCDs, each with its own L2.
__device__ __forceinline__ int xcd_tile(int w, int total) {
    const int q = total >> 3, r = total & 7, x = w & 7, i = w >> 3;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + i;
}

template <int BM, int BN, int WGM, int WGN, int D, bool IN_T, bool OUT_T, bool W_T>
struct GemmCfg {
    static constexpr int kWaves = WGM * WGN;
    static constexpr int kThreads = 64 * kWaves;
    static constexpr int WM = BM / WGM, WN = BN / WGN;
    static constexpr int kSubM = WM / 16, kSubN = WN / 16;
    static constexpr int kRes = OUT_T ? D : 1;            // A slabs of a BlockTrans stage
    static constexpr int kCPR = BN / kRes;                // internal columns per residue
    static constexpr int kRPW = WN >= kCPR ? WN / kCPR : 1;              // residues per wave
    static constexpr int kBPR = (WN >= kCPR ? kCPR : WN) / 16;           // MFMA blocks per residue per wave
    // A row-chunks (8 k values of one row) per stage and per thread
    static constexpr int kRowChunks = BM * (kStageK / 8);
    static constexpr int kRC = kRowChunks / kThreads;
    // 16-byte A vectors per row-chunk a BlockTrans stage loads
    static constexpr int kVecPerRC2 = (IN_T || OUT_T) ? D : 1;
    // B: 16-byte vectors (no transpose) or 8x8 blocks (transpose) per stage
    static constexpr int kVecB = BN * (kStageK / 8);
    static constexpr int kRB = (kVecB + kThreads - 1) / kThreads;
    static constexpr int kBlkB = (BN / 8) * (kStageK / 8);
    static constexpr int kRBT = (kBlkB + kThreads - 1) / kThreads;
    // LDS, in bf16 elements
    static constexpr int kSlab = BM * kStageK;
    static constexpr int kStageA = kRes * kSlab;
    static constexpr int kStageElems = kStageA + BN * kStageK;
    static constexpr int kLdsOperands = 2 * kStageElems * 2;   // bytes, two stage buffers
    // epilogue: WGM*16 rows of fp32 at a time
    static constexpr int kEpiRows = WGM * 16;
    static constexpr int kEpiPitch = BN + 4;
    static constexpr int kLdsEpi = kEpiRows * kEpiPitch * 4;
    static constexpr int kLds = kLdsOperands > kLdsEpi ? kLdsOperands : kLdsEpi;

    static_assert(BM % (16 * WGM) == 0 && BN % (16 * WGN) == 0, "wave tiles of whole MFMA blocks");
    static_assert(kRowChunks % kThreads == 0, "A row-chunks spread evenly over the threads");
    static_assert(!OUT_T || (kCPR % 16 == 0), "each MFMA column block holds one residue");
    static_assert(WN % kCPR == 0 || kCPR % WN == 0, "waves hold whole residues or parts of one");
    static_assert(kLds <= 160 * 1024, "LDS budget");
};

template <int BM, int BN, int WGM, int WGN, int D, bool IN_T, bool OUT_T, bool W_T, int OCC>
__global__ void __launch_bounds__(64 * WGM * WGN, OCC)
dyad_gemm_mfma(GemmArgs a) {
    using C = GemmCfg<BM, BN, WGM, WGN, D, IN_T, OUT_T, W_T>;
    using Comp1 = std::false_type;
    using Comp2 = std::true_type;
    constexpr int T = C::kThreads;
    __shared__ __attribute__((aligned(16))) unsigned char smem[C::kLds];
    uint16_t *lds = reinterpret_cast<uint16_t *>(smem);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int tile = xcd_tile(blockIdx.x, a.tiles_total);
    const int64_t m0 = (int64_t)(tile / a.tiles_n) * BM;
    const int n0 = (tile % a.tiles_n) * BN;        // first output column of the tile
    const int bk = (int)a.bk, bn = (int)a.bn, Kin = (int)a.Kin;
    const int g1 = n0 / bn;                        // output block = BlockDiag group
    const int jb = n0 - g1 * bn;                   // first BlockDiag weight row
    const int ks = bk / kStageK;                   // stages per component
    const int S = 2 * ks;

    const int wm0 = (wave / WGN) * C::WM;
    const int wn0 = (wave % WGN) * C::WN;

    // Buffers: A is this tile's token panel (rows past M fall outside its
    // range), W1 / W2 the whole weight tensors.
    const int64_t rows_left = a.M - m0;
    const uint64_t a_bytes = (uint64_t)(rows_left < BM ? rows_left : BM) * (uint64_t)Kin * 2u;
    const __amdgpu_buffer_rsrc_t rA = buffer_rsrc(a.in + m0 * a.Kin, (uint32_t)a_bytes);
    const uint32_t w_bytes = (uint32_t)(a.D * a.bn * a.bk * 2);
    const __amdgpu_buffer_rsrc_t rW1 = buffer_rsrc(a.W1, w_bytes);
    const __amdgpu_buffer_rsrc_t rW2 = buffer_rsrc(a.W2, w_bytes);

    // internal column q -> tile-local real column, and back
    auto real_col = [](int q) -> int { return OUT_T ? (q / C::kCPR) + D * (q % C::kCPR) : q; };
    auto internal_col = [](int p) -> int { return OUT_T ? (p % D) * C::kCPR + p / D : p; };

    // Per-thread byte offsets, fixed for the whole tile; stages add a scalar offset.
    uint32_t voA1[C::kRC], voA2[C::kRC];
#pragma unroll
    for (int q = 0; q < C::kRC; ++q) {
        const int rc = tid + q * T, row = rc >> 2, c = rc & 3;
        const uint32_t rowoff = (uint32_t)row * (uint32_t)Kin * 2u;
        voA1[q] = rowoff + (uint32_t)(g1 * bk + c * 8) * 2u;
        if constexpr (IN_T) voA2[q] = rowoff + (uint32_t)(c * 8 * D) * 2u;       // span of 8 k x D residues
        else if constexpr (OUT_T) voA2[q] = rowoff + (uint32_t)(c * 8) * 2u;     // + block r (scalar)
        else voA2[q] = voA1[q];
    }
    uint32_t voB1[W_T ? C::kRBT : C::kRB], voB2[W_T ? C::kRBT : C::kRB];
    if constexpr (!W_T) {
        // weight row of internal column col, chunk c of 8 k
#pragma unroll
        for (int q = 0; q < C::kRB; ++q) {
            const int v = (tid + q * T) % C::kVecB, col = v >> 2, c = v & 3;
            const int row1 = jb + real_col(col);
            int grp2 = g1, row2 = jb + col;
            if constexpr (OUT_T) { grp2 = col / C::kCPR; row2 = n0 / D + col % C::kCPR; }
            voB1[q] = (uint32_t)((g1 * bn + row1) * bk + c * 8) * 2u;
            voB2[q] = (uint32_t)((grp2 * bn + row2) * bk + c * 8) * 2u;
        }
    } else {
        // weights stored [grp][k][row]: 8x8 blocks of (8 k) x (8 consecutive rows)
#pragma unroll
        for (int q = 0; q < C::kRBT; ++q) {
            const int bid = (tid + q * T) % C::kBlkB;
            const int k8 = bid % (kStageK / 8), c8 = (bid / (kStageK / 8)) * 8;
            int grp2 = g1, row2 = jb + c8;                 // real (comp 1) / internal (comp 2) columns c8..c8+7
            if constexpr (OUT_T) { grp2 = c8 / C::kCPR; row2 = n0 / D + c8 % C::kCPR; }
            voB1[q] = (uint32_t)((g1 * bk + k8 * 8) * bn + jb + c8) * 2u;
            voB2[q] = (uint32_t)((grp2 * bk + k8 * 8) * bn + row2) * 2u;
        }
    }

    f32x4_t acc[C::kSubM][C::kSubN];
#pragma unroll
    for (int i = 0; i < C::kSubM; ++i)
#pragma unroll
        for (int j = 0; j < C::kSubN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    uint4 ra[C::kRC][C::kVecPerRC2];
    uint4 rb[W_T ? C::kRBT : C::kRB][W_T ? 8 : 1];

    // ---- global -> registers for stage s of component 1 or 2
    auto fetch = [&](auto comp, int s) {
        constexpr bool C2 = decltype(comp)::value;
        const uint32_t kk = (uint32_t)((C2 ? s - ks : s) * kStageK);
#pragma unroll
        for (int q = 0; q < C::kRC; ++q) {
            if constexpr (!C2 || !(IN_T || OUT_T)) {
                ra[q][0] = bload16(rA, C2 ? voA2[q] : voA1[q], kk * 2u);
            } else if constexpr (IN_T) {
#pragma unroll
                for (int d = 0; d < D; ++d) ra[q][d] = bload16(rA, voA2[q] + d * 16u, kk * D * 2u);
            } else {
#pragma unroll
                for (int r = 0; r < D; ++r) ra[q][r] = bload16(rA, voA2[q], ((uint32_t)(r * bk) + kk) * 2u);
            }
        }
        const __amdgpu_buffer_rsrc_t rW = C2 ? rW2 : rW1;
        if constexpr (!W_T) {
#pragma unroll
            for (int q = 0; q < C::kRB; ++q)
                if (C::kVecB % T == 0 || tid + q * T < C::kVecB)
                    rb[q][0] = bload16(rW, C2 ? voB2[q] : voB1[q], kk * 2u);
        } else {
#pragma unroll
            for (int q = 0; q < C::kRBT; ++q)
                if (C::kBlkB % T == 0 || tid + q * T < C::kBlkB) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        rb[q][e] = bload16(rW, C2 ? voB2[q] : voB1[q], (kk + e) * (uint32_t)bn * 2u);
                }
        }
    };

    // ---- registers -> LDS stage buffer
    auto stash = [&](auto comp, uint16_t *buf) {
        constexpr bool C2 = decltype(comp)::value;
        uint16_t *bufB = buf + C::kStageA;
#pragma unroll
        for (int q = 0; q < C::kRC; ++q) {
            const int rc = tid + q * T, row = rc >> 2, c = rc & 3;
            if constexpr (!C2 || !(IN_T || OUT_T)) {
                *reinterpret_cast<uint4 *>(buf + lds_off(row, c)) = ra[q][0];
            } else if constexpr (IN_T) {
                uint4 span[D];
#pragma unroll
                for (int d = 0; d < D; ++d) span[d] = ra[q][d];
                if constexpr (OUT_T)
                    deinterleave_all<D>(span, buf + lds_off(row, c), C::kSlab);
                else   // only residue g1 feeds this tile
                    *reinterpret_cast<uint4 *>(buf + lds_off(row, c)) = deinterleave_uniform<D>(span, g1);
            } else {
#pragma unroll
                for (int r = 0; r < D; ++r)
                    *reinterpret_cast<uint4 *>(buf + r * C::kSlab + lds_off(row, c)) = ra[q][r];
            }
        }
        if constexpr (!W_T) {
#pragma unroll
            for (int q = 0; q < C::kRB; ++q) {
                const int v = tid + q * T;
                if (C::kVecB % T == 0 || v < C::kVecB)
                    *reinterpret_cast<uint4 *>(bufB + lds_off(v >> 2, v & 3)) = rb[q][0];
            }
        } else {
#pragma unroll
            for (int q = 0; q < C::kRBT; ++q) {
                const int bid = tid + q * T;
                if (C::kBlkB % T == 0 || bid < C::kBlkB) {
                    const int k8 = bid % (kStageK / 8), c8 = (bid / (kStageK / 8)) * 8;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int col = C2 ? c8 + e : internal_col(c8 + e);
                        *reinterpret_cast<uint4 *>(bufB + lds_off(col, k8)) = column_of(rb[q], e);
                    }
                }
            }
        }
    };

    // ---- MFMA on one stage buffer
    auto compute = [&](auto comp, const uint16_t *buf) {
        constexpr bool C2 = decltype(comp)::value;
        const uint16_t *bufB = buf + C::kStageA;
        const int lr = lane & 15, lc = lane >> 4;
        bf16x8_t afrag[C::kSubM];
        if constexpr (!OUT_T || !C2) {
#pragma unroll
            for (int i = 0; i < C::kSubM; ++i)
                afrag[i] = *reinterpret_cast<const bf16x8_t *>(buf + lds_off(wm0 + i * 16 + lr, lc));
#pragma unroll
            for (int j = 0; j < C::kSubN; ++j) {
                const bf16x8_t bf = *reinterpret_cast<const bf16x8_t *>(bufB + lds_off(wn0 + j * 16 + lr, lc));
#pragma unroll
                for (int i = 0; i < C::kSubM; ++i)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag[i], bf, acc[i][j], 0, 0, 0);
            }
        } else {
#pragma unroll
            for (int rr = 0; rr < C::kRPW; ++rr) {
                const int r = (wn0 + rr * C::kCPR) / C::kCPR;
                const uint16_t *slab = buf + r * C::kSlab;
#pragma unroll
                for (int i = 0; i < C::kSubM; ++i)
                    afrag[i] = *reinterpret_cast<const bf16x8_t *>(slab + lds_off(wm0 + i * 16 + lr, lc));
#pragma unroll
                for (int jj = 0; jj < C::kBPR; ++jj) {
                    const int j = rr * C::kBPR + jj;
                    const bf16x8_t bf = *reinterpret_cast<const bf16x8_t *>(bufB + lds_off(wn0 + j * 16 + lr, lc));
#pragma unroll
                    for (int i = 0; i < C::kSubM; ++i)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag[i], bf, acc[i][j], 0, 0, 0);
                }
            }
        }
    };

    // ---- main loop.  Stage s (0 <= s < S) uses buffer s & 1; each iteration
    // stashes stage s+1, fetches stage s+2 and multiplies stage s.  Phases keep
    // the kind of every stage known at compile time.
    // (pointer arithmetic on the LDS array keeps these LDS accesses; an array of
    // pointers would turn them into flat ones)
    auto buf = [&](int idx) -> uint16_t * { return lds + (idx & 1) * C::kStageElems; };
    if (ks == 1) {
        fetch(Comp1{}, 0);
        stash(Comp1{}, buf(0));
        fetch(Comp2{}, 1);
        __syncthreads();
        stash(Comp2{}, buf(1));
        compute(Comp1{}, buf(0));
        __syncthreads();
        compute(Comp2{}, buf(1));
        __syncthreads();
    } else {
        fetch(Comp1{}, 0);
        stash(Comp1{}, buf(0));
        fetch(Comp1{}, 1);
        __syncthreads();
        int s = 0;
        for (; s + 2 < ks; ++s) {
            stash(Comp1{}, buf(s + 1));
            fetch(Comp1{}, s + 2);
            compute(Comp1{}, buf(s));
            __syncthreads();
        }
        // s = ks - 2: the stage after next is the first BlockTrans stage
        stash(Comp1{}, buf(s + 1));
        fetch(Comp2{}, s + 2);
        compute(Comp1{}, buf(s));
        __syncthreads();
        ++s;
        // s = ks - 1
        stash(Comp2{}, buf(s + 1));
        fetch(Comp2{}, s + 2);
        compute(Comp1{}, buf(s));
        __syncthreads();
        ++s;
        for (; s + 2 < S; ++s) {
            stash(Comp2{}, buf(s + 1));
            fetch(Comp2{}, s + 2);
            compute(Comp2{}, buf(s));
            __syncthreads();
        }
        stash(Comp2{}, buf(s + 1));
        compute(Comp2{}, buf(s));
        __syncthreads();
        ++s;
        compute(Comp2{}, buf(s));
        __syncthreads();
    }

    // ---- epilogue: per 16-row MFMA block row, accumulators -> LDS (real
    // column order, fp32) -> bias / GELU / GELU' -> bf16 -> coalesced stores
    float *ldsE = reinterpret_cast<float *>(smem);
    constexpr int kGroups = C::kEpiRows * (BN / 8);
#pragma unroll
    for (int i = 0; i < C::kSubM; ++i) {
#pragma unroll
        for (int j = 0; j < C::kSubN; ++j) {
            const int col = real_col(wn0 + j * 16 + (lane & 15));
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int er = (wave / WGN) * 16 + (lane >> 4) * 4 + v;
                ldsE[er * C::kEpiPitch + col] = acc[i][j][v];
            }
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < (kGroups + T - 1) / T; ++q) {
            const int gidx = tid + q * T;
            if (kGroups % T != 0 && gidx >= kGroups) break;
            const int er = gidx / (BN / 8), c8 = (gidx % (BN / 8)) * 8;
            const int64_t m = m0 + (er / 16) * C::WM + i * 16 + (er % 16);
            if (m < a.M) {
                float x[8];
                const float4 lo = *reinterpret_cast<const float4 *>(ldsE + er * C::kEpiPitch + c8);
                const float4 hi = *reinterpret_cast<const float4 *>(ldsE + er * C::kEpiPitch + c8 + 4);
                x[0] = lo.x; x[1] = lo.y; x[2] = lo.z; x[3] = lo.w;
                x[4] = hi.x; x[5] = hi.y; x[6] = hi.z; x[7] = hi.w;
                const int64_t off = m * a.Nout + n0 + c8;
                if (a.epilogue == kEpiGeluGrad) {
                    const uint4 h = ldg16(a.h_in + off);
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float hv = unpack_bf16(word_of(h, e >> 1), e & 1);
                        float cdf, pdf;
                        normal_cdf_pdf(hv, cdf, pdf);
                        x[e] *= fmaf(hv, pdf, cdf);
                    }
                } else {
                    if (a.bias) {
                        const uint4 b = ldg16(a.bias + n0 + c8);
#pragma unroll
                        for (int e = 0; e < 8; ++e) x[e] += unpack_bf16(word_of(b, e >> 1), e & 1);
                    }
                    if (a.epilogue == kEpiBiasGelu) {
                        if (a.h_out)
                            *reinterpret_cast<uint4 *>(a.h_out + off) =
                                make_uint4(pack_bf16(x[0], x[1]), pack_bf16(x[2], x[3]), pack_bf16(x[4], x[5]),
                                           pack_bf16(x[6], x[7]));
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            float cdf, pdf;
                            normal_cdf_pdf(x[e], cdf, pdf);
                            x[e] *= cdf;
                        }
                    }
                }
                *reinterpret_cast<uint4 *>(a.out + off) =
                    make_uint4(pack_bf16(x[0], x[1]), pack_bf16(x[2], x[3]), pack_bf16(x[4], x[5]), pack_bf16(x[6], x[7]));
            }
        }
        __syncthreads();
    }
}

}  // namespace dyad
