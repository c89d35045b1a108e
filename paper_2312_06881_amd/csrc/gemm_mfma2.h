// The Dyad grouped GEMM on gfx950 matrix cores, fused-stage form for large
// tiles of eight waves (bf16 in, fp32 accumulate).
//
// Same tile semantics as gemm_mfma.h (one output block per tile, residue-major
// internal columns with an output transpose, epilogue shared), but every
// pipeline stage carries 32 reduction indices of BOTH components: the
// BlockDiag operands (A1: the tile's input block, B1: W1) and the BlockTrans
// ones (A2: the de-interleaved input span or the per-residue input slabs, B2:
// W2).  Each stage therefore holds two MFMA k-steps, all stages have the same
// load shape, and one stage of prefetch covers twice the matrix work of a
// single-component stage.  The loop is uniform: stash stage s+1 from
// registers, issue the loads of stage s+2, multiply stage s, one barrier.
//
// With weights read transposed (input gradient) the weight stage is kept in
// its natural layout, 32 rows of the reduction index by BN columns (rows padded
// by 16 bytes), and the MFMA operand comes from ds_read_b64_tr_b16, so no
// transposes are done in registers.  Where the tile's columns are
// residue-major (output transpose), the BlockDiag weight columns are
// de-interleaved on their way into LDS, 8 D real columns at a time.
#pragma once

#include <type_traits>

#include "gemm_common.h"

namespace dyad {

template <int BM, int BN, int WGM, int WGN, int D, bool IN_T, bool OUT_T, bool W_T>
struct Gemm2Cfg {
    static constexpr int kWaves = WGM * WGN, kThreads = 64 * kWaves, kWGN = WGN;
    static constexpr int WM = BM / WGM, WN = BN / WGN;
    static constexpr int kSubM = WM / 16, kSubN = WN / 16;
    static constexpr int kRes = OUT_T ? D : 1;                          // A2 slabs
    static constexpr int kCPR = BN / kRes;                              // internal columns per residue
    static constexpr int kRPW = WN >= kCPR ? WN / kCPR : 1;             // residues per wave
    static constexpr int kBPR = (WN >= kCPR ? kCPR : WN) / 16;          // MFMA blocks per residue per wave
    // LDS bytes of one stage: A1 slab, kRes A2 slabs (BM rows of 64 bytes each),
    // then the two weight tiles
    static constexpr int kSlab = BM * kStageK * 2;
    static constexpr int kBRow = BN * 2 + 16;                           // transposed weights: row pitch
    static constexpr int kBBytes = W_T ? kStageK * kBRow : BN * kStageK * 2;
    static constexpr int kOffA2 = kSlab, kOffB1 = kSlab * (1 + kRes), kOffB2 = kOffB1 + kBBytes;
    static constexpr int kStage = kOffB2 + kBBytes;
    static constexpr int kLdsOperands = 2 * kStage;
    static constexpr int kEpiRows = WGM * 16, kEpiPitch = BN + 4, kEpiElems = kEpiRows * kEpiPitch;
    static constexpr int kLdsEpi = 2 * kEpiElems * 4;
    static constexpr int kLds = kLdsOperands > kLdsEpi ? kLdsOperands : kLdsEpi;
    // load slots per thread and stage
    static constexpr int kRowChunks = BM * (kStageK / 8);               // 16-byte pieces of an A slab
    static constexpr int kQA1 = (kRowChunks + kThreads - 1) / kThreads;
    static constexpr int kUnitsA2 = IN_T ? kRowChunks : kRes * kRowChunks;
    static constexpr int kQA2 = (kUnitsA2 + kThreads - 1) / kThreads;
    static constexpr int kVA2 = IN_T ? D : 1;                           // an input transpose loads spans
    static constexpr int kUnitsB = W_T ? kStageK * BN / 8 : BN * (kStageK / 8);
    static constexpr int kQB = (kUnitsB + kThreads - 1) / kThreads;
    static constexpr bool kB1Chunks = W_T && OUT_T && D > 1;
    static constexpr int kUnitsB1 = kB1Chunks ? kStageK * BN / (8 * D) : kUnitsB;
    static constexpr int kQB1 = (kUnitsB1 + kThreads - 1) / kThreads;
    static constexpr int kVB1 = kB1Chunks ? D : 1;

    static_assert(BM % (16 * WGM) == 0 && BN % (16 * WGN) == 0, "wave tiles of whole MFMA blocks");
    static_assert(kRowChunks % 64 == 0, "whole waves of A row-chunks");
    static_assert(!OUT_T || (BN % D == 0 && kCPR % 16 == 0), "each MFMA column block holds one residue");
    static_assert(WN % kCPR == 0 || kCPR % WN == 0, "waves hold whole residues or parts of one");
    static_assert(kLds <= 160 * 1024, "LDS budget");
};

// ONLY = 1 or 2: that component alone, into fp32 partial sums (a.part, slice
// a.slice0).  ONLY = 3: component 1 alone with the full epilogue, its sums
// first added to those of slice a.slice0 (read at the block-order place of
// each column when a.unperm).  Component 2 alone under an output transpose needs no output
// block per tile: its columns f = j*D + g take weight group f % D and row
// f / D whatever block f falls in.  The zero-padded forms (block-ordered
// operands, gemm_epilogue_pad): ONLY = 4 component 1 adding the slice of
// component 2 (run with ONLY = 1) under an output transpose, ONLY = 5 both
// components, the second reading its own input copy a.in2 at the first's
// places.
template <int BM, int BN, int WGM, int WGN, int D, bool IN_T, bool OUT_T, bool W_T, int ONLY = 0>
__global__ void __launch_bounds__(64 * WGM * WGN, 1)
dyad_gemm_mfma2(GemmArgs a) {
    using C = Gemm2Cfg<BM, BN, WGM, WGN, D, IN_T, OUT_T, W_T>;
    constexpr int T = C::kThreads;
    // ONLY 1, 3 and 4 run component 1 alone; 4 and 5 are the zero-padded forms
    static_assert(ONLY < 4 || (!IN_T && !OUT_T), "padded forms run on block-ordered operands");
    constexpr bool kComp1Only = ONLY == 1 || ONLY == 3 || ONLY == 4;
    __shared__ __attribute__((aligned(16))) unsigned char smem[C::kLds];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // work item -> (tile, split), the splits of a tile next to each other
    const int item = xcd_tile(blockIdx.x, a.tiles_total * a.splits);
    const int tile = item / a.splits, split = item % a.splits;
    const int tiles_m = a.tiles_total / a.tiles_n;
    const int64_t m0 = (int64_t)(a.n_major ? tile % tiles_m : tile / a.tiles_n) * BM;
    const int n0 = (a.n_major ? tile / tiles_m : tile % a.tiles_n) * BN;   // first output column of the tile
    const int bk = (int)a.bk, bn = (int)a.bn, Kin = (int)a.Kin;
    const int g1 = n0 / bn;                        // output block = BlockDiag group
    const int jb = n0 - g1 * bn;                   // first BlockDiag weight row / column
    const int S = bk / kStageK / a.splits;         // stages of this split (each both components)
    const int kofs = split * S;

    const int wm0 = (wave / WGN) * C::WM;
    const int wn0 = (wave % WGN) * C::WN;

    // Buffers: A is this tile's token panel (rows past M fall outside its
    // range), W1 / W2 the whole weight tensors.  Loads out of range read zero.
    const int64_t rows_left = a.M - m0;
    const uint64_t a_bytes = (uint64_t)(rows_left < BM ? rows_left : BM) * (uint64_t)Kin * 2u;
    const __amdgpu_buffer_rsrc_t rA = buffer_rsrc(a.in + m0 * a.Kin, (uint32_t)a_bytes);
    // component 2's input: with ONLY == 5 its own block-ordered copy
    const __amdgpu_buffer_rsrc_t rA2 = ONLY == 5 ? buffer_rsrc(a.in2 + m0 * a.Kin, (uint32_t)a_bytes) : rA;
    const uint32_t w_bytes = (uint32_t)(a.D * a.bn * a.bk * 2);
    const __amdgpu_buffer_rsrc_t rW1 = buffer_rsrc(a.W1, w_bytes);
    const __amdgpu_buffer_rsrc_t rW2 = buffer_rsrc(a.W2, w_bytes);

    // internal column q -> tile-local real column
    auto real_col = [](int q) -> int { return OUT_T ? (q / C::kCPR) + D * (q % C::kCPR) : q; };

    // ---- per-thread offsets, fixed for the tile; a stage adds a scalar offset
    // (slots past the tile's pieces, small tiles only: load out of range, store nothing)
    uint32_t voA1[C::kQA1], loA1[C::kQA1];
    bool okA1[C::kQA1], okA2[C::kQA2];
#pragma unroll
    for (int q = 0; q < C::kQA1; ++q) {
        const int rc = (tid + q * T) % C::kRowChunks, row = rc >> 2, c = rc & 3;
        okA1[q] = tid + q * T < C::kRowChunks;
        voA1[q] = okA1[q] ? (uint32_t)row * (uint32_t)Kin * 2u + (uint32_t)(g1 * bk + c * 8) * 2u : kNoLoad;
        loA1[q] = (uint32_t)lds_off(row, c) * 2u;
    }
    uint32_t voA2[C::kQA2], loA2[C::kQA2];
#pragma unroll
    for (int q = 0; q < C::kQA2; ++q) {
        const int p = (tid + q * T) % C::kUnitsA2;
        okA2[q] = tid + q * T < C::kUnitsA2;
        const int r = IN_T ? 0 : p / C::kRowChunks, rc = p % C::kRowChunks, row = rc >> 2, c = rc & 3;
        const uint32_t rowoff = (uint32_t)row * (uint32_t)Kin * 2u;
        if constexpr (IN_T) voA2[q] = rowoff + (uint32_t)(c * 8 * D) * 2u;            // span of 8 k x D residues
        else if constexpr (ONLY == 5) voA2[q] = rowoff + (uint32_t)(g1 * bk + c * 8) * 2u;   // block g1 of in2
        else voA2[q] = rowoff + (uint32_t)(r * bk + c * 8) * 2u;                      // residue r's input block
        loA2[q] = (uint32_t)(C::kOffA2 + r * C::kSlab) + (uint32_t)lds_off(row, c) * 2u;
        if (!okA2[q]) voA2[q] = kNoLoad;
    }
    uint32_t voB1[C::kQB1], loB1[C::kQB1], voB2[C::kQB], loB2[C::kQB];
    bool okB1[C::kQB1], okB2[C::kQB];
#pragma unroll
    for (int q = 0; q < C::kQB1; ++q) {
        const int v = tid + q * T;
        okB1[q] = v < C::kUnitsB1;
        if constexpr (!W_T) {
            // weight row of internal column col, chunk c of 8 k
            const int col = v >> 2, c = v & 3;
            voB1[q] = (uint32_t)((g1 * bn + jb + real_col(col)) * bk + c * 8) * 2u;
            loB1[q] = (uint32_t)(C::kOffB1 + lds_off(col, c) * 2);
        } else if constexpr (C::kB1Chunks) {
            // row j, real columns jb + 8 D u .. + 8 D - 1, split into one piece per residue
            const int per = BN / (8 * D), j = v / per, u = v % per;
            voB1[q] = (uint32_t)((g1 * bk + j) * bn + jb + 8 * D * u) * 2u;
            loB1[q] = (uint32_t)(C::kOffB1 + j * C::kBRow + 8 * u * 2);
        } else {
            const int j = v / (BN / 8), u = v % (BN / 8);
            voB1[q] = (uint32_t)((g1 * bk + j) * bn + jb + 8 * u) * 2u;
            loB1[q] = (uint32_t)(C::kOffB1 + j * C::kBRow + 8 * u * 2);
        }
        if (!okB1[q]) voB1[q] = kNoLoad;
    }
#pragma unroll
    for (int q = 0; q < C::kQB; ++q) {
        const int v = tid + q * T;
        okB2[q] = v < C::kUnitsB;
        if constexpr (!W_T) {
            const int col = v >> 2, c = v & 3;
            int grp2 = g1, row2 = jb + col;
            if constexpr (OUT_T) { grp2 = col / C::kCPR; row2 = n0 / D + col % C::kCPR; }
            voB2[q] = (uint32_t)((grp2 * bn + row2) * bk + c * 8) * 2u;
            loB2[q] = (uint32_t)(C::kOffB2 + lds_off(col, c) * 2);
        } else {
            // row j, internal columns 8 u .. 8 u + 7: residue r's columns t .. t + 7
            const int j = v / (BN / 8), col = 8 * (v % (BN / 8));
            int grp2 = g1, c2 = jb + col;
            if constexpr (OUT_T) { grp2 = col / C::kCPR; c2 = n0 / D + col % C::kCPR; }
            voB2[q] = (uint32_t)((grp2 * bk + j) * bn + c2) * 2u;
            loB2[q] = (uint32_t)(C::kOffB2 + j * C::kBRow + col * 2);
        }
        if (!okB2[q]) voB2[q] = kNoLoad;
    }

    f32x4_t acc[C::kSubM][C::kSubN];
#pragma unroll
    for (int i = 0; i < C::kSubM; ++i)
#pragma unroll
        for (int j = 0; j < C::kSubN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    uint4 ra1[C::kQA1], ra2[C::kQA2][C::kVA2], rb1[C::kQB1][C::kVB1], rb2[C::kQB];

    // ---- global -> registers: stage s (reduction indices 32 s .. 32 s + 31 of both components)
    auto fetch = [&](int s) {
        const uint32_t kk = (uint32_t)((s + kofs) * kStageK);
        if constexpr (ONLY != 2) {
#pragma unroll
            for (int q = 0; q < C::kQA1; ++q) ra1[q] = bload16(rA, voA1[q], kk * 2u);
        }
#pragma unroll
        for (int q = 0; q < (kComp1Only ? 0 : C::kQA2); ++q) {
            if constexpr (IN_T) {
#pragma unroll
                for (int d = 0; d < D; ++d) ra2[q][d] = bload16(rA, voA2[q] + d * 16u, kk * D * 2u);
            } else {
                ra2[q][0] = bload16(rA2, voA2[q], kk * 2u);
            }
        }
        const uint32_t kb = W_T ? kk * (uint32_t)bn * 2u : kk * 2u;
#pragma unroll
        for (int q = 0; q < (ONLY == 2 ? 0 : C::kQB1); ++q)
#pragma unroll
            for (int d = 0; d < C::kVB1; ++d) rb1[q][d] = bload16(rW1, voB1[q] + d * 16u, kb);
#pragma unroll
        for (int q = 0; q < (kComp1Only ? 0 : C::kQB); ++q) rb2[q] = bload16(rW2, voB2[q], kb);
    };

    // ---- registers -> LDS stage buffer
    auto stash = [&](unsigned char *buf) {
#pragma unroll
        for (int q = 0; q < (ONLY == 2 ? 0 : C::kQA1); ++q)
            if (C::kRowChunks % T == 0 || okA1[q]) *reinterpret_cast<uint4 *>(buf + loA1[q]) = ra1[q];
#pragma unroll
        for (int q = 0; q < (kComp1Only ? 0 : C::kQA2); ++q) {
            if (C::kUnitsA2 % T != 0 && !okA2[q]) continue;
            if constexpr (IN_T) {
                uint4 span[D];
#pragma unroll
                for (int d = 0; d < D; ++d) span[d] = ra2[q][d];
                if constexpr (OUT_T)
                    deinterleave_all<D>(span, reinterpret_cast<uint16_t *>(buf + loA2[q]), C::kSlab / 2);
                else   // only residue g1 feeds this tile
                    *reinterpret_cast<uint4 *>(buf + loA2[q]) = deinterleave_uniform<D>(span, g1);
            } else {
                *reinterpret_cast<uint4 *>(buf + loA2[q]) = ra2[q][0];
            }
        }
#pragma unroll
        for (int q = 0; q < (ONLY == 2 ? 0 : C::kQB1); ++q) {
            if (C::kUnitsB1 % T == 0 || okB1[q]) {
                if constexpr (C::kB1Chunks) {
                    uint4 span[D];
#pragma unroll
                    for (int d = 0; d < D; ++d) span[d] = rb1[q][d];
                    deinterleave_all<D>(span, reinterpret_cast<uint16_t *>(buf + loB1[q]), C::kCPR);
                } else {
                    *reinterpret_cast<uint4 *>(buf + loB1[q]) = rb1[q][0];
                }
            }
        }
#pragma unroll
        for (int q = 0; q < (kComp1Only ? 0 : C::kQB); ++q)
            if (C::kUnitsB % T == 0 || okB2[q]) *reinterpret_cast<uint4 *>(buf + loB2[q]) = rb2[q];
    };

    // ---- MFMA on one stage buffer: component 1, then component 2
    const int lr = lane & 15, lc = lane >> 4;
    const int trow = 8 * (lane >> 4) + ((lane & 15) >> 2), tcol = 4 * (lane & 3);
    auto bfrag = [&](const unsigned char *region, int j) -> bf16x8_t {
        if constexpr (W_T)
            return frag_tr((const lds_u8 *)(region + trow * C::kBRow + (wn0 + j * 16 + tcol) * 2), C::kBRow);
        else
            return *reinterpret_cast<const bf16x8_t *>(region + lds_off(wn0 + j * 16 + lr, lc) * 2);
    };
    auto compute = [&](const unsigned char *buf) {
        bf16x8_t afrag[C::kSubM];
        if constexpr (ONLY != 2) {
#pragma unroll
            for (int i = 0; i < C::kSubM; ++i)
                afrag[i] = *reinterpret_cast<const bf16x8_t *>(buf + lds_off(wm0 + i * 16 + lr, lc) * 2);
#pragma unroll
            for (int j = 0; j < C::kSubN; ++j) {
                const bf16x8_t bf = bfrag(buf + C::kOffB1, j);
#pragma unroll
                for (int i = 0; i < C::kSubM; ++i)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag[i], bf, acc[i][j], 0, 0, 0);
            }
        }
#pragma unroll
        for (int rr = 0; rr < (kComp1Only ? 0 : C::kRPW); ++rr) {
            const int r = OUT_T ? (wn0 + rr * C::kCPR) / C::kCPR : 0;
            const unsigned char *slab = buf + C::kOffA2 + r * C::kSlab;
#pragma unroll
            for (int i = 0; i < C::kSubM; ++i)
                afrag[i] = *reinterpret_cast<const bf16x8_t *>(slab + lds_off(wm0 + i * 16 + lr, lc) * 2);
            constexpr int kBlocks = OUT_T ? C::kBPR : C::kSubN;
#pragma unroll
            for (int jj = 0; jj < kBlocks; ++jj) {
                const int j = OUT_T ? rr * C::kBPR + jj : jj;
                const bf16x8_t bf = bfrag(buf + C::kOffB2, j);
#pragma unroll
                for (int i = 0; i < C::kSubM; ++i)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag[i], bf, acc[i][j], 0, 0, 0);
            }
        }
    };

    // ---- main loop: stage s uses buffer s & 1
    auto buf = [&](int idx) -> unsigned char * { return smem + (idx & 1) * C::kStage; };
    fetch(0);
    stash(buf(0));
    if (S == 1) {
        __syncthreads();
        compute(buf(0));
        __syncthreads();
    } else {
        fetch(1);
        __syncthreads();
        int s = 0;
        for (; s + 2 < S; ++s) {
            stash(buf(s + 1));
            fetch(s + 2);
            compute(buf(s));
            __syncthreads();
        }
        stash(buf(s + 1));
        compute(buf(s));
        __syncthreads();
        ++s;
        compute(buf(s));
        __syncthreads();
    }

    if constexpr (ONLY == 3)
        gemm_epilogue_as<C, BM, BN, D, OUT_T, false, true>(a, smem, acc, m0, n0, rows_left, tid, lane, wave, wn0,
                                                           split);
    else if constexpr (ONLY >= 4)
        gemm_epilogue_pad<C, BM, BN, ONLY == 4>(a, smem, acc, m0, n0, rows_left, tid, lane, wave, wn0);
    else
        gemm_epilogue<C, BM, BN, D, OUT_T>(a, smem, acc, m0, n0, rows_left, tid, lane, wave, wn0, split);
}

}  // namespace dyad
