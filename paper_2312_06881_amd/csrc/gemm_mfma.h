// The Dyad grouped GEMM on gfx950 matrix cores (bf16 in, fp32 accumulate).
//
// One workgroup computes an output tile of BM tokens x BN output features.
// Both weight components run in one K loop (the tile's accumulators take the
// BlockDiag and the BlockTrans products), so neither partial result leaves
// registers and no add or concatenation is materialised.
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
// BlockDiag stages first (with PF = 2 the components alternate and loads run
// one stage further ahead; see the main loop).  LDS holds two stage buffers: while the waves
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

#include "gemm_common.h"

namespace dyad {


template <int BM, int BN, int WGM, int WGN, int D, bool IN_T, bool OUT_T, bool W_T>
struct GemmCfg {
    static constexpr int kWaves = WGM * WGN, kWGN = WGN;
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
    // epilogue: WGM*16 rows of fp32 at a time, two such buffers
    static constexpr int kEpiRows = WGM * 16;
    static constexpr int kEpiPitch = BN + 4;
    static constexpr int kEpiElems = kEpiRows * kEpiPitch;
    static constexpr int kLdsEpi = 2 * kEpiElems * 4;
    static constexpr int kLds = kLdsOperands > kLdsEpi ? kLdsOperands : kLdsEpi;

    static_assert(BM % (16 * WGM) == 0 && BN % (16 * WGN) == 0, "wave tiles of whole MFMA blocks");
    static_assert(kRowChunks % kThreads == 0, "A row-chunks spread evenly over the threads");
    static_assert(!OUT_T || (kCPR % 16 == 0), "each MFMA column block holds one residue");
    static_assert(WN % kCPR == 0 || kCPR % WN == 0, "waves hold whole residues or parts of one");
    static_assert(kLds <= 160 * 1024, "LDS budget");
};

// GELU_IN: the pass's input is GELU(in) (a layer after a GELU, fed the
// stashed pre-activation): the activation is applied to the input operand as
// it is staged into LDS, so the activated tensor never exists in HBM.
template <int BM, int BN, int WGM, int WGN, int D, bool IN_T, bool OUT_T, bool W_T, int OCC, int PF = 1,
          bool GELU_IN = false>
__global__ void __launch_bounds__(64 * WGM * WGN, OCC)
dyad_gemm_mfma(GemmArgs a) {
    using C = GemmCfg<BM, BN, WGM, WGN, D, IN_T, OUT_T, W_T>;
    using Comp1 = std::false_type;
    using Comp2 = std::true_type;
    constexpr int T = C::kThreads;
    __shared__ __attribute__((aligned(16))) unsigned char smem[C::kLds];
    uint16_t *lds = reinterpret_cast<uint16_t *>(smem);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // work item -> (tile, split): the splits of a tile sit next to each other,
    // on one XCD, where they share the tile's token panel
    const int item = xcd_tile(blockIdx.x, a.tiles_total * a.splits);
    const int tile = item / a.splits, split = item % a.splits;
    const int64_t m0 = (int64_t)(tile / a.tiles_n) * BM;
    const int n0 = (tile % a.tiles_n) * BN;        // first output column of the tile
    const int bk = (int)a.bk, bn = (int)a.bn, Kin = (int)a.Kin;
    const int g1 = n0 / bn;                        // output block = BlockDiag group
    const int jb = n0 - g1 * bn;                   // first BlockDiag weight row
    const int ks = bk / kStageK / a.splits;        // stages per component in this split
    const int kofs = split * ks;                   // first stage of the split, per component
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

    // PF register sets of staged operands: the loads of a stage are issued PF
    // stages before its operands are written to LDS
    uint4 ras[PF][C::kRC][C::kVecPerRC2];
    uint4 rbs[PF][W_T ? C::kRBT : C::kRB][W_T ? 8 : 1];

    // ---- global -> registers (set `set`) for stage s of component 1 or 2
    auto fetch = [&](auto comp, int s, auto set) {
        constexpr bool C2 = decltype(comp)::value;
        auto &ra = ras[decltype(set)::value];
        auto &rb = rbs[decltype(set)::value];
        const uint32_t kk = (uint32_t)(((C2 ? s - ks : s) + kofs) * kStageK);
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

    // ---- registers (set `set`) -> LDS stage buffer
    // the input operand as staged: GELU(in) with GELU_IN, else in itself
    auto act = [](uint4 v) -> uint4 {
        if constexpr (GELU_IN) return gelu8(v);
        else return v;
    };
    auto stash = [&](auto comp, uint16_t *buf, auto set) {
        constexpr bool C2 = decltype(comp)::value;
        auto &ra = ras[decltype(set)::value];
        auto &rb = rbs[decltype(set)::value];
        uint16_t *bufB = buf + C::kStageA;
#pragma unroll
        for (int q = 0; q < C::kRC; ++q) {
            const int rc = tid + q * T, row = rc >> 2, c = rc & 3;
            if constexpr (!C2 || !(IN_T || OUT_T)) {
                *reinterpret_cast<uint4 *>(buf + lds_off(row, c)) = act(ra[q][0]);
            } else if constexpr (IN_T) {
                uint4 span[D];
                if constexpr (OUT_T) {
                    // every residue of the span is used: activate it whole
#pragma unroll
                    for (int d = 0; d < D; ++d) span[d] = act(ra[q][d]);
                    deinterleave_all<D>(span, buf + lds_off(row, c), C::kSlab);
                } else {   // only residue g1 feeds this tile: activate its 8 values
#pragma unroll
                    for (int d = 0; d < D; ++d) span[d] = ra[q][d];
                    *reinterpret_cast<uint4 *>(buf + lds_off(row, c)) = act(deinterleave_uniform<D>(span, g1));
                }
            } else {
#pragma unroll
                for (int r = 0; r < D; ++r)
                    *reinterpret_cast<uint4 *>(buf + r * C::kSlab + lds_off(row, c)) = act(ra[q][r]);
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
    using Set0 = std::integral_constant<int, 0>;
    using Set1 = std::integral_constant<int, 1>;
    if constexpr (PF == 2) {
        // Loads run two stages ahead, and the two components alternate: stage
        // 2j is the BlockDiag stage j, stage 2j+1 the BlockTrans stage j.  A
        // stage's kind, register set and LDS buffer all follow its parity, so
        // every iteration is straight-line code and the wait before each stash
        // leaves the next stage's loads in flight.  Iteration t stashes stage
        // t+1, fetches stage t+3 into the register set that stash freed, and
        // multiplies stage t.
        // (launched only with at least two stages per component, so that no
        // branch precedes the loop: a join there would make the compiler wait
        // for every load in flight)
        fetch(Comp1{}, 0, Set0{});
        fetch(Comp2{}, ks, Set1{});
        stash(Comp1{}, buf(0), Set0{});
        fetch(Comp1{}, 1, Set0{});
        __syncthreads();
        int j = 0;
        for (; j + 2 < ks; ++j) {
            stash(Comp2{}, buf(1), Set1{});          // BlockTrans stage j
            fetch(Comp2{}, ks + j + 1, Set1{});
            compute(Comp1{}, buf(0));                 // BlockDiag stage j
            __syncthreads();
            stash(Comp1{}, buf(0), Set0{});           // BlockDiag stage j+1
            fetch(Comp1{}, j + 2, Set0{});
            compute(Comp2{}, buf(1));                 // BlockTrans stage j
            __syncthreads();
        }
        stash(Comp2{}, buf(1), Set1{});               // j = ks - 2
        fetch(Comp2{}, ks + j + 1, Set1{});
        compute(Comp1{}, buf(0));
        __syncthreads();
        stash(Comp1{}, buf(0), Set0{});
        compute(Comp2{}, buf(1));
        __syncthreads();
        stash(Comp2{}, buf(1), Set1{});               // j = ks - 1
        compute(Comp1{}, buf(0));
        __syncthreads();
        compute(Comp2{}, buf(1));
        __syncthreads();
    } else if (ks == 1) {
        fetch(Comp1{}, 0, Set0{});
        stash(Comp1{}, buf(0), Set0{});
        fetch(Comp2{}, 1, Set0{});
        __syncthreads();
        stash(Comp2{}, buf(1), Set0{});
        compute(Comp1{}, buf(0));
        __syncthreads();
        compute(Comp2{}, buf(1));
        __syncthreads();
    } else {
        fetch(Comp1{}, 0, Set0{});
        stash(Comp1{}, buf(0), Set0{});
        fetch(Comp1{}, 1, Set0{});
        __syncthreads();
        int s = 0;
        for (; s + 2 < ks; ++s) {
            stash(Comp1{}, buf(s + 1), Set0{});
            fetch(Comp1{}, s + 2, Set0{});
            compute(Comp1{}, buf(s));
            __syncthreads();
        }
        // s = ks - 2: the stage after next is the first BlockTrans stage
        stash(Comp1{}, buf(s + 1), Set0{});
        fetch(Comp2{}, s + 2, Set0{});
        compute(Comp1{}, buf(s));
        __syncthreads();
        ++s;
        // s = ks - 1
        stash(Comp2{}, buf(s + 1), Set0{});
        fetch(Comp2{}, s + 2, Set0{});
        compute(Comp1{}, buf(s));
        __syncthreads();
        ++s;
        for (; s + 2 < S; ++s) {
            stash(Comp2{}, buf(s + 1), Set0{});
            fetch(Comp2{}, s + 2, Set0{});
            compute(Comp2{}, buf(s));
            __syncthreads();
        }
        stash(Comp2{}, buf(s + 1), Set0{});
        compute(Comp2{}, buf(s));
        __syncthreads();
        ++s;
        compute(Comp2{}, buf(s));
        __syncthreads();
    }

    gemm_epilogue<C, BM, BN, D, OUT_T>(a, smem, acc, m0, n0, rows_left, tid, lane, wave, wn0, split);
}

}  // namespace dyad
