// Weight and bias gradients of a Dyad layer on gfx950 matrix cores.
//
// dW_c[g][j][k] = sum_m dZ[m][row_c(g, j)] * X[m][col_c(g, k)] is, for each
// component c and group g, a GEMM whose reduction runs over the M tokens:
// A = dZ^T restricted to the group's rows, B = X^T restricted to its columns.
//
// Work split.  Work items are (token range "split", component, tile) and are
// numbered split-major; each XCD takes one contiguous run of them, so a split's
// slice of dZ and X is fetched from HBM by one XCD (two at a run boundary) and
// served to its workgroups from that XCD's L2.  A BlockDiag item (and a
// BlockTrans item without a stride, n_dyad = 1) is one group's BJ x BK tile.  A
// BlockTrans item whose operand is strided (columns j*D + g or k*D + g) covers
// all D groups at once, each with a (BJ/A) x (BK/B) tile for A*B = D: the
// strided columns of all groups are then one contiguous span of the input,
// loaded once with full-width loads and de-interleaved in registers, instead
// of every group reading the whole span for 1/D of it.  Every wave multiplies
// the same WJ x WK block in both kinds of item.  Each workgroup writes fp32
// partial sums to the workspace; a second kernel adds the splits in a fixed
// order, so the result is bitwise reproducible.
//
// Operands in LDS.  A stage holds 32 tokens of both operands in their natural
// token-major order: one row per token with each group's columns contiguous.
// Rows of whole 256-byte blocks have their 32-byte chunks XOR-swizzled by row
// (tr_swz), other rows are padded by 16 bytes, so that the fragment reads of
// 16 consecutive tokens spread over the banks.  The matrix cores need each lane's 8 values along
// the token axis; ds_read_b64_tr_b16 delivers exactly that from token-major
// rows (four 16-lane groups, each gathering 4 tokens x 16 columns and handing
// lane l the 4 tokens of column l), so no transpose is done in registers.
//
// Pipeline.  Two register sets of loads are in flight (stages s+2 and s+3
// while stage s is multiplied) and two LDS stage buffers alternate, so every
// load has two stages of matrix work to arrive and there is one barrier per
// stage.  Each thread owns the same load slots in every stage and issues every
// slot's loads (a slot past the stage's data loads out of range: zero, no
// memory traffic), so the wait counts are exact.
//
// Bias gradient.  In workgroups of component 1 whose column tile is the first,
// the waves also multiply their dZ fragments by a fragment of ones, which sums
// dZ over the tokens on the matrix cores; each wave of a row of waves takes
// every WKN-th fragment so the extra work is spread evenly.
#pragma once

#include "dyad_internal.h"
#include "mfma_common.h"

namespace dyad {

struct DwArgs {
    int64_t M, n_in, n_out, bi, bo;
    const uint16_t *dZ, *X;
    const uint16_t *dZ2, *X2;   // component 2's operands (dZ / X, or block-ordered copies)
    float *part;          // [splits][2][D][bo][bi]
    float *part_db;       // [splits][n_out]
    uint16_t *dW1, *dW2, *db;
    int direct;           // one split: the tiles store bf16 results, no partials
    int64_t tokens_per_split;
    int tiles_j, tiles_k; // BJ x BK tiles per (component, group)
    int splits, items;    // items = splits * 2 * D * tiles_j * tiles_k
    int want_db;
    int groups;           // D (the kernels on block-ordered operands take it at run time)
};

constexpr int kDwLdsBudget = 160 * 1024;

// Workgroup shape: WJN x WKN waves, each a WJ x WK block of 16 x 16 MFMA
// tiles; a one-group item is BJ x BK.
template <int BJ, int BK, int WJN, int WKN>
struct DwCfg {
    static constexpr int kWaves = WJN * WKN, kThreads = 64 * kWaves;
    static constexpr int WJ = BJ / WJN, WK = BK / WKN;
    static constexpr int kSubJ = WJ / 16, kSubK = WK / 16;
    static constexpr int kDbFr = (kSubJ + WKN - 1) / WKN;               // ones-products per wave
    // 8 waves run one workgroup per CU, 4 waves two; both leave 256 VGPRs a lane
    static constexpr int kMinBlocks = kWaves >= 8 ? 1 : 2;
    static_assert(WJ % 16 == 0 && WK % 16 == 0, "whole MFMA tiles per wave");
};

// LDS row of NG groups of w columns: groups of whole 256-byte blocks are
// swizzled (tr_swz), other rows keep a 16-byte pad.
constexpr bool dw_swz(int w) { return (w * 2) % 256 == 0; }
constexpr int dw_row(int ng, int w) { return ng * w * 2 + (dw_swz(w) ? 0 : 16); }

// Item layout: NG = GA * GB groups on a GA x GB grid of wave blocks, each group
// JT x KT; LDS rows hold the NG groups' columns side by side.
template <int BJ, int BK, int GA, int GB>
struct DwLayout {
    static constexpr int NG = GA * GB, JT = BJ / GA, KT = BK / GB;
    static constexpr bool kSwzA = dw_swz(JT), kSwzB = dw_swz(KT);
    static constexpr int kRowA = dw_row(NG, JT), kRowB = dw_row(NG, KT);
    static constexpr int kRegionA = kStageK * kRowA;
    static constexpr int kStageBytes = kRegionA + kStageK * kRowB;
};

// Group grid of an all-groups item: GA * GB = D with GA | WJN and GB | WKN,
// both stage buffers within the LDS share of a workgroup, least LDS traffic
// (GA*BK + GB*BJ columns per token); 0 when there is none.
template <int D, int BJ, int BK, int WJN, int WKN>
constexpr int mg_gb() {
    int best = 0, cost = 1 << 30;
    for (int gb = 1; gb <= D; gb *= 2) {
        if (D % gb != 0) break;
        const int ga = D / gb;
        if (WJN % ga || WKN % gb || BJ % (16 * ga) || BK % (16 * gb)) continue;
        const int bytes = 2 * kStageK * (dw_row(D, BJ / ga) + dw_row(D, BK / gb));
        if (bytes * DwCfg<BJ, BK, WJN, WKN>::kMinBlocks > kDwLdsBudget) continue;
        const int c = ga * BK + gb * BJ;
        if (c < cost) { cost = c; best = gb; }
    }
    return best;
}

// One operand side of an item's stage: NG groups of W columns each.
//   plain:        16-byte units of 8 columns, one load each;
//   strided, one group:  8 columns (j..j+7)*D + g, eight 2-byte loads;
//   strided, all groups: chunks of NJ columns of every group (NJ*D consecutive
//                 input columns, 16-byte loads) split into one NJ-column piece
//                 per group.
template <int D, int NG, int W, bool SPAN, int T>
struct DwSide {
    static constexpr int kKind = !SPAN ? 0 : (NG == 1 ? 1 : 2);
    static constexpr int kNJ = D >= 8 ? 32 / D : 8;
    static constexpr int kVec = kKind == 2 ? kNJ * D / 8 : 1;           // 16-byte loads per item
    static constexpr int kPerRow = kKind == 2 ? W / kNJ : NG * W / 8;   // items per token row
    static constexpr int kItems = kStageK * kPerRow;
    static constexpr int kSlots = (kItems + T - 1) / T;
    static_assert(kKind != 2 || NG == D, "a strided chunk feeds every group");
};

// Eight bf16 at base + voff + 2*D*e (e = 0..7), packed into 16 bytes.
template <int D>
__device__ __forceinline__ uint4 load_strided8(__amdgpu_buffer_rsrc_t r, uint32_t voff) {
    uint32_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) h[e] = __builtin_amdgcn_raw_buffer_load_b16(r, (int)(voff + 2u * D * e), 0, 0);
    return make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
}

// Residue R of NJ consecutive column groups held in NJ*D/8 16-byte vectors
// (input column j*D + r, residue fastest): the NJ values, packed.
template <int D, int NJ, int R>
__device__ __forceinline__ void piece_of(const uint4 *v, uint32_t (&o)[NJ / 2]) {
#pragma unroll
    for (int w = 0; w < NJ / 2; ++w) {
        const int e0 = (2 * w) * D + R, e1 = (2 * w + 1) * D + R;
        const uint32_t lo = word_of(v[e0 >> 3], (e0 & 7) >> 1);
        const uint32_t hi = word_of(v[e1 >> 3], (e1 & 7) >> 1);
        o[w] = __builtin_amdgcn_perm(hi, lo, perm_sel((e0 & 1) * 2, 4 + (e1 & 1) * 2));
    }
}

// Every residue's piece of a chunk into its group's columns: piece R at row
// byte lbyte + R * step of the (swizzled) row at `row`.
template <int D, int NJ, bool SWZ, int R = 0>
__device__ __forceinline__ void stash_pieces(const uint4 *v, unsigned char *row, int sw, int lbyte, int step) {
    uint32_t o[NJ / 2];
    piece_of<D, NJ, R>(v, o);
    // with the swizzle, step is a whole number of 256-byte blocks: the pieces stay step apart
    unsigned char *p = row + (SWZ ? tr_swz(sw, lbyte) : lbyte) + R * step;
    if constexpr (NJ == 8) *reinterpret_cast<uint4 *>(p) = make_uint4(o[0], o[1], o[2], o[3]);
    else if constexpr (NJ == 4) *reinterpret_cast<uint2 *>(p) = make_uint2(o[0], o[1]);
    else *reinterpret_cast<uint32_t *>(p) = o[0];
    if constexpr (R + 1 < D) stash_pieces<D, NJ, SWZ, R + 1>(v, row, sw, lbyte, step);
}

// Load slots of one side: global byte offsets (within a stage's rows) and LDS
// byte offsets (within the side's region) of this thread's items.
template <class S>
struct DwSlots {
    uint32_t vo[S::kSlots], lo[S::kSlots];   // lo: swizzled, or (strided chunks) the row start
    int lb[S::kSlots], sw[S::kSlots];          // strided chunks: unswizzled row byte and row swizzle
    bool ok[S::kSlots];
    uint4 r[2][S::kSlots][S::kVec];   // two stages in flight
};

// One item: component C2, groups g0.. (all groups when MG), tile (jt, kt) in
// units of the item's per-group JT x KT tile.  ONE: the split holds at most
// one 32-token stage (small batches), which runs straight through -- the
// pipelined loop would also issue the loads of four stages that read only
// zeros, and at 16 tokens those loads, not the stores, set the time.  Its own
// kernel instance, so the pipelined kernel's registers are unaffected.
// XG: the layer's input is GELU(X) (a layer after a GELU, given the stashed
// pre-activation): the activation is applied to the X operand as it is staged.
template <int D, int BJ, int BK, int WJN, int WKN, bool IN_T, bool OUT_T, bool C2, bool MG, bool ONE, bool XG>
__device__ __forceinline__ void dw_tile(const DwArgs &a, unsigned char *smem, int split, int g, int jt, int kt) {
    using C = DwCfg<BJ, BK, WJN, WKN>;
    constexpr int GB = MG ? mg_gb<D, BJ, BK, WJN, WKN>() : 1;
    constexpr int GA = MG ? D / GB : 1;
    using L = DwLayout<BJ, BK, GA, GB>;
    constexpr int T = C::kThreads;
    constexpr bool SPAN_A = C2 && OUT_T && D > 1;    // dZ columns j*D + g
    constexpr bool SPAN_B = C2 && IN_T && D > 1;     // X columns k*D + g
    using SA = DwSide<D, L::NG, L::JT, SPAN_A, T>;
    using SB = DwSide<D, L::NG, L::KT, SPAN_B, T>;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform, kept in a scalar register
    const int j0 = jt * L::JT, k0 = kt * L::KT;
    const int bo = (int)a.bo, bi = (int)a.bi;
    const uint32_t n_out = (uint32_t)a.n_out, n_in = (uint32_t)a.n_in;

    const int64_t t_begin = (int64_t)split * a.tokens_per_split;
    int64_t t_end = t_begin + a.tokens_per_split;
    if (t_end > a.M) t_end = a.M;
    int stages = t_end > t_begin ? (int)((t_end - t_begin + kStageK - 1) / kStageK) : 0;
    stages = (stages + 1) & ~1;   // whole stage pairs; the extra stage reads zeros

    // slot setup of one side: W columns per group starting at w0, groups of bw
    // columns in the input (plain), leading dimension ld
    auto setup = [&](auto side, auto swz, auto &sl, int w0, int bw, uint32_t ld, uint32_t region, uint32_t row) {
        using S = decltype(side);
        constexpr bool SWZ = decltype(swz)::value;
        constexpr int W = S::kPerRow * (S::kKind == 2 ? S::kNJ : 8) / (S::kKind == 0 ? L::NG : 1);
#pragma unroll
        for (int q = 0; q < S::kSlots; ++q) {
            const int i = tid + q * T;
            const int t = i / S::kPerRow, c = i % S::kPerRow;
            sl.ok[q] = i < S::kItems;
            uint32_t col, lcol;
            if constexpr (S::kKind == 0) {
                const int gg = c / (W / 8), cc = c % (W / 8);
                col = (uint32_t)((L::NG == 1 ? g : gg) * bw + w0 + 8 * cc);
                lcol = (uint32_t)(gg * W + 8 * cc);
            } else if constexpr (S::kKind == 1) {
                col = (uint32_t)((w0 + 8 * c) * D + g);
                lcol = (uint32_t)(8 * c);
            } else {
                col = (uint32_t)((w0 + S::kNJ * c) * D);
                lcol = (uint32_t)(S::kNJ * c);
            }
            sl.vo[q] = sl.ok[q] ? (uint32_t)t * ld * 2u + col * 2u : kNoLoad;
            sl.sw[q] = tr_sw(t);
            sl.lb[q] = (int)lcol * 2;
            sl.lo[q] = region + (uint32_t)t * row +
                       (S::kKind == 2 ? 0u : (uint32_t)(SWZ ? tr_swz(sl.sw[q], (int)lcol * 2) : (int)lcol * 2));
        }
    };
    DwSlots<SA> sa;
    DwSlots<SB> sb;
    setup(SA{}, std::bool_constant<L::kSwzA>{}, sa, j0, bo, n_out, 0u, (uint32_t)L::kRowA);
    setup(SB{}, std::bool_constant<L::kSwzB>{}, sb, k0, bi, n_in, (uint32_t)L::kRegionA, (uint32_t)L::kRowB);

    // ---- global -> registers: stage s into register set P.  Buffers start at
    // the stage's first token and end at the split's end, so tokens past it
    // read as zero.
    auto fetch_side = [&](auto side, auto &sl, auto set, __amdgpu_buffer_rsrc_t r, uint32_t rows) {
        using S = decltype(side);
        constexpr int P = decltype(set)::value;
#pragma unroll
        for (int q = 0; q < S::kSlots; ++q) {
            // one-stage splits skip the token rows past the batch (they read zero)
            // instead of issuing their loads
            if (ONE && (uint32_t)((tid + q * T) / S::kPerRow) >= rows) {
#pragma unroll
                for (int v = 0; v < (S::kKind == 1 ? 1 : S::kVec); ++v) sl.r[P][q][v] = make_uint4(0u, 0u, 0u, 0u);
            } else if constexpr (S::kKind == 1) {
                sl.r[P][q][0] = load_strided8<D>(r, sl.vo[q]);
            } else {
#pragma unroll
                for (int v = 0; v < S::kVec; ++v) sl.r[P][q][v] = bload16(r, sl.vo[q] + 16u * v, 0);
            }
        }
    };
    auto fetch = [&](auto set, int s) {
        const int64_t tok = t_begin + (int64_t)s * kStageK;
        const int64_t left = t_end - tok;
        const uint32_t rows = left <= 0 ? 0u : (uint32_t)(left < kStageK ? left : kStageK);
        const int64_t base = left <= 0 ? 0 : tok;
        fetch_side(SA{}, sa, set, buffer_rsrc((C2 ? a.dZ2 : a.dZ) + base * a.n_out, rows * n_out * 2u), rows);
        fetch_side(SB{}, sb, set, buffer_rsrc((C2 ? a.X2 : a.X) + base * a.n_in, rows * n_in * 2u), rows);
    };
    // ---- registers -> LDS stage buffer
    auto stash_side = [&](auto side, auto swz, auto &sl, auto set, unsigned char *buf, auto xg) {
        using S = decltype(side);
        constexpr bool SWZ = decltype(swz)::value;
        constexpr int P = decltype(set)::value;
        constexpr int W = S::kKind == 2 ? S::kPerRow * S::kNJ : 0;
#pragma unroll
        for (int q = 0; q < S::kSlots; ++q) {
            if constexpr (decltype(xg)::value) {
                // GELU(X): every loaded value feeds some group, so whole vectors are activated
#pragma unroll
                for (int v = 0; v < (S::kKind == 1 ? 1 : S::kVec); ++v) sl.r[P][q][v] = gelu8(sl.r[P][q][v]);
            }
            if (S::kItems % T == 0 || sl.ok[q]) {
                if constexpr (S::kKind == 2) stash_pieces<D, S::kNJ, SWZ>(sl.r[P][q], buf + sl.lo[q], sl.sw[q], sl.lb[q], 2 * W);
                else *reinterpret_cast<uint4 *>(buf + sl.lo[q]) = sl.r[P][q][0];
            }
        }
    };
    auto stash = [&](auto set, unsigned char *buf) {
        stash_side(SA{}, std::bool_constant<L::kSwzA>{}, sa, set, buf, std::false_type{});
        stash_side(SB{}, std::bool_constant<L::kSwzB>{}, sb, set, buf, std::bool_constant<XG>{});
    };

    f32x4_t acc[C::kSubJ][C::kSubK];
#pragma unroll
    for (int i = 0; i < C::kSubJ; ++i)
#pragma unroll
        for (int j = 0; j < C::kSubK; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    f32x4_t dacc[C::kDbFr];
#pragma unroll
    for (int d = 0; d < C::kDbFr; ++d) dacc[d] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const bool do_db = !C2 && a.want_db && kt == 0;

    // wave -> group of the item and position inside the group's tile
    const int wj = wave / WKN, wk = wave % WKN;
    constexpr int kWJG = WJN / GA, kWKG = WKN / GB;     // waves per group along j, k
    const int gw = (wj / kWJG) * GB + wk / kWKG;
    const int wj0 = (wj % kWJG) * C::WJ, wk0 = (wk % kWKG) * C::WK;
    // transpose-read lane offsets: token row 8*(lane/16) + (lane%16)/4, column 4*(lane%4)
    const int trow = 8 * (lane >> 4) + ((lane & 15) >> 2), tcol = 4 * (lane & 3);
    // (rows trow and trow + 4 share a swizzle, so frag_tr's second read is one 4-row step on)
    const int tsw = tr_sw(trow);
    const int rowA = trow * L::kRowA, colA = (gw * L::JT + wj0 + tcol) * 2;
    const int rowB = L::kRegionA + trow * L::kRowB, colB = (gw * L::KT + wk0 + tcol) * 2;
    const bf16x8_t ones = {(__bf16)1.0f, (__bf16)1.0f, (__bf16)1.0f, (__bf16)1.0f,
                           (__bf16)1.0f, (__bf16)1.0f, (__bf16)1.0f, (__bf16)1.0f};

    auto compute = [&](const unsigned char *buf) {
        const lds_u8 *b = (const lds_u8 *)buf;
        bf16x8_t af[C::kSubJ];
#pragma unroll
        for (int i = 0; i < C::kSubJ; ++i)
            af[i] = frag_tr(b + rowA + (L::kSwzA ? tr_swz(tsw, colA + 32 * i) : colA + 32 * i), L::kRowA);
#pragma unroll
        for (int j = 0; j < C::kSubK; ++j) {
            const bf16x8_t bf =
                frag_tr(b + rowB + (L::kSwzB ? tr_swz(tsw, colB + 32 * j) : colB + 32 * j), L::kRowB);
#pragma unroll
            for (int i = 0; i < C::kSubJ; ++i)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf, acc[i][j], 0, 0, 0);
        }
        if (do_db) {
#pragma unroll
            for (int i = 0; i < C::kSubJ; ++i)
                if (i % WKN == wk)
                    dacc[i / WKN] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], ones, dacc[i / WKN], 0, 0, 0);
        }
    };

    using Set0 = std::integral_constant<int, 0>;
    using Set1 = std::integral_constant<int, 1>;
    unsigned char *buf0 = smem, *buf1 = smem + L::kStageBytes;
    if constexpr (ONE) {
        fetch(Set0{}, 0);
        stash(Set0{}, buf0);
        __syncthreads();
        compute(buf0);
        __syncthreads();
    } else if (stages > 0) {
        fetch(Set0{}, 0);
        fetch(Set1{}, 1);
        stash(Set0{}, buf0);
        fetch(Set0{}, 2);
        __syncthreads();
        for (int s = 0; s < stages; s += 2) {
            // buf0: stage s; in flight: set 1 = stage s+1, set 0 = stage s+2
            stash(Set1{}, buf1);
            fetch(Set1{}, s + 3);
            compute(buf0);
            __syncthreads();
            // buf1: stage s+1; in flight: set 0 = stage s+2, set 1 = stage s+3
            stash(Set0{}, buf0);
            fetch(Set0{}, s + 4);
            compute(buf1);
            __syncthreads();
        }
    }

    // one split: bf16 results straight to dW1 / dW2 / db; else fp32 partial
    // sums -> workspace [split][comp][g][j][k], added by dyad_dw_reduce
    const int gout = MG ? gw : g;
    const int64_t per_comp = (int64_t)a.groups * bo * bi;
    if (a.direct) {
        // each 16-row slice of the wave's block goes through the wave's own
        // LDS area (the stage buffers are free after the last barrier) and
        // leaves as 16-byte row pieces
        uint16_t *dst = (C2 ? a.dW2 : a.dW1) + (int64_t)gout * bo * bi;
        uint16_t *slice = reinterpret_cast<uint16_t *>(smem) + wave * 16 * C::WK;
        constexpr int kPieces = 16 * C::WK / 8;
#pragma unroll
        for (int i = 0; i < C::kSubJ; ++i) {
#pragma unroll
            for (int j = 0; j < C::kSubK; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    slice[((lane >> 4) * 4 + v) * C::WK + j * 16 + (lane & 15)] = f32_to_bf16(acc[i][j][v]);
#pragma unroll
            for (int c0 = 0; c0 < kPieces; c0 += 64) {
                const int c = c0 + lane;
                if (kPieces % 64 != 0 && c >= kPieces) break;
                const int r = c / (C::WK / 8), q = c % (C::WK / 8);
                const uint4 v = *reinterpret_cast<const uint4 *>(slice + r * C::WK + q * 8);
                *reinterpret_cast<uint4 *>(dst + (int64_t)(j0 + wj0 + i * 16 + r) * bi + k0 + wk0 + q * 8) = v;
            }
        }
    } else {
        float *dst = a.part + ((int64_t)split * 2 + (C2 ? 1 : 0)) * per_comp + (int64_t)gout * bo * bi;
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
    }
    if (do_db && (lane & 15) == 0) {
        // every column of a ones-product holds the row sums; lane 16r holds rows 4r..4r+3
#pragma unroll
        for (int i = 0; i < C::kSubJ; ++i)
            if (i % WKN == wk) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int64_t f = g * bo + j0 + wj0 + i * 16 + (lane >> 4) * 4 + v;
                    if (a.direct) a.db[f] = f32_to_bf16(dacc[i / WKN][v]);
                    else a.part_db[(int64_t)split * a.n_out + f] = dacc[i / WKN][v];
                }
            }
    }
}

template <int D, int BJ, int BK, int WJN, int WKN, bool IN_T, bool OUT_T>
struct DwKernel {
    using C = DwCfg<BJ, BK, WJN, WKN>;
    static constexpr int kGB = mg_gb<D, BJ, BK, WJN, WKN>();
    // BlockTrans items cover all groups when an operand is strided and a group grid exists
    static constexpr bool kMG = D > 1 && (IN_T || OUT_T) && kGB > 0;
    static constexpr int kLds1 = 2 * DwLayout<BJ, BK, 1, 1>::kStageBytes;
    static constexpr int kLds2 = kMG ? 2 * DwLayout<BJ, BK, D / (kGB ? kGB : 1), kGB ? kGB : 1>::kStageBytes : kLds1;
    static constexpr int kLds = kLds1 > kLds2 ? kLds1 : kLds2;
    static_assert(kLds * C::kMinBlocks <= kDwLdsBudget, "LDS budget");
    static_assert(kLds >= C::kWaves * 16 * C::WK * 2, "the direct epilogue's slices fit the stage buffers");
};

template <int D, int BJ, int BK, int WJN, int WKN, bool IN_T, bool OUT_T, bool ONE, bool XG = false>
__global__ void __launch_bounds__(64 * WJN * WKN, (DwCfg<BJ, BK, WJN, WKN>::kMinBlocks))
dyad_dw_mfma(DwArgs a) {
    using K = DwKernel<D, BJ, BK, WJN, WKN, IN_T, OUT_T>;
    __shared__ __attribute__((aligned(16))) unsigned char smem[K::kLds];
    // work item -> (split, component, tile), split-major
    const int item = xcd_tile(blockIdx.x, a.items);
    const int tiles = a.groups * a.tiles_j * a.tiles_k;   // items per component and split
    const int split = item / (2 * tiles);
    const int t2 = item % (2 * tiles);
    const int comp = t2 / tiles, t = t2 % tiles;
    if (comp == 0 || !K::kMG) {
        const int kt = t % a.tiles_k;
        const int jt = (t / a.tiles_k) % a.tiles_j;
        const int g = t / (a.tiles_k * a.tiles_j);
        if (comp == 0) dw_tile<D, BJ, BK, WJN, WKN, IN_T, OUT_T, false, false, ONE, XG>(a, smem, split, g, jt, kt);
        else dw_tile<D, BJ, BK, WJN, WKN, IN_T, OUT_T, true, false, ONE, XG>(a, smem, split, g, jt, kt);
    } else if constexpr (K::kMG) {
        // all groups: (D / GB) * tiles_j x GB * tiles_k tiles of (BJ / GA) x (BK / GB)
        const int nk = K::kGB * a.tiles_k;
        dw_tile<D, BJ, BK, WJN, WKN, IN_T, OUT_T, true, true, ONE, XG>(a, smem, split, 0, t / nk, t % nk);
    }
}

// Adds the splits in order 0..S-1 and writes dW1, dW2 (and db) in bf16.
__global__ void __launch_bounds__(256) dyad_dw_reduce(const float *part, const float *part_db, int splits, int64_t per_comp,
                               int64_t n_out, uint16_t *dW1, uint16_t *dW2, uint16_t *db);

struct DwPlan {
    int BJ, BK, WJN, WKN, tiles_j, tiles_k, splits;
    int64_t tokens_per_split;
};

// Launches the weight-gradient kernel of plan `pl` and the split reduction.
template <int D, int BJ, int BK, int WJN, int WKN, bool IN_T, bool OUT_T, bool XG = false>
hipError_t launch_dw_cfg(const DwPass &p, const DwPlan &pl, hipStream_t s) {
    using C = DwCfg<BJ, BK, WJN, WKN>;
    DwArgs a;
    a.M = p.M; a.n_in = p.n_in; a.n_out = p.n_out; a.bi = p.bi; a.bo = p.bo;
    a.dZ = static_cast<const uint16_t *>(p.dZ);
    a.X = static_cast<const uint16_t *>(p.X);
    a.dZ2 = static_cast<const uint16_t *>(p.dZ2 ? p.dZ2 : p.dZ);
    a.X2 = static_cast<const uint16_t *>(p.X2 ? p.X2 : p.X);
    a.direct = pl.splits == 1;
    a.part = a.direct ? nullptr : static_cast<float *>(p.ws);
    a.part_db = a.direct ? nullptr : a.part + (int64_t)pl.splits * 2 * p.D * p.bo * p.bi;
    a.dW1 = static_cast<uint16_t *>(p.dW1);
    a.dW2 = static_cast<uint16_t *>(p.dW2);
    a.db = static_cast<uint16_t *>(p.db);
    a.tokens_per_split = pl.tokens_per_split;
    a.tiles_j = pl.tiles_j; a.tiles_k = pl.tiles_k;
    a.splits = pl.splits;
    a.groups = (int)p.D;
    a.items = pl.splits * 2 * a.groups * pl.tiles_j * pl.tiles_k;
    a.want_db = p.db != nullptr;
    if (pl.tokens_per_split >= p.M && p.M <= kStageK)   // one split of one stage
        dyad_dw_mfma<D, BJ, BK, WJN, WKN, IN_T, OUT_T, true, XG><<<(unsigned)a.items, C::kThreads, 0, s>>>(a);
    else
        dyad_dw_mfma<D, BJ, BK, WJN, WKN, IN_T, OUT_T, false, XG><<<(unsigned)a.items, C::kThreads, 0, s>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.direct) return e;
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

// Tile configurations, preferred first: BJ x BK weight tile on WJN x WKN waves.
// The last, sixteen waves, exists for all-groups items at n_dyad 16.
#define DYAD_DW_CONFIGS(X)  \
    X(256, 256, 2, 4)       \
    X(192, 256, 2, 4)       \
    X(256, 192, 4, 2)       \
    X(256, 128, 4, 2)       \
    X(128, 256, 2, 4)       \
    X(128, 128, 2, 2)       \
    X(128, 64, 2, 2)        \
    X(64, 128, 2, 2)        \
    X(64, 64, 2, 2)         \
    X(128, 128, 4, 4)

// Whether config (BJ, BK, WJN, WKN) has an all-groups layout at n_dyad D.
inline bool dw_mg_available(int D, int BJ, int BK, int WJN, int WKN) {
#define DYAD_DW_MG(J_, K_, WJ_, WK_)                                                     \
    if (BJ == J_ && BK == K_ && WJN == WJ_ && WKN == WK_) switch (D) {                   \
        case 2: return mg_gb<2, J_, K_, WJ_, WK_>() > 0;                                 \
        case 4: return mg_gb<4, J_, K_, WJ_, WK_>() > 0;                                 \
        case 8: return mg_gb<8, J_, K_, WJ_, WK_>() > 0;                                 \
        case 16: return mg_gb<16, J_, K_, WJ_, WK_>() > 0;                               \
        default: return false;                                                           \
    }
    DYAD_DW_CONFIGS(DYAD_DW_MG)
#undef DYAD_DW_MG
    return false;
}

// Per-variant launchers (one translation unit each); launch_dw_plain: both
// components on block-ordered operands (any n_dyad).
hipError_t launch_dw_plain(const DwPass &p, const DwPlan &pl, hipStream_t s);
hipError_t launch_dw_it(const DwPass &p, const DwPlan &pl, hipStream_t s);
hipError_t launch_dw_ot(const DwPass &p, const DwPlan &pl, hipStream_t s);
hipError_t launch_dw_dt(const DwPass &p, const DwPlan &pl, hipStream_t s);
// the same with X = GELU(X as passed) (DwPass::gelu_x)
hipError_t launch_dw_xg_it(const DwPass &p, const DwPlan &pl, hipStream_t s);
hipError_t launch_dw_xg_ot(const DwPass &p, const DwPlan &pl, hipStream_t s);
hipError_t launch_dw_xg_dt(const DwPass &p, const DwPlan &pl, hipStream_t s);

template <bool IN_T, bool OUT_T, bool XG = false>
hipError_t launch_dw_variant(const DwPass &p, const DwPlan &pl, hipStream_t s) {
#define DYAD_DW_CASE(J_, K_, WJ_, WK_)                                                      \
    if (pl.BJ == J_ && pl.BK == K_ && pl.WJN == WJ_ && pl.WKN == WK_) switch (p.D) {        \
        case 1: return launch_dw_cfg<1, J_, K_, WJ_, WK_, IN_T, OUT_T, XG>(p, pl, s);       \
        case 2: return launch_dw_cfg<2, J_, K_, WJ_, WK_, IN_T, OUT_T, XG>(p, pl, s);       \
        case 3: if constexpr (XG) return hipErrorNotSupported;                              \
                else return launch_dw_cfg<3, J_, K_, WJ_, WK_, IN_T, OUT_T, false>(p, pl, s); \
        case 4: return launch_dw_cfg<4, J_, K_, WJ_, WK_, IN_T, OUT_T, XG>(p, pl, s);       \
        case 6: if constexpr (XG) return hipErrorNotSupported;                              \
                else return launch_dw_cfg<6, J_, K_, WJ_, WK_, IN_T, OUT_T, false>(p, pl, s); \
        case 8: return launch_dw_cfg<8, J_, K_, WJ_, WK_, IN_T, OUT_T, XG>(p, pl, s);       \
        case 16: return launch_dw_cfg<16, J_, K_, WJ_, WK_, IN_T, OUT_T, XG>(p, pl, s);     \
        default: return hipErrorNotSupported;                                               \
    }
    DYAD_DW_CONFIGS(DYAD_DW_CASE)
#undef DYAD_DW_CASE
    return hipErrorNotSupported;
}

}  // namespace dyad
