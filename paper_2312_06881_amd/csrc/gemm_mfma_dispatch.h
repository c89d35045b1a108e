// Host-side tile choice and launch for the MFMA grouped GEMM (gemm_mfma.h).
#pragma once

#include "gemm_mfma.h"
#include "gemm_mfma2.h"

namespace dyad {


// Workgroups per CU: two 4-wave workgroups when both the tile's LDS and its
// registers fit twice (two caps a wave at 256 VGPRs, so accumulators above 128
// per lane need one); an 8-wave workgroup runs alone.
template <class C>
constexpr int occupancy() {
    const int acc_per_lane = C::WM * C::WN / 64;
    return (C::kThreads <= 256 && (160 * 1024) / C::kLds >= 2 && acc_per_lane <= 128) ? 2 : 1;
}

// Splits of the reduction for a launch of `tiles` output tiles: none when the
// tiles alone fill the GPU; otherwise the fewest that give about 384 work
// items, each split keeping at least `min_stages` stages per component, and no
// more than keep the fp32 partial sums (written and read once) within the
// bytes of the two weight tensors.
inline int gemm_splits(const GemmPass &p, int64_t tiles, int min_stages) {
    if (tiles >= 192) return 1;
    const int ks = (int)(p.bk / kStageK);
    const int64_t wbytes = 4 * p.D * p.bn * p.bk;
    int best = 1;
    for (int sp = 2; sp * min_stages <= ks; ++sp) {
        if (ks % sp != 0) continue;
        if ((int64_t)sp * p.M * p.Nout * 8 > wbytes) break;
        best = sp;
        if (tiles * sp >= 384) break;
    }
    return best;
}

// Workspace for `splits` partial sums of pass p on stream s; false (and no
// split) when none can be had.
inline bool gemm_split_ws(const GemmPass &p, int splits, hipStream_t s, GemmArgs &a) {
    a.part = nullptr;
    a.splits = 1;
    a.slice0 = 0;
    a.unperm = 0;
    if (splits <= 1) return false;
    void *ws = nullptr;
    if (split_workspace(s, (size_t)splits * (size_t)p.M * (size_t)p.Nout * sizeof(float), &ws) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    a.part = static_cast<float *>(ws);
    a.splits = splits;
    return true;
}

template <int BM, int BN, int WGM, int WGN, int D, bool IN_T, bool OUT_T, bool W_T, int PF = 1, bool GELU_IN = false>
hipError_t launch_tile(const GemmPass &p, hipStream_t s) {
    using C = GemmCfg<BM, BN, WGM, WGN, D, IN_T, OUT_T, W_T>;
    GemmArgs a{};
    // buffer offsets are 32-bit: one token panel of the input and of the output,
    // and one weight tensor, must fit
    if ((int64_t)BM * p.Kin * 2 >= ((int64_t)1 << 31) || (int64_t)BM * p.Nout * 2 >= ((int64_t)1 << 31) ||
        2 * p.D * p.bn * p.bk >= ((int64_t)1 << 31))
        return hipErrorNotSupported;
    if (PF == 2 && p.bk < 2 * kStageK) return hipErrorNotSupported;   // two stages per component
    a.M = p.M; a.Kin = p.Kin; a.Nout = p.Nout; a.bk = p.bk; a.bn = p.bn; a.D = p.D;
    a.in = static_cast<const uint16_t *>(p.in);
    a.W1 = static_cast<const uint16_t *>(p.W1);
    a.W2 = static_cast<const uint16_t *>(p.W2);
    a.bias = static_cast<const uint16_t *>(p.bias);
    a.h_in = static_cast<const uint16_t *>(p.h_in);
    a.out = static_cast<uint16_t *>(p.out);
    a.h_out = static_cast<uint16_t *>(p.h_out);
    a.epilogue = p.epilogue;
    const int64_t tiles_m = (p.M + BM - 1) / BM;
    const int64_t tiles_n = p.Nout / BN;
    if (tiles_m * tiles_n >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    a.tiles_n = (int)tiles_n;
    a.tiles_total = (int)(tiles_m * tiles_n);
    gemm_split_ws(p, gemm_splits(p, a.tiles_total, PF), s, a);
    dyad_gemm_mfma<BM, BN, WGM, WGN, D, IN_T, OUT_T, W_T, occupancy<C>(), PF, GELU_IN>
        <<<a.tiles_total * a.splits, C::kThreads, 0, s>>>(a);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && a.part) e = launch_split_reduce(p, a.part, a.splits, s);
    return e;
}

// Launch of a fused-stage tile (gemm_mfma2.h).
template <int BM, int BN, int WGM, int WGN, int D, bool IN_T, bool OUT_T, bool W_T>
hipError_t launch_tile2(const GemmPass &p, hipStream_t s) {
    using C = Gemm2Cfg<BM, BN, WGM, WGN, D, IN_T, OUT_T, W_T>;
    GemmArgs a{};
    if ((int64_t)BM * p.Kin * 2 >= ((int64_t)1 << 31) || (int64_t)BM * p.Nout * 2 >= ((int64_t)1 << 31) ||
        2 * p.D * p.bn * p.bk >= ((int64_t)1 << 31))
        return hipErrorNotSupported;
    a.M = p.M; a.Kin = p.Kin; a.Nout = p.Nout; a.bk = p.bk; a.bn = p.bn; a.D = p.D;
    a.in = static_cast<const uint16_t *>(p.in);
    a.W1 = static_cast<const uint16_t *>(p.W1);
    a.W2 = static_cast<const uint16_t *>(p.W2);
    a.bias = static_cast<const uint16_t *>(p.bias);
    a.h_in = static_cast<const uint16_t *>(p.h_in);
    a.out = static_cast<uint16_t *>(p.out);
    a.h_out = static_cast<uint16_t *>(p.h_out);
    a.epilogue = p.epilogue;
    const int64_t tiles_m = (p.M + BM - 1) / BM;
    const int64_t tiles_n = p.Nout / BN;
    if (tiles_m * tiles_n >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    a.tiles_n = (int)tiles_n;
    a.tiles_total = (int)(tiles_m * tiles_n);
    gemm_split_ws(p, gemm_splits(p, a.tiles_total, 1), s, a);
    dyad_gemm_mfma2<BM, BN, WGM, WGN, D, IN_T, OUT_T, W_T><<<a.tiles_total * a.splits, C::kThreads, 0, s>>>(a);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && a.part) e = launch_split_reduce(p, a.part, a.splits, s);
    return e;
}

// One component of a pass alone (fused-stage kernel, ONLY = 1 or 2) into
// slice `slice` of the fp32 partial sums `part`; with ONLY = 3, component 1
// into the pass's output with its epilogue, adding that slice (at the
// block-order place of each column with `unperm`).
template <int BM, int BN, int WGM, int WGN, int D, bool IN_T, bool OUT_T, bool W_T, int ONLY>
hipError_t launch_component(const GemmPass &p, float *part, int slice, bool unperm, hipStream_t s, int splits = 1) {
    using C = Gemm2Cfg<BM, BN, WGM, WGN, D, IN_T, OUT_T, W_T>;
    GemmArgs a{};
    if ((int64_t)BM * p.Kin * 2 >= ((int64_t)1 << 31) || (int64_t)BM * p.Nout * 4 >= ((int64_t)1 << 31) ||
        2 * p.D * p.bn * p.bk >= ((int64_t)1 << 31))
        return hipErrorNotSupported;
    a.M = p.M; a.Kin = p.Kin; a.Nout = p.Nout; a.bk = p.bk; a.bn = p.bn; a.D = p.D;
    a.in = static_cast<const uint16_t *>(p.in);
    a.W1 = static_cast<const uint16_t *>(p.W1);
    a.W2 = static_cast<const uint16_t *>(p.W2);
    a.bias = nullptr; a.h_in = nullptr; a.out = nullptr; a.h_out = nullptr;
    a.epilogue = kEpiBias;
    if constexpr (ONLY == 3) {
        a.bias = static_cast<const uint16_t *>(p.bias);
        a.h_in = static_cast<const uint16_t *>(p.h_in);
        a.out = static_cast<uint16_t *>(p.out);
        a.h_out = static_cast<uint16_t *>(p.h_out);
        a.epilogue = p.epilogue;
    }
    const int64_t tiles_m = (p.M + BM - 1) / BM;
    const int64_t tiles_n = p.Nout / BN;
    if (tiles_m * tiles_n >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    a.tiles_n = (int)tiles_n;
    a.tiles_total = (int)(tiles_m * tiles_n);
    // split s of the reduction (ONLY = 1 or 2) writes slice `slice` + s
    if (splits < 1 || (p.bk / kStageK) % splits != 0 || (splits > 1 && ONLY > 2)) return hipErrorNotSupported;
    a.part = part; a.splits = splits; a.slice0 = slice; a.unperm = unperm;
    // a few token panels over many weight tiles: the panels of one weight tile
    // run next to each other (on one XCD), which then reads those weights once
    a.n_major = tiles_m <= 8 && tiles_n >= 64;
    dyad_gemm_mfma2<BM, BN, WGM, WGN, D, IN_T, OUT_T, W_T, ONLY><<<a.tiles_total * splits, C::kThreads, 0, s>>>(a);
    return hipGetLastError();
}

// Whether a fused-stage tile fits (LDS of Gemm2Cfg, without instantiating it).
template <int BM, int BN, int WGM, int WGN, int D, bool IN_T, bool OUT_T, bool W_T>
constexpr bool tile2_ok() {
    const int res = OUT_T ? D : 1, cpr = BN / res, wn = BN / WGN;
    if (OUT_T && (BN % D != 0 || cpr % 16 != 0)) return false;
    if (wn % cpr != 0 && cpr % wn != 0) return false;
    if ((BM * 4) % 64 != 0) return false;
    const int slab = BM * kStageK * 2;
    const int bbytes = W_T ? kStageK * (BN * 2 + 16) : BN * kStageK * 2;
    const int operands = 2 * (slab * (1 + res) + 2 * bbytes);
    const int epi = 2 * (WGM * 16) * (BN + 4) * 4;
    return (operands > epi ? operands : epi) <= 160 * 1024;
}

// Tile choice.  Every tile stays inside one output block; with an output
// transpose every residue must get a multiple of 16 columns.  A BlockTrans
// stage with an output transpose stages one A slab per residue, so the token
// tile shrinks as n_dyad grows to keep both stage buffers in LDS.
//
// Large batches (at least one 8-wave workgroup per CU) first try 8-wave tiles,
// chosen by what the epilogue costs (measured on gfx950 at OPT-125m feed-forward
// shapes, n_dyad 4): with a plain or bias epilogue 256 x 192 (4 x 2 waves of
// 64 x 96); with GELU' (input gradient) 128 x 384 (2 x 4 waves of 64 x 96);
// with GELU after an output transpose 256 x 256 (2 x 4 waves of 128 x 64).
// The input gradient without an output transpose takes the fused-stage kernel
// (gemm_mfma2.h) instead.  Otherwise 4-wave tiles, two workgroups per CU.
// LDS bytes of a tile (as GemmCfg lays it out), without instantiating it
constexpr int gemm_lds(int BM, int BN, int WGM, int D, bool OUT_T) {
    const int operands = 2 * ((OUT_T ? D : 1) * BM * kStageK + BN * kStageK) * 2;
    const int epi = 2 * (WGM * 16) * (BN + 4) * 4;
    return operands > epi ? operands : epi;
}

// Under an output transpose every 16-column MFMA block holds one residue:
// BN splits into D residues of a multiple of 16 columns each.
constexpr bool out_cols_ok(int BN, int D) { return BN % D == 0 && (BN / D) % 16 == 0; }

// ... and each wave's columns hold whole residues or a part of one.
constexpr bool wave_cols_ok(int BN, int WGN, int D) {
    const int wn = BN / WGN, cpr = BN / D;
    return wn % cpr == 0 || cpr % wn == 0;
}

template <int BM, int BN, int WGM, int WGN, int D, bool OUT_T>
constexpr bool tile_ok() {
    return (!OUT_T || (out_cols_ok(BN, D) && wave_cols_ok(BN, WGN, D))) &&
           gemm_lds(BM, BN, WGM, D, OUT_T) <= 160 * 1024;
}

// The two components apart, for blocks too narrow for a tile (n_dyad 8 / 16
// with blocks of 64 or 128 columns).  Component 1 is a plain per-block GEMM on
// 64-column tiles.  Component 2 runs on the tiles of an output transpose,
// 256 columns j*D + g at a time across blocks, which use every residue of an
// input span; without an output transpose its sums are stored back at column
// g*bn + j.  Both write fp32 slices that the split reduction adds in order.
template <int D, bool IN_T, bool OUT_T, bool W_T>
hipError_t launch_components(const GemmPass &p, hipStream_t s) {
    if constexpr (D < 8) {
        return hipErrorNotSupported;
    } else {
        constexpr bool k64 = tile2_ok<64, 256, 2, 4, D, IN_T, true, W_T>();
        constexpr bool k32 = tile2_ok<32, 256, 1, 8, D, IN_T, true, W_T>();
        if constexpr (!k64 && !k32) {
            return hipErrorNotSupported;
        } else {
            if (p.bn % 64 != 0 || p.Nout % 256 != 0) return hipErrorNotSupported;
            // the two fp32 slices stay with the stream: at most 2 GiB of them
            const size_t bytes = 2 * (size_t)p.M * (size_t)p.Nout * sizeof(float);
            if (bytes > ((size_t)2 << 30)) return hipErrorNotSupported;
            void *ws = nullptr;
            if (split_workspace(s, bytes, &ws) != hipSuccess) {
                (void)hipGetLastError();
                return hipErrorNotSupported;
            }
            float *part = static_cast<float *>(ws);
            hipError_t e = launch_component<128, 64, 2, 2, D, IN_T, false, W_T, 1>(p, part, 0, false, s);
            if (e == hipSuccess) {
                if constexpr (k64) e = launch_component<64, 256, 2, 4, D, IN_T, true, W_T, 2>(p, part, 1, !OUT_T, s);
                else e = launch_component<32, 256, 1, 8, D, IN_T, true, W_T, 2>(p, part, 1, !OUT_T, s);
            }
            if (e == hipSuccess) e = launch_split_reduce(p, part, 2, s);
            return e;
        }
    }
}

// Large batches at n_dyad 8 and 16 with a transpose.  A fused tile under an
// output transpose holds every residue of its output columns and so reads the
// input panel D times over per column span; under an input transpose it reads
// whole spans of D residues for one.  Either way the operand traffic per tile
// outgrows the pass's HBM traffic at these widths.  Here the permutations
// leave the GEMM: an input transpose first de-interleaves the input once
// (residue g's columns k*D + g become the contiguous block g), both components
// then run as plain per-block GEMMs: component 2 (W2 on that block-ordered
// input) into an fp32 slice, then component 1 with the pass's epilogue, which
// adds the slice, read at the block-order place of each output column
// (column g*bn + j for output column j*D + g) under an output transpose.  The
// tokens run in chunks that keep the workspace (slice and de-interleaved
// input) within 2 GiB.
//
// A batch whose tiles give each CU at most one workgroup, over a reduction of
// at least 1024 (256 tokens of the wide layer: 256 tiles of 64 x 128 over
// 2048) splits the reduction of both components into S parts, each its own
// fp32 slice, so that every CU runs several workgroups with a shorter loop;
// the split reduction then adds component 1's slices and component 2's (read
// at the block-order place under an output transpose) in order and applies
// the epilogue.  Measured there: fc1 input gradient 93 -> 80 µs, fc2
// forward 87 -> 81 µs; over reductions of 512 (fc1 forward, fc2 input
// gradient, whose outputs are 4x wider) the slices cost more than the split
// saves (65 -> 104 µs).
template <int BM, int BN, int WGM, int WGN, int D, bool W_T>
hipError_t launch_permuted_as(const GemmPass &p, bool in_t, bool out_t, hipStream_t s) {
    const int64_t tiles = ((p.M + BM - 1) / BM) * (p.Nout / BN);
    int S = 1;
    while (tiles * S < 512 && S < 4 && (p.bk / kStageK) % (2 * S) == 0 && p.bk / kStageK / (2 * S) >= 16) S *= 2;
    const size_t per_tok = (in_t ? (size_t)p.Kin * 2 : 0) + (size_t)(S > 1 ? 2 * S : 1) * p.Nout * sizeof(float);
    const size_t cap = (size_t)2 << 30;
    int64_t mc = (int64_t)(cap / per_tok);
    if (mc >= p.M) mc = p.M;
    else mc -= mc % 256;
    if (mc < 1 || (mc < 256 && mc < p.M)) return hipErrorNotSupported;
    void *ws = nullptr;
    if (split_workspace(s, per_tok * (size_t)mc, &ws) != hipSuccess) {
        (void)hipGetLastError();
        return hipErrorNotSupported;
    }
    float *part = static_cast<float *>(ws);
    uint16_t *xp = reinterpret_cast<uint16_t *>(part + (S > 1 ? 2 * S : 1) * mc * p.Nout);
    hipError_t e = hipSuccess;
    for (int64_t m0 = 0; m0 < p.M && e == hipSuccess; m0 += mc) {
        GemmPass c = p;
        c.M = p.M - m0 < mc ? p.M - m0 : mc;
        c.in = static_cast<const uint16_t *>(p.in) + m0 * p.Kin;
        c.out = static_cast<uint16_t *>(p.out) + m0 * p.Nout;
        if (p.h_in) c.h_in = static_cast<const uint16_t *>(p.h_in) + m0 * p.Nout;
        if (p.h_out) c.h_out = static_cast<uint16_t *>(p.h_out) + m0 * p.Nout;
        GemmPass c2 = c;
        c2.W1 = p.W2;
        if (in_t) {
            e = launch_deinterleave(static_cast<const uint16_t *>(c.in), xp, c.M, p.bk, D, s);
            c2.in = xp;
        }
        if (S > 1) {
            // slices 0 .. S-1: component 1, S .. 2S-1: component 2 (block order)
            if (e == hipSuccess) e = launch_component<BM, BN, WGM, WGN, D, false, false, W_T, 1>(c, part, 0, false, s, S);
            if (e == hipSuccess) e = launch_component<BM, BN, WGM, WGN, D, false, false, W_T, 1>(c2, part, S, false, s, S);
            if (e == hipSuccess) e = launch_split_reduce(c, part, 2 * S, s, false, out_t ? S : 2 * S);
            continue;
        }
        if (e == hipSuccess) e = launch_component<BM, BN, WGM, WGN, D, false, false, W_T, 1>(c2, part, 0, false, s);
        if (e == hipSuccess) e = launch_component<BM, BN, WGM, WGN, D, false, false, W_T, 3>(c, part, 0, out_t, s);
    }
    return e;
}

// n_dyad 3 and 6 under an output transpose: with power-of-two blocks no
// tile of whole residues (a multiple of 16 columns of each of the D) lies
// within one block, so the components run apart on the de-interleaved form.
template <int D>
constexpr bool odd_residues() { return D == 3 || D == 6; }

template <int D, bool IN_T, bool OUT_T, bool W_T>
hipError_t launch_permuted(const GemmPass &p, hipStream_t s) {
    if constexpr ((D < 8 && !odd_residues<D>()) || (D >= 8 && 64 % D != 0) || (!IN_T && !OUT_T)) {
        return hipErrorNotSupported;
    } else {
        if (p.bk % kStageK != 0 || p.Nout % 8 != 0) return hipErrorNotSupported;
        // up to 1024 tokens, 128-token tiles: twice the workgroups, the weights
        // read twice; 128 x 128 where 128 x 256 would not give every CU a tile
        // (1.2x at 256 and 512 tokens, wide layer fc2 forward / fc1 input
        // gradient), and up to 512 tokens 64 x 128 where 128 x 128 would not
        // (another 1.1-1.2x at 256 tokens)
        const int64_t tm = (p.M + 127) / 128;
        if (p.bn % 128 == 0 && p.M <= 512 && tm * (p.Nout / 128) < 256)
            return launch_permuted_as<64, 128, 2, 2, D, W_T>(p, IN_T, OUT_T, s);
        if (p.bn % 128 == 0 && p.M <= 1024 && tm * (p.Nout / 256) < 256)
            return launch_permuted_as<128, 128, 2, 2, D, W_T>(p, IN_T, OUT_T, s);
        if (p.bn % 256 == 0 && p.M <= 1024) return launch_permuted_as<128, 256, 2, 4, D, W_T>(p, IN_T, OUT_T, s);
        if (p.bn % 256 == 0) return launch_permuted_as<256, 256, 2, 4, D, W_T>(p, IN_T, OUT_T, s);
        if (p.bn % 128 == 0) return launch_permuted_as<128, 128, 2, 2, D, W_T>(p, IN_T, OUT_T, s);
        if (p.bn % 64 == 0) return launch_permuted_as<128, 64, 2, 2, D, W_T>(p, IN_T, OUT_T, s);
        return hipErrorNotSupported;
    }
}

template <int D, bool IN_T, bool OUT_T, bool W_T>
hipError_t dispatch_tiles(const GemmPass &p, hipStream_t s) {
    if (p.bk % kStageK != 0) return hipErrorNotSupported;
    auto enough = [&](int bm, int bn_tile) { return ((p.M + bm - 1) / bm) * (p.Nout / bn_tile) >= 256; };
    if constexpr (D >= 8)
        if (permuted_pays((int)D, OUT_T, W_T, p.M, p.bk)) {
            const hipError_t e = launch_permuted<D, IN_T, OUT_T, W_T>(p, s);
            if (e != hipErrorNotSupported) return e;
        }
    if constexpr (odd_residues<D>() && OUT_T) return launch_permuted<D, IN_T, OUT_T, W_T>(p, s);
    if constexpr (D <= 4) {
        // the fused-stage kernel (natural-layout weights, transpose reads) wins
        // for the input gradient without an output transpose
        if constexpr (W_T && !OUT_T) {
            if (p.epilogue == kEpiGeluGrad) {
                if constexpr (tile2_ok<128, 384, 2, 4, D, IN_T, OUT_T, W_T>())
                    if (p.bn % 384 == 0 && enough(128, 384))
                        return launch_tile2<128, 384, 2, 4, D, IN_T, OUT_T, W_T>(p, s);
            } else {
                if constexpr (tile2_ok<256, 192, 4, 2, D, IN_T, OUT_T, W_T>())
                    if (p.bn % 192 == 0 && enough(256, 192))
                        return launch_tile2<256, 192, 4, 2, D, IN_T, OUT_T, W_T>(p, s);
            }
        }
        if (p.epilogue == kEpiBias) {
            // the forward pass keeps two stages of loads in flight when the
            // group is at least two stages deep (measured 3-8% faster at
            // OPT-125m fc2; the input gradient's transposed weights spill)
            if constexpr (tile_ok<256, 192, 4, 2, D, OUT_T>())
                if (p.bn % 192 == 0 && enough(256, 192)) {
                    if constexpr (!W_T)
                        if (p.bk >= 2 * kStageK) return launch_tile<256, 192, 4, 2, D, IN_T, OUT_T, W_T, 2>(p, s);
                    return launch_tile<256, 192, 4, 2, D, IN_T, OUT_T, W_T>(p, s);
                }
        } else if (p.epilogue == kEpiGeluGrad) {
            if constexpr (tile_ok<128, 384, 2, 4, D, OUT_T>())
                if (p.bn % 384 == 0 && enough(128, 384)) return launch_tile<128, 384, 2, 4, D, IN_T, OUT_T, W_T>(p, s);
            if constexpr (tile_ok<256, 192, 4, 2, D, OUT_T>())
                if (p.bn % 192 == 0 && enough(256, 192)) return launch_tile<256, 192, 4, 2, D, IN_T, OUT_T, W_T>(p, s);
        } else if constexpr (OUT_T && !W_T) {
            if constexpr (tile_ok<256, 256, 2, 4, D, OUT_T>())
                if (p.bn % 256 == 0 && enough(256, 256)) return launch_tile<256, 256, 2, 4, D, IN_T, OUT_T, W_T>(p, s);
        }
    }
    // Blocks of a multiple of 256 columns (OPT-350m, wider layers), from a tile
    // sweep at d = 1024 (n_dyad 4) and d = 2048 (n_dyad 8)
    if constexpr (D <= 8) {
        if (p.bn % 256 == 0) {
            if constexpr (W_T && (D <= 4 || !OUT_T)) {
                if constexpr (tile2_ok<128, 256, 2, 4, D, IN_T, OUT_T, W_T>())
                    if (enough(128, 256)) return launch_tile2<128, 256, 2, 4, D, IN_T, OUT_T, W_T>(p, s);
            } else if constexpr (D == 8 && OUT_T) {
                if constexpr (tile_ok<128, 256, 2, 4, D, OUT_T>())
                    if (enough(128, 256)) return launch_tile<128, 256, 2, 4, D, IN_T, OUT_T, W_T>(p, s);
            } else if constexpr (D == 8) {
                if constexpr (tile_ok<256, 256, 2, 4, D, OUT_T>())
                    if (enough(256, 256)) return launch_tile<256, 256, 2, 4, D, IN_T, OUT_T, W_T>(p, s);
            } else if (p.epilogue == kEpiBias) {
                if constexpr (OUT_T) {
                    if constexpr (tile_ok<256, 256, 2, 4, D, OUT_T>())
                        if (enough(256, 256)) return launch_tile<256, 256, 2, 4, D, IN_T, OUT_T, W_T>(p, s);
                } else {
                    if constexpr (tile_ok<256, 256, 4, 2, D, OUT_T>())
                        if (enough(256, 256)) return launch_tile<256, 256, 4, 2, D, IN_T, OUT_T, W_T>(p, s);
                }
            }
        }
    }
    // n_dyad 8 and 16 with an output transpose: a 256-column tile gives every
    // residue 16 or 32 columns; the D input slabs keep the token tile short
    if constexpr (D >= 8 && OUT_T) {
        if constexpr (tile2_ok<64, 256, 2, 4, D, IN_T, OUT_T, W_T>())
            if (p.bn % 256 == 0) return launch_tile2<64, 256, 2, 4, D, IN_T, OUT_T, W_T>(p, s);
        if constexpr (tile2_ok<32, 256, 1, 8, D, IN_T, OUT_T, W_T>())
            if (p.bn % 256 == 0) return launch_tile2<32, 256, 1, 8, D, IN_T, OUT_T, W_T>(p, s);
    }
    // An input transpose with narrow blocks: a tile inside one block would use
    // one residue of every span it loads
    if constexpr (IN_T && !OUT_T && D >= 8)
        if (p.bn < 256) {
            const hipError_t e = launch_components<D, IN_T, OUT_T, W_T>(p, s);
            if (e != hipErrorNotSupported) return e;
        }
    constexpr int BM = D >= 8 ? 64 : 128;
    // with an output transpose a 128 x 256 tile's D slabs need one workgroup per
    // CU; 64 x 256 keeps two, which measures faster
    constexpr int BM256 = OUT_T ? 64 : BM;
    if constexpr (D < 16 && tile_ok<BM256, 256, 2, 2, D, OUT_T>())
        if (p.bn % 256 == 0) return launch_tile<BM256, 256, 2, 2, D, IN_T, OUT_T, W_T>(p, s);
    if constexpr (tile_ok<BM, 192, 2, 2, D, OUT_T>())
        if (p.bn % 192 == 0) return launch_tile<BM, 192, 2, 2, D, IN_T, OUT_T, W_T>(p, s);
    if constexpr (tile_ok<BM, 128, 2, 2, D, OUT_T>())
        if (p.bn % 128 == 0) return launch_tile<BM, 128, 2, 2, D, IN_T, OUT_T, W_T>(p, s);
    if constexpr (tile_ok<BM, 64, 2, 2, D, OUT_T>())
        if (p.bn % 64 == 0) return launch_tile<BM, 64, 2, 2, D, IN_T, OUT_T, W_T>(p, s);
    // An output transpose whose blocks are too narrow for any tile above
    // (n_dyad 16 with blocks of 64 or 128 columns): the components run apart.
    if constexpr (OUT_T) return launch_components<D, IN_T, OUT_T, W_T>(p, s);
    return hipErrorNotSupported;
}

// Forward of a layer whose input is GELU(in) (GemmPass::gelu_in): the phased
// tiles, with the activation applied to the input operand as it is staged.
// Tiles as for the plain forward pass (8-wave 256 x 192 / 256 x 256 where the
// batch fills the GPU, else 4-wave tiles with split reductions), one stage of
// loads ahead.  An output transpose at n_dyad 8 / 16 has no such tile.
template <int D, bool IN_T, bool OUT_T>
hipError_t dispatch_gelu_in(const GemmPass &p, hipStream_t s) {
    if constexpr (OUT_T && D > 4) {
        return hipErrorNotSupported;
    } else {
        if (p.bk % kStageK != 0) return hipErrorNotSupported;
        auto enough = [&](int bm, int bn_tile) { return ((p.M + bm - 1) / bm) * (p.Nout / bn_tile) >= 256; };
        if constexpr (tile_ok<256, 192, 4, 2, D, OUT_T>())
            if (p.bn % 192 == 0 && enough(256, 192))
                return launch_tile<256, 192, 4, 2, D, IN_T, OUT_T, false, 1, true>(p, s);
        if constexpr (tile_ok<256, 256, 2, 4, D, OUT_T>())
            if (p.bn % 256 == 0 && enough(256, 256))
                return launch_tile<256, 256, 2, 4, D, IN_T, OUT_T, false, 1, true>(p, s);
        constexpr int BM = D >= 8 ? 64 : 128;
        constexpr int BM256 = OUT_T ? 64 : BM;
        if constexpr (D < 16 && tile_ok<BM256, 256, 2, 2, D, OUT_T>())
            if (p.bn % 256 == 0) return launch_tile<BM256, 256, 2, 2, D, IN_T, OUT_T, false, 1, true>(p, s);
        if constexpr (tile_ok<BM, 192, 2, 2, D, OUT_T>())
            if (p.bn % 192 == 0) return launch_tile<BM, 192, 2, 2, D, IN_T, OUT_T, false, 1, true>(p, s);
        if constexpr (tile_ok<BM, 128, 2, 2, D, OUT_T>())
            if (p.bn % 128 == 0) return launch_tile<BM, 128, 2, 2, D, IN_T, OUT_T, false, 1, true>(p, s);
        if constexpr (tile_ok<BM, 64, 2, 2, D, OUT_T>())
            if (p.bn % 64 == 0) return launch_tile<BM, 64, 2, 2, D, IN_T, OUT_T, false, 1, true>(p, s);
        return hipErrorNotSupported;
    }
}

template <bool IN_T, bool OUT_T>
hipError_t dispatch_d_gelu_in(const GemmPass &p, hipStream_t s) {
    switch (p.D) {
    case 1: return dispatch_gelu_in<1, IN_T, OUT_T>(p, s);
    case 2: return dispatch_gelu_in<2, IN_T, OUT_T>(p, s);
    case 4: return dispatch_gelu_in<4, IN_T, OUT_T>(p, s);
    case 8: return dispatch_gelu_in<8, IN_T, OUT_T>(p, s);
    case 16: return dispatch_gelu_in<16, IN_T, OUT_T>(p, s);
    default: return hipErrorNotSupported;
    }
}

template <bool IN_T, bool OUT_T, bool W_T>
hipError_t dispatch_d(const GemmPass &p, hipStream_t s) {
    switch (p.D) {
    case 1: return dispatch_tiles<1, IN_T, OUT_T, W_T>(p, s);
    case 2: return dispatch_tiles<2, IN_T, OUT_T, W_T>(p, s);
    case 3: return dispatch_tiles<3, IN_T, OUT_T, W_T>(p, s);
    case 4: return dispatch_tiles<4, IN_T, OUT_T, W_T>(p, s);
    case 6: return dispatch_tiles<6, IN_T, OUT_T, W_T>(p, s);
    case 8: return dispatch_tiles<8, IN_T, OUT_T, W_T>(p, s);
    case 16: return dispatch_tiles<16, IN_T, OUT_T, W_T>(p, s);
    default: return hipErrorNotSupported;
    }
}

// One per (pass, variant); each lives in its own translation unit.
hipError_t launch_mfma_fwd_it(const GemmPass &p, hipStream_t s);
hipError_t launch_mfma_fwd_ot(const GemmPass &p, hipStream_t s);
hipError_t launch_mfma_fwd_dt(const GemmPass &p, hipStream_t s);
hipError_t launch_mfma_dx_it(const GemmPass &p, hipStream_t s);
hipError_t launch_mfma_dx_ot(const GemmPass &p, hipStream_t s);
hipError_t launch_mfma_dx_dt(const GemmPass &p, hipStream_t s);
hipError_t launch_mfma_fwd_gin_it(const GemmPass &p, hipStream_t s);
hipError_t launch_mfma_fwd_gin_ot(const GemmPass &p, hipStream_t s);
hipError_t launch_mfma_fwd_gin_dt(const GemmPass &p, hipStream_t s);

}  // namespace dyad
