// Zero-padded forms of the grouped GEMM: for passes whose widths n_dyad does
// not divide, or whose blocks fit no tile (blocks of 154 or 615 columns at
// n_dyad 5, say), or whose n_dyad has no fused tile.  The zero-padded layer
// is the Dyad layer on widths D*bk x D*bn restricted to the real ones
// (block sizes rounded up, the rest zero), so its blocks can be padded
// further to whole tiles: the input becomes block-ordered copies with blocks
// of bkp = bk rounded up to 32 columns (component 1: block g of the input;
// component 2: residue g under an input transpose, else block g again), the
// weights copies of bnp x bkp blocks (bnp = bn rounded up to 64), zero in the
// padding, and the matrix cores run plain per-block tiles over them.
// Without an output transpose both components share each output column
// (K-concatenated, one pass); under one, component 2 first goes to an fp32
// slice that component 1's epilogue adds at the block-order place of each
// real column.  The epilogue writes real columns only (gemm_epilogue_pad).
#pragma once

#include "gemm_mfma2.h"

namespace dyad {

template <int BM, int BN, int WGM, int WGN, bool W_T, int ONLY>
hipError_t launch_pad_tile(const GemmArgs &a0, hipStream_t s) {
    using C = Gemm2Cfg<BM, BN, WGM, WGN, 1, false, false, W_T>;
    GemmArgs a = a0;
    const int64_t tiles_m = (a.M + BM - 1) / BM;
    const int64_t tiles_n = a.Nout / BN;
    if (a.Nout % BN != 0 || tiles_m * tiles_n >= ((int64_t)1 << 31)) return hipErrorNotSupported;
    a.tiles_n = (int)tiles_n;
    a.tiles_total = (int)(tiles_m * tiles_n);
    a.splits = 1;
    dyad_gemm_mfma2<BM, BN, WGM, WGN, 1, false, false, W_T, ONLY><<<a.tiles_total, C::kThreads, 0, s>>>(a);
    return hipGetLastError();
}

// The tiles of one padded form: ONLY = 1 (component 2 into the slice), 4
// (component 1 adding it) or 5 (both components).  Output blocks of a
// multiple of 256, 192, 128 or 64 columns, 8-wave tiles where they fill the GPU.
template <bool W_T, int ONLY>
hipError_t launch_pad_form(const GemmArgs &a, hipStream_t s) {
    const int64_t bnp = a.bn;
    auto enough = [&](int bm, int bn_tile) { return ((a.M + bm - 1) / bm) * (a.Nout / bn_tile) >= 256; };
    if (bnp % 256 == 0 && enough(256, 256)) return launch_pad_tile<256, 256, 2, 4, W_T, ONLY>(a, s);
    if (bnp % 192 == 0 && enough(256, 192)) return launch_pad_tile<256, 192, 4, 2, W_T, ONLY>(a, s);
    if (bnp % 128 == 0) return launch_pad_tile<128, 128, 2, 2, W_T, ONLY>(a, s);
    return launch_pad_tile<128, 64, 2, 2, W_T, ONLY>(a, s);
}

// Whole pass on the padded forms (GemmPass p: real widths and blocks).
// Token chunks keep the workspace (input copies and slice) within 2 GiB.
template <bool W_T>
hipError_t launch_padded_as(const GemmPass &p, hipStream_t s) {
    const int64_t D = p.D, bk = p.bk, bn = p.bn;
    const int64_t bkp = pad_up(bk, kStageK), bnp = pad_up(bn, 64);
    const int64_t Kp = D * bkp, Np = D * bnp;
    // 32-bit offsets: one tile's rows of the copies, slice and output
    if ((int64_t)256 * Np * 4 >= ((int64_t)1 << 31) || (int64_t)256 * Kp * 2 >= ((int64_t)1 << 31) ||
        D * bnp * bkp * 2 >= ((int64_t)1 << 31))
        return hipErrorNotSupported;
    const size_t wbytes = (size_t)(D * bnp * bkp * 2 + 255) / 256 * 256;
    const size_t per_tok = (size_t)Kp * 2 * (p.in_t ? 2 : 1) + (p.out_t ? (size_t)Np * 4 : 0);
    const size_t cap = (size_t)2 << 30;
    int64_t mc = (int64_t)((cap - 2 * wbytes) / per_tok);
    if (mc >= p.M) mc = p.M;
    else mc -= mc % 256;
    if (mc < 256 && mc < p.M) return hipErrorNotSupported;
    void *ws = nullptr;
    if (split_workspace(s, 2 * wbytes + per_tok * (size_t)mc + 256, &ws) != hipSuccess) {
        (void)hipGetLastError();
        return hipErrorNotSupported;
    }
    unsigned char *base = static_cast<unsigned char *>(ws);
    uint16_t *w1p = reinterpret_cast<uint16_t *>(base);
    uint16_t *w2p = reinterpret_cast<uint16_t *>(base + wbytes);
    uint16_t *x1 = reinterpret_cast<uint16_t *>(base + 2 * wbytes);
    uint16_t *x2 = p.in_t ? x1 + mc * Kp : x1;
    float *slice = reinterpret_cast<float *>(reinterpret_cast<unsigned char *>(x1) +
                                             (size_t)mc * Kp * 2 * (p.in_t ? 2 : 1));
    // weights as stored: [D][bn][bk], or [D][bk][bn] when read transposed
    const int64_t R = W_T ? bk : bn, Cc = W_T ? bn : bk, Rp = W_T ? bkp : bnp, Cp = W_T ? bnp : bkp;
    hipError_t e = launch_pad_matrix(static_cast<const uint16_t *>(p.W1), D, R, Cc, Rp, Cp, w1p, s);
    if (e == hipSuccess) e = launch_pad_matrix(static_cast<const uint16_t *>(p.W2), D, R, Cc, Rp, Cp, w2p, s);
    for (int64_t m0 = 0; m0 < p.M && e == hipSuccess; m0 += mc) {
        const int64_t mt = p.M - m0 < mc ? p.M - m0 : mc;
        e = launch_pad_rows(static_cast<const uint16_t *>(p.in) + m0 * p.Kin, mt, p.Kin, (int)D, bk, bkp, x1,
                            p.in_t ? x2 : nullptr, s);
        if (e != hipSuccess) break;
        GemmArgs a{};
        a.M = mt; a.Kin = Kp; a.Nout = Np; a.bk = bkp; a.bn = bnp; a.D = D;
        a.in = x1; a.in2 = x2; a.W1 = w1p; a.W2 = w2p;
        a.bias = static_cast<const uint16_t *>(p.bias);
        a.h_in = p.h_in ? static_cast<const uint16_t *>(p.h_in) + m0 * p.Nout : nullptr;
        a.out = static_cast<uint16_t *>(p.out) + m0 * p.Nout;
        a.h_out = p.h_out ? static_cast<uint16_t *>(p.h_out) + m0 * p.Nout : nullptr;
        a.epilogue = p.epilogue;
        a.Nout_r = p.Nout; a.bn_r = bn;
        a.slice0 = 0;
        if (p.out_t) {
            // component 2 (weights w2p on its input copy) into the slice, then
            // component 1 adding it at the block-order place of each real column
            GemmArgs c2 = a;
            c2.in = x2; c2.W1 = w2p; c2.part = slice; c2.unperm = 0;
            c2.bias = nullptr; c2.h_in = nullptr; c2.out = nullptr; c2.h_out = nullptr; c2.epilogue = kEpiBias;
            e = launch_pad_form<W_T, 1>(c2, s);
            a.part = slice; a.unperm = 1;
            if (e == hipSuccess) e = launch_pad_form<W_T, 4>(a, s);
        } else {
            a.part = nullptr; a.unperm = 0;
            e = launch_pad_form<W_T, 5>(a, s);
        }
    }
    return e;
}

}  // namespace dyad
