// Host-side tile choice and launch for the MFMA grouped GEMM (gemm_mfma.h).
#pragma once

#include "gemm_mfma.h"

namespace dyad {

template <int BM, int BN, int WM, int WN, int D, bool IN_T, bool OUT_T, bool W_T>
hipError_t launch_tile(const GemmPass &p, hipStream_t s) {
    GemmArgs a;
    a.M = p.M; a.Kin = p.Kin; a.Nout = p.Nout; a.bk = p.bk; a.bn = p.bn;
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
    dyad_gemm_mfma<BM, BN, WM, WN, D, IN_T, OUT_T, W_T><<<a.tiles_total, kThreads, 0, s>>>(a);
    return hipGetLastError();
}

// Picks the widest tile whose columns stay inside one output block and, with
// an output transpose, give every residue a multiple of 16 columns.
template <int D, bool IN_T, bool OUT_T, bool W_T>
hipError_t dispatch_tiles(const GemmPass &p, hipStream_t s) {
    if (p.bk % kStageK != 0) return hipErrorNotSupported;
    if constexpr (D <= 8) {
        if constexpr (!OUT_T || (128 / D) % 16 == 0)
            if (p.bn % 128 == 0) return launch_tile<128, 128, 64, 64, D, IN_T, OUT_T, W_T>(p, s);
        if constexpr (!OUT_T || (192 / D) % 16 == 0)
            if (p.bn % 192 == 0) return launch_tile<128, 192, 64, 96, D, IN_T, OUT_T, W_T>(p, s);
        if constexpr (!OUT_T || (64 / D) % 16 == 0)
            if (p.bn % 64 == 0) return launch_tile<128, 64, 64, 32, D, IN_T, OUT_T, W_T>(p, s);
    } else {
        if (p.bn % 256 == 0) return launch_tile<64, 256, 64, 64, D, IN_T, OUT_T, W_T>(p, s);
        if constexpr (!OUT_T)
            if (p.bn % 128 == 0) return launch_tile<64, 128, 32, 64, D, IN_T, OUT_T, W_T>(p, s);
    }
    return hipErrorNotSupported;
}

template <bool IN_T, bool OUT_T, bool W_T>
hipError_t dispatch_d(const GemmPass &p, hipStream_t s) {
    switch (p.D) {
    case 1: return dispatch_tiles<1, IN_T, OUT_T, W_T>(p, s);
    case 2: return dispatch_tiles<2, IN_T, OUT_T, W_T>(p, s);
    case 4: return dispatch_tiles<4, IN_T, OUT_T, W_T>(p, s);
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

}  // namespace dyad
