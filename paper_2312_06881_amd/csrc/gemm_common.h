// Pieces shared by the grouped-GEMM kernels: launch arguments and the
// epilogue (accumulators -> bias / GELU / GELU' -> bf16 output).
#pragma once

#include <type_traits>

#include "dyad_internal.h"
#include "mfma_common.h"

namespace dyad {

struct GemmArgs {
    int64_t M, Kin, Nout, bk, bn, D;
    const uint16_t *in, *W1, *W2, *bias, *h_in;
    uint16_t *out, *h_out;
    int epilogue;
    int tiles_n;        // output tiles per token panel
    int tiles_total;
    float *part;        // split reduction: fp32 partial sums [slices][M][Nout], else null
    int splits;         // workgroups along the reduction per tile
    int slice0;         // partial slice of split 0
    int unperm;         // partial sums of column j*D + g belong to column g*bn + j
    // zero-padded forms (gemm_epilogue_pad): component 2's block-ordered input,
    // and the real output width and block size (Nout and bn are the padded ones)
    const uint16_t *in2;
    int64_t Nout_r, bn_r;
    // tile order (fused-stage kernel): 0 token panels outer, so a workgroup's
    // neighbours on its XCD share its input rows; 1 output columns outer, so
    // they share its weights (few token panels, large weights)
    int n_major;
};

// Epilogue of a BM x BN tile whose accumulators sit in the MFMA layout (wave w
// owns rows (w / WGN) * WM + 16 i + 4 (lane / 16) + v and internal columns
// wn0 + 16 j + lane % 16).  C supplies kThreads, kWGN, WM, kSubM, kSubN,
// kEpiRows, kEpiPitch, kEpiElems and kCPR (internal columns per residue with an
// output transpose).  smem needs 2 * kEpiElems floats and must be free.  With
// a split reduction (a.part set) the tile's fp32 sums go to slice `split` of
// the partial sums instead, in real column order and without the epilogue.
// ADD: before the epilogue each sum gets the fp32 value of slice a.slice0 of
// a.part at its column, or with a.unperm at the block-order place of it
// (column g*bn + j for column j*D + g).
template <class C, int BM, int BN, int D, bool OUT_T, bool PARTIAL, bool ADD = false>
__device__ __forceinline__ void gemm_epilogue_as(const GemmArgs &a, unsigned char *smem,
                                                 const f32x4_t (&acc)[C::kSubM][C::kSubN], int64_t m0, int n0,
                                                 int64_t rows_left, int tid, int lane, int wave, int wn0,
                                                 int split) {
    constexpr int T = C::kThreads;
    auto internal_col = [](int p) -> int { return OUT_T ? (p % D) * C::kCPR + p / D : p; };
    // ---- epilogue: per 16-row MFMA block row, accumulators -> LDS (fp32, in
    // the tile's internal column order, so 16 lanes write 16 consecutive
    // words) -> real column order on the way out -> bias / GELU / GELU' ->
    // bf16 -> coalesced 16-byte stores.  Block rows alternate between two
    // staging buffers, so one barrier per block row suffices.  Bias and the
    // stashed pre-activations are loaded ahead of use (the latter one block row
    // ahead), so no global load latency sits between a block row's LDS round
    // trip and its stores.
    constexpr int kG8 = BN / 8;                          // 8-column groups per row
    constexpr int kGroups = C::kEpiRows * kG8;
    constexpr int kQ = (kGroups + T - 1) / T;            // groups per thread and block row
    constexpr bool kRagged = kGroups % T != 0;
    constexpr int kBiasQ = T % kG8 == 0 ? 1 : kQ;        // passes with distinct columns
    const bool grad = !PARTIAL && a.epilogue == kEpiGeluGrad;
    const bool act = !PARTIAL && a.epilogue == kEpiBiasGelu;
    const bool bias = !PARTIAL && a.bias != nullptr && !grad;
    const bool keep_h = act && a.h_out != nullptr;
    // The tile's rows as buffers: rows past the batch read zero and drop stores.
    const uint32_t rows_t = (uint32_t)(rows_left < BM ? rows_left : BM);
    const uint32_t o_bytes = rows_t * (uint32_t)a.Nout * 2u;
    const __amdgpu_buffer_rsrc_t rO = buffer_rsrc(a.out + m0 * a.Nout, o_bytes);
    const uint16_t *hbase = grad ? a.h_in : a.h_out;
    const __amdgpu_buffer_rsrc_t rH = buffer_rsrc((hbase ? hbase : a.out) + m0 * a.Nout, o_bytes);
    const uint32_t row16 = 16u * (uint32_t)a.Nout * 2u;  // bytes between block rows

    uint32_t voE[kQ];
    int c8of[kQ], erof[kQ];
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
        const int gidx = tid + q * T;
        erof[q] = gidx / kG8;
        c8of[q] = (gidx % kG8) * 8;
        const uint32_t row = (uint32_t)((erof[q] / 16) * C::WM + (erof[q] % 16));
        voE[q] = (row * (uint32_t)a.Nout + (uint32_t)(n0 + c8of[q])) * 2u;
    }
    uint4 bq[kBiasQ];
    if (bias) {
#pragma unroll
        for (int q = 0; q < kBiasQ; ++q) bq[q] = ldg16(a.bias + n0 + c8of[q]);
    }
    uint4 hq[2][kQ];
    float pa[ADD ? kQ : 1][8];
    const __amdgpu_buffer_rsrc_t rS =
        ADD ? buffer_rsrc(a.part + ((int64_t)a.slice0 * a.M + m0) * a.Nout, 2u * o_bytes) : rO;
    if (grad) {
#pragma unroll
        for (int q = 0; q < kQ; ++q) hq[0][q] = bload16_stream(rH, voE[q], 0);
    }

#pragma unroll
    for (int i = 0; i < C::kSubM; ++i) {
        float *ldsE = reinterpret_cast<float *>(smem) + (i & 1) * C::kEpiElems;
        if constexpr (ADD) {
            // this block row's slice values, in flight over the LDS round trip
#pragma unroll
            for (int q = 0; q < kQ; ++q) {
                const uint32_t vb = 2u * (voE[q] + (uint32_t)i * row16);
                if (a.unperm) {
                    const uint32_t rowb = vb - (uint32_t)(n0 + c8of[q]) * 4u;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int c = n0 + c8of[q] + e;
                        const uint32_t at = (uint32_t)((c % (int)a.D) * (int)a.bn + c / (int)a.D);
                        pa[q][e] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rS, (int)(rowb + 4u * at), 0, 0));
                    }
                } else {
                    const u32x4_t lo = __builtin_amdgcn_raw_buffer_load_b128(rS, (int)vb, 0, 0);
                    const u32x4_t hi = __builtin_amdgcn_raw_buffer_load_b128(rS, (int)(vb + 16u), 0, 0);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        pa[q][e] = __uint_as_float(lo[e]);
                        pa[q][4 + e] = __uint_as_float(hi[e]);
                    }
                }
            }
        }
#pragma unroll
        for (int j = 0; j < C::kSubN; ++j) {
            const int col = wn0 + j * 16 + (lane & 15);
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int er = (wave / C::kWGN) * 16 + (lane >> 4) * 4 + v;
                ldsE[er * C::kEpiPitch + col] = acc[i][j][v];
            }
        }
        __syncthreads();
        if (grad && i + 1 < C::kSubM) {
#pragma unroll
            for (int q = 0; q < kQ; ++q) hq[(i + 1) & 1][q] = bload16_stream(rH, voE[q] + (uint32_t)(i + 1) * row16, 0);
        }
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
            if (kRagged && tid + q * T >= kGroups) break;
            const float *rowE = ldsE + erof[q] * C::kEpiPitch;
            const int c8 = c8of[q];
            float x[8];
            if constexpr (OUT_T) {
                // real column c8 + e sits at internal column internal_col(c8 + e)
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] = rowE[internal_col(c8 + e)];
            } else {
                const float4 lo = *reinterpret_cast<const float4 *>(rowE + c8);
                const float4 hi = *reinterpret_cast<const float4 *>(rowE + c8 + 4);
                x[0] = lo.x; x[1] = lo.y; x[2] = lo.z; x[3] = lo.w;
                x[4] = hi.x; x[5] = hi.y; x[6] = hi.z; x[7] = hi.w;
            }
            const uint32_t vo = voE[q] + (uint32_t)i * row16;
            if constexpr (PARTIAL) {
                const __amdgpu_buffer_rsrc_t rP =
                    buffer_rsrc(a.part + ((int64_t)(a.slice0 + split) * a.M + m0) * a.Nout, 2u * o_bytes);
                if (a.unperm) {
                    // column c = j*D + g of the tile's output space is column g*bn + j
                    const uint32_t rowb = 2u * vo - (uint32_t)(n0 + c8) * 4u;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const int c = n0 + c8 + e;
                        const uint32_t real = (uint32_t)((c % (int)a.D) * (int)a.bn + c / (int)a.D);
                        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x[e]), rP, (int)(rowb + 4u * real), 0, 0);
                    }
                    continue;
                }
                const u32x4_t lo = {__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]), __float_as_uint(x[3])};
                const u32x4_t hi = {__float_as_uint(x[4]), __float_as_uint(x[5]), __float_as_uint(x[6]), __float_as_uint(x[7])};
                __builtin_amdgcn_raw_buffer_store_b128(lo, rP, (int)(2u * vo), 0, 0);
                __builtin_amdgcn_raw_buffer_store_b128(hi, rP, (int)(2u * vo + 16u), 0, 0);
                continue;
            }
            if constexpr (ADD) {
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] += pa[q][e];
            }
            if (grad) {
                const uint4 h = hq[i & 1][q];
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] *= gelu_grad(unpack_bf16(word_of(h, e >> 1), e & 1));
            } else {
                if (bias) {
                    const uint4 b = bq[kBiasQ == 1 ? 0 : q];
#pragma unroll
                    for (int e = 0; e < 8; ++e) x[e] += unpack_bf16(word_of(b, e >> 1), e & 1);
                }
                if (act) {
                    if (keep_h)
                        bstore16(rH, vo, make_uint4(pack_bf16(x[0], x[1]), pack_bf16(x[2], x[3]),
                                                    pack_bf16(x[4], x[5]), pack_bf16(x[6], x[7])));
#pragma unroll
                    for (int e = 0; e < 8; ++e) x[e] = gelu(x[e]);
                }
            }
            bstore16(rO, vo, make_uint4(pack_bf16(x[0], x[1]), pack_bf16(x[2], x[3]), pack_bf16(x[4], x[5]),
                                        pack_bf16(x[6], x[7])));
        }
    }
}

// Epilogue of a tile over zero-padded block-ordered operands (the padded
// forms of a pass whose widths or blocks fit no tile).  The tile's columns
// lie in one padded block g of a.bn columns; column n0 + t is real column
// cbase + t (cbase = g * a.bn_r + n0 % a.bn) while t < nt, the real columns
// left in the block and the row; the rest is padding and is dropped.  Real
// rows have a.Nout_r columns, and a real block need not start on a 16-byte
// boundary, so the accumulators are staged in LDS shifted by cbase % 8:
// 8-column units aligned in the real row are then aligned in LDS as well.
// Whole units (all 8 columns real) move as 16 bytes; the at most two ragged
// units of a row (the tile's ends) go element by element in a pass of their
// own, so no wave carries both forms.  Bias, the stashed pre-activation, the
// GELU' input and the output sit at real columns.  ADD: each sum first gets
// the fp32 sum of component 2 from slice a.slice0 of a.part (padded block
// order, rows of a.Nout) at column (c % D) * a.bn + c / D of real column c
// (component 2 under an output transpose).
template <class C, int BM, int BN, bool ADD>
__device__ __forceinline__ void gemm_epilogue_pad(const GemmArgs &a, unsigned char *smem,
                                                  const f32x4_t (&acc)[C::kSubM][C::kSubN], int64_t m0, int n0,
                                                  int64_t rows_left, int tid, int lane, int wave, int wn0) {
    constexpr int T = C::kThreads;
    constexpr int kPitch = BN + 12;                // room for the shift, rows 16-byte aligned
    constexpr int kElems = C::kEpiRows * kPitch;
    static_assert(2 * kElems * 4 <= C::kLds, "two shifted staging buffers fit the tile's LDS");
    const bool grad = a.epilogue == kEpiGeluGrad;
    const bool act = a.epilogue == kEpiBiasGelu;
    const bool bias = a.bias != nullptr && !grad;
    const bool keep_h = act && a.h_out != nullptr;
    const int D = (int)a.D, bnp = (int)a.bn, bnr = (int)a.bn_r;
    const uint32_t Nr = (uint32_t)a.Nout_r, Np = (uint32_t)a.Nout;
    const uint32_t rows_t = (uint32_t)(rows_left < BM ? rows_left : BM);
    const __amdgpu_buffer_rsrc_t rO = buffer_rsrc(a.out + m0 * a.Nout_r, rows_t * Nr * 2u);
    const uint16_t *hbase = grad ? a.h_in : a.h_out;
    const __amdgpu_buffer_rsrc_t rH = buffer_rsrc((hbase ? hbase : a.out) + m0 * a.Nout_r, rows_t * Nr * 2u);
    const __amdgpu_buffer_rsrc_t rS =
        buffer_rsrc(ADD ? a.part + ((int64_t)a.slice0 * a.M + m0) * a.Nout : nullptr, ADD ? rows_t * Np * 4u : 0u);
    const int g = n0 / bnp, j0 = n0 - g * bnp;
    const int cbase = g * bnr + j0;
    int nt = bnr - j0 < BN ? bnr - j0 : BN;
    if ((int)Nr - cbase < nt) nt = (int)Nr - cbase;
    const int sh = cbase & 7, ubase = cbase - sh;
    // units (8 LDS columns 8u .. 8u + 7 = real columns ubase + 8u ..): whole
    // ones u_lo .. u_hi - 1, ragged ones 0 (when shifted) and u_hi (when a tail is left)
    const bool vec = Nr % 8 == 0;
    const int u_lo = vec ? (sh ? 1 : 0) : 0, u_hi = vec && nt > 0 ? (nt + sh) / 8 : 0;
    const int n_whole = u_hi > u_lo ? u_hi - u_lo : 0;
    // a tail unit u_hi unless unit 0 already holds the tail (nt + sh < 8)
    const bool tail = (nt + sh) % 8 != 0 && !(sh && u_hi == 0);
    int n_rag = vec ? (sh ? 1 : 0) + (tail ? 1 : 0) : (nt + sh + 7) / 8;
    if (nt <= 0) n_rag = 0;

    // the epilogue of one unit; WHOLE: all 8 columns real (and 16-byte aligned)
    auto unit = [&](auto whole_tag, const float *ldsE, int erow, int u, int i) __attribute__((always_inline)) {
        constexpr bool WHOLE = decltype(whole_tag)::value;
        const int t0 = 8 * u - sh, r0 = ubase + 8 * u;
        const float *src = ldsE + erow * kPitch + 8 * u;
        const float4 lo = *reinterpret_cast<const float4 *>(src);
        const float4 hi = *reinterpret_cast<const float4 *>(src + 4);
        float x[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        const uint32_t row = (uint32_t)((erow / 16) * C::WM + (erow % 16) + i * 16);
        uint32_t vo[8];   // byte offsets of the unit's real columns; kNoLoad where absent
#pragma unroll
        for (int e = 0; e < 8; ++e)
            vo[e] = (WHOLE || (t0 + e >= 0 && t0 + e < nt)) ? (row * Nr + (uint32_t)(r0 + e)) * 2u : kNoLoad;
        const uint32_t vu = (row * Nr + (uint32_t)r0) * 2u;
        if constexpr (ADD) {
            // slice column (c % D) * bnp + c / D, stepped along the unit
            int res = r0 % D, quo = r0 / D;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const uint32_t so = vo[e] == kNoLoad ? kNoLoad : (row * Np + (uint32_t)(res * bnp + quo)) * 4u;
                x[e] += __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rS, (int)so, 0, 0));
                const bool wrap = ++res == D;
                res = wrap ? 0 : res;
                quo += wrap ? 1 : 0;
            }
        }
        if (bias) {
            if constexpr (WHOLE) {
                const uint4 b = ldg16(a.bias + r0);
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] += unpack_bf16(word_of(b, e >> 1), e & 1);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (vo[e] != kNoLoad) x[e] += bf16_to_f32(a.bias[r0 + e]);
            }
        }
        if (grad) {
            if constexpr (WHOLE) {
                const uint4 h = bload16_stream(rH, vu, 0);
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] *= gelu_grad(unpack_bf16(word_of(h, e >> 1), e & 1));
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint32_t h = __builtin_amdgcn_raw_buffer_load_b16(rH, (int)vo[e], 0, 0);
                    x[e] *= gelu_grad(__uint_as_float(h << 16));
                }
            }
        } else if (act) {
            if (keep_h) {
                if constexpr (WHOLE) {
                    bstore16(rH, vu, make_uint4(pack_bf16(x[0], x[1]), pack_bf16(x[2], x[3]), pack_bf16(x[4], x[5]),
                                                pack_bf16(x[6], x[7])));
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        __builtin_amdgcn_raw_buffer_store_b16((unsigned short)f32_to_bf16(x[e]), rH, (int)vo[e], 0, 0);
                }
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] = gelu(x[e]);
        }
        if constexpr (WHOLE) {
            bstore16(rO, vu, make_uint4(pack_bf16(x[0], x[1]), pack_bf16(x[2], x[3]), pack_bf16(x[4], x[5]),
                                        pack_bf16(x[6], x[7])));
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
                __builtin_amdgcn_raw_buffer_store_b16((unsigned short)f32_to_bf16(x[e]), rO, (int)vo[e], 0, 0);
        }
    };

#pragma unroll
    for (int i = 0; i < C::kSubM; ++i) {
        float *ldsE = reinterpret_cast<float *>(smem) + (i & 1) * kElems;
#pragma unroll
        for (int j = 0; j < C::kSubN; ++j) {
            const int col = wn0 + j * 16 + (lane & 15) + sh;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int er = (wave / C::kWGN) * 16 + (lane >> 4) * 4 + v;
                ldsE[er * kPitch + col] = acc[i][j][v];
            }
        }
        __syncthreads();
        for (int w = tid; w < C::kEpiRows * n_whole; w += T)
            unit(std::true_type{}, ldsE, w / n_whole, u_lo + w % n_whole, i);
        // ragged units: unit 0 when shifted, then unit u_hi (all units when rows are unaligned)
        for (int w = tid; w < C::kEpiRows * n_rag; w += T) {
            const int k = w % n_rag;
            const int u = vec ? (sh && k == 0 ? 0 : u_hi) : k;
            unit(std::false_type{}, ldsE, w / n_rag, u, i);
        }
    }
}

// The epilogue, or with a split reduction (a.part set) the fp32 partial sums:
// two inlined instances, so the bias / GELU / GELU' path carries no test of it.
template <class C, int BM, int BN, int D, bool OUT_T>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs &a, unsigned char *smem,
                                              const f32x4_t (&acc)[C::kSubM][C::kSubN], int64_t m0, int n0,
                                              int64_t rows_left, int tid, int lane, int wave, int wn0, int split) {
    if (a.part)
        gemm_epilogue_as<C, BM, BN, D, OUT_T, true>(a, smem, acc, m0, n0, rows_left, tid, lane, wave, wn0, split);
    else
        gemm_epilogue_as<C, BM, BN, D, OUT_T, false>(a, smem, acc, m0, n0, rows_left, tid, lane, wave, wn0, split);
}

}  // namespace dyad
