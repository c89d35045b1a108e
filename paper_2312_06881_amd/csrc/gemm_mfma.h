// The Dyad grouped GEMM on gfx950 matrix cores (bf16 in, fp32 accumulate).
//
// One workgroup computes an output tile of BM tokens x BN output features.
// Both weight components run in one K loop ("K-concat"): the tile's
// accumulators take the BlockDiag component's product first, then the
// BlockTrans component's, so neither partial result ever leaves registers.
//
// Tile columns.  Without an output transpose (out_t == 0) the BN columns lie
// in one output block g and use weight rows j0..j0+BN of group g in both
// components.  With an output transpose the BN columns still lie in one block
// g1 (which fixes the BlockDiag rows), but column f of the BlockTrans component
// comes from group f % D, row f / D.  The tile keeps its accumulator columns in
// "residue-major" order, internal column p = r*(BN/D) + t holding real column
// r + D*t, so that every 16-wide MFMA sub-tile of the BlockTrans product reads
// one group r and consecutive weight rows of it.  The store undoes the order.
//
// Operand staging.  Each K stage copies its operand tiles global -> registers
// -> LDS.  The BlockTrans component with an input transpose reads the input
// columns k*D + r: the stage loads the contiguous span of 32*D input columns
// that holds 32 consecutive k for every residue r, and de-interleaves it in
// registers into one [BM][32] slab per residue, so the strided view is never
// materialised in HBM and every global load stays a 16-byte contiguous load.
#pragma once

#include "dyad_device.h"
#include "dyad_internal.h"

namespace dyad {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;

constexpr int kStageK = 32;     // k per slab and per MFMA (v_mfma_f32_16x16x32_bf16)
constexpr int kLdsPadK = 8;     // bf16 elements of padding per LDS row
constexpr int kRowK = kStageK + kLdsPadK;
constexpr int kThreads = 256;   // four wave64s

struct GemmArgs {
    int64_t M, Kin, Nout, bk, bn;
    const uint16_t *in, *W1, *W2, *bias, *h_in;
    uint16_t *out, *h_out;
    int epilogue;
    int tiles_n;        // output tiles per token panel
    int tiles_total;
};

// Element e (0..8*D-1) of a run of D consecutive 16-byte vectors, as 16 bits.
template <int D>
__device__ __forceinline__ uint32_t elem16(const uint4 (&v)[D], int e) {
    const uint4 &q = v[e >> 3];
    const int w = (e >> 1) & 3;
    const uint32_t d = w == 0 ? q.x : w == 1 ? q.y : w == 2 ? q.z : q.w;
    return (e & 1) ? (d >> 16) : (d & 0xffffu);
}

// From 8*D consecutive input columns (8 k values x D residues, residue fastest),
// the 8 values of residue r as one 16-byte vector.
template <int D>
__device__ __forceinline__ uint4 deinterleave(const uint4 (&v)[D], int r) {
    uint4 o;
    o.x = elem16<D>(v, 0 * D + r) | (elem16<D>(v, 1 * D + r) << 16);
    o.y = elem16<D>(v, 2 * D + r) | (elem16<D>(v, 3 * D + r) << 16);
    o.z = elem16<D>(v, 4 * D + r) | (elem16<D>(v, 5 * D + r) << 16);
    o.w = elem16<D>(v, 6 * D + r) | (elem16<D>(v, 7 * D + r) << 16);
    return o;
}

__device__ __forceinline__ uint4 ldg16(const uint16_t *p) { return *reinterpret_cast<const uint4 *>(p); }

// Tile index -> (token panel, column tile), with consecutive tiles of one
// panel placed on one XCD (workgroups are dealt round-robin over 8 XCDs).
__device__ __forceinline__ int xcd_tile(int w, int total) {
    const int q = total >> 3, r = total & 7, x = w & 7, i = w >> 3;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + i;
}

template <int BM, int BN, int WM, int WN, int D, bool IN_T, bool OUT_T, bool W_T>
struct GemmTile {
    static constexpr int kWavesN = BN / WN;
    static constexpr int kSubM = WM / 16;
    static constexpr int kSubN = WN / 16;
    static constexpr int kColsPerRes = OUT_T ? BN / D : BN;
    // slabs of A held in LDS during a BlockTrans stage
    static constexpr int kSlabs2 = OUT_T ? D : 1;
    // 16-byte vectors of a [BM][32] slab, and per thread
    static constexpr int kVecA = BM * kStageK / 8;
    static constexpr int kVecAThr = kVecA / kThreads;
    // A vectors in flight per thread: span chunks of D vectors, or D slabs
    static constexpr int kRegA = kVecAThr * ((IN_T || OUT_T) ? D : 1);
    static constexpr int kVecB = BN * kStageK / 8;
    static constexpr int kRegB = kVecB / kThreads;
    static constexpr int kLdsA = kSlabs2 * BM * kRowK * 2;
    static constexpr int kLdsB = BN * kRowK * 2;
    static constexpr int kEpiRow = BN + 4;   // fp32 elements per LDS row in the epilogue
    static constexpr int kLdsEpi = BM * kEpiRow * 4;
    static constexpr int kLds = (kLdsA + kLdsB) > kLdsEpi ? (kLdsA + kLdsB) : kLdsEpi;

    static_assert(kVecA % kThreads == 0 && kVecB % kThreads == 0, "tile / thread mismatch");
    static_assert((BM / WM) * (BN / WN) == 4, "four waves per workgroup");
    static_assert(!OUT_T || (kColsPerRes % 16 == 0), "each MFMA column block must hold one residue");
    static_assert(kLds <= 160 * 1024, "LDS budget");
};

template <int BM, int BN, int WM, int WN, int D, bool IN_T, bool OUT_T, bool W_T>
__global__ void __launch_bounds__(kThreads, 1) dyad_gemm_mfma(GemmArgs a) {
    using T = GemmTile<BM, BN, WM, WN, D, IN_T, OUT_T, W_T>;
    __shared__ __attribute__((aligned(16))) unsigned char smem[T::kLds];
    uint16_t *ldsA = reinterpret_cast<uint16_t *>(smem);
    uint16_t *ldsB = reinterpret_cast<uint16_t *>(smem + T::kLdsA);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int tile = xcd_tile(blockIdx.x, a.tiles_total);
    const int64_t m0 = (int64_t)(tile / a.tiles_n) * BM;
    const int64_t n0 = (int64_t)(tile % a.tiles_n) * BN;   // first output column of the tile
    const int64_t g1 = n0 / a.bn;                          // output block (BlockDiag group)
    const int64_t jb = n0 - g1 * a.bn;                     // first BlockDiag weight row
    const int64_t bk = a.bk, bn = a.bn, Kin = a.Kin;
    const int ks = (int)(bk / kStageK);                    // stages per component

    const int wm0 = (wave / T::kWavesN) * WM;
    const int wn0 = (wave % T::kWavesN) * WN;

    f32x4_t acc[T::kSubM][T::kSubN];
#pragma unroll
    for (int i = 0; i < T::kSubM; ++i)
#pragma unroll
        for (int j = 0; j < T::kSubN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    uint4 ra[T::kRegA];
    uint4 rb[T::kRegB];

    // internal column p -> tile-local real column (and BlockDiag weight row offset)
    auto real_col = [](int p) -> int {
        return OUT_T ? (p / T::kColsPerRes) + D * (p % T::kColsPerRes) : p;
    };

    // ---- global -> registers for stage s (s < ks: BlockDiag, else BlockTrans)
    auto fetch = [&](int s) {
        const bool comp2 = s >= ks;
        const int64_t kk = (int64_t)(comp2 ? s - ks : s) * kStageK;
        // A
        if (!comp2 || !(IN_T || OUT_T)) {
            const int64_t col0 = g1 * bk + kk;
#pragma unroll
            for (int q = 0; q < T::kVecAThr; ++q) {
                const int v = tid + q * kThreads, row = v >> 2, c8 = (v & 3) * 8;
                const int64_t m = m0 + row;
                ra[q] = m < a.M ? ldg16(a.in + m * Kin + col0 + c8) : make_uint4(0, 0, 0, 0);
            }
        } else if (IN_T) {
            // span of 32*D columns holding k = kk..kk+31 for every residue
#pragma unroll
            for (int q = 0; q < T::kVecAThr; ++q) {
                const int c = tid + q * kThreads, row = c >> 2, tg = c & 3;
                const int64_t m = m0 + row;
                const uint16_t *src = a.in + m * Kin + (kk + tg * 8) * D;
#pragma unroll
                for (int d = 0; d < D; ++d)
                    ra[q * D + d] = m < a.M ? ldg16(src + d * 8) : make_uint4(0, 0, 0, 0);
            }
        } else {
            // OUT_T without IN_T: one [BM][32] slab from each input block r
#pragma unroll
            for (int r = 0; r < D; ++r)
#pragma unroll
                for (int q = 0; q < T::kVecAThr; ++q) {
                    const int v = tid + q * kThreads, row = v >> 2, c8 = (v & 3) * 8;
                    const int64_t m = m0 + row;
                    ra[r * T::kVecAThr + q] =
                        m < a.M ? ldg16(a.in + m * Kin + r * bk + kk + c8) : make_uint4(0, 0, 0, 0);
                }
        }
        // B: weight rows of internal columns p
        const uint16_t *W = comp2 ? a.W2 : a.W1;
        if (!W_T) {
#pragma unroll
            for (int q = 0; q < T::kRegB; ++q) {
                const int v = tid + q * kThreads, p = v >> 2, c8 = (v & 3) * 8;
                int64_t grp, row;
                if (!comp2) { grp = g1; row = jb + real_col(p); }
                else if (OUT_T) { grp = p / T::kColsPerRes; row = n0 / D + p % T::kColsPerRes; }
                else { grp = g1; row = jb + p; }
                rb[q] = ldg16(W + (grp * bn + row) * bk + kk + c8);
            }
        } else {
            // weights read transposed: element (row j, k) at W[grp][k][j]; load 8 j at one k
#pragma unroll
            for (int q = 0; q < T::kRegB; ++q) {
                const int v = tid + q * kThreads, k = v / (BN / 8), p8 = (v % (BN / 8)) * 8;
                int64_t grp, row;
                if (!comp2) { grp = g1; row = jb + p8; }                       // real cols p8..p8+7
                else if (OUT_T) { grp = p8 / T::kColsPerRes; row = n0 / D + p8 % T::kColsPerRes; }
                else { grp = g1; row = jb + p8; }
                rb[q] = ldg16(W + (grp * bk + kk + k) * bn + row);
            }
        }
    };

    // ---- registers -> LDS
    auto stash = [&](int s) {
        const bool comp2 = s >= ks;
        if (!comp2 || !(IN_T || OUT_T)) {
#pragma unroll
            for (int q = 0; q < T::kVecAThr; ++q) {
                const int v = tid + q * kThreads, row = v >> 2, c8 = (v & 3) * 8;
                *reinterpret_cast<uint4 *>(ldsA + row * kRowK + c8) = ra[q];
            }
        } else if (IN_T) {
#pragma unroll
            for (int q = 0; q < T::kVecAThr; ++q) {
                const int c = tid + q * kThreads, row = c >> 2, tg = c & 3;
                uint4 chunk[D];
#pragma unroll
                for (int d = 0; d < D; ++d) chunk[d] = ra[q * D + d];
                if (OUT_T) {
#pragma unroll
                    for (int r = 0; r < D; ++r)
                        *reinterpret_cast<uint4 *>(ldsA + (r * BM + row) * kRowK + tg * 8) =
                            deinterleave<D>(chunk, r);
                } else {
                    // only residue g1 feeds this tile's columns
                    uint4 o = make_uint4(0, 0, 0, 0);
#pragma unroll
                    for (int r = 0; r < D; ++r)
                        if (r == (int)g1) o = deinterleave<D>(chunk, r);
                    *reinterpret_cast<uint4 *>(ldsA + row * kRowK + tg * 8) = o;
                }
            }
        } else {
#pragma unroll
            for (int r = 0; r < D; ++r)
#pragma unroll
                for (int q = 0; q < T::kVecAThr; ++q) {
                    const int v = tid + q * kThreads, row = v >> 2, c8 = (v & 3) * 8;
                    *reinterpret_cast<uint4 *>(ldsA + (r * BM + row) * kRowK + c8) =
                        ra[r * T::kVecAThr + q];
                }
        }
        if (!W_T) {
#pragma unroll
            for (int q = 0; q < T::kRegB; ++q) {
                const int v = tid + q * kThreads, p = v >> 2, c8 = (v & 3) * 8;
                *reinterpret_cast<uint4 *>(ldsB + p * kRowK + c8) = rb[q];
            }
        } else {
#pragma unroll
            for (int q = 0; q < T::kRegB; ++q) {
                const int v = tid + q * kThreads, k = v / (BN / 8), p8 = (v % (BN / 8)) * 8;
                const uint32_t w[4] = {rb[q].x, rb[q].y, rb[q].z, rb[q].w};
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    // element e is real column (BlockDiag) / internal column (BlockTrans) p8+e
                    int p;
                    if (!comp2) {
                        const int c = p8 + e;   // real local column -> internal column
                        p = OUT_T ? (c % D) * T::kColsPerRes + c / D : c;
                    } else {
                        p = p8 + e;
                    }
                    ldsB[p * kRowK + k] = (uint16_t)((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xffffu));
                }
            }
        }
    };

    // ---- MFMA on the staged tiles
    auto compute = [&](int s) {
        const bool comp2 = s >= ks;
        const int kq = (lane >> 4) * 8;
        bf16x8_t bfrag[T::kSubN];
#pragma unroll
        for (int j = 0; j < T::kSubN; ++j)
            bfrag[j] = *reinterpret_cast<const bf16x8_t *>(ldsB + (wn0 + j * 16 + (lane & 15)) * kRowK + kq);
        if (!comp2 || !OUT_T) {
#pragma unroll
            for (int i = 0; i < T::kSubM; ++i) {
                const bf16x8_t afrag =
                    *reinterpret_cast<const bf16x8_t *>(ldsA + (wm0 + i * 16 + (lane & 15)) * kRowK + kq);
#pragma unroll
                for (int j = 0; j < T::kSubN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag, bfrag[j], acc[i][j], 0, 0, 0);
            }
        } else {
#pragma unroll
            for (int i = 0; i < T::kSubM; ++i) {
#pragma unroll
                for (int j = 0; j < T::kSubN; ++j) {
                    const int r = (wn0 + j * 16) / T::kColsPerRes;
                    const bf16x8_t afrag = *reinterpret_cast<const bf16x8_t *>(
                        ldsA + (r * BM + wm0 + i * 16 + (lane & 15)) * kRowK + kq);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag, bfrag[j], acc[i][j], 0, 0, 0);
                }
            }
        }
    };

    const int S = 2 * ks;
    fetch(0);
    for (int s = 0; s < S; ++s) {
        __syncthreads();
        stash(s);
        __syncthreads();
        if (s + 1 < S) fetch(s + 1);
        compute(s);
    }
    __syncthreads();

    // ---- epilogue: accumulators -> LDS (real column order) -> coalesced stores
    float *ldsE = reinterpret_cast<float *>(smem);
#pragma unroll
    for (int i = 0; i < T::kSubM; ++i)
#pragma unroll
        for (int j = 0; j < T::kSubN; ++j) {
            const int c = real_col(wn0 + j * 16 + (lane & 15));
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = wm0 + i * 16 + (lane >> 4) * 4 + v;
                ldsE[row * T::kEpiRow + c] = acc[i][j][v];
            }
        }
    __syncthreads();
    constexpr int kChunks = BM * BN / 8;
#pragma unroll
    for (int q = 0; q < kChunks / kThreads; ++q) {
        const int ch = tid + q * kThreads, row = ch / (BN / 8), c8 = (ch % (BN / 8)) * 8;
        const int64_t m = m0 + row;
        if (m >= a.M) continue;
        float x[8];
        const float4 lo = *reinterpret_cast<const float4 *>(ldsE + row * T::kEpiRow + c8);
        const float4 hi = *reinterpret_cast<const float4 *>(ldsE + row * T::kEpiRow + c8 + 4);
        x[0] = lo.x; x[1] = lo.y; x[2] = lo.z; x[3] = lo.w;
        x[4] = hi.x; x[5] = hi.y; x[6] = hi.z; x[7] = hi.w;
        const int64_t off = m * a.Nout + n0 + c8;
        if (a.epilogue == kEpiGeluGrad) {
            const uint4 h = ldg16(a.h_in + off);
            const uint32_t hw[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
            for (int e = 0; e < 8; ++e)
                x[e] *= gelu_grad_f32(bf16_to_f32((uint16_t)((e & 1) ? (hw[e >> 1] >> 16) : (hw[e >> 1] & 0xffffu))));
        } else {
            if (a.bias) {
                const uint4 b = ldg16(a.bias + n0 + c8);
                const uint32_t bw[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    x[e] += bf16_to_f32((uint16_t)((e & 1) ? (bw[e >> 1] >> 16) : (bw[e >> 1] & 0xffffu)));
            }
            if (a.epilogue == kEpiBiasGelu) {
                if (a.h_out) {
                    uint4 o;
                    o.x = f32_to_bf16(x[0]) | ((uint32_t)f32_to_bf16(x[1]) << 16);
                    o.y = f32_to_bf16(x[2]) | ((uint32_t)f32_to_bf16(x[3]) << 16);
                    o.z = f32_to_bf16(x[4]) | ((uint32_t)f32_to_bf16(x[5]) << 16);
                    o.w = f32_to_bf16(x[6]) | ((uint32_t)f32_to_bf16(x[7]) << 16);
                    *reinterpret_cast<uint4 *>(a.h_out + off) = o;
                }
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] = gelu_f32(x[e]);
            }
        }
        uint4 o;
        o.x = f32_to_bf16(x[0]) | ((uint32_t)f32_to_bf16(x[1]) << 16);
        o.y = f32_to_bf16(x[2]) | ((uint32_t)f32_to_bf16(x[3]) << 16);
        o.z = f32_to_bf16(x[4]) | ((uint32_t)f32_to_bf16(x[5]) << 16);
        o.w = f32_to_bf16(x[6]) | ((uint32_t)f32_to_bf16(x[7]) << 16);
        *reinterpret_cast<uint4 *>(a.out + off) = o;
    }
}

}  // namespace dyad
