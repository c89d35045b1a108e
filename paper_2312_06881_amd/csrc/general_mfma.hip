// Matrix-core forms of the general kernels (bf16): any n_dyad, any block
// sizes, zero-padded widths.
//
// Grouped GEMM (forward, input gradient).  It keeps the class decomposition of the vector
// kernel in kernels_simt.hip -- the output columns of class (g1, g2) all read
// input columns g1*bk + k (BlockDiag) and c2(g2, k) (BlockTrans), so a tile of
// 128 tokens x 128 columns of one class is a plain GEMM with K = 2*bk -- and
// multiplies on v_mfma_f32_16x16x32_bf16.  Operands are gathered element by
// element with 2-byte buffer loads (no alignment or divisibility is assumed;
// reads past a width or past the batch return zero), packed in pairs into the
// swizzled LDS rows the MFMA fragments read, double-buffered with one barrier
// per 32-deep chunk.  Every thread issues the same loads every chunk (invalid
// elements point past the buffer), so the compiler's wait counts stay exact.
//
// Weight gradient.  dWc[g][j][k] = sum_m dZ[m][row_c(g, j)] X[m][col_c(g, k)]
// as 128 x 128 tiles of (component, group) products over K = tokens, the
// tokens split across workgroups when the tiles alone would not fill the GPU;
// fp32 partials per split go to the workspace and are added in split order.
#include <type_traits>

#include "dyad_internal.h"
#include "mfma_common.h"

namespace dyad {
namespace {

constexpr int kGM = 128, kGN = 128;   // tokens x class columns per tile, 4 waves of 64 x 64
constexpr int kPairs = 8;             // element pairs per thread and operand per chunk

struct GClass {
    int64_t g1, g2, first, step, count;
};

__device__ __forceinline__ GClass gclass(const GemmPass &p, int64_t cls) {
    GClass c;
    const int64_t D = p.D;
    if (!p.out_t) {
        c.g1 = c.g2 = cls;
        c.first = cls * p.bn;
        c.step = 1;
        const int64_t end = min((cls + 1) * p.bn, p.Nout);
        c.count = end > c.first ? end - c.first : 0;
    } else {
        c.g1 = cls / D;
        c.g2 = cls % D;
        const int64_t lo = c.g1 * p.bn, hi = min((c.g1 + 1) * p.bn, p.Nout);
        c.first = lo + ((c.g2 - lo % D) % D + D) % D;   // first f >= lo with f % D == g2
        c.step = D;
        c.count = hi > c.first ? (hi - c.first + D - 1) / D : 0;
    }
    return c;
}

__device__ __forceinline__ uint32_t ld2(__amdgpu_buffer_rsrc_t r, uint32_t voff) {
    return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)voff, 0, 0);
}

__device__ __forceinline__ uint32_t ld4(__amdgpu_buffer_rsrc_t r, uint32_t voff) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, 0, 0);
}

// GM tokens x GN class columns per tile (4 waves of 64 x 64).  PAIRS: even
// input width and block size, so every (k, k+1) pair of a contiguous operand
// is one aligned 4-byte load.
template <int GM, int GN, bool PAIRS, bool IN_T, bool W_T>
__global__ void __launch_bounds__(256, 2) general_mfma_kernel(GemmPass p, int col_tiles, int row_tiles) {
    constexpr int kPA = GM / 16, kPB = GN / 16;        // element pairs per thread per chunk
    constexpr int kWGN = GN / 64;                      // waves along the columns
    __shared__ __attribute__((aligned(16))) uint16_t ldsA[2][GM * kStageK];
    __shared__ __attribute__((aligned(16))) uint16_t ldsB[2][GN * kStageK];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int b = blockIdx.x;
    const int rt = b % row_tiles, ct = (b / row_tiles) % col_tiles, cls = b / (row_tiles * col_tiles);
    const GClass cc = gclass(p, cls);
    const int t0 = ct * GN;
    if (t0 >= cc.count) return;                        // uniform: the whole block leaves
    const int64_t m0 = (int64_t)rt * GM;
    const int64_t rows_left = p.M - m0;
    const int bk = (int)p.bk, bn = (int)p.bn, D = (int)p.D, Kin = (int)p.Kin;
    const int nk = 2 * bk, chunks = (nk + kStageK - 1) / kStageK;

    const uint16_t *in = static_cast<const uint16_t *>(p.in);
    const uint32_t a_bytes = (uint32_t)((rows_left < GM ? rows_left : GM) * p.Kin * 2);
    const __amdgpu_buffer_rsrc_t rA = buffer_rsrc(in + m0 * p.Kin, a_bytes);
    const uint32_t w_bytes = (uint32_t)(p.D * p.bn * p.bk * 2);
    const __amdgpu_buffer_rsrc_t rW1 = buffer_rsrc(p.W1, w_bytes);
    const __amdgpu_buffer_rsrc_t rW2 = buffer_rsrc(p.W2, w_bytes);

    // Per-thread constants: A pair q is row arow[q], k pair akp[q]; B pair q is
    // class column bcol[q], k pair bkp[q], weights at bbase{1,2}[q] + k (-1 past the class).
    int arow[kPA], akp[kPA], bkp[kPB], bcol[kPB], bbase1[kPB], bbase2[kPB];
#pragma unroll
    for (int q = 0; q < kPA; ++q) {
        const int pi = tid + 256 * q;
        akp[q] = pi & 15;
        arow[q] = pi >> 4;
    }
#pragma unroll
    for (int q = 0; q < kPB; ++q) {
        const int pi = tid + 256 * q;
        int ci;
        if constexpr (W_T) { ci = pi & (GN - 1); bkp[q] = pi / GN; } else { bkp[q] = pi & 15; ci = pi >> 4; }
        bcol[q] = ci;
        const int64_t t = t0 + ci;
        bbase1[q] = bbase2[q] = -1;
        if (t < cc.count) {
            const int64_t f = cc.first + t * cc.step;
            const int64_t j1 = f - cc.g1 * p.bn, j2 = p.out_t ? f / p.D : j1;
            bbase1[q] = (int)(W_T ? cc.g1 * p.bk * p.bn + j1 : (cc.g1 * p.bn + j1) * p.bk);
            bbase2[q] = (int)(W_T ? cc.g2 * p.bk * p.bn + j2 : (cc.g2 * p.bn + j2) * p.bk);
        }
    }
    const int a_col1 = (int)(cc.g1 * bk);
    const int g2 = (int)cc.g2;

    // byte offset of element kq of the concatenated K (BlockDiag, then BlockTrans)
    auto a_off = [&](int q, int kq) __attribute__((always_inline)) -> uint32_t {
        if (kq >= nk) return kNoLoad;
        const int col = kq < bk ? a_col1 + kq : (IN_T ? (kq - bk) * D + g2 : g2 * bk + (kq - bk));
        if (col >= Kin) return kNoLoad;
        return (uint32_t)(arow[q] * Kin + col) * 2u;
    };
    auto b_off = [&](int q, int kq) __attribute__((always_inline)) -> uint32_t {
        if (kq >= nk || bbase1[q] < 0) return kNoLoad;
        const bool c2 = kq >= bk;
        const int k = c2 ? kq - bk : kq;
        return (uint32_t)((c2 ? bbase2[q] : bbase1[q]) + (W_T ? k * bn : k)) * 2u;
    };

    uint32_t ra[kPA], rb[kPB];                         // packed (k, k+1) pairs
    // Chunk kinds (uniform): 1 all BlockDiag, 2 all BlockTrans, 3 the chunk
    // that straddles k = bk, where every element picks its own form.
    auto fetch_kind = [&](auto kind, int k0) __attribute__((always_inline)) {
        constexpr int K = decltype(kind)::value;
#pragma unroll
        for (int q = 0; q < kPA; ++q) {
            const int kq = k0 + 2 * akp[q];
            const uint32_t o0 = a_off(q, kq), o1 = a_off(q, kq + 1);
            constexpr bool c1_pairs = PAIRS, c2_pairs = PAIRS && !IN_T;
            if constexpr ((K == 1 && c1_pairs) || (K == 2 && c2_pairs) || (K == 3 && c1_pairs && c2_pairs)) {
                ra[q] = ld4(rA, o0);
            } else if constexpr (K == 3 && c1_pairs) {
                // BlockDiag pairs contiguous, strided BlockTrans pairs element by element
                const bool c2 = kq >= bk;
                ra[q] = ld4(rA, c2 ? kNoLoad : o0) |
                        (ld2(rA, c2 ? o0 : kNoLoad) | (ld2(rA, c2 ? o1 : kNoLoad) << 16));
            } else {
                ra[q] = ld2(rA, o0) | (ld2(rA, o1) << 16);
            }
        }
#pragma unroll
        for (int q = 0; q < kPB; ++q) {
            const int kq = k0 + 2 * bkp[q];
            const uint32_t o0 = b_off(q, kq), o1 = b_off(q, kq + 1);
            if constexpr (PAIRS && !W_T) {
                if constexpr (K == 1) rb[q] = ld4(rW1, o0);
                else if constexpr (K == 2) rb[q] = ld4(rW2, o0);
                else rb[q] = ld4(rW1, kq < bk ? o0 : kNoLoad) | ld4(rW2, kq < bk ? kNoLoad : o0);
            } else {
                uint32_t h[2];
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const uint32_t o = e ? o1 : o0;
                    const int ke = kq + e;
                    if constexpr (K == 1) h[e] = ld2(rW1, o);
                    else if constexpr (K == 2) h[e] = ld2(rW2, o);
                    else h[e] = ld2(rW1, ke < bk ? o : kNoLoad) | ld2(rW2, ke < bk ? kNoLoad : o);
                }
                rb[q] = h[0] | (h[1] << 16);
            }
        }
    };
    auto fetch = [&](int c) __attribute__((always_inline)) {
        const int k0 = c * kStageK;
        if (k0 + kStageK <= bk) fetch_kind(std::integral_constant<int, 1>{}, k0);
        else if (k0 >= bk) fetch_kind(std::integral_constant<int, 2>{}, k0);
        else fetch_kind(std::integral_constant<int, 3>{}, k0);
    };
    auto stash = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < kPA; ++q)
            *reinterpret_cast<uint32_t *>(ldsA[buf] + lds_off(arow[q], akp[q] >> 2) + (akp[q] & 3) * 2) = ra[q];
#pragma unroll
        for (int q = 0; q < kPB; ++q)
            *reinterpret_cast<uint32_t *>(ldsB[buf] + lds_off(bcol[q], bkp[q] >> 2) + (bkp[q] & 3) * 2) = rb[q];
    };

    const int wm0 = (wave / kWGN) * 64, wn0 = (wave % kWGN) * 64;
    const int lr = lane & 15, lc = lane >> 4;
    f32x4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    fetch(0);
    stash(0);
    __syncthreads();
    for (int c = 0; c < chunks; ++c) {
        const int buf = c & 1;
        if (c + 1 < chunks) fetch(c + 1);
        const uint16_t *A = ldsA[buf], *B = ldsB[buf];
        bf16x8_t af[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const bf16x8_t *>(A + lds_off(wm0 + 16 * i + lr, lc));
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const bf16x8_t bf = *reinterpret_cast<const bf16x8_t *>(B + lds_off(wn0 + 16 * j + lr, lc));
#pragma unroll
            for (int i = 0; i < 4; ++i)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf, acc[i][j], 0, 0, 0);
        }
        if (c + 1 < chunks) stash(buf ^ 1);
        __syncthreads();
    }

    // Epilogue straight from the accumulators: lane holds rows 4*(lane/16)+v,
    // column lane%16 of each 16 x 16 block.
    uint16_t *out = static_cast<uint16_t *>(p.out);
    const uint16_t *bias = static_cast<const uint16_t *>(p.bias);
    const uint16_t *h_in = static_cast<const uint16_t *>(p.h_in);
    uint16_t *h_out = static_cast<uint16_t *>(p.h_out);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int64_t t = t0 + wn0 + 16 * j + lr;
        if (t >= cc.count) continue;
        const int64_t f = cc.first + t * cc.step;
        const float bv = (p.epilogue != kEpiGeluGrad && bias) ? bf16_to_f32(bias[f]) : 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t m = m0 + wm0 + 16 * i + 4 * lc + v;
                if (m >= p.M) continue;
                const int64_t e = m * p.Nout + f;
                float x = acc[i][j][v];
                if (p.epilogue == kEpiGeluGrad) {
                    x *= gelu_grad(bf16_to_f32(h_in[e]));
                } else {
                    x += bv;
                    if (p.epilogue == kEpiBiasGelu) {
                        if (h_out) h_out[e] = f32_to_bf16(x);
                        x = gelu(x);
                    }
                }
                out[e] = f32_to_bf16(x);
            }
    }
}

// One split's tile of dW for one component: rows j (dZ side), columns k (X
// side), K = tokens.  Operands sit in LDS token-major (one 272-byte row of 128
// entry columns per token, 16 bytes of pad) and the MFMA operands -- 8 tokens
// of one column per lane -- come from ds_read_b64_tr_b16.  ZP / XP: the
// operand's columns are contiguous with even offsets, so column pairs are one
// aligned 4-byte load.
constexpr int kDwPitch = 128 * 2 + 16;   // bytes per token row

template <bool ZP, bool XP>
__global__ void __launch_bounds__(256, 2) general_mfma_dw_kernel(DwPass p, int comp, int jt_n, int kt_n, int splits,
                                                                 int64_t tps, float *part) {
    __shared__ __attribute__((aligned(16))) unsigned char lds[2][2][kStageK * kDwPitch];   // [buffer][dZ, X]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int b = blockIdx.x;
    const int D = (int)p.D;
    const int kt = b % kt_n, jt = (b / kt_n) % jt_n, g = (b / (kt_n * jt_n)) % D;
    const int split = b / (kt_n * jt_n * D);
    const int bo = (int)p.bo, bi = (int)p.bi, n_out = (int)p.n_out, n_in = (int)p.n_in;
    const int j0 = jt * 128, k0 = kt * 128;
    const bool row_t = comp == 2 && p.out_t, col_t = comp == 2 && p.in_t;
    const int64_t m_lo = (int64_t)split * tps;
    const int64_t m_hi = min(m_lo + tps, p.M);
    const int rows = (int)(m_hi > m_lo ? m_hi - m_lo : 0);
    const int chunks = (rows + kStageK - 1) / kStageK;

    const __amdgpu_buffer_rsrc_t rZ =
        buffer_rsrc(static_cast<const uint16_t *>(p.dZ) + m_lo * p.n_out, (uint32_t)rows * (uint32_t)n_out * 2u);
    const __amdgpu_buffer_rsrc_t rX =
        buffer_rsrc(static_cast<const uint16_t *>(p.X) + m_lo * p.n_in, (uint32_t)rows * (uint32_t)n_in * 2u);

    // pair q: entry columns 2 cp, 2 cp + 1 of token row mm of the chunk
    int cp[kPairs], mm[kPairs], zc[kPairs][2], xc[kPairs][2];
#pragma unroll
    for (int q = 0; q < kPairs; ++q) {
        const int pi = tid + 256 * q;
        cp[q] = pi & 63;
        mm[q] = pi >> 6;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int j = j0 + 2 * cp[q] + h, k = k0 + 2 * cp[q] + h;
            const int row = row_t ? j * D + g : g * bo + j;
            const int col = col_t ? k * D + g : g * bi + k;
            zc[q][h] = (j < bo && row < n_out) ? row : -1;
            xc[q][h] = (k < bi && col < n_in) ? col : -1;
        }
    }
    uint32_t rz[kPairs], rx[kPairs];
    auto fetch = [&](int c) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < kPairs; ++q) {
            const uint32_t m = (uint32_t)(c * kStageK + mm[q]);
            auto off = [&](int col, int width) __attribute__((always_inline)) -> uint32_t {
                return col >= 0 ? (m * (uint32_t)width + (uint32_t)col) * 2u : kNoLoad;
            };
            if constexpr (ZP) rz[q] = ld4(rZ, off(zc[q][0], n_out));
            else rz[q] = ld2(rZ, off(zc[q][0], n_out)) | (ld2(rZ, off(zc[q][1], n_out)) << 16);
            if constexpr (XP) rx[q] = ld4(rX, off(xc[q][0], n_in));
            else rx[q] = ld2(rX, off(xc[q][0], n_in)) | (ld2(rX, off(xc[q][1], n_in)) << 16);
        }
    };
    auto stash = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < kPairs; ++q) {
            const int off = mm[q] * kDwPitch + 4 * cp[q];
            *reinterpret_cast<uint32_t *>(lds[buf][0] + off) = rz[q];
            *reinterpret_cast<uint32_t *>(lds[buf][1] + off) = rx[q];
        }
    };

    const int wm0 = (wave >> 1) * 64, wn0 = (wave & 1) * 64;
    const int lr = lane & 15, lc = lane >> 4;
    // transpose-read lane offsets: token row 8*(lane/16) + (lane%16)/4, column 4*(lane%4)
    const int trow = 8 * lc + (lr >> 2), tcol = 4 * (lane & 3);
    // db rides on the BlockDiag items of the first column tile: their dZ
    // fragments times a fragment of ones (one wave column, so once per row)
    const bool do_db = p.db && comp == 1 && kt == 0 && (wave & 1) == 0;
    const bf16x8_t ones = {(__bf16)1.0f, (__bf16)1.0f, (__bf16)1.0f, (__bf16)1.0f,
                           (__bf16)1.0f, (__bf16)1.0f, (__bf16)1.0f, (__bf16)1.0f};
    f32x4_t dacc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) dacc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    f32x4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (chunks > 0) {
        fetch(0);
        stash(0);
    }
    __syncthreads();
    for (int c = 0; c < chunks; ++c) {
        const int buf = c & 1;
        if (c + 1 < chunks) fetch(c + 1);
        const lds_u8 *Z = (const lds_u8 *)lds[buf][0], *Xs = (const lds_u8 *)lds[buf][1];
        bf16x8_t af[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) af[i] = frag_tr(Z + trow * kDwPitch + (wm0 + 16 * i + tcol) * 2, kDwPitch);
        if (do_db) {
#pragma unroll
            for (int i = 0; i < 4; ++i) dacc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], ones, dacc[i], 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const bf16x8_t bf = frag_tr(Xs + trow * kDwPitch + (wn0 + 16 * j + tcol) * 2, kDwPitch);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf, acc[i][j], 0, 0, 0);
        }
        if (c + 1 < chunks) stash(buf ^ 1);
        __syncthreads();
    }

    const int64_t per_comp = p.D * p.bo * p.bi;
    uint16_t *dW = static_cast<uint16_t *>(comp == 1 ? p.dW1 : p.dW2);
    float *dst = part ? part + (int64_t)split * 2 * per_comp + (comp - 1) * per_comp : nullptr;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int j = j0 + wm0 + 16 * i + 4 * lc + v;
            if (j >= bo) continue;
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const int k = k0 + wn0 + 16 * jj + lr;
                if (k >= bi) continue;
                const int64_t e = ((int64_t)g * bo + j) * bi + k;
                if (dst) dst[e] = acc[i][jj][v];
                else dW[e] = f32_to_bf16(acc[i][jj][v]);
            }
        }
    if (do_db && lr == 0) {
        float *dst_db = part ? part + (int64_t)splits * 2 * per_comp + (int64_t)split * n_out : nullptr;
        uint16_t *db = static_cast<uint16_t *>(p.db);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int j = j0 + wm0 + 16 * i + 4 * lc + v;
                const int f = g * bo + j;
                if (j >= bo || f >= n_out) continue;
                if (dst_db) dst_db[f] = dacc[i][v];
                else db[f] = f32_to_bf16(dacc[i][v]);
            }
    }
}

// dW (and db) = sum of the splits' partials, in split order.  Partials:
// [split][2 * per_comp] for dW1, dW2, then [split][n_out] for db.
__global__ void __launch_bounds__(256) general_dw_reduce(const float *part, int splits, int64_t per_comp,
                                                         int64_t n_out, uint16_t *dW1, uint16_t *dW2,
                                                         uint16_t *db) {
    const int64_t n_db = db ? n_out : 0;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < 2 * per_comp + n_db;
         e += (int64_t)gridDim.x * blockDim.x) {
        const bool is_db = e >= 2 * per_comp;
        const float *src = is_db ? part + (int64_t)splits * 2 * per_comp + (e - 2 * per_comp) : part + e;
        const int64_t stride = is_db ? n_out : 2 * per_comp;
        float s = 0.f;
        for (int q = 0; q < splits; ++q) s += src[(int64_t)q * stride];
        uint16_t *out = is_db ? db + (e - 2 * per_comp) : (e < per_comp ? dW1 + e : dW2 + (e - per_comp));
        *out = f32_to_bf16(s);
    }
}

struct GenDwPlan {
    int jt, kt, splits;
    int64_t tps;
};

bool gen_dw_plan(const DwPass &p, GenDwPlan &pl) {
    if (p.dtype != kBF16) return false;
    // 32-bit offsets within one split's token panel (checked with its rows below)
    pl.jt = (int)((p.bo + kGM - 1) / kGM);
    pl.kt = (int)((p.bi + kGN - 1) / kGN);
    const int64_t tiles = 2 * p.D * pl.jt * pl.kt;
    if (tiles >= ((int64_t)1 << 30)) return false;
    // each workgroup walks its tokens one 32-token chunk at a time with one
    // chunk in flight, so it is latency-bound: split the tokens until there
    // are ~2048 work items (8 per CU; measured best of 512-4096 at OPT-125m
    // widths, n_dyad 3, 5, 6), each at least 256 tokens deep
    int64_t splits = tiles >= 2048 ? 1 : (2048 + tiles - 1) / tiles;
    const int64_t max_splits = p.M / 256 > 0 ? p.M / 256 : 1;
    if (splits > max_splits) splits = max_splits;
    int64_t tps = (p.M + splits - 1) / splits;
    tps = (tps + kStageK - 1) / kStageK * kStageK;
    const int64_t wide = p.n_in > p.n_out ? p.n_in : p.n_out;
    // 32-bit offsets: a split's rows plus one chunk of overrun stay below 2^31 bytes
    if ((tps + kStageK) * wide * 2 >= ((int64_t)1 << 31)) {
        tps = (((int64_t)1 << 31) / (wide * 2) - kStageK) / kStageK * kStageK;
        if (tps < kStageK) return false;
    }
    pl.tps = tps > 0 ? tps : kStageK;
    pl.splits = (int)((p.M + pl.tps - 1) / pl.tps);
    if (pl.splits < 1) pl.splits = 1;
    return tiles * pl.splits < ((int64_t)1 << 31);
}

template <int GM, int GN, bool PAIRS, bool IN_T, bool W_T>
hipError_t launch_general_tile(const GemmPass &p, hipStream_t s) {
    if ((int64_t)GM * p.Kin * 2 >= ((int64_t)1 << 31)) return hipErrorNotSupported;
    const int64_t classes = p.out_t ? p.D * p.D : p.D;
    const int64_t per_class = p.out_t ? (p.bn + p.D - 1) / p.D + 1 : p.bn;
    const int64_t col_tiles = (per_class + GN - 1) / GN;
    const int64_t row_tiles = (p.M + GM - 1) / GM;
    const int64_t blocks = classes * col_tiles * row_tiles;
    if (blocks >= ((int64_t)1 << 31)) return hipErrorNotSupported;
    general_mfma_kernel<GM, GN, PAIRS, IN_T, W_T><<<(unsigned)blocks, 256, 0, s>>>(p, (int)col_tiles, (int)row_tiles);
    return hipGetLastError();
}

template <int GM, int GN>
hipError_t launch_general_gn(const GemmPass &p, hipStream_t s) {
    const bool pairs = p.Kin % 2 == 0 && p.bk % 2 == 0;
#define DYAD_GEN(PR, IT, WT) \
    if (pairs == PR && p.in_t == IT && p.w_t == WT) return launch_general_tile<GM, GN, PR, IT, WT>(p, s);
    DYAD_GEN(true, false, false) DYAD_GEN(true, false, true) DYAD_GEN(true, true, false) DYAD_GEN(true, true, true)
    DYAD_GEN(false, false, false) DYAD_GEN(false, false, true) DYAD_GEN(false, true, false) DYAD_GEN(false, true, true)
#undef DYAD_GEN
    return hipErrorNotSupported;
}

}  // namespace

hipError_t launch_general_mfma_gemm(const GemmPass &p, hipStream_t s) {
    if (p.dtype != kBF16) return hipErrorNotSupported;
    if (p.M == 0) return hipSuccess;
    // 32-bit buffer offsets: one weight tensor must fit
    if (p.D * p.bn * p.bk * 2 >= ((int64_t)1 << 31)) return hipErrorNotSupported;
    // classes narrower than 128 columns (an output transpose leaves bn / D per
    // class) take 256 x 64 tiles, which waste less of the tile
    const int64_t per_class = p.out_t ? (p.bn + p.D - 1) / p.D : p.bn;
    if (per_class <= 96) return launch_general_gn<256, 64>(p, s);
    return launch_general_gn<128, 128>(p, s);
}

bool general_dw_ok(const DwPass &p) {
    GenDwPlan pl;
    return gen_dw_plan(p, pl);
}

size_t general_dw_workspace(const DwPass &p) {
    GenDwPlan pl;
    if (!gen_dw_plan(p, pl) || pl.splits == 1) return 0;
    return (size_t)pl.splits * (size_t)(2 * p.D * p.bo * p.bi + p.n_out) * sizeof(float);
}

hipError_t launch_general_mfma_dw(const DwPass &p, hipStream_t s) {
    GenDwPlan pl;
    if (!gen_dw_plan(p, pl)) return hipErrorNotSupported;
    const int64_t per_comp = p.D * p.bo * p.bi;
    float *part = nullptr;
    if (pl.splits > 1) {
        if (!p.ws || p.ws_bytes < (size_t)pl.splits * (size_t)(2 * per_comp + p.n_out) * sizeof(float))
            return hipErrorInvalidValue;
        part = static_cast<float *>(p.ws);
    }
    // one launch per component: its operands' pair-load forms are fixed per launch
    const int64_t blocks = (int64_t)pl.splits * p.D * pl.jt * pl.kt;
    const bool z_ok = p.n_out % 2 == 0 && p.bo % 2 == 0, x_ok = p.n_in % 2 == 0 && p.bi % 2 == 0;
    hipError_t e = hipSuccess;
    for (int comp = 1; comp <= 2 && e == hipSuccess; ++comp) {
        const bool zp = z_ok && !(comp == 2 && p.out_t), xp = x_ok && !(comp == 2 && p.in_t);
        if (zp && xp) general_mfma_dw_kernel<true, true><<<(unsigned)blocks, 256, 0, s>>>(p, comp, pl.jt, pl.kt, pl.splits, pl.tps, part);
        else if (zp) general_mfma_dw_kernel<true, false><<<(unsigned)blocks, 256, 0, s>>>(p, comp, pl.jt, pl.kt, pl.splits, pl.tps, part);
        else if (xp) general_mfma_dw_kernel<false, true><<<(unsigned)blocks, 256, 0, s>>>(p, comp, pl.jt, pl.kt, pl.splits, pl.tps, part);
        else general_mfma_dw_kernel<false, false><<<(unsigned)blocks, 256, 0, s>>>(p, comp, pl.jt, pl.kt, pl.splits, pl.tps, part);
        e = hipGetLastError();
    }
    if (e != hipSuccess) return e;
    if (part) {
        int64_t grid = (2 * per_comp + p.n_out + 255) / 256;
        if (grid > 4096) grid = 4096;
        general_dw_reduce<<<(unsigned)grid, 256, 0, s>>>(part, pl.splits, per_comp, p.n_out,
                                                         static_cast<uint16_t *>(p.dW1),
                                                         static_cast<uint16_t *>(p.dW2),
                                                         static_cast<uint16_t *>(p.db));
        e = hipGetLastError();
    }
    return e;
}

}  // namespace dyad
