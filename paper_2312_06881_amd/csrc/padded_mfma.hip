// Zero-padded forms: the padding copies, the weight-gradient unpadding, and
// the grouped-GEMM entry (padded_mfma.h has the plan).
#include "padded_mfma.h"

namespace dyad {

// R token rows per workgroup (R * W about 8192 elements, so a narrow row
// does not leave most of the workgroup idle): the rows come into LDS with
// 16-byte loads (W % 8 == 0), then each thread assembles 8 consecutive
// padded columns of an output row from LDS and stores them as 16 bytes
// (bp % 8 == 0, so the 8 lie in one block).
__global__ void __launch_bounds__(256) pad_rows_kernel(const uint16_t *src, int64_t M, int W, int R, int D, int b,
                                                       int bp, uint16_t *dst1, uint16_t *dst2) {
    extern __shared__ u32x4_t row_lds[];
    const int64_t m0 = (int64_t)blockIdx.x * R;
    const int rows = M - m0 < R ? (int)(M - m0) : R;
    const int vpr = W / 8;                         // 16-byte vectors per row
    const u32x4_t *s = reinterpret_cast<const u32x4_t *>(src + m0 * W);
    for (int v = threadIdx.x; v < rows * vpr; v += 256) row_lds[v] = __builtin_nontemporal_load(s + v);
    __syncthreads();
    const int units = D * bp / 8;                  // 8-column units per output row
    const int64_t Wp = (int64_t)D * bp;
    for (int o = 0; o < 2; ++o) {
        uint16_t *dst = o == 0 ? dst1 : dst2;
        if (!dst) continue;
        for (int w = threadIdx.x; w < rows * units; w += 256) {
            const int rr = w / units, u = w - rr * units;
            const uint16_t *r = reinterpret_cast<const uint16_t *>(row_lds + rr * vpr);
            const int g = (8 * u) / bp, k0 = 8 * u - g * bp;
            uint32_t q[4];
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                uint32_t pair = 0;
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const int k = k0 + 2 * h + e;
                    const int col = o == 0 ? g * b + k : k * D + g;
                    const uint32_t v = (k < b && col < W) ? (uint32_t)r[col] : 0u;
                    pair |= v << (16 * e);
                }
                q[h] = pair;
            }
            *reinterpret_cast<uint4 *>(dst + (m0 + rr) * Wp + 8 * u) = make_uint4(q[0], q[1], q[2], q[3]);
        }
    }
}

hipError_t launch_pad_rows(const uint16_t *src, int64_t M, int64_t W, int D, int64_t b, int64_t bp,
                           uint16_t *dst1, uint16_t *dst2, hipStream_t s) {
    if (W % 8 != 0 || W > kPadMaxRow || bp % 8 != 0 || b > bp || M < 0 || (!dst1 && !dst2))
        return hipErrorNotSupported;
    if (M == 0) return hipSuccess;
    const int R = W >= 8192 ? 1 : (int)(8192 / W);   // at most 16 KB of LDS
    const int64_t blocks = (M + R - 1) / R;
    if (blocks >= ((int64_t)1 << 31)) return hipErrorNotSupported;
    pad_rows_kernel<<<(unsigned)blocks, 256, (size_t)R * W * 2, s>>>(src, M, (int)W, R, D, (int)b, (int)bp, dst1,
                                                                      dst2);
    return hipGetLastError();
}

// Zero-padded copy of D blocks of R x C (rows of C) as blocks of Rp x Cp.
__global__ void __launch_bounds__(256) pad_matrix_kernel(const uint16_t *src, int64_t D, int R, int C, int Rp,
                                                         int Cp, uint16_t *dst) {
    const int64_t units = D * Rp * (Cp / 8);
    for (int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x; u < units; u += (int64_t)gridDim.x * 256) {
        const int64_t g = u / ((int64_t)Rp * (Cp / 8));
        const int rem = (int)(u - g * Rp * (Cp / 8));
        const int r = rem / (Cp / 8), c0 = (rem % (Cp / 8)) * 8;
        uint32_t w[4];
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            uint32_t pair = 0;
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                const int c = c0 + 2 * h + e;
                const uint32_t v = (r < R && c < C) ? (uint32_t)src[(g * R + r) * C + c] : 0u;
                pair |= v << (16 * e);
            }
            w[h] = pair;
        }
        *reinterpret_cast<uint4 *>(dst + (g * Rp + r) * Cp + c0) = make_uint4(w[0], w[1], w[2], w[3]);
    }
}

hipError_t launch_pad_matrix(const uint16_t *src, int64_t D, int64_t R, int64_t C, int64_t Rp, int64_t Cp,
                             uint16_t *dst, hipStream_t s) {
    if (Cp % 8 != 0 || R > Rp || C > Cp || Rp * Cp >= ((int64_t)1 << 31)) return hipErrorNotSupported;
    const int64_t units = D * Rp * (Cp / 8);
    if (units == 0) return hipSuccess;
    int64_t grid = (units + 255) / 256;
    if (grid > 4096) grid = 4096;
    pad_matrix_kernel<<<(unsigned)grid, 256, 0, s>>>(src, D, (int)R, (int)C, (int)Rp, (int)Cp, dst);
    return hipGetLastError();
}

// Real weight (and bias) gradients from the padded ones: dW[g][j][k] from
// [g][j][k] of blocks bop x bip, db[c] from column (c / bo) * bop + c % bo.
__global__ void __launch_bounds__(256) unpad_dw_kernel(const uint16_t *p1, const uint16_t *p2, const uint16_t *pdb,
                                                       int64_t D, int bo, int bi, int bop, int bip, int64_t n_out,
                                                       uint16_t *dW1, uint16_t *dW2, uint16_t *db) {
    const int64_t per = D * bo * bi;
    const int64_t total = 2 * per + (db ? n_out : 0);
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
        if (e < 2 * per) {
            const int64_t i = e < per ? e : e - per;
            const int64_t g = i / ((int64_t)bo * bi);
            const int rem = (int)(i - g * bo * bi);
            const int j = rem / bi, k = rem % bi;
            const uint16_t v = (e < per ? p1 : p2)[(g * bop + j) * bip + k];
            (e < per ? dW1 : dW2)[i] = v;
        } else {
            const int64_t c = e - 2 * per;
            db[c] = pdb[(c / bo) * bop + c % bo];
        }
    }
}

hipError_t launch_unpad_dw(const uint16_t *p1, const uint16_t *p2, const uint16_t *pdb, int64_t D, int64_t bo,
                           int64_t bi, int64_t bop, int64_t bip, int64_t n_out, uint16_t *dW1, uint16_t *dW2,
                           uint16_t *db, hipStream_t s) {
    const int64_t total = 2 * D * bo * bi + (db ? n_out : 0);
    if (total == 0) return hipSuccess;
    int64_t grid = (total + 255) / 256;
    if (grid > 4096) grid = 4096;
    unpad_dw_kernel<<<(unsigned)grid, 256, 0, s>>>(p1, p2, pdb, D, (int)bo, (int)bi, (int)bop, (int)bip, n_out,
                                                   dW1, dW2, db);
    return hipGetLastError();
}

hipError_t launch_padded_gemm(const GemmPass &p, hipStream_t s) {
    if (p.dtype != kBF16 || p.gelu_in || p.M < kPadMinTokens) return hipErrorNotSupported;
    if (p.Kin % 8 != 0 || p.Kin > kPadMaxRow) return hipErrorNotSupported;
    return p.w_t ? launch_padded_dx(p, s) : launch_padded_fwd(p, s);
}

}  // namespace dyad
