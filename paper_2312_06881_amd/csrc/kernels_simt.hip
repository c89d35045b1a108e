// General kernels: any n_dyad, any block sizes, widths that n_dyad does not
// divide (zero-padded), both dtypes.  The fp32 path and every shape the MFMA
// kernels do not cover use them.  Arithmetic is fp32 FMA on the vector ALUs,
// tiled through LDS.
//
// Grouped GEMM (forward and input gradient).  The output columns of a pass
// fall into classes (g1, g2): g1 = f / bn is the BlockDiag group of column f
// and g2 its BlockTrans group (f % D with an output transpose, else g1).  All
// columns of one class read the same two input slabs -- columns g1*bk + k for
// BlockDiag and c2(g2, k) for BlockTrans -- so a tile of 64 tokens x 64 columns
// of one class is a plain GEMM with K = 2*bk over a gathered A.  Within a class,
// column t is f = g1*bn + t (no output transpose) or the t-th column of group
// g1 whose residue mod D is g2.  Reads past a width (zero-padding) return zero;
// columns past Nout do not exist.
//
// Weight gradient.  dWc[g][j][k] = sum_m dZ[m][row_c(g, j)] X[m][col_c(g, k)]:
// per (component, group) a GEMM of bo x bi over K = M tokens, tiled 64 x 64;
// the BlockDiag tiles of the first column tile also sum their dZ columns for
// db.  Token sums run in a fixed order.
#include "dyad_device.h"
#include "dyad_internal.h"

namespace dyad {
namespace {

constexpr int kT = 64;    // tile edge (tokens, columns)
constexpr int kKC = 16;   // K chunk staged in LDS

// One class of output columns of a grouped-GEMM pass.
struct ColClass {
    int64_t g1, g2, first, step, count;
    __device__ int64_t col(int64_t t) const { return first + t * step; }
};

__device__ __forceinline__ ColClass col_class(const GemmPass &p, int64_t cls) {
    ColClass c;
    const int64_t D = p.D;
    if (!p.out_t) {
        c.g1 = cls; c.g2 = cls;
        c.first = cls * p.bn; c.step = 1;
        const int64_t end = min((cls + 1) * p.bn, p.Nout);
        c.count = end > c.first ? end - c.first : 0;
    } else {
        c.g1 = cls / D; c.g2 = cls % D;
        const int64_t lo = c.g1 * p.bn, hi = min((c.g1 + 1) * p.bn, p.Nout);
        c.first = lo + ((c.g2 - lo % D) % D + D) % D;     // first f >= lo with f % D == g2
        c.step = D;
        c.count = hi > c.first ? (hi - c.first + D - 1) / D : 0;
    }
    return c;
}

template <typename T>
__global__ void __launch_bounds__(256) general_gemm_kernel(GemmPass p, int64_t col_tiles, int64_t row_tiles) {
    __shared__ float As[2][kKC][kT];
    __shared__ float Bs[2][kKC][kT];
    const T *in = static_cast<const T *>(p.in);
    const T *W1 = static_cast<const T *>(p.W1);
    const T *W2 = static_cast<const T *>(p.W2);
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;

    const int64_t b = blockIdx.x;
    const int64_t rt = b % row_tiles, ct = (b / row_tiles) % col_tiles, cls = b / (row_tiles * col_tiles);
    const ColClass cc = col_class(p, cls);
    const int64_t t0 = ct * kT, m0 = rt * kT;
    if (t0 >= cc.count) return;                        // uniform: the whole block leaves
    const int64_t bk = p.bk, bn = p.bn, D = p.D;
    const int64_t nk = 2 * bk;                          // BlockDiag k, then BlockTrans k
    const int64_t chunks = (nk + kKC - 1) / kKC;

    // Staging: 4 A and 4 B elements per thread per chunk.  Everything but the
    // chunk's k is fixed per thread, so it is worked out once here.
    int64_t a_row[4];            // m * Kin, or -1 past the batch
    int a_kk[4], b_kk[4];
    int64_t b_base1[4], b_base2[4];   // weight offsets at k = 0, or -1 past the class
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = tid + 256 * q;
        a_kk[q] = e % kKC;
        const int64_t m = m0 + e / kKC;
        a_row[q] = m < p.M ? m * p.Kin : -1;
        int ci;
        if (p.w_t) { ci = e % kT; b_kk[q] = e / kT; } else { b_kk[q] = e % kKC; ci = e / kKC; }
        const int64_t t = t0 + ci;
        b_base1[q] = b_base2[q] = -1;
        if (t < cc.count) {
            const int64_t f = cc.col(t);
            const int64_t j1 = f - cc.g1 * bn, j2 = p.out_t ? f / D : j1;
            b_base1[q] = p.w_t ? cc.g1 * bk * bn + j1 : (cc.g1 * bn + j1) * bk;
            b_base2[q] = p.w_t ? cc.g2 * bk * bn + j2 : (cc.g2 * bn + j2) * bk;
        }
    }
    const int64_t a_col1 = cc.g1 * bk;                     // BlockDiag input column at k = 0
    float ra[4], rb[4];
    auto fetch = [&](int64_t c0) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int64_t kq = c0 + a_kk[q];
            float v = 0.f;
            if (kq < nk && a_row[q] >= 0) {
                int64_t col;
                if (kq < bk) col = a_col1 + kq;
                else col = p.in_t ? (kq - bk) * D + cc.g2 : cc.g2 * bk + (kq - bk);
                if (col < p.Kin) v = load_f32(in, a_row[q] + col);
            }
            ra[q] = v;
            const int64_t kb = c0 + b_kk[q];
            float w = 0.f;
            if (kb < nk && b_base1[q] >= 0) {
                const bool c2 = kb >= bk;
                const int64_t k = c2 ? kb - bk : kb;
                const int64_t off = (c2 ? b_base2[q] : b_base1[q]) + (p.w_t ? k * bn : k);
                w = load_f32(c2 ? W2 : W1, off);
            }
            rb[q] = w;
        }
    };
    auto stash = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = tid + 256 * q;
            As[buf][e % kKC][e / kKC] = ra[q];
            if (p.w_t) Bs[buf][e / kT][e % kT] = rb[q];
            else Bs[buf][e % kKC][e / kKC] = rb[q];
        }
    };

    float acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

    fetch(0);
    stash(0);
    __syncthreads();
    for (int64_t c = 0; c < chunks; ++c) {
        const int buf = (int)(c & 1);
        if (c + 1 < chunks) fetch((c + 1) * kKC);
#pragma unroll
        for (int kk = 0; kk < kKC; ++kk) {
            float a[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[buf][kk][ty + 16 * i];
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[j] = Bs[buf][kk][tx + 16 * j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], bv[j], acc[i][j]);
        }
        if (c + 1 < chunks) stash(buf ^ 1);
        __syncthreads();
    }

    T *out = static_cast<T *>(p.out);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t m = m0 + ty + 16 * i;
        if (m >= p.M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t t = t0 + tx + 16 * j;
            if (t >= cc.count) continue;
            const int64_t f = cc.col(t);
            const int64_t e = m * p.Nout + f;
            float v = acc[i][j];
            if (p.epilogue == kEpiGeluGrad) {
                v *= gelu_grad_f32(load_f32(static_cast<const T *>(p.h_in), e));
            } else {
                if (p.bias) v += load_f32(static_cast<const T *>(p.bias), f);
                if (p.epilogue == kEpiBiasGelu) {
                    if (p.h_out) store_f32(static_cast<T *>(p.h_out), e, v);
                    v = gelu_f32(v);
                }
            }
            store_f32(out, e, v);
        }
    }
}

// dW tiles: (component, group, j tile, k tile), 64 x 64 entries each.
template <typename T>
__global__ void __launch_bounds__(256) general_dw_kernel(DwPass p, int64_t jt_n, int64_t kt_n) {
    __shared__ float As[2][kKC][kT];   // dZ[m][row(j)]
    __shared__ float Bs[2][kKC][kT];   // X[m][col(k)]
    const T *dZ = static_cast<const T *>(p.dZ);
    const T *X = static_cast<const T *>(p.X);
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int64_t b = blockIdx.x;
    const int64_t kt = b % kt_n, jt = (b / kt_n) % jt_n, gc = b / (kt_n * jt_n);
    const int comp = gc < p.D ? 1 : 2;
    const int64_t g = gc % p.D, D = p.D;
    const int64_t j0 = jt * kT, k0 = kt * kT;
    const bool row_t = comp == 2 && p.out_t, col_t = comp == 2 && p.in_t;
    const int64_t chunks = (p.M + kKC - 1) / kKC;
    // db[g*bo + j] = sum_m dZ[m][g*bo + j] is the BlockDiag tile's own dZ column
    // sum: the first column tile's threads of column 0 add up their A values
    const bool do_db = p.db && comp == 1 && kt == 0;
    float dbs[4] = {0.f, 0.f, 0.f, 0.f};

    float ra[4], rb[4];
    auto fetch = [&](int64_t c0) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = tid + 256 * q;
            const int ci = e % kT, mm = e / kT;   // entry index fastest: neighbouring columns
            const int64_t m = c0 + mm;
            float va = 0.f, vb = 0.f;
            if (m < p.M) {
                const int64_t j = j0 + ci, k = k0 + ci;
                const int64_t row = row_t ? j * D + g : g * p.bo + j;
                const int64_t col = col_t ? k * D + g : g * p.bi + k;
                if (j < p.bo && row < p.n_out) va = load_f32(dZ, m * p.n_out + row);
                if (k < p.bi && col < p.n_in) vb = load_f32(X, m * p.n_in + col);
            }
            ra[q] = va;
            rb[q] = vb;
        }
    };
    auto stash = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = tid + 256 * q;
            As[buf][e / kT][e % kT] = ra[q];
            Bs[buf][e / kT][e % kT] = rb[q];
        }
    };

    float acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
    if (chunks > 0) {
        fetch(0);
        stash(0);
    }
    __syncthreads();
    for (int64_t c = 0; c < chunks; ++c) {
        const int buf = (int)(c & 1);
        if (c + 1 < chunks) fetch((c + 1) * kKC);
#pragma unroll
        for (int mm = 0; mm < kKC; ++mm) {
            float a[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[buf][mm][ty + 16 * i];
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[j] = Bs[buf][mm][tx + 16 * j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], bv[j], acc[i][j]);
#pragma unroll
            for (int i = 0; i < 4; ++i) dbs[i] += a[i];
        }
        if (c + 1 < chunks) stash(buf ^ 1);
        __syncthreads();
    }

    if (do_db && tx == 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t j = j0 + ty + 16 * i, f = g * p.bo + j;
            if (j < p.bo && f < p.n_out) store_f32(static_cast<T *>(p.db), f, dbs[i]);
        }
    }
    T *dW = static_cast<T *>(comp == 1 ? p.dW1 : p.dW2);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t j = j0 + ty + 16 * i;
        if (j >= p.bo) continue;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int64_t k = k0 + tx + 16 * jj;
            if (k >= p.bi) continue;
            store_f32(dW, (g * p.bo + j) * p.bi + k, acc[i][jj]);
        }
    }
}

}  // namespace

hipError_t launch_simt_gemm(const GemmPass &p, hipStream_t s) {
    if (p.M == 0) return hipSuccess;
    const int64_t classes = p.out_t ? p.D * p.D : p.D;
    const int64_t per_class = p.out_t ? (p.bn + p.D - 1) / p.D + 1 : p.bn;
    const int64_t col_tiles = (per_class + kT - 1) / kT;
    const int64_t row_tiles = (p.M + kT - 1) / kT;
    const int64_t blocks = classes * col_tiles * row_tiles;
    if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    if (p.dtype == kF32)
        general_gemm_kernel<float><<<(unsigned)blocks, 256, 0, s>>>(p, col_tiles, row_tiles);
    else
        general_gemm_kernel<uint16_t><<<(unsigned)blocks, 256, 0, s>>>(p, col_tiles, row_tiles);
    return hipGetLastError();
}

hipError_t launch_simt_dw(const DwPass &p, hipStream_t s) {
    const int64_t jt = (p.bo + kT - 1) / kT, kt = (p.bi + kT - 1) / kT;
    const int64_t blocks = 2 * p.D * jt * kt;
    if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    if (p.dtype == kF32)
        general_dw_kernel<float><<<(unsigned)blocks, 256, 0, s>>>(p, jt, kt);
    else
        general_dw_kernel<uint16_t><<<(unsigned)blocks, 256, 0, s>>>(p, jt, kt);
    return hipGetLastError();
}

}  // namespace dyad
