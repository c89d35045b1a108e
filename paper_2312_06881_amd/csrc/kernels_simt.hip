// General kernels: any n_dyad, any block sizes, widths that n_dyad does not
// divide (zero-padded), both dtypes.  The fp32 path and every shape the MFMA
// kernels do not cover use them.  Arithmetic is fp32 FMA on the vector ALUs,
// tiled through LDS.
//
// Grouped GEMM (forward and input gradient).  The output columns of a pass
// fall into classes (g1, g2): g1 = f / bn is the BlockDiag group of column f
// and g2 its BlockTrans group (f % D with an output transpose, else g1).  All
// columns of one class read the same two input slabs -- columns g1*bk + k for
// BlockDiag and c2(g2, k) for BlockTrans -- so a tile of 128 tokens x 128 columns
// of one class is a plain GEMM with K = 2*bk over a gathered A.  Within a class,
// column t is f = g1*bn + t (no output transpose) or the t-th column of group
// g1 whose residue mod D is g2.  Reads past a width (zero-padding) return zero;
// columns past Nout do not exist.
//
// Weight gradient.  dWc[g][j][k] = sum_m dZ[m][row_c(g, j)] X[m][col_c(g, k)]:
// per (component, group) a GEMM of bo x bi over K = M tokens, tiled 128 x 128;
// the BlockDiag tiles of the first column tile also sum their dZ columns for
// db.  Token sums run in a fixed order.
#include "dyad_device.h"
#include "dyad_internal.h"

namespace dyad {
namespace {

constexpr int kT = 128;   // tile edge (tokens, columns); 8 x 8 outputs per thread
constexpr int kKC = 8;    // K chunk staged in LDS

// Rows (or columns) of a thread's 8 x 8 block: two groups of four, 64 apart,
// so that each group is one float4 read from LDS.
__device__ __forceinline__ int sub_of(int t4, int i) { return (i < 4 ? 0 : 64) + 4 * t4 + (i & 3); }

// acc[i][j] += a[i] * b[j] over one staged chunk; a and b are LDS rows of kT floats.
__device__ __forceinline__ void fma_block(const float *arow, const float *brow, int ty, int tx, float (&a)[8],
                                          float (&b)[8], float (&acc)[8][8]) {
    const float4 a0 = *reinterpret_cast<const float4 *>(arow + 4 * ty);
    const float4 a1 = *reinterpret_cast<const float4 *>(arow + 64 + 4 * ty);
    const float4 b0 = *reinterpret_cast<const float4 *>(brow + 4 * tx);
    const float4 b1 = *reinterpret_cast<const float4 *>(brow + 64 + 4 * tx);
    a[0] = a0.x; a[1] = a0.y; a[2] = a0.z; a[3] = a0.w; a[4] = a1.x; a[5] = a1.y; a[6] = a1.z; a[7] = a1.w;
    b[0] = b0.x; b[1] = b0.y; b[2] = b0.z; b[3] = b0.w; b[4] = b1.x; b[5] = b1.y; b[6] = b1.z; b[7] = b1.w;
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
}

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
__global__ void __launch_bounds__(256, 2) general_gemm_kernel(GemmPass p, int64_t col_tiles, int64_t row_tiles) {
    __shared__ __attribute__((aligned(16))) float As[2][kKC][kT];
    __shared__ __attribute__((aligned(16))) float Bs[2][kKC][kT];
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

    float acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = 0.f;

    fetch(0);
    stash(0);
    __syncthreads();
    for (int64_t c = 0; c < chunks; ++c) {
        const int buf = (int)(c & 1);
        if (c + 1 < chunks) fetch((c + 1) * kKC);
#pragma unroll 2
        for (int kk = 0; kk < kKC; ++kk) {
            float a[8], bv[8];
            fma_block(As[buf][kk], Bs[buf][kk], ty, tx, a, bv, acc);
        }
        if (c + 1 < chunks) stash(buf ^ 1);
        __syncthreads();
    }

    T *out = static_cast<T *>(p.out);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t m = m0 + sub_of(ty, i);
        if (m >= p.M) continue;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int64_t t = t0 + sub_of(tx, j);
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

// dW tiles: (component, group, j tile, k tile), 128 x 128 entries each.
template <typename T>
__global__ void __launch_bounds__(256, 2) general_dw_kernel(DwPass p, int64_t jt_n, int64_t kt_n, int64_t splits,
                                                            int64_t tps, float *part) {
    __shared__ __attribute__((aligned(16))) float As[2][kKC][kT];   // dZ[m][row(j)]
    __shared__ __attribute__((aligned(16))) float Bs[2][kKC][kT];   // X[m][col(k)]
    const T *dZ = static_cast<const T *>(p.dZ);
    const T *X = static_cast<const T *>(p.X);
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int64_t b = blockIdx.x;
    const int64_t kt = b % kt_n, jt = (b / kt_n) % jt_n, gc = (b / (kt_n * jt_n)) % (2 * p.D);
    const int64_t split = b / (kt_n * jt_n * 2 * p.D);
    const int64_t m_lo = split * tps, m_hi = min(m_lo + tps, p.M);
    const int comp = gc < p.D ? 1 : 2;
    const int64_t g = gc % p.D, D = p.D;
    const int64_t j0 = jt * kT, k0 = kt * kT;
    const bool row_t = comp == 2 && p.out_t, col_t = comp == 2 && p.in_t;
    const int64_t chunks = m_hi > m_lo ? (m_hi - m_lo + kKC - 1) / kKC : 0;
    // db[g*bo + j] = sum_m dZ[m][g*bo + j] is the BlockDiag tile's own dZ column
    // sum: the first column tile's threads of column 0 add up their A values
    const bool do_db = p.db && comp == 1 && kt == 0;
    float dbs[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};

    float ra[4], rb[4];
    auto fetch = [&](int64_t c0) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = tid + 256 * q;
            const int ci = e % kT, mm = e / kT;   // entry index fastest: neighbouring columns
            const int64_t m = m_lo + c0 + mm;
            float va = 0.f, vb = 0.f;
            if (m < m_hi) {
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

    float acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = 0.f;
    if (chunks > 0) {
        fetch(0);
        stash(0);
    }
    __syncthreads();
    for (int64_t c = 0; c < chunks; ++c) {
        const int buf = (int)(c & 1);
        if (c + 1 < chunks) fetch((c + 1) * kKC);
#pragma unroll 2
        for (int mm = 0; mm < kKC; ++mm) {
            float a[8], bv[8];
            fma_block(As[buf][mm], Bs[buf][mm], ty, tx, a, bv, acc);
#pragma unroll
            for (int i = 0; i < 8; ++i) dbs[i] += a[i];
        }
        if (c + 1 < chunks) stash(buf ^ 1);
        __syncthreads();
    }

    const int64_t per_comp = p.D * p.bo * p.bi;
    if (do_db && tx == 0) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int64_t j = j0 + sub_of(ty, i), f = g * p.bo + j;
            if (j >= p.bo || f >= p.n_out) continue;
            if (part) part[splits * 2 * per_comp + split * p.n_out + f] = dbs[i];
            else store_f32(static_cast<T *>(p.db), f, dbs[i]);
        }
    }
    T *dW = static_cast<T *>(comp == 1 ? p.dW1 : p.dW2);
    float *dst = part ? part + split * 2 * per_comp + (comp - 1) * per_comp : nullptr;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t j = j0 + sub_of(ty, i);
        if (j >= p.bo) continue;
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
            const int64_t k = k0 + sub_of(tx, jj);
            if (k >= p.bi) continue;
            const int64_t e = (g * p.bo + j) * p.bi + k;
            if (dst) dst[e] = acc[i][jj];
            else store_f32(dW, e, acc[i][jj]);
        }
    }
}

// dW, dW2, db = the splits' partials added in split order (layout as in
// general_dw_kernel: [split][2 * per_comp], then [split][n_out]).
template <typename T>
__global__ void __launch_bounds__(256) general_dw_reduce_t(const float *part, int64_t splits, int64_t per_comp,
                                                           int64_t n_out, T *dW1, T *dW2, T *db) {
    const int64_t n_db = db ? n_out : 0;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < 2 * per_comp + n_db;
         e += (int64_t)gridDim.x * blockDim.x) {
        const bool is_db = e >= 2 * per_comp;
        const float *src = is_db ? part + splits * 2 * per_comp + (e - 2 * per_comp) : part + e;
        const int64_t stride = is_db ? n_out : 2 * per_comp;
        float s = 0.f;
        for (int64_t q = 0; q < splits; ++q) s += src[q * stride];
        if (is_db) store_f32(db, e - 2 * per_comp, s);
        else if (e < per_comp) store_f32(dW1, e, s);
        else store_f32(dW2, e - per_comp, s);
    }
}

// Token splits of the vector weight gradient: one workgroup walks its tokens
// a chunk at a time, so split until there are ~1024 work items, each at least
// 512 tokens deep.
int64_t simt_dw_splits(const DwPass &p, int64_t tiles, int64_t &tps) {
    int64_t splits = tiles >= 1024 ? 1 : (1024 + tiles - 1) / tiles;
    const int64_t max_splits = p.M / 512 > 0 ? p.M / 512 : 1;
    if (splits > max_splits) splits = max_splits;
    tps = (p.M + splits - 1) / splits;
    if (tps < 1) tps = 1;
    return (p.M + tps - 1) / tps > 0 ? (p.M + tps - 1) / tps : 1;
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

size_t simt_dw_workspace(const DwPass &p) {
    const int64_t jt = (p.bo + kT - 1) / kT, kt = (p.bi + kT - 1) / kT;
    int64_t tps;
    const int64_t splits = simt_dw_splits(p, 2 * p.D * jt * kt, tps);
    return splits > 1 ? (size_t)splits * (size_t)(2 * p.D * p.bo * p.bi + p.n_out) * sizeof(float) : 0;
}

hipError_t launch_simt_dw(const DwPass &p, hipStream_t s) {
    const int64_t jt = (p.bo + kT - 1) / kT, kt = (p.bi + kT - 1) / kT;
    int64_t tps;
    const int64_t splits = simt_dw_splits(p, 2 * p.D * jt * kt, tps);
    const int64_t per_comp = p.D * p.bo * p.bi;
    float *part = nullptr;
    if (splits > 1) {
        if (!p.ws || p.ws_bytes < (size_t)splits * (size_t)(2 * per_comp + p.n_out) * sizeof(float))
            return hipErrorInvalidValue;
        part = static_cast<float *>(p.ws);
    }
    const int64_t blocks = splits * 2 * p.D * jt * kt;
    if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
    if (p.dtype == kF32)
        general_dw_kernel<float><<<(unsigned)blocks, 256, 0, s>>>(p, jt, kt, splits, tps, part);
    else
        general_dw_kernel<uint16_t><<<(unsigned)blocks, 256, 0, s>>>(p, jt, kt, splits, tps, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !part) return e;
    int64_t grid = (2 * per_comp + p.n_out + 255) / 256;
    if (grid > 4096) grid = 4096;
    if (p.dtype == kF32)
        general_dw_reduce_t<float><<<(unsigned)grid, 256, 0, s>>>(
            part, splits, per_comp, p.n_out, static_cast<float *>(p.dW1), static_cast<float *>(p.dW2),
            static_cast<float *>(p.db));
    else
        general_dw_reduce_t<uint16_t><<<(unsigned)grid, 256, 0, s>>>(
            part, splits, per_comp, p.n_out, static_cast<uint16_t *>(p.dW1), static_cast<uint16_t *>(p.dW2),
            static_cast<uint16_t *>(p.db));
    return hipGetLastError();
}

}  // namespace dyad
