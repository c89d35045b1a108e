// SIMT kernels: one thread per output element, fp32 accumulation in natural
// k order.  They accept any shape (any n_dyad, any block sizes, widths that
// n_dyad does not divide) and both dtypes; the fp32 path and every shape the
// MFMA kernels do not cover use them.
#include "dyad_device.h"
#include "dyad_internal.h"

namespace dyad {
namespace {

// out[m][f] of one grouped-GEMM pass (index maps in dyad_internal.h).
template <typename T>
__global__ void __launch_bounds__(256) simt_gemm_kernel(GemmPass p) {
    const T *in = static_cast<const T *>(p.in);
    const T *W1 = static_cast<const T *>(p.W1);
    const T *W2 = static_cast<const T *>(p.W2);
    const int64_t total = p.M * p.Nout;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t m = e / p.Nout, f = e % p.Nout;
        const T *x = in + m * p.Kin;
        // comp 1: block-diagonal, i = f / bn, j = f % bn; input columns past Kin
        // are zero-padding and are skipped
        int64_t i = f / p.bn, j = f % p.bn;
        float acc = 0.f;
        const int64_t k1 = min(p.bk, p.Kin - i * p.bk);
        for (int64_t k = 0; k < k1; ++k) {
            int64_t w = p.w_t ? (i * p.bk + k) * p.bn + j : (i * p.bn + j) * p.bk + k;
            acc += load_f32(W1, w) * load_f32(x, i * p.bk + k);
        }
        // comp 2: output column f came from (i, j) by the inverse of its output map
        if (p.out_t) { i = f % p.D; j = f / p.D; }
        const int64_t k2 = min(p.bk, p.in_t ? (p.Kin - i + p.D - 1) / p.D : p.Kin - i * p.bk);
        for (int64_t k = 0; k < k2; ++k) {
            int64_t w = p.w_t ? (i * p.bk + k) * p.bn + j : (i * p.bn + j) * p.bk + k;
            int64_t c = p.in_t ? k * p.D + i : i * p.bk + k;
            acc += load_f32(W2, w) * load_f32(x, c);
        }
        if (p.epilogue == kEpiGeluGrad) {
            acc *= gelu_grad_f32(load_f32(static_cast<const T *>(p.h_in), e));
        } else {
            if (p.bias) acc += load_f32(static_cast<const T *>(p.bias), f);
            if (p.epilogue == kEpiBiasGelu) {
                if (p.h_out) store_f32(static_cast<T *>(p.h_out), e, acc);
                acc = gelu_f32(acc);
            }
        }
        store_f32(static_cast<T *>(p.out), e, acc);
    }
}

// dW1, dW2: one thread per stored entry, sum over tokens in order.
template <typename T>
__global__ void __launch_bounds__(256) simt_dw_kernel(DwPass p) {
    const T *dZ = static_cast<const T *>(p.dZ);
    const T *X = static_cast<const T *>(p.X);
    const int64_t per = p.D * p.bo * p.bi;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < 2 * per;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int comp = e < per ? 1 : 2;
        const int64_t r = e % per, i = r / (p.bo * p.bi), j = (r / p.bi) % p.bo, k = r % p.bi;
        const int64_t row = (comp == 1 || !p.out_t) ? i * p.bo + j : j * p.D + i;
        const int64_t col = (comp == 1 || !p.in_t) ? i * p.bi + k : k * p.D + i;
        // an entry in a zero-padded row or column gets a zero gradient
        const int64_t M = (row < p.n_out && col < p.n_in) ? p.M : 0;
        float acc = 0.f;
        for (int64_t m = 0; m < M; ++m) acc += load_f32(dZ, m * p.n_out + row) * load_f32(X, m * p.n_in + col);
        store_f32(static_cast<T *>(comp == 1 ? p.dW1 : p.dW2), r, acc);
    }
}

template <typename T>
__global__ void __launch_bounds__(256) simt_db_kernel(DwPass p) {
    const T *dZ = static_cast<const T *>(p.dZ);
    for (int64_t f = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; f < p.n_out;
         f += (int64_t)gridDim.x * blockDim.x) {
        float acc = 0.f;
        for (int64_t m = 0; m < p.M; ++m) acc += load_f32(dZ, m * p.n_out + f);
        store_f32(static_cast<T *>(p.db), f, acc);
    }
}

unsigned grid_for(int64_t n) {
    int64_t g = (n + 255) / 256;
    if (g < 1) g = 1;
    if (g > 65536) g = 65536;
    return (unsigned)g;
}

}  // namespace

hipError_t launch_simt_gemm(const GemmPass &p, hipStream_t s) {
    if (p.M == 0) return hipSuccess;
    unsigned g = grid_for(p.M * p.Nout);
    if (p.dtype == kF32)
        simt_gemm_kernel<float><<<g, 256, 0, s>>>(p);
    else
        simt_gemm_kernel<uint16_t><<<g, 256, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_simt_dw(const DwPass &p, hipStream_t s) {
    unsigned g = grid_for(2 * p.D * p.bo * p.bi);
    if (p.dtype == kF32)
        simt_dw_kernel<float><<<g, 256, 0, s>>>(p);
    else
        simt_dw_kernel<uint16_t><<<g, 256, 0, s>>>(p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !p.db) return e;
    g = grid_for(p.n_out);
    if (p.dtype == kF32)
        simt_db_kernel<float><<<g, 256, 0, s>>>(p);
    else
        simt_db_kernel<uint16_t><<<g, 256, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace dyad
