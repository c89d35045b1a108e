// Internal interface between the C-ABI layer (dyad_abi.hip) and the kernel
// translation units.  Not installed; the public interface is include/dyad.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dyad {

enum Dtype { kF32 = 0, kBF16 = 1 };

// Epilogue applied to the fp32 accumulator of a grouped-GEMM pass.
enum Epilogue {
    kEpiBias = 0,      // out = acc + bias (bias may be null)
    kEpiBiasGelu = 1,  // pre = acc + bias; h_out = pre (if non-null); out = GELU(pre)
    kEpiGeluGrad = 2,  // out = acc * GELU'(h_in)
};

// One pass of the Dyad grouped GEMM, written for both the forward pass and the
// input gradient.  With D groups, per-group input width bk = ceil(Kin/D) and
// output width bn = ceil(Nout/D), for every token m and output feature f < Nout:
//   out[m][f] = sum over the stored entries (c, i, j, k) whose output column is f
//               and whose input column is < Kin
//               of Wc(i, j, k) * in[m][input column of (c, i, k)]
// (widths that D does not divide are zero-padded: the missing input columns
// read as zero and the output columns past Nout are never written).
// where
//   output column: comp 1 -> i*bn + j;  comp 2 -> out_t ? j*D + i : i*bn + j
//   input column:  comp 1 -> i*bk + k;  comp 2 -> in_t  ? k*D + i : i*bk + k
//   Wc(i, j, k) = w_t ? Wc[i][k][j] (stored [D][bk][bn]) : Wc[i][j][k] (stored [D][bn][bk]).
// Forward: in = X, out = Y, Kin = n_in, Nout = n_out, in_t = IT|DT, out_t = OT|DT, w_t = 0.
// Input gradient: in = dZ, out = dX, Kin = n_out, Nout = n_in, in_t = OT|DT,
// out_t = IT|DT, w_t = 1 (dX = W^T dZ reads every block transposed).
struct GemmPass {
    int64_t M, Kin, Nout, D, bk, bn;
    bool in_t, out_t, w_t;
    bool gelu_in;    // forward only: the input operand is GELU(in), formed as it is staged
    int dtype;       // Dtype
    int epilogue;    // Epilogue
    const void *in, *W1, *W2, *bias, *h_in;
    void *out, *h_out;
};

// Weight/bias gradient of one layer (forward-variant flags in_t/out_t):
//   dWc[i][j][k] = sum_m dZ[m][row_c(i, j)] * X[m][col_c(i, k)],  db[f] = sum_m dZ[m][f]
// row_c = comp 1 or !out_t ? i*bo + j : j*D + i;  col_c = comp 1 or !in_t ? i*bi + k : k*D + i.
// bi = ceil(n_in/D), bo = ceil(n_out/D); an entry with row_c >= n_out or
// col_c >= n_in touches only zero-padding and gets a zero gradient.
struct DwPass {
    int64_t M, n_in, n_out, D, bi, bo;
    bool in_t, out_t;
    int dtype;
    const void *dZ, *X;
    bool gelu_x;     // X is GELU(X as passed), formed as it is staged
    void *dW1, *dW2, *db;
    void *ws;
    size_t ws_bytes;
    // component 2's operands when they differ from dZ / X (block-ordered copies
    // of them, read with in_t / out_t false); null: dZ / X
    const void *dZ2, *X2;
};

// General kernels: any shape, any D, both dtypes (vector ALU, tiled).  The
// weight gradient splits the tokens through the workspace when the tiles alone
// would leave the GPU idle: simt_dw_workspace() bytes (0 for one split).
hipError_t launch_simt_gemm(const GemmPass &p, hipStream_t s);
size_t simt_dw_workspace(const DwPass &p);
hipError_t launch_simt_dw(const DwPass &p, hipStream_t s);

// General weight gradient on the matrix cores (bf16, any shape), token splits
// summed in order through the workspace: general_dw_workspace() bytes (0 when
// one split suffices or the path does not apply).
bool general_dw_ok(const DwPass &p);
size_t general_dw_workspace(const DwPass &p);
hipError_t launch_general_mfma_dw(const DwPass &p, hipStream_t s);

// General grouped GEMM on the matrix cores (bf16, any shape): operands
// gathered element by element.  hipErrorNotSupported for fp32 or offsets past
// 32 bits.
hipError_t launch_general_mfma_gemm(const GemmPass &p, hipStream_t s);

// Small-batch grouped GEMM (bf16, up to 32 tokens -- 256 for output-transposed
// input gradients at n_dyad 16 --, widths that n_dyad divides into blocks of a
// multiple of 128 columns): the reduction split over workgroups, fp32 partial
// sums in the stream's split workspace, added in a fixed order.
// hipErrorNotSupported (launching nothing) when skinny_ok() is false.
bool skinny_ok(const GemmPass &p);
hipError_t launch_skinny_gemm(const GemmPass &p, hipStream_t s);

// Split reductions of the grouped GEMM: a workspace of at least `bytes` for
// stream s (one per device and stream, kept between calls and regrown in
// stream order), and the kernel that adds `slices` fp32 partial sums
// [slices][M][Nout] in slice order and applies the pass's epilogue (with
// perm_last, the last slice holds block-order sums: output column j*D + g at
// column g*bn + j).
hipError_t split_workspace(hipStream_t s, size_t bytes, void **out);

// dyad_forward_noalloc: while a ScratchScope lives on the calling thread,
// split_workspace hands out its fixed buffer instead of the stream's pool
// buffer, and refuses any request larger than it (the pass then takes a
// plan that needs no buffer); it never allocates.
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;
struct ScratchScope {
    void *ptr;
    size_t bytes;
    const ScratchScope *prev;
    ScratchScope(void *p, size_t b);
    ~ScratchScope();
    ScratchScope(const ScratchScope &) = delete;
    ScratchScope &operator=(const ScratchScope &) = delete;
};
const ScratchScope *current_scratch();
// Device address of the fixed scratch array on the current device (looked up
// once per device with hipGetSymbolAddress).
hipError_t noalloc_scratch(void **out);
hipError_t launch_split_reduce(const GemmPass &p, const float *part, int slices, hipStream_t s,
                               bool perm_last = false, int perm_from = 1 << 30);

// out[n][g*bk + k] = in[n][k*D + g] for M token rows of D*bk bf16 values
// (bk a multiple of 32, D a divisor of 64, 16-byte aligned rows).
hipError_t launch_deinterleave(const uint16_t *in, uint16_t *out, int64_t M, int64_t bk, int D, hipStream_t s);

// Whether a bf16 pass at n_dyad 8 / 16 with a transpose (exact widths) takes the
// large-batch form that de-interleaves its input and runs the components as
// plain per-block GEMMs.  Measured on gfx950 against the fused tiles at 256 to
// 16384 tokens: at n_dyad 16 it wins from 2048 tokens with reduction blocks of
// 128 under an output transpose and 256 without, for the input gradient under
// an output transpose from blocks of 64 once the batch reaches 8192, and from
// 256 tokens with blocks of 512 (1.6-6.6x on the wide layer 8192 -> 32768 at
// 1024 tokens); at n_dyad 8 from 2048 tokens with blocks of 512.
inline bool permuted_pays(int D, bool out_t, bool w_t, int64_t M, int64_t bk) {
    if (D >= 16 && M >= 256 && bk >= 512) return true;
    if (M < 2048) return false;
    if (D >= 16) return bk >= (out_t ? 128 : 256) || (w_t && out_t && M >= 8192 && bk >= 64);
    return bk >= 512;
}

// Zero-padded forms (padded_mfma.h): block-ordered copies padded to whole
// tiles, for shapes the fused tiles refuse, from kPadMinTokens tokens.
constexpr int64_t kPadMinTokens = 512;     // below this the general kernels run
constexpr int64_t kPadMaxRow = 16384;      // widest row the padding copy stages in LDS
constexpr int64_t pad_up(int64_t v, int64_t q) { return (v + q - 1) / q * q; }
// dst1[m][g*bp + k] = src[m][g*b + k] and dst2[m][g*bp + k] = src[m][k*D + g]
// for k < b and a source column below W, else 0 (either output may be null).
hipError_t launch_pad_rows(const uint16_t *src, int64_t M, int64_t W, int D, int64_t b, int64_t bp,
                           uint16_t *dst1, uint16_t *dst2, hipStream_t s);
// dst[g][r][c] = src[g][r][c] for r < R and c < C, else 0 (dst is D x Rp x Cp).
hipError_t launch_pad_matrix(const uint16_t *src, int64_t D, int64_t R, int64_t C, int64_t Rp, int64_t Cp,
                             uint16_t *dst, hipStream_t s);
// dW1 / dW2 [D][bo][bi] and db [n_out] (nullable) from their padded forms
// [D][bop][bip] and [D * bop].
hipError_t launch_unpad_dw(const uint16_t *p1, const uint16_t *p2, const uint16_t *pdb, int64_t D, int64_t bo,
                           int64_t bi, int64_t bop, int64_t bip, int64_t n_out, uint16_t *dW1, uint16_t *dW2,
                           uint16_t *db, hipStream_t s);
// Forward / input gradient on the padded forms; hipErrorNotSupported, launching
// nothing, for fp32, an input activation, fewer than kPadMinTokens tokens, an
// input width that is not a multiple of 8 or above kPadMaxRow, or no workspace.
hipError_t launch_padded_gemm(const GemmPass &p, hipStream_t s);
hipError_t launch_padded_fwd(const GemmPass &p, hipStream_t s);
hipError_t launch_padded_dx(const GemmPass &p, hipStream_t s);

// MFMA grouped GEMM (bf16): returns hipErrorNotSupported, launching nothing,
// when the pass's shape has no matching tile configuration (zero-padded
// widths included).
hipError_t launch_mfma_gemm(const GemmPass &p, hipStream_t s);

// MFMA weight gradient (bf16): split over tokens, fixed-order reduction of the
// splits through the workspace (mfma_dw_workspace() bytes; 0 when one split
// covers the tokens and the tiles store the results directly).  When
// mfma_dw_ok() is false, launch_mfma_dw() returns hipErrorNotSupported.
bool mfma_dw_ok(const DwPass &p);
size_t mfma_dw_workspace(const DwPass &p);
hipError_t launch_mfma_dw(const DwPass &p, hipStream_t s);

}  // namespace dyad
