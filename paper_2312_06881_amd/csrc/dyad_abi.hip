// The C-ABI of libdyad (include/dyad.h): argument checks, the choice of kernel
// for each pass, and launches on the caller's stream.  Every check runs before
// the first HIP call.
#include "dyad.h"

#include <string.h>

#include "dyad_internal.h"

namespace {

using dyad::DwPass;
using dyad::GemmPass;

constexpr int64_t kMaxDim = (int64_t)1 << 31;   // any single width or token count
constexpr int64_t kMaxElems = (int64_t)1 << 40; // any single tensor, in elements

// Per-block size; a width that D does not divide is zero-padded up to D blocks.
int64_t block(int64_t n, int64_t D) { return (n + D - 1) / D; }

// The int a caller passed for an enum parameter.  A C caller may pass any
// int there; reading the parameter through its enum type would be undefined
// in C++ for values outside the enumerators' range, so its bytes are read as
// an int and every check works on that.
template <class E>
int enum_value(const E &e) {
    static_assert(sizeof(E) == sizeof(int), "C enums are int-sized");
    int v;
    memcpy(&v, &e, sizeof v);
    return v;
}

bool aligned16(const void *p) { return p == nullptr || ((uintptr_t)p & 15u) == 0; }

int check_sizes(int variant, int64_t n_in, int64_t n_out, int64_t D, int64_t M, int dtype) {
    if (variant != DYAD_IT && variant != DYAD_OT && variant != DYAD_DT) return DYAD_ERR_INVALID_ARG;
    if (dtype != DYAD_F32 && dtype != DYAD_BF16) return DYAD_ERR_DTYPE;
    if (n_in <= 0 || n_out <= 0 || D <= 0 || M < 0) return DYAD_ERR_INVALID_ARG;
    if (n_in >= kMaxDim || n_out >= kMaxDim || M >= kMaxDim) return DYAD_ERR_INVALID_ARG;
    if (M * n_in >= kMaxElems || M * n_out >= kMaxElems) return DYAD_ERR_INVALID_ARG;
    if (D >= kMaxDim || D * block(n_in, D) * block(n_out, D) >= kMaxElems) return DYAD_ERR_INVALID_ARG;
    return DYAD_OK;
}

bool in_transposed(int v) { return v == DYAD_IT || v == DYAD_DT; }
bool out_transposed(int v) { return v == DYAD_OT || v == DYAD_DT; }

int launch_status(hipError_t e) { return e == hipSuccess ? DYAD_OK : DYAD_ERR_LAUNCH; }

int run_gemm(const GemmPass &p, hipStream_t s) {
    hipError_t e = dyad::skinny_ok(p) ? dyad::launch_skinny_gemm(p, s) : hipErrorNotSupported;
    if (e == hipErrorNotSupported) e = dyad::launch_mfma_gemm(p, s);
    if (e == hipErrorNotSupported) e = dyad::launch_padded_gemm(p, s);
    if (e == hipErrorNotSupported) e = dyad::launch_general_mfma_gemm(p, s);
    if (e == hipErrorNotSupported) e = dyad::launch_simt_gemm(p, s);
    return launch_status(e);
}

// Workspace of the weight-gradient path the call will take: the MFMA kernels
// for shapes they cover, else the general matrix-core kernel (bf16), else the
// general vector kernel.
size_t dw_workspace(const DwPass &p) {
    if (dyad::mfma_dw_ok(p)) return dyad::mfma_dw_workspace(p);
    if (dyad::general_dw_ok(p)) return dyad::general_dw_workspace(p);
    return dyad::simt_dw_workspace(p);
}

}  // namespace

// dyad_forward and dyad_forward_noalloc: the same checks and plan; the
// latter runs with the fixed scratch array in place of the stream's buffer.
static int forward_impl(int variant, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M, int dtype,
                        const void *X, const void *W1, const void *W2, const void *bias, int act, void *Y,
                        void *H, hipStream_t stream, bool noalloc, int act_in = DYAD_ACT_NONE) {
    int rc = check_sizes(variant, n_in, n_out, n_dyad, M, dtype);
    if (rc) return rc;
    if (act != DYAD_ACT_NONE && act != DYAD_ACT_GELU) return DYAD_ERR_INVALID_ARG;
    if (act_in != DYAD_ACT_NONE && act_in != DYAD_ACT_GELU) return DYAD_ERR_INVALID_ARG;
    if (act_in == DYAD_ACT_GELU && dtype != DYAD_BF16) return DYAD_ERR_DTYPE;
    if (!W1 || !W2 || (M > 0 && (!X || !Y))) return DYAD_ERR_INVALID_ARG;
    if (act == DYAD_ACT_NONE) H = nullptr;
    if (!aligned16(X) || !aligned16(W1) || !aligned16(W2) || !aligned16(bias) || !aligned16(Y) ||
        !aligned16(H))
        return DYAD_ERR_ALIGN;
    if (M == 0) return DYAD_OK;
    GemmPass p{};
    p.M = M; p.Kin = n_in; p.Nout = n_out; p.D = n_dyad; p.bk = block(n_in, n_dyad); p.bn = block(n_out, n_dyad);
    p.in_t = in_transposed(variant); p.out_t = out_transposed(variant); p.w_t = false;
    p.dtype = dtype;
    p.epilogue = act == DYAD_ACT_GELU ? dyad::kEpiBiasGelu : dyad::kEpiBias;
    p.in = X; p.W1 = W1; p.W2 = W2; p.bias = bias; p.h_in = nullptr; p.out = Y; p.h_out = H;
    if (act_in == DYAD_ACT_GELU) {
        // only the matrix-core tiles apply an input activation; other shapes are refused
        p.gelu_in = true;
        const hipError_t e = dyad::launch_mfma_gemm(p, stream);
        return e == hipErrorNotSupported ? DYAD_ERR_SHAPE : launch_status(e);
    }
    if (!noalloc) return run_gemm(p, stream);
    void *scr = nullptr;
    if (dyad::noalloc_scratch(&scr) != hipSuccess) {
        (void)hipGetLastError();
        return DYAD_ERR_LAUNCH;
    }
    const dyad::ScratchScope scope(scr, dyad::kNoAllocScratchBytes);
    return run_gemm(p, stream);
}

extern "C" {

int dyad_forward(dyad_variant variant_arg, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M,
                 dyad_dtype dtype_arg, const void *X, const void *W1, const void *W2, const void *bias,
                 dyad_act act_arg, void *Y, void *H, hipStream_t stream) {
    return forward_impl(enum_value(variant_arg), n_in, n_out, n_dyad, M, enum_value(dtype_arg), X, W1, W2, bias,
                        enum_value(act_arg), Y, H, stream, false);
}

int dyad_forward_ex(dyad_variant variant_arg, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M,
                    dyad_dtype dtype_arg, dyad_act act_in_arg, const void *X, const void *W1, const void *W2,
                    const void *bias, dyad_act act_arg, void *Y, void *H, hipStream_t stream) {
    return forward_impl(enum_value(variant_arg), n_in, n_out, n_dyad, M, enum_value(dtype_arg), X, W1, W2, bias,
                        enum_value(act_arg), Y, H, stream, false, enum_value(act_in_arg));
}

int dyad_forward_noalloc(dyad_variant variant_arg, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M,
                         dyad_dtype dtype_arg, const void *X, const void *W1, const void *W2, const void *bias,
                         dyad_act act_arg, void *Y, void *H, hipStream_t stream) {
    return forward_impl(enum_value(variant_arg), n_in, n_out, n_dyad, M, enum_value(dtype_arg), X, W1, W2, bias,
                        enum_value(act_arg), Y, H, stream, true);
}

int dyad_backward_dx(dyad_variant variant_arg, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M,
                     dyad_dtype dtype_arg, const void *dZ, const void *W1, const void *W2, dyad_act act_in_arg,
                     const void *H_in, void *dX, hipStream_t stream) {
    const int variant = enum_value(variant_arg), dtype = enum_value(dtype_arg), act_in = enum_value(act_in_arg);
    int rc = check_sizes(variant, n_in, n_out, n_dyad, M, dtype);
    if (rc) return rc;
    if (act_in != DYAD_ACT_NONE && act_in != DYAD_ACT_GELU) return DYAD_ERR_INVALID_ARG;
    if (!W1 || !W2 || (M > 0 && (!dZ || !dX))) return DYAD_ERR_INVALID_ARG;
    if (act_in == DYAD_ACT_GELU && M > 0 && !H_in) return DYAD_ERR_INVALID_ARG;
    if (act_in == DYAD_ACT_NONE) H_in = nullptr;
    if (!aligned16(dZ) || !aligned16(W1) || !aligned16(W2) || !aligned16(H_in) || !aligned16(dX))
        return DYAD_ERR_ALIGN;
    if (M == 0) return DYAD_OK;
    GemmPass p{};
    p.M = M; p.Kin = n_out; p.Nout = n_in; p.D = n_dyad; p.bk = block(n_out, n_dyad); p.bn = block(n_in, n_dyad);
    p.in_t = out_transposed(variant); p.out_t = in_transposed(variant); p.w_t = true;
    p.dtype = dtype;
    p.epilogue = act_in == DYAD_ACT_GELU ? dyad::kEpiGeluGrad : dyad::kEpiBias;
    p.in = dZ; p.W1 = W1; p.W2 = W2; p.bias = nullptr; p.h_in = H_in; p.out = dX; p.h_out = nullptr;
    return run_gemm(p, stream);
}

static DwPass make_dw(int variant, int64_t n_in, int64_t n_out, int64_t D, int64_t M, int dtype) {
    DwPass p{};
    p.M = M; p.n_in = n_in; p.n_out = n_out; p.D = D; p.bi = block(n_in, D); p.bo = block(n_out, D);
    p.in_t = in_transposed(variant); p.out_t = out_transposed(variant); p.dtype = dtype;
    return p;
}

size_t dyad_dw_workspace_bytes(dyad_variant variant_arg, int64_t n_in, int64_t n_out, int64_t n_dyad,
                               int64_t M, dyad_dtype dtype_arg) {
    const int variant = enum_value(variant_arg), dtype = enum_value(dtype_arg);
    if (check_sizes(variant, n_in, n_out, n_dyad, M, dtype)) return 0;
    return dw_workspace(make_dw(variant, n_in, n_out, n_dyad, M, dtype));
}

size_t dyad_dw_workspace_bytes_ex(dyad_variant variant_arg, int64_t n_in, int64_t n_out, int64_t n_dyad,
                                  int64_t M, dyad_dtype dtype_arg, dyad_act act_in_arg) {
    const int variant = enum_value(variant_arg), dtype = enum_value(dtype_arg), act_in = enum_value(act_in_arg);
    if (check_sizes(variant, n_in, n_out, n_dyad, M, dtype)) return 0;
    if (act_in == DYAD_ACT_NONE) return dw_workspace(make_dw(variant, n_in, n_out, n_dyad, M, dtype));
    if (act_in != DYAD_ACT_GELU || dtype != DYAD_BF16) return 0;
    DwPass p = make_dw(variant, n_in, n_out, n_dyad, M, dtype);
    p.gelu_x = true;
    return dyad::mfma_dw_ok(p) ? dyad::mfma_dw_workspace(p) : 0;
}

static int backward_dw_impl(int variant, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M, int dtype,
                            int act_in, const void *dZ, const void *X, void *dW1, void *dW2, void *dbias,
                            void *workspace, size_t workspace_bytes, hipStream_t stream) {
    int rc = check_sizes(variant, n_in, n_out, n_dyad, M, dtype);
    if (rc) return rc;
    if (act_in != DYAD_ACT_NONE && act_in != DYAD_ACT_GELU) return DYAD_ERR_INVALID_ARG;
    if (act_in == DYAD_ACT_GELU && dtype != DYAD_BF16) return DYAD_ERR_DTYPE;
    if (!dW1 || !dW2 || (M > 0 && (!dZ || !X))) return DYAD_ERR_INVALID_ARG;
    if (!aligned16(dZ) || !aligned16(X) || !aligned16(dW1) || !aligned16(dW2) || !aligned16(dbias) ||
        !aligned16(workspace))
        return DYAD_ERR_ALIGN;
    DwPass p = make_dw(variant, n_in, n_out, n_dyad, M, dtype);
    p.gelu_x = act_in == DYAD_ACT_GELU;
    // an input activation runs on the matrix-core kernels only (an empty batch
    // has nothing to activate and takes the usual zero-gradient path)
    if (p.gelu_x && M > 0 && !dyad::mfma_dw_ok(p)) return DYAD_ERR_SHAPE;
    size_t need = dw_workspace(p);
    if (need > 0 && (!workspace || workspace_bytes < need)) return DYAD_ERR_WORKSPACE;
    p.dZ = dZ; p.X = X; p.dW1 = dW1; p.dW2 = dW2; p.db = dbias; p.ws = workspace; p.ws_bytes = workspace_bytes;
    hipError_t e = dyad::mfma_dw_ok(p) ? dyad::launch_mfma_dw(p, stream) : hipErrorNotSupported;
    if (e == hipErrorNotSupported && M > 0) e = dyad::launch_general_mfma_dw(p, stream);
    if (e == hipErrorNotSupported) e = dyad::launch_simt_dw(p, stream);
    return launch_status(e);
}

int dyad_backward_dw(dyad_variant variant_arg, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M,
                     dyad_dtype dtype_arg, const void *dZ, const void *X, void *dW1, void *dW2, void *dbias,
                     void *workspace, size_t workspace_bytes, hipStream_t stream) {
    return backward_dw_impl(enum_value(variant_arg), n_in, n_out, n_dyad, M, enum_value(dtype_arg), DYAD_ACT_NONE,
                            dZ, X, dW1, dW2, dbias, workspace, workspace_bytes, stream);
}

int dyad_backward_dw_ex(dyad_variant variant_arg, int64_t n_in, int64_t n_out, int64_t n_dyad, int64_t M,
                        dyad_dtype dtype_arg, dyad_act act_in_arg, const void *dZ, const void *X, void *dW1,
                        void *dW2, void *dbias, void *workspace, size_t workspace_bytes, hipStream_t stream) {
    return backward_dw_impl(enum_value(variant_arg), n_in, n_out, n_dyad, M, enum_value(dtype_arg),
                            enum_value(act_in_arg), dZ, X, dW1, dW2, dbias, workspace, workspace_bytes, stream);
}

const char *dyad_strerror(int status) {
    switch (status) {
    case DYAD_OK: return "ok";
    case DYAD_ERR_INVALID_ARG: return "invalid argument (enum, size or NULL pointer)";
    case DYAD_ERR_SHAPE: return "no kernel applies an input activation to this shape";
    case DYAD_ERR_ALIGN: return "pointer not 16-byte aligned";
    case DYAD_ERR_DTYPE: return "unsupported dtype";
    case DYAD_ERR_WORKSPACE: return "dW workspace missing or too small";
    case DYAD_ERR_LAUNCH: return "kernel launch failed";
    default: return "unknown status";
    }
}

}  // extern "C"
