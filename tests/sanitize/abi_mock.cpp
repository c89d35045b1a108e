// Host-only check of the C-ABI layer (dyad_abi.hip) under AddressSanitizer and
// UndefinedBehaviorSanitizer, with every kernel launcher replaced by a mock.
// The mocks record the pass they were handed and return an error chosen by
// the test, so the argument checks, the pass descriptions and the mapping of
// a failed launch to DYAD_ERR_LAUNCH run without a GPU.
#include <stdio.h>
#include <stdlib.h>

#include "dyad.h"
#include "dyad_internal.h"

namespace dyad {

hipError_t g_result = hipSuccess;   // what every mock launcher returns
int g_launches = 0;
GemmPass g_gemm{};
DwPass g_dw{};
size_t g_dw_ws = 0;                 // what the mock workspace query reports
const ScratchScope *g_scope = nullptr;       // innermost live ScratchScope
bool g_seen_scope = false;           // a ScratchScope was in force at the last forward launch,
void *g_seen_ptr = nullptr;          // with this buffer
size_t g_seen_bytes = 0;             // of this size

bool skinny_ok(const GemmPass &) { return false; }
hipError_t launch_skinny_gemm(const GemmPass &, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_mfma_gemm(const GemmPass &p, hipStream_t) {
    ++g_launches;
    g_gemm = p;
    const ScratchScope *sc = current_scratch();
    g_seen_scope = sc != nullptr;
    g_seen_ptr = sc ? sc->ptr : nullptr;
    g_seen_bytes = sc ? sc->bytes : 0;
    return g_result;
}
hipError_t launch_padded_gemm(const GemmPass &p, hipStream_t) { ++g_launches; g_gemm = p; return g_result; }
hipError_t launch_general_mfma_gemm(const GemmPass &p, hipStream_t) { ++g_launches; g_gemm = p; return g_result; }
hipError_t launch_simt_gemm(const GemmPass &p, hipStream_t) { ++g_launches; g_gemm = p; return g_result; }
bool mfma_dw_ok(const DwPass &) { return true; }
size_t mfma_dw_workspace(const DwPass &) { return g_dw_ws; }
bool general_dw_ok(const DwPass &) { return false; }
size_t general_dw_workspace(const DwPass &) { return 0; }
size_t simt_dw_workspace(const DwPass &) { return 0; }
hipError_t launch_mfma_dw(const DwPass &p, hipStream_t) { ++g_launches; g_dw = p; return g_result; }
hipError_t launch_general_mfma_dw(const DwPass &p, hipStream_t) { ++g_launches; g_dw = p; return g_result; }
hipError_t launch_simt_dw(const DwPass &p, hipStream_t) { ++g_launches; g_dw = p; return g_result; }

// the fixed scratch of dyad_forward_noalloc, mocked: a stand-in address
ScratchScope::ScratchScope(void *p, size_t b) : ptr(p), bytes(b), prev(g_scope) { g_scope = this; }
ScratchScope::~ScratchScope() { g_scope = prev; }
const ScratchScope *current_scratch() { return g_scope; }
hipError_t noalloc_scratch(void **out) { *out = (void *)0x400000; return hipSuccess; }

}  // namespace dyad

static int failures = 0;

#define EXPECT(cond)                                                             \
    do {                                                                         \
        if (!(cond)) {                                                           \
            fprintf(stderr, "FAILED line %d: %s\n", __LINE__, #cond);            \
            ++failures;                                                          \
        }                                                                        \
    } while (0)

// 16-byte aligned stand-in addresses: the mocks never dereference them.
static void *const A = (void *)0x100000, *const B = (void *)0x200000, *const C = (void *)0x300000;

static int fwd(int variant, int64_t n_in, int64_t n_out, int64_t D, int64_t M, int dtype, const void *X,
               int act, void *Y, void *H) {
    return dyad_forward((dyad_variant)variant, n_in, n_out, D, M, (dyad_dtype)dtype, X, A, B, nullptr,
                        (dyad_act)act, Y, H, nullptr);
}

int main() {
    using namespace dyad;
    // a valid forward reaches a launcher with the pass the header describes
    g_launches = 0;
    EXPECT(fwd(DYAD_DT, 768, 3072, 4, 100, DYAD_BF16, C, DYAD_ACT_GELU, C, C) == DYAD_OK);
    EXPECT(g_launches == 1);
    EXPECT(g_gemm.M == 100 && g_gemm.Kin == 768 && g_gemm.Nout == 3072 && g_gemm.bk == 192 && g_gemm.bn == 768);
    EXPECT(g_gemm.in_t && g_gemm.out_t && !g_gemm.w_t && g_gemm.epilogue == kEpiBiasGelu);
    // the input gradient swaps the roles: Kin = n_out, IT's input transpose becomes an output one
    EXPECT(dyad_backward_dx(DYAD_IT, 768, 3072, 4, 100, DYAD_BF16, C, A, B, DYAD_ACT_NONE, nullptr, C,
                            nullptr) == DYAD_OK);
    EXPECT(g_gemm.Kin == 3072 && g_gemm.Nout == 768 && !g_gemm.in_t && g_gemm.out_t && g_gemm.w_t);
    // zero-padded widths: blocks are ceil(width / n_dyad)
    EXPECT(fwd(DYAD_OT, 7, 6, 2, 5, DYAD_F32, C, DYAD_ACT_NONE, C, nullptr) == DYAD_OK);
    EXPECT(g_gemm.bk == 4 && g_gemm.bn == 3);

    // the no-allocation forward plans the same pass with the fixed scratch in scope
    EXPECT(!g_seen_scope);
    EXPECT(dyad_forward_noalloc(DYAD_DT, 768, 3072, 4, 100, DYAD_BF16, C, A, B, nullptr, DYAD_ACT_GELU, C, C,
                                nullptr) == DYAD_OK);
    EXPECT(g_seen_scope && g_seen_ptr == (void *)0x400000 && g_seen_bytes == kNoAllocScratchBytes);
    EXPECT(current_scratch() == nullptr);
    EXPECT(g_gemm.M == 100 && g_gemm.in_t && g_gemm.out_t && g_gemm.epilogue == kEpiBiasGelu);
    EXPECT(dyad_forward_noalloc(DYAD_IT, 64, 256, 4, 8, (dyad_dtype)7, C, A, B, nullptr, DYAD_ACT_NONE, C,
                                nullptr, nullptr) == DYAD_ERR_DTYPE);

    // a launch the runtime refuses is reported as DYAD_ERR_LAUNCH
    g_result = hipErrorLaunchFailure;
    EXPECT(fwd(DYAD_IT, 64, 256, 4, 8, DYAD_BF16, C, DYAD_ACT_NONE, C, nullptr) == DYAD_ERR_LAUNCH);
    EXPECT(dyad_backward_dx(DYAD_OT, 64, 256, 4, 8, DYAD_BF16, C, A, B, DYAD_ACT_NONE, nullptr, C, nullptr) ==
           DYAD_ERR_LAUNCH);
    g_dw_ws = 0;
    EXPECT(dyad_backward_dw(DYAD_DT, 64, 256, 4, 8, DYAD_BF16, C, C, A, B, nullptr, nullptr, 0, nullptr) ==
           DYAD_ERR_LAUNCH);
    g_result = hipErrorOutOfMemory;
    EXPECT(fwd(DYAD_IT, 64, 256, 4, 8, DYAD_BF16, C, DYAD_ACT_NONE, C, nullptr) == DYAD_ERR_LAUNCH);
    g_result = hipSuccess;

    // argument checks run before any launch
    g_launches = 0;
    EXPECT(fwd(3, 64, 256, 4, 8, DYAD_BF16, C, 0, C, nullptr) == DYAD_ERR_INVALID_ARG);
    EXPECT(fwd(DYAD_IT, 64, 256, 4, 8, 9, C, 0, C, nullptr) == DYAD_ERR_DTYPE);
    EXPECT(fwd(DYAD_IT, 0, 256, 4, 8, DYAD_BF16, C, 0, C, nullptr) == DYAD_ERR_INVALID_ARG);
    EXPECT(fwd(DYAD_IT, 64, 256, 0, 8, DYAD_BF16, C, 0, C, nullptr) == DYAD_ERR_INVALID_ARG);
    EXPECT(fwd(DYAD_IT, 64, 256, 4, -1, DYAD_BF16, C, 0, C, nullptr) == DYAD_ERR_INVALID_ARG);
    EXPECT(fwd(DYAD_IT, (int64_t)1 << 30, (int64_t)1 << 30, 2, 8, DYAD_BF16, C, 0, C, nullptr) ==
           DYAD_ERR_INVALID_ARG);
    EXPECT(fwd(DYAD_IT, INT64_MAX, 256, 4, 8, DYAD_BF16, C, 0, C, nullptr) == DYAD_ERR_INVALID_ARG);
    EXPECT(fwd(DYAD_IT, 64, 256, INT64_MAX, 8, DYAD_BF16, C, 0, C, nullptr) == DYAD_ERR_INVALID_ARG);
    EXPECT(fwd(DYAD_IT, 64, 256, 4, INT64_MAX, DYAD_BF16, C, 0, C, nullptr) == DYAD_ERR_INVALID_ARG);
    EXPECT(fwd(DYAD_IT, 64, 256, 4, 8, DYAD_BF16, nullptr, 0, C, nullptr) == DYAD_ERR_INVALID_ARG);
    EXPECT(fwd(DYAD_IT, 64, 256, 4, 8, DYAD_BF16, (char *)C + 8, 0, C, nullptr) == DYAD_ERR_ALIGN);
    EXPECT(fwd(DYAD_IT, 64, 256, 4, 8, DYAD_BF16, C, 7, C, nullptr) == DYAD_ERR_INVALID_ARG);
    EXPECT(dyad_backward_dx(DYAD_IT, 64, 256, 4, 8, DYAD_BF16, C, A, B, DYAD_ACT_GELU, nullptr, C, nullptr) ==
           DYAD_ERR_INVALID_ARG);
    EXPECT(g_launches == 0);
    // an empty batch is valid and launches nothing
    EXPECT(fwd(DYAD_IT, 64, 256, 4, 0, DYAD_BF16, nullptr, 0, nullptr, nullptr) == DYAD_OK);
    EXPECT(g_launches == 0);

    // the weight gradient refuses a missing or short workspace before launching
    g_dw_ws = 4096;
    EXPECT(dyad_dw_workspace_bytes(DYAD_IT, 64, 256, 4, 8, DYAD_BF16) == 4096);
    EXPECT(dyad_dw_workspace_bytes(DYAD_IT, 64, 256, 4, 8, (dyad_dtype)9) == 0);
    EXPECT(dyad_backward_dw(DYAD_IT, 64, 256, 4, 8, DYAD_BF16, C, C, A, B, nullptr, nullptr, 0, nullptr) ==
           DYAD_ERR_WORKSPACE);
    EXPECT(dyad_backward_dw(DYAD_IT, 64, 256, 4, 8, DYAD_BF16, C, C, A, B, nullptr, C, 4095, nullptr) ==
           DYAD_ERR_WORKSPACE);
    EXPECT(g_launches == 0);
    EXPECT(dyad_backward_dw(DYAD_OT, 64, 256, 4, 8, DYAD_BF16, C, C, A, B, C, C, 4096, nullptr) == DYAD_OK);
    EXPECT(g_launches == 1 && g_dw.ws == C && g_dw.ws_bytes == 4096 && !g_dw.in_t && g_dw.out_t);

    for (int code = -7; code <= 1; ++code) EXPECT(dyad_strerror(code) != nullptr);
    if (failures) return 1;
    printf("abi mock ok\n");
    return 0;
}
