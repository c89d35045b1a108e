// Weight-gradient planning (tile configuration and token splits), the
// fixed-order split reduction, and dispatch to the per-variant kernels.
#include "dw_mfma.h"

namespace dyad {

// Adds the splits in order 0..S-1 and writes dW1, dW2 (and db) in bf16.  The
// partial sums are read once and the results written once: both streamed
// (non-temporal).
__global__ void __launch_bounds__(256) dyad_dw_reduce(const float *part, const float *part_db, int splits,
                                                      int64_t per_comp, int64_t n_out, uint16_t *dW1,
                                                      uint16_t *dW2, uint16_t *db) {
    const int64_t n4 = 2 * per_comp / 4;            // float4 groups of the two components
    const int64_t nb4 = db ? n_out / 4 : 0;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n4 + nb4;
         e += (int64_t)gridDim.x * blockDim.x) {
        const bool is_db = e >= n4;
        const int64_t idx = is_db ? (e - n4) * 4 : e * 4;
        const float *src = is_db ? part_db + idx : part + idx;
        const int64_t stride = is_db ? n_out : 2 * per_comp;
        f32x4_t s = {0.f, 0.f, 0.f, 0.f};
        for (int q = 0; q < splits; ++q) s += __builtin_nontemporal_load(reinterpret_cast<const f32x4_t *>(src + q * stride));
        typedef __attribute__((ext_vector_type(2))) uint32_t u32x2_t;
        const u32x2_t o = {pack_bf16(s[0], s[1]), pack_bf16(s[2], s[3])};
        uint16_t *out = is_db ? db + idx : (idx < per_comp ? dW1 + idx : dW2 + (idx - per_comp));
        __builtin_nontemporal_store(o, reinterpret_cast<u32x2_t *>(out));
    }
}

namespace {

struct Cand { int BJ, BK, WJN, WKN; };
constexpr Cand kCands[] = {
#define DYAD_DW_CAND(J_, K_, WJ_, WK_) {J_, K_, WJ_, WK_},
    DYAD_DW_CONFIGS(DYAD_DW_CAND)
#undef DYAD_DW_CAND
};

bool choose(const DwPass &p, DwPlan &pl) {
    if (p.dtype != kBF16 || p.M <= 0) return false;
    if (p.n_in != p.D * p.bi || p.n_out != p.D * p.bo) return false;  // zero-padded widths
    // n_dyad 3 and 6 on the plain path only (no GELU-staging instances)
    const bool pow2 = p.D == 1 || p.D == 2 || p.D == 4 || p.D == 8 || p.D == 16;
    if (!pow2 && !((p.D == 3 || p.D == 6) && !p.gelu_x)) return false;
    // 32-bit buffer offsets within one stage (32 token rows of the wider operand)
    if ((int64_t)kStageK * (p.n_in > p.n_out ? p.n_in : p.n_out) * 2 >= ((int64_t)1 << 31)) return false;
    // A strided BlockTrans operand wants a configuration with an all-groups
    // layout; without one its items read the whole span per group.  At n_dyad
    // 16 the all-groups tiles (32 x 32 per group) pay off only when both
    // operands are strided (measured at d = 4096), and not for a batch of at
    // most 64 tokens, where the one-group 256 x 256 tiles measured 43 against
    // 53 us (wide layer 8192 -> 32768, 16 tokens).
    const bool want_mg = p.D > 1 && (p.in_t || p.out_t) && (p.D < 16 || (p.in_t && p.out_t && p.M > 64));
    // A batch of at most 32 tokens is one stage per tile, bound by the stores of
    // the result: 256 x 128 tiles on 4 x 2 waves measured best there (wide
    // layer 8192 -> 32768, n_dyad 16, 16 tokens: 19-24 us against 24-28 us for
    // 256 x 256), so they go first.
    const bool one_stage = p.M <= kStageK;
    for (int pass = want_mg ? 0 : 1; pass < 2; ++pass)
    for (int ci = one_stage ? -1 : 0; ci < (int)(sizeof(kCands) / sizeof(kCands[0])); ++ci) {
        const Cand c = ci < 0 ? Cand{256, 128, 4, 2} : kCands[ci];
        if (p.bo % c.BJ || p.bi % c.BK) continue;
        if (pass == 0 && !dw_mg_available((int)p.D, c.BJ, c.BK, c.WJN, c.WKN)) continue;
        pl.BJ = c.BJ; pl.BK = c.BK; pl.WJN = c.WJN; pl.WKN = c.WKN;
        pl.tiles_j = (int)(p.bo / c.BJ);
        pl.tiles_k = (int)(p.bi / c.BK);
        const int64_t tiles = 2 * p.D * (int64_t)pl.tiles_j * pl.tiles_k;
        // workgroup slots of the GPU: 256 CUs, one workgroup of 8 or more waves or two 4-wave ones each
        const int64_t slots = 256 * (c.WJN * c.WKN >= 8 ? 1 : 2);
        // as many token splits as fit in one round of slots, each at least 8 stages long
        int64_t splits = tiles >= slots ? 1 : slots / tiles;
        const int64_t max_splits = p.M / (8 * kStageK);
        if (splits > max_splits) splits = max_splits;
        if (splits < 1) splits = 1;
        int64_t tps = (p.M + splits - 1) / splits;
        tps = (tps + 2 * kStageK - 1) / (2 * kStageK) * (2 * kStageK);
        pl.tokens_per_split = tps;
        pl.splits = (int)((p.M + tps - 1) / tps);
        if (tiles * pl.splits >= ((int64_t)1 << 31)) return false;
        return true;
    }
    return false;
}

// Large batches at n_dyad 8 and 16 with a transpose: component 2's strided
// operands (dZ columns j*D + g, X columns k*D + g) are de-interleaved once into
// block-ordered copies in the caller's workspace (each at most 2 GiB), and
// both components then run on the plain tiles, whose operand reads are whole
// rows of one group instead of spans of all D.  Measured on gfx950 against
// the fused tiles, this pays at n_dyad 16 from 2048 tokens (1.1-1.6x at
// d = 1024, 3-4x on the wide layer 8192 -> 32768 at 32768 tokens) and from
// 256 with blocks of at least 512 (1.8-3.5x on the wide layer at 256 and
// 1024 tokens), and at n_dyad 8 from 8192 (at 2048 tokens it lost by up to 15%).
// At n_dyad 3 and 6 no all-groups layout exists (the group grid needs a power
// of two), so the fused tiles would gather a strided operand 2 bytes at a
// time: there the copies go first from 2048 tokens.
bool dw_permuted(const DwPass &p) {
    const bool odd = p.D == 3 || p.D == 6;
    if ((p.D != 8 && p.D != 16 && !odd) || (!p.in_t && !p.out_t)) return false;
    const bool wide = p.D == 16 && p.M >= 256 && p.bi >= 512 && p.bo >= 512;
    if (!wide && p.M < (p.D == 16 || odd ? 2048 : 8192)) return false;
    if ((p.out_t && p.bo % 32 != 0) || (p.in_t && p.bi % 32 != 0)) return false;
    const int64_t cap = (int64_t)1 << 31;
    return !(p.out_t && p.M * p.n_out * 2 > cap) && !(p.in_t && p.M * p.n_in * 2 > cap);
}

// The plan a pass runs with (for the permuted form, that of plain operands).
// With GELU(X) the fused form always runs: the activation is applied where X
// is staged, which the block-ordered copies would bypass.
bool plan(const DwPass &p, DwPlan &pl, bool *permuted) {
    *permuted = false;
    if (!p.gelu_x && dw_permuted(p)) {
        DwPass q = p;
        q.in_t = q.out_t = false;
        if (choose(q, pl)) {
            *permuted = true;
            return true;
        }
    }
    return choose(p, pl);
}

}  // namespace

bool mfma_dw_ok(const DwPass &p) {
    DwPlan pl;
    bool permuted;
    return plan(p, pl, &permuted);
}

// Partial-sum bytes of plan pl (one split writes the results directly).
static size_t plan_workspace(const DwPass &p, const DwPlan &pl) {
    if (pl.splits == 1) return 0;
    return (size_t)pl.splits * (size_t)(2 * p.D * p.bo * p.bi + p.n_out) * sizeof(float);
}

static size_t round256(size_t b) { return (b + 255) & ~(size_t)255; }

// Bytes of the block-ordered copies of the permuted form: dZ under an output
// transpose, X under an input transpose.
static size_t copy_bytes_z(const DwPass &p) { return p.out_t ? (size_t)p.M * (size_t)p.n_out * 2 : 0; }
static size_t copy_bytes_x(const DwPass &p) { return p.in_t ? (size_t)p.M * (size_t)p.n_in * 2 : 0; }

// Workspace of the plan a pass runs with: the partial sums, then (permuted
// form) the copies, each starting on a 256-byte boundary.  The library
// allocates nothing for the weight gradient; all of it comes from the caller.
size_t mfma_dw_workspace(const DwPass &p) {
    DwPlan pl;
    bool permuted;
    if (!plan(p, pl, &permuted)) return 0;
    size_t b = plan_workspace(p, pl);
    if (permuted) b = round256(b) + round256(copy_bytes_z(p)) + copy_bytes_x(p);
    return b;
}

hipError_t launch_mfma_dw(const DwPass &p, hipStream_t s) {
    DwPlan pl;
    bool permuted;
    if (!plan(p, pl, &permuted)) return hipErrorNotSupported;
    if (permuted) {
        // the caller's workspace holds mfma_dw_workspace(p) bytes (checked by
        // the C-ABI): partial sums first, then the copies
        DwPass q = p;
        q.in_t = q.out_t = false;
        const size_t zoff = round256(plan_workspace(p, pl));
        uint16_t *z2 = reinterpret_cast<uint16_t *>(static_cast<unsigned char *>(p.ws) + zoff);
        uint16_t *x2 = reinterpret_cast<uint16_t *>(reinterpret_cast<unsigned char *>(z2) +
                                                    round256(copy_bytes_z(p)));
        hipError_t e = hipSuccess;
        if (p.out_t) {
            e = launch_deinterleave(static_cast<const uint16_t *>(p.dZ), z2, p.M, p.bo, (int)p.D, s);
            q.dZ2 = z2;
        }
        if (e == hipSuccess && p.in_t) {
            e = launch_deinterleave(static_cast<const uint16_t *>(p.X), x2, p.M, p.bi, (int)p.D, s);
            q.X2 = x2;
        }
        return e == hipSuccess ? launch_dw_plain(q, pl, s) : e;
    }
    if (p.gelu_x) {
        if (p.in_t && !p.out_t) return launch_dw_xg_it(p, pl, s);
        if (!p.in_t && p.out_t) return launch_dw_xg_ot(p, pl, s);
        if (p.in_t && p.out_t) return launch_dw_xg_dt(p, pl, s);
        return hipErrorNotSupported;
    }
    if (p.in_t && !p.out_t) return launch_dw_it(p, pl, s);
    if (!p.in_t && p.out_t) return launch_dw_ot(p, pl, s);
    if (p.in_t && p.out_t) return launch_dw_dt(p, pl, s);
    return hipErrorNotSupported;
}

}  // namespace dyad
