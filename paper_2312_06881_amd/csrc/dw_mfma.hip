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
    // n_dyad 3 and 6 without GELU staging, and any n_dyad on block-ordered
    // operands (no transpose: the kernel takes n_dyad at run time)
    const bool pow2 = p.D == 1 || p.D == 2 || p.D == 4 || p.D == 8 || p.D == 16;
    const bool plain = !p.in_t && !p.out_t && !p.gelu_x;
    if (!pow2 && !plain && !((p.D == 3 || p.D == 6) && !p.gelu_x)) return false;
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

// Zero-padded form, for shapes no fused tile takes (widths n_dyad does not
// divide, blocks that are not whole tiles, an n_dyad without tiles):
// block-ordered copies of dZ and X with blocks padded to a multiple of 64
// (component 2's from the residues under a transpose), the plain tiles over
// them into padded gradients, then the real ones.  q: the padded pass.
bool dw_pad_pass(const DwPass &p, DwPass &q) {
    if (p.dtype != kBF16 || p.gelu_x || p.M < kPadMinTokens) return false;
    if (p.n_in % 8 != 0 || p.n_out % 8 != 0 || p.n_in > kPadMaxRow || p.n_out > kPadMaxRow) return false;
    q = p;
    q.bi = pad_up(p.bi, 64);
    q.bo = pad_up(p.bo, 64);
    q.n_in = p.D * q.bi;
    q.n_out = p.D * q.bo;
    q.in_t = q.out_t = false;
    // each copy within 2 GiB (32-bit buffer offsets across a split's tokens)
    const int64_t cap = (int64_t)1 << 31;
    return p.M * q.n_out * 2 <= cap && p.M * q.n_in * 2 <= cap;
}

enum class DwForm { kFused, kPermuted, kPadded };

// The plan a pass runs with (for the permuted and padded forms, that of their
// block-ordered pass).  With GELU(X) the fused form always runs: the
// activation is applied where X is staged, which the copies would bypass.
bool plan(const DwPass &p, DwPlan &pl, DwForm *form, DwPass *padded = nullptr) {
    *form = DwForm::kFused;
    if (!p.gelu_x && dw_permuted(p)) {
        DwPass q = p;
        q.in_t = q.out_t = false;
        if (choose(q, pl)) {
            *form = DwForm::kPermuted;
            return true;
        }
    }
    if (choose(p, pl)) return true;
    DwPass q;
    if (dw_pad_pass(p, q) && choose(q, pl)) {
        *form = DwForm::kPadded;
        if (padded) *padded = q;
        return true;
    }
    return false;
}

}  // namespace

bool mfma_dw_ok(const DwPass &p) {
    DwPlan pl;
    DwForm form;
    return plan(p, pl, &form);
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

// The padded form's workspace after the partial sums: the copies of dZ
// (component 1, then component 2 under an output transpose) and of X (the
// same under an input transpose), then the padded dW1, dW2 and db.
struct DwPadLayout {
    size_t z1, z2, x1, x2, w1, w2, db, end;
};
static DwPadLayout pad_layout(const DwPass &p, const DwPass &q, const DwPlan &pl) {
    DwPadLayout l;
    const size_t zb = round256((size_t)p.M * (size_t)q.n_out * 2), xb = round256((size_t)p.M * (size_t)q.n_in * 2);
    const size_t wb = round256((size_t)(q.D * q.bo * q.bi) * 2);
    l.z1 = round256(plan_workspace(q, pl));
    l.z2 = l.z1 + zb;
    l.x1 = l.z2 + (p.out_t ? zb : 0);
    l.x2 = l.x1 + xb;
    l.w1 = l.x2 + (p.in_t ? xb : 0);
    l.w2 = l.w1 + wb;
    l.db = l.w2 + wb;
    l.end = l.db + (size_t)q.n_out * 2;
    return l;
}

// Workspace of the plan a pass runs with: the partial sums, then (permuted
// and padded forms) the copies, each starting on a 256-byte boundary.  The
// library allocates nothing for the weight gradient; all of it comes from
// the caller.
size_t mfma_dw_workspace(const DwPass &p) {
    DwPlan pl;
    DwForm form;
    DwPass q;
    if (!plan(p, pl, &form, &q)) return 0;
    if (form == DwForm::kPadded) return pad_layout(p, q, pl).end;
    size_t b = plan_workspace(p, pl);
    if (form == DwForm::kPermuted) b = round256(b) + round256(copy_bytes_z(p)) + copy_bytes_x(p);
    return b;
}

hipError_t launch_mfma_dw(const DwPass &p, hipStream_t s) {
    DwPlan pl;
    DwForm form;
    DwPass q;
    if (!plan(p, pl, &form, &q)) return hipErrorNotSupported;
    if (form == DwForm::kPadded) {
        const DwPadLayout l = pad_layout(p, q, pl);
        unsigned char *ws = static_cast<unsigned char *>(p.ws);
        auto at = [&](size_t off) { return reinterpret_cast<uint16_t *>(ws + off); };
        DwPass r = q;
        r.dZ = at(l.z1);
        r.dZ2 = p.out_t ? at(l.z2) : nullptr;
        r.X = at(l.x1);
        r.X2 = p.in_t ? at(l.x2) : nullptr;
        r.dW1 = at(l.w1);
        r.dW2 = at(l.w2);
        r.db = p.db ? at(l.db) : nullptr;
        hipError_t e = launch_pad_rows(static_cast<const uint16_t *>(p.dZ), p.M, p.n_out, (int)p.D, p.bo, q.bo,
                                       at(l.z1), p.out_t ? at(l.z2) : nullptr, s);
        if (e == hipSuccess)
            e = launch_pad_rows(static_cast<const uint16_t *>(p.X), p.M, p.n_in, (int)p.D, p.bi, q.bi, at(l.x1),
                                p.in_t ? at(l.x2) : nullptr, s);
        if (e == hipSuccess) e = launch_dw_plain(r, pl, s);
        if (e == hipSuccess)
            e = launch_unpad_dw(at(l.w1), at(l.w2), at(l.db), p.D, p.bo, p.bi, q.bo, q.bi, p.n_out,
                                static_cast<uint16_t *>(p.dW1), static_cast<uint16_t *>(p.dW2),
                                static_cast<uint16_t *>(p.db), s);
        return e;
    }
    if (form == DwForm::kPermuted) {
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
