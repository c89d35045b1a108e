// Small-batch grouped GEMM (bf16; up to 32 tokens, and up to 256 for the
// output-transposed input gradients at n_dyad 16) for the forward pass and the
// input gradient: the regime where the weights are the traffic.
//
// With few tokens each weight entry takes part in at most 32 multiply-adds, so
// a pass is a stream of the two weight tensors from HBM and everything else is
// small.  What holds the tiled kernels back here is parallelism: a pass has too
// few output columns to give every CU a stream of its own.  This path splits
// the reduction instead.  Each component runs as its own grouped GEMM -- the
// rows j of block b against the input columns of block b (the slab b*bk + k,
// or the residue k*D + b under an input transpose) -- over one slice of k, and
// stores fp32 partial sums in a workspace at the pass's output columns (j*D + b
// under an output transpose, b*bn + j otherwise).  A second kernel adds the
// slices of both components in a fixed order, applies the epilogue and stores
// bf16, so results do not depend on scheduling.
//
// Operands.  With so little work per weight byte, what matters is how much of
// the stream is in flight: each wave issues every load of a reduction chunk
// up front -- its 16- or 32-token panel (16-byte loads along k, or 2-byte loads of
// the residue k*D + b under an input transpose), then 32 16-byte weight loads
// -- and multiplies once they land.  Untransposed [bn][bk] weight rows are
// contiguous along k: one load per lane and 16-row tile gives its MFMA operand.
// Transposed [bk][bn] weights are read as 8 x 8 bf16 blocks (8 rows along k of
// 8 consecutive output columns) and transposed in registers, so one lane's
// loads serve 8 tiles whose rows are the output columns j, j + 8, j + 16, ...
// of a 128-column strip.  The 8 waves of a workgroup split the reduction of
// their rows further and add their accumulators through LDS in wave order
// before storing the partial sums; above 32 tokens they split the batch
// instead, 32 tokens a wave, each looping over chunks of the reduction.
#include <mutex>
#include <vector>

#include "dyad_internal.h"
#include "mfma_common.h"

namespace dyad {
namespace {

constexpr int kSkWaves = 8;     // waves per workgroup
constexpr int kSkMaxTok = 256;

// One component of a pass.  A workgroup's 8 waves are tw along the tokens
// times kw along the reduction (each wave chunks x KR deep) times
// 8 / (tw kw) along the rows; each wave owns one row unit of 128 output
// columns (8 MFMA tiles) and 16 or 32 tokens.
struct SkComp {
    const uint16_t *W;   // [D][bn][bk], or [D][bk][bn] when the pass reads weights transposed
    int gather;          // input column k*D + b (else b*bk + k)
    int out_t;           // output column j*D + b (else b*bn + j)
    int kw;              // waves along the reduction in a workgroup
    int row_groups;      // workgroups along the rows of one block
    int slice0;          // partial slice of split 0
    int wgs;             // workgroups of this component
};

struct SkArgs {
    const uint16_t *in;  // [M][Kin]
    float *part;         // [slices][M][Nout] fp32 partial sums
    int M, Kin, Nout, bk, bn, D;
    int row_units;       // row units per block
    int tw;              // waves along the tokens in a workgroup (16 * MT tokens each)
    int chunks;          // KR-deep chunks per wave
    SkComp c[2];
};

__device__ __forceinline__ bf16x8_t as_frag(const uint4 &v) {
    const u32x4_t w = {v.x, v.y, v.z, v.w};
    return __builtin_bit_cast(bf16x8_t, w);
}

__device__ __forceinline__ uint32_t ld_b16(__amdgpu_buffer_rsrc_t r, uint32_t voff) {
    return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)voff, 0, 0);
}

template <bool W_T> struct SkShape {
    static constexpr int NA = 8;                 // 16-row A tiles per wave
    static constexpr int RU = 128;               // rows per row unit
};

// LDS for the reduction across the waves of a workgroup: at most 7 waves hand
// over NA x MT accumulator tiles of 64 lanes x 16 bytes.
template <int MT, bool W_T>
constexpr int sk_lds_bytes() { return (kSkWaves - 1) * SkShape<W_T>::NA * MT * 64 * 16; }

// One wave: for each KR-deep chunk of its reduction range, every load issued
// up front (the token panel, then the weights) and then the multiplies; after
// the last chunk a fixed-order sum over the workgroup's waves along k, and the
// partial sums stored.
template <int MT, bool W_T, bool GATHER, int KR, bool LOOP>
__device__ __forceinline__ void skinny_wave(const SkArgs &a, const SkComp &c, int bid, unsigned char *lds) {
    constexpr int STEPS = KR / 32;
    constexpr int NA = SkShape<W_T>::NA, RU = SkShape<W_T>::RU;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: scalar arithmetic
    const int lr = lane & 15, lg = lane >> 4;
    // tw and kw are powers of two: the wave's place by shifts, before any load
    const int tw_n = a.tw, kw_n = c.kw, tw_l = __builtin_ctz(tw_n), kw_l = __builtin_ctz(kw_n);
    const int rw_n = kSkWaves >> (tw_l + kw_l);
    const int wt = wave & (tw_n - 1), wk = (wave >> tw_l) & (kw_n - 1), wr = wave >> (tw_l + kw_l);
    const int rg = bid % c.row_groups;
    bid /= c.row_groups;
    const int blk = bid % a.D;
    const int split = bid / a.D;
    int ru = rg * rw_n + wr;
    const bool live = ru < a.row_units;
    ru = live ? ru : a.row_units - 1;                 // idle waves re-read a valid unit
    const int j0 = ru * RU;
    const int t0 = wt * 16 * MT;                      // the wave's first token
    const int kspan = a.chunks * KR;                  // the wave's reduction range
    const int kw0 = (split * kw_n + wk) * kspan;
    const int bk = a.bk, bn = a.bn, Kin = a.Kin, D = a.D;

    const int tok_left = a.M - t0;                    // tokens past the batch read zero
    const __amdgpu_buffer_rsrc_t rin =
        buffer_rsrc(a.in + (int64_t)t0 * Kin, tok_left > 0 ? (uint32_t)tok_left * (uint32_t)Kin * 2u : 0u);
    const __amdgpu_buffer_rsrc_t rw = buffer_rsrc(c.W, (uint32_t)D * (uint32_t)bn * (uint32_t)bk * 2u);

    f32x4_t acc[NA][MT];
#pragma unroll
    for (int i = 0; i < NA; ++i)
#pragma unroll
        for (int m = 0; m < MT; ++m) acc[i][m] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const int nch = LOOP ? a.chunks : 1;   // one chunk: straight-line code
    for (int ch = 0; ch < nch; ++ch) {
        const int k0 = kw0 + ch * KR;
        // B operands: token t0 + 16 m + lr, k = k0 + 32 s + 8 lg ..+7
        uint4 xin[STEPS][MT];
        uint32_t xg[STEPS][MT][8];
#pragma unroll
        for (int s = 0; s < STEPS; ++s)
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                const uint32_t row = (uint32_t)(16 * m + lr) * (uint32_t)Kin;
                const int k = k0 + 32 * s + 8 * lg;
                if constexpr (GATHER) {
#pragma unroll
                    for (int t = 0; t < 8; ++t) xg[s][m][t] = ld_b16(rin, (row + (uint32_t)((k + t) * D + blk)) * 2u);
                } else {
                    xin[s][m] = bload16(rin, (row + (uint32_t)(blk * bk + k)) * 2u, 0);
                }
            }
        // A operands
        uint4 w[STEPS][NA];
#pragma unroll
        for (int s = 0; s < STEPS; ++s)
#pragma unroll
            for (int i = 0; i < NA; ++i) {
                uint32_t off;
                if constexpr (W_T)   // row k0 + 32 s + 8 lg + i, columns j0 + 8 lr ..+7
                    off = ((uint32_t)(blk * bk + k0 + 32 * s + 8 * lg + i) * (uint32_t)bn + (uint32_t)(j0 + 8 * lr)) * 2u;
                else                 // row j0 + 16 i + lr, k = k0 + 32 s + 8 lg ..+7
                    off = ((uint32_t)(blk * bn + j0 + 16 * i + lr) * (uint32_t)bk + (uint32_t)(k0 + 32 * s + 8 * lg)) * 2u;
                w[s][i] = bload16(rw, off, 0);
            }

        // keep every load above the multiplies: the scheduler would otherwise
        // sink them next to their use and leave one step of the stream in flight
        __builtin_amdgcn_sched_barrier(0);

#pragma unroll
        for (int s = 0; s < STEPS; ++s) {
            bf16x8_t bf[MT];
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                if constexpr (GATHER) {
                    const uint4 v = make_uint4(xg[s][m][0] | (xg[s][m][1] << 16), xg[s][m][2] | (xg[s][m][3] << 16),
                                               xg[s][m][4] | (xg[s][m][5] << 16), xg[s][m][6] | (xg[s][m][7] << 16));
                    bf[m] = as_frag(v);
                } else {
                    bf[m] = as_frag(xin[s][m]);
                }
            }
#pragma unroll
            for (int i = 0; i < NA; ++i) {
                bf16x8_t af;
                if constexpr (W_T) af = as_frag(column_of(w[s], i));   // tile i: columns j0 + 8 r + i
                else af = as_frag(w[s][i]);
#pragma unroll
                for (int m = 0; m < MT; ++m)
                    acc[i][m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bf[m], acc[i][m], 0, 0, 0);
            }
        }
        if constexpr (LOOP) __builtin_amdgcn_sched_barrier(0);   // the next chunk's loads stay below
    }

    // waves k-split inside the workgroup: waves 1.. hand over, wave 0 adds in order
    if (kw_n > 1) {
        f32x4_t *slot = reinterpret_cast<f32x4_t *>(lds);
        if (wk > 0) {
            f32x4_t *mine = slot + (((wk - 1) * rw_n + wr) * tw_n + wt) * NA * MT * 64;
#pragma unroll
            for (int i = 0; i < NA; ++i)
#pragma unroll
                for (int m = 0; m < MT; ++m) mine[(i * MT + m) * 64 + lane] = acc[i][m];
        }
        __syncthreads();
        if (wk > 0) return;
        for (int q = 1; q < kw_n; ++q) {
            const f32x4_t *src = slot + (((q - 1) * rw_n + wr) * tw_n + wt) * NA * MT * 64;
#pragma unroll
            for (int i = 0; i < NA; ++i)
#pragma unroll
                for (int m = 0; m < MT; ++m) acc[i][m] += src[(i * MT + m) * 64 + lane];
        }
    }
    if (!live) return;

    // partial sums: lane holds output rows 4 lg + q of token column lr
    float *P = a.part + (int64_t)(c.slice0 + split) * a.M * a.Nout;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
        const int n = t0 + 16 * m + lr;
        if (n >= a.M) continue;
        float *row = P + (int64_t)n * a.Nout;
        if constexpr (!W_T) {
#pragma unroll
            for (int i = 0; i < NA; ++i) {
                const int j = j0 + 16 * i + 4 * lg;
                if (!c.out_t) {
                    *reinterpret_cast<f32x4_t *>(row + blk * bn + j) = acc[i][m];
                } else {
#pragma unroll
                    for (int q = 0; q < 4; ++q) row[(j + q) * D + blk] = acc[i][m][q];
                }
            }
        } else {
            // tile e, row 4 lg + q is output column j0 + 8 (4 lg + q) + e
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int j = j0 + 32 * lg + 8 * q;
                if (!c.out_t) {
                    float *dst = row + blk * bn + j;
                    *reinterpret_cast<f32x4_t *>(dst) = f32x4_t{acc[0][m][q], acc[1][m][q], acc[2][m][q], acc[3][m][q]};
                    *reinterpret_cast<f32x4_t *>(dst + 4) =
                        f32x4_t{acc[4][m][q], acc[5][m][q], acc[6][m][q], acc[7][m][q]};
                } else {
#pragma unroll
                    for (int e = 0; e < 8; ++e) row[(j + e) * D + blk] = acc[e][m][q];
                }
            }
        }
    }
}

// Both components in one launch: the first c[0].wgs workgroups run component 1.
// LOOP: waves take more than one chunk (batches above 32 tokens).
template <int MT, bool W_T, bool G2, int KR, bool LOOP>
__global__ void __launch_bounds__(64 * kSkWaves) skinny_part_kernel(SkArgs a) {
    __shared__ __attribute__((aligned(16))) unsigned char lds[sk_lds_bytes<MT, W_T>()];
    const int bid = blockIdx.x;
    if (bid < a.c[0].wgs) skinny_wave<MT, W_T, false, KR, LOOP>(a, a.c[0], bid, lds);
    else skinny_wave<MT, W_T, G2, KR, LOOP>(a, a.c[1], bid - a.c[0].wgs, lds);
}

// out[n][f] = epilogue(sum of the slices, in slice order); 8 columns per thread.
// PERM: slices perm_from .. slices-1 hold their sums in block order, output
// column j*D + g at column g*bn + j, and are read there.
template <bool PERM>
__global__ void __launch_bounds__(256) skinny_reduce_kernel(GemmPass p, const float *part, int slices, int perm_from) {
    const int64_t per_row = p.Nout / 8;
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= p.M * per_row) return;
    const int64_t n = idx / per_row, f = (idx % per_row) * 8;
    const int64_t e0 = n * p.Nout + f, stride = p.M * p.Nout;
    float x[8];
    {
        const f32x4_t lo = *reinterpret_cast<const f32x4_t *>(part + e0);
        const f32x4_t hi = *reinterpret_cast<const f32x4_t *>(part + e0 + 4);
#pragma unroll
        for (int v = 0; v < 4; ++v) { x[v] = lo[v]; x[4 + v] = hi[v]; }
    }
    for (int s = 1; s < slices; ++s) {
        if (PERM && s >= perm_from) {
            const float *row = part + s * stride + n * p.Nout;
            const int D = (int)p.D, bn = (int)p.bn;
#pragma unroll
            for (int v = 0; v < 8; ++v) {
                const int c = (int)f + v;
                x[v] += row[(c % D) * bn + c / D];
            }
            continue;
        }
        const float *src = part + s * stride + e0;
        const f32x4_t lo = *reinterpret_cast<const f32x4_t *>(src);
        const f32x4_t hi = *reinterpret_cast<const f32x4_t *>(src + 4);
#pragma unroll
        for (int v = 0; v < 4; ++v) { x[v] += lo[v]; x[4 + v] += hi[v]; }
    }
    uint32_t o[4], h[4];
    if (p.epilogue == kEpiGeluGrad) {
        const uint4 hv = *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(p.h_in) + e0);
        const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
#pragma unroll
        for (int w = 0; w < 4; ++w)
            o[w] = pack_bf16(x[2 * w] * gelu_grad(unpack_bf16(hw[w], 0)),
                             x[2 * w + 1] * gelu_grad(unpack_bf16(hw[w], 1)));
    } else {
        if (p.bias) {
            const uint4 bv = *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(p.bias) + f);
            const uint32_t bw[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                x[2 * w] += unpack_bf16(bw[w], 0);
                x[2 * w + 1] += unpack_bf16(bw[w], 1);
            }
        }
        if (p.epilogue == kEpiBiasGelu) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                h[w] = pack_bf16(x[2 * w], x[2 * w + 1]);
                o[w] = pack_bf16(gelu(x[2 * w]), gelu(x[2 * w + 1]));
            }
            if (p.h_out) *reinterpret_cast<uint4 *>(static_cast<uint16_t *>(p.h_out) + e0) = make_uint4(h[0], h[1], h[2], h[3]);
        } else {
#pragma unroll
            for (int w = 0; w < 4; ++w) o[w] = pack_bf16(x[2 * w], x[2 * w + 1]);
        }
    }
    *reinterpret_cast<uint4 *>(static_cast<uint16_t *>(p.out) + e0) = make_uint4(o[0], o[1], o[2], o[3]);
}

// ---- host: plan, workspace, launch ------------------------------------------------

// Reduction depth per wave and chunk: 128, i.e. 32 weight loads of 16 bytes
// per lane; 64 for batches above 32 tokens, whose waves loop over chunks and
// keep 32 tokens of accumulators.
int sk_depth(const GemmPass &p) {
    // (32 tokens of gathered transposed-weight operands also take 64: at 128
    // they spill)
    const bool deep = p.M <= 16 || (p.M <= 32 && !(p.w_t && p.in_t && p.D > 1));
    for (int kr = deep ? 128 : 64; kr >= 64; kr /= 2)
        if (p.bk % kr == 0) return kr;
    return 0;
}

// Workgroup shape and reduction split of a pass (both components alike).
struct SkPlan {
    int mt;              // 16-token MFMA column tiles per wave
    int tw;              // waves along the tokens
    int kw;              // waves along the reduction
    int chunks;          // KR-deep chunks per wave
    int row_groups;      // workgroups along the rows of one block
    int splits;          // workgroups along the reduction of one block
    int64_t wgs;         // workgroups per component
};

// Tokens: 16 (at most 16) or 32 per wave, tw waves covering the batch.  kw as
// large as the block allows, so each component leaves as few partial slices
// as possible, unless it idles more than a quarter of the waves along the
// rows.  Up to 32 tokens a wave takes one chunk, so all its loads are in flight
// at once; with more tokens the weights take part in more multiply-adds, and
// each wave takes as many chunks as still leave 128 workgroups per component.
bool sk_plan(const GemmPass &p, int kr, SkPlan &pl) {
    pl.mt = p.M <= 16 ? 1 : 2;
    pl.tw = 1;
    while (pl.tw * 16 * pl.mt < p.M) pl.tw *= 2;
    if (pl.tw > kSkWaves) return false;
    const int row_units = (int)(p.bn / 128);
    const int kunits = (int)(p.bk / kr);
    pl.kw = 1;
    pl.row_groups = (row_units + kSkWaves / pl.tw - 1) / (kSkWaves / pl.tw);
    for (int kw = kSkWaves / pl.tw; kw > 1; kw /= 2) {
        if (kunits % kw != 0) continue;
        const int rw = kSkWaves / (pl.tw * kw);
        const int groups = (row_units + rw - 1) / rw;
        if (4 * (groups * rw - row_units) > groups * rw) continue;
        pl.kw = kw;
        pl.row_groups = groups;
        break;
    }
    const int per = kunits / pl.kw;
    pl.chunks = 1;
    if (pl.tw > 1)
        for (int ch = per; ch > 1; --ch)
            if (per % ch == 0 && p.D * pl.row_groups * (per / ch) >= 128) {
                pl.chunks = ch;
                break;
            }
    pl.splits = per / pl.chunks;
    pl.wgs = p.D * pl.row_groups * pl.splits;
    return pl.wgs < ((int64_t)1 << 30);
}

template <int MT, bool W_T, bool G2>
hipError_t launch_part_kr(const SkArgs &a, int kr, hipStream_t s) {
    const dim3 grid((unsigned)(a.c[0].wgs + a.c[1].wgs)), block(64 * kSkWaves);
    if (a.chunks > 1) {
        if (kr != 64) return hipErrorNotSupported;
        skinny_part_kernel<MT, W_T, G2, 64, true><<<grid, block, 0, s>>>(a);
    } else if (kr == 128) {
        if constexpr (MT > 1 && W_T && G2) return hipErrorNotSupported;   // sk_depth gives 64
        else skinny_part_kernel<MT, W_T, G2, 128, false><<<grid, block, 0, s>>>(a);
    } else if (kr == 64) {
        skinny_part_kernel<MT, W_T, G2, 64, false><<<grid, block, 0, s>>>(a);
    } else {
        return hipErrorNotSupported;
    }
    return hipGetLastError();
}

template <int MT>
hipError_t launch_part_mt(const SkArgs &a, int kr, bool w_t, bool g2, hipStream_t s) {
    if (w_t) return g2 ? launch_part_kr<MT, true, true>(a, kr, s) : launch_part_kr<MT, true, false>(a, kr, s);
    return g2 ? launch_part_kr<MT, false, true>(a, kr, s) : launch_part_kr<MT, false, false>(a, kr, s);
}

// Partial-sum workspace: one buffer per (device, stream), from a
// stream-ordered pool per device, kept between calls and regrown in stream
// order (the old buffer is freed on the same stream), so calls on one stream
// reuse it in order and calls on different streams never share it.
struct StreamWorkspace {
    int dev;
    hipStream_t stream;
    void *ptr;
    size_t bytes;
};
std::mutex g_ws_mu;
hipMemPool_t g_pool[64] = {};
std::vector<StreamWorkspace> g_ws;

hipError_t pool_of(int dev, hipMemPool_t *out) {
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    if (!g_pool[dev]) {
        hipMemPoolProps props = {};
        props.allocType = hipMemAllocationTypePinned;
        props.handleTypes = hipMemHandleTypeNone;
        props.location.type = hipMemLocationTypeDevice;
        props.location.id = dev;
        hipMemPool_t pool = nullptr;
        hipError_t e = hipMemPoolCreate(&pool, &props);
        if (e != hipSuccess) return e;
        uint64_t keep = UINT64_MAX;   // keep freed blocks in the pool
        e = hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
        if (e != hipSuccess) {
            (void)hipMemPoolDestroy(pool);
            return e;
        }
        g_pool[dev] = pool;
    }
    *out = g_pool[dev];
    return hipSuccess;
}

}  // namespace

hipError_t split_workspace(hipStream_t s, size_t bytes, void **out) {
    if (const ScratchScope *sc = current_scratch()) {
        // the fixed scratch of dyad_forward_noalloc: never grown, never allocated
        if (bytes > sc->bytes) return hipErrorOutOfMemory;
        *out = sc->ptr;
        return hipSuccess;
    }
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(g_ws_mu);
    StreamWorkspace *w = nullptr;
    for (auto &x : g_ws)
        if (x.dev == dev && x.stream == s) w = &x;
    if (w && w->bytes >= bytes) {
        *out = w->ptr;
        return hipSuccess;
    }
    // No allocation (or regrowth) while the stream is being captured into a
    // graph: the buffer would belong to the graph, not to later eager calls.
    // The caller then takes a plan that needs no buffer.
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    e = hipStreamIsCapturing(s, &cap);
    if (e != hipSuccess) return e;
    if (cap != hipStreamCaptureStatusNone) return hipErrorNotSupported;
    hipMemPool_t pool;
    e = pool_of(dev, &pool);
    if (e != hipSuccess) return e;
    const size_t want = bytes < ((size_t)1 << 20) ? ((size_t)1 << 20) : bytes;
    void *p = nullptr;
    e = hipMallocFromPoolAsync(&p, want, pool, s);
    if (e != hipSuccess) return e;
    if (w) {
        (void)hipFreeAsync(w->ptr, s);
        w->ptr = p;
        w->bytes = want;
    } else {
        g_ws.push_back(StreamWorkspace{dev, s, p, want});
    }
    *out = p;
    return hipSuccess;
}

hipError_t launch_split_reduce(const GemmPass &p, const float *part, int slices, hipStream_t s, bool perm_last,
                               int perm_from) {
    if (p.Nout % 8 != 0) return hipErrorNotSupported;
    const int64_t threads = p.M * (p.Nout / 8);
    const unsigned blocks = (unsigned)((threads + 255) / 256);
    if (perm_last) perm_from = slices - 1;
    if (perm_from < 1) perm_from = 1;   // slice 0 is read in output order
    if (perm_from < slices)
        skinny_reduce_kernel<true><<<blocks, 256, 0, s>>>(p, part, slices, perm_from);
    else
        skinny_reduce_kernel<false><<<blocks, 256, 0, s>>>(p, part, slices, slices);
    return hipGetLastError();
}

// out[n][g*bk + k] = in[n][k*D + g] for a token row of D*bk elements: the
// input columns of residue g made the contiguous block g.  A group of 4*D
// threads moves 32 reduction indices of one row: 16-byte loads of the row
// span into LDS, then per thread 8 indices of one residue, stored as 16
// bytes.  A block holds 256 / (4*D) groups; where 4*D does not divide 256 its
// last threads have no group and stay idle.
__global__ void __launch_bounds__(256) deinterleave_kernel(const uint16_t *in, uint16_t *out, int64_t M, int bk,
                                                           int D) {
    __shared__ uint4 buf[256];
    const int tid = threadIdx.x, per = 4 * D;
    const int c = tid / per, pc = tid % per;
    const int spans = bk / 32;
    const int64_t gc = (int64_t)blockIdx.x * (256 / per) + c;
    const bool ok = c < 256 / per && gc < M * spans;
    const int64_t n = ok ? gc / spans : 0, kc = ok ? gc % spans : 0;
    const int64_t Kin = (int64_t)bk * D;
    if (ok) buf[tid] = *reinterpret_cast<const uint4 *>(in + n * Kin + kc * 32 * D + pc * 8);
    __syncthreads();
    if (!ok) return;
    const int g = pc / 4, k0 = (pc % 4) * 8;
    const uint16_t *span = reinterpret_cast<const uint16_t *>(buf + c * per);
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
        w[e] = (uint32_t)span[(k0 + 2 * e) * D + g] | ((uint32_t)span[(k0 + 2 * e + 1) * D + g] << 16);
    *reinterpret_cast<uint4 *>(out + n * Kin + (int64_t)g * bk + kc * 32 + k0) = make_uint4(w[0], w[1], w[2], w[3]);
}

hipError_t launch_deinterleave(const uint16_t *in, uint16_t *out, int64_t M, int64_t bk, int D, hipStream_t s) {
    if (D < 1 || D > 64 || bk % 32 != 0 || M < 0) return hipErrorNotSupported;
    if (M == 0) return hipSuccess;
    const int64_t groups = M * (bk / 32), per_block = 256 / (4 * D);
    const int64_t blocks = (groups + per_block - 1) / per_block;
    if (blocks >= ((int64_t)1 << 31)) return hipErrorNotSupported;
    deinterleave_kernel<<<(unsigned)blocks, 256, 0, s>>>(in, out, M, (int)bk, D);
    return hipGetLastError();
}

bool skinny_ok(const GemmPass &p) {
    if (p.dtype != kBF16 || p.M < 1 || p.M > kSkMaxTok) return false;
    // Above 32 tokens the waves of a workgroup split the batch and each reads
    // the same weights, which pays only against the 32-token tiles the tiled
    // kernels fall back to for an output transpose at n_dyad 16 with
    // transposed weights (input gradients of IT / DT; measured at the wide
    // layer with 256 tokens: 72-186 us against 171-220 us, while forward
    // passes and other input gradients took 1.2-2.8x longer than tiled).
    if (p.M > 32 && !(p.w_t && p.out_t && p.D >= 16)) return false;
    if (p.Kin != p.D * p.bk || p.Nout != p.D * p.bn) return false;
    // where the large-batch form (de-interleaved input, per-block GEMMs) pays,
    // it goes first (wide layer 8192 -> 32768 at 256 tokens: Dyad-IT fc1 input
    // gradient 49 us there against 73 here, with its split reduction and
    // weight-major tile order; the DT one 56 against 167)
    if (p.M > 32 && permuted_pays((int)p.D, p.out_t, p.w_t, p.M, p.bk)) return false;
    // 32-bit buffer offsets: the weights and the input panel
    if (2 * p.D * p.bn * p.bk >= ((int64_t)1 << 31) || 2 * p.M * p.Kin >= ((int64_t)1 << 31)) return false;
    if (p.bn % 128 != 0) return false;
    const int kr = sk_depth(p);
    SkPlan pl;
    return kr != 0 && sk_plan(p, kr, pl);
}

hipError_t launch_skinny_gemm(const GemmPass &p, hipStream_t s) {
    if (!skinny_ok(p)) return hipErrorNotSupported;
    const int kr = sk_depth(p);
    SkPlan pl;
    sk_plan(p, kr, pl);
    SkArgs a{};
    a.in = static_cast<const uint16_t *>(p.in);
    a.M = (int)p.M; a.Kin = (int)p.Kin; a.Nout = (int)p.Nout;
    a.bk = (int)p.bk; a.bn = (int)p.bn; a.D = (int)p.D;
    a.row_units = (int)(p.bn / 128);
    a.tw = pl.tw;
    a.chunks = pl.chunks;
    int slices = 0;
    for (int c = 0; c < 2; ++c) {
        SkComp &k = a.c[c];
        k.W = static_cast<const uint16_t *>(c == 0 ? p.W1 : p.W2);
        k.gather = c == 1 && p.in_t && p.D > 1;
        k.out_t = c == 1 && p.out_t;
        k.kw = pl.kw;
        k.row_groups = pl.row_groups;
        k.wgs = (int)pl.wgs;
        k.slice0 = slices;
        slices += pl.splits;
    }
    const size_t bytes = (size_t)slices * (size_t)p.M * (size_t)p.Nout * sizeof(float);
    void *ws = nullptr;
    if (split_workspace(s, bytes, &ws) != hipSuccess) {
        (void)hipGetLastError();      // no workspace: the tiled kernels take the pass
        return hipErrorNotSupported;
    }
    a.part = static_cast<float *>(ws);
    const bool g2 = a.c[1].gather != 0;
    hipError_t e = pl.mt == 1 ? launch_part_mt<1>(a, kr, p.w_t, g2, s) : launch_part_mt<2>(a, kr, p.w_t, g2, s);
    if (e == hipSuccess) e = launch_split_reduce(p, a.part, slices, s);
    return e;
}

}  // namespace dyad
