// Device helpers shared by the matrix-core kernels (grouped GEMM and weight
// gradient): vector types, buffer loads, register shuffles of bf16 data, the
// swizzled LDS row layout and the bf16 / normal-distribution epilogue math.
#pragma once

#include "dyad_device.h"

namespace dyad {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(2))) float f32x2_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;

constexpr int kStageK = 32;   // k per stage and per MFMA (v_mfma_f32_16x16x32_bf16)


// ---- buffer loads ------------------------------------------------------------

// Word 3 of a raw buffer resource on gfx9-family parts: 32-bit data, no swizzle.
constexpr int kBufferWord3 = 0x00020000;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kBufferWord3);
}

// Offset that every buffer range check rejects: the load reads zero.
constexpr uint32_t kNoLoad = 0x80000000u;

// 16 bytes at base + voff + soff; zero when voff lies past the buffer's range.
__device__ __forceinline__ uint4 bload16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ uint4 ldg16(const uint16_t *p) { return *reinterpret_cast<const uint4 *>(p); }

// ---- register shuffles ---------------------------------------------------------

// Word w (0..3) of a 16-byte vector, w known at compile time after unrolling.
__device__ __forceinline__ uint32_t word_of(const uint4 &v, int w) {
    const uint32_t lo = (w & 1) ? v.y : v.x;
    const uint32_t hi = (w & 1) ? v.w : v.z;
    return (w & 2) ? hi : lo;
}

// v_perm_b32 selector placing the 16-bit value at byte offset b of {hi:lo} in
// the low half and the one at byte offset c in the high half.
__host__ __device__ constexpr uint32_t perm_sel(int b, int c) {
    return (uint32_t)b | ((uint32_t)(b + 1) << 8) | ((uint32_t)c << 16) | ((uint32_t)(c + 1) << 24);
}

// Residue R (compile time) of 8 consecutive k values held in D consecutive
// 16-byte vectors (input column k*D + r, residue fastest), as one 16-byte
// vector of the 8 values.  Element e of the span sits in vector e / 8, word
// (e % 8) / 2, half e % 2; each output word takes two such halves with one
// v_perm_b32.
template <int D, int R>
__device__ __forceinline__ uint4 deinterleave(const uint4 (&v)[D]) {
    uint32_t o[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const int e0 = (2 * w) * D + R, e1 = (2 * w + 1) * D + R;
        const uint32_t a = word_of(v[e0 >> 3], (e0 & 7) >> 1);   // holds e0
        const uint32_t b = word_of(v[e1 >> 3], (e1 & 7) >> 1);   // holds e1
        // bytes 0-3 of {b:a} are a, bytes 4-7 are b
        o[w] = __builtin_amdgcn_perm(b, a, perm_sel((e0 & 1) * 2, 4 + (e1 & 1) * 2));
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
}

// Residue r (0 <= r < D, uniform across the workgroup, known only at run
// time) of the span, without branches: element e = 2wD + r sits in vector
// e / 8 (a compile-time base, plus one when r carries it over, which happens
// unless D divides 8), word (e % 8) / 2 and half e % 2, so each output word is
// a select or two and one v_perm_b32.  Branch-free code keeps a pipelined main
// loop straight-line, which the compiler needs to wait on exact load counts.
template <int D>
__device__ __forceinline__ uint32_t span_word(const uint4 (&v)[D], int c, int r) {
    // at most one carry: (c % 8) + r < 16 for every n_dyad up to 9, and c % 8 == 0 at 16
    static_assert(D <= 9 || D == 16, "one vector of carry");
    // element c + r, c a multiple of D fixed at compile time after unrolling;
    // when D divides 8 the vector is c / 8 for every r < D
    const int base = c >> 3;
    uint4 x = v[base];
    if constexpr (8 % D != 0)
        if (((c & 7) + r) >= 8) x = v[base + 1 < D ? base + 1 : base];
    return word_of(x, ((c + r) & 7) >> 1);
}

template <int D>
__device__ __forceinline__ uint4 deinterleave_uniform(const uint4 (&v)[D], int r) {
    uint32_t o[4];
    // elements 2wD + r and (2w + 1)D + r: halves r % 2 and (r + D) % 2
    const uint32_t sel = perm_sel((r & 1) * 2, 4 + ((r + D) & 1) * 2);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const uint32_t a = span_word<D>(v, 2 * w * D, r);
        const uint32_t b = span_word<D>(v, (2 * w + 1) * D, r);
        o[w] = __builtin_amdgcn_perm(b, a, sel);
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
}

// Every residue of the span into its own LDS slab (slab R at dst + R * slab).
template <int D, int R = 0>
__device__ __forceinline__ void deinterleave_all(const uint4 (&v)[D], uint16_t *dst, int slab) {
    *reinterpret_cast<uint4 *>(dst + R * slab) = deinterleave<D, R>(v);
    if constexpr (R + 1 < D) deinterleave_all<D, R + 1>(v, dst, slab);
}

// Column e (0..7) of an 8x8 block of bf16 given as 8 rows of 8: the 8 row values, packed.
__device__ __forceinline__ uint4 column_of(const uint4 (&r)[8], int e) {
    uint32_t o[4];
    const uint32_t sel = (e & 1) ? perm_sel(2, 6) : perm_sel(0, 4);
#pragma unroll
    for (int p = 0; p < 4; ++p)
        o[p] = __builtin_amdgcn_perm(word_of(r[2 * p + 1], e >> 1), word_of(r[2 * p], e >> 1), sel);
    return make_uint4(o[0], o[1], o[2], o[3]);
}

// ---- epilogue math -------------------------------------------------------------

// Two fp32 values as packed bf16, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
    const f32x2_t v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ float unpack_bf16(uint32_t w, int half) {
    return __uint_as_float(half ? (w & 0xffff0000u) : (w << 16));
}

// Upper tail P(N > |x|) of the standard normal, and exp(-x^2/2), which the
// density shares.  erfc(|x|/sqrt 2) uses the rational approximation 7.1.26 of
// Abramowitz & Stegun (absolute error below 1.5e-7 in erf, far below the bf16
// rounding of the results); the halving of erfc is folded into the polynomial.
__device__ __forceinline__ float normal_tail(float x, float &e) {
    const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f * 0.70710678118654752f, fabsf(x), 1.0f));
    const float poly =
        t * fmaf(t, fmaf(t, fmaf(t, fmaf(t, 0.5f * 1.061405429f, 0.5f * -1.453152027f), 0.5f * 1.421413741f),
                         0.5f * -0.284496736f),
                 0.5f * 0.254829592f);
    e = __builtin_amdgcn_exp2f(x * (x * -0.72134752044448170f));   // 2^(-x^2 log2(e) / 2)
    return poly * e;
}

// GELU(x) = x Phi(x); below zero Phi(x) is the tail itself, which keeps the
// relative accuracy of small negative outputs.
__device__ __forceinline__ float gelu(float x) {
    float e;
    const float xt = x * normal_tail(x, e);
    return x >= 0.f ? x - xt : xt;
}

// GELU'(x) = Phi(x) + x phi(x), phi(x) = exp(-x^2/2) / sqrt(2 pi).
__device__ __forceinline__ float gelu_grad(float x) {
    float e;
    const float tail = normal_tail(x, e);
    const float cdf = x >= 0.f ? 1.f - tail : tail;
    return fmaf(x * e, 0.3989422804014327f, cdf);
}

// GELU of 8 packed bf16 values, each computed in fp32 and rounded once to
// bf16 (RNE): the activated operand a layer after a GELU multiplies, formed as
// the operand is staged.
__device__ __forceinline__ uint4 gelu8(uint4 v) {
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int p = 0; p < 4; ++p) w[p] = pack_bf16(gelu(unpack_bf16(w[p], 0)), gelu(unpack_bf16(w[p], 1)));
    return make_uint4(w[0], w[1], w[2], w[3]);
}

// Cache policy of streamed data -- a pass's results, and the stashed
// pre-activations its epilogue reads once: non-temporal (the NT bit of the
// buffer instruction), so it does not displace the operand panels and weights
// the tiles re-read from the caches.  Measured on gfx950 at OPT-125m shapes:
// forward with GELU and stash 13 % faster, the GELU' input gradient 7-10 %,
// the other passes 4 %.
constexpr int kStreamPolicy = 2;

// 16 bytes to base + voff, streamed; dropped when voff lies past the buffer's range.
__device__ __forceinline__ void bstore16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint4 v) {
    const u32x4_t w = {v.x, v.y, v.z, v.w};
    __builtin_amdgcn_raw_buffer_store_b128(w, r, (int)voff, 0, kStreamPolicy);
}

// 16 bytes at base + voff + soff read once (streamed); zero past the buffer's range.
__device__ __forceinline__ uint4 bload16_stream(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, kStreamPolicy);
    return make_uint4(v.x, v.y, v.z, v.w);
}

// ---- transpose reads from LDS ---------------------------------------------------

typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4_t;
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4;
typedef __attribute__((address_space(3))) unsigned char lds_u8;

// MFMA operand (8 consecutive reduction indices of one column per lane) from
// LDS rows that run along the columns (one row per reduction index, `pitch`
// bytes apart): two ds_read_b64_tr_b16, rows t..t+3 and t+4..t+7.  In each
// 16-lane group, lane s supplies the address of row 8*(group) + s/4, columns
// 4*(s%4)..+3; lane l gets the 4 rows of column l.
__device__ __forceinline__ bf16x8_t frag_tr(const lds_u8 *p, int pitch) {
    const bf16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)p);
    const bf16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(p + 4 * pitch));
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Swizzle of token-major LDS rows read with ds_read_b64_tr_b16 (rows a
// multiple of 256 bytes): the 32-byte chunks of row r are XORed (within each
// 256-byte block) by (r & 3) | ((r >> 3) & 1) << 2.  The 16 rows one fragment
// read touches (8 g + 0..3, g = 0..3) then fall on every 32-byte bank group
// twice; measured on gfx950: 146 B/clk/CU against 103 for rows padded by 16
// bytes and 31 for plain 256-byte rows.
__host__ __device__ constexpr int tr_sw(int row) { return (row & 3) | (((row >> 3) & 1) << 2); }
__host__ __device__ constexpr int tr_swz(int sw, int byte) {
    const int c = byte >> 5;
    return ((((c & ~7) | ((c ^ sw) & 7))) << 5) | (byte & 31);
}
__host__ __device__ constexpr int round256(int bytes) { return (bytes + 255) & ~255; }

// ---- layout helpers --------------------------------------------------------------

// bf16 element offset of 16-byte chunk c (0..3) of LDS row `row` (rows of 32
// bf16, 64 bytes).  The chunk position is XORed with (row >> 1) & 3, which
// spreads the 16-byte fragment reads of 16 consecutive rows at one chunk over
// distinct banks (measured on gfx950: full LDS read bandwidth, where unswizzled
// 64-byte rows run at half of it).
__device__ __forceinline__ int lds_off(int row, int c) {
    return row * kStageK + ((c ^ (row >> 1)) & 3) * 8;
}

// Tile index of workgroup w, with consecutive tiles (one token panel's column
// tiles, then the next panel's) placed on one XCD: the hardware deals
// workgroups round-robin over the 8 XCDs, each with its own L2.
__device__ __forceinline__ int xcd_tile(int w, int total) {
    const int q = total >> 3, r = total & 7, x = w & 7, i = w >> 3;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + i;
}

}  // namespace dyad
