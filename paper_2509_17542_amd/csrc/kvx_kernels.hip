// gfx950 kernels of the KV-cache conversion: pack (source shards -> transfer
// tensor), unpack (transfer tensor -> paged cache) and the fused repack
// (source shards -> paged cache).
//
// Work decomposition: a work unit is one pass over part of a page's rows of
// one head segment: (layer, k/v plane) x (logical page of a request) x (head
// segment: the decode heads that come from one source shard) x (part).  A page
// holds ntok <= block_size tokens; a segment of n heads gives it ntok * n
// "rows" of head_dim elements.  Each row is covered by a power-of-two group of
// lanes, one per 16-byte chunk of the transfer-tensor row (global_load_dwordx4
// / global_store_dwordx4; a lane that dequantises 8-bit codes into a 16-bit
// cache writes two cache chunks), so a 256-thread workgroup covers 256 /
// lanes-per-row rows: one part.  The shard, its first head and the segment's
// place in the decode row are the same for the whole workgroup (scalar
// registers), so a lane's load address needs no table lookup; every lane
// issues its load(s), converts and stores once.
//
// Units are numbered plane-major, page, segment, then part, so consecutive
// units read consecutive source bytes.  The 1-D grid is dealt to the 8 XCDs
// round-robin (workgroup i runs on XCD i % 8); workgroup i takes unit
// (i % 8) * units_per_xcd + i / 8, so every XCD streams one contiguous run of
// units through its own L2 instead of every eighth unit of the whole stream.
//
// A paged source (the prefill side's own paged cache, with its own page size
// and block table) adds one lookup per row: the page of the row's token in
// the source block table.  Rows of one token are contiguous in a source page,
// as in a token-major source, so the unit and row order are the same.
//
// Destination pages of the paged cache are scattered over a pool of tens to
// hundreds of GiB, so their first touch often waits for an address
// translation.  The first workgroup of each page (part 0, segment 0) therefore
// also reads one dword of the destination page kPrefetchPages pages further
// along its XCD's run; the value is discarded, and the translation is cached by
// the time that page's workgroups store to it.  Row loads and stores are
// non-temporal: every row is read once and the destination is not read again
// by this launch.
//
// The path is a gather/scatter stream with no reuse and no contraction: the
// 16-bit conversions are bound by HBM bandwidth, the 8-bit ones (e4m3fn,
// e5m2, per-row scales) by the vector ALUs and HBM together.  There is no
// MFMA and no LDS staging of rows: rows are whole 16-byte vectors on both
// sides, so a [token][head] <-> [head][token] reorder is a change of row
// addresses only.  (The quantising kernels use LDS only to gather their 4-byte
// row scales into whole-line stores.)
#include <hip/hip_runtime.h>

#include <mutex>

#include "kvx_internal.h"

namespace kvx {
namespace {

// ---- element conversions ---------------------------------------------------

// fp16 bits -> bf16 bits, round to nearest even.  The widening to fp32 is
// exact (v_cvt_f32_f16); the rounding adds half an ulp of bf16 minus one plus
// the lowest kept bit, then truncates.  NaN keeps its sign and the top seven
// payload bits, with the quiet bit set.
__device__ __forceinline__ uint32_t f16_to_bf16(uint32_t h)
{
    if ((h & 0x7C00u) == 0x7C00u && (h & 0x03FFu))
        return (h & 0x8000u) | 0x7FC0u | ((h & 0x03FFu) >> 3);
    const _Float16 x = __builtin_bit_cast(_Float16, static_cast<unsigned short>(h));
    const uint32_t u = __float_as_uint(static_cast<float>(x));
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Magnitude q of a quotient (finite, >= 0, at most 448 plus an ulp) ->
// e4m3fn code without the sign: saturate at 448 (0x7E); below 2^-6 the grid
// step is 2^-9, so the code is q * 2^9 rounded to an even integer (8 is the
// code of 2^-6); above, round the fp32 fraction to 3 bits (ties to even) and
// rebias the exponent from 127 to 7.
__device__ __forceinline__ uint32_t e4m3_code(float q)
{
    if (q >= 448.0f) return 0x7Eu;
    if (q < 0x1p-6f) return static_cast<uint32_t>(__builtin_rintf(q * 512.0f));
    const uint32_t u = __float_as_uint(q);
    return ((u + 0x7FFFFu + ((u >> 20) & 1u)) >> 20) - (120u << 3);
}

// The same for OCP e5m2 (2 fraction bits, bias 15): saturate at 57344
// (0x7B); below 2^-14 the grid step is 2^-16; above, round the fp32 fraction
// to 2 bits (ties to even) and rebias the exponent from 127 to 15.
__device__ __forceinline__ uint32_t e5m2_code(float q)
{
    if (q >= 57344.0f) return 0x7Bu;
    if (q < 0x1p-14f) return static_cast<uint32_t>(__builtin_rintf(q * 65536.0f));
    const uint32_t u = __float_as_uint(q);
    return ((u + 0xFFFFFu + ((u >> 21) & 1u)) >> 21) - (112u << 2);
}

// The 8-bit transfer formats: e4m3fn (kE5 false) and e5m2 (kE5 true).  Both
// use S.1111111 (0x7F) for NaN, as the conversions write it.
template <bool kE5>
struct Fp8 {
    static constexpr float kMax = kE5 ? 57344.0f : 448.0f;  // largest finite value
    __device__ static __forceinline__ uint32_t code(float q)
    {
        return kE5 ? e5m2_code(q) : e4m3_code(q);
    }
    // hardware conversion of two fp32 values into bytes 0-1 (hi false) or
    // 2-3 (hi true) of `old`, round to nearest even
    __device__ static __forceinline__ int cvt_pk(float a, float b, int old, bool hi)
    {
        if constexpr (kE5)
            return hi ? __builtin_amdgcn_cvt_pk_bf8_f32(a, b, old, true)
                      : __builtin_amdgcn_cvt_pk_bf8_f32(a, b, old, false);
        else
            return hi ? __builtin_amdgcn_cvt_pk_fp8_f32(a, b, old, true)
                      : __builtin_amdgcn_cvt_pk_fp8_f32(a, b, old, false);
    }
};

// Correctly rounded a / s for a >= 0 and s in [2^-80, 2^100], given r, the
// reciprocal of s refined by one Newton step: two remainder corrections
// (Markstein), the unscaled form of the IEEE fp32 divide sequence.  No
// intermediate under- or overflows for quotients >= 2^-24; smaller quotients
// are only ever rounded to an 8-bit zero, which this result also gives.
__device__ __forceinline__ float quotient(float a, float s, float r)
{
    float q = a * r;
    float e = __builtin_fmaf(-s, q, a);
    q = __builtin_fmaf(e, r, q);
    e = __builtin_fmaf(-s, q, a);
    return __builtin_fmaf(e, r, q);
}

// a / s with one remainder correction, for the fast path's 8-bit codes.  Its
// result is not always the correctly rounded quotient, but its code always
// is that quotient's: the GPU test over every pair of finite 16-bit values
// (row maximum, element of no larger magnitude, both signs), bf16 and fp16
// sources, e4m3fn and e5m2 codes, finds every code equal to the oracle's,
// which rounds the exact quotient.  a may be negative: every step is odd in a
// (rounding to nearest is symmetric), and the residual is formed as s*q - a
// and subtracted, so a signed zero keeps its sign (q - (+0) * r is -0 for
// q = -0, where q + (+0) * r would be +0).
__device__ __forceinline__ float quotient_for_code(float a, float s, float r)
{
    const float q = a * r;
    return __builtin_fmaf(-__builtin_fmaf(s, q, -a), r, q);
}

// Maximum of m over each aligned group of 2^lg consecutive lanes (lg <= 6,
// wave-uniform).  Within a 16-lane DPP row the exchanges are VALU operands
// (quad_perm [1,0,3,2] and [2,3,0,1] pair lanes 1 and 2 apart; after those,
// row_half_mirror pairs the two quads of 8 lanes and row_mirror the two
// halves of 16), so no LDS permute and no wait is needed; wider groups (rows
// above 256 bytes) add xor shuffles.  Every lane of the wave must execute it.
__device__ __forceinline__ uint32_t group_max(uint32_t m, int lg)
{
    auto dpp = [](uint32_t v, auto ctrl) {
        return static_cast<uint32_t>(
            __builtin_amdgcn_update_dpp(0, static_cast<int>(v), decltype(ctrl)::value, 0xF, 0xF, false));
    };
    if (lg >= 1) m = max(m, dpp(m, std::integral_constant<int, 0xB1>{}));   // quad_perm 1,0,3,2
    if (lg >= 2) m = max(m, dpp(m, std::integral_constant<int, 0x4E>{}));   // quad_perm 2,3,0,1
    if (lg >= 3) m = max(m, dpp(m, std::integral_constant<int, 0x141>{}));  // row_half_mirror
    if (lg >= 4) m = max(m, dpp(m, std::integral_constant<int, 0x140>{}));  // row_mirror
    for (int o = 16; o < (1 << lg); o <<= 1)
        m = max(m, static_cast<uint32_t>(__shfl_xor(static_cast<int>(m), o)));
    return m;
}

// source format of a quantising conversion: fp16 or bf16
constexpr bool f16_source(int conv)
{
    return conv == kF16E4m3 || conv == kQdF16Bf16 || conv == kQdF16F16 || conv == kF16E5m2 ||
           conv == kQd5F16Bf16 || conv == kQd5F16F16;
}

// 8-bit format of a conversion that quantises or dequantises: e5m2, else e4m3fn
constexpr bool e5_conv(int conv)
{
    return conv == kBf16E5m2 || conv == kF16E5m2 || conv == kDq5Bf16 || conv == kDq5F16 ||
           conv == kQd5Bf16Bf16 || conv == kQd5F16Bf16 || conv == kQd5Bf16F16 ||
           conv == kQd5F16F16;
}

template <int CONV>
struct SrcFmt {
    static constexpr uint32_t kInf = f16_source(CONV) ? 0x7C00u : 0x7F80u;
    // 16-bit pattern (sign included) -> fp32, exactly
    __device__ static __forceinline__ float widen(uint32_t m)
    {
        if constexpr (f16_source(CONV))
            return static_cast<float>(
                __builtin_bit_cast(_Float16, static_cast<unsigned short>(m)));
        else
            return __uint_as_float(m << 16);
    }
};

// General path: one lane's 2*NW source elements (NW 32-bit words) -> 2*NW
// 8-bit codes, every case of the definition (NaN elements, zero rows, scales
// too small or too large for the two-step divide), element by element in
// software.  The row maximum is reduced over the lanes-per-row group (2^lg
// lanes, consecutive, so xor shuffles stay inside the group); every lane of the
// wave must execute the reduction.
template <int CONV, int NW>
__device__ __forceinline__ void fp8_codes_general(const uint32_t (&w)[NW], int lg,
                                                  float& scale_out, uint32_t (&out)[NW / 2])
{
    using F = SrcFmt<CONV>;
    using Q = Fp8<e5_conv(CONV)>;
    uint32_t m = 0;
#pragma unroll
    for (int k = 0; k < NW; ++k) {
        uint32_t lo = w[k] & 0x7FFFu, hi = (w[k] >> 16) & 0x7FFFu;
        lo = lo > F::kInf ? 0u : lo;  // NaN elements do not take part in the maximum
        hi = hi > F::kInf ? 0u : hi;
        m = max(m, max(lo, hi));
    }
    m = group_max(m, lg);
    const float amax = F::widen(m);
    const float s = amax / Q::kMax;  // IEEE divide
    scale_out = s;
    const bool fast = s >= 0x1p-80f && s <= 0x1p100f;
    const float r0 = __builtin_amdgcn_rcpf(s);
    const float r = __builtin_fmaf(__builtin_fmaf(-s, r0, 1.0f), r0, r0);
#pragma unroll
    for (int k = 0; k < NW / 2; ++k) out[k] = 0u;
#pragma unroll
    for (int k = 0; k < 2 * NW; ++k) {
        const uint32_t h = (w[k >> 1] >> ((k & 1) * 16)) & 0xFFFFu;
        const uint32_t mag = h & 0x7FFFu;
        uint32_t code;
        if (mag > F::kInf) {
            code = 0x7Fu;                       // NaN
        } else if (s == 0.0f) {
            code = 0u;                          // every finite element is zero
        } else if (fast) {
            code = Q::code(quotient(F::widen(mag), s, r));
        } else {
            const float q = F::widen(mag) / s;  // IEEE divide (tiny, huge or infinite scale)
            code = q != q ? 0x7Fu : Q::code(q);
        }
        out[k >> 2] |= (code | ((h >> 8) & 0x80u)) << ((k & 3) * 8);
    }
}

// One lane's 2*NW source elements -> 2*NW 8-bit codes.  Fast path for rows with
// no NaN and a scale in [2^-80, 2^100]: the row maximum from packed 16-bit
// maxima, the quotient x / s (quotient_for_code: the code of the exact
// quotient, sign included), and the hardware conversion
// v_cvt_pk_fp8_f32 / v_cvt_pk_bf8_f32 (round to nearest even, OCP e4m3fn and
// e5m2 on gfx950; they equal e4m3_code / e5m2_code on every fp32 magnitude up
// to 448 / 57344, and a quotient cannot round above those because |x| <=
// amax).  Other rows take the general path.  Every lane of the wave must
// execute this.
template <int CONV, int NW>
__device__ __forceinline__ void fp8_codes(const uint32_t (&w)[NW], int lg, float& scale_out,
                                          uint32_t (&out)[NW / 2])
{
    using F = SrcFmt<CONV>;
    using Q = Fp8<e5_conv(CONV)>;
    typedef unsigned short us2 __attribute__((ext_vector_type(2)));
    us2 mm = {0, 0};
#pragma unroll
    for (int k = 0; k < NW; ++k)  // magnitudes, NaN included
        mm = __builtin_elementwise_max(mm, __builtin_bit_cast(us2, w[k] & 0x7FFF7FFFu));
    uint32_t m = max(uint32_t(mm.x), uint32_t(mm.y));
    m = group_max(m, lg);
    // s = amax / fmax by the reciprocal and one remainder correction: equal
    // to the IEEE quotient for every 16-bit row maximum, and inside the fast
    // range exactly when the IEEE quotient is (the GPU test over every finite
    // bf16 and fp16 row maximum, both formats, compares each scale with the
    // oracle's IEEE quotient); NaN when the row holds a NaN or an infinity
    constexpr float kInv = 1.0f / Q::kMax;
    const float amax = F::widen(m);
    const float q0 = amax * kInv;
    const float s = __builtin_fmaf(__builtin_fmaf(-Q::kMax, q0, amax), kInv, q0);
    if (!(s >= 0x1p-80f && s <= 0x1p100f)) {
        fp8_codes_general<CONV, NW>(w, lg, scale_out, out);
        return;
    }
    scale_out = s;
    const float r0 = __builtin_amdgcn_rcpf(s);
    const float r = __builtin_fmaf(__builtin_fmaf(-s, r0, 1.0f), r0, r0);
#pragma unroll
    for (int d = 0; d < NW / 2; ++d) {  // output dword d = elements 4d .. 4d+3 = words 2d, 2d+1
        float q[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t h = (w[2 * d + (e >> 1)] >> ((e & 1) * 16)) & 0xFFFFu;
            q[e] = quotient_for_code(F::widen(h), s, r);  // the element's sign carried through
        }
        // bytes 2-3 of the first conversion's `old` operand are overwritten by
        // the second, so any register serves; q[0], dead after this
        // instruction, lets the result take its register (no copy of `old`)
        const int lo = Q::cvt_pk(q[0], q[1], __float_as_int(q[0]), false);
        out[d] = uint32_t(Q::cvt_pk(q[2], q[3], lo, true));
    }
}

// One lane's 16 source elements (two 16-byte vectors) -> 16 8-bit codes.
template <int CONV>
__device__ __forceinline__ uint4 to_fp8(const uint4 (&v)[2], int lg, float& scale_out)
{
    const uint32_t w[8] = {v[0].x, v[0].y, v[0].z, v[0].w, v[1].x, v[1].y, v[1].z, v[1].w};
    uint32_t out[4];
    fp8_codes<CONV, 8>(w, lg, scale_out, out);
    return make_uint4(out[0], out[1], out[2], out[3]);
}

// ---- dequantisation: 8-bit codes and a row scale -> 16-bit values -----------

// The product q * s is rounded to fp32 before its 16-bit conversion.  Left
// alone, the compiler folds the multiply and an f32 -> f16 conversion into
// one mixed-precision FMA (v_fma_mixlo_f16): that rounds the exact product
// once, straight to fp16, and adds +0, which drops the sign of a zero product.
// The empty asm makes the fp32 value opaque, so it is materialised as such.
template <typename T>
__device__ __forceinline__ T as_rounded(T v)
{
    __asm__("" : "+v"(v));
    return v;
}

// One code -> q * s rounded to the 16-bit format: the exact value of the code
// (e4m3fn: 3 fraction bits, bias 7, exponent field 0 subnormal, S.1111.111
// NaN; e5m2: 2 fraction bits, bias 15, exponent field 0 subnormal, all-ones
// exponent infinity (fraction 0) or NaN), one fp32 product, the conversion
// rounding to nearest even.  NaN codes and NaN products (0 * Inf) give the
// format's quiet NaN with the code's sign.
template <bool kBf16, bool kE5>
__device__ __forceinline__ uint32_t dequant1(uint32_t c, float s)
{
    const uint32_t sign = (c & 0x80u) << 8;
    const uint32_t qnan = kBf16 ? 0x7FC0u : 0x7E00u;
    float x;
    if constexpr (kE5) {
        const uint32_t e = (c >> 2) & 0x1Fu, m = c & 3u;
        if (e == 0x1Fu) {
            if (m) return sign | qnan;
            x = __builtin_inff();
        } else {
            x = e ? __builtin_ldexpf(float(4u + m), int(e) - 17) : float(m) * 0x1p-16f;
        }
    } else {
        const uint32_t e = (c >> 3) & 0xFu, m = c & 7u;
        if ((c & 0x7Fu) == 0x7Fu) return sign | qnan;
        x = e ? __builtin_ldexpf(float(8u + m), int(e) - 10) : float(m) * 0x1p-9f;
    }
    const float v = as_rounded((c & 0x80u ? -x : x) * s);
    if (v != v) return sign | qnan;
    if constexpr (kBf16)
        return __builtin_bit_cast(unsigned short, static_cast<__bf16>(v));
    else
        return __builtin_bit_cast(unsigned short, static_cast<_Float16>(v));
}

// Two codes (bytes 0-1 or 2-3 of a dword) -> their exact fp32 values, by the
// hardware decode (v_cvt_pk_f32_fp8 / v_cvt_pk_f32_bf8; finite codes only).
template <bool kE5, bool kHi>
__device__ __forceinline__ auto decode2(uint32_t c)
{
    if constexpr (kE5)
        return __builtin_amdgcn_cvt_pk_f32_bf8(int(c), kHi);
    else
        return __builtin_amdgcn_cvt_pk_f32_fp8(int(c), kHi);
}

// 8 codes (two dwords) -> 8 16-bit values.  Lanes whose codes are all finite
// and whose scale is finite: the hardware decode (exact), the fp32 product and
// the packed conversion; otherwise code by code.
template <bool kBf16, bool kE5>
__device__ __forceinline__ uint4 dequant8(uint32_t c0, uint32_t c1, float s)
{
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    // a byte that is not finite: e4m3fn (b & 0x7F) == 0x7F, exactly when
    // (b & 0x7F) + 1 sets bit 7; e5m2 (b & 0x7C) == 0x7C, exactly when
    // (b & 0x7C) + 4 sets bit 7 (no carry leaves the byte either way)
    const uint32_t mk = kE5 ? 0x7C7C7C7Cu : 0x7F7F7F7Fu, one = kE5 ? 0x04040404u : 0x01010101u;
    const uint32_t nan = (((c0 & mk) + one) | ((c1 & mk) + one)) & 0x80808080u;
    uint32_t o[4];
    if (!nan && __builtin_fabsf(s) <= 0x1.fffffep127f) {
        const f2 f[4] = {as_rounded(decode2<kE5, false>(c0) * s),
                         as_rounded(decode2<kE5, true>(c0) * s),
                         as_rounded(decode2<kE5, false>(c1) * s),
                         as_rounded(decode2<kE5, true>(c1) * s)};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if constexpr (kBf16)
                o[k] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f[k], b2));
            else
                o[k] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f[k], h2));
        }
    } else {
        const uint32_t c[2] = {c0, c1};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t w = c[k >> 1] >> ((k & 1) * 16);
            o[k] = dequant1<kBf16, kE5>(w & 0xFFu, s) |
                   (dequant1<kBf16, kE5>((w >> 8) & 0xFFu, s) << 16);
        }
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
}

// 8 fp16 -> 8 bf16.  Without NaN (the usual case): exact widening and the
// hardware v_cvt_pk_bf16_f32 (round to nearest even, the C semantics of a
// float -> bfloat conversion).  A NaN anywhere in the 8 sends them through
// f16_to_bf16, which fixes the NaN payload rule.
__device__ __forceinline__ uint4 to_bf16x8(const uint4& v)
{
    typedef unsigned short us2 __attribute__((ext_vector_type(2)));
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef __bf16 b2 __attribute__((ext_vector_type(2)));
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    us2 mm = {0, 0};
#pragma unroll
    for (int k = 0; k < 4; ++k)
        mm = __builtin_elementwise_max(mm, __builtin_bit_cast(us2, w[k] & 0x7FFF7FFFu));
    uint32_t o[4];
    if (max(uint32_t(mm.x), uint32_t(mm.y)) <= 0x7C00u) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const f2 f = __builtin_convertvector(__builtin_bit_cast(h2, w[k]), f2);
            o[k] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f, b2));
        }
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
            o[k] = f16_to_bf16(w[k] & 0xFFFFu) | (f16_to_bf16(w[k] >> 16) << 16);
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
}

// 8 bf16 -> 8 fp16.  Without NaN: exact widening to fp32 and the hardware
// fp32 -> fp16 conversion (round to nearest even, overflow to infinity, fp16
// subnormals kept).  A NaN anywhere in the 8 sends them element by element
// through the NaN rule: sign kept, quiet bit set, the 7 bf16 fraction bits at
// the top of the fp16 fraction; other elements take the same conversion.
__device__ __forceinline__ uint32_t bf16_to_f16(uint32_t b)
{
    if ((b & 0x7FFFu) > 0x7F80u) return (b & 0x8000u) | 0x7E00u | ((b & 0x7Fu) << 3);
    const _Float16 h = static_cast<_Float16>(__uint_as_float(b << 16));
    return __builtin_bit_cast(unsigned short, h);
}

__device__ __forceinline__ uint4 to_f16x8(const uint4& v)
{
    typedef unsigned short us2 __attribute__((ext_vector_type(2)));
    typedef float f2 __attribute__((ext_vector_type(2)));
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    us2 mm = {0, 0};
#pragma unroll
    for (int k = 0; k < 4; ++k)
        mm = __builtin_elementwise_max(mm, __builtin_bit_cast(us2, w[k] & 0x7FFF7FFFu));
    uint32_t o[4];
    if (max(uint32_t(mm.x), uint32_t(mm.y)) <= 0x7F80u) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const f2 f = {__uint_as_float(w[k] << 16), __uint_as_float(w[k] & 0xFFFF0000u)};
            o[k] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f, h2));
        }
    } else {
#pragma unroll
        for (int k = 0; k < 4; ++k)
            o[k] = bf16_to_f16(w[k] & 0xFFFFu) | (bf16_to_f16(w[k] >> 16) << 16);
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
}

// ---- the row kernel ----------------------------------------------------------

__device__ __forceinline__ uint32_t fdiv(uint32_t n, FastDiv f)
{
    return uint32_t((uint64_t(__umulhi(n, f.mul)) + n) >> f.shift);
}

// One 16-byte vector of a row that this launch reads once (source row or
// transfer-tensor row): a non-temporal load (global_load_dwordx4 ... nt), so
// the line is not kept in the caches at the expense of other data.
__device__ __forceinline__ uint4 load_stream(const char* p)
{
    typedef unsigned int v4u __attribute__((ext_vector_type(4)));
    const v4u v = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Read one dword at the start of the destination page of the unit
// kPrefetchPages pages after `unit` (same plane-major order), so that its
// address translation is cached before that page's workgroups store to it.
// The value is discarded; ids outside the pool are ignored.
__device__ __forceinline__ void warm_translation(const KArgs& a, uint32_t unit)
{
    const uint32_t fu = unit + uint32_t(kPrefetchPages) * a.parts * a.num_segs;
    if (fu >= a.units) return;
    const uint32_t page_unit = fdiv(fdiv(fu, a.div_parts), a.div_segs);
    const uint32_t plane = fdiv(page_unit, a.div_items) + a.dst_plane0;  // cache plane
    const Item it = a.items[page_unit - (plane - a.dst_plane0) * a.num_items];
    const int32_t b = a.bt[int64_t(it.req) * a.bt_stride + it.blk];
    if (b < 0 || b >= a.num_blocks) return;
    const volatile uint32_t* q = reinterpret_cast<const volatile uint32_t*>(
        static_cast<const char*>(a.dst) + plane * a.plane_bytes +
        int64_t(b) * a.block_size * a.hd * a.row_dst_bytes);
    (void)*q;
}

template <int MODE, int CONV, int ORDER>
__device__ __forceinline__ void convert_part(const KArgs& a)
{
    constexpr bool kFp8 = CONV == kBf16E4m3 || CONV == kF16E4m3 ||    // writes 8-bit codes
                          CONV == kBf16E5m2 || CONV == kF16E5m2;
    constexpr bool kQd = CONV == kQdBf16Bf16 || CONV == kQdF16Bf16 ||  // quantise + dequantise
                         CONV == kQdBf16F16 || CONV == kQdF16F16 || CONV == kQd5Bf16Bf16 ||
                         CONV == kQd5F16Bf16 || CONV == kQd5Bf16F16 || CONV == kQd5F16F16;
    constexpr bool kDq = CONV == kDq8Bf16 || CONV == kDq8F16 ||        // dequantising unpack
                         CONV == kDq5Bf16 || CONV == kDq5F16;
    constexpr bool kE5 = e5_conv(CONV);                                // e5m2 codes
    constexpr bool kQuant = kFp8 || kQd;                               // row maximum over lanes
    constexpr bool kScalesIn = CONV == kCopy8 || kDq;                  // unpack reads row scales
    constexpr bool kScales = kFp8 || CONV == kCopy8;                   // rows written with a scale
    constexpr bool kToBf16 = CONV == kDq8Bf16 || CONV == kQdBf16Bf16 || CONV == kQdF16Bf16 ||
                             CONV == kDq5Bf16 || CONV == kQd5Bf16Bf16 || CONV == kQd5F16Bf16;
    // Lanes follow the transfer-tensor row: lane `sub` of a row owns its 16-byte
    // chunk sub.  A dequantising lane owns the 16 codes of chunk sub and writes
    // them as the two 16-byte cache chunks sub and sub + cpr (and reads, for
    // the repack, the source chunks at the same places), so each load and
    // each store instruction covers one contiguous half row.
    constexpr bool kHalves = kDq || kQd;
    constexpr int kVecs = (kFp8 || kQd) ? 2 : 1;              // 16-byte loads per lane
    constexpr int kSrcEsz = CONV == kCopy8 ? 1 : 2;
    constexpr int kLaneElems = (kFp8 || CONV == kCopy8) ? 16 : 8;  // at the lane's first load
    static_assert(!kDq || MODE == kUnpack, "dequantisation reads the transfer tensor");
    static_assert(!kQd || MODE == kRepack, "quantise + dequantise is a repack");
    // Issue order.  "Early": the page lookups are scalar loads issued before
    // any lane-dependent branch and every lane issues its row load
    // unconditionally (lanes without a row read the buffer's first vector), so
    // the lookups, the row loads and the paged source's page lookup overlap
    // instead of following one another.  Measured faster for repacks from
    // paged sources (+16%) and 16-bit token-major rows (+2%); the head-major
    // and 8-bit paths measure 2-4% faster with the row load inside the
    // branch, and the pack from paged sources the same either way.
    constexpr bool kEarly =
        (ORDER == KVX_PAGED && MODE != kPack) ||
        (ORDER == KVX_THD && (CONV == kCopy16 || CONV == kF16Bf16 || CONV == kBf16F16));

    // XCD-contiguous unit of this workgroup -> (plane, page, segment, part)
    const uint32_t unit = (blockIdx.x % kXcds) * a.units_per_xcd + blockIdx.x / kXcds;
    if (unit >= a.units) return;  // the grid is rounded up to a multiple of kXcds
    const uint32_t q1 = fdiv(unit, a.div_parts);
    const uint32_t part = unit - q1 * a.parts;
    const uint32_t q2 = fdiv(q1, a.div_segs);
    const uint32_t sg = q1 - q2 * a.num_segs;
    const uint32_t plane = fdiv(q2, a.div_items);           // layer * 2 + k/v
    const uint32_t item = q2 - plane * a.num_items;
    if (plane >= a.planes || item >= a.num_items || sg >= a.num_segs || part >= a.parts) return;
    const Segment seg = a.seg[sg];
    const Item it = a.items[item];
    const int T = it.tokens;
    const int t0 = it.blk * a.block_size;
    const int seg_rows = min(a.block_size, T - t0) * seg.n;
    const int64_t row0 = (int64_t(plane) * T + t0) * a.hd;  // first row in transfer-tensor order
    const int lg = a.lg_lpr;

    int32_t b = 0;  // destination page (unpack, repack)
    if constexpr (kEarly && MODE != kPack) b = a.bt[int64_t(it.req) * a.bt_stride + it.blk];
    // Paged source whose parts never span two source pages: one page per
    // workgroup, looked up once (the part's first token must exist).
    int32_t sb_u = -1;
    uint32_t q_u = 0;
    if constexpr (ORDER == KVX_PAGED && MODE != kUnpack) {
        if (a.sbt_uniform) {
            const uint32_t tf = uint32_t(t0) + fdiv(part * uint32_t(kThreads >> lg), seg.div_n);
            if (tf < uint32_t(T)) {
                q_u = fdiv(tf, a.div_sbs);
                sb_u = a.sbt[int64_t(it.req) * a.sbt_stride + q_u];
            }
        }
    }

    const int sub = threadIdx.x & ((1 << lg) - 1);          // 16-byte chunk within the row
    const int r = int(part) * (kThreads >> lg) + (threadIdx.x >> lg);  // row within the segment
    int s, ii;  // token within the page, head within the segment
    bool ok;
    if constexpr (ORDER == KVX_HTD && MODE != kUnpack) {
        // head-major rows: consecutive lane groups read consecutive tokens of one
        // head, contiguous in a [head][token][dim] source
        ii = int(fdiv(uint32_t(r), a.div_bs));
        s = r - ii * a.block_size;
        ok = sub < a.cpr && ii < seg.n && s < seg_rows / seg.n;
    } else {
        s = int(fdiv(uint32_t(r), seg.div_n));
        ii = r - s * seg.n;
        ok = sub < a.cpr && r < seg_rows;
    }
    const int row = s * a.hd + seg.i0 + ii;                 // row within the page

    // source address of this lane's row (meaningful where ok)
    const char* base;
    const char* p = nullptr;
    const float* sp = nullptr;
    if constexpr (MODE == kUnpack) {
        base = static_cast<const char*>(a.wire_in);
        // a dequantising lane reads 8 codes at sub * 8 and 8 at (sub + cpr) * 8
        p = base + it.wire_data + (row0 + row) * a.row_wire_bytes + sub * (kDq ? 8 : 16);
        if constexpr (kScalesIn)
            sp = reinterpret_cast<const float*>(base + it.wire_scale) + row0 + row;
    } else {
        base = static_cast<const char*>(a.src[seg.slot]);
        const int h = seg.h0 + ii;                           // head within the shard
        int64_t e = 0;
        if constexpr (ORDER == KVX_THD) {
            e = (int64_t(plane + a.src_plane0) * T + t0 + s) * a.hs + h;
        } else if constexpr (ORDER == KVX_HTD) {
            e = (int64_t(plane + a.src_plane0) * a.hs + h) * T + t0 + s;
        } else {
            // the prefill side's own page of this token; a row whose page id
            // lies outside the source pool is neither read nor written
            const uint32_t t = uint32_t(t0 + s);
            int32_t sb = sb_u;
            uint32_t q = q_u;
            if (!a.sbt_uniform && ok) {
                q = fdiv(t, a.div_sbs);
                sb = a.sbt[int64_t(it.req) * a.sbt_stride + q];
            }
            ok = ok && sb >= 0 && sb < a.src_num_blocks;
            e = ((int64_t(plane + a.src_plane0) * a.src_num_blocks + sb) * a.src_block_size +
                 int64_t(t - q * uint32_t(a.src_block_size))) * a.hs + h;
        }
        p = base + (it.src_base + e * a.head_dim) * kSrcEsz + sub * (kLaneElems * kSrcEsz);
    }

    // byte distance from a lane's first load to its second
    const int second = kHalves ? a.cpr * (kDq ? 8 : 16) : 16;
    uint4 v[kVecs];
    float sc = 0.0f;
    if constexpr (kEarly) {
        // lanes without a row read the buffer's first vector (valid, cached)
        const char* pl = ok ? p : base;
        if constexpr (kDq) {
            const uint2 c0 = *reinterpret_cast<const uint2*>(pl);
            const uint2 c1 = *reinterpret_cast<const uint2*>(pl + (ok ? second : 0));
            v[0] = make_uint4(c0.x, c0.y, c1.x, c1.y);
        } else {
#pragma unroll
            for (int k = 0; k < kVecs; ++k)
                v[k] = load_stream(pl + (ok ? k * second : 0));
        }
        if constexpr (MODE == kUnpack && kScalesIn)
            sc = *(ok ? sp : reinterpret_cast<const float*>(base));
        // keep the loads here: the compiler would otherwise sink them below
        // the destination-page check, behind the scalar lookups
        __asm__ volatile("" ::: "memory");
        if constexpr (kQuant)
#pragma unroll
            for (int k = 0; k < kVecs; ++k)  // rows without data take part in the maximum as zeros
                if (!ok) v[k] = make_uint4(0u, 0u, 0u, 0u);
    } else {
#pragma unroll
        for (int k = 0; k < kVecs; ++k) v[k] = make_uint4(0u, 0u, 0u, 0u);
        if (ok) {
            if constexpr (kDq) {
                const uint2 c0 = *reinterpret_cast<const uint2*>(p);
                const uint2 c1 = *reinterpret_cast<const uint2*>(p + second);
                v[0] = make_uint4(c0.x, c0.y, c1.x, c1.y);
            } else {
#pragma unroll
                for (int k = 0; k < kVecs; ++k)
                    v[k] = load_stream(p + k * second);
            }
            if constexpr (MODE == kUnpack && kScalesIn)
                if (kDq || sub == 0) sc = *sp;  // every dequantising lane needs the scale
        }
        if constexpr (MODE != kPack) b = a.bt[int64_t(it.req) * a.bt_stride + it.blk];
    }

    char* dbase;
    float* sbase = nullptr;
    if constexpr (MODE == kPack) {
        dbase = static_cast<char*>(a.dst) + it.wire_data + row0 * a.row_dst_bytes;
        if constexpr (kScales)
            sbase = reinterpret_cast<float*>(static_cast<char*>(a.dst) + it.wire_scale) + row0;
    } else {
        if (part == 0 && sg == 0 && threadIdx.x == 0) warm_translation(a, unit);
        if (b < 0 || b >= a.num_blocks) return;  // not a page of the pool: nothing written
        const int64_t page_rows = int64_t(b) * a.block_size * a.hd;
        const uint32_t cplane = plane + a.dst_plane0;  // the cache's own layer
        dbase = static_cast<char*>(a.dst) + cplane * a.plane_bytes + page_rows * a.row_dst_bytes;
        if constexpr (kScales) sbase = a.dscale + cplane * a.plane_scales + page_rows;
    }

    uint4 out, out2;  // out2: a dequantising lane's second cache chunk
    if constexpr (kFp8) {
        out = to_fp8<CONV>(v, lg, sc);  // every lane takes part in the row reduction
    } else if constexpr (kQd) {
        const uint32_t w[8] = {v[0].x, v[0].y, v[0].z, v[0].w, v[1].x, v[1].y, v[1].z, v[1].w};
        uint32_t c[4];
        fp8_codes<CONV, 8>(w, lg, sc, c);  // every lane takes part in the row reduction
        out = dequant8<kToBf16, kE5>(c[0], c[1], sc);
        out2 = dequant8<kToBf16, kE5>(c[2], c[3], sc);
    } else if constexpr (kDq) {
        out = dequant8<kToBf16, kE5>(v[0].x, v[0].y, sc);
        out2 = dequant8<kToBf16, kE5>(v[0].z, v[0].w, sc);
    } else if constexpr (CONV == kF16Bf16)
        out = to_bf16x8(v[0]);
    else if constexpr (CONV == kBf16F16)
        out = to_f16x8(v[0]);
    else
        out = v[0];
    if (ok) {
        typedef unsigned int v4u __attribute__((ext_vector_type(4)));
        char* drow = dbase + int64_t(row) * a.row_dst_bytes;
        __builtin_nontemporal_store(__builtin_bit_cast(v4u, out),
                                    reinterpret_cast<v4u*>(drow + sub * 16));
        if constexpr (kHalves)
            __builtin_nontemporal_store(__builtin_bit_cast(v4u, out2),
                                        reinterpret_cast<v4u*>(drow + (sub + a.cpr) * 16));
        if constexpr (kScales && !kFp8)  // the 8-bit unpack: the scale it loaded
            if (sub == 0) __builtin_nontemporal_store(sc, sbase + row);
    }
    if constexpr (kFp8) {
        // The quantising launches' 4-byte row scales go out through LDS: lane
        // 0 of each row leaves its scale and destination slot there, and after
        // the barrier the first lanes of wave 0 store them all, so a
        // workgroup's 32 or so consecutive scales leave as one store
        // instruction covering whole cache lines instead of four 32-byte
        // pieces, one per wave.  Ordinary stores here: the L2 merges them into
        // whole lines.  Measured 2% faster on the fp8 decode cache than
        // non-temporal per-row stores; the 8-bit unpack, whose scales arrive
        // by a load rather than from the lanes' own arithmetic, measured 8%
        // slower this way and keeps the per-row store.
        __shared__ float lds_scale[kThreads];
        __shared__ int lds_slot[kThreads];  // the row's index in sbase, -1: not written
        if (sub == 0) {
            lds_scale[threadIdx.x >> lg] = sc;
            lds_slot[threadIdx.x >> lg] = ok ? row : -1;
        }
        __syncthreads();
        if (int(threadIdx.x) < (kThreads >> lg)) {
            const int slot = lds_slot[threadIdx.x];
            if (slot >= 0) sbase[slot] = lds_scale[threadIdx.x];
        }
    }
}

// One kernel name per operation, so traces tell them apart.
template <int CONV, int ORDER>
__global__ void __launch_bounds__(kThreads) kvx_pack_kernel(const KArgs a)
{
    convert_part<kPack, CONV, ORDER>(a);
}

template <int CONV, int ORDER>
__global__ void __launch_bounds__(kThreads) kvx_unpack_kernel(const KArgs a)
{
    convert_part<kUnpack, CONV, ORDER>(a);
}

template <int CONV, int ORDER>
__global__ void __launch_bounds__(kThreads) kvx_repack_kernel(const KArgs a)
{
    convert_part<kRepack, CONV, ORDER>(a);
}

template <int MODE, int CONV, int ORDER>
int go(const KArgs& a, void* stream)
{
    const void* fn;
    if constexpr (MODE == kPack)
        fn = reinterpret_cast<const void*>(&kvx_pack_kernel<CONV, ORDER>);
    else if constexpr (MODE == kUnpack)
        fn = reinterpret_cast<const void*>(&kvx_unpack_kernel<CONV, ORDER>);
    else
        fn = reinterpret_cast<const void*>(&kvx_repack_kernel<CONV, ORDER>);
    void* args[] = {const_cast<KArgs*>(&a)};
    const unsigned grid = a.units_per_xcd * kXcds;
    return int(hipLaunchKernel(fn, dim3(grid), dim3(kThreads), args, 0,
                               static_cast<hipStream_t>(stream)));
}

template <int MODE, int ORDER>
int go_conv(int conv, const KArgs& a, void* stream)
{
    switch (conv) {
    case kCopy16: return go<MODE, kCopy16, ORDER>(a, stream);
    case kF16Bf16: return go<MODE, kF16Bf16, ORDER>(a, stream);
    case kBf16F16: return go<MODE, kBf16F16, ORDER>(a, stream);
    case kBf16E4m3: return go<MODE, kBf16E4m3, ORDER>(a, stream);
    case kF16E4m3: return go<MODE, kF16E4m3, ORDER>(a, stream);
    case kBf16E5m2: return go<MODE, kBf16E5m2, ORDER>(a, stream);
    case kF16E5m2: return go<MODE, kF16E5m2, ORDER>(a, stream);
    default: break;
    }
    if constexpr (MODE == kRepack) {
        switch (conv) {
        case kQdBf16Bf16: return go<MODE, kQdBf16Bf16, ORDER>(a, stream);
        case kQdF16Bf16: return go<MODE, kQdF16Bf16, ORDER>(a, stream);
        case kQdBf16F16: return go<MODE, kQdBf16F16, ORDER>(a, stream);
        case kQdF16F16: return go<MODE, kQdF16F16, ORDER>(a, stream);
        case kQd5Bf16Bf16: return go<MODE, kQd5Bf16Bf16, ORDER>(a, stream);
        case kQd5F16Bf16: return go<MODE, kQd5F16Bf16, ORDER>(a, stream);
        case kQd5Bf16F16: return go<MODE, kQd5Bf16F16, ORDER>(a, stream);
        case kQd5F16F16: return go<MODE, kQd5F16F16, ORDER>(a, stream);
        default: break;
        }
    }
    return int(hipErrorInvalidValue);
}

// ---- the work-item table of the allocation-free repack ---------------------

// One workgroup: prefix sums of the pages and tokens of the requests (one
// thread, at most kNoAllocRequests terms), then every thread writes items
// idx = tid, tid + 256, ...: the request whose pages cover idx is the last one
// whose first page is <= idx (requests without pages share their first page
// with the next request and are skipped by that rule).  The source offset of a
// request is its preceding tokens times the elements of one token.
__global__ void __launch_bounds__(kThreads) kvx_items_kernel(const ItemsArgs a)
{
    __shared__ int32_t first[kNoAllocRequests + 1];
    __shared__ int64_t before[kNoAllocRequests + 1];
    const int R = a.num_requests;
    if (threadIdx.x == 0) {
        first[0] = 0;
        before[0] = 0;
        for (int r = 0; r < R; ++r) {
            first[r + 1] = first[r] + (a.lens[r] + a.block_size - 1) / a.block_size;
            before[r + 1] = before[r] + a.lens[r];
        }
    }
    __syncthreads();
    const int n = first[R];
    for (int idx = threadIdx.x; idx < n; idx += kThreads) {
        int lo = 0, hi = R - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) / 2;
            if (first[mid] <= idx) lo = mid;
            else hi = mid - 1;
        }
        Item it;
        it.src_base = before[lo] * a.src_elems_per_token;
        it.wire_data = 0;
        it.wire_scale = -1;
        it.req = lo;
        it.blk = idx - first[lo];
        it.tokens = a.lens[lo];
        it.pad = 0;
        a.items[idx] = it;
    }
}

}  // namespace

// Per device, for the calls that cannot allocate: their work-item table.
// Every call on a device rewrites it, so calls that overlap on one device
// race.  Host code never uses this name as an address: scratch_items() looks
// the device address up.
static __device__ __align__(256) Item scratch[kNoAllocItems];

int scratch_items(Item** out)
{
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static Item* table[kMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return int(e);
    if (dev < 0 || dev >= kMaxDevices) return int(hipErrorInvalidDevice);
    std::lock_guard<std::mutex> lock(mu);
    if (!table[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return int(e);
        table[dev] = static_cast<Item*>(p);
    }
    *out = table[dev];
    return int(hipSuccess);
}

int build_items(const ItemsArgs& a, void* stream)
{
    void* args[] = {const_cast<ItemsArgs*>(&a)};
    return int(hipLaunchKernel(reinterpret_cast<const void*>(&kvx_items_kernel), dim3(1),
                               dim3(kThreads), args, 0, static_cast<hipStream_t>(stream)));
}

int launch(int mode, int conv, int order, const KArgs& a, void* stream)
{
    if (mode == kUnpack) {
        if (conv == kCopy16) return go<kUnpack, kCopy16, KVX_THD>(a, stream);
        if (conv == kCopy8) return go<kUnpack, kCopy8, KVX_THD>(a, stream);
        if (conv == kDq8Bf16) return go<kUnpack, kDq8Bf16, KVX_THD>(a, stream);
        if (conv == kDq8F16) return go<kUnpack, kDq8F16, KVX_THD>(a, stream);
        if (conv == kDq5Bf16) return go<kUnpack, kDq5Bf16, KVX_THD>(a, stream);
        if (conv == kDq5F16) return go<kUnpack, kDq5F16, KVX_THD>(a, stream);
        return int(hipErrorInvalidValue);
    }
    if (mode == kPack) {
        if (order == KVX_THD) return go_conv<kPack, KVX_THD>(conv, a, stream);
        if (order == KVX_HTD) return go_conv<kPack, KVX_HTD>(conv, a, stream);
        return go_conv<kPack, KVX_PAGED>(conv, a, stream);
    }
    if (order == KVX_THD) return go_conv<kRepack, KVX_THD>(conv, a, stream);
    if (order == KVX_HTD) return go_conv<kRepack, KVX_HTD>(conv, a, stream);
    return go_conv<kRepack, KVX_PAGED>(conv, a, stream);
}

}  // namespace kvx
