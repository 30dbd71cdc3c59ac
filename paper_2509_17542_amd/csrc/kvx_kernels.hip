// gfx950 kernels of the KV-cache conversion: pack (source shards -> transfer
// tensor), unpack (transfer tensor -> paged cache) and the fused repack
// (source shards -> paged cache).
//
// Work decomposition: one workgroup per work unit = (logical page of a
// request, (layer, k/v) plane).  Units are numbered plane-major, so
// consecutive units read consecutive source bytes.  The 1-D grid is dealt to
// the 8 XCDs round-robin (workgroup i runs on XCD i % 8); workgroup i is mapped
// to unit (i % 8) * units_per_xcd + i / 8, so every XCD streams one contiguous
// run of units through its own L2 instead of every eighth page of the whole
// stream.  A page holds ntok <= block_size tokens x Hd heads = "rows" of
// head_dim elements, contiguous in both the paged cache and the transfer
// tensor.  Each row is covered by a power-of-two group of lanes, one 16-byte
// destination vector per lane (global_load_dwordx4 / global_store_dwordx4); a
// workgroup walks its rows in passes of threads / lanes-per-row rows and keeps
// U rows of loads in flight per lane before the first store.
//
// The path is a gather/scatter stream with no reuse and no contraction: it is
// bound by HBM bandwidth, so there is no MFMA and no LDS staging (every row is
// at least 128 contiguous bytes, i.e. whole cache lines on both sides, so a
// [token][head] <-> [head][token] reorder is a change of row addresses only).
#include <hip/hip_runtime.h>

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

// Correctly rounded a / s for a >= 0 and s in [2^-80, 2^100], given r, the
// reciprocal of s refined by one Newton step: two remainder corrections
// (Markstein), the unscaled form of the IEEE fp32 divide sequence.  No
// intermediate under- or overflows for quotients >= 2^-24; smaller quotients
// are only ever rounded to e4m3fn zero, which this result also gives.
__device__ __forceinline__ float quotient(float a, float s, float r)
{
    float q = a * r;
    float e = __builtin_fmaf(-s, q, a);
    q = __builtin_fmaf(e, r, q);
    e = __builtin_fmaf(-s, q, a);
    return __builtin_fmaf(e, r, q);
}

template <int CONV>
struct SrcFmt {
    static constexpr uint32_t kInf = CONV == kF16E4m3 ? 0x7C00u : 0x7F80u;
    // magnitude bits (sign cleared) -> fp32
    __device__ static __forceinline__ float widen(uint32_t m)
    {
        if constexpr (CONV == kF16E4m3)
            return static_cast<float>(
                __builtin_bit_cast(_Float16, static_cast<unsigned short>(m)));
        else
            return __uint_as_float(m << 16);
    }
};

// One lane's 16 source elements (two 16-byte vectors) -> 16 e4m3fn bytes.
// The row maximum is reduced over the lanes-per-row group (2^lg lanes,
// consecutive, so xor shuffles stay inside the group); every lane of the
// wave must execute this.
template <int CONV>
__device__ __forceinline__ uint4 to_e4m3(const uint4 (&v)[2], int lg, float& scale_out)
{
    using F = SrcFmt<CONV>;
    const uint32_t w[8] = {v[0].x, v[0].y, v[0].z, v[0].w, v[1].x, v[1].y, v[1].z, v[1].w};
    uint32_t m = 0;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        uint32_t lo = w[k] & 0x7FFFu, hi = (w[k] >> 16) & 0x7FFFu;
        lo = lo > F::kInf ? 0u : lo;  // NaN elements do not take part in the maximum
        hi = hi > F::kInf ? 0u : hi;
        m = max(m, max(lo, hi));
    }
    for (int o = 1; o < (1 << lg); o <<= 1)
        m = max(m, static_cast<uint32_t>(__shfl_xor(static_cast<int>(m), o)));
    const float amax = F::widen(m);
    const float s = amax / 448.0f;  // IEEE divide
    scale_out = s;
    const bool fast = s >= 0x1p-80f && s <= 0x1p100f;
    const float r0 = __builtin_amdgcn_rcpf(s);
    const float r = __builtin_fmaf(__builtin_fmaf(-s, r0, 1.0f), r0, r0);
    uint32_t out[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const uint32_t h = (w[k >> 1] >> ((k & 1) * 16)) & 0xFFFFu;
        const uint32_t mag = h & 0x7FFFu;
        uint32_t code;
        if (mag > F::kInf) {
            code = 0x7Fu;                       // NaN
        } else if (s == 0.0f) {
            code = 0u;                          // every finite element is zero
        } else if (fast) {
            code = e4m3_code(quotient(F::widen(mag), s, r));
        } else {
            const float q = F::widen(mag) / s;  // IEEE divide (tiny, huge or infinite scale)
            code = q != q ? 0x7Fu : e4m3_code(q);
        }
        out[k >> 2] |= (code | ((h >> 8) & 0x80u)) << ((k & 3) * 8);
    }
    return make_uint4(out[0], out[1], out[2], out[3]);
}

__device__ __forceinline__ uint4 to_bf16x8(const uint4& v)
{
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
        o[k] = f16_to_bf16(w[k] & 0xFFFFu) | (f16_to_bf16(w[k] >> 16) << 16);
    return make_uint4(o[0], o[1], o[2], o[3]);
}

// ---- the row kernel ----------------------------------------------------------

template <int MODE, int CONV, int ORDER, int THREADS, int U>
__device__ __forceinline__ void convert_rows(const KArgs& a)
{
    constexpr bool kFp8 = CONV == kBf16E4m3 || CONV == kF16E4m3;
    constexpr bool kScales = kFp8 || CONV == kCopy8;
    constexpr int kVecs = kFp8 ? 2 : 1;                       // 16-byte loads per lane per row
    constexpr int kSrcEsz = CONV == kCopy8 ? 1 : 2;
    constexpr int kLaneElems = (kFp8 || CONV == kCopy8) ? 16 : 8;

    // XCD-contiguous unit of this workgroup, then (plane, page)
    const int unit = int(blockIdx.x % kXcds) * a.units_per_xcd + int(blockIdx.x / kXcds);
    if (unit >= a.units) return;  // the grid is rounded up to a multiple of kXcds
    const int plane = unit / a.num_items;                    // layer * 2 + k/v
    const Item it = a.items[unit - plane * a.num_items];
    const int T = it.tokens;
    const int t0 = it.blk * a.block_size;
    const int rows = min(a.block_size, T - t0) * a.hd;
    const int64_t row0 = (int64_t(plane) * T + t0) * a.hd;  // first row in transfer-tensor order

    char* dbase;
    float* sbase = nullptr;
    int32_t b = 0;
    if constexpr (MODE == kPack) {
        dbase = static_cast<char*>(a.dst) + it.wire_data + row0 * a.row_dst_bytes;
        if constexpr (kScales)
            sbase = reinterpret_cast<float*>(static_cast<char*>(a.dst) + it.wire_scale) + row0;
    } else {
        b = a.bt[int64_t(it.req) * a.bt_stride + it.blk];
        const int64_t page_rows = int64_t(b) * a.block_size * a.hd;
        dbase = static_cast<char*>(a.dst) + plane * a.plane_bytes + page_rows * a.row_dst_bytes;
        if constexpr (kScales) sbase = a.dscale + plane * a.plane_scales + page_rows;
    }

    const int lg = a.lg_lpr;
    const int sub = threadIdx.x & ((1 << lg) - 1);          // 16-byte chunk within the row
    const int r0 = threadIdx.x >> lg;                        // first row of this lane group
    const int rpp = THREADS >> lg;                           // rows per pass
    const bool lane_ok = sub < a.cpr;
    int s = r0 / a.hd;                                       // token within the page
    int i = r0 - s * a.hd;                                   // decode head

    for (int pass = 0; pass < rows; pass += U * rpp) {      // uniform over the workgroup
        uint4 v[U][kVecs];
        float sc_in[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int row = pass + u * rpp + r0;
#pragma unroll
            for (int k = 0; k < kVecs; ++k) v[u][k] = make_uint4(0u, 0u, 0u, 0u);
            sc_in[u] = 0.0f;
            if (lane_ok && row < rows) {
                const char* p;
                if constexpr (MODE == kUnpack) {
                    p = static_cast<const char*>(a.wire_in) + it.wire_data +
                        (row0 + row) * a.row_dst_bytes;
                    if constexpr (kScales)
                        if (sub == 0)
                            sc_in[u] = reinterpret_cast<const float*>(
                                static_cast<const char*>(a.wire_in) + it.wire_scale)[row0 + row];
                } else {
                    const uint32_t hs = a.head_src[i];
                    const int h = int(hs & 0xFFFFu);
                    int64_t e;
                    if constexpr (ORDER == KVX_THD)
                        e = (int64_t(plane) * T + t0 + s) * a.hs + h;
                    else
                        e = (int64_t(plane) * a.hs + h) * T + t0 + s;
                    p = static_cast<const char*>(a.src[hs >> 16]) +
                        (it.src_base + e * a.head_dim) * kSrcEsz;
                }
                p += sub * (kLaneElems * kSrcEsz);
#pragma unroll
                for (int k = 0; k < kVecs; ++k) v[u][k] = reinterpret_cast<const uint4*>(p)[k];
            }
            s += a.dq;
            i += a.dr;
            if (i >= a.hd) {
                i -= a.hd;
                ++s;
            }
        }
        if constexpr (MODE != kPack)
            if (b < 0 || b >= a.num_blocks) return;  // not a page of the pool: nothing written
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int row = pass + u * rpp + r0;
            const bool ok = lane_ok && row < rows;
            uint4 out;
            float sc = sc_in[u];
            if constexpr (kFp8)
                out = to_e4m3<CONV>(v[u], lg, sc);
            else if constexpr (CONV == kF16Bf16)
                out = to_bf16x8(v[u][0]);
            else
                out = v[u][0];
            if (ok) {
                *reinterpret_cast<uint4*>(dbase + int64_t(row) * a.row_dst_bytes + sub * 16) = out;
                if constexpr (kScales)
                    if (sub == 0) sbase[row] = sc;
            }
        }
    }
}

// One kernel name per operation, so traces tell them apart.
template <int CONV, int ORDER, int THREADS, int U>
__global__ void __launch_bounds__(THREADS) kvx_pack_kernel(const KArgs a)
{
    convert_rows<kPack, CONV, ORDER, THREADS, U>(a);
}

template <int CONV, int ORDER, int THREADS, int U>
__global__ void __launch_bounds__(THREADS) kvx_unpack_kernel(const KArgs a)
{
    convert_rows<kUnpack, CONV, ORDER, THREADS, U>(a);
}

template <int CONV, int ORDER, int THREADS, int U>
__global__ void __launch_bounds__(THREADS) kvx_repack_kernel(const KArgs a)
{
    convert_rows<kRepack, CONV, ORDER, THREADS, U>(a);
}

template <int CONV>
struct Shape {
    static constexpr bool kFp8 = CONV == kBf16E4m3 || CONV == kF16E4m3;
    // 16-bit rows: 512 threads, 4 rows of 16-byte loads in flight per lane;
    // e4m3fn rows (two 16-byte loads per lane and row, VALU-heavy): 256 x 4
    static constexpr int kThreads = kFp8 ? 256 : 512;
    static constexpr int kU = 4;
};

template <int MODE, int CONV, int ORDER>
int go(const KArgs& a, void* stream)
{
    using S = Shape<CONV>;
    const void* fn;
    if constexpr (MODE == kPack)
        fn = reinterpret_cast<const void*>(&kvx_pack_kernel<CONV, ORDER, S::kThreads, S::kU>);
    else if constexpr (MODE == kUnpack)
        fn = reinterpret_cast<const void*>(&kvx_unpack_kernel<CONV, ORDER, S::kThreads, S::kU>);
    else
        fn = reinterpret_cast<const void*>(&kvx_repack_kernel<CONV, ORDER, S::kThreads, S::kU>);
    void* args[] = {const_cast<KArgs*>(&a)};
    const unsigned grid = unsigned(a.units_per_xcd) * kXcds;
    return int(hipLaunchKernel(fn, dim3(grid), dim3(S::kThreads), args, 0,
                               static_cast<hipStream_t>(stream)));
}

template <int MODE, int ORDER>
int go_conv(int conv, const KArgs& a, void* stream)
{
    switch (conv) {
    case kCopy16: return go<MODE, kCopy16, ORDER>(a, stream);
    case kF16Bf16: return go<MODE, kF16Bf16, ORDER>(a, stream);
    case kBf16E4m3: return go<MODE, kBf16E4m3, ORDER>(a, stream);
    case kF16E4m3: return go<MODE, kF16E4m3, ORDER>(a, stream);
    default: return int(hipErrorInvalidValue);
    }
}

}  // namespace

int threads_for(int conv)
{
    switch (conv) {
    case kBf16E4m3: return Shape<kBf16E4m3>::kThreads;
    case kF16E4m3: return Shape<kF16E4m3>::kThreads;
    case kCopy8: return Shape<kCopy8>::kThreads;
    case kF16Bf16: return Shape<kF16Bf16>::kThreads;
    default: return Shape<kCopy16>::kThreads;
    }
}

int launch(int mode, int conv, int order, const KArgs& a, void* stream)
{
    if (mode == kUnpack) {
        if (conv == kCopy16) return go<kUnpack, kCopy16, KVX_THD>(a, stream);
        if (conv == kCopy8) return go<kUnpack, kCopy8, KVX_THD>(a, stream);
        return int(hipErrorInvalidValue);
    }
    if (mode == kPack)
        return order == KVX_THD ? go_conv<kPack, KVX_THD>(conv, a, stream)
                                : go_conv<kPack, KVX_HTD>(conv, a, stream);
    return order == KVX_THD ? go_conv<kRepack, KVX_THD>(conv, a, stream)
                            : go_conv<kRepack, KVX_HTD>(conv, a, stream);
}

}  // namespace kvx
