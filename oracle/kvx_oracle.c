/*
 * kvx_oracle.c -- plain CPU oracle of the KV-cache conversion performed by the
 * heterogeneous compatible transmission module (paper Sec. III-B).
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the test suite, the smoke check and the
 * benchmark's CPU-baseline leg, never by the GPU library.
 *
 * What is computed, and where it comes from:
 *   - parallel-strategy alignment (Sec. III-B-3 and Fig. 4): a decode rank's
 *     heads are one contiguous range of the global KV heads, and the prefill
 *     ranks that overlap that range are merged (src TP > dst TP) or split
 *     (src TP < dst TP), as in the TP=4 -> TP=2 example of that subsection;
 *   - VRAM-management alignment (Sec. III-B-2 and Fig. 5): the prefill side's
 *     layout is flattened into a one-dimensional transfer tensor and then
 *     restored into the decode side's paged cache with its own page (block)
 *     size and layout;
 *   - precision alignment (named among the module's components in Sec. I):
 *     the decode side's element type.  The paper gives no rounding rule; the
 *     reading taken is IEEE round-to-nearest-even, and for the 8-bit
 *     formats (e4m3fn, e5m2) a per-(token, head) scale max|x| / (the
 *     format's largest finite value) in fp32 with a saturating cast.
 *
 * Casts are written from the format definitions: decode the bits to an exact
 * real value (double), round that value to the nearest point of the target
 * grid with ties to even, encode.  No bit tricks.
 *
 * Build: plain C99, no fast-math, no contraction (-ffp-contract=off), so the
 * one fp32 divide of the e4m3 path is the IEEE correctly rounded divide.
 */
#include "kvx_oracle.h"

#include <fenv.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ */
/* formats                                                              */
/* ------------------------------------------------------------------ */

typedef struct {
    int total_bits;  /* storage width */
    int exp_bits;
    int man_bits;    /* stored fraction bits */
    int bias;
} orc_fmt_desc;

static orc_fmt_desc fmt_desc(int fmt)
{
    orc_fmt_desc f;
    switch (fmt) {
    case ORC_FP16:   f.total_bits = 16; f.exp_bits = 5; f.man_bits = 10; f.bias = 15;  break;
    case ORC_BF16:   f.total_bits = 16; f.exp_bits = 8; f.man_bits = 7;  f.bias = 127; break;
    case ORC_E5M2:   f.total_bits = 8;  f.exp_bits = 5; f.man_bits = 2;  f.bias = 15;  break;
    default:         f.total_bits = 8;  f.exp_bits = 4; f.man_bits = 3;  f.bias = 7;   break;
    }
    return f;
}

int orc_is_fp8(int fmt) { return fmt == ORC_E4M3FN || fmt == ORC_E5M2; }

int orc_fmt_size(int fmt) { return orc_is_fp8(fmt) ? 1 : 2; }

/* Exact value of an encoded number.  IEEE-style formats (fp16, bf16 and OCP
 * e5m2): all-ones exponent is Inf (zero fraction) or NaN.  OCP e4m3fn: no
 * Inf; only S.1111.111 is NaN, and exponent field 15 with other fractions is
 * finite. */
double orc_decode(int fmt, uint32_t bits)
{
    orc_fmt_desc f = fmt_desc(fmt);
    uint32_t sign = (bits >> (f.total_bits - 1)) & 1u;
    uint32_t e = (bits >> f.man_bits) & ((1u << f.exp_bits) - 1u);
    uint32_t m = bits & ((1u << f.man_bits) - 1u);
    uint32_t emax_field = (1u << f.exp_bits) - 1u;
    double v;
    if (fmt == ORC_E4M3FN) {
        if (e == emax_field && m == ((1u << f.man_bits) - 1u))
            return sign ? -NAN : NAN;
    } else if (e == emax_field) {
        if (m != 0) return sign ? -NAN : NAN;
        return sign ? -INFINITY : INFINITY;
    }
    if (e == 0) /* subnormal: m * 2^(1 - bias - man_bits) */
        v = ldexp((double)m, 1 - f.bias - f.man_bits);
    else        /* normal: (2^man_bits + m) * 2^(e - bias - man_bits) */
        v = ldexp((double)((1u << f.man_bits) + m), (int)e - f.bias - f.man_bits);
    return sign ? -v : v;
}

/* Round a >= 0 (finite, exact in double) to the nearest point of the grid of
 * a binary format with `p` significand bits and minimum normal exponent
 * `emin`; ties go to the point with an even last significand bit.  The grid
 * spacing in the binade [2^E, 2^(E+1)) is 2^(E-p+1); below 2^emin it is the
 * subnormal spacing 2^(emin-p+1). */
static double rne_to_grid(double a, int p, int emin)
{
    int e;
    if (a == 0.0) return 0.0;
    (void)frexp(a, &e);          /* a in [2^(e-1), 2^e) */
    int E = e - 1;
    if (E < emin) E = emin;
    double spacing = ldexp(1.0, E - (p - 1));
    double n = a / spacing;      /* exact: power-of-two scaling */
    double r = nearbyint(n);     /* default mode: round half to even */
    return r * spacing;          /* exact */
}

/* Encode a magnitude that lies on the grid (and within the finite range)
 * with the given sign. */
static uint32_t encode(int fmt, uint32_t sign, double mag)
{
    orc_fmt_desc f = fmt_desc(fmt);
    int emin = 1 - f.bias;
    uint32_t s = sign << (f.total_bits - 1);
    if (mag == 0.0) return s;
    int e;
    (void)frexp(mag, &e);
    int E = e - 1;
    if (E < emin) { /* subnormal: exponent field 0, fraction = mag / 2^(emin - man_bits) */
        double frac = ldexp(mag, -(emin - f.man_bits));
        return s | (uint32_t)frac;
    }
    double frac = ldexp(mag, -(E - f.man_bits)) - ldexp(1.0, f.man_bits);
    return s | ((uint32_t)(E + f.bias) << f.man_bits) | (uint32_t)frac;
}

/* bf16 -> fp16.  Finite values: round the exact value to the fp16 grid (11
 * significand bits, emin = -14), ties to even; a rounded magnitude above the
 * largest finite fp16 (65504) overflows to infinity, as IEEE rounding to
 * nearest does.  Infinities stay infinite.  NaN (reading taken, as for fp16 ->
 * bf16): keep the sign, set the quiet bit, put the 7 bf16 fraction bits at
 * the top of the fp16 fraction. */
uint16_t orc_bf16_to_fp16(uint16_t b)
{
    uint32_t sign = (b >> 15) & 1u;
    double x = orc_decode(ORC_BF16, b);
    if (isnan(x))
        return (uint16_t)((sign << 15) | 0x7C00u | 0x0200u | ((b & 0x7Fu) << 3));
    if (isinf(x))
        return (uint16_t)((sign << 15) | 0x7C00u);
    double m = rne_to_grid(fabs(x), 11, -14);
    if (m > 65504.0)
        return (uint16_t)((sign << 15) | 0x7C00u);
    return (uint16_t)encode(ORC_FP16, sign, m);
}

/* float -> fp16 / bf16, round to nearest even; magnitudes that round above
 * the format's largest finite value become infinite. */
static uint16_t f32_to_16(int fmt, float v, uint32_t nan_sign)
{
    int bf = fmt == ORC_BF16;
    uint32_t sign = signbit(v) ? 1u : 0u;
    if (isnan(v))
        return (uint16_t)((nan_sign << 15) | (bf ? 0x7FC0u : 0x7E00u));
    if (isinf(v))
        return (uint16_t)((sign << 15) | (bf ? 0x7F80u : 0x7C00u));
    double m = bf ? rne_to_grid(fabs((double)v), 8, -126) : rne_to_grid(fabs((double)v), 11, -14);
    double maxf = bf ? ldexp(255.0, 120) : 65504.0;      /* (2 - 2^-7) 2^127, (2 - 2^-10) 2^15 */
    if (m > maxf)
        return (uint16_t)((sign << 15) | (bf ? 0x7F80u : 0x7C00u));
    return (uint16_t)encode(fmt, sign, m);
}

/* Dequantisation (reading R25): q * s as one fp32 product (round to nearest
 * even), then rounded to the cache format.  A NaN code, or a NaN product
 * (0 * Inf in a row whose scale is infinite), gives the quiet NaN with the
 * code's sign. */
void orc_dequant_row(int code_fmt, int cache_fmt, int D, const uint8_t *q, float s,
                     uint16_t *out)
{
    for (int d = 0; d < D; ++d) {
        uint32_t sign = (q[d] >> 7) & 1u;
        float x = (float)orc_decode(code_fmt, q[d]);      /* exact (or +-Inf / NaN) */
        float v = x * s;                                   /* fp32 product */
        out[d] = f32_to_16(cache_fmt, isnan(x) ? NAN : v, sign);
    }
}

/* fp16 -> bf16.  Finite values and infinities: round the exact value to the
 * bf16 grid (8 significand bits, emin = -126), ties to even; no fp16 value
 * can overflow bf16.  NaN (paper silent; reading taken): keep the sign, set
 * the quiet bit, keep the top 7 fraction bits of the fp16 payload. */
uint16_t orc_fp16_to_bf16(uint16_t h)
{
    uint32_t sign = (h >> 15) & 1u;
    double x = orc_decode(ORC_FP16, h);
    if (isnan(x))
        return (uint16_t)((sign << 15) | 0x7F80u | 0x0040u | ((h & 0x03FFu) >> 3));
    if (isinf(x))
        return (uint16_t)((sign << 15) | 0x7F80u);
    double m = rne_to_grid(fabs(x), 8, -126);
    return (uint16_t)encode(ORC_BF16, sign, m);
}

/* fp32 -> OCP e4m3fn, round to nearest even, saturating: any magnitude whose
 * rounding would exceed 448 (the largest finite value) gives +-448.  NaN gives
 * the NaN code S.1111.111 with the sign kept. */
uint8_t orc_f32_to_e4m3fn(float v)
{
    uint32_t sign = signbit(v) ? 1u : 0u;
    if (isnan(v)) return (uint8_t)((sign << 7) | 0x7Fu);
    double a = fabs((double)v);
    if (a >= 448.0) return (uint8_t)encode(ORC_E4M3FN, sign, 448.0);
    double m = rne_to_grid(a, 4, -6);
    if (m > 448.0) m = 448.0; /* unreachable: a < 448 and 448 is a grid point */
    return (uint8_t)encode(ORC_E4M3FN, sign, m);
}

/* fp32 -> OCP e5m2 (1 sign, 5 exponent bits with bias 15, 2 fraction bits;
 * largest finite value 57344 = 1.75 * 2^15, subnormals m * 2^-16), round to
 * nearest even, saturating like the e4m3fn cast (reading R26): a magnitude
 * whose rounding would exceed 57344, an infinity included, gives +-57344.
 * NaN gives S.11111.11 with the sign kept. */
uint8_t orc_f32_to_e5m2(float v)
{
    uint32_t sign = signbit(v) ? 1u : 0u;
    if (isnan(v)) return (uint8_t)((sign << 7) | 0x7Fu);
    double a = fabs((double)v);
    if (a >= 57344.0) return (uint8_t)encode(ORC_E5M2, sign, 57344.0);
    double m = rne_to_grid(a, 3, -14);
    if (m > 57344.0) m = 57344.0; /* unreachable: a < 57344 and 57344 is a grid point */
    return (uint8_t)encode(ORC_E5M2, sign, m);
}

/* Per-row scale: the largest magnitude over the row (NaN elements ignored),
 * divided by fmax, the 8-bit format's largest finite value, with one IEEE
 * fp32 divide. */
float orc_row_scale_to(const float *x, int n, float fmax)
{
    float amax = 0.0f;
    for (int d = 0; d < n; ++d) {
        if (isnan(x[d])) continue;
        float a = fabsf(x[d]);
        if (a > amax) amax = a;
    }
    return amax / fmax;
}

float orc_row_scale(const float *x, int n) { return orc_row_scale_to(x, n, 448.0f); }

void orc_f32_to_e5m2_n(const float *in, uint8_t *out, int64_t n)
{
    for (int64_t k = 0; k < n; ++k) out[k] = orc_f32_to_e5m2(in[k]);
}

void orc_bf16_to_fp16_n(const uint16_t *in, uint16_t *out, int64_t n)
{
    for (int64_t k = 0; k < n; ++k) out[k] = orc_bf16_to_fp16(in[k]);
}

void orc_fp16_to_bf16_n(const uint16_t *in, uint16_t *out, int64_t n)
{
    for (int64_t k = 0; k < n; ++k) out[k] = orc_fp16_to_bf16(in[k]);
}

void orc_f32_to_e4m3fn_n(const float *in, uint8_t *out, int64_t n)
{
    for (int64_t k = 0; k < n; ++k) out[k] = orc_f32_to_e4m3fn(in[k]);
}

void orc_decode_n(int fmt, const void *in, double *out, int64_t n)
{
    for (int64_t k = 0; k < n; ++k) {
        uint32_t b = orc_is_fp8(fmt) ? ((const uint8_t *)in)[k] : ((const uint16_t *)in)[k];
        out[k] = orc_decode(fmt, b);
    }
}

void orc_convert_row(int src_fmt, int dst_fmt, int D, const void *src_row, void *dst_row,
                     float *scale)
{
    const uint16_t *s = (const uint16_t *)src_row;
    if (src_fmt == dst_fmt) {               /* same type: bits unchanged */
        memcpy(dst_row, src_row, (size_t)D * (size_t)orc_fmt_size(src_fmt));
        return;
    }
    if (src_fmt == ORC_FP16 && dst_fmt == ORC_BF16) {
        uint16_t *o = (uint16_t *)dst_row;
        for (int d = 0; d < D; ++d) o[d] = orc_fp16_to_bf16(s[d]);
        return;
    }
    if (src_fmt == ORC_BF16 && dst_fmt == ORC_FP16) {
        uint16_t *o = (uint16_t *)dst_row;
        for (int d = 0; d < D; ++d) o[d] = orc_bf16_to_fp16(s[d]);
        return;
    }
    /* 16-bit float -> e4m3fn or e5m2 with a per-row fp32 scale */
    int e5 = dst_fmt == ORC_E5M2;
    float *x = (float *)calloc((size_t)D, sizeof(float));
    uint8_t *o = (uint8_t *)dst_row;
    if (!x) abort();
    for (int d = 0; d < D; ++d) x[d] = (float)orc_decode(src_fmt, s[d]); /* exact widening */
    float sc = orc_row_scale_to(x, D, e5 ? 57344.0f : 448.0f);
    *scale = sc;
    for (int d = 0; d < D; ++d) {
        uint32_t sign = (s[d] >> 15) & 1u;
        if (isnan(x[d]))
            o[d] = (uint8_t)((sign << 7) | 0x7Fu);
        else if (sc == 0.0f)                /* all finite elements are zero */
            o[d] = (uint8_t)(sign << 7);
        else {
            float v = x[d] / sc;
            /* An invalid quotient (Inf / Inf, in a row whose maximum is
             * infinite) has no defined sign; it takes the element's sign, as
             * every other quotient does (the scale is positive). */
            o[d] = isnan(v) ? (uint8_t)((sign << 7) | 0x7Fu)
                            : (e5 ? orc_f32_to_e5m2(v) : orc_f32_to_e4m3fn(v));
        }
    }
    free(x);
}

/* ------------------------------------------------------------------ */
/* index maps                                                          */
/* ------------------------------------------------------------------ */

int32_t orc_src_layers(const orc_problem *p) { return p->src_layers ? p->src_layers : p->layers; }
int32_t orc_cache_fmt(const orc_problem *p) { return p->cache_fmt ? p->cache_fmt : p->dst_fmt; }
int32_t orc_dst_layers(const orc_problem *p) { return p->dst_layers ? p->dst_layers : p->layers; }

int orc_validate(const orc_problem *p)
{
    if (!p) return -1;
    if (p->layers <= 0 || p->heads <= 0 || p->head_dim <= 0) return -1;
    /* the converted layers must lie inside both sides' layer ranges */
    if (p->src_layers < 0 || p->dst_layers < 0 || p->src_layer_offset < 0 ||
        p->dst_layer_offset < 0)
        return -1;
    if ((int64_t)p->src_layer_offset + p->layers > orc_src_layers(p)) return -1;
    if ((int64_t)p->dst_layer_offset + p->layers > orc_dst_layers(p)) return -1;
    if (p->src_tp <= 0 || p->dst_tp <= 0) return -1;
    /* each rank holds H / tp heads, or (tp a multiple of H) one replicated head */
    if (p->heads % p->src_tp != 0 && p->src_tp % p->heads != 0) return -1;
    if (p->heads % p->dst_tp != 0 && p->dst_tp % p->heads != 0) return -1;
    if (p->dst_rank < 0 || p->dst_rank >= p->dst_tp) return -1;
    if (p->block_size <= 0 || p->num_blocks <= 0) return -1;
    if (p->num_requests < 0 || (p->num_requests > 0 && !p->seq_lens)) return -1;
    for (int r = 0; r < p->num_requests; ++r)
        if (p->seq_lens[r] < 0) return -1;
    if (p->src_order != ORC_TOKEN_MAJOR && p->src_order != ORC_HEAD_MAJOR &&
        p->src_order != ORC_PAGED)
        return -1;
    if (p->src_order == ORC_PAGED) {
        if (p->src_block_size <= 0 || p->src_num_blocks <= 0) return -1;
        for (int r = 0; r < p->num_requests; ++r) {
            int64_t nb = ((int64_t)p->seq_lens[r] + p->src_block_size - 1) / p->src_block_size;
            if (nb > 0 && (!p->src_block_table || p->src_bt_stride < nb)) return -1;
        }
    }
    int sf = p->src_fmt, df = p->dst_fmt, cf = orc_cache_fmt(p);
    if (sf != ORC_FP16 && sf != ORC_BF16) return -2;
    /* a cache format other than the transfer format: only the dequantising
     * unpack of 8-bit codes (e4m3fn, e5m2) into fp16 / bf16 */
    if (cf != df && !(orc_is_fp8(df) && (cf == ORC_FP16 || cf == ORC_BF16))) return -2;
    if (sf == df) return 0;
    if (sf == ORC_FP16 && df == ORC_BF16) return 0;
    if (sf == ORC_BF16 && df == ORC_FP16) return 0;
    if (orc_is_fp8(df)) return 0;
    return -2;
}

/* Heads per rank.  With tp <= H a rank holds H / tp consecutive heads; with
 * tp a multiple of H every head is replicated on tp / H consecutive ranks and
 * a rank holds one head. */
int32_t orc_src_heads(const orc_problem *p)
{
    return p->src_tp <= p->heads ? p->heads / p->src_tp : 1;
}
int32_t orc_dst_heads(const orc_problem *p)
{
    return p->dst_tp <= p->heads ? p->heads / p->dst_tp : 1;
}

/* Decode-side head i of rank dst_rank is global head g = dst_rank*Hd + i (or,
 * replicated, g = dst_rank / (dst_tp / H)).  The prefill shard holding it is
 * g / Hs at local position g % Hs; replicated, the first of its replicas,
 * shard g * (src_tp / H), local position 0. */
void orc_head_source(const orc_problem *p, int i, int *shard, int *head)
{
    int H = p->heads;
    int g = p->dst_tp <= H ? p->dst_rank * (H / p->dst_tp) + i : p->dst_rank / (p->dst_tp / H);
    if (p->src_tp <= H) {
        int Hs = H / p->src_tp;
        *shard = g / Hs;
        *head = g % Hs;
    } else {
        *shard = g * (p->src_tp / H);
        *head = 0;
    }
}

/* Requests are stored back to back in every shard buffer, each one as
 * [layer][k/v][...Hs heads x T tokens...][dim]. */
int64_t orc_src_request_base(const orc_problem *p, int r)
{
    int64_t Hs = orc_src_heads(p);
    int64_t base = 0;
    if (p->src_order == ORC_PAGED) return 0; /* pages, not back-to-back requests */
    for (int q = 0; q < r; ++q)
        base += (int64_t)orc_src_layers(p) * 2 * p->seq_lens[q] * Hs * p->head_dim;
    return base;
}

/* element index of (r, l, kv, t, i, d) in its shard buffer, given the start
 * `base` of request r in that buffer */
static int64_t src_index_from(const orc_problem *p, int64_t base, int r, int l, int kv, int t,
                              int i, int d, int *shard)
{
    int j, h;
    orc_head_source(p, i, &j, &h);
    *shard = j;
    int64_t Hs = orc_src_heads(p);
    int64_t T = p->seq_lens[r];
    int64_t D = p->head_dim;
    int64_t plane = ((int64_t)p->src_layer_offset + l) * 2 + kv; /* in the source's layers */
    if (p->src_order == ORC_PAGED) {
        /* the prefill side's paged cache: token t sits in page
         * src_block_table[r][t / src_block_size], slot t % src_block_size */
        int64_t blk = p->src_block_table[(int64_t)r * p->src_bt_stride + t / p->src_block_size];
        int64_t slot = t % p->src_block_size;
        if (blk < 0 || blk >= p->src_num_blocks) return -1;
        return (((plane * p->src_num_blocks + blk) * p->src_block_size + slot) * Hs + h) * D + d;
    }
    if (p->src_order == ORC_TOKEN_MAJOR)
        return base + ((plane * T + t) * Hs + h) * D + d;
    return base + ((plane * Hs + h) * T + t) * D + d;
}

int64_t orc_src_index(const orc_problem *p, int r, int l, int kv, int t, int i, int d, int *shard)
{
    return src_index_from(p, orc_src_request_base(p, r), r, l, kv, t, i, d, shard);
}

/* decode-side paged cache: [layer][k/v][block][slot][Hd][dim] */
int64_t orc_cache_index(const orc_problem *p, int64_t block, int l, int kv, int slot, int i, int d)
{
    int64_t Hd = orc_dst_heads(p);
    int64_t plane = ((int64_t)p->dst_layer_offset + l) * 2 + kv; /* in the cache's layers */
    return (((plane * p->num_blocks + block) * p->block_size + slot) * Hd + i) * p->head_dim + d;
}

/* decode-side scales: [layer][k/v][block][slot][Hd] */
int64_t orc_cache_scale_index(const orc_problem *p, int64_t block, int l, int kv, int slot, int i)
{
    int64_t Hd = orc_dst_heads(p);
    int64_t plane = ((int64_t)p->dst_layer_offset + l) * 2 + kv;
    return ((plane * p->num_blocks + block) * p->block_size + slot) * Hd + i;
}

static int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }

/* Transfer tensor: request-major segments, each starting on a 256-byte
 * boundary; a segment is [layer][k/v][token][Hd][dim] in the destination type,
 * then (8-bit formats only) [layer][k/v][token][Hd] fp32 scales on the next 256-byte
 * boundary.  Returns the total size in bytes. */
int64_t orc_wire_layout(const orc_problem *p, int64_t *data_off, int64_t *scale_off)
{
    int64_t Hd = orc_dst_heads(p);
    int64_t esz = orc_fmt_size(p->dst_fmt);
    int64_t off = 0;
    for (int r = 0; r < p->num_requests; ++r) {
        int64_t rows = (int64_t)p->layers * 2 * p->seq_lens[r] * Hd;
        off = align256(off);
        if (data_off) data_off[r] = off;
        off += rows * p->head_dim * esz;
        if (orc_is_fp8(p->dst_fmt)) {
            off = align256(off);
            if (scale_off) scale_off[r] = off;
            off += rows * 4;
        } else if (scale_off) {
            scale_off[r] = -1;
        }
    }
    return align256(off);
}

/* Gather source row (r, l, kv, t, i) element by element and convert it.
 * Returns 0, writing nothing, when the row has no source (a source page id
 * outside the source pool). */
static int source_row_converted(const orc_problem *p, const void *const *shards, int64_t base,
                                int r, int l, int kv, int t, int i, uint16_t *tmp, void *out_row,
                                float *scale)
{
    for (int d = 0; d < p->head_dim; ++d) {
        int j;
        int64_t idx = src_index_from(p, base, r, l, kv, t, i, d, &j);
        if (idx < 0) return 0;
        tmp[d] = ((const uint16_t *)shards[j])[idx];
    }
    orc_convert_row(p->src_fmt, p->dst_fmt, p->head_dim, tmp, out_row, scale);
    return 1;
}

int orc_pack(const orc_problem *p, const void *const *shards, void *wire)
{
    int rc = orc_validate(p);
    if (rc) return rc;
    int Hd = orc_dst_heads(p), D = p->head_dim;
    int64_t esz = orc_fmt_size(p->dst_fmt);
    int64_t *doff = (int64_t *)malloc(sizeof(int64_t) * (size_t)(p->num_requests + 1));
    int64_t *soff = (int64_t *)malloc(sizeof(int64_t) * (size_t)(p->num_requests + 1));
    uint16_t *tmp = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)D);
    orc_wire_layout(p, doff, soff);
    uint8_t *w = (uint8_t *)wire;
    for (int r = 0; r < p->num_requests; ++r) {
        int T = p->seq_lens[r];
        int64_t base = orc_src_request_base(p, r);
        for (int l = 0; l < p->layers; ++l)
            for (int kv = 0; kv < 2; ++kv)
                for (int t = 0; t < T; ++t)
                    for (int i = 0; i < Hd; ++i) {
                        int64_t row = (((int64_t)l * 2 + kv) * T + t) * Hd + i;
                        float sc = 0.0f;
                        if (source_row_converted(p, shards, base, r, l, kv, t, i, tmp,
                                                 w + doff[r] + row * D * esz, &sc) &&
                            orc_is_fp8(p->dst_fmt))
                            memcpy(w + soff[r] + row * 4, &sc, 4);
                    }
    }
    free(doff); free(soff); free(tmp);
    return 0;
}

int orc_unpack(const orc_problem *p, const void *wire, void *cache, float *scales,
               const int32_t *block_table, int32_t bt_stride)
{
    int rc = orc_validate(p);
    if (rc) return rc;
    int Hd = orc_dst_heads(p), D = p->head_dim, bs = p->block_size;
    int64_t esz = orc_fmt_size(p->dst_fmt);
    int cf = orc_cache_fmt(p);
    int64_t cesz = orc_fmt_size(cf);
    int64_t *doff = (int64_t *)malloc(sizeof(int64_t) * (size_t)(p->num_requests + 1));
    int64_t *soff = (int64_t *)malloc(sizeof(int64_t) * (size_t)(p->num_requests + 1));
    orc_wire_layout(p, doff, soff);
    const uint8_t *w = (const uint8_t *)wire;
    uint8_t *c = (uint8_t *)cache;
    for (int r = 0; r < p->num_requests; ++r) {
        int T = p->seq_lens[r];
        for (int l = 0; l < p->layers; ++l)
            for (int kv = 0; kv < 2; ++kv)
                for (int t = 0; t < T; ++t) {
                    int64_t b = block_table[(int64_t)r * bt_stride + t / bs];
                    int slot = t % bs;
                    if (b < 0 || b >= p->num_blocks) continue;  /* not a page of the pool */
                    for (int i = 0; i < Hd; ++i) {
                        int64_t row = (((int64_t)l * 2 + kv) * T + t) * Hd + i;
                        if (cf != p->dst_fmt) {   /* dequantise the row */
                            float sc;
                            memcpy(&sc, w + soff[r] + row * 4, 4);
                            orc_dequant_row(p->dst_fmt, cf, D, w + doff[r] + row * D * esz, sc,
                                            (uint16_t *)(c + orc_cache_index(p, b, l, kv, slot, i, 0) * cesz));
                            continue;
                        }
                        memcpy(c + orc_cache_index(p, b, l, kv, slot, i, 0) * esz,
                               w + doff[r] + row * D * esz, (size_t)(D * esz));
                        if (orc_is_fp8(p->dst_fmt))
                            memcpy(&scales[orc_cache_scale_index(p, b, l, kv, slot, i)],
                                   w + soff[r] + row * 4, 4);
                    }
                }
    }
    free(doff); free(soff);
    return 0;
}

int orc_repack(const orc_problem *p, const void *const *shards, void *cache, float *scales,
               const int32_t *block_table, int32_t bt_stride)
{
    int rc = orc_validate(p);
    if (rc) return rc;
    int Hd = orc_dst_heads(p), D = p->head_dim, bs = p->block_size;
    int64_t esz = orc_fmt_size(p->dst_fmt);
    int cf = orc_cache_fmt(p);
    uint16_t *tmp = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)D);
    uint8_t *q = (uint8_t *)malloc((size_t)D);
    uint8_t *c = (uint8_t *)cache;
    for (int r = 0; r < p->num_requests; ++r) {
        int T = p->seq_lens[r];
        int64_t base = orc_src_request_base(p, r);
        for (int l = 0; l < p->layers; ++l)
            for (int kv = 0; kv < 2; ++kv)
                for (int t = 0; t < T; ++t) {
                    int64_t b = block_table[(int64_t)r * bt_stride + t / bs];
                    int slot = t % bs;
                    if (b < 0 || b >= p->num_blocks) continue;  /* not a page of the pool */
                    for (int i = 0; i < Hd; ++i) {
                        float sc = 0.0f;
                        if (cf != p->dst_fmt) {   /* quantise, then dequantise into the cache */
                            if (source_row_converted(p, shards, base, r, l, kv, t, i, tmp, q, &sc))
                                orc_dequant_row(p->dst_fmt, cf, D, q, sc,
                                                (uint16_t *)(c + orc_cache_index(p, b, l, kv, slot, i, 0) * 2));
                            continue;
                        }
                        if (source_row_converted(p, shards, base, r, l, kv, t, i, tmp,
                                                 c + orc_cache_index(p, b, l, kv, slot, i, 0) * esz,
                                                 &sc) &&
                            orc_is_fp8(p->dst_fmt))
                            scales[orc_cache_scale_index(p, b, l, kv, slot, i)] = sc;
                    }
                }
    }
    free(tmp);
    free(q);
    return 0;
}

int orc_expected_rows(const orc_problem *p, const void *const *shards, int r, int l, int kv,
                      int t0, int nt, void *out_rows, float *out_scales)
{
    int rc = orc_validate(p);
    if (rc) return rc;
    if (r < 0 || r >= p->num_requests || l < 0 || l >= p->layers || kv < 0 || kv > 1) return -1;
    if (t0 < 0 || nt < 0 || t0 + nt > p->seq_lens[r]) return -1;
    int Hd = orc_dst_heads(p), D = p->head_dim;
    int64_t esz = orc_fmt_size(p->dst_fmt);
    int cf = orc_cache_fmt(p);
    uint16_t *tmp = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)D);
    uint8_t *q = (uint8_t *)malloc((size_t)D);
    uint8_t *o = (uint8_t *)out_rows;
    int64_t base = orc_src_request_base(p, r);
    for (int t = t0; t < t0 + nt; ++t)
        for (int i = 0; i < Hd; ++i) {
            int64_t row = (int64_t)(t - t0) * Hd + i;
            float sc = 0.0f;
            if (cf != p->dst_fmt) {
                if (source_row_converted(p, shards, base, r, l, kv, t, i, tmp, q, &sc))
                    orc_dequant_row(p->dst_fmt, cf, D, q, sc, (uint16_t *)(o + row * D * 2));
                continue;
            }
            if (source_row_converted(p, shards, base, r, l, kv, t, i, tmp, o + row * D * esz, &sc) &&
                orc_is_fp8(p->dst_fmt) && out_scales)
                out_scales[row] = sc;
        }
    free(tmp);
    free(q);
    return 0;
}
