/*
 * kvx_oracle.h -- plain, slow CPU oracle for the KV-cache conversion of the
 * heterogeneous compatible transmission module (Sec. III-B of the paper:
 * precision alignment, VRAM-management alignment and parallel-strategy
 * alignment).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load this library.  It shares no code,
 * header, table or constant with the GPU library, and the GPU library never
 * calls it.
 *
 * Everything here is written from the plain definition of the result: nested
 * loops over (request, layer, k/v, token, head, dim), index maps written out
 * one formula per coordinate, and casts computed on exact real values in
 * double precision (decode -> round to the target grid -> encode).
 */
#ifndef KVX_ORACLE_H
#define KVX_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* element formats */
enum { ORC_FP16 = 1, ORC_BF16 = 2, ORC_E4M3FN = 3, ORC_E5M2 = 4 };
/* source storage orders: one (layer, k/v) plane of a request stored
 * contiguously, or the prefill side's own paged cache */
enum {
    ORC_TOKEN_MAJOR = 0, /* request r: [layer][k/v][token][head][dim] */
    ORC_HEAD_MAJOR = 1,  /* request r: [layer][k/v][head][token][dim] */
    ORC_PAGED = 2        /* shard pool [layer][k/v][src_num_blocks][src_block_size][head][dim],
                            token t of request r in page src_block_table[r][t / src_block_size] */
};

typedef struct {
    int32_t layers;      /* L */
    int32_t heads;       /* H, global KV heads */
    int32_t head_dim;    /* D */
    int32_t src_tp;      /* tensor-parallel degree of the prefill side */
    int32_t dst_tp;      /* tensor-parallel degree of the decode side */
    int32_t dst_rank;    /* which decode rank's head shard is produced */
    int32_t src_fmt;     /* ORC_FP16 or ORC_BF16 */
    int32_t dst_fmt;     /* ORC_FP16, ORC_BF16, ORC_E4M3FN or ORC_E5M2 */
    int32_t src_order;   /* ORC_TOKEN_MAJOR or ORC_HEAD_MAJOR */
    int32_t block_size;  /* tokens per destination page */
    int64_t num_blocks;  /* pages in the destination pool (per plane) */
    int32_t num_requests;
    const int32_t *seq_lens; /* [num_requests], tokens per request */
    /* ORC_PAGED sources only (ignored otherwise): the prefill side's pages */
    int32_t src_block_size;
    int64_t src_num_blocks;
    const int32_t *src_block_table; /* [num_requests][src_bt_stride] */
    int32_t src_bt_stride;
    /* Pipeline stages (layer ranges): the source buffers hold src_layers
     * layers and converted layer l is their layer src_layer_offset + l; the
     * cache holds dst_layers layers and layer l goes to its layer
     * dst_layer_offset + l.  0 layers means `layers` (offsets then 0). */
    int32_t src_layer_offset, src_layers;
    int32_t dst_layer_offset, dst_layers;
    /* Element format of the decode cache; 0 means dst_fmt.  A 16-bit cache
     * under an 8-bit dst_fmt is a dequantising unpack: the transfer tensor
     * carries 8-bit codes and scales, the cache their values q * s. */
    int32_t cache_fmt;
} orc_problem;

/* ---- casts (precision alignment) ---- */
double   orc_decode(int fmt, uint32_t bits);             /* exact value; NaN/Inf as such */
uint16_t orc_fp16_to_bf16(uint16_t h);                   /* IEEE round-to-nearest-even */
uint16_t orc_bf16_to_fp16(uint16_t b);                   /* RNE; overflow to +-Inf */
/* one row of 8-bit codes (e4m3fn or e5m2) back to a 16-bit format: each
 * value q * s (fp32 product), rounded to nearest even; NaN codes and NaN
 * products give the format's quiet NaN with the code's sign */
void     orc_dequant_row(int code_fmt, int cache_fmt, int D, const uint8_t *q, float s,
                         uint16_t *out);
int32_t  orc_cache_fmt(const orc_problem *p);
void     orc_bf16_to_fp16_n(const uint16_t *in, uint16_t *out, int64_t n);
uint8_t  orc_f32_to_e4m3fn(float v);                     /* RNE, saturating to +-448 */
uint8_t  orc_f32_to_e5m2(float v);                       /* RNE, saturating to +-57344 */
float    orc_row_scale(const float *x, int n);           /* max|x| / 448, fp32 divide */
float    orc_row_scale_to(const float *x, int n, float fmax); /* max|x| / fmax */
int      orc_is_fp8(int fmt);                            /* e4m3fn or e5m2 */
void     orc_fp16_to_bf16_n(const uint16_t *in, uint16_t *out, int64_t n);
void     orc_f32_to_e4m3fn_n(const float *in, uint8_t *out, int64_t n);
void     orc_f32_to_e5m2_n(const float *in, uint8_t *out, int64_t n);
void     orc_decode_n(int fmt, const void *in, double *out, int64_t n);
/* convert one row of D source elements to the destination format; *scale is
 * written only for an e4m3fn destination */
void     orc_convert_row(int src_fmt, int dst_fmt, int D, const void *src_row,
                         void *dst_row, float *scale);

/* ---- index maps (parallel-strategy and VRAM-management alignment) ---- */
int      orc_validate(const orc_problem *p);             /* 0 ok, -1 invalid, -2 unsupported */
void     orc_head_source(const orc_problem *p, int i, int *shard, int *head);
int32_t  orc_src_heads(const orc_problem *p);   /* heads per prefill shard (1 if replicated) */
int32_t  orc_dst_heads(const orc_problem *p);   /* heads per decode rank (1 if replicated) */
int64_t  orc_src_request_base(const orc_problem *p, int r);  /* elements; 0 for ORC_PAGED */
/* element index in shard *shard, or -1 when the token's source page id lies
 * outside [0, src_num_blocks) (ORC_PAGED): such a row is never written */
int64_t  orc_src_index(const orc_problem *p, int r, int l, int kv, int t, int i, int d, int *shard);
/* l is a converted layer (0..layers-1); the cache holds it at dst_layer_offset + l */
int64_t  orc_cache_index(const orc_problem *p, int64_t block, int l, int kv, int slot, int i, int d);
int64_t  orc_cache_scale_index(const orc_problem *p, int64_t block, int l, int kv, int slot, int i);
int32_t  orc_src_layers(const orc_problem *p);   /* layers held by the source buffers */
int32_t  orc_dst_layers(const orc_problem *p);   /* layers held by the cache */
/* wire ("one-dimensional tensor") segments: byte offsets per request */
int64_t  orc_wire_layout(const orc_problem *p, int64_t *data_off, int64_t *scale_off);
int      orc_fmt_size(int fmt);

/* ---- the three operations ----
 * A destination page id outside [0, num_blocks) is skipped, and so is a row
 * whose source page id lies outside the source pool: neither writes a byte. */
int orc_pack(const orc_problem *p, const void *const *shards, void *wire);
int orc_unpack(const orc_problem *p, const void *wire, void *cache, float *scales,
               const int32_t *block_table, int32_t bt_stride);
int orc_repack(const orc_problem *p, const void *const *shards, void *cache, float *scales,
               const int32_t *block_table, int32_t bt_stride);

/* expected cache rows of request r, plane (l, kv), tokens [t0, t0+nt): nt*Hd
 * rows in (token, head) order in the cache format, plus nt*Hd scales for an
 * e4m3fn cache; rows whose source page lies outside the source pool are left
 * as the caller filled them */
int orc_expected_rows(const orc_problem *p, const void *const *shards, int r, int l, int kv,
                      int t0, int nt, void *out_rows, float *out_scales);

#ifdef __cplusplus
}
#endif
#endif
