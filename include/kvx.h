/*
 * kvx.h -- C ABI of the KV-cache conversion library for MI355X (gfx950).
 *
 * The library implements the data path of the heterogeneous compatible
 * transmission module of "Disaggregated Prefill and Decoding Inference System
 * for Large Language Model Serving on Multi-Vendor GPUs" (Sec. III-B): the KV
 * cache that a prefill (P) instance produced is converted into the layout,
 * page size, element type and tensor-parallel head shard that a decode (D)
 * instance with another parallel strategy expects.  The three data components
 * of the module map to the calls below:
 *
 *   - parallel-strategy alignment (Sec. III-B-3, Fig. 4): a decode rank holds
 *     one contiguous range of the global KV heads; the prefill shards that
 *     overlap it are merged (src_tp > dst_tp) or split (src_tp < dst_tp);
 *   - VRAM-management alignment (Sec. III-B-2, Fig. 5): the prefill layout is
 *     flattened into a one-dimensional transfer tensor (kvx_pack) and restored
 *     into the decode side's paged cache with its own page size and layout
 *     (kvx_unpack); kvx_repack does both in one pass when both sides are on
 *     the same device;
 *   - precision alignment (Sec. I, contribution 1, named only): the decode
 *     element type.  Casts round to nearest even; the 8-bit casts use a
 *     per-(token, head) fp32 scale max|x| / fmax and saturate at +-fmax
 *     (e4m3fn: fmax 448, NaN S.1111.111; e5m2: fmax 57344, NaN S.11111.11);
 *     an 8-bit transfer tensor may be dequantised into a 16-bit cache
 *     (cache_dtype).
 *
 * Layouts (element indices; all dimensions row-major):
 *   source shard j (j = 0..src_tp-1) holds global heads [j*Hs, (j+1)*Hs),
 *     Hs = num_kv_heads / src_tp; requests are stored back to back, request r
 *     as [layer][k/v][token][Hs][dim] (KVX_THD) or [layer][k/v][Hs][token][dim]
 *     (KVX_HTD), T_r tokens, over the source's src_layers layers; or
 *     (KVX_PAGED) the shard is the prefill side's
 *     own paged cache [layer][k/v][src_num_blocks][src_block_size][Hs][dim]:
 *     token t of request r sits in page
 *     src_block_table[r*src_bt_stride + t/src_block_size], slot
 *     t % src_block_size, one source block table for all shards (both sides
 *     of Sec. III-B-2 use paged attention, each with its own page size);
 *   decode rank dst_rank holds global heads [dst_rank*Hd, (dst_rank+1)*Hd),
 *     Hd = num_kv_heads / dst_tp;
 *   cache:  [dst layer][k/v][num_blocks][block_size][Hd][dim] in the cache
 *     dtype (cache_dtype, else dst_dtype); token
 *     t of request r goes to page block_table[r*bt_stride + t/block_size],
 *     slot t % block_size;
 *   scales (8-bit cache only): [dst layer][k/v][num_blocks][block_size][Hd] fp32;
 *   transfer tensor: per request, starting on a 256-byte boundary,
 *     [layer][k/v][token][Hd][dim] in dst_dtype, then (8-bit only) on the
 *     next 256-byte boundary [layer][k/v][token][Hd] fp32 scales.
 * Bytes outside these positions (slots past the end of a request's last page,
 * pages not in a block-table row, transfer-tensor padding) are never written.
 * A page id outside its pool names no page: a decode page id outside
 * [0, num_blocks) writes nothing, and a row whose source page id lies outside
 * [0, src_num_blocks) is written neither to the cache (repack) nor to the
 * transfer tensor or its scale (pack).  kvx_unpack cannot see source page
 * ids: it copies whatever the transfer tensor holds at such a row, so after
 * a pack, an unpack (and the layer-streamed pipe) writes those rows with the
 * transfer tensor's earlier contents.
 *
 * Ownership: every buffer is caller-owned device memory; the library never
 * allocates or frees it.  A plan is library-owned: kvx_plan copies seq_lens
 * and allocates a small device table on the device current at that time.
 *
 * Streams: kvx_pack / kvx_unpack / kvx_repack (and the _paged forms) only
 * enqueue work on the given hipStream_t (passed as void*, NULL = default
 * stream) and return; buffers must stay alive until the stream reaches that
 * point.  A plan is immutable and may be used concurrently on several streams
 * of its device, from several host threads.
 *
 * Graphs: these calls (and kvx_repack_noalloc) launch kernels and nothing
 * else: no allocation, copy, memset or synchronisation.  Called on a stream
 * under HIP graph capture they are recorded, and each replay reads the
 * sources, block tables and transfer tensor as they are at replay time.  The
 * recorded kernels hold the plan's device table and the buffer addresses:
 * the plan and the buffers must outlive the graph.  Make the first
 * kvx_repack_noalloc call on a device outside capture (it looks the address
 * of its static table up once per device).
 *
 * Errors: every call returns a kvx_status; nothing is thrown and nothing
 * aborts.  kvx_last_error() gives a message for the calling thread's last
 * non-OK status.  A plan whose requests hold no tokens has nothing to move:
 * its launch calls return KVX_OK without inspecting any pointer.
 */
#ifndef KVX_H
#define KVX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVX_ABI_VERSION 9

typedef enum {
    KVX_OK = 0,
    KVX_EINVAL = -1,       /* invalid argument, shape or pointer */
    KVX_EUNSUPPORTED = -2, /* valid request this library does not implement */
    KVX_ENOMEM = -3,       /* host or device allocation failed (kvx_plan, kvx_pipe_create) */
    KVX_EDEVICE = -4       /* no usable device for the plan, or a HIP error */
} kvx_status;

typedef enum { KVX_FP16 = 1, KVX_BF16 = 2, KVX_FP8_E4M3FN = 3, KVX_FP8_E5M2 = 4 } kvx_dtype;

typedef enum {
    KVX_THD = 0,  /* [token][head][dim] within one (layer, k/v) plane of a request */
    KVX_HTD = 1,  /* [head][token][dim] */
    KVX_PAGED = 2 /* the prefill side's paged cache (kvx_pack_paged / kvx_repack_paged) */
} kvx_order;

typedef struct kvx_plan_s kvx_plan_t; /* opaque, library-owned */

/* The conversion problem, in the terms of Sec. III-B: the two parallel
 * strategies (src_tp, dst_tp, dst_rank), the page size and layout of the
 * decode side (block_size, num_blocks, src_order), the precision of each side
 * (src_dtype, dst_dtype), and the requests whose KV moves. */
typedef struct {
    int32_t num_layers;     /* L >= 1 */
    int32_t num_kv_heads;   /* H >= 1, global KV heads */
    int32_t head_dim;       /* D >= 1 */
    int32_t src_tp;         /* prefill TP degree; divides H or is a multiple of H */
    int32_t dst_tp;         /* decode TP degree; divides H or is a multiple of H */
    int32_t dst_rank;       /* 0 <= dst_rank < dst_tp */
    int32_t src_dtype;      /* kvx_dtype: KVX_FP16 or KVX_BF16 */
    int32_t dst_dtype;      /* kvx_dtype of the transfer tensor */
    int32_t src_order;      /* kvx_order */
    int32_t block_size;     /* tokens per decode page, >= 1 */
    int64_t num_blocks;     /* pages per (layer, k/v) plane of the pool, >= 1 */
    int32_t num_requests;   /* >= 0 */
    const int32_t *seq_lens;/* host array [num_requests], T_r >= 0; copied */
    /* KVX_PAGED sources only (ignored otherwise): */
    int32_t src_block_size; /* tokens per prefill-side page, >= 1 */
    int64_t src_num_blocks; /* pages per (layer, k/v) plane of each shard's pool, >= 1 */
    /* Pipeline stages: the source buffers hold src_layers layers and converted
     * layer l (0 <= l < num_layers) is their layer src_layer_offset + l; the
     * cache (and scales) hold dst_layers layers and receive layer l at
     * dst_layer_offset + l.  The transfer tensor carries the num_layers
     * converted layers only.  src_layers / dst_layers = 0 mean num_layers
     * (with offset 0).  All zero: both sides hold exactly the converted layers. */
    int32_t src_layer_offset;
    int32_t src_layers;
    int32_t dst_layer_offset;
    int32_t dst_layers;
    /* The decode cache's element type; 0 means dst_dtype.  With an 8-bit
     * transfer tensor, KVX_BF16 or KVX_FP16 asks for a dequantising unpack
     * (precision alignment, Sec. I, done on the receiving side): each element
     * of the cache is the product of its code's exact value and the
     * row's fp32 scale, computed in fp32 and rounded to nearest even to the
     * 16-bit type (fp16: overflow to infinity; an e5m2 infinity code gives
     * an infinite product); a NaN code, or a NaN product, gives that type's
     * quiet NaN (bf16 0x7FC0, fp16 0x7E00) with the code's sign.  The cache
     * then holds no scales.  The pack and the transfer tensor are those of
     * the plain 8-bit plan; the repack writes what its pack followed by this
     * unpack would. */
    int32_t cache_dtype;
} kvx_desc;

typedef struct {
    uint64_t wire_bytes;            /* transfer tensor size (multiple of 256) */
    int64_t total_tokens;           /* sum of T_r */
    /* algorithmic bytes per call: elements and scales read and written once */
    int64_t read_bytes_pack, write_bytes_pack;
    int64_t read_bytes_unpack, write_bytes_unpack;
    int64_t read_bytes_repack, write_bytes_repack;
    int32_t max_blocks_per_request; /* minimum valid bt_stride */
    int32_t num_items;              /* logical pages over all requests (per plane) */
    int32_t device;                 /* HIP device of the plan's tables, -1 = none */
    int32_t max_src_blocks_per_request; /* KVX_PAGED: minimum valid src_bt_stride; else 0 */
} kvx_plan_info;

/* Validate the problem and build a plan (host tables, plus a device table on
 * the current HIP device when one is usable; otherwise the plan is host-only
 * and the launch calls return KVX_EDEVICE).
 * Returns KVX_EINVAL for: NULL desc/out; a dimension <= 0; a TP degree that
 * neither divides H nor is a multiple of it; dst_rank outside [0, dst_tp);
 * block_size <= 0; num_blocks <= 0; num_requests < 0; NULL seq_lens with requests; T_r < 0;
 * an unknown order; for KVX_PAGED, src_block_size <= 0 or src_num_blocks <= 0;
 * a negative layer offset or count, or converted layers outside either side's
 * src_layers / dst_layers;
 * head_dim * element size not a multiple of 16 bytes on either side; an
 * unknown dtype.
 * KVX_EUNSUPPORTED for: a dtype pair outside {fp16->fp16, bf16->bf16,
 * fp16->bf16, bf16->fp16, fp16/bf16->e4m3fn, fp16/bf16->e5m2}; a cache_dtype
 * other than dst_dtype unless dst_dtype is 8-bit and cache_dtype 16-bit; a
 * transfer-tensor row (head_dim * dst element size) above 1024 bytes; more
 * than 1024 heads per decode rank; more than 65535 source heads per shard; a
 * decode rank whose heads form more than 64 head segments (runs of heads
 * from one source shard); 2*L > 65535; more than 2^24 - 8 work units in one
 * launch (logical pages, the sum over requests of ceil(T_r / block_size),
 * x 2L planes x head segments x workgroup passes per page; so at most
 * 2^23 - 4 pages); a decode cache, source shard or transfer tensor of 2^62
 * bytes or more.  KVX_ENOMEM / KVX_EDEVICE if the table cannot be
 * allocated. */
kvx_status kvx_plan(const kvx_desc *desc, kvx_plan_t **out);

kvx_status kvx_plan_info_get(const kvx_plan_t *plan, kvx_plan_info *info);

/* Byte offsets of request r's data and scale regions in the transfer tensor
 * (scale_off = -1 unless dst is 8-bit).  KVX_EINVAL for r out of range. */
kvx_status kvx_plan_segment(const kvx_plan_t *plan, int32_t r, int64_t *data_off,
                            int64_t *scale_off);

/* Sizes of the buffers that launches with this plan touch.  The launch calls
 * take bare pointers and cannot check them: these are what a caller
 * allocates and what a binding checks before it launches (host only).
 * KVX_EINVAL for a NULL argument. */
typedef struct {
    uint64_t wire_bytes;    /* transfer tensor, as kvx_plan_info.wire_bytes */
    uint64_t cache_bytes;   /* decode cache [dst layers][2][NB][bs][Hd][D] of the cache type */
    uint64_t scale_bytes;   /* its fp32 scales [dst layers][2][NB][bs][Hd]; 0 for a 16-bit cache */
    int32_t num_requests;   /* rows of the block table (and of a source block table) */
    int32_t src_tp;         /* entries of the src_shards array */
} kvx_buffer_sizes;

kvx_status kvx_plan_buffer_sizes(const kvx_plan_t *plan, kvx_buffer_sizes *out);

/* Bytes from the start of prefill shard j within which a pack or repack
 * reads: the shard's requests back to back (2 x src layers x T_r x Hs x D
 * elements each) for a contiguous source, its whole pool (2 x src layers x
 * src_num_blocks x src_block_size x Hs x D elements) for a paged one; 0 when
 * the decode rank reads nothing from shard j (its pointer may then be NULL)
 * or the plan has no tokens.  KVX_EINVAL for a NULL argument or j outside
 * [0, src_tp). */
kvx_status kvx_plan_shard_bytes(const kvx_plan_t *plan, int32_t j, uint64_t *bytes);

/* Frees the plan and its device table (synchronous; the caller ensures no
 * launch using it is still pending).  NULL is accepted. */
kvx_status kvx_plan_destroy(kvx_plan_t *plan);

/* Pack (VRAM-management alignment, prefill side, Sec. III-B-2): gather the
 * decode rank's heads from the source shards, cast to dst_dtype and write the
 * transfer tensor.
 *   src_shards: host array of src_tp device pointers, one per prefill shard in
 *               the layout above; shards the decode rank does not read may be
 *               NULL.  Each read pointer must be 16-byte aligned.
 *   wire:       device, >= wire_bytes, 16-byte aligned.
 * KVX_EINVAL for a NULL plan/array, a NULL or misaligned needed pointer, a
 * KVX_PAGED plan (use kvx_pack_paged); KVX_EDEVICE for a host-only plan, a
 * current device other than the plan's, or a launch error. */
kvx_status kvx_pack(const kvx_plan_t *plan, const void *const *src_shards, void *wire,
                    void *hip_stream);

/* Unpack (VRAM-management alignment, decode side): scatter the transfer
 * tensor into the paged cache (and the scales), with no cast unless
 * cache_dtype asks for the dequantisation described at kvx_desc.
 *   cache:       device [L][2][num_blocks][block_size][Hd][D] cache dtype, 16-byte aligned.
 *   scales:      device [L][2][num_blocks][block_size][Hd] fp32, 16-byte aligned;
 *                non-NULL if and only if the cache dtype is 8-bit.
 *   block_table: device int32 [num_requests][bt_stride]; the first
 *                ceil(T_r/block_size) entries of row r are used.  Contents are a
 *                caller contract (kvx_check_block_table checks them on the
 *                host); a page id outside [0, num_blocks) is skipped, never
 *                written.  Ids shared by two requests are two writers (a race).
 *   bt_stride:   >= max_blocks_per_request.
 * Errors as kvx_pack, plus KVX_EINVAL for a scales pointer whose presence does
 * not match the cache dtype, a NULL block table with pages to write, or a short
 * bt_stride. */
kvx_status kvx_unpack(const kvx_plan_t *plan, const void *wire, void *cache, float *scales,
                      const int32_t *block_table, int32_t bt_stride, void *hip_stream);

/* Repack: kvx_pack followed by kvx_unpack in one pass with no transfer tensor;
 * the cache and scales it writes are bit-identical to that pair's.
 * KVX_EINVAL for a KVX_PAGED plan (use kvx_repack_paged). */
kvx_status kvx_repack(const kvx_plan_t *plan, const void *const *src_shards, void *cache,
                      float *scales, const int32_t *block_table, int32_t bt_stride,
                      void *hip_stream);

/* Pack and repack from paged sources (plans with src_order KVX_PAGED): the
 * prefill side's own paged caches, one per shard, with their own page size
 * and block table (Sec. III-B-2), re-paged (and re-sharded and cast) into the
 * decode layout.  Results are those of the contiguous source the pages
 * describe.
 *   src_shards:      as kvx_pack; shard j points to its pool
 *                    [L][2][src_num_blocks][src_block_size][Hs][D].
 *   src_block_table: device int32 [num_requests][src_bt_stride]; the first
 *                    ceil(T_r/src_block_size) entries of row r are used.  A
 *                    page may appear in several rows (a shared prefix); an
 *                    id outside [0, src_num_blocks) leaves its rows unwritten.
 *   src_bt_stride:   >= max_src_blocks_per_request.
 * Errors as kvx_pack / kvx_repack, plus KVX_EINVAL for a plan whose source is
 * not KVX_PAGED, a NULL source block table with tokens to move, or a short
 * src_bt_stride. */
kvx_status kvx_pack_paged(const kvx_plan_t *plan, const void *const *src_shards,
                          const int32_t *src_block_table, int32_t src_bt_stride, void *wire,
                          void *hip_stream);
kvx_status kvx_repack_paged(const kvx_plan_t *plan, const void *const *src_shards,
                            const int32_t *src_block_table, int32_t src_bt_stride, void *cache,
                            float *scales, const int32_t *block_table, int32_t bt_stride,
                            void *hip_stream);

/* Repack without any allocation, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  The same conversion as kvx_plan + kvx_repack of *desc
 * (token- or head-major sources), with no plan: the work-item table that
 * kvx_plan would allocate lives in a static device array of the library (one
 * per device, 65536 entries of 40 bytes), written by a small kernel on
 * hip_stream before the repack kernel.  Nothing is allocated on the host
 * heap or the device; the call enqueues two kernels and returns.
 *   desc:        as kvx_plan (copied; seq_lens read during the call only);
 *                at most 256 requests and 65536 destination pages in all
 *                (sum of ceil(T_r / block_size)), else KVX_EUNSUPPORTED.
 *   other arguments: as kvx_repack.
 * Calls on one device share its table: calls that overlap on one device (two
 * streams, or two threads) race and must be ordered by the caller.  Errors:
 * those of kvx_plan and kvx_repack; KVX_EINVAL for a KVX_PAGED source;
 * KVX_EDEVICE when the table's device address cannot be found or a launch
 * fails. */
kvx_status kvx_repack_noalloc(const kvx_desc *desc, const void *const *src_shards, void *cache,
                              float *scales, const int32_t *block_table, int32_t bt_stride,
                              void *hip_stream);

/* Host-side check of a block table: every used entry in [0, num_blocks) and no
 * page used twice.  KVX_EINVAL (with a message) otherwise. */
kvx_status kvx_check_block_table(const kvx_plan_t *plan, const int32_t *host_block_table,
                                 int32_t bt_stride);

/* Host-side check of a source block table (KVX_PAGED plans): every used entry
 * in [0, src_num_blocks) and src_bt_stride >= max_src_blocks_per_request.
 * Pages shared between requests are allowed.  KVX_EINVAL otherwise. */
kvx_status kvx_check_src_block_table(const kvx_plan_t *plan, const int32_t *host_src_block_table,
                                     int32_t src_bt_stride);

/* ---- layer-streamed transfer through pinned host memory ----
 *
 * The transfer of Sec. III-B-1 moves the KV cache through a pinned host
 * memory pool, and the paper's conclusion names by-layer transmission as the
 * next step.  A pipe moves a plan's layers in chunks of chunk_layers layers:
 * each chunk is packed straight into a slot of a pinned host ring (the pack
 * kernel's stores cross the host link), copied into a device receive slot
 * (host to device) and unpacked into the cache, each stage on a stream of the
 * pipe.  With `slots` slots, chunk c + 1 is packed and chunk c - 1 unpacked
 * while chunk c crosses the bus.  The cache and scales written equal
 * kvx_pack followed by kvx_unpack of the whole plan (rows whose source page
 * id is outside the source pool take whatever their ring slot held).
 *
 * kvx_pipe_create allocates the pinned host ring (slots x the largest
 * chunk's transfer-tensor bytes, hipHostMalloc with hipHostMallocMapped),
 * device receive slots of the same size, three streams and their events, on
 * the plan's device.  The streams are CU-masked (hipExtStreamCreateWithCUMask,
 * default priority): the pack's covers half the device's CUs, the copy's and
 * the unpack's a quarter each, so that no stage waits for CUs another holds;
 * like streams created without flags, they synchronise with the null stream.
 * The plan must outlive the pipe.  A plan with no tokens gets a pipe that
 * allocates nothing and whose runs return KVX_OK at once (on any host).
 * KVX_EINVAL for a NULL plan or out, chunk_layers outside [1, num_layers] or
 * slots < 1; KVX_EDEVICE for a host-only plan with tokens or when the
 * streams cannot be created; KVX_ENOMEM if an allocation fails.
 *
 * kvx_pipe_run enqueues the whole transfer and returns: the pipe's streams
 * start after the caller's stream's earlier work and after the pipe's
 * previous run (runs of one pipe share the slots, so the pipe orders them
 * itself), and the caller's stream's later work waits for the last unpack.
 * On the legacy null stream (NULL or hipStreamLegacy) the pipe enqueues
 * nothing on the caller's stream, whose synchronisation with the pipe's
 * streams gives that order by itself; on any other stream it records an
 * event before the run and waits for one after it.  Work that the caller
 * puts on the legacy null stream between runs is ordered against the pipe's
 * streams by the runtime, which costs about 2.5% per run and the first few
 * times made the host wait 20-30 ms in that enqueue: transfers on a created
 * stream see neither.  Arguments as kvx_repack
 * (kvx_repack_paged for a paged plan, whose source block table is passed;
 * otherwise it must be NULL).  One pipe must not be used from two threads at
 * once; runs of different pipes may overlap.  A bad argument is reported
 * before anything is enqueued; a launch or enqueue failure part way through
 * returns its status with the cache partly written, and the caller's stream
 * and the pipe's next run still wait for the chunks already enqueued. */
typedef struct kvx_pipe_s kvx_pipe_t; /* opaque, library-owned */

typedef struct {
    int32_t chunk_layers;      /* layers per chunk (the last chunk may hold fewer) */
    int32_t num_chunks;
    int32_t slots;
    int32_t reserved;
    uint64_t slot_bytes;       /* transfer-tensor bytes of the largest chunk */
    uint64_t host_bytes;       /* pinned host ring: slots x slot_bytes */
    uint64_t device_bytes;     /* receive slots: slots x slot_bytes */
    uint64_t bus_bytes;        /* bytes each direction moves per run: the plan's wire bytes, by chunk */
} kvx_pipe_info;

kvx_status kvx_pipe_create(const kvx_plan_t *plan, int32_t chunk_layers, int32_t slots,
                           kvx_pipe_t **out);
kvx_status kvx_pipe_info_get(const kvx_pipe_t *pipe, kvx_pipe_info *info);
kvx_status kvx_pipe_run(kvx_pipe_t *pipe, const void *const *src_shards,
                        const int32_t *src_block_table, int32_t src_bt_stride, void *cache,
                        float *scales, const int32_t *block_table, int32_t bt_stride,
                        void *hip_stream);
/* Waits for the pipe's streams, then frees everything it allocated.  NULL is
 * accepted. */
kvx_status kvx_pipe_destroy(kvx_pipe_t *pipe);

/* Message for the calling thread's last non-OK status ("" if none). */
const char *kvx_last_error(void);

int32_t kvx_abi_version(void);

/* ---- P:D deployment planner (host only) ----
 *
 * The joint optimisation of parallel strategy and P:D ratio (Sec. III-C):
 * Eq. 1 picks the prefill instance's (dp, tp, pp, ep) that maximises the
 * throughput per GPU T_p / (dp*tp*pp) subject to l_p <= ttft (Eq. 2) and
 * m_p <= the GPU's VRAM (Eq. 3); Eq. 4 picks the decode instance's that
 * maximises its throughput subject to l_d <= tpot (Eq. 5) and m_d <= VRAM
 * (Eq. 6); the instance counts X : Y meet the request rate.  The paper
 * gives the structure of these equations, not the cost terms; the terms
 * used here are those of a decoder-only transformer:
 *   l_p = c_p / (lambda R) + e_p / (beta B)   c_p: 2 FLOPs per weight per
 *         token, causal attention 2*L*hq*D*b*s*(s+1), the LM head on the
 *         last token; split by tp (experts by ep); e_p: 2 ring all-reduces
 *         per layer (2(tp-1)/tp of b*s*h activations), pp-1 stage
 *         hand-overs, 2 expert all-to-alls per layer ((ep-1)/ep);
 *   m_p = weights on the most loaded GPU (attention, dense FFN and
 *         embedding/head split by tp, E/ep whole experts, layers split by
 *         pp) + one layer's activations + the batch's KV;
 *   l_d = (weights read per step + KV of b requests at the average context
 *         s_in + s_out/2) / (alpha B_vram) + e_d / (beta B);
 *   m_d = weights + activations + KV of b requests at s_in + s_out;
 *   T = dp * pp * b / l (pp batches in flight; requests/s for prefill,
 *         tokens/s for decode); X = ceil(qps / T_p), Y = ceil(qps * s_out / T_d).
 * KV per GPU uses H/tp heads, or one replicated head when tp is a multiple
 * of H.  Candidates: tp divides q_heads and divides H or is a multiple of
 * it (the head map of kvx_plan), pp divides L, ep = 1 for dense models or
 * divides E and dp*tp, batch a power of two <= max_batch, dp*tp*pp <=
 * max_gpus; visited in the order (GPUs, tp, pp, dp, ep, batch), the first
 * whose objective is within a relative 1e-9 of the best wins.  All sizes in
 * bytes, rates per second, times in seconds. */
typedef enum { KVX_PD_PREFILL = 0, KVX_PD_DECODE = 1 } kvx_pd_side;

typedef struct {
    int32_t layers, hidden, q_heads, kv_heads, head_dim, ffn_dim, vocab;
    int32_t experts;          /* FFN experts per layer, 1 = dense */
    int32_t active_experts;   /* experts per token (1 when dense) */
    int32_t reserved;
    double weight_bytes, kv_bytes, act_bytes;   /* bytes per element */
} kvx_pd_model;

typedef struct {
    double flops;       /* R: FLOP/s per GPU */
    double hbm_bytes;   /* B_vram: bytes/s per GPU */
    double vram;        /* M: bytes per GPU */
    double link_bytes;  /* B: interconnect bytes/s per GPU */
    double lambda, alpha, beta;  /* discount factors in (0, 1] */
    int32_t max_gpus;   /* GPUs one instance may use, 1..4096 */
    int32_t reserved;
} kvx_pd_gpu;

typedef struct {
    kvx_pd_model model;
    kvx_pd_gpu prefill, decode;
    int32_t prompt_tokens, output_tokens;   /* s_in, s_out >= 1 */
    double qps;          /* requests per second to serve, >= 0 */
    double ttft, tpot;   /* thresholds L_ttft, L_tpot (s), > 0 */
    int32_t max_batch;   /* largest batch tried, 1..2^20 */
    int32_t reserved;
} kvx_pd_problem;

typedef struct {
    int32_t dp, tp, pp, ep, batch, gpus;   /* gpus = dp*tp*pp; all 0 = no feasible strategy */
    double latency;      /* l_p or l_d */
    double vram;         /* m_p or m_d */
    double throughput;   /* T_p (requests/s) or T_d (tokens/s) */
    double objective;    /* T_p / gpus, or T_d */
} kvx_pd_choice;

typedef struct {
    kvx_pd_choice prefill, decode;
    int64_t prefill_instances, decode_instances;   /* X : Y (0 when either side is infeasible) */
    int64_t candidates_prefill, candidates_decode;
    int64_t feasible_prefill, feasible_decode;
} kvx_pd_solution;

/* The search of Eq. 1 and Eq. 4 (host only; no device is used).  KVX_EINVAL
 * for a NULL argument, a dimension < 1, active_experts > experts, a
 * non-positive byte size, rate, VRAM or threshold, a discount factor
 * outside (0, 1], max_gpus outside [1, 4096], prompt or output tokens < 1,
 * a negative qps or max_batch outside [1, 2^20]. */
kvx_status kvx_pd_search(const kvx_pd_problem *problem, kvx_pd_solution *out);

/* The cost terms of one strategy on one side (kvx_pd_side), without the
 * constraints: latency, vram, throughput and objective as in kvx_pd_choice.
 * Errors as kvx_pd_search, plus KVX_EINVAL for an unknown side or a
 * strategy value < 1. */
kvx_status kvx_pd_evaluate(const kvx_pd_problem *problem, int32_t side, int32_t dp, int32_t tp,
                           int32_t pp, int32_t ep, int32_t batch, kvx_pd_choice *out);

#ifdef __cplusplus
}
#endif
#endif /* KVX_H */
