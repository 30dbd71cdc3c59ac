// Host side of the C ABI: problem validation, the plan (head-shard map,
// request offsets, work items, transfer-tensor segments, byte accounting),
// argument checks and launch dispatch.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "kvx.h"
#include "kvx_host.h"
#include "kvx_internal.h"

using kvx::Item;


namespace {
thread_local std::string g_last_error;
}  // namespace

kvx_status kvx::fail(kvx_status s, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

namespace {

using kvx::fail;

bool is_fp8(int dt) { return dt == KVX_FP8_E4M3FN || dt == KVX_FP8_E5M2; }

bool is_dtype(int dt) { return dt == KVX_FP16 || dt == KVX_BF16 || is_fp8(dt); }

int dtype_size(int dt) { return is_fp8(dt) ? 1 : 2; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

// conversion kernel variant for a dtype pair, or -1 if unsupported
int pick_conv(int s, int d)
{
    if (s != KVX_FP16 && s != KVX_BF16) return -1;
    if (s == d) return kvx::kCopy16;
    if (s == KVX_FP16 && d == KVX_BF16) return kvx::kF16Bf16;
    if (s == KVX_BF16 && d == KVX_FP16) return kvx::kBf16F16;
    if (s == KVX_BF16 && d == KVX_FP8_E4M3FN) return kvx::kBf16E4m3;
    if (s == KVX_FP16 && d == KVX_FP8_E4M3FN) return kvx::kF16E4m3;
    if (s == KVX_BF16 && d == KVX_FP8_E5M2) return kvx::kBf16E5m2;
    if (s == KVX_FP16 && d == KVX_FP8_E5M2) return kvx::kF16E5m2;
    return -1;
}

// Heads per rank: H / tp, or 1 when tp is a multiple of H (each KV head is
// then replicated on tp / H consecutive ranks).
int heads_per_rank(int H, int tp) { return tp <= H ? H / tp : 1; }

// The cache's element type: dst_dtype, or the 16-bit type of a dequantising
// unpack of an 8-bit transfer tensor.
int cache_dtype_of(const kvx_desc& d) { return d.cache_dtype ? d.cache_dtype : d.dst_dtype; }

// repack kernel variant that quantises to the 8-bit format w and
// dequantises into a 16-bit cache c
int qd_conv(int s, int w, int c)
{
    if (w == KVX_FP8_E5M2) {
        if (s == KVX_BF16) return c == KVX_BF16 ? kvx::kQd5Bf16Bf16 : kvx::kQd5Bf16F16;
        return c == KVX_BF16 ? kvx::kQd5F16Bf16 : kvx::kQd5F16F16;
    }
    if (s == KVX_BF16) return c == KVX_BF16 ? kvx::kQdBf16Bf16 : kvx::kQdBf16F16;
    return c == KVX_BF16 ? kvx::kQdF16Bf16 : kvx::kQdF16F16;
}

int32_t src_layers_of(const kvx_desc& d) { return d.src_layers ? d.src_layers : d.num_layers; }
int32_t dst_layers_of(const kvx_desc& d) { return d.dst_layers ? d.dst_layers : d.num_layers; }

kvx_status validate(const kvx_desc* d)
{
    if (d->num_layers <= 0 || d->num_kv_heads <= 0 || d->head_dim <= 0)
        return fail(KVX_EINVAL, "num_layers, num_kv_heads and head_dim must be >= 1");
    if (d->src_tp <= 0 || d->dst_tp <= 0)
        return fail(KVX_EINVAL, "src_tp and dst_tp must be >= 1");
    if ((d->num_kv_heads % d->src_tp && d->src_tp % d->num_kv_heads) ||
        (d->num_kv_heads % d->dst_tp && d->dst_tp % d->num_kv_heads))
        return fail(KVX_EINVAL,
                    "num_kv_heads (%d) and each TP degree (src %d, dst %d) must divide one another",
                    d->num_kv_heads, d->src_tp, d->dst_tp);
    if (d->dst_rank < 0 || d->dst_rank >= d->dst_tp)
        return fail(KVX_EINVAL, "dst_rank %d outside [0, %d)", d->dst_rank, d->dst_tp);
    if (d->block_size <= 0) return fail(KVX_EINVAL, "block_size must be >= 1");
    if (d->num_blocks <= 0) return fail(KVX_EINVAL, "num_blocks must be >= 1");
    if (d->num_requests < 0) return fail(KVX_EINVAL, "num_requests must be >= 0");
    if (d->num_requests > 0 && !d->seq_lens) return fail(KVX_EINVAL, "seq_lens is NULL");
    for (int r = 0; r < d->num_requests; ++r)
        if (d->seq_lens[r] < 0) return fail(KVX_EINVAL, "seq_lens[%d] < 0", r);
    if (d->src_order != KVX_THD && d->src_order != KVX_HTD && d->src_order != KVX_PAGED)
        return fail(KVX_EINVAL, "unknown src_order %d", d->src_order);
    if (d->src_order == KVX_PAGED && (d->src_block_size <= 0 || d->src_num_blocks <= 0))
        return fail(KVX_EINVAL, "a paged source needs src_block_size >= 1 and src_num_blocks >= 1");
    if (!is_dtype(d->src_dtype)) return fail(KVX_EINVAL, "unknown src_dtype %d", d->src_dtype);
    if (!is_dtype(d->dst_dtype)) return fail(KVX_EINVAL, "unknown dst_dtype %d", d->dst_dtype);
    if (pick_conv(d->src_dtype, d->dst_dtype) < 0)
        return fail(KVX_EUNSUPPORTED, "dtype pair %d -> %d is not supported", d->src_dtype,
                    d->dst_dtype);
    const int cdt = cache_dtype_of(*d);
    if (!is_dtype(cdt)) return fail(KVX_EINVAL, "unknown cache_dtype %d", d->cache_dtype);
    if (cdt != d->dst_dtype && !(is_fp8(d->dst_dtype) && !is_fp8(cdt)))
        return fail(KVX_EUNSUPPORTED,
                    "cache_dtype %d differs from dst_dtype %d (only an 8-bit transfer tensor is "
                    "dequantised, into a 16-bit cache)", cdt, d->dst_dtype);
    if ((int64_t(d->head_dim) * dtype_size(d->src_dtype)) % 16 ||
        (int64_t(d->head_dim) * dtype_size(d->dst_dtype)) % 16)
        return fail(KVX_EINVAL, "head_dim %d: rows must be whole 16-byte vectors on both sides",
                    d->head_dim);
    if (int64_t(d->head_dim) * dtype_size(d->dst_dtype) > 16 * kvx::kMaxRowChunks)
        return fail(KVX_EUNSUPPORTED, "transfer-tensor rows above %d bytes",
                    16 * kvx::kMaxRowChunks);
    if (d->num_kv_heads / d->dst_tp > kvx::kMaxHeadsPerRank)
        return fail(KVX_EUNSUPPORTED, "more than %d heads per decode rank", kvx::kMaxHeadsPerRank);
    if (d->num_kv_heads / d->src_tp > 65535)
        return fail(KVX_EUNSUPPORTED, "more than 65535 heads per source shard");
    if (d->src_layer_offset < 0 || d->src_layers < 0 || d->dst_layer_offset < 0 ||
        d->dst_layers < 0)
        return fail(KVX_EINVAL, "negative layer offset or count");
    if (int64_t(d->src_layer_offset) + d->num_layers > src_layers_of(*d))
        return fail(KVX_EINVAL, "layers [%d, %d) outside the %d source layers", d->src_layer_offset,
                    d->src_layer_offset + d->num_layers, src_layers_of(*d));
    if (int64_t(d->dst_layer_offset) + d->num_layers > dst_layers_of(*d))
        return fail(KVX_EINVAL, "layers [%d, %d) outside the %d cache layers", d->dst_layer_offset,
                    d->dst_layer_offset + d->num_layers, dst_layers_of(*d));
    if (int64_t(src_layers_of(*d)) * 2 > 65535 || int64_t(dst_layers_of(*d)) * 2 > 65535)
        return fail(KVX_EUNSUPPORTED, "2 * layers above 65535");
    // every buffer stays below 2^62 bytes, so that the 64-bit offsets of the
    // planner and the kernels cannot overflow (sizes are compared in double
    // precision: relative error below 2^-50, far inside the 2x margin)
    const double lim = 4611686018427387904.0;  // 2^62
    const double hs = heads_per_rank(d->num_kv_heads, d->src_tp);
    const double hd = heads_per_rank(d->num_kv_heads, d->dst_tp);
    const double row_cache = hd * d->head_dim * dtype_size(cdt);
    if (2.0 * dst_layers_of(*d) * double(d->num_blocks) * d->block_size * row_cache > lim)
        return fail(KVX_EUNSUPPORTED, "decode cache above 2^62 bytes");
    const double row_src = hs * d->head_dim * dtype_size(d->src_dtype);
    double src = 0, wire = 0;
    if (d->src_order == KVX_PAGED)
        src = 2.0 * src_layers_of(*d) * double(d->src_num_blocks) * d->src_block_size * row_src;
    for (int r = 0; r < d->num_requests; ++r) {
        if (d->src_order != KVX_PAGED) src += 2.0 * src_layers_of(*d) * d->seq_lens[r] * row_src;
        wire += 2.0 * d->num_layers * d->seq_lens[r] * hd *
                    (double(d->head_dim) * dtype_size(d->dst_dtype) + 4) + 512;
    }
    if (src > lim) return fail(KVX_EUNSUPPORTED, "source shard above 2^62 bytes");
    if (wire > lim) return fail(KVX_EUNSUPPORTED, "transfer tensor above 2^62 bytes");
    return KVX_OK;
}

}  // namespace

extern "C" {

int32_t kvx_abi_version(void) { return KVX_ABI_VERSION; }

const char* kvx_last_error(void) { return g_last_error.c_str(); }

kvx_status kvx_plan(const kvx_desc* desc, kvx_plan_t** out)
{
    if (!desc || !out) return fail(KVX_EINVAL, "NULL desc or out");
    *out = nullptr;
    kvx_status st = validate(desc);
    if (st != KVX_OK) return st;

    kvx_plan_s* p = new (std::nothrow) kvx_plan_s();
    if (!p) return fail(KVX_ENOMEM, "host allocation failed");
    const kvx_desc& d = *desc;
    p->d = d;
    p->lens.assign(d.seq_lens, d.seq_lens + d.num_requests);
    p->d.seq_lens = p->lens.data();
    st = kvx::derive_shape(d, p->sh);
    if (st != KVX_OK) {
        delete p;
        return st;
    }
    const kvx::Shape& sh = p->sh;
    p->hs = sh.hs;
    p->hd = sh.hd;
    p->esz_src = sh.esz_src;
    p->esz_dst = sh.esz_dst;
    p->conv = sh.conv;
    p->cache_dtype = sh.cache_dtype;
    p->esz_cache = sh.esz_cache;
    p->dequant = sh.dequant;
    p->segs.assign(sh.segs, sh.segs + sh.nsegs);
    p->read_shards.assign(sh.read_shards, sh.read_shards + sh.nread);
    p->cpr = sh.cpr;
    p->lg_lpr = sh.lg_lpr;
    p->parts = sh.parts;
    p->parts_unpack = sh.parts_unpack;

    // requests: source offsets, transfer-tensor segments, work items
    const bool fp8 = is_fp8(d.dst_dtype);  // the transfer tensor carries scales
    const bool paged = d.src_order == KVX_PAGED;
    const int64_t L2 = int64_t(d.num_layers) * 2;
    int64_t src_off = 0, wire = 0, nitems = 0;
    p->wire_data.resize(d.num_requests);
    p->wire_scale.resize(d.num_requests);
    std::vector<int64_t> src_base(d.num_requests);
    for (int r = 0; r < d.num_requests; ++r) {
        const int64_t T = p->lens[r];
        const int64_t rows = L2 * T * p->hd;
        src_base[r] = paged ? 0 : src_off;  // a paged source is addressed through its pages
        src_off += 2 * int64_t(src_layers_of(d)) * T * p->hs * d.head_dim;
        if (paged)
            p->max_src_blocks = int32_t(std::max<int64_t>(
                p->max_src_blocks, (T + d.src_block_size - 1) / d.src_block_size));
        wire = align256(wire);
        p->wire_data[r] = wire;
        wire += rows * d.head_dim * p->esz_dst;
        if (fp8) {
            wire = align256(wire);
            p->wire_scale[r] = wire;
            wire += rows * 4;
        } else {
            p->wire_scale[r] = -1;
        }
        const int64_t nb = (T + d.block_size - 1) / d.block_size;
        p->max_blocks = int32_t(std::max<int64_t>(p->max_blocks, nb));
        nitems += nb;
        p->total_tokens += T;
        p->elems_rows += rows;
    }
    p->wire_bytes = uint64_t(align256(wire));
    p->src_elems = paged ? 2 * int64_t(src_layers_of(d)) * d.src_num_blocks * d.src_block_size *
                               p->hs * d.head_dim
                         : src_off;
    if (nitems * L2 * std::max<int64_t>(int64_t(p->parts) * int64_t(p->segs.size()),
                                        p->parts_unpack) > kvx::kMaxUnits) {
        delete p;
        return fail(KVX_EUNSUPPORTED, "more than %lld work units (pages x 2 x layers x parts)",
                    (long long)kvx::kMaxUnits);
    }
    p->items.reserve(size_t(std::max<int64_t>(nitems, 1)));
    for (int r = 0; r < d.num_requests; ++r) {
        const int nb = (p->lens[r] + d.block_size - 1) / d.block_size;
        for (int k = 0; k < nb; ++k)
            p->items.push_back(Item{src_base[r], p->wire_data[r], p->wire_scale[r], r, k,
                                    p->lens[r], 0});
    }

    // device table on the current device, when one is usable
    int dev = -1;
    if (!p->items.empty() && hipGetDevice(&dev) == hipSuccess && dev >= 0) {
        const size_t ib = p->items.size() * sizeof(Item);
        void* t = nullptr;
        if (hipMalloc(&t, ib) != hipSuccess) {
            delete p;
            return fail(KVX_ENOMEM, "device table allocation failed");
        }
        if (hipMemcpy(t, p->items.data(), ib, hipMemcpyHostToDevice) != hipSuccess) {
            (void)hipFree(t);
            delete p;
            return fail(KVX_EDEVICE, "device table upload failed");
        }
        p->device = dev;
        p->dev_table = t;
        p->dev_items = static_cast<const Item*>(t);
    } else if (!p->items.empty()) {
        (void)hipGetLastError();  // no device: host-only plan
    }
    *out = p;
    return KVX_OK;
}

kvx_status kvx_plan_info_get(const kvx_plan_t* p, kvx_plan_info* info)
{
    if (!p || !info) return fail(KVX_EINVAL, "NULL plan or info");
    std::memset(info, 0, sizeof *info);
    const int64_t D = p->d.head_dim;
    const int64_t rd = p->elems_rows * D * p->esz_src;
    const int64_t wr = p->elems_rows * D * p->esz_dst +
                       (is_fp8(p->d.dst_dtype) ? p->elems_rows * 4 : 0);
    const int64_t cw = p->elems_rows * D * p->esz_cache +
                       (is_fp8(p->cache_dtype) ? p->elems_rows * 4 : 0);
    info->wire_bytes = p->wire_bytes;
    info->total_tokens = p->total_tokens;
    info->read_bytes_pack = rd;
    info->write_bytes_pack = wr;
    info->read_bytes_unpack = wr;
    info->write_bytes_unpack = cw;
    info->read_bytes_repack = rd;
    info->write_bytes_repack = cw;
    info->max_blocks_per_request = p->max_blocks;
    info->num_items = int32_t(p->items.size());
    info->device = p->device;
    info->max_src_blocks_per_request = p->max_src_blocks;
    return KVX_OK;
}

kvx_status kvx_plan_segment(const kvx_plan_t* p, int32_t r, int64_t* data_off, int64_t* scale_off)
{
    if (!p) return fail(KVX_EINVAL, "NULL plan");
    if (r < 0 || r >= p->d.num_requests)
        return fail(KVX_EINVAL, "request %d outside [0, %d)", r, p->d.num_requests);
    if (data_off) *data_off = p->wire_data[r];
    if (scale_off) *scale_off = p->wire_scale[r];
    return KVX_OK;
}

kvx_status kvx_plan_buffer_sizes(const kvx_plan_t* p, kvx_buffer_sizes* out)
{
    if (!p || !out) return fail(KVX_EINVAL, "NULL plan or out");
    std::memset(out, 0, sizeof *out);
    const kvx_desc& d = p->d;
    const uint64_t slots = 2 * uint64_t(dst_layers_of(d)) * uint64_t(d.num_blocks) *
                           uint64_t(d.block_size) * uint64_t(p->hd);
    out->wire_bytes = p->wire_bytes;
    out->cache_bytes = slots * uint64_t(d.head_dim) * uint64_t(p->esz_cache);
    out->scale_bytes = is_fp8(p->cache_dtype) ? slots * 4 : 0;
    out->num_requests = d.num_requests;
    out->src_tp = d.src_tp;
    return KVX_OK;
}

kvx_status kvx_plan_shard_bytes(const kvx_plan_t* p, int32_t j, uint64_t* bytes)
{
    if (!p || !bytes) return fail(KVX_EINVAL, "NULL plan or bytes");
    if (j < 0 || j >= p->d.src_tp)
        return fail(KVX_EINVAL, "shard %d outside [0, %d)", j, p->d.src_tp);
    *bytes = 0;
    if (p->items.empty() ||
        std::find(p->read_shards.begin(), p->read_shards.end(), j) == p->read_shards.end())
        return KVX_OK;
    *bytes = uint64_t(p->src_elems) * uint64_t(p->esz_src);
    return KVX_OK;
}

kvx_status kvx_plan_destroy(kvx_plan_t* p)
{
    if (!p) return KVX_OK;
    if (p->dev_table) (void)hipFree(p->dev_table);
    delete p;
    return KVX_OK;
}

kvx_status kvx_check_block_table(const kvx_plan_t* p, const int32_t* bt, int32_t bt_stride)
{
    if (!p) return fail(KVX_EINVAL, "NULL plan");
    if (p->items.empty()) return KVX_OK;
    if (!bt) return fail(KVX_EINVAL, "NULL block table");
    if (bt_stride < p->max_blocks)
        return fail(KVX_EINVAL, "bt_stride %d < max_blocks_per_request %d", bt_stride, p->max_blocks);
    std::vector<int32_t> used;
    used.reserve(p->items.size());
    for (int r = 0; r < p->d.num_requests; ++r) {
        const int nb = (p->lens[r] + p->d.block_size - 1) / p->d.block_size;
        for (int k = 0; k < nb; ++k) {
            const int32_t b = bt[int64_t(r) * bt_stride + k];
            if (b < 0 || b >= p->d.num_blocks)
                return fail(KVX_EINVAL, "block_table[%d][%d] = %d outside [0, %lld)", r, k, b,
                            (long long)p->d.num_blocks);
            used.push_back(b);
        }
    }
    std::sort(used.begin(), used.end());
    for (size_t k = 1; k < used.size(); ++k)
        if (used[k] == used[k - 1]) return fail(KVX_EINVAL, "page %d is used twice", used[k]);
    return KVX_OK;
}

kvx_status kvx_check_src_block_table(const kvx_plan_t* p, const int32_t* sbt, int32_t sbt_stride)
{
    if (!p) return fail(KVX_EINVAL, "NULL plan");
    if (p->d.src_order != KVX_PAGED) return fail(KVX_EINVAL, "the plan's source is not paged");
    if (p->items.empty()) return KVX_OK;
    if (!sbt) return fail(KVX_EINVAL, "NULL source block table");
    if (sbt_stride < p->max_src_blocks)
        return fail(KVX_EINVAL, "src_bt_stride %d < max_src_blocks_per_request %d", sbt_stride,
                    p->max_src_blocks);
    for (int r = 0; r < p->d.num_requests; ++r) {
        const int nb = (p->lens[r] + p->d.src_block_size - 1) / p->d.src_block_size;
        for (int k = 0; k < nb; ++k) {
            const int32_t b = sbt[int64_t(r) * sbt_stride + k];
            if (b < 0 || b >= p->d.src_num_blocks)
                return fail(KVX_EINVAL, "src_block_table[%d][%d] = %d outside [0, %lld)", r, k, b,
                            (long long)p->d.src_num_blocks);
        }
    }
    return KVX_OK;
}

}  // extern "C"

kvx::FastDiv kvx::make_fastdiv(uint32_t d)
{
    uint32_t shift = 0;
    while ((uint64_t(1) << shift) < d) ++shift;
    const uint64_t mul = ((uint64_t(1) << 32) * ((uint64_t(1) << shift) - d)) / d + 1;
    return FastDiv{uint32_t(mul), shift};
}

kvx_status kvx::derive_shape(const kvx_desc& d, Shape& s)
{
    s = Shape();
    s.hs = heads_per_rank(d.num_kv_heads, d.src_tp);
    s.hd = heads_per_rank(d.num_kv_heads, d.dst_tp);
    s.esz_src = dtype_size(d.src_dtype);
    s.esz_dst = dtype_size(d.dst_dtype);
    s.conv = pick_conv(d.src_dtype, d.dst_dtype);
    s.cache_dtype = cache_dtype_of(d);
    s.esz_cache = dtype_size(s.cache_dtype);
    s.dequant = s.cache_dtype != d.dst_dtype;

    // parallel-strategy alignment: decode head i -> global head g -> (shard j,
    // head h within it); runs of decode heads with the same shard and
    // consecutive h form one head segment
    const int H = d.num_kv_heads;
    for (int i = 0; i < s.hd; ++i) {
        const int g = d.dst_tp <= H ? d.dst_rank * s.hd + i : d.dst_rank / (d.dst_tp / H);
        const int j = d.src_tp <= H ? g / s.hs : g * (d.src_tp / H);  // first replica
        const int h = d.src_tp <= H ? g % s.hs : 0;
        int slot = 0;
        while (slot < s.nread && s.read_shards[slot] != j) ++slot;
        Segment* last = s.nsegs ? &s.segs[s.nsegs - 1] : nullptr;
        if (last && last->slot == slot && last->h0 + last->n == h && last->i0 + last->n == i) {
            ++last->n;
            continue;
        }
        if (s.nsegs == kMaxReadShards)  // a new shard also starts a new segment: nread <= nsegs
            return fail(KVX_EUNSUPPORTED, "decode rank needs more than %d head segments",
                        kMaxReadShards);
        if (slot == s.nread) s.read_shards[s.nread++] = j;
        s.segs[s.nsegs++] = Segment{slot, h, i, 1, {0, 0}};
    }
    for (int k = 0; k < s.nsegs; ++k) s.segs[k].div_n = make_fastdiv(uint32_t(s.segs[k].n));

    // lanes per row: the smallest power of two covering the transfer-tensor
    // row's 16-byte chunks (a dequantising lane writes two cache chunks)
    s.cpr = d.head_dim * s.esz_dst / 16;
    while ((1 << s.lg_lpr) < s.cpr) ++s.lg_lpr;
    const int64_t rpp = kThreads >> s.lg_lpr;  // rows per workgroup pass
    int max_n = 0;
    for (int k = 0; k < s.nsegs; ++k) max_n = std::max(max_n, s.segs[k].n);
    s.parts = int32_t((int64_t(d.block_size) * max_n + rpp - 1) / rpp);
    s.parts_unpack = int32_t((int64_t(d.block_size) * s.hd + rpp - 1) / rpp);
    return KVX_OK;
}

namespace {

int conv_for(const kvx_plan_t* p, int mode)
{
    if (mode == kvx::kUnpack) {
        if (p->dequant) {
            if (p->d.dst_dtype == KVX_FP8_E5M2)
                return p->cache_dtype == KVX_BF16 ? kvx::kDq5Bf16 : kvx::kDq5F16;
            return p->cache_dtype == KVX_BF16 ? kvx::kDq8Bf16 : kvx::kDq8F16;
        }
        return p->esz_dst == 1 ? kvx::kCopy8 : kvx::kCopy16;
    }
    if (mode == kvx::kRepack && p->dequant)
        return qd_conv(p->d.src_dtype, p->d.dst_dtype, p->cache_dtype);
    return p->conv;
}

// The kernel arguments every launch mode shares, from the descriptor, its
// shape and the work-item table; the source (or transfer-tensor) pointers and
// a paged source's fields are set by the caller.
void fill_args(const kvx_desc& d, const kvx::Shape& s, int mode, uint32_t num_items,
               const Item* items, void* dst, float* scales, const int32_t* bt, int32_t bt_stride,
               int layer_shift, kvx::KArgs& a)
{
    a.dst = dst;
    a.dscale = scales;
    a.items = items;
    a.bt = bt;
    a.num_items = num_items;
    a.planes = uint32_t(2 * d.num_layers);
    a.src_plane0 = uint32_t(2 * (d.src_layer_offset + layer_shift));
    a.dst_plane0 = uint32_t(2 * (d.dst_layer_offset + layer_shift));
    if (mode == kvx::kUnpack) {  // transfer-tensor rows are already in decode order
        a.num_segs = 1;
        a.parts = uint32_t(s.parts_unpack);
        a.seg[0] = kvx::Segment{0, 0, 0, s.hd, kvx::make_fastdiv(uint32_t(s.hd))};
    } else {
        a.num_segs = uint32_t(s.nsegs);
        a.parts = uint32_t(s.parts);
        for (int k = 0; k < s.nsegs; ++k) a.seg[k] = s.segs[k];
    }
    const int64_t units = int64_t(num_items) * a.planes * a.num_segs * a.parts;
    a.units = uint32_t(units);
    a.units_per_xcd = uint32_t((units + kvx::kXcds - 1) / kvx::kXcds);
    a.div_parts = kvx::make_fastdiv(a.parts);
    a.div_segs = kvx::make_fastdiv(a.num_segs);
    a.div_items = kvx::make_fastdiv(a.num_items);
    a.div_bs = kvx::make_fastdiv(uint32_t(d.block_size));
    a.num_blocks = d.num_blocks;
    a.plane_bytes = d.num_blocks * d.block_size * int64_t(s.hd) * d.head_dim * s.esz_cache;
    a.plane_scales = d.num_blocks * d.block_size * int64_t(s.hd);
    a.bt_stride = bt_stride;
    a.block_size = d.block_size;
    a.hs = s.hs;
    a.hd = s.hd;
    a.head_dim = d.head_dim;
    a.row_wire_bytes = d.head_dim * s.esz_dst;
    a.row_dst_bytes = mode == kvx::kPack ? a.row_wire_bytes : d.head_dim * s.esz_cache;
    a.cpr = s.cpr;
    a.lg_lpr = s.lg_lpr;
}

// Shared argument checks of the launch calls; fills the kernel arguments.
// `paged_call` tells whether the entry point is a _paged one; it must match
// the plan's source order (the unpack reads no source and takes either).
kvx_status prepare(const kvx_plan_t* p, int mode, bool paged_call, const void* const* shards,
                   const int32_t* sbt, int32_t sbt_stride, const void* wire, void* dst,
                   float* scales, const int32_t* bt, int32_t bt_stride, kvx::KArgs& a,
                   int layer_shift = 0)
{
    if (!p) return fail(KVX_EINVAL, "NULL plan");
    const bool fp8 = is_fp8(p->cache_dtype);  // the cache holds scales
    const bool paged = p->d.src_order == KVX_PAGED;
    std::memset(&a, 0, sizeof a);
    if (mode != kvx::kUnpack && paged != paged_call)
        return fail(KVX_EINVAL, paged ? "the plan's source is paged: use kvx_pack_paged / kvx_repack_paged"
                                      : "the plan's source is not paged: use kvx_pack / kvx_repack");
    if (p->items.empty()) return KVX_OK;  // nothing to read or write: pointers are not used
    if (mode != kvx::kUnpack && paged) {
        if (!sbt) return fail(KVX_EINVAL, "NULL source block table");
        if (sbt_stride < p->max_src_blocks)
            return fail(KVX_EINVAL, "src_bt_stride %d < max_src_blocks_per_request %d", sbt_stride,
                        p->max_src_blocks);
    }
    if (mode != kvx::kUnpack) {
        if (!shards) return fail(KVX_EINVAL, "NULL src_shards array");
        for (size_t k = 0; k < p->read_shards.size(); ++k) {
            const int j = p->read_shards[k];
            const void* s = shards[j];
            if (!s) return fail(KVX_EINVAL, "src_shards[%d] is NULL", j);
            if (!aligned16(s)) return fail(KVX_EINVAL, "src_shards[%d] is not 16-byte aligned", j);
            a.src[k] = s;
        }
    } else {
        if (!wire) return fail(KVX_EINVAL, "NULL transfer tensor");
        if (!aligned16(wire)) return fail(KVX_EINVAL, "transfer tensor not 16-byte aligned");
        a.wire_in = wire;
    }
    if (!dst) return fail(KVX_EINVAL, mode == kvx::kPack ? "NULL transfer tensor" : "NULL cache");
    if (!aligned16(dst)) return fail(KVX_EINVAL, "destination not 16-byte aligned");
    if (mode != kvx::kPack) {
        if (fp8 != (scales != nullptr))
            return fail(KVX_EINVAL, fp8 ? "8-bit cache needs a scales buffer"
                                        : "scales given for a 16-bit cache");
        if (scales && !aligned16(scales)) return fail(KVX_EINVAL, "scales not 16-byte aligned");
        if (!p->items.empty() && !bt) return fail(KVX_EINVAL, "NULL block table");
        if (bt_stride < p->max_blocks)
            return fail(KVX_EINVAL, "bt_stride %d < max_blocks_per_request %d", bt_stride,
                        p->max_blocks);
    }
    if (p->device < 0) return fail(KVX_EDEVICE, "plan has no device tables (no HIP device)");
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess || cur != p->device)
        return fail(KVX_EDEVICE, "current device %d is not the plan's device %d", cur, p->device);

    const kvx_desc& d = p->d;
    fill_args(d, p->sh, mode, uint32_t(p->items.size()), p->dev_items, dst, scales, bt, bt_stride,
              layer_shift, a);
    if (mode != kvx::kUnpack && paged) {
        a.sbt = sbt;
        a.sbt_stride = sbt_stride;
        a.src_block_size = d.src_block_size;
        a.src_num_blocks = d.src_num_blocks;
        a.div_sbs = kvx::make_fastdiv(uint32_t(d.src_block_size));
        // A part of a segment of n heads covers rows [part*rpp, (part+1)*rpp),
        // i.e. tokens from part*rpp/n on.  When n divides rpp, a part holds
        // rpp/n whole tokens starting at a multiple of rpp/n; when rpp/n also
        // divides both page sizes, those tokens never straddle a source page.
        const int rpp = kvx::kThreads >> a.lg_lpr;
        bool uniform = true;
        for (const kvx::Segment& g : p->segs)
            if (rpp % g.n || d.src_block_size % (rpp / g.n) || d.block_size % (rpp / g.n))
                uniform = false;
        a.sbt_uniform = uniform;
    }
    return KVX_OK;
}

kvx_status run(const kvx_plan_t* p, int mode, const kvx::KArgs& a, void* stream)
{
    if (p->items.empty()) return KVX_OK;
    const int err = kvx::launch(mode, conv_for(p, mode), p->d.src_order, a, stream);
    if (err != 0)
        return fail(KVX_EDEVICE, "kernel launch failed: %s", hipGetErrorString(hipError_t(err)));
    return KVX_OK;
}

}  // namespace

kvx_status kvx::launch_shifted(const kvx_plan_t* p, int mode, int layer_shift,
                               const void* const* shards, const int32_t* sbt, int32_t sbt_stride,
                               const void* wire, void* dst, float* scales, const int32_t* bt,
                               int32_t bt_stride, void* stream)
{
    kvx::KArgs a;
    const bool paged = p && p->d.src_order == KVX_PAGED;
    kvx_status st = prepare(p, mode, paged, shards, sbt, sbt_stride, wire, dst, scales, bt,
                            bt_stride, a, layer_shift);
    return st != KVX_OK ? st : run(p, mode, a, stream);
}

extern "C" {

kvx_status kvx_pack(const kvx_plan_t* p, const void* const* shards, void* wire, void* stream)
{
    kvx::KArgs a;
    kvx_status st = prepare(p, kvx::kPack, false, shards, nullptr, 0, nullptr, wire, nullptr,
                            nullptr, 0, a);
    return st != KVX_OK ? st : run(p, kvx::kPack, a, stream);
}

kvx_status kvx_unpack(const kvx_plan_t* p, const void* wire, void* cache, float* scales,
                      const int32_t* bt, int32_t bt_stride, void* stream)
{
    kvx::KArgs a;
    kvx_status st = prepare(p, kvx::kUnpack, false, nullptr, nullptr, 0, wire, cache, scales, bt,
                            bt_stride, a);
    return st != KVX_OK ? st : run(p, kvx::kUnpack, a, stream);
}

kvx_status kvx_repack(const kvx_plan_t* p, const void* const* shards, void* cache, float* scales,
                      const int32_t* bt, int32_t bt_stride, void* stream)
{
    kvx::KArgs a;
    kvx_status st = prepare(p, kvx::kRepack, false, shards, nullptr, 0, nullptr, cache, scales,
                            bt, bt_stride, a);
    return st != KVX_OK ? st : run(p, kvx::kRepack, a, stream);
}

kvx_status kvx_pack_paged(const kvx_plan_t* p, const void* const* shards, const int32_t* sbt,
                          int32_t sbt_stride, void* wire, void* stream)
{
    kvx::KArgs a;
    kvx_status st = prepare(p, kvx::kPack, true, shards, sbt, sbt_stride, nullptr, wire, nullptr,
                            nullptr, 0, a);
    return st != KVX_OK ? st : run(p, kvx::kPack, a, stream);
}

kvx_status kvx_repack_paged(const kvx_plan_t* p, const void* const* shards, const int32_t* sbt,
                            int32_t sbt_stride, void* cache, float* scales, const int32_t* bt,
                            int32_t bt_stride, void* stream)
{
    kvx::KArgs a;
    kvx_status st = prepare(p, kvx::kRepack, true, shards, sbt, sbt_stride, nullptr, cache, scales,
                            bt, bt_stride, a);
    return st != KVX_OK ? st : run(p, kvx::kRepack, a, stream);
}

kvx_status kvx_repack_noalloc(const kvx_desc* desc, const void* const* shards, void* cache,
                              float* scales, const int32_t* bt, int32_t bt_stride, void* stream)
{
    if (!desc) return fail(KVX_EINVAL, "NULL desc");
    kvx_status st = validate(desc);
    if (st != KVX_OK) return st;
    const kvx_desc& d = *desc;
    if (d.src_order == KVX_PAGED)
        return fail(KVX_EINVAL, "kvx_repack_noalloc reads token- or head-major sources");
    if (d.num_requests > kvx::kNoAllocRequests)
        return fail(KVX_EUNSUPPORTED, "kvx_repack_noalloc takes at most %d requests (%d given)",
                    kvx::kNoAllocRequests, d.num_requests);
    kvx::Shape s;
    st = kvx::derive_shape(d, s);
    if (st != KVX_OK) return st;
    int64_t items = 0, max_blocks = 0;
    for (int r = 0; r < d.num_requests; ++r) {
        const int64_t nb = (int64_t(d.seq_lens[r]) + d.block_size - 1) / d.block_size;
        items += nb;
        max_blocks = std::max(max_blocks, nb);
    }
    if (items > kvx::kNoAllocItems)
        return fail(KVX_EUNSUPPORTED,
                    "kvx_repack_noalloc takes at most %d pages (%lld given): its work-item table "
                    "is a static array of that many entries", kvx::kNoAllocItems,
                    (long long)items);
    if (items == 0) return KVX_OK;  // nothing to read or write: pointers are not used
    if (items * 2 * d.num_layers * int64_t(s.nsegs) * s.parts > kvx::kMaxUnits)
        return fail(KVX_EUNSUPPORTED, "more than %lld work units (pages x 2 x layers x parts)",
                    (long long)kvx::kMaxUnits);

    kvx::KArgs a;
    std::memset(&a, 0, sizeof a);
    if (!shards) return fail(KVX_EINVAL, "NULL src_shards array");
    for (int k = 0; k < s.nread; ++k) {
        const int j = s.read_shards[k];
        if (!shards[j]) return fail(KVX_EINVAL, "src_shards[%d] is NULL", j);
        if (!aligned16(shards[j])) return fail(KVX_EINVAL, "src_shards[%d] is not 16-byte aligned", j);
        a.src[k] = shards[j];
    }
    const bool fp8 = is_fp8(s.cache_dtype);  // the cache holds scales
    if (!cache) return fail(KVX_EINVAL, "NULL cache");
    if (!aligned16(cache)) return fail(KVX_EINVAL, "destination not 16-byte aligned");
    if (fp8 != (scales != nullptr))
        return fail(KVX_EINVAL, fp8 ? "8-bit cache needs a scales buffer"
                                    : "scales given for a 16-bit cache");
    if (scales && !aligned16(scales)) return fail(KVX_EINVAL, "scales not 16-byte aligned");
    if (!bt) return fail(KVX_EINVAL, "NULL block table");
    if (bt_stride < max_blocks)
        return fail(KVX_EINVAL, "bt_stride %d < max_blocks_per_request %lld", bt_stride,
                    (long long)max_blocks);

    kvx::Item* table = nullptr;
    int e = kvx::scratch_items(&table);
    if (e != 0)
        return fail(KVX_EDEVICE, "static work-item table: %s", hipGetErrorString(hipError_t(e)));
    kvx::ItemsArgs ia;
    std::memset(&ia, 0, sizeof ia);
    for (int r = 0; r < d.num_requests; ++r) ia.lens[r] = d.seq_lens[r];
    ia.num_requests = d.num_requests;
    ia.block_size = d.block_size;
    ia.src_elems_per_token = 2 * int64_t(src_layers_of(d)) * s.hs * d.head_dim;
    ia.items = table;
    e = kvx::build_items(ia, stream);
    if (e != 0)
        return fail(KVX_EDEVICE, "work-item launch failed: %s", hipGetErrorString(hipError_t(e)));
    fill_args(d, s, kvx::kRepack, uint32_t(items), table, cache, scales, bt, bt_stride, 0, a);
    const int conv = s.dequant ? qd_conv(d.src_dtype, d.dst_dtype, s.cache_dtype) : s.conv;
    e = kvx::launch(kvx::kRepack, conv, d.src_order, a, stream);
    if (e != 0)
        return fail(KVX_EDEVICE, "kernel launch failed: %s", hipGetErrorString(hipError_t(e)));
    return KVX_OK;
}

}  // extern "C"
