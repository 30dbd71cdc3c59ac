// Host-side internals shared by the planner (kvx_plan.cpp) and the
// layer-streamed transfer (kvx_pipe.cpp): the plan object, the error setter
// and a launch with shifted layer offsets.  Not part of the C ABI.
#pragma once

#include <cstdint>
#include <vector>

#include "kvx.h"
#include "kvx_internal.h"

namespace kvx {

// What a problem descriptor fixes about the launches, independent of the
// requests' lengths: heads per rank, element sizes, the conversion, the head
// segments and the lanes and passes per row.  Fixed-size, so that it can be
// derived without allocating.
struct Shape {
    int hs = 0, hd = 0, esz_src = 0, esz_dst = 0, conv = 0;
    int cache_dtype = 0, esz_cache = 0;  // the cache's element type (dst_dtype unless dequantising)
    bool dequant = false;                // 8-bit transfer tensor, 16-bit cache
    // lanes per row (from the transfer-tensor row; a dequantising lane covers
    // two 16-byte cache chunks) and workgroup passes per (page, segment)
    int cpr = 0, lg_lpr = 0, parts = 0, parts_unpack = 0;
    int nsegs = 0;                       // head segments of the decode rank
    Segment segs[kMaxReadShards];
    int nread = 0;                       // prefill shards the decode rank reads, in slot order
    int read_shards[kMaxReadShards];
};

}  // namespace kvx

struct kvx_plan_s {
    kvx_desc d;                   // seq_lens points into lens
    kvx::Shape sh;                // the launches' shape (the fields below repeat it)
    std::vector<int32_t> lens;
    std::vector<int64_t> wire_data, wire_scale;  // per request, transfer-tensor offsets
    std::vector<kvx::Item> items;
    int hs = 0, hd = 0, esz_src = 0, esz_dst = 0, conv = 0;
    int cache_dtype = 0, esz_cache = 0;  // the cache's element type (dst_dtype unless dequantising)
    bool dequant = false;                // 8-bit transfer tensor, 16-bit cache
    std::vector<int> read_shards;  // prefill shards the decode rank reads, in slot order
    // lanes per row (from the transfer-tensor row; a dequantising lane covers
    // two 16-byte cache chunks) and workgroup passes per (page, segment)
    int cpr = 0, lg_lpr = 0, parts = 0, parts_unpack = 0;
    std::vector<kvx::Segment> segs;  // head segments of the decode rank
    int32_t max_blocks = 0;
    int32_t max_src_blocks = 0;   // paged sources: pages per request on the prefill side
    uint64_t wire_bytes = 0;
    int64_t src_elems = 0;        // elements of a read source shard the launches may touch
    int64_t total_tokens = 0;
    int64_t elems_rows = 0;       // sum over requests of L*2*T*Hd
    int device = -1;
    void* dev_table = nullptr;    // device copy of items
    const kvx::Item* dev_items = nullptr;
};

namespace kvx {

// The shape of a validated descriptor; KVX_EUNSUPPORTED when the decode rank
// needs more than kMaxReadShards head segments.
kvx_status derive_shape(const kvx_desc& d, Shape& s);

// Sets the calling thread's last-error message; returns s.
kvx_status fail(kvx_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// One pack / unpack / repack launch of plan p with both sides' layer offsets
// moved by layer_shift layers (the layers of a chunk of a larger plan); the
// argument checks of the public calls apply.  The source is paged exactly
// when the plan's is.
kvx_status launch_shifted(const kvx_plan_t* p, int mode, int layer_shift,
                          const void* const* shards, const int32_t* sbt, int32_t sbt_stride,
                          const void* wire, void* dst, float* scales, const int32_t* bt,
                          int32_t bt_stride, void* stream);

}  // namespace kvx
