// Internal declarations shared by the host planner (kvx_plan.cpp) and the
// gfx950 kernels (kvx_kernels.hip).
#pragma once

#include <cstdint>

#include "kvx.h"

namespace kvx {

constexpr int kThreads = 256;           // threads per workgroup (4 wave64)
constexpr int kMaxHeadsPerRank = 1024;  // Hd limit
constexpr int kMaxReadShards = 64;      // head segments (and so source shards) of a decode rank
constexpr int kMaxRowChunks = 64;       // 16-byte destination chunks per row (one wave)
constexpr int kXcds = 8;                // MI355X: workgroups are dealt round-robin to 8 XCDs
constexpr int kPrefetchPages = 32;      // pages ahead whose address translation a workgroup warms
// work units of one launch; the 1-D grid is this rounded up to a multiple of
// kXcds, and grid * kThreads stays below 2^32
constexpr int64_t kMaxUnits = (int64_t(1) << 24) - kXcds;

// Division by an invariant divisor d >= 1 (Granlund and Montgomery, 1994):
// n / d = (mulhi(n, mul) + n) >> shift for every 32-bit n, with
// shift = ceil(log2 d) and mul = floor(2^32 (2^shift - d) / d) + 1.
struct FastDiv {
    uint32_t mul;
    uint32_t shift;
};

// One logical page of one request, device resident: the unit of work of a
// workgroup in every (layer, k/v) plane.
struct Item {
    int64_t src_base;    // element offset of the request in every source shard (0 if paged)
    int64_t wire_data;   // byte offset of the request's data region in the transfer tensor
    int64_t wire_scale;  // byte offset of its scale region, -1 without scales
    int32_t req;         // request index (block-table row)
    int32_t blk;         // page index within the request
    int32_t tokens;      // T_r
    int32_t pad;
};

enum Mode : int { kPack = 0, kUnpack = 1, kRepack = 2 };

// element conversion performed by a launch
enum Conv : int {
    kCopy16 = 0,    // 16-bit bits unchanged
    kF16Bf16 = 1,   // fp16 -> bf16, round to nearest even
    kBf16E4m3 = 2,  // bf16 -> e4m3fn with per-row scale
    kF16E4m3 = 3,   // fp16 -> e4m3fn with per-row scale
    kCopy8 = 4,     // 8-bit bits unchanged (+ scale copy), unpack of an 8-bit format
    kBf16F16 = 5,   // bf16 -> fp16, round to nearest even, overflow to infinity
    // dequantising unpack: e4m3fn transfer tensor (+ scales) -> 16-bit cache
    kDq8Bf16 = 6,
    kDq8F16 = 7,
    // repack into a 16-bit cache through e4m3fn: quantise, then dequantise
    kQdBf16Bf16 = 8,
    kQdF16Bf16 = 9,
    kQdBf16F16 = 10,
    kQdF16F16 = 11,
    // the same with OCP e5m2 codes (scale max|x| / 57344)
    kBf16E5m2 = 12,
    kF16E5m2 = 13,
    kDq5Bf16 = 14,
    kDq5F16 = 15,
    kQd5Bf16Bf16 = 16,
    kQd5F16Bf16 = 17,
    kQd5Bf16F16 = 18,
    kQd5F16F16 = 19
};

// A run of the decode rank's heads that comes from one source shard: decode
// heads [i0, i0 + n) are heads [h0, h0 + n) of the shard at src[slot].
struct Segment {
    int32_t slot;
    int32_t h0;
    int32_t i0;
    int32_t n;
    FastDiv div_n;
};

// Kernel arguments (passed by value through the kernel-argument segment).
struct KArgs {
    const void* src[kMaxReadShards];  // the k-th shard the decode rank reads at src[k]
    Segment seg[kMaxReadShards];      // pack/repack: the head segments; unpack: one, all heads
    const void* wire_in;              // unpack source
    void* dst;                        // pack: transfer tensor; else cache
    float* dscale;                    // cache scales (unpack/repack into an 8-bit cache)
    const Item* items;
    const int32_t* bt;
    int64_t num_blocks;
    int64_t plane_bytes;              // cache bytes per (layer, k/v) plane
    int64_t plane_scales;             // cache scales per plane
    uint32_t units;                   // work units: planes x pages x segments x parts
    uint32_t units_per_xcd;           // grid / kXcds
    uint32_t num_items;               // logical pages per plane
    uint32_t planes;                  // 2 x converted layers
    uint32_t src_plane0;              // 2 x source layer offset (pipeline stages)
    uint32_t dst_plane0;              // 2 x cache layer offset
    uint32_t num_segs;
    uint32_t parts;                   // workgroup passes per (page, segment)
    FastDiv div_parts, div_segs, div_items, div_bs;
    int32_t bt_stride;
    int32_t block_size;
    int32_t hs;                       // heads per source shard
    int32_t hd;                       // heads per decode rank
    int32_t head_dim;
    int32_t row_dst_bytes;            // pack: transfer-tensor row bytes; else cache row bytes
    int32_t row_wire_bytes;           // transfer-tensor row bytes (the unpack's source rows)
    int32_t cpr;                      // 16-byte transfer-tensor chunks per row
    int32_t lg_lpr;                   // log2(lanes per row), lanes per row >= cpr
    // paged sources: the prefill side's pages
    const int32_t* sbt;               // source block table [requests][sbt_stride]
    int64_t src_num_blocks;           // pages per plane of each shard's pool
    int32_t sbt_stride;
    int32_t src_block_size;
    FastDiv div_sbs;
    int32_t sbt_uniform;              // every part lies in one source page
};

// Launch one conversion over a.units work units; returns a hipError_t value.
int launch(int mode, int conv, int order, const KArgs& a, void* stream);

// The allocation-free repack keeps its work-item table in a static device
// array of kNoAllocItems entries (40 B each: 2.5 MiB per device) and takes at
// most kNoAllocRequests requests, whose lengths travel in the arguments of the
// kernel that writes that table.
constexpr int kNoAllocItems = 65536;
constexpr int kNoAllocRequests = 256;

struct ItemsArgs {
    int32_t lens[kNoAllocRequests];   // tokens per request
    int32_t num_requests;
    int32_t block_size;               // destination page size
    int64_t src_elems_per_token;      // elements of one token in a source shard (2 x layers x Hs x D)
    Item* items;                      // the table to write
};

// The current device's static work-item table; the address is looked up once
// per device.  Returns a hipError_t value.
int scratch_items(Item** out);

// Enqueue the kernel that writes the work-item table of a.lens (one page of
// a request per item, requests in order) on `stream`.  Returns a hipError_t
// value.
int build_items(const ItemsArgs& a, void* stream);

FastDiv make_fastdiv(uint32_t d);

}  // namespace kvx
