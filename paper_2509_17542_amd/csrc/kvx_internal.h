// Internal declarations shared by the host planner (kvx_plan.cpp) and the
// gfx950 kernels (kvx_kernels.hip).
#pragma once

#include <cstdint>

#include "kvx.h"

namespace kvx {

constexpr int kThreads = 256;           // threads per workgroup (4 wave64)
constexpr int kMaxHeadsPerRank = 128;   // Hd limit (kernel-argument head table)
constexpr int kMaxReadShards = 64;      // source shards one decode rank may read
constexpr int kMaxRowChunks = 64;       // 16-byte destination chunks per row (one wave)
constexpr int kMaxItems = (1 << 24) - 1;  // workgroups along grid x (x * 256 threads < 2^32)

// Per request, device resident.
struct ReqInfo {
    int64_t src_base;    // element offset of the request in every source shard
    int64_t wire_data;   // byte offset of its data region in the transfer tensor
    int64_t wire_scale;  // byte offset of its scale region, -1 without scales
    int32_t tokens;      // T_r
    int32_t pad;
};

// One logical page of one request: the unit of work of a workgroup (per plane).
struct Item {
    int32_t req;
    int32_t blk;
};

enum Mode : int { kPack = 0, kUnpack = 1, kRepack = 2 };

// element conversion performed by a launch
enum Conv : int {
    kCopy16 = 0,    // 16-bit bits unchanged
    kF16Bf16 = 1,   // fp16 -> bf16, round to nearest even
    kBf16E4m3 = 2,  // bf16 -> e4m3fn with per-row scale
    kF16E4m3 = 3,   // fp16 -> e4m3fn with per-row scale
    kCopy8 = 4      // 8-bit bits unchanged (+ scale copy), unpack of e4m3fn
};

// Kernel arguments (passed by value through the kernel-argument segment).
struct KArgs {
    const void* src[kMaxReadShards];  // shard first_shard + k at src[k]
    const void* wire_in;              // unpack source
    void* dst;                        // pack: transfer tensor; else cache
    float* dscale;                    // cache scales (unpack/repack, e4m3fn)
    const Item* items;
    const ReqInfo* reqs;
    const int32_t* bt;
    int64_t num_blocks;
    int64_t plane_bytes;              // cache bytes per (layer, k/v) plane
    int64_t plane_scales;             // cache scales per plane
    int32_t bt_stride;
    int32_t block_size;
    int32_t hs;                       // heads per source shard
    int32_t hd;                       // heads per decode rank
    int32_t head_dim;
    int32_t row_dst_bytes;            // head_dim * dst element size
    int32_t cpr;                      // 16-byte destination chunks per row
    int32_t lg_lpr;                   // log2(lanes per row), lanes per row >= cpr
    int32_t dq, dr;                   // (rows per pass) / hd and % hd
    uint32_t head_src[kMaxHeadsPerRank];  // (shard slot << 16) | head within shard
};

// Launch one conversion; returns a hipError_t value (0 = success).
int launch(int mode, int conv, int order, const KArgs& a, int64_t num_items, int planes,
           void* stream);

}  // namespace kvx
