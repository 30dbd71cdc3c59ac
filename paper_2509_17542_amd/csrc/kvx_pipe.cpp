// Layer-streamed transfer through a pinned host ring: the plan's layers move
// in chunks, each packed straight into a slot of pinned host memory (the pack
// kernel's stores cross the host link), copied into a device receive slot and
// unpacked, with the stages of consecutive chunks overlapped on the pipe's
// three streams.  Writing the host slot from the kernel leaves the copy
// engines one direction only: two copies in opposite directions overlapped in
// some processes and ran one after the other in others.
//
// Each stage has a stream with a CU mask of its own: the pack on half the
// CUs, the host-to-device copy (which HIP runs as a blit kernel) and the
// unpack on a quarter each.  A pack bound by the host link keeps its
// workgroups resident for long; with all three stages free to use every CU,
// the copy of one chunk sometimes waited for CUs behind the next pack, and
// whether it did depended on how HIP had mapped the streams onto hardware
// queues (on the streams the process created earlier).  CU-masked streams
// block with the null stream like streams created without flags.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "kvx.h"
#include "kvx_host.h"
#include "kvx_internal.h"

struct kvx_pipe_s {
    const kvx_plan_t* plan = nullptr;
    int chunk_layers = 0, num_chunks = 0, slots = 0, device = -1;
    kvx_plan_t* full = nullptr;   // plan of chunk_layers layers
    kvx_plan_t* tail = nullptr;   // plan of the last, shorter chunk (or none)
    uint64_t slot_bytes = 0, bus_bytes = 0;
    char* host = nullptr;         // pinned ring, slots x slot_bytes, mapped for the device
    char* host_dev = nullptr;     // the ring's device address (the pack writes through it)
    char* recv = nullptr;         // device, slots x slot_bytes
    hipStream_t pack = nullptr, h2d = nullptr, unpack = nullptr;
    hipEvent_t start = nullptr;
    hipEvent_t ends[3] = {};      // the end of the last run on pack, h2d, unpack
    bool ran = false;             // ends hold a run
    std::vector<hipEvent_t> packed, received, unpacked;  // one per slot
};

namespace {

using kvx::fail;

void release(kvx_pipe_s* q)
{
    if (!q) return;
    for (hipStream_t s : {q->pack, q->h2d, q->unpack})
        if (s) (void)hipStreamSynchronize(s);
    for (auto* v : {&q->packed, &q->received, &q->unpacked})
        for (hipEvent_t e : *v)
            if (e) (void)hipEventDestroy(e);
    if (q->start) (void)hipEventDestroy(q->start);
    for (hipEvent_t e : q->ends)
        if (e) (void)hipEventDestroy(e);
    for (hipStream_t s : {q->pack, q->h2d, q->unpack})
        if (s) (void)hipStreamDestroy(s);
    if (q->host) (void)hipHostFree(q->host);
    if (q->recv) (void)hipFree(q->recv);
    kvx_plan_destroy(q->full);
    kvx_plan_destroy(q->tail);
    delete q;
}

// Plan of n layers starting where the parent plan's layers start; its launches
// are shifted to the chunk's first layer.
kvx_status chunk_plan(const kvx_plan_t* p, int n, kvx_plan_t** out)
{
    kvx_desc d = p->d;
    d.src_layers = d.src_layers ? d.src_layers : d.num_layers;
    d.dst_layers = d.dst_layers ? d.dst_layers : d.num_layers;
    d.num_layers = n;
    return kvx_plan(&d, out);
}

bool ok(hipError_t e) { return e == hipSuccess; }

// A stream whose kernels run on the CUs selected by `byte_mask` in every byte
// position it covers: CU i belongs to the stream when bit (i / 8) % 4 of
// byte_mask is set, so each of the 8 XCDs contributes CUs to it whether the
// mask's bits are dealt to the XCDs in runs of 32 or round-robin.  A device
// too small to give the stream any CU this way gives it all of them.
bool masked_stream(int device, unsigned byte_mask, hipStream_t* out)
{
    int cus = 0;
    if (!ok(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device)) ||
        cus <= 0)
        return false;
    std::vector<uint32_t> mask(size_t((cus + 31) / 32), 0u);
    bool any = false;
    for (int i = 0; i < cus; ++i)
        if ((byte_mask >> ((i / 8) % 4)) & 1u) {
            mask[size_t(i / 32)] |= 1u << (i % 32);
            any = true;
        }
    if (!any)
        for (int i = 0; i < cus; ++i) mask[size_t(i / 32)] |= 1u << (i % 32);
    return ok(hipExtStreamCreateWithCUMask(out, uint32_t(mask.size()), mask.data()));
}

// The legacy null stream needs no event either way: the pipe's streams,
// created without the non-blocking flag, start after its earlier work and its
// later work waits for them.  Any other caller stream gets an event each way.
bool legacy_stream(hipStream_t s) { return s == nullptr || s == hipStreamLegacy; }

// Records the end of this run on each of the pipe's streams; the next run's
// streams wait for all three, so runs of one pipe never overlap (they share
// the slots).
bool mark_ends(kvx_pipe_s* q)
{
    const hipStream_t st[3] = {q->pack, q->h2d, q->unpack};
    bool good = true;
    for (int i = 0; i < 3; ++i) good = ok(hipEventRecord(q->ends[i], st[i])) && good;
    q->ran = true;
    return good;
}

// A run that fails part way has chunks enqueued on the pipe's streams: the
// caller's stream still waits for them, so that buffers it releases after the
// failure are no longer in use, and so does the pipe's next run.
kvx_status stop(kvx_pipe_s* q, hipStream_t s0, kvx_status st)
{
    mark_ends(q);
    if (!legacy_stream(s0))
        for (hipEvent_t e : q->ends) (void)hipStreamWaitEvent(s0, e, 0);
    return st;
}

}  // namespace

extern "C" {

kvx_status kvx_pipe_create(const kvx_plan_t* p, int32_t chunk_layers, int32_t slots,
                           kvx_pipe_t** out)
{
    if (!p || !out) return fail(KVX_EINVAL, "NULL plan or out");
    *out = nullptr;
    const int L = p->d.num_layers;
    if (chunk_layers < 1 || chunk_layers > L)
        return fail(KVX_EINVAL, "chunk_layers %d outside [1, %d]", chunk_layers, L);
    if (slots < 1) return fail(KVX_EINVAL, "slots must be >= 1");
    if (p->items.empty()) {
        // no tokens: nothing to move, as for the plan's own launches; the pipe
        // holds no buffers, streams or events, and its runs return at once
        kvx_pipe_s* q = new (std::nothrow) kvx_pipe_s();
        if (!q) return fail(KVX_ENOMEM, "host allocation failed");
        q->plan = p;
        q->chunk_layers = chunk_layers;
        q->num_chunks = (L + chunk_layers - 1) / chunk_layers;
        q->slots = slots;
        q->device = p->device;
        *out = q;
        return KVX_OK;
    }
    if (p->device < 0) return fail(KVX_EDEVICE, "plan has no device tables (no HIP device)");
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess || cur != p->device)
        return fail(KVX_EDEVICE, "current device %d is not the plan's device %d", cur, p->device);

    kvx_pipe_s* q = new (std::nothrow) kvx_pipe_s();
    if (!q) return fail(KVX_ENOMEM, "host allocation failed");
    q->plan = p;
    q->chunk_layers = chunk_layers;
    q->num_chunks = (L + chunk_layers - 1) / chunk_layers;
    q->slots = slots;
    q->device = p->device;
    kvx_status st = chunk_plan(p, chunk_layers, &q->full);
    if (st == KVX_OK && L % chunk_layers) st = chunk_plan(p, L % chunk_layers, &q->tail);
    if (st != KVX_OK) {
        release(q);
        return st;
    }
    q->slot_bytes = q->full->wire_bytes;
    q->bus_bytes = uint64_t(L / chunk_layers) * q->full->wire_bytes +
                   (q->tail ? q->tail->wire_bytes : 0);
    const size_t ring = size_t(q->slot_bytes) * size_t(slots);
    if (ring) {
        // mapped pinned memory: the pack kernel stores to the ring through
        // its device address
        if (!ok(hipHostMalloc(reinterpret_cast<void**>(&q->host), ring, hipHostMallocMapped)) ||
            !ok(hipHostGetDevicePointer(reinterpret_cast<void**>(&q->host_dev), q->host, 0)) ||
            !ok(hipMalloc(reinterpret_cast<void**>(&q->recv), ring))) {
            (void)hipGetLastError();
            release(q);
            return fail(KVX_ENOMEM, "pipe buffers (2 x %zu bytes) could not be allocated", ring);
        }
    }
    bool good = masked_stream(q->device, 0x3u, &q->pack) &&    // half the CUs
                masked_stream(q->device, 0x4u, &q->h2d) &&     // a quarter
                masked_stream(q->device, 0x8u, &q->unpack) &&  // a quarter
                ok(hipEventCreateWithFlags(&q->start, hipEventDisableTiming));
    for (hipEvent_t& e : q->ends) good = good && ok(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    for (auto* v : {&q->packed, &q->received, &q->unpacked}) {
        v->assign(size_t(slots), nullptr);
        for (hipEvent_t& e : *v) good = good && ok(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    }
    if (!good) {
        (void)hipGetLastError();
        release(q);
        return fail(KVX_EDEVICE, "pipe streams or events could not be created");
    }
    *out = q;
    return KVX_OK;
}

kvx_status kvx_pipe_info_get(const kvx_pipe_t* q, kvx_pipe_info* info)
{
    if (!q || !info) return fail(KVX_EINVAL, "NULL pipe or info");
    std::memset(info, 0, sizeof *info);
    info->chunk_layers = q->chunk_layers;
    info->num_chunks = q->num_chunks;
    info->slots = q->slots;
    info->slot_bytes = q->slot_bytes;
    info->host_bytes = q->slot_bytes * uint64_t(q->slots);
    info->device_bytes = info->host_bytes;
    info->bus_bytes = q->bus_bytes;
    return KVX_OK;
}

kvx_status kvx_pipe_run(kvx_pipe_t* q, const void* const* shards, const int32_t* sbt,
                        int32_t sbt_stride, void* cache, float* scales, const int32_t* bt,
                        int32_t bt_stride, void* stream)
{
    if (!q) return fail(KVX_EINVAL, "NULL pipe");
    const bool paged = q->plan->d.src_order == KVX_PAGED;
    if (!paged && sbt) return fail(KVX_EINVAL, "source block table given for a contiguous source");
    if (q->plan->items.empty()) return KVX_OK;
    // the checks of the unpack side up front, so that a bad argument is
    // reported before anything is enqueued (the pack side's are the first
    // chunk's pack, which runs first)
    const bool fp8 = q->plan->cache_dtype == KVX_FP8_E4M3FN ||  // the cache holds scales
                     q->plan->cache_dtype == KVX_FP8_E5M2;
    if (!cache || (reinterpret_cast<uintptr_t>(cache) & 15u))
        return fail(KVX_EINVAL, "NULL or misaligned cache");
    if (fp8 != (scales != nullptr) || (reinterpret_cast<uintptr_t>(scales) & 15u))
        return fail(KVX_EINVAL, "scales must be given, 16-byte aligned, exactly for an 8-bit cache");
    if (!bt || bt_stride < q->plan->max_blocks)
        return fail(KVX_EINVAL, "NULL block table or bt_stride below %d", q->plan->max_blocks);
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess || cur != q->device)
        return fail(KVX_EDEVICE, "current device %d is not the pipe's device %d", cur, q->device);
    hipStream_t s0 = static_cast<hipStream_t>(stream);

    // The pipe's streams start after the caller's earlier work (implied for
    // the legacy null stream) and after the pipe's previous run.  Enqueuing
    // nothing on the null stream matters: with event records and waits on it
    // between runs, back-to-back runs measured 2-25% slower, the host
    // sometimes blocking in the enqueue.
    const bool legacy = legacy_stream(s0);
    if (!legacy && !ok(hipEventRecord(q->start, s0)))
        return fail(KVX_EDEVICE, "event record failed");
    for (hipStream_t s : {q->pack, q->h2d, q->unpack}) {
        if (!legacy && !ok(hipStreamWaitEvent(s, q->start, 0)))
            return fail(KVX_EDEVICE, "stream wait failed");
        if (q->ran)
            for (hipEvent_t e : q->ends)
                if (!ok(hipStreamWaitEvent(s, e, 0))) return fail(KVX_EDEVICE, "stream wait failed");
    }

    for (int c = 0; c < q->num_chunks; ++c) {
        const int s = c % q->slots;
        const bool reuse = c >= q->slots;  // slot s held chunk c - slots
        const kvx_plan_t* cp = (q->tail && c == q->num_chunks - 1) ? q->tail : q->full;
        const int shift = c * q->chunk_layers;
        const size_t bytes = size_t(cp->wire_bytes);
        char* host = q->host + size_t(s) * q->slot_bytes;
        char* host_dev = q->host_dev + size_t(s) * q->slot_bytes;
        char* recv = q->recv + size_t(s) * q->slot_bytes;

        // pack into the host slot: the slot's previous chunk must have been
        // copied to the device
        if (reuse && !ok(hipStreamWaitEvent(q->pack, q->received[s], 0)))
            return stop(q, s0, fail(KVX_EDEVICE, "stream wait failed"));
        kvx_status st = kvx::launch_shifted(cp, kvx::kPack, shift, shards, sbt, sbt_stride,
                                            nullptr, host_dev, nullptr, nullptr, 0, q->pack);
        if (st != KVX_OK) return stop(q, s0, st);
        bool good = ok(hipEventRecord(q->packed[s], q->pack));
        // host -> device: the receive slot must have been unpacked
        good = good && ok(hipStreamWaitEvent(q->h2d, q->packed[s], 0));
        if (reuse) good = good && ok(hipStreamWaitEvent(q->h2d, q->unpacked[s], 0));
        good = good && ok(hipMemcpyAsync(recv, host, bytes, hipMemcpyHostToDevice, q->h2d)) &&
               ok(hipEventRecord(q->received[s], q->h2d));
        // unpack
        good = good && ok(hipStreamWaitEvent(q->unpack, q->received[s], 0));
        if (!good)
            return stop(q, s0, fail(KVX_EDEVICE, "copy or event enqueue failed: %s",
                                    hipGetErrorString(hipGetLastError())));
        st = kvx::launch_shifted(cp, kvx::kUnpack, shift, nullptr, nullptr, 0, recv, cache,
                                 scales, bt, bt_stride, q->unpack);
        if (st != KVX_OK) return stop(q, s0, st);
        if (!ok(hipEventRecord(q->unpacked[s], q->unpack)))
            return stop(q, s0, fail(KVX_EDEVICE, "event record failed"));
    }
    // the caller's stream continues after the last unpack (the unpack stream
    // runs its chunks in order, each after its copy and its pack)
    if (!mark_ends(q)) return stop(q, s0, fail(KVX_EDEVICE, "event record failed"));
    if (!legacy && !ok(hipStreamWaitEvent(s0, q->ends[2], 0)))
        return stop(q, s0, fail(KVX_EDEVICE, "stream wait failed"));
    return KVX_OK;
}

kvx_status kvx_pipe_destroy(kvx_pipe_t* q)
{
    release(q);
    return KVX_OK;
}

}  // extern "C"
