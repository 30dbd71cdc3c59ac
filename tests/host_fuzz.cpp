// Host-side fuzz of the library's host code (kvx_plan.cpp, kvx_pd.cpp,
// kvx_pipe.cpp) under AddressSanitizer and UndefinedBehaviorSanitizer, built
// by tests/test_host_sanitizers.py with g++ (no GPU code: without a device,
// plans are host-only and the launch calls return KVX_EDEVICE before any
// kernel, so the kernel entry below is never reached).
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>
#include "kvx.h"
#include "kvx_internal.h"

namespace kvx {
int launch(int, int, int, const KArgs&, void*) { std::abort(); }  // never reached without a device
// the allocation-free repack's static table: no device here, as on a CPU machine
int scratch_items(Item**) { return int(hipErrorNoDevice); }
int build_items(const ItemsArgs&, void*) { std::abort(); }      // never reached without a table
}

int main()
{
    std::mt19937_64 rng(17542);
    auto pick = [&](std::initializer_list<int> v) { return *(v.begin() + rng() % v.size()); };
    auto pick64 = [&](std::initializer_list<int64_t> v) { return *(v.begin() + rng() % v.size()); };
    int ok = 0, rejected = 0;
    for (int it = 0; it < 100000; ++it) {
        std::vector<int32_t> lens(rng() % 6);
        for (auto& t : lens) t = int32_t(rng() % 300) - (rng() % 50 == 0 ? 5 : 0);
        kvx_desc d{};
        d.num_layers = pick({0, 1, 2, 3, 80, 40000});
        d.num_kv_heads = pick({1, 2, 4, 6, 8, 64, 1024, 4096});
        d.head_dim = pick({0, 4, 8, 16, 48, 64, 80, 128, 512, 1024, 2048});
        d.src_tp = pick({0, 1, 2, 3, 4, 8, 16, 64});
        d.dst_tp = pick({1, 2, 3, 4, 8, 16});
        d.dst_rank = int32_t(rng() % 20) - 2;
        d.src_dtype = pick({1, 2, 3, 4, 7});
        d.dst_dtype = pick({1, 2, 3, 4, 9});
        d.src_order = pick({0, 1, 2, 5});
        d.block_size = pick({0, 1, 5, 16, 64});
        d.num_blocks = pick64({0, 1, 64, 1 << 20, int64_t(1) << 45, int64_t(1) << 62});
        d.num_requests = int32_t(lens.size());
        d.seq_lens = lens.empty() ? nullptr : lens.data();
        d.src_block_size = pick({0, 5, 16});
        d.src_num_blocks = pick64({0, 8, 4096, int64_t(1) << 50});
        d.src_layer_offset = pick({0, 0, 1, -1});
        d.src_layers = pick({0, 0, 2, 100});
        d.dst_layer_offset = pick({0, 0, 2});
        d.dst_layers = pick({0, 0, 3, 100});
        d.cache_dtype = pick({0, 0, 1, 2, 3, 4, 6});
        // the allocation-free repack validates the same descriptor itself;
        // aligned stand-in pointers are never dereferenced on the host
        {
            std::vector<const void*> sh(size_t(std::max(d.src_tp, 1)),
                                        reinterpret_cast<const void*>(uintptr_t(0x10000)));
            void* c = reinterpret_cast<void*>(uintptr_t(0x20000));
            float* sc = (it & 1) ? reinterpret_cast<float*>(uintptr_t(0x30000)) : nullptr;
            const int32_t* t = reinterpret_cast<const int32_t*>(uintptr_t(0x40000));
            const kvx_status st = kvx_repack_noalloc(&d, sh.data(), c, sc, t, 1 << 20, nullptr);
            if (st == KVX_OK) {
                int64_t tokens = 0;
                for (int32_t x : lens) tokens += x;
                if (tokens != 0) std::abort();   // only an empty problem needs no device
            }
        }
        kvx_plan_t* p = nullptr;
        if (kvx_plan(&d, &p) != KVX_OK) { ++rejected; continue; }
        ++ok;
        kvx_plan_info info;
        kvx_plan_info_get(p, &info);
        kvx_buffer_sizes sz;
        kvx_plan_buffer_sizes(p, &sz);
        for (int j = -1; j <= d.src_tp; ++j) {
            uint64_t n = 0;
            kvx_plan_shard_bytes(p, j, &n);
        }
        for (int r = -1; r <= d.num_requests; ++r) {
            int64_t a, b;
            kvx_plan_segment(p, r, &a, &b);
        }
        std::vector<int32_t> bt(size_t(d.num_requests) * (info.max_blocks_per_request + 1));
        for (size_t k = 0; k < bt.size(); ++k) bt[k] = int32_t(k) - 1;
        kvx_check_block_table(p, bt.data(), info.max_blocks_per_request + 1);
        if (d.src_order == KVX_PAGED)
            kvx_check_src_block_table(p, bt.data(), info.max_src_blocks_per_request);
        kvx_pipe_t* q = nullptr;
        // host-only plan: EDEVICE, unless it has no tokens (a pipe that moves
        // nothing, whose run returns at once)
        if (kvx_pipe_create(p, 1, 2, &q) == KVX_OK) {
            if (kvx_pipe_run(q, nullptr, nullptr, 0, nullptr, nullptr, nullptr, 0, nullptr) !=
                KVX_OK) {
                std::printf("pipe of a plan without tokens failed to run\n");
                return 1;
            }
            kvx_pipe_destroy(q);
        }
        kvx_plan_destroy(p);
    }
    // mostly valid problems: every head map, order, dtype and layer range
    for (int it = 0; it < 50000; ++it) {
        std::vector<int32_t> lens(1 + rng() % 5);
        for (auto& t : lens) t = int32_t(rng() % 200);
        kvx_desc d{};
        const int H = pick({1, 2, 4, 8, 64});
        d.num_layers = pick({1, 2, 3});
        d.num_kv_heads = H;
        d.head_dim = pick({16, 64, 128, 512});
        d.src_tp = pick({1, 2, 4, 8, 16, 64});
        d.dst_tp = pick({1, 2, 4, 8, 16});
        d.dst_rank = int32_t(rng() % d.dst_tp);
        d.src_dtype = pick({1, 2});
        d.dst_dtype = pick({1, 2, 3, 4});
        d.src_order = pick({0, 1, 2});
        d.block_size = pick({1, 5, 16, 64});
        d.num_blocks = 4096;
        d.num_requests = int32_t(lens.size());
        d.seq_lens = lens.data();
        d.src_block_size = pick({5, 16, 24});
        d.src_num_blocks = 4096;
        d.src_layers = d.num_layers + pick({0, 1});
        d.src_layer_offset = int32_t(rng() % (d.src_layers - d.num_layers + 1));
        d.cache_dtype = (d.dst_dtype >= 3) ? pick({0, 1, 2}) : 0;
        kvx_plan_t* p = nullptr;
        if (kvx_plan(&d, &p) != KVX_OK) { ++rejected; continue; }
        ++ok;
        kvx_plan_info info;
        kvx_plan_info_get(p, &info);
        kvx_plan_destroy(p);
    }
    int pd_ok = 0;
    for (int it = 0; it < 3000; ++it) {
        kvx_pd_problem pr{};
        pr.model = kvx_pd_model{pick({1, 2, 32, 80}), pick({64, 4096}), pick({1, 8, 32, 64}),
                                pick({1, 2, 8}), pick({64, 128}), pick({128, 14336}), pick({100, 32000}),
                                pick({1, 1, 4, 8}), pick({1, 2}), 0, 2.0, 2.0, 2.0};
        kvx_pd_gpu g{2.5e15, 8e12, 288e9, 1e12, 0.5, 0.8, 0.7, pick({0, 1, 8, 16}), 0};
        pr.prefill = g;
        pr.decode = g;
        pr.prompt_tokens = pick({0, 1, 4096});
        pr.output_tokens = pick({1, 512});
        pr.qps = 10.0;
        pr.ttft = 2.0;
        pr.tpot = 0.05;
        pr.max_batch = pick({0, 1, 256, 1 << 20});
        kvx_pd_solution s;
        if (kvx_pd_search(&pr, &s) == KVX_OK) ++pd_ok;
        kvx_pd_choice c;
        kvx_pd_evaluate(&pr, it % 3, 1 + it % 4, 1 + it % 8, 1, 1, 1 + it % 7, &c);
    }
    std::printf("plans ok %d rejected %d; pd searches ok %d\n", ok, rejected, pd_ok);
    return 0;
}
