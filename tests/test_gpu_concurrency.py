"""One plan used at once from several host threads, each on its own stream (a
plan is immutable and may serve any number of streams of its device): every
thread repacks its own sources into its own pool, five times, while the
others do the same; each pool is then compared with the oracle, byte for
byte.  ctypes releases the interpreter lock during the C call, so the
threads are inside the library at the same time."""
from __future__ import annotations

import threading

import numpy as np
import pytest
import torch

from cases import SMALL, inputs
from gpu_util import DEV, check_shapes, desc_for, dev_u16, log, oracle_pool, pool

import paper_2509_17542_amd as K

pytestmark = pytest.mark.gpu

THREADS = 4
LAUNCHES = 5


@pytest.mark.parametrize("name", ["llama3_70b_small_r1", "fp8_small", "qwen_htd_small"])
def test_one_plan_from_several_threads_and_streams(name):
    w = SMALL[name]
    lens, bt, stride, shards = inputs(w)
    plan = K.kvx_plan(desc_for(w, lens))
    # each thread's sources: the workload's values rotated by its own offset
    variants = [[None if s is None else np.roll(s, 101 * k) for s in shards]
                for k in range(THREADS)]
    dsh = [[dev_u16(s) for s in v] for v in variants]
    for d in dsh:
        check_shapes(w, lens, bt, stride, d, w.layers)
    bt_d = torch.from_numpy(np.ascontiguousarray(bt, dtype=np.int32)).to(DEV)
    pools = [pool(w, w.layers) for _ in range(THREADS)]
    streams = [torch.cuda.Stream() for _ in range(THREADS)]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())  # the pools' fills come first
    start = threading.Barrier(THREADS)
    errors = []

    def work(k):
        try:
            start.wait()
            for _ in range(LAUNCHES):
                K.kvx_repack(plan, dsh[k], pools[k][0], pools[k][1], bt_d, stride, streams[k])
        except Exception as e:  # reported by the main thread
            errors.append((k, e))

    log(f"concurrency {name}: {THREADS} threads x {LAUNCHES} launches")
    threads = [threading.Thread(target=work, args=(k,)) for k in range(THREADS)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for k in range(THREADS):
        want_c, want_s = oracle_pool(w, lens, bt, stride, variants[k])
        cache, scales = pools[k]
        assert np.array_equal(cache.cpu().numpy(), want_c), f"thread {k}: cache"
        if want_s is not None:
            assert np.array_equal(scales.view(torch.uint8).cpu().numpy(), want_s.view(np.uint8)), \
                f"thread {k}: scales"
