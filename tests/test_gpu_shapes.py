"""GPU parity at the limits of the lane layout, whole pools against the
oracle, byte for byte: rows of 16 to 2048 bytes (one lane per row up to a
whole wave, chunk counts that are not powers of two, 8-bit row maxima
exchanged across 64 lanes), 1024 heads on a decode rank and 64 head
segments; repack, pack and unpack.  Also the largest launch a plan accepts
(2^24 - 8 work units, the largest grid the kernels use)."""
import numpy as np
import pytest
import torch

from cases import L8B, SMALL_SHAPES, inputs, oracle_problem
from gpu_util import gpu_run, log, oracle_pool

import oracle as O

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


@pytest.fixture(autouse=True)
def _release_device_memory():
    yield
    import gc
    gc.collect()
    torch.cuda.empty_cache()


def _eq(a, b):
    return np.array_equal(np.asarray(a).view(np.uint8), np.asarray(b).view(np.uint8))


@pytest.mark.parametrize("name", list(SMALL_SHAPES))
def test_shapes_repack(name):
    w = SMALL_SHAPES[name]
    lens, bt, stride, shards = inputs(w)
    log(f"shape repack {name}: D={w.head_dim}, H={w.heads}, TP {w.src_tp}->{w.dst_tp}")
    cache, scales, _ = gpu_run("repack", w, lens, bt, stride, shards)
    want_c, want_s = oracle_pool(w, lens, bt, stride, shards)
    assert _eq(cache.cpu().numpy(), want_c)
    if want_s is not None:
        assert _eq(scales.cpu().numpy(), want_s)


@pytest.mark.parametrize("name", list(SMALL_SHAPES))
def test_shapes_pack_and_unpack(name):
    w = SMALL_SHAPES[name]
    lens, bt, stride, shards = inputs(w)
    log(f"shape pack/unpack {name}")
    _, _, wire = gpu_run("pack", w, lens, bt, stride, shards)
    want = O.pack(oracle_problem(O, w, lens), shards)
    assert _eq(wire.cpu().numpy()[:want.size], want)
    cache, scales, _ = gpu_run("unpack", w, lens, bt, stride, None, wire_in=want)
    want_c, want_s = oracle_pool(w, lens, bt, stride, shards, op="unpack", wire=want)
    assert _eq(cache.cpu().numpy(), want_c)
    if want_s is not None:
        assert _eq(scales.cpu().numpy(), want_s)


# 2^24 - 8 work units: one-token pages of one 16-byte row (a single KV head of
# 8 bf16 elements), one unit per page in each of the two planes of one layer
UNIT_LIMIT_PAGES = (1 << 23) - 4
UNIT_LIMIT = L8B.replace(name="unit_limit", heads=1, head_dim=8, layers=1, total_layers=1,
                         block_size=1, num_blocks=UNIT_LIMIT_PAGES, num_requests=1,
                         lens_override=(UNIT_LIMIT_PAGES,))


def test_work_unit_limit_repack_pack_unpack():
    """The largest launch: 16,777,208 workgroups, every page of the pool
    written once in random order; whole pool and transfer tensor against the
    oracle."""
    w = UNIT_LIMIT
    lens, bt, stride, shards = inputs(w)
    log(f"unit limit: {int(lens.sum())} one-token pages, repack")
    cache, _, _ = gpu_run("repack", w, lens, bt, stride, shards)
    want_c, _ = oracle_pool(w, lens, bt, stride, shards)
    assert _eq(cache.cpu().numpy(), want_c)
    del cache
    log("unit limit: pack")
    _, _, wire = gpu_run("pack", w, lens, bt, stride, shards)
    want = O.pack(oracle_problem(O, w, lens), shards)
    assert _eq(wire.cpu().numpy()[:want.size], want)
    del wire
    log("unit limit: unpack")
    cache, _, _ = gpu_run("unpack", w, lens, bt, stride, None, wire_in=want)
    assert _eq(cache.cpu().numpy(), want_c)
