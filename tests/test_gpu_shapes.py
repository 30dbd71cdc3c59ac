"""GPU parity at the limits of the lane layout, whole pools against the
oracle, byte for byte: rows of 16 to 2048 bytes (one lane per row up to a
whole wave, chunk counts that are not powers of two, 8-bit row maxima
exchanged across 64 lanes), 1024 heads on a decode rank and 64 head
segments; repack, pack and unpack."""
import numpy as np
import pytest
import torch

from cases import SMALL_SHAPES, inputs, oracle_problem
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
