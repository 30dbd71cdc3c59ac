"""GPU parity of paged sources (the prefill side's own paged cache, with its
own page size and block table): kvx_pack_paged / kvx_repack_paged through the
C ABI against the oracle, byte for byte.

Small cases compare every byte of the destination pool or transfer tensor,
sentinels included; the full-size paged workloads run in the launch
configuration the benchmark times and are checked on sampled requests and
planes plus sampled unused pages."""
import numpy as np
import pytest
import torch

from cases import FULL, SMALL_PAGED, inputs, oracle_problem
from gpu_util import check_sampled, check_unused_pages, gpu_run, log, oracle_pool

import oracle as O
import workload as W

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


@pytest.mark.parametrize("name", list(SMALL_PAGED))
def test_repack_paged_small(name):
    w = SMALL_PAGED[name]
    lens, bt, stride, shards = inputs(w)
    log(f"repack_paged {name} lens={list(lens)}")
    cache, scales, _ = gpu_run("repack", w, lens, bt, stride, shards)
    want_c, want_s = oracle_pool(w, lens, bt, stride, shards)
    assert _eq(cache.cpu().numpy(), want_c)
    if want_s is not None:
        assert _eq(scales.cpu().numpy(), want_s)


@pytest.mark.parametrize("name", list(SMALL_PAGED))
def test_pack_paged_small(name):
    w = SMALL_PAGED[name]
    lens, bt, stride, shards = inputs(w)
    log(f"pack_paged {name}")
    _, _, wire = gpu_run("pack", w, lens, bt, stride, shards)
    want = O.pack(oracle_problem(O, w, lens), shards)
    assert _eq(wire.cpu().numpy()[:want.size], want)


@pytest.mark.parametrize("name", ["paged16_tp4to2_bs32_small", "paged16_e4m3_bs24"])
def test_pack_paged_then_unpack_equals_repack_paged(name):
    w = SMALL_PAGED[name]
    lens, bt, stride, shards = inputs(w)
    log(f"pack_paged+unpack {name}")
    c1, s1, _ = gpu_run("repack", w, lens, bt, stride, shards)
    c2, s2, _ = gpu_run("pack_unpack", w, lens, bt, stride, shards)
    assert torch.equal(c1, c2)
    if s1 is not None:
        assert torch.equal(s1.view(torch.int32), s2.view(torch.int32))


def test_source_pages_outside_the_pool_are_skipped():
    """Source page ids outside [0, src_num_blocks) give no row (the kernel's
    own bounds check): those decode slots keep the sentinel, as the oracle's."""
    w = SMALL_PAGED["paged24_bs16_r1"]
    lens, bt, stride, shards = inputs(w)
    sbt, _ = W.src_block_table(w, lens)
    bad = sbt.copy()
    bad[0, 1] = -1
    bad[2, 0] = w.src_num_blocks
    bad[1, 2] = 1 << 30
    log("repack_paged with out-of-pool source page ids")
    cache, _, _ = gpu_run("repack", w, lens, bt, stride, shards, sbt=bad)
    want, _ = oracle_pool(w, lens, bt, stride, shards, sbt=bad)
    assert _eq(cache.cpu().numpy(), want)
    assert int((cache == W.SENTINEL).sum()) > int((torch.from_numpy(
        oracle_pool(w, lens, bt, stride, shards)[0]) == W.SENTINEL).sum())


def test_shared_prefix_pages_are_read_twice():
    """Two requests whose first source pages are the same page (a shared
    prefix): both get that page's tokens."""
    w = SMALL_PAGED["paged16_bs64_small"]
    lens, bt, stride, shards = inputs(w)
    sbt, _ = W.src_block_table(w, lens)
    shared = sbt.copy()
    shared[1, 0] = shared[0, 0]
    log("repack_paged with a shared source page")
    cache, _, _ = gpu_run("repack", w, lens, bt, stride, shards, sbt=shared)
    want, _ = oracle_pool(w, lens, bt, stride, shards, sbt=shared)
    assert _eq(cache.cpu().numpy(), want)


def _full_paged_case(name, extra_planes=2, n_req=4):
    w = FULL[name]
    rng = np.random.default_rng(11)
    log(f"full {name}: generating the prefill-side pools")
    lens, bt, stride, shards = inputs(w)
    log(f"full {name}: repack_paged on GPU ({int(lens.sum())} tokens)")
    cache, scales, _ = gpu_run("repack", w, lens, bt, stride, shards)
    edge = [(0, 0), (w.layers - 1, 1)]
    n1 = check_sampled(w, lens, bt, shards, cache, scales, w.layers, edge, range(len(lens)), rng)
    picks = rng.choice(len(lens), min(n_req, len(lens)), replace=False)
    planes = [(int(rng.integers(w.layers)), int(rng.integers(2))) for _ in range(extra_planes)]
    n2 = check_sampled(w, lens, bt, shards, cache, scales, w.layers, planes, picks, rng)
    check_unused_pages(w, lens, bt, cache, w.layers, rng)
    log(f"full {name}: {n1 + n2} rows checked")


def test_full_llama3_8b_paged16_bs64():
    _full_paged_case("llama3_8b_paged16_bf16_bs64")


def test_full_llama3_70b_paged16_tp4to2_bs32():
    _full_paged_case("llama3_70b_paged16_tp4to2_bf16_bs32")
