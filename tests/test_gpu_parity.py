"""GPU parity: the HIP path (through the C ABI) against the oracle, byte for
byte (layout work and casts are exact, so the tolerance is 0 ULP).

Small cases compare every byte of the destination pool (or transfer tensor),
sentinels included.  Cast sweeps cover every fp16 pattern and every finite
bf16 value under many row scales.  Full-size workloads run in the launch
configuration the benchmark times and are checked on sampled requests and
planes (every request in the first and last plane), plus sampled unused
pages."""
import numpy as np
import pytest
import torch

from cases import (FULL, SMALL, e4m3_sweep_rows, inputs, oracle_problem, pad_rows,
                   read_shards, sweep_case, wire_size)
from gpu_util import (DEV, check_sampled, check_unused_pages, desc_for, dev_u16, gpu_run, log,
                      oracle_pool, pool)

import oracle as O
import paper_2509_17542_amd as K
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


# ---- small cases: whole pools ----------------------------------------------------

@pytest.mark.parametrize("name", list(SMALL))
def test_repack_small(name):
    w = SMALL[name]
    lens, bt, stride, shards = inputs(w)
    log(f"repack {name} lens={list(lens)}")
    cache, scales, _ = gpu_run("repack", w, lens, bt, stride, shards)
    want_c, want_s = oracle_pool(w, lens, bt, stride, shards)
    assert _eq(cache.cpu().numpy(), want_c)
    if want_s is not None:
        assert _eq(scales.cpu().numpy(), want_s)


@pytest.mark.parametrize("name", list(SMALL))
def test_pack_small(name):
    w = SMALL[name]
    lens, bt, stride, shards = inputs(w)
    log(f"pack {name}")
    _, _, wire = gpu_run("pack", w, lens, bt, stride, shards)
    want = O.pack(oracle_problem(O, w, lens), shards)
    got = wire.cpu().numpy()[:want.size]
    assert _eq(got, want)


@pytest.mark.parametrize("name", list(SMALL))
def test_unpack_small(name):
    """Unpack alone, fed the oracle's transfer tensor."""
    w = SMALL[name]
    lens, bt, stride, shards = inputs(w)
    wire = O.pack(oracle_problem(O, w, lens), shards)
    log(f"unpack {name}")
    cache, scales, _ = gpu_run("unpack", w, lens, bt, stride, None, wire_in=wire)
    want_c, want_s = oracle_pool(w, lens, bt, stride, shards, op="unpack", wire=wire)
    assert _eq(cache.cpu().numpy(), want_c)
    if want_s is not None:
        assert _eq(scales.cpu().numpy(), want_s)


@pytest.mark.parametrize("name", ["tiny", "llama3_70b_small_r1", "qwen_htd_small", "fp8_small",
                                  "fp16_e4m3_htd_empty"])
def test_pack_then_unpack_equals_repack(name):
    w = SMALL[name]
    lens, bt, stride, shards = inputs(w)
    log(f"pack+unpack {name}")
    c1, s1, _ = gpu_run("pack_unpack", w, lens, bt, stride, shards)
    c2, s2, _ = gpu_run("repack", w, lens, bt, stride, shards)
    assert torch.equal(c1, c2)
    if s1 is not None:
        assert torch.equal(s1.view(torch.int32), s2.view(torch.int32))


def test_page_ids_outside_the_pool_are_skipped():
    """A block-table entry outside [0, num_blocks) is not a page: nothing is
    written for it (the kernel's own bounds check), the other pages are."""
    w = SMALL["llama3_8b_small"]
    lens, bt, stride, shards = inputs(w)
    bad = bt.copy()
    bad[0, 1] = -1
    bad[1, 0] = w.num_blocks + 5
    log("repack with out-of-pool page ids")
    cache, _, _ = gpu_run("repack", w, lens, bad, stride, shards)
    want, _ = oracle_pool(w, lens, bt, stride, shards)
    page = w.block_size * w.hd * w.head_dim * 2
    want = want.reshape(w.layers, 2, w.num_blocks, page)
    want[:, :, bt[0, 1]] = W.SENTINEL
    want[:, :, bt[1, 0]] = W.SENTINEL
    assert _eq(cache.cpu().numpy(), want.reshape(-1))


def test_empty_batch_is_a_no_op():
    w = SMALL["llama3_8b_small"].replace(lens_override=(0, 0), num_requests=2)
    lens, bt, stride, shards = inputs(w)
    cache, _, _ = gpu_run("repack", w, lens, bt, stride, shards)
    assert bool((cache == W.SENTINEL).all())


# ---- cast sweeps --------------------------------------------------------------------

def test_fp16_to_bf16_every_pattern():
    rows = np.arange(65536, dtype=np.uint32).astype(np.uint16).reshape(512, 128)
    w, lens, bt, shards = sweep_case("fp16", "bf16", rows)
    log("fp16->bf16 all 65536 patterns")
    cache, _, _ = gpu_run("repack", w, lens, bt, bt.shape[1], shards)
    want, _ = oracle_pool(w, lens, bt, bt.shape[1], shards)
    assert _eq(cache.cpu().numpy(), want)


def test_bf16_to_fp16_every_pattern():
    rows = np.arange(65536, dtype=np.uint32).astype(np.uint16).reshape(512, 128)
    w, lens, bt, shards = sweep_case("bf16", "fp16", rows)
    log("bf16->fp16 all 65536 patterns")
    cache, _, _ = gpu_run("repack", w, lens, bt, bt.shape[1], shards)
    want, _ = oracle_pool(w, lens, bt, bt.shape[1], shards)
    assert _eq(cache.cpu().numpy(), want)


@pytest.mark.parametrize("fmt", ["bf16", "fp16"])
def test_e4m3_sweep(fmt):
    rng = np.random.default_rng(2024)
    if fmt == "bf16":
        # row maxima over the whole bf16 range: subnormal, tiny, around 448,
        # around the fast-path limits 2^-80 * 448 and 2^100 * 448, the largest
        amaxes = sorted(set([0x0001, 0x0040, 0x0080, 0x00FF, 0x0100, 0x0F00, 0x1000, 0x1080,
                             0x3F80, 0x3F81, 0x43E0, 0x43DF, 0x43E1, 0x4000, 0x7F7F, 0x7F00,
                             0x7200, 0x71FF, 0x7201, 0x2000, 0x1F00, 0x1F80])
                        | set(rng.integers(1, 0x7F80, 40).tolist()))
    else:
        amaxes = sorted(set([0x0001, 0x0200, 0x03FF, 0x0400, 0x3C00, 0x5F00, 0x5EFF, 0x7BFF,
                             0x1000, 0x2000]) | set(rng.integers(1, 0x7C00, 24).tolist()))
    rows = pad_rows(e4m3_sweep_rows(fmt, amaxes, rng))
    w, lens, bt, shards = sweep_case(fmt, "e4m3fn", rows)
    log(f"{fmt}->e4m3fn sweep: {rows.shape[0]} rows, {len(amaxes)} row maxima")
    cache, scales, _ = gpu_run("repack", w, lens, bt, bt.shape[1], shards)
    want_c, want_s = oracle_pool(w, lens, bt, bt.shape[1], shards)
    got_c = cache.cpu().numpy()
    bad = np.nonzero(got_c != want_c)[0]
    assert bad.size == 0, f"{bad.size} bytes differ, first at {bad[:8]}"
    assert _eq(scales.cpu().numpy(), want_s)


# ---- full-size workloads (the benchmark's launch configuration) ------------------

def _full_case(name, layer0=0, nlayers=None, extra_planes=2, n_req=4):
    w = FULL[name]
    nlayers = nlayers or w.layers
    rng = np.random.default_rng(7)
    log(f"full {name}: generating layers {layer0}..{layer0 + nlayers - 1}")
    lens = W.seq_lens(w)
    bt, stride = W.block_table(w, lens)
    shards = W.source_shards(w, lens, layer0, nlayers, read_shards(w))
    log(f"full {name}: repack on GPU ({int(lens.sum())} tokens)")
    cache, scales, _ = gpu_run("repack", w, lens, bt, stride, shards, nlayers)
    # every request in the first and the last plane; a few requests in random planes
    edge = [(0, 0), (nlayers - 1, 1)]
    n1 = check_sampled(w, lens, bt, shards, cache, scales, nlayers, edge, range(len(lens)), rng)
    picks = rng.choice(len(lens), min(n_req, len(lens)), replace=False)
    planes = [(int(rng.integers(nlayers)), int(rng.integers(2))) for _ in range(extra_planes)]
    n2 = check_sampled(w, lens, bt, shards, cache, scales, nlayers, planes, picks, rng)
    check_unused_pages(w, lens, bt, cache, nlayers, rng)
    log(f"full {name}: {n1 + n2} rows checked")


def test_full_llama3_8b():
    _full_case("llama3_8b_bf16_bs16")


def test_full_llama3_70b_shard():
    _full_case("llama3_70b_tp4to2_bf16_bs32")


def test_full_qwen7b_htd():
    _full_case("qwen7b_htd_fp16_bf16_bs64")


def test_full_tiny():
    _full_case("tiny_tp1to2_fp16_bf16")


def test_full_qwen7b_gqa_replicated_tp8():
    _full_case("qwen7b_gqa_tp1to8_r5_fp16_bf16_bs64")


def test_full_llama3_8b_bf16_to_fp16():
    _full_case("llama3_8b_bf16_fp16_bs16")


@pytest.mark.parametrize("group", [0, 15])
def test_full_fp8_decode_layer_group(group):
    w = FULL["fp8_decode_61l_bf16_e4m3_bs16"]
    l0, nl = w.group_layers(group)
    _full_case(w.name, l0, nl, extra_planes=1, n_req=3)


@pytest.mark.parametrize("name", ["llama3_8b_bf16_bs16", "llama3_70b_tp4to2_bf16_bs32",
                                  "qwen7b_htd_fp16_bf16_bs64", "fp8_decode_61l_bf16_e4m3_bs16"])
def test_full_pack_then_unpack(name):
    """The benchmark's pack and unpack at full size: the transfer tensor on
    sampled (request, plane) segments against the oracle's rows (every request
    in the first and last plane), then the unpack of that same device
    transfer tensor on sampled pages, plus sampled unused pages."""
    w = FULL[name]   # the fp8 decode workload: its first 4-layer group
    rng = np.random.default_rng(11)
    lens = W.seq_lens(w)
    bt, stride = W.block_table(w, lens)
    log(f"full {name}: generating inputs")
    shards = W.source_shards(w, lens, 0, w.layers, read_shards(w))
    plan = K.kvx_plan(desc_for(w, lens))
    info = K.kvx_plan_info_get(plan)
    dsh = [dev_u16(s) for s in shards]
    wire = torch.full((int(info.wire_bytes),), W.SENTINEL, dtype=torch.uint8, device=DEV)
    log(f"full {name}: pack on GPU")
    K.kvx_pack(plan, dsh, wire)
    torch.cuda.synchronize()
    p = oracle_problem(O, w, lens)
    doff, soff, _ = O.wire_layout(p)
    row = w.head_dim * wire_size(w)
    samples = [(r, 0, 0) for r in range(len(lens))] + \
              [(r, w.layers - 1, 1) for r in range(len(lens))] + \
              [(int(rng.integers(len(lens))), int(rng.integers(w.layers)), int(rng.integers(2)))
               for _ in range(4)]
    for r, l, kv in samples:
        T = int(lens[r])
        want, want_s = O.expected_rows(p, shards, r, l, kv, 0, T)
        off = int(doff[r]) + (l * 2 + kv) * T * w.hd * row
        got = wire[off:off + T * w.hd * row].cpu().numpy()
        assert np.array_equal(got, want.reshape(-1)), (name, r, l, kv)
        if want_s is not None:
            so = int(soff[r]) + (l * 2 + kv) * T * w.hd * 4
            gs = wire[so:so + T * w.hd * 4].cpu().numpy()
            assert np.array_equal(gs.view(np.uint32), want_s.view(np.uint32)), (name, r, l, kv)
    log(f"full {name}: unpack on GPU")
    del dsh
    cache, scales = pool(w, w.layers)
    K.kvx_unpack(plan, wire, cache, scales, torch.from_numpy(bt).to(DEV), stride)
    torch.cuda.synchronize()
    edge = [(0, 0), (w.layers - 1, 1)]
    n = check_sampled(w, lens, bt, shards, cache, scales, w.layers, edge, range(len(lens)), rng)
    check_unused_pages(w, lens, bt, cache, w.layers, rng)
    log(f"full {name}: {len(samples)} transfer-tensor segments, {n} cache rows checked")
