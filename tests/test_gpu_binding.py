"""The binding refuses tensor arguments that do not hold what the plan's
launches touch (a kernel would otherwise read or write past them), before
anything is launched: a cache, wire, scale or shard one byte short, host
tensors, non-contiguous views and block tables that are not int32.  The
sizes come from kvx_plan_buffer_sizes / kvx_plan_shard_bytes."""
import numpy as np
import pytest
import torch

from cases import SMALL, SMALL_PAGED, inputs
from gpu_util import desc_for, dev_u16, log, pool

import paper_2509_17542_amd as K
import workload as W

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def _setup(w):
    lens, bt, stride, shards = inputs(w)
    plan = K.kvx_plan(desc_for(w, lens))
    dsh = [dev_u16(s) for s in shards]
    cache, scales = pool(w, w.layers)
    bt_d = torch.from_numpy(bt).cuda()
    return plan, dsh, cache, scales, bt_d, stride


@pytest.mark.parametrize("name", ["llama3_8b_small", "fp8_small"])
def test_short_or_wrong_tensors_are_refused(name):
    w = SMALL[name]
    log(f"binding checks {name}")
    plan, dsh, cache, scales, bt_d, stride = _setup(w)
    sz = K.kvx_plan_buffer_sizes(plan)
    assert cache.numel() == sz.cache_bytes
    with pytest.raises(ValueError, match="holds"):
        K.kvx_repack(plan, dsh, cache[:-1], scales, bt_d, stride)
    j = next(j for j in range(w.src_tp) if plan.shard_bytes[j])
    short = list(dsh)
    short[j] = dsh[j][:plan.shard_bytes[j] // 2 - 1]
    with pytest.raises(ValueError, match=f"src_shards\\[{j}\\]"):
        K.kvx_repack(plan, short, cache, scales, bt_d, stride)
    with pytest.raises(ValueError, match="device tensor"):
        K.kvx_repack(plan, [None if s is None else s.cpu() for s in dsh], cache, scales, bt_d,
                     stride)
    with pytest.raises(ValueError, match="int32"):
        K.kvx_repack(plan, dsh, cache, scales, bt_d.long(), stride)
    with pytest.raises(ValueError, match="holds"):
        K.kvx_repack(plan, dsh, cache, scales, bt_d[:-1], stride)
    with pytest.raises(ValueError, match="contiguous"):
        K.kvx_repack(plan, dsh, cache.view(2, -1)[:, ::2], scales, bt_d, stride)
    if scales is not None:
        with pytest.raises(ValueError, match="scales"):
            K.kvx_repack(plan, dsh, cache, scales[:-1], bt_d, stride)
    wire = torch.empty(int(sz.wire_bytes), dtype=torch.uint8, device="cuda")
    with pytest.raises(ValueError, match="wire"):
        K.kvx_pack(plan, dsh, wire[:-16])
    with pytest.raises(ValueError, match="wire"):
        K.kvx_unpack(plan, wire[:-16], cache, scales, bt_d, stride)
    # nothing was written by the refused calls
    assert bool((cache == W.SENTINEL).all())
    # the same arguments at their sizes go through
    K.kvx_repack(plan, dsh, cache, scales, bt_d, stride)
    torch.cuda.synchronize()
    assert not bool((cache == W.SENTINEL).all())


def test_paged_source_table_is_checked():
    w = SMALL_PAGED["paged16_bs64_small"]
    lens = W.seq_lens(w)
    plan, dsh, cache, scales, bt_d, stride = _setup(w)
    sbt, sstride = W.src_block_table(w, lens)
    sbt_d = torch.from_numpy(np.ascontiguousarray(sbt, dtype=np.int32)).cuda()
    assert plan.shard_bytes[0] == 2 * w.layers * 2 * w.src_num_blocks * w.src_block_size * \
        w.hs * w.head_dim
    with pytest.raises(ValueError, match="src_block_table"):
        K.kvx_repack_paged(plan, dsh, sbt_d[:-1], sstride, cache, scales, bt_d, stride)
    with pytest.raises(ValueError, match="src_block_table"):
        K.kvx_repack_paged(plan, dsh, sbt_d.long(), sstride, cache, scales, bt_d, stride)
    K.kvx_repack_paged(plan, dsh, sbt_d, sstride, cache, scales, bt_d, stride)
    torch.cuda.synchronize()
