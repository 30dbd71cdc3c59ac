"""GPU parity of every conversion in every source order (the cases of
cases.MATRIX): for each source type, transfer-tensor type and cache type the
library accepts, from token-major, head-major and paged sources, the pack,
the unpack (fed the oracle's transfer tensor) and the repack through the C
ABI against the oracle, byte for byte over the whole transfer tensor or pool,
sentinels included.  Every kernel instantiation of the library runs here."""
import numpy as np
import pytest
import torch

from cases import MATRIX, inputs, oracle_problem
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


@pytest.mark.parametrize("name", list(MATRIX))
def test_matrix_case(name):
    w = MATRIX[name]
    lens, bt, stride, shards = inputs(w)
    wire_want = O.pack(oracle_problem(O, w, lens), shards)
    log(f"matrix {name}: pack")
    _, _, wire = gpu_run("pack", w, lens, bt, stride, shards)
    assert _eq(wire.cpu().numpy()[:wire_want.size], wire_want)
    for op in ("unpack", "repack"):
        log(f"matrix {name}: {op}")
        if op == "unpack":
            cache, scales, _ = gpu_run("unpack", w, lens, bt, stride, None, wire_in=wire_want)
            want_c, want_s = oracle_pool(w, lens, bt, stride, shards, op="unpack", wire=wire_want)
        else:
            cache, scales, _ = gpu_run("repack", w, lens, bt, stride, shards)
            want_c, want_s = oracle_pool(w, lens, bt, stride, shards)
        assert _eq(cache.cpu().numpy(), want_c), op
        if want_s is not None:
            assert _eq(scales.cpu().numpy(), want_s), op
