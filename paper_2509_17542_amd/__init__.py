"""Python binding of the kvx C ABI (include/kvx.h): argument marshalling only.

Every step of the conversion runs in the gfx950 kernels of libkvx.so; this
module converts Python arguments (ints, torch tensors) to the C types and
turns non-OK statuses into KvxError.  torch is imported first so that the
library binds to the HIP runtime torch already loaded; torch serves only for
device memory and streams.

Importing fails loudly (ImportError) when libkvx.so has not been built.
"""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (loads the process's HIP runtime before libkvx.so)

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libkvx.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"kvx HIP library not built: {LIB_PATH} is missing "
                      "(run `python -m paper_2509_17542_amd.build`)")

_lib = ctypes.CDLL(LIB_PATH)

# the struct layouts below are those of this version of include/kvx.h
ABI_VERSION = 9
if _lib.kvx_abi_version() != ABI_VERSION:
    raise ImportError(f"{LIB_PATH} implements kvx ABI {_lib.kvx_abi_version()}, this binding "
                      f"ABI {ABI_VERSION}: rebuild the library")

OK, EINVAL, EUNSUPPORTED, ENOMEM, EDEVICE = 0, -1, -2, -3, -4
FP16, BF16, E4M3FN, E5M2 = 1, 2, 3, 4
THD, HTD, PAGED = 0, 1, 2
_STATUS = {0: "KVX_OK", -1: "KVX_EINVAL", -2: "KVX_EUNSUPPORTED", -3: "KVX_ENOMEM",
           -4: "KVX_EDEVICE"}


class KvxError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


class kvx_desc(ctypes.Structure):
    _fields_ = [
        ("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("src_tp", ctypes.c_int32), ("dst_tp", ctypes.c_int32),
        ("dst_rank", ctypes.c_int32), ("src_dtype", ctypes.c_int32),
        ("dst_dtype", ctypes.c_int32), ("src_order", ctypes.c_int32),
        ("block_size", ctypes.c_int32), ("num_blocks", ctypes.c_int64),
        ("num_requests", ctypes.c_int32), ("seq_lens", ctypes.POINTER(ctypes.c_int32)),
        ("src_block_size", ctypes.c_int32), ("src_num_blocks", ctypes.c_int64),
        ("src_layer_offset", ctypes.c_int32), ("src_layers", ctypes.c_int32),
        ("dst_layer_offset", ctypes.c_int32), ("dst_layers", ctypes.c_int32),
        ("cache_dtype", ctypes.c_int32),
    ]


class kvx_plan_info(ctypes.Structure):
    _fields_ = [
        ("wire_bytes", ctypes.c_uint64), ("total_tokens", ctypes.c_int64),
        ("read_bytes_pack", ctypes.c_int64), ("write_bytes_pack", ctypes.c_int64),
        ("read_bytes_unpack", ctypes.c_int64), ("write_bytes_unpack", ctypes.c_int64),
        ("read_bytes_repack", ctypes.c_int64), ("write_bytes_repack", ctypes.c_int64),
        ("max_blocks_per_request", ctypes.c_int32), ("num_items", ctypes.c_int32),
        ("device", ctypes.c_int32), ("max_src_blocks_per_request", ctypes.c_int32),
    ]


class kvx_buffer_sizes(ctypes.Structure):
    _fields_ = [
        ("wire_bytes", ctypes.c_uint64), ("cache_bytes", ctypes.c_uint64),
        ("scale_bytes", ctypes.c_uint64), ("num_requests", ctypes.c_int32),
        ("src_tp", ctypes.c_int32),
    ]


class kvx_pipe_info(ctypes.Structure):
    _fields_ = [
        ("chunk_layers", ctypes.c_int32), ("num_chunks", ctypes.c_int32),
        ("slots", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("slot_bytes", ctypes.c_uint64), ("host_bytes", ctypes.c_uint64),
        ("device_bytes", ctypes.c_uint64), ("bus_bytes", ctypes.c_uint64),
    ]


class kvx_pd_model(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("layers", "hidden", "q_heads", "kv_heads",
                                              "head_dim", "ffn_dim", "vocab", "experts",
                                              "active_experts", "reserved")] + \
               [(n, ctypes.c_double) for n in ("weight_bytes", "kv_bytes", "act_bytes")]


class kvx_pd_gpu(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in ("flops", "hbm_bytes", "vram", "link_bytes",
                                               "lam", "alpha", "beta")] + \
               [("max_gpus", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class kvx_pd_problem(ctypes.Structure):
    _fields_ = [("model", kvx_pd_model), ("prefill", kvx_pd_gpu), ("decode", kvx_pd_gpu),
                ("prompt_tokens", ctypes.c_int32), ("output_tokens", ctypes.c_int32),
                ("qps", ctypes.c_double), ("ttft", ctypes.c_double), ("tpot", ctypes.c_double),
                ("max_batch", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class kvx_pd_choice(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("dp", "tp", "pp", "ep", "batch", "gpus")] + \
               [(n, ctypes.c_double) for n in ("latency", "vram", "throughput", "objective")]


class kvx_pd_solution(ctypes.Structure):
    _fields_ = [("prefill", kvx_pd_choice), ("decode", kvx_pd_choice)] + \
               [(n, ctypes.c_int64) for n in ("prefill_instances", "decode_instances",
                                              "candidates_prefill", "candidates_decode",
                                              "feasible_prefill", "feasible_decode")]


PD_PREFILL, PD_DECODE = 0, 1

_vp = ctypes.c_void_p
_i32 = ctypes.c_int32
_lib.kvx_plan.restype = ctypes.c_int
_lib.kvx_plan.argtypes = [ctypes.POINTER(kvx_desc), ctypes.POINTER(_vp)]
_lib.kvx_plan_info_get.restype = ctypes.c_int
_lib.kvx_plan_info_get.argtypes = [_vp, ctypes.POINTER(kvx_plan_info)]
_lib.kvx_plan_segment.restype = ctypes.c_int
_lib.kvx_plan_segment.argtypes = [_vp, _i32, ctypes.POINTER(ctypes.c_int64),
                                  ctypes.POINTER(ctypes.c_int64)]
_lib.kvx_plan_buffer_sizes.restype = ctypes.c_int
_lib.kvx_plan_buffer_sizes.argtypes = [_vp, ctypes.POINTER(kvx_buffer_sizes)]
_lib.kvx_plan_shard_bytes.restype = ctypes.c_int
_lib.kvx_plan_shard_bytes.argtypes = [_vp, _i32, ctypes.POINTER(ctypes.c_uint64)]
_lib.kvx_plan_destroy.restype = ctypes.c_int
_lib.kvx_plan_destroy.argtypes = [_vp]
_lib.kvx_pack.restype = ctypes.c_int
_lib.kvx_pack.argtypes = [_vp, _vp, _vp, _vp]
_lib.kvx_unpack.restype = ctypes.c_int
_lib.kvx_unpack.argtypes = [_vp, _vp, _vp, _vp, _vp, _i32, _vp]
_lib.kvx_repack.restype = ctypes.c_int
_lib.kvx_repack.argtypes = [_vp, _vp, _vp, _vp, _vp, _i32, _vp]
_lib.kvx_pack_paged.restype = ctypes.c_int
_lib.kvx_pack_paged.argtypes = [_vp, _vp, _vp, _i32, _vp, _vp]
_lib.kvx_repack_paged.restype = ctypes.c_int
_lib.kvx_repack_paged.argtypes = [_vp, _vp, _vp, _i32, _vp, _vp, _vp, _i32, _vp]
_lib.kvx_repack_noalloc.restype = ctypes.c_int
_lib.kvx_repack_noalloc.argtypes = [ctypes.POINTER(kvx_desc), _vp, _vp, _vp, _vp, _i32, _vp]
_lib.kvx_check_block_table.restype = ctypes.c_int
_lib.kvx_check_block_table.argtypes = [_vp, _vp, _i32]
_lib.kvx_check_src_block_table.restype = ctypes.c_int
_lib.kvx_check_src_block_table.argtypes = [_vp, _vp, _i32]
_lib.kvx_pipe_create.restype = ctypes.c_int
_lib.kvx_pipe_create.argtypes = [_vp, _i32, _i32, ctypes.POINTER(_vp)]
_lib.kvx_pipe_info_get.restype = ctypes.c_int
_lib.kvx_pipe_info_get.argtypes = [_vp, ctypes.POINTER(kvx_pipe_info)]
_lib.kvx_pipe_run.restype = ctypes.c_int
_lib.kvx_pipe_run.argtypes = [_vp, _vp, _vp, _i32, _vp, _vp, _vp, _i32, _vp]
_lib.kvx_pipe_destroy.restype = ctypes.c_int
_lib.kvx_pipe_destroy.argtypes = [_vp]
_lib.kvx_last_error.restype = ctypes.c_char_p
_lib.kvx_last_error.argtypes = []
_lib.kvx_abi_version.restype = ctypes.c_int32
_lib.kvx_abi_version.argtypes = []
_lib.kvx_pd_search.restype = ctypes.c_int
_lib.kvx_pd_search.argtypes = [ctypes.POINTER(kvx_pd_problem), ctypes.POINTER(kvx_pd_solution)]
_lib.kvx_pd_evaluate.restype = ctypes.c_int
_lib.kvx_pd_evaluate.argtypes = [ctypes.POINTER(kvx_pd_problem)] + [_i32] * 6 + \
    [ctypes.POINTER(kvx_pd_choice)]

EXPORTS = ("kvx_plan", "kvx_plan_info_get", "kvx_plan_segment", "kvx_plan_buffer_sizes",
           "kvx_plan_shard_bytes", "kvx_plan_destroy", "kvx_pack",
           "kvx_unpack", "kvx_repack", "kvx_pack_paged", "kvx_repack_paged", "kvx_repack_noalloc",
           "kvx_check_block_table", "kvx_check_src_block_table", "kvx_pipe_create",
           "kvx_pipe_info_get", "kvx_pipe_run", "kvx_pipe_destroy", "kvx_last_error",
           "kvx_abi_version", "kvx_pd_search", "kvx_pd_evaluate")


def _check(status: int) -> None:
    if status != OK:
        raise KvxError(status, kvx_last_error())


def _addr(x) -> int | None:
    """Device (or host) address of a tensor, an int, or None."""
    if x is None:
        return None
    if isinstance(x, torch.Tensor):
        return x.data_ptr()
    return int(x)


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


class Plan:
    """Owns a kvx_plan_t*; destroyed with kvx_plan_destroy.  Holds the sizes
    its launches touch (kvx_plan_buffer_sizes, kvx_plan_shard_bytes) for the
    checks of tensor arguments."""

    _destroy = _lib.kvx_plan_destroy  # kept reachable during interpreter shutdown

    def __init__(self, handle: int):
        self.handle = handle
        self.sizes = kvx_buffer_sizes()
        _check(_lib.kvx_plan_buffer_sizes(self, ctypes.byref(self.sizes)))
        self.shard_bytes = []
        b = ctypes.c_uint64()
        for j in range(self.sizes.src_tp):
            _check(_lib.kvx_plan_shard_bytes(self, j, ctypes.byref(b)))
            self.shard_bytes.append(b.value)
        info = kvx_plan_info()
        _check(_lib.kvx_plan_info_get(self, ctypes.byref(info)))
        self.touches = info.num_items > 0   # launches read or write anything

    def __del__(self):
        h, self.handle = getattr(self, "handle", None), None
        if h:
            self._destroy(h)

    @property
    def _as_parameter_(self):
        return ctypes.c_void_p(self.handle)


class Pipe:
    """Owns a kvx_pipe_t*; destroyed with kvx_pipe_destroy.  Keeps its plan
    alive."""

    _destroy = _lib.kvx_pipe_destroy

    def __init__(self, handle: int, plan: "Plan"):
        self.handle = handle
        self.plan = plan

    def __del__(self):
        h, self.handle = getattr(self, "handle", None), None
        if h:
            self._destroy(h)

    @property
    def _as_parameter_(self):
        return ctypes.c_void_p(self.handle)


def make_desc(num_layers, num_kv_heads, head_dim, src_tp, dst_tp, dst_rank, src_dtype, dst_dtype,
              src_order, block_size, num_blocks, seq_lens, src_block_size=0, src_num_blocks=0,
              src_layer_offset=0, src_layers=0, dst_layer_offset=0, dst_layers=0,
              cache_dtype=0):
    """kvx_desc plus the int32 array its seq_lens points into (src_block_size
    and src_num_blocks matter only for a PAGED source; the layer fields
    describe pipeline stages, 0 = the converted layers; cache_dtype 0 = the
    cache holds dst_dtype, FP16 / BF16 with an E4M3FN dst_dtype = the
    dequantising unpack)."""
    lens = (ctypes.c_int32 * max(len(seq_lens), 1))(*[int(t) for t in seq_lens])
    d = kvx_desc(num_layers, num_kv_heads, head_dim, src_tp, dst_tp, dst_rank, src_dtype,
                 dst_dtype, src_order, block_size, num_blocks, len(seq_lens),
                 ctypes.cast(lens, ctypes.POINTER(ctypes.c_int32)), src_block_size,
                 src_num_blocks, src_layer_offset, src_layers, dst_layer_offset, dst_layers,
                 cache_dtype)
    d._lens = lens
    return d


def kvx_plan(desc: kvx_desc) -> Plan:
    h = _vp()
    _check(_lib.kvx_plan(ctypes.byref(desc), ctypes.byref(h)))
    return Plan(h.value)


def kvx_plan_info_get(plan: Plan) -> kvx_plan_info:
    info = kvx_plan_info()
    _check(_lib.kvx_plan_info_get(plan, ctypes.byref(info)))
    return info


def kvx_plan_segment(plan: Plan, r: int) -> tuple[int, int]:
    d, s = ctypes.c_int64(), ctypes.c_int64()
    _check(_lib.kvx_plan_segment(plan, r, ctypes.byref(d), ctypes.byref(s)))
    return d.value, s.value


def kvx_plan_buffer_sizes(plan: Plan) -> kvx_buffer_sizes:
    out = kvx_buffer_sizes()
    _check(_lib.kvx_plan_buffer_sizes(plan, ctypes.byref(out)))
    return out


def kvx_plan_shard_bytes(plan: Plan, j: int) -> int:
    b = ctypes.c_uint64()
    _check(_lib.kvx_plan_shard_bytes(plan, j, ctypes.byref(b)))
    return b.value


def kvx_plan_destroy(plan: Plan) -> None:
    h, plan.handle = plan.handle, None
    _check(_lib.kvx_plan_destroy(h))


def _need(x, nbytes: int, what: str, dtype=None) -> None:
    """A torch tensor argument must be a contiguous device tensor (of `dtype`
    where given) holding at least the `nbytes` the plan's launches touch
    through it.  Bare addresses (ints) and None pass unchecked: the C calls
    check NULL and alignment, sizes are the caller's contract there."""
    if not isinstance(x, torch.Tensor) or nbytes <= 0:
        return
    if x.device.type != "cuda":
        raise ValueError(f"{what} must be a device tensor, not one on {x.device}")
    if not x.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if dtype is not None and x.dtype != dtype:
        raise ValueError(f"{what} must be {dtype}, not {x.dtype}")
    have = x.numel() * x.element_size()
    if have < nbytes:
        raise ValueError(f"{what} holds {have} bytes; the plan touches {nbytes}")


def _shard_array(plan: Plan, shards):
    """The host array of src_tp shard addresses, each read shard checked."""
    shards = list(shards)
    if len(shards) < plan.sizes.src_tp:
        raise ValueError(f"{len(shards)} source shards given; the plan has src_tp = "
                         f"{plan.sizes.src_tp}")
    arr = (_vp * max(len(shards), 1))()
    for j, s in enumerate(shards):
        if j < plan.sizes.src_tp:
            _need(s, plan.shard_bytes[j], f"src_shards[{j}]")
        arr[j] = _addr(s)
    return arr


def _table_bytes(plan: Plan, stride: int) -> int:
    """int32 bytes of a [num_requests][stride] block table, if launches read it."""
    return 4 * plan.sizes.num_requests * max(int(stride), 0) if plan.touches else 0


def _need_pool(plan: Plan, cache, scales, block_table, bt_stride: int) -> None:
    if not plan.touches:
        return
    _need(cache, plan.sizes.cache_bytes, "cache")
    _need(scales, plan.sizes.scale_bytes, "scales", torch.float32)
    _need(block_table, _table_bytes(plan, bt_stride), "block_table", torch.int32)


def kvx_pack(plan: Plan, src_shards, wire, stream=None) -> None:
    if plan.touches:
        _need(wire, plan.sizes.wire_bytes, "wire")
    _check(_lib.kvx_pack(plan, _shard_array(plan, src_shards), _addr(wire), _stream(stream)))


def kvx_unpack(plan: Plan, wire, cache, scales, block_table, bt_stride: int, stream=None) -> None:
    if plan.touches:
        _need(wire, plan.sizes.wire_bytes, "wire")
    _need_pool(plan, cache, scales, block_table, bt_stride)
    _check(_lib.kvx_unpack(plan, _addr(wire), _addr(cache), _addr(scales), _addr(block_table),
                           bt_stride, _stream(stream)))


def kvx_repack(plan: Plan, src_shards, cache, scales, block_table, bt_stride: int,
               stream=None) -> None:
    _need_pool(plan, cache, scales, block_table, bt_stride)
    _check(_lib.kvx_repack(plan, _shard_array(plan, src_shards), _addr(cache), _addr(scales),
                           _addr(block_table), bt_stride, _stream(stream)))


def kvx_repack_noalloc(desc: kvx_desc, src_shards, cache, scales, block_table, bt_stride: int,
                       stream=None) -> None:
    """kvx_repack of `desc` with no plan and no allocation (the C call keeps
    its work-item table in a static device array).  Tensor arguments are
    checked against the sizes the descriptor implies: every shard given must
    hold one shard's bytes, whether the decode rank reads it or not."""
    lens = [desc.seq_lens[r] for r in range(desc.num_requests)]
    if sum(lens) > 0:
        H, D = desc.num_kv_heads, desc.head_dim
        hs = H // desc.src_tp if 0 < desc.src_tp <= H else 1
        hd = H // desc.dst_tp if 0 < desc.dst_tp <= H else 1
        cdt = desc.cache_dtype or desc.dst_dtype
        esz = 1 if cdt in (E4M3FN, E5M2) else 2
        src_layers = desc.src_layers or desc.num_layers
        dst_layers = desc.dst_layers or desc.num_layers
        slots = 2 * dst_layers * desc.num_blocks * desc.block_size * hd
        _need(cache, slots * D * esz, "cache")
        _need(scales, slots * 4 if esz == 1 else 0, "scales", torch.float32)
        _need(block_table, 4 * desc.num_requests * max(int(bt_stride), 0), "block_table",
              torch.int32)
        for j, sh in enumerate(src_shards):
            _need(sh, 2 * src_layers * sum(lens) * hs * D * 2, f"src_shards[{j}]")
    arr = (_vp * max(len(src_shards), 1))()
    for j, sh in enumerate(src_shards):
        arr[j] = _addr(sh)
    _check(_lib.kvx_repack_noalloc(ctypes.byref(desc), arr, _addr(cache), _addr(scales),
                                   _addr(block_table), bt_stride, _stream(stream)))


def kvx_pack_paged(plan: Plan, src_shards, src_block_table, src_bt_stride: int, wire,
                   stream=None) -> None:
    if plan.touches:
        _need(wire, plan.sizes.wire_bytes, "wire")
    _need(src_block_table, _table_bytes(plan, src_bt_stride), "src_block_table", torch.int32)
    _check(_lib.kvx_pack_paged(plan, _shard_array(plan, src_shards), _addr(src_block_table),
                               src_bt_stride, _addr(wire), _stream(stream)))


def kvx_repack_paged(plan: Plan, src_shards, src_block_table, src_bt_stride: int, cache, scales,
                     block_table, bt_stride: int, stream=None) -> None:
    _need_pool(plan, cache, scales, block_table, bt_stride)
    _need(src_block_table, _table_bytes(plan, src_bt_stride), "src_block_table", torch.int32)
    _check(_lib.kvx_repack_paged(plan, _shard_array(plan, src_shards), _addr(src_block_table),
                                 src_bt_stride, _addr(cache), _addr(scales), _addr(block_table),
                                 bt_stride, _stream(stream)))


def _host_table(table):
    """(keep-alive object, address) of a contiguous int32 host table."""
    if isinstance(table, torch.Tensor):
        if table.device.type != "cpu" or table.dtype != torch.int32:
            raise ValueError("a host block table must be an int32 CPU tensor or array")
        keep = table.contiguous()
        return keep, keep.data_ptr()
    import numpy as np
    keep = np.ascontiguousarray(table, dtype=np.int32)
    return keep, keep.ctypes.data


def kvx_check_block_table(plan: Plan, host_block_table, bt_stride: int) -> None:
    """host_block_table: a contiguous int32 numpy array or CPU tensor."""
    keep, ptr = _host_table(host_block_table)
    _check(_lib.kvx_check_block_table(plan, ptr, bt_stride))
    del keep


def kvx_check_src_block_table(plan: Plan, host_src_block_table, src_bt_stride: int) -> None:
    """host_src_block_table: a contiguous int32 numpy array or CPU tensor."""
    keep, ptr = _host_table(host_src_block_table)
    _check(_lib.kvx_check_src_block_table(plan, ptr, src_bt_stride))
    del keep


def kvx_last_error() -> str:
    return _lib.kvx_last_error().decode()


def kvx_abi_version() -> int:
    return int(_lib.kvx_abi_version())


def kvx_pipe_create(plan: Plan, chunk_layers: int, slots: int) -> Pipe:
    h = _vp()
    _check(_lib.kvx_pipe_create(plan, chunk_layers, slots, ctypes.byref(h)))
    return Pipe(h.value, plan)


def kvx_pipe_info_get(pipe: Pipe) -> kvx_pipe_info:
    info = kvx_pipe_info()
    _check(_lib.kvx_pipe_info_get(pipe, ctypes.byref(info)))
    return info


def kvx_pipe_run(pipe: Pipe, src_shards, src_block_table, src_bt_stride: int, cache, scales,
                 block_table, bt_stride: int, stream=None) -> None:
    _need_pool(pipe.plan, cache, scales, block_table, bt_stride)
    _need(src_block_table, _table_bytes(pipe.plan, src_bt_stride), "src_block_table", torch.int32)
    _check(_lib.kvx_pipe_run(pipe, _shard_array(pipe.plan, src_shards), _addr(src_block_table),
                             src_bt_stride, _addr(cache), _addr(scales), _addr(block_table),
                             bt_stride, _stream(stream)))


def kvx_pipe_destroy(pipe: Pipe) -> None:
    h, pipe.handle = pipe.handle, None
    _check(_lib.kvx_pipe_destroy(h))


def kvx_pd_search(problem: kvx_pd_problem) -> kvx_pd_solution:
    out = kvx_pd_solution()
    _check(_lib.kvx_pd_search(ctypes.byref(problem), ctypes.byref(out)))
    return out


def kvx_pd_evaluate(problem: kvx_pd_problem, side: int, dp: int, tp: int, pp: int, ep: int,
                    batch: int) -> kvx_pd_choice:
    out = kvx_pd_choice()
    _check(_lib.kvx_pd_evaluate(ctypes.byref(problem), side, dp, tp, pp, ep, batch,
                                ctypes.byref(out)))
    return out
