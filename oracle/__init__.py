"""Plain CPU oracle of the KV-cache conversion (paper Sec. III-B).

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It wraps
``liboracle.so`` (built from ``kvx_oracle.c`` with gcc) through ctypes and
shares nothing with the GPU library: its own problem struct, its own index
maps, its own casts.

Arrays are numpy: 16-bit source elements as ``uint16`` bit patterns, the
destination as raw ``uint8`` bytes, scales as ``float32``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kvx_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

FP16, BF16, E4M3FN, E5M2 = 1, 2, 3, 4
TOKEN_MAJOR, HEAD_MAJOR, PAGED = 0, 1, 2
FMT_SIZE = {FP16: 2, BF16: 2, E4M3FN: 1, E5M2: 1}
FP8 = (E4M3FN, E5M2)

GCC_CMD = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-fPIC", "-shared",
           "-ffp-contract=off", "-fno-fast-math", "-o", _LIB_PATH, _SRC, "-lm"]


def build() -> str:
    """Compile liboracle.so next to its source."""
    subprocess.run(GCC_CMD, check=True)
    return _LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.POINTER
        vp = ctypes.c_void_p
        L.orc_decode.restype = ctypes.c_double
        L.orc_decode.argtypes = [ctypes.c_int, ctypes.c_uint32]
        L.orc_fp16_to_bf16.restype = ctypes.c_uint16
        L.orc_fp16_to_bf16.argtypes = [ctypes.c_uint16]
        L.orc_f32_to_e4m3fn.restype = ctypes.c_uint8
        L.orc_f32_to_e4m3fn.argtypes = [ctypes.c_float]
        L.orc_row_scale.restype = ctypes.c_float
        L.orc_row_scale.argtypes = [vp, ctypes.c_int]
        L.orc_fp16_to_bf16_n.argtypes = [vp, vp, ctypes.c_int64]
        L.orc_bf16_to_fp16_n.argtypes = [vp, vp, ctypes.c_int64]
        L.orc_dequant_row.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, vp,
                                      ctypes.c_float, vp]
        L.orc_f32_to_e5m2_n.argtypes = [vp, vp, ctypes.c_int64]
        L.orc_row_scale_to.restype = ctypes.c_float
        L.orc_row_scale_to.argtypes = [vp, ctypes.c_int, ctypes.c_float]
        L.orc_src_heads.restype = ctypes.c_int32
        L.orc_src_heads.argtypes = [P(Problem)]
        L.orc_dst_heads.restype = ctypes.c_int32
        L.orc_dst_heads.argtypes = [P(Problem)]
        L.orc_f32_to_e4m3fn_n.argtypes = [vp, vp, ctypes.c_int64]
        L.orc_decode_n.argtypes = [ctypes.c_int, vp, vp, ctypes.c_int64]
        L.orc_convert_row.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, vp, vp, vp]
        L.orc_validate.restype = ctypes.c_int
        L.orc_validate.argtypes = [P(Problem)]
        L.orc_head_source.argtypes = [P(Problem), ctypes.c_int, P(ctypes.c_int), P(ctypes.c_int)]
        L.orc_src_request_base.restype = ctypes.c_int64
        L.orc_src_request_base.argtypes = [P(Problem), ctypes.c_int]
        L.orc_src_index.restype = ctypes.c_int64
        L.orc_src_index.argtypes = [P(Problem)] + [ctypes.c_int] * 6 + [P(ctypes.c_int)]
        L.orc_cache_index.restype = ctypes.c_int64
        L.orc_cache_index.argtypes = [P(Problem), ctypes.c_int64] + [ctypes.c_int] * 5
        L.orc_cache_scale_index.restype = ctypes.c_int64
        L.orc_cache_scale_index.argtypes = [P(Problem), ctypes.c_int64] + [ctypes.c_int] * 4
        L.orc_wire_layout.restype = ctypes.c_int64
        L.orc_wire_layout.argtypes = [P(Problem), vp, vp]
        L.orc_pack.restype = ctypes.c_int
        L.orc_pack.argtypes = [P(Problem), vp, vp]
        L.orc_unpack.restype = ctypes.c_int
        L.orc_unpack.argtypes = [P(Problem), vp, vp, vp, vp, ctypes.c_int32]
        L.orc_repack.restype = ctypes.c_int
        L.orc_repack.argtypes = [P(Problem), vp, vp, vp, vp, ctypes.c_int32]
        L.orc_expected_rows.restype = ctypes.c_int
        L.orc_expected_rows.argtypes = [P(Problem), vp] + [ctypes.c_int] * 5 + [vp, vp]
        _lib = L
    return _lib


class Problem(ctypes.Structure):
    _fields_ = [
        ("layers", ctypes.c_int32), ("heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("src_tp", ctypes.c_int32), ("dst_tp", ctypes.c_int32), ("dst_rank", ctypes.c_int32),
        ("src_fmt", ctypes.c_int32), ("dst_fmt", ctypes.c_int32), ("src_order", ctypes.c_int32),
        ("block_size", ctypes.c_int32), ("num_blocks", ctypes.c_int64),
        ("num_requests", ctypes.c_int32), ("seq_lens", ctypes.POINTER(ctypes.c_int32)),
        ("src_block_size", ctypes.c_int32), ("src_num_blocks", ctypes.c_int64),
        ("src_block_table", ctypes.POINTER(ctypes.c_int32)), ("src_bt_stride", ctypes.c_int32),
        ("src_layer_offset", ctypes.c_int32), ("src_layers", ctypes.c_int32),
        ("dst_layer_offset", ctypes.c_int32), ("dst_layers", ctypes.c_int32),
        ("cache_fmt", ctypes.c_int32),
    ]


class OracleProblem:
    """Problem description plus the arrays it points into (seq_lens, and for a
    PAGED source the source block table [num_requests][src_bt_stride])."""

    def __init__(self, layers, heads, head_dim, src_tp, dst_tp, dst_rank, src_fmt, dst_fmt,
                 src_order, block_size, num_blocks, seq_lens, src_block_size=0,
                 src_num_blocks=0, src_block_table=None, src_bt_stride=0, src_layer_offset=0,
                 src_layers=0, dst_layer_offset=0, dst_layers=0, cache_fmt=0):
        self.seq_lens = np.ascontiguousarray(np.asarray(seq_lens, dtype=np.int32))
        self.src_block_table = None
        sbt = ctypes.POINTER(ctypes.c_int32)()
        if src_block_table is not None:
            self.src_block_table = np.ascontiguousarray(np.asarray(src_block_table, dtype=np.int32))
            sbt = self.src_block_table.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        self.c = Problem(layers, heads, head_dim, src_tp, dst_tp, dst_rank, src_fmt, dst_fmt,
                         src_order, block_size, num_blocks, len(self.seq_lens),
                         self.seq_lens.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                         src_block_size, src_num_blocks, sbt, src_bt_stride, src_layer_offset,
                         src_layers, dst_layer_offset, dst_layers, cache_fmt)

    def __getattr__(self, name):
        return getattr(self.__dict__["c"], name)

    @property
    def hs(self):
        return lib().orc_src_heads(self.ref())

    @property
    def hd(self):
        return lib().orc_dst_heads(self.ref())

    @property
    def dst_layers_held(self):
        return self.c.dst_layers or self.c.layers

    @property
    def dst_size(self):
        """element size of the transfer tensor"""
        return FMT_SIZE[self.c.dst_fmt]

    @property
    def cache_fmt_eff(self):
        return self.c.cache_fmt or self.c.dst_fmt

    @property
    def cache_size(self):
        return FMT_SIZE[self.cache_fmt_eff]

    def ref(self):
        return ctypes.byref(self.c)


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else ctypes.c_void_p(0)


def _shard_ptrs(shards):
    arr = (ctypes.c_void_p * len(shards))()
    for j, s in enumerate(shards):
        if s is not None:
            assert s.dtype.itemsize == 2 and s.flags["C_CONTIGUOUS"]
            arr[j] = s.ctypes.data
    return arr


# ---- casts -----------------------------------------------------------------

def decode(fmt: int, bits: np.ndarray) -> np.ndarray:
    bits = np.ascontiguousarray(bits, dtype=np.uint8 if fmt in FP8 else np.uint16)
    out = np.empty(bits.shape, dtype=np.float64)
    lib().orc_decode_n(fmt, _ptr(bits), _ptr(out), bits.size)
    return out


def fp16_to_bf16(bits: np.ndarray) -> np.ndarray:
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.empty_like(bits)
    lib().orc_fp16_to_bf16_n(_ptr(bits), _ptr(out), bits.size)
    return out


def dequant_row(cache_fmt: int, q: np.ndarray, s, code_fmt: int = E4M3FN) -> np.ndarray:
    """8-bit codes (uint8, e4m3fn or e5m2) of one row and their fp32 scale ->
    16-bit bits."""
    q = np.ascontiguousarray(q, dtype=np.uint8)
    out = np.empty(q.size, dtype=np.uint16)
    lib().orc_dequant_row(code_fmt, cache_fmt, q.size, _ptr(q), ctypes.c_float(float(s)),
                          _ptr(out))
    return out


def bf16_to_fp16(bits: np.ndarray) -> np.ndarray:
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.empty_like(bits)
    lib().orc_bf16_to_fp16_n(_ptr(bits), _ptr(out), bits.size)
    return out


def f32_to_e4m3fn(v: np.ndarray) -> np.ndarray:
    v = np.ascontiguousarray(v, dtype=np.float32)
    out = np.empty(v.shape, dtype=np.uint8)
    lib().orc_f32_to_e4m3fn_n(_ptr(v), _ptr(out), v.size)
    return out


def f32_to_e5m2(v: np.ndarray) -> np.ndarray:
    v = np.ascontiguousarray(v, dtype=np.float32)
    out = np.empty(v.shape, dtype=np.uint8)
    lib().orc_f32_to_e5m2_n(_ptr(v), _ptr(out), v.size)
    return out


def row_scale(x: np.ndarray, fmax: float = 448.0) -> np.float32:
    x = np.ascontiguousarray(x, dtype=np.float32)
    return np.float32(lib().orc_row_scale_to(_ptr(x), x.size, ctypes.c_float(fmax)))


def convert_row(src_fmt: int, dst_fmt: int, row_bits: np.ndarray):
    """Convert one row (uint16 bit patterns); returns (dst bytes, scale or None)."""
    row_bits = np.ascontiguousarray(row_bits, dtype=np.uint16)
    D = row_bits.size
    out = np.empty(D * FMT_SIZE[dst_fmt], dtype=np.uint8)
    sc = np.zeros(1, dtype=np.float32)
    lib().orc_convert_row(src_fmt, dst_fmt, D, _ptr(row_bits), _ptr(out), _ptr(sc))
    return out, (sc[0] if dst_fmt in FP8 else None)


# ---- index maps --------------------------------------------------------------

def validate(p: OracleProblem) -> int:
    return lib().orc_validate(p.ref())


def head_source(p: OracleProblem, i: int):
    j, h = ctypes.c_int(), ctypes.c_int()
    lib().orc_head_source(p.ref(), i, ctypes.byref(j), ctypes.byref(h))
    return j.value, h.value


def src_index(p: OracleProblem, r, l, kv, t, i, d):
    j = ctypes.c_int()
    idx = lib().orc_src_index(p.ref(), r, l, kv, t, i, d, ctypes.byref(j))
    return j.value, idx


def cache_index(p: OracleProblem, block, l, kv, slot, i, d):
    return lib().orc_cache_index(p.ref(), block, l, kv, slot, i, d)


def wire_layout(p: OracleProblem):
    R = len(p.seq_lens)
    data_off = np.zeros(max(R, 1), dtype=np.int64)
    scale_off = np.zeros(max(R, 1), dtype=np.int64)
    total = lib().orc_wire_layout(p.ref(), _ptr(data_off), _ptr(scale_off))
    return data_off[:R], scale_off[:R], int(total)


def cache_bytes(p: OracleProblem) -> int:
    return p.dst_layers_held * 2 * p.num_blocks * p.block_size * p.hd * p.head_dim * p.cache_size


def scale_count(p: OracleProblem) -> int:
    return p.dst_layers_held * 2 * p.num_blocks * p.block_size * p.hd


# ---- the operations ------------------------------------------------------------

def _check(rc):
    if rc != 0:
        raise ValueError(f"oracle rejected the problem (code {rc})")


def pack(p: OracleProblem, shards, wire=None, sentinel=0xA5):
    if wire is None:
        wire = np.full(wire_layout(p)[2], sentinel, dtype=np.uint8)
    _check(lib().orc_pack(p.ref(), _shard_ptrs(shards), _ptr(wire)))
    return wire


def unpack(p: OracleProblem, wire, cache, scales, block_table, bt_stride):
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    _check(lib().orc_unpack(p.ref(), _ptr(wire), _ptr(cache), _ptr(scales), _ptr(bt), bt_stride))
    return cache, scales


def repack(p: OracleProblem, shards, cache, scales, block_table, bt_stride):
    bt = np.ascontiguousarray(block_table, dtype=np.int32)
    _check(lib().orc_repack(p.ref(), _shard_ptrs(shards), _ptr(cache), _ptr(scales), _ptr(bt),
                            bt_stride))
    return cache, scales


def expected_rows(p: OracleProblem, shards, r, l, kv, t0, nt, sentinel=0xA5):
    """Expected cache rows (nt*Hd, D*esize bytes, in the cache format) and
    scales (or None).  Rows with no source (a source page outside the source
    pool) keep the sentinel bytes, as the destination does."""
    row_bytes = p.head_dim * p.cache_size
    out = np.full((nt * p.hd, row_bytes), sentinel, dtype=np.uint8)
    sc = np.full(nt * p.hd * 4, sentinel, dtype=np.uint8).view(np.float32)
    _check(lib().orc_expected_rows(p.ref(), _shard_ptrs(shards), r, l, kv, t0, nt, _ptr(out),
                                   _ptr(sc)))
    return out, (sc if p.cache_fmt_eff in FP8 else None)
