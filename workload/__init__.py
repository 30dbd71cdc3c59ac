"""Seeded synthetic KV-cache workloads, shared by the tests and the benchmark.

This module draws random numbers and arranges them in the prefill side's
storage order (which heads each prefill shard stores, token- or head-major
buffers, or the prefill side's own pages); it holds none of the conversion's
arithmetic (no head map to the decode side, no decode paging, no casts of the
method).  Values are keyed by
logical coordinates (request, layer, k/v, global head, token, dim), so a
different shard split or storage order of the same workload holds the same
values.

The C core (``gen.c``) is a counter-based splitmix64 stream; see its header.
Streams: 1 sequence lengths, 2 block-table permutation, 3 values,
4 outlier mask, 5 outlier sign, 6 per-(layer, k/v, head) scale, 7 the
prefill side's own block-table permutation (paged sources).
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB_PATH = os.path.join(_HERE, "libkvxgen.so")
GCC_CMD = ["gcc", "-std=c99", "-O2", "-Wall", "-fPIC", "-shared", "-pthread", "-o", _LIB_PATH,
           _SRC, "-lm"]

SENTINEL = 0xA5

S_LENS, S_TABLE, S_VALUES, S_OUTLIER, S_OUTSIGN, S_HEADSCALE, S_SRC_TABLE = 1, 2, 3, 4, 5, 6, 7


def build() -> str:
    subprocess.run(GCC_CMD, check=True)
    return _LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        u64, u32, i64, vp = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int64, ctypes.c_void_p
        L.wl_word.restype = u64
        L.wl_word.argtypes = [u64, u32, u64]
        L.wl_uniform.restype = ctypes.c_double
        L.wl_uniform.argtypes = [u64, u32, u64]
        L.wl_normal.restype = ctypes.c_double
        L.wl_normal.argtypes = [u64, u32, u64]
        L.wl_fill_normal.argtypes = [u64, u32, u64, i64, ctypes.c_double, vp, ctypes.c_int]
        L.wl_fill_normal_blocks.argtypes = [u64, u32, vp, i64, i64, ctypes.c_double, vp,
                                            ctypes.c_int]
        L.wl_fill_uniform.argtypes = [u64, u32, u64, i64, vp]
        L.wl_select.restype = i64
        L.wl_select.argtypes = [u64, u32, u64, i64, ctypes.c_double, vp]
        L.wl_permutation.argtypes = [u64, u32, i64, vp]
        _lib = L
    return _lib


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    layers: int            # layers handled by one plan (a layer group for grouped runs)
    total_layers: int      # layers of the model; values are keyed by the global layer
    heads: int             # global KV heads
    head_dim: int
    src_tp: int
    dst_tp: int
    dst_rank: int
    src_dtype: str         # "fp16" | "bf16"
    dst_dtype: str         # "fp16" | "bf16" | "e4m3fn" | "e5m2"
    src_order: str         # "thd" = [token][head][dim], "htd" = [head][token][dim],
                           # "paged" = the prefill side's own paged cache
    block_size: int
    num_blocks: int
    num_requests: int
    len_lo: int
    len_hi: int
    seed: int
    sigma: float = 1.0
    outlier_frac: float = 0.0
    outlier_value: float = 0.0
    head_scale_log10: tuple | None = None
    lens_override: tuple | None = None   # explicit tokens per request (edge cases)
    src_block_size: int = 0  # "paged" sources: tokens per prefill-side page
    src_num_blocks: int = 0  # "paged" sources: pages per (layer, k/v) plane of each shard's pool
    src_pp: int = 1          # prefill pipeline stages: equal layer ranges, one buffer set each
    cache_dtype: str = ""    # decode cache type when it differs from dst_dtype (dequantising unpack)

    @property
    def cdt(self):
        """element type of the decode cache"""
        return self.cache_dtype or self.dst_dtype

    @property
    def hs(self):
        """heads per prefill shard: H / src_tp, or 1 when src_tp is a multiple
        of H (each head then lives on src_tp / H consecutive shards)"""
        return self.heads // self.src_tp if self.src_tp <= self.heads else 1

    @property
    def hd(self):
        """heads per decode rank, likewise (sizes the decode pool)"""
        return self.heads // self.dst_tp if self.dst_tp <= self.heads else 1

    def shard_heads(self, j: int) -> tuple[int, int]:
        """Global heads [g0, g1) that prefill shard j stores."""
        if self.src_tp <= self.heads:
            return j * self.hs, (j + 1) * self.hs
        g = j // (self.src_tp // self.heads)
        return g, g + 1


    @property
    def layer_groups(self):
        return math.ceil(self.total_layers / self.layers)

    def group_layers(self, g: int) -> tuple[int, int]:
        """(first global layer, layer count) of layer group g."""
        l0 = g * self.layers
        return l0, min(self.layers, self.total_layers - l0)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The workloads: the decode-side shapes of four model families plus a tiny
# one, then variants of them (paged sources, pipeline stages, replicated GQA
# heads, other casts and 8-bit formats).  Sizes: layers x KV heads x
# head_dim, tokens per request.
WORKLOADS = {
    w.name: w
    for w in [
        # 2 layers, 4 heads, dim 64, one 256-token request, TP1 -> TP2 rank 0,
        # fp16 -> bf16, 64-block pool of 16-token pages
        Workload("tiny_tp1to2_fp16_bf16", 2, 2, 4, 64, 1, 2, 0, "fp16", "bf16", "thd",
                 16, 64, 1, 256, 256, seed=17542),
        # Llama-3-8B KV shape: 32 layers, 8 heads, dim 128; 16 requests of
        # 512..4096 tokens; bf16 re-layout into 16-token pages of a 65536-page pool
        Workload("llama3_8b_bf16_bs16", 32, 32, 8, 128, 1, 1, 0, "bf16", "bf16", "thd",
                 16, 65536, 16, 512, 4096, seed=17543),
        # Llama-3-70B shard: 80 layers, 8 heads, dim 128; 8 requests of
        # 1024..8192 tokens; prefill TP4 -> decode TP2 rank 0 (merges shards 0, 1);
        # 32-token pages, 16384-page pool
        Workload("llama3_70b_tp4to2_bf16_bs32", 80, 80, 8, 128, 4, 2, 0, "bf16", "bf16", "thd",
                 32, 16384, 8, 1024, 8192, seed=17544),
        # Qwen-7B-style GQA: 28 layers, 4 heads, dim 128; 32 requests of
        # 128..2048 tokens; fp16 head-major source, sigma 2 with 0.1% outliers at
        # +-60000 -> bf16 token-major 64-token pages, 8192-page pool
        Workload("qwen7b_htd_fp16_bf16_bs64", 28, 28, 4, 128, 1, 1, 0, "fp16", "bf16", "htd",
                 64, 8192, 32, 128, 2048, seed=17545, sigma=2.0, outlier_frac=0.001,
                 outlier_value=60000.0),
        # fp8 decode cache: 61 layers (run as groups of 4), 8 heads, dim 128;
        # 64 requests of 256..16384 tokens; bf16 with a per-(layer, k/v, head)
        # scale 10^U(-2, 2) -> e4m3fn + fp32 per-(token, head) scale, 16-token
        # pages of a 2^20-page pool
        Workload("fp8_decode_61l_bf16_e4m3_bs16", 4, 61, 8, 128, 1, 1, 0, "bf16", "e4m3fn", "thd",
                 16, 1 << 20, 64, 256, 16384, seed=17546, head_scale_log10=(-2.0, 2.0)),
        # paged -> paged, Llama-3-8B KV shape: the prefill side's own cache of
        # 16-token pages (4096-page pool) re-paged into 64-token decode pages
        # (4096-page pool); 16 requests of 512..4096 tokens, bf16
        Workload("llama3_8b_paged16_bf16_bs64", 32, 32, 8, 128, 1, 1, 0, "bf16", "bf16", "paged",
                 64, 4096, 16, 512, 4096, seed=17547, src_block_size=16, src_num_blocks=4096),
        # paged -> paged with a TP change, Llama-3-70B shard: prefill TP4 caches
        # of 16-token pages (4096-page pool per shard) -> decode TP2 rank 0 with
        # 32-token pages (16384-page pool); 8 requests of 1024..8192 tokens, bf16
        Workload("llama3_70b_paged16_tp4to2_bf16_bs32", 80, 80, 8, 128, 4, 2, 0, "bf16", "bf16",
                 "paged", 32, 16384, 8, 1024, 8192, seed=17548, src_block_size=16,
                 src_num_blocks=4096),
        # the Llama-3-8B workload (same seed, same values) from a prefill side
        # in 2 pipeline stages of 16 layers, each with its own buffers, into
        # one decode cache: one plan per stage
        Workload("llama3_8b_pp2to1_bf16_bs16", 32, 32, 8, 128, 1, 1, 0, "bf16", "bf16", "thd",
                 16, 65536, 16, 512, 4096, seed=17543, src_pp=2),
        # the Qwen-7B-style GQA workload (4 KV heads, same seed and values) into
        # a decode side with tensor parallelism 8: rank 5 holds a replica of
        # KV head 2; 16 KiB pages of one head
        Workload("qwen7b_gqa_tp1to8_r5_fp16_bf16_bs64", 28, 28, 4, 128, 1, 8, 5, "fp16", "bf16",
                 "htd", 64, 8192, 32, 128, 2048, seed=17545, sigma=2.0, outlier_frac=0.001,
                 outlier_value=60000.0),
        # the Llama-3-8B workload (same seed and values) cast bf16 -> fp16
        Workload("llama3_8b_bf16_fp16_bs16", 32, 32, 8, 128, 1, 1, 0, "bf16", "fp16", "thd",
                 16, 65536, 16, 512, 4096, seed=17543),
        # the Llama-3-8B workload (same seed and values) moved as e4m3fn codes
        # with per-(token, head) scales and dequantised into a bf16 cache
        Workload("llama3_8b_bf16_e4m3_bf16_bs16", 32, 32, 8, 128, 1, 1, 0, "bf16", "e4m3fn",
                 "thd", 16, 65536, 16, 512, 4096, seed=17543, cache_dtype="bf16"),
        # the Llama-3-8B workload (same seed and values) into an e5m2 cache with
        # per-(token, head) fp32 scales
        Workload("llama3_8b_bf16_e5m2_bs16", 32, 32, 8, 128, 1, 1, 0, "bf16", "e5m2", "thd",
                 16, 65536, 16, 512, 4096, seed=17543),
    ]
}


def seq_lens(w: Workload) -> np.ndarray:
    """T_r = lo + floor(u_r * (hi - lo + 1)), or the explicit lengths."""
    if w.lens_override is not None:
        return np.asarray(w.lens_override, dtype=np.int32)
    u = np.empty(w.num_requests, dtype=np.float64)
    lib().wl_fill_uniform(w.seed, S_LENS, 0, w.num_requests, u.ctypes.data)
    lens = w.len_lo + np.floor(u * (w.len_hi - w.len_lo + 1)).astype(np.int64)
    return np.minimum(lens, w.len_hi).astype(np.int32)


def permutation(seed: int, n: int, stream: int = S_TABLE) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)
    lib().wl_permutation(seed, stream, n, out.ctypes.data)
    return out


def block_table(w: Workload, lens: np.ndarray, consecutive: bool = False) -> tuple[np.ndarray, int]:
    """Pages for each request, drawn in order from a seeded permutation of the
    pool (or, with consecutive=True, pages 0, 1, 2, ... in request order: the
    same page counts with no scatter).  Returns ([R, stride] int32 with -1 in
    unused entries, stride)."""
    nblk = [(int(t) + w.block_size - 1) // w.block_size for t in lens]
    stride = max(nblk + [1])
    need = sum(nblk)
    if need > w.num_blocks:
        raise ValueError(f"{w.name}: {need} pages needed, pool has {w.num_blocks}")
    perm = np.arange(w.num_blocks, dtype=np.int64) if consecutive else \
        permutation(w.seed, w.num_blocks)
    bt = np.full((len(lens), stride), -1, dtype=np.int32)
    pos = 0
    for r, n in enumerate(nblk):
        bt[r, :n] = perm[pos:pos + n]
        pos += n
    return bt, stride


def src_stages(w: Workload) -> list[tuple[int, int]]:
    """(first layer, layer count) of each prefill pipeline stage: w.layers
    split into w.src_pp ranges as equal as possible, earlier stages larger."""
    q, rem = divmod(w.layers, w.src_pp)
    out, l0 = [], 0
    for k in range(w.src_pp):
        n = q + (1 if k < rem else 0)
        out.append((l0, n))
        l0 += n
    return out


def src_block_table(w: Workload, lens: np.ndarray) -> tuple[np.ndarray, int]:
    """The prefill side's pages for each request ("paged" sources), drawn in
    order from a seeded permutation of its pool (stream 7).  The same table
    serves every prefill shard.  Returns ([R, stride] int32, -1 in unused
    entries, stride)."""
    sbs = w.src_block_size
    nblk = [(int(t) + sbs - 1) // sbs for t in lens]
    stride = max(nblk + [1])
    need = sum(nblk)
    if need > w.src_num_blocks:
        raise ValueError(f"{w.name}: {need} source pages needed, pool has {w.src_num_blocks}")
    perm = permutation(w.seed, w.src_num_blocks, S_SRC_TABLE)
    sbt = np.full((len(lens), stride), -1, dtype=np.int32)
    pos = 0
    for r, n in enumerate(nblk):
        sbt[r, :n] = perm[pos:pos + n]
        pos += n
    return sbt, stride


def _request_value_base(w: Workload, lens: np.ndarray, r: int) -> int:
    return int(sum(w.total_layers * 2 * w.heads * int(t) * w.head_dim for t in lens[:r]))


def logical_values(w: Workload, lens: np.ndarray, r: int, layer0: int, nlayers: int,
                   heads: tuple[int, int] | None = None, out: np.ndarray | None = None
                   ) -> np.ndarray:
    """float32 values of request r, layers [layer0, layer0+nlayers), global
    heads [g0, g1) (default all), shaped [layer][k/v][head][token][dim].

    Element (l, kv, g, t, d) is draw number
    base(r) + (((l*2 + kv)*H + g)*T + t)*D + d of the value stream, base(r)
    being the element count of all earlier requests over all layers."""
    T = int(lens[r])
    H, D = w.heads, w.head_dim
    g0, g1 = heads if heads is not None else (0, H)
    shape = (nlayers, 2, g1 - g0, T, D)
    if out is not None:   # caller-provided scratch (reused, so no fresh pages per request)
        x = out.reshape(-1)[:int(np.prod(shape))].reshape(shape)
    else:
        x = np.empty(shape, dtype=np.float32)
    if x.size == 0:
        return x
    base = _request_value_base(w, lens, r)
    n = T * D
    # one block of T*D consecutive draws per (layer, k/v, head)
    li, kv, g = np.meshgrid(np.arange(nlayers), np.arange(2), np.arange(g0, g1), indexing="ij")
    starts = (base + (((layer0 + li) * 2 + kv) * H + g) * n).astype(np.uint64).reshape(-1)
    lib().wl_fill_normal_blocks(w.seed, S_VALUES, starts.ctypes.data, starts.size, n, w.sigma,
                                x.ctypes.data, _threads())
    if w.outlier_frac > 0:
        flat_all = x.reshape(starts.size, n)
        idx = np.empty(n, dtype=np.int64)
        for b, start in enumerate(starts.tolist()):
            c = lib().wl_select(w.seed, S_OUTLIER, start, n, w.outlier_frac, idx.ctypes.data)
            for k in idx[:c]:
                neg = lib().wl_uniform(w.seed, S_OUTSIGN, start + int(k)) < 0.5
                flat_all[b, k] = -w.outlier_value if neg else w.outlier_value
    if w.head_scale_log10 is not None:
        lo, hi = w.head_scale_log10
        u = np.empty(w.total_layers * 2 * H, dtype=np.float64)
        lib().wl_fill_uniform(w.seed, S_HEADSCALE, 0, u.size, u.ctypes.data)
        sc = (10.0 ** (lo + (hi - lo) * u)).astype(np.float32).reshape(w.total_layers, 2, H)
        x *= sc[layer0:layer0 + nlayers, :, g0:g1, None, None]
    return x


def _to_bits(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float32 to the 16-bit storage type (torch's round-to-nearest-even)
    and return the bit patterns as uint16."""
    import torch
    t = torch.from_numpy(x).to(_TORCH_DTYPE[dtype]())
    return t.view(torch.int16).numpy().view(np.uint16)


_TORCH_DTYPE = {"fp16": lambda: __import__("torch").float16,
                "bf16": lambda: __import__("torch").bfloat16}


def source_shards(w: Workload, lens: np.ndarray, layer0: int = 0, nlayers: int | None = None,
                  shards: list[int] | None = None) -> list[np.ndarray | None]:
    """Prefill-side shard buffers (uint16 bit patterns), one per source TP rank.

    Shard j holds global heads [j*Hs, (j+1)*Hs); requests are stored back to
    back, each as [layer][k/v][token][head][dim] ("thd") or
    [layer][k/v][head][token][dim] ("htd").  A "paged" shard is instead the
    prefill side's pool [layer][k/v][src_num_blocks][src_block_size][head][dim]:
    token t of request r sits in page src_block_table(w, lens)[r][t //
    src_block_size], slot t % src_block_size; slots holding no token keep the
    sentinel bytes.  Values are rounded from float32 to the storage type by
    torch (round to nearest even).  Shards not listed in `shards` (default:
    all of them) are None."""
    import torch
    if nlayers is None:
        nlayers = w.layers
    if shards is None:
        shards = list(range(w.src_tp))
    Hs, D = w.hs, w.head_dim
    if w.src_order == "paged":
        return _paged_source_shards(w, lens, layer0, nlayers, shards)
    per_shard = sum(nlayers * 2 * int(t) * Hs * D for t in lens)
    out: list[np.ndarray | None] = [None] * w.src_tp
    for j in shards:
        out[j] = np.empty(per_shard, dtype=np.uint16)   # first touched by torch's copy below
    scratch = np.empty(max([nlayers * 2 * int(t) * Hs * D for t in lens] + [1]), np.float32)
    tdt = _TORCH_DTYPE[w.src_dtype]()
    off = 0
    for r in range(len(lens)):
        T = int(lens[r])
        n = nlayers * 2 * T * Hs * D
        if n == 0:
            continue
        for j in shards:
            vals = torch.from_numpy(
                logical_values(w, lens, r, layer0, nlayers, w.shard_heads(j), scratch))
            dst = torch.from_numpy(out[j][off:off + n].view(np.int16)).view(tdt)
            if w.src_order == "thd":
                dst.view(nlayers, 2, T, Hs, D).copy_(vals.permute(0, 1, 3, 2, 4))
            else:
                dst.view(nlayers, 2, Hs, T, D).copy_(vals)
        off += n
    return out


def _paged_source_shards(w: Workload, lens: np.ndarray, layer0: int, nlayers: int,
                         shards: list[int]) -> list[np.ndarray | None]:
    import torch
    Hs, D, sbs, nbs = w.hs, w.head_dim, w.src_block_size, w.src_num_blocks
    sbt, _ = src_block_table(w, lens)
    out: list[np.ndarray | None] = [None] * w.src_tp
    for j in shards:
        out[j] = np.full(nlayers * 2 * nbs * sbs * Hs * D, SENTINEL * 0x0101, dtype=np.uint16)
    scratch = np.empty(max([nlayers * 2 * int(t) * Hs * D for t in lens] + [1]), np.float32)
    tdt = _TORCH_DTYPE[w.src_dtype]()
    for r in range(len(lens)):
        T = int(lens[r])
        if T == 0 or nlayers == 0:
            continue
        nb = (T + sbs - 1) // sbs
        full = T // sbs
        for j in shards:
            vals = torch.from_numpy(
                logical_values(w, lens, r, layer0, nlayers, w.shard_heads(j), scratch))
            x = vals.permute(0, 1, 3, 2, 4).to(tdt).view(torch.int16).numpy()  # [l][kv][t][h][d]
            pool = out[j].view(np.int16).reshape(nlayers, 2, nbs, sbs, Hs, D)
            ids = sbt[r, :nb]
            if full:
                pool[:, :, ids[:full]] = x[:, :, :full * sbs].reshape(nlayers, 2, full, sbs, Hs, D)
            if T > full * sbs:
                pool[:, :, ids[full], :T - full * sbs] = x[:, :, full * sbs:]
    return out
