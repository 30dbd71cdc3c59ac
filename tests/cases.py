"""Workload cases and helpers shared by the test modules.

Small cases keep the structure of the five full workloads (same heads,
head_dim, TP mapping, dtypes, orders and page sizes) with fewer layers,
requests and tokens, so the oracle finishes in well under a second while
still spanning several pages per request and a ragged last page."""
from __future__ import annotations

import numpy as np
import torch

import workload as W

FULL = W.WORKLOADS
TINY = FULL["tiny_tp1to2_fp16_bf16"]
L8B = FULL["llama3_8b_bf16_bs16"]
L70B = FULL["llama3_70b_tp4to2_bf16_bs32"]
QWEN = FULL["qwen7b_htd_fp16_bf16_bs64"]
FP8 = FULL["fp8_decode_61l_bf16_e4m3_bs16"]
P8B = FULL["llama3_8b_paged16_bf16_bs64"]
P70B = FULL["llama3_70b_paged16_tp4to2_bf16_bs32"]

SMALL = {
    "tiny": TINY,
    "llama3_8b_small": L8B.replace(name="llama3_8b_small", layers=2, total_layers=2,
                                   num_requests=3, len_lo=17, len_hi=100, num_blocks=64),
    "llama3_70b_small_r0": L70B.replace(name="llama3_70b_small_r0", layers=2, total_layers=2,
                                        num_requests=2, len_lo=33, len_hi=90, num_blocks=16),
    "llama3_70b_small_r1": L70B.replace(name="llama3_70b_small_r1", layers=2, total_layers=2,
                                        num_requests=2, len_lo=33, len_hi=90, num_blocks=16,
                                        dst_rank=1),
    "qwen_htd_small": QWEN.replace(name="qwen_htd_small", layers=2, total_layers=2,
                                   num_requests=3, len_lo=10, len_hi=150, num_blocks=16),
    "fp8_small": FP8.replace(name="fp8_small", layers=2, total_layers=3, num_requests=3,
                             len_lo=5, len_hi=70, num_blocks=64),
    # split: prefill TP2 -> decode TP4, rank 3 (second half of shard 1)
    "split_tp2to4_r3": L8B.replace(name="split_tp2to4_r3", layers=2, total_layers=2, src_tp=2,
                                   dst_tp=4, dst_rank=3, num_requests=2, len_lo=20, len_hi=50,
                                   num_blocks=16),
    # merge everything: prefill TP8 -> decode TP1, head-major fp16 -> bf16
    "merge_tp8to1_htd": QWEN.replace(name="merge_tp8to1_htd", heads=8, layers=1, total_layers=1,
                                     src_tp=8, dst_tp=1, num_requests=2, len_lo=3, len_hi=40,
                                     block_size=16, num_blocks=16),
    # ratio that is not a power of two: 6 heads, prefill TP2 -> decode TP3 rank 1
    "tp2to3_r1_fp8": FP8.replace(name="tp2to3_r1_fp8", heads=6, layers=2, total_layers=2,
                                 src_tp=2, dst_tp=3, dst_rank=1, num_requests=2, len_lo=1,
                                 len_hi=33, num_blocks=16),
    # fp16 -> e4m3fn, head-major, with an empty request in the batch
    "fp16_e4m3_htd_empty": QWEN.replace(name="fp16_e4m3_htd_empty", dst_dtype="e4m3fn",
                                        layers=1, total_layers=1, num_requests=4,
                                        lens_override=(37, 0, 16, 1), block_size=16,
                                        num_blocks=16, seed=99),
    # GQA with more ranks than KV heads: 4 heads, decode TP8 rank 5 holds the
    # replicated head 2
    "gqa_rep_tp1to8_r5": QWEN.replace(name="gqa_rep_tp1to8_r5", layers=2, total_layers=2,
                                      src_order="thd", dst_tp=8, dst_rank=5, num_requests=2,
                                      len_lo=9, len_hi=70, block_size=16, num_blocks=16),
    # replicated prefill shards: 4 heads over prefill TP8 (shard j holds head
    # j // 2) -> decode TP2 rank 1 (heads 2, 3), bf16 -> e4m3fn
    "gqa_src_rep_tp8to2_r1": FP8.replace(name="gqa_src_rep_tp8to2_r1", heads=4, layers=2,
                                         total_layers=2, src_tp=8, dst_tp=2, dst_rank=1,
                                         num_requests=2, len_lo=5, len_hi=40, num_blocks=16),
    # both sides replicated: 2 heads, prefill TP4 -> decode TP8 rank 7, head-major
    "gqa_both_rep_tp4to8_r7": QWEN.replace(name="gqa_both_rep_tp4to8_r7", heads=2, layers=1,
                                          total_layers=1, src_tp=4, dst_tp=8, dst_rank=7,
                                          num_requests=2, len_lo=3, len_hi=50, block_size=16,
                                          num_blocks=16),
    # bf16 -> fp16 with values up to about 4 sigma = 160000: many overflow to
    # infinity, the rest round to nearest even (subnormals from the tail)
    "bf16_fp16_overflow": L8B.replace(name="bf16_fp16_overflow", dst_dtype="fp16", layers=2,
                                      total_layers=2, num_requests=2, len_lo=20, len_hi=60,
                                      num_blocks=16, sigma=40000.0),
    "bf16_fp16_small_values": L8B.replace(name="bf16_fp16_small_values", dst_dtype="fp16",
                                          layers=1, total_layers=1, num_requests=1,
                                          len_lo=40, len_hi=40, num_blocks=8, sigma=1e-6),
}

# Dequantising unpack: e4m3fn codes and scales in the transfer tensor, a
# 16-bit decode cache holding q * s.
SMALL_DEQUANT = {
    "dequant_bf16_e4m3_bf16": FP8.replace(name="dequant_bf16_e4m3_bf16", cache_dtype="bf16",
                                          layers=2, total_layers=3, num_requests=3, len_lo=5,
                                          len_hi=70, num_blocks=64),
    "dequant_fp16_e4m3_fp16_htd": QWEN.replace(name="dequant_fp16_e4m3_fp16_htd",
                                               dst_dtype="e4m3fn", cache_dtype="fp16", layers=2,
                                               total_layers=2, num_requests=3, len_lo=10,
                                               len_hi=150, num_blocks=16),
    "dequant_paged_tp4to2_bf16": P70B.replace(name="dequant_paged_tp4to2_bf16", dst_dtype="e4m3fn",
                                              cache_dtype="bf16", layers=2, total_layers=2,
                                              num_requests=2, len_lo=33, len_hi=90,
                                              num_blocks=16, src_num_blocks=24),
    "dequant_fp16_e4m3_bf16_empty": QWEN.replace(name="dequant_fp16_e4m3_bf16_empty",
                                                 dst_dtype="e4m3fn", cache_dtype="bf16", layers=1,
                                                 total_layers=1, num_requests=4,
                                                 lens_override=(37, 0, 16, 1), block_size=16,
                                                 num_blocks=16, seed=98),
}

# e5m2 transfer tensors: the e4m3fn scheme with OCP e5m2 codes (scale
# max|x| / 57344); caches holding the codes and scales, or dequantised.
SMALL_E5M2 = {
    "e5m2_bf16": FP8.replace(name="e5m2_bf16", dst_dtype="e5m2", layers=2, total_layers=2,
                             num_requests=3, len_lo=5, len_hi=70, num_blocks=64),
    "e5m2_fp16_htd_tp2to4": QWEN.replace(name="e5m2_fp16_htd_tp2to4", dst_dtype="e5m2",
                                         layers=2, total_layers=2, src_tp=2, dst_tp=4,
                                         dst_rank=3, num_requests=3, len_lo=10, len_hi=150,
                                         num_blocks=16),
    "e5m2_paged_tp4to2": P70B.replace(name="e5m2_paged_tp4to2", dst_dtype="e5m2", layers=2,
                                      total_layers=2, num_requests=2, len_lo=33, len_hi=90,
                                      num_blocks=16, src_num_blocks=24),
    "e5m2_dequant_bf16": FP8.replace(name="e5m2_dequant_bf16", dst_dtype="e5m2",
                                     cache_dtype="bf16", layers=2, total_layers=2,
                                     num_requests=3, len_lo=5, len_hi=70, num_blocks=64),
    "e5m2_dequant_fp16_empty": QWEN.replace(name="e5m2_dequant_fp16_empty", dst_dtype="e5m2",
                                            cache_dtype="fp16", layers=1, total_layers=1,
                                            num_requests=4, lens_override=(37, 0, 16, 1),
                                            block_size=16, num_blocks=16, seed=99),
}

# Shapes at the limits of the lane layout: rows of 16 to 2048 bytes (1 to 64
# lanes per row, chunk counts that are not powers of two), 1024 heads per
# decode rank, 64 head segments.
_S = dict(layers=1, total_layers=1, num_requests=2, len_lo=5, len_hi=40, num_blocks=16)
SMALL_SHAPES = {
    # 1024-byte rows: 64 lanes per row, a whole wave; 4 rows per pass
    "hd512_bf16": L8B.replace(name="hd512_bf16", heads=2, head_dim=512, **_S),
    # 1024-byte e4m3fn rows: the row maximum exchanges beyond a 16-lane row
    "hd1024_e4m3": FP8.replace(name="hd1024_e4m3", heads=2, head_dim=1024, **_S),
    # ... dequantised into 2048-byte bf16 cache rows
    "hd1024_e4m3_bf16": FP8.replace(name="hd1024_e4m3_bf16", heads=2, head_dim=1024,
                                    cache_dtype="bf16", **_S),
    # 160-byte rows: 10 chunks on 16 lanes; TP1 -> TP2
    "hd80_fp16_bf16": TINY.replace(name="hd80_fp16_bf16", head_dim=80, **_S),
    # 48-byte 8-bit rows from head-major fp16: 3 chunks on 4 lanes
    "hd48_fp16_e5m2": QWEN.replace(name="hd48_fp16_e5m2", head_dim=48, dst_dtype="e5m2",
                                   block_size=16, **_S),
    "hd48_fp16_e4m3_fp16": QWEN.replace(name="hd48_fp16_e4m3_fp16", head_dim=48,
                                        dst_dtype="e4m3fn", cache_dtype="fp16", block_size=16,
                                        **_S),
    # 16-byte e4m3fn rows: one lane per row, 256 rows per pass; 256 heads
    "hd16_e4m3_256heads": FP8.replace(name="hd16_e4m3_256heads", heads=256, head_dim=16,
                                      block_size=4, **_S),
    # 16-byte bf16 rows and the most heads a decode rank may hold (1024)
    "hd8_bf16_1024heads": L8B.replace(name="hd8_bf16_1024heads", heads=1024, head_dim=8,
                                      block_size=2, **dict(_S, num_blocks=64)),
    # the most head segments (64): prefill TP64 -> decode TP1
    "tp64to1_64segs": L8B.replace(name="tp64to1_64segs", heads=64, head_dim=16, src_tp=64,
                                  **_S),
}

# Paged sources (the prefill side's own paged cache), same shapes as the two
# full paged workloads plus page-size ratios that do not divide each other.
SMALL_PAGED = {
    "paged16_bs64_small": P8B.replace(name="paged16_bs64_small", layers=2, total_layers=2,
                                      num_requests=3, len_lo=17, len_hi=150, num_blocks=16,
                                      src_num_blocks=48),
    "paged16_tp4to2_bs32_small": P70B.replace(name="paged16_tp4to2_bs32_small", layers=2,
                                              total_layers=2, num_requests=2, len_lo=33,
                                              len_hi=90, num_blocks=16, src_num_blocks=24),
    # 24-token prefill pages -> 16-token decode pages (neither divides the other)
    "paged24_bs16_r1": P70B.replace(name="paged24_bs16_r1", layers=1, total_layers=1,
                                    dst_rank=1, num_requests=3, len_lo=1, len_hi=80,
                                    block_size=16, num_blocks=32, src_block_size=24,
                                    src_num_blocks=16),
    # 16 -> 24-token pages, bf16 -> e4m3fn, one empty request
    "paged16_e4m3_bs24": FP8.replace(name="paged16_e4m3_bs24", src_order="paged", layers=2,
                                     total_layers=3, num_requests=3, lens_override=(50, 0, 7),
                                     block_size=24, num_blocks=16, src_block_size=16,
                                     src_num_blocks=16),
    # fp16 -> bf16 split TP1 -> TP2 rank 0 from 5-token prefill pages
    "paged5_fp16_split": TINY.replace(name="paged5_fp16_split", src_order="paged", num_requests=2,
                                      len_lo=3, len_hi=40, lens_override=None,
                                      src_block_size=5, src_num_blocks=24),
}



def random_workloads(seed: int, n: int) -> dict:
    """n small valid workloads drawn over every option of the descriptor:
    heads 1..16 with every TP degree that divides them or that they divide
    (replicated heads included), any decode rank, all dtype pairs and
    dequantising caches, the three source orders, head_dim 8..1024, page
    sizes that are not powers of two, empty requests, value scales over five
    decades.  Each pool stays under 8 MiB so that the oracle runs in
    milliseconds."""
    rng = np.random.default_rng(seed)
    out = {}
    while len(out) < n:
        H = int(rng.choice([1, 2, 3, 4, 6, 8, 12, 16]))
        tps = [t for t in range(1, H + 1) if H % t == 0] + [2 * H, 4 * H]
        src_tp, dst_tp = int(rng.choice(tps)), int(rng.choice(tps))
        src = str(rng.choice(["fp16", "bf16"]))
        dst = str(rng.choice(["fp16", "bf16", "e4m3fn", "e5m2"]))
        cache = str(rng.choice(["fp16", "bf16"])) if dst in FP8_NAMES and rng.random() < 0.4 else ""
        esz = 1 if dst in FP8_NAMES else 2
        dims = [d for d in (8, 16, 24, 32, 40, 48, 64, 80, 96, 128, 192, 256, 512, 1024)
                if d * esz <= 1024 and (d * esz) % 16 == 0]
        D = int(rng.choice(dims))
        order = str(rng.choice(["thd", "htd", "paged"]))
        bs = int(rng.choice([1, 2, 3, 5, 8, 16, 17, 32, 64]))
        R = int(rng.integers(0, 6))
        lens = [0 if rng.random() < 0.15 else int(rng.integers(1, 121)) for _ in range(R)]
        L = int(rng.integers(1, 4))
        nb = sum((t + bs - 1) // bs for t in lens) + int(rng.integers(0, 7))
        sbs = snb = 0
        if order == "paged":
            sbs = int(rng.choice([1, 3, 4, 7, 16, 32]))
            snb = max(1, sum((t + sbs - 1) // sbs for t in lens) + int(rng.integers(0, 7)))
        hd = H // dst_tp if dst_tp <= H else 1
        hs = H // src_tp if src_tp <= H else 1
        csz = 1 if (cache or dst) in FP8_NAMES else 2
        if L * 2 * max(nb, 1) * bs * hd * D * csz > 8 << 20 or \
                L * 2 * max(sum(lens), snb * sbs) * hs * D * 2 > 8 << 20:
            continue
        sigma = float(10.0 ** rng.uniform(-2.0, 2.5))
        frac = float(rng.choice([0.0, 0.01]))
        k = len(out)
        out[f"rand{k}"] = W.Workload(
            f"rand{k}", L, L, H, D, src_tp, dst_tp, int(rng.integers(0, dst_tp)), src, dst, order,
            bs, max(nb, 1), R, 0, 0, seed=int(rng.integers(1, 1 << 30)), sigma=sigma,
            outlier_frac=frac, outlier_value=float(rng.uniform(100.0, 60000.0)),
            head_scale_log10=(-2.0, 2.0) if rng.random() < 0.3 else None,
            lens_override=tuple(lens), src_block_size=sbs, src_num_blocks=snb, cache_dtype=cache)
    return out



def out_of_pool(table, limit, rng, frac=0.1):
    """A copy of a block table with about `frac` of its used entries (>= 0)
    replaced by ids outside [0, limit): -1 .. -3 or limit .. limit + 99.
    Rows that map to such a page are neither read nor written."""
    t = np.array(table, dtype=np.int32, copy=True)
    used = np.argwhere(t >= 0)
    pick = used[rng.random(len(used)) < frac]
    for i, j in pick:
        t[i, j] = -int(rng.integers(1, 4)) if rng.random() < 0.5 else limit + int(rng.integers(0, 100))
    return t

FP8_NAMES = ("e4m3fn", "e5m2")
RANDOM = random_workloads(2509_17542, 64)
# 8-bit formats: torch dtype and largest finite value (the scale's divisor)
_FP8 = {"e4m3fn": (torch.float8_e4m3fn, 448.0), "e5m2": (torch.float8_e5m2, 57344.0)}


def fmt_codes(mod):
    """dtype name -> the integer code used by `mod` (oracle or GPU binding)."""
    return {"fp16": mod.FP16, "bf16": mod.BF16, "e4m3fn": mod.E4M3FN, "e5m2": mod.E5M2}


def dst_size(w):
    """element size of the decode cache"""
    return 1 if w.cdt in FP8_NAMES else 2


def wire_size(w):
    """element size of the transfer tensor"""
    return 1 if w.dst_dtype in FP8_NAMES else 2


def oracle_problem(O, w, lens, layers=None, sbt=None):
    """The oracle's problem for workload w; a paged source takes the
    generator's source block table unless `sbt` ([R, stride] int32) is given."""
    f = fmt_codes(O)
    order = {"thd": O.TOKEN_MAJOR, "htd": O.HEAD_MAJOR, "paged": O.PAGED}[w.src_order]
    extra = {}
    if w.src_order == "paged":
        if sbt is None:
            sbt, _ = W.src_block_table(w, lens)
        extra = dict(src_block_size=w.src_block_size, src_num_blocks=w.src_num_blocks,
                     src_block_table=sbt, src_bt_stride=sbt.shape[1])
    if w.cache_dtype:
        extra["cache_fmt"] = f[w.cache_dtype]
    return O.OracleProblem(layers or w.layers, w.heads, w.head_dim, w.src_tp, w.dst_tp,
                           w.dst_rank, f[w.src_dtype], f[w.dst_dtype], order, w.block_size,
                           w.num_blocks, lens, **extra)


def rank_heads(w):
    """Global heads [g0, g1) of the produced decode rank: [rank*Hd,
    (rank+1)*Hd), or the one head rank // (dst_tp / H) when dst_tp is a
    multiple of H (tensor parallelism replicates KV heads then)."""
    if w.dst_tp <= w.heads:
        return w.dst_rank * w.hd, (w.dst_rank + 1) * w.hd
    g = w.dst_rank // (w.dst_tp // w.heads)
    return g, g + 1


def read_shards(w):
    """Prefill shards that store a head of the produced decode rank (with
    replicated heads, every replica): the ones the test inputs need."""
    lo, hi = rank_heads(w)
    return [j for j in range(w.src_tp) if w.shard_heads(j)[0] < hi and w.shard_heads(j)[1] > lo]


def inputs(w, layer0=0, nlayers=None):
    lens = W.seq_lens(w)
    bt, stride = W.block_table(w, lens)
    shards = W.source_shards(w, lens, layer0, nlayers, read_shards(w))
    return lens, bt, stride, shards


# ---- library-only construction of what the decode side must see ------------

_TDT = {"fp16": torch.float16, "bf16": torch.bfloat16}


def consumer_rows(w, lens, r, layer0, nlayers):
    """Expected decode-side rows of request r, built only from the generator's
    logical values and torch library conversions:
    returns (rows uint8 [L][2][T][Hd][D*esize], scales float32 [L][2][T][Hd] or None).

    Heads: the decode rank holds global heads [rank*Hd, (rank+1)*Hd), or the
    one head rank // (dst_tp / H) when dst_tp is a multiple of H.
    Casts: same type = bits; fp16->bf16 and bf16->fp16 = torch .to();
    a 16-bit cache under an 8-bit transfer = q.float() * s then .to();
    e4m3fn = s = amax/448 in fp32, q = clamp(x/s, +-448).to(float8_e4m3fn),
    e5m2 the same with 57344 and float8_e5m2."""
    heads = rank_heads(w)
    x = torch.from_numpy(W.logical_values(w, lens, r, layer0, nlayers, heads))
    x = x.to(_TDT[w.src_dtype])                                     # [L][2][Hd][T][D]
    x = x.permute(0, 1, 3, 2, 4).contiguous()                      # [L][2][T][Hd][D]
    if x.numel() == 0:   # an empty request: no rows (torch cannot view empty tensors as bytes)
        row = w.head_dim * (1 if w.cdt in FP8_NAMES else 2)
        return (np.zeros((*x.shape[:4], row), np.uint8),
                np.zeros(x.shape[:4], np.float32) if w.cdt in FP8_NAMES else None)
    if w.dst_dtype == w.src_dtype:
        return x.view(torch.uint8).numpy().reshape(*x.shape[:4], 2 * w.head_dim), None
    if w.dst_dtype in ("bf16", "fp16"):
        y = x.to(_TDT[w.dst_dtype])
        return y.view(torch.uint8).numpy().reshape(*y.shape[:4], 2 * w.head_dim), None
    tq, fmax = _FP8[w.dst_dtype]
    xf = x.float()
    s = xf.abs().amax(dim=-1) / torch.tensor(fmax)
    v = xf / s[..., None]
    q = v.clamp(-fmax, fmax).to(tq).view(torch.uint8)
    zero_rows = (s == 0)[..., None].expand_as(q)
    signed_zero = torch.where(torch.signbit(xf), 0x80, 0).to(torch.uint8)
    q = torch.where(zero_rows, signed_zero, q)
    if w.cdt not in FP8_NAMES:   # dequantising unpack: q * s in fp32, then the 16-bit cast
        y = (q.view(tq).float() * s[..., None]).to(_TDT[w.cdt])
        return y.view(torch.uint8).numpy().reshape(*y.shape[:4], 2 * w.head_dim), None
    return q.numpy(), s.numpy()


def gather_pages(cache_u8, w, lens, bt, r, nlayers, scales=None):
    """What a paged-attention reader sees for request r: the pages listed in
    its block-table row, in order, cut at T tokens.  cache_u8 is the whole
    destination pool as bytes; returns rows shaped like consumer_rows."""
    T = int(lens[r])
    nblk = (T + w.block_size - 1) // w.block_size
    row = w.head_dim * dst_size(w)
    c = cache_u8.reshape(nlayers, 2, w.num_blocks, w.block_size, w.hd, row)
    pages = c[:, :, bt[r, :nblk]]                                   # [L][2][nblk][bs][Hd][row]
    rows = pages.reshape(nlayers, 2, nblk * w.block_size, w.hd, row)[:, :, :T]
    sc = None
    if scales is not None:
        s = scales.reshape(nlayers, 2, w.num_blocks, w.block_size, w.hd)
        sc = s[:, :, bt[r, :nblk]].reshape(nlayers, 2, nblk * w.block_size, w.hd)[:, :, :T]
    return rows, sc


def written_mask(w, lens, bt, nlayers):
    """Bytes of the pool that the conversion must write (per page slot)."""
    m = np.zeros((nlayers, 2, w.num_blocks, w.block_size), dtype=bool)
    for r, T in enumerate(lens):
        for k in range((int(T) + w.block_size - 1) // w.block_size):
            n = min(w.block_size, int(T) - k * w.block_size)
            m[:, :, bt[r, k], :n] = True
    return m


def double_rounding_scales(bits):
    """fp32 scales s for which some e4m3fn value q makes the fp32 product q * s
    land exactly on a midpoint of a format with `bits` significand bits (11:
    fp16, 8: bf16) while the exact product does not: rounding q * s to fp32
    first, then to that format, differs from rounding the exact product
    once.  One scale per (q, midpoint) pair tried."""
    def rne(x, p):
        e = np.floor(np.log2(abs(x)))
        step = 2.0 ** (p - 1 - e)
        return np.rint(x * step) / step

    out = []
    for q in (1.875, 1.625, 1.375, 1.125, 1.75, 1.25):
        for mid in (1 + 2.0 ** -bits, 1 + 3 * 2.0 ** -bits, 1.5 + 2.0 ** -bits):
            s0 = np.float32(mid / q)
            for k in range(1, 41):
                s = s0
                for _ in range(k // 2):
                    s = np.nextafter(s, np.float32(np.inf if k % 2 else -np.inf))
                p = q * float(s)                    # exact in float64
                if rne(float(np.float32(p)), bits) != rne(p, bits):
                    out.append(float(s))
                    break
    return out


# ---- cast sweeps: rows of chosen bit patterns in a one-request workload ----

def sweep_case(src, dst, rows_bits):
    """One request whose 2*T rows (layer 0, k then v) are the given rows
    (uint16 [2T, 128]); TP1, one head, 16-token pages in order."""
    n = rows_bits.shape[0]
    assert n % 32 == 0
    T = n // 2
    w = W.Workload("sweep", 1, 1, 1, 128, 1, 1, 0, src, dst, "thd", 16, T // 16, 1, T, T, seed=1)
    lens = np.array([T], dtype=np.int32)
    bt = np.arange(T // 16, dtype=np.int32)[None, :]
    return w, lens, bt, [np.ascontiguousarray(rows_bits.reshape(-1))]


def pad_rows(rows):
    n = -(-rows.shape[0] // 32) * 32
    out = np.zeros((n, 128), dtype=np.uint16)
    out[:rows.shape[0]] = rows
    return out


def e4m3_sweep_rows(fmt, amaxes, rng):
    """Rows [amax, x_1..x_127] covering every finite pattern x with |x| <= amax
    (both signs) for each amax, plus NaN/Inf/zero rows."""
    allp = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    inf = 0x7C00 if fmt == "fp16" else 0x7F80
    mag = allp & 0x7FFF
    finite = allp[mag < inf]
    out = []
    for a in amaxes:
        xs = finite[(finite & 0x7FFF) <= a]
        xs = rng.permutation(xs)
        k = -(-xs.size // 127)
        xs = np.concatenate([xs, np.zeros(k * 127 - xs.size, np.uint16)]).reshape(k, 127)
        pos = rng.integers(0, 128, k)
        rows = np.empty((k, 128), np.uint16)
        for j in range(k):
            rows[j] = np.insert(xs[j], pos[j], a | (rng.integers(0, 2) << 15))
        out.append(rows)
    special = np.zeros((6, 128), np.uint16)
    special[1, :] = 0x8000                         # all -0
    special[2, 5] = inf | 0x1                      # a NaN in a zero row
    special[3, :] = 0x3C00 if fmt == "fp16" else 0x3F80
    special[3, 7] = inf                            # +Inf sets the row maximum
    special[4, :64] = (inf | 0x40) | 0x8000        # half NaN, rest zero
    special[5, :] = rng.integers(0, 0x7800, 128)
    special[5, 9] = inf | 0x20                     # one NaN among finite values
    special[5, 11] = inf | 0x8000                  # and -Inf: the row maximum is Inf
    out.append(special)
    return np.concatenate(out)


# ---- exhaustive 8-bit sweep: every row maximum, every element under it ----

FINITE_MAX = {"bf16": 0x7F7F, "fp16": 0x7BFF}   # largest finite magnitude pattern
NAN_BITS = {"bf16": 0x7FC0, "fp16": 0x7E00}     # a quiet NaN of each format


def pair_rows(fmt, mags, nan=False, block=512, threads=None):
    """Rows of 128 16-bit patterns such that, for each magnitude pattern m in
    `mags` (finite, > 0), some rows have row maximum exactly m and together
    hold every finite pattern x with |x| <= m, in both signs.  Each row holds
    127 of those patterns (the last row of each m padded with +0) plus m
    itself at column (row index mod 128), its sign flipping every 128 rows,
    so the maximum visits every lane of a row.  With nan=True each row holds
    126 patterns, m and a NaN (sign and payload varying by row) at column
    (row index + 64) mod 128: rows whose row maximum, and so their scale, is
    finite but which contain a NaN.  Returns uint16 [rows, 128]."""
    from concurrent.futures import ThreadPoolExecutor
    import os

    mags = np.asarray(mags, dtype=np.int64)
    assert mags.size and mags.min() >= 1 and mags.max() <= FINITE_MAX[fmt]
    per = 127 - int(nan)                       # patterns per row besides m (and the NaN)
    k_all = -(-(2 * (mags + 1)) // per)        # rows per maximum
    first_all = np.cumsum(k_all) - k_all       # first row of each maximum
    out = np.empty((int(k_all.sum()), 128), dtype=np.uint16)
    col = np.arange(128, dtype=np.int32)[None, :]

    def fill(b):
        m_b, k_b = mags[b:b + block], k_all[b:b + block]
        r0, n = int(first_all[b]), int(k_b.sum())
        m = np.repeat(m_b, k_b).astype(np.int32)[:, None]      # row maximum of each row
        i = (np.arange(r0, r0 + n) - np.repeat(first_all[b:b + block], k_b)).astype(np.int32)
        g = np.arange(r0, r0 + n, dtype=np.int64)              # global row index
        pos = (g % 128).astype(np.int32)[:, None]
        npos = (pos + 64) % 128
        # value index under m of each column (the columns of m and the NaN skipped)
        v = (i * per)[:, None] + col
        v -= col > pos
        if nan:
            v -= col > npos
        neg = v > m                                            # second half: the negative patterns
        v -= np.where(neg, m + 1, 0)
        v |= np.where(neg, 0x8000, 0)
        v[v >= 0x8000 + m + 1] = 0                             # padding past -m: +0
        rows = np.arange(n)
        v[rows, pos[:, 0]] = m[:, 0] | (((g // 128) & 1) << 15).astype(np.int32)
        if nan:
            v[rows, npos[:, 0]] = NAN_BITS[fmt] | (g % 7 + 1) | (((g // 2) & 1) << 15)
        out[r0:r0 + n] = v

    with ThreadPoolExecutor(threads or min(16, os.cpu_count() or 1)) as ex:
        list(ex.map(fill, range(0, mags.size, block)))
    return out

# Every conversion in every source order: each (source type, transfer-tensor
# type, cache type) the library accepts, from token-major, head-major and
# paged sources, so that every kernel instantiation runs.  Each case merges
# two prefill shards (TP2 -> TP1: two head segments), has a ragged last page
# and an empty request, and varies the row size with the order (head_dim 128
# token-major, 64 head-major, 256 paged; paged sources use 12-token pages
# against 16-token decode pages).  8-bit transfers draw per-head scales over
# four decades; bf16 -> fp16 draws values up to about 2^17, so some overflow.
_MATRIX_TYPES = [("bf16", ""), ("fp16", ""), ("e4m3fn", ""), ("e5m2", ""),
                 ("e4m3fn", "bf16"), ("e4m3fn", "fp16"), ("e5m2", "bf16"), ("e5m2", "fp16")]


def _matrix():
    out = {}
    seed = 600
    for src in ("bf16", "fp16"):
        for dst, cache in _MATRIX_TYPES:
            for order, hdim in (("thd", 128), ("htd", 64), ("paged", 256)):
                if src == dst and not cache and order != "paged":
                    continue  # a plain copy: the small and paged cases above cover it
                seed += 1
                name = f"mx_{src}_{dst}{'_' + cache if cache else ''}_{order}"
                w = W.Workload(name, 2, 2, 4, hdim, 2, 1, 0, src, dst, order, 16, 24, 3, 1, 45,
                               seed=seed, lens_override=(45, 0, 19),
                               sigma=30000.0 if (src, dst) == ("bf16", "fp16") else 1.0,
                               head_scale_log10=(-2.0, 2.0) if dst in ("e4m3fn", "e5m2") else None,
                               src_block_size=12 if order == "paged" else 0,
                               src_num_blocks=16 if order == "paged" else 0,
                               cache_dtype=cache)
                out[name] = w
    return out


MATRIX = _matrix()
