"""Plain oracle of the joint optimisation of parallel strategy and P:D ratio
(Sec. III-C, Eq. 1-6).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: the test suite and
the benchmark may call it; the library never does.  Plain Python loops over
every candidate strategy, each cost term written out as its own expression,
in float64.

What the paper fixes (Sec. III-C):
  Eq. 1  prefill: maximise T_p / (dp*tp*pp) over (dp, tp, pp, ep) subject to
         l_p <= L_ttft and m_p <= M_p;
  Eq. 2  l_p = c_p / (lambda R_p) + e_p / (beta B_p);
  Eq. 3  m_p = m_p^weight + m_p^activation;
  Eq. 4  decode: maximise sum_y T_y^d / Y over (dp, tp, pp, ep, Y) subject to
         l_d <= L_tpot and m_d <= M_d;
  Eq. 5  l_d = e_d^VRAM / (alpha B_d^VRAM) + e_d^comm / (beta B_d);
  Eq. 6  m_d = m_d^weight + m_d^activation + m_d^KV.
What it leaves open, and the readings taken here (R27-R31):
  R27  the cost terms: a decoder-only transformer (attention with hq query and
       H KV heads of dim D, a gated FFN of three h x F matrices per expert,
       RMSNorm weights, untied embedding and LM head); FLOPs 2 per
       multiply-add, causal attention; tensor parallelism splits attention,
       dense FFNs and the embedding/head by tp, expert parallelism places
       E/ep whole experts per GPU, pipeline parallelism splits layers by pp;
       TP all-reduces 2 per layer (ring: 2(tp-1)/tp of the bytes), PP hands
       the hidden states over pp-1 times, EP all-to-alls 2 per layer.
  R28  throughput: an instance keeps pp batches in flight, dp replicas:
       T = dp * pp * batch / l (requests/s for prefill, tokens/s for decode);
       the pp batches in flight keep their KV on the GPUs, so the KV held per
       GPU does not shrink with pp.
  R29  the batch size is a search variable (powers of two up to max_batch);
       decode reads the KV of an average context s_in + s_out / 2 per step
       and holds the full s_in + s_out.
  R30  instances: X = ceil(qps / T_p) prefill and Y = ceil(qps * s_out / T_d)
       decode instances (all D instances alike, so sum_y T_y / Y = T_d).
  R31  candidates: tp divides hq and either divides H or is a multiple of it
       (the KV conversion's head map), pp divides L, ep = 1 for dense models
       or divides E and dp*tp; dp*tp*pp <= max_gpus.  Ties (objectives within
       a relative 1e-9) go to the smallest (gpus, tp, pp, dp, ep, batch).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

TIE = 1e-9


@dataclass
class Model:
    layers: int
    hidden: int
    q_heads: int
    kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    experts: int = 1
    active_experts: int = 1
    weight_bytes: float = 2.0
    kv_bytes: float = 2.0
    act_bytes: float = 2.0


@dataclass
class Gpu:
    flops: float        # R, FLOP/s per GPU
    hbm_bytes: float    # B^VRAM, bytes/s per GPU
    vram: float         # M, bytes per GPU
    link_bytes: float   # B, interconnect bytes/s per GPU
    lam: float = 1.0
    alpha: float = 1.0
    beta: float = 1.0
    max_gpus: int = 8


@dataclass
class Problem:
    model: Model
    prefill: Gpu
    decode: Gpu
    prompt_tokens: int
    output_tokens: int
    qps: float
    ttft: float
    tpot: float
    max_batch: int = 256


@dataclass
class Choice:
    dp: int = 0
    tp: int = 0
    pp: int = 0
    ep: int = 0
    batch: int = 0
    gpus: int = 0
    latency: float = 0.0
    vram: float = 0.0
    throughput: float = 0.0
    objective: float = 0.0


@dataclass
class Solution:
    prefill: Choice = field(default_factory=Choice)
    decode: Choice = field(default_factory=Choice)
    prefill_instances: int = 0
    decode_instances: int = 0
    candidates_prefill: int = 0
    candidates_decode: int = 0
    feasible_prefill: int = 0
    feasible_decode: int = 0


# ---- model sizes (R27) --------------------------------------------------------

def attention_weights(m: Model) -> int:
    """Q, K, V and O projections of one layer (elements)."""
    q = m.hidden * m.q_heads * m.head_dim
    k = m.hidden * m.kv_heads * m.head_dim
    v = m.hidden * m.kv_heads * m.head_dim
    o = m.q_heads * m.head_dim * m.hidden
    return q + k + v + o


def expert_weights(m: Model) -> int:
    """Gate, up and down matrices of one FFN expert (elements)."""
    return 3 * m.hidden * m.ffn_dim


def router_weights(m: Model) -> int:
    """The expert router of one layer (h x E), none for a dense model."""
    return m.hidden * m.experts if m.experts > 1 else 0


def parameters(m: Model) -> int:
    """All weights: per layer attention, E experts, the router and two
    RMSNorm vectors; the final norm; untied embedding and LM head."""
    per_layer = (attention_weights(m) + m.experts * expert_weights(m) + router_weights(m)
                 + 2 * m.hidden)
    return m.layers * per_layer + m.hidden + 2 * m.vocab * m.hidden


def kv_heads_per_gpu(m: Model, tp: int) -> int:
    """H / tp, or one (replicated) head when tp is a multiple of H."""
    return m.kv_heads // tp if tp <= m.kv_heads else 1


def weights_per_gpu(m: Model, tp: int, pp: int, ep: int) -> float:
    """Bytes of weights on the most loaded GPU: its stage's layers (attention
    split by tp; a dense FFN split by tp, experts E/ep whole per GPU; router
    and norms whole) plus the embedding and the LM head split by tp (both on
    one GPU when pp = 1, one of them on the first or last stage otherwise)
    and the final norm."""
    layers = m.layers / pp
    if m.experts == 1:
        ffn = expert_weights(m) / tp
    else:
        ffn = (m.experts / ep) * expert_weights(m)
    per_layer = attention_weights(m) / tp + ffn + router_weights(m) + 2 * m.hidden
    tables = (2 if pp == 1 else 1) * m.vocab * m.hidden / tp
    return m.weight_bytes * (layers * per_layer + tables + m.hidden)


# ---- prefill (Eq. 1-3) -----------------------------------------------------------

def prefill_flops(m: Model, b: int, s: int):
    """FLOPs of one batch of b prompts of s tokens, by part: (attention
    projections, experts (k per token), causal attention scores and context,
    the LM head on each request's last token)."""
    proj = 2 * b * s * m.layers * attention_weights(m)
    ffn = 2 * b * s * m.layers * m.active_experts * expert_weights(m)
    attn = 2 * m.layers * m.q_heads * m.head_dim * b * s * (s + 1)
    head = 2 * b * m.vocab * m.hidden
    return proj, ffn, attn, head


def comm_bytes(m: Model, tokens: float, tp: int, pp: int, ep: int) -> float:
    """Bytes each GPU moves on the critical path for `tokens` hidden states:
    2 ring all-reduces per layer (TP), pp - 1 stage hand-overs (PP), 2
    all-to-alls per layer (EP)."""
    hid = tokens * m.hidden * m.act_bytes
    e_tp = m.layers * 2 * (2 * (tp - 1) / tp) * hid if tp > 1 else 0.0
    e_pp = (pp - 1) * hid
    e_ep = (m.layers * 2 * m.active_experts * hid * (ep - 1) / ep
            if (m.experts > 1 and ep > 1) else 0.0)
    return e_tp + e_pp + e_ep


def activations_per_gpu(m: Model, tokens: float, tp: int) -> float:
    """One layer's working set for `tokens` tokens: hidden states in and out,
    query and attention output, the FFN's three intermediates (split by tp)."""
    return tokens * (4 * m.hidden + 3 * m.active_experts * m.ffn_dim / tp) * m.act_bytes


def kv_per_gpu(m: Model, tokens: float, tp: int) -> float:
    """KV bytes of `tokens` tokens over all layers on one GPU (R28: the pp
    batches in flight hold their KV, so the layer split does not reduce it)."""
    return tokens * 2 * m.layers * kv_heads_per_gpu(m, tp) * m.head_dim * m.kv_bytes


def prefill_cost(p: Problem, dp: int, tp: int, pp: int, ep: int, b: int):
    """(l_p, m_p, T_p) of Eq. 2, Eq. 3 and R28."""
    m, g, s = p.model, p.prefill, p.prompt_tokens
    proj, ffn, attn, head = prefill_flops(m, b, s)
    ffn_split = tp if m.experts == 1 else ep
    c_crit = (proj + attn + head) / tp + ffn / ffn_split
    e_comm = comm_bytes(m, b * s, tp, pp, ep)
    l_p = c_crit / (g.lam * g.flops) + e_comm / (g.beta * g.link_bytes)          # Eq. 2
    m_p = (weights_per_gpu(m, tp, pp, ep)                                        # Eq. 3
           + activations_per_gpu(m, b * s, tp) + kv_per_gpu(m, b * s, tp))
    t_p = dp * pp * b / l_p
    return l_p, m_p, t_p


# ---- decode (Eq. 4-6) --------------------------------------------------------------

def decode_cost(p: Problem, dp: int, tp: int, pp: int, ep: int, b: int):
    """(l_d, m_d, T_d) of Eq. 5, Eq. 6 and R28-R29."""
    m, g = p.model, p.decode
    # weights read per step: every layer's attention share, the experts the
    # batch touches on this GPU (at most its E/ep, at most b*k), router and
    # norms, the LM head share (the embedding lookup reads b rows: ignored)
    if m.experts == 1:
        ffn_read = expert_weights(m) / tp
    else:
        ffn_read = min(m.experts / ep, b * m.active_experts) * expert_weights(m)
    w_read = m.weight_bytes * (m.layers * (attention_weights(m) / tp + ffn_read
                                           + router_weights(m) + 2 * m.hidden)
                               + m.vocab * m.hidden / tp)
    ctx_read = p.prompt_tokens + p.output_tokens / 2
    e_vram = w_read + kv_per_gpu(m, b * ctx_read, tp)
    e_comm = comm_bytes(m, b, tp, pp, ep)
    l_d = e_vram / (g.alpha * g.hbm_bytes) + e_comm / (g.beta * g.link_bytes)   # Eq. 5
    ctx_held = p.prompt_tokens + p.output_tokens
    m_d = (weights_per_gpu(m, tp, pp, ep) + activations_per_gpu(m, b, tp)      # Eq. 6
           + kv_per_gpu(m, b * ctx_held, tp))
    t_d = dp * pp * b / l_d
    return l_d, m_d, t_d


# ---- candidates and search (Eq. 1, Eq. 4, R30-R31) ---------------------------------

def candidates(m: Model, max_gpus: int, max_batch: int):
    """Every (dp, tp, pp, ep, batch) allowed by R31, in the tie-break order."""
    out = []
    for dp in range(1, max_gpus + 1):
        for tp in range(1, max_gpus + 1):
            if m.q_heads % tp:
                continue
            if m.kv_heads % tp and tp % m.kv_heads:
                continue
            for pp in range(1, max_gpus + 1):
                if m.layers % pp or dp * tp * pp > max_gpus:
                    continue
                eps = [1] if m.experts == 1 else [e for e in range(1, m.experts + 1)
                                                  if m.experts % e == 0 and (dp * tp) % e == 0]
                for ep in eps:
                    b = 1
                    while b <= max_batch:
                        out.append((dp, tp, pp, ep, b))
                        b *= 2
    out.sort(key=lambda c: (c[0] * c[1] * c[2], c[1], c[2], c[0], c[3], c[4]))
    return out


def _best(rows):
    """rows: (key tuple, objective, choice) of feasible candidates in key order."""
    if not rows:
        return Choice()
    top = max(r[1] for r in rows)
    for _, obj, ch in rows:
        if obj >= top * (1 - TIE):
            return ch
    return Choice()


def search(p: Problem) -> Solution:
    sol = Solution()
    rows = []
    for (dp, tp, pp, ep, b) in candidates(p.model, p.prefill.max_gpus, p.max_batch):
        sol.candidates_prefill += 1
        l_p, m_p, t_p = prefill_cost(p, dp, tp, pp, ep, b)
        if l_p <= p.ttft and m_p <= p.prefill.vram:                              # Eq. 1 (c1), (c2)
            obj = t_p / (dp * tp * pp)                                           # Eq. 1 objective
            rows.append(((dp, tp, pp, ep, b), obj,
                         Choice(dp, tp, pp, ep, b, dp * tp * pp, l_p, m_p, t_p, obj)))
    sol.feasible_prefill = len(rows)
    sol.prefill = _best(rows)
    rows = []
    for (dp, tp, pp, ep, b) in candidates(p.model, p.decode.max_gpus, p.max_batch):
        sol.candidates_decode += 1
        l_d, m_d, t_d = decode_cost(p, dp, tp, pp, ep, b)
        if l_d <= p.tpot and m_d <= p.decode.vram:                               # Eq. 4 (c1), (c2)
            rows.append(((dp, tp, pp, ep, b), t_d,                               # Eq. 4 objective
                         Choice(dp, tp, pp, ep, b, dp * tp * pp, l_d, m_d, t_d, t_d)))
    sol.feasible_decode = len(rows)
    sol.decode = _best(rows)
    if sol.prefill.gpus and sol.decode.gpus:                                     # R30
        sol.prefill_instances = math.ceil(p.qps / sol.prefill.throughput)
        sol.decode_instances = math.ceil(p.qps * p.output_tokens / sol.decode.throughput)
    return sol
