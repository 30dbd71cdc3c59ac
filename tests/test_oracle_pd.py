"""Pins of the oracle of the P:D planner (Sec. III-C, Eq. 1-6 under readings
R27-R31) to things other than itself: published parameter counts of four
models (the weight model of R27), the KV bytes per token everyone quotes,
hand-worked cost terms, properties of the constrained maximisation (more
VRAM or a looser threshold never lowers the optimum; the per-GPU prefill
objective does not depend on dp), and an independent brute force over the
candidates that checks the search and its tie rule."""
import itertools
import math

import pytest

from conftest import golden_lines

from oracle import pd as P

LLAMA2_7B = P.Model(32, 4096, 32, 32, 128, 11008, 32000)
LLAMA3_8B = P.Model(32, 4096, 32, 8, 128, 14336, 128256)
LLAMA3_70B = P.Model(80, 8192, 64, 8, 128, 28672, 128256)
MIXTRAL = P.Model(32, 4096, 32, 8, 128, 14336, 32000, experts=8, active_experts=2)
TINY = P.Model(2, 8, 2, 1, 4, 16, 10)


@pytest.mark.parametrize("m,count", [(LLAMA2_7B, 6_738_415_616), (LLAMA3_8B, 8_030_261_248),
                                     (LLAMA3_70B, 70_553_706_496), (MIXTRAL, 46_702_792_704)])
def test_parameter_counts_match_published(m, count):
    """The published parameter counts of these checkpoints (model cards)."""
    assert P.parameters(m) == count


def test_kv_bytes_per_token():
    """bf16 KV per token: 2 (K, V) x layers x KV heads x head_dim x 2 bytes,
    128 KiB for Llama-3-8B, 320 KiB for Llama-3-70B, 512 KiB for Llama-2-7B."""
    assert P.kv_per_gpu(LLAMA3_8B, 1, 1) == 128 * 1024
    assert P.kv_per_gpu(LLAMA3_70B, 1, 1) == 320 * 1024
    assert P.kv_per_gpu(LLAMA2_7B, 1, 1) == 512 * 1024
    assert P.kv_per_gpu(LLAMA3_70B, 1, 2) == 160 * 1024
    assert P.kv_per_gpu(LLAMA3_70B, 1, 16) == 40 * 1024      # one replicated head per GPU


def _tiny_problem(**kw):
    g = P.Gpu(1000.0, 1000.0, 1e9, 100.0, 0.5, 0.5, 0.5)
    base = dict(model=TINY, prefill=g, decode=g, prompt_tokens=3, output_tokens=2, qps=1.0,
                ttft=100.0, tpot=100.0)
    base.update(kw)
    return P.Problem(**base)


def test_hand_worked_costs():
    rows = golden_lines("pd_costs.txt")
    assert len(rows) == 3
    p = _tiny_problem()
    for ln in rows:
        f = ln.split()
        side, (dp, tp, pp, ep, b) = f[0], map(int, f[1:6])
        lat, mem, thr = float(f[6]), float(f[7]), float(f[8])
        cost = P.prefill_cost if side == "prefill" else P.decode_cost
        l, m, t = cost(p, dp, tp, pp, ep, b)
        assert l == pytest.approx(lat, rel=1e-12) and m == mem and t == pytest.approx(thr, rel=1e-12), ln


def test_prefill_flops_approach_two_per_parameter():
    """Short prompts: projections and experts cost 2 FLOPs per weight per
    token (the usual 2N rule, embedding table aside)."""
    proj, ffn, attn, head = P.prefill_flops(LLAMA3_8B, 1, 1)
    per_layer = P.attention_weights(LLAMA3_8B) + P.expert_weights(LLAMA3_8B)
    assert proj + ffn == 2 * LLAMA3_8B.layers * per_layer
    assert attn == 2 * 32 * 32 * 128 * 2      # one token attends to itself: QK and PV


def _mi355x(**kw):
    base = dict(flops=2.5e15, hbm_bytes=8e12, vram=288e9, link_bytes=7 * 153e9, lam=0.5,
                alpha=0.8, beta=0.7, max_gpus=8)
    base.update(kw)
    return P.Gpu(**base)


def _problem(m=LLAMA3_70B, **kw):
    base = dict(model=m, prefill=_mi355x(), decode=_mi355x(), prompt_tokens=2048,
                output_tokens=256, qps=20.0, ttft=2.0, tpot=0.05, max_batch=64)
    base.update(kw)
    return P.Problem(**base)


def _brute(p, side):
    """Independent enumeration: every (dp, tp, pp, ep, batch) within the limits
    of R31, filtered, maximised; the tie rule applied by sorting."""
    m = p.model
    g = p.prefill if side == "p" else p.decode
    best = []
    for dp, tp, pp, k in itertools.product(range(1, 9), range(1, 9), range(1, 9), range(0, 9)):
        b = 2 ** k
        if b > p.max_batch or dp * tp * pp > g.max_gpus:
            continue
        if m.q_heads % tp or (m.kv_heads % tp and tp % m.kv_heads) or m.layers % pp:
            continue
        eps = [1] if m.experts == 1 else [e for e in range(1, 9)
                                          if m.experts % e == 0 and (dp * tp) % e == 0]
        for ep in eps:
            if side == "p":
                l, mem, t = P.prefill_cost(p, dp, tp, pp, ep, b)
                ok, obj = l <= p.ttft and mem <= g.vram, t / (dp * tp * pp)
            else:
                l, mem, t = P.decode_cost(p, dp, tp, pp, ep, b)
                ok, obj = l <= p.tpot and mem <= g.vram, t
            if ok:
                best.append((obj, (dp * tp * pp, tp, pp, dp, ep, b)))
    top = max(o for o, _ in best)
    keys = sorted(k for o, k in best if o >= top * (1 - P.TIE))
    return top, keys[0], len(best)


@pytest.mark.parametrize("m", [LLAMA3_8B, LLAMA3_70B, MIXTRAL])
def test_search_matches_brute_force(m):
    p = _problem(m)
    sol = P.search(p)
    for side, ch, feas in (("p", sol.prefill, sol.feasible_prefill),
                           ("d", sol.decode, sol.feasible_decode)):
        top, key, n = _brute(p, side)
        assert n == feas
        assert ch.objective == pytest.approx(top, rel=1e-12)
        assert (ch.gpus, ch.tp, ch.pp, ch.dp, ch.ep, ch.batch) == key
    assert sol.prefill_instances == math.ceil(p.qps / sol.prefill.throughput)
    assert sol.decode_instances == math.ceil(p.qps * p.output_tokens / sol.decode.throughput)


def test_looser_constraints_never_lower_the_optimum():
    base = P.search(_problem())
    for kw in (dict(ttft=4.0), dict(tpot=0.1), dict(prefill=_mi355x(vram=400e9)),
               dict(decode=_mi355x(vram=400e9))):
        s = P.search(_problem(**kw))
        assert s.prefill.objective >= base.prefill.objective * (1 - 1e-12)
        assert s.decode.objective >= base.decode.objective * (1 - 1e-12)


def test_prefill_objective_does_not_depend_on_dp():
    p = _problem(LLAMA3_8B)
    for tp, pp, b in ((1, 1, 4), (2, 2, 8), (8, 1, 1)):
        objs = [P.prefill_cost(p, dp, tp, pp, 1, b)[2] / (dp * tp * pp)
                for dp in range(1, 8 // (tp * pp) + 1)]
        assert max(objs) == pytest.approx(min(objs), rel=1e-12)


def test_infeasible_problem_has_no_choice():
    sol = P.search(_problem(ttft=1e-6))
    assert sol.feasible_prefill == 0 and sol.prefill.gpus == 0 and sol.prefill_instances == 0
    sol = P.search(_problem(decode=_mi355x(vram=1e9)))
    assert sol.feasible_decode == 0 and sol.decode.gpus == 0 and sol.decode_instances == 0


def test_tensor_parallel_degrees_follow_the_head_map():
    """Only degrees the KV conversion supports: tp divides H or is a multiple
    of H (and divides the query heads)."""
    tps = {c[1] for c in P.candidates(LLAMA3_70B, 64, 1)}
    assert tps == {1, 2, 4, 8, 16, 32, 64}
    tps = {c[1] for c in P.candidates(P.Model(28, 3584, 28, 4, 128, 18944, 152064), 8, 1)}
    assert tps == {1, 2, 4}           # 28 query heads: 8 does not divide them


def test_instance_counts_hand_worked():
    """R30 on the tiny model with one candidate per side (1 GPU, batch 1):
    prefill T_p = 1 / 14.912 requests/s (first row of pd_costs.txt); decode
    at batch 1 reads the 2528 weight bytes of that file plus the KV of a
    4-token context (4 x 2 x 2 layers x 1 head x 4 dims x 2 B = 128 B), so
    l_d = 2656 / 500 = 5.312 s and T_d = 1 / 5.312 tokens/s.  At 0.5
    requests/s of 2 output tokens: X = ceil(0.5 x 14.912) = ceil(7.456) = 8
    prefill and Y = ceil(0.5 x 2 x 5.312) = ceil(5.312) = 6 decode
    instances."""
    g = P.Gpu(1000.0, 1000.0, 1e9, 100.0, 0.5, 0.5, 0.5, max_gpus=1)
    p = _tiny_problem(prefill=g, decode=g, qps=0.5, max_batch=1)
    sol = P.search(p)
    assert sol.decode.latency == pytest.approx(5.312, rel=1e-12)
    assert (sol.prefill_instances, sol.decode_instances) == (8, 6)


def test_tie_goes_to_fewest_gpus():
    """R31's tie rule on a case where it decides.  With an unlimited
    interconnect every prefill strategy's compute splits exactly, so the
    per-GPU objective b / (l_p tp) is the same for all of them; 280 kB of
    VRAM leaves out tp = 1 with pp = 1 or 2 (weights and one layer's
    activations do not fit) and admits tp = 2 with pp = 1 and tp = 1 with
    pp = 4.  Among equal objectives the fewest GPUs win: tp 2, pp 1 (2 GPUs)
    over tp 1, pp 4 (4 GPUs), although the latter has the smaller tp."""
    m = P.Model(4, 64, 4, 1, 16, 16, 100)
    g = P.Gpu(1e9, 1e9, 280000.0, 1e30, max_gpus=4)
    p = P.Problem(m, g, g, 256, 2, 1.0, 1e9, 1e9, max_batch=1)
    assert P.prefill_cost(p, 1, 1, 1, 1, 1)[1] > g.vram
    assert P.prefill_cost(p, 1, 1, 2, 1, 1)[1] > g.vram
    a, b = P.prefill_cost(p, 1, 2, 1, 1, 1), P.prefill_cost(p, 1, 1, 4, 1, 1)
    assert a[1] <= g.vram and b[1] <= g.vram
    assert a[2] / 2 == pytest.approx(b[2] / 4, rel=1e-12)
    ch = P.search(p).prefill
    assert (ch.dp, ch.tp, ch.pp, ch.gpus) == (1, 2, 1, 2)
