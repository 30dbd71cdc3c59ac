// Joint optimisation of parallel strategy and P:D ratio (Sec. III-C): the
// search of Eq. 1 over the prefill instance's (dp, tp, pp, ep) and of Eq. 4
// over the decode instance's, with the latency models of Eq. 2 and Eq. 5 and
// the memory models of Eq. 3 and Eq. 6.  The paper leaves every cost term
// open; the model below is a decoder-only transformer:
//   - weights: attention Q/K/V/O, a gated FFN (three h x F matrices) per
//     expert, a router per layer when there are experts, two norm vectors
//     per layer and a final one, untied embedding and LM head;
//   - placement: tp splits attention, dense FFNs and the embedding/head; ep
//     places E/ep whole experts on a GPU; pp splits layers (the embedding
//     and the head sit on the first and last stage);
//   - FLOPs: 2 per multiply-add; causal attention; the prefill's LM head on
//     each request's last token;
//   - communication: 2 ring all-reduces per layer (2(tp-1)/tp of the bytes
//     per GPU), pp-1 stage hand-overs, 2 all-to-alls per layer for experts;
//   - throughput: pp batches in flight per replica, dp replicas, so the KV
//     held per GPU does not shrink with pp; decode reads the KV of the
//     average context s_in + s_out/2 and holds s_in + s_out;
//   - the batch is a search variable (powers of two); instances
//     X = ceil(qps / T_p), Y = ceil(qps * s_out / T_d).
// Candidates: tp divides the query heads and either divides the KV heads or
// is a multiple of them (what the KV conversion's head map supports), pp
// divides the layers, ep = 1 (dense) or divides E and dp*tp, dp*tp*pp GPUs
// at most max_gpus.  They are visited in the order (GPUs, tp, pp, dp, ep,
// batch); among objectives within a relative 1e-9 of the best, the first wins.
#include <cmath>
#include <cstring>
#include <vector>

#include "kvx.h"
#include "kvx_host.h"

namespace {

using kvx::fail;

constexpr double kTie = 1e-9;

// Element counts of the model's weight groups (R27).
struct Weights {
    double attn;    // Q, K, V, O of one layer
    double expert;  // one gated FFN
    double router;  // one layer's router (0 when dense)
    double norms;   // one layer's two norm vectors
    double table;   // embedding or LM head

    explicit Weights(const kvx_pd_model& m)
    {
        const double h = m.hidden, d = m.head_dim;
        attn = 2.0 * h * m.q_heads * d + 2.0 * h * m.kv_heads * d;
        expert = 3.0 * h * m.ffn_dim;
        router = m.experts > 1 ? h * m.experts : 0.0;
        norms = 2.0 * h;
        table = double(m.vocab) * h;
    }
};

struct Strategy {
    int dp, tp, pp, ep, batch;
};

class Evaluator {
public:
    explicit Evaluator(const kvx_pd_problem& p) : p_(p), m_(p.model), w_(p.model) {}

    // weights held by the most loaded GPU (bytes)
    double held_weights(const Strategy& s) const
    {
        const double ffn = dense() ? w_.expert / s.tp : (double(m_.experts) / s.ep) * w_.expert;
        const double layer = w_.attn / s.tp + ffn + w_.router + w_.norms;
        const double tables = (s.pp == 1 ? 2.0 : 1.0) * w_.table / s.tp;
        return m_.weight_bytes * (double(m_.layers) / s.pp * layer + tables + m_.hidden);
    }

    // KV bytes of `tokens` tokens on one GPU (every layer: pp batches in flight)
    double kv(double tokens, int tp) const
    {
        const int heads = tp <= m_.kv_heads ? m_.kv_heads / tp : 1;
        return tokens * 2.0 * m_.layers * heads * m_.head_dim * m_.kv_bytes;
    }

    // one layer's working activations for `tokens` tokens on one GPU
    double work(double tokens, int tp) const
    {
        return tokens * (4.0 * m_.hidden + 3.0 * m_.active_experts * double(m_.ffn_dim) / tp) *
               m_.act_bytes;
    }

    // bytes a GPU sends on the critical path for `tokens` hidden states
    double comm(double tokens, const Strategy& s) const
    {
        const double x = tokens * m_.hidden * m_.act_bytes;
        double e = (s.pp - 1) * x;
        if (s.tp > 1) e += 2.0 * m_.layers * x * 2.0 * (s.tp - 1) / s.tp;
        if (!dense() && s.ep > 1) e += 2.0 * m_.layers * m_.active_experts * x * (s.ep - 1) / s.ep;
        return e;
    }

    // Eq. 2 and Eq. 3 for one prefill batch; T_p in requests/s
    kvx_pd_choice prefill(const Strategy& s) const
    {
        const kvx_pd_gpu& g = p_.prefill;
        const double b = s.batch, n = p_.prompt_tokens, L = m_.layers;
        const double tokens = b * n;
        const double split_part = 2.0 * tokens * L * w_.attn +                        // projections
                                  2.0 * L * m_.q_heads * m_.head_dim * b * n * (n + 1.0) +  // attention
                                  2.0 * b * w_.table;                                  // LM head
        const double experts = 2.0 * tokens * L * m_.active_experts * w_.expert;
        const double c = split_part / s.tp + experts / (dense() ? s.tp : s.ep);
        kvx_pd_choice r = base(s);
        r.latency = c / (g.lambda * g.flops) + comm(tokens, s) / (g.beta * g.link_bytes);
        r.vram = held_weights(s) + work(tokens, s.tp) + kv(tokens, s.tp);
        r.throughput = double(s.dp) * s.pp * b / r.latency;
        r.objective = r.throughput / double(s.dp * s.tp * s.pp);
        return r;
    }

    // Eq. 5 and Eq. 6 for one decode step; T_d in tokens/s
    kvx_pd_choice decode(const Strategy& s) const
    {
        const kvx_pd_gpu& g = p_.decode;
        const double b = s.batch;
        double touched;  // expert weights one GPU reads per layer and step
        if (dense())
            touched = w_.expert / s.tp;
        else
            touched = std::fmin(double(m_.experts) / s.ep, b * m_.active_experts) * w_.expert;
        const double weights = m_.weight_bytes *
                               (m_.layers * (w_.attn / s.tp + touched + w_.router + w_.norms) +
                                w_.table / s.tp);
        const double ctx_read = p_.prompt_tokens + p_.output_tokens / 2.0;
        const double ctx_held = double(p_.prompt_tokens) + p_.output_tokens;
        kvx_pd_choice r = base(s);
        r.latency = (weights + kv(b * ctx_read, s.tp)) / (g.alpha * g.hbm_bytes) +
                    comm(b, s) / (g.beta * g.link_bytes);
        r.vram = held_weights(s) + work(b, s.tp) + kv(b * ctx_held, s.tp);
        r.throughput = double(s.dp) * s.pp * b / r.latency;
        r.objective = r.throughput;
        return r;
    }

    bool dense() const { return m_.experts == 1; }

    // candidate strategies for a side, in the tie-break order
    std::vector<Strategy> candidates(int max_gpus) const
    {
        std::vector<Strategy> out;
        for (int gpus = 1; gpus <= max_gpus; ++gpus)
            for (int tp = 1; tp <= gpus; ++tp) {
                if (gpus % tp || m_.q_heads % tp) continue;
                if (m_.kv_heads % tp && tp % m_.kv_heads) continue;
                for (int pp = 1; pp <= gpus / tp; ++pp) {
                    if ((gpus / tp) % pp || m_.layers % pp) continue;
                    const int dp = gpus / (tp * pp);
                    for (int ep = 1; ep <= (dense() ? 1 : m_.experts); ++ep) {
                        if (!dense() && (m_.experts % ep || (dp * tp) % ep)) continue;
                        for (int b = 1; b <= p_.max_batch; b *= 2) out.push_back({dp, tp, pp, ep, b});
                    }
                }
            }
        return out;
    }

private:
    static kvx_pd_choice base(const Strategy& s)
    {
        kvx_pd_choice r;
        std::memset(&r, 0, sizeof r);
        r.dp = s.dp;
        r.tp = s.tp;
        r.pp = s.pp;
        r.ep = s.ep;
        r.batch = s.batch;
        r.gpus = s.dp * s.tp * s.pp;
        return r;
    }

    const kvx_pd_problem& p_;
    const kvx_pd_model& m_;
    Weights w_;
};

bool positive(double x) { return x > 0.0 && std::isfinite(x); }

kvx_status check_gpu(const kvx_pd_gpu& g, const char* side)
{
    if (!positive(g.flops) || !positive(g.hbm_bytes) || !positive(g.vram) ||
        !positive(g.link_bytes))
        return fail(KVX_EINVAL, "%s GPU: flops, hbm_bytes, vram and link_bytes must be > 0", side);
    if (!(g.lambda > 0 && g.lambda <= 1) || !(g.alpha > 0 && g.alpha <= 1) ||
        !(g.beta > 0 && g.beta <= 1))
        return fail(KVX_EINVAL, "%s GPU: discount factors must lie in (0, 1]", side);
    if (g.max_gpus < 1 || g.max_gpus > 4096)
        return fail(KVX_EINVAL, "%s GPU: max_gpus %d outside [1, 4096]", side, g.max_gpus);
    return KVX_OK;
}

kvx_status check(const kvx_pd_problem* p)
{
    if (!p) return fail(KVX_EINVAL, "NULL problem");
    const kvx_pd_model& m = p->model;
    if (m.layers < 1 || m.hidden < 1 || m.q_heads < 1 || m.kv_heads < 1 || m.head_dim < 1 ||
        m.ffn_dim < 1 || m.vocab < 1 || m.experts < 1 || m.active_experts < 1)
        return fail(KVX_EINVAL, "model dimensions must be >= 1");
    if (m.active_experts > m.experts)
        return fail(KVX_EINVAL, "active_experts %d above experts %d", m.active_experts, m.experts);
    if (!positive(m.weight_bytes) || !positive(m.kv_bytes) || !positive(m.act_bytes))
        return fail(KVX_EINVAL, "bytes per element must be > 0");
    kvx_status st = check_gpu(p->prefill, "prefill");
    if (st == KVX_OK) st = check_gpu(p->decode, "decode");
    if (st != KVX_OK) return st;
    if (p->prompt_tokens < 1 || p->output_tokens < 1)
        return fail(KVX_EINVAL, "prompt_tokens and output_tokens must be >= 1");
    if (!(p->qps >= 0) || !std::isfinite(p->qps) || !positive(p->ttft) || !positive(p->tpot))
        return fail(KVX_EINVAL, "qps must be >= 0, ttft and tpot > 0");
    if (p->max_batch < 1 || p->max_batch > (1 << 20))
        return fail(KVX_EINVAL, "max_batch %d outside [1, 2^20]", p->max_batch);
    return KVX_OK;
}

// The first candidate (in visiting order) whose objective is within kTie of
// the best feasible one; gpus = 0 when none is feasible.
kvx_pd_choice pick(const std::vector<kvx_pd_choice>& feasible)
{
    kvx_pd_choice none;
    std::memset(&none, 0, sizeof none);
    double top = 0.0;
    for (const kvx_pd_choice& c : feasible) top = std::fmax(top, c.objective);
    for (const kvx_pd_choice& c : feasible)
        if (c.objective >= top * (1.0 - kTie)) return c;
    return none;
}

}  // namespace

extern "C" {

kvx_status kvx_pd_evaluate(const kvx_pd_problem* p, int32_t side, int32_t dp, int32_t tp,
                           int32_t pp, int32_t ep, int32_t batch, kvx_pd_choice* out)
{
    kvx_status st = check(p);
    if (st != KVX_OK) return st;
    if (!out) return fail(KVX_EINVAL, "NULL out");
    if (side != KVX_PD_PREFILL && side != KVX_PD_DECODE)
        return fail(KVX_EINVAL, "side %d is neither KVX_PD_PREFILL nor KVX_PD_DECODE", side);
    if (dp < 1 || tp < 1 || pp < 1 || ep < 1 || batch < 1)
        return fail(KVX_EINVAL, "dp, tp, pp, ep and batch must be >= 1");
    const Evaluator ev(*p);
    const Strategy s{dp, tp, pp, ep, batch};
    *out = side == KVX_PD_PREFILL ? ev.prefill(s) : ev.decode(s);
    return KVX_OK;
}

kvx_status kvx_pd_search(const kvx_pd_problem* p, kvx_pd_solution* out)
{
    kvx_status st = check(p);
    if (st != KVX_OK) return st;
    if (!out) return fail(KVX_EINVAL, "NULL out");
    std::memset(out, 0, sizeof *out);
    const Evaluator ev(*p);

    std::vector<kvx_pd_choice> ok;
    const std::vector<Strategy> pc = ev.candidates(p->prefill.max_gpus);
    for (const Strategy& s : pc) {
        const kvx_pd_choice c = ev.prefill(s);
        if (c.latency <= p->ttft && c.vram <= p->prefill.vram) ok.push_back(c);  // Eq. 1 (c1), (c2)
    }
    out->candidates_prefill = int64_t(pc.size());
    out->feasible_prefill = int64_t(ok.size());
    out->prefill = pick(ok);

    ok.clear();
    const std::vector<Strategy> dc = ev.candidates(p->decode.max_gpus);
    for (const Strategy& s : dc) {
        const kvx_pd_choice c = ev.decode(s);
        if (c.latency <= p->tpot && c.vram <= p->decode.vram) ok.push_back(c);   // Eq. 4 (c1), (c2)
    }
    out->candidates_decode = int64_t(dc.size());
    out->feasible_decode = int64_t(ok.size());
    out->decode = pick(ok);

    if (out->prefill.gpus && out->decode.gpus) {
        out->prefill_instances = int64_t(std::ceil(p->qps / out->prefill.throughput));
        out->decode_instances =
            int64_t(std::ceil(p->qps * p->output_tokens / out->decode.throughput));
    }
    return KVX_OK;
}

}  // extern "C"
