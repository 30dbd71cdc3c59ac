"""Mutation test of the oracle's pins.

Each mutant plants one plausible mistake in a copy of the oracle package (a
dropped term, a wrong sign, index or constant, a transposed operand, a wrong
rounding or saturation rule, a mistaken reading of the planner's cost
model), builds it, and runs the oracle's pin tests (tests/test_oracle_*.py)
against the copy in a child pytest (-x).  Every mutant must make a pin fail;
the unmodified copy must pass.  Children run in parallel, each given the pin
file expected to catch its mutant first, so the run stays short.
"""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle")
PINS = sorted(p for p in glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py"))
              if os.path.basename(p) != os.path.basename(__file__))
C = "kvx_oracle.c"
PD = "pd.py"

# (name, file, text to replace, replacement, pin file to run first)
MUTANTS = [
    # decoding of the formats
    ("e4m3_nan_whole_top_binade", C,
     "if (e == emax_field && m == ((1u << f.man_bits) - 1u))", "if (e == emax_field)", "casts"),
    ("subnormal_exponent_off_by_one", C,
     "v = ldexp((double)m, 1 - f.bias - f.man_bits);", "v = ldexp((double)m, -f.bias - f.man_bits);",
     "casts"),
    ("bf16_bias", C, "f.man_bits = 7;  f.bias = 127;", "f.man_bits = 7;  f.bias = 126;", "casts"),
    # rounding to a grid
    ("ties_away_from_zero", C, "double r = nearbyint(n);", "double r = floor(n + 0.5);", "casts"),
    ("truncation", C, "double r = nearbyint(n);", "double r = floor(n);", "casts"),
    ("no_subnormal_spacing", C, "if (E < emin) E = emin;", "(void)emin;", "casts"),
    ("subnormal_encoding", C, "double frac = ldexp(mag, -(emin - f.man_bits));",
     "double frac = ldexp(mag, -(emin - f.man_bits) - 1);", "casts"),
    # fp16 <-> bf16
    ("fp16_nan_payload_shift", C, "((h & 0x03FFu) >> 3)", "((h & 0x03FFu) >> 2)", "casts"),
    ("fp16_nan_no_quiet_bit", C, "0x7F80u | 0x0040u |", "0x7F80u |", "casts"),
    ("fp16_to_bf16_sign_dropped", C, "return (uint16_t)encode(ORC_BF16, sign, m);",
     "return (uint16_t)encode(ORC_BF16, 0, m);", "casts"),
    ("bf16_to_fp16_overflow_threshold", C, "    if (m > 65504.0)\n", "    if (m > 61440.0)\n",
     "casts"),
    ("bf16_nan_payload_shift", C, "((b & 0x7Fu) << 3)", "((b & 0x7Fu) << 2)", "casts"),
    # 8-bit casts
    ("e4m3_overflow_to_nan", C,
     "if (a >= 448.0) return (uint8_t)encode(ORC_E4M3FN, sign, 448.0);",
     "if (a >= 448.0) return (uint8_t)((sign << 7) | 0x7Fu);", "casts"),
    ("e4m3_min_exponent", C, "rne_to_grid(a, 4, -6)", "rne_to_grid(a, 4, -7)", "casts"),
    ("e4m3_one_bit_short", C, "rne_to_grid(a, 4, -6)", "rne_to_grid(a, 3, -6)", "casts"),
    ("e5m2_overflow_to_inf", C,
     "if (a >= 57344.0) return (uint8_t)encode(ORC_E5M2, sign, 57344.0);",
     "if (a >= 57344.0) return (uint8_t)((sign << 7) | 0x7Cu);", "e5m2"),
    ("e5m2_min_exponent", C, "rne_to_grid(a, 3, -14)", "rne_to_grid(a, 3, -15)", "e5m2"),
    ("e5m2_one_bit_extra", C, "rne_to_grid(a, 3, -14)", "rne_to_grid(a, 4, -14)", "e5m2"),
    ("e5m2_nan_code", C,
     "if (isnan(v)) return (uint8_t)((sign << 7) | 0x7Fu);\n    double a = fabs((double)v);\n"
     "    if (a >= 57344.0)",
     "if (isnan(v)) return (uint8_t)((sign << 7) | 0x7Eu);\n    double a = fabs((double)v);\n"
     "    if (a >= 57344.0)", "e5m2"),
    ("scale_over_224", C, "return amax / fmax;", "return amax / (fmax * 0.5f);", "casts"),
    ("scale_signed_maximum", C, "float a = fabsf(x[d]);", "float a = x[d];", "casts"),
    ("zero_row_sign_dropped", C, "o[d] = (uint8_t)(sign << 7);", "o[d] = 0;", "casts"),
    ("nan_element_code", C,
     "if (isnan(x[d]))\n            o[d] = (uint8_t)((sign << 7) | 0x7Fu);",
     "if (isnan(x[d]))\n            o[d] = (uint8_t)((sign << 7) | 0x7Eu);", "casts"),
    ("quotient_by_reciprocal", C, "float v = x[d] / sc;", "float v = x[d] * (1.0f / sc);",
     "casts"),
    ("invalid_quotient_unsigned", C, "o[d] = isnan(v) ? (uint8_t)((sign << 7) | 0x7Fu)",
     "o[d] = isnan(v) ? (uint8_t)0x7Fu", "casts"),
    ("e5m2_scale_divisor", C, "e5 ? 57344.0f : 448.0f", "e5 ? 448.0f : 448.0f", "e5m2"),
    ("e5m2_rows_cast_as_e4m3", C, ": (e5 ? orc_f32_to_e5m2(v) : orc_f32_to_e4m3fn(v));",
     ": orc_f32_to_e4m3fn(v);", "e5m2"),
    # dequantisation
    ("dequant_codes_as_e4m3", C, "float x = (float)orc_decode(code_fmt, q[d]);",
     "float x = (float)orc_decode(ORC_E4M3FN, q[d]);", "e5m2"),
    ("dequant_nan_sign", C, "out[d] = f32_to_16(cache_fmt, isnan(x) ? NAN : v, sign);",
     "out[d] = f32_to_16(cache_fmt, isnan(x) ? NAN : v, 0);", "dequant"),
    ("dequant_scale_dropped", C, "float v = x * s;", "float v = x;", "dequant"),
    ("fp16_overflow_threshold", C, "double maxf = bf ? ldexp(255.0, 120) : 65504.0;",
     "double maxf = bf ? ldexp(255.0, 120) : 65472.0;", "dequant"),
    # head map (parallel-strategy alignment)
    ("head_modulo_all_heads", C, "*head = g % Hs;", "*head = g % H;", "layout"),
    ("shard_without_rank_offset", C, "*shard = g / Hs;", "*shard = i / Hs;", "layout"),
    ("replica_shard_not_scaled", C, "*shard = g * (p->src_tp / H);", "*shard = g;", "layout"),
    ("replicated_head_modulo", C, "p->dst_rank / (p->dst_tp / H)", "p->dst_rank % H", "layout"),
    ("replication_rejected", C,
     "if (p->heads % p->dst_tp != 0 && p->dst_tp % p->heads != 0) return -1;",
     "if (p->heads % p->dst_tp != 0) return -1;", "layout"),
    ("replicated_rank_two_heads", C,
     "return p->dst_tp <= p->heads ? p->heads / p->dst_tp : 1;",
     "return p->dst_tp <= p->heads ? p->heads / p->dst_tp : 2;", "layout"),
    # index maps (VRAM-management alignment)
    ("token_major_read_head_major", C, "return base + ((plane * T + t) * Hs + h) * D + d;",
     "return base + ((plane * Hs + h) * T + t) * D + d;", "layout"),
    ("head_major_read_token_major", C, "return base + ((plane * Hs + h) * T + t) * D + d;",
     "return base + ((plane * T + t) * Hs + h) * D + d;", "layout"),
    ("kv_swapped", C,
     "int64_t plane = ((int64_t)p->src_layer_offset + l) * 2 + kv; /* in the source's layers */",
     "int64_t plane = ((int64_t)p->src_layer_offset + l) * 2 + (1 - kv);", "layout"),
    ("request_stride_converted_layers", C,
     "base += (int64_t)orc_src_layers(p) * 2 * p->seq_lens[q] * Hs * p->head_dim;",
     "base += (int64_t)p->layers * 2 * p->seq_lens[q] * Hs * p->head_dim;", "layers"),
    ("slot_reversed", C,
     "return (((plane * p->num_blocks + block) * p->block_size + slot) * Hd + i) * p->head_dim + d;",
     "return (((plane * p->num_blocks + block) * p->block_size + (p->block_size - 1 - slot)) * Hd"
     " + i) * p->head_dim + d;", "layout"),
    ("cache_layer_offset_dropped", C,
     "int64_t plane = ((int64_t)p->dst_layer_offset + l) * 2 + kv; /* in the cache's layers */",
     "int64_t plane = ((int64_t)l) * 2 + kv;", "layers"),
    ("scale_layer_offset_dropped", C,
     "int64_t plane = ((int64_t)p->dst_layer_offset + l) * 2 + kv;\n    return ((plane",
     "int64_t plane = ((int64_t)l) * 2 + kv;\n    return ((plane", "layers"),
    ("source_layer_offset_dropped", C,
     "int64_t plane = ((int64_t)p->src_layer_offset + l) * 2 + kv; /* in the source's layers */",
     "int64_t plane = ((int64_t)l) * 2 + kv;", "layers"),
    ("no_wire_alignment", C,
     "static int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }",
     "static int64_t align256(int64_t x) { return x; }", "layout"),
    ("wire_rows_16_bit", C, "off += rows * p->head_dim * esz;", "off += rows * p->head_dim * 2;",
     "layout"),
    # paged sources
    ("source_page_from_modulo", C,
     "p->src_block_table[(int64_t)r * p->src_bt_stride + t / p->src_block_size]",
     "p->src_block_table[(int64_t)r * p->src_bt_stride + t % p->src_block_size]", "paged"),
    ("source_slot_from_division", C, "int64_t slot = t % p->src_block_size;",
     "int64_t slot = t / p->src_block_size;", "paged"),
    ("source_table_stride", C,
     "p->src_block_table[(int64_t)r * p->src_bt_stride + t / p->src_block_size]",
     "p->src_block_table[(int64_t)r * p->src_block_size + t / p->src_block_size]", "paged"),
    ("source_plane_term_dropped", C,
     "return (((plane * p->src_num_blocks + blk) * p->src_block_size + slot) * Hs + h) * D + d;",
     "return (((blk) * p->src_block_size + slot) * Hs + h) * D + d;", "paged"),
    ("source_pool_uses_decode_count", C, "(plane * p->src_num_blocks + blk)",
     "(plane * p->num_blocks + blk)", "paged"),
    # the P:D planner (Eq. 1-6 under readings R27-R31)
    ("pd_output_projection_kv_heads", PD, "o = m.q_heads * m.head_dim * m.hidden",
     "o = m.kv_heads * m.head_dim * m.hidden", "pd"),
    ("pd_two_ffn_matrices", PD, "return 3 * m.hidden * m.ffn_dim", "return 2 * m.hidden * m.ffn_dim",
     "pd"),
    ("pd_tied_embedding", PD, "return m.layers * per_layer + m.hidden + 2 * m.vocab * m.hidden",
     "return m.layers * per_layer + m.hidden + 1 * m.vocab * m.hidden", "pd"),
    ("pd_ring_factor", PD, "(2 * (tp - 1) / tp)", "(2 * (tp - 1))", "pd"),
    ("pd_prefill_throughput_without_pp", PD, "t_p = dp * pp * b / l_p", "t_p = dp * b / l_p", "pd"),
    ("pd_kv_one_tensor", PD,
     "return tokens * 2 * m.layers * kv_heads_per_gpu(m, tp) * m.head_dim * m.kv_bytes",
     "return tokens * 1 * m.layers * kv_heads_per_gpu(m, tp) * m.head_dim * m.kv_bytes", "pd"),
    ("pd_objective_ignores_pp", PD, "obj = t_p / (dp * tp * pp)", "obj = t_p / (dp * tp)", "pd"),
    ("pd_tie_order", PD,
     "out.sort(key=lambda c: (c[0] * c[1] * c[2], c[1], c[2], c[0], c[3], c[4]))",
     "out.sort(key=lambda c: (c[1], c[2], c[0], c[3], c[4]))", "pd"),
    ("pd_decode_full_context", PD, "ctx_read = p.prompt_tokens + p.output_tokens / 2",
     "ctx_read = p.prompt_tokens + p.output_tokens", "pd"),
    ("pd_decode_instances_per_request", PD,
     "sol.decode_instances = math.ceil(p.qps * p.output_tokens / sol.decode.throughput)",
     "sol.decode_instances = math.ceil(p.qps / sol.decode.throughput)", "pd"),
]


def _copy(tmp, name, mutant):
    d = os.path.join(tmp, name)
    dst = os.path.join(d, "oracle")
    shutil.copytree(ORACLE, dst, ignore=shutil.ignore_patterns("*.so", "__pycache__"))
    if mutant is not None:
        _, fname, old, new, _ = mutant
        path = os.path.join(dst, fname)
        text = open(path).read()
        assert text.count(old) == 1, f"{name}: the text to replace occurs {text.count(old)} times"
        with open(path, "w") as f:
            f.write(text.replace(old, new))
    subprocess.run(["gcc", "-std=c99", "-O2", "-fPIC", "-shared", "-ffp-contract=off",
                    "-fno-fast-math", "-o", os.path.join(dst, "liboracle.so"),
                    os.path.join(dst, C), "-lm"], check=True, capture_output=True)
    return d


def _pins(first):
    lead = [p for p in PINS if os.path.basename(p) == f"test_oracle_{first}.py"]
    return lead + [p for p in PINS if p not in lead]


def _run(tmp, name, mutant):
    d = _copy(tmp, name, mutant)
    env = dict(os.environ, KVX_ORACLE_COPY=d, OMP_NUM_THREADS="1")
    first = mutant[4] if mutant else "casts"
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu", *_pins(first)], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=900)
    return name, r.returncode, (r.stdout + r.stderr)[-600:]


def test_mutants_are_unique_and_named():
    names = [m[0] for m in MUTANTS]
    assert len(set(names)) == len(names)
    assert all(m[1] in (C, PD) and m[2] != m[3] for m in MUTANTS)
    assert len(MUTANTS) >= 40


@pytest.mark.timeout(1800)
def test_every_mutant_fails_a_pin(tmp_path):
    assert os.environ.get("KVX_ORACLE_COPY") is None, "the harness must not run inside a child"
    assert all("mutants" not in os.path.basename(p) for p in PINS)
    workers = max(1, min(8, os.cpu_count() or 1))
    jobs = [("unmodified", None)] + [(m[0], m) for m in MUTANTS]
    with ThreadPoolExecutor(workers) as ex:
        results = list(ex.map(lambda j: _run(str(tmp_path), *j), jobs))
    base = results[0]
    assert base[1] == 0, f"the unmodified copy fails its pins:\n{base[2]}"
    survivors = [(n, rc, out) for n, rc, out in results[1:] if rc != 1]
    assert not survivors, "mutants not caught by a failing pin:\n" + "\n".join(
        f"{n} (exit {rc}): {out[-300:]}" for n, rc, out in survivors)
