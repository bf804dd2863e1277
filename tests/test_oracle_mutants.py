"""Mutation check of the oracle's pins: each plausible mistake planted in a
copy of the oracle source (on the CPU) must make at least one pin fail."""
import os
import re
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(os.path.dirname(HERE), "oracle", "kvo.c")

# (name, exact text in kvo.c, replacement, which occurrence (0-based))
MUTANTS = [
    ("rope_sign", "hu[i] = to_work(a * c - b * s, dt);", "hu[i] = to_work(a * c + b * s, dt);", 0),
    ("rope_frequency", "pow(theta, -(double)(2 * i) / (double)d)", "pow(theta, -(double)(i) / (double)d)", 0),
    ("rope_pairing", "double a = hu[i], b = hu[i + half];", "double a = hu[2 * (i / 2)], b = hu[2 * (i / 2) + 1];", 0),
    ("dropped_norm_gain", "rnd(load(g, dt, j) * xr[j] * inv, dt)", "rnd(xr[j] * inv, dt)", 0),
    ("norm_sum_not_mean", "inv = 1.0 / sqrt(ss / (double)H + eps);", "inv = 1.0 / sqrt(ss + eps);", 0),
    ("gqa_modulo_grouping", "kvh = h / g,", "kvh = h % nkv,", 0),
    ("no_softmax_scale", "z[j] = s * scale;", "z[j] = s;", 0),
    ("no_softmax_denominator", "rnd(to_work(o / den, dt), dt)", "rnd(to_work(o, dt), dt)", 0),
    ("v_from_k_plane", "arena_off(m, ar, l, 1, slot_of(ar, table, j))", "arena_off(m, ar, l, 0, slot_of(ar, table, j))", 0),
    ("no_attention_residual", "x[idx] = to_work(x[idx] + a[idx], dt);", "x[idx] = to_work(a[idx], dt);", 0),
    ("no_ffn_residual", "x[idx] = to_work(x[idx] + a[idx], dt);", "x[idx] = to_work(a[idx], dt);", 1),
    ("sigmoid_not_silu", "gv / (1.0 + exp(-gv))", "1.0 / (1.0 + exp(-gv))", 0),
    ("dropped_up_projection", "rnd(to_work(silu * up[idx], dt), dt)", "rnd(to_work(silu, dt), dt)", 0),
    ("slot_offset", "table[p / ar->block_size] * ar->block_size + p % ar->block_size",
     "table[p / ar->block_size] * ar->block_size + (p + 1) % ar->block_size", 0),
    ("bf16_truncation", "u += 0x7fffu + ((u >> 16) & 1u);", "u += 0u;", 0),
    ("gate_up_swapped", "project(lw->w_gate, dt, F, H, a, cnt, gate);", "project(lw->w_up, dt, F, H, a, cnt, gate);", 0),
    ("k_not_rotated", "rope_row(k + r * nkv * d, (int)nkv, (int)d, p, m->rope_theta, dt);", ";", 0),
    ("position_plus_one", "double phi = (double)pos * inv_freq;", "double phi = (double)(pos + 1) * inv_freq;", 0),
    ("no_rounding_of_q", "q[r * nq * d + e] = rnd(q[r * nq * d + e], dt);", "q[r * nq * d + e] = q[r * nq * d + e];", 0),
    ("final_norm_gain_from_lm_head", "rmsnorm(hidden, final_norm, m->dtype, H, m->rms_eps, n, a);",
     "rmsnorm(hidden, lm_head, m->dtype, H, m->rms_eps, n, a);", 0),
    ("logits_of_unnormed_residual", "project(lm_head, m->dtype, V, H, a, n, z);",
     "project(lm_head, m->dtype, V, H, hidden, n, z);", 0),
    ("decode_step_position_plus_one", "layer_step(m, &layers[l], l, x, positions[r], 1, table, arena, kv_only, scratch);",
     "layer_step(m, &layers[l], l, x, positions[r] + 1, 1, table, arena, kv_only, scratch);", 0),
    ("decode_step_first_table", "const int32_t* table = block_tables + (int64_t)r * max_blocks;",
     "const int32_t* table = block_tables;", 2),
    ("q_norm_skipped", "head_rmsnorm(q, lw->q_norm, dt, cnt, nq, d, m->rms_eps);", ";", 0),
    ("q_norm_with_k_gain", "head_rmsnorm(q, lw->q_norm, dt, cnt, nq, d, m->rms_eps);",
     "head_rmsnorm(q, lw->k_norm, dt, cnt, nq, d, m->rms_eps);", 0),
    ("head_norm_sum_not_mean", "inv = 1.0 / sqrt(ss / (double)d + eps);", "inv = 1.0 / sqrt(ss + eps);", 0),
    ("bias_dropped", "to_work(dot_row(W, dt, i, K, A + r * K) + load(b, dt, i), dt)",
     "to_work(dot_row(W, dt, i, K, A + r * K), dt)", 0),
    ("v_bias_from_k", "project_bias(lw->wv, lw->bv, dt, nkv * d, H, a, cnt, v);",
     "project_bias(lw->wv, lw->bk, dt, nkv * d, H, a, cnt, v);", 0),
    ("rebuild_from_positions_from_zero", "layer_step(m, &layers[l], l, x, s, cnt, table, arena, kv_only, scratch);",
     "layer_step(m, &layers[l], l, x, 0, cnt, table, arena, kv_only, scratch);", 0),
    ("rebuild_from_token_offset", "    off += cnt;", "    off += lens[r];", 0),
    ("rebuild_from_first_tokens", "embed_rows(m, embed, tokens + off, cnt, x);", "embed_rows(m, embed, tokens, cnt, x);", 0),
    ("digest_key_multiplier", "u ^ (uint32_t)(i * 0x9E3779B9u)", "u ^ (uint32_t)(i * 0x9E3779B1u)", 0),
    ("digest_unkeyed", "u ^ (uint32_t)(i * 0x9E3779B9u)", "u", 0),
    ("digest_key_restarts_per_plane", "for (s = 0; s < nslots; ++s) {", "for (s = 0, i = 0; s < nslots; ++s) {", 0),
    ("digest_big_endian_words", "(uint32_t)p[4 * w] | (uint32_t)p[4 * w + 1] << 8 |",
     "(uint32_t)p[4 * w + 3] | (uint32_t)p[4 * w + 2] << 8 |", 0),
    ("digest_one_slot_too_many", "for (s = 0; s < nslots; ++s) {", "for (s = 0; s <= nslots && s < a->block_size; ++s) {", 0),
    ("digest_k_plane_only", "for (kv = 0; kv < 2; ++kv)\n      for (s = 0; s < nslots",
     "for (kv = 0; kv < 1; ++kv)\n      for (s = 0; s < nslots", 0),
    ("digest_linear_not_square", "sum += (uint64_t)x * (uint64_t)x;", "sum += (uint64_t)x;", 0),
    ("verify_counts_all_matches", "if (leading && dg == committed[e]) intact[r] = j + 1;",
     "if (dg == committed[e]) intact[r] += 1;", 0),
    ("verify_tail_block_full", "const int32_t n = lens[r] - j * B < B ? lens[r] - j * B : B;",
     "const int32_t n = B;", 0),
    # rounding sites of the Qwen variants
    ("qk_norm_output_rounded_before_rope", "for (e = 0; e < d; ++e) hu[e] = to_work(load(g, dt, e) * hu[e] * inv, dt);",
     "for (e = 0; e < d; ++e) hu[e] = rnd(load(g, dt, e) * hu[e] * inv, dt);", 0),
    ("bias_added_after_rounding", "to_work(dot_row(W, dt, i, K, A + r * K) + load(b, dt, i), dt)",
     "to_work(to_work(dot_row(W, dt, i, K, A + r * K), dt) + load(b, dt, i), dt)", 0),
    ("qk_norm_gain_after_rope", [
        ("for (e = 0; e < d; ++e) hu[e] = to_work(load(g, dt, e) * hu[e] * inv, dt);",
         "for (e = 0; e < d; ++e) hu[e] = to_work(hu[e] * inv, dt);", 0),
        ("rope_row(k + r * nkv * d, (int)nkv, (int)d, p, m->rope_theta, dt);",
         "rope_row(k + r * nkv * d, (int)nkv, (int)d, p, m->rope_theta, dt);\n"
         "    if (m->qk_norm) {\n"
         "      for (e = 0; e < nq * d; ++e) q[r * nq * d + e] = to_work(load(lw->q_norm, dt, e % d) * q[r * nq * d + e], dt);\n"
         "      for (e = 0; e < nkv * d; ++e) k[r * nkv * d + e] = to_work(load(lw->k_norm, dt, e % d) * k[r * nkv * d + e], dt);\n"
         "    }", 0)], None, None),
    ("round_p_ignored", "z[j] = rnd(to_work(exp2(z[j] * M_LOG2E - c), dt), dt);", "z[j] = exp2(z[j] * M_LOG2E - c);", 0),
    ("round_p_denominator_unrounded",
     "        z[j] = rnd(to_work(exp2(z[j] * M_LOG2E - c), dt), dt);\n        den += z[j];",
     "        den += exp2(z[j] * M_LOG2E - c);\n        z[j] = rnd(to_work(exp2(z[j] * M_LOG2E - c), dt), dt);", 0),
    ("round_p_anchored_at_the_exact_max", "const double c = ceil(zmax * M_LOG2E);",
     "const double c = zmax * M_LOG2E;", 0),
    # causal mask, norm, rotation, gather and projection mix-ups
    ("causal_mask_one_key_ahead", "kvh = h / g, p = p0 + r;",
     "kvh = h / g, p = (r + 1 < cnt) ? p0 + r + 1 : p0 + r;", 0),
    ("causal_mask_without_the_diagonal", "kvh = h / g, p = p0 + r;", "kvh = h / g, p = p0 + r - 1;", 0),
    ("norm_eps_outside_the_root", "inv = 1.0 / sqrt(ss / (double)H + eps);",
     "inv = 1.0 / (sqrt(ss / (double)H) + eps);", 0),
    ("ffn_norm_with_attention_gain", "rmsnorm(x, lw->ffn_norm, dt, H, m->rms_eps, cnt, a);",
     "rmsnorm(x, lw->attn_norm, dt, H, m->rms_eps, cnt, a);", 0),
    ("q_not_rotated", "rope_row(q + r * nq * d, (int)nq, (int)d, p, m->rope_theta, dt);", ";", 0),
    ("v_rotated", "rope_row(k + r * nkv * d, (int)nkv, (int)d, p, m->rope_theta, dt);",
     "rope_row(k + r * nkv * d, (int)nkv, (int)d, p, m->rope_theta, dt);\n"
     "    rope_row(v + r * nkv * d, (int)nkv, (int)d, p, m->rope_theta, dt);", 0),
    ("embedding_row_off_by_one", "load(embed, m->dtype, (int64_t)tok[r] * H + j)",
     "load(embed, m->dtype, (((int64_t)tok[r] + 1) % m->vocab) * H + j)", 0),
    ("wo_transposed", "project(lw->wo, dt, H, nq * d, u, cnt, a);",
     "if (H == nq * d) {\n"
     "    for (idx = 0; idx < cnt * H; ++idx) {\n"
     "      const int64_t rr = idx / H, ii = idx % H;\n"
     "      double s = 0.0;\n"
     "      int64_t kk;\n"
     "      for (kk = 0; kk < H; ++kk) s += load(lw->wo, dt, kk * H + ii) * u[rr * H + kk];\n"
     "      a[idx] = to_work(s, dt);\n"
     "    }\n"
     "  } else project(lw->wo, dt, H, nq * d, u, cnt, a);", 0),
    ("down_reads_up_not_swiglu", "project(lw->w_down, dt, H, F, gate, cnt, a);",
     "project(lw->w_down, dt, H, F, up, cnt, a);", 0),
    ("k_written_to_layer_zero", "store(ar->base, dt, arena_off(m, ar, l, 0, slot) + e",
     "store(ar->base, dt, arena_off(m, ar, 0, 0, slot) + e", 0),
    # RoPE precision: the angle in fp64, cos and sin rounded once to the working precision
    ("rope_cos_sin_unrounded", "if (dt != KVO_F64) { c = (double)(float)c; s = (double)(float)s; }", ";", 0),
    ("rope_angle_in_fp32", "double phi = (double)pos * inv_freq;",
     "double phi = (double)((float)pos * (float)inv_freq);", 0),
    # the layer-0 K/V helper that samples expected rows at full size
    ("layer0_helper_without_eps", "inv = 1.0 / sqrt(ss / (double)H + m->rms_eps);",
     "inv = 1.0 / sqrt(ss / (double)H);", 0),
    ("layer0_helper_gain_dropped", "a[j] = rnd(load(layer0->attn_norm, dt, j) * x[j] * inv, dt);",
     "a[j] = rnd(x[j] * inv, dt);", 0),
    ("layer0_helper_position_zero",
     "rope_row(k, m->num_kv_heads, m->head_dim, positions[i], m->rope_theta, dt);",
     "rope_row(k, m->num_kv_heads, m->head_dim, 0, m->rope_theta, dt);", 0),
]


def _patch(text, old, new, occ):
    if isinstance(old, list):  # several sites: a list of (old, new, occurrence)
        for o, n, k in old:
            text = _patch(text, o, n, k)
        return text
    idx = -1
    for _ in range(occ + 1):
        idx = text.find(old, idx + 1)
        assert idx >= 0, f"anchor not found: {old}"
    return text[:idx] + new + text[idx + len(old):]


def _run_mutant(tmp, name, old, new, occ):
    d = os.path.join(tmp, name)
    os.makedirs(d, exist_ok=True)
    src = open(SRC).read()
    shutil.copy(os.path.join(os.path.dirname(SRC), "kvo.h"), d)
    with open(os.path.join(d, "kvo.c"), "w") as f:
        f.write(_patch(src, old, new, occ))
    lib = oracle.build(os.path.join(d, "kvo.c"), os.path.join(d, "libkvo.so"), ["-I", d])
    env = dict(os.environ, OMP_NUM_THREADS="2")
    p = subprocess.run([sys.executable, os.path.join(HERE, "oracle_pins.py"), lib],
                       capture_output=True, text=True, timeout=600, env=env)
    m = re.search(r"(\d+) of (\d+) pins failed", p.stdout)
    caught = (int(m.group(1)) if m else 1) if p.returncode == 0 or m is None else int(m.group(1))
    return name, caught, p.stdout[-2000:] + p.stderr[-500:]


def test_every_anchor_exists():
    src = open(SRC).read()
    for name, old, new, occ in MUTANTS:
        _patch(src, old, new, occ)


def test_mutants_are_caught(tmp_path):
    with ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(lambda m: _run_mutant(str(tmp_path), *m), MUTANTS))
    missed = [(n, out) for n, caught, out in results if caught == 0]
    assert not missed, "mutants not caught by any pin: " + ", ".join(n for n, _ in missed)
