"""Host-side checks of bench.py: the one-GPU guard, and the algorithmic work
it prices the roofline with, recounted here from the model's weight
matrices and a brute-force count of causal (query, key) pairs."""
import json
import os
import subprocess
import sys
import types

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2608_14635_amd import workloads as W  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert p.returncode == 2
    msg = json.loads(p.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def _matrices(s, last):
    """(out, in) of every projection a layer multiplies by; the last layer
    needs only the K and V projections."""
    H, d, nq, nkv, F = s.hidden, s.head_dim, s.num_q_heads, s.num_kv_heads, s.ffn_dim
    if last:
        return [(nkv * d, H), (nkv * d, H)]
    return [(nq * d, H), (nkv * d, H), (nkv * d, H), (H, nq * d), (F, H), (F, H), (H, F)]


def _causal_pairs(n):
    return sum(1 for q in range(n) for k in range(n) if k <= q)


def test_algorithmic_work_recounted():
    for s in (W.LLAMA8B, W.QWEN14B, W.TINY_F32):
        lens = np.array([1, 5, 64], dtype=np.int64)
        wl = types.SimpleNamespace(shape=s, lens=lens, total_tokens=int(lens.sum()))
        got = bench.algorithmic_work(wl)
        L = s.num_layers
        macs_tok = sum(o * i for l in range(L) for o, i in _matrices(s, l == L - 1))
        assert got["linear_flops"] == 2 * macs_tok * wl.total_tokens
        # attention of layers 0..L-2: per q head and causal pair, q.k and p.v
        # (d multiply-adds each)
        pairs = sum(_causal_pairs(int(n)) for n in lens)
        assert got["attn_flops"] == (L - 1) * s.num_q_heads * pairs * 2 * 2 * s.head_dim
        # bytes: every weight element once (norm gains included, the last
        # layer's K and V projections and the embedding rows gathered), and
        # the K and V rows written
        e = s.elem_bytes
        w_elems = sum(o * i for l in range(L) for o, i in _matrices(s, l == L - 1))
        gains = (L - 1) * 2 * s.hidden + s.hidden
        kv = wl.total_tokens * L * 2 * s.num_kv_heads * s.head_dim * e
        emb = wl.total_tokens * s.hidden * e
        assert got["kv_bytes"] == kv
        assert got["bytes"] == (w_elems + gains) * e + kv + emb


def test_linear_flops_per_token_of_the_8b_shape():
    # 13.54 GFLOP per token of projections for the 8B shape (the figure the
    # measurement plan states for the benchmark configuration)
    wl = types.SimpleNamespace(shape=W.LLAMA8B, lens=np.array([1]), total_tokens=1)
    assert abs(bench.algorithmic_work(wl)["linear_flops"] / 1e9 - 13.54) < 0.005


def test_decode_step_bytes_recounted():
    # one decode step: each weight matrix element and gain once, the LM head
    # and final gain once, one embedding row per request, and per layer the K
    # and V rows of every context key (brute-force over keys) plus the new rows
    for s in (W.LLAMA8B, W.QWEN3_8B, W.TINY_BF16):
        ctx = [1, 7, 300]
        e, L = s.elem_bytes, s.num_layers
        mats = sum(o * i for o, i in _matrices(s, False)) * L
        gains = 2 * s.hidden * L + s.hidden
        head = s.vocab * s.hidden
        emb = len(ctx) * s.hidden
        row = s.num_kv_heads * s.head_dim
        kv = sum(1 for n in ctx for _ in range(n)) * L * 2 * row
        new = len(ctx) * L * 2 * row
        assert bench.decode_step_bytes(s, ctx) == (mats + gains + head + emb + kv + new) * e


def test_decode_step_bytes_of_the_8b_benchmark():
    # the figure the benchmark prices the decode step with: 16 requests over
    # the 8B workload's 128,325 context tokens
    wl = W.config2()
    assert bench.decode_step_bytes(W.LLAMA8B, wl.lens) == 31831891968
