"""Pins of the CPU oracle against facts fixed outside the oracle itself.

Each pin is a function of an `oracle.Oracle` instance that raises
AssertionError when the oracle violates it.  They are run on the real
oracle by test_oracle_pins.py and on deliberately broken copies of the oracle
source by test_oracle_mutants.py (every planted mistake must trip at least
one pin).  Running this file directly with a library path runs every pin on
that library and prints the names of the pins that failed.

What pins what:
  * textbook PyTorch fp64 forward (library rms_norm / linear / causal GQA
    scaled_dot_product_attention / silu / rotate-half RoPE): whole forward
  * closed forms: Wq = 0 gives uniform causal attention (mean of V rows);
    position 0 leaves K unrotated; a two-layer worked example whose every
    K, V and final residual value is derived by hand (golden/worked_example.txt)
  * invariants: prefill == token-by-token decode through the arena; rotary
    pair norms and the rotation angle; relative-position dot products;
    GQA == MHA with duplicated KV heads; causality; batch independence;
    idempotence over garbage; exact placement and untouched bits
  * library routine: fp32 -> bf16 rounding against torch's conversion
  * rebuild from a retained prefix: two-phase rebuild == full rebuild
    (causality), start 0 == rebuild, start = length is a no-op, the suffix
    reads the prefix K/V the arena holds, shared-prefix block copies
  * block commit digests: closed forms on arenas built to cancel the word
    keys (N c^2, one changed word), bit flips always detected, bytes outside
    the covered slots ignored, leading-intact counts with planted corruption
"""
from __future__ import annotations

import ast
import dataclasses
import math
import operator
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2608_14635_amd import workloads as W  # noqa: E402

F32, BF16, F64 = W.F32, W.BF16, W.F64

# A GQA variant of the tiny fp32 decoder (group 2) so that pins see grouping.
TINY_GQA = dataclasses.replace(W.TINY_F32, num_q_heads=4, num_kv_heads=2, ffn_dim=344)
TINY_BF16_2L = W.TINY_BF16.with_layers(2)


# ----------------------------------------------------------------------
# helpers
# ----------------------------------------------------------------------
def as_float(a: np.ndarray, dt: int) -> np.ndarray:
    if dt == BF16:
        return W.bf16_bits_to_f32(a).astype(np.float64)
    if a.dtype == np.uint32:
        return a.view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def weights_in(w: dict, src_dt: int, dst_dt: int) -> dict:
    """Re-express materialized weights exactly in another container dtype."""
    if src_dt == dst_dt:
        return w
    f = W.weights_as_f32(w, src_dt)
    if dst_dt == F64:
        cv = lambda a: a.astype(np.float64)  # noqa: E731
    elif dst_dt == F32:
        cv = lambda a: a.astype(np.float32)  # noqa: E731
    else:
        cv = W.f32_to_bf16_bits
    return {"embed": cv(f["embed"]), "layers": [{k: cv(v) for k, v in lw.items()} for lw in f["layers"]]}


def run(o, shape, w, wl, dt=None, mode="prefill", arena=None, final_hidden=False, round_p=False):
    dt = shape.dtype if dt is None else dt
    a = W.host_arena(wl, dt) if arena is None else arena
    fh = o.rebuild(shape, w, wl.tokens, wl.lens, wl.block_tables, a, wl.block_size,
                   wl.num_blocks, mode=mode, dtype=dt, final_hidden=final_hidden, round_p=round_p)
    return (a, fh) if final_hidden else a


def view(wl, shape, a):
    return a.reshape(shape.num_layers, 2, wl.num_blocks, wl.block_size, shape.num_kv_heads,
                     shape.head_dim)


def gather(wl, shape, a, r):
    """K, V of request r as [L, n, nkv, d] read through its block table."""
    v = view(wl, shape, a)
    n = int(wl.lens[r])
    p = np.arange(n)
    blocks = wl.block_tables[r, p // wl.block_size]
    slots = p % wl.block_size
    return v[:, 0, blocks, slots], v[:, 1, blocks, slots]


def written_mask(wl, shape):
    m = np.zeros((shape.num_layers, 2, wl.num_blocks, wl.block_size), bool)
    for r in range(wl.num_requests):
        p = np.arange(int(wl.lens[r]))
        m[:, :, wl.block_tables[r, p // wl.block_size], p % wl.block_size] = True
    return m


def normwise(g, o):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    den = np.max(np.abs(o))
    err = float(np.max(np.abs(g - o)) / den) if den > 0 else float(np.max(np.abs(g - o)))
    return err if np.isfinite(err) else np.inf  # NaN would vanish in a max() fold


# ----------------------------------------------------------------------
# pins
# ----------------------------------------------------------------------
def pin_decode_equals_prefill_f32(o):
    wl = W.config1()
    w = W.host_weights(wl.shape, seed=3)
    a = run(o, wl.shape, w, wl)
    b = run(o, wl.shape, w, wl, mode="decode")
    assert np.array_equal(a, b), "prefill and decode arenas differ (fp32)"


def pin_decode_equals_prefill_bf16(o):
    shape = TINY_BF16_2L
    wl = W.small_workload(shape, [1, 17, 40], seed=5)
    w = W.host_weights(shape, seed=4)
    a = run(o, shape, w, wl)
    b = run(o, shape, w, wl, mode="decode")
    assert np.array_equal(a, b), "prefill and decode arenas differ (bf16)"


def pin_placement_and_untouched(o):
    shape = W.TINY_F32
    wl = W.small_workload(shape, [5, 16, 33, 0, 47], seed=9, other_live_frac=0.3)
    w = W.host_weights(shape, seed=5)
    before = W.host_arena(wl)
    after = run(o, shape, w, wl, arena=before.copy())
    vb = view(wl, shape, before).reshape(shape.num_layers, 2, wl.num_blocks, wl.block_size, -1)
    va = view(wl, shape, after).reshape(vb.shape)
    m = written_mask(wl, shape)
    changed = np.any(va != vb, axis=-1)
    assert np.array_equal(changed, m), "written slots differ from the listed slots"
    assert np.array_equal(va[~m], vb[~m]), "an unlisted slot was modified"
    # every written value is finite (no sentinel leaked into a result)
    assert np.all(np.isfinite(va[m].view(np.float32))), "non-finite value written"


def pin_table_permutation(o):
    shape = W.TINY_F32
    lens = [20, 33, 7]
    wl1 = W.small_workload(shape, lens, seed=21, other_live_frac=0.0)
    wl2 = W.small_workload(shape, lens, seed=22, other_live_frac=0.4)
    wl2.tokens = wl1.tokens.copy()
    assert not np.array_equal(wl1.block_tables, wl2.block_tables)
    w = W.host_weights(shape, seed=6)
    a1 = run(o, shape, w, wl1)
    a2 = run(o, shape, w, wl2)
    for r in range(len(lens)):
        k1, v1 = gather(wl1, shape, a1, r)
        k2, v2 = gather(wl2, shape, a2, r)
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2), "placement depends on the table"


def pin_causality(o):
    shape = W.TINY_F32
    wl = W.small_workload(shape, [50], seed=31, other_live_frac=0.0)
    w = W.host_weights(shape, seed=7)
    a = run(o, shape, w, wl)
    j = 23
    wl2 = dataclasses.replace(wl, tokens=wl.tokens.copy())
    wl2.tokens[j] = (wl2.tokens[j] + 1) % shape.vocab
    b = run(o, shape, w, wl2)
    ka, va = gather(wl, shape, a, 0)
    kb, vb = gather(wl2, shape, b, 0)
    assert np.array_equal(ka[:, :j], kb[:, :j]) and np.array_equal(va[:, :j], vb[:, :j]), \
        "a later token changed earlier K/V"
    assert not np.array_equal(ka[:, j:], kb[:, j:]), "the changed token had no effect"
    assert not np.array_equal(ka[1, j + 1:], kb[1, j + 1:]), "layer-1 K after j ignored token j"


def pin_uniform_attention_closed_form(o):
    """Wq = 0 makes every score 0, so attention is the plain mean of the
    visible V rows; with Wo = I and a zero down projection the residual after
    the layer is x0 + mean_{j<=p} V_{kv(h)}."""
    shape = dataclasses.replace(TINY_GQA, num_layers=1, dtype=F64)
    H, d, nq, nkv = shape.hidden, shape.head_dim, shape.num_q_heads, shape.num_kv_heads
    assert nq * d == H
    wl = W.small_workload(shape, [1, 9, 30], seed=41, other_live_frac=0.0)
    w = weights_in(W.host_weights(dataclasses.replace(shape, dtype=F32), seed=8), F32, F64)
    lw = w["layers"][0]
    lw["wq"] = np.zeros_like(lw["wq"])
    lw["wo"] = np.eye(H, dtype=np.float64)
    lw["w_down"] = np.zeros_like(lw["w_down"])
    a, fh = run(o, shape, w, wl, final_hidden=True)
    off = wl.request_offsets()
    g = nq // nkv
    for r in range(wl.num_requests):
        n = int(wl.lens[r])
        _, V = gather(wl, shape, a, r)
        V = V[0]  # [n, nkv, d]
        x0 = w["embed"][wl.tokens[off[r]:off[r + 1]]]
        u = fh[off[r]:off[r + 1]] - x0
        mean = np.cumsum(V, axis=0) / np.arange(1, n + 1)[:, None, None]
        expect = np.concatenate([mean[:, h // g] for h in range(nq)], axis=1)
        assert np.max(np.abs(u - expect)) <= 1e-12 * max(1.0, np.max(np.abs(expect))), \
            "uniform-attention closed form violated"


_EXPR_FUNCS = {"cos": math.cos, "sin": math.sin, "exp": math.exp, "sqrt": math.sqrt}
_EXPR_OPS = {ast.Add: operator.add, ast.Sub: operator.sub, ast.Mult: operator.mul,
             ast.Div: operator.truediv, ast.Pow: operator.pow}


def _eval_expr(text: str, env: dict) -> float:
    """Value of a fixture expression: numbers, names bound by earlier `let`
    lines, + - * / **, unary minus and cos/sin/exp/sqrt of one argument."""
    def ev(n):
        if isinstance(n, ast.Constant) and isinstance(n.value, (int, float)):
            return float(n.value)
        if isinstance(n, ast.Name):
            return env[n.id]
        if isinstance(n, ast.UnaryOp) and isinstance(n.op, ast.USub):
            return -ev(n.operand)
        if isinstance(n, ast.BinOp) and type(n.op) in _EXPR_OPS:
            return _EXPR_OPS[type(n.op)](ev(n.left), ev(n.right))
        if (isinstance(n, ast.Call) and isinstance(n.func, ast.Name)
                and n.func.id in _EXPR_FUNCS and len(n.args) == 1 and not n.keywords):
            return _EXPR_FUNCS[n.func.id](ev(n.args[0]))
        raise ValueError(f"unsupported expression: {text}")
    return ev(ast.parse(text.strip(), mode="eval").body)


def _worked_example(path: str):
    """Model, weights, requests and hand-derived expectations of the worked
    example fixture (its header states the format)."""
    kw, arena, reqs, embed, weights, env, expect = {}, {}, [], {}, {}, {}, []
    for raw in open(path):
        line = raw.split("#", 1)[0].strip()
        if not line:
            continue
        word, _, rest = line.partition(" ")
        if word in ("shape", "arena"):
            for item in rest.split():
                k, v = item.split("=")
                (kw if word == "shape" else arena)[k] = float(v)
        elif word == "request":
            f = dict(item.split("=") for item in rest.split())
            reqs.append(([int(t) for t in f["tokens"].split(",")],
                         [int(b) for b in f["blocks"].split(",")]))
        elif word == "let":
            name, _, expr = rest.partition("=")
            env[name.strip()] = _eval_expr(expr, env)
        else:
            head, _, values = line.partition(":")
            head = head.split()
            if word == "embed":
                embed[int(head[1])] = [float(x) for x in values.split()]
            elif word == "weight":
                rows = [[float(x) for x in r.split()] for r in values.split("|")]
                weights[(int(head[1]), head[2])] = np.array(rows if len(rows) > 1 else rows[0])
            elif word in ("K", "V", "hidden"):
                key = tuple(int(x) for x in head[1:])
                expect.append((word, key, [_eval_expr(e, env) for e in values.split(",")]))
            else:
                raise ValueError(f"unknown fixture line: {line}")
    shape = W.ModelShape(int(kw["layers"]), int(kw["hidden"]), int(kw["q_heads"]),
                         int(kw["kv_heads"]), int(kw["head_dim"]), int(kw["ffn"]),
                         int(kw["vocab"]), kw["eps"], kw["theta"], F64)
    w = {"embed": np.array([embed[t] for t in range(shape.vocab)], np.float64),
         "layers": [{k: np.ascontiguousarray(weights[(l, k)], np.float64) for k in W.LAYER_KEYS}
                    for l in range(shape.num_layers)]}
    B, NB = int(arena["block_size"]), int(arena["num_blocks"])
    max_blocks = max(len(b) for _, b in reqs)
    tables = np.full((len(reqs), max_blocks), -1, np.int32)
    for r, (_, b) in enumerate(reqs):
        tables[r, :len(b)] = b
    wl = W.Workload("worked_example", shape, np.array([len(t) for t, _ in reqs], np.int32),
                    np.array([t for toks, _ in reqs for t in toks], np.int32), B, NB, max_blocks,
                    tables, np.zeros(0, np.int64), 0)
    return shape, w, wl, expect


def pin_worked_example_by_hand(o):
    """Every K and V the rebuild writes, and the residual after the last layer,
    of a two-layer model equal to values derived by hand in closed form (fp64
    mode); every other arena element keeps its fill value."""
    shape, w, wl, expect = _worked_example(os.path.join(os.path.dirname(__file__), "golden",
                                                       "worked_example.txt"))
    fill = -7.0
    arena = np.full(wl.arena_elems(), fill, np.float64)
    a, fh = run(o, shape, w, wl, arena=arena, final_hidden=True)
    v = view(wl, shape, a)
    off = wl.request_offsets()
    seen = np.zeros(v.shape[:4], bool)
    for kind, key, want in expect:
        if kind == "hidden":
            r, p = key
            got = fh[off[r] + p]
        else:
            l, r, p = key
            blk, slot = wl.block_tables[r, p // wl.block_size], p % wl.block_size
            got = v[l, 0 if kind == "K" else 1, blk, slot].reshape(-1)
            seen[l, 0 if kind == "K" else 1, blk, slot] = True
        want = np.array(want)
        assert np.all(np.abs(got - want) <= 1e-12 * np.maximum(1.0, np.abs(want))), \
            f"worked example {kind} {key}: oracle {got} vs hand-derived {want}"
    assert np.array_equal(seen, written_mask(wl, shape)), "worked example does not cover every written slot"
    assert np.all(v[~seen] == fill), "worked example: an unlisted arena element changed"


def pin_position0_unrotated(o):
    import torch
    import torch.nn.functional as F
    shape = dataclasses.replace(TINY_GQA, dtype=F64)
    w = weights_in(W.host_weights(dataclasses.replace(shape, dtype=F32), seed=9), F32, F64)
    toks = np.array([3, 500, 1023], np.int32)
    k, v = o.layer0_kv(shape, w["embed"], w["layers"][0], toks, np.zeros(3, np.int32))
    lw = w["layers"][0]
    x = torch.from_numpy(w["embed"][toks])
    a = F.rms_norm(x, (shape.hidden,), weight=torch.from_numpy(lw["attn_norm"]), eps=shape.rms_eps)
    kk = F.linear(a, torch.from_numpy(lw["wk"])).numpy()
    vv = F.linear(a, torch.from_numpy(lw["wv"])).numpy()
    assert normwise(k, kk) < 1e-12 and normwise(v, vv) < 1e-12, "position-0 K/V is not W a"


def pin_rope_rotation(o):
    shape = dataclasses.replace(TINY_GQA, dtype=F64)
    d, nkv, half = shape.head_dim, shape.num_kv_heads, shape.head_dim // 2
    w = weights_in(W.host_weights(dataclasses.replace(shape, dtype=F32), seed=10), F32, F64)
    tok = 77
    for p in (1, 5, 1000):
        k, _ = o.layer0_kv(shape, w["embed"], w["layers"][0], np.array([tok, tok], np.int32),
                           np.array([0, p], np.int32))
        k0 = k[0].reshape(nkv, d)
        kp = k[1].reshape(nkv, d)
        i = np.arange(half)
        n0 = np.hypot(k0[:, i], k0[:, i + half])
        npn = np.hypot(kp[:, i], kp[:, i + half])
        assert np.allclose(n0, npn, rtol=1e-12, atol=0), "rotary pair norm not preserved"
        ang = np.arctan2(kp[:, i + half], kp[:, i]) - np.arctan2(k0[:, i + half], k0[:, i])
        expect = p * shape.rope_theta ** (-2.0 * i / d)
        diff = np.angle(np.exp(1j * (ang - expect[None, :])))
        assert np.max(np.abs(diff)) < 1e-9, "rotation angle differs from p * theta^(-2i/d)"


def pin_rope_relative(o):
    shape = dataclasses.replace(TINY_GQA, dtype=F64)
    d, nkv = shape.head_dim, shape.num_kv_heads
    w = weights_in(W.host_weights(dataclasses.replace(shape, dtype=F32), seed=12), F32, F64)
    tok = 123
    pos = np.array([3, 10, 3 + 57, 10 + 57], np.int32)
    k, _ = o.layer0_kv(shape, w["embed"], w["layers"][0], np.full(4, tok, np.int32), pos)
    k = k.reshape(4, nkv, d)
    d1 = np.einsum("hd,hd->h", k[0], k[1])
    d2 = np.einsum("hd,hd->h", k[2], k[3])
    assert np.allclose(d1, d2, rtol=1e-11, atol=1e-14), "dot products depend on absolute position"


def pin_gqa_equals_mha(o):
    shape = dataclasses.replace(TINY_GQA, num_layers=2)
    g = shape.num_q_heads // shape.num_kv_heads
    d = shape.head_dim
    wl = W.small_workload(shape, [13, 40], seed=51, other_live_frac=0.0)
    w = W.host_weights(shape, seed=13)
    a = run(o, shape, w, wl)
    mha = dataclasses.replace(shape, num_kv_heads=shape.num_q_heads)
    wm = {"embed": w["embed"], "layers": []}
    for lw in w["layers"]:
        lm = dict(lw)
        for key in ("wk", "wv"):
            rows = lw[key].reshape(shape.num_kv_heads, d, -1)
            lm[key] = np.ascontiguousarray(np.repeat(rows, g, axis=0).reshape(mha.num_kv_heads * d, -1))
        wm["layers"].append(lm)
    wlm = dataclasses.replace(wl, shape=mha)
    am = run(o, mha, wm, wlm)
    for r in range(wl.num_requests):
        k, v = gather(wl, shape, a, r)
        km, vm = gather(wlm, mha, am, r)
        for h in range(mha.num_kv_heads):
            assert np.array_equal(km[:, :, h], k[:, :, h // g]), "GQA K != MHA K"
            assert np.array_equal(vm[:, :, h], v[:, :, h // g]), "GQA V != MHA V"


def _torch_compare(o, shape, wl, w, dt, rounding, tol, min_exact=None, round_p=False):
    import torch_ref
    a = run(o, shape, w, wl, dt=dt, round_p=round_p)
    w64 = torch_ref.weights_f64(w, dt)
    refs = torch_ref.forward_batch(shape, w64, wl, rounding, round_p)
    worst, exact, total = 0.0, 0, 0
    for r in range(wl.num_requests):
        if refs[r] is None:
            continue
        K, V = gather(wl, shape, a, r)
        Kr, Vr = refs[r][0].numpy(), refs[r][1].numpy()
        for l in range(shape.num_layers):
            for got, ref in ((K[l], Kr[l]), (V[l], Vr[l])):
                gf = as_float(got, dt)
                for h in range(shape.num_kv_heads):
                    worst = max(worst, normwise(gf[:, h], ref[:, h]))
                exact += int(np.sum(gf == ref))
                total += gf.size
    assert worst <= tol, f"oracle vs textbook torch: {worst:.3e} > {tol:.1e}"
    if min_exact is not None:
        assert exact >= min_exact * total, f"only {exact}/{total} values bit-exact"


def pin_torch_f64(o):
    wl = W.config1()
    shape = dataclasses.replace(wl.shape, dtype=F64)
    w = weights_in(W.host_weights(wl.shape, seed=14), F32, F64)
    _torch_compare(o, shape, dataclasses.replace(wl, shape=shape), w, F64, None, 1e-10)


def pin_torch_f64_gqa(o):
    shape = dataclasses.replace(TINY_GQA, dtype=F64)
    wl = W.small_workload(shape, [1, 16, 45], seed=61, other_live_frac=0.2)
    w = weights_in(W.host_weights(dataclasses.replace(shape, dtype=F32), seed=15), F32, F64)
    _torch_compare(o, shape, wl, w, F64, None, 1e-10)


def pin_torch_f32_rounding(o):
    wl = W.config1()
    w = W.host_weights(wl.shape, seed=16)
    _torch_compare(o, wl.shape, wl, w, F32, "f32", 1e-6, min_exact=0.999)


def pin_torch_bf16_rounding(o):
    shape = TINY_BF16_2L
    wl = W.small_workload(shape, [1, 17, 70], seed=71)
    w = W.host_weights(shape, seed=17)
    _torch_compare(o, shape, wl, w, BF16, "bf16", 1e-3, min_exact=0.999)


def pin_torch_bf16_rounding_round_p(o):
    """round_p mode against the same torch forward with the attention written
    out and its weights rounded before P.V and the denominator; the mode
    must change the result (P rounding is not a no-op)."""
    shape = TINY_BF16_2L
    wl = W.small_workload(shape, [1, 17, 70], seed=71)
    w = W.host_weights(shape, seed=17)
    _torch_compare(o, shape, wl, w, BF16, "bf16", 1e-3, min_exact=0.999, round_p=True)
    plain, rp = run(o, shape, w, wl), run(o, shape, w, wl, round_p=True)
    assert not np.array_equal(plain, rp), "round_p left the bf16 rebuild unchanged"


def pin_bf16_rounding_matches_torch(o):
    import torch
    rng = np.random.default_rng(5)
    specials = np.array([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, 3.4e38, -3.4e38, 1e-40, -1e-40,
                         1.00390625, 1.01171875, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8,
                         65504.0, 2 ** -126, 2 ** -133], np.float32)
    bits = rng.integers(0, 2 ** 32, size=20000, dtype=np.uint64).astype(np.uint32)
    vals = np.concatenate([specials, bits.view(np.float32)])
    vals = vals[~np.isnan(vals)]
    ref = torch.from_numpy(vals).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([o.round_bf16(float(x)) for x in vals], np.uint16)
    assert np.array_equal(got, ref), "bf16 rounding differs from torch"


def pin_batch_independence(o):
    shape = W.TINY_F32
    wl = W.small_workload(shape, [30, 64, 17], seed=81, other_live_frac=0.1)
    w = W.host_weights(shape, seed=18)
    a = run(o, shape, w, wl)
    for r in range(wl.num_requests):
        off = wl.request_offsets()
        single = dataclasses.replace(wl, lens=wl.lens[r:r + 1].copy(),
                                     tokens=wl.tokens[off[r]:off[r + 1]].copy(),
                                     block_tables=wl.block_tables[r:r + 1].copy())
        b = run(o, shape, w, single)
        k1, v1 = gather(wl, shape, a, r)
        k2, v2 = gather(single, shape, b, 0)
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2), "result depends on the batch"


def pin_idempotent_over_garbage(o):
    shape = W.TINY_F32
    wl = W.small_workload(shape, [25, 40], seed=91, other_live_frac=0.2)
    w = W.host_weights(shape, seed=19)
    clean = run(o, shape, w, wl)
    garbage = W.host_arena(wl)
    vg = view(wl, shape, garbage)
    rng = np.random.default_rng(3)
    m = written_mask(wl, shape)
    junk = rng.integers(0, 2 ** 32, size=vg[m].shape, dtype=np.uint64).astype(np.uint32)
    vg[m] = junk  # arbitrary bits, NaNs included, in every target slot
    half = clean.copy()
    vh = view(wl, shape, half)
    vh[:, :, :, : wl.block_size // 2] = view(wl, shape, garbage)[:, :, :, : wl.block_size // 2]
    for start in (garbage, half):
        again = run(o, shape, w, wl, arena=start.copy())
        assert np.array_equal(again, clean), "rebuild depends on prior slot contents"


def pin_layer0_helper_matches_rebuild(o):
    shape = TINY_BF16_2L
    wl = W.small_workload(shape, [3, 50], seed=101)
    w = W.host_weights(shape, seed=20)
    a = run(o, shape, w, wl)
    pos = np.concatenate([np.arange(n) for n in wl.lens]).astype(np.int32)
    k, v = o.layer0_kv(shape, w["embed"], w["layers"][0], wl.tokens, pos)
    off = wl.request_offsets()
    for r in range(wl.num_requests):
        K, V = gather(wl, shape, a, r)
        assert np.array_equal(K[0].reshape(len(K[0]), -1), k[off[r]:off[r + 1]])
        assert np.array_equal(V[0].reshape(len(V[0]), -1), v[off[r]:off[r + 1]])


def pin_empty_and_single(o):
    shape = W.TINY_F32
    wl = W.small_workload(shape, [0, 1, 0], seed=111, other_live_frac=0.0)
    w = W.host_weights(shape, seed=21)
    before = W.host_arena(wl)
    after = run(o, shape, w, wl, arena=before.copy())
    m = written_mask(wl, shape)
    assert m.sum() == shape.num_layers * 2
    vb = view(wl, shape, before).reshape(*m.shape, -1)
    va = view(wl, shape, after).reshape(*m.shape, -1)
    assert np.array_equal(va[~m], vb[~m])
    # n = 1: attention over one key returns V_0, so layer 1 sees x0 + Wo V_0 + FFN;
    # the 1-token request alone equals the same request inside any batch
    single = W.small_workload(shape, [1], seed=111, other_live_frac=0.0)
    single.tokens = wl.tokens.copy()
    b = run(o, shape, w, single)
    k1, v1 = gather(wl, shape, after, 1)
    k2, v2 = gather(single, shape, b, 0)
    assert np.array_equal(k1, k2) and np.array_equal(v1, v2)


# ----------------------------------------------------------------------
# the Qwen attention variants: per-head q/k RMSNorm (Qwen3), q/k/v bias (Qwen2.5)
# ----------------------------------------------------------------------
VARIANTS = {"qk_norm": dict(qk_norm=True), "qkv_bias": dict(qkv_bias=True),
            "both": dict(qk_norm=True, qkv_bias=True)}


def pin_torch_variants_f64(o):
    for name, kw in VARIANTS.items():
        base = dataclasses.replace(TINY_GQA, **kw)
        shape = dataclasses.replace(base, dtype=F64)
        wl = W.small_workload(base, [5, 19, 1], seed=150, other_live_frac=0.0)
        w = weights_in(W.host_weights(base, seed=51), F32, F64)
        _torch_compare(o, shape, dataclasses.replace(wl, shape=shape), w, F64, None, 1e-10)


def pin_torch_variants_rounding(o):
    """The variants' rounding sites (bias joined to the fp64 sum before its one
    rounding to fp32; the head norm's output kept in working precision until q
    and k are rounded after RoPE) against the torch forward with the same
    sites emulated, held to the base model's bar: the bound and the share of
    bit-identical values of pin_torch_f32_rounding / pin_torch_bf16_rounding."""
    for name, kw in VARIANTS.items():
        for base, rounding, tol in ((dataclasses.replace(TINY_GQA, **kw), "f32", 1e-6),
                                    (dataclasses.replace(TINY_BF16_2L, **kw), "bf16", 1e-3)):
            wl = W.small_workload(base, [5, 19], seed=151, other_live_frac=0.0)
            w = W.host_weights(base, seed=52)
            _torch_compare(o, base, wl, w, base.dtype, rounding, tol, min_exact=0.999)


def pin_qk_norm_scale_invariance(o):
    """With the per-head norm (and eps = 0) q and k do not depend on the scale
    of Wq and Wk: scaling both by 3 leaves every K/V output unchanged up to
    fp64 rounding, while it does change them without the norm."""
    for qk in (True, False):
        shape = dataclasses.replace(TINY_GQA, dtype=F64, qk_norm=qk, rms_eps=0.0)
        wl = W.small_workload(shape, [7, 12], seed=152, other_live_frac=0.0)
        w = weights_in(W.host_weights(dataclasses.replace(shape, dtype=F32), seed=53), F32, F64)
        w3 = {"embed": w["embed"], "layers": [dict(lw) for lw in w["layers"]]}
        for lw in w3["layers"]:
            lw["wq"] = lw["wq"] * 3.0
            lw["wk"] = lw["wk"] * 3.0
        a1 = run(o, shape, w, wl, dt=F64)
        a3 = run(o, shape, w3, wl, dt=F64)
        err = normwise(a3[np.isfinite(a3)], a1[np.isfinite(a1)])
        if qk:
            assert err < 1e-12, err
        else:
            assert err > 1e-3, err


def pin_value_bias_closed_form(o):
    """With Wv = 0 every value row is the bias: V of every layer equals
    rnd(bv) at every position, and attention returns exactly that row."""
    shape = dataclasses.replace(TINY_BF16_2L, qkv_bias=True)
    wl = W.small_workload(shape, [3, 17], seed=153, other_live_frac=0.0)
    w = W.host_weights(shape, seed=54)
    for lw in w["layers"]:
        lw["wv"] = np.zeros_like(lw["wv"])
    a = run(o, shape, w, wl)
    for r in range(wl.num_requests):
        _, V = gather(wl, shape, a, r)
        for l in range(shape.num_layers):
            bv = w["layers"][l]["bv"].reshape(shape.num_kv_heads, shape.head_dim)
            assert np.array_equal(V[l], np.broadcast_to(bv, V[l].shape))


# ----------------------------------------------------------------------
# resumed decode (the step after the rebuild): final norm, LM head, greedy
# ----------------------------------------------------------------------
def _head_in(head: dict, src_dt: int, dst_dt: int) -> dict:
    if src_dt == dst_dt:
        return head
    f = {k: (W.bf16_bits_to_f32(v) if src_dt == BF16 else v.astype(np.float32)) for k, v in head.items()}
    if dst_dt == F64:
        return {k: v.astype(np.float64) for k, v in f.items()}
    if dst_dt == F32:
        return {k: v.astype(np.float32) for k, v in f.items()}
    return {k: W.f32_to_bf16_bits(v) for k, v in f.items()}


def pin_logits_torch(o):
    """Final norm + LM head against the textbook torch formula, in the fp64
    pin mode (no rounding) and with the bf16 rounding contract emulated."""
    import torch_ref  # noqa: E402 - tests/ is on sys.path when pins run
    shape = W.TINY_BF16
    head = W.host_head_weights(shape, seed=31)
    rng = np.random.default_rng(5)
    x = rng.standard_normal((3, shape.hidden)) * 0.7
    x32 = x.astype(np.float32).astype(np.float64)
    z64 = o.logits(shape, _head_in(head, BF16, F64), x, dtype=F64)
    t64 = torch_ref.logits(shape, head["final_norm"], head["lm_head"], x, BF16, None).numpy()
    assert normwise(z64, t64) < 1e-6, normwise(z64, t64)
    zb = o.logits(shape, head, x32)
    tb = torch_ref.logits(shape, head["final_norm"], head["lm_head"], x32, BF16, "bf16").numpy()
    # the normed activations are bf16: both sides round the same fp32 values
    assert normwise(zb, tb) < 1e-5, normwise(zb, tb)


def pin_logits_onehot_closed_form(o):
    """A residual row c*e_k normalizes to a single entry g_k*c/sqrt(c^2/H+eps),
    so every logit is one product: W[v][k] times that entry."""
    shape = dataclasses.replace(W.TINY_F32, vocab=257)
    head = W.host_head_weights(shape, seed=32)
    H = shape.hidden
    ks, cs = [3, 100, H - 1], [2.5, -0.75, 13.0]
    x = np.zeros((len(ks), H))
    for i, (k, c) in enumerate(zip(ks, cs)):
        x[i, k] = c
    z = o.logits(shape, head, x)
    g = head["final_norm"].astype(np.float64)
    wl = head["lm_head"].astype(np.float64)
    for i, (k, c) in enumerate(zip(ks, cs)):
        a = np.float64(np.float32(g[k] * c / math.sqrt(c * c / H + shape.rms_eps)))
        expect = (wl[:, k] * a).astype(np.float32)
        assert np.array_equal(z[i], expect), np.max(np.abs(z[i] - expect))


def pin_greedy_lowest_index(o):
    import oracle as _o
    z = np.array([[1.0, 3.0, 3.0, -1.0], [0.0, 0.0, 0.0, 0.0], [-5.0, -4.0, -4.5, -4.0]], np.float32)
    assert list(_o.greedy(z)) == [1, 0, 1]


def _resume(o, shape, w, head, wl, prefix_mode, steps):
    """Greedy continuation of every request of wl: its prefix (all but the last
    token) rebuilt by prefill or fed token by token, then the last token and
    each generated one decoded at the next position.  Returns (tokens
    [steps, R], last logits, arena)."""
    import oracle as _o
    R = wl.num_requests
    lens = wl.lens.astype(np.int64)
    pre = dataclasses.replace(wl, lens=(lens - 1).astype(wl.lens.dtype),
                              tokens=np.concatenate([wl.tokens[o0:o1 - 1] for o0, o1 in
                                                     zip(wl.request_offsets()[:-1], wl.request_offsets()[1:])]))
    a = W.host_arena(wl)
    if prefix_mode == "prefill":
        o.rebuild(shape, w, pre.tokens, pre.lens, pre.block_tables, a, wl.block_size, wl.num_blocks)
    else:
        for p in range(int(pre.lens.max())):
            rs = [r for r in range(R) if p < pre.lens[r]]
            toks = [pre.tokens[pre.request_offsets()[r] + p] for r in rs]
            o.decode_step(shape, w, toks, [p] * len(rs), wl.block_tables[rs], a, wl.block_size,
                          wl.num_blocks, final_hidden=False)
    offs = wl.request_offsets()
    cur = np.array([wl.tokens[offs[r + 1] - 1] for r in range(R)], np.int32)
    pos = (lens - 1).astype(np.int32)
    out, z = [], None
    for _ in range(steps):
        fh = o.decode_step(shape, w, cur, pos, wl.block_tables, a, wl.block_size, wl.num_blocks)
        z = o.logits(shape, head, fh)
        cur = _o.greedy(z)
        out.append(cur.copy())
        pos = pos + 1
    return np.array(out), z, a


def _resume_workload(shape, lens, steps, seed):
    wl = W.small_workload(shape, [n + steps for n in lens], seed=seed, other_live_frac=0.0)
    offs = wl.request_offsets()
    toks = np.concatenate([wl.tokens[offs[r]:offs[r] + lens[r]] for r in range(len(lens))])
    return dataclasses.replace(wl, lens=np.array(lens, dtype=wl.lens.dtype), tokens=toks)


def pin_decode_step_chain_equals_decode(o):
    """Stepping the oracle position by position over a request equals its
    token-by-token decode mode, arena and final residual bit for bit."""
    shape = W.TINY_F32
    w = W.host_weights(shape, seed=33)
    wl = W.small_workload(shape, [5, 19], seed=133, other_live_frac=0.0)
    a_ref, fh_ref = run(o, shape, w, wl, mode="decode", final_hidden=True)
    a = W.host_arena(wl)
    offs = wl.request_offsets()
    for r in range(wl.num_requests):
        for p in range(int(wl.lens[r])):
            fh = o.decode_step(shape, w, [wl.tokens[offs[r] + p]], [p], wl.block_tables[r:r + 1], a,
                               wl.block_size, wl.num_blocks)
            assert np.array_equal(fh[0], fh_ref[offs[r] + p])
    assert np.array_equal(a, a_ref)


def pin_resume_from_rebuild_equals_decode_built(o):
    """The paper's recoverability criterion on the oracle: generation resumed
    from a rebuilt (prefill) arena continues exactly as from the arena the
    original token-by-token generation built."""
    for shape in (W.TINY_F32, TINY_BF16_2L):
        w = W.host_weights(shape, seed=34)
        head = W.host_head_weights(shape, seed=35)
        wl = _resume_workload(shape, [1, 6, 23], steps=5, seed=134)
        t_re, z_re, a_re = _resume(o, shape, w, head, wl, "prefill", 5)
        t_de, z_de, a_de = _resume(o, shape, w, head, wl, "decode", 5)
        assert np.array_equal(t_re, t_de) and np.array_equal(z_re, z_de)
        assert np.array_equal(a_re, a_de)


# --------------------------------------------------------------------------
# rebuild from a retained prefix
# --------------------------------------------------------------------------
def _piece(wl, lo, hi):
    """Packed tokens of positions lo[r] .. hi[r]-1 of every request."""
    offs = wl.request_offsets()
    parts = [wl.tokens[offs[r] + int(lo[r]):offs[r] + int(hi[r])] for r in range(wl.num_requests)]
    return np.concatenate(parts).astype(np.int32) if parts else np.zeros(0, np.int32)


def pin_rebuild_from_split_equals_full(o):
    """A position's K/V depend only on the tokens up to it (causality):
    rebuilding positions [0, s) and then [s, n) from the retained prefix gives
    the full rebuild's arena bit for bit, with s at 0, at n, at and inside
    block boundaries, for fp32 and bf16 models."""
    for shape, seed in ((TINY_GQA, 51), (TINY_BF16_2L, 52)):
        w = W.host_weights(shape, seed=seed)
        wl = W.small_workload(shape, [1, 17, 40, 33, 0, 9], block_size=8, seed=150 + seed,
                              other_live_frac=0.25)
        B, NB = wl.block_size, wl.num_blocks
        full = W.host_arena(wl)
        o.rebuild(shape, w, wl.tokens, wl.lens, wl.block_tables, full, B, NB)
        starts = np.array([0, 16, 23, 33, 0, 9], np.int32)
        two = W.host_arena(wl)
        zero = np.zeros_like(starts)
        o.rebuild(shape, w, _piece(wl, zero, starts), starts, wl.block_tables, two, B, NB)
        o.rebuild_from(shape, w, _piece(wl, starts, wl.lens), wl.lens, starts, wl.block_tables, two, B, NB)
        assert np.array_equal(two, full), shape


def pin_rebuild_from_boundaries(o):
    """Start 0 is the plain rebuild (bit for bit); start = length changes
    nothing at all."""
    shape = TINY_GQA
    w = W.host_weights(shape, seed=53)
    wl = W.small_workload(shape, [5, 16, 29], seed=153, other_live_frac=0.25)
    B, NB = wl.block_size, wl.num_blocks
    a = W.host_arena(wl)
    o.rebuild(shape, w, wl.tokens, wl.lens, wl.block_tables, a, B, NB)
    b = W.host_arena(wl)
    zero = np.zeros(wl.num_requests, np.int32)
    o.rebuild_from(shape, w, wl.tokens, wl.lens, zero, wl.block_tables, b, B, NB)
    assert np.array_equal(a, b)
    c = a.copy()
    o.rebuild_from(shape, w, np.zeros(0, np.int32), wl.lens, wl.lens, wl.block_tables, c, B, NB)
    assert np.array_equal(a, c)


def pin_rebuild_from_reads_retained_prefix(o):
    """The recomputed positions attend to the prefix K/V the arena holds: with
    one request's prefix slots holding another model's K/V, its recomputed
    layer-0 K/V (which precede any attention) are unchanged, its later
    layers' change, and the other requests are untouched."""
    shape = TINY_GQA
    w, w2 = W.host_weights(shape, seed=54), W.host_weights(shape, seed=55)
    wl = W.small_workload(shape, [24, 24], block_size=8, seed=154, other_live_frac=0.0)
    B, NB = wl.block_size, wl.num_blocks
    starts = np.array([16, 16], np.int32)
    good, bad = W.host_arena(wl), W.host_arena(wl)
    o.rebuild(shape, w, wl.tokens, wl.lens, wl.block_tables, good, B, NB)
    o.rebuild(shape, w2, wl.tokens, wl.lens, wl.block_tables, bad, B, NB)
    mixed = good.copy()
    view_m = mixed.reshape(shape.num_layers, 2, NB, B, -1)
    view_b = bad.reshape(shape.num_layers, 2, NB, B, -1)
    for j in range(2):  # request 1's two prefix blocks from the other model
        view_m[:, :, wl.block_tables[1, j]] = view_b[:, :, wl.block_tables[1, j]]
    o.rebuild_from(shape, w, _piece(wl, starts, wl.lens), wl.lens, starts, wl.block_tables, mixed, B, NB)
    vg = good.reshape(shape.num_layers, 2, NB, B, -1)
    blk0, blk1 = wl.block_tables[0, 2], wl.block_tables[1, 2]   # the recomputed block
    assert np.array_equal(view_m[:, :, blk0], vg[:, :, blk0])
    assert np.array_equal(view_m[0, :, blk1], vg[0, :, blk1])
    assert not np.array_equal(view_m[1:, :, blk1], vg[1:, :, blk1])


def pin_shared_prefix_block_copy(o):
    """Shared-prefix reuse: requests beginning with the same S tokens (S a
    multiple of the block size); the first is rebuilt in full, its first S/B
    blocks are copied into the others' first blocks, and the others are
    rebuilt from S: the arena equals the full rebuild of every request."""
    shape = TINY_BF16_2L
    w = W.host_weights(shape, seed=56)
    wl = W.small_workload(shape, [40, 21, 16, 57], block_size=8, seed=156, other_live_frac=0.25)
    B, NB, S = wl.block_size, wl.num_blocks, 16
    offs = wl.request_offsets()
    toks = wl.tokens.copy()
    for r in range(1, wl.num_requests):
        toks[offs[r]:offs[r] + S] = toks[:S]
    wl = dataclasses.replace(wl, tokens=toks)
    full = W.host_arena(wl)
    o.rebuild(shape, w, wl.tokens, wl.lens, wl.block_tables, full, B, NB)
    arena = W.host_arena(wl)
    first = dataclasses.replace(wl, lens=wl.lens[:1], tokens=wl.tokens[:wl.lens[0]],
                                block_tables=wl.block_tables[:1])
    o.rebuild(shape, w, first.tokens, first.lens, first.block_tables, arena, B, NB)
    view = arena.reshape(shape.num_layers, 2, NB, B, -1)
    for r in range(1, wl.num_requests):
        for j in range(S // B):
            view[:, :, wl.block_tables[r, j]] = view[:, :, wl.block_tables[0, j]]
    starts = np.array([wl.lens[0]] + [S] * (wl.num_requests - 1), np.int32)
    o.rebuild_from(shape, w, _piece(wl, starts, wl.lens), wl.lens, starts, wl.block_tables, arena, B, NB)
    assert np.array_equal(arena, full)


# --------------------------------------------------------------------------
# block commit digests
# --------------------------------------------------------------------------
DIGEST_GEOMS = (dataclasses.replace(W.TINY_F32, num_layers=3, num_q_heads=2, num_kv_heads=2, head_dim=8),
                dataclasses.replace(W.TINY_BF16, num_layers=2, num_q_heads=6, num_kv_heads=3, head_dim=8))
GOLDEN = 0x9E3779B9
M64 = (1 << 64) - 1


def _digest_arena(shape, B=4, NB=5, seed=0):
    """Random raw arena bits plus its 32-bit word view [L, 2, NB, B, words per row]."""
    rng = np.random.default_rng(seed)
    el = np.uint16 if shape.dtype == BF16 else np.uint32
    n = shape.num_layers * 2 * NB * B * shape.num_kv_heads * shape.head_dim
    a = rng.integers(0, np.iinfo(el).max, size=n, dtype=el, endpoint=True)
    wr = shape.num_kv_heads * shape.head_dim * a.itemsize // 4
    return a, a.view(np.uint32).reshape(shape.num_layers, 2, NB, B, wr)


def _keys(n):
    return ((np.arange(n, dtype=np.uint64) * np.uint64(GOLDEN)) & np.uint64(0xFFFFFFFF)).astype(np.uint32)


def pin_digest_keyed_closed_form(o):
    """Covered words set to key_i XOR c (keys in the order layer, K|V, slot,
    word) make every squared term c^2: digest = N c^2 mod 2^64, whatever the
    bytes outside the covered slots hold; c = 0 gives 0; nslots = 0 gives 0."""
    for shape in DIGEST_GEOMS:
        for blk, ns, c in ((0, 4, 0), (2, 3, 1), (4, 1, 0xFFFFFFFF), (3, 2, 0x12345678)):
            a, words = _digest_arena(shape, seed=blk)
            L, _, NB, B, wr = words.shape
            N = L * 2 * ns * wr
            words[:, :, blk, :ns, :] = (_keys(N) ^ np.uint32(c)).reshape(L, 2, ns, wr)
            got = o.block_digest(shape, a, B, NB, blk, ns)
            assert got == (N * c * c) & M64, (shape.dtype, blk, ns, c, got)
        assert o.block_digest(shape, a, B, NB, 1, 0) == 0


def pin_digest_one_changed_word(o):
    """From the keyed arena, word j set to key_j XOR c' gives
    (N-1) c^2 + c'^2 mod 2^64, for words at plane, slot and row boundaries."""
    for shape in DIGEST_GEOMS:
        a, words = _digest_arena(shape, seed=7)
        L, _, NB, B, wr = words.shape
        blk, ns, c = 1, 3, 0xDEADBEEF
        N = L * 2 * ns * wr
        keys = _keys(N)
        view = words[:, :, blk, :ns, :]
        view[...] = (keys ^ np.uint32(c)).reshape(L, 2, ns, wr)
        for j in (0, wr - 1, wr, ns * wr - 1, ns * wr, N // 2 + 1, N - wr, N - 1):
            l, rem = divmod(j, 2 * ns * wr)
            kv, rem = divmod(rem, ns * wr)
            s, w = divmod(rem, wr)
            for c2 in (0, 5, 0xFFFFFFFF):
                saved = view[l, kv, s, w]
                view[l, kv, s, w] = keys[j] ^ np.uint32(c2)
                got = o.block_digest(shape, a, B, NB, blk, ns)
                view[l, kv, s, w] = saved
                assert got == ((N - 1) * c * c + c2 * c2) & M64, (shape.dtype, j, c2)


def pin_digest_detects_every_bit_flip(o):
    """Changing one 32-bit word x to x' changes (x^k)^2 by a nonzero amount
    below 2^64 in magnitude, so any change of one covered word is detected;
    check every bit of a few words of each plane."""
    for shape in DIGEST_GEOMS:
        a, words = _digest_arena(shape, seed=11)
        L, _, NB, B, wr = words.shape
        blk, ns = 2, B
        ref = o.block_digest(shape, a, B, NB, blk, ns)
        for l in range(L):
            for kv in range(2):
                for (s, w) in ((0, 0), (B - 1, wr - 1)):
                    for bit in range(32):
                        words[l, kv, blk, s, w] ^= np.uint32(1 << bit)
                        assert o.block_digest(shape, a, B, NB, blk, ns) != ref, (l, kv, s, w, bit)
                        words[l, kv, blk, s, w] ^= np.uint32(1 << bit)
        assert o.block_digest(shape, a, B, NB, blk, ns) == ref


def pin_digest_covers_exactly_its_slots(o):
    """Bytes of other blocks and of slots >= nslots do not enter the digest;
    the same contents moved to another block give the same digest."""
    for shape in DIGEST_GEOMS:
        a, words = _digest_arena(shape, seed=13)
        L, _, NB, B, wr = words.shape
        blk, ns = 3, 2
        ref = o.block_digest(shape, a, B, NB, blk, ns)
        rng = np.random.default_rng(5)
        for other in range(NB):
            if other != blk:
                words[:, :, other] = rng.integers(0, 2**32, size=words[:, :, other].shape, dtype=np.uint64).astype(np.uint32)
        words[:, :, blk, ns:] = 0
        assert o.block_digest(shape, a, B, NB, blk, ns) == ref
        words[:, :, 0, :ns] = words[:, :, blk, :ns]
        assert o.block_digest(shape, a, B, NB, 0, ns) == ref
        assert o.block_digest(shape, a, B, NB, blk, ns + 1) != ref


def pin_verify_leading_intact_counts(o):
    """Committed digests of a rebuilt arena, then corruption planted in chosen
    blocks: each request's leading-intact count is the index of its first
    corrupted block; tail slots past a request's length and blocks of other
    requests do not count against it."""
    shape = W.TINY_F32
    w = W.host_weights(shape, seed=41)
    wl = W.small_workload(shape, [5, 16, 33, 0, 47], block_size=8, seed=141, other_live_frac=0.2)
    image = W.host_arena(wl)
    o.rebuild(shape, w, wl.tokens, wl.lens, wl.block_tables, image, wl.block_size, wl.num_blocks)
    committed, intact = o.verify(shape, image, wl.block_size, wl.num_blocks, wl.lens, wl.block_tables)
    nb = (wl.lens + wl.block_size - 1) // wl.block_size
    assert committed.size == nb.sum() and np.all(intact == 0) or nb.sum() == 0
    _, intact = o.verify(shape, image, wl.block_size, wl.num_blocks, wl.lens, wl.block_tables, committed)
    assert np.array_equal(intact, nb)
    B = wl.block_size
    row = shape.num_kv_heads * shape.head_dim
    arena6 = image.view(np.float32).reshape(shape.num_layers, 2, wl.num_blocks, B, row)
    # tail slots of request 2 (33 tokens: block 4 holds slot 0 only) and a free block
    arena6[1, 0, wl.block_tables[2, 4], 1:] = np.float32(7.0)
    for b in wl.other_live[:2]:
        arena6[0, 1, b] += np.float32(1.0)
    _, intact = o.verify(shape, image, B, wl.num_blocks, wl.lens, wl.block_tables, committed)
    assert np.array_equal(intact, nb)
    # request 1: block 1 (V plane, last layer); request 4: block 2 and block 5
    arena6[shape.num_layers - 1, 1, wl.block_tables[1, 1], B - 1, row - 1] *= np.float32(-1.0)
    arena6[0, 0, wl.block_tables[4, 2], 0, 0] = np.float32(0.5)
    arena6[0, 0, wl.block_tables[4, 5], 0, 0] = np.float32(0.25)
    _, intact = o.verify(shape, image, B, wl.num_blocks, wl.lens, wl.block_tables, committed)
    assert intact.tolist() == [nb[0], 1, nb[2], 0, 2], intact.tolist()


PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]


if __name__ == "__main__":
    import oracle
    inst = oracle.Oracle(sys.argv[1])
    failed = []
    for pin in PINS:
        try:
            pin(inst)
        except Exception as e:  # noqa: BLE001 - any failure counts as caught
            failed.append(f"{pin.__name__}: {type(e).__name__}: {str(e)[:80]}")
    for f in failed:
        print("FAILED", f)
    print(f"{len(failed)} of {len(PINS)} pins failed")
