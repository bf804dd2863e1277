"""GPU parity at the sizes the benchmark runs, through the C ABI.

The oracle cannot run a whole 8B-shaped rebuild of 128K tokens (hours of fp64
work), so these tests compare outputs it can compute one by one:

* layer-0 K/V of every token (they depend only on the tokens and positions);
* layer-1 K/V at sampled positions of a two-layer rebuild: the oracle first
  writes layer-0 K/V of every position of the request, then runs its decode
  step (one token at a time, keys read back from its arena) at each sampled
  position, which is the prefill's result for that row bit for bit (the
  oracle's prefill and decode modes are pinned equal) and depends on
  layer-0 attention over every earlier key and on the layer-0 output and
  FFN products of that row;
* one resumed decode step over the rebuilt contexts of a one-layer model
  (paged attention over the whole context, final norm, LM head, argmax).

Tolerances as everywhere: max normwise error per (layer, K|V, kv head)
tensor of 2e-2 for bf16; the decode step's K/V rows and each request's
logits likewise; untouched arena contents bit-exact.
"""
import dataclasses
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from paper_2608_14635_amd import harness as Hn  # noqa: E402
from paper_2608_14635_amd import kvr  # noqa: E402
from paper_2608_14635_amd import workloads as W  # noqa: E402

import parity_util as PU  # noqa: E402

pytestmark = pytest.mark.gpu
TOL = PU.TOL[W.BF16]


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def token_positions(wl):
    """(request, position) of every token in packed order."""
    req = np.repeat(np.arange(wl.num_requests), wl.lens)
    pos = np.concatenate([np.arange(n) for n in wl.lens]).astype(np.int32) if wl.total_tokens \
        else np.zeros(0, np.int32)
    return req, pos


def oracle_layer0(oracle_lib, wl, h0, step=16384):
    """Oracle layer-0 K and V rows [T, nkv*d] of every token of wl."""
    _, pos = token_positions(wl)
    toks = wl.tokens.astype(np.int32)
    kd = wl.shape.num_kv_heads * wl.shape.head_dim
    K = np.empty((wl.total_tokens, kd), np.uint16)
    V = np.empty((wl.total_tokens, kd), np.uint16)
    for c0 in range(0, wl.total_tokens, step):
        c1 = min(wl.total_tokens, c0 + step)
        K[c0:c1], V[c0:c1] = oracle_lib.layer0_kv(wl.shape, h0["embed"], h0["layer0"], toks[c0:c1],
                                                 pos[c0:c1])
        say(f"  oracle layer-0 K/V of tokens {c0}..{c1 - 1}")
    return K, V


class NormErr:
    """Running max |g - o| and max |o| per kv head."""

    def __init__(self, nkv):
        self.num, self.den = np.zeros(nkv), np.zeros(nkv)
        self.same = self.total = 0

    def add(self, g_bits, o_bits, nkv, d):
        gf = W.bf16_bits_to_f32(g_bits).reshape(-1, nkv, d).astype(np.float64)
        of = W.bf16_bits_to_f32(o_bits).reshape(-1, nkv, d).astype(np.float64)
        self.num = np.maximum(self.num, np.abs(gf - of).max(axis=(0, 2)))
        self.den = np.maximum(self.den, np.abs(of).max(axis=(0, 2)))
        self.same += int(np.sum(g_bits == o_bits))
        self.total += g_bits.size

    def err(self):
        err = float(np.max(self.num / np.where(self.den > 0, self.den, 1.0)))
        return err if np.isfinite(err) else np.inf  # NaN would vanish in a max() fold

    def exact(self):
        return self.same / max(1, self.total)


def device_rows(arena, layer, plane, wl, req, pos):
    """Arena rows [n, nkv*d] (bf16 bits) at the slots of (req, pos), gathered on the device."""
    B = wl.block_size
    blk = torch.as_tensor(wl.block_tables[req, pos // B].astype(np.int64), device="cuda")
    sl = torch.as_tensor((pos % B).astype(np.int64), device="cuda")
    return arena.bits[layer, plane][blk, sl].cpu().numpy().view(np.uint16).reshape(len(pos), -1)


def compare_layer0_every_token(arena, wl, K0, V0, label, step=16384):
    req, pos = token_positions(wl)
    nkv, d = wl.shape.num_kv_heads, wl.shape.head_dim
    errs = {"K": NormErr(nkv), "V": NormErr(nkv)}
    for c0 in range(0, wl.total_tokens, step):
        c1 = min(wl.total_tokens, c0 + step)
        for name, plane, ref in (("K", 0, K0), ("V", 1, V0)):
            g = device_rows(arena, 0, plane, wl, req[c0:c1], pos[c0:c1])
            errs[name].add(g, ref[c0:c1], nkv, d)
    for name in ("K", "V"):
        say(f"  {label}: layer-0 {name} over all {wl.total_tokens} tokens: normwise "
            f"{errs[name].err():.3e}, bit-exact {errs[name].exact():.4f}")
        assert errs[name].err() <= TOL


def oracle_arena_with_layer0(wl, shape, K0, V0, req_ids=None):
    """Host arena of `shape`'s geometry: sentinel everywhere, and layer-0 K/V
    of the listed requests' positions (every request by default) at their
    slots, taken from the oracle's rows K0/V0."""
    s = shape
    sen = W.SENTINEL_BITS[W.BF16]
    a = np.full((s.num_layers, 2, wl.num_blocks, wl.block_size, s.num_kv_heads * s.head_dim), sen,
                np.uint16)
    req, pos = token_positions(wl)
    keep = np.ones(len(req), bool) if req_ids is None else np.isin(req, req_ids)
    blk = wl.block_tables[req[keep], pos[keep] // wl.block_size]
    sl = pos[keep] % wl.block_size
    a[0, 0, blk, sl] = K0[keep]
    a[0, 1, blk, sl] = V0[keep]
    return a.reshape(-1)


def sample_positions(n, rng, extra=4):
    """Positions of one request: both ends, block and tile edges, random ones."""
    edges = [0, 1, 15, 16, 63, 64, 255, 256, 1023, 1024, 4095, 4096, 16383, 16384, 32767, 32768,
             n // 2, n - 2, n - 1]
    p = {x for x in edges if 0 <= x < n}
    p |= set(rng.integers(0, n, size=extra).tolist()) if n > 0 else set()
    return np.array(sorted(p), np.int32)


def sampled_layer1(oracle_lib, wl2, host_w2, ora2, samples):
    """Oracle layer-1 K/V at sampled (request, position) pairs of a two-layer
    model, over an arena holding layer-0 K/V of every earlier position:
    one decode step per pair.  Returns the K, V rows [n, nkv*d] (layers 0, 1)."""
    req = np.array([r for r, _ in samples], np.int64)
    pos = np.array([p for _, p in samples], np.int32)
    offs = wl2.request_offsets()
    toks = wl2.tokens[offs[req] + pos].astype(np.int32)
    oracle_lib.decode_step(wl2.shape, host_w2, toks, pos, wl2.block_tables[req], ora2,
                           wl2.block_size, wl2.num_blocks, final_hidden=False)
    s = wl2.shape
    v = ora2.reshape(s.num_layers, 2, wl2.num_blocks, wl2.block_size, -1)
    blk, sl = wl2.block_tables[req, pos // wl2.block_size], pos % wl2.block_size
    return req, pos, v[:, :, blk, sl]


def compare_sampled(arena, wl, req, pos, rows, label):
    """GPU arena rows at the sampled slots against the oracle's, per layer and plane."""
    s = wl.shape
    nkv, d = s.num_kv_heads, s.head_dim
    worst = 0.0
    for l in range(s.num_layers):
        for plane, name in ((0, "K"), (1, "V")):
            e = NormErr(nkv)
            e.add(device_rows(arena, l, plane, wl, req, pos), rows[l, plane], nkv, d)
            say(f"  {label}: layer-{l} {name} at {len(pos)} sampled positions: normwise {e.err():.3e}, "
                f"bit-exact {e.exact():.4f}")
            worst = max(worst, e.err())
    assert worst <= TOL


def gpu_rebuild_into(wl, model, fill=0xFF):
    arena = Hn.DeviceArena(wl)
    arena.bind()
    ws, nbytes = Hn.alloc_workspace(wl.shape, wl.num_requests, wl.total_tokens, wl.total_tokens,
                                    fill=fill)
    kvr.kv_rebuild(model.weights, wl.tokens, wl.lens, wl.block_tables, arena.handle, ws.data_ptr(),
                   nbytes, Hn.stream_ptr())
    torch.cuda.synchronize()
    del ws
    return arena


# --------------------------------------------------------------------------
# the full 8B benchmark workload: 16 requests, 128,325 tokens
# --------------------------------------------------------------------------
def test_config2_full_batch(oracle_lib):
    """All 32 layers: device invariants and layer-0 K/V of every token.
    Two layers: layer-1 K/V at sampled positions of every request (attention
    over up to 16K keys, the O, gate/up and down products at 128,896 rows).
    One layer: a resumed decode step of all 16 requests over their whole
    contexts, in the benchmark's launch configuration."""
    wl = W.config2()
    s = wl.shape
    say(f"config2 full: R={wl.num_requests} T={wl.total_tokens} NB={wl.num_blocks} "
        f"lens {sorted(wl.lens.tolist())}")
    model = Hn.device_model_random(s, seed=2, gain_std=0.1)
    h0 = Hn.host_copy_layer0(model)
    K0, V0 = oracle_layer0(oracle_lib, wl, h0)

    # ---- all 32 layers ----
    arena = gpu_rebuild_into(wl, model)
    inv = arena.check_invariants()
    say(f"  32 layers: device invariants {inv}")
    assert inv == {"free_changed": 0, "live_changed": 0, "tail_changed": 0, "written_bad": 0}
    compare_layer0_every_token(arena, wl, K0, V0, "32 layers")
    arena.release()
    del arena
    torch.cuda.empty_cache()

    # ---- two layers: layer-1 K/V at sampled positions of every request ----
    m2 = Hn.first_layers(model, 2)
    wl2 = dataclasses.replace(wl, shape=m2.shape)
    arena2 = gpu_rebuild_into(wl2, m2)
    inv = arena2.check_invariants()
    assert inv == {"free_changed": 0, "live_changed": 0, "tail_changed": 0, "written_bad": 0}
    compare_layer0_every_token(arena2, wl2, K0, V0, "2 layers")
    rng = np.random.default_rng(7)
    samples = [(r, int(p)) for r in range(wl.num_requests)
               for p in sample_positions(int(wl.lens[r]), rng, extra=3)]
    host_w2 = {"embed": h0["embed"], "layers": [h0["layer0"], Hn.host_copy_layer(model, 1)]}
    ora2 = oracle_arena_with_layer0(wl2, m2.shape, K0, V0)
    say(f"  oracle: layer-1 K/V at {len(samples)} sampled positions")
    req, pos, rows = sampled_layer1(oracle_lib, wl2, host_w2, ora2, samples)
    # the oracle's decode-mode layer-0 rows are its prefill rows, bit for bit
    offs = wl.request_offsets()
    assert np.array_equal(rows[0, 0], K0[offs[req] + pos]) and np.array_equal(rows[0, 1], V0[offs[req] + pos])
    compare_sampled(arena2, wl2, req, pos, rows, "2 layers")
    arena2.release()
    del arena2, ora2
    torch.cuda.empty_cache()

    # ---- one layer: resumed decode over every request's whole context ----
    m1 = Hn.first_layers(model, 1)
    wl1 = dataclasses.replace(wl, shape=m1.shape)
    arena1 = gpu_rebuild_into(wl1, m1)
    compare_layer0_every_token(arena1, wl1, K0, V0, "1 layer")
    head = Hn.device_head_random(s, seed=0x5EED00FF)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    head["final_norm"] = (1.0 + 0.1 * torch.randn(s.hidden, device="cuda", generator=gen)).to(torch.bfloat16)
    lens = wl.lens.astype(np.int64)
    last = np.array([wl.tokens[offs[r + 1] - 1] for r in range(wl.num_requests)], np.int32)
    pos = (lens - 1).astype(np.int32)
    nbytes = kvr.kv_decode_workspace_bytes(m1.shape, wl.num_requests, int(pos.max()) + 1)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    nxt = torch.zeros(wl.num_requests, dtype=torch.int32, device="cuda")
    logits = torch.zeros((wl.num_requests, s.vocab), dtype=torch.float32, device="cuda")
    kvr.kv_decode_step(m1.weights, head["final_norm"].data_ptr(), head["lm_head"].data_ptr(), last,
                       pos, wl.block_tables, arena1.handle, ws.data_ptr(), nbytes, nxt.data_ptr(),
                       logits.data_ptr(), Hn.stream_ptr())
    torch.cuda.synchronize()
    tok_g, z_g = nxt.cpu().numpy(), logits.cpu().numpy()
    kg = device_rows(arena1, 0, 0, wl1, np.arange(wl.num_requests), pos)
    vg = device_rows(arena1, 0, 1, wl1, np.arange(wl.num_requests), pos)
    ora1 = oracle_arena_with_layer0(wl1, m1.shape, K0, V0)
    host_w1 = {"embed": h0["embed"], "layers": [h0["layer0"]]}
    head_h = Hn.host_copy_head(model, head)
    say("  oracle: decode step of 16 requests over their contexts")
    fh = oracle_lib.decode_step(m1.shape, host_w1, last, pos, wl.block_tables, ora1, wl.block_size,
                                wl.num_blocks)
    z_o = oracle_lib.logits(m1.shape, head_h, fh)
    v1 = ora1.reshape(1, 2, wl.num_blocks, wl.block_size, -1)
    blk, sl = wl.block_tables[np.arange(wl.num_requests), pos // wl.block_size], pos % wl.block_size
    nkv, d = s.num_kv_heads, s.head_dim
    ek, ev = NormErr(nkv), NormErr(nkv)
    ek.add(kg, v1[0, 0, blk, sl], nkv, d)
    ev.add(vg, v1[0, 1, blk, sl], nkv, d)
    z_err = max(float(np.max(np.abs(z_g[r].astype(np.float64) - z_o[r])) / np.max(np.abs(z_o[r])))
                for r in range(wl.num_requests))
    say(f"  decode step: K rows {ek.err():.3e}, V rows {ev.err():.3e}, logits {z_err:.3e}; "
        f"gpu tokens {tok_g.tolist()} oracle {oracle.greedy(z_o).tolist()}")
    assert ek.err() <= TOL and ev.err() <= TOL and z_err <= TOL
    for r, t in enumerate(tok_g):
        z = z_o[r].astype(np.float64)
        assert z[t] >= z.max() - TOL * np.max(np.abs(z)), (r, int(t), int(np.argmax(z)))
    arena1.release()


# --------------------------------------------------------------------------
# 32B widths at the longest lengths of the 32B workload (64K keys)
# --------------------------------------------------------------------------
def test_qwen32b_64k_two_layers(oracle_lib):
    """Two layers at 32B widths over a 65,536-token request (the longest the
    32B workload draws) and two short ones: layer-0 K/V of every token and
    layer-1 K/V at sampled positions, i.e. attention over up to 64K keys."""
    shape = W.QWEN32B.with_layers(2)
    wl = W.small_workload(shape, [65536, 300, 17], block_size=16, seed=501, other_live_frac=0.3)
    say(f"qwen32b 2 layers lens={wl.lens.tolist()} NB={wl.num_blocks}")
    model = Hn.device_model_random(shape, seed=502, gain_std=0.1)
    host_w = Hn.host_copy_all(model)
    h0 = {"embed": host_w["embed"], "layer0": host_w["layers"][0]}
    arena = gpu_rebuild_into(wl, model)
    inv = arena.check_invariants()
    say(f"  device invariants {inv}")
    assert inv == {"free_changed": 0, "live_changed": 0, "tail_changed": 0, "written_bad": 0}
    K0, V0 = oracle_layer0(oracle_lib, wl, h0)
    compare_layer0_every_token(arena, wl, K0, V0, "32B 2 layers")
    rng = np.random.default_rng(8)
    samples = [(r, int(p)) for r in range(wl.num_requests)
               for p in sample_positions(int(wl.lens[r]), rng, extra=6 if r == 0 else 2)]
    ora = oracle_arena_with_layer0(wl, shape, K0, V0)
    say(f"  oracle: layer-1 K/V at {len(samples)} sampled positions")
    req, pos, rows = sampled_layer1(oracle_lib, wl, host_w, ora, samples)
    compare_sampled(arena, wl, req, pos, rows, "32B 2 layers")
    arena.release()


# --------------------------------------------------------------------------
# long key loops at a small width, compared in full
# --------------------------------------------------------------------------
def test_tiny_bf16_long_requests_in_full(oracle_lib):
    """Two layers of the small bf16 decoder over requests of 8192 and 4097
    tokens (128 and 65 key tiles, a ragged tail) plus short ones, every
    written K/V element compared with the oracle's full rebuild."""
    shape = W.TINY_BF16.with_layers(2)
    wl = W.small_workload(shape, [8192, 1, 4097, 300, 64], seed=511, other_live_frac=0.25)
    say(f"tiny bf16 2 layers lens={wl.lens.tolist()}")
    host_w = W.host_weights(shape, seed=512, gain_std=0.1)
    image = W.host_arena(wl)
    model = Hn.device_model_from_host(shape, host_w)
    arena = Hn.DeviceArena(wl, host_image=image)
    arena.bind()
    ws, nbytes = Hn.alloc_workspace(shape, wl.num_requests, wl.total_tokens, wl.total_tokens, fill=0xFF)
    kvr.kv_rebuild(model.weights, wl.tokens, wl.lens, wl.block_tables, arena.handle, ws.data_ptr(),
                   nbytes, Hn.stream_ptr())
    torch.cuda.synchronize()
    g = arena.to_host()
    arena.release()
    o = image.copy()
    oracle_lib.rebuild(shape, host_w, wl.tokens, wl.lens, wl.block_tables, o, wl.block_size,
                       wl.num_blocks)
    worst, rep = PU.compare(wl, g, o, image)
    say(f"  worst per-layer K/V error {np.array2string(worst.T, precision=2)}; {rep}")
    assert rep["unwritten_changed"] == 0 and rep["written_nonfinite"] == 0
    assert rep["worst"] <= TOL
