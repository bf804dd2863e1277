"""GPU parity of the resumed decode step (kv_decode_step, through the C ABI)
against the CPU oracle, and the paper's recoverability criterion on the GPU:
generation resumed from a rebuilt arena continues as from the arena the
token-by-token generation built.

Tolerances as for the rebuild: normwise 1e-4 (fp32) / 2e-2 (bf16) on the K/V
rows the step writes and on each request's logits (max |g - o| / max |o|).
The greedy token is an argmax decided on each side in fp32: the GPU's choice
must be a maximum of the oracle's logits up to that tolerance, and every
other arena bit is unchanged by a step."""
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

SHAPES = {
    "tiny_f32": W.TINY_F32,
    "tiny_bf16": W.TINY_BF16,
    # real 8B widths, 2 layers, a reduced vocabulary for the host-side LM head
    "llama8b_2l": dataclasses.replace(W.LLAMA8B.with_layers(2), vocab=2048),
    # the paper's model family: per-head q/k RMSNorm
    "qwen3_8b_2l": dataclasses.replace(W.QWEN3_8B.with_layers(2), vocab=2048),
    # 6 q heads per kv head, q/k/v bias (Qwen2.5 widths)
    "qwen25_1_5b_2l": dataclasses.replace(W.QWEN25_1_5B.with_layers(2), vocab=2048),
    # 16 q heads per kv head
    "g16_bf16": dataclasses.replace(W.TINY_BF16, num_q_heads=32, num_kv_heads=2),
    # a vocabulary of whole 64-row blocks: the LM head runs as a few-row
    # product into row-major logits (the other bf16 vocabularies here take the
    # transposed product)
    "tiny_bf16_v1024": dataclasses.replace(W.TINY_BF16, vocab=1024),
    # two layers of the small decoder, for long contexts the oracle still
    # rebuilds in seconds
    "tiny_bf16_2l": W.TINY_BF16.with_layers(2),
}
# (shape, prefix lengths, block size): the default cases plus block size 32
# and a batch of 40 requests (three 16-row tiles in the few-row products)
CASES = {n: (n, None, 16) for n in SHAPES}
CASES["tiny_bf16_b32"] = ("tiny_bf16", [1, 31, 32, 33, 97], 32)
CASES["tiny_bf16_40req"] = ("tiny_bf16", [1 + (7 * i) % 90 for i in range(40)], 16)
# the row-major LM head with two and three 16-row tiles of requests
CASES["tiny_bf16_v1024_20req"] = ("tiny_bf16_v1024", [1 + (5 * i) % 60 for i in range(20)], 16)
CASES["tiny_bf16_v1024_40req"] = ("tiny_bf16_v1024", [1 + (7 * i) % 90 for i in range(40)], 16)
# the edges of the few-row products: one full 16-row tile, their largest batch
# (64 rows), and one request more (the general split-K path, with the residual
# sum and the norm as separate kernels)
CASES["tiny_bf16_v1024_16req"] = ("tiny_bf16_v1024", [1 + (11 * i) % 70 for i in range(16)], 16)
CASES["tiny_bf16_v1024_64req"] = ("tiny_bf16_v1024", [1 + (13 * i) % 50 for i in range(64)], 16)
CASES["tiny_bf16_v1024_65req"] = ("tiny_bf16_v1024", [1 + (13 * i) % 50 for i in range(65)], 16)
# long contexts: 8192 keys split into 128 ranges of 64 keys (the split's cap),
# a ragged 5000-key context, and 16 requests of 1-2K keys (31 ranges each)
CASES["tiny_bf16_2l_long"] = ("tiny_bf16_2l", [8192, 5000, 1], 16)
CASES["tiny_bf16_2l_16req_1k_2k"] = ("tiny_bf16_2l", [1024 + 61 * i for i in range(16)], 16)


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def resume_workload(shape, prefix_lens, steps, seed, block_size=16):
    """Block tables sized for prefix + steps tokens; tokens and lens hold the prefixes."""
    wl = W.small_workload(shape, [n + steps for n in prefix_lens], block_size=block_size, seed=seed,
                          other_live_frac=0.25)
    offs = wl.request_offsets()
    toks = np.concatenate([wl.tokens[offs[r]:offs[r] + prefix_lens[r]] for r in range(len(prefix_lens))])
    return dataclasses.replace(wl, lens=np.array(prefix_lens, dtype=wl.lens.dtype), tokens=toks)


def split_last(wl):
    """(workload of the prefixes without their last token, last tokens)."""
    offs = wl.request_offsets()
    last = np.array([wl.tokens[offs[r + 1] - 1] for r in range(wl.num_requests)], np.int32)
    toks = np.concatenate([wl.tokens[offs[r]:offs[r + 1] - 1] for r in range(wl.num_requests)])
    return dataclasses.replace(wl, lens=(wl.lens - 1).astype(wl.lens.dtype), tokens=toks), last


class GpuDecoder:
    def __init__(self, wl, model, head_dev, max_position):
        self.wl, self.model, self.head = wl, model, head_dev
        R = wl.num_requests
        self.nbytes = kvr.kv_decode_workspace_bytes(wl.shape, R, max_position)
        self.ws = torch.empty(self.nbytes, dtype=torch.uint8, device="cuda")
        self.next = torch.zeros(R, dtype=torch.int32, device="cuda")
        self.logits = torch.zeros((R, wl.shape.vocab), dtype=torch.float32, device="cuda")

    def step(self, arena, tokens, positions, rows=None, want_logits=True):
        rows = np.arange(self.wl.num_requests) if rows is None else np.asarray(rows)
        n = len(rows)
        kvr.kv_decode_step(self.model.weights, self.head["final_norm"].data_ptr(),
                           self.head["lm_head"].data_ptr(), tokens, positions,
                           self.wl.block_tables[rows], arena.handle, self.ws.data_ptr(), self.nbytes,
                           self.next.data_ptr(), self.logits.data_ptr() if want_logits else 0,
                           Hn.stream_ptr())
        torch.cuda.synchronize()
        return self.next[:n].cpu().numpy().copy(), self.logits[:n].cpu().numpy().copy()


def slot_rows(wl, arena_bits, positions):
    """K/V rows [L, 2, R, nkv*d] at each request's slot for positions[r]."""
    s = wl.shape
    v = arena_bits.reshape(s.num_layers, 2, wl.num_blocks, wl.block_size, s.num_kv_heads * s.head_dim)
    blk = np.array([wl.block_tables[r, p // wl.block_size] for r, p in enumerate(positions)])
    sl = np.array([p % wl.block_size for p in positions])
    return v[:, :, blk, sl]


def rel(g, o):
    g, o = np.asarray(g, np.float64), np.asarray(o, np.float64)
    den = np.max(np.abs(o))
    err = float(np.max(np.abs(g - o)) / (den if den > 0 else 1.0))
    return err if np.isfinite(err) else np.inf  # NaN would vanish in a max() fold


def assert_valid_argmax(gpu_tok, ora_logits, tol):
    for r, t in enumerate(gpu_tok):
        z = ora_logits[r].astype(np.float64)
        assert z[t] >= z.max() - tol * np.max(np.abs(z)), (r, t, int(np.argmax(z)), z[t], z.max())


@pytest.mark.parametrize("name", list(CASES))
def test_decode_step_matches_oracle(oracle_lib, name):
    sname, prefix, B = CASES[name]
    shape = SHAPES[sname]
    tol = PU.TOL[shape.dtype]
    if prefix is None:
        prefix = [1, 6, 23, 300] if sname != "tiny_f32" else [1, 6, 23, 100]
    wl = resume_workload(shape, prefix, steps=2, seed=201, block_size=B)
    pre, last = split_last(wl)
    say(f"[decode parity] {name}: {len(prefix)} prefixes {prefix[:8]}, block size {B}")
    head = W.host_head_weights(shape, seed=42)
    if shape.hidden <= 512:
        host_w = W.host_weights(shape, seed=41, gain_std=0.1)
        model = Hn.device_model_from_host(shape, host_w)
    else:
        model = Hn.device_model_random(shape, seed=41, gain_std=0.1)
        host_w = Hn.host_copy_all(model)
    head_dev = Hn.device_head_from_host(shape, head)
    image = W.host_arena(pre)
    arena = Hn.DeviceArena(pre, host_image=image)
    arena.bind()
    # GPU: rebuild the prefixes without their last token, then one decode step
    ws, nbytes = Hn.alloc_workspace(shape, pre.num_requests, pre.total_tokens, max(pre.total_tokens, 1))
    kvr.kv_rebuild(model.weights, pre.tokens, pre.lens, pre.block_tables, arena.handle, ws.data_ptr(),
                   nbytes, Hn.stream_ptr())
    torch.cuda.synchronize()
    before = arena.to_host()
    pos = (np.array(prefix) - 1).astype(np.int32)
    dec = GpuDecoder(pre, model, head_dev, int(pos.max()) + 1)
    tok_g, z_g = dec.step(arena, last, pos)
    after = arena.to_host()
    # oracle: the same two steps on its own arena
    ora = image.copy()
    oracle_lib.rebuild(shape, host_w, pre.tokens, pre.lens, pre.block_tables, ora, pre.block_size,
                       pre.num_blocks)
    fh = oracle_lib.decode_step(shape, host_w, last, pos, pre.block_tables, ora, pre.block_size,
                                pre.num_blocks)
    z_o = oracle_lib.logits(shape, head, fh)
    # K/V rows of the step
    g_rows, o_rows = slot_rows(pre, after, pos), slot_rows(pre, ora, pos)
    kv_err = rel(PU.to_float(g_rows, shape.dtype), PU.to_float(o_rows, shape.dtype))
    z_err = max(rel(z_g[r], z_o[r]) for r in range(len(prefix)))
    say(f"  step K/V error {kv_err:.2e}, logits error {z_err:.2e} (tol {tol}); "
        f"gpu tokens {tok_g.tolist()} oracle {oracle.greedy(z_o).tolist()}")
    assert kv_err < tol and z_err < tol
    assert_valid_argmax(tok_g, z_o, tol)
    assert np.array_equal(tok_g, np.argmax(z_g, axis=1))
    # nothing but the step's slots changed
    mask = np.ones(before.shape, bool)
    s = shape
    m6 = mask.reshape(s.num_layers, 2, pre.num_blocks, pre.block_size, -1)
    for r, p in enumerate(pos):
        m6[:, :, pre.block_tables[r, p // pre.block_size], p % pre.block_size] = False
    assert np.array_equal(after[mask], before[mask])
    # the same step without a logits buffer: the same tokens, and it rewrites
    # the same K/V rows
    tok_n, _ = dec.step(arena, last, pos, want_logits=False)
    assert np.array_equal(tok_n, tok_g)
    assert np.array_equal(arena.to_host(), after)


@pytest.mark.parametrize("name", ["tiny_f32", "tiny_bf16"])
def test_resume_from_rebuild_equals_decode_built(oracle_lib, name):
    """T-resume: greedy continuations from the rebuilt arena and from an arena
    built token by token with decode steps agree (up to near-ties of the
    logits, after which they may diverge), and so do the arenas."""
    shape = SHAPES[name]
    tol = PU.TOL[shape.dtype]
    steps = 6
    prefix = [1, 6, 23, 50]
    wl = resume_workload(shape, prefix, steps=steps, seed=202)
    pre, last = split_last(wl)
    say(f"[resume] {name}: prefixes {prefix}, {steps} greedy steps")
    host_w = W.host_weights(shape, seed=43, gain_std=0.1)
    head = W.host_head_weights(shape, seed=44)
    model = Hn.device_model_from_host(shape, host_w)
    head_dev = Hn.device_head_from_host(shape, head)
    max_pos = max(prefix) + steps
    dec = GpuDecoder(pre, model, head_dev, max_pos)
    conts = {}
    arenas = {}
    for mode in ("rebuild", "decode"):
        arena = Hn.DeviceArena(pre, host_image=W.host_arena(pre))
        arena.bind()
        if mode == "rebuild":
            ws, nbytes = Hn.alloc_workspace(shape, pre.num_requests, pre.total_tokens,
                                            max(pre.total_tokens, 1))
            kvr.kv_rebuild(model.weights, pre.tokens, pre.lens, pre.block_tables, arena.handle,
                           ws.data_ptr(), nbytes, Hn.stream_ptr())
            torch.cuda.synchronize()
        else:
            offs = pre.request_offsets()
            for p in range(int(pre.lens.max())):
                rows = [r for r in range(pre.num_requests) if p < pre.lens[r]]
                toks = [pre.tokens[offs[r] + p] for r in rows]
                kvr.kv_decode_step(model.weights, head_dev["final_norm"].data_ptr(),
                                   head_dev["lm_head"].data_ptr(), toks, [p] * len(rows),
                                   pre.block_tables[rows], arena.handle, dec.ws.data_ptr(),
                                   dec.nbytes, dec.next.data_ptr(), 0, Hn.stream_ptr())
            torch.cuda.synchronize()
        cur, pos = last.copy(), (np.array(prefix) - 1).astype(np.int32)
        toks, zs = [], []
        for _ in range(steps):
            t, z = dec.step(arena, cur, pos)
            toks.append(t)
            zs.append(z)
            cur, pos = t, pos + 1
        conts[mode] = (np.array(toks), zs)
        arenas[mode] = arena.to_host()
    (ta, za), (tb, zb) = conts["rebuild"], conts["decode"]
    say(f"  rebuild path {ta.T.tolist()}\n  decode path  {tb.T.tolist()}")
    for r in range(pre.num_requests):
        for i in range(steps):
            if ta[i, r] != tb[i, r]:
                z = za[i][r]
                gap = abs(float(z[ta[i, r]]) - float(z[tb[i, r]]))
                say(f"  request {r} diverges at step {i}: logit gap {gap:.3e}")
                assert gap <= tol * np.max(np.abs(z)), "continuations differ without a near-tie"
                break
            assert rel(za[i][r], zb[i][r]) < tol
    # K/V of every prefix position agree between the two arenas within tolerance
    full = dataclasses.replace(pre, lens=pre.lens + 1)
    _, rep = PU.compare(full, arenas["decode"], arenas["rebuild"], arenas["rebuild"])
    say(f"  arenas: {rep}")
    assert rep["written_nonfinite"] == 0 and rep["worst"] < tol
