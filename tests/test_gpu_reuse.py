"""Rebuild from a retained prefix on the GPU (include/kvr_reuse.h) against the
oracle's kvo_rebuild_from: positions start..len-1 recomputed, the prefix K/V
read from the arena.  Tolerances as for the rebuild (normwise per layer, K|V,
kv head); prefix slots, untouched blocks and tail slots bit-exact; and with
starts on multiples of 64 (where the attention's query grouping matches the
full rebuild's) the result is the full rebuild's, bit for bit."""
import dataclasses
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_14635_amd import harness as Hn  # noqa: E402
from paper_2608_14635_amd import kvr  # noqa: E402
from paper_2608_14635_amd import workloads as W  # noqa: E402

import parity_util as PU  # noqa: E402

pytestmark = pytest.mark.gpu
LLAMA8B_2L = W.LLAMA8B.with_layers(2)
# workspaces start as all-ones bytes (NaN in bf16 and fp32), so that a read of
# an element no kernel wrote shows up as a non-finite result, whatever the
# caching allocator handed back
POISON = 0xFF


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def piece(wl, lo, hi):
    offs = wl.request_offsets()
    parts = [wl.tokens[offs[r] + int(lo[r]):offs[r] + int(hi[r])] for r in range(wl.num_requests)]
    return np.concatenate(parts).astype(np.int32) if parts else np.zeros(0, np.int32)


def model_for(shape, seed):
    if shape.hidden <= 512:
        host_w = W.host_weights(shape, seed=seed, gain_std=0.1)
        return Hn.device_model_from_host(shape, host_w), host_w
    model = Hn.device_model_random(shape, seed=seed, gain_std=0.1)
    return model, Hn.host_copy_all(model)


def gpu_from(model, wl, arena, tokens, lens, starts, tables):
    rows = int((np.asarray(lens) - np.asarray(starts)).sum())
    keys = int(np.asarray(lens).sum())
    nbytes = kvr.kv_rebuild_from_workspace_bytes(wl.shape, len(lens), rows, keys, max(rows, 1))
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda").fill_(POISON)
    kvr.kv_rebuild_from(model.weights, tokens, lens, starts, tables, arena.handle, ws.data_ptr(),
                        nbytes, Hn.stream_ptr())
    torch.cuda.synchronize()


def gpu_full(model, wl, arena, tokens, lens, tables):
    T = int(np.asarray(lens).sum())
    ws, nbytes = Hn.alloc_workspace(wl.shape, len(lens), T, max(T, 1), fill=POISON)
    kvr.kv_rebuild(model.weights, tokens, lens, tables, arena.handle, ws.data_ptr(), nbytes,
                   Hn.stream_ptr())
    torch.cuda.synchronize()


CASES = {
    "tiny_bf16": (W.TINY_BF16, [300, 129, 64, 0, 255, 40], [64, 72, 64, 0, 128, 8], 16),
    "tiny_f32": (W.TINY_F32, [100, 33, 64], [64, 24, 8], 16),
    "llama8b_2l": (LLAMA8B_2L, [1, 300, 520, 17], [0, 256, 200, 16], 16),
    "qwen3_8b_2l_b32": (W.QWEN3_8B.with_layers(2), [333, 64, 129], [128, 32, 96], 32),
}


@pytest.mark.parametrize("name", list(CASES))
def test_rebuild_from_matches_oracle(oracle_lib, name):
    shape, lens, starts, B = CASES[name]
    wl = W.small_workload(shape, lens, block_size=B, seed=601, other_live_frac=0.25)
    starts = np.array(starts, np.int32)
    zero = np.zeros_like(starts)
    say(f"[rebuild from] {name}: lens {lens} starts {starts.tolist()} B {B}")
    model, host_w = model_for(shape, 602)
    image = W.host_arena(wl)
    # GPU: the prefixes first, then the rest from them
    arena = Hn.DeviceArena(wl, host_image=image)
    arena.bind()
    if starts.sum():
        gpu_full(model, wl, arena, piece(wl, zero, starts), starts, wl.block_tables)
    before = arena.to_host().copy()
    gpu_from(model, wl, arena, piece(wl, starts, wl.lens), wl.lens, starts, wl.block_tables)
    got = arena.to_host()
    # oracle: its own prefixes first, then the same call over them
    ora = image.copy()
    if starts.sum():
        oracle_lib.rebuild(shape, host_w, piece(wl, zero, starts), starts, wl.block_tables, ora, B,
                           wl.num_blocks)
    oracle_lib.rebuild_from(shape, host_w, piece(wl, starts, wl.lens), wl.lens, starts, wl.block_tables,
                            ora, B, wl.num_blocks)
    worst, rep = PU.compare(wl, got, ora, image)
    say(f"  vs oracle: worst {worst.max():.2e}; {rep}")
    assert rep["unwritten_changed"] == 0 and rep["written_nonfinite"] == 0
    assert rep["worst"] <= PU.TOL[shape.dtype]
    # prefix slots untouched, bit for bit
    v = shape.num_layers, 2, wl.num_blocks, B, -1
    gb, bb = got.reshape(v), before.reshape(v)
    for r, s0 in enumerate(starts):
        for p in range(int(s0)):
            blk, sl = wl.block_tables[r, p // B], p % B
            assert np.array_equal(gb[:, :, blk, sl], bb[:, :, blk, sl]), (r, p)
    # the full rebuild, bit for bit where the starts are on multiples of 64
    full = Hn.DeviceArena(wl, host_image=image)
    full.bind()
    gpu_full(model, wl, full, wl.tokens, wl.lens, wl.block_tables)
    fh = full.to_host().reshape(v)
    for r, s0 in enumerate(starts):
        if s0 % 64 == 0:
            for p in range(int(wl.lens[r])):
                blk, sl = wl.block_tables[r, p // B], p % B
                assert np.array_equal(gb[:, :, blk, sl], fh[:, :, blk, sl]), (name, r, p)
    arena.release()
    full.release()


def test_shared_prefix_blocks_in_one_call(oracle_lib):
    """A leader request computes a shared 128-token prefix; followers list the
    leader's prefix blocks read-only and start after them, all in one call:
    equal to the oracle on the same tables, and each follower's own positions
    equal to a full rebuild of it on its own blocks, bit for bit."""
    shape, B, S = W.TINY_BF16, 16, 128
    lens = [200, 150, 128, 300]
    wl = W.small_workload(shape, lens, block_size=B, seed=611, other_live_frac=0.25)
    offs = wl.request_offsets()
    toks = wl.tokens.copy()
    for r in range(1, wl.num_requests):
        toks[offs[r]:offs[r] + S] = toks[:S]
    wl = dataclasses.replace(wl, tokens=toks)
    shared = wl.block_tables.copy()
    for r in range(1, wl.num_requests):
        shared[r, :S // B] = wl.block_tables[0, :S // B]
    starts = np.array([0] + [S] * (wl.num_requests - 1), np.int32)
    model, host_w = model_for(shape, 612)
    image = W.host_arena(wl)
    arena = Hn.DeviceArena(wl, host_image=image)
    arena.bind()
    say(f"[shared prefix] lens {lens}, {S} shared tokens in the leader's blocks")
    assert kvr.kv_rebuild_from_check(shape, B, wl.num_blocks, piece(wl, starts, wl.lens), wl.lens,
                                     starts, shared) == kvr.KV_OK
    gpu_from(model, wl, arena, piece(wl, starts, wl.lens), wl.lens, starts, shared)
    got = arena.to_host()
    ora = image.copy()
    oracle_lib.rebuild_from(shape, host_w, piece(wl, starts, wl.lens), wl.lens, starts, shared, ora, B,
                            wl.num_blocks)
    swl = dataclasses.replace(wl, block_tables=shared)
    worst, rep = PU.compare(swl, got, ora, image)
    say(f"  vs oracle: worst {worst.max():.2e}; {rep}")
    assert rep["written_nonfinite"] == 0 and rep["worst"] <= PU.TOL[shape.dtype]
    full = Hn.DeviceArena(wl, host_image=image)
    full.bind()
    gpu_full(model, wl, full, wl.tokens, wl.lens, wl.block_tables)
    v = shape.num_layers, 2, wl.num_blocks, B, -1
    gb, fh = got.reshape(v), full.to_host().reshape(v)
    for r in range(wl.num_requests):
        for p in range(int(wl.lens[r])):
            g = gb[:, :, shared[r, p // B], p % B]
            f = fh[:, :, wl.block_tables[r, p // B], p % B]
            assert np.array_equal(g, f), (r, p)
    arena.release()
    full.release()


def test_decode_after_shared_prefix_rebuild(oracle_lib):
    """Generation resumes over an arena whose requests share prefix blocks: one
    decode step per request lists the shared blocks read-only and writes its
    own last block; step K/V rows and logits match the oracle's step over the
    oracle's arena, every greedy token is a maximum of the oracle's logits."""
    shape, B, S = W.TINY_BF16, 16, 128
    lens = [200, 150, 300]
    wl = W.small_workload(shape, lens, block_size=B, seed=613, other_live_frac=0.25)
    offs = wl.request_offsets()
    toks = wl.tokens.copy()
    for r in range(1, wl.num_requests):
        toks[offs[r]:offs[r] + S] = toks[:S]
    wl = dataclasses.replace(wl, tokens=toks)
    shared = wl.block_tables.copy()
    for r in range(1, wl.num_requests):
        shared[r, :S // B] = wl.block_tables[0, :S // B]
    starts = np.array([0] + [S] * (wl.num_requests - 1), np.int32)
    model, host_w = model_for(shape, 614)
    head = W.host_head_weights(shape, seed=615)
    head_dev = Hn.device_head_from_host(shape, head)
    image = W.host_arena(wl)
    arena = Hn.DeviceArena(wl, host_image=image)
    arena.bind()
    say(f"[decode after shared prefix] lens {lens}, {S} shared tokens")
    gpu_from(model, wl, arena, piece(wl, starts, wl.lens), wl.lens, starts, shared)
    rebuilt = arena.to_host().copy()
    ora = image.copy()
    oracle_lib.rebuild_from(shape, host_w, piece(wl, starts, wl.lens), wl.lens, starts, shared, ora, B,
                            wl.num_blocks)
    # one step per request: its last token again at its last position
    pos = (wl.lens - 1).astype(np.int32)
    last = np.array([toks[offs[r + 1] - 1] for r in range(wl.num_requests)], np.int32)
    assert kvr.kv_decode_check(shape, B, wl.num_blocks, last, pos, shared) == kvr.KV_OK
    R = wl.num_requests
    nbytes = kvr.kv_decode_workspace_bytes(shape, R, int(pos.max()) + 1)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    nxt = torch.zeros(R, dtype=torch.int32, device="cuda")
    logits = torch.zeros((R, shape.vocab), dtype=torch.float32, device="cuda")
    kvr.kv_decode_step(model.weights, head_dev["final_norm"].data_ptr(), head_dev["lm_head"].data_ptr(),
                       last, pos, shared, arena.handle, ws.data_ptr(), nbytes, nxt.data_ptr(),
                       logits.data_ptr(), Hn.stream_ptr())
    torch.cuda.synchronize()
    got = arena.to_host()
    fh = oracle_lib.decode_step(shape, host_w, last, pos, shared, ora, B, wl.num_blocks)
    z_o = oracle_lib.logits(shape, head, fh)
    z_g = logits.cpu().numpy()
    v = shape.num_layers, 2, wl.num_blocks, B, -1
    blk, sl = shared[np.arange(R), pos // B], pos % B
    g_rows = PU.to_float(got.reshape(v)[:, :, blk, sl], shape.dtype).astype(np.float64)
    o_rows = PU.to_float(ora.reshape(v)[:, :, blk, sl], shape.dtype).astype(np.float64)
    kv_err = float(np.max(np.abs(g_rows - o_rows)) / np.max(np.abs(o_rows)))
    z_err = max(float(np.max(np.abs(z_g[r] - z_o[r])) / np.max(np.abs(z_o[r]))) for r in range(R))
    tol = PU.TOL[shape.dtype]
    say(f"  step K/V error {kv_err:.2e}, logits error {z_err:.2e}")
    assert kv_err <= tol and z_err <= tol
    for r, t in enumerate(nxt.cpu().numpy()):
        z = z_o[r].astype(np.float64)
        assert z[t] >= z.max() - tol * np.max(np.abs(z)), (r, int(t), int(np.argmax(z)))
    # the shared prefix blocks are read, never written
    pref = shared[0, :S // B]
    assert np.array_equal(got.reshape(v)[:, :, pref], rebuilt.reshape(v)[:, :, pref])
    arena.release()


def test_partial_recovery_from_first_damaged_block(oracle_lib):
    """Flush-free recovery at block granularity: commit digests after a full
    rebuild, damage blocks of two requests, verify, and rebuild each damaged
    request from its first damaged block only.  With 64-slot blocks the
    starts are multiples of 64, so the recovered arena reproduces the
    committed digests exactly."""
    shape, B = W.TINY_BF16, 64
    lens = [300, 129, 64, 255]
    wl = W.small_workload(shape, lens, block_size=B, seed=621, other_live_frac=0.25)
    model, host_w = model_for(shape, 622)
    arena = Hn.DeviceArena(wl, host_image=W.host_arena(wl))
    arena.bind()
    gpu_full(model, wl, arena, wl.tokens, wl.lens, wl.block_tables)
    reference = arena.to_host().copy()
    E = kvr.num_entries(wl.lens, B)
    vb = kvr.kv_verify_workspace_bytes(wl.num_requests, E)
    vws = torch.empty(max(vb, 256), dtype=torch.uint8, device="cuda")
    committed = torch.empty(E, dtype=torch.int64, device="cuda")
    intact = torch.empty(wl.num_requests, dtype=torch.int32, device="cuda")
    kvr.kv_block_digests(arena.handle, wl.lens, wl.block_tables, vws.data_ptr(), vb, committed.data_ptr(),
                         Hn.stream_ptr())
    arena.bits[1, 1, int(wl.block_tables[0, 3]), 5] = 0          # request 0, block 3
    arena.bits[0, 0, int(wl.block_tables[3, 2]), 0, 1, :8] = 7   # request 3, block 2
    kvr.kv_verify(arena.handle, wl.lens, wl.block_tables, committed.data_ptr(), vws.data_ptr(), vb,
                  intact.data_ptr(), 0, Hn.stream_ptr())
    torch.cuda.synchronize()
    got = intact.cpu().numpy()
    nb = (wl.lens + B - 1) // B
    say(f"[partial recovery] intact blocks {got.tolist()} of {nb.tolist()}")
    assert got.tolist() == [3, nb[1], nb[2], 2]
    starts = (np.minimum(got, nb) * B).clip(max=wl.lens).astype(np.int32)
    gpu_from(model, wl, arena, piece(wl, starts, wl.lens), wl.lens, starts, wl.block_tables)
    assert np.array_equal(arena.to_host(), reference), "recovered arena differs from the full rebuild"
    kvr.kv_verify(arena.handle, wl.lens, wl.block_tables, committed.data_ptr(), vws.data_ptr(), vb,
                  intact.data_ptr(), 0, Hn.stream_ptr())
    torch.cuda.synchronize()
    assert np.array_equal(intact.cpu().numpy(), nb)
    arena.release()


def test_rebuild_from_errors_leave_arena_untouched():
    shape = W.TINY_BF16
    wl = W.small_workload(shape, [40, 33], seed=631, other_live_frac=0.25)
    model, _ = model_for(shape, 632)
    image = W.host_arena(wl)
    arena = Hn.DeviceArena(wl, host_image=image)
    arena.bind()
    starts = np.array([8, 12], np.int32)   # 12: not a multiple of 8
    with pytest.raises(kvr.KvError) as e:
        gpu_from(model, wl, arena, piece(wl, starts, wl.lens), wl.lens, starts, wl.block_tables)
    assert e.value.status == kvr.KV_EINVAL
    assert np.array_equal(arena.to_host(), image)
    arena.release()
