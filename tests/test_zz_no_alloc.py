"""The allocation-free verification (kv_verify_noalloc, include/kvr_verify.h)
against kv_verify with a workspace, through the C ABI: digests and
leading-intact counts are integer results, so they must be bit-identical.
Two calls in a row share the library's scratch array, the second over a
smaller request set; a call needing more scratch than the array holds is
refused before any device work."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_14635_amd import harness as Hn  # noqa: E402
from paper_2608_14635_amd import kvr  # noqa: E402
from paper_2608_14635_amd import workloads as W  # noqa: E402

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def fill_random(arena, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    flat = arena.bits.view(-1)
    flat.copy_(torch.randint(-(1 << 15), 1 << 15, (flat.numel(),), generator=g, device="cuda",
                             dtype=flat.dtype))


def with_workspace(arena, lens, tables, B, committed):
    E = kvr.num_entries(lens, B)
    nbytes = kvr.kv_verify_workspace_bytes(len(lens), E)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda")
    dg = torch.full((max(E, 1),), -1, dtype=torch.int64, device="cuda")
    intact = torch.full((len(lens),), -5, dtype=torch.int32, device="cuda")
    kvr.kv_verify(arena.handle, lens, tables, committed.data_ptr(), ws.data_ptr(), nbytes,
                  intact.data_ptr(), dg.data_ptr(), Hn.stream_ptr())
    torch.cuda.synchronize()
    return dg[:E].cpu().numpy(), intact.cpu().numpy()


def without_workspace(arena, lens, tables, B, committed, want_digests=True):
    E = kvr.num_entries(lens, B)
    dg = torch.full((max(E, 1),), -1, dtype=torch.int64, device="cuda")
    intact = torch.full((len(lens),), -5, dtype=torch.int32, device="cuda")
    kvr.kv_verify_noalloc(arena.handle, lens, tables, committed.data_ptr(), intact.data_ptr(),
                          dg.data_ptr() if want_digests else 0, Hn.stream_ptr())
    torch.cuda.synchronize()
    return (dg[:E].cpu().numpy() if want_digests else None), intact.cpu().numpy()


def test_verify_noalloc_matches_verify_with_workspace():
    shape = W.TINY_BF16.with_layers(2)
    lens = [1, 300, 0, 17, 64, 1000, 33, 255]
    B = 16
    wl = W.small_workload(shape, lens, block_size=B, seed=601, other_live_frac=0.2)
    say(f"[noalloc] {len(lens)} requests {lens}, {wl.num_blocks} blocks")
    arena = Hn.DeviceArena(wl)
    arena.bind()
    fill_random(arena, 7)
    E = kvr.num_entries(wl.lens, B)
    nbytes = kvr.kv_verify_workspace_bytes(wl.num_requests, E)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda")
    committed = torch.zeros(E, dtype=torch.int64, device="cuda")
    kvr.kv_block_digests(arena.handle, wl.lens, wl.block_tables, ws.data_ptr(), nbytes,
                         committed.data_ptr(), Hn.stream_ptr())
    torch.cuda.synchronize()
    # damage: one word in request 1's third block, one in request 5's first
    for r, j in ((1, 2), (5, 0)):
        blk = int(wl.block_tables[r, j])
        arena.bits[1, 0, blk, 3, 0, 5] ^= 1
    torch.cuda.synchronize()

    # call 1: the whole set
    dg_w, in_w = with_workspace(arena, wl.lens, wl.block_tables, B, committed)
    dg_n, in_n = without_workspace(arena, wl.lens, wl.block_tables, B, committed)
    say(f"  call 1: intact {in_n.tolist()} (with workspace {in_w.tolist()})")
    assert np.array_equal(dg_n, dg_w) and np.array_equal(in_n, in_w)
    nb = (wl.lens + B - 1) // B
    assert in_n[1] == 2 and in_n[5] == 0 and in_n[3] == nb[3]

    # call 2: a smaller set (three requests, their own entries of the commit records)
    sel = [5, 1, 6]
    offs = np.concatenate([[0], np.cumsum(nb)])
    com2 = torch.cat([committed[offs[r]:offs[r + 1]] for r in sel])
    lens2, tab2 = wl.lens[sel], wl.block_tables[sel]
    dg_w2, in_w2 = with_workspace(arena, lens2, tab2, B, com2)
    dg_n2, in_n2 = without_workspace(arena, lens2, tab2, B, com2)
    say(f"  call 2: intact {in_n2.tolist()} (with workspace {in_w2.tolist()})")
    assert np.array_equal(dg_n2, dg_w2) and np.array_equal(in_n2, in_w2)
    assert in_n2.tolist() == [0, 2, int(nb[6])]

    # the digests kept in the scratch array when the caller takes none
    _, in_n3 = without_workspace(arena, wl.lens, wl.block_tables, B, committed, want_digests=False)
    assert np.array_equal(in_n3, in_w)

    # more scratch than the array holds: refused on the host
    big = np.zeros((1, kvr.KV_VERIFY_NOALLOC_SCRATCH_BYTES // 4 + 1), np.int32)
    intact = torch.zeros(1, dtype=torch.int32, device="cuda")
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_verify_noalloc(arena.handle, [B], big, committed.data_ptr(), intact.data_ptr())
    assert e.value.status == kvr.KV_ENOMEM and "scratch" in e.value.message
    arena.release()
