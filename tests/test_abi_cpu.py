"""C-ABI library checks that need no GPU: it loads, exports every function
the headers declare, sizes workspaces, and rejects invalid requests with the
documented status codes before touching any device."""
import ctypes as C
import dataclasses
import glob
import os
import re

import numpy as np
import pytest

from paper_2608_14635_amd import kvr
from paper_2608_14635_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(kvr.LIB_PATH):
        from paper_2608_14635_amd import build
        build.build()
    return kvr.lib()


def declared_functions():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names.update(re.findall(r"\b(kv_[a-z_]+)\s*\(", text))
    return sorted(names)


def test_exports_every_declared_function(L):
    decl = declared_functions()
    assert len(decl) >= 13
    for name in decl:
        assert hasattr(L, name), f"{name} declared but not exported"
    assert set(decl) == set(kvr.exported_symbols())


def test_workspace_bytes(L):
    s = W.LLAMA8B
    assert kvr.kv_rebuild_workspace_bytes(dataclasses.replace(s, head_dim=64), 4, 1000, 1000) == 0
    a = kvr.kv_rebuild_workspace_bytes(s, 16, 100000, 16384)
    b = kvr.kv_rebuild_workspace_bytes(s, 16, 100000, 65536)
    c = kvr.kv_rebuild_workspace_bytes(s, 16, 200000, 65536)
    assert 0 < a < b < c
    # activations dominate: fp32 residual + bf16 buffers per wave token
    per_tok = 4 * s.hidden + 2 * (s.hidden + 2 * s.num_q_heads * s.head_dim + s.ffn_dim)
    assert b >= 65536 * per_tok


def _valid(shape=W.TINY_BF16, lens=(5, 16, 33), B=16, NB=20, seed=0):
    rng = np.random.default_rng(seed)
    lens = np.array(lens, np.int32)
    toks = rng.integers(0, shape.vocab, size=int(lens.sum())).astype(np.int32)
    need = (lens + B - 1) // B
    perm = rng.permutation(NB).astype(np.int32)
    tables = np.full((len(lens), int(need.max())), -1, np.int32)
    o = 0
    for r, k in enumerate(need):
        tables[r, :k] = perm[o:o + k]
        o += k
    return shape, B, NB, toks, lens, tables


def test_check_accepts_valid(L):
    s, B, NB, toks, lens, tables = _valid()
    assert kvr.kv_rebuild_check(s, B, NB, toks, lens, tables) == kvr.KV_OK


@pytest.mark.parametrize("case,expect", [
    ("token_high", kvr.KV_ERANGE), ("token_negative", kvr.KV_ERANGE),
    ("block_high", kvr.KV_ERANGE), ("block_negative", kvr.KV_ERANGE),
    ("alias_within", kvr.KV_EALIAS), ("alias_across", kvr.KV_EALIAS),
    ("capacity", kvr.KV_ECAPACITY), ("negative_len", kvr.KV_EINVAL),
    ("bad_shape", kvr.KV_EINVAL), ("zero_blocks", kvr.KV_EINVAL),
])
def test_check_errors(L, case, expect):
    s, B, NB, toks, lens, tables = _valid()
    toks, lens, tables = toks.copy(), lens.copy(), tables.copy()
    if case == "token_high":
        toks[7] = s.vocab
    elif case == "token_negative":
        toks[0] = -1
    elif case == "block_high":
        tables[2, 1] = NB
    elif case == "block_negative":
        tables[1, 0] = -5
    elif case == "alias_within":
        tables[2, 2] = tables[2, 0]
    elif case == "alias_across":
        tables[2, 0] = tables[0, 0]
    elif case == "capacity":
        tables = tables[:, :2]
    elif case == "negative_len":
        lens[1] = -1
    elif case == "bad_shape":
        s = dataclasses.replace(s, head_dim=64)
    elif case == "zero_blocks":
        NB = 0
    assert kvr.kv_rebuild_check(s, B, NB, toks, lens, tables) == expect
    assert kvr.kv_last_error() != ""


def test_check_ignores_unused_table_entries(L):
    s, B, NB, toks, lens, tables = _valid()
    wide = np.full((tables.shape[0], tables.shape[1] + 3), 10 ** 6, np.int32)
    wide[:, :tables.shape[1]] = tables
    need = (lens + B - 1) // B
    for r in range(len(lens)):
        wide[r, need[r]:] = 10 ** 6  # garbage past ceil(n / B) is ignored
    assert kvr.kv_rebuild_check(s, B, NB, toks, lens, wide) == kvr.KV_OK


def test_zero_length_requests(L):
    s, B, NB, toks, lens, tables = _valid(lens=(0, 3, 0))
    assert kvr.kv_rebuild_check(s, B, NB, toks, lens, tables) == kvr.KV_OK
    empty = kvr.kv_rebuild_check(s, B, NB, np.zeros(0, np.int32), np.zeros(0, np.int32),
                                 np.zeros((0, 0), np.int32))
    assert empty == kvr.KV_OK


def test_null_pointers(L):
    s, B, NB, toks, lens, tables = _valid()
    d = kvr.make_desc(s)
    i32p = C.POINTER(C.c_int32)
    tab = np.ascontiguousarray(tables)
    st = L.kv_rebuild_check(C.byref(d), B, NB, None, lens.ctypes.data_as(i32p), len(lens),
                            tab.ctypes.data_as(i32p), tab.shape[1])
    assert st == kvr.KV_EINVAL
    st = L.kv_rebuild_check(C.byref(d), B, NB, toks.ctypes.data_as(i32p), None, len(lens),
                            tab.ctypes.data_as(i32p), tab.shape[1])
    assert st == kvr.KV_EINVAL
    assert L.kv_rebuild_check(None, B, NB, None, None, 0, None, 0) == kvr.KV_EINVAL


def test_bind_rejects_bad_arguments_before_device_access(L):
    s = W.TINY_BF16
    need = s.num_layers * 2 * 10 * 16 * s.num_kv_heads * s.head_dim * 2
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_arena_bind(0, need, s, 16, 10)
    assert e.value.status == kvr.KV_EINVAL
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_arena_bind(0x10000, need - 1, s, 16, 10)  # never dereferenced: geometry fails first
    assert e.value.status == kvr.KV_EINVAL
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_arena_bind(0x10000, need, dataclasses.replace(s, dtype=7), 16, 10)
    assert e.value.status == kvr.KV_EINVAL


def test_bind_forced_probe_failure(L, monkeypatch):
    s = W.TINY_BF16
    need = s.num_layers * 2 * 10 * 16 * s.num_kv_heads * s.head_dim * 2
    monkeypatch.setenv("KVR_DEBUG_FAIL_PROBE", "1")
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_arena_bind(0x10000, need, s, 16, 10)
    assert e.value.status == kvr.KV_EDEVICE


def test_unknown_handles_are_rejected(L):
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_arena_release(0x1234)
    assert e.value.status == kvr.KV_ESTATE
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_rebuild_stage(0x1234, [1], [1], [[0]], 0x10000, 1 << 20)
    assert e.value.status == kvr.KV_ESTATE
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_plan_release(0x1234)
    assert e.value.status == kvr.KV_ESTATE


# ---- resumed decode: host-side checks (no device access) -----------------
def _decode_valid(shape=W.TINY_BF16, positions=(0, 15, 40), B=16, NB=12):
    pos = np.array(positions, np.int32)
    toks = (np.arange(len(pos)) * 7 % shape.vocab).astype(np.int32)
    need = pos // B + 1
    mb = int(need.max()) + 1
    tables = np.full((len(pos), mb), -1, np.int32)
    nxt = 0
    for r, n in enumerate(need):
        tables[r, :n] = np.arange(nxt, nxt + n)
        nxt += n
    return shape, toks, pos, tables, B, NB


def test_decode_workspace_bytes(L):
    s = W.LLAMA8B
    assert kvr.kv_decode_workspace_bytes(s, 0, 100) == 0
    assert kvr.kv_decode_workspace_bytes(s, 4, 0) == 0
    a = kvr.kv_decode_workspace_bytes(s, 4, 1000)
    b = kvr.kv_decode_workspace_bytes(s, 4, 65536)
    c = kvr.kv_decode_workspace_bytes(s, 16, 65536)
    assert 0 < a < b < c
    # transposed logits of the LM head: vocab x (requests padded to 256) fp32
    assert a >= s.vocab * 256 * 4


def test_decode_check_valid(L):
    shape, toks, pos, tables, B, NB = _decode_valid()
    assert kvr.kv_decode_check(shape, B, NB, toks, pos, tables) == kvr.KV_OK
    # zero requests is a no-op
    assert kvr.kv_decode_check(shape, B, NB, [], [], np.zeros((0, 0), np.int32)) == kvr.KV_OK


@pytest.mark.parametrize("case,expect", [
    ("negative_position", kvr.KV_EINVAL),
    ("token_out_of_range", kvr.KV_ERANGE),
    ("block_out_of_range", kvr.KV_ERANGE),
    ("needs_more_blocks", kvr.KV_ECAPACITY),
    ("alias_across_requests", kvr.KV_EALIAS),
    ("alias_within_request", kvr.KV_EALIAS),
    ("two_writers_of_one_block", kvr.KV_EALIAS),
])
def test_decode_check_errors(L, case, expect):
    shape, toks, pos, tables, B, NB = _decode_valid()
    if case == "negative_position":
        pos[1] = -1
    elif case == "token_out_of_range":
        toks[2] = shape.vocab
    elif case == "block_out_of_range":
        tables[2, 1] = NB
    elif case == "needs_more_blocks":
        pos[2] = B * tables.shape[1]
    elif case == "alias_across_requests":
        tables[2, 0] = tables[1, 0]
    elif case == "alias_within_request":
        tables[2, 2] = tables[2, 0]
    elif case == "two_writers_of_one_block":
        tables[1, 0] = tables[0, 0]
    assert kvr.kv_decode_check(shape, B, NB, toks, pos, tables) == expect


def test_decode_check_allows_shared_read_only_blocks(L):
    """Full prefix blocks the step only reads may be listed by several
    requests (a shared system prompt), and twice by one request; the block
    each request writes stays exclusive."""
    shape, B, NB = W.TINY_BF16, 16, 12
    pos = np.array([40, 47, 33], np.int32)
    toks = np.array([1, 2, 3], np.int32)
    tables = np.array([[0, 1, 2], [0, 1, 3], [0, 0, 4]], np.int32)
    assert kvr.kv_decode_check(shape, B, NB, toks, pos, tables) == kvr.KV_OK
    tables[2, 2] = 1  # request 2 would write block 1, which requests 0 and 1 read
    assert kvr.kv_decode_check(shape, B, NB, toks, pos, tables) == kvr.KV_EALIAS


def test_decode_check_ignores_unused_entries(L):
    shape, toks, pos, tables, B, NB = _decode_valid()
    tables[0, 1:] = 10 ** 6        # past position 0's block: never read
    assert kvr.kv_decode_check(shape, B, NB, toks, pos, tables) == kvr.KV_OK


def test_decode_step_rejects_unknown_arena(L):
    shape, toks, pos, tables, B, NB = _decode_valid()
    w = kvr.Weights(kvr.make_desc(shape), 0x1000, [{k: 0x1000 for k in kvr.LAYER_FIELDS}] * shape.num_layers)
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_decode_step(w, 0x1000, 0x1000, toks, pos, tables, 0x1234, 0x10000, 1 << 20, 0x2000)
    assert e.value.status == kvr.KV_ESTATE


def _blob(pid: int, device: int = 0) -> bytes:
    h = kvr.kv_ipc_handle()
    h.owner_pid, h.device, h.bytes = pid, device, 4096
    return bytes(h)


def _dead_pid() -> int:
    import subprocess
    import sys
    p = subprocess.Popen([sys.executable, "-c", "pass"])
    p.wait()
    return p.pid


def test_ipc_handle_is_plain_bytes(L):
    assert C.sizeof(kvr.kv_ipc_handle) == 96
    info = kvr.kv_ipc_handle_info(_blob(1234, 3))
    assert info == {"offset": 0, "bytes": 4096, "owner_pid": 1234, "device": 3}
    with pytest.raises(ValueError):
        kvr.kv_ipc_handle_info(b"\0" * 95)


def test_ipc_owner_liveness(L):
    assert kvr.kv_ipc_owner_alive(_blob(os.getpid())) == kvr.KV_OK
    assert kvr.kv_ipc_owner_alive(_blob(os.getppid())) == kvr.KV_OK
    assert kvr.kv_ipc_owner_alive(_blob(_dead_pid())) == kvr.KV_ESTATE
    assert kvr.kv_ipc_owner_alive(_blob(0)) == kvr.KV_EINVAL


def test_ipc_open_refuses_before_device_access(L):
    # a dead owner: the state it held is gone, nothing is mapped
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_ipc_open(_blob(_dead_pid()))
    assert e.value.status == kvr.KV_ESTATE and "gone" in e.value.message
    # the owner itself may not import its own allocation
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_ipc_open(_blob(os.getpid()))
    assert e.value.status == kvr.KV_EINVAL
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_ipc_close(0x1000)
    assert e.value.status == kvr.KV_ESTATE
    assert L.kv_ipc_export(None, 16, None) == kvr.KV_EINVAL


def test_ipc_export_refuses_two_gib_before_device_access(L):
    """Handles are limited to allocations below 2 GiB; a range of 2 GiB or more
    is refused on the host, before HIP is asked about the pointer."""
    h = kvr.kv_ipc_handle()
    assert L.kv_ipc_export(C.c_void_p(0x1000), 2 << 30, C.byref(h)) == kvr.KV_EINVAL
    assert "2 GiB" in kvr.kv_last_error()
    assert L.kv_ipc_export(C.c_void_p(0x1000), (2 << 30) + 4096, C.byref(h)) == kvr.KV_EINVAL


def test_verify_workspace_bytes(L):
    assert kvr.kv_verify_workspace_bytes(-1, 5) == 0 and kvr.kv_verify_workspace_bytes(2, -1) == 0
    a = kvr.kv_verify_workspace_bytes(4, 100)
    b = kvr.kv_verify_workspace_bytes(4, 1000)
    assert 0 < a < b and b >= 1000 * (8 + 1 + 8)
    assert kvr.num_entries([0, 1, 16, 17, 33], 16) == 0 + 1 + 1 + 2 + 3


def test_verify_rejects_unknown_arena_and_null_records(L):
    lens, tables = np.array([3, 20], np.int32), np.zeros((2, 2), np.int32)
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_block_digests(0x1234, lens, tables, 0x10000, 1 << 20, 0x2000)
    assert e.value.status == kvr.KV_ESTATE
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_verify(0x1234, lens, tables, 0, 0x10000, 1 << 20, 0x3000)
    assert e.value.status == kvr.KV_EINVAL and "committed" in e.value.message
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_verify(0x1234, lens, tables, 0x4000, 0x10000, 1 << 20, 0x3000)
    assert e.value.status == kvr.KV_ESTATE


def _from_valid(B=16):
    shape = W.TINY_BF16
    lens = np.array([40, 64, 0, 17], np.int32)
    starts = np.array([32, 16, 0, 8], np.int32)
    NB = 20
    rng = np.random.default_rng(3)
    tables = np.full((4, 4), -1, np.int32)
    nxt = 0
    for r, n in enumerate(lens):
        for j in range((n + B - 1) // B):
            tables[r, j] = nxt
            nxt += 1
    toks = rng.integers(0, shape.vocab, size=int((lens - starts).sum())).astype(np.int32)
    return shape, toks, lens, starts, tables, B, NB


def test_rebuild_from_workspace_bytes(L):
    s = W.LLAMA8B
    a = kvr.kv_rebuild_from_workspace_bytes(s, 4, 1000, 1000, 1000)
    b = kvr.kv_rebuild_from_workspace_bytes(s, 4, 1000, 9000, 1000)
    assert 0 < a < b
    assert kvr.kv_rebuild_from_workspace_bytes(s, 4, 1000, 999, 1000) == 0
    # with no prefix it sizes like the plain rebuild's workspace at one wave
    assert a >= kvr.kv_rebuild_workspace_bytes(s, 4, 1000, 1000)


def test_rebuild_from_check(L):
    shape, toks, lens, starts, tables, B, NB = _from_valid()
    assert kvr.kv_rebuild_from_check(shape, B, NB, toks, lens, starts, tables) == kvr.KV_OK
    # starts = 0 is the plain rebuild's check
    full = np.concatenate([np.arange(n) % shape.vocab for n in lens]).astype(np.int32)
    assert kvr.kv_rebuild_from_check(shape, B, NB, full, lens, np.zeros(4, np.int32), tables) == kvr.KV_OK
    assert kvr.kv_rebuild_check(shape, B, NB, full, lens, tables) == kvr.KV_OK
    bad = starts.copy(); bad[0] = 41          # past the length
    assert kvr.kv_rebuild_from_check(shape, B, NB, toks, lens, bad, tables) == kvr.KV_EINVAL
    bad = starts.copy(); bad[1] = 12          # not a multiple of 8
    assert kvr.kv_rebuild_from_check(shape, B, NB, toks, lens, bad, tables) == kvr.KV_EINVAL
    bad = starts.copy(); bad[3] = 17          # = length: nothing to compute, any value allowed
    assert kvr.kv_rebuild_from_check(shape, B, NB, toks[:-9], lens, bad, tables) == kvr.KV_OK
    # a prefix block may be shared read-only, also with an earlier writer
    t = tables.copy(); t[1, 0] = tables[0, 0]  # request 1 reads request 0's first block
    assert kvr.kv_rebuild_from_check(shape, B, NB, toks, lens, starts, t) == kvr.KV_OK
    t = tables.copy(); t[0, 0] = tables[3, 1]  # request 0 reads what request 3 writes later
    assert kvr.kv_rebuild_from_check(shape, B, NB, toks, lens, starts, t) == kvr.KV_EALIAS
    t = tables.copy(); t[1, 1] = tables[0, 2]  # two writers
    assert kvr.kv_rebuild_from_check(shape, B, NB, toks, lens, starts, t) == kvr.KV_EALIAS
    t = tables.copy(); t[0, 0] = NB            # out of range, read-only block included
    assert kvr.kv_rebuild_from_check(shape, B, NB, toks, lens, starts, t) == kvr.KV_ERANGE
    assert L.kv_rebuild_from_check(C.byref(kvr.make_desc(shape)), B, NB, None, None, None, 1, None, 4) == kvr.KV_EINVAL
