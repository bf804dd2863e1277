"""Thin ctypes binding of libkvr.so (include/kvr.h, include/kvr_decode.h,
include/kvr_ipc.h, include/kvr_verify.h, include/kvr_reuse.h, include/kvr_profile.h).

Argument marshalling only: every step of the rebuild runs in the library's
HIP kernels.  Device buffers are passed as integer addresses (for example a
torch tensor's data_ptr()), host arrays as numpy int32 arrays, streams as the
integer value of a hipStream_t (torch.cuda.Stream.cuda_stream).  Errors raise
KvError carrying the library's status code and message.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Iterable, Optional, Sequence, Tuple

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libkvr.so")

KV_OK, KV_EINVAL, KV_ERANGE, KV_EALIAS, KV_ECAPACITY, KV_EDEVICE, KV_ENOMEM, KV_ESTATE = \
    0, -1, -2, -3, -4, -5, -6, -7
STATUS_NAMES = {0: "KV_OK", -1: "KV_EINVAL", -2: "KV_ERANGE", -3: "KV_EALIAS", -4: "KV_ECAPACITY",
                -5: "KV_EDEVICE", -6: "KV_ENOMEM", -7: "KV_ESTATE"}
KV_F32, KV_BF16 = 0, 1
PROF_CLASSES = ("rope", "norm", "gemm_qkv", "attention", "gemm_o", "gemm_gateup", "gemm_down")
LAYER_FIELDS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down",
                "q_norm", "k_norm", "bq", "bk", "bv")
OPTIONAL_FIELDS = ("q_norm", "k_norm", "bq", "bk", "bv")


class KvError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


class kv_model_desc(C.Structure):
    _fields_ = [("num_layers", C.c_int32), ("hidden", C.c_int32), ("num_q_heads", C.c_int32),
                ("num_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn_dim", C.c_int32),
                ("vocab", C.c_int32), ("rms_eps", C.c_double), ("rope_theta", C.c_double),
                ("dtype", C.c_int32), ("qk_norm", C.c_int32), ("qkv_bias", C.c_int32)]


class kv_layer_weights(C.Structure):
    _fields_ = [(k, C.c_void_p) for k in LAYER_FIELDS]


class kv_weights(C.Structure):
    _fields_ = [("desc", kv_model_desc), ("embed", C.c_void_p),
                ("layers", C.POINTER(kv_layer_weights))]


class kv_ipc_handle(C.Structure):
    _fields_ = [("ipc", C.c_uint8 * 64), ("offset", C.c_uint64), ("bytes", C.c_uint64),
                ("owner_pid", C.c_int64), ("device", C.c_int32), ("reserved", C.c_int32)]


_lib: Optional[C.CDLL] = None


def lib() -> C.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2608_14635_amd.build` (there is no fallback path)")
    L = C.CDLL(LIB_PATH)
    i32p = C.POINTER(C.c_int32)
    vp = C.c_void_p
    L.kv_last_error.restype = C.c_char_p
    L.kv_rebuild_workspace_bytes.restype = C.c_uint64
    L.kv_rebuild_workspace_bytes.argtypes = [C.POINTER(kv_model_desc), C.c_int32, C.c_int64, C.c_int64]
    L.kv_rebuild_check.restype = C.c_int
    L.kv_rebuild_check.argtypes = [C.POINTER(kv_model_desc), C.c_int32, C.c_int64, i32p, i32p,
                                   C.c_int32, i32p, C.c_int32]
    L.kv_arena_bind.restype = C.c_int
    L.kv_arena_bind.argtypes = [vp, C.c_uint64, C.POINTER(kv_model_desc), C.c_int32, C.c_int64,
                                C.c_int32, C.POINTER(vp)]
    L.kv_arena_release.restype = C.c_int
    L.kv_arena_release.argtypes = [vp]
    L.kv_rebuild.restype = C.c_int
    L.kv_rebuild.argtypes = [C.POINTER(kv_weights), i32p, i32p, C.c_int32, i32p, C.c_int32, vp,
                             vp, C.c_uint64, vp]
    L.kv_rebuild_stage.restype = C.c_int
    L.kv_rebuild_stage.argtypes = [vp, i32p, i32p, C.c_int32, i32p, C.c_int32, vp, C.c_uint64, vp,
                                   C.POINTER(vp)]
    L.kv_rebuild_execute.restype = C.c_int
    L.kv_rebuild_execute.argtypes = [C.POINTER(kv_weights), vp, vp]
    L.kv_plan_release.restype = C.c_int
    L.kv_plan_release.argtypes = [vp]
    L.kv_plan_info.restype = C.c_int
    L.kv_plan_info.argtypes = [vp, C.POINTER(C.c_int32), C.POINTER(C.c_int64)]
    L.kv_decode_workspace_bytes.restype = C.c_uint64
    L.kv_decode_workspace_bytes.argtypes = [C.POINTER(kv_model_desc), C.c_int32, C.c_int64]
    L.kv_decode_check.restype = C.c_int
    L.kv_decode_check.argtypes = [C.POINTER(kv_model_desc), C.c_int32, C.c_int64, i32p, i32p,
                                  C.c_int32, i32p, C.c_int32]
    L.kv_decode_step.restype = C.c_int
    L.kv_decode_step.argtypes = [C.POINTER(kv_weights), vp, vp, i32p, i32p, C.c_int32, i32p,
                                 C.c_int32, vp, vp, C.c_uint64, vp, vp, vp]
    L.kv_rebuild_from_workspace_bytes.restype = C.c_uint64
    L.kv_rebuild_from_workspace_bytes.argtypes = [C.POINTER(kv_model_desc), C.c_int32, C.c_int64,
                                                  C.c_int64, C.c_int64]
    L.kv_rebuild_from_check.restype = C.c_int
    L.kv_rebuild_from_check.argtypes = [C.POINTER(kv_model_desc), C.c_int32, C.c_int64, i32p, i32p,
                                        i32p, C.c_int32, i32p, C.c_int32]
    L.kv_rebuild_from.restype = C.c_int
    L.kv_rebuild_from.argtypes = [C.POINTER(kv_weights), i32p, i32p, i32p, C.c_int32, i32p, C.c_int32,
                                  vp, vp, C.c_uint64, vp]
    L.kv_rebuild_stage_from.restype = C.c_int
    L.kv_rebuild_stage_from.argtypes = [vp, i32p, i32p, i32p, C.c_int32, i32p, C.c_int32, vp,
                                        C.c_uint64, vp, C.POINTER(vp)]
    L.kv_verify_workspace_bytes.restype = C.c_uint64
    L.kv_verify_workspace_bytes.argtypes = [C.c_int32, C.c_int64]
    L.kv_block_digests.restype = C.c_int
    L.kv_block_digests.argtypes = [vp, i32p, C.c_int32, i32p, C.c_int32, vp, C.c_uint64, vp, vp]
    L.kv_verify.restype = C.c_int
    L.kv_verify.argtypes = [vp, i32p, C.c_int32, i32p, C.c_int32, vp, vp, C.c_uint64, vp, vp, vp]
    L.kv_verify_noalloc.restype = C.c_int
    L.kv_verify_noalloc.argtypes = [vp, i32p, C.c_int32, i32p, C.c_int32, vp, vp, vp, vp]
    hp = C.POINTER(kv_ipc_handle)
    L.kv_ipc_export.restype = C.c_int
    L.kv_ipc_export.argtypes = [vp, C.c_uint64, hp]
    L.kv_ipc_owner_alive.restype = C.c_int
    L.kv_ipc_owner_alive.argtypes = [hp]
    L.kv_ipc_open.restype = C.c_int
    L.kv_ipc_open.argtypes = [hp, C.POINTER(vp)]
    L.kv_ipc_close.restype = C.c_int
    L.kv_ipc_close.argtypes = [vp]
    L.kv_profile_enable.restype = C.c_int
    L.kv_profile_enable.argtypes = [vp, C.c_int32]
    L.kv_profile_read.restype = C.c_int
    L.kv_profile_read.argtypes = [vp, C.POINTER(C.c_double), C.POINTER(C.c_int64),
                                  C.POINTER(C.c_double), C.c_int32]
    L.kv_profile_reset.restype = C.c_int
    L.kv_profile_reset.argtypes = [vp]
    _lib = L
    return L


def kv_last_error() -> str:
    return lib().kv_last_error().decode()


def _check(st: int) -> None:
    if st != KV_OK:
        raise KvError(st, kv_last_error())


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(C.POINTER(C.c_int32)) if a.size else None


def make_desc(shape) -> kv_model_desc:
    """kv_model_desc from any object with the ModelShape fields."""
    return kv_model_desc(shape.num_layers, shape.hidden, shape.num_q_heads, shape.num_kv_heads,
                         shape.head_dim, shape.ffn_dim, shape.vocab, float(shape.rms_eps),
                         float(shape.rope_theta), int(shape.dtype),
                         int(getattr(shape, "qk_norm", False)), int(getattr(shape, "qkv_bias", False)))


class Weights:
    """Owns the ctypes kv_weights struct and its host layer array."""

    def __init__(self, desc: kv_model_desc, embed_ptr: int, layer_ptrs: Sequence[Dict[str, int]]):
        self._layers = (kv_layer_weights * len(layer_ptrs))()
        for i, lp in enumerate(layer_ptrs):
            for k in LAYER_FIELDS:
                if k in OPTIONAL_FIELDS and k not in lp:
                    continue
                setattr(self._layers[i], k, lp[k])
        self.c = kv_weights(desc, embed_ptr, C.cast(self._layers, C.POINTER(kv_layer_weights)))


def _tables2d(tables, n_req: int) -> Tuple[np.ndarray, int]:
    t = _i32(tables)
    if t.ndim != 2:
        t = t.reshape(n_req, -1) if n_req else t.reshape(0, 0)
    return t, int(t.shape[1]) if t.ndim == 2 else 0


def kv_rebuild_workspace_bytes(shape_or_desc, num_requests: int, total_tokens: int,
                               wave_tokens: int) -> int:
    d = shape_or_desc if isinstance(shape_or_desc, kv_model_desc) else make_desc(shape_or_desc)
    return int(lib().kv_rebuild_workspace_bytes(C.byref(d), num_requests, total_tokens, wave_tokens))


def kv_rebuild_check(shape_or_desc, block_size: int, num_blocks: int, tokens, lens, tables) -> int:
    """Host-only validation; returns the status code (no exception)."""
    d = shape_or_desc if isinstance(shape_or_desc, kv_model_desc) else make_desc(shape_or_desc)
    tok, ln = _i32(tokens), _i32(lens)
    tab, mb = _tables2d(tables, len(ln))
    return int(lib().kv_rebuild_check(C.byref(d), block_size, num_blocks, _ptr(tok), _ptr(ln),
                                      len(ln), _ptr(tab), mb))


def kv_arena_bind(base: int, nbytes: int, shape_or_desc, block_size: int, num_blocks: int,
                  device: int = 0) -> int:
    d = shape_or_desc if isinstance(shape_or_desc, kv_model_desc) else make_desc(shape_or_desc)
    h = C.c_void_p()
    _check(lib().kv_arena_bind(C.c_void_p(base), nbytes, C.byref(d), block_size, num_blocks,
                               device, C.byref(h)))
    return h.value


def kv_arena_release(arena: int) -> None:
    _check(lib().kv_arena_release(C.c_void_p(arena)))


def kv_rebuild(weights: Weights, tokens, lens, tables, arena: int, workspace: int,
               workspace_bytes: int, stream: int = 0) -> None:
    tok, ln = _i32(tokens), _i32(lens)
    tab, mb = _tables2d(tables, len(ln))
    _check(lib().kv_rebuild(C.byref(weights.c), _ptr(tok), _ptr(ln), len(ln), _ptr(tab), mb,
                            C.c_void_p(arena), C.c_void_p(workspace), workspace_bytes,
                            C.c_void_p(stream)))


def kv_rebuild_stage(arena: int, tokens, lens, tables, workspace: int, workspace_bytes: int,
                     stream: int = 0) -> int:
    tok, ln = _i32(tokens), _i32(lens)
    tab, mb = _tables2d(tables, len(ln))
    plan = C.c_void_p()
    _check(lib().kv_rebuild_stage(C.c_void_p(arena), _ptr(tok), _ptr(ln), len(ln), _ptr(tab), mb,
                                  C.c_void_p(workspace), workspace_bytes, C.c_void_p(stream),
                                  C.byref(plan)))
    return plan.value


def kv_rebuild_execute(weights: Weights, plan: int, stream: int = 0) -> None:
    _check(lib().kv_rebuild_execute(C.byref(weights.c), C.c_void_p(plan), C.c_void_p(stream)))


def kv_plan_release(plan: int) -> None:
    _check(lib().kv_plan_release(C.c_void_p(plan)))


def kv_plan_info(plan: int) -> Tuple[int, int]:
    nw, mx = C.c_int32(), C.c_int64()
    _check(lib().kv_plan_info(C.c_void_p(plan), C.byref(nw), C.byref(mx)))
    return nw.value, mx.value


def kv_rebuild_from_workspace_bytes(shape_or_desc, num_requests: int, total_rows: int,
                                    total_keys: int, wave_rows: int) -> int:
    d = shape_or_desc if isinstance(shape_or_desc, kv_model_desc) else make_desc(shape_or_desc)
    return int(lib().kv_rebuild_from_workspace_bytes(C.byref(d), num_requests, total_rows, total_keys,
                                                     wave_rows))


def kv_rebuild_from_check(shape_or_desc, block_size: int, num_blocks: int, tokens, lens, starts,
                          tables) -> int:
    """Host-only validation of a rebuild from retained prefixes; the status code."""
    d = shape_or_desc if isinstance(shape_or_desc, kv_model_desc) else make_desc(shape_or_desc)
    tok, ln, st = _i32(tokens), _i32(lens), _i32(starts)
    tab, mb = _tables2d(tables, len(ln))
    return int(lib().kv_rebuild_from_check(C.byref(d), block_size, num_blocks, _ptr(tok), _ptr(ln),
                                           _ptr(st), len(ln), _ptr(tab), mb))


def kv_rebuild_from(weights: Weights, tokens, lens, starts, tables, arena: int, workspace: int,
                    workspace_bytes: int, stream: int = 0) -> None:
    """Recompute positions starts[r] .. lens[r]-1; tokens are those positions' tokens only."""
    tok, ln, st = _i32(tokens), _i32(lens), _i32(starts)
    tab, mb = _tables2d(tables, len(ln))
    _check(lib().kv_rebuild_from(C.byref(weights.c), _ptr(tok), _ptr(ln), _ptr(st), len(ln), _ptr(tab),
                                 mb, C.c_void_p(arena), C.c_void_p(workspace), workspace_bytes,
                                 C.c_void_p(stream)))


def kv_rebuild_stage_from(arena: int, tokens, lens, starts, tables, workspace: int,
                          workspace_bytes: int, stream: int = 0) -> int:
    tok, ln, st = _i32(tokens), _i32(lens), _i32(starts)
    tab, mb = _tables2d(tables, len(ln))
    plan = C.c_void_p()
    _check(lib().kv_rebuild_stage_from(C.c_void_p(arena), _ptr(tok), _ptr(ln), _ptr(st), len(ln),
                                       _ptr(tab), mb, C.c_void_p(workspace), workspace_bytes,
                                       C.c_void_p(stream), C.byref(plan)))
    return plan.value


def kv_decode_workspace_bytes(shape_or_desc, num_requests: int, max_position: int) -> int:
    d = shape_or_desc if isinstance(shape_or_desc, kv_model_desc) else make_desc(shape_or_desc)
    return int(lib().kv_decode_workspace_bytes(C.byref(d), num_requests, max_position))


def kv_decode_check(shape_or_desc, block_size: int, num_blocks: int, tokens, positions,
                    tables) -> int:
    """Host-only validation of a decode step; returns the status code."""
    d = shape_or_desc if isinstance(shape_or_desc, kv_model_desc) else make_desc(shape_or_desc)
    tok, pos = _i32(tokens), _i32(positions)
    tab, mb = _tables2d(tables, len(tok))
    return int(lib().kv_decode_check(C.byref(d), block_size, num_blocks, _ptr(tok), _ptr(pos),
                                     len(tok), _ptr(tab), mb))


def kv_decode_step(weights: Weights, final_norm: int, lm_head: int, tokens, positions, tables,
                   arena: int, workspace: int, workspace_bytes: int, next_tokens: int,
                   logits: int = 0, stream: int = 0) -> None:
    """One greedy decode step; next_tokens / logits are device addresses."""
    tok, pos = _i32(tokens), _i32(positions)
    tab, mb = _tables2d(tables, len(tok))
    _check(lib().kv_decode_step(C.byref(weights.c), C.c_void_p(final_norm), C.c_void_p(lm_head),
                                _ptr(tok), _ptr(pos), len(tok), _ptr(tab), mb, C.c_void_p(arena),
                                C.c_void_p(workspace), workspace_bytes, C.c_void_p(stream),
                                C.c_void_p(next_tokens), C.c_void_p(logits or None)))


def num_entries(lens, block_size: int) -> int:
    """Blocks a request set occupies: sum of ceil(len / block_size)."""
    ln = _i32(lens).astype(np.int64)
    return int(((ln + block_size - 1) // block_size).sum())


def kv_verify_workspace_bytes(num_requests: int, entries: int) -> int:
    return int(lib().kv_verify_workspace_bytes(num_requests, entries))


def kv_block_digests(arena: int, lens, tables, workspace: int, workspace_bytes: int, digests: int,
                     stream: int = 0) -> None:
    """Commit digests (device uint64 [entries]) of every block the requests occupy."""
    ln = _i32(lens)
    tab, mb = _tables2d(tables, len(ln))
    _check(lib().kv_block_digests(C.c_void_p(arena), _ptr(ln), len(ln), _ptr(tab), mb,
                                  C.c_void_p(workspace), workspace_bytes, C.c_void_p(stream),
                                  C.c_void_p(digests)))


def kv_verify(arena: int, lens, tables, committed: int, workspace: int, workspace_bytes: int,
              intact: int, digests: int = 0, stream: int = 0) -> None:
    """Per request, the count of leading blocks matching their committed digests
    (device int32 [R] at `intact`); current digests optionally at `digests`."""
    ln = _i32(lens)
    tab, mb = _tables2d(tables, len(ln))
    _check(lib().kv_verify(C.c_void_p(arena), _ptr(ln), len(ln), _ptr(tab), mb,
                           C.c_void_p(committed), C.c_void_p(workspace), workspace_bytes,
                           C.c_void_p(stream), C.c_void_p(digests or None), C.c_void_p(intact)))


# bytes of device scratch the allocation-free verification holds per device
KV_VERIFY_NOALLOC_SCRATCH_BYTES = 16 << 20


def kv_verify_noalloc(arena: int, lens, tables, committed: int, intact: int, digests: int = 0,
                      stream: int = 0) -> None:
    """kv_verify without a workspace: its scratch is the library's own device
    array (callers that cannot allocate)."""
    ln = _i32(lens)
    tab, mb = _tables2d(tables, len(ln))
    _check(lib().kv_verify_noalloc(C.c_void_p(arena), _ptr(ln), len(ln), _ptr(tab), mb,
                                   C.c_void_p(committed), C.c_void_p(stream),
                                   C.c_void_p(digests or None), C.c_void_p(intact)))


def kv_ipc_export(ptr: int, nbytes: int) -> bytes:
    """Owner side: the handle of device memory [ptr, ptr+nbytes) as plain bytes."""
    h = kv_ipc_handle()
    _check(lib().kv_ipc_export(C.c_void_p(ptr), nbytes, C.byref(h)))
    return bytes(h)


def _handle(blob: bytes) -> kv_ipc_handle:
    if len(blob) != C.sizeof(kv_ipc_handle):
        raise ValueError(f"an IPC handle is {C.sizeof(kv_ipc_handle)} bytes, got {len(blob)}")
    return kv_ipc_handle.from_buffer_copy(blob)


def kv_ipc_handle_info(blob: bytes) -> Dict[str, int]:
    h = _handle(blob)
    return {"offset": h.offset, "bytes": h.bytes, "owner_pid": h.owner_pid, "device": h.device}


def kv_ipc_owner_alive(blob: bytes) -> int:
    """Status code: KV_OK when the owner process exists, KV_ESTATE when it is gone."""
    h = _handle(blob)
    return int(lib().kv_ipc_owner_alive(C.byref(h)))


def kv_ipc_open(blob: bytes) -> int:
    """Importer side: the device address the owner exported."""
    h = _handle(blob)
    p = C.c_void_p()
    _check(lib().kv_ipc_open(C.byref(h), C.byref(p)))
    return p.value


def kv_ipc_close(ptr: int) -> None:
    _check(lib().kv_ipc_close(C.c_void_p(ptr)))


def kv_profile_enable(arena: int, enable: bool = True) -> None:
    _check(lib().kv_profile_enable(C.c_void_p(arena), 1 if enable else 0))


def kv_profile_read(arena: int) -> Dict[str, Dict[str, float]]:
    n = len(PROF_CLASSES)
    ms, la, fl = (C.c_double * n)(), (C.c_int64 * n)(), (C.c_double * n)()
    _check(lib().kv_profile_read(C.c_void_p(arena), ms, la, fl, n))
    return {name: {"ms": ms[i], "launches": int(la[i]), "flops": fl[i]}
            for i, name in enumerate(PROF_CLASSES)}


def kv_profile_reset(arena: int) -> None:
    _check(lib().kv_profile_reset(C.c_void_p(arena)))


def exported_symbols() -> Iterable[str]:
    return ("kv_arena_bind", "kv_arena_release", "kv_rebuild_workspace_bytes", "kv_rebuild_check",
            "kv_rebuild", "kv_rebuild_stage", "kv_rebuild_execute", "kv_plan_release",
            "kv_plan_info", "kv_last_error", "kv_profile_enable", "kv_profile_read",
            "kv_profile_reset", "kv_decode_workspace_bytes", "kv_decode_check", "kv_decode_step",
            "kv_ipc_export", "kv_ipc_owner_alive", "kv_ipc_open", "kv_ipc_close",
            "kv_verify_workspace_bytes", "kv_block_digests", "kv_verify", "kv_verify_noalloc",
            "kv_rebuild_from_workspace_bytes", "kv_rebuild_from_check", "kv_rebuild_from",
            "kv_rebuild_stage_from")
