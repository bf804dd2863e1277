"""Python handle on the CPU oracle (oracle/kvo.c).  TEST INFRASTRUCTURE ONLY.

Only tests, the package smoke check and the benchmark's CPU-baseline leg may
import this module.  It compiles kvo.c with gcc (OpenMP, no fast-math, no FMA
contraction) into oracle/libkvo.so and calls it through ctypes.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import time
from typing import Dict, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kvo.c")
_LIB = os.path.join(_HERE, "libkvo.so")

KVO_F32, KVO_BF16, KVO_F64 = 0, 1, 2
_NP = {KVO_F32: np.float32, KVO_BF16: np.uint16, KVO_F64: np.float64}


def build(src: str = _SRC, out: str = _LIB, extra_flags: Sequence[str] = ()) -> str:
    """Compile the oracle (also used by mutation tests on patched copies)."""
    cmd = ["gcc", "-O2", "-std=gnu11", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
           "-fno-fast-math", "-I", _HERE, *extra_flags, src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    os.replace(out + ".tmp", out)
    return out


class _Model(C.Structure):
    _fields_ = [("num_layers", C.c_int32), ("hidden", C.c_int32), ("num_q_heads", C.c_int32),
                ("num_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn_dim", C.c_int32),
                ("vocab", C.c_int32), ("rms_eps", C.c_double), ("rope_theta", C.c_double),
                ("dtype", C.c_int32), ("qk_norm", C.c_int32), ("qkv_bias", C.c_int32),
                ("round_p", C.c_int32)]


_LAYER_KEYS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down",
               "q_norm", "k_norm", "bq", "bk", "bv")
_OPTIONAL = ("q_norm", "k_norm", "bq", "bk", "bv")


class _Layer(C.Structure):
    _fields_ = [(k, C.c_void_p) for k in _LAYER_KEYS]


class _Arena(C.Structure):
    _fields_ = [("base", C.c_void_p), ("block_size", C.c_int32), ("num_blocks", C.c_int64)]


class Oracle:
    """ctypes wrapper around one compiled copy of the oracle."""

    def __init__(self, lib_path: Optional[str] = None):
        path = lib_path or _LIB
        if lib_path is None and (not os.path.exists(path)
                                 or os.path.getmtime(path) < os.path.getmtime(_SRC)):
            build()
        self.lib = C.CDLL(path)
        I32P = C.POINTER(C.c_int32)
        for name in ("kvo_rebuild", "kvo_decode"):
            f = getattr(self.lib, name)
            f.restype = C.c_int
            f.argtypes = [C.POINTER(_Model), C.c_void_p, C.POINTER(_Layer), I32P, I32P, C.c_int32,
                          I32P, C.c_int32, C.POINTER(_Arena), C.c_void_p]
        self.lib.kvo_rebuild_from.restype = C.c_int
        self.lib.kvo_rebuild_from.argtypes = [C.POINTER(_Model), C.c_void_p, C.POINTER(_Layer), I32P,
                                              I32P, I32P, C.c_int32, I32P, C.c_int32,
                                              C.POINTER(_Arena), C.c_void_p]
        self.lib.kvo_decode_step.restype = C.c_int
        self.lib.kvo_decode_step.argtypes = [C.POINTER(_Model), C.c_void_p, C.POINTER(_Layer), I32P,
                                             I32P, C.c_int32, I32P, C.c_int32, C.POINTER(_Arena),
                                             C.c_void_p]
        self.lib.kvo_logits.restype = C.c_int
        self.lib.kvo_logits.argtypes = [C.POINTER(_Model), C.c_void_p, C.c_void_p, C.c_void_p,
                                        C.c_int64, C.c_void_p]
        self.lib.kvo_layer0_kv.restype = C.c_int
        self.lib.kvo_layer0_kv.argtypes = [C.POINTER(_Model), C.c_void_p, C.POINTER(_Layer),
                                           I32P, I32P, C.c_int64, C.c_void_p, C.c_void_p]
        self.lib.kvo_time_layers.restype = C.c_int
        self.lib.kvo_time_layers.argtypes = [C.POINTER(_Model), C.c_void_p, C.POINTER(_Layer),
                                             I32P, C.c_int32, C.c_int32]
        self.lib.kvo_block_digest.restype = C.c_uint64
        self.lib.kvo_block_digest.argtypes = [C.POINTER(_Model), C.POINTER(_Arena), C.c_int64,
                                              C.c_int32, C.POINTER(C.c_int)]
        self.lib.kvo_verify.restype = C.c_int
        self.lib.kvo_verify.argtypes = [C.POINTER(_Model), C.POINTER(_Arena), I32P, C.c_int32, I32P,
                                        C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p]
        self.lib.kvo_round_bf16.restype = C.c_uint16
        self.lib.kvo_round_bf16.argtypes = [C.c_float]
        self.lib.kvo_num_threads.restype = C.c_int

    # -- marshalling -------------------------------------------------
    @staticmethod
    def _model(shape, dtype: Optional[int] = None, num_layers: Optional[int] = None,
               round_p: bool = False) -> _Model:
        return _Model(num_layers if num_layers is not None else shape.num_layers, shape.hidden,
                      shape.num_q_heads, shape.num_kv_heads, shape.head_dim, shape.ffn_dim,
                      shape.vocab, float(shape.rms_eps), float(shape.rope_theta),
                      shape.dtype if dtype is None else dtype,
                      int(getattr(shape, "qk_norm", False)), int(getattr(shape, "qkv_bias", False)),
                      int(round_p))

    @staticmethod
    def _check(a: np.ndarray, dt: int) -> np.ndarray:
        assert a.dtype == _NP[dt] and a.flags.c_contiguous, (a.dtype, dt)
        return a

    def _layers(self, weights: Dict, dt: int):
        arr = (_Layer * len(weights["layers"]))()
        for i, lw in enumerate(weights["layers"]):
            for k, _ in _Layer._fields_:
                if k in _OPTIONAL and k not in lw:
                    continue
                setattr(arr[i], k, self._check(lw[k], dt).ctypes.data)
        return arr

    @staticmethod
    def _i32(a) -> np.ndarray:
        return np.ascontiguousarray(a, dtype=np.int32)

    # -- calls --------------------------------------------------------
    def rebuild(self, shape, weights: Dict, tokens, lens, tables, arena: np.ndarray,
                block_size: int, num_blocks: int, mode: str = "prefill",
                dtype: Optional[int] = None, final_hidden: bool = False, round_p: bool = False):
        """Run the oracle in place on `arena` (raw host array of the dtype).
        Returns the final fp64 hidden state [T, H] when final_hidden is set.
        round_p: attention weights rounded to the dtype before P.V (kvo.h)."""
        dt = shape.dtype if dtype is None else dtype
        m = self._model(shape, dt, round_p=round_p)
        tokens, lens = self._i32(tokens), self._i32(lens)
        tables = self._i32(tables)
        max_blocks = tables.shape[1] if tables.ndim == 2 else 0
        layers = self._layers(weights, dt)
        emb = self._check(weights["embed"], dt)
        need = shape.num_layers * 2 * num_blocks * block_size * shape.num_kv_heads * shape.head_dim
        assert arena.dtype == _NP[dt] or (dt != KVO_F64 and arena.itemsize == np.dtype(_NP[dt]).itemsize)
        assert arena.flags.c_contiguous and arena.size >= need, "arena smaller than its geometry"
        assert tokens.shape[0] == int(lens.sum())
        assert tables.ndim == 2 and tables.shape[0] == len(lens)
        ar = _Arena(arena.ctypes.data, block_size, num_blocks)
        fh = np.zeros((int(lens.sum()), shape.hidden), np.float64) if final_hidden else None
        fn = self.lib.kvo_rebuild if mode == "prefill" else self.lib.kvo_decode
        I32P = C.POINTER(C.c_int32)
        rc = fn(C.byref(m), emb.ctypes.data, layers, tokens.ctypes.data_as(I32P),
                lens.ctypes.data_as(I32P), len(lens), tables.ctypes.data_as(I32P), max_blocks,
                C.byref(ar), fh.ctypes.data if fh is not None else None)
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        return fh

    def rebuild_from(self, shape, weights: Dict, tokens, lens, starts, tables, arena: np.ndarray,
                     block_size: int, num_blocks: int, dtype: Optional[int] = None,
                     final_hidden: bool = False):
        """Recompute positions starts[r] .. lens[r]-1 in place on `arena`, the
        prefixes' K/V being read from it; tokens holds the recomputed
        positions' tokens only (kvo.h defines it)."""
        dt = shape.dtype if dtype is None else dtype
        m = self._model(shape, dt)
        tokens, lens, starts = self._i32(tokens), self._i32(lens), self._i32(starts)
        tables = self._i32(tables)
        max_blocks = tables.shape[1] if tables.ndim == 2 else 0
        layers = self._layers(weights, dt)
        emb = self._check(weights["embed"], dt)
        ar = self._arena(shape, arena, block_size, num_blocks, dt)
        assert tokens.shape[0] == int((lens - starts).sum()) and len(starts) == len(lens)
        nrows = int((lens - starts).sum())
        fh = np.zeros((nrows, shape.hidden), np.float64) if final_hidden else None
        I32P = C.POINTER(C.c_int32)
        rc = self.lib.kvo_rebuild_from(C.byref(m), emb.ctypes.data, layers, tokens.ctypes.data_as(I32P),
                                       lens.ctypes.data_as(I32P), starts.ctypes.data_as(I32P), len(lens),
                                       tables.ctypes.data_as(I32P), max_blocks, C.byref(ar),
                                       fh.ctypes.data if fh is not None else None)
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        return fh

    def decode_step(self, shape, weights: Dict, tokens, positions, tables, arena: np.ndarray,
                    block_size: int, num_blocks: int, dtype: Optional[int] = None,
                    final_hidden: bool = True):
        """One resumed-generation step in place on `arena`: token tokens[r] at
        position positions[r] of request r.  Returns the final fp64 residual
        [R, H] (needed for the logits) when final_hidden is set."""
        dt = shape.dtype if dtype is None else dtype
        m = self._model(shape, dt)
        tokens, positions = self._i32(tokens), self._i32(positions)
        tables = self._i32(tables)
        R = tokens.shape[0]
        assert positions.shape[0] == R and tables.ndim == 2 and tables.shape[0] == R
        need = shape.num_layers * 2 * num_blocks * block_size * shape.num_kv_heads * shape.head_dim
        assert arena.flags.c_contiguous and arena.size >= need, "arena smaller than its geometry"
        ar = _Arena(arena.ctypes.data, block_size, num_blocks)
        fh = np.zeros((R, shape.hidden), np.float64) if final_hidden else None
        I32P = C.POINTER(C.c_int32)
        rc = self.lib.kvo_decode_step(C.byref(m), self._check(weights["embed"], dt).ctypes.data,
                                      self._layers(weights, dt), tokens.ctypes.data_as(I32P),
                                      positions.ctypes.data_as(I32P), R,
                                      tables.ctypes.data_as(I32P), tables.shape[1], C.byref(ar),
                                      fh.ctypes.data if fh is not None else None)
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        return fh

    def logits(self, shape, head: Dict, hidden: np.ndarray, dtype: Optional[int] = None):
        """Final RMSNorm + LM head of rows of the final residual: fp32 [n, vocab]."""
        dt = shape.dtype if dtype is None else dtype
        m = self._model(shape, dt)
        hidden = np.ascontiguousarray(hidden, dtype=np.float64)
        n = hidden.shape[0]
        out = np.zeros((n, shape.vocab), np.float32)
        rc = self.lib.kvo_logits(C.byref(m), self._check(head["final_norm"], dt).ctypes.data,
                                 self._check(head["lm_head"], dt).ctypes.data,
                                 hidden.ctypes.data, n, out.ctypes.data)
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        return out

    def layer0_kv(self, shape, embed: np.ndarray, layer0: Dict, tokens, positions,
                  dtype: Optional[int] = None):
        dt = shape.dtype if dtype is None else dtype
        m = self._model(shape, dt)
        tokens, positions = self._i32(tokens), self._i32(positions)
        n = tokens.shape[0]
        kvd = shape.num_kv_heads * shape.head_dim
        k = np.zeros((n, kvd), _NP[dt])
        v = np.zeros((n, kvd), _NP[dt])
        lay = self._layers({"layers": [layer0]}, dt)
        I32P = C.POINTER(C.c_int32)
        rc = self.lib.kvo_layer0_kv(C.byref(m), self._check(embed, dt).ctypes.data, lay,
                                    tokens.ctypes.data_as(I32P), positions.ctypes.data_as(I32P),
                                    n, k.ctypes.data, v.ctypes.data)
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        return k, v

    def time_layers(self, shape, weights: Dict, tokens, num_layers: int) -> float:
        """Wall time of `num_layers` full layers over one request of len(tokens)."""
        dt = shape.dtype
        m = self._model(shape, dt)
        tokens = self._i32(tokens)
        lay = self._layers(weights, dt)
        I32P = C.POINTER(C.c_int32)
        t0 = time.perf_counter()
        rc = self.lib.kvo_time_layers(C.byref(m), self._check(weights["embed"], dt).ctypes.data,
                                      lay, tokens.ctypes.data_as(I32P), tokens.shape[0], num_layers)
        t1 = time.perf_counter()
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        return t1 - t0

    def _arena(self, shape, arena: np.ndarray, block_size: int, num_blocks: int, dt: int):
        need = shape.num_layers * 2 * num_blocks * block_size * shape.num_kv_heads * shape.head_dim
        assert arena.itemsize == np.dtype(_NP[dt]).itemsize
        assert arena.flags.c_contiguous and arena.size >= need, "arena smaller than its geometry"
        return _Arena(arena.ctypes.data, block_size, num_blocks)

    def block_digest(self, shape, arena: np.ndarray, block_size: int, num_blocks: int, block: int,
                     nslots: int, dtype: Optional[int] = None) -> int:
        """Commit digest of slots [0, nslots) of one block (kvo.h defines it)."""
        dt = shape.dtype if dtype is None else dtype
        m = self._model(shape, dt)
        ar = self._arena(shape, arena, block_size, num_blocks, dt)
        ok = C.c_int()
        v = self.lib.kvo_block_digest(C.byref(m), C.byref(ar), block, nslots, C.byref(ok))
        if ok.value != 0:
            raise ValueError("oracle rejected its arguments")
        return int(v)

    def verify(self, shape, arena: np.ndarray, block_size: int, num_blocks: int, lens, tables,
               committed=None, dtype: Optional[int] = None):
        """(digests [entries] uint64, intact [R] int32): every used block's
        digest, request by request, and the count of leading blocks per request
        whose digest equals `committed` (all zeros when committed is None)."""
        dt = shape.dtype if dtype is None else dtype
        m = self._model(shape, dt)
        ar = self._arena(shape, arena, block_size, num_blocks, dt)
        lens, tables = self._i32(lens), self._i32(tables)
        max_blocks = tables.shape[1] if tables.ndim == 2 else 0
        n = int(sum((int(x) + block_size - 1) // block_size for x in lens))
        dg = np.zeros(max(n, 1), np.uint64)
        com = (np.zeros(max(n, 1), np.uint64) if committed is None
               else np.ascontiguousarray(committed, dtype=np.uint64))
        assert com.size >= n
        intact = np.zeros(max(len(lens), 1), np.int32)
        I32P = C.POINTER(C.c_int32)
        rc = self.lib.kvo_verify(C.byref(m), C.byref(ar), lens.ctypes.data_as(I32P), len(lens),
                                 tables.ctypes.data_as(I32P), max_blocks, com.ctypes.data,
                                 dg.ctypes.data, intact.ctypes.data)
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        return dg[:n], intact[:len(lens)]

    def round_bf16(self, x: float) -> int:
        return int(self.lib.kvo_round_bf16(float(x)))

    def num_threads(self) -> int:
        return int(self.lib.kvo_num_threads())


def greedy(logits: np.ndarray) -> np.ndarray:
    """Greedy next tokens: the lowest index among equal maxima of each row."""
    return np.argmax(np.asarray(logits), axis=-1).astype(np.int32)


_default: Optional[Oracle] = None


def get() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default
