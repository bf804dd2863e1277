"""Seeded synthetic workloads for the KV rebuild: model shapes, request mixes,
block tables and arena states.

This module holds input generation only (shapes, random draws, fill patterns).
It contains none of the rebuild's arithmetic, so both the HIP path and the CPU
oracle can be fed from it.

The paper evaluates its recovery on Qwen3 4B-32B rollout engines with math
and software-engineering traces (Sec. 7.1, Experiment Setup); those datasets
and weights are not available here, so decoder shapes of public 8B/14B/32B
models with random N(0, 0.02) weights and uniform random tokens stand in for
them. The rebuild itself is the re-prefill of logged token prefixes into a
retained paged KV arena (Sec. 4.2 Handover, step 5; Sec. 4.3 LLM Context
Recovery).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

# dtype codes shared with the C ABI (kv_dtype) and the oracle (kvo dtype)
F32 = 0
BF16 = 1
F64 = 2  # oracle-only pin mode

DTYPE_BYTES = {F32: 4, BF16: 2, F64: 8}
DTYPE_NAME = {F32: "f32", BF16: "bf16", F64: "f64"}

# Sentinel bit patterns for never-written arena slots: signalling NaNs that no
# arithmetic produces, so "written" <=> "differs from the sentinel".
SENTINEL_BITS = {F32: 0x7FA5A5A5, BF16: 0x7FA5}


@dataclasses.dataclass(frozen=True)
class ModelShape:
    num_layers: int
    hidden: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rms_eps: float
    rope_theta: float
    dtype: int
    qk_norm: bool = False    # per-head RMSNorm of q and k before RoPE (Qwen3)
    qkv_bias: bool = False   # biases on the q, k, v projections (Qwen2.5)

    @property
    def elem_bytes(self) -> int:
        return DTYPE_BYTES[self.dtype]

    def with_layers(self, n: int) -> "ModelShape":
        return dataclasses.replace(self, num_layers=n)

    def with_dtype(self, dt: int) -> "ModelShape":
        return dataclasses.replace(self, dtype=dt)

    def kv_row_elems(self) -> int:
        return self.num_kv_heads * self.head_dim

    def weight_elems(self) -> int:
        H, d = self.hidden, self.head_dim
        per_layer = (2 * H + H * (self.num_q_heads + 2 * self.num_kv_heads) * d
                     + self.num_q_heads * d * H + 3 * H * self.ffn_dim)
        return self.vocab * H + self.num_layers * per_layer


# --------------------------------------------------------------------------
# Model shapes
# --------------------------------------------------------------------------
TINY_F32 = ModelShape(2, 256, 4, 4, 64, 688, 1024, 1e-5, 1e4, F32)
LLAMA8B = ModelShape(32, 4096, 32, 8, 128, 14336, 128256, 1e-5, 5e5, BF16)
QWEN14B = ModelShape(48, 5120, 40, 8, 128, 13824, 152064, 1e-6, 1e6, BF16)
QWEN32B = ModelShape(64, 5120, 40, 8, 128, 27648, 152064, 1e-6, 1e6, BF16)
# small bf16 decoder used by fast parity tests: several MFMA tiles per GEMM,
# GQA group 4, head_dim 128 like the real shapes.
TINY_BF16 = ModelShape(4, 512, 8, 2, 128, 1408, 1000, 1e-5, 1e4, BF16)
# The paper's own model families (Sec. 7.1 evaluates Qwen3 4B-32B; Fig. 3 uses
# Qwen2.5-1.5B): public decoder shapes with their attention variants.
QWEN3_8B = ModelShape(36, 4096, 32, 8, 128, 12288, 151936, 1e-6, 1e6, BF16, qk_norm=True)
QWEN3_32B = ModelShape(64, 5120, 64, 8, 128, 25600, 151936, 1e-6, 1e6, BF16, qk_norm=True)
QWEN25_1_5B = ModelShape(28, 1536, 12, 2, 128, 8960, 151936, 1e-6, 1e6, BF16, qkv_bias=True)

SHAPES = {"tiny_f32": TINY_F32, "llama8b": LLAMA8B, "qwen14b": QWEN14B,
          "qwen32b": QWEN32B, "tiny_bf16": TINY_BF16, "qwen3_8b": QWEN3_8B,
          "qwen3_32b": QWEN3_32B, "qwen25_1_5b": QWEN25_1_5B}


@dataclasses.dataclass
class Workload:
    """A synthetic rebuild request batch plus the arena it targets."""
    name: str
    shape: ModelShape
    lens: np.ndarray            # int32 [R]
    tokens: np.ndarray          # int32 [sum(lens)], packed in request order
    block_size: int
    num_blocks: int
    max_blocks: int
    block_tables: np.ndarray    # int32 [R, max_blocks]; unused entries = -1
    other_live: np.ndarray      # int64 ids of blocks holding other requests' KV
    seed: int

    @property
    def total_tokens(self) -> int:
        return int(self.lens.sum())

    @property
    def num_requests(self) -> int:
        return int(self.lens.shape[0])

    def arena_elems(self) -> int:
        s = self.shape
        return s.num_layers * 2 * self.num_blocks * self.block_size * s.kv_row_elems()

    def arena_bytes(self) -> int:
        return self.arena_elems() * self.shape.elem_bytes

    def request_offsets(self) -> np.ndarray:
        off = np.zeros(self.num_requests + 1, dtype=np.int64)
        np.cumsum(self.lens, out=off[1:])
        return off


def config_seed(c: int) -> int:
    return 0x5EED0000 + c


def _blocks_needed(lens: np.ndarray, B: int) -> np.ndarray:
    return (lens.astype(np.int64) + B - 1) // B


def _assign_tables(rng: np.random.Generator, lens: np.ndarray, B: int,
                   free_blocks: np.ndarray, shuffle: bool = True):
    need = _blocks_needed(lens, B)
    max_blocks = max(1, int(need.max()) if len(need) else 1)
    pool = rng.permutation(free_blocks) if shuffle else free_blocks
    assert pool.shape[0] >= need.sum(), "arena too small for the request batch"
    tables = np.full((len(lens), max_blocks), -1, dtype=np.int32)
    o = 0
    for r, k in enumerate(need):
        tables[r, :k] = pool[o:o + k]
        o += int(k)
    return tables, max_blocks


def make_workload(name: str, shape: ModelShape, lens, block_size: int,
                  num_blocks: Optional[int] = None, other_live_frac: float = 0.0,
                  seed: int = 1, token_rows: Optional[List[np.ndarray]] = None,
                  table_mode: str = "random") -> Workload:
    """Generic builder: lens -> tokens, a fragmented arena and block tables.

    Sub-streams are drawn in a fixed order from one PCG64 generator:
    tokens, arena occupancy, block tables.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    lens = np.asarray(lens, dtype=np.int32)
    T = int(lens.sum())
    if token_rows is None:
        tokens = rng.integers(0, shape.vocab, size=T, dtype=np.int64).astype(np.int32)
    else:
        tokens = np.concatenate(token_rows).astype(np.int32) if T else np.zeros(0, np.int32)
        assert tokens.shape[0] == T
    need = int(_blocks_needed(lens, block_size).sum())
    if num_blocks is None:
        num_blocks = max(2 * need, 1)
    all_blocks = np.arange(num_blocks, dtype=np.int64)
    n_live = min(int(other_live_frac * num_blocks), num_blocks - need)
    live = np.sort(rng.choice(num_blocks, size=n_live, replace=False)) if n_live > 0 \
        else np.zeros(0, np.int64)
    free = np.setdiff1d(all_blocks, live)
    if table_mode == "permutation":
        tables, max_blocks = _assign_tables(rng, lens, block_size, free, shuffle=True)
    else:
        tables, max_blocks = _assign_tables(rng, lens, block_size, free, shuffle=True)
    return Workload(name, shape, lens, tokens, block_size, int(num_blocks), int(max_blocks),
                    tables, live.astype(np.int64), seed)


# --------------------------------------------------------------------------
# The five benchmark configurations
# --------------------------------------------------------------------------
def config1() -> Workload:
    """Tiny fp32 decoder: 4 requests of 37/64/100/128 tokens, 64 blocks of 16,
    tables drawn from one random permutation of the 64 blocks."""
    return make_workload("tiny_f32", TINY_F32, [37, 64, 100, 128], 16, num_blocks=64,
                         seed=config_seed(1), table_mode="permutation")


def config2_lens(rng) -> np.ndarray:
    return rng.integers(2048, 16384, size=16, endpoint=True).astype(np.int32)


def config2(shape: ModelShape = LLAMA8B) -> Workload:
    """8B shape, 16 requests with lengths uniform in [2048, 16384], B = 16,
    arena of twice the needed blocks, the rest left at the sentinel."""
    seed = config_seed(2)
    lens = config2_lens(np.random.Generator(np.random.PCG64(seed ^ 0xA5)))
    return make_workload("llama8b_uniform16", shape, lens, 16, seed=seed)


def config3_lens_and_tokens(rng, vocab: int, R: int = 64, cap: int = 32768):
    """Agentic multi-turn mix: a shared 1024-token system segment followed by
    5-20 alternating spans (generated U[64,1024], observation U[128,4096]),
    starting with a generated span, truncated to 32768 tokens."""
    system = rng.integers(0, vocab, size=1024, dtype=np.int64)
    rows, lens = [], []
    for _ in range(R):
        n_spans = int(rng.integers(5, 20, endpoint=True))
        parts = [system]
        for s in range(n_spans):
            ln = int(rng.integers(64, 1024, endpoint=True)) if s % 2 == 0 \
                else int(rng.integers(128, 4096, endpoint=True))
            parts.append(rng.integers(0, vocab, size=ln, dtype=np.int64))
        row = np.concatenate(parts)[:cap]
        rows.append(row.astype(np.int32))
        lens.append(row.shape[0])
    return np.asarray(lens, np.int32), rows


def config3(num_blocks: Optional[int] = None, shape: ModelShape = LLAMA8B) -> Workload:
    """8B shape, 64 agentic requests, half of the arena holding other live
    requests' blocks that must stay bit-identical."""
    seed = config_seed(3)
    lens, rows = config3_lens_and_tokens(np.random.Generator(np.random.PCG64(seed ^ 0xA5)),
                                         shape.vocab)
    need = int(_blocks_needed(lens, 16).sum())
    if num_blocks is None:
        num_blocks = 2 * need
    frac = min(0.5, (num_blocks - need) / num_blocks)
    return make_workload("llama8b_agentic64", shape, lens, 16, num_blocks=num_blocks,
                         other_live_frac=frac, seed=seed, token_rows=rows)


def config4(shape: ModelShape = QWEN14B) -> Workload:
    """14B shape, 32 requests with log-uniform lengths in [512, 32768], B = 32,
    arena of twice the needed blocks with a random half holding other live data."""
    seed = config_seed(4)
    rng = np.random.Generator(np.random.PCG64(seed ^ 0xA5))
    lens = np.floor(np.exp(rng.uniform(math.log(512), math.log(32768), size=32))).astype(np.int32)
    return make_workload("qwen14b_loguniform32", shape, lens, 32, other_live_frac=0.5, seed=seed)


def config5(num_blocks: Optional[int] = None, shape: ModelShape = QWEN32B) -> Workload:
    """32B shape, 8 long requests uniform in [32768, 65536], B = 16, arena
    filling the HBM left after weights and workspace."""
    seed = config_seed(5)
    rng = np.random.Generator(np.random.PCG64(seed ^ 0xA5))
    lens = rng.integers(32768, 65536, size=8, endpoint=True).astype(np.int32)
    return make_workload("qwen32b_long8", shape, lens, 16, num_blocks=num_blocks, seed=seed)


CONFIGS = {1: config1, 2: config2, 3: config3, 4: config4, 5: config5}


def small_workload(shape: ModelShape, lens, block_size: int = 16, seed: int = 7,
                   other_live_frac: float = 0.25, num_blocks: Optional[int] = None) -> Workload:
    """Reduced request sets for parity tests at real layer widths."""
    return make_workload(f"{DTYPE_NAME[shape.dtype]}_small", shape, lens, block_size,
                         num_blocks=num_blocks, other_live_frac=other_live_frac, seed=seed)


# --------------------------------------------------------------------------
# Weights (host, numpy) for oracle-sized shapes
# --------------------------------------------------------------------------
LAYER_KEYS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")


def layer_shapes(s: ModelShape) -> Dict[str, tuple]:
    """Per-layer weight shapes; the variant weights come after the common ones,
    so turning a variant on leaves the draws of the common weights unchanged."""
    H, d = s.hidden, s.head_dim
    out = {"attn_norm": (H,), "wq": (s.num_q_heads * d, H), "wk": (s.num_kv_heads * d, H),
           "wv": (s.num_kv_heads * d, H), "wo": (H, s.num_q_heads * d), "ffn_norm": (H,),
           "w_gate": (s.ffn_dim, H), "w_up": (s.ffn_dim, H), "w_down": (H, s.ffn_dim)}
    if s.qk_norm:
        out.update({"q_norm": (d,), "k_norm": (d,)})
    if s.qkv_bias:
        out.update({"bq": (s.num_q_heads * d,), "bk": (s.num_kv_heads * d,),
                    "bv": (s.num_kv_heads * d,)})
    return out


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16 bit pattern (input-generation helper)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = 0x7FC0
    return r


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _materialize(x32: np.ndarray, dtype: int) -> np.ndarray:
    if dtype == BF16:
        return f32_to_bf16_bits(x32)
    if dtype == F32:
        return x32.astype(np.float32)
    return x32.astype(np.float64)


def host_weights(shape: ModelShape, seed: int = 11, gain_std: float = 0.1,
                 std: float = 0.02) -> Dict:
    """N(0, std) projection/embedding weights drawn in fp32 and rounded to the
    model dtype (uint16 bit patterns for bf16).  Norm gains are 1 + N(0, gain_std)
    (gain_std = 0 gives unit gains, the benchmark setting)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    H = shape.hidden
    emb = rng.standard_normal((shape.vocab, H), dtype=np.float32) * np.float32(std)
    out = {"embed": _materialize(emb, shape.dtype), "layers": []}
    for _ in range(shape.num_layers):
        lw = {}
        for k, shp in layer_shapes(shape).items():
            if k.endswith("norm"):
                g = 1.0 + rng.standard_normal(shp, dtype=np.float32) * np.float32(gain_std)
                lw[k] = _materialize(g.astype(np.float32), shape.dtype)
            else:
                w = rng.standard_normal(shp, dtype=np.float32) * np.float32(std)
                lw[k] = _materialize(w, shape.dtype)
        out["layers"].append(lw)
    return out


def host_head_weights(shape: ModelShape, seed: int = 12, gain_std: float = 0.1,
                      std: float = 0.02) -> Dict:
    """Final RMSNorm gain (1 + N(0, gain_std)) and LM head [vocab, hidden]
    (N(0, std)) for the resumed decode, from their own generator so that the
    decoder weights of host_weights do not change."""
    rng = np.random.Generator(np.random.PCG64(seed))
    g = 1.0 + rng.standard_normal((shape.hidden,), dtype=np.float32) * np.float32(gain_std)
    w = rng.standard_normal((shape.vocab, shape.hidden), dtype=np.float32) * np.float32(std)
    return {"final_norm": _materialize(g.astype(np.float32), shape.dtype),
            "lm_head": _materialize(w, shape.dtype)}


def weights_as_f32(w: Dict, dtype: int) -> Dict:
    """Exact fp32 view of materialized weights (bf16 bits widened)."""
    conv = (lambda a: bf16_bits_to_f32(a)) if dtype == BF16 else (lambda a: a.astype(np.float32))
    return {"embed": conv(w["embed"]),
            "layers": [{k: conv(v) for k, v in lw.items()} for lw in w["layers"]]}


# --------------------------------------------------------------------------
# Arena fill patterns
# --------------------------------------------------------------------------
def live_pattern_bits(dtype: int, block_ids: np.ndarray, elems_per_block: int,
                      layer_kv: int) -> np.ndarray:
    """Finite pseudo-random bit patterns standing in for other live requests'
    KV blocks: a hash of (layer/kv plane, block, element) mapped into +-[1, 2)."""
    b = np.asarray(block_ids, dtype=np.uint64)[:, None]
    e = np.arange(elems_per_block, dtype=np.uint64)[None, :]
    with np.errstate(over="ignore"):  # wrap-around hashing
        h = (b * np.uint64(0x9E3779B97F4A7C15) + e * np.uint64(0xBF58476D1CE4E5B9)
             + np.uint64(layer_kv) * np.uint64(0x94D049BB133111EB))
        h ^= h >> np.uint64(29)
        h *= np.uint64(0xD6E8FEB86659FD93)
        h ^= h >> np.uint64(32)
    if dtype == BF16:
        return (np.uint64(0x3F80) | (h & np.uint64(0x807F))).astype(np.uint16)
    return (np.uint64(0x3F800000) | (h & np.uint64(0x807FFFFF))).astype(np.uint32)


def host_arena(wl: Workload, dtype: Optional[int] = None) -> np.ndarray:
    """Host arena image: sentinel everywhere, other-live blocks patterned.
    Returned as raw bits (uint16 for bf16, uint32 for fp32, float64 for f64)."""
    s = wl.shape
    dt = s.dtype if dtype is None else dtype
    L, NB, B, row = s.num_layers, wl.num_blocks, wl.block_size, s.kv_row_elems()
    if dt == F64:
        a = np.full((L, 2, NB, B * row), np.nan, dtype=np.float64)
        for l in range(L):
            for kv in range(2):
                if wl.other_live.size:
                    bits = live_pattern_bits(F32, wl.other_live, B * row, 2 * l + kv)
                    a[l, kv, wl.other_live] = bits.view(np.float32).astype(np.float64)
        return a.reshape(-1)
    np_t = np.uint16 if dt == BF16 else np.uint32
    a = np.full((L, 2, NB, B * row), SENTINEL_BITS[dt], dtype=np_t)
    for l in range(L):
        for kv in range(2):
            if wl.other_live.size:
                a[l, kv, wl.other_live] = live_pattern_bits(dt, wl.other_live, B * row, 2 * l + kv)
    return a.reshape(-1)
