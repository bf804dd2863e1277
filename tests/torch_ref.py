"""Textbook decoder prefill written with PyTorch library primitives
(F.rms_norm, F.linear, F.scaled_dot_product_attention with causal masking and
grouped KV heads, F.silu, rotate-half RoPE), in float64 on the CPU.

It is an independent second implementation used to pin the oracle (it does
not share code with it).  `rounding` selects whether the declared rounding
sites are emulated: None (pure fp64), "f32" or "bf16".
"""
from __future__ import annotations

from typing import Dict, List, Optional, Tuple

import math

import numpy as np
import torch
import torch.nn.functional as F

from paper_2608_14635_amd import workloads as W


def _t(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.asarray(a, dtype=np.float64).copy())


def weights_f64(w: Dict, dtype: int) -> Dict:
    f = W.weights_as_f32(w, dtype) if dtype != W.F64 else w
    return {"embed": _t(f["embed"]), "layers": [{k: _t(v) for k, v in lw.items()} for lw in f["layers"]]}


def _rotate_half(x: torch.Tensor) -> torch.Tensor:
    x1, x2 = x.chunk(2, dim=-1)
    return torch.cat((-x2, x1), dim=-1)


def forward(shape: W.ModelShape, w64: Dict, tokens: np.ndarray,
            rounding: Optional[str] = None, round_p: bool = False
            ) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """One request.  Returns K [L, n, nkv, d], V [L, n, nkv, d] (rounded as
    stored) and the final residual [n, H].  round_p: attention written out
    as softmax weights 2^(z log2 e - c) with c the row max in log2 units
    rounded up, rounded like an op output, then (P V) / sum(P), instead of
    scaled_dot_product_attention."""
    n = len(tokens)
    H, d, nq, nkv = shape.hidden, shape.head_dim, shape.num_q_heads, shape.num_kv_heads

    def work(x):
        return x if rounding is None else x.to(torch.float32).to(torch.float64)

    def rnd(x):
        if rounding is None:
            return x
        x = x.to(torch.float32)
        if rounding == "bf16":
            x = x.to(torch.bfloat16)
        return x.to(torch.float64)

    pos = torch.arange(n, dtype=torch.float64)
    inv_freq = float(shape.rope_theta) ** (-torch.arange(0, d, 2, dtype=torch.float64) / d)
    ang = pos[:, None] * inv_freq[None, :]
    cos, sin = torch.cos(ang), torch.sin(ang)
    if rounding is not None:
        cos, sin = work(cos), work(sin)
    cos = torch.cat((cos, cos), dim=-1)[:, None, :]
    sin = torch.cat((sin, sin), dim=-1)[:, None, :]

    x = work(w64["embed"][torch.as_tensor(tokens, dtype=torch.long)])
    Ks, Vs = [], []
    for lw in w64["layers"]:
        a = rnd(F.rms_norm(x, (H,), weight=lw["attn_norm"], eps=float(shape.rms_eps)))
        q = work(F.linear(a, lw["wq"], lw.get("bq"))).view(n, nq, d)
        k = work(F.linear(a, lw["wk"], lw.get("bk"))).view(n, nkv, d)
        v = work(F.linear(a, lw["wv"], lw.get("bv"))).view(n, nkv, d)
        if getattr(shape, "qk_norm", False):
            q = work(F.rms_norm(q, (d,), weight=lw["q_norm"], eps=float(shape.rms_eps)))
            k = work(F.rms_norm(k, (d,), weight=lw["k_norm"], eps=float(shape.rms_eps)))
        q = rnd(work(q * cos + _rotate_half(q) * sin))
        k = rnd(work(k * cos + _rotate_half(k) * sin))
        v = rnd(v)
        Ks.append(k)
        Vs.append(v)
        if round_p:
            g = nq // nkv
            qh = q.transpose(0, 1)                                   # [nq, n, d]
            kh = k.transpose(0, 1).repeat_interleave(g, dim=0)       # [nq, n, d]
            vh = v.transpose(0, 1).repeat_interleave(g, dim=0)
            z = torch.matmul(qh, kh.transpose(1, 2).contiguous()) / math.sqrt(d)
            z = z.masked_fill(torch.triu(torch.ones(n, n, dtype=torch.bool), 1), float("-inf"))
            # weights relative to a power of two of the row max (log2 units)
            c = torch.ceil(z.amax(dim=-1, keepdim=True) * (1.0 / math.log(2.0)))
            pw = rnd(work(torch.exp2(z * (1.0 / math.log(2.0)) - c)))
            o = (torch.matmul(pw, vh) / pw.sum(dim=-1, keepdim=True))[None]
        else:
            o = F.scaled_dot_product_attention(q.transpose(0, 1)[None], k.transpose(0, 1)[None],
                                               v.transpose(0, 1)[None], is_causal=True,
                                               enable_gqa=True)
        u = rnd(work(o[0].transpose(0, 1).reshape(n, nq * d)))
        x = work(x + work(F.linear(u, lw["wo"])))
        b = rnd(F.rms_norm(x, (H,), weight=lw["ffn_norm"], eps=float(shape.rms_eps)))
        g = work(F.linear(b, lw["w_gate"]))
        up = work(F.linear(b, lw["w_up"]))
        h = rnd(work(F.silu(g) * up))
        x = work(x + work(F.linear(h, lw["w_down"])))
    return torch.stack(Ks), torch.stack(Vs), x


def forward_batch(shape, w64, wl: W.Workload, rounding=None, round_p: bool = False) -> List:
    off = wl.request_offsets()
    out = []
    for r in range(wl.num_requests):
        toks = wl.tokens[off[r]:off[r + 1]]
        if len(toks) == 0:
            out.append(None)
            continue
        out.append(forward(shape, w64, toks, rounding, round_p))
    return out


def logits(shape: W.ModelShape, final_norm: np.ndarray, lm_head: np.ndarray, x: np.ndarray,
           dtype: int, rounding: Optional[str] = None) -> torch.Tensor:
    """Final RMSNorm + LM head of final residual rows x [n, H] (float64 in),
    with the declared rounding of the norm output emulated as in forward()."""
    conv = (lambda a: W.bf16_bits_to_f32(a)) if dtype == W.BF16 else (lambda a: a)
    g, wl = _t(conv(final_norm)), _t(conv(lm_head))
    a = F.rms_norm(_t(x), (shape.hidden,), weight=g, eps=float(shape.rms_eps))
    if rounding is not None:
        a = a.to(torch.float32)
        if rounding == "bf16":
            a = a.to(torch.bfloat16)
        a = a.to(torch.float64)
    z = F.linear(a, wl)
    return z if rounding is None else z.to(torch.float32).to(torch.float64)
