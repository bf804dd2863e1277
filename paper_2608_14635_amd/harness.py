"""Device-side plumbing shared by the benchmark, the smoke check and the GPU
tests: allocating weights, arenas and workspaces with torch, seeded fills of
the arena (sentinel and other-live patterns), and arena invariant checks.

Nothing here computes any part of the rebuild; PyTorch only provides device
memory and streams.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np
import torch

from . import kvr
from . import workloads as W

_TORCH_BITS = {W.BF16: torch.int16, W.F32: torch.int32}
_TORCH_VAL = {W.BF16: torch.bfloat16, W.F32: torch.float32}


def _signed(bits: int, dt: int) -> int:
    width = 16 if dt == W.BF16 else 32
    return bits - (1 << width) if bits >= (1 << (width - 1)) else bits


@dataclasses.dataclass
class DeviceModel:
    shape: W.ModelShape
    embed: torch.Tensor
    layers: List[Dict[str, torch.Tensor]]
    weights: kvr.Weights


def _bind_weights(shape, embed, layers) -> kvr.Weights:
    ptrs = [{k: t.data_ptr() for k, t in lw.items()} for lw in layers]
    return kvr.Weights(kvr.make_desc(shape), embed.data_ptr(), ptrs)


def device_model_from_host(shape: W.ModelShape, host_w: Dict, device="cuda") -> DeviceModel:
    """Copy materialized host weights (workloads.host_weights) to the device."""
    def up(a):
        t = torch.from_numpy(np.ascontiguousarray(a))
        if shape.dtype == W.BF16:
            t = t.view(torch.int16).view(torch.bfloat16)
        return t.to(device)
    embed = up(host_w["embed"])
    layers = [{k: up(v) for k, v in lw.items()} for lw in host_w["layers"]]
    return DeviceModel(shape, embed, layers, _bind_weights(shape, embed, layers))


def device_model_random(shape: W.ModelShape, seed: int = 1234, device="cuda",
                        std: float = 0.02, gain_std: float = 0.0) -> DeviceModel:
    """N(0, std) weights drawn on the device (fp32, rounded to the dtype) and
    norm gains 1 + N(0, gain_std) (unit gains by default, the benchmark
    setting); used for the full-size configurations."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    dt = _TORCH_VAL[shape.dtype]

    def rnd(*shp):
        out = torch.empty(*shp, dtype=dt, device=device)
        flat = out.view(-1)
        chunk = 1 << 26
        for i in range(0, flat.numel(), chunk):
            n = min(chunk, flat.numel() - i)
            flat[i:i + n] = (torch.randn(n, generator=g, device=device, dtype=torch.float32) * std).to(dt)
        return out

    embed = rnd(shape.vocab, shape.hidden)
    layers = []
    for _ in range(shape.num_layers):
        lw = {}
        for k, shp in W.layer_shapes(shape).items():
            if k.endswith("norm"):
                gn = torch.randn(*shp, generator=g, device=device, dtype=torch.float32)
                lw[k] = (1.0 + gn * gain_std).to(dt)
            else:
                lw[k] = rnd(*shp)
        layers.append(lw)
    return DeviceModel(shape, embed, layers, _bind_weights(shape, embed, layers))


def model_view(shape: W.ModelShape, embed: torch.Tensor, layers: List[Dict[str, torch.Tensor]]) -> DeviceModel:
    """A model over existing device tensors (an embedding table and layer weights)."""
    return DeviceModel(shape, embed, layers, _bind_weights(shape, embed, layers))


def upload(shape: W.ModelShape, a: np.ndarray, device="cuda") -> torch.Tensor:
    """A host array in oracle format (bf16 bits or fp32) as a device tensor of the model dtype."""
    t = torch.from_numpy(np.ascontiguousarray(a))
    if shape.dtype == W.BF16:
        t = t.view(torch.int16).view(torch.bfloat16)
    return t.to(device)


def first_layers(model: DeviceModel, n: int) -> DeviceModel:
    """The same device weights seen as an n-layer model (its first n layers)."""
    shape = model.shape.with_layers(n)
    layers = model.layers[:n]
    return DeviceModel(shape, model.embed, layers, _bind_weights(shape, model.embed, layers))


def device_head_from_host(shape: W.ModelShape, head: Dict, device="cuda") -> Dict[str, torch.Tensor]:
    """Final-norm gain and LM head of the resumed decode (workloads.host_head_weights) on the device."""
    out = {}
    for k, a in head.items():
        t = torch.from_numpy(np.ascontiguousarray(a))
        if shape.dtype == W.BF16:
            t = t.view(torch.int16).view(torch.bfloat16)
        out[k] = t.to(device)
    return out


def device_head_random(shape: W.ModelShape, seed: int = 4321, device="cuda",
                       std: float = 0.02) -> Dict[str, torch.Tensor]:
    """Unit final-norm gain and an N(0, std) LM head drawn on the device."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    dt = _TORCH_VAL[shape.dtype]
    lm = torch.empty(shape.vocab, shape.hidden, dtype=dt, device=device)
    flat = lm.view(-1)
    chunk = 1 << 26
    for i in range(0, flat.numel(), chunk):
        n = min(chunk, flat.numel() - i)
        flat[i:i + n] = (torch.randn(n, generator=g, device=device, dtype=torch.float32) * std).to(dt)
    return {"final_norm": torch.ones(shape.hidden, dtype=dt, device=device), "lm_head": lm}


def _down(model: DeviceModel, t: torch.Tensor) -> np.ndarray:
    if model.shape.dtype == W.BF16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def host_copy_all(model: DeviceModel) -> Dict:
    """All weights back on the host in oracle format (small models only)."""
    return {"embed": _down(model, model.embed),
            "layers": [{k: _down(model, v) for k, v in lw.items()} for lw in model.layers]}


def host_copy_head(model: DeviceModel, head: Dict[str, torch.Tensor]) -> Dict:
    """Final-norm gain and LM head back on the host in oracle format."""
    return {k: _down(model, v) for k, v in head.items()}


def host_copy_layer(model: DeviceModel, l: int) -> Dict:
    """Layer l's weights back on the host in oracle format."""
    return {k: _down(model, v) for k, v in model.layers[l].items()}


def host_copy_layer0(model: DeviceModel) -> Dict:
    """Layer-0 weights and embedding back on the host in oracle format."""
    def down(t):
        if model.shape.dtype == W.BF16:
            return t.view(torch.int16).cpu().numpy().view(np.uint16)
        return t.cpu().numpy()
    return {"embed": down(model.embed), "layer0": {k: down(v) for k, v in model.layers[0].items()}}


# --------------------------------------------------------------------------
# Arena
# --------------------------------------------------------------------------
class DeviceArena:
    """Arena tensor in the paged layout [L, 2, NB, B, nkv, d] (raw bits)."""

    def __init__(self, wl: W.Workload, device="cuda", host_image: Optional[np.ndarray] = None,
                 progress=None):
        s = wl.shape
        self.wl = wl
        self.dt = s.dtype
        self.shape6 = (s.num_layers, 2, wl.num_blocks, wl.block_size, s.num_kv_heads, s.head_dim)
        bits_t = _TORCH_BITS[self.dt]
        # other-live blocks of a host image keep a device copy for the checks;
        # device-filled arenas regenerate their pattern instead
        self.live_ref: Optional[torch.Tensor] = None
        if host_image is not None:
            arr = host_image.view(np.int16 if self.dt == W.BF16 else np.int32)
            self.bits = torch.from_numpy(arr.copy()).to(device).view(self.shape6)
            if wl.other_live.size:
                live = torch.as_tensor(wl.other_live, device=self.bits.device)
                self.live_ref = self.bits[:, :, live].clone()
        else:
            self.bits = torch.empty(self.shape6, dtype=bits_t, device=device)
            self.fill_initial(progress)
        self.handle: Optional[int] = None

    @property
    def nbytes(self) -> int:
        return self.bits.numel() * self.bits.element_size()

    def ptr(self) -> int:
        return self.bits.data_ptr()

    def sentinel(self) -> int:
        return _signed(W.SENTINEL_BITS[self.dt], self.dt)

    def _chunk_blocks(self) -> int:
        """Blocks per chunk so that one chunk of one plane is about 64 MiB."""
        B, nkv, d = self.shape6[3:]
        return max(1, (64 << 20) // (B * nkv * d * self.bits.element_size()))

    def _base_pattern(self) -> torch.Tensor:
        """Fixed finite bit pattern over the elements of one block."""
        if getattr(self, "_base", None) is None:
            B, nkv, d = self.shape6[3:]
            e = torch.arange(B * nkv * d, device=self.bits.device, dtype=torch.int64)
            h = (e * 2654435761 + 97531)
            h = (h ^ (h >> 13)) * 1274126177
            h = h ^ (h >> 16)
            if self.dt == W.BF16:
                bits = (h & 0x807F) | 0x3F80
                bits = torch.where(bits >= 0x8000, bits - 0x10000, bits).to(torch.int16)
            else:
                bits = (h & 0x807FFFFF) | 0x3F800000
                bits = torch.where(bits >= 0x80000000, bits - 0x100000000, bits).to(torch.int32)
            self._base = bits
        return self._base

    def live_pattern(self, blocks: torch.Tensor, layer_kv: int) -> torch.Tensor:
        """Deterministic finite bit patterns for other-live blocks, computed
        on the device: [len(blocks), B, nkv, d].  A fixed per-element pattern
        XOR a per-(block, layer, K|V) hash confined to the sign and mantissa
        bits, so every value stays finite and the fill runs at copy speed."""
        B, nkv, d = self.shape6[3:]
        h = blocks.to(torch.int64) * 40503 + layer_kv * 97531 + 12345
        h = (h ^ (h >> 7)) * 1274126177
        h = h ^ (h >> 16)
        if self.dt == W.BF16:
            m = h & 0x807F
            m = torch.where(m >= 0x8000, m - 0x10000, m).to(torch.int16)
        else:
            m = h & 0x807FFFFF
            m = torch.where(m >= 0x80000000, m - 0x100000000, m).to(torch.int32)
        return (self._base_pattern()[None, :] ^ m[:, None]).view(len(blocks), B, nkv, d)

    def fill_initial(self, progress=None) -> None:
        self.bits.fill_(self.sentinel())
        live = torch.as_tensor(self.wl.other_live, device=self.bits.device)
        if live.numel() == 0:
            return
        ch = self._chunk_blocks()
        for l in range(self.shape6[0]):
            for kv in range(2):
                for i in range(0, live.numel(), ch):
                    blk = live[i:i + ch]
                    self.bits[l, kv, blk] = self.live_pattern(blk, 2 * l + kv)
            if progress:
                progress(f"fill layer {l + 1}/{self.shape6[0]}")

    def bind(self, device: int = 0) -> int:
        s = self.wl.shape
        self.handle = kvr.kv_arena_bind(self.ptr(), self.nbytes, s, self.wl.block_size,
                                        self.wl.num_blocks, device)
        return self.handle

    def release(self) -> None:
        if self.handle is not None:
            kvr.kv_arena_release(self.handle)
            self.handle = None

    def to_host(self) -> np.ndarray:
        a = self.bits.cpu().numpy()
        return a.view(np.uint16 if self.dt == W.BF16 else np.uint32).reshape(-1)

    # ---- invariants, checked on the device --------------------------------
    def check_invariants(self, progress=None) -> Dict[str, int]:
        """Bit-exact checks at any size, in chunks of about 64 MiB: unlisted
        blocks keep their fill (sentinel or other-live pattern), tail slots of
        each request's last block keep the sentinel, every written slot is
        finite and not the sentinel.  Returns counts of violations per kind."""
        wl = self.wl
        dev = self.bits.device
        L, _, NB, B = self.shape6[:4]
        listed = torch.zeros(NB, dtype=torch.bool, device=dev)
        ntab = ((wl.lens.astype(np.int64) + B - 1) // B)
        ids = np.concatenate([wl.block_tables[r, :ntab[r]] for r in range(wl.num_requests)]) \
            if wl.num_requests else np.zeros(0, np.int32)
        ids_t = torch.as_tensor(ids.astype(np.int64), device=dev)
        listed[ids_t] = True
        is_live = torch.zeros(NB, dtype=torch.bool, device=dev)
        if wl.other_live.size:
            is_live[torch.as_tensor(wl.other_live, device=dev)] = True
        live_index = None
        if self.live_ref is not None:
            # position of each other-live block within the snapshot
            live_index = torch.full((NB,), -1, dtype=torch.int64, device=dev)
            live_index[torch.as_tensor(wl.other_live, device=dev)] = torch.arange(
                wl.other_live.size, device=dev)
        free = ~listed & ~is_live
        # tail slots: (block, slot) of last blocks with slot >= n % B
        tail_b, tail_s = [], []
        for r in range(wl.num_requests):
            n = int(wl.lens[r])
            if n == 0 or n % B == 0:
                continue
            blk = int(wl.block_tables[r, (n - 1) // B])
            for sl in range(n % B, B):
                tail_b.append(blk)
                tail_s.append(sl)
        tail_b = torch.as_tensor(tail_b, dtype=torch.int64, device=dev)
        tail_s = torch.as_tensor(tail_s, dtype=torch.int64, device=dev)
        sen = self.sentinel()
        ch = self._chunk_blocks()
        bad = {"free_changed": 0, "live_changed": 0, "tail_changed": 0, "written_bad": 0}
        for l in range(L):
            for kv in range(2):
                plane = self.bits[l, kv]
                for c0 in range(0, NB, ch):
                    c1 = min(NB, c0 + ch)
                    sl = plane[c0:c1]
                    fr = free[c0:c1]
                    bad["free_changed"] += int(((sl != sen) & fr[:, None, None, None]).sum())
                    lv = torch.nonzero(is_live[c0:c1]).flatten()
                    if lv.numel():
                        if live_index is not None:
                            ref = self.live_ref[l, kv, live_index[lv + c0]]
                        else:
                            ref = self.live_pattern(lv + c0, 2 * l + kv)
                        bad["live_changed"] += int((sl[lv] != ref).sum())
                if tail_b.numel():
                    bad["tail_changed"] += int((plane[tail_b, tail_s] != sen).sum())
                # written slots = slots of listed blocks except the tails: finite values
                for i in range(0, ids_t.numel(), ch):
                    blk = ids_t[i:i + ch]
                    vals = plane[blk].view(_TORCH_VAL[self.dt])
                    bad["written_bad"] += int((~torch.isfinite(vals)).sum())
                if tail_b.numel():
                    tails = plane[tail_b, tail_s].view(_TORCH_VAL[self.dt])
                    bad["written_bad"] -= int((~torch.isfinite(tails)).sum())
            if progress:
                progress(f"check layer {l + 1}/{L}")
        return bad


def alloc_workspace(shape: W.ModelShape, num_requests: int, total_tokens: int,
                    wave_tokens: int, device="cuda", fill=None):
    """A rebuild workspace; `fill` (a byte value) overwrites its contents
    first, e.g. 0xFF so that any read of a never-written element yields NaN."""
    nbytes = kvr.kv_rebuild_workspace_bytes(shape, num_requests, total_tokens, wave_tokens)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
    if fill is not None:
        ws.fill_(fill)
    return ws, nbytes


def stream_ptr() -> int:
    return torch.cuda.current_stream().cuda_stream
