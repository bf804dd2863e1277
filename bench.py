"""KV-rebuild benchmark on one MI355X.

    python bench.py [--gpus 1] [--steps 5] [--warmup 1] [--config 2]

A step is one full kv_rebuild call of the configuration's whole request
batch: host validation and wave planning, the metadata upload, embedding
gather, every layer's norms, QKV GEMM + RoPE + arena scatter, attention,
output projection and SwiGLU FFN, with weights and arena resident in HBM.
The default workload is the 8B-shaped decoder with 16 requests of 2048-16384
tokens.  Prints one JSON line; `value` is total tokens over the wall time of
the K timed steps, and the per-step HIP-event median is reported beside it,
as is the device time of a pre-staged plan (kv_rebuild_execute).
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2517.0   # MI355X dense bf16 MFMA (256 CU x 2.4 GHz x 4096 flop/clk)
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0

# kernel class -> sources whose text fixes that kernel's code
KERNEL_SOURCES = {
    "gemm_qkv": ["gemm_bf16.hip", "epilogue.h", "common.h", "launch.h"],
    "gemm_o": ["gemm_bf16.hip", "epilogue.h", "common.h", "launch.h"],
    "gemm_gateup": ["gemm_bf16.hip", "epilogue.h", "common.h", "launch.h"],
    "gemm_down": ["gemm_bf16.hip", "epilogue.h", "common.h", "launch.h"],
    "attention": ["attention.hip", "common.h", "launch.h"],
    "verify": ["verify.hip", "launch.h"],
}


def kernel_source_hash(kernel: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES.get(kernel, []):
        with open(os.path.join(ROOT, "paper_2608_14635_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed counter runs (profiles/traffic.json),
    or None when they were taken on other kernel sources or another workload."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f).get(kernel)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_sha") != kernel_source_hash(kernel) or rec.get("workload") != workload:
        return None
    return rec.get("bytes_per_launch")


def decode_step_bytes(s, ctx_lens) -> int:
    """Algorithmic HBM bytes of one decode step over requests whose contexts
    (the step's own position included) have the lengths ctx_lens: every layer's
    weights (Q/K/V/O and gate/up/down projections, both norm gains), the final
    norm gain and the LM head once; each request's embedding row; every
    context key's K and V row once per layer; the step's new K and V rows."""
    e = s.elem_bytes
    H, F, d, nq, nkv, L = s.hidden, s.ffn_dim, s.head_dim, s.num_q_heads, s.num_kv_heads, s.num_layers
    R = len(ctx_lens)
    w_layer = (H * (nq + 2 * nkv) * d + nq * d * H + 3 * H * F + 2 * H) * e
    weights = L * w_layer + (s.vocab * H + H) * e + R * H * e
    kv_read = int(sum(int(n) for n in ctx_lens)) * L * 2 * nkv * d * e
    kv_write = R * L * 2 * nkv * d * e
    return weights + kv_read + kv_write


def resume_decode(wl, model, arena, Hn, kvr, W, steps, stream, log):
    """Resumed generation over the rebuilt arena: one greedy decode step per
    request, timed with HIP events.  Each step decodes every request's last
    prefix token again at its own position (rewriting that slot), so it
    attends over the whole rebuilt context.  HBM-bound: the weights are read
    once per step and every request's K/V context once per layer."""
    import numpy as np
    import torch
    s = wl.shape
    R = wl.num_requests
    offs = wl.request_offsets()
    lens = wl.lens.astype(np.int64)
    live = lens > 0
    rows = np.nonzero(live)[0]
    toks = np.array([wl.tokens[offs[r + 1] - 1] for r in rows], np.int32)
    pos = (lens[rows] - 1).astype(np.int32)
    head = Hn.device_head_random(s, seed=0x5EED00FF)
    nbytes = kvr.kv_decode_workspace_bytes(s, len(rows), int(pos.max()) + 1)
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    nxt = torch.zeros(len(rows), dtype=torch.int32, device="cuda")

    def step():
        kvr.kv_decode_step(model.weights, head["final_norm"].data_ptr(), head["lm_head"].data_ptr(),
                           toks, pos, wl.block_tables[rows], arena.handle, ws.data_ptr(), nbytes,
                           nxt.data_ptr(), 0, stream)
    step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    total = decode_step_bytes(s, lens[rows])
    out = {"steps": steps, "requests": int(len(rows)), "ms_per_step": ms,
           "tokens_per_s": len(rows) / (ms / 1e3), "context_tokens": int(lens[rows].sum()),
           "hbm_bytes_per_step": total, "achieved_GBps": total / (ms / 1e3) / 1e9,
           "hbm_frac": total / (ms / 1e3) / 1e9 / PEAK_HBM_GBS,
           "next_tokens": nxt.cpu().numpy().tolist()[:8]}
    log(f"[bench] resume decode: {ms:.2f} ms per step of {len(rows)} requests, "
        f"{out['achieved_GBps']:.0f} GB/s ({100 * out['hbm_frac']:.1f}% of HBM)")
    return out


def flush_free(wl, model, arena, ws_rebuild, Hn, kvr, reps, stream, log):
    """Flush-free recovery over the rebuilt arena: commit digests of every
    block the requests occupy, then time the verification scan (HBM-bound:
    every covered byte read once, HIP events on the library's stream), and
    one recovery of a single damaged request (verify + rebuild of that request
    only) against the full flush-and-refill rebuild."""
    import numpy as np
    import torch
    s, B = wl.shape, wl.block_size
    E = kvr.num_entries(wl.lens, B)
    R = wl.num_requests
    nbytes = kvr.kv_verify_workspace_bytes(R, E)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device="cuda")
    committed = torch.empty(max(E, 1), dtype=torch.int64, device="cuda")
    intact = torch.empty(max(R, 1), dtype=torch.int32, device="cuda")
    kvr.kv_block_digests(arena.handle, wl.lens, wl.block_tables, ws.data_ptr(), nbytes,
                         committed.data_ptr(), stream)

    def verify():
        kvr.kv_verify(arena.handle, wl.lens, wl.block_tables, committed.data_ptr(), ws.data_ptr(),
                      nbytes, intact.data_ptr(), 0, stream)
    verify()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        verify()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    nb = (wl.lens + B - 1) // B
    all_intact = bool(np.array_equal(intact[:R].cpu().numpy(), nb))
    covered = int(wl.lens.astype(np.int64).sum()) * s.num_layers * 2 * s.num_kv_heads * s.head_dim * s.elem_bytes
    moved = covered + 8 * E + E + 4 * (R + 1) + 8 * E + 4 * R
    # one damaged request (the median-length one), damaged in its middle block:
    # (a) verify, then rebuild that request alone; (b) verify, then rebuild it
    # from its first damaged block, rounded down to a multiple of 256
    # positions (where the recomputed values are the full rebuild's bit for
    # bit, so the committed digests stay valid)
    r = int(np.argsort(wl.lens)[R // 2])
    blk = int(wl.block_tables[r, int(nb[r]) // 2])
    offs = wl.request_offsets()

    def damage():
        arena.bits[s.num_layers - 1, 1, blk, 0, 0, 0] ^= 1
        torch.cuda.synchronize()

    damage()
    t0 = time.perf_counter()
    verify()
    got = intact[:R].cpu().numpy()
    bad = np.nonzero(got < nb)[0]
    toks = np.concatenate([wl.tokens[offs[i]:offs[i] + wl.lens[i]] for i in bad]) if bad.size else \
        np.zeros(0, np.int32)
    kvr.kv_rebuild(model.weights, toks, wl.lens[bad], wl.block_tables[bad], arena.handle,
                   ws_rebuild[0].data_ptr(), ws_rebuild[1], stream)
    torch.cuda.synchronize()
    rec_ms = (time.perf_counter() - t0) * 1e3
    verify()
    healed = bool(np.array_equal(intact[:R].cpu().numpy(), nb))
    damage()
    t0 = time.perf_counter()
    verify()
    got = intact[:R].cpu().numpy()
    bad = np.nonzero(got < nb)[0]
    starts = ((got[bad] * B) // 256 * 256).astype(np.int32)
    toks = np.concatenate([wl.tokens[offs[i] + st:offs[i] + wl.lens[i]] for i, st in zip(bad, starts)]) \
        if bad.size else np.zeros(0, np.int32)
    kvr.kv_rebuild_from(model.weights, toks, wl.lens[bad], starts, wl.block_tables[bad], arena.handle,
                        ws_rebuild[0].data_ptr(), ws_rebuild[1], stream)
    torch.cuda.synchronize()
    from_ms = (time.perf_counter() - t0) * 1e3
    verify()
    healed_from = bool(np.array_equal(intact[:R].cpu().numpy(), nb))
    out = {"entries": E, "verify_ms": ms, "covered_bytes": covered, "bytes_per_launch": moved,
           "achieved_GBps": moved / (ms / 1e3) / 1e9, "hbm_frac": moved / (ms / 1e3) / 1e9 / PEAK_HBM_GBS,
           "traffic": measured_traffic("verify", wl.name), "source_sha": kernel_source_hash("verify"),
           "all_intact_after_rebuild": all_intact,
           "one_damaged_request": {"request": r, "tokens": int(wl.lens[r]),
                                   "detected": bad.tolist(), "recovery_ms": rec_ms,
                                   "intact_after": healed,
                                   "from_position": int(starts[0]) if bad.size else None,
                                   "recovery_from_block_ms": from_ms,
                                   "intact_after_from_block": healed_from}}
    log(f"[bench] verify scan: {ms:.3f} ms over {E} blocks, {out['achieved_GBps']:.0f} GB/s "
        f"({100 * out['hbm_frac']:.1f}% of HBM); one damaged request recovered in {rec_ms:.1f} ms, "
        f"from its damaged block in {from_ms:.1f} ms")
    return out


def shared_prefix(wl, model, arena, ws, nbytes, kvr, S, steps, stream, log):
    """Requests that all begin with the same S tokens (S a multiple of the
    block size): request 0 computes them, the others list its first S/B
    blocks read-only and start at S, all in one call (kv_rebuild_from).
    Timed with HIP events like the main rebuild; covered positions are all
    of every request's."""
    import numpy as np
    import torch
    R, B = wl.num_requests, wl.block_size
    offs = wl.request_offsets()
    head = wl.tokens[offs[0]:offs[0] + S]
    if S % B or any(wl.lens[r] < S or not np.array_equal(wl.tokens[offs[r]:offs[r] + S], head)
                    for r in range(R)):
        raise SystemExit(f"--shared-prefix {S}: the requests do not all begin with the same {S} tokens "
                         f"(or {S} is not a multiple of the block size {B})")
    tables = wl.block_tables.copy()
    tables[1:, :S // B] = tables[0, :S // B]
    starts = np.array([0] + [S] * (R - 1), np.int32)
    toks = np.concatenate([wl.tokens[offs[r] + starts[r]:offs[r] + wl.lens[r]] for r in range(R)])
    plan = kvr.kv_rebuild_stage_from(arena.handle, toks, wl.lens, starts, tables, ws.data_ptr(), nbytes,
                                     stream)
    kvr.kv_rebuild_execute(model.weights, plan, stream)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        kvr.kv_rebuild_execute(model.weights, plan, stream)
    e1.record()
    torch.cuda.synchronize()
    kvr.kv_plan_release(plan)
    ms = e0.elapsed_time(e1) / steps
    covered, computed = int(wl.lens.sum()), int(len(toks))
    out = {"shared_tokens": S, "requests": R, "positions_covered": covered,
           "positions_computed": computed, "ms_per_step": ms,
           "covered_tokens_per_s": covered / (ms / 1e3)}
    log(f"[bench] shared prefix of {S}: {computed} of {covered} positions computed, {ms:.1f} ms per "
        f"step, {out['covered_tokens_per_s']:.0f} covered tokens/s")
    return out


def algorithmic_work(wl):
    """Flops and HBM bytes the method must spend (last layer: K/V projections only)."""
    s = wl.shape
    H, d, nq, nkv, F, L = s.hidden, s.head_dim, s.num_q_heads, s.num_kv_heads, s.ffn_dim, s.num_layers
    lin_tok = 2.0 * ((L - 1) * (H * (nq + 2 * nkv) * d + nq * d * H + 3 * H * F) + 2 * H * nkv * d)
    n = wl.lens.astype(np.float64)
    attn = float(np.sum(2.0 * nq * d * n * (n + 1))) * (L - 1)
    flops = lin_tok * wl.total_tokens + attn
    e = s.elem_bytes
    w_layer = H * (nq + 2 * nkv) * d + nq * d * H + 3 * H * F + 2 * H
    weights = ((L - 1) * w_layer + 2 * nkv * d * H + H) * e
    kv = wl.total_tokens * L * 2 * nkv * d * e
    emb = wl.total_tokens * H * e
    return {"flops": flops, "linear_flops": lin_tok * wl.total_tokens, "attn_flops": attn,
            "bytes": float(weights + kv + emb), "kv_bytes": float(kv)}


def host_info():
    """Host CPU facts for the CPU baseline: nproc, the lscpu model name."""
    model = platform.processor()
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                model = line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    return {"nproc": os.cpu_count(), "lscpu_model": model}


# CPU-baseline sample plans: (fit lengths n1, n2; all-layer check length)
CPU_PLANS = {"bounded": (1024, 4096, 64), "full": (1024, 4096, 512)}


def _oracle_forward_time(o, s, embed, layer, tokens, L, log):
    """Wall time of a complete L-layer oracle forward over one request, run one
    layer per call: each layer's output rows, rounded to the model's dtype,
    are the next call's input rows, and a line is printed per layer.  Layer
    0's weights serve every layer (the time depends only on the shapes), and
    every layer is run whole, the last one included."""
    import dataclasses
    from paper_2608_14635_amd import workloads as W
    n = len(tokens)
    one = dataclasses.replace(s, num_layers=1, vocab=n)
    nb = (n + 15) // 16
    tables = np.arange(nb, dtype=np.int32)[None, :]
    ids = np.arange(n, dtype=np.int32)
    lens = np.array([n], dtype=np.int32)
    rows = np.ascontiguousarray(embed[np.asarray(tokens)])
    arena = np.zeros(2 * nb * 16 * s.num_kv_heads * s.head_dim, dtype=embed.dtype)
    total = 0.0
    for l in range(L):
        t0 = time.perf_counter()
        fh = o.rebuild(one, {"embed": rows, "layers": [layer]}, ids, lens, tables, arena, 16, nb,
                       final_hidden=True)
        total += time.perf_counter() - t0
        if s.dtype == W.BF16:
            rows = W.f32_to_bf16_bits(fh.astype(np.float32))
        else:
            rows = np.ascontiguousarray(fh.astype(embed.dtype))
        log(f"[bench] oracle check: layer {l + 1}/{L} over {n} tokens, {total:.1f}s so far")
    return total


def cpu_baseline(wl, model, Hn, plan: str = "bounded", log=lambda m: None):
    """Time the CPU oracle on a bounded sample of the same workload and model
    the whole rebuild from it: one transformer layer of the workload's shape
    over one request at two lengths gives t_layer(n) = a n + b n^2 (fitted),
    layer-0 K/V rows of 128 tokens give c, the last layer's per-token cost,
    and t = sum_r (L-1) t_layer(n_r) + c n_r.  The model is checked against a
    complete all-layer oracle run over one request.  Both plans fit at
    n = 1024 and 4096 (about a minute of CPU work for the 8B shape on 16
    threads: shorter requests make the quadratic attention term too small for
    requests of up to 16K tokens); "full" checks on 512 tokens (three more
    minutes), "bounded" on 64.  A tiny model's whole rebuild is timed instead
    (median of 5)."""
    import oracle
    from paper_2608_14635_amd import workloads as W
    o = oracle.get()
    s = wl.shape
    info = host_info()
    if s.num_layers == 2 and s.hidden <= 512:
        # a tiny model: the whole rebuild of the workload, median of 5 runs
        host_w = Hn.host_copy_all(model)
        times = []
        for _ in range(5):
            arena = W.host_arena(wl)
            t0 = time.perf_counter()
            o.rebuild(s, host_w, wl.tokens, wl.lens, wl.block_tables, arena, wl.block_size, wl.num_blocks)
            times.append(time.perf_counter() - t0)
        t = float(np.median(times))
        return {"value": wl.total_tokens / t, "unit": "tokens/s", "cores": o.num_threads(), "kind": "oracle",
                "plan": "whole", "nproc": info["nproc"], "lscpu_model": info["lscpu_model"],
                "omp_threads": o.num_threads(),
                "sample": f"the whole oracle rebuild of the workload's {wl.total_tokens} tokens, median of 5 runs "
                          f"({t * 1e3:.1f} ms)"}
    host = Hn.host_copy_layer0(model)
    layer_w = {"embed": host["embed"], "layers": [host["layer0"]]}
    rng = np.random.default_rng(99)
    n1, n2, nm = CPU_PLANS[plan]
    t1 = o.time_layers(s, layer_w, rng.integers(0, s.vocab, n1), 1)
    log(f"[bench] oracle: one layer over {n1} tokens in {t1:.1f}s")
    t2 = o.time_layers(s, layer_w, rng.integers(0, s.vocab, n2), 1)
    log(f"[bench] oracle: one layer over {n2} tokens in {t2:.1f}s")
    b = max(0.0, (t2 / n2 - t1 / n1) / (n2 - n1))
    a = max(1e-12, t1 / n1 - b * n1)
    nk = 128
    tk0 = time.perf_counter()
    o.layer0_kv(s, host["embed"], host["layer0"], rng.integers(0, s.vocab, nk),
                rng.integers(0, 4096, nk))
    c = (time.perf_counter() - tk0) / nk
    log(f"[bench] oracle: layer-0 K/V rows of {nk} tokens in {c * nk:.2f}s")
    n = wl.lens.astype(np.float64)
    L = s.num_layers
    t_pred = float(np.sum((L - 1) * (a * n + b * n * n) + c * n))
    # check of the model: a complete oracle forward of all layers over one request
    tm = _oracle_forward_time(o, s, host["embed"], host["layer0"], rng.integers(0, s.vocab, nm), L, log)
    tm_pred = L * (a * nm + b * nm * nm)
    return {"value": wl.total_tokens / t_pred, "unit": "tokens/s", "cores": o.num_threads(),
            "kind": "oracle", "plan": plan,
            "nproc": info["nproc"], "lscpu_model": info["lscpu_model"],
            "omp_threads": o.num_threads(),
            "fit": {"n1": n1, "t1_s": t1, "n2": n2, "t2_s": t2, "a_s_per_token": a,
                    "b_s_per_token2": b, "c_s_per_token": c},
            "model_check": {"tokens": nm, "layers": L, "measured_s": tm, "predicted_s": tm_pred,
                            "ratio": tm / tm_pred},
            "sample": (f"oracle timed on one layer of the same shape at n={n1} ({t1:.1f}s) and "
                       f"n={n2} ({t2:.1f}s) plus layer-0 K/V rows of {nk} tokens ({c * nk:.2f}s); "
                       f"fitted t_layer(n)=a*n+b*n^2 extrapolated to {L} layers x "
                       f"{wl.num_requests} requests (modelled from measured per-layer timings, "
                       f"{t_pred:.0f}s predicted); checked by a complete {L}-layer forward, one layer per call, over "
                       f"{nm} tokens ({tm:.1f}s measured, {tm_pred:.1f}s predicted)")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--model", default="",
                    help="run the configuration's request mix on another decoder shape "
                         "(e.g. qwen3_8b, qwen3_32b, qwen25_1_5b: the paper's model families)")
    ap.add_argument("--wave-tokens", type=int, default=0, help="0 = largest that fits")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-baseline", choices=sorted(CPU_PLANS), default="bounded",
                    help="CPU-oracle sample plan (n=1024/4096 fit; all-layer check on 64 tokens, full: 512)")
    ap.add_argument("--no-check", action="store_true")
    ap.add_argument("--decode-steps", type=int, default=4,
                    help="resumed-decode steps timed after the rebuild (0 = none)")
    ap.add_argument("--shared-prefix", type=int, default=0,
                    help="also time a rebuild whose requests share their first N tokens' blocks")
    ap.add_argument("--verify-reps", type=int, default=20,
                    help="timed block-digest verification scans after the rebuild (0 = skip)")
    ap.add_argument("--copy-probe", type=int, default=0,
                    help="only copy this many bytes device-to-device (counter calibration)")
    args = ap.parse_args()
    if args.copy_probe:
        import torch
        n = args.copy_probe // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n * 4}))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    import torch
    from paper_2608_14635_amd import harness as Hn
    from paper_2608_14635_amd import kvr
    from paper_2608_14635_amd import workloads as W

    torch.cuda.set_device(0)
    cfg = args.config
    shape = {1: W.TINY_F32, 2: W.LLAMA8B, 3: W.LLAMA8B, 4: W.QWEN14B, 5: W.QWEN32B}[cfg]
    if args.model:
        shape = W.SHAPES[args.model]
    log = lambda m: print(m, file=sys.stderr, flush=True)  # noqa: E731

    log(f"[bench] config {cfg}: generating weights on the device")
    model = Hn.device_model_random(shape, seed=0x5EED0000 + cfg)
    torch.cuda.synchronize()
    if cfg in (3, 5):
        # arena fills the HBM left after weights and workspace (2 GiB margin)
        probe = W.CONFIGS[cfg](num_blocks=1 << 30, shape=shape)
        wave = args.wave_tokens or min(probe.total_tokens, 131072)
        ws_bytes = kvr.kv_rebuild_workspace_bytes(shape, probe.num_requests, probe.total_tokens, wave)
        free, _ = torch.cuda.mem_get_info()
        per_block = shape.num_layers * 2 * 16 * shape.kv_row_elems() * shape.elem_bytes
        nb = int((free - ws_bytes - (2 << 30)) // per_block)
        wl = W.CONFIGS[cfg](num_blocks=nb, shape=shape)
    else:
        wl = W.CONFIGS[cfg](shape=shape) if cfg != 1 else W.CONFIGS[cfg]()
    T = wl.total_tokens
    wave = args.wave_tokens or min(T, 131072 if cfg != 5 else 65536)
    log(f"[bench] R={wl.num_requests} T={T} NB={wl.num_blocks} arena={wl.arena_bytes() / 2**30:.1f} GiB")
    big = wl.arena_bytes() > (32 << 30)
    arena = Hn.DeviceArena(wl, progress=log if big else None)
    arena.bind(0)
    ws, nbytes = Hn.alloc_workspace(shape, wl.num_requests, T, wave)
    stream = Hn.stream_ptr()
    plan = kvr.kv_rebuild_stage(arena.handle, wl.tokens, wl.lens, wl.block_tables, ws.data_ptr(),
                                nbytes, stream)
    n_waves, max_wave = kvr.kv_plan_info(plan)
    torch.cuda.synchronize()

    for i in range(args.warmup):
        kvr.kv_rebuild(model.weights, wl.tokens, wl.lens, wl.block_tables, arena.handle, ws.data_ptr(),
                       nbytes, stream)
        torch.cuda.synchronize()
        log(f"[bench] warmup {i + 1}/{args.warmup} done")

    # timed steps: whole kv_rebuild calls (metadata staged from host arrays
    # every call), HIP events around each on the library's stream
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record()
    for i in range(args.steps):
        kvr.kv_rebuild(model.weights, wl.tokens, wl.lens, wl.block_tables, arena.handle, ws.data_ptr(),
                       nbytes, stream)
        evs[i + 1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_wall = (t1 - t0) * 1e3 / args.steps
    step_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]
    ms_median = float(np.median(step_ms))
    log(f"[bench] {args.steps} steps: {ms_wall:.1f} ms/step wall, median {ms_median:.1f} ms "
        f"(events {', '.join(f'{x:.1f}' for x in step_ms)})")

    # the device work of a pre-staged plan alone (metadata already in HBM)
    ex0, ex1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ex0.record()
    for i in range(args.steps):
        kvr.kv_rebuild_execute(model.weights, plan, stream)
    ex1.record()
    torch.cuda.synchronize()
    ms_exec = ex0.elapsed_time(ex1) / args.steps

    # one profiled step: per-kernel-class device time via HIP events inside the library
    kvr.kv_profile_reset(arena.handle)
    kvr.kv_profile_enable(arena.handle, True)
    kvr.kv_rebuild_execute(model.weights, plan, stream)
    torch.cuda.synchronize()
    prof = kvr.kv_profile_read(arena.handle)
    kvr.kv_profile_enable(arena.handle, False)
    kvr.kv_plan_release(plan)

    check = None
    if not args.no_check:
        check = arena.check_invariants(progress=log if big else None)
        log(f"[bench] arena invariants after the last rebuild: {check}")

    work = algorithmic_work(wl)
    peak = PEAK_FP32_TFLOPS if shape.dtype == W.F32 else PEAK_BF16_TFLOPS
    sec = ms_wall / 1e3
    dom = max((k for k in prof if prof[k]["launches"]), key=lambda k: prof[k]["ms"])
    dom_t = prof[dom]["ms"] / 1e3
    dom_tf = prof[dom]["flops"] / dom_t / 1e12 if dom_t > 0 else 0.0
    gemm_keys = ("gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down")
    gemm_ms = sum(prof[k]["ms"] for k in gemm_keys)
    gemm_tf = sum(prof[k]["flops"] for k in gemm_keys) / (gemm_ms / 1e3) / 1e12 if gemm_ms else 0.0

    # the verification runs over the rebuilt arena before resumed decode
    # rewrites each request's last slot (decode rounds differently from the
    # prefill, so its rows would need commit records of their own)
    ff = None
    if args.verify_reps > 0 and wl.num_requests > 0:
        ff = flush_free(wl, model, arena, (ws, nbytes), Hn, kvr, args.verify_reps, stream, log)

    dec = None
    if args.decode_steps > 0 and wl.num_requests > 0:
        dec = resume_decode(wl, model, arena, Hn, kvr, W, args.decode_steps, stream, log)

    sp = None
    if args.shared_prefix > 0:
        sp = shared_prefix(wl, model, arena, ws, nbytes, kvr, args.shared_prefix, max(1, args.steps), stream,
                           log)

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        cpu = cpu_baseline(wl, model, Hn, args.cpu_baseline, log)
        log(f"[bench] cpu baseline {cpu}")

    dt_name = "bf16" if shape.dtype == W.BF16 else "f32"
    out = {
        "metric": "KV-rebuild prefix tokens/sec (1 GPU) + MFMA/HBM roofline fraction",
        "value": T / sec, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_wall, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": dt_name, "data": "synthetic",
        "config": {"workload": wl.name + (f"@{args.model}" if args.model else ""),
                   "requests": wl.num_requests, "total_tokens": T,
                   "block_size": wl.block_size, "num_blocks": wl.num_blocks,
                   "layers": shape.num_layers, "hidden": shape.hidden,
                   "heads": f"{shape.num_q_heads}/{shape.num_kv_heads}x{shape.head_dim}",
                   "ffn": shape.ffn_dim, "vocab": shape.vocab, "waves": n_waves,
                   "max_wave_tokens": max_wave, "weights": "random N(0,0.02)"},
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": dom_tf, "peak": peak,
                     "unit": "TFLOP/s", "frac": dom_tf / peak,
                     "traffic": measured_traffic(dom, wl.name),
                     "launches": prof[dom]["launches"],
                     "avg_launch_ms": prof[dom]["ms"] / max(1, prof[dom]["launches"]),
                     "flop_per_launch": prof[dom]["flops"] / max(1, prof[dom]["launches"]),
                     "source_sha": kernel_source_hash(dom)},
        "end_to_end": {"algorithmic_tflop": work["flops"] / 1e12,
                       "mfma_frac": work["flops"] / sec / 1e12 / peak,
                       "hbm_frac": work["bytes"] / sec / 1e9 / PEAK_HBM_GBS,
                       "gemm_tflops": gemm_tf, "gemm_frac": gemm_tf / peak,
                       "median_ms_per_step": ms_median, "step_ms_events": step_ms,
                       "staged_plan_ms": ms_exec,
                       "staged_plan_tokens_per_s": T / (ms_exec / 1e3)},
        "kernel_classes": {k: {"ms": round(v["ms"], 3), "launches": v["launches"],
                               "tflops": (v["flops"] / (v["ms"] / 1e3) / 1e12) if v["ms"] and v["flops"] else None}
                           for k, v in prof.items()},
        "arena_check": check,
        "resume_decode": dec,
        "flush_free": ff,
        "shared_prefix": sp,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    arena.release()


if __name__ == "__main__":
    main()
