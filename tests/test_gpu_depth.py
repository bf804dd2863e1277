"""Parity through every layer of the 8B, 14B and 32B shapes, through the C ABI.

Random N(0, 0.02) decoders carry any difference in one bf16 rounding decision
down the fp32 residual stream and widen it layer by layer: two runs of the
oracle that differ only in how the attention weights are rounded, or only in
the last bit of one weight, drift apart by more than 2e-2 (normwise, per
layer and K|V plane) within the first 32 layers.  So parity at depth is
checked in two ways:

* every layer from a common input: for each layer l, the GPU and the oracle
  both run layers l and l+1 from the same input rows (a table the oracle
  produced, one layer at a time, from the embeddings), and layer l's and l+1's
  K/V must match within the stated 2e-2 -- at every depth, with nothing
  accumulated from earlier layers;
* end to end: the GPU's K/V of every layer against the oracle in the mode
  that rounds P as the GPU does, printed beside the oracle's own drift (that
  mode against the plain one, and the plain oracle against itself with one
  weight changed by one bf16 ulp); the GPU must stay within 2e-2 over the
  first layers and within 1.5x that drift plus 5e-3 everywhere.  A kernel
  mistake (index, sign, position) shows up as errors of order 1.

Request lengths are short because the oracle's fp64 forward costs about 0.44
(8B), 0.55 (14B) and 0.97 (32B) GFLOP per token per layer.
"""
import dataclasses
import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_14635_amd import harness as Hn  # noqa: E402
from paper_2608_14635_amd import kvr  # noqa: E402
from paper_2608_14635_amd import workloads as W  # noqa: E402

import parity_util as PU  # noqa: E402

pytestmark = pytest.mark.gpu
TOL = PU.TOL[W.BF16]

CASES = {
    "llama8b": (W.LLAMA8B, [1, 17, 40]),
    "qwen14b": (W.QWEN14B, [1, 17, 40]),
    "qwen32b": (W.QWEN32B, [1, 17]),
}
# Requests of 1, 17 and 300 tokens: minutes of the oracle's fp64 forward on
# 16 host threads per test (8B about 3 and 4, 14B about 7 and 10, 32B about
# 16 end to end), so they run only when KVR_DEPTH_LONG=1 is set; the 32B
# shape's layer-by-layer test (about 25 minutes) is left out.
LONG = os.environ.get("KVR_DEPTH_LONG") == "1"
if LONG:
    CASES["llama8b_300"] = (W.LLAMA8B, [1, 17, 300])
    CASES["qwen14b_300"] = (W.QWEN14B, [1, 17, 300])
    CASES["qwen32b_300"] = (W.QWEN32B, [1, 17, 300])
    # the 8B shape with a 1000-token request too: about 12 minutes end to end and
    # 2 x 9 minutes layer by layer (KVR_DEPTH_LAYERS=0:16, 16:31)
    CASES["llama8b_1000"] = (W.LLAMA8B, [1, 17, 300, 1000])


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def exact_frac(a, b, wl):
    """Share of written K/V elements of every layer that are bit-identical, per layer."""
    s = wl.shape
    m = PU.written_mask(wl)
    va = a.reshape(s.num_layers, 2, wl.num_blocks, wl.block_size, -1)
    vb = b.reshape(va.shape)
    return np.array([np.mean(va[l][m[l]] == vb[l][m[l]]) for l in range(s.num_layers)])


def gpu_rebuild(wl, model, image):
    arena = Hn.DeviceArena(wl, host_image=image)
    arena.bind()
    ws, nbytes = Hn.alloc_workspace(wl.shape, wl.num_requests, wl.total_tokens, wl.total_tokens, fill=0xFF)
    kvr.kv_rebuild(model.weights, wl.tokens, wl.lens, wl.block_tables, arena.handle, ws.data_ptr(), nbytes,
                   Hn.stream_ptr())
    torch.cuda.synchronize()
    out = arena.to_host()
    arena.release()
    return out


@pytest.mark.parametrize("name", list(CASES))
def test_end_to_end_all_layers(oracle_lib, name):
    shape, lens = CASES[name]
    wl = W.small_workload(shape, lens, block_size=16, seed=411, other_live_frac=0.3)
    say(f"{name}: all {shape.num_layers} layers end to end, lens={lens}")
    model = Hn.device_model_random(shape, seed=412, gain_std=0.1)
    host_w = Hn.host_copy_all(model)
    image = W.host_arena(wl)
    g = gpu_rebuild(wl, model, image)
    del model
    torch.cuda.empty_cache()
    o = image.copy()
    oracle_lib.rebuild(shape, host_w, wl.tokens, wl.lens, wl.block_tables, o, wl.block_size, wl.num_blocks)
    say("  oracle (definition) done")
    o_p = image.copy()
    oracle_lib.rebuild(shape, host_w, wl.tokens, wl.lens, wl.block_tables, o_p, wl.block_size,
                       wl.num_blocks, round_p=True)
    say("  oracle (P rounded) done")
    gpu_p, rep = PU.compare(wl, g, o_p, image)
    gpu_o, _ = PU.compare(wl, g, o, image)
    drift, _ = PU.compare(wl, o_p, o, image)
    np.set_printoptions(precision=3, linewidth=240)
    say(f"  GPU vs oracle (P rounded as the GPU): {gpu_p.max(axis=1)}")
    say(f"  GPU vs oracle (definition):           {gpu_o.max(axis=1)}")
    say(f"  oracle, P rounded vs definition:      {drift.max(axis=1)}")
    say(f"  bit-identical share, GPU vs P-rounded oracle: {exact_frac(g, o_p, wl)}")
    say(f"  bit-identical share, GPU vs definition:       {exact_frac(g, o, wl)}")
    envelope = drift
    if name in ("llama8b", "llama8b_300"):
        # the oracle against itself with the last bit of one layer-0 value
        # weight flipped: the model's own sensitivity to one rounding-sized change
        w1 = {"embed": host_w["embed"], "layers": [dict(lw) for lw in host_w["layers"]]}
        wv = w1["layers"][0]["wv"].copy()
        wv.reshape(-1)[12345] ^= 1
        w1["layers"][0]["wv"] = wv
        o_1 = image.copy()
        oracle_lib.rebuild(shape, w1, wl.tokens, wl.lens, wl.block_tables, o_1, wl.block_size,
                           wl.num_blocks)
        sens, _ = PU.compare(wl, o_1, o, image)
        say(f"  oracle, one weight one ulp off:       {sens.max(axis=1)}")
        # the change grows with depth (observed: 0.005 after one layer, 0.02 by layer 28)
        assert sens.max(axis=1)[-4:].max() > 3 * sens.max(axis=1)[1], sens.max(axis=1)
        envelope = np.maximum(drift, sens)
    assert rep["unwritten_changed"] == 0 and rep["written_nonfinite"] == 0
    assert gpu_p[:4].max() <= TOL, gpu_p[:4]
    bound = np.maximum(TOL, 1.5 * envelope + 5e-3)
    assert np.all(gpu_p <= bound), (gpu_p, bound)


@pytest.mark.parametrize("name", list(CASES))
def test_every_layer_from_common_input(oracle_lib, name):
    # KVR_DEPTH_LAYERS="a:b" checks the pairs l = a..b-1 only (the oracle still
    # forms every earlier layer's input), so a long case can be split over runs
    rng = os.environ.get("KVR_DEPTH_LAYERS", "")
    if name in ("qwen32b_300", "llama8b_1000") and not rng:
        pytest.skip("this case's layer-by-layer oracle takes about 20-25 minutes; "
                    "run it in parts with KVR_DEPTH_LAYERS")
    shape, lens = CASES[name]
    wl = W.small_workload(shape, lens, block_size=16, seed=421, other_live_frac=0.3)
    L, T = shape.num_layers, wl.total_tokens
    say(f"{name}: layers l, l+1 from the oracle's layer-l input, l = 0..{L - 2}, lens={lens}")
    model = Hn.device_model_random(shape, seed=422, gain_std=0.1)
    host_w = Hn.host_copy_all(model)
    # rows of the input table are the packed tokens: token i of the batch is row i
    one = dataclasses.replace(shape, num_layers=1, vocab=T)
    two = dataclasses.replace(shape, num_layers=2, vocab=T)
    wl1 = dataclasses.replace(wl, shape=one, tokens=np.arange(T, dtype=np.int32))
    wl2 = dataclasses.replace(wl, shape=two, tokens=np.arange(T, dtype=np.int32))
    table = np.ascontiguousarray(host_w["embed"][wl.tokens])  # layer-0 input rows
    worst = np.zeros(L - 1)
    lo, hi = (int(v) for v in rng.split(":")) if rng else (0, L - 1)
    for l in range(min(hi, L - 1)):
        if l < lo:
            # only the next layer's input rows (see below)
            single = {"embed": table, "layers": [host_w["layers"][l]]}
            fh = oracle_lib.rebuild(one, single, wl1.tokens, wl1.lens, wl1.block_tables, W.host_arena(wl1),
                                    wl1.block_size, wl1.num_blocks, final_hidden=True)
            table = W.f32_to_bf16_bits(fh.astype(np.float32))
            say(f"  layer {l}: input rows of layer {l + 1} formed")
            continue
        pair = {"embed": table, "layers": [host_w["layers"][l], host_w["layers"][l + 1]]}
        image = W.host_arena(wl2)
        o = image.copy()
        oracle_lib.rebuild(two, pair, wl2.tokens, wl2.lens, wl2.block_tables, o, wl2.block_size,
                           wl2.num_blocks)
        dev = Hn.model_view(two, Hn.upload(two, table), [model.layers[l], model.layers[l + 1]])
        g = gpu_rebuild(wl2, dev, image)
        err, rep = PU.compare(wl2, g, o, image)
        assert rep["unwritten_changed"] == 0 and rep["written_nonfinite"] == 0
        worst[l] = err.max()
        say(f"  layers {l}, {l + 1}: worst K/V error {worst[l]:.2e}")
        # the next layer's input rows: this layer's output residual (oracle), rounded to bf16
        single = {"embed": table, "layers": [host_w["layers"][l]]}
        fh = oracle_lib.rebuild(one, single, wl1.tokens, wl1.lens, wl1.block_tables, W.host_arena(wl1),
                                wl1.block_size, wl1.num_blocks, final_hidden=True)
        table = W.f32_to_bf16_bits(fh.astype(np.float32))
    np.set_printoptions(precision=4, linewidth=240)
    say(f"  worst K/V error of layers l, l+1 per l: {worst}")
    assert worst.max() <= TOL, worst
