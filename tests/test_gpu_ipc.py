"""Cross-process retained state (include/kvr_ipc.h) on the GPU.

An owner process (ipc_owner.py) holds the weights and the arena; this process
plays the replacement worker: it checks the owner, opens both through IPC
handles, binds the arena (which runs the health probe) and rebuilds into it
(Sec. 4.2, Handover steps 1-4).  The owner's arena must then hold exactly
what an in-process rebuild produces (bit-identical, deterministic kernels),
within the oracle tolerance of the oracle, and reuse must be refused once
the owner has exited."""
import json
import os
import select
import subprocess
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_14635_amd import harness as Hn  # noqa: E402
from paper_2608_14635_amd import kvr  # noqa: E402
from paper_2608_14635_amd import workloads as W  # noqa: E402

import parity_util as PU  # noqa: E402

pytestmark = pytest.mark.gpu
OWNER = os.path.join(os.path.dirname(os.path.abspath(__file__)), "ipc_owner.py")


def say(msg):
    print(msg, flush=True)


def read_tagged(proc, tag, timeout_s):
    """Next stdout line of `proc` starting with `tag` (the rest of it)."""
    while True:
        ready, _, _ = select.select([proc.stdout], [], [], timeout_s)
        if not ready:
            raise TimeoutError(f"owner sent no {tag} line within {timeout_s} s")
        line = proc.stdout.readline()
        if not line:
            raise RuntimeError(f"owner exited (status {proc.wait()}) before {tag}")
        if line.startswith(tag):
            return line[len(tag):].strip()


@pytest.mark.parametrize("spec", [
    {"shape": "tiny_bf16", "lens": [1, 17, 300, 129, 0, 255], "seed": 401, "wseed": 402,
     "other_live_frac": 0.25},
    {"shape": "tiny_f32", "lens": [33, 64, 7], "seed": 403, "wseed": 404, "other_live_frac": 0.5},
], ids=["tiny_bf16", "tiny_f32"])
def test_rebuild_into_state_owned_by_another_process(oracle_lib, tmp_path, spec):
    shape = W.SHAPES[spec["shape"]]
    wl = W.small_workload(shape, spec["lens"], seed=spec["seed"],
                          other_live_frac=spec["other_live_frac"])
    host_w = W.host_weights(shape, seed=spec["wseed"])
    image = W.host_arena(wl)
    say(f"ipc {spec['shape']} lens={spec['lens']}: starting the owner process")
    owner = subprocess.Popen([sys.executable, "-u", OWNER, json.dumps(spec)],
                             stdin=subprocess.PIPE, stdout=subprocess.PIPE, text=True)
    try:
        msg = json.loads(read_tagged(owner, "HANDLES ", 100))
        pool_h, arena_h = bytes.fromhex(msg["pool"]), bytes.fromhex(msg["arena"])
        info = kvr.kv_ipc_handle_info(arena_h)
        assert info["owner_pid"] == owner.pid == msg["pid"]
        assert info["bytes"] == image.nbytes
        assert kvr.kv_ipc_owner_alive(pool_h) == kvr.KV_OK

        say("  open the owner's weights and arena, bind, rebuild")
        pool = kvr.kv_ipc_open(pool_h)
        arena_ptr = kvr.kv_ipc_open(arena_h)
        lay = msg["layout"]
        weights = kvr.Weights(kvr.make_desc(shape), pool + lay["embed"],
                              [{k: pool + o for k, o in lw.items()} for lw in lay["layers"]])
        handle = kvr.kv_arena_bind(arena_ptr, info["bytes"], shape, wl.block_size,
                                   wl.num_blocks, 0)
        T = wl.total_tokens
        ws, nbytes = Hn.alloc_workspace(shape, wl.num_requests, T, max(T, 1))
        kvr.kv_rebuild(weights, wl.tokens, wl.lens, wl.block_tables, handle, ws.data_ptr(),
                       nbytes, Hn.stream_ptr())
        torch.cuda.synchronize()
        kvr.kv_arena_release(handle)
        kvr.kv_ipc_close(arena_ptr)
        kvr.kv_ipc_close(pool)

        path = str(tmp_path / "owner_arena.npy")
        owner.stdin.write(f"dump {path}\n")
        owner.stdin.flush()
        read_tagged(owner, "DUMPED", 60)
        elem = np.uint16 if shape.dtype == W.BF16 else np.uint32
        got = np.load(path).view(elem).reshape(-1)

        say("  in-process rebuild of the same request set")
        model = Hn.device_model_from_host(shape, host_w)
        local = Hn.DeviceArena(wl, host_image=image)
        local.bind()
        kvr.kv_rebuild(model.weights, wl.tokens, wl.lens, wl.block_tables, local.handle,
                       ws.data_ptr(), nbytes, Hn.stream_ptr())
        torch.cuda.synchronize()
        want = local.to_host()
        local.release()
        assert np.array_equal(got, want), "rebuild through IPC differs from the in-process one"

        ora = image.copy()
        oracle_lib.rebuild(shape, host_w, wl.tokens, wl.lens, wl.block_tables, ora,
                           wl.block_size, wl.num_blocks)
        worst, rep = PU.compare(wl, got, ora, image)
        say(f"  owner's arena vs oracle: worst {worst.max():.2e}; {rep}")
        assert rep["unwritten_changed"] == 0 and rep["written_nonfinite"] == 0
        assert rep["worst"] <= PU.TOL[shape.dtype]

        owner.stdin.write("exit\n")
        owner.stdin.flush()
        assert owner.wait(timeout=60) == 0
        say("  owner gone: reuse must be refused")
        assert kvr.kv_ipc_owner_alive(arena_h) == kvr.KV_ESTATE
        with pytest.raises(kvr.KvError) as e:
            kvr.kv_ipc_open(arena_h)
        assert e.value.status == kvr.KV_ESTATE
    finally:
        if owner.poll() is None:
            owner.kill()
            owner.wait()


def test_export_refuses_allocations_of_two_gib():
    """A handle covers its whole allocation, and allocations of 2 GiB or more
    are refused before any handle is created; a small allocation exports."""
    big = torch.empty((2 << 30) + 4096, dtype=torch.uint8, device="cuda")
    with pytest.raises(kvr.KvError) as e:
        kvr.kv_ipc_export(big.data_ptr() + 4096, 4096)
    assert e.value.status == kvr.KV_EINVAL and "2 GiB" in e.value.message
    del big
    torch.cuda.empty_cache()
    small = torch.empty(1 << 19, dtype=torch.uint8, device="cuda")  # small pool: 2 MiB segments
    assert len(kvr.kv_ipc_export(small.data_ptr(), 1 << 19)) > 0
