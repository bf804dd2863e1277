"""Owner process for the cross-process test: it holds the decoder weights and
the KV arena in its own device memory and hands them out as IPC handles, the
way independent owner processes keep retained state alive across a worker
failure (Sec. 4.1, state isolation; Sec. 6, shadow-worker integration).

    python -u ipc_owner.py '<json spec>'

Spec keys: shape (a workloads.SHAPES name), lens, seed (workload), wseed
(weights), other_live_frac.  Prints one line "HANDLES {json}" with the hex
handles of the weight pool and the arena and each weight's byte offset in the
pool, then serves stdin commands until "exit" or end of input:
    dump <path>   synchronise and save the arena bits (.npy); prints "DUMPED"
Weights go into one pool at 256-byte aligned offsets, so the importer maps a
single allocation for all of them."""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import torch  # noqa: E402

from paper_2608_14635_amd import kvr  # noqa: E402
from paper_2608_14635_amd import workloads as W  # noqa: E402


def main() -> int:
    spec = json.loads(sys.argv[1])
    shape = W.SHAPES[spec["shape"]]
    wl = W.small_workload(shape, spec["lens"], seed=spec["seed"],
                          other_live_frac=spec["other_live_frac"])
    host_w = W.host_weights(shape, seed=spec["wseed"])

    arrays, layout = [], {"embed": 0, "layers": []}
    cursor = 0

    def place(a: np.ndarray) -> int:
        nonlocal cursor
        off = cursor
        arrays.append((off, np.ascontiguousarray(a).view(np.uint8).reshape(-1)))
        cursor = (off + a.nbytes + 255) // 256 * 256
        return off

    layout["embed"] = place(host_w["embed"])
    for lw in host_w["layers"]:
        layout["layers"].append({k: place(v) for k, v in lw.items()})
    pool = torch.empty(cursor, dtype=torch.uint8, device="cuda")
    for off, a in arrays:
        pool[off:off + a.size].copy_(torch.from_numpy(a))

    image = W.host_arena(wl)
    arena = torch.from_numpy(image.view(np.uint8).copy()).to("cuda")
    torch.cuda.synchronize()

    msg = {"pool": kvr.kv_ipc_export(pool.data_ptr(), cursor).hex(),
           "arena": kvr.kv_ipc_export(arena.data_ptr(), arena.numel()).hex(),
           "layout": layout, "pid": os.getpid()}
    print("HANDLES " + json.dumps(msg), flush=True)
    for line in sys.stdin:
        cmd = line.split()
        if not cmd:
            continue
        if cmd[0] == "dump":
            torch.cuda.synchronize()
            np.save(cmd[1], arena.cpu().numpy())
            print("DUMPED", flush=True)
        elif cmd[0] == "exit":
            break
        else:
            print(f"unknown command {cmd[0]}", file=sys.stderr, flush=True)
            return 2
    torch.cuda.synchronize()
    return 0


if __name__ == "__main__":
    sys.exit(main())
