"""Single-launch backward ablation: what the text-gradient update of the
appendix's in-GPU backward algorithm costs on this GPU, against the two-launch
backward of infcl_bwd.

    python -m paper_2410_17243_amd.ablation [--config 2] [--reps 5]

Prints one JSON line: the two-launch backward time, the time of the dT update
traffic alone (infcl_ablation_dt_atomics, hardware fp32 atomics) for row blocks
of 128 rows (the most whose dI accumulators fit the register file at d = 512)
and 256 rows, its bytes, and the HBM-bandwidth floor of the same update done as
a plain read-modify-write (read and write of every 32 x d tile per row block at
8 TB/s).  The update alone already bounds the single-launch backward from below.
"""

from __future__ import annotations

import argparse
import json
import sys


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--reps", type=int, default=5)
    a = ap.parse_args(argv)

    import numpy as np
    import torch

    import paper_2410_17243_amd as infcl
    from paper_2410_17243_amd import synth

    cfg = synth.WORKLOADS[a.config]
    b, d = cfg["b"], cfg["d"]
    dev = torch.device("cuda:0")
    img_np, txt_np = synth.clip_pairs(b, d, cfg["sigma"], seed=0, dtype=cfg["dtype"])
    tdt = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}[cfg["dtype"]]
    if cfg["dtype"] == "f32":
        img = torch.from_numpy(img_np).to(dev)
        txt = torch.from_numpy(txt_np).to(dev)
    else:
        img = torch.from_numpy(img_np.view(np.int16)).view(tdt).to(dev)
        txt = torch.from_numpy(txt_np.view(np.int16)).view(tdt).to(dev)
    sc = torch.tensor([cfg["scale"]], dtype=torch.float32, device=dev).reshape(())
    f = infcl.clip_loss_fwd(img, txt, sc)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(a.reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / a.reps

    bwd_ms = timed(lambda: infcl.clip_loss_bwd(img, txt, sc, f))
    dT = torch.zeros((b, d), dtype=torch.float32, device=dev)
    out = {"workload": f"b={b} d={d} {cfg['dtype']}", "two_launch_backward_ms": bwd_ms, "update": []}
    for bm in (128, 256):
        dT.zero_()
        ms = timed(lambda: infcl.infcl_ablation_dt_atomics(dT, bm))
        nwg = -(-b // bm)
        want = float(nwg * (a.reps + 1))
        exact = bool(torch.all(dT == want).item())
        payload = nwg * b * d * 4  # bytes added per launch
        out["update"].append({
            "row_block": bm, "ms": ms, "atomic_payload_GiB": payload / 2**30,
            "payload_rate_TBps": payload / (ms * 1e-3) / 1e12,
            "rmw_floor_ms_at_8TBps": 2 * payload / 8e12 * 1e3, "exact": exact,
            "ratio_to_two_launch_backward": ms / bwd_ms,
        })
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
