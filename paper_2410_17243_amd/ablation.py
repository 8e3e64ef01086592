"""Single-launch backward ablation: the appendix's in-GPU backward (one sweep,
each similarity tile and its softmax weights computed once, the text-gradient
tile updated in memory for every tile, with atomics) against the two-launch
backward of infcl_bwd (two sweeps, the similarity tile recomputed, every
gradient written once).

    python -m paper_2410_17243_amd.ablation [--config 2] [--reps 5]

Prints one JSON line: the time of each backward on the workload's inputs, the
MFMA flops each executes (the single launch 6 b^2 d, the two launches
8 b^2 d), and the single launch's atomic payload (ceil(b / 64) additions of
every text-gradient element).
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
    if cfg["dtype"] != "bf16" or d not in (256, 512):
        raise SystemExit("the single-launch backward covers bf16 inputs with d = 256 or 512")
    dev = torch.device("cuda:0")
    img_np, txt_np = synth.clip_pairs(b, d, cfg["sigma"], seed=0, dtype="bf16")
    img = torch.from_numpy(img_np.view(np.int16)).view(torch.bfloat16).to(dev)
    txt = torch.from_numpy(txt_np.view(np.int16)).view(torch.bfloat16).to(dev)
    sc = torch.tensor([cfg["scale"]], dtype=torch.float32, device=dev).reshape(())
    f = infcl.clip_loss_fwd(img, txt, sc)
    ws = f["workspace"]
    dimg = torch.empty((b, d), dtype=torch.float32, device=dev)
    dtxt = torch.empty((b, d), dtype=torch.float32, device=dev)
    ds = torch.empty((), dtype=torch.float32, device=dev)

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

    two = timed(lambda: infcl.infcl_bwd(img, txt, sc, f["lse_r"], f["lse_c"], f["aux"], None, dimg, dtxt, ds, ws))
    two_ds = float(ds.item())
    one = timed(lambda: infcl.infcl_ablation_bwd_single(img, txt, sc, f["lse_r"], f["lse_c"], f["aux"], None, dimg,
                                                        dtxt, ds, ws))
    one_ds = float(ds.item())
    nwg = -(-b // 64)
    payload = nwg * b * d * 4
    out = {
        "workload": f"b={b} d={d} bf16, sigma={cfg['sigma']}, s={cfg['scale']}",
        "two_launch_backward_ms": two,
        "single_launch_backward_ms": one,
        "ratio_single_to_two": one / two,
        "executed_mfma_tflop": {"two_launch": 8.0 * b * b * d / 1e12, "single_launch": 6.0 * b * b * d / 1e12},
        "single_launch_atomic_payload_GiB": payload / 2**30,
        "single_launch_atomic_payload_rate_TBps": payload / (one * 1e-3) / 1e12,
        "dscale": {"two_launch": two_ds, "single_launch": one_ds},
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
