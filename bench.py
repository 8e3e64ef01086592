#!/usr/bin/env python3
"""Benchmark of the tiled symmetric InfoNCE loss (forward + backward) on one MI355X.

A step is one full pass of the loss: infcl_fwd (similarity tiles, online
row/column log-sum-exp, per-sample terms, loss) followed by infcl_bwd (both
gradient sweeps and dscale) over one batch of synthetic CLIP-shaped embeddings
already resident in HBM.  The metric is similarity entries per second,
b^2 / (time of one forward + backward).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 3]

The default workload is b = 131072 pairs, d = 768, bf16, s = 100 (the largest
of the five configurations whose default run, 20 timed steps, finishes in a few
minutes; b = 1048576 and b = 4194304 take 8 s and 2 min per step and are run
with --config 4 / 5 and fewer steps).

Prints one JSON line.  Only one GPU is used; --gpus above 1 exits with a message.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

BF16_PEAK = 2.5e15      # MI355X dense bf16 MFMA, FLOP/s
FP32_MFMA_PEAK = 157.3e12
HBM_PEAK = 8.0e12       # MI355X HBM3E, bytes/s
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "traffic.json")
PROFILE_MFMA = os.path.join(ROOT, "profiles", "mfma_busy.json")


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3, help="workload configuration 1..5 (default 3)")
    ap.add_argument("--shards", type=int, default=1,
                    help="run each step as this many shards of the batch (one GPU's share each, "
                         "infcl_fwd_shard / _finish / infcl_bwd_shard) one after another on this device")
    ap.add_argument("--b", type=int, default=None,
                    help="batch size instead of the configuration's own (same d, input type, noise and scale; "
                         "used for counters that wrap on long launches)")
    ap.add_argument("--dtype", choices=["bf16", "f16", "f32"], default=None,
                    help="input type instead of the configuration's own (same shapes and scale)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-b", type=int, default=None,
                    help="batch size of the oracle sample timed on the host (default: the workload's b when the "
                         "oracle finishes it in about 40 s, else the largest multiple of 4096 that does in 20 s)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 256 MiB device copy three times (reference for the HBM byte counters)")
    return ap.parse_args()


def source_hash(*names) -> str:
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2410_17243_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(kernel: str, workload: str, src: str):
    """HBM bytes per launch from the committed rocprofv3 counter runs, or None
    when absent or taken on a different kernel source."""
    try:
        with open(PROFILE_TRAFFIC) as f:
            e = json.load(f)[f"{kernel}|{workload}"]
        return e["bytes_per_launch"] if e.get("source_hash") == src else None
    except (OSError, KeyError, ValueError):
        return None


def load_mfma_busy(kernel: str, d: int, src: str):
    """MFMA-pipe occupancy of the kernel at width d from the committed counter
    runs (busy cycles over elapsed cycles at the running clock), with the
    batch it was measured at; None when absent or taken on other source."""
    try:
        with open(PROFILE_MFMA) as f:
            e = json.load(f)[f"{kernel}|d={d}"]
        return {"busy": e["busy"], "measured_at": e["measured_at"], "clock_ghz": e.get("clock_ghz")} \
            if e.get("source_hash") == src else None
    except (OSError, KeyError, ValueError):
        return None


def sysfs_reading():
    """(shader clock MHz, temperature C) of card 0 from sysfs, or None where
    absent: the clock is the starred level of pp_dpm_sclk, the temperature
    the hottest hwmon sensor of the card.  Read from files; no program is run."""
    import glob
    import re
    sclk = temp = None
    for dev in sorted(glob.glob("/sys/class/drm/card*/device")):
        try:
            with open(os.path.join(dev, "pp_dpm_sclk")) as f:
                for line in f:
                    if line.rstrip().endswith("*"):
                        m = re.search(r"(\d+)\s*[Mm][Hh]z", line)
                        sclk = float(m.group(1)) if m else None
            temps = []
            for t in glob.glob(os.path.join(dev, "hwmon", "hwmon*", "temp*_input")):
                with open(t) as f:
                    temps.append(int(f.read().strip()) / 1000.0)
            temp = max(temps) if temps else None
        except (OSError, ValueError):
            continue
        if sclk is not None:
            break
    return sclk, temp


def device_info(torch):
    """Name, architecture and CU count of device 0, and its shader clock and
    temperature right after the timed steps (None where sysfs does not show
    them)."""
    pr = torch.cuda.get_device_properties(0)
    sclk, temp = sysfs_reading()
    return {"name": pr.name, "arch": getattr(pr, "gcnArchName", None), "cus": pr.multi_processor_count,
            "sclk_mhz_after": sclk, "temp_c_after": temp}


def cpu_sample_b(b, d):
    """Batch size of the oracle sample: the oracle costs about 10 b^2 d fp64
    flops plus 4 b^2 exponentials; on 16 host cores b = 24576 at d = 512 took
    18 s.  The whole batch when that estimate is under 40 s, else the largest
    multiple of 4096 estimated at 20 s."""
    def est(n):
        return 18.0 * (n / 24576.0) ** 2 * (d / 512.0)
    if est(b) <= 40.0:
        return b
    return max(4096, int(24576 * math.sqrt(20.0 / 18.0 * 512.0 / d)) // 4096 * 4096)


def cpu_baseline(cfg, sample_b):
    """The fp64 oracle (as it stands) on a bounded sample of the same workload."""
    import oracle
    from oracle.infonce import _threads
    from paper_2410_17243_amd import synth

    img, txt = synth.clip_pairs(sample_b, cfg["d"], cfg["sigma"], seed=0, dtype=cfg["dtype"])
    I = synth.as_f64(img, cfg["dtype"])
    T = synth.as_f64(txt, cfg["dtype"])
    s = float(__import__("numpy").float32(cfg["scale"]))
    t0 = time.perf_counter()
    oracle.forward_backward(I, T, s)
    dt = time.perf_counter() - t0
    return {
        "value": sample_b * sample_b / dt,
        "unit": "entries/s",
        "cores": _threads(),
        "kind": "oracle",
        "sample": (f"full fp64 oracle forward+backward at b={sample_b}" +
                   (" (the whole workload)" if sample_b == cfg["b"] else
                    f" (the first {sample_b} pairs of the b={cfg['b']} workload)") +
                   f", same generator, d={cfg['d']}, sigma={cfg['sigma']}, s={cfg['scale']}, seed 0: {dt:.2f} s"),
    }


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {a.gpus}): the library has no collective path. "
              "Its shard entry points compute one GPU's share of a batch sharded over n GPUs; "
              "--shards n times all n shares one after another on this device.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    if a.calibrate_copy:
        x = torch.empty((256 << 20) // 4, dtype=torch.float32, device="cuda:0").uniform_()
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "device copy", "bytes_per_copy": 256 << 20, "copies": 3}))
        return

    import paper_2410_17243_amd as infcl
    from paper_2410_17243_amd import synth

    cfg = dict(synth.WORKLOADS[a.config])
    if a.dtype is not None:
        cfg["dtype"] = a.dtype
    if a.b is not None:
        cfg["b"] = a.b
    b, d, dt_name = cfg["b"], cfg["d"], cfg["dtype"]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    # the largest workloads take seconds to minutes per step: say so on stderr
    # (after every forward and backward, so that no silence lasts a whole step)
    progress = b >= (1 << 20)
    t_start = time.perf_counter()

    def note(msg):
        if progress:  # with the seconds since start: per-shard times and their trend under sustained load
            print(f"[bench config {a.config} +{time.perf_counter() - t_start:.1f} s] {msg}", file=sys.stderr, flush=True)

    note("generating inputs on the host")
    img_np, txt_np = synth.clip_pairs(b, d, cfg["sigma"], seed=0, dtype=dt_name)
    if dt_name in ("bf16", "f16"):
        tdt = torch.bfloat16 if dt_name == "bf16" else torch.float16
        img = torch.from_numpy(img_np.view(np.int16)).view(tdt).to(dev)
        txt = torch.from_numpy(txt_np.view(np.int16)).view(tdt).to(dev)
    else:
        img = torch.from_numpy(img_np).to(dev)
        txt = torch.from_numpy(txt_np).to(dev)
    del img_np, txt_np
    scale = torch.tensor([cfg["scale"]], dtype=torch.float32, device=dev).reshape(())

    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats(dev)
    base_mem = torch.cuda.memory_allocated(dev)
    # outputs and workspace, allocated once (torch owns every buffer)
    ws = infcl.workspace_for(img)
    loss = torch.empty((), dtype=torch.float32, device=dev)
    loss64 = torch.empty((), dtype=torch.float64, device=dev)
    lse_r = torch.empty(b, dtype=torch.float32, device=dev)
    lse_c = torch.empty(b, dtype=torch.float32, device=dev)
    aux = torch.empty(3 * b, dtype=torch.float32, device=dev)
    dimg = torch.empty((b, d), dtype=torch.float32, device=dev)
    dtxt = torch.empty((b, d), dtype=torch.float32, device=dev)
    dscale = torch.empty((), dtype=torch.float32, device=dev)

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        infcl.infcl_fwd(img, txt, scale, loss, loss64, lse_r, lse_c, aux, ws)
        if ev is not None:
            ev[1].record()
        if progress:
            torch.cuda.synchronize()
            note("forward done")
        infcl.infcl_bwd(img, txt, scale, lse_r, lse_c, aux, None, dimg, dtxt, dscale, ws)
        if ev is not None:
            ev[2].record()

    if a.shards > 1:
        # the same step as a.shards shards, each a separate call; on very large
        # batches every shard call is waited for and reported
        from paper_2410_17243_amd import shards as shd

        del ws
        sws = [infcl.workspace_for(img) for _ in shd.shard_bounds(b, a.shards)]
        sh_out = {"lse_r": lse_r, "lse_c": lse_c, "aux": aux, "dimg": dimg, "dtxt": dtxt}

        def step(ev=None):  # noqa: F811
            def on_step(name):
                if ev is not None and name == "forward finished":
                    ev[1].record()
                if progress:
                    torch.cuda.synchronize()
                    note(name)
            if ev is not None:
                ev[0].record()
            r = shd.sharded_forward_backward(img, txt, scale, a.shards, on_step=on_step, workspaces=sws, out=sh_out)
            loss64.copy_(r["loss64"])
            if ev is not None:
                ev[2].record()

    note(f"inputs resident (b={b}, d={d}); first step")
    step()
    torch.cuda.synchronize()
    note("first step done")
    peak_bytes = torch.cuda.max_memory_allocated(dev)
    for w in range(a.warmup):
        note(f"warm-up step {w + 1}/{a.warmup}")
        step()
    torch.cuda.synchronize()

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(a.steps)]
    stream = torch.cuda.current_stream(dev)  # the stream the library launches on
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(a.steps):
        step(evs[k])
        if progress:
            torch.cuda.synchronize()
            note(f"timed step {k + 1}/{a.steps}: {evs[k][0].elapsed_time(evs[k][2]):.1f} ms")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    fwd_ms = [e[0].elapsed_time(e[1]) for e in evs]
    bwd_ms = [e[1].elapsed_time(e[2]) for e in evs]
    step_ms = [e[0].elapsed_time(e[2]) for e in evs]
    gpu_total_ms = evs[0][0].elapsed_time(evs[-1][2])
    ms_per_step = gpu_total_ms / a.steps
    ms_wall = wall * 1e3 / a.steps
    assert math.isfinite(float(loss64.item())), "non-finite loss"

    entries = float(b) * float(b)
    value = entries / (ms_per_step * 1e-3)
    bwd_launch_ms = sum(bwd_ms) / len(bwd_ms) / 2.0   # two sweep launches per infcl_bwd call
    # 16-bit inputs with d = 768 or 1024 run the single-pass wide-row sweep
    bwd_kernel = "bwd_wide" if dt_name != "f32" and d in (768, 1024) else "bwd_sweep"
    fwd_launch_ms = sum(fwd_ms) / len(fwd_ms)
    peak = FP32_MFMA_PEAK if dt_name == "f32" else BF16_PEAK  # fp16 and bf16 dense MFMA peaks are equal
    alg_bwd_launch = 3.0 * entries * d      # half of the 6 b^2 d algorithmic backward flops
    alg_fwd_launch = 2.0 * entries * d
    achieved = alg_bwd_launch / (bwd_launch_ms * 1e-3)
    workload = f"symmetric InfoNCE forward+backward, b={b} d={d} {dt_name}, sigma={cfg['sigma']}, s={cfg['scale']}"
    if a.shards > 1:
        workload += f", as {a.shards} shards"
    fwd_kernel = "fwd_sweep2" if dt_name != "f32" else "fwd_sweep"  # 16-bit widths run padded to a multiple of 128
    src = source_hash("bwd.hip", "bwd_wide.hip", "bwd.hpp", "sweep.hpp", "common.hpp")
    traffic = load_traffic(bwd_kernel, workload, src)
    # roofline bound from the arithmetic intensity: flops per HBM byte (the
    # measured bytes when the counters are current, else the compulsory ones:
    # both inputs read, one gradient written) against the ridge point
    hbm_bytes = traffic if traffic else (2.0 * b * d * img.element_size() + 4.0 * b * d)
    intensity = alg_bwd_launch / hbm_bytes
    ridge = peak / HBM_PEAK

    out = {
        "metric": "similarity entries/s (b^2 per forward+backward pass)",
        "value": value,
        "unit": "entries/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dt_name,
        "data": "synthetic (seeded CLIP-shaped unit-norm pairs; no dataset)",
        "config": {"workload": workload, "b": b, "d": d, "input_dtype": dt_name, "sigma": cfg["sigma"],
                   "scale": cfg["scale"], "seed": 0},
        "mfma_frac_algorithmic": 8.0 * entries * d / (ms_per_step * 1e-3) / peak,
        "mfma_frac_executed": 10.0 * entries * d / (ms_per_step * 1e-3) / peak,
        "fwd_ms": fwd_launch_ms,
        "bwd_ms": 2.0 * bwd_launch_ms,
        "fwd_entries_per_s": entries / (fwd_launch_ms * 1e-3),
        "bwd_entries_per_s": entries / (2.0 * bwd_launch_ms * 1e-3),
        "ms_per_step_host_wall": ms_wall,
        "step_ms_min": min(step_ms),
        "peak_hbm_bytes": int(peak_bytes - base_mem + (img.numel() + txt.numel()) * img.element_size()),
        "roofline": {
            "kernel": f"{bwd_kernel} (one of the two backward launches)",
            "bound": "mfma" if intensity >= ridge else "hbm",
            "intensity_flop_per_byte": intensity,
            "ridge_flop_per_byte": ridge,
            "achieved": achieved / 1e12,
            "peak": peak / 1e12,
            "unit": "TFLOP/s",
            "frac": achieved / peak,
            "traffic": traffic,
            "mfma_busy": load_mfma_busy(bwd_kernel, d, src),
            "algorithmic_flops_per_launch": alg_bwd_launch,
            "avg_launch_ms": bwd_launch_ms,
            "forward": {"kernel": fwd_kernel,
                        "achieved": alg_fwd_launch / (fwd_launch_ms * 1e-3) / 1e12,
                        "frac": alg_fwd_launch / (fwd_launch_ms * 1e-3) / peak, "avg_launch_ms": fwd_launch_ms,
                        "mfma_busy": load_mfma_busy(fwd_kernel, d, source_hash("fwd2.hip", "sweep.hpp", "common.hpp"))},
        },
        "cpu_baseline": None,
        "device": device_info(torch),
    }
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, min(a.cpu_sample_b or cpu_sample_b(b, d), b))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
