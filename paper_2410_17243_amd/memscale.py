"""Peak device memory of one forward + backward against the batch size.

    python -m paper_2410_17243_amd.memscale [--d 512] [--max-b 1048576]

For each b (powers of two from 4096) it measures torch's peak allocated bytes
around one infcl forward + backward (inputs, outputs and workspace are all
torch allocations; the library allocates nothing), and the same for the
materialised-S formulation the tiled method replaces: S = s * I T^T in fp32,
cross-entropy over rows and columns with torch, autograd backward.  The
materialised baseline is run until it runs out of memory.  Inputs are the
seeded synthetic CLIP-shaped pairs generated on the device (bf16).  Prints one
JSON line per b and a summary line.
"""

from __future__ import annotations

import argparse
import json
import sys

import torch
import torch.nn.functional as F


def _pairs(b: int, d: int, sigma: float = 1.0, seed: int = 0):
    g = torch.Generator(device="cuda").manual_seed(seed)
    x = torch.randn(b, d, device="cuda", generator=g)
    n = torch.randn(b, d, device="cuda", generator=g)
    img = F.normalize(x, dim=1).to(torch.bfloat16)
    txt = F.normalize(x + sigma * n, dim=1).to(torch.bfloat16)
    return img, txt


def _peak(fn) -> tuple[int, float]:
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    torch.cuda.reset_peak_memory_stats()
    base = torch.cuda.memory_allocated()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    fn()
    e1.record()
    torch.cuda.synchronize()
    return torch.cuda.max_memory_allocated() - base, e0.elapsed_time(e1)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--d", type=int, default=512)
    ap.add_argument("--max-b", type=int, default=1 << 20)
    ap.add_argument("--scale", type=float, default=14.29)
    a = ap.parse_args()

    import paper_2410_17243_amd as infcl

    rows = []
    materialised_ok = True
    b = 4096
    while b <= a.max_b:
        img, txt = _pairs(b, a.d)
        sc = torch.tensor([a.scale], dtype=torch.float32, device="cuda").reshape(())
        in_bytes = img.numel() * img.element_size() * 2

        def tiled():
            f = infcl.clip_loss_fwd(img, txt, sc)
            infcl.clip_loss_bwd(img, txt, sc, f)

        tb, tms = _peak(tiled)
        row = {"b": b, "d": a.d, "inputs_bytes": in_bytes, "tiled_peak_bytes": tb, "tiled_ms": round(tms, 3)}
        if materialised_ok:
            def materialised():
                I = img.float().requires_grad_()
                T = txt.float().requires_grad_()
                S = a.scale * (I @ T.t())
                lab = torch.arange(b, device="cuda")
                loss = 0.5 * (F.cross_entropy(S, lab) + F.cross_entropy(S.t(), lab))
                loss.backward()

            try:
                mb, mms = _peak(materialised)
                row.update({"materialised_peak_bytes": mb, "materialised_ms": round(mms, 3)})
            except torch.cuda.OutOfMemoryError:
                materialised_ok = False
                row["materialised_peak_bytes"] = "out of memory"
                torch.cuda.empty_cache()
        rows.append(row)
        print(json.dumps(row), flush=True)
        del img, txt
        b *= 2
    per_sample = [(r["tiled_peak_bytes"]) / r["b"] for r in rows]
    print(json.dumps({"summary": "peak bytes per sample, tiled path", "min": min(per_sample),
                      "max": max(per_sample),
                      "device_bytes": torch.cuda.get_device_properties(0).total_memory}), flush=True)


if __name__ == "__main__":
    sys.exit(main())
