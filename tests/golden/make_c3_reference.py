"""Write the fp64 oracle's results for the b = 131072 workload to
tests/golden/c3_oracle.npz.

Workload: b = 131072, d = 768, bf16 inputs from the seeded generator
(sigma = 0.5, seed 0), s = 100 as the float32 value the GPU sees.  The full
oracle (forward and backward) takes several minutes on a few host cores, longer
than a test should, so its outputs are stored once:

  loss, dscale                 fp64 scalars
  lse_r, lse_c                 [b] row / column log-sum-exp (float64)
  ell_r, ell_c                 [b] per-sample terms r_i - x_ii, c_j - x_jj (float64)
  input_sha256                 hash of the generator's bf16 bits (img then txt),
                               so that a test notices a generator change

Only ``oracle`` and the input generator are called; nothing here touches the
GPU path.

    python tests/golden/make_c3_reference.py
"""

import hashlib
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2410_17243_amd import synth  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c3_oracle.npz")


def input_hash(img, txt) -> str:
    h = hashlib.sha256()
    h.update(np.ascontiguousarray(img).tobytes())
    h.update(np.ascontiguousarray(txt).tobytes())
    return h.hexdigest()


def main():
    c = synth.WORKLOADS[3]
    b, d = c["b"], c["d"]
    s = float(np.float32(c["scale"]))
    img, txt = synth.clip_pairs(b, d, c["sigma"], seed=0, dtype="bf16")
    I = synth.as_f64(img, "bf16")
    T = synth.as_f64(txt, "bf16")
    t0 = time.perf_counter()
    fwd = oracle.forward(I, T, s)
    print(f"forward {time.perf_counter() - t0:.1f} s, loss {fwd['loss']:.9e}", flush=True)
    _, _, dscale = oracle.backward(I, T, s, fwd)
    print(f"backward done {time.perf_counter() - t0:.1f} s, dscale {dscale:.9e}", flush=True)
    np.savez_compressed(OUT, loss=np.float64(fwd["loss"]), dscale=np.float64(dscale), lse_r=fwd["lse_r"],
                        lse_c=fwd["lse_c"], ell_r=fwd["ell_r"], ell_c=fwd["ell_c"], b=b, d=d, scale=s,
                        sigma=c["sigma"], input_sha256=input_hash(img, txt))
    print(f"wrote {OUT}")


if __name__ == "__main__":
    main()
