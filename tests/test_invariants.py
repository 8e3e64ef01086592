"""Invariants of the loss on the GPU path (no reference implementation needed):

* permuting the pairs permutes r, c, the per-sample terms and the gradient rows
  and leaves the loss and dscale unchanged;
* swapping the modalities (img <-> txt) swaps r <-> c and dimg <-> dtxt and
  leaves the loss and dscale unchanged;
* the result does not depend on how the rows are partitioned (one GPU's share
  of n shards, n = 1, 2, 3, 7, against each other);
* the calls are bitwise reproducible, for every kind of sweep (resident-rows
  and streamed forwards; 128-row and wide backwards; bf16, fp16, fp32).

The exact rewrite (Sec. 3.1, Eq. 2-5) makes these hold up to floating-point
rounding: tiles, merges and partitions only change the order of additions.
Bars: loss and dscale relative 1e-5 (fp64 accumulation of per-sample terms
that differ by fp32 merge rounding), r and c within gpu_util.lse_tol,
gradients max|diff|/max|ref| <= 2e-3 (a tenth of the parity bar: only the
rounding of G' to the 16-bit type can differ).
"""

import numpy as np
import pytest
import torch

from gpu_util import device_inputs, f32_scale, lse_tol, max_rel, run, synth
from paper_2410_17243_amd.shards import sharded_forward_backward

pytestmark = pytest.mark.gpu

CASES = [(1500, 512, "bf16"), (1100, 768, "bf16"), (900, 1024, "f16"), (700, 256, "f32")]


def _close(a, b, s, d, grad_tol=2e-3):
    assert a["loss64"] == pytest.approx(b["loss64"], rel=1e-5)
    assert np.all(np.abs(a["lse_r"] - b["lse_r"]) <= lse_tol(s, d, b["lse_r"]))
    assert np.all(np.abs(a["lse_c"] - b["lse_c"]) <= lse_tol(s, d, b["lse_c"]))
    assert max_rel(a["dI"], b["dI"]) <= grad_tol and max_rel(a["dT"], b["dT"]) <= grad_tol
    assert a["dscale"] == pytest.approx(b["dscale"], rel=1e-5, abs=1e-12)


@pytest.mark.parametrize("b,d,dtype", CASES)
def test_pair_permutation(b, d, dtype):
    img, txt = synth.clip_pairs(b, d, 1.0, seed=31, dtype=dtype)
    s = f32_scale(14.29)
    perm = np.random.default_rng(5).permutation(b)
    g = run(img, txt, dtype, s)
    p = run(img[perm], txt[perm], dtype, s)
    gp = {k: (v[perm] if isinstance(v, np.ndarray) else v) for k, v in g.items()}
    print(f"loss {g['loss64']:.12e} permuted {p['loss64']:.12e}; dI {max_rel(p['dI'], gp['dI']):.2e}", flush=True)
    _close(p, gp, s, d)


@pytest.mark.parametrize("b,d,dtype", CASES)
def test_modality_swap(b, d, dtype):
    img, txt = synth.clip_pairs(b, d, 1.0, seed=32, dtype=dtype)
    s = f32_scale(14.29)
    g = run(img, txt, dtype, s)
    w = run(txt, img, dtype, s)
    sw = dict(g)
    sw.update(lse_r=g["lse_c"], lse_c=g["lse_r"], dI=g["dT"], dT=g["dI"], ell_r=g["ell_c"], ell_c=g["ell_r"])
    print(f"loss {g['loss64']:.12e} swapped {w['loss64']:.12e}; dI {max_rel(w['dI'], sw['dI']):.2e}", flush=True)
    _close(w, sw, s, d)
    np.testing.assert_array_equal(w["u_diag"], g["u_diag"])


@pytest.mark.parametrize("d,dtype", [(512, "bf16"), (768, "bf16")])
def test_partition_count(d, dtype):
    b = 1000
    img, txt = synth.clip_pairs(b, d, 1.0, seed=33, dtype=dtype)
    s = f32_scale(14.29)
    I, T = device_inputs(img, txt, dtype)
    sc = torch.tensor([s], dtype=torch.float32, device=I.device)
    outs = []
    for n in (1, 2, 3, 7):
        o = sharded_forward_backward(I, T, sc, n)
        torch.cuda.synchronize()
        aux = o["aux"].cpu().numpy().astype(np.float64)
        outs.append({"loss64": float(o["loss64"].item()), "lse_r": o["lse_r"].cpu().numpy().astype(np.float64),
                     "lse_c": o["lse_c"].cpu().numpy().astype(np.float64), "ell_r": aux[:b],
                     "dI": o["dimg"].cpu().numpy().astype(np.float64), "dT": o["dtxt"].cpu().numpy().astype(np.float64),
                     "dscale": float(o["dscale64"].item())})
    for n, o in zip((2, 3, 7), outs[1:]):
        print(f"n={n}: loss {o['loss64']:.12e} (n=1 {outs[0]['loss64']:.12e})", flush=True)
        _close(o, outs[0], s, d)


@pytest.mark.parametrize("b,d,dtype", [(3000, 256, "bf16"), (2000, 768, "bf16"), (1500, 1024, "f16"),
                                       (1100, 512, "f32")])
def test_deterministic_bitwise(b, d, dtype):
    img, txt = synth.clip_pairs(b, d, 1.0, seed=11, dtype=dtype)
    s = f32_scale(14.29)
    a = run(img, txt, dtype, s)
    c = run(img, txt, dtype, s)
    for k in ("loss64", "loss", "dscale"):
        assert a[k] == c[k], k
    for k in ("lse_r", "lse_c", "ell_r", "ell_c", "u_diag", "dI", "dT"):
        assert np.array_equal(a[k], c[k]), k
