"""Parity at b = 4194304 (d = 768, s = 14.29: one GPU's full CLIP-ViT-L/14-shaped
batch) on the generator's inputs, against the exact sampled oracle.

About 100 s on an MI355X host, most of it drawing the 6.4 billion input values
and their fp64 copies (about 70 GB of host memory).  What it checks:
  * the whole forward: r_i, r_i - x_ii for 96 seeded rows and c_j, c_j - x_jj
    for 96 seeded columns against the sampled oracle (independent of the GPU),
    and the loss against the mean of the exported per-sample terms;
  * the backward of three 64-sample ranges through the shard entry point (the
    whole-batch kernels and 64-bit offsets; every own row sweeps all 4M swept
    rows), containing the first, a middle and the last sample: their dimg and
    dtxt rows against fp64 rows built from the inputs, the oracle's
    log-sum-exp of the own row and the GPU's of the other side.
"""

import numpy as np
import pytest
import torch

import oracle
import paper_2410_17243_amd as infcl
from gpu_util import device_inputs, f32_scale, grad_rows, lse_tol, max_rel, synth

pytestmark = pytest.mark.gpu


def test_sampled_b4194304_d768():
    c = synth.WORKLOADS[5]
    b, d, s = c["b"], c["d"], f32_scale(c["scale"])
    print(f"b={b} d={d} s={s}: drawing the inputs", flush=True)
    img, txt = synth.clip_pairs(b, d, c["sigma"], seed=0, dtype="bf16")
    I, T = device_inputs(img, txt, "bf16")
    sc = torch.tensor([s], dtype=torch.float32, device="cuda").reshape(())
    print("forward", flush=True)
    f = infcl.clip_loss_fwd(I, T, sc)
    torch.cuda.synchronize()
    lse_r = f["lse_r"].cpu().numpy().astype(np.float64)
    lse_c = f["lse_c"].cpu().numpy().astype(np.float64)
    aux = f["aux"].cpu().numpy().astype(np.float64)
    ell_r, ell_c = aux[:b], aux[b:2 * b]
    loss64 = float(f["loss64"].item())

    rng = np.random.default_rng(4321)
    rows = np.sort(rng.choice(b, size=96, replace=False))
    rows[0], rows[-1] = 0, b - 1
    I64 = synth.as_f64(img, "bf16")
    T64 = synth.as_f64(txt, "bf16")
    print("sampled oracle", flush=True)
    sr = oracle.sampled_rows(I64, T64, s, rows)
    sc_ = oracle.sampled_cols(I64, T64, s, rows)
    err_r = np.max(np.abs(lse_r[rows] - sr["lse"]))
    err_c = np.max(np.abs(lse_c[rows] - sc_["lse"]))
    rel_r = np.max(np.abs(ell_r[rows] - sr["ell"]) / sr["ell"])
    rel_c = np.max(np.abs(ell_c[rows] - sc_["ell"]) / sc_["ell"])
    print(f"  loss {loss64:.9e}; lse_r err {err_r:.2e} lse_c err {err_c:.2e}; "
          f"ell rel err rows {rel_r:.2e} cols {rel_c:.2e}", flush=True)
    assert np.all(np.abs(lse_r[rows] - sr["lse"]) <= lse_tol(s, d, sr["lse"]))
    assert np.all(np.abs(lse_c[rows] - sc_["lse"]) <= lse_tol(s, d, sc_["lse"]))
    assert rel_r <= 2e-2 and rel_c <= 2e-2
    assert loss64 == pytest.approx((np.sum(ell_r, dtype=np.float64) + np.sum(ell_c, dtype=np.float64)) / (2 * b),
                                   rel=1e-6)

    # the backward of three ranges of own samples around sampled indices
    mid = int(rows[len(rows) // 2])
    for r0 in (0, (mid // 32) * 32, b - 64):
        bs = 64
        own = rows[(rows >= r0) & (rows < r0 + bs)]
        print(f"backward of samples [{r0}, {r0 + bs}): sampled rows {own.tolist()}", flush=True)
        dI = torch.empty((bs, d), dtype=torch.float32, device="cuda")
        dT = torch.empty((bs, d), dtype=torch.float32, device="cuda")
        dsp = torch.empty(1, dtype=torch.float64, device="cuda")
        infcl.infcl_bwd_shard(I, T, sc, r0, bs, f["lse_r"], f["lse_c"], f["aux"], None, dI, dT, dsp, f["workspace"])
        torch.cuda.synchronize()
        k = np.searchsorted(rows, own)
        dI_ref = grad_rows(I64, T64, s, own, sr["lse"][k], lse_c, sr["ell"][k], ell_c[own], b)
        dT_ref = grad_rows(T64, I64, s, own, sc_["lse"][k], lse_r, sc_["ell"][k], ell_r[own], b)
        dIg = dI.cpu().numpy().astype(np.float64)[own - r0]
        dTg = dT.cpu().numpy().astype(np.float64)[own - r0]
        e1, e2 = max_rel(dIg, dI_ref), max_rel(dTg, dT_ref)
        print(f"  dimg rows {e1:.2e} dtxt rows {e2:.2e}", flush=True)
        assert e1 <= 2e-2 and e2 <= 2e-2
