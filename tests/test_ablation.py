"""The single-launch backward of the ablation (infcl_ablation_bwd_single:
one sweep, G' once per tile, atomic text-gradient updates) against the fp64
oracle at the parity bars, and against the two-launch backward of infcl_bwd
on the same forward outputs.  The atomic additions make dtxt order-dependent,
so the comparisons are to tolerance, not bitwise."""

import numpy as np
import pytest
import torch

import oracle
import paper_2410_17243_amd as infcl
from gpu_util import device_inputs, f32_scale, max_rel, run, synth

pytestmark = pytest.mark.gpu


def _single(I, T, s, dloss=1.0):
    sc = torch.tensor([s], dtype=torch.float32, device=I.device)
    f = infcl.clip_loss_fwd(I, T, sc)
    b, d = I.shape
    dimg = torch.empty((b, d), dtype=torch.float32, device=I.device)
    dtxt = torch.full((b, d), float("nan"), dtype=torch.float32, device=I.device)  # zeroed by the call
    ds = torch.empty((), dtype=torch.float32, device=I.device)
    dl = torch.tensor(dloss, dtype=torch.float32, device=I.device)
    infcl.infcl_ablation_bwd_single(I, T, sc.reshape(()), f["lse_r"], f["lse_c"], f["aux"], dl, dimg, dtxt, ds,
                                    f["workspace"])
    torch.cuda.synchronize()
    return dimg.cpu().numpy().astype(np.float64), dtxt.cpu().numpy().astype(np.float64), float(ds.item())


@pytest.mark.parametrize("b,d,s,sigma", [(1, 256, 14.29, 1.0), (100, 256, 14.29, 1.0), (1000, 512, 14.29, 1.0),
                                         (2100, 512, 100.0, 0.5), (777, 256, 50.0, 1.0)])
def test_single_launch_matches_oracle(b, d, s, sigma):
    img, txt = synth.clip_pairs(b, d, sigma, seed=b + d, dtype="bf16")
    s = f32_scale(s)
    I, T = device_inputs(img, txt, "bf16")
    dI, dT, ds = _single(I, T, s, dloss=0.6)
    fwd, rI, rT, rds = oracle.forward_backward(synth.as_f64(img, "bf16"), synth.as_f64(txt, "bf16"), s, dloss=0.6)
    print(f"b={b} d={d}: dI {max_rel(dI, rI):.2e} dT {max_rel(dT, rT):.2e} ds {ds:.6e} ref {rds:.6e}", flush=True)
    if b == 1:
        assert np.all(dI == 0) and np.all(dT == 0) and ds == 0
        return
    assert max_rel(dI, rI) <= 2e-2 and max_rel(dT, rT) <= 2e-2
    assert abs(ds - rds) <= 2e-2 * abs(rds) + 1e-6 * max(np.max(np.abs(rI)), 1e-30)


def test_single_launch_matches_two_launch_b32768():
    c = synth.WORKLOADS[2]
    b, d, s = c["b"], c["d"], f32_scale(c["scale"])
    img, txt = synth.clip_pairs(b, d, c["sigma"], seed=0, dtype="bf16")
    I, T = device_inputs(img, txt, "bf16")
    dI, dT, ds = _single(I, T, s)
    two = run(img, txt, "bf16", s, I=I, T=T)
    e1, e2 = max_rel(dI, two["dI"]), max_rel(dT, two["dT"])
    print(f"against infcl_bwd: dI {e1:.2e} dT {e2:.2e} ds {ds:.9e} / {two['dscale']:.9e}", flush=True)
    assert e1 <= 1e-5 and e2 <= 1e-4
    assert ds == pytest.approx(two["dscale"], rel=1e-5)
