"""Python binding: checks made before anything reaches the library (wrong
sizes, types and devices raise instead of handing the kernels bad pointers)."""

import pytest
import torch

import paper_2410_17243_amd as infcl
from gpu_util import device_inputs, synth


def test_host_tensors_are_rejected():
    x = torch.zeros((4, 128), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        infcl.clip_loss_fwd(x, x, torch.ones((), dtype=torch.float32))


@pytest.mark.gpu
def test_backward_checks_forward_tensors_and_workspace():
    b, d = 300, 128
    img, txt = synth.clip_pairs(b, d, 1.0, seed=8, dtype="bf16")
    I, T = device_inputs(img, txt, "bf16")
    sc = torch.tensor(14.29, dtype=torch.float32, device=I.device)
    f = infcl.clip_loss_fwd(I, T, sc)
    for key, bad in [("lse_r", f["lse_r"][:-1]), ("lse_c", f["lse_c"].double()), ("aux", f["aux"][: 2 * b]),
                     ("lse_r", f["lse_r"].cpu())]:
        g = dict(f)
        g[key] = bad
        with pytest.raises(ValueError):
            infcl.clip_loss_bwd(I, T, sc, g)
    with pytest.raises(ValueError):
        infcl.clip_loss_bwd(I, T, sc, f, dloss=torch.ones(2, device=I.device))
    with pytest.raises(ValueError):
        infcl.clip_loss_bwd(I, T, sc, f, workspace=f["workspace"].cpu())
    with pytest.raises(ValueError):
        infcl.clip_loss_fwd(I, T, sc, workspace=torch.empty(16, dtype=torch.float32, device=I.device))
    # a workspace on the right device but too small is the library's error
    with pytest.raises(infcl.InfclError):
        infcl.clip_loss_fwd(I, T, sc, workspace=torch.empty(256, dtype=torch.uint8, device=I.device))
    # the valid call still works after the rejected ones
    dI, dT, ds = infcl.clip_loss_bwd(I, T, sc, f)
    torch.cuda.synchronize()
    assert torch.isfinite(dI).all() and torch.isfinite(dT).all() and torch.isfinite(ds)
