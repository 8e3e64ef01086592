"""The C ABI under HIP graph capture: the library allocates nothing and clears
nothing with memset nodes, so a captured forward + backward replays to the
same bits as the eager calls, replay after replay."""

import pytest
import torch

import paper_2410_17243_amd as infcl
from gpu_util import device_inputs, synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("b,d,dtype,grad16", [(1000, 512, "bf16", False), (777, 768, "bf16", False),
                                              (600, 256, "f16", False),
                                              (513, 200, "bf16", True)])  # padded width, bf16 gradients
def test_captured_step_replays_bitwise(b, d, dtype, grad16):
    img, txt = synth.clip_pairs(b, d, 1.0, seed=31, dtype=dtype)
    I, T = device_inputs(img, txt, dtype)
    dev = I.device
    sc = torch.tensor([14.29], dtype=torch.float32, device=dev).reshape(())
    dl = torch.tensor([0.5], dtype=torch.float32, device=dev).reshape(())
    ws = infcl.workspace_for(I)
    out = {
        "loss": torch.empty((), dtype=torch.float32, device=dev),
        "loss64": torch.empty((), dtype=torch.float64, device=dev),
        "lse_r": torch.empty(b, dtype=torch.float32, device=dev),
        "lse_c": torch.empty(b, dtype=torch.float32, device=dev),
        "aux": torch.empty(3 * b, dtype=torch.float32, device=dev),
        "dimg": torch.empty((b, d), dtype=I.dtype if grad16 else torch.float32, device=dev),
        "dtxt": torch.empty((b, d), dtype=I.dtype if grad16 else torch.float32, device=dev),
        "dscale": torch.empty((), dtype=torch.float32, device=dev),
    }

    def step():
        infcl.infcl_fwd(I, T, sc, out["loss"], out["loss64"], out["lse_r"], out["lse_c"], out["aux"], ws)
        infcl.infcl_bwd(I, T, sc, out["lse_r"], out["lse_c"], out["aux"], dl, out["dimg"], out["dtxt"],
                        out["dscale"], ws)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in out.items()}

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        for v in out.values():  # eager work between replays: clobber every output
            v.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in out:
            assert torch.equal(out[k], ref[k]), (rep, k)
