"""Loss memory is linear in the batch size (the claim of Table 1 and Fig. 1:
the tiled loss never holds the b x b matrix).

For several b, torch's peak allocated bytes around one forward + backward
through the binding (every buffer is a torch allocation: outputs, gradients
and the workspace; the library allocates nothing) must equal what those
buffers take, and the bytes per sample must not grow with b.
"""

import pytest
import torch
import torch.nn.functional as F

import paper_2410_17243_amd as infcl

pytestmark = pytest.mark.gpu


def _round512(n):
    return max(512, (n + 511) // 512 * 512)


def _pairs(b, d, dtype):
    g = torch.Generator(device="cuda").manual_seed(b + d)
    x = torch.randn(b, d, device="cuda", generator=g)
    n = torch.randn(b, d, device="cuda", generator=g)
    return F.normalize(x, dim=1).to(dtype), F.normalize(x + n, dim=1).to(dtype)


@pytest.mark.parametrize("d,dtype,code", [(512, torch.bfloat16, infcl.INFCL_BF16),
                                          (768, torch.bfloat16, infcl.INFCL_BF16),
                                          (1024, torch.float16, infcl.INFCL_F16)])
def test_loss_memory_linear_in_b(d, dtype, code):
    sc = torch.tensor([14.29], dtype=torch.float32, device="cuda")
    per_sample = []
    for b in (8192, 16384, 32768, 65536):
        img, txt = _pairs(b, d, dtype)
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        f = infcl.clip_loss_fwd(img, txt, sc)
        dI, dT, ds = infcl.clip_loss_bwd(img, txt, sc, f)
        torch.cuda.synchronize()
        peak = torch.cuda.max_memory_allocated() - base
        ws = infcl.infcl_workspace_size(b, d, code)
        bufs = [4, 8, 4 * b, 4 * b, 12 * b, ws, 4 * b * d, 4 * b * d, 4]
        expect = sum(_round512(n) for n in bufs)
        print(f"d={d} b={b}: peak {peak} B, expected {expect} B, {peak / b:.1f} B/sample "
              f"(workspace {ws / b:.1f})", flush=True)
        # the caching allocator may hand out a block up to 1 MiB larger than asked
        assert expect <= peak <= expect + 4 * (1 << 20)
        per_sample.append(peak / b)
        del f, dI, dT, ds, img, txt
    # linear: bytes per sample settle to 8 d + 20 + workspace per sample
    assert max(per_sample[1:]) <= per_sample[1] * 1.01
    slope = 8 * d + 20 + infcl.infcl_workspace_size(1 << 20, d, code) / (1 << 20)
    assert per_sample[-1] == pytest.approx(slope, rel=0.01)
