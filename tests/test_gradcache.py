"""Gradient-cache driver: encoder-parameter gradients against an fp64 CPU
reference (fp64 encoders, the oracle's embedding gradients), chunk-size
independence, and the memory it saves."""

import pytest
import torch

import oracle
from gpu_util import f32_scale, max_rel
from paper_2410_17243_amd.gradcache import chunks, gradcache_step


class _Enc(torch.nn.Module):
    """Small random-initialised encoder: two linear layers and L2 normalisation."""

    def __init__(self, din, hidden, dout):
        super().__init__()
        self.l1 = torch.nn.Linear(din, hidden)
        self.l2 = torch.nn.Linear(hidden, dout)

    def forward(self, x):
        y = self.l2(torch.nn.functional.gelu(self.l1(x)))
        return y / torch.linalg.vector_norm(y, dim=1, keepdim=True)


def _setup(b, din_i, din_t, hidden, dout, seed):
    torch.manual_seed(seed)
    ei, et = _Enc(din_i, hidden, dout), _Enc(din_t, hidden, dout)
    g = torch.Generator().manual_seed(seed + 1)
    xi = torch.randn((b, din_i), generator=g)
    xt = xi[:, :din_t] + 0.5 * torch.randn((b, din_t), generator=g)  # paired inputs
    return ei, et, xi, xt


def _grads(*mods):
    return [p.grad.detach().double().cpu().numpy() for m in mods for p in m.parameters()]


@pytest.mark.gpu
def test_gradcache_against_fp64_reference():
    b, s = 1000, f32_scale(14.29)
    ei, et, xi, xt = _setup(b, 64, 48, 256, 128, seed=3)
    # fp64 CPU reference: same weights, the embeddings the loss sees (bf16),
    # the oracle's gradient, backpropagated through fp64 encoders
    ei64, et64 = _Enc(64, 256, 128).double(), _Enc(48, 256, 128).double()
    ei64.load_state_dict({k: v.double() for k, v in ei.state_dict().items()})
    et64.load_state_dict({k: v.double() for k, v in et.state_dict().items()})
    ei, et = ei.cuda(), et.cuda()
    sc = torch.tensor([s], dtype=torch.float32, device="cuda")
    loss, dscale = gradcache_step(ei, et, xi.cuda(), xt.cuda(), sc, chunk=256)
    g_gpu = _grads(ei, et)
    with torch.no_grad():
        EI = ei(xi.cuda()).to(torch.bfloat16).double().cpu().numpy()
        ET = et(xt.cuda()).to(torch.bfloat16).double().cpu().numpy()
    fwd, dI, dT, ds = oracle.forward_backward(EI, ET, s)
    oi, ot = ei64(xi.double()), et64(xt.double())
    oi.backward(torch.from_numpy(dI))
    ot.backward(torch.from_numpy(dT))
    g_ref = _grads(ei64, et64)
    errs = [max_rel(a, r) for a, r in zip(g_gpu, g_ref)]
    print(f"loss {float(loss):.6e} ref {fwd['loss']:.6e}; parameter gradient errors {['%.1e' % e for e in errs]}",
          flush=True)
    assert float(loss) == pytest.approx(fwd["loss"], rel=1e-3)
    assert float(dscale) == pytest.approx(ds, rel=2e-2)
    assert max(errs) <= 2e-2


@pytest.mark.gpu
def test_gradcache_chunk_independence():
    b = 777
    ei, et, xi, xt = _setup(b, 32, 32, 128, 128, seed=5)
    ei, et = ei.cuda(), et.cuda()
    xi, xt = xi.cuda(), xt.cuda()
    sc = torch.tensor([f32_scale(20.0)], dtype=torch.float32, device="cuda")
    res = []
    for chunk in (b, 128, 100):
        for m in (ei, et):
            m.zero_grad(set_to_none=True)
        loss, ds = gradcache_step(ei, et, xi, xt, sc, chunk=chunk)
        res.append((float(loss), float(ds), _grads(ei, et)))
    for loss, ds, g in res[1:]:
        assert loss == pytest.approx(res[0][0], rel=1e-5)
        assert ds == pytest.approx(res[0][1], rel=1e-3)
        assert max(max_rel(a, r) for a, r in zip(g, res[0][2])) <= 1e-2


@pytest.mark.gpu
def test_gradcache_bounds_encoder_memory():
    """Peak device memory of one step: chunks of 1024 samples against the
    whole batch in one chunk (b = 16384, hidden width 2048)."""
    b = 16384
    ei, et, xi, xt = _setup(b, 64, 64, 2048, 256, seed=7)
    ei, et = ei.cuda(), et.cuda()
    xi, xt = xi.cuda(), xt.cuda()
    sc = torch.tensor([f32_scale(14.29)], dtype=torch.float32, device="cuda")
    peaks = {}
    for chunk in (b, 1024):
        for m in (ei, et):
            m.zero_grad(set_to_none=True)
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        gradcache_step(ei, et, xi, xt, sc, chunk=chunk)
        torch.cuda.synchronize()
        peaks[chunk] = torch.cuda.max_memory_allocated() - base
    print(f"peak bytes above resident: whole batch {peaks[b] / 2**20:.1f} MiB, chunks of 1024 "
          f"{peaks[1024] / 2**20:.1f} MiB", flush=True)
    assert peaks[1024] < 0.5 * peaks[b]


def test_chunks_cover_the_batch():
    assert chunks(10, 4) == [(0, 4), (4, 8), (8, 10)]
    assert chunks(3, 8) == [(0, 3)]
    with pytest.raises(ValueError):
        chunks(5, 0)
