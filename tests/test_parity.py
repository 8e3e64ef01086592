"""GPU path vs the fp64 oracle, element by element, on seeded synthetic inputs.

Bars (bf16 embeddings, fp32 accumulation): loss relative error <= 1e-3;
gradients max|diff| / max|ref| <= 2e-2; dscale relative <= 2e-2; the row and
column log-sum-exp within the fp32-accumulation bound of gpu_util.lse_tol.
fp32 embeddings: loss <= 1e-5 relative, gradients <= 1e-4 (the G' operand of
the second product stays fp32 there).  fp16 embeddings: the same bars as bf16
for the loss and log-sum-exp; gradients and dscale <= 2.5e-3: G' is rounded to
fp16 (unit roundoff 2^-11) instead of bf16 (2^-8), and both bars are about
five unit roundoffs of the G' type (5 * 2^-8 = 1.95e-2, 5 * 2^-11 = 2.4e-3).
"""

import math

import numpy as np
import pytest

import oracle
from gpu_util import f32_scale, lse_tol, max_rel, run, synth

pytestmark = pytest.mark.gpu


def _check(gpu, ref, dI, dT, ds, s, d, dtype, loss_tol=None, grad_tol=None):
    loss_tol = loss_tol or {"bf16": 1e-3, "f16": 1e-3, "f32": 1e-5}[dtype]
    grad_tol = grad_tol or {"bf16": 2e-2, "f16": 2.5e-3, "f32": 1e-4}[dtype]
    print(f"loss gpu {gpu['loss64']:.9e} ref {ref['loss']:.9e} | lse_r err {np.max(np.abs(gpu['lse_r'] - ref['lse_r'])):.2e}"
          f" lse_c err {np.max(np.abs(gpu['lse_c'] - ref['lse_c'])):.2e} | dI {max_rel(gpu['dI'], dI):.2e}"
          f" dT {max_rel(gpu['dT'], dT):.2e} | ds gpu {gpu['dscale']:.6e} ref {ds:.6e}", flush=True)
    assert gpu["loss64"] == pytest.approx(ref["loss"], rel=loss_tol, abs=1e-30)
    assert gpu["loss"] == pytest.approx(ref["loss"], rel=max(loss_tol, 2e-7), abs=1e-37)
    tol = lse_tol(s, d, ref["lse_r"])
    assert np.all(np.abs(gpu["lse_r"] - ref["lse_r"]) <= tol)
    assert np.all(np.abs(gpu["lse_c"] - ref["lse_c"]) <= lse_tol(s, d, ref["lse_c"]))
    assert np.all(gpu["ell_r"] >= 0) and np.all(gpu["ell_c"] >= 0)
    assert max_rel(gpu["dI"], dI) <= grad_tol
    assert max_rel(gpu["dT"], dT) <= grad_tol
    scale_g = max(np.max(np.abs(dI)), np.max(np.abs(dT)), 1e-30)
    assert abs(gpu["dscale"] - ds) <= grad_tol * abs(ds) + 1e-6 * scale_g


def _case(b, d, s, sigma=1.0, dtype="bf16", seed=0, mode="clip", dloss=1.0):
    img, txt = synth.clip_pairs(b, d, sigma, seed=seed, dtype=dtype, mode=mode)
    I = synth.as_f64(img, dtype)
    T = synth.as_f64(txt, dtype)
    s32 = f32_scale(s)
    fwd, dI, dT, ds = oracle.forward_backward(I, T, s32, dloss=dloss)
    gpu = run(img, txt, dtype, s32, dloss=dloss)
    return gpu, fwd, dI, dT, ds, s32


@pytest.mark.parametrize("b", [1, 2, 3, 17, 64, 65, 255, 256, 257, 1000, 1023, 1025, 2048])
def test_ragged_batch_bf16(b):
    gpu, fwd, dI, dT, ds, s = _case(b, 128, 14.29, seed=b)
    _check(gpu, fwd, dI, dT, ds, s, 128, "bf16")


@pytest.mark.parametrize("d", [256, 384, 512, 640, 768, 896, 1024])
def test_feature_widths_bf16(d):
    gpu, fwd, dI, dT, ds, s = _case(777, d, 14.29, seed=d)
    _check(gpu, fwd, dI, dT, ds, s, d, "bf16")


@pytest.mark.parametrize("s,sigma", [(1.0, 1.0), (14.29, 1.0), (50.0, 1.0), (100.0, 0.5)])
def test_scales_bf16(s, sigma):
    gpu, fwd, dI, dT, ds, s32 = _case(1536, 512, s, sigma=sigma, seed=7)
    _check(gpu, fwd, dI, dT, ds, s32, 512, "bf16")


def _case_bits(img, txt, s):
    """Oracle and GPU on given bf16 bit arrays."""
    I = synth.as_f64(img, "bf16")
    T = synth.as_f64(txt, "bf16")
    s32 = f32_scale(s)
    fwd, dI, dT, ds = oracle.forward_backward(I, T, s32)
    return run(img, txt, "bf16", s32), fwd, dI, dT, ds, s32


@pytest.mark.parametrize("d", [256, 768])
def test_sign_flipped_pairs_bf16(d):
    """txt_i = -img_i for a third of the pairs (in runs of 37), s = 100: the
    diagonal values sit at +-144 in base-2 units, so row and column references
    lie far apart and far above most entries (d = 768: the 4-wave forward and
    the wide backward)."""
    b = 1500
    img, _ = synth.clip_pairs(b, d, 0.3, seed=21, dtype="bf16")
    txt = img.copy()
    flip = (np.arange(b) // 37) % 3 == 0
    txt[flip] ^= np.uint16(0x8000)
    gpu, fwd, dI, dT, ds, s = _case_bits(img, txt, 100.0)
    _check(gpu, fwd, dI, dT, ds, s, d, "bf16")


@pytest.mark.parametrize("d", [384, 896])
def test_mixed_row_norms_bf16(d):
    """Rows scaled by 2^-2 .. 2^2 (exact in bf16): entries of one tile spread
    over a range several times that of unit rows."""
    b = 1300
    img, txt = synth.clip_pairs(b, d, 1.0, seed=23, dtype="bf16")
    fi = synth.as_f64(img, "bf16") * (2.0 ** ((np.arange(b) % 5) - 2))[:, None]
    ft = synth.as_f64(txt, "bf16") * (2.0 ** ((np.arange(b) * 3 % 5) - 2))[:, None]
    img2 = synth.f32_to_bf16_bits(fi.astype(np.float32))
    txt2 = synth.f32_to_bf16_bits(ft.astype(np.float32))
    gpu, fwd, dI, dT, ds, s = _case_bits(img2, txt2, 14.29)
    # entries reach 16 s in magnitude: the fp32 log-sum-exp bound scales with it
    _check(gpu, fwd, dI, dT, ds, 16.0 * s, d, "bf16")


def test_weak_positive_reading_bf16():
    """Noise added to the unit vector itself: positives barely above the negatives."""
    gpu, fwd, dI, dT, ds, s = _case(1200, 256, 14.29, mode="weak", seed=3)
    _check(gpu, fwd, dI, dT, ds, s, 256, "bf16")


def test_dloss_scaling_bf16():
    gpu, fwd, dI, dT, ds, s = _case(700, 256, 20.0, dloss=-0.37, seed=5)
    _check(gpu, fwd, dI, dT, ds, s, 256, "bf16")


@pytest.mark.parametrize("b,d", [(1, 128), (65, 128), (1025, 256), (777, 512), (777, 640), (700, 768), (600, 1024)]
                         + [(300, d) for d in range(128, 1025, 128)])
def test_fp16_inputs(b, d):
    """IEEE half embeddings (the paper's mixed-precision training type): the
    resident-rows forward (8 waves at d <= 512, 4 above), the 128-row backward
    and the wide backward (d = 768, 1024)."""
    gpu, fwd, dI, dT, ds, s = _case(b, d, 14.29, dtype="f16", seed=b + d)
    _check(gpu, fwd, dI, dT, ds, s, d, "f16")


@pytest.mark.parametrize("s,sigma", [(50.0, 1.0), (100.0, 0.5)])
def test_fp16_scales(s, sigma):
    gpu, fwd, dI, dT, ds, s32 = _case(1536, 512, s, sigma=sigma, dtype="f16", seed=11)
    _check(gpu, fwd, dI, dT, ds, s32, 512, "f16")


@pytest.mark.parametrize("b,d", [(1, 64), (17, 64), (1024, 512)] + [(300, d) for d in range(64, 513, 64)])
def test_fp32_inputs(b, d):
    gpu, fwd, dI, dT, ds, s = _case(b, d, 1.0 / 0.07, dtype="f32", seed=b)
    _check(gpu, fwd, dI, dT, ds, s, d, "f32")


def test_config1_fp32_workload():
    """b=1024, d=512, fp32, sigma=1, s=1/0.07, seed 0: the whole small workload."""
    c = synth.WORKLOADS[1]
    gpu, fwd, dI, dT, ds, s = _case(c["b"], c["d"], c["scale"], sigma=c["sigma"], dtype="f32", seed=0)
    _check(gpu, fwd, dI, dT, ds, s, c["d"], "f32")


@pytest.mark.parametrize("d,dtype", [(8, "bf16"), (72, "bf16"), (200, "bf16"), (1000, "bf16"), (24, "f16"),
                                     (520, "f16"), (4, "f32"), (36, "f32"), (100, "f32"), (500, "f32")])
def test_widths_between_kernel_widths(d, dtype):
    """Widths the sweeps are not built for (16-bit: not a multiple of 128; f32:
    not a multiple of 64) go through the C ABI as they are: the library runs
    the sweeps on zero-padded copies and drops the padding's gradients.  Zero
    features add nothing to any dot product, so the results are those of the
    unpadded batch (checked against the oracle at d) and, bit for bit, those
    of the same inputs padded by the caller (the same kernels on the same
    values)."""
    b = 513
    img, txt = synth.clip_pairs(b, d, 1.0, seed=d, dtype=dtype)
    s = f32_scale(14.29)
    gpu = run(img, txt, dtype, s)
    fwd, dI, dT, ds = oracle.forward_backward(synth.as_f64(img, dtype), synth.as_f64(txt, dtype), s)
    assert gpu["dI"].shape == (b, d) and gpu["dT"].shape == (b, d)
    _check(gpu, fwd, dI, dT, ds, s, d, dtype)
    q = 64 if dtype == "f32" else 128
    dp = -(-d // q) * q
    pi = np.zeros((b, dp), dtype=img.dtype)
    pt = np.zeros((b, dp), dtype=txt.dtype)
    pi[:, :d] = img
    pt[:, :d] = txt
    padded = run(pi, pt, dtype, s)
    assert np.all(padded["dI"][:, d:] == 0) and np.all(padded["dT"][:, d:] == 0)
    for k in ("loss64", "loss", "dscale"):
        assert gpu[k] == padded[k], k
    for k in ("lse_r", "lse_c", "ell_r", "ell_c", "u_diag"):
        np.testing.assert_array_equal(gpu[k], padded[k], err_msg=k)
    np.testing.assert_array_equal(gpu["dI"], padded["dI"][:, :d])
    np.testing.assert_array_equal(gpu["dT"], padded["dT"][:, :d])


@pytest.mark.parametrize("b,d,dtype", [(777, 512, "bf16"), (700, 768, "bf16"), (600, 1024, "f16"), (513, 384, "f16"),
                                       (513, 200, "bf16")])
def test_gradients_in_the_input_type(b, d, dtype):
    """Gradient type = the inputs' 16-bit type (the 128-row sweep at d = 384
    and 512, the wide sweeps at 768 and 1024, a zero-padded width at 200): the
    kernels round the fp32 accumulators once, to nearest even, when storing,
    so the 16-bit gradients are the fp32 gradients of the same inputs rounded
    (torch's cast), bit for bit, on the whole batch, on a shard and through
    the autograd function; dscale does not change."""
    import torch

    import paper_2410_17243_amd as infcl
    from gpu_util import device_inputs

    img, txt = synth.clip_pairs(b, d, 1.0, seed=b + d, dtype=dtype)
    I, T = device_inputs(img, txt, dtype)
    sc = torch.tensor([f32_scale(14.29)], dtype=torch.float32, device=I.device)
    f = infcl.clip_loss_fwd(I, T, sc)
    dl = torch.tensor([0.7], dtype=torch.float32, device=I.device)
    g32 = infcl.clip_loss_bwd(I, T, sc, f, dloss=dl)
    g16 = infcl.clip_loss_bwd(I, T, sc, f, dloss=dl, grad_dtype=I.dtype)
    assert g16[0].dtype == g16[1].dtype == I.dtype
    assert torch.equal(g16[0], g32[0].to(I.dtype)) and torch.equal(g16[1], g32[1].to(I.dtype))
    assert torch.equal(g16[2], g32[2])
    # a shard of own rows [64, 64 + 300)
    r0, bs = 64, 300
    ds = torch.empty((), dtype=torch.float64, device=I.device)
    s32 = [torch.empty((bs, d), dtype=torch.float32, device=I.device) for _ in range(2)]
    s16 = [torch.empty((bs, d), dtype=I.dtype, device=I.device) for _ in range(2)]
    for out in (s32, s16):
        infcl.infcl_bwd_shard(I, T, sc.reshape(()), r0, bs, f["lse_r"], f["lse_c"], f["aux"], None, out[0], out[1], ds,
                              f["workspace"])
    assert torch.equal(s16[0], s32[0].to(I.dtype)) and torch.equal(s16[1], s32[1].to(I.dtype))
    # the autograd function returns gradients in the inputs' dtype
    Ia, Ta = I.clone().requires_grad_(), T.clone().requires_grad_()
    sa = sc.reshape(()).clone().requires_grad_()
    infcl.clip_loss(Ia, Ta, sa).backward()
    ref = infcl.clip_loss_bwd(I, T, sc, f)
    assert Ia.grad.dtype == I.dtype
    assert torch.equal(Ia.grad, ref[0].to(I.dtype)) and torch.equal(Ta.grad, ref[1].to(I.dtype))
    torch.cuda.synchronize()
