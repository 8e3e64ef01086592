"""GPU path vs closed forms that hold at any size (inputs exact in bf16).

A: identical embeddings: every x_ij = s, so r_i = c_j = s + log b and L = log b.
B: one-hot pairs I_i = T_i = e_i (d >= b): L = log1p((b-1) e^{-s}), exact even
   where L is far below the float range (s = 100); dscale = -(b-1)/(e^s + b - 1).
C: periodic one-hot I_i = T_i = e_{i mod d} (b > d): with n_i the size of i's
   class, r_i = c_i = log(n_i e^s + b - n_i), and the gradients have per-class
   closed forms; this covers the full path (all tiles, partial merges, ragged
   ends) at the benchmark shapes.
"""

import math

import numpy as np
import pytest
import torch

from gpu_util import f32_scale, lse_tol, max_rel, run

pytestmark = pytest.mark.gpu


def _onehot(b, d, period):
    I = np.zeros((b, d), dtype=np.uint16)
    I[np.arange(b), np.arange(b) % period] = 0x3F80  # bf16 1.0
    return I


@pytest.mark.parametrize("b,s", [(1000, 14.29), (4097, 100.0), (32768, 14.29)])
def test_A_identical(b, s):
    d = 128
    I = np.zeros((b, d), dtype=np.uint16)
    I[:, 5] = 0x3F80
    g = run(I, I.copy(), "bf16", f32_scale(s))
    assert g["loss64"] == pytest.approx(math.log(b), rel=1e-6)
    np.testing.assert_allclose(g["lse_r"], f32_scale(s) + math.log(b), rtol=1e-6)
    np.testing.assert_allclose(g["lse_c"], f32_scale(s) + math.log(b), rtol=1e-6)
    # exact gradient is 0; what remains is bf16 rounding of G' = 2/b, summed over a row
    k = f32_scale(s) / (2 * b)
    assert np.max(np.abs(g["dI"])) <= 2 * k * 2.0 ** -8 * 2
    assert abs(g["dscale"]) <= 1e-6


def _closed_B(b, s):
    Z = math.exp(s) + b - 1
    return math.log1p((b - 1) * math.exp(-s)), math.log(Z), -(b - 1) / Z, (s / b) * (-(b - 1) / Z), (s / b) / Z


@pytest.mark.parametrize("b,d,s", [(128, 128, 100.0), (100, 128, 14.29), (512, 512, 50.0), (1000, 1024, 100.0)])
def test_B_one_hot_pairs(b, d, s):
    s32 = f32_scale(s)
    I = _onehot(b, d, d)
    g = run(I, I.copy(), "bf16", s32)
    loss, lse, ds, gdiag, goff = _closed_B(b, s32)
    assert g["loss64"] == pytest.approx(loss, rel=1e-3)
    np.testing.assert_allclose(g["lse_r"], lse, rtol=1e-6)
    np.testing.assert_allclose(g["lse_c"], lse, rtol=1e-6)
    if s <= 20:  # at larger s the exact gradients are below the float range
        assert abs(g["dscale"] - ds) <= 2e-2 * abs(ds) + 2.0 ** -120
        ref = np.full((b, b), goff)
        np.fill_diagonal(ref, gdiag)
        assert max_rel(g["dI"][:, :b], ref) <= 2e-2
        assert max_rel(g["dT"][:, :b], ref) <= 2e-2


def _closed_C(b, d, s):
    """Closed forms for periodic one-hot inputs, plus the per-element error
    bound of the GPU's arithmetic: bf16 rounding of every G' term (relative
    2^-9) in the second product, and float exponentials that flush results
    below 2^-126 to zero:  bound[i, f] = (s/2b) (2^-9 sum_j |G'_ij| |T_jf| + 2^-120)."""
    cls = np.arange(b) % d
    n = np.bincount(cls, minlength=d).astype(np.float64)
    es = math.exp(s)
    Zc = n * es + (b - n)
    r = np.log(Zc)[cls]
    ell = np.log(n + (b - n) * math.exp(-s))           # r_i - s per class
    loss = math.fsum(r - s) / b
    coef = np.zeros((d, d))   # coef[class of i][class kappa]
    absg = np.zeros((d, d))   # sum_j |G'_ij| over j in class kappa (before the s/2b factor)
    for c in range(d):
        row = n * (1.0 / Zc[c] + 1.0 / Zc) / (2 * b)
        row[c] = -(b - n[c]) / (b * Zc[c])      # n e^s / (b Z) - 1/b without cancellation
        coef[c] = s * row
        a = n * (1.0 / Zc[c] + 1.0 / Zc)
        a[c] = (n[c] - 1) * 2 * es / Zc[c] + abs(2 * math.expm1(-ell[c]))
        absg[c] = a
    ds = -(1.0 / b) * math.fsum((b - n[cls]) / Zc[cls])
    bound = (s / (2 * b)) * (2.0 ** -9 * absg[cls] + 2.0 ** -120)
    return loss, r, coef[cls], ds, bound


@pytest.mark.parametrize("b,d,s", [(32768, 512, 14.29), (131072, 768, 100.0), (163840, 768, 50.0), (5000, 128, 50.0),
                                   (33000, 256, 14.29)])
def test_C_periodic_one_hot(b, d, s):
    s32 = f32_scale(s)
    I = _onehot(b, d, d)
    g = run(I, I.copy(), "bf16", s32)
    loss, r, dI, ds, bound = _closed_C(b, d, s32)
    excess_I = np.max(np.abs(g["dI"] - dI) / (bound + 1e-3 * np.max(np.abs(dI))))
    excess_T = np.max(np.abs(g["dT"] - dI) / (bound + 1e-3 * np.max(np.abs(dI))))
    # at s = 100 the exact gradients (~1e-44) are below the float range: the
    # check then reduces to "within the rounding bound of zero"
    print(f"C b={b} d={d} s={s}: loss {g['loss64']:.9e} vs {loss:.9e}, dI err/bound {excess_I:.2e}, "
          f"dT err/bound {excess_T:.2e}, ds {g['dscale']:.6e} vs {ds:.6e}", flush=True)
    assert g["loss64"] == pytest.approx(loss, rel=1e-4)
    assert np.all(np.abs(g["lse_r"] - r) <= lse_tol(s32, d, r))
    assert np.all(np.abs(g["lse_c"] - r) <= lse_tol(s32, d, r))
    # Identical embeddings make the own-class gradient a difference of nearly
    # equal sums, so the bar is the bf16 rounding bound of G', element by element
    # (plus 1e-3 of the largest entry for the fp32 exponentials and accumulation).
    assert excess_I <= 1.0 and excess_T <= 1.0
    assert abs(g["dscale"] - ds) <= 2e-2 * abs(ds) + 2.0 ** -120


def _device_onehot(b, d):
    x = torch.zeros(b, d, dtype=torch.bfloat16, device="cuda")
    i = torch.arange(b, device="cuda")
    x[i, i % d] = 1.0
    return x


def _check_C_on_device(b, d, s32, f, grads=None):
    """Closed form C checked on the device, rows in chunks (the full-size
    matrices stay on the GPU; only maxima come back)."""
    n = np.bincount(np.arange(b) % d, minlength=d).astype(np.float64)
    es = math.exp(s32)
    Zc = n * es + (b - n)
    loss = math.fsum(n * np.log(n + (b - n) * math.exp(-s32))) / b
    r_cls = torch.tensor(np.log(Zc), dtype=torch.float64, device="cuda")
    tol_cls = torch.tensor(lse_tol(s32, d, np.log(Zc)), dtype=torch.float64, device="cuda")
    assert f["loss64"].item() == pytest.approx(loss, rel=1e-4)
    idx = torch.arange(b, device="cuda") % d
    for key in ("lse_r", "lse_c"):
        err = (f[key].double() - r_cls[idx]).abs() - tol_cls[idx]
        assert err.max().item() <= 0.0, key
    if grads is None:
        return
    dI, dT, dscale = grads
    ds_ref = -(1.0 / b) * math.fsum(n * (b - n) / Zc)
    assert abs(dscale - ds_ref) <= 2e-2 * abs(ds_ref) + 2.0 ** -120
    worst = max(_check_C_grad_rows(b, d, s32, g, 0) for g in (dI, dT))
    print(f"  closed form C at b={b}: gradient error / bound {worst:.2e}", flush=True)
    assert worst <= 1.0


def _check_C_grad_rows(b, d, s32, g, r0):
    """Largest |g - closed form C| / bound over the rows of g, which hold the
    gradients of samples r0, r0 + 1, ... (class (r0 + i) mod d)."""
    n = np.bincount(np.arange(b) % d, minlength=d).astype(np.float64)
    es = math.exp(s32)
    Zc = n * es + (b - n)
    # per class c: expected row coef[c] and bound[c] (see _closed_C)
    coef = np.zeros((d, d))
    absg = np.zeros((d, d))
    ell = np.log(n + (b - n) * math.exp(-s32))
    for c in range(d):
        row = n * (1.0 / Zc[c] + 1.0 / Zc) / (2 * b)
        row[c] = -(b - n[c]) / (b * Zc[c])
        coef[c] = s32 * row
        a = n * (1.0 / Zc[c] + 1.0 / Zc)
        a[c] = (n[c] - 1) * 2 * es / Zc[c] + abs(2 * math.expm1(-ell[c]))
        absg[c] = a
    bound = (s32 / (2 * b)) * (2.0 ** -9 * absg + 2.0 ** -120)
    coef_t = torch.tensor(coef, dtype=torch.float64, device="cuda")
    slack = torch.tensor(bound + 1e-3 * np.max(np.abs(coef)), dtype=torch.float64, device="cuda")
    worst = 0.0
    for c0 in range(0, g.shape[0], 65536):
        c1 = min(g.shape[0], c0 + 65536)
        c = (torch.arange(c0, c1, device="cuda") + r0) % d
        worst = max(worst, ((g[c0:c1].double() - coef_t[c]).abs() / slack[c]).max().item())
    return worst


@pytest.mark.parametrize("b,d,s,with_bwd", [(1048576, 1024, 50.0, True), (4194304, 768, 14.29, False)])
def test_C_periodic_full_size(b, d, s, with_bwd):
    """Closed form C at the two largest workloads, inputs built on the device:
    b = 1M, d = 1024, s = 50 forward and backward; b = 4M, d = 768 forward and
    the backward of two ranges of own samples (the whole backward takes
    minutes; every own row sweeps all 4M swept rows either way)."""
    import paper_2410_17243_amd as infcl

    s32 = f32_scale(s)
    I = _device_onehot(b, d)
    T = I.clone()
    sc = torch.tensor([s32], dtype=torch.float32, device="cuda").reshape(())
    print(f"closed form C at b={b} d={d} s={s}: forward", flush=True)
    f = infcl.clip_loss_fwd(I, T, sc)
    torch.cuda.synchronize()
    grads = None
    if with_bwd:
        print("  backward", flush=True)
        dI, dT, dscale = infcl.clip_loss_bwd(I, T, sc, f)
        torch.cuda.synchronize()
        grads = (dI, dT, float(dscale.item()))
    _check_C_on_device(b, d, s32, f, grads)
    if not with_bwd:
        # the backward for two ranges of own samples against all b swept
        # samples (the shard entry point; same kernels and 64-bit offsets as
        # the whole-batch backward): the last 65536 samples, and a ragged
        # range in the middle; dscale_part is the range's share of dL/ds
        n = np.bincount(np.arange(b) % d, minlength=d).astype(np.float64)
        Zc = n * math.exp(s32) + (b - n)
        for r0, bs in ((b - 65536, 65536), (b // 2 + 32 * 7, 65523)):
            print(f"  backward of samples [{r0}, {r0 + bs})", flush=True)
            dI = torch.empty((bs, d), dtype=torch.float32, device="cuda")
            dT = torch.empty((bs, d), dtype=torch.float32, device="cuda")
            dsp = torch.empty(1, dtype=torch.float64, device="cuda")
            infcl.infcl_bwd_shard(I, T, sc, r0, bs, f["lse_r"], f["lse_c"], f["aux"], None, dI, dT, dsp,
                                  f["workspace"])
            torch.cuda.synchronize()
            worst = max(_check_C_grad_rows(b, d, s32, g, r0) for g in (dI, dT))
            cls = np.arange(r0, r0 + bs) % d
            ds_ref = -(1.0 / b) * math.fsum((b - n[cls]) / Zc[cls])
            print(f"    gradient error / bound {worst:.2e}; dscale part {dsp.item():.6e} vs {ds_ref:.6e}", flush=True)
            assert worst <= 1.0
            assert abs(dsp.item() - ds_ref) <= 2e-2 * abs(ds_ref)
