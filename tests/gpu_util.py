"""Shared helpers for the GPU tests: upload generator output, call the C ABI
through the Python binding, bring results back as numpy."""

import math

import numpy as np
import torch

import paper_2410_17243_amd as infcl
from paper_2410_17243_amd import synth


def device_inputs(img, txt, dtype):
    if dtype in ("bf16", "f16"):
        tdt = torch.bfloat16 if dtype == "bf16" else torch.float16
        I = torch.from_numpy(img.view(np.int16)).view(tdt).cuda()
        T = torch.from_numpy(txt.view(np.int16)).view(tdt).cuda()
    else:
        I = torch.from_numpy(np.ascontiguousarray(img, dtype=np.float32)).cuda()
        T = torch.from_numpy(np.ascontiguousarray(txt, dtype=np.float32)).cuda()
    return I, T


def run(img, txt, dtype, s, dloss=1.0, I=None, T=None):
    """Forward + backward through the C ABI; returns numpy results."""
    if I is None:
        I, T = device_inputs(img, txt, dtype)
    sc = torch.tensor([s], dtype=torch.float32, device=I.device)
    f = infcl.clip_loss_fwd(I, T, sc)
    dl = torch.tensor([dloss], dtype=torch.float32, device=I.device)
    dI, dT, ds = infcl.clip_loss_bwd(I, T, sc, f, dloss=dl)
    torch.cuda.synchronize()
    b = I.shape[0]
    aux = f["aux"].cpu().numpy().astype(np.float64)
    return {
        "loss": float(f["loss"].item()),
        "loss64": float(f["loss64"].item()),
        "lse_r": f["lse_r"].cpu().numpy().astype(np.float64),
        "lse_c": f["lse_c"].cpu().numpy().astype(np.float64),
        "ell_r": aux[:b],
        "ell_c": aux[b:2 * b],
        "u_diag": aux[2 * b:],
        "dI": dI.cpu().numpy().astype(np.float64),
        "dT": dT.cpu().numpy().astype(np.float64),
        "dscale": float(ds.item()),
    }


def f32_scale(s):
    """The logit scale as the float32 value the GPU sees."""
    return float(np.float32(s))


def lse_tol(s, d, ref):
    """Absolute tolerance of a float32 log-sum-exp of s*<a,b> over unit-norm bf16
    rows: fp32 accumulation of d exact products (about sqrt(d) * 2^-24 relative,
    with a x16 margin) scaled by s, plus the float32 rounding of the result."""
    return 16.0 * abs(s) * math.sqrt(d) * 2.0 ** -24 + 4.0 * 2.0 ** -24 * np.abs(ref) + 1e-6


def max_rel(a, ref):
    m = np.max(np.abs(ref))
    return float(np.max(np.abs(a - ref)) / m) if m > 0 else float(np.max(np.abs(a)))


def grad_rows(A, B, s, rows, lse_own_rows, lse_other_all, ell_own_rows, ell_other_rows, b):
    """fp64 rows of dOwn = k G' Other for own rows `rows` (own = A, other = B,
    k = s / 2b): G'_ij = exp(x_ij - lse_own_i) + exp(x_ij - lse_other_j) off
    the diagonal, expm1(-ell_own_i) + expm1(-ell_other_i) on it."""
    k = s / (2.0 * b)
    x = s * (A[rows] @ B.T)
    g = np.exp(x - lse_own_rows[:, None]) + np.exp(x - lse_other_all[None, :])
    g[np.arange(len(rows)), rows] = np.expm1(-ell_own_rows) + np.expm1(-ell_other_rows)
    return k * (g @ B)


__all__ = ["device_inputs", "run", "f32_scale", "grad_rows", "lse_tol", "max_rel", "synth"]
