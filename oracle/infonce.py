"""fp64 oracle: symmetric InfoNCE loss and its gradients, written from the definition.

TEST INFRASTRUCTURE ONLY (see the package docstring): the product path never
imports this module.

Notation (paper Sec. 2.2, Eq. 1; the paper writes c for the feature width):
  I, T      image / text features, shape [b, d], used exactly as given
            (no normalisation inside the loss);
  s         the logit scale (1/temperature), omitted in Eq. 1 "for simplicity";
  x_ij      s * <I_i, T_j>, the scaled similarity;
  r_i       log sum_j exp(x_ij)          (row log-sum-exp, Eq. 2's second term)
  c_j       log sum_i exp(x_ij)          (column log-sum-exp, the symmetric half)
  L         (1/2b) * ( sum_i (r_i - x_ii) + sum_j (c_j - x_jj) )
            i.e. the mean of Eq. 1's image->text loss and its text->image twin.

Readings taken where the paper is silent or loose (each is pinned by a test):
  * weighting of the two directions: their mean (Eq. 1 defines one direction and
    calls the other symmetric);
  * the scale multiplies the dot product; dscale is dL/ds for s itself;
  * positives are the diagonal (Eq. 1's x_ii); any other equal pair is a negative.

Cancellation-free but exact rewrites (no approximation is made anywhere):
  * r_i - x_ii = softplus(LSE_{j != i} x_ij - x_ii), so each per-sample term is
    computed from the off-diagonal log-sum-exp (Eq. 2's two parts never get
    subtracted as large numbers);
  * dL/dx_ij = (1/2b)(P^r_ij + P^c_ij) - (1/b) delta_ij with
    P^r_ij = exp(x_ij - r_i), P^c_ij = exp(x_ij - c_j) (Eq. 6-7 completed);
    on the diagonal P^r_ii - 1 = expm1(-(r_i - x_ii));
  * dL/ds = (1/2b) sum_{i != j} [P^r_ij + P^c_ij ... ] written with differences
    (u_ij - u_ii) of the unscaled dot products u = <I_i, T_j>, using that each
    row of P^r and each column of P^c sums to one.

The similarity matrix is materialised in blocks of whole rows (plain dense
algebra, no online merging): rows are complete inside one block, and the
column statistics take two passes (max first, then the shifted sum), which is
the textbook stable log-sum-exp, not the paper's serial merge of Eq. 4.
"""

from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_BLOCK_BYTES = 128 << 20  # bytes of one fp64 block of whole rows of S


def _threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return max(1, os.cpu_count() or 1)


def _row_blocks(b: int):
    rows = max(1, min(b, _BLOCK_BYTES // (8 * max(b, 1))))
    return [(r0, min(b, r0 + rows)) for r0 in range(0, b, rows)]


def _as64(a) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype != np.float64:
        a = a.astype(np.float64)
    return np.ascontiguousarray(a)


def softplus(z):
    """log(1 + e^z), evaluated without overflow or cancellation."""
    z = np.asarray(z, dtype=np.float64)
    return np.maximum(z, 0.0) + np.log1p(np.exp(-np.abs(z)))


def _pmap(fn, items, threads):
    if threads <= 1 or len(items) <= 1:
        return [fn(it) for it in items]
    with ThreadPoolExecutor(max_workers=threads) as ex:
        return list(ex.map(fn, items))


def forward(I, T, s, threads: int | None = None) -> dict:
    """Loss, row/column log-sum-exp and per-sample terms (Eq. 1-2, symmetric).

    Returns a dict with (all fp64):
      loss     scalar L
      lse_r    r_i = log sum_j exp(x_ij)
      lse_c    c_j = log sum_i exp(x_ij)
      ell_r    r_i - x_ii  (row per-sample loss, >= 0)
      ell_c    c_j - x_jj  (column per-sample loss, >= 0)
      x_diag   x_ii
      u_diag   <I_i, T_i>  (unscaled)
    """
    I = _as64(I)
    T = _as64(T)
    s = float(s)
    b, d = I.shape
    assert T.shape == (b, d)
    threads = threads or _threads()
    blocks = _row_blocks(b)

    def pass_rows(blk):
        r0, r1 = blk
        u = I[r0:r1] @ T.T                      # unscaled dot products
        x = s * u                               # x_ij of Eq. 1
        idx = np.arange(r0, r1)
        u_diag = u[idx - r0, idx].copy()
        x_diag = x[idx - r0, idx].copy()
        x[idx - r0, idx] = -np.inf              # off-diagonal view
        m = np.max(x, axis=1)                   # row max over j != i
        safe = np.where(np.isfinite(m), m, 0.0)
        with np.errstate(divide="ignore"):     # b == 1: empty off-diagonal set -> -inf
            lse_off = safe + np.log(np.sum(np.exp(x - safe[:, None]), axis=1))
        col_max = np.max(x, axis=0)             # column max over this block's i != j
        return u_diag, x_diag, lse_off, col_max

    res = _pmap(pass_rows, blocks, threads)
    u_diag = np.concatenate([r[0] for r in res]) if b else np.zeros(0)
    x_diag = np.concatenate([r[1] for r in res]) if b else np.zeros(0)
    lse_off_r = np.concatenate([r[2] for r in res]) if b else np.zeros(0)
    col_max = np.full(b, -np.inf)
    for r in res:
        col_max = np.maximum(col_max, r[3])
    col_safe = np.where(np.isfinite(col_max), col_max, 0.0)

    def pass_cols(blk):
        r0, r1 = blk
        x = s * (I[r0:r1] @ T.T)
        idx = np.arange(r0, r1)
        x[idx - r0, idx] = -np.inf
        return np.sum(np.exp(x - col_safe[None, :]), axis=0)

    col_sum = np.zeros(b)
    for part in _pmap(pass_cols, blocks, threads):   # fixed block order
        col_sum += part
    with np.errstate(divide="ignore"):
        lse_off_c = col_safe + np.log(col_sum)

    # Per-sample terms: r_i - x_ii = softplus(LSE_{j!=i} x_ij - x_ii); an empty
    # off-diagonal set (b == 1) gives LSE = -inf and a zero term.
    ell_r = softplus(lse_off_r - x_diag)
    ell_c = softplus(lse_off_c - x_diag)
    loss = (math.fsum(ell_r) + math.fsum(ell_c)) / (2.0 * b) if b else 0.0
    return {
        "loss": loss,
        "lse_r": x_diag + ell_r,
        "lse_c": x_diag + ell_c,
        "ell_r": ell_r,
        "ell_c": ell_c,
        "x_diag": x_diag,
        "u_diag": u_diag,
    }


def backward(I, T, s, fwd: dict, dloss: float = 1.0, threads: int | None = None):
    """Exact gradients (dI, dT, dscale) of dloss * L.

    Chain rule of Eq. 6 with dL/dx_ij = (1/2b)(P^r_ij + P^c_ij) - (1/b) delta_ij,
    which for the image->text half alone reduces to Eq. 7's closed form
    (-T_i + sum_j e^{x_ij - l_i} T_j)/b; dx_ij/dI_i = s T_j, dx_ij/dT_j = s I_i,
    dx_ij/ds = u_ij.
    """
    I = _as64(I)
    T = _as64(T)
    s = float(s)
    b, d = I.shape
    threads = threads or _threads()
    lse_r, lse_c = fwd["lse_r"], fwd["lse_c"]
    ell_r, ell_c, u_diag = fwd["ell_r"], fwd["ell_c"], fwd["u_diag"]
    k = dloss * s / (2.0 * b)

    def blk_grad(blk):
        r0, r1 = blk
        u = I[r0:r1] @ T.T
        x = s * u
        idx = np.arange(r0, r1)
        pr = np.exp(x - lse_r[r0:r1, None])     # P^r
        pc = np.exp(x - lse_c[None, :])         # P^c
        g = pr + pc                             # 2b * dL/dx off the diagonal
        g[idx - r0, idx] = np.expm1(-ell_r[r0:r1]) + np.expm1(-ell_c[r0:r1])
        # dscale pieces, with the diagonal terms (which are zero) removed
        du_r = u - u_diag[r0:r1, None]
        du_c = u - u_diag[None, :]
        pr_off = pr.copy()
        pc_off = pc.copy()
        pr_off[idx - r0, idx] = 0.0
        pc_off[idx - r0, idx] = 0.0
        ds_part = math.fsum(np.sum(pr_off * du_r, axis=1)) + math.fsum(np.sum(pc_off * du_c, axis=1))
        dI_blk = k * (g @ T)
        dT_part = k * (g.T @ I[r0:r1])
        return dI_blk, dT_part, ds_part

    blocks = _row_blocks(b)
    dI = np.zeros((b, d))
    dT = np.zeros((b, d))
    ds_parts = []
    # blocks in groups of `threads`, each group's results added in block order
    # before the next group starts: a block's dT part is a whole [b, d] array,
    # so holding every block's part at once would need (b / rows) b d 8 bytes
    for g0 in range(0, len(blocks), threads):
        group = blocks[g0:g0 + threads]
        for (r0, r1), (dI_blk, dT_part, ds_part) in zip(group, _pmap(blk_grad, group, threads)):
            dI[r0:r1] = dI_blk
            dT += dT_part
            ds_parts.append(ds_part)
    dscale = dloss * math.fsum(ds_parts) / (2.0 * b)
    return dI, dT, dscale


def forward_backward(I, T, s, dloss: float = 1.0, threads: int | None = None):
    fwd = forward(I, T, s, threads=threads)
    dI, dT, dscale = backward(I, T, s, fwd, dloss=dloss, threads=threads)
    return fwd, dI, dT, dscale


def sampled_rows(I, T, s, rows) -> dict:
    """Exact row statistics (r_i, ell_r_i, x_ii) for a subset of rows only.

    Costs |rows| * b * d; used where the full oracle would take hours.
    """
    I = _as64(I)
    T = _as64(T)
    s = float(s)
    rows = np.asarray(rows, dtype=np.int64)
    x = s * (I[rows] @ T.T)
    x_diag = x[np.arange(len(rows)), rows].copy()
    x[np.arange(len(rows)), rows] = -np.inf
    m = np.max(x, axis=1)
    safe = np.where(np.isfinite(m), m, 0.0)
    with np.errstate(divide="ignore"):
        lse_off = safe + np.log(np.sum(np.exp(x - safe[:, None]), axis=1))
    ell = softplus(lse_off - x_diag)
    return {"lse": x_diag + ell, "ell": ell, "x_diag": x_diag}


def sampled_cols(I, T, s, cols) -> dict:
    """Exact column statistics (c_j, ell_c_j, x_jj) for a subset of columns."""
    return sampled_rows(T, I, s, cols)   # S^T = s * T I^T: columns are rows of the swap
