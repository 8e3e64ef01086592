"""Full-size parity against the fp64 oracle, independent of the GPU path.

* b = 32768, d = 512, bf16, s = 14.29 (the benchmark's shapes): the full oracle
  runs in the test (about half a minute on 16 host cores) and every output is
  compared element by element: loss and loss64, all r_i and c_j, all per-sample
  terms, dimg and dtxt, dscale.
* b = 131072, d = 768, bf16, s = 100: the full oracle takes minutes, so its
  results are stored in tests/golden/c3_oracle.npz by
  tests/golden/make_c3_reference.py (which calls only the oracle and the input
  generator).  Compared: loss, dscale, all r_i, c_j and per-sample terms; for 96
  seeded rows and columns (first and last included) the gradient rows, computed
  in fp64 from the inputs and the oracle's own log-sum-exp vectors (no GPU value
  enters a reference).

Bars: loss relative 1e-3; gradients max|diff|/max|ref| <= 2e-2; dscale relative
2e-2; r, c within the fp32-accumulation bound of gpu_util.lse_tol; per-sample
terms relative 2e-2 (they are what the loss sums).
"""

import hashlib
import math
import os

import numpy as np
import pytest

import oracle
from gpu_util import f32_scale, lse_tol, max_rel, run, synth

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "c3_oracle.npz")


def _check_forward(g, ref, s, d, rows=None):
    """loss, every r_i / c_j and per-sample term against the reference."""
    print(f"loss gpu {g['loss64']:.9e} ref {float(ref['loss']):.9e}; "
          f"lse_r err {np.max(np.abs(g['lse_r'] - ref['lse_r'])):.2e} lse_c err "
          f"{np.max(np.abs(g['lse_c'] - ref['lse_c'])):.2e}", flush=True)
    assert g["loss64"] == pytest.approx(float(ref["loss"]), rel=1e-3, abs=1e-300)
    assert np.all(np.abs(g["lse_r"] - ref["lse_r"]) <= lse_tol(s, d, ref["lse_r"]))
    assert np.all(np.abs(g["lse_c"] - ref["lse_c"]) <= lse_tol(s, d, ref["lse_c"]))
    for k in ("ell_r", "ell_c"):
        r = np.asarray(ref[k])
        rel = np.abs(g[k] - r) / np.maximum(np.abs(r), 1e-300)
        print(f"  {k} max rel err {np.max(rel):.2e}", flush=True)
        assert np.max(rel) <= 2e-2, k


def test_full_oracle_b32768_d512():
    c = synth.WORKLOADS[2]
    b, d, s = c["b"], c["d"], f32_scale(c["scale"])
    img, txt = synth.clip_pairs(b, d, c["sigma"], seed=0, dtype="bf16")
    g = run(img, txt, "bf16", s)
    fwd, dI, dT, ds = oracle.forward_backward(synth.as_f64(img, "bf16"), synth.as_f64(txt, "bf16"), s)
    _check_forward(g, fwd, s, d)
    assert g["loss"] == pytest.approx(fwd["loss"], rel=1e-3)
    e1, e2 = max_rel(g["dI"], dI), max_rel(g["dT"], dT)
    print(f"  dI {e1:.2e} dT {e2:.2e} dscale gpu {g['dscale']:.9e} ref {ds:.9e}", flush=True)
    assert e1 <= 2e-2 and e2 <= 2e-2
    assert g["dscale"] == pytest.approx(ds, rel=2e-2)


def _grad_rows(A, B, s, rows, lse_own, lse_other, ell_own, ell_other, b):
    """fp64 rows of dOwn = k G' Other for own rows `rows`, from the oracle's
    log-sum-exp vectors (own = A, other = B)."""
    k = s / (2.0 * b)
    x = s * (A[rows] @ B.T)
    g = np.exp(x - lse_own[rows][:, None]) + np.exp(x - lse_other[None, :])
    g[np.arange(len(rows)), rows] = np.expm1(-ell_own[rows]) + np.expm1(-ell_other[rows])
    return k * (g @ B)


@pytest.mark.skipif(not os.path.exists(GOLDEN), reason="stored oracle results absent: run tests/golden/make_c3_reference.py")
def test_stored_oracle_b131072_d768_s100():
    ref = np.load(GOLDEN, allow_pickle=False)
    c = synth.WORKLOADS[3]
    b, d, s = c["b"], c["d"], f32_scale(c["scale"])
    assert int(ref["b"]) == b and int(ref["d"]) == d and float(ref["scale"]) == s
    img, txt = synth.clip_pairs(b, d, c["sigma"], seed=0, dtype="bf16")
    h = hashlib.sha256()
    h.update(img.tobytes())
    h.update(txt.tobytes())
    assert h.hexdigest() == str(ref["input_sha256"]), "generator output differs from the stored reference's"
    g = run(img, txt, "bf16", s)
    _check_forward(g, ref, s, d)
    assert g["dscale"] == pytest.approx(float(ref["dscale"]), rel=2e-2)
    # the loss is the mean of the per-sample terms the GPU exported
    assert g["loss64"] == pytest.approx((math.fsum(g["ell_r"]) + math.fsum(g["ell_c"])) / (2 * b), rel=1e-6)
    I = synth.as_f64(img, "bf16")
    T = synth.as_f64(txt, "bf16")
    rows = np.sort(np.random.default_rng(1234).choice(b, size=96, replace=False))
    rows[0], rows[-1] = 0, b - 1
    dI_ref = _grad_rows(I, T, s, rows, ref["lse_r"], ref["lse_c"], ref["ell_r"], ref["ell_c"], b)
    dT_ref = _grad_rows(T, I, s, rows, ref["lse_c"], ref["lse_r"], ref["ell_c"], ref["ell_r"], b)
    e1, e2 = max_rel(g["dI"][rows], dI_ref), max_rel(g["dT"][rows], dT_ref)
    print(f"  dI rows {e1:.2e} dT rows {e2:.2e}; dscale gpu {g['dscale']:.9e} ref {float(ref['dscale']):.9e}",
          flush=True)
    assert e1 <= 2e-2 and e2 <= 2e-2
