"""Pins of the fp64 oracle against facts that do not come from the oracle itself.

Every pin here is independent of the oracle's own code path:
  * closed forms A-D derived by hand from the loss definition (Sec. 2.2, Eq. 1
    and its symmetric text->image half);
  * a library routine: torch float64 cross-entropy on a materialised similarity
    matrix, with torch autograd for the gradients;
  * brute force: the definition in pure-Python loops (math.exp / math.log) on
    tiny inputs;
  * central finite differences of the loss for the gradients (Eq. 6-8);
  * invariants that hold at any size.
The last block plants mistakes into the oracle and checks a pin catches each.
"""

import math

import numpy as np
import pytest
import torch

import oracle
from oracle import infonce
from paper_2410_17243_amd import synth


def _rand(b, d, seed=0, unit=True):
    rng = np.random.default_rng(seed)
    I = rng.standard_normal((b, d))
    T = I + 0.7 * rng.standard_normal((b, d))
    if unit:
        I /= np.linalg.norm(I, axis=1, keepdims=True)
        T /= np.linalg.norm(T, axis=1, keepdims=True)
    return I, T


# ---------------------------------------------------------------- closed forms

@pytest.mark.parametrize("b,s", [(2, 1.0), (7, 14.29), (64, 100.0), (300, 50.0)])
def test_closed_form_A_identical(b, s):
    """All embeddings equal to one unit vector: L = log b, r = c = s + log b, zero gradients."""
    d = 5
    e = np.zeros(d)
    e[2] = 1.0
    I = np.tile(e, (b, 1))
    T = I.copy()
    fwd, dI, dT, ds = oracle.forward_backward(I, T, s, dloss=1.0)
    assert fwd["loss"] == pytest.approx(math.log(b), rel=1e-13)
    np.testing.assert_allclose(fwd["lse_r"], s + math.log(b), rtol=1e-13)
    np.testing.assert_allclose(fwd["lse_c"], s + math.log(b), rtol=1e-13)
    assert np.max(np.abs(dI)) < 1e-13 * s
    assert np.max(np.abs(dT)) < 1e-13 * s
    assert abs(ds) < 1e-13


def _closed_B(b, s, dloss):
    Z = math.exp(s) + b - 1
    p = math.exp(s) / Z
    q = 1.0 / Z
    loss = math.log1p((b - 1) * math.exp(-s))
    lse = math.log(Z)
    ds = -dloss * (b - 1) / Z
    g = np.full((b, b), q)
    np.fill_diagonal(g, -(b - 1) / Z)   # p - 1, written without cancellation
    dI = (s * dloss / b) * g  # row i: (p-1) e_i + q sum_{j != i} e_j, embedded in d >= b
    return loss, lse, ds, dI


@pytest.mark.parametrize("b,s", [(16, 100.0), (16, 14.29), (5, 1.0), (40, 60.0)])
def test_closed_form_B_one_hot_pairs(b, s):
    """I_i = T_i = e_i (d >= b): L = log1p((b-1) e^-s), exact even where L ~ 1e-43."""
    d = b + 3
    I = np.zeros((b, d))
    I[np.arange(b), np.arange(b)] = 1.0
    T = I.copy()
    dloss = 0.75
    fwd, dI, dT, ds = oracle.forward_backward(I, T, s, dloss=dloss)
    loss, lse, ds_ref, dI_ref = _closed_B(b, s, dloss)
    assert fwd["loss"] == pytest.approx(loss, rel=1e-12)
    np.testing.assert_allclose(fwd["lse_r"], lse, rtol=1e-14)
    np.testing.assert_allclose(fwd["lse_c"], lse, rtol=1e-14)
    assert ds == pytest.approx(ds_ref, rel=1e-12)
    np.testing.assert_allclose(dI[:, :b], dI_ref, rtol=1e-12, atol=0)
    np.testing.assert_allclose(dT[:, :b], dI_ref, rtol=1e-12, atol=0)
    assert np.all(dI[:, b:] == 0) and np.all(dT[:, b:] == 0)


def _closed_C(b, d, s, dloss):
    """Periodic one-hot I_i = T_i = e_{i mod d}: per-class closed forms, O(b d)."""
    cls = np.arange(b) % d
    n = np.bincount(cls, minlength=d).astype(np.float64)   # class sizes
    es = math.exp(s)
    Zc = n * es + (b - n)                                   # Z per class
    r = np.log(Zc)[cls]
    loss = math.fsum(r - s) / b
    dI = np.zeros((b, d))
    for i in range(b):
        ci = cls[i]
        coef = n * (1.0 / Zc[ci] + 1.0 / Zc) / (2 * b)      # other classes
        coef[ci] = n[ci] * es / (b * Zc[ci]) - 1.0 / b       # own class
        coef[n == 0] = 0.0
        dI[i] = dloss * s * coef
    ds = -(dloss / b) * math.fsum(((b - n[cls]) / Zc[cls]))
    return loss, r, dI, ds


@pytest.mark.parametrize("b,d,s", [(50, 8, 14.29), (37, 5, 100.0), (64, 64, 3.0), (129, 16, 50.0)])
def test_closed_form_C_periodic(b, d, s):
    I = np.zeros((b, d))
    I[np.arange(b), np.arange(b) % d] = 1.0
    T = I.copy()
    dloss = 1.3
    fwd, dI, dT, ds = oracle.forward_backward(I, T, s, dloss=dloss)
    loss, r, dI_ref, ds_ref = _closed_C(b, d, s, dloss)
    assert fwd["loss"] == pytest.approx(loss, rel=1e-12)
    np.testing.assert_allclose(fwd["lse_r"], r, rtol=1e-13)
    np.testing.assert_allclose(fwd["lse_c"], r, rtol=1e-13)
    np.testing.assert_allclose(dI, dI_ref, rtol=1e-10, atol=1e-13 * abs(dloss * s))
    np.testing.assert_allclose(dT, dI_ref, rtol=1e-10, atol=1e-13 * abs(dloss * s))
    assert ds == pytest.approx(ds_ref, rel=1e-10)


def test_closed_form_D_single_pair():
    I, T = _rand(1, 9, seed=3)
    fwd, dI, dT, ds = oracle.forward_backward(I, T, 37.0, dloss=2.0)
    assert fwd["loss"] == 0.0
    assert np.all(dI == 0) and np.all(dT == 0) and ds == 0.0
    np.testing.assert_allclose(fwd["lse_r"], fwd["x_diag"])


# ------------------------------------------------------- library routine (torch)

def _torch_ref(I, T, s, dloss):
    It = torch.tensor(I, dtype=torch.float64, requires_grad=True)
    Tt = torch.tensor(T, dtype=torch.float64, requires_grad=True)
    st = torch.tensor(s, dtype=torch.float64, requires_grad=True)
    S = st * (It @ Tt.T)
    lab = torch.arange(I.shape[0])
    loss = 0.5 * (torch.nn.functional.cross_entropy(S, lab) + torch.nn.functional.cross_entropy(S.T, lab))
    (loss * dloss).backward()
    return (loss.item(), torch.logsumexp(S, 1).detach().numpy(), torch.logsumexp(S, 0).detach().numpy(),
            It.grad.numpy(), Tt.grad.numpy(), st.grad.item())


@pytest.mark.parametrize("b,d,s,seed", [(3, 4, 1.0, 0), (17, 8, 14.29, 1), (256, 64, 14.29, 2),
                                         (200, 32, 50.0, 3), (1025, 16, 5.0, 4)])
def test_against_torch_cross_entropy(b, d, s, seed):
    I, T = _rand(b, d, seed=seed)
    dloss = 0.8
    fwd, dI, dT, ds = oracle.forward_backward(I, T, s, dloss=dloss, threads=2)
    loss, lr, lc, gI, gT, gs = _torch_ref(I, T, s, dloss)
    assert fwd["loss"] == pytest.approx(loss, rel=1e-11)
    np.testing.assert_allclose(fwd["lse_r"], lr, rtol=1e-12)
    np.testing.assert_allclose(fwd["lse_c"], lc, rtol=1e-12)
    sc = max(np.max(np.abs(gI)), np.max(np.abs(gT)))
    np.testing.assert_allclose(dI, gI, rtol=0, atol=1e-10 * sc)
    np.testing.assert_allclose(dT, gT, rtol=0, atol=1e-10 * sc)
    assert ds == pytest.approx(gs, rel=1e-9, abs=1e-13)


def test_against_torch_non_normalised_inputs():
    """The loss uses its inputs as given (no normalisation inside)."""
    rng = np.random.default_rng(11)
    I = 3.0 * rng.standard_normal((40, 6))
    T = 0.5 * rng.standard_normal((40, 6))
    fwd, dI, dT, ds = oracle.forward_backward(I, T, 2.0)
    loss, lr, lc, gI, gT, gs = _torch_ref(I, T, 2.0, 1.0)
    assert fwd["loss"] == pytest.approx(loss, rel=1e-12)
    np.testing.assert_allclose(dI, gI, rtol=1e-9, atol=1e-14)
    np.testing.assert_allclose(dT, gT, rtol=1e-9, atol=1e-14)
    assert ds == pytest.approx(gs, rel=1e-9)


# --------------------------------------------------------------- brute force

def _brute_loss(I, T, s):
    b = len(I)
    x = [[s * sum(I[i][k] * T[j][k] for k in range(len(I[0]))) for j in range(b)] for i in range(b)]
    li = [-math.log(math.exp(x[i][i]) / sum(math.exp(x[i][j]) for j in range(b))) for i in range(b)]
    lt = [-math.log(math.exp(x[j][j]) / sum(math.exp(x[i][j]) for i in range(b))) for j in range(b)]
    return 0.5 * (sum(li) / b + sum(lt) / b), x


@pytest.mark.parametrize("b,d,s", [(1, 3, 2.0), (2, 2, 1.0), (3, 4, 7.0), (5, 3, 14.29)])
def test_brute_force_tiny(b, d, s):
    I, T = _rand(b, d, seed=b + d)
    loss, x = _brute_loss(I.tolist(), T.tolist(), s)
    fwd = oracle.forward(I, T, s)
    assert fwd["loss"] == pytest.approx(loss, rel=1e-12, abs=1e-15)
    for i in range(b):
        assert fwd["lse_r"][i] == pytest.approx(math.log(sum(math.exp(v) for v in x[i])), rel=1e-13)
        assert fwd["lse_c"][i] == pytest.approx(math.log(sum(math.exp(x[k][i]) for k in range(b))), rel=1e-13)
        assert fwd["x_diag"][i] == pytest.approx(x[i][i], rel=1e-13, abs=1e-15)


# --------------------------------------------------------- finite differences

@pytest.mark.parametrize("b,d,s", [(2, 3, 1.0), (5, 4, 14.29), (16, 6, 3.0), (9, 9, 30.0)])
def test_finite_differences(b, d, s):
    I, T = _rand(b, d, seed=7 * b + d, unit=False)
    dloss = 1.7
    _, dI, dT, ds = oracle.forward_backward(I, T, s, dloss=dloss)
    h = 1e-6

    def L(I_, T_, s_):
        return dloss * oracle.forward(I_, T_, s_)["loss"]

    fdI = np.zeros_like(I)
    fdT = np.zeros_like(T)
    for i in range(b):
        for k in range(d):
            Ip, Im = I.copy(), I.copy()
            Ip[i, k] += h
            Im[i, k] -= h
            fdI[i, k] = (L(Ip, T, s) - L(Im, T, s)) / (2 * h)
            Tp, Tm = T.copy(), T.copy()
            Tp[i, k] += h
            Tm[i, k] -= h
            fdT[i, k] = (L(I, Tp, s) - L(I, Tm, s)) / (2 * h)
    hs = 1e-6 * max(1.0, s)
    fds = (L(I, T, s + hs) - L(I, T, s - hs)) / (2 * hs)
    sc = max(np.max(np.abs(fdI)), np.max(np.abs(fdT)), 1e-3)
    np.testing.assert_allclose(dI, fdI, rtol=0, atol=2e-7 * sc)
    np.testing.assert_allclose(dT, fdT, rtol=0, atol=2e-7 * sc)
    assert ds == pytest.approx(fds, rel=1e-6, abs=1e-8)


# ---------------------------------------------------------------- invariants

def test_invariants():
    b, d, s = 120, 24, 20.0
    I, T = _rand(b, d, seed=5)
    fwd, dI, dT, ds = oracle.forward_backward(I, T, s, dloss=1.0)
    # <dI, I>_F = <dT, T>_F = s * dscale
    assert np.sum(dI * I) == pytest.approx(s * ds, rel=1e-10)
    assert np.sum(dT * T) == pytest.approx(s * ds, rel=1e-10)
    # per-sample terms are non-negative
    assert np.all(fwd["ell_r"] >= 0) and np.all(fwd["ell_c"] >= 0)
    # pair permutation
    perm = np.random.default_rng(0).permutation(b)
    f2, dI2, dT2, ds2 = oracle.forward_backward(I[perm], T[perm], s)
    assert f2["loss"] == pytest.approx(fwd["loss"], rel=1e-12)
    np.testing.assert_allclose(f2["lse_r"], fwd["lse_r"][perm], rtol=1e-13)
    np.testing.assert_allclose(dI2, dI[perm], rtol=1e-10, atol=1e-15)
    np.testing.assert_allclose(dT2, dT[perm], rtol=1e-10, atol=1e-15)
    assert ds2 == pytest.approx(ds, rel=1e-10)
    # image <-> text swap
    f3, dI3, dT3, ds3 = oracle.forward_backward(T, I, s)
    assert f3["loss"] == pytest.approx(fwd["loss"], rel=1e-12)
    np.testing.assert_allclose(f3["lse_r"], fwd["lse_c"], rtol=1e-13)
    np.testing.assert_allclose(dI3, dT, rtol=1e-10, atol=1e-15)
    assert ds3 == pytest.approx(ds, rel=1e-10)
    # linearity in dloss
    _, dI4, dT4, ds4 = oracle.forward_backward(I, T, s, dloss=-2.5)
    np.testing.assert_allclose(dI4, -2.5 * dI, rtol=1e-12)
    assert ds4 == pytest.approx(-2.5 * ds, rel=1e-12)
    # scale homogeneity: L(aI, T, s) = L(I, T, a s)
    assert oracle.forward(3.0 * I, T, s)["loss"] == pytest.approx(oracle.forward(I, T, 3.0 * s)["loss"], rel=1e-12)


def test_block_size_independence(monkeypatch):
    """The row-block size of the materialisation is not part of the arithmetic."""
    I, T = _rand(300, 16, seed=9)
    ref = oracle.forward_backward(I, T, 14.29, threads=1)
    monkeypatch.setattr(infonce, "_BLOCK_BYTES", 8 * 300 * 7)   # 7-row blocks
    got = oracle.forward_backward(I, T, 14.29, threads=3)
    assert got[0]["loss"] == pytest.approx(ref[0]["loss"], rel=1e-13)
    np.testing.assert_allclose(got[0]["lse_c"], ref[0]["lse_c"], rtol=1e-14)
    np.testing.assert_allclose(got[1], ref[1], rtol=1e-12, atol=1e-16)
    np.testing.assert_allclose(got[2], ref[2], rtol=1e-12, atol=1e-16)


def test_sampled_rows_and_cols_match_full():
    I, T = _rand(500, 12, seed=13)
    full = oracle.forward(I, T, 30.0)
    rows = np.array([0, 7, 123, 499])
    sr = oracle.sampled_rows(I, T, 30.0, rows)
    sc = oracle.sampled_cols(I, T, 30.0, rows)
    np.testing.assert_allclose(sr["lse"], full["lse_r"][rows], rtol=1e-14)
    np.testing.assert_allclose(sr["ell"], full["ell_r"][rows], rtol=1e-12)
    np.testing.assert_allclose(sc["lse"], full["lse_c"][rows], rtol=1e-14)
    np.testing.assert_allclose(sc["ell"], full["ell_c"][rows], rtol=1e-12)


def test_generator_inputs_workload_sanity():
    """Config-2-shaped generator output at reduced b: loss is finite and below log b."""
    img, txt = synth.clip_pairs(2048, 64, 1.0, seed=0, dtype="bf16")
    I = synth.as_f64(img, "bf16")
    T = synth.as_f64(txt, "bf16")
    f = oracle.forward(I, T, 14.29)
    assert 0.0 < f["loss"] < math.log(2048)


# ------------------------------------------------------------ planted mistakes

# Each (old, new) pair plants one plausible slip into a copy of the oracle's
# source; at least one of the independent pins below must then fail.
MUTANTS = [
    ("np.maximum(z, 0.0) + np.log1p(np.exp(-np.abs(z)))", "np.maximum(z, 0.0)"),          # dropped log1p term
    ("x[idx - r0, idx] = -np.inf              # off-diagonal view", "pass"),              # diagonal kept in LSE_off
    ("dT_part = k * (g.T @ I[r0:r1])", "dT_part = k * (g @ I[r0:r1])"),                  # transposed operand
    ("np.expm1(-ell_r[r0:r1])", "np.expm1(ell_r[r0:r1])"),                               # sign slip on the diagonal
    ("k = dloss * s / (2.0 * b)", "k = dloss * s / b"),                                  # wrong weighting (grad)
    ("pc = np.exp(x - lse_c[None, :])", "pc = np.exp(x - lse_c[r0:r1, None])"),          # row/col index swap
    ("du_c = u - u_diag[None, :]", "du_c = u - u_diag[r0:r1, None]"),                    # wrong diagonal in dscale
    ("/ (2.0 * b) if b else 0.0", "/ b if b else 0.0"),                                  # sum, not mean, of the halves
    ("lse_off_c = col_safe + np.log(col_sum)", "lse_off_c = np.log(col_sum)"),           # dropped shift
    ("pr = np.exp(x - lse_r[r0:r1, None])", "pr = np.exp(x - lse_r[r0:r1, None] - 1e-9)"),  # tiny bias
]


def _mutated_module(old, new):
    import inspect
    import types
    src = inspect.getsource(infonce)
    assert src.count(old) == 1, old
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src.replace(old, new), "oracle_mutant", "exec"), mod.__dict__)
    return mod


def _pins_pass(mod):
    """Fast independent pins: closed forms A and B, torch reference, <dI, I> invariant."""
    ok = True
    e = np.zeros((10, 3))
    e[:, 0] = 1.0
    fA = mod.forward_backward(e, e, 5.0)
    ok &= abs(fA[0]["loss"] - math.log(10)) <= 1e-12 * math.log(10)
    b = 16
    I = np.zeros((b, b + 1))
    I[np.arange(b), np.arange(b)] = 1.0
    fB = mod.forward_backward(I, I, 100.0)
    lB, _, dsB, _ = _closed_B(b, 100.0, 1.0)
    ok &= abs(fB[0]["loss"] - lB) <= 1e-10 * lB and abs(fB[3] - dsB) <= 1e-10 * abs(dsB)
    I3, T3 = _rand(12, 5, seed=21)
    f3 = mod.forward_backward(I3, T3, 4.0)
    loss, lr, lc, gI, gT, gs = _torch_ref(I3, T3, 4.0, 1.0)
    ok &= abs(f3[0]["loss"] - loss) <= 1e-11 * loss
    ok &= bool(np.allclose(f3[1], gI, rtol=1e-9, atol=1e-13)) and bool(np.allclose(f3[2], gT, rtol=1e-9, atol=1e-13))
    ok &= abs(f3[3] - gs) <= 1e-9 * abs(gs) + 1e-13
    return bool(ok)


def test_unmutated_oracle_passes_mutation_pins():
    assert _pins_pass(infonce)


@pytest.mark.parametrize("old,new", MUTANTS, ids=[f"m{i}" for i in range(len(MUTANTS))])
def test_planted_mistake_is_caught(old, new):
    assert not _pins_pass(_mutated_module(old, new))
