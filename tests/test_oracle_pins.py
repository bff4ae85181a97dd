"""Pins of the float64 oracle against facts other than itself.

Each test ties the oracle to a hand-worked example, a closed form computed
with a different algorithm (LAPACK Householder QR, SVD), or an identity of the
mathematics.  Together they make a plausible mistake anywhere in the oracle
(a dropped error term, a wrong sign, a transposed operand, a missing
orthogonalisation, a wrong warm start) fail at least one test; the mutant
tests in test_oracle_mutants.py check exactly that.
"""

import json
import math
import os

import numpy as np
import pytest

import oracle
from workloads import bf16_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _val(s):
    if isinstance(s, (int, float)):
        return float(s)
    s = s.replace("sqrt", "math.sqrt(").strip()
    # close the sqrt( opened above: sqrt5 -> math.sqrt(5)
    out, i = "", 0
    while i < len(s):
        if s.startswith("math.sqrt(", i):
            j = i + len("math.sqrt(")
            k = j
            while k < len(s) and s[k].isdigit():
                k += 1
            out += "math.sqrt(" + s[j:k] + ")"
            i = k
        else:
            out += s[i]
            i += 1
    return float(eval(out, {"math": math}))


def _arr(rows):
    return np.array([[_val(x) for x in row] for row in rows], dtype=np.float64)


def _case_inputs(c):
    M = np.array(c["M"], dtype=np.float32)
    e = np.array(c["err_prev"], dtype=np.float32)
    Q0 = np.array(c["Q0"], dtype=np.float32)
    return M, e, Q0


# ----------------------------------------------------------------------------
# hand-worked examples (tests/golden/handworked.json)
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("case", json.load(open(os.path.join(GOLDEN, "handworked.json")))["cases"],
                         ids=lambda c: c["name"])
def test_handworked(case):
    M, e, Q0 = _case_inputs(case)
    out = oracle.step(M, "f32", e, Q0, case["rank"], case["iters"])
    for key in ("P", "Q", "M_hat", "err"):
        np.testing.assert_allclose(out[key], _arr(case[key]), rtol=0, atol=1e-14, err_msg=key)


def test_bf16_lift_and_rne_fixture():
    cases = json.load(open(os.path.join(GOLDEN, "bf16_rne.json")))["cases"]
    f32 = np.array([int(c["f32_bits"], 16) for c in cases], dtype=np.uint32).view(np.float32)
    want = np.array([int(c["bf16_bits"], 16) for c in cases], dtype=np.uint16)
    got = bf16_bits(f32)
    np.testing.assert_array_equal(got, want)
    # the oracle's lift of bf16 bits: 0x3F82 = 1 + 2^-6, 0xC000 = -2
    lifted = oracle.lift(np.array([0x3F82, 0xC000, 0x0000, 0x8000], dtype=np.uint16), "bf16")
    assert lifted[0] == 1 + 2.0 ** -6 and lifted[1] == -2.0 and lifted[2] == 0.0
    assert math.copysign(1.0, lifted[3]) == -1.0


# ----------------------------------------------------------------------------
# P1: closed form.  For full-rank iterates M_hat = Pi_range(K) A with
# K = (A A^T)^(t-1) A Q0, computed here with LAPACK Householder QR.
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("t", [1, 2, 3])
@pytest.mark.parametrize("shape,r", [((60, 40), 5), ((37, 90), 7), ((50, 50), 1)])
def test_closed_form_projection(shape, r, t):
    g = np.random.default_rng(100 + t)
    m, n = shape
    M = g.standard_normal((m, n)).astype(np.float32)
    e = (0.3 * g.standard_normal((m, n))).astype(np.float32)
    Q0 = g.standard_normal((n, r)).astype(np.float32)
    out = oracle.step(M, "f32", e, Q0, r, t)
    A = M.astype(np.float64) + e.astype(np.float64)
    K = A @ Q0.astype(np.float64)
    for _ in range(t - 1):
        K = A @ (A.T @ K)
        K, _ = np.linalg.qr(K)          # re-basis only; the span is unchanged
    Qk, _ = np.linalg.qr(K)
    want = Qk @ (Qk.T @ A)
    np.testing.assert_allclose(out["M_hat"], want, rtol=0, atol=1e-11 * np.abs(A).max())
    np.testing.assert_allclose(out["err"], A - want, rtol=0, atol=1e-11 * np.abs(A).max())
    # returned Q is the unnormalised right factor A^T P_hat
    np.testing.assert_allclose(out["Q"], A.T @ out["P"], rtol=0, atol=1e-11 * np.abs(A).max() * m)


# ----------------------------------------------------------------------------
# P2: the invariants of the method
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("k,r", [(3, 5), (5, 5), (1, 4)])
def test_exact_recovery_of_low_rank(k, r):
    g = np.random.default_rng(7 + k)
    m, n = 48, 33
    # exactly rank-k float64 input (err_prev carries it; M is zero)
    A = g.standard_normal((m, k)) @ g.standard_normal((k, n))
    M = np.zeros((m, n), np.float32)
    Q0 = g.standard_normal((n, r)).astype(np.float32)
    out = oracle.step(M, "f32", A, Q0, r, 1)
    assert np.linalg.norm(out["err"]) <= 1e-12 * np.linalg.norm(A)


@pytest.mark.parametrize("t", [1, 2])
def test_orthonormal_P(t):
    g = np.random.default_rng(11)
    M = g.standard_normal((70, 45)).astype(np.float32)
    Q0 = g.standard_normal((45, 9)).astype(np.float32)
    P = oracle.step(M, "f32", np.zeros_like(M), Q0, 9, t)["P"]
    np.testing.assert_allclose(P.T @ P, np.eye(9), rtol=0, atol=1e-10)


def test_conservation_mhat_plus_err_is_input():
    g = np.random.default_rng(12)
    M = g.standard_normal((64, 30)).astype(np.float32)
    e = g.standard_normal((64, 30)).astype(np.float32)
    Q0 = g.standard_normal((30, 6)).astype(np.float32)
    out = oracle.step(M, "f32", e, Q0, 6, 2)
    A = M.astype(np.float64) + e
    assert np.abs(out["M_hat"] + out["err"] - A).max() <= 1e-14 * np.abs(A).max()


@pytest.mark.parametrize("shape", [(40, 12), (12, 40), (25, 25)])
def test_full_rank_reconstructs(shape):
    g = np.random.default_rng(13)
    m, n = shape
    r = min(m, n)
    M = g.standard_normal((m, n)).astype(np.float32)
    Q0 = g.standard_normal((n, r)).astype(np.float32)
    out = oracle.step(M, "f32", np.zeros_like(M), Q0, r, 1)
    np.testing.assert_allclose(out["M_hat"], M.astype(np.float64), rtol=0, atol=1e-12)


def test_svd_agreement_after_many_iterations():
    """Eckart-Young: with a spectral gap the iteration converges to A_r."""
    g = np.random.default_rng(14)
    m, n, r = 8, 6, 3
    U, _ = np.linalg.qr(g.standard_normal((m, n)))
    V, _ = np.linalg.qr(g.standard_normal((n, n)))
    s = np.array([10, 8, 6, 2, 1, 0.5])
    A = (U * s) @ V.T
    Q0 = g.standard_normal((n, r)).astype(np.float32)
    out = oracle.step(np.zeros((m, n), np.float32), "f32", A, Q0, r, 60)
    Uu, ss, Vt = np.linalg.svd(A)
    Ar = (Uu[:, :r] * ss[:r]) @ Vt[:r]
    np.testing.assert_allclose(out["M_hat"], Ar, rtol=0, atol=1e-12)


def test_svd_convergence_rate():
    """The subspace error after t rounds decays like (s_{r+1}/s_r)^(2t)."""
    g = np.random.default_rng(15)
    m, n, r = 30, 20, 2
    U, _ = np.linalg.qr(g.standard_normal((m, n)))
    V, _ = np.linalg.qr(g.standard_normal((n, n)))
    s = np.concatenate([[4.0, 3.0, 1.5], 0.1 * np.ones(n - 3)])
    A = (U * s) @ V.T
    Ar = (U[:, :r] * s[:r]) @ V[:, :r].T
    Q0 = g.standard_normal((n, r)).astype(np.float32)
    errs = []
    for t in (2, 4, 6):
        out = oracle.step(np.zeros((m, n), np.float32), "f32", A, Q0, r, t)
        errs.append(np.linalg.norm(out["M_hat"] - Ar))
    ratio = (1.5 / 3.0) ** 4          # two extra rounds
    assert errs[1] / errs[0] < 4 * ratio and errs[2] / errs[1] < 4 * ratio


# ----------------------------------------------------------------------------
# P3: further identities
# ----------------------------------------------------------------------------
def _rand_step(seed=20, m=55, n=38, r=6, t=1, dtype="f32"):
    g = np.random.default_rng(seed)
    x = g.standard_normal((m, n))
    M = x.astype(np.float32) if dtype == "f32" else bf16_bits(x.astype(np.float32))
    e = (0.5 * g.standard_normal((m, n))).astype(np.float32)
    Q0 = g.standard_normal((n, r)).astype(np.float32)
    return M, e, Q0


def test_residual_orthogonal_to_P():
    M, e, Q0 = _rand_step()
    out = oracle.step(M, "f32", e, Q0, 6, 1)
    assert np.abs(out["P"].T @ out["err"]).max() <= 1e-13 * np.abs(out["A"]).max()


def test_pythagoras():
    M, e, Q0 = _rand_step(t=2)
    out = oracle.step(M, "f32", e, Q0, 6, 2)
    a2 = np.sum(out["A"] ** 2)
    assert abs(np.sum(out["M_hat"] ** 2) + np.sum(out["err"] ** 2) - a2) <= 1e-13 * a2


def test_error_feedback_telescopes():
    """Sec. 5.1 (Eqs. gstar -> restruct): summed over S steps, the values sent
    plus the last residual equal the true inputs plus the first residual."""
    g = np.random.default_rng(21)
    m, n, r, S = 40, 24, 3, 8
    err = (0.1 * g.standard_normal((m, n))).astype(np.float64)
    err0 = err.copy()
    Q = g.standard_normal((n, r))
    sent = np.zeros((m, n))
    true = np.zeros((m, n))
    for s in range(S):
        M = g.standard_normal((m, n)).astype(np.float32)
        out = oracle.step(M, "f32", err, Q, r, 1)
        sent += out["M_hat"]
        true += M
        err, Q = out["err"], out["Q"]
    np.testing.assert_allclose(sent + err, true + err0, rtol=0, atol=1e-12)


def test_warm_start_invariances():
    M, e, Q0 = _rand_step(seed=22, r=5)
    base = oracle.step(M, "f32", e, Q0, 5, 2)
    g = np.random.default_rng(23)
    Rt = np.triu(g.standard_normal((5, 5)))
    Rt[np.diag_indices(5)] = np.abs(Rt[np.diag_indices(5)]) + 0.5
    tri = oracle.step(M, "f32", e, Q0.astype(np.float64) @ Rt, 5, 2)
    np.testing.assert_allclose(tri["P"], base["P"], rtol=0, atol=1e-10)
    X = g.standard_normal((5, 5)) + 3 * np.eye(5)
    gen = oracle.step(M, "f32", e, Q0.astype(np.float64) @ X, 5, 2)
    np.testing.assert_allclose(gen["M_hat"], base["M_hat"], rtol=0, atol=1e-10)


def test_scale_equivariance():
    M, e, Q0 = _rand_step(seed=24)
    base = oracle.step(M, "f32", e, Q0, 6, 1)
    sc = oracle.step((4 * M).astype(np.float32), "f32", 4 * e.astype(np.float64), Q0, 6, 1)
    np.testing.assert_allclose(sc["M_hat"], 4 * base["M_hat"], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(sc["P"], base["P"], rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------
# P4: the orthogonalisation choice.  CholeskyQR (the GPU's method) and MGS2
# (the oracle's) give the same Q-factor for full-rank P.
# ----------------------------------------------------------------------------
def test_cholesky_qr_equals_mgs2():
    g = np.random.default_rng(30)
    P = g.standard_normal((200, 16)) @ np.diag(np.logspace(0, -3, 16))
    L = np.linalg.cholesky(P.T @ P)
    Pc = np.linalg.solve(L, P.T).T          # P L^-T
    np.testing.assert_allclose(oracle.mgs2(P), Pc, rtol=0, atol=1e-9)
    Qh, Rh = np.linalg.qr(P)
    Qh = Qh * np.sign(np.diag(Rh))
    np.testing.assert_allclose(oracle.mgs2(P), Qh, rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------
# degenerate cases the method has
# ----------------------------------------------------------------------------
def test_zero_input_gives_zero_factors():
    M = np.zeros((20, 10), np.float32)
    Q0 = np.random.default_rng(1).standard_normal((10, 3)).astype(np.float32)
    out = oracle.step(M, "f32", np.zeros_like(M), Q0, 3, 2)
    for key in ("P", "Q", "M_hat", "err"):
        assert not out[key].any(), key


def test_rank_deficient_zeroes_dependent_columns():
    g = np.random.default_rng(31)
    m, n, r = 30, 20, 4
    A = np.outer(g.standard_normal(m), g.standard_normal(n))    # rank 1
    Q0 = g.standard_normal((n, r)).astype(np.float32)
    out = oracle.step(np.zeros((m, n), np.float32), "f32", A, Q0, r, 1)
    P = out["P"]
    assert np.count_nonzero(np.linalg.norm(P, axis=0)) == 1
    np.testing.assert_allclose(out["M_hat"], A, rtol=0, atol=1e-12)


def test_bf16_input_path():
    """bf16 inputs are lifted exactly: same result as the equivalent fp32 input."""
    M, e, Q0 = _rand_step(seed=40, dtype="bf16")
    widened = (M.astype(np.uint32) << 16).view(np.float32)
    a = oracle.step(M, "bf16", e, Q0, 6, 1)
    b = oracle.step(widened, "f32", e, Q0, 6, 1)
    for key in ("P", "Q", "M_hat", "err"):
        np.testing.assert_array_equal(a[key], b[key])


def test_batched_is_independent_steps():
    items = [_rand_step(seed=50 + j, m=20 + j, n=15) for j in range(3)]
    outs = oracle.step_batched([(M, "f32", e, Q) for (M, e, Q) in items], 6, 2)
    for (M, e, Q), o in zip(items, outs):
        ref = oracle.step(M, "f32", e, Q, 6, 2)
        np.testing.assert_array_equal(o["M_hat"], ref["M_hat"])


def test_argument_errors():
    M = np.zeros((5, 4), np.float32)
    with pytest.raises(ValueError):
        oracle.step(M, "f32", M, np.zeros((4, 5), np.float32), 5, 1)
    with pytest.raises(ValueError):
        oracle.step(M, "f32", M, np.zeros((4, 2), np.float32), 2, 0)
    with pytest.raises(TypeError):
        oracle.step(M, "bf16", M, np.zeros((4, 2), np.float32), 2, 1)
