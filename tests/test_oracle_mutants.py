"""Planted mistakes in (copies of) the oracle must fail at least one pin.

Each mutant is the oracle's step with one plausible mistake.  The pins are
the same facts test_oracle_pins.py checks (hand-worked fixture, LAPACK closed
form, telescoping identity, residual orthogonality).  The real oracle passes
all of them; every mutant must fail at least one.  Mistakes are planted on
the CPU only, in local functions; the oracle module itself is not modified.
"""

import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle.powerlr import lift, mgs2

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _make_step(*, err_sign=1.0, use_err=True, transpose_q=False, orth=True,
               resid_from_m=False, warm=True, iters_delta=0, norm_q=False,
               mhat_transposed=False):
    def step(M, dt, err_prev, Q, rank, iters):
        Mf = lift(M, dt)
        A = Mf + err_sign * np.asarray(err_prev, np.float64) if use_err else Mf.copy()
        Qc = np.asarray(Q, np.float64)
        if not warm:
            Qc = np.ones_like(Qc)
        P_hat = None
        for _ in range(max(1, iters + iters_delta)):
            P = A @ Qc
            P_hat = mgs2(P) if orth else P / np.maximum(np.linalg.norm(P, axis=0), 1e-300)
            Qc = (A @ P_hat) if transpose_q else (A.T @ P_hat)
            if norm_q:
                Qc = Qc / np.linalg.norm(Qc, axis=0)
        M_hat = (Qc @ P_hat.T).T if mhat_transposed else P_hat @ Qc.T
        if mhat_transposed:
            M_hat = M_hat.T if M_hat.shape != A.shape else M_hat.T
        err = (Mf - M_hat) if resid_from_m else (A - M_hat)
        return {"P": P_hat, "Q": Qc, "M_hat": M_hat, "err": err, "A": A}
    return step


MUTANTS = {
    "dropped_err_term": _make_step(use_err=False),
    "wrong_err_sign": _make_step(err_sign=-1.0),
    "transposed_right_product": _make_step(transpose_q=True),
    "no_orthogonalisation": _make_step(orth=False),
    "residual_ignores_err_prev": _make_step(resid_from_m=True),
    "cold_start": _make_step(warm=False),
    "one_round_too_many": _make_step(iters_delta=1),
    "normalised_Q": _make_step(norm_q=True),
    "transposed_decompression": _make_step(mhat_transposed=True),
}


def _val(s):
    if isinstance(s, (int, float)):
        return float(s)
    expr = s
    for d in "2356789":
        expr = expr.replace(f"sqrt{d}", f"math.sqrt({d})")
    return float(eval(expr, {"math": math}))


def pin_handworked(step):
    for c in json.load(open(os.path.join(GOLDEN, "handworked.json")))["cases"]:
        M = np.array(c["M"], np.float32)
        e = np.array(c["err_prev"], np.float32)
        Q0 = np.array(c["Q0"], np.float32)
        try:
            out = step(M, "f32", e, Q0, c["rank"], c["iters"])
        except ValueError:
            return False
        for key in ("Q", "M_hat", "err"):
            want = np.array([[_val(x) for x in row] for row in c[key]])
            if out[key].shape != want.shape or not np.allclose(out[key], want, atol=1e-12, rtol=0):
                return False
    return True


def pin_closed_form(step):
    g = np.random.default_rng(5)
    for (m, n, r, t) in ((24, 24, 3, 1), (24, 24, 3, 2), (30, 18, 4, 1)):
        M = g.standard_normal((m, n)).astype(np.float32)
        e = (0.5 * g.standard_normal((m, n))).astype(np.float32)
        Q0 = g.standard_normal((n, r)).astype(np.float32)
        try:
            out = step(M, "f32", e, Q0, r, t)
        except ValueError:
            return False
        A = M.astype(np.float64) + e
        K = A @ Q0.astype(np.float64)
        for _ in range(t - 1):
            K = A @ (A.T @ K)
        Qk, _ = np.linalg.qr(K)
        want = Qk @ (Qk.T @ A)
        if out["M_hat"].shape != want.shape or not np.allclose(out["M_hat"], want, atol=1e-10, rtol=0):
            return False
        if not np.allclose(out["err"], A - want, atol=1e-10, rtol=0):
            return False
    return True


def pin_telescoping(step):
    g = np.random.default_rng(6)
    m, n, r = 16, 16, 2
    err = 0.1 * g.standard_normal((m, n))
    err0 = err.copy()
    Q = g.standard_normal((n, r))
    sent = np.zeros((m, n))
    true = np.zeros((m, n))
    for _ in range(5):
        M = g.standard_normal((m, n)).astype(np.float32)
        try:
            out = step(M, "f32", err, Q, r, 1)
        except ValueError:
            return False
        sent += out["M_hat"]
        true += M
        err, Q = out["err"], out["Q"]
    return np.allclose(sent + err, true + err0, atol=1e-11, rtol=0)


def pin_orthogonal_residual(step):
    g = np.random.default_rng(8)
    M = g.standard_normal((20, 20)).astype(np.float32)
    Q0 = g.standard_normal((20, 4)).astype(np.float32)
    out = step(M, "f32", np.zeros_like(M), Q0, 4, 1)
    P = out["P"]
    return (np.allclose(P.T @ P, np.eye(4), atol=1e-10)
            and np.abs(P.T @ out["err"]).max() < 1e-10)


PINS = [pin_handworked, pin_closed_form, pin_telescoping, pin_orthogonal_residual]


def test_real_oracle_passes_every_pin():
    for pin in PINS:
        assert pin(oracle.step), pin.__name__


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_fails_a_pin(name):
    mutant = MUTANTS[name]
    results = {}
    for pin in PINS:
        try:
            results[pin.__name__] = pin(mutant)
        except Exception:
            results[pin.__name__] = False
    assert not all(results.values()), f"mutant {name} passed every pin: {results}"
