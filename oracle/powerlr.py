"""Float64 CPU oracle for the low-rank power-iteration compressor with error feedback.

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously-correct
reference that the GPU library is checked against.  Only the test suite,
the smoke check and the CPU-baseline leg of the benchmark may import it; the
product path (the C-ABI library and its Python binding) never does, and this
module imports nothing from the product path.

What it computes (Optimus-CC, arXiv 2301.09830):

* Sec. 2.3 (Background, low-rank approximation): the compressor is PowerSGD's
  power iteration, run once per call and warm-started from the factor of the
  previous call.  Sec. 8 (Implementation) states the paper adopted the PowerSGD
  compressor for both the inter-stage and the data-parallel traffic.
* Sec. 5.1 (Lazy error propagation), Eq. (star2): the compression error of one
  call is kept in memory and added to the input of the next call.

The paper never writes the compressor out, so the steps below are the
textbook block power (subspace) iteration in PowerSGD's form:

    A   = M + err_prev                 error-feedback add
    repeat t times:
        P  = A Q                       left product
        P^ = orth(P)                   thin-QR Q-factor, positive R diagonal
        Q  = A^T P^                    right product (Q is not orthonormalised)
    M^  = P^ Q^T                       decompression
    err = A - M^                       residual kept for the next call

``orth`` is modified Gram-Schmidt with one re-orthogonalisation pass (MGS2).
A column whose residual norm after both passes is at most ``tol`` times the
largest original column norm of P is set to zero (rank deficiency; the paper
is silent on it).  Sign convention of the residual: err = input - M^, i.e. the
negative of the paper's epsilon in Eq. (star2), which is "sent - true".

Every array is lifted exactly from its stored dtype to float64 first
(fp32 -> float64 exactly; bf16 bit patterns -> fp32 -> float64 exactly).

Parity status: every public function is pinned by the CPU tests against
closed forms, LAPACK QR, SVD and hand-worked examples; none is "parity
unpinned".
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "lift",
    "mgs2",
    "compress",
    "decompress",
    "err_update",
    "step",
    "step_batched",
    "RANK_TOL",
]

#: relative residual threshold under which MGS2 declares a column dependent.
RANK_TOL = 1e-10


def lift(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 copy of a stored array.

    ``dtype`` is "f32" (x is float32) or "bf16" (x holds bf16 bit patterns as
    uint16: the bf16 value is the fp32 number whose upper 16 bits they are).
    """
    if dtype == "f32":
        if x.dtype != np.float32:
            raise TypeError("f32 data must be stored as numpy float32")
        return x.astype(np.float64)
    if dtype == "bf16":
        if x.dtype != np.uint16:
            raise TypeError("bf16 data must be stored as uint16 bit patterns")
        widened = (x.astype(np.uint32) << np.uint32(16)).view(np.float32)
        return widened.astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def mgs2(P: np.ndarray, tol: float = RANK_TOL) -> np.ndarray:
    """Orthonormal basis of the columns of P by modified Gram-Schmidt, 2 passes.

    Column j of the result is P[:, j] with its components along the already
    accepted columns 0..j-1 removed (twice, one projection at a time), then
    scaled to unit norm.  This is the Q-factor of the thin QR decomposition
    with a positive R diagonal.  A column whose remaining norm is at most
    ``tol * max_k ||P[:, k]||`` is returned as zero and later columns are not
    projected against it.
    """
    P = np.asarray(P, dtype=np.float64)
    m, r = P.shape
    out = np.zeros((m, r), dtype=np.float64)
    scale = max((float(np.linalg.norm(P[:, k])) for k in range(r)), default=0.0)
    accepted: list[int] = []
    for j in range(r):
        v = P[:, j].copy()
        for _ in range(2):
            for k in accepted:
                v -= (out[:, k] @ v) * out[:, k]
        norm = float(np.linalg.norm(v))
        if norm <= tol * scale or norm == 0.0:
            continue
        out[:, j] = v / norm
        accepted.append(j)
    return out


def compress(A: np.ndarray, Q: np.ndarray, iters: int):
    """Power iteration on the error-fed input A (float64), warm-started at Q.

    Returns (P_hat, Q_new): P_hat (m x r) orthonormal, Q_new = A^T P_hat (n x r).
    Sec. 2.3: one power-iteration round per call, reusing the previous factor.
    """
    if iters < 1:
        raise ValueError("iters must be >= 1")
    Q = np.asarray(Q, dtype=np.float64)
    P_hat = None
    for _ in range(iters):
        P = A @ Q
        P_hat = mgs2(P)
        Q = A.T @ P_hat
    return P_hat, Q


def decompress(P_hat: np.ndarray, Q: np.ndarray) -> np.ndarray:
    """M_hat = P_hat Q^T, the low-rank reconstruction (Sec. 9.6 decompression)."""
    return np.asarray(P_hat, np.float64) @ np.asarray(Q, np.float64).T


def err_update(A: np.ndarray, M_hat: np.ndarray) -> np.ndarray:
    """err_new = (M + err_prev) - M_hat, the residual kept in memory (Sec. 5.1)."""
    return A - M_hat


def step(M: np.ndarray, m_dtype: str, err_prev: np.ndarray, Q: np.ndarray,
         rank: int, iters: int) -> dict:
    """One compress + decompress + error-update call on stored-dtype inputs.

    M: m x n, stored dtype ``m_dtype`` ("f32" or "bf16" bits); err_prev: m x n
    float32 (or float64, used as is); Q: n x rank warm start (float32 or
    float64).  Returns float64 arrays P (= P_hat), Q (new), M_hat, err and A.
    The returned Q and err are the state of the next call (Sec. 2.3 warm start,
    Sec. 5.1 lazy error propagation).
    """
    Mf = lift(M, m_dtype)
    m, n = Mf.shape
    if not (1 <= rank <= min(m, n)):
        raise ValueError("rank must satisfy 1 <= rank <= min(m, n)")
    Q = np.asarray(Q)
    if Q.shape != (n, rank):
        raise ValueError("Q must be n x rank")
    A = Mf + np.asarray(err_prev, dtype=np.float64)
    P_hat, Q_new = compress(A, Q.astype(np.float64), iters)
    M_hat = decompress(P_hat, Q_new)
    err = err_update(A, M_hat)
    return {"P": P_hat, "Q": Q_new, "M_hat": M_hat, "err": err, "A": A}


def step_batched(items, rank: int, iters: int) -> list:
    """Independent ``step`` per matrix; items are (M, m_dtype, err_prev, Q)."""
    return [step(M, dt, e, Q, rank, iters) for (M, dt, e, Q) in items]
