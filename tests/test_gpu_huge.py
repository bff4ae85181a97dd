"""A step on a matrix of more than 2^31 elements (49152 x 45056), at a small
and a large rank: every element offset past 2^31 has to be formed in 64 bits.

The oracle is not run at this size.  Inputs are seeded normal draws made on
the device, and the checks are properties every step satisfies at any size,
taken on the whole matrix where that is cheap on the GPU and on rows and
columns sampled at both ends (the last rows start past element 2^31):
  M_hat + err == M + err_prev (one fp32 rounding of err), every element;
  P_hat^T P_hat == I;
  Q == A^T P_hat on sampled columns (float64 on the host);
  M_hat == P_hat Q^T on sampled rows (float64 on the host).
"""

import numpy as np
import pytest

from gpu_util import torch_mod

pytestmark = pytest.mark.gpu

SHAPE = (49152, 45056)   # 2,214,592,512 elements


def _say(msg: str) -> None:
    print(f"[huge] {msg}", flush=True)


@pytest.mark.parametrize("dtype,rank", [("bf16", 16), ("f32", 64)])
def test_step_past_2pow31_elements(dtype, rank):
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    m, n = SHAPE
    assert m * n > 2 ** 31 and (m - 1) * n > 2 ** 31
    _say(f"{m}x{n} {dtype} rank {rank}: drawing inputs")
    g = torch.Generator(device="cuda")
    g.manual_seed(20230123 + rank)
    M = torch.randn((m, n), generator=g, device="cuda", dtype=torch.float32)
    if dtype == "bf16":
        M = M.to(torch.bfloat16)
    err = torch.randn((m, n), generator=g, device="cuda", dtype=torch.float32).mul_(0.01)
    Q = torch.randn((n, rank), generator=g, device="cuda", dtype=torch.float32)
    err_prev = err.clone()
    rows = [0, 1, m // 2, m - 2, m - 1]
    cols = [0, n // 2, n - 1]
    A_cols = (M[:, cols].float() + err[:, cols]).double().cpu().numpy()

    _say("step")
    P, Mh = optcc.occ_step(M, err, Q, rank, 1)
    torch.cuda.synchronize()

    _say("M_hat + err == A on every element")
    worst, amax = 0.0, 0.0
    for r0 in range(0, m, 4096):
        A = M[r0:r0 + 4096].float() + err_prev[r0:r0 + 4096]
        amax = max(amax, A.abs().max().item())
        worst = max(worst, (Mh[r0:r0 + 4096].double() + err[r0:r0 + 4096].double()
                            - A.double()).abs().max().item())
        del A
    assert worst <= 2 * np.finfo(np.float32).eps * amax, f"M_hat + err != A ({worst:.3e})"

    _say("P_hat orthonormal, Q and M_hat on sampled columns and rows")
    Ph = P.double().cpu().numpy()
    Qh = Q.double().cpu().numpy()
    orth = np.abs(Ph.T @ Ph - np.eye(rank)).max()
    assert orth <= 1e-5, f"P_hat^T P_hat - I = {orth:.3e}"
    q_ref = A_cols.T @ Ph                       # rows `cols` of A^T P_hat
    for i, c in enumerate(cols):
        scale = np.linalg.norm(A_cols[:, i])
        dq = np.abs(Qh[c] - q_ref[i]).max()
        assert dq <= 1e-4 * scale, f"Q row {c}: {dq:.3e} (|A col| {scale:.3e})"
    Mh_rows = Mh[rows].double().cpu().numpy()
    m_ref = Ph[rows] @ Qh.T
    dm = np.abs(Mh_rows - m_ref).max()
    assert dm <= 1e-5 * np.abs(m_ref).max(), f"M_hat rows: {dm:.3e}"
    _say(f"ok: M_hat + err vs A {worst:.2e}, orth {orth:.2e}, M_hat rows {dm:.2e}")
    del M, err, err_prev, Mh, P, Q
    torch.cuda.empty_cache()
