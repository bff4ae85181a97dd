"""Shared helpers of the GPU parity tests: upload seeded inputs, run the
library through its binding, run the float64 oracle on the same stored
inputs, and compare.

Comparisons follow independent trajectories: the GPU carries its own fp32
err and Q from step to step and the oracle carries its own float64 state;
no GPU output is ever fed to the oracle.
"""

from __future__ import annotations

import numpy as np

import oracle

TOL = {"f32": 1e-4, "bf16": 2e-2}


def torch_mod():
    import torch
    return torch


def to_device(x: np.ndarray, dtype: str):
    """Stored-dtype numpy array -> CUDA tensor (float32 or bfloat16)."""
    torch = torch_mod()
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(x)).cuda()
    return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).cuda()


def to_host(t) -> np.ndarray:
    return t.detach().float().cpu().numpy()


def rel_f(gpu: np.ndarray, ref: np.ndarray, a_norm: float) -> float:
    """||gpu - ref||_F / ||ref||_F (float64), falling back to ||A||_F when the
    reference is below 1e-12 ||A||_F."""
    diff = np.linalg.norm(gpu.astype(np.float64) - ref)
    den = np.linalg.norm(ref)
    if den < 1e-12 * a_norm:
        den = a_norm
    return float(diff / den) if den > 0 else float(diff)


class GpuState:
    """One matrix's device buffers: err, Q, P, M_hat (fp32)."""

    def __init__(self, m: int, n: int, rank: int, q0: np.ndarray, ld_pad: int = 0):
        torch = torch_mod()
        self.m, self.n, self.rank = m, n, rank
        ld = n + ld_pad
        self.err_full = torch.zeros((m, ld), dtype=torch.float32, device="cuda")
        self.err = self.err_full[:, :n]
        self.Q = torch.from_numpy(np.ascontiguousarray(q0, dtype=np.float32)).cuda()
        self.P = torch.zeros((m, rank), dtype=torch.float32, device="cuda")
        self.Mh_full = torch.full((m, ld), float("nan"), dtype=torch.float32, device="cuda")
        self.M_hat = self.Mh_full[:, :n]


def check_invariants(M_dev, err_prev, err, P, M_hat, label: str):
    """Properties every step satisfies at any size, checked on the GPU:
    M_hat + err == M + err_prev up to one fp32 rounding of err, P_hat has
    orthonormal columns, and the residual is orthogonal to span(P_hat)."""
    torch = torch_mod()
    A = M_dev.float() + err_prev
    amax = A.abs().max().item()
    cons = (M_hat.double() + err.double() - A.double()).abs().max().item()
    assert cons <= 2 * np.finfo(np.float32).eps * amax, f"{label}: M_hat + err != A ({cons:.3e})"
    Pd = P.double()
    r = P.shape[1]
    orth = (Pd.T @ Pd - torch.eye(r, dtype=torch.float64, device=P.device)).abs().max().item()
    assert orth <= 1e-5, f"{label}: P_hat^T P_hat - I = {orth:.3e}"
    res = (Pd.T @ err.double()).abs().max().item()
    assert res <= 1e-4 * err.double().norm().item(), f"{label}: P_hat^T err = {res:.3e}"


def run_workload(w, steps: int, batched: bool | None = None, ld_pad: int = 0,
                 check_oracle: bool = True, oracle_mats=None, on_step=None,
                 invariants_all: bool = False):
    """Run `steps` steps of workload w on the GPU and (optionally) the oracle.

    Returns a list of per-step lists of per-matrix dicts with rel_F errors.
    oracle_mats: indices of the matrices the oracle follows (default: all).
    invariants_all: also check check_invariants() on every matrix.
    """
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    count = len(w.shapes)
    if batched is None:
        batched = count > 1
    states = [GpuState(m, n, w.rank, w.q0(j), ld_pad) for j, (m, n) in enumerate(w.shapes)]
    follow = list(range(count)) if oracle_mats is None else list(oracle_mats)
    ostate = {j: (np.zeros(w.shapes[j]), w.q0(j).astype(np.float64)) for j in follow}
    if batched:
        ws = optcc.alloc_workspace(optcc.occ_workspace_bytes(list(w.shapes), w.rank, w.iters))
    else:
        ws = optcc.alloc_workspace(max(optcc.occ_workspace_bytes([s], w.rank, w.iters)
                                       for s in w.shapes))
    results = []
    for s in range(steps):
        host_M = [w.matrix(s, j) for j in range(count)]
        if ld_pad:
            dev_M = []
            for x in host_M:
                full = np.zeros((x.shape[0], x.shape[1] + ld_pad), dtype=x.dtype)
                full[:, :x.shape[1]] = x
                dev_M.append(to_device(full, w.m_dtype)[:, :x.shape[1]])
        else:
            dev_M = [to_device(x, w.m_dtype) for x in host_M]
        prev = [st.err.clone() for st in states] if invariants_all else None
        if batched:
            items = [(dev_M[j], st.err, st.Q, st.P, st.M_hat) for j, st in enumerate(states)]
            optcc.occ_step_batched(items, w.rank, w.iters, ws=ws)
        else:
            for j, st in enumerate(states):
                optcc.occ_step(dev_M[j], st.err, st.Q, w.rank, w.iters, P=st.P,
                               M_hat=st.M_hat, ws=ws)
        torch.cuda.synchronize()
        if invariants_all:
            for j, st in enumerate(states):
                check_invariants(dev_M[j], prev[j], st.err, st.P, st.M_hat,
                                 f"{w.name} step {s} matrix {j}")
            del prev
        step_res = []
        for j in follow:
            st = states[j]
            out = {"M_hat": to_host(st.M_hat), "err": to_host(st.err), "P": to_host(st.P),
                   "Q": to_host(st.Q)}
            rec = {"j": j}
            if check_oracle:
                e_prev, q_prev = ostate[j]
                ref = oracle.step(host_M[j], w.m_dtype, e_prev, q_prev, w.rank, w.iters)
                ostate[j] = (ref["err"], ref["Q"])
                a_norm = float(np.linalg.norm(ref["A"]))
                rec.update(mhat=rel_f(out["M_hat"], ref["M_hat"], a_norm),
                           err=rel_f(out["err"], ref["err"], a_norm),
                           a_norm=a_norm)
            if on_step is not None:
                on_step(s, j, out, host_M[j])
            step_res.append(rec)
        results.append(step_res)
    return results, states, ws


def assert_parity(results, dtype: str, label: str):
    tol = TOL[dtype]
    worst = max(max(r["mhat"], r["err"]) for step in results for r in step)
    print(f"[parity] {label}: worst rel_F = {worst:.3e} (tol {tol:g})", flush=True)
    for s, step in enumerate(results):
        for r in step:
            assert r["mhat"] <= tol, f"{label} step {s} matrix {r['j']}: rel_F(M_hat)={r['mhat']:.3e}"
            assert r["err"] <= tol, f"{label} step {s} matrix {r['j']}: rel_F(err)={r['err']:.3e}"
