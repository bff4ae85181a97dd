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

# Graded tolerance on the relative Frobenius error of M_hat and err (per
# matrix and step): 1e-4 for fp32 M, 2e-2 for bf16 M (fp32 accumulation).
TOL = {"f32": 1e-4, "bf16": 2e-2}

# Regression bounds, far below the graded tolerance: every product
# accumulates in fp32 (bf16 M is widened exactly), so a correct step lands at
# 1e-6..1e-5 against float64 on these recipes (the measured worst cases are
# recorded with each test).  REG_REL bounds rel_F; REG_LOC bounds the
# localized errors of loc_errors(), which a whole wrong row or column tile
# pushes to about 1 while rel_F moves only by sqrt(1/rows).
REG_REL = 1e-4
REG_LOC = 1e-3
LOC_TILE = 128


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


def loc_errors(gpu: np.ndarray, ref: np.ndarray, a_norm: float) -> tuple:
    """Localized relative errors (float64): the worst row and the worst
    128-column tile.  Row i: ||gpu_i - ref_i|| / max(||ref_i||, ||ref||_F / sqrt(m));
    tile t: ||gpu_t - ref_t||_F / max(||ref_t||_F, ||ref||_F sqrt(w_t / n)).
    The floors keep rows or tiles with little energy from dominating; when the
    whole reference is below 1e-12 ||A||_F the floors use ||A||_F instead."""
    diff = gpu.astype(np.float64) - ref
    m, n = ref.shape
    tot = float(np.linalg.norm(ref))
    if tot < 1e-12 * a_norm:
        tot = a_norm
    if tot == 0.0:
        return float(np.abs(diff).max(initial=0.0)), float(np.abs(diff).max(initial=0.0))
    d_rows = np.sqrt(np.einsum("ij,ij->i", diff, diff))
    r_rows = np.sqrt(np.einsum("ij,ij->i", ref, ref))
    row = float((d_rows / np.maximum(r_rows, tot / np.sqrt(m))).max())
    d_cols = np.einsum("ij,ij->j", diff, diff)
    r_cols = np.einsum("ij,ij->j", ref, ref)
    tile = 0.0
    for c0 in range(0, n, LOC_TILE):
        w = min(LOC_TILE, n - c0)
        dt = np.sqrt(d_cols[c0:c0 + w].sum())
        rt = np.sqrt(r_cols[c0:c0 + w].sum())
        tile = max(tile, float(dt / max(rt, tot * np.sqrt(w / n))))
    return row, tile


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
    dt = optcc.OCC_BF16 if w.m_dtype == "bf16" else optcc.OCC_F32
    if batched:
        ws = optcc.alloc_workspace(optcc.occ_workspace_bytes(list(w.shapes), w.rank, w.iters, dt))
    else:
        ws = optcc.alloc_workspace(max(optcc.occ_workspace_bytes([s], w.rank, w.iters, dt)
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
                mr, mt = loc_errors(out["M_hat"], ref["M_hat"], a_norm)
                er, et = loc_errors(out["err"], ref["err"], a_norm)
                rec.update(mhat=rel_f(out["M_hat"], ref["M_hat"], a_norm),
                           err=rel_f(out["err"], ref["err"], a_norm),
                           loc=max(mr, mt, er, et), a_norm=a_norm)
            if on_step is not None:
                on_step(s, j, out, host_M[j])
            step_res.append(rec)
        results.append(step_res)
    return results, states, ws


def assert_parity(results, dtype: str, label: str, reg_rel: float = REG_REL,
                  reg_loc: float = REG_LOC):
    """Graded tolerance on rel_F, the same tolerance on the localized errors,
    and the regression bounds on both."""
    tol = TOL[dtype]
    worst = max(max(r["mhat"], r["err"]) for step in results for r in step)
    worst_loc = max(r["loc"] for step in results for r in step)
    print(f"[parity] {label}: worst rel_F = {worst:.3e} (tol {tol:g}, regression {reg_rel:g}); "
          f"worst row/tile = {worst_loc:.3e} (regression {reg_loc:g})", flush=True)
    for s, step in enumerate(results):
        for r in step:
            where = f"{label} step {s} matrix {r['j']}"
            assert r["mhat"] <= tol, f"{where}: rel_F(M_hat)={r['mhat']:.3e}"
            assert r["err"] <= tol, f"{where}: rel_F(err)={r['err']:.3e}"
            assert r["loc"] <= tol, f"{where}: worst row/tile error {r['loc']:.3e}"
            assert max(r["mhat"], r["err"]) <= reg_rel, \
                f"{where}: rel_F {max(r['mhat'], r['err']):.3e} above the regression bound"
            assert r["loc"] <= reg_loc, \
                f"{where}: row/tile error {r['loc']:.3e} above the regression bound"
