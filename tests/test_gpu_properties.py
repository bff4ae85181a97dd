"""GPU-side properties: invariants at fp32 level, bitwise identities between
entry points, determinism, resume, numeric flags and degenerate inputs."""

import numpy as np
import pytest

from gpu_util import to_device, to_host, torch_mod
from workloads import WORKLOADS, Workload

pytestmark = pytest.mark.gpu


def _inputs(m=513, n=300, rank=16, dtype="bf16", seed=5):
    w = WORKLOADS[2].scaled([(m, n)], rank=rank, m_dtype=dtype)
    M = w.matrix(seed, 0)
    return w, M, w.q0(0)


def _run_step(M_dev, err, Q, rank, iters, flags_write=True):
    from paper_2301_09830_amd import optcc
    P, Mh = optcc.occ_step(M_dev, err, Q, rank, iters, write_mhat=flags_write)
    torch_mod().cuda.synchronize()
    return P, Mh


# Ranks on both kernel paths: padded rank <= 16 and padded rank 32..128.
SMALL_LARGE = [16, 64]


@pytest.mark.parametrize("rank", SMALL_LARGE + [128])
def test_invariants_fp32_level(rank):
    torch = torch_mod()
    w, M, q0 = _inputs(rank=rank)
    Md = to_device(M, "bf16")
    err0 = torch.randn(M.shape, device="cuda") * 0.01
    err = err0.clone()
    Q = torch.from_numpy(q0).cuda()
    P, Mh = _run_step(Md, err, Q, rank, 1)
    A = Md.float() + err0
    Pd = P.double()
    eye = Pd.T @ Pd
    assert torch.allclose(eye, torch.eye(rank, dtype=torch.float64, device="cuda"), atol=1e-5)
    # conservation: M_hat + err_new == A up to one fp32 rounding of err
    diff = (Mh.double() + err.double() - A.double()).abs().max().item()
    assert diff <= 2 * np.finfo(np.float32).eps * A.abs().max().item()
    # residual orthogonal to span(P_hat)
    ortho = (Pd.T @ err.double()).abs().max().item()
    assert ortho <= 1e-4 * err.double().norm().item()


@pytest.mark.parametrize("rank,dtype", [(12, "bf16"), (40, "bf16"), (64, "f32"), (100, "f32")])
def test_fused_equals_unfused_bitwise(rank, dtype):
    """occ_step (large ranks: A stored over err, later passes read it back)
    equals occ_compress (re-reads M + err_prev) + occ_decompress +
    occ_err_update bit for bit."""
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    w, M, q0 = _inputs(m=700, n=260, rank=rank, dtype=dtype)
    Md = to_device(M, dtype)
    err = torch.randn(M.shape, device="cuda") * 0.02
    err_a, err_b = err.clone(), err.clone()
    Qa = torch.from_numpy(q0).cuda()
    Qb = Qa.clone()
    P1, Mh1 = optcc.occ_step(Md, err_a, Qa, rank, 2)
    P2 = optcc.occ_compress(Md, err_b, Qb, rank, 2)
    if dtype == "bf16":
        Mh2 = optcc.occ_decompress_ex(P2, Qb, optcc.OCC_DEC_SPLIT_BF16)
    else:
        Mh2 = optcc.occ_decompress(P2, Qb)
    optcc.occ_err_update(Md, err_b, Mh2, err_new=err_b)
    torch.cuda.synchronize()
    for x, y in ((P1, P2), (Qa, Qb), (Mh1, Mh2), (err_a, err_b)):
        assert torch.equal(x.view(torch.int32), y.view(torch.int32))


@pytest.mark.parametrize("rank", [40, 128])
def test_split_decompress_close_to_fp32(rank):
    """occ_decompress_ex with OCC_DEC_SPLIT_BF16 above rank 16 uses the split
    bf16 products of the fused step (two bf16 parts per factor, about 2^-16
    relative per element); occ_decompress stays at fp32 rounding.  Both
    against float64."""
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    g = torch.Generator(device="cuda").manual_seed(3)
    P = torch.randn((700, rank), device="cuda", generator=g)
    Q = torch.randn((260, rank), device="cuda", generator=g)
    ref = P.double() @ Q.double().T
    a = optcc.occ_decompress(P, Q)
    b = optcc.occ_decompress_ex(P, Q, optcc.OCC_DEC_SPLIT_BF16)
    torch.cuda.synchronize()
    rel_a = ((a.double() - ref).norm() / ref.norm()).item()
    rel_b = ((b.double() - ref).norm() / ref.norm()).item()
    print(f"[decompress] rank {rank}: fp32 {rel_a:.2e}, split bf16 {rel_b:.2e}", flush=True)
    assert rel_a <= 1e-6
    assert rel_b <= 1e-4


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("rank,n", [(8, 200), (64, 200), (8, 224), (16, 512), (4, 96)])
def test_compress_without_error_buffer(rank, n, dtype):
    """No error buffer equals a zero one bit for bit.  At rank <= 16 with
    whole 32-column K-steps (n = 96, 224, 512) the zero buffer takes the left
    product's LDS-tile path and no buffer the register path, so this also
    pins the tile layouts (bf16 and fp32 M) to the register loads."""
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    w, M, q0 = _inputs(m=300, n=n, rank=rank, dtype=dtype)
    Md = to_device(M, dtype)
    Qa = torch.from_numpy(q0).cuda()
    Qb = Qa.clone()
    zero = torch.zeros(M.shape, device="cuda")
    Pa = optcc.occ_compress(Md, None, Qa, rank, 1)
    Pb = optcc.occ_compress(Md, zero, Qb, rank, 1)
    torch.cuda.synchronize()
    assert torch.equal(Pa, Pb) and torch.equal(Qa, Qb)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("rank", [32, 64, 128])
def test_large_rank_tile_paths_match_scalar_paths(rank, dtype):
    """Rank > 16, 224 columns: with 16-byte aligned rows the left and right
    products take their LDS-tile paths; with a leading dimension of n + 1
    every pass takes its scalar path.  The products see the same operands in
    the same order, so the two runs agree bit for bit."""
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    m, n = 1000, 224
    w, M, q0 = _inputs(m=m, n=n, rank=rank, dtype=dtype)
    e0 = np.random.default_rng(7).standard_normal((m, n)).astype(np.float32) * 1e-2
    out = []
    for pad in (0, 1):
        full = np.zeros((m, n + pad), dtype=M.dtype)
        full[:, :n] = M
        Md = to_device(full, dtype)[:, :n]
        err_full = torch.zeros((m, n + pad), device="cuda")
        err = err_full[:, :n]
        err.copy_(torch.from_numpy(e0).cuda())
        Q = torch.from_numpy(q0).cuda()
        Mh_full = torch.zeros((m, n + pad), device="cuda")
        P = torch.empty((m, rank), device="cuda")
        optcc.occ_step(Md, err, Q, rank, 2, P=P, M_hat=Mh_full[:, :n])
        torch.cuda.synchronize()
        out.append((P, Q, Mh_full[:, :n].contiguous(), err.contiguous()))
    for a, b, name in zip(out[0], out[1], ("P", "Q", "M_hat", "err")):
        assert torch.equal(a, b), f"{dtype} rank {rank}: {name} differs between the tile and scalar paths"


@pytest.mark.parametrize("rank", [16, 48])
def test_batched_equals_single_bitwise(rank):
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    # (2080, 96): more row blocks than the other matrices together, so the
    # batch's grids are dominated by one matrix
    shapes = [(300, 96), (96, 96), (400, 96), (96, 384), (77, 130), (2080, 96)]
    w = WORKLOADS[3].scaled(shapes, rank=rank)
    mats = [to_device(w.matrix(0, j), "f32") for j in range(len(shapes))]
    errs = [torch.randn(s, device="cuda") * 1e-3 for s in shapes]
    qs = [torch.from_numpy(w.q0(j)).cuda() for j in range(len(shapes))]
    single, batch = [], []
    for j, (m, n) in enumerate(shapes):
        e, q = errs[j].clone(), qs[j].clone()
        P, Mh = optcc.occ_step(mats[j], e, q, rank, 2)
        single.append((P, Mh, e, q))
    items = []
    for j, (m, n) in enumerate(shapes):
        items.append((mats[j], errs[j].clone(), qs[j].clone(),
                      torch.empty((m, rank), device="cuda"), torch.empty((m, n), device="cuda")))
    optcc.occ_step_batched(items, rank, 2)
    torch.cuda.synchronize()
    for (P, Mh, e, q), (_, eb, qb, Pb, Mhb) in zip(single, items):
        assert torch.equal(P, Pb) and torch.equal(Mh, Mhb) and torch.equal(e, eb) and torch.equal(q, qb)


@pytest.mark.parametrize("rank", [16, 128])
def test_deterministic_run_to_run(rank):
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    w, M, q0 = _inputs(m=2048, n=1024, rank=rank)
    Md = to_device(M, "bf16")
    outs = []
    for _ in range(2):
        err = torch.zeros(M.shape, device="cuda")
        Q = torch.from_numpy(q0).cuda()
        for _s in range(3):
            P, Mh = optcc.occ_step(Md, err, Q, rank, 1)
        torch.cuda.synchronize()
        outs.append((P.clone(), Mh.clone(), err.clone(), Q.clone()))
    for x, y in zip(*outs):
        assert torch.equal(x, y)


@pytest.mark.parametrize("rank", [16, 64])
def test_resume_from_saved_state_bitwise(rank):
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    w = WORKLOADS[2].scaled([(640, 384)], rank=rank)
    Ms = [to_device(w.matrix(s, 0), "bf16") for s in range(6)]
    err = torch.zeros((640, 384), device="cuda")
    Q = torch.from_numpy(w.q0(0)).cuda()
    for s in range(6):
        optcc.occ_step(Ms[s], err, Q, rank, 1)
    torch.cuda.synchronize()
    ref = (err.clone(), Q.clone())
    err = torch.zeros((640, 384), device="cuda")
    Q = torch.from_numpy(w.q0(0)).cuda()
    for s in range(3):
        optcc.occ_step(Ms[s], err, Q, rank, 1)
    saved = (err.cpu().numpy().copy(), Q.cpu().numpy().copy())     # checkpoint
    err = torch.from_numpy(saved[0]).cuda()
    Q = torch.from_numpy(saved[1]).cuda()
    for s in range(3, 6):
        optcc.occ_step(Ms[s], err, Q, rank, 1)
    torch.cuda.synchronize()
    assert torch.equal(err, ref[0]) and torch.equal(Q, ref[1])


@pytest.mark.parametrize("rank", SMALL_LARGE)
def test_no_mhat_flag_matches_full_step(rank):
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    w, M, q0 = _inputs(m=500, n=260, rank=rank)
    Md = to_device(M, "bf16")
    e1 = torch.zeros(M.shape, device="cuda")
    e2 = e1.clone()
    q1 = torch.from_numpy(q0).cuda()
    q2 = q1.clone()
    P1, _ = optcc.occ_step(Md, e1, q1, rank, 1)
    P2, Mh2 = optcc.occ_step(Md, e2, q2, rank, 1, write_mhat=False)
    torch.cuda.synchronize()
    assert Mh2 is None
    assert torch.equal(e1, e2) and torch.equal(P1, P2) and torch.equal(q1, q2)


@pytest.mark.parametrize("rank", [8, 64])
def test_zero_input_sets_rank_deficient_flag(rank):
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    M = torch.zeros((200, 100), device="cuda")
    err = torch.zeros_like(M)
    Q = torch.randn((100, rank), device="cuda")
    ws = optcc.alloc_workspace(optcc.occ_workspace_bytes([(200, 100)], rank, 1))
    P, Mh = optcc.occ_step(M, err, Q, rank, 1, ws=ws)
    flags = optcc.occ_get_flags(ws, clear=True)
    assert flags & optcc.OCC_F_RANK_DEFICIENT
    assert not (flags & optcc.OCC_F_NONFINITE)
    assert not P.any() and not Mh.any() and not err.any() and not Q.any()
    assert optcc.occ_get_flags(ws) == 0


@pytest.mark.parametrize("rank,full", [(8, 40), (48, 100)])
def test_exact_low_rank_recovery_and_full_rank(rank, full):
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    g = np.random.default_rng(3)
    A = (g.standard_normal((300, 3)) @ g.standard_normal((3, 120))).astype(np.float32)
    M = torch.from_numpy(A).cuda()
    err = torch.zeros_like(M)
    Q = torch.from_numpy(g.standard_normal((120, rank)).astype(np.float32)).cuda()
    P, Mh = optcc.occ_step(M, err, Q, rank, 1)
    torch.cuda.synchronize()
    assert err.norm().item() <= 1e-5 * M.norm().item()
    # rank = min(m, n): reconstruction equals the input.  An orthonormal
    # warm start keeps cond(P) <= cond(B)^3 (about 50 for a 3:1 Gaussian),
    # so the fp32 subspace error stays far below the bound.
    B = torch.from_numpy(g.standard_normal((3 * full, full)).astype(np.float32)).cuda()
    errb = torch.zeros_like(B)
    q_orth, _ = np.linalg.qr(g.standard_normal((full, full)))
    Qb = torch.from_numpy(q_orth.astype(np.float32)).cuda()
    P, Mh = optcc.occ_step(B, errb, Qb, full, 2)
    torch.cuda.synchronize()
    assert (Mh - B).norm().item() <= 1e-4 * B.norm().item()


@pytest.mark.parametrize("rank", [4, 96])
def test_nonfinite_input_propagates_and_flags(rank):
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    M = torch.randn((256, 128), device="cuda")
    M[17, 5] = float("nan")
    err = torch.zeros_like(M)
    Q = torch.randn((128, rank), device="cuda")
    ws = optcc.alloc_workspace(optcc.occ_workspace_bytes([(256, 128)], rank, 1))
    P, Mh = optcc.occ_step(M, err, Q, rank, 1, ws=ws)
    flags = optcc.occ_get_flags(ws)
    assert flags & optcc.OCC_F_NONFINITE
    assert torch.isnan(Mh).any() and torch.isnan(err).any()


@pytest.mark.parametrize("split", [False, True])
@pytest.mark.parametrize("rank,pad", [(4, 0), (16, 0), (16, 3), (40, 0), (40, 3), (64, 0), (128, 0),
                                      (128, 5)])
def test_decompress_bf16_output_is_rne_of_fp32(rank, pad, split):
    """OCC_DEC_OUT_BF16 stores every element of M_hat rounded to nearest even
    from the fp32 value the same call computes without it: bitwise equal to
    torch's fp32 -> bf16 conversion (also round to nearest even) of the fp32
    output, on the vector store path (pad 0) and the element path (ld =
    n + pad)."""
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    g = torch.Generator(device="cuda").manual_seed(11 + rank)
    m, n = 700, 260
    P = torch.randn((m, rank), device="cuda", generator=g)
    Q = torch.randn((n, rank), device="cuda", generator=g) * 1e-3
    base = optcc.OCC_DEC_SPLIT_BF16 if split else 0
    ref = optcc.occ_decompress_ex(P, Q, base)
    out_full = torch.zeros((m, n + pad), dtype=torch.bfloat16, device="cuda")
    out = optcc.occ_decompress_ex(P, Q, base | optcc.OCC_DEC_OUT_BF16, M_hat=out_full[:, :n])
    torch.cuda.synchronize()
    want = ref.to(torch.bfloat16)
    assert torch.equal(out.contiguous().view(torch.int16), want.view(torch.int16))
    if pad:
        assert not out_full[:, n:].float().any(), "bf16 stores ran past the row"


@pytest.mark.parametrize("shape,rank,iters,wkey", [((1000, 512), 16, 1, 2), ((700, 512), 128, 2, 5),
                                                   ((1000, 4096), 16, 1, 2)])
def test_sender_receiver_round_trip(shape, rank, iters, wkey):
    """Compressed backpropagation across a stage boundary (Sec. 5, 5.1): the
    sending stage runs occ_step without M_hat over consecutive micro-batches,
    carrying err (lazy error propagation) and Q; only P_hat and Q cross; the
    receiving stage rebuilds the gradient with occ_decompress_ex.

    - In fp32 (with the split products of the sender's bf16 step) the
      receiver's M_hat is bitwise the M_hat a fused step would have written.
    - In bf16 (OCC_DEC_OUT_BF16) every element is that value rounded to
      nearest even, so against the float64 oracle its relative Frobenius error
      is at most 2^-9 (the bf16 rounding) plus the fp32 step's own error
      (regression bound 1e-4): bound 2^-9 + 1e-4.  Per row and per 128-column
      tile the same 2^-9 plus the localized regression bound 1e-3.
    - Error feedback telescopes (Eq. (star2) summed over micro-batches): the
      sum of what the receiver got plus the sender's last error equals the sum
      of the true gradients plus the first error, to fp32 rounding."""
    import numpy as np

    import oracle
    from gpu_util import loc_errors, rel_f, to_device, to_host
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    w = WORKLOADS[wkey].scaled([shape], rank=rank, iters=iters)
    m, n = shape
    split = optcc.OCC_DEC_SPLIT_BF16
    err_s = torch.zeros((m, n), device="cuda")         # sender, no M_hat
    err_f = torch.zeros((m, n), device="cuda")         # reference fused step
    Q_s = torch.from_numpy(w.q0(0)).cuda()
    Q_f = Q_s.clone()
    o_err, o_q = np.zeros((m, n)), w.q0(0).astype(np.float64)
    got = torch.zeros((m, n), dtype=torch.float64, device="cuda")
    true = torch.zeros((m, n), dtype=torch.float64, device="cuda")
    bound = 2.0 ** -9 + 1e-4
    for s in range(4):
        Mh = w.matrix(s, 0)
        Md = to_device(Mh, "bf16")
        P_s, _ = optcc.occ_step(Md, err_s, Q_s, rank, iters, write_mhat=False)
        P_f, Mh_f = optcc.occ_step(Md, err_f, Q_f, rank, iters)
        recv32 = optcc.occ_decompress_ex(P_s, Q_s, split)
        recv16 = optcc.occ_decompress_ex(P_s, Q_s, split | optcc.OCC_DEC_OUT_BF16)
        got += recv32.double()
        true += Md.double()
        torch.cuda.synchronize()
        assert torch.equal(recv32, Mh_f), f"step {s}: receiver M_hat differs from the fused step"
        assert torch.equal(err_s, err_f) and torch.equal(Q_s, Q_f)
        ref = oracle.step(Mh, "bf16", o_err, o_q, rank, iters)
        o_err, o_q = ref["err"], ref["Q"]
        a_norm = float(np.linalg.norm(ref["A"]))
        r16 = to_host(recv16)
        rel = rel_f(r16, ref["M_hat"], a_norm)
        row, tile = loc_errors(r16, ref["M_hat"], a_norm)
        print(f"[cb] {m}x{n} r{rank} step {s}: bf16 M_hat rel_F {rel:.3e}, row {row:.3e}, "
              f"tile {tile:.3e} (bound {bound:.3e})", flush=True)
        assert rel <= bound and max(row, tile) <= 2.0 ** -9 + 1e-3
    lhs = got + err_s.double()
    amax = true.abs().max().item()
    tele = (lhs - true).abs().max().item()
    assert tele <= 4 * 4 * np.finfo(np.float32).eps * amax, f"telescoping off by {tele:.3e}"


@pytest.mark.parametrize("rank", [64, 128])
def test_compress_bf16_large_rank_documented_workspace(rank):
    """occ_compress on a bf16 matrix large enough for several column and row
    splits, with exactly the workspace occ_compress_workspace_bytes documents
    for that dtype; the result equals the fused step's P_hat and Q bitwise."""
    from paper_2301_09830_amd import optcc
    torch = torch_mod()
    m, n = 8192, 4096
    w = WORKLOADS[5].scaled([(m, n)], rank=rank, signal_rank=160)
    Md = to_device(w.matrix(0, 0), "bf16")
    nbytes = optcc.occ_compress_workspace_bytes(m, n, rank, 2, optcc.OCC_BF16)
    ws = optcc.alloc_workspace(nbytes)
    assert ws.numel() == max(nbytes, 256)
    Qa = torch.from_numpy(w.q0(0)).cuda()
    Qb = Qa.clone()
    Pa = optcc.occ_compress(Md, None, Qa, rank, 2, ws=ws)
    err = torch.zeros((m, n), device="cuda")
    Pb, _ = optcc.occ_step(Md, err, Qb, rank, 2, write_mhat=False)
    torch.cuda.synchronize()
    assert torch.equal(Pa, Pb) and torch.equal(Qa, Qb)
