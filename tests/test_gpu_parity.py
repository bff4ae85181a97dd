"""GPU parity: liboptcc (through its binding) against the float64 oracle.

Sizes are chosen so the oracle finishes in seconds while the kernels still
see several tiles and ragged tails; the full-size workloads are in
test_gpu_full.py.  Tolerance (relative Frobenius error of M_hat and of err):
1e-4 for fp32 M, 2e-2 for bf16 M (fp32 accumulation).
"""

import numpy as np
import pytest

from gpu_util import TOL, assert_parity, rel_f, run_workload, to_device, to_host, torch_mod
from workloads import WORKLOADS, Workload, high_snr

pytestmark = pytest.mark.gpu


def test_config1_full_size():
    res, _, _ = run_workload(WORKLOADS[1], 1)
    assert_parity(res, "f32", "gauss_1024 r4 t1")


def test_config2_ragged_multistep():
    w = WORKLOADS[2].scaled([(1000, 700)])
    res, _, _ = run_workload(w, 4)
    assert_parity(res, "bf16", "act_grad 1000x700 r16 t1 x4 steps")


def test_config2_high_snr_ragged():
    w = high_snr(WORKLOADS[2].scaled([(777, 520)]))
    res, _, _ = run_workload(w, 3)
    assert_parity(res, "bf16", "act_grad high-SNR 777x520", reg_rel=5e-4, reg_loc=5e-3)


@pytest.mark.parametrize("shape", [(1000, 512), (1000, 4096)])
def test_config2_high_snr_lds_tiles(shape):
    """High-SNR recipe at widths that are multiples of 32: the rank-16 left
    product takes its LDS-tile path, as on the full-size input."""
    w = high_snr(WORKLOADS[2].scaled([shape]))
    res, _, _ = run_workload(w, 3)
    assert_parity(res, "bf16", f"act_grad high-SNR {shape[0]}x{shape[1]} (LDS tiles)",
                  reg_rel=5e-4, reg_loc=5e-3)


@pytest.mark.parametrize("rank", [1, 3, 4, 8, 16, 17, 32, 64, 100, 128])
@pytest.mark.parametrize("iters", [1, 2])
def test_rank_sweep_fp32(rank, iters):
    w = Workload(90, "sweep", ((300, 257),), "f32", rank, iters, 2, "gauss", std=1.0)
    res, _, _ = run_workload(w, 2)
    assert_parity(res, "f32", f"sweep 300x257 r{rank} t{iters}")


@pytest.mark.parametrize("rank", [4, 16, 32])
def test_max_iterations(rank):
    """OCC_MAX_ITERS (64) power-iteration rounds per step on a low-rank matrix
    whose spectrum (1/j, j = 1..48, noise 1e-4) separates every leading
    subspace used here: the rounds contract towards it, so the fp32 and
    float64 trajectories stay together through all 64."""
    w = Workload(91, "maxiter", ((300, 257),), "f32", rank, 64, 2, "lowrank",
                 signal_rank=48, noise=1e-4)
    res, _, _ = run_workload(w, 2)
    assert_parity(res, "f32", f"lowrank 300x257 r{rank} t64")


@pytest.mark.parametrize("rank", [4, 16, 33, 128])
def test_rank_sweep_bf16(rank):
    w = WORKLOADS[2].scaled([(600, 333)], rank=rank, signal_rank=48)
    res, _, _ = run_workload(w, 2)
    assert_parity(res, "bf16", f"bf16 600x333 r{rank}")


@pytest.mark.parametrize("shape", [(1000, 512), (77, 32), (300, 96), (4100, 224)])
@pytest.mark.parametrize("rank", [3, 8, 16])
def test_bf16_whole_ksteps_lds_tiles(shape, rank):
    """bf16 M whose width is a multiple of 32 columns takes the left product's
    LDS-tile path: ragged rows, fewer K-steps than waves, padded and unpadded
    ranks."""
    w = WORKLOADS[2].scaled([shape], rank=rank)
    res, _, _ = run_workload(w, 2)
    assert_parity(res, "bf16", f"bf16 {shape[0]}x{shape[1]} r{rank} (LDS tiles)")


@pytest.mark.parametrize("shape,rank", [(s, r) for r in (32, 64, 128)
                                        for s in ((1000, 512), (4100, 224), (130, 128), (300, 160))]
                         + [((77, 32), 32), ((77, 96), 64)])
def test_bf16_large_rank_whole_columns(shape, rank):
    """bf16 M at rank > 16 whose width is a multiple of 32 columns: the left
    products and the right product stage the stored A through LDS tiles, the
    right product its P_hat^T operand from 16-row tiles.  Covers several row
    splits with a ragged last group (4100 rows), a single ragged group (77),
    waves whose columns run past n (96, 160 and 224 columns at ranks 32 and
    64) and waves wholly past n (160 and 224 columns at rank 128).  The bound
    is the split-product accuracy bound of the test below."""
    w = WORKLOADS[5].scaled([shape], rank=rank, signal_rank=160)
    res, _, _ = run_workload(w, 2)
    assert_parity(res, "bf16", f"bf16 {shape[0]}x{shape[1]} r{rank} (LDS tiles)")
    worst = max(max(r["mhat"], r["err"]) for step in res for r in step)
    assert worst <= 5e-4, f"split products off: {worst:.3e}"


@pytest.mark.parametrize("shape,rank", [(s, r) for r in (32, 64, 128)
                                        for s in ((1000, 512), (4100, 224), (130, 128), (300, 160))]
                         + [((77, 32), 32), ((77, 96), 64)])
def test_fp32_large_rank_whole_columns(shape, rank):
    """fp32 M at rank > 16 whose width is a multiple of 32 columns: the left
    products stage A through LDS tiles and the right product stages the
    stored A and the P_hat rows by DMA several groups ahead.  The same edge
    cases as the bf16 test above (ragged last groups, waves past n)."""
    w = WORKLOADS[3].scaled([shape], rank=rank)
    res, _, _ = run_workload(w, 2)
    assert_parity(res, "f32", f"fp32 {shape[0]}x{shape[1]} r{rank} (LDS tiles)")


def test_config3_stage_batched_small():
    shapes = [(3 * 96, 96), (96, 96), (4 * 96, 96), (96, 4 * 96)] * 2
    w = WORKLOADS[3].scaled(shapes)
    res, _, _ = run_workload(w, 2, batched=True)
    assert_parity(res, "f32", "stage weights h=96 x2 layers, batched")


def test_config4_zipf_small():
    w = WORKLOADS[4].scaled([(2000, 300)], tokens=400)
    res, _, _ = run_workload(w, 2)
    assert_parity(res, "f32", "embedding 2000x300 zipf")


def test_config5_batched_small():
    w = WORKLOADS[5].scaled([(700, 520)] * 2, signal_rank=160)
    res, _, _ = run_workload(w, 2, batched=True)
    assert_parity(res, "bf16", "act_grad 2x700x520 r128 t2 batched")


@pytest.mark.parametrize("shape", [(700, 520), (700, 512)])
def test_config5_high_snr_small(shape):
    """High-SNR rank-128 recipe; 512 columns take the LDS-tile paths."""
    w = high_snr(WORKLOADS[5].scaled([shape], signal_rank=160))
    res, _, _ = run_workload(w, 2)
    assert_parity(res, "bf16", f"act_grad high-SNR {shape[0]}x{shape[1]} r128 t2",
                  reg_rel=5e-4, reg_loc=5e-3)


@pytest.mark.parametrize("rank,iters,ratio", [(8, 2, 1.5), (16, 2, 1.2), (12, 3, 1.2), (32, 2, 1.1),
                                              (64, 2, 1.05), (128, 2, 1.025)])
def test_ill_conditioned_iterates_second_pass(rank, iters, ratio):
    """Geometric spectrum ratio^-j: the power iterates P have condition
    number ratio^((2t-1)(r-1)) between 1e3 and 1e5 (1.05^189 = 1.0e4 at rank
    64, 1.025^381 = 1.2e4 at rank 128), so the Cholesky diagonal spans more
    than 1e3 and the CholeskyQR second pass runs, on the small-rank kernel up
    to rank 16 and on the blocked fp64 Cholesky above.  (Much larger
    condition numbers exceed what an fp32 P can resolve.)  The recipe's
    "noise" field carries the ratio."""
    w = Workload(93, "geom", ((400, 300),), "f32", rank, iters, 2, "geom",
                 signal_rank=rank + 8, noise=ratio)
    res, _, _ = run_workload(w, 2)
    assert_parity(res, "f32", f"geometric {ratio}^-j r{rank} t{iters}")


@pytest.mark.parametrize("kind", ["lowrank", "geom"])
def test_batched_small_rank_split_sums(kind):
    """One batched small-rank step (one factor block per matrix in the right
    product's launch) over matrices whose right products have many row
    splits: 2000, 4000, 8000 and 16000 rows of 96 columns give 63, 125, 250
    and 500 splits, whose sums the finishing kernel shares over 2, 4, 8 and 16
    threads per element; 20000 x 96 has more row blocks than left-product
    blocks (each block takes several); 300 x 257 is wide.  "geom" makes the
    power iterates of every matrix ill-conditioned enough for the second
    CholeskyQR pass inside the batch."""
    shapes = ((2000, 96), (4000, 96), (8000, 96), (16000, 96), (20000, 96), (300, 257))
    if kind == "lowrank":
        w = Workload(94, "mixed", shapes, "f32", 8, 2, 2, "lowrank", signal_rank=48, noise=1e-3)
    else:
        w = Workload(95, "mixed_geom", shapes, "f32", 8, 2, 2, "geom", signal_rank=16, noise=1.5)
    res, _, _ = run_workload(w, 2, batched=True)
    assert_parity(res, "f32", f"batched {kind} r8 t2, {len(shapes)} matrices")


@pytest.mark.parametrize("shape,rank,iters", [((20000, 96), 16, 1), ((9000, 130), 8, 2),
                                              ((8193, 64), 4, 1)])
def test_tall_small_rank_chunked_orthogonalisation(shape, rank, iters):
    """More than 64 x 128 rows at rank <= 16: the orthogonalisation kernel
    runs 64 blocks, each forming P_hat for several consecutive 128-row chunks
    (8193 rows: one block takes the single row of the last chunk)."""
    w = Workload(94, "tall", (shape,), "f32", rank, iters, 2, "gauss", std=1.0)
    res, _, _ = run_workload(w, 2)
    assert_parity(res, "f32", f"tall {shape[0]}x{shape[1]} r{rank} t{iters}")


def test_tall_small_rank_second_pass():
    """A tall matrix with ill-conditioned iterates (geometric spectrum 1.2^-j,
    rank 16, t = 2): the second CholeskyQR pass runs with capped blocks."""
    w = Workload(95, "geom_tall", ((12000, 64),), "f32", 16, 2, 2, "geom", signal_rank=24,
                 noise=1.2)
    res, _, _ = run_workload(w, 2)
    assert_parity(res, "f32", "geometric 1.2^-j 12000x64 r16 t2")


@pytest.mark.parametrize("shape,rank", [((1, 1), 1), ((5, 3), 3), ((64, 1), 1), ((1, 100), 1),
                                        ((65, 33), 8), ((3, 200), 2)])
def test_tiny_shapes(shape, rank):
    w = Workload(91, "tiny", (shape,), "f32", rank, 1, 1, "gauss", std=1.0)
    res, _, _ = run_workload(w, 1)
    assert_parity(res, "f32", f"tiny {shape} r{rank}")


def test_unaligned_leading_dimension():
    w = Workload(92, "ldpad", ((130, 75),), "f32", 8, 2, 2, "gauss", std=1.0)
    res, _, _ = run_workload(w, 2, ld_pad=1)
    assert_parity(res, "f32", "ld = n + 1 (scalar path)")
    wb = WORKLOADS[2].scaled([(130, 75)], rank=8)
    res, _, _ = run_workload(wb, 2, ld_pad=3)
    assert_parity(res, "bf16", "bf16 ld = n + 3 (scalar path)")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("ld_pad", [1, 2])
@pytest.mark.parametrize("rank", [32, 64, 128])
def test_large_rank_padded_rows(rank, ld_pad, dtype):
    """Rows of pitch n + 1 (a multiple of 4: 16-byte accesses, with a ragged
    last piece of 3 columns) and n + 2 (element accesses) at padded ranks
    32-128, where the reconstruction stores straight from the MFMA layout
    (rank 32, 128, bf16) or through an LDS tile by rows (fp32 rank 64).  The
    padding columns of err and M_hat must never be written."""
    shape = (300, 151)
    if dtype == "f32":
        w = Workload(95, "ldpad_large", (shape,), "f32", rank, 2, 2, "gauss", std=1.0)
    else:
        w = WORKLOADS[5].scaled([shape], rank=rank)
    res, states, _ = run_workload(w, 2, ld_pad=ld_pad)
    assert_parity(res, dtype, f"{dtype} {shape} rank {rank} ld = n + {ld_pad}")
    torch = torch_mod()
    st = states[0]
    assert bool(torch.isnan(st.Mh_full[:, shape[1]:]).all()), "M_hat padding written"
    assert bool((st.err_full[:, shape[1]:] == 0).all()), "err padding written"


@pytest.mark.parametrize("snr", [False, True])
@pytest.mark.parametrize("rank", [32, 64, 128])
def test_bf16_large_rank_split_products_accuracy(rank, snr):
    """bf16 M at rank > 16 runs its left and right products and the
    reconstruction on the bf16 matrix cores with each operand split as
    x = x_hi + x_lo (x - x_hi - x_lo below 2^-16 |x|).  The split must keep the
    result close to fp32 arithmetic: measured 1e-5 (noise-dominated) to 7e-5
    (high SNR, where err is 1 % of A) against the float64 oracle with the
    products split.  Dropping the lo parts would leave bf16 operands (2^-9
    relative), about 2e-3 per product, so the bound 5e-4 -- well inside the
    2e-2 bf16 tolerance -- catches a broken split."""
    w = WORKLOADS[5].scaled([(700, 520)], rank=rank, signal_rank=160)
    if snr:
        w = high_snr(w)
    res, _, _ = run_workload(w, 2)
    worst = max(max(r["mhat"], r["err"]) for step in res for r in step)
    print(f"[split] bf16 700x520 rank {rank} high_snr={snr}: worst rel_F = {worst:.3e}", flush=True)
    assert worst <= 5e-4
