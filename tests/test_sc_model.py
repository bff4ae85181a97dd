"""Selective stage compression model (Sec. 7) on the host: the
one-forward-one-backward pipeline simulation and the stage selection.  No
device is touched.

Pins: the 1F1B schedule's closed forms (no hop latency: the last stage-0
backward ends at (m + S - 1)(F + B), the pipeline-bubble result for uniform
stages, and stage s finishes s backward passes earlier because the last
micro-batch's backward runs down the stages one after the other; one
micro-batch with hop latency p: S(F + B) + 2(S - 1)p - s(B + p)), a
hand-simulated 2-stage case, and the selection against brute force over every
choice of stages."""

import itertools
import os
import random

import pytest

from paper_2301_09830_amd import build as buildmod
from paper_2301_09830_amd import optcc


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not os.path.exists(buildmod.LIB):
        buildmod.build()
    optcc.lib()


@pytest.mark.parametrize("S,m,F,B", [(1, 5, 1.0, 2.0), (4, 4, 1.0, 2.0), (4, 16, 0.7, 1.3),
                                     (8, 32, 2.0, 2.0), (3, 9, 1.0, 3.0)])
def test_1f1b_closed_form_without_hop_latency(S, m, F, B):
    done, end = optcc.occ_pipeline_1f1b(S, m, F, B, 0.0)
    t0 = (m + S - 1) * (F + B)
    assert end == pytest.approx(t0, rel=1e-12)
    for s in range(S):
        assert done[s] == pytest.approx(t0 - s * B, rel=1e-12)


@pytest.mark.parametrize("S,F,B,p", [(2, 1.0, 2.0, 0.5), (4, 1.0, 1.0, 0.25), (6, 0.5, 1.5, 1.0)])
def test_1f1b_single_micro_batch_with_hops(S, F, B, p):
    done, _ = optcc.occ_pipeline_1f1b(S, 1, F, B, p)
    for s in range(S):
        assert done[s] == pytest.approx(S * (F + B) + 2 * (S - 1) * p - s * (B + p), rel=1e-12)


def test_1f1b_hand_simulated_two_stages():
    # stage 1: F0 [1,2] B0 [2,4] F1 [4,5] B1 [5,7]; stage 0: F0 [0,1] F1 [1,2] B0 [4,6] B1 [7,9]
    done, end = optcc.occ_pipeline_1f1b(2, 2, 1.0, 2.0, 0.0)
    assert done == [9.0, 7.0] and end == 9.0


def test_1f1b_later_stages_finish_first():
    done, _ = optcc.occ_pipeline_1f1b(8, 24, 1.0, 2.1, 0.05)
    assert all(done[s] > done[s + 1] for s in range(7))


def _brute(stages, k):
    best = None
    for j in range(k + 1):
        for sub in itertools.combinations(range(len(stages)), j):
            end = max(b + (z + c2 if s in sub else c) for s, (b, c, c2, z) in enumerate(stages))
            best = end if best is None else min(best, end)
    return best


def test_selection_matches_brute_force():
    rng = random.Random(5)
    for _ in range(300):
        S = rng.randint(1, 7)
        stages = [(rng.uniform(0, 10), rng.uniform(0, 5), rng.uniform(0, 2), rng.uniform(0, 3))
                  for _ in range(S)]
        k = rng.randint(0, S)
        sel, end = optcc.occ_sc_select(stages, k)
        assert sum(sel) <= k
        got = max(b + (z + c2 if sel[s] else c) for s, (b, c, c2, z) in enumerate(stages))
        assert got == pytest.approx(end, rel=1e-12)
        assert end == pytest.approx(_brute(stages, k), rel=1e-12)


def test_selection_under_1f1b_starts_from_the_earliest_stage():
    """Uniform stages of a 1F1B pipeline: the exchange of stage 0 ends last,
    so it is compressed first, then stage 1, and so on (the order Sec. 7
    describes); a budget of 75 % of 4 stages compresses stages 0-2."""
    done, _ = optcc.occ_pipeline_1f1b(4, 16, 1.0, 2.0, 0.1)
    stages = [(d, 6.0, 0.5, 0.4) for d in done]
    for k, want in ((1, [1, 0, 0, 0]), (2, [1, 1, 0, 0]), (3, [1, 1, 1, 0])):
        sel, _ = optcc.occ_sc_select(stages, k)
        assert sel == want


def test_selection_stops_when_compression_does_not_pay():
    # compressing costs more than the exchange it replaces: nothing chosen
    sel, end = optcc.occ_sc_select([(10.0, 1.0, 0.5, 2.0), (9.0, 1.0, 0.5, 2.0)], 2)
    assert sel == [0, 0] and end == 11.0


def test_invalid_arguments():
    with pytest.raises(optcc.OccError):
        optcc.occ_pipeline_1f1b(0, 4, 1.0, 1.0)
    with pytest.raises(optcc.OccError):
        optcc.occ_pipeline_1f1b(4, 4, -1.0, 1.0)
    with pytest.raises(optcc.OccError):
        optcc.occ_sc_select([(1.0, float("nan"), 0.0, 0.0)], 1)
    with pytest.raises(optcc.OccError):
        optcc.occ_sc_select([(1.0, 1.0, 0.0, 0.0)], -1)
