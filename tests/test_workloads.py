"""Seeded input generators: determinism, shapes and recipe statistics."""

import hashlib

import numpy as np

from workloads import WORKLOADS, high_snr


def _digest(a):
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def test_table_shapes_and_dtypes():
    w = WORKLOADS
    assert w[1].shapes == ((1024, 1024),) and w[1].m_dtype == "f32" and w[1].rank == 4
    assert w[2].shapes == ((8192, 4096),) and w[2].m_dtype == "bf16" and w[2].rank == 16
    assert len(w[3].shapes) == 36 and w[3].rank == 32 and w[3].iters == 2
    assert {s for s in w[3].shapes} == {(9216, 3072), (3072, 3072), (12288, 3072), (3072, 12288)}
    assert w[4].shapes == ((51200, 3072),) and w[4].rank == 64
    assert w[5].shapes == ((16384, 8192),) * 4 and w[5].rank == 128 and w[5].iters == 2
    assert w[3].elements == 1_019_215_872 and w[5].elements == 536_870_912


def test_config1_literal_seeds():
    w = WORKLOADS[1]
    M = w.matrix(0, 0)
    np.testing.assert_array_equal(M, np.random.default_rng(0).standard_normal((1024, 1024)).astype(np.float32))
    np.testing.assert_array_equal(w.q0(0), np.random.default_rng(1).standard_normal((1024, 4)).astype(np.float32))


def test_deterministic_and_step_dependent():
    w = WORKLOADS[2].scaled([(300, 200)])
    a, b = w.matrix(0, 0), w.matrix(0, 0)
    assert a.dtype == np.uint16 and _digest(a) == _digest(b)
    assert _digest(w.matrix(1, 0)) != _digest(a)
    assert _digest(w.q0(0)) == _digest(w.q0(0))


def test_lowrank_recipe_spectrum():
    w = WORKLOADS[2].scaled([(400, 300)], noise=0.0)
    x = (w.matrix(0, 0).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    s = np.linalg.svd(x, compute_uv=False)
    np.testing.assert_allclose(s[:32], 1.0 / np.arange(1, 33), rtol=2e-2)
    assert s[32] < 0.05 * s[31]          # bf16 rounding noise only


def test_high_snr_scales_signal():
    w = high_snr(WORKLOADS[2].scaled([(256, 128)]))
    x = (w.matrix(0, 0).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert 0.5 < np.sqrt(np.mean(x ** 2)) < 2.0


def test_zipf_embedding_rows():
    w = WORKLOADS[4]
    M = w.matrix(0, 0)
    nz = np.flatnonzero(np.abs(M).sum(axis=1))
    assert 2300 < nz.size < 2600
    assert nz[0] == 0                         # the most frequent token is row 0
    counts = np.abs(M[nz[:4]]).std(axis=1)
    assert counts[0] > counts[3]              # the frequent row accumulates more draws
