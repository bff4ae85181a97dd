"""Seeded synthetic inputs for the compressor (shared by tests, bench and smoke).

This module holds input generation only: random draws, casts to the stored
dtype and the workload table.  It contains none of the compressor's
arithmetic, so both the GPU library's tests and the float64 oracle can consume
its arrays.

The paper's tensors are Megatron GPT gradients (Sec. 9.1) that are not
available; each recipe below stands in for one kind of traffic the paper
compresses, with the shapes of the five workloads:

1. "gauss_1024": a 1024x1024 fp32 matrix of i.i.d. N(0,1) entries (seed 0),
   rank 4, initial Q of N(0,1) entries (seed 1), one step.
2. "act_grad_8192x4096": an inter-stage activation gradient (Sec. 5: micro-batch
   4 x seq 2048 flattened against hidden 4096), bf16, a rank-32 signal with
   singular values 1/k plus N(0, 0.01) noise, rank 16, 1 power iteration,
   8 consecutive steps carrying err and Q.
3. "stage_weights_h3072": the data-parallel weight gradients of one pipeline
   stage (Sec. 7) of an h=3072 GPT: 9 layers x {QKV 9216x3072, proj 3072x3072,
   fc1 12288x3072, fc2 3072x12288}, fp32 N(0, 1e-3), rank 32, 2 iterations.
4. "embedding_51200x3072": an embedding gradient (Sec. 6): 8192 Zipf(1.1)
   token ids over a 51200 vocabulary, each adding an N(0, 1e-2) row, fp32,
   rank 64, 1 iteration.
5. "act_grad_4x16384x8192": four large bf16 inter-stage gradients with a
   decaying rank-256 signal plus noise, rank 128, 2 iterations, batched.

Random streams: numpy PCG64 seeded with SeedSequence([config, step, matrix,
role]), role 0 = values/noise, 1 = initial Q, 2 = left singular factor U,
3 = right singular factor V, 4 = token ids.  "N(0, x)" means standard
deviation x.  The signal subspaces (U, V) of workloads 2 and 5 are drawn once
(step 0) and kept for every step; the noise is fresh each step, as consecutive
gradients share their dominant subspace.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

ROLE_VALUES, ROLE_Q0, ROLE_U, ROLE_V, ROLE_TOKENS = 0, 1, 2, 3, 4


def stream(config: int, step: int, mat: int, role: int) -> np.random.Generator:
    """The PCG64 generator of one (config, step, matrix, role) stream."""
    return np.random.default_rng(np.random.SeedSequence([config, step, mat, role]))


def bf16_bits(x) -> np.ndarray:
    """Round float32 values to bf16, round-to-nearest-even; returns uint16 bits.

    NaN stays NaN (quiet bit forced), infinities stay infinite, values that
    round past the largest finite bf16 become infinity (IEEE behaviour).
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    rounded = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint32)
    nan = np.isnan(x)
    if nan.any():
        rounded = np.where(nan, ((u >> np.uint64(16)) | np.uint64(0x40)).astype(np.uint32),
                           rounded)
    return (rounded & np.uint32(0xFFFF)).astype(np.uint16)


def to_stored(x64: np.ndarray, dtype: str) -> np.ndarray:
    """float64 -> fp32 (RNE) -> stored dtype ("f32": float32, "bf16": uint16 bits)."""
    x32 = np.asarray(x64).astype(np.float32)
    if dtype == "f32":
        return x32
    if dtype == "bf16":
        return bf16_bits(x32)
    raise ValueError(dtype)


def haar(g: np.random.Generator, rows: int, k: int) -> np.ndarray:
    """rows x k matrix with orthonormal columns, Haar-distributed."""
    z = g.standard_normal((rows, k))
    q, r = np.linalg.qr(z)
    d = np.sign(np.diag(r))
    d[d == 0] = 1.0
    return q * d


def gauss(config: int, step: int, mat: int, m: int, n: int, std: float) -> np.ndarray:
    return std * stream(config, step, mat, ROLE_VALUES).standard_normal((m, n))


def lowrank_plus_noise(config: int, step: int, mat: int, m: int, n: int,
                       k: int, noise: float, signal_scale: float = 1.0) -> np.ndarray:
    """U diag(1/j, j=1..k) V^T * signal_scale + noise * Z (float64)."""
    k = min(k, m, n)
    u = haar(stream(config, 0, mat, ROLE_U), m, k)
    v = haar(stream(config, 0, mat, ROLE_V), n, k)
    s = signal_scale / np.arange(1, k + 1, dtype=np.float64)
    out = (u * s) @ v.T
    out += noise * stream(config, step, mat, ROLE_VALUES).standard_normal((m, n))
    return out


def geometric_spectrum(config: int, step: int, mat: int, m: int, n: int, k: int,
                       ratio: float) -> np.ndarray:
    """U diag(ratio^-j, j=0..k-1) V^T (float64): a steeply decaying spectrum
    whose power iterates are badly conditioned (exercises CholeskyQR2)."""
    k = min(k, m, n)
    u = haar(stream(config, step, mat, ROLE_U), m, k)
    v = haar(stream(config, step, mat, ROLE_V), n, k)
    return (u * ratio ** -np.arange(k, dtype=np.float64)) @ v.T


def zipf_rows(config: int, step: int, mat: int, vocab: int, hidden: int,
              tokens: int, exponent: float = 1.1, std: float = 1e-2) -> np.ndarray:
    """Embedding-gradient rows: `tokens` Zipf ids, each adding an N(0, std) row.

    Ids are drawn with replacement from P(k) ~ k^-exponent, k = 1..vocab, by
    inverse CDF; id k-1 is the row, so the most frequent token is row 0.
    Duplicate ids accumulate (scatter-add, as in an embedding backward).
    """
    w = np.arange(1, vocab + 1, dtype=np.float64) ** (-exponent)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    u = stream(config, step, mat, ROLE_TOKENS).random(tokens)
    ids = np.minimum(np.searchsorted(cdf, u, side="right"), vocab - 1)
    vals = std * stream(config, step, mat, ROLE_VALUES).standard_normal((tokens, hidden))
    uniq, inv = np.unique(ids, return_inverse=True)
    acc = np.zeros((uniq.size, hidden), dtype=np.float64)
    np.add.at(acc, inv, vals)
    out = np.zeros((vocab, hidden), dtype=np.float64)
    out[uniq] = acc
    return out


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: shapes, stored dtype, rank, iterations, steps."""

    key: int
    name: str
    shapes: tuple          # ((m, n), ...) one entry per matrix
    m_dtype: str           # "f32" or "bf16"
    rank: int
    iters: int
    steps: int
    kind: str              # recipe: gauss | lowrank | zipf | geom | gauss1024
    std: float = 1.0
    signal_rank: int = 0
    noise: float = 0.0
    tokens: int = 0
    signal_scale: float = 1.0
    notes: str = field(default="", compare=False)

    @property
    def elements(self) -> int:
        return sum(m * n for m, n in self.shapes)

    @property
    def m_bytes(self) -> int:
        return self.elements * (2 if self.m_dtype == "bf16" else 4)

    def matrix(self, step: int, j: int) -> np.ndarray:
        """Stored-dtype input matrix j of step `step`."""
        m, n = self.shapes[j]
        c = self.key
        if self.kind == "gauss1024":
            x = np.random.default_rng(0).standard_normal((m, n))
        elif self.kind == "gauss":
            x = gauss(c, step, j, m, n, self.std)
        elif self.kind == "lowrank":
            x = lowrank_plus_noise(c, step, j, m, n, self.signal_rank, self.noise,
                                   self.signal_scale)
        elif self.kind == "zipf":
            x = zipf_rows(c, step, j, m, n, self.tokens)
        elif self.kind == "geom":
            x = geometric_spectrum(c, step, j, m, n, self.signal_rank, self.noise)
        else:
            raise ValueError(self.kind)
        return to_stored(x, self.m_dtype)

    def q0(self, j: int) -> np.ndarray:
        """Initial warm-start factor Q (n x rank, fp32 N(0,1))."""
        n = self.shapes[j][1]
        if self.kind == "gauss1024":
            g = np.random.default_rng(1)
        else:
            g = stream(self.key, 0, j, ROLE_Q0)
        return g.standard_normal((n, self.rank)).astype(np.float32)

    def scaled(self, shapes, name: str | None = None, **kw) -> "Workload":
        """Same recipe at other shapes (parity cases the oracle finishes fast)."""
        d = dict(self.__dict__)
        d.update(shapes=tuple(tuple(s) for s in shapes), name=name or self.name + "_scaled")
        d.update(kw)
        d.pop("notes", None)
        return Workload(**d)


def _stage_shapes(layers: int = 9, h: int = 3072):
    per_layer = ((3 * h, h), (h, h), (4 * h, h), (h, 4 * h))
    return tuple(s for _ in range(layers) for s in per_layer)


WORKLOADS = {
    1: Workload(1, "gauss_1024", ((1024, 1024),), "f32", 4, 1, 1, "gauss1024"),
    2: Workload(2, "act_grad_8192x4096", ((8192, 4096),), "bf16", 16, 1, 8, "lowrank",
                signal_rank=32, noise=0.01),
    3: Workload(3, "stage_weights_h3072", _stage_shapes(), "f32", 32, 2, 2, "gauss",
                std=1e-3),
    4: Workload(4, "embedding_51200x3072", ((51200, 3072),), "f32", 64, 1, 2, "zipf",
                tokens=8192),
    5: Workload(5, "act_grad_4x16384x8192", ((16384, 8192),) * 4, "bf16", 128, 2, 2,
                "lowrank", signal_rank=256, noise=0.01),
}


def high_snr(w: Workload) -> Workload:
    """Diagnostic variant: signal scaled to unit-RMS entries over 1 % noise."""
    m, n = w.shapes[0]
    k = np.arange(1, w.signal_rank + 1, dtype=np.float64)
    alpha = float(np.sqrt(m * n) / np.linalg.norm(1.0 / k))
    return w.scaled(w.shapes, name=w.name + "_snr", signal_scale=alpha)

