"""Host-side checks of the C ABI: it loads, exports what the header declares,
and rejects bad arguments before touching the device.  No kernel runs here:
every call below fails validation on the host and returns an error code."""

import ctypes
import os

import pytest

from paper_2301_09830_amd import build as buildmod
from paper_2301_09830_amd import optcc


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(buildmod.LIB):
        buildmod.build()
    return optcc.lib()


def test_exports_every_declared_symbol(L):
    names = optcc.header_symbols()
    assert "occ_step" in names and "occ_step_batched" in names and len(names) >= 12
    for name in names:
        assert hasattr(L, name), name
        assert name in optcc._SIGS, f"binding lacks {name}"


def test_abi_version_and_status_strings(L):
    assert optcc.occ_abi_version() == 2
    for code in range(11):
        assert optcc.occ_status_str(code)
    assert "unknown" in optcc.occ_status_str(99)


def _mat(rows=64, cols=32, ld=None, dtype=optcc.OCC_F32, base=1 << 20):
    a = optcc.occ_mat_t()
    a.M = base
    a.m_dtype = dtype
    a.rows, a.cols = rows, cols
    a.ldm = cols if ld is None else ld
    a.err = base + (1 << 24)
    a.lde = cols
    a.P = base + (2 << 24)
    a.Q = base + (3 << 24)
    a.M_hat = base + (4 << 24)
    a.ldh = cols
    return a


def _step(L, mat, rank=4, iters=1, flags=0, ws=1 << 32, ws_bytes=1 << 30):
    return L.occ_step(ctypes.byref(mat), rank, iters, flags, ws, ws_bytes, None)


def test_argument_errors_are_host_side(L):
    assert _step(L, _mat(), rank=0) == 3           # OCC_E_RANK
    assert _step(L, _mat(), rank=33) == 3          # rank > cols
    assert _step(L, _mat(rows=200, cols=200), rank=129) == 3
    assert _step(L, _mat(), iters=0) == 4          # OCC_E_ITERS
    assert _step(L, _mat(), iters=65) == 4
    assert _step(L, _mat(ld=16)) == 2              # ld < cols: OCC_E_SHAPE
    assert _step(L, _mat(rows=0)) == 2
    assert _step(L, _mat(dtype=7)) == 5            # OCC_E_DTYPE
    m = _mat(); m.P = 0
    assert _step(L, m) == 1                        # OCC_E_NULL
    m = _mat(); m.M_hat = 0
    assert _step(L, m) == 1                        # M_hat needed unless OCC_NO_MHAT
    m = _mat(); m.err = m.err + 2
    assert _step(L, m) == 6                        # OCC_E_ALIGN
    m = _mat(); m.Q = m.P + 16
    assert _step(L, m) == 7                        # OCC_E_ALIAS
    assert _step(L, _mat(), ws=0) == 8             # OCC_E_WORKSPACE
    assert _step(L, _mat(), ws=(1 << 32) + 4) == 8
    assert _step(L, _mat(), ws_bytes=100) == 8
    assert _step(L, _mat(), flags=8) == 10         # OCC_E_FLAGS
    assert L.occ_step(None, 4, 1, 0, 1 << 32, 1 << 30, None) == 1


def test_batched_errors(L):
    arr = (optcc.occ_mat_t * 2)(_mat(), _mat(base=1 << 30))
    assert L.occ_step_batched(arr, 0, 4, 1, 0, 1 << 40, 1 << 30, None) == 2
    arr[1].m_dtype = optcc.OCC_BF16
    assert L.occ_step_batched(arr, 2, 4, 1, 0, 1 << 40, 1 << 30, None) == 5
    arr = (optcc.occ_mat_t * 2)(_mat(), _mat())     # same buffers twice: overlap
    assert L.occ_step_batched(arr, 2, 4, 1, 0, 1 << 40, 1 << 30, None) == 7


def test_other_entry_points_validate(L):
    # decompress: rank > n
    assert L.occ_decompress(1 << 20, 1 << 21, 10, 3, 4, 1 << 22, 3, None) == 3
    # decompress: output overlaps P
    assert L.occ_decompress(1 << 20, 1 << 24, 10, 8, 4, (1 << 20) + 8, 8, None) == 7
    # decompress_ex: unknown flag bit, bf16 output misaligned for its element size
    assert L.occ_decompress_ex(1 << 20, 1 << 24, 10, 8, 4, 4, 1 << 26, 8, None) == 10
    assert L.occ_decompress_ex(1 << 20, 1 << 24, 10, 8, 4, 2, (1 << 26) + 1, 8, None) == 6
    # decompress_ex: a bf16 M_hat of 10 x 8 at ld 8 spans 160 bytes; a P 100
    # bytes after its start overlaps it
    assert L.occ_decompress_ex((1 << 26) + 100, 1 << 24, 10, 8, 4, 2, 1 << 26, 8, None) == 7
    # err_update: err_new overlapping M
    assert L.occ_err_update(1 << 20, 0, 4, 4, 4, 1 << 24, 4, 1 << 26, 4, (1 << 20) + 4,
                            None) == 7
    # err_update: unknown dtype, leading dimension below cols
    assert L.occ_err_update(1 << 20, 3, 4, 4, 4, 1 << 24, 4, 1 << 26, 4, 1 << 24, None) == 5
    assert L.occ_err_update(1 << 20, 0, 4, 4, 4, 1 << 24, 3, 1 << 26, 4, 1 << 24, None) == 2
    # compress: missing workspace
    assert L.occ_compress(1 << 20, 0, 16, 16, 16, None, 0, 1 << 24, 1 << 26, 2, 1, None, 0,
                          None) == 8
    assert L.occ_workspace_init(None, 1024, None) == 1
    flags = ctypes.c_uint32()
    assert L.occ_get_flags(None, ctypes.byref(flags), 0, None) == 1


def test_compress_workspace_follows_dtype(L):
    """The compress-only workspace is sized for the M dtype it will run on
    (the large-rank tiling depends on it); an unknown dtype gives 0."""
    for dt in (optcc.OCC_F32, optcc.OCC_BF16):
        a = L.occ_compress_workspace_bytes(8192, 4096, dt, 128, 2)
        arr = (optcc.occ_mat_t * 1)()
        arr[0].rows, arr[0].cols, arr[0].ldm, arr[0].m_dtype = 8192, 4096, 4096, dt
        assert a > 0 and a == L.occ_workspace_bytes(arr, 1, 128, 2)
    assert L.occ_compress_workspace_bytes(8192, 4096, 5, 16, 1) == 0


def test_workspace_size_is_deterministic_and_grows(L):
    a = optcc.occ_workspace_bytes([(8192, 4096)], 16, 1)
    b = optcc.occ_workspace_bytes([(8192, 4096)], 16, 1)
    c = optcc.occ_workspace_bytes([(8192, 4096)] * 2, 16, 1)
    assert a == b and a > 0 and c > 2 * a - 4096
    assert a % 256 == 0
    assert optcc.occ_workspace_bytes([(8192, 4096)], 0, 1) == 0     # invalid rank -> 0
    # config sizes stay modest relative to the 288 GB HBM
    w5 = optcc.occ_workspace_bytes([(16384, 8192)] * 4, 128, 2)
    assert w5 < 2 << 30


def test_rows_step_validates_on_the_host(L):
    a = _mat(rows=64, cols=32)
    ws, nb = 1 << 32, 1 << 30
    rows = 1 << 36
    # fewer listed rows than the rank, more rows than the matrix, negative count
    assert L.occ_step_rows(ctypes.byref(a), rows, 3, 4, 1, 0, ws, nb, None) == 3
    assert L.occ_step_rows(ctypes.byref(a), rows, 65, 4, 1, 0, ws, nb, None) == 2
    assert L.occ_step_rows(ctypes.byref(a), rows, -1, 4, 1, 0, ws, nb, None) == 2
    # missing row list, unaligned row list, list overlapping err
    assert L.occ_step_rows(ctypes.byref(a), None, 10, 4, 1, 0, ws, nb, None) == 1
    assert L.occ_step_rows(ctypes.byref(a), rows + 2, 10, 4, 1, 0, ws, nb, None) == 6
    assert L.occ_step_rows(ctypes.byref(a), a.err + 64, 10, 4, 1, 0, ws, nb, None) == 7
    # workspace too small for the listed rows, unknown flag
    need = L.occ_step_rows_workspace_bytes(10, 32, 0, 4, 1)
    assert need > 0
    assert L.occ_step_rows(ctypes.byref(a), rows, 10, 4, 1, 0, ws, need - 256, None) == 8
    assert L.occ_step_rows(ctypes.byref(a), rows, 10, 4, 1, 2, ws, nb, None) == 10
    assert L.occ_step_rows(None, rows, 10, 4, 1, 0, ws, nb, None) == 1


def test_rows_workspace_grows_with_the_list(L):
    a = L.occ_step_rows_workspace_bytes(100, 3072, 0, 64, 1)
    b = L.occ_step_rows_workspace_bytes(2500, 3072, 0, 64, 1)
    dense = optcc.occ_workspace_bytes([(51200, 3072)], 64, 1)
    assert 0 < a < b < dense
    assert L.occ_step_rows_workspace_bytes(0, 3072, 0, 64, 1) == 256
    assert L.occ_step_rows_workspace_bytes(10, 3072, 0, 64, 1) == 0     # rows < rank


def test_noalloc_rejects_calls_beyond_its_static_workspace(L):
    """The 36 stage-weight matrices need about 386 MiB of workspace, beyond the
    64 MiB static array: rejected on the host before any device call."""
    from workloads import WORKLOADS
    shapes = WORKLOADS[3].shapes
    arr = (optcc.occ_mat_t * len(shapes))()
    for j, (m, n) in enumerate(shapes):
        arr[j] = _mat(rows=m, cols=n, base=(j + 1) << 34)
    assert optcc.occ_workspace_bytes(list(shapes), 32, 2) > optcc.OCC_NOALLOC_MAX_BYTES
    assert L.occ_step_batched_noalloc(arr, len(shapes), 32, 2, 0, None, None) == 8
    assert L.occ_step_batched_noalloc(arr, len(shapes), 32, 2, 4, None, None) == 10
