"""The C-ABI library without a GPU: it loads, exports every declared symbol,
and rejects bad arguments on the host before launching anything."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2507_23035_amd import oasis

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "oasis.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(oasis.LIB_PATH):
        from paper_2507_23035_amd import build
        build.build()
    return oasis.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(oasis_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for fn in ("oasis_build_lut", "oasis_quantize_act", "oasis_lut_gemm",
               "oasis_outlier_compensate", "oasis_outlier_compensate_rows"):
        assert fn in names


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", oasis.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(l.split()[-1] for l in out.splitlines() if l.strip())
    for fn in declared_functions():
        assert fn in exported, fn
        assert hasattr(lib, fn)
    assert set(oasis.EXPORTS) <= exported


def test_status_strings(lib):
    assert lib.oasis_status_str(0) == b"ok"
    for s in range(-10, 0):
        assert lib.oasis_status_str(s) != b"unknown status"
    assert lib.oasis_version().startswith(b"oasis")


# Host buffers stand in for device pointers: every call below fails its
# argument check before anything touches them.
BUF = np.zeros(1 << 16, dtype=np.uint8)
P = BUF.ctypes.data          # 16-byte aligned by numpy for this size
MIS = P + 2                  # misaligned
A256 = (P + 255) & ~255      # 256-byte aligned, inside BUF (workspace checks)


def _cb(vals):
    return np.asarray(vals, dtype=np.float16).view(np.uint16)


def test_build_lut_errors(lib):
    asc = _cb(np.linspace(-1, 1, 16))
    cw = _cb(np.linspace(-1, 1, 16))
    assert lib.oasis_build_lut(None, 4, cw.ctypes.data, 4, P, None) == -1
    assert lib.oasis_build_lut(asc.ctypes.data, 5, cw.ctypes.data, 4, P, None) == -3
    assert lib.oasis_build_lut(asc.ctypes.data, 4, cw.ctypes.data, 0, P, None) == -3
    desc = _cb(np.linspace(1, -1, 16))
    assert lib.oasis_build_lut(desc.ctypes.data, 4, cw.ctypes.data, 4, P, None) == -5
    dup = _cb([0.0, 0.5, 0.5, 1.0])
    assert lib.oasis_build_lut(dup.ctypes.data, 2, cw.ctypes.data, 4, P, None) == -5
    bad = _cb([0.0, np.inf])
    assert lib.oasis_build_lut(bad.ctypes.data, 1, cw.ctypes.data, 4, P, None) == -5
    nanw = _cb([0.0, np.nan])
    assert lib.oasis_build_lut(asc.ctypes.data, 4, nanw.ctypes.data, 1, P, None) == -5
    assert lib.oasis_build_lut(asc.ctypes.data, 4, cw.ctypes.data, 4, MIS, None) == -6


def test_quantize_errors(lib):
    q = lib.oasis_quantize_act
    assert q(P, 4, 12, P, 4, 1, 0, P, P, P, P, P, None) == -2        # d_in % 8
    assert q(P, -1, 16, P, 4, 1, 0, P, P, P, P, P, None) == -2
    assert q(P, 4, 16, P, 0, 1, 0, P, P, P, P, P, None) == -3
    assert q(P, 4, 16, P, 4, 17, 0, P, P, P, P, P, None) == -4
    assert q(P, 4, 16, P, 4, -1, 0, P, P, P, P, P, None) == -4
    assert q(P, 4, 16, P, 4, 1, 3, P, P, P, P, P, None) == -7       # modes 0..2
    assert q(P, 4, 65544, P, 4, 1, 0, P, P, P, P, P, None) == -9
    assert q(P, 4, 32768, P, 4, 32768, 0, P, P, P, P, P, None) == -9   # LDS budget
    assert q(None, 4, 16, P, 4, 1, 0, P, P, P, P, P, None) == -1
    assert q(P, 4, 16, P, 4, 1, 0, P, P, None, P, P, None) == -1
    assert q(MIS, 4, 16, P, 4, 1, 0, P, P, P, P, P, None) == -6
    assert q(P, 0, 16, None, 4, 1, 0, None, None, None, None, None, None) == 0   # empty


def test_build_lut_quantize_errors(lib):
    f = lib.oasis_build_lut_quantize_act
    ca = _cb(np.linspace(-1, 1, 16))
    cw = _cb(np.linspace(-1, 1, 16))
    A, W = ca.ctypes.data, cw.ctypes.data
    assert f(None, 4, W, 4, P, P, 4, 16, 1, 0, P, P, P, P, P, None) == -1
    assert f(A, 4, W, 4, None, P, 4, 16, 1, 0, P, P, P, P, P, None) == -1
    assert f(A, 4, W, 4, P, P, 4, 12, 1, 0, P, P, P, P, P, None) == -2
    assert f(A, 5, W, 4, P, P, 4, 16, 1, 0, P, P, P, P, P, None) == -3
    assert f(A, 4, W, 4, P, P, 4, 16, 17, 0, P, P, P, P, P, None) == -4
    desc = _cb(np.linspace(1, -1, 16))
    assert f(desc.ctypes.data, 4, W, 4, P, P, 4, 16, 1, 0, P, P, P, P, P, None) == -5
    assert f(A, 4, W, 4, MIS, P, 4, 16, 1, 0, P, P, P, P, P, None) == -6
    assert f(A, 4, W, 4, P, MIS, 4, 16, 1, 0, P, P, P, P, P, None) == -6
    assert f(A, 4, W, 4, P, P, 4, 16, 1, 3, P, P, P, P, P, None) == -7
    assert f(A, 4, W, 4, P, P, 4, 65544, 1, 0, P, P, P, P, P, None) == -9
    assert f(A, 4, W, 4, P, None, 4, 16, 1, 0, P, P, P, P, P, None) == -1


def test_quantize_static_errors(lib):
    f = lib.oasis_quantize_act_static
    f.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                  ctypes.c_int, ctypes.c_int, ctypes.c_float, ctypes.c_float] + \
        [ctypes.c_void_p] * 5 + [ctypes.c_void_p]
    assert f(P, 4, 12, P, 4, 1, 0, 2.0, -2.0, P, P, P, P, P, None) == -2
    assert f(P, 4, 16, P, 5, 1, 0, 2.0, -2.0, P, P, P, P, P, None) == -3
    assert f(P, 4, 16, P, 4, 17, 0, 2.0, -2.0, P, P, P, P, P, None) == -4
    assert f(P, 4, 16, P, 4, 1, 0, -2.0, 2.0, P, P, P, P, P, None) == -7     # lo >= hi
    assert f(P, 4, 16, P, 4, 1, 3, 2.0, -2.0, P, P, P, P, P, None) == -7     # mode
    assert f(P, 4, 16, P, 4, 1, 0, float("nan"), -2.0, P, P, P, P, P, None) == -7
    assert f(None, 4, 16, P, 4, 1, 0, 2.0, -2.0, P, P, P, P, P, None) == -1
    assert f(MIS, 4, 16, P, 4, 1, 0, 2.0, -2.0, P, P, P, P, P, None) == -6
    assert f(P, 0, 16, None, 4, 1, 0, 2.0, -2.0, None, None, None, None, None, None) == 0


def test_build_lut_quantize_static_errors(lib):
    f = lib.oasis_build_lut_quantize_act_static
    ca = _cb(np.linspace(-1, 1, 16))
    cw = _cb(np.linspace(-1, 1, 16))
    A, W = ca.ctypes.data, cw.ctypes.data
    assert f(None, 4, W, 4, P, P, 4, 16, 1, 0, 2.0, -2.0, P, P, P, P, P, None) == -1
    assert f(A, 4, W, 4, P, P, 4, 12, 1, 0, 2.0, -2.0, P, P, P, P, P, None) == -2
    assert f(A, 4, W, 5, P, P, 4, 16, 1, 0, 2.0, -2.0, P, P, P, P, P, None) == -3
    assert f(A, 4, W, 4, P, P, 4, 16, 17, 0, 2.0, -2.0, P, P, P, P, P, None) == -4
    assert f(A, 4, W, 4, P, P, 4, 16, 1, 0, -2.0, 2.0, P, P, P, P, P, None) == -7   # lo >= hi
    assert f(A, 4, W, 4, P, P, 4, 16, 1, 3, 2.0, -2.0, P, P, P, P, P, None) == -7
    assert f(A, 4, W, 4, MIS, P, 4, 16, 1, 0, 2.0, -2.0, P, P, P, P, P, None) == -6


def test_cluster_and_detect_errors(lib):
    c = lib.oasis_cluster_act
    assert c(P, 4, 12, P, 4, 0, P, P, None) == -2
    assert c(P, 4, 16, P, 5, 0, P, P, None) == -3
    assert c(P, 4, 16, P, 4, 3, P, P, None) == -7
    assert c(P, 4, 16, P, 4, 2, P, P, None) == -7   # the inlier scale needs the lists
    assert c(None, 4, 16, P, 4, 0, P, P, None) == -1
    assert c(P, 4, 16, P, 4, 0, MIS, P, None) == -6
    d = lib.oasis_detect_outliers
    assert d(P, 4, 16, P, 4, 17, 0, P, P, P, None) == -4
    assert d(P, 4, 16, P, 4, 2, 0, None, P, P, None) == -1
    assert d(P, 4, 16, P, 4, 0, 0, None, None, None, None) == 0   # k = 0: nothing to do
    assert d(P, 4, 65544, P, 4, 1, 0, P, P, P, None) == -9
    assert d(P, 4, 16, P, 4, 1, 2, P, P, P, None) == -7


def test_fused_gemm_errors(lib):
    f = lib.oasis_lut_gemm_compensated
    assert f(P, P, 4, 20, P, P, 8, P, 4, 4, P, P, P, 1, P, 0, None) == -2
    assert f(P, P, 4, 16, P, P, 8, P, 4, 4, P, P, P, 17, P, 0, None) == -4
    assert f(P, P, 4, 16, P, P, 8, P, 4, 4, None, P, P, 1, P, 0, None) == -1
    assert f(P, P, 4, 16, P, P, 8, P, 4, 4, P, P, MIS, 1, P, 0, None) == -6


def test_gemm_errors(lib):
    g = lib.oasis_lut_gemm
    assert g(P, P, 4, 20, P, P, 8, P, 4, 4, 1, P, 0, None) == -2
    assert g(P, P, 4, 16, P, P, -8, P, 4, 4, 1, P, 0, None) == -2
    assert g(P, P, 4, 16, P, P, 8, P, 4, 9, 1, P, 0, None) == -3
    assert g(P, P, 4, 16, P, P, 8, P, 4, 4, 2, P, 0, None) == -7
    assert g(None, P, 4, 16, P, P, 8, P, 4, 4, 1, P, 0, None) == -1
    assert g(P, P, 4, 16, MIS, P, 8, P, 4, 4, 1, P, 0, None) == -6
    assert g(P, P, 0, 16, P, P, 8, P, 4, 4, 1, P, 0, None) == 0      # empty


def test_compensate_errors(lib):
    c = lib.oasis_outlier_compensate
    assert c(P, P, P, 4, 3, P, P, 4, P, 20, 8, P, 1, None) == -2
    assert c(P, P, P, 4, 17, P, P, 4, P, 16, 8, P, 1, None) == -4
    assert c(P, P, P, 4, 3, P, P, 5, P, 16, 8, P, 1, None) == -3
    assert c(None, P, P, 4, 3, P, P, 4, P, 16, 8, P, 1, None) == -1
    assert c(P, P, P, 4, 3, P, P, 4, P, 16, 8, MIS, 1, None) == -6
    assert c(P, P, P, 0, 3, P, P, 4, P, 16, 8, P, 1, None) == 0
    # codes of 2^31 bytes (d_in / 8 * d_out words): 32-bit buffer offsets
    assert c(P, P, P, 100, 3, P, P, 4, P, 65536, 65536, P, 1, None) == -9


def test_compensate_rows_errors(lib):
    c = lib.oasis_outlier_compensate_rows
    assert c(P, P, P, 4, 3, P, P, 4, P, 20, 8, P, 1, None) == -2
    assert c(P, P, P, 4, 17, P, P, 4, P, 16, 8, P, 1, None) == -4
    assert c(P, P, P, 4, 3, P, P, 5, P, 16, 8, P, 1, None) == -3
    assert c(None, P, P, 4, 3, P, P, 4, P, 16, 8, P, 1, None) == -1
    assert c(P, P, P, 4, 3, P, P, 4, P, 16, 8, MIS, 1, None) == -6
    assert c(P, P, P, 4, 3, P, P, 4, P, 65536, 65536, P, 1, None) == -9  # 2^31 bytes of codes
    assert c(P, P, P, 0, 3, P, P, 4, P, 16, 8, P, 1, None) == 0


def test_pack_weight_rows_matches_oracle_packing():
    from oracle import oasis_oracle as O
    rng = np.random.default_rng(6)
    for shape in [(24, 13), (8, 16), (5, 1), (3, 40)]:
        w = rng.integers(0, 16, shape).astype(np.uint8)
        got = oasis.pack_weight_rows(w)
        assert got.shape == (shape[0], (shape[1] + 7) // 8)
        assert np.array_equal(got, O.pack_weight_rows(w))
        # every nibble back in place, zeros past the last column
        cols = np.arange(8 * got.shape[1])
        nib = (got[:, cols // 8] >> (4 * (cols % 8)).astype(np.uint32)) & 15
        assert np.array_equal(nib[:, :shape[1]], w) and not nib[:, shape[1]:].any()


def test_fused_rows_errors(lib):
    g = lib.oasis_lut_gemm_compensated_rows
    assert g(P, P, 4, 12, P, P, P, 8, P, 4, 4, P, P, P, 2, P, 0, None) == -2
    assert g(P, P, 4, 16, P, None, P, 8, P, 4, 4, P, P, P, 2, P, 0, None) == -1   # rows needed
    assert g(P, P, 4, 16, P, MIS, P, 8, P, 4, 4, P, P, P, 2, P, 0, None) == -6
    assert g(P, P, 4, 16, P, P, P, 8, P, 4, 4, P, P, P, 17, P, 0, None) == -4


def test_percol_errors(lib):
    g = lib.oasis_lut_gemm_compensated_percol
    assert g(P, P, 4, 12, P, P, 8, P, P, 4, 4, P, P, P, 2, P, 0, None) == -2
    assert g(P, P, 4, 16, P, P, 8, P, None, 4, 4, P, P, P, 2, P, 0, None) == -1
    assert g(P, P, 4, 16, P, P, 8, P, P + 1, 4, 4, P, P, P, 2, P, 0, None) == -6
    assert g(P, P, 4, 16, P, P, 8, P, P + 2, 4, 4, P, P, P, 2, P, 0, None) == -6  # 16 B
    assert g(P, P, 33, 16, P, P, 8, P, P, 4, 4, P, P, P, 17, P, 0, None) == -4  # any n
    assert g(P, P, 4, 16, P, P, 8, P, P, 4, 4, P, P, P, 17, P, 0, None) == -4


def test_pack_weight_indices_matches_oracle_packing():
    from oracle import oasis_oracle as O
    rng = np.random.default_rng(5)
    w = rng.integers(0, 16, (24, 13)).astype(np.uint8)
    assert np.array_equal(oasis.pack_weight_indices(w), O.pack_weight_indices(w))
    with pytest.raises(oasis.OasisError):
        oasis.pack_weight_indices(np.zeros((12, 4), dtype=np.uint8))


def test_binding_refuses_host_tensors():
    """The wrappers pass raw addresses: a tensor that is not on the GPU (or,
    on a GPU, not contiguous or of the wrong element type) is refused before
    any call."""
    torch = pytest.importorskip("torch")
    t = torch.zeros(16, dtype=torch.float32)
    with pytest.raises(ValueError, match="CUDA"):
        oasis._ptr(t, "f32")
    assert oasis._ptr(None, "f32") is None


def test_compensate_split_errors(lib):
    c = lib.oasis_outlier_compensate_split
    c.argtypes = [ctypes.c_void_p] * 3 + [ctypes.c_int] * 2 + [ctypes.c_void_p] * 3 + \
        [ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
         ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    wsz = lib.oasis_outlier_compensate_split_workspace
    wsz.restype = ctypes.c_size_t
    wsz.argtypes = [ctypes.c_int] * 4
    need = wsz(4, 16, 8, 3)
    assert need > 0 and wsz(4, 16, 8, 3) == need and wsz(-1, 16, 8, 3) == 0
    ok = (P, P, P, 4, 3, P, P, P, 4, P, 16, 8, P, 1)
    assert c(P, P, P, 4, 3, P, P, P, 4, P, 20, 8, P, 1, P, need, None) == -2
    assert c(P, P, P, 4, 17, P, P, P, 4, P, 16, 8, P, 1, P, need, None) == -4
    assert c(P, P, P, 4, 3, P, P, P, 5, P, 16, 8, P, 1, P, need, None) == -3
    assert c(P, P, P, 4, 3, P, None, P, 4, P, 16, 8, P, 1, P, need, None) == -1   # idx_wr
    assert c(P, P, P, 4, 3, MIS, P, P, 4, P, 16, 8, P, 1, P, need, None) == -6
    assert c(*ok, None, need, None) == -10                       # no workspace
    assert c(*ok, A256 + 16, need, None) == -10                  # not 256-byte aligned
    assert c(*ok, A256, 64, None) == -10                         # too small (need > 64)
    assert c(P, P, P, 4, 3, P, P, P, 4, P, 65536, 65536, P, 1, P, 1 << 40, None) == -9
    assert c(P, P, P, 0, 3, P, P, P, 4, P, 16, 8, P, 1, None, 0, None) == 0   # no tokens


def test_gemm_compensated_split_errors(lib):
    g = lib.oasis_lut_gemm_compensated_split
    g.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                  ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                  ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_size_t,
                  ctypes.c_void_p]
    assert g(P, P, 40, 12, P, P, P, 8, P, 4, 4, P, P, P, 2, P, 0, P, 1 << 20, None) == -2
    assert g(P, P, 40, 64, P, P, P, 8, P, 4, 5, P, P, P, 2, P, 0, P, 1 << 20, None) == -3
    assert g(P, P, 40, 64, P, P, P, 8, P, 4, 4, P, P, P, 65, P, 0, P, 1 << 20, None) == -4
    assert g(P, P, 40, 64, P, None, P, 8, P, 4, 4, P, P, P, 2, P, 0, P, 1 << 20, None) == -1
    assert g(P, P, 40, 64, MIS, P, P, 8, P, 4, 4, P, P, P, 2, P, 0, P, 1 << 20, None) == -6
    # many tokens with lists: the workspace is required, 256-byte aligned, large enough
    assert g(P, P, 40, 64, P, P, P, 8, P, 4, 4, P, P, P, 2, P, 0, None, 1 << 20, None) == -10
    assert g(P, P, 40, 64, P, P, P, 8, P, 4, 4, P, P, P, 2, P, 0, A256 + 16, 1 << 20, None) == -10
    assert g(P, P, 40, 64, P, P, P, 8, P, 4, 4, P, P, P, 2, P, 0, A256, 64, None) == -10
    assert g(P, P, 0, 64, P, P, P, 8, P, 4, 4, P, P, P, 2, P, 0, None, 0, None) == 0
