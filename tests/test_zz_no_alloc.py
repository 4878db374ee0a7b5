"""The no-allocation entry point against the workspace one, through the C ABI:
two calls in a row (the second smaller, over the scratch the first left),
each within the parity bound of the other; and the size limit."""
import ctypes

import numpy as np
import pytest

from paper_2507_23035_amd import oasis, synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

RTOL, ATOL, ATOL_RMS = 1e-3, 1e-2, 1e-4


def close(y, ref):
    y = y.cpu().numpy().astype(np.float64)
    ref = ref.cpu().numpy().astype(np.float64)
    rms = np.sqrt(np.mean(ref * ref, axis=-1, keepdims=True))
    bound = np.maximum(RTOL * np.abs(ref), np.minimum(ATOL, ATOL_RMS * rms))
    return bool(np.all(np.abs(y - ref) <= bound))


def run_case(lib, n, d_in, d_out, k, seed):
    print(f"no-alloc case n={n} d_in={d_in} d_out={d_out} k={k} seed={seed}", flush=True)
    L = synth.make_layer(synth.custom(n, d_in, d_out, k, seed=seed))
    dev = torch.device("cuda:0")
    s = L.spec
    x = torch.from_numpy(L.x.view(np.int16).copy()).to(dev)
    lut = oasis.build_lut(L.cb_a, s.b_a, L.cb_w, s.b_w)
    idx_w = torch.from_numpy(oasis.pack_weight_indices(L.w_idx).view(np.int32)).to(dev)
    idx_wr = torch.from_numpy(oasis.pack_weight_rows(L.w_idx).view(np.int32)).to(dev)
    s_w = torch.from_numpy(L.s_w).to(dev)
    q = oasis.quantize_act(x, lut, s.b_a, k)
    ref = oasis.lut_gemm_compensated_split(q["idx_act"], q["act_scale"], idx_w, idx_wr, s_w, lut,
                                           s.b_a, s.b_w, q["max_idx"], q["min_idx"],
                                           q["residual"])
    y = torch.full((n, d_out), float("nan"), dtype=torch.float32, device=dev)
    st = lib.oasis_lut_gemm_compensated_split_noalloc(
        q["idx_act"].data_ptr(), q["act_scale"].data_ptr(), n, d_in, idx_w.data_ptr(),
        idx_wr.data_ptr(), s_w.data_ptr(), d_out, lut.data_ptr(), s.b_a, s.b_w,
        q["max_idx"].data_ptr(), q["min_idx"].data_ptr(), q["residual"].data_ptr(), k,
        y.data_ptr(), 0, torch.cuda.current_stream().cuda_stream)
    assert st == 0, lib.oasis_status_str(st)
    torch.cuda.synchronize()
    assert close(y, ref), "no-alloc result differs from the workspace entry point"
    # accumulate into a preset y
    y.fill_(0.25)
    st = lib.oasis_lut_gemm_compensated_split_noalloc(
        q["idx_act"].data_ptr(), q["act_scale"].data_ptr(), n, d_in, idx_w.data_ptr(),
        idx_wr.data_ptr(), s_w.data_ptr(), d_out, lut.data_ptr(), s.b_a, s.b_w,
        q["max_idx"].data_ptr(), q["min_idx"].data_ptr(), q["residual"].data_ptr(), k,
        y.data_ptr(), 1, torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    assert close(y - 0.25, ref)


def test_no_alloc_matches_workspace_entry_point():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib = oasis.load()
    run_case(lib, 300, 1024, 520, 24, 71)   # heavy channels inside the GEMM
    run_case(lib, 70, 512, 136, 8, 72)      # smaller, over the scratch the first call left
    run_case(lib, 40, 264, 100, 5, 73)      # d_in not a multiple of 64: split, then the GEMM


def test_no_alloc_rejects_sizes_beyond_its_scratch():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib = oasis.load()
    need = lib.oasis_outlier_compensate_split_workspace(40000, 8192, 28672, 64)
    assert need > 32 << 20
    buf = torch.zeros(1 << 16, dtype=torch.uint8, device="cuda")
    p = buf.data_ptr()
    # rejected on the host before anything is launched (no pointer is read)
    st = lib.oasis_lut_gemm_compensated_split_noalloc(p, p, 40000, 8192, p, p, p, 28672, p, 4, 4,
                                                      p, p, p, 64, p, 0, None)
    assert st == -9
