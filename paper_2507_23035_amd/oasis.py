"""ctypes binding of liboasis.so, the C ABI of the OASIS hot path.

Argument marshalling only: every step runs in the library's HIP kernels.
torch supplies device memory and the current HIP stream.  There is no
fallback: if the library is missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboasis.so")

SCALE_ABSMAX = 0
SCALE_NONE = 1
SCALE_INLIER = 2
ALGO_LUT = 0
ALGO_MFMA = 1
LUT_BLOCK_BYTES = 256 * 4 + 16 * 2 + 16 * 2

EXPORTS = ("oasis_status_str", "oasis_version", "oasis_build_lut", "oasis_quantize_act",
           "oasis_cluster_act", "oasis_detect_outliers",
           "oasis_lut_gemm", "oasis_outlier_compensate", "oasis_outlier_compensate_rows",
           "oasis_lut_gemm_compensated", "oasis_pack_weight_indices", "oasis_pack_weight_rows",
           "oasis_build_lut_quantize_act", "oasis_quantize_act_static",
           "oasis_build_lut_quantize_act_static", "oasis_lut_gemm_compensated_percol",
           "oasis_lut_gemm_compensated_rows", "oasis_outlier_compensate_split",
           "oasis_outlier_compensate_split_workspace", "oasis_lut_gemm_compensated_split",
           "oasis_lut_gemm_compensated_split_noalloc")


class OasisError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn} failed with status {status}: {msg}")
        self.status = status


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load liboasis.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with paper_2507_23035_amd.build.build()")
    lib = ctypes.CDLL(path)
    P, I = ctypes.c_void_p, ctypes.c_int
    lib.oasis_status_str.restype = ctypes.c_char_p
    lib.oasis_status_str.argtypes = [I]
    lib.oasis_version.restype = ctypes.c_char_p
    lib.oasis_version.argtypes = []
    lib.oasis_build_lut.restype = I
    lib.oasis_build_lut.argtypes = [P, I, P, I, P, P]
    lib.oasis_quantize_act.restype = I
    lib.oasis_quantize_act.argtypes = [P, I, I, P, I, I, I, P, P, P, P, P, P]
    F = ctypes.c_float
    lib.oasis_quantize_act_static.restype = I
    lib.oasis_quantize_act_static.argtypes = [P, I, I, P, I, I, I, F, F, P, P, P, P, P, P]
    lib.oasis_build_lut_quantize_act_static.restype = I
    lib.oasis_build_lut_quantize_act_static.argtypes = [P, I, P, I, P, P, I, I, I, I, F, F, P, P,
                                                        P, P, P, P]
    lib.oasis_build_lut_quantize_act.restype = I
    lib.oasis_build_lut_quantize_act.argtypes = [P, I, P, I, P, P, I, I, I, I, P, P, P, P, P, P]
    lib.oasis_cluster_act.restype = I
    lib.oasis_cluster_act.argtypes = [P, I, I, P, I, I, P, P, P]
    lib.oasis_detect_outliers.restype = I
    lib.oasis_detect_outliers.argtypes = [P, I, I, P, I, I, I, P, P, P, P]
    lib.oasis_lut_gemm.restype = I
    lib.oasis_lut_gemm.argtypes = [P, P, I, I, P, P, I, P, I, I, I, P, I, P]
    lib.oasis_outlier_compensate.restype = I
    lib.oasis_outlier_compensate.argtypes = [P, P, P, I, I, P, P, I, P, I, I, P, I, P]
    lib.oasis_lut_gemm_compensated.restype = I
    lib.oasis_lut_gemm_compensated.argtypes = [P, P, I, I, P, P, I, P, I, I, P, P, P, I, P, I, P]
    lib.oasis_lut_gemm_compensated_rows.restype = I
    lib.oasis_lut_gemm_compensated_rows.argtypes = [P, P, I, I, P, P, P, I, P, I, I, P, P, P, I,
                                                    P, I, P]
    lib.oasis_lut_gemm_compensated_percol.restype = I
    lib.oasis_lut_gemm_compensated_percol.argtypes = [P, P, I, I, P, P, I, P, P, I, I, P, P, P, I,
                                                      P, I, P]
    lib.oasis_outlier_compensate_rows.restype = I
    lib.oasis_outlier_compensate_rows.argtypes = [P, P, P, I, I, P, P, I, P, I, I, P, I, P]
    S = ctypes.c_size_t
    lib.oasis_outlier_compensate_split_workspace.restype = S
    lib.oasis_outlier_compensate_split_workspace.argtypes = [I, I, I, I]
    lib.oasis_outlier_compensate_split.restype = I
    lib.oasis_outlier_compensate_split.argtypes = [P, P, P, I, I, P, P, P, I, P, I, I, P, I, P, S,
                                                   P]
    lib.oasis_lut_gemm_compensated_split.restype = I
    lib.oasis_lut_gemm_compensated_split.argtypes = [P, P, I, I, P, P, P, I, P, I, I, P, P, P, I,
                                                     P, I, P, S, P]
    lib.oasis_lut_gemm_compensated_split_noalloc.restype = I
    lib.oasis_lut_gemm_compensated_split_noalloc.argtypes = [P, P, I, I, P, P, P, I, P, I, I, P,
                                                             P, P, I, P, I, P]
    lib.oasis_pack_weight_indices.restype = I
    lib.oasis_pack_weight_indices.argtypes = [P, I, I, P]
    lib.oasis_pack_weight_rows.restype = I
    lib.oasis_pack_weight_rows.argtypes = [P, I, I, P]
    _lib = lib
    return lib


def _check(fn: str, status: int) -> None:
    if status != 0:
        raise OasisError(fn, status, load().oasis_status_str(status).decode())


# element kinds of the tensors the calls take: fp16 values travel as their
# bit patterns, so float16 and int16 tensors both qualify
_KINDS = {
    "u8": ("uint8", "int8"),
    "f16": ("float16", "int16", "uint16"),
    "i32": ("int32", "uint32"),
    "f32": ("float32",),
}


def _ptr(t, kind: Optional[str] = None) -> Optional[int]:
    """Device address of a tensor the library reads or writes as packed
    row-major memory: it must be a contiguous CUDA tensor of the right element
    kind (a strided view would be read as if it were packed)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"expected a CUDA tensor, got one on {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"expected a contiguous tensor, got strides {tuple(t.stride())}")
    if kind is not None and str(t.dtype).split(".")[-1] not in _KINDS[kind]:
        raise ValueError(f"expected a {'/'.join(_KINDS[kind])} tensor, got {t.dtype}")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _fp16_bits(cb) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(cb, dtype=np.float16)).view(np.uint16)


# ----------------------------------------------------------------------------
def pack_weight_indices(w_idx: np.ndarray) -> np.ndarray:
    """uint8 [d_in][d_out] codes -> uint32 [d_in/8][d_out] words (host)."""
    w = np.ascontiguousarray(w_idx, dtype=np.uint8)
    d_in, d_out = w.shape
    out = np.empty((d_in // 8, d_out), dtype=np.uint32)
    _check("oasis_pack_weight_indices",
           load().oasis_pack_weight_indices(w.ctypes.data, d_in, d_out, out.ctypes.data))
    return out


def pack_weight_rows(w_idx: np.ndarray) -> np.ndarray:
    """uint8 [d_in][d_out] codes -> uint32 [d_in][ceil(d_out/8)] row-layout words (host)."""
    w = np.ascontiguousarray(w_idx, dtype=np.uint8)
    d_in, d_out = w.shape
    out = np.empty((d_in, (d_out + 7) // 8), dtype=np.uint32)
    _check("oasis_pack_weight_rows",
           load().oasis_pack_weight_rows(w.ctypes.data, d_in, d_out, out.ctypes.data))
    return out


def build_lut(cb_act, b_a: int, cb_wgt, b_w: int, out=None, stream=None):
    """Cartesian product LUT block (device uint8 tensor of 1088 bytes)."""
    import torch
    if out is None:
        out = torch.empty(LUT_BLOCK_BYTES, dtype=torch.uint8, device="cuda")
    ca = _fp16_bits(cb_act)
    cw = _fp16_bits(cb_wgt)
    _check("oasis_build_lut", load().oasis_build_lut(ca.ctypes.data, b_a, cw.ctypes.data, b_w,
                                                     _ptr(out, "u8"), _stream(stream)))
    return out


def quantize_act(x, lut, b_a: int, k: int, scale_mode: int = SCALE_ABSMAX,
                 out: Optional[Dict] = None, stream=None) -> Dict:
    """Scale, activation codes, outlier lists and residuals of every token."""
    import torch
    n, d_in = x.shape
    dev = x.device
    if out is None:
        out = {
            "idx_act": torch.empty((n, d_in // 2), dtype=torch.uint8, device=dev),
            "act_scale": torch.empty(n, dtype=torch.float32, device=dev),
            "max_idx": torch.empty((n, k), dtype=torch.int32, device=dev),
            "min_idx": torch.empty((n, k), dtype=torch.int32, device=dev),
            "residual": torch.empty((n, 2 * k), dtype=torch.float32, device=dev),
        }
    _check("oasis_quantize_act", load().oasis_quantize_act(
        _ptr(x, "f16"), n, d_in, _ptr(lut, "u8"), b_a, k, scale_mode, _ptr(out["idx_act"], "u8"),
        _ptr(out["act_scale"], "f32"), _ptr(out["max_idx"], "i32") if k else None,
        _ptr(out["min_idx"], "i32") if k else None, _ptr(out["residual"], "f32") if k else None,
        _stream(stream)))
    return out


def quantize_act_static(x, lut, b_a: int, k: int, thr_hi: float, thr_lo: float,
                        scale_mode: int = SCALE_ABSMAX, out: Optional[Dict] = None,
                        stream=None) -> Dict:
    """OASIS-S: scale and codes, outlier lists from fixed thresholds (k places
    per side, channel -1 / residual 0 where unused)."""
    import torch
    n, d_in = x.shape
    dev = x.device
    if out is None:
        out = {
            "idx_act": torch.empty((n, d_in // 2), dtype=torch.uint8, device=dev),
            "act_scale": torch.empty(n, dtype=torch.float32, device=dev),
            "max_idx": torch.empty((n, k), dtype=torch.int32, device=dev),
            "min_idx": torch.empty((n, k), dtype=torch.int32, device=dev),
            "residual": torch.empty((n, 2 * k), dtype=torch.float32, device=dev),
        }
    _check("oasis_quantize_act_static", load().oasis_quantize_act_static(
        _ptr(x, "f16"), n, d_in, _ptr(lut, "u8"), b_a, k, scale_mode, float(thr_hi), float(thr_lo),
        _ptr(out["idx_act"], "u8"), _ptr(out["act_scale"], "f32"), _ptr(out["max_idx"], "i32") if k else None,
        _ptr(out["min_idx"], "i32") if k else None, _ptr(out["residual"], "f32") if k else None,
        _stream(stream)))
    return out


def build_lut_quantize_act(cb_act, b_a: int, cb_wgt, b_w: int, x, k: int,
                           scale_mode: int = SCALE_ABSMAX, lut=None, out: Optional[Dict] = None,
                           stream=None):
    """build_lut then quantize_act in one launch; returns (lut, quantize outputs)."""
    import torch
    n, d_in = x.shape
    dev = x.device
    if lut is None:
        lut = torch.empty(LUT_BLOCK_BYTES, dtype=torch.uint8, device=dev)
    if out is None:
        out = {
            "idx_act": torch.empty((n, d_in // 2), dtype=torch.uint8, device=dev),
            "act_scale": torch.empty(n, dtype=torch.float32, device=dev),
            "max_idx": torch.empty((n, k), dtype=torch.int32, device=dev),
            "min_idx": torch.empty((n, k), dtype=torch.int32, device=dev),
            "residual": torch.empty((n, 2 * k), dtype=torch.float32, device=dev),
        }
    ca = _fp16_bits(cb_act)
    cw = _fp16_bits(cb_wgt)
    _check("oasis_build_lut_quantize_act", load().oasis_build_lut_quantize_act(
        ca.ctypes.data, b_a, cw.ctypes.data, b_w, _ptr(lut, "u8"), _ptr(x, "f16"), n, d_in, k, scale_mode,
        _ptr(out["idx_act"], "u8"), _ptr(out["act_scale"], "f32"), _ptr(out["max_idx"], "i32") if k else None,
        _ptr(out["min_idx"], "i32") if k else None, _ptr(out["residual"], "f32") if k else None,
        _stream(stream)))
    return lut, out


def build_lut_quantize_act_static(cb_act, b_a: int, cb_wgt, b_w: int, x, k: int, thr_hi: float,
                                  thr_lo: float, scale_mode: int = SCALE_ABSMAX, lut=None,
                                  out: Optional[Dict] = None, stream=None):
    """build_lut then quantize_act_static (OASIS-S) in one launch; returns (lut, outputs)."""
    import torch
    n, d_in = x.shape
    dev = x.device
    if lut is None:
        lut = torch.empty(LUT_BLOCK_BYTES, dtype=torch.uint8, device=dev)
    if out is None:
        out = {
            "idx_act": torch.empty((n, d_in // 2), dtype=torch.uint8, device=dev),
            "act_scale": torch.empty(n, dtype=torch.float32, device=dev),
            "max_idx": torch.empty((n, k), dtype=torch.int32, device=dev),
            "min_idx": torch.empty((n, k), dtype=torch.int32, device=dev),
            "residual": torch.empty((n, 2 * k), dtype=torch.float32, device=dev),
        }
    ca = _fp16_bits(cb_act)
    cw = _fp16_bits(cb_wgt)
    _check("oasis_build_lut_quantize_act_static", load().oasis_build_lut_quantize_act_static(
        ca.ctypes.data, b_a, cw.ctypes.data, b_w, _ptr(lut, "u8"), _ptr(x, "f16"), n, d_in, k, scale_mode,
        float(thr_hi), float(thr_lo), _ptr(out["idx_act"], "u8"), _ptr(out["act_scale"], "f32"),
        _ptr(out["max_idx"], "i32") if k else None, _ptr(out["min_idx"], "i32") if k else None,
        _ptr(out["residual"], "f32") if k else None, _stream(stream)))
    return lut, out


def cluster_act(x, lut, b_a: int, scale_mode: int = SCALE_ABSMAX, out: Optional[Dict] = None,
                stream=None) -> Dict:
    """Scale and activation codes only (the main branch's inputs)."""
    import torch
    n, d_in = x.shape
    if out is None:
        out = {"idx_act": torch.empty((n, d_in // 2), dtype=torch.uint8, device=x.device),
               "act_scale": torch.empty(n, dtype=torch.float32, device=x.device)}
    _check("oasis_cluster_act", load().oasis_cluster_act(
        _ptr(x, "f16"), n, d_in, _ptr(lut, "u8"), b_a, scale_mode, _ptr(out["idx_act"], "u8"),
        _ptr(out["act_scale"], "f32"), _stream(stream)))
    return out


def detect_outliers(x, lut, b_a: int, k: int, scale_mode: int = SCALE_ABSMAX,
                    out: Optional[Dict] = None, stream=None) -> Dict:
    """Outlier lists and residuals only (the outlier branch's inputs)."""
    import torch
    n, d_in = x.shape
    if out is None:
        out = {"max_idx": torch.empty((n, k), dtype=torch.int32, device=x.device),
               "min_idx": torch.empty((n, k), dtype=torch.int32, device=x.device),
               "residual": torch.empty((n, 2 * k), dtype=torch.float32, device=x.device)}
    _check("oasis_detect_outliers", load().oasis_detect_outliers(
        _ptr(x, "f16"), n, d_in, _ptr(lut, "u8"), b_a, k, scale_mode,
        _ptr(out["max_idx"], "i32") if k else None, _ptr(out["min_idx"], "i32") if k else None,
        _ptr(out["residual"], "f32") if k else None, _stream(stream)))
    return out


def lut_gemm(idx_act, act_scale, idx_w, w_scale, lut, b_a: int, b_w: int, algo: int = ALGO_MFMA,
             y=None, accumulate: bool = False, stream=None):
    """Main branch Y* (y = Y*, or y += Y* with accumulate)."""
    import torch
    n = idx_act.shape[0]
    d_in = idx_act.shape[1] * 2
    d_out = idx_w.shape[1]
    if y is None:
        y = torch.empty((n, d_out), dtype=torch.float32, device=idx_act.device)
    _check("oasis_lut_gemm", load().oasis_lut_gemm(
        _ptr(idx_act, "u8"), _ptr(act_scale, "f32"), n, d_in, _ptr(idx_w, "i32"), _ptr(w_scale, "f32"), d_out, _ptr(lut, "u8"),
        b_a, b_w, algo, _ptr(y, "f32"), 1 if accumulate else 0, _stream(stream)))
    return y


def outlier_compensate(max_idx, min_idx, residual, idx_w, lut, b_w: int, w_scale, d_in: int,
                       y=None, accumulate: bool = True, stream=None):
    """Outlier branch Y' (y += Y' with accumulate, else y = Y')."""
    import torch
    n, k = max_idx.shape
    d_out = idx_w.shape[1]
    if y is None:
        y = torch.empty((n, d_out), dtype=torch.float32, device=max_idx.device)
    _check("oasis_outlier_compensate", load().oasis_outlier_compensate(
        _ptr(max_idx, "i32") if k else None, _ptr(min_idx, "i32") if k else None,
        _ptr(residual, "f32") if k else None, n, k, _ptr(idx_w, "i32"), _ptr(lut, "u8"), b_w, _ptr(w_scale, "f32"), d_in,
        d_out, _ptr(y, "f32"), 1 if accumulate else 0, _stream(stream)))
    return y


def outlier_compensate_rows(max_idx, min_idx, residual, idx_wr, lut, b_w: int, w_scale,
                            d_in: int, y=None, accumulate: bool = True, stream=None):
    """Outlier branch Y' from the row-layout codes (y += Y' with accumulate, else y = Y')."""
    import torch
    n, k = max_idx.shape
    d_out = w_scale.shape[0]
    if y is None:
        y = torch.empty((n, d_out), dtype=torch.float32, device=max_idx.device)
    _check("oasis_outlier_compensate_rows", load().oasis_outlier_compensate_rows(
        _ptr(max_idx, "i32") if k else None, _ptr(min_idx, "i32") if k else None,
        _ptr(residual, "f32") if k else None, n, k, _ptr(idx_wr, "i32"), _ptr(lut, "u8"), b_w, _ptr(w_scale, "f32"), d_in,
        d_out, _ptr(y, "f32"), 1 if accumulate else 0, _stream(stream)))
    return y


def split_workspace_bytes(n: int, d_in: int, d_out: int, k: int) -> int:
    """Bytes of device workspace outlier_compensate_split needs."""
    return int(load().oasis_outlier_compensate_split_workspace(n, d_in, d_out, k))


def outlier_compensate_split(max_idx, min_idx, residual, idx_w, idx_wr, lut, b_w: int, w_scale,
                             d_in: int, y=None, accumulate: bool = True, workspace=None,
                             stream=None):
    """Outlier branch Y' split by channel: the heavy channels as a dense MFMA
    contraction, the other entries from the row-layout codes (y += Y' with
    accumulate, else y = Y').  workspace: a uint8 CUDA tensor of at least
    split_workspace_bytes(...) bytes (allocated here when None)."""
    import torch
    n, k = max_idx.shape
    d_out = w_scale.shape[0]
    if y is None:
        y = torch.empty((n, d_out), dtype=torch.float32, device=max_idx.device)
    need = split_workspace_bytes(n, d_in, d_out, k)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=max_idx.device)
    _check("oasis_outlier_compensate_split", load().oasis_outlier_compensate_split(
        _ptr(max_idx, "i32") if k else None, _ptr(min_idx, "i32") if k else None,
        _ptr(residual, "f32") if k else None, n, k, _ptr(idx_w, "i32"), _ptr(idx_wr, "i32"),
        _ptr(lut, "u8"), b_w, _ptr(w_scale, "f32"), d_in, d_out, _ptr(y, "f32"),
        1 if accumulate else 0, _ptr(workspace, "u8"), workspace.numel(), _stream(stream)))
    return y


def lut_gemm_compensated(idx_act, act_scale, idx_w, w_scale, lut, b_a: int, b_w: int, max_idx,
                         min_idx, residual, y=None, accumulate: bool = False, stream=None):
    """Main branch plus outlier compensation in one call: y (+)= Y* + Y'."""
    import torch
    n = idx_act.shape[0]
    d_in = idx_act.shape[1] * 2
    d_out = idx_w.shape[1]
    k = max_idx.shape[1]
    if y is None:
        y = torch.empty((n, d_out), dtype=torch.float32, device=idx_act.device)
    _check("oasis_lut_gemm_compensated", load().oasis_lut_gemm_compensated(
        _ptr(idx_act, "u8"), _ptr(act_scale, "f32"), n, d_in, _ptr(idx_w, "i32"), _ptr(w_scale, "f32"), d_out, _ptr(lut, "u8"),
        b_a, b_w, _ptr(max_idx, "i32") if k else None, _ptr(min_idx, "i32") if k else None,
        _ptr(residual, "f32") if k else None, k, _ptr(y, "f32"), 1 if accumulate else 0, _stream(stream)))
    return y


def lut_gemm_compensated_rows(idx_act, act_scale, idx_w, idx_wr, w_scale, lut, b_a: int,
                              b_w: int, max_idx, min_idx, residual, y=None,
                              accumulate: bool = False, stream=None):
    """lut_gemm_compensated with the outlier branch reading the row-layout codes."""
    import torch
    n = idx_act.shape[0]
    d_in = idx_act.shape[1] * 2
    d_out = idx_w.shape[1]
    k = max_idx.shape[1]
    if y is None:
        y = torch.empty((n, d_out), dtype=torch.float32, device=idx_act.device)
    _check("oasis_lut_gemm_compensated_rows", load().oasis_lut_gemm_compensated_rows(
        _ptr(idx_act, "u8"), _ptr(act_scale, "f32"), n, d_in, _ptr(idx_w, "i32"), _ptr(idx_wr, "i32") if k else None,
        _ptr(w_scale, "f32"), d_out, _ptr(lut, "u8"), b_a, b_w, _ptr(max_idx, "i32") if k else None,
        _ptr(min_idx, "i32") if k else None, _ptr(residual, "f32") if k else None, k, _ptr(y, "f32"),
        1 if accumulate else 0, _stream(stream)))
    return y


def lut_gemm_compensated_split(idx_act, act_scale, idx_w, idx_wr, w_scale, lut, b_a: int,
                               b_w: int, max_idx, min_idx, residual, y=None,
                               accumulate: bool = False, workspace=None, stream=None):
    """Main branch plus compensation for many tokens, the heavy channels of the
    split compensation inside the GEMM (y (+)= Y* + Y').  workspace: a uint8
    CUDA tensor of at least split_workspace_bytes(...) bytes (allocated here
    when None)."""
    import torch
    n = idx_act.shape[0]
    d_in = idx_act.shape[1] * 2
    d_out = idx_w.shape[1]
    k = max_idx.shape[1]
    if y is None:
        y = torch.empty((n, d_out), dtype=torch.float32, device=idx_act.device)
    if workspace is None:
        workspace = torch.empty(max(1, split_workspace_bytes(n, d_in, d_out, k)),
                                dtype=torch.uint8, device=idx_act.device)
    _check("oasis_lut_gemm_compensated_split", load().oasis_lut_gemm_compensated_split(
        _ptr(idx_act, "u8"), _ptr(act_scale, "f32"), n, d_in, _ptr(idx_w, "i32"),
        _ptr(idx_wr, "i32") if k else None, _ptr(w_scale, "f32"), d_out, _ptr(lut, "u8"), b_a,
        b_w, _ptr(max_idx, "i32") if k else None, _ptr(min_idx, "i32") if k else None,
        _ptr(residual, "f32") if k else None, k, _ptr(y, "f32"), 1 if accumulate else 0,
        _ptr(workspace, "u8"), workspace.numel(), _stream(stream)))
    return y


def lut_gemm_compensated_percol(idx_act, act_scale, idx_w, w_scale, lut, cb_cols, b_a: int,
                                b_w: int, max_idx, min_idx, residual, y=None,
                                accumulate: bool = False, stream=None):
    """lut_gemm_compensated with a weight codebook per output channel
    (cb_cols: fp16 device tensor [d_out][16]); one GEMV launch per 32 tokens."""
    import torch
    n = idx_act.shape[0]
    d_in = idx_act.shape[1] * 2
    d_out = idx_w.shape[1]
    k = max_idx.shape[1]
    if y is None:
        y = torch.empty((n, d_out), dtype=torch.float32, device=idx_act.device)
    _check("oasis_lut_gemm_compensated_percol", load().oasis_lut_gemm_compensated_percol(
        _ptr(idx_act, "u8"), _ptr(act_scale, "f32"), n, d_in, _ptr(idx_w, "i32"), _ptr(w_scale, "f32"), d_out, _ptr(lut, "u8"),
        _ptr(cb_cols, "f16"), b_a, b_w, _ptr(max_idx, "i32") if k else None, _ptr(min_idx, "i32") if k else None,
        _ptr(residual, "f32") if k else None, k, _ptr(y, "f32"), 1 if accumulate else 0, _stream(stream)))
    return y


def forward(x, lut, idx_w, w_scale, b_a: int, b_w: int, k: int, scale_mode: int = SCALE_ABSMAX,
            algo: int = ALGO_MFMA, out: Optional[Dict] = None, y=None, fused: bool = False,
            stream=None) -> Dict:
    """Whole hot path of one layer: Y = Y* + Y'.

    fused=False: quantize, compensation (y = Y'), then the main branch merged
    into it (y += Y*).  fused=True: quantize, then one call that produces both
    terms (matrix-core path only).
    """
    q = quantize_act(x, lut, b_a, k, scale_mode, out=out, stream=stream)
    if fused:
        y = lut_gemm_compensated(q["idx_act"], q["act_scale"], idx_w, w_scale, lut, b_a, b_w,
                                 q["max_idx"], q["min_idx"], q["residual"], y=y,
                                 accumulate=False, stream=stream)
    else:
        y = outlier_compensate(q["max_idx"], q["min_idx"], q["residual"], idx_w, lut, b_w,
                               w_scale, x.shape[1], y=y, accumulate=False, stream=stream)
        lut_gemm(q["idx_act"], q["act_scale"], idx_w, w_scale, lut, b_a, b_w, algo, y=y,
                 accumulate=True, stream=stream)
    q["y"] = y
    return q


_side_streams: Dict = {}


def forward_lookahead(x, lut, idx_w, w_scale, b_a: int, b_w: int, k: int,
                      scale_mode: int = SCALE_ABSMAX, algo: int = ALGO_MFMA,
                      out: Optional[Dict] = None, y=None, side_stream=None) -> Dict:
    """Whole hot path with the look-ahead schedule of Sec. III-C on two streams.

    Main stream: cluster the whole token, then the LUT-GEMM (y = Y*).  Side
    stream, concurrently: outlier detection and residuals.  The main stream
    then waits for the side stream and merges the compensation (y += Y').
    """
    import torch
    main = torch.cuda.current_stream()
    if side_stream is None:
        side_stream = _side_streams.setdefault(main.device, torch.cuda.Stream(device=main.device))
    n, d_in = x.shape
    if out is None:
        out = {
            "idx_act": torch.empty((n, d_in // 2), dtype=torch.uint8, device=x.device),
            "act_scale": torch.empty(n, dtype=torch.float32, device=x.device),
            "max_idx": torch.empty((n, k), dtype=torch.int32, device=x.device),
            "min_idx": torch.empty((n, k), dtype=torch.int32, device=x.device),
            "residual": torch.empty((n, 2 * k), dtype=torch.float32, device=x.device),
        }
    side_stream.wait_stream(main)                      # x and lut are ready
    with torch.cuda.stream(side_stream):
        detect_outliers(x, lut, b_a, k, scale_mode, out=out, stream=side_stream)
    cluster_act(x, lut, b_a, scale_mode, out=out, stream=main)
    y = lut_gemm(out["idx_act"], out["act_scale"], idx_w, w_scale, lut, b_a, b_w, algo, y=y,
                 accumulate=False, stream=main)
    main.wait_stream(side_stream)                      # outlier branch done
    for key in ("max_idx", "min_idx", "residual"):
        out[key].record_stream(side_stream)
    x.record_stream(side_stream)
    outlier_compensate(out["max_idx"], out["min_idx"], out["residual"], idx_w, lut, b_w, w_scale,
                       d_in, y=y, accumulate=True, stream=main)
    out["y"] = y
    return out

