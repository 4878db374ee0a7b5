"""Seeded synthetic workloads for the OASIS W4A4 linear layer.

This module only draws random data and prepares the offline inputs of one
quantized linear layer; it performs none of the hot-path arithmetic (no
clustering of activations, no outlier selection, no LUT, no GEMM).  Both the
CPU oracle and the HIP path are fed from it.

The paper evaluates trained LLM layers on WikiText-2 / C4 activations, which
are not available here; the synthetic recipe below stands in for them (same
shapes as the LLM projections the paper names, heavy-tailed activations with a
few large-magnitude channels, Gaussian weights).

Offline preparation (done here, once per layer, never timed):
  * per-output-channel weight scale s_j = fp16(max_p |W[p, j]|)           (Sec. III-A)
  * one weight codebook shared by the whole matrix, fitted by K-Means on
    W / s (Eq. (1)), fp16, ascending                                      (Sec. III-A)
  * weight indices = nearest centroid of W[p, j] / s_j                    (Eq. (1))
  * activation codebook fitted offline by K-Means on absmax-normalised
    calibration tokens drawn from the same distribution                  (Sec. III-A, V-A)
"""
from __future__ import annotations

from dataclasses import dataclass, replace
from typing import Dict, Optional

import numpy as np

FP16_MAX = 65504.0


@dataclass(frozen=True)
class LayerSpec:
    """Shape and value distribution of one synthetic linear layer."""

    name: str
    n: int            # tokens
    d_in: int         # reduction length (input channels)
    d_out: int        # output channels
    k: int            # outliers per side per token (max list and min list)
    dist: str = "t"   # "normal" or "t" (Student-t)
    nu: float = 3.0   # Student-t degrees of freedom
    outlier_frac: float = 0.01   # fraction of heavy channels (ignored if outlier_count set)
    outlier_count: Optional[int] = None
    outlier_scale: float = 50.0
    w_sigma: float = 0.02
    b_a: int = 4
    b_w: int = 4
    calib_tokens: int = 128
    seed: int = 0

    @property
    def heavy_channels(self) -> int:
        if self.outlier_count is not None:
            return min(self.outlier_count, self.d_in)
        return int(np.floor(self.outlier_frac * self.d_in))


# The five layer shapes of the workload set: a tiny layer, a LLaMA-7B-class
# decode GEMV, the 7B MLP up- and down-projections at prefill, and a
# 70B-class MLP projection at prefill and decode (same weights).
CONFIGS: Dict[str, LayerSpec] = {
    "tiny_4x256x256": LayerSpec("tiny_4x256x256", 4, 256, 256, 4, dist="normal",
                                outlier_count=4, outlier_scale=20.0, w_sigma=0.02),
    "decode_8x4096x4096": LayerSpec("decode_8x4096x4096", 8, 4096, 4096, 32, dist="t", nu=3.0,
                                    outlier_frac=0.01, outlier_scale=50.0, w_sigma=0.02),
    "prefill_up_2048x4096x11008": LayerSpec("prefill_up_2048x4096x11008", 2048, 4096, 11008, 32,
                                            dist="t", nu=3.0, outlier_frac=0.01,
                                            outlier_scale=50.0, w_sigma=0.02),
    "prefill_down_2048x11008x4096": LayerSpec("prefill_down_2048x11008x4096", 2048, 11008, 4096, 128,
                                              dist="t", nu=2.0, outlier_frac=0.02,
                                              outlier_scale=100.0, w_sigma=0.02),
    "large_prefill_4096x8192x28672": LayerSpec("large_prefill_4096x8192x28672", 4096, 8192, 28672, 64,
                                               dist="t", nu=3.0, outlier_frac=0.01,
                                               outlier_scale=50.0, w_sigma=0.01),
    "large_decode_16x8192x28672": LayerSpec("large_decode_16x8192x28672", 16, 8192, 28672, 64,
                                            dist="t", nu=3.0, outlier_frac=0.01,
                                            outlier_scale=50.0, w_sigma=0.01),
}


def _streams(seed: int):
    ss = np.random.SeedSequence(seed)
    kx, kw, kc, kcal = ss.spawn(4)
    return (np.random.default_rng(kx), np.random.default_rng(kw),
            np.random.default_rng(kc), np.random.default_rng(kcal))


def _draw_tokens(rng, spec: LayerSpec, n: int, heavy: np.ndarray) -> np.ndarray:
    if spec.dist == "normal":
        x = rng.standard_normal((n, spec.d_in))
    elif spec.dist == "t":
        x = rng.standard_t(spec.nu, size=(n, spec.d_in))
    else:
        raise ValueError(f"unknown distribution {spec.dist!r}")
    if heavy.size:
        x[:, heavy] *= spec.outlier_scale
    return x


def to_fp16_saturating(x: np.ndarray) -> np.ndarray:
    """Clip to the finite fp16 range, then round to nearest even."""
    return np.clip(x, -FP16_MAX, FP16_MAX).astype(np.float16)


def kmeans_1d(values: np.ndarray, n_clusters: int, rng, iters: int = 50) -> np.ndarray:
    """Plain Lloyd K-Means on scalars with k-means++ seeding (Eq. (1)).

    Returns strictly ascending fp16 centroids (ties nudged apart by one ulp).
    """
    v = np.asarray(values, dtype=np.float64).ravel()
    # k-means++ seeding
    cents = [v[rng.integers(v.size)]]
    d2 = (v - cents[0]) ** 2
    for _ in range(1, n_clusters):
        tot = d2.sum()
        if tot <= 0:
            cents.append(v[rng.integers(v.size)])
        else:
            cents.append(v[rng.choice(v.size, p=d2 / tot)])
        d2 = np.minimum(d2, (v - cents[-1]) ** 2)
    c = np.sort(np.array(cents))
    for _ in range(iters):
        mids = 0.5 * (c[1:] + c[:-1])
        lab = np.searchsorted(mids, v)
        sums = np.bincount(lab, weights=v, minlength=n_clusters)
        cnt = np.bincount(lab, minlength=n_clusters)
        newc = np.where(cnt > 0, sums / np.maximum(cnt, 1), c)
        newc = np.sort(newc)
        if np.allclose(newc, c, rtol=0, atol=1e-12):
            c = newc
            break
        c = newc
    h = c.astype(np.float16)
    # enforce strictly ascending fp16 values
    for i in range(1, h.size):
        if not h[i] > h[i - 1]:
            h[i] = np.nextafter(h[i - 1], np.float16(np.inf))
    return h


def nearest_index(values: np.ndarray, codebook: np.ndarray) -> np.ndarray:
    """Offline weight quantization: index of the nearest centroid (Eq. (1))."""
    c = codebook.astype(np.float64)
    mids = 0.5 * (c[1:] + c[:-1])
    return np.searchsorted(mids, values).astype(np.uint8)


@dataclass
class Layer:
    spec: LayerSpec
    x: np.ndarray          # fp16 [n][d_in]
    w_idx: np.ndarray      # uint8 [d_in][d_out], values < 2^b_w
    cb_w: np.ndarray       # fp16 [2^b_w] weight codebook (shared by the matrix)
    s_w: np.ndarray        # fp32 [d_out] per-output-channel scale (fp16-representable)
    cb_a: np.ndarray       # fp16 [2^b_a] activation codebook, strictly ascending
    heavy: np.ndarray      # heavy (outlier) channel ids used by the generator
    clipped: int           # number of activations saturated to the fp16 range


_W_CACHE: Dict[tuple, tuple] = {}


def _weights(spec: LayerSpec, rng_w):
    key = (spec.d_in, spec.d_out, spec.w_sigma, spec.b_w, spec.seed)
    if key in _W_CACHE:
        return _W_CACHE[key]
    w = rng_w.standard_normal((spec.d_in, spec.d_out), dtype=np.float32)
    w *= np.float32(spec.w_sigma)
    s = np.abs(w).max(axis=0).astype(np.float16)
    s = np.where(s == 0, np.float16(1.0), s).astype(np.float16)
    s32 = s.astype(np.float32)
    wn = w / s32[None, :]
    flat = wn.ravel()
    samp = flat if flat.size <= (1 << 20) else flat[rng_w.choice(flat.size, 1 << 20, replace=False)]
    cb_w = kmeans_1d(samp, 1 << spec.b_w, rng_w)
    w_idx = nearest_index(wn, cb_w)
    out = (w_idx, cb_w, s32)
    if spec.d_in * spec.d_out >= (1 << 24):
        _W_CACHE.clear()
        _W_CACHE[key] = out
    return out


def make_layer(spec: LayerSpec) -> Layer:
    """Generate one layer: activations, quantized weights and both codebooks."""
    rng_x, rng_w, rng_c, rng_cal = _streams(spec.seed)
    heavy = np.sort(rng_c.choice(spec.d_in, spec.heavy_channels, replace=False)) \
        if spec.heavy_channels else np.zeros(0, dtype=np.int64)
    x64 = _draw_tokens(rng_x, spec, spec.n, heavy)
    clipped = int(np.count_nonzero(np.abs(x64) > FP16_MAX))
    x = to_fp16_saturating(x64)
    w_idx, cb_w, s_w = _weights(spec, rng_w)
    cal = to_fp16_saturating(_draw_tokens(rng_cal, spec, spec.calib_tokens, heavy)).astype(np.float64)
    am = np.abs(cal).max(axis=1, keepdims=True)
    am[am == 0] = 1.0
    cb_a = kmeans_1d(cal / am, 1 << spec.b_a, rng_cal)
    return Layer(spec, x, w_idx, cb_w, s_w, cb_a, heavy, clipped)


def percol_codebooks(layer: Layer) -> np.ndarray:
    """Per-output-channel weight codebooks (fp16 [d_out][2^b_w]) for the
    per-column variant: column j's codebook is the shared one scaled by u_j in
    [0.75, 1.25] and shifted by v_j ~ N(0, 0.02^2), rounded to fp16, from a
    stream of its own (the layer's other streams are untouched)."""
    spec = layer.spec
    rng = np.random.default_rng(np.random.SeedSequence([spec.seed, 0x9E37]))
    u = rng.uniform(0.75, 1.25, spec.d_out)
    v = 0.02 * rng.standard_normal(spec.d_out)
    cb = layer.cb_w.astype(np.float64)[None, :] * u[:, None] + v[:, None]
    return cb.astype(np.float16)


def static_thresholds(layer: Layer, k: int):
    """Offline outlier thresholds for OASIS-S (Sec. V-A): the mean over the
    layer's calibration tokens of the k-th largest and the k-th smallest
    value, as fp32 (thr_hi, thr_lo)."""
    spec = layer.spec
    _, _, _, rng_cal = _streams(spec.seed)
    cal = to_fp16_saturating(_draw_tokens(rng_cal, spec, spec.calib_tokens, layer.heavy))
    srt = np.sort(cal.astype(np.float64), axis=1)
    return float(np.float32(srt[:, -k].mean())), float(np.float32(srt[:, k - 1].mean()))


def config(name: str, **overrides) -> LayerSpec:
    spec = CONFIGS[name]
    return replace(spec, **overrides) if overrides else spec


def custom(n: int, d_in: int, d_out: int, k: int, seed: int = 0, **kw) -> LayerSpec:
    """A small layer with the decode recipe, for ragged / edge-case tests."""
    base = dict(dist="t", nu=3.0, outlier_frac=0.01, outlier_scale=50.0, w_sigma=0.02)
    base.update(kw)
    return LayerSpec(f"custom_{n}x{d_in}x{d_out}_k{k}_s{seed}", n, d_in, d_out, k, seed=seed, **base)
