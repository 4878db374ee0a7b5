"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a value
printed in the paper, Eq. (1) written independently, brute force on tiny
inputs, the textbook matmul of raw data, or a closed form.  None of them needs
a GPU.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import oasis_oracle as O
from paper_2507_23035_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def small_layer(n=5, d_in=64, d_out=48, k=3, seed=1, **kw):
    return synth.make_layer(synth.custom(n, d_in, d_out, k, seed=seed, **kw))


# ---------------------------------------------------------------- Sec. III-C1
def test_worked_residual_example():
    g = json.load(open(os.path.join(GOLDEN, "worked_residuals.json")))
    cb = np.array(g["codebook"], dtype=np.float16)
    x = np.array([g["token"]], dtype=np.float16)
    q = O.quantize_act(x, cb, g["b_a"], 1, mode=O.SCALE_NONE)
    pmax, pmin = g["outlier_channels"]["max"], g["outlier_channels"]["min"]
    assert q["max_idx"][0, 0] == pmax and q["min_idx"][0, 0] == pmin
    cent = cb.astype(np.float64)[q["a"][0]]
    assert abs(cent[pmax] - g["expected_centroid"]["max"]) < 1e-3
    assert abs(cent[pmin] - g["expected_centroid"]["min"]) < 1e-3
    assert abs(q["residual"][0, 0] - g["expected_residual"]["max"]) < g["tolerance"]
    assert abs(q["residual"][0, 1] - g["expected_residual"]["min"]) < g["tolerance"]
    # sign convention: residual = original - quantized
    assert q["residual"][0, 0] > 0 > q["residual"][0, 1]


# ---------------------------------------------------------------- Sec. IV-C
def _all_finite_fp16():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    v = bits.view(np.float16)
    return v[np.isfinite(v)]


@pytest.mark.parametrize("b_a", [1, 3, 4])
@pytest.mark.parametrize("t", [1.0, 0.375, 37.5])
def test_clustering_matches_eq1_exhaustively(b_a, t):
    """Boundary rule == Eq. (1) argmin for every finite fp16 value; on an exact
    midpoint the half-open interval sends the value to the upper centroid."""
    rng = np.random.default_rng(b_a)
    cb = np.sort(rng.standard_normal(1 << b_a)).astype(np.float16)
    cb = np.unique(cb)
    assert cb.size == (1 << b_a)
    xs = _all_finite_fp16()
    # keep the scaled values finite in fp16 terms
    xs = xs[np.abs(xs.astype(np.float64)) < 60000]
    x = xs.reshape(1, -1)
    tt = np.array([t], dtype=np.float32)
    rule = O.cluster(x, tt, cb, b_a)[0].astype(np.int64)
    # Eq. (1) written independently: squared distance to every scaled centroid
    cents = t * cb.astype(np.float64)
    d = (x[0].astype(np.float64)[:, None] - cents[None, :]) ** 2
    best = d.min(axis=1, keepdims=True)
    ties = (d == best)
    nearest_hi = (ties * np.arange(cb.size)[None, :]).max(axis=1)
    assert np.array_equal(rule, nearest_hi)
    assert rule.min() >= 0 and rule.max() <= cb.size - 1


def test_clustering_rejects_unsorted_codebook():
    with pytest.raises(ValueError):
        O.cluster_boundaries(np.array([0.5, 0.1], dtype=np.float16), 1)


# ---------------------------------------------------------------- Sec. IV-D
def _brute_rank_lists(x, k):
    """Position of every element in pop order, from pairwise comparisons only."""
    x = [float(v) for v in x]
    N = len(x)
    mx = [None] * k
    mn = [None] * k
    for p in range(N):
        r_hi = sum(1 for q in range(N) if x[q] > x[p] or (x[q] == x[p] and q < p))
        r_lo = sum(1 for q in range(N) if x[q] < x[p] or (x[q] == x[p] and q < p))
        if r_hi < k:
            mx[r_hi] = p
        if r_lo < k:
            mn[r_lo] = p
    return mx, mn


def _tiny_vectors():
    rng = np.random.default_rng(7)
    out = []
    for N in [1, 2, 3, 5, 8, 13, 16, 32, 37]:
        out.append(rng.standard_normal(N).astype(np.float16))
        out.append(rng.integers(-2, 3, N).astype(np.float16))         # many ties
        z = np.zeros(N, dtype=np.float16)
        z[::2] = np.float16(-0.0)                                       # -0 and +0
        out.append(z)
        out.append(np.full(N, 3.5, dtype=np.float16))                   # constant
    return out


@pytest.mark.parametrize("vi", range(36))
def test_topk_sort_orizuru_and_bruteforce_agree(vi):
    x = _tiny_vectors()[vi]
    N = x.size
    for k in sorted({0, 1, N // 2, N}):
        mx, mn = O.topk_lists(x.reshape(1, -1), k)
        bmx, bmn = _brute_rank_lists(x, k)
        assert list(mx[0]) == bmx and list(mn[0]) == bmn
        tree = O.Orizuru(x)
        tmx, tmn = tree.topk(k)
        assert tmx == bmx and tmn == bmn


def test_orizuru_node14_pop():
    """8-leaf tree with the maximum 9 at element 6: the first pop reads bits
    '110' from the root and lands on leaf node 14 (Sec. IV-D)."""
    x = np.array([3, 1, 4, 1, 5, 2, 9, 6], dtype=np.float16)
    tree = O.Orizuru(x)
    leaf, path = tree.pop("p")
    assert leaf == 14 and path == "110"
    assert int("1" + path, 2) == 14


@pytest.mark.parametrize("N", [2, 4, 8, 16, 64, 256])
@pytest.mark.parametrize("k", [0, 1, 2])
def test_orizuru_comparison_count(N, k):
    """Init N-1 (max) + N/2-1 (min, leaf level reused) comparisons, then
    log2 N per pop per tree: at most 1.5N + 2k log2 N (Sec. IV-D)."""
    rng = np.random.default_rng(N + k)
    x = rng.standard_normal(N).astype(np.float16)
    tree = O.Orizuru(x)
    assert tree.comparisons == N - 1 + N // 2 - 1
    tree.topk(k)
    L = int(math.log2(N))
    assert tree.comparisons == int(1.5 * N) - 2 + 2 * k * L
    assert tree.comparisons <= 1.5 * N + 2 * k * L


# ---------------------------------------------------------------- Sec. III-B
def test_lut_gemm_direct_counts_dequant_agree():
    L = small_layer(n=3, d_in=40, d_out=7, k=2, seed=3)
    t = O.act_scale(L.x)
    a = O.cluster(L.x, t, L.cb_a, 4)
    lut = O.build_lut(L.cb_a, L.cb_w, 4, 4)
    y1 = O.lut_gemm(a, L.w_idx, lut, t, L.s_w, 4)
    y2 = O.lut_gemm_counts(a, L.w_idx, lut, t, L.s_w, 4, 4)
    y3 = O.dequant_matmul(a, L.w_idx, L.cb_a, L.cb_w, t, L.s_w)
    np.testing.assert_allclose(y1, y3, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(y2, y3, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("b_a,b_w", [(4, 4), (3, 4), (2, 3), (1, 1)])
def test_exact_grid_reduces_to_textbook_matmul(b_a, b_w):
    """Activations that sit exactly on their token's centroids and weights that
    sit exactly on s_j * C_W: with k = 0 the method must give the plain matmul
    of the raw inputs (pins scales, concat order and LUT orientation)."""
    rng = np.random.default_rng(11)
    n, K, N = 4, 32, 12
    # dyadic centroids so that every product below is exact in fp16
    ca = np.sort(rng.choice(np.arange(-16, 17), 1 << b_a, replace=False)).astype(np.float64) / 16
    ca[np.argmax(np.abs(ca))] = np.sign(ca[np.argmax(np.abs(ca))]) * 1.0
    cw = rng.choice(np.arange(-8, 9), 1 << b_w, replace=False).astype(np.float64) / 8
    t = 2.0 ** rng.integers(-2, 4, n)
    s = 2.0 ** rng.integers(-6, -1, N)
    a = rng.integers(0, 1 << b_a, (n, K))
    a[:, 0] = np.argmax(np.abs(ca))                  # absmax of each token = t_i
    w = rng.integers(0, 1 << b_w, (K, N))
    X = (t[:, None] * ca[a]).astype(np.float16)
    W = s[None, :] * cw[w]
    assert np.array_equal(X.astype(np.float64), t[:, None] * ca[a])
    res = O.forward(X, w.astype(np.uint8), cw.astype(np.float16), s.astype(np.float32),
                    ca.astype(np.float16), b_a, b_w, 0)
    assert np.array_equal(res["t"].astype(np.float64), t)
    assert np.array_equal(res["a"].astype(np.int64), a)
    ref = X.astype(np.float64) @ W
    np.testing.assert_allclose(res["y"], ref, rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------- Sec. III-C
def test_k0_is_pure_codebook_gemm():
    L = small_layer(k=0)
    r = O.forward(L.x, L.w_idx, L.cb_w, L.s_w, L.cb_a, 4, 4, 0)
    assert r["residual"].shape == (L.spec.n, 0)
    assert np.all(r["y_comp"] == 0)
    ref = O.dequant_matmul(r["a"], L.w_idx, L.cb_a, L.cb_w, r["t"], L.s_w)
    np.testing.assert_allclose(r["y"], ref, rtol=1e-12, atol=1e-12)


def test_all_channels_outliers_recover_exact_gemm():
    """With every channel kept in fp16 the result is the GEMM of the original
    fp16 activations with the dequantized weights (up to the fp32 rounding of
    each residual)."""
    L = small_layer(n=4, d_in=32, d_out=20, k=32)
    r = O.forward(L.x, L.w_idx, L.cb_w, L.s_w, L.cb_a, 4, 4, 32)
    what = L.cb_w.astype(np.float64)[L.w_idx] * L.s_w.astype(np.float64)[None, :]
    ref = L.x.astype(np.float64) @ what
    scale = np.abs(L.x.astype(np.float64)) @ np.abs(what)
    assert np.all(np.abs(r["y"] - ref) <= 2.0 ** -22 * scale + 1e-12)


@pytest.mark.parametrize("seed,k", [(0, 1), (1, 3), (2, 8), (3, 20)])
def test_lookahead_equals_conventional_scheme(seed, k):
    """Y* + Y' equals quantized inliers plus fp16 outliers (Sec. II-C)."""
    L = small_layer(n=6, d_in=24, d_out=10, k=k, seed=seed)
    x = L.x.copy()
    if seed == 3:
        x[0, :] = np.float16(2.0)                   # constant token: lists overlap
    r = O.forward(x, L.w_idx, L.cb_w, L.s_w, L.cb_a, 4, 4, k)
    what = L.cb_w.astype(np.float64)[L.w_idx] * L.s_w.astype(np.float64)[None, :]
    xh = r["t"].astype(np.float64)[:, None] * L.cb_a.astype(np.float64)[r["a"]]
    mixed = xh.copy()
    for i in range(x.shape[0]):
        outl = set(r["max_idx"][i]) | set(r["min_idx"][i])
        for p in outl:
            mixed[i, p] = float(x[i, p])
    ref = mixed @ what
    scale = np.abs(mixed) @ np.abs(what)
    assert np.all(np.abs(r["y"] - ref) <= 2.0 ** -22 * scale + 1e-12)


def test_duplicate_channels_compensated_once():
    x = np.full((1, 8), 1.5, dtype=np.float16)
    cb = np.array([-1, -0.5, 0.25, 0.75], dtype=np.float16)
    q = O.quantize_act(x, cb, 2, 4)
    assert list(q["max_idx"][0]) == [0, 1, 2, 3]
    assert list(q["min_idx"][0]) == [0, 1, 2, 3]
    assert np.all(q["residual"][0, 4:] == 0)
    assert np.all(q["residual"][0, :4] != 0)


# ---------------------------------------------------------------- per-column codebooks (R14)
def test_percol_by_hand():
    """One token, two channels, two columns with their own codebooks; t = 1
    (mode NONE), C_A = (-1, 1), codes a = (1, 0)."""
    x = np.array([[1.0, -1.0]], dtype=np.float16)
    cb_a = np.array([-1.0, 1.0], dtype=np.float16)
    w_idx = np.array([[0, 1], [1, 0]], dtype=np.uint8)            # [p][j]
    cols = np.array([[0.5, 2.0], [-1.0, 4.0]], dtype=np.float16)  # C_W[j][w]
    s_w = np.array([1.0, 0.5], dtype=np.float32)
    r = O.forward_percol(x, w_idx, cols, s_w, cb_a, 1, 1, 0, mode=O.SCALE_NONE)
    # y_0 = 1 * (1 * 0.5 + (-1) * 2.0) = -1.5;  y_1 = 0.5 * (1 * 4.0 + (-1) * -1.0) = 2.5
    assert list(r["y"][0]) == [-1.5, 2.5]


def test_percol_equal_rows_is_the_shared_codebook():
    L = small_layer(n=4, d_in=40, d_out=12, k=3, seed=9)
    cols = np.tile(L.cb_w, (L.spec.d_out, 1))
    a = O.forward(L.x, L.w_idx, L.cb_w, L.s_w, L.cb_a, 4, 4, 3)
    b = O.forward_percol(L.x, L.w_idx, cols, L.s_w, L.cb_a, 4, 4, 3)
    assert np.array_equal(a["y"], b["y"])


def test_percol_lut_gemm_equals_dequant_matmul():
    L = small_layer(n=5, d_in=48, d_out=11, k=2, seed=10)
    cols = synth.percol_codebooks(L)
    q = O.quantize_act(L.x, L.cb_a, 4, 2)
    lut = O.build_lut_percol(L.cb_a, cols, 4, 4)
    ys = O.lut_gemm_percol(q["a"], L.w_idx, lut, q["t"], L.s_w, 4)
    xh = q["t"].astype(np.float64)[:, None] * L.cb_a.astype(np.float64)[q["a"]]
    ref = xh @ O.dequant_weights_percol(L.w_idx, cols, L.s_w)
    np.testing.assert_allclose(ys, ref, rtol=1e-12, atol=1e-12)


def test_percol_all_channels_listed_recover_exact_gemm():
    L = small_layer(n=3, d_in=16, d_out=9, k=16, seed=11)
    cols = synth.percol_codebooks(L)
    r = O.forward_percol(L.x, L.w_idx, cols, L.s_w, L.cb_a, 4, 4, 16)
    what = O.dequant_weights_percol(L.w_idx, cols, L.s_w)
    ref = L.x.astype(np.float64) @ what
    scale = np.abs(L.x.astype(np.float64)) @ np.abs(what)
    assert np.all(np.abs(r["y"] - ref) <= 2.0 ** -22 * scale + 1e-12)


# ---------------------------------------------------------------- inlier scale (R13)
def test_inlier_scale_by_hand():
    """k = 1: the max list takes 10, the min list -2; the inliers' absmax is 3.
    Boundaries of C_A = (-1, -0.5, 0.25, 0.75) are (-0.75, -0.125, 0.5), scaled
    by t = 3: (-2.25, -0.375, 1.5)."""
    x = np.array([[10, 1, -2, 0.5, -0.25, 3]], dtype=np.float16)
    cb = np.array([-1, -0.5, 0.25, 0.75], dtype=np.float16)
    q = O.quantize_act(x, cb, 2, 1, mode=O.SCALE_INLIER)
    assert q["t"][0] == np.float32(3.0)
    assert list(q["a"][0]) == [3, 2, 1, 2, 2, 3]
    assert list(q["max_idx"][0]) == [0] and list(q["min_idx"][0]) == [2]
    assert list(q["residual"][0]) == [np.float32(10 - 3 * 0.75), np.float32(-2 - 3 * -0.5)]


def test_inlier_scale_is_the_absmax_of_the_unlisted():
    L = small_layer(n=6, d_in=96, k=5, seed=7)
    q = O.quantize_act(L.x, L.cb_a, 4, 5, mode=O.SCALE_INLIER)
    ta = O.act_scale(L.x)
    for i in range(L.spec.n):
        listed = set(q["max_idx"][i]) | set(q["min_idx"][i])
        rest = np.abs(np.delete(L.x[i].astype(np.float64), sorted(listed)))
        assert q["t"][i] == np.float32(rest.max()) <= ta[i]
    q0 = O.quantize_act(L.x, L.cb_a, 4, 0, mode=O.SCALE_INLIER)
    assert np.array_equal(q0["t"], ta)               # no outliers: the absmax


def test_inlier_scale_all_channels_listed():
    """Every channel listed: t = 0, the main branch vanishes and the outlier
    branch alone gives the GEMM of the fp16 activations."""
    L = small_layer(n=3, d_in=16, d_out=12, k=16)
    r = O.forward(L.x, L.w_idx, L.cb_w, L.s_w, L.cb_a, 4, 4, 16, mode=O.SCALE_INLIER)
    assert np.all(r["t"] == 0) and np.all(r["y_star"] == 0)
    what = L.cb_w.astype(np.float64)[L.w_idx] * L.s_w.astype(np.float64)[None, :]
    ref = L.x.astype(np.float64) @ what
    np.testing.assert_allclose(r["y"], ref, rtol=1e-12, atol=1e-9)


@pytest.mark.parametrize("seed,k", [(4, 2), (5, 6)])
def test_inlier_lookahead_equals_conventional_scheme(seed, k):
    L = small_layer(n=5, d_in=32, d_out=9, k=k, seed=seed)
    r = O.forward(L.x, L.w_idx, L.cb_w, L.s_w, L.cb_a, 4, 4, k, mode=O.SCALE_INLIER)
    what = L.cb_w.astype(np.float64)[L.w_idx] * L.s_w.astype(np.float64)[None, :]
    mixed = r["t"].astype(np.float64)[:, None] * L.cb_a.astype(np.float64)[r["a"]]
    for i in range(L.spec.n):
        for p in set(r["max_idx"][i]) | set(r["min_idx"][i]):
            mixed[i, p] = float(L.x[i, p])
    ref = mixed @ what
    scale = np.abs(mixed) @ np.abs(what)
    assert np.all(np.abs(r["y"] - ref) <= 2.0 ** -22 * scale + 1e-12)


# ---------------------------------------------------------------- Sec. V-A, OASIS-S
def test_static_lists_by_hand():
    """Fixed thresholds: the channels at or beyond them, in channel order,
    capped at k per side, -1 in the places left (read by hand)."""
    x = np.array([[0.5, 3.0, -4.0, 2.5, -0.125, 7.0, -1.0, 2.0]], dtype=np.float16)
    mx, mn = O.static_lists(x, 2.5, -1.0, 4)
    assert mx.tolist() == [[1, 3, 5, -1]]
    assert mn.tolist() == [[2, 6, -1, -1]]
    mx, mn = O.static_lists(x, 2.5, -1.0, 2)
    assert mx.tolist() == [[1, 3]] and mn.tolist() == [[2, 6]]
    # a threshold between two fp16 values: 2.4 keeps 2.5 and drops 2.0
    mx, _ = O.static_lists(x, 2.4, -9.0, 8)
    assert mx[0, :3].tolist() == [1, 3, 5] and mx[0, 3] == -1


def test_static_lists_equal_topk_sets_at_the_kth_values():
    """With the thresholds at a token's k-th largest and k-th smallest value
    (distinct values) the static lists hold exactly the top-k sets."""
    rng = np.random.default_rng(4)
    for k in (1, 3, 10):
        x = rng.permutation(np.arange(-50, 50)).astype(np.float16)[None, :] / np.float16(8)
        x = x.astype(np.float16)
        srt = np.sort(x[0].astype(np.float64))
        mx, mn = O.static_lists(x, srt[-k], srt[k - 1], k)
        tmx, tmn = O.topk_lists(x, k)
        assert set(mx[0].tolist()) == set(tmx[0].tolist())
        assert set(mn[0].tolist()) == set(tmn[0].tolist())


@pytest.mark.parametrize("seed", [0, 1])
def test_static_forward_equals_conventional_scheme(seed):
    """OASIS-S still gives quantized inliers plus fp16 outliers (Sec. II-C),
    unused places adding nothing."""
    L = small_layer(n=6, d_in=24, d_out=10, k=3, seed=seed)
    r = O.forward(L.x, L.w_idx, L.cb_w, L.s_w, L.cb_a, 4, 4, 3, thresholds=(1.5, -1.5))
    what = L.cb_w.astype(np.float64)[L.w_idx] * L.s_w.astype(np.float64)[None, :]
    mixed = r["t"].astype(np.float64)[:, None] * L.cb_a.astype(np.float64)[r["a"]]
    for i in range(L.x.shape[0]):
        for p in set(r["max_idx"][i]) | set(r["min_idx"][i]):
            if p >= 0:
                mixed[i, p] = float(L.x[i, p])
    assert (r["max_idx"] == -1).any()        # some places unused
    ref = mixed @ what
    scale = np.abs(mixed) @ np.abs(what)
    assert np.all(np.abs(r["y"] - ref) <= 2.0 ** -22 * scale + 1e-12)
    assert np.all(r["residual"][:, :3][r["max_idx"] == -1] == 0)


# ---------------------------------------------------------------- Table I
def test_cost_model_closed_forms():
    c = O.cost_model(4096, 4096, 4, 4)
    assert c["waq_lut_size"] == 256
    assert c["woq_lut_size"] / c["waq_lut_size"] == 64
    assert c["waq_group"] / c["woq_group"] == 1024
    assert c["woq_reduction_flops"] / c["waq_reduction_flops"] == 16


def test_pack_roundtrip():
    rng = np.random.default_rng(0)
    a = rng.integers(0, 16, (3, 24)).astype(np.uint8)
    assert np.array_equal(O.unpack_act_indices(O.pack_act_indices(a), 24), a)
    w = rng.integers(0, 16, (16, 5)).astype(np.uint8)
    pw = O.pack_weight_indices(w)
    for p in range(16):
        for j in range(5):
            assert (int(pw[p // 8, j]) >> (4 * (p % 8))) & 0xF == w[p, j]


# Hand-written packings of the three index layouts the library exchanges
# (activation codes: channel 2q in the low nibble of byte q; weight codes,
# GEMM layout: channel 8b+e of column j at bits 4e..4e+3 of word (b, j);
# row layout: column 8m+c of channel p at bits 4c..4c+3 of word (p, m)).
def check_act_packing(pack, unpack):
    assert np.array_equal(pack(np.array([[1, 2, 3, 4]], dtype=np.uint8)),
                          np.array([[0x21, 0x43]], dtype=np.uint8))
    assert np.array_equal(pack(np.array([[15, 0, 0, 10], [7, 8, 9, 6]], dtype=np.uint8)),
                          np.array([[0x0F, 0xA0], [0x87, 0x69]], dtype=np.uint8))
    assert np.array_equal(unpack(np.array([[0x21, 0x43]], dtype=np.uint8), 4),
                          np.array([[1, 2, 3, 4]], dtype=np.uint8))


def test_act_packing_by_hand():
    check_act_packing(O.pack_act_indices, O.unpack_act_indices)


def test_act_packing_pin_catches_a_nibble_swap():
    """The hand pin fails for a packer (and unpacker) with the nibbles swapped,
    a mistake the round trip alone cannot see."""
    def pack_swapped(a):
        a = np.asarray(a, dtype=np.uint8)
        return (a[:, 1::2] | (a[:, 0::2] << 4)).astype(np.uint8)

    def unpack_swapped(p, K):
        p = np.asarray(p, dtype=np.uint8)
        out = np.zeros((p.shape[0], K), dtype=np.uint8)
        out[:, 1::2] = p & 0xF
        out[:, 0::2] = p >> 4
        return out

    a = np.arange(8, dtype=np.uint8).reshape(1, 8)
    assert np.array_equal(unpack_swapped(pack_swapped(a), 8), a)   # round trip holds
    with pytest.raises(AssertionError):
        check_act_packing(pack_swapped, unpack_swapped)


def test_weight_packing_by_hand():
    w = np.zeros((8, 2), dtype=np.uint8)
    w[:, 0] = np.arange(1, 9)            # channel e of column 0 holds e + 1
    w[:, 1] = 15 - np.arange(8)          # channel e of column 1 holds 15 - e
    assert np.array_equal(O.pack_weight_indices(w),
                          np.array([[0x87654321, 0x89ABCDEF]], dtype=np.uint32))
    w16 = np.zeros((16, 1), dtype=np.uint8)
    w16[9, 0] = 5                         # channel 9 = word 1, nibble 1
    assert np.array_equal(O.pack_weight_indices(w16), np.array([[0], [0x50]], dtype=np.uint32))


def test_weight_row_packing_by_hand():
    w = np.arange(1, 11, dtype=np.uint8).reshape(1, 10)   # columns 0..9 of channel 0
    assert np.array_equal(O.pack_weight_rows(w),
                          np.array([[0x87654321, 0x000000A9]], dtype=np.uint32))
    w2 = np.zeros((2, 3), dtype=np.uint8)
    w2[1, 2] = 12                         # channel 1, column 2: word (1, 0), nibble 2
    assert np.array_equal(O.pack_weight_rows(w2), np.array([[0], [0xC00]], dtype=np.uint32))
