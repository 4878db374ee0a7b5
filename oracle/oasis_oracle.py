"""CPU oracle for the OASIS hot path (arXiv 2507.23035).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this
module: only the tests, the smoke check and the CPU-baseline leg of the
benchmark use it.  It shares no code with the HIP library.

A plain, slow, obviously-correct restatement of what the paper's method
computes, in numpy.  Floating point is fp64 except where the method fixes a
narrower precision (the LUT entries, the clustering boundaries and the
residuals are defined on fp16/fp32 values; see the readings below).

Notation follows the paper: n tokens, K = d_in input channels, N = d_out
output channels, n_A / n_W bit-widths (b_a, b_w here), C_A / C_W the
activation / weight codebooks, k outliers per side per token.

Readings taken where the paper is silent or loose (each one is listed in the
design notes of the repository):
  R1  The weight codebook is shared by the whole matrix and every output
      channel has its own scale s_j (Sec. III-A), so a single Cartesian
      product LUT exists (Sec. III-B).
  R2  Per-token scale t_i = max_p |x_ip| over all channels, outliers
      included ("absmax"); "none" sets t_i = 1.  The token's centroids are
      t_i * C_A (Sec. III-A).
  R3  k is per side: k largest and k smallest per token (Sec. III-A, IV-D).
  R4  Ties go to the lower channel index in both lists; lists are in pop
      order (largest first / smallest first) (Sec. IV-D, "Dealing with ties").
  R5  A channel present in both lists is compensated once: its min-list
      residual is 0.
  R6  Clustering follows the mid-point boundary rule of Sec. IV-C:
      b_c = (c_c + c_{c+1}) / 2 evaluated in fp32, scaled boundary
      P_c = fp32(t * b_c), cluster index = #{c : x >= P_c} (half-open
      intervals [b_{c-1}, b_c)).
  R7  LUT entries are fp32(C_A[a]) * fp32(C_W[w]), exact in fp32, indexed by
      the concatenation (a << n_W) | w (Sec. III-B, IV-A).
  R8  Residual r = fp32(x - fp32(t * C_A[a])), one fp32 rounding (the
      Error Calculation Unit of Sec. IV-A, in fp32 instead of fp16).
  R9  Accumulation is exact-ish (fp64 here); the GPU accumulates in fp32.
  R12 OASIS-S (Sec. V-A: thresholds reused from the offline calibration):
      the max list holds the channels with x >= thr_hi, the min list those
      with x <= thr_lo, in channel order, at most k each; unused places hold
      channel -1 and residual 0.
  R13 Inlier scale ("inlier"): t_i = max |x_ip| over the channels in neither
      list, so the main branch's centroids span only the values it keeps
      (the outliers are compensated exactly, Sec. III-A, III-C); t_i = 0 when
      every channel is listed (the outlier branch then carries the whole
      product).  The lists come first, so this mode has no look-ahead split.
  R14 Per-output-channel weight codebooks (an extension the paper leaves
      open, Sec. III-A): column j has its own C_W[j], so each column has its
      own LUT slice C_A (x) C_W[j], lut_j[(a << n_W) | w] = C_A[a] * C_W[j][w];
      s_j still scales the column.  A shared codebook is the case of equal rows.
"""
from __future__ import annotations

import math
from typing import Dict, List, Tuple

import numpy as np

SCALE_ABSMAX = 0
SCALE_NONE = 1
SCALE_INLIER = 2


# --------------------------------------------------------------------------
# Sec. III-B: the Cartesian product LUT, built offline from the two codebooks
# --------------------------------------------------------------------------
def build_lut(cb_a: np.ndarray, cb_w: np.ndarray, b_a: int, b_w: int) -> np.ndarray:
    """All products of an activation centroid and a weight centroid.

    Entry for the concatenated index (a << b_w) | w holds C_A[a] * C_W[w].
    The product of two fp16 numbers needs at most 22 significant bits, so it
    is exact in fp32; the oracle forms it in fp64 and checks that.
    """
    ca = np.asarray(cb_a, dtype=np.float16)[: 1 << b_a].astype(np.float64)
    cw = np.asarray(cb_w, dtype=np.float16)[: 1 << b_w].astype(np.float64)
    lut = np.zeros(1 << (b_a + b_w), dtype=np.float64)
    for a in range(1 << b_a):
        for w in range(1 << b_w):
            lut[(a << b_w) | w] = ca[a] * cw[w]
    out = lut.astype(np.float32)
    assert np.array_equal(out.astype(np.float64), lut), "LUT product not exact in fp32"
    return out


# --------------------------------------------------------------------------
# Sec. III-A: per-token scale of the activation codebook
# --------------------------------------------------------------------------
def act_scale(x: np.ndarray, mode: int = SCALE_ABSMAX) -> np.ndarray:
    """t_i: absmax over the token's channels (a max of fp16 values, exact)."""
    x = np.asarray(x, dtype=np.float16)
    if mode == SCALE_NONE:
        return np.ones(x.shape[0], dtype=np.float32)
    if mode != SCALE_ABSMAX:
        raise ValueError("unknown scale mode")
    if x.shape[1] == 0:
        return np.zeros(x.shape[0], dtype=np.float32)
    return np.abs(x.astype(np.float64)).max(axis=1).astype(np.float32)


# --------------------------------------------------------------------------
# Sec. IV-C: Clustering Unit (mid-point boundaries, half-open intervals)
# --------------------------------------------------------------------------
def cluster_boundaries(cb_a: np.ndarray, b_a: int) -> np.ndarray:
    """b_c = (c_c + c_{c+1}) / 2 for adjacent centroids, in fp32."""
    c = np.asarray(cb_a, dtype=np.float16)[: 1 << b_a].astype(np.float32)
    if not np.all(c[1:] > c[:-1]):
        raise ValueError("activation codebook must be strictly ascending")
    return ((c[:-1] + c[1:]) * np.float32(0.5)).astype(np.float32)


def cluster(x: np.ndarray, t: np.ndarray, cb_a: np.ndarray, b_a: int) -> np.ndarray:
    """Activation index of every channel (outliers included, Sec. III-C1).

    The token's centroids are t * C_A, so its boundaries are t * b_c.  A value
    in [t*b_{c-1}, t*b_c) belongs to cluster c; the index equals the number of
    scaled boundaries that are <= x.
    """
    x32 = np.asarray(x, dtype=np.float16).astype(np.float32)
    bnd = cluster_boundaries(cb_a, b_a)
    t32 = np.asarray(t, dtype=np.float32)
    out = np.zeros(x32.shape, dtype=np.uint8)
    for c in range(bnd.size):
        scaled = (t32 * bnd[c]).astype(np.float32)          # fp32 product
        out += (x32 >= scaled[:, None]).astype(np.uint8)
    return out


# --------------------------------------------------------------------------
# Sec. IV-D: dynamic top-k outlier detection (k largest and k smallest)
# --------------------------------------------------------------------------
def topk_lists(x: np.ndarray, k: int) -> Tuple[np.ndarray, np.ndarray]:
    """Max list and min list of every token, in pop order, ties to lower index.

    The max list is the first k channels of a stable sort by value descending;
    the min list the first k of a stable sort by value ascending.  -0 and +0
    compare equal.
    """
    x64 = np.asarray(x, dtype=np.float16).astype(np.float64)
    if not np.all(np.isfinite(x64)):
        raise ValueError("activations must be finite")
    if k < 0 or k > x64.shape[1]:
        raise ValueError("k out of range")
    mx = np.argsort(-x64, axis=1, kind="stable")[:, :k].astype(np.int32)
    mn = np.argsort(x64, axis=1, kind="stable")[:, :k].astype(np.int32)
    return mx, mn


class Orizuru:
    """Literal emulation of the two-fold binary tree of Sec. IV-D.

    Heap numbering: root is node 1, internal nodes 1..M-1, leaves M..2M-1
    (leaf M+e holds element e).  M is N rounded up to a power of two; padded
    leaves are unavailable in both trees from the start.  A node's bit selects
    its left (0) or right (1) child.  The max tree takes the right child only
    if its value is strictly larger, the min tree only if strictly smaller, so
    ties go left in both (reading of "reversed comparison results": the
    operands of the strict comparison are swapped).  A popped element is
    masked (acts as -inf in the max tree, +inf in the min tree) and only the
    ancestors of its leaf are re-evaluated, one comparison per level.
    """

    def __init__(self, values):
        self.x = [float(v) for v in values]
        n = len(self.x)
        self.n = n
        self.M = 1 << max(1, math.ceil(math.log2(max(n, 2))))
        self.L = int(math.log2(self.M))
        self.avail_p = [e < n for e in range(self.M)]
        self.avail_q = [e < n for e in range(self.M)]
        self.p = [0] * self.M      # max-tree bits, index = node number
        self.q = [0] * self.M      # min-tree bits
        self.comparisons = 0
        self._init()

    # value presented by a node to its parent
    def _val(self, node: int, tree: str) -> float:
        M = self.M
        bits = self.p if tree == "p" else self.q
        avail = self.avail_p if tree == "p" else self.avail_q
        while node < M:
            node = 2 * node + bits[node]
        e = node - M
        if avail[e]:
            return self.x[e]
        return -math.inf if tree == "p" else math.inf

    def _compare(self, node: int, tree: str) -> None:
        left = self._val(2 * node, tree)
        right = self._val(2 * node + 1, tree)
        self.comparisons += 1
        if tree == "p":
            self.p[node] = 1 if right > left else 0
        else:
            self.q[node] = 1 if right < left else 0

    def _init(self) -> None:
        M = self.M
        # leaf level of the max tree: nodes M/2 .. M-1, N/2 comparisons
        for node in range(M // 2, M):
            self._compare(node, "p")
        # the min tree reuses those comparisons (operands swapped) where both
        # leaves are real; pairs touching padding are decided by availability
        for node in range(M // 2, M):
            e_l, e_r = 2 * node - M, 2 * node + 1 - M
            if e_l < self.n and e_r < self.n:
                xl, xr = self.x[e_l], self.x[e_r]
                self.q[node] = 1 if xr < xl else 0
            else:
                self._compare(node, "q")
        # remaining levels, bottom-up, for both trees
        for level_start in [M >> s for s in range(2, self.L + 1)]:
            for node in range(level_start, 2 * level_start):
                self._compare(node, "p")
        for level_start in [M >> s for s in range(2, self.L + 1)]:
            for node in range(level_start, 2 * level_start):
                self._compare(node, "q")

    def _path(self, tree: str) -> Tuple[int, str]:
        bits = self.p if tree == "p" else self.q
        node, path = 1, ""
        while node < self.M:
            path += str(bits[node])
            node = 2 * node + bits[node]
        return node, path

    def pop(self, tree: str) -> Tuple[int, str]:
        """Pop the root's element; returns (leaf node number, path bits)."""
        leaf, path = self._path(tree)
        e = leaf - self.M
        (self.avail_p if tree == "p" else self.avail_q)[e] = False
        node = leaf // 2
        while node >= 1:
            self._compare(node, tree)
            node //= 2
        return leaf, path

    def topk(self, k: int) -> Tuple[List[int], List[int]]:
        mx = [self.pop("p")[0] - self.M for _ in range(k)]
        mn = [self.pop("q")[0] - self.M for _ in range(k)]
        return mx, mn


# --------------------------------------------------------------------------
# Sec. III-C: look-ahead residuals of the outliers
# --------------------------------------------------------------------------
def inlier_scale(x: np.ndarray, max_idx: np.ndarray, min_idx: np.ndarray) -> np.ndarray:
    """R13: t_i = max |x_ip| over the channels in neither list (0 if none)."""
    xv = np.asarray(x, dtype=np.float16).astype(np.float64)
    n, K = xv.shape
    t = np.zeros(n, dtype=np.float32)
    for i in range(n):
        listed = set(int(p) for p in max_idx[i] if p >= 0) | \
            set(int(p) for p in min_idx[i] if p >= 0)
        rest = [abs(xv[i, p]) for p in range(K) if p not in listed]
        t[i] = np.float32(max(rest)) if rest else np.float32(0.0)
    return t


def dequant_act(a: np.ndarray, t: np.ndarray, cb_a: np.ndarray) -> np.ndarray:
    """x_hat = fp32(t * C_A[a]): exact, the product of two fp16 values."""
    ca = np.asarray(cb_a, dtype=np.float16).astype(np.float32)
    return (np.asarray(t, dtype=np.float32)[:, None] * ca[a]).astype(np.float32)


def residuals(x: np.ndarray, t: np.ndarray, a: np.ndarray, cb_a: np.ndarray,
              max_idx: np.ndarray, min_idx: np.ndarray) -> np.ndarray:
    """Residual of every listed outlier: its fp16 value minus its quantized value.

    Layout [n][2k]: the max list's residuals, then the min list's.  A min-list
    channel that also appears in the token's max list gets residual 0 so the
    union of the two lists is compensated exactly once.
    """
    n, k = max_idx.shape
    x32 = np.asarray(x, dtype=np.float16).astype(np.float32)
    xh = dequant_act(a, t, cb_a)
    r = np.zeros((n, 2 * k), dtype=np.float32)
    for i in range(n):
        in_max = set(int(p) for p in max_idx[i] if p >= 0)
        for e in range(k):
            p = int(max_idx[i, e])
            if p >= 0:                      # -1: an unused place (R12)
                r[i, e] = np.float32(x32[i, p] - xh[i, p])
        for e in range(k):
            p = int(min_idx[i, e])
            if p >= 0:
                r[i, k + e] = np.float32(0.0) if p in in_max else np.float32(x32[i, p] - xh[i, p])
    return r


# --------------------------------------------------------------------------
# Sec. III-B: WAQ LUT-GEMM (concatenate, count, weighted sum)
# --------------------------------------------------------------------------
def lut_gemm(a: np.ndarray, w_idx: np.ndarray, lut: np.ndarray, t: np.ndarray,
             s_w: np.ndarray, b_w: int, tokens=None) -> np.ndarray:
    """Y*[i, j] = t_i * s_j * sum_p LUT[(a_ip << b_w) | w_pj]  (fp64 sum).

    Step 1 concatenates the two indices of every (p, j) pair, step 3 fetches
    the LUT entry the concatenated index selects and reduces along the input
    channels.  `tokens` restricts the computation to a subset of rows.
    """
    rows = range(a.shape[0]) if tokens is None else tokens
    lut64 = np.asarray(lut, dtype=np.float32).astype(np.float64)
    w = np.asarray(w_idx, dtype=np.uint8)
    out = np.zeros((len(rows), w.shape[1]), dtype=np.float64)
    for r, i in enumerate(rows):
        acc = np.zeros(w.shape[1], dtype=np.float64)
        for p in range(w.shape[0]):
            concat = (int(a[i, p]) << b_w) | w[p].astype(np.intp)
            acc += lut64[concat]
        out[r] = float(t[i]) * np.asarray(s_w, dtype=np.float64) * acc
    return out


def lut_gemm_counts(a: np.ndarray, w_idx: np.ndarray, lut: np.ndarray, t: np.ndarray,
                    s_w: np.ndarray, b_a: int, b_w: int) -> np.ndarray:
    """Same product through the count formulation (Sec. III-B, Sec. IV-B).

    For every output (i, j) the concatenated indices are counted (the Index
    Counter's one-hot decode + row sums) and the reduction becomes a weighted
    sum of the 2^(n_A+n_W) LUT entries with the counts as weights.
    """
    n, K = a.shape
    N = w_idx.shape[1]
    nbins = 1 << (b_a + b_w)
    lut64 = np.asarray(lut, dtype=np.float32).astype(np.float64)
    out = np.zeros((n, N), dtype=np.float64)
    for i in range(n):
        for j in range(N):
            concat = (a[i].astype(np.int64) << b_w) | w_idx[:, j].astype(np.int64)
            onehot = np.zeros((nbins, K), dtype=np.int64)
            onehot[concat, np.arange(K)] = 1
            counts = onehot.sum(axis=1)
            out[i, j] = float(t[i]) * float(s_w[j]) * float(np.dot(counts, lut64[:nbins]))
    return out


def dequant_matmul(a: np.ndarray, w_idx: np.ndarray, cb_a: np.ndarray, cb_w: np.ndarray,
                   t: np.ndarray, s_w: np.ndarray) -> np.ndarray:
    """Conventional path: dequantize both operands, then a plain matmul (fp64)."""
    xh = np.asarray(t, dtype=np.float64)[:, None] * \
        np.asarray(cb_a, dtype=np.float16).astype(np.float64)[a]
    wh = np.asarray(cb_w, dtype=np.float16).astype(np.float64)[w_idx] * \
        np.asarray(s_w, dtype=np.float64)[None, :]
    return xh @ wh


# --------------------------------------------------------------------------
# R14: per-output-channel weight codebooks
# --------------------------------------------------------------------------
def build_lut_percol(cb_a: np.ndarray, cb_w_cols: np.ndarray, b_a: int, b_w: int) -> np.ndarray:
    """lut[j][(a << b_w) | w] = fp32(C_A[a]) * fp32(C_W[j][w]) for every column j."""
    ca = np.asarray(cb_a, dtype=np.float16)[: 1 << b_a].astype(np.float32)
    cw = np.asarray(cb_w_cols, dtype=np.float16)[:, : 1 << b_w].astype(np.float32)
    out = np.zeros((cw.shape[0], 1 << (b_a + b_w)), dtype=np.float32)
    for j in range(cw.shape[0]):
        for a_ in range(1 << b_a):
            for w in range(1 << b_w):
                out[j, (a_ << b_w) | w] = ca[a_] * cw[j, w]
    return out


def lut_gemm_percol(a: np.ndarray, w_idx: np.ndarray, lut_cols: np.ndarray, t: np.ndarray,
                    s_w: np.ndarray, b_w: int, tokens=None) -> np.ndarray:
    """Y*[i, j] = t_i * s_j * sum_p lut_j[(a_ip << b_w) | w_pj]: every column
    looks its concatenated indices up in its own LUT slice (fp64 sum)."""
    rows = range(a.shape[0]) if tokens is None else tokens
    lut64 = np.asarray(lut_cols, dtype=np.float32).astype(np.float64)
    w = np.asarray(w_idx, dtype=np.intp)
    cols = np.arange(w.shape[1])
    out = np.zeros((len(rows), w.shape[1]), dtype=np.float64)
    for r, i in enumerate(rows):
        acc = np.zeros(w.shape[1], dtype=np.float64)
        for p in range(w.shape[0]):
            acc += lut64[cols, (int(a[i, p]) << b_w) | w[p]]
        out[r] = float(t[i]) * np.asarray(s_w, dtype=np.float64) * acc
    return out


def dequant_weights_percol(w_idx: np.ndarray, cb_w_cols: np.ndarray,
                           s_w: np.ndarray) -> np.ndarray:
    """w_hat[p, j] = s_j * C_W[j][w_pj] (fp64)."""
    cw = np.asarray(cb_w_cols, dtype=np.float16).astype(np.float64)
    w = np.asarray(w_idx, dtype=np.intp)
    return cw[np.arange(w.shape[1])[None, :], w] * np.asarray(s_w, dtype=np.float64)[None, :]


def outlier_compensate_percol(max_idx: np.ndarray, min_idx: np.ndarray, r: np.ndarray,
                              w_idx: np.ndarray, cb_w_cols: np.ndarray, s_w: np.ndarray,
                              tokens=None) -> np.ndarray:
    """Y'[i, j] = sum over listed outliers p of r_ip * s_j * C_W[j][w_pj] (fp64)."""
    n, k = max_idx.shape
    rows = range(n) if tokens is None else tokens
    cw = np.asarray(cb_w_cols, dtype=np.float16).astype(np.float64)
    s = np.asarray(s_w, dtype=np.float64)
    cols = np.arange(w_idx.shape[1])
    out = np.zeros((len(rows), w_idx.shape[1]), dtype=np.float64)
    for rr, i in enumerate(rows):
        chans = list(max_idx[i]) + list(min_idx[i])
        for e, p in enumerate(chans):
            if r[i, e] != 0:
                out[rr] += float(r[i, e]) * cw[cols, w_idx[int(p)].astype(np.intp)] * s
    return out


def forward_percol(x, w_idx, cb_w_cols, s_w, cb_a, b_a: int, b_w: int, k: int,
                   mode: int = SCALE_ABSMAX, tokens=None) -> Dict[str, np.ndarray]:
    """The whole path with per-column weight codebooks (R14)."""
    q = quantize_act(x, cb_a, b_a, k, mode)
    lut = build_lut_percol(cb_a, cb_w_cols, b_a, b_w)
    ys = lut_gemm_percol(q["a"], w_idx, lut, q["t"], s_w, b_w, tokens=tokens)
    yc = outlier_compensate_percol(q["max_idx"], q["min_idx"], q["residual"], w_idx,
                                   cb_w_cols, s_w, tokens=tokens)
    q.update({"lut": lut, "y_star": ys, "y_comp": yc, "y": ys + yc})
    return q


# --------------------------------------------------------------------------
# Sec. III-C2: error compensation of the outliers
# --------------------------------------------------------------------------
def outlier_compensate(max_idx: np.ndarray, min_idx: np.ndarray, r: np.ndarray,
                       w_idx: np.ndarray, cb_w: np.ndarray, s_w: np.ndarray,
                       tokens=None) -> np.ndarray:
    """Y'[i, j] = sum over listed outliers p of r_ip * s_j * C_W[w_pj]  (fp64).

    Each outlier's channel index fetches one input channel (a row) of the
    weight index matrix, which is dequantized and scaled by the residual.
    """
    n, k = max_idx.shape
    rows = range(n) if tokens is None else tokens
    cw = np.asarray(cb_w, dtype=np.float16).astype(np.float64)
    s = np.asarray(s_w, dtype=np.float64)
    out = np.zeros((len(rows), w_idx.shape[1]), dtype=np.float64)
    for rr, i in enumerate(rows):
        chans = list(max_idx[i]) + list(min_idx[i])
        for e, p in enumerate(chans):
            if r[i, e] != 0:
                out[rr] += float(r[i, e]) * cw[w_idx[int(p)]] * s
    return out


# --------------------------------------------------------------------------
# The whole hot path for one linear layer
# --------------------------------------------------------------------------
def quantize_act(x: np.ndarray, cb_a: np.ndarray, b_a: int, k: int,
                 mode: int = SCALE_ABSMAX) -> Dict[str, np.ndarray]:
    """Per-token scale, activation indices, outlier lists and residuals."""
    mx, mn = topk_lists(x, k)
    t = inlier_scale(x, mx, mn) if mode == SCALE_INLIER else act_scale(x, mode)
    a = cluster(x, t, cb_a, b_a)
    r = residuals(x, t, a, cb_a, mx, mn)
    return {"t": t, "a": a, "max_idx": mx, "min_idx": mn, "residual": r}


def static_lists(x: np.ndarray, thr_hi: float, thr_lo: float,
                 k: int) -> Tuple[np.ndarray, np.ndarray]:
    """OASIS-S outlier lists (R12): channels at or beyond the fixed thresholds,
    in channel order, at most k per side, -1 in the places left."""
    xv = np.asarray(x, dtype=np.float16).astype(np.float64)
    hi, lo = float(np.float32(thr_hi)), float(np.float32(thr_lo))
    n = xv.shape[0]
    mx = np.full((n, k), -1, dtype=np.int32)
    mn = np.full((n, k), -1, dtype=np.int32)
    for i in range(n):
        up = [p for p in range(xv.shape[1]) if xv[i, p] >= hi][:k]
        dn = [p for p in range(xv.shape[1]) if xv[i, p] <= lo][:k]
        mx[i, :len(up)] = up
        mn[i, :len(dn)] = dn
    return mx, mn


def quantize_act_static(x: np.ndarray, cb_a: np.ndarray, b_a: int, k: int, thr_hi: float,
                        thr_lo: float, mode: int = SCALE_ABSMAX) -> Dict[str, np.ndarray]:
    """OASIS-S: scale and indices as in quantize_act, lists from fixed thresholds."""
    mx, mn = static_lists(x, thr_hi, thr_lo, k)
    t = inlier_scale(x, mx, mn) if mode == SCALE_INLIER else act_scale(x, mode)
    a = cluster(x, t, cb_a, b_a)
    r = residuals(x, t, a, cb_a, mx, mn)
    return {"t": t, "a": a, "max_idx": mx, "min_idx": mn, "residual": r}


def forward(x, w_idx, cb_w, s_w, cb_a, b_a: int, b_w: int, k: int,
            mode: int = SCALE_ABSMAX, tokens=None, thresholds=None) -> Dict[str, np.ndarray]:
    """Look-ahead LUT-GEMM plus error compensation: Y = Y* + Y' (Sec. III-C);
    thresholds = (thr_hi, thr_lo) selects OASIS-S lists (R12)."""
    q = quantize_act(x, cb_a, b_a, k, mode) if thresholds is None else \
        quantize_act_static(x, cb_a, b_a, k, thresholds[0], thresholds[1], mode)
    lut = build_lut(cb_a, cb_w, b_a, b_w)
    ys = lut_gemm(q["a"], w_idx, lut, q["t"], s_w, b_w, tokens=tokens)
    yc = outlier_compensate(q["max_idx"], q["min_idx"], q["residual"], w_idx, cb_w, s_w,
                            tokens=tokens)
    q.update({"lut": lut, "y_star": ys, "y_comp": yc, "y": ys + yc})
    return q


# --------------------------------------------------------------------------
# Packing of the index tensors exchanged with the library (oracle's own code)
# --------------------------------------------------------------------------
def pack_act_indices(a: np.ndarray) -> np.ndarray:
    """[n][K] indices -> [n][K/2] bytes, channel 2q in the low nibble of byte q."""
    a = np.asarray(a, dtype=np.uint8)
    return (a[:, 0::2] | (a[:, 1::2] << 4)).astype(np.uint8)


def unpack_act_indices(packed: np.ndarray, K: int) -> np.ndarray:
    p = np.asarray(packed, dtype=np.uint8)
    out = np.zeros((p.shape[0], K), dtype=np.uint8)
    out[:, 0::2] = p & 0xF
    out[:, 1::2] = p >> 4
    return out


def pack_weight_indices(w_idx: np.ndarray) -> np.ndarray:
    """[K][N] indices -> [K/8][N] 32-bit words; channel 8b+e at bits 4e..4e+3."""
    w = np.asarray(w_idx, dtype=np.uint32)
    K, N = w.shape
    out = np.zeros((K // 8, N), dtype=np.uint32)
    for e in range(8):
        out |= w[e::8, :] << np.uint32(4 * e)
    return out


def pack_weight_rows(w_idx: np.ndarray) -> np.ndarray:
    """[K][N] indices -> [K][ceil(N/8)] 32-bit words; column 8m+c of row p at
    bits 4c..4c+3 of word (p, m), zero past N (one input channel per row)."""
    w = np.asarray(w_idx, dtype=np.uint32)
    K, N = w.shape
    Np = (N + 7) // 8 * 8
    wp = np.zeros((K, Np), dtype=np.uint32)
    wp[:, :N] = w
    out = np.zeros((K, Np // 8), dtype=np.uint32)
    for c in range(8):
        out |= wp[:, c::8] << np.uint32(4 * c)
    return out


# --------------------------------------------------------------------------
# Table I / Sec. II-B: closed-form cost of the LUT schemes
# --------------------------------------------------------------------------
def cost_model(K: int, N: int, n_a: int, n_w: int, mu: int = 4) -> Dict[str, float]:
    """LUT size, group size and reduction FLOPs of the WOQ and WAQ LUT schemes."""
    return {
        "woq_lut_size": (2 ** mu) * K / mu,
        "waq_lut_size": 2 ** (n_a + n_w),
        "woq_group": mu,
        "waq_group": K,
        "woq_reduction_flops": (K / mu) * n_w * N,
        "waq_reduction_flops": (2 ** (n_a + n_w)) * N,
    }
