"""Benchmark of the OASIS hot path on one MI355X.

A step is one pass of the whole path over one synthetic layer: build the LUT
block and quantize the activations (scale, codes, top-k outliers, residuals)
in one launch, then the LUT-GEMM and the outlier compensation (one fused call
for few tokens; --path selects the schedule).  (Building the LUT block on a
second stream, overlapping the previous step, was slower: the cross-stream
waits inside the graph cost more than the 1.7 us launch they hide; building
it inside the quantize launch removes that launch.)
Inputs are resident in HBM when timing starts; the weight codes are rotated
over enough copies (> 512 MiB in total) that the 256 MiB last-level cache
cannot serve them.  The timed steps are captured once into one HIP graph and
replayed (no host launch gaps); per-call durations come from HIP events
around back-to-back launches of each call, queued behind a spin kernel so
that every launch is waiting before the GPU gets to it.

With no arguments the line is the largest layer: 4096 tokens x 8192 x 28672
(prefill, k = 64 per side), with the decode of 16 tokens through the same
weights as its "decode" part.  --config NAME times one other layer.

Prints ONE JSON line (rank 0).
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import re
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "effective TOPS (2*n*d_in*d_out/s) + HBM GB/s, % of roofline, at decode & prefill"
HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0


def gemm_bytes(n, d_in, d_out, k=0, merge=True):
    """Algorithmic HBM bytes of one main-branch launch: weight codes (0.5 B
    each), activation codes (0.5 B each), both scale vectors, Y written once
    (read too when the GEMM merges into a compensation term written before
    it), and with k > 0 the outlier lists and residuals it compensates from
    (the weight rows those need are rows the same launch streams anyway)."""
    y = (8 if merge else 4) * n * d_out
    return d_in * d_out // 2 + n * d_in // 2 + 4 * n + 4 * d_out + y + 16 * n * k


def step_bytes(n, d_in, d_out, k, fused):
    """Algorithmic HBM bytes of one whole step (LUT block ignored: 1 KiB)."""
    quant = 2 * n * d_in + n * d_in // 2 + 4 * n + 16 * n * k       # x in; codes, t, lists out
    if fused:
        return quant + gemm_bytes(n, d_in, d_out, k, merge=False)
    comp = 16 * n * k + 2 * n * k * d_out // 2 + 4 * d_out + 4 * n * d_out
    return quant + comp + gemm_bytes(n, d_in, d_out)


def call_bytes(n, d_in, d_out, k, path):
    """Algorithmic HBM bytes per launch of every call of the path."""
    x, codes = 2 * n * d_in, n * d_in // 2
    lists = 16 * n * k                       # two int32 lists + 2k fp32 residuals
    # outlier branch: one input channel of the index matrix (d_out/2 bytes) per
    # listed outlier, the lists, the scales, y written (read too if merging)
    comp_y = (8 if path == "lookahead" else 4) * n * d_out
    comp = 2 * n * k * d_out // 2 + lists + 4 * d_out + comp_y
    return {
        "build_lut": 2 * 32 + 1088,
        "quantize_act": x + codes + 4 * n + lists,
        "build_lut_quantize_act": x + codes + 4 * n + lists + 1088,
        "build_lut_quantize_act_static": x + codes + 4 * n + lists + 1088,
        "quantize_act_static": x + codes + 4 * n + lists,
        "cluster_act": x + codes + 4 * n,
        "detect_outliers": x + lists,
        "outlier_compensate": comp,
        "lut_gemm": gemm_bytes(n, d_in, d_out, merge=path == "separate"),
        "lut_gemm_compensated": gemm_bytes(n, d_in, d_out, k, merge=False),
        # the row-layout copy of a listed channel, where the launch reads it,
        # duplicates codes the operation needs once: not counted
        "lut_gemm_compensated_rows": gemm_bytes(n, d_in, d_out, k, merge=False),
        # the compacted lists' rows are part of comp; y written by the lists'
        # kernel and merged by the GEMM
        "lut_gemm_compensated_split": gemm_bytes(n, d_in, d_out) + comp - 4 * d_out,
        # + the columns' own codebooks (16 fp16 each)
        "lut_gemm_compensated_percol": gemm_bytes(n, d_in, d_out, k, merge=False) + 32 * d_out,
    }


KERNEL_SOURCES = {
    "build_lut": ["lut.hip"],
    "quantize_act": ["quantize.hip"], "cluster_act": ["quantize.hip"],
    "build_lut_quantize_act": ["quantize.hip"], "quantize_act_static": ["quantize.hip"],
    "build_lut_quantize_act_static": ["quantize.hip"],
    "detect_outliers": ["quantize.hip"],
    "outlier_compensate": ["compensate.hip", "split.hip", "lut_gemm.hip"],
    "lut_gemm": ["lut_gemm.hip"], "lut_gemm_compensated": ["lut_gemm.hip", "compensate.hip"],
    "lut_gemm_compensated_rows": ["lut_gemm.hip", "compensate.hip"],
    "lut_gemm_compensated_split": ["lut_gemm.hip", "compensate.hip", "split.hip"],
    "lut_gemm_compensated_percol": ["lut_gemm.hip"],
}


def source_digest(call):
    """sha256 of the HIP sources a call's kernels are built from (+ common.h)."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[call] + ["common.h"]:
        with open(os.path.join(ROOT, "paper_2507_23035_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(call, workload):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE
    summary, scaled by the copy-kernel calibration; None if there is none or
    the kernel source changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path)).get(f"{call}|{workload}")
    if not rec or rec.get("source_sha256") != source_digest(call):
        return None
    return rec.get("hbm_bytes_per_launch")


CALL_SYMBOLS = {   # kernel symbol fragment of each call's dominant kernel
    "build_lut": "k_build_lut", "quantize_act": "k_quantize<", "cluster_act": "k_quantize<",
    "build_lut_quantize_act": "k_quantize<", "quantize_act_static": "k_quantize<",
    "build_lut_quantize_act_static": "k_quantize<",
    "detect_outliers": "k_quantize<", "outlier_compensate": "k_compensate",
    "lut_gemm": "k_gemm_mfma", "lut_gemm_compensated": "k_gemm_mfma",
    "lut_gemm_compensated_rows": "k_gemm_mfma",
    "lut_gemm_compensated_split": "k_gemm_mfma",
    "lut_gemm_compensated_percol": "k_gemm_mfma",
}


def _pmc_rows(d, counter):
    import csv
    import glob
    rows = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        rows += [r for r in csv.DictReader(open(f)) if r.get("Counter_Name") == counter]
    return rows


def summarize_pmc(root, workload, path):
    """Turn four rocprofv3 --pmc runs (subdirectories fetch/, write/ of the
    bench, cal_fetch/, cal_write/ of --calibrate-copy) into per-launch HBM
    bytes for every call of the path, written to profiles/traffic.json."""
    cal = {}
    for c, sub in (("FETCH_SIZE", "cal_fetch"), ("WRITE_SIZE", "cal_write")):
        vals = [float(r["Counter_Value"]) for r in _pmc_rows(os.path.join(root, sub), c)]
        cal[c] = max(vals) / float(256 << 20)      # counter units per byte (copy of 256 MiB)
    out_path = os.path.join(ROOT, "profiles", "traffic.json")
    db = json.load(open(out_path)) if os.path.exists(out_path) else {}
    lines = [f"| call | kernel | dispatches | FETCH_SIZE | WRITE_SIZE | HBM bytes/launch |",
             "|---|---|---|---|---|---|"]
    names = {"fused": ["build_lut_quantize_act", "lut_gemm_compensated_rows"],
             "split": ["build_lut_quantize_act", "lut_gemm"],
             "separate": ["build_lut_quantize_act", "outlier_compensate", "lut_gemm"],
             "lookahead": ["cluster_act", "detect_outliers", "lut_gemm",
                           "outlier_compensate"]}[path]
    for call in names:
        sym = CALL_SYMBOLS[call]
        vals = {}
        for c, sub in (("FETCH_SIZE", "fetch"), ("WRITE_SIZE", "write")):
            rs = [r for r in _pmc_rows(os.path.join(root, sub), c) if sym in r["Kernel_Name"]]
            if call == "lut_gemm":  # the main-branch kernel alone: a tile kernel's value
                # operand and heavy-block variants (5th and 6th template arguments) are not
                rs = [r for r in rs if not re.search(
                    r"k_gemm_mfma_tile<\d+, \d+, \d+, \d+, (true, \w+|\w+, true)",
                    r["Kernel_Name"])]
            if call in ("cluster_act", "detect_outliers", "quantize_act",
                        "build_lut_quantize_act"):
                want = {"cluster_act": "true, false", "detect_outliers": "false, true",
                        "quantize_act": "true, true", "build_lut_quantize_act": "true, true"}[call]
                rs = [r for r in rs if want in r["Kernel_Name"]]
            vals[c] = (len(rs), sum(float(r["Counter_Value"]) for r in rs) / max(1, len(rs)))
        if not vals["FETCH_SIZE"][0]:
            continue
        hbm = vals["FETCH_SIZE"][1] / cal["FETCH_SIZE"] + vals["WRITE_SIZE"][1] / cal["WRITE_SIZE"]
        db[f"{call}|{workload}"] = {"source_sha256": source_digest(call),
                                    "fetch_counter": vals["FETCH_SIZE"][1],
                                    "write_counter": vals["WRITE_SIZE"][1],
                                    "copy_factor_fetch": cal["FETCH_SIZE"],
                                    "copy_factor_write": cal["WRITE_SIZE"],
                                    "hbm_bytes_per_launch": round(hbm)}
        lines.append(f"| {call} | {sym} | {vals['FETCH_SIZE'][0]} | {vals['FETCH_SIZE'][1]:.1f} "
                     f"| {vals['WRITE_SIZE'][1]:.1f} | {hbm:.0f} |")
    with open(out_path, "w") as fh:
        json.dump(db, fh, indent=1, sort_keys=True)
    print(f"copy calibration: FETCH_SIZE {cal['FETCH_SIZE']:.6g} and WRITE_SIZE "
          f"{cal['WRITE_SIZE']:.6g} counter units per byte")
    print("\n".join(lines))


def calibrate_copy(mib):
    """A plain device copy of known size (the counter calibration run)."""
    import torch
    nbytes = mib << 20
    a = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(10):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "copy", "bytes_read_per_copy": nbytes,
                      "bytes_written_per_copy": nbytes, "copies": 10}), flush=True)


_CPU = {}   # the layer the forked oracle workers read (set before the pool forks)


def _oracle_tokens(sl):
    """Oracle forward of tokens sl[0]:sl[1] of the layer (one worker, one thread)."""
    from threadpoolctl import threadpool_limits
    from oracle import oasis_oracle as O
    L, mode, cols = _CPU["layer"], _CPU["mode"], _CPU["cols"]
    s = L.spec
    x = L.x[sl[0]:sl[1]]
    with threadpool_limits(limits=1):
        if cols is None:
            O.forward(x, L.w_idx, L.cb_w, L.s_w, L.cb_a, s.b_a, s.b_w, s.k, mode=mode)
        else:
            O.forward_percol(x, L.w_idx, cols, L.s_w, L.cb_a, s.b_a, s.b_w, s.k, mode=mode)
    return sl[1] - sl[0]


def cpu_baseline(layer, mode=0, cols=None, max_procs=16, per_proc=8, single=8):
    """The oracle's forward (quantize, LUT-GEMM, compensation; numpy) timed on
    the host, on a bounded sample: the first tokens of the layer (at most
    per_proc per worker), each token a whole row of the output.  All cores:
    one single-threaded worker process per core (at most max_procs), median
    of 3 runs; one thread: `single` tokens, once.  Run before the GPU is touched (the
    workers are forked).  Rates are effective TOPS over the sampled tokens."""
    import multiprocessing as mp
    s = layer.spec
    _CPU.update(layer=layer, mode=mode, cols=cols)
    procs = max(1, min(max_procs, os.cpu_count() or 1, s.n))
    ntok = min(s.n, procs * per_proc)
    per = -(-ntok // procs)
    chunks = [(i, min(ntok, i + per)) for i in range(0, ntok, per)]
    runs = []
    ctx = mp.get_context("fork")
    with ctx.Pool(procs) as pool:
        for _ in range(3):
            t0 = time.perf_counter()
            done = sum(pool.map(_oracle_tokens, chunks))
            runs.append(time.perf_counter() - t0)
    el = sorted(runs)[1]
    ops = 2.0 * done * s.d_in * s.d_out
    ns = min(s.n, single)
    t0 = time.perf_counter()
    _oracle_tokens((0, ns))
    el1 = time.perf_counter() - t0
    whole = "the whole layer" if done == s.n else f"{done} of {s.n} tokens (extrapolates linearly)"
    return {"value": round(ops / el / 1e12, 6), "unit": "effective TOPS", "cores": procs,
            "kind": "oracle",
            "sample": f"{s.name}: oracle forward (numpy, fp64) of {whole}, {procs} worker "
                      f"processes of one thread, {per} tokens each, median of 3 runs "
                      f"({el:.2f} s); one thread: {ns} tokens in {el1:.2f} s",
            "single_thread_value": round(2.0 * ns * s.d_in * s.d_out / el1 / 1e12, 6)}


def layer_spec(args, name):
    """The spec of layer `name` with the variant options applied."""
    from paper_2507_23035_amd import synth
    spec = synth.config(name)
    if args.bits_a and args.bits_a != spec.b_a:
        spec = dataclasses.replace(spec, b_a=args.bits_a, name=f"{spec.name}_a{args.bits_a}")
    if args.scale == "inlier":
        spec = dataclasses.replace(spec, name=f"{spec.name}_inlier")
    if args.percol:
        spec = dataclasses.replace(spec, name=f"{spec.name}_percol")
    if args.oasis_s:
        spec = dataclasses.replace(spec, name=f"{spec.name}_oasis_s")
    return spec


class Weights:
    """Device copies of one layer's weight codes (both layouts), rotated over
    enough copies that the last-level cache cannot serve them; shared by the
    layers with the same weights."""

    def __init__(self, layer, copies, dev):
        import torch
        from paper_2507_23035_amd import oasis
        d_in, d_out = layer.w_idx.shape
        wbytes = d_in * d_out // 2
        self.copies = copies or max(1, min(64, (512 << 20) // wbytes + 1))
        packed = oasis.pack_weight_indices(layer.w_idx).view(np.int32)
        self.idx_w = [torch.from_numpy(packed).to(dev) for _ in range(self.copies)]
        rows = oasis.pack_weight_rows(layer.w_idx).view(np.int32)
        self.idx_wr = [torch.from_numpy(rows).to(dev) for _ in range(self.copies)]
        self.s_w = torch.from_numpy(layer.s_w).to(dev)


def run_workload(args, layer, weights, dev, side):
    """Time one layer's step (graph replay of `args.steps` steps) and every
    call of it; returns the fields of its JSON line."""
    import torch
    from paper_2507_23035_amd import oasis, synth
    s = layer.spec
    n, d_in, d_out, k, b_a, b_w = s.n, s.d_in, s.d_out, s.k, s.b_a, s.b_w
    scale = oasis.SCALE_INLIER if args.scale == "inlier" else oasis.SCALE_ABSMAX
    thr = None
    if args.oasis_s:   # thresholds at the k-th extremes; twice the places per side
        thr = synth.static_thresholds(layer, k)
        k = 2 * k
    algo = oasis.ALGO_MFMA if args.algo == "mfma" else oasis.ALGO_LUT
    copies, idx_w, idx_wr, s_w = weights.copies, weights.idx_w, weights.idx_wr, weights.s_w
    x = torch.from_numpy(layer.x.view(np.int16).copy()).to(dev)
    cb_a, cb_w = layer.cb_a, layer.cb_w
    lut = torch.empty(oasis.LUT_BLOCK_BYTES, dtype=torch.uint8, device=dev)
    q = {
        "idx_act": torch.empty((n, d_in // 2), dtype=torch.uint8, device=dev),
        "act_scale": torch.empty(n, dtype=torch.float32, device=dev),
        "max_idx": torch.empty((n, k), dtype=torch.int32, device=dev),
        "min_idx": torch.empty((n, k), dtype=torch.int32, device=dev),
        "residual": torch.empty((n, 2 * k), dtype=torch.float32, device=dev),
    }
    y = torch.empty((n, d_out), dtype=torch.float32, device=dev)
    # scratch of the split compensation (many tokens), allocated once
    ws = torch.empty(max(1, oasis.split_workspace_bytes(n, d_in, d_out, k)), dtype=torch.uint8,
                     device=dev)
    path = args.path
    if path == "auto":
        if (n <= 32 or args.percol) and algo == oasis.ALGO_MFMA:
            path = "fused"
        else:
            path = "split" if algo == oasis.ALGO_MFMA else "separate"
    # per-column codebooks (--percol): fp16 [d_out][16], entries past 2^b_w zero
    cols_dev = None
    if args.percol:
        cols_np = synth.percol_codebooks(layer)
        full = np.zeros((d_out, 16), dtype=np.float16)
        full[:, : cols_np.shape[1]] = cols_np
        cols_dev = torch.from_numpy(full.view(np.int16).copy()).to(dev)

    # Every call of the path, with the arguments the step uses (c = weight copy).
    calls = {
        "build_lut": lambda c: oasis.build_lut(cb_a, b_a, cb_w, b_w, out=lut),
        "quantize_act": lambda c: oasis.quantize_act(x, lut, b_a, k, scale, out=q),
        "build_lut_quantize_act": lambda c: oasis.build_lut_quantize_act(
            cb_a, b_a, cb_w, b_w, x, k, scale, lut=lut, out=q),
        "quantize_act_static": lambda c: oasis.quantize_act_static(x, lut, b_a, k, thr[0], thr[1],
                                                                   scale, out=q),
        "build_lut_quantize_act_static": lambda c: oasis.build_lut_quantize_act_static(
            cb_a, b_a, cb_w, b_w, x, k, thr[0], thr[1], scale, lut=lut, out=q),
        "cluster_act": lambda c: oasis.cluster_act(x, lut, b_a, out=q),
        "detect_outliers": lambda c: oasis.detect_outliers(x, lut, b_a, k, out=q),
        "outlier_compensate": lambda c: oasis.outlier_compensate_split(
            q["max_idx"], q["min_idx"], q["residual"], idx_w[c], idx_wr[c], lut, b_w, s_w, d_in,
            y=y, accumulate=False, workspace=ws),
        # adds into y only where the path merges there (the separate schedule);
        # the split and look-ahead schedules run it first, writing y
        "lut_gemm": lambda c: oasis.lut_gemm(q["idx_act"], q["act_scale"], idx_w[c], s_w, lut,
                                             b_a, b_w, algo, y=y,
                                             accumulate=path == "separate"),
        "lut_gemm_compensated": lambda c: oasis.lut_gemm_compensated(
            q["idx_act"], q["act_scale"], idx_w[c], s_w, lut, b_a, b_w, q["max_idx"],
            q["min_idx"], q["residual"], y=y),
        "lut_gemm_compensated_rows": lambda c: oasis.lut_gemm_compensated_rows(
            q["idx_act"], q["act_scale"], idx_w[c], idx_wr[c], s_w, lut, b_a, b_w, q["max_idx"],
            q["min_idx"], q["residual"], y=y),
        "lut_gemm_compensated_split": lambda c: oasis.lut_gemm_compensated_split(
            q["idx_act"], q["act_scale"], idx_w[c], idx_wr[c], s_w, lut, b_a, b_w, q["max_idx"],
            q["min_idx"], q["residual"], y=y, workspace=ws),
        "lut_gemm_compensated_percol": lambda c: oasis.lut_gemm_compensated_percol(
            q["idx_act"], q["act_scale"], idx_w[c], s_w, lut, cols_dev, b_a, b_w, q["max_idx"],
            q["min_idx"], q["residual"], y=y),
    }

    def fused_gemm(c, L, qq, yy=None):
        """The fused path's GEMM + compensation call."""
        if args.percol:
            return oasis.lut_gemm_compensated_percol(qq["idx_act"], qq["act_scale"], idx_w[c], s_w,
                                                     L, cols_dev, b_a, b_w, qq["max_idx"],
                                                     qq["min_idx"], qq["residual"], y=yy)
        return oasis.lut_gemm_compensated_rows(qq["idx_act"], qq["act_scale"], idx_w[c],
                                               idx_wr[c], s_w, L, b_a, b_w, qq["max_idx"],
                                               qq["min_idx"], qq["residual"], y=yy)
    if path == "fused":
        gemm_name = "lut_gemm_compensated_percol" if args.percol else "lut_gemm_compensated_rows"
        names = (["build_lut_quantize_act_static"] if thr else ["build_lut_quantize_act"]) + \
            [gemm_name]
    elif path == "lookahead":
        names = ["build_lut", "cluster_act", "detect_outliers", "lut_gemm", "outlier_compensate"]
        gemm_name = "lut_gemm"
    elif path == "split":
        # the step's two calls, then the main-branch GEMM and the split
        # compensation each on their own (what the GEMM call's kernels cost)
        names = (["build_lut_quantize_act_static"] if thr else ["build_lut_quantize_act"]) + \
            ["lut_gemm_compensated_split", "lut_gemm", "outlier_compensate"]
        gemm_name = "lut_gemm"
    else:
        names = (["build_lut_quantize_act_static"] if thr else ["build_lut_quantize_act"]) + \
            ["outlier_compensate", "lut_gemm"]
        gemm_name = "lut_gemm"

    def quantize(L):
        """LUT block + quantization in one launch (a second one for the inlier scale)."""
        if thr:
            oasis.build_lut_quantize_act_static(cb_a, b_a, cb_w, b_w, x, k, thr[0], thr[1], scale,
                                                lut=L, out=q)
        else:
            oasis.build_lut_quantize_act(cb_a, b_a, cb_w, b_w, x, k, scale, lut=L, out=q)

    def step(i):
        """Step i (weight copy i mod copies)."""
        c = i % copies
        main = torch.cuda.current_stream()
        L = lut
        if path == "fused":
            # the LUT block is rebuilt with every step (Sec. IV-A builds it once
            # per layer), inside the quantize launch
            quantize(L)
            fused_gemm(c, L, q, y)
        elif path == "split":
            quantize(L)
            oasis.lut_gemm_compensated_split(q["idx_act"], q["act_scale"], idx_w[c], idx_wr[c],
                                             s_w, L, b_a, b_w, q["max_idx"], q["min_idx"],
                                             q["residual"], y=y, workspace=ws)
        elif path == "lookahead":
            oasis.build_lut(cb_a, b_a, cb_w, b_w, out=L)
            # main branch and outlier detection run concurrently (Sec. III-C)
            side.wait_stream(main)
            with torch.cuda.stream(side):
                oasis.detect_outliers(x, L, b_a, k, out=q, stream=side)
            oasis.cluster_act(x, L, b_a, out=q)
            oasis.lut_gemm(q["idx_act"], q["act_scale"], idx_w[c], s_w, L, b_a, b_w, algo,
                           y=y, accumulate=False)
            main.wait_stream(side)
            oasis.outlier_compensate_split(q["max_idx"], q["min_idx"], q["residual"], idx_w[c],
                                           idx_wr[c], L, b_w, s_w, d_in, y=y, accumulate=True,
                                           workspace=ws)
        else:
            quantize(L)
            oasis.outlier_compensate_split(q["max_idx"], q["min_idx"], q["residual"], idx_w[c],
                                           idx_wr[c], L, b_w, s_w, d_in, y=y, accumulate=False,
                                           workspace=ws)
            oasis.lut_gemm(q["idx_act"], q["act_scale"], idx_w[c], s_w, L, b_a, b_w, algo, y=y,
                           accumulate=True)

    nsteps = args.steps

    def capture(count, first):
        """One HIP graph holding `count` consecutive steps (rotating weight copies)."""
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(first, first + count):
                step(i)
        return g

    # prime the library and the allocator outside capture
    for i in range(2):
        step(i)
    torch.cuda.synchronize()
    mode = "eager" if args.eager else "graph"
    if mode == "graph":
        try:
            g_warm = capture(args.warmup, 0) if args.warmup else None
            g_timed = capture(nsteps, args.warmup)
        except Exception as e:
            if args.verbose:
                print(f"graph capture failed ({e}); timing eager launches", file=sys.stderr)
            mode = "eager"
            torch.cuda.synchronize()

    # ---- timed region: exactly `nsteps` steps, wall clock, synchronized on both sides
    if mode == "graph":
        if g_warm is not None:
            g_warm.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        g_timed.replay()
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
    else:
        for i in range(args.warmup):
            step(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.warmup, args.warmup + nsteps):
            step(i)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0

    # ---- the schedule keeps every dependence: the last timed step's output
    # equals one eager, single-stream pass over the same weight copy (the
    # kernels are deterministic, so bit for bit)
    y_sched = y.clone()
    last = args.warmup + nsteps - 1
    c_last = last % copies
    oasis.build_lut(cb_a, b_a, cb_w, b_w, out=lut)
    q1 = oasis.quantize_act(x, lut, b_a, k, scale) if not thr else \
        oasis.quantize_act_static(x, lut, b_a, k, thr[0], thr[1], scale)
    if path == "fused":
        y_ref = fused_gemm(c_last, lut, q1)
    elif path == "split":
        y_ref = oasis.lut_gemm_compensated_split(q1["idx_act"], q1["act_scale"], idx_w[c_last],
                                                 idx_wr[c_last], s_w, lut, b_a, b_w,
                                                 q1["max_idx"], q1["min_idx"], q1["residual"],
                                                 workspace=ws)
    else:
        if path == "lookahead":
            y_ref = oasis.lut_gemm(q1["idx_act"], q1["act_scale"], idx_w[c_last], s_w, lut, b_a,
                                   b_w, algo)
            oasis.outlier_compensate_split(q1["max_idx"], q1["min_idx"], q1["residual"],
                                           idx_w[c_last], idx_wr[c_last], lut, b_w, s_w, d_in,
                                           y=y_ref, accumulate=True, workspace=ws)
        else:
            y_ref = oasis.outlier_compensate_split(q1["max_idx"], q1["min_idx"], q1["residual"],
                                                   idx_w[c_last], idx_wr[c_last], lut, b_w, s_w,
                                                   d_in, accumulate=False, workspace=ws)
            oasis.lut_gemm(q1["idx_act"], q1["act_scale"], idx_w[c_last], s_w, lut, b_a, b_w,
                           algo, y=y_ref, accumulate=True)
    torch.cuda.synchronize()
    schedule_ok = bool(torch.equal(y_sched, y_ref)) if algo == oasis.ALGO_MFMA else bool(
        torch.allclose(y_sched, y_ref, rtol=1e-4, atol=1e-3))
    if not schedule_ok:
        print(f"bench.py: {s.name}: the timed schedule's output differs from an eager pass",
              file=sys.stderr)
    del y_sched, y_ref, q1

    # ---- per-call durations: `nsteps` back-to-back launches of one call (same
    # arguments, rotating weight copies) queued behind a spin kernel, so the
    # GPU never waits for the host; one HIP event pair around the batch on the
    # stream the calls launch on (the current stream).
    kern_us = {}
    stream = torch.cuda.current_stream()
    for nm in names:
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(int(2.4e9 * (0.002 + nsteps * 60e-6)))  # longer than the host needs
        e0.record(stream)
        for i in range(nsteps):
            calls[nm]((args.warmup + i) % copies)
        e1.record(stream)
        torch.cuda.synchronize()
        kern_us[nm] = e0.elapsed_time(e1) * 1e3 / nsteps
    fused = path == "fused"
    ms_per_step = elapsed * 1e3 / nsteps
    ops = 2.0 * n * d_in * d_out
    value = ops / (ms_per_step * 1e-3) / 1e12

    # ---- roofline of the dominant kernel: the longest call that is one
    # kernel (the split call runs the lists' kernel, its preparation and the
    # GEMM; the GEMM alone is timed as lut_gemm)
    kbytes = call_bytes(n, d_in, d_out, k, path)
    composite = {"lut_gemm_compensated_split", "outlier_compensate"} if path == "split" else set()
    dom = max((nm for nm in names if nm not in composite), key=lambda nm: kern_us[nm])

    def roof(nm):
        us = kern_us[nm]
        if nm in ("lut_gemm", "lut_gemm_compensated", "lut_gemm_compensated_rows",
                  "lut_gemm_compensated_percol") and n > 32:
            tflops = ops / (us * 1e-6) / 1e12
            r = {"bound": "mfma", "achieved": round(tflops, 2), "peak": MFMA_F16_PEAK_TFLOPS,
                 "unit": "TFLOP/s", "frac": round(tflops / MFMA_F16_PEAK_TFLOPS, 4),
                 "flops_per_launch": ops}
        else:
            gbs = kbytes[nm] / (us * 1e-6) / 1e9
            r = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                 "frac": round(gbs / HBM_PEAK_GBS, 4), "bytes_per_launch": kbytes[nm]}
        r["traffic"] = measured_traffic(nm, s.name)
        r["kernel"] = nm
        r["kernel_us"] = round(us, 3)
        return r

    out = {
        "workload": s.name,
        "value": round(value, 3),
        "ms_per_step": round(ms_per_step, 5),
        "config": {"workload": s.name, "n": n, "d_in": d_in, "d_out": d_out, "k_per_side": k,
                   "b_a": b_a, "b_w": b_w, "algo": args.algo, "launch": mode,
                   "path": path, "outliers": "static" if thr else "top-k",
                   "scale": args.scale,
                   "weight_codebooks": "per-column" if args.percol else "shared",
                   "weight_copies": copies},
        "schedule_check": schedule_ok,
        "step_hbm_gbs": round(step_bytes(n, d_in, d_out, k, fused) / (ms_per_step * 1e-3) / 1e9, 1),
        "kernel_us": {kk: round(v, 3) for kk, v in kern_us.items()},
        "roofline": roof(dom),
        "roofline_main_branch": roof(gemm_name),
    }
    del q, y, x, ws
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="large_prefill_4096x8192x28672")
    ap.add_argument("--decode-config", default="auto",
                    help="the layer timed as the line's decode part: 'auto' (16 tokens through "
                         "the same weights when --config is the large prefill layer), a layer "
                         "name, or 'none'")
    ap.add_argument("--algo", default="mfma", choices=["mfma", "lut"])
    ap.add_argument("--oasis-s", action="store_true",
                    help="OASIS-S: outliers from fixed thresholds (the mean k-th extreme "
                         "values of the calibration tokens), 2k places per side")
    ap.add_argument("--bits-a", type=int, default=0, choices=[0, 1, 2, 3, 4],
                    help="activation bits (0: the config's, 4); 3 is the paper's W4A3 point")
    ap.add_argument("--scale", default="absmax", choices=["absmax", "inlier"],
                    help="per-token scale: absmax of all channels, or of the channels in "
                         "neither outlier list (a second quantize launch; no look-ahead)")
    ap.add_argument("--percol", action="store_true",
                    help="an independent weight codebook per output channel (fused GEMV, "
                         "one launch per 32 tokens)")
    ap.add_argument("--copies", type=int, default=0, help="weight copies (0: auto, >512 MiB)")
    ap.add_argument("--eager", action="store_true", help="launch eagerly instead of graphs")
    ap.add_argument("--path", default="auto",
                    choices=["auto", "fused", "split", "separate", "lookahead"],
                    help="fused: one call for Y* + Y' (default for <= 32 tokens); split: the "
                         "compensation split by channel, heavy channels inside the GEMM "
                         "(default for more tokens); separate: split compensation, then the "
                         "GEMM; lookahead: outlier detection on a second stream beside the "
                         "main-branch GEMM")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--verbose", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (counter calibration)")
    ap.add_argument("--summarize-pmc", default="", metavar="DIR",
                    help="only summarize rocprofv3 --pmc runs under DIR into profiles/")
    args = ap.parse_args()
    if args.summarize_pmc:
        summarize_pmc(args.summarize_pmc, layer_spec(args, args.config).name,
                      "fused" if args.path == "auto" else args.path)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: this build runs on one GPU only; --gpus must be 1 (no figure at "
              "several GPUs is measured)", file=sys.stderr)
        sys.exit(2)
    if args.scale == "inlier" and args.path == "lookahead":
        print("bench.py: --scale inlier has no look-ahead schedule (the scale needs the lists)",
              file=sys.stderr)
        sys.exit(2)
    if args.percol and (args.path not in ("auto", "fused") or args.algo != "mfma"):
        print("bench.py: --percol runs the fused MFMA GEMV (32 tokens per launch)",
              file=sys.stderr)
        sys.exit(2)
    if args.oasis_s and args.path == "lookahead":
        print("bench.py: --oasis-s has no look-ahead schedule (no top-k to overlap)",
              file=sys.stderr)
        sys.exit(2)
    dec_name = args.decode_config
    if dec_name == "auto":
        dec_name = "large_decode_16x8192x28672" \
            if args.config == "large_prefill_4096x8192x28672" else "none"

    from paper_2507_23035_amd import synth
    scale_mode = 2 if args.scale == "inlier" else 0
    specs = [layer_spec(args, args.config)]
    if dec_name != "none":
        specs.append(layer_spec(args, dec_name))
    def progress(msg):
        print(f"bench.py: {msg}", file=sys.stderr, flush=True)

    layers = []
    if not args.calibrate_copy:
        for sp in specs:
            layers.append(synth.make_layer(sp))
            progress(f"layer {sp.name} generated")

    # ---- the oracle on the host cores, before anything touches the GPU (its
    # worker processes are forked)
    cpu = {}
    if not args.no_cpu_baseline and not args.calibrate_copy:
        for L in layers:
            cols = synth.percol_codebooks(L) if args.percol else None
            cpu[L.spec.name] = cpu_baseline(L, mode=scale_mode, cols=cols)
            progress(f"oracle timed on {L.spec.name}: {cpu[L.spec.name]['sample']}")

    import torch
    from paper_2507_23035_amd import oasis

    if not torch.cuda.is_available():
        print("bench.py: no GPU", file=sys.stderr)
        sys.exit(1)
    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy)
        return
    oasis.load()
    dev = torch.device("cuda:0")
    side = torch.cuda.Stream()
    parts = []
    wsets = {}
    for L in layers:
        key = (L.w_idx.shape, id(L.w_idx))
        if key not in wsets:
            wsets[key] = Weights(L, args.copies, dev)
        parts.append(run_workload(args, L, wsets[key], dev, side))
        progress(f"{L.spec.name}: {parts[-1]['ms_per_step'] * 1e3:.1f} us per step")
    head = parts[0]
    out = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "effective TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": head["config"],
        "schedule_check": head["schedule_check"],
        "step_hbm_gbs": head["step_hbm_gbs"],
        "kernel_us": head["kernel_us"],
        "roofline": head["roofline"],
        "roofline_main_branch": head["roofline_main_branch"],
    }
    if specs[0].name in cpu:
        out["cpu_baseline"] = cpu[specs[0].name]
    if len(parts) > 1:
        dec = {kk: v for kk, v in parts[1].items() if kk != "workload"}
        dec["unit"] = "effective TOPS"
        if specs[1].name in cpu:
            dec["cpu_baseline"] = cpu[specs[1].name]
        out["decode"] = dec
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
