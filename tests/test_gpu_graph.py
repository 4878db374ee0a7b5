"""HIP-graph replay of whole steps of the path (the way bench.py times them):
every replay, with other tokens copied in and eager launches in between,
equals the eager launches on the same input bit for bit."""
import numpy as np
import pytest
import torch

from paper_2507_23035_amd import oasis, synth

pytestmark = pytest.mark.gpu


def token_variants(x):
    """Other valid fp16 token batches of the same shape."""
    return [x, -x, x[::-1], np.roll(x, 3, axis=1)]


@pytest.mark.parametrize("schedule", ["fused", "fused_percol", "separate", "lookahead", "split",
                                      "split_noalloc"])
def test_graph_replays_match_eager(schedule):
    name = "decode_8x4096x4096" if schedule.startswith("fused") else None
    if name:
        spec = synth.config(name)
    elif schedule.startswith("split"):   # d_in a multiple of 64: heavy channels in the GEMM
        spec = synth.custom(70, 1024, 300, 20, seed=72)
    else:
        spec = synth.custom(70, 1032, 300, 20, seed=71)
    L = synth.make_layer(spec)
    s = L.spec
    print(f"case graph {schedule} n={s.n} d_in={s.d_in} d_out={s.d_out} k={s.k}", flush=True)
    dev = torch.device("cuda:0")
    idx_w = torch.from_numpy(oasis.pack_weight_indices(L.w_idx).view(np.int32)).to(dev)
    idx_wr = torch.from_numpy(oasis.pack_weight_rows(L.w_idx).view(np.int32)).to(dev)
    s_w = torch.from_numpy(L.s_w).to(dev)
    full = np.zeros((s.d_out, 16), dtype=np.float16)
    full[:, : 1 << s.b_w] = synth.percol_codebooks(L)
    cols = torch.from_numpy(full.view(np.int16).copy()).to(dev)
    xs = [torch.from_numpy(np.ascontiguousarray(v).view(np.int16).copy()).to(dev)
          for v in token_variants(L.x)]
    x = xs[0].clone()
    lut, q = oasis.build_lut_quantize_act(L.cb_a, s.b_a, L.cb_w, s.b_w, x, s.k)
    y = torch.empty((s.n, s.d_out), dtype=torch.float32, device=dev)
    side = torch.cuda.Stream()
    ws = torch.empty(oasis.split_workspace_bytes(s.n, s.d_in, s.d_out, s.k), dtype=torch.uint8,
                     device=dev)
    lib = oasis.load()

    def step():
        if schedule == "lookahead":
            main = torch.cuda.current_stream()
            oasis.build_lut(L.cb_a, s.b_a, L.cb_w, s.b_w, out=lut)
            side.wait_stream(main)
            with torch.cuda.stream(side):
                oasis.detect_outliers(x, lut, s.b_a, s.k, out=q, stream=side)
            oasis.cluster_act(x, lut, s.b_a, out=q)
            oasis.lut_gemm(q["idx_act"], q["act_scale"], idx_w, s_w, lut, s.b_a, s.b_w, y=y)
            main.wait_stream(side)
            oasis.outlier_compensate_rows(q["max_idx"], q["min_idx"], q["residual"], idx_wr, lut,
                                          s.b_w, s_w, s.d_in, y=y, accumulate=True)
            return
        oasis.build_lut_quantize_act(L.cb_a, s.b_a, L.cb_w, s.b_w, x, s.k, lut=lut, out=q)
        if schedule == "fused":
            oasis.lut_gemm_compensated_rows(q["idx_act"], q["act_scale"], idx_w, idx_wr, s_w, lut,
                                            s.b_a, s.b_w, q["max_idx"], q["min_idx"],
                                            q["residual"], y=y)
        elif schedule == "split":
            oasis.lut_gemm_compensated_split(q["idx_act"], q["act_scale"], idx_w, idx_wr, s_w, lut,
                                             s.b_a, s.b_w, q["max_idx"], q["min_idx"],
                                             q["residual"], y=y, workspace=ws)
        elif schedule == "split_noalloc":
            st = lib.oasis_lut_gemm_compensated_split_noalloc(
                q["idx_act"].data_ptr(), q["act_scale"].data_ptr(), s.n, s.d_in,
                idx_w.data_ptr(), idx_wr.data_ptr(), s_w.data_ptr(), s.d_out, lut.data_ptr(),
                s.b_a, s.b_w, q["max_idx"].data_ptr(), q["min_idx"].data_ptr(),
                q["residual"].data_ptr(), s.k, y.data_ptr(), 0,
                torch.cuda.current_stream().cuda_stream)
            assert st == 0
        elif schedule == "fused_percol":
            oasis.lut_gemm_compensated_percol(q["idx_act"], q["act_scale"], idx_w, s_w, lut, cols,
                                              s.b_a, s.b_w, q["max_idx"], q["min_idx"],
                                              q["residual"], y=y)
        else:
            oasis.outlier_compensate_rows(q["max_idx"], q["min_idx"], q["residual"], idx_wr, lut,
                                          s.b_w, s_w, s.d_in, y=y, accumulate=False)
            oasis.lut_gemm(q["idx_act"], q["act_scale"], idx_w, s_w, lut, s.b_a, s.b_w, y=y,
                           accumulate=True)

    step()  # prime the library outside capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        for v, xv in enumerate(xs):
            x.copy_(xv)
            step()
            torch.cuda.synchronize()
            y_eager = y.clone()
            q_eager = {key: t.clone() for key, t in q.items()}
            y.fill_(float("nan"))
            for t in q.values():
                t.fill_(90)
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(y, y_eager), f"replay {rep}, tokens {v}: y"
            for key, t in q.items():
                assert torch.equal(t, q_eager[key]), f"replay {rep}, tokens {v}: {key}"
