"""Benchmark of the P4Q hot path on one MI355X.

One step = one pass of the whole hot path over one batch:
  1. quantization-aware selection: B x N visual tokens -> K kept + T text
     (p4q_select), the pruned sequence X [M = B(K+T), h];
  2. per-token int4 quantization of X, of the attention-output stand-in and
     of the MLP-activation stand-in (p4q_quant_act);
  3. the seven W4A4 linears of one decoder layer on those codes
     (p4q_w4a4_linear): q/k/v/gate/up on X, o_proj, down_proj, as four
     launches: q|k|v and gate|up run as one GEMM each on row-concatenated
     weights (fused projections, as serving stacks store them).
Weights are quantized once, before timing (offline RTN, as in the paper).
Four copies of the layer's weights rotate across steps so that successive
steps read weights like successive decoder layers would (101 MB per layer at
7B, i.e. not resident in the 256 MB MALL across the rotation).

Timing: W untimed steps, then K timed steps between two synchronizations and
a start / end event pair on the launch stream; inside them each step records
three events only (after the selector, the quantize calls and the GEMMs), from
which the per-phase mean, median, p10 and p90 are reported.

Prints ONE JSON line.  value = W4A4 linear ops of the step / step time (TOPS);
roofline = the GEMM phase against the int8 MFMA peak (published, and measured
by a microbenchmark of this device); the selector's token rate and HBM
fraction beside it.  Also reported, outside the timed steps: the same step at
batch 1 (LLaVA-NeXT-7B, K = 320 / 640) and at the 13B stress shape, the hot-
cache GEMM rate, the fused RMSNorm + quantize prologue, the attention prefill,
the calibration step, the three-stage selector and the decode-step GEMV, and
the oracle's rate on the host's cores (all of them and one).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

INT8_PEAK_TOPS = 5000.0      # MI355X dense int8 MFMA
FP16_PEAK_TFLOPS = 2500.0    # MI355X dense fp16 MFMA
FP32_PEAK_TFLOPS = 157.3     # MI355X dense fp32
HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
N_WEIGHT_SETS = 4


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="next7b_b16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true", help="skip the decode GEMV measurement")
    ap.add_argument("--no-calib", action="store_true", help="skip the calibration-step measurement")
    ap.add_argument("--calib-only", action="store_true",
                    help="measure only the calibration step (for profiling it alone)")
    ap.add_argument("--decode-only", action="store_true",
                    help="measure only the decode GEMV layer (for profiling it alone)")
    ap.add_argument("--no-select-full", action="store_true",
                    help="skip the three-stage selector measurement")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy (HBM counter calibration)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the batch-1 and 13B-shape configurations")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip the MFMA and HBM microbenchmarks")
    ap.add_argument("--step-only", action="store_true",
                    help="only the timed steps of --config (for profiling them alone)")
    return ap.parse_args()


def setup(cfg, dev):
    import torch
    import paper_2609_34867_amd as p4q
    from workload import selector_inputs, weight, attn_standin, mlp_standin

    si = selector_inputs(cfg)
    t = lambda a: torch.from_numpy(a).to(dev)
    st = {
        "vis": t(si.vis), "con": t(si.concepts), "text": t(si.text),
        "attn": t(attn_standin(cfg)), "mlp": t(mlp_standin(cfg)),
    }
    st["idx"] = torch.empty((cfg.B, cfg.K), dtype=torch.int32, device=dev)
    st["tok"] = torch.empty((cfg.B, cfg.K + cfg.T, cfg.d), dtype=torch.float16, device=dev)
    st["ws"] = p4q.select_workspace(cfg.B, cfg.N, cfg.d, cfg.J, dev)
    M = cfg.M
    st["xq"] = (torch.empty((M, cfg.d // 2), dtype=torch.uint8, device=dev),
                torch.empty((M,), dtype=torch.float32, device=dev))
    st["aq"] = (torch.empty((M, cfg.d // 2), dtype=torch.uint8, device=dev),
                torch.empty((M,), dtype=torch.float32, device=dev))
    f = st["mlp"].shape[1]
    st["mq"] = (torch.empty((M, f // 2), dtype=torch.uint8, device=dev),
                torch.empty((M,), dtype=torch.float32, device=dev))
    out_dt = torch.bfloat16 if cfg.out_dtype == "bf16" else torch.float16
    q = {}
    for li, lin in enumerate(cfg.linears):
        q[lin.name] = p4q.quant_act(t(weight(cfg, li)))     # offline weight RTN
    weights = []
    for gname, members, src in launch_groups(cfg):
        weights.append((torch.cat([q[m][0] for m in members]),
                        torch.cat([q[m][1] for m in members])))
    del q
    torch.cuda.synchronize()
    st["weights"] = [[(wc.clone(), ws.clone()) for (wc, ws) in weights]
                     for _ in range(N_WEIGHT_SETS)]
    st["y"] = [torch.empty((M, wc.shape[0]), dtype=out_dt, device=dev) for (wc, _) in weights]
    # split-K workspaces of the small-M launches (none at large M), allocated
    # once so that no allocation happens inside the timed steps
    k_in = {"x": cfg.d, "attn": cfg.d, "mlp": f}
    st["gemm_ws"] = [p4q.w4a4_linear_workspace(M, wc.shape[0], k_in[src], dev)
                     for (wc, _), (_, _, src) in zip(weights, launch_groups(cfg))]
    del weights
    torch.cuda.synchronize()
    return st


def launch_groups(cfg):
    """The layer's linears as launches: linears that read the same input run as
    one GEMM on row-concatenated weights (q|k|v and gate|up), the layout serving
    stacks keep their fused projections in.  Returns (name, members, source)."""
    groups, seen = [], set()
    for lin in cfg.linears:
        if lin.name in seen:
            continue
        if lin.name == "q_proj":
            members = ["q_proj", "k_proj", "v_proj"]
            name = "qkv"
        elif lin.name == "gate_proj":
            members = ["gate_proj", "up_proj"]
            name = "gate_up"
        else:
            members, name = [lin.name], lin.name
        seen.update(members)
        groups.append((name, members, lin.source))
    return groups


PHASES = ("select", "quant_act", "gemm")


def step(cfg, st, layer, marks=None):
    """One hot-path pass: the selector, the three quantize calls, the four
    GEMM launches, in that order on the current stream.  `marks`, when given,
    holds three pre-created events recorded after the selector, after the
    quantize calls and after the GEMMs (the phase boundaries; the step's
    start is the previous step's last mark), so a timed step records three
    events and nothing else."""
    import paper_2609_34867_amd as p4q

    p4q.select(st["vis"], st["con"], st["text"], cfg.K, idx_out=st["idx"], tokens_out=st["tok"],
               workspace=st["ws"])
    if marks:
        marks[0].record()
    x = st["tok"].view(cfg.M, cfg.d)
    p4q.quant_act(x, codes=st["xq"][0], scales=st["xq"][1])
    p4q.quant_act(st["attn"], codes=st["aq"][0], scales=st["aq"][1])
    p4q.quant_act(st["mlp"], codes=st["mq"][0], scales=st["mq"][1])
    if marks:
        marks[1].record()
    W = st["weights"][layer % N_WEIGHT_SETS]
    src = {"x": st["xq"], "attn": st["aq"], "mlp": st["mq"]}
    for gi, (gname, members, source) in enumerate(launch_groups(cfg)):
        a = src[source]
        p4q.w4a4_linear(a[0], a[1], W[gi][0], W[gi][1], y=st["y"][gi],
                        workspace=st["gemm_ws"][gi])
    if marks:
        marks[2].record()


def timed_steps(cfg, st, steps, warmup):
    """`warmup` untimed steps, then `steps` timed ones bracketed by
    synchronizations and a start / end event pair on the launch stream (the
    stream the binding passes to every call).  Returns the mean ms per step
    and the per-step duration of each phase (ms, from the phase marks)."""
    import torch

    for i in range(warmup):
        step(cfg, st, i)
    mk = lambda: torch.cuda.Event(enable_timing=True)
    marks = [[mk(), mk(), mk()] for _ in range(steps)]
    start, end = mk(), mk()
    torch.cuda.synchronize()
    start.record()
    for i in range(steps):
        step(cfg, st, i, marks[i])
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / steps
    phases = {p: [] for p in PHASES}
    prev = start
    for m in marks:
        phases["select"].append(prev.elapsed_time(m[0]))
        phases["quant_act"].append(m[0].elapsed_time(m[1]))
        phases["gemm"].append(m[1].elapsed_time(m[2]))
        prev = m[2]
    return ms, phases


def dist(v):
    """mean, median, p10 and p90 of per-step durations (ms)."""
    a = np.asarray(v, dtype=np.float64)
    return {"mean": round(float(a.mean()), 5), "median": round(float(np.median(a)), 5),
            "p10": round(float(np.percentile(a, 10)), 5),
            "p90": round(float(np.percentile(a, 90)), 5)}


def selector_bytes(cfg):
    """Algorithmic HBM bytes of one selector call: the features once, the kept
    rows again, the text rows, the pruned sequence written."""
    return (cfg.B * cfg.N * cfg.d * 2 + cfg.B * cfg.K * cfg.d * 2 + cfg.B * cfg.T * cfg.d * 2
            + cfg.M * cfg.d * 2)


def gemm_hot(cfg, st, reps=10):
    """The step's four GEMM launches on one weight copy, repeated: operands
    stay in the 256 MB MALL as far as they fit (the hot-cache number beside
    the rotated, cold one of the timed steps)."""
    import torch
    import paper_2609_34867_amd as p4q

    W = st["weights"][0]
    src = {"x": st["xq"], "attn": st["aq"], "mlp": st["mq"]}

    def run():
        for gi, (gname, members, source) in enumerate(launch_groups(cfg)):
            a = src[source]
            p4q.w4a4_linear(a[0], a[1], W[gi][0], W[gi][1], y=st["y"][gi],
                            workspace=st["gemm_ws"][gi])
    run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def config_result(cfg, ms, phases, peak_meas=None):
    """Per-configuration figures of the timed steps."""
    ops = cfg.linear_ops()
    g, s = dist(phases["gemm"]), dist(phases["select"])
    tops = ops / (g["mean"] * 1e-3) / 1e12
    sel_gbs = selector_bytes(cfg) / (s["mean"] * 1e-3) / 1e9
    out = {"workload": workload_name(cfg), "ms_per_step": round(ms, 4),
           "gemm_tops": round(tops, 2), "gemm_frac_int8_peak": round(tops / INT8_PEAK_TOPS, 4),
           "gemm_floor_ms": round(ops / (INT8_PEAK_TOPS * 1e12) * 1e3, 4),
           "selector_us": round(s["mean"] * 1e3, 2),
           "selector_tokens_per_s": round(cfg.B * cfg.N / (s["mean"] * 1e-3), 1),
           "selector_gbs": round(sel_gbs, 1), "selector_hbm_frac": round(sel_gbs / HBM_PEAK_GBS, 4),
           "selector_floor_us": round(selector_bytes(cfg) / (HBM_PEAK_GBS * 1e9) * 1e6, 2),
           "phase_ms": {k: dist(v) for k, v in phases.items()}}
    if peak_meas:
        out["gemm_frac_measured_mfma_peak"] = round(tops / peak_meas, 4)
    return out


def workload_name(cfg):
    return (f"{cfg.name}: select K={cfg.K} of N={cfg.N} tokens x d={cfg.d} fp16 for B={cfg.B} "
            f"image(s) + T={cfg.T} text, then 7 W4A4 linears (h={cfg.d}, "
            f"f={cfg.linears[4].n_out}) at M={cfg.M} as 4 launches (q|k|v, o, gate|up, down), "
            f"{cfg.out_dtype} out")


def peaks(dev):
    """Measured ceilings of this device: the int8 MFMA microbenchmark (random
    operands, 2 work-groups of 4 wavefronts per CU) and a streaming read of
    2 GiB (2 work-groups of 4 wavefronts per CU, the fastest of 2 to 64 per
    CU in a sweep on this MI355X: 6.98 TB/s against 5.6-6.0 with more)."""
    import torch
    import paper_2609_34867_amd as p4q

    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    out = torch.empty(4 * cus * 256 * 8, dtype=torch.int32, device=dev)

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            work = fn()
        e1.record()
        torch.cuda.synchronize()
        return work, e0.elapsed_time(e1) / reps
    ops, ms = timed(lambda: p4q.diag_mfma_i8(2 * cus, 4096, out), 5)
    src = torch.empty(1 << 31, dtype=torch.uint8, device=dev)
    src.fill_(1)
    nb, ms_r = timed(lambda: p4q.diag_stream_read(src, 2 * cus, out), 5)
    del src
    return {"mfma_i8_tops": round(ops / (ms * 1e-3) / 1e12, 1),
            "hbm_read_gbs": round(nb / (ms_r * 1e-3) / 1e9, 1),
            "cus": cus,
            "note": "int8 MFMA: 2 x 4 wavefronts per CU each issuing 16 independent "
                    "v_mfma_i32_16x16x64_i8 per round on pseudo-random operands; HBM: one "
                    "streaming read of 2 GiB, 16-byte non-temporal loads, 2 work-groups per CU"}


def cpu_baseline(cfg):
    """The oracle on a bounded sample of the same workload, scaled to the step:
    every image through the selector and 8192 of the pruned rows through
    every quantize + linear (weights quantized beforehand, untimed), with the
    BLAS threads of the host (the oracle's selector and quantizer loops are
    single-threaded Python / NumPy); then the same on one image and 1024 rows
    with one BLAS thread."""
    import oracle
    from threadpoolctl import threadpool_limits
    from workload import selector_inputs, weight, attn_standin, mlp_standin

    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    si = selector_inputs(cfg, samples=list(range(cfg.B)))
    wq = [oracle.quant_act(weight(cfg, li)) for li in range(len(cfg.linears))]   # offline, untimed

    def run(n_img, rows):
        toks = []
        t0 = time.perf_counter()
        for b in range(n_img):
            toks.append(oracle.select(si.vis[b], si.concepts[b], si.text[b], cfg.K)[1])
        t_sel = (time.perf_counter() - t0) / n_img
        xs = {"x": np.concatenate(toks)[:rows],
              "attn": attn_standin(cfg, rows), "mlp": mlp_standin(cfg, rows)}
        t_lin = 0.0
        for li, lin in enumerate(cfg.linears):
            t0 = time.perf_counter()
            ap, sa = oracle.quant_act(xs[lin.source])
            oracle.w4a4_linear(ap, sa, wq[li][0], wq[li][1], cfg.out_dtype)
            t_lin += time.perf_counter() - t0
        return t_sel, t_lin, cfg.B * t_sel + (cfg.M / rows) * t_lin

    rows = min(8192, cfg.B * (cfg.K + cfg.T))
    t_sel, t_lin, t_full = run(cfg.B, rows)
    with threadpool_limits(limits=1):
        rows1 = min(1024, cfg.K + cfg.T)
        t_sel1, t_lin1, t_full1 = run(1, rows1)
    return {"value": round(cfg.linear_ops() / t_full / 1e12, 6), "unit": "TOPS",
            "cores": threads, "kind": "oracle",
            "scaled_from_sample": True,
            "sample": (f"{cfg.B} of {cfg.B} images through the selector ({cfg.B * t_sel:.1f}s) and "
                       f"{rows} of {cfg.M} rows through quantize + all 7 linears ({t_lin:.1f}s), "
                       f"scaled to the full step ({t_full:.0f}s)"),
            "value_1thread": round(cfg.linear_ops() / t_full1 / 1e12, 6),
            "sample_1thread": (f"1 image through the selector ({t_sel1:.1f}s) and {rows1} rows "
                               f"through quantize + all 7 linears ({t_lin1:.1f}s) with one BLAS "
                               f"thread, scaled to the full step ({t_full1:.0f}s)")}


def decode_gemv(dev, steps=20):
    """Decode-step W4A4 linears of the 13B-shape layer (h = 5120, f = 13824)
    at M in {1, 4, 16}: HBM-bound, reported against the 8 TB/s peak.  The
    linears that share an input run as one launch on row-concatenated weights
    (q|k|v and gate|up, as serving stacks store them), so a layer is 4
    launches: qkv, o, gate_up, down.  Four weight copies (634 MB) rotate so
    the 158.8 MB of packed weights of a layer come from HBM, not from the
    256 MB MALL."""
    import torch
    import paper_2609_34867_amd as p4q
    from workload import CONFIGS, weight, gemv_activations

    cfg = CONFIGS["stress13b_b8"]
    names = [lin.name for lin in cfg.linears]
    q = {}
    for li, lin in enumerate(cfg.linears):
        q[lin.name] = p4q.quant_act(torch.from_numpy(weight(cfg, li)).to(dev))
    groups = [("qkv", ["q_proj", "k_proj", "v_proj"]), ("o", ["o_proj"]),
              ("gate_up", ["gate_proj", "up_proj"]), ("down", ["down_proj"])]
    fused = []
    for gname, members in groups:
        wc = torch.cat([q[m][0] for m in members])
        ws = torch.cat([q[m][1] for m in members])
        fused.append((gname, wc, ws, cfg.linears[names.index(members[0])].k_in))
    del q
    torch.cuda.synchronize()
    copies = [[(wc.clone(), ws.clone()) for (_, wc, ws, _) in fused] for _ in range(N_WEIGHT_SETS)]
    wbytes = sum(wc.numel() + 4 * ws.numel() for (_, wc, ws, _) in fused)
    del fused
    kins = [cfg.linears[names.index(members[0])].k_in for _, members in groups]
    out = {}
    for M in cfg.gemv_M:
        acts = {}
        for k_in in set(kins):
            x = torch.from_numpy(gemv_activations(cfg, M, k_in)).to(dev)
            acts[k_in] = p4q.quant_act(x)
        ys = [torch.empty((M, wc.shape[0]), dtype=torch.bfloat16, device=dev)
              for (wc, _) in copies[0]]

        def layer(i):
            W = copies[i % N_WEIGHT_SETS]
            for gi, k_in in enumerate(kins):
                a = acts[k_in]
                p4q.w4a4_linear(a[0], a[1], W[gi][0], W[gi][1], y=ys[gi])

        def timed(run):
            for i in range(5):
                run(i)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for i in range(steps):
                run(i)
            e1.record()
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) * 1e3 / steps

        us_eager = timed(layer)
        # the decode loop of a server replays captured graphs: one per weight copy
        graphs = []
        for i in range(N_WEIGHT_SETS):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                layer(i)
            graphs.append(g)
        us = timed(lambda i: graphs[i % N_WEIGHT_SETS].replay())
        del graphs
        nbytes = wbytes + sum(M * (k // 2 + 4) for k in kins) + sum(y.numel() * 2 for y in ys)
        out[str(M)] = {"us_per_layer": round(us_eager, 2), "gbs": round(nbytes / us_eager / 1e3, 1),
                       "hbm_frac": round(nbytes / us_eager / 1e3 / HBM_PEAK_GBS, 4),
                       "us_per_layer_graph": round(us, 2)}
    return {"workload": "13b-shape decode step: 7 W4A4 linears (h=5120, f=13824) as 4 launches "
                        "(qkv, o, gate_up, down on row-concatenated weights), bf16 out, "
                        f"{wbytes / 1e6:.1f} MB of packed weights per layer; us_per_layer: the "
                        "launches queued from Python (they run ahead of the GPU); "
                        "us_per_layer_graph: the same launches replayed as a captured HIP graph "
                        "(the kernels take as long either way, the replay adds launch cost)",
            "M": out}


def selector_full(cfg, dev, reps=10):
    """The three-stage selector (Query Relevance, Visual Saliency, Visual
    Diversity at the paper's 0.3 / 0.2 / 0.5 split of K) on the same batch of
    features, with the CLS-attention stand-in.  Its dominant kernels are the
    code Gram matrix on the int8 MFMA path (2 B N^2 d ops counted for the
    full matrix; the kernel computes the upper half and mirrors it) and the
    sequential greedy scan (K - kq - ks dependent steps per sample)."""
    import torch
    import paper_2609_34867_amd as p4q
    from workload import selector_inputs, cls_attention

    si = selector_inputs(cfg)
    t = lambda a: torch.from_numpy(a).to(dev)
    vis, con, txt = t(si.vis), t(si.concepts), t(si.text)
    cls = t(np.stack([cls_attention(cfg.cfg_id, cfg.N, b) for b in range(cfg.B)]))
    kq, ks, kd = p4q.select_budgets(cfg.K)
    idx = torch.empty((cfg.B, cfg.K), dtype=torch.int32, device=dev)
    tok = torch.empty((cfg.B, cfg.K + cfg.T, cfg.d), dtype=vis.dtype, device=dev)
    ws = p4q.select_full_workspace(cfg.B, cfg.N, cfg.d, cfg.J, cfg.K, dev)
    run = lambda: p4q.select_full(vis, con, cls, txt, cfg.K, kq, ks, idx_out=idx, tokens_out=tok,
                                  workspace=ws)
    for _ in range(3):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del ws
    return {"workload": f"{cfg.name}: three-stage selection of K={cfg.K} (kq={kq}, ks={ks}, "
                        f"kd={kd}) of N={cfg.N} tokens x d={cfg.d} for B={cfg.B} images + "
                        f"T={cfg.T} text",
            "ms": round(ms, 4), "tokens_per_s": round(cfg.B * cfg.N / (ms * 1e-3), 1),
            "greedy_steps_per_sample": kd,
            "gram_ops_full_matrix": 2 * cfg.B * cfg.N * cfg.N * cfg.d}


def prologue(cfg, st, dev, reps=20):
    """The fused decoder prologue (p4q_rmsnorm_quant: per-token int4 of
    RMSNorm(X) * gamma) on the step's pruned sequence X [M, d], next to the
    plain quantize-and-pack of X.  HBM-bound: algorithmic bytes = read X
    (2 B/element) + gamma + codes (0.5 B/element) + scales; an unfused
    RMSNorm would also write and re-read the normalized rows."""
    import torch
    import paper_2609_34867_amd as p4q
    from workload import norm_weight

    x = st["tok"].view(cfg.M, cfg.d)
    g = torch.from_numpy(norm_weight(cfg)).to(dev)
    codes, scales = st["xq"]

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / reps

    us = timed(lambda: p4q.rmsnorm_quant(x, g, 1e-5, codes=codes, scales=scales))
    us_plain = timed(lambda: p4q.quant_act(x, codes=codes, scales=scales))
    nbytes = cfg.M * cfg.d * 2 + cfg.d * 2 + cfg.M * cfg.d // 2 + 4 * cfg.M
    return {"workload": f"per-token int4 of RMSNorm(X) * gamma, X = the pruned sequence "
                        f"[M={cfg.M}, d={cfg.d}] fp16",
            "us": round(us, 2), "gbs": round(nbytes / us / 1e3, 1),
            "hbm_frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4),
            "us_plain_quant_act": round(us_plain, 2),
            "unfused_extra_bytes": 2 * cfg.M * cfg.d * 2}


def attention(cfg, dev, reps=20):
    """Causal attention prefill of the decoder layer on the pruned sequence
    (B samples x K+T tokens, 32 heads of 128) reading q, k, v out of one fused
    q|k|v buffer, fp16.  Bound by the MFMA work: 4 B H D sum_t (t+1) flops
    (the causal half), fp16 dense peak 2500 TFLOP/s."""
    import torch
    import paper_2609_34867_amd as p4q

    B, L, D = cfg.B, cfg.K + cfg.T, 128
    H = cfg.d // D
    g = torch.Generator(device="cpu").manual_seed(7)
    qkv = torch.randn((B * L, 3 * H * D), generator=g, dtype=torch.float32).to(torch.float16).to(dev)
    out = torch.empty((B * L, H * D), dtype=torch.float16, device=dev)
    run = lambda: p4q.attention_prefill(qkv[:, :H * D], qkv[:, H * D:2 * H * D], qkv[:, 2 * H * D:],
                                        B, H, True, out=out)
    for _ in range(3):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    flops = 4 * B * H * D * (L * (L + 1) // 2)
    return {"workload": f"causal attention prefill, B={B} x L={L} tokens, H={H} heads of {D}, "
                        "fp16 q|k|v from one fused buffer",
            "us": round(us, 2), "tflops": round(flops / us / 1e6, 1),
            "mfma_frac": round(flops / us / 1e6 / FP16_PEAK_TFLOPS, 4)}


def calibration(dev, reps=20, M=384, N=12288, K=4096):
    """One pruning-aware calibration step of a W4A4 fake-quantized linear
    (loss + gradients for the diagonal scales and clipping factors) at the
    LLaVA-NeXT-7B q|k|v shape on one pruned calibration sample: M = 320 kept
    visual + 64 text tokens, N = 3 x 4096, K = 4096.  Synthetic inputs of the
    workload's calibration recipe (seeded on the GPU: the host generator's
    float64 target matmul would dominate the set-up)."""
    import torch
    import paper_2609_34867_amd as p4q
    g = torch.Generator(device=dev).manual_seed(11)
    x = torch.randn((M, K), generator=g, device=dev, dtype=torch.float32)
    ch = torch.randperm(K, generator=g, device=dev)[:8]
    x[:, ch] *= 20.0
    w = torch.randn((N, K), generator=g, device=dev, dtype=torch.float32) * 0.02
    x, w = x.to(torch.float16), w.to(torch.float16)
    target = x.float() @ w.float().T
    sigma = torch.exp(0.3 * torch.randn(K, generator=g, device=dev))
    sigma[ch] *= 20.0 ** 0.3
    clip_w = 0.75 + 0.25 * torch.rand(N, generator=g, device=dev)
    ws = p4q.calib_linear_workspace(M, N, K, dev)
    outs = (torch.empty(1, device=dev), torch.empty(K, device=dev), torch.empty(1, device=dev),
            torch.empty(N, device=dev))
    run = lambda: p4q.calib_linear_grad(x, w, target, sigma, 0.9, clip_w, workspace=ws, out=outs)
    for _ in range(3):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    mnk = M * N * K
    # time the matrix units need at their dense peaks: the int8 forward GEMM
    # (2MNK ops) and the two bf16 backward products (2MNK flops each)
    floor_us = 2 * mnk / (INT8_PEAK_TOPS * 1e6) + 4 * mnk / (FP16_PEAK_TFLOPS * 1e6)
    return {"workload": f"calibration step of one W4A4 linear: M={M} (320 kept visual + 64 text "
                        f"tokens), N={N} (q|k|v), K={K}, fp16; loss + d sigma, d clip_a, d clip_w",
            "us": round(us, 2), "steps_per_s": round(1e6 / us, 1),
            "mfma_floor_us": round(floor_us, 2), "mfma_frac": round(floor_us / us, 4)}


def calibration_block(dev, reps=10, M=384, d=4096, f=11008, H=32):
    """One pruning-aware calibration step of a whole W4A4 fake-quantized
    LLaVA-NeXT-7B decoder block (loss + gradients of every linear group's
    diagonal scales and clipping factors) on one pruned calibration sample
    (320 kept visual + 64 text tokens).  Synthetic inputs of the block
    recipe drawn on the GPU; the target, the full-precision block's output,
    is computed in the untimed set-up with plain torch fp32 operations."""
    import torch
    import paper_2609_34867_amd as p4q
    g = torch.Generator(device=dev).manual_seed(13)
    rn = lambda *sh: torch.randn(*sh, generator=g, device=dev, dtype=torch.float32)
    x = rn(M, d)
    ch = torch.randperm(d, generator=g, device=dev)[:8]
    x[:, ch] *= 20.0
    x = x.half()
    w = {k: (rn(*sh) * 0.02).half() for k, sh in
         (("qkv", (3 * d, d)), ("o", (d, d)), ("gu", (2 * f, d)), ("down", (d, f)))}
    g1, g2 = (1.0 + 0.1 * rn(d)).half(), (1.0 + 0.1 * rn(d)).half()
    sig = torch.exp(0.3 * rn(3 * d + f))
    sig[ch] *= 20.0 ** 0.3
    clip_w = 0.75 + 0.25 * torch.rand(5 * d + 2 * f, generator=g, device=dev)
    clip_a = [0.9, 0.95, 0.85, 0.9]
    with torch.no_grad():                                  # full-precision target
        D = d // H

        def rms(v, gm):
            return (v * torch.rsqrt((v * v).mean(1, keepdim=True) + 1e-5) * gm.float()).half().float()
        xf = x.float()
        qkv = (rms(xf, g1) @ w["qkv"].float().T).half().float()
        i = torch.arange(D // 2, device=dev, dtype=torch.float64)
        ang = torch.arange(M, device=dev, dtype=torch.float64)[:, None] * 10000.0 ** (-2 * i / D)
        c, sn = torch.cos(ang).float()[:, None, :], torch.sin(ang).float()[:, None, :]

        def rope(z):
            a, b = z[..., :D // 2], z[..., D // 2:]
            return torch.cat([a * c - b * sn, b * c + a * sn], -1).half().float()
        q = rope(qkv[:, :d].reshape(M, H, D)).transpose(0, 1).contiguous()
        k = rope(qkv[:, d:2 * d].reshape(M, H, D)).transpose(0, 1).contiguous()
        v = qkv[:, 2 * d:].reshape(M, H, D).transpose(0, 1).contiguous()
        S = torch.matmul(q, k.transpose(1, 2).contiguous()) / D ** 0.5
        S = S.masked_fill(~torch.tril(torch.ones(M, M, device=dev, dtype=torch.bool)), float("-inf"))
        O = torch.matmul(torch.softmax(S, -1), v).transpose(0, 1).reshape(M, d).half().float()
        h = (xf + (O @ w["o"].float().T).half().float()).half().float()
        gu = (rms(h, g2) @ w["gu"].float().T).half().float()
        a = (torch.nn.functional.silu(gu[:, :f]) * gu[:, f:]).half().float()
        target = (h + (a @ w["down"].float().T).half().float()).half().float().contiguous()
        del qkv, q, k, v, S, O, h, gu, a
    ws = p4q.calib_block_workspace(M, d, f, H, dev)
    outs = (torch.empty(1, device=dev), torch.empty(3 * d + f, device=dev),
            torch.empty(4, device=dev), torch.empty(5 * d + 2 * f, device=dev))
    run = lambda: p4q.calib_block_grad(x, target, w["qkv"], w["o"], w["gu"], w["down"], g1, g2, H,
                                       sig, clip_a, clip_w, workspace=ws, out=outs)
    for _ in range(3):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    mnk = M * (3 * d * d + d * d + 2 * f * d + d * f)
    attn = 6 * 2 * H * M * M * D            # 6 fp32 products per head (full tiles)
    # the matrix units' floor: int8 forward GEMMs, two bf16 backward
    # contractions per group, the attention products at the fp32 peak
    floor_us = (2 * mnk / (INT8_PEAK_TOPS * 1e6) + 4 * mnk / (FP16_PEAK_TFLOPS * 1e6)
                + attn / (FP32_PEAK_TFLOPS * 1e6))
    del ws
    return {"workload": f"calibration step of one W4A4 LLaVA-NeXT-7B decoder block: M={M} (320 kept "
                        f"visual + 64 text tokens), d={d}, f={f}, {H} heads, fp16; loss + d sigma, "
                        f"d clip_a, d clip_w of the 4 linear groups",
            "us": round(us, 2), "steps_per_s": round(1e6 / us, 1),
            "mfma_floor_us": round(floor_us, 2), "mfma_frac": round(floor_us / us, 4)}


def copy_calibration(dev, nbytes=1 << 30, reps=5):
    """A plain device-to-device copy of known size, run so that the HBM
    counters (FETCH_SIZE, WRITE_SIZE) can be scaled to bytes: the counter
    reading of one copy dispatch corresponds to exactly `nbytes` read and
    `nbytes` written."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "dispatches": reps}), flush=True)


def traffic_from_profile():
    """HBM bytes per GEMM launch from the committed counter summary, or None
    when the GEMM source changed after the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "hbm_traffic_w4a4_gemm_llava_next_b16.md")
    src = os.path.join(ROOT, "paper_2609_34867_amd", "csrc", "w4a4_gemm.hip")
    try:
        fields = dict(l.strip("- \n").split(": ", 1) for l in open(path)
                      if l.startswith("- ") and ": " in l)
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
        if fields.get("w4a4_gemm.hip sha256") != sha:
            return None
        return int(fields["hbm bytes per launch"])
    except (OSError, KeyError, ValueError):
        return None


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(this build shows the per-GPU kernels; sharding across GPUs is not run)", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2609_34867_amd as p4q
    from workload import CONFIGS

    cfg = CONFIGS[args.config]
    dev = torch.device("cuda:0")
    if args.copy_calibration:
        copy_calibration(dev)
        return
    if args.calib_only:
        print(json.dumps({"calibration_step": calibration(dev),
                          "calibration_block_step": calibration_block(dev)}), flush=True)
        return
    if args.decode_only:
        print(json.dumps({"decode_gemv": decode_gemv(dev)}), flush=True)
        return
    st = setup(cfg, dev)
    ms, phases = timed_steps(cfg, st, args.steps, args.warmup)
    if args.step_only:
        print(json.dumps(config_result(cfg, ms, phases)), flush=True)
        return
    pk = None if args.no_peaks else peaks(dev)
    main_cfg = config_result(cfg, ms, phases, pk and pk["mfma_i8_tops"])

    ops = cfg.linear_ops()
    gemm_ms = main_cfg["phase_ms"]["gemm"]["mean"]
    gemm_tops = main_cfg["gemm_tops"]
    res = {
        "metric": "W4A4 GEMM TOPS (% int8 MFMA peak) + selector tokens/s, LLaVA-NeXT-7B shape",
        "value": round(ops / (ms * 1e-3) / 1e12, 3),
        "unit": "TOPS",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int4 (int8 MFMA, int32 acc)", "data": "synthetic",
        "config": {"workload": workload_name(cfg),
                   "B": cfg.B, "N": cfg.N, "d": cfg.d, "K": cfg.K, "T": cfg.T, "J": cfg.J,
                   "M": cfg.M, "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "achieved": round(gemm_tops, 2), "peak": INT8_PEAK_TOPS,
                     "unit": "TOPS", "frac": round(gemm_tops / INT8_PEAK_TOPS, 4),
                     "traffic": traffic_from_profile(), "kernel": "k_w4a4_gemm_pt",
                     "per_launch": "2*M*n_out*k_in int ops, averaged over the 4 launches of a step "
                                   "(HIP events around the step's GEMM phase); traffic in HBM "
                                   "bytes per launch"},
        "gemm_tops": round(gemm_tops, 2),
        "selector_tokens_per_s": main_cfg["selector_tokens_per_s"],
        "selector_gbs": main_cfg["selector_gbs"],
        "selector_hbm_frac": main_cfg["selector_hbm_frac"],
        "phase_ms": main_cfg["phase_ms"],
        "lib": p4q.version(),
    }
    if pk:
        res["measured_peaks"] = pk
        res["roofline"]["peak_measured"] = pk["mfma_i8_tops"]
        res["roofline"]["frac_measured"] = round(gemm_tops / pk["mfma_i8_tops"], 4)
        res["selector_frac_measured_read_peak"] = round(main_cfg["selector_gbs"] / pk["hbm_read_gbs"], 4)
    hot_ms = gemm_hot(cfg, st)
    res["gemm_hot_cache"] = {"ms": round(hot_ms, 4),
                             "tops": round(ops / (hot_ms * 1e-3) / 1e12, 2),
                             "note": "the 4 launches on one weight copy, repeated (the timed "
                                     "steps rotate 4 copies: cold weights)"}
    res["prologue_rmsnorm_quant"] = prologue(cfg, st, dev)
    del st
    torch.cuda.empty_cache()
    if not args.no_configs:
        others = {}
        for name in ("next7b_b1_k320", "next7b_b1_k640", "stress13b_b8"):
            c = CONFIGS[name]
            sc = setup(c, dev)
            cms, cph = timed_steps(c, sc, 20, 5)
            others[name] = config_result(c, cms, cph, pk and pk["mfma_i8_tops"])
            del sc
            torch.cuda.empty_cache()
        res["configs"] = others
    res["attention_prefill"] = attention(cfg, dev)
    if not args.no_calib:
        res["calibration_step"] = calibration(dev)
        res["calibration_block_step"] = calibration_block(dev)
    if not args.no_select_full:
        res["selector_full"] = selector_full(cfg, dev)
    if not args.no_decode:
        torch.cuda.empty_cache()
        res["decode_gemv"] = decode_gemv(dev)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(cfg)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
