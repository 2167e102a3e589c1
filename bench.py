"""Benchmark of the OrbitQuant quantized-linear hot path on one MI355X.

A step is one pass of the online path over one batch: for each linear of the workload the
fused RPBH activation quantizer (rpbh_quantize_act) followed by the LUT-decode GEMM
(orbit_qlinear), on inputs already resident in HBM.  The offline weight pass
(quantize_weights_offline) and the host-side plan/codebook construction are timed once,
separately, and reported beside the step.

Default workload: the video-DiT MLP, W4A4, 32760 latent-patch + 512 text tokens,
5120 -> 13824 -> 5120 (two quantized linears per step).

Prints ONE JSON line (rank 0).  Kernel durations come from HIP events recorded on the stream
the kernels are launched on (torch's current stream).
"""

import argparse
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "orbit_qlinear TFLOP/s + rpbh_quantize_act GB/s (% of MI355X roofline)"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak (the same for fp16)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=25)
    ap.add_argument("--workload", default="c4_video_mlp_w4a4", choices=["c4_video_mlp_w4a4", "c1_single_w4a4"])
    ap.add_argument("--cpu-baseline-rows", type=int, default=12288,
                    help="token rows of the oracle's timed CPU sample (0 disables it)")
    ap.add_argument("--trunk-steps", type=int, default=2,
                    help="timed steps of the 40-block video trunk sweep (config 5); 0 skips it")
    ap.add_argument("--adaln-steps", type=int, default=10,
                    help="timed steps of the AdaLN INT4 modulation projections (FLUX-shaped); 0 skips them")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run one plain device-to-device copy of this many MiB before the step, so that a "
                         "counter profile of this run holds a kernel of known traffic to scale by")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="per-kernel HBM bytes measured with rocprofv3 counters (optional)")
    ap.add_argument("--part-reps", type=int, default=10,
                    help="timed launches of each layer kernel on its own (the roofline's per-kernel times)")
    ap.add_argument("--config-reps", type=int, default=10,
                    help="timed launches per linear of the other workloads' configurations (0 skips them)")
    ap.add_argument("--image-reps", type=int, default=10,
                    help="timed launches per shape of the per-image rotation cost (0 skips it)")
    ap.add_argument("--cpu-one-thread-rows", type=int, default=1536,
                    help="token rows of the oracle's single-thread CPU sample (0 disables it)")
    ap.add_argument("--extras", type=int, default=1,
                    help="0 skips the entries after the step (block-size rule, rotation classes, fused "
                         "epilogue, MLP chain, W4A6), e.g. for counter profiles of the step alone")
    ap.add_argument("--cpu-baseline-worker", default=None, help=argparse.SUPPRESS)
    return ap.parse_args()


def source_digest():
    """Digest of the kernel sources; traffic counters taken from other sources are not used."""
    import hashlib
    h = hashlib.sha256()
    for f in ("rpbh_quantize.hip", "rpbh_quantize_row.hip", "lut_gemm.hip"):
        with open(os.path.join(ROOT, "paper_2607_02461_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def quant_bytes(M, K, bits):
    """Algorithmic bytes of one quantizer launch: bf16 rows in, packed codes + fp32 norms out."""
    return M * (2 * K + K * bits // 8 + 4)


def main():
    args = parse()
    if args.cpu_baseline_worker:
        cpu_baseline_worker(args.cpu_baseline_worker)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; --gpus must be 1 "
                                   "(rows shard across GPUs with no exchange, see the design notes)"}))
        sys.exit(2)
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(2)

    import paper_2607_02461_amd as oq
    from paper_2607_02461_amd import workloads

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = workloads.WORKLOADS[args.workload]

    # ---- inputs (synthetic, seeded) ------------------------------------------------------
    if wl is workloads.C4:
        Xu, Xd, Wu, Wd = workloads.c4_inputs(device=dev)
        lin_inputs = [(wl.linears[0], Xu, Wu), (wl.linears[1], Xd, Wd)]
    else:
        X, W = workloads.c1_inputs(device=dev)
        lin_inputs = [(wl.linears[0], X, W)]
    torch.cuda.synchronize()

    # ---- offline stage: plans + codebooks on the host, weight pass on the GPU -------------
    t0 = time.perf_counter()
    plans, cbs = {}, {}
    for lin, _, _ in lin_inputs:
        plans[lin.K] = oq.rpbh_plan(lin.K, lin.h, wl.plan_seed)
        cbs[(lin.ba, lin.K)] = oq.lloydmax_codebook(lin.ba, lin.K)
        cbs[(lin.bw, lin.K)] = oq.lloydmax_codebook(lin.bw, lin.K)
    host_offline_s = time.perf_counter() - t0

    layers = []
    for lin, X, W in lin_inputs:
        wc = torch.empty((lin.N, lin.K * lin.bw // 8), dtype=torch.uint8, device=dev)
        wn = torch.empty((lin.N,), dtype=torch.bfloat16, device=dev)
        xc = torch.empty((lin.M, lin.K * lin.ba // 8), dtype=torch.uint8, device=dev)
        xn = torch.empty((lin.M,), dtype=torch.float32, device=dev)
        Y = torch.empty((lin.M, lin.N), dtype=torch.float32, device=dev)
        # the K-split workspace of the rows the 128x128 kernel runs (c1: all; c4 down: its last 504)
        wsp = torch.empty(max(16, oq.orbit_qlinear_workspace_size(lin.M, lin.N, lin.K)), dtype=torch.uint8,
                          device=dev)
        layers.append(dict(lin=lin, X=X, W=W, wc=wc, wn=wn, xc=xc, xn=xn, Y=Y, ws=wsp,
                           plan=plans[lin.K], cba=cbs[(lin.ba, lin.K)], cbw=cbs[(lin.bw, lin.K)]))

    def weight_pass():
        for L in layers:
            oq.quantize_weights_offline(L["plan"], L["cbw"], L["W"], 1e-10, L["wc"], L["wn"])

    weight_pass()  # also uploads the plan tables
    torch.cuda.synchronize()
    wp_reps = 5
    ws, we = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ws.record()
    for _ in range(wp_reps):
        weight_pass()
    we.record()
    torch.cuda.synchronize()
    weight_pass_ms = ws.elapsed_time(we) / wp_reps
    weight_bytes = sum(L["lin"].N * (2 * L["lin"].K + L["lin"].K * L["lin"].bw // 8 + 2) for L in layers)

    # a plain device-to-device copy: the attainable HBM rate beside the 8 TB/s peak, and (with
    # --copy-calibration-mib) a kernel of known traffic in counter profiles of this run
    copy_mib = args.copy_calibration_mib if args.copy_calibration_mib > 0 else 1024
    src = torch.empty(copy_mib << 20, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record()
    for _ in range(5):
        dst.copy_(src)
    c1.record()
    torch.cuda.synchronize()
    copy_ms = c0.elapsed_time(c1) / 5
    hbm_copy = {"bytes_read_plus_written": 2 * (copy_mib << 20), "ms": copy_ms,
                "gbs": 2 * (copy_mib << 20) / (copy_ms * 1e-3) / 1e9,
                "frac_of_hbm": 2 * (copy_mib << 20) / (copy_ms * 1e-3) / 1e9 / HBM_PEAK_GBS}
    del src, dst

    # ---- the step --------------------------------------------------------------------------
    nl = len(layers)

    def step(ev=None):
        for i, L in enumerate(layers):
            if ev is not None:
                ev[4 * i].record()
            oq.rpbh_quantize_act(L["plan"], L["cba"], L["X"], 1e-10, L["xc"], L["xn"])
            if ev is not None:
                ev[4 * i + 1].record()
                ev[4 * i + 2].record()
            oq.orbit_qlinear_ws(L["cba"], L["xc"], L["xn"], L["cbw"], L["wc"], L["wn"], L["ws"], out=L["Y"])
            if ev is not None:
                ev[4 * i + 3].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4 * nl)] for _ in range(args.steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall0 = time.perf_counter()
    start.record()
    for s in range(args.steps):
        step(events[s])
    end.record()
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - t_wall0
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / args.steps

    q_all = np.array([[ev[4 * i].elapsed_time(ev[4 * i + 1]) for i in range(nl)] for ev in events])
    g_all = np.array([[ev[4 * i + 2].elapsed_time(ev[4 * i + 3]) for i in range(nl)] for ev in events])
    quant_ms = q_all.mean(axis=0)
    gemm_ms = g_all.mean(axis=0)

    flops = np.array([2.0 * L["lin"].M * L["lin"].N * L["lin"].K for L in layers])
    qbytes = np.array([quant_bytes(L["lin"].M, L["lin"].K, L["lin"].ba) for L in layers], dtype=np.float64)
    gemm_tflops = flops.sum() / (gemm_ms.sum() * 1e-3) / 1e12
    quant_gbs = qbytes.sum() / (quant_ms.sum() * 1e-3) / 1e9
    step_tflops = flops.sum() / (ms_per_step * 1e-3) / 1e12

    traffic = None
    if os.path.exists(args.traffic):
        try:
            t = json.load(open(args.traffic))
            if t.get("workload") == wl.name and t.get("source_digest") == source_digest():
                traffic = t
        except (OSError, ValueError):
            traffic = None

    # The layer's kernels, each launch timed alone with HIP events on the stream it runs on: the
    # rows the 256x256 kernel takes and the rows the 128x128 kernel takes (split over K with the
    # workspace, then the reduction), as orbit_qlinear_schedule names them
    parts = [p for L in layers for p in gemm_parts(oq, L, args.part_reps)]
    dom = [p for p in parts if p["kernel"].startswith("lut_gemm_big")]
    if not dom:   # a layer too small for the large kernel (c1): its split kernel pair dominates
        dom = parts
    dom_flops = sum(p["flops"] for p in dom)
    dom_ms = sum(p["ms"] for p in dom)
    roofline = {
        "kernel": dom[0]["kernel"],
        "bound": "mfma",
        "achieved": dom_flops / (dom_ms * 1e-3) / 1e12,
        "peak": MFMA_PEAK_TFLOPS,
        "unit": "TFLOP/s",
        "frac": dom_flops / (dom_ms * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS,
        "traffic": (traffic or {}).get("gemm_bytes_per_launch"),
        "achieved_is": "2*rows*N*K of each launch of this kernel in the step / its HIP-event launch time, "
                       "over the launches listed in 'launches'",
        "launches": [p for p in parts if p["kernel"] == dom[0]["kernel"]],
        "other_launches": [p for p in parts if p["kernel"] != dom[0]["kernel"]],
        "call_ms_in_step": [float(v) for v in gemm_ms],
        "workspace_bytes": [oq.orbit_qlinear_workspace_size(L["lin"].M, L["lin"].N, L["lin"].K) for L in layers],
    }
    # The quantizer's launches timed alone as well (back to back between one event pair); inside the
    # step each one follows a GEMM, whose power draw holds the clock down for a while.
    # Rows of K = 1024 .. 16384 (a multiple of 128 and of h) with h = 128 .. 1024 run the
    # one-row-per-workgroup kernel; its last template argument is log2(h / 128).
    q_alone = []
    for L in layers:
        fn = (lambda L=L: oq.rpbh_quantize_act(L["plan"], L["cba"], L["X"], 1e-10, L["xc"], L["xn"]))
        q_alone.append(_timed_back_to_back(fn, args.part_reps))
    qkern = [(f"rpbh_quantize_row_kernel<{L['lin'].ba}, false, {L['lin'].h.bit_length() - 8}>"
              if 128 <= L["lin"].h <= 1024 and L["lin"].K % 128 == 0 and L["lin"].K % L["lin"].h == 0
              and 1024 <= L["lin"].K <= 16384 else
              f"rpbh_quantize_kernel<{L['lin'].ba}, false, {'true' if L['lin'].h > 128 else 'false'}, true>")
             for L in layers]
    qa_gbs = float(qbytes.sum()) / (sum(q_alone) * 1e-3) / 1e9
    roofline_q = {
        "kernel": qkern[0] if len(set(qkern)) == 1 else qkern,
        "bound": "hbm",
        "achieved": qa_gbs,
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": qa_gbs / HBM_PEAK_GBS,
        "traffic": (traffic or {}).get("quant_bytes_per_launch"),
        "achieved_is": "algorithmic bytes of the step's quantizer launches / their average HIP-event time, each "
                       "layer's launch repeated back to back between one event pair; 'in_step' gives the same "
                       "launches inside the step",
        "launches": [{"linear": L["lin"].name, "M": L["lin"].M, "K": L["lin"].K, "bits": L["lin"].ba,
                      "ms": q_alone[i], "algorithmic_bytes": float(qbytes[i]),
                      "gbs": float(qbytes[i]) / (q_alone[i] * 1e-3) / 1e9,
                      "frac": float(qbytes[i]) / (q_alone[i] * 1e-3) / 1e9 / HBM_PEAK_GBS}
                     for i, L in enumerate(layers)],
        "in_step": {"gbs": quant_gbs, "frac": quant_gbs / HBM_PEAK_GBS, "ms": [float(v) for v in quant_ms]},
        "attainable_copy_gbs": hbm_copy["gbs"],
    }

    paper_h = rot = fused = chain = a6 = None
    if args.extras:
        paper_h, rot, fused, chain, a6 = extras_entries(oq, workloads, wl, dev, layers, flops, gemm_ms)
        # the rule's rate against the same layer's h = 128 launch, both timed back to back
        for i, L in enumerate(layers):
            e = paper_h[L["lin"].name]
            e["rate_vs_h128"] = q_alone[i] / e["ms"]
        # what the vendor library's dense bf16 matmul attains on the same shapes (context for the
        # GEMM's fraction of the nominal peak)
        dn = rot["dense_bf16_matmul"]
        roofline["attainable_dense_bf16_matmul_tflops"] = {L["lin"].name: dn[L["lin"].name]["tflops"] for L in layers}

    configs = None
    if args.config_reps > 0:
        configs = configs_sweep(oq, workloads, dev, args.config_reps)

    per_image = None
    if args.image_reps > 0:
        per_image = rotation_per_image(oq, dev, args.image_reps)

    adaln = None
    if args.adaln_steps > 0:
        adaln = adaln_sweep(oq, workloads, dev, args.adaln_steps)

    trunk = None
    if args.trunk_steps > 0:
        trunk = trunk_sweep(oq, workloads, dev, args.trunk_steps)

    cpu = None
    if args.cpu_baseline_rows > 0:
        step()                     # the step's own outputs back in place (later entries reused buffers)
        torch.cuda.synchronize()
        cpu = cpu_baseline(layers, args.cpu_baseline_rows, one_thread_rows=args.cpu_one_thread_rows, parity=True)

    out = {
        "metric": METRIC,
        "value": step_tflops,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": wl.name,
            "description": wl.description,
            "linears": [{"name": L["lin"].name, "M": L["lin"].M, "K": L["lin"].K, "N": L["lin"].N,
                         "bits": f"W{L['lin'].bw}A{L['lin'].ba}", "h": L["lin"].h} for L in layers],
            "value_is": "GEMM flops of the step / step time (quantizer + GEMM per linear)",
            "arith": "quantizer fp32; GEMM bf16 MFMA operands (levels dequantized to bf16), fp32 accumulate",
            # inputs above the 256 MB Infinity Cache stream from HBM on every step
            "cache": "cold" if min(L["X"].numel() * 2 for L in layers) > (256 << 20) else "warm",
        },
        "components": {
            "orbit_qlinear_tflops": gemm_tflops,
            "orbit_qlinear_frac_of_bf16_peak": gemm_tflops / MFMA_PEAK_TFLOPS,
            "rpbh_quantize_act_gbs": quant_gbs,
            "rpbh_quantize_act_frac_of_hbm": quant_gbs / HBM_PEAK_GBS,
            "quant_ms": [float(v) for v in quant_ms],
            "gemm_ms": [float(v) for v in gemm_ms],
            "quant_ms_median": [float(v) for v in np.median(q_all, axis=0)],
            "quant_ms_min": [float(v) for v in q_all.min(axis=0)],
            "gemm_ms_median": [float(v) for v in np.median(g_all, axis=0)],
            "gemm_ms_min": [float(v) for v in g_all.min(axis=0)],
            "weight_pass_ms": weight_pass_ms,
            "weight_pass_gbs": weight_bytes / (weight_pass_ms * 1e-3) / 1e9,
            "host_plan_codebook_s": host_offline_s,
            "wall_s_timed_region": wall_s,
        },
        "roofline": roofline,
        "roofline_quantizer": roofline_q,
        "hbm_copy": hbm_copy,
        "parity": (cpu or {}).pop("parity", None),
        "configs": configs,
        "rotation_per_image": per_image,
        "quantizer_paper_block_rule": paper_h,
        "rotation_classes": rot,
        "fused_epilogue": fused,
        "mlp_chain": chain,
        "w4a6": a6,
        "trunk_c5": trunk,
        "adaln_int4": adaln,
        "cpu_baseline": cpu,
        "env": {"torch": torch.__version__, "hip": torch.version.hip, "device": torch.cuda.get_device_name(0),
                "host_cpu_count": os.cpu_count(),
                "arch": torch.cuda.get_device_properties(0).gcnArchName,
                "compute_units": torch.cuda.get_device_properties(0).multi_processor_count,
                "memory_gib": torch.cuda.get_device_properties(0).total_memory / 2 ** 30},
    }
    print(json.dumps(out), flush=True)


def extras_entries(oq, workloads, wl, dev, layers, flops, gemm_ms):
    """The entries after the step: the paper's block-size rule, the rotation classes, the fused
    epilogue, the MLP chain and the W4A6 recipe, each timed on the step's own inputs."""
    # NEXT row: the activation quantizer with the paper's block-size rule (largest power of two
    # dividing d: 1024 for 5120, 512 for 13824), same inputs, timed alone
    paper_h = {}
    for L in layers:
        lin = L["lin"]
        plan_p = oq.rpbh_plan(lin.K, 0, wl.plan_seed)
        _warm(lambda: oq.rpbh_quantize_act(plan_p, L["cba"], L["X"], 1e-10, L["xc"], L["xn"]))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(10):
            oq.rpbh_quantize_act(plan_p, L["cba"], L["X"], 1e-10, L["xc"], L["xn"])
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 10
        qb = quant_bytes(lin.M, lin.K, lin.ba)
        paper_h[lin.name] = {"h": plan_p.h, "ms": ms, "gbs": qb / (ms * 1e-3) / 1e9,
                             "frac_of_hbm": qb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}

    # NEXT row: the rotation classes of the paper's ablation (Table 4), on the up-projection input:
    # fused quantizer time with RPBH and with Block-RHT (RPBH without the permutation) at h = 128
    # and at the paper's rule, and the dense-rotation alternative as a bf16 GEMM X Q^T (rotation
    # only, the cost the structured rotations avoid)
    L0 = layers[0]
    K0 = L0["lin"].K

    def time_quant(plan_v, reps=10, X=None, cb=None, xc=None, xn=None):
        X = L0["X"] if X is None else X
        cb, xc, xn = (L0["cba"], L0["xc"], L0["xn"]) if cb is None else (cb, xc, xn)
        _warm(lambda: oq.rpbh_quantize_act(plan_v, cb, X, 1e-10, xc, xn))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            oq.rpbh_quantize_act(plan_v, cb, X, 1e-10, xc, xn)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    rot = {}
    for hh in (128, 0):
        pr = oq.rpbh_plan(K0, hh, wl.plan_seed)
        _, signs = pr.arrays()
        pb = oq.rpbh_plan_from_arrays(K0, pr.h, np.arange(K0), signs)
        rot[f"rpbh_h{pr.h}_ms"] = time_quant(pr)
        rot[f"block_rht_h{pr.h}_ms"] = time_quant(pb)
    # the Haar rotation itself is drawn on the host: only its application is timed
    gq = torch.Generator()
    gq.manual_seed(7)
    Q, _ = torch.linalg.qr(torch.randn((K0, K0), generator=gq, dtype=torch.float32))
    Qt = Q.t().contiguous().to(torch.bfloat16).to(dev)
    del Q
    Xr = torch.empty((L0["lin"].M, K0), dtype=torch.bfloat16, device=dev)
    _warm(lambda: torch.matmul(L0["X"], Qt, out=Xr))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        torch.matmul(L0["X"], Qt, out=Xr)
    e1.record()
    torch.cuda.synchronize()
    rot["dense_haar_rotation_gemm_ms"] = e0.elapsed_time(e1) / 5
    rot["shape"] = f"{L0['lin'].M} x {K0}"
    del Qt, Xr
    # The paper's own layer computation (fake quantization): operands dequantized to BF16 and the
    # matmul in BF16.  The matmul alone, by the vendor library (hipBLASLt through torch), on each
    # layer's shape with its bf16 inputs, beside the LUT-decode GEMM's launches on the same shape.
    dense = {"what": "torch.matmul (hipBLASLt) of the layer's bf16 X and bf16 W^T into bf16, the matmul of the "
                     "paper's dequantize-then-BF16 path without its dequantization passes"}
    for L in layers:
        lin = L["lin"]
        Wt = L["W"].t().contiguous()
        Yd = torch.empty((lin.M, lin.N), dtype=torch.bfloat16, device=dev)
        ms = _timed_back_to_back(lambda: torch.matmul(L["X"], Wt, out=Yd), 5)
        dense[lin.name] = {"M": lin.M, "K": lin.K, "N": lin.N, "ms": ms,
                           "tflops": 2.0 * lin.M * lin.N * lin.K / (ms * 1e-3) / 1e12}
        del Wt, Yd
    # Full RHT (one Hadamard block over the whole row, no permutation) needs a power-of-two d: the
    # first 4096 channels of the same input (a strided view; 2048 of c1's 3072), against RPBH and
    # Block-RHT there
    K1 = 4096 if K0 >= 4096 else 2048
    X1 = L0["X"][:, :K1]
    cb1 = oq.lloydmax_codebook(L0["lin"].ba, K1)
    xc1 = torch.empty((L0["lin"].M, K1 * L0["lin"].ba // 8), dtype=torch.uint8, device=dev)
    xn1 = torch.empty((L0["lin"].M,), dtype=torch.float32, device=dev)
    d4 = {"shape": f"{L0['lin'].M} x {K1}"}
    for hh in (128, K1):
        pr = oq.rpbh_plan(K1, hh, wl.plan_seed)
        _, signs = pr.arrays()
        pb = oq.rpbh_plan_from_arrays(K1, hh, np.arange(K1), signs)
        d4[f"rpbh_h{hh}_ms"] = time_quant(pr, X=X1, cb=cb1, xc=xc1, xn=xn1)
        d4[f"{'full_rht' if hh == K1 else 'block_rht'}_h{hh}_ms"] = time_quant(pb, X=X1, cb=cb1, xc=xc1, xn=xn1)
    rot[f"d{K1}"] = d4
    del xc1, xn1

    # NEXT row: the up-projection with the MLP's GELU and a bf16 output fused into the epilogue
    # (the form that feeds the next quantizer), against the plain fp32 GEMM on the same codes
    Yb = torch.empty((L0["lin"].M, L0["lin"].N), dtype=torch.bfloat16, device=dev)
    _warm(lambda: oq.orbit_qlinear_ws(L0["cba"], L0["xc"], L0["xn"], L0["cbw"], L0["wc"], L0["wn"], L0["ws"],
                                      gelu=True, out_dtype=torch.bfloat16, out=Yb))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        oq.orbit_qlinear_ws(L0["cba"], L0["xc"], L0["xn"], L0["cbw"], L0["wc"], L0["wn"], L0["ws"], gelu=True,
                            out_dtype=torch.bfloat16, out=Yb)
    e1.record()
    torch.cuda.synchronize()
    fused_ms = e0.elapsed_time(e1) / 5
    fused = {"linear": L0["lin"].name, "epilogue": "GELU(erf) + bf16 output", "ms": fused_ms,
             "tflops": float(flops[0]) / (fused_ms * 1e-3) / 1e12, "plain_fp32_ms": float(gemm_ms[0])}

    # NEXT row: the MLP as a model runs it, the fused up-projection's bf16 output feeding the
    # down-projection's quantizer directly, against the same chain with an fp32 up output, GELU
    # and the bf16 cast as separate torch ops
    chain = None
    if len(layers) > 1:   # c4's two projections (c1 is a single linear)
        L1 = layers[1]
        H = Yb

        def chain_fused():
            oq.rpbh_quantize_act(L0["plan"], L0["cba"], L0["X"], 1e-10, L0["xc"], L0["xn"])
            oq.orbit_qlinear_ws(L0["cba"], L0["xc"], L0["xn"], L0["cbw"], L0["wc"], L0["wn"], L0["ws"], gelu=True,
                                out_dtype=torch.bfloat16, out=H)
            oq.rpbh_quantize_act(L1["plan"], L1["cba"], H, 1e-10, L1["xc"], L1["xn"])
            oq.orbit_qlinear_ws(L1["cba"], L1["xc"], L1["xn"], L1["cbw"], L1["wc"], L1["wn"], L1["ws"], out=L1["Y"])

        def chain_unfused():
            oq.rpbh_quantize_act(L0["plan"], L0["cba"], L0["X"], 1e-10, L0["xc"], L0["xn"])
            oq.orbit_qlinear_ws(L0["cba"], L0["xc"], L0["xn"], L0["cbw"], L0["wc"], L0["wn"], L0["ws"], out=L0["Y"])
            H.copy_(torch.nn.functional.gelu(L0["Y"]))
            oq.rpbh_quantize_act(L1["plan"], L1["cba"], H, 1e-10, L1["xc"], L1["xn"])
            oq.orbit_qlinear_ws(L1["cba"], L1["xc"], L1["xn"], L1["cbw"], L1["wc"], L1["wn"], L1["ws"], out=L1["Y"])

        chain = {"layers": f"{L0['lin'].name} -> GELU -> {L1['lin'].name}"}
        for name, fn in (("fused_ms", chain_fused), ("unfused_ms", chain_unfused)):
            _warm(fn)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(3):
                fn()
            e1.record()
            torch.cuda.synchronize()
            chain[name] = e0.elapsed_time(e1) / 3
        chain["fused_tflops"] = float(flops[0] + flops[1]) / (chain["fused_ms"] * 1e-3) / 1e12
    del Yb

    # NEXT row: the video recipe's 6-bit activations (W4A6, the paper's Wan setting) on the
    # up-projection: the quantizer writing 6-bit codes and the GEMM decoding them
    cb6 = oq.lloydmax_codebook(6, K0)
    xc6 = torch.empty((L0["lin"].M, K0 * 6 // 8), dtype=torch.uint8, device=dev)
    plan0 = L0["plan"]
    _warm(lambda: oq.rpbh_quantize_act(plan0, cb6, L0["X"], 1e-10, xc6, L0["xn"]))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        oq.rpbh_quantize_act(plan0, cb6, L0["X"], 1e-10, xc6, L0["xn"])
    e1.record()
    torch.cuda.synchronize()
    q6_ms = e0.elapsed_time(e1) / 10
    _warm(lambda: oq.orbit_qlinear(cb6, xc6, L0["xn"], L0["cbw"], L0["wc"], L0["wn"], L0["Y"]))
    e0.record()
    for _ in range(5):
        oq.orbit_qlinear(cb6, xc6, L0["xn"], L0["cbw"], L0["wc"], L0["wn"], L0["Y"])
    e1.record()
    torch.cuda.synchronize()
    g6_ms = e0.elapsed_time(e1) / 5
    q6_bytes = quant_bytes(L0["lin"].M, K0, 6)
    a6 = {"linear": L0["lin"].name, "quant_ms": q6_ms, "quant_gbs": q6_bytes / (q6_ms * 1e-3) / 1e9,
          "gemm_ms": g6_ms, "gemm_tflops": float(flops[0]) / (g6_ms * 1e-3) / 1e12}
    del xc6

    rot["dense_bf16_matmul"] = dense
    return paper_h, rot, fused, chain, a6


# Untimed work ahead of each per-launch measurement.  After an idle spell the GPU's clock takes tens
# of milliseconds of load to come back: c4-shaped GEMMs issued after 2 s idle ran 18% slower than
# in steady state over their first ~12 ms and 4% slower over the next 12 ms.
WARM_MS = 100.0


def _warm(fn, before=None, min_ms=WARM_MS):
    """Untimed launches of fn (each after `before`) until at least min_ms of wall time has passed."""
    t0 = time.perf_counter()
    n = 1
    while True:
        for _ in range(n):
            if before is not None:
                before()
            fn()
        torch.cuda.synchronize()
        if (time.perf_counter() - t0) * 1e3 >= min_ms:
            return
        n = min(2 * n, 64)


def _timed_back_to_back(fn, reps):
    """Average time of one of `reps` launches of fn issued back to back between one pair of HIP
    events on the current stream (after WARM_MS of untimed launches): the rate of a kernel run in a
    sequence, without an event pair around every launch (which adds several microseconds to a
    0.1 ms launch)."""
    _warm(fn)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def _timed(fn, reps, before=None):
    """Mean, median and minimum of `reps` launches of fn, each bracketed by its own HIP events on the
    current stream; `before` (untimed) runs ahead of each launch, and WARM_MS of both ahead of the
    first."""
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    _warm(fn, before)
    for e0, e1 in ev:
        if before is not None:
            before()
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    t = np.array([e0.elapsed_time(e1) for e0, e1 in ev])
    return float(t.mean()), float(np.median(t)), float(t.min())


def gemm_parts(oq, L, reps):
    """The kernel launches of one layer call, each timed alone: rows [0, rows_large) on the 256x256
    kernel, then rows [rows_large, M) on the 128x128 kernel, split over K with the layer's workspace
    and followed by the reduction when the schedule splits them.  Each part is the same launch the
    whole call makes (the same rows, operands and split)."""
    lin = L["lin"]
    M, N, K = lin.M, lin.N, lin.K
    rows, splits = oq.orbit_qlinear_schedule(M, N, K)
    out = []
    for r0, r1 in ((0, rows), (rows, M)):
        if r1 <= r0:
            continue
        xc, xn, Y = L["xc"][r0:r1], L["xn"][r0:r1], L["Y"][r0:r1]
        big = r0 == 0 and rows > 0

        def call():
            oq.orbit_qlinear_ws(L["cba"], xc, xn, L["cbw"], L["wc"], L["wn"], L["ws"], out=Y)

        mean, med, mn = _timed(call, reps)
        fl = 2.0 * (r1 - r0) * N * K
        name = (f"lut_gemm_big<{lin.ba},{lin.bw}>" if big else
                f"lut_gemm_kernel<{lin.ba},{lin.bw},{'true' if splits > 1 else 'false'}>"
                + ("+lut_gemm_reduce" if splits > 1 else ""))
        out.append({"linear": lin.name, "kernel": name, "rows": [r0, r1], "N": N, "K": K, "splits": 1 if big else splits,
                    "flops": fl, "ms": mean, "ms_median": med, "ms_min": mn,
                    "tflops": fl / (mean * 1e-3) / 1e12, "frac": fl / (mean * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS})
    return out


def configs_sweep(oq, workloads, dev, reps):
    """Every linear of the other workload configurations at its bit pair, the quantizer and the layer
    each timed launch by launch: the single layer (c1), the image-DiT MLP at W4A4 and W3A4 (c2,
    timestep 0), the image-DiT attention projections at W2A4 and W3A3 (c3), and the video recipe's
    W4A6 on the c4 up-projection.  Inputs smaller than the 256 MB Infinity Cache are evicted before
    each timed launch by writing a 512 MB buffer, so every launch streams its operands from HBM."""
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)

    def evict():
        flush.fill_(0)

    jobs = []
    X1, W1 = workloads.c1_inputs(device=dev)
    jobs.append(("c1_single_w4a4", workloads.C1.linears[0], X1, W1, workloads.C1.plan_seed))
    Xu, Xd = workloads.c2_up_acts(0, device=dev), workloads.c2_down_acts(0, device=dev)
    Wu, Wd = workloads.c2_weights(device=dev)
    for lin in workloads.C2.linears:
        X, W = (Xu, Wu) if lin.name.startswith("up") else (Xd, Wd)
        jobs.append(("c2_image_mlp", lin, X, W, workloads.C2.plan_seed))
    Xq, Xo, Wq, Wo = workloads.c3_inputs(device=dev)
    for lin in workloads.C3.linears:
        X, W = (Xq, Wq) if lin.name.startswith("qkv") else (Xo, Wo)
        jobs.append(("c3_image_attn", lin, X, W, workloads.C3.plan_seed))
    fr, tpf, txt = workloads.C4.extra["frames"], workloads.C4.extra["tokens_per_frame"], workloads.C4.extra["text_tokens"]
    up = workloads.C4.linears[0]
    X4 = workloads.video_acts(fr * tpf, txt, up.K, 4, fr, workloads.C4.data_seed, 0, device=dev)
    W4 = workloads.gaussian_weights(up.N, up.K, 0.015, workloads.C4.data_seed, 0, device=dev)
    jobs.append(("c4_video_mlp_w4a6", workloads.Linear("up_w4a6", up.M, up.K, up.N, 4, 6), X4, W4,
                 workloads.C4.plan_seed))

    res = []
    for wname, lin, X, W, seed in jobs:
        plan = oq.rpbh_plan(lin.K, lin.h, seed)
        cba, cbw = oq.lloydmax_codebook(lin.ba, lin.K), oq.lloydmax_codebook(lin.bw, lin.K)
        wc, wn = oq.quantize_weights_offline(plan, cbw, W)
        xc = torch.empty((lin.M, lin.K * lin.ba // 8), dtype=torch.uint8, device=dev)
        xn = torch.empty((lin.M,), dtype=torch.float32, device=dev)
        Y = torch.empty((lin.M, lin.N), dtype=torch.float32, device=dev)
        ws = torch.empty(max(16, oq.orbit_qlinear_workspace_size(lin.M, lin.N, lin.K)), dtype=torch.uint8, device=dev)
        cold = X.numel() * 2 > (256 << 20)
        q = _timed(lambda: oq.rpbh_quantize_act(plan, cba, X, 1e-10, xc, xn), reps, None if cold else evict)
        g = _timed(lambda: oq.orbit_qlinear_ws(cba, xc, xn, cbw, wc, wn, ws, out=Y), reps, evict)
        qb = quant_bytes(lin.M, lin.K, lin.ba)
        fl = 2.0 * lin.M * lin.N * lin.K
        rows, splits = oq.orbit_qlinear_schedule(lin.M, lin.N, lin.K)
        res.append({"workload": wname, "linear": lin.name, "M": lin.M, "K": lin.K, "N": lin.N,
                    "bits": f"W{lin.bw}A{lin.ba}", "h": lin.h, "schedule": {"rows_large": rows, "splits": splits},
                    "quant_ms": q[0], "quant_ms_min": q[2], "quant_gbs": qb / (q[0] * 1e-3) / 1e9,
                    "quant_frac_of_hbm": qb / (q[0] * 1e-3) / 1e9 / HBM_PEAK_GBS,
                    "gemm_ms": g[0], "gemm_ms_min": g[2], "gemm_tflops": fl / (g[0] * 1e-3) / 1e12,
                    "gemm_frac_of_bf16_peak": fl / (g[0] * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS})
        del wc, wn, xc, xn, Y, ws
    del flush
    return {"cache": "cold: operands below 256 MB evicted before every timed launch", "linears": res}


# FLUX.1-shaped image DiT at 1024^2 (hidden 3072, MLP 12288): the activation inputs the quantized
# projections read per denoising step, as (tokens, d, count).  Each of the 19 double-stream blocks
# has an image stream (4096 tokens) and a text stream (512 tokens), each reading three inputs of
# width 3072 (attention QKV, attention output, FFN up) and one of 12288 (FFN down); each of the 38
# single-stream blocks (4608 tokens) reads one of 3072 (its fused QKV and FFN up) and one of
# 3072 + 12288 = 15360 (its fused output projection).  4 steps per image (the schnell sampler).
FLUX_ROTATION_INPUTS = ((4096, 3072, 19 * 3), (4096, 12288, 19), (512, 3072, 19 * 3), (512, 12288, 19),
                        (4608, 3072, 38), (4608, 15360, 38))
FLUX_STEPS = 4
# the paper's per-image activation-rotation latency on one H100 (FLUX.1-schnell, 1024^2), seconds
PAPER_H100_ROTATION_S = {"rpbh": 0.451, "block_rht": 0.381, "full_rht": 0.452, "dense_haar": 11.65}


def rotation_per_image(oq, dev, reps):
    """Analogue of the paper's per-image activation-rotation latency (FLUX.1-schnell at 1024^2, all
    quantized layers and steps): for each rotation class, the fused quantizer (rotation, norm, 4-bit
    encode) timed once per input shape, times how often a step reads that shape, times 4 steps.
    Dense Haar is the rotation alone, a bf16 GEMM X Q^T with a d x d matrix (a random one: the GEMM's
    time does not depend on Q being orthogonal).  Inputs are synthetic N(0, 1) rows, timed back to
    back (warm: in a model each input was just written by the previous layer)."""
    g = torch.Generator(device=dev)
    g.manual_seed(11)
    per_shape, tot = [], {"rpbh_h128": 0.0, "rpbh_paper_rule": 0.0, "block_rht_h128": 0.0,
                          "block_rht_paper_rule": 0.0, "dense_haar": 0.0}
    for M, d, count in FLUX_ROTATION_INPUTS:
        X = torch.randn((M, d), generator=g, device=dev).to(torch.bfloat16)
        cb = oq.lloydmax_codebook(4, d)
        xc = torch.empty((M, d // 2), dtype=torch.uint8, device=dev)
        xn = torch.empty((M,), dtype=torch.float32, device=dev)
        row = {"M": M, "d": d, "per_step": count}
        for hh, tag in ((128, "h128"), (0, "paper_rule")):
            pr = oq.rpbh_plan(d, hh, 0)
            _, signs = pr.arrays()
            pb = oq.rpbh_plan_from_arrays(d, pr.h, np.arange(d), signs)
            for name, plan in (("rpbh", pr), ("block_rht", pb)):
                ms = _timed_back_to_back(lambda: oq.rpbh_quantize_act(plan, cb, X, 1e-10, xc, xn), reps)
                row[f"{name}_{tag}_ms"] = ms
                row[f"{name}_{tag}_h"] = pr.h
                tot[f"{name}_{tag}"] += ms * count * FLUX_STEPS
        Q = (torch.randn((d, d), generator=g, device=dev) / d ** 0.5).to(torch.bfloat16)
        Xr = torch.empty((M, d), dtype=torch.bfloat16, device=dev)
        ms = _timed_back_to_back(lambda: torch.matmul(X, Q, out=Xr), max(3, reps // 2))
        row["dense_haar_ms"] = ms
        tot["dense_haar"] += ms * count * FLUX_STEPS
        per_shape.append(row)
        del X, xc, xn, Q, Xr
    return {"model": "FLUX.1-shaped image DiT, 1024^2, 4 steps, 4608 tokens (4096 image + 512 text)",
            "seconds_per_image": {k: v * 1e-3 for k, v in tot.items()},
            "quantizer_includes": "rotation + norm + 4-bit Lloyd-Max encode and pack (the fused kernel)",
            "paper_h100_rotation_only_s": PAPER_H100_ROTATION_S,
            "shapes": per_shape}


def trunk_sweep(oq, workloads, dev, steps, warmup=1):
    """The video-DiT trunk sweep: per denoising step, the activation quantizer and the GEMM of
    every linear of 40 blocks (QKV, out, FFN up, FFN down at M = 32760), summed over the 160
    calls; and the offline weight pass over all 160 weight matrices.  Every layer of input width d
    shares the one rotation Pi_d (Sec. 4.2), so the weight rows of one width form one row set: the
    pass quantizes it in one launch per width (two here), each matrix's codes and norms being a row
    range of the result.  The same pass as 160 launches, one per matrix, is timed beside it.
    Weights are generated outside the timing.  One activation draw per input width serves every
    block."""
    wl = workloads.C5
    acts = workloads.c5_acts(device=dev)
    M = workloads.C5_M
    plans = {K: oq.rpbh_plan(K, 128, wl.plan_seed) for K in acts}
    cbs = {K: oq.lloydmax_codebook(4, K) for K in acts}
    xc = {K: torch.empty((M, K // 2), dtype=torch.uint8, device=dev) for K in acts}
    xn = {K: torch.empty((M,), dtype=torch.float32, device=dev) for K in acts}
    Yflat = torch.empty(max(M * lin.N for lin in wl.linears), dtype=torch.float32, device=dev)

    # the 160 bf16 weight matrices (19.7 GB) as row ranges of one [rows, d] buffer per width
    rows = {K: 0 for K in acts}
    spans = []
    for b in range(wl.repeat):
        for li, lin in enumerate(wl.linears):
            spans.append((lin, rows[lin.K], rows[lin.K] + lin.N))
            rows[lin.K] += lin.N
    Wcat = {K: torch.empty((n, K), dtype=torch.bfloat16, device=dev) for K, n in rows.items()}
    ccat = {K: torch.empty((n, K // 2), dtype=torch.uint8, device=dev) for K, n in rows.items()}
    ncat = {K: torch.empty((n,), dtype=torch.bfloat16, device=dev) for K, n in rows.items()}
    for i, (lin, r0, r1) in enumerate(spans):
        b, li = divmod(i, len(wl.linears))
        Wcat[lin.K][r0:r1].copy_(workloads.c5_weight(b, li, device=dev))
    wcodes = [ccat[lin.K][r0:r1] for lin, r0, r1 in spans]
    wnorms = [ncat[lin.K][r0:r1] for lin, r0, r1 in spans]
    wp_bytes = float(sum(n * (2 * K + K // 2 + 2) for K, n in rows.items()))
    n_weights = sum(n * K for K, n in rows.items())

    def timed(fn):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1)

    def batched():
        for K in rows:
            oq.quantize_weights_offline(plans[K], cbs[K], Wcat[K], 1e-10, ccat[K], ncat[K])

    def per_matrix():
        for lin, r0, r1 in spans:
            oq.quantize_weights_offline(plans[lin.K], cbs[lin.K], Wcat[lin.K][r0:r1], 1e-10, ccat[lin.K][r0:r1],
                                        ncat[lin.K][r0:r1])

    # an untimed pass first: the first writes into freshly allocated output memory are several
    # times slower than later ones.  Then the pass as one launch per matrix (its results checked
    # against the untimed pass), and twice as one launch per width.
    batched()
    torch.cuda.synchronize()
    ref = {K: (ccat[K].clone(), ncat[K].clone()) for K in rows}
    per_matrix_ms = timed(per_matrix)
    same = all(torch.equal(ref[K][0], ccat[K]) and torch.equal(ref[K][1], ncat[K]) for K in rows)
    wp_runs = [timed(batched) for _ in range(2)]
    wp_ms = float(np.mean(wp_runs))
    del Wcat, ref

    def step(ev=None):
        for b in range(wl.repeat):
            for li, lin in enumerate(wl.linears):
                i = b * len(wl.linears) + li
                if ev is not None:
                    ev[4 * i].record()
                oq.rpbh_quantize_act(plans[lin.K], cbs[lin.K], acts[lin.K], 1e-10, xc[lin.K], xn[lin.K])
                if ev is not None:
                    ev[4 * i + 1].record()
                    ev[4 * i + 2].record()
                oq.orbit_qlinear(cbs[lin.K], xc[lin.K], xn[lin.K], cbs[lin.K], wcodes[i], wnorms[i],
                                 Yflat[:M * lin.N].view(M, lin.N))
                if ev is not None:
                    ev[4 * i + 3].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    n = wl.repeat * len(wl.linears)
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4 * n)] for _ in range(steps)]
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s0.record()
    for k in range(steps):
        step(events[k])
    s1.record()
    torch.cuda.synchronize()
    step_ms = s0.elapsed_time(s1) / steps
    q_ms = sum(ev[4 * i].elapsed_time(ev[4 * i + 1]) for ev in events for i in range(n)) / steps
    g_ms = sum(ev[4 * i + 2].elapsed_time(ev[4 * i + 3]) for ev in events for i in range(n)) / steps
    flops = wl.repeat * sum(2.0 * M * lin.N * lin.K for lin in wl.linears)
    qbytes = wl.repeat * sum(quant_bytes(M, lin.K, 4) for lin in wl.linears)
    return {"workload": wl.name, "blocks": wl.repeat, "linears_per_step": n, "M": M, "steps": steps,
            "step_ms": step_ms, "step_tflops": flops / (step_ms * 1e-3) / 1e12,
            "gemm_ms_sum": g_ms, "gemm_tflops": flops / (g_ms * 1e-3) / 1e12,
            "gemm_frac_of_bf16_peak": flops / (g_ms * 1e-3) / 1e12 / MFMA_PEAK_TFLOPS,
            "quant_ms_sum": q_ms, "quant_gbs": qbytes / (q_ms * 1e-3) / 1e9,
            "quant_frac_of_hbm": qbytes / (q_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "weight_pass_ms": wp_ms, "weight_pass_gbs": wp_bytes / (wp_ms * 1e-3) / 1e9,
            "weight_pass_frac_of_hbm": wp_bytes / (wp_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "weight_pass_launches": len(rows), "weight_pass_runs_ms": wp_runs,
            "weight_pass_rows": {str(K): n for K, n in rows.items()},
            "weight_pass_per_matrix": {"launches": len(spans), "ms": per_matrix_ms,
                                       "gbs": wp_bytes / (per_matrix_ms * 1e-3) / 1e9,
                                       "codes_and_norms_equal": bool(same)},
            "weights": n_weights, "weight_code_bytes": int(sum(c.numel() for c in wcodes))}


def adaln_sweep(oq, workloads, dev, steps, warmup=2):
    """The adjacent layer type: every AdaLN modulation projection of a FLUX-shaped image DiT at INT4
    weight round-to-nearest (group 64), one BF16 conditioning token.  Timed two ways per step:
    the 76 projections one call each, and as one call over their concatenated weight rows (all
    of them read the same conditioning vector).  Each way is captured in a graph (the launches
    are a few microseconds long) and every replay is checked against the eager result.  The
    offline pass over all 3.2e9 weights is timed launch by launch, generation outside."""
    K = workloads.ADALN_K
    sizes = [N for N, count in workloads.ADALN_LAYERS for _ in range(count)]
    Ntot = sum(sizes)
    q = torch.empty((Ntot, K // 2), dtype=torch.uint8, device=dev)
    sc = torch.empty((Ntot, K // 64), dtype=torch.float16, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wp_ms, row = 0.0, 0
    for i, N in enumerate(sizes):
        W = workloads.adaln_weights(N, i, device=dev)
        torch.cuda.synchronize()
        e0.record()
        oq.adaln_int4_quantize_weights(W, q[row:row + N], sc[row:row + N])
        e1.record()
        torch.cuda.synchronize()
        wp_ms += e0.elapsed_time(e1)
        row += N
        del W
    X = workloads.adaln_tokens(1, device=dev)
    Y_each = torch.empty((1, Ntot), device=dev)
    Y_all = torch.empty((1, Ntot), device=dev)
    offs = np.cumsum([0] + sizes)

    def each():
        for i in range(len(sizes)):
            a, b = int(offs[i]), int(offs[i + 1])
            oq.adaln_int4_linear(X, q[a:b], sc[a:b], out=Y_each[:, a:b])

    def batched():
        oq.adaln_int4_linear(X, q, sc, out=Y_all)

    out = {"layers": len(sizes), "K": K, "M": 1, "weights": Ntot * K,
           "weight_bytes": Ntot * (K // 2 + 2 * (K // 64)), "weight_pass_ms": wp_ms,
           "weight_pass_gbs": Ntot * (2 * K + K // 2 + 2 * (K // 64)) / (wp_ms * 1e-3) / 1e9}
    for name, fn, Y in (("per_layer", each, Y_each), ("batched", batched, Y_all)):
        fn()
        torch.cuda.synchronize()
        ref = Y.clone()
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            fn()
        ok = True
        for _ in range(warmup):
            Y.zero_()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            ok = ok and bool(torch.equal(Y, ref))
        _warm(g.replay)
        e0.record()
        for _ in range(steps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        ok = ok and bool(torch.equal(Y, ref))
        gbs = out["weight_bytes"] / (ms * 1e-3) / 1e9
        out[name] = {"ms": ms, "gbs": gbs, "frac_of_hbm": gbs / HBM_PEAK_GBS, "replays_match_eager": ok}
    out["batched_equals_per_layer"] = bool(torch.equal(Y_all, Y_each))
    del q, sc
    return out


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        return os.cpu_count()


def _oracle_pass(oracle, prepared, rows, min_seconds):
    """Oracle work on the host: every prepared linear's rows quantized and contracted in fp64, passes
    repeated until `rows` rows and at least `min_seconds` are done.  Returns (flops, seconds, passes,
    the last pass's activation codes per linear)."""
    t0 = time.perf_counter()
    flops, done, passes, last = 0.0, 0, 0, []
    while done < rows or time.perf_counter() - t0 < min_seconds:
        last = []
        for lin, plan, cba, cbw, cw, r, X in prepared:
            cx, s, U = oracle.quantize_act(X, plan, cba)
            oracle.qlinear(cx, s, cba.levels, cw, r, cbw.levels)
            flops += 2.0 * X.shape[0] * lin.N * lin.K
            last.append((cx, s, U))
        done += prepared[0][6].shape[0]
        passes += 1
    return flops, time.perf_counter() - t0, passes, last


def cpu_baseline(layers, rows, min_seconds=10.0, one_thread_rows=0, parity=False):
    """The fp64 oracle timed on the host cores on a bounded sample: `rows` token rows through
    every linear of the step (quantize + contraction), with the BLAS library's own thread count, and
    (one_thread_rows > 0) a smaller sample in a child process limited to one thread.  The oracle's
    weight codes are made once, outside the timing, as the GPU's offline weight pass is outside the
    step.  With parity=True the same oracle results are compared with the GPU's outputs of the step
    (activation and weight codes, norms, and 256 output rows against the oracle contraction of the
    GPU's own codes); the counts go to a 'parity' entry."""
    import oracle
    prepared = []
    for L in layers:
        lin = L["lin"]
        plan = oracle.rpbh_plan(lin.K, lin.h, 0)
        cba, cbw = oracle.lloydmax_codebook(lin.ba, lin.K), oracle.lloydmax_codebook(lin.bw, lin.K)
        W = L["W"].float().cpu().numpy().astype(np.float64)
        cw, r, Uw = oracle.quantize_weights(W, plan, cbw)
        del W
        X = L["X"][:rows].float().cpu().numpy().astype(np.float64)
        prepared.append((lin, plan, cba, cbw, cw, r, X))
        L["_oracle_w"] = (cw, r, Uw) if parity else None
    # a workload with fewer rows than the sample asks for (c1: 256) repeats its rows, and passes
    # continue until at least min_seconds of work, so that the rate is not a timer artefact
    flops, dt, passes, last = _oracle_pass(oracle, prepared, rows, min_seconds)
    n = prepared[0][6].shape[0]
    out = {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": _blas_threads(), "kind": "oracle",
           "host_cpu_count": os.cpu_count(),
           "sample": f"{n} token rows through every linear of the step (quantize + fp64 contraction), "
                     f"{passes} pass{'es' if passes > 1 else ''}, {dt:.1f} s, BLAS threads as the library "
                     f"chose; same metric unit as the GPU value",
           "seconds": dt}
    if one_thread_rows > 0:
        out["one_thread"] = cpu_baseline_one_thread(prepared, one_thread_rows, min_seconds)
    if parity:
        out["parity"] = parity_vs_oracle(oracle, layers, prepared, last)
    return out


def parity_vs_oracle(oracle, layers, prepared, last, gemm_rows=256, band=1e-5):
    """The GPU's outputs of the step against the oracle on the baseline's sample: codes equal off
    near-ties (|u - tau| > 1e-5); within a near-tie only the two codes across the nearest threshold are
    nearest centroids (Eq. (3) ties there), so other codes count as invalid.  Norms to 1e-5 (s) and
    one bf16 ulp (r').  The layer on gemm_rows rows against the fp64 contraction of the GPU's own codes,
    norms and bf16 levels: relative Frobenius error and the worst element over the per-element bar
    1e-4 s_n r'_i ||a_n|| ||b_i||."""
    res = []
    for L, (lin, plan, cba, cbw, cw, r, X), (cx, s, Ux) in zip(layers, prepared, last):
        n = X.shape[0]
        gx = oracle.from_labels(oracle.unpack_codes(L["xc"][:n].cpu().numpy(), lin.ba, lin.K), lin.ba)
        gw = oracle.from_labels(oracle.unpack_codes(L["wc"].cpu().numpy(), lin.bw, lin.K), lin.bw)
        _, _, Uw = L.pop("_oracle_w")
        entry = {"linear": lin.name, "act_rows": n, "weight_rows": lin.N}
        for tag, g, c, U, th in (("act", gx, cx, Ux, cba.thresholds), ("weights", gw, cw, Uw, cbw.thresholds)):
            near = oracle.near_tie_mask(U, th, band)
            j = oracle.nearest_threshold(U, th)
            mism = g != c
            entry[tag] = {"codes": int(g.size), "near_ties": int(near.sum()),
                          "near_tie_mismatches": int(np.sum(mism & near)),
                          "near_tie_invalid": int(np.sum(mism & near & (g != j) & (g != j + 1))),
                          "mismatches_off_tie": int(np.sum(mism & ~near))}
        gs = L["xn"][:n].cpu().numpy().astype(np.float64)
        gr = L["wn"].float().cpu().numpy().astype(np.float64)
        ulp = np.ldexp(1.0, np.frexp(np.maximum(r, 1e-30))[1] - 8)
        entry["s_max_rel_err"] = float(np.max(np.abs(gs - s) / np.maximum(s, 1e-30)))
        entry["r_max_err_bf16_ulps"] = float(np.max(np.abs(gr - r) / ulp))
        m = min(gemm_rows, n)
        la, lw = oracle.bf16_round(cba.levels), oracle.bf16_round(cbw.levels)
        ref = oracle.qlinear(gx[:m], gs[:m], la, gw, gr, lw)
        Y = L["Y"][:m].double().cpu().numpy()
        unit = (gs[:m] * np.linalg.norm(la[gx[:m]], axis=1))[:, None] * (gr * np.linalg.norm(lw[gw], axis=1))[None, :]
        entry["gemm_rows"] = m
        entry["gemm_rel_f"] = float(np.linalg.norm(Y - ref) / np.linalg.norm(ref))
        entry["gemm_worst_elem_over_bar"] = float(np.max(np.abs(Y - ref) / np.maximum(1e-4 * unit, 1e-300)))
        res.append(entry)
    ok = all(e[t]["mismatches_off_tie"] == 0 and e[t]["near_tie_invalid"] == 0 for e in res for t in ("act", "weights"))
    ok = ok and all(e["s_max_rel_err"] <= 1e-5 and e["r_max_err_bf16_ulps"] <= 1.0 and e["gemm_rel_f"] <= 2e-3
                    and e["gemm_worst_elem_over_bar"] <= 1.0 for e in res)
    return {"passed": bool(ok), "band": band, "linears": res}


def cpu_baseline_one_thread(prepared, rows, min_seconds):
    """The same oracle work in a child process with every BLAS/OpenMP pool at one thread, on the
    first `rows` rows of the sample (the pools are sized when numpy loads, so it takes a process of
    its own)."""
    import subprocess
    import tempfile
    tmp = tempfile.mkdtemp(prefix="orbit_cpu1_")
    path = os.path.join(tmp, "sample.npz")
    arrays = {}
    for i, (lin, plan, cba, cbw, cw, r, X) in enumerate(prepared):
        arrays[f"X{i}"] = X[:rows]
        arrays[f"cw{i}"] = cw.astype(np.uint8)
        arrays[f"r{i}"] = r
        arrays[f"shape{i}"] = np.array([lin.M, lin.K, lin.N, lin.bw, lin.ba, lin.h], dtype=np.int64)
    arrays["min_seconds"] = np.array([min_seconds])
    np.savez(path, **arrays)
    env = dict(os.environ)
    for v in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS", "BLIS_NUM_THREADS"):
        env[v] = "1"
    try:
        r = subprocess.run([sys.executable, os.path.abspath(__file__), "--cpu-baseline-worker", path],
                           capture_output=True, text=True, env=env, timeout=600)
        line = [l for l in r.stdout.splitlines() if l.startswith("{")]
        res = json.loads(line[-1]) if r.returncode == 0 and line else {"error": r.stderr[-500:]}
    finally:
        for f in os.listdir(tmp):
            os.remove(os.path.join(tmp, f))
        os.rmdir(tmp)
    return res


def cpu_baseline_worker(path):
    """Child process of cpu_baseline_one_thread: times the oracle on the saved sample, prints JSON."""
    import oracle
    z = np.load(path)
    prepared, i = [], 0
    while f"X{i}" in z:
        M, K, N, bw, ba, h = (int(v) for v in z[f"shape{i}"])
        from paper_2607_02461_amd.workloads import Linear
        lin = Linear(f"linear{i}", M, K, N, bw, ba, h)
        prepared.append((lin, oracle.rpbh_plan(K, h, 0), oracle.lloydmax_codebook(ba, K),
                         oracle.lloydmax_codebook(bw, K), z[f"cw{i}"].astype(np.int64), z[f"r{i}"], z[f"X{i}"]))
        i += 1
    rows = prepared[0][6].shape[0]
    flops, dt, passes, _ = _oracle_pass(oracle, prepared, rows, float(z["min_seconds"][0]))
    print(json.dumps({"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": _blas_threads(), "kind": "oracle",
                      "sample": f"{rows} token rows through every linear of the step (quantize + fp64 contraction), "
                                f"{passes} pass{'es' if passes > 1 else ''}, {dt:.1f} s, one thread",
                      "seconds": dt}), flush=True)


if __name__ == "__main__":
    main()
