"""Benchmark: the NVFP4 W4A4 + RAC MoE layer forward on one MI355X.

One step = the whole hot path (route, quantise X with RAC statistics,
channel selection and masked residual, W13 grouped GEMM with fused residual
and SwiGLU, quantise h, W2 grouped GEMM, combine) over one batch of the
workload, with inputs already resident in HBM.  Weight banks and inputs are
rotated over several copies so the weights never stay in the 256 MB MALL
between steps.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload NAME]
    python bench.py --copy-bytes N     # plain device copy, for counter calibration

The headline workload is the largest one that fits a GPU (4096 tokens,
H = 4096, I = 1536); `per_config` adds the other MoE workloads, timed in the
same run.  Step times are the median of per-step HIP-event intervals over
the K timed steps (the mean beside it).  `roofline` describes the dominant
kernel (the W13 grouped GEMM): its algorithmic bytes (decode) or FLOPs
(prefill) per launch over its average duration, timed with HIP events
recorded on the layer's stream at the stage boundaries, against the
published peak and against the achievable peak measured by the library's
probes in the same run.  `roofline.traffic` is the kernel's measured HBM
traffic per launch, taken from the counter summary under profiles/ when that
summary was made from the current GEMM source (its SHA-256 is recorded
there), else null.  `cpu_baseline` times the CPU oracle's whole forward on a
token sample of the headline workload.
"""

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE-layer tokens/s + effective TFLOP/s (% of MFMA peak) or GB/s (% HBM), 1 GPU"
PEAK_HBM_GBS = 8000.0
PEAK_F16_TFLOPS = 2500.0     # dense f16/bf16 MFMA (the operand type of exact NVFP4 here)
PEAK_FP8_TFLOPS = 5000.0
PEAK_FP4_TFLOPS = 10100.0
NVFP4_BYTES_PER_ELEM = 0.5625   # 4-bit code + one E4M3 byte per 16 elements

HEADLINE = "moe_prefill_t4096_h4096"
PER_CONFIG = ["moe_decode_t256_h2048", "moe_prefill_t8192_h2048", "moe_zipf_decode_t64_h4096",
              "moe_prefill_t4096_h4096"]
DECODE = {"moe_decode_t256_h2048", "moe_zipf_decode_t64_h4096", "dense_t16_k256_n128"}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--copies", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-comparisons", action="store_true",
                    help="skip the FP8 / MXFP4 layers and the K_s = 0 / 50%% rows")
    ap.add_argument("--no-per-config", action="store_true",
                    help="time the headline workload only")
    ap.add_argument("--ks-sweep", action="store_true",
                    help="add a K_s sweep (0, 12.5, 25, 50, 75, 100%% of the channels and the "
                         "configured K_s): step time and compensated-activation error")
    ap.add_argument("--cpu-tokens", type=int, default=8,
                    help="tokens of the headline batch in the oracle's timed sample")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only run a plain device-to-device copy of this many bytes "
                         "(5 times), the reference kernel for HBM counter calibration")
    return ap.parse_args()


GEMM_SRC = os.path.join(ROOT, "paper_2607_15810_amd", "csrc", "gemm.hip")
PROFILES = os.path.join(ROOT, "profiles")


def gemm_source_hash():
    with open(GEMM_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(workload):
    """HBM bytes per W13 launch from profiles/w13_traffic_<workload>.txt, or
    None when that summary is missing or was taken from another GEMM source."""
    path = os.path.join(PROFILES, f"w13_traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("gemm_source_sha256") != gemm_source_hash():
        return None
    try:
        return int(float(vals["hbm_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def copy_only(nbytes):
    import torch
    n = max(1, nbytes // 4)
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n * 4, "launches": 5}))


def algorithmic(wl, counts):
    """Algorithmic bytes and FLOPs of one step and of the W13 launch.

    Bytes: NVFP4 weights of the touched experts, X in and y out (bf16), the
    router logits (f32); intermediates (codes, residual, h, z) are the
    implementation's own traffic and are not counted.  FLOPs: 2*R*(H*2I +
    I*H) for the expert GEMMs plus 2*R*Ks*2I for the residual.
    """
    T, H, I, k, Ks = wl.T, wl.H, wl.I, wl.k, wl.Ks
    R = T * k
    touched = int(np.count_nonzero(counts))
    w13_bytes = touched * 2 * I * H * NVFP4_BYTES_PER_ELEM
    w2_bytes = touched * H * I * NVFP4_BYTES_PER_ELEM
    step_bytes = w13_bytes + w2_bytes + T * H * 2 * 2 + T * wl.E * 4
    w13_flops = 2.0 * R * 2 * I * H + 2.0 * R * Ks * 2 * I
    step_flops = w13_flops + 2.0 * R * I * H
    # the W13 launch reads its weights, the NVFP4 activations and residual,
    # and writes h (bf16)
    w13_launch_bytes = w13_bytes + 2 * T * H * NVFP4_BYTES_PER_ELEM + R * I * 2
    return dict(touched=touched, step_bytes=step_bytes, step_flops=step_flops,
                w13_bytes=w13_launch_bytes, w13_flops=w13_flops)


def _oracle_banks(inp, experts):
    """The oracle's own quantisation of the given experts' weights (the others
    stay zero and receive no rows); experts are independent, so they are
    quantised on a pool of threads."""
    import concurrent.futures as cf
    from oracle import quant as OQ
    wl = inp.wl
    banks = []
    for src, N, K in ((inp.w13, 2 * wl.I, wl.H), (inp.w2, wl.H, wl.I)):
        b = dict(codes=np.zeros((wl.E, N, K), np.uint8),
                 scales=np.zeros((wl.E, N, K // 16), np.uint8),
                 gscale=np.ones((wl.E, 2), np.float32))

        def one(e, b=b, src=src):
            q = OQ.quantize(src[e].float().numpy())
            b["codes"][e], b["scales"][e] = q["codes"], q["scales"]
            b["gscale"][e] = (q["s_enc"], q["s_dec"])

        with cf.ThreadPoolExecutor(min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(one, [int(e) for e in experts]))
        banks.append(b)
    return banks


def cpu_baseline(name, n_tok):
    """The oracle's free-running forward of the whole layer (routing, Q_A of X
    with RAC, W13 + SwiGLU, Q_A(h), W2, combine; float64 contractions), timed
    on the host cores on the first n_tok tokens of the workload's batch.  The
    oracle quantises the touched experts' weights itself first (not timed:
    weights are quantised once per weight sync, not per forward)."""
    from oracle import layer as OL, route as ORt
    from paper_2607_15810_amd import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    wl = synth.WORKLOADS[name]
    lg_all = synth.generate(name, with_weights=False)
    x = lg_all.x[:n_tok].float().numpy()
    lg = lg_all.logits[:n_tok].numpy()
    touched = np.unique(ORt.topk_fast(lg, wl.k))
    inp = synth.generate(name, experts=touched)
    t_q = time.perf_counter()
    W13, W2 = _oracle_banks(inp, touched)
    t_q = time.perf_counter() - t_q
    reps, t_sum = 0, 0.0
    while reps == 0 or (t_sum < 10.0 and reps < 100):
        t0 = time.perf_counter()
        OL.moe_layer(x, lg, W13, W2, wl.k, wl.Ks)
        t_sum += time.perf_counter() - t0
        reps += 1
    per = t_sum / reps
    return dict(value=round(n_tok / per, 2), unit="tokens/s", cores=int(threads), kind="oracle",
                sample=(f"{reps} free-running forwards of the whole layer (float64 numpy oracle) "
                        f"on the first {n_tok} tokens of the {name} batch ({n_tok * wl.k} expert "
                        f"rows over {touched.size} experts), {per:.3f} s each; the oracle's own "
                        f"weight quantisation of those experts ({t_q:.1f} s) is not timed"),
                seconds_measured=round(t_sum, 3))


def measure_ceilings():
    """Achievable peaks on this GPU: a 4 GiB streaming read and a register-only
    f16 MFMA loop (the library's probes), each the best of 3 launches."""
    import torch
    from paper_2607_15810_amd import quads as Q
    L = Q.lib()
    s = torch.cuda.current_stream().cuda_stream
    nbytes = 4 << 30
    buf = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    out = torch.empty(L.qd_probe_hbm_read_out_count(), dtype=torch.int32, device="cuda")
    best = None
    for _ in range(4):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        Q.call("qd_probe_hbm_read", buf.data_ptr(), nbytes, out.data_ptr(), s)
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b)
        best = ms if best is None else min(best, ms)
    hbm = nbytes / (best * 1e-3) / 1e9
    del buf
    wg, rounds = 2048, 2000
    outm = torch.empty(wg, dtype=torch.float32, device="cuda")
    mfma = {}
    for rnd in (0, 1):
        best = None
        for _ in range(4):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            Q.call("qd_probe_mfma_f16", rounds, wg, rnd, outm.data_ptr(), s)
            b.record()
            torch.cuda.synchronize()
            ms = a.elapsed_time(b)
            best = ms if best is None else min(best, ms)
        mfma[rnd] = L.qd_probe_mfma_f16_flops(rounds, wg) / (best * 1e-3) / 1e12
    torch.cuda.empty_cache()
    return {"hbm_read_GBps": round(hbm, 1), "mfma_f16_TFLOPs": round(mfma[1], 1),
            "mfma_f16_low_toggle_TFLOPs": round(mfma[0], 1),
            "how": "streaming 16-byte reads of 4 GiB; 16 independent v_mfma_f32_32x32x16_f16 "
                   "chains per wave, 8 waves per CU, best of 4 launches: mfma_f16_TFLOPs on "
                   "random operand bits (the power-limited rate real data sees), "
                   "mfma_f16_low_toggle_TFLOPs on slowly varying operands"}


def clone_bank(b):
    from paper_2607_15810_amd import ops
    return ops.NVFP4Tensor(b.codes.clone(), b.scales.clone(), b.gscale.clone(), b.groups,
                           b.rows, b.cols,
                           b.scales_frag.clone() if b.scales_frag is not None else None)


def measure(args, name, ceil, headline):
    """Time one workload: the step (median and mean over args.steps), the
    stages, and the W13 roofline.  With headline=True also the HIP-graph
    replay, the comparison rows and the K_s sweep."""
    import torch
    from paper_2607_15810_amd import ops, synth
    from paper_2607_15810_amd import quads as Q
    wl = synth.WORKLOADS[name]
    t_gen = time.perf_counter()
    inp = synth.generate(name)
    t_gen = time.perf_counter() - t_gen
    print(f"[bench] generated {name} in {t_gen:.1f} s", file=sys.stderr, flush=True)
    dev = "cuda"
    x0 = inp.x.to(dev)
    lg0 = inp.logits.to(dev)
    w13_0 = ops.quantize_weight(inp.w13.to(dev))
    w2_0 = ops.quantize_weight(inp.w2.to(dev))
    torch.cuda.synchronize()
    copies = max(1, args.copies)
    banks = [(w13_0, w2_0)] + [(clone_bank(w13_0), clone_bank(w2_0)) for _ in range(copies - 1)]
    xs = [x0] + [x0.clone() for _ in range(copies - 1)]
    lgs = [lg0] + [lg0.clone() for _ in range(copies - 1)]
    n_ws = Q.lib().qd_moe_layer_workspace(wl.T, wl.H, wl.E, wl.k, wl.I)
    ws = torch.empty(n_ws, dtype=torch.uint8, device=dev)
    layers = [ops.MoELayer(b13, b2, wl.T, wl.k, wl.Ks, ws=ws) for b13, b2 in banks]
    y = torch.empty((wl.T, wl.H), dtype=torch.bfloat16, device=dev)

    for i in range(args.warmup):
        c = i % copies
        layers[c](xs[c], lgs[c], y)
    torch.cuda.synchronize()
    counts = np.diff(layers[0].views()["offsets"].cpu().numpy())

    # timed region 1: the layer alone, an event between consecutive steps
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record()
    for i in range(args.steps):
        c = i % copies
        layers[c](xs[c], lgs[c], y)
        evs[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    ms_mean = evs[0].elapsed_time(evs[-1]) / args.steps
    ms_step = float(np.median(per_step))

    # timed region 2: the same steps with HIP events recorded by the library
    # at the stage boundaries on the layer's stream -> per-stage times and
    # the W13 kernel's duration for the roofline
    n_ev = len(Q.STAGE_NAMES) + 1
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(n_ev)] for _ in range(args.steps)]
    for ee in events:          # create the underlying HIP events
        for e in ee:
            e.record()
    torch.cuda.synchronize()
    start2 = torch.cuda.Event(enable_timing=True)
    end2 = torch.cuda.Event(enable_timing=True)
    start2.record()
    for i in range(args.steps):
        c = i % copies
        layers[c](xs[c], lgs[c], y, events=events[i])
    end2.record()
    torch.cuda.synchronize()
    ms_step_ev = start2.elapsed_time(end2) / args.steps
    stage_ms = np.zeros(n_ev - 1)
    for ee in events:
        for s in range(n_ev - 1):
            stage_ms[s] += ee[s].elapsed_time(ee[s + 1])
    stage_ms /= args.steps

    alg = algorithmic(wl, counts)
    tok_s = wl.T / (ms_step * 1e-3)
    step_gbs = alg["step_bytes"] / (ms_step * 1e-3) / 1e9
    step_tflops = alg["step_flops"] / (ms_step * 1e-3) / 1e12
    w13_ms = stage_ms[Q.STAGE_NAMES.index("w13")]
    decode = name in DECODE
    # the W13 launch runs the decode kernel when the rows per expert are few
    skinny = Q.lib().moe_w4a4_grouped_gemm_amax_count(
        wl.T * wl.k, 2 * wl.I, wl.H, wl.E, wl.Ks, Q.QD_EPI_SWIGLU) <= 1024
    kname = ("gemm_skinny_kernel" if skinny else "gemm_tile_kernel") + \
        " (W13 + fused RAC residual + SwiGLU)"
    traffic = measured_traffic(name)
    if decode:
        achieved = alg["w13_bytes"] / (w13_ms * 1e-3) / 1e9
        roof = dict(bound="hbm", achieved=round(achieved, 1), peak=PEAK_HBM_GBS, unit="GB/s",
                    frac=round(achieved / PEAK_HBM_GBS, 4), traffic=traffic,
                    kernel=kname, algorithmic_bytes=int(alg["w13_bytes"]),
                    avg_ms=round(w13_ms, 5))
        if ceil:
            roof["measured_peak"] = ceil["hbm_read_GBps"]
            roof["frac_of_measured"] = round(achieved / ceil["hbm_read_GBps"], 4)
    else:
        achieved = alg["w13_flops"] / (w13_ms * 1e-3) / 1e12
        roof = dict(bound="mfma", achieved=round(achieved, 1), peak=PEAK_F16_TFLOPS,
                    unit="TFLOP/s", frac=round(achieved / PEAK_F16_TFLOPS, 4), traffic=traffic,
                    kernel=kname, algorithmic_flops=alg["w13_flops"], avg_ms=round(w13_ms, 5),
                    frac_of_fp8_peak=round(achieved / PEAK_FP8_TFLOPS, 4),
                    frac_of_fp4_peak=round(achieved / PEAK_FP4_TFLOPS, 4))
        if ceil:
            roof["measured_peak"] = ceil["mfma_f16_TFLOPs"]
            roof["frac_of_measured"] = round(achieved / ceil["mfma_f16_TFLOPs"], 4)
    res = {
        "workload": name, "tokens": wl.T, "hidden": wl.H, "experts": wl.E, "top_k": wl.k,
        "intermediate": wl.I, "rac_channels": wl.Ks, "touched_experts": alg["touched"],
        "weight_copies": copies,
        "ms_per_step": round(ms_step, 5), "ms_per_step_mean": round(ms_mean, 5),
        "ms_per_step_min": round(float(per_step.min()), 5),
        "tokens_per_s": round(tok_s, 1),
        "effective": {"GB/s": round(step_gbs, 1), "frac_hbm": round(step_gbs / PEAK_HBM_GBS, 4),
                      "TFLOP/s": round(step_tflops, 2),
                      "frac_f16_mfma": round(step_tflops / PEAK_F16_TFLOPS, 4),
                      "frac_fp8_mfma": round(step_tflops / PEAK_FP8_TFLOPS, 4),
                      "frac_fp4_mfma": round(step_tflops / PEAK_FP4_TFLOPS, 4)},
        "stage_ms": {n: round(float(v), 5) for n, v in zip(Q.STAGE_NAMES, stage_ms)},
        "ms_per_step_with_stage_events": round(ms_step_ev, 5),
        "wall_ms_per_step": round(wall * 1e3 / args.steps, 5),
        "roofline": roof,
    }
    print(f"[bench] {name}: {ms_step:.4f} ms/step (median), {ms_mean:.4f} mean",
          file=sys.stderr, flush=True)
    if headline:
        # the same steps replayed from HIP graphs (one captured layer call per
        # weight copy): what a serving loop that captures its step sees
        graphs = []
        for c in range(copies):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                layers[c](xs[c], lgs[c], y)
            graphs.append(g)
        ms_graph = time_steps([g.replay for g in graphs], args.steps, args.warmup)
        res["hip_graph"] = dict(ms_per_step=round(ms_graph, 5),
                                value=round(wl.T / (ms_graph * 1e-3), 1), unit="tokens/s")
        del graphs
        if not args.no_comparisons:
            res["comparisons"] = comparisons(args, wl, inp, banks, xs, lgs, ms_step, ws)
        if args.ks_sweep:
            res["ks_sweep"] = ks_sweep(args, wl, banks, xs, lgs, ws)
    del layers, banks, xs, lgs, ws, y, inp
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU; --gpus {args.gpus} is not supported: the layer is "
              "built and measured on a single MI355X (no collectives, no sharding)",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_bytes:
        copy_only(args.copy_bytes)
        return
    import torch
    from paper_2607_15810_amd import synth
    from paper_2607_15810_amd import quads as Q

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    Q.lib()
    wl = synth.WORKLOADS[args.workload]
    if wl.dense:
        print("the dense GEMM workload is a parity case, not a bench line", file=sys.stderr)
        sys.exit(2)
    ceil = measure_ceilings()
    print(f"[bench] ceilings {ceil}", file=sys.stderr, flush=True)
    head = measure(args, args.workload, ceil, headline=True)
    out = {
        "metric": METRIC,
        "value": head["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "ms_per_step_mean": head["ms_per_step_mean"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "nvfp4 (e2m1 x e4m3 decoded exactly to f16 MFMA operands, f32 accumulate)",
        "data": "synthetic",
        "config": {k: head[k] for k in ("workload", "tokens", "hidden", "experts", "top_k",
                                        "intermediate", "rac_channels", "touched_experts",
                                        "weight_copies")},
        "roofline": head["roofline"],
        "measured_ceilings": ceil,
    }
    for k in ("effective", "stage_ms", "ms_per_step_with_stage_events", "wall_ms_per_step",
              "ms_per_step_min", "hip_graph", "comparisons", "ks_sweep"):
        if k in head:
            out[k] = head[k]
    if not args.no_per_config:
        pc = {}
        for name in PER_CONFIG:
            if name == args.workload:
                continue
            r = measure(args, name, ceil, headline=False)
            pc[name] = {k: r[k] for k in ("ms_per_step", "ms_per_step_mean", "tokens_per_s",
                                          "touched_experts", "stage_ms", "roofline",
                                          "effective")}
        out["per_config"] = pc
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.workload, args.cpu_tokens)
    print(json.dumps(out))


def time_steps(fns, steps, warmup):
    """Average ms per call of fns[i % len(fns)]() over `steps` calls after
    `warmup`, bracketed by synchronisations (HIP events on torch's stream)."""
    import torch
    for i in range(warmup):
        fns[i % len(fns)]()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(steps):
        fns[i % len(fns)]()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def comparisons(args, wl, inp, banks, xs, lgs, ms_step, ws):
    """The measurement rows beside the headline: the FP8 W8A8 layer (same
    routing and shapes, per-token / per-channel E4M3, no residual), the
    MXFP4 W4A4 layer (the hardware's native FP4 format, no residual), the
    plain NVFP4 W4A4 layer (K_s = 0), RAC at K_s = 50% of the channels, RAC
    at both the W13 and the W2 inputs, per-expert channel sets, the block
    entry point with RMSNorm and router folded in, and the trainer-side
    W4A16 forward."""
    import torch
    from paper_2607_15810_amd import ops
    dev = "cuda"
    res = {}
    steps, warm = max(args.steps, 10), max(args.warmup, 3)
    y = torch.empty((wl.T, wl.H), dtype=torch.bfloat16, device=dev)
    # FP8 W8A8 layer, as many weight copies as the headline rotates
    w13c, w13d = ops.fp8_quantize_rows(inp.w13.to(dev))
    w2c, w2d = ops.fp8_quantize_rows(inp.w2.to(dev))
    f8 = [(w13c, w13d, w2c, w2d)] + [tuple(t.clone() for t in (w13c, w13d, w2c, w2d))
                                     for _ in range(len(banks) - 1)]
    lay8 = [ops.FP8MoELayer(*b, wl.T, wl.k) for b in f8]
    ms8 = time_steps([lambda c=c: lay8[c](xs[c], lgs[c], y) for c in range(len(f8))], steps, warm)
    res["fp8_w8a8"] = dict(ms_per_step=round(ms8, 5), value=round(wl.T / (ms8 * 1e-3), 1),
                           unit="tokens/s", nvfp4_rac_speedup=round(ms8 / ms_step, 3),
                           weight_bytes_per_param=1.0)
    del lay8, f8, w13c, w13d, w2c, w2d
    # MXFP4 W4A4 layer (E8M0 per 32 elements, the FP4 MFMA's own block
    # scales; no tensor scale, no residual): what exact NVFP4 costs here
    m13c, m13s = ops.mxfp4_quantize_rows(inp.w13.to(dev))
    m2c, m2s = ops.mxfp4_quantize_rows(inp.w2.to(dev))
    mx = [(m13c, m13s, m2c, m2s)] + [tuple(t.clone() for t in (m13c, m13s, m2c, m2s))
                                     for _ in range(len(banks) - 1)]
    laym = [ops.MXFP4MoELayer(*b, wl.T, wl.k) for b in mx]
    msm = time_steps([lambda c=c: laym[c](xs[c], lgs[c], y) for c in range(len(mx))], steps, warm)
    res["mxfp4_w4a4"] = dict(ms_per_step=round(msm, 5), value=round(wl.T / (msm * 1e-3), 1),
                             unit="tokens/s", nvfp4_rac_speedup=round(msm / ms_step, 3),
                             weight_bytes_per_param=0.53125)
    del laym, mx, m13c, m13s, m2c, m2s
    # the NVFP4 layer without RAC, with K_s = H / 2 (the paper's k = 50%),
    # and with RAC at the W2 input too (the same fraction of I channels)
    ks2 = max(1, round(wl.Ks * wl.I / wl.H)) if wl.Ks else 0
    for name, ks, k2 in (("w4a4_ks0", 0, 0), ("rac_ks_half", wl.H // 2, 0),
                         ("rac_w13_and_w2", wl.Ks, ks2)):
        lays = [ops.MoELayer(b13, b2, wl.T, wl.k, ks, ws=ws, Ks2=k2) for b13, b2 in banks]
        ms = time_steps([lambda c=c: lays[c](xs[c], lgs[c], y) for c in range(len(lays))],
                        steps, warm)
        res[name] = dict(ms_per_step=round(ms, 5), value=round(wl.T / (ms * 1e-3), 1),
                         unit="tokens/s", rac_channels=ks,
                         time_vs_headline=round(ms / ms_step, 3))
        if k2:
            res[name]["rac_channels_w2"] = k2
    # one RAC channel set per expert (each expert's own rows rank the
    # channels; reading L7), at the configured K_s
    lpe = [ops.MoELayerPerExpert(b13, b2, wl.T, wl.k, wl.Ks) for b13, b2 in banks]
    mspe = time_steps([lambda c=c: lpe[c](xs[c], lgs[c], y) for c in range(len(lpe))], steps, warm)
    res["rac_per_expert_sets"] = dict(ms_per_step=round(mspe, 5),
                                      value=round(wl.T / (mspe * 1e-3), 1), unit="tokens/s",
                                      rac_channels=wl.Ks,
                                      time_vs_headline=round(mspe / ms_step, 3))
    # the block input path: RMSNorm and the router folded into the layer's
    # first launch (qd_moe_block_forward, the workload's activations as the
    # hidden state) against the same steps as separate launches (torch's
    # RMSNorm arithmetic and bf16 router product, then the layer)
    from paper_2607_15810_amd import synth
    gamma, w_r = synth.block_params(wl.H, wl.E, seed=wl.index)
    gamma, w_r = gamma.to(dev), w_r.to(dev)
    w_rt = w_r.t().contiguous()
    gf = gamma.float()
    blks = [ops.MoEBlock(b13, b2, wl.T, wl.k, wl.Ks, gamma, w_r) for b13, b2 in banks]
    msb = time_steps([lambda c=c: blks[c](xs[c], y) for c in range(len(blks))], steps, warm)
    lays = [ops.MoELayer(b13, b2, wl.T, wl.k, wl.Ks, ws=ws) for b13, b2 in banks]

    def unfused(c):
        hf = xs[c].float()
        xn = (hf * torch.rsqrt(hf.pow(2).mean(-1, keepdim=True) + 1e-6) * gf).to(torch.bfloat16)
        lg = torch.mm(xn, w_rt).float()
        lays[c](xn, lg, y)

    msu = time_steps([lambda c=c: unfused(c) for c in range(len(lays))], steps, warm)
    res["block_norm_router_fused"] = dict(ms_per_step=round(msb, 5),
                                          value=round(wl.T / (msb * 1e-3), 1), unit="tokens/s",
                                          unfused_ms_per_step=round(msu, 5),
                                          speedup_vs_unfused=round(msu / msb, 3),
                                          time_vs_headline=round(msb / ms_step, 3))
    del blks, lays
    # the trainer-side forward on the same weights (Sec. 3.2: bf16
    # activations, fake-quantised NVFP4 weights, no activation quantiser)
    lay16 = [ops.W4A16MoELayer(b13, b2, wl.k) for b13, b2 in banks]
    ms16 = time_steps([lambda c=c: lay16[c](xs[c], lgs[c]) for c in range(len(lay16))], steps, warm)
    flop = 2.0 * wl.T * wl.k * (2 * wl.I * wl.H + wl.H * wl.I)
    res["w4a16_trainer_forward"] = dict(ms_per_step=round(ms16, 5),
                                        value=round(wl.T / (ms16 * 1e-3), 1), unit="tokens/s",
                                        gemm_tflops=round(flop / (ms16 * 1e-3) / 1e12, 1),
                                        time_vs_headline=round(ms16 / ms_step, 3))
    # train/inference alignment (the analogue of the paper's layer-output
    # comparison, Sec. 4): relative L2 distance of each rollout layer's output
    # from the trainer-side W4A16 forward on the same weights and tokens
    b13, b2 = banks[0]
    y_train = lay16[0](xs[0], lgs[0]).float()
    ref = torch.linalg.vector_norm(y_train).item()

    def gap(y):
        return round(torch.linalg.vector_norm(y.float() - y_train).item() / max(ref, 1e-30), 6)

    mism = {}
    for name, ks, k2 in (("w4a4_ks0", 0, 0), ("nvfp4_rac", wl.Ks, 0), ("rac_ks_half", wl.H // 2, 0),
                         ("rac_w13_and_w2", wl.Ks, ks2)):
        lay = ops.MoELayer(b13, b2, wl.T, wl.k, ks, ws=ws, Ks2=k2)
        mism[name] = gap(lay(xs[0], lgs[0]))
    mism["rac_per_expert_sets"] = gap(lpe[0](xs[0], lgs[0]))
    del lpe
    res["train_infer_rel_l2"] = mism
    del lay16
    torch.cuda.synchronize()
    return res


def ks_sweep(args, wl, banks, xs, lgs, ws):
    """Throughput against the number of compensated channels (the paper's
    K_s sweep, Sec. 3.3 / its ablation on k): per K_s the layer's step time
    and the relative error of the compensated activation,
    ||x - (x_hat - r_hat_S)|| / ||x|| (x_hat, r_hat_S the dequantised NVFP4
    activation and masked residual, all from the library's own calls)."""
    import torch
    from paper_2607_15810_amd import ops
    dev = "cuda"
    steps, warm = max(args.steps, 10), max(args.warmup, 3)
    y = torch.empty((wl.T, wl.H), dtype=torch.bfloat16, device=dev)
    x = xs[0]
    xf = x.float()
    nx = torch.linalg.vector_norm(xf).item()
    xq, scores, ramax = ops.quantize_act(x, rac=True)
    xhat = ops.dequantize(xq)[0]
    points = sorted({0, wl.Ks} | {max(1, round(f * wl.H)) for f in (0.125, 0.25, 0.5, 0.75, 1.0)})
    rows = []
    for ks in points:
        lays = [ops.MoELayer(b13, b2, wl.T, wl.k, ks, ws=ws) for b13, b2 in banks]
        ms = time_steps([lambda c=c: lays[c](xs[c], lgs[c], y) for c in range(len(lays))],
                        steps, warm)
        comp = xhat
        if ks:
            _, rq, _, _ = ops.select_channels(x, xq, ks, scores, ramax)
            comp = xhat - ops.dequantize(rq)[0]
        err = torch.linalg.vector_norm(xf - comp).item() / max(nx, 1e-30)
        rows.append(dict(rac_channels=ks, frac=round(ks / wl.H, 4), ms_per_step=round(ms, 5),
                         value=round(wl.T / (ms * 1e-3), 1), act_rel_err=round(err, 6)))
        del lays
    torch.cuda.synchronize()
    return rows


if __name__ == "__main__":
    main()
