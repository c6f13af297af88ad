"""Benchmark of the RFQ forward path on one MI355X.

One step = the whole hot path over one batch of the Qwen3-VL-like up-projection
(X 4096x4096 bf16 with 0.5% outlier channels x50, W 4096x12288 fp32 master):
  1. rfq_quantize_weight  W[N][K] fp32 -> MXFP4 codes + scales
  2. rfq_quantize_act     X[M][K] bf16 -> primary + residual MXFP4
  3. rfq_gemm             Z = (deq q + deq r) deq(w)^T, bf16 out
Inputs are resident in HBM before the timed region; three input sets are
rotated so that no step finds its inputs in the 256 MB last-level cache.

value = executed FP4 flops of the step (4*M*N*K: the primary and the residual
contraction) / step time.  The product's duration comes from HIP events
recorded on its launch stream around it in every timed step; the roofline
object reports it (the dominant kernel) against the dense MXFP4 matrix-core
peak.  The two quantizers are timed over back-to-back launches after the
timed region.  The oracle (plain C) is timed on a bounded sample of
the same step on the host cores.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
"""
import argparse
import json
import os
import sys
import time

import numpy as np

REPO = os.path.dirname(os.path.abspath(__file__))
if REPO not in sys.path:
    sys.path.insert(0, REPO)

PEAK_FP4_TFLOPS = 10100.0     # MI355X dense MXFP4 matrix cores
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 matrix cores
N_SETS = 3
EV_EVERY = 4                  # product events on every 4th timed step (all input sets alike)
Q_SETS = 9                    # 9 x 64 MiB quantizer inputs: over twice the 256 MB last-level cache
PHI_MARGINS = (2, 4, 6)       # scale-threshold phi: median primary scale byte + margin
MFMA_LOOP_ITERS = 512         # register-only MFMA loop: iterations per launch (2.1 GFLOP each)
METRIC = "RFQ-MXFP4 GEMM TFLOP/s + quantizer GB/s (Qwen3-VL-like 4096×4096×12288)"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    # Untimed steps before the timed region: about 0.1 s of GPU work, after
    # which the GPU's clock has settled (measured on MI355X: the first tens
    # of milliseconds of sustained matrix-core load run 10-20% slower).
    p.add_argument("--warmup", type=int, default=400)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extras", action="store_true",
                   help="skip the secondary workloads and the accuracy diagnostics")
    p.add_argument("--cpu-rows", type=int, default=8,
                   help="activation rows in the oracle's sample of the step")
    args = p.parse_args()
    if args.steps < 1 or args.warmup < 0:
        p.error("--steps must be at least 1 and --warmup at least 0")
    return args


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the RFQ path is data parallel over "
              "tokens and this benchmark runs and reports a single MI355X "
              "(got --gpus %d)." % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_26581_amd as rfq
    from paper_2608_26581_amd import workloads as wl

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wk = wl.WORKLOADS["qwen"]
    M, K = wk.M, wk.K
    N = wk.weights[0][2]

    # ---- inputs: N_SETS independent draws, resident on the device
    xs, ws, outs = [], [], []
    for s in range(N_SETS):
        d = wl.generate(wk, seed=s)
        xs.append(torch.from_numpy(d["x_bf16"].view(np.int16)).to(dev).view(torch.bfloat16))
        ws.append(torch.from_numpy(d["w"]).to(dev))
        del d
    for s in range(N_SETS):
        outs.append({
            "wc": torch.empty((N, K // 2), dtype=torch.uint8, device=dev),
            "ws": torch.empty((N, K // 32), dtype=torch.uint8, device=dev),
            "q": [torch.empty((M, K // 2), dtype=torch.uint8, device=dev),
                  torch.empty((M, K // 32), dtype=torch.uint8, device=dev),
                  torch.empty((M, K // 2), dtype=torch.uint8, device=dev),
                  torch.empty((M, K // 32), dtype=torch.uint8, device=dev)],
            "z": torch.empty((M, N), dtype=torch.bfloat16, device=dev),
        })
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    def step(i, ev=None):
        """One pass of the path; with ev, HIP events bracket the product (the
        roofline kernel) on its launch stream."""
        s = i % N_SETS
        o = outs[s]
        rfq.rfq_quantize_weight(ws[s], out=(o["wc"], o["ws"]), stream=stream)
        rfq.rfq_quantize_act(xs[s], out=o["q"], stream=stream)
        if ev is not None:
            ev[0].record(stream)
        rfq.rfq_gemm(*o["q"], o["wc"], o["ws"], out=o["z"], stream=stream)
        if ev is not None:
            ev[1].record(stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # Timed region: the K steps.  A pair of events around the product of every
    # step adds about 5 us to each step (measured on one MI355X: 239.4 against
    # 234.4 us without events); around every EV_EVERY-th product it adds
    # nothing measurable and gives the same average product time (185.0
    # against 185.1 us), so the product is timed on that uniform sample of
    # the timed launches.
    sampled = [i for i in range(args.steps) if i % EV_EVERY == 0]
    evs = {i: [torch.cuda.Event(enable_timing=True) for _ in range(2)] for i in sampled}
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for i in range(args.steps):
        step(i, evs.get(i))
    t1.record(stream)
    torch.cuda.synchronize()
    total_ms = t0.elapsed_time(t1)
    ms_step = total_ms / args.steps
    gm_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs.values()]))

    # The two quantizers of the step, each timed over back-to-back launches
    # on the same rotated inputs (outside the timed region).
    wq_ms = _per_launch_ms(torch, stream, lambda i: rfq.rfq_quantize_weight(
        ws[i % N_SETS], out=(outs[i % N_SETS]["wc"], outs[i % N_SETS]["ws"]), stream=stream), 30)
    xq_ms = _per_launch_ms(torch, stream, lambda i: rfq.rfq_quantize_act(
        xs[i % N_SETS], out=outs[i % N_SETS]["q"], stream=stream), 30)

    exec_flops = 4.0 * M * N * K
    # Operand and result bytes of one product: q, r and w codes and scales, bf16 Z.
    gemm_bytes = 2 * (M * K // 2 + M * K // 32) + (N * K // 2 + N * K // 32) + 2 * M * N
    value = exec_flops / (ms_step * 1e-3) / 1e12
    gemm_tflops = exec_flops / (gm_ms * 1e-3) / 1e12
    xq_bytes = M * K * 2 + 2 * (M * K // 2 + M * K // 32)
    wq_bytes = N * K * 4 + N * K // 2 + N * K // 32
    xq_gbs = xq_bytes / (xq_ms * 1e-3) / 1e9
    wq_gbs = wq_bytes / (wq_ms * 1e-3) / 1e9

    # ---- quantizer alone on the 8192x4096 bf16 workload (pure bandwidth)
    qk = wl.WORKLOADS["quant"]
    # Q_SETS 64 MiB inputs (rows of one draw rotated on the device) so that no
    # launch finds its input in the 256 MB last-level cache.
    d = wl.generate(qk, seed=100)
    x0 = torch.from_numpy(d["x_bf16"].view(np.int16)).to(dev).view(torch.bfloat16)
    del d
    qx = [torch.roll(x0, shifts=997 * s, dims=0).contiguous() for s in range(Q_SETS)]
    del x0
    qo = [torch.empty((qk.M, qk.K // 2), dtype=torch.uint8, device=dev),
          torch.empty((qk.M, qk.K // 32), dtype=torch.uint8, device=dev),
          torch.empty((qk.M, qk.K // 2), dtype=torch.uint8, device=dev),
          torch.empty((qk.M, qk.K // 32), dtype=torch.uint8, device=dev)]
    for i in range(20):
        rfq.rfq_quantize_act(qx[i % Q_SETS], out=qo, stream=stream)
    # Back-to-back launches between one pair of events: an event recorded
    # between two short kernels adds a few microseconds of its own.
    qreps = 200
    qa = torch.cuda.Event(enable_timing=True)
    qb = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    qa.record(stream)
    for i in range(qreps):
        rfq.rfq_quantize_act(qx[i % Q_SETS], out=qo, stream=stream)
    qb.record(stream)
    torch.cuda.synchronize()
    q_ms = qa.elapsed_time(qb) / qreps
    q_bytes = qk.M * qk.K * 2 + 2 * (qk.M * qk.K // 2 + qk.M * qk.K // 32)
    quant_gbs = q_bytes / (q_ms * 1e-3) / 1e9

    # ---- plain copy of 1 GiB as the achievable-bandwidth calibration
    src = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    c0 = torch.cuda.Event(enable_timing=True)
    c1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    c0.record(stream)
    for _ in range(10):
        dst.copy_(src)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_gbs = 2 * src.numel() * 4 * 10 / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del src, dst

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp4-e2m1 (fp32 accumulate)",
        "data": "synthetic",
        "config": {
            "workload": "Qwen3-VL-like MLP up-projection: X 4096x4096 bf16 N(0,1) with 0.5% "
                        "outlier channels x50, W 4096x12288 N(0,0.02) fp32 master; step = "
                        "weight quantize + RFQ activation quantize + RFQ GEMM (phi=1), bf16 Z",
            "M": M, "K": K, "N": N, "phi": 1, "z_dtype": "bf16", "input_sets": N_SETS,
        },
        "components": {
            "rfq_gemm": {"ms": round(gm_ms, 5), "exec_tflops": round(gemm_tflops, 1),
                         "effective_tflops": round(gemm_tflops / 2, 1)},
            "quantize_act": {"ms": round(xq_ms, 5), "gbs": round(xq_gbs, 1),
                             "bytes": xq_bytes},
            "quantize_weight": {"ms": round(wq_ms, 5), "gbs": round(wq_gbs, 1),
                                "bytes": wq_bytes},
            "quantizer_8192x4096_bf16": {"ms": round(q_ms, 5), "gbs": round(quant_gbs, 1),
                                         "frac_hbm": round(quant_gbs / PEAK_HBM_GBS, 4),
                                         "bytes": q_bytes},
            "copy_1GiB_gbs": round(copy_gbs, 1),
        },
        "roofline": {
            "kernel": "rfq_gemm_large_kernel",
            "bound": "mfma",
            "achieved": round(gemm_tflops, 1),
            "peak": PEAK_FP4_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(gemm_tflops / PEAK_FP4_TFLOPS, 4),
            "traffic": None,
            "algorithmic_bytes": gemm_bytes,
        },
    }
    rec = recorded_traffic()
    if rec is not None:
        result["roofline"]["traffic"] = rec["read_bytes"] + rec["write_bytes"]
        result["roofline"]["traffic_read_write"] = [rec["read_bytes"], rec["write_bytes"]]
    if not args.no_extras:
        result["components"].update(secondary(torch, rfq, wl, xs[0], ws[0], stream))
        result["accuracy"] = accuracy(torch, rfq, xs[0], ws[0])
    del xs, ws, outs, qx, qo
    torch.cuda.empty_cache()

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wk, args.cpu_rows)
    print(json.dumps(result), flush=True)


TRAFFIC_RECORD = os.path.join(REPO, "profiles", "rfq_gemm_large_qwen_hbm_counters.md")


def recorded_traffic(path=TRAFFIC_RECORD):
    """HBM bytes per launch of the product, from the FETCH_SIZE / WRITE_SIZE
    counter passes summarised in `path` (calibrated against a plain copy).
    The record names the sources it was measured on with their SHA-256; if
    any of them has changed since, the figure no longer describes this
    kernel and None is returned."""
    import hashlib
    try:
        with open(path) as f:
            lines = [ln for ln in f if ln.startswith("<!-- traffic-record ")]
    except OSError:
        return None
    if not lines:
        return None
    rec = json.loads(lines[0][len("<!-- traffic-record "):].rsplit("-->", 1)[0])
    for rel, digest in rec["sources"].items():
        try:
            with open(os.path.join(REPO, rel), "rb") as f:
                if hashlib.sha256(f.read()).hexdigest() != digest:
                    return None
        except OSError:
            return None
    return rec


# Seconds of back-to-back launches before a secondary measurement: on MI355X
# the clock drops a few milliseconds into sustained matrix-core load and
# settles again over the following ~100 ms, so every variant is timed in the
# settled state (the headline steps get their own --warmup instead).
SETTLE_S = 0.12


def _per_launch_ms(torch, stream, fn, reps, settle_s=SETTLE_S):
    """Mean time of `reps` back-to-back launches between one pair of events,
    after the same launches have run back to back for settle_s seconds."""
    t0 = time.perf_counter()
    i = 0
    while True:
        for _ in range(8):
            fn(i)
            i += 1
        torch.cuda.synchronize()
        if time.perf_counter() - t0 >= settle_s:
            break
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for i in range(reps):
        fn(i)
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / reps


def _graph_ms(torch, layer, layers, reps=20):
    """Per-layer time of `layers` calls of layer(i) captured in one HIP graph
    (warmed up on a side stream first, as capture requires) and replayed
    `reps` times between one pair of events."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(layers):
            layer(i)
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(layers):
            layer(i)
    graph.replay()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        graph.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / (reps * layers)


def secondary(torch, rfq, wl, x, w, stream):
    """Rates reported beside the headline step: the product without the
    residual (plain MXFP4), the bf16 matrix product of the same shape
    (hipBLASLt through torch), decode-sized products (1 and 16 activation
    rows, codes in and streaming form), the product on the Wan2.2-DiT-like
    shape, and the chained SwiGLU MLP block (quantize -> gate and up
    products -> SwiGLU + quantize -> down product, weights quantized
    beforehand)."""
    out = {}
    M, K = x.shape
    N = w.shape[0]
    q = rfq.rfq_quantize_act(x)
    wq = rfq.rfq_quantize_weight(w)
    z = torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    ms = _per_launch_ms(torch, stream, lambda i: rfq.rfq_gemm(
        q[0], q[1], None, None, *wq, out=z, stream=stream), 20)
    out["rfq_gemm_plain_mxfp4"] = {"ms": round(ms, 5),
                                   "exec_tflops": round(2.0 * M * N * K / ms / 1e9, 1)}
    wt = w.to(torch.bfloat16).t().contiguous()
    ms = _per_launch_ms(torch, stream, lambda i: torch.matmul(x, wt, out=z), 20)
    out["bf16_matmul"] = {"ms": round(ms, 5), "tflops": round(2.0 * M * N * K / ms / 1e9, 1)}
    # The vendor's block-scaled FP4 product (hipBLASLt through torch) on the
    # same primary codes: one plain MXFP4 contraction.
    try:
        a4 = q[0].view(torch.float4_e2m1fn_x2)
        b4 = wq[0].view(torch.float4_e2m1fn_x2).t()
        sa = q[1].view(torch.float8_e8m0fnu)
        sb = wq[1].view(torch.float8_e8m0fnu)
        ms = _per_launch_ms(torch, stream, lambda i: torch._scaled_mm(
            a4, b4, sa, sb, out_dtype=torch.bfloat16), 20)
        out["hipblaslt_mxfp4_scaled_mm"] = {
            "ms": round(ms, 5), "exec_tflops": round(2.0 * M * N * K / ms / 1e9, 1)}
    except (AttributeError, RuntimeError, ValueError, NotImplementedError) as e:
        out["hipblaslt_mxfp4_scaled_mm"] = {"unavailable": str(e)[:120]}
    # The FP4 matrix cores' sustained rate without memory traffic: the
    # register-only MFMA loop of the library (the product's instruction,
    # workgroup shape and accumulator pattern), with random and with
    # constant operand bits; about 0.2 ms per launch.
    loop = {}
    sink = torch.empty(rfq.MFMA_LOOP_ITEMS, dtype=torch.float32, device=x.device)
    for mode, rnd in (("random_operands", True), ("constant_operands", False)):
        ms = _per_launch_ms(torch, stream, lambda i: rfq.rfq_mfma_fp4_loop(
            MFMA_LOOP_ITERS, random_operands=rnd, sink=sink, stream=stream), 20)
        loop[mode] = {"ms": round(ms, 5), "tflops": round(
            MFMA_LOOP_ITERS * rfq.MFMA_LOOP_FLOPS_PER_ITER / ms / 1e9, 1)}
    out["mfma_fp4_register_loop"] = loop
    # The same loop on the bf16 matrix cores the HiF4 product runs on.
    loop = {}
    for mode, rnd in (("random_operands", True), ("constant_operands", False)):
        ms = _per_launch_ms(torch, stream, lambda i: rfq.rfq_mfma_bf16_loop(
            MFMA_LOOP_ITERS, random_operands=rnd, sink=sink, stream=stream), 20)
        loop[mode] = {"ms": round(ms, 5), "tflops": round(
            MFMA_LOOP_ITERS * rfq.MFMA_BF16_LOOP_FLOPS_PER_ITER / ms / 1e9, 1)}
    out["mfma_bf16_register_loop"] = loop
    # Fallback indicator by the scale-threshold rule (phi = 1 on tiles holding
    # a primary scale byte >= the median + margin): residual work only where
    # outliers are, at three thresholds; exec_tflops counts the MFMA work
    # done (2MNK plus 2MNK times the fraction of tiles on).
    med = int(q[1].float().median().item())
    sweep = []
    for margin in PHI_MARGINS:
        phi = rfq.rfq_fallback_map(None, q[1], rfq.RFQ_PHI_SCALE_AT_LEAST, med + margin)
        ms = _per_launch_ms(torch, stream, lambda i: rfq.rfq_gemm_phi(
            *q, *wq, phi, out=z, stream=stream), 20)
        on = float(phi.float().mean().item())
        sweep.append({"margin": margin, "threshold_byte": med + margin, "tiles_on": round(on, 4),
                      "ms": round(ms, 5),
                      "exec_tflops": round((2.0 + 2.0 * on) * M * N * K / ms / 1e9, 1)})
        del phi
    out["rfq_gemm_phi_scale_threshold"] = sweep
    del q, z, wt

    # HiF4 form (64-element blocks, E6M2 macro scale, micro-exponents): the
    # quantizer (primary + residual of the bf16 activations) and the product,
    # which decodes to bf16 and runs the bf16 matrix cores (no HiF4 format
    # there), so its rate is set against the 2.5 PFLOP/s dense bf16 peak.
    bf16_loop = out["mfma_bf16_register_loop"]["random_operands"]["tflops"]
    hq = rfq.rfq_hif4_quantize(x)
    hw = rfq.rfq_hif4_quantize(w, residual=False)
    ms = _per_launch_ms(torch, stream, lambda i: rfq.rfq_hif4_quantize(x, out=hq, stream=stream),
                        20)
    hbytes = M * K * x.element_size() + 2 * (M * K // 2 + M * K // 64 * 4)
    out["hif4_quantize_act"] = {"ms": round(ms, 5), "gb_per_s": round(hbytes / ms / 1e6, 1)}
    z = torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    for res in (True, False):
        ms = _per_launch_ms(torch, stream, lambda i: rfq.rfq_hif4_gemm(
            hq[0], hq[1], hq[2] if res else None, hq[3] if res else None, hw[0], hw[1], out=z,
            stream=stream), 10)
        tf = (4.0 if res else 2.0) * M * N * K / ms / 1e9
        out["hif4_gemm" if res else "hif4_gemm_plain"] = {
            "ms": round(ms, 5), "exec_tflops": round(tf, 1),
            "frac_of_bf16_peak": round(tf / (PEAK_BF16_TFLOPS), 4),
            "frac_of_bf16_loop_random": round(tf / bf16_loop, 4)}
    # The product given a workspace (rfq_hif4_gemm_split): at this size the
    # weights are decoded to bf16 into it on every call, then multiplied.
    ms = _per_launch_ms(torch, stream, lambda i: rfq.rfq_hif4_gemm(
        *hq, hw[0], hw[1], out=z, stream=stream, split=True), 10)
    tf = 4.0 * M * N * K / ms / 1e9
    out["hif4_gemm_workspace"] = {"ms": round(ms, 5), "exec_tflops": round(tf, 1),
                                  "frac_of_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
                                  "frac_of_bf16_loop_random": round(tf / bf16_loop, 4),
                                  "workspace_bytes": rfq.rfq_hif4_gemm_workspace_bytes(M, N, K)}
    # The same product with the weights decoded to bf16 once (exact; constant
    # weights, or weights re-quantized once per training step).
    wv = rfq.rfq_hif4_dequant(hw[0], hw[1], out_dtype=torch.bfloat16)
    ms = _per_launch_ms(torch, stream, lambda i: rfq.rfq_hif4_gemm_wbf16(
        *hq, wv, out=z, stream=stream), 10)
    tf = 4.0 * M * N * K / ms / 1e9
    out["hif4_gemm_bf16_weights"] = {"ms": round(ms, 5), "exec_tflops": round(tf, 1),
                                     "frac_of_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
                                     "frac_of_bf16_loop_random": round(tf / bf16_loop, 4)}
    del hq, hw, z, wv

    # Decode-sized products on the same weight: few activation rows, codes in
    # (rfq_quantize_act + rfq_gemm, whose few-row kernel streams W) and the
    # streaming form (rfq_gemm_stream, activations quantized inside the
    # product).  Ten weight copies (267 MB, beyond the last-level cache) are
    # rotated, as a model's many layers would be.
    wcs = [(torch.roll(wq[0], 97 * s, 0), torch.roll(wq[1], 97 * s, 0)) for s in range(10)]
    w_bytes = N * K // 2 + N * K // 32
    for md in (1, 16):
        xd = x[:md].contiguous()
        qd = rfq.rfq_quantize_act(xd)
        zd = torch.empty((md, N), dtype=torch.bfloat16, device=x.device)

        def codes_path(i):
            rfq.rfq_quantize_act(xd, out=qd, stream=stream)
            rfq.rfq_gemm(*qd, *wcs[i % 10], out=zd, stream=stream)

        ms_c = _per_launch_ms(torch, stream, codes_path, 50)
        ms_s = _per_launch_ms(torch, stream, lambda i: rfq.rfq_gemm_stream(
            xd, *wcs[i % 10], out=zd, stream=stream), 50)
        # The same ten layers captured once into a HIP graph and replayed:
        # the launch overhead of back-to-back calls leaves the timing.
        gc_ms = _graph_ms(torch, lambda i: (rfq.rfq_quantize_act(xd, out=qd),
                                            rfq.rfq_gemm(*qd, *wcs[i], out=zd)), 10)
        gs_ms = _graph_ms(torch, lambda i: rfq.rfq_gemm_stream(xd, *wcs[i], out=zd), 10)
        out["decode_%dx%dx%d" % (md, K, N)] = {
            "quantize_then_gemm_ms": round(ms_c, 5), "stream_ms": round(ms_s, 5),
            "w_gbs_quantize_then_gemm": round(w_bytes / ms_c / 1e6, 1),
            "w_gbs_stream": round(w_bytes / ms_s / 1e6, 1),
            "hip_graph_quantize_then_gemm_ms": round(gc_ms, 5),
            "hip_graph_stream_ms": round(gs_ms, 5)}
    del wq, wcs

    # HiF4 at the same decode shapes (few-row HiF4 kernel; codes in).
    hw = rfq.rfq_hif4_quantize(w, residual=False)
    hws = [(torch.roll(hw[0], 97 * s, 0), torch.roll(hw[1], 97 * s, 0)) for s in range(10)]
    for md in (1, 16):
        xd = x[:md].contiguous()
        hq = rfq.rfq_hif4_quantize(xd)
        zd = torch.empty((md, N), dtype=torch.bfloat16, device=x.device)

        def hif4_path(i):
            rfq.rfq_hif4_quantize(xd, out=hq, stream=stream)
            rfq.rfq_hif4_gemm(*hq, *hws[i % 10], out=zd, stream=stream)

        ms = _per_launch_ms(torch, stream, hif4_path, 50)
        out["hif4_decode_%dx%dx%d" % (md, K, N)] = {
            "quantize_then_gemm_ms": round(ms, 5),
            "w_gbs": round((N * K // 2 + N * K // 64 * 4) / ms / 1e6, 1)}
    del hw, hws

    # Wan2.2-DiT-like product: X 32768x5120, W 5120x13824.
    d = wl.generate(wl.WORKLOADS["wan"], seed=0)
    xw = torch.from_numpy(d["x_bf16"].view(np.int16)).to(x.device).view(torch.bfloat16)
    ww = torch.from_numpy(d["w"]).to(x.device)
    del d
    Mw, Kw = xw.shape
    Nw = ww.shape[0]
    q = rfq.rfq_quantize_act(xw)
    wq = rfq.rfq_quantize_weight(ww)
    del xw, ww
    z = torch.empty((Mw, Nw), dtype=torch.bfloat16, device=x.device)
    ms = _per_launch_ms(torch, stream, lambda i: rfq.rfq_gemm(*q, *wq, out=z, stream=stream), 5)
    out["rfq_gemm_wan_32768x5120x13824"] = {
        "ms": round(ms, 5), "exec_tflops": round(4.0 * Mw * Nw * Kw / ms / 1e9, 1)}
    del q, wq, z
    torch.cuda.empty_cache()

    # SwiGLU MLP block on the Qwen3-VL-like activations.
    d = wl.generate(wl.WORKLOADS["swiglu"], seed=0)
    dev = x.device
    xs = torch.from_numpy(d["x_bf16"].view(np.int16)).to(dev).view(torch.bfloat16)
    wg = rfq.rfq_quantize_weight(torch.from_numpy(d["w_gate"]).to(dev))
    wu = rfq.rfq_quantize_weight(torch.from_numpy(d["w_up"]).to(dev))
    wd32 = torch.from_numpy(d["w_down"]).to(dev)
    wd = rfq.rfq_quantize_weight(wd32)
    del d
    Ms, Ks = xs.shape
    Nh = wg[0].shape[0]
    q = [torch.empty((Ms, Ks // 2), dtype=torch.uint8, device=dev),
         torch.empty((Ms, Ks // 32), dtype=torch.uint8, device=dev),
         torch.empty((Ms, Ks // 2), dtype=torch.uint8, device=dev),
         torch.empty((Ms, Ks // 32), dtype=torch.uint8, device=dev)]
    g = torch.empty((Ms, Nh), dtype=torch.bfloat16, device=dev)
    u = torch.empty_like(g)
    h = [torch.empty((Ms, Nh // 2), dtype=torch.uint8, device=dev),
         torch.empty((Ms, Nh // 32), dtype=torch.uint8, device=dev),
         torch.empty((Ms, Nh // 2), dtype=torch.uint8, device=dev),
         torch.empty((Ms, Nh // 32), dtype=torch.uint8, device=dev)]
    y = torch.empty((Ms, Ks), dtype=torch.bfloat16, device=dev)

    def block(i):
        rfq.rfq_quantize_act(xs, out=q, stream=stream)
        rfq.rfq_gemm(*q, *wg, out=g, stream=stream)
        rfq.rfq_gemm(*q, *wu, out=u, stream=stream)
        rfq.rfq_swiglu_quantize_act(g, u, out=h, stream=stream)
        rfq.rfq_gemm(*h, *wd, out=y, stream=stream)

    ms = _per_launch_ms(torch, stream, block, 10)
    flops = 4.0 * Ms * Ks * Nh * 3
    out["swiglu_mlp_block_4096x4096x12288"] = {
        "ms": round(ms, 5), "exec_tflops": round(flops / ms / 1e9, 1),
        "stages": "quantize X; RFQ gate and up products (N=12288 each); SwiGLU + RFQ "
                  "quantize (K=12288); RFQ down product; bf16 outputs"}

    # The same block with SwiGLU + quantization fused into the gate/up product.
    wgu = (rfq.interleave_gate_up(wg[0], wu[0]), rfq.interleave_gate_up(wg[1], wu[1]))
    del g, u

    def fused(i):
        rfq.rfq_quantize_act(xs, out=q, stream=stream)
        rfq.rfq_gemm_swiglu_quantize(*q, *wgu, out=h, stream=stream)
        rfq.rfq_gemm(*h, *wd, out=y, stream=stream)

    ms = _per_launch_ms(torch, stream, fused, 10)
    out["swiglu_mlp_block_fused_4096x4096x12288"] = {
        "ms": round(ms, 5), "exec_tflops": round(flops / ms / 1e9, 1),
        "stages": "quantize X; RFQ gate/up product (N=24576) with SwiGLU + RFQ quantize "
                  "in its epilogue; RFQ down product; bf16 output"}

    # Batched-decode and prefill-sized token counts through the block's
    # products: the gate product (12288 x 4096 weights; few-row kernel at 64
    # rows, 128-wide tiles above) and the down product (4096 x 12288
    # weights), the latter with K unsplit (rfq_gemm) and split over
    # workgroups (rfq_gemm_split).
    for mp in (64, 256, 512):
        qp = [t[:mp] for t in q]
        hp = [t[:mp] for t in h]
        gp = torch.empty((mp, Nh), dtype=torch.bfloat16, device=dev)
        yp = torch.empty((mp, Ks), dtype=torch.bfloat16, device=dev)
        ms_g = _per_launch_ms(torch, stream, lambda i: rfq.rfq_gemm(
            *qp, *wg, out=gp, stream=stream), 20)
        ms_d = _per_launch_ms(torch, stream, lambda i: rfq.rfq_gemm(
            *hp, *wd, out=yp, stream=stream), 20)
        nb = rfq.rfq_gemm_workspace_bytes(mp, Ks, Nh)
        ws = torch.empty(max(nb, 16), dtype=torch.uint8, device=dev)
        ms_s = _per_launch_ms(torch, stream, lambda i: rfq.rfq_gemm_split(
            *hp, *wd, ws, out=yp, stream=stream), 20)
        fl = 4.0 * mp * Ks * Nh
        out["prefill_%d_rows" % mp] = {
            "gate_ms": round(ms_g, 5), "gate_exec_tflops": round(fl / ms_g / 1e9, 1),
            "down_ms": round(ms_d, 5), "down_exec_tflops": round(fl / ms_d / 1e9, 1),
            "down_split_ms": round(ms_s, 5), "down_split_exec_tflops": round(fl / ms_s / 1e9, 1),
            "down_split_workspace_bytes": nb}

    # The down product in HiF4 at 256 rows (activations N(0,1) in bf16; the
    # tile product with K unsplit and split over workgroups).
    hwd = rfq.rfq_hif4_quantize(wd32, residual=False)
    del wd32
    mp = 256
    hx = rfq.rfq_hif4_quantize(torch.randn((mp, Nh), device=dev).to(torch.bfloat16))
    yp = torch.empty((mp, Ks), dtype=torch.bfloat16, device=dev)
    ms_d = _per_launch_ms(torch, stream, lambda i: rfq.rfq_hif4_gemm(
        *hx, hwd[0], hwd[1], out=yp, stream=stream), 20)
    nb = rfq.rfq_hif4_gemm_workspace_bytes(mp, Ks, Nh)
    ws = torch.empty(max(nb, 16), dtype=torch.uint8, device=dev)
    ms_s = _per_launch_ms(torch, stream, lambda i: rfq.rfq_hif4_gemm_split(
        *hx, hwd[0], hwd[1], ws, out=yp, stream=stream), 20)
    fl = 4.0 * mp * Ks * Nh
    out["hif4_prefill_%d_rows" % mp] = {
        "down_ms": round(ms_d, 5), "down_exec_tflops": round(fl / ms_d / 1e9, 1),
        "down_split_ms": round(ms_s, 5), "down_split_exec_tflops": round(fl / ms_s / 1e9, 1),
        "down_split_workspace_bytes": nb}
    return out


def accuracy(torch, rfq, x, w, nrows=64):
    """Relative Frobenius errors against the fp64 product of the unquantized
    activations (bf16 values) and the fp32 master weights, on `nrows` rows
    spread over the batch: bf16 matrix product, plain MXFP4, RFQ, and the
    weight-only floor X deq(Q(W))."""
    M = x.shape[0]
    rows = torch.arange(0, M, max(M // nrows, 1), device=x.device)[:nrows]
    x64 = x[rows].double()
    zt = x64 @ w.double().t()
    nt = torch.linalg.norm(zt)

    def rel(z):
        return float(torch.linalg.norm(z[rows].double() - zt) / nt)

    q = rfq.rfq_quantize_act(x)
    wq = rfq.rfq_quantize_weight(w)
    wt = w.to(torch.bfloat16).t().contiguous()
    out = {
        "bf16_matmul": rel(torch.matmul(x, wt)),
        "plain_mxfp4": rel(rfq.rfq_gemm(q[0], q[1], None, None, *wq)),
        "rfq": rel(rfq.rfq_gemm(*q, *wq)),
    }
    med = int(q[1].float().median().item())
    for margin in PHI_MARGINS:
        phi = rfq.rfq_fallback_map(None, q[1], rfq.RFQ_PHI_SCALE_AT_LEAST, med + margin)
        out["rfq_phi_scale_threshold_margin%d" % margin] = rel(rfq.rfq_gemm_phi(*q, *wq, phi))
    hq = rfq.rfq_hif4_quantize(x)
    hw = rfq.rfq_hif4_quantize(w, residual=False)
    out["plain_hif4"] = rel(rfq.rfq_hif4_gemm(hq[0], hq[1], None, None, hw[0], hw[1]))
    out["rfq_hif4"] = rel(rfq.rfq_hif4_gemm(*hq, hw[0], hw[1]))
    del hq, hw
    wdq = rfq.rfq_dequant(*wq).double()
    out["weight_only_floor"] = float(torch.linalg.norm(x64 @ wdq.t() - zt) / nt)
    out["rows"] = int(rows.numel())
    return {k: (round(v, 6) if isinstance(v, float) else v) for k, v in out.items()}


def cpu_baseline(wk, rows):
    """The oracle, as it stands, on a bounded sample of one step: the whole
    weight quantization plus `rows` activation rows through the activation
    quantizer and the product (all N outputs).  Scaled to a full step as
    t_w + (M / rows) * (t_x + t_gemm)."""
    import oracle
    from paper_2608_26581_amd import workloads as wl
    o = oracle.default()
    d = wl.generate(wk, seed=0)
    M, K = d["x"].shape
    N = d["w"].shape[0]
    t = time.perf_counter()
    wc, wsc, _, _ = o.quantize(d["w"], residual=False)
    t_w = time.perf_counter() - t
    t = time.perf_counter()
    q = o.quantize(d["x"][:rows])
    t_x = time.perf_counter() - t
    t = time.perf_counter()
    o.gemm(*q, wc, wsc)
    t_g = time.perf_counter() - t
    t_step = t_w + (M / rows) * (t_x + t_g)
    # The same with one thread, on a smaller sample: 1/16 of the weight rows
    # and one activation row.
    cores = o.num_threads()
    o.set_num_threads(1)
    wrows = max(N // 16, 1)
    t = time.perf_counter()
    o.quantize(d["w"][:wrows], residual=False)
    t_w1 = (time.perf_counter() - t) * (N / wrows)
    t = time.perf_counter()
    q1 = o.quantize(d["x"][:1])
    o.gemm(*q1, wc, wsc)
    t_r1 = time.perf_counter() - t
    o.set_num_threads(cores)
    t_step1 = t_w1 + M * t_r1
    return {
        "value": round(4.0 * M * N * K / t_step / 1e12, 6),
        "unit": "TFLOP/s",
        "cores": cores,
        "single_thread_value": round(4.0 * M * N * K / t_step1 / 1e12, 7),
        "cpu": _cpu_model(),
        "kind": "oracle",
        "sample": "full weight quantization (%dx%d) + %d activation rows through the RFQ "
                  "quantizer and the fp64 product against all %d outputs; scaled to the "
                  "%d-row step (t_w=%.2fs t_x=%.3fs t_gemm=%.2fs); single_thread_value: 1/%d "
                  "of the weight rows and 1 activation row on one thread, scaled the same "
                  "way" % (N, K, rows, N, M, t_w, t_x, t_g, N // wrows),
    }


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


if __name__ == "__main__":
    main()
