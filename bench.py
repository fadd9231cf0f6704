#!/usr/bin/env python3
"""Benchmark: FQT backward of one Transformer-FFN shaped linear layer on one MI355X.

Workload: X [8192, 1024], W [4096, 1024], G [8192, 4096] float32 (1% outlier
gradient rows), grad_X quantizer BHQ 5-bit with block size 64, grad_W
quantizer 8-bit stochastic PTQ, X and W 8-bit deterministic PTQ.  A step is
one fqt_linear_backward call (statistics, BHQ plan, all quantizers, both int8
contractions and their dequantizing epilogues) on inputs resident in HBM.

Prints one JSON line: the int8 throughput of the whole layer backward
(2 * 2 N d_in d_out ops per step / step time), per-phase times from HIP
events recorded in a second run of the same steps, the roofline of the
dominant kernel (the fused quantizer launch, against HBM, with its measured
vector-ALU busy share beside it) and the CPU oracle timed on a bounded
sample of the same layer, single-threaded and on all host cores.  Extra legs:
the multi-layer chain, the low-bit grad_W quantizer, sub-8-bit contractions,
the paper's conv layer, every ResNet-50 conv shape at batch 256 for three
gradient quantizers, and the seed-batched quantizer over 1000 seeds.
"""
import argparse
import json
import os
import sys
import time

N, D_IN, D_OUT = 8192, 1024, 4096
QB_X = ("bhq", 5, 64)
QB_W = ("ptq", 8, 0)
HBM_PEAK_GBS = 8000.0            # MI355X HBM3E
INT8_PEAK_TOPS = 5000.0          # MI355X dense int8 matrix cores
CPU_SAMPLE_ROWS = N          # the whole layer: about 15 s of oracle work per thread setting


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-chain", action="store_true", help="skip every leg beyond the layer backward")
    ap.add_argument("--legs", default="chain,shift,bf6,conv,resnet,seeds",
                    help="comma list of the legs beyond the layer backward (chain, shift, bf6, conv, resnet, seeds)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="after timing, run a plain 256 MiB elementwise pass (traffic-counter calibration)")
    return ap.parse_args()


TRAFFIC_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "traffic_linear_ffn_bhq5.txt")
COUNTER_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "counters_linear_ffn_bhq5.json")
SEEDS_COUNTER_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "counters_seed_batch.json")
# kernel of each phase in the rocprofv3 summaries (name prefixes)
PHASE_KERNEL = {
    "quant_G": ("quant_fused_kernel<2, 64, 1>",),
    "gemm_gradX": ("gemm_i8_kernel<fqt::TileCfg<256", ", 3, 64, true>"),
    "gemm_gradW": ("gemm_i8_kernel<fqt::TileCfg<128", ", 1, 0, true>"),
}


def measured_traffic(phase):
    """HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE summary, if it
    was taken on the current kernel sources; else None."""
    try:
        from paper_2010_14298_amd import profiling
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        if t.get("kernel_sources") != profiling.source_hash():
            return None
        for name, v in t["kernels"].items():
            if all(part in name for part in PHASE_KERNEL[phase]):
                return v["bytes"]
    except (OSError, ValueError, KeyError):
        return None
    return None


def measured_counters(phase, path=COUNTER_FILE, parts=None):
    """Counter summary of one kernel (a phase's, or the kernel whose name holds
    every string of `parts`) from committed rocprofv3 passes, if they were taken
    on the current kernel sources; else None."""
    try:
        from paper_2010_14298_amd import profiling
        with open(path) as f:
            t = json.load(f)
        if t.get("kernel_sources") != profiling.source_hash():
            return None
        for name, v in t["kernels"].items():
            if all(part in name for part in (parts or PHASE_KERNEL[phase])):
                return v
    except (OSError, ValueError, KeyError):
        return None
    return None


def cpu_baseline(X, W, G):
    """The oracle, as is, on the first CPU_SAMPLE_ROWS samples (all of them) of the same layer:
    its quantizers (Q_f, Q_theta, Q_b1, Q_b2) and its contractions (float64
    products of the dequantized operands) timed apart, with one thread and
    with every host core (numpy's BLAS threads)."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits
    from oracle import backward as BW
    from oracle import quantizers as Q
    n = CPU_SAMPLE_ROWS
    Xs, Gs = X[:n], G[:n]

    def step():
        t0 = time.perf_counter()
        qx = Q.quantize_ptq(Xs, 8, False)
        qw = Q.quantize_ptq(W, 8, False)
        qb1 = BW.quantize_gradient(Gs, QB_W, 0, 0)
        qb2 = BW.quantize_gradient(Gs, QB_X, 0, 1)
        t1 = time.perf_counter()
        Xr, Wr, G1r, G2r = (Q.dequantize(q) for q in (qx, qw, qb1, qb2))
        gW = (G1r.T @ Xr).astype(np.float32)
        gX = (G2r @ Wr).astype(np.float32)
        t2 = time.perf_counter()
        return t1 - t0, t2 - t1

    ops = 2.0 * 2.0 * n * D_IN * D_OUT
    res = {}
    for label, limit in (("one_core", 1), ("all_cores", None)):
        if limit is None:
            tq, tc = step()
            threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        else:
            with threadpool_limits(limits=limit):
                tq, tc = step()
            threads = 1
        res[label] = {"quantizers_s": round(tq, 3), "contractions_s": round(tc, 3),
                      "TOPS": ops / (tq + tc) / 1e12, "threads": int(threads)}
    a = res["all_cores"]
    return {"value": a["TOPS"], "unit": "TOPS", "cores": a["threads"], "kind": "oracle",
            "sample": (f"the whole layer ({N} samples)" if n == N else f"first {n} of {N} samples of the layer")
                      + f", full d_in and d_out, BHQ-5 k=64; {a['quantizers_s'] + a['contractions_s']:.1f} s "
                      "on all cores",
            "per_step": res}


CHAIN_WIDTHS = (1024, 4096, 4096, 1024)   # FFN-like ReLU MLP: up, square, down


def measured_peaks(fqt, torch):
    """The machine's own ceilings: the library's register-only int8 matrix-core
    loop and its streaming copy, timed with HIP events."""
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    fqt.fqt_probe_mfma_i8(100, sink)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    ops = fqt.fqt_probe_mfma_i8(10000, sink)
    e1.record()
    torch.cuda.synchronize()
    mfma = ops / (e0.elapsed_time(e1) * 1e-3) / 1e12
    src = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    fqt.fqt_probe_copy(src, dst)
    e0.record()
    moved = sum(fqt.fqt_probe_copy(src, dst) for _ in range(5))
    e1.record()
    torch.cuda.synchronize()
    copy = moved / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    return {"mfma_i8_TOPS": round(mfma, 1), "copy_GBps": round(copy, 1),
            "mfma_frac_of_spec": round(mfma / INT8_PEAK_TOPS, 4), "copy_frac_of_spec": round(copy / HBM_PEAK_GBS, 4)}


def chain_bench(args, fqt, synth, torch):
    """The multi-layer chain: forward (Q_f, Q_theta, int8 product, ReLU) and FQT
    backward (Q_b2 = BHQ 5-bit, Q_b1 = PTQ 8-bit, ReLU masks) of a 3-layer MLP
    on N tokens, timed with HIP events on the library's stream."""
    import numpy as np
    X, Ws, _ = synth.mlp(seed=0, n=N, widths=CHAIN_WIDTHS)
    _, _, Gtop = synth.linear_outlier(seed=1, n=N, d_in=8, d_out=CHAIN_WIDTHS[-1])
    dX, dG = torch.from_numpy(X).cuda(), torch.from_numpy(Gtop).cuda()
    dWs = [torch.from_numpy(W).cuda() for W in Ws]
    specs = [QB_X] * len(dWs)
    steps = max(1, args.steps // 4)
    for i in range(max(1, args.warmup // 4)):
        acts, _ = fqt.mlp_forward(dX, dWs)
        fqt.mlp_backward(acts, dWs, dG, specs, [i] * len(dWs), qb_w=QB_W)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    fwd, bwd = [], []
    for i in range(steps):
        ev[0].record()
        acts, _ = fqt.mlp_forward(dX, dWs)
        ev[1].record()
        fqt.mlp_backward(acts, dWs, dG, specs, [3 * i + j for j in range(len(dWs))], qb_w=QB_W)
        ev[2].record()
        torch.cuda.synchronize()
        fwd.append(ev[0].elapsed_time(ev[1]))
        bwd.append(ev[1].elapsed_time(ev[2]))
    layer_ops = sum(2.0 * N * CHAIN_WIDTHS[i] * CHAIN_WIDTHS[i + 1] for i in range(len(dWs)))
    f_ms, b_ms = float(np.mean(fwd)), float(np.mean(bwd))
    return {"workload": f"ReLU MLP {'-'.join(map(str, CHAIN_WIDTHS))}, N={N}; forward + FQT backward "
                        "(Q_b2 = BHQ 5-bit block 64, Q_b1 = PTQ 8-bit)",
            "steps": steps, "forward_ms": round(f_ms, 4), "backward_ms": round(b_ms, 4),
            "ms_per_step": round(f_ms + b_ms, 4),
            "forward_TOPS": round(layer_ops / (f_ms * 1e-3) / 1e12, 2),
            "backward_TOPS": round(2.0 * layer_ops / (b_ms * 1e-3) / 1e12, 2),
            "TOPS": round(3.0 * layer_ops / ((f_ms + b_ms) * 1e-3) / 1e12, 2)}


def shift_bench(args, fqt, torch, dX, dW, dG):
    """The same layer backward with a low-bit grad_W quantizer carrying
    per-sample power-of-two scales (Q_b1 = shift 4-bit), HIP events."""
    import numpy as np
    qb_w = ("shift", 4, 0)
    cfg = fqt.cfg_struct(QB_X, qb_w, 8, 8, 0)
    ws = torch.empty(fqt.fqt_linear_backward_workspace(N, D_IN, D_OUT, cfg), dtype=torch.uint8, device="cuda")
    gW = torch.empty((D_OUT, D_IN), dtype=torch.float32, device="cuda")
    gX = torch.empty((N, D_IN), dtype=torch.float32, device="cuda")
    steps = max(1, args.steps // 4)
    for i in range(max(1, args.warmup // 4)):
        fqt.fqt_linear_backward(dX, dW, dG, qb_x=QB_X, qb_w=qb_w, seed=i, grad_W=gW, grad_X=gX, ws=ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        fqt.fqt_linear_backward(dX, dW, dG, qb_x=QB_X, qb_w=qb_w, seed=i, grad_W=gW, grad_X=gX, ws=ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    return {"workload": "the same layer backward, Q_b1 = per-tensor range with per-sample power-of-two "
                        "steps, 4-bit (shifted codes, E = 4)", "steps": steps, "ms_per_step": round(ms, 4),
            "TOPS": round(2.0 * 2.0 * N * D_IN * D_OUT / (ms * 1e-3) / 1e12, 2)}


def conv_bench(args, fqt, synth, torch, qb_w=None):
    """The conv layer of the paper's overhead example (N = 128, C = 64, 56 x 56;
    a 3 x 3, 64 -> 64, stride-1 conv): the whole FQT backward with Q_b2 = BHQ
    5-bit across samples (block 64), Q_b1 = PTQ 8-bit (or per sample: grad_W
    in one K block per sample), HIP events."""
    qb_w = qb_w or QB_W
    n, c, h, o, k = 128, 64, 56, 64, 3
    X, W, G = synth.conv_layer(seed=0, n=n, c=c, h=h, w=h, o=o, k=k, stride=1, pad=1)
    dX, dW, dG = (torch.from_numpy(a).cuda() for a in (X, W, G))
    gW = torch.empty(W.shape, dtype=torch.float32, device="cuda")
    gX = torch.empty(X.shape, dtype=torch.float32, device="cuda")
    ws = None
    for i in range(3):
        _, _, ws = fqt.fqt_conv_backward_im2col(dX, dW, dG, 1, 1, qb_x=QB_X, qb_w=qb_w, seed=i, grad_W=gW,
                                                 grad_X=gX, ws=ws)
    torch.cuda.synchronize()
    steps = max(2, args.steps // 10)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(steps):
        fqt.fqt_conv_backward_im2col(dX, dW, dG, 1, 1, qb_x=QB_X, qb_w=qb_w, seed=i, grad_W=gW, grad_X=gX, ws=ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    ops = 2.0 * 2.0 * n * h * h * (c * k * k) * o
    return {"workload": "conv 3x3 64->64, 56x56, batch 128, stride 1 (the paper's overhead-example layer); "
                        "Q_b2 = BHQ 5-bit across samples (block 64), Q_b1 = %s %d-bit" % (qb_w[0].upper(), qb_w[1]),
            "steps": steps,
            "ms_per_step": round(ms, 4), "TOPS": round(ops / (ms * 1e-3) / 1e12, 2)}


def resnet_sweep(args, fqt, synth, torch):
    """Every ResNet-50 v1.5 conv shape (stem to stage 4) at batch 256: the whole
    FQT conv backward per layer for three gradient quantizers (Q_b2 = BHQ
    5-bit block 64, PSQ 8-bit, PTQ 8-bit; Q_b1 = PTQ 8-bit), HIP events.
    Inputs drawn on the device with the recipe of synth.conv_layer:
    post-ReLU half-normal X (N(0,1) at the stem), He-init W, per-sample
    LogNormal(0, 2) gradient scales.  The stem's input is the image, which
    takes no gradient in training: its row and the network total run it
    without grad_X (NULL), and its full backward is reported beside them."""
    import math
    n = 256
    specs = (("bhq5", ("bhq", 5, 64)), ("psq8", ("psq", 8, 0)), ("ptq8", ("ptq", 8, 0)))
    gen = torch.Generator(device="cuda").manual_seed(0)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = max(2, args.steps // 40)
    layers, net = [], {name: [0.0, 0.0] for name, _ in specs}
    for (c, o, k, stride, h, count) in synth.RESNET50_CONVS:
        pad = k // 2
        ho = (h + 2 * pad - k) // stride + 1
        X = torch.randn((n, h, h, c), generator=gen, device="cuda")
        if c != 3:
            X.clamp_(min=0.0)
        W = torch.randn((o, k, k, c), generator=gen, device="cuda") * math.sqrt(2.0 / (k * k * c))
        G = torch.exp(2.0 * torch.randn((n, 1, 1, 1), generator=gen, device="cuda")) * \
            torch.randn((n, ho, ho, o), generator=gen, device="cuda")
        ops = 2.0 * 2.0 * n * ho * ho * o * k * k * c
        row = {"shape": f"{c}->{o} k{k} s{stride} {h}->{ho}", "count": count, "GOP": round(ops / 1e9, 2)}
        gW, gX = torch.empty_like(W), torch.empty_like(X)
        stem = c == 3
        if stem:
            row["input_grad"] = False
            row["GOP"] = round(ops / 2 / 1e9, 2)  # the grad_W contraction only

        def timed(spec, input_grad):
            ws = None
            for i in range(2):
                _, _, ws = fqt.fqt_conv_backward_im2col(X, W, G, stride, pad, qb_x=spec, qb_w=QB_W, seed=i,
                                                         grad_W=gW, grad_X=gX, ws=ws, input_grad=input_grad)
            torch.cuda.synchronize()
            e0.record()
            for i in range(reps):
                fqt.fqt_conv_backward_im2col(X, W, G, stride, pad, qb_x=spec, qb_w=QB_W, seed=i, grad_W=gW,
                                             grad_X=gX, ws=ws, input_grad=input_grad)
            e1.record()
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / reps

        for name, spec in specs:
            lops = ops / 2 if stem else ops  # grad_W only
            ms = timed(spec, not stem)
            row[name] = {"ms": round(ms, 4), "TOPS": round(lops / (ms * 1e-3) / 1e12, 2)}
            if stem:
                row[name]["ms_with_input_grad"] = round(timed(spec, True), 4)
            net[name][0] += count * ms
            net[name][1] += count * lops
        layers.append(row)
        del X, W, G, gW, gX
    torch.cuda.empty_cache()
    return {"workload": "ResNet-50 v1.5 conv layers at batch 256 (224 x 224), every unique shape; whole FQT conv "
                        "backward per layer (the stem without its input gradient)", "steps_per_layer": reps,
            "layers": layers,
            "network": {name: {"ms": round(v[0], 3), "TOPS": round(v[1] / (v[0] * 1e-3) / 1e12, 2)}
                        for name, v in net.items()}}


def seeds_bench(args, fqt, synth, torch):
    """The seed-batched quantizer on the 4096 x 4096 single-outlier gradient:
    1000 seeds per quantizer and width in one launch each (G read once, every
    seed's codes drawn and summed per element), HIP events; draws per second,
    and the vector-ALU busy share of each quantizer's launches from the
    committed counter summary (all widths together)."""
    _, _, G = synth.linear_single_outlier(seed=0)
    dG = torch.from_numpy(G).cuda()
    S = 1000
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    res = {}
    for kind, k in (("ptq", 0), ("psq", 0), ("bhq", 64)):
        for bits in (4, 5, 6, 8):
            out = fqt.fqt_quantize_seeds(dG, kind, bits, 4, block_size=k)
            torch.cuda.synchronize()
            e0.record()
            out = fqt.fqt_quantize_seeds(dG, kind, bits, S, block_size=k, seed=0, stream=1, ws=out["ws"])
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1)
            r = {"ms": round(ms, 3), "draws_per_s": round(S * G.size / (ms * 1e-3), 1)}
            if bits == 5:
                s1 = out["sum_c"].double()
                var = (out["sum_c2"].double() - s1 * s1 / S) / (S - 1)
                r["sum_code_variance"] = round(float(var.sum()), 1)
            res[f"{kind}{bits}"] = r
        mode = {"ptq": 0, "psq": 1, "bhq": 2}[kind]
        cnt = measured_counters(None, SEEDS_COUNTER_FILE, (f"quant_seeds_kernel<{mode}, {k}>",))
        if cnt and "VALUBusy" in cnt:
            res[f"{kind}_valu_busy_pct"] = cnt["VALUBusy"]
    return {"workload": "4096 x 4096 gradient, N(0,1) with one row x 1000; 1000 seeds (keys 0..999) per "
                        "quantizer; PTQ / PSQ / BHQ block 64 at 4, 5, 6, 8 bits", "seeds": S, "runs": res}


def bf6_bench(args, fqt, torch):
    """Exact contraction of 4-bit codes: 6-bit float matrix cores (e3m2
    operands, packed in the call) against the int8 matrix cores, on the two
    contraction shapes of the layer; each call ends in int64 accumulators."""
    res = {}
    gen = torch.Generator(device="cuda").manual_seed(0)
    for name, (M, Nn, K) in {"gradX_shape": (N, D_IN, D_OUT), "gradW_shape": (D_OUT, D_IN, N)}.items():
        A = torch.randint(-8, 8, (M, K), dtype=torch.int8, device="cuda", generator=gen)
        B = torch.randint(-8, 8, (Nn, K), dtype=torch.int8, device="cuda", generator=gen)
        C = torch.empty((M, Nn), dtype=torch.int64, device="cuda")
        ws6 = torch.empty(fqt.fqt_gemm_s4s4_bf6_workspace(M, Nn, K), dtype=torch.uint8, device="cuda")
        ws8 = torch.empty(fqt.fqt_gemm_workspace(M, Nn, K), dtype=torch.uint8, device="cuda")
        calls = {"bf6": lambda: fqt.fqt_gemm_s4s4_bf6(A, B, ws=ws6, C=C),
                 "int8": lambda: fqt.fqt_gemm_s8s8_s64(A, B, ws=ws8)}
        row = {"M": M, "N": Nn, "K": K}
        for key, fn in calls.items():
            for _ in range(3):
                fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            reps = max(2, args.steps // 10)
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            row[key + "_call_ms"] = round(e0.elapsed_time(e1) / reps, 4)
        res[name] = row
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(the layer backward runs on a single MI355X)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch
    from paper_2010_14298_amd import fqt, synth

    fqt.load()
    X, W, G = synth.linear_outlier(seed=0, n=N, d_in=D_IN, d_out=D_OUT)
    dX, dW, dG = (torch.from_numpy(a).cuda() for a in (X, W, G))
    grad_W = torch.empty((D_OUT, D_IN), dtype=torch.float32, device="cuda")
    grad_X = torch.empty((N, D_IN), dtype=torch.float32, device="cuda")
    cfg = fqt.cfg_struct(QB_X, QB_W, 8, 8, 0)
    ws = torch.empty(fqt.fqt_linear_backward_workspace(N, D_IN, D_OUT, cfg), dtype=torch.uint8, device="cuda")

    def step(seed, trace=None):
        fqt.fqt_linear_backward(dX, dW, dG, qb_x=QB_X, qb_w=QB_W, seed=seed, grad_W=grad_W, grad_X=grad_X,
                                ws=ws, trace=trace)

    for i in range(args.warmup):
        step(1000 + i)
    torch.cuda.synchronize()
    if fqt.fqt_workspace_status(ws) != 0:
        raise RuntimeError("non-finite data reported by the workspace status")
    # timed region: K whole steps, nothing else on the stream
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    # per-kernel durations: the same K steps again with HIP events recorded by the
    # library around each phase on this stream (the markers add ~0.05 ms per step,
    # so they stay out of the timed region above)
    traces = [fqt.make_trace() for _ in range(args.steps)]
    for i in range(args.steps):
        step(i, traces[i])
    torch.cuda.synchronize()
    phase_ms = np.mean([fqt.trace_ms(t) for t in traces], axis=0)
    for t in traces:
        fqt.free_trace(t)
    phases = dict(zip(fqt.PHASE_NAMES, [round(float(v), 5) for v in phase_ms]))

    gemm_ops = 2.0 * N * D_IN * D_OUT               # per contraction
    value = 2.0 * gemm_ops / (ms_step * 1e-3) / 1e12
    nd = float(N) * D_OUT
    nxw = float(N) * D_IN + float(D_OUT) * D_IN
    # the quantizer launch: read G, write Q_b2 and Q_b1 codes; read X and W, write their codes
    quant_bytes = (4 + 2) * nd + (4 + 1) * nxw
    t_quant_g = phases["quant_G"] * 1e-3
    t_quantizer = (phases["stats"] + phases["scales_plan"] + phases["quant_G"]) * 1e-3
    kernels = {
        "gemm_gradX": {"bound": "mfma", "t": phases["gemm_gradX"] * 1e-3, "work": gemm_ops, "unit": "TOP/s",
                       "peak": INT8_PEAK_TOPS, "scale": 1e12},
        "gemm_gradW": {"bound": "mfma", "t": phases["gemm_gradW"] * 1e-3, "work": gemm_ops, "unit": "TOP/s",
                       "peak": INT8_PEAK_TOPS, "scale": 1e12},
        # the fused quantizer launch against HBM: algorithmic bytes (each input
        # read once, each code written once); its vector-ALU busy share, from
        # the committed counters, goes beside it
        "quant_G": {"bound": "hbm", "t": t_quant_g, "work": quant_bytes, "unit": "GB/s", "peak": HBM_PEAK_GBS,
                    "scale": 1e9},
    }
    measured = measured_peaks(fqt, torch)
    per_kernel = {}
    for name, k in kernels.items():
        ach = k["work"] / k["t"] / k["scale"]
        per_kernel[name] = {"bound": k["bound"], "achieved": round(ach, 2), "peak": k["peak"], "unit": k["unit"],
                            "frac": round(ach / k["peak"], 4), "ms": round(k["t"] * 1e3, 4)}
        mp = {"mfma": measured["mfma_i8_TOPS"], "hbm": measured["copy_GBps"]}.get(k["bound"])
        if mp:
            per_kernel[name]["measured_peak"] = mp
            per_kernel[name]["frac_measured"] = round(ach / mp, 4)
    for name in kernels:
        cnt = measured_counters(name)
        if cnt:
            per_kernel[name]["counters"] = cnt
    dom = max(kernels, key=lambda n: kernels[n]["t"])
    roof = dict(per_kernel[dom])
    roof.pop("ms")
    roof.pop("counters", None)
    roof["kernel"] = dom
    roof["traffic"] = measured_traffic(dom)
    cnt = measured_counters(dom)
    if cnt and "VALUBusy" in cnt:
        roof["valu_busy_pct"] = cnt["VALUBusy"]
    out = {
        "metric": "FQT layer-backward int8 TOPS + quantizer HBM GB/s (BHQ 5-bit) vs roofline",
        "value": round(value, 3),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8 contractions, f32 quantizers, f64 epilogue",
        "data": "synthetic",
        "config": {"workload": "linear FQT backward, N=8192 tokens, d_in=1024, d_out=4096, 1% outlier gradient "
                               "rows; Q_b2 = BHQ 5-bit block 64, Q_b1 = PTQ 8-bit, Q_f = Q_theta = PTQ 8-bit",
                   "global_batch": N, "parallelism": "single GPU"},
        "quantizer_GBps": round(quant_bytes / t_quantizer / 1e9, 2),
        "quant_G_pass_GBps": round(quant_bytes / t_quant_g / 1e9, 2),
        "phases_ms": phases,
        "measured_peaks": measured,
        "kernels": per_kernel,
        "roofline": roof,
    }
    legs = set() if args.no_chain else set(args.legs.split(","))
    if "chain" in legs:
        out["chain"] = chain_bench(args, fqt, synth, torch)
    if "shift" in legs:
        out["shift_gradW"] = shift_bench(args, fqt, torch, dX, dW, dG)
    if "bf6" in legs:
        out["sub8bit_mfma"] = bf6_bench(args, fqt, torch)
    if "conv" in legs:
        out["conv_layer"] = conv_bench(args, fqt, synth, torch)
        out["conv_layer_per_sample_b1"] = conv_bench(args, fqt, synth, torch, qb_w=("psq", 8, 0))
    if "resnet" in legs:
        out["resnet50_batch256"] = resnet_sweep(args, fqt, synth, torch)
    if "seeds" in legs:
        out["seed_batch"] = seeds_bench(args, fqt, synth, torch)
    if args.copy_probe:
        # a plain elementwise pass: reads 256 MiB, writes 256 MiB
        src = torch.ones(64 * 1024 * 1024, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(X, W, G)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
