"""Benchmark: compensated W4A16 decode of a Llama-3.1-8B-shaped decoder layer.

One step = the seven compensated linears of the layer (q, k, v, o, gate, up,
down; 4-bit, group 128; per-matrix ranks from the seeded allocator under a
budget of 64 x 7) decoding one batch of tokens through the C ABI, issued as
the layer's four compensation windows in dependency order: Q/K/V (one window:
they read the same input), O, gate/up (one window), down.  Weights are
seeded N(0, 0.02) draws quantized by the library on the GPU; compensation
factors are seeded fp16 stand-ins (the forward's cost does not depend on their
values).  Steps rotate over enough distinct copies of the layer (>= 1.5 GiB)
that every step streams its weights from HBM, not from the 256 MB Infinity
Cache.  Each step is a captured HIP graph of the four window calls, so host launch
overhead is outside the timed region; the inputs are resident in HBM.

Prints one JSON line: whole-job algorithmic HBM throughput (GB/s) of the step,
the roofline of the dominant call (the gate matrix, 14336 x 4096) timed with
HIP events on the stream it runs on, and the fp64 CPU oracle timed on the
same layer.
"""

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=240)
    p.add_argument("--warmup", type=int, default=24)
    p.add_argument("--tokens", type=int, default=1)
    p.add_argument("--rotate-gib", type=float, default=1.5)
    p.add_argument("--no-cpu-baseline", action="store_true")
    return p.parse_args()


def algorithmic_bytes(spec, T):
    """HBM bytes a compensated decode must move at minimum: packed codes,
    fp16 scales and zeros, the used rows of A and columns of B, activations in
    and fp16 outputs out."""
    q = spec.d_out * spec.d_in * spec.bits // 8
    sz = 2 * 2 * spec.d_out * (spec.d_in // spec.group_size)
    ab = 2 * spec.rank * (spec.d_in + spec.d_out)
    return q + sz + ab + 2 * T * spec.d_in + 2 * T * spec.d_out


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: the compensated linear runs on a single device; "
              "multi-GPU sharding is described in DESIGN.md and not run.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2605_05819_amd import cl, workloads as wl

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    T = args.tokens
    layer = wl.llama_layer()
    specs = layer.linears

    # ---- one layer on the device (library quantizer), then copies
    base = []
    for m, spec in enumerate(specs):
        W = torch.from_numpy(wl.weight((spec.d_out, spec.d_in), layer.index, 0, m)).to(dev)
        w = cl.quantize_pack(W, spec.bits, spec.group_size)
        del W
        A, B = wl.standin_factors(spec.d_out, spec.d_in, spec.r_max, layer.index, 0, m)
        c = cl.LowRank(torch.from_numpy(A).to(dev), torch.from_numpy(B).to(dev), spec.r_max, spec.rank)
        base.append((w, c))
    torch.cuda.synchronize()
    layer_bytes = sum(w.q.numel() * 4 + w.scales.numel() * 4 + c.A.numel() * 2 + c.B.numel() * 2
                      for w, c in base)
    ncopies = max(2, int(np.ceil(args.rotate_gib * 2 ** 30 / layer_bytes)))
    copies = [base]
    for _ in range(ncopies - 1):
        copies.append([(cl.QWeight(w.q.clone(), w.scales.clone(), w.zeros.clone(), w.d_out, w.d_in, w.bits,
                                   w.group_size), cl.LowRank(c.A.clone(), c.B.clone(), c.r_max, c.rank))
                       for w, c in base])
    xs, ys, wss = [], [], []
    for m, spec in enumerate(specs):
        x = wl.activation((T, spec.d_in), layer.index, 0, m)
        xs.append(torch.from_numpy(x.bits.view(np.int16)).view(torch.float16).to(dev))
        ys.append(torch.empty((T, spec.d_out), dtype=torch.float16, device=dev))
        wss.append(cl.workspace(cl.linear_workspace(base[m][0], base[m][1], T), dev))
    torch.cuda.synchronize()

    stream = torch.cuda.Stream()

    def capture(fn):
        """A HIP graph of fn() recorded on `stream` (after one eager run)."""
        with torch.cuda.stream(stream):
            fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            fn()
        torch.cuda.synchronize()
        return g

    # the layer's compensation windows: matrices that read the same input
    names = [s.name for s in specs]
    windows = [[names.index(n) for n in grp] for grp in (("q", "k", "v"), ("o",), ("gate", "up"), ("down",))]
    wxs = [xs[grp[0]] for grp in windows]          # one input per window
    wwss = [cl.workspace(cl.window_workspace([base[m][0] for m in grp], [base[m][1] for m in grp], T), dev)
            for grp in windows]

    def layer_calls(k):
        def run():
            for wi, grp in enumerate(windows):
                cl.linear_decode_window([copies[k][m][0] for m in grp], [copies[k][m][1] for m in grp],
                                        wxs[wi], ys=[ys[m] for m in grp], ws=wwss[wi], stream=stream)
        return run

    step_graphs = [capture(layer_calls(k)) for k in range(ncopies)]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(graphs, n):
        """Average ms per replay of n replays cycling through graphs, with
        events on the stream the kernels run on."""
        with torch.cuda.stream(stream):
            for i in range(min(n, len(graphs))):
                graphs[i % len(graphs)].replay()
            stream.synchronize()
            e0.record(stream)
            for i in range(n):
                graphs[i % len(graphs)].replay()
            e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    with torch.cuda.stream(stream):
        for i in range(args.warmup):
            step_graphs[i % ncopies].replay()
    torch.cuda.synchronize()
    ms_step = timed(step_graphs, args.steps)
    step_bytes = sum(algorithmic_bytes(s, T) for s in specs)
    value = step_bytes / (ms_step * 1e-3) / 1e9

    # ---- per matrix: graphs of one call on each copy, back to back
    per_matrix_us = {}
    per_matrix_gbs = {}
    for m, spec in enumerate(specs):
        def calls(m=m):
            for k in range(ncopies):
                w, c = copies[k][m]
                cl.linear_decode(w, c, xs[m], y=ys[m], ws=wss[m], stream=stream)
        g = capture(calls)
        us = timed([g], 20) * 1e3 / ncopies
        per_matrix_us[spec.name] = round(us, 3)
        per_matrix_gbs[spec.name] = round(algorithmic_bytes(spec, T) / us / 1e3, 1)
    gi = [s.name for s in specs].index("gate")
    gate_us = per_matrix_us["gate"]
    gate_bytes = algorithmic_bytes(specs[gi], T)
    achieved = gate_bytes / (gate_us * 1e-6) / 1e9

    cpu = None if args.no_cpu_baseline else cpu_baseline(specs, layer, T)

    out = {
        "metric": "achieved HBM GB/s + us/call, compensated W4A16 decode linear; prefill TFLOP/s",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u4 codes x fp16 activations, fp32 accumulate, fp16 out",
        "data": "synthetic",
        "config": {"workload": "llama8b-decoder-layer: 7 compensated linears in 4 windows (qkv|o|gate,up|down), "
                               "w4 g128, ranks %s, T=%d decode" % ("/".join(str(s.rank) for s in specs), T),
                   "tokens": T, "step_bytes": step_bytes, "rotating_copies": ncopies,
                   "per_matrix_us": per_matrix_us, "per_matrix_gbs": per_matrix_gbs},
        "roofline": {"bound": "hbm", "kernel": "cl_linear_decode on gate 14336x4096 (prepare + backbone launches)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "us_per_launch": gate_us,
                     "bytes_per_launch": gate_bytes, "traffic": None},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


def cpu_baseline(specs, layer, T):
    """The fp64 oracle on the same layer (all seven matrices, every row):
    unpack + dequantize + forward, median of 5 after one warm-up."""
    from oracle import linear, quant
    from paper_2605_05819_amd import workloads as wl
    prepared = []
    nbytes = 0
    for m, spec in enumerate(specs):
        W = wl.weight((spec.d_out, spec.d_in), layer.index, 0, m)
        Q, s, z = quant.quantize_pack(W, spec.bits, spec.group_size)
        A, B = wl.standin_factors(spec.d_out, spec.d_in, spec.r_max, layer.index, 0, m)
        x = wl.activation((T, spec.d_in), layer.index, 0, m).values
        prepared.append((Q, s, z, spec, A, B, x))
        nbytes += algorithmic_bytes(spec, T)

    def run():
        for Q, s, z, spec, A, B, x in prepared:
            linear.forward_packed(Q, s, z, spec.bits, spec.group_size, A, B, spec.rank, x)

    run()
    times = []
    for _ in range(5):
        t0 = time.perf_counter()
        run()
        times.append(time.perf_counter() - t0)
    sec = float(np.median(times))
    try:
        import threadpoolctl
        threads = max(i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()) or 1
    except Exception:
        threads = os.cpu_count()
    return {"value": round(nbytes / sec / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": "whole layer (7 matrices, all rows), T=%d, median of 5 runs of %.2f s" % (T, sec)}


if __name__ == "__main__":
    main()
