"""Benchmark: compensated W4A16 decode of a Llama-3.1-8B-shaped decoder layer.

One step = the seven compensated linears of the layer (q, k, v, o, gate, up,
down; 4-bit, group 128; per-matrix ranks from the seeded allocator under a
budget of 64 x 7) decoding one batch of tokens through the C ABI.  Weights are
seeded N(0, 0.02) draws quantized by the library on the GPU; compensation
factors are seeded fp16 stand-ins (the forward's cost does not depend on their
values).  Steps rotate over enough distinct copies of the layer (>= 1 GiB) that
every step streams its weights from HBM rather than from the 256 MB
Infinity Cache.

Prints one JSON line: whole-job algorithmic HBM throughput (GB/s), the
roofline of the dominant kernel (the gate matrix's decode launch, timed with
HIP events on the stream it runs on) and the fp64 CPU oracle timed on a
bounded sample of the same layer.
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
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--tokens", type=int, default=1)
    p.add_argument("--rotate-gib", type=float, default=1.5)
    p.add_argument("--no-cpu-baseline", action="store_true")
    return p.parse_args()


def algorithmic_bytes(spec, T):
    """HBM bytes a compensated decode must move at minimum: packed codes,
    fp16 scales and zeros, the used factor rows/columns, activations in and
    fp16 outputs out."""
    q = spec.d_out * spec.d_in * spec.bits // 8
    sz = 2 * 2 * spec.d_out * (spec.d_in // spec.group_size)
    ab = 2 * spec.rank * (spec.d_in + spec.d_out)
    return q + sz + ab + 2 * T * spec.d_in + 2 * T * spec.d_out


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: the compensated linear runs on a single device "
              "(multi-GPU sharding is described in DESIGN.md, not run).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2605_05819_amd import cl, workloads as wl

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    T = args.tokens
    layer = wl.llama_layer()
    specs = layer.linears

    # ---- build one layer on the device (library quantizer), then copies
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

    stream = torch.cuda.current_stream()

    def step(i):
        lay = copies[i % ncopies]
        for m in range(len(specs)):
            w, c = lay[m]
            cl.linear_decode(w, c, xs[m], y=ys[m], ws=wss[m], stream=stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(args.steps):
        step(i)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    step_bytes = sum(algorithmic_bytes(s, T) for s in specs)
    value = step_bytes / (ms_step * 1e-3) / 1e9

    # ---- dominant kernel: the gate matrix's decode, one launch per call,
    # timed back to back over the rotating copies on the same stream
    gi = [s.name for s in specs].index("gate")
    n_calls = max(50, args.steps)
    for i in range(10):
        w, c = copies[i % ncopies][gi]
        cl.linear_decode(w, c, xs[gi], y=ys[gi], ws=wss[gi], stream=stream)
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(n_calls):
        w, c = copies[i % ncopies][gi]
        cl.linear_decode(w, c, xs[gi], y=ys[gi], ws=wss[gi], stream=stream)
    e1.record(stream)
    torch.cuda.synchronize()
    gate_us = e0.elapsed_time(e1) * 1e3 / n_calls
    gate_bytes = algorithmic_bytes(specs[gi], T)
    achieved = gate_bytes / (gate_us * 1e-6) / 1e9

    per_matrix_us = {}
    for m, spec in enumerate(specs):
        e0.record(stream)
        for i in range(50):
            w, c = copies[i % ncopies][m]
            cl.linear_decode(w, c, xs[m], y=ys[m], ws=wss[m], stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        per_matrix_us[spec.name] = round(e0.elapsed_time(e1) * 1e3 / 50, 2)

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
        "dtype": "u4 codes, fp16 activations, fp32 accumulate",
        "data": "synthetic",
        "config": {"workload": "llama8b-decoder-layer 7 linears w4g128 ranks %s, T=%d decode" %
                   ("/".join(str(s.rank) for s in specs), T),
                   "tokens": T, "step_bytes": step_bytes, "rotating_copies": ncopies,
                   "per_matrix_us": per_matrix_us},
        "roofline": {"bound": "hbm", "kernel": "gate 14336x4096 decode call", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "us_per_launch": round(gate_us, 3), "bytes_per_launch": gate_bytes, "traffic": None},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


def cpu_baseline(specs, layer, T):
    """The fp64 oracle on a bounded sample: the first 2048 rows of each of the
    seven matrices (about a third of the layer), same inputs, median of 3."""
    from oracle import linear, quant
    from paper_2605_05819_amd import workloads as wl
    rows = 2048
    prepared = []
    nbytes = 0
    for m, spec in enumerate(specs):
        W = wl.weight((spec.d_out, spec.d_in), layer.index, 0, m)[:rows]
        Q, s, z = quant.quantize_pack(W, spec.bits, spec.group_size)
        A, B = wl.standin_factors(spec.d_out, spec.d_in, spec.r_max, layer.index, 0, m)
        x = wl.activation((T, spec.d_in), layer.index, 0, m).values
        prepared.append((Q, s, z, spec, A, B[:rows], x))
        sub = wl.LinearSpec(spec.name, min(rows, spec.d_out), spec.d_in, spec.bits, spec.group_size,
                            spec.r_max, spec.rank)
        nbytes += algorithmic_bytes(sub, T)

    def run():
        for Q, s, z, spec, A, B, x in prepared:
            linear.forward_packed(Q, s, z, spec.bits, spec.group_size, A, B, spec.rank, x)

    run()
    times = []
    for _ in range(3):
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
            "sample": "first %d rows of each of the 7 layer matrices, T=%d, median of 3 (%.2f s each)" %
                      (rows, T, sec)}


if __name__ == "__main__":
    main()
