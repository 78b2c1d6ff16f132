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
Cache.  Each step is a captured HIP graph of the four window calls, so host
launch overhead is outside the timed region; the inputs are resident in HBM.

Prints one JSON line: whole-job algorithmic HBM throughput (GB/s) of the step,
the roofline of the dominant call (the gate matrix, 14336 x 4096) timed with
HIP events on the stream it runs on, the fp64 CPU oracle timed on a bounded
sample of the same layer, and (unless --no-extras) the other measured
workloads: the layer at 4 and 16 tokens, the gate,up window against the gated
call (SiLU(gate x) * (up x) fused), the 2-bit layer with its gate rank
sweep, the 3-bit layer (the paper's INT3 setting), prefill (M = 2048) in
TFLOP/s and the 48-layer MoE decode.

--copy-calibration runs only a plain 256 MiB device-to-device copy (the
reference kernel for scaling HBM traffic counters) and prints its size;
--only {decode,tokens,glu,layer2bit,layer3bit,prefill,moe} runs one workload (for
profiling): "decode" prints the line above without extras or CPU baseline,
the others print their own results.
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
MFMA_F16_PEAK_TFLOPS = 2500.0

# HBM traffic of one gate-matrix decode call (prepare + backbone), from
# rocprofv3 FETCH_SIZE and WRITE_SIZE passes over `bench.py --only decode`,
# scaled by the same counters on a plain 256 MiB device copy (FETCH_SIZE
# reads half the copied bytes: x2; WRITE_SIZE exact: x1).  Valid only for the
# kernel sources it was measured on (their SHA-256 below); null otherwise.
GATE_TRAFFIC = {"fetch_bytes": (32397 + 702) * 1024, "write_bytes": (56 + 9) * 1024,
                "sources": ("paper_2605_05819_amd/csrc/decode.hip", "paper_2605_05819_amd/csrc/gemv_common.h",
                            "paper_2605_05819_amd/csrc/cl_device.h"),
                "sha256": "76689c5865a48b68b7b4974a54f1e488aa645dd7171892eb4b680c3c3b1db176"}


def sources_sha256(paths):
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def gate_traffic():
    if GATE_TRAFFIC["sha256"] != sources_sha256(GATE_TRAFFIC["sources"]):
        return None
    return GATE_TRAFFIC["fetch_bytes"] + GATE_TRAFFIC["write_bytes"]


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=240)
    p.add_argument("--warmup", type=int, default=24)
    p.add_argument("--tokens", type=int, default=1)
    p.add_argument("--rotate-gib", type=float, default=1.5)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extras", action="store_true")
    p.add_argument("--copy-calibration", action="store_true")
    p.add_argument("--only", choices=("decode", "single", "tokens", "glu", "layer2bit", "layer3bit", "prefill",
                                       "moe", "cpu"),
                   default=None,
                   help="run one workload and print its own JSON line (for profiling)")
    return p.parse_args()


def algorithmic_bytes(spec, T, rank=None):
    """HBM bytes a compensated decode must move at minimum: packed codes,
    fp16 scales and zeros, the used rows of A and columns of B, activations in
    and fp16 outputs out."""
    r = spec.rank if rank is None else rank
    q = spec.d_out * spec.d_in * spec.bits // 8       # 3-bit: 12 bytes per 32 codes
    sz = 2 * 2 * spec.d_out * (spec.d_in // spec.group_size)
    ab = 2 * r * (spec.d_in + spec.d_out)
    return q + sz + ab + 2 * T * spec.d_in + 2 * T * spec.d_out


class Timer:
    """HIP graphs captured and replayed on one stream, timed with events
    recorded on that stream."""

    def __init__(self, torch):
        self.torch = torch
        self.stream = torch.cuda.Stream()
        self.e0 = torch.cuda.Event(enable_timing=True)
        self.e1 = torch.cuda.Event(enable_timing=True)

    def capture(self, fn):
        torch = self.torch
        with torch.cuda.stream(self.stream):
            fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=self.stream):
            fn()
        torch.cuda.synchronize()
        return g

    def spread(self, graphs, n):
        """p10 / p50 / p90 of single replays, in ms: an event after every
        replay (a separate pass, after the timed region)."""
        torch = self.torch
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
        with torch.cuda.stream(self.stream):
            evs[0].record(self.stream)
            for i in range(n):
                graphs[i % len(graphs)].replay()
                evs[i + 1].record(self.stream)
        torch.cuda.synchronize()
        d = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(n))
        return d[n // 10], d[n // 2], d[(9 * n) // 10]

    def time(self, graphs, n, warm=None):
        """Average ms per replay of n replays cycling through graphs."""
        torch = self.torch
        with torch.cuda.stream(self.stream):
            for i in range(min(n, len(graphs)) if warm is None else warm):
                graphs[i % len(graphs)].replay()
            self.stream.synchronize()
            self.e0.record(self.stream)
            for i in range(n):
                graphs[i % len(graphs)].replay()
            self.e1.record(self.stream)
        torch.cuda.synchronize()
        return self.e0.elapsed_time(self.e1) / n


def device_layer(torch, cl, wl, layer, dev, rotate_gib):
    """The layer quantized by the library, plus copies for HBM-cold steps."""
    base = []
    for m, spec in enumerate(layer.linears):
        W = torch.from_numpy(wl.weight((spec.d_out, spec.d_in), layer.index, 0, m)).to(dev)
        w = cl.quantize_pack(W, spec.bits, spec.group_size)
        del W
        A, B = wl.standin_factors(spec.d_out, spec.d_in, spec.r_max, layer.index, 0, m)
        c = cl.LowRank(torch.from_numpy(A).to(dev), torch.from_numpy(B).to(dev), spec.r_max, spec.rank)
        base.append((w, c))
    torch.cuda.synchronize()
    layer_bytes = sum(w.q.numel() * 4 + w.scales.numel() * 4 + c.A.numel() * 2 + c.B.numel() * 2 for w, c in base)
    ncopies = max(2, int(np.ceil(rotate_gib * 2 ** 30 / layer_bytes)))
    copies = [base]
    for _ in range(ncopies - 1):
        copies.append([(cl.QWeight(w.q.clone(), w.scales.clone(), w.zeros.clone(), w.d_out, w.d_in, w.bits,
                                   w.group_size), cl.LowRank(c.A.clone(), c.B.clone(), c.r_max, c.rank))
                       for w, c in base])
    return copies


WINDOWS = (("q", "k", "v"), ("o",), ("gate", "up"), ("down",))


def layer_step(torch, cl, wl, timer, copies, layer, T, dev, steps, warmup, spread=None):
    """ms per step of the layer's four windows (graph per copy), and the
    inputs/outputs used; with a dict as spread, also the p10 / p50 / p90 of
    single steps from a separate pass of as many steps."""
    specs = layer.linears
    names = [s.name for s in specs]
    windows = [[names.index(n) for n in grp] for grp in WINDOWS]
    xs, ys = [], []
    for m, spec in enumerate(specs):
        x = wl.activation((T, spec.d_in), layer.index, 0, m)
        xs.append(torch.from_numpy(x.bits.view(np.int16)).view(torch.float16).to(dev))
        ys.append(torch.empty((T, spec.d_out), dtype=torch.float16, device=dev))
    base = copies[0]
    wxs = [xs[grp[0]] for grp in windows]
    wwss = [cl.workspace(cl.window_workspace([base[m][0] for m in grp], [base[m][1] for m in grp], T), dev)
            for grp in windows]

    def calls(k):
        def run():
            for wi, grp in enumerate(windows):
                cl.linear_decode_window([copies[k][m][0] for m in grp], [copies[k][m][1] for m in grp],
                                        wxs[wi], ys=[ys[m] for m in grp], ws=wwss[wi], stream=timer.stream)
        return run

    graphs = [timer.capture(calls(k)) for k in range(len(copies))]
    ms = timer.time(graphs, steps, warm=warmup)
    if spread is not None:
        spread["p10"], spread["p50"], spread["p90"] = (round(v, 5) for v in timer.spread(graphs, steps))
    return ms, xs, ys


def per_matrix(torch, cl, timer, copies, specs, xs, ys, T, dev, rank=None, m_only=None):
    """us per single-linear call of each matrix (graph of one call per copy)."""
    out = {}
    for m, spec in enumerate(specs):
        if m_only is not None and m != m_only:
            continue
        cs = []
        for k in range(len(copies)):
            w, c = copies[k][m]
            cs.append((w, c if rank is None else cl.LowRank(c.A, c.B, c.r_max, rank)))
        ws = cl.workspace(cl.linear_workspace(cs[0][0], cs[0][1], T), dev)

        def run():
            for w, c in cs:
                cl.linear_decode(w, c, xs[m], y=ys[m], ws=ws, stream=timer.stream)
        g = timer.capture(run)
        out[spec.name] = timer.time([g], 20) * 1e3 / len(cs)
    return out


def bench_tokens(torch, cl, wl, timer, copies, layer, dev):
    """The layer step at 4 and 16 decode tokens."""
    res = {}
    for T in (4, 16):
        ms, _, _ = layer_step(torch, cl, wl, timer, copies, layer, T, dev, 200, 24)
        b = sum(algorithmic_bytes(s, T) for s in layer.linears)
        res["layer_T%d" % T] = {"ms_per_step": round(ms, 5), "gbs": round(b / (ms * 1e-3) / 1e9, 1)}
    return res


def bench_glu(torch, cl, wl, timer, copies, layer, dev):
    """The gate,up window alone, the window followed by torch's SiLU and
    product (the unfused gated MLP input), and the gated call (SiLU(gate x) *
    (up x) in the backbone launch) at 1 and 16 tokens: us per call over the
    copies."""
    names = [s.name for s in layer.linears]
    gi, ui = names.index("gate"), names.index("up")
    d_in, d_out = layer.linears[gi].d_in, layer.linears[gi].d_out
    res = {}
    for T in (1, 16):
        x = torch.from_numpy(wl.activation((T, d_in), layer.index, 0, gi).bits.view(np.int16)).view(
            torch.float16).to(dev)
        yg, yu, h = (torch.empty((T, d_out), dtype=torch.float16, device=dev) for _ in range(3))
        pairs = [([k[gi][0], k[ui][0]], [k[gi][1], k[ui][1]]) for k in copies]
        ws = cl.workspace(cl.window_workspace(*pairs[0], T), dev)

        def win():
            for w2, c2 in pairs:
                cl.linear_decode_window(w2, c2, x, ys=[yg, yu], ws=ws, stream=timer.stream)

        def win_then_torch():
            for w2, c2 in pairs:
                cl.linear_decode_window(w2, c2, x, ys=[yg, yu], ws=ws, stream=timer.stream)
                torch.mul(torch.nn.functional.silu(yg), yu, out=h)

        def glu():
            for w2, c2 in pairs:
                cl.linear_decode_glu(w2, c2, x, h=h, ws=ws, stream=timer.stream)
        gw, gt, gg = timer.capture(win), timer.capture(win_then_torch), timer.capture(glu)
        res["T%d" % T] = {"window_us": round(timer.time([gw], 20) * 1e3 / len(pairs), 3),
                          "window_then_torch_silu_mul_us": round(timer.time([gt], 20) * 1e3 / len(pairs), 3),
                          "glu_us": round(timer.time([gg], 20) * 1e3 / len(pairs), 3)}
    return res


def bench_layer2bit(torch, cl, wl, timer, dev, rotate_gib):
    """The 2-bit group-64 layer (ranks up to 256 under 128 x 7) at one token,
    the rank sweep r in {0, 32, 128, 256} on its 14336 x 4096 gate, and the
    layer at 4 and 16 tokens (MFMA backbone)."""
    layer2 = wl.llama_layer_2bit()
    copies2 = device_layer(torch, cl, wl, layer2, dev, rotate_gib)
    ms2, xs2, ys2 = layer_step(torch, cl, wl, timer, copies2, layer2, 1, dev, 80, 8)
    b2 = sum(algorithmic_bytes(s, 1) for s in layer2.linears)
    sweep = {}
    g2 = [s.name for s in layer2.linears].index("gate")
    for r in (0, 32, 128, 256):
        u = per_matrix(torch, cl, timer, copies2, layer2.linears, xs2, ys2, 1, dev, rank=r, m_only=g2)["gate"]
        sweep["r%d" % r] = {"us": round(u, 3), "gbs": round(algorithmic_bytes(layer2.linears[g2], 1, r) / u / 1e3, 1)}
    many = {}
    for T in (4, 16):
        msT, _, _ = layer_step(torch, cl, wl, timer, copies2, layer2, T, dev, 80, 8)
        bT = sum(algorithmic_bytes(s, T) for s in layer2.linears)
        many["T%d" % T] = {"ms_per_step": round(msT, 5), "gbs": round(bT / (msT * 1e-3) / 1e9, 1)}
    return {"ms_per_step": round(ms2, 5), "gbs": round(b2 / (ms2 * 1e-3) / 1e9, 1),
            "ranks": "/".join(str(s.rank) for s in layer2.linears), "gate_rank_sweep": sweep, **many}


def bench_single(torch, cl, wl, timer, dev, rotate_gib):
    """The 1024 x 1024 linear (4-bit g128, rank 16, one token): us per call
    over enough copies to exceed the Infinity Cache, one graph of every
    copy's call replayed."""
    spec = wl.single_linear().linears[0]
    W = torch.from_numpy(wl.weight((spec.d_out, spec.d_in), 0)).to(dev)
    w = cl.quantize_pack(W, spec.bits, spec.group_size)
    A, B = wl.standin_factors(spec.d_out, spec.d_in, spec.r_max, 0)
    c = cl.LowRank(torch.from_numpy(A).to(dev), torch.from_numpy(B).to(dev), spec.r_max, spec.rank)
    per = w.q.numel() * 4 + w.scales.numel() * 4 + c.A.numel() * 2 + c.B.numel() * 2
    n = max(2, int(np.ceil(rotate_gib * 2 ** 30 / per)))
    copies = [(w, c)] + [(cl.QWeight(w.q.clone(), w.scales.clone(), w.zeros.clone(), w.d_out, w.d_in, w.bits,
                                      w.group_size), cl.LowRank(c.A.clone(), c.B.clone(), c.r_max, c.rank))
                         for _ in range(n - 1)]
    x = torch.from_numpy(wl.activation((1, spec.d_in), 0).bits.view(np.int16)).view(torch.float16).to(dev)
    y = torch.empty((1, spec.d_out), dtype=torch.float16, device=dev)
    ws = cl.workspace(cl.linear_workspace(w, c, 1), dev)

    def run():
        for wk, ck in copies:
            cl.linear_decode(wk, ck, x, y=y, ws=ws, stream=timer.stream)
    g = timer.capture(run)
    us = timer.time([g], 5) * 1e3 / n
    nbytes = algorithmic_bytes(spec, 1)
    return {"us_per_call": round(us, 3), "gbs": round(nbytes / us / 1e3, 1), "bytes_per_call": nbytes,
            "copies": n}


def bench_layer3bit(torch, cl, wl, timer, dev, rotate_gib):
    """The 3-bit group-128 layer (the paper's INT3 dense setting; ranks
    from {0, 16, 32, 64, 128} under 64 x 7) at 1, 4 and 16 tokens (dot2
    backbone at one token, MFMA from three)."""
    layer3 = wl.llama_layer_3bit()
    copies3 = device_layer(torch, cl, wl, layer3, dev, rotate_gib)
    res = {"ranks": "/".join(str(s.rank) for s in layer3.linears)}
    for T in (1, 4, 16):
        ms3, xs3, ys3 = layer_step(torch, cl, wl, timer, copies3, layer3, T, dev, 80, 8)
        b3 = sum(algorithmic_bytes(s, T) for s in layer3.linears)
        res["T%d" % T] = {"ms_per_step": round(ms3, 5), "gbs": round(b3 / (ms3 * 1e-3) / 1e9, 1),
                          "step_bytes": b3}
        if T == 1:
            g3 = [s.name for s in layer3.linears].index("gate")
            u = per_matrix(torch, cl, timer, copies3, layer3.linears, xs3, ys3, 1, dev, m_only=g3)["gate"]
            res["gate_T1"] = {"us": round(u, 3), "gbs": round(algorithmic_bytes(layer3.linears[g3], 1) / u / 1e3, 1)}
    return res


def bench_prefill(torch, cl, wl, timer, dev):
    """M = 2048 tokens through 4096 x 4096 and 14336 x 4096, rank 64, 4-bit
    codes with fp16 and bf16 activations, and 3-bit codes (the paper's INT3
    setting) with fp16 activations through 14336 x 4096: us per call and
    TFLOP/s (2MNK + 2Mr(K + N)); and, for scale, torch's fp16 matrix
    product of the same shape (2MNK)."""
    M, r = 2048, 64
    res = {}
    for (N, K, bits) in ((4096, 4096, 4), (14336, 4096, 4), (14336, 4096, 3)):
        W = torch.from_numpy(wl.weight((N, K), 3, 0, N)).to(dev)
        w = cl.quantize_pack(W, bits, 128)
        del W
        A, B = wl.standin_factors(N, K, r, 3, 0, N)
        c = cl.LowRank(torch.from_numpy(A).to(dev), torch.from_numpy(B).to(dev), r, r)
        for act in (("fp16", "bf16") if bits == 4 else ("fp16",)):
            x = wl.activation((M, K), 3, 0, N, dtype=act)
            dt = torch.float16 if act == "fp16" else torch.bfloat16
            X = torch.from_numpy(x.bits.view(np.int16)).view(dt).to(dev)
            Y = torch.empty((M, N), dtype=torch.float16, device=dev)
            need = cl.prefill_workspace(w, c, M)
            ws = cl.workspace(need, dev) if need else None
            g = timer.capture(lambda: cl.linear_prefill(w, c, X, Y=Y, ws=ws, stream=timer.stream))
            us = timer.time([g], 30) * 1e3
            flops = 2.0 * M * N * K + 2.0 * M * r * (K + N)
            key = "%dx%d_%s" % (N, K, act) if bits == 4 else "%dx%d_w3_%s" % (N, K, act)
            res[key] = {"us": round(us, 2), "tflops": round(flops / us / 1e6, 1)}
        if bits != 4:
            continue
        # reference: the bare fp16 contraction through torch (hipBLASLt) on
        # the same shape, no dequantization and no rank term
        Xr = torch.randn((M, K), dtype=torch.float16, device=dev)
        Wt = torch.randn((K, N), dtype=torch.float16, device=dev)
        Yr = torch.empty((M, N), dtype=torch.float16, device=dev)
        g = timer.capture(lambda: torch.mm(Xr, Wt, out=Yr))
        us = timer.time([g], 30) * 1e3
        res["%dx%d_torch_mm_fp16_reference" % (N, K)] = {"us": round(us, 2),
                                                         "tflops": round(2.0 * M * N * K / us / 1e6, 1)}
        del Xr, Wt, Yr
    return res


def bench_moe(torch, cl, wl, timer, dev):
    """48 stacked MoE layers (128 experts, gate/up 768 x 2048, down
    2048 x 768, 4-bit g128, per-expert ranks from {0, 8, 16, 32}), top-8
    routing: per layer gate and up as one window on the token's input, down
    on each slot's input; and the same layers chained as in a model (down on
    SiLU(gate) * up of the window's outputs, formed by the gated down call).  Codes, scales and factors of the stacked experts are seeded random
    device data (the cost does not depend on the values).  GB/s counts only the
    routed experts' bytes."""
    L, E, K = wl.MOE_LAYERS, wl.MOE_EXPERTS, wl.MOE_TOPK
    gen = torch.Generator(device=dev)
    gen.manual_seed(5)
    mats = (("gate", 0), ("up", 1), ("down", 2))
    layers = {}
    for name, m in mats:
        d_out, d_in = wl.MOE_SHAPES[name]
        lst = []
        for l in range(L):
            q = torch.randint(-2 ** 31, 2 ** 31 - 1, (E, d_out, d_in // 8), dtype=torch.int32, device=dev,
                              generator=gen)
            s = (torch.rand((E, d_out, d_in // 128), device=dev, generator=gen) * 0.004 + 0.005).half()
            z = torch.randint(0, 16, (E, d_out, d_in // 128), device=dev, generator=gen).half()
            A = (torch.randn((E, 32, d_in), device=dev, generator=gen) * 0.05).half()
            B = (torch.randn((E, d_out, 32), device=dev, generator=gen) * 0.05).half()
            ranks = torch.from_numpy(wl.moe_expert_ranks(5, l, m)).to(dev)
            lst.append(cl.MoeExperts(q, s, z, A, B, ranks, E, d_out, d_in, 4, 128, 32))
        layers[name] = lst
    res = {}
    for T in (1, 8, 64):
        ids = [torch.from_numpy(wl.routing(T, 5, l)[0]).to(dev) for l in range(L)]
        xs = {n: torch.from_numpy(wl.activation((T, K, wl.MOE_SHAPES[n][1]) if n == "down"
                                                else (T, wl.MOE_SHAPES[n][1]), 5, 0, m).bits.view(np.int16))
              .view(torch.float16).to(dev) for n, m in mats}
        ys = {n: torch.empty((T, K, wl.MOE_SHAPES[n][0]), dtype=torch.float16, device=dev) for n, _ in mats}
        ws_gu = cl.workspace(cl.moe_window_workspace([layers["gate"][0], layers["up"][0]], T, K, False), dev)
        ws_dn = cl.workspace(cl.moe_workspace(layers["down"][0], T, K, True), dev)
        ws_gd = cl.workspace(cl.moe_gated_workspace(layers["down"][0], T, K), dev)

        def run():
            # gate and up share the token's input and routing: one window
            for l in range(L):
                cl.moe_linear_decode_window([layers["gate"][l], layers["up"][l]], xs["gate"], ids[l],
                                            ys=[ys["gate"], ys["up"]], ws=ws_gu, stream=timer.stream)
                cl.moe_linear_decode(layers["down"][l], xs["down"], ids[l], y=ys["down"], ws=ws_dn,
                                     stream=timer.stream)
        def chain():
            # the FFN as it runs in a model: the gate/up window's outputs feed
            # the down call, which forms SiLU(gate) * up as it reads them
            for l in range(L):
                cl.moe_linear_decode_window([layers["gate"][l], layers["up"][l]], xs["gate"], ids[l],
                                            ys=[ys["gate"], ys["up"]], ws=ws_gu, stream=timer.stream)
                cl.moe_linear_decode_gated(layers["down"][l], ys["gate"], ys["up"], ids[l], y=ys["down"], ws=ws_gd,
                                           stream=timer.stream)
        g = timer.capture(run)
        us = timer.time([g], 10) * 1e3
        us_chain = timer.time([timer.capture(chain)], 10) * 1e3
        nbytes = 0
        for l in range(L):
            routed = np.unique(ids[l].cpu().numpy())
            for n, _ in mats:
                d_out, d_in = wl.MOE_SHAPES[n]
                rk = layers[n][l].ranks.cpu().numpy()
                for e in routed:
                    nbytes += d_out * d_in // 2 + 4 * d_out * (d_in // 128) + 2 * int(rk[e]) * (d_in + d_out)
                nbytes += 2 * xs[n].numel() + 2 * ys[n].numel()
        res["T%d" % T] = {"us_per_layer": round(us / L, 2), "gbs": round(nbytes / us / 1e3, 1),
                          "bytes_per_layer": nbytes // L, "gated_chain_us_per_layer": round(us_chain / L, 2)}
    return res


def copy_calibration(torch, dev):
    n = 64 << 20                                   # 256 MiB of fp32
    a = torch.ones(n, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": 4 * n, "copy_calibration_bytes_written": 4 * n,
                      "calls": 5}))


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: the compensated linear runs on a single device; "
              "multi-GPU sharding is described in DESIGN.md and not run.", file=sys.stderr)
        sys.exit(2)

    if args.only == "cpu":                          # the oracle baselines alone (no GPU)
        print(json.dumps({"cpu_oracle": cpu_oracle_workloads()}))
        return

    import torch
    from paper_2605_05819_amd import cl, workloads as wl

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        copy_calibration(torch, dev)
        return
    timer = Timer(torch)
    T = args.tokens
    layer = wl.llama_layer()
    specs = layer.linears
    only = args.only
    if only in ("prefill", "moe"):
        fn = bench_prefill if only == "prefill" else bench_moe
        print(json.dumps({only: fn(torch, cl, wl, timer, dev)}))
        return
    if only == "layer2bit":
        print(json.dumps({"layer_2bit_g64_T1": bench_layer2bit(torch, cl, wl, timer, dev, args.rotate_gib)}))
        return
    if only == "layer3bit":
        print(json.dumps({"layer_3bit_g128": bench_layer3bit(torch, cl, wl, timer, dev, args.rotate_gib)}))
        return
    if only == "single":
        print(json.dumps({"single_1024x1024_r16": bench_single(torch, cl, wl, timer, dev, args.rotate_gib)}))
        return

    copies = device_layer(torch, cl, wl, layer, dev, args.rotate_gib)
    ncopies = len(copies)
    if only == "tokens":
        print(json.dumps(bench_tokens(torch, cl, wl, timer, copies, layer, dev)))
        return
    if only == "glu":
        print(json.dumps({"gate_up_window_vs_glu": bench_glu(torch, cl, wl, timer, copies, layer, dev)}))
        return

    step_spread = {}
    ms_step, xs, ys = layer_step(torch, cl, wl, timer, copies, layer, T, dev, args.steps, args.warmup,
                                 spread=step_spread)
    step_bytes = sum(algorithmic_bytes(s, T) for s in specs)
    value = step_bytes / (ms_step * 1e-3) / 1e9

    us = per_matrix(torch, cl, timer, copies, specs, xs, ys, T, dev)
    per_matrix_us = {k: round(v, 3) for k, v in us.items()}
    per_matrix_gbs = {s.name: round(algorithmic_bytes(s, T) / us[s.name] / 1e3, 1) for s in specs}
    gi = [s.name for s in specs].index("gate")
    gate_us = us["gate"]
    gate_bytes = algorithmic_bytes(specs[gi], T)
    achieved = gate_bytes / (gate_us * 1e-6) / 1e9

    extras = None
    if only is None and not args.no_extras:
        extras = {"single_1024x1024_r16": bench_single(torch, cl, wl, timer, dev, args.rotate_gib)}
        extras.update(bench_tokens(torch, cl, wl, timer, copies, layer, dev))
        extras["gate_up_window_vs_glu"] = bench_glu(torch, cl, wl, timer, copies, layer, dev)
        del copies
        torch.cuda.empty_cache()
        extras["layer_2bit_g64_T1"] = bench_layer2bit(torch, cl, wl, timer, dev, args.rotate_gib)
        torch.cuda.empty_cache()
        extras["layer_3bit_g128"] = bench_layer3bit(torch, cl, wl, timer, dev, args.rotate_gib)
        torch.cuda.empty_cache()
        extras["prefill_M2048_r64"] = bench_prefill(torch, cl, wl, timer, dev)
        extras["moe_48_layers"] = bench_moe(torch, cl, wl, timer, dev)

    cpu = None if (args.no_cpu_baseline or only) else cpu_baseline(layer, T)
    if extras is not None and not args.no_cpu_baseline:
        extras["cpu_oracle"] = cpu_oracle_workloads()

    out = {
        "metric": "achieved HBM GB/s + us/call, compensated W4A16 decode linear; prefill TFLOP/s",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "step_ms_spread": dict(step_spread, note="single steps of a separate pass after the timed region, an "
                                                 "event after each (each event lengthens its step: compare "
                                                 "the spread's width, not its level, with ms_per_step)"),
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
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "us_per_launch": round(gate_us, 3),
                     "bytes_per_launch": gate_bytes, "traffic": gate_traffic()},
        "cpu_baseline": cpu,
    }
    if extras is not None:
        pf = extras["prefill_M2048_r64"]["14336x4096_fp16"]
        extras["prefill_roofline"] = {"bound": "mfma", "kernel": "cl_linear_prefill 14336x4096 M=2048 r=64 fp16",
                                      "achieved": pf["tflops"], "peak": MFMA_F16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                      "frac": round(pf["tflops"] / MFMA_F16_PEAK_TFLOPS, 4)}
        out["extras"] = extras
    print(json.dumps(out))


def cpu_baseline(layer, T):
    """The fp64 oracle (unpack + dequantize + forward) on the whole layer
    (all seven matrices, every row): median of 3 runs after one warm-up."""
    from oracle import linear, quant
    from paper_2605_05819_amd import workloads as wl
    prepared = []
    nbytes = 0
    for m, spec in enumerate(layer.linears):
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
    for _ in range(3):
        t0 = time.perf_counter()
        run()
        times.append(time.perf_counter() - t0)
    sec = float(np.median(times))
    threads, ncpu = host_threads()
    return {"value": round(nbytes / sec / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "cpu_count": ncpu,
            "sample": "whole layer (7 matrices, all rows, %d bytes), T=%d, median of 3 runs of %.2f s; "
                      "numpy elementwise steps on one thread, BLAS products on %d threads of %d host CPUs"
                      % (nbytes, T, sec, threads, ncpu)}


def host_threads():
    """(BLAS threads the oracle's matrix products use, os.cpu_count())."""
    try:
        import threadpoolctl
        threads = max(i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()) or 1
    except Exception:
        threads = os.cpu_count()
    return threads, os.cpu_count()


def _median_time(fn, reps, warm=True):
    if warm:
        fn()
    ts = []
    for _ in range(reps):
        t0 = time.perf_counter()
        fn()
        ts.append(time.perf_counter() - t0)
    return float(np.median(ts))


def cpu_oracle_workloads():
    """The fp64 oracle (unpack + dequantize + forward, as it stands) timed on
    bounded samples of the other workloads, in each workload's unit: the
    1024 x 1024 linear (median of 5), the 2-bit gate rank sweep (one run per
    rank, one warm-up run before the first), prefill on a 256-token sample of
    the 2048 tokens (TFLOP/s; the cost is linear in tokens) and the
    128-expert MoE gate and down at 1 and 8 tokens (routed bytes / time; one
    warm-up run at 1 token)."""
    from oracle import linear, moe, quant
    from paper_2605_05819_amd import workloads as wl
    threads, ncpu = host_threads()
    out = {"cores": threads, "cpu_count": ncpu}
    # 1024 x 1024, rank 16, one token
    spec = wl.single_linear().linears[0]
    W = wl.weight((spec.d_out, spec.d_in), 0)
    Q, s, z = quant.quantize_pack(W, 4, 128)
    A, B = wl.standin_factors(spec.d_out, spec.d_in, spec.r_max, 0)
    x = wl.activation((1, spec.d_in), 0).values
    sec = _median_time(lambda: linear.forward_packed(Q, s, z, 4, 128, A, B, spec.rank, x), 5)
    out["single_1024x1024_r16"] = {"us_per_call": round(sec * 1e6, 1),
                                   "gbs": round(algorithmic_bytes(spec, 1) / sec / 1e9, 4)}
    # 2-bit gate, rank sweep
    layer2 = wl.llama_layer_2bit()
    g2 = [l.name for l in layer2.linears].index("gate")
    sp2 = layer2.linears[g2]
    W = wl.weight((sp2.d_out, sp2.d_in), layer2.index, 0, g2)
    Q, s, z = quant.quantize_pack(W, 2, 64)
    A, B = wl.standin_factors(sp2.d_out, sp2.d_in, 256, layer2.index, 0, g2)
    x = wl.activation((1, sp2.d_in), layer2.index, 0, g2).values
    sweep = {}
    for r in (0, 32, 128, 256):
        sec = _median_time(lambda: linear.forward_packed(Q, s, z, 2, 64, A, B, r, x), 1, warm=r == 0)
        sweep["r%d" % r] = {"s": round(sec, 3), "gbs": round(algorithmic_bytes(sp2, 1, r) / sec / 1e9, 4)}
    out["gate_2bit_rank_sweep"] = sweep
    # prefill, 256 of the 2048 tokens, rank 64
    Ms, r = 256, 64
    pf = {}
    for (N, K) in ((4096, 4096), (14336, 4096)):
        W = wl.weight((N, K), 3, 0, N)
        Q, s, z = quant.quantize_pack(W, 4, 128)
        A, B = wl.standin_factors(N, K, r, 3, 0, N)
        X = wl.activation((Ms, K), 3, 0, N).values
        sec = _median_time(lambda: linear.forward_packed(Q, s, z, 4, 128, A, B, r, X), 1)
        flops = 2.0 * Ms * N * K + 2.0 * Ms * r * (K + N)
        pf["%dx%d" % (N, K)] = {"s": round(sec, 3), "tflops": round(flops / sec / 1e12, 5)}
    out["prefill_sample_M256_r64"] = pf
    # MoE: 128 stand-in experts of gate (shared input) and down (per-slot input)
    E, k = wl.MOE_EXPERTS, wl.MOE_TOPK
    mo = {}
    for name, m in (("gate", 0), ("down", 2)):
        d_out, d_in = wl.MOE_SHAPES[name]
        Qe, se, ze = wl.standin_codes(E, d_out, d_in, 4, 128, 5, 0, m)
        ranks = wl.moe_expert_ranks(5, 0, m)
        packed = []
        for e in range(E):
            Ae, Be = wl.standin_factors(d_out, d_in, 32, 5, 0, m, e)
            packed.append((Qe[e], se[e], ze[e], Ae, Be))
        rows = np.arange(d_out)
        for T in (1, 8):
            ids, _ = wl.routing(T, 5, 0)
            X = wl.activation((T, k, d_in) if name == "down" else (T, d_in), 5, 0, m).values
            sec = _median_time(lambda: moe.forward_rows(packed, ranks, X, ids, name == "down", rows, 4, 128), 1,
                               warm=T == 1)
            nbytes = sum(d_out * d_in // 2 + 4 * d_out * (d_in // 128) + 2 * int(ranks[e]) * (d_in + d_out)
                         for e in np.unique(ids)) + 2 * X.size + 2 * T * k * d_out
            mo["%s_T%d" % (name, T)] = {"s": round(sec, 3), "gbs": round(nbytes / sec / 1e9, 4)}
    out["moe_layer_sample"] = mo
    return out


if __name__ == "__main__":
    main()
