"""Report (not a test): the relative L2 error of the library against the
fp64 oracle on the benchmark workloads, for the results table.

    python tests/report_rel_l2.py        (on an MI355X, from the repository root)

The 1024 x 1024 rank-16 linear over its whole output; the Llama-8B gate
matrix (4-, 2- and 3-bit codes) at 1, 4 and 16 tokens on 200 sampled rows;
the 2048-token prefill of 14336 x 4096 (4- and 3-bit, fp16 and bf16
activations) on 100 rows x 64 tokens.  The oracle quantizes the sampled rows
itself, as the parity tests do."""
import os, sys, json
sys.path.insert(0, os.getcwd())
import numpy as np, torch
from oracle import linear, quant
from paper_2605_05819_amd import cl, workloads as wl
from tests.helpers import dev_f16, dev_u16, out_to_numpy, rel_l2
out = {}
# the 1024 x 1024 linear: the whole output
spec = wl.single_linear().linears[0]
W = wl.weight((spec.d_out, spec.d_in), 0)
w = cl.quantize_pack(torch.from_numpy(W).cuda(), 4, 128)
Q, s, z = quant.quantize_pack(W, 4, 128)
A, B = wl.standin_factors(spec.d_out, spec.d_in, spec.r_max, 0)
c = cl.LowRank(dev_f16(A), dev_f16(B), spec.r_max, spec.rank)
x = wl.activation((1, spec.d_in), 0)
y = out_to_numpy(cl.linear_decode(w, c, dev_u16(x.bits, torch.float16), out_dtype=torch.float32))
out["linear_1024x1024_r16_T1"] = rel_l2(y, linear.forward_packed(Q, s, z, 4, 128, A, B, spec.rank, x.values))
# the gate matrix, 200 sampled rows
for tag, mk, bits, G in (("gate_w4", wl.llama_layer, 4, 128), ("gate_w2", wl.llama_layer_2bit, 2, 64),
                         ("gate_w3", wl.llama_layer_3bit, 3, 128)):
    layer = mk(); gi = [l.name for l in layer.linears].index("gate"); sp = layer.linears[gi]
    W = wl.weight((sp.d_out, sp.d_in), layer.index, 0, gi)
    w = cl.quantize_pack(torch.from_numpy(W).cuda(), bits, G)
    A, B = wl.standin_factors(sp.d_out, sp.d_in, sp.r_max, layer.index, 0, gi)
    c = cl.LowRank(dev_f16(A), dev_f16(B), sp.r_max, sp.rank)
    rows = np.random.default_rng(1).choice(sp.d_out, 200, replace=False)
    Qr, sr, zr = quant.quantize_pack(W[rows], bits, G)
    for T in (1, 4, 16):
        x = wl.activation((T, sp.d_in), layer.index, 0, gi)
        y = out_to_numpy(cl.linear_decode(w, c, dev_u16(x.bits, torch.float16), out_dtype=torch.float32))[:, rows]
        out["%s_T%d" % (tag, T)] = rel_l2(y, linear.forward_packed(Qr, sr, zr, bits, G, A, B[rows], sp.rank, x.values))
# prefill 14336 x 4096, M = 2048, sampled rows and tokens
M, N, K, r = 2048, 14336, 4096, 64
W = wl.weight((N, K), 4, 0, N)
for bits in (4, 3):
    w = cl.quantize_pack(torch.from_numpy(W).cuda(), bits, 128)
    A, B = wl.standin_factors(N, K, 64, 4, 0, N)
    c = cl.LowRank(dev_f16(A), dev_f16(B), 64, r)
    for act in ("fp16", "bf16"):
        x = wl.activation((M, K), 4, 0, N, dtype=act)
        y = out_to_numpy(cl.linear_prefill(w, c, dev_u16(x.bits, torch.float16 if act == "fp16" else torch.bfloat16),
                                           out_dtype=torch.float32))
        g = np.random.default_rng(2)
        rows = g.choice(N, 100, replace=False); toks = g.choice(M, 64, replace=False)
        Qr, sr, zr = quant.quantize_pack(W[rows], bits, 128)
        ref = linear.forward_packed(Qr, sr, zr, bits, 128, A, B[rows], r, x.values[toks])
        out["prefill_14336x4096_w%d_%s" % (bits, act)] = rel_l2(y[np.ix_(toks, rows)], ref)
print(json.dumps({k: float("%.3g" % v) for k, v in out.items()}))
