"""Thin Python binding of ``libcl.so`` (the C ABI declared in ``include/cl.h``).

Argument marshalling only: every step of the layer runs in the HIP kernels of
the library.  PyTorch provides device memory and the current stream.  If the
library has not been built, :func:`lib` raises -- there is no fallback path.
"""

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcl.so")

CL_OK, CL_EINVAL, CL_EUNSUPPORTED, CL_EWORKSPACE, CL_EHIP = range(5)
CL_FP16, CL_BF16, CL_FP32 = 1, 2, 3
STATUS_NAMES = {0: "CL_OK", 1: "CL_EINVAL", 2: "CL_EUNSUPPORTED", 3: "CL_EWORKSPACE", 4: "CL_EHIP"}

_DTYPE_CODE = {torch.float16: CL_FP16, torch.bfloat16: CL_BF16, torch.float32: CL_FP32}


class ClError(RuntimeError):
    def __init__(self, status, message):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), message))
        self.status = status


class QWeightC(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("scales", ctypes.c_void_p), ("zeros", ctypes.c_void_p),
                ("d_out", ctypes.c_int32), ("d_in", ctypes.c_int32), ("bits", ctypes.c_int32),
                ("group_size", ctypes.c_int32)]


class LowRankC(ctypes.Structure):
    _fields_ = [("A", ctypes.c_void_p), ("B", ctypes.c_void_p), ("r_max", ctypes.c_int32),
                ("rank", ctypes.c_int32)]


_lib = None

_SIGNATURES = {
    "cl_last_error": (ctypes.c_char_p, []),
    "cl_quantize_pack": (ctypes.c_int32, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                          ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_void_p]),
    "cl_dequantize": (ctypes.c_int32, [ctypes.POINTER(QWeightC), ctypes.c_void_p, ctypes.c_void_p]),
    "cl_linear_workspace": (ctypes.c_size_t, [ctypes.POINTER(QWeightC), ctypes.POINTER(LowRankC), ctypes.c_int32]),
    "cl_linear_decode": (ctypes.c_int32, [ctypes.POINTER(QWeightC), ctypes.POINTER(LowRankC), ctypes.c_void_p,
                                          ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                          ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "cl_prefill_workspace": (ctypes.c_size_t, [ctypes.POINTER(QWeightC), ctypes.POINTER(LowRankC), ctypes.c_int32]),
    "cl_linear_prefill": (ctypes.c_int32, [ctypes.POINTER(QWeightC), ctypes.POINTER(LowRankC), ctypes.c_void_p,
                                           ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                           ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "cl_build_compensation_workspace": (ctypes.c_size_t, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]),
    "cl_build_compensation": (ctypes.c_int32, [ctypes.c_void_p, ctypes.POINTER(QWeightC), ctypes.c_int32,
                                               ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                               ctypes.c_size_t, ctypes.c_void_p]),
    "cl_moe_workspace": (ctypes.c_size_t, [ctypes.POINTER(QWeightC), ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                            ctypes.c_int32, ctypes.c_int32]),
    "cl_moe_linear_decode": (ctypes.c_int32, [ctypes.POINTER(QWeightC), ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                              ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                              ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                              ctypes.c_size_t, ctypes.c_void_p]),
    "cl_moe_window_workspace": (ctypes.c_size_t, [ctypes.c_int32, ctypes.POINTER(QWeightC), ctypes.c_void_p,
                                                  ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]),
    "cl_moe_linear_decode_window": (ctypes.c_int32, [ctypes.c_int32, ctypes.POINTER(QWeightC), ctypes.c_void_p,
                                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                                     ctypes.c_int32,
                                                     ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                                     ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                                     ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "cl_linear_window_workspace": (ctypes.c_size_t, [ctypes.c_int32, ctypes.POINTER(QWeightC),
                                                     ctypes.POINTER(LowRankC), ctypes.c_int32]),
    "cl_linear_decode_window": (ctypes.c_int32, [ctypes.c_int32, ctypes.POINTER(QWeightC), ctypes.POINTER(LowRankC),
                                                 ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                                 ctypes.POINTER(ctypes.c_void_p), ctypes.c_int32, ctypes.c_void_p,
                                                 ctypes.c_size_t, ctypes.c_void_p]),
    "cl_allocate_ranks": (ctypes.c_int32, [ctypes.c_int32, ctypes.POINTER(ctypes.c_void_p),
                                           ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_double),
                                           ctypes.c_double, ctypes.c_double, ctypes.POINTER(ctypes.c_int32),
                                           ctypes.c_int32, ctypes.c_int32, ctypes.c_double,
                                           ctypes.POINTER(ctypes.c_int32)]),
    "cl_layer_sensitivity": (ctypes.c_int32, [ctypes.c_int32, ctypes.POINTER(ctypes.c_double), ctypes.c_int32,
                                              ctypes.POINTER(ctypes.c_double)]),
    "cl_linear_decode_glu": (ctypes.c_int32, [ctypes.POINTER(QWeightC), ctypes.POINTER(LowRankC), ctypes.c_void_p,
                                              ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                              ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
}


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libcl.so is not built; run `python -m paper_2605_05819_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype, fn.argtypes = res, args
        _lib = handle
    return _lib


def _check(status):
    if status != CL_OK:
        raise ClError(status, lib().cl_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


@dataclass
class QWeight:
    """A packed backbone on the device: q uint32-as-int32 [d_out][d_in*bits/32],
    scales/zeros fp16 [d_out][d_in/group_size]."""
    q: torch.Tensor
    scales: torch.Tensor
    zeros: torch.Tensor
    d_out: int
    d_in: int
    bits: int
    group_size: int

    def c(self):
        return QWeightC(self.q.data_ptr(), self.scales.data_ptr(), self.zeros.data_ptr(),
                        self.d_out, self.d_in, self.bits, self.group_size)


@dataclass
class LowRank:
    """Compensation factors on the device: A fp16 [r_max][d_in], B fp16
    [d_out][r_max]; ``rank`` leading factors are applied."""
    A: Optional[torch.Tensor]
    B: Optional[torch.Tensor]
    r_max: int
    rank: int

    def c(self):
        return LowRankC(0 if self.A is None else self.A.data_ptr(),
                        0 if self.B is None else self.B.data_ptr(), self.r_max, self.rank)


def quantize_pack(W, bits, group_size, stream=None):
    """``cl_quantize_pack`` on a float32 device tensor; returns a QWeight."""
    d_out, d_in = W.shape
    dev = W.device
    q = torch.empty((d_out, d_in * bits // 32), dtype=torch.int32, device=dev)
    s = torch.empty((d_out, d_in // group_size), dtype=torch.float16, device=dev)
    z = torch.empty_like(s)
    _check(lib().cl_quantize_pack(_ptr(W), d_out, d_in, bits, group_size, _ptr(q), _ptr(s), _ptr(z),
                                  _stream(stream)))
    return QWeight(q, s, z, d_out, d_in, bits, group_size)


def dequantize(w, stream=None):
    out = torch.empty((w.d_out, w.d_in), dtype=torch.float32, device=w.q.device)
    qc = w.c()
    _check(lib().cl_dequantize(ctypes.byref(qc), _ptr(out), _stream(stream)))
    return out


def linear_workspace(w, c, tokens):
    qc = w.c()
    lc = c.c() if c is not None else None
    return lib().cl_linear_workspace(ctypes.byref(qc), ctypes.byref(lc) if lc else None, tokens)


def workspace(nbytes, device):
    """A device workspace of at least ``nbytes`` (torch allocations are
    256-byte aligned)."""
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def linear_decode(w, c, x, out_dtype=torch.float16, y=None, ws=None, stream=None):
    """``cl_linear_decode``: x [T][d_in] fp16/bf16 -> y [T][d_out] of out_dtype."""
    T = x.shape[0]
    if y is None:
        y = torch.empty((T, w.d_out), dtype=out_dtype, device=x.device)
    if ws is None:
        ws = workspace(linear_workspace(w, c, T), x.device)
    qc = w.c()
    lc = c.c() if c is not None else None
    _check(lib().cl_linear_decode(ctypes.byref(qc), ctypes.byref(lc) if lc else None, _ptr(x), T,
                                  _DTYPE_CODE[x.dtype], _ptr(y), _DTYPE_CODE[y.dtype], _ptr(ws),
                                  0 if ws is None else ws.numel(), _stream(stream)))
    return y


def _window_structs(ws_, cs):
    n = len(ws_)
    qa = (QWeightC * n)(*[w.c() for w in ws_])
    la = None
    if cs is not None and any(c is not None for c in cs):
        la = (LowRankC * n)(*[(c.c() if c is not None else LowRankC(0, 0, 0, 0)) for c in cs])
    return qa, la


def window_workspace(ws_, cs, tokens):
    qa, la = _window_structs(ws_, cs)
    return lib().cl_linear_window_workspace(len(ws_), qa, la, tokens)


def linear_decode_window(ws_, cs, x, out_dtype=torch.float16, ys=None, ws=None, stream=None):
    """``cl_linear_decode_window``: n linears sharing x [T][d_in]; returns the
    list of outputs y_i [T][d_out_i]."""
    T = x.shape[0]
    n = len(ws_)
    if ys is None:
        ys = [torch.empty((T, w.d_out), dtype=out_dtype, device=x.device) for w in ws_]
    qa, la = _window_structs(ws_, cs)
    if ws is None:
        ws = workspace(lib().cl_linear_window_workspace(n, qa, la, T), x.device)
    yp = (ctypes.c_void_p * n)(*[y.data_ptr() for y in ys])
    _check(lib().cl_linear_decode_window(n, qa, la, _ptr(x), T, _DTYPE_CODE[x.dtype], yp,
                                         _DTYPE_CODE[ys[0].dtype], _ptr(ws), ws.numel(), _stream(stream)))
    return ys


def linear_decode_glu(gate_up, cs, x, out_dtype=torch.float16, h=None, ws=None, stream=None):
    """``cl_linear_decode_glu``: h = SiLU(gate x) * (up x) [T][d_out] for
    gate_up = (gate, up) and their factors cs (or None)."""
    T = x.shape[0]
    if h is None:
        h = torch.empty((T, gate_up[0].d_out), dtype=out_dtype, device=x.device)
    qa, la = _window_structs(gate_up, cs)
    if ws is None:
        ws = workspace(lib().cl_linear_window_workspace(2, qa, la, T), x.device)
    _check(lib().cl_linear_decode_glu(qa, la, _ptr(x), T, _DTYPE_CODE[x.dtype], _ptr(h), _DTYPE_CODE[h.dtype],
                                      _ptr(ws), ws.numel(), _stream(stream)))
    return h


def allocate_ranks(sigmas, sens, layer_score, r_std, levels, r_max, tau=0.01):
    """``cl_allocate_ranks`` (host code): ranks of one compensation window
    from the linears' descending singular values (sequences of float32),
    their sensitivities and the layer score; returns a list of ints."""
    n = len(sigmas)
    arrs = [np.ascontiguousarray(np.asarray(sg, dtype=np.float32)) for sg in sigmas]
    sp = (ctypes.c_void_p * n)(*[a.ctypes.data for a in arrs])
    ln = (ctypes.c_int32 * n)(*[a.size for a in arrs])
    sd = (ctypes.c_double * n)(*[float(v) for v in sens])
    lv = (ctypes.c_int32 * len(levels))(*[int(v) for v in levels])
    out = (ctypes.c_int32 * n)()
    _check(lib().cl_allocate_ranks(n, sp, ln, sd, float(layer_score), float(r_std), lv, len(levels), int(r_max),
                                   float(tau), out))
    return list(out)


def layer_sensitivity(D, K):
    """``cl_layer_sensitivity`` (host code): layer scores from layer-level
    sensitivities, the top K scoring 1."""
    L = len(D)
    d = (ctypes.c_double * L)(*[float(v) for v in D])
    out = (ctypes.c_double * L)()
    _check(lib().cl_layer_sensitivity(L, d, int(K), out))
    return list(out)


def prefill_workspace(w, c, M):
    qc = w.c()
    lc = c.c() if c is not None else None
    return lib().cl_prefill_workspace(ctypes.byref(qc), ctypes.byref(lc) if lc else None, M)


def linear_prefill(w, c, X, out_dtype=torch.float16, Y=None, ws=None, stream=None):
    """``cl_linear_prefill``: X [M][d_in] fp16/bf16 -> Y [M][d_out] of out_dtype."""
    M = X.shape[0]
    if Y is None:
        Y = torch.empty((M, w.d_out), dtype=out_dtype, device=X.device)
    need = prefill_workspace(w, c, M)
    if ws is None and need:
        ws = workspace(need, X.device)
    qc = w.c()
    lc = c.c() if c is not None else None
    _check(lib().cl_linear_prefill(ctypes.byref(qc), ctypes.byref(lc) if lc else None, _ptr(X), M,
                                   _DTYPE_CODE[X.dtype], _ptr(Y), _DTYPE_CODE[Y.dtype], _ptr(ws),
                                   0 if ws is None else ws.numel(), _stream(stream)))
    return Y


@dataclass
class MoeExperts:
    """Stacked experts of one MoE projection on the device: q [E][d_out][...],
    scales/zeros [E][d_out][d_in/G], A [E][r_max][d_in], B [E][d_out][r_max],
    ranks int32 [E]."""
    q: torch.Tensor
    scales: torch.Tensor
    zeros: torch.Tensor
    A: Optional[torch.Tensor]
    B: Optional[torch.Tensor]
    ranks: Optional[torch.Tensor]
    num_experts: int
    d_out: int
    d_in: int
    bits: int
    group_size: int
    r_max: int

    def expert0(self):
        return QWeightC(self.q.data_ptr(), self.scales.data_ptr(), self.zeros.data_ptr(), self.d_out, self.d_in,
                        self.bits, self.group_size)


def moe_workspace(ex, T, k, x_per_slot):
    q0 = ex.expert0()
    return lib().cl_moe_workspace(ctypes.byref(q0), ex.r_max, ex.num_experts, T, k, int(bool(x_per_slot)))


def moe_linear_decode(ex, x, topk_ids, out_dtype=torch.float16, y=None, ws=None, stream=None):
    """``cl_moe_linear_decode``: x [T][d_in] (shared) or [T][k][d_in] (per
    slot), topk_ids int32 [T][k] -> y [T][k][d_out]."""
    T, k = topk_ids.shape
    x_per_slot = x.dim() == 3
    if y is None:
        y = torch.empty((T, k, ex.d_out), dtype=out_dtype, device=x.device)
    if ws is None:
        ws = workspace(moe_workspace(ex, T, k, x_per_slot), x.device)
    q0 = ex.expert0()
    _check(lib().cl_moe_linear_decode(ctypes.byref(q0), _ptr(ex.A), _ptr(ex.B), ex.r_max, _ptr(ex.ranks),
                                      ex.num_experts, _ptr(x), int(x_per_slot), _ptr(topk_ids), T, k,
                                      _DTYPE_CODE[x.dtype], _ptr(y), _DTYPE_CODE[y.dtype], _ptr(ws), ws.numel(),
                                      _stream(stream)))
    return y


def _moe_window_arrays(exs):
    n = len(exs)
    q0 = (QWeightC * n)(*[ex.expert0() for ex in exs])
    A = (ctypes.c_void_p * n)(*[_ptr(ex.A) for ex in exs])
    B = (ctypes.c_void_p * n)(*[_ptr(ex.B) for ex in exs])
    rm = (ctypes.c_int32 * n)(*[ex.r_max for ex in exs])
    rk = (ctypes.c_void_p * n)(*[_ptr(ex.ranks) for ex in exs])
    return n, q0, A, B, rm, rk


def moe_window_workspace(exs, T, k, x_per_slot):
    n, q0, _, _, rm, _ = _moe_window_arrays(exs)
    return lib().cl_moe_window_workspace(n, q0, rm, exs[0].num_experts, T, k, int(bool(x_per_slot)))


def moe_linear_decode_window(exs, x, topk_ids, out_dtype=torch.float16, ys=None, ws=None, stream=None,
                             slot_ranks=None):
    """``cl_moe_linear_decode_window``: the MoE linears ``exs`` (same d_in,
    bits, group size and expert count) over one routing and one activation
    tensor -> one ``y [T][k][d_out_i]`` per linear.  ``slot_ranks``: None, or
    one device int32 ``[T][k]`` tensor (or None) per linear, used in place of
    the experts' ranks."""
    T, k = topk_ids.shape
    x_per_slot = x.dim() == 3
    if ys is None:
        ys = [torch.empty((T, k, ex.d_out), dtype=out_dtype, device=x.device) for ex in exs]
    if ws is None:
        ws = workspace(moe_window_workspace(exs, T, k, x_per_slot), x.device)
    n, q0, A, B, rm, rk = _moe_window_arrays(exs)
    yp = (ctypes.c_void_p * n)(*[_ptr(y) for y in ys])
    sr = None if slot_ranks is None else (ctypes.c_void_p * n)(*[_ptr(r) for r in slot_ranks])
    _check(lib().cl_moe_linear_decode_window(n, q0, A, B, rm, rk, sr, exs[0].num_experts, _ptr(x), int(x_per_slot),
                                             _ptr(topk_ids), T, k, _DTYPE_CODE[x.dtype], yp,
                                             _DTYPE_CODE[ys[0].dtype], _ptr(ws), ws.numel(), _stream(stream)))
    return ys


def build_compensation(W, w, r_max, stream=None):
    """``cl_build_compensation``: fp32 weight ``W`` [d_out][d_in] and its
    packed backbone ``w`` -> ``(A fp16 [r_max][d_in], B fp16 [d_out][r_max],
    sigma fp32 [min(d_out, d_in)])``.  Waits on the stream once per sweep."""
    A = torch.empty((r_max, w.d_in), dtype=torch.float16, device=W.device)
    B = torch.empty((w.d_out, r_max), dtype=torch.float16, device=W.device)
    sigma = torch.empty((min(w.d_out, w.d_in),), dtype=torch.float32, device=W.device)
    nbytes = lib().cl_build_compensation_workspace(w.d_out, w.d_in, r_max)
    ws = workspace(nbytes, W.device)
    q = w.c()
    _check(lib().cl_build_compensation(_ptr(W), ctypes.byref(q), r_max, _ptr(A), _ptr(B), _ptr(sigma), _ptr(ws),
                                       ws.numel(), _stream(stream)))
    return A, B, sigma
