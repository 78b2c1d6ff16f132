"""Thin Python binding of ``libcl.so`` (the C ABI declared in ``include/cl.h``).

Argument marshalling only: every step of the layer runs in the HIP kernels of
the library.  PyTorch provides device memory and the current stream.  If the
library has not been built, :func:`lib` raises -- there is no fallback path.
The environment variable CL_LIBRARY, when set, names another build of the same
library to load instead (the host-sanitized build, for instance).
"""

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

LIB_PATH = os.environ.get("CL_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcl.so")

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
    "cl_linear_decode_noalloc": (ctypes.c_int32, [ctypes.POINTER(QWeightC), ctypes.POINTER(LowRankC),
                                                  ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                                  ctypes.c_int32, ctypes.c_void_p]),
    "cl_prefill_workspace": (ctypes.c_size_t, [ctypes.POINTER(QWeightC), ctypes.POINTER(LowRankC), ctypes.c_int32]),
    "cl_linear_prefill": (ctypes.c_int32, [ctypes.POINTER(QWeightC), ctypes.POINTER(LowRankC), ctypes.c_void_p,
                                           ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                           ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "cl_build_compensation_workspace": (ctypes.c_size_t, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]),
    "cl_build_compensation_sweeps": (ctypes.c_int32, []),
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
    "cl_moe_linear_decode_gated": (ctypes.c_int32, [ctypes.POINTER(QWeightC), ctypes.c_void_p, ctypes.c_void_p,
                                                    ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                                    ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                                    ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                                    ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "cl_moe_gated_workspace": (ctypes.c_size_t, [ctypes.POINTER(QWeightC), ctypes.c_int32, ctypes.c_int32,
                                                  ctypes.c_int32, ctypes.c_int32]),
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
    "cl_moe_status": (ctypes.c_int32, [ctypes.c_void_p]),
    "cl_linear_decode_glu": (ctypes.c_int32, [ctypes.POINTER(QWeightC), ctypes.POINTER(LowRankC), ctypes.c_void_p,
                                              ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                                              ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
}


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("%s is not built; run `python -m paper_2605_05819_amd.build`" % LIB_PATH)
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


# ---------------------------------------------------------------- validation
# The C ABI sees raw pointers and sizes only, so a tensor of the wrong dtype,
# shape or layout would be read as something else.  Every call below checks
# its tensors first (dtype, contiguity and shape of all of them, then that
# they are on the GPU) and raises ValueError on a mismatch.

def _need(cond, msg):
    if not cond:
        raise ValueError(msg)


class _Checked(list):
    """Tensors whose layout passed, for the device check that follows."""

    def on_gpu(self):
        for name, t in self:
            _need(t.device.type == "cuda", "%s must be on the GPU (got %s)" % (name, t.device))


def _dev_tensor(t, name, dtypes, shape=None, chk=None):
    _need(isinstance(t, torch.Tensor), "%s must be a torch.Tensor" % name)
    _need(t.dtype in dtypes, "%s must have dtype %s (got %s)" % (name, " or ".join(map(str, dtypes)), t.dtype))
    _need(t.is_contiguous(), "%s must be contiguous" % name)
    if shape is not None:
        _need(tuple(t.shape) == tuple(shape), "%s must have shape %s (got %s)" % (name, tuple(shape), tuple(t.shape)))
    if chk is None:
        _need(t.device.type == "cuda", "%s must be on the GPU (got %s)" % (name, t.device))
    else:
        chk.append((name, t))


_ACT = (torch.float16, torch.bfloat16)
_OUT = (torch.float16, torch.bfloat16, torch.float32)
_I32 = (torch.int32,)


def _check_qweight(w, chk, name="w"):
    _need(w.d_out > 0 and w.d_in > 0 and w.bits > 0 and w.group_size > 0, "%s: sizes must be positive" % name)
    _need((w.d_in * w.bits) % 32 == 0 and w.d_in % w.group_size == 0, "%s: d_in does not fit the packing" % name)
    _dev_tensor(w.q, name + ".q", _I32, (w.d_out, w.d_in * w.bits // 32), chk=chk)
    _dev_tensor(w.scales, name + ".scales", (torch.float16,), (w.d_out, w.d_in // w.group_size), chk=chk)
    _dev_tensor(w.zeros, name + ".zeros", (torch.float16,), (w.d_out, w.d_in // w.group_size), chk=chk)


def _check_lowrank(c, w, chk, name="c"):
    if c is None or c.rank == 0 and c.A is None and c.B is None:
        return
    _need(0 <= c.rank <= c.r_max, "%s: need 0 <= rank <= r_max" % name)
    _dev_tensor(c.A, name + ".A", (torch.float16,), (c.r_max, w.d_in), chk=chk)
    _dev_tensor(c.B, name + ".B", (torch.float16,), (w.d_out, c.r_max), chk=chk)


def _check_act(x, chk, name, d_in, lead=None):
    _dev_tensor(x, name, _ACT, chk=chk)
    _need(x.dim() >= 2 and x.shape[-1] == d_in, "%s must be [..][%d] (got %s)" % (name, d_in, tuple(x.shape)))
    if lead is not None:
        _need(tuple(x.shape[:-1]) == tuple(lead), "%s must have shape %s (got %s)"
              % (name, tuple(lead) + (d_in,), tuple(x.shape)))


def _check_ws(ws, need, chk, name="ws"):
    if ws is None:
        return
    _dev_tensor(ws, name, (torch.uint8,), chk=chk)
    _need(ws.numel() >= need, "%s holds %d bytes, %d needed" % (name, ws.numel(), need))


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
    chk = _Checked()
    _check_qweight(w, chk)
    _check_lowrank(c, w, chk)
    _check_act(x, chk, "x", w.d_in)
    _need(x.dim() == 2, "x must be [T][d_in]")
    T = x.shape[0]
    if y is None:
        y = torch.empty((T, w.d_out), dtype=out_dtype, device=x.device)
    _dev_tensor(y, "y", _OUT, (T, w.d_out), chk)
    chk.on_gpu()
    need = linear_workspace(w, c, T)
    if ws is None:
        ws = workspace(need, x.device)
    _check_ws(ws, need, None)
    qc = w.c()
    lc = c.c() if c is not None else None
    _check(lib().cl_linear_decode(ctypes.byref(qc), ctypes.byref(lc) if lc else None, _ptr(x), T,
                                  _DTYPE_CODE[x.dtype], _ptr(y), _DTYPE_CODE[y.dtype], _ptr(ws),
                                  0 if ws is None else ws.numel(), _stream(stream)))
    return y


def linear_decode_noalloc(w, c, x, out_dtype=torch.float16, y=None, stream=None):
    """``cl_linear_decode_noalloc``: as :func:`linear_decode`, with the
    library's per-device scratch in place of a workspace (calls overlapping
    on one device race)."""
    chk = _Checked()
    _check_qweight(w, chk)
    _check_lowrank(c, w, chk)
    _check_act(x, chk, "x", w.d_in)
    _need(x.dim() == 2, "x must be [T][d_in]")
    T = x.shape[0]
    if y is None:
        y = torch.empty((T, w.d_out), dtype=out_dtype, device=x.device)
    _dev_tensor(y, "y", _OUT, (T, w.d_out), chk)
    chk.on_gpu()
    qc = w.c()
    lc = c.c() if c is not None else None
    _check(lib().cl_linear_decode_noalloc(ctypes.byref(qc), ctypes.byref(lc) if lc else None, _ptr(x), T,
                                          _DTYPE_CODE[x.dtype], _ptr(y), _DTYPE_CODE[y.dtype], _stream(stream)))
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
    n = len(ws_)
    _need(cs is None or len(cs) == n, "one factor set per linear")
    _need(all(w.d_in == ws_[0].d_in and w.bits == ws_[0].bits and w.group_size == ws_[0].group_size for w in ws_),
          "the linears of a window must share d_in, bits and group size")
    chk = _Checked()
    for i, w in enumerate(ws_):
        _check_qweight(w, chk, "w[%d]" % i)
        _check_lowrank(None if cs is None else cs[i], w, chk, "c[%d]" % i)
    _check_act(x, chk, "x", ws_[0].d_in)
    _need(x.dim() == 2, "x must be [T][d_in]")
    T = x.shape[0]
    if ys is None:
        ys = [torch.empty((T, w.d_out), dtype=out_dtype, device=x.device) for w in ws_]
    _need(len(ys) == n, "one output per linear")
    for i, (w, y) in enumerate(zip(ws_, ys)):
        _dev_tensor(y, "ys[%d]" % i, _OUT, (T, w.d_out), chk)
    chk.on_gpu()
    qa, la = _window_structs(ws_, cs)
    need = lib().cl_linear_window_workspace(n, qa, la, T)
    if ws is None:
        ws = workspace(need, x.device)
    _check_ws(ws, need, None)
    yp = (ctypes.c_void_p * n)(*[y.data_ptr() for y in ys])
    _check(lib().cl_linear_decode_window(n, qa, la, _ptr(x), T, _DTYPE_CODE[x.dtype], yp,
                                         _DTYPE_CODE[ys[0].dtype], _ptr(ws), ws.numel(), _stream(stream)))
    return ys


def linear_decode_glu(gate_up, cs, x, out_dtype=torch.float16, h=None, ws=None, stream=None):
    """``cl_linear_decode_glu``: h = SiLU(gate x) * (up x) [T][d_out] for
    gate_up = (gate, up) and their factors cs (or None)."""
    _need(len(gate_up) == 2 and (cs is None or len(cs) == 2), "gate_up and cs are (gate, up) pairs")
    chk = _Checked()
    for i, w in enumerate(gate_up):
        _check_qweight(w, chk, ("gate", "up")[i])
        _check_lowrank(None if cs is None else cs[i], w, chk, ("gate", "up")[i] + " factors")
    _check_act(x, chk, "x", gate_up[0].d_in)
    _need(x.dim() == 2, "x must be [T][d_in]")
    T = x.shape[0]
    if h is None:
        h = torch.empty((T, gate_up[0].d_out), dtype=out_dtype, device=x.device)
    _dev_tensor(h, "h", _OUT, (T, gate_up[0].d_out), chk)
    chk.on_gpu()
    qa, la = _window_structs(gate_up, cs)
    need = lib().cl_linear_window_workspace(2, qa, la, T)
    if ws is None:
        ws = workspace(need, x.device)
    _check_ws(ws, need, None)
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
    chk = _Checked()
    _check_qweight(w, chk)
    _check_lowrank(c, w, chk)
    _check_act(X, chk, "X", w.d_in)
    _need(X.dim() == 2, "X must be [M][d_in]")
    M = X.shape[0]
    if Y is None:
        Y = torch.empty((M, w.d_out), dtype=out_dtype, device=X.device)
    _dev_tensor(Y, "Y", _OUT, (M, w.d_out), chk)
    chk.on_gpu()
    need = prefill_workspace(w, c, M)
    if ws is None and need:
        ws = workspace(need, X.device)
    _check_ws(ws, need, None)
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


def _check_experts(ex, chk, name="ex"):
    """Stacked experts: q [E][d_out][d_in*bits/32], scales/zeros
    [E][d_out][d_in/G], and with r_max > 0 A [E][r_max][d_in],
    B [E][d_out][r_max], ranks [E]."""
    E = ex.num_experts
    _need(E >= 1 and ex.d_out > 0 and ex.d_in > 0 and ex.group_size > 0, "%s: sizes must be positive" % name)
    _need((ex.d_in * ex.bits) % 32 == 0 and ex.d_in % ex.group_size == 0, "%s: d_in does not fit the packing" % name)
    _dev_tensor(ex.q, name + ".q", _I32, (E, ex.d_out, ex.d_in * ex.bits // 32), chk)
    _dev_tensor(ex.scales, name + ".scales", (torch.float16,), (E, ex.d_out, ex.d_in // ex.group_size), chk)
    _dev_tensor(ex.zeros, name + ".zeros", (torch.float16,), (E, ex.d_out, ex.d_in // ex.group_size), chk)
    if ex.r_max > 0:
        _dev_tensor(ex.A, name + ".A", (torch.float16,), (E, ex.r_max, ex.d_in), chk)
        _dev_tensor(ex.B, name + ".B", (torch.float16,), (E, ex.d_out, ex.r_max), chk)
        _dev_tensor(ex.ranks, name + ".ranks", _I32, (E,), chk)


def _check_moe_inputs(exs, x, topk_ids, ys, chk):
    for i, ex in enumerate(exs):
        _check_experts(ex, chk, "experts[%d]" % i)
        _need(ex.num_experts == exs[0].num_experts and ex.d_in == exs[0].d_in, "the linears of a window must "
              "share the expert count and d_in")
    _dev_tensor(topk_ids, "topk_ids", _I32, chk=chk)
    _need(topk_ids.dim() == 2, "topk_ids must be [T][k]")
    T, k = topk_ids.shape
    _check_act(x, chk, "x", exs[0].d_in)
    _need(tuple(x.shape[:-1]) in ((T,), (T, k)), "x must be [T][d_in] or [T][k][d_in] with (T, k) = %s (got %s)"
          % ((T, k), tuple(x.shape)))
    for i, (ex, y) in enumerate(zip(exs, ys)):
        _dev_tensor(y, "y[%d]" % i, _OUT, (T, k, ex.d_out), chk)


def moe_workspace(ex, T, k, x_per_slot):
    q0 = ex.expert0()
    return lib().cl_moe_workspace(ctypes.byref(q0), ex.r_max, ex.num_experts, T, k, int(bool(x_per_slot)))


def moe_linear_decode(ex, x, topk_ids, out_dtype=torch.float16, y=None, ws=None, stream=None):
    """``cl_moe_linear_decode``: x [T][d_in] (shared) or [T][k][d_in] (per
    slot), topk_ids int32 [T][k] -> y [T][k][d_out]."""
    _need(isinstance(topk_ids, torch.Tensor) and topk_ids.dim() == 2, "topk_ids must be a [T][k] tensor")
    T, k = topk_ids.shape
    x_per_slot = x.dim() == 3
    if y is None:
        y = torch.empty((T, k, ex.d_out), dtype=out_dtype, device=x.device)
    chk = _Checked()
    _check_moe_inputs([ex], x, topk_ids, [y], chk)
    chk.on_gpu()
    need = moe_workspace(ex, T, k, x_per_slot)
    if ws is None:
        ws = workspace(need, x.device)
    _check_ws(ws, need, None)
    q0 = ex.expert0()
    _check(lib().cl_moe_linear_decode(ctypes.byref(q0), _ptr(ex.A), _ptr(ex.B), ex.r_max, _ptr(ex.ranks),
                                      ex.num_experts, _ptr(x), int(x_per_slot), _ptr(topk_ids), T, k,
                                      _DTYPE_CODE[x.dtype], _ptr(y), _DTYPE_CODE[y.dtype], _ptr(ws), ws.numel(),
                                      _stream(stream)))
    return y


def moe_gated_workspace(ex, T, k):
    q0 = ex.expert0()
    return lib().cl_moe_gated_workspace(ctypes.byref(q0), ex.r_max, ex.num_experts, T, k)


def moe_linear_decode_gated(ex, g, u, topk_ids, out_dtype=torch.float16, y=None, ws=None, stream=None,
                            slot_ranks=None):
    """``cl_moe_linear_decode_gated``: the down projection of SiLU(g) * u,
    with g and u the slots' gate and up outputs [T][k][d_in] (fp16 or bf16,
    one dtype), topk_ids int32 [T][k] -> y [T][k][d_out].  ``slot_ranks``:
    None or a device int32 [T][k] tensor used in place of the experts'
    ranks."""
    _need(isinstance(topk_ids, torch.Tensor) and topk_ids.dim() == 2, "topk_ids must be a [T][k] tensor")
    T, k = topk_ids.shape
    _need(isinstance(g, torch.Tensor) and isinstance(u, torch.Tensor) and g.dim() == 3 and
          tuple(u.shape) == tuple(g.shape) and u.dtype == g.dtype, "g and u must be [T][k][d_in] of one dtype")
    if y is None:
        y = torch.empty((T, k, ex.d_out), dtype=out_dtype, device=g.device)
    chk = _Checked()
    _check_moe_inputs([ex], g, topk_ids, [y], chk)
    _check_act(u, chk, "u", ex.d_in)
    if slot_ranks is not None:
        _dev_tensor(slot_ranks, "slot_ranks", _I32, (T, k), chk)
    chk.on_gpu()
    need = moe_gated_workspace(ex, T, k)
    if ws is None:
        ws = workspace(need, g.device)
    _check_ws(ws, need, None)
    q0 = ex.expert0()
    _check(lib().cl_moe_linear_decode_gated(ctypes.byref(q0), _ptr(ex.A), _ptr(ex.B), ex.r_max, _ptr(ex.ranks),
                                            _ptr(slot_ranks), ex.num_experts, _ptr(g), _ptr(u), _ptr(topk_ids), T,
                                            k, _DTYPE_CODE[g.dtype], _ptr(y), _DTYPE_CODE[y.dtype], _ptr(ws),
                                            ws.numel(), _stream(stream)))
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
    _need(isinstance(topk_ids, torch.Tensor) and topk_ids.dim() == 2, "topk_ids must be a [T][k] tensor")
    T, k = topk_ids.shape
    x_per_slot = x.dim() == 3
    if ys is None:
        ys = [torch.empty((T, k, ex.d_out), dtype=out_dtype, device=x.device) for ex in exs]
    _need(len(ys) == len(exs), "one output per linear")
    chk = _Checked()
    _check_moe_inputs(exs, x, topk_ids, ys, chk)
    if slot_ranks is not None:
        _need(len(slot_ranks) == len(exs), "one slot-rank table (or None) per linear")
        for i, r in enumerate(slot_ranks):
            if r is not None:
                _dev_tensor(r, "slot_ranks[%d]" % i, _I32, (T, k), chk)
    chk.on_gpu()
    need = moe_window_workspace(exs, T, k, x_per_slot)
    if ws is None:
        ws = workspace(need, x.device)
    _check_ws(ws, need, None)
    n, q0, A, B, rm, rk = _moe_window_arrays(exs)
    yp = (ctypes.c_void_p * n)(*[_ptr(y) for y in ys])
    sr = None if slot_ranks is None else (ctypes.c_void_p * n)(*[_ptr(r) for r in slot_ranks])
    _check(lib().cl_moe_linear_decode_window(n, q0, A, B, rm, rk, sr, exs[0].num_experts, _ptr(x), int(x_per_slot),
                                             _ptr(topk_ids), T, k, _DTYPE_CODE[x.dtype], yp,
                                             _DTYPE_CODE[ys[0].dtype], _ptr(ws), ws.numel(), _stream(stream)))
    return ys


def moe_status(stream=None):
    """``cl_moe_status``: waits for the stream, then raises ClError
    (CL_EINVAL) if a MoE call on this device met a routing id outside
    0..E-1 since the last check (the record is cleared)."""
    _check(lib().cl_moe_status(_stream(stream)))


def build_compensation_sweeps():
    """``cl_build_compensation_sweeps``: Jacobi sweeps of this thread's last
    :func:`build_compensation` call."""
    return int(lib().cl_build_compensation_sweeps())


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
