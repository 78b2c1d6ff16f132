"""The C-ABI library loads, exports every entry point its header declares, and
rejects bad arguments with the documented status before touching the GPU."""

import ctypes
import os
import re

import pytest

from paper_2605_05819_amd import cl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cl.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cl_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = cl.lib()
    names = declared_functions()
    assert "cl_linear_decode" in names and "cl_quantize_pack" in names
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_covers_every_declared_symbol():
    assert set(declared_functions()) <= set(cl._SIGNATURES)


FAKE = 0x100000  # a 256-byte aligned non-null address; never dereferenced


def _qw(**kw):
    d = dict(q=FAKE, scales=FAKE, zeros=FAKE, d_out=64, d_in=256, bits=4, group_size=128)
    d.update(kw)
    return cl.QWeightC(**d)


def _decode(qw, lr=None, T=1, act=cl.CL_FP16, out=cl.CL_FP16, x=FAKE, y=FAKE, ws=FAKE, ws_bytes=1 << 20):
    lib = cl.lib()
    return lib.cl_linear_decode(ctypes.byref(qw), ctypes.byref(lr) if lr else None, ctypes.c_void_p(x), T, act,
                                ctypes.c_void_p(y), out, ctypes.c_void_p(ws), ws_bytes, None)


@pytest.mark.parametrize("kw,status,needle", [
    (dict(bits=3), cl.CL_EUNSUPPORTED, "3-bit"),
    (dict(bits=8), cl.CL_EUNSUPPORTED, "bits"),
    (dict(group_size=100), cl.CL_EINVAL, "group_size"),
    (dict(group_size=16), cl.CL_EINVAL, "group_size"),     # a 16-byte run would straddle groups
    (dict(d_in=320), cl.CL_EINVAL, "multiple of group_size"),
    (dict(d_out=0), cl.CL_EINVAL, "positive"),
    (dict(q=0), cl.CL_EINVAL, "null"),
    (dict(q=FAKE + 8), cl.CL_EINVAL, "16-byte"),
    (dict(scales=FAKE + 1), cl.CL_EINVAL, "2-byte"),
])
def test_decode_rejects_bad_weight_descriptors(kw, status, needle):
    assert _decode(_qw(**kw)) == status
    assert needle in cl.lib().cl_last_error().decode()


def test_decode_rejects_bad_calls():
    lib = cl.lib()
    qw = _qw()
    bad_rank = cl.LowRankC(FAKE, FAKE, 16, 17)
    assert _decode(qw, bad_rank) == cl.CL_EINVAL and b"rank" in lib.cl_last_error()
    assert _decode(qw, cl.LowRankC(FAKE, FAKE, 512, 16)) == cl.CL_EINVAL
    assert _decode(qw, cl.LowRankC(0, FAKE, 16, 16)) == cl.CL_EINVAL
    assert _decode(qw, cl.LowRankC(FAKE + 2, FAKE, 16, 16)) == cl.CL_EINVAL
    assert _decode(qw, T=0) == cl.CL_EINVAL
    assert _decode(qw, T=65) == cl.CL_EINVAL
    assert _decode(qw, act=cl.CL_FP32) == cl.CL_EINVAL
    assert _decode(qw, out=7) == cl.CL_EINVAL
    assert _decode(qw, x=0) == cl.CL_EINVAL
    assert _decode(qw, x=FAKE + 2) == cl.CL_EINVAL
    lr = cl.LowRankC(FAKE, FAKE, 16, 16)
    assert _decode(qw, lr, ws=0) == cl.CL_EWORKSPACE
    assert _decode(qw, lr, ws_bytes=16) == cl.CL_EWORKSPACE
    assert b"workspace" in lib.cl_last_error()
    assert _decode(qw, lr, ws=FAKE + 16) == cl.CL_EINVAL


def test_workspace_query_is_pure_and_sized_by_rank_and_tokens():
    lib = cl.lib()
    _decode(_qw(bits=3))
    before = lib.cl_last_error()
    qw = _qw()
    lr = cl.LowRankC(FAKE, FAKE, 64, 32)
    n1 = lib.cl_linear_workspace(ctypes.byref(qw), ctypes.byref(lr), 1)
    n4 = lib.cl_linear_workspace(ctypes.byref(qw), ctypes.byref(lr), 4)
    assert n1 >= 32 * 4 and n4 - n1 >= 3 * 32 * 4       # A x for every token
    assert 0 < lib.cl_linear_workspace(ctypes.byref(qw), None, 4) < n4     # rank 0: activations only
    assert lib.cl_linear_workspace(ctypes.byref(_qw(bits=3)), ctypes.byref(lr), 1) == 0
    assert lib.cl_last_error() == before


def test_quantize_pack_and_dequantize_validate():
    lib = cl.lib()
    p = ctypes.c_void_p(FAKE)
    assert lib.cl_quantize_pack(p, 64, 256, 3, 128, p, p, p, None) == cl.CL_EUNSUPPORTED
    assert lib.cl_quantize_pack(p, 64, 256, 4, 96, p, p, p, None) == cl.CL_EINVAL
    assert lib.cl_quantize_pack(None, 64, 256, 4, 128, p, p, p, None) == cl.CL_EINVAL
    assert lib.cl_quantize_pack(p, 64, 256, 4, 128, ctypes.c_void_p(FAKE + 4), p, p, None) == cl.CL_EINVAL
    qw = _qw(zeros=0)
    assert lib.cl_dequantize(ctypes.byref(qw), p, None) == cl.CL_EINVAL
    qw = _qw()
    assert lib.cl_dequantize(ctypes.byref(qw), None, None) == cl.CL_EINVAL


def test_window_validation():
    lib = cl.lib()
    q = (cl.QWeightC * 3)(_qw(), _qw(d_out=32), _qw(d_in=512))
    yp = (ctypes.c_void_p * 3)(FAKE, FAKE, FAKE)
    args = lambda n, qa, **kw: lib.cl_linear_decode_window(
        n, qa, None, ctypes.c_void_p(FAKE), kw.get("T", 1), cl.CL_FP16, yp, cl.CL_FP16,
        ctypes.c_void_p(FAKE), 1 << 20, None)
    assert args(0, q) == cl.CL_EINVAL
    assert args(9, q) == cl.CL_EINVAL
    assert args(3, q) == cl.CL_EINVAL and b"share d_in" in lib.cl_last_error()
    assert lib.cl_linear_window_workspace(3, q, None, 1) == 0
    q2 = (cl.QWeightC * 2)(_qw(), _qw(d_out=32))
    n2 = lib.cl_linear_window_workspace(2, q2, None, 1)
    assert n2 > 0
    ybad = (ctypes.c_void_p * 2)(FAKE, 0)
    assert lib.cl_linear_decode_window(2, q2, None, ctypes.c_void_p(FAKE), 1, cl.CL_FP16, ybad, cl.CL_FP16,
                                       ctypes.c_void_p(FAKE), 1 << 20, None) == cl.CL_EINVAL
