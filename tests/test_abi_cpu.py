"""The C-ABI library loads, exports every function include/qlinear.h declares,
and rejects bad arguments before touching the GPU (CPU only: no call here
reaches a kernel launch or any HIP runtime call)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qlinear.h")
LIB = os.path.join(ROOT, "paper_2607_08526_amd", "libqlinear.so")

OK, INVALID, SHAPE, ALIGN, RANGE, UNSUPPORTED, HIP = range(7)
Q4, INT8, F32, BF16 = 4, 8, 0, 1
ACT_NONE, ACT_GELU = 0, 1


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(qlinear_\w+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        pytest.fail(f"{LIB} not built (run __graft_entry__.build())")
    import torch  # noqa: F401  (same HIP runtime the GPU tests use)
    lib = ctypes.CDLL(LIB)
    i64, vp, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    lib.qlinear_codes_bytes.argtypes = [ci, i64, i64]
    lib.qlinear_codes_bytes.restype = ctypes.c_size_t
    lib.qlinear_scales_bytes.argtypes = [i64, i64]
    lib.qlinear_scales_bytes.restype = ctypes.c_size_t
    lib.qlinear_quantize.argtypes = [ci, vp, i64, i64, vp, vp, vp]
    lib.qlinear_forward.argtypes = [ci, vp, ci, i64, i64, vp, vp, i64, vp, vp]
    lib.qlinear_status_string.restype = ctypes.c_char_p
    return lib


def test_header_declares_the_boundary():
    assert declared_functions() == sorted([
        "qlinear_codes_bytes", "qlinear_scales_bytes", "qlinear_quantize",
        "qlinear_forward", "qlinear_block_forward", "qlinear_forward_ep",
        "qlinear_block_forward_ep", "qlinear_quantize_act", "qlinear_forward_w8a8",
        "qlinear_steer", "qlinear_attention", "qlinear_status_string",
        "qlinear_force_path", "qlinear_block_forward_ep_noalloc"])


def test_force_path_values(lib):
    """The path knob takes the seven documented values (setting it launches
    nothing) and rejects others; left at automatic choice."""
    for p in range(7):
        assert lib.qlinear_force_path(p) == OK
    for bad in (-1, 7, 99):
        assert lib.qlinear_force_path(bad) == INVALID
    assert lib.qlinear_force_path(0) == OK


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_size_helpers(lib):
    assert lib.qlinear_codes_bytes(INT8, 6144, 2048) == 6144 * 2048
    assert lib.qlinear_codes_bytes(Q4, 6144, 2048) == 6144 * 1024
    assert lib.qlinear_codes_bytes(5, 6144, 2048) == 0
    assert lib.qlinear_codes_bytes(16, 6144, 2048) == 2 * 6144 * 2048  # fp16 weights
    assert lib.qlinear_scales_bytes(6144, 2048) == 6144 * 64 * 2
    assert lib.qlinear_scales_bytes(6144, 2047) == 0
    assert lib.qlinear_scales_bytes(0, 64) == 0


def test_status_strings(lib):
    for s in range(7):
        assert lib.qlinear_status_string(s)
    assert lib.qlinear_status_string(99) == b"unknown status"


# fake, never dereferenced device addresses (every call below fails its checks
# before any HIP call, or is the M == 0 no-op)
A16 = 0x10000
A2 = 0x10002
A1 = 0x10001


def fwd(lib, fmt=INT8, X=A16, xdt=BF16, M=4, K=64, codes=A16, scales=A16, N=16, Y=A16):
    return lib.qlinear_forward(fmt, X, xdt, M, K, codes, scales, N, Y, None)


def test_forward_argument_errors(lib):
    assert fwd(lib, fmt=5) == INVALID
    assert fwd(lib, xdt=2) == INVALID
    assert fwd(lib, K=48) == SHAPE
    assert fwd(lib, K=0) == SHAPE
    assert fwd(lib, N=0) == SHAPE
    assert fwd(lib, M=-1) == SHAPE
    assert fwd(lib, X=None) == INVALID
    assert fwd(lib, codes=None) == INVALID
    assert fwd(lib, scales=None) == INVALID
    assert fwd(lib, Y=None) == INVALID
    assert fwd(lib, X=A2) == ALIGN
    assert fwd(lib, codes=A2) == ALIGN
    assert fwd(lib, scales=A1) == ALIGN
    assert fwd(lib, Y=A2) == ALIGN
    assert fwd(lib, M=1 << 31) == UNSUPPORTED
    # M == 0 is a successful no-op even without activation/output buffers
    assert fwd(lib, M=0, X=None, Y=None) == OK


def test_quantize_argument_errors(lib):
    q = lambda fmt=INT8, W=A16, N=8, K=64, c=A16, s=A16: lib.qlinear_quantize(fmt, W, N, K, c, s, None)
    assert q(fmt=3) == INVALID
    assert q(K=40) == SHAPE
    assert q(N=0) == SHAPE
    assert q(W=None) == INVALID
    assert q(c=None) == INVALID
    assert q(W=A2) == ALIGN
    assert q(c=A2) == ALIGN
    assert q(s=A1) == ALIGN
    assert q(N=1 << 40) == UNSUPPORTED


def test_block_forward_argument_errors(lib):
    from paper_2607_08526_amd.qlinear import _Linear
    arr = (_Linear * 2)()
    arr[0] = _Linear(INT8, A16, BF16, 4, 64, 16, A16, A16, A16)
    arr[1] = _Linear(INT8, A16, BF16, 4, 48, 16, A16, A16, A16)  # bad K
    assert lib.qlinear_block_forward(arr, 2, None) == SHAPE
    assert lib.qlinear_block_forward(arr, 0, None) == INVALID
    assert lib.qlinear_block_forward(arr, 9, None) == INVALID
    assert lib.qlinear_block_forward(None, 1, None) == INVALID
    empty = (_Linear * 1)()
    empty[0] = _Linear(Q4, None, BF16, 0, 64, 16, A16, A16, None)
    assert lib.qlinear_block_forward(empty, 1, None) == OK  # all layers empty: no-op


def fwd_ep(lib, bias=None, act=ACT_NONE, residual=None, ydt=F32, Y=A16, M=4, ep=True,
           sdir=None, sstr=None):
    from paper_2607_08526_amd.qlinear import _Epilogue
    e = _Epilogue(bias, act, residual, ydt, sdir, 1.0, sstr)
    return lib.qlinear_forward_ep(INT8, A16, BF16, M, 64, A16, A16, 16, Y,
                                  ctypes.byref(e) if ep else None, None)


def test_forward_ep_argument_errors(lib):
    from paper_2607_08526_amd.qlinear import _Epilogue
    i64, vp, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    lib.qlinear_forward_ep.argtypes = [ci, vp, ci, i64, i64, vp, vp, i64, vp,
                                       ctypes.POINTER(_Epilogue), vp]
    assert fwd_ep(lib, act=2) == INVALID
    assert fwd_ep(lib, act=-1) == INVALID
    assert fwd_ep(lib, ydt=2) == INVALID
    assert fwd_ep(lib, bias=A2) == ALIGN
    assert fwd_ep(lib, residual=A2) == ALIGN
    # bf16 Y needs 2-byte alignment only; fp32 Y needs 4
    assert fwd_ep(lib, Y=A2, ydt=F32, M=0) == OK
    assert fwd_ep(lib, Y=A1, ydt=BF16) == ALIGN
    assert fwd_ep(lib, Y=A2, ydt=F32) == ALIGN
    # an in-place residual add needs fp32 Y
    assert fwd_ep(lib, residual=A16, Y=A16, ydt=BF16) == INVALID
    # steering needs its device strength; 4-byte alignment
    assert fwd_ep(lib, sdir=A16, sstr=None) == INVALID
    assert fwd_ep(lib, sdir=A2, sstr=A16) == ALIGN
    assert fwd_ep(lib, sdir=A16, sstr=A2) == ALIGN
    assert fwd_ep(lib, sdir=None, sstr=A2, M=0) == OK
    # the checks of qlinear_forward still apply; no epilogue is the plain call
    assert lib.qlinear_forward_ep(5, A16, BF16, 4, 64, A16, A16, 16, A16, None, None) == INVALID
    assert fwd_ep(lib, M=0, ep=False) == OK


def test_block_forward_ep_argument_errors(lib):
    from paper_2607_08526_amd.qlinear import _Epilogue, _Linear, _LinearEp
    lib.qlinear_block_forward_ep.argtypes = [ctypes.POINTER(_LinearEp), ctypes.c_int,
                                             ctypes.c_void_p]
    arr = (_LinearEp * 2)()
    arr[0] = _LinearEp(_Linear(INT8, A16, BF16, 4, 64, 16, A16, A16, A16),
                       _Epilogue(A16, ACT_GELU, None, F32))
    arr[1] = _LinearEp(_Linear(INT8, A16, BF16, 4, 64, 16, A16, A16, A16),
                       _Epilogue(None, 7, None, F32))  # unknown act
    assert lib.qlinear_block_forward_ep(arr, 2, None) == INVALID
    arr[1] = _LinearEp(_Linear(INT8, A16, BF16, 4, 64, 16, A16, A16, A1),
                       _Epilogue(None, ACT_NONE, None, BF16))  # odd bf16 Y
    assert lib.qlinear_block_forward_ep(arr, 2, None) == ALIGN
    assert lib.qlinear_block_forward_ep(arr, 0, None) == INVALID
    assert lib.qlinear_block_forward_ep(arr, 9, None) == INVALID
    empty = (_LinearEp * 1)()
    empty[0] = _LinearEp(_Linear(Q4, None, BF16, 0, 64, 16, A16, A16, None),
                         _Epilogue(None, ACT_GELU, None, BF16))
    assert lib.qlinear_block_forward_ep(empty, 1, None) == OK


def test_w8a8_argument_errors(lib):
    from paper_2607_08526_amd.qlinear import _Epilogue
    i64, vp, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    lib.qlinear_quantize_act.argtypes = [vp, ci, i64, i64, vp, vp, vp]
    lib.qlinear_forward_w8a8.argtypes = [vp, vp, i64, i64, vp, vp, i64, vp,
                                         ctypes.POINTER(_Epilogue), vp]
    qa = lambda X=A16, xdt=BF16, M=4, K=64, q=A16, s=A16: lib.qlinear_quantize_act(
        X, xdt, M, K, q, s, None)
    assert qa(xdt=2) == INVALID
    assert qa(K=48) == SHAPE
    assert qa(M=-1) == SHAPE
    assert qa(X=None) == INVALID
    assert qa(q=None) == INVALID
    assert qa(X=A2) == ALIGN
    assert qa(q=A2) == ALIGN
    assert qa(s=A1) == ALIGN
    assert qa(M=1 << 31) == UNSUPPORTED
    assert qa(M=0, X=None, q=None, s=None) == OK

    def fw(q=A16, s=A16, M=4, K=64, c=A16, sc=A16, N=16, Y=A16, ep=None):
        return lib.qlinear_forward_w8a8(q, s, M, K, c, sc, N, Y,
                                        ctypes.byref(ep) if ep is not None else None, None)
    assert fw(K=40) == SHAPE
    assert fw(N=0) == SHAPE
    assert fw(c=None) == INVALID
    assert fw(sc=None) == INVALID
    assert fw(q=None) == INVALID
    assert fw(Y=None) == INVALID
    assert fw(q=A2) == ALIGN
    assert fw(c=A2) == ALIGN
    assert fw(s=A1) == ALIGN
    assert fw(Y=A2) == ALIGN
    assert fw(ep=_Epilogue(None, 5, None, F32)) == INVALID
    assert fw(Y=A1, ep=_Epilogue(None, ACT_NONE, None, BF16)) == ALIGN
    assert fw(M=0, q=None, s=None, Y=None) == OK


def test_steer_argument_errors(lib):
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    lib.qlinear_steer.argtypes = [vp, i64, i64, vp, ctypes.c_float, vp, vp]
    st = lambda h=A16, M=4, N=16, d=A16, s=A16: lib.qlinear_steer(h, M, N, d, 1.0, s, None)
    assert st(N=0) == SHAPE
    assert st(M=-1) == SHAPE
    assert st(d=None) == INVALID
    assert st(s=None) == INVALID
    assert st(h=None) == INVALID
    assert st(h=A2) == ALIGN
    assert st(d=A1) == ALIGN
    assert st(M=1 << 31) == UNSUPPORTED
    assert st(M=0, h=None) == OK


def test_attention_argument_errors(lib):
    i64, vp, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    lib.qlinear_attention.argtypes = [vp, i64, vp, i64, vp, i64, i64, i64, i64, i64,
                                      ctypes.c_float, vp, i64, ci, vp]

    def at(q=A16, ld=128, B=1, T=8, H=2, dh=64, scale=0.125, o=A16, ldo=128, odt=F32):
        return lib.qlinear_attention(q, ld, A16, ld, A16, ld, B, T, H, dh, scale, o, ldo, odt,
                                     None)
    assert at(odt=2) == INVALID
    assert at(T=0) == SHAPE
    assert at(ld=64) == SHAPE
    assert at(ldo=100) == SHAPE
    assert at(dh=32, ld=64, ldo=64) == UNSUPPORTED
    assert at(B=40000, H=2) == UNSUPPORTED
    assert at(q=None) == INVALID
    assert at(scale=float("nan")) == INVALID
    assert at(scale=-0.5) == INVALID
    assert at(q=A2) == ALIGN
    assert at(ld=132) == ALIGN
    assert at(o=0x10008, odt=F32) == ALIGN
    assert at(ldo=130) == ALIGN
