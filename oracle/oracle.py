"""ctypes front end of the fp64 oracle (test infrastructure only).

Functions take and return numpy arrays on the host.  Formats follow the
quantized-weight layout of the library under test: int8 codes [N][K] or q4
codes [N][K/2] (low nibble = even k), fp16 scale bit patterns [N][K/32],
activations fp32 or bf16 bit patterns (uint16) [M][K].
"""
import ctypes
import os

import numpy as np

from . import build as _build

FMT_Q4 = 4
FMT_INT8 = 8
DT_F32 = 0
DT_BF16 = 1
BLOCK = 32
ACT_NONE = 0
ACT_GELU = 1

OK = 0
ERR_INVALID = 1
ERR_SHAPE = 2
ERR_RANGE = 4

_LIBS = {}


def load(path=None):
    """Load (building first if absent) the oracle library at `path`."""
    path = path or _build.LIB
    if path not in _LIBS:
        if not os.path.exists(path):
            _build.build(out=path)
        lib = ctypes.CDLL(path)
        i64, p = ctypes.c_int64, ctypes.c_void_p
        lib.oracle_f64_to_f16.argtypes = [ctypes.c_double]
        lib.oracle_f64_to_f16.restype = ctypes.c_uint16
        lib.oracle_f16_to_f64.argtypes = [ctypes.c_uint16]
        lib.oracle_f16_to_f64.restype = ctypes.c_double
        lib.oracle_bf16_to_f64.argtypes = [ctypes.c_uint16]
        lib.oracle_bf16_to_f64.restype = ctypes.c_double
        lib.oracle_quantize.argtypes = [ctypes.c_int, p, i64, i64, p, p]
        lib.oracle_quantize.restype = ctypes.c_int
        lib.oracle_dequantize.argtypes = [ctypes.c_int, p, p, i64, i64, p]
        lib.oracle_dequantize.restype = ctypes.c_int
        lib.oracle_forward.argtypes = [ctypes.c_int, p, ctypes.c_int, i64, i64, p, p, i64, p]
        lib.oracle_forward.restype = ctypes.c_int
        lib.oracle_forward_rows.argtypes = [ctypes.c_int, p, ctypes.c_int, i64, i64, p, p,
                                            i64, p, i64, p]
        lib.oracle_forward_rows.restype = ctypes.c_int
        lib.oracle_forward_f16_rows.argtypes = [p, ctypes.c_int, i64, i64, p, i64, p, i64, p]
        lib.oracle_forward_f16_rows.restype = ctypes.c_int
        lib.oracle_epilogue.argtypes = [p, i64, i64, p, p, ctypes.c_int, p]
        lib.oracle_epilogue.restype = ctypes.c_int
        lib.oracle_quantize_act.argtypes = [p, ctypes.c_int, i64, i64, p, p]
        lib.oracle_quantize_act.restype = ctypes.c_int
        lib.oracle_forward_w8a8_rows.argtypes = [p, p, i64, i64, p, p, i64, p, i64, p]
        lib.oracle_forward_w8a8_rows.restype = ctypes.c_int
        lib.oracle_steer.argtypes = [p, i64, i64, p, ctypes.c_double, ctypes.c_double]
        lib.oracle_steer.restype = ctypes.c_int
        lib.oracle_attention_rows.argtypes = [p, i64, p, i64, p, i64, i64, i64, i64, i64,
                                              ctypes.c_double, p, i64, p]
        lib.oracle_attention_rows.restype = ctypes.c_int
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = ctypes.c_int
        _LIBS[path] = lib
    return _LIBS[path]


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def codes_shape(fmt, N, K):
    return (N, K) if fmt == FMT_INT8 else (N, K // 2)


class OracleError(RuntimeError):
    def __init__(self, status):
        super().__init__(f"oracle status {status}")
        self.status = status


class Oracle:
    """Bound view of one oracle library build (the default one, or a
    deliberately altered copy used to show that the pins catch mistakes)."""

    def __init__(self, path=None):
        self.lib = load(path)

    def num_threads(self):
        return int(self.lib.oracle_num_threads())

    # number formats
    def f64_to_f16(self, v):
        return int(self.lib.oracle_f64_to_f16(float(v)))

    def f16_to_f64(self, h):
        return float(self.lib.oracle_f16_to_f64(int(h)))

    def bf16_to_f64(self, b):
        return float(self.lib.oracle_bf16_to_f64(int(b)))

    # quantizer
    def quantize(self, fmt, W):
        """Returns (codes uint8, scales uint16); raises OracleError."""
        W = np.ascontiguousarray(W, dtype=np.float32)
        N, K = W.shape
        codes = np.zeros(codes_shape(fmt, N, K), dtype=np.uint8)
        scales = np.zeros((N, K // BLOCK if K % BLOCK == 0 else 1), dtype=np.uint16)
        st = self.lib.oracle_quantize(fmt, _ptr(W), N, K, _ptr(codes), _ptr(scales))
        if st != OK:
            raise OracleError(st)
        return codes, scales

    def quantize_status(self, fmt, W):
        W = np.ascontiguousarray(W, dtype=np.float32)
        N, K = W.shape
        codes = np.zeros(codes_shape(fmt, N, max(K, 2)), dtype=np.uint8)
        scales = np.zeros((N, max(K // BLOCK, 1)), dtype=np.uint16)
        return self.lib.oracle_quantize(fmt, _ptr(W), N, K, _ptr(codes), _ptr(scales))

    def dequantize(self, fmt, codes, scales, N, K):
        codes = np.ascontiguousarray(codes, dtype=np.uint8)
        scales = np.ascontiguousarray(scales, dtype=np.uint16)
        out = np.empty((N, K), dtype=np.float64)
        st = self.lib.oracle_dequantize(fmt, _ptr(codes), _ptr(scales), N, K, _ptr(out))
        if st != OK:
            raise OracleError(st)
        return out

    # forward
    def forward(self, fmt, X, xdt, codes, scales, N, rows=None):
        """Y (fp64) = X * dequant(codes, scales)^T, optionally only for the
        listed rows of X.  X is fp32 (xdt=DT_F32) or bf16 bits (DT_BF16)."""
        X = np.ascontiguousarray(X, dtype=np.float32 if xdt == DT_F32 else np.uint16)
        M, K = X.shape
        codes = np.ascontiguousarray(codes, dtype=np.uint8)
        scales = np.ascontiguousarray(scales, dtype=np.uint16)
        if rows is None:
            Y = np.empty((M, N), dtype=np.float64)
            st = self.lib.oracle_forward(fmt, _ptr(X), xdt, M, K, _ptr(codes), _ptr(scales),
                                         N, _ptr(Y))
        else:
            rows = np.ascontiguousarray(rows, dtype=np.int64)
            Y = np.empty((len(rows), N), dtype=np.float64)
            st = self.lib.oracle_forward_rows(fmt, _ptr(X), xdt, M, K, _ptr(codes),
                                              _ptr(scales), N, _ptr(rows), len(rows), _ptr(Y))
        if st != OK:
            raise OracleError(st)
        return Y


    def forward_f16(self, X, xdt, W16, rows=None):
        """Y (fp64) = X * W^T for fp16 weight bit patterns W16 [N][K] (the
        unquantized reference), optionally only for the listed rows of X."""
        X = np.ascontiguousarray(X, dtype=np.float32 if xdt == DT_F32 else np.uint16)
        W16 = np.ascontiguousarray(W16, dtype=np.uint16)
        M, K = X.shape
        N = W16.shape[0]
        rows_arr = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
        nrows = M if rows is None else len(rows_arr)
        Y = np.empty((nrows, N), dtype=np.float64)
        st = self.lib.oracle_forward_f16_rows(
            _ptr(X), xdt, M, K, _ptr(W16), N,
            None if rows_arr is None else _ptr(rows_arr), nrows, _ptr(Y))
        if st != OK:
            raise OracleError(st)
        return Y


    def epilogue(self, Y, bias=None, act=ACT_NONE, residual=None, rows=None):
        """act(Y + bias[n]) + residual[m][n] (fp64) on a product Y of the
        listed rows of X (all rows if None); returns a new array."""
        Y = np.array(Y, dtype=np.float64, order="C", copy=True)
        nrows, N = Y.shape
        b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        r = None if residual is None else np.ascontiguousarray(residual, dtype=np.float32)
        rw = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
        st = self.lib.oracle_epilogue(_ptr(Y), nrows, N, None if rw is None else _ptr(rw),
                                      None if b is None else _ptr(b), act,
                                      None if r is None else _ptr(r))
        if st != OK:
            raise OracleError(st)
        return Y

    # attention (R10)
    def attention(self, Q, K, V, B, T, H, dh, scale=None, rows=None):
        """Softmax attention (fp64) of bf16 bit-pattern operands Q, K, V, each
        [B*T][>= H*dh] (row strides from their shapes): returns O [nrows][H*dh]
        for the listed query rows (b * T + t; all if None)."""
        Q = np.ascontiguousarray(Q, dtype=np.uint16)
        K = np.ascontiguousarray(K, dtype=np.uint16)
        V = np.ascontiguousarray(V, dtype=np.uint16)
        scale = 1.0 / np.sqrt(dh) if scale is None else scale
        rows_arr = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
        nrows = B * T if rows is None else len(rows_arr)
        O = np.empty((nrows, H * dh), dtype=np.float64)
        st = self.lib.oracle_attention_rows(
            _ptr(Q), Q.shape[1], _ptr(K), K.shape[1], _ptr(V), V.shape[1], B, T, H, dh,
            float(scale), None if rows_arr is None else _ptr(rows_arr), nrows, _ptr(O))
        if st != OK:
            raise OracleError(st)
        return O

    # steering (R9)
    def steer(self, Y, direction, hnorm, alpha):
        """Y + alpha * hnorm * direction[n] on every row (Eq. 2), fp64; a
        new array."""
        Y = np.array(Y, dtype=np.float64, order="C", copy=True)
        d = np.ascontiguousarray(direction, dtype=np.float32)
        nrows, N = Y.shape
        st = self.lib.oracle_steer(_ptr(Y), nrows, N, _ptr(d), float(hnorm), float(alpha))
        if st != OK:
            raise OracleError(st)
        return Y

    # W8A8 (R8)
    def quantize_act(self, X, xdt):
        """Per-token int8 quantization of X: (q int8 [M][K], s fp16 bits
        [M]); raises OracleError."""
        X = np.ascontiguousarray(X, dtype=np.float32 if xdt == DT_F32 else np.uint16)
        M, K = X.shape
        q = np.zeros((M, K), dtype=np.int8)
        s = np.zeros(M, dtype=np.uint16)
        st = self.lib.oracle_quantize_act(_ptr(X), xdt, M, K, _ptr(q), _ptr(s))
        if st != OK:
            raise OracleError(st)
        return q, s

    def forward_w8a8(self, qx, sx, codes, scales, N, rows=None):
        """Y (fp64) from per-token int8 activations (qx, sx) and int8
        weights (codes, scales), optionally only for the listed rows."""
        qx = np.ascontiguousarray(qx, dtype=np.int8)
        sx = np.ascontiguousarray(sx, dtype=np.uint16)
        codes = np.ascontiguousarray(codes, dtype=np.uint8)
        scales = np.ascontiguousarray(scales, dtype=np.uint16)
        M, K = qx.shape
        rows_arr = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
        nrows = M if rows is None else len(rows_arr)
        Y = np.empty((nrows, N), dtype=np.float64)
        st = self.lib.oracle_forward_w8a8_rows(
            _ptr(qx), _ptr(sx), M, K, _ptr(codes), _ptr(scales), N,
            None if rows_arr is None else _ptr(rows_arr), nrows, _ptr(Y))
        if st != OK:
            raise OracleError(st)
        return Y


_DEFAULT = None


def default():
    global _DEFAULT
    if _DEFAULT is None:
        _DEFAULT = Oracle()
    return _DEFAULT
