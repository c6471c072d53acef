"""Python binding of libqlinear.so (include/qlinear.h).

Argument marshalling only: every step of quantization and of the forward
product runs in the library's HIP kernels.  PyTorch provides device memory
and the current HIP stream.  There is no fallback: if the library is missing
or the process has no GPU, calls raise.
"""
import ctypes
import os

import torch

from . import build as _build

FMT_Q4 = 4
FMT_INT8 = 8
FMT_F16 = 16  # unquantized fp16 weights (forward only; scales unused)
DT_F32 = 0
DT_BF16 = 1
ACT_NONE = 0
ACT_GELU = 1  # exact GELU, x * Phi(x)
BLOCK = 32
MAX_GROUP = 8

STATUS = {
    0: "QL_OK", 1: "QL_ERR_INVALID", 2: "QL_ERR_SHAPE", 3: "QL_ERR_ALIGN",
    4: "QL_ERR_RANGE", 5: "QL_ERR_UNSUPPORTED", 6: "QL_ERR_HIP",
}

EXPORTS = [
    "qlinear_codes_bytes", "qlinear_scales_bytes", "qlinear_quantize",
    "qlinear_forward", "qlinear_block_forward", "qlinear_forward_ep",
    "qlinear_block_forward_ep", "qlinear_quantize_act", "qlinear_forward_w8a8",
    "qlinear_steer", "qlinear_attention", "qlinear_status_string",
    "qlinear_force_path", "qlinear_block_forward_ep_noalloc",
]

PATH_AUTO, PATH_GEMV, PATH_STREAM, PATH_SKINNY, PATH_TILED, PATH_WIDE, PATH_MID = range(7)


class QLinearError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class _Linear(ctypes.Structure):
    _fields_ = [
        ("fmt", ctypes.c_int),
        ("X", ctypes.c_void_p),
        ("xdt", ctypes.c_int),
        ("M", ctypes.c_int64),
        ("K", ctypes.c_int64),
        ("N", ctypes.c_int64),
        ("codes", ctypes.c_void_p),
        ("scales", ctypes.c_void_p),
        ("Y", ctypes.c_void_p),
    ]


class _Epilogue(ctypes.Structure):
    _fields_ = [
        ("bias", ctypes.c_void_p),
        ("act", ctypes.c_int),
        ("residual", ctypes.c_void_p),
        ("ydt", ctypes.c_int),
        ("steer_dir", ctypes.c_void_p),
        ("steer_norm", ctypes.c_float),
        ("steer_strength", ctypes.c_void_p),
        ("y_bf16_copy", ctypes.c_void_p),
    ]


class _LinearEp(ctypes.Structure):
    _fields_ = [("lin", _Linear), ("ep", _Epilogue)]


_LIB = None


def lib_path():
    return _build.LIB


def _hip_runtimes_mapped():
    paths = set()
    with open("/proc/self/maps") as f:
        for line in f:
            p = line.split()[-1] if len(line.split()) >= 6 else ""
            if "libamdhip64.so" in p:
                paths.add(os.path.realpath(p))
    return paths


def load():
    """Load libqlinear.so (built in-tree by build.py); raises if absent."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = lib_path()
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with "
                          "`python -m paper_2607_08526_amd.build` (no CPU fallback exists)")
    # torch's HIP runtime is loaded first (import above), so the library's
    # libamdhip64.so.7 dependency resolves to that same copy: device pointers
    # and streams from torch are then valid inside the library.
    lib = ctypes.CDLL(path)
    i64, vp, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    lib.qlinear_codes_bytes.argtypes = [ci, i64, i64]
    lib.qlinear_codes_bytes.restype = ctypes.c_size_t
    lib.qlinear_scales_bytes.argtypes = [i64, i64]
    lib.qlinear_scales_bytes.restype = ctypes.c_size_t
    lib.qlinear_quantize.argtypes = [ci, vp, i64, i64, vp, vp, vp]
    lib.qlinear_quantize.restype = ci
    lib.qlinear_forward.argtypes = [ci, vp, ci, i64, i64, vp, vp, i64, vp, vp]
    lib.qlinear_forward.restype = ci
    lib.qlinear_block_forward.argtypes = [ctypes.POINTER(_Linear), ci, vp]
    lib.qlinear_forward_ep.argtypes = [ci, vp, ci, i64, i64, vp, vp, i64, vp,
                                       ctypes.POINTER(_Epilogue), vp]
    lib.qlinear_forward_ep.restype = ci
    lib.qlinear_block_forward_ep.argtypes = [ctypes.POINTER(_LinearEp), ci, vp]
    lib.qlinear_block_forward_ep.restype = ci
    lib.qlinear_block_forward_ep_noalloc.argtypes = [ctypes.POINTER(_LinearEp), ci, vp]
    lib.qlinear_block_forward_ep_noalloc.restype = ci
    lib.qlinear_quantize_act.argtypes = [vp, ci, i64, i64, vp, vp, vp]
    lib.qlinear_quantize_act.restype = ci
    lib.qlinear_forward_w8a8.argtypes = [vp, vp, i64, i64, vp, vp, i64, vp,
                                         ctypes.POINTER(_Epilogue), vp]
    lib.qlinear_forward_w8a8.restype = ci
    lib.qlinear_steer.argtypes = [vp, i64, i64, vp, ctypes.c_float, vp, vp]
    lib.qlinear_steer.restype = ci
    lib.qlinear_attention.argtypes = [vp, i64, vp, i64, vp, i64, i64, i64, i64, i64,
                                      ctypes.c_float, vp, i64, ci, vp]
    lib.qlinear_attention.restype = ci
    lib.qlinear_block_forward.restype = ci
    lib.qlinear_force_path.argtypes = [ci]
    lib.qlinear_force_path.restype = ci
    lib.qlinear_status_string.argtypes = [ci]
    lib.qlinear_status_string.restype = ctypes.c_char_p
    if len(_hip_runtimes_mapped()) > 1:
        raise ImportError(f"two HIP runtimes are mapped: {_hip_runtimes_mapped()}")
    _LIB = lib
    return lib


def _check(status):
    if status != 0:
        raise QLinearError(status, load().qlinear_status_string(status).decode())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


# Argument checks of the binding.  The library receives bare pointers and
# sizes, so a tensor of the wrong dtype, shape or layout would be read or
# written out of bounds; these checks run before the library is called.
_TWO_BYTE = (torch.int16, torch.uint16, torch.bfloat16, torch.float16)
_BF16_BITS = (torch.bfloat16, torch.int16, torch.uint16)


def _require(t, name, dtypes, shape=None, min_cols=None):
    """t must be a contiguous (or, with min_cols, unit-column-stride 2-D)
    device tensor of one of `dtypes`, with `shape` (None entries: any)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor, not {type(t).__name__}")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} must have dtype {' or '.join(str(d) for d in dtypes)}, "
                        f"not {t.dtype}")
    if shape is not None:
        if t.dim() != len(shape) or any(w is not None and w != h for w, h in zip(shape, t.shape)):
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected "
                             f"{tuple('*' if w is None else w for w in shape)}")
    if min_cols is not None:
        if t.dim() != 2 or t.stride(1) != 1 or t.shape[1] < min_cols or \
                (t.shape[0] > 1 and t.stride(0) < min_cols):
            raise ValueError(f"{name} must be a 2-D row view with unit column stride and at "
                             f"least {min_cols} columns per row")
    elif not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _on_device(*tensors):
    """Every tensor given (None skipped) must be device memory; checked
    after the dtype and shape checks of a call."""
    for t in tensors:
        if t is not None and not t.is_cuda:
            raise ValueError("every tensor argument must be a device (cuda) tensor")


def _require_weights(fmt, codes, scales, N, K):
    if fmt == FMT_F16:
        _require(codes, "codes (fp16 weights)", _TWO_BYTE, (N, K))
        return
    if fmt not in (FMT_INT8, FMT_Q4):
        raise ValueError(f"unknown weight format {fmt}")
    if K % BLOCK:
        raise ValueError(f"K = {K} is not a multiple of {BLOCK}")
    _require(codes, "codes", (torch.uint8, torch.int8), (N, K if fmt == FMT_INT8 else K // 2))
    _require(scales, "scales", _TWO_BYTE, (N, K // BLOCK))


def _require_x(X):
    if not isinstance(X, torch.Tensor) or X.dim() != 2:
        raise ValueError("activations X must be a 2-D tensor [M][K]")
    _require(X, "X", (torch.float32,) + _BF16_BITS)
    return X.shape


def _require_y(Y, M, N, ydtypes=(torch.float32,)):
    _require(Y, "Y", ydtypes, (M, N))


def _require_ep(bias, residual, M, N):
    if bias is not None:
        _require(bias, "bias", (torch.float32,), (N,))
    if residual is not None:
        _require(residual, "residual", (torch.float32,), (M, N))


def _require_ycopy(ycopy, Y, M, N):
    if ycopy is None:
        return
    _require(ycopy, "ycopy", _BF16_BITS, (M, N))
    if Y.dtype != torch.float32:
        raise ValueError("a bf16 copy is taken of an fp32 output only")


def _require_steer(steer, N):
    if steer is None:
        return
    d, hnorm, strength = steer
    _require(d, "steering direction", (torch.float32,), (N,))
    _require(strength, "steering strength", (torch.float32,))
    if strength.numel() < 1:
        raise ValueError("steering strength must hold one element")


def codes_bytes(fmt, N, K):
    return int(load().qlinear_codes_bytes(fmt, N, K))


def scales_bytes(N, K):
    return int(load().qlinear_scales_bytes(N, K))


def empty_codes(fmt, N, K, device="cuda"):
    return torch.empty((N, K) if fmt == FMT_INT8 else (N, K // 2), dtype=torch.uint8,
                       device=device)


def empty_scales(N, K, device="cuda"):
    # fp16 bit patterns; int16 storage so torch never reinterprets them
    return torch.empty((N, K // BLOCK), dtype=torch.int16, device=device)


def quantize(fmt, W, codes=None, scales=None, stream=None):
    """Quantize fp32 W [N][K] (device) -> (codes, scales).  Synchronous."""
    if fmt not in (FMT_INT8, FMT_Q4):
        raise ValueError(f"quantize takes FMT_INT8 or FMT_Q4, not {fmt}")
    _require(W, "W", (torch.float32,), (None, None))
    N, K = W.shape
    if K % BLOCK:
        raise ValueError(f"K = {K} is not a multiple of {BLOCK}")
    codes = empty_codes(fmt, N, K, W.device) if codes is None else codes
    scales = empty_scales(N, K, W.device) if scales is None else scales
    _require_weights(fmt, codes, scales, N, K)
    _on_device(W, codes, scales)
    _check(load().qlinear_quantize(fmt, _ptr(W), N, K, _ptr(codes), _ptr(scales),
                                   _stream(stream)))
    return codes, scales


def _xdt(X):
    if X.dtype == torch.float32:
        return DT_F32
    if X.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        return DT_BF16
    raise TypeError(f"activations must be float32 or bfloat16, not {X.dtype}")


def forward(fmt, X, codes, scales, N, Y=None, stream=None):
    """Y [M][N] fp32 = X [M][K] . dequant(codes, scales)^T.  Asynchronous.
    FMT_F16: codes are the fp16 weights [N][K] (any 2-byte dtype), scales
    None."""
    M, K = _require_x(X)
    _require_weights(fmt, codes, scales, N, K)
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float32, device=X.device)
    _require_y(Y, M, N)
    _on_device(X, codes, scales, Y)
    _check(load().qlinear_forward(fmt, _ptr(X), _xdt(X), M, K, _ptr(codes), _ptr(scales), N,
                                  _ptr(Y), _stream(stream)))
    return Y


def _ydt(Y):
    if Y.dtype == torch.float32:
        return DT_F32
    if Y.dtype == torch.bfloat16:
        return DT_BF16
    raise TypeError(f"outputs must be float32 or bfloat16, not {Y.dtype}")


def _epilogue(Y, bias, act, residual, steer=None, ycopy=None):
    """steer: None, or (direction fp32 [N], hnorm float, strength: a device
    fp32 tensor of one element, re-read by every launch); ycopy: None, or a
    bf16 [M][N] tensor that receives a bf16 copy of the (fp32) output."""
    if steer is None:
        return _Epilogue(_ptr(bias), act, _ptr(residual), _ydt(Y), None, 0.0, None, _ptr(ycopy))
    d, hnorm, strength = steer
    return _Epilogue(_ptr(bias), act, _ptr(residual), _ydt(Y), _ptr(d), float(hnorm),
                     _ptr(strength), _ptr(ycopy))


def forward_ep(fmt, X, codes, scales, N, Y=None, bias=None, act=ACT_NONE, residual=None,
               ydtype=torch.float32, steer=None, stream=None, ycopy=None):
    """forward() with the layer epilogue fused into the output store:
    Y = act(X . W^T + bias) + residual (+ alpha * hnorm * d), Y fp32 or bf16
    (ydtype, or Y's dtype when Y is given).  bias fp32 [N], residual fp32
    [M][N] (may be Y itself for fp32 Y), each optional; steer = (d fp32 [N],
    hnorm, strength) adds the steering term with alpha = strength[0] read on
    the device by the launch (skipped exactly when alpha is 0); ycopy (bf16
    [M][N]) receives a bf16 copy of an fp32 Y.  Asynchronous."""
    M, K = _require_x(X)
    _require_weights(fmt, codes, scales, N, K)
    if Y is None:
        Y = torch.empty((M, N), dtype=ydtype, device=X.device)
    _require_y(Y, M, N, (torch.float32, torch.bfloat16))
    _require_ep(bias, residual, M, N)
    _require_steer(steer, N)
    _require_ycopy(ycopy, Y, M, N)
    ep = _epilogue(Y, bias, act, residual, steer, ycopy)
    _on_device(X, codes, scales, Y, bias, residual, ycopy, *(steer[::2] if steer else ()))
    _check(load().qlinear_forward_ep(fmt, _ptr(X), _xdt(X), M, K, _ptr(codes), _ptr(scales), N,
                                     _ptr(Y), ctypes.byref(ep), _stream(stream)))
    return Y


def make_group(entries):
    """ctypes array for block_forward from (fmt, X, codes, scales, N, Y) tuples.
    The array holds the device addresses of the tensors and keeps references
    to the tensors themselves, so they live as long as the array (a freed
    tensor's memory may be returned to the driver, e.g. when a graph capture
    empties torch's cache, and a later launch would then fault)."""
    if not 1 <= len(entries) <= MAX_GROUP:
        raise ValueError(f"a group holds 1 to {MAX_GROUP} linears, not {len(entries)}")
    arr = (_Linear * len(entries))()
    for i, (fmt, X, codes, scales, N, Y) in enumerate(entries):
        M, K = _require_x(X)
        _require_weights(fmt, codes, scales, N, K)
        _require_y(Y, M, N)
        _on_device(X, codes, scales, Y)
        arr[i] = _Linear(fmt, X.data_ptr(), _xdt(X), M, K, N, codes.data_ptr(),
                         scales.data_ptr() if scales is not None else 0, Y.data_ptr())
    arr._tensors = [tuple(e) for e in entries]
    return arr


def block_forward(entries, stream=None, group=None):
    """Grouped forward of up to 8 independent linears (one DiT block's QKV,
    out, FFN-up, FFN-down).  entries: (fmt, X, codes, scales, N, Y) tuples.
    Asynchronous.  A prepared `group` (make_group) skips re-marshalling."""
    arr = group if group is not None else make_group(entries)
    _check(load().qlinear_block_forward(arr, len(arr), _stream(stream)))
    return [e[5] for e in entries] if entries is not None else None


def make_group_ep(entries):
    """ctypes array for block_forward_ep from (fmt, X, codes, scales, N, Y,
    bias, act, residual[, steer[, ycopy]]) tuples (bias/residual/steer/ycopy
    None for none; Y fp32 or bf16; ycopy a bf16 [M][N] copy of an fp32 Y).
    The array keeps references to every tensor it points to (see
    make_group)."""
    if not 1 <= len(entries) <= MAX_GROUP:
        raise ValueError(f"a group holds 1 to {MAX_GROUP} linears, not {len(entries)}")
    arr = (_LinearEp * len(entries))()
    for i, e in enumerate(entries):
        fmt, X, codes, scales, N, Y, bias, act, residual = e[:9]
        steer = e[9] if len(e) > 9 else None
        ycopy = e[10] if len(e) > 10 else None
        M, K = _require_x(X)
        _require_weights(fmt, codes, scales, N, K)
        _require_y(Y, M, N, (torch.float32, torch.bfloat16))
        _require_ep(bias, residual, M, N)
        _require_steer(steer, N)
        _require_ycopy(ycopy, Y, M, N)
        _on_device(X, codes, scales, Y, bias, residual, ycopy, *(steer[::2] if steer else ()))
        lin = _Linear(fmt, X.data_ptr(), _xdt(X), M, K, N, codes.data_ptr(),
                      scales.data_ptr() if scales is not None else 0, Y.data_ptr())
        arr[i] = _LinearEp(lin, _epilogue(Y, bias, act, residual, steer, ycopy))
    arr._tensors = [tuple(e) for e in entries]
    return arr


def block_forward_ep(entries, stream=None, group=None):
    """block_forward with an epilogue per layer: entries are (fmt, X, codes,
    scales, N, Y, bias, act, residual) tuples.  Asynchronous."""
    arr = group if group is not None else make_group_ep(entries)
    _check(load().qlinear_block_forward_ep(arr, len(arr), _stream(stream)))
    return [e[5] for e in entries] if entries is not None else None


def block_forward_ep_noalloc(entries, stream=None, group=None):
    """block_forward_ep through the entry point that allocates nothing: its
    workspace is the library's static scratch (128 MiB per device).  Calls
    that may overlap on one device must be ordered by the caller.
    Asynchronous."""
    arr = group if group is not None else make_group_ep(entries)
    _check(load().qlinear_block_forward_ep_noalloc(arr, len(arr), _stream(stream)))
    return [e[5] for e in entries] if entries is not None else None


def quantize_act(X, qx=None, sx=None, stream=None):
    """Per-token int8 quantization of activations X [M][K] (fp32 or bf16):
    returns (qx int8 [M][K], sx fp16 bits as int16 [M]).  Asynchronous."""
    M, K = _require_x(X)
    if qx is None:
        qx = torch.empty((M, K), dtype=torch.int8, device=X.device)
    if sx is None:
        sx = torch.empty(M, dtype=torch.int16, device=X.device)
    _require(qx, "qx", (torch.int8,), (M, K))
    _require(sx, "sx", _TWO_BYTE, (M,))
    _on_device(X, qx, sx)
    _check(load().qlinear_quantize_act(_ptr(X), _xdt(X), M, K, _ptr(qx), _ptr(sx),
                                       _stream(stream)))
    return qx, sx


def forward_w8a8(qx, sx, codes, scales, N, Y=None, bias=None, act=ACT_NONE, residual=None,
                 ydtype=torch.float32, steer=None, stream=None):
    """W8A8 product of per-token int8 activations (quantize_act) and int8
    weights (quantize(FMT_INT8, ...)), with the layer epilogue (arguments as
    forward_ep).  Asynchronous."""
    _require(qx, "qx", (torch.int8,), (None, None))
    M, K = qx.shape
    _require(sx, "sx", _TWO_BYTE, (M,))
    _require_weights(FMT_INT8, codes, scales, N, K)
    if Y is None:
        Y = torch.empty((M, N), dtype=ydtype, device=qx.device)
    _require_y(Y, M, N, (torch.float32, torch.bfloat16))
    _require_ep(bias, residual, M, N)
    _require_steer(steer, N)
    ep = _epilogue(Y, bias, act, residual, steer)
    _on_device(qx, sx, codes, scales, Y, bias, residual, *(steer[::2] if steer else ()))
    _check(load().qlinear_forward_w8a8(_ptr(qx), _ptr(sx), M, K, _ptr(codes), _ptr(scales), N,
                                       _ptr(Y), ctypes.byref(ep), _stream(stream)))
    return Y


def steer(h, direction, hnorm, strength, stream=None):
    """h += alpha * hnorm * direction on every row, in place (Eq. 2), with
    alpha = strength[0] read on the device at run time (skipped exactly when
    alpha is 0).  Asynchronous."""
    _require(h, "h", (torch.float32,), (None, None))
    M, N = h.shape
    _require_steer((direction, hnorm, strength), N)
    _on_device(h, direction, strength)
    _check(load().qlinear_steer(_ptr(h), M, N, _ptr(direction), float(hnorm), _ptr(strength),
                                _stream(stream)))
    return h


def attention(q, k, v, B, T, H, dh=64, scale=None, O=None, odtype=torch.float32, stream=None):
    """Softmax self-attention over each sequence's T keys.  q, k, v: bf16 (or
    int16 bit patterns) 2-D row views [B*T][>= H*dh] with unit column stride
    (e.g. column slices of a fused QKV output).  Returns O [B*T][H*dh] fp32
    or bf16.  Asynchronous."""
    for name, t in (("q", q), ("k", k), ("v", v)):
        _require(t, name, _BF16_BITS, min_cols=H * dh)
        if t.shape[0] != B * T:
            raise ValueError(f"{name} has {t.shape[0]} rows, expected B * T = {B * T}")
    if O is None:
        O = torch.empty((B * T, H * dh), dtype=odtype, device=q.device)
    _require(O, "O", (torch.float32, torch.bfloat16), min_cols=H * dh)
    if O.shape[0] != B * T:
        raise ValueError(f"O has {O.shape[0]} rows, expected B * T = {B * T}")
    odt = DT_BF16 if O.dtype == torch.bfloat16 else DT_F32
    scale = 1.0 / float(dh) ** 0.5 if scale is None else scale
    _on_device(q, k, v, O)
    _check(load().qlinear_attention(_ptr(q), q.stride(0), _ptr(k), k.stride(0), _ptr(v),
                                    v.stride(0), B, T, H, dh, float(scale), _ptr(O),
                                    O.stride(0), odt, _stream(stream)))
    return O


class forced_path:
    """Context manager: every quantized forward call inside it runs on one
    kernel (PATH_GEMV, PATH_STREAM, PATH_SKINNY, PATH_TILED, PATH_WIDE or PATH_MID;
    qlinear_force_path).  Process-wide; restores automatic choice on exit."""

    def __init__(self, path):
        self.path = path

    def __enter__(self):
        _check(load().qlinear_force_path(self.path))
        return self

    def __exit__(self, *exc):
        _check(load().qlinear_force_path(PATH_AUTO))
        return False


class QuantizedLinear:
    """A linear layer's weight held only as codes + scales on the device.

    from_float() quantizes and keeps no full-precision copy: the compressed
    weight replaces the original (the caller drops its fp32 tensor).
    """

    def __init__(self, fmt, codes, scales, N, K):
        self.fmt, self.codes, self.scales, self.N, self.K = fmt, codes, scales, N, K

    @classmethod
    def from_float(cls, W, fmt):
        codes, scales = quantize(fmt, W)
        return cls(fmt, codes, scales, W.shape[0], W.shape[1])

    def __call__(self, X, Y=None, stream=None):
        return forward(self.fmt, X, self.codes, self.scales, self.N, Y, stream)
