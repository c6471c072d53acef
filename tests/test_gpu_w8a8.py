"""GPU parity of the W8A8 path (qlinear_quantize_act, qlinear_forward_w8a8)
against the oracle.

Activation codes and scales must match the oracle bit for bit.  Outputs
from the same codes: each block's integer sum is exact on both sides, and
the GPU folds the blocks into an fp32 accumulator (one rounding per block)
and multiplies by the row scale (one more), so element by element
|Y_gpu - Y_ref| <= (K/32 + 1) * 2^-24 * (|X_d| |W_d|^T)[m][n], with X_d, W_d
the dequantized operands; exact constructions must match exactly.
"""
import numpy as np
import pytest

import synth_inputs as si
from oracle import oracle as O

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU (run with -m 'not gpu' on a CPU host)")
    from paper_2607_08526_amd import qlinear as ql
    ql.load()
    return torch, ql


def dev(torch, A, dtype=np.float32):
    A = np.ascontiguousarray(A, dtype=dtype)
    if dtype == np.uint16:
        A = A.view(np.int16)
    return torch.from_numpy(A).cuda()


def f16(bits):
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def quant_act_gpu(gpu, X, xdt):
    torch, ql = gpu
    Xd = dev(torch, X, np.float32 if xdt == O.DT_F32 else np.uint16)
    q, s = ql.quantize_act(Xd)
    torch.cuda.synchronize()
    return q.cpu().numpy(), s.cpu().numpy().view(np.uint16)


def forward_gpu(gpu, q, s, codes, scales, N, **ep):
    torch, ql = gpu
    Y = ql.forward_w8a8(dev(torch, q, np.int8), dev(torch, s, np.uint16),
                        dev(torch, codes, np.uint8), dev(torch, scales, np.uint16), N, **ep)
    torch.cuda.synchronize()
    return Y.float().cpu().numpy().astype(np.float64)


def bound(orc, q, s, codes, scales, N):
    K = q.shape[1]
    Xd = np.abs(f16(s)[:, None] * q.astype(np.float64))
    Wd = np.abs(orc.dequantize(O.FMT_INT8, codes, scales, N, K))
    return (K // 32 + 1) * 2.0 ** -24 * (Xd @ Wd.T) + 1e-30


@pytest.mark.parametrize("xdt", [O.DT_BF16, O.DT_F32])
def test_quantize_act_bitexact(gpu, orc, xdt):
    """Rows of 32 to 8192 activations, ragged row counts, with exact .5
    ties, zero rows, one huge value among tiny ones, wide magnitude ranges."""
    rng = np.random.default_rng(7000 + xdt)
    for M, K in ((1, 32), (7, 96), (33, 2048), (130, 8192), (3, 8224)):
        Xf = (rng.standard_normal((M, K)) * 10.0 ** rng.integers(-4, 5, (M, 1))).astype(np.float32)
        if M > 2:
            Xf[1] = 0.0
            Xf[2, :4] = [127.0, 0.5, -2.5, 3.5]
            Xf[2, 4:] = np.clip(Xf[2, 4:], -100.0, 100.0)
        X = Xf if xdt == O.DT_F32 else si.f32_to_bf16_bits(Xf)
        qg, sg = quant_act_gpu(gpu, X, xdt)
        qr, sr = orc.quantize_act(X, xdt)
        assert np.array_equal(sg, sr), (M, K, np.argwhere(sg != sr)[:4])
        assert np.array_equal(qg, qr), (M, K, np.argwhere(qg != qr)[:4])


def test_quantize_act_bad_rows(gpu, orc):
    """A row with a NaN or Inf, or whose scale would overflow fp16, gets the
    NaN scale and zero codes; the other rows are untouched."""
    rng = np.random.default_rng(7010)
    X = rng.standard_normal((5, 64)).astype(np.float32)
    X[1, 3] = np.nan
    X[2, 60] = -np.inf
    X[3, 0] = 65520.0 * 127
    qg, sg = quant_act_gpu(gpu, X, O.DT_F32)
    for m in (1, 2, 3):
        assert sg[m] == 0x7E00 and np.all(qg[m] == 0)
    qr, sr = orc.quantize_act(X[[0, 4]], O.DT_F32)
    assert np.array_equal(qg[[0, 4]], qr) and np.array_equal(sg[[0, 4]], sr)


@pytest.mark.parametrize("M,N,K", [(1, 1, 32), (5, 17, 96), (64, 128, 64), (127, 200, 320),
                                   (129, 130, 2048), (300, 520, 1024), (40, 77, 8192)])
def test_forward_w8a8_ragged(gpu, orc, M, N, K):
    """Row and column counts around the 128 x 128 tile, K with an odd number
    of 32-blocks (a half-filled last stage), long K."""
    W, X = si.small_case(7100 + M + N + K, M, N, K)
    codes, scales = orc.quantize(O.FMT_INT8, W)
    q, s = orc.quantize_act(X, O.DT_BF16)
    Yg = forward_gpu(gpu, q, s, codes, scales, N)
    Yr = orc.forward_w8a8(q, s, codes, scales, N)
    B = bound(orc, q, s, codes, scales, N)
    bad = np.abs(Yg - Yr) > B
    assert not bad.any(), (np.argwhere(bad)[:4], Yg[bad][:4], Yr[bad][:4])
    assert np.array_equal(Yg, forward_gpu(gpu, q, s, codes, scales, N))


def test_forward_w8a8_integer_exact(gpu, orc):
    """Integer activations with row absmax 127 and W = c * 2^-12: the
    product is an exact integer matmul times 2^-12."""
    rng = np.random.default_rng(7200)
    M, N, K = 150, 140, 512
    Xi = rng.integers(-127, 128, (M, K))
    Xi[:, 5] = -127
    C = rng.integers(-127, 128, (N, K))
    C.reshape(N, K // 32, 32)[:, :, 1] = -127
    q, s = quant_act_gpu(gpu, si.f32_to_bf16_bits(Xi.astype(np.float32)), O.DT_BF16)
    assert np.array_equal(q, Xi) and np.all(s == 0x3C00)
    codes, scales = orc.quantize(O.FMT_INT8, (C * 2.0 ** -12).astype(np.float32))
    Yg = forward_gpu(gpu, q, s, codes, scales, N)
    assert np.array_equal(Yg, (Xi @ C.T).astype(np.float64) * 2.0 ** -12)


def test_forward_w8a8_epilogue_and_nan_rows(gpu, orc):
    """The layer epilogue applies to the W8A8 product (bias, GELU, residual,
    bf16 outputs), and a row with the NaN scale comes out NaN."""
    torch, ql = gpu
    M, N, K = 70, 96, 256
    W, X = si.small_case(7300, M, N, K)
    codes, scales = orc.quantize(O.FMT_INT8, W)
    q, s = orc.quantize_act(X, O.DT_BF16)
    rng = np.random.default_rng(7301)
    bias = (rng.standard_normal(N) * 0.5).astype(np.float32)
    resid = rng.standard_normal((M, N)).astype(np.float32)
    P = orc.forward_w8a8(q, s, codes, scales, N)
    B = bound(orc, q, s, codes, scales, N)
    for act, yd in ((O.ACT_GELU, torch.float32), (O.ACT_GELU, torch.bfloat16)):
        Yg = forward_gpu(gpu, q, s, codes, scales, N, bias=dev(torch, bias), act=act,
                         residual=dev(torch, resid), ydtype=yd)
        Yr = orc.epilogue(P, bias, act, resid)
        lim = 1.13 * B + 1e-6 * (np.abs(Yr) + np.max(np.abs(P)) + np.max(np.abs(bias)))
        if yd == torch.bfloat16:
            lim = lim + 2.0 ** -8 * np.abs(Yr)
        assert np.all(np.abs(Yg - Yr) <= lim), yd
    s2 = s.copy()
    s2[3] = 0x7E00
    Yg = forward_gpu(gpu, q, s2, codes, scales, N)
    assert np.all(np.isnan(Yg[3])) and not np.isnan(np.delete(Yg, 3, axis=0)).any()


def test_forward_w8a8_block_shapes_sampled(gpu, orc):
    """One DiT block's four linears at full size (2048 tokens, d = 2048):
    GPU activation quantization and product, checked on sampled rows."""
    torch, ql = gpu
    xa, xb = si.block_activations()
    rows = np.array([0, 1, 777, 1500, 2047])
    for i, (_, N, K) in enumerate(si.block_linears()):
        X = xb if K == xb.shape[1] else xa
        W = si.block_weights(i, 7400)
        cd, sd = ql.quantize(ql.FMT_INT8, dev(torch, W))
        qd, sxd = ql.quantize_act(dev(torch, X, np.uint16))
        Y = ql.forward_w8a8(qd, sxd, cd, sd, N)
        torch.cuda.synchronize()
        q, s = orc.quantize_act(X[rows], O.DT_BF16)
        assert np.array_equal(qd.cpu().numpy()[rows], q)
        assert np.array_equal(sxd.cpu().numpy().view(np.uint16)[rows], s)
        codes, scales = cd.cpu().numpy().view(np.uint8), sd.cpu().numpy().view(np.uint16)
        Yr = orc.forward_w8a8(q, s, codes, scales, N)
        B = bound(orc, q, s, codes, scales, N)
        assert np.all(np.abs(Y.cpu().numpy()[rows].astype(np.float64) - Yr) <= B), i
