"""Pins of the fp64 oracle against what the mathematics fixes (CPU only).

The paper prints no worked quantization example, so the oracle is pinned by
exact-rational rounding rules, brute force on small inputs, invariants of
the symmetric absmax block quantizer, constructions whose answer is known in
closed form, and agreement with library routines (numpy) on special cases.
"""
from fractions import Fraction

import numpy as np
import pytest

import exact
from oracle import oracle as O

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")

QMAX = {O.FMT_INT8: 127, O.FMT_Q4: 7}
FMTS = [O.FMT_INT8, O.FMT_Q4]


def decode_codes(fmt, codes, N, K):
    """Signed codes [N][K] from the stored bytes (numpy bit operations)."""
    if fmt == O.FMT_INT8:
        return codes.view(np.int8).astype(np.int64).reshape(N, K)
    lo = (codes & 0x0F).astype(np.int64)
    hi = (codes >> 4).astype(np.int64)
    out = np.empty((N, K), dtype=np.int64)
    out[:, 0::2] = lo
    out[:, 1::2] = hi
    return np.where(out >= 8, out - 16, out)


def f16_vals(bits):
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


# --------------------------------------------------------------------------
# fp64 -> fp16 conversion helper: exhaustive over the fp16 grid
# --------------------------------------------------------------------------

def test_f16_decode_all_patterns(orc):
    bits = np.arange(0, 0x10000, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([orc.f16_to_f64(int(b)) for b in bits])
    finite = np.isfinite(ref)
    assert np.array_equal(got[finite], ref[finite])
    assert np.array_equal(np.signbit(got[finite]), np.signbit(ref[finite]))
    assert np.all(np.isnan(got[np.isnan(ref)]))
    assert np.array_equal(got[np.isinf(ref)], ref[np.isinf(ref)])


def test_f16_encode_exact_values_roundtrip(orc):
    bits = np.concatenate([np.arange(0, 0x7C01), np.arange(0x8000, 0xFC01)]).astype(np.uint16)
    vals = bits.view(np.float16).astype(np.float64)
    got = np.array([orc.f64_to_f16(float(v)) for v in vals], dtype=np.uint16)
    assert np.array_equal(got, bits)


def test_f16_encode_midpoints_and_neighbours(orc):
    """Every midpoint between consecutive positive fp16 values (and the one
    past 65504) must tie to the even significand; one fp64 ulp either side
    must go to the nearer neighbour.  Checked against the exact grid search
    and against numpy's direct float64 -> float16 cast."""
    bits = np.arange(0, 0x7C00, dtype=np.uint16)
    lo = bits.view(np.float16).astype(np.float64)
    hi = np.append(lo[1:], 65536.0)
    mids = (lo + hi) / 2  # exact in fp64
    for v in list(mids) + list(np.nextafter(mids, 0)) + list(np.nextafter(mids, np.inf)):
        for sv in (v, -v):
            got = orc.f64_to_f16(float(sv))
            want = exact.f16_round_exact(Fraction(float(sv)))
            assert got == want, (sv, hex(got), hex(want))
    # numpy as a second witness on the same points
    pts = np.concatenate([mids, np.nextafter(mids, 0), np.nextafter(mids, np.inf)])
    ref = pts.astype(np.float16).view(np.uint16)
    got = np.array([orc.f64_to_f16(float(v)) for v in pts], dtype=np.uint16)
    assert np.array_equal(got, ref)


def test_f16_encode_special_values(orc):
    assert orc.f64_to_f16(65504.0) == 0x7BFF
    assert orc.f64_to_f16(65519.999) == 0x7BFF
    assert orc.f64_to_f16(65520.0) == 0x7C00
    assert orc.f64_to_f16(-1e300) == 0xFC00
    assert orc.f64_to_f16(float("inf")) == 0x7C00
    assert orc.f64_to_f16(2.0 ** -24) == 0x0001
    assert orc.f64_to_f16(2.0 ** -25) == 0x0000  # tie to even (0)
    assert orc.f64_to_f16(3 * 2.0 ** -25) == 0x0002  # tie between 1 and 2 quanta -> 2
    assert orc.f64_to_f16(-0.0) == 0x8000
    assert orc.f64_to_f16(1.0) == 0x3C00
    assert (orc.f64_to_f16(float("nan")) & 0x7C00) == 0x7C00
    assert (orc.f64_to_f16(float("nan")) & 0x03FF) != 0


def test_bf16_decode(orc):
    rng = np.random.default_rng(7)
    b = rng.integers(0, 0x10000, 5000).astype(np.uint16)
    ref = (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    got = np.array([orc.bf16_to_f64(int(x)) for x in b])
    fin = np.isfinite(ref)
    assert np.array_equal(got[fin], ref[fin])


# --------------------------------------------------------------------------
# quantizer: scales and codes against exact brute force
# --------------------------------------------------------------------------

def adversarial_blocks(Q):
    """Hand-built 32-wide blocks that stress each rule."""
    blocks = []
    z = np.zeros(32, np.float32)
    blocks.append(z.copy())                                 # all zero -> s = 0
    b = z.copy(); b[5] = 0.75; blocks.append(b)             # single non-zero
    b = z.copy(); b[0] = -0.5; b[31] = 0.5; blocks.append(b)  # +-absmax both signs
    b = np.full(32, -0.0, np.float32); b[3] = 1.0; blocks.append(b)  # negative zeros
    # exact .5 ties: with absmax = Q * 2^-4 (s = 2^-4 exactly) put w = (c + 1/2) s
    s = np.float32(2.0 ** -4)
    b = (np.arange(32) - 16 + 0.5).astype(np.float32) * s
    b = np.clip(b, -(Q - 0.5) * s, (Q - 0.5) * s)
    b[0] = Q * s
    blocks.append(b.astype(np.float32))
    # tiny block -> subnormal fp16 scale
    b = (np.linspace(-1, 1, 32) * 1e-6).astype(np.float32); blocks.append(b)
    # very tiny -> scale rounds to 0 even though the block is non-zero
    b = z.copy(); b[7] = 1e-9; blocks.append(b)
    # absmax/Q right below the fp16 overflow threshold
    b = z.copy(); b[9] = np.float32(65519.0 * Q); b[10] = -1.0; blocks.append(b)
    # largest finite scale exactly
    b = z.copy(); b[1] = np.float32(65504.0 * Q); blocks.append(b)
    # values that sit near half-integers after division by a non-power-of-2 scale
    rng = np.random.default_rng(11)
    b = (rng.standard_normal(32) * 0.3).astype(np.float32)
    s_bits = exact.block_scale_bits(b, Q)
    sv = float(exact.f16_value(s_bits))
    b[1:8] = ((np.arange(7) - 3 + 0.5) * sv).astype(np.float32)
    blocks.append(b)
    return blocks


def random_blocks(seed, nblocks, std):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((nblocks, 32)) * std).astype(np.float32)


@pytest.mark.parametrize("fmt", FMTS)
def test_scales_and_codes_bruteforce(orc, fmt):
    Q = QMAX[fmt]
    blocks = adversarial_blocks(Q) + list(random_blocks(fmt, 24, 0.02)) \
        + list(random_blocks(fmt + 1, 8, 3.0)) + list(random_blocks(fmt + 2, 8, 1e-5))
    W = np.stack(blocks).astype(np.float32)  # each block a row of K = 32
    N = W.shape[0]
    codes, scales = orc.quantize(fmt, W)
    C = decode_codes(fmt, codes, N, 32)
    cands = range(-Q, Q + 1) if fmt == O.FMT_Q4 else None
    for n in range(N):
        sb = exact.block_scale_bits(W[n], Q)
        assert int(scales[n, 0]) == sb, (n, hex(int(scales[n, 0])), hex(sb))
        s = exact.f16_value(sb)
        for k in range(32):
            if cands is not None or n < 14:
                want = exact.nearest_code(Fraction(float(W[n, k])), s, Q)
            else:  # int8 random rows: exact rounding of the exact quotient
                want = 0 if s == 0 else max(-Q, min(Q, round(Fraction(float(W[n, k])) / s)))
            assert C[n, k] == want, (n, k, W[n, k], C[n, k], want)


def test_half_integer_ties_go_to_even(orc):
    # s = 2^-4 exactly for int8 when absmax = 127 * 2^-4
    s = 2.0 ** -4
    w = np.zeros(32, np.float32)
    w[0] = 127 * s
    ties = [0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 99.5, 100.5, -126.5]
    for i, t in enumerate(ties):
        w[1 + i] = t * s
    codes, scales = orc.quantize(O.FMT_INT8, w[None, :])
    C = decode_codes(O.FMT_INT8, codes, 1, 32)[0]
    assert int(scales[0, 0]) == 0x2C00  # 2^-4
    assert list(C[1:1 + len(ties)]) == [0, 2, 2, 0, -2, -2, 100, 100, -126]


def test_q4_packing_layout(orc):
    """Byte j of a row holds code 2j (low nibble) and 2j+1 (high nibble)."""
    s = 2.0 ** -3
    want = [7, -1, 1, -7, 0, 3, -3, 2] + [0] * 24
    w = np.array(want, np.float32) * np.float32(s)
    codes, scales = orc.quantize(O.FMT_Q4, w[None, :])
    assert scales[0, 0] == 0x3000  # 2^-3
    b = codes[0]
    assert b[0] == (7 | (0xF << 4))      # 7, -1
    assert b[1] == (1 | (0x9 << 4))      # 1, -7
    assert b[2] == (0 | (3 << 4))        # 0, 3
    assert b[3] == (0xD | (2 << 4))      # -3, 2


# --------------------------------------------------------------------------
# invariants I1-I3 on DiT-like weights
# --------------------------------------------------------------------------

@pytest.mark.parametrize("fmt", FMTS)
def test_invariants_roundtrip_maxcode_idempotent(orc, fmt):
    Q = QMAX[fmt]
    rng = np.random.default_rng(100 + fmt)
    N, K = 96, 512
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    codes, scales = orc.quantize(fmt, W)
    C = decode_codes(fmt, codes, N, K)
    S = f16_vals(scales)
    assert np.all(np.abs(S) >= 2.0 ** -14)  # normal scales: invariants apply
    Srep = np.repeat(S, 32, axis=1)
    # I1: round-trip error at most half a scale (exact in fp64)
    err = np.abs(W.astype(np.float64) - C * Srep)
    assert np.all(err <= Srep / 2)
    # I3: every block holds a code of magnitude exactly Q
    assert np.all(np.abs(C).reshape(N, K // 32, 32).max(axis=2) == Q)
    # codes within [-Q, Q]
    assert np.all(np.abs(C) <= Q)
    # I2: re-quantizing the dequantized weights reproduces codes and scales
    Wd = orc.dequantize(fmt, codes, scales, N, K)
    assert np.array_equal(Wd.astype(np.float32).astype(np.float64), Wd)  # exact in fp32
    codes2, scales2 = orc.quantize(fmt, Wd.astype(np.float32))
    assert np.array_equal(codes2, codes)
    assert np.array_equal(scales2, scales)


# --------------------------------------------------------------------------
# closed forms: power-of-two weights and integer matmuls
# --------------------------------------------------------------------------

@pytest.mark.parametrize("fmt", FMTS)
def test_power_of_two_weights_exact(orc, fmt):
    """W = c * 2^-12 with one +-Q per block: s = 2^-12 and codes = c exactly,
    and Y for integer X is the exact dyadic X.C^T * 2^-12."""
    Q = QMAX[fmt]
    rng = np.random.default_rng(5 + fmt)
    N, K, M = 24, 256, 9
    C = rng.integers(-Q, Q + 1, (N, K))
    C.reshape(N, K // 32, 32)[:, :, 0] = rng.choice([-Q, Q], (N, K // 32))
    W = (C * 2.0 ** -12).astype(np.float32)
    codes, scales = orc.quantize(fmt, W)
    assert np.all(scales == 0x0C00)  # 2^-12
    assert np.array_equal(decode_codes(fmt, codes, N, K), C)
    Xi = rng.integers(-8, 9, (M, K))
    for xdt, X in ((O.DT_F32, Xi.astype(np.float32)),
                   (O.DT_BF16, (Xi.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16))):
        Y = orc.forward(fmt, X, xdt, codes, scales, N)
        want = (Xi @ C.T).astype(np.float64) * 2.0 ** -12
        assert np.array_equal(Y, want)


@pytest.mark.parametrize("fmt", FMTS)
def test_unit_scale_integer_matmul(orc, fmt):
    """Codes set by hand with s = 1.0: Y equals numpy's int64 matmul."""
    Q = QMAX[fmt]
    rng = np.random.default_rng(31 + fmt)
    M, N, K = 7, 13, 96
    C = rng.integers(-Q - 1, Q + 1, (N, K))  # includes -128 / -8 as stored codes
    if fmt == O.FMT_INT8:
        codes = C.astype(np.int8).view(np.uint8)
    else:
        u = (C & 0xF).astype(np.uint8)
        codes = (u[:, 0::2] | (u[:, 1::2] << 4)).astype(np.uint8)
    scales = np.full((N, K // 32), 0x3C00, np.uint16)
    Xi = rng.integers(-100, 101, (M, K))
    Y = orc.forward(fmt, Xi.astype(np.float32), O.DT_F32, codes, scales, N)
    assert np.array_equal(Y, (Xi @ C.T).astype(np.float64))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("xdt", [O.DT_F32, O.DT_BF16])
def test_forward_matches_dequantized_matmul(orc, fmt, xdt):
    import synth_inputs as si
    W, X = si.small_case(40 + fmt + xdt, 33, 70, 192, xdt)
    codes, scales = orc.quantize(fmt, W)
    Y = orc.forward(fmt, X, xdt, codes, scales, 70)
    Wd = orc.dequantize(fmt, codes, scales, 70, 192)
    Xd = X.astype(np.float64) if xdt == O.DT_F32 else si.bf16_bits_to_f32(X).astype(np.float64)
    ref = Xd @ Wd.T
    assert np.max(np.abs(Y - ref)) <= 1e-12 * np.max(np.abs(ref))
    # the dequantized weights themselves against the decoded codes x scales
    C = decode_codes(fmt, codes, 70, 192)
    assert np.array_equal(Wd, C * np.repeat(f16_vals(scales), 32, axis=1))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("K", [32, 64])
def test_forward_bruteforce_tiny(orc, fmt, K):
    import synth_inputs as si
    for xdt in (O.DT_F32, O.DT_BF16):
        W, X = si.small_case(70 + K + fmt + xdt, 3, 4, K, xdt)
        codes, scales = orc.quantize(fmt, W)
        C = decode_codes(fmt, codes, 4, K)
        Y = orc.forward(fmt, X, xdt, codes, scales, 4)
        Xf = X if xdt == O.DT_F32 else si.bf16_bits_to_f32(X)
        for m in range(3):
            for n in range(4):
                want = exact.dot_exact(Xf[m], C[n], scales[n])
                bound = sum(abs(Fraction(float(Xf[m, k])) * int(C[n, k])) for k in range(K))
                bound *= max(exact.f16_value(int(s)) for s in scales[n])
                assert abs(Fraction(Y[m, n]) - want) <= Fraction(1, 10 ** 15) * bound


def test_forward_rows_subset_matches_full(orc):
    import synth_inputs as si
    W, X = si.small_case(91, 20, 40, 128, O.DT_BF16)
    codes, scales = orc.quantize(O.FMT_Q4, W)
    full = orc.forward(O.FMT_Q4, X, O.DT_BF16, codes, scales, 40)
    rows = np.array([19, 0, 7, 7])
    part = orc.forward(O.FMT_Q4, X, O.DT_BF16, codes, scales, 40, rows=rows)
    assert np.array_equal(part, full[rows])


# --------------------------------------------------------------------------
# unquantized reference: fp16 weights (R6)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("xdt", [O.DT_F32, O.DT_BF16])
def test_forward_f16_integer_bruteforce(orc, xdt):
    """Small integers are exact in fp16, bf16 and fp32: the product is an
    integer matmul, checked against exact integer arithmetic (a transposed
    or mis-indexed operand fails on the non-square shapes)."""
    rng = np.random.default_rng(61 + xdt)
    M, N, K = 5, 7, 96
    Xi = rng.integers(-100, 101, (M, K))
    Wi = rng.integers(-2048, 2049, (N, K))
    W16 = Wi.astype(np.float16).view(np.uint16)
    X = Xi.astype(np.float32)
    if xdt == O.DT_BF16:
        import synth_inputs as si
        X = si.f32_to_bf16_bits(X)
    Y = orc.forward_f16(X, xdt, W16)
    assert np.array_equal(Y, (Xi @ Wi.T).astype(np.float64))
    rows = np.array([4, 0, 2])
    assert np.array_equal(orc.forward_f16(X, xdt, W16, rows=rows), Y[rows])


@pytest.mark.parametrize("fmt", FMTS)
def test_forward_f16_equals_quantized_at_power_of_two_scales(orc, fmt):
    """With power-of-two scales every dequantized weight c * s is exact in
    fp16, so the unquantized product of those fp16 weights must equal the
    quantized product (itself pinned above) exactly: both are sums of exact
    fp64 products well inside 53 bits."""
    import synth_inputs as si
    rng = np.random.default_rng(71 + fmt)
    Q = QMAX[fmt]
    M, N, K = 6, 9, 256
    C = rng.integers(-Q - 1, Q + 1, (N, K))
    e = rng.integers(-8, -5, (N, K // 32))
    scales = (np.float16(2.0) ** e.astype(np.float16)).astype(np.float16).view(np.uint16)
    if fmt == O.FMT_INT8:
        codes = C.astype(np.int8).view(np.uint8)
    else:
        u = (C & 0xF).astype(np.uint8)
        codes = (u[:, 0::2] | (u[:, 1::2] << 4)).astype(np.uint8)
    Wd = C * np.repeat(2.0 ** e, 32, axis=1)
    W16 = Wd.astype(np.float16)
    assert np.array_equal(W16.astype(np.float64), Wd)  # exact in fp16
    X = si.f32_to_bf16_bits(rng.standard_normal((M, K), dtype=np.float32))
    assert np.array_equal(orc.forward_f16(X, O.DT_BF16, W16.view(np.uint16)),
                          orc.forward(fmt, X, O.DT_BF16, codes, scales, N))


def test_forward_f16_subnormal_and_signed_zero_weights(orc):
    """fp16 subnormal weights decode exactly (2^-24 steps) and -0 adds
    nothing."""
    K = 64
    W16 = np.zeros((3, K), np.uint16)
    W16[0, :] = 0x0001            # 2^-24
    W16[1, :] = 0x83FF            # -(1023 * 2^-24), largest negative subnormal
    W16[2, :] = 0x8000            # -0
    X = np.ones((2, K), np.float32)
    X[1] = 2.0
    Y = orc.forward_f16(X, O.DT_F32, W16)
    assert np.array_equal(Y[:, 0], np.array([K, 2 * K]) * 2.0 ** -24)
    assert np.array_equal(Y[:, 1], -np.array([K, 2 * K]) * 1023 * 2.0 ** -24)
    assert np.array_equal(Y[:, 2], np.zeros(2))


# --------------------------------------------------------------------------
# epilogue (R7): act(P + bias) + residual
# --------------------------------------------------------------------------

def test_epilogue_gelu_normal_cdf_values(orc):
    """GELU(x) = x * Phi(x) at points where the standard normal CDF is a
    textbook value: Phi(0) = 1/2, Phi(1) = 0.8413447460685429,
    Phi(-1) = 0.15865525393145707, Phi(2) = 0.9772498680518208, and
    GELU(x) -> x (resp. 0) far in the right (left) tail."""
    x = np.array([[0.0, 1.0, -1.0, 2.0, 40.0, -40.0]])
    want = np.array([0.0, 0.8413447460685429, -0.15865525393145707,
                     2 * 0.9772498680518208, 40.0, 0.0])
    got = orc.epilogue(x, act=O.ACT_GELU)[0]
    assert np.allclose(got, want, rtol=2e-16, atol=1e-300)


def test_epilogue_bias_residual_exact_and_order(orc):
    """Bias indexed by output column, residual by the product's source row
    (a row subset), act between them: with act = GELU the result is
    GELU(P + b) + r, not GELU(P + b + r) and not GELU(P) + b + r."""
    rng = np.random.default_rng(81)
    M, N = 6, 5
    P = rng.integers(-50, 51, (M, N)).astype(np.float64)
    b = rng.integers(-50, 51, N).astype(np.float32)
    r = rng.integers(-50, 51, (M, N)).astype(np.float32)
    assert np.array_equal(orc.epilogue(P, bias=b, residual=r), P + b + r)
    rows = np.array([4, 1])
    assert np.array_equal(orc.epilogue(P[rows], bias=b, residual=r, rows=rows),
                          (P + b + r)[rows])
    # order: 1 + (-1) = 0 through GELU gives 0; then + residual
    P1 = np.array([[1.0]])
    got = orc.epilogue(P1, bias=np.float32([-1.0]), act=O.ACT_GELU,
                       residual=np.float32([[3.0]]))
    assert got[0, 0] == 3.0


# --------------------------------------------------------------------------
# attention (softmax over all keys of the same sequence)
# --------------------------------------------------------------------------

def bf16_exact(rng, shape, scale=1.0):
    """bf16 bit patterns of N(0, scale^2) draws, and their exact values."""
    bits = bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))
    return bits, bf16_vals(bits)


def test_attention_zero_queries_average_values(orc):
    """Q = 0: every score is 0, the weights are uniform and each output is
    the mean of its sequence's value rows (numpy's mean)."""
    rng = np.random.default_rng(91)
    B, T, H, dh = 2, 9, 3, 8
    Q = np.zeros((B * T, H * dh), np.uint16)
    K, _ = bf16_exact(rng, (B * T, H * dh))
    V, Vv = bf16_exact(rng, (B * T, H * dh))
    O = orc.attention(Q, K, V, B, T, H, dh)
    for b in range(B):
        want = Vv[b * T:(b + 1) * T].mean(axis=0)
        assert np.allclose(O[b * T:(b + 1) * T], want[None, :], rtol=0, atol=1e-15)


def test_attention_single_key_returns_its_value(orc):
    """T = 1: the only weight is 1 and the output is the value row itself,
    exactly."""
    rng = np.random.default_rng(92)
    Q, _ = bf16_exact(rng, (3, 16))
    K, _ = bf16_exact(rng, (3, 16))
    V, Vv = bf16_exact(rng, (3, 16))
    assert np.array_equal(orc.attention(Q, K, V, 3, 1, 2, 8), Vv)


def test_attention_two_keys_sigmoid(orc):
    """Two keys: the weights are the logistic function of the score
    difference, w1 = 1 / (1 + e^(s2 - s1))."""
    rng = np.random.default_rng(93)
    dh = 16
    Q, Qv = bf16_exact(rng, (2, dh))
    K, Kv = bf16_exact(rng, (2, dh))
    V, Vv = bf16_exact(rng, (2, dh))
    O = orc.attention(Q, K, V, 1, 2, 1, dh, scale=0.25)
    for t in range(2):
        s1, s2 = 0.25 * Qv[t] @ Kv[0], 0.25 * Qv[t] @ Kv[1]
        w1 = 1.0 / (1.0 + np.exp(s2 - s1))
        assert np.allclose(O[t], w1 * Vv[0] + (1 - w1) * Vv[1], rtol=1e-14, atol=1e-15)


def test_attention_dominant_key(orc):
    """A key whose score exceeds all others by more than 800 takes all the
    weight (e^-800 underflows): the output is exactly its value row."""
    rng = np.random.default_rng(94)
    T, dh = 6, 8
    Q = bf16_bits(np.full((T, dh), 4.0, np.float32))
    Kf = (rng.standard_normal((T, dh)) * 0.1).astype(np.float32)
    Kf[3] = 64.0
    K = bf16_bits(Kf)
    V, Vv = bf16_exact(rng, (T, dh))
    O = orc.attention(Q, K, V, 1, T, 1, dh, scale=1.0)
    assert np.array_equal(O, np.repeat(Vv[3:4], T, axis=0))


def test_attention_key_permutation_and_heads(orc):
    """Permuting the keys together with their values leaves the output
    unchanged (up to summation order), the batches do not mix, heads are
    independent, and a row subset is the same rows of the full result."""
    rng = np.random.default_rng(95)
    B, T, H, dh = 2, 12, 2, 8
    Q, _ = bf16_exact(rng, (B * T, H * dh))
    K, _ = bf16_exact(rng, (B * T, H * dh))
    V, _ = bf16_exact(rng, (B * T, H * dh))
    O = orc.attention(Q, K, V, B, T, H, dh)
    perm = np.concatenate([rng.permutation(T), T + rng.permutation(T)])
    assert np.allclose(orc.attention(Q, K[perm], V[perm], B, T, H, dh), O, rtol=1e-13, atol=1e-14)
    K2, V2 = K.copy(), V.copy()
    K2[T:], V2[T:] = bf16_exact(rng, (T, H * dh))[0], bf16_exact(rng, (T, H * dh))[0]
    assert np.array_equal(orc.attention(Q, K2, V2, B, T, H, dh)[:T], O[:T])
    K3 = K.copy()
    K3[:, dh:] = bf16_exact(rng, (B * T, dh))[0]
    O3 = orc.attention(Q, K3, V, B, T, H, dh)
    assert np.array_equal(O3[:, :dh], O[:, :dh]) and not np.allclose(O3[:, dh:], O[:, dh:])
    rows = np.array([23, 0, 11, 12])
    assert np.array_equal(orc.attention(Q, K, V, B, T, H, dh, rows=rows), O[rows])


# --------------------------------------------------------------------------
# steering: additive injection (Eq. 2)
# --------------------------------------------------------------------------

def unit_direction(rng, N):
    d = rng.standard_normal(N)
    return (d / np.linalg.norm(d)).astype(np.float32)


def test_steer_zero_strength_is_identity(orc):
    """alpha = 0 leaves every value bit for bit, -0.0 and NaN included."""
    rng = np.random.default_rng(71)
    Y = rng.standard_normal((5, 16))
    Y[0, 0], Y[1, 1] = -0.0, np.nan
    out = orc.steer(Y, unit_direction(rng, 16), 3.5, 0.0)
    assert np.array_equal(out.view(np.uint64), Y.view(np.uint64))


def test_steer_rank_one_shift(orc):
    """Every row moves by the same vector, of length alpha * ||h_bar|| along
    the unit direction d (cosine 1), and the shift is linear in alpha
    (dyadic strengths: exact)."""
    rng = np.random.default_rng(72)
    N = 64
    d = unit_direction(rng, N)
    Y = rng.standard_normal((7, N))
    hnorm = 12.5
    for alpha in (0.25, 0.5, 1.0):
        shift = orc.steer(np.zeros_like(Y), d, hnorm, alpha)
        assert np.all(shift == shift[0])
        assert abs(np.linalg.norm(shift[0]) - alpha * hnorm * np.linalg.norm(d.astype(np.float64))) \
            <= 1e-13 * alpha * hnorm
        cosv = shift[0] @ d.astype(np.float64) / np.linalg.norm(shift[0]) / np.linalg.norm(
            d.astype(np.float64))
        assert abs(cosv - 1.0) < 1e-15
        assert np.array_equal(orc.steer(Y, d, hnorm, alpha), Y + shift)
    s1 = orc.steer(np.zeros((1, N)), d, hnorm, 0.25)
    s2 = orc.steer(np.zeros((1, N)), d, hnorm, 0.5)
    assert np.array_equal(2 * s1, s2)


# --------------------------------------------------------------------------
# W8A8: per-token int8 activations against int8 weights
# --------------------------------------------------------------------------

def bf16_bits(x):
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def bf16_vals(bits):
    return (np.asarray(bits, dtype=np.uint32) << 16).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("xdt", [O.DT_F32, O.DT_BF16])
def test_act_quant_bruteforce(orc, xdt):
    """Per-token scale = the fp16 nearest to the exact row absmax / 127 (grid
    search in rationals), codes = the nearest multiple of the scale among
    -127..127 (all candidates tried), ties to even; rows with exact .5 ties,
    a zero row, a row of one huge and many tiny values."""
    rng = np.random.default_rng(61)
    M, K = 6, 64
    Xf = rng.standard_normal((M, K)).astype(np.float32)
    Xf[1] = 0.0
    Xf[2] = np.float32(1e-6) * rng.standard_normal(K).astype(np.float32)
    Xf[2, 5] = np.float32(300.0)
    Xf[3, :4] = [127.0, 0.5, 1.5, -2.5]  # scale 1: exact ties
    Xf[3, 4:] = np.clip(Xf[3, 4:], -100, 100)
    X = Xf if xdt == O.DT_F32 else bf16_bits(Xf)
    vals = Xf.astype(np.float64) if xdt == O.DT_F32 else bf16_vals(X)
    q, sx = orc.quantize_act(X, xdt)
    for m in range(M):
        sb = exact.block_scale_bits(vals[m], 127)
        assert sx[m] == sb, (m, sx[m], sb)
        sv = exact.f16_value(sb)
        for k in range(K):
            assert q[m, k] == exact.nearest_code(vals[m, k], sv, 127), (m, k)
    assert np.all(q[1] == 0) and sx[1] == 0
    assert list(q[3, :4]) == [127, 0, 2, -2]


def test_act_quant_equals_weight_quantizer_one_block(orc):
    """With K = 32 a row is one block: the per-token activation quantizer and
    the (separately pinned) int8 weight quantizer give the same codes and
    scales."""
    rng = np.random.default_rng(62)
    X = (rng.standard_normal((40, 32)) * 10.0 ** rng.integers(-3, 4, (40, 1))).astype(np.float32)
    q, sx = orc.quantize_act(X, O.DT_F32)
    c, s = orc.quantize(O.FMT_INT8, X)
    assert np.array_equal(q.view(np.uint8), c)
    assert np.array_equal(sx, s[:, 0])


def test_act_quant_invariants(orc):
    """DiT-like activation rows (bf16, K = 2048): |x - s q| <= s / 2, every
    row reaches +-127, and re-quantizing the dequantized rows is the
    identity."""
    rng = np.random.default_rng(63)
    Xf = (rng.standard_normal((16, 2048)) * rng.uniform(0.1, 10, (16, 1))).astype(np.float32)
    X = bf16_bits(Xf)
    q, sx = orc.quantize_act(X, O.DT_BF16)
    s = f16_vals(sx)[:, None]
    x = bf16_vals(X)
    assert np.all(np.abs(x - s * q) <= s / 2)
    assert np.all(np.max(np.abs(q.astype(np.int64)), axis=1) == 127)
    q2, s2 = orc.quantize_act((s * q).astype(np.float32), O.DT_F32)
    assert np.array_equal(q2, q) and np.array_equal(s2, sx)


def test_act_quant_range_errors(orc):
    X = np.ones((3, 64), np.float32)
    for bad in (np.nan, np.inf, 65520.0 * 127):
        Xb = X.copy()
        Xb[1, 7] = bad
        with pytest.raises(O.OracleError):
            orc.quantize_act(Xb, O.DT_F32)


def test_forward_w8a8_integer_exact(orc):
    """Integer activations whose row absmax is 127 (scale 1, codes = X) and
    W = c * 2^-12 with +-127 in every block (scale 2^-12, codes = c): Y is
    the exact integer matmul times 2^-12."""
    rng = np.random.default_rng(64)
    M, N, K = 9, 7, 256
    Xi = rng.integers(-127, 128, (M, K))
    Xi[:, 3] = 127
    C = rng.integers(-127, 128, (N, K))
    C.reshape(N, K // 32, 32)[:, :, 0] = 127
    q, sx = orc.quantize_act(Xi.astype(np.float32), O.DT_F32)
    assert np.array_equal(q, Xi) and np.all(sx == 0x3C00)
    codes, scales = orc.quantize(O.FMT_INT8, (C * 2.0 ** -12).astype(np.float32))
    Y = orc.forward_w8a8(q, sx, codes, scales, N)
    assert np.array_equal(Y, (Xi @ C.T).astype(np.float64) * 2.0 ** -12)


def test_forward_w8a8_matches_dequantized_matmul(orc):
    """Y against numpy's fp64 matmul of the dequantized activations and
    weights, (s_x q)(s_w c)^T; and the row-subset form."""
    rng = np.random.default_rng(65)
    M, N, K = 20, 33, 320
    X = bf16_bits(rng.standard_normal((M, K)).astype(np.float32))
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    q, sx = orc.quantize_act(X, O.DT_BF16)
    codes, scales = orc.quantize(O.FMT_INT8, W)
    Xd = f16_vals(sx)[:, None] * q.astype(np.float64)
    Wd = orc.dequantize(O.FMT_INT8, codes, scales, N, K)
    ref = Xd @ Wd.T
    Y = orc.forward_w8a8(q, sx, codes, scales, N)
    assert np.max(np.abs(Y - ref)) <= 1e-12 * np.max(np.abs(ref))
    rows = np.array([19, 0, 7])
    assert np.array_equal(orc.forward_w8a8(q, sx, codes, scales, N, rows=rows), Y[rows])


def test_forward_w8a8_exact_rationals_tiny(orc):
    """Tiny shapes in exact rationals: s_x * sum_b s_b * sum_k q c."""
    rng = np.random.default_rng(66)
    M, N, K = 2, 3, 64
    X = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((N, K)) * 0.05).astype(np.float32)
    q, sx = orc.quantize_act(X, O.DT_F32)
    codes, scales = orc.quantize(O.FMT_INT8, W)
    c = codes.view(np.int8)
    Y = orc.forward_w8a8(q, sx, codes, scales, N)
    for m in range(M):
        for n in range(N):
            want = exact.f16_value(sx[m]) * exact.dot_exact(q[m], c[n], scales[n])
            assert abs(Fraction(Y[m, n]) - want) <= abs(want) * Fraction(1, 2 ** 50)


# --------------------------------------------------------------------------
# error conventions
# --------------------------------------------------------------------------

@pytest.mark.parametrize("fmt", FMTS)
def test_range_errors(orc, fmt):
    Q = QMAX[fmt]
    base = np.zeros((2, 64), np.float32)
    for bad in (np.nan, np.inf, -np.inf):
        W = base.copy(); W[1, 40] = bad
        assert orc.quantize_status(fmt, W) == O.ERR_RANGE
    W = base.copy(); W[0, 3] = np.float32(65520.0 * Q)   # scale rounds to inf
    assert orc.quantize_status(fmt, W) == O.ERR_RANGE
    W = base.copy(); W[0, 3] = np.float32(65504.0 * Q)   # largest finite scale: fine
    assert orc.quantize_status(fmt, W) == O.OK


def test_shape_errors(orc):
    assert orc.quantize_status(O.FMT_INT8, np.zeros((2, 48), np.float32)) == O.ERR_SHAPE
    assert orc.quantize_status(3, np.zeros((2, 64), np.float32)) == O.ERR_INVALID
