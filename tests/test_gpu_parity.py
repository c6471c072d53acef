"""GPU parity: the HIP library (through its C ABI) against the fp64 oracle.

Codes and scales must match the oracle bit for bit.  Outputs must satisfy
max |Y_gpu - Y_ref| / max |Y_ref| <= 2e-3 for bf16 activations and <= 1e-5
for fp32 activations (Y_ref the fp64 oracle result); constructions whose
exact answer is representable must match exactly.
"""
import numpy as np
import pytest

import synth_inputs as si
from oracle import oracle as O

pytestmark = pytest.mark.gpu

TOL = {O.DT_BF16: 2e-3, O.DT_F32: 1e-5}
QMAX = {O.FMT_INT8: 127, O.FMT_Q4: 7}


@pytest.fixture(scope="module")
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU (run with -m 'not gpu' on a CPU host)")
    from paper_2607_08526_amd import qlinear as ql
    ql.load()
    return torch, ql


def dev_w(torch, W):
    return torch.from_numpy(np.ascontiguousarray(W, dtype=np.float32)).cuda()


def dev_x(torch, X, xdt):
    if xdt == O.DT_F32:
        return torch.from_numpy(np.ascontiguousarray(X, dtype=np.float32)).cuda()
    return torch.from_numpy(np.ascontiguousarray(X, dtype=np.uint16).view(np.int16)).cuda()


def host_codes(c):
    return c.cpu().numpy().astype(np.uint8)


def host_scales(s):
    return s.cpu().numpy().view(np.uint16)


def rel_err(Yg, Yr):
    return float(np.max(np.abs(Yg.astype(np.float64) - Yr)) / np.max(np.abs(Yr)))


def quantize_both(gpu, orc, fmt, W):
    torch, ql = gpu
    cg, sg = ql.quantize(fmt, dev_w(torch, W))
    cr, sr = orc.quantize(fmt, W)
    cg, sg = host_codes(cg), host_scales(sg)
    assert np.array_equal(sg, sr), f"scales differ at {np.argwhere(sg != sr)[:5]}"
    assert np.array_equal(cg, cr), f"codes differ at {np.argwhere(cg != cr)[:5]}"
    return cr, sr


def forward_gpu(gpu, fmt, X, xdt, codes, scales, N):
    torch, ql = gpu
    cd = torch.from_numpy(codes).cuda()
    sd = torch.from_numpy(scales.view(np.int16)).cuda()
    Y = ql.forward(fmt, dev_x(torch, X, xdt), cd, sd, N)
    torch.cuda.synchronize()
    return Y.cpu().numpy()


# --------------------------------------------------------------------------
# quantizer: bit-exact
# --------------------------------------------------------------------------

@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
@pytest.mark.parametrize("N,K", [(1, 32), (3, 96), (70, 320), (257, 1024)])
def test_quantize_bitexact_small(gpu, orc, fmt, N, K):
    W, _ = si.small_case(N * 7 + K + fmt, 1, N, K)
    quantize_both(gpu, orc, fmt, W)


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_quantize_bitexact_adversarial(gpu, orc, fmt):
    import test_oracle_pins as pins
    blocks = pins.adversarial_blocks(QMAX[fmt])
    blocks += list(pins.random_blocks(fmt + 1, 64, 3.0)) + list(pins.random_blocks(fmt + 2, 64, 1e-5))
    W = np.stack(blocks).astype(np.float32).reshape(-1, 64)  # two blocks per row
    quantize_both(gpu, orc, fmt, W)


@pytest.mark.parametrize("name", ["single_int8", "single_q4"])
def test_quantize_bitexact_single_configs(gpu, orc, name):
    cfg = getattr(si, name)()
    quantize_both(gpu, orc, cfg["fmt"], cfg["W"])


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_quantize_range_errors(gpu, fmt):
    torch, ql = gpu
    W = np.zeros((4, 64), np.float32)
    for bad in (np.nan, np.inf):
        Wb = W.copy(); Wb[2, 33] = bad
        with pytest.raises(ql.QLinearError) as e:
            ql.quantize(fmt, dev_w(torch, Wb))
        assert e.value.status == 4
    Wb = W.copy(); Wb[1, 0] = np.float32(65520.0 * QMAX[fmt])
    with pytest.raises(ql.QLinearError) as e:
        ql.quantize(fmt, dev_w(torch, Wb))
    assert e.value.status == 4
    Wb = W.copy(); Wb[1, 0] = np.float32(65504.0 * QMAX[fmt])
    ql.quantize(fmt, dev_w(torch, Wb))  # the largest finite scale is fine


# --------------------------------------------------------------------------
# forward: ragged shapes across every tile configuration
# --------------------------------------------------------------------------

MS = [1, 2, 15, 16, 17, 33, 64, 65, 127, 130, 257]
NKS = [(16, 32), (70, 96), (200, 320)]


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
@pytest.mark.parametrize("xdt", [O.DT_BF16, O.DT_F32])
@pytest.mark.parametrize("N,K", NKS)
def test_forward_ragged(gpu, orc, fmt, xdt, N, K):
    for M in MS:
        W, X = si.small_case(1000 + M + N + K + fmt + xdt, M, N, K, xdt)
        codes, scales = quantize_both(gpu, orc, fmt, W)
        Yg = forward_gpu(gpu, fmt, X, xdt, codes, scales, N)
        Yr = orc.forward(fmt, X, xdt, codes, scales, N)
        e = rel_err(Yg, Yr)
        assert e <= TOL[xdt], (M, N, K, e)


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_forward_large_m_ragged_tiles(gpu, orc, fmt):
    """The large-M bf16 path (M > 64, K % 256 == 0) at row and column counts
    that leave partial 128 x 256 tiles, several K steps (odd and even ring
    positions) and one-step K."""
    for (M, N, K) in ((65, 200, 512), (130, 256, 768), (257, 300, 256), (300, 520, 1280),
                      (129, 17, 1024)):
        W, X = si.small_case(70 + M + N + K + fmt, M, N, K)
        codes, scales = quantize_both(gpu, orc, fmt, W)
        Yg = forward_gpu(gpu, fmt, X, O.DT_BF16, codes, scales, N)
        Yr = orc.forward(fmt, X, O.DT_BF16, codes, scales, N)
        e = rel_err(Yg, Yr)
        assert e <= TOL[O.DT_BF16], (M, N, K, e)


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_forward_mid_m(gpu, orc, fmt):
    """The mid-M exact kernel (32 < M <= 256, K % 256 == 0): partial
    128 x 128 tiles in both directions (a single row tile below 65 rows),
    one-chunk and long reductions, K
    parts summed by a second launch (up to 16 parts), the paper's 214-token
    rows and the 256-row single-layer workload's shape.  Exact per-block
    form: within 1e-5 of the oracle; every output written (Y starts as NaN);
    results repeat bit for bit."""
    torch, ql = gpu
    cases = [(65, 130, 256), (100, 129, 8192), (128, 2048, 2048), (129, 300, 1024),
             (200, 1000, 4096), (214, 1027, 1536), (256, 6144, 1536), (97, 8192, 512),
             (33, 520, 2048), (48, 2049, 8192), (64, 300, 768)]
    for M, N, K in cases:
        W, X = si.small_case(90 + M + N + K + fmt, M, N, K)
        codes, scales = quantize_both(gpu, orc, fmt, W)
        cd = torch.from_numpy(codes).cuda()
        sd = torch.from_numpy(scales.view(np.int16)).cuda()
        xd = dev_x(torch, X, O.DT_BF16)
        outs = []
        for _ in range(2):
            Y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
            ql.forward(fmt, xd, cd, sd, N, Y)
            torch.cuda.synchronize()
            outs.append(Y.cpu().numpy())
        assert np.isfinite(outs[0]).all(), (M, N, K)
        Yr = orc.forward(fmt, X, O.DT_BF16, codes, scales, N)
        e = rel_err(outs[0], Yr)
        assert e <= 1e-5, (M, N, K, e)
        assert np.array_equal(outs[0], outs[1]), (M, N, K)


def test_mid_split_graph_replay(gpu, orc):
    """The mid-M path's K parts, whose partial outputs pass through the
    stream's workspace to the sum launch: a captured call replayed several
    times, with and without other calls in between that overwrite that
    workspace (a large-M call, a mid-M call with 16 parts), equals the eager
    result bit for bit every time."""
    torch, ql = gpu
    fmt = O.FMT_Q4
    shapes = {"mid": (128, 2048, 2048), "wide": (640, 1024, 4096), "ext": (100, 129, 8192)}
    data = {}
    for name, (M, N, K) in shapes.items():
        W, X = si.small_case(500 + M + N + K, M, N, K)
        codes, scales = orc.quantize(fmt, W)
        data[name] = (dev_x(torch, X, O.DT_BF16), torch.from_numpy(codes).cuda(),
                      torch.from_numpy(scales.view(np.int16)).cuda(), N,
                      torch.empty((M, N), dtype=torch.float32, device="cuda"), (X, codes, scales))

    def run(name):
        xd, cd, sd, N, Y, _ = data[name]
        ql.forward(fmt, xd, cd, sd, N, Y)

    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        run("wide")  # sizes the workspace beyond the mid call's needs
        run("mid")
    s.synchronize()
    ref = data["mid"][4].clone()
    X, codes, scales = data["mid"][5]
    assert rel_err(ref.cpu().numpy(), orc.forward(fmt, X, O.DT_BF16, codes, scales, 2048)) <= 1e-5
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        run("mid")
    for rep in range(4):
        data["mid"][4].fill_(float("nan"))
        if rep % 2 == 1:
            with torch.cuda.stream(s):
                run("wide" if rep == 1 else "ext")
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            g.replay()
        s.synchronize()
        assert torch.equal(data["mid"][4], ref), rep


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_forward_streaming_ragged(gpu, orc, fmt):
    """The weight-streaming path (M <= 32, K % 256 == 0; M <= 4 goes to the
    GEMV when it fits): row counts around its 8- to 64-row workgroups,
    K lengths that leave some wavefronts or K parts short or empty and that
    cross the 32-block scale runs, activation stages of 8, 16 and 32 rows,
    and long reductions cut into K parts summed by a second launch (results
    repeat bit for bit)."""
    cases = [(1, 1, 256), (2, 7, 512), (3, 9, 768), (4, 16, 2304), (5, 17, 256),
             (8, 100, 1280), (15, 300, 2048), (16, 4100, 512), (16, 4111, 1024),
             (1, 5000, 8448), (9, 4096, 256), (6, 4097, 768), (17, 300, 2048),
             (24, 4100, 1024), (32, 513, 2304), (31, 2048, 8192), (20, 7, 256),
             (32, 4096, 256), (32, 100, 8192), (12, 777, 4352), (29, 65, 12288),
             (8, 2049, 8192)]
    for M, N, K in cases:
        W, X = si.small_case(80 + M + N + K + fmt, M, N, K)
        codes, scales = quantize_both(gpu, orc, fmt, W)
        Yg = forward_gpu(gpu, fmt, X, O.DT_BF16, codes, scales, N)
        Yr = orc.forward(fmt, X, O.DT_BF16, codes, scales, N)
        e = rel_err(Yg, Yr)
        assert e <= TOL[O.DT_BF16], (M, N, K, e)
        if K >= 4096:
            assert np.array_equal(Yg, forward_gpu(gpu, fmt, X, O.DT_BF16, codes, scales, N))


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_forward_gemv_shapes(gpu, orc, fmt):
    """The wavefront-reduction GEMV (M <= 4, K % 256 == 0, K <= 8192): every
    M, lanes with one to four blocks and with a ragged last block round
    (K / 32 not a multiple of 64), row counts that leave wavefronts of the
    last workgroup without rows, the largest staged activation (4 x 8192)."""
    for (M, N, K) in ((1, 1, 256), (2, 13, 2048), (3, 4097, 2304), (4, 1000, 4352),
                      (1, 8191, 8192), (4, 300, 8192), (2, 64, 6144), (3, 5, 7936)):
        W, X = si.small_case(40 + M + N + K + fmt, M, N, K)
        codes, scales = quantize_both(gpu, orc, fmt, W)
        Yg = forward_gpu(gpu, fmt, X, O.DT_BF16, codes, scales, N)
        Yr = orc.forward(fmt, X, O.DT_BF16, codes, scales, N)
        e = rel_err(Yg, Yr)
        assert e <= TOL[O.DT_BF16], (M, N, K, e)


@pytest.mark.parametrize("K", [4096, 16384, 16640])
def test_forward_long_rows(gpu, orc, K):
    """Large-M bf16 path at reduction lengths that exercise every row width
    of the activation pre-pass (held in registers up to K = 16384, two reads
    beyond)."""
    M, N = 80, 48
    for fmt in (O.FMT_INT8, O.FMT_Q4):
        W, X = si.small_case(40 + K + fmt, M, N, K)
        codes, scales = quantize_both(gpu, orc, fmt, W)
        Yg = forward_gpu(gpu, fmt, X, O.DT_BF16, codes, scales, N)
        Yr = orc.forward(fmt, X, O.DT_BF16, codes, scales, N)
        assert rel_err(Yg, Yr) <= TOL[O.DT_BF16], (fmt, K)


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_forward_row_scales_far_apart(gpu, orc, fmt):
    """Activation rows scaled by 2^-100 .. 2^100 (and one all-zero row): each
    row's own relative error stays within the tolerance, on the small-M path
    and on the large-M path (per-row power-of-two shifts)."""
    rng = np.random.default_rng(91 + fmt)
    N, K = 96, 256
    for M in (40, 200):
        W, X0 = si.small_case(92 + M + fmt, M, N, K, O.DT_F32)
        e = rng.integers(-100, 101, M).astype(np.float64)
        Xf = (X0.astype(np.float64) * 2.0 ** e[:, None]).astype(np.float32)
        Xf[M // 2] = 0.0
        X = si.f32_to_bf16_bits(Xf)
        codes, scales = quantize_both(gpu, orc, fmt, W)
        Yg = forward_gpu(gpu, fmt, X, O.DT_BF16, codes, scales, N).astype(np.float64)
        Yr = orc.forward(fmt, X, O.DT_BF16, codes, scales, N)
        assert np.all(Yg[M // 2] == 0.0)
        for m in range(M):
            if m == M // 2:
                continue
            err = np.max(np.abs(Yg[m] - Yr[m])) / np.max(np.abs(Yr[m]))
            assert err <= TOL[O.DT_BF16], (M, m, err)


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_forward_block_scales_far_apart(gpu, orc, fmt):
    """Weight rows whose blocks lie many binary decades apart (block
    magnitudes 2^-20 .. 2^16 within one row, rows whose largest block
    exceeds 2^15 so that the large-M path shifts them down, rows of tiny
    blocks only), on the exact small-M path (M = 40) and the folded large-M
    path (M = 200).

    Bound, element by element: the large-M path enters each weight as
    fp16(c * s') with s' = s * 2^f and f set by the row's largest scale.
    When s' is a normal fp16 (s at least Q * 2^-28 of the row's largest
    scale) that is one rounding, relative error <= 2^-11; below it s' itself
    is rounded to a subnormal, an absolute error <= (Q + 2) * 2^-25 in the
    shifted units, i.e. <= (Q + 2) * Q * smax * 2^-39 per unit of |x|.  The
    fp32 accumulation adds <= K * 2^-24 of sum |x| |w|.  So
      |Yg - Yr| <= (2^-11 + (K + 8) 2^-24) (|X| |W|^T)[m][n]
                   + (Q + 2) Q smax[n] 2^-39 sum_k |X[m][k]|."""
    Q = QMAX[fmt]
    rng = np.random.default_rng(3100 + fmt)
    N, K = 64, 1024
    nb = K // 32
    u = rng.integers(-20, 17, (N, nb)).astype(np.float64)
    u[0] = 16.0            # every block large: negative row shift
    u[1] = -20.0           # every block tiny: large positive row shift
    u[2, ::2], u[2, 1::2] = 16.0, -20.0   # 36 binary decades inside one row
    u[3, 0] = 16.0         # one large block, the rest random
    W = (rng.standard_normal((N, K)) * np.repeat(2.0 ** u, 32, axis=1)).astype(np.float32)
    codes, scales = quantize_both(gpu, orc, fmt, W)
    Wd = orc.dequantize(fmt, codes, scales, N, K)
    smax = np.max(np.abs(Wd), axis=1) / Q
    for M in (40, 200):
        X = si.small_case(3200 + M + fmt, M, 1, K)[1]
        Xv = si.bf16_bits_to_f32(X).astype(np.float64)
        Yg = forward_gpu(gpu, fmt, X, O.DT_BF16, codes, scales, N).astype(np.float64)
        Yr = orc.forward(fmt, X, O.DT_BF16, codes, scales, N)
        A = np.abs(Xv) @ np.abs(Wd).T
        lim = (2.0 ** -11 + (K + 8) * 2.0 ** -24) * A + \
            (Q + 2) * Q * 2.0 ** -39 * np.outer(np.abs(Xv).sum(axis=1), smax)
        bad = np.argwhere(np.abs(Yg - Yr) > lim)
        assert len(bad) == 0, (M, bad[:5], (Yg - Yr)[tuple(bad[0])], lim[tuple(bad[0])])
        assert rel_err(Yg, Yr) <= TOL[O.DT_BF16]


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
@pytest.mark.parametrize("xdt", [O.DT_BF16, O.DT_F32])
def test_forward_power_of_two_exact(gpu, orc, fmt, xdt):
    """W = c * 2^-12, integer X: the exact result is representable, so the
    GPU must reproduce it exactly."""
    Q = QMAX[fmt]
    rng = np.random.default_rng(17 + fmt + xdt)
    N, K = 80, 512
    for M in (5, 40, 200):
        C = rng.integers(-Q, Q + 1, (N, K))
        C.reshape(N, K // 32, 32)[:, :, 3] = rng.choice([-Q, Q], (N, K // 32))
        W = (C * 2.0 ** -12).astype(np.float32)
        codes, scales = quantize_both(gpu, orc, fmt, W)
        Xi = rng.integers(-8, 9, (M, K)).astype(np.float32)
        X = Xi if xdt == O.DT_F32 else si.f32_to_bf16_bits(Xi)
        Yg = forward_gpu(gpu, fmt, X, xdt, codes, scales, N)
        want = (Xi.astype(np.int64) @ C.T).astype(np.float64) * 2.0 ** -12
        assert np.array_equal(Yg.astype(np.float64), want)
        assert np.array_equal(Yg.astype(np.float64), orc.forward(fmt, X, xdt, codes, scales, N))


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_forward_stored_extreme_codes_exact(gpu, orc, fmt):
    """Codes set by hand (including the never-produced -128 / -8) with unit
    scales and integer activations: Y is an exact integer matmul."""
    Q = QMAX[fmt]
    rng = np.random.default_rng(23 + fmt)
    M, N, K = 37, 48, 96
    C = rng.integers(-Q - 1, Q + 1, (N, K))
    C[:, 0] = -Q - 1
    if fmt == O.FMT_INT8:
        codes = C.astype(np.int8).view(np.uint8)
    else:
        u = (C & 0xF).astype(np.uint8)
        codes = (u[:, 0::2] | (u[:, 1::2] << 4)).astype(np.uint8)
    scales = np.full((N, K // 32), 0x3C00, np.uint16)
    Xi = rng.integers(-100, 101, (M, K)).astype(np.float32)
    for xdt, X in ((O.DT_F32, Xi), (O.DT_BF16, si.f32_to_bf16_bits(Xi))):
        Yg = forward_gpu(gpu, fmt, X, xdt, codes, scales, N)
        assert np.array_equal(Yg.astype(np.int64), Xi.astype(np.int64) @ C.T)


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_forward_in_kernel_reduction(gpu, orc, fmt):
    """Single layers whose split plan adds the K parts inside the large-M
    kernel (more parts than one wave of workgroups: 700 or 768 tokens x 2048
    x 2048, 6 x 8 output tiles in 4 parts of 8 steps each; each part stores
    its partial tile and the last part to arrive adds them in part order).
    Every output starts NaN-filled; all rows against the oracle (700: a
    ragged last row tile); a second call repeats the first bit for bit."""
    torch, ql = gpu
    N, K = 2048, 2048
    W, _ = si.small_case(3600 + fmt, 1, N, K)
    codes, scales = quantize_both(gpu, orc, fmt, W)
    cd = torch.from_numpy(codes).cuda()
    sd = torch.from_numpy(scales.view(np.int16)).cuda()
    for M in (768, 700):
        _, X = si.small_case(3610 + M, M, 1, K)
        Xd = dev_x(torch, X, O.DT_BF16)
        Y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        ql.forward(fmt, Xd, cd, sd, N, Y)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(Y).all()), M
        Yg = Y.cpu().numpy()
        Yr = orc.forward(fmt, X, O.DT_BF16, codes, scales, N)
        assert rel_err(Yg, Yr) <= TOL[O.DT_BF16], M
        Y.fill_(float("nan"))
        ql.forward(fmt, Xd, cd, sd, N, Y)
        torch.cuda.synchronize()
        assert np.array_equal(Y.cpu().numpy(), Yg), M


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_forward_split_reduction(gpu, orc, fmt):
    """Large-M shapes with few output tiles and long reductions, which the
    fp16 path cuts into K parts summed by a separate launch (the plan when
    all parts fit in one wave of workgroups): single layers and a grouped
    call mixing reduction lengths over two activations; uneven last parts
    (K / 64 not a multiple of the part length), ragged tiles; results repeat
    bit for bit.  The in-kernel reduction has tests of its own."""
    torch, ql = gpu
    for (M, N, K) in ((300, 520, 4096), (129, 260, 8448), (2048, 64, 2304)):
        W, X = si.small_case(90 + M + N + K + fmt, M, N, K)
        codes, scales = quantize_both(gpu, orc, fmt, W)
        Yg = forward_gpu(gpu, fmt, X, O.DT_BF16, codes, scales, N)
        Yr = orc.forward(fmt, X, O.DT_BF16, codes, scales, N)
        assert rel_err(Yg, Yr) <= TOL[O.DT_BF16], (M, N, K)
        assert np.array_equal(Yg, forward_gpu(gpu, fmt, X, O.DT_BF16, codes, scales, N))
    # one grouped launch: short and long reductions over two activations
    M = 384
    _, xa = si.small_case(95, M, 1, 512)
    _, xb = si.small_case(96, M, 1, 4096)
    shapes = [(700, 512), (256, 4096), (1000, 512)]
    entries, refs = [], []
    for i, (N, K) in enumerate(shapes):
        W, _ = si.small_case(97 + i, 1, N, K)
        cd, sd = ql.quantize(fmt, dev_w(torch, W))
        cr, sr = orc.quantize(fmt, W)
        X = xa if K == 512 else xb
        Y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        entries.append((fmt, dev_x(torch, X, O.DT_BF16), cd, sd, N, Y))
        refs.append(orc.forward(fmt, X, O.DT_BF16, cr, sr, N))
    ql.block_forward(entries)
    torch.cuda.synchronize()
    for e, Yr in zip(entries, refs):
        assert rel_err(e[5].cpu().numpy(), Yr) <= TOL[O.DT_BF16]


def test_forward_deterministic(gpu, orc):
    torch, ql = gpu
    W, X = si.small_case(5, 300, 520, 1024, O.DT_BF16)
    codes, scales = orc.quantize(O.FMT_Q4, W)
    a = forward_gpu(gpu, O.FMT_Q4, X, O.DT_BF16, codes, scales, 520)
    b = forward_gpu(gpu, O.FMT_Q4, X, O.DT_BF16, codes, scales, 520)
    assert np.array_equal(a, b)


def test_forward_on_side_stream(gpu, orc):
    torch, ql = gpu
    W, X = si.small_case(6, 50, 130, 256, O.DT_BF16)
    codes, scales = orc.quantize(O.FMT_INT8, W)
    s = torch.cuda.Stream()
    cd = torch.from_numpy(codes).cuda()
    sd = torch.from_numpy(scales.view(np.int16)).cuda()
    xd = dev_x(torch, X, O.DT_BF16)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        Y = ql.forward(O.FMT_INT8, xd, cd, sd, 130)
    s.synchronize()
    e = rel_err(Y.cpu().numpy(), orc.forward(O.FMT_INT8, X, O.DT_BF16, codes, scales, 130))
    assert e <= TOL[O.DT_BF16]


def test_forward_graph_workspace(gpu, orc):
    """Captured graphs and the per-stream workspace.  A graph captured on a
    stream whose workspace an eager call has sized keeps that buffer when a
    later, larger call on the stream grows the workspace; a capture that
    needs more than its stream's workspace allocates for itself.  Every
    replay, with eager work and synchronization in between, equals the eager
    result bit for bit."""
    torch, ql = gpu
    fmt = O.FMT_Q4
    small, large = (300, 520, 1024), (640, 1024, 4096)
    data = {}
    for (M, N, K) in (small, large):
        W, X = si.small_case(300 + M + K, M, N, K)
        codes, scales = orc.quantize(fmt, W)
        data[(M, N, K)] = (dev_x(torch, X, O.DT_BF16), torch.from_numpy(codes).cuda(),
                           torch.from_numpy(scales.view(np.int16)).cuda(),
                           orc.forward(fmt, X, O.DT_BF16, codes, scales, N))
    Ys = torch.empty(small[:2], dtype=torch.float32, device="cuda")
    Yl = torch.empty(large[:2], dtype=torch.float32, device="cuda")

    def run(shape, Y):
        xd, cd, sd, _ = data[shape]
        ql.forward(fmt, xd, cd, sd, shape[1], Y)

    s, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        run(small, Ys)
    s.synchronize()
    eager_s = Ys.clone()
    assert rel_err(eager_s.cpu().numpy(), data[small][3]) <= TOL[O.DT_BF16]
    g1 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g1, stream=s):
        run(small, Ys)
    with torch.cuda.stream(s):
        run(large, Yl)  # grows the workspace of s
    s.synchronize()
    eager_l = Yl.clone()
    assert rel_err(eager_l.cpu().numpy(), data[large][3]) <= TOL[O.DT_BF16]
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g2, stream=s2):  # nothing sized on s2 yet
        run(large, Yl)
    for _ in range(3):
        Ys.fill_(float("nan"))
        Yl.fill_(float("nan"))
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            g1.replay()
        s.synchronize()
        assert torch.equal(Ys, eager_s)
        with torch.cuda.stream(s):
            run(large, Yl)
        s.synchronize()
        assert torch.equal(Yl, eager_l)
        Yl.fill_(float("nan"))
        torch.cuda.synchronize()
        with torch.cuda.stream(s2):
            g2.replay()
        s2.synchronize()
        assert torch.equal(Yl, eager_l)


# --------------------------------------------------------------------------
# unquantized reference: fp16 weights through the same large-M kernel
# --------------------------------------------------------------------------

def f16_bits(W):
    return np.ascontiguousarray(W, dtype=np.float32).astype(np.float16).view(np.uint16)


def test_forward_f16_weights(gpu, orc):
    """fp16 weights (QL_FMT_F16) against the oracle's unquantized product:
    ragged row and column counts, one to several 64-k steps, small M (the
    same kernel serves every M), a split long reduction; results repeat bit
    for bit."""
    torch, ql = gpu
    for (M, N, K) in ((1, 40, 256), (65, 200, 512), (300, 520, 1280), (129, 17, 1024),
                      (214, 3072, 1024), (128, 64, 8192)):
        W, X = si.small_case(500 + M + N + K, M, N, K)
        W16 = f16_bits(W)
        wd = torch.from_numpy(W16.view(np.int16)).cuda()
        Y = ql.forward(ql.FMT_F16, dev_x(torch, X, O.DT_BF16), wd, None, N)
        torch.cuda.synchronize()
        Yg = Y.cpu().numpy()
        Yr = orc.forward_f16(X, O.DT_BF16, W16)
        e = rel_err(Yg, Yr)
        assert e <= TOL[O.DT_BF16], (M, N, K, e)
        Y2 = ql.forward(ql.FMT_F16, dev_x(torch, X, O.DT_BF16), wd, None, N)
        torch.cuda.synchronize()
        assert np.array_equal(Yg, Y2.cpu().numpy())


def test_forward_f16_block_and_errors(gpu, orc):
    """A grouped call of one block's four fp16-weight linears (every row
    against the oracle), and the calls the format does not take."""
    torch, ql = gpu
    xa, xb = si.paper_activations(1)
    d = si.PAPER_WIDTHS[1][1]
    entries, refs = [], []
    rows = np.arange(xa.shape[0])
    for i, (_, N, K) in enumerate(si.block_linears(d)):
        W16 = f16_bits(si.paper_weight(1, 0, i))
        X = xb if K == 4 * d else xa
        Y = torch.full((X.shape[0], N), float("nan"), dtype=torch.float32, device="cuda")
        entries.append((ql.FMT_F16, dev_x(torch, X, O.DT_BF16),
                        torch.from_numpy(W16.view(np.int16)).cuda(), None, N, Y))
        refs.append(orc.forward_f16(X, O.DT_BF16, W16, rows=rows))
    ql.block_forward(entries)
    torch.cuda.synchronize()
    for e, Yr in zip(entries, refs):
        assert bool(torch.isfinite(e[5]).all())
        assert rel_err(e[5].cpu().numpy()[rows], Yr) <= TOL[O.DT_BF16]
    w = torch.zeros((16, 512), dtype=torch.int16, device="cuda")
    for X, status in ((torch.zeros((4, 512), dtype=torch.float32, device="cuda"), 5),
                      (torch.zeros((4, 512), dtype=torch.int16, device="cuda"), None)):
        if status is None:
            ql.forward(ql.FMT_F16, X, w, None, 16)
            continue
        with pytest.raises(ql.QLinearError) as err:
            ql.forward(ql.FMT_F16, X, w, None, 16)
        assert err.value.status == status  # fp32 activations: unsupported
    with pytest.raises(ql.QLinearError) as err:
        ql.forward(ql.FMT_F16, torch.zeros((4, 96), dtype=torch.int16, device="cuda"),
                   torch.zeros((16, 96), dtype=torch.int16, device="cuda"), None, 16)
    assert err.value.status == 5  # K % 256 != 0: unsupported


# --------------------------------------------------------------------------
# the workload configurations
# --------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["single_int8", "single_q4"])
def test_single_linear_configs(gpu, orc, name):
    cfg = getattr(si, name)()
    fmt, W, X, xdt = cfg["fmt"], cfg["W"], cfg["X"], cfg["xdt"]
    codes, scales = quantize_both(gpu, orc, fmt, W)
    Yg = forward_gpu(gpu, fmt, X, xdt, codes, scales, W.shape[0])
    Yr = orc.forward(fmt, X, xdt, codes, scales, W.shape[0])
    e = rel_err(Yg, Yr)
    print(f"{name}: max err / |y|inf = {e:.3e}")
    assert e <= TOL[xdt]


def sample_rows(M, k, seed):
    rng = np.random.default_rng(seed)
    rows = set([0, M - 1]) | set(rng.choice(M, size=min(k, M), replace=False).tolist())
    return np.array(sorted(rows), dtype=np.int64)


def tile_rows(M, k, seed, tile=128):
    """At least k distinct rows of an M-row output: one random row inside
    every `tile`-row band (so every row tile of a grouped launch is sampled),
    the first and last rows, and random others up to k."""
    rng = np.random.default_rng(seed)
    rows = {0, M - 1}
    for t0 in range(0, M, tile):
        rows.add(int(rng.integers(t0, min(t0 + tile, M))))
    rest = [r for r in rng.permutation(M).tolist() if r not in rows]
    rows |= set(rest[:max(0, k - len(rows))])
    return np.array(sorted(rows), dtype=np.int64)


def run_block(gpu, orc, fmt, weights, xa, xb, rows, check_codes=True):
    """One DiT block's four linears through qlinear_block_forward.  Every Y
    starts NaN-filled: the whole output of every linear must be finite (every
    element written) and the sampled rows must match the oracle (all N
    columns)."""
    torch, ql = gpu
    xa_d, xb_d = dev_x(torch, xa, O.DT_BF16), dev_x(torch, xb, O.DT_BF16)
    entries, host = [], []
    for i, W in enumerate(weights):
        N, K = W.shape
        cd, sd = ql.quantize(fmt, dev_w(torch, W))
        if check_codes:
            cr, sr = orc.quantize(fmt, W)
            assert np.array_equal(host_scales(sd), sr)
            assert np.array_equal(host_codes(cd), cr)
        else:
            cr, sr = host_codes(cd), host_scales(sd)
        Y = torch.full((xa.shape[0], N), float("nan"), dtype=torch.float32, device="cuda")
        entries.append((fmt, xb_d if K == 4 * xa.shape[1] else xa_d, cd, sd, N, Y))
        host.append((cr, sr, N, K))
    ql.block_forward(entries)
    torch.cuda.synchronize()
    errs = []
    for i, ((fmt_, X_d, cd, sd, N, Y), (cr, sr, N_, K)) in enumerate(zip(entries, host)):
        assert bool(torch.isfinite(Y).all()), f"linear {i}: unwritten (NaN) or non-finite outputs"
        X = xb if K == 4 * xa.shape[1] else xa
        Yr = orc.forward(fmt, X, O.DT_BF16, cr, sr, N, rows=rows)
        Yg = Y.cpu().numpy()[rows]
        errs.append(rel_err(Yg, Yr))
    return errs


def test_block_int8_config(gpu, orc):
    xa, xb = si.block_activations()
    weights = [si.block_int8_weight(i) for i in range(4)]
    rows = tile_rows(xa.shape[0], 64, 0)
    assert len(rows) >= 64
    errs = run_block(gpu, orc, O.FMT_INT8, weights, xa, xb, rows)
    print("block int8 errs", errs)
    assert max(errs) <= TOL[O.DT_BF16]


@pytest.fixture(scope="module")
def block_x():
    return si.block_activations()


@pytest.mark.parametrize("blk", range(si.N_BLOCKS))
def test_step_q4_config_every_block(gpu, orc, block_x, blk):
    """All 24 blocks of the q4 denoising step: codes and scales bit for bit,
    every output finite, 64 rows (one in every 128-row tile) x all N of each
    linear against the oracle."""
    xa, xb = block_x
    weights = [si.step_q4_weight(blk, i) for i in range(4)]
    rows = tile_rows(xa.shape[0], 64, 1000 + blk)
    errs = run_block(gpu, orc, O.FMT_Q4, weights, xa, xb, rows)
    print(f"step q4 block {blk} errs", errs)
    assert max(errs) <= TOL[O.DT_BF16]


@pytest.mark.parametrize("w", range(len(si.PAPER_WIDTHS)))
@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_paper_width_block(gpu, orc, w, fmt):
    """The last block of each of the paper's DiT widths (d = 1024, 1536) at
    the token count of one 10 s clip (214 rows: partial 128-row tiles, few
    tiles per layer), every output row against the oracle."""
    xa, xb = si.paper_activations(w)
    blk = si.PAPER_WIDTHS[w][2] - 1
    weights = [si.paper_weight(w, blk, i) for i in range(4)]
    errs = run_block(gpu, orc, fmt, weights, xa, xb, np.arange(xa.shape[0]))
    print(f"paper width {si.PAPER_WIDTHS[w][0]} fmt {fmt} errs", errs)
    assert max(errs) <= TOL[O.DT_BF16]


@pytest.mark.parametrize("v,fmt,N,K", si.skinny_variants())
def test_skinny_configs(gpu, orc, v, fmt, N, K):
    W = si.skinny_weight(v, N, K)
    codes, scales = quantize_both(gpu, orc, fmt, W)
    for M in si.SKINNY_M:
        X = si.skinny_activations(M, K)
        Yg = forward_gpu(gpu, fmt, X, O.DT_BF16, codes, scales, N)
        rows = np.arange(M) if M <= 32 else sample_rows(M, 30, M)
        Yr = orc.forward(fmt, X, O.DT_BF16, codes, scales, N, rows=rows)
        e = rel_err(Yg[rows], Yr)
        print(f"skinny v{v} M={M}: {e:.3e}")
        assert e <= TOL[O.DT_BF16]


def test_block_forward_mixed_group(gpu, orc):
    """Layers of different formats / activation dtypes in one call."""
    torch, ql = gpu
    specs = [(O.FMT_INT8, O.DT_BF16, 40, 96, 64), (O.FMT_Q4, O.DT_BF16, 40, 200, 128),
             (O.FMT_INT8, O.DT_F32, 17, 64, 96), (O.FMT_Q4, O.DT_F32, 3, 48, 32),
             (O.FMT_Q4, O.DT_BF16, 0, 16, 32)]
    entries, refs = [], []
    for i, (fmt, xdt, M, N, K) in enumerate(specs):
        W, X = si.small_case(300 + i, M, N, K, xdt)
        cd, sd = ql.quantize(fmt, dev_w(torch, W))
        cr, sr = orc.quantize(fmt, W)
        Y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        entries.append((fmt, dev_x(torch, X, xdt), cd, sd, N, Y))
        refs.append(orc.forward(fmt, X, xdt, cr, sr, N) if M > 0 else None)
    ql.block_forward(entries)
    torch.cuda.synchronize()
    for (fmt, xdt, M, N, K), e, Yr in zip(specs, entries, refs):
        if M == 0:
            continue
        assert rel_err(e[5].cpu().numpy(), Yr) <= TOL[xdt]


# --------------------------------------------------------------------------
# the same shapes through every kernel that takes them (qlinear_force_path)
# --------------------------------------------------------------------------

EXACT_PATHS = ("GEMV", "STREAM", "SKINNY", "TILED", "MID")


def takes(path, M, K):
    """Shape limits of each forced kernel (include/qlinear.h)."""
    return {"GEMV": 1 <= M <= 4 and K % 256 == 0 and K <= 8192,
            "STREAM": M <= 32 and K % 256 == 0,
            "SKINNY": M <= 64,
            "TILED": True,
            "WIDE": K % 256 == 0,
            "MID": K % 256 == 0}[path]


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_forced_paths_agree(gpu, orc, fmt):
    """Each shape runs through every kernel that takes it: the exact kernels
    (GEMV, streaming, few-row MFMA, tiled MFMA, mid-M) each within 1e-5 of the
    oracle and within 2e-6 of one another; the large-M fp16 path within the
    bf16 tolerance.  A kernel that cannot take a shape refuses it
    (QL_ERR_UNSUPPORTED) and leaves Y untouched."""
    torch, ql = gpu
    shapes = [(1, 300, 2048), (3, 257, 1024), (4, 64, 8192), (8, 300, 2048), (17, 200, 512),
              (32, 513, 2304), (64, 96, 768), (130, 260, 1280), (40, 48, 96)]
    try:
        for (M, N, K) in shapes:
            W, X = si.small_case(7000 + M + N + K + fmt, M, N, K)
            codes, scales = quantize_both(gpu, orc, fmt, W)
            cd = torch.from_numpy(codes).cuda()
            sd = torch.from_numpy(scales.view(np.int16)).cuda()
            xd = dev_x(torch, X, O.DT_BF16)
            Yr = orc.forward(fmt, X, O.DT_BF16, codes, scales, N)
            got = {}
            for name in EXACT_PATHS + ("WIDE",):
                Y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
                ql.load().qlinear_force_path(getattr(ql, "PATH_" + name))
                if not takes(name, M, K):
                    with pytest.raises(ql.QLinearError) as err:
                        ql.forward(fmt, xd, cd, sd, N, Y)
                    assert err.value.status == 5, (name, M, K)
                    torch.cuda.synchronize()
                    assert bool(torch.isnan(Y).all()), (name, M, K)
                    continue
                ql.forward(fmt, xd, cd, sd, N, Y)
                torch.cuda.synchronize()
                got[name] = Y.cpu().numpy().astype(np.float64)
                tol = TOL[O.DT_BF16] if name == "WIDE" else 1e-5
                assert rel_err(got[name], Yr) <= tol, (name, M, N, K, rel_err(got[name], Yr))
            exact = [got[p] for p in EXACT_PATHS if p in got]
            assert len(exact) >= 1
            for Ya in exact[1:]:
                assert rel_err(Ya, exact[0]) <= 2e-6, (M, N, K)
    finally:
        ql.load().qlinear_force_path(ql.PATH_AUTO)


def test_forced_path_fp32_activations(gpu, orc):
    """fp32 activations: only the tiled kernel takes them; the few-row and
    fp16-path kernels refuse."""
    torch, ql = gpu
    M, N, K = 12, 40, 256
    W, X = si.small_case(7100, M, N, K, O.DT_F32)
    codes, scales = orc.quantize(O.FMT_INT8, W)
    cd = torch.from_numpy(codes).cuda()
    sd = torch.from_numpy(scales.view(np.int16)).cuda()
    xd = dev_x(torch, X, O.DT_F32)
    try:
        for name in ("GEMV", "STREAM", "SKINNY", "WIDE", "MID"):
            ql.load().qlinear_force_path(getattr(ql, "PATH_" + name))
            with pytest.raises(ql.QLinearError) as err:
                ql.forward(O.FMT_INT8, xd, cd, sd, N)
            assert err.value.status == 5, name
        ql.load().qlinear_force_path(ql.PATH_TILED)
        Yg = ql.forward(O.FMT_INT8, xd, cd, sd, N)
        torch.cuda.synchronize()
        assert rel_err(Yg.cpu().numpy(), orc.forward(O.FMT_INT8, X, O.DT_F32, codes, scales, N)) <= 1e-5
    finally:
        ql.load().qlinear_force_path(ql.PATH_AUTO)


# --------------------------------------------------------------------------
# few-row grouped launches: a whole block's weights in one launch
# --------------------------------------------------------------------------

@pytest.fixture(scope="module")
def skinny_block():
    """The four d = 2048 linears of the int8 block workload's weights (seeds
    2..5) and their q4 codes from the same draws."""
    return [si.block_int8_weight(i) for i in range(4)]


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
@pytest.mark.parametrize("M", [1, 3, 8, 32])
def test_block_forward_few_rows_grouped(gpu, orc, skinny_block, fmt, M):
    """One block's four linears (QKV 2048->6144, out, FFN-up 2048->8192,
    FFN-down 8192->2048) at the few-row sizes: the GEMV (M <= 4) and the
    streaming kernel (M <= 32) each take the four layers in one launch, the
    streaming kernel's K-split layers share one sum launch.  Every output
    NaN-filled beforehand, every row against the oracle; a second call
    repeats the first bit for bit."""
    torch, ql = gpu
    rng = np.random.default_rng(7300 + M + fmt)
    xa = si.activations(rng, M, 2048, si.DT_BF16)
    xb = si.activations(rng, M, 8192, si.DT_BF16)
    entries, host = [], []
    for W in skinny_block:
        N, K = W.shape
        cd, sd = ql.quantize(fmt, dev_w(torch, W))
        X = xb if K == 8192 else xa
        Y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        entries.append((fmt, dev_x(torch, X, O.DT_BF16), cd, sd, N, Y))
        host.append((X, host_codes(cd), host_scales(sd), N))
    ql.block_forward(entries)
    torch.cuda.synchronize()
    first = [e[5].clone() for e in entries]
    ql.block_forward(entries)
    torch.cuda.synchronize()
    for e, Y1, (X, cr, sr, N) in zip(entries, first, host):
        assert torch.equal(e[5], Y1)
        Yr = orc.forward(fmt, X, O.DT_BF16, cr, sr, N)
        assert rel_err(e[5].cpu().numpy(), Yr) <= 1e-5, (M, N)


def test_block_forward_few_rows_mixed_m(gpu, orc):
    """One call whose layers have different row counts: GEMV layers of two
    row counts (two launches), streaming layers of two row counts in one
    launch (activation stage of the larger), some with K parts."""
    torch, ql = gpu
    specs = [(1, 300, 2048), (4, 257, 8192), (1, 64, 512), (9, 500, 8192), (30, 129, 1024),
             (4, 1000, 256)]
    for fmt in (O.FMT_INT8, O.FMT_Q4):
        entries, refs = [], []
        for i, (M, N, K) in enumerate(specs):
            W, X = si.small_case(7400 + i + fmt, M, N, K)
            cd, sd = ql.quantize(fmt, dev_w(torch, W))
            Y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
            entries.append((fmt, dev_x(torch, X, O.DT_BF16), cd, sd, N, Y))
            refs.append(orc.forward(fmt, X, O.DT_BF16, host_codes(cd), host_scales(sd), N))
        ql.block_forward(entries)
        torch.cuda.synchronize()
        for (M, N, K), e, Yr in zip(specs, entries, refs):
            assert rel_err(e[5].cpu().numpy(), Yr) <= 1e-5, (fmt, M, N, K)


@pytest.mark.parametrize("fmt", [O.FMT_INT8, O.FMT_Q4])
def test_tiled_kernel_k_parts(gpu, orc, fmt):
    """The tiled exact kernel cuts long reductions into K parts when a call
    has too few tiles for the GPU (partials added by the sum launch): fp32
    activations at the single-linear workload's shape (64 x 1024 x 1024),
    an odd block count (the last 64-k step is half a step) in the last
    part, bf16 mid-M shapes forced onto the tiled kernel, and a split layer
    with its epilogue applied by the sum launch.  Results repeat bit for
    bit."""
    torch, ql = gpu
    cases = [(64, 1024, 1024, O.DT_F32), (40, 512, 2080, O.DT_F32), (7, 300, 4128, O.DT_F32),
             (128, 2048, 8192, O.DT_BF16), (214, 1024, 4096, O.DT_BF16),
             (256, 1536, 6144, O.DT_BF16)]
    try:
        for (M, N, K, xdt) in cases:
            W, X = si.small_case(7500 + M + N + K + fmt, M, N, K, xdt)
            codes, scales = quantize_both(gpu, orc, fmt, W)
            ql.load().qlinear_force_path(ql.PATH_TILED if xdt == O.DT_BF16 else ql.PATH_AUTO)
            Yg = forward_gpu(gpu, fmt, X, xdt, codes, scales, N)
            Yr = orc.forward(fmt, X, xdt, codes, scales, N)
            assert rel_err(Yg, Yr) <= (1e-5 if xdt == O.DT_F32 else 2e-6), (M, N, K, rel_err(Yg, Yr))
            assert np.array_equal(Yg, forward_gpu(gpu, fmt, X, xdt, codes, scales, N))
        # a split layer with bias, GELU and a residual, applied after the sum
        M, N, K = 64, 1024, 1024
        W, X = si.small_case(7600 + fmt, M, N, K, O.DT_F32)
        codes, scales = quantize_both(gpu, orc, fmt, W)
        rng = np.random.default_rng(7601)
        bias = (rng.standard_normal(N) * 0.5).astype(np.float32)
        resid = rng.standard_normal((M, N)).astype(np.float32)
        Y = torch.from_numpy(resid.copy()).cuda()
        ql.forward_ep(fmt, dev_x(torch, X, O.DT_F32), torch.from_numpy(codes).cuda(),
                      torch.from_numpy(scales.view(np.int16)).cuda(), N, Y=Y,
                      bias=torch.from_numpy(bias).cuda(), act=ql.ACT_GELU, residual=Y)
        torch.cuda.synchronize()
        P = orc.forward(fmt, X, O.DT_F32, codes, scales, N)
        Yr = orc.epilogue(P, bias, O.ACT_GELU, resid)
        lim = 1.13 * 1e-5 * np.max(np.abs(P)) + 1e-6 * (np.abs(Yr) + np.max(np.abs(P)))
        assert np.all(np.abs(Y.cpu().numpy().astype(np.float64) - Yr) <= lim)
    finally:
        ql.load().qlinear_force_path(ql.PATH_AUTO)
