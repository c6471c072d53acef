"""GPU parity of the steering injection (Eq. 2: h + alpha ||h_bar|| d on every
token) against the oracle: as an operation of its own (qlinear_steer) and
fused into the epilogue of every kernel that stores final outputs.

At alpha = 0 the output must be bit for bit the unsteered one.  Otherwise,
element by element, |Y_gpu - Y_ref| stays within the bound of the unsteered
path plus the fp32 roundings of the steering term (alpha * hnorm, times
d[n], added): 4 * 2^-24 * (|alpha hnorm d[n]| + |Y_ref|).  A captured graph
re-reads the strength at every replay: replays with new strengths equal
eager calls bit for bit.
"""
import numpy as np
import pytest

import synth_inputs as si
from oracle import oracle as O

pytestmark = pytest.mark.gpu

TOL = {O.DT_BF16: 2e-3, O.DT_F32: 1e-5}
EPS = 4 * 2.0 ** -24


@pytest.fixture(scope="module")
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU (run with -m 'not gpu' on a CPU host)")
    from paper_2607_08526_amd import qlinear as ql
    ql.load()
    return torch, ql


def dev_f32(torch, A):
    return torch.from_numpy(np.ascontiguousarray(A, dtype=np.float32)).cuda()


def dev_x(torch, X, xdt):
    if xdt == O.DT_F32:
        return dev_f32(torch, X)
    return torch.from_numpy(np.ascontiguousarray(X, dtype=np.uint16).view(np.int16)).cuda()


def unit(rng, N):
    d = rng.standard_normal(N)
    return (d / np.linalg.norm(d)).astype(np.float32)


def steer_bound(d, hnorm, alpha, Yr):
    return EPS * (np.abs(np.float64(alpha) * hnorm * d.astype(np.float64))[None, :] + np.abs(Yr))


@pytest.mark.parametrize("N", [2048, 77])
def test_steer_op(gpu, orc, N):
    """The operation alone, 16-byte groups (N % 4 == 0) and single elements;
    alpha = 0 leaves h bit for bit (signed zeros and NaN included)."""
    torch, ql = gpu
    rng = np.random.default_rng(8000 + N)
    M, hnorm = 300, 8.0
    h0 = rng.standard_normal((M, N)).astype(np.float32)
    h0[0, 0], h0[1, 1], h0[2, 2] = -0.0, np.nan, np.inf
    d = unit(rng, N)
    dd = dev_f32(torch, d)
    strength = torch.zeros(1, dtype=torch.float32, device="cuda")
    for alpha in (0.0, 0.15, 1.0, 0.0):
        strength.fill_(alpha)
        h = dev_f32(torch, h0)
        ql.steer(h, dd, hnorm, strength)
        torch.cuda.synchronize()
        hg = h.cpu().numpy()
        if alpha == 0.0:
            assert np.array_equal(hg.view(np.uint32), h0.view(np.uint32))
            continue
        ref = orc.steer(h0.astype(np.float64), d, hnorm, alpha)
        fin = np.isfinite(ref)
        assert np.all(np.abs(hg[fin] - ref[fin]) <= steer_bound(d, hnorm, alpha, ref)[fin])
        assert np.isnan(hg[1, 1]) and hg[2, 2] == np.inf


# (fmt, xdt, M, N, K): each kernel that stores final outputs
PATHS = [
    (O.FMT_Q4, O.DT_BF16, 3, 4097, 2048),     # GEMV
    (O.FMT_INT8, O.DT_BF16, 16, 4100, 512),   # weight streaming, one K part
    (O.FMT_Q4, O.DT_BF16, 8, 2048, 8192),     # weight streaming + split sum
    (O.FMT_INT8, O.DT_BF16, 20, 70, 320),     # small-M MFMA
    (O.FMT_Q4, O.DT_F32, 40, 200, 320),       # MFMA kernel, fp32 activations
    (O.FMT_Q4, O.DT_BF16, 300, 520, 1280),    # fp16 path
    (O.FMT_INT8, O.DT_BF16, 300, 520, 4096),  # fp16 path, parts summed by split sum
    (O.FMT_Q4, O.DT_BF16, 129, 17, 1024),     # fp16 path, element-by-element store
]


@pytest.mark.parametrize("fmt,xdt,M,N,K", PATHS)
def test_steer_in_epilogue(gpu, orc, fmt, xdt, M, N, K):
    torch, ql = gpu
    W, X = si.small_case(8100 + M + N + K, M, N, K, xdt)
    cd, sd = ql.quantize(fmt, dev_f32(torch, W))
    cr, sr = orc.quantize(fmt, W)
    Xd = dev_x(torch, X, xdt)
    rng = np.random.default_rng(N)
    bias = (rng.standard_normal(N) * 0.5).astype(np.float32)
    resid = rng.standard_normal((M, N)).astype(np.float32)
    d, hnorm = unit(rng, N), 20.0
    bd, rd, dd = dev_f32(torch, bias), dev_f32(torch, resid), dev_f32(torch, d)
    strength = torch.zeros(1, dtype=torch.float32, device="cuda")
    P = orc.forward(fmt, X, xdt, cr, sr, N)
    # with bias and residual, steering alone (the per-column term without
    # any other), and steering with GELU into bf16 outputs
    for b_, r_, act, ydt in ((True, True, O.ACT_NONE, torch.float32),
                             (False, False, O.ACT_NONE, torch.float32),
                             (True, False, O.ACT_GELU, torch.bfloat16)):
        kw = dict(bias=bd if b_ else None, residual=rd if r_ else None, act=act, ydtype=ydt)
        plain = ql.forward_ep(fmt, Xd, cd, sd, N, **kw)
        base = orc.epilogue(P, bias if b_ else None, act, resid if r_ else None)
        for alpha in (0.0, 0.25):
            strength.fill_(alpha)
            Y = ql.forward_ep(fmt, Xd, cd, sd, N, steer=(dd, hnorm, strength), **kw)
            torch.cuda.synchronize()
            if alpha == 0.0:
                assert torch.equal(Y.view(torch.int16) if ydt == torch.bfloat16 else Y.view(
                    torch.int32), plain.view(torch.int16) if ydt == torch.bfloat16 else
                    plain.view(torch.int32))
                continue
            Yg = Y.float().cpu().numpy()
            Yr = orc.steer(base, d, hnorm, alpha)
            lim = 1.13 * TOL[xdt] * np.max(np.abs(P)) \
                + 1e-6 * (np.abs(Yr) + np.max(np.abs(P)) + np.max(np.abs(bias))) \
                + steer_bound(d, hnorm, alpha, Yr)
            if ydt == torch.bfloat16:
                lim = lim + 2.0 ** -8 * np.abs(Yr)
            assert np.all(np.abs(Yg - Yr) <= lim), (M, N, K, b_, act)


def test_steer_w8a8(gpu, orc):
    """The W8A8 product takes the same steering term."""
    torch, ql = gpu
    M, N, K = 70, 96, 256
    W, X = si.small_case(8200, M, N, K)
    codes, scales = orc.quantize(O.FMT_INT8, W)
    q, s = orc.quantize_act(X, O.DT_BF16)
    rng = np.random.default_rng(8201)
    d, hnorm = unit(rng, N), 5.0
    strength = torch.full((1,), 0.5, dtype=torch.float32, device="cuda")
    args = (torch.from_numpy(q).cuda(), torch.from_numpy(s.view(np.int16)).cuda(),
            torch.from_numpy(codes).cuda(), torch.from_numpy(scales.view(np.int16)).cuda(), N)
    Y = ql.forward_w8a8(*args, steer=(dev_f32(torch, d), hnorm, strength))
    torch.cuda.synchronize()
    P = orc.forward_w8a8(q, s, codes, scales, N)
    Yr = orc.steer(P, d, hnorm, 0.5)
    Xd = np.abs(np.asarray(s, np.uint16).view(np.float16).astype(np.float64)[:, None] * q)
    Wd = np.abs(orc.dequantize(O.FMT_INT8, codes, scales, N, K))
    lim = (K // 32 + 1) * 2.0 ** -24 * (Xd @ Wd.T) + steer_bound(d, hnorm, 0.5, Yr)
    assert np.all(np.abs(Y.cpu().numpy() - Yr) <= lim)


def test_steer_graph_strength_refresh(gpu, orc):
    """One block's grouped call with steering on the FFN-down output, and the
    steering operation on a residual stream, captured once in a HIP graph;
    every replay re-reads the strength: replays at alpha = 0.5, 0, 1, 0
    equal eager calls at those strengths bit for bit, and alpha = 0 equals
    the unsteered call."""
    torch, ql = gpu
    M, d_model = 256, 512
    rng = np.random.default_rng(8300)
    xa = torch.from_numpy(si.f32_to_bf16_bits(rng.standard_normal((M, d_model)).astype(
        np.float32)).view(np.int16)).cuda()
    xb = torch.from_numpy(si.f32_to_bf16_bits(rng.standard_normal((M, 4 * d_model)).astype(
        np.float32)).view(np.int16)).cuda()
    lin = si.block_linears(d_model)
    ws = [ql.quantize(ql.FMT_Q4, dev_f32(torch, (rng.standard_normal((N, K)) * 0.02)))
          for _, N, K in lin]
    dvec = dev_f32(torch, unit(rng, d_model))
    strength = torch.zeros(1, dtype=torch.float32, device="cuda")
    h0 = dev_f32(torch, rng.standard_normal((M, d_model)))

    def make(steered):
        Ys = [torch.zeros((M, N), dtype=torch.float32, device="cuda") for _, N, _ in lin]
        ents = []
        for i, ((_, N, K), (c, s)) in enumerate(zip(lin, ws)):
            X = xb if K == 4 * d_model else xa
            st = (dvec, 7.0, strength) if steered and i == 3 else None
            ents.append((ql.FMT_Q4, X, c, s, N, Ys[i], None, ql.ACT_NONE, None, st))
        return Ys, ql.make_group_ep(ents)

    Ys, grp = make(True)
    h = h0.clone()

    def step():
        ql.block_forward_ep(None, group=grp)
        h.copy_(h0)
        ql.steer(h, dvec, 3.0, strength)

    def snapshot():
        return [Y.cpu().numpy().copy() for Y in Ys] + [h.cpu().numpy().copy()]

    eager = {}
    for alpha in (0.5, 0.0, 1.0):
        strength.fill_(alpha)
        step()
        torch.cuda.synchronize()
        eager[alpha] = snapshot()
    Yp, gp = make(False)
    ql.block_forward_ep(None, group=gp)
    torch.cuda.synchronize()
    for a, b in zip(eager[0.0][:4], [Y.cpu().numpy() for Y in Yp]):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert np.array_equal(eager[0.0][4], h0.cpu().numpy())

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()  # sizes the stream's workspace before the capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        step()
    for alpha in (0.5, 0.0, 1.0, 0.0):
        strength.fill_(alpha)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(snapshot(), eager[alpha]):
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), alpha
    Yr = orc.steer(np.zeros((1, d_model)), dvec.cpu().numpy(), 7.0, 1.0)
    assert np.allclose(eager[1.0][3] - eager[0.0][3], Yr, atol=1e-4)
