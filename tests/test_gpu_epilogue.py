"""GPU parity of the fused layer epilogue (qlinear_forward_ep and
qlinear_block_forward_ep): Y = act(X . W^T + bias) + residual, stored as fp32
or bf16, against the oracle's product followed by its epilogue (fp64).

Bound, element by element: the product's error is at most TOL * max|P|
(the forward bar); the GELU's slope never exceeds 1.13, so after the
epilogue the error is at most 1.13 * TOL * max|P| plus fp32 rounding of the
epilogue's own operations (a few units of 2^-24 of the values involved,
allowed as 1e-6 of them).  bf16 outputs add one rounding to bf16 (at most
2^-9 of |Y|, allowed as 2^-8).  Exact constructions (integer products,
integer bias and residual) must match exactly, and their bf16 outputs must
be torch's round-to-nearest-even conversion of the exact value.
"""
import numpy as np
import pytest

import synth_inputs as si
from oracle import oracle as O

pytestmark = pytest.mark.gpu

TOL = {O.DT_BF16: 2e-3, O.DT_F32: 1e-5}
GELU_SLOPE = 1.13


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


def host_y(torch, Y):
    return Y.float().cpu().numpy().astype(np.float64)


def check(Yg, Pr, Yr, bias, xdt, ybf16, what):
    bmax = 0.0 if bias is None else float(np.max(np.abs(bias)))
    pmax = float(np.max(np.abs(Pr)))
    bound = GELU_SLOPE * TOL[xdt] * pmax + 1e-6 * (np.abs(Yr) + pmax + bmax)
    if ybf16:
        bound = bound + 2.0 ** -8 * np.abs(Yr)
    bad = np.abs(Yg - Yr) > bound
    assert not bad.any(), (what, np.argwhere(bad)[:4], Yg[bad][:4], Yr[bad][:4])


# (fmt, xdt, M, N, K): one shape per kernel that stores final outputs
PATHS = [
    (O.FMT_Q4, O.DT_BF16, 3, 4097, 2048),     # wavefront GEMV (M <= 4)
    (O.FMT_INT8, O.DT_BF16, 16, 4100, 512),   # weight streaming, one K part
    (O.FMT_Q4, O.DT_BF16, 8, 2049, 8192),     # weight streaming, K parts + sum launch
    (O.FMT_INT8, O.DT_BF16, 20, 70, 320),     # small-M MFMA (K % 256 != 0)
    (O.FMT_Q4, O.DT_F32, 40, 200, 320),       # MFMA kernel, fp32 activations
    (O.FMT_INT8, O.DT_BF16, 200, 77, 288),    # MFMA kernel, 128-row tiles
    (O.FMT_Q4, O.DT_BF16, 300, 520, 1280),    # fp16 path, no split
    (O.FMT_INT8, O.DT_BF16, 300, 520, 4096),  # fp16 path, K parts + sum launch
    (O.FMT_Q4, O.DT_BF16, 129, 17, 1024),     # fp16 path, ragged tiles, N % 4 != 0
]

# (bias, act, residual, Y dtype): every operation, each store width
EPILOGUES = [
    (True, O.ACT_GELU, True, "f32"),
    (True, O.ACT_GELU, False, "bf16"),
    (False, O.ACT_NONE, True, "bf16"),
    (False, O.ACT_NONE, "inplace", "f32"),
    (True, O.ACT_NONE, False, "f32"),
]


def run_ep(gpu, fmt, X, xdt, cd, sd, N, bias, act, resid, ydt):
    torch, ql = gpu
    M = X.shape[0]
    Xd = dev_x(torch, X, xdt)
    bd = None if bias is None else dev_f32(torch, bias)
    if resid is not None and ydt == "inplace":
        Y = dev_f32(torch, resid)
        rd = Y
    else:
        dt = torch.bfloat16 if ydt == "bf16" else torch.float32
        Y = torch.full((M, N), float("nan"), dtype=dt, device="cuda")
        rd = None if resid is None else dev_f32(torch, resid)
    ql.forward_ep(fmt, Xd, cd, sd, N, Y=Y, bias=bd, act=act, residual=rd)
    torch.cuda.synchronize()
    return host_y(torch, Y)


@pytest.mark.parametrize("fmt,xdt,M,N,K", PATHS)
def test_epilogue_every_path(gpu, orc, fmt, xdt, M, N, K):
    torch, ql = gpu
    W, X = si.small_case(3000 + M + N + K + fmt, M, N, K, xdt)
    cd, sd = ql.quantize(fmt, dev_f32(torch, W))
    cr, sr = orc.quantize(fmt, W)
    assert np.array_equal(cd.cpu().numpy().astype(np.uint8), cr)
    Pr = orc.forward(fmt, X, xdt, cr, sr, N)
    rng = np.random.default_rng(M + N + K)
    for use_b, act, use_r, ydt in EPILOGUES:
        bias = (rng.standard_normal(N) * 0.5).astype(np.float32) if use_b else None
        resid = rng.standard_normal((M, N)).astype(np.float32) if use_r else None
        Yr = orc.epilogue(Pr, bias, act, resid)
        Yg = run_ep(gpu, fmt, X, xdt, cd, sd, N, bias, act, resid,
                    "inplace" if use_r == "inplace" else ydt)
        check(Yg, Pr, Yr, bias, xdt, ydt == "bf16", (M, N, K, use_b, act, use_r, ydt))


def test_epilogue_f16_weights(gpu, orc):
    """fp16 weights take the same epilogue (the fp16 path's kernel at small
    and large M, with and without K parts)."""
    torch, ql = gpu
    for (M, N, K) in ((2, 40, 256), (214, 520, 1280), (128, 64, 8192)):
        W, X = si.small_case(3100 + M + N + K, M, N, K)
        W16 = np.ascontiguousarray(W, dtype=np.float32).astype(np.float16).view(np.uint16)
        wd = torch.from_numpy(W16.view(np.int16)).cuda()
        Pr = orc.forward_f16(X, O.DT_BF16, W16)
        rng = np.random.default_rng(N)
        bias = (rng.standard_normal(N) * 0.5).astype(np.float32)
        resid = rng.standard_normal((M, N)).astype(np.float32)
        for act, ydt in ((O.ACT_GELU, "f32"), (O.ACT_GELU, "bf16")):
            Yr = orc.epilogue(Pr, bias, act, resid)
            Yg = run_ep(gpu, ql.FMT_F16, X, O.DT_BF16, wd, None, N, bias, act, resid, ydt)
            check(Yg, Pr, Yr, bias, O.DT_BF16, ydt == "bf16", (M, N, K, ydt))


@pytest.mark.parametrize("M", [3, 16, 40, 200])
def test_epilogue_exact_and_bf16_rounding(gpu, orc, M):
    """W = c * 2^-12 with integer activations, an integer bias and residual:
    P + bias + residual is exact in fp32, so fp32 outputs must equal it and
    bf16 outputs must be its round-to-nearest-even bf16 value (torch's CPU
    conversion), ties included."""
    torch, ql = gpu
    rng = np.random.default_rng(3200 + M)
    N, K = 80, 512
    C = rng.integers(-127, 128, (N, K))
    C.reshape(N, K // 32, 32)[:, :, 3] = rng.choice([-127, 127], (N, K // 32))
    W = (C * 2.0 ** -12).astype(np.float32)
    cd, sd = ql.quantize(O.FMT_INT8, dev_f32(torch, W))
    Xi = rng.integers(-8, 9, (M, K)).astype(np.float32)
    X = si.f32_to_bf16_bits(Xi)
    bias = rng.integers(-1000, 1001, N).astype(np.float32)
    resid = rng.integers(-1000, 1001, (M, N)).astype(np.float32)
    exact = ((Xi.astype(np.int64) @ C.T) * 2.0 ** -12 + bias.astype(np.float64)[None, :]
             + resid.astype(np.float64))
    assert np.array_equal(exact.astype(np.float32).astype(np.float64), exact)
    Yf = run_ep(gpu, O.FMT_INT8, X, O.DT_BF16, cd, sd, N, bias, O.ACT_NONE, resid, "f32")
    assert np.array_equal(Yf, exact)
    Yb = run_ep(gpu, O.FMT_INT8, X, O.DT_BF16, cd, sd, N, bias, O.ACT_NONE, resid, "bf16")
    want = torch.from_numpy(exact.astype(np.float32)).to(torch.bfloat16).float().numpy()
    assert np.array_equal(Yb, want.astype(np.float64))


def test_epilogue_gelu_special_values(gpu, orc):
    """Zero products give GELU(0) = 0; a product of -40 gives -0 or a
    denormal-free tiny value in fp32 (the oracle's value rounds to zero);
    large positive products pass through unchanged."""
    torch, ql = gpu
    M, N, K = 4, 8, 256
    W = np.zeros((N, K), np.float32)
    W[:, 0] = [0.0, -40.0, 40.0, 1.0, -1.0, 3.0, -3.0, 0.5]
    cd, sd = ql.quantize(O.FMT_INT8, dev_f32(torch, W))
    cr, sr = orc.quantize(O.FMT_INT8, W)
    Xi = np.zeros((M, K), np.float32)
    Xi[:, 0] = 1.0
    X = si.f32_to_bf16_bits(Xi)
    Pr = orc.forward(O.FMT_INT8, X, O.DT_BF16, cr, sr, N)
    Yr = orc.epilogue(Pr, None, O.ACT_GELU, None)
    Yg = run_ep(gpu, O.FMT_INT8, X, O.DT_BF16, cd, sd, N, None, O.ACT_GELU, None, "f32")
    assert np.all(Yg[:, 0] == 0.0)
    assert np.all(np.abs(Yg[:, 1]) < 1e-30)
    assert np.all(Yg[:, 2] == Pr[:, 2])
    assert np.max(np.abs(Yg - Yr)) <= 4e-6 * np.max(np.abs(Yr))


def test_block_forward_ep_grouped(gpu, orc):
    """One grouped call with a different epilogue per layer: the fp16 path's
    grouped launch with K parts (mixed reduction lengths over two
    activations; summed by the separate launch, which applies the
    epilogues), and a small-M group on the streaming kernels."""
    torch, ql = gpu
    for M, shapes in ((384, [(700, 512), (256, 4096), (1000, 512)]),
                      (24, [(3072, 1024), (1024, 4096), (4096, 1024)])):
        for fmt in (O.FMT_INT8, O.FMT_Q4):
            _, xa = si.small_case(3300 + M, M, 1, 1024 if M == 24 else 512)
            _, xb = si.small_case(3301 + M, M, 1, 4096)
            eps = [(True, O.ACT_GELU, None, "bf16"), (False, O.ACT_NONE, "inplace", "f32"),
                   (True, O.ACT_GELU, True, "f32")]
            rng = np.random.default_rng(M + fmt)
            entries, refs = [], []
            for i, ((N, K), (use_b, act, use_r, ydt)) in enumerate(zip(shapes, eps)):
                W, _ = si.small_case(3310 + i + M, 1, N, K)
                cd, sd = ql.quantize(fmt, dev_f32(torch, W))
                cr, sr = orc.quantize(fmt, W)
                X = xb if K == 4096 else xa
                bias = (rng.standard_normal(N) * 0.5).astype(np.float32) if use_b else None
                resid = rng.standard_normal((M, N)).astype(np.float32) if use_r else None
                if use_r == "inplace":
                    Y = dev_f32(torch, resid)
                    rd = Y
                else:
                    dt = torch.bfloat16 if ydt == "bf16" else torch.float32
                    Y = torch.full((M, N), float("nan"), dtype=dt, device="cuda")
                    rd = None if resid is None else dev_f32(torch, resid)
                bd = None if bias is None else dev_f32(torch, bias)
                entries.append((fmt, dev_x(torch, X, O.DT_BF16), cd, sd, N, Y, bd, act, rd))
                Pr = orc.forward(fmt, X, O.DT_BF16, cr, sr, N)
                refs.append((Pr, orc.epilogue(Pr, bias, act, resid), bias, ydt == "bf16"))
            ql.block_forward_ep(entries)
            torch.cuda.synchronize()
            for e, (Pr, Yr, bias, yb) in zip(entries, refs):
                check(host_y(torch, e[5]), Pr, Yr, bias, O.DT_BF16, yb, (M, fmt, e[4]))


def test_block_forward_ep_routed_layers(gpu, orc):
    """A grouped call on the large-M path mixing layers whose epilogue takes
    groups of four outputs with layers that the host routes through plain
    partials and the sum launch: an odd N, and a bias that is 4-byte but not
    16-byte aligned; long reductions cut into parts in the same launch."""
    torch, ql = gpu
    M = 384
    _, xa = si.small_case(3400, M, 1, 512)
    _, xb = si.small_case(3401, M, 1, 4096)
    rng = np.random.default_rng(3402)
    shapes = [(702, 512), (256, 4096), (1000, 512), (257, 4096)]
    entries, refs = [], []
    for fmt in (O.FMT_Q4, O.FMT_INT8):
        entries.clear()
        refs.clear()
        for i, (N, K) in enumerate(shapes):
            W, _ = si.small_case(3410 + i, 1, N, K)
            cd, sd = ql.quantize(fmt, dev_f32(torch, W))
            cr, sr = orc.quantize(fmt, W)
            X = xb if K == 4096 else xa
            bias = (rng.standard_normal(N) * 0.5).astype(np.float32)
            if i == 2:  # a bias view one float past a 16-byte boundary
                store = dev_f32(torch, np.concatenate([[0.0], bias]).astype(np.float32))
                bd = store[1:]
            else:
                bd = dev_f32(torch, bias)
            act = O.ACT_GELU if i % 2 else O.ACT_NONE
            resid = rng.standard_normal((M, N)).astype(np.float32)
            Y = dev_f32(torch, resid)  # in-place residual add
            entries.append((fmt, dev_x(torch, X, O.DT_BF16), cd, sd, N, Y, bd, act, Y))
            P = orc.forward(fmt, X, O.DT_BF16, cr, sr, N)
            refs.append((P, orc.epilogue(P, bias, act, resid), bias))
        ql.block_forward_ep(entries)
        torch.cuda.synchronize()
        for e, (P, Yr, bias) in zip(entries, refs):
            check(host_y(torch, e[5]), P, Yr, bias, O.DT_BF16, False, (fmt, e[4]))


@pytest.mark.parametrize("fmt,xdt,M,N,K", PATHS)
def test_epilogue_bf16_copy_every_path(gpu, orc, fmt, xdt, M, N, K):
    """The bf16 copy of an fp32 output (the residual stream's copy that the
    next linear reads), on every store path: an in-place residual add with
    bias and the copy; the fp32 output within the epilogue bound, and the
    copy equal to the round-to-nearest-even bf16 of the fp32 output, bit for
    bit (NaN-filled beforehand, so every element is written).  A copy of a
    bf16 output, or one aliasing Y or the residual, is refused."""
    torch, ql = gpu
    W, X = si.small_case(3500 + M + N + K + fmt, M, N, K, xdt)
    cd, sd = ql.quantize(fmt, dev_f32(torch, W))
    cr, sr = orc.quantize(fmt, W)
    Pr = orc.forward(fmt, X, xdt, cr, sr, N)
    rng = np.random.default_rng(3600 + M + N)
    bias = (rng.standard_normal(N) * 0.5).astype(np.float32)
    resid = rng.standard_normal((M, N)).astype(np.float32)
    Xd = dev_x(torch, X, xdt)
    Y = dev_f32(torch, resid)
    copy = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
    ql.forward_ep(fmt, Xd, cd, sd, N, Y=Y, bias=dev_f32(torch, bias), residual=Y, ycopy=copy)
    torch.cuda.synchronize()
    Yg = host_y(torch, Y)
    check(Yg, Pr, orc.epilogue(Pr, bias, O.ACT_NONE, resid), bias, xdt, False, (M, N, K))
    want = si.f32_to_bf16_bits(Yg.astype(np.float32))
    assert np.array_equal(copy.view(torch.int16).cpu().numpy().view(np.uint16), want)
    Yb = torch.zeros((M, N), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError):  # a copy of a bf16 output
        ql.forward_ep(fmt, Xd, cd, sd, N, Y=Yb, ycopy=copy)
    alias = Y.view(-1).view(torch.bfloat16)[:M * N].view(M, N)  # same address as Y
    with pytest.raises(ql.QLinearError) as err:
        ql.forward_ep(fmt, Xd, cd, sd, N, Y=Y, residual=Y, ycopy=alias)
    assert err.value.status == 1


def test_block_forward_ep_in_kernel_reduction(gpu, orc):
    """A DiT block at d = 1024 and 768 tokens, the shape class (a few hundred
    to ~1500 tokens) whose split plan adds the K parts inside the large-M
    kernel: more parts than one wave of workgroups (FFN-down in 4 parts of
    16 steps, the other layers in 2 of 8), each part stores its partial
    tile, and the last part to arrive adds them in part order and applies
    the layer's epilogue (QKV + bias -> bf16; out-projection + bias + a
    residual; FFN-up + bias -> GELU -> bf16; FFN-down + bias added in place
    into its residual with a bf16 copy).  Every output starts NaN-filled and
    must be finite everywhere; 64 rows (one in every 128-row tile) x all
    columns against the oracle; the copy equals the rounded fp32 output bit
    for bit; a second call repeats the first bit for bit."""
    torch, ql = gpu
    M, d = 768, 1024
    rng = np.random.default_rng(3500)
    rows = np.array(sorted({0, M - 1} | {int(rng.integers(t, t + 128)) for t in range(0, M, 128)}
                           | set(rng.choice(M, 56, replace=False).tolist())), dtype=np.int64)
    _, xa = si.small_case(3501, M, 1, d)
    _, xb = si.small_case(3502, M, 1, 4 * d)
    for fmt in (O.FMT_Q4, O.FMT_INT8):
        entries, refs = [], []
        copy = torch.full((M, d), -1, dtype=torch.int16, device="cuda")
        for i, (_, N, K) in enumerate(si.block_linears(d)):
            W, _ = si.small_case(3510 + i, 1, N, K)
            cd, sd = ql.quantize(fmt, dev_f32(torch, W))
            cr, sr = orc.quantize(fmt, W)
            X = xb if K == 4 * d else xa
            bias = (rng.standard_normal(N) * 0.5).astype(np.float32)
            act = O.ACT_GELU if i == 2 else O.ACT_NONE
            resid = rng.standard_normal((M, N)).astype(np.float32) if i in (1, 3) else None
            ybf16 = i in (0, 2)
            if i == 3:
                resid3 = resid
                Y = dev_f32(torch, resid)  # in place, with its bf16 copy
                rd, yc = Y, copy.view(torch.bfloat16)
            else:
                Y = torch.full((M, N), float("nan"), device="cuda",
                               dtype=torch.bfloat16 if ybf16 else torch.float32)
                rd, yc = (None if resid is None else dev_f32(torch, resid)), None
            entries.append((fmt, dev_x(torch, X, O.DT_BF16), cd, sd, N, Y, dev_f32(torch, bias),
                            act, rd, None, yc))
            Pr = orc.forward(fmt, X, O.DT_BF16, cr, sr, N, rows=rows)
            Yr = orc.epilogue(Pr, bias, act, None if resid is None else resid[rows])
            refs.append((Pr, Yr, bias, ybf16))
        g = ql.make_group_ep(entries)
        ql.block_forward_ep(None, group=g)
        torch.cuda.synchronize()
        first = [e[5].clone() for e in entries] + [copy.clone()]
        for e, (Pr, Yr, bias, yb) in zip(entries, refs):
            assert bool(torch.isfinite(e[5].float()).all()), (fmt, e[4])
            check(host_y(torch, e[5])[rows], Pr, Yr, bias, O.DT_BF16, yb, (fmt, e[4]))
        assert torch.equal(copy.view(torch.bfloat16), entries[3][5].to(torch.bfloat16))
        # again from the same inputs: NaN-filled outputs, the in-place layer
        # back at its residual
        for i, e in enumerate(entries):
            if i == 3:
                e[5].copy_(dev_f32(torch, resid3))
            else:
                e[5].fill_(float("nan"))
        copy.fill_(-1)
        ql.block_forward_ep(None, group=g)
        torch.cuda.synchronize()
        again = [e[5] for e in entries] + [copy]
        assert all(torch.equal(a_, b_) for a_, b_ in zip(first, again)), fmt
