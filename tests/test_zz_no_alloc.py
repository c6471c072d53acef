"""The entry point that allocates nothing (qlinear_block_forward_ep_noalloc),
called through the C ABI, against the pool-workspace entry point it is a
variant of (qlinear_block_forward_ep) and against the oracle.

Both entry points run the same kernels on the same inputs, so their outputs
must agree bit for bit; the outputs must also meet the forward bar against
the oracle (max |Y - Y_ref| / max |Y_ref| <= 2e-3 for bf16 activations, with
the layer epilogue applied to the oracle's product).  Two calls in a row use
the static scratch, the second with a smaller input; a call whose workspace
exceeds the scratch is refused before anything is enqueued.
"""
import numpy as np
import pytest

import synth_inputs as si
from oracle import oracle as O

pytestmark = pytest.mark.gpu

TOL = 2e-3
SCRATCH_BYTES = 128 << 20


@pytest.fixture(scope="module")
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU (run with -m 'not gpu' on a CPU host)")
    from paper_2607_08526_amd import qlinear as ql
    ql.load()
    return torch, ql


def block(gpu, orc, fmt, d, M, seed):
    """One block's four linears at width d and M tokens: quantized weights,
    bf16 activations, and epilogues of every kind (QKV + bias -> bf16, out +
    in-place residual, FFN-up + bias -> GELU -> bf16, FFN-down plain)."""
    torch, ql = gpu
    rng = np.random.default_rng(seed)
    xa = si.activations(rng, M, d, si.DT_BF16)
    xb = si.activations(rng, M, 4 * d, si.DT_BF16)
    dx = lambda X: torch.from_numpy(X.view(np.int16)).cuda()
    xs = {d: (xa, dx(xa)), 4 * d: (xb, dx(xb))}
    layers = []
    for i, (name, N, K) in enumerate(si.block_linears(d)):
        W = si.weights(rng, N, K)
        codes, scales = ql.quantize(fmt, torch.from_numpy(W).cuda())
        bias = rng.standard_normal(N).astype(np.float32) * np.float32(0.5)
        resid = rng.standard_normal((M, N)).astype(np.float32)
        spec = {"qkv": (bias, O.ACT_NONE, None, torch.bfloat16),
                "out": (None, O.ACT_NONE, resid, torch.float32),
                "ffn_up": (bias, O.ACT_GELU, None, torch.bfloat16),
                "ffn_down": (None, O.ACT_NONE, None, torch.float32)}[name]
        layers.append((name, N, K, codes, scales, spec))
    return xs, layers


def entries_for(gpu, xs, layers, fmt, M):
    """Fresh outputs (NaN-filled, residuals re-loaded) and the entry tuples."""
    torch, ql = gpu
    out = []
    for name, N, K, codes, scales, (bias, act, resid, ydt) in layers:
        if resid is not None:
            Y = torch.from_numpy(resid.copy()).cuda()  # in-place residual add
            r = Y
        else:
            Y = torch.full((M, N), float("nan"), dtype=ydt, device="cuda")
            r = None
        b = None if bias is None else torch.from_numpy(bias).cuda()
        out.append((fmt, xs[K][1], codes, scales, N, Y, b, act, r))
    return out


def run_both(gpu, orc, fmt, d, M, seed, check_rows):
    torch, ql = gpu
    xs, layers = block(gpu, orc, fmt, d, M, seed)
    ref = entries_for(gpu, xs, layers, fmt, M)
    ql.block_forward_ep(ref)
    torch.cuda.synchronize()
    got = entries_for(gpu, xs, layers, fmt, M)
    ql.block_forward_ep_noalloc(got)
    torch.cuda.synchronize()
    rows = check_rows
    for (name, N, K, codes, scales, (bias, act, resid, ydt)), e_ref, e_got in zip(layers, ref, got):
        Yref, Ygot = e_ref[5], e_got[5]
        assert bool(torch.isfinite(Ygot).all()), name
        assert torch.equal(Yref, Ygot), f"{name}: no-alloc output differs from the pool path"
        cr = codes.cpu().numpy().astype(np.uint8)
        sr = scales.cpu().numpy().view(np.uint16)
        X = xs[K][0]
        P = orc.forward(fmt, X, O.DT_BF16, cr, sr, N, rows=rows)
        Yr = orc.epilogue(P, bias=bias, act=act, residual=resid, rows=rows)
        Yg = Ygot.float().cpu().numpy().astype(np.float64)[rows]
        bound = 1.13 * TOL * np.max(np.abs(P)) + 1e-6 * (np.abs(Yr) + np.max(np.abs(P)))
        if ydt == torch.bfloat16:
            bound = bound + 2.0 ** -8 * np.abs(Yr)
        assert np.all(np.abs(Yg - Yr) <= bound), name


def test_no_alloc_matches_pool_entry_two_calls(gpu, orc):
    """First call: a block at d = 1024 and 300 tokens (the large-M path,
    pre-pass copies and split partials in the scratch).  Second call, smaller:
    the same block shape at 8 tokens (the streaming kernel with K parts summed
    by a second launch, partials in the scratch)."""
    run_both(gpu, orc, O.FMT_Q4, 1024, 300, 11, np.array([0, 1, 77, 128, 200, 255, 299]))
    run_both(gpu, orc, O.FMT_INT8, 1024, 8, 12, np.arange(8))


def test_no_alloc_refuses_oversized_workspace(gpu, orc):
    """A layer whose fp16 activation copy alone (8192 x 10240 x 2 bytes =
    160 MiB) exceeds the scratch: QL_ERR_UNSUPPORTED, nothing enqueued (Y
    keeps its NaN fill); the same call through the pool entry point works."""
    torch, ql = gpu
    M, N, K = 8192, 64, 10240
    assert M * K * 2 > SCRATCH_BYTES
    X = torch.zeros((M, K), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros((N, K), dtype=torch.float32, device="cuda")
    codes, scales = ql.quantize(O.FMT_Q4, W)
    Y = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    e = [(O.FMT_Q4, X, codes, scales, N, Y, None, O.ACT_NONE, None)]
    with pytest.raises(ql.QLinearError) as err:
        ql.block_forward_ep_noalloc(e)
    assert err.value.status == 5
    torch.cuda.synchronize()
    assert bool(torch.isnan(Y).all())
    ql.block_forward_ep(e)
    torch.cuda.synchronize()
    assert bool((Y == 0).all())


def test_no_alloc_largest_dit_layer(gpu, orc):
    """The DiT step's largest single call: FFN-down (8192 -> 2048, q4) alone
    at 2048 tokens, K cut into parts with partial tiles in the scratch
    (about 101 MB of workspace): bit for bit the pool path, sampled rows
    against the oracle."""
    torch, ql = gpu
    rng = np.random.default_rng(13)
    M, N, K = 2048, 2048, 8192
    W = si.weights(rng, N, K)
    X = si.activations(rng, M, K, si.DT_BF16)
    codes, scales = ql.quantize(O.FMT_Q4, torch.from_numpy(W).cuda())
    Xd = torch.from_numpy(X.view(np.int16)).cuda()
    Ys = [torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda") for _ in range(2)]
    ql.block_forward_ep([(O.FMT_Q4, Xd, codes, scales, N, Ys[0], None, O.ACT_NONE, None)])
    ql.block_forward_ep_noalloc([(O.FMT_Q4, Xd, codes, scales, N, Ys[1], None, O.ACT_NONE, None)])
    torch.cuda.synchronize()
    assert bool(torch.isfinite(Ys[1]).all())
    assert torch.equal(Ys[0], Ys[1])
    rows = np.array([0, 127, 128, 1000, 2047])
    cr = codes.cpu().numpy().astype(np.uint8)
    sr = scales.cpu().numpy().view(np.uint16)
    Yr = orc.forward(O.FMT_Q4, X, O.DT_BF16, cr, sr, N, rows=rows)
    Yg = Ys[1].cpu().numpy().astype(np.float64)[rows]
    assert np.max(np.abs(Yg - Yr)) / np.max(np.abs(Yr)) <= TOL
