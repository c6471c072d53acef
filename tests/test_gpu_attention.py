"""GPU parity of the fused self-attention (qlinear_attention) against the
oracle's fp64 softmax attention.

The kernel rounds the probabilities to bf16 before the value product and
accumulates in fp32; the row sum uses the unrounded probabilities.  Each
probability is off by at most 2^-9 of itself, so |O_gpu - O_ref| <=
2^-9 * max_j |V_j| per channel, plus fp32 and exp2 rounding; the test allows
2^-8 * max|V| (over the sequence and head) + 2^-16 * max|V|.  bf16 outputs
add one rounding (2^-8 |O_ref|).
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


def bf16(rng, shape, scale=1.0):
    return si.f32_to_bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))


def vals(bits):
    return (np.asarray(bits, np.uint32) << 16).view(np.float32).astype(np.float64)


def check(Og, Or, V, B, T, H, dh, obf16):
    Vv = np.abs(vals(V))
    for b in range(B):
        for h in range(H):
            sl = (slice(b * T, (b + 1) * T), slice(h * dh, (h + 1) * dh))
            vmax = np.max(Vv[b * T:(b + 1) * T, h * dh:(h + 1) * dh])
            lim = (2.0 ** -8 + 2.0 ** -16) * vmax
            if obf16:
                lim = lim + 2.0 ** -8 * np.abs(Or[sl])
            err = np.abs(Og[sl] - Or[sl])
            assert np.all(err <= lim), (b, h, np.max(err), vmax)


def run(gpu, Q, K, V, B, T, H, dh, odt="f32", scale=None):
    torch, ql = gpu
    t = lambda A: torch.from_numpy(np.ascontiguousarray(A).view(np.int16)).cuda()
    Og = ql.attention(t(Q), t(K), t(V), B, T, H, dh, scale=scale,
                      odtype=torch.bfloat16 if odt == "bf16" else torch.float32)
    torch.cuda.synchronize()
    return Og.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("B,T,H", [(1, 1, 1), (2, 77, 3), (1, 64, 2), (2, 200, 2),
                                   (1, 129, 1), (1, 1024, 2)])
def test_attention_ragged(gpu, orc, B, T, H):
    """Sequence lengths of one key, a partial key tile, exactly one tile,
    several tiles with a ragged tail and a partial query tile, and 1024."""
    dh = 64
    rng = np.random.default_rng(9000 + B * 1000 + T + H)
    Q, K, V = (bf16(rng, (B * T, H * dh)) for _ in range(3))
    Or = orc.attention(Q, K, V, B, T, H, dh)
    for odt in ("f32", "bf16"):
        check(run(gpu, Q, K, V, B, T, H, dh, odt), Or, V, B, T, H, dh, odt == "bf16")


def test_attention_peaked_and_flat(gpu, orc):
    """Large scores (a few keys take nearly all the weight: the running
    maximum moves across tiles) and zero scale (uniform weights: the mean of
    V)."""
    B, T, H, dh = 1, 300, 2, 64
    rng = np.random.default_rng(9100)
    Q, K, V = bf16(rng, (B * T, H * dh), 3.0), bf16(rng, (B * T, H * dh), 3.0), \
        bf16(rng, (B * T, H * dh))
    check(run(gpu, Q, K, V, B, T, H, dh), orc.attention(Q, K, V, B, T, H, dh), V, B, T, H,
          dh, False)
    Og = run(gpu, Q, K, V, B, T, H, dh, scale=0.0)
    assert np.allclose(Og, np.repeat(vals(V).mean(axis=0, keepdims=True), T, axis=0),
                       atol=2.0 ** -8 * np.max(np.abs(vals(V))))


def test_attention_fused_qkv_full_size_sampled(gpu, orc):
    """The DiT shape: 2 sequences (the guidance branches) x 1024 tokens,
    d = 2048 (32 heads of 64), read in place from one fused QKV tensor
    [2048][6144] (ld = 3 d).  O starts NaN-filled and must be finite
    everywhere; 64 query rows (one in every 32-row band of both sequences,
    plus each sequence's first and last row) x every head against the
    oracle; a second call repeats the first bit for bit."""
    torch, ql = gpu
    B, T, H, dh = 2, 1024, 32, 64
    d = H * dh
    rng = np.random.default_rng(9200)
    QKV = bf16(rng, (B * T, 3 * d))
    qkv = torch.from_numpy(QKV.view(np.int16)).cuda()
    O1 = torch.full((B * T, d), float("nan"), dtype=torch.float32, device="cuda")
    Og = ql.attention(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:], B, T, H, dh, O=O1)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(Og).all())
    rows = {0, T - 1, T, 2 * T - 1}
    for b0 in range(0, B * T, 32):
        rows.add(int(rng.integers(b0, b0 + 32)))
    rows = np.array(sorted(rows))
    assert len(rows) >= 64
    Or = orc.attention(QKV[:, :d], QKV[:, d:2 * d], QKV[:, 2 * d:], B, T, H, dh, rows=rows)
    Vv = np.abs(vals(QKV[:, 2 * d:]))
    Ogh = Og.cpu().numpy()[rows]
    for b in range(B):
        sel = (rows >= b * T) & (rows < (b + 1) * T)
        for h in range(H):
            cols = slice(h * dh, (h + 1) * dh)
            vmax = np.max(Vv[b * T:(b + 1) * T, cols])
            lim = (2.0 ** -8 + 2.0 ** -16) * vmax
            assert np.max(np.abs(Ogh[sel, cols] - Or[sel, cols])) <= lim, (b, h)
    Og2 = ql.attention(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:], B, T, H, dh)
    torch.cuda.synchronize()
    assert torch.equal(Og, Og2)
