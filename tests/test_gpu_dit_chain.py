"""A chained DiT denoising step on the GPU: two blocks whose linears feed
one another, captured as one HIP graph, with the steering injection of
Eq. 2 at one block and its strength changed between replays.

Per block (the block's linears and attention as the paper's transformer
runs them; the normalizations and modulation are outside this library):

    qkv   = bf16(hb_in . Wqkv^T + bqkv)
    att   = bf16(attention(qkv))
    h_mid = h_in + att . Wout^T + bout           (hb_mid = bf16(h_mid))
    up    = bf16(GELU(hb_mid . Wup^T + bup))
    h_out = h_mid + up . Wdown^T + bdown [+ alpha ||h_bar|| d]
                                                 (hb_out = bf16(h_out))

with q4 weights.  The bf16 copies hb_* come from the same kernel that
writes the fp32 residual stream (the epilogue's bf16 copy).

Checks against the oracle (fp64), on every row:

1. Stage by stage, element by element (the parity check of the chain):
   each stage's GPU output against the oracle applied to that stage's GPU
   inputs, within the bound of the one operation (the forward bar
   2e-3 * max |P| through the epilogue, the attention bound 2^-8 max |V|,
   one bf16 rounding for bf16 outputs); the bf16 copies must equal the
   round-to-nearest-even of the fp32 outputs bit for bit.  The first
   stage's input is the same on both sides, so by induction the GPU chain
   is the oracle's composition up to these per-stage errors.
2. End to end: the GPU's final residual stream against the oracle's own
   composition (forward, epilogue, attention, steer, with bf16 rounding at
   the same points), held under 1e-2 of max |h|, five times the forward
   bar.  This is a sanity bound, not a derived one: a worst-case
   element-wise propagation (each linear multiplies an element's bound by
   sum_k |w_k|, 4 to 16 here, and the softmax by e^(2D)) overflows within
   two blocks, so the element-by-element parity is check 1's.
"""
import numpy as np
import pytest

import synth_inputs as si
from oracle import oracle as O

pytestmark = pytest.mark.gpu

TOL = 2e-3
GELU_SLOPE = 1.13
SLACK = 1e-6       # fp32 rounding of the epilogue's adds (a few 2^-24)
BF = 2.0 ** -8     # difference of two bf16 roundings, relative
ATT = 2.0 ** -8 + 2.0 ** -16   # the attention kernel's bound, per max |V|


@pytest.fixture(scope="module")
def gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU (run with -m 'not gpu' on a CPU host)")
    from paper_2607_08526_amd import qlinear as ql
    ql.load()
    return torch, ql


def bits_val(b):
    return si.bf16_bits_to_f32(np.asarray(b, np.uint16)).astype(np.float64)


def to_bits(x):
    return si.f32_to_bf16_bits(np.asarray(x, np.float64).astype(np.float32))


def host_bits(t):
    import torch
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


class Model:
    """Two blocks of q4 weights and fp32 biases (host and device copies)."""

    def __init__(self, gpu, orc, d, nblk, seed):
        torch, ql = gpu
        rng = np.random.default_rng(seed)
        self.d, self.blocks = d, []
        for b in range(nblk):
            layers = []
            for name, N, K in si.block_linears(d):
                W = si.weights(rng, N, K)
                cd, sd = ql.quantize(ql.FMT_Q4, torch.from_numpy(W).cuda())
                codes = cd.cpu().numpy().astype(np.uint8)
                scales = sd.cpu().numpy().view(np.uint16)
                bias = (rng.standard_normal(N) * 0.1).astype(np.float32)
                layers.append(dict(N=N, K=K, cd=cd, sd=sd, codes=codes, scales=scales,
                                   Wd=orc.dequantize(O.FMT_Q4, codes, scales, N, K),
                                   bias=bias, bias_d=torch.from_numpy(bias).cuda()))
            self.blocks.append(layers)
        dvec = rng.standard_normal(d).astype(np.float32)
        self.dir = (dvec / np.linalg.norm(dvec.astype(np.float64))).astype(np.float32)
        self.hnorm = 12.0


def gpu_chain(gpu, model, h0, B, T, steer_block):
    """Device buffers of every stage (none reused, so that all of them can
    be checked after a replay) and the call sequence of the chain."""
    torch, ql = gpu
    d, M, H = model.d, B * T, model.d // 64
    h_in = torch.from_numpy(h0).cuda()
    hb_in = torch.from_numpy(to_bits(h0).view(np.int16)).cuda()
    strength = torch.zeros(1, dtype=torch.float32, device="cuda")
    direction = torch.from_numpy(model.dir).cuda()
    st, calls = [], []
    bf = lambda n: torch.empty((M, n), dtype=torch.bfloat16, device="cuda")
    f32 = lambda n: torch.full((M, n), float("nan"), dtype=torch.float32, device="cuda")
    for b, L in enumerate(model.blocks):
        s = dict(qkv=bf(3 * d), att=bf(d), h_mid=f32(d), hb_mid=bf(d), up=bf(4 * d),
                 h_out=f32(d), hb_out=bf(d), h_in=h_in, hb_in=hb_in)
        steer = (direction, model.hnorm, strength) if b == steer_block else None
        g_qkv = ql.make_group_ep([(ql.FMT_Q4, hb_in, L[0]["cd"], L[0]["sd"], L[0]["N"], s["qkv"],
                                   L[0]["bias_d"], ql.ACT_NONE, None)])
        g_out = ql.make_group_ep([(ql.FMT_Q4, s["att"], L[1]["cd"], L[1]["sd"], L[1]["N"],
                                   s["h_mid"], L[1]["bias_d"], ql.ACT_NONE, h_in, None,
                                   s["hb_mid"])])
        g_up = ql.make_group_ep([(ql.FMT_Q4, s["hb_mid"], L[2]["cd"], L[2]["sd"], L[2]["N"],
                                  s["up"], L[2]["bias_d"], ql.ACT_GELU, None)])
        g_down = ql.make_group_ep([(ql.FMT_Q4, s["up"], L[3]["cd"], L[3]["sd"], L[3]["N"],
                                    s["h_out"], L[3]["bias_d"], ql.ACT_NONE, s["h_mid"], steer,
                                    s["hb_out"])])
        qv = s["qkv"].view(torch.int16)
        calls.append((g_qkv, (qv[:, :d], qv[:, d:2 * d], qv[:, 2 * d:], s["att"]), g_out, g_up,
                      g_down))
        st.append(s)
        h_in, hb_in = s["h_out"], s["hb_out"]

    def run():
        for g_qkv, (q, k, v, att), g_out, g_up, g_down in calls:
            ql.block_forward_ep(None, group=g_qkv)
            ql.attention(q, k, v, B, T, H, O=att)
            ql.block_forward_ep(None, group=g_out)
            ql.block_forward_ep(None, group=g_up)
            ql.block_forward_ep(None, group=g_down)

    # the groups hold raw pointers: every tensor they point to must stay
    # alive as long as they are replayed
    run.keep = (direction, strength)
    return st, run, strength


def snapshot(torch, st):
    torch.cuda.synchronize()
    return [{k: v.clone() for k, v in s.items()} for s in st]


def lin_ref(orc, L, X_bits):
    return orc.forward(O.FMT_Q4, X_bits, O.DT_BF16, L["codes"], L["scales"], L["N"])


def check_stages(orc, model, snap, B, T, alpha, steer_block):
    """Check 1: every stage against the oracle on that stage's GPU inputs."""
    d, H = model.d, model.d // 64
    for b, (L, s) in enumerate(zip(model.blocks, snap)):
        g = {k: v.cpu().numpy() if v.dtype.is_floating_point and v.dtype.itemsize == 4 else
             None for k, v in s.items()}
        bits = {k: host_bits(v) for k, v in s.items() if v.dtype.itemsize == 2}
        h_in = s["h_in"].cpu().numpy().astype(np.float64)
        # QKV + bias -> bf16
        P = lin_ref(orc, L[0], bits["hb_in"])
        Yr = orc.epilogue(P, bias=L[0]["bias"])
        lim = TOL * np.max(np.abs(P)) + SLACK * (np.abs(Yr) + np.max(np.abs(P))) + BF * np.abs(Yr)
        assert np.all(np.abs(bits_val(bits["qkv"]) - Yr) <= lim), ("qkv", b)
        # attention -> bf16, on the GPU's qkv
        q = bits["qkv"]
        Or = orc.attention(q[:, :d], q[:, d:2 * d], q[:, 2 * d:], B, T, H, 64)
        Vv = np.abs(bits_val(q[:, 2 * d:]))
        for sb in range(B):
            for hh in range(H):
                rs, cs = slice(sb * T, (sb + 1) * T), slice(hh * 64, (hh + 1) * 64)
                lim = ATT * np.max(Vv[rs, cs]) + BF * np.abs(Or[rs, cs])
                assert np.all(np.abs(bits_val(bits["att"])[rs, cs] - Or[rs, cs]) <= lim), \
                    ("attention", b, sb, hh)
        # out-proj + bias + residual (fp32) and its bf16 copy
        P = lin_ref(orc, L[1], bits["att"])
        Yr = orc.epilogue(P, bias=L[1]["bias"]) + h_in
        lim = TOL * np.max(np.abs(P)) + SLACK * (np.abs(Yr) + np.abs(h_in) + np.max(np.abs(P)))
        assert np.all(np.abs(g["h_mid"] - Yr) <= lim), ("out-proj", b)
        assert np.array_equal(bits["hb_mid"], si.f32_to_bf16_bits(g["h_mid"])), ("hb_mid", b)
        # FFN-up + bias -> GELU -> bf16
        P = lin_ref(orc, L[2], bits["hb_mid"])
        Yr = orc.epilogue(P, bias=L[2]["bias"], act=O.ACT_GELU)
        lim = GELU_SLOPE * TOL * np.max(np.abs(P)) + SLACK * (np.abs(Yr) + np.max(np.abs(P))) \
            + BF * np.abs(Yr)
        assert np.all(np.abs(bits_val(bits["up"]) - Yr) <= lim), ("ffn-up", b)
        # FFN-down + bias + residual (+ steering) and its bf16 copy
        P = lin_ref(orc, L[3], bits["up"])
        h_mid = g["h_mid"].astype(np.float64)
        Yr = orc.epilogue(P, bias=L[3]["bias"]) + h_mid
        if b == steer_block:
            Yr = orc.steer(Yr, model.dir, model.hnorm, alpha)
        lim = TOL * np.max(np.abs(P)) + SLACK * (np.abs(Yr) + np.abs(h_mid) + np.max(np.abs(P)))
        assert np.all(np.abs(g["h_out"] - Yr) <= lim), ("ffn-down", b)
        assert np.array_equal(bits["hb_out"], si.f32_to_bf16_bits(g["h_out"])), ("hb_out", b)


def check_end_to_end(orc, model, h0, h_final, B, T, alpha, steer_block):
    """Check 2: the oracle's own composition, free running from h0."""
    d, H = model.d, model.d // 64
    h = h0.astype(np.float64)
    hb_bits = to_bits(h0)
    for b, L in enumerate(model.blocks):
        qkv_bits = to_bits(orc.epilogue(lin_ref(orc, L[0], hb_bits), bias=L[0]["bias"]))
        att_bits = to_bits(orc.attention(qkv_bits[:, :d], qkv_bits[:, d:2 * d],
                                         qkv_bits[:, 2 * d:], B, T, H, 64))
        h = orc.epilogue(lin_ref(orc, L[1], att_bits), bias=L[1]["bias"]) + h
        hb_bits = to_bits(h)
        up_bits = to_bits(orc.epilogue(lin_ref(orc, L[2], hb_bits), bias=L[2]["bias"],
                                       act=O.ACT_GELU))
        h = orc.epilogue(lin_ref(orc, L[3], up_bits), bias=L[3]["bias"]) + h
        if b == steer_block:
            h = orc.steer(h, model.dir, model.hnorm, alpha)
        hb_bits = to_bits(h)
    err = float(np.max(np.abs(h_final.astype(np.float64) - h)) / np.max(np.abs(h)))
    assert err <= 1e-2, err
    return err


@pytest.mark.parametrize("B,T", [(2, 96), (2, 12)])
def test_dit_chain_graph_with_steering(gpu, orc, B, T):
    """Two chained blocks at d = 256 (4 heads): 2 x 96 tokens (every linear
    on the large-M fp16 path) and 2 x 12 tokens (the few-row kernels).  The
    chain is captured once; replays at strength 0, 0.25 and 0 again each
    equal an eager run at the same strength bit for bit, and pass both
    checks.  Steering changes only what follows the steered block, and
    strength 0 gives back the unsteered result bit for bit."""
    torch, ql = gpu
    d, steer_block = 256, 0
    model = Model(gpu, orc, d, 2, 4200 + T)
    h0 = np.random.default_rng(4300 + T).standard_normal((B * T, d)).astype(np.float32)
    st, run, strength = gpu_chain(gpu, model, h0, B, T, steer_block)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    eager = {}
    for a in (0.0, 0.25):
        strength.fill_(a)
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            run()
        s.synchronize()
        eager[a] = snapshot(torch, st)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        run()
    results = {}
    for a in (0.0, 0.25, 0.0):
        # every output of the chain NaN-filled (the first block's inputs kept)
        for s_ in st:
            for k, t in s_.items():
                if k not in ("h_in", "hb_in"):
                    t.fill_(float("nan"))
        strength.fill_(a)
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            g.replay()
        s.synchronize()
        snap = snapshot(torch, st)
        for s_e, s_r in zip(eager[a], snap):
            for k in s_e:
                assert torch.equal(s_e[k], s_r[k]), (a, k)
        results[a] = snap
    # steering: the steered block's FFN-down output moves by alpha ||h|| d
    # exactly where the epilogue adds it; nothing before it changes
    for k in ("qkv", "att", "h_mid", "hb_mid", "up"):
        assert torch.equal(results[0.0][steer_block][k], results[0.25][steer_block][k])
    assert not torch.equal(results[0.0][steer_block]["h_out"], results[0.25][steer_block]["h_out"])
    for a in (0.0, 0.25):
        check_stages(orc, model, results[a], B, T, a, steer_block)
        e = check_end_to_end(orc, model, h0, results[a][-1]["h_out"].cpu().numpy(), B, T, a,
                             steer_block)
        print(f"B={B} T={T} alpha={a}: end-to-end max err / max|h| {e:.2e}")
