"""Seeded synthetic inputs for the block-quantized linear layers.

This module only draws inputs; it holds none of the quantizer's or the
product's arithmetic, so both the fp64 oracle's tests and the GPU library's
tests and benchmark can take their inputs from here.

Recipe (stands in for the trained DiT weights and real prompts, which are not
available): weights W ~ N(0, 0.02) drawn as fp32 [N][K] (out x in);
activations X ~ N(0, 1) drawn as fp32 [M][K] and, for bf16 workloads, rounded
to bf16 (round to nearest even).  Everything comes from
numpy.random.default_rng(seed).standard_normal(..., dtype=float32); when one
generator yields both, W is drawn before X.

Workloads (the DiT shapes the paper's medium model implies: width d, FFN 4d,
2 classifier-free-guidance branches x 1024 latent frames = 2048 tokens):
  single_int8   int8, W 1024x1024, X fp32 64x1024, seed 0
  single_q4     q4 FFN-up, W 6144x1536, X bf16 256x1536, seed 1
  block_int8    one block d=2048: QKV 2048->6144, out 2048->2048,
                FFN-up 2048->8192, FFN-down 8192->2048; W seeds 2..5,
                X bf16 2048x2048 and 2048x8192 from seed 6
  step_q4       24 such blocks, q4; W seeds 100 + 4*block + i, X as above
  skinny        int8/q4 x (N,K) in {(8192,2048),(2048,8192)} x M in
                {1,8,32,128}, bf16 X; W seed 200 + variant, X seed 300 + M
  paper widths  the paper's two DiT configurations (small-music: 20 blocks at
                d = 1024; medium: 24 blocks at d = 1536; Related Work,
                generative audio models, and Experiments, setup) at the
                token count of one 10 s clip: ~107 latent frames at ~10.7 Hz
                (Methodology, the runtime) x 2 guidance branches = 214;
                W seeds 1000 * (width index + 1) + 4 * block + i, X seed
                900 + width index
"""
import numpy as np

FMT_Q4 = 4
FMT_INT8 = 8
DT_F32 = 0
DT_BF16 = 1

W_STD = np.float32(0.02)

D_MODEL = 2048
TOKENS = 2 * 1024
N_BLOCKS = 24

# (name, N, K) of the four linears of one DiT block at width d
def block_linears(d=D_MODEL):
    return [("qkv", 3 * d, d), ("out", d, d), ("ffn_up", 4 * d, d), ("ffn_down", d, 4 * d)]


# (name, d, blocks) of the paper's DiT configurations, and the tokens of a
# 10 s clip with both guidance branches
PAPER_WIDTHS = [("small_music", 1024, 20), ("medium", 1536, 24)]
PAPER_TOKENS = 2 * 107

SKINNY_SHAPES = [(8192, 2048), (2048, 8192)]
SKINNY_M = [1, 8, 32, 128]


def f32_to_bf16_bits(x):
    """bf16 bit patterns (uint16) of fp32 values, round to nearest even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    nan = np.isnan(x)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    out = rounded.astype(np.uint16)
    out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b):
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def weights(rng, N, K):
    return rng.standard_normal((N, K), dtype=np.float32) * W_STD


def activations(rng, M, K, xdt):
    x = rng.standard_normal((M, K), dtype=np.float32)
    return x if xdt == DT_F32 else f32_to_bf16_bits(x)


def single_int8():
    rng = np.random.default_rng(0)
    W = weights(rng, 1024, 1024)
    X = activations(rng, 64, 1024, DT_F32)
    return dict(fmt=FMT_INT8, W=W, X=X, xdt=DT_F32)


def single_q4():
    rng = np.random.default_rng(1)
    W = weights(rng, 6144, 1536)
    X = activations(rng, 256, 1536, DT_BF16)
    return dict(fmt=FMT_Q4, W=W, X=X, xdt=DT_BF16)


def block_activations(M=TOKENS, d=D_MODEL, seed=6):
    """(X of width d shared by QKV/out/FFN-up, X of width 4d for FFN-down)."""
    rng = np.random.default_rng(seed)
    xa = activations(rng, M, d, DT_BF16)
    xb = activations(rng, M, 4 * d, DT_BF16)
    return xa, xb


def block_weights(i, seed_base, d=D_MODEL):
    name, N, K = block_linears(d)[i]
    return weights(np.random.default_rng(seed_base + i), N, K)


def block_int8_weight(i, d=D_MODEL):
    return block_weights(i, 2, d)


def step_q4_weight(blk, i, d=D_MODEL):
    return block_weights(i, 100 + 4 * blk, d)


def paper_weight(w, blk, i):
    """Weight i of block blk of paper width w (index into PAPER_WIDTHS)."""
    d = PAPER_WIDTHS[w][1]
    return block_weights(i, 1000 * (w + 1) + 4 * blk, d)


def paper_activations(w):
    d = PAPER_WIDTHS[w][1]
    return block_activations(M=PAPER_TOKENS, d=d, seed=900 + w)


def skinny_variants():
    """[(variant index, fmt, N, K)] in seed order."""
    out = []
    v = 0
    for fmt in (FMT_INT8, FMT_Q4):
        for N, K in SKINNY_SHAPES:
            out.append((v, fmt, N, K))
            v += 1
    return out


def skinny_weight(v, N, K):
    return weights(np.random.default_rng(200 + v), N, K)


def skinny_activations(M, K):
    return activations(np.random.default_rng(300 + M), M, K, DT_BF16)


def small_case(seed, M, N, K, xdt=DT_BF16, w_std=W_STD):
    """A small random case (same recipe) for parity tests at ragged sizes."""
    rng = np.random.default_rng(seed)
    W = rng.standard_normal((N, K), dtype=np.float32) * np.float32(w_std)
    X = activations(rng, M, K, xdt)
    return W, X
