"""The Python binding's argument checks (CPU only).

The library takes bare pointers and sizes, so the binding must refuse
tensors whose dtype, shape or layout does not match what it passes on:
such a call would otherwise read or write out of bounds on the device.
These checks run before the library is loaded, so host tensors exercise
them here; a well-formed host tensor is refused for not being on the
device.
"""
import pytest
import torch

from paper_2607_08526_amd import qlinear as ql

M, N, K = 4, 64, 128


def x_bf16(m=M, k=K):
    return torch.zeros((m, k), dtype=torch.bfloat16)


def weights(fmt=ql.FMT_INT8, n=N, k=K):
    codes = torch.zeros((n, k if fmt == ql.FMT_INT8 else k // 2), dtype=torch.uint8)
    scales = torch.zeros((n, k // 32), dtype=torch.int16)
    return codes, scales


def test_quantize_rejects():
    with pytest.raises(TypeError):
        ql.quantize(ql.FMT_INT8, torch.zeros((N, K), dtype=torch.float16))
    with pytest.raises(ValueError):
        ql.quantize(ql.FMT_INT8, torch.zeros((N, K), dtype=torch.float32).t())  # not contiguous
    with pytest.raises(ValueError):
        ql.quantize(ql.FMT_INT8, torch.zeros((N, 100), dtype=torch.float32))  # K % 32
    with pytest.raises(ValueError):
        ql.quantize(ql.FMT_F16, torch.zeros((N, K), dtype=torch.float32))  # not a quantized fmt
    codes, scales = weights(ql.FMT_Q4)
    with pytest.raises(ValueError):  # int8 codes shape needed, q4 given
        ql.quantize(ql.FMT_INT8, torch.zeros((N, K), dtype=torch.float32), codes, scales)
    with pytest.raises(ValueError):  # host tensor
        ql.quantize(ql.FMT_INT8, torch.zeros((N, K), dtype=torch.float32))


def test_forward_rejects():
    codes, scales = weights()
    with pytest.raises(TypeError):  # fp16 activations are not a taken dtype
        ql.forward(ql.FMT_INT8, torch.zeros((M, K), dtype=torch.float16), codes, scales, N)
    with pytest.raises(ValueError):  # X not 2-D
        ql.forward(ql.FMT_INT8, torch.zeros(K, dtype=torch.bfloat16), codes, scales, N)
    with pytest.raises(ValueError):  # X not contiguous
        ql.forward(ql.FMT_INT8, torch.zeros((K, M), dtype=torch.bfloat16).t(), codes, scales, N)
    with pytest.raises(ValueError):  # codes for another N
        ql.forward(ql.FMT_INT8, x_bf16(), codes, scales, N + 1)
    with pytest.raises(ValueError):  # q4 codes read as int8
        ql.forward(ql.FMT_INT8, x_bf16(), weights(ql.FMT_Q4)[0], scales, N)
    with pytest.raises(ValueError):  # scales shape
        ql.forward(ql.FMT_INT8, x_bf16(), codes, scales[:, :2], N)
    with pytest.raises(TypeError):  # scales dtype (4-byte)
        ql.forward(ql.FMT_INT8, x_bf16(), codes, scales.float(), N)
    with pytest.raises(TypeError):  # Y must be fp32
        ql.forward(ql.FMT_INT8, x_bf16(), codes, scales, N, Y=torch.zeros((M, N), dtype=torch.bfloat16))
    with pytest.raises(ValueError):  # Y shape
        ql.forward(ql.FMT_INT8, x_bf16(), codes, scales, N, Y=torch.zeros((M, N - 1)))
    with pytest.raises(ValueError):  # Y not contiguous
        ql.forward(ql.FMT_INT8, x_bf16(), codes, scales, N, Y=torch.zeros((N, M)).t())
    with pytest.raises(ValueError):  # fp16 weights of the wrong shape
        ql.forward(ql.FMT_F16, x_bf16(), torch.zeros((N, K + 2), dtype=torch.float16), None, N)
    with pytest.raises(ValueError):  # well formed, but host memory
        ql.forward(ql.FMT_INT8, x_bf16(), codes, scales, N)


def test_forward_ep_rejects():
    codes, scales = weights()
    with pytest.raises(TypeError):  # fp16 Y
        ql.forward_ep(ql.FMT_INT8, x_bf16(), codes, scales, N, Y=torch.zeros((M, N), dtype=torch.float16))
    with pytest.raises(ValueError):  # bias length
        ql.forward_ep(ql.FMT_INT8, x_bf16(), codes, scales, N, bias=torch.zeros(N - 1))
    with pytest.raises(TypeError):  # bias dtype
        ql.forward_ep(ql.FMT_INT8, x_bf16(), codes, scales, N, bias=torch.zeros(N, dtype=torch.float64))
    with pytest.raises(ValueError):  # residual shape
        ql.forward_ep(ql.FMT_INT8, x_bf16(), codes, scales, N, residual=torch.zeros((M + 1, N)))
    with pytest.raises(ValueError):  # steering direction length
        ql.forward_ep(ql.FMT_INT8, x_bf16(), codes, scales, N,
                      steer=(torch.zeros(N + 1), 1.0, torch.zeros(1)))
    with pytest.raises(ValueError):  # empty strength
        ql.forward_ep(ql.FMT_INT8, x_bf16(), codes, scales, N,
                      steer=(torch.zeros(N), 1.0, torch.zeros(0)))


def test_group_rejects():
    codes, scales = weights()
    good = (ql.FMT_INT8, x_bf16(), codes, scales, N, torch.zeros((M, N)))
    with pytest.raises(ValueError):
        ql.make_group([])
    with pytest.raises(ValueError):
        ql.make_group([good] * (ql.MAX_GROUP + 1))
    with pytest.raises(ValueError):  # Y of another layer's shape
        ql.make_group([good, (ql.FMT_INT8, x_bf16(), codes, scales, N, torch.zeros((M, 2 * N)))])
    with pytest.raises(ValueError):
        ql.make_group([good])  # host tensors
    with pytest.raises(ValueError):  # residual shape in an epilogue group
        ql.make_group_ep([good + (None, ql.ACT_NONE, torch.zeros((M, N + 1)))])


def test_w8a8_steer_rejects():
    codes, scales = weights()
    qx = torch.zeros((M, K), dtype=torch.int8)
    with pytest.raises(TypeError):  # uint8 activation codes
        ql.forward_w8a8(qx.to(torch.uint8), torch.zeros(M, dtype=torch.int16), codes, scales, N)
    with pytest.raises(ValueError):  # one scale per row
        ql.forward_w8a8(qx, torch.zeros(M + 1, dtype=torch.int16), codes, scales, N)
    with pytest.raises(ValueError):  # q4 weights
        ql.forward_w8a8(qx, torch.zeros(M, dtype=torch.int16), weights(ql.FMT_Q4)[0], scales, N)
    with pytest.raises(ValueError):
        ql.quantize_act(x_bf16(), qx=torch.zeros((M, K - 32), dtype=torch.int8))
    with pytest.raises(TypeError):
        ql.quantize_act(x_bf16(), sx=torch.zeros(M, dtype=torch.float32))
    with pytest.raises(TypeError):
        ql.steer(torch.zeros((M, N), dtype=torch.bfloat16), torch.zeros(N), 1.0, torch.zeros(1))
    with pytest.raises(ValueError):
        ql.steer(torch.zeros((M, N)), torch.zeros(N - 1), 1.0, torch.zeros(1))


def test_attention_rejects():
    B, T, H = 2, 8, 2
    qkv = torch.zeros((B * T, 3 * H * 64), dtype=torch.bfloat16)
    q, k, v = qkv[:, :128], qkv[:, 128:256], qkv[:, 256:]
    with pytest.raises(TypeError):  # fp16 O would receive fp32 rows
        ql.attention(q, k, v, B, T, H, O=torch.zeros((B * T, H * 64), dtype=torch.float16))
    with pytest.raises(ValueError):  # O rows
        ql.attention(q, k, v, B, T, H, O=torch.zeros((B * T - 1, H * 64)))
    with pytest.raises(ValueError):  # O too narrow
        ql.attention(q, k, v, B, T, H, O=torch.zeros((B * T, H * 64 - 4)))
    with pytest.raises(ValueError):  # q rows
        ql.attention(q[:-1], k, v, B, T, H)
    with pytest.raises(ValueError):  # q too narrow for H heads
        ql.attention(q[:, :64], k, v, B, T, H)
    with pytest.raises(TypeError):  # fp32 q
        ql.attention(q.float(), k, v, B, T, H)
    with pytest.raises(ValueError):  # column stride
        ql.attention(qkv[:, ::3], k, v, B, T, H)
    with pytest.raises(ValueError):  # host tensors
        ql.attention(q, k, v, B, T, H)


def test_groups_keep_their_tensors(monkeypatch):
    """A group array holds only device addresses; it must also keep the
    tensors alive, or a tensor dropped by the caller could have its memory
    handed back to the driver (torch empties its cache when a graph capture
    begins) while the group still points at it.  Host tensors stand in for
    device ones here: the device check is switched off and nothing is
    launched."""
    import gc
    import weakref
    monkeypatch.setattr(ql, "_on_device", lambda *a: None)
    codes, scales = weights()
    X, Y = x_bf16(), torch.zeros((M, N), dtype=torch.float32)
    bias, strength, d = torch.zeros(N), torch.zeros(1), torch.zeros(N)
    refs = [weakref.ref(t) for t in (codes, scales, X, Y, bias, strength, d)]
    g = ql.make_group([(ql.FMT_INT8, X, codes, scales, N, Y)])
    ge = ql.make_group_ep([(ql.FMT_INT8, X, codes, scales, N, Y, bias, ql.ACT_NONE, None,
                            (d, 3.0, strength))])
    del codes, scales, X, Y, bias, strength, d
    gc.collect()
    assert all(r() is not None for r in refs)
    del g, ge
    gc.collect()
    assert all(r() is None for r in refs)
