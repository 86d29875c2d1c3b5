"""Parity of incremental decoding with the oracle's whole-sequence layer.

The decoder produces the output of one token per sequence per call; the
layer is causal, so token t's output must equal row t of the layer applied to
the whole sequence.  Each case decodes every token of seeded inputs (from an
empty state, or after a chunked prefill of whole blocks that hands its memory
state to the decoder) and compares the stacked outputs with the float64
oracle's Y, max|gpu - ref| / max|ref| <= 2e-2 (bf16) or 1e-4 (float32).
"""

import numpy as np
import pytest

from test_gpu_parity import compare, inputs, say, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu


def oracle_y(B, T, D, H, L, X, W, gamma, residual):
    from oracle import bcmt_oracle as orc
    from paper_2608_13578_amd.inputs import to_f64
    Y, _ = orc.forward(X.astype(np.float64), to_f64(W), L, H, gamma, residual)
    return Y


def gpu_decode(torch, B, T, D, H, L, dtype, X, W, gamma, residual, prefill=0):
    """Decodes tokens prefill..T-1; the first `prefill` tokens (whole blocks)
    go through the chunked forward, whose outgoing state starts the decoder.
    Returns the outputs of all T tokens."""
    from paper_2608_13578_amd.layer import DecodeBuffers, LayerBuffers, to_device, to_host64
    Xd = to_device(X, dtype)
    ys = []
    carry = None
    if prefill:
        assert prefill % L == 0
        lb = LayerBuffers(B, prefill, D, H, L, gamma=gamma, dtype=dtype, residual=residual)
        lb.set_params(W)
        Yp = lb.new_activation()
        carry = lb.new_carry()
        lb.forward_chunk(Xd[:, :prefill].contiguous(), Yp, None, carry)
        ys.append(to_host64(Yp))
    db = DecodeBuffers(B, D, H, L, gamma=gamma, dtype=dtype, residual=residual)
    db.set_params(W)
    db.reset(carry)
    out = torch.empty((B, T - prefill, D), dtype=Xd.dtype, device="cuda")
    y = torch.empty((B, D), dtype=Xd.dtype, device="cuda")
    for t in range(prefill, T):
        x = Xd[:, t].contiguous()
        db.step(t - prefill, x, y)
        out[:, t - prefill] = y
    torch.cuda.synchronize()
    ys.append(to_host64(out))
    return np.concatenate(ys, axis=1)


CASES = [
    # name, B, T, D, H, L, dtype, w_std, gamma, residual, prefill
    ("bf16-L32", 2, 100, 256, 4, 32, "bf16", 0.02, 0.8, False, 0),
    ("f32-L16-residual", 3, 70, 128, 2, 16, "f32", 0.05, 0.9, True, 0),
    ("bf16-stress", 2, 96, 128, 2, 32, "bf16", 2 / np.sqrt(128), 0.8, False, 0),
    ("f32-gamma0-L8", 1, 50, 192, 3, 8, "f32", 0.05, 0.0, False, 0),
    # 10 sequences: two groups of eight in the matrix-vector products
    ("bf16-B10", 10, 40, 256, 4, 16, "bf16", 0.02, 0.8, False, 0),
    ("f32-B10-stress", 10, 48, 128, 2, 16, "f32", 2 / np.sqrt(128), 0.8, True, 0),
    # decoding after a prefill of whole blocks
    ("bf16-prefill", 2, 200, 256, 4, 32, "bf16", 0.02, 0.8, False, 96),
    ("f32-prefill", 2, 90, 128, 2, 16, "f32", 0.05, 0.8, True, 48),
    # every token completes a block (one-token blocks), and two-token
    # blocks after a prefill of five
    ("f32-L1", 2, 20, 128, 2, 1, "f32", 0.05, 0.8, False, 0),
    ("bf16-L2-prefill", 2, 30, 128, 2, 2, "bf16", 0.02, 0.8, False, 10),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_decode_matches_layer(torch_cuda, case):
    name, B, T, D, H, L, dtype, ws, gamma, res, pre = case
    say(f"decode {name}: B={B} T={T} D={D} H={H} L={L} {dtype} prefill={pre}")
    X, W, _ = inputs(B, T, D, dtype, w_std=ws)
    gpu = gpu_decode(torch_cuda, B, T, D, H, L, dtype, X, W, gamma, res, prefill=pre)
    ref = oracle_y(B, T, D, H, L, X, W, gamma, res)
    compare({"Y": gpu}, {"Y": ref}, dtype, f"decode-{name}")


def test_decode_measured_shape(torch_cuda):
    """B=8, D=768, H=12, L=128 (the measured layer's shape), 288 tokens: two
    whole blocks and part of a third, from an empty state."""
    B, T, D, H, L = 8, 288, 768, 12, 128
    X, W, _ = inputs(B, T, D, "bf16")
    gpu = gpu_decode(torch_cuda, B, T, D, H, L, "bf16", X, W, 0.8, False)
    ref = oracle_y(B, T, D, H, L, X, W, 0.8, False)
    compare({"Y": gpu}, {"Y": ref}, "bf16", "decode-B8-D768-L128")


def test_decode_long_context_shape(torch_cuda):
    """B=2, D=1024, H=16, L=256: a 512-token prefill through the chunked
    forward, then 300 decoded tokens across a block boundary."""
    B, T, D, H, L = 2, 812, 1024, 16, 256
    X, W, _ = inputs(B, T, D, "bf16")
    gpu = gpu_decode(torch_cuda, B, T, D, H, L, "bf16", X, W, 0.8, False, prefill=512)
    ref = oracle_y(B, T, D, H, L, X, W, 0.8, False)
    compare({"Y": gpu}, {"Y": ref}, "bf16", "decode-B2-D1024-L256")
    compare({"Y": gpu[:, 512:]}, {"Y": ref[:, 512:]}, "bf16", "decode-B2-D1024-L256-decoded")


def test_decode_repeats_exactly(torch_cuda):
    """Two decoders over the same tokens give identical outputs (the
    products' K partials are added in a fixed order)."""
    B, T, D, H, L = 4, 40, 256, 4, 16
    X, W, _ = inputs(B, T, D, "bf16")
    a = gpu_decode(torch_cuda, B, T, D, H, L, "bf16", X, W, 0.8, False)
    b = gpu_decode(torch_cuda, B, T, D, H, L, "bf16", X, W, 0.8, False)
    assert np.array_equal(a, b)
