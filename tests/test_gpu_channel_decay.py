"""Parity of the per-channel decay (BCMT_FLAG_CHANNEL_DECAY) with the oracle.

Channel d of the memory runs the recurrence of Sec. 3.5 with its own decay;
the backward returns one decay gradient per channel.  Cases cover both
memory paths (up to 32 blocks per sequence: the single-kernel scan; more:
the parallel scans), chunked execution with a per-channel state, and
decoding.  Bounds: 2e-2 (bf16) and 1e-4 (float32), max|gpu - ref| / max|ref|
per tensor, the per-channel decay gradient included.
"""

import numpy as np
import pytest

from test_gpu_parity import GRADS, compare, inputs, say, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu


def decays(D, seed=4, lo=0.3, hi=0.95):
    return np.random.default_rng(seed).uniform(lo, hi, D).astype(np.float32)


def run_gpu(torch, B, T, D, H, L, dtype, X, W, dY, gamma, residual=False):
    from paper_2608_13578_amd.layer import LayerBuffers, to_device, to_host64
    lb = LayerBuffers(B, T, D, H, L, gamma=gamma, dtype=dtype, residual=residual)
    lb.set_params(W)
    Xd, dYd = to_device(X, dtype), to_device(dY, dtype)
    Yd, dXd = lb.new_activation(), lb.new_activation()
    g = lb.new_grads()
    lb.forward(Xd, Yd)
    lb.backward(Xd, dYd, dXd, g)
    torch.cuda.synchronize()
    out = {"Y": to_host64(Yd), "dX": to_host64(dXd)}
    for k in GRADS:
        out[k] = to_host64(g[k])
    if "dgamma_ch" in g:
        out["dgamma_ch"] = to_host64(g["dgamma_ch"])
    out["dgamma"] = float(g["dgamma"][0].item())
    return out


def run_oracle(L, H, X, W, dY, gamma, residual=False):
    from oracle import bcmt_oracle as orc
    from paper_2608_13578_amd.inputs import to_f64
    Y, c = orc.forward(X.astype(np.float64), to_f64(W), L, H, np.asarray(gamma, np.float64),
                       residual)
    g = orc.backward(c, dY.astype(np.float64))
    out = {"Y": Y, "dX": g["dX"], "dgamma_ch": g["dgamma"]}
    for k in GRADS:
        out[k] = g[k]
    return out


CASES = [
    # name, B, T, D, H, L, dtype, w_std, residual
    ("f32-fused", 2, 256, 128, 2, 32, "f32", 0.05, False),
    ("bf16-fused", 2, 1024, 256, 4, 128, "bf16", 0.02, False),
    ("f32-long-scans", 2, 1200, 128, 2, 16, "f32", 0.05, True),
    ("bf16-long-scans", 2, 2560, 256, 4, 32, "bf16", 0.02, False),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_channel_decay_parity(torch_cuda, case):
    name, B, T, D, H, L, dtype, ws, res = case
    say(f"channel decay {name}: B={B} T={T} D={D} H={H} L={L} {dtype}")
    X, W, dY = inputs(B, T, D, dtype, w_std=ws)
    g = decays(D)
    gpu = run_gpu(torch_cuda, B, T, D, H, L, dtype, X, W, dY, g, res)
    ref = run_oracle(L, H, X, W, dY, g, res)
    compare({k: gpu[k] for k in ref}, ref, dtype, name)


@pytest.mark.parametrize("dtype,T,L", [("bf16", 1024, 128), ("f32", 1200, 16)])
def test_equal_channels_are_the_single_decay(torch_cuda, dtype, T, L):
    """Every channel at 0.8 gives the scalar-decay layer.  The scalar decay
    scans the projected summaries (S W_m); a per-channel decay scans S and
    then projects the memory (W_m mixes channels, so only one decay lets the
    two orders agree), so the two agree to rounding, on the single-kernel
    path (8 blocks) and on the parallel scans (75 blocks).  The per-channel
    decay gradients add up to the scalar one."""
    B, D, H = 2, 128, 2
    X, W, dY = inputs(B, T, D, dtype, w_std=0.05)
    a = run_gpu(torch_cuda, B, T, D, H, L, dtype, X, W, dY, 0.8)
    b = run_gpu(torch_cuda, B, T, D, H, L, dtype, X, W, dY, np.full(D, 0.8, np.float32))
    keys = ("Y", "dX") + tuple(k for k in GRADS if k != "dgamma")
    compare({k: b[k] for k in keys}, {k: a[k] for k in keys}, dtype, "equal-channels")
    tol = 1e-4 if dtype == "f32" else 2e-2
    assert abs(b["dgamma_ch"].sum() - a["dgamma"]) <= tol * abs(a["dgamma"])


def test_channel_decay_chunks(torch_cuda):
    """Chained chunks with a per-channel state (Z as [B, D]) against the
    oracle's chunks: outputs, states, gradients and state gradients."""
    from test_gpu_chunks import compare_chunks, gpu_chunks, oracle_chunks
    torch = torch_cuda
    B, D, H, L = 2, 128, 2, 16
    cuts = [0, 320, 800, 1024]  # 20 and 30 blocks (single kernel), then 14
    X, W, dY = inputs(B, cuts[-1], D, "f32", w_std=0.05)
    g = decays(D)
    gpu = gpu_chunks(torch, B, cuts, D, H, L, "f32", X, W, dY, g)
    ref = oracle_chunks(B, cuts, D, H, L, X, W, dY, np.asarray(g, np.float64))
    ref["dgamma_ch"] = ref.pop("dgamma")  # one value per channel
    gpu.pop("dgamma")
    compare_chunks(gpu, ref, "f32", "channel-decay-chunks")


def test_channel_decay_decode(torch_cuda):
    """Decoding with a per-channel decay equals the whole-sequence layer."""
    from test_gpu_decode import gpu_decode
    B, T, D, H, L = 2, 160, 256, 4, 32
    X, W, _ = inputs(B, T, D, "bf16")
    g = decays(D)
    gpu = gpu_decode(torch_cuda, B, T, D, H, L, "bf16", X, W, g, False, prefill=64)
    from oracle import bcmt_oracle as orc
    from paper_2608_13578_amd.inputs import to_f64
    ref, _ = orc.forward(X.astype(np.float64), to_f64(W), L, H, np.asarray(g, np.float64))
    compare({"Y": gpu}, {"Y": ref}, "bf16", "channel-decay-decode")


def test_multi_scale_memory(torch_cuda):
    """A multi-scale memory: four groups of channels, each with its own
    decay (0.5, 0.8, 0.95, 0.99) and so its own memory over its channels,
    as one per-channel decay vector; against the oracle."""
    B, T, D, H, L = 2, 1024, 256, 4, 64
    X, W, dY = inputs(B, T, D, "bf16", w_std=0.02)
    g = np.repeat(np.array([0.5, 0.8, 0.95, 0.99], np.float32), D // 4)
    gpu = run_gpu(torch_cuda, B, T, D, H, L, "bf16", X, W, dY, g)
    ref = run_oracle(L, H, X, W, dY, g)
    compare({k: gpu[k] for k in ref}, ref, "bf16", "multi-scale")
