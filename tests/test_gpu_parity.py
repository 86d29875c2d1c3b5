"""Parity of the HIP layer (through the C ABI) with the float64 oracle.

Each case draws seeded inputs, runs forward + backward on cuda:0, runs the
oracle on the same (bf16-rounded where applicable) values, and compares every
output tensor with max|gpu - ref| / max|ref|: at most 2e-2 for bf16 and 1e-4
for float32, except for the bf16 cases listed in tolerances.py, whose bounds
per tensor are derived from the float64 rounding model (bf16_model.py).
"""

import os
import sys

import numpy as np
import pytest

import tolerances as tl
from conftest import maxabs_rel

pytestmark = pytest.mark.gpu

GRADS = ("dWq", "dWk", "dWv", "dWo", "dWm", "dWg", "dwp")


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "no GPU visible"
    from paper_2608_13578_amd import bcmt as abi
    if not os.path.exists(abi.LIB_PATH):
        from paper_2608_13578_amd.build import build
        build()
    abi.lib()
    return torch


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def run_gpu(torch, B, T, D, H, L, dtype, X, W, dY=None, gamma=0.8, residual=False):
    from paper_2608_13578_amd.layer import LayerBuffers, to_device, to_host64
    lb = LayerBuffers(B, T, D, H, L, gamma=gamma, dtype=dtype, residual=residual)
    lb.set_params(W)
    Xd = to_device(X, dtype)
    Yd = lb.new_activation()
    lb.forward(Xd, Yd)
    out = {}
    if dY is not None:
        dYd = to_device(dY, dtype)
        dXd = lb.new_activation()
        g = lb.new_grads()
        lb.backward(Xd, dYd, dXd, g)
        torch.cuda.synchronize()
        out["dX"] = to_host64(dXd)
        for k in GRADS:
            out[k] = to_host64(g[k])
        out["dgamma"] = float(g["dgamma"][0].item())
    torch.cuda.synchronize()
    out["Y"] = to_host64(Yd)
    return out


def run_oracle(B, T, D, H, L, X, W, dY=None, gamma=0.8, residual=False):
    from oracle import bcmt_oracle as orc
    from paper_2608_13578_amd.inputs import to_f64
    Y, cache = orc.forward(X.astype(np.float64), to_f64(W), L, H, gamma, residual)
    out = {"Y": Y}
    if dY is not None:
        out.update(orc.backward(cache, dY.astype(np.float64)))
    return out


def inputs(B, T, D, dtype, seed=0, x_std=1.0, w_std=0.02):
    from paper_2608_13578_amd.inputs import make_layer_inputs, make_upstream_grad
    bf = dtype == "bf16"
    X, [W] = make_layer_inputs(B, T, D, seed=seed, x_std=x_std, w_std=w_std, bf16=bf)
    dY = make_upstream_grad(B, T, D, seed=seed + 1, bf16=bf)
    return X, W, dY


def compare(gpu, ref, dtype, label):
    """Every output within its bound (tolerances.bound of the case)."""
    errs = {}
    for k, v in ref.items():
        if k == "dgamma":
            errs[k] = abs(gpu[k] - v) / max(abs(v), 1e-30)
        else:
            errs[k] = maxabs_rel(gpu[k], v)
    say(f"[{label}] " + " ".join(f"{k}={e:.2e}" for k, e in errs.items()))
    bad = {k: (e, tl.bound(label, k, dtype)) for k, e in errs.items()
           if not (e <= tl.bound(label, k, dtype))}
    assert not bad, f"{label}: above the bound (error, bound): {bad}"


CASES = [
    # name, B, T, D, H, L, dtype, x_std, w_std, gamma, residual
    ("c1-f32", 1, 256, 128, 2, 64, "f32", 0.02, 0.02, 0.8, False),
    ("c1-f32-stress", 1, 256, 128, 2, 64, "f32", 1.0, 2 / np.sqrt(128), 0.8, False),
    ("c1-bf16", 1, 256, 128, 2, 64, "bf16", 1.0, 0.02, 0.8, False),
    ("bf16-stress", 2, 256, 128, 2, 64, "bf16", 1.0, 2 / np.sqrt(128), 0.8, False),
    ("f32-ragged-L48", 2, 200, 128, 2, 48, "f32", 1.0, 0.05, 0.8, False),
    ("f32-single-block", 2, 192, 128, 2, 256, "f32", 1.0, 0.05, 0.8, False),
    ("f32-L32-gamma0", 2, 160, 192, 3, 32, "f32", 1.0, 0.05, 0.0, False),
    ("f32-residual-L20", 1, 130, 192, 3, 20, "f32", 1.0, 0.05, 0.9, True),
    ("bf16-ragged-T1000", 1, 1000, 256, 4, 128, "bf16", 1.0, 2 / np.sqrt(256), 0.8, False),
    ("bf16-L1024-dense", 1, 1024, 256, 4, 1024, "bf16", 1.0, 0.02, 0.8, False),
    ("bf16-L256", 2, 1024, 256, 4, 256, "bf16", 1.0, 0.02, 0.8, True),
    # 512 blocks per sequence: the W_m products and the look-back scans
    # across workgroups (32 segments of 16 blocks per sequence)
    ("f32-many-blocks-L8", 2, 4096, 128, 2, 8, "f32", 1.0, 0.05, 0.8, False),
    # the look-back scans with a ragged last segment (126 blocks: 7 segments
    # of 16 and one of 14) and a ragged last block (3 tokens)
    ("f32-look-back-ragged", 1, 1003, 128, 2, 8, "f32", 1.0, 0.05, 0.8, False),
    # 160 blocks per sequence (the look-back scans and the W_m products),
    # ragged, at the paper's decay and at 0.9 (there the decay gradient is a
    # small sum of large terms of both signs: its bound comes from the
    # rounding model).
    ("bf16-many-blocks-L16", 2, 2550, 256, 4, 16, "bf16", 1.0, 0.02, 0.8, False),
    ("bf16-many-blocks-L16-g0.9", 2, 2550, 256, 4, 16, "bf16", 1.0, 0.02, 0.9, False),
    # heads of 16 and 32 dimensions (the paper's model uses 16): ragged
    # blocks, a stress distribution, one long block staged in many chunks
    ("f32-dh16-ragged-L48", 2, 200, 128, 8, 48, "f32", 1.0, 0.05, 0.8, False),
    ("f32-dh32-stress-residual", 1, 256, 128, 4, 64, "f32", 1.0, 2 / np.sqrt(128), 0.8, True),
    ("f32-dh16-one-block-T300", 1, 300, 64, 4, 512, "f32", 1.0, 0.05, 0.8, False),
    ("bf16-dh16-L128", 2, 512, 128, 8, 128, "bf16", 1.0, 0.02, 0.8, False),
    ("bf16-dh32-L1000", 1, 1000, 128, 4, 1000, "bf16", 1.0, 0.02, 0.8, False),
    # the bf16 matrix-core kernels' three launch shapes (blocks of at most
    # 32, at most 64, and longer), each with ragged blocks
    ("bf16-dh16-ragged-L20", 2, 150, 128, 8, 20, "bf16", 1.0, 0.02, 0.8, False),
    ("bf16-dh32-ragged-L48", 2, 200, 128, 4, 48, "bf16", 1.0, 0.02, 0.8, True),
    ("bf16-dh16-stress-L200", 1, 450, 64, 4, 200, "bf16", 1.0, 2 / np.sqrt(64), 0.8, False),
    # degenerate blocks: every token a block of its own (attention returns
    # V and pooling returns H, so the exact dW_q, dW_k and dw_p are zero and
    # the metric takes the absolute error; the memory is a decayed average
    # of earlier tokens), blocks of two tokens with a one-token last block,
    # and sequences of one token
    ("f32-L1", 1, 40, 128, 2, 1, "f32", 1.0, 0.05, 0.8, False),
    ("bf16-L2-ragged", 2, 67, 128, 2, 2, "bf16", 1.0, 0.02, 0.8, False),
    ("f32-T1", 2, 1, 128, 2, 64, "f32", 1.0, 0.05, 0.8, False),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_parity_small(torch_cuda, case):
    name, B, T, D, H, L, dtype, xs, ws, gamma, res = case
    say(f"case {name}: B={B} T={T} D={D} H={H} L={L} {dtype}")
    X, W, dY = inputs(B, T, D, dtype, x_std=xs, w_std=ws)
    gpu = run_gpu(torch_cuda, B, T, D, H, L, dtype, X, W, dY, gamma=gamma, residual=res)
    ref = run_oracle(B, T, D, H, L, X, W, dY, gamma=gamma, residual=res)
    if name in tl.DERIVED:  # the rounding model's case is this one
        assert tl.DERIVED[name][:5] == (B, T, D, H, L)
        assert np.isclose(tl.DERIVED[name][5], ws) and tl.DERIVED[name][6:8] == (gamma, res)
    compare(gpu, ref, dtype, name)


@pytest.mark.parametrize("gamma", [0.7, 0.8, 0.9])
def test_parity_gpt2_small_shape(torch_cuda, gamma):
    """The GPT-2-small-shaped layer at the paper's maximum context:
    B=8, T=1024, L=128, D=768, H=12, bf16, activations N(0,1), weights
    N(0, 0.02^2); at the paper's decay 0.8 and at the ends of the range of
    its sensitivity remark (Sec. 3.5)."""
    B, T, D, H, L = 8, 1024, 768, 12, 128
    say(f"case c2: B=8 T=1024 D=768 H=12 L=128 bf16 gamma={gamma}")
    X, W, dY = inputs(B, T, D, "bf16")
    gpu = run_gpu(torch_cuda, B, T, D, H, L, "bf16", X, W, dY, gamma=gamma)
    ref = run_oracle(B, T, D, H, L, X, W, dY, gamma=gamma)
    compare(gpu, ref, "bf16", f"c2-gamma{gamma}")


def test_forward_is_deterministic_and_causal(torch_cuda):
    """Forward has no atomics: two runs are bit-identical.  Changing tokens
    after t leaves outputs up to t bit-identical (Sec. 3.6)."""
    torch = torch_cuda
    from paper_2608_13578_amd.layer import LayerBuffers, to_device
    B, T, D, H, L = 2, 256, 128, 2, 64
    say("case causality: B=2 T=256 D=128 L=64 bf16")
    X, W, _ = inputs(B, T, D, "bf16")
    lb = LayerBuffers(B, T, D, H, L, dtype="bf16")
    lb.set_params(W)
    Xd = to_device(X, "bf16")
    Y1 = lb.new_activation()
    Y2 = lb.new_activation()
    lb.forward(Xd, Y1)
    lb.forward(Xd, Y2)
    torch.cuda.synchronize()
    assert torch.equal(Y1, Y2)
    for t in (0, 63, 64, 100, 200):
        X2 = Xd.clone()
        X2[:, t + 1:] = torch.randn_like(X2[:, t + 1:].float()).to(X2.dtype)
        Y3 = lb.new_activation()
        lb.forward(X2, Y3)
        torch.cuda.synchronize()
        assert torch.equal(Y1[:, :t + 1], Y3[:, :t + 1]), t
        assert not torch.equal(Y1[:, t + 1:], Y3[:, t + 1:]), t


def test_forward_is_deterministic_on_the_look_back_scans(torch_cuda):
    """Two sequences of 160 blocks take the look-back scans, whose
    workgroups wait for one another's published aggregates: the forward is
    still bit-identical from run to run."""
    torch = torch_cuda
    from paper_2608_13578_amd.layer import LayerBuffers, to_device
    B, T, D, H, L = 2, 2560, 256, 4, 16
    say(f"case look-back forward determinism: B={B} T={T} D={D} L={L} bf16")
    X, W, _ = inputs(B, T, D, "bf16")
    lb = LayerBuffers(B, T, D, H, L, dtype="bf16")
    lb.set_params(W)
    Xd = to_device(X, "bf16")
    Ys = []
    for _ in range(3):
        Y = lb.new_activation()
        lb.forward(Xd, Y)
        torch.cuda.synchronize()
        Ys.append(Y)
    for Y in Ys[1:]:
        assert torch.equal(Ys[0], Y)


@pytest.mark.parametrize("T,L,per_channel", [(1024, 128, False), (2560, 16, False),
                                              (2560, 16, True)],
                         ids=["fused-memory", "long-scan", "long-scan-per-channel"])
def test_backward_is_deterministic(torch_cuda, T, L, per_channel):
    """Every gradient, the decay gradient included, is reduced in a fixed
    order (per-workgroup partials, no atomics): repeated backward passes
    give the same bits, on the single-kernel memory path (8 blocks), the
    look-back scans across workgroups (160 blocks of two sequences, one
    decay: every segment folds the aggregates before it in a fixed order)
    and the per-channel scans."""
    torch = torch_cuda
    from paper_2608_13578_amd.layer import LayerBuffers, to_device
    B, D, H = 2, 256, 4
    say(f"case backward determinism: B={B} T={T} D={D} L={L} per_channel={per_channel}")
    X, W, dY = inputs(B, T, D, "bf16")
    gamma = np.linspace(0.7, 0.9, D) if per_channel else 0.8
    lb = LayerBuffers(B, T, D, H, L, gamma=gamma, dtype="bf16")
    lb.set_params(W)
    Xd, dYd = to_device(X, "bf16"), to_device(dY, "bf16")
    Yd, dXd = lb.new_activation(), lb.new_activation()
    lb.forward(Xd, Yd)
    runs = []
    for _ in range(3):
        g = lb.new_grads()
        lb.backward(Xd, dYd, dXd, g)
        torch.cuda.synchronize()
        runs.append({k: v.clone() for k, v in g.items()})
    dg = "dgamma_ch" if per_channel else "dgamma"
    assert float(runs[0][dg].abs().max()) > 0.0
    for r in runs[1:]:
        for k in runs[0]:
            assert torch.equal(runs[0][k], r[k]), k


def test_accumulate_flag(torch_cuda):
    """BCMT_FLAG_ACCUM_WGRAD adds into the gradient buffers."""
    torch = torch_cuda
    from paper_2608_13578_amd.layer import LayerBuffers, to_device
    B, T, D, H, L = 1, 256, 128, 2, 64
    say("case accumulate: B=1 T=256 D=128 L=64 f32")
    X, W, dY = inputs(B, T, D, "f32", w_std=0.05)
    lb = LayerBuffers(B, T, D, H, L, dtype="f32")
    lb.set_params(W)
    Xd, dYd = to_device(X, "f32"), to_device(dY, "f32")
    Yd = lb.new_activation()
    lb.forward(Xd, Yd)
    g1 = lb.new_grads()
    lb.backward(Xd, dYd, None, g1)
    acc = LayerBuffers(B, T, D, H, L, dtype="f32", accumulate=True)
    acc.params = lb.params
    acc.saved = lb.saved
    g2 = lb.new_grads()
    acc.backward(Xd, dYd, None, g2)
    acc.backward(Xd, dYd, None, g2)
    torch.cuda.synchronize()
    for k in GRADS + ("dgamma",):
        a, b = g1[k], g2[k]
        assert torch.allclose(2 * a, b, rtol=1e-5, atol=1e-6 * float(a.abs().max()) + 1e-30), k
