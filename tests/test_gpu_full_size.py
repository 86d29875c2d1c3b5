"""Parity at the full sizes of the measured workloads, on sampled outputs.

Sequences are independent and the layer is causal (Sec. 3.6), so the
outputs of a token prefix of chosen sequences depend on that region of the
input alone.  The HIP path runs the full-size launch (the configuration the
benchmark times, or the larger long-context and block-size ones); the
upstream gradient is zero outside the sampled region; the float64 oracle runs
the region alone.  Then Y and dX agree on the region, dX is exactly zero
outside it, and every weight, w_p and decay gradient equals the region's.
Tolerances as in test_gpu_parity: max-abs-rel <= 2e-2 in bf16; the 12-layer
stack's w_p and decay gradients have bounds derived from the rounding model
(tolerances.STACK).
"""

import sys

import numpy as np
import pytest

import tolerances as tl
from conftest import maxabs_rel

pytestmark = pytest.mark.gpu

TOL_BF16 = tl.TOL_BF16
GRADS = ("dWq", "dWk", "dWv", "dWo", "dWm", "dWg", "dwp")


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "no GPU visible"
    from paper_2608_13578_amd import bcmt as abi
    abi.lib()
    return torch


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def sampled_case(torch, label, B, T, D, H, L, rows, P, n_layers=1, residual=False, gamma=0.8):
    from oracle import bcmt_oracle as orc
    from paper_2608_13578_amd.inputs import make_layer_inputs, make_upstream_grad, to_f64
    from paper_2608_13578_amd.layer import LayerBuffers, to_device, to_host64
    say(f"case {label}: B={B} T={T} D={D} H={H} L={L} layers={n_layers} "
        f"sampled sequences {rows}, tokens < {P}")
    X, Ws = make_layer_inputs(B, T, D, seed=0, x_std=1.0, w_std=0.02, bf16=True,
                              n_layers=n_layers)
    dY = make_upstream_grad(B, T, D, seed=1, bf16=True)
    keep = np.zeros((B, T, 1), dtype=np.float32)
    keep[rows, :P] = 1.0
    dY = dY * keep

    # full-size launch on the GPU: forward through the stack, then backward
    layers = []
    xs = [to_device(X, "bf16")]
    for W in Ws:
        lb = LayerBuffers(B, T, D, H, L, gamma=gamma, dtype="bf16", residual=residual)
        lb.set_params(W)
        y = lb.new_activation()
        lb.forward(xs[-1], y)
        layers.append(lb)
        xs.append(y)
    g = to_device(dY, "bf16")
    grads = [None] * n_layers
    for li in reversed(range(n_layers)):
        lb = layers[li]
        dx = lb.new_activation()
        gr = lb.new_grads()
        lb.backward(xs[li], g, dx, gr)
        grads[li] = gr
        g = dx
    torch.cuda.synchronize()
    Y = to_host64(xs[-1])
    dX = to_host64(g)
    say(f"[{label}] GPU pass done")

    # the oracle on the sampled region alone
    Xr = X[rows, :P].astype(np.float64)
    dYr = dY[rows, :P].astype(np.float64)
    Wr = [to_f64(W) for W in Ws]
    if n_layers == 1:
        Yr, cache = orc.forward(Xr, Wr[0], L, H, gamma, residual)
        gr_ref = [orc.backward(cache, dYr)]
        dXr = gr_ref[0]["dX"]
    else:
        Yr, caches = orc.stack_forward(Xr, Wr, L, H, gamma, residual)
        dXr, gr_ref = orc.stack_backward(caches, dYr)

    errs = {"Y": maxabs_rel(Y[rows, :P], Yr), "dX": maxabs_rel(dX[rows, :P], dXr)}
    outside = dX.copy()
    outside[rows, :P] = 0.0
    assert not np.any(outside), f"{label}: dX nonzero outside the sampled region"
    for li in range(n_layers):
        for k in GRADS:
            errs[f"{k}[{li}]"] = maxabs_rel(to_host64(grads[li][k]), gr_ref[li][k])
        dg = float(grads[li]["dgamma"][0].item())
        ref = gr_ref[li]["dgamma"]
        errs[f"dgamma[{li}]"] = abs(dg - ref) / max(abs(ref), 1e-30)
    worst = max(errs, key=errs.get)
    say(f"[{label}] worst {worst}={errs[worst]:.2e}; Y={errs['Y']:.2e} dX={errs['dX']:.2e}")
    def tol(k):
        if n_layers > 1:
            return tl.STACK["bounds"].get(k.split("[")[0], TOL_BF16)
        return tl.bound(label, k)
    bad = {k: e for k, e in errs.items() if not (e <= tol(k))}
    assert not bad, f"{label}: above tolerance: {bad}"


@pytest.mark.parametrize("L", [32, 64, 128, 256, 1024])
def test_block_size_sweep(torch_cuda, L):
    """B=16, T=1024, D=768, H=12, bf16; sequences 0 and 15 checked whole."""
    sampled_case(torch_cuda, f"sweep-L{L}", 16, 1024, 768, 12, L, rows=[0, 15], P=1024)


@pytest.mark.parametrize("L", [64, 128, 256, 512, 1024])
def test_paper_model_shape(torch_cuda, L):
    """The paper's model width: B=16, T=1024, D=128 with 8 heads of 16
    dimensions, bf16, the block sizes it sweeps and the dense limit L = T.
    All 16 sequences are checked whole: the decay gradient of a couple of
    sequences alone is a small, heavily cancelling sum (two sequences at
    L = 128 give a scalar the bf16 path misses by 5e-2, while the float32
    path matches it to 1e-6 and all 16 sequences give 8.6e-3).  The dense
    limit (no memory, dgamma = 0) checks sequences 0 and 15."""
    rows = [0, 15] if L >= 1024 else list(range(16))
    sampled_case(torch_cuda, f"paper-shape-L{L}", 16, 1024, 128, 8, L, rows=rows, P=1024)


def test_paper_model_shape_two_sequences(torch_cuda):
    """The paper's model width at L = 128 with two sequences checked (0 and
    15), the decay gradient included (its bound is derived from the rounding
    model: tolerances.SAMPLED)."""
    B, T, D, H, L, _, gamma, rows, _ = tl.SAMPLED["paper-shape-L128-two"]
    sampled_case(torch_cuda, "paper-shape-L128-two", B, T, D, H, L, rows=list(rows), P=1024,
                 gamma=gamma)


@pytest.mark.parametrize("T,rows,P", [(4096, [0], 4096), (16384, [0, 1], 1024),
                                      (65536, [0, 1], 1024)])
def test_long_context(torch_cuda, T, rows, P):
    """B=2, D=1024, H=16, L=256, bf16, T up to 65536 (256 blocks)."""
    sampled_case(torch_cuda, f"long-T{T}", 2, T, 1024, 16, 256, rows=rows, P=P)


def test_twelve_layer_stack(torch_cuda):
    """Forward + backward of 12 residual layers at B=8, T=1024, D=768, H=12,
    L=128, bf16; sequence 3 checked whole."""
    s = tl.STACK
    assert (s["B"], s["T"], s["D"], s["H"], s["L"], s["layers"]) == (8, 1024, 768, 12, 128, 12)
    sampled_case(torch_cuda, "stack-12", 8, 1024, 768, 12, 128, rows=list(s["rows"]), P=1024,
                 n_layers=12, residual=True)


@pytest.mark.timeout(900)
def test_long_context_tail(torch_cuda):
    """The long-context launch (B=2, T=65536, D=1024, H=16, L=256, bf16)
    checked at the END of a sequence: the upstream gradient is sequence 0's
    last 1024 tokens (blocks 252-255), so the memory carries information
    from all 252 earlier blocks into the compared outputs (Sec. 3.5).

    The float64 reference is the oracle run as chunks with its carried state:
    the blocks before token START only through their state (N, Z), the last
    TAIL tokens with a forward and backward pass.  Gradients reaching blocks
    before START through the memory are scaled by at most 0.8**48 (the
    decay over the 48 blocks between START and the first token with an
    upstream gradient), so the reference drops terms of relative size below
    1e-4; the GPU's own dX on those tokens is checked to be that small.

    The decay gradient here is a sum over four blocks that cancels heavily;
    its bound is derived as for the cases of tolerances.py, from the bf16
    rounding model run on the same tail with the same incoming state (the
    model without jitter and two jittered realisations), computed here."""
    torch = torch_cuda
    from oracle import bcmt_oracle as orc
    from paper_2608_13578_amd.inputs import make_layer_inputs, make_upstream_grad, to_f64
    from paper_2608_13578_amd.layer import LayerBuffers, to_device, to_host64
    B, T, D, H, L, gamma = 2, 65536, 1024, 16, 256, 0.8
    P0 = T - 1024                      # first token with an upstream gradient
    TAIL = 1024 + 48 * L               # tokens the reference runs in full
    START = T - TAIL
    CH = 8192                          # forward chunk of the state-only part
    say(f"case long-tail: B={B} T={T} D={D} H={H} L={L}; dY on sequence 0, tokens >= {P0}")
    X, [W] = make_layer_inputs(B, T, D, seed=0, x_std=1.0, w_std=0.02, bf16=True)
    dY = make_upstream_grad(B, T, D, seed=1, bf16=True)
    dY[1] = 0.0
    dY[0, :P0] = 0.0

    lb = LayerBuffers(B, T, D, H, L, gamma=gamma, dtype="bf16")
    lb.set_params(W)
    Xd = to_device(X, "bf16")
    Yd = lb.new_activation()
    lb.forward(Xd, Yd)
    dXd = lb.new_activation()
    g = lb.new_grads()
    lb.backward(Xd, to_device(dY, "bf16"), dXd, g)
    torch.cuda.synchronize()
    Yg = to_host64(Yd[0, P0:])
    dXg = to_host64(dXd[0])
    gg = {k: to_host64(g[k]) for k in GRADS}
    gg["dgamma"] = float(g["dgamma"][0].item())
    del Yd, dXd, Xd, lb, g
    say("[long-tail] GPU pass done")

    Wf = to_f64(W)
    x0 = X[:1].astype(np.float64)
    carry = (np.zeros((1, D)), np.zeros(1))
    for a in range(0, START, CH):
        b = min(a + CH, START)
        _, c = orc.forward(x0[:, a:b], Wf, L, H, gamma, carry=carry)
        carry = c["carry_out"]
        say(f"[long-tail] oracle state through token {b}")
    Yr, c = orc.forward(x0[:, START:], Wf, L, H, gamma, carry=carry)
    dYt = dY[:1, START:].astype(np.float64)
    ref = orc.backward(c, dYt)
    del c
    say("[long-tail] oracle tail done")
    import bf16_model as bm
    model_dg = 0.0
    for rnd in [bm.rounder()] + [bm.rounder(jitter=tl.JITTER, seed=k) for k in range(2)]:
        _, cm = bm.forward(x0[:, START:], Wf, L, H, gamma, rnd, carry=carry)
        dg = bm.backward(cm, dYt, rnd)["dgamma"]
        model_dg = max(model_dg, abs(dg - ref["dgamma"]) / abs(ref["dgamma"]))
        del cm
        say(f"[long-tail] rounding model: dgamma error {model_dg:.2e}")

    errs = {"Y": maxabs_rel(Yg, Yr[0, P0 - START:]),
            "dX": maxabs_rel(dXg[START:], ref["dX"][0])}
    for k in GRADS:
        errs[k] = maxabs_rel(gg[k], ref[k])
    errs["dgamma"] = abs(gg["dgamma"] - ref["dgamma"]) / abs(ref["dgamma"])
    before = float(np.abs(dXg[:START]).max() / np.abs(dXg).max())
    say("[long-tail] " + " ".join(f"{k}={e:.2e}" for k, e in errs.items())
        + f"; dX before the reference's tokens {before:.1e}")
    assert before <= 1e-4
    tol = {"dgamma": max(TOL_BF16, tl.MARGIN * model_dg)}
    bad = {k: e for k, e in errs.items() if not (e <= tol.get(k, TOL_BF16))}
    assert not bad, f"long-tail: above tolerance: {bad} (dgamma bound {tol['dgamma']:.2e})"
