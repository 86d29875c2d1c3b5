"""Parity of the language-model entry points (bcmt_model_*) with the oracle.

The GPU model keeps activations in bf16 (the residual stream included) with
float32 accumulation; the oracle runs in float64 on the same bf16-valued
weights and float32 LayerNorm parameters.  Bounds: the loss to 2e-3
absolute (about 5e-4 of log V), every gradient array to 2e-2 of its largest
element (the layer's bf16 bound; for the benchmarked model, the arrays listed
in tolerances.LM have bounds derived from the rounding model), and the AdamW
update, which is float32 arithmetic on the same inputs, to 1e-6.
"""

import numpy as np
import pytest

import tolerances as tl
from test_gpu_parity import say, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

LOSS_TOL = 2e-3
GRAD_TOL = 2e-2


def oracle_params(arrs, n_layer):
    from paper_2608_13578_amd.inputs import MODEL_LAYER_ARRAYS
    f = [np.asarray(a, dtype=np.float64) for a in arrs]
    P = {"E": f[0], "Pe": f[1], "lnf_g": f[-2], "lnf_b": f[-1], "layers": []}
    for l in range(n_layer):
        a = dict(zip(MODEL_LAYER_ARRAYS, f[2 + 13 * l: 2 + 13 * (l + 1)]))
        P["layers"].append({"ln1_g": a["ln1_g"], "ln1_b": a["ln1_b"], "ln2_g": a["ln2_g"],
                            "ln2_b": a["ln2_b"], "W1": a["W1"], "W2": a["W2"],
                            "mix": {k: a[k] for k in ("Wq", "Wk", "Wv", "Wo", "Wm", "Wg", "wp")}})
    return P


def run(torch, V, d, H, nl, B, T, L, gamma, seed=0, opt=None):
    from paper_2608_13578_amd.inputs import make_model_inputs
    from paper_2608_13578_amd.model import ModelBuffers
    arrs, tok, tgt = make_model_inputs(V, d, T, nl, B, seed=seed)
    mb = ModelBuffers(V, d, H, nl, B, T, L, gamma)
    mb.set_params(arrs)
    tk = torch.from_numpy(tok).cuda()
    tg = torch.from_numpy(tgt).cuda()
    mb.step(tk, tg, opt)
    torch.cuda.synchronize()
    return mb, arrs, tok, tgt, tk, tg


CASES = [
    # name, V, d, H, n_layer, B, T, L
    ("bcmt-L32", 97, 64, 4, 2, 2, 96, 32),
    ("dense", 97, 64, 4, 2, 2, 96, 96),
    ("bcmt-dh32-ragged", 300, 128, 4, 1, 2, 100, 48),
    # the paper's vocabulary: rows of 50304 padded logits, 7 register steps
    # per thread in the loss kernel, 47 masked padding columns
    ("bcmt-vocab50257", 50257, 64, 2, 1, 1, 40, 16),
    # the benchmarked model (d = 128, 6 layers of 8 heads of 16, L = 128,
    # the GPT-2 vocabulary) on one sequence of 1024 tokens
    ("bcmt-bench-shape", 50257, 128, 8, 6, 1, 1024, 128),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_model_parity(torch_cuda, case):
    from oracle import model_oracle as mo
    name, V, d, H, nl, B, T, L = case
    gamma = 0.8
    say(f"model {name}: V={V} d={d} H={H} layers={nl} B={B} T={T} L={L}")
    mb, arrs, tok, tgt, _, _ = run(torch_cuda, V, d, H, nl, B, T, L, gamma)
    loss_ref, cache = mo.forward(tok.astype(np.int64), tgt.astype(np.int64),
                                 oracle_params(arrs, nl), L, H, gamma)
    G = mo.flatten(mo.backward(cache))
    loss = float(mb.loss.item())
    bounds = tl.LM["bounds"] if name == tl.LM["case"] else {}
    if bounds:
        s = tl.LM
        assert (V, d, H, nl, B, T, L) == (s["V"], s["d"], s["H"], s["layers"], s["B"], s["T"],
                                          s["L"])
    worst = []
    for nm, g, r in zip(mb.names, mb.arrays(mb.grads), G):
        g, r = np.asarray(g).reshape(-1), np.asarray(r).reshape(-1)
        err = float(np.abs(g - r).max() / max(np.abs(r).max(), 1e-30))
        worst.append((err / bounds.get(nm, GRAD_TOL), err, nm))
    worst.sort(reverse=True)
    say(f"[{name}] loss {loss:.6f} vs {loss_ref:.6f}; worst grads "
        + " ".join(f"{n}={e:.2e}" for _, e, n in worst[:4]))
    assert abs(loss - loss_ref) <= LOSS_TOL
    assert worst[0][0] <= 1.0, worst[:3]


def test_model_adamw_update(torch_cuda):
    """One step with AdamW: params = adamw(initial, the step's gradients);
    the bf16 copy holds the rounded update."""
    torch = torch_cuda
    from oracle import model_oracle as mo
    opt = {"lr": 1e-3, "beta1": 0.9, "beta2": 0.95, "eps": 1e-8, "weight_decay": 0.1}
    mb, arrs, *_ = run(torch, 97, 64, 4, 1, 2, 64, 32, 0.8, opt=opt)
    p0 = np.zeros(mb.n)
    for a, (off, cnt) in zip(arrs, mb.layout):
        p0[off:off + np.asarray(a).size] = np.asarray(a, dtype=np.float64).reshape(-1)
    g = mb.grads.double().cpu().numpy()
    m, v = np.zeros(mb.n), np.zeros(mb.n)
    mo.adamw_step(p0, g, m, v, 1, opt["lr"], opt["beta1"], opt["beta2"], opt["eps"],
                  opt["weight_decay"])
    got = mb.params.double().cpu().numpy()
    assert np.abs(got - p0).max() <= 1e-6 * max(1.0, np.abs(p0).max())
    assert np.array_equal(mb.params_bf16.float().cpu().numpy(),
                          mb.params.bfloat16().float().cpu().numpy())


def test_model_trains(torch_cuda):
    """Twenty AdamW steps on one fixed batch drive its loss well down, and
    the loss of a repeated step without an update is identical."""
    torch = torch_cuda
    opt = {"lr": 3e-3, "weight_decay": 0.0}
    mb, arrs, tok, tgt, tk, tg = run(torch, 97, 64, 4, 2, 2, 96, 32, 0.8, opt=opt)
    first = float(mb.loss.item())
    for _ in range(19):
        mb.step(tk, tg, opt)
    mb.step(tk, tg, None)
    torch.cuda.synchronize()
    a = float(mb.loss.item())
    mb.step(tk, tg, None)
    torch.cuda.synchronize()
    b = float(mb.loss.item())
    say(f"loss {first:.4f} -> {a:.4f}")
    assert a < 0.5 * first
    assert a == b
