"""Float64 model of where the bf16 language-model step rounds (test
infrastructure).

The language model of the benchmarks (the decoder of Sec. 4.1 around the
BCMT layer; oracle/model_oracle.py is its exact form) keeps its residual
stream and activations in bf16 on the GPU.  This module repeats the oracle's
forward and backward in float64, rounding to bf16 where the GPU step stores
a value in bf16, and runs the mixing layer through bf16_model (the layer's
own rounding points).  Rounded here, in the order of the step:
  forward   the embedded input, each LayerNorm output, the sum of the
            residual and the mixing layer's output, U = LN2(x) W1 and
            GELU(U), the residual after the MLP;
  backward  the gradient of the logits, (softmax - onehot) / (B T); the
            residual-stream gradient after every LayerNorm backward; the
            gradient of U (taking GELU's derivative at the stored U); the
            gradient of LN2's output; the mixing layer's input gradient.
The loss and the head's log-sum-exp are float32 on the GPU and exact here.
"""

import numpy as np

import bf16_model as bm
from oracle import model_oracle as mo


def forward(tokens, targets, P, L, h, gamma, rnd):
    B, T = tokens.shape
    r = lambda x: rnd("lm", x)
    x = r(P["E"][tokens] + P["Pe"][:T][None])
    caches = []
    for lp in P["layers"]:
        a, c1 = mo.layer_norm(x, lp["ln1_g"], lp["ln1_b"])
        a = r(a)
        y, cmix = bm.forward(a, lp["mix"], L, h, gamma, rnd)
        xm = r(x + y)
        bn, c2 = mo.layer_norm(xm, lp["ln2_g"], lp["ln2_b"])
        bn = r(bn)
        u = r(bn @ lp["W1"])
        m = r(mo.gelu(u))
        x = r(xm + m @ lp["W2"])
        caches.append((c1, cmix, c2, bn, u, m))
    f, cf = mo.layer_norm(x, P["lnf_g"], P["lnf_b"])
    f = r(f)
    logits = f @ P["E"].T
    loss, dlogits = mo.cross_entropy(logits, targets)
    return loss, dict(tokens=tokens, P=P, caches=caches, cf=cf, f=f, dlogits=r(dlogits))


def backward(cache, rnd):
    P, tokens = cache["P"], cache["tokens"]
    B, T = tokens.shape
    r = lambda x: rnd("lm", x)
    dlogits = cache["dlogits"]
    G = {"E": dlogits.reshape(-1, dlogits.shape[-1]).T @ cache["f"].reshape(-1, P["E"].shape[1])}
    df = dlogits @ P["E"]
    dx, G["lnf_g"], G["lnf_b"] = mo.layer_norm_backward(df, cache["cf"])
    dx = r(dx)
    G["layers"] = [None] * len(P["layers"])
    for i in reversed(range(len(P["layers"]))):
        lp = P["layers"][i]
        c1, cmix, c2, bn, u, m = cache["caches"][i]
        g = {}
        g["W2"] = m.reshape(-1, m.shape[-1]).T @ dx.reshape(-1, dx.shape[-1])
        du = r((dx @ lp["W2"].T) * mo.gelu_grad(u))
        g["W1"] = bn.reshape(-1, bn.shape[-1]).T @ du.reshape(-1, du.shape[-1])
        dbn = r(du @ lp["W1"].T)
        dxm, g["ln2_g"], g["ln2_b"] = mo.layer_norm_backward(dbn, c2)
        dx = r(dx + dxm)
        gm = bm.backward(cmix, dx, rnd)
        g["mix"] = {k: gm["d" + k] for k in ("Wq", "Wk", "Wv", "Wo", "Wm", "Wg", "wp")}
        da, g["ln1_g"], g["ln1_b"] = mo.layer_norm_backward(gm["dX"], c1)
        dx = r(dx + da)
        G["layers"][i] = g
    np.add.at(G["E"], tokens.reshape(-1), dx.reshape(-1, dx.shape[-1]))
    G["Pe"] = np.zeros_like(P["Pe"])
    G["Pe"][:T] = dx.sum(axis=0)
    return G
