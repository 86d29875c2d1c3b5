"""Float64 CPU oracle of a language model built from BCMT layers.

TEST INFRASTRUCTURE ONLY, under the same rules as bcmt_oracle: only the test
suite, the smoke check and the CPU-baseline leg of the benchmark may import
it, and it imports nothing from the product package.

The paper evaluates BCMT inside a decoder-only language model (Sec. 4.1:
d_model = 128, 6 layers, 8 heads, batch 16; the Dense baseline has the same
architecture) but does not spell out the parts around the token-mixing
layer.  The readings used here (all listed in the design notes):
  * token embedding E [V, d] plus a learned absolute position embedding
    Pe [T, d] (the usual decoder of the period; the paper names none);
  * pre-LN blocks: x <- x + mix(LN1(x)); x <- x + MLP(LN2(x)), where mix is
    the BCMT layer of Sec. 3 (for the Dense model: the same layer with one
    block, L >= T, i.e. plain causal attention, Sec. 4.1);
  * MLP: x W1 -> GELU (tanh form) -> W2, hidden width 4d, no biases (the
    BCMT layer has none either);
  * LayerNorm with gain and bias, eps = 1e-5, over the feature axis;
  * final LayerNorm, then logits = f E^T (head tied to the embedding);
  * loss = mean over all B T positions of -log softmax(logits)[target];
  * the memory decay is a fixed hyperparameter (not trained);
  * AdamW (decoupled decay, bias-corrected moments), applied to every
    parameter, with the hyperparameters passed in.

Every function below writes out its definition directly; the backward is
the chain rule taken by hand, pinned by finite differences in the tests.
"""

import numpy as np

from oracle import bcmt_oracle as layer

LN_EPS = 1e-5
GELU_C = np.sqrt(2.0 / np.pi)
GELU_A = 0.044715


def gelu(u):
    """GELU, tanh form: 0.5 u (1 + tanh(c (u + a u^3)))."""
    return 0.5 * u * (1.0 + np.tanh(GELU_C * (u + GELU_A * u ** 3)))


def gelu_grad(u):
    """d gelu / du of the tanh form."""
    t = np.tanh(GELU_C * (u + GELU_A * u ** 3))
    return 0.5 * (1.0 + t) + 0.5 * u * (1.0 - t * t) * GELU_C * (1.0 + 3.0 * GELU_A * u * u)


def layer_norm(x, g, b):
    """LayerNorm over the last axis; returns (y, cache)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + LN_EPS)
    xh = (x - mu) * rstd
    return xh * g + b, (xh, rstd, g)


def layer_norm_backward(dy, cache):
    """Gradients (dx, dg, db) of sum(dy * y), summed over all leading axes."""
    xh, rstd, g = cache
    dxh = dy * g
    dx = rstd * (dxh - dxh.mean(axis=-1, keepdims=True)
                 - xh * (dxh * xh).mean(axis=-1, keepdims=True))
    lead = tuple(range(dy.ndim - 1))
    return dx, (dy * xh).sum(axis=lead), dy.sum(axis=lead)


def cross_entropy(logits, targets):
    """Mean of -log softmax(logits)[target]; returns (loss, dlogits)."""
    m = logits.max(axis=-1, keepdims=True)
    e = np.exp(logits - m)
    z = e.sum(axis=-1, keepdims=True)
    lse = (m + np.log(z))[..., 0]
    picked = np.take_along_axis(logits, targets[..., None], axis=-1)[..., 0]
    n = targets.size
    loss = float((lse - picked).sum() / n)
    d = e / z
    np.put_along_axis(d, targets[..., None],
                      np.take_along_axis(d, targets[..., None], axis=-1) - 1.0, axis=-1)
    return loss, d / n


def init_params(V, d, T, n_layer, seed=0, w_std=0.02):
    """A seeded float64 parameter set (normal weights, unit LN gains)."""
    rng = np.random.default_rng(seed)
    P = {"E": rng.standard_normal((V, d)) * w_std,
         "Pe": rng.standard_normal((T, d)) * w_std,
         "lnf_g": np.ones(d), "lnf_b": np.zeros(d), "layers": []}
    for _ in range(n_layer):
        lp = {"ln1_g": np.ones(d), "ln1_b": np.zeros(d),
              "ln2_g": np.ones(d), "ln2_b": np.zeros(d),
              "W1": rng.standard_normal((d, 4 * d)) * w_std,
              "W2": rng.standard_normal((4 * d, d)) * w_std,
              "mix": {k: rng.standard_normal((d, d)) * w_std
                      for k in ("Wq", "Wk", "Wv", "Wo", "Wm", "Wg")}}
        lp["mix"]["wp"] = rng.standard_normal(d) * w_std
        P["layers"].append(lp)
    return P


def forward(tokens, targets, P, L, h, gamma):
    """Loss of the model on tokens [B, T] with next-token targets [B, T]."""
    B, T = tokens.shape
    x = P["E"][tokens] + P["Pe"][:T][None]
    caches = []
    for lp in P["layers"]:
        a, c1 = layer_norm(x, lp["ln1_g"], lp["ln1_b"])
        y, cmix = layer.forward(a, lp["mix"], L, h, gamma)
        x = x + y
        bn, c2 = layer_norm(x, lp["ln2_g"], lp["ln2_b"])
        u = bn @ lp["W1"]
        m = gelu(u)
        x = x + m @ lp["W2"]
        caches.append((c1, cmix, c2, bn, u, m))
    f, cf = layer_norm(x, P["lnf_g"], P["lnf_b"])
    logits = f @ P["E"].T
    loss, dlogits = cross_entropy(logits, targets)
    return loss, dict(tokens=tokens, P=P, caches=caches, cf=cf, f=f, dlogits=dlogits)


def backward(cache):
    """Gradients of the loss for every parameter (same structure as P)."""
    P, tokens = cache["P"], cache["tokens"]
    B, T = tokens.shape
    dlogits = cache["dlogits"]
    G = {"E": dlogits.reshape(-1, dlogits.shape[-1]).T @ cache["f"].reshape(-1, P["E"].shape[1])}
    df = dlogits @ P["E"]
    dx, G["lnf_g"], G["lnf_b"] = layer_norm_backward(df, cache["cf"])
    G["layers"] = [None] * len(P["layers"])
    for i in reversed(range(len(P["layers"]))):
        lp = P["layers"][i]
        c1, cmix, c2, bn, u, m = cache["caches"][i]
        g = {}
        # x_out = x_mid + gelu(LN2(x_mid) W1) W2
        g["W2"] = m.reshape(-1, m.shape[-1]).T @ dx.reshape(-1, dx.shape[-1])
        du = (dx @ lp["W2"].T) * gelu_grad(u)
        g["W1"] = bn.reshape(-1, bn.shape[-1]).T @ du.reshape(-1, du.shape[-1])
        dbn = du @ lp["W1"].T
        dxm, g["ln2_g"], g["ln2_b"] = layer_norm_backward(dbn, c2)
        dx = dx + dxm
        # x_mid = x_in + mix(LN1(x_in))
        gm = layer.backward(cmix, dx)
        g["mix"] = {k: gm["d" + k] for k in ("Wq", "Wk", "Wv", "Wo", "Wm", "Wg", "wp")}
        da, g["ln1_g"], g["ln1_b"] = layer_norm_backward(gm["dX"], c1)
        dx = dx + da
        G["layers"][i] = g
    # embedding lookups (the tied head's part is already in G["E"])
    np.add.at(G["E"], tokens.reshape(-1), dx.reshape(-1, dx.shape[-1]))
    G["Pe"] = np.zeros_like(P["Pe"])
    G["Pe"][:T] = dx.sum(axis=0)
    return G


def adamw_step(p, g, m, v, t, lr, beta1, beta2, eps, wd):
    """One AdamW update of arrays p, m, v (in place) at step t >= 1:
    p *= 1 - lr wd; m = b1 m + (1 - b1) g; v = b2 v + (1 - b2) g^2;
    p -= lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps)."""
    p *= 1.0 - lr * wd
    m *= beta1
    m += (1.0 - beta1) * g
    v *= beta2
    v += (1.0 - beta2) * g * g
    mh = m / (1.0 - beta1 ** t)
    vh = v / (1.0 - beta2 ** t)
    p -= lr * mh / (np.sqrt(vh) + eps)


def flatten(tree):
    """The parameter (or gradient) arrays in a fixed order, as a list."""
    out = [tree["E"], tree["Pe"]]
    for lp in tree["layers"]:
        out += [lp["ln1_g"], lp["ln1_b"]]
        out += [lp["mix"][k] for k in ("Wq", "Wk", "Wv", "Wo", "Wm", "Wg", "wp")]
        out += [lp["ln2_g"], lp["ln2_b"], lp["W1"], lp["W2"]]
    out += [tree["lnf_g"], tree["lnf_b"]]
    return out
