"""Pins of the language-model oracle (oracle/model_oracle.py).

Each part is checked against something other than its own formula: exact
identities of GELU, LayerNorm invariants, the uniform-logit cross-entropy,
AdamW's closed form at step 1, and central finite differences of the whole
model's loss in every parameter group.
"""

import numpy as np
import pytest

from oracle import model_oracle as mo


def test_gelu_identities():
    """The tanh form satisfies gelu(u) - gelu(-u) = u exactly, gelu(0) = 0,
    gelu(u) -> u and gelu(-u) -> 0 for large u, and its derivative matches
    central differences."""
    u = np.linspace(-6, 6, 97)
    assert np.allclose(mo.gelu(u) - mo.gelu(-u), u, rtol=0, atol=1e-14)
    assert mo.gelu(np.array(0.0)) == 0.0
    assert abs(mo.gelu(np.array(12.0)) - 12.0) < 1e-12 and abs(mo.gelu(np.array(-12.0))) < 1e-12
    h = 1e-5
    fd = (mo.gelu(u + h) - mo.gelu(u - h)) / (2 * h)
    assert np.allclose(mo.gelu_grad(u), fd, rtol=0, atol=1e-9)


def test_layer_norm_invariants_and_gradient():
    """Unit gain, zero bias: every row has mean 0 and mean square
    var / (var + eps); a shift or positive scale of a row does not change
    the output; the backward matches central differences."""
    rng = np.random.default_rng(0)
    x = rng.standard_normal((3, 5, 16)) * 2 + 1
    g, b = np.ones(16), np.zeros(16)
    y, _ = mo.layer_norm(x, g, b)
    var = x.var(axis=-1)
    assert np.allclose(y.mean(axis=-1), 0, atol=1e-14)
    assert np.allclose((y ** 2).mean(axis=-1), var / (var + mo.LN_EPS), rtol=1e-12)
    y2, _ = mo.layer_norm(3.0 * x + 7.0, g, b)
    assert np.allclose(y2, mo.layer_norm(3.0 * x, g, b)[0], atol=1e-12)
    g, b = rng.standard_normal(16), rng.standard_normal(16)
    dy = rng.standard_normal(x.shape)
    _, c = mo.layer_norm(x, g, b)
    dx, dg, db = mo.layer_norm_backward(dy, c)
    f = lambda xx, gg, bb: float((mo.layer_norm(xx, gg, bb)[0] * dy).sum())
    for arr, grad in ((x, dx), (g, dg), (b, db)):
        v = rng.standard_normal(arr.shape)
        e = 1e-6
        args = [x, g, b]
        i = [id(x), id(g), id(b)].index(id(arr))
        ap, am = list(args), list(args)
        ap[i], am[i] = arr + e * v, arr - e * v
        fd = (f(*ap) - f(*am)) / (2 * e)
        assert abs(fd - (grad * v).sum()) < 1e-7 * max(1.0, abs(fd))


def test_cross_entropy_uniform_and_gradient():
    """Equal logits give log V whatever the targets; the gradient is
    (softmax - onehot) / N, checked by central differences."""
    rng = np.random.default_rng(1)
    V = 13
    t = rng.integers(0, V, (2, 7))
    loss, _ = mo.cross_entropy(np.full((2, 7, V), 0.3), t)
    assert abs(loss - np.log(V)) < 1e-14
    z = rng.standard_normal((2, 7, V)) * 3
    loss, d = mo.cross_entropy(z, t)
    v = rng.standard_normal(z.shape)
    e = 1e-6
    fd = (mo.cross_entropy(z + e * v, t)[0] - mo.cross_entropy(z - e * v, t)[0]) / (2 * e)
    assert abs(fd - (d * v).sum()) < 1e-8
    assert np.allclose(d.sum(axis=-1), 0, atol=1e-15)


def test_adamw_first_step_closed_form():
    """At step 1 the bias-corrected moments are g and g^2, so a parameter
    moves by -lr g / (|g| + eps) after the decoupled decay p (1 - lr wd);
    with g = 0 only the decay acts."""
    p = np.array([1.0, -2.0, 0.5, 3.0])
    g = np.array([0.1, -4.0, 0.0, 1e-3])
    m, v = np.zeros(4), np.zeros(4)
    lr, wd, eps = 1e-2, 0.1, 1e-8
    want = p * (1 - lr * wd) - lr * g / (np.abs(g) + eps)
    mo.adamw_step(p, g, m, v, 1, lr, 0.9, 0.999, eps, wd)
    assert np.allclose(p, want, rtol=1e-12, atol=0)


def _tiny(L, seed=0):
    V, d, T, B, h, nl = 11, 32, 20, 2, 2, 2
    P = mo.init_params(V, d, T, nl, seed=seed, w_std=0.3)
    rng = np.random.default_rng(seed + 5)
    for lp in P["layers"]:  # non-trivial LayerNorm parameters
        for k in ("ln1_g", "ln2_g"):
            lp[k] = 1 + 0.3 * rng.standard_normal(d)
        for k in ("ln1_b", "ln2_b"):
            lp[k] = 0.3 * rng.standard_normal(d)
    P["lnf_g"] = 1 + 0.3 * rng.standard_normal(d)
    P["lnf_b"] = 0.3 * rng.standard_normal(d)
    tok = rng.integers(0, V, (B, T))
    tgt = np.roll(tok, -1, axis=1)
    return P, tok, tgt, L, h


@pytest.mark.parametrize("L", [8, 32])
def test_model_gradients_finite_differences(L):
    """Central differences of the loss along a random direction in every
    parameter array (L = 8: memory across three blocks; L = 32 >= T: the
    Dense model)."""
    P, tok, tgt, L, h = _tiny(L)
    gamma = 0.7
    loss, c = mo.forward(tok, tgt, P, L, h, gamma)
    G = mo.backward(c)
    params, grads = mo.flatten(P), mo.flatten(G)
    rng = np.random.default_rng(9)
    for arr, grad in zip(params, grads):
        v = rng.standard_normal(arr.shape)
        e = 1e-5
        arr += e * v
        lp = mo.forward(tok, tgt, P, L, h, gamma)[0]
        arr -= 2 * e * v
        lm = mo.forward(tok, tgt, P, L, h, gamma)[0]
        arr += e * v
        fd = (lp - lm) / (2 * e)
        ana = float((grad * v).sum())
        assert abs(fd - ana) <= 1e-6 * max(1e-3, abs(ana)) + 1e-9, (arr.shape, fd, ana)


def test_untrained_loss_is_near_log_vocab():
    """With small weights the logits are nearly equal, so the loss is close
    to log V; an embedding row that appears only as a target gets gradient
    only through the tied head."""
    V, d, T = 50, 32, 16
    P = mo.init_params(V, d, T, 1, seed=3, w_std=1e-3)
    rng = np.random.default_rng(4)
    tok = rng.integers(0, V - 1, (2, T))  # token V-1 never appears as an input
    tgt = np.full((2, T), V - 1)
    loss, c = mo.forward(tok, tgt, P, 16, 2, 0.8)
    assert abs(loss - np.log(V)) < 1e-2
    G = mo.backward(c)
    head_only = c["dlogits"].reshape(-1, V).T @ c["f"].reshape(-1, d)
    assert np.allclose(G["E"][V - 1], head_only[V - 1], rtol=1e-12, atol=1e-15)
