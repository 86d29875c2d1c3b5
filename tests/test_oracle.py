"""Pins of the float64 oracle against what the paper and mathematics fix.

None of these tests re-types the oracle's own formulas: each compares it with
a library routine, a hand-derived value, a closed form, an invariant of the
method, or finite differences.
"""

import os

import numpy as np
import pytest
import torch

from oracle import bcmt_oracle as orc
from paper_2608_13578_amd.inputs import make_layer_inputs, make_upstream_grad, to_f64

from conftest import maxabs_rel

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _layer(B, T, D, seed=0, x_std=1.0, w_std=0.02):
    X, [W] = make_layer_inputs(B, T, D, seed=seed, x_std=x_std, w_std=w_std)
    return X.astype(np.float64), to_f64(W)


def _sdpa(Q, K, V, h, mask=None, is_causal=False):
    """torch's scaled_dot_product_attention in float64 on [B, T, D] inputs."""
    B, T, D = Q.shape
    dh = D // h

    def heads(x):
        return torch.from_numpy(x).reshape(B, T, h, dh).transpose(1, 2)

    out = torch.nn.functional.scaled_dot_product_attention(
        heads(Q), heads(K), heads(V), attn_mask=mask, is_causal=is_causal)
    return out.transpose(1, 2).reshape(B, T, D).numpy()


def _read_golden(name):
    sections = {}
    cur = None
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("["):
                cur = line.strip("[]")
                sections[cur] = []
                continue
            sections[cur].append([float(v) for v in line.split()])
    return sections


# ---------------------------------------------------------------- P1 / P2

def test_single_block_is_dense_causal_attention():
    """L >= T: one block, so the local stage is dense causal MHA (Sec. 3.2-3.3)
    and the shifted memory is zero, hence Y == H exactly (Sec. 3.5)."""
    X, P = _layer(2, 48, 64)
    Y, c = orc.forward(X, P, L=64, h=4, gamma=0.8)
    ref = _sdpa(c["Q"], c["K"], c["V"], 4, is_causal=True)
    assert maxabs_rel(c["Hcat"], ref) < 1e-12
    assert np.array_equal(Y, c["Hloc"])


@pytest.mark.parametrize("T,L", [(64, 16), (70, 16), (40, 64), (33, 1)])
def test_block_attention_is_block_diagonal_causal(T, L):
    """Attention confined to blocks equals library attention under a
    block-diagonal causal mask, and dense causal attention run on each block
    separately (Sec. 3.3, 3.6), including a partial last block."""
    X, P = _layer(2, T, 32)
    Y, c = orc.forward(X, P, L=L, h=2, gamma=0.8)
    t = np.arange(T)
    mask = (t[None, :] <= t[:, None]) & (t[None, :] // L == t[:, None] // L)
    ref = _sdpa(c["Q"], c["K"], c["V"], 2, mask=torch.from_numpy(mask))
    assert maxabs_rel(c["Hcat"], ref) < 1e-12
    for s, e in orc.block_ranges(T, L):
        part = _sdpa(c["Q"][:, s:e].copy(), c["K"][:, s:e].copy(),
                     c["V"][:, s:e].copy(), 2, is_causal=True)
        assert maxabs_rel(c["Hcat"][:, s:e], part) < 1e-12


def test_block_count_and_ranges():
    """N_b = ceil(T / L); all blocks have L tokens except possibly the last."""
    assert orc.n_blocks(1024, 128) == 8
    assert orc.n_blocks(1000, 128) == 8
    assert orc.n_blocks(1, 128) == 1
    r = orc.block_ranges(1000, 128)
    assert r[0] == (0, 128) and r[-1] == (896, 1000)
    assert sum(e - s for s, e in r) == 1000


# ---------------------------------------------------------------- P3

def test_pooling_uniform_when_wp_zero():
    """W_p = 0 gives equal scores, so each summary is the block mean (Sec. 3.4)."""
    X, P = _layer(2, 40, 32)
    P["wp"] = np.zeros_like(P["wp"])
    _, c = orc.forward(X, P, L=16, h=2, gamma=0.8)
    for i, (s, e) in enumerate(orc.block_ranges(40, 16)):
        assert np.allclose(c["S"][:, i], c["Hloc"][:, s:e].mean(axis=1), rtol=0, atol=1e-15)
    assert np.allclose(c["a"].reshape(2, -1).sum(axis=1), [3.0, 3.0])


def test_pooling_selects_argmax_for_large_wp():
    """A large W_p makes the block softmax one-hot on the top-scoring token."""
    X, P = _layer(1, 32, 16)
    _, c0 = orc.forward(X, P, L=16, h=2, gamma=0.8)
    H = c0["Hloc"]
    P2 = dict(P)
    P2["wp"] = P["wp"] * 1e6
    _, c = orc.forward(X, P2, L=16, h=2, gamma=0.8)
    for i, (s, e) in enumerate(orc.block_ranges(32, 16)):
        top = s + int(np.argmax(H[0, s:e] @ P2["wp"]))
        assert np.allclose(c["S"][0, i], H[0, top], atol=1e-12)
        assert abs(c["a"][0, s:e].sum() - 1.0) < 1e-14


# ---------------------------------------------------------------- P4

def test_memory_normaliser_golden():
    """Row sums of the decay weights equal (1 - 0.8^i)/(1 - 0.8) (Sec. 3.5)."""
    g = _read_golden("memory_gamma0.8.txt")
    _, _, z = orc.memory_weights(6, 0.8)
    for i, zi in g["normaliser"]:
        assert abs(z[int(i) - 1] - zi) < 1e-14


def test_memory_impulse_golden():
    """Hand-derived memory of the impulse summaries (1, 0, 0, 0)."""
    g = _read_golden("memory_gamma0.8.txt")
    S = np.array([[1.0], [0.0], [0.0], [0.0]])
    M = orc.exp_memory(S, 0.8)
    for i, num, den in g["impulse"]:
        assert abs(M[int(i) - 1, 0] - num / den) < 1e-15


def test_memory_matches_recurrence():
    """The literal double sum equals the decayed recurrence
    N_i = g N_{i-1} + S_i, Z_i = g Z_{i-1} + 1, M_i = N_i / Z_i."""
    rng = np.random.default_rng(5)
    S = rng.standard_normal((3, 37, 8))
    for gamma in (0.0, 0.3, 0.8, 0.95):
        M = orc.exp_memory(S, gamma)
        N = np.zeros((3, 8))
        Z = 0.0
        for i in range(37):
            N = gamma * N + S[:, i]
            Z = gamma * Z + 1.0
            assert np.allclose(M[:, i], N / Z, rtol=1e-13, atol=1e-14)


def test_memory_special_cases():
    """gamma = 0 gives M = S; constant summaries give that constant (convex
    combination); gamma = 1 (the limit) gives the cumulative mean."""
    rng = np.random.default_rng(6)
    S = rng.standard_normal((2, 11, 5))
    assert np.array_equal(orc.exp_memory(S, 0.0), S)
    c = np.broadcast_to(rng.standard_normal((2, 1, 5)), (2, 11, 5))
    assert np.allclose(orc.exp_memory(c, 0.8), c, rtol=1e-14, atol=1e-15)
    cum = np.cumsum(S, axis=1) / np.arange(1, 12)[None, :, None]
    assert np.allclose(orc.exp_memory(S, 1.0), cum, rtol=1e-13, atol=1e-14)
    # close to the limit: within O((1 - gamma) * N_b) of the cumulative mean
    assert np.abs(orc.exp_memory(S, 0.999) - cum).max() < 0.05


# ---------------------------------------------------------------- P5 / P6 / P7

@pytest.mark.parametrize("t", [0, 15, 16, 40, 63])
def test_causality_bit_identical(t):
    """Changing tokens after t leaves outputs up to t bit-identical (Sec. 3.6)."""
    X, P = _layer(2, 64, 32)
    Y, _ = orc.forward(X, P, L=16, h=2, gamma=0.8)
    X2 = X.copy()
    X2[:, t + 1:] += np.random.default_rng(7).standard_normal(X2[:, t + 1:].shape)
    Y2, _ = orc.forward(X2, P, L=16, h=2, gamma=0.8)
    assert np.array_equal(Y[:, :t + 1], Y2[:, :t + 1])
    if t < 63:
        assert not np.array_equal(Y[:, t + 1:], Y2[:, t + 1:])


def test_causality_nan_poison_across_block_boundary():
    """NaN in every token after a block boundary cannot reach earlier blocks."""
    X, P = _layer(1, 64, 32)
    Y, _ = orc.forward(X, P, L=16, h=2, gamma=0.8)
    X2 = X.copy()
    X2[:, 32:] = np.nan
    with np.errstate(invalid="ignore"):
        Y2, _ = orc.forward(X2, P, L=16, h=2, gamma=0.8)
    assert np.array_equal(Y[:, :32], Y2[:, :32])


def test_first_block_has_no_memory():
    """M_causal of block 1 is zero, so Y == H there (Sec. 3.5)."""
    X, P = _layer(2, 64, 32)
    Y, c = orc.forward(X, P, L=16, h=2, gamma=0.8)
    assert np.array_equal(Y[:, :16], c["Hloc"][:, :16])
    assert not np.allclose(Y[:, 16:], c["Hloc"][:, 16:])


def test_last_block_only_changes_last_block():
    """The last block's summary never reaches any output (shift by one)."""
    X, P = _layer(2, 64, 32)
    Y, _ = orc.forward(X, P, L=16, h=2, gamma=0.8)
    X2 = X.copy()
    X2[:, 48:] *= 1.7
    Y2, _ = orc.forward(X2, P, L=16, h=2, gamma=0.8)
    assert np.array_equal(Y[:, :48], Y2[:, :48])


def test_honly_when_wm_zero():
    """W_m = 0 removes the memory path: Y == H, the HOnly variant (Sec. 4.5)."""
    X, P = _layer(2, 64, 32)
    P["Wm"] = np.zeros_like(P["Wm"])
    Y, c = orc.forward(X, P, L=16, h=2, gamma=0.8)
    assert np.array_equal(Y, c["Hloc"])


def test_zero_gate_weights_give_half_gate():
    """W_g = 0 gives sigmoid(0) = 1/2 exactly, so Y = H + M_tokens / 2."""
    X, P = _layer(2, 64, 32)
    P["Wg"] = np.zeros_like(P["Wg"])
    Y, c = orc.forward(X, P, L=16, h=2, gamma=0.8)
    blk = np.arange(64) // 16
    assert np.all(c["G"] == 0.5)
    assert np.array_equal(Y, c["Hloc"] + 0.5 * c["Mcausal"][:, blk])


def test_sigmoid_matches_library():
    """The gate's sigmoid (Sec. 3.8) equals scipy's expit, including far into
    saturation where a naive 1/(1+exp(-u)) overflows."""
    from scipy.special import expit
    u = np.concatenate([np.linspace(-50, 50, 1001), [-800.0, -745.0, 745.0, 800.0]])
    assert np.allclose(orc.sigmoid(u), expit(u), rtol=1e-15, atol=1e-300)
    assert orc.sigmoid(np.array([-800.0]))[0] < 1e-300
    assert orc.sigmoid(np.array([800.0]))[0] == 1.0


# ---------------------------------------------------------------- P8

FD_SHAPE = dict(B=2, T=64, D=32, h=2, L=16)


def _loss_and_grads(X, layers, dY, gamma, residual, stack):
    if stack:
        Y, caches = orc.stack_forward(X, layers, FD_SHAPE["L"], FD_SHAPE["h"], gamma, residual)
        dX, grads = orc.stack_backward(caches, dY)
        return float((Y * dY).sum()), dX, grads
    Y, cache = orc.forward(X, layers[0], FD_SHAPE["L"], FD_SHAPE["h"], gamma, residual)
    g = orc.backward(cache, dY)
    return float((Y * dY).sum()), g["dX"], [g]


def _loss(X, layers, dY, gamma, residual, stack):
    """The layer output Y; the loss sum(dY * Y) is formed from differences of
    outputs so that the large residual term cancels elementwise first."""
    if stack:
        Y, _ = orc.stack_forward(X, layers, FD_SHAPE["L"], FD_SHAPE["h"], gamma, residual)
    else:
        Y, _ = orc.forward(X, layers[0], FD_SHAPE["L"], FD_SHAPE["h"], gamma, residual)
    return Y


@pytest.mark.parametrize("w_std,n_layers,residual", [
    (0.02, 1, False), (0.3, 1, False), (0.02, 1, True), (0.3, 1, True),
    # deep stacks with 0.3-std weights blow activations up to ~1e11, where a
    # finite-difference step can no longer resolve the derivative
    (0.02, 12, True), (0.06, 12, True)])
def test_gradients_finite_differences(w_std, n_layers, residual):
    """Directional central differences of sum(dY * Y) against the analytic
    gradients, for X, every weight of every layer, and the decay."""
    B, T, D = FD_SHAPE["B"], FD_SHAPE["T"], FD_SHAPE["D"]
    X, layers = make_layer_inputs(B, T, D, seed=0, x_std=1.0, w_std=w_std, n_layers=n_layers)
    X = X.astype(np.float64)
    layers = [to_f64(w) for w in layers]
    dY = make_upstream_grad(B, T, D, seed=1).astype(np.float64)
    gamma = 0.8
    stack = n_layers > 1
    _, dX, grads = _loss_and_grads(X, layers, dY, gamma, residual, stack)
    rng = np.random.default_rng(11)

    def check(analytic_dir, f_plus_minus, scale, bound):
        # fourth-order central stencil with a step of 1e-3 of the tensor's
        # scale; the error is normalised by |grad| |v| (the Cauchy-Schwarz
        # bound of the directional derivative), since a random direction can
        # make the directional derivative itself arbitrarily small
        eps = 1e-3 * scale
        f = f_plus_minus
        diff = 8 * (f(eps) - f(-eps)) - (f(2 * eps) - f(-2 * eps))
        fd = float((diff * dY).sum()) / (12 * eps)
        err = abs(fd - analytic_dir) / max(bound, 1e-300)
        assert err < 1e-6, (fd, analytic_dir, err)

    v = rng.standard_normal(X.shape)
    check(float((dX * v).sum()),
          lambda e: _loss(X + e * v, layers, dY, gamma, residual, stack),
          np.abs(X).max() / np.abs(v).max(), np.linalg.norm(dX) * np.linalg.norm(v))
    for li in ([0, n_layers - 1] if stack else [0]):
        for name in orc.PARAM_NAMES:
            v = rng.standard_normal(layers[li][name].shape)
            gname = "d" + name
            ana = float((grads[li][gname] * v).sum())

            def f(e, name=name, v=v, li=li):
                ls = [dict(w) for w in layers]
                ls[li][name] = layers[li][name] + e * v
                return _loss(X, ls, dY, gamma, residual, stack)

            check(ana, f, np.abs(layers[li][name]).max() / np.abs(v).max(),
                  np.linalg.norm(grads[li][gname]) * np.linalg.norm(v))
    # decay: one shared value feeds every layer, so its derivative is the sum
    ana = sum(g["dgamma"] for g in grads)
    check(ana, lambda e: _loss(X, layers, dY, gamma + e, residual, stack), 0.1, abs(ana))


def test_gradients_coordinates():
    """Single-coordinate central differences on sampled entries."""
    B, T, D = FD_SHAPE["B"], FD_SHAPE["T"], FD_SHAPE["D"]
    X, [W] = make_layer_inputs(B, T, D, seed=3, x_std=1.0, w_std=0.3)
    X = X.astype(np.float64)
    W = to_f64(W)
    dY = make_upstream_grad(B, T, D, seed=1).astype(np.float64)
    Y, cache = orc.forward(X, W, FD_SHAPE["L"], FD_SHAPE["h"], 0.8, False)
    g = orc.backward(cache, dY)
    rng = np.random.default_rng(12)
    tensors = dict(X=X, **W)
    for name, arr in tensors.items():
        grad = g["d" + name]
        gmax = np.abs(grad).max()
        for _ in range(12):
            idx = tuple(int(rng.integers(0, s)) for s in arr.shape)
            eps = 1e-4 * max(1.0, abs(arr[idx]))

            def L_at(delta):
                t2 = {k: v.copy() for k, v in tensors.items()}
                t2[name][idx] += delta
                Xp = t2.pop("X")
                Yp, _ = orc.forward(Xp, t2, FD_SHAPE["L"], FD_SHAPE["h"], 0.8, False)
                return float((Yp * dY).sum())

            fd = (8 * (L_at(eps) - L_at(-eps)) - (L_at(2 * eps) - L_at(-2 * eps))) / (12 * eps)
            assert abs(fd - grad[idx]) <= 1e-6 * gmax, (name, idx, fd, grad[idx])


def test_decay_gradient_forward_mode():
    """dgamma equals the forward-mode derivative of the recurrence:
    N'_i = g N'_{i-1} + N_{i-1}, Z'_i = g Z'_{i-1} + Z_{i-1},
    dgamma = sum_i dM_i . (N'_i - M_i Z'_i) / Z_i."""
    X, P = _layer(2, 96, 32, w_std=0.3)
    dY = make_upstream_grad(2, 96, 32, seed=1).astype(np.float64)
    for gamma in (0.0, 0.5, 0.8):
        Y, c = orc.forward(X, P, L=16, h=2, gamma=gamma)
        g = orc.backward(c, dY)
        # recover dM from the same chain: dM = shift(dMcausal) @ Wm^T
        blk = np.arange(96) // 16
        dMtok = dY * c["G"]
        nb = 6
        dMc = np.stack([dMtok[:, i * 16:(i + 1) * 16].sum(axis=1) for i in range(nb)], axis=1)
        dMp = np.zeros_like(dMc)
        dMp[:, :-1] = dMc[:, 1:]
        dM = dMp @ P["Wm"].T
        S = c["S"]
        N = np.zeros_like(S[:, 0])
        Np = np.zeros_like(N)
        Z = 0.0
        Zp = 0.0
        total = 0.0
        for i in range(nb):
            Np, Zp = gamma * Np + N, gamma * Zp + Z
            N, Z = gamma * N + S[:, i], gamma * Z + 1.0
            M = N / Z
            total += float((dM[:, i] * (Np - M * Zp)).sum() / Z)
        assert abs(total - g["dgamma"]) <= 1e-12 * max(1.0, abs(total))
        del blk


def test_single_block_zero_memory_gradients():
    """With one block the memory path is inactive: the gate, memory, pooling
    and decay gradients vanish exactly."""
    X, P = _layer(2, 32, 32, w_std=0.3)
    dY = make_upstream_grad(2, 32, 32, seed=1).astype(np.float64)
    Y, c = orc.forward(X, P, L=32, h=2, gamma=0.8)
    g = orc.backward(c, dY)
    for k in ("dWg", "dWm", "dwp"):
        assert np.all(g[k] == 0.0)
    assert g["dgamma"] == 0.0
