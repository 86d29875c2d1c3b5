"""The bf16 rounding model and the parity bounds derived from it.

bf16_model.py repeats the layer in float64 and rounds to bf16 exactly where
the GPU path stores a value or feeds it to the matrix cores in bf16.  Pins:
with no rounding it is the oracle; each rounding point reaches the outputs
it should; and the derived bounds in tolerances.py follow from its jittered
ensembles.
"""

import numpy as np
import pytest

import bf16_model as bm
import tolerances as tl
from oracle import bcmt_oracle as orc
from paper_2608_13578_amd.inputs import make_layer_inputs, make_upstream_grad, to_f64

pytestmark = pytest.mark.slow


def _err(a, b):
    """max|a - b| / max|b| (|a - b| where b is zero: the single block's)."""
    den = abs(b) if np.ndim(b) == 0 else np.abs(b).max()
    num = abs(a - b) if np.ndim(b) == 0 else np.abs(a - b).max()
    return float(num / den) if den > 0 else float(num)


def _case(B, T, D, w_std, seed=0):
    X, [W] = make_layer_inputs(B, T, D, seed=seed, x_std=1.0, w_std=w_std, bf16=True)
    dY = make_upstream_grad(B, T, D, seed=seed + 1, bf16=True).astype(np.float64)
    return X.astype(np.float64), to_f64(W), dY


def _exact(X, W, L, H, gamma, dY, residual=False):
    Y, cache = orc.forward(X, W, L, H, gamma, residual)
    g = orc.backward(cache, dY)
    g["Y"] = Y
    return g


def _model(X, W, L, H, gamma, dY, rnd, residual=False):
    Y, cache = bm.forward(X, W, L, H, gamma, rnd, residual)
    g = bm.backward(cache, dY, rnd)
    g["Y"] = Y
    return g


@pytest.mark.parametrize("L,residual", [(20, True), (16, False), (130, False)])
def test_model_without_rounding_is_the_oracle(L, residual):
    """No rounding point active: the oracle's outputs and gradients, with 7
    blocks (L=20), 40 blocks (L=16) and a single block (L=130)."""
    X, W, dY = _case(2, 130 if L != 16 else 640, 64, 0.3)
    H = 4
    ref = _exact(X, W, L, H, 0.8, dY, residual)
    got = _model(X, W, L, H, 0.8, dY, bm.rounder(points=()), residual)
    for k in ref:
        assert _err(got[k], ref[k]) < 1e-12, k


def test_each_rounding_point_reaches_its_outputs():
    """Rounding one point alone changes exactly the outputs downstream of it
    (a misplaced or dead point fails here)."""
    X, W, dY = _case(1, 96, 64, 0.3)
    ref = _exact(X, W, 16, 4, 0.8, dY)
    fwd_only = {"y": {"Y"}}
    bwd = {"du": {"dWg", "dX", "dWq", "dWk", "dWv", "dWo", "dwp", "dgamma", "dWm"},
           "pb": {"dWm"}, "pbwd": {"dWv", "dX"}, "dx": {"dX"}, "mt": {"dWm", "Y", "dWg", "dX"},
           "dz": {"dWq", "dWk", "dX"}}
    for p in bm.POINTS:
        got = _model(X, W, 16, 4, 0.8, dY, bm.rounder(points=(p,)))
        moved = {k for k in ref if _err(got[k], ref[k]) > 1e-10}
        assert moved, f"rounding at {p} changes nothing"
        want = fwd_only.get(p) or bwd.get(p)
        if want is not None:
            assert moved <= want | {"Y"} and (moved & want), (p, moved)


@pytest.mark.parametrize("case", list(tl.DERIVED))
def test_derived_bounds_follow_from_the_model(case):
    """Each listed bound is between MARGIN and 2 * MARGIN times the largest
    error of its tensor over the jittered ensemble; every tensor left at the
    regular bound stays below it with the margin."""
    B, T, D, H, L, w_std, gamma, residual, bounds = tl.DERIVED[case]
    X, W, dY = _case(B, T, D, w_std)
    ref = _exact(X, W, L, H, gamma, dY, residual)
    worst = {}
    for k in range(tl.ENSEMBLE):
        got = _model(X, W, L, H, gamma, dY, bm.rounder(jitter=tl.JITTER, seed=k), residual)
        for key in ref:
            if key in ("dN_in", "dZ_in"):
                continue
            worst[key] = max(worst.get(key, 0.0), _err(got[key], ref[key]))
    print(case, " ".join(f"{k}={v:.2e}" for k, v in worst.items()))
    for key, e in worst.items():
        b = tl.bound(case, key)
        assert b >= tl.MARGIN * e, (case, key, e, b)
        if key in bounds:
            assert b <= 2 * tl.MARGIN * e, (case, key, e, b)


@pytest.mark.parametrize("case", list(tl.SAMPLED))
def test_sampled_bounds_follow_from_the_model(case):
    """The same for full-size launches checked on sampled sequences: the
    model and the oracle run on those sequences alone."""
    B, T, D, H, L, w_std, gamma, rows, bounds = tl.SAMPLED[case]
    X, W, dY = _case(B, T, D, w_std)
    X, dY = X[list(rows)], dY[list(rows)]
    ref = _exact(X, W, L, H, gamma, dY)
    worst = {}
    for k in range(tl.ENSEMBLE):
        got = _model(X, W, L, H, gamma, dY, bm.rounder(jitter=tl.JITTER, seed=k))
        for key in ref:
            worst[key] = max(worst.get(key, 0.0), _err(got[key], ref[key]))
    print(case, " ".join(f"{k}={v:.2e}" for k, v in worst.items()))
    for key, e in worst.items():
        b = tl.bound(case, key)
        assert b >= tl.MARGIN * e, (case, key, e, b)
        if key in bounds:
            assert b <= 2 * tl.MARGIN * e, (case, key, e, b)


@pytest.mark.parametrize("case", list(tl.DERIVED_FORWARD))
def test_derived_forward_bounds_follow_from_the_model(case):
    """The same for the cases compared on the forward output alone."""
    B, T, D, H, L, w_std, gamma, residual, bounds = tl.DERIVED_FORWARD[case]
    X, W, _ = _case(B, T, D, w_std)
    Y = orc.forward(X, W, L, H, gamma, residual)[0]
    worst = max(_err(bm.forward(X, W, L, H, gamma, bm.rounder(jitter=tl.JITTER, seed=k),
                                residual)[0], Y) for k in range(tl.ENSEMBLE))
    print(case, f"Y={worst:.2e}")
    assert tl.MARGIN * worst <= bounds["Y"] <= 2 * tl.MARGIN * worst


def test_stack_bounds_follow_from_the_model():
    """The 12-layer stack's bounds per kind of tensor (w_p and decay
    gradients of all layers) against the model of the stack on the compared
    sequence, with the same margin rule; all other tensors stay within the
    regular bound with the margin."""
    s = tl.STACK
    X, Ws = make_layer_inputs(s["B"], s["T"], s["D"], seed=0, x_std=1.0, w_std=s["w_std"],
                              bf16=True, n_layers=s["layers"])
    dY = make_upstream_grad(s["B"], s["T"], s["D"], seed=1, bf16=True)
    rows = list(s["rows"])
    Xr, dYr = X[rows].astype(np.float64), dY[rows].astype(np.float64)
    Wr = [to_f64(W) for W in Ws]
    L, H, gamma = s["L"], s["H"], s["gamma"]
    Yr, caches = orc.stack_forward(Xr, Wr, L, H, gamma, True)
    dXr, gref = orc.stack_backward(caches, dYr)
    worst = {}
    rounders = [bm.rounder()] + [bm.rounder(jitter=tl.JITTER, seed=k)
                                  for k in range(tl.STACK_ENSEMBLE)]
    for rnd in rounders:
        Ym, dXm, gm = bm.stack(Xr, Wr, L, H, gamma, dYr, rnd)
        cur = {"Y": _err(Ym, Yr), "dX": _err(dXm, dXr)}
        for li in range(s["layers"]):
            for k in ("dWq", "dWk", "dWv", "dWo", "dWm", "dWg", "dwp", "dgamma"):
                cur[k] = max(cur.get(k, 0.0), _err(gm[li][k], gref[li][k]))
        for k, v in cur.items():
            worst[k] = max(worst.get(k, 0.0), v)
    print("stack", " ".join(f"{k}={v:.2e}" for k, v in worst.items()))
    for k, e in worst.items():
        b = s["bounds"].get(k, tl.TOL_BF16)
        assert b >= tl.MARGIN * e, (k, e, b)
        if k in s["bounds"]:
            assert b <= 2 * tl.MARGIN * e, (k, e, b)


def _lm_params(arrs, n_layer):
    from paper_2608_13578_amd.inputs import MODEL_LAYER_ARRAYS
    f = [np.asarray(a, dtype=np.float64) for a in arrs]
    P = {"E": f[0], "Pe": f[1], "lnf_g": f[-2], "lnf_b": f[-1], "layers": []}
    for l in range(n_layer):
        a = dict(zip(MODEL_LAYER_ARRAYS, f[2 + 13 * l: 2 + 13 * (l + 1)]))
        P["layers"].append({k: a[k] for k in ("ln1_g", "ln1_b", "ln2_g", "ln2_b", "W1", "W2")})
        P["layers"][-1]["mix"] = {k: a[k] for k in ("Wq", "Wk", "Wv", "Wo", "Wm", "Wg", "wp")}
    return P


def test_lm_model_without_rounding_is_the_oracle():
    import lm_bf16_model as lmm
    from oracle import model_oracle as mo
    from paper_2608_13578_amd.inputs import make_model_inputs
    arrs, tok, tgt = make_model_inputs(97, 64, 96, 2, 2, seed=0)
    P = _lm_params(arrs, 2)
    tok, tgt = tok.astype(np.int64), tgt.astype(np.int64)
    loss, c = mo.forward(tok, tgt, P, 32, 4, 0.8)
    G = mo.flatten(mo.backward(c))
    none = bm.rounder(points=())
    loss_m, cm = lmm.forward(tok, tgt, P, 32, 4, 0.8, none)
    Gm = mo.flatten(lmm.backward(cm, none))
    assert abs(loss_m - loss) < 1e-12
    for a, b in zip(Gm, G):
        assert _err(np.asarray(a), np.asarray(b)) < 1e-11


def test_lm_bounds_follow_from_the_model():
    """The benchmarked language model's per-array bounds (tolerances.LM)
    against lm_bf16_model, with the same margin rule; every other array stays
    within the regular bound with the margin."""
    import lm_bf16_model as lmm
    from oracle import model_oracle as mo
    from paper_2608_13578_amd.inputs import make_model_inputs, model_array_names
    s = tl.LM
    arrs, tok, tgt = make_model_inputs(s["V"], s["d"], s["T"], s["layers"], s["B"], seed=0)
    P = _lm_params(arrs, s["layers"])
    tok, tgt = tok.astype(np.int64), tgt.astype(np.int64)
    _, c = mo.forward(tok, tgt, P, s["L"], s["H"], s["gamma"])
    G = mo.flatten(mo.backward(c))
    names = model_array_names(s["layers"])
    worst = {}
    rounders = [bm.rounder()] + [bm.rounder(jitter=tl.JITTER, seed=k)
                                  for k in range(1, tl.LM_ENSEMBLE)]
    for rnd in rounders:
        _, cm = lmm.forward(tok, tgt, P, s["L"], s["H"], s["gamma"], rnd)
        Gm = mo.flatten(lmm.backward(cm, rnd))
        for nm, a, b in zip(names, Gm, G):
            worst[nm] = max(worst.get(nm, 0.0), _err(np.asarray(a), np.asarray(b)))
    print("lm", " ".join(f"{k}={v:.2e}" for k, v in sorted(worst.items(), key=lambda kv: -kv[1])[:8]))
    for k, e in worst.items():
        b = s["bounds"].get(k, tl.TOL_BF16)
        assert b >= tl.MARGIN * e, (k, e, b)
        if k in s["bounds"]:
            assert b <= 2 * tl.MARGIN * e, (k, e, b)


def test_model_with_carry_without_rounding_is_the_oracle():
    """The chunked form (an incoming memory state) of the model, with no
    rounding, is the oracle's chunk."""
    X, W, dY = _case(2, 640, 64, 0.3)
    rng = np.random.default_rng(5)
    Z = np.array([3.0, 1.5])
    N = Z[:, None] * rng.standard_normal((2, 64)) * 0.5
    Y, c = orc.forward(X, W, 16, 4, 0.8, carry=(N, Z))
    ref = orc.backward(c, dY)
    ref["Y"] = Y
    none = bm.rounder(points=())
    Ym, cm = bm.forward(X, W, 16, 4, 0.8, none, carry=(N, Z))
    got = bm.backward(cm, dY, none)
    got["Y"] = Ym
    for k in ref:
        assert _err(np.asarray(got[k]), np.asarray(ref[k])) < 1e-12, k
