"""Seeded synthetic inputs for the BCMT layer.

This module holds no arithmetic of the method: it only draws Gaussian arrays
from a seeded NumPy generator and rounds them to bfloat16 when asked.  The same
arrays feed the HIP library and the CPU oracle.

Draw order for one layer: X, then Wq, Wk, Wv, Wo, wp, Wm, Wg (each
``standard_normal(...) * std`` in float32).  An upstream gradient dY comes from
its own generator.  Weights are input-major [D_in, D_out] so that y = x @ W.
"""

import numpy as np

WEIGHT_ORDER = ("Wq", "Wk", "Wv", "Wo", "wp", "Wm", "Wg")


def bf16_round(x):
    """Round float32 values to the nearest bfloat16 (ties to even).

    Returns (float32 array holding the rounded values, uint16 bit patterns).
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    r = ((u + bias) & np.uint32(0xFFFF0000)).astype(np.uint32)
    return r.view(np.float32), (r >> np.uint32(16)).astype(np.uint16)


def _draw(rng, shape, std):
    return rng.standard_normal(shape, dtype=np.float32) * np.float32(std)


def layer_weights(rng, D, w_std):
    """One layer's weights, drawn in WEIGHT_ORDER (float32)."""
    out = {}
    for name in WEIGHT_ORDER:
        shape = (D,) if name == "wp" else (D, D)
        out[name] = _draw(rng, shape, w_std)
    return out


def make_layer_inputs(B, T, D, seed=0, x_std=1.0, w_std=0.02, bf16=False,
                      n_layers=1):
    """X [B, T, D] and ``n_layers`` weight sets, from one generator.

    When ``bf16`` is true every array is rounded to bfloat16 values (kept in
    float32), so that both sides see exactly the same numbers.
    Returns (X, [weights per layer]).
    """
    rng = np.random.default_rng(seed)
    X = _draw(rng, (B, T, D), x_std)
    layers = [layer_weights(rng, D, w_std) for _ in range(n_layers)]
    if bf16:
        X = bf16_round(X)[0]
        layers = [{k: bf16_round(v)[0] for k, v in w.items()} for w in layers]
    return X, layers


def make_upstream_grad(B, T, D, seed=1, std=1.0, bf16=False):
    """Upstream gradient dY ~ N(0, std^2) from its own generator."""
    rng = np.random.default_rng(seed)
    g = _draw(rng, (B, T, D), std)
    if bf16:
        g = bf16_round(g)[0]
    return g


def to_f64(layer):
    """Float64 copy of a weight dict (for the oracle)."""
    return {k: np.asarray(v, dtype=np.float64) for k, v in layer.items()}
