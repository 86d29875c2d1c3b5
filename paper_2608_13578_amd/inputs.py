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


# ---- language model (flat parameter order of the model entry points)

MODEL_LAYER_ARRAYS = ("ln1_g", "ln1_b", "Wq", "Wk", "Wv", "Wo", "Wm", "Wg", "wp", "ln2_g",
                      "ln2_b", "W1", "W2")


def model_array_names(n_layer):
    """Names of the flat parameter vector's arrays, in order."""
    names = ["E", "Pe"]
    for l in range(n_layer):
        names += [f"{l}.{k}" for k in MODEL_LAYER_ARRAYS]
    return names + ["lnf_g", "lnf_b"]


def make_model_inputs(V, d, T, n_layer, B, seed=0, w_std=0.1, ln_std=0.2):
    """A seeded model parameter set and a token batch.

    Returns (arrays, tokens, targets): float32 arrays in model_array_names
    order with the matrices (E, Pe, W*) rounded to bfloat16 values and the
    LayerNorm gains 1 + N(0, ln_std^2), biases and wp N(0, ...); tokens
    uniform in [0, V) as int32 [B, T] and targets the tokens shifted by one
    (the last position takes a fresh draw)."""
    rng = np.random.default_rng(seed)
    out = [bf16_round(_draw(rng, (V, d), w_std))[0], bf16_round(_draw(rng, (T, d), w_std))[0]]
    for _ in range(n_layer):
        for k in MODEL_LAYER_ARRAYS:
            if k.endswith("_g"):
                out.append((1 + _draw(rng, (d,), ln_std)).astype(np.float32))
            elif k.endswith("_b"):
                out.append(_draw(rng, (d,), ln_std))
            elif k == "wp":
                out.append(bf16_round(_draw(rng, (d,), w_std))[0])
            elif k == "W1":
                out.append(bf16_round(_draw(rng, (d, 4 * d), w_std))[0])
            elif k == "W2":
                out.append(bf16_round(_draw(rng, (4 * d, d), w_std))[0])
            else:
                out.append(bf16_round(_draw(rng, (d, d), w_std))[0])
    out.append((1 + _draw(rng, (d,), ln_std)).astype(np.float32))
    out.append(_draw(rng, (d,), ln_std))
    tokens = rng.integers(0, V, (B, T)).astype(np.int32)
    targets = np.concatenate([tokens[:, 1:], rng.integers(0, V, (B, 1)).astype(np.int32)], axis=1)
    return out, tokens, targets
