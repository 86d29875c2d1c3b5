"""Derives the per-array parity bounds of the benchmarked language model
(tolerances.LM) from its float64 bf16 rounding model (test infrastructure).

    python tests/lm_bounds.py [realizations]

runs lm_bf16_model on the case of tolerances.LM with the exact rounder and
(realizations - 1) jittered ones (tolerances.JITTER, seeds 1, 2, ...), takes
each array's largest max-abs-relative error against the float64 oracle,
and prints MARGIN times it, rounded up to 1e-3, for the arrays whose bound
exceeds the regular bf16 bound.  Only oracle/ and the rounding models run.
"""

import math
import os
import sys
from concurrent.futures import ProcessPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)
sys.path.insert(0, os.path.dirname(HERE))

import bf16_model as bm  # noqa: E402
import lm_bf16_model as lmm  # noqa: E402
import tolerances as tl  # noqa: E402
from oracle import model_oracle as mo  # noqa: E402


def _case():
    from paper_2608_13578_amd.inputs import MODEL_LAYER_ARRAYS, make_model_inputs
    s = tl.LM
    arrs, tok, tgt = make_model_inputs(s["V"], s["d"], s["T"], s["layers"], s["B"], seed=0)
    f = [np.asarray(a, dtype=np.float64) for a in arrs]
    P = {"E": f[0], "Pe": f[1], "lnf_g": f[-2], "lnf_b": f[-1], "layers": []}
    for l in range(s["layers"]):
        a = dict(zip(MODEL_LAYER_ARRAYS, f[2 + 13 * l: 2 + 13 * (l + 1)]))
        P["layers"].append({k: a[k] for k in ("ln1_g", "ln1_b", "ln2_g", "ln2_b", "W1", "W2")})
        P["layers"][-1]["mix"] = {k: a[k] for k in ("Wq", "Wk", "Wv", "Wo", "Wm", "Wg", "wp")}
    return P, tok.astype(np.int64), tgt.astype(np.int64)


def _err(a, b):
    a, b = np.asarray(a).reshape(-1), np.asarray(b).reshape(-1)
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-300))


def realization_errors(seed):
    """{array: error} of one realization (seed 0: no jitter)."""
    from paper_2608_13578_amd.inputs import model_array_names
    s = tl.LM
    P, tok, tgt = _case()
    _, c = mo.forward(tok, tgt, P, s["L"], s["H"], s["gamma"])
    G = mo.flatten(mo.backward(c))
    rnd = bm.rounder() if seed == 0 else bm.rounder(jitter=tl.JITTER, seed=seed)
    _, cm = lmm.forward(tok, tgt, P, s["L"], s["H"], s["gamma"], rnd)
    Gm = mo.flatten(lmm.backward(cm, rnd))
    names = model_array_names(s["layers"])
    return {nm: _err(a, b) for nm, a, b in zip(names, Gm, G)}


def derive(n, workers=4):
    worst = {}
    with ProcessPoolExecutor(workers) as ex:
        for e in ex.map(realization_errors, range(n)):
            for k, v in e.items():
                worst[k] = max(worst.get(k, 0.0), v)
    bounds = {}
    for k, v in worst.items():
        b = math.ceil(tl.MARGIN * v * 1000.0) / 1000.0
        if b > tl.TOL_BF16:
            bounds[k] = b
    return worst, bounds


if __name__ == "__main__":
    n = int(sys.argv[1]) if len(sys.argv) > 1 else tl.LM_DERIVE
    worst, bounds = derive(n)
    print(f"{n} realizations; largest errors:",
          " ".join(f"{k}={v:.2e}" for k, v in sorted(worst.items(), key=lambda kv: -kv[1])[:10]))
    print("bounds =", {k: bounds[k] for k in sorted(bounds, key=lambda k: (len(k), k))})
