"""Float64 model of where the bf16 GPU path rounds (test infrastructure).

The bf16 layer keeps its activations, and the operands it feeds the matrix
cores, in bfloat16 while it accumulates in float32.  This module repeats the
layer of Sec. 3.2-3.8 (and the chain rule through it) in float64 and rounds a
value to bf16 at each place where the GPU path stores it or hands it to the
matrix cores in bf16, and nowhere else.  The gap between this model and the
exact oracle is the error that bf16 storage alone causes; it is what the
parity bounds of the bf16 stress cases are derived from.

The points where a value is rounded (``POINTS``):
  qkv   Q, K, V as stored by the projection (Sec. 3.3);
  pfwd  the softmax probabilities as the operand of the value product;
  o     the attention output, stored; its row sums with dO give delta;
  h     the output projection H (Sec. 3.3), stored; pooling reads it;
  st    the block summaries as the operand of the W_m product (the memory
        path projects S and scans the projections);
  mt    the memory M as the operand of the W_m weight gradient (and of the
        W_m product of an incoming state's memory);
  g     the gate, stored for the backward pass in fp16 (the output uses it
        unrounded);
  y     the layer output (Sec. 3.8), stored;
  du    the gate pre-activation gradient, stored;
  pb    the block sums of dY * G (the shifted context gradient) as the
        operand of the W_m weight gradient (the memory gradient takes them
        as a pair hi + lo of bf16 values, which is float32-accurate);
  dh    the gradient of H, stored;
  do    the gradient of the attention output, stored;
  dz    the softmax-input gradient as the operand of the dQ / dK products;
  pbwd  the recomputed probabilities as the operand of the dV product;
  dqkv  dQ, dK, dV, stored;
  dx    the input gradient, stored.

``rounder(points, jitter, seed)`` builds the rounding function.  With a
jitter j > 0 each value is first multiplied by (1 + j * N(0, 1)): the GPU
sums in float32, in its own order, so its value before a rounding differs
from the float64 one in the last float32 bits, amplified where sums cancel,
and the bf16 rounding of some elements goes the other way.  The rounded
results of these problems are very sensitive to such flips (a peaked softmax
turns one flipped element of Q into a different probability row), so the
error of one realisation says little; a jittered ensemble samples the spread
of errors that bf16 storage can produce.

Only the test suite imports this module; it uses the oracle's small helpers
(block ranges, softmax, memory weights) and nothing from the GPU package
except the bf16 rounding of the seeded-input module, which holds no layer
arithmetic.
"""

import numpy as np

from oracle import bcmt_oracle as orc
from paper_2608_13578_amd.inputs import bf16_round

POINTS = ("qkv", "pfwd", "o", "h", "st", "mt", "g", "y", "du", "pb", "dh", "do", "dz", "pbwd",
          "dqkv", "dx")
# points stored as fp16 rather than bf16
FP16_POINTS = ("g",)
# with the language model around the layer (lm_bf16_model): its own tensors
ALL_POINTS = POINTS + ("lm",)


def rounder(points=ALL_POINTS, jitter=0.0, seed=0):
    """rnd(point, x): x rounded to bf16 (fp16 for FP16_POINTS) if ``point`` is
    in ``points``."""
    rng = np.random.default_rng(seed)
    active = set(points)

    def rnd(point, x):
        if point not in active:
            return x
        x = np.asarray(x, dtype=np.float64)
        if jitter > 0.0:
            x = x * (1.0 + jitter * rng.standard_normal(x.shape))
        if point in FP16_POINTS:
            return x.astype(np.float32).astype(np.float16).astype(np.float64)
        return bf16_round(x.astype(np.float32))[0].astype(np.float64)
    return rnd


def exact(point, x):
    return x


def _heads(M, b0, b1, h):
    B, _, D = M.shape
    n = b1 - b0
    return M[:, b0:b1].reshape(B, n, h, D // h).transpose(0, 2, 1, 3)


def _wgrad(A, B):
    """sum over batch and tokens of A[b, t]^T B[b, t] (as one matrix product)."""
    return A.reshape(-1, A.shape[-1]).T @ B.reshape(-1, B.shape[-1])


def _unheads(m):
    B, h, n, dh = m.shape
    return m.transpose(0, 2, 1, 3).reshape(B, n, h * dh)


def forward(X, W, L, h, gamma, rnd, residual=False, carry=None):
    """The layer with bf16 rounding at the GPU path's points; (Y, cache).

    ``carry`` = (N_in, Z_in): X is a chunk after earlier blocks, as in the
    oracle; the incoming memory N_in / Z_in is projected from its bf16
    value, and the chunk's projections continue the decayed sum from it."""
    X = np.asarray(X, dtype=np.float64)
    B, T, D = X.shape
    nb = orc.n_blocks(T, L)
    blk = np.arange(T) // L
    ranges = orc.block_ranges(T, L)
    dh = D // h
    Q, K, V = (rnd("qkv", X @ W[k]) for k in ("Wq", "Wk", "Wv"))
    O = np.zeros_like(X)
    probs = []
    for (b0, b1) in ranges:
        n = b1 - b0
        z = _heads(Q, b0, b1, h) @ _heads(K, b0, b1, h).transpose(0, 1, 3, 2) / np.sqrt(dh)
        z = np.where(np.tril(np.ones((n, n), dtype=bool)), z, -np.inf)
        A = orc.softmax_last(z)
        probs.append(A)
        O[:, b0:b1] = _unheads(rnd("pfwd", A) @ _heads(V, b0, b1, h))
    O = rnd("o", O)
    Hl = rnd("h", O @ W["Wo"])
    s = Hl @ W["wp"]
    a = np.zeros_like(s)
    S = np.zeros((B, nb, D))
    for i, (b0, b1) in enumerate(ranges):
        a[:, b0:b1] = orc.softmax_last(s[:, b0:b1])
        S[:, i] = np.einsum("bt,btd->bd", a[:, b0:b1], Hl[:, b0:b1])
    extra = {}
    Qm = rnd("st", S) @ W["Wm"]  # the projected summaries, scanned like S
    if carry is not None:
        N_in, Z_in = (np.asarray(a, dtype=np.float64) for a in carry)
        M, Nacc, Zacc = orc.exp_memory_carry(S, gamma, N_in, Z_in)
        Mext = np.concatenate([orc.carry_memory(N_in, Z_in)[:, None], M], axis=1)
        Mt = rnd("mt", Mext)
        Pc = Mt[:, 0] @ W["Wm"]
        P = orc.exp_memory_carry(Qm, gamma, Pc * Z_in[:, None], Z_in)[0]
        C = np.concatenate([Pc[:, None], P[:, :-1]], axis=1)
        extra = dict(N_in=N_in, Z_in=Z_in, Mext=Mext, Nacc=Nacc, Zacc=Zacc)
    else:
        Aw = orc.memory_weights(nb, gamma)[0]
        M = np.einsum("ij,bjd->bid", Aw, S)
        Mt = rnd("mt", M)
        P = np.einsum("ij,bjd->bid", Aw, Qm)
        C = np.zeros_like(P)
        C[:, 1:] = P[:, :-1]
    G = orc.sigmoid(Hl @ W["Wg"])
    Y = Hl + G * C[:, blk]
    if residual:
        Y = Y + X
    Y = rnd("y", Y)
    cache = dict(X=X, W=W, L=L, h=h, gamma=float(gamma), residual=residual, Q=Q, K=K, V=V,
                 probs=probs, O=O, Hl=Hl, a=a, S=S, Mt=Mt, C=C, G=rnd("g", G), **extra)
    return Y, cache


def backward(cache, dY, rnd):
    """Gradients of sum(dY * Y) with the GPU path's bf16 roundings."""
    c = cache
    W, L, h, gamma = c["W"], c["L"], c["h"], c["gamma"]
    X, Hl, G, C = c["X"], c["Hl"], c["G"], c["C"]
    dY = np.asarray(dY, dtype=np.float64)
    B, T, D = X.shape
    nb = orc.n_blocks(T, L)
    blk = np.arange(T) // L
    ranges = orc.block_ranges(T, L)
    dh = D // h
    dU = rnd("du", dY * C[:, blk] * G * (1.0 - G))
    dC = np.stack([(dY * G)[:, b0:b1].sum(axis=1) for b0, b1 in ranges], axis=1)
    dWg = _wgrad(Hl, dU)
    extra = {}
    if "Mext" in c:
        # the incoming memory feeds block 0: P-bar has one more row in front
        dWm = _wgrad(c["Mt"][:, :-1], rnd("pb", dC))
        mem = dict(P=W, S=c["S"], Mext=c["Mext"], Nacc=c["Nacc"], Zacc=c["Zacc"],
                   N_in=c["N_in"], Z_in=c["Z_in"], gamma=gamma, per_channel=False)
        dS, _, dgamma, extra = orc._memory_carry_backward(mem, dC, None)
    else:
        Pb = np.zeros_like(dC)
        Pb[:, :-1] = dC[:, 1:]
        dWm = _wgrad(c["Mt"], rnd("pb", Pb))
        dM = Pb @ W["Wm"].T
        # M = A(gamma) S: dS = A^T dM and dgamma = sum dM . (dA/dgamma) S.
        Aw, w, z = orc.memory_weights(nb, gamma)
        dS = np.einsum("ij,bid->bjd", Aw, dM)
        dist = np.arange(nb)[:, None] - np.arange(nb)[None, :]
        dw = np.where(dist >= 1, dist * np.power(gamma, np.where(dist >= 1, dist - 1, 0)), 0.0)
        dA = (dw - Aw * dw.sum(axis=1)[:, None]) / z[:, None]
        dgamma = float(np.einsum("ij,bid,bjd->", dA, dM, c["S"]))
    dH = dY + dU @ W["Wg"].T
    dwp = np.zeros(D)
    for i, (b0, b1) in enumerate(ranges):
        a = c["a"][:, b0:b1]
        Hb = Hl[:, b0:b1]
        da = np.einsum("bd,btd->bt", dS[:, i], Hb)
        ds = a * (da - np.einsum("bd,bd->b", dS[:, i], c["S"][:, i])[:, None])
        dH[:, b0:b1] += a[:, :, None] * dS[:, i][:, None, :] + ds[:, :, None] * W["wp"]
        dwp += np.einsum("bt,btd->d", ds, Hb)
    dH = rnd("dh", dH)
    dWo = _wgrad(c["O"], dH)
    dO = rnd("do", dH @ W["Wo"].T)
    dQ, dK, dV = np.zeros_like(X), np.zeros_like(X), np.zeros_like(X)
    for bi, (b0, b1) in enumerate(ranges):
        A = c["probs"][bi]
        q, k, v = (_heads(t, b0, b1, h) for t in (c["Q"], c["K"], c["V"]))
        do, o = _heads(dO, b0, b1, h), _heads(c["O"], b0, b1, h)
        delta = (do * o).sum(axis=-1, keepdims=True)
        dz = rnd("dz", A * (do @ v.transpose(0, 1, 3, 2) - delta))
        dQ[:, b0:b1] = _unheads(dz @ k / np.sqrt(dh))
        dK[:, b0:b1] = _unheads(dz.transpose(0, 1, 3, 2) @ q / np.sqrt(dh))
        dV[:, b0:b1] = _unheads(rnd("pbwd", A).transpose(0, 1, 3, 2) @ do)
    dQ, dK, dV = (rnd("dqkv", t) for t in (dQ, dK, dV))
    dX = dQ @ W["Wq"].T + dK @ W["Wk"].T + dV @ W["Wv"].T
    if c["residual"]:
        dX = dX + dY
    dX = rnd("dx", dX)
    return dict(dX=dX, dWq=_wgrad(X, dQ), dWk=_wgrad(X, dK), dWv=_wgrad(X, dV), dWo=dWo, dWm=dWm,
                dWg=dWg, dwp=dwp, dgamma=dgamma, **extra)


def stack(X, layers, L, h, gamma, dY, rnd, residual=True):
    """A stack of layers (each layer's output is the next one's input) with
    its backward; returns (Y, dX, [gradients per layer])."""
    caches = []
    for W in layers:
        X, cache = forward(X, W, L, h, gamma, rnd, residual)
        caches.append(cache)
    g = dY
    grads = [None] * len(layers)
    for i in reversed(range(len(layers))):
        grads[i] = backward(caches[i], g, rnd)
        g = grads[i]["dX"]
    return X, g, grads
