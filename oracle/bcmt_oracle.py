"""Float64 CPU oracle of the BCMT token-mixing layer (forward and backward).

TEST INFRASTRUCTURE ONLY.  This module is the slow, plainly written reference
that the HIP implementation is checked against.  Only the test suite, the
smoke check and the CPU-baseline leg of the benchmark may import it; the
product path never does, and this module imports nothing from the product
package.

Every function follows "BCMT: Blockwise Causal Memory Transformer"
(arXiv 2608.13578).  Section numbers below are the paper's.

Notation (the paper overloads two letters, so they are renamed here):
  * the memory decay, written alpha in Sec. 3.5, is ``gamma`` here;
  * the pooling softmax weights, also written alpha in Sec. 3.4, are ``a``;
  * ``h`` is the number of heads and ``dh = D / h`` the head width (Sec. 3.3);
  * ``Hloc`` is the local representation H of Sec. 3.3 (the paper reuses H).

Readings of points the paper leaves open (all listed in the design notes):
  * no biases anywhere (none appear in any equation of Sec. 3.3-3.8);
  * the causal mask of Sec. 3.3 keeps the diagonal (a token attends to itself
    and to earlier tokens of its block, Sec. 3.6) and is applied by exclusion;
  * the pooling softmax of Sec. 3.4 runs over all tokens of a block (the
    one-block shift of Sec. 3.5 is what keeps the layer causal);
  * a partial last block (Sec. 3.2) gets attention, pooling and broadcast over
    its own tokens only;
  * gamma = 0 uses 0**0 = 1, so the memory equals the block's own summary;
  * the residual form Y = X + layer(X) exists only for stacking layers; the
    paper's layer output is exactly Y = H + G * M_tokens (Sec. 3.8);
  * the paper states no backward pass; the one here is derived by hand and
    pinned by finite differences in the tests.

Per-channel decay: ``gamma`` may also be one decay per feature channel
([D]); each channel then has its own recurrence of Sec. 3.5 (and its own
normaliser Z), and the decay gradient is per channel.  This generalises the
paper's single decay (its suggested extension); a scalar is the paper's.

Chunked execution: a sequence cut at block boundaries into consecutive
chunks gives the same layer when each chunk starts the recurrence of Sec. 3.5
from the state the previous chunk ended with.  That state (the "carry") is
N = sum_j gamma^(k-j) S_j and Z = sum_j gamma^(k-j) over all earlier blocks j
(k the last of them); the first block of a chunk receives M = N / Z projected
by W_m, and Z = 0 stands for an empty history (the start of a sequence).

Parity status: forward pinned by library attention (dense / block-diagonal
causal), closed forms of the memory normaliser, convexity, gamma limits,
HOnly / W_m = 0 and W_g = 0 identities, and causality; backward pinned by
central finite differences; the carry pinned by chunked runs equal to the
whole sequence's (values and gradients) and by finite differences.
End-to-end values beyond those pins have no printed worked example in the
paper ("parity unpinned" beyond the pins).
"""

import numpy as np

PARAM_NAMES = ("Wq", "Wk", "Wv", "Wo", "Wm", "Wg", "wp")


def n_blocks(T, L):
    """Number of blocks, the ceiling of T / L (Sec. 3.2)."""
    return -(-T // L)


def block_ranges(T, L):
    """Contiguous, non-overlapping [start, end) token ranges (Sec. 3.2)."""
    return [(s, min(s + L, T)) for s in range(0, T, L)]


def sigmoid(u):
    """Logistic sigmoid (Sec. 3.8), evaluated without overflow."""
    out = np.empty_like(u)
    pos = u >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-u[pos]))
    e = np.exp(u[~pos])
    out[~pos] = e / (1.0 + e)
    return out


def softmax_last(z):
    """Max-subtracted softmax over the last axis."""
    z = z - z.max(axis=-1, keepdims=True)
    e = np.exp(z)
    return e / e.sum(axis=-1, keepdims=True)


def memory_weights(n, gamma):
    """Row-normalised weights of the exponential causal memory (Sec. 3.5).

    A[i, j] = gamma**(i-j) / sum_{j'<=i} gamma**(i-j') for j <= i, else 0, so
    that M = A @ S.  Each row is a convex combination.  Indices are 0-based.
    Also returns the unnormalised weights and their row sums.
    """
    i = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    lower = j <= i
    expo = np.where(lower, i - j, 0)
    w = np.where(lower, np.power(float(gamma), expo), 0.0)  # 0**0 == 1
    z = w.sum(axis=1)
    return w / z[:, None], w, z


def exp_memory(S, gamma):
    """M^(i) = sum_{j<=i} gamma^(i-j) S^(j) / sum_{j<=i} gamma^(i-j) (Sec. 3.5).

    S: [..., N_b, D] block summaries.  Written as the literal double sum, each
    memory vector touching only the summaries j <= i.
    """
    n = S.shape[-2]
    A, _, _ = memory_weights(n, gamma)
    M = np.empty_like(S)
    for i in range(n):
        M[..., i, :] = np.einsum("j,...jd->...d", A[i, :i + 1], S[..., :i + 1, :])
    return M


def _per_channel(gamma, D):
    """The decay as one value per channel [D] (a scalar repeated)."""
    return np.broadcast_to(np.asarray(gamma, dtype=np.float64), (D,))


def _z_channels(Z, D):
    """A normaliser shared by the channels ([B]) or per channel ([B, D]),
    as [B, D]."""
    Z = np.asarray(Z, dtype=np.float64)
    return np.repeat(Z[:, None], D, axis=1) if Z.ndim == 1 else Z


def exp_memory_carry(S, gamma, N_in, Z_in):
    """The memory of Sec. 3.5 for blocks that follow earlier ones.

    S: [B, n, D] summaries of this chunk's blocks; N_in [B, D] and Z_in
    ([B], or [B, D] per channel) aggregate the earlier blocks
    (N_in = sum_j gamma^(-1-j) S_j and Z_in = sum_j gamma^(-1-j) over blocks
    j < 0).  gamma is a scalar or one decay per channel [D].  Block i of the
    chunk then has the double sums of Sec. 3.5 over every block up to it,
    channel by channel:
      N_i = sum_{0<=j<=i} gamma^(i-j) S_j + gamma^(i+1) N_in,
      Z_i = sum_{0<=j<=i} gamma^(i-j)     + gamma^(i+1) Z_in,
    and M_i = N_i / Z_i.  Returns M, N and Z, all [B, n, D].
    """
    B, n, D = S.shape
    g = _per_channel(gamma, D)
    Zc = _z_channels(Z_in, D)
    N = np.zeros((B, n, D))
    Z = np.zeros((B, n, D))
    for i in range(n):
        for j in range(i + 1):
            N[:, i] += g ** (i - j) * S[:, j]
            Z[:, i] += g ** (i - j)
        N[:, i] += g ** (i + 1) * N_in
        Z[:, i] += g ** (i + 1) * Zc
    return N / Z, N, Z


def carry_memory(N_in, Z_in):
    """M = N / Z of the earlier blocks, or 0 for an empty history (Z = 0)."""
    N_in = np.asarray(N_in, dtype=np.float64)
    Z = _z_channels(Z_in, N_in.shape[1])
    safe = np.where(Z > 0, Z, 1.0)
    return np.where(Z > 0, N_in / safe, 0.0)


def block_causal_attention(Q, K, V, L, h):
    """Dense causal multi-head attention confined to each block (Sec. 3.3, 3.6).

    Q, K, V: [B, T, D].  Head i uses columns i*dh .. (i+1)*dh-1.  Within a
    block, query t sees keys u of the same block with u <= t.  Returns the
    concatenated head outputs [B, T, D] and the attention probabilities of
    every block, list of [B, h, Lb, Lb].
    """
    B, T, D = Q.shape
    dh = D // h
    out = np.zeros_like(Q)
    probs = []
    for s, e in block_ranges(T, L):
        n = e - s
        q = Q[:, s:e].reshape(B, n, h, dh).transpose(0, 2, 1, 3)
        k = K[:, s:e].reshape(B, n, h, dh).transpose(0, 2, 1, 3)
        v = V[:, s:e].reshape(B, n, h, dh).transpose(0, 2, 1, 3)
        z = q @ k.transpose(0, 1, 3, 2) / np.sqrt(dh)
        keep = np.tril(np.ones((n, n), dtype=bool))
        z = np.where(keep, z, -np.inf)  # excluded entries, whatever their value
        A = softmax_last(z)
        probs.append(A)
        o = A @ v
        out[:, s:e] = o.transpose(0, 2, 1, 3).reshape(B, n, D)
    return out, probs


def forward(X, P, L, h, gamma, residual=False, carry=None):
    """One BCMT token-mixing layer, X [B, T, D] -> Y [B, T, D] (Sec. 3.2-3.8).

    P: dict of float64 weights Wq, Wk, Wv, Wo, Wm, Wg [D, D] (input-major, so
    that y = x @ W) and wp [D].  Returns (Y, cache) with every intermediate.

    ``carry`` = (N_in [B, D], Z_in [B]) makes X a chunk that follows earlier
    blocks of the same sequences (see exp_memory_carry); the state after the
    chunk's last block is then cache["carry_out"] = (N_out, Z_out).  With a
    per-channel ``gamma`` [D] the normalisers are per channel: Z_in and
    Z_out are [B, D].
    """
    X = np.asarray(X, dtype=np.float64)
    B, T, D = X.shape
    nb = n_blocks(T, L)
    blk = np.arange(T) // L

    # Sec. 3.3: per-head projections and block-local causal attention.
    Q = X @ P["Wq"]
    K = X @ P["Wk"]
    V = X @ P["Wv"]
    Hcat, probs = block_causal_attention(Q, K, V, L, h)
    # Sec. 3.3: head concatenation and output projection; blocks concatenated.
    Hloc = Hcat @ P["Wo"]

    # Sec. 3.4: pooling scores, per-block softmax, adaptive summaries.
    s = Hloc @ P["wp"]                       # [B, T]
    a = np.zeros_like(s)
    S = np.zeros((B, nb, D))
    for i, (b0, b1) in enumerate(block_ranges(T, L)):
        a[:, b0:b1] = softmax_last(s[:, b0:b1])
        S[:, i] = np.einsum("bt,btd->bd", a[:, b0:b1], Hloc[:, b0:b1])

    # Sec. 3.5: normalised exponential memory, projection, one-block shift.
    per_channel = np.ndim(gamma) > 0
    if per_channel and carry is None:
        carry = (np.zeros((B, D)), np.zeros((B, D)))
    if carry is None:
        M = exp_memory(S, gamma)
        Mproj = M @ P["Wm"]
        Mcausal = np.zeros_like(Mproj)
        Mcausal[:, 1:] = Mproj[:, :-1]
        extra = {}
    else:
        N_in = np.asarray(carry[0], dtype=np.float64)
        Z_in = np.asarray(carry[1], dtype=np.float64)
        M, Nacc, Zacc = exp_memory_carry(S, gamma, N_in, Z_in)
        # The earlier blocks' memory precedes this chunk's first block.
        Mext = np.concatenate([carry_memory(N_in, Z_in)[:, None], M], axis=1)
        Mproj = Mext @ P["Wm"]
        Mcausal = Mproj[:, :-1].copy()
        Z_out = Zacc[:, -1].copy() if per_channel else Zacc[:, -1, 0].copy()
        extra = dict(N_in=N_in, Z_in=Z_in, Mext=Mext, Nacc=Nacc, Zacc=Zacc,
                     per_channel=per_channel, carry_out=(Nacc[:, -1].copy(), Z_out))

    # Sec. 3.7: broadcast to tokens; Sec. 3.8: gate and injection.
    Mtok = Mcausal[:, blk]                   # [B, T, D]
    U = Hloc @ P["Wg"]
    G = sigmoid(U)
    Y = Hloc + G * Mtok
    if residual:
        Y = Y + X
    cache = dict(X=X, P=P, L=L, h=h,
                 gamma=np.asarray(gamma, dtype=np.float64) if per_channel else float(gamma),
                 residual=residual,
                 Q=Q, K=K, V=V, probs=probs, Hcat=Hcat, Hloc=Hloc, s=s, a=a,
                 S=S, M=M, Mproj=Mproj, Mcausal=Mcausal, U=U, G=G, **extra)
    return Y, cache


def backward(cache, dY, dcarry=None):
    """Gradients of sum(dY * Y) for the layer of ``forward``.

    The paper gives no backward pass; this is the chain rule applied to the
    forward steps in reverse order.  Weight gradients are summed over the
    batch.  Returns a dict with dX, dWq, dWk, dWv, dWo, dWm, dWg, dwp, dgamma.

    For a chunk (``forward`` with a carry) the loss also holds
    sum(dN_out * N_out) + sum(dZ_out * Z_out) with ``dcarry`` = (dN_out,
    dZ_out) (None: zero), and the result adds dN_in and dZ_in, the gradients
    of the incoming state.
    """
    c = cache
    P, L, h, gamma = c["P"], c["L"], c["h"], c["gamma"]
    X, Hloc, G, Mcausal = c["X"], c["Hloc"], c["G"], c["Mcausal"]
    dY = np.asarray(dY, dtype=np.float64)
    B, T, D = X.shape
    nb = n_blocks(T, L)
    blk = np.arange(T) // L
    ranges = block_ranges(T, L)

    # Gate and injection: Y = Hloc + G * Mtok, G = sigmoid(Hloc @ Wg).
    dH = dY.copy()
    dG = dY * Mcausal[:, blk]
    dU = dG * G * (1.0 - G)
    dMtok = dY * G
    dWg = np.einsum("btd,bte->de", Hloc, dU)
    dH += dU @ P["Wg"].T
    # Broadcast: each block's memory vector is summed over its tokens.
    dMcausal = np.zeros((B, nb, D))
    for i, (b0, b1) in enumerate(ranges):
        dMcausal[:, i] = dMtok[:, b0:b1].sum(axis=1)

    extra = {}
    if "carry_out" not in c:
        # Shift and projection: Mcausal[i] = Mproj[i-1], Mproj = M @ Wm.
        dMproj = np.zeros_like(dMcausal)
        dMproj[:, :-1] = dMcausal[:, 1:]
        dWm = np.einsum("bid,bie->de", c["M"], dMproj)
        dM = dMproj @ P["Wm"].T

        # Memory M = A(gamma) @ S with A the normalised decay weights.
        A, w, z = memory_weights(nb, gamma)
        dS = np.einsum("ij,bid->bjd", A, dM)
        i_idx = np.arange(nb)[:, None]
        j_idx = np.arange(nb)[None, :]
        dist = i_idx - j_idx
        lower = dist >= 0
        # d/dgamma of gamma**(i-j): (i-j) * gamma**(i-j-1), zero on the diagonal.
        dw = np.where(dist >= 1, dist * np.power(float(gamma), np.where(dist >= 1, dist - 1, 0)), 0.0)
        dw = np.where(lower, dw, 0.0)
        dz = dw.sum(axis=1)
        dA = (dw - A * dz[:, None]) / z[:, None]
        dgamma = float(np.einsum("ij,bid,bjd->", dA, dM, c["S"]))
    else:
        dS, dWm, dgamma, extra = _memory_carry_backward(c, dMcausal, dcarry)

    # Pooling: S_i = sum_t a_t Hloc[t], a = softmax(Hloc @ wp) per block.
    dwp = np.zeros(D)
    for i, (b0, b1) in enumerate(ranges):
        a = c["a"][:, b0:b1]                          # [B, n]
        Hb = Hloc[:, b0:b1]                           # [B, n, D]
        da = np.einsum("bd,btd->bt", dS[:, i], Hb)
        ds = a * (da - np.einsum("bt,bt->b", a, da)[:, None])
        dH[:, b0:b1] += a[:, :, None] * dS[:, i][:, None, :] + ds[:, :, None] * P["wp"]
        dwp += np.einsum("bt,btd->d", ds, Hb)

    # Output projection: Hloc = Hcat @ Wo.
    dWo = np.einsum("btd,bte->de", c["Hcat"], dH)
    dHcat = dH @ P["Wo"].T

    # Block-local causal attention, per block and head.
    dh = D // h
    dQ = np.zeros_like(X)
    dK = np.zeros_like(X)
    dV = np.zeros_like(X)
    for bi, (b0, b1) in enumerate(ranges):
        n = b1 - b0
        Ab = c["probs"][bi]                           # [B, h, n, n]

        def heads(M_):
            return M_[:, b0:b1].reshape(B, n, h, dh).transpose(0, 2, 1, 3)

        q, k, v, do = heads(c["Q"]), heads(c["K"]), heads(c["V"]), heads(dHcat)
        dv = Ab.transpose(0, 1, 3, 2) @ do
        dA_ = do @ v.transpose(0, 1, 3, 2)
        dz_ = Ab * (dA_ - (dA_ * Ab).sum(axis=-1, keepdims=True))
        dq = dz_ @ k / np.sqrt(dh)
        dk = dz_.transpose(0, 1, 3, 2) @ q / np.sqrt(dh)

        def unheads(m):
            return m.transpose(0, 2, 1, 3).reshape(B, n, D)

        dQ[:, b0:b1] = unheads(dq)
        dK[:, b0:b1] = unheads(dk)
        dV[:, b0:b1] = unheads(dv)

    # Q/K/V projections.
    dWq = np.einsum("btd,bte->de", X, dQ)
    dWk = np.einsum("btd,bte->de", X, dK)
    dWv = np.einsum("btd,bte->de", X, dV)
    dX = dQ @ P["Wq"].T + dK @ P["Wk"].T + dV @ P["Wv"].T
    if c["residual"]:
        dX = dX + dY
    return dict(dX=dX, dWq=dWq, dWk=dWk, dWv=dWv, dWo=dWo, dWm=dWm, dWg=dWg,
                dwp=dwp, dgamma=dgamma, **extra)


def _memory_carry_backward(c, dMcausal, dcarry):
    """Chain rule through exp_memory_carry and the projection of a chunk.

    Differentiates the double sums of exp_memory_carry directly, channel by
    channel: with dN_i = dM_i / Z_i (+ dN_out at the last block) and
    dZ_i = -dM_i M_i / Z_i (+ dZ_out at the last block),
      dS_j    = sum_{i>=j} gamma^(i-j) dN_i,
      dN_in   = sum_i gamma^(i+1) dN_i + dM_prev / Z_in,
      dZ_in   = sum_i gamma^(i+1) dZ_i - dM_prev M_prev / Z_in,
      dgamma  = sum_i sum_{j<i} (i-j) gamma^(i-j-1) (dN_i S_j + dZ_i)
              + sum_i (i+1) gamma^i (dN_i N_in + dZ_i Z_in),
    summed over the sequences, where M_prev = N_in / Z_in is the earlier
    blocks' memory (its terms are absent where Z_in = 0).  With a single
    decay (and one normaliser shared by the channels) dgamma and dZ_in are
    the sums of these over the channels.  Returns dS, dWm, dgamma and
    {dN_in, dZ_in}.
    """
    P = c["P"]
    S, Mext, Nacc, Zacc = c["S"], c["Mext"], c["Nacc"], c["Zacc"]
    N_in = c["N_in"]
    B, n, D = S.shape
    g = _per_channel(c["gamma"], D)
    Zc_in = _z_channels(c["Z_in"], D)
    # Mcausal[i] = Mproj[i] with Mproj = Mext @ Wm; Mproj's last row is unused.
    dMproj = np.zeros((B, n + 1, D))
    dMproj[:, :n] = dMcausal
    dWm = np.einsum("bid,bie->de", Mext, dMproj)
    dMext = dMproj @ P["Wm"].T
    dM_prev, dM = dMext[:, 0], dMext[:, 1:]
    M = Mext[:, 1:]

    dN = dM / Zacc
    dZ = -dM * M / Zacc                      # per channel
    if dcarry is not None:
        dN[:, -1] += np.asarray(dcarry[0], dtype=np.float64)
        dZo = np.asarray(dcarry[1], dtype=np.float64)
        if c["per_channel"]:
            dZ[:, -1] += dZo
        else:  # the shared normaliser: its gradient enters once
            dZ[:, -1, 0] += dZo

    dS = np.zeros_like(S)
    dN_in = np.zeros((B, D))
    dZ_in = np.zeros((B, D))
    dgamma = np.zeros(D)
    for i in range(n):
        for j in range(i + 1):
            dS[:, j] += g ** (i - j) * dN[:, i]
            if j < i:
                dgamma += (i - j) * g ** (i - j - 1) * (
                    np.sum(dN[:, i] * S[:, j], axis=0) + np.sum(dZ[:, i], axis=0))
        dN_in += g ** (i + 1) * dN[:, i]
        dZ_in += g ** (i + 1) * dZ[:, i]
        dgamma += (i + 1) * (g ** i if i > 0 else np.ones(D)) * (
            np.sum(dN[:, i] * N_in, axis=0) + np.sum(dZ[:, i] * Zc_in, axis=0))
    has = Zc_in > 0
    safe = np.where(has, Zc_in, 1.0)
    M_prev = carry_memory(N_in, c["Z_in"])
    dN_in += np.where(has, dM_prev / safe, 0.0)
    dZ_in -= np.where(has, dM_prev * M_prev / safe, 0.0)
    if not c["per_channel"]:
        return dS, dWm, float(dgamma.sum()), dict(dN_in=dN_in, dZ_in=dZ_in.sum(axis=1))
    return dS, dWm, dgamma, dict(dN_in=dN_in, dZ_in=dZ_in)


def stack_forward(X, layers, L, h, gamma, residual=True):
    """A stack of layers, X_{l+1} = X_l + layer_l(X_l) when ``residual``."""
    caches = []
    for P in layers:
        X, cache = forward(X, P, L, h, gamma, residual=residual)
        caches.append(cache)
    return X, caches


def stack_backward(caches, dY):
    """Backward through ``stack_forward``; returns dX and per-layer grads.

    dgamma of each layer is reported separately (each layer has its own decay
    input, even when all share one value).
    """
    grads = []
    g = dY
    for cache in reversed(caches):
        gr = backward(cache, g)
        grads.append(gr)
        g = gr["dX"]
    grads.reverse()
    return g, grads
