"""The allocation-free forward entry point (bcmt_layer_forward_noalloc).

It runs the forward pass with its workspace in the library's own device
array instead of a caller buffer.  Its output must equal that of
bcmt_layer_forward on the same inputs bit for bit (same kernels, no
atomics), and the activations it saves must give the same backward pass.
Three calls in a row on one GPU, each with a smaller input than the one
before, check that a call does not depend on what the previous call left in
the array.
"""

import numpy as np
import pytest

from test_gpu_parity import GRADS, inputs, say, torch_cuda  # noqa: F401

pytestmark = pytest.mark.gpu

CALLS = [
    # B, T, D, H, L, dtype: the measured layer; then 160 blocks of 16 tokens
    # (the memory path whose W_m product keeps split-K partials in the
    # scratch); then a small float32 layer with a ragged last block
    (8, 1024, 768, 12, 128, "bf16"),
    (2, 2560, 512, 8, 16, "bf16"),
    (1, 300, 256, 4, 64, "f32"),
]


def test_noalloc_forward_matches_forward(torch_cuda):
    torch = torch_cuda
    from paper_2608_13578_amd import bcmt as abi
    from paper_2608_13578_amd.layer import LayerBuffers, to_device
    for (B, T, D, H, L, dt) in CALLS:
        say(f"noalloc forward: B={B} T={T} D={D} H={H} L={L} {dt}")
        cfg_ws = abi.bcmt_workspace_bytes(abi.make_config(B, T, D, H, L, 0.8, dt),
                                          abi.BCMT_PASS_FORWARD)
        assert 0 < cfg_ws <= abi.BCMT_NOALLOC_SCRATCH_BYTES
        X, W, dY = inputs(B, T, D, dt)
        lb = LayerBuffers(B, T, D, H, L, dtype=dt)
        lb.set_params(W)
        Xd, dYd = to_device(X, dt), to_device(dY, dt)
        # the existing entry point, with its own workspace
        Y1 = lb.new_activation()
        lb.forward(Xd, Y1)
        g1 = lb.new_grads()
        lb.backward(Xd, dYd, None, g1)
        # the allocation-free one, into a separate saved buffer
        Y2 = lb.new_activation()
        saved2 = torch.empty_like(lb.saved)
        abi.bcmt_layer_forward_noalloc(lb.cfg, Xd, lb.params, Y2, saved2)
        lb.saved = saved2
        g2 = lb.new_grads()
        lb.backward(Xd, dYd, None, g2)
        torch.cuda.synchronize()
        assert torch.equal(Y1, Y2), "outputs differ"
        for k in GRADS:
            assert torch.equal(g1[k], g2[k]), k
        # the decay gradient too is reduced in a fixed order
        assert torch.equal(g1["dgamma"], g2["dgamma"]), "dgamma"
