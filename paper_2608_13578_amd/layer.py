"""Device buffers around one BCMT layer, for callers that hold torch tensors.

Allocates the `saved` activations and the two workspaces through torch's
allocator (plumbing only) and forwards to the C ABI in ``bcmt``.  The layer's
arithmetic runs entirely in the library's HIP kernels.
"""

import sys

import numpy as np
import torch

from . import bcmt as abi

TORCH_DTYPE = {"bf16": torch.bfloat16, "f32": torch.float32}


def to_device(arr, dtype, device="cuda"):
    """numpy float32 values -> device tensor of the compute type (exact when
    the values are already representable, as the seeded inputs are)."""
    t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(device)
    return t.to(TORCH_DTYPE[dtype]).contiguous()


def to_host64(t):
    """Device tensor -> float64 numpy array."""
    return t.detach().float().cpu().numpy().astype(np.float64)


class SideStream:
    """A caller-owned second stream (default priority) and the two events the
    backward passes use to fork work onto it and join it back (bcmt_side).
    The events come from bcmt_side_events_create: no timing and no
    system-scope fence on record, since they only order two streams of the
    device."""

    def __init__(self, device="cuda"):
        self.stream = torch.cuda.Stream(device=device)
        self._ev = abi.bcmt_side()
        with torch.cuda.device(self.stream.device):
            abi.bcmt_side_events_create(self._ev)
        self.fork, self.join = self._ev.fork, self._ev.join

    def __del__(self):
        ev = getattr(self, "_ev", None)
        if sys.is_finalizing():
            return  # the process is ending: the events go with it
        if ev is not None and (ev.fork or ev.join):
            try:
                torch.cuda.synchronize(self.stream.device)
                abi.bcmt_side_events_destroy(ev)
            except Exception:
                pass


class LayerBuffers:
    """Holds a config, device weights and the scratch buffers of one layer."""

    def __init__(self, B, T, D, H, L, gamma=0.8, dtype="bf16", residual=False,
                 accumulate=False, device="cuda", side=True):
        """gamma: the decay, or one decay per channel ([D] array: sets
        BCMT_FLAG_CHANNEL_DECAY; its values go to the device as gamma_ch).
        side: run the backward's weight-gradient products on a second stream
        (True: one made here; a SideStream; or None for one stream)."""
        self.dtype = dtype
        self.side = SideStream(device) if side is True else side
        self.device = device
        self.gamma_ch = None
        if np.ndim(gamma) > 0:
            self.gamma_ch = torch.tensor(np.asarray(gamma, dtype=np.float32), device=device)
            gamma = 0.0
        self.cfg = abi.make_config(B, T, D, H, L, gamma, dtype, residual, accumulate,
                                   channel_decay=self.gamma_ch is not None)
        st = abi.bcmt_validate(self.cfg)
        if st != abi.BCMT_OK:
            raise abi.BcmtError(st, "bcmt_validate")
        self.shape = (B, T, D)
        u8 = dict(dtype=torch.uint8, device=device)
        self.saved = torch.empty(abi.bcmt_saved_bytes(self.cfg), **u8)
        self.ws_fwd = torch.empty(max(256, abi.bcmt_workspace_bytes(self.cfg, abi.BCMT_PASS_FORWARD)), **u8)
        self.ws_bwd = torch.empty(max(256, abi.bcmt_workspace_bytes(self.cfg, abi.BCMT_PASS_BACKWARD)), **u8)
        self.params = None

    def set_params(self, weights):
        """weights: dict of numpy float32 arrays (input-major [D, D], wp [D])."""
        self.params = {k: to_device(weights[k], self.dtype, self.device) for k in abi.PARAM_NAMES}
        if self.gamma_ch is not None:
            self.params["gamma_ch"] = self.gamma_ch
        return self.params

    def new_activation(self):
        return torch.empty(self.shape, dtype=TORCH_DTYPE[self.dtype], device=self.device)

    def new_grads(self):
        D = self.shape[2]
        f = dict(dtype=torch.float32, device=self.device)
        g = {n: torch.zeros((D, D), **f) for n in ("dWq", "dWk", "dWv", "dWo", "dWm", "dWg")}
        g["dwp"] = torch.zeros((D,), **f)
        g["dgamma"] = torch.zeros((4,), **f)  # 16 bytes, value in element 0
        if self.gamma_ch is not None:
            g["dgamma_ch"] = torch.zeros((D,), **f)
        return g

    def forward(self, X, Y, stream=None):
        abi.bcmt_layer_forward(self.cfg, X, self.params, Y, self.saved, self.ws_fwd, stream=stream)

    def backward(self, X, dY, dX, grads, stream=None):
        abi.bcmt_layer_backward(self.cfg, X, self.params, self.saved, dY, dX, grads, self.ws_bwd,
                                stream=stream, side=self.side)

    def new_carry(self):
        """A zeroed memory state (N [B, D], Z [B] or [B, D] with a per-channel
        decay, float32): an empty history."""
        B, _, D = self.shape
        f = dict(dtype=torch.float32, device=self.device)
        zshape = (B, D) if self.gamma_ch is not None else (B,)
        return torch.zeros((B, D), **f), torch.zeros(zshape, **f)

    def forward_chunk(self, X, Y, carry_in, carry_out, stream=None):
        abi.bcmt_layer_forward_chunk(self.cfg, X, self.params, carry_in, Y, carry_out, self.saved,
                                     self.ws_fwd, stream=stream)

    def backward_chunk(self, X, dY, dcarry_out, dX, dcarry_in, grads, stream=None):
        abi.bcmt_layer_backward_chunk(self.cfg, X, self.params, self.saved, dY, dcarry_out, dX,
                                      dcarry_in, grads, self.ws_bwd, stream=stream,
                                      side=self.side)


class DecodeBuffers:
    """Decode state and workspace for B sequences decoded in step."""

    def __init__(self, B, D, H, L, gamma=0.8, dtype="bf16", residual=False, device="cuda"):
        self.dtype = dtype
        self.device = device
        self.gamma_ch = None
        if np.ndim(gamma) > 0:
            self.gamma_ch = torch.tensor(np.asarray(gamma, dtype=np.float32), device=device)
            gamma = 0.0
        self.cfg = abi.make_config(B, 1, D, H, L, gamma, dtype, residual,
                                   channel_decay=self.gamma_ch is not None)
        u8 = dict(dtype=torch.uint8, device=device)
        n = abi.bcmt_decode_state_bytes(self.cfg)
        if n == 0:
            raise abi.BcmtError(abi.BCMT_ERR_UNSUPPORTED, "bcmt_decode_state_bytes")
        self.state = torch.empty(n, **u8)
        self.ws = torch.empty(max(256, abi.bcmt_decode_workspace_bytes(self.cfg)), **u8)
        self.shape = (B, D)
        self.params = None

    def set_params(self, weights):
        self.params = {k: to_device(weights[k], self.dtype, self.device) for k in abi.PARAM_NAMES}
        if self.gamma_ch is not None:
            self.params["gamma_ch"] = self.gamma_ch
        return self.params

    def reset(self, carry_in=None, stream=None):
        abi.bcmt_decode_reset(self.cfg, self.params, carry_in, self.state, self.ws, stream=stream)

    def step(self, t, x, y, stream=None):
        abi.bcmt_decode_step(self.cfg, self.params, t, x, y, self.state, self.ws, stream=stream)
