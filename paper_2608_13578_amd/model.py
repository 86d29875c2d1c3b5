"""Device buffers for the language model entry points (bcmt_model_*).

Allocation and argument marshalling only: the forward, backward and AdamW
steps run in the library's kernels.
"""

import numpy as np
import torch

from . import bcmt as abi
from .inputs import model_array_names


class ModelBuffers:
    """Flat float32 master parameters, their bf16 copy, gradients, AdamW
    moments, the loss and the workspace for one model configuration."""

    def __init__(self, V, d, H, n_layer, B, T, L, gamma=0.8, device="cuda", side=True):
        from .layer import SideStream
        self.side = SideStream(device) if side is True else side
        self.cfg = abi.make_model_config(V, d, H, n_layer, B, T, L, gamma)
        self.n = abi.bcmt_model_param_count(self.cfg)
        if self.n == 0:
            raise ValueError("invalid model configuration")
        self.names = model_array_names(n_layer)
        self.layout = [abi.bcmt_model_param_array(self.cfg, i) for i in range(len(self.names))]
        f32 = dict(dtype=torch.float32, device=device)
        self.params = torch.zeros(self.n, **f32)
        self.params_bf16 = torch.zeros(self.n, dtype=torch.bfloat16, device=device)
        self.grads = torch.zeros(self.n, **f32)
        self.m = torch.zeros(self.n, **f32)
        self.v = torch.zeros(self.n, **f32)
        self.loss = torch.zeros(1, **f32)
        self.ws_bytes = abi.bcmt_model_workspace_bytes(self.cfg)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        self.B, self.T, self.V = B, T, V
        self.step_count = 0

    def set_params(self, arrays):
        """Arrays in model_array_names order (E may have fewer rows than the
        padded vocabulary: the rest stay zero)."""
        host = np.zeros(self.n, dtype=np.float32)
        for a, (off, cnt) in zip(arrays, self.layout):
            flat = np.asarray(a, dtype=np.float32).reshape(-1)
            host[off:off + flat.size] = flat
        self.params.copy_(torch.from_numpy(host))
        abi.bcmt_model_cast(self.cfg, self.params, self.params_bf16)

    def arrays(self, flat):
        """Split a flat device vector into host float64 arrays (E cut to V rows)."""
        h = flat.detach().float().cpu().numpy().astype(np.float64)
        d = self.cfg.d
        out = []
        for name, (off, cnt) in zip(self.names, self.layout):
            a = h[off:off + cnt]
            if name == "E":
                a = a.reshape(-1, d)[:self.V]
            out.append(a)
        return out

    def step(self, tokens, targets, opt=None):
        """One training step; opt is a dict of AdamW hyperparameters or None."""
        o = None
        if opt is not None:
            self.step_count += 1
            o = abi.bcmt_adamw(opt["lr"], opt.get("beta1", 0.9), opt.get("beta2", 0.999),
                               opt.get("eps", 1e-8), opt.get("weight_decay", 0.01),
                               self.step_count)
        abi.bcmt_model_train_step(self.cfg, tokens, targets, self.params, self.params_bf16,
                                  self.grads, self.m, self.v, o, self.loss, self.ws, self.ws_bytes,
                                  side=self.side)
