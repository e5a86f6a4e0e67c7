"""A stack of PQ layers run through the C ABI on one stream (no host syncs).

Used for the AlexNet-shaped forward: conv (ReLU fused in the gather's
epilogue) -> max-pool -> ... -> FC.  Every layer is one library call; the
activations between layers are torch tensors used as device memory only.
"""
from __future__ import annotations

from typing import List, Optional

import numpy as np
import torch

from . import api


class DeviceLayer:
    def __init__(self, spec: dict, device):
        self.kind = spec["kind"]
        if self.kind == "pool":
            self.k, self.s = spec["k"], spec["s"]
            return
        self.D = torch.from_numpy(np.ascontiguousarray(spec["D"])).to(device)
        self.codes = torch.from_numpy(np.ascontiguousarray(spec["codes"])).to(device)
        self.relu = bool(spec["relu"])
        self.bias = None
        if spec.get("bias") is not None:
            self.bias = torch.from_numpy(np.ascontiguousarray(spec["bias"], dtype=np.float32)).to(device)
        if self.kind == "conv":
            self.stride, self.pad = spec["stride"], spec["pad"]

    def __call__(self, h: torch.Tensor) -> torch.Tensor:
        if self.kind == "pool":
            return api.maxpool2d(h, self.k, self.s)
        if self.kind == "conv":
            return api.conv_forward(h, self.D, self.codes, self.stride, self.pad, self.bias, self.relu)
        return api.fc_forward(h.reshape(h.shape[0], -1), self.D, self.codes, self.bias, self.relu)


class Network:
    """Layers from workloads.generate(...)['layers'], resident on ``device``."""

    def __init__(self, layer_specs: List[dict], device="cuda:0"):
        self.layers = [DeviceLayer(s, device) for s in layer_specs]

    def forward(self, x: torch.Tensor, keep: Optional[list] = None) -> torch.Tensor:
        h = x
        for L in self.layers:
            h = L(h)
            if keep is not None:
                keep.append(h)
        return h
