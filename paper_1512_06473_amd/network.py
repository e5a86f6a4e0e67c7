"""A stack of PQ layers run through the C ABI on one stream (no host syncs).

Used for the AlexNet-shaped forward: conv (ReLU fused in the gather's
epilogue) -> max-pool -> ... -> FC.  A conv layer followed by a max-pool is
one library call (qcnn_conv_pool_forward: the pooling is taken where the
conv's split partial sums are added); every other layer is one call of its
own.  With ``use_plans`` (the default) each conv and FC layer is prepared
once per input shape (qcnn_conv_plan_create / qcnn_fc_plan_create: codes
re-laid for the kernel, codebooks and bias copied) and each forward is a
qcnn_plan_forward; the results are the per-call entry points' bit for bit.
The activations between calls are torch tensors used as device memory only.
"""
from __future__ import annotations

from typing import List, Optional

import numpy as np
import torch

from . import api


class DeviceLayer:
    """One library call: a conv, FC or pool layer, or a conv and the max-pool
    after it.  ``specs`` holds the layer specs it covers (one or two)."""

    def __init__(self, spec: dict, device, pool: Optional[dict] = None, use_plans: bool = True):
        self.kind = spec["kind"]
        self.use_plans = use_plans
        self._plans = {}
        self.specs = [spec] if pool is None else [spec, pool]
        self.pool = None if pool is None else (pool["k"], pool["s"])
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

    @property
    def name(self) -> str:
        return "+".join(s["kind"] for s in self.specs)

    def _plan(self, shape):
        plan = self._plans.get(shape)
        if plan is None:
            if self.kind == "conv":
                plan = api.ConvPlan(shape, self.D, self.codes, self.stride, self.pad, self.bias, self.relu, self.pool)
            else:
                plan = api.FcPlan(shape[0], self.D, self.codes, self.bias, self.relu)
            self._plans[shape] = plan
        return plan

    def __call__(self, h: torch.Tensor) -> torch.Tensor:
        if self.kind == "pool":
            return api.maxpool2d(h, self.k, self.s)
        if self.kind == "fc" and h.dim() != 2:
            h = h.reshape(h.shape[0], -1)
        if self.use_plans:
            return self._plan(tuple(h.shape))(h)
        if self.kind == "conv":
            if self.pool is not None:
                return api.conv_pool_forward(h, self.D, self.codes, self.stride, self.pad, self.pool[0],
                                             self.pool[1], self.bias, self.relu)
            return api.conv_forward(h, self.D, self.codes, self.stride, self.pad, self.bias, self.relu)
        return api.fc_forward(h, self.D, self.codes, self.bias, self.relu)


class Network:
    """Layers from workloads.generate(...)['layers'], resident on ``device``.
    ``fuse_pools``: a conv followed by a max-pool becomes one call;
    ``use_plans``: conv and FC layers run through prepared plans."""

    def __init__(self, layer_specs: List[dict], device="cuda:0", fuse_pools: bool = True, use_plans: bool = True):
        self.layers = []
        i = 0
        while i < len(layer_specs):
            s = layer_specs[i]
            nxt = layer_specs[i + 1] if i + 1 < len(layer_specs) else None
            if fuse_pools and s["kind"] == "conv" and nxt is not None and nxt["kind"] == "pool":
                self.layers.append(DeviceLayer(s, device, pool=nxt, use_plans=use_plans))
                i += 2
            else:
                self.layers.append(DeviceLayer(s, device, use_plans=use_plans))
                i += 1

    def forward(self, x: torch.Tensor, keep: Optional[list] = None) -> torch.Tensor:
        h = x
        for L in self.layers:
            h = L(h)
            if keep is not None:
                keep.append(h)
        return h
