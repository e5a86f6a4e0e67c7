"""Quantizing a stack of layers with error correction, one layer after the
other (Sec. 3.3.3, multi-layer error correction).

Layer l is quantized from the inputs it sees in the network whose layers
1 .. l-1 are already quantized (S), against the responses of the original,
unquantized network (T): the error that earlier layers introduced is then
part of what layer l's error correction minimises.  Per layer: k-means on
the dense weights (Eq. (4) / (6), `qcnn_pq_kmeans`) gives the starting
sub-codebooks and codes, then `sweeps` sweeps of error correction
(`qcnn_ec_fc` / `qcnn_ec_conv`).  The quantized network then advances with
the library's PQ forward (bias and ReLU fused) and max-pool.

The original network belongs to the caller: for every PQ layer it supplies
the desired responses T, the original layer's linear response W * S_orig on
the original network's own inputs (no bias, before the ReLU), as fp32.  Every
step here is a library call; nothing is computed in torch.
"""
from __future__ import annotations

from typing import List, Optional

import torch

from . import api


def quantize_network(x: torch.Tensor, specs: List[dict], targets: List[Optional[torch.Tensor]], sweeps: int = 1,
                     inner: int = 1, kmeans_iters: int = 4, record: Optional[list] = None) -> List[Optional[dict]]:
    """Quantize `specs` layer by layer on the calibration batch x (fp32 NCHW).

    Each spec: {"kind": "conv", "W": [C_t][C_s][d_k][d_k], "bias": [C_t] or
    None, "stride", "pad", "relu", "D0": [M][K][C'_s]} or the same with
    "kind": "fc" and W [C_t][C_s] (no stride or pad), or {"kind": "pool",
    "k", "s"}.  ``targets`` runs parallel to ``specs``: None for a pool, else
    the original layer's linear response T, fp32 [N][C_t][H_o][W_o] (conv) or
    [N][C_t] (FC).  Tensors on one device, fp32.  Returns, per spec, None for a
    pool or {"D", "codes", "objective"} (objective: the error-correction
    history of Eq. (8) / (14)).  If `record` is a list, (S, T) of every PQ
    layer is appended to it.
    """
    if len(targets) != len(specs):
        raise ValueError("targets must run parallel to specs")
    hq = x  # activations of the network quantized so far
    out: List[Optional[dict]] = []
    for spec, T in zip(specs, targets):
        if spec["kind"] == "pool":
            hq = api.maxpool2d(hq, spec["k"], spec["s"])
            out.append(None)
            continue
        if T is None or T.dtype != torch.float32 or not T.is_contiguous():
            raise ValueError("each PQ layer needs its target responses as a contiguous fp32 tensor")
        W = spec["W"]
        D, codes, _ = api.pq_kmeans(W, spec["D0"], kmeans_iters)
        if spec["kind"] == "conv":
            S = hq
            obj = api.ec_conv(S, T, D, codes, spec["stride"], spec["pad"], sweeps, inner)
            hq = api.conv_forward(hq, D, codes, spec["stride"], spec["pad"], spec.get("bias"), spec["relu"])
        else:
            S = hq.reshape(hq.shape[0], -1).contiguous()
            obj = api.ec_fc(S, T, D, codes, sweeps, inner)
            hq = api.fc_forward(S, D, codes, spec.get("bias"), spec["relu"])
        if record is not None:
            record.append((S, T))
        out.append({"D": D, "codes": codes, "objective": obj})
    return out
