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

The original network is the caller's dense weights; its responses T =
W * S_orig are the desired outputs the method is given, computed here in
float64 (torch unfold + matmul on the device) and rounded to fp32; the
original network's activations are kept in fp32.  Only the quantized path
and the error correction are library calls.
"""
from __future__ import annotations

from typing import List, Optional

import torch
import torch.nn.functional as F

from . import api


def dense_response(h: torch.Tensor, spec: dict) -> torch.Tensor:
    """The original layer's linear response W * h in float64 (no bias)."""
    W = spec["W"].double()
    if spec["kind"] == "fc":
        return h.reshape(h.shape[0], -1).double() @ W.t().contiguous()
    Ct, Cs, dk, _ = W.shape
    N, _, H, Wd = h.shape
    Ho = api.out_size(H, dk, spec["stride"], spec["pad"])
    Wo = api.out_size(Wd, dk, spec["stride"], spec["pad"])
    cols = F.unfold(h.double(), dk, padding=spec["pad"], stride=spec["stride"])  # [N][Cs dk dk][Ho Wo]
    y = torch.matmul(W.reshape(Ct, -1), cols)
    return y.reshape(N, Ct, Ho, Wo)


def quantize_network(x: torch.Tensor, specs: List[dict], sweeps: int = 1, inner: int = 1, kmeans_iters: int = 4,
                     record: Optional[list] = None) -> List[Optional[dict]]:
    """Quantize `specs` layer by layer on the calibration batch x (fp32 NCHW).

    Each spec: {"kind": "conv", "W": [C_t][C_s][d_k][d_k], "bias": [C_t] or
    None, "stride", "pad", "relu", "D0": [M][K][C'_s]} or the same with
    "kind": "fc" and W [C_t][C_s] (no stride or pad), or {"kind": "pool",
    "k", "s"}.  Tensors on one device, fp32.  Returns, per spec, None for a
    pool or {"D", "codes", "objective"} (objective: the error-correction
    history of Eq. (8) / (14)).  If `record` is a list, (S, T) of every PQ
    layer is appended to it.
    """
    hq = x  # activations of the network quantized so far
    ho = x  # activations of the original network
    out: List[Optional[dict]] = []
    for spec in specs:
        if spec["kind"] == "pool":
            hq = api.maxpool2d(hq, spec["k"], spec["s"])
            ho = api.maxpool2d(ho, spec["k"], spec["s"])
            out.append(None)
            continue
        lin = dense_response(ho, spec)
        T = lin.float().contiguous()
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
        bias = spec.get("bias")
        if bias is not None:
            lin = lin + (bias.double()[None, :, None, None] if spec["kind"] == "conv" else bias.double()[None, :])
        if spec["relu"]:
            lin = torch.clamp_min(lin, 0.0)
        ho = lin.float().contiguous()
        out.append({"D": D, "codes": codes, "objective": obj})
    return out
