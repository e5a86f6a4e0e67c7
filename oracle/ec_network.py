"""Multi-layer error correction -- TEST INFRASTRUCTURE ONLY (imported by
tests/ and nothing in the product package).

Paper: Wu et al., CVPR 2016, Sec. 3.3.3.  The layers are quantized one after
another; layer l is quantized with, as inputs S, the layer's inputs in the
network whose earlier layers are already quantized, and, as desired
responses T, the layer's responses in the original network.  Per layer: the
k-means quantizer (Eq. (4) / (6); the C oracle's `pq_kmeans`) starts it, then
error correction (Eq. (8)-(12), `oracle.ec`; Eq. (13)-(21), `oracle.ec_conv`).

Readings (M1-M3 in the design notes):
  M1 T is the original layer's linear response W * S_orig (no bias, before
     the ReLU): the quantized layer keeps the original bias, so matching the
     linear part is what Eq. (8) / (14) asks;
  M2 activations are kept in fp32 on both networks: T and the original
     network's activations are float64 sums rounded to fp32; the quantized
     network's activations are its PQ forward (Eq. (5) / (7)) with the
     learned sub-codebooks rounded to fp32, bias and ReLU, rounded to fp32;
  M3 max-pool layers pass both networks' activations through unchanged in
     kind (no parameters).
"""
from __future__ import annotations

import numpy as np

from oracle import ec, ec_conv
from oracle import oracle as O


def dense_linear(h, spec):
    """W * h in float64 (no bias): FC over flattened inputs, conv as a
    cross-correlation with stride and zero padding (one offset at a time)."""
    W = np.asarray(spec["W"], np.float64)
    h = np.asarray(h, np.float64)
    if spec["kind"] == "fc":
        return h.reshape(h.shape[0], -1) @ W.T
    Ct, Cs, dk, _ = W.shape
    N, _, H, Wd = h.shape
    s, p = spec["stride"], spec["pad"]
    Ho, Wo = (H + 2 * p - dk) // s + 1, (Wd + 2 * p - dk) // s + 1
    hp = np.zeros((N, Cs, H + 2 * p, Wd + 2 * p))
    hp[:, :, p:p + H, p:p + Wd] = h
    y = np.zeros((N, Ct, Ho, Wo))
    for ky in range(dk):
        for kx in range(dk):
            win = hp[:, :, ky:ky + s * (Ho - 1) + 1:s, kx:kx + s * (Wo - 1) + 1:s]
            y += np.einsum("tc,nchw->nthw", W[:, :, ky, kx], win)
    return y


def original_responses(x, specs):
    """The desired responses T of every PQ layer (None for a pool): the
    original network run on x, T = W * S_orig in float64 rounded to fp32
    (M1, M2); the next layer sees bias + ReLU of the float64 response,
    rounded to fp32, or the pool of the fp32 activations (M3)."""
    ho = np.asarray(x, np.float32)
    out = []
    for spec in specs:
        if spec["kind"] == "pool":
            ho = O.maxpool(ho, spec["k"], spec["s"]).astype(np.float32)
            out.append(None)
            continue
        lin = dense_linear(ho, spec)                              # M1
        out.append(lin.astype(np.float32))
        bias = spec.get("bias")
        if bias is not None:
            b = np.asarray(bias, np.float64)
            lin = lin + (b[None, :, None, None] if spec["kind"] == "conv" else b[None, :])
        if spec["relu"]:
            lin = np.maximum(lin, 0.0)
        ho = lin.astype(np.float32)
    return out


def quantize_network(x, specs, sweeps=1, inner=1, kmeans_iters=4):
    """Returns, per spec, None for a pool or (D float64, codes, objective
    history, S, T) for a PQ layer."""
    hq = np.asarray(x, np.float32)
    out = []
    for spec, T in zip(specs, original_responses(x, specs)):
        if spec["kind"] == "pool":
            hq = O.maxpool(hq, spec["k"], spec["s"]).astype(np.float32)
            out.append(None)
            continue
        W = np.asarray(spec["W"], np.float32)
        D, codes, _ = O.pq_kmeans(W, np.asarray(spec["D0"], np.float32), kmeans_iters)
        bias = spec.get("bias")
        if spec["kind"] == "conv":
            S = hq
            D, codes, hist = ec_conv.ec_conv(S, T, D, codes, spec["stride"], spec["pad"], sweeps, inner)
            D32 = D.astype(np.float32)                            # M2
            hq = O.conv_lut(hq, D32, codes, spec["stride"], spec["pad"], bias=bias,
                            relu=spec["relu"]).astype(np.float32)
        else:
            S = hq.reshape(hq.shape[0], -1)
            D, codes, hist = ec.ec_fc(S, T, D, codes, sweeps, inner)
            D32 = D.astype(np.float32)
            hq = O.fc_lut(S, D32, codes, bias=bias, relu=spec["relu"]).astype(np.float32)
        out.append((D, codes, hist, S, T))
    return out
