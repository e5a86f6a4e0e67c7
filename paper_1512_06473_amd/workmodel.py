"""Work and traffic model of the product-quantized layer forward.

Table 1 of the paper (Sec. 3.4) gives the test-phase cost of a conv and an FC
layer, dense vs quantized, in FLOPs (the paper counts one multiply-add as one
FLOP, e.g. 7.29e8 for AlexNet in Table 3) and in bytes of stored parameters:

  conv  FLOPs  dense  d_t^2 C_t d_k^2 C_s          Q-CNN  d_s^2 C_s K + d_t^2 C_t d_k^2 M
  FC    FLOPs  dense  C_s C_t                      Q-CNN  C_s K + C_t M
  conv  bytes  dense  4 d_k^2 C_s C_t              Q-CNN  4 C_s K + d_k^2 M C_t log2(K) / 8
  FC    bytes  dense  4 C_s C_t                    Q-CNN  4 C_s K + M C_t log2(K) / 8

The same counts, restricted to the receptive-field pairs that fall inside the
input (zero padding contributes nothing), give the algorithmic work of the
MI355X kernels:

* table entries  N d_s^2 M K, each a C'_s-term inner product;
* gathers        one per valid (image, c_t, p_t, p_k, m) -- one table read and
                 one fp32 add each;
* LDS bytes      4 per gather read + 4 per table entry written;
* HBM bytes      input + output + codes + codebooks, each moved once.

Grouped convolutions (the original AlexNet's conv2, conv4, conv5) are modelled
as ``groups`` independent layers, which Table 4's figures require.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional

# MI355X figures used for roofline fractions.
N_CU = 256
CLOCK_HZ = 2.4e9
HBM_PEAK_BPS = 8.0e12                  # HBM3E, published
LDS_READ_BYTES_PER_CLK_PER_CU = 256    # gfx950 LDS read port (128-bit reads)
LDS_PEAK_BPS = N_CU * CLOCK_HZ * LDS_READ_BYTES_PER_CLK_PER_CU   # 157.3e12
VALU_LANE_OPS_PER_CLK_PER_CU = 64      # 4 SIMD x 16 lanes, unpacked fp32
VALU_PEAK_OPS = N_CU * CLOCK_HZ * VALU_LANE_OPS_PER_CLK_PER_CU   # 39.3e12 adds/s


def out_size(n: int, k: int, s: int, p: int) -> int:
    span = n + 2 * p - k
    return span // s + 1 if span >= 0 else 0


# --------------------------------------------------------------------------
# Table 1, per layer (per image), paper convention: 1 FLOP = 1 multiply-add.

def conv_flops_dense(ds_t: int, Ct: int, dk: int, Cs: int, groups: int = 1) -> int:
    return groups * ds_t * ds_t * (Ct // groups) * dk * dk * (Cs // groups)


def conv_flops_qcnn(ds_s: int, ds_t: int, Cs: int, Ct: int, dk: int, Csp: int, K: int,
                    groups: int = 1) -> int:
    cs, ct = Cs // groups, Ct // groups
    M = cs // Csp
    return groups * (ds_s * ds_s * cs * K + ds_t * ds_t * ct * dk * dk * M)


def fc_flops_dense(Cs: int, Ct: int) -> int:
    return Cs * Ct


def fc_flops_qcnn(Cs: int, Ct: int, Csp: int, K: int) -> int:
    return Cs * K + Ct * (Cs // Csp)


def conv_bytes_dense(Cs: int, Ct: int, dk: int, groups: int = 1) -> float:
    return 4.0 * dk * dk * (Cs // groups) * Ct


def conv_bytes_qcnn(Cs: int, Ct: int, dk: int, Csp: int, K: int, groups: int = 1) -> float:
    cs, ct = Cs // groups, Ct // groups
    M = cs // Csp
    return groups * (4.0 * cs * K + dk * dk * M * ct * math.log2(K) / 8.0)


def fc_bytes_dense(Cs: int, Ct: int) -> float:
    return 4.0 * Cs * Ct


def fc_bytes_qcnn(Cs: int, Ct: int, Csp: int, K: int) -> float:
    return 4.0 * Cs * K + (Cs // Csp) * Ct * math.log2(K) / 8.0


# --------------------------------------------------------------------------
# Algorithmic work of one launch on the MI355X path.

@dataclass
class LayerWork:
    dense_macs: int        # multiply-adds of the equivalent dense layer (valid taps)
    lut_entries: int       # N d_s^2 M K
    gathers: int           # valid (n, c_t, p_t, p_k, m) tuples
    hbm_bytes: int         # x + y + codes + codebooks (+ bias)
    lds_bytes: int         # 4 * (gathers + lut_entries)

    @property
    def dense_flops(self) -> int:
        return 2 * self.dense_macs


def _valid_taps_1d(n_in: int, n_out: int, k: int, s: int, p: int) -> int:
    """Number of (output index, kernel index) pairs whose input index is inside."""
    c = 0
    for o in range(n_out):
        for kk in range(k):
            i = o * s - p + kk
            if 0 <= i < n_in:
                c += 1
    return c


def conv_work(N: int, Cs: int, H: int, W: int, Ct: int, dk: int, stride: int, pad: int,
              Csp: int, K: int, bias: bool = False) -> LayerWork:
    M = Cs // Csp
    Ho, Wo = out_size(H, dk, stride, pad), out_size(W, dk, stride, pad)
    taps = _valid_taps_1d(H, Ho, dk, stride, pad) * _valid_taps_1d(W, Wo, dk, stride, pad)
    gathers = N * Ct * taps * M
    lut = N * H * W * M * K
    hbm = 4 * N * Cs * H * W + 4 * N * Ct * Ho * Wo + Ct * dk * dk * M + 4 * M * K * Csp
    if bias:
        hbm += 4 * Ct
    return LayerWork(dense_macs=N * Ct * taps * Cs, lut_entries=lut, gathers=gathers,
                     hbm_bytes=hbm, lds_bytes=4 * (gathers + lut))


def fc_work(N: int, Cs: int, Ct: int, Csp: int, K: int, bias: bool = False) -> LayerWork:
    M = Cs // Csp
    gathers = N * Ct * M
    lut = N * M * K
    hbm = 4 * N * Cs + 4 * N * Ct + Ct * M + 4 * M * K * Csp
    if bias:
        hbm += 4 * Ct
    return LayerWork(dense_macs=N * Ct * Cs, lut_entries=lut, gathers=gathers,
                     hbm_bytes=hbm, lds_bytes=4 * (gathers + lut))


def lut_build_work(N: int, Cs: int, H: int, W: int, Csp: int, K: int) -> LayerWork:
    """qcnn_lut_build: reads x and the codebooks, writes the whole table."""
    M = Cs // Csp
    lut = N * H * W * M * K
    return LayerWork(dense_macs=lut * Csp, lut_entries=lut, gathers=0,
                     hbm_bytes=4 * N * Cs * H * W + 4 * M * K * Csp + 4 * lut,
                     lds_bytes=0)


def maxpool_work(N: int, C: int, H: int, W: int, k: int, s: int) -> LayerWork:
    Ho, Wo = out_size(H, k, s, 0), out_size(W, k, s, 0)
    return LayerWork(dense_macs=0, lut_entries=0, gathers=0,
                     hbm_bytes=4 * N * C * (H * W + Ho * Wo), lds_bytes=0)


def workload_work(wl, N: Optional[int] = None):
    """Per-layer LayerWork list for a workloads.Workload (pool layers included)."""
    from .workloads import Conv, FC, Pool  # shapes only
    n = wl.N if N is None else N
    shape = tuple(wl.in_shape)
    out = []
    for L in wl.layers:
        if isinstance(L, Pool):
            C, H, W = shape
            out.append(("pool", maxpool_work(n, C, H, W, L.k, L.s)))
            shape = (C, out_size(H, L.k, L.s, 0), out_size(W, L.k, L.s, 0))
        elif isinstance(L, Conv):
            C, H, W = shape
            out.append(("conv", conv_work(n, C, H, W, L.Ct, L.dk, L.stride, L.pad, L.Csp, L.K)))
            shape = (L.Ct, out_size(H, L.dk, L.stride, L.pad), out_size(W, L.dk, L.stride, L.pad))
        else:
            Cs = int(math.prod(shape))
            out.append(("fc", fc_work(n, Cs, L.Ct, L.Csp, L.K)))
            shape = (L.Ct,)
    return out


def call_work(wl, N: Optional[int] = None, fuse_pools: bool = True):
    """Per-library-call (name, LayerWork) list for a workloads.Workload, as
    network.Network issues them: with ``fuse_pools`` a conv followed by a
    max-pool is one call ("conv+pool"), whose HBM bytes are the conv's
    without its full output map and with the pooled map instead."""
    from .workloads import Conv, Pool  # shapes only
    n = wl.N if N is None else N
    layers = list(wl.layers)
    per = workload_work(wl, N)
    shape = tuple(wl.in_shape)
    out = []
    i = 0
    while i < len(layers):
        L = layers[i]
        kind, lw = per[i]
        if isinstance(L, Conv):
            C, H, W = shape
            shape = (L.Ct, out_size(H, L.dk, L.stride, L.pad), out_size(W, L.dk, L.stride, L.pad))
            nxt = layers[i + 1] if i + 1 < len(layers) else None
            if fuse_pools and isinstance(nxt, Pool):
                Ct, Ho, Wo = shape
                Hp, Wp = out_size(Ho, nxt.k, nxt.s, 0), out_size(Wo, nxt.k, nxt.s, 0)
                hbm = lw.hbm_bytes - 4 * n * Ct * Ho * Wo + 4 * n * Ct * Hp * Wp
                out.append(("conv+pool", LayerWork(dense_macs=lw.dense_macs, lut_entries=lw.lut_entries,
                                                   gathers=lw.gathers, hbm_bytes=hbm, lds_bytes=lw.lds_bytes)))
                shape = (Ct, Hp, Wp)
                i += 2
                continue
        elif isinstance(L, Pool):
            C, H, W = shape
            shape = (C, out_size(H, L.k, L.s, 0), out_size(W, L.k, L.s, 0))
        else:
            shape = (L.Ct,)
        out.append((kind, lw))
        i += 1
    return out
