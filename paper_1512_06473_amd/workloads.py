"""Seeded synthetic workloads for the product-quantized layer forward.

This module only draws random inputs of the right shapes; it holds none of the
method's arithmetic.  Both the HIP path (tests, benchmark) and the CPU oracle
receive exactly the bytes it produces.

Stand-in for the paper's data: the paper evaluates on ILSVRC-12 activations
with trained AlexNet / VGG-16 weights (Sec. 5.2), neither of which is
available here.  Inputs are therefore synthetic with the layer shapes of those
networks:

* activations x = |N(0, 1)| (half-normal, non-negative like post-ReLU maps),
  drawn in float64 and cast to fp32;
* sub-codebooks D[m][k][j] = sigma * N(0, 1) cast to fp32, shape [M][K][C'_s];
* codes uniform in [0, K) as uint8, conv [C_t][d_k][d_k][M], FC [C_t][M].

Generator: numpy ``Generator(PCG64(seed))``; draw order x, then for each PQ
layer in network order its D then its codes.  Each workload has a
seed of its own (1 to 5, in the order of the table below).

``integer=True`` gives the exact-arithmetic variant used for bit-exact index
checks: x in {0..7}, D in {-8..8} (integers as fp32), so every partial sum of
every layer stays far below 2**24 and fp32 sums are exact in any order.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple, Union

import numpy as np


@dataclass(frozen=True)
class Conv:
    Cs: int
    Ct: int
    dk: int
    stride: int
    pad: int
    Csp: int
    K: int
    relu: bool = False
    sigma: float = 0.05

    @property
    def M(self) -> int:
        return self.Cs // self.Csp


@dataclass(frozen=True)
class FC:
    Cs: int
    Ct: int
    Csp: int
    K: int
    relu: bool = False
    sigma: float = 0.01

    @property
    def M(self) -> int:
        return self.Cs // self.Csp


@dataclass(frozen=True)
class Pool:
    k: int = 3
    s: int = 2


Layer = Union[Conv, FC, Pool]


@dataclass(frozen=True)
class Workload:
    name: str
    title: str
    N: int
    in_shape: Tuple[int, ...]
    layers: Tuple[Layer, ...]
    seed: int


def _alexnet_layers() -> Tuple[Layer, ...]:
    # AlexNet-shaped stack without groups or LRN: conv1 at C'_s=3, K=64 (M=1),
    # conv2..conv5 at C'_s=4, K=128, FC at C'_s=4, K=32, ReLU everywhere but fc8.
    return (
        Conv(3, 96, 11, 4, 0, 3, 64, True, 0.05),
        Pool(3, 2),
        Conv(96, 256, 5, 1, 2, 4, 128, True, 0.05),
        Pool(3, 2),
        Conv(256, 384, 3, 1, 1, 4, 128, True, 0.05),
        Conv(384, 384, 3, 1, 1, 4, 128, True, 0.05),
        Conv(384, 256, 3, 1, 1, 4, 128, True, 0.05),
        Pool(3, 2),
        FC(9216, 4096, 4, 32, True, 0.01),
        FC(4096, 4096, 4, 32, True, 0.01),
        FC(4096, 1000, 4, 32, False, 0.01),
    )


WORKLOADS = {
    "small_conv_n1": Workload("small_conv_n1", "single PQ conv 1x16x14x14 -> 32, 3x3 s1 p1, C's=4, K=16",
                     1, (16, 14, 14), (Conv(16, 32, 3, 1, 1, 4, 16, False, 0.1),), 1),
    "alexnet_conv3_n32": Workload("alexnet_conv3_n32", "AlexNet-conv3-shaped PQ conv 32x256x13x13 -> 384, 3x3 p1, C's=4, K=128",
                     32, (256, 13, 13), (Conv(256, 384, 3, 1, 1, 4, 128, False, 0.05),), 2),
    "alexnet_fc6_n128": Workload("alexnet_fc6_n128", "fc6-shaped PQ FC 128x9216 -> 4096, C's=4, K=32",
                     128, (9216,), (FC(9216, 4096, 4, 32, False, 0.01),), 3),
    "vgg16_conv3_n16": Workload("vgg16_conv3_n16", "VGG-16-conv3-shaped PQ conv 16x256x56x56 -> 256, 3x3 p1, C's=8, K=128",
                     16, (256, 56, 56), (Conv(256, 256, 3, 1, 1, 8, 128, False, 0.05),), 4),
    "alexnet_n64": Workload("alexnet_n64", "AlexNet-shaped PQ forward, batch 64, 227x227, 5 conv + 3 pool + 3 FC",
                     64, (3, 227, 227), _alexnet_layers(), 5),
}


def layer_dict(L: Layer, D: Optional[np.ndarray] = None, codes: Optional[np.ndarray] = None) -> dict:
    if isinstance(L, Pool):
        return {"kind": "pool", "k": L.k, "s": L.s}
    if isinstance(L, Conv):
        return {"kind": "conv", "D": D, "codes": codes, "stride": L.stride, "pad": L.pad,
                "relu": L.relu, "spec": L}
    return {"kind": "fc", "D": D, "codes": codes, "relu": L.relu, "spec": L}


def draw_layer(rng: np.random.Generator, L: Layer, integer: bool = False):
    """Sub-codebooks then codes of one PQ layer."""
    M = L.M
    if integer:
        D = rng.integers(-8, 9, size=(M, L.K, L.Csp)).astype(np.float32)
    else:
        D = (L.sigma * rng.standard_normal((M, L.K, L.Csp))).astype(np.float32)
    if isinstance(L, Conv):
        codes = rng.integers(0, L.K, size=(L.Ct, L.dk, L.dk, M), dtype=np.uint8)
    else:
        codes = rng.integers(0, L.K, size=(L.Ct, M), dtype=np.uint8)
    return D, codes


def draw_input(rng: np.random.Generator, shape, integer: bool = False) -> np.ndarray:
    if integer:
        return rng.integers(0, 8, size=shape).astype(np.float32)
    return np.abs(rng.standard_normal(shape)).astype(np.float32)


def generate(name: str, seed: Optional[int] = None, integer: bool = False,
             N: Optional[int] = None) -> dict:
    """Inputs of workload ``name``: {'x': fp32, 'layers': [layer dicts], 'spec': Workload}.

    ``N`` overrides the batch (the draws of the codebooks and codes do not
    depend on it, but those of x do, so a smaller N is a different sample).
    """
    wl = WORKLOADS[name]
    rng = np.random.Generator(np.random.PCG64(wl.seed if seed is None else seed))
    n = wl.N if N is None else N
    x = draw_input(rng, (n,) + tuple(wl.in_shape), integer)
    layers = []
    for L in wl.layers:
        if isinstance(L, Pool):
            layers.append(layer_dict(L))
        else:
            D, codes = draw_layer(rng, L, integer)
            layers.append(layer_dict(L, D, codes))
    return {"x": x, "layers": layers, "spec": wl}


def random_conv(rng: np.random.Generator, N, Cs, H, W, Ct, dk, stride, pad, Csp, K,
                integer=False, sigma=0.1):
    """One conv layer of arbitrary shape (for edge-case tests)."""
    L = Conv(Cs, Ct, dk, stride, pad, Csp, K, False, sigma)
    x = draw_input(rng, (N, Cs, H, W), integer)
    D, codes = draw_layer(rng, L, integer)
    return x, D, codes


def random_fc(rng: np.random.Generator, N, Cs, Ct, Csp, K, integer=False, sigma=0.1):
    """One FC layer of arbitrary shape (for edge-case tests)."""
    L = FC(Cs, Ct, Csp, K, False, sigma)
    x = draw_input(rng, (N, Cs), integer)
    D, codes = draw_layer(rng, L, integer)
    return x, D, codes


# ------------------------------------------------------------ quantizer inputs
# Dense weights for the parameter quantization (Eq. (4), (6)): W [C_t][C_s]
# [d_k][d_k] (d_k = 1: a fully-connected layer) = sigma * N(0, 1), and initial
# sub-codebooks [M][K][C'_s] drawn from the same distribution (the k-means
# start is an input).  ``integer=True`` draws both in {-4..4}: every distance
# and every mean of such vectors is then exact or nearly so, which pins ties.

QUANT_LAYERS = {
    # name: (C_t, C_s, d_k, C'_s, K) -- AlexNet conv3 and fc6 shapes of the headline workloads
    "conv3": (384, 256, 3, 4, 128),
    "fc6": (4096, 9216, 1, 4, 32),
}


def random_quant(rng: np.random.Generator, Ct, Cs, dk, Csp, K, integer=False, sigma=0.05):
    M = Cs // Csp
    if integer:
        W = rng.integers(-4, 5, (Ct, Cs, dk, dk)).astype(np.float32)
        D = rng.integers(-4, 5, (M, K, Csp)).astype(np.float32)
    else:
        W = (sigma * rng.standard_normal((Ct, Cs, dk, dk))).astype(np.float32)
        D = (sigma * rng.standard_normal((M, K, Csp))).astype(np.float32)
    if dk == 1:
        W = W.reshape(Ct, Cs)
    return W, D
