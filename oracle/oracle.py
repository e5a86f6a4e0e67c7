"""ctypes front end of the CPU oracle (qcnn_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, by __graft_entry__.smoke() and by
the cpu_baseline leg of bench.py, never by the product package.  Everything
here is marshalling (numpy arrays in, float64 arrays out) plus the layer-by-
layer composition of a whole network from the oracle's own layer functions.

Paper: Wu et al., "Quantized Convolutional Neural Networks for Mobile Devices",
CVPR 2016 -- Sec. 3.1 Eq. (5) (fully-connected layer) and Sec. 3.2 Eq. (7)
(convolutional layer), each computed through the table of sub-codeword inner
products and, independently, as a dense layer on the rebuilt weights.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "qcnn_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

ERRORS = {-1: "bad argument", -2: "bad shape", -3: "K out of range", -4: "code >= K", -5: "out of memory"}


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (plain C, -O2, no fast-math, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _signatures():
    P, I = ctypes.c_void_p, ctypes.c_int
    return {
        "qo_lut": [P, I, I, I, I, P, I, I, I, P, P],
        "qo_conv_lut": [P, I, I, I, I, P, I, I, I, P, I, I, I, I, P, I, P, P],
        "qo_conv_direct": [P, I, I, I, I, P, I, I, I, P, I, I, I, I, P, I, P],
        "qo_conv_points": [P, I, I, I, I, P, I, I, I, P, I, I, I, I, P, I, P, I, P, P],
        "qo_fc_lut": [P, I, I, P, I, I, I, P, I, P, I, P, P],
        "qo_fc_direct": [P, I, I, P, I, I, I, P, I, P, I, P],
        "qo_fc_points": [P, I, I, P, I, I, I, P, I, P, I, P, I, P, P],
        "qo_maxpool": [P, I, I, I, I, I, I, P],
        "qo_pq_assign": [P, I, I, I, P, I, I, I, P, P],
        "qo_pq_distances": [P, I, I, I, P, I, I, I, P, P, P],
        "qo_pq_update": [P, I, I, I, P, I, I, I, P, P, P],
        "qo_pq_kmeans": [P, I, I, I, I, I, I, I, P, P, P],
        "qo_threads": [],
        "qo_set_threads": [I],
        "qo_code_bits": [I],
        "qo_pack_codes": [P, ctypes.c_longlong, I, P],
        "qo_unpack_codes": [P, ctypes.c_longlong, I, P],
    }


def load(path: str):
    """Load an oracle shared library (the default build, or another build of
    the same source, e.g. a deliberately broken copy in a pin test)."""
    cdll = ctypes.CDLL(path)
    for name, args in _signatures().items():
        f = getattr(cdll, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    return cdll


_lib = None
_override = None


def use(cdll) -> None:
    """Route the functions below to ``cdll`` (None restores the default)."""
    global _override
    _override = cdll


def lib():
    global _lib
    if _override is not None:
        return _override
    if _lib is None:
        _lib = load(build())
    return _lib


class OracleError(RuntimeError):
    pass


def _chk(rc: int) -> None:
    if rc != 0:
        raise OracleError(ERRORS.get(rc, "error %d" % rc))


def _f32(a):
    a = np.ascontiguousarray(a, dtype=np.float32)
    return a, a.ctypes.data


def _u8(a):
    a = np.ascontiguousarray(a, dtype=np.uint8)
    return a, a.ctypes.data


def _opt_f32(a):
    if a is None:
        return None, None
    return _f32(a)


def threads() -> int:
    return lib().qo_threads()


def set_threads(n: int) -> None:
    """Thread count of the oracle's parallel loops (for timing it)."""
    lib().qo_set_threads(int(n))


def out_size(n: int, k: int, s: int, p: int) -> int:
    span = n + 2 * p - k
    return span // s + 1 if span >= 0 else 0


def lut(x, D, with_bound=False):
    """Table of Sec. 3.1/3.2: [N][M][K][H][W] float64 (and the |term| sums)."""
    x, xp = _f32(x)
    D, Dp = _f32(D)
    N, Cs, H, W = x.shape
    M, K, Csp = D.shape
    out = np.empty((N, M, K, H, W), np.float64)
    ab = np.empty_like(out) if with_bound else None
    _chk(lib().qo_lut(xp, N, Cs, H, W, Dp, M, K, Csp, out.ctypes.data,
                      ab.ctypes.data if ab is not None else None))
    return (out, ab) if with_bound else out


def conv_lut(x, D, codes, stride=1, pad=0, bias=None, relu=False, with_bound=False):
    """Conv layer through the table, Eq. (7): [N][C_t][H_o][W_o] float64."""
    x, xp = _f32(x)
    D, Dp = _f32(D)
    codes, cp = _u8(codes)
    bias, bp = _opt_f32(bias)
    N, Cs, H, W = x.shape
    M, K, Csp = D.shape
    Ct, dk, dk2, M2 = codes.shape
    assert dk == dk2 and M2 == M
    Ho, Wo = out_size(H, dk, stride, pad), out_size(W, dk, stride, pad)
    y = np.empty((N, Ct, max(Ho, 0), max(Wo, 0)), np.float64)
    ab = np.empty_like(y) if with_bound else None
    _chk(lib().qo_conv_lut(xp, N, Cs, H, W, Dp, M, K, Csp, cp, Ct, dk, stride, pad, bp,
                           int(bool(relu)), y.ctypes.data,
                           ab.ctypes.data if ab is not None else None))
    return (y, ab) if with_bound else y


def conv_direct(x, D, codes, stride=1, pad=0, bias=None, relu=False):
    """Conv layer as a dense cross-correlation on the rebuilt kernel, Eq. (1)/(7)."""
    x, xp = _f32(x)
    D, Dp = _f32(D)
    codes, cp = _u8(codes)
    bias, bp = _opt_f32(bias)
    N, Cs, H, W = x.shape
    M, K, Csp = D.shape
    Ct, dk, _, _ = codes.shape
    Ho, Wo = out_size(H, dk, stride, pad), out_size(W, dk, stride, pad)
    y = np.empty((N, Ct, max(Ho, 0), max(Wo, 0)), np.float64)
    _chk(lib().qo_conv_direct(xp, N, Cs, H, W, Dp, M, K, Csp, cp, Ct, dk, stride, pad, bp,
                              int(bool(relu)), y.ctypes.data))
    return y


def conv_points(x, D, codes, pts, stride=1, pad=0, bias=None, relu=False):
    """Selected responses (n, c_t, yo, xo) of the conv layer: (values, bounds)."""
    x, xp = _f32(x)
    D, Dp = _f32(D)
    codes, cp = _u8(codes)
    bias, bp = _opt_f32(bias)
    pts = np.ascontiguousarray(pts, dtype=np.int32).reshape(-1, 4)
    N, Cs, H, W = x.shape
    M, K, Csp = D.shape
    Ct, dk, _, _ = codes.shape
    y = np.empty(len(pts), np.float64)
    ab = np.empty(len(pts), np.float64)
    _chk(lib().qo_conv_points(xp, N, Cs, H, W, Dp, M, K, Csp, cp, Ct, dk, stride, pad, bp,
                              int(bool(relu)), pts.ctypes.data, len(pts), y.ctypes.data,
                              ab.ctypes.data))
    return y, ab


def fc_lut(x, D, codes, bias=None, relu=False, with_bound=False):
    """FC layer through the table, Eq. (5): [N][C_t] float64."""
    x, xp = _f32(x)
    D, Dp = _f32(D)
    codes, cp = _u8(codes)
    bias, bp = _opt_f32(bias)
    N, Cs = x.shape
    M, K, Csp = D.shape
    Ct, M2 = codes.shape
    assert M2 == M
    y = np.empty((N, Ct), np.float64)
    ab = np.empty_like(y) if with_bound else None
    _chk(lib().qo_fc_lut(xp, N, Cs, Dp, M, K, Csp, cp, Ct, bp, int(bool(relu)), y.ctypes.data,
                         ab.ctypes.data if ab is not None else None))
    return (y, ab) if with_bound else y


def fc_direct(x, D, codes, bias=None, relu=False):
    """FC layer as a dense product with the rebuilt weights, Eq. (2)/(5)."""
    x, xp = _f32(x)
    D, Dp = _f32(D)
    codes, cp = _u8(codes)
    bias, bp = _opt_f32(bias)
    N, Cs = x.shape
    M, K, Csp = D.shape
    Ct, _ = codes.shape
    y = np.empty((N, Ct), np.float64)
    _chk(lib().qo_fc_direct(xp, N, Cs, Dp, M, K, Csp, cp, Ct, bp, int(bool(relu)), y.ctypes.data))
    return y


def fc_points(x, D, codes, pts, bias=None, relu=False):
    """Selected responses (n, c_t) of the FC layer: (values, bounds)."""
    x, xp = _f32(x)
    D, Dp = _f32(D)
    codes, cp = _u8(codes)
    bias, bp = _opt_f32(bias)
    pts = np.ascontiguousarray(pts, dtype=np.int32).reshape(-1, 2)
    N, Cs = x.shape
    M, K, Csp = D.shape
    Ct, _ = codes.shape
    y = np.empty(len(pts), np.float64)
    ab = np.empty(len(pts), np.float64)
    _chk(lib().qo_fc_points(xp, N, Cs, Dp, M, K, Csp, cp, Ct, bp, int(bool(relu)),
                            pts.ctypes.data, len(pts), y.ctypes.data, ab.ctypes.data))
    return y, ab


def maxpool(x, k=3, s=2):
    """k x k / stride s max pooling, no padding (network glue)."""
    x, xp = _f32(x)
    N, C, H, W = x.shape
    y = np.empty((N, C, out_size(H, k, s, 0), out_size(W, k, s, 0)), np.float64)
    _chk(lib().qo_maxpool(xp, N, C, H, W, k, s, y.ctypes.data))
    return y


def network(x, layers, absolute=False, layer_inputs=None):
    """Run a stack of PQ layers and pools through the oracle.

    ``layers`` is a list of dicts from the workload generator: kind 'conv'
    (D, codes, stride, pad, relu), 'fc' (D, codes, relu) or 'pool' (k, s).
    Each layer takes the fp32 rounding of the previous layer's float64 output,
    as the GPU path would receive it.  With ``absolute`` every value is
    replaced by its magnitude and ReLU is dropped (|x|, |D|, no ReLU): that
    network's output bounds the sum of |terms| that reach each final output.
    If ``layer_inputs`` is a list, the fp32 input of every layer is appended.
    Returns the float64 output of the last layer.
    """
    h = np.abs(x) if absolute else x
    for L in layers:
        h32 = np.ascontiguousarray(h, dtype=np.float32)
        if layer_inputs is not None:
            layer_inputs.append(h32)
        if L["kind"] == "pool":
            h = maxpool(h32, L["k"], L["s"])
            continue
        D = np.abs(L["D"]) if absolute else L["D"]
        relu = bool(L["relu"]) and not absolute
        if L["kind"] == "conv":
            h = conv_lut(h32, D, L["codes"], L["stride"], L["pad"], None, relu)
        else:
            h = fc_lut(h32.reshape(h32.shape[0], -1), D, L["codes"], None, relu)
    return h


# ---------------------------------------------------------------- quantizer
# Sec. 3.1 Eq. (4) and Sec. 3.2 Eq. (6): k-means per subspace over the
# sub-vectors of W [C_t][C_s][d_k][d_k] (d_k = 1: a fully-connected layer).

def _wshape(W):
    W = np.ascontiguousarray(W, dtype=np.float32)
    if W.ndim == 2:
        W = W.reshape(W.shape[0], W.shape[1], 1, 1)
    Ct, Cs, dk, dk2 = W.shape
    assert dk == dk2
    return W, Ct, Cs, dk


def pq_assign(W, D):
    """Nearest sub-codeword per sub-vector (Eq. (4)/(6): float64 distances,
    ties to the lowest index).  Returns codes [C_t][d_k][d_k][M] (FC:
    [C_t][M]) and the per-subspace float64 objective ||D B - W||^2."""
    fc = np.ndim(W) == 2
    W, Ct, Cs, dk = _wshape(W)
    D, Dp = _f32(D)
    M, K, Csp = D.shape
    codes = np.empty((Ct, dk, dk, M), np.uint8)
    obj = np.empty(M, np.float64)
    _chk(lib().qo_pq_assign(W.ctypes.data, Ct, Cs, dk, Dp, M, K, Csp, codes.ctypes.data, obj.ctypes.data))
    return (codes.reshape(Ct, M) if fc else codes), obj


def pq_distances(W, D, codes):
    """For an assignment made elsewhere: per sub-vector (codes' shape) the
    float64 distance to the named sub-codeword and the float64 minimum over
    all K, as (dcode, dmin)."""
    W, Ct, Cs, dk = _wshape(W)
    D, Dp = _f32(D)
    M, K, Csp = D.shape
    shape = np.shape(codes)
    codes, cp = _u8(np.asarray(codes).reshape(Ct, dk, dk, M))
    dcode = np.empty((Ct, dk, dk, M), np.float64)
    dmin = np.empty_like(dcode)
    _chk(lib().qo_pq_distances(W.ctypes.data, Ct, Cs, dk, Dp, M, K, Csp, cp, dcode.ctypes.data, dmin.ctypes.data))
    return dcode.reshape(shape), dmin.reshape(shape)


def pq_update(W, codes, D):
    """Each sub-codeword becomes the mean of its sub-vectors (float64 sum in
    sub-vector order, rounded to fp32); unused ones keep their value.
    Returns the new codebooks [M][K][C'_s] fp32 and the counts [M][K]."""
    W, Ct, Cs, dk = _wshape(W)
    D, Dp = _f32(D)
    M, K, Csp = D.shape
    codes, cp = _u8(np.asarray(codes).reshape(Ct, dk, dk, M))
    out = np.empty_like(D)
    counts = np.empty((M, K), np.int32)
    _chk(lib().qo_pq_update(W.ctypes.data, Ct, Cs, dk, cp, M, K, Csp, Dp, out.ctypes.data,
                            counts.ctypes.data))
    return out, counts


def pq_kmeans(W, D_init, iters):
    """iters x (assign, update) then a final assignment.  Returns the learned
    codebooks, the codes and the float64 objective of every assignment
    (length iters + 1)."""
    fc = np.ndim(W) == 2
    W, Ct, Cs, dk = _wshape(W)
    D = np.array(D_init, dtype=np.float32, copy=True, order="C")
    M, K, Csp = D.shape
    codes = np.empty((Ct, dk, dk, M), np.uint8)
    obj = np.empty(iters + 1, np.float64)
    _chk(lib().qo_pq_kmeans(W.ctypes.data, Ct, Cs, dk, M, K, Csp, int(iters), D.ctypes.data,
                            codes.ctypes.data, obj.ctypes.data))
    return D, (codes.reshape(Ct, M) if fc else codes), obj


# ------------------------------------------------------------- packed codes
# Table 1 (Sec. 3.4): log2 K bits per quantization index.  Stream format in
# qcnn_oracle.c (reading R6b): code i is bits i b .. i b + b - 1, least
# significant bit first, b = bits that hold 0 .. K-1.

def code_bits(K: int) -> int:
    b = lib().qo_code_bits(int(K))
    _chk(min(b, 0))
    return b


def packed_nbytes(n: int, K: int) -> int:
    """Bytes of the packed stream of n codes: ceil(n b / 8)."""
    return (int(n) * code_bits(K) + 7) // 8


def pack_codes(codes, K: int):
    """uint8 codes (any shape, C order) -> the packed stream (uint8, ceil(n b / 8) bytes)."""
    c, cp = _u8(np.asarray(codes).reshape(-1))
    out = np.zeros(max(packed_nbytes(c.size, K), 1), np.uint8)
    _chk(lib().qo_pack_codes(cp, c.size, int(K), out.ctypes.data))
    return out[:packed_nbytes(c.size, K)]


def unpack_codes(packed, n: int, K: int):
    """The packed stream of n codes -> uint8 codes [n]."""
    p = np.ascontiguousarray(np.asarray(packed, dtype=np.uint8))
    if p.size == 0:
        p = np.zeros(1, np.uint8)
    out = np.empty(max(int(n), 1), np.uint8)
    _chk(lib().qo_unpack_codes(p.ctypes.data, int(n), int(K), out.ctypes.data))
    return out[:int(n)]
