"""Python binding of the C ABI (include/qcnn.h): argument marshalling only.

torch tensors supply device memory and the current HIP stream; every step of
the computation runs in the library's HIP kernels.  Functions take and return
torch tensors on a ROCm device; outputs are allocated with torch.empty when
``out`` is not given.
"""
from __future__ import annotations

import ctypes
from typing import Optional, Tuple

import torch

from ._lib import check, lib


def _stream(t: torch.Tensor) -> int:
    return torch.cuda.current_stream(t.device).cuda_stream


def _need(t: torch.Tensor, name: str, dtype: torch.dtype, ndim: int, device=None) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if t.dim() != ndim:
        raise ValueError("%s must have %d dims, got shape %s" % (name, ndim, tuple(t.shape)))
    if not t.is_cuda:
        raise ValueError("%s must be on a GPU device" % name)
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, expected %s" % (name, t.device, device))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def out_size(n: int, k: int, stride: int = 1, pad: int = 0) -> int:
    return lib().qcnn_out_size(n, k, stride, pad)


def lut_build(x: torch.Tensor, codebooks: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Table of sub-codeword inner products [N][M][K][H][W] (qcnn_lut_build).

    x: [N][C_s][H][W] (or [N][C_s] for an FC input) fp32; codebooks [M][K][C'_s] fp32.
    """
    x4 = x if x.dim() == 4 else x.reshape(x.shape[0], x.shape[1], 1, 1)
    _need(x4, "x", torch.float32, 4)
    _need(codebooks, "codebooks", torch.float32, 3, x.device)
    N, Cs, H, W = x4.shape
    M, K, Csp = codebooks.shape
    if out is None:
        out = torch.empty((N, M, K, H, W), dtype=torch.float32, device=x.device)
    _need(out, "out", torch.float32, 5, x.device)
    if tuple(out.shape) != (N, M, K, H, W):
        raise ValueError("out has shape %s, expected %s" % (tuple(out.shape), (N, M, K, H, W)))
    check(lib().qcnn_lut_build(x4.data_ptr(), N, Cs, H, W, codebooks.data_ptr(), M, K, Csp,
                               out.data_ptr(), _stream(x)), "qcnn_lut_build")
    return out


def conv_forward(x: torch.Tensor, codebooks: torch.Tensor, codes: torch.Tensor, stride: int = 1, pad: int = 0,
                 bias: Optional[torch.Tensor] = None, relu: bool = False,
                 out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """PQ conv layer forward, Eq. (7) (qcnn_conv_forward).

    x [N][C_s][H][W] fp32, codebooks [M][K][C'_s] fp32, codes uint8 [C_t][d_k][d_k][M],
    bias [C_t] fp32 or None.  Returns y [N][C_t][H_o][W_o].
    """
    return _conv_call("qcnn_conv_forward", x, codebooks, codes, stride, pad, bias, relu, out)


def conv_forward_noalloc(x: torch.Tensor, codebooks: torch.Tensor, codes: torch.Tensor, stride: int, pad: int,
                         bias: Optional[torch.Tensor], relu: bool, out: torch.Tensor) -> torch.Tensor:
    """conv_forward that allocates nothing (qcnn_conv_forward_noalloc): the
    temporaries live in the library's static device scratch; the caller
    brings ``out``.  Raises QcnnError (QCNN_ERR_WORKSPACE) for a layer whose
    temporaries do not fit; calls that overlap on one device race."""
    if out is None:
        raise ValueError("conv_forward_noalloc needs the caller's output tensor")
    return _conv_call("qcnn_conv_forward_noalloc", x, codebooks, codes, stride, pad, bias, relu, out)


def conv_pool_forward(x: torch.Tensor, codebooks: torch.Tensor, codes: torch.Tensor, stride: int, pad: int,
                      pool_k: int, pool_s: int, bias: Optional[torch.Tensor] = None, relu: bool = False,
                      out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """conv_forward followed by pool_k x pool_k / stride pool_s max pooling
    (qcnn_conv_pool_forward), equal bit for bit to conv_forward then
    maxpool2d.  Returns y [N][C_t][H_p][W_p]."""
    return _conv_call("qcnn_conv_pool_forward", x, codebooks, codes, stride, pad, bias, relu, out,
                      pool=(int(pool_k), int(pool_s)))


def _conv_call(entry, x, codebooks, codes, stride, pad, bias, relu, out, pool=None):
    _need(x, "x", torch.float32, 4)
    _need(codebooks, "codebooks", torch.float32, 3, x.device)
    _need(codes, "codes", torch.uint8, 4, x.device)
    N, Cs, H, W = x.shape
    M, K, Csp = codebooks.shape
    Ct, dk, dk2, M2 = codes.shape
    if dk != dk2 or M2 != M:
        raise ValueError("codes shape %s does not match [C_t][d_k][d_k][M=%d]" % (tuple(codes.shape), M))
    Ho, Wo = out_size(H, dk, stride, pad), out_size(W, dk, stride, pad)
    if pool is not None:
        Ho, Wo = out_size(Ho, pool[0], pool[1], 0), out_size(Wo, pool[0], pool[1], 0)
    bp = 0
    if bias is not None:
        _need(bias, "bias", torch.float32, 1, x.device)
        if bias.shape[0] != Ct:
            raise ValueError("bias must have C_t=%d entries" % Ct)
        bp = bias.data_ptr()
    if out is None:
        out = torch.empty((N, Ct, max(Ho, 0), max(Wo, 0)), dtype=torch.float32, device=x.device)
    _need(out, "out", torch.float32, 4, x.device)
    if tuple(out.shape) != (N, Ct, Ho, Wo):
        raise ValueError("out has shape %s, expected %s" % (tuple(out.shape), (N, Ct, Ho, Wo)))
    extra = () if pool is None else pool
    check(getattr(lib(), entry)(x.data_ptr(), N, Cs, H, W, codebooks.data_ptr(), M, K, Csp,
                                codes.data_ptr(), Ct, dk, stride, pad, bp or None, int(bool(relu)),
                                *extra, out.data_ptr(), _stream(x)), entry)
    return out


class _Plan:
    """A layer prepared for repeated forwards on inputs of one shape
    (qcnn_plan_forward / qcnn_plan_destroy); made by ConvPlan or FcPlan."""

    def _create(self, entry, dev, in_shape, out_shape, *args):
        self._ptr = None
        handle = ctypes.c_void_p()
        with torch.cuda.device(dev):
            check(getattr(lib(), entry)(*args, ctypes.byref(handle), torch.cuda.current_stream(dev).cuda_stream),
                  entry)
        self._ptr = handle
        self.device = dev
        self.in_shape = tuple(in_shape)
        self.out_shape = tuple(out_shape)

    def __call__(self, x: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
        if self._ptr is None:
            raise ValueError("the plan is closed")
        _need(x, "x", torch.float32, len(self.in_shape), self.device)
        if tuple(x.shape) != self.in_shape:
            raise ValueError("x has shape %s, the plan's is %s" % (tuple(x.shape), self.in_shape))
        if out is None:
            out = torch.empty(self.out_shape, dtype=torch.float32, device=self.device)
        _need(out, "out", torch.float32, len(self.out_shape), self.device)
        if tuple(out.shape) != self.out_shape:
            raise ValueError("out has shape %s, expected %s" % (tuple(out.shape), self.out_shape))
        check(lib().qcnn_plan_forward(self._ptr, x.data_ptr(), out.data_ptr(), _stream(x)), "qcnn_plan_forward")
        return out

    def close(self) -> None:
        """Frees the plan (after its device has finished its work)."""
        if getattr(self, "_ptr", None) is not None:
            ptr, self._ptr = self._ptr, None
            with torch.cuda.device(self.device):
                check(lib().qcnn_plan_destroy(ptr), "qcnn_plan_destroy")

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _bias_arg(bias, Ct, dev) -> int:
    if bias is None:
        return 0
    _need(bias, "bias", torch.float32, 1, dev)
    if bias.shape[0] != Ct:
        raise ValueError("bias must have C_t=%d entries" % Ct)
    return bias.data_ptr()


class ConvPlan(_Plan):
    """A PQ conv layer prepared for inputs of shape in_shape (N, C_s, H, W)
    (qcnn_conv_plan_create).  codebooks [M][K][C'_s] fp32; codes uint8
    [C_t][d_k][d_k][M], or with ``packed=(C_t, d_k)`` their packed stream
    (pack_codes); bias [C_t] or None; pool None or (pool_k, pool_s).  The
    plan keeps its own copies: the tensors given may change afterwards.
    ``plan(x)`` equals conv_forward (or conv_pool_forward) with the same
    arguments, bit for bit, without re-laying the codes on every call."""

    def __init__(self, in_shape, codebooks: torch.Tensor, codes: torch.Tensor, stride: int = 1, pad: int = 0,
                 bias: Optional[torch.Tensor] = None, relu: bool = False, pool=None, packed=None):
        self._ptr = None
        dev = codebooks.device
        _need(codebooks, "codebooks", torch.float32, 3, dev)
        N, Cs, H, W = (int(v) for v in in_shape)
        M, K, Csp = codebooks.shape
        keep = codes
        if packed is None:
            _need(codes, "codes", torch.uint8, 4, dev)
            Ct, dk, dk2, M2 = codes.shape
            if dk != dk2 or M2 != M:
                raise ValueError("codes shape %s does not match [C_t][d_k][d_k][M=%d]" % (tuple(codes.shape), M))
            cptr = codes.data_ptr()
        else:
            Ct, dk = (int(v) for v in packed)
            cptr, keep = _packed_codes_arg(codes, Ct * dk * dk * M, K, dev)
        bp = _bias_arg(bias, Ct, dev)
        pk, ps = (0, 0) if pool is None else (int(pool[0]), int(pool[1]))
        Ho, Wo = out_size(H, dk, stride, pad), out_size(W, dk, stride, pad)
        if pool is not None:
            Ho, Wo = out_size(Ho, pk, ps, 0), out_size(Wo, pk, ps, 0)
        self._create("qcnn_conv_plan_create", dev, (N, Cs, H, W), (N, Ct, Ho, Wo), N, Cs, H, W,
                     codebooks.data_ptr(), M, K, Csp, cptr, int(packed is not None), Ct, dk, stride, pad,
                     bp or None, int(bool(relu)), pk, ps)
        del keep


class FcPlan(_Plan):
    """A PQ fully-connected layer prepared for inputs [N][C_s]
    (qcnn_fc_plan_create).  codebooks [M][K][C'_s] fp32; codes uint8
    [C_t][M], or with ``packed=C_t`` their packed stream; bias [C_t] or None.
    ``plan(x)`` equals fc_forward with the same arguments, bit for bit."""

    def __init__(self, N: int, codebooks: torch.Tensor, codes: torch.Tensor,
                 bias: Optional[torch.Tensor] = None, relu: bool = False, packed=None):
        self._ptr = None
        dev = codebooks.device
        _need(codebooks, "codebooks", torch.float32, 3, dev)
        M, K, Csp = codebooks.shape
        keep = codes
        if packed is None:
            _need(codes, "codes", torch.uint8, 2, dev)
            Ct, M2 = codes.shape
            if M2 != M:
                raise ValueError("codes shape %s does not match [C_t][M=%d]" % (tuple(codes.shape), M))
            cptr = codes.data_ptr()
        else:
            Ct = int(packed)
            cptr, keep = _packed_codes_arg(codes, Ct * M, K, dev)
        bp = _bias_arg(bias, Ct, dev)
        N, Cs = int(N), M * Csp
        self._create("qcnn_fc_plan_create", dev, (N, Cs), (N, Ct), N, Cs, codebooks.data_ptr(), M, K, Csp, cptr,
                     int(packed is not None), Ct, bp or None, int(bool(relu)))
        del keep


def fc_forward(x: torch.Tensor, codebooks: torch.Tensor, codes: torch.Tensor,
               bias: Optional[torch.Tensor] = None, relu: bool = False,
               out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """PQ fully-connected layer forward, Eq. (5) (qcnn_fc_forward).

    x [N][C_s] fp32 (any trailing shape is flattened), codebooks [M][K][C'_s],
    codes uint8 [C_t][M], bias [C_t] or None.  Returns y [N][C_t].
    """
    if x.dim() != 2:
        x = x.reshape(x.shape[0], -1)
    _need(x, "x", torch.float32, 2)
    _need(codebooks, "codebooks", torch.float32, 3, x.device)
    _need(codes, "codes", torch.uint8, 2, x.device)
    N, Cs = x.shape
    M, K, Csp = codebooks.shape
    Ct, M2 = codes.shape
    if M2 != M:
        raise ValueError("codes shape %s does not match [C_t][M=%d]" % (tuple(codes.shape), M))
    bp = 0
    if bias is not None:
        _need(bias, "bias", torch.float32, 1, x.device)
        if bias.shape[0] != Ct:
            raise ValueError("bias must have C_t=%d entries" % Ct)
        bp = bias.data_ptr()
    if out is None:
        out = torch.empty((N, Ct), dtype=torch.float32, device=x.device)
    _need(out, "out", torch.float32, 2, x.device)
    if tuple(out.shape) != (N, Ct):
        raise ValueError("out has shape %s, expected %s" % (tuple(out.shape), (N, Ct)))
    check(lib().qcnn_fc_forward(x.data_ptr(), N, Cs, codebooks.data_ptr(), M, K, Csp, codes.data_ptr(), Ct,
                                bp or None, int(bool(relu)), out.data_ptr(), _stream(x)), "qcnn_fc_forward")
    return out


# ---------------------------------------------------------------- packed codes
# Table 1 (Sec. 3.4): log2 K bits per quantization index.  Format and limits
# are those of include/qcnn.h.

def code_bits(K: int) -> int:
    """Bits per packed code (qcnn_code_bits): 0 for K = 1, else ceil(log2 K)."""
    b = lib().qcnn_code_bits(int(K))
    if b < 0:
        raise ValueError("K must be in [1, 256], got %d" % K)
    return b


def packed_bytes(n: int, K: int) -> int:
    """Bytes of the packed form of n codes (qcnn_packed_bytes): 4 ceil(n b / 32)."""
    code_bits(K)
    return int(lib().qcnn_packed_bytes(int(n), int(K)))


def pack_codes(codes: torch.Tensor, K: int, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """uint8 codes (any shape, contiguous) -> packed stream, uint8 [packed_bytes(numel, K)]."""
    _need(codes, "codes", torch.uint8, codes.dim())
    n = codes.numel()
    nb = packed_bytes(n, K)
    if out is None:
        out = torch.empty(max(nb, 1), dtype=torch.uint8, device=codes.device)[:nb]
    _need(out, "out", torch.uint8, 1, codes.device)
    if out.numel() != nb:
        raise ValueError("out must have %d bytes, got %d" % (nb, out.numel()))
    check(lib().qcnn_pack_codes(codes.data_ptr(), n, int(K), out.data_ptr() if nb else None, _stream(codes)),
          "qcnn_pack_codes")
    return out


def unpack_codes(packed: torch.Tensor, shape, K: int, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Packed stream -> uint8 codes of the given shape (qcnn_unpack_codes)."""
    _need(packed, "packed", torch.uint8, 1)
    shape = tuple(int(v) for v in shape)
    n = 1
    for v in shape:
        n *= v
    if packed.numel() != packed_bytes(n, K):
        raise ValueError("packed must have %d bytes, got %d" % (packed_bytes(n, K), packed.numel()))
    if out is None:
        out = torch.empty(shape, dtype=torch.uint8, device=packed.device)
    _need(out, "out", torch.uint8, len(shape), packed.device)
    if tuple(out.shape) != shape:
        raise ValueError("out has shape %s, expected %s" % (tuple(out.shape), shape))
    check(lib().qcnn_unpack_codes(packed.data_ptr() if packed.numel() else None, n, int(K), out.data_ptr(),
                                  _stream(packed)), "qcnn_unpack_codes")
    return out


def _packed_codes_arg(packed: torch.Tensor, n: int, K: int, device) -> int:
    _need(packed, "packed_codes", torch.uint8, 1, device)
    if packed.numel() != packed_bytes(n, K):
        raise ValueError("packed_codes must have %d bytes, got %d" % (packed_bytes(n, K), packed.numel()))
    if packed.numel() == 0:  # K = 1 stores nothing; the library still wants an aligned pointer
        packed = torch.zeros(4, dtype=torch.uint8, device=device)
    return packed.data_ptr(), packed


def conv_forward_packed(x: torch.Tensor, codebooks: torch.Tensor, packed_codes: torch.Tensor, C_t: int, d_k: int,
                        stride: int = 1, pad: int = 0, bias: Optional[torch.Tensor] = None, relu: bool = False,
                        out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """conv_forward with packed codes (qcnn_conv_forward_packed): packed_codes is
    the packed stream of codes [C_t][d_k][d_k][M]."""
    _need(x, "x", torch.float32, 4)
    _need(codebooks, "codebooks", torch.float32, 3, x.device)
    N, Cs, H, W = x.shape
    M, K, Csp = codebooks.shape
    ptr, keep = _packed_codes_arg(packed_codes, C_t * d_k * d_k * M, K, x.device)
    Ho, Wo = out_size(H, d_k, stride, pad), out_size(W, d_k, stride, pad)
    bp = 0
    if bias is not None:
        _need(bias, "bias", torch.float32, 1, x.device)
        if bias.shape[0] != C_t:
            raise ValueError("bias must have C_t=%d entries" % C_t)
        bp = bias.data_ptr()
    if out is None:
        out = torch.empty((N, C_t, max(Ho, 0), max(Wo, 0)), dtype=torch.float32, device=x.device)
    _need(out, "out", torch.float32, 4, x.device)
    if tuple(out.shape) != (N, C_t, Ho, Wo):
        raise ValueError("out has shape %s, expected %s" % (tuple(out.shape), (N, C_t, Ho, Wo)))
    check(lib().qcnn_conv_forward_packed(x.data_ptr(), N, Cs, H, W, codebooks.data_ptr(), M, K, Csp, ptr, C_t, d_k,
                                         stride, pad, bp or None, int(bool(relu)), out.data_ptr(), _stream(x)),
          "qcnn_conv_forward_packed")
    return out


def fc_forward_packed(x: torch.Tensor, codebooks: torch.Tensor, packed_codes: torch.Tensor, C_t: int,
                      bias: Optional[torch.Tensor] = None, relu: bool = False,
                      out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """fc_forward with packed codes (qcnn_fc_forward_packed): packed_codes is the
    packed stream of codes [C_t][M]."""
    if x.dim() != 2:
        x = x.reshape(x.shape[0], -1)
    _need(x, "x", torch.float32, 2)
    _need(codebooks, "codebooks", torch.float32, 3, x.device)
    N, Cs = x.shape
    M, K, Csp = codebooks.shape
    ptr, keep = _packed_codes_arg(packed_codes, C_t * M, K, x.device)
    bp = 0
    if bias is not None:
        _need(bias, "bias", torch.float32, 1, x.device)
        if bias.shape[0] != C_t:
            raise ValueError("bias must have C_t=%d entries" % C_t)
        bp = bias.data_ptr()
    if out is None:
        out = torch.empty((N, C_t), dtype=torch.float32, device=x.device)
    _need(out, "out", torch.float32, 2, x.device)
    if tuple(out.shape) != (N, C_t):
        raise ValueError("out has shape %s, expected %s" % (tuple(out.shape), (N, C_t)))
    check(lib().qcnn_fc_forward_packed(x.data_ptr(), N, Cs, codebooks.data_ptr(), M, K, Csp, ptr, C_t,
                                       bp or None, int(bool(relu)), out.data_ptr(), _stream(x)),
          "qcnn_fc_forward_packed")
    return out


def ec_fc(S: torch.Tensor, T: torch.Tensor, codebooks: torch.Tensor, codes: torch.Tensor, sweeps: int = 1,
          inner: int = 1, objective: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Error-corrected quantization of a FC layer, Eq. (8)-(12) (qcnn_ec_fc).

    S [N][C_s] layer inputs, T [N][C_t] desired responses (fp32); codebooks
    [M][K][C'_s] fp32 and codes uint8 [C_t][M] are updated in place.  Returns
    the objective history, float64 [1 + sweeps M].
    """
    _need(S, "S", torch.float32, 2)
    _need(T, "T", torch.float32, 2, S.device)
    _need(codebooks, "codebooks", torch.float32, 3, S.device)
    _need(codes, "codes", torch.uint8, 2, S.device)
    N, Cs = S.shape
    Ct = T.shape[1]
    M, K, Csp = codebooks.shape
    if T.shape[0] != N or tuple(codes.shape) != (Ct, M):
        raise ValueError("shapes: S %s, T %s, codes %s, codebooks %s" % (tuple(S.shape), tuple(T.shape),
                                                                          tuple(codes.shape), tuple(codebooks.shape)))
    if objective is None:
        objective = torch.empty(1 + sweeps * M, dtype=torch.float64, device=S.device)
    _need(objective, "objective", torch.float64, 1, S.device)
    if objective.numel() != 1 + sweeps * M:
        raise ValueError("objective must have 1 + sweeps M = %d entries" % (1 + sweeps * M))
    check(lib().qcnn_ec_fc(S.data_ptr(), N, Cs, T.data_ptr(), Ct, codebooks.data_ptr(), M, K, Csp, codes.data_ptr(),
                           int(sweeps), int(inner), objective.data_ptr(), _stream(S)), "qcnn_ec_fc")
    return objective


def ec_conv(S: torch.Tensor, T: torch.Tensor, codebooks: torch.Tensor, codes: torch.Tensor, stride: int = 1,
            pad: int = 0, sweeps: int = 1, inner: int = 1,
            objective: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Error-corrected quantization of a conv layer, Eq. (13), App. B
    (qcnn_ec_conv).

    S [N][C_s][H][W] layer inputs, T [N][C_t][H_o][W_o] desired responses
    (fp32); codebooks [M][K][C'_s] fp32 and codes uint8 [C_t][d_k][d_k][M] are
    updated in place.  Returns the objective history, float64 [1 + sweeps M].
    """
    _need(S, "S", torch.float32, 4)
    _need(T, "T", torch.float32, 4, S.device)
    _need(codebooks, "codebooks", torch.float32, 3, S.device)
    _need(codes, "codes", torch.uint8, 4, S.device)
    N, Cs, H, W = S.shape
    Ct, dk = codes.shape[0], codes.shape[1]
    M, K, Csp = codebooks.shape
    Ho, Wo = out_size(H, dk, stride, pad), out_size(W, dk, stride, pad)
    if tuple(T.shape) != (N, Ct, Ho, Wo) or tuple(codes.shape) != (Ct, dk, dk, M):
        raise ValueError("shapes: S %s, T %s, codes %s, codebooks %s" % (tuple(S.shape), tuple(T.shape),
                                                                          tuple(codes.shape), tuple(codebooks.shape)))
    if objective is None:
        objective = torch.empty(1 + sweeps * M, dtype=torch.float64, device=S.device)
    _need(objective, "objective", torch.float64, 1, S.device)
    if objective.numel() != 1 + sweeps * M:
        raise ValueError("objective must have 1 + sweeps M = %d entries" % (1 + sweeps * M))
    check(lib().qcnn_ec_conv(S.data_ptr(), N, Cs, H, W, T.data_ptr(), Ct, dk, int(stride), int(pad),
                             codebooks.data_ptr(), M, K, Csp, codes.data_ptr(), int(sweeps), int(inner),
                             objective.data_ptr(), _stream(S)), "qcnn_ec_conv")
    return objective


def maxpool2d(x: torch.Tensor, k: int = 3, s: int = 2, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """k x k / stride s max pooling, no padding (qcnn_maxpool2d): network glue."""
    _need(x, "x", torch.float32, 4)
    N, C, H, W = x.shape
    Ho, Wo = out_size(H, k, s, 0), out_size(W, k, s, 0)
    if out is None:
        out = torch.empty((N, C, max(Ho, 0), max(Wo, 0)), dtype=torch.float32, device=x.device)
    _need(out, "out", torch.float32, 4, x.device)
    check(lib().qcnn_maxpool2d(x.data_ptr(), N, C, H, W, k, s, out.data_ptr(), _stream(x)), "qcnn_maxpool2d")
    return out


def timing_enable(enable: bool = True) -> None:
    """Switch the library's kernel timing on or off (events around each call's main kernel)."""
    check(lib().qcnn_timing_enable(1 if enable else 0), "qcnn_timing_enable")


def timing_read() -> Tuple[float, int]:
    """(summed milliseconds, launches) of the main kernels timed since the last read."""
    ms = ctypes.c_double(0.0)
    n = ctypes.c_longlong(0)
    check(lib().qcnn_timing_read(ctypes.byref(ms), ctypes.byref(n)), "qcnn_timing_read")
    return ms.value, n.value


def timing_read_each(capacity: int = 4096):
    """Per-launch milliseconds of the main kernels timed since the last read
    (launch order; at most ``capacity`` of them)."""
    buf = (ctypes.c_double * max(1, capacity))()
    n = ctypes.c_longlong(0)
    check(lib().qcnn_timing_read_each(buf, capacity, ctypes.byref(n)), "qcnn_timing_read_each")
    return [buf[i] for i in range(min(n.value, capacity))]


def probe_lds(device=None) -> dict:
    """Measured LDS read peak of the device (qcnn_probe_lds): bytes per clock
    per CU, the shader clock under load (GHz) and bytes per second."""
    dev = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    vals = [ctypes.c_double(0.0) for _ in range(3)]
    with torch.cuda.device(dev):
        check(lib().qcnn_probe_lds(*[ctypes.byref(v) for v in vals], torch.cuda.current_stream(dev).cuda_stream),
              "qcnn_probe_lds")
    return {"bytes_per_clk_cu": vals[0].value, "clock_ghz": vals[1].value, "bytes_per_s": vals[2].value}


def probe_valu(device=None) -> dict:
    """Measured VALU issue costs (qcnn_probe_valu): shader clocks per wave64
    instruction per SIMD of v_add_f32, DPP v_add_f32 and v_mad_u32_u24."""
    dev = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    vals = [ctypes.c_double(0.0) for _ in range(3)]
    with torch.cuda.device(dev):
        check(lib().qcnn_probe_valu(*[ctypes.byref(v) for v in vals], torch.cuda.current_stream(dev).cuda_stream),
              "qcnn_probe_valu")
    return {"add_clk": vals[0].value, "dpp_add_clk": vals[1].value, "mad_clk": vals[2].value}


def probe_hbm(nbytes: int = 2 << 30, device=None) -> dict:
    """Measured HBM stream rates (qcnn_probe_hbm) over two buffers of
    ``nbytes``: read, write and copy (read + written) bytes per second."""
    dev = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    rd, wr, cp = ctypes.c_double(0.0), ctypes.c_double(0.0), ctypes.c_double(0.0)
    check(lib().qcnn_probe_hbm(src.data_ptr(), dst.data_ptr(), src.numel() * 4, ctypes.byref(rd), ctypes.byref(wr),
                               ctypes.byref(cp), _stream(src)), "qcnn_probe_hbm")
    del src, dst
    return {"read_bytes_per_s": rd.value, "write_bytes_per_s": wr.value, "copy_bytes_per_s": cp.value,
            "buffer_bytes": nbytes}


# ------------------------------------------------------ parameter quantization

def _quant_w(W: torch.Tensor):
    """W [C_t][C_s][d_k][d_k] (or [C_t][C_s] for an FC layer) -> (C_t, C_s, d_k)."""
    if W.dim() == 2:
        return W.shape[0], W.shape[1], 1
    _need(W, "W", torch.float32, 4)
    Ct, Cs, dk, dk2 = W.shape
    if dk != dk2:
        raise ValueError("W must be [C_t][C_s][d_k][d_k]")
    return Ct, Cs, dk


def _codes_shape(W, M):
    return (W.shape[0], M) if W.dim() == 2 else (W.shape[0], W.shape[2], W.shape[3], M)


def _need_shaped(t: torch.Tensor, name: str, dtype: torch.dtype, shape, device) -> None:
    """A caller-supplied buffer: dtype, exact shape, device, contiguity."""
    _need(t, name, dtype, len(shape), device)
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))


def pq_assign(W: torch.Tensor, codebooks: torch.Tensor, codes: Optional[torch.Tensor] = None,
              objective: Optional[torch.Tensor] = None):
    """Nearest sub-codeword of every sub-vector (Eq. (4)/(6) assignment step,
    qcnn_pq_assign).  Returns (codes uint8, per-subspace objective float64 [M])."""
    if W.dim() == 2:
        _need(W, "W", torch.float32, 2)
    Ct, Cs, dk = _quant_w(W)
    _need(codebooks, "codebooks", torch.float32, 3, W.device)
    M, K, Csp = codebooks.shape
    if codes is None:
        codes = torch.empty(_codes_shape(W, M), dtype=torch.uint8, device=W.device)
    _need_shaped(codes, "codes", torch.uint8, _codes_shape(W, M), W.device)
    if objective is None:
        objective = torch.empty(M, dtype=torch.float64, device=W.device)
    _need_shaped(objective, "objective", torch.float64, (M,), W.device)
    check(lib().qcnn_pq_assign(W.data_ptr(), Ct, Cs, dk, codebooks.data_ptr(), M, K, Csp, codes.data_ptr(),
                               objective.data_ptr(), _stream(W)), "qcnn_pq_assign")
    return codes, objective


def pq_update(W: torch.Tensor, codes: torch.Tensor, codebooks: torch.Tensor, counts: Optional[torch.Tensor] = None):
    """Each sub-codeword becomes the mean of its sub-vectors (update step,
    qcnn_pq_update); ``codebooks`` is updated in place and returned with the
    counts [M][K] int32."""
    if W.dim() == 2:
        _need(W, "W", torch.float32, 2)
    Ct, Cs, dk = _quant_w(W)
    _need(codebooks, "codebooks", torch.float32, 3, W.device)
    M, K, Csp = codebooks.shape
    _need_shaped(codes, "codes", torch.uint8, _codes_shape(W, M), W.device)
    if counts is None:
        counts = torch.empty((M, K), dtype=torch.int32, device=W.device)
    _need_shaped(counts, "counts", torch.int32, (M, K), W.device)
    check(lib().qcnn_pq_update(W.data_ptr(), Ct, Cs, dk, codes.data_ptr(), M, K, Csp, codebooks.data_ptr(),
                               counts.data_ptr(), _stream(W)), "qcnn_pq_update")
    return codebooks, counts


def pq_kmeans(W: torch.Tensor, init_codebooks: torch.Tensor, iters: int):
    """Learn sub-codebooks and codes by k-means (qcnn_pq_kmeans): iters x
    (assignment, update) and a final assignment.  Returns (codebooks, codes,
    objective float64 [iters + 1]); ``init_codebooks`` is not modified."""
    if W.dim() == 2:
        _need(W, "W", torch.float32, 2)
    Ct, Cs, dk = _quant_w(W)
    _need(init_codebooks, "init_codebooks", torch.float32, 3, W.device)
    D = init_codebooks.clone()
    M, K, Csp = D.shape
    codes = torch.empty(_codes_shape(W, M), dtype=torch.uint8, device=W.device)
    objective = torch.empty(int(iters) + 1, dtype=torch.float64, device=W.device)
    check(lib().qcnn_pq_kmeans(W.data_ptr(), Ct, Cs, dk, M, K, Csp, int(iters), D.data_ptr(), codes.data_ptr(),
                               objective.data_ptr(), _stream(W)), "qcnn_pq_kmeans")
    return D, codes, objective
