"""ctypes loader for libqcnn.so (the HIP kernels behind the C ABI of include/qcnn.h).

There is no fallback: if the library is missing or fails to load, every call
raises.  Build it with ``python -m paper_1512_06473_amd.build``.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libqcnn.so")

P, I = ctypes.c_void_p, ctypes.c_int

# Entry points declared in include/qcnn.h, with their argument types.
SIGNATURES = {
    "qcnn_lut_build": ([P, I, I, I, I, P, I, I, I, P, P], I),
    "qcnn_conv_forward": ([P, I, I, I, I, P, I, I, I, P, I, I, I, I, P, I, P, P], I),
    "qcnn_fc_forward": ([P, I, I, P, I, I, I, P, I, P, I, P, P], I),
    "qcnn_maxpool2d": ([P, I, I, I, I, I, I, P, P], I),
    "qcnn_pq_assign": ([P, I, I, I, P, I, I, I, P, P, P], I),
    "qcnn_pq_update": ([P, I, I, I, P, I, I, I, P, P, P], I),
    "qcnn_pq_kmeans": ([P, I, I, I, I, I, I, I, P, P, P, P], I),
    "qcnn_out_size": ([I, I, I, I], I),
    "qcnn_status_string": ([I], ctypes.c_char_p),
    "qcnn_version": ([], I),
    "qcnn_conv_forward_noalloc": ([P, I, I, I, I, P, I, I, I, P, I, I, I, I, P, I, P, P], I),
    "qcnn_conv_pool_forward": ([P, I, I, I, I, P, I, I, I, P, I, I, I, I, P, I, I, I, P, P], I),
    "qcnn_conv_forward_packed": ([P, I, I, I, I, P, I, I, I, P, I, I, I, I, P, I, P, P], I),
    "qcnn_conv_plan_create": ([I, I, I, I, P, I, I, I, P, I, I, I, I, I, P, I, I, I, ctypes.POINTER(P), P], I),
    "qcnn_fc_plan_create": ([I, I, P, I, I, I, P, I, I, P, I, ctypes.POINTER(P), P], I),
    "qcnn_plan_forward": ([P, P, P, P], I),
    "qcnn_plan_destroy": ([P], I),
    "qcnn_fc_forward_packed": ([P, I, I, P, I, I, I, P, I, P, I, P, P], I),
    "qcnn_code_bits": ([I], I),
    "qcnn_packed_bytes": ([ctypes.c_size_t, I], ctypes.c_size_t),
    "qcnn_pack_codes": ([P, ctypes.c_size_t, I, P, P], I),
    "qcnn_unpack_codes": ([P, ctypes.c_size_t, I, P, P], I),
    "qcnn_ec_fc": ([P, I, I, P, I, P, I, I, I, P, I, I, P, P], I),
    "qcnn_ec_conv": ([P, I, I, I, I, P, I, I, I, I, P, I, I, I, P, I, I, P, P], I),
    "qcnn_timing_enable": ([I], I),
    "qcnn_timing_read_each": ([ctypes.POINTER(ctypes.c_double), ctypes.c_longlong,
                               ctypes.POINTER(ctypes.c_longlong)], I),
    "qcnn_probe_valu": ([ctypes.POINTER(ctypes.c_double)] * 3 + [P], I),
    "qcnn_probe_lds": ([ctypes.POINTER(ctypes.c_double)] * 3 + [P], I),
    "qcnn_probe_hbm": ([P, P, ctypes.c_size_t] + [ctypes.POINTER(ctypes.c_double)] * 3 + [P], I),
    "qcnn_timing_read": ([ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_longlong)], I),
}

STATUS = {0: "QCNN_OK", 1: "QCNN_ERR_NULL", 2: "QCNN_ERR_SHAPE", 3: "QCNN_ERR_K_RANGE",
          4: "QCNN_ERR_CODE_RANGE", 5: "QCNN_ERR_HIP", 6: "QCNN_ERR_UNSUPPORTED", 7: "QCNN_ERR_ALIAS", 8: "QCNN_ERR_WORKSPACE"}

_lib = None


class QcnnError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = lib().qcnn_status_string(status).decode()
        super().__init__("%s: %s (%s)" % (where, STATUS.get(status, status), msg))


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libqcnn.so is not built (expected at %s); run "
                              "`python -m paper_1512_06473_amd.build`" % LIB_PATH)
        cdll = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in SIGNATURES.items():
            f = getattr(cdll, name)
            f.argtypes = args
            f.restype = res
        _lib = cdll
    return _lib


def check(status: int, where: str) -> None:
    if status != 0:
        raise QcnnError(status, where)
