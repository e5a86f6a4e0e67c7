"""C ABI checks that need no GPU: the library loads, exports every entry point
include/qcnn.h declares, and rejects bad arguments on the host before any HIP
call (fake device pointers are safe here because validation fails first)."""
import ctypes
import os
import re

import pytest

from paper_1512_06473_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qcnn.h")

FAKE = 0x10000      # never dereferenced: validation rejects the call first
FAKE2 = 0x800000


@pytest.fixture(scope="module")
def L():
    return _lib.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(qcnn_[a-z0-9_]+)\s*\(", text)))


def test_header_and_binding_agree():
    decl = declared_functions()
    assert decl == sorted(_lib.SIGNATURES), (decl, sorted(_lib.SIGNATURES))


def test_exports_every_declared_symbol(L):
    for name in declared_functions():
        assert hasattr(L, name), name


def test_exported_dynamic_symbols():
    # Plain C names (no C++ mangling) in the dynamic symbol table.
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True, text=True).stdout
    names = set(line.split()[-1] for line in out.splitlines() if line.strip())
    for name in declared_functions():
        assert name in names, name


def test_version_status_outsize(L):
    assert L.qcnn_version() == 1
    for code, name in _lib.STATUS.items():
        s = L.qcnn_status_string(code)
        assert isinstance(s, bytes) and len(s) > 0
    assert L.qcnn_status_string(99) == b"unknown status"
    assert L.qcnn_out_size(13, 3, 1, 1) == 13
    assert L.qcnn_out_size(227, 11, 4, 0) == 55
    assert L.qcnn_out_size(27, 5, 1, 2) == 27
    assert L.qcnn_out_size(55, 3, 2, 0) == 27
    assert L.qcnn_out_size(2, 3, 1, 0) == 0
    assert L.qcnn_out_size(0, 1, 1, 0) == 0


def conv(L, entry="qcnn_conv_forward", **kw):
    a = dict(x=FAKE, N=2, Cs=8, H=5, W=5, D=FAKE, M=2, K=16, Csp=4, codes=FAKE, Ct=4, dk=3, s=1, p=1,
             bias=None, relu=0, y=FAKE2, stream=None)
    a.update(kw)
    return getattr(L, entry)(a["x"], a["N"], a["Cs"], a["H"], a["W"], a["D"], a["M"], a["K"], a["Csp"],
                               a["codes"], a["Ct"], a["dk"], a["s"], a["p"], a["bias"], a["relu"], a["y"],
                               a["stream"])


def fc(L, **kw):
    a = dict(x=FAKE, N=2, Cs=8, D=FAKE, M=2, K=16, Csp=4, codes=FAKE, Ct=4, bias=None, relu=0, y=FAKE2,
             stream=None)
    a.update(kw)
    return L.qcnn_fc_forward(a["x"], a["N"], a["Cs"], a["D"], a["M"], a["K"], a["Csp"], a["codes"], a["Ct"],
                             a["bias"], a["relu"], a["y"], a["stream"])


NULL, SHAPE, KR, UNSUP, ALIAS = 1, 2, 3, 6, 7


@pytest.mark.parametrize("kw,want", [
    (dict(x=None), NULL), (dict(D=None), NULL), (dict(codes=None), NULL), (dict(y=None), NULL),
    (dict(N=0), SHAPE), (dict(Cs=0), SHAPE), (dict(H=0), SHAPE), (dict(W=-1), SHAPE), (dict(Ct=0), SHAPE),
    (dict(dk=0), SHAPE), (dict(s=0), SHAPE), (dict(p=-1), SHAPE), (dict(M=3), SHAPE), (dict(Csp=3), SHAPE),
    (dict(K=0), KR), (dict(K=257), KR), (dict(K=-5), KR),
    (dict(H=1, W=1, p=0), SHAPE),                 # 3x3 kernel on 1x1 input: empty output
    (dict(Cs=34, M=2, Csp=17), UNSUP),           # C's > 16
    (dict(codes=FAKE + 1), UNSUP),                # codes not 4-byte aligned
    (dict(N=70000), UNSUP),                       # grid limit
    (dict(y=FAKE), ALIAS),                        # output == input
    (dict(y=FAKE + 64), ALIAS),                   # output starts inside the input
    (dict(bias=FAKE2 + 16), ALIAS),               # bias inside the output
    (dict(N=60000, Cs=1 << 14, M=1 << 12, H=1 << 12, W=1 << 12, p=0), SHAPE),  # element count overflow
])
def test_conv_rejects(L, kw, want):
    assert conv(L, **kw) == want
    # the allocation-free variant validates the same way, before any HIP call
    assert conv(L, "qcnn_conv_forward_noalloc", **kw) == want


def conv_pool(L, pk=3, ps=2, **kw):
    a = dict(x=FAKE, N=2, Cs=8, H=5, W=5, D=FAKE, M=2, K=16, Csp=4, codes=FAKE, Ct=4, dk=3, s=1, p=1,
             bias=None, relu=0, y=FAKE2, stream=None)
    a.update(kw)
    return L.qcnn_conv_pool_forward(a["x"], a["N"], a["Cs"], a["H"], a["W"], a["D"], a["M"], a["K"], a["Csp"],
                                    a["codes"], a["Ct"], a["dk"], a["s"], a["p"], a["bias"], a["relu"], pk, ps,
                                    a["y"], a["stream"])


@pytest.mark.parametrize("kw,want", [
    (dict(x=None), NULL), (dict(codes=None), NULL), (dict(y=None), NULL),
    (dict(N=0), SHAPE), (dict(Ct=0), SHAPE), (dict(M=3), SHAPE), (dict(K=0), KR),
    (dict(codes=FAKE + 1), UNSUP), (dict(y=FAKE + 64), ALIAS), (dict(bias=FAKE2 + 16), ALIAS),
    (dict(pk=0), SHAPE), (dict(ps=0), SHAPE), (dict(pk=-1, ps=-1), SHAPE),
    (dict(pk=6), SHAPE),                          # window larger than the 5x5 conv output
])
def test_conv_pool_rejects(L, kw, want):
    pk, ps = kw.pop("pk", 3), kw.pop("ps", 2)
    assert conv_pool(L, pk, ps, **kw) == want


def plan_create(L, plan_out=True, **kw):
    a = dict(N=2, Cs=8, H=5, W=5, D=FAKE, M=2, K=16, Csp=4, codes=FAKE, packed=0, Ct=4, dk=3, s=1, p=1,
             bias=None, relu=0, pk=0, ps=0, stream=None)
    a.update(kw)
    handle = ctypes.c_void_p(0xdead0)
    st = L.qcnn_conv_plan_create(a["N"], a["Cs"], a["H"], a["W"], a["D"], a["M"], a["K"], a["Csp"], a["codes"],
                                 a["packed"], a["Ct"], a["dk"], a["s"], a["p"], a["bias"], a["relu"], a["pk"],
                                 a["ps"], ctypes.byref(handle) if plan_out else None, a["stream"])
    return st, handle.value


@pytest.mark.parametrize("kw,want", [
    (dict(D=None), NULL), (dict(codes=None), NULL), (dict(plan_out=False), NULL),
    (dict(N=0), SHAPE), (dict(H=0), SHAPE), (dict(Ct=0), SHAPE), (dict(M=3), SHAPE), (dict(p=-1), SHAPE),
    (dict(K=0), KR), (dict(K=257), KR), (dict(K=0, packed=1), KR),
    (dict(H=1, W=1, p=0), SHAPE),                 # empty conv output
    (dict(pk=3), SHAPE), (dict(ps=2), SHAPE),     # one of the pooling sizes 0
    (dict(pk=-1, ps=-1), SHAPE), (dict(pk=6, ps=1), SHAPE),  # negative; window past the 5x5 map
    (dict(Cs=34, M=2, Csp=17), UNSUP),           # C's > 16
    (dict(codes=FAKE + 1), UNSUP), (dict(codes=FAKE + 2, packed=1), UNSUP),  # codes not 4-byte aligned
    (dict(N=70000), UNSUP),                       # grid limit
])
def test_conv_plan_create_rejects(L, kw, want):
    st, handle = plan_create(L, **kw)
    assert st == want
    assert handle == 0xdead0  # *plan is not written on an error


def fc_plan_create(L, plan_out=True, **kw):
    a = dict(N=2, Cs=8, D=FAKE, M=2, K=16, Csp=4, codes=FAKE, packed=0, Ct=4, bias=None, relu=0, stream=None)
    a.update(kw)
    handle = ctypes.c_void_p(0xdead0)
    st = L.qcnn_fc_plan_create(a["N"], a["Cs"], a["D"], a["M"], a["K"], a["Csp"], a["codes"], a["packed"], a["Ct"],
                               a["bias"], a["relu"], ctypes.byref(handle) if plan_out else None, a["stream"])
    return st, handle.value


@pytest.mark.parametrize("kw,want", [
    (dict(D=None), NULL), (dict(codes=None), NULL), (dict(plan_out=False), NULL),
    (dict(N=0), SHAPE), (dict(Ct=0), SHAPE), (dict(M=3), SHAPE), (dict(Cs=0), SHAPE),
    (dict(K=0), KR), (dict(K=257, packed=1), KR),
    (dict(Cs=34, M=2, Csp=17), UNSUP), (dict(codes=FAKE + 1), UNSUP), (dict(N=70000), UNSUP),
])
def test_fc_plan_create_rejects(L, kw, want):
    st, handle = fc_plan_create(L, **kw)
    assert st == want
    assert handle == 0xdead0


def test_plan_forward_and_destroy_without_gpu(L):
    assert L.qcnn_plan_forward(None, FAKE, FAKE2, None) == NULL
    assert L.qcnn_plan_destroy(None) == 0  # NULL is accepted, like free(NULL)


def test_noalloc_rejects_layers_beyond_its_scratch(L):
    # AlexNet conv3 at N = 64 (256 -> 384, 13x13, 3x3 pad 1, C's = 4, K = 128)
    # needs more temporaries than the static scratch holds: refused on the
    # host, before any HIP call (the fake addresses are never touched).
    X, Y, D, C = 1 << 40, 2 << 40, 3 << 40, 4 << 40
    st = L.qcnn_conv_forward_noalloc(X, 64, 256, 13, 13, D, 64, 128, 4, C, 384, 3, 1, 1, None, 0, Y, None)
    assert st == 8 and _lib.STATUS[st] == "QCNN_ERR_WORKSPACE"
    assert b"noalloc" in L.qcnn_status_string(8)


@pytest.mark.parametrize("kw,want", [
    (dict(x=None), NULL), (dict(codes=None), NULL), (dict(y=None), NULL),
    (dict(N=0), SHAPE), (dict(Ct=0), SHAPE), (dict(M=3), SHAPE), (dict(K=300), KR),
    (dict(codes=FAKE + 2), UNSUP), (dict(y=FAKE), ALIAS),
])
def test_fc_rejects(L, kw, want):
    assert fc(L, **kw) == want


def test_lut_and_pool_reject(L):
    assert L.qcnn_lut_build(None, 1, 8, 4, 4, FAKE, 2, 16, 4, FAKE2, None) == NULL
    assert L.qcnn_lut_build(FAKE, 1, 8, 4, 4, FAKE, 2, 0, 4, FAKE2, None) == KR
    assert L.qcnn_lut_build(FAKE, 1, 8, 0, 4, FAKE, 2, 16, 4, FAKE2, None) == SHAPE
    assert L.qcnn_lut_build(FAKE, 1, 8, 4, 4, FAKE, 2, 16, 4, FAKE, None) == ALIAS
    assert L.qcnn_maxpool2d(None, 1, 1, 5, 5, 3, 2, FAKE2, None) == NULL
    assert L.qcnn_maxpool2d(FAKE, 1, 1, 2, 2, 3, 2, FAKE2, None) == SHAPE
    assert L.qcnn_maxpool2d(FAKE, 1, 1, 5, 5, 3, 0, FAKE2, None) == SHAPE
    assert L.qcnn_maxpool2d(FAKE, 1, 1, 5, 5, 3, 2, FAKE, None) == ALIAS


def test_python_binding_rejects_host_tensors():
    import torch
    from paper_1512_06473_amd import api
    x = torch.zeros(1, 8, 5, 5)
    D = torch.zeros(2, 16, 4)
    codes = torch.zeros(4, 3, 3, 2, dtype=torch.uint8)
    with pytest.raises(ValueError, match="GPU"):
        api.conv_forward(x, D, codes, 1, 1)
    with pytest.raises(TypeError):
        api.conv_forward(x.double(), D, codes, 1, 1)


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "nope.so"))
    with pytest.raises(ImportError, match="not built"):
        _lib.lib()


def test_timing_calls_without_gpu(L):
    # Nothing recorded yet: reading returns zero launches without touching HIP.
    ms = ctypes.c_double(-1.0)
    n = ctypes.c_longlong(-1)
    assert L.qcnn_timing_read(None, ctypes.byref(n)) == NULL
    assert L.qcnn_timing_read(ctypes.byref(ms), None) == NULL
    assert L.qcnn_timing_enable(0) == 0
    assert L.qcnn_timing_read(ctypes.byref(ms), ctypes.byref(n)) == 0
    assert ms.value == 0.0 and n.value == 0
    buf = (ctypes.c_double * 4)()
    assert L.qcnn_timing_read_each(None, 4, ctypes.byref(n)) == NULL
    assert L.qcnn_timing_read_each(buf, 4, None) == NULL
    assert L.qcnn_timing_read_each(buf, -1, ctypes.byref(n)) == SHAPE
    assert L.qcnn_timing_read_each(buf, 4, ctypes.byref(n)) == 0 and n.value == 0


def test_probes_reject_bad_arguments(L):
    d = ctypes.c_double(0.0)
    assert L.qcnn_probe_lds(None, ctypes.byref(d), ctypes.byref(d), None) == NULL
    assert L.qcnn_probe_valu(ctypes.byref(d), None, ctypes.byref(d), None) == NULL
    r = ctypes.byref(d)
    assert L.qcnn_probe_hbm(None, FAKE2, 1024, r, r, r, None) == NULL
    assert L.qcnn_probe_hbm(FAKE, FAKE2, 1024, None, r, r, None) == NULL
    assert L.qcnn_probe_hbm(FAKE, FAKE2, 1024, r, None, r, None) == NULL
    assert L.qcnn_probe_hbm(FAKE, FAKE2, 8, r, r, r, None) == SHAPE
    assert L.qcnn_probe_hbm(FAKE + 4, FAKE2, 1024, r, r, r, None) == UNSUP
    assert L.qcnn_probe_hbm(FAKE, FAKE + 512, 1024, r, r, r, None) == ALIAS


def test_quantizer_rejects(L):
    # W [4][8][3][3] at FAKE, codebooks [2][16][4] at FAKE2, codes elsewhere.
    C = 0x2000000
    assert L.qcnn_pq_assign(None, 4, 8, 3, FAKE2, 2, 16, 4, C, None, None) == NULL
    assert L.qcnn_pq_assign(FAKE, 4, 8, 3, None, 2, 16, 4, C, None, None) == NULL
    assert L.qcnn_pq_assign(FAKE, 0, 8, 3, FAKE2, 2, 16, 4, C, None, None) == SHAPE
    assert L.qcnn_pq_assign(FAKE, 4, 8, 0, FAKE2, 2, 16, 4, C, None, None) == SHAPE
    assert L.qcnn_pq_assign(FAKE, 4, 8, 3, FAKE2, 3, 16, 4, C, None, None) == SHAPE
    assert L.qcnn_pq_assign(FAKE, 4, 8, 3, FAKE2, 2, 257, 4, C, None, None) == KR
    assert L.qcnn_pq_assign(FAKE, 4, 34, 3, FAKE2, 2, 16, 17, C, None, None) == UNSUP
    assert L.qcnn_pq_assign(FAKE, 4, 8, 3, FAKE2, 2, 16, 4, FAKE + 8, None, None) == ALIAS
    assert L.qcnn_pq_update(FAKE, 4, 8, 3, C, 2, 16, 4, None, None, None) == NULL
    assert L.qcnn_pq_update(FAKE, 4, 8, 3, C, 2, 0, 4, FAKE2, None, None) == KR
    assert L.qcnn_pq_update(FAKE, 4, 8, 3, C, 2, 16, 4, FAKE + 4, None, None) == ALIAS
    assert L.qcnn_pq_kmeans(FAKE, 4, 8, 3, 2, 16, 4, -1, FAKE2, C, None, None) == SHAPE
    assert L.qcnn_pq_kmeans(FAKE, 4, 8, 3, 2, 16, 4, 3, FAKE2, C, FAKE2 + 8, None) == ALIAS


# ------------------------------------------------------------- packed codes

def test_code_bits_and_packed_bytes(L):
    # Table 1 (Sec. 3.4): log2 K bits per index; whole dwords per stream.
    assert [L.qcnn_code_bits(K) for K in (1, 2, 3, 4, 16, 32, 33, 100, 128, 129, 256)] == \
        [0, 1, 2, 2, 4, 5, 6, 7, 7, 8, 8]
    assert L.qcnn_code_bits(0) == -1 and L.qcnn_code_bits(257) == -1
    assert L.qcnn_packed_bytes(0, 32) == 0
    assert L.qcnn_packed_bytes(3, 32) == 4          # 15 bits -> one dword
    assert L.qcnn_packed_bytes(7, 32) == 8          # 35 bits -> two dwords
    assert L.qcnn_packed_bytes(4096 * 2304, 32) == 4096 * 2304 * 5 // 8  # fc6 at 4/32: Table 1's bytes exactly
    assert L.qcnn_packed_bytes(1000, 1) == 0
    assert L.qcnn_packed_bytes(5, 0) == 0 and L.qcnn_packed_bytes(5, 300) == 0


def test_pack_unpack_rejects_bad_arguments(L):
    assert L.qcnn_pack_codes(FAKE, 4, 0, FAKE2, None) == KR
    assert L.qcnn_pack_codes(FAKE, 4, 257, FAKE2, None) == KR
    assert L.qcnn_pack_codes(None, 4, 16, FAKE2, None) == NULL
    assert L.qcnn_pack_codes(FAKE, 4, 16, None, None) == NULL
    assert L.qcnn_pack_codes(FAKE, 4, 16, FAKE2 + 2, None) == UNSUP     # packed not 4-byte aligned
    assert L.qcnn_pack_codes(FAKE + 1, 4, 16, FAKE2, None) == UNSUP     # codes not 4-byte aligned
    assert L.qcnn_pack_codes(FAKE, 64, 16, FAKE + 8, None) == ALIAS     # packed overlaps codes
    assert L.qcnn_pack_codes(None, 0, 16, None, None) == 0              # nothing to do, nothing launched
    assert L.qcnn_pack_codes(FAKE, 9, 1, None, None) == 0               # K = 1 stores nothing
    assert L.qcnn_unpack_codes(FAKE, 4, 0, FAKE2, None) == KR
    assert L.qcnn_unpack_codes(None, 4, 16, FAKE2, None) == NULL
    assert L.qcnn_unpack_codes(FAKE, 4, 16, None, None) == NULL
    assert L.qcnn_unpack_codes(FAKE + 2, 4, 16, FAKE2, None) == UNSUP
    assert L.qcnn_unpack_codes(FAKE, 64, 16, FAKE + 4, None) == ALIAS
    assert L.qcnn_unpack_codes(None, 0, 16, None, None) == 0


def test_packed_forwards_reject_bad_arguments(L):
    def convp(**kw):
        a = dict(x=FAKE, N=2, Cs=8, H=5, W=5, D=FAKE, M=2, K=16, Csp=4, codes=FAKE, Ct=4, dk=3, s=1, p=1,
                 bias=None, relu=0, y=FAKE2, stream=None)
        a.update(kw)
        return L.qcnn_conv_forward_packed(a["x"], a["N"], a["Cs"], a["H"], a["W"], a["D"], a["M"], a["K"], a["Csp"],
                                          a["codes"], a["Ct"], a["dk"], a["s"], a["p"], a["bias"], a["relu"], a["y"],
                                          a["stream"])

    def fcp(**kw):
        a = dict(x=FAKE, N=2, Cs=8, D=FAKE, M=2, K=16, Csp=4, codes=FAKE, Ct=4, bias=None, relu=0, y=FAKE2,
                 stream=None)
        a.update(kw)
        return L.qcnn_fc_forward_packed(a["x"], a["N"], a["Cs"], a["D"], a["M"], a["K"], a["Csp"], a["codes"],
                                        a["Ct"], a["bias"], a["relu"], a["y"], a["stream"])

    assert convp(K=0) == KR and fcp(K=300) == KR
    assert convp(codes=None) == NULL and fcp(codes=None) == NULL
    assert convp(Cs=9) == SHAPE and fcp(Cs=9) == SHAPE
    assert convp(codes=FAKE + 2) == UNSUP and fcp(codes=FAKE + 2) == UNSUP
    # the packed stream is smaller than the byte codes: y may start right after it
    assert convp(y=FAKE + 32) == ALIAS       # 72 codes at 4 bits = 36 bytes: y overlaps their last dword
    assert fcp(y=FAKE + 4) == ALIAS          # 8 codes at 4 bits = one dword


def test_ec_fc_rejects_bad_arguments(L):
    def ec(**kw):
        a = dict(S=FAKE, N=8, Cs=8, T=FAKE2, Ct=4, D=FAKE2 + 4096, M=2, K=16, Csp=4, codes=FAKE2 + 8192,
                 sweeps=1, inner=1, obj=None, stream=None)
        a.update(kw)
        return L.qcnn_ec_fc(a["S"], a["N"], a["Cs"], a["T"], a["Ct"], a["D"], a["M"], a["K"], a["Csp"], a["codes"],
                            a["sweeps"], a["inner"], a["obj"], a["stream"])

    assert ec(S=None) == NULL and ec(T=None) == NULL and ec(D=None) == NULL and ec(codes=None) == NULL
    assert ec(Cs=9) == SHAPE and ec(Ct=0) == SHAPE and ec(N=0) == SHAPE
    assert ec(sweeps=-1) == SHAPE and ec(inner=0) == SHAPE
    assert ec(K=0) == KR and ec(K=257) == KR
    assert ec(M=1, Csp=17, Cs=17) == UNSUP
    assert ec(D=FAKE + 16) == ALIAS                  # codebooks inside S
    assert ec(codes=FAKE2 + 4) == ALIAS              # codes inside T
    assert ec(obj=FAKE2 + 4096 + 8) == ALIAS         # objective inside the codebooks


def test_ec_fc_rejects_too_many_outputs(L):
    assert L.qcnn_ec_fc(FAKE, 8, 8, FAKE2, 65537, FAKE2 + (1 << 24), 2, 16, 4, FAKE2 + (1 << 25), 1, 1, None,
                        None) == UNSUP


def test_ec_conv_rejects_bad_arguments(L):
    def ec(**kw):
        a = dict(S=FAKE, N=2, Cs=8, H=5, W=5, T=FAKE2, Ct=4, dk=3, stride=1, pad=1, D=FAKE2 + 4096, M=2, K=16,
                 Csp=4, codes=FAKE2 + 8192, sweeps=1, inner=1, obj=None, stream=None)
        a.update(kw)
        return L.qcnn_ec_conv(a["S"], a["N"], a["Cs"], a["H"], a["W"], a["T"], a["Ct"], a["dk"], a["stride"],
                              a["pad"], a["D"], a["M"], a["K"], a["Csp"], a["codes"], a["sweeps"], a["inner"],
                              a["obj"], a["stream"])

    assert ec(S=None) == NULL and ec(T=None) == NULL and ec(D=None) == NULL and ec(codes=None) == NULL
    assert ec(Cs=9) == SHAPE and ec(Ct=0) == SHAPE and ec(N=0) == SHAPE and ec(H=0) == SHAPE
    assert ec(dk=0) == SHAPE and ec(stride=0) == SHAPE and ec(pad=-1) == SHAPE
    assert ec(dk=7, pad=0) == SHAPE                  # kernel larger than the padded input
    assert ec(sweeps=-1) == SHAPE and ec(inner=0) == SHAPE
    assert ec(K=0) == KR and ec(K=257) == KR
    assert ec(M=1, Csp=16, Cs=16) == UNSUP           # C'_s > 8 on this path
    assert ec(Ct=2000, dk=3) == UNSUP                # C_t d_k^2 > 16384
    assert ec(D=FAKE + 16) == ALIAS                  # codebooks inside S
    assert ec(codes=FAKE2 + 4) == ALIAS              # codes inside T
    assert ec(obj=FAKE2 + 4096 + 8) == ALIAS         # objective inside the codebooks
