"""The Table 1 cost model (Sec. 3.4) against the figures the paper prints.

The benchmark's dense-equivalent FLOP/s and its roofline byte counts come from
workmodel.py; these tests pin that arithmetic to Tables 2-9.
"""
import json
import os

import pytest

from paper_1512_06473_amd import workmodel as wm
from paper_1512_06473_amd import workloads as wl

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_tables.json")))

# Grouped AlexNet conv layers: (d_s, d_t, C_s, C_t, d_k, groups).
ALEX_CONV = [(227, 55, 3, 96, 11, 1), (27, 27, 96, 256, 5, 2), (13, 13, 256, 384, 3, 1),
             (13, 13, 384, 384, 3, 2), (13, 13, 384, 256, 3, 2)]
ALEX_FC = [(9216, 4096), (4096, 4096), (4096, 1000)]


def _alex_conv_flops(csp, K):
    dense = q = 0
    for i, (ds, dt, cs, ct, dk, g) in enumerate(ALEX_CONV):
        dense += wm.conv_flops_dense(dt, ct, dk, cs, g)
        q += wm.conv_flops_qcnn(ds, dt, cs, ct, dk, 3 if i == 0 else csp, K, g)
    return dense, q


def test_table4_conv2_speedup():
    g = GOLD["table4_alexnet_conv2_speedup"]
    L = g["layer"]
    for csp, K, printed in g["rows"]:
        d = wm.conv_flops_dense(L["dt"], L["Ct"], L["dk"], L["Cs"], L["groups"])
        q = wm.conv_flops_qcnn(L["ds"], L["dt"], L["Cs"], L["Ct"], L["dk"], csp, K, L["groups"])
        assert abs(d / q - printed) <= g["tol"], (csp, K, d / q, printed)


def test_table4_needs_groups():
    # Without the two groups the 4/64 row would be 3.85x, not the printed 3.70x.
    d = wm.conv_flops_dense(27, 256, 5, 96, 1)
    q = wm.conv_flops_qcnn(27, 27, 96, 256, 5, 4, 64, 1)
    assert abs(d / q - 3.70) > 0.1


def test_table5_all_conv_speedup():
    g = GOLD["table5_alexnet_all_conv_speedup"]
    for csp, K, printed in g["rows"]:
        d, q = _alex_conv_flops(csp, K)
        assert abs(d / q - printed) <= g["tol"], (csp, K, d / q, printed)


def test_table6_fc6_compression():
    g = GOLD["table6_caffenet_fc6_compression"]
    for csp, K, printed in g["rows"]:
        r = wm.fc_bytes_dense(9216, 4096) / wm.fc_bytes_qcnn(9216, 4096, csp, K)
        assert abs(r - printed) <= g["tol"], (csp, K, r, printed)


def test_table7_all_fc_compression():
    g = GOLD["table7_caffenet_all_fc_compression"]
    for csp, K, printed in g["rows"]:
        dense = sum(wm.fc_bytes_dense(a, b) for a, b in ALEX_FC)
        q = (wm.fc_bytes_qcnn(9216, 4096, csp, K) + wm.fc_bytes_qcnn(4096, 4096, csp, K)
             + wm.fc_bytes_qcnn(4096, 1000, 1, 16))
        assert abs(dense / q - printed) <= g["tol"], (csp, K, dense / q, printed)


def test_table8_whole_net_speedup():
    g = GOLD["table8_alexnet_whole_net_speedup"]
    for fcsp, K, printed in g["rows"]:
        d, q = _alex_conv_flops(8, 128)
        d += sum(wm.fc_flops_dense(a, b) for a, b in ALEX_FC)
        q += (wm.fc_flops_qcnn(9216, 4096, fcsp, K) + wm.fc_flops_qcnn(4096, 4096, fcsp, K)
              + wm.fc_flops_qcnn(4096, 1000, 1, 16))
        assert abs(d / q - printed) <= g["tol"], (fcsp, d / q, printed)


def test_table2_mnist_compression():
    g = GOLD["table2_mnist_compression"]
    for arch, printed in g["rows"]:
        dims = [int(v) for v in arch.split("-")]
        pairs = list(zip(dims[:-1], dims[1:]))
        hidden, out = pairs[:-1], pairs[-1]
        dense = sum(wm.fc_bytes_dense(a, b) for a, b in pairs)
        q = sum(wm.fc_bytes_qcnn(a, b, 4, 32) for a, b in hidden) + wm.fc_bytes_dense(*out)
        assert abs(dense / q - printed) <= g["tol"], (arch, dense / q, printed)


def _alexnet_params():
    n = 0
    for ds, dt, cs, ct, dk, g in ALEX_CONV:
        n += ct * (cs // g) * dk * dk + ct
    for a, b in ALEX_FC:
        n += a * b + b
    return n


def test_table9_and_table3_storage():
    n = _alexnet_params()
    assert n == 60965224
    mib = 4 * n / 2 ** 20
    g = GOLD["table9_alexnet_storage_mb"]
    assert abs(mib - g["value"]) <= g["tol"]
    g3 = GOLD["table3_alexnet_bytes"]
    assert abs(4 * n - g3["value"]) <= g3["tol"]


def test_valid_taps_brute_force():
    # Valid receptive-field pairs counted by brute force over a 2-D grid.
    for (H, W, dk, s, p) in [(13, 13, 3, 1, 1), (227, 227, 11, 4, 0), (27, 27, 5, 1, 2), (7, 5, 3, 2, 1)]:
        Ho, Wo = wm.out_size(H, dk, s, p), wm.out_size(W, dk, s, p)
        brute = sum(1 for yo in range(Ho) for xo in range(Wo) for ky in range(dk) for kx in range(dk)
                    if 0 <= yo * s - p + ky < H and 0 <= xo * s - p + kx < W)
        w = wm.conv_work(1, 4, H, W, 1, dk, s, p, 4, 2)
        assert w.gathers == brute  # 1 image, 1 channel, M = 1


def test_workload_counts():
    # Figures quoted for the five workloads: valid gathers and table entries.
    w2 = wm.workload_work(wl.WORKLOADS["alexnet_conv3_n32"])[0][1]
    assert w2.gathers == 32 * 384 * 64 * (13 * 13 * 9 - 4 * 13 * 3 + 4)
    assert w2.lut_entries == 32 * 169 * 64 * 128
    w3 = wm.workload_work(wl.WORKLOADS["alexnet_fc6_n128"])[0][1]
    assert w3.gathers == 128 * 4096 * 2304
    assert w3.dense_macs == 128 * 9216 * 4096
    w5 = wm.workload_work(wl.WORKLOADS["alexnet_n64"])
    kinds = [k for k, _ in w5]
    assert kinds == ["conv", "pool", "conv", "pool", "conv", "conv", "conv", "pool", "fc", "fc", "fc"]
    # conv1 gathers: 55x55 outputs, all 11x11 taps valid (227 = 54*4 + 11), M = 1.
    assert w5[0][1].gathers == 64 * 96 * 55 * 55 * 121
