"""GPU parity of every conv kernel family on the shapes the default one serves.

The library picks one kernel per layer (the flattened-grid kernel where it
can tile the layer).  QCNN_CONV_KERNEL = half puts the two-table kernel
(conv_half.hip: half-wave table rows, a builder wave, two tables in LDS)
first, = generic forces the simple per-subspace kernel, and
QCNN_TABLE_BUILD = valu makes the default kernel build its tables with
vector fused multiply-adds instead of MFMA (the comparison variant); each is
checked here against the CPU oracle on the headline layer (full size, float within
the bound and integer data bit for bit) and on stride-1 edge shapes (ragged
tiles and channel blocks, column strips, 1x1 kernels, every K block count).
"""
import os

import numpy as np
import pytest
import torch

from paper_1512_06473_amd import workloads as wl

pytestmark = pytest.mark.gpu

RTOL, ATOL = 1e-5, 1e-6

STRIDE1_SHAPES = [
    # N, Cs, H, W, Ct, dk, pad, Csp, K
    (1, 16, 14, 14, 32, 3, 1, 4, 16),       # column strips (W + pad > 14)
    (3, 12, 11, 9, 33, 3, 1, 4, 32),        # ragged channel block, odd map
    (3, 12, 13, 13, 200, 3, 1, 4, 9),       # K not a multiple of 16
    (2, 20, 10, 11, 7, 3, 0, 5, 32),        # pad 0, two channel groups
    (1, 18, 9, 14, 33, 3, 2, 6, 1),         # pad 2, K = 1
    (5, 16, 7, 12, 13, 3, 1, 8, 64),
    (2, 512, 6, 6, 16, 3, 1, 2, 16),        # many subspaces, split over workgroups
    (4, 32, 8, 8, 40, 1, 0, 4, 128),        # 1x1
    (2, 10, 8, 8, 7, 1, 0, 5, 9),           # 1x1, C's = 5
    (1, 7, 3, 3, 5, 3, 1, 1, 7),            # C's = 1, tiny map
    (2, 16, 10, 90, 20, 3, 1, 4, 128),      # wide map, ragged last strip
    (1, 64, 57, 57, 9, 3, 1, 8, 128),       # positions far beyond one tile
    (1, 8, 1, 1, 4, 3, 1, 4, 1),            # 1x1 input
]


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


@pytest.fixture(params=["half", "generic", "valu"])
def kernel(request, monkeypatch):
    if request.param == "valu":  # the default kernel with its tables built on the vector ALUs
        monkeypatch.delenv("QCNN_CONV_KERNEL", raising=False)
        monkeypatch.setenv("QCNN_TABLE_BUILD", "valu")
    else:
        monkeypatch.setenv("QCNN_CONV_KERNEL", request.param)
    return request.param


def T(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def run_conv(dev, x, D, codes, s, p, bias=None, relu=False):
    from paper_1512_06473_amd import api
    y = api.conv_forward(T(x, dev), T(D, dev), T(codes, dev), s, p, None if bias is None else T(bias, dev), relu)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def check(y, ref, A, what, exact=False):
    y = np.asarray(y, np.float64)
    assert y.shape == ref.shape, (what, y.shape, ref.shape)
    if exact:
        bad = y != ref
        assert not bad.any(), "%s: %d of %d differ (integer data must be bit-exact)" % (what, bad.sum(), bad.size)
        return
    err = np.abs(y - ref)
    lim = RTOL * A + ATOL
    bad = err > lim
    assert not bad.any(), "%s: %d of %d outside the bound; worst err/limit %.3g" % (
        what, int(bad.sum()), bad.size, float((err / lim).max()))


@pytest.mark.parametrize("integer", [False, True])
def test_headline_layer(dev, oracle, kernel, integer):
    d = wl.generate("alexnet_conv3_n32", integer=integer)
    L = d["layers"][0]
    y = run_conv(dev, d["x"], L["D"], L["codes"], L["stride"], L["pad"])
    ref, A = oracle.conv_lut(d["x"], L["D"], L["codes"], L["stride"], L["pad"], with_bound=True)
    check(y, ref, A, "alexnet_conv3_n32 %s integer=%s" % (kernel, integer), exact=integer)


@pytest.mark.parametrize("shape", STRIDE1_SHAPES)
def test_stride1_shapes(dev, oracle, kernel, shape):
    N, Cs, H, W, Ct, dk, p, Csp, K = shape
    rng = np.random.Generator(np.random.PCG64(sum(shape) + 17))
    x, D, codes = wl.random_conv(rng, N, Cs, H, W, Ct, dk, 1, p, Csp, K)
    b = rng.standard_normal(Ct).astype(np.float32)
    for bias, relu in [(None, False), (b, True)]:
        y = run_conv(dev, x, D, codes, 1, p, bias, relu)
        ref, A = oracle.conv_lut(x, D, codes, 1, p, bias=bias, relu=relu, with_bound=True)
        check(y, ref, A, "%s %s bias=%s relu=%s" % (kernel, shape, bias is not None, relu))
    xi, Di, ci = wl.random_conv(rng, N, Cs, H, W, Ct, dk, 1, p, Csp, K, integer=True)
    check(run_conv(dev, xi, Di, ci, 1, p), oracle.conv_lut(xi, Di, ci, 1, p), None, "%s int %s" % (kernel, shape),
          exact=True)


def test_default_kernel_unchanged_by_env_cleanup(dev, oracle):
    # With the switches unset the default kernel serves the layer again (they
    # are read per call).
    os.environ.pop("QCNN_CONV_KERNEL", None)
    os.environ.pop("QCNN_TABLE_BUILD", None)
    d = wl.generate("small_conv_n1")
    L = d["layers"][0]
    y = run_conv(dev, d["x"], L["D"], L["codes"], L["stride"], L["pad"])
    ref, A = oracle.conv_lut(d["x"], L["D"], L["codes"], L["stride"], L["pad"], with_bound=True)
    check(y, ref, A, "small_conv_n1 default kernel")
