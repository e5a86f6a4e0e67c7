"""Seeded random sweep of conv layer shapes on the GPU against the CPU oracle
(Eq. (7)).

Each case draws a layer: batch, channels, map size, kernel, stride and
padding, C'_s and K, including shapes where the planner picks the
stride-phase or row-group layouts, column strips, ragged channel blocks
(6, 8 or 12 channels per wave) and split subspaces.  Every case runs through
qcnn_conv_forward and through a prepared plan (which must agree bit for
bit), on float data (within the bound of the tolerance reading) and on
integer data (bit for bit with the oracle).  The shapes are kept small
enough for the oracle to finish each case in well under a second.
"""
import numpy as np
import pytest
import torch

from paper_1512_06473_amd import workloads as wl

pytestmark = pytest.mark.gpu

RTOL, ATOL = 1e-5, 1e-6
NCASES = 48


def draw_shape(rng):
    while True:
        dk = int(rng.choice([1, 2, 3, 3, 3, 4, 5, 5, 7, 11]))
        stride = int(rng.choice([1, 1, 1, 2, 2, 3, 4])) if dk > 1 else int(rng.choice([1, 2]))
        pad = int(rng.integers(0, dk // 2 + 2))
        Csp = int(rng.choice([1, 2, 3, 4, 4, 4, 5, 8, 16]))
        M = int(rng.integers(1, max(2, 96 // Csp) + 1))
        Cs = M * Csp
        K = int(rng.choice([1, 2, 7, 16, 32, 64, 100, 128, 256]))
        Ct = int(rng.integers(1, 300))
        N = int(rng.integers(1, 5))
        H = int(rng.integers(1, 40))
        W = int(rng.integers(1, 70))
        Ho = (H + 2 * pad - dk) // stride + 1
        Wo = (W + 2 * pad - dk) // stride + 1
        if Ho < 1 or Wo < 1:
            continue
        # keep the oracle's work (outputs x taps x subspaces) small
        if N * Ct * Ho * Wo * dk * dk * M > 6e7:
            continue
        return N, Cs, H, W, Ct, dk, stride, pad, Csp, K


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


@pytest.fixture(scope="module")
def api():
    from paper_1512_06473_amd import api as a
    return a


def T(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def bits(t):
    return t.cpu().numpy().view(np.uint32)


SHAPES = [draw_shape(np.random.Generator(np.random.PCG64(9000 + i))) for i in range(NCASES)]


@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_random_conv_shape(api, dev, oracle, shape):
    N, Cs, H, W, Ct, dk, st, pad, Csp, K = shape
    print("random conv", shape, flush=True)
    rng = np.random.Generator(np.random.PCG64(sum(shape) * 7 + 1))
    for integer in (False, True):
        x, D, codes = wl.random_conv(rng, N, Cs, H, W, Ct, dk, st, pad, Csp, K, integer=integer)
        bias = (rng.integers(-3, 4, size=Ct) if integer else rng.standard_normal(Ct)).astype(np.float32)
        relu = bool(rng.integers(0, 2))
        xd, Dd, cd, bd = T(x, dev), T(D, dev), T(codes, dev), T(bias, dev)
        y = api.conv_forward(xd, Dd, cd, st, pad, bd, relu)
        plan = api.ConvPlan((N, Cs, H, W), Dd, cd, st, pad, bd, relu)
        yp = plan(xd)
        torch.cuda.synchronize()
        assert np.array_equal(bits(y), bits(yp)), "plan differs from the per-call forward"
        ref, A = oracle.conv_lut(x, D, codes, st, pad, bias=bias, relu=relu, with_bound=True)
        got = y.cpu().numpy().astype(np.float64)
        assert got.shape == ref.shape
        if integer:
            diff = got != ref
            assert not diff.any(), "%d of %d differ" % (int(diff.sum()), diff.size)
        else:
            err = np.abs(got - ref)
            lim = RTOL * A + ATOL
            assert np.all(err <= lim), float((err / lim).max())
        plan.close()
