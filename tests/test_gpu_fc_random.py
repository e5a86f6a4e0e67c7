"""Seeded random sweep of fully-connected layer shapes on the GPU against the
CPU oracle (Eq. (5)).

Each case draws a layer: batch (1 to 300 images, so the tiled kernel's image
blocks and the per-image path both run), C_s, C'_s (1 to 16), K (1 to 256)
and C_t (1 to 5000, ragged channel blocks), with or without bias and ReLU.
Every case runs through qcnn_fc_forward and through a prepared plan (which
must agree bit for bit), on float data (within the bound of the tolerance
reading) and on integer data (bit for bit with the oracle).
"""
import numpy as np
import pytest
import torch

from paper_1512_06473_amd import workloads as wl

pytestmark = pytest.mark.gpu

RTOL, ATOL = 1e-5, 1e-6
NCASES = 40


def draw_shape(rng):
    while True:
        Csp = int(rng.choice([1, 2, 3, 4, 4, 4, 5, 8, 12, 16]))
        M = int(rng.integers(1, max(2, 1200 // Csp) + 1))
        Cs = M * Csp
        K = int(rng.choice([1, 2, 7, 16, 16, 32, 64, 100, 128, 256]))
        Ct = int(rng.integers(1, 5000))
        N = int(rng.choice([1, 2, 5, 17, 64, 65, 128, 130, 300]))
        if N * Ct * M > 8e7:  # the oracle's work (outputs x subspaces)
            continue
        return N, Cs, Ct, Csp, K


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


SHAPES = [draw_shape(np.random.Generator(np.random.PCG64(7000 + i))) for i in range(NCASES)]


@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_random_fc_shape(api, dev, oracle, shape):
    N, Cs, Ct, Csp, K = shape
    print("random fc", shape, flush=True)
    rng = np.random.Generator(np.random.PCG64(sum(shape) * 11 + 3))
    for integer in (False, True):
        x, D, codes = wl.random_fc(rng, N, Cs, Ct, Csp, K, integer=integer)
        use_bias = bool(rng.integers(0, 2))
        bias = None
        if use_bias:
            bias = (rng.integers(-3, 4, size=Ct) if integer else rng.standard_normal(Ct)).astype(np.float32)
        relu = bool(rng.integers(0, 2))
        xd, Dd, cd = T(x, dev), T(D, dev), T(codes, dev)
        bd = T(bias, dev) if use_bias else None
        y = api.fc_forward(xd, Dd, cd, bd, relu)
        plan = api.FcPlan(N, Dd, cd, bd, relu)
        yp = plan(xd)
        torch.cuda.synchronize()
        assert np.array_equal(bits(y), bits(yp)), "plan differs from the per-call forward"
        ref, A = oracle.fc_lut(x, D, codes, bias=bias, relu=relu, with_bound=True)
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
