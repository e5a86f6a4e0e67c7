"""GPU parity of the fused conv + max-pool call (qcnn_conv_pool_forward).

Two references for every case:
* the library's own two calls, qcnn_conv_forward then qcnn_maxpool2d, on
  the same inputs: the fused call must equal them bit for bit (the pooled
  split-sum kernel adds the splits in the same order and takes exact
  maxima);
* the CPU oracle's conv (Eq. (7)) with float64 window maxima: within the
  window maximum of the conv's bound (|max a - max b| <= max |a - b|), and
  bit for bit on integer data.
Layers whose subspaces the flat kernel splits over workgroups (small
batches, AlexNet conv2 and conv5 shapes) take the pooled split-sum kernel;
the others (conv1's strided layout at one split, the two-table and the
generic kernels) pool a full map in the workspace.
"""
import numpy as np
import pytest
import torch

from paper_1512_06473_amd import workloads as wl

pytestmark = pytest.mark.gpu

RTOL, ATOL = 1e-5, 1e-6

# N, C_s, H, W, C_t, d_k, stride, pad, C's, K, pool k, pool s, bias, relu
CASES = [
    (2, 96, 27, 27, 256, 5, 1, 2, 4, 128, 3, 2, True, True),    # AlexNet conv2 + pool2
    (4, 384, 13, 13, 256, 3, 1, 1, 4, 128, 3, 2, True, True),   # AlexNet conv5 + pool3
    (1, 3, 227, 227, 96, 11, 4, 0, 3, 64, 3, 2, False, True),   # AlexNet conv1 + pool1
    (3, 64, 13, 13, 40, 3, 1, 1, 4, 32, 2, 2, False, False),    # ragged windows (13 -> 6)
    (2, 32, 11, 9, 33, 3, 1, 1, 4, 16, 3, 3, True, False),      # stride = window, odd map
    (1, 48, 10, 10, 24, 3, 1, 1, 4, 16, 1, 1, False, True),     # 1x1 windows: the conv itself
    (2, 16, 7, 7, 12, 3, 1, 1, 4, 8, 7, 1, True, True),         # one window over the whole map
    (2, 32, 16, 16, 20, 1, 1, 0, 4, 16, 2, 2, False, True),     # 1x1 conv
    (9, 64, 13, 13, 64, 3, 1, 1, 4, 32, 3, 2, True, True),      # two image groups, the last of one image
    (1, 16, 100, 100, 16, 3, 1, 1, 4, 16, 2, 2, False, True),   # 10000 outputs per map: pools a full map
]


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


@pytest.fixture(scope="module")
def api():
    from paper_1512_06473_amd import api as a
    return a


@pytest.fixture(params=["default", "half", "generic"])
def kernel(request, monkeypatch):
    if request.param == "default":
        monkeypatch.delenv("QCNN_CONV_KERNEL", raising=False)
    else:
        monkeypatch.setenv("QCNN_CONV_KERNEL", request.param)
    monkeypatch.delenv("QCNN_TABLE_BUILD", raising=False)
    return request.param


def T(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def pool64(a, k, s):
    """k x k / stride s window maxima of a float64 array (no padding)."""
    Hp, Wp = (a.shape[2] - k) // s + 1, (a.shape[3] - k) // s + 1
    out = None
    for dy in range(k):
        for dx in range(k):
            v = a[:, :, dy:dy + s * (Hp - 1) + 1:s, dx:dx + s * (Wp - 1) + 1:s]
            out = v.copy() if out is None else np.maximum(out, v)
    return out


def draw(case, integer):
    N, Cs, H, W, Ct, dk, st, pad, Csp, K, pk, ps, has_bias, relu = case
    rng = np.random.Generator(np.random.PCG64(1000 + CASES.index(case) + (500 if integer else 0)))
    L = wl.Conv(Cs, Ct, dk, st, pad, Csp, K, relu, 0.05)
    D, codes = wl.draw_layer(rng, L, integer)
    x = wl.draw_input(rng, (N, Cs, H, W), integer)
    bias = None
    if has_bias:
        bias = (rng.integers(-4, 5, size=Ct) if integer else 0.1 * rng.standard_normal(Ct)).astype(np.float32)
    return x, D, codes, bias


@pytest.mark.parametrize("integer", [False, True])
@pytest.mark.parametrize("case", CASES, ids=[str(c[:10]) for c in CASES])
def test_conv_pool(api, dev, oracle, kernel, case, integer):
    N, Cs, H, W, Ct, dk, st, pad, Csp, K, pk, ps, has_bias, relu = case
    if kernel == "half" and (st != 1 or dk not in (1, 3)):
        pytest.skip("the two-table kernel serves stride-1 1x1 / 3x3 layers; others fall to the default")
    print("conv_pool", kernel, case, integer, flush=True)
    x, D, codes, bias = draw(case, integer)
    xd, Dd, cd = T(x, dev), T(D, dev), T(codes, dev)
    bd = None if bias is None else T(bias, dev)
    y = api.conv_pool_forward(xd, Dd, cd, st, pad, pk, ps, bd, relu)
    z = api.conv_forward(xd, Dd, cd, st, pad, bd, relu)
    y2 = api.maxpool2d(z, pk, ps)
    torch.cuda.synchronize()
    y, y2 = y.cpu().numpy(), y2.cpu().numpy()
    assert y.shape == y2.shape
    assert np.array_equal(y.view(np.uint32), y2.view(np.uint32)), "fused call differs from conv then max-pool"
    ref, A = oracle.conv_lut(x, D, codes, st, pad, bias=bias, relu=relu, with_bound=True)
    ref, A = pool64(ref, pk, ps), pool64(A, pk, ps)
    assert y.shape == ref.shape
    if integer:
        assert np.array_equal(y.astype(np.float64), ref), int((y != ref).sum())
    else:
        err = np.abs(y.astype(np.float64) - ref)
        assert np.all(err <= RTOL * A + ATOL), float((err / (RTOL * A + ATOL)).max())


def test_conv_pool_two_calls_and_streams(api, dev, oracle):
    """A split layer then a non-split one on one stream, then the split layer
    on a side stream: the workspace and partial-sum buffers are reused in
    stream order."""
    a, b = CASES[1], CASES[2]
    xa, Da, ca, ba = draw(a, False)
    xb, Db, cb, bb = draw(b, False)
    ya = api.conv_pool_forward(T(xa, dev), T(Da, dev), T(ca, dev), a[6], a[7], a[10], a[11], T(ba, dev), a[13])
    yb = api.conv_pool_forward(T(xb, dev), T(Db, dev), T(cb, dev), b[6], b[7], b[10], b[11], None, b[13])
    s = torch.cuda.Stream(dev)
    with torch.cuda.stream(s):
        ya2 = api.conv_pool_forward(T(xa, dev), T(Da, dev), T(ca, dev), a[6], a[7], a[10], a[11], T(ba, dev),
                                    a[13])
    torch.cuda.synchronize()
    assert torch.equal(ya, ya2)
    ref, A = oracle.conv_lut(xb, Db, cb, b[6], b[7], relu=b[13], with_bound=True)
    ref, A = pool64(ref, b[10], b[11]), pool64(A, b[10], b[11])
    err = np.abs(yb.cpu().numpy().astype(np.float64) - ref)
    assert np.all(err <= RTOL * A + ATOL)


def test_conv_pool_rejects(api, dev):
    x, D, codes, _ = draw(CASES[3], False)
    xd, Dd, cd = T(x, dev), T(D, dev), T(codes, dev)
    from paper_1512_06473_amd._lib import QcnnError
    for pk, ps in [(0, 1), (2, 0), (14, 1)]:  # empty window, zero stride, window past the 13x13 map
        with pytest.raises((QcnnError, ValueError)):
            api.conv_pool_forward(xd, Dd, cd, 1, 1, pk, ps)
