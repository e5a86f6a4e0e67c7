"""The allocation-free conv forward (qcnn_conv_forward_noalloc) against
qcnn_conv_forward, called through the C ABI.

Both run the same plan and kernels; only the home of the temporaries
differs (the library's static device scratch instead of its per-stream
buffer), so the outputs must agree bit for bit.  Each case makes two
allocation-free calls in a row, the second on a smaller input, so that the
second runs over the first one's leftovers in the shared scratch; the
smaller call is also held to the oracle's bound (Eq. (7)).  One case per
conv kernel family: the flattened-grid kernel with split partial sums (the
AlexNet conv3 layer at N = 32), the two-table kernel, and the generic
kernel (stride 4, no temporaries).  A layer too large for the scratch is
refused with QCNN_ERR_WORKSPACE and leaves the output untouched.
"""
import numpy as np
import pytest
import torch

from paper_1512_06473_amd import api
from paper_1512_06473_amd import workloads as wl
from paper_1512_06473_amd._lib import lib

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def T(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def call(entry, x, D, codes, stride, pad, bias, relu, y):
    N, Cs, H, W = x.shape
    M, K, Csp = D.shape
    Ct, dk = codes.shape[0], codes.shape[1]
    stream = torch.cuda.current_stream(x.device).cuda_stream
    return getattr(lib(), entry)(x.data_ptr(), N, Cs, H, W, D.data_ptr(), M, K, Csp, codes.data_ptr(), Ct, dk,
                                 stride, pad, None if bias is None else bias.data_ptr(), int(relu), y.data_ptr(),
                                 stream)


def layer(rng, dev, shape, integer=False):
    N, Cs, H, W, Ct, dk, s, p, Csp, K = shape
    x, D, codes = wl.random_conv(rng, N, Cs, H, W, Ct, dk, s, p, Csp, K, integer=integer)
    bias = (rng.integers(-3, 4, Ct) if integer else rng.standard_normal(Ct)).astype(np.float32)
    Ho, Wo = api.out_size(H, dk, s, p), api.out_size(W, dk, s, p)
    return dict(x=x, D=D, codes=codes, bias=bias, s=s, p=p, xd=T(x, dev), Dd=T(D, dev), cd=T(codes, dev),
                bd=T(bias, dev), shape=(N, Ct, Ho, Wo))


CASES = [
    # (kernel family forced, big shape, smaller shape):
    # N, Cs, H, W, Ct, dk, stride, pad, C's, K
    (None, (32, 256, 13, 13, 384, 3, 1, 1, 4, 128), (4, 256, 13, 13, 384, 3, 1, 1, 4, 128)),
    ("half", (8, 64, 13, 13, 96, 3, 1, 1, 4, 64), (2, 32, 9, 11, 40, 3, 1, 1, 4, 64)),
    ("generic", (4, 3, 67, 67, 32, 11, 4, 0, 3, 64), (1, 3, 35, 35, 20, 11, 4, 0, 3, 64)),
]


@pytest.mark.parametrize("kernel,big,small", CASES, ids=["flat", "half", "generic"])
@pytest.mark.parametrize("integer", [False, True])
def test_noalloc_equals_conv_forward(dev, oracle, monkeypatch, kernel, big, small, integer):
    if kernel is not None:
        monkeypatch.setenv("QCNN_CONV_KERNEL", kernel)
    else:
        monkeypatch.delenv("QCNN_CONV_KERNEL", raising=False)
    rng = np.random.Generator(np.random.PCG64(sum(big) + integer))
    calls = [layer(rng, dev, big, integer), layer(rng, dev, small, integer)]
    print("noalloc", kernel, big, small, integer, flush=True)
    got = []
    for c in calls:  # two allocation-free calls in a row, the second smaller
        y = torch.full(c["shape"], float("nan"), device=dev)
        st = call("qcnn_conv_forward_noalloc", c["xd"], c["Dd"], c["cd"], c["s"], c["p"], c["bd"], True, y)
        assert st == 0, st
        got.append(y)
    torch.cuda.synchronize()
    for c, y in zip(calls, got):
        ref = torch.full(c["shape"], float("nan"), device=dev)
        assert call("qcnn_conv_forward", c["xd"], c["Dd"], c["cd"], c["s"], c["p"], c["bd"], True, ref) == 0
        torch.cuda.synchronize()
        assert torch.equal(y, ref), "noalloc differs from qcnn_conv_forward %s" % (c["shape"],)
    c, y = calls[1], got[1].cpu().numpy()
    if integer:
        want = oracle.conv_lut(c["x"], c["D"], c["codes"], c["s"], c["p"], bias=c["bias"], relu=True)
        assert np.array_equal(y, want)
    else:
        want, A = oracle.conv_lut(c["x"], c["D"], c["codes"], c["s"], c["p"], bias=c["bias"], relu=True,
                                  with_bound=True)
        assert np.all(np.abs(y - want) <= 1e-5 * A + 1e-6)


def test_noalloc_python_binding(dev):
    rng = np.random.Generator(np.random.PCG64(8))
    c = layer(rng, dev, (3, 16, 11, 12, 24, 3, 1, 1, 4, 32))
    out = torch.empty(c["shape"], device=dev)
    y = api.conv_forward_noalloc(c["xd"], c["Dd"], c["cd"], 1, 1, c["bd"], True, out)
    ref = api.conv_forward(c["xd"], c["Dd"], c["cd"], 1, 1, c["bd"], True)
    torch.cuda.synchronize()
    assert y is out and torch.equal(y, ref)


def test_noalloc_refuses_layers_beyond_its_scratch(dev):
    from paper_1512_06473_amd._lib import QcnnError
    rng = np.random.Generator(np.random.PCG64(9))
    x = torch.from_numpy(np.abs(rng.standard_normal((64, 256, 13, 13))).astype(np.float32)).to(dev)
    D = torch.zeros((64, 128, 4), device=dev)
    codes = torch.zeros((384, 3, 3, 64), dtype=torch.uint8, device=dev)
    y = torch.full((64, 384, 13, 13), 7.0, device=dev)
    with pytest.raises(QcnnError) as err:
        api.conv_forward_noalloc(x, D, codes, 1, 1, None, False, y)
    assert err.value.status == 8
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())


def test_noalloc_under_graph_capture(dev):
    """The allocation-free forward recorded into a HIP graph (the callers it
    is for): each replay, with eager work and a synchronization between
    replays and a new input copied into the captured input buffer each time,
    equals the eager qcnn_conv_forward on that input bit for bit.  The layer
    is split over workgroups, so the captured work includes the code
    re-layout, the gather kernel and the split-sum kernel."""
    rng = np.random.Generator(np.random.PCG64(10))
    c = layer(rng, dev, (4, 256, 13, 13, 384, 3, 1, 1, 4, 128))
    y = torch.empty(c["shape"], device=dev)
    # one eager call first: per-device set-up (the scratch address, kernel
    # attributes) happens outside the capture
    assert call("qcnn_conv_forward_noalloc", c["xd"], c["Dd"], c["cd"], 1, 1, c["bd"], True, y) == 0
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream(dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            st = call("qcnn_conv_forward_noalloc", c["xd"], c["Dd"], c["cd"], 1, 1, c["bd"], True, y)
    assert st == 0, st
    torch.cuda.synchronize()
    for rep in range(4):
        xn = np.abs(rng.standard_normal(c["x"].shape)).astype(np.float32)
        c["xd"].copy_(T(xn, dev))
        ref = torch.full(c["shape"], float("nan"), device=dev)
        assert call("qcnn_conv_forward", c["xd"], c["Dd"], c["cd"], 1, 1, c["bd"], True, ref) == 0
        torch.cuda.synchronize()
        y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref), "replay %d differs from the eager forward" % rep
