"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bar (fp32 outputs): |gpu - oracle| <= 1e-5 * sum|terms| + 1e-6 per element,
where sum|terms| is the oracle's sum of the magnitudes of every product that
enters the output.  Integer-valued inputs (x in 0..7, D in -8..8) keep every
partial sum exact in fp32, so there the comparison is bit-exact: that checks
all code, subspace, offset, stride and padding indexing.
"""
import numpy as np
import pytest
import torch

from paper_1512_06473_amd import workloads as wl

pytestmark = pytest.mark.gpu

RTOL, ATOL = 1e-5, 1e-6


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


def assert_bound(gpu, ref, A, what):
    gpu = np.asarray(gpu, np.float64)
    assert gpu.shape == ref.shape, (what, gpu.shape, ref.shape)
    assert np.all(np.isfinite(gpu)), what + ": non-finite output"
    err = np.abs(gpu - ref)
    lim = RTOL * A + ATOL
    bad = err > lim
    assert not bad.any(), "%s: %d of %d outside the bound; worst err/limit %.3g" % (
        what, int(bad.sum()), bad.size, float((err / lim).max()))


def assert_exact(gpu, ref, what):
    gpu = np.asarray(gpu)
    assert gpu.shape == ref.shape, (what, gpu.shape, ref.shape)
    diff = gpu.astype(np.float64) != ref
    assert not diff.any(), "%s: %d of %d differ (integer data must be bit-exact)" % (what, int(diff.sum()), diff.size)


def pool64(a, k, s):
    """k x k / stride s window maxima of a float64 array [N][C][H][W] (no
    padding), for references and bounds that must not be rounded."""
    Hp, Wp = (a.shape[2] - k) // s + 1, (a.shape[3] - k) // s + 1
    out = None
    for dy in range(k):
        for dx in range(k):
            v = a[:, :, dy:dy + s * (Hp - 1) + 1:s, dx:dx + s * (Wp - 1) + 1:s]
            out = v.copy() if out is None else np.maximum(out, v)
    return out


def run_conv(api, dev, x, D, codes, s, p, bias=None, relu=False):
    y = api.conv_forward(T(x, dev), T(D, dev), T(codes, dev), s, p,
                         None if bias is None else T(bias, dev), relu)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def run_fc(api, dev, x, D, codes, bias=None, relu=False):
    y = api.fc_forward(T(x, dev), T(D, dev), T(codes, dev), None if bias is None else T(bias, dev), relu)
    torch.cuda.synchronize()
    return y.cpu().numpy()


# ------------------------------------------------------------ headline configs

@pytest.mark.parametrize("integer", [False, True])
@pytest.mark.parametrize("cfg", ["small_conv_n1", "alexnet_conv3_n32"])
def test_conv_config_full(api, dev, oracle, cfg, integer):
    d = wl.generate(cfg, integer=integer)
    L = d["layers"][0]
    y = run_conv(api, dev, d["x"], L["D"], L["codes"], L["stride"], L["pad"])
    ref, A = oracle.conv_lut(d["x"], L["D"], L["codes"], L["stride"], L["pad"], with_bound=True)
    if integer:
        assert_exact(y, ref, cfg + " integer")
    else:
        assert_bound(y, ref, A, cfg)


@pytest.mark.parametrize("integer", [False, True])
def test_fc_config_full(api, dev, oracle, integer):
    d = wl.generate("alexnet_fc6_n128", integer=integer)
    L = d["layers"][0]
    y = run_fc(api, dev, d["x"], L["D"], L["codes"])
    ref, A = oracle.fc_lut(d["x"], L["D"], L["codes"], with_bound=True)
    if integer:
        assert_exact(y, ref, "alexnet_fc6_n128 integer")
    else:
        assert_bound(y, ref, A, "alexnet_fc6_n128")


@pytest.mark.parametrize("integer", [False, True])
@pytest.mark.timeout(600)
def test_vgg16_conv3_n16_full(api, dev, oracle, integer):
    # Full-size VGG-conv3-shaped layer (16 x 256 x 56 x 56 -> 256, C's = 8,
    # K = 128): every one of the 12.8 M outputs against the oracle.
    d = wl.generate("vgg16_conv3_n16", integer=integer)
    L = d["layers"][0]
    y = run_conv(api, dev, d["x"], L["D"], L["codes"], L["stride"], L["pad"])
    if integer:
        assert_exact(y, oracle.conv_lut(d["x"], L["D"], L["codes"], L["stride"], L["pad"]), "vgg16_conv3_n16 integer")
    else:
        ref, A = oracle.conv_lut(d["x"], L["D"], L["codes"], L["stride"], L["pad"], with_bound=True)
        assert_bound(y, ref, A, "vgg16_conv3_n16")


@pytest.mark.timeout(600)
def test_alexnet_n64_every_layer_and_end_to_end(api, dev, oracle):
    from paper_1512_06473_amd.network import Network
    d = wl.generate("alexnet_n64")
    net = Network(d["layers"], dev)
    keep = []
    out = net.forward(T(d["x"], dev), keep)
    torch.cuda.synchronize()
    acts = [d["x"]] + [k.cpu().numpy() for k in keep]
    assert sum(len(L.specs) for L in net.layers) == len(d["layers"])
    assert [L.name for L in net.layers].count("conv+pool") == 3
    # Every library call, every output: the oracle gets the GPU's own fp32
    # input of that call, so each call is held to its own bound.  A conv
    # with its max-pool: the pooled oracle output, bounded by the window
    # maximum of the conv's bound (|max a - max b| <= max |a - b|).
    for i, L in enumerate(net.layers):
        spec = L.specs[0]
        hin, hout = acts[i], acts[i + 1]
        what = "alexnet_n64 call %d (%s)" % (i, L.name)
        if spec["kind"] == "pool":
            assert_exact(hout, oracle.maxpool(hin, spec["k"], spec["s"]), what)
        elif spec["kind"] == "conv":
            ref, A = oracle.conv_lut(hin, spec["D"], spec["codes"], spec["stride"], spec["pad"],
                                     relu=spec["relu"], with_bound=True)
            if len(L.specs) == 2:
                k, s = L.specs[1]["k"], L.specs[1]["s"]
                ref, A = pool64(ref, k, s), pool64(A, k, s)
            assert_bound(hout, ref, A, what)
        else:
            ref, A = oracle.fc_lut(hin.reshape(hin.shape[0], -1), spec["D"], spec["codes"], relu=spec["relu"],
                                   with_bound=True)
            assert_bound(hout, ref, A, what)
    # End to end on all 64 images: the oracle network in float64 from the same
    # input, bounded by the absolute network (|x|, |D|, no ReLU).
    ref = oracle.network(d["x"], d["layers"])
    A = oracle.network(d["x"], d["layers"], absolute=True)
    assert_bound(out.cpu().numpy(), ref, A, "alexnet_n64 end to end (64 images)")


# ----------------------------------------------------------------- table export

@pytest.mark.parametrize("shape", [(1, 16, 14, 14, 4, 16), (32, 256, 13, 13, 4, 128), (128, 9216, 1, 1, 4, 32),
                                   (3, 6, 5, 7, 3, 64), (2, 40, 9, 9, 8, 256), (2, 5, 3, 4, 5, 1)])
def test_lut_build(api, dev, oracle, shape):
    N, Cs, H, W, Csp, K = shape
    rng = np.random.Generator(np.random.PCG64(sum(shape)))
    x, D, _ = wl.random_conv(rng, N, Cs, H, W, 1, 1, 1, 0, Csp, K)
    L = api.lut_build(T(x, dev), T(D, dev))
    torch.cuda.synchronize()
    ref, A = oracle.lut(x, D, with_bound=True)
    assert_bound(L.cpu().numpy(), ref, A, "lut %s" % (shape,))
    xi, Di, _ = wl.random_conv(rng, N, Cs, H, W, 1, 1, 1, 0, Csp, K, integer=True)
    Li = api.lut_build(T(xi, dev), T(Di, dev))
    torch.cuda.synchronize()
    assert_exact(Li.cpu().numpy(), oracle.lut(xi, Di), "lut integer %s" % (shape,))


# ----------------------------------------------------------------- edge shapes

CONV_EDGE = [
    # N, Cs, H, W, Ct, dk, stride, pad, Csp, K
    (1, 16, 14, 14, 32, 3, 1, 1, 4, 16),
    (3, 12, 11, 9, 33, 3, 1, 1, 4, 32),      # C_t not a multiple of the channel block, odd map
    (2, 3, 47, 47, 20, 11, 4, 0, 3, 64),     # conv1-like, stride 4, 11x11
    (2, 24, 15, 15, 17, 5, 1, 2, 4, 128),    # conv2-like 5x5 pad 2
    (1, 40, 9, 70, 5, 3, 1, 1, 8, 256),      # wide map (several column tiles), K = 256
    (2, 10, 8, 8, 7, 1, 1, 0, 5, 9),         # 1x1 kernel, C's = 5 (runtime-length path)
    (1, 32, 6, 6, 3, 3, 2, 3, 16, 8),        # pad > d_k/2, C's = 16
    (4, 2, 5, 5, 65, 2, 3, 1, 1, 2),         # even kernel, stride 3, C's = 1
    (1, 8, 1, 1, 4, 3, 1, 1, 4, 1),          # 1x1 input, only the centre tap is inside; K = 1
    (2, 6, 30, 1, 3, 3, 2, 1, 2, 4),         # one-column map
    (1, 64, 57, 57, 9, 3, 1, 1, 8, 128),     # positions far beyond one tile
    # stride-1 shapes for the flattened-grid kernel: grid widths of every
    # residue mod 4, pad 0..2, K not a multiple of 16, C's of 1..8, ragged
    # channel blocks and tiles, long subspace ranges (split over blocks)
    (3, 12, 13, 13, 200, 3, 1, 1, 4, 9),
    (2, 20, 10, 11, 7, 3, 1, 0, 5, 32),
    (1, 18, 9, 14, 33, 3, 1, 2, 6, 1),
    (5, 16, 7, 12, 13, 3, 1, 1, 8, 64),
    (2, 6, 16, 5, 3, 3, 1, 1, 3, 100),
    (2, 512, 6, 6, 16, 3, 1, 1, 2, 16),
    (4, 32, 8, 8, 40, 1, 1, 0, 4, 128),
    (1, 7, 3, 3, 5, 3, 1, 1, 1, 7),
    # maps too wide for one table row: cut into column strips (ragged last strip)
    (2, 16, 10, 90, 20, 3, 1, 1, 4, 128),
    (1, 8, 12, 201, 4, 3, 1, 0, 8, 64),
    (1, 16, 5, 61, 140, 3, 1, 1, 8, 128),
    # stride phases and kernel-row groups (virtual subspaces), incl. padded tap grids
    (2, 12, 21, 19, 30, 3, 2, 1, 6, 40),     # 3x3 stride 2, two 4-channel groups
    (1, 9, 33, 29, 10, 7, 3, 2, 3, 24),      # 7x7 stride 3: 9 phases of 3x3 grids
    (3, 20, 9, 40, 70, 5, 1, 2, 5, 128),     # 5x5 pad 2, row groups, C's = 5
    (2, 8, 11, 11, 9, 5, 1, 0, 8, 100),      # 5x5 pad 0
    (1, 6, 12, 12, 5, 4, 2, 1, 2, 16),       # even kernel, stride 2
    # stride phases with 6 channels per wave: ragged channel blocks of 96, split subspaces
    (2, 12, 25, 25, 200, 3, 2, 1, 4, 32),    # 3x3 stride 2: three channel blocks, 12 splits
    (1, 64, 23, 23, 100, 5, 2, 2, 4, 64),    # 5x5 stride 2: 3x3 phase grids with a zero row, 16 splits
]


@pytest.mark.parametrize("shape", CONV_EDGE)
def test_conv_edge(api, dev, oracle, shape):
    N, Cs, H, W, Ct, dk, s, p, Csp, K = shape
    rng = np.random.Generator(np.random.PCG64(sum(shape) + 7))
    x, D, codes = wl.random_conv(rng, N, Cs, H, W, Ct, dk, s, p, Csp, K)
    b = rng.standard_normal(Ct).astype(np.float32)
    for bias, relu in [(None, False), (b, True)]:
        y = run_conv(api, dev, x, D, codes, s, p, bias, relu)
        ref, A = oracle.conv_lut(x, D, codes, s, p, bias=bias, relu=relu, with_bound=True)
        assert_bound(y, ref, A, "conv %s bias=%s relu=%s" % (shape, bias is not None, relu))
    xi, Di, ci = wl.random_conv(rng, N, Cs, H, W, Ct, dk, s, p, Csp, K, integer=True)
    assert_exact(run_conv(api, dev, xi, Di, ci, s, p), oracle.conv_lut(xi, Di, ci, s, p), "conv int %s" % (shape,))


FC_EDGE = [
    # N, Cs, Ct, Csp, K
    (1, 64, 10, 4, 32),
    (65, 96, 257, 4, 32),     # one image past a wave, C_t past a block
    (130, 300, 1000, 3, 16),
    (64, 4096, 1000, 4, 32),  # fc8-shaped, one wave of images
    (7, 48, 33, 1, 16),       # C's = 1, K = 16 (the paper's fc8 setting)
    (5, 80, 70, 8, 256),
    (3, 10, 5, 5, 1),         # K = 1, runtime-length C's
    (96, 640, 300, 8, 64),    # K = 64 (four codeword blocks), C's = 8
    (200, 192, 70, 4, 48),    # K = 48, two image blocks, ragged channels
    (128, 68, 40, 4, 32),     # M = 17: the last phase holds one subspace
]


@pytest.mark.parametrize("shape", FC_EDGE)
def test_fc_edge(api, dev, oracle, shape):
    N, Cs, Ct, Csp, K = shape
    rng = np.random.Generator(np.random.PCG64(sum(shape) + 3))
    x, D, codes = wl.random_fc(rng, N, Cs, Ct, Csp, K)
    b = rng.standard_normal(Ct).astype(np.float32)
    for bias, relu in [(None, False), (b, True)]:
        y = run_fc(api, dev, x, D, codes, bias, relu)
        ref, A = oracle.fc_lut(x, D, codes, bias=bias, relu=relu, with_bound=True)
        assert_bound(y, ref, A, "fc %s bias=%s relu=%s" % (shape, bias is not None, relu))
    xi, Di, ci = wl.random_fc(rng, N, Cs, Ct, Csp, K, integer=True)
    assert_exact(run_fc(api, dev, xi, Di, ci), oracle.fc_lut(xi, Di, ci), "fc int %s" % (shape,))


@pytest.mark.parametrize("shape", [(64, 96, 55, 55, 3, 2), (2, 5, 13, 13, 3, 2), (1, 2, 7, 9, 2, 3), (1, 1, 3, 3, 3, 1)])
def test_maxpool(api, dev, oracle, shape):
    N, C, H, W, k, s = shape
    x = np.random.Generator(np.random.PCG64(1)).standard_normal((N, C, H, W)).astype(np.float32)
    y = api.maxpool2d(T(x, dev), k, s)
    torch.cuda.synchronize()
    assert_exact(y.cpu().numpy(), oracle.maxpool(x, k, s), "maxpool %s" % (shape,))


# ------------------------------------------------------------------ semantics

def test_side_stream_and_determinism(api, dev, oracle):
    d = wl.generate("alexnet_fc6_n128", N=64)
    L = d["layers"][0]
    x, D, c = T(d["x"], dev), T(L["D"], dev), T(L["codes"], dev)
    s = torch.cuda.Stream(dev)
    with torch.cuda.stream(s):
        y1 = api.fc_forward(x, D, c)
        y2 = api.fc_forward(x, D, c)
    s.synchronize()
    assert torch.equal(y1, y2), "repeated calls must be bitwise identical"
    ref, A = oracle.fc_lut(d["x"], L["D"], L["codes"], with_bound=True)
    assert_bound(y1.cpu().numpy(), ref, A, "fc on a side stream")


def test_workspace_streams_and_growth(api, dev, oracle):
    # Conv and FC calls interleaved over two streams with no syncs between
    # them, in an order that grows each stream's workspace and shrinks it
    # back: every output must still match the oracle exactly.
    rng = np.random.Generator(np.random.PCG64(2024))
    conv_shapes = [(1, 16, 14, 14, 32, 3, 1, 1, 4, 16), (4, 64, 13, 13, 48, 3, 1, 1, 4, 64),
                   (2, 24, 15, 15, 17, 5, 1, 2, 4, 128)]
    fc_shapes = [(65, 96, 257, 4, 32), (7, 48, 33, 1, 16)]
    conv_in = [wl.random_conv(rng, *sh, integer=True) for sh in conv_shapes]
    fc_in = [wl.random_fc(rng, *sh, integer=True) for sh in fc_shapes]
    streams = [torch.cuda.Stream(dev), torch.cuda.Stream(dev)]
    jobs = []
    for rep in range(2):
        for i, (sh, (x, D, c)) in enumerate(zip(conv_shapes, conv_in)):
            with torch.cuda.stream(streams[(i + rep) % 2]):
                y = api.conv_forward(T(x, dev), T(D, dev), T(c, dev), sh[6], sh[7])
            jobs.append(("conv", i, y))
        for i, (x, D, c) in enumerate(fc_in):
            with torch.cuda.stream(streams[(i + rep + 1) % 2]):
                y = api.fc_forward(T(x, dev), T(D, dev), T(c, dev))
            jobs.append(("fc", i, y))
    for st in streams:
        st.synchronize()
    for kind, i, y in jobs:
        if kind == "conv":
            x, D, c = conv_in[i]
            ref = oracle.conv_lut(x, D, c, conv_shapes[i][6], conv_shapes[i][7])
        else:
            x, D, c = fc_in[i]
            ref = oracle.fc_lut(x, D, c)
        assert_exact(y.cpu().numpy(), ref, "%s %d across streams" % (kind, i))


def test_out_of_range_codes_are_clamped(api, dev, oracle):
    # Precondition violation: codes >= K.  The kernels clamp them to K - 1.
    rng = np.random.Generator(np.random.PCG64(77))
    x, D, codes = wl.random_conv(rng, 1, 8, 6, 6, 4, 3, 1, 1, 4, 16, integer=True)
    bad = codes.copy()
    bad[::2] = 200
    y = run_conv(api, dev, x, D, bad, 1, 1)
    assert_exact(y, oracle.conv_lut(x, D, np.minimum(bad, 15), 1, 1), "clamped codes")
