"""GPU checks of the prepared conv layer (qcnn_conv_plan_create,
qcnn_plan_forward, qcnn_plan_destroy).

A plan's forward must equal the per-call entry point with the same
arguments bit for bit: qcnn_conv_forward without pooling, and
qcnn_conv_pool_forward with it (both are compared with the CPU oracle's
Eq. (7) in their own test files; one case here is also compared with the
oracle directly).  Layers cover the flat kernel with and without subspace
splits (the split sum, the pooled split sum, a full map pooled after an
unsplit layer), the strided and row-group layouts, and layers that other
kernels run (C'_s = 16, K = 256, and the kernel forced at creation through
QCNN_CONV_KERNEL), where the plan keeps a copy of the caller's codes.
"""
import numpy as np
import pytest
import torch

from paper_1512_06473_amd import workloads as wl

pytestmark = pytest.mark.gpu

RTOL, ATOL = 1e-5, 1e-6

# N, C_s, H, W, C_t, d_k, stride, pad, C's, K, pool (k, s) or None, bias, relu
CASES = [
    (4, 256, 13, 13, 384, 3, 1, 1, 4, 128, None, False, False),    # AlexNet conv3 shape, split
    (4, 384, 13, 13, 256, 3, 1, 1, 4, 128, (3, 2), True, True),    # conv5 + pool3: pooled split sum
    (1, 3, 227, 227, 96, 11, 4, 0, 3, 64, (3, 2), True, True),     # conv1 + pool1: unsplit, full map pooled
    (2, 96, 27, 27, 256, 5, 1, 2, 4, 128, (3, 2), True, True),     # conv2 + pool2: 2x5 row groups
    (2, 32, 16, 16, 20, 1, 1, 0, 4, 16, None, True, False),        # 1x1 conv
    (2, 64, 9, 9, 24, 3, 1, 1, 16, 32, None, True, True),          # C's = 16: not the flat kernel
    (1, 32, 8, 8, 16, 3, 1, 1, 4, 256, (2, 2), False, True),       # K = 256: not the flat kernel
    (3, 64, 13, 13, 40, 3, 1, 1, 4, 32, (2, 2), False, False),     # ragged windows
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


def T(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def draw(case, integer, seed=0):
    N, Cs, H, W, Ct, dk, st, pad, Csp, K, pool, has_bias, relu = case
    rng = np.random.Generator(np.random.PCG64(3000 + seed + CASES.index(case) + (500 if integer else 0)))
    L = wl.Conv(Cs, Ct, dk, st, pad, Csp, K, relu, 0.05)
    D, codes = wl.draw_layer(rng, L, integer)
    x = wl.draw_input(rng, (N, Cs, H, W), integer)
    bias = None
    if has_bias:
        bias = (rng.integers(-4, 5, size=Ct) if integer else 0.1 * rng.standard_normal(Ct)).astype(np.float32)
    return x, D, codes, bias


def per_call(api, case, xd, Dd, cd, bd):
    N, Cs, H, W, Ct, dk, st, pad, Csp, K, pool, has_bias, relu = case
    if pool is None:
        return api.conv_forward(xd, Dd, cd, st, pad, bd, relu)
    return api.conv_pool_forward(xd, Dd, cd, st, pad, pool[0], pool[1], bd, relu)


def bits(t):
    return t.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("kernel", ["default", "half", "generic"])
@pytest.mark.parametrize("integer", [False, True])
@pytest.mark.parametrize("case", CASES, ids=[str(c[:10]) for c in CASES])
def test_plan_equals_per_call(api, dev, monkeypatch, case, integer, kernel):
    N, Cs, H, W, Ct, dk, st, pad, Csp, K, pool, has_bias, relu = case
    if kernel == "default":
        monkeypatch.delenv("QCNN_CONV_KERNEL", raising=False)
    else:
        monkeypatch.setenv("QCNN_CONV_KERNEL", kernel)
    print("conv_plan", kernel, case, integer, flush=True)
    x, D, codes, bias = draw(case, integer)
    xd, Dd, cd = T(x, dev), T(D, dev), T(codes, dev)
    bd = None if bias is None else T(bias, dev)
    plan = api.ConvPlan((N, Cs, H, W), Dd, cd, st, pad, bd, relu, pool)
    y = plan(xd)
    y2 = plan(xd)  # a second forward of the same plan
    ref = per_call(api, case, xd, Dd, cd, bd)
    torch.cuda.synchronize()
    assert tuple(y.shape) == tuple(ref.shape) == plan.out_shape
    assert np.array_equal(bits(y), bits(ref)), "plan differs from the per-call forward"
    assert np.array_equal(bits(y2), bits(ref))
    plan.close()


def test_plan_against_oracle(api, dev, oracle):
    """The AlexNet conv3 case against the CPU oracle's Eq. (7), float data."""
    case = CASES[0]
    N, Cs, H, W, Ct, dk, st, pad, Csp, K, pool, has_bias, relu = case
    x, D, codes, bias = draw(case, False)
    plan = api.ConvPlan((N, Cs, H, W), T(D, dev), T(codes, dev), st, pad)
    y = plan(T(x, dev)).cpu().numpy().astype(np.float64)
    ref, A = oracle.conv_lut(x, D, codes, st, pad, with_bound=True)
    err = np.abs(y - ref)
    assert np.all(err <= RTOL * A + ATOL), float((err / (RTOL * A + ATOL)).max())


def test_plan_keeps_its_own_copies(api, dev):
    """Changing or freeing the caller's codebooks, codes and bias after
    creation does not change the plan's results."""
    case = CASES[1]
    N, Cs, H, W, Ct, dk, st, pad, Csp, K, pool, has_bias, relu = case
    x, D, codes, bias = draw(case, False)
    xd, Dd, cd, bd = T(x, dev), T(D, dev), T(codes, dev), T(bias, dev)
    ref = per_call(api, case, xd, Dd, cd, bd)
    plan = api.ConvPlan((N, Cs, H, W), Dd, cd, st, pad, bd, relu, pool)
    Dd.mul_(3.0)
    cd.copy_(torch.flip(cd, dims=[0]))
    bd.fill_(7.0)
    del Dd, cd, bd
    torch.cuda.empty_cache()
    y = plan(xd)
    torch.cuda.synchronize()
    assert np.array_equal(bits(y), bits(ref))


def test_plan_from_packed_codes(api, dev):
    """A plan from the packed code stream equals one from the byte codes
    (K = 100: 7 bits per code)."""
    case = (2, 64, 13, 13, 48, 3, 1, 1, 4, 100, None, True, True)
    N, Cs, H, W, Ct, dk, st, pad, Csp, K, pool, has_bias, relu = case
    rng = np.random.Generator(np.random.PCG64(77))
    L = wl.Conv(Cs, Ct, dk, st, pad, Csp, K, relu, 0.05)
    D, codes = wl.draw_layer(rng, L, False)
    x = wl.draw_input(rng, (N, Cs, H, W), False)
    bias = (0.1 * rng.standard_normal(Ct)).astype(np.float32)
    xd, Dd, cd, bd = T(x, dev), T(D, dev), T(codes, dev), T(bias, dev)
    packed = api.pack_codes(cd.reshape(-1), K)
    p_bytes = api.ConvPlan((N, Cs, H, W), Dd, cd, st, pad, bd, relu)
    p_packed = api.ConvPlan((N, Cs, H, W), Dd, packed, st, pad, bd, relu, packed=(Ct, dk))
    a, b = p_bytes(xd), p_packed(xd)
    torch.cuda.synchronize()
    assert np.array_equal(bits(a), bits(b))


def test_plan_rejects_a_code_out_of_range(api, dev):
    from paper_1512_06473_amd._lib import QcnnError
    case = CASES[4]
    N, Cs, H, W, Ct, dk, st, pad, Csp, K, pool, has_bias, relu = case
    x, D, codes, bias = draw(case, False)
    codes = codes.copy()
    codes.reshape(-1)[37] = K + 3
    with pytest.raises(QcnnError) as ei:
        api.ConvPlan((N, Cs, H, W), T(D, dev), T(codes, dev), st, pad)
    assert ei.value.status == 4  # QCNN_ERR_CODE_RANGE


def test_plan_rejects_overlapping_output(api, dev):
    from paper_1512_06473_amd import _lib
    case = CASES[4]  # 2x32x16x16 -> 2x20x16x16: y fits inside x's storage
    N, Cs, H, W, Ct, dk, st, pad, Csp, K, pool, has_bias, relu = case
    x, D, codes, bias = draw(case, False)
    xd = T(x, dev)
    plan = api.ConvPlan((N, Cs, H, W), T(D, dev), T(codes, dev), st, pad)
    y = xd.reshape(-1)[:N * Ct * H * W].view(N, Ct, H, W)
    st_ = _lib.lib().qcnn_plan_forward(plan._ptr, xd.data_ptr(), y.data_ptr(),
                                       torch.cuda.current_stream(dev).cuda_stream)
    assert st_ == 7  # QCNN_ERR_ALIAS; nothing launched
    assert torch.equal(xd, T(x, dev))


def test_plan_on_two_streams(api, dev):
    """Forwards of one plan on two streams at once (the plan is only read;
    each stream has its own workspace)."""
    case = CASES[0]
    N, Cs, H, W, Ct, dk, st, pad, Csp, K, pool, has_bias, relu = case
    x, D, codes, bias = draw(case, False)
    xd = T(x, dev)
    plan = api.ConvPlan((N, Cs, H, W), T(D, dev), T(codes, dev), st, pad)
    ref = plan(xd)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(dev), torch.cuda.Stream(dev)
    outs = []
    for s in (s1, s2, s1, s2):
        with torch.cuda.stream(s):
            outs.append(plan(xd))
    torch.cuda.synchronize()
    for o in outs:
        assert torch.equal(o, ref)


def test_plan_headline_full_size(api, dev):
    """The 32-image AlexNet conv3 layer, the benchmark's configuration:
    equal to the per-call forward bit for bit, float and integer data."""
    for integer in (False, True):
        d = wl.generate("alexnet_conv3_n32", integer=integer)
        L0 = d["layers"][0]
        x, D, codes = d["x"], L0["D"], L0["codes"]
        xd, Dd, cd = T(x, dev), T(D, dev), T(codes, dev)
        plan = api.ConvPlan(tuple(xd.shape), Dd, cd, 1, 1)
        y = plan(xd)
        ref = api.conv_forward(xd, Dd, cd, 1, 1)
        torch.cuda.synchronize()
        assert np.array_equal(bits(y), bits(ref))


def test_plan_closed_and_shape_checks(api, dev):
    case = CASES[4]
    N, Cs, H, W, Ct, dk, st, pad, Csp, K, pool, has_bias, relu = case
    x, D, codes, bias = draw(case, False)
    plan = api.ConvPlan((N, Cs, H, W), T(D, dev), T(codes, dev), st, pad)
    with pytest.raises(ValueError):
        plan(T(x[:1], dev))  # another batch size than the plan's
    plan.close()
    plan.close()  # a second close does nothing
    with pytest.raises(ValueError):
        plan(T(x, dev))


def test_plan_keeps_the_kernel_chosen_at_creation(api, dev, monkeypatch):
    """A plan made under QCNN_CONV_KERNEL=generic keeps the generic kernel
    after the variable is unset (float data: the kernels sum in different
    orders, so the bits tell them apart)."""
    case = CASES[7]
    N, Cs, H, W, Ct, dk, st, pad, Csp, K, pool, has_bias, relu = case
    x, D, codes, bias = draw(case, False)
    xd, Dd, cd = T(x, dev), T(D, dev), T(codes, dev)
    monkeypatch.setenv("QCNN_CONV_KERNEL", "generic")
    plan = api.ConvPlan((N, Cs, H, W), Dd, cd, st, pad, None, relu, pool)
    ref_generic = per_call(api, case, xd, Dd, cd, None)
    monkeypatch.delenv("QCNN_CONV_KERNEL")
    ref_default = per_call(api, case, xd, Dd, cd, None)
    y = plan(xd)
    torch.cuda.synchronize()
    assert np.array_equal(bits(y), bits(ref_generic))
    assert not np.array_equal(bits(ref_default), bits(ref_generic))  # the case does tell them apart
