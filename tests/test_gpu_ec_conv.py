"""GPU error-corrected quantization of a conv layer (Sec. 3.3.2 Eq. (13),
App. B Eq. (14)-(21)) through the C ABI, against the float64 oracle
(oracle/ec_conv.py).

The oracle follows the appendix on dense arrays (residuals Q and P formed
explicitly, the least squares of Eq. (19) built row by row, the error of
Eq. (21) summed for every candidate); the GPU works through the Gram blocks
of the shifted inputs and their correlations with the residual.  Both are
float64, so on inputs without near ties the codes must be equal and the
sub-codebooks and the objective history must agree to float64 rounding (the
GPU rounds the sub-codebooks to fp32 at the end).
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


@pytest.fixture(scope="module")
def api():
    from paper_1512_06473_amd import api as a
    return a


def T_(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def problem(rng, N, Cs, H, W, Ct, dk, st, pd, Csp, K, dead=None):
    S = np.maximum(rng.standard_normal((N, Cs, H, W)), 0).astype(np.float32)
    if dead is not None:
        S[:, dead] = 0.0
    Wt = (0.2 * rng.standard_normal((Ct, Cs, dk, dk))).astype(np.float64)
    Ho, Wo = (H + 2 * pd - dk) // st + 1, (W + 2 * pd - dk) // st + 1
    Sp = np.zeros((N, Cs, H + 2 * pd, W + 2 * pd))
    Sp[:, :, pd:pd + H, pd:pd + W] = S
    T = np.zeros((N, Ct, Ho, Wo))
    for ky in range(dk):
        for kx in range(dk):
            win = Sp[:, :, ky:ky + st * (Ho - 1) + 1:st, kx:kx + st * (Wo - 1) + 1:st]
            T += np.einsum("tc,nchw->nthw", Wt[:, :, ky, kx], win)
    T = (T + 0.01 * rng.standard_normal(T.shape)).astype(np.float32)
    D0 = (0.2 * rng.standard_normal((Cs // Csp, K, Csp))).astype(np.float32)
    c0 = rng.integers(0, K, (Ct, dk, dk, Cs // Csp)).astype(np.uint8)
    return S, T, D0, c0


def run_gpu(api, dev, S, T, D0, c0, st, pd, sweeps, inner):
    D = T_(D0, dev)
    c = T_(c0, dev)
    obj = api.ec_conv(T_(S, dev), T_(T, dev), D, c, st, pd, sweeps, inner)
    torch.cuda.synchronize()
    return D.cpu().numpy(), c.cpu().numpy(), obj.cpu().numpy()


# (N, C_s, H, W, C_t, d_k, stride, pad, C'_s, K, sweeps, inner, dead channels)
CASES = [
    (3, 8, 6, 6, 10, 3, 1, 1, 4, 8, 1, 1, None),
    (2, 6, 7, 5, 12, 3, 2, 1, 3, 5, 1, 2, None),     # stride 2, ragged map
    (2, 8, 5, 5, 9, 2, 1, 0, 2, 4, 2, 1, None),      # even kernel, no padding, two sweeps
    (4, 4, 4, 4, 6, 1, 1, 0, 4, 8, 1, 1, None),      # 1x1 kernel
    (1, 16, 9, 9, 20, 5, 1, 2, 8, 16, 1, 1, None),   # 5x5, C'_s = 8
    (2, 6, 6, 6, 40, 3, 1, 1, 6, 16, 1, 1, None),    # more (c, p) pairs than one sort chunk
    (2, 4, 5, 5, 6, 3, 1, 1, 4, 1, 1, 1, None),      # K = 1
    (1, 4, 5, 5, 8, 3, 1, 1, 4, 256, 1, 1, None),    # K = 256, most sub-codewords unused
    (2, 8, 6, 6, 12, 3, 1, 1, 4, 6, 1, 2, [1, 6]),   # input channels zero everywhere
    (2, 4, 5, 5, 6, 3, 1, 1, 4, 8, 0, 1, None),      # no sweep: the starting objective only
    (1, 4, 4, 4, 600, 3, 1, 1, 4, 32, 1, 1, None),   # 5400 pairs: 22 sort chunks, 3 channel blocks
    (1, 8, 4, 4, 200, 3, 1, 1, 8, 256, 1, 1, None),  # normal matrices too large to precompute in LDS
]


@pytest.mark.parametrize("case", CASES, ids=[str(c[:12]) for c in CASES])
def test_ec_conv_matches_oracle(api, dev, case):
    from oracle import ec_conv
    N, Cs, H, W, Ct, dk, st, pd, Csp, K, sweeps, inner, dead = case
    rng = np.random.Generator(np.random.PCG64(abs(hash(case[:12])) % (2 ** 32)))
    S, T, D0, c0 = problem(rng, N, Cs, H, W, Ct, dk, st, pd, Csp, K, dead)
    print("ec_conv", case, flush=True)
    D, c, obj = run_gpu(api, dev, S, T, D0, c0, st, pd, sweeps, inner)
    Dr, cr, hr = ec_conv.ec_conv(S, T, D0, c0, st, pd, sweeps, inner)
    assert np.array_equal(c, cr), "assignments differ in %d places" % int((c != cr).sum())
    scale = max(float(np.abs(Dr).max()), 1e-30)
    assert np.allclose(D, Dr, rtol=1e-6, atol=1e-7 * scale), float(np.abs(D - Dr).max())
    assert obj.shape == hr.shape
    assert np.allclose(obj, hr, rtol=1e-9, atol=1e-9 * hr[0]), (obj[:4], hr[:4])
    assert np.all(np.diff(obj) <= 1e-9 * obj[0])
    if dead is not None:
        for ch in dead:
            m, j = divmod(ch, Csp)
            used = np.unique(c[:, :, :, m])
            assert np.all(D[m][used, j] == 0.0)


def test_ec_conv_1x1_equals_fc(api, dev):
    """A 1x1 kernel (stride 1, no padding) is the FC problem over every pixel:
    the two entry points give the same result."""
    rng = np.random.Generator(np.random.PCG64(8))
    N, Cs, H, W, Ct, Csp, K = 3, 16, 5, 4, 24, 4, 8
    S = np.maximum(rng.standard_normal((N, Cs, H, W)), 0).astype(np.float32)
    T = rng.standard_normal((N, Ct, H, W)).astype(np.float32)
    D0 = (0.2 * rng.standard_normal((Cs // Csp, K, Csp))).astype(np.float32)
    c0 = rng.integers(0, K, (Ct, 1, 1, Cs // Csp)).astype(np.uint8)
    D, c, obj = run_gpu(api, dev, S, T, D0, c0, 1, 0, 1, 2)
    Df, cf = T_(D0, dev), T_(c0[:, 0, 0, :], dev)
    of = api.ec_fc(T_(S.transpose(0, 2, 3, 1).reshape(-1, Cs), dev), T_(T.transpose(0, 2, 3, 1).reshape(-1, Ct), dev),
                   Df, cf, 1, 2)
    torch.cuda.synchronize()
    assert np.array_equal(c[:, 0, 0, :], cf.cpu().numpy())
    assert np.allclose(D, Df.cpu().numpy(), rtol=1e-6, atol=1e-7)
    assert np.allclose(obj, of.cpu().numpy(), rtol=1e-9)


def test_ec_conv_lowers_response_error_of_kmeans(api, dev):
    """From the k-means quantizer of a conv layer (Eq. (6)), one sweep lowers
    the response error (the AlexNet conv3 layer shape on 8 images)."""
    rng = np.random.Generator(np.random.PCG64(9))
    N, Cs, H, Ct, dk, Csp, K = 8, 256, 13, 384, 3, 4, 128
    S = np.maximum(rng.standard_normal((N, Cs, H, H)), 0).astype(np.float32)
    Wt = (0.02 * rng.standard_normal((Ct, Cs, dk, dk))).astype(np.float32)
    Sd, Wd = T_(S, dev), T_(Wt, dev)
    Td = torch.nn.functional.conv2d(Sd, Wd, padding=1)
    D0 = T_((0.02 * rng.standard_normal((Cs // Csp, K, Csp))).astype(np.float32), dev)
    D, codes, _ = api.pq_kmeans(Wd, D0, 3)
    obj = api.ec_conv(Sd, Td.contiguous(), D, codes, 1, 1, 1, 1)
    torch.cuda.synchronize()
    o = obj.cpu().numpy()
    assert np.all(np.diff(o) <= 1e-9 * o[0])
    assert o[-1] < 0.7 * o[0], (o[0], o[-1])
    y = api.conv_forward(Sd, D, codes, 1, 1)
    err = float(((y.double() - Td.double()) ** 2).sum())
    assert abs(err - o[-1]) <= 1e-4 * o[-1], (err, o[-1])


def test_ec_conv_full_size_first_step(api, dev):
    """The AlexNet conv3 shape (256 -> 384, 3x3, pad 1, 13x13, C'_s = 4,
    K = 128) at full layer size on 4 images: after one GPU sweep, subspace 0's
    sub-codebook and codes are those of the first step, which the oracle
    replays from the same start; the first objective entries agree too."""
    from oracle import ec_conv
    rng = np.random.Generator(np.random.PCG64(14))
    N, Cs, H, Ct, dk, Csp, K = 4, 256, 13, 384, 3, 4, 128
    S, T, D0, c0 = problem(rng, N, Cs, H, H, Ct, dk, 1, 1, Csp, K)
    D, c, obj = run_gpu(api, dev, S, T, D0, c0, 1, 1, 1, 1)
    M = Cs // Csp
    S64, T64 = S.astype(np.float64), T.astype(np.float64).reshape(N, Ct, -1)
    Dr = D0.astype(np.float64)
    cm = [c0[:, :, :, m].reshape(Ct, dk * dk) for m in range(M)]
    ss = [ec_conv.shifted(S64[:, m * Csp:(m + 1) * Csp], dk, 1, 1) for m in range(M)]
    Y = sum(ec_conv.contribution(ss[m], Dr[m], cm[m]) for m in range(M))
    h0 = float(np.sum((T64 - Y) ** 2))
    old = ec_conv.contribution(ss[0], Dr[0], cm[0])
    D1, c1 = ec_conv.subspace_step(ss[0], T64 - Y + old, Dr[0], cm[0], 1)
    Y = Y - old + ec_conv.contribution(ss[0], D1, c1)
    h1 = float(np.sum((T64 - Y) ** 2))
    assert np.array_equal(c[:, :, :, 0].reshape(Ct, -1), c1)
    assert np.allclose(D[0], D1, rtol=1e-6, atol=1e-7 * float(np.abs(D1).max()))
    assert np.allclose(obj[:2], [h0, h1], rtol=1e-9), (obj[:2], h0, h1)
