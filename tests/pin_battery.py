"""A compact battery of oracle pins that needs only numpy, run in a child
process against a given build of the oracle (see test_oracle_mutants.py).

Every reference here is independent of the oracle's code: hand-worked values,
a numpy dense convolution / matrix product on kernels rebuilt from the codes
(Eq. (4), (6)), numpy einsum for the table (Sec. 3.1 test phase), and for the
packed indices (Table 1) Python integers and the compression ratios the paper
prints for fc6 (Table 6).
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402
from paper_1512_06473_amd import workloads as wl  # noqa: E402


def dense_conv(x, Wt, stride, pad, bias=None):
    """Plain numpy cross-correlation (float64), one kernel offset at a time."""
    N, Cs, H, W = x.shape
    Ct, _, dk, _ = Wt.shape
    Ho, Wo = (H + 2 * pad - dk) // stride + 1, (W + 2 * pad - dk) // stride + 1
    xp = np.zeros((N, Cs, H + 2 * pad, W + 2 * pad))
    xp[:, :, pad:pad + H, pad:pad + W] = x
    y = np.zeros((N, Ct, Ho, Wo))
    for ky in range(dk):
        for kx in range(dk):
            win = xp[:, :, ky:ky + stride * (Ho - 1) + 1:stride, kx:kx + stride * (Wo - 1) + 1:stride]
            y += np.einsum("tc,nchw->nthw", Wt[:, :, ky, kx], win)
    if bias is not None:
        y += bias[None, :, None, None]
    return y


def rebuilt_conv(D, codes):
    M, K, Csp = D.shape
    Ct, dk, _, _ = codes.shape
    sub = D[np.arange(M)[None, None, None, :], codes.astype(np.int64)]
    return sub.transpose(0, 3, 4, 1, 2).reshape(Ct, M * Csp, dk, dk).astype(np.float64)


def rebuilt_fc(D, codes):
    M = D.shape[0]
    sub = D[np.arange(M)[None, :], codes.astype(np.int64)]
    return sub.reshape(codes.shape[0], -1).astype(np.float64)


def subvectors(W, Csp):
    """Sub-vectors of W [C_t][C_s][d_k][d_k] grouped by subspace:
    [M][C_t d_k d_k][C'_s], in (c_t, ky, kx) order (numpy reshapes only)."""
    Ct, Cs, dk, _ = W.shape
    return W.reshape(Ct, Cs // Csp, Csp, dk, dk).transpose(1, 0, 3, 4, 2).reshape(Cs // Csp, -1, Csp)


def quant_checks(rng):
    out = []
    # K = 1: the single sub-codeword is the mean of every sub-vector (Eq. (4)
    # with one indicator row), the objective the total squared deviation.
    W = rng.standard_normal((5, 6, 3, 3)).astype(np.float32)
    V = subvectors(W.astype(np.float64), 3)
    D, codes, o64 = O.pq_kmeans(W, np.zeros((2, 1, 3), np.float32), 1)
    mean = V.mean(axis=1)
    out.append(("quant K=1 mean", np.allclose(D[:, 0], mean, rtol=1e-6, atol=1e-7) and not codes.any()))
    dev = ((V - mean[:, None, :]) ** 2).sum()
    out.append(("quant K=1 objective", abs(o64[-1] - dev) <= 1e-6 * dev))
    # A pool of R distinct sub-vectors per subspace and the pool among the
    # initial sub-codewords: every sub-vector is matched exactly, error 0.
    Ct, Cs, dk, Csp, K, R = 7, 8, 2, 4, 16, 5
    M = Cs // Csp
    pool = rng.integers(-9, 10, (M, R, Csp)).astype(np.float32)
    pool[:, :, 0] = np.arange(R)[None, :] * 20  # distinct rows
    r = rng.integers(0, R, (M, Ct * dk * dk))
    V = pool[np.arange(M)[:, None], r]  # [M][n][Csp]
    W = V.reshape(M, Ct, dk, dk, Csp).transpose(1, 0, 4, 2, 3).reshape(Ct, Cs, dk, dk)
    D0 = (rng.standard_normal((M, K, Csp)) * 100 + 1000).astype(np.float32)
    perm = rng.permutation(K)[:R]
    D0[:, perm] = pool
    codes, o64 = O.pq_assign(W, D0)
    got = codes.reshape(Ct * dk * dk, M).T
    out.append(("quant exact pool", np.array_equal(got, perm[r]) and o64.sum() == 0.0))
    # Nearest sub-codeword: against float64 distances from numpy.
    for shape in [(9, 12, 3, 4, 16), (33, 8, 1, 2, 64), (4, 6, 5, 3, 7)]:
        Ct, Cs, dk, Csp, K = shape
        W, D = wl.random_quant(rng, Ct, Cs, dk, Csp, K)
        W4 = W.reshape(Ct, Cs, dk, dk)
        codes, o64 = O.pq_assign(W, D)
        V = subvectors(W4.astype(np.float64), Csp)
        dist = ((V[:, :, None, :] - D.astype(np.float64)[:, None, :, :]) ** 2).sum(-1)  # [M][n][K]
        got = codes.reshape(Ct * dk * dk, Cs // Csp).T
        chosen = np.take_along_axis(dist, got[:, :, None].astype(np.int64), 2)[..., 0]
        best = dist.min(-1)
        # float64 on both sides: the chosen distance is the minimum up to the
        # order of C's float64 additions
        out.append(("quant nearest %s" % (shape,), np.all(chosen <= best * (1 + 1e-13) + 1e-300)))
        # and the distances the oracle reports for a given assignment are
        # these same float64 distances
        dcode, dmin = O.pq_distances(W, D, codes)
        out.append(("quant distances %s" % (shape,),
                    np.allclose(dcode.reshape(-1, Cs // Csp).T, chosen, rtol=1e-13, atol=0)
                    and np.allclose(dmin.reshape(-1, Cs // Csp).T, best, rtol=1e-13, atol=0)))
        rec = ((V - D.astype(np.float64)[np.arange(Cs // Csp)[:, None], got]) ** 2).sum(axis=(1, 2))
        out.append(("quant objective = ||DB - W||^2 %s" % (shape,), np.allclose(o64, rec, rtol=1e-10, atol=1e-14)))
        # Update: the mean of each cluster; an unused sub-codeword keeps its value.
        D[:, -1] = 1e3  # far from every sub-vector: never chosen
        codes, _ = O.pq_assign(W, D)
        got = codes.reshape(Ct * dk * dk, Cs // Csp).T
        Dn, cnt = O.pq_update(W, codes, D)
        ok = True
        for m in range(Cs // Csp):
            for k in range(K):
                sel = V[m][got[m] == k]
                ok &= cnt[m, k] == len(sel)
                if len(sel):
                    ok &= np.allclose(Dn[m, k], sel.mean(0), rtol=1e-6, atol=1e-8)
                else:
                    ok &= np.array_equal(Dn[m, k], D[m, k])
        out.append(("quant update means %s" % (shape,), bool(ok) and (cnt[:, -1] == 0).all()))
    # Integer data: distances are exact, so the decision must be numpy's
    # argmin (the first minimum: ties to the lowest index).
    Ct, Cs, dk, Csp, K = 20, 12, 3, 3, 40
    W, D = wl.random_quant(rng, Ct, Cs, dk, Csp, K, integer=True)
    codes, _ = O.pq_assign(W, D)
    V = subvectors(W.astype(np.float64), Csp)
    dist = ((V[:, :, None, :] - D.astype(np.float64)[:, None, :, :]) ** 2).sum(-1)
    out.append(("quant ties to lowest index", np.array_equal(codes.reshape(-1, Cs // Csp).T, dist.argmin(-1))))
    # Lloyd iterations never raise the objective; the final codes are the
    # assignment to the final sub-codewords.
    W, D0 = wl.random_quant(rng, 40, 16, 3, 4, 32)
    D, codes, o64 = O.pq_kmeans(W, D0, 6)
    out.append(("quant objective non-increasing", np.all(np.diff(o64) <= 1e-6 * o64[:-1])))
    c2, _ = O.pq_assign(W, D)
    out.append(("quant final codes match codebooks", np.array_equal(codes, c2)))
    # Eq. (6) = Eq. (4) over the gathered sub-vectors: quantizing a conv layer
    # is quantizing the FC matrix whose rows are its (c_t, p_k) kernels' columns.
    Wf = W.transpose(0, 2, 3, 1).reshape(-1, W.shape[1])
    Df, cf, o64f = O.pq_kmeans(Wf, D0, 6)
    out.append(("quant conv = fc on gathered sub-vectors",
                np.array_equal(D, Df) and np.array_equal(codes.reshape(cf.shape), cf) and np.array_equal(o64, o64f)))
    return out


def _pool_np(h, k, s):
    N, C, H, W = h.shape
    Ho, Wo = (H - k) // s + 1, (W - k) // s + 1
    return np.array([[[[h[n, c, s * i:s * i + k, s * j:s * j + k].max() for j in range(Wo)] for i in range(Ho)]
                      for c in range(C)] for n in range(N)])


def network_checks(rng, Om=None):
    """Pins of the oracle's network composition (oracle.network): the
    hand-worked stack of tests/golden/network_handworked.json, and a random
    conv -> pool -> conv -> pool -> FC -> FC stack against the same layers
    written as numpy dense products on the rebuilt weights (Eq. (4), (6)),
    fp32 rounding of every layer's input, NCHW flatten before the first FC;
    in absolute mode (|x|, |D|, no ReLU) the same composition on magnitudes,
    which bounds |y| elementwise.  ``Om`` replaces the oracle module (a copy
    with a planted mistake)."""
    Om = Om or O
    out = []
    g = json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                                    "network_handworked.json")))
    x = np.array(g["x"], np.float32)
    layers = [dict(kind="conv", D=np.array(g["conv"]["D"], np.float32),
                   codes=np.array(g["conv"]["codes"], np.uint8), stride=1, pad=0, relu=True),
              dict(kind="pool", k=2, s=1),
              dict(kind="fc", D=np.array(g["fc"]["D"], np.float32),
                   codes=np.array(g["fc"]["codes"], np.uint8), relu=False)]
    try:
        out.append(("network hand-worked stack",
                    np.array_equal(Om.network(x, layers), np.array(g["y"], np.float64))))
        out.append(("network hand-worked absolute stack",
                    np.array_equal(Om.network(x, layers, absolute=True), np.array(g["y_absolute"], np.float64))))
    except Exception:
        out.append(("network hand-worked stack", False))

    def reference(xx, specs, absolute):
        h = np.abs(xx).astype(np.float64) if absolute else xx.astype(np.float64)
        for L in specs:
            h = h.astype(np.float32).astype(np.float64)  # fp32 input of every layer
            if L["kind"] == "pool":
                h = _pool_np(h, L["k"], L["s"])
                continue
            D = np.abs(L["D"]) if absolute else L["D"]
            if L["kind"] == "conv":
                h = dense_conv(h, rebuilt_conv(D, L["codes"]), L["stride"], L["pad"])
            else:
                h = h.reshape(h.shape[0], -1) @ rebuilt_fc(D, L["codes"]).T
            if L["relu"] and not absolute:
                h = np.maximum(h, 0.0)
        return h

    Ls = []
    # 9x9 -> conv p1 9x9 -> pool 3/2 4x4 -> conv p0 2x2 -> pool 2/1 1x1 -> fc 8 -> fc 3
    for (Cs, Ct, p, Csp, K, pk, ps) in [(4, 6, 1, 2, 8, 3, 2), (6, 8, 0, 3, 16, 2, 1)]:
        Ls.append(dict(kind="conv", D=(0.3 * rng.standard_normal((Cs // Csp, K, Csp))).astype(np.float32),
                       codes=rng.integers(0, K, (Ct, 3, 3, Cs // Csp)).astype(np.uint8), stride=1, pad=p,
                       relu=True))
        Ls.append(dict(kind="pool", k=pk, s=ps))
    for (Cs, Ct, Csp, K, relu) in [(8, 10, 2, 4, True), (10, 3, 5, 8, False)]:
        Ls.append(dict(kind="fc", D=(0.3 * rng.standard_normal((Cs // Csp, K, Csp))).astype(np.float32),
                       codes=rng.integers(0, K, (Ct, Cs // Csp)).astype(np.uint8), relu=relu))
    x = rng.standard_normal((3, 4, 9, 9)).astype(np.float32)
    # a spatial FC input too: conv -> pool 2x2 map -> fc, where the flatten order matters
    Ls2 = [dict(kind="conv", D=(0.3 * rng.standard_normal((2, 8, 2))).astype(np.float32),
                codes=rng.integers(0, 8, (3, 3, 3, 2)).astype(np.uint8), stride=1, pad=1, relu=True),
           dict(kind="pool", k=3, s=2),
           dict(kind="fc", D=(0.3 * rng.standard_normal((4, 8, 3))).astype(np.float32),
                codes=rng.integers(0, 8, (5, 4)).astype(np.uint8), relu=False)]
    x2 = rng.standard_normal((2, 4, 5, 5)).astype(np.float32)
    for name, xx, specs in [("network stack", x, Ls), ("network spatial flatten", x2, Ls2)]:
        try:
            y = Om.network(xx, specs)
            A = Om.network(xx, specs, absolute=True)
            r, ra = reference(xx, specs, False), reference(xx, specs, True)
            # intermediate fp32 roundings may land one unit apart: 1e-6 of the magnitude sum
            out.append((name + " = numpy composition",
                        y.shape == r.shape and bool(np.all(np.abs(y - r) <= 1e-6 * ra + 1e-12))))
            out.append((name + " absolute = numpy composition on magnitudes",
                        A.shape == ra.shape and bool(np.all(np.abs(A - ra) <= 1e-6 * ra + 1e-12))))
            out.append((name + " absolute bounds |y|", bool(np.all(np.abs(y) <= A * (1 + 1e-6) + 1e-12))))
        except Exception:
            out.append((name + " = numpy composition", False))
    return out


def pack_checks(rng):
    """Packed quantization indices (Table 1: log2 K bits each; reading R6b)."""
    out = []
    gold = json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "packed_codes.json")))
    for c in gold["cases"]:
        got = O.pack_codes(np.array(c["codes"], np.uint8), c["K"])
        out.append(("packed hand-worked K=%d" % c["K"], got.tolist() == c["bytes"]))
        back = O.unpack_codes(np.array(c["bytes"], np.uint8), len(c["codes"]), c["K"])
        out.append(("unpacked hand-worked K=%d" % c["K"], back.tolist() == c["codes"]))
    for K in [1, 2, 3, 5, 16, 31, 32, 33, 64, 100, 127, 128, 129, 200, 255, 256]:
        n = int(rng.integers(1, 300))
        codes = rng.integers(0, K, n).astype(np.uint8)
        b = max(K - 1, 0).bit_length()
        # the stream as one integer, sum code_i 2^(i b), in little-endian bytes
        ref = sum(int(v) << (i * b) for i, v in enumerate(codes)).to_bytes((n * b + 7) // 8, "little")
        got = O.pack_codes(codes, K)
        out.append(("packed big-int K=%d" % K, bytes(got.tobytes()) == ref))
        out.append(("packed round trip K=%d" % K, np.array_equal(O.unpack_codes(got, n, K), codes)))
    # the code bytes of Table 1 reproduce the paper's printed compression of
    # CaffeNet fc6 (Table 6) when the index array is really packed
    for csp, K, printed in [(2, 16, 15.06), (3, 16, 21.94), (3, 32, 16.70), (4, 32, 21.33)]:
        M = 9216 // csp
        nbytes = O.pack_codes(np.zeros(4096 * M, np.uint8), K).size
        r = 4.0 * 9216 * 4096 / (4.0 * 9216 * K + nbytes)
        out.append(("packed fc6 compression %d/%d" % (csp, K), abs(r - printed) <= 0.005))
    return out


def ec_checks(rng, E=None):
    """Error correction for a FC layer (Sec. 3.3.1, Eq. (8)-(12)); E is the
    module under test (default: the oracle's)."""
    if E is None:
        from oracle import ec as E
    out = []
    # Eq. (8) with S = I is || W - D B ||^2 column by column: one round of
    # (sub-codebook, assignment) update is a k-means update then an
    # assignment (Eq. (4)).  Well separated clusters, so no decision is close.
    Ct, Cs, Csp, K = 60, 12, 4, 5
    M = Cs // Csp
    centers = rng.standard_normal((M, K, Csp)) * 10
    lab = rng.integers(0, K, (Ct, M))
    W = np.stack([centers[m][lab[:, m]] for m in range(M)], 1).reshape(Ct, Cs)
    W = (W + 0.01 * rng.standard_normal(W.shape)).astype(np.float32)
    D0 = (centers + rng.standard_normal(centers.shape)).astype(np.float32)
    c0, _ = O.pq_assign(W, D0)
    D, codes, hist = E.ec_fc(np.eye(Cs), W.T.astype(np.float64), D0, c0, sweeps=1, inner=1)
    D1, _ = O.pq_update(W, c0, D0)
    c1, _ = O.pq_assign(W, D1)
    out.append(("ec S=I sub-codebooks = k-means update", np.allclose(D, D1, rtol=1e-6, atol=1e-6)))
    out.append(("ec S=I assignment = k-means assignment", np.array_equal(codes, c1)))
    # general inputs
    N, Cs, Ct, Csp, K = 40, 12, 30, 3, 6
    M = Cs // Csp
    S = rng.standard_normal((N, Cs))
    Wt = rng.standard_normal((Ct, Cs))
    T = S @ Wt.T + 0.1 * rng.standard_normal((N, Ct))
    D0 = rng.standard_normal((M, K, Csp))
    c0 = rng.integers(0, K, (Ct, M)).astype(np.uint8)
    D, codes, hist = E.ec_fc(S, T, D0, c0, sweeps=2, inner=2)
    out.append(("ec objective non-increasing", bool(np.all(np.diff(hist) <= 1e-9 * hist[0]))))
    out.append(("ec objective decreases", hist[-1] < 0.9 * hist[0]))
    What = np.stack([D[m][codes[:, m]] for m in range(M)], 1).reshape(Ct, Cs)
    out.append(("ec objective = response error", abs(float(np.sum((T - S @ What.T) ** 2)) - hist[-1])
                <= 1e-9 * hist[0]))
    # one subspace step against library least squares and a brute-force argmin
    m = 1
    Sm = S[:, m * Csp:(m + 1) * Csp]
    R = rng.standard_normal((N, Ct))
    Dm, cm = E.subspace_step(Sm, R, D0[m], c0[:, m], inner=1)
    ok = True
    for k in range(K):
        Lk = np.flatnonzero(c0[:, m] == k)
        if Lk.size:
            A = np.vstack([Sm] * Lk.size)
            bb = np.concatenate([R[:, c] for c in Lk])
            ok &= np.allclose(Dm[k], np.linalg.lstsq(A, bb, rcond=None)[0], rtol=1e-9, atol=1e-12)
        else:
            ok &= np.array_equal(Dm[k], D0[m][k])
    out.append(("ec sub-codebook = least squares (lstsq)", bool(ok)))
    brute = np.array([np.argmin([np.sum((R[:, c] - Sm @ Dm[k]) ** 2) for k in range(K)]) for c in range(Ct)])
    out.append(("ec assignment = brute-force Eq. (12)", np.array_equal(cm, brute)))
    # a channel that is zero on every image: its coordinate of every updated
    # sub-codeword is 0 (reading E4), and the fit equals least squares
    S2 = S.copy()
    S2[:, m * Csp + 1] = 0.0
    Sm2 = S2[:, m * Csp:(m + 1) * Csp]
    Dz, _ = E.subspace_step(Sm2, R, D0[m], c0[:, m], inner=1)
    used = np.unique(c0[:, m])
    out.append(("ec dead channel gives a zero coordinate", bool(np.all(Dz[used, 1] == 0.0))))
    ok = True
    for k in used:
        Lk = np.flatnonzero(c0[:, m] == k)
        ok &= np.allclose(Dz[k], np.linalg.lstsq(np.vstack([Sm2] * Lk.size),
                                                 np.concatenate([R[:, c] for c in Lk]), rcond=None)[0],
                          rtol=1e-9, atol=1e-12)
    out.append(("ec dead channel fit = min-norm least squares", bool(ok)))
    # an exact quantized layer stays exact
    Dt = rng.standard_normal((M, K, Csp))
    ct = rng.integers(0, K, (Ct, M)).astype(np.uint8)
    Wq = np.stack([Dt[m][ct[:, m]] for m in range(M)], 1).reshape(Ct, Cs)
    D, codes, hist = E.ec_fc(S, S @ Wq.T, Dt, ct, sweeps=1, inner=1)
    out.append(("ec lossless start stays lossless", hist[-1] <= 1e-18 * float(np.sum((S @ Wq.T) ** 2)) + 1e-20
                and np.array_equal(codes, ct)))
    return out


def _bf_patch(Sm, n, yo, xo, ky, kx, stride, pad):
    """The input sub-vector at p_s = p_t s - pad + p_k, or 0 outside."""
    y, x = yo * stride - pad + ky, xo * stride - pad + kx
    if 0 <= y < Sm.shape[2] and 0 <= x < Sm.shape[3]:
        return Sm[n, :, y, x].astype(np.float64)
    return np.zeros(Sm.shape[1])


def _bf_channel(Sm, Dm, codes_c, dk, stride, pad, Ho, Wo, skip=()):
    """One channel's response of subspace m, [N][H_o][W_o], by loops: the sum
    over kernel positions (except those in `skip`) of D_{code}^T S_{p_s}."""
    N = Sm.shape[0]
    out = np.zeros((N, Ho, Wo))
    for n in range(N):
        for yo in range(Ho):
            for xo in range(Wo):
                for ky in range(dk):
                    for kx in range(dk):
                        if ky * dk + kx not in skip:
                            out[n, yo, xo] += Dm[codes_c[ky * dk + kx]] @ _bf_patch(Sm, n, yo, xo, ky, kx,
                                                                                     stride, pad)
    return out


def ec_conv_checks(rng, E=None):
    """Error correction for a conv layer (Sec. 3.3.2 Eq. (13), App. B Eq.
    (14)-(21)); E is the module under test (default: the oracle's)."""
    if E is None:
        from oracle import ec_conv as E
    from oracle import ec as F
    out = []
    # the quantized response equals the C oracle's conv forward (Eq. (7))
    ok = True
    for (N, Cs, H, W, Ct, dk, st, pd, Csp, K) in [(2, 6, 7, 6, 5, 3, 1, 1, 3, 4), (1, 4, 9, 8, 3, 3, 2, 2, 2, 5),
                                                  (2, 4, 5, 5, 4, 2, 1, 0, 4, 3)]:
        S = rng.standard_normal((N, Cs, H, W)).astype(np.float32)
        D = rng.standard_normal((Cs // Csp, K, Csp)).astype(np.float32)
        c = rng.integers(0, K, (Ct, dk, dk, Cs // Csp)).astype(np.uint8)
        ok &= np.allclose(E.forward(S, D, c, st, pd), O.conv_direct(S, D, c, st, pd), rtol=1e-12, atol=1e-12)
    out.append(("ec conv response = C oracle conv", bool(ok)))
    # a 1x1 kernel (stride 1, no padding) is the FC case over every pixel
    N, Cs, H, W, Ct, Csp, K = 3, 8, 3, 2, 7, 2, 4
    M = Cs // Csp
    S = rng.standard_normal((N, Cs, H, W))
    T = rng.standard_normal((N, Ct, H, W))
    D0 = rng.standard_normal((M, K, Csp))
    c0 = rng.integers(0, K, (Ct, 1, 1, M)).astype(np.uint8)
    D, codes, hist = E.ec_conv(S, T, D0, c0, 1, 0, sweeps=2, inner=2)
    Df, cf, hf = F.ec_fc(S.transpose(0, 2, 3, 1).reshape(-1, Cs), T.transpose(0, 2, 3, 1).reshape(-1, Ct),
                         D0, c0[:, 0, 0, :], sweeps=2, inner=2)
    out.append(("ec conv 1x1 = FC over pixels: codes", np.array_equal(codes[:, 0, 0, :], cf)))
    out.append(("ec conv 1x1 = FC over pixels: sub-codebooks", np.allclose(D, Df, rtol=1e-9, atol=1e-12)))
    out.append(("ec conv 1x1 = FC over pixels: objective", np.allclose(hist, hf, rtol=1e-9)))
    # one subspace: the codebook update against least squares built by loops
    # (sub-codewords in order, each with the latest others), and the
    # assignment update against every candidate's error for that channel
    # (inputs with a strong per-channel mean, so that neighbouring kernel
    # positions see correlated inputs and one position's code moves the
    # best code of another)
    N, Csp, H, W, Ct, dk, st, pd, K = 2, 2, 4, 5, 8, 2, 1, 1, 3
    Sm = 0.3 * rng.standard_normal((N, Csp, H, W)) + rng.standard_normal((1, Csp, 1, 1))
    Ho, Wo = (H + 2 * pd - dk) // st + 1, (W + 2 * pd - dk) // st + 1
    R = rng.standard_normal((N, Ct, Ho, Wo))
    Dm0 = rng.standard_normal((K, Csp))
    cm = rng.integers(0, K, (Ct, dk * dk)).astype(np.uint8)
    cm[0, :2] = 1  # a channel with two positions on one sub-codeword
    s = E.shifted(Sm, dk, st, pd)
    Rf = R.reshape(N, Ct, -1)
    Dg = E.update_codebook(s, Rf, Dm0.copy(), cm)
    Db = Dm0.copy()
    for k in range(K):
        rows, rhs = [], []
        for c in range(Ct):
            mine = [p for p in range(dk * dk) if cm[c, p] == k]
            if not mine:
                continue
            Q = R[:, c] - _bf_channel(Sm, Db, cm[c], dk, st, pd, Ho, Wo, skip=mine)
            for n in range(N):
                for yo in range(Ho):
                    for xo in range(Wo):
                        rows.append(sum(_bf_patch(Sm, n, yo, xo, p // dk, p % dk, st, pd) for p in mine))
                        rhs.append(Q[n, yo, xo])
        if rows:
            Db[k] = np.linalg.lstsq(np.array(rows), np.array(rhs), rcond=None)[0]
    out.append(("ec conv codebook update = sequential least squares", np.allclose(Dg, Db, rtol=1e-9, atol=1e-12)))
    cg = E.update_assignment(s, Rf, Dg.copy(), cm.copy())
    cb = cm.copy()
    for p in range(dk * dk):
        for c in range(Ct):
            errs = []
            for k in range(K):
                trial = cb[c].copy()
                trial[p] = k
                errs.append(np.sum((R[:, c] - _bf_channel(Sm, Dg, trial, dk, st, pd, Ho, Wo)) ** 2))
            cb[c, p] = int(np.argmin(errs))
    out.append(("ec conv assignment update = brute force, positions in order", np.array_equal(cg, cb)))
    # whole descent: monotone, ends at the response error it reports
    N, Cs, H, W, Ct, dk, st, pd, Csp, K = 2, 6, 6, 5, 5, 3, 1, 1, 3, 4
    M = Cs // Csp
    S = rng.standard_normal((N, Cs, H, W))
    Wt = rng.standard_normal((Ct, Cs, dk, dk))
    T = dense_conv(S, Wt, st, pd) + 0.1 * rng.standard_normal((N, Ct, H, W))
    D0 = rng.standard_normal((M, K, Csp))
    c0 = rng.integers(0, K, (Ct, dk, dk, M)).astype(np.uint8)
    D, codes, hist = E.ec_conv(S, T, D0, c0, st, pd, sweeps=2, inner=1)
    out.append(("ec conv objective non-increasing", bool(np.all(np.diff(hist) <= 1e-9 * hist[0]))))
    out.append(("ec conv objective decreases", hist[-1] < 0.9 * hist[0]))
    Y = dense_conv(S, rebuilt_conv(D, codes), st, pd)
    out.append(("ec conv objective = response error", abs(float(np.sum((T - Y) ** 2)) - hist[-1])
                <= 1e-9 * hist[0]))
    # an exactly quantized layer stays exact
    Dt = rng.standard_normal((M, K, Csp))
    ct = rng.integers(0, K, (Ct, dk, dk, M)).astype(np.uint8)
    Tq = dense_conv(S, rebuilt_conv(Dt, ct), st, pd)
    D, codes, hist = E.ec_conv(S, Tq, Dt, ct, st, pd, sweeps=1, inner=1)
    out.append(("ec conv lossless start stays lossless",
                hist[-1] <= 1e-18 * float(np.sum(Tq ** 2)) + 1e-20 and np.array_equal(codes, ct)))
    # an input channel that is zero everywhere: its coordinate of every
    # updated sub-codeword is 0 (pivot rule)
    S2 = S.copy()
    S2[:, 1] = 0.0
    D, codes, hist = E.ec_conv(S2, T, D0, c0, st, pd, sweeps=1, inner=1)
    used = np.unique(codes[:, :, :, 0])
    out.append(("ec conv dead channel gives a zero coordinate", bool(np.all(D[0][used, 1] == 0.0))))
    return out


def small_network(rng, lossless=False):
    """A conv -> pool -> conv -> FC stack with synthetic weights (and, with
    lossless, weights that are exactly quantized by their D0 and codes)."""
    specs = []
    shapes = [("conv", 6, 4, 3, 1, 1, 2, 4), ("pool", 2, 2), ("conv", 8, 6, 3, 1, 1, 3, 4), ("fc", 5, 8 * 3 * 3, 1, 0, 0, 4, 4)]
    for sh in shapes:
        if sh[0] == "pool":
            specs.append({"kind": "pool", "k": sh[1], "s": sh[2]})
            continue
        kind, Ct, Cs, dk, st, pd, Csp, K = sh
        M = Cs // Csp
        D0 = (0.5 * rng.standard_normal((M, K, Csp))).astype(np.float32)
        if lossless:
            codes = rng.integers(0, K, (Ct, dk, dk, M)).astype(np.uint8)
            W = rebuilt_conv(D0, codes).astype(np.float32)
        else:
            W = (0.5 * rng.standard_normal((Ct, Cs, dk, dk))).astype(np.float32)
        spec = {"kind": kind, "W": W if kind == "conv" else W.reshape(Ct, Cs), "D0": D0,
                "bias": (0.1 * rng.standard_normal(Ct)).astype(np.float32), "relu": kind == "conv"}
        if kind == "conv":
            spec.update(stride=st, pad=pd)
        specs.append(spec)
    x = np.maximum(rng.standard_normal((3, 4, 6, 6)), 0).astype(np.float32)
    return x, specs


def ec_network_checks(rng, E=None):
    """Multi-layer error correction (Sec. 3.3.3); E is the module under test
    (default: the oracle's)."""
    if E is None:
        from oracle import ec_network as E
    out = []
    x, specs = small_network(rng)
    res = E.quantize_network(x, specs, sweeps=1, inner=1, kmeans_iters=2)
    # layer 1: S is the input and T its original linear response
    D, codes, hist, S, T = res[0]
    out.append(("ecn layer 1 S = input", np.array_equal(S, x)))
    W1 = specs[0]["W"].astype(np.float64)
    out.append(("ecn layer 1 T = W * x", np.allclose(T, dense_conv(x.astype(np.float64), W1, 1, 1), rtol=1e-6,
                                                    atol=1e-6)))
    # layer 2: S = max-pool of layer 1's quantized forward (C oracle), T = W2
    # times the pooled original activations (bias, ReLU)
    h1q = O.conv_lut(x, D.astype(np.float32), codes, 1, 1, bias=specs[0]["bias"], relu=True).astype(np.float32)
    S2 = O.maxpool(h1q, 2, 2).astype(np.float32)
    h1o = np.maximum(dense_conv(x.astype(np.float64), W1, 1, 1) + specs[0]["bias"][None, :, None, None], 0)
    S2o = O.maxpool(h1o.astype(np.float32), 2, 2)
    D2, codes2, hist2, S_2, T_2 = res[2]
    out.append(("ecn layer 2 S = pooled quantized forward", np.array_equal(S_2, S2)))
    out.append(("ecn layer 2 T = W2 * pooled original activations",
                np.allclose(T_2, dense_conv(S2o.astype(np.float64), specs[2]["W"].astype(np.float64), 1, 1),
                            rtol=1e-6, atol=1e-6)))
    # layer 3 (FC) on the flattened quantized activations
    h2q = O.conv_lut(S2, D2.astype(np.float32), codes2, 1, 1, bias=specs[2]["bias"], relu=True).astype(np.float32)
    out.append(("ecn FC S = flattened quantized activations", np.array_equal(res[3][3], h2q.reshape(3, -1))))
    out.append(("ecn objectives non-increasing",
                all(np.all(np.diff(r[2]) <= 1e-9 * r[2][0]) for r in res if r is not None)))
    # every layer's codes are those of error correction from k-means on W
    D1k, c1k, _ = O.pq_kmeans(specs[0]["W"], specs[0]["D0"], 2)
    from oracle import ec_conv as EC
    Dr, cr, hr = EC.ec_conv(x, T, D1k, c1k, 1, 1, 1, 1)
    out.append(("ecn layer 1 = k-means then conv error correction", np.array_equal(cr, codes) and
                np.allclose(Dr, D, rtol=1e-12, atol=1e-15)))
    # weights that their D0 quantizes exactly: every layer stays lossless and
    # the quantized network's activations equal the original's
    x, specs = small_network(rng, lossless=True)
    res = E.quantize_network(x, specs, sweeps=1, inner=1, kmeans_iters=2)
    ok = True
    for r, spec in zip(res, specs):
        if r is not None:
            ok &= r[2][-1] <= 1e-12 * max(float(np.sum(r[4].astype(np.float64) ** 2)), 1e-30)
    out.append(("ecn lossless network stays lossless", bool(ok)))
    return out


def checks():
    out = []
    # hand-worked (see test_oracle.py for the arithmetic)
    x = np.array([[[[1, 2, 0], [0, 1, 3], [2, 0, 1]], [[0, 1, 1], [2, 0, 0], [1, 1, 2]]]], np.float32)
    D = np.array([[[2], [-1]], [[1], [3]]], np.float32)
    c = np.zeros((1, 2, 2, 2), np.uint8)
    c[0, 0, 0], c[0, 0, 1], c[0, 1, 0], c[0, 1, 1] = [0, 1], [1, 0], [1, 1], [0, 0]
    out.append(("hand conv", np.array_equal(O.conv_lut(x, D, c, 1, 0), [[[[9, 13], [7, 6]]]])))
    x = np.arange(1, 10, dtype=np.float32).reshape(1, 1, 3, 3)
    c = np.zeros((1, 3, 3, 1), np.uint8)
    c[0, 1, 1, 0] = 1
    b = np.array([-4], np.float32)
    out.append(("hand conv s2p1", np.array_equal(
        O.conv_lut(x, np.array([[[1], [-2]]], np.float32), c, 2, 1, bias=b, relu=True),
        [[[[5, 3], [0, 0]]]])))
    out.append(("hand fc", np.array_equal(
        O.fc_lut(np.array([[1, 2, 3, 4]], np.float32),
                 np.array([[[1, 0], [0, 1]], [[1, 1], [2, -1]]], np.float32),
                 np.array([[0, 1], [1, 0]], np.uint8)), [[3, 9]])))
    rng = np.random.Generator(np.random.PCG64(1234))
    for shape in [(2, 8, 7, 6, 5, 3, 1, 1, 4, 16), (1, 6, 9, 7, 3, 3, 2, 1, 3, 8),
                  (1, 3, 15, 15, 2, 7, 4, 0, 3, 16), (1, 8, 6, 6, 3, 5, 1, 2, 4, 32)]:
        N, Cs, H, W, Ct, dk, s, p, Csp, K = shape
        x, D, codes = wl.random_conv(rng, N, Cs, H, W, Ct, dk, s, p, Csp, K)
        bias = rng.standard_normal(Ct).astype(np.float32)
        ref = dense_conv(x.astype(np.float64), rebuilt_conv(D, codes), s, p, bias.astype(np.float64))
        y, A = O.conv_lut(x, D, codes, s, p, bias=bias, with_bound=True)
        out.append(("conv lut %s" % (shape,), y.shape == ref.shape and np.allclose(y, ref, rtol=1e-11, atol=1e-11)))
        out.append(("conv direct %s" % (shape,),
                    np.allclose(O.conv_direct(x, D, codes, s, p, bias=bias), ref, rtol=1e-11, atol=1e-11)))
        Aref = dense_conv(np.abs(x).astype(np.float64), np.abs(rebuilt_conv(D, codes)), s, p,
                          np.abs(bias).astype(np.float64))
        out.append(("conv bound %s" % (shape,), np.allclose(A, Aref, rtol=1e-11, atol=1e-11)))
        pts = np.array([[0, Ct - 1, y.shape[2] - 1, 0], [N - 1, 0, 0, y.shape[3] - 1]], np.int32)
        v, a = O.conv_points(x, D, codes, pts, s, p, bias=bias)
        out.append(("conv points %s" % (shape,), np.allclose(v, ref[tuple(pts.T)], rtol=1e-11, atol=1e-11)
                    and np.allclose(a, Aref[tuple(pts.T)], rtol=1e-11, atol=1e-11)))
    x, D, _ = wl.random_conv(rng, 2, 12, 4, 5, 1, 1, 1, 0, 3, 7)
    L = O.lut(x, D)
    want = np.einsum("mkj,nmjhw->nmkhw", D.astype(np.float64), x.astype(np.float64).reshape(2, 4, 3, 4, 5))
    out.append(("lut einsum", np.allclose(L, want, rtol=1e-12, atol=1e-12)))
    for (N, Cs, Ct, Csp, K) in [(3, 12, 7, 4, 8), (2, 9, 5, 3, 32)]:
        x, D, codes = wl.random_fc(rng, N, Cs, Ct, Csp, K)
        bias = rng.standard_normal(Ct).astype(np.float32)
        ref = x.astype(np.float64) @ rebuilt_fc(D, codes).T + bias
        y, A = O.fc_lut(x, D, codes, bias=bias, with_bound=True)
        out.append(("fc lut", np.allclose(y, ref, rtol=1e-11, atol=1e-11)))
        out.append(("fc direct", np.allclose(O.fc_direct(x, D, codes, bias=bias), ref, rtol=1e-11, atol=1e-11)))
        Aref = np.abs(x).astype(np.float64) @ np.abs(rebuilt_fc(D, codes)).T + np.abs(bias)
        out.append(("fc bound", np.allclose(A, Aref, rtol=1e-11, atol=1e-11)))
        pts = np.array([[N - 1, Ct - 1], [0, 1]], np.int32)
        v, a = O.fc_points(x, D, codes, pts, bias=bias)
        out.append(("fc points", np.allclose(v, ref[tuple(pts.T)], rtol=1e-11, atol=1e-11)))
    xm = rng.standard_normal((1, 2, 7, 9)).astype(np.float32)
    ym = O.maxpool(xm, 3, 2)
    ref = np.array([[[[xm[0, ch, 2 * i:2 * i + 3, 2 * j:2 * j + 3].max() for j in range(4)] for i in range(3)]
                     for ch in range(2)]])
    out.append(("maxpool", np.array_equal(ym, ref)))
    out += quant_checks(rng)
    out += network_checks(rng)
    out += pack_checks(rng)
    out += ec_checks(rng)
    return out


def run(libpath=None):
    if libpath:
        O.use(O.load(libpath))
    res = checks()
    bad = [name for name, ok in res if not ok]
    for name in bad:
        print("FAILED:", name)
    return 1 if bad else 0


if __name__ == "__main__":
    sys.exit(run(sys.argv[1] if len(sys.argv) > 1 else None))
