"""Error-corrected quantization of a convolutional layer -- TEST
INFRASTRUCTURE ONLY (imported by tests/ and nothing in the product package).

Paper: Wu et al., "Quantized Convolutional Neural Networks for Mobile
Devices", CVPR 2016, Sec. 3.3.2 (Eq. (13)) and Appendix B (Eq. (14)-(21)).
With the input feature maps S_n and desired responses T_n of a conv layer on
N images, the sub-codebooks D^(m) (shared by every kernel position p_k) and
the assignments B^(m)_{p_k} minimise

    sum_{n, p_t} || sum_{(p_k, p_s)} sum_m (D^(m) B^(m)_{p_k})^T S^(m)_{n, p_s} - T_{n, p_t} ||^2

by block coordinate descent over the subspaces.  For subspace m the residual
of the others is R^(m) (Eq. (15)), and Eq. (16) is minimised by

  * the sub-codebook update: the sub-codewords one after another (k = 0 ..
    K-1, each with the latest values of the others); for sub-codeword k the
    residual Q_k (Eq. (18)) takes out of R^(m) the contribution of every
    kernel position whose sub-codeword is not k, and D_k is the least-squares
    fit of Eq. (19) to Q_k over the images, output positions and channels;
  * the assignment update: the kernel positions one after another (p_k in
    row-major (ky, kx) order, each with the latest assignments of the
    others); for position p_k the residual P_{p_k} (Eq. (20)) takes out of
    R^(m) the contribution of every other position, and each channel takes
    the sub-codeword of least squared error (Eq. (21)), tried exhaustively.

Everything is float64, computed from the definitions on dense arrays (no
Gram-matrix shortcuts).  Readings of what the appendix leaves open or
garbles (C1-C4 in the design notes; E1-E4 and E6 of the FC case carry over):
  C1 Eq. (18) uses c_t both free and summed: Q_k(c_t) = R(c_t) minus, for
     the kernel positions p_k whose sub-codeword for channel c_t is not k,
     D_{k(c_t, p_k)}^T S_{n, p_s}; Eq. (19) sums the squared error over every
     channel that has at least one position coded k (for the others it does
     not depend on D_k);
  C2 Eq. (20) reads "p'_k != p_k", with p'_s the input position paired with
     p'_k; the error of Eq. (21) is summed over n and p_t;
  C3 p_s = p_t s - pad + p_k (cross-correlation, the forward's reading R2);
     positions outside the input hold S = 0 (R3);
  C4 the least squares of Eq. (19) is solved through its normal equations
     with the elimination and pivot rule of the FC case (E4), the scale
     being the largest diagonal entry of its normal matrix; a sub-codeword
     that no position of any channel uses keeps its value; Eq. (21) ties go
     to the lowest k.
"""
from __future__ import annotations

import numpy as np

from oracle.ec import solve_normal


def out_size(n, k, stride, pad):
    return (n + 2 * pad - k) // stride + 1


def shifted(Sm, dk, stride, pad):
    """s[n][o][p][j] = S^(m)[n][j][yo s - pad + ky][xo s - pad + kx] (0 outside
    the input), o = yo W_o + xo, p = ky d_k + kx: the input sub-vector that
    kernel position p meets at output position o (C3)."""
    N, Csp, H, W = Sm.shape
    Ho, Wo = out_size(H, dk, stride, pad), out_size(W, dk, stride, pad)
    Sp = np.zeros((N, Csp, H + 2 * pad + dk, W + 2 * pad + dk), np.float64)
    Sp[:, :, pad:pad + H, pad:pad + W] = Sm
    s = np.zeros((N, Ho * Wo, dk * dk, Csp), np.float64)
    for ky in range(dk):
        for kx in range(dk):
            win = Sp[:, :, ky:ky + (Ho - 1) * stride + 1:stride, kx:kx + (Wo - 1) * stride + 1:stride]
            s[:, :, ky * dk + kx, :] = win.reshape(N, Csp, Ho * Wo).transpose(0, 2, 1)
    return s


def contribution(s, Dm, codes_m, positions=None):
    """sum over kernel positions p (all, or those listed) of
    D^(m)_{k(c, p)}^T s_p: [N][C_t][O].  codes_m [C_t][P]."""
    N, O, P, Csp = s.shape
    Ct = codes_m.shape[0]
    out = np.zeros((N, Ct, O), np.float64)
    for p in (range(P) if positions is None else positions):
        out += np.einsum("noj,cj->nco", s[:, :, p, :], Dm[codes_m[:, p]])
    return out


def update_codebook(s, R, Dm, codes_m):
    """Eq. (17)-(19), the sub-codewords in order (C1, C4).  Updates Dm."""
    N, O, P, Csp = s.shape
    K = Dm.shape[0]
    for k in range(K):
        mine = codes_m == k                                 # [C_t][P]
        chans = np.flatnonzero(mine.any(axis=1))
        if chans.size == 0:
            continue
        A_rows, Q_rows = [], []
        for c in chans:
            A = s[:, :, mine[c], :].sum(axis=2)             # [N][O][C's]
            other = np.flatnonzero(~mine[c])
            Q = R[:, c, :].copy()
            for p in other:                                 # Eq. (18)
                Q -= s[:, :, p, :] @ Dm[codes_m[c, p]]
            A_rows.append(A.reshape(-1, Csp))
            Q_rows.append(Q.reshape(-1))
        A = np.vstack(A_rows)
        Q = np.concatenate(Q_rows)
        Dm[k] = solve_normal(A.T @ A, A.T @ Q)              # Eq. (19)
    return Dm


def update_assignment(s, R, Dm, codes_m):
    """Eq. (20)-(21), the kernel positions in order (C2).  Updates codes_m."""
    N, O, P, Csp = s.shape
    K = Dm.shape[0]
    Ct = codes_m.shape[0]
    for p in range(P):
        for c in range(Ct):
            Pp = R[:, c, :].copy()                          # Eq. (20)
            for q in range(P):
                if q != p:
                    Pp -= s[:, :, q, :] @ Dm[codes_m[c, q]]
            err = [float(np.sum((s[:, :, p, :] @ Dm[k] - Pp) ** 2)) for k in range(K)]
            codes_m[c, p] = int(np.argmin(err))             # Eq. (21), first minimum
    return codes_m


def subspace_step(s, R, Dm, codes_m, inner=1):
    """Eq. (16)-(21) for one subspace: s from shifted(), R [N][C_t][O]
    (Eq. (15)), Dm [K][C's], codes_m [C_t][P].  Returns updated copies."""
    Dm = np.array(Dm, dtype=np.float64, copy=True)
    codes_m = np.array(codes_m, dtype=np.uint8, copy=True)
    for _ in range(inner):
        update_codebook(s, R, Dm, codes_m)
        update_assignment(s, R, Dm, codes_m)
    return Dm, codes_m


def forward(S, D, codes, stride, pad):
    """The quantized layer's response [N][C_t][H_o][W_o] (the left sum of
    Eq. (14)); codes [C_t][d_k][d_k][M]."""
    N, Cs, H, W = S.shape
    M, K, Csp = D.shape
    Ct, dk = codes.shape[0], codes.shape[1]
    Ho, Wo = out_size(H, dk, stride, pad), out_size(W, dk, stride, pad)
    Y = np.zeros((N, Ct, Ho * Wo), np.float64)
    for m in range(M):
        s = shifted(S[:, m * Csp:(m + 1) * Csp], dk, stride, pad)
        Y += contribution(s, D[m], codes[:, :, :, m].reshape(Ct, dk * dk))
    return Y.reshape(N, Ct, Ho, Wo)


def ec_conv(S, T, D0, codes0, stride, pad, sweeps=1, inner=1):
    """Error-corrected quantization of a conv layer (Eq. (13)-(21)).

    S [N][C_s][H][W], T [N][C_t][H_o][W_o] (fp32 or fp64), D0 [M][K][C's],
    codes0 [C_t][d_k][d_k][M].  Returns (D float64, codes uint8 in the same
    layouts, objective history: Eq. (14) at the start and after every
    subspace step)."""
    S = np.asarray(S, np.float64)
    T = np.asarray(T, np.float64)
    D = np.array(D0, dtype=np.float64, copy=True)
    codes = np.array(codes0, dtype=np.uint8, copy=True)
    N, Cs, H, W = S.shape
    M, K, Csp = D.shape
    Ct, dk = codes.shape[0], codes.shape[1]
    Tf = T.reshape(N, Ct, -1)
    ss = [shifted(S[:, m * Csp:(m + 1) * Csp], dk, stride, pad) for m in range(M)]
    cm = [codes[:, :, :, m].reshape(Ct, dk * dk) for m in range(M)]
    Y = sum(contribution(ss[m], D[m], cm[m]) for m in range(M))
    hist = [float(np.sum((Tf - Y) ** 2))]
    for _ in range(sweeps):
        for m in range(M):
            old = contribution(ss[m], D[m], cm[m])
            R = Tf - Y + old                                # Eq. (15)
            D[m], cm[m] = subspace_step(ss[m], R, D[m], cm[m], inner)
            Y = Y - old + contribution(ss[m], D[m], cm[m])
            hist.append(float(np.sum((Tf - Y) ** 2)))
    for m in range(M):
        codes[:, :, :, m] = cm[m].reshape(Ct, dk, dk)
    return D, codes, np.array(hist)
