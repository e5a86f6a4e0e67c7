"""Error-corrected quantization of a fully-connected layer -- TEST
INFRASTRUCTURE ONLY (imported by tests/ and nothing in the product package).

Paper: Wu et al., "Quantized Convolutional Neural Networks for Mobile
Devices", CVPR 2016, Sec. 3.3.1.  Given the inputs S_n and the desired
responses T_n of a fully-connected layer on N images, the sub-codebooks D^(m)
and assignments B^(m) minimise the response error of Eq. (8),

    sum_n || T_n - sum_m (D^(m) B^(m))^T S_n^(m) ||^2,

by block coordinate descent over the subspaces.  For subspace m the residual
of the other subspaces is R_n^(m) (Eq. (9)); Eq. (10) is then minimised by
alternating

  * the sub-codebook update (Eq. (11)): for each sub-codeword k, the least
    squares problem over the images and the output channels L_k assigned
    to it, min_{D_k} sum_n sum_{c in L_k} (R_n(c) - D_k^T S_n^(m))^2; its
    normal equations are |L_k| G D_k = sum_{c in L_k} P_c with
    G = S^(m)T S^(m) and P_c = S^(m)T r_c (r_c = R(:, c));
  * the assignment update (Eq. (12)): k*(c) = argmin_k
    sum_n (R_n(c) - D_k^T S_n^(m))^2 = ||r_c||^2 - 2 D_k^T P_c + D_k^T G D_k.

Everything is float64.  Readings of what the paper leaves open (E1-E6 in the
design notes):
  E1 the descent starts from given sub-codebooks and assignments (those of
     the k-means quantizer of Eq. (4) in practice);
  E2 a sweep visits m = 0 .. M-1 in order; for each subspace, `inner`
     rounds of (sub-codebook update, then assignment update), the order in
     which the paper states them;
  E3 a sub-codeword that no output channel uses keeps its value;
  E4 the normal equations are solved by elimination in channel order
     without row exchanges; a pivot <= 1e-12 times the largest diagonal
     entry of G marks a direction the inputs do not span (for instance a
     channel that is zero on every image): that coordinate of D_k is set
     to 0 and its row and column are left out;
  E5 the assignment minimises D_k^T G D_k - 2 D_k^T P_c (the constant
     ||r_c||^2 dropped), ties to the lowest k;
  E6 the reported objective is Eq. (8) after each subspace step, plus the
     starting value.
"""
from __future__ import annotations

import numpy as np

PIVOT_REL = 1e-12


def solve_normal(G, b):
    """E4: x with G x = b by elimination in order, small pivots dropped."""
    n = G.shape[0]
    A = np.array(G, dtype=np.float64, copy=True)
    y = np.array(b, dtype=np.float64, copy=True)
    scale = float(np.max(np.diag(G))) if n else 0.0
    live = np.zeros(n, bool)
    for j in range(n):
        if A[j, j] <= PIVOT_REL * scale or A[j, j] <= 0.0:
            continue  # a direction S^(m) does not span: x_j = 0
        live[j] = True
        for i in range(j + 1, n):
            f = A[i, j] / A[j, j]
            A[i, j:] -= f * A[j, j:]
            y[i] -= f * y[j]
    x = np.zeros(n, np.float64)
    for j in range(n - 1, -1, -1):
        if live[j]:
            s = y[j] - sum(A[j, i] * x[i] for i in range(j + 1, n) if live[i])
            x[j] = s / A[j, j]
    return x


def subspace_step(Sm, R, Dm, codes_m, inner=1):
    """Eq. (10)-(12) for one subspace: Sm [N][C's], R [N][C_t] (Eq. (9)),
    Dm [K][C's] and codes_m [C_t] (updated copies are returned)."""
    Dm = np.array(Dm, dtype=np.float64, copy=True)
    codes_m = np.array(codes_m, copy=True)
    K = Dm.shape[0]
    G = Sm.T @ Sm
    P = Sm.T @ R                                    # [C's][C_t]
    for _ in range(inner):
        for k in range(K):                          # Eq. (11)
            Lk = codes_m == k
            if Lk.any():
                Dm[k] = solve_normal(G, P[:, Lk].sum(axis=1)) / Lk.sum()
        q = np.einsum("kj,ji,ki->k", Dm, G, Dm)     # D_k^T G D_k
        cost = q[:, None] - 2.0 * (Dm @ P)          # Eq. (12) without ||r_c||^2
        codes_m = np.argmin(cost, axis=0).astype(np.uint8)  # first minimum
    return Dm, codes_m


def forward(S, D, codes):
    """sum_m (D^(m) B^(m))^T S^(m): the quantized layer's response [N][C_t]."""
    M, K, Csp = D.shape
    Y = np.zeros((S.shape[0], codes.shape[0]), np.float64)
    for m in range(M):
        Y += S[:, m * Csp:(m + 1) * Csp] @ D[m][codes[:, m]].T
    return Y


def ec_fc(S, T, D0, codes0, sweeps=1, inner=1):
    """Error-corrected quantization of a FC layer (Eq. (8)-(12)).

    S [N][C_s], T [N][C_t] (fp32 or fp64), D0 [M][K][C's], codes0 [C_t][M].
    Returns (D float64 [M][K][C's], codes uint8 [C_t][M], objective history:
    Eq. (8) at the start and after every subspace step).
    """
    S = np.asarray(S, np.float64)
    T = np.asarray(T, np.float64)
    D = np.array(D0, dtype=np.float64, copy=True)
    codes = np.array(codes0, dtype=np.uint8, copy=True)
    M, K, Csp = D.shape
    Y = forward(S, D, codes)
    hist = [float(np.sum((T - Y) ** 2))]
    for _ in range(sweeps):
        for m in range(M):
            Sm = S[:, m * Csp:(m + 1) * Csp]
            old = Sm @ D[m][codes[:, m]].T
            R = T - Y + old                          # Eq. (9)
            D[m], codes[:, m] = subspace_step(Sm, R, D[m], codes[:, m], inner)
            Y = Y - old + Sm @ D[m][codes[:, m]].T
            hist.append(float(np.sum((T - Y) ** 2)))
    return D, codes, np.array(hist)
