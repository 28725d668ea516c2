"""numpy brute force of the routed layer for tiny shapes (fp64).

TEST INFRASTRUCTURE ONLY.  A second, independent formulation that builds the
explicit matrices -- the full N x N attention matrix of every head, the full
[N, L] gate activations -- instead of looping row by row.  Used to cross-check
the C oracle on tiny inputs (N up to a few hundred).
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf, expit, softmax


def pool(Q, W, U, w):
    """Eq.1-2 on explicit matrices; returns q_pool [H,d], alpha [H,N]."""
    Q = np.asarray(Q, np.float64)
    N, H, d = Q.shape
    qp = np.zeros((H, d))
    al = np.zeros((H, N))
    for h in range(H):
        Qh = Q[:, h, :]                                  # [N, d]
        G = np.tanh(Qh @ np.asarray(W[h], np.float64).T) * expit(Qh @ np.asarray(U[h], np.float64).T)
        a = G @ np.asarray(w[h], np.float64)             # [N]
        al[h] = softmax(a)
        qp[h] = al[h] @ Qh
    return qp, al


def route(K, V, qp, scale):
    K = np.asarray(K, np.float64)
    V = np.asarray(V, np.float64)
    N, H, d = K.shape
    r = np.zeros((H, N))
    for h in range(H):
        r[h] = softmax(scale * (K[:, h, :] @ qp[h]))
    s = r.max(axis=1)
    C = np.einsum("hn,nhd->hd", r, V)
    mean = V.mean(axis=0)
    return s, C, mean, r


def attention(Q, K, V, h, scale):
    Qh = np.asarray(Q, np.float64)[:, h, :]
    Kh = np.asarray(K, np.float64)[:, h, :]
    Vh = np.asarray(V, np.float64)[:, h, :]
    A = softmax(scale * Qh @ Kh.T, axis=1)
    return A @ Vh, A


def _act(x, act):
    return np.maximum(x, 0.0) if act == 1 else 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def surrogate(V, C_h, surr, h, act=0):
    Vh = np.asarray(V, np.float64)[:, h, :]
    N, d = Vh.shape
    Z = np.concatenate([Vh, np.broadcast_to(C_h, (N, d))], axis=1)   # [N, 2d]
    f = lambda k: np.asarray(surr[k][h], np.float64)
    Hg = _act(Z @ f("g_w1").T + f("g_b1"), act)
    Hd = _act(Z @ f("d_w1").T + f("d_b1"), act)
    gam = expit(Hg @ f("g_w2").T + f("g_b2"))
    dl = Hd @ f("d_w2").T + f("d_b2")
    return C_h[None, :] + gam * dl
