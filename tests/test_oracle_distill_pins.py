"""Pins of the oracle's distillation targets and losses (Section 4.4,
Eq.8-11).  CPU only.

Column maxima of the teacher's attention are checked against the explicit
attention matrix built with numpy (an independent formulation), invariants
(every entry in (0, 1], each query's column sums to one so the column maxima
sum to at least one) and planted closed forms; the KL term against scipy's
relative entropy; the latent loss against closed forms."""
import numpy as np
import pytest
import scipy.stats
import torch

import oracle

RNG = np.random.default_rng(88)


def explicit_attention(Q, K, h):
    """A[k, q] = softmax over keys of q . k / sqrt(d) (numpy, float64)."""
    q = Q[:, h, :].astype(np.float64)
    k = K[:, h, :].astype(np.float64)
    L = q @ k.T / np.sqrt(q.shape[1])            # [q, k]
    E = np.exp(L - L.max(axis=1, keepdims=True))
    return (E / E.sum(axis=1, keepdims=True)).T  # [k, q]


@pytest.mark.parametrize("N", [1, 2, 7, 64, 130])
def test_colmax_against_explicit_matrix(N):
    Q = RNG.normal(size=(N, 3, 64)).astype(np.float32)
    K = RNG.normal(size=(N, 3, 64)).astype(np.float32)
    for h in range(3):
        A = explicit_attention(Q, K, h)
        p = oracle.attention_colmax(Q, K, h)
        np.testing.assert_allclose(p, A.max(axis=1), rtol=1e-12, atol=1e-15)
        # s_attn: the largest entry of A is the largest column maximum
        assert abs(p.max() - A.max()) < 1e-12


def test_colmax_invariants_and_subset():
    N = 90
    Q = RNG.normal(size=(N, 2, 64)).astype(np.float32)
    K = RNG.normal(size=(N, 2, 64)).astype(np.float32)
    p = oracle.attention_colmax(Q, K, 0)
    assert (p > 0).all() and (p <= 1).all()
    assert p.sum() >= 1 - 1e-12
    keys = np.array([89, 0, 45, 3])
    np.testing.assert_array_equal(oracle.attention_colmax(Q, K, 0, keys=keys), p[keys])
    one = oracle.attention_colmax(Q[:1], K[:1], 1)
    np.testing.assert_array_equal(one, [1.0])


def test_colmax_planted_key():
    """Every query puts weight e^L / (e^L + N - 1) on a key whose logit is L
    above the (zero) others: that key's column maximum is that weight, every
    other key's is 1 / (e^L + N - 1)."""
    N, L = 50, 4.0
    Q = np.zeros((N, 1, 64), np.float32)
    Q[:, 0, 0] = 1.0
    K = np.zeros((N, 1, 64), np.float32)
    K[17, 0, 0] = 8.0 * L
    p = oracle.attention_colmax(Q, K, 0)
    den = np.exp(L) + N - 1
    assert abs(p[17] - np.exp(L) / den) < 1e-13
    np.testing.assert_allclose(np.delete(p, 17), 1.0 / den, rtol=1e-12)


def test_teacher_delta_closed_forms():
    N = 40
    Q = RNG.normal(size=(N, 2, 64)).astype(np.float32)
    K = RNG.normal(size=(N, 2, 64)).astype(np.float32)
    V = np.tile(RNG.normal(size=(1, 2, 64)).astype(np.float32), (N, 1, 1))
    # identical values: attention returns them unchanged, so (A - I) V = 0
    np.testing.assert_allclose(oracle.teacher_delta_rows(Q, K, V, 1), 0, atol=1e-13)
    V2 = RNG.normal(size=(N, 2, 64)).astype(np.float32)
    d = oracle.teacher_delta_rows(Q, K, V2, 0, rows=[3, 9])
    A = explicit_attention(Q, K, 0)
    ref = A.T @ V2[:, 0, :].astype(np.float64) - V2[:, 0, :]
    np.testing.assert_allclose(d, ref[[3, 9]], atol=1e-12)


def test_router_loss():
    p = RNG.uniform(0.01, 1, 300)
    r = RNG.dirichlet(np.ones(300))
    kl = scipy.stats.entropy(p / p.sum(), r)
    lam = 0.7
    assert abs(oracle.router_loss(p, r, lam) - (kl + lam * abs(p.max() - r.max()))) < 1e-12
    # identical distributions with equal maxima: zero loss
    assert abs(oracle.router_loss(r, r, 5.0)) < 1e-15
    # the KL term compares normalised distributions: scaling p changes only
    # the max term
    assert abs(oracle.router_loss(3 * p, r, 0.0) - kl) < 1e-12


def test_latent_loss():
    a = RNG.normal(size=(30, 64))
    assert abs(oracle.latent_loss(a, a, 2.0)) < 1e-12
    # same direction, twice the length: the norm of the difference only
    assert abs(oracle.latent_loss(2 * a, a, 3.0) - np.linalg.norm(a)) < 1e-10
    # orthogonal: norm of the difference plus lambda
    b = np.zeros_like(a)
    b[:, 0] = 1.0
    c = np.zeros_like(a)
    c[:, 1] = 2.0
    expect = np.sqrt(30 * 1 + 30 * 4) + 0.5
    assert abs(oracle.latent_loss(b, c, 0.5) - expect) < 1e-12
    cos = torch.nn.functional.cosine_similarity(torch.from_numpy(a.ravel()),
                                                torch.from_numpy((a + 0.3).ravel()), dim=0)
    expect = np.linalg.norm(0.3 * np.ones_like(a)) + 1.5 * (1 - float(cos))
    assert abs(oracle.latent_loss(a, a + 0.3, 1.5) - expect) < 1e-10
