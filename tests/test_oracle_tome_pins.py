"""Pins of the oracle's token merging (ToMe's bipartite soft matching before the
routed attention; the paper's ToMe combination).  CPU only.

The metric's rounding is checked against torch's float32 -> bfloat16
conversion; the destination split against counts worked out by hand; the
matching, the selection and the rows against a pure-Python brute force over
every (source, destination) pair on tiny inputs; planted cases fix the
decisions that matter (a source equal to a destination in direction, a long
destination beaten by a better-aligned short one, exact ties broken by token
index); merge and unmerge against invariants (counts, sums, identity when
nothing is merged, identity on groups of identical tokens)."""
import math

import numpy as np
import pytest
import torch

import oracle

RNG = np.random.default_rng(77)


def test_metric_rounding_matches_torch_bf16():
    x = RNG.normal(size=4000).astype(np.float32) * np.float32(3.0)
    # values halfway between two bf16 numbers (ties to even, both parities)
    base = (np.arange(1, 200, dtype=np.uint32) << 16) | np.uint32(0x3F800000)
    halfway = (base | np.uint32(0x8000)).view(np.float32)
    vals = np.concatenate([x, halfway, -halfway, np.float32([0.0, -0.0, 1e-30, 3e38])])
    K = vals.reshape(-1, 1, 1)
    got = oracle.tome_metric(K).ravel()
    ref = torch.from_numpy(vals).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(got, ref)


def test_metric_is_head_sum():
    k = RNG.normal(size=(30, 1, 8)).astype(np.float32)
    # all 16 heads equal: the sum is 16 k exactly (a power of two)
    K = np.repeat(k, 16, axis=1)
    ref = torch.from_numpy(16 * k[:, 0, :]).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(oracle.tome_metric(K), ref)
    # only head 5 nonzero: the metric is that head, rounded
    K = np.zeros((30, 16, 8), np.float32)
    K[:, 5, :] = k[:, 0, :]
    ref = torch.from_numpy(k[:, 0, :]).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(oracle.tome_metric(K), ref)


@pytest.mark.parametrize("S,P,M,g,ndst", [
    (3, 15, 12, 3, 33),     # 10 patches: g = 2 leaves 10 sources, g = 3 leaves 12
    (3, 15, 10, 2, 35),
    (2, 1374, 1000, 4, 1374 + 5 + 343),
    (4, 9, 0, 1, 36),       # nothing merged: every token a destination
    (100, 1374, 123660, 12, 137400 - 99 * (1369 - 115)),
    (100, 1374, 103050, 5, 137400 - 99 * (1369 - 274)),
])
def test_split_counts(S, P, M, g, ndst):
    is_dst, gg = oracle.tome_split(S, P, M)
    assert gg == g and int(is_dst.sum()) == ndst
    view = is_dst.reshape(S, P)
    assert view[0].all() and view[:, :5].all()
    if S > 1 and g > 1:
        # the patch lattice of a later view: indices 0, g, 2g, ...
        np.testing.assert_array_equal(np.nonzero(view[1, 5:])[0], np.arange(0, P - 5, g))
    if g > 1:   # g is the smallest stride that leaves M sources
        n_prev = (S - 1) * ((P - 5) - -(-(P - 5) // (g - 1)))
        assert n_prev < M


def test_split_rejects_too_many():
    with pytest.raises(ValueError):
        oracle.tome_split(2, 15, 10)   # at most 9 sources (patch 0 stays)
    with pytest.raises(ValueError):
        oracle.tome_split(1, 15, 1)    # one view: no sources at all


def brute_plan(K, S, P, M):
    """Every (source, destination) pair in pure Python; cosines with math.fsum."""
    N = S * P
    m = oracle.tome_metric(K)
    is_dst, _ = oracle.tome_split(S, P, M)
    dst = [t for t in range(N) if is_dst[t]]
    src = [t for t in range(N) if not is_dst[t]]

    def cos(a, b):
        na = math.sqrt(math.fsum(x * x for x in m[a]))
        nb = math.sqrt(math.fsum(x * x for x in m[b]))
        if na == 0 or nb == 0:
            return 0.0
        return math.fsum(x * y for x, y in zip(m[a], m[b])) / (na * nb)

    best, score = {}, {}
    for a in src:
        cands = [(cos(a, b), -b) for b in dst]
        c, nb = max(cands)
        best[a], score[a] = -nb, c
    order = sorted(src, key=lambda a: (-score[a], a))
    merged = set(order[:M])
    row, r = {}, 0
    for t in range(N):
        if t not in merged:
            row[t] = r
            r += 1
    for a in merged:
        row[a] = row[best[a]]
    return best, score, merged, [row[t] for t in range(N)], r


@pytest.mark.parametrize("S,P,M,seed", [(3, 15, 12, 0), (3, 15, 5, 1), (4, 12, 9, 2),
                                        (2, 20, 13, 3)])
def test_plan_against_brute_force(S, P, M, seed):
    rng = np.random.default_rng(seed)
    K = rng.normal(size=(S * P, 3, 8)).astype(np.float32)
    # a few near-copies of destinations so that some similarities are high
    K[P + 6] = K[2] * 1.7
    K[(S - 1) * P + 7] = K[P] + 0.01
    pl = oracle.tome_plan(K, S, P, M, nthreads=2)
    best, score, merged, row, nrows = brute_plan(K, S, P, M)
    for i, a in enumerate(pl["srcs"]):
        assert pl["best"][i] == best[a]
        assert abs(pl["score"][i] - score[a]) < 1e-12
        assert bool(pl["merged"][i]) == (a in merged)
    np.testing.assert_array_equal(pl["row"], row)
    assert pl["nrows"] == nrows == S * P - M


def test_cosine_not_dot_product():
    """A long destination that is badly aligned loses to a short, aligned one."""
    S, P = 2, 7   # 2 patches per view; view 1: patch 0 destination, patch 1 source
    K = np.zeros((S * P, 1, 4), np.float32)
    K[:, 0, 3] = 1.0                              # all tokens alike in feature 3
    K[0, 0] = [100.0, 100.0, 0.0, 1.0]            # long, half aligned
    K[1, 0] = [0.5, 0.0, 0.0, 0.0]                # short, aligned with the source
    K[P + 6, 0] = [1.0, 0.0, 0.0, 0.0]            # the source
    srcs, best, score = oracle.tome_match(K, S, P, 1)
    assert list(srcs) == [P + 6] and best[0] == 1 and abs(score[0] - 1.0) < 1e-15


def test_planted_copies_merge_first_and_ties_by_index():
    S, P = 3, 15
    K = RNG.normal(size=(S * P, 2, 8)).astype(np.float32)
    is_dst, _ = oracle.tome_split(S, P, 6)
    srcs = np.nonzero(~is_dst)[0]
    # three sources that point exactly along destination 4 (cosine 1)
    planted = [srcs[5], srcs[1], srcs[3]]
    for a, f in zip(planted, (2.0, 0.5, 4.0)):
        K[a] = K[4] * f
    K[7] = K[4] * 2.0   # a second destination along the same direction (exact scaling)
    pl = oracle.tome_plan(K, S, P, 2)
    got = set(pl["srcs"][pl["merged"]])
    # all three tie at cosine 1: the two lowest token indices win
    assert got == set(sorted(planted)[:2])
    # and each ties between destinations 4 and 7: the first in token order
    for a in planted:
        assert pl["best"][list(pl["srcs"]).index(a)] == 4


def test_nothing_merged_is_identity():
    S, P = 3, 11
    K = RNG.normal(size=(S * P, 2, 8)).astype(np.float32)
    pl = oracle.tome_plan(K, S, P, 0)
    np.testing.assert_array_equal(pl["row"], np.arange(S * P))
    X = RNG.normal(size=(S * P, 2, 8)).astype(np.float32)
    np.testing.assert_array_equal(oracle.tome_merge(X, pl["row"], pl["nrows"]), X)


def test_merge_sums_and_counts():
    S, P, M = 4, 13, 20
    K = RNG.normal(size=(S * P, 2, 8)).astype(np.float32)
    pl = oracle.tome_plan(K, S, P, M)
    X = RNG.normal(size=(S * P, 5)).astype(np.float32)
    Xm = oracle.tome_merge(X, pl["row"], pl["nrows"])
    size = np.bincount(pl["row"], minlength=pl["nrows"])
    assert size.sum() == S * P and (size >= 1).all() and pl["nrows"] == S * P - M
    np.testing.assert_allclose((Xm * size[:, None]).sum(0), X.astype(np.float64).sum(0),
                               rtol=1e-12, atol=1e-12)
    # a row of one token is that token
    one = np.nonzero(size == 1)[0]
    first = {r: t for t, r in reversed(list(enumerate(pl["row"])))}
    for r in one[:10]:
        np.testing.assert_array_equal(Xm[r], X[first[r]])


def test_unmerge_of_identical_groups_is_identity():
    S, P, M = 3, 15, 9
    K = RNG.normal(size=(S * P, 2, 8)).astype(np.float32)
    pl = oracle.tome_plan(K, S, P, M)
    X = RNG.normal(size=(pl["nrows"], 3)).astype(np.float32)
    Xt = X[pl["row"]]                 # every token a copy of its row
    back = oracle.tome_unmerge(oracle.tome_merge(Xt, pl["row"], pl["nrows"]), pl["row"])
    np.testing.assert_array_equal(back, Xt)
