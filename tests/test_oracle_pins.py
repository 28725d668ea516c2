"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these compare the oracle with a retyping of its own formulas: they
use library routines (torch scaled-dot-product attention, scipy softmax and
erf), closed forms (planted keys, zero queries, one-hot router rows),
invariants (rows summing to one, token-permutation equivariance, identical
views) and the explicit-matrix brute force on tiny shapes.  Each is chosen
so that a plausible mistake (a dropped term, a wrong sign or index, a
transposed operand, softmax over the wrong axis or per view) fails one.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
from scipy.special import erf, expit, softmax

import oracle
from oracle import brute
from paper_2609_23733_amd import synth

pytestmark = pytest.mark.filterwarnings("ignore")
GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))


def small(S, P, H=4, d=64, L=64, dtype="f32", n_full=None, sharp=True, key=(9, 0), modes=None):
    if n_full is None:
        n_full = H // 2
    return synth.make_layer(S, P, dtype=dtype, n_full=n_full, key=key, sharp=sharp, H=H, d=d,
                            L=L, modes=modes)


def np32(t):
    return oracle.as_f32(t)


# ---------------------------------------------------------------- constants

def test_paper_constants_match_oracle_defaults():
    assert oracle.TAU_LOW == GOLD["tau_low"]["value"]
    assert oracle.TAU_HIGH == GOLD["tau_high"]["value"]
    assert synth.HIDDEN == GOLD["hidden"]["value"]
    assert synth.H_HEADS == GOLD["heads_per_layer"]["value"]
    assert synth.HEAD_DIM == GOLD["head_dim"]["value"]
    assert synth.BASE_SEED == GOLD["seed"]["value"]


# ------------------------------------------------- P1: FULL == library SDPA

@pytest.mark.parametrize("S,P", [(1, 37), (2, 61), (3, 50)])
def test_full_equals_torch_sdpa_fp64(S, P):
    x = small(S, P, H=3)
    Q, K, V = (torch.from_numpy(np32(t)).double() for t in (x.Q, x.K, x.V))
    ref = torch.nn.functional.scaled_dot_product_attention(
        Q.permute(1, 0, 2), K.permute(1, 0, 2), V.permute(1, 0, 2)).permute(1, 0, 2).numpy()
    for h in range(3):
        y = oracle.full_rows(x.Q, x.K, x.V, h)
        np.testing.assert_allclose(y, ref[:, h, :], rtol=1e-12, atol=1e-13)


def test_full_rows_subset_matches_all_rows():
    x = small(2, 40, H=2)
    allr = oracle.full_rows(x.Q, x.K, x.V, 1)
    rows = np.array([0, 7, 79], np.int64)
    np.testing.assert_array_equal(oracle.full_rows(x.Q, x.K, x.V, 1, rows), allr[rows])


def test_global_attention_spans_views_not_frames():
    """With S > 1 the FULL branch attends over all views (global), which is
    different from per-view (frame) attention computed by SDPA per view."""
    S, P = 3, 20
    x = small(S, P, H=1)
    y = oracle.full_rows(x.Q, x.K, x.V, 0)
    Q, K, V = (torch.from_numpy(np32(t)).double()[:, 0, :] for t in (x.Q, x.K, x.V))
    frame = torch.cat([torch.nn.functional.scaled_dot_product_attention(
        Q[s * P:(s + 1) * P][None], K[s * P:(s + 1) * P][None], V[s * P:(s + 1) * P][None])[0]
        for s in range(S)]).numpy()
    glob = torch.nn.functional.scaled_dot_product_attention(Q[None], K[None], V[None])[0].numpy()
    np.testing.assert_allclose(y, glob, rtol=1e-12, atol=1e-13)
    assert np.abs(y - frame).max() > 1e-3


def test_s1_global_equals_frame_attention():
    x = small(1, 33, H=2)
    for h in range(2):
        Q, K, V = (torch.from_numpy(np32(t)).double()[:, h, :] for t in (x.Q, x.K, x.V))
        frame = torch.nn.functional.scaled_dot_product_attention(Q[None], K[None], V[None])[0]
        np.testing.assert_allclose(oracle.full_rows(x.Q, x.K, x.V, h), frame.numpy(),
                                   rtol=1e-12, atol=1e-13)


# ----------------------------------------------------- P2: weights sum to one

def test_pool_and_route_weights_sum_to_one():
    x = small(2, 45, H=4)
    qp, a, al = oracle.router_pool(x.Q, x.W, x.U, x.w, want_weights=True)
    np.testing.assert_allclose(al.sum(axis=1), 1.0, atol=1e-12)
    assert (al > 0).all()
    s, C, mean, r = oracle.router_route(x.K, x.V, qp, want_r=True)
    np.testing.assert_allclose(r.sum(axis=1), 1.0, atol=1e-12)
    np.testing.assert_allclose(s, r.max(axis=1), rtol=0, atol=0)
    # s lies in [1/N, 1]
    N = x.N
    assert (s >= 1.0 / N - 1e-15).all() and (s <= 1.0).all()


# ----------------------------------------------- gated pooling structure pins

def test_pool_gate_structure_closed_form():
    """Eq.1 with W = beta*I, U = gamma*I (gamma large: sigmoid ~ step) and w = e_c:
    a_i = tanh(beta q_{i,c}) * sigmoid(gamma q_{i,c}); alpha = softmax_i(a).
    Fails if tanh/sigmoid are swapped, if the gate multiplies the wrong row, or
    if the softmax runs over the wrong axis."""
    N, H, d = 31, 2, 64
    rng = np.random.default_rng(1)
    Q = rng.normal(size=(N, H, d)).astype(np.float32)
    beta, gamma, c = 0.75, 4.0, 5
    W = np.stack([beta * np.eye(d, dtype=np.float32)] * H)
    U = np.stack([gamma * np.eye(d, dtype=np.float32)] * H)
    w = np.zeros((H, d), np.float32)
    w[:, c] = 1.0
    qp, a, al = oracle.router_pool(Q, W, U, w, want_weights=True)
    for h in range(H):
        x = Q[:, h, c].astype(np.float64)
        ref_a = np.tanh(beta * x) * expit(gamma * x)
        np.testing.assert_allclose(a[h], ref_a, rtol=1e-13, atol=1e-15)
        ref_al = softmax(ref_a)
        np.testing.assert_allclose(al[h], ref_al, rtol=1e-12)
        np.testing.assert_allclose(qp[h], ref_al @ Q[:, h, :].astype(np.float64), rtol=1e-12,
                                   atol=1e-14)


def test_pool_w_zero_gives_mean_query():
    """W = 0 => tanh(0) = 0 => alpha uniform => q_pool = mean of the queries
    (the paper's 'mean query' ablation, component ablation table)."""
    x = small(2, 30, H=3)
    W0 = torch.zeros_like(x.W)
    qp = oracle.router_pool(x.Q, W0, x.U, x.w)
    np.testing.assert_allclose(qp, np32(x.Q).astype(np.float64).mean(axis=0), rtol=1e-12,
                               atol=1e-15)


# ------------------------------------------------- P3: permutation equivariance

def test_token_permutation_equivariance():
    x = small(2, 40, H=4, n_full=2, modes=np.array([2, 1, 0, 2], np.uint8))
    rng = np.random.default_rng(3)
    pi = rng.permutation(x.N)
    Q, K, V = np32(x.Q), np32(x.K), np32(x.V)
    base = oracle.routed_layer(Q, K, V, x.W, x.U, x.w, x.surr, modes=x.modes)
    perm = oracle.routed_layer(Q[pi], K[pi], V[pi], x.W, x.U, x.w, x.surr, modes=x.modes)
    for k in ("q_pool", "s", "C", "mean"):
        np.testing.assert_allclose(perm[k], base[k], rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(perm["Y"], base["Y"][pi], rtol=1e-11, atol=1e-14)
    # the routing scores are also permutation invariant, so threshold modes are
    np.testing.assert_array_equal(oracle.assign(perm["s"], 0), oracle.assign(base["s"], 0))


# ----------------------------------------------------- P4: identical views

def test_identical_views():
    """S copies of one view: FULL, SURR and MEAN outputs equal those of the
    single view, q_pool equals it, and the saliency divides by S (the peak
    routing weight is shared by S identical keys)."""
    P, S = 23, 4
    one = small(1, P, H=3, modes=np.array([2, 1, 0], np.uint8))
    Q1, K1, V1 = np32(one.Q), np32(one.K), np32(one.V)
    Qs, Ks, Vs = (np.concatenate([a] * S) for a in (Q1, K1, V1))
    r1 = oracle.routed_layer(Q1, K1, V1, one.W, one.U, one.w, one.surr, modes=one.modes)
    rs = oracle.routed_layer(Qs, Ks, Vs, one.W, one.U, one.w, one.surr, modes=one.modes)
    np.testing.assert_allclose(rs["q_pool"], r1["q_pool"], rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(rs["s"], r1["s"] / S, rtol=1e-11)
    np.testing.assert_allclose(rs["C"], r1["C"], rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(rs["Y"], np.concatenate([r1["Y"]] * S), rtol=1e-10, atol=1e-13)


# ------------------------------------------------------- P5: brute force

@pytest.mark.parametrize("N", [1, 2, 3, 5, 17, 64, 130])
def test_tiny_shapes_against_brute_force(N):
    H = 16
    modes = np.array([2, 1, 0, 2] * 4, np.uint8)
    x = synth.make_layer(1, N, dtype="f32", key=(11, N), sharp=True, H=H, modes=modes)
    Q, K, V = np32(x.Q), np32(x.K), np32(x.V)
    ref_qp, ref_al = brute.pool(Q, np32(x.W), np32(x.U), np32(x.w))
    scale = 1.0 / 8.0
    ref_s, ref_C, ref_mean, ref_r = brute.route(K, V, ref_qp, scale)
    out = oracle.routed_layer(Q, K, V, x.W, x.U, x.w, x.surr, modes=x.modes)
    np.testing.assert_allclose(out["q_pool"], ref_qp, rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(out["s"], ref_s, rtol=1e-11)
    np.testing.assert_allclose(out["C"], ref_C, rtol=1e-11, atol=1e-14)
    np.testing.assert_allclose(out["mean"], ref_mean, rtol=1e-11, atol=1e-15)
    surr = {k: np32(v) for k, v in x.surr.items()}
    for h in range(H):
        if modes[h] == 2:
            ref = brute.attention(Q, K, V, h, scale)[0]
        elif modes[h] == 1:
            ref = brute.surrogate(V, ref_C[h], surr, h)
        else:
            ref = np.broadcast_to(ref_mean[h], (N, 64))
        np.testing.assert_allclose(out["Y"][:, h, :], ref, rtol=1e-10, atol=1e-13)


# ------------------------------------------------------- P6: zero queries

def test_zero_queries_three_way_equality():
    """Q = 0: alpha and r are uniform, s = 1/N, q_pool = 0 and C = mean.  Then
    FULL (uniform attention), MEAN and SURR with a zero correction layer all
    return the value mean."""
    N, H = 57, 3
    x = small(1, N, H=H, modes=np.array([2, 1, 0], np.uint8))
    Q0 = np.zeros((N, H, 64), np.float32)
    surr = {k: np32(v).copy() for k, v in x.surr.items()}
    surr["d_w2"][:] = 0.0
    surr["d_b2"][:] = 0.0
    out = oracle.routed_layer(Q0, x.K, x.V, x.W, x.U, x.w, surr, modes=x.modes)
    np.testing.assert_array_equal(out["q_pool"], 0.0)
    np.testing.assert_allclose(out["s"], 1.0 / N, rtol=1e-14)
    np.testing.assert_allclose(out["C"], out["mean"], rtol=1e-12, atol=1e-16)
    mean = np32(x.V).astype(np.float64).mean(axis=0)
    for h in range(H):
        np.testing.assert_allclose(out["Y"][:, h, :], np.broadcast_to(mean[h], (N, 64)),
                                   rtol=1e-12, atol=1e-16)


# --------------------------------------------------- P7/P9: planted key

def planted(N, Lval, H=1, d=64, jstar=None, seed=5):
    """All queries equal q = e_0 (so q_pool = q), keys with k_j[0] = 0 except
    k_{j*}[0] = 8 * Lval; other coordinates random.  With scale 1/sqrt(64):
    t_j = 0 for j != j*, t_{j*} = Lval, hence s = e^L / (e^L + N - 1)."""
    rng = np.random.default_rng(seed)
    if jstar is None:
        jstar = N // 3
    Q = np.zeros((N, H, d), np.float32)
    Q[:, :, 0] = 1.0
    K = rng.normal(size=(N, H, d)).astype(np.float32)
    K[:, :, 0] = 0.0
    K[jstar, :, 0] = np.float32(8.0 * Lval)
    V = rng.normal(size=(N, H, d)).astype(np.float32)
    return Q, K, V, jstar


def s_closed(N, Lval):
    return math.exp(Lval) / (math.exp(Lval) + N - 1)


@pytest.mark.parametrize("N", [2, 97, 2748])
@pytest.mark.parametrize("Lval", [0.0, 1.5, 6.25])
def test_planted_key_saliency_closed_form(N, Lval):
    Q, K, V, js = planted(N, Lval)
    rng = np.random.default_rng(0)
    W = rng.uniform(-.1, .1, size=(1, 64, 64)).astype(np.float32)
    U = rng.uniform(-.1, .1, size=(1, 64, 64)).astype(np.float32)
    w = rng.uniform(-.1, .1, size=(1, 64)).astype(np.float32)
    qp = oracle.router_pool(Q, W, U, w)
    np.testing.assert_allclose(qp[0], np.eye(64)[0], atol=1e-15)
    Lexact = float(np.float32(8.0 * Lval)) / 8.0
    s, C, mean = oracle.router_route(K, V, qp)
    assert abs(s[0] - s_closed(N, Lexact)) <= 1e-12 * max(1.0, s[0])
    # C = sum_j r_j v_j with the closed-form weights
    rj = np.full(N, 1.0 / (math.exp(Lexact) + N - 1))
    rj[js] = math.exp(Lexact) / (math.exp(Lexact) + N - 1)
    np.testing.assert_allclose(C[0], rj @ V[:, 0, :].astype(np.float64), rtol=1e-11, atol=1e-14)


def L_for(N, s):
    """Planted logit placing the saliency at s: e^L / (e^L + N - 1) = s."""
    return math.log(s * (N - 1) / (1.0 - s))


@pytest.mark.parametrize("N", [2748, 10992])
def test_threshold_rule_on_planted_saliency(N):
    """Eq.4 on planted saliencies placed 1e-3 either side of each threshold."""
    cases = [(0.20 + 1e-3, 2), (0.20 - 1e-3, 1), (0.01 + 1e-3, 1), (0.01 - 1e-3, 0),
             (0.5, 2), (0.05, 1)]
    for target, mode in cases:
        if target * N < 1.0 + 1e-9:
            continue
        Q, K, V, _ = planted(N, L_for(N, target))
        qp = oracle.router_pool(Q, np.zeros((1, 64, 64), np.float32),
                                np.zeros((1, 64, 64), np.float32), np.zeros((1, 64), np.float32))
        s, _, _ = oracle.router_route(K, V, qp)
        assert abs(s[0] - target) < 2e-6
        assert oracle.assign(s, oracle.RULE_THRESHOLD)[0] == mode


def test_threshold_inclusivity_and_nan():
    tl, th = np.float32(0.01), np.float32(0.2)
    s = np.array([float(th), float(tl), np.nextafter(float(th), 0), np.nextafter(float(tl), 1),
                  1.0, 0.0, np.nan])
    np.testing.assert_array_equal(oracle.assign(s, 0), [2, 0, 1, 1, 2, 0, 2])


def test_large_planted_logit_one_hot_context():
    """L large => r one-hot at j* => C -> v_{j*} (P9)."""
    N = 300
    Q, K, V, js = planted(N, 60.0)
    qp = np.eye(64)[:1]
    s, C, _ = oracle.router_route(K, V, qp)
    assert s[0] >= 1.0 - 1e-15
    np.testing.assert_allclose(C[0], V[js, 0, :].astype(np.float64), rtol=1e-12, atol=1e-20)


# ---------------------------------------------- P10: linear-logit mode router

def test_router_logits_one_hot_rows():
    H, Din = 16, 1024
    rng = np.random.default_rng(2)
    u = rng.normal(size=Din).astype(np.float32)
    cols = rng.choice(Din, size=3 * H, replace=False)
    Wr = np.zeros((3 * H, Din), np.float32)
    Wr[np.arange(3 * H), cols] = 1.0
    br = rng.normal(size=3 * H).astype(np.float32)
    lg = oracle.router_logits(u, Wr, br)
    np.testing.assert_array_equal(lg.reshape(-1), u[cols].astype(np.float64) + br)


def test_argmax_ties_and_nan():
    lg = np.array([[1.0, 1.0, 0.0], [0.0, 2.0, 2.0], [3.0, 3.0, 3.0], [0.0, 0.0, 1.0],
                   [np.nan, 0.0, 0.0], [-1.0, -2.0, -3.0]])
    np.testing.assert_array_equal(oracle.assign(lg, 1), [0, 1, 0, 2, 2, 0])


@pytest.mark.parametrize("wl", ["s2_f32", "s8_bf16", "s32_bf16", "s100_bf16"])
def test_generated_router_hits_target_modes_with_margin(wl):
    """The seeded workload routers (weights only; no tokens needed) produce the
    target modes under the oracle's logits, with top-1 minus top-2 >= 1e-3."""
    cfg = synth.WORKLOADS[wl]
    x = synth.make_layer(1, 3, dtype=cfg["dtype"], n_full=cfg["n_full"], key=(7, 0))
    lg = oracle.router_logits(x.u, x.Wr, x.br)
    modes = oracle.assign(lg, 1)
    np.testing.assert_array_equal(modes, x.modes)
    srt = np.sort(lg, axis=1)
    assert (srt[:, 2] - srt[:, 1] >= 1e-3).all()
    assert (modes == 2).sum() == cfg["n_full"]


def test_buckets_grouping():
    modes = np.array([2, 0, 1, 2, 0, 0, 1, 2], np.uint8)
    c, lst = oracle.buckets(modes)
    np.testing.assert_array_equal(c, [3, 2, 3])
    np.testing.assert_array_equal(lst, [1, 4, 5, 2, 6, 0, 3, 7])


# ----------------------------------------------------- surrogate pins

def _identity_surr(H, d, L, act, which):
    z = lambda *s: np.zeros(s, np.float32)
    s = {"g_w1": z(H, L, 2 * d), "g_b1": z(H, L), "g_w2": z(H, d, L), "g_b2": z(H, d),
         "d_w1": z(H, L, 2 * d), "d_b1": z(H, L), "d_w2": z(H, d, L), "d_b2": z(H, d)}
    s["g_b2"][:] = 0.7       # gamma = sigmoid(0.7) everywhere
    off = 0 if which == "v" else d
    for h in range(H):
        s["d_w1"][h, np.arange(L), off + np.arange(L)] = 1.0
        s["d_w2"][h, np.arange(d), np.arange(L)] = 1.0
    return s


@pytest.mark.parametrize("act", [0, 1])
@pytest.mark.parametrize("which", ["v", "C"])
def test_surrogate_closed_form(act, which):
    """Correction MLP acting on one half of z = [v; C] through identities:
    y = C + sigmoid(0.7) * act(v) (or act(C)).  Pins the concat order, the
    gate/correction roles, GELU against scipy's erf and ReLU."""
    N, H, d = 19, 2, 64
    rng = np.random.default_rng(4)
    V = rng.normal(size=(N, H, d)).astype(np.float32)
    C = rng.normal(size=(H, d))
    s = _identity_surr(H, d, d, act, which)
    f = (lambda x: np.maximum(x, 0)) if act == 1 else (lambda x: 0.5 * x * (1 + erf(x / np.sqrt(2))))
    for h in range(H):
        y = oracle.surr_rows(V, C[h], s, h, act=act)
        src = V[:, h, :].astype(np.float64) if which == "v" else np.broadcast_to(C[h], (N, d))
        g = expit(float(np.float32(0.7)))
        np.testing.assert_allclose(y, C[h] + g * f(src), rtol=1e-13, atol=1e-15)


def test_surrogate_gate_modulates():
    """A zero correction (delta = 0) leaves exactly the context (Eq.7)."""
    x = small(1, 16, H=2)
    s = {k: np32(v).copy() for k, v in x.surr.items()}
    s["d_w2"][:] = 0
    s["d_b2"][:] = 0
    C = np.random.default_rng(0).normal(size=64)
    np.testing.assert_array_equal(oracle.surr_rows(x.V, C, s, 1), np.broadcast_to(C, (16, 64)))


# ------------------------------------ ablation variants (component study,
# ------------------------------------ compute-mode study)

def test_binary_rules():
    """Two-branch routing (no surrogate): threshold form is FULL if s >= tau_high
    else MEAN -- a score between the thresholds, SURR under Eq.4, becomes MEAN;
    argmax form compares only the MEAN and FULL logits (MEAN on a tie), even
    when the SURR logit is the largest.  NaN goes to FULL."""
    th, tl = float(np.float32(0.2)), float(np.float32(0.01))
    s = np.array([th, np.nextafter(th, 0), 0.05, tl, 0.0, 1.0, np.nan])
    np.testing.assert_array_equal(oracle.assign(s, oracle.RULE_THRESHOLD), [2, 1, 1, 0, 0, 2, 2])
    np.testing.assert_array_equal(oracle.assign(s, oracle.RULE_THRESHOLD_BINARY),
                                  [2, 0, 0, 0, 0, 2, 2])
    lg = np.array([[1.0, 5.0, 0.0], [0.0, 9.0, 2.0], [3.0, 3.0, 3.0], [0.0, 0.0, 1.0],
                   [np.nan, 0.0, 0.0], [0.0, np.nan, -1.0]])
    np.testing.assert_array_equal(oracle.assign(lg, oracle.RULE_ARGMAX_BINARY),
                                  [0, 2, 0, 2, 2, 0])


def test_mean_query_equals_gated_pooling_with_zero_w():
    """Mean-query ablation: q_pool = mean_i q_i, the same value that the
    gated pooling of Eq.1-2 gives when W = 0 (uniform alpha)."""
    x = small(2, 40, H=3)
    W0 = np.zeros_like(np32(x.W))
    gated = oracle.router_pool(x.Q, W0, x.U, x.w)
    np.testing.assert_allclose(oracle.router_pool_mean(x.Q), gated, rtol=1e-12, atol=1e-15)
    out = oracle.routed_layer(x.Q, x.K, x.V, x.W, x.U, x.w, x.surr, modes=x.modes,
                              pool=oracle.POOL_MEAN)
    np.testing.assert_allclose(out["q_pool"], gated, rtol=1e-12, atol=1e-15)


def test_mean_context_matches_base_when_routing_is_uniform():
    """Mean-context ablation: the surrogate sees the value mean instead of C_h.
    With Q = 0 the routing is uniform, C_h = mean_h, and both variants agree;
    with real queries they differ."""
    N, H = 33, 2
    modes = np.array([1, 1], np.uint8)
    x = small(1, N, H=H, modes=modes)
    Q0 = np.zeros((N, H, 64), np.float32)
    a = oracle.routed_layer(Q0, x.K, x.V, x.W, x.U, x.w, x.surr, modes=modes)
    b = oracle.routed_layer(Q0, x.K, x.V, x.W, x.U, x.w, x.surr, modes=modes,
                            surr_variant=oracle.SURR_MEAN_CONTEXT)
    np.testing.assert_allclose(a["Y"], b["Y"], rtol=1e-11, atol=1e-14)
    c = oracle.routed_layer(x.Q, x.K, x.V, x.W, x.U, x.w, x.surr, modes=modes)
    e = oracle.routed_layer(x.Q, x.K, x.V, x.W, x.U, x.w, x.surr, modes=modes,
                            surr_variant=oracle.SURR_MEAN_CONTEXT)
    assert np.abs(c["Y"] - e["Y"]).max() > 1e-6
    # and it is Eq.7 evaluated at the value mean
    for h in range(H):
        ref = brute.surrogate(np32(x.V), e["mean"][h], x.surr, h)
        np.testing.assert_allclose(e["Y"][:, h, :], ref, rtol=1e-10, atol=1e-13)


def test_no_residual_is_zero_correction():
    """No-residual ablation: y = C_h, which is what Eq.7 gives when the
    correction MLP's output layer is zero."""
    x = small(1, 21, H=2)
    s = {k: np32(v).copy() for k, v in x.surr.items()}
    s["d_w2"][:] = 0
    s["d_b2"][:] = 0
    C = np.random.default_rng(1).normal(size=64)
    np.testing.assert_array_equal(oracle.surr_rows(x.V, C, x.surr, 0, variant=oracle.SURR_NO_RESIDUAL),
                                  oracle.surr_rows(x.V, C, s, 0))


def test_add_identity_closed_form():
    """Identity-added reading: y = v + C_h + gamma (.) delta; with a zero
    correction layer y = v + C_h exactly."""
    x = small(1, 23, H=2)
    s = {k: np32(v).copy() for k, v in x.surr.items()}
    s["d_w2"][:] = 0
    s["d_b2"][:] = 0
    C = np.random.default_rng(2).normal(size=64)
    y = oracle.surr_rows(x.V, C, s, 1, variant=oracle.SURR_ADD_IDENTITY)
    np.testing.assert_allclose(y, np32(x.V)[:, 1, :].astype(np.float64) + C, rtol=1e-15,
                               atol=1e-15)


def _phi(x):
    return np.where(x > 0, x + 1.0, np.exp(np.minimum(x, 0.0)))


@pytest.mark.parametrize("N", [1, 2, 7, 64, 129])
def test_linear_attention_against_matrix_form(N):
    """Linear attention (phi = elu + 1): the oracle's row-by-row definition
    against the explicit matrix A = phi(Q) phi(K)^T, rows normalised, times V."""
    rng = np.random.default_rng(N)
    H, d = 2, 64
    Q = rng.normal(size=(N, H, d)).astype(np.float32)
    K = rng.normal(size=(N, H, d)).astype(np.float32)
    V = rng.normal(size=(N, H, d)).astype(np.float32)
    for h in range(H):
        A = _phi(Q[:, h].astype(np.float64)) @ _phi(K[:, h].astype(np.float64)).T
        ref = (A / A.sum(axis=1, keepdims=True)) @ V[:, h].astype(np.float64)
        np.testing.assert_allclose(oracle.linattn_rows(Q, K, V, h), ref, rtol=1e-11, atol=1e-13)


def test_linear_attention_special_cases():
    """Equal keys give equal weights: y_i = mean of V for every query.  For any
    keys the weights are positive, so y lies in the per-coordinate hull of V;
    a joint permutation of the key and value rows changes nothing."""
    rng = np.random.default_rng(11)
    N, H, d = 50, 1, 64
    Q = rng.normal(size=(N, H, d)).astype(np.float32)
    V = rng.normal(size=(N, H, d)).astype(np.float32)
    K = np.broadcast_to(rng.normal(size=(1, H, d)), (N, H, d)).astype(np.float32).copy()
    y = oracle.linattn_rows(Q, K, V, 0)
    np.testing.assert_allclose(y, np.broadcast_to(V[:, 0].astype(np.float64).mean(axis=0), (N, d)),
                               rtol=1e-12, atol=1e-14)
    K = rng.normal(size=(N, H, d)).astype(np.float32)
    y = oracle.linattn_rows(Q, K, V, 0)
    assert (y <= V[:, 0].max(axis=0) + 1e-12).all() and (y >= V[:, 0].min(axis=0) - 1e-12).all()
    pi = rng.permutation(N)
    np.testing.assert_allclose(oracle.linattn_rows(Q, K[pi], V[pi], 0), y, rtol=1e-12, atol=1e-14)
