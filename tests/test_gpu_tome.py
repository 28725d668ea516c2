"""GPU parity of token merging before the routed attention (the paper's ToMe
combination, read as ToMe's bipartite soft matching) against the oracle,
through the C ABI.

Decisions (each source's destination, the merged set) are taken in fp32 on
the GPU and in fp64 by the oracle from the same bf16 metric, so near-ties may
go either way: the GPU's choice must be a maximum within rounding (its oracle
similarity within 2e-6 of the oracle's best), its similarity must match the
oracle's for that choice within 2e-6, and the merged sources must be the most
similar ones within 4e-6.  Planted inputs with margins (and exact ties broken
by token index) make every decision unique: there the plan must equal the
oracle's exactly.  Given the GPU's decisions, the rows and the member lists
are compared exactly, the merged rows within half an ulp of their format (plus
fp32 summation error), unmerging exactly, and the routed layer on the merged
rows with the layer's own bar.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2609_23733_amd import synth
from test_gpu_parity import check_y, log, oracle_layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_23733_amd import vp
    vp.load_library()


def test_tome_element_offsets_past_2_32():
    """N = 3053 x 1374 = 4,194,822 tokens at merging ratio 0.9: token rows of
    [N, 16, 64] inputs pass 2^32 elements from token 2^22 on.  The plan is
    checked as at S = 100 (64 sampled decisions against the oracle, rows and
    member lists of every token exactly); merged rows whose members lie past
    the boundary on a sample; the unmerged [N, 16, 64] output against the
    merged rows it copies, bitwise."""
    from paper_2609_23733_amd import vp
    S, P = 3053, synth.TOKENS_PER_VIEW
    N = S * P
    M = int(0.9 * N)
    log("tome element offsets past 2^32: N=%d M=%d" % (N, M))
    K = synth.stored(synth.normal((N, 16, 64), synth.derive_seed(48, S, 0), 1.0, "cuda"), "bf16")
    plan = run_plan(K, S, P, M)
    Kc = K.cpu()
    is_dst, _ = oracle.tome_split(S, P, M)
    nsrc = int((~is_dst).sum())
    sample = synth.sample_rows(nsrc, 64, synth.derive_seed(48, S, 1))
    check_plan(Kc, S, P, M, plan, "N=%d" % N, srcs_sample=sample)
    X = synth.stored(synth.normal((N, 16, 64), synth.derive_seed(48, S, 2), 1.0, "cuda"), "bf16")
    Xm = vp.tome_merge(X, plan)
    back = vp.tome_unmerge(Xm, plan)
    torch.cuda.synchronize()
    assert torch.equal(back, Xm[plan.row.long()])
    rs = plan.row_start.cpu().numpy().astype(np.int64)
    mem = plan.members.cpu().numpy().astype(np.int64)
    row = plan.row.cpu().numpy().astype(np.int64)
    high = np.unique(row[2 ** 22:])
    pick = synth.sample_rows(high.shape[0], 24, synth.derive_seed(48, S, 3))
    rows = np.unique(np.concatenate([high[pick], [row[2 ** 22 - 1], row[N - 1]]]))
    toks = np.concatenate([mem[rs[r]:rs[r + 1]] for r in rows])
    assert toks.max() >= 2 ** 22
    lab = np.concatenate([np.full(rs[r + 1] - rs[r], i) for i, r in enumerate(rows)])
    Xs = X[torch.from_numpy(toks).cuda()].cpu()
    ref = oracle.tome_merge(Xs, lab, rows.shape[0])
    g = Xm[torch.from_numpy(rows).cuda()].double().cpu().numpy()
    bound = merged_bound(ref, rs[rows + 1] - rs[rows], float(Xs.float().abs().max()), True)
    log("N=%d merge worst err/bound = %.3f" % (N, float((np.abs(g - ref) / bound).max())))
    assert (np.abs(g - ref) <= bound).all()


def run_plan(K, S, P, M):
    from paper_2609_23733_amd import vp
    plan = vp.TomePlan(S, P, M, want_best=True)
    vp.tome_plan(K.cuda(), plan)
    torch.cuda.synchronize()
    return plan


def expected_csr(row, kept, nrows):
    N = row.shape[0]
    order = np.lexsort((np.arange(N), ~kept, row))   # by row, own token first, then tokens
    starts = np.concatenate([[0], np.cumsum(np.bincount(row, minlength=nrows))])
    return order, starts


def check_plan(K, S, P, M, plan, label, srcs_sample=None):
    """Validity of the GPU's decisions, exactness of everything derived from
    them.  Returns the GPU's merged flags over the sources."""
    N = S * P
    row = plan.row.cpu().numpy().astype(np.int64)
    rs = plan.row_start.cpu().numpy().astype(np.int64)
    mem = plan.members.cpu().numpy().astype(np.int64)
    best = plan.best.cpu().numpy().astype(np.int64)
    score = plan.score.cpu().numpy().astype(np.float64)
    is_dst, _ = oracle.tome_split(S, P, M)
    np.testing.assert_array_equal(best == -1, is_dst)
    srcs = np.nonzero(~is_dst)[0]
    gb = best[srcs]
    merged = row[srcs] == row[gb]
    assert int(merged.sum()) == M, (label, int(merged.sum()), M)
    # the GPU's own selection: merged = the M largest (score, lower token)
    if 0 < M < srcs.shape[0]:
        assert score[srcs][merged].min() >= score[srcs][~merged].max()
    # decisions against the oracle (all sources, or a sample at full size)
    m = oracle.tome_metric(K)
    nm = np.sqrt((m * m).sum(1))
    sel = np.arange(srcs.shape[0]) if srcs_sample is None else srcs_sample
    a, b = srcs[sel], gb[sel]
    den = nm[a] * nm[b]
    cos_g = np.where(den > 0, (m[a] * m[b]).sum(1) / np.where(den > 0, den, 1.0), 0.0)
    err_s = np.abs(score[a] - cos_g).max()
    _, ob, os_ = oracle.tome_match(K, S, P, M, srcs=a)
    gap = (os_ - cos_g).max()
    log("%s: score err %.2e, best-choice gap %.2e, %d of %d choices differ" %
        (label, err_s, gap, int((ob != b).sum()), a.shape[0]))
    assert err_s <= 2e-6 and gap <= 2e-6
    if srcs_sample is None and 0 < M < srcs.shape[0]:
        assert os_[merged].min() >= os_[~merged].max() - 4e-6
    # rows and member lists, exactly, given the GPU's decisions
    r_exp, nrows = oracle.tome_rows(N, srcs, gb, merged)
    assert nrows == plan.nrows == N - M
    np.testing.assert_array_equal(row, r_exp)
    kept = np.ones(N, bool)
    kept[srcs[merged]] = False
    order, starts = expected_csr(row, kept, nrows)
    np.testing.assert_array_equal(rs, starts)
    np.testing.assert_array_equal(mem, order)
    return srcs, gb, merged


@pytest.mark.parametrize("S,P,M", [(3, 15, 12), (3, 15, 5), (4, 1374, 2748), (8, 1374, 8244),
                                   (16, 1374, 19785), (2, 300, 1)])
def test_plan_random(S, P, M):
    log("tome plan S=%d P=%d M=%d" % (S, P, M))
    K = synth.stored(synth.normal((S * P, 16, 64), synth.derive_seed(40, S, M), 1.0), "bf16")
    plan = run_plan(K, S, P, M)
    check_plan(K, S, P, M, plan, "S=%d P=%d M=%d" % (S, P, M))


@pytest.mark.parametrize("S,P,M,nspecial", [(3, 40, 78, 0), (4, 20, 42, 5), (5, 1374, 5472, 5),
                                            (3, 8, 0, 3)])
def test_plan_edges(S, P, M, nspecial):
    """No special tokens; every possible source merged (each later view keeps
    only patch 0: 2 x 39, 3 x 14 and 4 x 1368 sources); nothing merged."""
    from paper_2609_23733_amd import vp
    log("tome edges S=%d P=%d M=%d nspecial=%d" % (S, P, M, nspecial))
    K = synth.stored(synth.normal((S * P, 16, 64), synth.derive_seed(47, S, M), 1.0), "bf16")
    plan = vp.TomePlan(S, P, M, nspecial, want_best=True)
    vp.tome_plan(K.cuda(), plan)
    torch.cuda.synchronize()
    ref = oracle.tome_plan(K, S, P, M, nspecial)
    assert plan.g == ref["g"] and plan.nrows == ref["nrows"] == S * P - M
    best = plan.best.cpu().numpy()
    np.testing.assert_array_equal(best == -1, ref["is_dst"])
    if M == (~ref["is_dst"]).sum():   # every source merged: rows are decided by the choices
        srcs = ref["srcs"]
        r_exp, _ = oracle.tome_rows(S * P, srcs, best[srcs], np.ones(srcs.shape[0], bool))
        np.testing.assert_array_equal(plan.row.cpu().numpy(), r_exp)
    if M == 0:
        np.testing.assert_array_equal(plan.row.cpu().numpy(), np.arange(S * P))
        np.testing.assert_array_equal(plan.members.cpu().numpy(), np.arange(S * P))


def planted_keys(S, P, seed):
    """Random keys; 40 sources are power-of-two multiples of one destination
    (exact cosine ties on both sides), 100 more are noisy copies of other
    destinations with distinct similarities near 1."""
    N = S * P
    K = synth.normal((N, 16, 64), seed, 1.0).float()
    is_dst, _ = oracle.tome_split(S, P, 1)
    rng = np.random.default_rng(seed)
    srcs = np.nonzero(~is_dst)[0]
    dsts = np.nonzero(is_dst)[0]
    pick = rng.choice(srcs, 140, replace=False)
    d0 = dsts[7]
    for i, a in enumerate(pick[:40]):
        K[a] = K[d0] * (2.0 ** (i % 4 - 1))
    eps = np.linspace(0.02, 0.3, 100)
    for a, e, d in zip(pick[40:], eps, rng.choice(dsts, 100)):
        K[a] = K[d] + e * synth.normal((16, 64), int(a), 1.0).float()
    return K.to(torch.bfloat16), sorted(pick[:40])


@pytest.mark.parametrize("M", [20, 40, 100])
def test_plan_planted_exact(M):
    """Unique decisions: the whole plan equals the oracle's; with M = 20 the
    threshold falls inside the tied group, which is cut by token index."""
    S, P = 4, 1374
    log("tome planted M=%d" % M)
    K, tied = planted_keys(S, P, 41)
    plan = run_plan(K, S, P, M)
    srcs, gb, merged = check_plan(K, S, P, M, plan, "planted M=%d" % M)
    ref = oracle.tome_plan(K, S, P, M)
    np.testing.assert_array_equal(merged, ref["merged"])
    np.testing.assert_array_equal(gb[merged], ref["best"][ref["merged"]])
    np.testing.assert_array_equal(plan.row.cpu().numpy(), ref["row"])
    if M == 20:
        assert set(srcs[merged]) == set(tied[:20])


def merged_bound(ref, sizes, X_abs_max, bf16):
    """A row of c tokens: fp32 sums err by at most c 2^-24 max|X| (bound with
    a factor 2), the division and the output rounding by half an ulp."""
    c = np.asarray(sizes, np.float64).reshape((-1,) + (1,) * (ref.ndim - 1))
    sums = c * 2.0 ** -23 * X_abs_max
    return (2.0 ** -8 if bf16 else 2.0 ** -23) * np.abs(ref) + sums + 1e-30


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_merge_unmerge(dtype):
    from paper_2609_23733_amd import vp
    S, P, M = 8, 1374, 8244
    log("tome merge/unmerge %s" % dtype)
    K = synth.stored(synth.normal((S * P, 16, 64), 42, 1.0), "bf16")
    plan = run_plan(K, S, P, M)
    X = synth.stored(synth.normal((S * P, 16, 64), 43, 1.0), dtype)
    Xm = vp.tome_merge(X.cuda(), plan)
    back = vp.tome_unmerge(Xm, plan)
    torch.cuda.synchronize()
    row = plan.row.cpu().numpy().astype(np.int64)
    ref = oracle.tome_merge(X, row, plan.nrows)
    g = Xm.double().cpu().numpy()
    err = np.abs(g - ref)
    sizes = np.bincount(row, minlength=plan.nrows)
    bound = merged_bound(ref, sizes, float(X.float().abs().max()), dtype == "bf16")
    log("merge worst err/bound = %.3f" % float((err / bound).max()))
    assert (err <= bound).all()
    assert torch.equal(back, Xm[plan.row.long()])
    if dtype == "bf16":   # the fused Q/K/V merge gives the same rows, bitwise
        X2 = synth.stored(synth.normal((S * P, 16, 64), 44, 1.0), dtype).cuda()
        X3 = synth.stored(synth.normal((S * P, 16, 64), 45, 1.0), dtype).cuda()
        out = [torch.empty_like(Xm) for _ in range(3)]
        vp.tome_merge_qkv(X.cuda(), X2, X3, plan, *out)
        assert torch.equal(out[0], Xm) and torch.equal(out[1], vp.tome_merge(X2, plan))
        assert torch.equal(out[2], vp.tome_merge(X3, plan))
    # deterministic: a second plan and merge are bitwise equal
    plan2 = run_plan(K, S, P, M)
    assert torch.equal(plan2.members, plan.members) and torch.equal(plan2.row, plan.row)
    assert torch.equal(vp.tome_merge(X.cuda(), plan2), Xm)


def test_tome_layer_small():
    """Plan, merge, routed layer on the merged rows and unmerge, against the
    oracle's routed layer on the merged rows."""
    from paper_2609_23733_amd import vp
    S, M = 4, 2748
    log("tome layer S=4")
    x = synth.make_layer(S, dtype="bf16", n_full=4, key=(44, 0))
    tl = vp.TomeLayer(x, M, want_best=True, y_dtype=torch.bfloat16)
    Y = tl.step()
    torch.cuda.synchronize()
    check_plan(x.K, S, synth.TOKENS_PER_VIEW, M, tl.plan, "layer plan")
    row = tl.plan.row.cpu().numpy().astype(np.int64)
    sizes = np.bincount(row, minlength=tl.plan.nrows)
    for nm_, X, Xm in (("Q", x.Q, tl.Qm), ("K", x.K, tl.Km), ("V", x.V, tl.Vm)):
        ref = oracle.tome_merge(X, row, tl.plan.nrows)
        err = np.abs(Xm.double().cpu().numpy() - ref)
        assert (err <= merged_bound(ref, sizes, float(X.float().abs().max()), True)).all(), nm_
    xm = dataclasses.replace(x, S=1, P=tl.plan.nrows, Q=tl.Qm.cpu(), K=tl.Km.cpu(),
                             V=tl.Vm.cpu())
    ref = oracle_layer(xm)
    np.testing.assert_array_equal(tl.layer.modes.cpu().numpy(), ref["modes"])
    check_y(tl.layer.Y.double().cpu().numpy(), ref["Y"], "bf16", True, label="tome layer S=4")
    assert torch.equal(Y, tl.layer.Y[tl.plan.row.long()])


@pytest.mark.parametrize("ratio", [0.75, 0.9])
def test_tome_full_size_sampled(ratio):
    """S = 100 views (N = 137,400) at the paper's merging ratios: decisions of
    512 sampled sources against the oracle, rows and member lists of every
    token exactly, merged rows and the layer's output on 64 sampled rows."""
    from paper_2609_23733_amd import vp
    S, P = 100, synth.TOKENS_PER_VIEW
    N = S * P
    M = int(ratio * N)
    log("tome full size ratio %.2f" % ratio)
    x = synth.make_layer(S, dtype="bf16", n_full=4, key=(S, 0), qkv_device="cuda")
    tl = vp.TomeLayer(x, M, want_best=True, y_dtype=torch.bfloat16)
    Y = tl.step()
    torch.cuda.synchronize()
    Kc = x.K.cpu()
    is_dst, _ = oracle.tome_split(S, P, M)
    nsrc = int((~is_dst).sum())
    sample = synth.sample_rows(nsrc, 512, synth.derive_seed(S, 45, int(ratio * 100)))
    check_plan(Kc, S, P, M, tl.plan, "full ratio %.2f" % ratio, srcs_sample=sample)
    # merged rows on a sample of rows
    rs = tl.plan.row_start.cpu().numpy().astype(np.int64)
    mem = tl.plan.members.cpu().numpy().astype(np.int64)
    rows = synth.sample_rows(tl.plan.nrows, 64, synth.derive_seed(S, 46, int(ratio * 100)))
    toks = np.concatenate([mem[rs[r]:rs[r + 1]] for r in rows])
    lab = np.concatenate([np.full(rs[r + 1] - rs[r], i) for i, r in enumerate(rows)])
    for nm_, X, Xm in (("Q", x.Q, tl.Qm), ("K", x.K, tl.Km), ("V", x.V, tl.Vm)):
        Xs = X[torch.from_numpy(toks).cuda()].cpu()
        ref = oracle.tome_merge(Xs, lab, rows.shape[0])
        g = Xm[torch.from_numpy(rows).cuda()].double().cpu().numpy()
        bound = merged_bound(ref, rs[rows + 1] - rs[rows], float(Xs.float().abs().max()), True)
        assert (np.abs(g - ref) <= bound).all(), nm_
    # the layer on the merged rows: router and modes on all rows, outputs on the sample
    xm = dataclasses.replace(x, S=1, P=tl.plan.nrows, Q=tl.Qm.cpu(), K=tl.Km.cpu(),
                             V=tl.Vm.cpu())
    ref = oracle_layer(xm, rows=rows, full_rows_sel=rows)
    np.testing.assert_array_equal(tl.layer.modes.cpu().numpy(), ref["modes"])
    for h in range(16):
        if ref["modes"][h] == 2:
            ref["Y"][:, h, :] = ref["Y_full_rows"][h]
    Yg = tl.layer.Y[torch.from_numpy(rows).cuda()].double().cpu().numpy()
    check_y(Yg, ref["Y"], "bf16", True, label="tome full ratio %.2f" % ratio)
    assert torch.equal(Y, tl.layer.Y[tl.plan.row.long()])
