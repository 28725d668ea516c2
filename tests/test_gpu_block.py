"""GPU parity of the dense block around the routed layer (Algorithm 1 steps
1, 3, 4) against the fp64 oracle, through the C ABI.

Bars (bf16 operands and outputs, fp32 arithmetic):
  - Q, K, V of vp_block_qkv: the layer's bound, max |err| <= 2e-2 * RMS +
    2^-8 |ref| (RMS the smaller of the head's and the layer's), per head;
  - vp_block_out: on the block's update U = X_out - X, max |err| <= 2e-2 *
    RMS(U_ref) + 2^-8 |X_out_ref| (the half-ulp of the stored output);
  - the whole block (qkv, routed layer, out) against the oracle's
    composition: the same bar on the update.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_23733_amd import synth
from test_gpu_parity import check_y, log, rms

pytestmark = pytest.mark.gpu

D = 1024


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_23733_amd import vp
    vp.load_library()


def weights(key):
    return {k: v.cuda() for k, v in synth.make_block_weights(key).items()}


def check_update(out_g, X, ref, label, rows=None):
    """out_g: GPU block output [R, D]; X: block input rows [R, D] (stored);
    ref: oracle block output rows [R, D] float64."""
    Xs = X.double().cpu().numpy()
    g = out_g.double().cpu().numpy()
    U_ref = ref - Xs
    bound = 2e-2 * rms(U_ref) + 2.0 ** -8 * np.abs(ref)
    err = np.abs((g - Xs) - U_ref)
    ratio = float((err / bound).max())
    log("%s worst err/bound = %.3f (update rms %.3e)" % (label, ratio, rms(U_ref)))
    assert (err <= bound).all(), "%s: max err %.3e, ratio %.3f" % (label, err.max(), ratio)


@pytest.mark.parametrize("S,P", [(1, 1), (1, 5), (1, 256), (1, 300), (1, 513), (1, 1374), (2, 1374)])
def test_block_qkv(S, P):
    from paper_2609_23733_amd import vp
    log("block qkv S=%d P=%d" % (S, P))
    wt = synth.make_block_weights((20, P))
    X = synth.make_block_input(S, P, key=(20, P))
    pos = synth.token_positions(S, P)
    ws = torch.empty(vp.block_workspace_bytes(S, P), dtype=torch.uint8, device="cuda")
    Q, K, V = vp.block_qkv(X.cuda(), torch.from_numpy(pos).cuda(),
                           {k: v.cuda() for k, v in wt.items()}, S, P, ws)
    torch.cuda.synchronize()
    rq, rk, rv = oracle.block_qkv(X, pos, wt)
    for nm, g, r in (("Q", Q, rq), ("K", K, rk), ("V", V, rv)):
        check_y(g.double().cpu().numpy(), r, "bf16", True, label="qkv %s S=%d P=%d" % (nm, S, P))


@pytest.mark.parametrize("S,P", [(1, 1), (1, 255), (1, 300), (1, 513), (2, 1374)])
def test_block_out(S, P):
    from paper_2609_23733_amd import vp
    log("block out S=%d P=%d" % (S, P))
    wt = synth.make_block_weights((21, P))
    X = synth.make_block_input(S, P, key=(21, P))
    Y = synth.stored(synth.normal((S * P, D), synth.derive_seed(21, P, 99), 0.1), "bf16")
    ws = torch.empty(vp.block_workspace_bytes(S, P), dtype=torch.uint8, device="cuda")
    out = vp.block_out(X.cuda(), Y.cuda(), {k: v.cuda() for k, v in wt.items()}, S, P, ws)
    torch.cuda.synchronize()
    ref, _ = oracle.block_out(X, Y, wt)
    check_update(out, X, ref, "out S=%d P=%d" % (S, P))


def test_block_out_in_place():
    """X_out may be X itself."""
    from paper_2609_23733_amd import vp
    log("block out in place")
    wt = {k: v.cuda() for k, v in synth.make_block_weights((22, 0)).items()}
    X = synth.make_block_input(1, 700, key=(22, 0)).cuda()
    Y = synth.stored(synth.normal((700, D), 5, 0.1), "bf16").cuda()
    ws = torch.empty(vp.block_workspace_bytes(1, 700), dtype=torch.uint8, device="cuda")
    a = vp.block_out(X, Y, wt, 1, 700, ws)
    Xc = X.clone()
    vp.block_out(Xc, Y, wt, 1, 700, ws, X_out=Xc)
    torch.cuda.synchronize()
    assert torch.equal(a, Xc)


def test_block_full_size_sampled():
    """S = 100 views (N = 137,400): both stages on every token, compared on 64
    sampled rows (each output row depends only on its own input row)."""
    from paper_2609_23733_amd import vp
    S, P = 100, synth.TOKENS_PER_VIEW
    N = S * P
    log("block full size S=100")
    wt = synth.make_block_weights((23, 0))
    wd = {k: v.cuda() for k, v in wt.items()}
    X = synth.make_block_input(S, P, key=(23, 0), device="cuda")
    pos = synth.token_positions(S, P)
    ws = torch.empty(vp.block_workspace_bytes(S, P), dtype=torch.uint8, device="cuda")
    Q, K, V = vp.block_qkv(X, torch.from_numpy(pos).cuda(), wd, S, P, ws)
    Y = synth.stored(synth.normal((N, D), synth.derive_seed(23, 0, 99), 0.1, "cuda"), "bf16")
    out = vp.block_out(X, Y, wd, S, P, ws)
    torch.cuda.synchronize()
    rows = synth.sample_rows(N, 64, synth.derive_seed(23, 0, 20))
    rt = torch.from_numpy(rows).cuda()
    Xr = X[rt].cpu()
    rq, rk, rv = oracle.block_qkv(Xr, pos[rows], wt)
    for nm, g, r in (("Q", Q, rq), ("K", K, rk), ("V", V, rv)):
        check_y(g[rt].double().cpu().numpy(), r, "bf16", True, label="S=100 %s" % nm)
    ref, _ = oracle.block_out(Xr, Y[rt].cpu(), wt)
    check_update(out[rt], Xr, ref, "S=100 out")


def test_block_element_offsets_past_2_32():
    """N = 3053 x 1374 = 4,194,822 tokens: the FFN's 4096-wide hidden rows
    pass 2^32 elements from token 2^20 on, the 1024-wide rows of X, Q, K, V
    and the update from token 2^22.  Both stages on every token; sampled rows
    on both sides of both boundaries and the last row."""
    from paper_2609_23733_amd import vp
    S, P = 3053, synth.TOKENS_PER_VIEW
    N = S * P
    log("block element offsets past 2^32: N=%d" % N)
    wt = synth.make_block_weights((25, 0))
    wd = {k: v.cuda() for k, v in wt.items()}
    X = synth.make_block_input(S, P, key=(25, 0), device="cuda")
    pos = synth.token_positions(S, P)
    ws = torch.empty(vp.block_workspace_bytes(S, P), dtype=torch.uint8, device="cuda")
    Q, K, V = vp.block_qkv(X, torch.from_numpy(pos).cuda(), wd, S, P, ws)
    Y = synth.stored(synth.normal((N, D), synth.derive_seed(25, 0, 99), 0.1, "cuda"), "bf16")
    out = vp.block_out(X, Y, wd, S, P, ws)
    torch.cuda.synchronize()
    edges = [2 ** 20 - 1, 2 ** 20, 2 ** 22 - 1, 2 ** 22, N - 2, N - 1]
    rows = np.unique(np.concatenate([synth.sample_rows(N, 26, synth.derive_seed(25, 0, 20)),
                                     np.array(edges)])).astype(np.int64)
    rt = torch.from_numpy(rows).cuda()
    Xr = X[rt].cpu()
    rq, rk, rv = oracle.block_qkv(Xr, pos[rows], wt)
    for nm, g, r in (("Q", Q, rq), ("K", K, rk), ("V", V, rv)):
        check_y(g[rt].double().cpu().numpy(), r, "bf16", True, label="N=%d %s" % (N, nm))
    ref, _ = oracle.block_out(Xr, Y[rt].cpu(), wt)
    check_update(out[rt], Xr, ref, "N=%d out" % N)


@pytest.mark.parametrize("dtype_note", ["bf16"])
def test_whole_block(dtype_note):
    """qkv -> routed layer (router, modes, attention) -> out, against the
    oracle's composition of the same steps; the mode router is steered to a
    fixed mix with margins, so both sides route identically."""
    from paper_2609_23733_amd import vp
    S, P = 2, synth.TOKENS_PER_VIEW
    log("whole block S=2")
    modes = np.array([2, 1, 0, 2, 2, 1, 0, 0, 1, 2, 0, 1, 2, 0, 1, 2], np.uint8)
    lay = synth.make_layer(S, P, dtype="bf16", key=(24, 0), modes=modes)
    wt = synth.make_block_weights((24, 0))
    X = synth.make_block_input(S, P, key=(24, 0))
    pos = synth.token_positions(S, P)
    blk = vp.PrimeBlock(lay, wt, pos)
    out = blk.step(X.cuda())
    out2 = blk.step(X.cuda())
    torch.cuda.synchronize()
    assert torch.equal(out, out2)
    np.testing.assert_array_equal(blk.layer.modes.cpu().numpy(), modes)
    rq, rk, rv = oracle.block_qkv(X, pos, wt)
    ref_l = oracle.routed_layer(rq, rk, rv, lay.W, lay.U, lay.w, lay.surr, u=lay.u, Wr=lay.Wr,
                                br=lay.br, rule=oracle.RULE_ARGMAX)
    np.testing.assert_array_equal(ref_l["modes"], modes)
    ref, _ = oracle.block_out(X, ref_l["Y"].reshape(S * P, D), wt)
    check_update(out, X, ref, "whole block")


def test_whole_block_tome():
    """The block with token merging before its routed layer: qkv on all
    tokens, the plan on the block's K, the routed layer on the merged rows,
    unmerge, out -- against the oracle's composition of the same steps with
    the GPU's merge decisions (checked for validity against the oracle)."""
    from paper_2609_23733_amd import vp
    from test_gpu_tome import check_plan
    S, P = 4, synth.TOKENS_PER_VIEW
    M = (S * P) // 2
    log("whole block with token merging S=4")
    modes = np.array([2, 1, 0, 2, 2, 1, 0, 0, 1, 2, 0, 1, 2, 0, 1, 2], np.uint8)
    lay = synth.make_layer(S, P, dtype="bf16", key=(25, 0), modes=modes)
    wt = synth.make_block_weights((25, 0))
    X = synth.make_block_input(S, P, key=(25, 0))
    pos = synth.token_positions(S, P)
    blk = vp.PrimeBlock(lay, wt, pos, tome_M=M)
    blk.tome.plan = vp.TomePlan(S, P, M, want_best=True)
    out = blk.step(X.cuda())
    torch.cuda.synchronize()
    check_plan(blk.K.cpu(), S, P, M, blk.tome.plan, "block plan")
    row = blk.tome.plan.row.cpu().numpy().astype(np.int64)
    nrows = blk.tome.plan.nrows
    rq, rk, rv = oracle.block_qkv(X, pos, wt)
    mq, mk, mv = (oracle.tome_merge(t.astype(np.float32), row, nrows) for t in (rq, rk, rv))
    ref_l = oracle.routed_layer(mq, mk, mv, lay.W, lay.U, lay.w, lay.surr, u=lay.u, Wr=lay.Wr,
                                br=lay.br, rule=oracle.RULE_ARGMAX)
    np.testing.assert_array_equal(ref_l["modes"], modes)
    Y = oracle.tome_unmerge(ref_l["Y"], row)
    ref, _ = oracle.block_out(X, Y.reshape(S * P, D), wt)
    check_update(out, X, ref, "whole block with merging")

