"""The C-ABI library loads, exports every symbol the header declares, and
rejects bad arguments on the host before anything is enqueued (CPU only:
every call here fails validation, so no kernel is launched)."""
import ctypes
import os
import re

import pytest
import torch

from paper_2609_23733_amd import vp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vggt_prime.h")

FAKE = 0x10000          # 256-byte aligned fake device address (never dereferenced)
FAKE_ODD = 0x10002      # misaligned


def header_functions():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(vp_\w+)\s*\(", txt, re.M)))


@pytest.fixture(scope="module")
def lib():
    return vp.load_library()


def test_exports_every_declared_symbol(lib):
    names = header_functions()
    assert set(names) == set(vp.EXPORTS)
    for n in names:
        assert getattr(lib, n) is not None


def test_status_strings(lib):
    for code in range(5):
        assert lib.vp_status_string(code)
    assert lib.vp_last_error() == b""


def shape(S=2, P=1374, H=16, d=64, dt=vp.VP_BF16):
    return vp.vp_shape(S, P, H, d, dt)


def test_workspace_bytes(lib):
    f = lambda s: lib.vp_workspace_bytes(ctypes.byref(s))
    assert f(shape(S=0)) == 0
    assert f(shape(H=17)) == 0
    assert f(shape(d=32)) == 0
    assert f(shape(dt=7)) == 0
    a, b = f(shape(S=2)), f(shape(S=8))
    assert 0 < a < b
    assert a % 256 == 0
    # bf16 needs room for the packed values of up to H FULL heads
    assert f(shape(dt=vp.VP_BF16)) > f(shape(dt=vp.VP_F32))


def rw(L=64, W=FAKE, scale=0.0, pool=vp.POOL_GATED):
    return vp.vp_router_weights(W, FAKE, FAKE, L, scale, pool)


def rs(q=FAKE):
    return vp.vp_router_state(q, FAKE, FAKE, FAKE, FAKE)


def call_score(lib, shp=None, Q=FAKE, w=None, st=None, ws=FAKE, ws_bytes=1 << 40):
    shp = shp or shape()
    w = w or rw()
    st = st or rs()
    return lib.vp_router_score(ctypes.byref(shp), Q, FAKE, FAKE, ctypes.byref(w), ctypes.byref(st),
                               ws, ws_bytes, None)


def test_router_score_validation(lib):
    assert call_score(lib, shp=shape(S=0)) == vp.VP_ERR_INVALID_ARG
    assert call_score(lib, shp=shape(H=0)) == vp.VP_ERR_INVALID_ARG
    assert call_score(lib, shp=shape(H=17)) == vp.VP_ERR_UNSUPPORTED
    assert call_score(lib, shp=shape(d=128)) == vp.VP_ERR_UNSUPPORTED
    assert call_score(lib, shp=shape(S=1 << 20, P=1 << 10)) == vp.VP_ERR_UNSUPPORTED
    assert call_score(lib, shp=shape(dt=5)) == vp.VP_ERR_INVALID_ARG
    assert call_score(lib, Q=None) == vp.VP_ERR_INVALID_ARG
    assert call_score(lib, Q=FAKE_ODD) == vp.VP_ERR_INVALID_ARG
    assert call_score(lib, w=rw(W=None)) == vp.VP_ERR_INVALID_ARG
    assert call_score(lib, w=rw(L=32)) == vp.VP_ERR_UNSUPPORTED
    assert call_score(lib, w=rw(scale=float("nan"))) == vp.VP_ERR_INVALID_ARG
    assert call_score(lib, st=rs(q=None)) == vp.VP_ERR_INVALID_ARG
    assert call_score(lib, ws=None) == vp.VP_ERR_INVALID_ARG
    assert call_score(lib, ws=FAKE + 64) == vp.VP_ERR_INVALID_ARG
    assert call_score(lib, ws_bytes=1024) == vp.VP_ERR_WORKSPACE
    assert lib.vp_router_score(None, FAKE, FAKE, FAKE, None, None, FAKE, 1 << 40, None) == \
        vp.VP_ERR_INVALID_ARG
    # pooling mode: unknown values are rejected; the mean query reads no W, U, w
    # (a NULL W then passes validation and the next check, the workspace, fails)
    assert call_score(lib, w=rw(pool=2)) == vp.VP_ERR_INVALID_ARG
    assert call_score(lib, w=rw(pool=-1)) == vp.VP_ERR_INVALID_ARG
    assert call_score(lib, w=rw(W=None, pool=vp.POOL_MEAN), ws_bytes=1024) == \
        vp.VP_ERR_WORKSPACE
    assert call_score(lib, w=rw(W=None, pool=vp.POOL_GATED), ws_bytes=1024) == \
        vp.VP_ERR_INVALID_ARG


def test_router_score_noalloc_validation(lib):
    """The allocation-free router rejects the same arguments as vp_router_score
    on the host, before it looks up its scratch or enqueues anything."""
    f = lambda shp=None, Q=FAKE, w=None, st=None: lib.vp_router_score_noalloc(
        ctypes.byref(shp or shape()), Q, FAKE, FAKE, ctypes.byref(w or rw()),
        ctypes.byref(st or rs()), None)
    assert f(shp=shape(S=0)) == vp.VP_ERR_INVALID_ARG
    assert f(shp=shape(H=17)) == vp.VP_ERR_UNSUPPORTED
    assert f(shp=shape(d=128)) == vp.VP_ERR_UNSUPPORTED
    assert f(shp=shape(S=1 << 20, P=1 << 10)) == vp.VP_ERR_UNSUPPORTED
    assert f(Q=None) == vp.VP_ERR_INVALID_ARG
    assert f(Q=FAKE_ODD) == vp.VP_ERR_INVALID_ARG
    assert f(w=rw(W=None)) == vp.VP_ERR_INVALID_ARG
    assert f(w=rw(L=32)) == vp.VP_ERR_UNSUPPORTED
    assert f(w=rw(pool=2)) == vp.VP_ERR_INVALID_ARG
    assert f(st=rs(q=None)) == vp.VP_ERR_INVALID_ARG
    assert lib.vp_router_score_noalloc(None, FAKE, FAKE, FAKE, None, None, None) == \
        vp.VP_ERR_INVALID_ARG


def test_router_logits_validation(lib):
    f = lib.vp_router_logits
    B = vp.VP_BF16
    assert f(None, FAKE, FAKE, 16, 1024, 3, B, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, None, FAKE, 16, 1024, 3, B, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, FAKE, FAKE, 0, 1024, 3, B, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, FAKE, FAKE, 17, 1024, 3, B, FAKE, None) == vp.VP_ERR_UNSUPPORTED
    assert f(FAKE, FAKE, FAKE, 16, 0, 3, B, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, FAKE, FAKE, 16, 1 << 20, 3, B, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, FAKE, FAKE, 16, 1024, 3, 9, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE + 1, FAKE, FAKE, 16, 1024, 3, B, FAKE, None) == vp.VP_ERR_INVALID_ARG
    # M: the number of modes, which Eq.4 fixes at 3
    assert f(FAKE, FAKE, FAKE, 16, 1024, 0, B, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, FAKE, FAKE, 16, 1024, 2, B, FAKE, None) == vp.VP_ERR_UNSUPPORTED
    assert f(FAKE, FAKE, FAKE, 16, 1024, 4, B, FAKE, None) == vp.VP_ERR_UNSUPPORTED


def test_assign_validation(lib):
    f = lib.vp_assign_heads
    T, A = vp.RULE_THRESHOLD, vp.RULE_ARGMAX
    assert f(None, 16, 1, T, 0.01, 0.2, FAKE, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, 16, 1, T, 0.01, 0.2, None, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, 16, 1, T, 0.01, 0.2, FAKE, None, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, 0, 1, T, 0.01, 0.2, FAKE, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, 17, 1, T, 0.01, 0.2, FAKE, FAKE, None) == vp.VP_ERR_UNSUPPORTED
    assert f(FAKE, 16, 1, 4, 0.01, 0.2, FAKE, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, 16, 1, -1, 0.01, 0.2, FAKE, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, 16, 1, T, 0.3, 0.2, FAKE, FAKE, None) == vp.VP_ERR_INVALID_ARG
    # the binary threshold rule checks its thresholds like Eq.4 does
    assert f(FAKE, 16, 1, vp.RULE_THRESHOLD_BINARY, 0.3, 0.2, FAKE, FAKE, None) == \
        vp.VP_ERR_INVALID_ARG
    assert f(FAKE, 16, 1, vp.RULE_THRESHOLD_BINARY, 0.01, float("inf"), FAKE, FAKE, None) == \
        vp.VP_ERR_INVALID_ARG
    assert f(FAKE, 16, 1, T, -0.1, 0.2, FAKE, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, 16, 1, T, float("nan"), 0.2, FAKE, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE + 2, 16, 1, T, 0.01, 0.2, FAKE, FAKE, None) == vp.VP_ERR_INVALID_ARG
    # M: one score per head for the threshold rules, three logits for argmax
    assert f(FAKE, 16, 0, T, 0.01, 0.2, FAKE, FAKE, None) == vp.VP_ERR_INVALID_ARG
    assert f(FAKE, 16, 3, T, 0.01, 0.2, FAKE, FAKE, None) == vp.VP_ERR_UNSUPPORTED
    assert f(FAKE, 16, 3, vp.RULE_THRESHOLD_BINARY, 0.01, 0.2, FAKE, FAKE, None) == \
        vp.VP_ERR_UNSUPPORTED
    assert f(FAKE, 16, 1, A, 0.01, 0.2, FAKE, FAKE, None) == vp.VP_ERR_UNSUPPORTED
    assert f(FAKE, 16, 2, vp.RULE_ARGMAX_BINARY, 0.01, 0.2, FAKE, FAKE, None) == \
        vp.VP_ERR_UNSUPPORTED


def sw(L=64, act=0, g_w1=FAKE, variant=vp.SURR_EQ7):
    return vp.vp_surrogate_weights(g_w1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, L, act,
                                   variant)


def call_attn(lib, shp=None, Q=FAKE, modes=FAKE, st=None, s=None, Y=FAKE, ydt=vp.VP_BF16,
              ws=FAKE, ws_bytes=1 << 40):
    shp = shp or shape()
    st = st or rs()
    s = s or sw()
    return lib.vp_routed_global_attention(ctypes.byref(shp), Q, FAKE, FAKE, modes, FAKE,
                                          ctypes.byref(st), ctypes.byref(s), Y, ydt, ws, ws_bytes,
                                          None)


def test_routed_attention_validation(lib):
    assert call_attn(lib, shp=shape(P=0)) == vp.VP_ERR_INVALID_ARG
    assert call_attn(lib, shp=shape(H=20)) == vp.VP_ERR_UNSUPPORTED
    assert call_attn(lib, Q=None) == vp.VP_ERR_INVALID_ARG
    assert call_attn(lib, modes=None) == vp.VP_ERR_INVALID_ARG
    assert call_attn(lib, Y=None) == vp.VP_ERR_INVALID_ARG
    assert call_attn(lib, Y=FAKE + 8) == vp.VP_ERR_INVALID_ARG
    assert call_attn(lib, ydt=3) == vp.VP_ERR_INVALID_ARG
    assert call_attn(lib, s=sw(L=16)) == vp.VP_ERR_UNSUPPORTED
    assert call_attn(lib, s=sw(act=7)) == vp.VP_ERR_INVALID_ARG
    assert call_attn(lib, s=sw(g_w1=None)) == vp.VP_ERR_INVALID_ARG
    assert call_attn(lib, ws_bytes=10) == vp.VP_ERR_WORKSPACE
    assert lib.vp_routed_global_attention(ctypes.byref(shape()), FAKE, FAKE, FAKE, FAKE, FAKE,
                                          None, ctypes.byref(sw()), FAKE, 1, FAKE, 1 << 40,
                                          None) == vp.VP_ERR_INVALID_ARG
    # surrogate variants: unknown values are rejected; the weight-free ablations
    # accept NULL weights (the workspace check fails next), the others do not
    assert call_attn(lib, s=sw(variant=5)) == vp.VP_ERR_INVALID_ARG
    assert call_attn(lib, s=sw(variant=-1)) == vp.VP_ERR_INVALID_ARG
    for v in (vp.SURR_NO_RESIDUAL, vp.SURR_LINEAR_ATTN):
        assert call_attn(lib, s=sw(g_w1=None, variant=v), ws_bytes=10) == vp.VP_ERR_WORKSPACE
    for v in (vp.SURR_EQ7, vp.SURR_MEAN_CONTEXT, vp.SURR_ADD_IDENTITY):
        assert call_attn(lib, s=sw(g_w1=None, variant=v), ws_bytes=10) == vp.VP_ERR_INVALID_ARG


def call_linear(lib, Q=FAKE, s=None, ws=FAKE, ws_bytes=1 << 40):
    s = s or sw()
    return lib.vp_linear_heads(ctypes.byref(shape()), Q, FAKE, FAKE, FAKE, ctypes.byref(rs()),
                               ctypes.byref(s), FAKE, vp.VP_BF16, ws, ws_bytes, None)


def test_linear_heads_validation(lib):
    lin = sw(variant=vp.SURR_LINEAR_ATTN)
    # linear attention reads Q and K and keeps its sums in the workspace
    assert call_linear(lib, Q=None, s=lin) == vp.VP_ERR_INVALID_ARG
    assert call_linear(lib, Q=FAKE_ODD, s=lin) == vp.VP_ERR_INVALID_ARG
    assert call_linear(lib, ws=None, s=lin) == vp.VP_ERR_INVALID_ARG
    assert call_linear(lib, ws_bytes=10, s=lin) == vp.VP_ERR_WORKSPACE
    assert call_linear(lib, s=sw(variant=9)) == vp.VP_ERR_INVALID_ARG
    assert call_linear(lib, s=sw(act=3)) == vp.VP_ERR_INVALID_ARG
    assert lib.vp_linear_heads(ctypes.byref(shape()), FAKE, FAKE, FAKE, FAKE, None,
                               ctypes.byref(sw()), FAKE, vp.VP_BF16, FAKE, 1 << 40, None) == \
        vp.VP_ERR_INVALID_ARG


def test_binding_rejects_cpu_tensors():
    x = torch.zeros(4, 16, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        vp.router_score(x, x, x, torch.zeros(16, 64, 64, dtype=torch.bfloat16),
                        torch.zeros(16, 64, 64, dtype=torch.bfloat16),
                        torch.zeros(16, 64, dtype=torch.bfloat16), 1, 4,
                        torch.zeros(10, dtype=torch.uint8))


# ------------------------------------------------------------------ block

def bw(mat=FAKE, vec=FAKE, eps=0.0, base=0.0):
    f = dict(ln1_w=vec, ln1_b=vec, w_qkv=mat, b_qkv=vec, w_o=mat, b_o=vec, ls1=vec, ln2_w=vec,
             ln2_b=vec, w_fc1=mat, b_fc1=vec, w_fc2=mat, b_fc2=vec, ls2=vec, ln_eps=eps,
             rope_base=base)
    return vp.vp_block_weights(**f)


def test_block_workspace_bytes(lib):
    f = lambda s: lib.vp_block_workspace_bytes(ctypes.byref(s))
    assert f(shape(dt=vp.VP_F32)) == 0          # bf16 layers only
    assert f(shape(H=8)) == 0                   # model width 1024 only
    assert f(shape(S=0)) == 0
    n = f(shape(S=2, P=1374))
    assert n >= 2 * 1374 * 1024 * 2 * 6 and n % 256 == 0


def call_qkv(lib, shp=None, X=FAKE, pos=FAKE, w=None, Q=FAKE, ws=FAKE, ws_bytes=1 << 40):
    return lib.vp_block_qkv(ctypes.byref(shp or shape()), X, pos, ctypes.byref(w or bw()), Q,
                            FAKE, FAKE, ws, ws_bytes, None)


def call_out(lib, shp=None, X=FAKE, Y=FAKE, w=None, Xo=FAKE, ws=FAKE, ws_bytes=1 << 40):
    return lib.vp_block_out(ctypes.byref(shp or shape()), X, Y, ctypes.byref(w or bw()), Xo, ws,
                            ws_bytes, None)


def test_block_validation(lib):
    for call in (call_qkv, call_out):
        assert call(lib, shp=shape(dt=vp.VP_F32)) == vp.VP_ERR_UNSUPPORTED
        assert call(lib, shp=shape(H=4)) == vp.VP_ERR_UNSUPPORTED
        assert call(lib, shp=shape(P=0)) == vp.VP_ERR_INVALID_ARG
        assert call(lib, X=None) == vp.VP_ERR_INVALID_ARG
        assert call(lib, X=FAKE_ODD) == vp.VP_ERR_INVALID_ARG
        assert call(lib, w=bw(mat=None)) == vp.VP_ERR_INVALID_ARG
        assert call(lib, w=bw(mat=FAKE + 8)) == vp.VP_ERR_INVALID_ARG
        assert call(lib, w=bw(vec=None)) == vp.VP_ERR_INVALID_ARG
        assert call(lib, w=bw(vec=FAKE + 2)) == vp.VP_ERR_INVALID_ARG
        assert call(lib, w=bw(eps=-1.0)) == vp.VP_ERR_INVALID_ARG
        assert call(lib, w=bw(eps=float("nan"))) == vp.VP_ERR_INVALID_ARG
        assert call(lib, w=bw(base=0.5)) == vp.VP_ERR_INVALID_ARG
        assert call(lib, ws=None) == vp.VP_ERR_INVALID_ARG
        assert call(lib, ws=FAKE + 16) == vp.VP_ERR_INVALID_ARG
        assert call(lib, ws_bytes=1024) == vp.VP_ERR_WORKSPACE
    assert call_qkv(lib, pos=None) == vp.VP_ERR_INVALID_ARG
    assert call_qkv(lib, pos=FAKE + 4) == vp.VP_ERR_INVALID_ARG
    assert call_qkv(lib, Q=None) == vp.VP_ERR_INVALID_ARG
    assert call_out(lib, Y=None) == vp.VP_ERR_INVALID_ARG
    assert call_out(lib, Xo=FAKE + 2) == vp.VP_ERR_INVALID_ARG


# ------------------------------------------------------- distillation

def test_distill_validation(lib):
    f = lambda s: lib.vp_teacher_workspace_bytes(ctypes.byref(s))
    assert f(shape(dt=vp.VP_F32)) == 0 and f(shape()) > lib.vp_workspace_bytes(ctypes.byref(shape()))
    assert lib.vp_loss_workspace_bytes(ctypes.byref(shape())) > 0
    tt = lambda shp=None, Q=FAKE, cm=FAKE, ydt=vp.VP_BF16, ws=FAKE, nb=1 << 40: \
        lib.vp_teacher_targets(ctypes.byref(shp or shape()), Q, FAKE, FAKE, cm, FAKE, FAKE, ydt,
                               ws, nb, None)
    assert tt(shp=shape(dt=vp.VP_F32)) == vp.VP_ERR_UNSUPPORTED
    assert tt(Q=None) == vp.VP_ERR_INVALID_ARG
    assert tt(cm=FAKE + 2) == vp.VP_ERR_INVALID_ARG
    assert tt(ydt=4) == vp.VP_ERR_INVALID_ARG
    assert tt(ws=None) == vp.VP_ERR_INVALID_ARG
    assert tt(nb=100) == vp.VP_ERR_WORKSPACE
    rl = lambda K=FAKE, st=None, scale=0.0, lam=1.0, nb=1 << 40: \
        lib.vp_router_loss(ctypes.byref(shape()), K, st if st is not None else ctypes.byref(rs()),
                           scale, FAKE, FAKE, lam, FAKE, FAKE, nb, None)
    assert rl(K=None) == vp.VP_ERR_INVALID_ARG
    assert rl(scale=-1.0) == vp.VP_ERR_INVALID_ARG
    assert rl(lam=float("inf")) == vp.VP_ERR_INVALID_ARG
    assert rl(nb=16) == vp.VP_ERR_WORKSPACE
    assert lib.vp_router_loss(ctypes.byref(shape()), FAKE, None, 0.0, FAKE, FAKE, 1.0, FAKE,
                              FAKE, 1 << 40, None) == vp.VP_ERR_INVALID_ARG
    ll = lambda A=FAKE, dt=vp.VP_BF16, lam=1.0, nb=1 << 40: \
        lib.vp_latent_loss(ctypes.byref(shape()), A, FAKE, dt, lam, FAKE, FAKE, nb, None)
    assert ll(A=None) == vp.VP_ERR_INVALID_ARG
    assert ll(A=FAKE_ODD) == vp.VP_ERR_INVALID_ARG
    assert ll(dt=3) == vp.VP_ERR_INVALID_ARG
    assert ll(lam=float("nan")) == vp.VP_ERR_INVALID_ARG
    assert ll(nb=16) == vp.VP_ERR_WORKSPACE


@pytest.mark.parametrize("S,P,M", [(3, 15, 12), (3, 15, 10), (2, 1374, 1000), (4, 9, 0),
                                   (100, 1374, 123660), (100, 1374, 103050), (500, 1374, 515250)])
def test_tome_split_matches_oracle(lib, S, P, M):
    import oracle
    is_dst, g = oracle.tome_split(S, P, M)
    gg, nrows = vp.tome_split(S, P, M)
    assert gg == g and nrows == S * P - M


def test_tome_validation(lib):
    g, nr = ctypes.c_int64(0), ctypes.c_int64(0)
    sp = lambda shp=None, M=12, ns=5: lib.vp_tome_split(ctypes.byref(shp or shape(S=3, P=15)), M,
                                                        ns, ctypes.byref(g), ctypes.byref(nr))
    assert sp() == vp.VP_OK and g.value == 3 and nr.value == 33
    # 10 patches per view: at most 2 x 9 sources (patch 0 of a view is always a destination)
    assert sp(M=18) == vp.VP_OK and g.value == 10 and sp(M=19) == vp.VP_ERR_INVALID_ARG
    assert sp(M=-1) == vp.VP_ERR_INVALID_ARG
    assert sp(ns=15) == vp.VP_ERR_INVALID_ARG and sp(ns=-1) == vp.VP_ERR_INVALID_ARG
    assert sp(shp=shape(S=1, P=15), M=1) == vp.VP_ERR_INVALID_ARG
    assert sp(shp=shape(S=1, P=15), M=0) == vp.VP_OK and nr.value == 15
    assert lib.vp_tome_workspace_bytes(ctypes.byref(shape(S=3, P=15))) > 0
    pl = lambda shp=None, K=FAKE, M=12, row=FAKE, rs_=FAKE, mem=FAKE, best=None, ws=FAKE, \
        nb=1 << 40: lib.vp_tome_plan(ctypes.byref(shp or shape(S=3, P=15)), K, M, 5, row, rs_,
                                     mem, best, None, ws, nb, None)
    assert pl(shp=shape(S=3, P=15, dt=vp.VP_F32)) == vp.VP_ERR_UNSUPPORTED
    assert pl(K=None) == vp.VP_ERR_INVALID_ARG and pl(K=FAKE_ODD) == vp.VP_ERR_INVALID_ARG
    assert pl(M=40) == vp.VP_ERR_INVALID_ARG
    assert pl(row=None) == vp.VP_ERR_INVALID_ARG and pl(mem=FAKE + 2) == vp.VP_ERR_INVALID_ARG
    assert pl(best=FAKE + 1) == vp.VP_ERR_INVALID_ARG
    assert pl(ws=None) == vp.VP_ERR_INVALID_ARG and pl(ws=FAKE + 64) == vp.VP_ERR_INVALID_ARG
    assert pl(nb=1024) == vp.VP_ERR_WORKSPACE
    mg = lambda X=FAKE, nrows=33, rs_=FAKE, out=FAKE: lib.vp_tome_merge(
        ctypes.byref(shape(S=3, P=15)), X, nrows, rs_, FAKE, out, None)
    assert mg(X=None) == vp.VP_ERR_INVALID_ARG and mg(out=FAKE_ODD) == vp.VP_ERR_INVALID_ARG
    assert mg(nrows=0) == vp.VP_ERR_INVALID_ARG and mg(nrows=46) == vp.VP_ERR_INVALID_ARG
    assert mg(rs_=None) == vp.VP_ERR_INVALID_ARG
    um = lambda Y=FAKE, nrows=33, row=FAKE: lib.vp_tome_unmerge(
        ctypes.byref(shape(S=3, P=15)), FAKE, nrows, row, Y, None)
    assert um(Y=None) == vp.VP_ERR_INVALID_ARG and um(row=FAKE + 2) == vp.VP_ERR_INVALID_ARG
    assert um(nrows=-1) == vp.VP_ERR_INVALID_ARG


def test_tome_merge_qkv_validation(lib):
    f = lambda shp=None, Q=FAKE, Km=FAKE, nrows=33: lib.vp_tome_merge_qkv(
        ctypes.byref(shp or shape(S=3, P=15)), Q, FAKE, FAKE, nrows, FAKE, FAKE, FAKE, Km, FAKE,
        None)
    assert f(shp=shape(S=3, P=15, dt=vp.VP_F32)) == vp.VP_ERR_UNSUPPORTED
    assert f(Q=None) == vp.VP_ERR_INVALID_ARG and f(Km=FAKE_ODD) == vp.VP_ERR_INVALID_ARG
    assert f(nrows=0) == vp.VP_ERR_INVALID_ARG and f(nrows=46) == vp.VP_ERR_INVALID_ARG
