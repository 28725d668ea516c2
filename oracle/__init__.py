"""fp64 CPU oracle of the VGGT-Prime routed global-attention layer.

TEST INFRASTRUCTURE ONLY.  Imported by the tests, by the smoke check and by
the benchmark's CPU-baseline leg; never by the GPU library or its binding.
It shares no code with the GPU path (only the seeded input generators are
common).  The arithmetic lives in ``vp_oracle.c`` (plain C, double precision,
written from the paper's equations); this module loads it, composes the
layer in the paper's order and adds the trivial MEAN broadcast.

Pins (tests/test_oracle_pins.py) tie every function here to something other
than itself: library routines (scaled-dot-product attention, softmax, erf),
closed forms (planted key, zero queries, one-hot router rows), invariants
(rows summing to one, token-permutation equivariance, S identical views) and
a numpy brute force on tiny shapes.  The surrogate MLP's exact architecture is
a reading of the paper (it gives only "a lightweight MLP" of hidden size 64):
its structure is pinned by closed-form special cases, but no paper number
fixes it -- parity unpinned as to the architecture itself.  Likewise the
feature map of the linear-attention ablation (phi = elu + 1, the map of the
kernelised attention the paper cites) is a reading: the computation given phi
is pinned against its explicit-matrix form, the choice of phi is unpinned.
The paper gives no steps for its token-merging combination either: the merging
rule here (ToMe's bipartite soft matching on the head-summed keys) is a
reading, its computation pinned by a brute force and planted decisions, the
choice of rule parity unpinned.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "vp_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

MODE_MEAN, MODE_SURR, MODE_FULL = 0, 1, 2
RULE_THRESHOLD, RULE_ARGMAX, RULE_THRESHOLD_BINARY, RULE_ARGMAX_BINARY = 0, 1, 2, 3
POOL_GATED, POOL_MEAN = 0, 1
SURR_EQ7, SURR_MEAN_CONTEXT, SURR_NO_RESIDUAL, SURR_ADD_IDENTITY, SURR_LINEAR_ATTN = 0, 1, 2, 3, 4
ACT_GELU, ACT_RELU = 0, 1
TAU_LOW, TAU_HIGH = 0.01, 0.20   # Section 4.2 and implementation details
TOME_SPECIAL = 5                 # special tokens per view (camera + registers), never merged
LN_EPS, ROPE_BASE = 1e-6, 100.0  # readings for the block around the layer


def build(force: bool = False) -> str:
    """Compile vp_oracle.c with gcc (strict IEEE double; no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-o", tmp, _SRC,
                               "-lm", "-lpthread"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            # VP_ORACLE_LIB names a prebuilt variant (the mutation tests plant
            # mistakes in a copy of vp_oracle.c and check that the pins fail).
            path = os.environ.get("VP_ORACLE_LIB")
            if not path:
                path = build()
            lib = ctypes.CDLL(path)
            P = ctypes.c_void_p
            i64, i32, dbl, flt = ctypes.c_int64, ctypes.c_int, ctypes.c_double, ctypes.c_float
            lib.or_router_pool.argtypes = [P, i64, i32, i32, i32, P, P, P, P, P, P, i32]
            lib.or_router_route.argtypes = [P, P, i64, i32, i32, P, dbl, P, P, P, P, i32]
            lib.or_router_logits.argtypes = [P, P, P, i32, i32, P]
            lib.or_assign.argtypes = [P, i32, i32, flt, flt, P]
            lib.or_full_rows.argtypes = [P, P, P, i64, i32, i32, i32, P, i64, dbl, P, i32]
            lib.or_surr_rows.argtypes = [P, i64, i32, i32, i32, i32, i32, i32, P, P, P, P, P, P,
                                         P, P, P, P, i64, P, i32]
            lib.or_linattn_rows.argtypes = [P, P, P, i64, i32, i32, i32, P, i64, P, i32]
            lib.or_layernorm.argtypes = [P, i64, i32, P, P, dbl, P, i32]
            lib.or_rope2d.argtypes = [P, i64, i32, i32, P, dbl, i32]
            lib.or_gelu.argtypes = [P, i64]
            lib.or_attention_colmax.argtypes = [P, P, i64, i32, i32, i32, dbl, P, i64, P, i32]
            lib.or_tome_metric.argtypes = [P, i64, i32, i32, P]
            lib.or_tome_split.argtypes = [i64, i64, i64, i64, P]
            lib.or_tome_split.restype = i64
            lib.or_tome_match.argtypes = [P, i64, i32, P, P, i64, P, P, i32]
            lib.or_tome_select.argtypes = [P, P, i64, i64, P]
            lib.or_tome_rows.argtypes = [i64, P, P, P, i64, P]
            lib.or_tome_rows.restype = i64
            lib.or_tome_merge.argtypes = [P, i64, i64, P, i64, P]
            lib.or_threads_used.argtypes = [i32]
            lib.or_threads_used.restype = i32
            _lib = lib
    return _lib


def as_f32(x) -> np.ndarray:
    """Stored values as a C-contiguous float32 array (exact for bf16 and fp32)."""
    if hasattr(x, "detach"):
        x = x.detach().float().cpu().numpy()
    return np.ascontiguousarray(x, dtype=np.float32)


def default_threads() -> int:
    """Oracle worker threads: VP_ORACLE_THREADS, else min(16, CPU count)."""
    env = os.environ.get("VP_ORACLE_THREADS")
    if env:
        return max(1, int(env))
    return max(1, min(16, os.cpu_count() or 1))


def _nt(n):
    return default_threads() if not n else int(n)


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def threads_used(nthreads: int = 0) -> int:
    return _load().or_threads_used(_nt(nthreads))


# ------------------------------------------------------------------ steps

def router_pool(Q, W, U, w, nthreads=0, want_weights=False):
    """Eq.1-2: gated attention pooling.  Returns q_pool [H, d] (and a, alpha [H, N])."""
    Q, W, U, w = as_f32(Q), as_f32(W), as_f32(U), as_f32(w)
    N, H, d = Q.shape
    L = W.shape[1]
    qp = np.zeros((H, d), np.float64)
    a = np.zeros((H, N), np.float64) if want_weights else None
    al = np.zeros((H, N), np.float64) if want_weights else None
    _load().or_router_pool(_p(Q), N, H, d, L, _p(W), _p(U), _p(w), _p(qp), _p(a), _p(al),
                           _nt(nthreads))
    return (qp, a, al) if want_weights else qp


def router_pool_mean(Q):
    """Mean-query ablation (component study): q_pool = (1/N) sum_i q_i."""
    return as_f32(Q).astype(np.float64).mean(axis=0)


def router_route(K, V, q_pool, scale=None, nthreads=0, want_r=False):
    """Eq.3 and Eq.5: single-query attention r_h, saliency s_h = max r_h,
    context C_h = r_h V_h and value mean.  Returns (s [H], C [H,d], mean [H,d] [, r])."""
    K, V = as_f32(K), as_f32(V)
    N, H, d = K.shape
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    qp = np.ascontiguousarray(q_pool, dtype=np.float64)
    s = np.zeros(H, np.float64)
    C = np.zeros((H, d), np.float64)
    mean = np.zeros((H, d), np.float64)
    r = np.zeros((H, N), np.float64) if want_r else None
    _load().or_router_route(_p(K), _p(V), N, H, d, _p(qp), float(scale), _p(r), _p(s), _p(C),
                            _p(mean), _nt(nthreads))
    return (s, C, mean, r) if want_r else (s, C, mean)


def router_logits(u, Wr, br):
    """Linear-logit mode router of the synthetic workloads: [H, 3] logits."""
    u, Wr, br = as_f32(u), as_f32(Wr), as_f32(br)
    R, Din = Wr.shape
    out = np.zeros(R, np.float64)
    _load().or_router_logits(_p(u), _p(Wr), _p(br), R, Din, _p(out))
    return out.reshape(R // 3, 3)


def assign(scores, rule, tau_low=TAU_LOW, tau_high=TAU_HIGH):
    """Eq.4 (threshold on s_h), first-argmax of per-head logits, or their
    two-branch (MEAN / FULL only) forms of the compute-mode ablation."""
    sc = np.ascontiguousarray(scores, dtype=np.float64)
    H = sc.shape[0]
    modes = np.zeros(H, np.uint8)
    _load().or_assign(_p(sc), H, int(rule), float(tau_low), float(tau_high), _p(modes))
    return modes


def buckets(modes):
    """Counts per mode and head ids grouped by mode (MEAN, SURR, FULL), each
    group in ascending head order."""
    modes = np.asarray(modes)
    counts = np.array([(modes == m).sum() for m in range(3)], np.int32)
    lst = np.concatenate([np.nonzero(modes == m)[0] for m in range(3)]).astype(np.int32)
    return counts, lst


def full_rows(Q, K, V, h, rows=None, scale=None, nthreads=0):
    """Algorithm 1 FULL branch for head h on the given query rows: [R, d]."""
    Q, K, V = as_f32(Q), as_f32(K), as_f32(V)
    N, H, d = Q.shape
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    if rows is None:
        nr, rp = N, None
    else:
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        nr, rp = rows.shape[0], rows
    Y = np.zeros((nr, d), np.float64)
    _load().or_full_rows(_p(Q), _p(K), _p(V), N, H, d, int(h), _p(rp), nr, float(scale), _p(Y),
                         _nt(nthreads))
    return Y


def surr_rows(V, C_h, surr, h, rows=None, act=ACT_GELU, nthreads=0, variant=SURR_EQ7):
    """Eq.5-7 SURR branch for head h: [R, d].  ``surr`` holds the per-head
    stacked weights g_w1 [H,L,2d], g_b1 [H,L], g_w2 [H,d,L], g_b2 [H,d], d_*.
    ``variant``: SURR_EQ7, SURR_NO_RESIDUAL (y = C_h) or SURR_ADD_IDENTITY
    (y = v + Eq.7); the mean-context ablation is SURR_EQ7 with C_h = mean."""
    V = as_f32(V)
    N, H, d = V.shape
    wt = {k: np.ascontiguousarray(as_f32(v)[h]) for k, v in surr.items()}
    L = wt["g_w1"].shape[0]
    C_h = np.ascontiguousarray(C_h, dtype=np.float64)
    if rows is None:
        nr, rp = N, None
    else:
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        nr, rp = rows.shape[0], rows
    Y = np.zeros((nr, d), np.float64)
    _load().or_surr_rows(_p(V), N, H, d, int(h), L, int(act), int(variant), _p(C_h),
                         _p(wt["g_w1"]),
                         _p(wt["g_b1"]), _p(wt["g_w2"]), _p(wt["g_b2"]), _p(wt["d_w1"]),
                         _p(wt["d_b1"]), _p(wt["d_w2"]), _p(wt["d_b2"]), _p(rp), nr, _p(Y),
                         _nt(nthreads))
    return Y


def linattn_rows(Q, K, V, h, rows=None, nthreads=0):
    """Linear attention of head h (the compute-mode ablation's alternative to
    the surrogate; phi = elu + 1) on the given query rows: [R, d]."""
    Q, K, V = as_f32(Q), as_f32(K), as_f32(V)
    N, H, d = Q.shape
    if rows is None:
        nr, rp = N, None
    else:
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        nr, rp = rows.shape[0], rows
    Y = np.zeros((nr, d), np.float64)
    _load().or_linattn_rows(_p(Q), _p(K), _p(V), N, H, d, int(h), _p(rp), nr, _p(Y),
                            _nt(nthreads))
    return Y


def routed_layer(Q, K, V, W, U, w, surr, u=None, Wr=None, br=None, rule=RULE_ARGMAX,
                 tau_low=TAU_LOW, tau_high=TAU_HIGH, modes=None, rows=None, full_rows_sel=None,
                 act=ACT_GELU, scale_router=None, scale_attn=None, nthreads=0,
                 pool=POOL_GATED, surr_variant=SURR_EQ7):
    """The routed global-attention layer (Algorithm 1 step 2, Eq.1-7), in order:
    router pooling, single-query routing, mode assignment, per-head outputs,
    concatenation over heads.

    ``rows``: query rows at which Y is evaluated (all if None).
    ``full_rows_sel``: for FULL heads only, evaluate these rows instead (the
    row sample used at sizes where exact attention over every row is too slow);
    the returned ``Y_full_rows`` then holds them.
    ``modes``: explicit modes (bypasses the rule, e.g. to force every head FULL).
    ``pool``: POOL_GATED (Eq.1-2) or POOL_MEAN (mean-query ablation).
    ``surr_variant``: how SURR heads are computed (Eq.5-7 or an ablation).
    """
    Q32 = as_f32(Q)
    N, H, d = Q32.shape
    q_pool = router_pool(Q32, W, U, w, nthreads) if pool == POOL_GATED else router_pool_mean(Q32)
    s, C, mean = router_route(K, V, q_pool, scale_router, nthreads)
    logits = None
    if modes is None:
        if rule in (RULE_THRESHOLD, RULE_THRESHOLD_BINARY):
            modes = assign(s, rule, tau_low, tau_high)
        else:
            if u is None:   # default router input: the pooled queries of all heads
                u = q_pool.reshape(-1).astype(np.float32)
            logits = router_logits(u, Wr, br)
            modes = assign(logits, rule)
    modes = np.asarray(modes, np.uint8)
    nrow = N if rows is None else len(rows)
    Y = np.zeros((nrow, H, d), np.float64)
    Yf = {}
    for h in range(H):
        m = int(modes[h])
        if m == MODE_FULL:
            if full_rows_sel is not None:
                Yf[h] = full_rows(Q32, K, V, h, full_rows_sel, scale_attn, nthreads)
                Y[:, h, :] = np.nan
            else:
                Y[:, h, :] = full_rows(Q32, K, V, h, rows, scale_attn, nthreads)
        elif m == MODE_SURR:
            if surr_variant == SURR_LINEAR_ATTN:
                Y[:, h, :] = linattn_rows(Q32, K, V, h, rows, nthreads)
            elif surr_variant == SURR_MEAN_CONTEXT:
                Y[:, h, :] = surr_rows(V, mean[h], surr, h, rows, act, nthreads, SURR_EQ7)
            else:
                Y[:, h, :] = surr_rows(V, C[h], surr, h, rows, act, nthreads, surr_variant)
        else:
            Y[:, h, :] = mean[h][None, :]     # Algorithm 1: broadcast of the value mean
    return dict(q_pool=q_pool, s=s, C=C, mean=mean, logits=logits, modes=modes, Y=Y,
                Y_full_rows=Yf)


# ------------------------------------------- dense block around the layer

def layernorm(X, g, b, eps=LN_EPS, nthreads=0):
    """Algorithm 1, LN: per row, (x - mean) / sqrt(var + eps) * g + b.  X: stored
    values or float64 rows."""
    if hasattr(X, "detach"):
        X = as_f32(X)
    X = np.ascontiguousarray(X, dtype=np.float64)
    N, D = X.shape
    g, b = as_f32(g), as_f32(b)
    Y = np.zeros((N, D), np.float64)
    _load().or_layernorm(_p(X), N, D, _p(g), _p(b), float(eps), _p(Y), _nt(nthreads))
    return Y


def rope2d(T, pos, base=ROPE_BASE, nthreads=0):
    """The positional information of QKV_h(., P): 2D rotary encoding of each
    head's features by the token's (row, column) coordinates.  T: [N, H, d]
    float64 (rotated copy returned); pos: [N, 2] int."""
    T = np.array(T, dtype=np.float64, order="C", copy=True)
    N, H, d = T.shape
    pos = np.ascontiguousarray(pos, dtype=np.int32)
    _load().or_rope2d(_p(T), N, H, d, _p(pos), float(base), _nt(nthreads))
    return T


def gelu(X):
    """GELU with the exact normal CDF (erf form)."""
    X = np.array(X, dtype=np.float64, order="C", copy=True)
    _load().or_gelu(_p(X), X.size)
    return X


def linear(X, W, b):
    """y = x W^T + b in float64 (W [out, in] as stored; a library matmul)."""
    X = np.asarray(X, dtype=np.float64)
    return X @ as_f32(W).astype(np.float64).T + as_f32(b).astype(np.float64)


def block_qkv(X, pos, wt, H=16, eps=LN_EPS, base=ROPE_BASE, nthreads=0):
    """Algorithm 1 steps (1)-(2a): X~ = LN_1(X); (Q_h, K_h, V_h) = QKV_h(X~, P),
    the projection followed by the rotary encoding of Q and K.
    X [N, D] -> Q, K, V [N, H, D/H] float64."""
    Xn = layernorm(X, wt["ln1_w"], wt["ln1_b"], eps, nthreads)
    N, D = Xn.shape
    qkv = linear(Xn, wt["w_qkv"], wt["b_qkv"])
    d = D // H
    Q = rope2d(qkv[:, :D].reshape(N, H, d), pos, base, nthreads)
    K = rope2d(qkv[:, D:2 * D].reshape(N, H, d), pos, base, nthreads)
    V = qkv[:, 2 * D:].reshape(N, H, d).copy()
    return Q, K, V


def block_out(X, Y, wt, eps=LN_EPS, nthreads=0):
    """Algorithm 1 steps (3)-(4): X_attn = X + LS_1(Y W_O); the block output
    X_attn + LS_2(FFN(LN_2(X_attn))), FFN = Linear -> GELU -> Linear.
    X, Y [N, D] stored values (Y = Concat of the head outputs; [N, H, d] is
    accepted) -> (block output, X_attn), float64."""
    X64 = as_f32(X).astype(np.float64)
    N = X64.shape[0]
    Y64 = (as_f32(Y) if hasattr(Y, "detach") else np.asarray(Y)).astype(np.float64)
    A = linear(Y64.reshape(N, -1), wt["w_o"], wt["b_o"])
    Xa = X64 + as_f32(wt["ls1"]).astype(np.float64) * A
    Z = layernorm(Xa, wt["ln2_w"], wt["ln2_b"], eps, nthreads)
    F = linear(gelu(linear(Z, wt["w_fc1"], wt["b_fc1"])), wt["w_fc2"], wt["b_fc2"])
    return Xa + as_f32(wt["ls2"]).astype(np.float64) * F, Xa


# ------------------------------------------ distillation targets and losses

def attention_colmax(Q, K, h, keys=None, scale=None, nthreads=0):
    """Eq.8: p^T_{h,k} = max over queries q of the teacher's post-softmax
    attention A_{h,k,q} (every query attends all N keys).  Returns [N] (or the
    listed keys) float64."""
    Q, K = as_f32(Q), as_f32(K)
    N, H, d = Q.shape
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    if keys is None:
        nk, kp = N, None
    else:
        kp = np.ascontiguousarray(keys, dtype=np.int64)
        nk = kp.shape[0]
    p = np.zeros(nk, np.float64)
    _load().or_attention_colmax(_p(Q), _p(K), N, H, d, int(h), float(scale), _p(kp), nk, _p(p),
                                _nt(nthreads))
    return p


def teacher_delta_rows(Q, K, V, h, rows=None, nthreads=0):
    """Eq.10: Delta^T_h = (A_h - I) V_h on the given rows: softmax attention of
    the rows minus their own values.  [R, d] float64."""
    Y = full_rows(Q, K, V, h, rows, None, nthreads)
    Vh = as_f32(V)[:, h, :].astype(np.float64)
    return Y - (Vh if rows is None else Vh[np.asarray(rows)])


def router_loss(p, r, lam=1.0):
    """Eq.9 for one head: KL(p_bar || r_bar) + lam |max p - max r|, with p_bar
    and r_bar the key distributions p / sum p and r / sum r (0 log 0 = 0)."""
    p = np.asarray(p, np.float64)
    r = np.asarray(r, np.float64)
    pb, rb = p / p.sum(), r / r.sum()
    nz = pb > 0
    kl = float(np.sum(pb[nz] * (np.log(pb[nz]) - np.log(rb[nz]))))
    return kl + lam * abs(float(p.max()) - float(r.max()))


def latent_loss(dhat, dT, lam=1.0):
    """Eq.11 for one head: ||dhat - dT||_2 + lam (1 - cos(dhat, dT)), the norm and
    the cosine taken over all N x d entries."""
    a = np.asarray(dhat, np.float64).ravel()
    b = np.asarray(dT, np.float64).ravel()
    cos = float(a @ b) / (np.sqrt(float(a @ a)) * np.sqrt(float(b @ b)))
    return float(np.sqrt(float((a - b) @ (a - b)))) + lam * (1.0 - cos)


# ----------------------------------------------------------- token merging
# ToMe's bipartite soft matching (Bolya et al., ICLR 2023) before the routed
# attention, in the reading stated in vp_oracle.c: head-sum key metric rounded
# to bf16, destinations = view 0 + special tokens + a stride-g patch lattice,
# cosine matching, the M most similar sources merged by mean, unmerge by copy.

def tome_metric(K):
    """m_i = bf16(sum over heads of K_{i,h}) (fp32 head-order sum): [N, d] float64."""
    K = as_f32(K)
    N, H, d = K.shape
    m = np.empty((N, d), np.float64)
    _load().or_tome_metric(_p(K), N, H, d, _p(m))
    return m


def tome_split(S, P, M, nspecial=TOME_SPECIAL):
    """(is_dst [S*P] bool, g): the destination set for merging M tokens."""
    is_dst = np.zeros(S * P, np.uint8)
    g = _load().or_tome_split(int(S), int(P), int(nspecial), int(M), _p(is_dst))
    if g < 0:
        raise ValueError("cannot merge %d of %d tokens" % (M, S * P))
    return is_dst.astype(bool), int(g)


def tome_match(K, S, P, M, srcs=None, nspecial=TOME_SPECIAL, nthreads=0):
    """Most similar destination token and its cosine similarity for the listed
    source tokens (all sources when srcs is None): (srcs, best, score)."""
    is_dst, _ = tome_split(S, P, M, nspecial)
    m = tome_metric(K)
    if srcs is None:
        srcs = np.nonzero(~is_dst)[0]
    srcs = np.ascontiguousarray(srcs, dtype=np.int64)
    best = np.empty(srcs.shape[0], np.int64)
    score = np.empty(srcs.shape[0], np.float64)
    _load().or_tome_match(_p(m), m.shape[0], m.shape[1], _p(is_dst.astype(np.uint8)), _p(srcs),
                          srcs.shape[0], _p(best), _p(score), _nt(nthreads))
    return srcs, best, score


def tome_select(srcs, score, M):
    """merged [nsrc] bool: the M sources ranked first by (similarity desc, token asc)."""
    srcs = np.ascontiguousarray(srcs, dtype=np.int64)
    score = np.ascontiguousarray(score, dtype=np.float64)
    merged = np.zeros(srcs.shape[0], np.uint8)
    _load().or_tome_select(_p(srcs), _p(score), srcs.shape[0], int(M), _p(merged))
    return merged.astype(bool)


def tome_rows(N, srcs, best, merged):
    """(row [N] int64, nrows): merged-sequence row of every token."""
    srcs = np.ascontiguousarray(srcs, dtype=np.int64)
    best = np.ascontiguousarray(best, dtype=np.int64)
    row = np.empty(int(N), np.int64)
    n = _load().or_tome_rows(int(N), _p(srcs), _p(best),
                             _p(np.ascontiguousarray(merged, dtype=np.uint8)), srcs.shape[0],
                             _p(row))
    return row, int(n)


def tome_plan(K, S, P, M, nspecial=TOME_SPECIAL, nthreads=0):
    """The whole merge plan for merging M of the S*P tokens."""
    is_dst, g = tome_split(S, P, M, nspecial)
    srcs, best, score = tome_match(K, S, P, M, None, nspecial, nthreads)
    merged = tome_select(srcs, score, M)
    row, nrows = tome_rows(S * P, srcs, best, merged)
    return dict(is_dst=is_dst, g=g, srcs=srcs, best=best, score=score, merged=merged, row=row,
                nrows=nrows)


def tome_merge(X, row, nrows):
    """Rows of the merged sequence: the mean of each row's tokens.  X [N, ...]
    -> [nrows, ...] float64."""
    X = as_f32(X)
    N = X.shape[0]
    F = int(np.prod(X.shape[1:])) if X.ndim > 1 else 1
    out = np.empty((int(nrows), F), np.float64)
    _load().or_tome_merge(_p(np.ascontiguousarray(X.reshape(N, F))), N, F,
                          _p(np.ascontiguousarray(row, dtype=np.int64)), int(nrows), _p(out))
    return out.reshape((int(nrows),) + X.shape[1:])


def tome_unmerge(Y, row):
    """Every token takes its row's output: Y [nrows, ...] -> [N, ...]."""
    return np.asarray(Y)[np.asarray(row)]
