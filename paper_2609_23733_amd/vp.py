"""Python binding of libvggtprime.so (include/vggt_prime.h).

Argument marshalling only: every step of the layer runs in the HIP kernels of
the library.  Tensors are torch CUDA (HIP) tensors; each call enqueues on the
current torch stream and returns without synchronising.  There is no CPU
fallback: if the library is not built, loading fails with an error.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Dict, Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libvggtprime.so")

VP_OK, VP_ERR_INVALID_ARG, VP_ERR_UNSUPPORTED, VP_ERR_WORKSPACE, VP_ERR_HIP = range(5)
VP_F32, VP_BF16 = 0, 1
MODE_MEAN, MODE_SURR, MODE_FULL = 0, 1, 2
RULE_THRESHOLD, RULE_ARGMAX, RULE_THRESHOLD_BINARY, RULE_ARGMAX_BINARY = 0, 1, 2, 3
POOL_GATED, POOL_MEAN = 0, 1
SURR_EQ7, SURR_MEAN_CONTEXT, SURR_NO_RESIDUAL, SURR_ADD_IDENTITY, SURR_LINEAR_ATTN = range(5)
ACT_GELU_ERF, ACT_RELU = 0, 1
MAX_HEADS, HEAD_DIM, HIDDEN = 16, 64, 64
BUCKETS_LEN = 3 + MAX_HEADS + 1
TAU_LOW, TAU_HIGH = 0.01, 0.20

EXPORTS = ("vp_workspace_bytes", "vp_router_score", "vp_router_score_noalloc",
           "vp_router_logits", "vp_assign_heads",
           "vp_routed_global_attention", "vp_gather_full_heads", "vp_full_head_attention",
           "vp_linear_heads", "vp_status_string", "vp_last_error", "vp_block_workspace_bytes",
           "vp_block_qkv", "vp_block_out", "vp_teacher_workspace_bytes", "vp_loss_workspace_bytes",
           "vp_teacher_targets", "vp_router_loss", "vp_latent_loss", "vp_tome_split",
           "vp_tome_workspace_bytes", "vp_tome_plan", "vp_tome_merge", "vp_tome_merge_qkv",
           "vp_tome_unmerge")
TOME_SPECIAL = 5   # special tokens per view (camera + registers), never merged
MODEL_DIM = MAX_HEADS * HEAD_DIM
BLOCK_VECS = ("ln1_w", "ln1_b", "b_qkv", "b_o", "ls1", "ln2_w", "ln2_b", "b_fc1", "b_fc2", "ls2")
BLOCK_MATS = ("w_qkv", "w_o", "w_fc1", "w_fc2")


class vp_shape(ctypes.Structure):
    _fields_ = [("S", ctypes.c_int64), ("P", ctypes.c_int64), ("H", ctypes.c_int32),
                ("d", ctypes.c_int32), ("dtype", ctypes.c_int)]


class vp_router_weights(ctypes.Structure):
    _fields_ = [("W", ctypes.c_void_p), ("U", ctypes.c_void_p), ("w", ctypes.c_void_p),
                ("L", ctypes.c_int32), ("scale", ctypes.c_float), ("pool", ctypes.c_int)]


class vp_router_state(ctypes.Structure):
    _fields_ = [("q_pool", ctypes.c_void_p), ("stats", ctypes.c_void_p),
                ("score", ctypes.c_void_p), ("ctx", ctypes.c_void_p), ("vmean", ctypes.c_void_p)]


class vp_surrogate_weights(ctypes.Structure):
    _fields_ = [("g_w1", ctypes.c_void_p), ("g_w2", ctypes.c_void_p), ("d_w1", ctypes.c_void_p),
                ("d_w2", ctypes.c_void_p), ("g_b1", ctypes.c_void_p), ("g_b2", ctypes.c_void_p),
                ("d_b1", ctypes.c_void_p), ("d_b2", ctypes.c_void_p), ("L", ctypes.c_int32),
                ("act", ctypes.c_int), ("variant", ctypes.c_int)]


class vp_block_weights(ctypes.Structure):
    _fields_ = [("ln1_w", ctypes.c_void_p), ("ln1_b", ctypes.c_void_p),
                ("w_qkv", ctypes.c_void_p), ("b_qkv", ctypes.c_void_p),
                ("w_o", ctypes.c_void_p), ("b_o", ctypes.c_void_p), ("ls1", ctypes.c_void_p),
                ("ln2_w", ctypes.c_void_p), ("ln2_b", ctypes.c_void_p),
                ("w_fc1", ctypes.c_void_p), ("b_fc1", ctypes.c_void_p),
                ("w_fc2", ctypes.c_void_p), ("b_fc2", ctypes.c_void_p), ("ls2", ctypes.c_void_p),
                ("ln_eps", ctypes.c_float), ("rope_base", ctypes.c_float)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libvggtprime.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("libvggtprime.so is not built (%s); run "
                           "`python -c 'import __graft_entry__ as g; g.build()'`" % path)
    lib = ctypes.CDLL(path)
    P, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    lib.vp_workspace_bytes.argtypes = [ctypes.POINTER(vp_shape)]
    lib.vp_workspace_bytes.restype = ctypes.c_size_t
    lib.vp_router_score.argtypes = [ctypes.POINTER(vp_shape), P, P, P,
                                    ctypes.POINTER(vp_router_weights),
                                    ctypes.POINTER(vp_router_state), P, ctypes.c_size_t, P]
    lib.vp_router_score_noalloc.argtypes = [ctypes.POINTER(vp_shape), P, P, P,
                                            ctypes.POINTER(vp_router_weights),
                                            ctypes.POINTER(vp_router_state), P]
    lib.vp_router_logits.argtypes = [P, P, P, i32, i32, i32, ctypes.c_int, P, P]
    lib.vp_assign_heads.argtypes = [P, i32, i32, ctypes.c_int, f32, f32, P, P, P]
    lib.vp_routed_global_attention.argtypes = [ctypes.POINTER(vp_shape), P, P, P, P, P,
                                               ctypes.POINTER(vp_router_state),
                                               ctypes.POINTER(vp_surrogate_weights), P,
                                               ctypes.c_int, P, ctypes.c_size_t, P]
    lib.vp_gather_full_heads.argtypes = [ctypes.POINTER(vp_shape), P, P, P, P, ctypes.c_size_t,
                                         P]
    lib.vp_full_head_attention.argtypes = [ctypes.POINTER(vp_shape), P, P, P, P, P, ctypes.c_int,
                                           P, ctypes.c_size_t, P]
    lib.vp_linear_heads.argtypes = [ctypes.POINTER(vp_shape), P, P, P, P,
                                    ctypes.POINTER(vp_router_state),
                                    ctypes.POINTER(vp_surrogate_weights), P, ctypes.c_int, P,
                                    ctypes.c_size_t, P]
    lib.vp_block_workspace_bytes.argtypes = [ctypes.POINTER(vp_shape)]
    lib.vp_block_workspace_bytes.restype = ctypes.c_size_t
    lib.vp_block_qkv.argtypes = [ctypes.POINTER(vp_shape), P, P, ctypes.POINTER(vp_block_weights),
                                 P, P, P, P, ctypes.c_size_t, P]
    lib.vp_block_out.argtypes = [ctypes.POINTER(vp_shape), P, P, ctypes.POINTER(vp_block_weights),
                                 P, P, ctypes.c_size_t, P]
    for f in ("vp_teacher_workspace_bytes", "vp_loss_workspace_bytes"):
        getattr(lib, f).argtypes = [ctypes.POINTER(vp_shape)]
        getattr(lib, f).restype = ctypes.c_size_t
    lib.vp_teacher_targets.argtypes = [ctypes.POINTER(vp_shape), P, P, P, P, P, P, ctypes.c_int,
                                       P, ctypes.c_size_t, P]
    lib.vp_router_loss.argtypes = [ctypes.POINTER(vp_shape), P, ctypes.POINTER(vp_router_state),
                                   f32, P, P, f32, P, P, ctypes.c_size_t, P]
    lib.vp_latent_loss.argtypes = [ctypes.POINTER(vp_shape), P, P, ctypes.c_int, f32, P, P,
                                   ctypes.c_size_t, P]
    lib.vp_tome_split.argtypes = [ctypes.POINTER(vp_shape), i64, i32, ctypes.POINTER(i64),
                                  ctypes.POINTER(i64)]
    lib.vp_tome_workspace_bytes.argtypes = [ctypes.POINTER(vp_shape)]
    lib.vp_tome_workspace_bytes.restype = ctypes.c_size_t
    lib.vp_tome_plan.argtypes = [ctypes.POINTER(vp_shape), P, i64, i32, P, P, P, P, P, P,
                                 ctypes.c_size_t, P]
    lib.vp_tome_merge.argtypes = [ctypes.POINTER(vp_shape), P, i64, P, P, P, P]
    lib.vp_tome_merge_qkv.argtypes = [ctypes.POINTER(vp_shape), P, P, P, i64, P, P, P, P, P, P]
    lib.vp_tome_unmerge.argtypes = [ctypes.POINTER(vp_shape), P, i64, P, P, P]
    for f in ("vp_tome_split", "vp_tome_plan", "vp_tome_merge", "vp_tome_merge_qkv",
              "vp_tome_unmerge"):
        getattr(lib, f).restype = ctypes.c_int
    for f in ("vp_router_score", "vp_router_score_noalloc", "vp_router_logits", "vp_assign_heads",
              "vp_routed_global_attention", "vp_gather_full_heads", "vp_full_head_attention",
              "vp_linear_heads", "vp_block_qkv", "vp_block_out", "vp_teacher_targets",
              "vp_router_loss", "vp_latent_loss"):
        getattr(lib, f).restype = ctypes.c_int
    lib.vp_status_string.argtypes = [ctypes.c_int]
    lib.vp_status_string.restype = ctypes.c_char_p
    lib.vp_last_error.argtypes = []
    lib.vp_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


class VPError(RuntimeError):
    def __init__(self, code: int, where: str):
        lib = load_library()
        msg = lib.vp_status_string(code).decode()
        if code == VP_ERR_HIP:
            msg += ": " + lib.vp_last_error().decode()
        super().__init__("%s failed: %s (status %d)" % (where, msg, code))
        self.code = code


def _check(code: int, where: str):
    if code != VP_OK:
        raise VPError(code, where)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return VP_BF16
    if t.dtype == torch.float32:
        return VP_F32
    raise TypeError("unsupported dtype %s" % t.dtype)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _need(t: torch.Tensor, name: str, shape=None, dtype=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a tensor" % name)
    if not t.is_cuda:
        raise ValueError("%s must be a GPU tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    if dtype is not None and t.dtype != dtype:
        raise ValueError("%s has dtype %s, expected %s" % (name, t.dtype, dtype))


def make_shape(S: int, P: int, H: int, dtype: torch.dtype) -> vp_shape:
    return vp_shape(S, P, H, HEAD_DIM, VP_BF16 if dtype == torch.bfloat16 else VP_F32)


def workspace_bytes(S: int, P: int, H: int = MAX_HEADS, dtype=torch.bfloat16) -> int:
    n = load_library().vp_workspace_bytes(ctypes.byref(make_shape(S, P, H, dtype)))
    if n == 0:
        raise ValueError("invalid shape")
    return int(n)


def alloc_workspace(S: int, P: int, H: int = MAX_HEADS, dtype=torch.bfloat16,
                    device="cuda") -> torch.Tensor:
    # torch's caching allocator returns 512-byte aligned blocks
    return torch.empty(workspace_bytes(S, P, H, dtype), dtype=torch.uint8, device=device)


@dataclass
class RouterState:
    q_pool: torch.Tensor   # [H, d]
    stats: torch.Tensor    # [H, 2]  (m, l)
    score: torch.Tensor    # [H]
    ctx: torch.Tensor      # [H, d]
    vmean: torch.Tensor    # [H, d]

    @staticmethod
    def empty(H: int, device="cuda") -> "RouterState":
        f = lambda *s: torch.empty(*s, dtype=torch.float32, device=device)
        return RouterState(f(H, HEAD_DIM), f(H, 2), f(H), f(H, HEAD_DIM), f(H, HEAD_DIM))

    def c(self) -> vp_router_state:
        return vp_router_state(self.q_pool.data_ptr(), self.stats.data_ptr(),
                               self.score.data_ptr(), self.ctx.data_ptr(), self.vmean.data_ptr())


def router_score(Q, K, V, W, U, w, S: int, P: int, ws: torch.Tensor, scale: float = 0.0,
                 out: Optional[RouterState] = None, pool: int = POOL_GATED) -> RouterState:
    """Router (Eq.1-3) plus context and value mean: see vp_router_score.
    ``pool=POOL_MEAN`` pools by the plain query mean (W, U, w may be None)."""
    N, H = S * P, Q.shape[1]
    for t, nm in ((Q, "Q"), (K, "K"), (V, "V")):
        _need(t, nm, (N, H, HEAD_DIM), Q.dtype)
    if pool == POOL_GATED:
        _need(W, "W", (H, HIDDEN, HEAD_DIM), Q.dtype)
        _need(U, "U", (H, HIDDEN, HEAD_DIM), Q.dtype)
        _need(w, "w", (H, HIDDEN), Q.dtype)
    _need(ws, "ws")
    if out is None:
        out = RouterState.empty(H, Q.device)
    ptr = lambda t: None if t is None else t.data_ptr()
    rw = vp_router_weights(ptr(W), ptr(U), ptr(w), HIDDEN, float(scale), int(pool))
    shp = make_shape(S, P, H, Q.dtype)
    st = out.c()
    _check(load_library().vp_router_score(ctypes.byref(shp), _ptr(Q), _ptr(K), _ptr(V),
                                          ctypes.byref(rw), ctypes.byref(st), _ptr(ws),
                                          ws.numel() * ws.element_size(), _stream()),
           "vp_router_score")
    return out


def router_score_noalloc(Q, K, V, W, U, w, S: int, P: int, scale: float = 0.0,
                         out: Optional[RouterState] = None,
                         pool: int = POOL_GATED) -> RouterState:
    """router_score without a workspace: the library keeps the partial sums in
    its own static device array (see vp_router_score_noalloc)."""
    N, H = S * P, Q.shape[1]
    for t, nm in ((Q, "Q"), (K, "K"), (V, "V")):
        _need(t, nm, (N, H, HEAD_DIM), Q.dtype)
    if pool == POOL_GATED:
        _need(W, "W", (H, HIDDEN, HEAD_DIM), Q.dtype)
        _need(U, "U", (H, HIDDEN, HEAD_DIM), Q.dtype)
        _need(w, "w", (H, HIDDEN), Q.dtype)
    if out is None:
        out = RouterState.empty(H, Q.device)
    ptr = lambda t: None if t is None else t.data_ptr()
    rw = vp_router_weights(ptr(W), ptr(U), ptr(w), HIDDEN, float(scale), int(pool))
    shp = make_shape(S, P, H, Q.dtype)
    st = out.c()
    _check(load_library().vp_router_score_noalloc(ctypes.byref(shp), _ptr(Q), _ptr(K), _ptr(V),
                                                  ctypes.byref(rw), ctypes.byref(st),
                                                  _stream()),
           "vp_router_score_noalloc")
    return out


def router_logits(u, Wr, br, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Linear-logit mode router of the synthetic workloads: [H, 3] fp32."""
    R, Din = Wr.shape
    H = R // 3
    _need(u, "u", (Din,), torch.float32)
    _need(Wr, "Wr")
    _need(br, "br", (R,), torch.float32)
    if out is None:
        out = torch.empty(H, 3, dtype=torch.float32, device=u.device)
    _need(out, "logits", (H, 3), torch.float32)
    _check(load_library().vp_router_logits(_ptr(u), _ptr(Wr), _ptr(br), H, Din, 3, _dt(Wr),
                                           _ptr(out), _stream()), "vp_router_logits")
    return out


def assign_heads(scores, rule: int, tau_low: float = TAU_LOW, tau_high: float = TAU_HIGH,
                 modes: Optional[torch.Tensor] = None, buckets: Optional[torch.Tensor] = None):
    """Mode assignment (Eq.4 / argmax).  Returns (modes uint8 [H], buckets int32 [20])."""
    H = scores.shape[0]
    _need(scores, "scores", None, torch.float32)
    if modes is None:
        modes = torch.empty(H, dtype=torch.uint8, device=scores.device)
    if buckets is None:
        buckets = torch.empty(BUCKETS_LEN, dtype=torch.int32, device=scores.device)
    _need(modes, "modes", (H,), torch.uint8)
    _need(buckets, "buckets", (BUCKETS_LEN,), torch.int32)
    M = 3 if rule in (RULE_ARGMAX, RULE_ARGMAX_BINARY) else 1
    _check(load_library().vp_assign_heads(_ptr(scores), H, M, int(rule), float(tau_low),
                                          float(tau_high), _ptr(modes), _ptr(buckets),
                                          _stream()), "vp_assign_heads")
    return modes, buckets


_SURR_KEYS = ("g_w1", "g_w2", "d_w1", "d_w2", "g_b1", "g_b2", "d_b1", "d_b2")


def _surr_struct(surr, H, dtype, act, variant=SURR_EQ7):
    if variant in (SURR_NO_RESIDUAL, SURR_LINEAR_ATTN):   # no MLP weight is read
        return vp_surrogate_weights(*([None] * 8), HIDDEN, int(act), int(variant))
    for k in ("g_w1", "d_w1"):
        _need(surr[k], k, (H, HIDDEN, 2 * HEAD_DIM), dtype)
    for k in ("g_w2", "d_w2"):
        _need(surr[k], k, (H, HEAD_DIM, HIDDEN), dtype)
    for k in ("g_b1", "d_b1"):
        _need(surr[k], k, (H, HIDDEN), torch.float32)
    for k in ("g_b2", "d_b2"):
        _need(surr[k], k, (H, HEAD_DIM), torch.float32)
    return vp_surrogate_weights(*(surr[k].data_ptr() for k in _SURR_KEYS), HIDDEN, int(act),
                                int(variant))


def _qkv(Q, K, V, S, P):
    N, H = S * P, Q.shape[1]
    for t, nm in ((Q, "Q"), (K, "K"), (V, "V")):
        _need(t, nm, (N, H, HEAD_DIM), Q.dtype)
    return N, H


def routed_global_attention(Q, K, V, modes, buckets, state: RouterState,
                            surr: Dict[str, torch.Tensor], S: int, P: int, ws: torch.Tensor,
                            y_dtype=None, act: int = ACT_GELU_ERF,
                            Y: Optional[torch.Tensor] = None,
                            surr_variant: int = SURR_EQ7) -> torch.Tensor:
    """Routed global attention (Algorithm 1 step 2): Y [N, H, d]."""
    N, H = _qkv(Q, K, V, S, P)
    _need(modes, "modes", (H,), torch.uint8)
    _need(buckets, "buckets", (BUCKETS_LEN,), torch.int32)
    if y_dtype is None:
        y_dtype = Q.dtype
    if Y is None:
        Y = torch.empty(N, H, HEAD_DIM, dtype=y_dtype, device=Q.device)
    _need(Y, "Y", (N, H, HEAD_DIM), y_dtype)
    sw = _surr_struct(surr, H, Q.dtype, act, surr_variant)
    shp = make_shape(S, P, H, Q.dtype)
    st = state.c()
    _check(load_library().vp_routed_global_attention(
        ctypes.byref(shp), _ptr(Q), _ptr(K), _ptr(V), _ptr(modes), _ptr(buckets),
        ctypes.byref(st), ctypes.byref(sw), _ptr(Y), _dt(Y), _ptr(ws),
        ws.numel() * ws.element_size(), _stream()), "vp_routed_global_attention")
    return Y


def gather_full_heads(K, V, buckets, S: int, P: int, ws: torch.Tensor):
    """Stage 1 of routed_global_attention: pack V of the FULL heads."""
    N, H = S * P, V.shape[1]
    _need(K, "K", (N, H, HEAD_DIM), V.dtype)
    _need(V, "V", (N, H, HEAD_DIM))
    _need(buckets, "buckets", (BUCKETS_LEN,), torch.int32)
    shp = make_shape(S, P, H, V.dtype)
    _check(load_library().vp_gather_full_heads(ctypes.byref(shp), _ptr(K), _ptr(V), _ptr(buckets),
                                               _ptr(ws), ws.numel() * ws.element_size(),
                                               _stream()), "vp_gather_full_heads")


def full_head_attention(Q, K, V, buckets, S: int, P: int, ws: torch.Tensor, Y: torch.Tensor):
    """Stage 2: exact softmax attention of every FULL head into Y."""
    N, H = _qkv(Q, K, V, S, P)
    _need(buckets, "buckets", (BUCKETS_LEN,), torch.int32)
    _need(Y, "Y", (N, H, HEAD_DIM))
    shp = make_shape(S, P, H, Q.dtype)
    _check(load_library().vp_full_head_attention(ctypes.byref(shp), _ptr(Q), _ptr(K), _ptr(V),
                                                 _ptr(buckets), _ptr(Y), _dt(Y), _ptr(ws),
                                                 ws.numel() * ws.element_size(), _stream()),
           "vp_full_head_attention")


def linear_heads(V, modes, state: RouterState, surr, S: int, P: int, Y: torch.Tensor,
                 act: int = ACT_GELU_ERF, surr_variant: int = SURR_EQ7, Q=None, K=None,
                 ws: Optional[torch.Tensor] = None):
    """Stage 3: SURR and MEAN heads into Y (Q, K and ws: linear attention only)."""
    N, H = S * P, V.shape[1]
    _need(V, "V", (N, H, HEAD_DIM))
    _need(modes, "modes", (H,), torch.uint8)
    _need(Y, "Y", (N, H, HEAD_DIM))
    if surr_variant == SURR_LINEAR_ATTN:
        _need(Q, "Q", (N, H, HEAD_DIM), V.dtype)
        _need(K, "K", (N, H, HEAD_DIM), V.dtype)
        _need(ws, "ws")
    sw = _surr_struct(surr, H, V.dtype, act, surr_variant)
    shp = make_shape(S, P, H, V.dtype)
    st = state.c()
    nws = 0 if ws is None else ws.numel() * ws.element_size()
    _check(load_library().vp_linear_heads(ctypes.byref(shp), _ptr(Q), _ptr(K), _ptr(V),
                                          _ptr(modes), ctypes.byref(st), ctypes.byref(sw),
                                          _ptr(Y), _dt(Y), _ptr(ws), nws, _stream()),
           "vp_linear_heads")


class RoutedLayer:
    """One routed global-attention layer on the GPU: holds the weights, the
    router state and the workspace, and runs the four library calls in order
    (router_score, [router_logits], assign_heads, routed_global_attention)."""

    def __init__(self, inp, rule: int = RULE_ARGMAX, y_dtype=None, act: int = ACT_GELU_ERF,
                 tau_low: float = TAU_LOW, tau_high: float = TAU_HIGH, device="cuda",
                 pool: int = POOL_GATED, surr_variant: int = SURR_EQ7,
                 ws: Optional[torch.Tensor] = None, Y: Optional[torch.Tensor] = None):
        """``ws`` and ``Y`` may be shared by layers that run one after another
        on one stream (a stack); they are allocated when not given."""
        x = inp.to(device)
        self.x = x
        self.S, self.P, self.H = x.S, x.P, x.H
        self.rule, self.act = rule, act
        self.pool, self.surr_variant = pool, surr_variant
        self.tau_low, self.tau_high = tau_low, tau_high
        self.y_dtype = y_dtype if y_dtype is not None else x.Q.dtype
        self.ws = ws if ws is not None else alloc_workspace(x.S, x.P, x.H, x.Q.dtype, device)
        self.state = RouterState.empty(x.H, device)
        self.logits = torch.empty(x.H, 3, dtype=torch.float32, device=device)
        self.modes = torch.empty(x.H, dtype=torch.uint8, device=device)
        self.buckets = torch.empty(BUCKETS_LEN, dtype=torch.int32, device=device)
        self.Y = Y if Y is not None else torch.empty(x.N, x.H, HEAD_DIM, dtype=self.y_dtype,
                                                     device=device)

    def step(self, Q=None, K=None, V=None, events=None, stages=None) -> torch.Tensor:
        """One pass of the layer.  ``events`` = (start, end) torch.cuda.Events
        recorded around the FULL-head attention stage on the current stream;
        ``stages`` = six events recorded before the router, after the router,
        after the mode assignment, after the bucket gather, after the FULL
        heads and after the SURR/MEAN heads."""
        x = self.x
        Q = x.Q if Q is None else Q
        K = x.K if K is None else K
        V = x.V if V is None else V
        rec = (lambda i: stages[i].record()) if stages is not None else (lambda i: None)
        rec(0)
        router_score(Q, K, V, x.W, x.U, x.w, self.S, self.P, self.ws, out=self.state,
                     pool=self.pool)
        rec(1)
        if self.rule in (RULE_ARGMAX, RULE_ARGMAX_BINARY):
            router_logits(x.u, x.Wr, x.br, out=self.logits)
            scores = self.logits
        else:
            scores = self.state.score
        assign_heads(scores, self.rule, self.tau_low, self.tau_high, self.modes, self.buckets)
        rec(2)
        if events is None and stages is None:
            routed_global_attention(Q, K, V, self.modes, self.buckets, self.state, x.surr,
                                    self.S, self.P, self.ws, self.y_dtype, self.act, self.Y,
                                    self.surr_variant)
        else:
            # the same three stages, with events between them
            gather_full_heads(K, V, self.buckets, self.S, self.P, self.ws)
            rec(3)
            if events is not None:
                events[0].record()
            full_head_attention(Q, K, V, self.buckets, self.S, self.P, self.ws, self.Y)
            if events is not None:
                events[1].record()
            rec(4)
            linear_heads(V, self.modes, self.state, x.surr, self.S, self.P, self.Y, self.act,
                         self.surr_variant, Q, K, self.ws)
            rec(5)
        return self.Y


class LayerGraph:
    """One pass of a RoutedLayer captured as a HIP graph (torch.cuda.CUDAGraph):
    the same library launches on the same buffers, replayed without per-call
    host work.  The layer's buffers (weights, workspace, router state, modes,
    Y) stay owned by the layer; replay() overwrites Y."""

    def __init__(self, layer: "RoutedLayer"):
        self.layer = layer
        side = torch.cuda.Stream()   # default priority
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            layer.step()             # one eager pass before capture
        torch.cuda.current_stream().wait_stream(side)
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            layer.step()

    def replay(self) -> torch.Tensor:
        self.graph.replay()
        return self.layer.Y


# ------------------------------------------- dense block around the layer

def block_workspace_bytes(S: int, P: int) -> int:
    n = load_library().vp_block_workspace_bytes(ctypes.byref(make_shape(S, P, MAX_HEADS,
                                                                        torch.bfloat16)))
    if n == 0:
        raise ValueError("invalid block shape")
    return int(n)


def _block_struct(w: Dict[str, torch.Tensor], eps: float = 0.0, rope_base: float = 0.0):
    D = MODEL_DIM
    shapes = {"w_qkv": (3 * D, D), "w_o": (D, D), "w_fc1": (4 * D, D), "w_fc2": (D, 4 * D),
              "b_qkv": (3 * D,), "b_fc1": (4 * D,)}
    for k in BLOCK_MATS:
        _need(w[k], k, shapes[k], torch.bfloat16)
    for k in BLOCK_VECS:
        _need(w[k], k, shapes.get(k, (D,)), torch.float32)
    names = [f[0] for f in vp_block_weights._fields_[:14]]
    return vp_block_weights(*[w[k].data_ptr() for k in names], float(eps), float(rope_base))


def block_qkv(X, pos, w, S: int, P: int, ws: torch.Tensor, Q=None, K=None, V=None):
    """LN_1, QKV projection and rotary encoding: Q, K, V [N, H, d] bf16."""
    N = S * P
    _need(X, "X", (N, MODEL_DIM), torch.bfloat16)
    _need(pos, "pos", (N, 2), torch.int32)
    _need(ws, "ws")
    out = []
    for t, nm in ((Q, "Q"), (K, "K"), (V, "V")):
        if t is None:
            t = torch.empty(N, MAX_HEADS, HEAD_DIM, dtype=torch.bfloat16, device=X.device)
        _need(t, nm, (N, MAX_HEADS, HEAD_DIM), torch.bfloat16)
        out.append(t)
    bw = _block_struct(w)
    shp = make_shape(S, P, MAX_HEADS, torch.bfloat16)
    _check(load_library().vp_block_qkv(ctypes.byref(shp), _ptr(X), _ptr(pos), ctypes.byref(bw),
                                       _ptr(out[0]), _ptr(out[1]), _ptr(out[2]), _ptr(ws),
                                       ws.numel() * ws.element_size(), _stream()),
           "vp_block_qkv")
    return tuple(out)


def block_out(X, Y, w, S: int, P: int, ws: torch.Tensor, X_out=None):
    """W_O, LayerScale, residual, LN_2, FFN, LayerScale, residual: [N, D] bf16."""
    N = S * P
    _need(X, "X", (N, MODEL_DIM), torch.bfloat16)
    _need(Y, "Y")
    if Y.numel() != N * MODEL_DIM or Y.dtype != torch.bfloat16:
        raise ValueError("Y must be [N, %d] bf16" % MODEL_DIM)
    _need(ws, "ws")
    if X_out is None:
        X_out = torch.empty_like(X)
    _need(X_out, "X_out", (N, MODEL_DIM), torch.bfloat16)
    bw = _block_struct(w)
    shp = make_shape(S, P, MAX_HEADS, torch.bfloat16)
    _check(load_library().vp_block_out(ctypes.byref(shp), _ptr(X), _ptr(Y), ctypes.byref(bw),
                                       _ptr(X_out), _ptr(ws), ws.numel() * ws.element_size(),
                                       _stream()), "vp_block_out")
    return X_out


class PrimeBlock:
    """One global-attention block of Algorithm 1 on the GPU: block_qkv, the
    routed layer on the block's own Q, K, V (router_score, [router_logits],
    assign_heads, routed_global_attention) and block_out; with ``tome_M``, the
    routed layer runs on the block's tokens merged down by tome_M (TomeLayer)
    and its output is unmerged before block_out."""

    def __init__(self, layer_inp, block_w: Dict[str, torch.Tensor], pos, device="cuda",
                 shared: Optional[Dict[str, torch.Tensor]] = None,
                 tome_M: Optional[int] = None, **layer_kw):
        """``shared``: buffers that blocks run one after another on one stream
        may share (make_shared()); allocated per block when not given."""
        self.S, self.P = layer_inp.S, layer_inp.P
        sh = shared if shared is not None else PrimeBlock.make_shared(self.S, self.P, device)
        self.w = {k: v.to(device) for k, v in block_w.items()}
        self.pos = pos if isinstance(pos, torch.Tensor) and pos.is_cuda else \
            torch.as_tensor(pos, dtype=torch.int32).to(device)
        if tome_M is None:
            self.tome = None
            self.layer = RoutedLayer(layer_inp, y_dtype=torch.bfloat16, device=device,
                                     ws=sh["layer_ws"], Y=sh["Y"], **layer_kw)
        else:
            self.tome = TomeLayer(layer_inp, tome_M, device=device, y_dtype=torch.bfloat16,
                                  Y=sh["Y"], **layer_kw)
            self.layer = self.tome.layer
        self.ws = sh["block_ws"]
        self.Q, self.K, self.V = sh["Q"], sh["K"], sh["V"]

    @staticmethod
    def make_shared(S: int, P: int, device="cuda") -> Dict[str, torch.Tensor]:
        N = S * P
        e = lambda: torch.empty(N, MAX_HEADS, HEAD_DIM, dtype=torch.bfloat16, device=device)
        return {"Q": e(), "K": e(), "V": e(), "Y": e(),
                "layer_ws": alloc_workspace(S, P, MAX_HEADS, torch.bfloat16, device),
                "block_ws": torch.empty(block_workspace_bytes(S, P), dtype=torch.uint8,
                                        device=device)}

    def step(self, X, X_out=None, events=None):
        """X [N, D] bf16 -> block output [N, D] bf16.  ``events``: optional
        list of torch.cuda.Event pairs (qkv, attention, out) to time stages."""
        ev = events or [None, None, None]
        def rec(i, j):
            if ev[i] is not None:
                ev[i][j].record()
        rec(0, 0)
        block_qkv(X, self.pos, self.w, self.S, self.P, self.ws, self.Q, self.K, self.V)
        rec(0, 1)
        rec(1, 0)
        if self.tome is None:
            Y = self.layer.step(self.Q, self.K, self.V)
        else:
            Y = self.tome.step(self.Q, self.K, self.V)
        rec(1, 1)
        rec(2, 0)
        out = block_out(X, Y, self.w, self.S, self.P, self.ws, X_out)
        rec(2, 1)
        return out


# ------------------------------------------- distillation targets and losses

def teacher_targets(Q, K, V, S: int, P: int, y_dtype=torch.bfloat16, ws=None):
    """Eq.8 and Eq.10 of the teacher (every head FULL): (colmax [H, N] fp32,
    smax [H] fp32, delta [N, H, d] y_dtype)."""
    N, H = _qkv(Q, K, V, S, P)
    shp = make_shape(S, P, H, Q.dtype)
    lib = load_library()
    if ws is None:
        n = lib.vp_teacher_workspace_bytes(ctypes.byref(shp))
        if n == 0:
            raise ValueError("teacher targets need a bf16 layer")
        ws = torch.empty(n, dtype=torch.uint8, device=Q.device)
    colmax = torch.empty(H, N, dtype=torch.float32, device=Q.device)
    smax = torch.empty(H, dtype=torch.float32, device=Q.device)
    delta = torch.empty(N, H, HEAD_DIM, dtype=y_dtype, device=Q.device)
    _check(lib.vp_teacher_targets(ctypes.byref(shp), _ptr(Q), _ptr(K), _ptr(V), _ptr(colmax),
                                  _ptr(smax), _ptr(delta), _dt(delta), _ptr(ws),
                                  ws.numel() * ws.element_size(), _stream()),
           "vp_teacher_targets")
    return colmax, smax, delta


def _loss_ws(shp, device):
    n = load_library().vp_loss_workspace_bytes(ctypes.byref(shp))
    return torch.empty(n, dtype=torch.uint8, device=device)


def router_loss(K, state: RouterState, colmax, smax, S: int, P: int, lam: float = 1.0,
                scale: float = 0.0):
    """Eq.9 per head: [H] fp32."""
    N, H = S * P, K.shape[1]
    _need(K, "K", (N, H, HEAD_DIM), torch.bfloat16)
    _need(colmax, "colmax", (H, N), torch.float32)
    _need(smax, "smax", (H,), torch.float32)
    shp = make_shape(S, P, H, K.dtype)
    ws = _loss_ws(shp, K.device)
    loss = torch.empty(H, dtype=torch.float32, device=K.device)
    st = state.c()
    _check(load_library().vp_router_loss(ctypes.byref(shp), _ptr(K), ctypes.byref(st),
                                         float(scale), _ptr(colmax), _ptr(smax), float(lam),
                                         _ptr(loss), _ptr(ws), ws.numel(), _stream()),
           "vp_router_loss")
    return loss


def latent_loss(D_hat, D_t, S: int, P: int, lam: float = 1.0):
    """Eq.11 per head: [H] fp32."""
    N, H = S * P, D_hat.shape[1]
    _need(D_hat, "D_hat", (N, H, HEAD_DIM))
    _need(D_t, "D_t", (N, H, HEAD_DIM), D_hat.dtype)
    shp = make_shape(S, P, H, D_hat.dtype)
    ws = _loss_ws(shp, D_hat.device)
    loss = torch.empty(H, dtype=torch.float32, device=D_hat.device)
    _check(load_library().vp_latent_loss(ctypes.byref(shp), _ptr(D_hat), _ptr(D_t), _dt(D_hat),
                                         float(lam), _ptr(loss), _ptr(ws), ws.numel(),
                                         _stream()), "vp_latent_loss")
    return loss


# ------------------------------------------------------------ token merging

def tome_split(S: int, P: int, M: int, nspecial: int = TOME_SPECIAL):
    """(g, nrows) for merging M of the S*P tokens (host only)."""
    shp = make_shape(S, P, MAX_HEADS, torch.bfloat16)
    g, nrows = ctypes.c_int64(0), ctypes.c_int64(0)
    _check(load_library().vp_tome_split(ctypes.byref(shp), int(M), int(nspecial),
                                        ctypes.byref(g), ctypes.byref(nrows)), "vp_tome_split")
    return g.value, nrows.value


def tome_workspace_bytes(S: int, P: int) -> int:
    return load_library().vp_tome_workspace_bytes(
        ctypes.byref(make_shape(S, P, MAX_HEADS, torch.bfloat16)))


class TomePlan:
    """Device arrays of a merge plan: row [N], row_start [nrows + 1], members
    [N] (int32), and optionally best [N] int32 / score [N] fp32."""

    def __init__(self, S, P, M, nspecial=TOME_SPECIAL, device="cuda", want_best=False):
        self.S, self.P, self.M, self.nspecial = S, P, M, nspecial
        self.g, self.nrows = tome_split(S, P, M, nspecial)
        N = S * P
        self.row = torch.empty(N, dtype=torch.int32, device=device)
        self.row_start = torch.empty(self.nrows + 1, dtype=torch.int32, device=device)
        self.members = torch.empty(N, dtype=torch.int32, device=device)
        self.best = torch.empty(N, dtype=torch.int32, device=device) if want_best else None
        self.score = torch.empty(N, dtype=torch.float32, device=device) if want_best else None
        self.ws = torch.empty(tome_workspace_bytes(S, P), dtype=torch.uint8, device=device)


def tome_plan(K, plan: TomePlan) -> TomePlan:
    """Fill `plan` from the keys K [N, H, 64] (bf16)."""
    S, P = plan.S, plan.P
    N, H = S * P, K.shape[1]
    _need(K, "K", (N, H, HEAD_DIM), torch.bfloat16)
    shp = make_shape(S, P, H, K.dtype)
    _check(load_library().vp_tome_plan(ctypes.byref(shp), _ptr(K), int(plan.M),
                                       int(plan.nspecial), _ptr(plan.row), _ptr(plan.row_start),
                                       _ptr(plan.members), _ptr(plan.best), _ptr(plan.score),
                                       _ptr(plan.ws), plan.ws.numel(), _stream()), "vp_tome_plan")
    return plan


def tome_merge(X, plan: TomePlan, out=None):
    """Rows of the merged sequence: X [N, H, 64] -> [nrows, H, 64] (means)."""
    N, H = plan.S * plan.P, X.shape[1]
    _need(X, "X", (N, H, HEAD_DIM))
    if out is None:
        out = torch.empty(plan.nrows, H, HEAD_DIM, dtype=X.dtype, device=X.device)
    _need(out, "out", (plan.nrows, H, HEAD_DIM), X.dtype)
    shp = make_shape(plan.S, plan.P, H, X.dtype)
    _check(load_library().vp_tome_merge(ctypes.byref(shp), _ptr(X), plan.nrows,
                                        _ptr(plan.row_start), _ptr(plan.members), _ptr(out),
                                        _stream()), "vp_tome_merge")
    return out


def tome_merge_qkv(Q, K, V, plan: TomePlan, Qm, Km, Vm):
    """Q, K, V (bf16) merged in one pass: the same rows as three tome_merge calls."""
    N, H = plan.S * plan.P, Q.shape[1]
    for nm, t in (("Q", Q), ("K", K), ("V", V)):
        _need(t, nm, (N, H, HEAD_DIM), torch.bfloat16)
    for nm, t in (("Qm", Qm), ("Km", Km), ("Vm", Vm)):
        _need(t, nm, (plan.nrows, H, HEAD_DIM), torch.bfloat16)
    shp = make_shape(plan.S, plan.P, H, Q.dtype)
    _check(load_library().vp_tome_merge_qkv(ctypes.byref(shp), _ptr(Q), _ptr(K), _ptr(V),
                                            plan.nrows, _ptr(plan.row_start),
                                            _ptr(plan.members), _ptr(Qm), _ptr(Km), _ptr(Vm),
                                            _stream()), "vp_tome_merge_qkv")
    return Qm, Km, Vm


def tome_unmerge(Ym, plan: TomePlan, out=None):
    """Every token takes its row's output: [nrows, H, 64] -> [N, H, 64]."""
    N, H = plan.S * plan.P, Ym.shape[1]
    _need(Ym, "Ym", (plan.nrows, H, HEAD_DIM))
    if out is None:
        out = torch.empty(N, H, HEAD_DIM, dtype=Ym.dtype, device=Ym.device)
    _need(out, "out", (N, H, HEAD_DIM), Ym.dtype)
    shp = make_shape(plan.S, plan.P, H, Ym.dtype)
    _check(load_library().vp_tome_unmerge(ctypes.byref(shp), _ptr(Ym), plan.nrows,
                                          _ptr(plan.row), _ptr(out), _stream()),
           "vp_tome_unmerge")
    return out


class TomeLayer:
    """Token merging around a routed layer: the plan from K, Q/K/V merged, the
    routed layer on the nrows merged rows (one sequence), its output unmerged
    to all S*P tokens."""

    def __init__(self, inp, M: int, nspecial: int = TOME_SPECIAL, device="cuda",
                 want_best=False, Y: Optional[torch.Tensor] = None, **layer_kw):
        """``Y``: the unmerged output [N, H, 64] (allocated when not given)."""
        import dataclasses
        x = inp.to(device)
        self.x = x
        self.plan = TomePlan(x.S, x.P, M, nspecial, device, want_best)
        nr = self.plan.nrows
        dt = x.Q.dtype if x.Q is not None else torch.bfloat16
        mk = lambda: torch.empty(nr, x.H, HEAD_DIM, dtype=dt, device=device)
        self.Qm, self.Km, self.Vm = mk(), mk(), mk()
        merged = dataclasses.replace(x, S=1, P=nr, Q=self.Qm, K=self.Km, V=self.Vm)
        self.layer = RoutedLayer(merged, device=device, **layer_kw)
        self.Y = Y if Y is not None else torch.empty(x.N, x.H, HEAD_DIM,
                                                     dtype=self.layer.y_dtype, device=device)

    def step(self, Q=None, K=None, V=None, events=None) -> torch.Tensor:
        x = self.x
        Q = x.Q if Q is None else Q
        K = x.K if K is None else K
        V = x.V if V is None else V
        tome_plan(K, self.plan)
        if Q.dtype == torch.bfloat16:
            tome_merge_qkv(Q, K, V, self.plan, self.Qm, self.Km, self.Vm)
        else:
            tome_merge(Q, self.plan, self.Qm)
            tome_merge(K, self.plan, self.Km)
            tome_merge(V, self.plan, self.Vm)
        Ym = self.layer.step(events=events)
        return tome_unmerge(Ym, self.plan, self.Y)

