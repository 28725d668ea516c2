"""Seeded synthetic inputs for the routed global-attention layer.

This module is the only code shared by the fp64 oracle tests and the GPU path.
It draws random tensors and arranges them; it computes none of the layer's
arithmetic (no pooling, no routing scores, no attention, no surrogate MLP).
The single piece of arithmetic it does hold is input construction for the
linear-logit mode router used by the synthetic workloads: a float64 dot
product of the stored router weight rows with the stored router input, used
only to place the bias so that a chosen mode wins by a chosen margin. Tests
re-derive the logits independently with the oracle and check the margin.

Shapes follow the VGGT aggregator as the paper describes it (Section 3: 24
global-attention layers of 16 heads; implementation details: hidden size 64
for router and surrogate, seed 67). Tokens per view P = 1374
(1 camera + 4 register + 37 x 37 patch tokens), head dimension d = 64, and
Q/K/V are laid out [S*P, H, d] row-major.

Value recipe (iid, synthetic, standing in for the paper's benchmark scenes,
which are not available here):
  Q, K, V               ~ N(0, 1) / sqrt(d)         (``sharp=True``: N(0, 1))
  router W_h, U_h, w_h  ~ U(-1/sqrt(64), 1/sqrt(64))
  surrogate layer 1     ~ U(-1/sqrt(2d), 1/sqrt(2d)), layer 2 ~ U(-1/sqrt(L), 1/sqrt(L))
  surrogate biases      ~ U(-1/sqrt(fan_in), 1/sqrt(fan_in)), kept fp32
  mode-router input u   ~ N(0, 1) / sqrt(d), 1024 entries, fp32
  mode-router W_r, b_r  ~ U(-1/32, 1/32) before steering
Every tensor except biases and u is rounded (round-to-nearest-even) to the
workload's storage dtype; all later arithmetic sees only the stored values.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional, Sequence

import numpy as np
import torch

BASE_SEED = 67          # the paper's training seed (implementation details)
H_HEADS = 16            # heads per global-attention layer (Section 3)
HEAD_DIM = 64           # per-head dimension d
HIDDEN = 64             # router and surrogate hidden size (implementation details)
TOKENS_PER_VIEW = 1374  # 1 camera + 4 register + 37*37 patch tokens
N_MODES = 3             # MEAN=0 < SURR=1 < FULL=2, ordered by compute
MODE_MEAN, MODE_SURR, MODE_FULL = 0, 1, 2

_MASK64 = (1 << 64) - 1

TENSOR_IDS = {
    "Q": 1, "K": 2, "V": 3, "W": 4, "U": 5, "w": 6,
    "u": 7, "Wr": 8, "br": 9, "perm": 10, "margin": 11,
    "g_w1": 12, "g_b1": 13, "g_w2": 14, "g_b2": 15,
    "d_w1": 16, "d_b1": 17, "d_w2": 18, "d_b2": 19,
    "rows": 20,
    "X": 30, "ln1_w": 31, "ln1_b": 32, "w_qkv": 33, "b_qkv": 34, "w_o": 35, "b_o": 36,
    "ls1": 37, "ln2_w": 38, "ln2_b": 39, "w_fc1": 40, "b_fc1": 41, "w_fc2": 42, "b_fc2": 43,
    "ls2": 44,
}
SPECIAL_TOKENS = 5      # camera + 4 register tokens at the start of every view
PATCH_GRID = 37         # patch tokens per row of the 37 x 37 grid


def splitmix64(x: int) -> int:
    """One SplitMix64 output for state ``x`` (Steele, Lea, Flood 2014)."""
    z = (x + 0x9E3779B97F4A7C15) & _MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
    return z ^ (z >> 31)


def derive_seed(*keys: int) -> int:
    """Chain SplitMix64 over the base seed and integer keys; returns a 63-bit seed."""
    s = BASE_SEED
    for k in keys:
        s = splitmix64(s ^ (int(k) & _MASK64))
    return s & ((1 << 63) - 1)


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def normal(shape, seed: int, std: float = 1.0, device="cpu") -> torch.Tensor:
    g = _gen(seed, device)
    t = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
    return t.mul_(std)


def uniform(shape, seed: int, bound: float, device="cpu") -> torch.Tensor:
    g = _gen(seed, device)
    t = torch.rand(*shape, generator=g, device=device, dtype=torch.float32)
    return t.mul_(2.0 * bound).sub_(bound)


def torch_dtype(name: str) -> torch.dtype:
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def stored(t: torch.Tensor, dtype: str) -> torch.Tensor:
    """Round to the storage dtype (RNE for bf16)."""
    return t.to(torch_dtype(dtype))


def target_modes(n_full: int, seed: int, H: int = H_HEADS,
                 n_surr: Optional[int] = None) -> np.ndarray:
    """Seeded head -> mode map: a random permutation of the heads, the first
    ``n_full`` FULL, then ``n_surr`` SURR (default: half of the rest, rounded
    down), the remaining MEAN.  MEAN >= SURR mirrors the paper's measured mix
    (about 50% mean, 42% surrogate, 8% full: routing distribution table)."""
    if not 0 <= n_full <= H:
        raise ValueError("n_full out of range")
    rest = H - n_full
    if n_surr is None:
        n_surr = rest // 2
    if not 0 <= n_surr <= rest:
        raise ValueError("n_surr out of range")
    g = np.random.Generator(np.random.PCG64(seed))
    perm = g.permutation(H)
    modes = np.full(H, MODE_MEAN, dtype=np.uint8)
    modes[perm[:n_full]] = MODE_FULL
    modes[perm[n_full:n_full + n_surr]] = MODE_SURR
    return modes


def steer_bias(u: np.ndarray, W_r: np.ndarray, b_r: np.ndarray,
               modes: np.ndarray, margins: np.ndarray) -> np.ndarray:
    """Input construction for the linear-logit mode router: raise the bias of
    each head's target mode so that its logit exceeds the runner-up by
    ``margins[h]`` (computed in float64 on the stored values).  Returns the
    steered fp32 bias.  Not part of the layer; see module docstring."""
    H = modes.shape[0]
    raw = W_r.astype(np.float64) @ u.astype(np.float64) + b_r.astype(np.float64)
    raw = raw.reshape(H, N_MODES)
    b = b_r.astype(np.float64).reshape(H, N_MODES).copy()
    for h in range(H):
        t = int(modes[h])
        others = [raw[h, m] for m in range(N_MODES) if m != t]
        gap = max(others) - raw[h, t]
        b[h, t] += max(gap, 0.0) + float(margins[h])
    return b.reshape(-1).astype(np.float32)


@dataclasses.dataclass
class LayerInputs:
    S: int
    P: int
    H: int
    d: int
    L: int
    dtype: str
    Q: torch.Tensor          # [N, H, d] dtype
    K: torch.Tensor
    V: torch.Tensor
    W: torch.Tensor          # [H, L, d] dtype     (gated pooling, Eq.1)
    U: torch.Tensor          # [H, L, d] dtype
    w: torch.Tensor          # [H, L]    dtype
    u: torch.Tensor          # [H*d]     fp32      (mode-router input)
    Wr: torch.Tensor         # [H*3, H*d] dtype
    br: torch.Tensor         # [H*3]     fp32 (steered)
    surr: Dict[str, torch.Tensor]   # g_w1 [H,L,2d], g_b1 [H,L], g_w2 [H,d,L], g_b2 [H,d], d_*
    modes: np.ndarray        # [H] uint8 target modes

    @property
    def N(self) -> int:
        return self.S * self.P

    def to(self, device) -> "LayerInputs":
        f = {}
        for fld in dataclasses.fields(self):
            v = getattr(self, fld.name)
            if isinstance(v, torch.Tensor):
                v = v.to(device)
            elif isinstance(v, dict):
                v = {k: t.to(device) for k, t in v.items()}
            f[fld.name] = v
        return LayerInputs(**f)


def make_layer(S: int, P: int = TOKENS_PER_VIEW, dtype: str = "bf16", n_full: int = 8,
               n_surr: Optional[int] = None, key: Sequence[int] = (0, 0),
               qkv_device="cpu", sharp: bool = False, H: int = H_HEADS,
               d: int = HEAD_DIM, L: int = HIDDEN,
               modes: Optional[np.ndarray] = None, with_qkv: bool = True) -> LayerInputs:
    """Seeded inputs of one routed global-attention layer.

    ``key`` = (workload id, layer index) selects the seed stream.  Q/K/V are
    drawn on ``qkv_device`` (a CUDA device for the large workloads); the small
    weight tensors are always drawn on the CPU.  ``with_qkv=False`` leaves
    Q/K/V empty (a layer inside a block, whose Q/K/V come from the block).
    """
    N = S * P
    sd = lambda name: derive_seed(*key, TENSOR_IDS[name])
    std = 1.0 if sharp else 1.0 / np.sqrt(d)
    if with_qkv:
        Q = stored(normal((N, H, d), sd("Q"), std, qkv_device), dtype)
        K = stored(normal((N, H, d), sd("K"), std, qkv_device), dtype)
        V = stored(normal((N, H, d), sd("V"), 1.0 / np.sqrt(d), qkv_device), dtype)
    else:
        Q = K = V = torch.empty(0, dtype=torch_dtype(dtype))

    bw = 1.0 / np.sqrt(d)
    W = stored(uniform((H, L, d), sd("W"), bw), dtype)
    U = stored(uniform((H, L, d), sd("U"), bw), dtype)
    w = stored(uniform((H, L), sd("w"), 1.0 / np.sqrt(L)), dtype)

    Din = H * d
    u = stored(normal((Din,), sd("u"), 1.0 / np.sqrt(d)), dtype).float()
    Wr = stored(uniform((H * N_MODES, Din), sd("Wr"), 1.0 / 32), dtype)
    br0 = uniform((H * N_MODES,), sd("br"), 1.0 / 32)
    if modes is None:
        modes = target_modes(n_full, sd("perm"), H, n_surr)
    modes = np.asarray(modes, dtype=np.uint8)
    mg = np.random.Generator(np.random.PCG64(sd("margin")))
    margins = mg.uniform(2e-3, 2e-2, size=H)
    br = torch.from_numpy(steer_bias(u.numpy(), Wr.float().numpy(), br0.numpy(), modes, margins))

    b1 = 1.0 / np.sqrt(2 * d)
    b2 = 1.0 / np.sqrt(L)
    surr = {
        "g_w1": stored(uniform((H, L, 2 * d), sd("g_w1"), b1), dtype),
        "g_b1": uniform((H, L), sd("g_b1"), b1),
        "g_w2": stored(uniform((H, d, L), sd("g_w2"), b2), dtype),
        "g_b2": uniform((H, d), sd("g_b2"), b2),
        "d_w1": stored(uniform((H, L, 2 * d), sd("d_w1"), b1), dtype),
        "d_b1": uniform((H, L), sd("d_b1"), b1),
        "d_w2": stored(uniform((H, d, L), sd("d_w2"), b2), dtype),
        "d_b2": uniform((H, d), sd("d_b2"), b2),
    }
    return LayerInputs(S=S, P=P, H=H, d=d, L=L, dtype=dtype, Q=Q, K=K, V=V, W=W, U=U, w=w,
                       u=u, Wr=Wr, br=br, surr=surr, modes=modes)


def sample_rows(N: int, R: int, seed: int) -> np.ndarray:
    """R distinct seeded query rows of N (sorted), always including the last row
    so that the ragged tail of a tiled kernel is sampled."""
    R = min(R, N)
    g = np.random.Generator(np.random.PCG64(seed))
    rows = g.choice(N, size=R, replace=False)
    rows[-1] = N - 1
    return np.unique(rows).astype(np.int64)


# Workloads (S views x 1374 tokens, 16 heads x 64), with the head mix each uses.
WORKLOADS = {
    "s2_f32":   dict(S=2,   dtype="f32",  n_full=8),
    "s8_bf16":  dict(S=8,   dtype="bf16", n_full=8),
    "s32_bf16": dict(S=32,  dtype="bf16", n_full=4),
    "s100_bf16": dict(S=100, dtype="bf16", n_full=4),
    "s500_bf16": dict(S=500, dtype="bf16", n_full=4),
}


# ----------------------------------------------------- block around the layer
#
# Inputs of the dense block of Algorithm 1 (LN_1, QKV with positions, W_O,
# LayerScale, LN_2, FFN) for D = H * d = 1024 and FFN width 4 D:
#   X                       ~ N(0, 1)                        (stored dtype)
#   LN gains ~ U(0.5, 1.5), LN biases ~ U(-0.1, 0.1)        (fp32)
#   W_qkv, W_o, W_fc1       ~ U(-1/sqrt(D), 1/sqrt(D))      (stored dtype)
#   W_fc2                   ~ U(-1/sqrt(4D), 1/sqrt(4D))    (stored dtype)
#   biases                  ~ U(-0.02, 0.02)                 (fp32)
#   LayerScale LS_1, LS_2   ~ U(0.5, 1.5)                    (fp32; large enough
#                             that both residual branches matter in parity tests)
# Positions: the SPECIAL_TOKENS tokens of a view at (0, 0), patch k of the view
# at (k // PATCH_GRID + 1, k % PATCH_GRID + 1).

BLOCK_KEYS = ("ln1_w", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o", "ls1", "ln2_w", "ln2_b",
              "w_fc1", "b_fc1", "w_fc2", "b_fc2", "ls2")


def token_positions(S: int, P: int = TOKENS_PER_VIEW) -> np.ndarray:
    """(row, column) of every token of S views of P tokens: int32 [S * P, 2]."""
    t = np.arange(P)
    k = t - SPECIAL_TOKENS
    rc = np.stack([k // PATCH_GRID + 1, k % PATCH_GRID + 1], axis=1)
    rc[t < SPECIAL_TOKENS] = 0
    return np.ascontiguousarray(np.tile(rc, (S, 1)), dtype=np.int32)


def make_block_weights(key: Sequence[int] = (0, 0), dtype: str = "bf16", H: int = H_HEADS,
                       d: int = HEAD_DIM) -> Dict[str, torch.Tensor]:
    """Seeded weights of one dense block (CPU tensors)."""
    D = H * d
    sd = lambda name: derive_seed(*key, TENSOR_IDS[name])
    u = lambda name, shape, lo, hi: uniform(shape, sd(name), (hi - lo) / 2) + (hi + lo) / 2
    mat = lambda name, shape, fan: stored(uniform(shape, sd(name), 1.0 / np.sqrt(fan)), dtype)
    return {
        "ln1_w": u("ln1_w", (D,), 0.5, 1.5), "ln1_b": u("ln1_b", (D,), -0.1, 0.1),
        "w_qkv": mat("w_qkv", (3 * D, D), D), "b_qkv": u("b_qkv", (3 * D,), -0.02, 0.02),
        "w_o": mat("w_o", (D, D), D), "b_o": u("b_o", (D,), -0.02, 0.02),
        "ls1": u("ls1", (D,), 0.5, 1.5),
        "ln2_w": u("ln2_w", (D,), 0.5, 1.5), "ln2_b": u("ln2_b", (D,), -0.1, 0.1),
        "w_fc1": mat("w_fc1", (4 * D, D), D), "b_fc1": u("b_fc1", (4 * D,), -0.02, 0.02),
        "w_fc2": mat("w_fc2", (D, 4 * D), 4 * D), "b_fc2": u("b_fc2", (D,), -0.02, 0.02),
        "ls2": u("ls2", (D,), 0.5, 1.5),
    }


def make_block_input(S: int, P: int = TOKENS_PER_VIEW, key: Sequence[int] = (0, 0),
                     dtype: str = "bf16", D: int = H_HEADS * HEAD_DIM, device="cpu"):
    """Seeded block input tokens X [S * P, D] in the stored dtype."""
    return stored(normal((S * P, D), derive_seed(*key, TENSOR_IDS["X"]), 1.0, device), dtype)
