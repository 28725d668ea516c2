"""Pins of the oracle's dense block around the routed layer (Algorithm 1,
steps 1, 3 and 4): LayerNorm, the 2D rotary encoding of the positional
information, GELU, the linear layers and their composition.  CPU only.

Each function is tied to something other than its own code: library
routines (torch layer_norm and gelu in float64), an independent formulation
(the rotation as a complex multiplication), invariants (rotation preserves
norms and makes dot products depend only on position differences), published
constants (the standard normal CDF at 1) and closed forms of the block
with zeroed weights."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2609_23733_amd import synth

RNG = np.random.default_rng(2024)


# ----------------------------------------------------------------- LayerNorm

def test_layernorm_matches_torch():
    X = RNG.normal(size=(37, 1024)).astype(np.float32) * 3 + 1
    g = RNG.uniform(0.5, 1.5, 1024).astype(np.float32)
    b = RNG.uniform(-0.1, 0.1, 1024).astype(np.float32)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(X).double(), (1024,),
                                         torch.from_numpy(g).double(),
                                         torch.from_numpy(b).double(), eps=1e-6).numpy()
    np.testing.assert_allclose(oracle.layernorm(X, g, b), ref, rtol=0, atol=1e-12)


def test_layernorm_closed_forms():
    g = RNG.uniform(0.5, 1.5, 64).astype(np.float32)
    b = RNG.uniform(-0.1, 0.1, 64).astype(np.float32)
    # a constant row has zero variance: every output is the bias
    const = np.full((3, 64), 2.5, np.float32)
    np.testing.assert_array_equal(oracle.layernorm(const, g, b), np.tile(b, (3, 1)))
    # without eps the output is invariant to an affine map of the row
    x = RNG.normal(size=(4, 64))
    one = np.ones(64, np.float32)
    zero = np.zeros(64, np.float32)
    y1 = oracle.layernorm(x, one, zero, eps=0.0)
    y2 = oracle.layernorm(7.0 * x - 3.0, one, zero, eps=0.0)
    np.testing.assert_allclose(y1, y2, atol=1e-12)
    # and has zero mean and unit (biased) variance per row
    np.testing.assert_allclose(y1.mean(axis=1), 0, atol=1e-12)
    np.testing.assert_allclose((y1 ** 2).mean(axis=1), 1, atol=1e-12)


# ----------------------------------------------------------- rotary encoding

def _pairs(T):
    """Complex view of the rotated planes of [N, H, 64]: half (0 row, 1
    column) and pair j -> feature j + 32 half and j + 16 + 32 half."""
    z = np.empty(T.shape[:-1] + (2, 16), complex)
    for half in range(2):
        z[..., half, :] = T[..., 32 * half:32 * half + 16] + 1j * T[..., 32 * half + 16:32 * half + 32]
    return z


def test_rope_is_a_complex_rotation():
    """Independent formulation: each plane (j, j + 16) of a half is the complex
    number u + i w multiplied by exp(i p w_j), w_j = base^(-j/16), p the row
    (first half) or column (second half) coordinate."""
    N, H = 11, 3
    T = RNG.normal(size=(N, H, 64))
    pos = RNG.integers(0, 40, size=(N, 2)).astype(np.int32)
    R = oracle.rope2d(T, pos)
    z, zr = _pairs(T), _pairs(R)
    w = 100.0 ** (-np.arange(16) / 16.0)
    for half in range(2):
        rot = np.exp(1j * pos[:, half, None] * w[None, :])[:, None, :]
        np.testing.assert_allclose(zr[:, :, half, :], z[:, :, half, :] * rot, atol=1e-12)


def test_rope_identity_norm_and_relative_position():
    N, H = 9, 2
    T = RNG.normal(size=(N, H, 64))
    zero = np.zeros((N, 2), np.int32)
    np.testing.assert_array_equal(oracle.rope2d(T, zero), T)
    pos = RNG.integers(0, 38, size=(N, 2)).astype(np.int32)
    R = oracle.rope2d(T, pos)
    # every rotated plane keeps its length
    np.testing.assert_allclose(np.abs(_pairs(R)), np.abs(_pairs(T)), atol=1e-12)
    # <R(p) q, R(p') k> = <q, R(p' - p) k>: only position differences matter
    q = RNG.normal(size=(1, 1, 64))
    k = RNG.normal(size=(1, 1, 64))
    p1 = np.array([[5, 9]], np.int32)
    p2 = np.array([[12, 3]], np.int32)
    lhs = float((oracle.rope2d(q, p1) * oracle.rope2d(k, p2)).sum())
    shift = np.array([[7, -6]], np.int32)
    rhs = float((q * oracle.rope2d(k, shift)).sum())
    assert abs(lhs - rhs) < 1e-12
    # frequency 0 of the row half rotates by exactly the row coordinate
    e = np.zeros((1, 1, 64))
    e[0, 0, 0] = 1.0
    r = oracle.rope2d(e, np.array([[3, 0]], np.int32))
    assert abs(r[0, 0, 0] - math.cos(3)) < 1e-15 and abs(r[0, 0, 16] - math.sin(3)) < 1e-15
    assert np.count_nonzero(np.abs(r) > 1e-15) == 2


# ---------------------------------------------------------------------- GELU

def test_gelu_library_and_identities():
    x = np.linspace(-8, 8, 1001)
    ref = torch.nn.functional.gelu(torch.from_numpy(x), approximate="none").numpy()
    np.testing.assert_allclose(oracle.gelu(x), ref, atol=1e-15)
    # GELU(x) - GELU(-x) = x, and GELU(1) = Phi(1) (standard normal CDF table)
    np.testing.assert_allclose(oracle.gelu(x) - oracle.gelu(-x), x, atol=1e-12)
    assert abs(oracle.gelu(np.array([1.0]))[0] - 0.8413447460685429) < 1e-15


# ------------------------------------------------------------ linear, block

def test_linear_identity_weight():
    X = RNG.normal(size=(5, 8))
    b = RNG.normal(size=8).astype(np.float32)
    np.testing.assert_allclose(oracle.linear(X, np.eye(8, dtype=np.float32), b),
                               X + b.astype(np.float64), atol=1e-15)


def small_block(seed=5):
    wt = synth.make_block_weights((seed, 0), dtype="f32", H=2, d=64)
    X = synth.make_block_input(1, 7, key=(seed, 0), dtype="f32", D=128)
    return X, wt


def test_block_out_closed_forms():
    """W_O = 0: X_attn = X + LS_1 b_O; W_fc2 = 0 as well: the output adds
    LS_2 b_fc2 (the FFN reduces to its last bias)."""
    X, wt = small_block()
    Y = torch.randn(7, 128, generator=torch.Generator().manual_seed(1))
    wt["w_o"] = torch.zeros_like(wt["w_o"])
    wt["w_fc2"] = torch.zeros_like(wt["w_fc2"])
    out, Xa = oracle.block_out(X, Y, wt)
    X64 = X.double().numpy()
    f64 = lambda k: wt[k].double().numpy()
    np.testing.assert_allclose(Xa, X64 + f64("ls1") * f64("b_o"), atol=1e-12)
    np.testing.assert_allclose(out, Xa + f64("ls2") * f64("b_fc2"), atol=1e-12)


def test_block_out_matches_torch_modules():
    """The composition against torch's own layers in float64."""
    X, wt = small_block(6)
    Y = torch.randn(7, 128, generator=torch.Generator().manual_seed(2), dtype=torch.float64)
    out, Xa = oracle.block_out(X, Y.float(), wt)
    d = {k: v.double() for k, v in wt.items()}
    Yf = Y.float().double()
    xa = X.double() + d["ls1"] * torch.nn.functional.linear(Yf, d["w_o"], d["b_o"])
    z = torch.nn.functional.layer_norm(xa, (128,), d["ln2_w"], d["ln2_b"], eps=1e-6)
    f = torch.nn.functional.linear(
        torch.nn.functional.gelu(torch.nn.functional.linear(z, d["w_fc1"], d["b_fc1"])),
        d["w_fc2"], d["b_fc2"])
    np.testing.assert_allclose(Xa, xa.numpy(), atol=1e-12)
    np.testing.assert_allclose(out, (xa + d["ls2"] * f).numpy(), atol=1e-12)


def test_block_qkv_without_positions_and_equivariance():
    X, wt = small_block(7)
    zero = np.zeros((7, 2), np.int32)
    Q, K, V = oracle.block_qkv(X, zero, wt, H=2)
    d = {k: v.double() for k, v in wt.items()}
    xn = torch.nn.functional.layer_norm(X.double(), (128,), d["ln1_w"], d["ln1_b"], eps=1e-6)
    qkv = torch.nn.functional.linear(xn, d["w_qkv"], d["b_qkv"]).numpy()
    np.testing.assert_allclose(Q.reshape(7, 128), qkv[:, :128], atol=1e-12)
    np.testing.assert_allclose(K.reshape(7, 128), qkv[:, 128:256], atol=1e-12)
    np.testing.assert_allclose(V.reshape(7, 128), qkv[:, 256:], atol=1e-12)
    # permuting tokens together with their positions permutes the outputs
    pos = synth.token_positions(1, 7)
    pi = np.array([3, 0, 6, 1, 5, 2, 4])
    a = oracle.block_qkv(X, pos, wt, H=2)
    b = oracle.block_qkv(X[torch.from_numpy(pi)], pos[pi], wt, H=2)
    for u, v in zip(a, b):
        np.testing.assert_allclose(u[pi], v, atol=1e-12)
    # V carries no positional rotation
    np.testing.assert_allclose(a[2], V, atol=1e-12)


@pytest.mark.parametrize("P", [1, 6, 40])
def test_token_positions(P):
    pos = synth.token_positions(2, P)
    assert pos.shape == (2 * P, 2) and pos.dtype == np.int32
    assert (pos[:min(P, 5)] == 0).all()
    if P > 5:
        assert tuple(pos[5]) == (1, 1)
    np.testing.assert_array_equal(pos[:P], pos[P:])
