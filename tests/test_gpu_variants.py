"""GPU parity of the ablation variants of the routed layer (Section 5.3:
component study, Table 5; compute-mode study, Table 6) against the fp64
oracle, through the C ABI:
  - binary routing (MEAN / FULL only), threshold and logit forms;
  - mean query instead of gated attention pooling;
  - mean context, no residual correction, identity added (surrogate forms);
  - linear attention (phi = elu + 1) in place of the surrogate.
Tolerances are those of the base layer (tests/test_gpu_parity.py)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_23733_amd import synth
from test_gpu_parity import (check_router, check_y, log, oracle_layer, planted_inputs, rms,
                             run_gpu)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_23733_amd import vp
    vp.load_library()


ALL_MODES = np.array([2, 1, 0, 2, 2, 1, 0, 0, 1, 2, 0, 1, 2, 0, 1, 2], np.uint8)
TWO_MODES = np.array([2, 0, 0, 2, 0, 2, 2, 0, 0, 0, 2, 0, 2, 0, 0, 2], np.uint8)
VARIANTS = [oracle.SURR_MEAN_CONTEXT, oracle.SURR_NO_RESIDUAL, oracle.SURR_ADD_IDENTITY,
            oracle.SURR_LINEAR_ATTN]


# ------------------------------------------------------------ binary routing

def test_binary_assign_boundaries_and_nan():
    from paper_2609_23733_amd import vp
    log("binary assign boundaries")
    tl, th = np.float32(0.01), np.float32(0.2)
    s = np.array([th, tl, np.nextafter(th, 0), np.nextafter(tl, 1), 1.0, 0.0, np.nan, 0.05],
                 np.float32)
    modes, buckets = vp.assign_heads(torch.from_numpy(s).cuda(), vp.RULE_THRESHOLD_BINARY)
    torch.cuda.synchronize()
    want = oracle.assign(s.astype(np.float64), oracle.RULE_THRESHOLD_BINARY, tl, th)
    np.testing.assert_array_equal(want, [2, 0, 0, 0, 2, 0, 2, 0])
    np.testing.assert_array_equal(modes.cpu().numpy(), want)
    counts, lst = oracle.buckets(want)
    b = buckets.cpu().numpy()
    np.testing.assert_array_equal(b[:3], counts)
    np.testing.assert_array_equal(b[3:3 + len(lst)], lst)
    assert b[19] & 1
    # logits: ties go to MEAN; a NaN in a compared logit -> FULL + flag; the
    # SURR logit is never compared (a NaN there changes nothing)
    lg = np.array([[1, 1, 0], [0, 2, 2], [3, 3, 3], [0, 0, 1], [-1, -2, -3], [0, 9, -1],
                   [0, np.nan, -1]], np.float32)
    modes, buckets = vp.assign_heads(torch.from_numpy(lg).cuda(), vp.RULE_ARGMAX_BINARY)
    torch.cuda.synchronize()
    want = oracle.assign(lg.astype(np.float64), oracle.RULE_ARGMAX_BINARY)
    np.testing.assert_array_equal(want, [0, 2, 0, 2, 0, 0, 0])
    np.testing.assert_array_equal(modes.cpu().numpy(), want)
    assert buckets.cpu().numpy()[19] == 0
    lg[4, 0] = np.nan
    modes, buckets = vp.assign_heads(torch.from_numpy(lg).cuda(), vp.RULE_ARGMAX_BINARY)
    torch.cuda.synchronize()
    assert modes.cpu().numpy()[4] == 2 and buckets.cpu().numpy()[19] & 1


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_binary_argmax_layer(dtype):
    """Logit routing restricted to MEAN and FULL; the target modes win by the
    steering margin, so the MEAN-vs-FULL comparison has that margin too."""
    log("binary argmax layer %s" % dtype)
    x = synth.make_layer(1, 1000, dtype=dtype, key=(11, 0), sharp=True, modes=TWO_MODES,
                         qkv_device="cuda")
    layer = run_gpu(x, rule=oracle.RULE_ARGMAX_BINARY, y_dtype=torch.float32)
    ref = oracle_layer(x, rule=oracle.RULE_ARGMAX_BINARY)
    np.testing.assert_array_equal(ref["modes"], TWO_MODES)
    check_router(layer, ref, oracle.RULE_ARGMAX_BINARY)
    check_y(layer.Y.double().cpu().numpy(), ref["Y"], dtype, False, label="binary argmax")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_binary_threshold_layer_planted(dtype):
    """Planted saliencies on both sides of tau_high and between the two
    thresholds (SURR under Eq.4, MEAN under the binary rule)."""
    N = 2748
    log("binary threshold planted %s" % dtype)
    targets = [0.22, 0.18, 0.014, 0.006, 0.6, 0.05, 0.1, 0.3,
               0.015, 0.005, 0.25, 0.12, 0.9, 0.02, 0.17, 0.23]
    x = planted_inputs(N, targets, dtype)
    ref = oracle_layer(x, rule=oracle.RULE_THRESHOLD_BINARY)
    assert (np.abs(ref["s"] - 0.2) >= 1e-3).all()
    assert set(ref["modes"].tolist()) == {0, 2}
    layer = run_gpu(x.to("cuda"), rule=oracle.RULE_THRESHOLD_BINARY, y_dtype=torch.float32)
    check_router(layer, ref, oracle.RULE_THRESHOLD_BINARY)
    check_y(layer.Y.double().cpu().numpy(), ref["Y"], dtype, False, label="binary planted")


# ---------------------------------------------------------------- mean query

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("S,P", [(1, 1), (1, 300), (2, 1000)])
def test_mean_query(dtype, S, P):
    """Router with the plain query mean as pooled query: q_pool, s, C and the
    SURR heads (which read C) follow it; modes come from the logit router."""
    log("mean query %s S=%d P=%d" % (dtype, S, P))
    x = synth.make_layer(S, P, dtype=dtype, key=(12, S * P), sharp=True, modes=ALL_MODES,
                         qkv_device="cuda")
    layer = run_gpu(x, y_dtype=torch.float32, pool=oracle.POOL_MEAN)
    ref = oracle_layer(x, pool=oracle.POOL_MEAN)
    q_mean = x.Q.double().mean(dim=0).cpu().numpy()
    assert np.abs(ref["q_pool"] - q_mean).max() <= 1e-12
    check_router(layer, ref, oracle.RULE_ARGMAX)
    check_y(layer.Y.double().cpu().numpy(), ref["Y"], dtype, False, label="mean query")


# ------------------------------------------------------- surrogate variants

@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("P", [1, 65, 1000])
def test_surrogate_variants(variant, dtype, P):
    """Every head mode present; SURR heads computed by the variant; ragged
    token counts around the 64-token tiles and 512/256-token blocks."""
    log("surrogate variant %d %s P=%d" % (variant, dtype, P))
    x = synth.make_layer(2, P, dtype=dtype, key=(13, P), sharp=True, modes=ALL_MODES,
                         qkv_device="cuda")
    layer = run_gpu(x, y_dtype=torch.float32, surr_variant=variant)
    ref = oracle_layer(x, surr_variant=variant)
    check_router(layer, ref, oracle.RULE_ARGMAX)
    check_y(layer.Y.double().cpu().numpy(), ref["Y"], dtype, False,
            label="variant %d P=%d" % (variant, P))


@pytest.mark.parametrize("variant", VARIANTS)
def test_surrogate_variants_bf16_output(variant):
    log("surrogate variant %d, bf16 Y" % variant)
    x = synth.make_layer(2, 700, dtype="bf16", key=(14, 0), sharp=True, n_full=4,
                         qkv_device="cuda")
    layer = run_gpu(x, y_dtype=torch.bfloat16, surr_variant=variant)
    ref = oracle_layer(x, surr_variant=variant)
    check_router(layer, ref, oracle.RULE_ARGMAX)
    check_y(layer.Y.double().cpu().numpy(), ref["Y"], "bf16", True, label="variant %d" % variant)


def test_no_residual_is_the_context_and_identity_adds_v():
    """Closed forms on the GPU outputs alone: no residual gives C_h on every
    row; identity-added minus Eq.7 is V exactly up to fp32 rounding."""
    log("no residual / identity closed forms")
    x = synth.make_layer(1, 777, dtype="f32", key=(15, 0), sharp=True, modes=ALL_MODES,
                         qkv_device="cuda")
    surr = [h for h in range(16) if ALL_MODES[h] == 1]
    a = run_gpu(x, y_dtype=torch.float32, surr_variant=oracle.SURR_NO_RESIDUAL)
    ctx = a.state.ctx.cpu().numpy()
    Ya = a.Y.cpu().numpy()
    for h in surr:
        np.testing.assert_array_equal(Ya[:, h, :], np.broadcast_to(ctx[h], Ya[:, h, :].shape))
    b = run_gpu(x, y_dtype=torch.float32, surr_variant=oracle.SURR_EQ7).Y.double().cpu().numpy()
    c = run_gpu(x, y_dtype=torch.float32,
                surr_variant=oracle.SURR_ADD_IDENTITY).Y.double().cpu().numpy()
    V = x.V.double().cpu().numpy()
    for h in surr:
        assert np.abs(c[:, h] - b[:, h] - V[:, h]).max() <= 1e-6
    for h in range(16):
        if ALL_MODES[h] != 1:   # other heads do not depend on the variant
            assert np.array_equal(c[:, h], b[:, h]) and np.array_equal(Ya[:, h], b[:, h])


def test_linear_attention_uniform_keys_give_value_mean():
    """All keys equal: every weight phi(q).phi(k) is the same, so each row of
    a linear-attention head is the mean value token."""
    log("linear attention, equal keys")
    x = synth.make_layer(1, 999, dtype="f32", key=(16, 0), sharp=True, modes=ALL_MODES,
                         qkv_device="cuda")
    x.K = x.K[:1].expand_as(x.K).contiguous()
    layer = run_gpu(x, y_dtype=torch.float32, surr_variant=oracle.SURR_LINEAR_ATTN)
    Y = layer.Y.double().cpu().numpy()
    vm = x.V.double().mean(dim=0).cpu().numpy()
    for h in range(16):
        if ALL_MODES[h] == 1:
            err = np.abs(Y[:, h] - vm[h]).max()
            assert err <= 1e-4 * rms(vm[h]), (h, err)


def test_variant_stages_and_determinism():
    """The three-stage path (gather, FULL, linear heads with Q, K and the
    workspace) equals the one-call path bit for bit, and reruns are bitwise
    identical, for the linear-attention variant."""
    from paper_2609_23733_amd import vp
    log("linear attention stages / determinism")
    x = synth.make_layer(4, 1374, dtype="bf16", key=(17, 0), n_full=4, qkv_device="cuda")
    layer = vp.RoutedLayer(x, y_dtype=torch.bfloat16, surr_variant=vp.SURR_LINEAR_ATTN,
                           pool=vp.POOL_MEAN)
    Y1 = layer.step().clone()
    ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    Y2 = layer.step(events=ev).clone()
    Y3 = layer.step().clone()
    torch.cuda.synchronize()
    assert torch.equal(Y1, Y2) and torch.equal(Y1, Y3)


# ------------------------------------------------------------ full size

@pytest.mark.parametrize("variant,pool", [(oracle.SURR_LINEAR_ATTN, oracle.POOL_GATED),
                                          (oracle.SURR_ADD_IDENTITY, oracle.POOL_MEAN)])
def test_variants_full_size_sampled(variant, pool):
    """S = 100 views (N = 137,400), bf16 operands and output, four FULL heads:
    router and modes on all tokens, every head on sampled rows."""
    cfg = synth.WORKLOADS["s100_bf16"]
    log("full size s100 variant %d pool %d" % (variant, pool))
    x = synth.make_layer(cfg["S"], dtype="bf16", n_full=4, key=(cfg["S"], 0), qkv_device="cuda")
    layer = run_gpu(x, y_dtype=torch.bfloat16, pool=pool, surr_variant=variant)
    rows = synth.sample_rows(x.N, 64, synth.derive_seed(cfg["S"], 0, 21))
    ref = oracle_layer(x, rows=rows, full_rows_sel=rows, pool=pool, surr_variant=variant)
    check_router(layer, ref, oracle.RULE_ARGMAX)
    Yg = layer.Y[torch.from_numpy(rows).cuda()].double().cpu().numpy()
    for h in range(16):
        if ref["modes"][h] == 2:
            ref["Y"][:, h, :] = ref["Y_full_rows"][h]
    check_y(Yg, ref["Y"], "bf16", True, label="s100 variant %d pool %d" % (variant, pool))
