"""Benchmark of the routed global-attention layer on one MI355X.

A step is one pass of the whole layer on device-resident inputs:
router_score -> router_logits -> assign_heads -> routed global attention
(bucket gather, FULL-head attention, SURR/MEAN heads).  The headline
workload is S = 100 views x 1374 tokens (N = 137,400), 16 heads x 64, bf16
operands with fp32 accumulation, bf16 Y, 4 of 16 heads routed FULL by the
seeded linear-logit mode router.  The JSON line also carries the latency of
the other view counts and full-head counts (`by_workload`), the roofline of
the FULL-head kernel, and the fp64 CPU oracle timed on a bounded sample.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
"""
import argparse
import dataclasses
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "routed global-attn layer latency (ms) + TFLOP/s & % bf16 MFMA peak vs S"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3       # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0
P_TOKENS = 1374
HEADS, D, L = 16, 64, 64

# HBM traffic of k_flash_bf16 on the headline workload (S=100, 4 FULL heads),
# from two rocprofv3 --pmc passes (FETCH_SIZE, then WRITE_SIZE; KiB per
# dispatch) over this bench, each scaled by the same counter on a plain 1 GiB
# device-to-device copy (bench.py --copy-calibration): the copy reads FETCH_SIZE
# = 524305 KiB for 1 GiB read (x2.0) and WRITE_SIZE = 1048576 KiB for 1 GiB
# written (x1.0).  Valid only for the kernel source it was measured on.
FLASH_TRAFFIC = {
    "source_sha256": "f98be6b14a04ba6c40fa84e0c8dce862feb05c74357ab2f902ba95c9f40c2df7",
    "S": 100, "n_full": 4,
    "fetch_kib": 1545636, "write_kib": 122449,
    "copy_fetch_kib": 524305, "copy_write_kib": 1048576, "copy_bytes": 1 << 30,
}


def flash_traffic(S, n_full):
    """Measured HBM bytes per launch of the FULL-head kernel, or None when the
    kernel source or the workload differs from the measured one."""
    import hashlib
    src = os.path.join(ROOT, "paper_2609_23733_amd", "csrc", "flash.hip")
    t = FLASH_TRAFFIC
    if (S, n_full) != (t["S"], t["n_full"]):
        return None
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != t["source_sha256"]:
        return None
    fetch = t["fetch_kib"] * 1024 * t["copy_bytes"] / (t["copy_fetch_kib"] * 1024)
    write = t["write_kib"] * 1024 * t["copy_bytes"] / (t["copy_write_kib"] * 1024)
    return int(round(fetch + write))


def flops_full(N, n_full):
    """Algorithmic FULL-head work: QK^T and PV, 2 * N^2 * d each."""
    return 4.0 * N * N * D * n_full


def layer_flops(N, n_full, n_surr, n_mean):
    """Algorithmic work of the whole layer (complexity terms of the paper's
    appendix): FULL 4 N^2 d per head; router N H (4 d L + 2 L + 2 d) plus the
    single-query pass 4 N H d; SURR 8 d L N per head; MEAN N d per head."""
    router = N * HEADS * (4 * D * L + 2 * L + 2 * D) + 4 * N * HEADS * D
    return flops_full(N, n_full) + router + 8 * D * L * N * n_surr + N * D * n_mean


STAGES = ("router", "assign", "gather", "full", "linear")


def measure(layer, steps, warmup):
    """Average ms per layer pass over `steps` passes (HIP events around all of
    them), and per-stage averages from events recorded between the stages."""
    import torch
    for _ in range(warmup):
        layer.step()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(steps)]
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for k in range(steps):
        layer.step(stages=ev[k])
    t1.record()
    torch.cuda.synchronize()
    ms_step = t0.elapsed_time(t1) / steps
    stage = {name: sum(e[i].elapsed_time(e[i + 1]) for e in ev) / steps
             for i, name in enumerate(STAGES)}
    return ms_step, stage


def measure_graph(layer, steps, warmup):
    """Average ms per replay of the layer captured as a HIP graph (the same
    launches without per-call host work), HIP events around `steps` replays."""
    import torch
    from paper_2609_23733_amd import vp
    g = vp.LayerGraph(layer)
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        g.replay()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    del g
    return ms


def stage_bytes(N, n_full, n_surr, n_mean, b_in, b_out):
    """Algorithmic HBM bytes per stage: the router reads Q, K and V once; the
    gather reads K and V of each FULL head and writes its fp16 K and V^T
    tiles; SURR heads read V and write Y, MEAN heads write Y."""
    return {"router": 3.0 * N * HEADS * D * b_in,
            "gather": float(N) * D * n_full * (2 * b_in + 2 * 2) if b_in == 2 else 0.0,
            "linear": float(N) * D * (n_surr * (b_in + b_out) + n_mean * b_out)}


WIDE_QK_SCALE = 1.3   # sharp Q and K scaled by this: item bounds near 30 log2 units


def run_workload(S, n_full, steps, warmup, seed_key, dtype="bf16", sharp=False, wide=False):
    """One layer configuration; `wide` scales the sharp Q and K so that every
    FULL work item's logit bound exceeds the zero-reference window (running
    reference points throughout the FULL stage)."""
    import torch
    from paper_2609_23733_amd import synth, vp
    x = synth.make_layer(S, P_TOKENS, dtype=dtype, n_full=n_full, key=seed_key,
                         qkv_device="cuda", sharp=sharp or wide)
    if wide:
        x.Q = (x.Q.float() * WIDE_QK_SCALE).to(x.Q.dtype)
        x.K = (x.K.float() * WIDE_QK_SCALE).to(x.K.dtype)
    ydt = torch.bfloat16 if dtype == "bf16" else torch.float32
    layer = vp.RoutedLayer(x, y_dtype=ydt)
    ms_step, stage = measure(layer, steps, warmup)
    modes = layer.modes.cpu().numpy()
    counts = [int((modes == m).sum()) for m in range(3)]
    assert counts[2] == n_full, "router did not produce the target FULL count"
    ms_graph = measure_graph(layer, steps, warmup)
    N = S * P_TOKENS
    fl = layer_flops(N, counts[2], counts[1], counts[0])
    ff = flops_full(N, counts[2])
    peak = PEAK_BF16_TFLOPS if dtype == "bf16" else PEAK_FP32_TFLOPS
    b_in = 2 if dtype == "bf16" else 4
    b_out = 2 if ydt == torch.bfloat16 else 4
    byt = stage_bytes(N, counts[2], counts[1], counts[0], b_in, b_out)
    gbs = {k: round(v / stage[k] / 1e6, 1) for k, v in byt.items() if v and stage[k] > 0}
    full_ms = stage["full"]
    inputs = ("sharp N(0,1) Q/K x%g" % WIDE_QK_SCALE if wide else
              "sharp N(0,1) Q/K" if sharp else "N(0,1/64)")
    rec = dict(S=S, N=N, dtype=dtype, inputs=inputs,
               n_full=counts[2], n_surr=counts[1], n_mean=counts[0],
               ms=round(ms_step, 4), tflops=round(fl / ms_step / 1e9, 2),
               frac_peak=round(fl / ms_step / 1e9 / peak, 4),
               full_kernel_ms=round(full_ms, 4),
               full_kernel_tflops=round(ff / full_ms / 1e9, 2) if ff else None,
               full_kernel_frac=round(ff / full_ms / 1e9 / peak, 4) if ff else None,
               peak_tflops=peak,
               stage_ms={k: round(v, 4) for k, v in stage.items()},
               hbm_gbs=gbs,
               non_full_frac=round(1.0 - full_ms / ms_step, 4),
               ms_graph_replay=round(ms_graph, 4))
    return rec, layer, x


# Ablation variants of the layer (Section 5.3, Tables 5-6), timed on the
# headline inputs: (name, assignment rule, pooling, SURR-head variant).
VARIANTS = (
    ("eq7", 1, 0, 0),
    ("binary_argmax", 3, 0, 0),
    ("mean_query", 1, 1, 0),
    ("mean_context", 1, 0, 1),
    ("no_residual", 1, 0, 2),
    ("add_identity", 1, 0, 3),
    ("linear_attention", 1, 0, 4),
)


def linattn_flops(N, n_surr):
    """Linear attention per (token, SURR head): sum phi(k) v^T and sum phi(k)
    (2 d^2 + d), then phi(q)^T S and phi(q) . z (2 d^2 + 2 d)."""
    return float(N) * n_surr * (4 * D * D + 3 * D)


def run_variants(x, steps, warmup):
    """Layer latency per variant, and the SURR/MEAN stage (vp_linear_heads)
    alone, timed with HIP events over `steps` launches."""
    import torch
    from paper_2609_23733_amd import vp
    out = []
    for name, rule, pool, sv in VARIANTS:
        layer = vp.RoutedLayer(x, rule=rule, y_dtype=torch.bfloat16, pool=pool, surr_variant=sv)
        ms_step, stage = measure(layer, steps, warmup)
        full_avg = stage["full"]
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        xd = layer.x   # the layer's device copy of the inputs
        lin = lambda: vp.linear_heads(xd.V, layer.modes, layer.state, xd.surr, xd.S, xd.P,
                                      layer.Y, layer.act, sv, xd.Q, xd.K, layer.ws)
        for _ in range(warmup):
            lin()
        torch.cuda.synchronize()
        t0.record()
        for _ in range(steps):
            lin()
        t1.record()
        torch.cuda.synchronize()
        lin_ms = t0.elapsed_time(t1) / steps
        modes = layer.modes.cpu().numpy()
        counts = [int((modes == m).sum()) for m in range(3)]
        rec = dict(variant=name, ms=round(ms_step, 4), full_kernel_ms=round(full_avg, 4),
                   linear_stage_ms=round(lin_ms, 4), n_full=counts[2], n_surr=counts[1],
                   n_mean=counts[0])
        if sv == 4 and counts[1]:
            fl = linattn_flops(x.N, counts[1])
            ach = fl / lin_ms / 1e9
            rec["roofline"] = {"kernel": "k_linattn_partial + k_linattn_combine + "
                                         "k_linattn_apply (+ MEAN broadcast)",
                               "bound": "alu", "achieved": round(ach, 2),
                               "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                               "frac": round(ach / PEAK_FP32_TFLOPS, 4),
                               "algorithmic_flop_per_launch": fl}
        out.append(rec)
        del layer
    torch.cuda.empty_cache()
    return out


def block_gemm_flops(N):
    """Projections of one block: QKV (3D), W_O (D), FFN (4D and back), D = 1024."""
    Dm = HEADS * D
    return 2.0 * N * Dm * (3 * Dm + Dm + 4 * Dm + 4 * Dm)


def run_block(S, n_full, steps, warmup):
    """One global block of Algorithm 1 (LN_1, QKV with rotary positions, the
    routed layer, W_O, LayerScale, LN_2, FFN): per-stage latency from HIP
    events, and the projections' MFMA roofline."""
    import torch
    from paper_2609_23733_amd import synth, vp
    lay = synth.make_layer(S, P_TOKENS, dtype="bf16", n_full=n_full, key=(S, 7), with_qkv=False)
    blk = vp.PrimeBlock(lay, synth.make_block_weights((S, 7)), synth.token_positions(S, P_TOKENS))
    X = synth.make_block_input(S, P_TOKENS, key=(S, 7), device="cuda")
    Xo = torch.empty_like(X)
    for _ in range(warmup):
        blk.step(X, Xo)
    torch.cuda.synchronize()
    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in range(3)] for _ in range(steps)]
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for k in range(steps):
        blk.step(X, Xo, events=evs[k])
    t1.record()
    torch.cuda.synchronize()
    stage = [sum(e[i][0].elapsed_time(e[i][1]) for e in evs) / steps for i in range(3)]
    N = S * P_TOKENS
    fl = block_gemm_flops(N)
    ach = fl / (stage[0] + stage[2]) / 1e9
    return dict(S=S, N=N, n_full=int((blk.layer.modes == 2).sum()),
                ms=round(t0.elapsed_time(t1) / steps, 4), qkv_ms=round(stage[0], 4),
                routed_layer_ms=round(stage[1], 4), out_ms=round(stage[2], 4),
                roofline={"kernel": "k_gemm (QKV, W_O, FFN) + k_layernorm", "bound": "mfma",
                          "achieved": round(ach, 2), "peak": PEAK_BF16_TFLOPS,
                          "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                          "algorithmic_flop_per_launch": fl})


def run_stack(S, layers, steps, warmup, tome_ratio=None):
    """A stack of global blocks with independent seeded weights, layer l + 1
    taking layer l's output; FULL-head counts drawn from {1, ..., 6} per
    layer.  Per-layer latency from HIP events around each block.  With
    ``tome_ratio``, every block merges that fraction of its tokens before its
    routed layer and unmerges after it."""
    import numpy as np
    import torch
    from paper_2609_23733_amd import synth, vp
    rng = np.random.Generator(np.random.PCG64(synth.derive_seed(S, 500)))
    n_full = rng.integers(1, 7, size=layers)
    sh = vp.PrimeBlock.make_shared(S, P_TOKENS)
    pos = torch.from_numpy(synth.token_positions(S, P_TOKENS)).cuda()
    M = None if tome_ratio is None else int(tome_ratio * S * P_TOKENS)
    blocks = [vp.PrimeBlock(synth.make_layer(S, P_TOKENS, dtype="bf16", n_full=int(n_full[l]),
                                             key=(S, 100 + l), with_qkv=False),
                            synth.make_block_weights((S, 100 + l)), pos, shared=sh, tome_M=M)
              for l in range(layers)]
    X0 = synth.make_block_input(S, P_TOKENS, key=(S, 100), device="cuda")
    X = torch.empty_like(X0)

    def once(evs=None):
        X.copy_(X0)
        for l, b in enumerate(blocks):
            if evs is not None:
                evs[l][0].record()
            b.step(X, X)
            if evs is not None:
                evs[l][1].record()
    for _ in range(warmup):
        once()
    torch.cuda.synchronize()
    per = np.zeros(layers)
    for _ in range(steps):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(layers)]
        once(evs)
        torch.cuda.synchronize()
        per += [a.elapsed_time(b) for a, b in evs]
    per /= steps
    got = [int((b.layer.modes == 2).sum()) for b in blocks]
    out = dict(S=S, N=S * P_TOKENS, layers=layers, n_full=got,
               per_layer_ms=[round(float(v), 3) for v in per],
               total_ms=round(float(per.sum()), 3))
    if tome_ratio is not None:
        out = dict(tome_ratio=tome_ratio, merged_rows=blocks[0].tome.plan.nrows,
                   total_ms=out["total_ms"], per_layer_ms=out["per_layer_ms"], n_full=got)
    del blocks, sh
    torch.cuda.empty_cache()
    return out


def run_layer_stack(S, layers, steps, warmup):
    """A stack of routed layers at S views, each with its own seeded Q/K/V
    (drawn on the device before timing: 4.2 GB per layer at S = 500, all 24
    resident in HBM), router and surrogate weights, and a FULL-head count
    drawn from {1, ..., 6}; the layers share one workspace and output buffer.
    HIP events around each layer; MFMA work 4 N^2 d per FULL head."""
    import numpy as np
    import torch
    from paper_2609_23733_amd import synth, vp
    rng = np.random.Generator(np.random.PCG64(synth.derive_seed(S, 600)))
    n_full = rng.integers(1, 7, size=layers)
    N = S * P_TOKENS
    ws = vp.alloc_workspace(S, P_TOKENS, HEADS, torch.bfloat16)
    Y = torch.empty(N, HEADS, D, dtype=torch.bfloat16, device="cuda")
    lys = []
    for l in range(layers):
        x = synth.make_layer(S, P_TOKENS, dtype="bf16", n_full=int(n_full[l]), key=(S, 600 + l),
                             qkv_device="cuda")
        lys.append(vp.RoutedLayer(x, y_dtype=torch.bfloat16, ws=ws, Y=Y))
    torch.cuda.synchronize()

    def once(evs=None):
        for l, ly in enumerate(lys):
            if evs is not None:
                evs[l][0].record()
            ly.step()
            if evs is not None:
                evs[l][1].record()
    for _ in range(warmup):
        once()
    torch.cuda.synchronize()
    per = np.zeros(layers)
    for _ in range(steps):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(layers)]
        once(evs)
        torch.cuda.synchronize()
        per += [a.elapsed_time(b) for a, b in evs]
    per /= steps
    got = [int((ly.modes == 2).sum()) for ly in lys]
    fl = sum(flops_full(N, n) for n in got)
    tot = float(per.sum())
    del lys, ws, Y
    torch.cuda.empty_cache()
    return dict(S=S, N=N, layers=layers, n_full=got, qkv="independent seeded Q/K/V per layer",
                per_layer_ms=[round(float(v), 2) for v in per],
                total_ms=round(tot, 1), tflops=round(fl / tot / 1e9, 1),
                frac_bf16_peak=round(fl / tot / 1e9 / PEAK_BF16_TFLOPS, 4))


def run_teacher(S, steps, warmup):
    """Distillation targets of a teacher layer (every head FULL; Eq.8, Eq.10)
    and the two losses (Eq.9, Eq.11) on the same inputs: HIP-event latency
    and the algorithmic MFMA work per head: 4 N^2 d for the attention behind
    Delta^T (which also yields each query's softmax normaliser) + 2 N^2 d for
    the column maxima.  (The residual products that keep the teacher's logits
    exact are implementation work and not counted.)"""
    import torch
    from paper_2609_23733_amd import synth, vp
    x = synth.make_layer(S, P_TOKENS, dtype="bf16", key=(S, 9), qkv_device="cuda")
    Q, K, V = x.Q, x.K, x.V
    N = S * P_TOKENS
    shp = vp.make_shape(S, P_TOKENS, HEADS, torch.bfloat16)
    import ctypes
    ws = torch.empty(vp.load_library().vp_teacher_workspace_bytes(ctypes.byref(shp)),
                     dtype=torch.uint8, device="cuda")
    lws = vp.alloc_workspace(S, P_TOKENS, HEADS, torch.bfloat16)
    st = vp.router_score(Q, K, V, x.W.cuda(), x.U.cuda(), x.w.cuda(), S, P_TOKENS, lws)

    def timed(f):
        for _ in range(warmup):
            f()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            out = f()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / steps, out
    t_ms, (colmax, smax, delta) = timed(lambda: vp.teacher_targets(Q, K, V, S, P_TOKENS, ws=ws))
    r_ms, _ = timed(lambda: vp.router_loss(K, st, colmax, smax, S, P_TOKENS))
    l_ms, _ = timed(lambda: vp.latent_loss(delta, delta, S, P_TOKENS))
    fl = 6.0 * N * N * D * HEADS
    ach = fl / t_ms / 1e9
    return dict(S=S, N=N, heads=HEADS, teacher_targets_ms=round(t_ms, 3),
                router_loss_ms=round(r_ms, 4), latent_loss_ms=round(l_ms, 4),
                roofline={"kernel": "k_flash_bf16<teacher> + k_colmax + k_sub_v",
                          "bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_BF16_TFLOPS,
                          "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                          "algorithmic_flop_per_launch": fl})


def run_tome(S, n_full, ratios, steps, warmup, unmerged_ms):
    """Token merging around the routed layer (the paper's ToMe combination):
    plan, merge of Q/K/V, the routed layer on the merged rows, unmerge; HIP-
    event time of each stage, and the speedup over the unmerged layer."""
    import torch
    from paper_2609_23733_amd import synth, vp
    x = synth.make_layer(S, P_TOKENS, dtype="bf16", n_full=n_full, key=(S, 0), qkv_device="cuda")
    N = S * P_TOKENS
    out = []
    for ratio in ratios:
        M = int(ratio * N)
        tl = vp.TomeLayer(x, M, y_dtype=torch.bfloat16)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]

        def step(rec):
            if rec:
                ev[0].record()
            vp.tome_plan(x.K, tl.plan)
            if rec:
                ev[1].record()
            vp.tome_merge_qkv(x.Q, x.K, x.V, tl.plan, tl.Qm, tl.Km, tl.Vm)
            if rec:
                ev[2].record()
            Ym = tl.layer.step()
            if rec:
                ev[3].record()
            vp.tome_unmerge(Ym, tl.plan, tl.Y)
            if rec:
                ev[4].record()
        for _ in range(warmup):
            step(False)
        torch.cuda.synchronize()
        acc = [0.0] * 4
        for _ in range(steps):
            step(True)
            torch.cuda.synchronize()
            for i in range(4):
                acc[i] += ev[i].elapsed_time(ev[i + 1])
        t = [a / steps for a in acc]
        tot = sum(t)
        out.append(dict(ratio=ratio, M=M, rows=tl.plan.nrows, stride_g=tl.plan.g,
                        plan_ms=round(t[0], 4), merge_ms=round(t[1], 4), layer_ms=round(t[2], 4),
                        unmerge_ms=round(t[3], 4), total_ms=round(tot, 4),
                        speedup_vs_unmerged=round(unmerged_ms / tot, 2)))
        del tl
        torch.cuda.empty_cache()
    return dict(S=S, N=N, n_full=n_full, unmerged_layer_ms=round(unmerged_ms, 4), by_ratio=out)


def host_cpus():
    """What the host offers the oracle: logical CPUs, the CPUs this process may
    run on, the cgroup CPU quota (if any) and the CPU model string."""
    info = {"nproc": os.cpu_count()}
    try:
        info["affinity"] = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        info["affinity"] = None
    try:
        q, per = open("/sys/fs/cgroup/cpu.max").read().split()[:2]
        info["cgroup_quota_cpus"] = None if q == "max" else round(int(q) / int(per), 2)
    except (OSError, ValueError):
        info["cgroup_quota_cpus"] = None
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    info["model"] = model
    return info


# CPUs that one GPU's share of the box provides (the oracle's thread cap there).
CPU_SHARE = 16


def cpu_baseline(x, rows_per_head=800):
    """The fp64 oracle on a bounded sample of the same layer: the router over
    all N tokens, then `rows_per_head` query rows of every FULL and SURR head,
    extrapolated linearly to all N rows (every row costs the same).  It runs
    on every CPU the process may use, up to the per-GPU share of the box."""
    import oracle
    from paper_2609_23733_amd import synth
    host = host_cpus()
    avail = [v for v in (host["nproc"], host["affinity"], CPU_SHARE) if v]
    if host["cgroup_quota_cpus"]:
        avail.append(max(1, int(host["cgroup_quota_cpus"])))
    nt = max(1, min(avail))
    os.environ["VP_ORACLE_THREADS"] = str(nt)
    Q, K, V = oracle.as_f32(x.Q), oracle.as_f32(x.K), oracle.as_f32(x.V)
    N = Q.shape[0]
    t0 = time.perf_counter()
    qp = oracle.router_pool(Q, x.W, x.U, x.w)
    s, C, mean = oracle.router_route(K, V, qp)
    lg = oracle.router_logits(x.u, x.Wr, x.br)
    modes = oracle.assign(lg, oracle.RULE_ARGMAX)
    t_router = time.perf_counter() - t0
    rows = synth.sample_rows(N, rows_per_head, synth.derive_seed(500, 0, 20))
    t_rows = 0.0
    for h in range(Q.shape[1]):
        t1 = time.perf_counter()
        if modes[h] == 2:
            oracle.full_rows(Q, K, V, h, rows)
        elif modes[h] == 1:
            oracle.surr_rows(V, C[h], x.surr, h, rows)
        t_rows += time.perf_counter() - t1
    total = t_router + t_rows * N / len(rows)
    return dict(value=round(total * 1e3, 1), unit="ms", cores=oracle.threads_used(),
                kind="oracle", host=host,
                sample="router over all %d tokens (%.1f s) + %d sampled query rows per FULL and "
                       "SURR head (%.1f s), extrapolated to %d rows; MEAN heads free"
                       % (N, t_router, len(rows), t_rows, N),
                measured_s=round(t_router + t_rows, 1))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--n-full", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-variants", action="store_true")
    ap.add_argument("--no-block", action="store_true")
    ap.add_argument("--no-teacher", action="store_true")
    ap.add_argument("--no-tome", action="store_true")
    ap.add_argument("--no-stack500", action="store_true",
                    help="skip the 24-layer routed stack at S=500")
    ap.add_argument("--stack", type=int, default=0, metavar="S",
                    help="also time a 24-block stack at S views (e.g. 500)")
    ap.add_argument("--workload", default=None, metavar="S,NFULL[,sharp|wide|f32]",
                    help="time only this workload and print its record (for profiling runs)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy three times (the "
                         "reference for scaling the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    torch.cuda.set_device(0)
    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": 1 << 30, "launches": 3}))
        return
    from paper_2609_23733_amd import vp
    vp.load_library()
    if args.workload:
        f = args.workload.split(",")
        S, nf = int(f[0]), int(f[1])
        sharp, wide = "sharp" in f[2:], "wide" in f[2:]
        dt = "f32" if "f32" in f[2:] else "bf16"
        rec, _, _ = run_workload(S, nf, args.steps, args.warmup,
                                 (S, 3 if sharp or wide else 0), dtype=dt, sharp=sharp,
                                 wide=wide)
        print(json.dumps(rec))
        return

    head, layer, x = run_workload(100, args.n_full, args.steps, args.warmup, (100, 0))
    by = [head]
    variants = None
    if not args.no_variants:
        variants = run_variants(x, args.steps, args.warmup)
    del layer
    torch.cuda.empty_cache()
    block = None
    if not args.no_block:
        block = run_block(100, args.n_full, args.steps, args.warmup)
    tome = None
    if not args.no_tome:
        tome = run_tome(100, args.n_full, (0.75, 0.9), max(3, args.steps // 2), 2, head["ms"])
        torch.cuda.empty_cache()
    teacher = None
    if not args.no_teacher:
        teacher = run_teacher(100, max(2, args.steps // 4), 1)
        torch.cuda.empty_cache()
    stack500 = None
    if not args.no_stack500:
        stack500 = run_layer_stack(500, 24, 1, 1)
    stack = None
    if args.stack:
        stack = run_stack(args.stack, 24, 2, 1)
        stack["tome"] = [run_stack(args.stack, 24, 2, 1, r) for r in (0.75, 0.9)]
        for t in stack["tome"]:
            t["speedup_vs_unmerged_stack"] = round(stack["total_ms"] / t["total_ms"], 2)
    if not args.no_sweep:
        # S = 2 in fp32 (the fp32 FULL kernel against the fp32 matrix peak), the
        # other view counts and FULL-head counts, and S = 100 with sharp FULL
        # heads (logit bounds past the zero-reference window: EXT items, whose
        # reference point moves only on fp16 overflow) and with sharper ones
        # (bounds past the EXT window too: WIDE items, running reference points).
        sweep = ((2, 8, "f32", ""), (8, 8, "bf16", ""), (32, 4, "bf16", ""),
                 (32, 16, "bf16", ""), (100, 2, "bf16", ""), (100, 8, "bf16", ""),
                 (100, 16, "bf16", ""), (500, 4, "bf16", ""), (100, 4, "bf16", "sharp"),
                 (100, 4, "bf16", "wide"))
        for S, nf, dt, kind in sweep:
            r, lyr, _ = run_workload(S, nf, args.steps, args.warmup, (S, 3 if kind else 0),
                                     dtype=dt, sharp=kind == "sharp", wide=kind == "wide")
            by.append(r)
            del lyr
            torch.cuda.empty_cache()
        ref16 = [r for r in by if r["S"] == 100 and r["n_full"] == 16]
        if ref16:
            for r in by:
                if r["S"] == 100 and r["inputs"] == head["inputs"]:
                    r["speedup_vs_all_full"] = round(ref16[0]["ms"] / r["ms"], 3)
                    r["ideal_speedup"] = round(16.0 / max(r["n_full"], 1), 3)

    ff = flops_full(head["N"], head["n_full"])
    achieved = ff / head["full_kernel_ms"] / 1e9
    out = {
        "metric": METRIC,
        "value": head["ms"],
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms"],
        "higher_is_better": False,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded iid N(0,1/64) Q/K/V, seeded router and surrogate weights)",
        "config": {"workload": "S=100 views x 1374 tokens (N=137400), 16 heads x 64, bf16 "
                               "operands, fp32 accumulate, bf16 Y, %d of 16 heads FULL"
                               % head["n_full"],
                   "S": 100, "P": P_TOKENS, "N": head["N"], "heads": HEADS, "head_dim": D,
                   "n_full": head["n_full"], "n_surr": head["n_surr"], "n_mean": head["n_mean"],
                   "layout": "Q/K/V [S*P, 16, 64] row-major"},
        "tflops": head["tflops"],
        "frac_bf16_peak": head["frac_peak"],
        "roofline": {"kernel": "k_flash_bf16", "bound": "mfma", "achieved": round(achieved, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": flash_traffic(100, head["n_full"]),
                     "contraction": "fp16 MFMA 32x32x16 (bf16 Q, K converted to fp16; P and "
                                    "the per-head power-of-two-scaled V in fp16), fp32 "
                                    "accumulate; the fp16 and bf16 dense MFMA peaks are equal",
                     "algorithmic_flop_per_launch": ff,
                     "avg_launch_ms": round(head["full_kernel_ms"], 4)},
        "hbm": {"router_gbs": head["hbm_gbs"].get("router"),
                "gather_gbs": head["hbm_gbs"].get("gather"),
                "linear_heads_gbs": head["hbm_gbs"].get("linear"),
                "peak_gbs": PEAK_HBM_GBS,
                "note": "algorithmic bytes / HIP-event stage time: router = vp_router_score "
                        "(Q, K, V read once), gather = vp_gather_full_heads (K, V read, fp16 K "
                        "and V^T written per FULL head), linear = vp_linear_heads"},
        "by_workload": by,
    }
    if variants is not None:
        out["variants"] = variants
    if block is not None:
        out["block"] = block
    if tome is not None:
        out["tome"] = tome
    if teacher is not None:
        out["teacher"] = teacher
    if stack500 is not None:
        out["layer_stack_s500"] = stack500
    if stack is not None:
        out["stack"] = stack
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(x)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
