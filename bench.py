#!/usr/bin/env python3
"""Benchmark of the DPara drafter hot path on one MI355X.

One step = one steady-state round for the whole batch, all in libdpara's HIP kernels:
    dpara_ctx_append (r+1 new feature rows per request, incremental projection)
    -> dpara_backbone_all_boundaries (all gamma+1 boundaries, tree mask)
    -> dpara_verify_greedy (planted target logits)
    -> dpara_select_and_head (gather branch r, LM head, gamma-step AR head)
Inputs are resident in HBM before the timed region.  Before each append the
context length is rewound by the append size, so every round runs at the
workload's context length (a steady state at fixed context).

Prints one JSON line.  Besides the metric's own configuration (Qwen3-8B-shaped drafter,
batch 1, context 2048) the default run also measures, on the same clock: the batch-16 and
14B batch-8 configurations (`other_configs`), the single-GPU full round with the 36-layer
target at batch 1 and 16 (`full_round`: verification, backbone, both concurrent, the serial
step, the overlapped round eager and as one graph), the head per batch size with the
verification it must hide in (`serial_head_share`), and the CPU oracle on a bounded sample of
the same unit of work (`cpu_baseline`).  `--gpus N` with N > 1 exits: the path runs on one GPU
(requests would shard independently across GPUs).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "all-boundary backbone rounds/sec + head µs/round at b=1..16; % HBM/MFMA peak"
PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
PEAK_F32_TFLOPS = 157.3
COPY_PROBE_BYTES = 256 << 20
GATEUP_KERNEL_SMALL_M = "gemm_adir_kernel<2, 4, 0>"  # the gate/up SwiGLU GEMM at <= 320 rows


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def gateup_work(shape, M):
    """Algorithmic bytes and flops of one gate/up SwiGLU GEMM launch over M rows."""
    esz = 2 if shape.dtype == "bf16" else 4
    H, F = shape.hidden, shape.ffn
    bytes_ = 2 * F * H * esz + M * H * esz + M * F * esz
    flops = 2.0 * M * (2 * F) * H
    return bytes_, flops


def backbone_work(shape, B, ctx_lens):
    """Algorithmic bytes (weights + context K/V read + reps written) and flops of one backbone call."""
    esz = 2 if shape.dtype == "bf16" else 4
    H, F, nq, nkv, hd, L, g = (shape.hidden, shape.ffn, shape.n_q_heads, shape.n_kv_heads, shape.head_dim,
                               shape.n_layers, shape.gamma)
    R = (g + 1) ** 2
    M = B * R
    per_layer_w = (nq + 2 * nkv) * hd * H + nq * hd * H + 3 * F * H
    wbytes = L * per_layer_w * esz
    kv_bytes = L * sum(int(n) for n in ctx_lens) * 2 * nkv * hd * esz
    reps_bytes = B * (g + 1) * g * H * 4
    dense = 2.0 * M * per_layer_w * L
    return wbytes + kv_bytes + reps_bytes, dense + attention_flops(shape, ctx_lens)


def attention_flops(shape, ctx_lens):
    """Algorithmic flops of the backbone's attention (all layers): QK^T and PV over the keys
    each row sees under the tree mask (the whole context plus its visible in-block keys)."""
    nq, hd, L, g = shape.n_q_heads, shape.head_dim, shape.n_layers, shape.gamma
    R = (g + 1) ** 2
    vis_in_block = (g + 1) * (g + 2) // 2 + sum(g * (r + 1 + g) for r in range(g + 1))
    return sum(4.0 * nq * hd * (R * int(n) + vis_in_block) * L for n in ctx_lens)


def host_cores():
    """(threads this process may run on, CPU model name) of the host."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return n, model


def cpu_baseline(wl, weights, ri, min_seconds=10.0, max_rounds=8):
    """The CPU oracle on a bounded sample of the same unit of work as one GPU step, for request 0:
    the context's K/V are projected once beforehand (the GPU keeps them in its cache too), then
    each timed round appends the K/V of the r+1 new rows at their positions, runs every layer over
    the (gamma+1)^2 tree rows, the final norm, greedy verify and select + AR head, with the
    oracle's own functions in float64.  Rounds repeat for about min_seconds (at most max_rounds);
    the time per round is scaled by the batch (requests are independent)."""
    import numpy as np
    from oracle import dpara_oracle as O
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas = None
    n_aff, model = host_cores()
    s = wl.shape
    mode = "bf16" if s.dtype == "bf16" else "f32"
    rnd = O.Rounding(mode)
    g, R = s.gamma, s.rows
    r = int(ri.accept_planted[0])
    n_b = int(ri.ctx_lens[0])
    base = n_b - (r + 1)
    feats, new = ri.ctx_feats[0][:base], ri.new_feats[0][:r + 1]
    ck = [O.context_kv(s, weights, l, feats, 0, rnd) for l in range(s.n_layers)]
    vis, pos = O.tree_visibility(g), O.row_positions(g, n_b)
    x0 = np.empty((R, s.hidden), np.float64)
    for j in range(g + 1):
        x0[j] = weights["embed"][int(ri.spine[0, j])]
    x0[g + 1:] = weights["mask_emb"][None, :]
    n, t = 0, time.perf_counter()
    while n < max_rounds and (n == 0 or time.perf_counter() - t < min_seconds):
        x = rnd.r32(x0)
        for l in range(s.n_layers):
            kn, vn = O.context_kv(s, weights, l, new, base, rnd)
            x = O.layer_forward(s, weights, l, x, pos, np.concatenate([ck[l][0], kn]),
                                np.concatenate([ck[l][1], vn]), vis, rnd)
        reps = rnd.r32(O.rmsnorm(x[g + 1:], weights["final_norm"], s.rms_eps)).reshape(g + 1, g, s.hidden)
        rr, bonus, _ = O.verify_greedy(ri.target_logits[0], ri.spine[0])
        O.select_and_head(s, weights, reps, rr, bonus, mode)
        n += 1
    dt = time.perf_counter() - t
    per_round = dt / n * wl.batch
    return {"value": 1.0 / per_round, "unit": "rounds/s", "cores": n_aff, "blas_threads": blas,
            "cpu_model": model, "kind": "oracle",
            "unit_of_work": (f"one round as the GPU step runs it: K/V of the {r + 1} appended rows, "
                             f"{s.n_layers} layers over the {R} tree rows at context {n_b}, final norm, greedy "
                             f"verify, select + AR head over vocabulary {s.vocab}"),
            "sample": (f"{n} rounds of request 0 in {dt:.1f} s (context K/V of {base} cached positions "
                       f"projected once beforehand, untimed)"
                       + (f"; scaled x{wl.batch} to the batch" if wl.batch > 1 else ""))}


def full_round(wl, steps, warmup, drafter=None):
    """Single-GPU full round: the target's verification forward and the drafter's append +
    all-boundary backbone on two streams, joined by an event, then greedy verify on the
    target logits and select + AR head (Algorithm 1 with the colocated placement), eager and
    captured as one HIP graph (fork onto the two streams and join inside the capture).
    Returns the overlap figures (ms)."""
    import numpy as np
    import torch
    from paper_2609_27396_amd import dpara as D
    from paper_2609_27396_amd import synth
    from paper_2609_27396_amd.harness import DeviceRound

    shape, B = wl.shape, wl.batch
    tshape = synth.QWEN3_8B_TARGET
    t0 = time.time()
    weights = None if drafter is not None else synth.make_weights(shape, seed=wl.seed_w)
    ri = synth.make_round(wl)
    dr = DeviceRound(shape, weights, ri, drafter=drafter)
    prepare_head(dr)
    cap = dr.ctx_cap
    tgt = D.DeviceTarget(tshape, None, seed=100)
    tctx = D.DeviceContext(tshape, B, cap)
    synth.device_normal_(tctx.k, 201)
    synth.device_normal_(tctx.v, 202)
    tctx.ctx_len[:B] = torch.from_numpy(ri.ctx_lens.astype(np.int32)).cuda()
    tws = D.Workspace(tgt.cfg, B, cap, target=True)
    logits = torch.empty((B, shape.gamma + 1, shape.vocab), dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    log(f"[bench] full round b={B} set up in {time.time() - t0:.1f} s (target {tshape.n_layers} layers on device)")

    n_new_h = ri.accept_planted.astype(np.int32) + 1
    n_new = torch.from_numpy(n_new_h).cuda()
    base_len = torch.from_numpy((ri.ctx_lens - n_new_h).astype(np.int32)).cuda()
    s_draft, s_ver = torch.cuda.Stream(), torch.cuda.Stream()

    def draft(st):
        with torch.cuda.stream(st):
            dr.ctx.ctx_len[:B].copy_(base_len)
            dr.append(n_new, stream=st)
            dr.backbone(stream=st)

    def verify_pass(st):
        with torch.cuda.stream(st):
            D.target_forward(tgt, tctx, dr.spine, logits, tws, stream=st)

    def serial(st):
        with torch.cuda.stream(st):
            D.verify_greedy(dr.d, logits, dr.spine, dr.accept, dr.bonus, dr.targmax, dr.ws, stream=st)
            dr.head(stream=st)

    def round_(overlap=True):
        cur = torch.cuda.current_stream()
        s_draft.wait_stream(cur)
        s_ver.wait_stream(cur)
        draft(s_draft)
        if not overlap:
            s_ver.wait_stream(s_draft)
        verify_pass(s_ver)
        s_ver.wait_stream(s_draft)  # barrier: (r, b) and all branches ready
        serial(s_ver)
        cur.wait_stream(s_ver)

    def timed(fn, k):
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(k):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / k

    def only(fn, st):
        def go():
            st.wait_stream(torch.cuda.current_stream())
            fn(st)
            torch.cuda.current_stream().wait_stream(st)
        return go

    def both():
        cur = torch.cuda.current_stream()
        s_draft.wait_stream(cur)
        s_ver.wait_stream(cur)
        draft(s_draft)
        verify_pass(s_ver)
        cur.wait_stream(s_draft)
        cur.wait_stream(s_ver)

    for _ in range(warmup):
        round_()
    K = steps
    t_v = timed(only(verify_pass, s_ver), K)
    t_bb = timed(only(draft, s_draft), K)
    t_serial = timed(only(serial, s_ver), K)
    t_both = timed(both, K)
    t_seq = timed(lambda: round_(overlap=False), K)
    ms = timed(round_, K)
    # the whole round as one graph: fork onto the two streams and join inside the capture
    graph = torch.cuda.CUDAGraph()
    cs = torch.cuda.Stream()
    cs.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cs):
        with torch.cuda.graph(graph, stream=cs):
            round_()
    torch.cuda.synchronize()
    for _ in range(warmup):
        graph.replay()
    graph_ms = timed(graph.replay, K)
    assert dr.status() == 0, f"device status {dr.status()}"
    out = {"batch": B, "ctx": int(ri.ctx_lens[0]), "target_layers": tshape.n_layers,
           "target_verify_ms": t_v, "append_backbone_ms": t_bb, "both_concurrent_ms": t_both,
           "serial_verify_head_ms": t_serial, "round_overlapped_ms": ms, "round_sequential_ms": t_seq,
           "round_graph_ms": graph_ms, "backbone_hidden_fraction": (t_v + t_bb - t_both) / t_bb,
           "paper_model_ms": max(t_v, t_bb) + t_serial, "serial_share_of_verify": t_serial / t_v}
    del graph, dr, tgt, tctx, tws, logits
    torch.cuda.empty_cache()
    return out


def target_verify_sweep(batches, steps, warmup, ctx=2048):
    """The verification forward alone (the 36-layer Qwen3-8B-shaped random target, gamma+1 = 17
    tokens per request at context `ctx`) at each batch size: the denominator of the serial head's
    share of a round.  Milliseconds per call."""
    import torch
    from paper_2609_27396_amd import dpara as D
    from paper_2609_27396_amd import synth
    ts = synth.QWEN3_8B_TARGET
    bmax = max(batches)
    cap = (ctx + 2 * (ts.gamma + 1) + 63) // 64 * 64
    tgt = D.DeviceTarget(ts, None, seed=100)
    tctx = D.DeviceContext(ts, bmax, cap)
    synth.device_normal_(tctx.k, 201)
    synth.device_normal_(tctx.v, 202)
    tctx.ctx_len.fill_(ctx)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(7)
    out = {}
    for B in batches:
        tws = D.Workspace(tgt.cfg, B, cap, target=True)
        block = torch.randint(0, ts.vocab, (B, ts.gamma + 1), generator=gen, device="cuda", dtype=torch.int32)
        logits = torch.empty((B, ts.gamma + 1, ts.vocab), dtype=torch.bfloat16, device="cuda")
        for _ in range(warmup):
            D.target_forward(tgt, tctx, block, logits, tws)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            D.target_forward(tgt, tctx, block, logits, tws)
        e1.record()
        torch.cuda.synchronize()
        out[str(B)] = e0.elapsed_time(e1) / steps
        del tws, logits
    del tgt, tctx
    torch.cuda.empty_cache()
    return out


def recorded_traffic(kernel: str):
    """HBM bytes per launch of `kernel` from the committed counter summary (two rocprofv3 --pmc
    passes, FETCH_SIZE and WRITE_SIZE, scaled on a plain copy of known size), or None when the
    summary is missing or the kernel's source changed since the counters were taken."""
    import hashlib
    here = os.path.dirname(os.path.abspath(__file__))
    try:
        with open(os.path.join(here, "profiles", "traffic_qwen3_8b_b1.md")) as f:
            line = next(l for l in f if l.startswith("traffic-json: "))
        rec = json.loads(line[len("traffic-json: "):])
        with open(os.path.join(here, rec["source"]), "rb") as f:
            digest = hashlib.sha256(f.read()).hexdigest()
    except (OSError, StopIteration, ValueError, KeyError):
        return None
    if rec.get("kernel") != kernel or rec.get("source_sha256") != digest:
        return None
    return float(rec["bytes_per_launch"])


def prepare_head(dr):
    """Weight preparation at load time (outside every timed region): the AR head's max row
    norm and the embedding's max row norm, constants of the weights that the bound-pruned head
    steps and the hi-plane candidate ranking use."""
    if dr.shape.ar_rank in (64, 128, 256):
        dr.d.prepare_head(dr.ws)
        if dr.shape.dtype == "bf16":
            dr.d.prepare_candidates(dr.ws)


def fuse_timing(shape, rows=(17, 2048), n_feat=3, iters=20):
    """Feature fusion (the step before the cache update) alone: f = RMSNorm(fc [h_1; h_2;
    h_3]) * g for a round's rows at b=1 and for a 2048-row prefill, on device-generated
    weights and hidden states (microseconds per call, and the call's weight + row bytes
    over its time)."""
    import torch
    from paper_2609_27396_amd import dpara as D, synth
    fus = D.DeviceFusion(shape, None, n_feat)
    H = shape.hidden
    out = {}
    for n in rows:
        hid = synth.device_normal_(torch.empty((n, n_feat * H), dtype=torch.bfloat16, device="cuda"), 13 + n)
        f = torch.empty((n, H), dtype=torch.bfloat16, device="cuda")
        ws = torch.empty(D.dpara_fuse_workspace_bytes(fus.cfg, n, n_feat), dtype=torch.uint8, device="cuda")
        for _ in range(3):
            D.fuse_features(fus, hid, f, ws)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            D.fuse_features(fus, hid, f, ws)
        e1.record()
        torch.cuda.synchronize()
        us = 1000.0 * e0.elapsed_time(e1) / iters
        nbytes = H * n_feat * H * 2 + n * n_feat * H * 2 + n * H * 2
        out[str(n)] = {"us": us, "GB_s": nbytes / us / 1e3}
    return out


def head_sweep(dr, shape, batches=(1, 2, 4, 8, 16), iters=20):
    """Select + AR head alone at several batch sizes, on synthetic branch representations
    (microseconds per call): the plain call (gather, LM head over gamma rows, gamma AR
    steps), the off-serial-path variant: the branch-candidates call (every branch row's
    LM head with top-2 tiles, timed on its own) and the serial call that uses them, and the
    sampling variant: the sampled head and the speculative-sampling verification."""
    import torch
    from paper_2609_27396_amd import dpara as D
    g, H, V = shape.gamma, shape.hidden, shape.vocab
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1234)
    out = {"plain_us": {}, "plain_fallback": {}, "candidates_us": {}, "cand_serial_us": {}, "cand_fallback": {},
           "sampled_head_us": {}, "sampled_verify_us": {}}

    def timed(call):
        for _ in range(3):
            call()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            call()
        e1.record()
        torch.cuda.synchronize()
        return 1000.0 * e0.elapsed_time(e1) / iters

    for B in batches:
        ws = D.Workspace(dr.d.cfg, B, 64)
        reps = torch.randn((B, g + 1, g, H), generator=gen, device="cuda", dtype=torch.float32)
        acc = torch.randint(0, g + 1, (B,), generator=gen, device="cuda", dtype=torch.int32)
        bon = torch.randint(0, V, (B,), generator=gen, device="cuda", dtype=torch.int32)
        drafts = torch.empty((B, g), dtype=torch.int32, device="cuda")
        nspine = torch.empty((B, g + 1), dtype=torch.int32, device="cuda")
        k = str(B)
        out["plain_us"][k] = timed(lambda: D.select_and_head(dr.d, reps, acc, bon, None, drafts, nspine, None, ws))
        out["plain_fallback"][k] = ws.head_fallback()
        cand = D.branch_candidates_buffer(dr.d, B)
        out["candidates_us"][k] = timed(lambda: D.branch_candidates(dr.d, reps, cand, ws))
        out["cand_serial_us"][k] = timed(
            lambda: D.select_and_head_cand(dr.d, reps, cand, acc, bon, None, drafts, nspine, None, ws))
        out["cand_fallback"][k] = ws.head_fallback()
        # sampling variant: the sampled head (full head with Gumbel noise, draft scores out)
        # and the speculative-sampling verification of a block
        scores = torch.randn((B, g, V), generator=gen, device="cuda", dtype=torch.float32)
        out["sampled_head_us"][k] = timed(lambda: D.select_and_head_sampled(
            dr.d, reps, acc, bon, None, drafts, nspine, None, 1.0, 77, scores, ws))
        tl = torch.randn((B, g + 1, V), generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
        out["sampled_verify_us"][k] = timed(lambda: D.verify_sampled(dr.d, tl, scores, nspine, 1.0, 78, acc, bon, ws))
        assert ws.status() == 0, f"device status {ws.status()}"
        del ws, reps, cand, scores, tl
    return out


def step_bench(wl, dr, ri, steps, warmup, graph=True, prof_steps=5):
    """Time the steady-state step (rewind, append, backbone, verify, select + head) of a prepared
    DeviceRound: eager, as HIP graph replays, and per phase (the library's HIP events on the
    launching stream).  Returns the figures of one configuration."""
    import numpy as np
    import torch
    from paper_2609_27396_amd import dpara as D

    shape, B = wl.shape, wl.batch
    n_new_h = (ri.accept_planted.astype(np.int32) + 1)
    n_new = torch.from_numpy(n_new_h).cuda()
    base_len = torch.from_numpy((ri.ctx_lens - n_new_h).astype(np.int32)).cuda()

    def step():
        dr.ctx.ctx_len[:B].copy_(base_len)
        dr.append(n_new)
        dr.backbone()
        dr.verify()
        dr.head()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    assert dr.status() == 0, f"device status {dr.status()}"
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    log(f"[bench] {wl.name}: {steps} steps: {ms:.3f} ms/step")

    # the same step captured into a HIP graph and replayed (same kernels, same work)
    graph_ms = None
    if graph:
        g = torch.cuda.CUDAGraph()
        cs = torch.cuda.Stream()
        cs.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cs):
            with torch.cuda.graph(g, stream=cs):
                step()
        torch.cuda.synchronize()
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        ev0.record()
        for _ in range(steps):
            g.replay()
        ev1.record()
        torch.cuda.synchronize()
        graph_ms = ev0.elapsed_time(ev1) / steps
        assert dr.status() == 0, f"device status {dr.status()}"
        del g

    D.dpara_profile_enable(True)
    for _ in range(prof_steps):
        step()
    torch.cuda.synchronize()
    phases = {}
    for ph in D.PHASES:
        tot, n = D.dpara_profile_read(ph)
        if n:
            phases[ph] = {"ms_per_step": tot / prof_steps, "launches_per_step": n / prof_steps,
                          "avg_us": 1000.0 * tot / n}
    D.dpara_profile_enable(False)
    sum_ms = lambda names: sum(phases.get(p, {}).get("ms_per_step", 0.0) for p in names)
    backbone_ms = sum_ms(["assemble", "rmsnorm", "qkv_gemm", "qk_norm_rope", "attn_ctx", "attn_merge", "o_gemm",
                          "gateup_gemm", "down_gemm", "final_norm"])

    # roofline of the dominant kernel: the gate/up SwiGLU GEMM
    M = B * shape.rows
    gb, gf = gateup_work(shape, M)
    g_avg_s = phases["gateup_gemm"]["avg_us"] * 1e-6
    peak_flops = PEAK_BF16_TFLOPS if shape.dtype == "bf16" else PEAK_F32_TFLOPS
    if gb / (PEAK_HBM_GBS * 1e9) >= gf / (peak_flops * 1e12):
        roof = {"bound": "hbm", "achieved": gb / g_avg_s / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    else:
        roof = {"bound": "mfma", "achieved": gf / g_avg_s / 1e12, "peak": peak_flops, "unit": "TFLOP/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["kernel"] = GATEUP_KERNEL_SMALL_M if M <= 320 else "gemm_pipe_kernel (gate/up SwiGLU)"
    roof["traffic"] = recorded_traffic(roof["kernel"]) if wl.name == "qwen3_8b_b1" else None
    roof["algorithmic_bytes_per_launch"] = gb
    roof["algorithmic_flops_per_launch"] = gf
    roof["avg_launch_us"] = g_avg_s * 1e6

    bb_bytes, bb_flops = backbone_work(shape, B, ri.ctx_lens)
    bb_s = backbone_ms * 1e-3
    return {
        "ms_per_step": ms, "rounds_per_s": 1000.0 / ms, "graph_ms_per_step": graph_ms,
        "roofline": roof,
        "backbone": {"ms": backbone_ms, "rounds_per_s": 1000.0 / backbone_ms, "algorithmic_GB": bb_bytes / 1e9,
                     "GFLOP": bb_flops / 1e9, "GB_s": bb_bytes / bb_s / 1e9, "TFLOP_s": bb_flops / bb_s / 1e12,
                     "hbm_frac": bb_bytes / bb_s / 1e9 / PEAK_HBM_GBS,
                     "mfma_frac": bb_flops / bb_s / 1e12 / peak_flops},
        # attention (MFMA pass + fold) against the bf16 peak, counting each useful product once
        "attention": {"us_per_layer": 1000.0 * sum_ms(["attn_ctx", "attn_merge"]) / shape.n_layers,
                      "TFLOP_s": attention_flops(shape, ri.ctx_lens) / (sum_ms(["attn_ctx", "attn_merge"]) * 1e-3) / 1e12,
                      "mfma_frac": attention_flops(shape, ri.ctx_lens) / (sum_ms(["attn_ctx", "attn_merge"]) * 1e-3)
                      / 1e12 / peak_flops},
        "head_us_per_round": 1000.0 * sum_ms(["gather", "lm_head", "ar_step"]),
        "head_full_fallback": dr.head_fallback(),
        "verify_us_per_round": 1000.0 * sum_ms(["verify"]),
        "append_us_per_round": 1000.0 * sum_ms(["append_gemm", "append_store"]),
        "phases": phases,
    }


def workload_config(wl, ri):
    s = wl.shape
    return {"workload": wl.name, "batch": wl.batch, "gamma": s.gamma,
            "ctx": int(ri.ctx_lens[0]) if wl.ctx_min == wl.ctx_max else [wl.ctx_min, wl.ctx_max],
            "layers": s.n_layers, "hidden": s.hidden, "heads": [s.n_q_heads, s.n_kv_heads],
            "head_dim": s.head_dim, "ffn": s.ffn, "vocab": s.vocab, "ar_rank": s.ar_rank,
            "rows_per_request": s.rows}


def other_config(name, steps, warmup, drafter=None):
    """Step figures of another configuration (batch 16 at ragged contexts, the 14B shape at batch
    8), on its own seeded inputs; the drafter weights are reused when the shape and seed match."""
    import torch
    from paper_2609_27396_amd import synth
    from paper_2609_27396_amd.harness import DeviceRound
    wl = synth.WORKLOADS[name]
    t0 = time.time()
    weights = None if drafter is not None else synth.make_weights(wl.shape, seed=wl.seed_w)
    ri = synth.make_round(wl)
    dr = DeviceRound(wl.shape, weights, ri, drafter=drafter)
    prepare_head(dr)
    torch.cuda.synchronize()
    log(f"[bench] {name} set up in {time.time() - t0:.1f} s")
    res = step_bench(wl, dr, ri, steps, warmup)
    res["config"] = workload_config(wl, ri)
    del dr, weights
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="qwen3_8b_b1")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-head-sweep", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the other configurations (batch 16, 14B batch 8) and the full rounds")
    ap.add_argument("--head-sweep-batches", default="1,2,4,8,16",
                    help="comma-separated batch sizes of the head sweep")
    ap.add_argument("--no-graph", action="store_true", help="skip timing the step as HIP graph replays")
    ap.add_argument("--copy-probe", action="store_true",
                    help="first run a plain 256 MiB device copy 3 times (known HBM bytes, to scale "
                         "profiler traffic counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); requests are independent, so several "
              f"GPUs would each run this path on their own share of the batch.", file=sys.stderr)
        sys.exit(2)

    import dataclasses

    import torch
    from paper_2609_27396_amd import synth
    from paper_2609_27396_amd.harness import DeviceRound

    wl = synth.WORKLOADS[args.workload]
    shape = wl.shape
    log(f"[bench] workload {wl.name}: {wl.description}")
    if args.copy_probe:
        src = torch.ones(COPY_PROBE_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if wl.name == "full_round":
        res = full_round(wl, args.steps, args.warmup)
        out = {"metric": METRIC, "value": 1000.0 / res["round_overlapped_ms"], "unit": "rounds/s", "n_gpus": 1,
               "steps": args.steps, "warmup": args.warmup, "ms_per_step": res["round_overlapped_ms"],
               "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
               "data": "synthetic", "config": {"workload": wl.name, "batch": wl.batch, "gamma": shape.gamma},
               "overlap": res}
        print(json.dumps(out), flush=True)
        return
    t0 = time.time()
    weights = synth.make_weights(shape, seed=wl.seed_w)
    ri = synth.make_round(wl)
    log(f"[bench] inputs generated in {time.time() - t0:.1f} s")
    dr = DeviceRound(shape, weights, ri)
    prepare_head(dr)
    torch.cuda.synchronize()
    log(f"[bench] weights resident, context prefilled ({time.time() - t0:.1f} s)")

    res = step_bench(wl, dr, ri, args.steps, args.warmup, graph=not args.no_graph)
    out = {
        "metric": METRIC, "value": res["rounds_per_s"], "unit": "rounds/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": res["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": shape.dtype, "data": "synthetic",
        "config": workload_config(wl, ri),
    }
    out.update({k: v for k, v in res.items() if k not in ("ms_per_step", "rounds_per_s")})
    if shape.dtype == "bf16" and not args.no_head_sweep:
        hs = head_sweep(dr, shape, batches=tuple(int(x) for x in args.head_sweep_batches.split(",")))
        out["head_us_by_batch"] = hs.pop("plain_us")
        out["head_variants_by_batch"] = hs
        out["fuse_by_rows"] = fuse_timing(shape)
    if not args.no_extra and wl.name == "qwen3_8b_b1":
        # the other configurations of the metric and the single-GPU full rounds, on this run's clock
        k, w = min(args.steps, 10), min(args.warmup, 3)
        out["other_configs"] = {
            "qwen3_8b_b16": other_config("qwen3_8b_b16", k, w, drafter=dr.d),
            "qwen3_14b_b8": other_config("qwen3_14b_b8", k, w),
        }
        fr = synth.WORKLOADS["full_round"]
        out["full_round"] = {
            "b1": full_round(dataclasses.replace(fr, name="full_round_b1", batch=1), k, w, drafter=dr.d),
            "b16": full_round(fr, k, w, drafter=dr.d),
        }
        if "head_us_by_batch" in out:
            tv = target_verify_sweep([int(b) for b in out["head_us_by_batch"]], k, w)
            hv = out["head_variants_by_batch"]
            out["serial_head_share"] = {
                "target_verify_ms": tv,
                "plain_head": {b: out["head_us_by_batch"][b] / 1000.0 / tv[b] for b in tv},
                "candidates_head": {b: hv["cand_serial_us"][b] / 1000.0 / tv[b] for b in tv},
                "candidates_off_path_fits": {b: hv["candidates_us"][b] / 1000.0 <= tv[b] for b in tv},
            }
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample ...")
        out["cpu_baseline"] = cpu_baseline(wl, weights, ri)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
