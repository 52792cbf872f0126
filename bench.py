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

Prints one JSON line (see the fields below).  `--gpus N` with N > 1 exits: the
path runs on one GPU (requests would shard independently across GPUs).
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
    vis_in_block = (g + 1) * (g + 2) // 2 + sum(g * (r + 1 + g) for r in range(g + 1))
    attn = 0.0
    for n in ctx_lens:
        attn += 4.0 * nq * hd * (R * int(n) + vis_in_block) * L
    return wbytes + kv_bytes + reps_bytes, dense + attn


def cpu_baseline(wl, weights, ri, min_seconds=10.0, max_rounds=8):
    """The CPU oracle (as it stands) on a bounded sample: full rounds of request 0, repeated
    until about min_seconds of CPU work (at most max_rounds), the mean time per round."""
    from oracle import dpara_oracle as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = os.cpu_count() or 1
    mode = "bf16" if wl.shape.dtype == "bf16" else "f32"
    n, t = 0, time.perf_counter()
    while n < max_rounds and (n == 0 or time.perf_counter() - t < min_seconds):
        O.dpara_round(wl.shape, weights, ri.ctx_feats[0], ri.spine[0], ri.target_logits[0], mode)
        n += 1
    dt = time.perf_counter() - t
    per_round = dt / n * wl.batch  # a batch round = B requests; scaled linearly from request 0
    return {"value": 1.0 / per_round, "unit": "rounds/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"{n} full rounds (context K/V projection of {int(ri.ctx_lens[0])} positions, all-boundary "
                       f"backbone, greedy verify, select + AR head) of request 0, {dt:.1f} s"
                       + (f", scaled x{wl.batch} to the batch" if wl.batch > 1 else ""))}


def full_round(args, wl):
    """Single-GPU full round: the target's verification forward and the drafter's append +
    all-boundary backbone on two streams, joined by an event, then greedy verify on the
    target logits and select + AR head (Algorithm 1 with the colocated placement)."""
    import numpy as np
    import torch
    from paper_2609_27396_amd import dpara as D
    from paper_2609_27396_amd import synth
    from paper_2609_27396_amd.harness import DeviceRound

    shape, B = wl.shape, wl.batch
    tshape = synth.QWEN3_8B_TARGET
    t0 = time.time()
    weights = synth.make_weights(shape, seed=wl.seed_w)
    ri = synth.make_round(wl)
    dr = DeviceRound(shape, weights, ri)
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
    log(f"[bench] full round set up in {time.time() - t0:.1f} s (target {tshape.n_layers} layers on device)")

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
        start = torch.cuda.Event()
        start.record(torch.cuda.current_stream())
        s_draft.wait_event(start)
        s_ver.wait_event(start)
        draft(s_draft)
        if not overlap:
            s_ver.wait_stream(s_draft)
        verify_pass(s_ver)
        s_ver.wait_stream(s_draft)  # barrier: (r, b) and all branches ready
        serial(s_ver)
        torch.cuda.current_stream().wait_stream(s_ver)

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
        start = torch.cuda.Event()
        start.record(torch.cuda.current_stream())
        s_draft.wait_event(start)
        s_ver.wait_event(start)
        draft(s_draft)
        verify_pass(s_ver)
        torch.cuda.current_stream().wait_stream(s_draft)
        torch.cuda.current_stream().wait_stream(s_ver)

    for _ in range(args.warmup):
        round_()
    K = args.steps
    t_v = timed(only(verify_pass, s_ver), K)
    t_bb = timed(only(draft, s_draft), K)
    t_serial = timed(only(serial, s_ver), K)
    t_both = timed(both, K)
    t_seq = timed(lambda: round_(overlap=False), K)
    ms = timed(round_, K)
    assert dr.status() == 0
    hidden = (t_v + t_bb - t_both) / t_bb
    out = {
        "metric": METRIC, "value": 1000.0 / ms, "unit": "rounds/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.name, "batch": B, "gamma": shape.gamma, "ctx": int(ri.ctx_lens[0]),
                   "drafter_layers": shape.n_layers, "target_layers": tshape.n_layers, "hidden": shape.hidden,
                   "vocab": shape.vocab},
        "overlap": {"target_verify_ms": t_v, "append_backbone_ms": t_bb, "both_concurrent_ms": t_both,
                    "serial_verify_head_ms": t_serial, "round_overlapped_ms": ms, "round_sequential_ms": t_seq,
                    "backbone_hidden_fraction": hidden,
                    "paper_model_ms": max(t_v, t_bb) + t_serial,
                    "serial_share_of_verify": t_serial / t_v},
    }
    print(json.dumps(out), flush=True)


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
    norm, a constant of the weights that the bound-pruned head steps use."""
    if dr.shape.ar_rank in (64, 128, 256):
        dr.d.prepare_head(dr.ws)


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


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="qwen3_8b_b1")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-head-sweep", action="store_true")
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

    import numpy as np
    import torch
    from paper_2609_27396_amd import dpara as D
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
        full_round(args, wl)
        return
    t0 = time.time()
    weights = synth.make_weights(shape, seed=wl.seed_w)
    ri = synth.make_round(wl)
    log(f"[bench] inputs generated in {time.time() - t0:.1f} s")
    dr = DeviceRound(shape, weights, ri)
    prepare_head(dr)
    torch.cuda.synchronize()
    log(f"[bench] weights resident, context prefilled ({time.time() - t0:.1f} s)")

    B = wl.batch
    n_new_h = (ri.accept_planted.astype(np.int32) + 1)
    n_new = torch.from_numpy(n_new_h).cuda()
    base_len = torch.from_numpy((ri.ctx_lens - n_new_h).astype(np.int32)).cuda()

    def step():
        dr.ctx.ctx_len[:B].copy_(base_len)
        dr.append(n_new)
        dr.backbone()
        dr.verify()
        dr.head()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    assert dr.status() == 0, f"device status {dr.status()}"
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(args.steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / args.steps
    log(f"[bench] {args.steps} steps: {ms:.3f} ms/step")

    # the same step captured into a HIP graph and replayed K times (same kernels, same work)
    graph_ms = None
    if not args.no_graph:
        g = torch.cuda.CUDAGraph()
        cs = torch.cuda.Stream()
        cs.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cs):
            with torch.cuda.graph(g, stream=cs):
                step()
        torch.cuda.synchronize()
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        ev0.record()
        for _ in range(args.steps):
            g.replay()
        ev1.record()
        torch.cuda.synchronize()
        graph_ms = ev0.elapsed_time(ev1) / args.steps
        assert dr.status() == 0, f"device status {dr.status()}"
        log(f"[bench] {args.steps} graph replays: {graph_ms:.3f} ms/step")

    # per-phase durations (HIP events recorded by the library on the launching stream)
    prof_steps = 5
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
    head_us = 1000.0 * sum_ms(["gather", "lm_head", "ar_step"])

    # roofline of the dominant kernel: the gate/up SwiGLU GEMM
    M = B * shape.rows
    gb, gf = gateup_work(shape, M)
    g_avg_s = phases["gateup_gemm"]["avg_us"] * 1e-6
    peak_flops = PEAK_BF16_TFLOPS if shape.dtype == "bf16" else PEAK_F32_TFLOPS
    hbm_bound = gb / (PEAK_HBM_GBS * 1e9) >= gf / (peak_flops * 1e12)
    if hbm_bound:
        roof = {"bound": "hbm", "achieved": gb / g_avg_s / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    else:
        roof = {"bound": "mfma", "achieved": gf / g_avg_s / 1e12, "peak": peak_flops, "unit": "TFLOP/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["kernel"] = "gemm_adir_kernel<2, 4>" if M <= 320 else "gemm_pipe_kernel (gate/up SwiGLU)"
    roof["traffic"] = recorded_traffic(roof["kernel"]) if wl.name == "qwen3_8b_b1" else None
    roof["algorithmic_bytes_per_launch"] = gb
    roof["algorithmic_flops_per_launch"] = gf
    roof["avg_launch_us"] = g_avg_s * 1e6

    bb_bytes, bb_flops = backbone_work(shape, B, ri.ctx_lens)
    bb_s = backbone_ms * 1e-3
    out = {
        "metric": METRIC, "value": 1000.0 / ms, "unit": "rounds/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": shape.dtype, "data": "synthetic",
        "config": {"workload": wl.name, "batch": B, "gamma": shape.gamma,
                   "ctx": int(ri.ctx_lens[0]) if wl.ctx_min == wl.ctx_max else [wl.ctx_min, wl.ctx_max],
                   "layers": shape.n_layers, "hidden": shape.hidden, "heads": [shape.n_q_heads, shape.n_kv_heads],
                   "head_dim": shape.head_dim, "ffn": shape.ffn, "vocab": shape.vocab, "ar_rank": shape.ar_rank,
                   "rows_per_request": shape.rows},
        "roofline": roof,
        "backbone": {"ms": backbone_ms, "algorithmic_GB": bb_bytes / 1e9, "GFLOP": bb_flops / 1e9,
                     "GB_s": bb_bytes / bb_s / 1e9, "TFLOP_s": bb_flops / bb_s / 1e12,
                     "hbm_frac": bb_bytes / bb_s / 1e9 / PEAK_HBM_GBS,
                     "mfma_frac": bb_flops / bb_s / 1e12 / peak_flops},
        "head_us_per_round": head_us,
        "head_full_fallback": dr.head_fallback(),
        "verify_us_per_round": 1000.0 * sum_ms(["verify"]),
        "append_us_per_round": 1000.0 * sum_ms(["append_gemm", "append_store"]),
        "phases": phases,
        "graph_ms_per_step": graph_ms,
    }
    if shape.dtype == "bf16" and not args.no_head_sweep:
        hs = head_sweep(dr, shape, batches=tuple(int(x) for x in args.head_sweep_batches.split(",")))
        out["head_us_by_batch"] = hs.pop("plain_us")
        out["head_variants_by_batch"] = hs
    if shape.dtype == "bf16" and not args.no_head_sweep:
        out["fuse_by_rows"] = fuse_timing(shape)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample ...")
        out["cpu_baseline"] = cpu_baseline(wl, weights, ri)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
