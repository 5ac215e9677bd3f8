"""Benchmark of the FarSkip MoE block forward on one MI355X.

One step = one pass of the whole hot path over one batch: router + top-k,
dispatch plan + pack, the dispatch stand-in copy on a second stream, shared
and routed grouped SwiGLU experts, Combine and the deferred residual add
(fs_moe_block_forward BEGIN + FINISH).  The default workload is the
Llama-4-Scout-shaped layer (8192 tokens, d 5120, 16 experts top-1 sigmoid
with a uniform selection bias, one shared expert, expert FFN 8192, bf16),
the largest single-GPU workload, inputs resident in HBM.  The same step is
then timed on the DeepSeek-V2-Lite-shaped layer and the DeepSeek-V3-shaped
prefill and decode ranks (``--extra``), reported under ``workloads``.

    python bench.py [--steps K] [--warmup W] [--config NAME] [--extra A,B] [--gpus 1]

Prints one JSON line.
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "MoE-block tokens/sec per GPU; grouped-GEMM % bf16 MFMA peak; permute % HBM"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_FP8_TFLOPS = 5000.0      # MI355X dense fp8 MFMA
PEAK_F32_VALU_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def measured_traffic(cfg_name):
    """HBM bytes per launch of the routed gate/up GEMM from the rocprofv3
    FETCH_SIZE / WRITE_SIZE runs kept under profiles/, if they were taken on
    this workload with the current kernel source; otherwise None."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"gate_up_gemm_{cfg_name}_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    src = os.path.join(ROOT, rec["source"])
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec["source_sha256"]:
        return None
    return rec["hbm_bytes_per_launch"]


KERNEL_NAMES = ("router", "topk", "plan", "pack", "gate_up", "down", "combine", "shared_gate_up",
                "shared_down", "dispatch_copy", "next_layer", "combine_copy", "allreduce_copy",
                "quantize")


def kernel_table(L):
    """Average launch time of each profiled kernel (library HIP events on the
    stream each one runs on) since the last fs_profile_reset."""
    out = {}
    for kid, nm in enumerate(KERNEL_NAMES):
        ms, n = L.fs_profile_read(kid)
        if n:
            out[nm] = {"us_per_launch": 1e3 * ms / n, "launches": n}
    return out


KERNELS_NOTE = ("per-launch us from library HIP events: gate_up from the timed steps, where only "
                "its events are on; the others from an untimed pass of as many steps with "
                "every kernel's events on")


def time_steps(L, run, steps, warmup, stream):
    """Warm up, then time `steps` runs between torch events on `stream`.
    Only the routed gate/up pass (the roofline's kernel) carries the
    library's HIP events in those steps: every timed kernel adds stream
    events, which slow a step of short kernels by up to a fifth.  A second,
    untimed pass of `steps` runs with every kernel's events on gives the
    other kernels' times.  Returns (ms per step, per-kernel table whose
    gate_up entry comes from the timed steps)."""
    import torch
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    L.fs_profile_reset()
    L.fs_profile_select([L.FS_K_GATE_UP])
    L.fs_profile_enable(True)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(steps):
        run()
    b.record(stream)
    torch.cuda.synchronize()
    L.fs_profile_enable(False)
    ms = a.elapsed_time(b) / steps
    timed_gu = kernel_table(L).get("gate_up")
    L.fs_profile_reset()
    L.fs_profile_select(None)
    L.fs_profile_enable(True)
    for _ in range(steps):
        run()
    torch.cuda.synchronize()
    L.fs_profile_enable(False)
    table = kernel_table(L)
    if timed_gu is not None:
        table["gate_up"] = timed_gu
    return ms, table


def ffn_roofs(rows, groups, d, F, es, fp8):
    """(bytes, flops, MFMA peak) of an FFN's gate/up and down passes.  FP8:
    1-byte weights and input codes, H written in bf16, and the down pass
    includes H's quantisation (read H, write its codes) before reading the
    codes."""
    if not fp8:
        mm = (PEAK_BF16_TFLOPS if es == 2 else PEAK_F32_VALU_TFLOPS) * 1e12
        return ((groups * 2 * F * d + rows * d + rows * F) * es, 2.0 * rows * d * 2 * F, mm), \
               ((groups * d * F + rows * F + rows * d) * es, 2.0 * rows * d * F, mm)
    mm = PEAK_FP8_TFLOPS * 1e12
    return (groups * 2 * F * d + rows * d + 2 * rows * F + 4 * rows, 2.0 * rows * d * 2 * F, mm), \
           (groups * d * F + 2 * rows * F + 2 * rows * F + 4 * rows + 2 * rows * d,
            2.0 * rows * d * F, mm)


def step_roofs(cfg, M, active, fp8_routed=False, fp8_shared=False):
    """Algorithmic (bytes, flops, roof time in us) of each step of one pass,
    at HBM 8 TB/s, bf16 MFMA 2.5 PFLOP/s, fp8 MFMA 5.0 PFLOP/s and fp32
    vector 157.3 TFLOP/s.  With FP8 routed experts the N token rows are
    quantised once before pack, and pack moves codes (1 byte) and scales."""
    es = cfg.elem_bytes
    N, d, k, E, F = cfg.n_tokens, cfg.hidden, cfg.top_k, cfg.n_experts, cfg.ffn
    SF = cfg.n_shared * cfg.ffn_shared
    hbm, valu = PEAK_HBM_GBS * 1e9, PEAK_F32_VALU_TFLOPS * 1e12
    gu, dn = ffn_roofs(M, active, d, F, es, fp8_routed)
    steps = {
        "router": (N * d * es + E * d * es + N * E * 4, 2.0 * N * d * E, valu),
        "topk": (N * E * 4 + N * k * 8, 0.0, valu),
        "plan": (12 * N * k, 0.0, valu),
        "pack": ((N * d + N * k * d + 4 * N + 4 * N * k + 4 * N * k) if fp8_routed
                 else (N * d * es + N * k * d * es + 4 * N * k), 0.0, valu),
        "gate_up": gu,
        "down": dn,
        "combine": (N * k * d * es + 8 * N * k + 2 * N * d * es, 0.0, valu),
    }
    if fp8_routed:
        steps["quantize"] = (N * d * es + N * d + 4 * N, 0.0, valu)
    if SF:
        steps["shared_gate_up"], steps["shared_down"] = ffn_roofs(N, 1, d, SF, es, fp8_shared)
        steps["partial"] = (3 * N * d * es, 0.0, valu)
        if fp8_shared:
            b, f, p = steps["quantize"] if "quantize" in steps else (0, 0.0, valu)
            steps["quantize"] = (b + N * d * es + N * d + 4 * N, f, p)
    return {k2: (b, f, 1e6 * max(b / hbm, f / peak)) for k2, (b, f, peak) in steps.items()}


def cpu_baseline(cfg, wl, sample_tokens):
    """The oracle, as it stands, on the first `sample_tokens` tokens of this
    rank: the whole block for those tokens, timed on the host."""
    import numpy as np
    import threadpoolctl

    import oracle
    f64 = lambda t: None if t is None else t.detach().float().cpu().numpy().astype(np.float64)
    if sample_tokens <= 0:
        # about 1 TFLOP of fp64 work per pass: router, the k routed experts
        # (local ones only when R > 1: about k / R per token) and the shared
        # experts, 6 d F flops per SwiGLU row
        per_token = 2 * cfg.hidden * cfg.n_experts + 6 * cfg.hidden * (
            cfg.top_k / cfg.ep_size * cfg.ffn + cfg.n_shared * cfg.ffn_shared)
        sample_tokens = max(64, int(1e12 / per_token))
    n = min(sample_tokens, cfg.n_tokens)
    x = f64(wl.x[:n])
    wr, bias = f64(wl.w_router), f64(wl.bias)
    gu, dn = f64(wl.w_gate_up), f64(wl.w_down)
    sgu, sdn = f64(wl.sh_gate_up), f64(wl.sh_down)
    yr = f64(wl.y_remote)
    info = threadpoolctl.threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info] or [1])
    def one_pass():
        if cfg.ep_size == 1:
            ref = oracle.moe_block(cfg.scaled(n_tokens=n), x[None], wr, bias, gu, dn, sgu, sdn)
            routed, shared = ref["routed"], ref["shared"]
        else:
            z32 = oracle.logits_routing_f32(x, wr)
            ids, w, _, _ = oracle.route(z32, cfg.score, cfg.top_k, cfg.n_groups, cfg.topk_groups,
                                        cfg.norm_topk, cfg.routed_scale, bias)
            # the sample's own plan; the other ranks' experts return their
            # rows at its positions in the return buffer
            plan = oracle.dispatch_plan(ids, cfg.n_experts, cfg.ep_size)
            s2r = plan["slot_to_row"]
            rows = [[yr[s2r[t * cfg.top_k + j]] for j in range(cfg.top_k)] for t in range(n)]
            routed = oracle.moe_tokens_direct(cfg, x, ids, w, lambda e: (gu[e], dn[e]), rows)
            shared = oracle.shared_ffn(x, sgu, sdn)
        oracle.residual_add(x, shared, routed)

    # repeat whole passes until about 10 s of host work (at most 30 s)
    passes, t0 = 0, time.perf_counter()
    while True:
        one_pass()
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= 10.0 or dt * (passes + 1) / passes > 30.0:
            break
    return {"value": n * passes / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"first {n} of {cfg.n_tokens} tokens of this workload, whole block in fp64 "
                      f"NumPy, {passes} pass(es) in {dt:.1f} s; host affinity "
                      f"{len(os.sched_getaffinity(0))} cores"}


def bench_layers(args, cfg, torch, L):
    """L stacked layers (attention stand-in + MoE block each) in the
    two-window FarSkip schedule on two streams and in the regular schedule
    on one; one JSON line with both times and Eq. 9's budget per layer."""
    import paper_2511_11505_amd as fs
    from paper_2511_11505_amd.stack import LayerStack
    from workloads.generate import merge_shared, stack_layers

    dev = "cuda:0"
    t0 = time.perf_counter()
    layers = stack_layers(cfg, args.layers, dev)
    st = LayerStack(cfg, layers, device=dev, merge_shared=merge_shared)
    if cfg.ep_size > 1:
        for (lc, wl, _, _), blk in zip(layers, st.blocks):
            blk.set_max_recv_rows(fs.prepare_remote_sources(blk, wl.x_all, wl.w_router, wl.bias,
                                                            wl.y_remote))
    x = layers[0][1].x
    comm = torch.cuda.Stream(device=dev)
    compute = torch.cuda.current_stream()
    torch.cuda.synchronize()
    log(f"setup {time.perf_counter() - t0:.1f}s: {args.layers} layers of {cfg.name}")

    def timed(run):
        return time_steps(L, run, args.steps, args.warmup, compute)

    ms_fs, k_fs = timed(lambda: st.farskip(x, compute=compute, comm=comm))
    ms_rg, k_rg = timed(lambda: st.regular(x, compute=compute))
    us = lambda k, name: k[name]["us_per_launch"] if name in k else 0.0
    link = None
    if args.link_gbs > 0:
        # both schedules again, every stand-in copy paced at the time the
        # all-to-all of its buffer takes on 8 GPUs joined by 7 links each
        with L.standin_link(7, args.link_gbs * 1e9, args.link_wgs):
            ms_fs_l, k_fs_l = timed(lambda: st.farskip(x, compute=compute, comm=comm))
            ms_rg_l, k_rg_l = timed(lambda: st.regular(x, compute=compute))
        link = {"links": 7, "link_gbs": args.link_gbs, "workgroups": args.link_wgs,
                "copy_model_us_each": round(cfg.cap * cfg.hidden * cfg.elem_bytes / 8
                                            / (args.link_gbs * 1e9) * 1e6, 2),
                "farskip_ms_per_step": ms_fs_l, "regular_ms_per_step": ms_rg_l,
                "speedup_vs_regular": ms_rg_l / ms_fs_l,
                "farskip_copy_us": {n: round(us(k_fs_l, n), 2) for n in ("dispatch_copy", "combine_copy")},
                "regular_copy_us": {n: round(us(k_rg_l, n), 2) for n in ("dispatch_copy", "combine_copy")},
                "kernels_us": {k2: round(v["us_per_launch"], 2) for k2, v in k_fs_l.items()},
                "note": "both schedules measured with each Dispatch and Combine stand-in copy "
                        "run on link_wgs workgroups and paced to the time the all-to-all of its "
                        "buffer takes on a node of 8 GPUs (1/8 of the buffer per link at "
                        "link_gbs, all links at once); the link rate is emulated, the overlap, "
                        "the copies' CU and HBM use and the schedule are measured"}
    per_layer = ms_fs * 1e3 / args.layers
    gate = sum(us(k_fs, n) for n in ("router", "topk", "plan", "pack"))
    routed = us(k_fs, "gate_up") + us(k_fs, "down")
    comm_us = us(k_fs, "dispatch_copy") + us(k_fs, "combine_copy")
    N = cfg.n_tokens
    # model: the regular schedule with its blocking copies taking the time
    # an all-to-all of the same buffers would take on an 8-GPU xGMI node
    # (1/8 of the buffer per peer at 153 GB/s, links in parallel); the
    # FarSkip schedule keeps its measured time while the copies fit Eq. 9's
    # window
    xgmi_us = cfg.cap * cfg.hidden * cfg.elem_bytes / 8 / 153e9 * 1e6
    rg_copies_ms = args.layers * (us(k_rg, "dispatch_copy") + us(k_rg, "combine_copy")) / 1e3
    rg_xgmi_ms = ms_rg - rg_copies_ms + args.layers * 2 * xgmi_us / 1e3
    res = {
        "metric": "FarSkip stacked-layer tokens/sec per GPU (attention stand-in + MoE block per layer)",
        "value": N / (ms_fs * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_fs, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {args.layers} stacked layers, two-window FarSkip "
                               f"schedule (Dispatch and Combine stand-in copies on a second stream)",
                   "layers": args.layers, "tokens": N, "hidden": cfg.hidden,
                   "experts": cfg.n_experts, "top_k": cfg.top_k, "ffn": cfg.ffn,
                   "shared": cfg.n_shared, "ffn_shared": cfg.ffn_shared,
                   "ep_size": cfg.ep_size, "dtype": cfg.dtype},
        "regular_ms_per_step": ms_rg,
        "speedup_vs_regular": ms_rg / ms_fs,
        "xgmi_model": {"copy_us_each": round(xgmi_us, 2),
                       "regular_ms_per_step": round(rg_xgmi_ms, 4),
                       "speedup_vs_regular": round(rg_xgmi_ms / ms_fs, 4),
                       "farskip_copies_fit_window": 2 * xgmi_us <= per_layer - routed - gate,
                       "note": "regular schedule with its measured blocking copies replaced by "
                               "all-to-all time on an 8-GPU xGMI node (model, not a measurement)"},
        "link_emulated": link,
        "eq9_per_layer_us": {"dispatch_plus_combine": round(comm_us, 2),
                             "layer": round(per_layer, 2), "routed_experts": round(routed, 2),
                             "gate": round(gate, 2),
                             "window": round(per_layer - routed - gate, 2),
                             "fits": comm_us <= per_layer - routed - gate},
        "kernels_us_note": KERNELS_NOTE,
        "kernels_us": {k2: round(v["us_per_launch"], 2) for k2, v in k_fs.items()},
        "kernels_us_regular": {k2: round(v["us_per_launch"], 2) for k2, v in k_rg.items()},
    }
    st.close()
    print(json.dumps(res), flush=True)


def bench_replicated(args, cfg, torch, L):
    """L stacked layers of the replicated-activation (all-reduce) variant on
    one rank: the FarSkip schedule with the all-reduce stand-in copies on a
    second stream, the same order on one stream, and the regular schedule;
    one JSON line with the times, Tab. 5's two overlap windows and the
    roofline of the gathered routed gate/up GEMM."""
    import numpy as np

    from paper_2511_11505_amd.replicated import ReplicatedStack
    from workloads.generate import merge_shared, stack_layers, tp_attention_slice, tp_shared_slice

    dev = "cuda:0"
    t0 = time.perf_counter()
    R, r = cfg.ep_size, cfg.ep_rank
    layers = stack_layers(cfg, args.layers, dev)
    gl = []
    for _, wl, w_a, w_b in layers:
        sh_gu = sh_dn = None
        if cfg.n_shared:
            sh_gu, sh_dn = tp_shared_slice(*merge_shared(wl.sh_gate_up, wl.sh_down), R, r)
        wa_r, wb_r = tp_attention_slice(w_a, w_b, R, r)
        gl.append(dict(w_router=wl.w_router, bias=wl.bias, w_gate_up=wl.w_gate_up,
                       w_down=wl.w_down, sh_gate_up=sh_gu, sh_down=sh_dn, w_a=wa_r, w_b=wb_r))
    x = layers[0][1].x
    del layers
    st = ReplicatedStack(cfg, gl, device=dev)
    comm = torch.cuda.Stream(device=dev)
    compute = torch.cuda.current_stream()
    # rows this rank's experts receive, per layer (untimed pass)
    st.farskip(x, compute=compute, comm=comm, keep_ids=True)
    torch.cuda.synchronize()
    lo, hi = r * cfg.n_local, (r + 1) * cfg.n_local
    rows, active = [], []
    for ids in st.kept_ids:
        ids = ids.cpu().numpy()
        local = ids[(ids >= lo) & (ids < hi)]
        rows.append(local.size)
        active.append(np.unique(local).size)
    st.kept_ids = []
    log(f"setup {time.perf_counter() - t0:.1f}s: {args.layers} replicated layers of {cfg.name}, "
        f"local rows per layer {rows}")

    def timed(run):
        return time_steps(L, run, args.steps, args.warmup, compute)

    ms_fs, k_fs = timed(lambda: st.farskip(x, compute=compute, comm=comm))
    if args.farskip_only:
        line = {"schedule": "farskip", "ms_per_step": ms_fs,
                "kernels_us": {k2: round(v["us_per_launch"], 2) for k2, v in k_fs.items()}}
        if args.link_gbs > 0:
            # then with the link-paced all-reduce stand-ins
            with L.standin_link(7, args.link_gbs * 1e9, args.link_wgs):
                ms_l, k_l = timed(lambda: st.farskip(x, compute=compute, comm=comm))
            line["link_emulated"] = {"ms_per_step": ms_l, "kernels_us": {
                k2: round(v["us_per_launch"], 2) for k2, v in k_l.items()}}
        print(json.dumps(line), flush=True)
        return
    ms_serial, _ = timed(lambda: st.farskip(x, compute=compute, comm=None))
    ms_rg, k_rg = timed(lambda: st.regular(x, compute=compute))
    us = lambda k, name: k[name]["us_per_launch"] if name in k else 0.0
    link = None
    if args.link_gbs > 0:
        # both schedules again, every all-reduce stand-in paced at the time
        # a ring all-reduce of its message takes over the 7 links of each
        # of 8 GPUs
        with L.standin_link(7, args.link_gbs * 1e9, args.link_wgs):
            ms_fs_l, k_fs_l = timed(lambda: st.farskip(x, compute=compute, comm=comm))
            ms_rg_l, k_rg_l = timed(lambda: st.regular(x, compute=compute))
        link = {"links": 7, "link_gbs": args.link_gbs, "workgroups": args.link_wgs,
                "allreduce_model_us": round(2 * cfg.n_tokens * cfg.hidden * cfg.elem_bytes / 8
                                            / (args.link_gbs * 1e9) * 1e6, 2),
                "farskip_ms_per_step": ms_fs_l, "regular_ms_per_step": ms_rg_l,
                "speedup_vs_regular": ms_rg_l / ms_fs_l,
                "farskip_copy_us": round(us(k_fs_l, "allreduce_copy"), 2),
                "regular_copy_us": round(us(k_rg_l, "allreduce_copy"), 2),
                "kernels_us": {k2: round(v["us_per_launch"], 2) for k2, v in k_fs_l.items()},
                "note": "both schedules measured with each all-reduce stand-in copy run on "
                        "link_wgs workgroups and paced to the time a ring all-reduce of the "
                        "message takes over every link of a node of 8 GPUs (link_gbs per "
                        "direction); the link rate is emulated, the overlap, the copies' CU "
                        "and HBM use and the schedule are measured"}
    N, d, F, es = cfg.n_tokens, cfg.hidden, cfg.ffn, cfg.elem_bytes
    per_layer = ms_fs * 1e3 / args.layers
    attention = 2 * us(k_fs, "next_layer")
    routed = sum(us(k_fs, n) for n in ("router", "topk", "plan", "gate_up", "down", "combine"))
    shared = us(k_fs, "shared_gate_up") + us(k_fs, "shared_down")
    copy = us(k_fs, "allreduce_copy")
    msg_bytes = N * d * es
    # ring all-reduce of one [N, d] message over R ranks moves 2 (R-1)/R of
    # it through each rank: at the bus bandwidth of App. B's accelerator
    # (400 GB/s) and at the rate of 7 xGMI links of 153 GB/s
    ring = 2.0 * (R - 1) / R * msg_bytes
    ar_400 = ring / 400e9 * 1e6
    ar_links = ring / (7 * 153e9) * 1e6
    M = float(np.mean(rows))
    act = float(np.mean(active))
    bytes_gu = (act * 2 * F * d + M * d + M * F) * es
    flops_gu = 2.0 * M * d * 2 * F
    t_gu = us(k_fs, "gate_up") * 1e-6
    hbm_gbs, tflops = bytes_gu / t_gu / 1e9, flops_gu / t_gu / 1e12
    mfma_bound = flops_gu / (PEAK_BF16_TFLOPS * 1e12) >= bytes_gu / (PEAK_HBM_GBS * 1e9)
    roof = ({"bound": "mfma", "achieved": round(tflops, 2), "peak": PEAK_BF16_TFLOPS,
             "unit": "TFLOP/s", "frac": round(tflops / PEAK_BF16_TFLOPS, 4)} if mfma_bound else
            {"bound": "hbm", "achieved": round(hbm_gbs, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
             "frac": round(hbm_gbs / PEAK_HBM_GBS, 4)})
    roof.update({"kernel": "gathered routed gate/up SwiGLU GEMM", "traffic": None,
                 "algorithmic_bytes_per_launch": int(bytes_gu),
                 "algorithmic_flops_per_launch": flops_gu, "local_rows": round(M, 1),
                 "experts_with_rows": round(act, 2),
                 "mfma_frac": round(tflops / PEAK_BF16_TFLOPS, 4),
                 "hbm_frac": round(hbm_gbs / PEAK_HBM_GBS, 4)})
    rg_copies_ms = args.layers * 2 * us(k_rg, "allreduce_copy") / 1e3
    model = lambda t_ar: {
        "allreduce_us": round(t_ar, 2),
        "regular_ms_per_step": round(ms_rg - rg_copies_ms + args.layers * 2 * t_ar / 1e3, 4),
        "farskip_ms_per_step": round(ms_fs + args.layers * (max(0.0, t_ar - routed)
                                                            + max(0.0, t_ar - attention)) / 1e3, 4),
        "attention_shared_ar_hidden": t_ar <= routed,
        "routed_ar_hidden": t_ar <= attention}
    m400, mlinks = model(ar_400), model(ar_links)
    for m in (m400, mlinks):
        m["speedup_vs_regular"] = round(m["regular_ms_per_step"] / m["farskip_ms_per_step"], 4)
    res = {
        "metric": "replicated-activation FarSkip stacked-layer tokens/sec per GPU "
                  "(one EP/TP rank: attention and shared-expert blocks, own routed experts)",
        "value": N / (ms_fs * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_fs, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {args.layers} stacked layers, replicated activations, "
                               f"rank {r} of EP = TP = {R}; all-reduce stand-in copies on a second "
                               f"stream", "layers": args.layers, "tokens": N, "hidden": d,
                   "experts": cfg.n_experts, "top_k": cfg.top_k, "ep_size": R,
                   "local_rows_per_layer": rows},
        "serial_ms_per_step": ms_serial,
        "regular_ms_per_step": ms_rg,
        "speedup_vs_regular": ms_rg / ms_fs,
        "roofline": roof,
        "tab5_windows_per_layer_us": {
            "layer": round(per_layer, 2), "attention": round(attention, 2),
            "shared": round(shared, 2), "routed_experts": round(routed, 2),
            "allreduce_copy": round(copy, 2),
            "note": "the attention + shared all-reduce hides behind the routed experts, "
                    "the routed all-reduce behind the next attention"},
        "link_emulated": link,
        "allreduce_model": {"message_bytes": msg_bytes, "at_400GBs_bus": m400,
                            "at_7_xgmi_links": mlinks,
                            "note": "measured times with each stand-in copy replaced by a ring "
                                    "all-reduce of the message over R ranks (model, not a "
                                    "measurement); FarSkip pays only what exceeds its window"},
        "kernels_us_note": KERNELS_NOTE,
        "kernels_us": {k2: round(v["us_per_launch"], 2) for k2, v in k_fs.items()},
        "kernels_us_regular": {k2: round(v["us_per_launch"], 2) for k2, v in k_rg.items()},
    }
    print(json.dumps(res), flush=True)


EXTRA_DEFAULT = "dsv2lite,dsv3_prefill,dsv3_decode"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="scout")
    ap.add_argument("--extra", default=EXTRA_DEFAULT,
                    help="comma-separated workloads also timed in the same run (same steps), "
                         "reported under 'workloads' in the JSON line; '' for none")
    ap.add_argument("--cpu-sample", type=int, default=0,
                    help="tokens of the workload the oracle runs on the host (0: as many as about "
                         "1 TFLOP of fp64 work per pass)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--serial", action="store_true", help="no second stream")
    ap.add_argument("--rotate", type=int, default=4, help="input sets rotated across steps")
    ap.add_argument("--graph", action="store_true",
                    help="also time the step captured as a HIP graph and replayed")
    ap.add_argument("--layers", type=int, default=0,
                    help="run this many stacked layers in the two-window schedule and the regular one "
                         "(replicated-activation workloads always run stacked layers, 4 by default)")
    ap.add_argument("--fp8", choices=("routed", "all"), default=None,
                    help="run the routed (or routed and shared) experts in FP8 E4M3")
    ap.add_argument("--farskip-only", action="store_true",
                    help="replicated-activation workloads: time only the two-stream FarSkip schedule, "
                         "with HBM-speed and then link-paced copies (for kernel traces)")
    ap.add_argument("--link-gbs", type=float, default=153.0,
                    help="stacked-layer runs: also time both schedules with every stand-in copy "
                         "paced at the time its collective takes on a node of 8 GPUs joined by "
                         "links of this many GB/s per direction (0: skip)")
    ap.add_argument("--link-wgs", type=int, default=128,
                    help="workgroups of each link-paced stand-in copy")
    ap.add_argument("--vendor-reference", action="store_true",
                    help="also time the block's GEMM passes as plain hipBLASLt GEMMs (context)")
    ap.add_argument("--no-shared-beside", action="store_true",
                    help="skip the extra timing of the side-stream phase order (kernel traces "
                         "then hold the default order's launches only)")
    ap.add_argument("--overlap", action="store_true",
                    help="run the next-layer stand-in (d x d linear) between BEGIN and FINISH and "
                         "compare with a serial run")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the library has no multi-GPU path (asked for {args.gpus})",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2511_11505_amd import _lib as L
    from workloads import CONFIGS

    cfg = CONFIGS[args.config]
    torch.cuda.set_device(0)
    if cfg.ep_mode == "allreduce":
        args.layers = args.layers or 4
        return bench_replicated(args, cfg, torch, L)
    if args.layers > 0:
        return bench_layers(args, cfg, torch, L)
    res = bench_block(args, cfg, torch, L, with_cpu=not args.no_cpu_baseline)
    extra = [n for n in args.extra.split(",") if n and n != cfg.name]
    if extra:
        res["workloads_note"] = ("the same step timed on the other block workloads in this run "
                                 "(same steps and warm-up, no CPU leg); roofline as in the headline")
        res["workloads"] = {}
        for name in extra:
            torch.cuda.empty_cache()
            r2 = bench_block(args, CONFIGS[name], torch, L, with_cpu=False)
            res["workloads"][name] = {key: r2[key] for key in (
                "value", "unit", "ms_per_step", "config", "roofline", "ffn", "permute_frac_hbm",
                "step_roofline_frac", "block_roofline_frac", "kernels_us", "vendor_reference",
                "shared_beside")
                if key in r2}
            torch.cuda.empty_cache()
    print(json.dumps(res), flush=True)


def vendor_reference(cfg, blk, wl, kernels, torch):
    """The block's four GEMM passes as plain hipBLASLt GEMMs (torch.matmul),
    for context: the routed passes as one GEMM per local expert with the
    block's own row counts, the shared passes as one dense GEMM each.  They
    do less than the library's passes (no row gather or scatter, no SwiGLU
    epilogue), on random inputs of the same shapes and distribution."""
    dev = "cuda:0"
    d, F, E_loc = cfg.hidden, cfg.ffn, cfg.n_local
    lo = cfg.ep_rank * E_loc
    counts = blk.t["src_counts"][:, lo:lo + E_loc].sum(0).tolist()
    dt = torch.bfloat16
    g = torch.Generator(device=dev).manual_seed(7)
    xs = [torch.randn((n, d), generator=g, device=dev, dtype=torch.float32).to(dt) for n in counts]
    hs = [torch.randn((n, F), generator=g, device=dev, dtype=torch.float32).to(dt) for n in counts]

    def timed(fn, reps=10):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps * 1e3

    def routed(inputs, w):
        for e, xe in enumerate(inputs):
            if xe.shape[0]:
                torch.matmul(xe, w[e].t())
    M = sum(counts)
    ref = {"gate_up": timed(lambda: routed(xs, wl.w_gate_up)),
           "down": timed(lambda: routed(hs, wl.w_down))}
    flops = {"gate_up": 2.0 * M * d * 2 * F, "down": 2.0 * M * F * d}
    if cfg.n_shared > 0 and blk.weights_keep[4] is not None:
        sh_gu, sh_dn = blk.weights_keep[4], blk.weights_keep[5]
        Fs = sh_dn.shape[1]
        x = torch.randn((cfg.n_tokens, d), generator=g, device=dev, dtype=torch.float32).to(dt)
        h = torch.randn((cfg.n_tokens, Fs), generator=g, device=dev, dtype=torch.float32).to(dt)
        ref["shared_gate_up"] = timed(lambda: torch.matmul(x, sh_gu.t()))
        ref["shared_down"] = timed(lambda: torch.matmul(h, sh_dn.t()))
        # the library's shared FFN alone (in the block it runs beside the
        # Dispatch stand-in copy)
        from paper_2511_11505_amd import _lib as L
        ws = torch.empty((max(L.fs_workspace_size(blk.desc, L.FS_OP_GROUPED_FFN, cfg.n_tokens, Fs), 256),),
                         dtype=torch.uint8, device=dev)
        y = torch.empty((cfg.n_tokens, d), dtype=dt, device=dev)
        run = lambda: L.fs_grouped_expert_ffn(blk.desc, 1, Fs, x, None, None, cfg.n_tokens, sh_gu,
                                              sh_dn, y, ws)
        for _ in range(3):
            run()
        torch.cuda.synchronize()
        L.fs_profile_reset()
        L.fs_profile_select([L.FS_K_SHARED_GATE_UP, L.FS_K_SHARED_DOWN])
        L.fs_profile_enable(True)
        for _ in range(10):
            run()
        torch.cuda.synchronize()
        L.fs_profile_enable(False)
        alone = kernel_table(L)
        L.fs_profile_reset()
        L.fs_profile_select(None)
        flops["shared_gate_up"] = 2.0 * cfg.n_tokens * d * 2 * Fs
        flops["shared_down"] = 2.0 * cfg.n_tokens * Fs * d
    else:
        alone = {}
    out = {}
    frac = lambda k, us: round(flops[k] / us / 1e6 / PEAK_BF16_TFLOPS, 4)
    for k, us in ref.items():
        ours = kernels.get(k, {}).get("us_per_launch")
        out[k] = {"hipblaslt_us": round(us, 2), "hipblaslt_frac": frac(k, us),
                  "ours_us": round(ours, 2) if ours else None,
                  "ours_frac": frac(k, ours) if ours else None}
        if k in alone:
            out[k]["ours_alone_us"] = round(alone[k]["us_per_launch"], 2)
            out[k]["ours_alone_frac"] = frac(k, alone[k]["us_per_launch"])
    return {"passes": out, "note": "hipBLASLt (torch.matmul) on the same GEMM shapes: routed passes as "
            "one GEMM per local expert with the block's row counts, shared passes dense; plain GEMMs "
            "without the library's gather, scatter and SwiGLU epilogue; fractions of the 2.5 PFLOP/s "
            "bf16 peak; ours_us inside the block step, ours_alone_us the library's shared FFN "
            "(fs_grouped_expert_ffn, one group) run alone"}


def bench_block(args, cfg, torch, L, with_cpu):
    """Time fs_moe_block_forward (BEGIN + FINISH) on one workload; returns
    the result dict of the JSON line."""
    import paper_2511_11505_amd as fs
    from workloads import make_workload
    from workloads.generate import merge_shared, source_tokens

    dev = "cuda:0"
    t_setup = time.perf_counter()
    wl = make_workload(cfg, dev)
    sh_gu = sh_dn = None
    if cfg.n_shared > 0:
        sh_gu, sh_dn = merge_shared(wl.sh_gate_up, wl.sh_down)
    # decode-sized routed passes (a few rows per local expert) stream the
    # experts' weights in fragment order
    fo = cfg.dtype == "bf16" and cfg.cap <= 64 * cfg.n_local
    blk = fs.MoEBlock(cfg, wl.w_router, wl.bias, wl.w_gate_up, wl.w_down, sh_gu, sh_dn, device=dev,
                      fp8=args.fp8, fragment_order=fo)
    M = cfg.cap
    if cfg.ep_size > 1:
        M = fs.prepare_remote_sources(blk, wl.x_all, wl.w_router, wl.bias, wl.y_remote)
        blk.set_max_recv_rows(M)
    # rotating input sets so the 256 MB last-level cache does not hold them
    xs = [wl.x] + [source_tokens(cfg.scaled(seed=cfg.seed + 1000 + i), dev, cfg.ep_rank)
                   for i in range(1, max(1, args.rotate))]
    partials = [torch.empty_like(wl.x) for _ in xs]
    comm = None if args.serial else torch.cuda.Stream(device=dev)
    compute = torch.cuda.current_stream()
    torch.cuda.synchronize()
    log(f"setup {time.perf_counter() - t_setup:.1f}s: {cfg.name}, rows on local experts M={M}")

    dt_id = L.FS_F32 if cfg.dtype == "f32" else L.FS_BF16
    nxts = [torch.empty_like(wl.x) for _ in xs] if args.overlap else None
    outs = [torch.empty_like(wl.x) for _ in xs] if args.overlap else None

    side = torch.cuda.Stream(device=dev)

    def step(i, comm_stream, beside=False):
        j = i % len(xs)
        if beside:
            # the shared experts on a side stream beside the routed experts:
            # GATE, then SHARED on `side` while EXPERTS runs on `compute`;
            # COMBINE adds into the partial input SHARED wrote, so it waits
            blk.phase(L.FS_PHASE_GATE, xs[j], compute=compute, comm=comm_stream)
            side.wait_stream(compute)
            blk.phase(L.FS_PHASE_SHARED, xs[j], partial_out=partials[j], compute=side,
                      comm=comm_stream)
            blk.phase(L.FS_PHASE_EXPERTS, xs[j], compute=compute, comm=comm_stream)
            compute.wait_stream(side)
            blk.phase(L.FS_PHASE_COMBINE, xs[j], residual_io=partials[j], compute=compute,
                      comm=comm_stream)
            return
        blk.begin(xs[j], partials[j], compute=compute, comm=comm_stream)
        if args.overlap:
            # the far-skipped next layer reads the partial input while the
            # Dispatch stand-in is in flight; its output joins the residual
            # before the deferred routed add (Eq. 7)
            L.fs_dense_linear(dt_id, cfg.n_tokens, cfg.hidden, cfg.hidden, partials[j], wl.w_next,
                              nxts[j], stream=compute)
            L.fs_farskip_residual(blk.desc, outs[j], partials[j], nxts[j], stream=compute)
            blk.finish(xs[j], outs[j], compute=compute, comm=comm_stream)
        else:
            blk.finish(xs[j], partials[j], compute=compute, comm=comm_stream)

    def timed(comm_stream, beside=False):
        n = [0]

        def run():
            step(n[0], comm_stream, beside)
            n[0] += 1
        return time_steps(L, run, args.steps, args.warmup, compute)

    ms, kernels = timed(comm)
    shared_beside = None
    if comm is not None and not args.overlap and not getattr(args, "no_shared_beside", False):
        # the same step with the shared experts beside the routed experts;
        # the two passes then share the GPU, so the per-kernel table and the
        # roofline stay the default schedule's
        ms_sb, _ = timed(comm, beside=True)
        shared_beside = {"ms_per_step": ms_sb, "tokens_per_s": cfg.n_tokens / (ms_sb * 1e-3),
                         "note": "shared experts on a side stream beside the routed experts "
                                 "(GATE; SHARED on the side stream while EXPERTS runs; COMBINE "
                                 "after both), same kernels and results"}
    serial = timed(None) if (args.overlap and comm is not None) else None
    graph = None
    if args.graph:
        # one HIP graph per input set, captured on a side stream (the comm
        # stream joins the capture through the library's events), replayed
        # in rotation; the per-kernel table stays the eager run's
        graphs = []
        side = torch.cuda.Stream(device=dev)
        for j in range(len(xs)):
            gr = torch.cuda.CUDAGraph()
            side.wait_stream(compute)
            with torch.cuda.stream(side):
                with torch.cuda.graph(gr):
                    cur = torch.cuda.current_stream()
                    blk.begin(xs[j], partials[j], compute=cur, comm=comm)
                    if args.overlap:
                        L.fs_dense_linear(dt_id, cfg.n_tokens, cfg.hidden, cfg.hidden, partials[j],
                                          wl.w_next, nxts[j], stream=cur)
                        L.fs_farskip_residual(blk.desc, outs[j], partials[j], nxts[j], stream=cur)
                        blk.finish(xs[j], outs[j], compute=cur, comm=comm)
                    else:
                        blk.finish(xs[j], partials[j], compute=cur, comm=comm)
            compute.wait_stream(side)
            graphs.append(gr)
        torch.cuda.synchronize()
        for i in range(args.warmup):
            graphs[i % len(graphs)].replay()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(compute)
        for i in range(args.steps):
            graphs[i % len(graphs)].replay()
        b.record(compute)
        torch.cuda.synchronize()
        gms = a.elapsed_time(b) / args.steps
        graph = {"ms_per_step": gms, "tokens_per_s": cfg.n_tokens / (gms * 1e-3),
                 "note": "the same step captured as one HIP graph per input set and replayed"}

    es = cfg.elem_bytes
    N, d, k, E = cfg.n_tokens, cfg.hidden, cfg.top_k, cfg.n_experts
    lo = cfg.ep_rank * cfg.n_local
    rows_per_expert = blk.t["src_counts"][:, lo:lo + cfg.n_local].sum(0)
    active = int((rows_per_expert > 0).sum().item())
    fp8_routed, fp8_shared = args.fp8 is not None, args.fp8 == "all" and cfg.n_shared > 0
    roofs = step_roofs(cfg, M, active, fp8_routed, fp8_shared)
    us = lambda name: kernels[name]["us_per_launch"] if name in kernels else None
    peak_f = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_F32_VALU_TFLOPS
    if fp8_routed:
        peak_f = PEAK_FP8_TFLOPS

    # roofline of the dominant kernel, the routed gate/up SwiGLU GEMM: its
    # algorithmic work is 2 M d 2F flops and (active experts' gate/up weights
    # + M input rows + M rows of H) bytes; the bound is the roof that takes
    # longer, and both fractions are given.
    roof = None
    if us("gate_up"):
        bytes_gu, flops_gu, _ = roofs["gate_up"]
        t = us("gate_up") * 1e-6
        if flops_gu / (peak_f * 1e12) >= bytes_gu / (PEAK_HBM_GBS * 1e9):
            achieved, peak, unit = flops_gu / t / 1e12, peak_f, "TFLOP/s"
            bound = "mfma" if cfg.dtype == "bf16" else "alu"
        else:
            achieved, peak, unit, bound = bytes_gu / t / 1e9, PEAK_HBM_GBS, "GB/s", "hbm"
        roof = {"bound": bound, "kernel": ("FP8 " if fp8_routed else "") + "gate_up SwiGLU grouped GEMM",
                "achieved": round(achieved, 2), "peak": peak, "unit": unit,
                "frac": round(achieved / peak, 4),
                "traffic": None if fp8_routed else measured_traffic(cfg.name),
                "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                "algorithmic_flops_per_launch": flops_gu,
                "algorithmic_bytes_per_launch": bytes_gu, "experts_with_rows": active,
                "mfma_frac": round(flops_gu / t / 1e12 / peak_f, 4),
                "hbm_frac": round(bytes_gu / t / 1e9 / PEAK_HBM_GBS, 4)}

    # the whole FFNs (gate/up + down): routed and shared separately, against
    # the MFMA peak (2 M 3 d F flops) and HBM (weights + activations; the
    # decode metric)
    ffn = {}
    for name, gu_k, dn_k in (("routed", "gate_up", "down"), ("shared", "shared_gate_up", "shared_down")):
        if us(gu_k) and us(dn_k):
            t = (us(gu_k) + us(dn_k)) * 1e-6
            b = roofs[gu_k][0] + roofs[dn_k][0]
            f = roofs[gu_k][1] + roofs[dn_k][1]
            p_ffn = PEAK_FP8_TFLOPS if (fp8_routed if name == "routed" else fp8_shared) else \
                (PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_F32_VALU_TFLOPS)
            ffn[name] = {"us": round(t * 1e6, 2), "tflops": round(f / t / 1e12, 2),
                         "mfma_frac": round(f / t / 1e12 / p_ffn, 4),
                         "hbm_gbs": round(b / t / 1e9, 1), "hbm_frac": round(b / t / 1e9 / PEAK_HBM_GBS, 4)}
    # permute kernels and the router against their roofs (algorithmic bytes;
    # the router against max(bytes / HBM, flops / fp32 vector peak))
    steps_frac = {}
    for name in ("router", "topk", "pack", "combine"):
        if us(name):
            steps_frac[name] = round(roofs[name][2] / us(name), 4)
    hbm = {name: roofs[name][0] / (us(name) * 1e-6) / 1e9 for name in ("pack", "combine") if us(name)}
    # the block against the sum of its steps' roofs (the Dispatch copy is
    # excluded: on a multi-GPU node it is network time, overlapped)
    t_roof = sum(r[2] for r in roofs.values())
    overlap = None
    if args.overlap:
        copy_bytes = cfg.cap * d * (1 if fp8_routed else es) + (4 * cfg.cap if fp8_routed else 0)
        overlap = {"next_layer_us": us("next_layer"), "dispatch_copy_us": us("dispatch_copy"),
                   "dispatch_bytes": copy_bytes,
                   "xgmi_equivalent_us": round(copy_bytes / 8 / 153e9 * 1e6, 2),
                   "note": "xgmi_equivalent_us: the same buffer spread over an 8-GPU node, 1/8 per "
                           "peer at 153 GB/s per link, all links in parallel"}
        if serial is not None:
            ms_s, k_s = serial
            overlap["ms_per_step_serial"] = ms_s
            overlap["slowdown_under_copy"] = {
                name: round(kernels[name]["us_per_launch"] / k_s[name]["us_per_launch"] - 1, 4)
                for name in ("shared_gate_up", "shared_down", "next_layer", "gate_up")
                if name in kernels and name in k_s}
    res = {
        "metric": METRIC,
        "value": N / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": (f"fp8_e4m3 {'routed and shared' if fp8_shared else 'routed'} experts, "
                  f"{cfg.dtype} elsewhere") if fp8_routed else cfg.dtype,
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: FarSkip MoE block forward, {N} tokens, d {d}, {E} experts "
                               f"top-{k} {cfg.score}, FFN {cfg.ffn}, {cfg.n_shared} shared, EP rank "
                               f"{cfg.ep_rank} of {cfg.ep_size}, {cfg.dtype}"
                               + (", with the next-layer stand-in between BEGIN and FINISH"
                                  if args.overlap else "")
                               + (f", FP8 E4M3 experts ({args.fp8})" if fp8_routed else ""),
                   "tokens": N, "hidden": d, "experts": E, "top_k": k, "ffn": cfg.ffn,
                   "shared": cfg.n_shared, "ep_size": cfg.ep_size, "rows_local_experts": M,
                   "second_stream": comm is not None, "next_layer": bool(args.overlap),
                   "fragment_ordered_experts": fo},
        "roofline": roof,
        "grouped_gemm_frac_bf16_peak": None if roof is None else roof["mfma_frac"],
        "ffn": ffn,
        "permute_frac_hbm": {k2: round(v / PEAK_HBM_GBS, 4) for k2, v in hbm.items()},
        "step_roofline_frac": steps_frac,
        "block_roofline_frac": round(t_roof / (ms * 1e3), 4),
        "kernels_us_note": KERNELS_NOTE,
        "kernels_us": {k2: round(v["us_per_launch"], 2) for k2, v in kernels.items()},
    }
    if overlap is not None:
        res["overlap"] = overlap
    if graph is not None:
        res["graph"] = graph
    if shared_beside is not None:
        res["shared_beside"] = shared_beside
    if fp8_routed:
        res["grouped_gemm_frac_bf16_peak"] = None
        res["grouped_gemm_frac_fp8_peak"] = None if roof is None else roof["mfma_frac"]
    if getattr(args, "vendor_reference", False) and cfg.dtype == "bf16" and not fp8_routed:
        res["vendor_reference"] = vendor_reference(cfg, blk, wl, kernels, torch)
    if with_cpu and not fp8_routed:
        try:
            res["cpu_baseline"] = cpu_baseline(cfg, wl, args.cpu_sample)
        except Exception as e:  # report, do not hide the GPU number
            res["cpu_baseline"] = {"error": repr(e)}
    blk.close()
    del blk, wl, xs, partials
    return res


if __name__ == "__main__":
    main()
