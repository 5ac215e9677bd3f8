"""Benchmark of the FarSkip MoE block forward on one MI355X.

One step = one pass of the whole hot path over one batch: router + top-k,
dispatch plan + pack, the dispatch stand-in copy on a second stream, shared
and routed grouped SwiGLU experts, Combine and the deferred residual add
(fs_moe_block_forward BEGIN + FINISH).  The default workload is the
DeepSeek-V2-Lite-shaped layer (4096 tokens, d 2048, 64 experts top-6, two
shared experts of width 1408, bf16), inputs resident in HBM.

    python bench.py [--steps K] [--warmup W] [--config NAME] [--gpus 1]

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
    if os.environ.get("FS_GEMM_TILE") not in (None, "", str(rec.get("tile", ""))):
        return None
    return rec["hbm_bytes_per_launch"]


def kernel_table(L, steps):
    names = {L.FS_K_ROUTER: "router", L.FS_K_TOPK: "topk", L.FS_K_PLAN: "plan", L.FS_K_PACK: "pack",
             L.FS_K_GATE_UP: "gate_up", L.FS_K_DOWN: "down", L.FS_K_COMBINE: "combine"}
    out = {}
    for kid, nm in names.items():
        ms, n = L.fs_profile_read(kid)
        if n:
            out[nm] = {"us_per_launch": 1e3 * ms / n, "launches": n}
    return out


def cpu_baseline(cfg, wl, sample_tokens):
    """The oracle, as it stands, on the first `sample_tokens` tokens of this
    rank: the whole block for those tokens, timed on the host."""
    import numpy as np
    import threadpoolctl

    import oracle
    f64 = lambda t: None if t is None else t.detach().float().cpu().numpy().astype(np.float64)
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
            rows = [[yr[t * cfg.top_k + j] for j in range(cfg.top_k)] for t in range(n)]
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="dsv2lite")
    ap.add_argument("--cpu-sample", type=int, default=4096,
                    help="tokens of the workload the oracle runs on the host")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--serial", action="store_true", help="no second stream")
    ap.add_argument("--rotate", type=int, default=4, help="input sets rotated across steps")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for {args.gpus})",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2511_11505_amd as fs
    from paper_2511_11505_amd import _lib as L
    from workloads import CONFIGS, make_workload
    from workloads.generate import merge_shared, source_tokens

    cfg = CONFIGS[args.config]
    dev = "cuda:0"
    torch.cuda.set_device(0)
    t_setup = time.perf_counter()
    wl = make_workload(cfg, dev)
    sh_gu = sh_dn = None
    if cfg.n_shared > 0:
        sh_gu, sh_dn = merge_shared(wl.sh_gate_up, wl.sh_down)
    blk = fs.MoEBlock(cfg, wl.w_router, wl.bias, wl.w_gate_up, wl.w_down, sh_gu, sh_dn, device=dev)
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

    def step(i):
        j = i % len(xs)
        blk.begin(xs[j], partials[j], compute=compute, comm=comm)
        blk.finish(xs[j], partials[j], compute=compute, comm=comm)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    L.fs_profile_reset()
    L.fs_profile_enable(True)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(compute)
    for i in range(args.steps):
        step(i)
    end.record(compute)
    torch.cuda.synchronize()
    L.fs_profile_enable(False)
    ms = start.elapsed_time(end) / args.steps
    kernels = kernel_table(L, args.steps)

    # roofline of the dominant kernel: the routed gate/up SwiGLU GEMM.  Its
    # algorithmic work is 2 M d 2F flops; its algorithmic HBM bytes are the
    # weights of the experts that received rows, the M input rows and the M
    # rows of H it writes.  The bound is the roof that takes longer.
    es = cfg.elem_bytes
    flops_gate_up = 2.0 * M * cfg.hidden * 2 * cfg.ffn
    lo = cfg.ep_rank * cfg.n_local
    rows_per_expert = blk.t["src_counts"][:, lo:lo + cfg.n_local].sum(0)
    active = int((rows_per_expert > 0).sum().item())
    bytes_gate_up = (active * 2 * cfg.ffn * cfg.hidden + M * cfg.hidden + M * cfg.ffn) * es
    gu = kernels.get("gate_up")
    roof = None
    if gu:
        t = gu["us_per_launch"] * 1e-6
        peak_f = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_F32_VALU_TFLOPS
        compute_bound = flops_gate_up / (peak_f * 1e12) >= bytes_gate_up / (PEAK_HBM_GBS * 1e9)
        if compute_bound:
            achieved, peak, unit = flops_gate_up / t / 1e12, peak_f, "TFLOP/s"
            bound = "mfma" if cfg.dtype == "bf16" else "alu"
        else:
            achieved, peak, unit, bound = bytes_gate_up / t / 1e9, PEAK_HBM_GBS, "GB/s", "hbm"
        roof = {"bound": bound, "kernel": "gate_up SwiGLU grouped GEMM",
                "achieved": round(achieved, 2), "peak": peak, "unit": unit,
                "frac": round(achieved / peak, 4), "traffic": measured_traffic(cfg.name),
                "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                "algorithmic_flops_per_launch": flops_gate_up,
                "algorithmic_bytes_per_launch": bytes_gate_up, "experts_with_rows": active,
                "mfma_frac": round(flops_gate_up / t / 1e12 / peak_f, 4),
                "hbm_frac": round(bytes_gate_up / t / 1e9 / PEAK_HBM_GBS, 4)}
    # permute kernels against HBM (algorithmic bytes)
    N, d, k, E = cfg.n_tokens, cfg.hidden, cfg.top_k, cfg.n_experts
    hbm = {}
    if "pack" in kernels:
        b = N * d * es + N * k * d * es + 4 * N * k
        hbm["pack"] = b / (kernels["pack"]["us_per_launch"] * 1e-6) / 1e9
    if "combine" in kernels:
        b = N * k * d * es + 8 * N * k + 2 * N * d * es
        hbm["combine"] = b / (kernels["combine"]["us_per_launch"] * 1e-6) / 1e9
    if "router" in kernels:
        flops = 2.0 * N * d * E
        kernels["router"]["tflops"] = flops / (kernels["router"]["us_per_launch"] * 1e-6) / 1e12
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
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: FarSkip MoE block forward, {N} tokens, d {d}, {E} experts "
                               f"top-{k} {cfg.score}, FFN {cfg.ffn}, {cfg.n_shared} shared, EP rank "
                               f"{cfg.ep_rank} of {cfg.ep_size}, {cfg.dtype}",
                   "tokens": N, "hidden": d, "experts": E, "top_k": k, "ffn": cfg.ffn,
                   "shared": cfg.n_shared, "ep_size": cfg.ep_size, "rows_local_experts": M,
                   "second_stream": comm is not None},
        "roofline": roof,
        "grouped_gemm_frac_bf16_peak": None if roof is None else roof["mfma_frac"],
        "permute_frac_hbm": {k2: round(v / PEAK_HBM_GBS, 4) for k2, v in hbm.items()},
        "kernels_us": {k2: round(v["us_per_launch"], 2) for k2, v in kernels.items()},
    }
    if not args.no_cpu_baseline:
        try:
            res["cpu_baseline"] = cpu_baseline(cfg, wl, args.cpu_sample)
        except Exception as e:  # report, do not hide the GPU number
            res["cpu_baseline"] = {"error": repr(e)}
    blk.close()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
