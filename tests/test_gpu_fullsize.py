"""GPU parity at the full sizes of the five workloads, in the launch
configuration bench.py times (two streams, BEGIN then FINISH), on outputs the
oracle computes one by one:

* router logits of sampled tokens, bit for bit;
* routing ids of every token (non-near-tie tokens bit for bit) and the whole
  dispatch plan bit for bit, from the oracle's routing of all tokens;
* the block's residual and partial outputs of sampled tokens, with every
  local expert evaluated in fp64 and the other ranks' rows taken from the
  return buffer at the oracle's plan positions.
"""

import numpy as np
import pytest
import torch

import oracle
from paper_2511_11505_amd import MoEBlock, prepare_remote_sources
from tests._util import TOL, f64, rel_err
from workloads import CONFIGS, make_workload
from workloads.generate import merge_shared

pytestmark = [pytest.mark.gpu, pytest.mark.slow,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]
DEV = "cuda"
N_SAMPLE = 10


def sample_tokens(N, n, seed):
    g = np.random.default_rng(seed)
    picks = set([0, N - 1]) | set(g.choice(N, size=min(n, N), replace=False).tolist())
    return np.array(sorted(picks))[:max(n, 2)]


def check_valid_choice(cfg, z, bias, ids, tau=1e-6):
    """A selection that a rounding within tau could produce: distinct ids, at
    most topk_groups groups, each selected key within tau of the k-th best
    key of its allowed set."""
    k, E = cfg.top_k, cfg.n_experts
    assert len(set(ids.tolist())) == k and all(0 <= e < E for e in ids)
    zz = np.asarray(z, np.float64)
    keys = zz if cfg.score == "softmax" else 1 / (1 + np.exp(-zz)) + (0 if bias is None else bias)
    if cfg.n_groups > 1:
        gsz = E // cfg.n_groups
        groups = set(int(e) // gsz for e in ids)
        assert len(groups) <= cfg.topk_groups
        gs = np.sort(keys.reshape(cfg.n_groups, gsz), axis=1)[:, -2:].sum(1)
        gbest = np.sort(gs)[::-1][cfg.topk_groups - 1]
        assert all(gs[g] >= gbest - 2 * tau for g in groups)
        allowed = np.concatenate([keys[g * gsz:(g + 1) * gsz] for g in groups])
    else:
        allowed = keys
    kth = np.sort(allowed)[::-1][k - 1]
    assert all(keys[e] >= kth - 2 * tau for e in ids)


@pytest.mark.parametrize("name", ["tiny", "dsv2lite", "scout", "dsv3_prefill", "dsv3_decode"])
def test_fullsize_block(name):
    cfg = CONFIGS[name]
    wl = make_workload(cfg, DEV)
    sh_gu = sh_dn = None
    if cfg.n_shared > 0:
        sh_gu, sh_dn = merge_shared(wl.sh_gate_up, wl.sh_down)
    blk = MoEBlock(cfg, wl.w_router, wl.bias, wl.w_gate_up, wl.w_down, sh_gu, sh_dn, device=DEV)
    if cfg.ep_size > 1:
        blk.set_max_recv_rows(prepare_remote_sources(blk, wl.x_all, wl.w_router, wl.bias, wl.y_remote))
    comm = torch.cuda.Stream()
    x = wl.x
    partial = torch.empty_like(x)
    blk.begin(x, partial, comm=comm)
    blk.finish(x, partial, comm=comm)     # residual_io = partial: x + shared + routed
    torch.cuda.synchronize()
    out = partial

    N, k, E = cfg.n_tokens, cfg.top_k, cfg.n_experts
    # routing of every token in the routing precision, then the plan
    xs32 = f64(x).astype(np.float32)
    wr32 = f64(wl.w_router).astype(np.float32)
    z_ref = oracle.logits_routing_f32(xs32, wr32)
    bias = None if wl.bias is None else f64(wl.bias)
    ids_ref, w_ref, near, _ = oracle.route(z_ref, cfg.score, k, cfg.n_groups, cfg.topk_groups,
                                           cfg.norm_topk, cfg.routed_scale, bias)
    z_gpu = blk.t["logits"].cpu().numpy()
    samp = sample_tokens(N, N_SAMPLE, cfg.seed)
    assert np.array_equal(z_gpu[samp], z_ref[samp]), "router logits differ bitwise"
    assert np.array_equal(z_gpu, z_ref), "router logits differ bitwise"
    ids_gpu = blk.t["topk_ids"].cpu().numpy()
    assert np.array_equal(ids_gpu[~near], ids_ref[~near])
    # near ties: a sanity bound on their count (each token has about a dozen
    # rounded decisions with gaps of order 1e-2, so a few per thousand), and
    # every GPU choice there must still be a valid top-k within the margin
    assert near.sum() <= max(2, N // 200), f"{near.sum()} near-tie tokens"
    for t in np.where(near)[0]:
        check_valid_choice(cfg, z_ref[t], bias, ids_gpu[t])
    assert rel_err(blk.t["topk_w"].cpu().numpy()[~near], w_ref[~near]) <= 2e-6
    plan = oracle.dispatch_plan(ids_ref, E, cfg.ep_size)
    if np.array_equal(ids_gpu, ids_ref):
        assert np.array_equal(blk.t["slot_to_row"].cpu().numpy(), plan["slot_to_row"])
        assert np.array_equal(blk.t["rank_offsets"].cpu().numpy(), plan["rank_offsets"])
        r = cfg.ep_rank
        assert np.array_equal(blk.t["src_counts"][r].cpu().numpy(), plan["counts"])
        assert np.array_equal(blk.t["src_offsets"][r].cpu().numpy(), plan["offsets"])

    # outputs of sampled tokens (skipping near ties, whose experts may differ).
    # With R > 1 the rows returned by other ranks sit at plan positions; if a
    # near tie changed any id, those positions can shift, so only tokens whose
    # experts are all local are compared then.
    samp = np.array([t for t in samp if not near[t]])
    if cfg.ep_size > 1 and not np.array_equal(ids_gpu, ids_ref):
        lo, hi = cfg.ep_rank * cfg.n_local, (cfg.ep_rank + 1) * cfg.n_local
        samp = np.array([t for t in samp if np.all((ids_ref[t] >= lo) & (ids_ref[t] < hi))])
        if samp.size == 0:
            pytest.skip("near ties moved the return rows of every sampled token")
    xs = f64(x)[samp]
    cache = {}

    def expert(e_local):
        if e_local not in cache:
            cache[e_local] = (f64(wl.w_gate_up[e_local]), f64(wl.w_down[e_local]))
        return cache[e_local]

    yr = None if wl.y_remote is None else f64(wl.y_remote)
    remote = [[yr[plan["slot_to_row"][t * k + j]] if yr is not None else None for j in range(k)]
              for t in samp]
    routed = oracle.moe_tokens_direct(cfg, xs, ids_ref[samp], w_ref[samp], expert, remote)
    shared = np.zeros_like(xs)
    if cfg.n_shared > 0:
        shared = oracle.shared_ffn(xs, f64(wl.sh_gate_up), f64(wl.sh_down))
    want = oracle.residual_add(xs, shared, routed)
    tol = TOL[cfg.dtype]
    assert rel_err(f64(out)[samp], want) <= tol
    blk.close()


@pytest.mark.parametrize("name", ["dsv2lite", "dsv3_prefill", "dsv3_decode"])
def test_fullsize_block_fp8(name):
    """The block with FP8 routed experts (FP8 dispatch) at full size: the
    residual output of sampled tokens against the oracle's FP8 experts (its
    own E4M3 quantisation of the bf16 weights and of each token row, H
    rounded to bf16 and quantised per row), shared experts in bf16."""
    from oracle import fp8 as of8
    cfg = CONFIGS[name]
    wl = make_workload(cfg, DEV)
    sh_gu = sh_dn = None
    if cfg.n_shared > 0:
        sh_gu, sh_dn = merge_shared(wl.sh_gate_up, wl.sh_down)
    blk = MoEBlock(cfg, wl.w_router, wl.bias, wl.w_gate_up, wl.w_down, sh_gu, sh_dn, device=DEV,
                   fp8="routed")
    if cfg.ep_size > 1:
        blk.set_max_recv_rows(prepare_remote_sources(blk, wl.x_all, wl.w_router, wl.bias, wl.y_remote))
    comm = torch.cuda.Stream()
    x = wl.x
    partial = torch.empty_like(x)
    blk.begin(x, partial, comm=comm)
    blk.finish(x, partial, comm=comm)
    torch.cuda.synchronize()

    N, k, E = cfg.n_tokens, cfg.top_k, cfg.n_experts
    z_ref = oracle.logits_routing_f32(f64(x).astype(np.float32), f64(wl.w_router).astype(np.float32))
    bias = None if wl.bias is None else f64(wl.bias)
    ids_ref, w_ref, near, _ = oracle.route(z_ref, cfg.score, k, cfg.n_groups, cfg.topk_groups,
                                           cfg.norm_topk, cfg.routed_scale, bias)
    ids_gpu = blk.t["topk_ids"].cpu().numpy()
    assert np.array_equal(ids_gpu[~near], ids_ref[~near])
    # the plan of the GPU's own selection, bit for bit; the rows other ranks
    # return sit at its positions, so near ties elsewhere do not matter
    plan = oracle.dispatch_plan(ids_gpu, E, cfg.ep_size)
    assert np.array_equal(blk.t["slot_to_row"].cpu().numpy(), plan["slot_to_row"])
    samp = np.array([t for t in sample_tokens(N, 3, cfg.seed + 1) if not near[t]])
    lo = cfg.ep_rank * cfg.n_local
    yr = None if wl.y_remote is None else f64(wl.y_remote)
    cache = {}

    def fp8_expert(el):
        if el not in cache:
            gq, gs = of8.quantize_rows(f64(wl.w_gate_up[el]).astype(np.float32))
            dq, ds = of8.quantize_rows(f64(wl.w_down[el]).astype(np.float32))
            cache[el] = (gq, gs, dq, ds)
        return cache[el]

    xs = f64(x)[samp]
    routed = np.zeros_like(xs)
    for i, t in enumerate(samp):
        for j in range(k):
            e = int(ids_ref[t, j])
            if lo <= e < lo + cfg.n_local:
                y = of8.swiglu_fp8(xs[i:i + 1], *fp8_expert(e - lo))[0][0]
            else:
                y = yr[plan["slot_to_row"][t * k + j]]
            routed[i] += w_ref[t, j] * y
    shared = np.zeros_like(xs)
    if cfg.n_shared > 0:
        shared = oracle.shared_ffn(xs, f64(wl.sh_gate_up), f64(wl.sh_down))
    want = oracle.residual_add(xs, shared, routed)
    assert rel_err(f64(partial)[samp], want) <= TOL["bf16"]
    blk.close()
