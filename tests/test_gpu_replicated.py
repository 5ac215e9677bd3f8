"""GPU parity of the replicated-activation (all-reduce) inference variant:
local rows, gathered expert GEMMs, partial Combine, the all-reduce stand-in
and the stacked FarSkip / regular schedules, against oracle.allreduce.

Integers (plan, local rows) are compared bit for bit; floating point to the
block tolerance (bf16 2e-2, fp32 1e-5 max relative error), L times it for
an L-layer stack (see tests/test_gpu_stack.py for why)."""

import numpy as np
import pytest
import torch

import oracle
from oracle import allreduce as ar
from paper_2511_11505_amd import _lib as L
from paper_2511_11505_amd.replicated import ReplicatedStack
from tests._util import TOL, f64, rel_err
from tests.test_gpu_stack import choosers
from workloads import CONFIGS, make_workload
from workloads.generate import (merge_shared, stack_layers, synthetic_topk_ids, tp_attention_slice,
                                tp_shared_slice)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]
DEV = "cuda"

# Small replicated-activation workloads: several ranks (never only rank 0),
# ragged token counts, group-limited routing, a tensor-parallel block of the
# shared experts that straddles two experts (dsv2_ar_s).
SMALL_AR = {
    "tiny_ar": CONFIGS["dsv2_ar"].scaled(
        name="tiny_ar", n_tokens=128, hidden=256, n_experts=8, top_k=2, ffn=512, n_shared=1,
        ffn_shared=256, n_groups=1, topk_groups=1, routed_scale=1.0, norm_topk=True,
        ep_size=4, ep_rank=1, dtype="f32", seed=11),
    "dsv2_ar_s": CONFIGS["dsv2_ar"].scaled(
        name="dsv2_ar_s", n_tokens=333, hidden=512, n_experts=32, ffn=256, n_shared=3,
        ffn_shared=256, ep_size=4, ep_rank=2, seed=12),
    "scout_ar_s": CONFIGS["scout_ar"].scaled(
        name="scout_ar_s", n_tokens=517, hidden=1024, ffn=384, ffn_shared=512, ep_size=4,
        ep_rank=3, seed=13),
}


class _Rows:
    """fp64 copies of single experts of a device weight tensor, on demand."""

    def __init__(self, t):
        self.t = t

    def __getitem__(self, i):
        return f64(self.t[i])


def u8(n):
    return torch.empty((max(int(n), 256),), dtype=torch.uint8, device=DEV)


def plan_and_local_rows(cfg, desc, ids):
    N, k, E, R = cfg.n_tokens, cfg.top_k, cfg.n_experts, cfg.ep_size
    i32 = dict(dtype=torch.int32, device=DEV)
    t = dict(counts=torch.empty(E, **i32), offsets=torch.empty(E + 1, **i32),
             rank_offsets=torch.empty(R + 1, **i32), s2r=torch.empty(N * k, **i32),
             r2s=torch.empty(N * k, **i32),
             local_tokens=torch.full((max(N * min(k, cfg.n_local), 1),), -7, **i32),
             local_offsets=torch.empty(cfg.n_local + 1, **i32))
    L.fs_dispatch_pack(desc, ids, None, t["counts"], t["offsets"], t["rank_offsets"], t["s2r"],
                       t["r2s"], None, u8(L.fs_workspace_size(desc, L.FS_OP_DISPATCH_PACK)))
    L.fs_local_rows(desc, t["offsets"], t["rank_offsets"], t["r2s"], t["local_tokens"],
                    t["local_offsets"])
    return t


@pytest.mark.parametrize("name,skew", [("tiny_ar", 0.0), ("dsv2_ar_s", 0.0), ("scout_ar_s", 0.0),
                                       ("dsv2_ar_s", 3.0)])
def test_local_rows_gathered_ffn_partial_combine(name, skew):
    cfg = SMALL_AR[name]
    N, k, E, R, r = cfg.n_tokens, cfg.top_k, cfg.n_experts, cfg.ep_size, cfg.ep_rank
    desc = L.make_desc(cfg)
    wl = make_workload(cfg, DEV)
    ids = synthetic_topk_ids(N, E, k, cfg.seed, DEV, skew=skew)
    g = torch.Generator(device=DEV).manual_seed(cfg.seed)
    w = torch.rand((N, k), generator=g, device=DEV, dtype=torch.float32) + 0.05
    t = plan_and_local_rows(cfg, desc, ids)
    torch.cuda.synchronize()
    ids_np = ids.cpu().numpy()
    plan = oracle.dispatch_plan(ids_np, E, R)
    for key, okey in (("counts", "counts"), ("offsets", "offsets"), ("rank_offsets", "rank_offsets"),
                      ("s2r", "slot_to_row"), ("r2s", "row_to_slot")):
        assert np.array_equal(t[key].cpu().numpy(), plan[okey]), key
    tokens, offsets = ar.local_rows(ids_np, E, R, r)
    M = len(tokens)
    assert np.array_equal(t["local_tokens"].cpu().numpy()[:M], tokens)
    assert np.array_equal(t["local_offsets"].cpu().numpy(), offsets)
    # entries past M_r are left alone
    assert (t["local_tokens"].cpu().numpy()[M:] == -7).all()

    max_rows = N * min(k, cfg.n_local)
    y = torch.empty((max_rows, cfg.hidden), dtype=wl.x.dtype, device=DEV)
    L.fs_grouped_expert_ffn_gathered(desc, cfg.n_local, cfg.ffn, wl.x, t["local_tokens"],
                                     t["local_offsets"], max_rows, wl.w_gate_up, wl.w_down, y,
                                     u8(L.fs_workspace_size(desc, L.FS_OP_GROUPED_FFN, max_rows,
                                                            cfg.ffn)))
    part = torch.empty_like(wl.x)
    L.fs_combine_partial(desc, y, t["s2r"], t["rank_offsets"], w, part)
    torch.cuda.synchronize()
    x64 = f64(wl.x)
    gu, dn = f64(wl.w_gate_up), f64(wl.w_down)
    y_want = ar.routed_partial_rows(x64, tokens, offsets, gu, dn)
    assert rel_err(f64(y[:M]), y_want) <= TOL[cfg.dtype]
    # Rows of tokens with no local selection must be exact zeros; the
    # tolerance applies to the others (zero rows would lower the rms floor
    # of rel_err by the fraction of tokens without a local expert).
    lo, hi = r * cfg.n_local, (r + 1) * cfg.n_local
    has = ((ids_np >= lo) & (ids_np < hi)).any(axis=1)
    got = f64(part)
    assert np.array_equal(got[~has], np.zeros_like(got[~has]))
    # the partial Combine alone, on the GPU's expert rows: only its own rounding
    comb = ar.combine_partial(f64(y[:M]), tokens, offsets, ids_np, f64(w), E, R, r)
    assert rel_err(got[has], comb[has]) <= (1e-6 if cfg.dtype == "f32" else 8e-3)
    # end to end against the token-by-token definition
    want = ar.routed_partial(x64, ids_np, f64(w), E, R, r, gu, dn)
    assert rel_err(got[has], want[has]) <= TOL[cfg.dtype]


def test_rank_without_rows():
    # Every token picks experts of rank 0 only; rank 3 has no rows: empty
    # local offsets, and the partial is all zeros.
    cfg = SMALL_AR["tiny_ar"].scaled(ep_rank=3)
    desc = L.make_desc(cfg)
    N, k = cfg.n_tokens, cfg.top_k
    wl = make_workload(cfg, DEV)
    ids = torch.tensor([[0, 1] if t % 2 else [1, 0] for t in range(N)], dtype=torch.int32, device=DEV)
    t = plan_and_local_rows(cfg, desc, ids)
    max_rows = N * min(k, cfg.n_local)
    y = torch.empty((max_rows, cfg.hidden), dtype=wl.x.dtype, device=DEV)
    L.fs_grouped_expert_ffn_gathered(desc, cfg.n_local, cfg.ffn, wl.x, t["local_tokens"],
                                     t["local_offsets"], max_rows, wl.w_gate_up, wl.w_down, y,
                                     u8(L.fs_workspace_size(desc, L.FS_OP_GROUPED_FFN, max_rows,
                                                            cfg.ffn)))
    part = torch.full_like(wl.x, 3.0)
    L.fs_combine_partial(desc, y, t["s2r"], t["rank_offsets"],
                         torch.ones((N, k), dtype=torch.float32, device=DEV), part)
    torch.cuda.synchronize()
    assert np.array_equal(t["local_offsets"].cpu().numpy(), np.zeros(cfg.n_local + 1, np.int32))
    assert torch.equal(part, torch.zeros_like(part))


def test_allreduce_standin_copies_and_rejects_overlap():
    cfg = SMALL_AR["dsv2_ar_s"]
    desc = L.make_desc(cfg)
    src = torch.randn((cfg.n_tokens, cfg.hidden), device=DEV).to(torch.bfloat16)
    dst = torch.empty_like(src)
    L.fs_allreduce_standin(desc, dst, src)
    L.fs_allreduce_standin(desc, src, src)          # in place: a no-op
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    big = torch.empty((2 * cfg.n_tokens, cfg.hidden), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(L.FsError):
        L.fs_allreduce_standin(desc, big[8:], big)


def rank_layers(cfg, layers):
    """(GPU layer dicts with rank r's tensor-parallel blocks, oracle layer
    dicts with the full shared experts and attention weights)."""
    R, r = cfg.ep_size, cfg.ep_rank
    gl, ol = [], []
    np_ = lambda t: None if t is None else f64(t)
    for _, wl, w_a, w_b in layers:
        sh_gu = sh_dn = None
        if cfg.n_shared:
            sh_gu, sh_dn = tp_shared_slice(*merge_shared(wl.sh_gate_up, wl.sh_down), R, r)
        wa_r, wb_r = tp_attention_slice(w_a, w_b, R, r)
        gl.append(dict(w_router=wl.w_router, bias=wl.bias, w_gate_up=wl.w_gate_up,
                       w_down=wl.w_down, sh_gate_up=sh_gu, sh_down=sh_dn, w_a=wa_r, w_b=wb_r))
        ol.append(dict(w_router=f64(wl.w_router), bias=np_(wl.bias), w_gate_up=f64(wl.w_gate_up),
                       w_down=f64(wl.w_down), sh_gate_up=np_(wl.sh_gate_up),
                       sh_down=np_(wl.sh_down), w_a=f64(w_a), w_b=f64(w_b)))
    return gl, ol


@pytest.mark.parametrize("name,n_layers", [("tiny_ar", 3), ("dsv2_ar_s", 3), ("scout_ar_s", 2)])
def test_replicated_stack_matches_oracle(name, n_layers):
    cfg = SMALL_AR[name]
    layers = stack_layers(cfg, n_layers, DEV)
    gl, ol = rank_layers(cfg, layers)
    st = ReplicatedStack(cfg, gl, device=DEV)
    x = layers[0][1].x
    tol = TOL[cfg.dtype] * n_layers

    comm = torch.cuda.Stream()
    fs = st.farskip(x, comm=comm, keep_ids=True).clone()
    torch.cuda.synchronize()
    ids_fs = [i.cpu().numpy() for i in st.kept_ids]
    z_fs = [z.cpu().numpy() for z in st.kept_logits]
    fs_serial = st.farskip(x, comm=None).clone()
    torch.cuda.synchronize()
    assert torch.equal(fs, fs_serial)
    # the all-reduce stand-ins paced at the modelled link time copy the same bytes
    with L.standin_link(7, 153e9, 64):
        fs_link = st.farskip(x, comm=comm).clone()
        rg_link = st.regular(x).clone()
        torch.cuda.synchronize()
    assert torch.equal(fs, fs_link)
    near = []
    want_fs, _ = ar.farskip_ar_stack(cfg, f64(x), ol,
                                     ids_given=choosers(cfg, ids_fs, z_fs, ol, near))
    assert rel_err(f64(fs), want_fs) <= tol

    rg = st.regular(x, keep_ids=True).clone()
    torch.cuda.synchronize()
    ids_rg = [i.cpu().numpy() for i in st.kept_ids]
    z_rg = [z.cpu().numpy() for z in st.kept_logits]
    want_rg, _ = ar.regular_ar_stack(cfg, f64(x), ol,
                                     ids_given=choosers(cfg, ids_rg, z_rg, ol, near))
    assert rel_err(f64(rg), want_rg) <= tol
    assert torch.equal(rg, rg_link)
    print(f"[replicated {name}] (near-tie tokens, max logit difference / rms) per layer, "
          f"FarSkip then regular: {near}")
    assert rel_err(f64(fs), want_rg) > 2 * rel_err(f64(fs), want_fs)
    assert rel_err(f64(rg), want_fs) > 2 * rel_err(f64(rg), want_rg)
    st.close()


@pytest.mark.parametrize("name", ["dsv2_ar", "scout_ar"])
def test_fullsize_partial_on_sampled_tokens(name):
    # The full-size workload through the same calls the stack makes, in the
    # launch configuration the benchmark times; sampled tokens against the
    # oracle, ranks 0 and R-1.
    base = CONFIGS[name]
    for r in (0, base.ep_size - 1):
        cfg = base.scaled(ep_rank=r)
        layers = stack_layers(cfg, 1, DEV)
        gl, _ = rank_layers(cfg, layers)
        wl = layers[0][1]
        st = ReplicatedStack(cfg, gl, device=DEV)
        st._routed(wl.x, gl[0], torch.cuda.current_stream())
        torch.cuda.synchronize()
        g = np.random.default_rng(cfg.seed + r)
        all_ids = st.ids.cpu().numpy()
        lo, hi = r * cfg.n_local, (r + 1) * cfg.n_local
        local = ((all_ids >= lo) & (all_ids < hi)).any(axis=1)
        sample = np.sort(np.concatenate([g.choice(np.flatnonzero(local), 6, replace=False),
                                         g.choice(np.flatnonzero(~local), 2, replace=False)]))
        xs = f64(wl.x[torch.from_numpy(sample).to(DEV)])
        z32 = oracle.logits_routing_f32(xs.astype(np.float32), f64(wl.w_router))
        bias = None if wl.bias is None else f64(wl.bias)
        own, w_own, near, _ = oracle.route(z32, cfg.score, cfg.top_k, cfg.n_groups,
                                           cfg.topk_groups, cfg.norm_topk, cfg.routed_scale, bias)
        ids = st.ids.cpu().numpy()[sample]
        assert np.array_equal(ids[~near], own[~near])
        w = oracle.route_given(z32, ids, cfg.score, cfg.norm_topk, cfg.routed_scale)
        assert rel_err(f64(st.w)[sample], w) <= 1e-5
        want = ar.routed_partial(xs, ids, w, cfg.n_experts, cfg.ep_size, r,
                                 _Rows(wl.w_gate_up), _Rows(wl.w_down))
        got = f64(st.routed)[sample]
        has = ((ids >= lo) & (ids < hi)).any(axis=1)
        assert np.array_equal(got[~has], np.zeros_like(got[~has]))
        assert rel_err(got[has], want[has]) <= TOL[cfg.dtype]
        st.close()
        del layers, gl, st
        torch.cuda.empty_cache()
