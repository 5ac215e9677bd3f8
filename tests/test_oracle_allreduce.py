"""Pins of the oracle's replicated-activation (all-reduce) inference variant.

Each check ties oracle/allreduce.py to something it does not share code
with: the all-to-all block and stacks of oracle/moe.py (written as pack,
receive and Combine), the plan's stable sort, brute-force masks, or closed
identities (partial sums over the R ranks add up to the full terms).
"""

import numpy as np
import pytest

import oracle
from oracle import allreduce as ar


def rng(seed):
    return np.random.default_rng(seed)


def _cfg(**kw):
    from workloads.configs import MoEConfig
    base = dict(name="t", n_tokens=13, hidden=8, n_experts=6, top_k=2, ffn=4,
                score="softmax", norm_topk=False, dtype="f32", seed=0, ep_mode="allreduce")
    base.update(kw)
    return MoEConfig(**base)


def _experts(cfg, g):
    E, F, d = cfg.n_experts, cfg.ffn, cfg.hidden
    gu = 0.3 * g.standard_normal((E, 2 * F, d))
    dn = 0.3 * g.standard_normal((E, d, F))
    return gu, dn


def _routing(cfg, x, wr, bias=None):
    z = oracle.logits_routing_f32(x, wr)
    ids, w, _, _ = oracle.route(z, cfg.score, cfg.top_k, cfg.n_groups, cfg.topk_groups,
                                cfg.norm_topk, cfg.routed_scale, bias)
    return ids, w


def _case(cfg, seed):
    g = rng(seed)
    x = g.standard_normal((cfg.n_tokens, cfg.hidden)).astype(np.float32)
    wr = (0.5 * g.standard_normal((cfg.n_experts, cfg.hidden))).astype(np.float32)
    gu, dn = _experts(cfg, g)
    ids, w = _routing(cfg, x, wr)
    return x, wr, gu, dn, ids, w


@pytest.mark.parametrize("R", [1, 2, 3, 6])
def test_local_rows_are_the_plans_rank_blocks(R):
    # Rank r's rows are the plan's rows [rank_offsets[r], rank_offsets[r+1])
    # (stable sort by expert), read back to their tokens.
    cfg = _cfg(ep_size=R, n_tokens=29, top_k=3)
    _, _, _, _, ids, _ = _case(cfg, 1)
    plan = oracle.dispatch_plan(ids, cfg.n_experts, R)
    total = 0
    for r in range(R):
        tokens, offsets = ar.local_rows(ids, cfg.n_experts, R, r)
        lo, hi = plan["rank_offsets"][r], plan["rank_offsets"][r + 1]
        assert np.array_equal(tokens, plan["row_to_slot"][lo:hi] // cfg.top_k)
        e0 = r * cfg.n_local
        assert np.array_equal(offsets, plan["offsets"][e0:e0 + cfg.n_local + 1] - lo)
        total += len(tokens)
    assert total == cfg.n_tokens * cfg.top_k


@pytest.mark.parametrize("kw", [dict(ep_size=3), dict(ep_size=2, score="sigmoid", norm_topk=True),
                                dict(ep_size=6, top_k=3)])
def test_routed_partials_sum_to_the_block(kw):
    # The all-reduce of the R ranks' partial sums is the whole routed MoE
    # output, as the all-to-all block computes it on one rank owning every
    # expert (plan, pack, grouped experts, Combine).
    cfg = _cfg(**kw)
    x, wr, gu, dn, _, _ = _case(cfg, 2)
    full = _cfg(**{**kw, "ep_size": 1, "ep_mode": "a2a"})
    blk = oracle.moe_block(full, x[None], wr, None, gu, dn)
    ids, w = blk["me"]["ids"], blk["me"]["w"]
    E_loc = cfg.n_local
    total = sum(ar.routed_partial(x, ids, w, cfg.n_experts, cfg.ep_size, r,
                                  gu[r * E_loc:(r + 1) * E_loc], dn[r * E_loc:(r + 1) * E_loc])
                for r in range(cfg.ep_size))
    assert np.allclose(total, blk["routed"], rtol=1e-12, atol=1e-12)


def test_routed_partial_is_zero_for_tokens_without_local_experts():
    cfg = _cfg(ep_size=3, n_tokens=4)
    g = rng(3)
    x = g.standard_normal((4, cfg.hidden))
    gu, dn = _experts(cfg, g)
    ids = np.array([[2, 3], [0, 5], [4, 1], [3, 2]], np.int32)   # rank 1 owns experts 2, 3
    w = np.abs(g.standard_normal((4, 2))) + 0.1
    part = ar.routed_partial(x, ids, w, 6, 3, 1, gu[2:4], dn[2:4])
    assert np.array_equal(part[1], np.zeros(cfg.hidden))
    assert np.array_equal(part[2], np.zeros(cfg.hidden))
    # token 0 selects both local experts: the sum of the two weighted outputs
    want = sum(w[0, j] * oracle.swiglu(x[0:1], gu[ids[0, j]], dn[ids[0, j]])[0] for j in range(2))
    assert np.allclose(part[0], want, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("R,r", [(1, 0), (3, 0), (3, 2), (6, 4)])
def test_grouped_rows_then_partial_combine_is_the_partial(R, r):
    # The grouped formulation (rows of each local expert, then a Combine
    # restricted to local selections) equals the token-by-token definition.
    cfg = _cfg(ep_size=R, n_tokens=31, top_k=3)
    x, _, gu, dn, ids, w = _case(cfg, 4)
    E_loc = cfg.n_local
    gu_r, dn_r = gu[r * E_loc:(r + 1) * E_loc], dn[r * E_loc:(r + 1) * E_loc]
    tokens, offsets = ar.local_rows(ids, cfg.n_experts, R, r)
    y = ar.routed_partial_rows(x, tokens, offsets, gu_r, dn_r)
    got = ar.combine_partial(y, tokens, offsets, ids, w, cfg.n_experts, R, r)
    want = ar.routed_partial(x, ids, w, cfg.n_experts, R, r, gu_r, dn_r)
    assert np.allclose(got, want, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("S,Fs,R", [(2, 6, 3), (2, 6, 4), (1, 8, 8), (3, 4, 2)])
def test_shared_partials_sum_to_the_shared_experts(S, Fs, R):
    # Splitting the merged hidden units over R ranks (blocks may straddle
    # two experts) and adding the partials gives the S shared experts' sum.
    g = rng(5)
    d = 8
    x = g.standard_normal((7, d))
    sh_gu = 0.3 * g.standard_normal((S, 2 * Fs, d))
    sh_dn = 0.3 * g.standard_normal((S, d, Fs))
    total = sum(ar.shared_partial(x, sh_gu, sh_dn, R, r) for r in range(R))
    assert np.allclose(total, oracle.shared_ffn(x, sh_gu, sh_dn), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("R", [1, 2, 4])
def test_attention_partials_sum_to_the_stand_in(R):
    g = rng(6)
    d = 8
    p = g.standard_normal((5, d))
    lw = dict(w_a=g.standard_normal((d, d)), w_b=g.standard_normal((d, d)))
    total = sum(ar.attention_partial(p, lw["w_a"], lw["w_b"], R, r) for r in range(R))
    assert np.allclose(total, oracle.attention_stand_in(p, lw), rtol=1e-12, atol=1e-12)


def _layers(cfg, g, L, rank_experts=True, zero_down=False, shared=True):
    d = cfg.hidden
    layers = []
    for _ in range(L):
        wr = (0.5 * g.standard_normal((cfg.n_experts, d))).astype(np.float32)
        gu, dn = _experts(cfg, g)
        if zero_down:
            dn[:] = 0
        lo = cfg.ep_rank * cfg.n_local
        if rank_experts:
            gu, dn = gu[lo:lo + cfg.n_local], dn[lo:lo + cfg.n_local]
        lw = dict(w_router=wr, bias=None, w_gate_up=gu, w_down=dn,
                  w_a=0.4 * g.standard_normal((d, d)), w_b=0.4 * g.standard_normal((d, d)))
        if shared and cfg.n_shared:
            lw["sh_gate_up"] = 0.3 * g.standard_normal((cfg.n_shared, 2 * cfg.ffn_shared, d))
            lw["sh_down"] = 0.3 * g.standard_normal((cfg.n_shared, d, cfg.ffn_shared))
        layers.append(lw)
    return layers


@pytest.mark.parametrize("kw", [dict(), dict(n_shared=2, ffn_shared=4, score="sigmoid", norm_topk=True)])
def test_one_rank_stacks_are_the_all_to_all_stacks(kw):
    # With R = 1 every partial is the full term and the all-reduce is the
    # identity: the variant's FarSkip and regular stacks are those of the
    # all-to-all formulation (Eqs. 6-8), up to the order of fp64 additions.
    cfg = _cfg(ep_size=1, **kw)
    g = rng(7)
    x = g.standard_normal((cfg.n_tokens, cfg.hidden))
    layers = _layers(cfg, g, 3)
    a2a = _cfg(ep_size=1, ep_mode="a2a", **kw)
    o_ar, t_ar = ar.farskip_ar_stack(cfg, x, layers)
    o_a2a, t_a2a = oracle.farskip_stack(a2a, x, layers)
    assert np.allclose(o_ar, o_a2a, rtol=1e-12, atol=1e-12)
    assert all(np.array_equal(a["ids"], b["ids"]) for a, b in zip(t_ar, t_a2a))
    r_ar, _ = ar.regular_ar_stack(cfg, x, layers)
    r_a2a, _ = oracle.regular_stack(a2a, x, layers)
    assert np.allclose(r_ar, r_a2a, rtol=1e-12, atol=1e-12)
    assert not np.allclose(o_ar, r_ar)


def test_ar_stack_conservation():
    # Eq. 7 on one rank: the final residual minus the input is the sum of
    # every layer's attention, shared and routed partials, each once.
    cfg = _cfg(ep_size=2, ep_rank=1, n_shared=1, ffn_shared=6)
    g = rng(8)
    x = g.standard_normal((cfg.n_tokens, cfg.hidden))
    layers = _layers(cfg, g, 4)
    o, terms = ar.farskip_ar_stack(cfg, x, layers)
    total = sum(t["attn"] + t["shared"] + t["routed"] for t in terms)
    assert np.allclose(o - x, total, rtol=1e-12, atol=1e-12)
    assert all(t["routed"].any() for t in terms)


def test_ar_stack_zero_moe_output_equals_regular():
    cfg = _cfg(ep_size=3, ep_rank=2)
    g = rng(9)
    x = g.standard_normal((cfg.n_tokens, cfg.hidden))
    layers = _layers(cfg, g, 3, zero_down=True)
    fs, _ = ar.farskip_ar_stack(cfg, x, layers)
    rg, _ = ar.regular_ar_stack(cfg, x, layers)
    assert np.array_equal(fs, rg)


def test_ar_stack_attention_does_not_see_the_previous_routed_output():
    # The dependency FarSkip drops: layer 1's attention partial does not
    # change with layer 0's routed experts; layer 1's routed partial does.
    cfg = _cfg(ep_size=2, ep_rank=0)
    g = rng(10)
    x = g.standard_normal((cfg.n_tokens, cfg.hidden))
    layers = _layers(cfg, g, 2)
    other = [dict(lw) for lw in layers]
    other[0]["w_down"] = 2.0 * layers[0]["w_down"]
    _, t1 = ar.farskip_ar_stack(cfg, x, layers)
    _, t2 = ar.farskip_ar_stack(cfg, x, other)
    assert np.array_equal(t1[1]["attn"], t2[1]["attn"])
    assert not np.allclose(t1[1]["routed"], t2[1]["routed"])
    _, r1 = ar.regular_ar_stack(cfg, x, layers)
    _, r2 = ar.regular_ar_stack(cfg, x, other)
    assert not np.allclose(r1[1]["attn"], r2[1]["attn"])
