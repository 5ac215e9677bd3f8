"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Every check here compares the oracle with something other than itself: a
hand-derived value, a closed form, an exact integer result, a library routine
(stable argsort, bincount, scipy softmax), brute force over subsets, or an
invariant of the FarSkip residual (Section 3, Eqs. 6-8).  The paper prints no
worked numeric example for the block, so there is no printed fixture.
"""

import itertools
import math

import numpy as np
import pytest
import scipy.special

import oracle


def rng(seed):
    return np.random.default_rng(seed)


def bf16_values(a):
    """Round fp32 values to bf16-representable fp32 values (RNE)."""
    u = np.asarray(a, np.float32).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32)


# ---------------------------------------------------------------- O1 logits
def test_routing_logits_exact_on_integers():
    # Small integers: every partial sum is an integer below 2^24, so the fp32
    # order-fixed sum must equal the exact integer matmul, for a d that is not
    # a multiple of the slice length (ragged last slice).
    g = rng(0)
    x = g.integers(-8, 9, size=(5, 700)).astype(np.float32)
    w = g.integers(-8, 9, size=(7, 700)).astype(np.float32)
    exact = x.astype(np.int64) @ w.astype(np.int64).T
    z = oracle.logits_routing_f32(x, w)
    assert np.array_equal(z.astype(np.int64), exact)
    assert np.array_equal(oracle.logits_f64(x, w), exact.astype(np.float64))


def test_routing_logits_order_hand_value():
    # d = 512 = two slices.  Slice 0 holds 2^24 followed by 255 ones: every
    # fp32 add of 1 to 2^24 rounds back to 2^24 (tie to even), so slice 0
    # sums to 2^24.  Slice 1 holds 256 ones and sums to 256 exactly.  The
    # final add gives 2^24 + 256, which is representable.  The exact sum
    # would be 2^24 + 511.
    x = np.ones((1, 512), np.float32)
    w = np.ones((1, 512), np.float32)
    w[0, 0] = 2.0 ** 24
    z = oracle.logits_routing_f32(x, w)
    assert z[0, 0] == np.float32(16777472.0)
    assert oracle.logits_f64(x, w)[0, 0] == 16777216.0 + 511.0


def test_routing_logits_error_bound():
    # Recursive-summation error bound: each product rounds once and passes
    # through at most (slice - 1) + n_slices additions.
    g = rng(1)
    d = 2048 + 192
    x = bf16_values(g.standard_normal((16, d)))
    w = bf16_values(0.02 * g.standard_normal((24, d)))
    z32 = oracle.logits_routing_f32(x, w).astype(np.float64)
    z64 = oracle.logits_f64(x, w)
    n_add = oracle.ROUTER_SLICE + math.ceil(d / oracle.ROUTER_SLICE) + 1
    u = 2.0 ** -24
    bound = 1.01 * n_add * u * (np.abs(x.astype(np.float64)) @ np.abs(w.astype(np.float64)).T)
    assert np.all(np.abs(z32 - z64) <= bound)


# ---------------------------------------------------------------- O2-O6 route
def test_route_sigmoid_hand_example():
    # z = [0, ln 3, -ln 3, ln 7] -> sigmoid = [1/2, 3/4, 1/4, 7/8].
    z = np.array([[0.0, math.log(3), -math.log(3), math.log(7)]])
    ids, w, near, _ = oracle.route(z, "sigmoid", 2, norm_topk=False)
    assert ids.tolist() == [[3, 1]]
    assert np.allclose(w, [[7 / 8, 3 / 4]], rtol=0, atol=1e-15)
    ids, w, near, _ = oracle.route(z, "sigmoid", 2, norm_topk=True, routed_scale=2.5)
    assert np.allclose(w, [[2.5 * 7 / 13, 2.5 * 6 / 13]], rtol=0, atol=1e-15)
    assert not near.any()


def test_route_bias_changes_selection_not_weights():
    z = np.array([[2.0, 1.0, 0.0, -1.0]])
    bias = np.array([0.0, 0.0, 0.0, 5.0])
    ids, w, _, _ = oracle.route(z, "sigmoid", 1, bias=bias)
    assert ids.tolist() == [[3]]
    assert w[0, 0] == pytest.approx(1.0 / (1.0 + math.exp(1.0)), abs=1e-15)


def test_route_softmax_weights_and_ties():
    g = rng(2)
    z = g.standard_normal((9, 6)).astype(np.float32)
    # k = E, no renormalisation: weights are the softmax over all experts,
    # checked against scipy's softmax.
    ids, w, near, _ = oracle.route(z, "softmax", 6)
    p = scipy.special.softmax(z.astype(np.float64), axis=1)
    assert np.allclose(np.take_along_axis(p, ids.astype(np.int64), axis=1), w, atol=1e-15)
    assert np.allclose(w.sum(1), 1.0, atol=1e-14)
    assert not near.any()
    # equal logits: the lower expert index wins and comes first
    zt = np.array([[0.5, 1.0, 1.0, 1.0, -2.0]], np.float32)
    ids, _, _, _ = oracle.route(zt, "softmax", 2)
    assert ids.tolist() == [[1, 2]]


def _brute_route(keys, k, G, tg):
    """Selection by exhaustive search: the kept groups are the tg-subset of
    groups with the largest total group score, where a group's score is the
    largest sum over pairs of its keys; the selected experts are the k-subset
    of allowed experts with the largest key sum; slot order by key."""
    E = len(keys)
    gsz = E // G
    if G > 1:
        def gscore(gi):
            ks = keys[gi * gsz:(gi + 1) * gsz]
            return max(a + b for a, b in itertools.combinations(ks, 2)) if gsz >= 2 else ks[0]
        gs = [gscore(gi) for gi in range(G)]
        best = max(itertools.combinations(range(G), tg), key=lambda c: sum(gs[i] for i in c))
        allowed = [e for e in range(E) if e // gsz in best]
    else:
        allowed = list(range(E))
    sel = max(itertools.combinations(allowed, k), key=lambda c: sum(keys[e] for e in c))
    return sorted(sel, key=lambda e: -keys[e])


@pytest.mark.parametrize("score,G,tg,k", [("softmax", 1, 1, 3), ("sigmoid", 1, 1, 2),
                                          ("sigmoid", 4, 2, 3), ("softmax", 3, 1, 2),
                                          ("sigmoid", 2, 1, 1)])
def test_route_matches_brute_force(score, G, tg, k):
    g = rng(3)
    E = 12
    bias = 0.3 * g.standard_normal(E) if score == "sigmoid" else None
    for _ in range(40):
        z = g.standard_normal((1, E))
        ids, _, near, _ = oracle.route(z, score, k, G, tg, bias=bias)
        keys = z[0] if score == "softmax" else 1 / (1 + np.exp(-z[0])) + bias
        assert ids[0].tolist() == _brute_route(list(keys), k, G, tg)
        assert not near.any()


def test_route_flags_near_ties():
    z = np.array([[0.3, 0.3 + 1e-9, -1.0]])
    _, _, near, margin = oracle.route(z, "sigmoid", 1)
    assert near[0] and margin[0] < 1e-6
    _, _, near, _ = oracle.route(np.array([[0.3, 0.9, -1.0]]), "sigmoid", 1)
    assert not near[0]


# ---------------------------------------------------------------- O7-O8 plan/pack
def test_plan_hand_example():
    ids = np.array([[1, 0], [0, 2], [1, 2]])
    p = oracle.dispatch_plan(ids, 3, ep_size=3)
    assert p["counts"].tolist() == [2, 2, 2]
    assert p["offsets"].tolist() == [0, 2, 4, 6]
    assert p["slot_to_row"].tolist() == [2, 0, 1, 4, 3, 5]
    assert p["row_to_slot"].tolist() == [1, 2, 0, 4, 3, 5]
    assert p["rank_offsets"].tolist() == [0, 2, 4, 6]


@pytest.mark.parametrize("N,E,k,R", [(1, 4, 1, 1), (37, 16, 4, 4), (200, 64, 6, 8), (5, 8, 8, 2)])
def test_plan_is_stable_sort_and_bijection(N, E, k, R):
    g = rng(N + E)
    ids = np.stack([g.choice(E, size=k, replace=False) for _ in range(N)])
    p = oracle.dispatch_plan(ids, E, R)
    flat = ids.reshape(-1)
    assert np.array_equal(p["counts"], np.bincount(flat, minlength=E))
    assert np.array_equal(p["offsets"], np.concatenate([[0], np.cumsum(np.bincount(flat, minlength=E))]))
    assert np.array_equal(p["row_to_slot"], np.argsort(flat, kind="stable"))
    assert np.array_equal(np.sort(p["slot_to_row"]), np.arange(N * k))
    assert np.array_equal(p["row_to_slot"][p["slot_to_row"]], np.arange(N * k))
    assert np.array_equal(p["rank_offsets"], p["offsets"][::E // R])
    x = g.standard_normal((N, 3))
    send = oracle.pack(x, p["slot_to_row"], k)
    assert np.array_equal(send, x[np.argsort(flat, kind="stable") // k])


# ---------------------------------------------------------------- O9 receive
def test_receive_rows_decomposition():
    g = rng(5)
    R, N, E, k, r = 4, 19, 16, 3, 2
    E_loc, cap = E // R, N * k
    plans, ids_all = [], []
    for s in range(R):
        ids = np.stack([g.choice(E, size=k, replace=False) for _ in range(N)])
        ids_all.append(ids)
        plans.append(oracle.dispatch_plan(ids, E, R))
    rows, goff = oracle.receive_rows(np.stack([p["counts"] for p in plans]),
                                     np.stack([p["offsets"] for p in plans]), cap, r, E_loc)
    # brute force: scan every source's slots in (source, token) order
    for e in range(E_loc):
        want = []
        for s in range(R):
            for t in range(N):
                for j in range(k):
                    if ids_all[s][t, j] == r * E_loc + e:
                        want.append(s * cap + plans[s]["slot_to_row"][t * k + j])
        assert rows[goff[e]:goff[e + 1]].tolist() == want


# ---------------------------------------------------------------- O10 SwiGLU
def test_swiglu_scalar_and_roles():
    # d = F = 1: x = 2, gate 1, up 3, down 0.5 -> SiLU(2) * 6 * 0.5
    y = oracle.swiglu([[2.0]], [[1.0], [3.0]], [[0.5]])
    assert y[0, 0] == pytest.approx(3.0 * 2.0 / (1.0 + math.exp(-2.0)), rel=1e-15)
    assert oracle.silu([1.0])[0] == pytest.approx(0.7310585786300049, rel=1e-15)
    assert oracle.silu([0.0])[0] == 0.0
    assert oracle.silu([-800.0])[0] == 0.0


def test_swiglu_identity_weights():
    g = rng(6)
    d = 5
    x = g.standard_normal((4, d))
    gu = np.concatenate([np.eye(d), np.eye(d)])
    y = oracle.swiglu(x, gu, np.eye(d))
    assert np.allclose(y, x * x / (1 + np.exp(-x)), rtol=1e-14, atol=0)
    # a permuted down projection moves output columns
    P = np.eye(d)[::-1]
    assert np.allclose(oracle.swiglu(x, gu, P), (x * x / (1 + np.exp(-x)))[:, ::-1], rtol=1e-14)


# ---------------------------------------------------------------- whole block
def _tiny_cfg(**kw):
    from workloads.configs import MoEConfig
    base = dict(name="t", n_tokens=11, hidden=8, n_experts=6, top_k=2, ffn=4,
                score="softmax", norm_topk=False, dtype="f32", seed=0, next_linear=True)
    base.update(kw)
    return MoEConfig(**base)


def _tiny_inputs(cfg, g):
    R, N, d, E, F = cfg.ep_size, cfg.n_tokens, cfg.hidden, cfg.n_experts, cfg.ffn
    x_all = g.standard_normal((R, N, d)).astype(np.float32)
    wr = (0.5 * g.standard_normal((E, d))).astype(np.float32)
    gu = (0.3 * g.standard_normal((cfg.n_local, 2 * F, d))).astype(np.float32)
    dn = (0.3 * g.standard_normal((cfg.n_local, d, F))).astype(np.float32)
    bias = (0.1 * g.standard_normal(E)).astype(np.float32) if cfg.score == "sigmoid" else None
    yr = g.standard_normal((cfg.cap, d)).astype(np.float32) if R > 1 else None
    return x_all, wr, bias, gu, dn, yr


@pytest.mark.parametrize("kw", [dict(), dict(score="sigmoid", norm_topk=True),
                                dict(score="sigmoid", n_groups=3, topk_groups=2, top_k=3),
                                dict(ep_size=3, ep_rank=1), dict(ep_size=2, ep_rank=0, score="sigmoid")])
def test_block_packed_equals_dense_masked(kw):
    # P6: evaluate every expert on every token and mask by the selection;
    # no plan, no pack.  Remote experts' rows come from the return buffer.
    cfg = _tiny_cfg(**kw)
    g = rng(7)
    x_all, wr, bias, gu, dn, yr = _tiny_inputs(cfg, g)
    out = oracle.moe_block(cfg, x_all, wr, bias, gu, dn, y_remote=yr)
    me = out["me"]
    x = x_all[cfg.ep_rank].astype(np.float64)
    dense = np.zeros_like(x)
    lo = cfg.ep_rank * cfg.n_local
    for t in range(cfg.n_tokens):
        for j in range(cfg.top_k):
            e = me["ids"][t, j]
            if lo <= e < lo + cfg.n_local:
                ye = (oracle.silu(x[t] @ gu[e - lo][:cfg.ffn].T) * (x[t] @ gu[e - lo][cfg.ffn:].T)) @ dn[e - lo].T
            else:
                ye = yr[me["plan"]["slot_to_row"][t * cfg.top_k + j]]
            dense[t] += me["w"][t, j] * ye
    assert np.allclose(out["routed"], dense, rtol=1e-12, atol=1e-12)


def test_block_ep_decomposition():
    # P8: the R-rank path gives each received row the output of its expert
    # applied to the token that sent it.
    cfg = _tiny_cfg(ep_size=3, ep_rank=2, n_experts=6)
    g = rng(8)
    x_all, wr, bias, gu, dn, yr = _tiny_inputs(cfg, g)
    out = oracle.moe_block(cfg, x_all, wr, bias, gu, dn, y_remote=yr)
    for e in range(cfg.n_local):
        for row in out["group_rows"][out["group_offsets"][e]:out["group_offsets"][e + 1]]:
            s, pos = divmod(int(row), cfg.cap)
            slot = out["src"][s]["plan"]["row_to_slot"][pos]
            t = slot // cfg.top_k
            assert out["src"][s]["ids"][t, slot % cfg.top_k] == cfg.ep_rank * cfg.n_local + e
            want = oracle.swiglu(x_all[s][t:t + 1], gu[e], dn[e])[0]
            assert np.allclose(out["y"][row], want, rtol=1e-13, atol=1e-13)


def test_dense_mixture_special_case():
    # P7: k = E with softmax and no renormalisation is the dense mixture
    # sum_e p_e MLP_e(x) with p the softmax over all experts.
    cfg = _tiny_cfg(top_k=6)
    g = rng(9)
    x_all, wr, _, gu, dn, _ = _tiny_inputs(cfg, g)
    out = oracle.moe_block(cfg, x_all, wr, None, gu, dn)
    x = x_all[0].astype(np.float64)
    p = scipy.special.softmax(oracle.logits_routing_f32(x_all[0], wr).astype(np.float64), axis=1)
    want = sum(p[:, e:e + 1] * oracle.swiglu(x, gu[e], dn[e]) for e in range(6))
    assert np.allclose(out["routed"], want, rtol=1e-12, atol=1e-12)


def test_identical_experts_reduce_to_dense_mlp():
    # P5: identical experts with renormalised top-k weights: sum_j G_j = 1,
    # so the MoE equals the one MLP, whatever the routing.
    cfg = _tiny_cfg(score="sigmoid", norm_topk=True, top_k=3)
    g = rng(10)
    x_all, wr, bias, gu, dn, _ = _tiny_inputs(cfg, g)
    gu[:] = gu[0]
    dn[:] = dn[0]
    out = oracle.moe_block(cfg, x_all, wr, bias, gu, dn)
    x = x_all[0].astype(np.float64)
    g1 = x @ gu[0][:cfg.ffn].T.astype(np.float64)
    u1 = x @ gu[0][cfg.ffn:].T.astype(np.float64)
    want = (g1 / (1 + np.exp(-g1)) * u1) @ dn[0].T.astype(np.float64)
    assert np.allclose(out["routed"], want, rtol=1e-12, atol=1e-12)
    # E = 1, k = 1: a plain MLP
    cfg1 = _tiny_cfg(n_experts=1, top_k=1)
    out1 = oracle.moe_block(cfg1, x_all, wr[:1], None, gu[:1], dn[:1])
    assert np.allclose(out1["routed"], want, rtol=1e-12, atol=1e-12)


def test_shared_experts_sum():
    g = rng(11)
    x = g.standard_normal((3, 4))
    a = g.standard_normal((2, 6, 4))
    b = g.standard_normal((2, 4, 3))
    want = oracle.swiglu(x, a[0], b[0]) + oracle.swiglu(x, a[1], b[1])
    assert np.allclose(oracle.shared_ffn(x, a, b), want, rtol=1e-14)


# ---------------------------------------------------------------- O14 FarSkip pair
def test_zero_moe_output_farskip_equals_regular():
    # P3 (Eq. 6 vs Eq. 7 with f = 0): with zero routed output the FarSkip
    # pair and the regular pair are the same computation.
    cfg = _tiny_cfg()
    g = rng(12)
    x_all, wr, _, gu, dn, _ = _tiny_inputs(cfg, g)
    dn[:] = 0
    out = oracle.moe_block(cfg, x_all, wr, None, gu, dn)
    assert not out["routed"].any()
    wn = g.standard_normal((cfg.hidden, cfg.hidden))
    shared = g.standard_normal(out["x"].shape)
    fs, _, _ = oracle.farskip_pair(out["x"], shared, out["routed"], wn)
    rg, _, _ = oracle.regular_pair(out["x"], shared, out["routed"], wn)
    assert np.array_equal(fs, rg)


def test_farskip_conservation_and_dropped_input():
    # P4 (Eq. 7, Section 3): every block output is added once into the final
    # residual; the next layer's input lacks exactly the routed output.
    g = rng(13)
    x, sh, ro = g.standard_normal((3, 4, 5))
    wn = g.standard_normal((5, 5))
    out, partial, nxt = oracle.farskip_pair(x, sh, ro, wn)
    assert np.allclose(out - x, sh + nxt + ro, rtol=1e-14, atol=1e-14)
    assert np.allclose(partial, x + sh, rtol=0, atol=0)
    assert np.allclose(nxt, (x + sh) @ wn.T, rtol=1e-14)
    rout, r1, rn = oracle.regular_pair(x, sh, ro, wn)
    assert np.allclose(rn, (x + sh + ro) @ wn.T, rtol=1e-14)
    # a stack of L FarSkip layers: the final residual holds every layer's
    # outputs exactly once, and layer l+1's dense input misses only layer l's
    # routed part.
    L = 4
    o = x.copy()
    total = x.copy()
    pending = np.zeros_like(x)
    for layer in range(L):
        o = o + pending
        shl, rol = g.standard_normal((2, 4, 5))
        out_l, part_l, nxt_l = oracle.farskip_pair(o, shl, rol, wn)
        assert np.allclose(part_l, o + shl)
        total = total + shl + nxt_l + rol
        o = out_l - rol
        pending = rol
    o = o + pending
    assert np.allclose(o, total, rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------- stacked layers
def _stack_layers(cfg, g, L, zero_down=False, zero_attention=False, shared=True):
    d, F = cfg.hidden, cfg.ffn
    layers = []
    for _ in range(L):
        _, wr, bias, gu, dn, _ = _tiny_inputs(cfg, g)
        if zero_down:
            dn[:] = 0
        lw = dict(w_router=wr, bias=bias, w_gate_up=gu, w_down=dn,
                  w_a=0.4 * g.standard_normal((d, d)), w_b=0.4 * g.standard_normal((d, d)))
        if zero_attention:
            lw["w_a"][:] = 0
        if shared and cfg.n_shared:
            lw["sh_gate_up"] = 0.3 * g.standard_normal((cfg.n_shared, 2 * cfg.ffn_shared, d))
            lw["sh_down"] = 0.3 * g.standard_normal((cfg.n_shared, d, cfg.ffn_shared))
        layers.append(lw)
    return layers


def test_stack_zero_moe_output_equals_regular():
    # With zero MoE output (zero down projections, no shared experts) the
    # FarSkip and the regular stacks are the same computation (Eq. 6 vs
    # Eq. 7 with f = 0), bit for bit in fp64.
    cfg = _tiny_cfg()
    g = rng(20)
    x = g.standard_normal((cfg.n_tokens, cfg.hidden))
    layers = _stack_layers(cfg, g, 3, zero_down=True)
    fs, _ = oracle.farskip_stack(cfg, x, layers)
    rg, _ = oracle.regular_stack(cfg, x, layers)
    assert np.array_equal(fs, rg)


@pytest.mark.parametrize("kw", [dict(), dict(n_shared=2, ffn_shared=3, score="sigmoid", norm_topk=True)])
def test_stack_conservation(kw):
    # Eq. 7 over L layers: the final residual minus the input is the sum of
    # every layer's attention, shared and routed outputs, each once.
    cfg = _tiny_cfg(**kw)
    g = rng(21)
    x = g.standard_normal((cfg.n_tokens, cfg.hidden))
    layers = _stack_layers(cfg, g, 4)
    o, terms = oracle.farskip_stack(cfg, x, layers)
    total = sum(t["attn"] + t["shared"] + t["routed"] for t in terms)
    assert np.allclose(o - x, total, rtol=1e-12, atol=1e-12)
    assert any(t["routed"].any() for t in terms)


def test_stack_one_layer_is_the_block():
    # One layer with a zero attention stand-in is the MoE block on x:
    # o = x + shared + routed, with both from the block computed directly.
    cfg = _tiny_cfg(n_shared=1, ffn_shared=4)
    g = rng(22)
    x = g.standard_normal((cfg.n_tokens, cfg.hidden)).astype(np.float32)
    layers = _stack_layers(cfg, g, 1, zero_attention=True)
    lw = layers[0]
    o, terms = oracle.farskip_stack(cfg, x, layers)
    blk = oracle.moe_block(cfg, x[None], lw["w_router"], lw["bias"], lw["w_gate_up"], lw["w_down"],
                           lw["sh_gate_up"], lw["sh_down"])
    assert np.array_equal(o, (x.astype(np.float64) + 0 + blk["shared"]) + blk["routed"])
    rg, _ = oracle.regular_stack(cfg, x, layers)
    assert np.array_equal(o, rg)


def test_stack_attention_does_not_see_the_previous_routed_output():
    # The one dependency FarSkip drops (Section 3): layer k's attention reads
    # p_{k-1}, which lacks layer k-1's routed output.  Changing layer 0's
    # experts leaves layer 1's attention unchanged in the FarSkip stack and
    # changes it in the regular stack; layer 1's experts see it in both.
    cfg = _tiny_cfg()
    g = rng(23)
    x = g.standard_normal((cfg.n_tokens, cfg.hidden))
    layers = _stack_layers(cfg, g, 2)
    other = [dict(lw) for lw in layers]
    other[0]["w_down"] = 2.0 * layers[0]["w_down"]
    _, t1 = oracle.farskip_stack(cfg, x, layers)
    _, t2 = oracle.farskip_stack(cfg, x, other)
    assert np.array_equal(t1[1]["attn"], t2[1]["attn"])
    assert not np.allclose(t1[1]["routed"], t2[1]["routed"])
    _, r1 = oracle.regular_stack(cfg, x, layers)
    _, r2 = oracle.regular_stack(cfg, x, other)
    assert not np.allclose(r1[1]["attn"], r2[1]["attn"])


def test_route_given_matches_route_on_its_own_selection():
    # The weights of a given selection are route()'s weights when the given
    # selection is route()'s own, for every scoring mode.
    g = rng(24)
    z = g.standard_normal((9, 12)).astype(np.float32)
    for score, norm in (("softmax", False), ("softmax", True), ("sigmoid", True), ("sigmoid", False)):
        ids, w, _, _ = oracle.route(z, score, 3, norm_topk=norm, routed_scale=2.5)
        assert np.allclose(oracle.route_given(z, ids, score, norm, 2.5), w, rtol=1e-15, atol=0)
    # and a given selection changes the block output only through the routing
    cfg = _tiny_cfg()
    x_all, wr, bias, gu, dn, _ = _tiny_inputs(cfg, rng(25))
    own = oracle.moe_block(cfg, x_all, wr, bias, gu, dn)
    same = oracle.moe_block(cfg, x_all, wr, bias, gu, dn, ids_given=own["me"]["ids"])
    assert np.array_equal(own["routed"], same["routed"])
    flipped = own["me"]["ids"][:, ::-1].copy()   # same experts, other slot order
    other = oracle.moe_block(cfg, x_all, wr, bias, gu, dn, ids_given=flipped)
    assert np.allclose(own["routed"], other["routed"], rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- token-by-token MoE
def _dense_mask_routed(cfg, x, ids, w, gu, dn, y_rows):
    """MoE(A) = sum_j G_j MLP^j(A) (Section 2.1) as a dense mixture: every
    local expert evaluated on every token at once, weighted by a gate matrix
    G [N, E] that is zero off the selection; the rows of experts on other
    ranks come from y_rows[t, j]."""
    N, k = ids.shape
    lo = cfg.ep_rank * cfg.n_local
    G = np.zeros((N, cfg.n_experts))
    np.put_along_axis(G, ids.astype(np.int64), w, axis=1)
    out = np.zeros_like(x)
    for e in range(cfg.n_local):
        h = x @ gu[e][:cfg.ffn].T.astype(np.float64)
        u = x @ gu[e][cfg.ffn:].T.astype(np.float64)
        out += G[:, lo + e:lo + e + 1] * ((h / (1 + np.exp(-h)) * u) @ dn[e].T.astype(np.float64))
    remote = (ids < lo) | (ids >= lo + cfg.n_local)
    out += np.einsum("tj,tjd->td", np.where(remote, w, 0.0), y_rows)
    return out


@pytest.mark.parametrize("kw", [dict(), dict(ep_size=3, ep_rank=1),
                                dict(ep_size=2, ep_rank=1, score="sigmoid", norm_topk=True),
                                dict(score="sigmoid", n_groups=3, topk_groups=2, top_k=3,
                                     ep_size=3, ep_rank=2)])
def test_tokens_direct_equals_dense_mask_and_packed_block(kw):
    # moe_tokens_direct evaluates the experts token by token with no plan or
    # pack.  It must equal (1) the dense gate-matrix mixture and (2) the
    # packed data flow of moe_block (pinned above), with the rows of other
    # ranks' experts taken from the return buffer at the plan row of each
    # (token, slot).  Ranks other than 0 make a local index off by the
    # rank's first expert fail, and every case mixes local and remote rows.
    cfg = _tiny_cfg(n_tokens=17, **kw)
    g = rng(26)
    x_all, wr, bias, gu, dn, yr = _tiny_inputs(cfg, g)
    out = oracle.moe_block(cfg, x_all, wr, bias, gu, dn, y_remote=yr)
    me = out["me"]
    ids, w, k = me["ids"], me["w"], cfg.top_k
    lo = cfg.ep_rank * cfg.n_local
    local = (ids >= lo) & (ids < lo + cfg.n_local)
    assert local.any()
    if cfg.ep_size > 1:
        assert (~local).any()
    s2r = me["plan"]["slot_to_row"]
    y_rows = np.zeros((cfg.n_tokens, k, cfg.hidden))
    if yr is not None:
        y_rows = yr.astype(np.float64)[s2r.reshape(cfg.n_tokens, k)]
    x = x_all[cfg.ep_rank].astype(np.float64)
    direct = oracle.moe_tokens_direct(cfg, x, ids, w, lambda e: (gu[e], dn[e]), y_rows)
    assert np.allclose(direct, _dense_mask_routed(cfg, x, ids, w, gu, dn, y_rows),
                       rtol=1e-12, atol=1e-12)
    assert np.allclose(direct, out["routed"], rtol=1e-12, atol=1e-12)
    # tokens are independent: a subset in any order gives the same rows
    sub = np.array([5, 0, 16, 9])
    part = oracle.moe_tokens_direct(cfg, x[sub], ids[sub], w[sub], lambda e: (gu[e], dn[e]),
                                    y_rows[sub])
    assert np.allclose(part, direct[sub], rtol=1e-14, atol=1e-14)


def test_tokens_direct_hand_value():
    # One local expert of width 1 with gate and up weights e_0 and down
    # weights 1: MLP(x) = SiLU(x_0) * x_0 in every output column.  Token
    # x_0 = 2 with weight 0.5 gives 0.5 * 2 * 2 / (1 + e^-2); a remote row of
    # 3s with weight 0.25 adds 0.75.
    cfg = _tiny_cfg(n_tokens=1, hidden=2, n_experts=2, top_k=2, ffn=1, ep_size=2, ep_rank=1)
    gu = np.array([[[1.0, 0.0], [1.0, 0.0]]])
    dn = np.array([[[1.0], [1.0]]])
    x = np.array([[2.0, -7.0]])
    ids = np.array([[1, 0]])
    w = np.array([[0.5, 0.25]])
    got = oracle.moe_tokens_direct(cfg, x, ids, w, lambda e: (gu[e], dn[e]),
                                   [[None, np.array([3.0, 3.0])]])
    want = 0.5 * 4.0 / (1.0 + math.exp(-2.0)) + 0.75
    assert np.allclose(got, [[want, want]], rtol=1e-15, atol=0)


def test_route_margin_kinds():
    # Softmax selection is never a near tie for the kernel (it compares the
    # logits themselves), but a perturbed input can flip a close pair:
    # "all" covers every decision, "set" only those that change which
    # experts are selected.
    z = np.array([[0.5, 0.5 + 2e-9, -1.0, 0.1], [2.0, 1.0, 0.0, -1.0],
                  [3.0, 1.0, 1.0 - 1e-9, -1.0]])
    _, _, near, margin = oracle.route(z, "softmax", 2)
    assert not near.any() and np.all(np.isinf(margin))
    ids, _, near, margin = oracle.route(z, "softmax", 2, margins="all")
    assert near.tolist() == [True, False, True]
    assert ids[0].tolist() == [1, 0]
    # row 1: gaps 2 - 1 (slot order) and 1 - 0 (last kept vs first dropped)
    assert margin[1] == 1.0
    _, _, near, margin = oracle.route(z, "softmax", 2, margins="set")
    # row 0: the close pair are both selected (only their order is close)
    assert near.tolist() == [False, False, True]
    assert margin[0] == 0.5 - 0.1 and margin[1] == 1.0
    # sigmoid: "kernel" and "all" agree
    a = oracle.route(z, "sigmoid", 2)[3]
    b = oracle.route(z, "sigmoid", 2, margins="all")[3]
    assert np.array_equal(a, b)
    # groups: the group boundary counts for "set", the order of kept groups
    # does not
    zg = np.array([[1.0, 0.0, 1.0 + 1e-9, 0.0, -3.0, -3.0]])
    m_all = oracle.route(zg, "softmax", 2, n_groups=3, topk_groups=2, margins="all")[3]
    m_set = oracle.route(zg, "softmax", 2, n_groups=3, topk_groups=2, margins="set")[3]
    assert m_all[0] < 1e-8 and m_set[0] == 1.0


def test_block_selection_callback():
    # A callable ids_given sees the logits, the oracle's own ids and the
    # margins of its set decisions, and its result replaces the selection.
    cfg = _tiny_cfg(score="sigmoid", n_groups=3, topk_groups=2, top_k=3)
    x_all, wr, bias, gu, dn, _ = _tiny_inputs(cfg, rng(27))
    own = oracle.moe_block(cfg, x_all, wr, bias, gu, dn)
    seen = {}

    def keep_own(z32, ids, margin):
        seen.update(z32=z32, ids=ids, margin=margin)
        return ids

    same = oracle.moe_block(cfg, x_all, wr, bias, gu, dn, ids_given=keep_own)
    assert np.array_equal(same["routed"], own["routed"])
    assert np.array_equal(seen["ids"], own["me"]["ids"])
    assert np.array_equal(seen["z32"], own["me"]["z32"])
    m_set = oracle.route(seen["z32"], cfg.score, cfg.top_k, cfg.n_groups, cfg.topk_groups,
                         cfg.norm_topk, cfg.routed_scale, bias, margins="set")[3]
    assert np.array_equal(seen["margin"], m_set)
    flipped = oracle.moe_block(cfg, x_all, wr, bias, gu, dn,
                               ids_given=lambda z, ids, m: ids[:, ::-1].copy())
    assert np.allclose(flipped["routed"], own["routed"], rtol=1e-12, atol=1e-12)
