"""Plain NumPy definitions of the FarSkip MoE block forward (test oracle).

Notation follows the paper: tokens A (here x, shape [N, d]), router weights
W_R [E, d], experts MLP^j with gate/up/down weights, EP size R with rank r
owning the contiguous experts [r*E/R, (r+1)*E/R).

Readings where the paper is silent (all listed in the design notes):
  * the expert MLP of Section 2.1, sigma(A W1^T . g(A W2^T)) W3^T, is read as
    SwiGLU: sigma = identity, g = SiLU on the gate projection, "." a Hadamard
    product;
  * the router selection function s() of Section 2.1 is a per-workload
    choice: softmax over all E experts (selection key = the logit), or
    sigmoid (selection key = sigmoid(z) + selection bias, weights use the
    unbiased sigmoid), optionally group-limited (group score = sum of the two
    largest keys in the group), top-k in descending key order, ties to the
    lower index, optional renormalisation over the k weights, then a scale;
  * Dispatch sends one row per (token, selected expert); rows of one expert
    are in ascending token order and experts are rank-blocked, so the send
    buffer is expert- and rank-contiguous.
"""

import numpy as np

# Router reduction order: the hidden dimension is cut into consecutive
# slices of this many elements.
ROUTER_SLICE = 256


# --------------------------------------------------------------------------
# O1: router logits  z = x W_R^T   (Section 2.1, G(A) = s(A W_R^T))
# --------------------------------------------------------------------------
def logits_f64(x, w_router):
    """Exact-definition logits in fp64."""
    return np.asarray(x, np.float64) @ np.asarray(w_router, np.float64).T


def logits_routing_f32(x, w_router, slice_len=ROUTER_SLICE):
    """fp32 logits summed in the router's fixed order.

    For every (token t, expert e): the hidden dimension is cut into slices of
    ``slice_len`` consecutive elements; within a slice the products
    fl32(x[t,i] * w[e,i]) are added one at a time in ascending i, starting
    from zero; the slice sums are then added one at a time in ascending slice
    order, starting from zero.  Every operation rounds to fp32.  This is the
    precision the routing decision is taken in.
    """
    x32 = np.asarray(x, np.float32)
    w32 = np.asarray(w_router, np.float32)
    N, d = x32.shape
    E = w32.shape[0]
    z = np.zeros((N, E), np.float32)
    for s0 in range(0, d, slice_len):
        p = np.zeros((N, E), np.float32)
        for i in range(s0, min(s0 + slice_len, d)):
            p += np.multiply.outer(x32[:, i], w32[:, i])
        z += p
    return z


# --------------------------------------------------------------------------
# O2-O6: scores, group limit, top-k, weights  (Section 2.1, s())
# --------------------------------------------------------------------------
def route(z32, score, top_k, n_groups=1, topk_groups=1, norm_topk=False,
          routed_scale=1.0, bias=None, tau=1e-6, margins="kernel"):
    """Select top_k experts per token from fp32 logits.

    Returns (ids [N,k] int32 in descending key order, weights [N,k] fp64,
    near_tie [N] bool, margin [N] fp64).

    ``near_tie`` flags tokens where a decision the kernel takes with rounded
    transcendental keys or rounded group sums is closer than ``tau``: either
    selection or slot order may then legitimately differ.  Softmax selection
    compares the fp32 logits themselves and is never flagged.

    ``margins`` chooses the decisions the margin covers: "kernel" (the
    above), "all" (every decision of either score: gaps between consecutive
    selected keys, between the last selected and the first rejected key,
    and the group decisions) or "set" (only the decisions that change which
    experts and groups are selected: the last selected against the first
    rejected key and group).  The last two serve logits that are themselves
    perturbed, as a stacked layer's input carries roundings.
    """
    if margins not in ("kernel", "all", "set"):
        raise ValueError(margins)
    z = np.asarray(z32, np.float64)
    N, E = z.shape
    if score == "softmax":
        if bias is not None:
            raise ValueError("a selection bias is defined for sigmoid scoring only")
        zmax = z.max(axis=1, keepdims=True)
        ex = np.exp(z - zmax)
        base = ex / ex.sum(axis=1, keepdims=True)   # probabilities over all E
        keys = z.copy()
        keys_rounded = margins != "kernel"
    elif score == "sigmoid":
        with np.errstate(over="ignore"):
            base = 1.0 / (1.0 + np.exp(-z))
        keys = base + (0.0 if bias is None else np.asarray(bias, np.float64)[None, :])
        keys_rounded = True
    else:
        raise ValueError(score)

    margin = np.full(N, np.inf)
    idx_e = np.broadcast_to(np.arange(E), (N, E))
    if n_groups > 1:
        gsz = E // n_groups
        kg = keys.reshape(N, n_groups, gsz)
        top2 = -np.sort(-kg, axis=2)[:, :, :2]
        gscore = top2.sum(axis=2) if gsz >= 2 else top2[:, :, 0]
        idx_g = np.broadcast_to(np.arange(n_groups), (N, n_groups))
        gorder = np.lexsort((idx_g, -gscore), axis=1)
        keep = gorder[:, :topk_groups]
        allowed = np.zeros((N, n_groups), bool)
        np.put_along_axis(allowed, keep, True, axis=1)
        keys = np.where(np.repeat(allowed, gsz, axis=1), keys, -np.inf)
        gs_sorted = np.take_along_axis(gscore, gorder, axis=1)
        if topk_groups < n_groups:
            margin = np.minimum(margin, gs_sorted[:, topk_groups - 1] - gs_sorted[:, topk_groups])
        if topk_groups > 1 and margins != "set":
            margin = np.minimum(margin, np.min(np.diff(-gs_sorted[:, :topk_groups], axis=1), axis=1))

    order = np.lexsort((idx_e, -keys), axis=1)
    ids = order[:, :top_k]
    if keys_rounded:
        ks = np.take_along_axis(keys, order, axis=1)
        if top_k < E:
            nxt = ks[:, top_k]
            gap = ks[:, top_k - 1] - nxt
            margin = np.minimum(margin, np.where(np.isfinite(nxt), gap, np.inf))
        if top_k > 1 and margins != "set":
            margin = np.minimum(margin, np.min(ks[:, :top_k - 1] - ks[:, 1:top_k], axis=1))
    w = np.take_along_axis(base, ids, axis=1)
    if norm_topk:
        w = w / w.sum(axis=1, keepdims=True)
    w = w * routed_scale
    return ids.astype(np.int32), w, margin < tau, margin


def route_given(z32, ids, score, norm_topk=False, routed_scale=1.0):
    """Weights of a given selection (ids [N,k], slot order as given) from
    fp32 logits: the softmax probability over all E or the sigmoid (no
    bias), then the optional renormalisation and the scale, as route()
    computes them for its own selection."""
    z = np.asarray(z32, np.float64)
    if score == "softmax":
        ex = np.exp(z - z.max(axis=1, keepdims=True))
        base = ex / ex.sum(axis=1, keepdims=True)
    else:
        base = 1.0 / (1.0 + np.exp(-z))
    w = np.take_along_axis(base, np.asarray(ids, np.int64), axis=1)
    if norm_topk:
        w = w / w.sum(axis=1, keepdims=True)
    return w * routed_scale


# --------------------------------------------------------------------------
# O7-O8: Dispatch plan and pack  (Section 2.1, Dispatch: permutation of A
# followed by the all-to-all)
# --------------------------------------------------------------------------
def dispatch_plan(ids, n_experts, ep_size=1):
    """counts[E], offsets[E+1], rank_offsets[R+1], slot_to_row[N*k],
    row_to_slot[N*k] (all int32).  Slot t*k+j is token t's j-th selection;
    rows are ordered by (expert, token)."""
    ids = np.asarray(ids)
    N, k = ids.shape
    counts = np.zeros(n_experts, np.int64)
    for e in ids.reshape(-1):
        counts[e] += 1
    offsets = np.zeros(n_experts + 1, np.int64)
    for e in range(n_experts):
        offsets[e + 1] = offsets[e] + counts[e]
    slot_to_row = np.empty(N * k, np.int64)
    seen = np.zeros(n_experts, np.int64)
    for t in range(N):
        for j in range(k):
            e = ids[t, j]
            slot_to_row[t * k + j] = offsets[e] + seen[e]
            seen[e] += 1
    row_to_slot = np.empty(N * k, np.int64)
    row_to_slot[slot_to_row] = np.arange(N * k)
    e_loc = n_experts // ep_size
    rank_offsets = np.array([offsets[r * e_loc] for r in range(ep_size + 1)], np.int64)
    i32 = lambda a: a.astype(np.int32)
    return dict(counts=i32(counts), offsets=i32(offsets), rank_offsets=i32(rank_offsets),
                slot_to_row=i32(slot_to_row), row_to_slot=i32(row_to_slot))


def pack(x, slot_to_row, top_k):
    """send[slot_to_row[t*k+j]] = x[t]."""
    x = np.asarray(x)
    send = np.empty((x.shape[0] * top_k, x.shape[1]), x.dtype)
    for s, row in enumerate(np.asarray(slot_to_row)):
        send[row] = x[s // top_k]
    return send


# --------------------------------------------------------------------------
# O9: rows landing on this rank's experts (receive side of Dispatch)
# --------------------------------------------------------------------------
def receive_rows(src_counts, src_offsets, cap, ep_rank, n_local):
    """Receive buffer layout: source s's whole send buffer sits at rows
    [s*cap, (s+1)*cap).  For each local expert e (ascending), rows of source
    0, 1, ... R-1 in that source's send order.  Returns (group_rows [M],
    group_offsets [n_local+1]) as int32."""
    src_counts = np.asarray(src_counts)
    src_offsets = np.asarray(src_offsets)
    R = src_counts.shape[0]
    rows, goff = [], [0]
    for e in range(n_local):
        ge = ep_rank * n_local + e
        for s in range(R):
            start = s * cap + int(src_offsets[s, ge])
            rows.extend(range(start, start + int(src_counts[s, ge])))
        goff.append(len(rows))
    return np.array(rows, np.int32), np.array(goff, np.int32)


# --------------------------------------------------------------------------
# O10/O13: expert MLP (Section 2.1, read as SwiGLU) and shared experts
# --------------------------------------------------------------------------
def silu(v):
    v = np.asarray(v, np.float64)
    with np.errstate(over="ignore"):
        return v / (1.0 + np.exp(-v))


def swiglu(X, w_gate_up, w_down):
    """(SiLU(X Wg^T) * (X Wu^T)) Wd^T with Wg = rows [0,F), Wu = rows [F,2F)."""
    X = np.asarray(X, np.float64)
    gu = np.asarray(w_gate_up, np.float64)
    F = gu.shape[0] // 2
    g = X @ gu[:F].T
    u = X @ gu[F:].T
    return (silu(g) * u) @ np.asarray(w_down, np.float64).T


def shared_ffn(x, sh_gate_up, sh_down):
    """Sum over the always-on shared experts (Section 2.1)."""
    out = np.zeros((np.asarray(x).shape[0], np.asarray(sh_down).shape[1]), np.float64)
    for s in range(len(sh_gate_up)):
        out += swiglu(x, sh_gate_up[s], sh_down[s])
    return out


# --------------------------------------------------------------------------
# O12: Combine  (Section 2.1: weighted sum of the returned expert outputs)
# --------------------------------------------------------------------------
def combine(y_ret, slot_to_row, weights):
    """routed[t] = sum_j w[t,j] * y_ret[slot_to_row[t*k+j]], j ascending."""
    w = np.asarray(weights, np.float64)
    N, k = w.shape
    y = np.asarray(y_ret, np.float64)
    out = np.zeros((N, y.shape[1]), np.float64)
    s2r = np.asarray(slot_to_row)
    for j in range(k):
        out += w[:, j:j + 1] * y[s2r[np.arange(N) * k + j]]
    return out


def residual_add(*terms):
    out = np.zeros_like(np.asarray(terms[0], np.float64))
    for t in terms:
        out = out + np.asarray(t, np.float64)
    return out


def dense_linear(a, w):
    """out = a w^T (the next-layer stand-in)."""
    return np.asarray(a, np.float64) @ np.asarray(w, np.float64).T


# --------------------------------------------------------------------------
# The whole block on rank r (packed formulation, O1-O13)
# --------------------------------------------------------------------------
def _given(ids_given, cfg, z32, own, bias):
    """The selection a caller substitutes: an [N, k] array, or a callable
    taking (z32, own ids, set-decision margins) and returning one."""
    if callable(ids_given):
        _, _, _, margin = route(z32, cfg.score, cfg.top_k, cfg.n_groups, cfg.topk_groups,
                                cfg.norm_topk, cfg.routed_scale, bias, margins="set")
        return ids_given(z32, own, margin)
    return ids_given


def moe_block(cfg, x_all, w_router, bias, w_gate_up, w_down, sh_gate_up=None,
              sh_down=None, y_remote=None, ids_given=None):
    """Every step of the block on rank cfg.ep_rank, following the data flow
    router -> top-k -> plan -> pack -> all-to-all -> experts -> return ->
    combine.  For R > 1 the other ranks' routing and sends are computed here
    too.  ids_given (optional) replaces this rank's own selection (the
    weights still come from its logits): an [N, k] array, or a callable
    (z32, own ids, margins of the set decisions) -> [N, k] ids, so that a
    caller can take the other side's selection only where rounding in an
    earlier layer may have moved a near tie.  Returns a dict of every
    intermediate."""
    R, r, k, E = cfg.ep_size, cfg.ep_rank, cfg.top_k, cfg.n_experts
    E_loc, cap = cfg.n_local, cfg.cap
    src = []
    for s in range(R):
        xs = np.asarray(x_all[s])
        z32 = logits_routing_f32(xs, w_router)
        ids, w, near, margin = route(z32, cfg.score, k, cfg.n_groups, cfg.topk_groups,
                                     cfg.norm_topk, cfg.routed_scale, bias)
        if s == r and ids_given is not None:
            ids = np.asarray(_given(ids_given, cfg, z32, ids, bias), np.int32)
            w = route_given(z32, ids, cfg.score, cfg.norm_topk, cfg.routed_scale)
        plan = dispatch_plan(ids, E, R)
        send = pack(xs, plan["slot_to_row"], k)
        src.append(dict(z32=z32, ids=ids, w=w, near_tie=near, margin=margin, plan=plan, send=send))
    src_counts = np.stack([s["plan"]["counts"] for s in src])
    src_offsets = np.stack([s["plan"]["offsets"] for s in src])
    group_rows, group_offsets = receive_rows(src_counts, src_offsets, cap, r, E_loc)
    recv = np.concatenate([s["send"] for s in src], axis=0)         # [R*cap, d]
    d = recv.shape[1]
    y = np.zeros((R * cap, d), np.float64)
    for e in range(E_loc):
        rows = group_rows[group_offsets[e]:group_offsets[e + 1]]
        if len(rows):
            y[rows] = swiglu(recv[rows], w_gate_up[e], w_down[e])
    me = src[r]
    lo, hi = me["plan"]["rank_offsets"][r], me["plan"]["rank_offsets"][r + 1]
    if R > 1:
        y_ret = np.array(y_remote, np.float64, copy=True)
    else:
        y_ret = np.zeros((cap, d), np.float64)
    y_ret[lo:hi] = y[r * cap + lo:r * cap + hi]
    routed = combine(y_ret, me["plan"]["slot_to_row"], me["w"])
    x = np.asarray(x_all[r], np.float64)
    shared = shared_ffn(x, sh_gate_up, sh_down) if cfg.n_shared > 0 else np.zeros_like(x)
    return dict(src=src, me=me, src_counts=src_counts, src_offsets=src_offsets,
                group_rows=group_rows, group_offsets=group_offsets, recv=recv, y=y,
                y_ret=y_ret, routed=routed, shared=shared, x=x)


def moe_tokens_direct(cfg, x_tokens, ids, weights, expert_weights, y_remote_rows=None):
    """MoE(A) = sum_j G_j MLP^j(A) token by token (Section 2.1), with no pack.

    ``expert_weights(e_local)`` returns (gate_up, down) of a local expert.
    For experts owned by other ranks, ``y_remote_rows[t][j]`` supplies the
    returned row.  Used on sampled tokens of the full-size workloads."""
    x_tokens = np.asarray(x_tokens, np.float64)
    n, d = x_tokens.shape
    out = np.zeros((n, d), np.float64)
    lo = cfg.ep_rank * cfg.n_local
    for t in range(n):
        for j in range(ids.shape[1]):
            e = int(ids[t, j])
            if lo <= e < lo + cfg.n_local:
                gu, dn = expert_weights(e - lo)
                y = swiglu(x_tokens[t:t + 1], gu, dn)[0]
            else:
                y = np.asarray(y_remote_rows[t][j], np.float64)
            out[t] += weights[t, j] * y
    return out


# --------------------------------------------------------------------------
# O14: the FarSkip block pair and the regular pair (Section 3, Eqs. 6-8)
# --------------------------------------------------------------------------
def farskip_pair(x, shared, routed, w_next):
    """FarSkip: the next layer reads attn-in = o_{k-1} + shared (Eq. 8b, the
    partial input) without this block's routed output, which is added into
    the residual afterwards (Eq. 7).  Returns (out, partial, next_out)."""
    x = np.asarray(x, np.float64)
    partial = x + shared
    nxt = dense_linear(partial, w_next)
    return x + shared + nxt + routed, partial, nxt


def regular_pair(x, shared, routed, w_next):
    """Regular residual stream (Eq. 6): the next layer reads the full o_k."""
    r1 = np.asarray(x, np.float64) + shared + routed
    nxt = dense_linear(r1, w_next)
    return r1 + nxt, r1, nxt


# --------------------------------------------------------------------------
# Stacked layers: the FarSkip connectivity of Section 3 (Eqs. 7-8) and the
# regular one (Eq. 6), each layer an attention stand-in (a bias-free linear
# for part (a), one for part (b), as Section 4.1 splits attention) and an
# MoE block.  R = 1: every source token is this rank's.
# --------------------------------------------------------------------------
def _layer_moe(cfg, o, lw, ids_given=None):
    """Shared and routed outputs of one layer's MoE block on input o, and
    its routing (logits, ids, margin)."""
    blk = moe_block(cfg, o[None], lw["w_router"], lw.get("bias"), lw["w_gate_up"], lw["w_down"],
                    lw.get("sh_gate_up"), lw.get("sh_down"), ids_given=ids_given)
    me = blk["me"]
    return blk["shared"], blk["routed"], dict(z32=me["z32"], ids=me["ids"], margin=me["margin"])


def attention_stand_in(p, lw):
    """Part (a) then part (b) of the attention stand-in: (p Wa^T) Wb^T."""
    return dense_linear(dense_linear(p, lw["w_a"]), lw["w_b"])


def farskip_stack(cfg, x, layers, ids_given=None):
    """L FarSkip layers.  Layer k's attention reads the partial output
    p_{k-1} (everything but layer k-1's routed output, Eq. 8b); its shared
    and routed experts read the outdated o_{k-1} (Eq. 8a);
    p_k = o_{k-1} + attn_k + shared_k and o_k = p_k + routed_k (Eq. 7).
    p_{-1} = o_{-1} = x.  ids_given[k] (optional) is layer k's selection
    (see moe_block).  Returns the final o and the per-layer terms."""
    o = p = np.asarray(x, np.float64)
    terms = []
    for k, lw in enumerate(layers):
        attn = attention_stand_in(p, lw)
        shared, routed, rt = _layer_moe(cfg, o, lw, None if ids_given is None else ids_given[k])
        p = o + attn + shared
        o = p + routed
        terms.append(dict(attn=attn, shared=shared, routed=routed, p=p, o=o, **rt))
    return o, terms


def regular_stack(cfg, x, layers, ids_given=None):
    """L regular layers (Eq. 6): o'_k = o_{k-1} + attn(o_{k-1}), then
    o_k = o'_k + shared(o'_k) + routed(o'_k)."""
    o = np.asarray(x, np.float64)
    terms = []
    for k, lw in enumerate(layers):
        attn = attention_stand_in(o, lw)
        o1 = o + attn
        shared, routed, rt = _layer_moe(cfg, o1, lw, None if ids_given is None else ids_given[k])
        o = o1 + shared + routed
        terms.append(dict(attn=attn, shared=shared, routed=routed, o=o, **rt))
    return o, terms
