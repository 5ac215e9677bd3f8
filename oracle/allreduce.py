"""The inference variant with replicated activations -- TEST INFRASTRUCTURE ONLY.

Section 2.1 notes that inference engines replace Dispatch and Combine by an
all-reduce: every rank holds all N tokens, routes all of them (the router is
duplicated), runs only the experts it owns, and the per-rank partial sums
are added over the R ranks.  Section 4.2 describes the FarSkip schedule for
this setting: the routed-expert all-reduce is started asynchronously and
joined only before the next layer's MoE, overlapping the next attention;
the attention output (tensor-parallel, so also a partial sum) and the
shared-expert output are added into one message and all-reduced once,
overlapping the routed experts.  Tab. 5 gives which computation hides
which all-reduce.

On one GPU an all-reduce over R ranks has one participant: the sum of one
rank's partial is that partial.  ``farskip_ar_stack`` / ``regular_ar_stack``
take that stand-in (identity) explicitly, so they describe exactly what one
rank computes; summed over the R ranks' partials (``routed_partial``,
``shared_partial`` and ``attention_partial`` for r = 0..R-1) every term is
the full-model term (pinned in the tests).

Tensor-parallel splits (readings where the paper only names the
parallelism):
  * shared experts: the merged SwiGLU of width W = S * F_s (hidden units
    expert-major: expert 0's F_s units, then expert 1's, ...) is split into
    R contiguous blocks of W / R hidden units; rank r owns the gate and up
    rows and the down columns of block r;
  * attention stand-in (two bias-free d x d linears, part (a) then part
    (b)): rank r owns rows [r d/R, (r+1) d/R) of W_a (column parallel) and
    the same columns of W_b (row parallel).

Floating point is fp64 on the exact input values, as in ``moe.py``.
"""

import numpy as np

from .moe import _given, dense_linear, logits_routing_f32, route, route_given, silu


def expert_range(n_experts, ep_size, ep_rank):
    """Rank r owns experts [r*E/R, (r+1)*E/R) (Section 2.1)."""
    e_loc = n_experts // ep_size
    return ep_rank * e_loc, (ep_rank + 1) * e_loc


def local_rows(ids, n_experts, ep_size, ep_rank):
    """Rows landing on rank r's experts when every rank holds every token.

    For each local expert (ascending) the tokens that selected it, in
    ascending token order.  Returns (tokens [M_r] int32: the token of each
    row, offsets [E/R + 1] int32: where each local expert's rows start)."""
    ids = np.asarray(ids)
    lo, hi = expert_range(n_experts, ep_size, ep_rank)
    tokens, offsets = [], [0]
    for e in range(lo, hi):
        for t in range(ids.shape[0]):
            if e in ids[t]:
                tokens.append(t)
        offsets.append(len(tokens))
    return np.array(tokens, np.int32), np.array(offsets, np.int32)


def _swiglu_one(xrow, gate_up, down):
    gu = np.asarray(gate_up, np.float64)
    F = gu.shape[0] // 2
    h = silu(gu[:F] @ xrow) * (gu[F:] @ xrow)
    return np.asarray(down, np.float64) @ h


def routed_partial(x, ids, weights, n_experts, ep_size, ep_rank, w_gate_up, w_down):
    """Rank r's share of MoE(A) = sum_j G_j MLP^j(A): for each token, the sum
    over its selections j whose expert rank r owns of w[t,j] *
    MLP^{ids[t,j]}(x_t), j ascending; tokens with no such selection get a
    zero row.  w_gate_up / w_down hold rank r's experts only ([E/R, ...])."""
    x = np.asarray(x, np.float64)
    ids = np.asarray(ids)
    w = np.asarray(weights, np.float64)
    lo, hi = expert_range(n_experts, ep_size, ep_rank)
    out = np.zeros_like(x)
    for t in range(x.shape[0]):
        for j in range(ids.shape[1]):
            e = int(ids[t, j])
            if lo <= e < hi:
                out[t] += w[t, j] * _swiglu_one(x[t], w_gate_up[e - lo], w_down[e - lo])
    return out


def routed_partial_rows(x, tokens, offsets, w_gate_up, w_down):
    """The expert outputs of rank r's rows (the grouped order of
    ``local_rows``): row i is MLP^{e}(x[tokens[i]]) for the local expert e
    whose block holds i.  Returns [M_r, d]."""
    x = np.asarray(x, np.float64)
    y = np.zeros((len(tokens), x.shape[1]), np.float64)
    for e in range(len(offsets) - 1):
        rows = np.arange(offsets[e], offsets[e + 1])
        if len(rows):
            X = x[np.asarray(tokens)[rows]]
            gu = np.asarray(w_gate_up[e], np.float64)
            F = gu.shape[0] // 2
            H = silu(X @ gu[:F].T) * (X @ gu[F:].T)
            y[rows] = H @ np.asarray(w_down[e], np.float64).T
    return y


def combine_partial(y_local, tokens, offsets, ids, weights, n_experts, ep_size, ep_rank):
    """The partial Combine of rank r from its rows' outputs: token t's j-th
    selection, when local, is the row of expert ids[t,j] holding token t;
    its output enters with weight w[t,j], j ascending."""
    ids = np.asarray(ids)
    w = np.asarray(weights, np.float64)
    y = np.asarray(y_local, np.float64)
    lo, hi = expert_range(n_experts, ep_size, ep_rank)
    N = ids.shape[0]
    out = np.zeros((N, y.shape[1]), np.float64)
    tokens = np.asarray(tokens)
    for t in range(N):
        for j in range(ids.shape[1]):
            e = int(ids[t, j])
            if lo <= e < hi:
                block = np.arange(offsets[e - lo], offsets[e - lo + 1])
                row = block[tokens[block] == t]
                out[t] += w[t, j] * y[int(row[0])]
    return out


def shared_partial(x, sh_gate_up, sh_down, ep_size, ep_rank):
    """Rank r's tensor-parallel share of the shared experts: the merged
    hidden units [r W/R, (r+1) W/R) of the S experts' SwiGLUs (expert-major
    order).  Summed over r it is the sum of the S shared experts."""
    x = np.asarray(x, np.float64)
    S = len(sh_gate_up)
    Fs = np.asarray(sh_gate_up[0]).shape[0] // 2
    W = S * Fs
    lo, hi = ep_rank * W // ep_size, (ep_rank + 1) * W // ep_size
    out = np.zeros((x.shape[0], np.asarray(sh_down[0]).shape[0]), np.float64)
    for u in range(lo, hi):
        s, f = divmod(u, Fs)
        gu = np.asarray(sh_gate_up[s], np.float64)
        g = x @ gu[f]
        up = x @ gu[Fs + f]
        out += np.outer(silu(g) * up, np.asarray(sh_down[s], np.float64)[:, f])
    return out


def attention_partial(p, w_a, w_b, ep_size, ep_rank):
    """Rank r's tensor-parallel share of the attention stand-in
    (p W_a^T) W_b^T: rows [r d/R, (r+1) d/R) of W_a, the same columns of
    W_b.  Summed over r it is the whole stand-in."""
    d = np.asarray(w_a).shape[0]
    lo, hi = ep_rank * d // ep_size, (ep_rank + 1) * d // ep_size
    wa = np.asarray(w_a, np.float64)[lo:hi]
    wb = np.asarray(w_b, np.float64)[:, lo:hi]
    return dense_linear(dense_linear(p, wa), wb)


def allreduce_one_rank(partial):
    """The all-reduce over ranks as seen by a single participant."""
    return np.asarray(partial, np.float64)


def _route_all(cfg, o, lw, ids_given):
    z32 = logits_routing_f32(o, lw["w_router"])
    ids, w, near, margin = route(z32, cfg.score, cfg.top_k, cfg.n_groups, cfg.topk_groups,
                                 cfg.norm_topk, cfg.routed_scale, lw.get("bias"))
    if ids_given is not None:
        ids = np.asarray(_given(ids_given, cfg, z32, ids, lw.get("bias")), np.int32)
        w = route_given(z32, ids, cfg.score, cfg.norm_topk, cfg.routed_scale)
    return ids, w, dict(z32=z32, ids=ids, margin=margin)


def _layer_partials(cfg, o, lw, ids_given):
    ids, w, rt = _route_all(cfg, o, lw, ids_given)
    R, r = cfg.ep_size, cfg.ep_rank
    routed = routed_partial(o, ids, w, cfg.n_experts, R, r, lw["w_gate_up"], lw["w_down"])
    shared = (shared_partial(o, lw["sh_gate_up"], lw["sh_down"], R, r) if cfg.n_shared > 0
              else np.zeros_like(np.asarray(o, np.float64)))
    return shared, routed, rt


def farskip_ar_stack(cfg, x, layers, ids_given=None):
    """L FarSkip layers of the replicated-activation variant on rank r.
    Layer k: attention partial A_k on p_{k-1}; shared partial S_k and
    routed partial R_k on o_{k-1} (Eq. 8a); the message A_k + S_k is
    all-reduced once, p_k = o_{k-1} + AR(A_k + S_k); o_k = p_k + AR(R_k)
    (Eq. 7).  p_{-1} = o_{-1} = x; AR is ``allreduce_one_rank``.  layers[k]
    holds w_router, bias, rank r's w_gate_up / w_down, the full sh_gate_up /
    sh_down and the full w_a / w_b."""
    o = p = np.asarray(x, np.float64)
    terms = []
    for k, lw in enumerate(layers):
        attn = attention_partial(p, lw["w_a"], lw["w_b"], cfg.ep_size, cfg.ep_rank)
        shared, routed, rt = _layer_partials(cfg, o, lw, None if ids_given is None else ids_given[k])
        p = o + allreduce_one_rank(attn + shared)
        o = p + allreduce_one_rank(routed)
        terms.append(dict(attn=attn, shared=shared, routed=routed, p=p, o=o, **rt))
    return o, terms


def regular_ar_stack(cfg, x, layers, ids_given=None):
    """L regular layers of the same variant (Eq. 6): o' = o + AR(A(o)),
    then o = o' + AR(S(o') + R(o')) -- one all-reduce after attention and
    one after the MLP, each blocking."""
    o = np.asarray(x, np.float64)
    terms = []
    for k, lw in enumerate(layers):
        attn = attention_partial(o, lw["w_a"], lw["w_b"], cfg.ep_size, cfg.ep_rank)
        o1 = o + allreduce_one_rank(attn)
        shared, routed, rt = _layer_partials(cfg, o1, lw, None if ids_given is None else ids_given[k])
        o = o1 + allreduce_one_rank(shared + routed)
        terms.append(dict(attn=attn, shared=shared, routed=routed, o=o, **rt))
    return o, terms
