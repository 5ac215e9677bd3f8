"""Seeded synthetic inputs.

Every tensor is drawn with torch's Philox generator on the device that runs
the case, seeded from (config seed, tensor tag, index) through numpy's
SeedSequence, so any single tensor (one expert's weights, one virtual rank's
tokens) can be regenerated on its own.  Values are drawn in fp32 and, for
bf16 workloads, rounded to bf16 by round-to-nearest-even.

Distributions: tokens x ~ N(0, 1); router, expert, shared-expert and
next-layer weights ~ N(0, 0.02^2) (0.02 is the standard deviation); the
selection bias is none, uniform(-0.1, 0.1), or a Zipf(s) popularity bias
b_e = -beta * s * ln(rank_e) over a seeded permutation rank of 1..E; the
synthetic expert-output rows returned by the other ranks ~ N(0, y_std^2).

No routing, GEMM, combine or residual arithmetic lives here.
"""

from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import torch

# tensor tags
TAG_X, TAG_ROUTER, TAG_BIAS, TAG_GATE_UP, TAG_DOWN = 0, 1, 2, 3, 4
TAG_SH_GATE_UP, TAG_SH_DOWN, TAG_NEXT, TAG_Y_REMOTE = 5, 6, 7, 8
TAG_ATT_A, TAG_ATT_B, TAG_LAYER = 9, 10, 11

WEIGHT_STD = 0.02
Y_REMOTE_STD = 1.8   # close to the rms of one expert's output at d=7168, F=2048


def _seed(seed, tag, idx=0):
    state = np.random.SeedSequence([int(seed), int(tag), int(idx)]).generate_state(2, np.uint32)
    return int(state[0]) | (int(state[1] & 0x7FFFFFFF) << 32)


def _gen(device, seed, tag, idx=0):
    g = torch.Generator(device=device)
    g.manual_seed(_seed(seed, tag, idx))
    return g


def torch_dtype(name):
    return torch.float32 if name == "f32" else torch.bfloat16


def bf16_round(a):
    """fp32 numpy array -> bf16 bit patterns (uint16), round-to-nearest-even."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def normal(shape, std, dtype, device, seed, tag, idx=0):
    g = _gen(device, seed, tag, idx)
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    return t.to(torch_dtype(dtype))


def selection_bias(cfg, device):
    """fp32 [E] selection bias, or None."""
    if cfg.bias == "none":
        return None
    g = _gen(device, cfg.seed, TAG_BIAS)
    if cfg.bias == "uniform":
        return torch.rand(cfg.n_experts, generator=g, device=device, dtype=torch.float32) * 0.2 - 0.1
    if cfg.bias == "zipf":
        rank = torch.randperm(cfg.n_experts, generator=g, device=device).to(torch.float64) + 1.0
        return (-cfg.zipf_beta * cfg.zipf_s * torch.log(rank)).to(torch.float32)
    raise ValueError(cfg.bias)


@dataclass
class Workload:
    cfg: object
    device: str
    x_all: torch.Tensor                 # [R, N, d]: tokens of every (virtual) source rank
    w_router: torch.Tensor              # [E, d]
    bias: Optional[torch.Tensor]        # [E] fp32 or None
    w_gate_up: torch.Tensor             # [E_loc, 2F, d]: rows [0,F) gate, [F,2F) up
    w_down: torch.Tensor                # [E_loc, d, F]
    sh_gate_up: Optional[torch.Tensor]  # [S, 2F_s, d] per shared expert
    sh_down: Optional[torch.Tensor]     # [S, d, F_s]
    w_next: Optional[torch.Tensor]      # [d, d] next-layer stand-in
    y_remote: Optional[torch.Tensor]    # [N*k, d] rows returned by the other ranks' experts
    extra: dict = field(default_factory=dict)

    @property
    def x(self):
        """This rank's tokens, the MoE input o_{k-1}: its own (all-to-all) or
        the replicated token set (all-reduce)."""
        return self.x_all[0 if self.cfg.ep_mode == "allreduce" else self.cfg.ep_rank]


def expert_weights(cfg, device, e_local):
    """(gate_up [2F, d], down [d, F]) of one local expert, regenerated alone."""
    gu = normal((2 * cfg.ffn, cfg.hidden), WEIGHT_STD, cfg.dtype, device, cfg.seed, TAG_GATE_UP, e_local)
    dn = normal((cfg.hidden, cfg.ffn), WEIGHT_STD, cfg.dtype, device, cfg.seed, TAG_DOWN, e_local)
    return gu, dn


def source_tokens(cfg, device, src):
    return normal((cfg.n_tokens, cfg.hidden), 1.0, cfg.dtype, device, cfg.seed, TAG_X, src)


def make_workload(cfg, device="cpu", with_experts=True):
    R, N, d, E, F = cfg.ep_size, cfg.n_tokens, cfg.hidden, cfg.n_experts, cfg.ffn
    dt = torch_dtype(cfg.dtype)
    x_all = torch.empty((cfg.n_sources, N, d), dtype=dt, device=device)
    for s in range(cfg.n_sources):
        x_all[s] = source_tokens(cfg, device, s)
    w_router = normal((E, d), WEIGHT_STD, cfg.dtype, device, cfg.seed, TAG_ROUTER)
    bias = selection_bias(cfg, device)
    E_loc = cfg.n_local
    if with_experts:
        w_gate_up = torch.empty((E_loc, 2 * F, d), dtype=dt, device=device)
        w_down = torch.empty((E_loc, d, F), dtype=dt, device=device)
        for e in range(E_loc):
            w_gate_up[e], w_down[e] = expert_weights(cfg, device, e)
    else:
        w_gate_up = w_down = None
    sh_gu = sh_dn = None
    if cfg.n_shared > 0:
        Fs = cfg.ffn_shared
        sh_gu = torch.stack([normal((2 * Fs, d), WEIGHT_STD, cfg.dtype, device, cfg.seed, TAG_SH_GATE_UP, s)
                             for s in range(cfg.n_shared)])
        sh_dn = torch.stack([normal((d, Fs), WEIGHT_STD, cfg.dtype, device, cfg.seed, TAG_SH_DOWN, s)
                             for s in range(cfg.n_shared)])
    w_next = normal((d, d), WEIGHT_STD, cfg.dtype, device, cfg.seed, TAG_NEXT) if cfg.next_linear else None
    y_remote = None
    if R > 1 and cfg.ep_mode == "a2a":
        y_remote = normal((cfg.cap, d), Y_REMOTE_STD, cfg.dtype, device, cfg.seed, TAG_Y_REMOTE)
    return Workload(cfg, device, x_all, w_router, bias, w_gate_up, w_down, sh_gu, sh_dn, w_next, y_remote)


def merge_shared(sh_gate_up, sh_down):
    """Lay S shared experts out as one SwiGLU of width S*F_s (a weight-layout
    transform done once at load time): gate rows of all experts, then up rows;
    down columns concatenated along F."""
    S, twoF, d = sh_gate_up.shape
    Fs = twoF // 2
    gate = sh_gate_up[:, :Fs, :].reshape(S * Fs, d)
    up = sh_gate_up[:, Fs:, :].reshape(S * Fs, d)
    gu = torch.cat([gate, up], dim=0).contiguous()
    dn = sh_down.permute(1, 0, 2).reshape(d, S * Fs).contiguous()
    return gu, dn


def tp_shared_slice(gate_up, down, ep_size, ep_rank):
    """Rank r's tensor-parallel block of a merged shared-expert SwiGLU of
    width W (gate_up [2W, d], down [d, W]): hidden units
    [r W/R, (r+1) W/R), as (gate_up [2W/R, d], down [d, W/R]), contiguous
    (a weight-layout transform)."""
    W = down.shape[1]
    lo, hi = ep_rank * W // ep_size, (ep_rank + 1) * W // ep_size
    gu = torch.cat([gate_up[lo:hi], gate_up[W + lo:W + hi]], dim=0).contiguous()
    return gu, down[:, lo:hi].contiguous()


def tp_attention_slice(w_a, w_b, ep_size, ep_rank):
    """Rank r's tensor-parallel block of the attention stand-in: rows
    [r d/R, (r+1) d/R) of w_a, the same columns of w_b (contiguous)."""
    d = w_a.shape[0]
    lo, hi = ep_rank * d // ep_size, (ep_rank + 1) * d // ep_size
    return w_a[lo:hi].contiguous(), w_b[:, lo:hi].contiguous()


def synthetic_topk_ids(n_tokens, n_experts, top_k, seed, device="cpu", skew=0.0):
    """Distinct expert ids per token, seeded; optional popularity skew.
    Used to drive the dispatch-plan kernels with ids that do not come from a
    router."""
    g = _gen(device, seed, 99)
    w = torch.ones(n_experts, dtype=torch.float32, device=device)
    if skew > 0:
        w = (torch.arange(n_experts, device=device, dtype=torch.float32) + 1.0) ** (-skew)
    w = w.expand(n_tokens, n_experts).contiguous()
    ids = torch.multinomial(w, top_k, replacement=False, generator=g)
    return ids.to(torch.int32)


def layer_seed(seed, layer):
    """Seed of layer `layer` of a stack built on a workload of seed `seed`."""
    return int(np.random.SeedSequence([int(seed), TAG_LAYER, int(layer)]).generate_state(1, np.uint32)[0])


def stack_layers(cfg, n_layers, device):
    """Weights of n_layers stacked layers: each an MoE block drawn like a
    workload of its own seed, plus two d x d attention stand-in linears
    (part (a), part (b)) ~ N(0, 0.02^2).  Returns a list of
    (layer config, Workload, w_a, w_b)."""
    out = []
    for k in range(n_layers):
        lc = cfg.scaled(seed=layer_seed(cfg.seed, k))
        wl = make_workload(lc, device)
        w_a = normal((cfg.hidden, cfg.hidden), WEIGHT_STD, cfg.dtype, device, lc.seed, TAG_ATT_A)
        w_b = normal((cfg.hidden, cfg.hidden), WEIGHT_STD, cfg.dtype, device, lc.seed, TAG_ATT_B)
        out.append((lc, wl, w_a, w_b))
    return out
