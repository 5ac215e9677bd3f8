"""The allocation-free dispatch entry point (fs_dispatch_pack_noalloc),
called through the C ABI, against fs_dispatch_pack with a caller workspace
on the same inputs: every plan array and the send buffer bit for bit, on
calls in a row whose shapes shrink (each call finds the previous call's
contents in the library's fixed scratch), and against the oracle's plan."""

import numpy as np
import pytest
import torch

import oracle
from paper_2511_11505_amd import _lib as L
from workloads import CONFIGS
from workloads.generate import synthetic_topk_ids

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]
DEV = "cuda"


def outputs(cfg):
    N, E, k, R = cfg.n_tokens, cfg.n_experts, cfg.top_k, cfg.ep_size
    i32 = dict(dtype=torch.int32, device=DEV)
    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    return dict(counts=torch.full((E,), -7, **i32), offsets=torch.full((E + 1,), -7, **i32),
                rank_offsets=torch.full((R + 1,), -7, **i32),
                slot_to_row=torch.full((N * k,), -7, **i32),
                row_to_slot=torch.full((N * k,), -7, **i32),
                send=torch.full((N * k, cfg.hidden), -3.0, dtype=dt, device=DEV))


def both(cfg, seed):
    N, E, k = cfg.n_tokens, cfg.n_experts, cfg.top_k
    print(f"\n[no_alloc] N {N} E {E} k {k} R {cfg.ep_size} d {cfg.hidden} {cfg.dtype}", flush=True)
    ids = synthetic_topk_ids(N, E, k, seed=seed, device=DEV, skew=1.1)
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    x = torch.randn((N, cfg.hidden), generator=g, device=DEV)
    x = x.to(torch.float32 if cfg.dtype == "f32" else torch.bfloat16)
    desc = L.make_desc(cfg)
    ref, got = outputs(cfg), outputs(cfg)
    ws = torch.empty((max(L.fs_workspace_size(desc, L.FS_OP_DISPATCH_PACK), 256),),
                     dtype=torch.uint8, device=DEV)
    L.fs_dispatch_pack(desc, ids, x, ref["counts"], ref["offsets"], ref["rank_offsets"],
                       ref["slot_to_row"], ref["row_to_slot"], ref["send"], ws)
    L.fs_dispatch_pack_noalloc(desc, ids, x, got["counts"], got["offsets"], got["rank_offsets"],
                               got["slot_to_row"], got["row_to_slot"], got["send"])
    torch.cuda.synchronize()
    for key in ref:
        assert torch.equal(got[key].view(torch.int16) if key == "send" and cfg.dtype == "bf16"
                           else got[key], ref[key].view(torch.int16)
                           if key == "send" and cfg.dtype == "bf16" else ref[key]), key
    plan = oracle.dispatch_plan(ids.cpu().numpy(), E, cfg.ep_size)
    for key in ("counts", "offsets", "rank_offsets", "slot_to_row", "row_to_slot"):
        assert np.array_equal(got[key].cpu().numpy(), plan[key]), key


def test_no_alloc_dispatch_matches_workspace_entry_point():
    # DeepSeek-V3-shaped rank (three plan kernels, 64 x 256 scratch pairs),
    # then a smaller DeepSeek-V2-Lite-shaped batch (three kernels again,
    # stale scratch from the first call), then a decode-sized batch (the
    # one-workgroup plan), then the largest shape the scratch holds
    base = CONFIGS["dsv3_prefill"]
    both(base, 1)
    both(CONFIGS["dsv2lite"].scaled(n_tokens=1000), 2)
    both(base.scaled(n_tokens=64), 3)
    both(CONFIGS["tiny"].scaled(n_tokens=32768, n_experts=512, top_k=4, hidden=128), 4)
