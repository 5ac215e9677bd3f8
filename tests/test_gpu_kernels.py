"""GPU parity of each step of the hot path against the CPU oracle, through the
C ABI, at sizes the oracle finishes in seconds that span several tiles and a
ragged tail.  Integers are compared bit for bit, floats with rel_err against
the stated tolerance."""

import numpy as np
import pytest
import torch

import oracle
from paper_2511_11505_amd import _lib as L
from paper_2511_11505_amd.block import fragment_ordered
from tests._util import TOL, f64, rel_err
from workloads import CONFIGS, make_workload
from workloads.generate import synthetic_topk_ids

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]
DEV = "cuda"

# Small variants of the five workloads: several router slices (one ragged),
# several GEMM tiles, ragged token counts.
SMALL = {
    "tiny": CONFIGS["tiny"],
    "tiny_ragged": CONFIGS["tiny"].scaled(n_tokens=77, name="tiny_ragged"),
    "dsv2lite_s": CONFIGS["dsv2lite"].scaled(n_tokens=333, hidden=512, ffn=256, ffn_shared=128,
                                             name="dsv2lite_s"),
    "scout_s": CONFIGS["scout"].scaled(n_tokens=517, hidden=640, ffn=384, ffn_shared=384,
                                       name="scout_s"),
    "dsv3_prefill_s": CONFIGS["dsv3_prefill"].scaled(n_tokens=150, hidden=512, ffn=256,
                                                     ffn_shared=256, name="dsv3_prefill_s"),
    "dsv3_decode_s": CONFIGS["dsv3_decode"].scaled(n_tokens=9, hidden=384, ffn=192, ffn_shared=192,
                                                   name="dsv3_decode_s"),
}


def ws_for(desc, op, rows=0, ffn=0):
    return torch.empty((max(L.fs_workspace_size(desc, op, rows, ffn), 256),), dtype=torch.uint8,
                       device=DEV)


def route_gpu(cfg, x, w_router, bias, logits_in=None):
    desc = L.make_desc(cfg)
    N, E, k = cfg.n_tokens, cfg.n_experts, cfg.top_k
    logits = torch.empty((N, E), dtype=torch.float32, device=DEV)
    ids = torch.empty((N, k), dtype=torch.int32, device=DEV)
    w = torch.empty((N, k), dtype=torch.float32, device=DEV)
    L.fs_router_topk(desc, x, w_router, bias, logits_in, logits, ids, w,
                     ws_for(desc, L.FS_OP_ROUTER_TOPK))
    torch.cuda.synchronize()
    return logits, ids, w


def check_ids(cfg, ids_gpu, ids_ref, near):
    """Bit-exact ids except on near-tie tokens, where the selection must still
    be a valid top-k set (checked by the caller's keys)."""
    g = ids_gpu.cpu().numpy()
    assert g.shape == ids_ref.shape
    far = ~near
    bad = np.where(np.any(g[far] != ids_ref[far], axis=1))[0]
    assert bad.size == 0, f"{cfg.name}: {bad.size} non-tie tokens routed differently"
    for t in np.where(near)[0]:
        assert len(set(g[t].tolist())) == cfg.top_k
        assert all(0 <= e < cfg.n_experts for e in g[t])
    return int(near.sum())


# router-only cases: 37 tokens over five slices of the hidden dimension;
# 160 experts (a ragged last 64-expert range) over 300 tokens (a ragged last
# 32-token tile); 8190 tokens over 512 experts, enough output tiles to run
# without splitting the hidden dimension, two slices of it (one ragged);
ROUTER_EXTRA = {
    "dsv3_decode_m": CONFIGS["dsv3_decode"].scaled(n_tokens=37, hidden=1280, ffn=192,
                                                   ffn_shared=192, name="dsv3_decode_m"),
    "e160": CONFIGS["dsv2lite"].scaled(n_tokens=300, hidden=640, n_experts=160, ffn=256,
                                       ffn_shared=128, name="e160"),
    "wide_unsplit": CONFIGS["dsv3_prefill"].scaled(n_tokens=8190, hidden=384, n_experts=512,
                                                   ep_size=1, ffn=256, ffn_shared=128,
                                                   name="wide_unsplit"),
    # the 16-expert matrix-core kernel: one slice (no split; 700 tokens, a
    # ragged third 256-token tile); 6 experts (padded expert rows) over 4.5
    # slices (the last one 128 wide), one slice per workgroup
    "e16_unsplit": CONFIGS["scout"].scaled(n_tokens=700, hidden=256, ffn=256, ffn_shared=256,
                                           name="e16_unsplit"),
    "e6_split": CONFIGS["dsv2lite"].scaled(n_tokens=1100, hidden=1152, n_experts=6, top_k=2,
                                           ffn=256, ffn_shared=128, name="e6_split"),
    # enough tiles x slices for two slices per workgroup: 9 tiles x 58
    # slices (the last 128 wide), workgroup 28 taking slices 56 and 57
    "e16_two_slices": CONFIGS["scout"].scaled(n_tokens=2148, hidden=14720, ffn=256,
                                              ffn_shared=256, name="e16_two_slices"),
    # decode-sized: 36 slices summed by the top-k kernel (four batches of
    # eight loads and a ragged tail of four)
    "decode_36_slices": CONFIGS["dsv3_decode"].scaled(n_tokens=20, hidden=9216, ffn=128,
                                                      ffn_shared=128, name="decode_36_slices"),
}


@pytest.mark.parametrize("name", list(SMALL) + list(ROUTER_EXTRA))
def test_router_logits_bitexact_and_topk(name):
    cfg = SMALL.get(name) or ROUTER_EXTRA[name]
    wl = make_workload(cfg, DEV, with_experts=False)
    for s in range(cfg.ep_size):
        x = wl.x_all[s]
        logits, ids, w = route_gpu(cfg, x, wl.w_router, wl.bias)
        z_ref = oracle.logits_routing_f32(f64(x).astype(np.float32), f64(wl.w_router).astype(np.float32))
        z_gpu = logits.cpu().numpy()
        assert np.array_equal(z_gpu, z_ref), (
            f"{name} src {s}: logits differ bitwise at {np.argwhere(z_gpu != z_ref)[:5].tolist()}")
        bias = None if wl.bias is None else f64(wl.bias)
        ids_ref, w_ref, near, _ = oracle.route(z_ref, cfg.score, cfg.top_k, cfg.n_groups,
                                               cfg.topk_groups, cfg.norm_topk, cfg.routed_scale, bias)
        check_ids(cfg, ids, ids_ref, near)
        far = ~near
        assert rel_err(w.cpu().numpy()[far], w_ref[far]) <= 2e-6


# groups of 16, 24, 32 and 64 experts, over 64 to 512 experts (one to
# eight per lane)
@pytest.mark.parametrize("score,G,TG,k,E", [("softmax", 1, 1, 4, 40), ("sigmoid", 4, 2, 3, 96),
                                            ("sigmoid", 8, 4, 8, 256), ("softmax", 16, 3, 5, 512),
                                            ("sigmoid", 1, 1, 32, 200), ("sigmoid", 16, 5, 6, 256),
                                            ("softmax", 4, 2, 4, 256), ("sigmoid", 4, 2, 3, 64),
                                            ("sigmoid", 4, 3, 4, 128), ("softmax", 8, 2, 6, 192)])
def test_topk_from_given_logits(score, G, TG, k, E):
    # Quantised logits create exact ties: selection must break them toward
    # the lower expert (softmax compares the logits themselves).
    cfg = CONFIGS["tiny"].scaled(n_tokens=301, n_experts=E, top_k=k, score=score, n_groups=G,
                                 topk_groups=TG, norm_topk=(score == "sigmoid"), routed_scale=1.5)
    g = torch.Generator(device="cpu").manual_seed(11)
    z = (torch.randint(-6, 7, (cfg.n_tokens, E), generator=g).float() * 0.25)
    bias = (torch.rand(E, generator=g) * 0.2 - 0.1) if score == "sigmoid" else None
    logits_in = z.to(DEV)
    _, ids, w = route_gpu(cfg, None, None, None if bias is None else bias.to(DEV), logits_in=logits_in)
    ids_ref, w_ref, near, _ = oracle.route(z.numpy(), score, k, G, TG, cfg.norm_topk, 1.5,
                                           None if bias is None else bias.numpy().astype(np.float64))
    n_near = check_ids(cfg, ids, ids_ref, near)
    if score == "softmax" and G == 1:
        assert n_near == 0
    assert rel_err(w.cpu().numpy()[~near], w_ref[~near]) <= 2e-6


def plan_gpu(cfg, ids, x):
    desc = L.make_desc(cfg)
    N, E, k, R, d = cfg.n_tokens, cfg.n_experts, cfg.top_k, cfg.ep_size, cfg.hidden
    i32 = torch.int32
    out = dict(counts=torch.empty(E, dtype=i32, device=DEV),
               offsets=torch.empty(E + 1, dtype=i32, device=DEV),
               rank_offsets=torch.empty(R + 1, dtype=i32, device=DEV),
               slot_to_row=torch.empty(N * k, dtype=i32, device=DEV),
               row_to_slot=torch.empty(N * k, dtype=i32, device=DEV),
               send=torch.empty((N * k, d), dtype=x.dtype, device=DEV))
    L.fs_dispatch_pack(desc, ids, x, out["counts"], out["offsets"], out["rank_offsets"],
                       out["slot_to_row"], out["row_to_slot"], out["send"],
                       ws_for(desc, L.FS_OP_DISPATCH_PACK))
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("N,E,k,R,dtype", [(1, 8, 2, 1, "f32"), (63, 16, 1, 4, "bf16"),
                                           (64, 64, 6, 1, "bf16"), (65, 64, 6, 8, "bf16"),
                                           (512, 512, 32, 4, "bf16"), (1000, 256, 8, 8, "bf16"),
                                           (777, 512, 32, 4, "f32"), (4096, 16, 1, 1, "bf16"),
                                           (4200, 256, 4, 8, "bf16"), (4096, 256, 8, 8, "bf16"),
                                           (8192, 16, 1, 1, "bf16"), (20000, 64, 8, 8, "bf16")])
def test_plan_pack_bitexact(N, E, k, R, dtype):
    # up to tiles x slots = 2^23 the plan runs in one workgroup per 64-token
    # tile that counts every slot (4096 x 8: 2^21), beyond (20000 x 8) in
    # three kernels
    cfg = CONFIGS["tiny"].scaled(n_tokens=N, n_experts=E, top_k=k, ep_size=R, hidden=128, dtype=dtype)
    ids = synthetic_topk_ids(N, E, k, seed=N + E, device=DEV, skew=1.1)
    x = torch.randn((N, 128), device=DEV).to(torch.float32 if dtype == "f32" else torch.bfloat16)
    out = plan_gpu(cfg, ids, x)
    ref = oracle.dispatch_plan(ids.cpu().numpy(), E, R)
    for key in ("counts", "offsets", "rank_offsets", "slot_to_row", "row_to_slot"):
        assert np.array_equal(out[key].cpu().numpy(), ref[key]), key
    send_ref = oracle.pack(x.cpu().float().numpy(), ref["slot_to_row"], k)
    assert np.array_equal(out["send"].cpu().float().numpy(), send_ref)


def test_receive_rows_bitexact():
    cfg = CONFIGS["dsv3_prefill"].scaled(n_tokens=300, ep_rank=5)
    R, N, E, k = cfg.ep_size, cfg.n_tokens, cfg.n_experts, cfg.top_k
    plans = [oracle.dispatch_plan(synthetic_topk_ids(N, E, k, seed=s, skew=0.7).numpy(), E, R)
             for s in range(R)]
    cnt = np.stack([p["counts"] for p in plans])
    off = np.stack([p["offsets"] for p in plans])
    rows_ref, goff_ref = oracle.receive_rows(cnt, off, cfg.cap, cfg.ep_rank, cfg.n_local)
    rows = torch.full((R * cfg.cap,), -7, dtype=torch.int32, device=DEV)
    goff = torch.empty(cfg.n_local + 1, dtype=torch.int32, device=DEV)
    L.fs_receive_rows(L.make_desc(cfg), torch.from_numpy(cnt).to(DEV), torch.from_numpy(off).to(DEV),
                      rows, goff)
    torch.cuda.synchronize()
    assert np.array_equal(goff.cpu().numpy(), goff_ref)
    assert np.array_equal(rows.cpu().numpy()[:len(rows_ref)], rows_ref)


def ragged_groups(G, total_hint, seed):
    g = np.random.default_rng(seed)
    counts = g.integers(0, 2 * total_hint // G + 1, size=G)
    counts[0] = 0                   # an empty group
    counts[min(1, G - 1)] = 1       # a single row
    if G > 2:
        counts[2] = 300             # several m-tiles with a ragged tail
    return counts


@pytest.mark.parametrize("dtype,G,d,F,gather", [("f32", 5, 256, 512, False), ("f32", 3, 128, 192, True),
                                                ("bf16", 6, 512, 256, False), ("bf16", 4, 384, 320, True),
                                                ("bf16", 1, 256, 128, False), ("bf16", 5, 768, 384, True)])
def test_grouped_ffn(dtype, G, d, F, gather):
    counts = ragged_groups(G, 600, seed=G + d)
    M = int(counts.sum())
    goff = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    gen = torch.Generator(device=DEV).manual_seed(d + F)
    n_src = M + 37
    X = torch.randn((n_src, d), generator=gen, device=DEV).to(tdt)
    wgu = (0.05 * torch.randn((G, 2 * F, d), generator=gen, device=DEV)).to(tdt)
    wd = (0.05 * torch.randn((G, d, F), generator=gen, device=DEV)).to(tdt)
    rows = torch.randperm(n_src, generator=gen, device=DEV)[:M].to(torch.int32) if gather else None
    out = torch.full((n_src, d), float("nan"), device=DEV).to(tdt)
    cfg = CONFIGS["tiny"].scaled(hidden=d, ffn=F, dtype=dtype)
    desc = L.make_desc(cfg)
    L.fs_grouped_expert_ffn(desc, G, F, X, rows, torch.from_numpy(goff).to(DEV), M, wgu, wd, out,
                            ws_for(desc, L.FS_OP_GROUPED_FFN, M, F))
    torch.cuda.synchronize()
    Xn, gun, dnn = f64(X), f64(wgu), f64(wd)
    rr = rows.cpu().numpy() if gather else np.arange(M)
    outn = f64(out)
    for gi in range(G):
        sel = rr[goff[gi]:goff[gi + 1]]
        if len(sel) == 0:
            continue
        want = oracle.swiglu(Xn[sel], gun[gi], dnn[gi])
        assert rel_err(outn[sel], want) <= TOL[dtype], f"group {gi}"
    untouched = np.setdiff1d(np.arange(n_src), rr)
    assert np.all(np.isnan(outn[untouched]))


@pytest.mark.parametrize("counts,d,F,gather", [([12000, 0, 9001, 1, 8000, 11111], 256, 128, True),
                                               ([12000, 0, 9001, 1, 8000, 11111], 512, 256, False)])
def test_grouped_ffn_many_tiles(counts, d, F, gather):
    """More 128-row tiles than workgroups, so the interleaved ring runs on
    from tile to tile (the last blocks of a tile prefetch the next tile's
    first ones; gathered rows through scalar loads), with K rings of 2, 4
    and 8 blocks; element by element against the oracle."""
    counts = np.array(counts)
    G, M = len(counts), int(counts.sum())
    goff = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    gen = torch.Generator(device=DEV).manual_seed(d + 5 * F)
    n_src = M + 37
    X = torch.randn((n_src, d), generator=gen, device=DEV).to(torch.bfloat16)
    wgu = (0.05 * torch.randn((G, 2 * F, d), generator=gen, device=DEV)).to(torch.bfloat16)
    wd = (0.05 * torch.randn((G, d, F), generator=gen, device=DEV)).to(torch.bfloat16)
    rows = torch.randperm(n_src, generator=gen, device=DEV)[:M].to(torch.int32) if gather else None
    out = torch.full((n_src, d), float("nan"), device=DEV).to(torch.bfloat16)
    desc = L.make_desc(CONFIGS["tiny"].scaled(hidden=d, ffn=F, dtype="bf16"))
    L.fs_grouped_expert_ffn(desc, G, F, X, rows, torch.from_numpy(goff).to(DEV), M, wgu, wd, out,
                            ws_for(desc, L.FS_OP_GROUPED_FFN, M, F))
    torch.cuda.synchronize()
    Xn, gun, dnn, outn = f64(X), f64(wgu), f64(wd), f64(out)
    rr = rows.cpu().numpy() if gather else np.arange(M)
    for gi in range(G):
        sel = rr[goff[gi]:goff[gi + 1]]
        if len(sel):
            assert rel_err(outn[sel], oracle.swiglu(Xn[sel], gun[gi], dnn[gi])) <= TOL["bf16"], f"group {gi}"
    assert np.all(np.isnan(outn[np.setdiff1d(np.arange(n_src), rr)]))


def test_grouped_ffn_wide_tiles():
    """Two long groups (4100 and 2050 rows, both ragged) of a dense-shaped
    pass with a short down K and a 4096-wide output (the shape of a
    prefill's shared expert); sampled rows of each group (the first 64, 64
    from the middle, the last 300: its ragged tiles) against the oracle
    element by element."""
    counts = np.array([4100, 2050])
    d, F = 4096, 256
    G, M = len(counts), int(counts.sum())
    goff = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    gen = torch.Generator(device=DEV).manual_seed(4100)
    n_src = M + 11
    X = torch.randn((n_src, d), generator=gen, device=DEV).to(torch.bfloat16)
    wgu = (0.05 * torch.randn((G, 2 * F, d), generator=gen, device=DEV)).to(torch.bfloat16)
    wd = (0.05 * torch.randn((G, d, F), generator=gen, device=DEV)).to(torch.bfloat16)
    rows = torch.randperm(n_src, generator=gen, device=DEV)[:M].to(torch.int32)
    out = torch.full((n_src, d), float("nan"), device=DEV).to(torch.bfloat16)
    desc = L.make_desc(CONFIGS["tiny"].scaled(hidden=d, ffn=F, dtype="bf16"))
    L.fs_grouped_expert_ffn(desc, G, F, X, rows, torch.from_numpy(goff).to(DEV), M, wgu, wd, out,
                            ws_for(desc, L.FS_OP_GROUPED_FFN, M, F))
    torch.cuda.synchronize()
    rr = rows.cpu().numpy()
    for gi in range(G):
        n = counts[gi]
        pick = np.concatenate([np.arange(64), np.arange(n // 2 - 32, n // 2 + 32), np.arange(n - 300, n)])
        sel = rr[goff[gi] + pick]
        want = oracle.swiglu(f64(X[torch.from_numpy(sel).to(DEV).long()]), f64(wgu[gi]), f64(wd[gi]))
        assert rel_err(f64(out[torch.from_numpy(sel).to(DEV).long()]), want) <= TOL["bf16"], f"group {gi}"
    assert torch.isnan(out[torch.from_numpy(np.setdiff1d(np.arange(n_src), rr)).to(DEV).long()]).all()


@pytest.mark.parametrize("counts,d,F,gather", [([100, 0, 170, 50], 1024, 1024, True),
                                               ([41, 300, 7], 2048, 512, False)])
def test_grouped_ffn_split_k(counts, d, F, gather):
    """Few tiles and long K: the interleaved-ring passes split K into slices
    with fp32 partials summed in slice order (gate/up and down here);
    element by element against the oracle."""
    counts = np.array(counts)
    G, M = len(counts), int(counts.sum())
    goff = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    gen = torch.Generator(device=DEV).manual_seed(d + 3 * F)
    n_src = M + 9
    X = torch.randn((n_src, d), generator=gen, device=DEV).to(torch.bfloat16)
    wgu = (0.05 * torch.randn((G, 2 * F, d), generator=gen, device=DEV)).to(torch.bfloat16)
    wd = (0.05 * torch.randn((G, d, F), generator=gen, device=DEV)).to(torch.bfloat16)
    rows = torch.randperm(n_src, generator=gen, device=DEV)[:M].to(torch.int32) if gather else None
    out = torch.full((n_src, d), float("nan"), device=DEV).to(torch.bfloat16)
    desc = L.make_desc(CONFIGS["tiny"].scaled(hidden=d, ffn=F, dtype="bf16"))
    L.fs_grouped_expert_ffn(desc, G, F, X, rows, torch.from_numpy(goff).to(DEV), M, wgu, wd, out,
                            ws_for(desc, L.FS_OP_GROUPED_FFN, M, F))
    torch.cuda.synchronize()
    Xn, gun, dnn, outn = f64(X), f64(wgu), f64(wd), f64(out)
    rr = rows.cpu().numpy() if gather else np.arange(M)
    for gi in range(G):
        sel = rr[goff[gi]:goff[gi + 1]]
        if len(sel):
            assert rel_err(outn[sel], oracle.swiglu(Xn[sel], gun[gi], dnn[gi])) <= TOL["bf16"], f"group {gi}"
    assert np.all(np.isnan(outn[np.setdiff1d(np.arange(n_src), rr)]))


@pytest.mark.parametrize("counts,d,F,gather", [
    ([0, 1, 64, 65, 130], 768, 320, True),     # m-chunks of 64, split K 6 / 2 slices (3 + 2 blocks)
    ([37], 512, 256, False),                   # one group (a decode shared expert), K 256: streamed
    ([50], 1024, 512, True),                   # one group, K 512: the skinny down pass
    ([64], 512, 1024, False),                  # a full 64-row group, skinny down (K 1024)
    ([1], 512, 512, True),                     # one row, skinny down
    ([3, 0, 5, 9, 1, 0, 2, 7], 384, 192, True),  # many small groups
])
def test_grouped_ffn_streaming(counts, d, F, gather):
    """Groups averaging at most 64 rows take the weight-streaming kernel (with
    split K when its tiles are few); the down pass of one group of at most 64
    rows takes the skinny kernel where K % 512 == 0; element by element
    against the oracle."""
    counts = np.array(counts)
    G, M = len(counts), int(counts.sum())
    goff = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    gen = torch.Generator(device=DEV).manual_seed(d * 7 + F)
    n_src = M + 11
    X = torch.randn((n_src, d), generator=gen, device=DEV).to(torch.bfloat16)
    wgu = (0.05 * torch.randn((G, 2 * F, d), generator=gen, device=DEV)).to(torch.bfloat16)
    wd = (0.05 * torch.randn((G, d, F), generator=gen, device=DEV)).to(torch.bfloat16)
    rows = torch.randperm(n_src, generator=gen, device=DEV)[:M].to(torch.int32) if gather else None
    out = torch.full((n_src, d), float("nan"), device=DEV).to(torch.bfloat16)
    desc = L.make_desc(CONFIGS["tiny"].scaled(hidden=d, ffn=F, dtype="bf16"))
    L.fs_grouped_expert_ffn(desc, G, F, X, rows, torch.from_numpy(goff).to(DEV), M, wgu, wd, out,
                            ws_for(desc, L.FS_OP_GROUPED_FFN, M, F))
    torch.cuda.synchronize()
    Xn, gun, dnn, outn = f64(X), f64(wgu), f64(wd), f64(out)
    rr = rows.cpu().numpy() if gather else np.arange(M)
    for gi in range(G):
        sel = rr[goff[gi]:goff[gi + 1]]
        if len(sel):
            assert rel_err(outn[sel], oracle.swiglu(Xn[sel], gun[gi], dnn[gi])) <= TOL["bf16"], f"group {gi}"
    assert np.all(np.isnan(outn[np.setdiff1d(np.arange(n_src), rr)]))


# n not a multiple of 256 takes 128 x 128 tiles: one K block (no cross-tile
# prefetch), exactly the three blocks a tile prefetches, and the
# tensor-parallel attention part [4096 x 5120] x [5120 x 640] with a ragged m
@pytest.mark.parametrize("dtype,m,n,kd", [("f32", 70, 128, 256), ("bf16", 300, 256, 512), ("bf16", 1, 128, 64),
                                         ("bf16", 2049, 768, 640), ("bf16", 333, 640, 512),
                                         ("bf16", 129, 384, 64), ("bf16", 257, 384, 192),
                                         ("bf16", 4099, 640, 5120)])
def test_dense_linear(dtype, m, n, kd):
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    gen = torch.Generator(device=DEV).manual_seed(m)
    a = torch.randn((m, kd), generator=gen, device=DEV).to(tdt)
    w = (0.05 * torch.randn((n, kd), generator=gen, device=DEV)).to(tdt)
    out = torch.empty((m, n), dtype=tdt, device=DEV)
    L.fs_dense_linear(L.FS_F32 if dtype == "f32" else L.FS_BF16, m, n, kd, a, w, out)
    torch.cuda.synchronize()
    assert rel_err(out, oracle.dense_linear(f64(a), f64(w))) <= TOL[dtype]


# the last two cases have wide rows (640 and 544 16-byte chunks)
@pytest.mark.parametrize("dtype,N,k,d,shared", [("f32", 37, 2, 256, False), ("bf16", 130, 8, 512, True),
                                                ("bf16", 5, 1, 128, False), ("bf16", 67, 8, 5120, True),
                                                ("f32", 33, 6, 2176, False)])
def test_combine_and_residual(dtype, N, k, d, shared):
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    cfg = CONFIGS["tiny"].scaled(n_tokens=N, top_k=k, hidden=d, n_experts=16, dtype=dtype)
    desc = L.make_desc(cfg)
    ids = synthetic_topk_ids(N, 16, k, seed=N)
    plan = oracle.dispatch_plan(ids.numpy(), 16, 1)
    gen = torch.Generator(device=DEV).manual_seed(d)
    y = torch.randn((N * k, d), generator=gen, device=DEV).to(tdt)
    w = torch.rand((N, k), generator=gen, device=DEV)
    sh = torch.randn((N, d), generator=gen, device=DEV).to(tdt) if shared else None
    resid = torch.randn((N, d), generator=gen, device=DEV).to(tdt)
    resid0 = resid.clone()
    routed = torch.empty((N, d), dtype=tdt, device=DEV)
    s2r = torch.from_numpy(plan["slot_to_row"]).to(DEV)
    L.fs_combine_unpack(desc, y, s2r, w, sh, routed, resid)
    torch.cuda.synchronize()
    acc = oracle.combine(f64(y), plan["slot_to_row"], f64(w))
    if shared:
        acc = acc + f64(sh)
    assert rel_err(routed, acc) <= TOL[dtype]
    assert rel_err(resid, oracle.residual_add(f64(resid0), acc)) <= TOL[dtype]
    # the plain FarSkip residual add, out of place and in place
    out = torch.empty_like(resid)
    L.fs_farskip_residual(desc, out, resid0, routed, sh)
    torch.cuda.synchronize()
    extra = [f64(sh)] if shared else []
    assert rel_err(out, oracle.residual_add(f64(resid0), f64(routed), *extra)) <= TOL[dtype]
    want_inplace = oracle.residual_add(f64(resid0), f64(routed))
    L.fs_farskip_residual(desc, resid0, resid0, routed)
    torch.cuda.synchronize()
    assert rel_err(resid0, want_inplace) <= TOL[dtype]


def test_profile_select_times_only_the_selected_kernels():
    """fs_profile_select: with only the gate/up pass selected, a grouped FFN
    records gate/up launches and no down launches; with all selected, both."""
    G, per, d, F = 4, 100, 256, 256
    M = G * per
    gen = torch.Generator(device=DEV).manual_seed(5)
    X = torch.randn((M, d), generator=gen, device=DEV).to(torch.bfloat16)
    wgu = (0.05 * torch.randn((G, 2 * F, d), generator=gen, device=DEV)).to(torch.bfloat16)
    wd = (0.05 * torch.randn((G, d, F), generator=gen, device=DEV)).to(torch.bfloat16)
    goff = torch.arange(0, M + 1, per, dtype=torch.int32, device=DEV)
    out = torch.empty((M, d), dtype=torch.bfloat16, device=DEV)
    desc = L.make_desc(CONFIGS["tiny"].scaled(hidden=d, ffn=F, dtype="bf16"))
    ws = ws_for(desc, L.FS_OP_GROUPED_FFN, M, F)
    try:
        for sel, want_down in (([L.FS_K_GATE_UP], 0), (None, 2)):
            L.fs_profile_reset()
            L.fs_profile_select(sel)
            L.fs_profile_enable(True)
            for _ in range(2):
                L.fs_grouped_expert_ffn(desc, G, F, X, None, goff, M, wgu, wd, out, ws)
            torch.cuda.synchronize()
            L.fs_profile_enable(False)
            ms_gu, n_gu = L.fs_profile_read(L.FS_K_GATE_UP)
            assert n_gu == 2 and ms_gu > 0
            assert L.fs_profile_read(L.FS_K_DOWN)[1] == want_down
    finally:
        L.fs_profile_enable(False)
        L.fs_profile_select(None)
        L.fs_profile_reset()


def test_fragment_order_layout():
    # block (g, c) of a matrix holds, at lane l, row 32 g + l % 32 and
    # columns 16 c + 8 (l / 32) .. + 7: a plain reshape of the row-major
    # matrix, checked bit for bit
    gen = torch.Generator(device=DEV).manual_seed(5)
    w = torch.randn((3, 96, 48), generator=gen, device=DEV).to(torch.bfloat16)
    fo = fragment_ordered(w)
    torch.cuda.synchronize()
    a = w.view(torch.int16).cpu().numpy().reshape(3, 3, 32, 3, 2, 8)   # [m][g][r][c][h][e]
    want = a.transpose(0, 1, 3, 4, 2, 5).reshape(-1)                   # [m][g][c][h][r][e]
    assert np.array_equal(fo.view(torch.int16).cpu().numpy().reshape(-1), want)


@pytest.mark.parametrize("counts,d,F,gather", [
    ([0, 1, 64, 65, 130], 768, 256, True),      # empty, single-row, one and three 64-row tiles
    ([37], 512, 128, False),                    # one group
    ([3, 0, 5, 9, 1, 0, 2, 7], 256, 384, True),   # many small groups, K of 4 blocks (tail)
    ([20, 113, 0, 61, 2], 1024, 640, True),     # K rings of 16 and 10 blocks (ragged tails)
    # 320 tiles per pass: workgroups take two (K of 16 and 8 blocks)
    ([100] * 40, 1024, 512, True),
])
def test_grouped_ffn_fragment_order(counts, d, F, gather):
    """The grouped SwiGLU FFN on fragment-ordered weights (weights streamed
    straight into the matrix units' registers), element by element against
    the oracle; rows outside the groups are never written."""
    counts = np.array(counts)
    G, M = len(counts), int(counts.sum())
    goff = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    gen = torch.Generator(device=DEV).manual_seed(d * 3 + F)
    n_src = M + 13
    X = torch.randn((n_src, d), generator=gen, device=DEV).to(torch.bfloat16)
    wgu = (0.05 * torch.randn((G, 2 * F, d), generator=gen, device=DEV)).to(torch.bfloat16)
    wd = (0.05 * torch.randn((G, d, F), generator=gen, device=DEV)).to(torch.bfloat16)
    rows = torch.randperm(n_src, generator=gen, device=DEV)[:M].to(torch.int32) if gather else None
    out = torch.full((n_src, d), float("nan"), device=DEV).to(torch.bfloat16)
    desc = L.make_desc(CONFIGS["tiny"].scaled(hidden=d, ffn=F, dtype="bf16"))
    L.fs_grouped_expert_ffn_fo(desc, G, F, X, rows, torch.from_numpy(goff).to(DEV), M,
                               fragment_ordered(wgu), fragment_ordered(wd), out,
                               ws_for(desc, L.FS_OP_GROUPED_FFN, M, F))
    torch.cuda.synchronize()
    Xn, gun, dnn, outn = f64(X), f64(wgu), f64(wd), f64(out)
    rr = rows.cpu().numpy() if gather else np.arange(M)
    for gi in range(G):
        sel = rr[goff[gi]:goff[gi + 1]]
        if len(sel):
            assert rel_err(outn[sel], oracle.swiglu(Xn[sel], gun[gi], dnn[gi])) <= TOL["bf16"], f"group {gi}"
    assert np.all(np.isnan(outn[np.setdiff1d(np.arange(n_src), rr)]))
