"""GPU parity of the FP8 (E4M3) experts against oracle.fp8.

Row quantisation is compared bit for bit (codes and scales).  The FP8
SwiGLU FFN is compared step by step on the same quantised operands:
  * H (bf16) against the oracle's fp64 gate/up product of the same x and
    weight codes, then rounded like the kernel: only fp32 accumulation and
    the bf16 rounding of H separate them;
  * the codes and scales of H, bit for bit against the oracle's quantiser
    applied to the GPU's H (H is the quantiser's input, so the decision is
    taken on the same value);
  * the output against the oracle's fp64 down product of those H codes;
and end to end against the unquantised SwiGLU, within the error FP8
brings (3 mantissa bits on both operands of both GEMMs).

Tolerance for the step comparisons: max relative error (floored at the
rms) 1e-2, between the bf16 output rounding (2^-9 relative) and the block
tolerance; measured values are printed."""

import numpy as np
import pytest
import torch

import oracle
from oracle import fp8 as of8
from paper_2511_11505_amd import _lib as L
from tests._util import f64, rel_err
from workloads import CONFIGS

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]
DEV = "cuda"
STEP_TOL = 1e-2


def quantize(t):
    rows, cols = t.shape
    codes = torch.empty((rows, cols), dtype=torch.uint8, device=DEV)
    scales = torch.empty((rows,), dtype=torch.float32, device=DEV)
    L.fs_quantize_fp8(L.FS_F32 if t.dtype == torch.float32 else L.FS_BF16, rows, cols, t, codes, scales)
    return codes, scales


def np_u8(t):
    return t.cpu().numpy().astype(np.uint8)


# 1024 rows and more take one wave per row for bf16 rows up to 8192 wide
# (16 columns: two vectors, most lanes idle; 2064: a ragged 16-vector row;
# 8192 the widest; 8208 falls back to a workgroup per row)
@pytest.mark.parametrize("dtype,rows,cols", [("bf16", 37, 512), ("f32", 21, 256), ("bf16", 1, 7168),
                                             ("bf16", 300, 2048), ("bf16", 1030, 16),
                                             ("bf16", 1500, 2048), ("bf16", 1025, 2064),
                                             ("bf16", 1024, 8192), ("bf16", 1024, 8208)])
def test_quantize_rows_bit_exact(dtype, rows, cols):
    g = torch.Generator(device=DEV).manual_seed(rows * 7 + cols)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    x = torch.randn((rows, cols), generator=g, device=DEV)
    # rows of very different magnitudes, an all-zero row, negative zeros,
    # exact fp8 midpoints after scaling, and a row whose amax is negative
    x *= torch.exp(torch.linspace(-8, 8, rows, device=DEV))[:, None]
    if rows > 3:
        x[1] = 0
        x[2, : cols // 2] = -0.0
        x[3] = torch.tensor([448.0, -232.0, 240.0, 13.0, -0.5], device=DEV).repeat(cols // 5 + 1)[:cols]
        x[3, 5] = -448.0
    x = x.to(tdt)
    codes, scales = quantize(x)
    torch.cuda.synchronize()
    want_c, want_s = of8.quantize_rows(x.float().cpu().numpy())
    assert np.array_equal(scales.cpu().numpy().view(np.uint32), want_s.view(np.uint32))
    assert np.array_equal(np_u8(codes), want_c)


def ffn_case(G, F, d, counts, gather, seed):
    g = torch.Generator(device=DEV).manual_seed(seed)
    M = int(sum(counts))
    n_src = max(M, 1) + 5
    x = torch.randn((n_src, d), generator=g, device=DEV).to(torch.bfloat16)
    wgu = (0.02 * torch.randn((G, 2 * F, d), generator=g, device=DEV)).to(torch.bfloat16)
    wdn = (0.02 * torch.randn((G, d, F), generator=g, device=DEV)).to(torch.bfloat16)
    goff = torch.tensor(np.concatenate([[0], np.cumsum(counts)]), dtype=torch.int32, device=DEV)
    rows = None
    if gather:
        rows = torch.randperm(n_src, generator=g, device=DEV)[:M].to(torch.int32)
    return x, wgu, wdn, goff, rows, M


# Every pass runs on 128 x 256 FP8 tiles (eight waves); [2304] is one dense
# group that fills the CUs; the last case but one has few tiles and long
# K, so both passes split K; the last has more tiles than workgroups with
# two-block K rings (the ring runs on from tile to tile)
FFN_CASES = [([0, 1, 64, 65, 130], 256, 512, True),
             ([37], 128, 256, False),
             ([3, 0, 5, 300, 1, 0, 2, 7], 384, 768, True),
             ([513, 700], 512, 1024, False),
             ([2304], 4096, 256, False),
             ([100, 0, 170, 50], 1024, 2048, True),
             ([12000, 0, 9001, 1, 8000, 11111], 256, 256, True)]
# the FP8 fragment-order kernels (weights streamed into registers) on the
# cases of a few rows per group, and one dense group (36 row tiles)
FO_CASES = [c for i, c in enumerate(FFN_CASES) if i in (0, 1, 2, 4, 5)] + [
    # 320 tiles per pass, two per workgroup, K of 8 and 4 blocks; then a
    # down pass of K = 2 blocks
    ([100] * 40, 512, 1024, True),
    ([100] * 40, 256, 1024, True)]


def test_fragment_order_fp8_layout():
    # fragment (g, c), half h of a code matrix holds, at lane l, row
    # 32 g + l % 32 and columns 64 c + 32 (l / 32) + 16 h .. + 15: a plain
    # reshape of the row-major matrix, checked bit for bit
    from paper_2511_11505_amd import fragment_ordered_fp8
    gen = torch.Generator(device=DEV).manual_seed(6)
    w = torch.randint(0, 256, (3, 96, 192), generator=gen, device=DEV, dtype=torch.int32).to(torch.uint8)
    fo = fragment_ordered_fp8(w)
    torch.cuda.synchronize()
    a = np_u8(w).reshape(3, 3, 32, 3, 2, 2, 16)        # [m][g][r][c][l/32][h][byte]
    want = a.transpose(0, 1, 3, 5, 4, 2, 6).reshape(-1)  # [m][g][c][h][l/32][r][byte]
    assert np.array_equal(np_u8(fo).reshape(-1), want)


@pytest.mark.parametrize("counts,F,d,gather,fo", [c + (False,) for c in FFN_CASES]
                         + [c + (True,) for c in FO_CASES])
def test_grouped_ffn_fp8_steps(counts, F, d, gather, fo):
    G = len(counts)
    x, wgu, wdn, goff, rows, M = ffn_case(G, F, d, counts, gather, seed=sum(counts) + F)
    cfg = CONFIGS["tiny"].scaled(hidden=d, ffn=F, dtype="bf16")
    desc = L.make_desc(cfg)
    xq, xs = quantize(x)
    gq, gs = quantize(wgu.reshape(G * 2 * F, d))
    dq, ds = quantize(wdn.reshape(G * d, F))
    out = torch.full((x.shape[0], d), float("nan"), dtype=torch.bfloat16, device=DEV)
    ws_bytes = L.fs_workspace_size(desc, L.FS_OP_GROUPED_FFN_FP8, M, F)
    ws = torch.empty((ws_bytes,), dtype=torch.uint8, device=DEV)
    if fo:
        from paper_2511_11505_amd import fragment_ordered_fp8
        L.fs_grouped_expert_ffn_fp8_fo(desc, G, F, xq, xs, rows, goff, M,
                                       fragment_ordered_fp8(gq.reshape(G, 2 * F, d)), gs,
                                       fragment_ordered_fp8(dq.reshape(G, d, F)), ds, out, ws)
    else:
        L.fs_grouped_expert_ffn_fp8(desc, G, F, xq, xs, rows, goff, M, gq.reshape(G, 2 * F, d), gs,
                                    dq.reshape(G, d, F), ds, out, ws)
    torch.cuda.synchronize()
    a = lambda n: (n + 255) // 256 * 256
    H = ws[: M * F * 2].view(torch.bfloat16).reshape(M, F)
    Hq = ws[a(2 * M * F): a(2 * M * F) + M * F].reshape(M, F)
    Hs = ws[a(2 * M * F) + a(M * F): a(2 * M * F) + a(M * F) + 4 * M].view(torch.float32)
    xq_n, xs_n = np_u8(xq), xs.cpu().numpy()
    gq_n, gs_n = np_u8(gq).reshape(G, 2 * F, d), gs.cpu().numpy().reshape(G, 2 * F)
    dq_n, ds_n = np_u8(dq).reshape(G, d, F), ds.cpu().numpy().reshape(G, d)
    # the codes the oracle is about to use are the oracle's own quantisation
    # of the bf16 activations and weights, bit for bit
    for got_c, got_s, src_t in ((xq_n, xs_n, x), (gq_n.reshape(-1, d), gs_n.reshape(-1), wgu),
                                (dq_n.reshape(-1, F), ds_n.reshape(-1), wdn)):
        want_c, want_s = of8.quantize_rows(src_t.float().cpu().numpy().reshape(got_c.shape))
        assert np.array_equal(got_c, want_c)
        assert np.array_equal(got_s.view(np.uint32), want_s.view(np.uint32))
    src = np.arange(M) if rows is None else rows.cpu().numpy()
    goff_n = goff.cpu().numpy()
    H_n, Hq_n, Hs_n, out_n = f64(H), np_u8(Hq), Hs.cpu().numpy(), f64(out)
    errs = []
    for e in range(G):
        r0, r1 = goff_n[e], goff_n[e + 1]
        if r1 == r0:
            continue
        sel = src[r0:r1]
        h_want = of8.swiglu_fp8_hidden(xq_n[sel], xs_n[sel], gq_n[e], gs_n[e])
        errs.append(rel_err(H_n[r0:r1], h_want))
        c_want, s_want = of8.quantize_rows(H_n[r0:r1])
        assert np.array_equal(Hq_n[r0:r1], c_want)
        assert np.array_equal(Hs_n[r0:r1].view(np.uint32), s_want.view(np.uint32))
        y_want = of8.scaled_gemm(Hq_n[r0:r1], Hs_n[r0:r1], dq_n[e], ds_n[e])
        errs.append(rel_err(out_n[sel], y_want))
        # end to end against the unquantised expert: the FP8 error
        ref = oracle.swiglu(f64(x[torch.from_numpy(sel).to(DEV)]), f64(wgu[e]), f64(wdn[e]))
        d_rms = np.sqrt(np.mean((out_n[sel] - ref) ** 2)) / np.sqrt(np.mean(ref ** 2))
        assert d_rms <= 0.08, d_rms
    print("max step errors", max(errs))
    assert max(errs) <= STEP_TOL
    # rows of x that no group reads keep their NaN fill only where out is not written
    if rows is not None:
        untouched = np.setdiff1d(np.arange(x.shape[0]), src)
        assert np.all(np.isnan(out_n[untouched]))


# ---------------------------------------------------------------- FP8 dispatch
@pytest.mark.parametrize("N,E,k,R,d", [(77, 16, 2, 1, 256), (300, 64, 6, 4, 512), (9, 256, 8, 8, 1024)])
def test_dispatch_pack_fp8_bit_exact(N, E, k, R, d):
    # plan equal to the oracle's; every send row holds the E4M3 codes and
    # the scale of its token row (oracle quantisation), an all-zero token
    # included
    from paper_2511_11505_amd.block import fp8_row_views
    from workloads.generate import synthetic_topk_ids
    cfg = CONFIGS["tiny"].scaled(n_tokens=N, n_experts=E, top_k=k, ep_size=R, hidden=d, dtype="bf16")
    desc = L.make_desc(cfg)
    ids = synthetic_topk_ids(N, E, k, seed=N + d, device=DEV)
    g = torch.Generator(device=DEV).manual_seed(N)
    x = (torch.randn((N, d), generator=g, device=DEV) *
         torch.exp(4 * torch.rand((N, 1), generator=g, device=DEV) - 2)).to(torch.bfloat16)
    x[N // 2] = 0
    cap = N * k
    i32 = dict(dtype=torch.int32, device=DEV)
    counts, offsets, ro = torch.empty(E, **i32), torch.empty(E + 1, **i32), torch.empty(R + 1, **i32)
    s2r, r2s = torch.empty(cap, **i32), torch.empty(cap, **i32)
    buf = torch.full((cap, d), float("nan"), dtype=torch.bfloat16, device=DEV)   # a bf16-sized buffer
    codes, scales = fp8_row_views(buf, cap, d)
    ws = torch.empty((L.fs_workspace_size(desc, L.FS_OP_DISPATCH_PACK_FP8),), dtype=torch.uint8, device=DEV)
    L.fs_dispatch_pack_fp8(desc, ids, x, counts, offsets, ro, s2r, r2s, codes, scales, ws)
    torch.cuda.synchronize()
    plan = oracle.dispatch_plan(ids.cpu().numpy(), E, R)
    for key, t in (("counts", counts), ("offsets", offsets), ("rank_offsets", ro),
                   ("slot_to_row", s2r), ("row_to_slot", r2s)):
        assert np.array_equal(t.cpu().numpy(), plan[key]), key
    qc, qs = of8.quantize_rows(f64(x).astype(np.float32))
    tok = plan["row_to_slot"] // k
    assert np.array_equal(np_u8(codes), qc[tok])
    assert np.array_equal(scales.cpu().numpy(), qs[tok])


# ---------------------------------------------------------------- FP8 experts inside the block
FP8_BLOCKS = {
    "dsv2lite_f8s": CONFIGS["dsv2lite"].scaled(n_tokens=333, hidden=512, ffn=256, ffn_shared=128,
                                               name="dsv2lite_f8s"),
    "dsv3_prefill_f8s": CONFIGS["dsv3_prefill"].scaled(n_tokens=150, hidden=512, ffn=256,
                                                       ffn_shared=256, ep_rank=3,
                                                       name="dsv3_prefill_f8s"),
    "dsv3_decode_f8s": CONFIGS["dsv3_decode"].scaled(n_tokens=9, hidden=512, ffn=256,
                                                     ffn_shared=256, name="dsv3_decode_f8s"),
}


@pytest.mark.parametrize("name,fo", [(n, False) for n in FP8_BLOCKS] + [("dsv3_decode_f8s", True)])
def test_block_fp8_chain(name, fo):
    # The block with FP8 experts: (a) gate and plan equal the bf16 block's
    # bit for bit, and its send and receive rows (FP8 dispatch) are the
    # codes and scales of the bf16 block's rows; (b) the local expert rows and the shared output
    # equal the standalone FP8 FFN on the same inputs bit for bit (that FFN
    # is checked step by step against the oracle above); (c) Combine and the
    # residual add against the oracle on the GPU's rows; (d) the FP8 block
    # stays within FP8's error of the bf16 block.
    from paper_2511_11505_amd import MoEBlock, fp8_row_views, prepare_remote_sources
    from tests._util import TOL
    from workloads import make_workload
    from workloads.generate import merge_shared

    cfg = FP8_BLOCKS[name]
    wl = make_workload(cfg, DEV)
    sh_gu, sh_dn = merge_shared(wl.sh_gate_up, wl.sh_down)
    comm = torch.cuda.Stream()
    blocks, outs = {}, {}
    for mode in (None, "all"):
        blk = MoEBlock(cfg, wl.w_router, wl.bias, wl.w_gate_up, wl.w_down, sh_gu, sh_dn,
                       device=DEV, fp8=mode, fragment_order=fo)
        if cfg.ep_size > 1:
            blk.set_max_recv_rows(prepare_remote_sources(blk, wl.x_all, wl.w_router, wl.bias,
                                                         wl.y_remote))
        x = wl.x
        partial, out = torch.empty_like(x), x.clone()
        blk.begin(x, partial, comm=comm)
        blk.finish(x, out, comm=comm)
        torch.cuda.synchronize()
        blocks[mode], outs[mode] = blk, (out, partial)
    b16, b8 = blocks[None], blocks["all"]
    R, r, cap, E_loc = cfg.ep_size, cfg.ep_rank, b8.cap, cfg.n_local
    for key in ("topk_ids", "topk_w", "slot_to_row", "row_to_slot", "src_counts", "src_offsets",
                "rank_offsets"):
        assert torch.equal(b16.t[key], b8.t[key]), key
    d = cfg.hidden
    for key, rows_n in (("send", cap), ("recv", R * cap)):
        codes8, scales8 = fp8_row_views(b8.t[key], rows_n, d)
        codes16, scales16 = quantize(b16.t[key])
        assert torch.equal(codes8, codes16) and torch.equal(scales8, scales16), key
    if R > 1:
        assert torch.equal(b16.t["group_offsets"], b8.t["group_offsets"])
        m = int(b8.t["group_offsets"][E_loc].item())
        assert torch.equal(b16.t["group_rows"][:m], b8.t["group_rows"][:m])   # entries past M unwritten
        in_rows, rows, goff = b16.t["recv"], b8.t["group_rows"], b8.t["group_offsets"]
    else:
        in_rows, rows, goff = b16.t["send"], None, b8.t["src_offsets"][r]
    M = int(goff[E_loc].item())
    q = b8.fp8_weights
    xq, xs = quantize(in_rows)
    y_ref = torch.full_like(b8.t["y"], float("nan"))
    desc = b8.desc
    ws = torch.empty((L.fs_workspace_size(desc, L.FS_OP_GROUPED_FFN_FP8, b8.max_recv_rows, cfg.ffn),),
                     dtype=torch.uint8, device=DEV)
    if fo:
        # the block streams the FP8-fragment-ordered codes (decode)
        L.fs_grouped_expert_ffn_fp8_fo(desc, E_loc, cfg.ffn, xq, xs, rows, goff, b8.max_recv_rows,
                                       q["w_gate_up_fp8_fo"], q["s_gate_up"], q["w_down_fp8_fo"],
                                       q["s_down"], y_ref, ws)
    else:
        L.fs_grouped_expert_ffn_fp8(desc, E_loc, cfg.ffn, xq, xs, rows, goff, b8.max_recv_rows,
                                    q["w_gate_up_fp8"], q["s_gate_up"], q["w_down_fp8"], q["s_down"],
                                    y_ref, ws)
    x = wl.x
    xq_s, xs_s = quantize(x)
    sh_ref = torch.empty_like(x)
    W = cfg.n_shared * cfg.ffn_shared
    ws_s = torch.empty((L.fs_workspace_size(desc, L.FS_OP_GROUPED_FFN_FP8, cfg.n_tokens, W),),
                       dtype=torch.uint8, device=DEV)
    L.fs_grouped_expert_ffn_fp8(desc, 1, W, xq_s, xs_s, None, None, cfg.n_tokens,
                                q["ws_gate_up_fp8"], q["ss_gate_up"], q["ws_down_fp8"], q["ss_down"],
                                sh_ref, ws_s)
    torch.cuda.synchronize()
    idx = rows[:M].long() if rows is not None else torch.arange(M, device=DEV)
    assert torch.equal(b8.t["y"][idx], y_ref[idx])
    assert torch.equal(b8.t["shared_out"], sh_ref)
    out8, partial8 = outs["all"]
    s2r = b8.t["slot_to_row"].cpu().numpy()
    routed = oracle.combine(f64(b8.y_ret()), s2r, f64(b8.t["topk_w"]))
    assert rel_err(out8, f64(x) + routed) <= TOL["bf16"]
    assert rel_err(partial8, f64(x) + f64(b8.t["shared_out"])) <= TOL["bf16"]
    rms = lambda a: np.sqrt(np.mean(a * a))
    for a8, a16 in ((b8.t["y"][idx], b16.t["y"][idx]), (b8.t["shared_out"], b16.t["shared_out"])):
        assert rms(f64(a8) - f64(a16)) <= 0.08 * rms(f64(a16))
    for blk in blocks.values():
        blk.close()
