"""GPU parity of the whole FarSkip MoE block (fs_moe_block_forward) against
the oracle, plus the invariants the FarSkip connectivity fixes (Section 3,
Eqs. 6-8) and the race check of the two-stream schedule."""

import numpy as np
import pytest
import torch

import oracle
from paper_2511_11505_amd import MoEBlock, prepare_remote_sources
from paper_2511_11505_amd import _lib as L
from tests._util import TOL, f64, rel_err
from tests.test_gpu_kernels import SMALL
from workloads import make_workload
from workloads.generate import merge_shared

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]
DEV = "cuda"


def build_block(cfg, wl, w_down=None):
    sh_gu = sh_dn = None
    if cfg.n_shared > 0:
        sh_gu, sh_dn = merge_shared(wl.sh_gate_up, wl.sh_down)
    blk = MoEBlock(cfg, wl.w_router, wl.bias, wl.w_gate_up,
                   wl.w_down if w_down is None else w_down, sh_gu, sh_dn, device=DEV)
    if cfg.ep_size > 1:
        M = prepare_remote_sources(blk, wl.x_all, wl.w_router, wl.bias, wl.y_remote)
        blk.set_max_recv_rows(M)
    return blk


def dtype_id(cfg):
    return L.FS_F32 if cfg.dtype == "f32" else L.FS_BF16


def farskip_gpu(blk, wl, comm=None):
    """BEGIN -> next layer on the partial input -> FINISH (deferred add)."""
    cfg = blk.cfg
    x = wl.x
    partial, nxt, out = torch.empty_like(x), torch.empty_like(x), torch.empty_like(x)
    blk.begin(x, partial, comm=comm)
    L.fs_dense_linear(dtype_id(cfg), cfg.n_tokens, cfg.hidden, cfg.hidden, partial, wl.w_next, nxt)
    L.fs_farskip_residual(blk.desc, out, partial, nxt)
    blk.finish(x, out, comm=comm)
    torch.cuda.synchronize()
    return out, partial, nxt


def regular_gpu(blk, wl):
    """The regular stream (Eq. 6): the next layer reads the full o_k."""
    cfg = blk.cfg
    x = wl.x
    r1, nxt, out = torch.empty_like(x), torch.empty_like(x), torch.empty_like(x)
    blk.run(L.FS_PHASE_ALL, x, r1, r1)
    L.fs_dense_linear(dtype_id(cfg), cfg.n_tokens, cfg.hidden, cfg.hidden, r1, wl.w_next, nxt)
    L.fs_farskip_residual(blk.desc, out, r1, nxt)
    torch.cuda.synchronize()
    return out


def oracle_block(cfg, wl, w_down=None):
    np32 = lambda t: None if t is None else f64(t)
    return oracle.moe_block(cfg, f64(wl.x_all), f64(wl.w_router), np32(wl.bias), f64(wl.w_gate_up),
                            f64(wl.w_down) if w_down is None else f64(w_down), np32(wl.sh_gate_up),
                            np32(wl.sh_down), np32(wl.y_remote))


@pytest.mark.parametrize("name", list(SMALL))
def test_block_matches_oracle(name):
    cfg = SMALL[name]
    wl = make_workload(cfg, DEV)
    blk = build_block(cfg, wl)
    comm = torch.cuda.Stream()
    out, partial, nxt = farskip_gpu(blk, wl, comm=comm)
    ref = oracle_block(cfg, wl)
    me = ref["me"]
    near = me["near_tie"]
    ids = blk.t["topk_ids"].cpu().numpy()
    far = ~near
    assert np.array_equal(ids[far], me["ids"][far]), "routing differs on non-tie tokens"
    any_near = any(s["near_tie"].any() for s in ref["src"])
    if not any_near:
        plan = me["plan"]
        r = cfg.ep_rank
        assert np.array_equal(blk.t["slot_to_row"].cpu().numpy(), plan["slot_to_row"])
        assert np.array_equal(blk.t["row_to_slot"].cpu().numpy(), plan["row_to_slot"])
        assert np.array_equal(blk.t["rank_offsets"].cpu().numpy(), plan["rank_offsets"])
        assert np.array_equal(blk.t["src_counts"].cpu().numpy(), ref["src_counts"])
        assert np.array_equal(blk.t["src_offsets"].cpu().numpy(), ref["src_offsets"])
        assert np.array_equal(blk.t["send"].cpu().float().numpy(), me["send"].astype(np.float32))
        if cfg.ep_size > 1:
            M = len(ref["group_rows"])
            assert np.array_equal(blk.t["group_rows"][:M].cpu().numpy(), ref["group_rows"])
            assert np.array_equal(blk.t["group_offsets"].cpu().numpy(), ref["group_offsets"])
            rows = ref["group_rows"]
        else:
            rows = np.arange(cfg.cap)
        # every expert-output row this GPU computed
        assert rel_err(f64(blk.t["y"])[rows], ref["y"][rows]) <= TOL[cfg.dtype]
        assert blk.max_recv_rows == len(rows)
    want_out, want_partial, want_next = oracle.farskip_pair(ref["x"], ref["shared"], ref["routed"],
                                                            f64(wl.w_next))
    tol = TOL[cfg.dtype]
    assert rel_err(partial, want_partial) <= tol
    assert rel_err(nxt, want_next) <= tol
    assert rel_err(f64(out)[far], want_out[far]) <= tol
    blk.close()


@pytest.mark.parametrize("name", ["tiny", "dsv2lite_s", "dsv3_prefill_s"])
def test_two_stream_run_is_race_free(name):
    # The copy on the comm stream is ordered by events: a NaN-poisoned
    # receive slot must leave no trace, and the result must equal the
    # serial run bit for bit.
    cfg = SMALL[name]
    wl = make_workload(cfg, DEV)
    blk = build_block(cfg, wl)
    serial, _, _ = farskip_gpu(blk, wl, comm=None)
    r = cfg.ep_rank
    slot = blk.t["recv"][r * blk.cap:(r + 1) * blk.cap]
    comm = torch.cuda.Stream()
    for _ in range(3):
        slot.fill_(float("nan"))
        torch.cuda.synchronize()
        over, _, _ = farskip_gpu(blk, wl, comm=comm)
        assert torch.equal(over, serial)
        assert not torch.isnan(over).any()
    blk.close()


@pytest.mark.parametrize("name", ["tiny", "dsv2lite_s", "dsv3_prefill_s", "dsv3_decode_s"])
def test_shared_experts_beside_routed_equal_default(name):
    # The shared experts may run on a side stream while the routed experts
    # run (GATE; SHARED on the side stream; EXPERTS; COMBINE once SHARED is
    # done): the same kernels, disjoint workspace regions, so the block's
    # output equals the default order bit for bit.  The partial input is
    # NaN-poisoned first, so COMBINE reading it before SHARED wrote it shows.
    cfg = SMALL[name]
    wl = make_workload(cfg, DEV)
    blk = build_block(cfg, wl)
    x = wl.x
    compute = torch.cuda.current_stream()
    comm, side = torch.cuda.Stream(), torch.cuda.Stream()
    want = torch.empty_like(x)
    blk.begin(x, want, compute=compute, comm=comm)
    blk.finish(x, want, compute=compute, comm=comm)
    torch.cuda.synchronize()
    for _ in range(3):
        got = torch.full_like(x, float("nan"))
        torch.cuda.synchronize()
        blk.phase(L.FS_PHASE_GATE, x, compute=compute, comm=comm)
        side.wait_stream(compute)
        blk.phase(L.FS_PHASE_SHARED, x, partial_out=got, compute=side, comm=comm)
        blk.phase(L.FS_PHASE_EXPERTS, x, compute=compute, comm=comm)
        compute.wait_stream(side)
        blk.phase(L.FS_PHASE_COMBINE, x, residual_io=got, compute=compute, comm=comm)
        torch.cuda.synchronize()
        assert not torch.isnan(got).any()
        assert torch.equal(got, want)
    blk.close()


@pytest.mark.parametrize("name", ["tiny", "scout_s", "dsv3_decode_s"])
def test_zero_moe_output_farskip_equals_regular(name):
    # Eq. 6 vs Eq. 7 with a zero routed output: the two connectivities are
    # the same computation, bit for bit on the GPU.
    cfg = SMALL[name]
    wl = make_workload(cfg, DEV)
    zero_down = torch.zeros_like(wl.w_down)
    blk = build_block(cfg, wl, w_down=zero_down)
    if cfg.ep_size > 1:
        blk.y_ret().zero_()
    fs_out, _, _ = farskip_gpu(blk, wl)
    reg_out = regular_gpu(blk, wl)
    assert torch.equal(fs_out, reg_out)
    blk.close()


def test_farskip_differs_from_regular_only_through_the_dropped_input():
    # With a non-zero routed output the next layer's input differs by exactly
    # the routed output: out_fs - out_reg = W_next (partial) - W_next (partial + routed).
    cfg = SMALL["tiny"]
    wl = make_workload(cfg, DEV)
    blk = build_block(cfg, wl)
    fs_out, partial, _ = farskip_gpu(blk, wl)
    reg_out = regular_gpu(blk, wl)
    ref = oracle_block(cfg, wl)
    wn = f64(wl.w_next)
    want = oracle.dense_linear(ref["x"] + ref["shared"], wn) - oracle.dense_linear(
        ref["x"] + ref["shared"] + ref["routed"], wn)
    got = f64(fs_out) - f64(reg_out)
    # Each output is an fp32 sum rounded a few times (residual adds, the
    # next-layer GEMM): the difference carries at most a few ulps of the
    # outputs' magnitude, which cancellation does not shrink.
    ulp = 2.0 ** -23 * max(np.abs(f64(fs_out)).max(), np.abs(f64(reg_out)).max())
    assert np.max(np.abs(got - want)) <= 16 * ulp
    assert np.abs(want).max() > 100 * 16 * ulp   # the dropped input is visible
    blk.close()
