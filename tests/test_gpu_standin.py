"""GPU checks of the link-paced stand-in copies (fs_standin_link): the
bytes arrive bit for bit on every copy path (16-, 4-byte units, partial
chunks, tail bytes, one or many workgroups), the copy takes the time of the
modelled collective, and a block or a stack computes the same result with
the link model on as with HBM-speed copies."""

import pytest
import torch

from paper_2511_11505_amd import _lib as L
from tests.test_gpu_kernels import SMALL

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]
DEV = "cuda"


def ar_desc(n_tokens, hidden, dtype):
    cfg = SMALL["tiny"].scaled(n_tokens=n_tokens, hidden=hidden, dtype=dtype)
    return L.make_desc(cfg)


@pytest.mark.parametrize("n,d,dtype,wgs", [(1, 128, "f32", 64), (64, 128, "bf16", 64),
                                           (64, 128, "f32", 64), (128, 128, "f32", 64),
                                           (128, 128, "f32", 1), (4099, 1024, "bf16", 64),
                                           (4099, 1024, "bf16", 5), (777, 384, "f32", 3)])
def test_paced_allreduce_copy_is_exact(n, d, dtype, wgs):
    # sizes: one partial chunk (512 bytes, 16 KB), exactly one and two
    # chunks (32 KB each), many rounds of chunks over 64, 5, 3 and one
    # workgroup(s)
    desc = ar_desc(n, d, dtype)
    dt = torch.float32 if dtype == "f32" else torch.bfloat16
    g = torch.Generator(device="cpu").manual_seed(n * 31 + d)
    src = torch.randn((n, d), generator=g).to(dt).to(DEV)
    dst = torch.full_like(src, float("nan"))
    with L.standin_link(7, 153e9, wgs):
        L.fs_allreduce_standin(desc, dst, src)
    torch.cuda.synchronize()
    assert torch.equal(dst.view(torch.uint8 if dtype == "bf16" else torch.int32),
                       src.view(torch.uint8 if dtype == "bf16" else torch.int32))
    assert L.fs_standin_link_get() == (0, 0.0, 0)


def test_paced_copy_takes_the_link_time():
    # a 64 MiB ring all-reduce over 8 GPUs joined by 153 GB/s links: twice
    # B / (8 * 153 GB/s); the schedule forbids finishing early, and alone on
    # the GPU 64 workgroups keep up with it
    n, d = 32768, 1024
    desc = ar_desc(n, d, "bf16")
    src = torch.ones((n, d), dtype=torch.bfloat16, device=DEV)
    dst = torch.empty_like(src)
    want_us = 2 * src.numel() * 2 / (8 * 153e9) * 1e6
    s = torch.cuda.current_stream()
    times = []
    with L.standin_link(7, 153e9, 64):
        for _ in range(3):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(s)
            L.fs_allreduce_standin(desc, dst, src, stream=s)
            b.record(s)
            torch.cuda.synchronize()
            times.append(a.elapsed_time(b) * 1e3)
    print(f"[paced copy] 64 MiB all-reduce stand-in: model {want_us:.1f} us, measured "
          f"{', '.join(f'{t:.1f}' for t in times)} us")
    assert min(times) >= 0.98 * want_us
    assert min(times) <= 1.3 * want_us + 20.0
    assert torch.equal(dst, src)


@pytest.mark.parametrize("rank", [0, 1])
def test_block_fp8_dispatch_with_link_model(rank):
    # FP8 routed experts on 8 ranks with 1998 rows per slot: the Dispatch
    # copy of the scales (7992 bytes) takes 16-byte units and an 8-byte tail
    # on rank 0, and 4-byte units on rank 1, whose slot starts 8 bytes past
    # a 16-byte boundary.  The block computes the same bits either way.
    from paper_2511_11505_amd import MoEBlock, fp8_row_views, prepare_remote_sources
    from tests.test_gpu_fp8 import FP8_BLOCKS
    from workloads import make_workload
    from workloads.generate import merge_shared

    cfg = FP8_BLOCKS["dsv2lite_f8s"].scaled(ep_size=8, ep_rank=rank, name=f"dsv2lite_f8s_r{rank}")
    assert cfg.cap * 4 % 16 == 8 and cfg.ep_rank * cfg.cap * 4 % 16 == 8 * rank
    wl = make_workload(cfg, DEV)
    sh_gu, sh_dn = merge_shared(wl.sh_gate_up, wl.sh_down)
    blk = MoEBlock(cfg, wl.w_router, wl.bias, wl.w_gate_up, wl.w_down, sh_gu, sh_dn, device=DEV,
                   fp8="routed")
    blk.set_max_recv_rows(prepare_remote_sources(blk, wl.x_all, wl.w_router, wl.bias, wl.y_remote))
    comm = torch.cuda.Stream()
    res = []
    for link in (False, True):
        partial, out = torch.empty_like(wl.x), wl.x.clone()
        if link:
            # slot r of the receive buffer (codes and scales) must be
            # written again by the copy
            codes, scales = fp8_row_views(blk.t["recv"], cfg.ep_size * cfg.cap, cfg.hidden)
            codes[rank * cfg.cap:(rank + 1) * cfg.cap].fill_(0xFF)
            scales[rank * cfg.cap:(rank + 1) * cfg.cap].fill_(float("nan"))
            with L.standin_link(7, 153e9, 16):
                blk.begin(wl.x, partial, comm=comm)
                blk.finish(wl.x, out, comm=comm)
        else:
            blk.begin(wl.x, partial, comm=comm)
            blk.finish(wl.x, out, comm=comm)
        torch.cuda.synchronize()
        res.append((out.clone(), partial.clone(), blk.t["y"].clone(), blk.t["recv"].clone()))
    for a, b in zip(*res):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    blk.close()
