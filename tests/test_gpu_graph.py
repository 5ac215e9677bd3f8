"""HIP-graph capture of the block and of the stacked two-window schedule
(both streams, events only): every replay, with the program's own eager
work and synchronisations between replays, equals the eager result bit for
bit."""

import pytest
import torch

from paper_2511_11505_amd import MoEBlock, prepare_remote_sources
from paper_2511_11505_amd import _lib as L
from paper_2511_11505_amd.stack import LayerStack
from tests.test_gpu_kernels import SMALL
from workloads import make_workload
from workloads.generate import merge_shared, source_tokens, stack_layers

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]
DEV = "cuda"


def block_for(cfg):
    wl = make_workload(cfg, DEV)
    sh_gu = sh_dn = None
    if cfg.n_shared > 0:
        sh_gu, sh_dn = merge_shared(wl.sh_gate_up, wl.sh_down)
    blk = MoEBlock(cfg, wl.w_router, wl.bias, wl.w_gate_up, wl.w_down, sh_gu, sh_dn, device=DEV,
                   with_return=True)
    if cfg.ep_size > 1:
        blk.set_max_recv_rows(prepare_remote_sources(blk, wl.x_all, wl.w_router, wl.bias, wl.y_remote))
    return blk, wl


@pytest.mark.parametrize("name", ["dsv2lite_s", "dsv3_decode_s", "tiny"])
def test_block_graph_replays_equal_eager(name):
    cfg = SMALL[name]
    blk, wl = block_for(cfg)
    comm = torch.cuda.Stream()
    x = wl.x
    other = source_tokens(cfg.scaled(seed=cfg.seed + 77), DEV, cfg.ep_rank)
    out = torch.empty_like(x)

    def step(inp, res):
        s = torch.cuda.current_stream()
        blk.begin(inp, res, compute=s, comm=comm)
        blk.finish(inp, res, compute=s, comm=comm)

    step(x, out)
    torch.cuda.synchronize()
    eager = out.clone()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g):
            step(x, out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    scratch = torch.empty_like(x)
    for i in range(3):
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {i}"
        step(other, scratch)          # eager work on the same block between replays
        torch.cuda.synchronize()
    blk.close()


@pytest.mark.parametrize("link", [False, True])
def test_stack_graph_replays_equal_eager(link):
    # link: the Dispatch and Combine stand-ins captured as link-paced copy
    # kernels (fs_standin_link), whose pacing starts from each replay's own
    # clock
    cfg = SMALL["dsv2lite_s"]
    layers = stack_layers(cfg, 2, DEV)
    st = LayerStack(cfg, layers, device=DEV, merge_shared=merge_shared)
    comm = torch.cuda.Stream()
    x = layers[0][1].x
    eager = st.farskip(x, comm=comm).clone()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with L.standin_link(*((7, 153e9, 32) if link else (0,))):
        with torch.cuda.stream(side):
            with torch.cuda.graph(g):
                res = st.farskip(x, compute=torch.cuda.current_stream(), comm=comm)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for i in range(3):
        res.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(res, eager), f"replay {i}"
        st.regular(x)                 # eager work between replays
        torch.cuda.synchronize()
    st.close()
