"""One FarSkip MoE block on one EP rank: caller-side buffers around the C ABI.

``MoEBlock`` owns the device buffers and workspace of one block and calls
``fs_moe_block_forward`` for its two phases (Section 3 connectivity, Section
4.1 schedule).  ``prepare_remote_sources`` sets up, on one GPU, what the
other EP ranks would have sent: their routing and packed send buffers land
in their receive slots, their counts in the source-count rows, and the
Combine return rows of other ranks' experts in this rank's return slot.
With ``fp8`` the expert weights are quantised once, at construction, by the
library's row quantiser, and the block runs those experts in FP8.
All arithmetic runs in the library's kernels; torch only allocates memory.
"""

import torch

from . import _lib as L
from ._lib import make_desc


def _dt(cfg):
    return torch.float32 if cfg.dtype == "f32" else torch.bfloat16


def _quantize(w):
    """E4M3 codes and per-row scales of a weight tensor [..., cols] (rows
    are its output channels), through the library's quantiser."""
    rows, cols = w.numel() // w.shape[-1], w.shape[-1]
    codes = torch.empty(w.shape, dtype=torch.uint8, device=w.device)
    scales = torch.empty(w.shape[:-1], dtype=torch.float32, device=w.device)
    L.fs_quantize_fp8(L.FS_F32 if w.dtype == torch.float32 else L.FS_BF16, rows, cols,
                      w.contiguous(), codes, scales)
    return codes, scales


def fragment_ordered(w):
    """MFMA fragment-order copy of bf16 weight matrices [..., rows, cols]
    (fs_expert_weights_fragment_order)."""
    rows, cols = w.shape[-2], w.shape[-1]
    out = torch.empty_like(w)
    L.fs_expert_weights_fragment_order(L.FS_BF16, w.numel() // (rows * cols), rows, cols,
                                       w.contiguous(), out)
    return out


def fragment_ordered_fp8(codes):
    """FP8 fragment-order copy of E4M3 code matrices [..., rows, cols]
    (fs_expert_weights_fragment_order_fp8)."""
    rows, cols = codes.shape[-2], codes.shape[-1]
    out = torch.empty_like(codes)
    L.fs_expert_weights_fragment_order_fp8(codes.numel() // (rows * cols), rows, cols,
                                           codes.contiguous(), out)
    return out


def fp8_row_views(buf, rows, d):
    """Views of an FP8 row buffer of `rows` rows held in the device tensor
    buf (any dtype, contiguous): codes [rows, d] uint8 at byte 0, scales
    [rows] fp32 at byte rows * d rounded up to a multiple of 256."""
    raw = buf.reshape(-1).view(torch.uint8)
    at = (rows * d + 255) // 256 * 256
    if raw.numel() < at + 4 * rows:
        raise ValueError("buffer too small for the FP8 rows")
    return raw[:rows * d].view(rows, d), raw[at:at + 4 * rows].view(torch.float32)


class MoEBlock:
    def __init__(self, cfg, w_router, sel_bias, w_gate_up, w_down, ws_gate_up=None, ws_down=None,
                 max_recv_rows=None, device="cuda", with_comm=True, with_return=False, fp8=None,
                 fragment_order=False):
        """fp8: None (bf16 experts), "routed" (FP8 routed experts) or "all"
        (FP8 routed and shared experts).  fragment_order: also keep the
        routed experts' weights (and with fp8 their codes) in MFMA fragment
        order (converted once, by the library), which the block streams for
        passes of few rows per expert (decode)."""
        if fp8 not in (None, "routed", "all"):
            raise ValueError(f"fp8 must be None, 'routed' or 'all', not {fp8!r}")
        self.cfg = cfg
        self.fp8 = fp8
        self.desc = make_desc(cfg)
        R, N, d, E, k = cfg.ep_size, cfg.n_tokens, cfg.hidden, cfg.n_experts, cfg.top_k
        cap = N * k
        self.cap = cap
        self.max_recv_rows = cap if max_recv_rows is None else int(max_recv_rows)
        dt = _dt(cfg)
        i32 = torch.int32
        dev = device
        self.t = dict(
            logits=torch.empty((N, E), dtype=torch.float32, device=dev),
            topk_ids=torch.empty((N, k), dtype=i32, device=dev),
            topk_w=torch.empty((N, k), dtype=torch.float32, device=dev),
            src_counts=torch.zeros((R, E), dtype=i32, device=dev),
            src_offsets=torch.zeros((R, E + 1), dtype=i32, device=dev),
            rank_offsets=torch.empty((R + 1,), dtype=i32, device=dev),
            slot_to_row=torch.empty((cap,), dtype=i32, device=dev),
            row_to_slot=torch.empty((cap,), dtype=i32, device=dev),
            send=torch.empty((cap, d), dtype=dt, device=dev),
            recv=torch.empty((R * cap, d), dtype=dt, device=dev) if (R > 1 or with_comm) else None,
            group_rows=torch.empty((R * cap,), dtype=i32, device=dev) if R > 1 else None,
            group_offsets=torch.empty((E // R + 1,), dtype=i32, device=dev) if R > 1 else None,
            y=torch.empty((R * cap, d), dtype=dt, device=dev),
            shared_out=torch.empty((N, d), dtype=dt, device=dev) if cfg.n_shared > 0 else None,
            ret=torch.empty((cap, d), dtype=dt, device=dev) if with_return else None,
        )
        q = dict()
        if fp8:
            q["w_gate_up_fp8"], q["s_gate_up"] = _quantize(w_gate_up)
            q["w_down_fp8"], q["s_down"] = _quantize(w_down)
            if fp8 == "all" and ws_gate_up is not None:
                q["ws_gate_up_fp8"], q["ss_gate_up"] = _quantize(ws_gate_up)
                q["ws_down_fp8"], q["ss_down"] = _quantize(ws_down)
        if fragment_order and fp8:
            q["w_gate_up_fp8_fo"] = fragment_ordered_fp8(q["w_gate_up_fp8"])
            q["w_down_fp8_fo"] = fragment_ordered_fp8(q["w_down_fp8"])
        elif fragment_order:
            q["w_gate_up_fo"] = fragment_ordered(w_gate_up)
            q["w_down_fo"] = fragment_ordered(w_down)
        self.fp8_weights = q
        self.weights_keep = (w_router, sel_bias, w_gate_up, w_down, ws_gate_up, ws_down)
        self.weights = L.fs_moe_weights(L.ptr(w_router), L.ptr(sel_bias), L.ptr(w_gate_up),
                                        L.ptr(w_down), L.ptr(ws_gate_up), L.ptr(ws_down),
                                        *[L.ptr(q.get(n)) for n, _ in L.fs_moe_weights._fields_[6:]])
        self.buffers = L.fs_block_buffers(*[L.ptr(self.t[n]) for n, _ in L.fs_block_buffers._fields_])
        self.ws_op = L.FS_OP_BLOCK_FP8 if fp8 else L.FS_OP_BLOCK
        ws_bytes = L.fs_workspace_size(self.desc, self.ws_op, self.max_recv_rows)
        self.ws = torch.empty((max(ws_bytes, 256),), dtype=torch.uint8, device=dev)
        self.sync = L.fs_block_sync_create()

    def close(self):
        if self.sync:
            L.fs_block_sync_destroy(self.sync)
            self.sync = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_max_recv_rows(self, m):
        m = int(m)
        if m != self.max_recv_rows:
            self.max_recv_rows = m
            ws_bytes = L.fs_workspace_size(self.desc, self.ws_op, m)
            if ws_bytes > self.ws.numel():
                self.ws = torch.empty((ws_bytes,), dtype=torch.uint8, device=self.ws.device)

    def run(self, phase, residual_in, partial_out, residual_io, compute=None, comm=None):
        L.fs_moe_block_forward(self.desc, phase, self.weights, residual_in, partial_out,
                               residual_io, self.buffers, self.max_recv_rows, self.ws,
                               sync=self.sync if comm is not None else None,
                               compute=compute, comm=comm)

    def phase(self, phase, residual_in, partial_out=None, residual_io=None, compute=None,
              comm=None):
        """One of the finer phases (FS_PHASE_GATE / SHARED / EXPERTS / COMBINE)."""
        self.run(phase, residual_in, partial_out, residual_io, compute, comm)

    def begin(self, residual_in, partial_out, compute=None, comm=None):
        self.run(L.FS_PHASE_BEGIN, residual_in, partial_out, None, compute, comm)

    def finish(self, residual_in, residual_io, compute=None, comm=None):
        self.run(L.FS_PHASE_FINISH, residual_in, None, residual_io, compute, comm)

    def y_ret(self):
        r = self.cfg.ep_rank
        return self.t["y"][r * self.cap:(r + 1) * self.cap]


def prepare_remote_sources(block, x_all, w_router, sel_bias, y_remote, stream=None):
    """Single-GPU stand-in for the other EP ranks (R > 1).

    For every source rank s != r, run the library's router + top-k and plan
    + pack on that rank's tokens; the packed send buffer is written straight
    into receive slot s and the counts / offsets into row s.  With FP8
    routed experts the sources pack FP8 rows (fs_dispatch_pack_fp8) into
    slot s of the receive buffer's codes and scales.  Fill this
    rank's Combine-return slot with the rows other ranks' experts send back.
    Then run this rank's routing once to learn how many rows land on the
    local experts (what the counts exchange tells the receiver) and return
    that number."""
    cfg = block.cfg
    R, r, N, E, k = cfg.ep_size, cfg.ep_rank, cfg.n_tokens, cfg.n_experts, cfg.top_k
    cap = block.cap
    t = block.t
    dev = t["send"].device
    desc = block.desc
    ids = torch.empty((N, k), dtype=torch.int32, device=dev)
    w = torch.empty((N, k), dtype=torch.float32, device=dev)
    ro = torch.empty((R + 1,), dtype=torch.int32, device=dev)
    s2r = torch.empty((cap,), dtype=torch.int32, device=dev)
    r2s = torch.empty((cap,), dtype=torch.int32, device=dev)
    ws_r = torch.empty((max(L.fs_workspace_size(desc, L.FS_OP_ROUTER_TOPK), 256),), dtype=torch.uint8, device=dev)
    ws_p = torch.empty((max(L.fs_workspace_size(desc, L.FS_OP_DISPATCH_PACK), 256),), dtype=torch.uint8, device=dev)
    fp8 = block.fp8 is not None
    if fp8:
        # FP8 routed experts: every source packs FP8 rows, into its slot of
        # the receive buffer's codes and scales
        ws_p = torch.empty((max(L.fs_workspace_size(desc, L.FS_OP_DISPATCH_PACK_FP8), 256),),
                           dtype=torch.uint8, device=dev)
        recv_codes, recv_scales = fp8_row_views(t["recv"], R * cap, cfg.hidden)
        send_codes, send_scales = fp8_row_views(t["send"], cap, cfg.hidden)
    for s in range(R):
        L.fs_router_topk(desc, x_all[s], w_router, sel_bias, None, None, ids, w, ws_r, stream)
        if fp8:
            if s != r:
                codes_s, scales_s = recv_codes[s * cap:(s + 1) * cap], recv_scales[s * cap:(s + 1) * cap]
            else:
                codes_s, scales_s = send_codes, send_scales
            L.fs_dispatch_pack_fp8(desc, ids, x_all[s], t["src_counts"][s], t["src_offsets"][s], ro,
                                   s2r, r2s, codes_s, scales_s, ws_p, stream)
        else:
            send_s = t["recv"][s * cap:(s + 1) * cap] if s != r else t["send"]
            L.fs_dispatch_pack(desc, ids, x_all[s], t["src_counts"][s], t["src_offsets"][s], ro, s2r,
                               r2s, send_s, ws_p, stream)
    if y_remote is not None:
        block.y_ret().copy_(y_remote)
    torch.cuda.synchronize()
    lo = r * (E // R)
    return int(t["src_counts"][:, lo:lo + E // R].sum().item())
