"""Stacked layers of the replicated-activation (all-reduce) inference variant
on one GPU: the FarSkip schedule of Section 4.2 and the regular one, both
driving the library's entry points.

Every rank holds all N tokens.  Rank r runs the tensor-parallel share of
the attention stand-in (rows of W_a / columns of W_b) and of the shared
experts (a block of their merged hidden units), routes every token, runs
its own experts on the rows that selected them (gathered straight from the
token matrix) and combines them into a partial sum.  Partial sums are
all-reduced; on one GPU the all-reduce is `fs_allreduce_standin`, a copy on
the stream the collective would use.

FarSkip, layer k (p: partial residual, o: full residual; Eqs. 7, 8):
    attn  = (p Wa_r^T) Wb_r^T                on compute, overlapping AR(routed_{k-1})
    join AR(routed_{k-1});  o = p + AR(routed_{k-1})
    shared = shared_r(o); msg = attn + shared; AR(msg) on comm
    router, plan, local rows, gathered experts, partial Combine -> routed_k
                                             (overlapping AR(msg))
    join AR(msg); p = o + AR(msg); AR(routed_k) on comm
The last layer's routed all-reduce is joined at the end: o = p + AR(routed).
Tab. 5: the attention + shared all-reduce hides behind the routed experts,
the routed all-reduce behind the next attention.

Regular (Eq. 6): o' = o + AR(attn(o)); o = o' + AR(shared(o') + routed(o')),
each all-reduce blocking on `compute`.

This module only orders the calls and owns the buffers.
"""

import torch

from . import _lib as L


class ReplicatedStack:
    def __init__(self, cfg, layers, device="cuda"):
        """layers: one dict per layer of device tensors: w_router [E, d],
        bias [E] fp32 or None, w_gate_up [E/R, 2F, d] and w_down [E/R, d, F]
        (this rank's experts), sh_gate_up [2W/R, d] and sh_down [d, W/R]
        (this rank's block of the merged shared experts, or None), w_a
        [d/R, d] and w_b [d, d/R] (this rank's attention stand-in block)."""
        if cfg.ep_mode != "allreduce":
            raise ValueError("ReplicatedStack needs a replicated-activation workload")
        self.cfg, self.layers = cfg, layers
        self.desc = L.make_desc(cfg)
        self.dtype_id = L.FS_F32 if cfg.dtype == "f32" else L.FS_BF16
        N, d, E, k, R = cfg.n_tokens, cfg.hidden, cfg.n_experts, cfg.top_k, cfg.ep_size
        E_loc = cfg.n_local
        self.max_rows = N * min(k, E_loc)
        self.w_sh = layers[0]["sh_down"].shape[1] if layers[0].get("sh_down") is not None else 0
        dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
        i32 = dict(dtype=torch.int32, device=device)
        nd = lambda: torch.empty((N, d), dtype=dt, device=device)
        self.ids = torch.empty((N, k), **i32)
        self.w = torch.empty((N, k), dtype=torch.float32, device=device)
        self.counts = torch.empty((E,), **i32)
        self.offsets = torch.empty((E + 1,), **i32)
        self.rank_offsets = torch.empty((R + 1,), **i32)
        self.s2r = torch.empty((N * k,), **i32)
        self.r2s = torch.empty((N * k,), **i32)
        self.local_tokens = torch.empty((max(self.max_rows, 1),), **i32)
        self.local_offsets = torch.empty((E_loc + 1,), **i32)
        self.y_local = torch.empty((max(self.max_rows, 1), d), dtype=dt, device=device)
        self.a = torch.empty((N, d // R), dtype=dt, device=device)
        self.attn, self.shared, self.routed, self.msg = nd(), nd(), nd(), nd()
        self.ar_msg, self.ar_routed, self.ar_attn = nd(), nd(), nd()
        self.p, self.o, self.o1 = nd(), nd(), nd()
        u8 = lambda n: torch.empty((max(int(n), 1),), dtype=torch.uint8, device=device)
        self.ws_router = u8(L.fs_workspace_size(self.desc, L.FS_OP_ROUTER_TOPK))
        self.ws_plan = u8(L.fs_workspace_size(self.desc, L.FS_OP_DISPATCH_PACK))
        ffn_ws = L.fs_workspace_size(self.desc, L.FS_OP_GROUPED_FFN, self.max_rows, cfg.ffn)
        if self.w_sh:
            ffn_ws = max(ffn_ws, L.fs_workspace_size(self.desc, L.FS_OP_GROUPED_FFN, N, self.w_sh))
        self.ws_ffn = u8(ffn_ws)
        # per-layer copies of the selections, kept when a schedule runs with
        # keep_ids=True (for checking routing against a reference)
        self.kept_ids = []
        self.kept_logits = []

    def close(self):
        pass

    # ------------------------------------------------------------ one layer's parts
    def _attention(self, p, lw, stream):
        N, d, R = self.cfg.n_tokens, self.cfg.hidden, self.cfg.ep_size
        L.fs_dense_linear(self.dtype_id, N, d // R, d, p, lw["w_a"], self.a, stream=stream)
        L.fs_dense_linear(self.dtype_id, N, d, d // R, self.a, lw["w_b"], self.attn, stream=stream)

    def _shared(self, o, lw, stream):
        """shared_r(o) into self.shared; returns it (None without shared experts)."""
        if not self.w_sh:
            return None
        L.fs_grouped_expert_ffn(self.desc, 1, self.w_sh, o, None, None, self.cfg.n_tokens,
                                lw["sh_gate_up"], lw["sh_down"], self.shared, self.ws_ffn,
                                stream=stream)
        return self.shared

    def _routed(self, o, lw, stream, keep_ids=False):
        """This rank's routed partial sum on o into self.routed."""
        c = self.cfg
        logits = None
        if keep_ids:
            if getattr(self, "logits", None) is None:
                self.logits = torch.empty((c.n_tokens, c.n_experts), dtype=torch.float32,
                                          device=self.ids.device)
            logits = self.logits
        L.fs_router_topk(self.desc, o, lw["w_router"], lw.get("bias"), None, logits, self.ids,
                         self.w, self.ws_router, stream=stream)
        if keep_ids:
            with torch.cuda.stream(stream):
                self.kept_ids.append(self.ids.clone())
                self.kept_logits.append(self.logits.clone())
        L.fs_dispatch_pack(self.desc, self.ids, None, self.counts, self.offsets, self.rank_offsets,
                           self.s2r, self.r2s, None, self.ws_plan, stream=stream)
        L.fs_local_rows(self.desc, self.offsets, self.rank_offsets, self.r2s, self.local_tokens,
                        self.local_offsets, stream=stream)
        L.fs_grouped_expert_ffn_gathered(self.desc, c.n_local, c.ffn, o, self.local_tokens,
                                         self.local_offsets, self.max_rows, lw["w_gate_up"],
                                         lw["w_down"], self.y_local, self.ws_ffn, stream=stream)
        L.fs_combine_partial(self.desc, self.y_local, self.s2r, self.rank_offsets, self.w,
                             self.routed, stream=stream)

    def _add(self, out, a, b, stream, c=None):
        L.fs_farskip_residual(self.desc, out, a, b, c, stream=stream)

    # ------------------------------------------------------------ schedules
    def farskip(self, x, compute=None, comm=None, keep_ids=False):
        """FarSkip schedule on input x; returns the buffer holding o_{L-1}.
        With comm None the same order runs on one stream."""
        compute = compute or torch.cuda.current_stream()
        self.kept_ids = []
        self.kept_logits = []
        side = comm or compute
        p = o = x
        routed_done = None
        for k, lw in enumerate(self.layers):
            self._attention(p, lw, compute)
            if k > 0:
                if routed_done is not None:
                    compute.wait_event(routed_done)
                self._add(self.o, p, self.ar_routed, compute)
                o = self.o
            sh = self._shared(o, lw, compute)
            msg = self.attn
            if sh is not None:
                self._add(self.msg, self.attn, sh, compute)
                msg = self.msg
            msg_ready = torch.cuda.Event()
            msg_ready.record(compute)
            side.wait_event(msg_ready)
            L.fs_allreduce_standin(self.desc, self.ar_msg, msg, stream=side)
            msg_done = torch.cuda.Event()
            msg_done.record(side)
            self._routed(o, lw, compute, keep_ids)
            compute.wait_event(msg_done)
            self._add(self.p, o, self.ar_msg, compute)
            p = self.p
            routed_ready = torch.cuda.Event()
            routed_ready.record(compute)
            side.wait_event(routed_ready)
            L.fs_allreduce_standin(self.desc, self.ar_routed, self.routed, stream=side)
            routed_done = torch.cuda.Event()
            routed_done.record(side)
        compute.wait_event(routed_done)
        self._add(self.o, p, self.ar_routed, compute)
        return self.o

    def regular(self, x, compute=None, keep_ids=False):
        """Regular schedule on input x, every all-reduce blocking on
        `compute`; returns the buffer holding o_{L-1}."""
        compute = compute or torch.cuda.current_stream()
        self.kept_ids = []
        self.kept_logits = []
        o = x
        for lw in self.layers:
            self._attention(o, lw, compute)
            L.fs_allreduce_standin(self.desc, self.ar_attn, self.attn, stream=compute)
            self._add(self.o1, o, self.ar_attn, compute)
            sh = self._shared(self.o1, lw, compute)
            self._routed(self.o1, lw, compute, keep_ids)
            msg = self.routed
            if sh is not None:
                self._add(self.msg, sh, self.routed, compute)
                msg = self.msg
            L.fs_allreduce_standin(self.desc, self.ar_msg, msg, stream=compute)
            self._add(self.o, self.o1, self.ar_msg, compute)
            o = self.o
        return self.o
