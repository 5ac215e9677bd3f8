"""Stacked FarSkip MoE layers on one GPU: the two-window schedule of
Section 4.1 and the regular schedule, both driving the library's phases.

Each layer is an attention stand-in (two bias-free d x d linears: part (a),
then part (b), as Section 4.1 splits attention around the Dispatch call) and
one MoE block (`MoEBlock` with a Combine return buffer).

FarSkip (Section 3 connectivity, Section 4.1 order), layer k on `compute`,
with p the partial residual (everything but the previous routed output):
    a   = p Wa^T                       attention part (a), on p_{k-1}
    COMBINE_{k-1}                      p += routed_{k-1}: p is now o_{k-1}
    GATE_k(o_{k-1})                    router, top-k, plan, pack; Dispatch on `comm`
    b   = a Wb^T                       attention part (b): overlaps Dispatch
    EXPERTS_k                          joins Dispatch; routed experts; Combine on `comm`
    SHARED_k(o_{k-1}) -> q             q = o_{k-1} + shared_k
    q  += b                            q = p_k (Eq. 7 without routed_k)
The Combine copy of layer k overlaps SHARED_k and layer k+1's part (a); the
last layer's COMBINE closes the stack.  Only the gate and the routed experts
stay outside both windows (Eq. 9).

Regular (Eq. 6): o' = o + Wb(Wa o); the block on o' with every copy
blocking on `compute`; o = o' + shared + routed.

Every arithmetic step runs in the library's kernels; this module only
orders the calls and owns the buffers.
"""

import torch

from . import _lib as L
from .block import MoEBlock


class LayerStack:
    def __init__(self, cfg, layers, device="cuda", merge_shared=None):
        """layers: list of (layer config, Workload, w_a, w_b) as made by
        workloads.generate.stack_layers; merge_shared lays out the shared
        experts as one SwiGLU (workloads.generate.merge_shared)."""
        self.cfg = cfg
        self.dtype_id = L.FS_F32 if cfg.dtype == "f32" else L.FS_BF16
        self.blocks, self.w_a, self.w_b = [], [], []
        for lc, wl, w_a, w_b in layers:
            sh_gu = sh_dn = None
            if lc.n_shared > 0:
                sh_gu, sh_dn = merge_shared(wl.sh_gate_up, wl.sh_down)
            blk = MoEBlock(lc, wl.w_router, wl.bias, wl.w_gate_up, wl.w_down, sh_gu, sh_dn,
                           device=device, with_comm=True, with_return=True)
            self.blocks.append(blk)
            self.w_a.append(w_a)
            self.w_b.append(w_b)
        N, d = cfg.n_tokens, cfg.hidden
        dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
        self.buf = [torch.empty((N, d), dtype=dt, device=device) for _ in range(2)]
        self.a = torch.empty((N, d), dtype=dt, device=device)
        self.b = torch.empty((N, d), dtype=dt, device=device)
        self.o1 = torch.empty((N, d), dtype=dt, device=device)

    def close(self):
        for blk in self.blocks:
            blk.close()

    def _linear(self, x, w, out, stream):
        N, d = self.cfg.n_tokens, self.cfg.hidden
        L.fs_dense_linear(self.dtype_id, N, d, d, x, w, out, stream=stream)

    def farskip(self, x, compute=None, comm=None):
        """FarSkip schedule on input x; returns the buffer holding o_{L-1}.
        With comm None the same order runs on one stream, copies blocking."""
        p, prev = x, None
        for k, blk in enumerate(self.blocks):
            q = self.buf[k % 2]
            self._linear(p, self.w_a[k], self.a, compute)
            if prev is not None:
                prev.phase(L.FS_PHASE_COMBINE, p, residual_io=p, compute=compute, comm=comm)
            blk.phase(L.FS_PHASE_GATE, p, compute=compute, comm=comm)
            self._linear(self.a, self.w_b[k], self.b, compute)
            blk.phase(L.FS_PHASE_EXPERTS, p, compute=compute, comm=comm)
            blk.phase(L.FS_PHASE_SHARED, p, partial_out=q, compute=compute, comm=comm)
            L.fs_farskip_residual(blk.desc, q, q, self.b, stream=compute)
            p, prev = q, blk
        prev.phase(L.FS_PHASE_COMBINE, p, residual_io=p, compute=compute, comm=comm)
        return p

    def regular(self, x, compute=None):
        """Regular schedule on input x (one stream, every copy blocking);
        returns the buffer holding o_{L-1}."""
        o = x
        for k, blk in enumerate(self.blocks):
            q = self.buf[k % 2]
            self._linear(o, self.w_a[k], self.a, compute)
            self._linear(self.a, self.w_b[k], self.b, compute)
            L.fs_farskip_residual(blk.desc, self.o1, o, self.b, stream=compute)
            blk.run(L.FS_PHASE_ALL, self.o1, q, q, compute=compute, comm=None)
            o = q
        return o
