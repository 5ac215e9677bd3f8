"""ctypes binding of libfarskip.so (include/farskip.h).

Argument marshalling only: torch tensors are passed as raw device pointers
(``data_ptr()``), streams as ``hipStream_t`` handles.  Every step of the
path runs in the library's HIP kernels.  There is no fallback: if the
library is missing, loading raises.
"""

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libfarskip.so")

FS_OK, FS_ERR_INVALID, FS_ERR_UNSUPPORTED, FS_ERR_WORKSPACE, FS_ERR_HIP = range(5)
FS_F32, FS_BF16 = 0, 1
FS_SOFTMAX, FS_SIGMOID = 0, 1
(FS_PHASE_ALL, FS_PHASE_BEGIN, FS_PHASE_FINISH, FS_PHASE_GATE, FS_PHASE_SHARED, FS_PHASE_EXPERTS,
 FS_PHASE_COMBINE) = range(7)
(FS_OP_ROUTER_TOPK, FS_OP_DISPATCH_PACK, FS_OP_GROUPED_FFN, FS_OP_BLOCK, FS_OP_GROUPED_FFN_FP8,
 FS_OP_BLOCK_FP8, FS_OP_DISPATCH_PACK_FP8) = range(7)
(FS_K_ROUTER, FS_K_TOPK, FS_K_PLAN, FS_K_PACK, FS_K_GATE_UP, FS_K_DOWN,
 FS_K_COMBINE, FS_K_SHARED_GATE_UP, FS_K_SHARED_DOWN, FS_K_DISPATCH_COPY, FS_K_DENSE,
 FS_K_COMBINE_COPY, FS_K_ALLREDUCE_COPY, FS_K_QUANTIZE, FS_K_COUNT) = range(15)
FS_ABI_VERSION = 9

_i32, _i64, _f32, _vp, _sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t


class FsError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{status_name(status)}: {message}")
        self.status = status


class fs_moe_desc(ctypes.Structure):
    _fields_ = [("abi_version", _i32), ("n_tokens", _i32), ("hidden", _i32),
                ("n_experts", _i32), ("top_k", _i32), ("n_groups", _i32),
                ("topk_groups", _i32), ("score", _i32), ("norm_topk", _i32),
                ("routed_scale", _f32), ("ffn", _i32), ("n_shared", _i32),
                ("ffn_shared", _i32), ("ep_size", _i32), ("ep_rank", _i32), ("dtype", _i32)]


class fs_moe_weights(ctypes.Structure):
    _fields_ = [("w_router", _vp), ("sel_bias", _vp), ("w_gate_up", _vp), ("w_down", _vp),
                ("ws_gate_up", _vp), ("ws_down", _vp),
                ("w_gate_up_fp8", _vp), ("s_gate_up", _vp), ("w_down_fp8", _vp), ("s_down", _vp),
                ("ws_gate_up_fp8", _vp), ("ss_gate_up", _vp), ("ws_down_fp8", _vp),
                ("ss_down", _vp), ("w_gate_up_fo", _vp), ("w_down_fo", _vp),
                ("w_gate_up_fp8_fo", _vp), ("w_down_fp8_fo", _vp)]


class fs_block_buffers(ctypes.Structure):
    _fields_ = [(n, _vp) for n in ("logits", "topk_ids", "topk_w", "src_counts", "src_offsets",
                                   "rank_offsets", "slot_to_row", "row_to_slot", "send", "recv",
                                   "group_rows", "group_offsets", "y", "shared_out", "ret")]


_SIGS = {
    "fs_status_string": (ctypes.c_char_p, [_i32]),
    "fs_last_error_message": (ctypes.c_char_p, []),
    "fs_abi_version": (_i32, []),
    "fs_workspace_size": (_i32, [ctypes.POINTER(fs_moe_desc), _i32, _i64, _i32, ctypes.POINTER(_sz)]),
    "fs_router_topk": (_i32, [ctypes.POINTER(fs_moe_desc), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "fs_dispatch_pack": (_i32, [ctypes.POINTER(fs_moe_desc), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "fs_dispatch_pack_fp8": (_i32, [ctypes.POINTER(fs_moe_desc), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                    _sz, _vp]),
    "fs_dispatch_pack_noalloc": (_i32, [ctypes.POINTER(fs_moe_desc), _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                        _vp, _vp]),
    "fs_receive_rows": (_i32, [ctypes.POINTER(fs_moe_desc), _vp, _vp, _vp, _vp, _vp]),
    "fs_local_rows": (_i32, [ctypes.POINTER(fs_moe_desc), _vp, _vp, _vp, _vp, _vp, _vp]),
    "fs_grouped_expert_ffn_gathered": (_i32, [ctypes.POINTER(fs_moe_desc), _i32, _i32, _vp, _vp, _vp,
                                              _i64, _vp, _vp, _vp, _vp, _sz, _vp]),
    "fs_grouped_expert_ffn": (_i32, [ctypes.POINTER(fs_moe_desc), _i32, _i32, _vp, _vp, _vp, _i64,
                                     _vp, _vp, _vp, _vp, _sz, _vp]),
    "fs_grouped_expert_ffn_fo": (_i32, [ctypes.POINTER(fs_moe_desc), _i32, _i32, _vp, _vp, _vp, _i64,
                                        _vp, _vp, _vp, _vp, _sz, _vp]),
    "fs_expert_weights_fragment_order": (_i32, [_i32, _i64, _i32, _i32, _vp, _vp, _vp]),
    "fs_combine_unpack": (_i32, [ctypes.POINTER(fs_moe_desc), _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "fs_quantize_fp8": (_i32, [_i32, _i64, _i32, _vp, _vp, _vp, _vp]),
    "fs_grouped_expert_ffn_fp8": (_i32, [ctypes.POINTER(fs_moe_desc), _i32, _i32, _vp, _vp, _vp, _vp,
                                         _i64, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "fs_grouped_expert_ffn_fp8_fo": (_i32, [ctypes.POINTER(fs_moe_desc), _i32, _i32, _vp, _vp, _vp,
                                            _vp, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "fs_expert_weights_fragment_order_fp8": (_i32, [_i64, _i32, _i32, _vp, _vp, _vp]),
    "fs_combine_partial": (_i32, [ctypes.POINTER(fs_moe_desc), _vp, _vp, _vp, _vp, _vp, _vp]),
    "fs_allreduce_standin": (_i32, [ctypes.POINTER(fs_moe_desc), _vp, _vp, _vp]),
    "fs_standin_link": (_i32, [_i32, ctypes.c_double, _i32]),
    "fs_standin_link_get": (_i32, [ctypes.POINTER(_i32), ctypes.POINTER(ctypes.c_double),
                                   ctypes.POINTER(_i32)]),
    "fs_farskip_residual": (_i32, [ctypes.POINTER(fs_moe_desc), _vp, _vp, _vp, _vp, _vp]),
    "fs_block_sync_create": (_i32, [ctypes.POINTER(_vp)]),
    "fs_block_sync_destroy": (_i32, [_vp]),
    "fs_moe_block_forward": (_i32, [ctypes.POINTER(fs_moe_desc), _i32, ctypes.POINTER(fs_moe_weights),
                                    _vp, _vp, _vp, ctypes.POINTER(fs_block_buffers), _i64, _vp, _sz,
                                    _vp, _vp, _vp]),
    "fs_dense_linear": (_i32, [_i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp]),
    "fs_profile_enable": (_i32, [_i32]),
    "fs_profile_select": (_i32, [ctypes.c_uint32]),
    "fs_profile_read": (_i32, [_i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_i64)]),
    "fs_profile_reset": (_i32, []),
}
EXPORTS = tuple(_SIGS)

_lib = None


def load(path=LIB_PATH):
    """Load libfarskip.so once.  Raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise FsError(FS_ERR_INVALID, f"{path} is not built; run python -m paper_2511_11505_amd.build")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def status_name(status):
    try:
        return load().fs_status_string(status).decode()
    except Exception:  # the library itself failed to load
        return f"status {status}"


def _check(status):
    if status != FS_OK:
        raise FsError(status, load().fs_last_error_message().decode())


def ptr(t):
    """Device pointer of a tensor (or an int address); None -> NULL."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def stream_handle(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _ws(ws):
    if ws is None:
        return None, 0
    if isinstance(ws, tuple):
        return ws
    return ws.data_ptr(), ws.numel() * ws.element_size()


def make_desc(cfg):
    """fs_moe_desc of a workload configuration."""
    return fs_moe_desc(
        FS_ABI_VERSION, cfg.n_tokens, cfg.hidden, cfg.n_experts, cfg.top_k, cfg.n_groups,
        cfg.topk_groups if cfg.n_groups > 1 else 1,
        FS_SOFTMAX if cfg.score == "softmax" else FS_SIGMOID, int(cfg.norm_topk),
        float(cfg.routed_scale), cfg.ffn, cfg.n_shared, cfg.ffn_shared if cfg.n_shared else 0,
        cfg.ep_size, cfg.ep_rank, FS_F32 if cfg.dtype == "f32" else FS_BF16)


# ---------------------------------------------------------------- entry points
def fs_abi_version():
    return load().fs_abi_version()


def fs_workspace_size(desc, op, max_rows=0, ffn=0):
    out = _sz(0)
    _check(load().fs_workspace_size(ctypes.byref(desc), op, max_rows, ffn, ctypes.byref(out)))
    return out.value


def fs_router_topk(desc, x, w_router, sel_bias, logits_in, logits_out, topk_ids, topk_w, ws,
                   stream=None):
    wp, wb = _ws(ws)
    _check(load().fs_router_topk(ctypes.byref(desc), ptr(x), ptr(w_router), ptr(sel_bias),
                                 ptr(logits_in), ptr(logits_out), ptr(topk_ids), ptr(topk_w),
                                 wp, wb, stream_handle(stream)))


def fs_dispatch_pack(desc, topk_ids, x, expert_counts, expert_offsets, rank_offsets, slot_to_row,
                     row_to_slot, send, ws, stream=None):
    wp, wb = _ws(ws)
    _check(load().fs_dispatch_pack(ctypes.byref(desc), ptr(topk_ids), ptr(x), ptr(expert_counts),
                                   ptr(expert_offsets), ptr(rank_offsets), ptr(slot_to_row),
                                   ptr(row_to_slot), ptr(send), wp, wb, stream_handle(stream)))


def fs_dispatch_pack_noalloc(desc, topk_ids, x, expert_counts, expert_offsets, rank_offsets,
                             slot_to_row, row_to_slot, send, stream=None):
    _check(load().fs_dispatch_pack_noalloc(ctypes.byref(desc), ptr(topk_ids), ptr(x),
                                           ptr(expert_counts), ptr(expert_offsets),
                                           ptr(rank_offsets), ptr(slot_to_row), ptr(row_to_slot),
                                           ptr(send), stream_handle(stream)))


def fs_dispatch_pack_fp8(desc, topk_ids, x, expert_counts, expert_offsets, rank_offsets, slot_to_row,
                         row_to_slot, send_codes, send_scales, ws, stream=None):
    wp, wb = _ws(ws)
    _check(load().fs_dispatch_pack_fp8(ctypes.byref(desc), ptr(topk_ids), ptr(x), ptr(expert_counts),
                                       ptr(expert_offsets), ptr(rank_offsets), ptr(slot_to_row),
                                       ptr(row_to_slot), ptr(send_codes), ptr(send_scales), wp, wb,
                                       stream_handle(stream)))


def fs_receive_rows(desc, src_counts, src_offsets, group_rows, group_offsets, stream=None):
    _check(load().fs_receive_rows(ctypes.byref(desc), ptr(src_counts), ptr(src_offsets),
                                  ptr(group_rows), ptr(group_offsets), stream_handle(stream)))


def fs_local_rows(desc, expert_offsets, rank_offsets, row_to_slot, local_tokens, local_offsets,
                  stream=None):
    _check(load().fs_local_rows(ctypes.byref(desc), ptr(expert_offsets), ptr(rank_offsets),
                                ptr(row_to_slot), ptr(local_tokens), ptr(local_offsets),
                                stream_handle(stream)))


def fs_grouped_expert_ffn_gathered(desc, n_groups, ffn, x, gather_rows, group_offsets, max_rows,
                                   w_gate_up, w_down, y, ws, stream=None):
    wp, wb = _ws(ws)
    _check(load().fs_grouped_expert_ffn_gathered(ctypes.byref(desc), n_groups, ffn, ptr(x),
                                                 ptr(gather_rows), ptr(group_offsets), max_rows,
                                                 ptr(w_gate_up), ptr(w_down), ptr(y), wp, wb,
                                                 stream_handle(stream)))


def fs_grouped_expert_ffn_fo(desc, n_groups, ffn, in_rows, group_rows, group_offsets, max_rows,
                             w_gate_up_fo, w_down_fo, out_rows, ws, stream=None):
    wp, wb = _ws(ws)
    _check(load().fs_grouped_expert_ffn_fo(ctypes.byref(desc), n_groups, ffn, ptr(in_rows),
                                           ptr(group_rows), ptr(group_offsets), max_rows,
                                           ptr(w_gate_up_fo), ptr(w_down_fo), ptr(out_rows), wp,
                                           wb, stream_handle(stream)))


def fs_expert_weights_fragment_order(dtype, n_mats, rows, cols, src, dst, stream=None):
    _check(load().fs_expert_weights_fragment_order(dtype, n_mats, rows, cols, ptr(src), ptr(dst),
                                                   stream_handle(stream)))


def fs_grouped_expert_ffn(desc, n_groups, ffn, in_rows, group_rows, group_offsets, max_rows,
                          w_gate_up, w_down, out_rows, ws, stream=None):
    wp, wb = _ws(ws)
    _check(load().fs_grouped_expert_ffn(ctypes.byref(desc), n_groups, ffn, ptr(in_rows),
                                        ptr(group_rows), ptr(group_offsets), max_rows,
                                        ptr(w_gate_up), ptr(w_down), ptr(out_rows), wp, wb,
                                        stream_handle(stream)))


def fs_combine_unpack(desc, y_ret, slot_to_row, topk_w, shared_out, routed_out, residual,
                      stream=None):
    _check(load().fs_combine_unpack(ctypes.byref(desc), ptr(y_ret), ptr(slot_to_row), ptr(topk_w),
                                    ptr(shared_out), ptr(routed_out), ptr(residual),
                                    stream_handle(stream)))


def fs_quantize_fp8(dtype, rows, cols, src, codes, scales, stream=None):
    _check(load().fs_quantize_fp8(dtype, rows, cols, ptr(src), ptr(codes), ptr(scales),
                                  stream_handle(stream)))


def fs_grouped_expert_ffn_fp8(desc, n_groups, ffn, x_codes, x_scales, group_rows, group_offsets,
                              max_rows, w_gate_up, s_gate_up, w_down, s_down, out_rows, ws,
                              stream=None):
    wp, wb = _ws(ws)
    _check(load().fs_grouped_expert_ffn_fp8(ctypes.byref(desc), n_groups, ffn, ptr(x_codes),
                                            ptr(x_scales), ptr(group_rows), ptr(group_offsets),
                                            max_rows, ptr(w_gate_up), ptr(s_gate_up), ptr(w_down),
                                            ptr(s_down), ptr(out_rows), wp, wb,
                                            stream_handle(stream)))


def fs_grouped_expert_ffn_fp8_fo(desc, n_groups, ffn, x_codes, x_scales, group_rows, group_offsets,
                                 max_rows, w_gate_up_fo, s_gate_up, w_down_fo, s_down, out_rows, ws,
                                 stream=None):
    wp, wb = _ws(ws)
    _check(load().fs_grouped_expert_ffn_fp8_fo(ctypes.byref(desc), n_groups, ffn, ptr(x_codes),
                                               ptr(x_scales), ptr(group_rows), ptr(group_offsets),
                                               max_rows, ptr(w_gate_up_fo), ptr(s_gate_up),
                                               ptr(w_down_fo), ptr(s_down), ptr(out_rows), wp, wb,
                                               stream_handle(stream)))


def fs_expert_weights_fragment_order_fp8(n_mats, rows, cols, src, dst, stream=None):
    _check(load().fs_expert_weights_fragment_order_fp8(n_mats, rows, cols, ptr(src), ptr(dst),
                                                       stream_handle(stream)))


def fs_combine_partial(desc, y_local, slot_to_row, rank_offsets, topk_w, partial_out, stream=None):
    _check(load().fs_combine_partial(ctypes.byref(desc), ptr(y_local), ptr(slot_to_row),
                                     ptr(rank_offsets), ptr(topk_w), ptr(partial_out),
                                     stream_handle(stream)))


def fs_allreduce_standin(desc, out, partial, stream=None):
    _check(load().fs_allreduce_standin(ctypes.byref(desc), ptr(out), ptr(partial),
                                       stream_handle(stream)))


def fs_standin_link(links, link_bytes_per_s=0.0, workgroups=0):
    _check(load().fs_standin_link(int(links), float(link_bytes_per_s), int(workgroups)))


def fs_standin_link_get():
    n, b, w = _i32(), ctypes.c_double(), _i32()
    _check(load().fs_standin_link_get(ctypes.byref(n), ctypes.byref(b), ctypes.byref(w)))
    return n.value, b.value, w.value


class standin_link:
    """Context manager: the stand-in copies inside follow a node of
    links + 1 GPUs joined by links of link_bytes_per_s per direction
    (fs_standin_link); the previous setting comes back on exit."""

    def __init__(self, links=7, link_bytes_per_s=153e9, workgroups=128):
        self.args = (links, link_bytes_per_s, workgroups)

    def __enter__(self):
        self.prev = fs_standin_link_get()
        fs_standin_link(*self.args)
        return self

    def __exit__(self, *exc):
        fs_standin_link(*self.prev)


def fs_farskip_residual(desc, out, residual, deferred, extra=None, stream=None):
    _check(load().fs_farskip_residual(ctypes.byref(desc), ptr(out), ptr(residual), ptr(deferred),
                                      ptr(extra), stream_handle(stream)))


def fs_dense_linear(dtype, m, n, kdim, a, w, out, stream=None):
    _check(load().fs_dense_linear(dtype, m, n, kdim, ptr(a), ptr(w), ptr(out), stream_handle(stream)))


def fs_block_sync_create():
    h = _vp()
    _check(load().fs_block_sync_create(ctypes.byref(h)))
    return h.value


def fs_block_sync_destroy(h):
    _check(load().fs_block_sync_destroy(h))


def fs_moe_block_forward(desc, phase, weights, residual_in, partial_out, residual_io, buffers,
                         max_recv_rows, ws, sync=None, compute=None, comm=None):
    wp, wb = _ws(ws)
    _check(load().fs_moe_block_forward(ctypes.byref(desc), phase, ctypes.byref(weights),
                                       ptr(residual_in), ptr(partial_out), ptr(residual_io),
                                       ctypes.byref(buffers), max_recv_rows, wp, wb, sync,
                                       stream_handle(compute),
                                       None if comm is None else stream_handle(comm)))


def fs_profile_enable(on=True):
    _check(load().fs_profile_enable(int(on)))


def fs_profile_select(kernels=None):
    """Time only the given fs_kernel_id values (None: all)."""
    mask = (1 << FS_K_COUNT) - 1 if kernels is None else sum(1 << int(k) for k in set(kernels))
    _check(load().fs_profile_select(mask))


def fs_profile_read(kernel):
    ms, n = ctypes.c_double(0), _i64(0)
    _check(load().fs_profile_read(kernel, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def fs_profile_reset():
    _check(load().fs_profile_reset())
