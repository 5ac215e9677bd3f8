"""FarSkip MoE block forward on AMD Instinct MI355X (gfx950).

The hot path is libfarskip.so (C ABI in include/farskip.h): router and top-k,
dispatch plan and pack, grouped SwiGLU experts on MFMA, Combine with the
deferred FarSkip residual add, and the two-phase block driver; for the
replicated-activation inference variant, the local rows, the gathered
expert GEMMs, the partial Combine and the all-reduce stand-in.  This package
is its ctypes binding plus small owners of device buffers that order the
calls: one block (block.py), stacked layers in the two-window schedule
(stack.py) and stacked replicated-activation layers (replicated.py).
"""

from . import _lib  # noqa: F401
from ._lib import (  # noqa: F401
    FsError, make_desc, load, fs_abi_version, fs_workspace_size, fs_router_topk,
    fs_dispatch_pack, fs_dispatch_pack_fp8, fs_receive_rows, fs_grouped_expert_ffn, fs_combine_unpack,
    fs_local_rows, fs_grouped_expert_ffn_gathered, fs_combine_partial, fs_allreduce_standin,
    fs_quantize_fp8, fs_grouped_expert_ffn_fp8, fs_expert_weights_fragment_order,
    fs_grouped_expert_ffn_fo, fs_grouped_expert_ffn_fp8_fo, fs_expert_weights_fragment_order_fp8,
    fs_standin_link, fs_standin_link_get, standin_link,
    fs_farskip_residual, fs_dense_linear, fs_block_sync_create, fs_block_sync_destroy,
    fs_moe_block_forward, fs_profile_enable, fs_profile_select, fs_profile_read, fs_profile_reset,
)
from .block import (MoEBlock, fp8_row_views, fragment_ordered, fragment_ordered_fp8,  # noqa: F401
                    prepare_remote_sources)
