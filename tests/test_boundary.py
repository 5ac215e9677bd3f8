"""The C ABI boundary on the host: the library loads, exports every function
include/farskip.h declares, and rejects bad arguments before any HIP call
(these tests make no compute call and need no GPU)."""

import ctypes
import os
import re

import pytest

from paper_2511_11505_amd import _lib as L
from workloads import CONFIGS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "farskip.h")


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fs_[a-z_0-9]+)\s*\(", src)))


def test_library_loads_and_exports_every_declared_symbol():
    lib = L.load()
    declared = header_functions()
    assert len(declared) >= 17
    for name in declared:
        assert hasattr(lib, name), name
    assert set(declared) == set(L.EXPORTS)
    assert L.fs_abi_version() == L.FS_ABI_VERSION


def test_binding_constants_match_the_header():
    """Every enumerator the header defines has the same value in the binding."""
    src = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    enums = re.findall(r"\b(FS_[A-Z0-9_]+)\s*=\s*(\d+)\s*[,}\n]", src)
    assert len(enums) >= 20
    for name, value in enums:
        assert getattr(L, name) == int(value), name
    assert L.fs_profile_read(L.FS_K_COUNT - 1) == (0.0, 0)
    with pytest.raises(L.FsError):
        L.fs_profile_read(L.FS_K_COUNT)
    with pytest.raises(L.FsError):
        L.fs_profile_select([L.FS_K_COUNT])
    L.fs_profile_select([L.FS_K_GATE_UP, L.FS_K_DOWN])
    L.fs_profile_select(None)


def test_status_strings():
    lib = L.load()
    assert lib.fs_status_string(0) == b"FS_OK"
    assert lib.fs_status_string(3) == b"FS_ERR_WORKSPACE"


def desc(name="dsv3_prefill", **kw):
    d = L.make_desc(CONFIGS[name])
    for k, v in kw.items():
        setattr(d, k, v)
    return d


FAKE = 1 << 20  # a 16-byte aligned non-null address; never dereferenced


def expect(status, fn, *args, **kw):
    with pytest.raises(L.FsError) as e:
        fn(*args, **kw)
    assert e.value.status == status, str(e.value)
    return str(e.value)


@pytest.mark.parametrize("field,value,status", [
    ("abi_version", L.FS_ABI_VERSION + 1, L.FS_ERR_INVALID),
    ("n_tokens", -1, L.FS_ERR_INVALID),
    ("hidden", 0, L.FS_ERR_INVALID),
    ("hidden", 7168 + 64, L.FS_ERR_UNSUPPORTED),
    ("top_k", 0, L.FS_ERR_INVALID),
    ("top_k", 300, L.FS_ERR_INVALID),
    ("n_experts", 1024, L.FS_ERR_UNSUPPORTED),
    ("n_groups", 7, L.FS_ERR_INVALID),
    ("topk_groups", 9, L.FS_ERR_INVALID),
    ("score", 5, L.FS_ERR_INVALID),
    ("ffn", 100, L.FS_ERR_UNSUPPORTED),
    ("ep_size", 3, L.FS_ERR_INVALID),
    ("ep_rank", 8, L.FS_ERR_INVALID),
    ("dtype", 9, L.FS_ERR_INVALID),
])
def test_descriptor_checks(field, value, status):
    d = desc(**{field: value})
    expect(status, L.fs_workspace_size, d, L.FS_OP_ROUTER_TOPK)


def test_topk_groups_limit():
    d = desc(topk_groups=1, top_k=32)      # 32 experts per group: ok
    assert L.fs_workspace_size(d, L.FS_OP_BLOCK, 1000) > 0
    d = desc(topk_groups=1, n_groups=64, top_k=5)   # 4 experts per kept group < 5
    expect(L.FS_ERR_INVALID, L.fs_workspace_size, d, L.FS_OP_ROUTER_TOPK)


def test_token_count_limit():
    d = desc(n_tokens=(1 << 31) // 64)
    expect(L.FS_ERR_UNSUPPORTED, L.fs_workspace_size, d, L.FS_OP_ROUTER_TOPK)


def test_workspace_sizes_grow_with_rows():
    d = desc()
    a = L.fs_workspace_size(d, L.FS_OP_GROUPED_FFN, 1000, 2048)
    b = L.fs_workspace_size(d, L.FS_OP_GROUPED_FFN, 2000, 2048)
    assert b > a >= 1000 * 2048 * 2
    blk = L.fs_workspace_size(d, L.FS_OP_BLOCK, 32768)
    assert blk >= L.fs_workspace_size(d, L.FS_OP_GROUPED_FFN, 32768, 2048)
    expect(L.FS_ERR_INVALID, L.fs_workspace_size, d, 17)
    expect(L.FS_ERR_INVALID, L.fs_workspace_size, d, L.FS_OP_GROUPED_FFN, -1, 64)


def test_router_argument_checks():
    d = desc()
    msg = expect(L.FS_ERR_INVALID, L.fs_router_topk, d, None, FAKE, None, None, None, FAKE, FAKE,
                 (FAKE, 1 << 30), stream=0)
    assert "x" in msg
    expect(L.FS_ERR_INVALID, L.fs_router_topk, d, FAKE + 4, FAKE, None, None, None, FAKE, FAKE,
           (FAKE, 1 << 30), stream=0)
    expect(L.FS_ERR_WORKSPACE, L.fs_router_topk, d, FAKE, FAKE, None, None, None, FAKE, FAKE,
           (FAKE, 16), stream=0)
    ds = desc("dsv2lite")
    expect(L.FS_ERR_UNSUPPORTED, L.fs_router_topk, ds, FAKE, FAKE, FAKE, None, None, FAKE, FAKE,
           (FAKE, 1 << 30), stream=0)


def test_other_entry_point_checks():
    d = desc()
    expect(L.FS_ERR_INVALID, L.fs_dispatch_pack, d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE,
           (FAKE, 1 << 30), stream=0)
    expect(L.FS_ERR_WORKSPACE, L.fs_dispatch_pack, d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
           (FAKE, 8), stream=0)
    # the allocation-free dispatch: pointer checks, and shapes beyond its
    # fixed scratch rejected before any HIP call
    expect(L.FS_ERR_INVALID, L.fs_dispatch_pack_noalloc, d, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None,
           FAKE, stream=0)
    big = desc("dsv2lite", n_experts=512, n_tokens=(262144 // 512) * 64 + 1)
    msg = expect(L.FS_ERR_UNSUPPORTED, L.fs_dispatch_pack_noalloc, big, FAKE, FAKE, FAKE, FAKE, FAKE,
                 FAKE, FAKE, FAKE, stream=0)
    assert "scratch" in msg
    expect(L.FS_ERR_INVALID, L.fs_grouped_expert_ffn, d, 32, 2048, FAKE, None, None, 100, FAKE, FAKE,
           FAKE, (FAKE, 1 << 40), stream=0)
    # fragment order: bf16 only, whole 32-row x 16-column blocks, no overlap
    expect(L.FS_ERR_UNSUPPORTED, L.fs_expert_weights_fragment_order, L.FS_F32, 2, 64, 64, FAKE,
           FAKE + (1 << 20), stream=0)
    expect(L.FS_ERR_UNSUPPORTED, L.fs_expert_weights_fragment_order, L.FS_BF16, 2, 48, 64, FAKE,
           FAKE + (1 << 20), stream=0)
    expect(L.FS_ERR_INVALID, L.fs_expert_weights_fragment_order, L.FS_BF16, 2, 64, 64, FAKE,
           FAKE + 4096, stream=0)
    expect(L.FS_ERR_UNSUPPORTED, L.fs_grouped_expert_ffn_fo, desc("tiny"), 8, 512, FAKE, None,
           FAKE, 100, FAKE, FAKE, FAKE, (FAKE, 1 << 40), stream=0)
    expect(L.FS_ERR_WORKSPACE, L.fs_grouped_expert_ffn_fo, d, 32, 2048, FAKE, None, FAKE, 100,
           FAKE, FAKE, FAKE, (FAKE, 64), stream=0)
    # FP8 fragment order: whole 32-row x 64-byte fragments, no overlap; its
    # FFN: the FP8 FFN's shapes and workspace
    expect(L.FS_ERR_UNSUPPORTED, L.fs_expert_weights_fragment_order_fp8, 2, 64, 96, FAKE,
           FAKE + (1 << 20), stream=0)
    expect(L.FS_ERR_UNSUPPORTED, L.fs_expert_weights_fragment_order_fp8, 2, 48, 128, FAKE,
           FAKE + (1 << 20), stream=0)
    expect(L.FS_ERR_INVALID, L.fs_expert_weights_fragment_order_fp8, 2, 64, 128, FAKE,
           FAKE + 4096, stream=0)
    expect(L.FS_ERR_INVALID, L.fs_expert_weights_fragment_order_fp8, -1, 64, 128, FAKE,
           FAKE + (1 << 20), stream=0)
    expect(L.FS_ERR_UNSUPPORTED, L.fs_grouped_expert_ffn_fp8_fo, d, 32, 100, FAKE, FAKE, None, FAKE,
           100, FAKE, FAKE, FAKE, FAKE, FAKE, (FAKE, 1 << 40), stream=0)
    expect(L.FS_ERR_WORKSPACE, L.fs_grouped_expert_ffn_fp8_fo, d, 32, 2048, FAKE, FAKE, None, FAKE,
           100, FAKE, FAKE, FAKE, FAKE, FAKE, (FAKE, 64), stream=0)
    expect(L.FS_ERR_UNSUPPORTED, L.fs_grouped_expert_ffn, d, 32, 100, FAKE, None, FAKE, 100, FAKE,
           FAKE, FAKE, (FAKE, 1 << 40), stream=0)
    expect(L.FS_ERR_WORKSPACE, L.fs_grouped_expert_ffn, d, 32, 2048, FAKE, None, FAKE, 100, FAKE,
           FAKE, FAKE, (FAKE, 64), stream=0)
    expect(L.FS_ERR_INVALID, L.fs_combine_unpack, d, FAKE, FAKE, FAKE, None, None, None, stream=0)
    expect(L.FS_ERR_INVALID, L.fs_farskip_residual, d, FAKE, None, FAKE, stream=0)
    expect(L.FS_ERR_UNSUPPORTED, L.fs_dense_linear, L.FS_BF16, 4, 100, 64, FAKE, FAKE, FAKE, stream=0)
    expect(L.FS_ERR_INVALID, L.fs_dense_linear, 5, 4, 128, 64, FAKE, FAKE, FAKE, stream=0)


def test_block_checks():
    cfg = CONFIGS["dsv3_prefill"]
    d = L.make_desc(cfg)
    w = L.fs_moe_weights(FAKE, None, FAKE, FAKE, FAKE, FAKE)
    b = L.fs_block_buffers(*([FAKE] * 14))
    expect(L.FS_ERR_INVALID, L.fs_moe_block_forward, d, 9, w, FAKE, FAKE, FAKE, b, 1000,
           (FAKE, 1 << 40), compute=0)
    expect(L.FS_ERR_WORKSPACE, L.fs_moe_block_forward, d, L.FS_PHASE_ALL, w, FAKE, FAKE, FAKE, b,
           1000, (FAKE, 64), compute=0)
    expect(L.FS_ERR_INVALID, L.fs_moe_block_forward, d, L.FS_PHASE_ALL, w, FAKE, FAKE, FAKE, b,
           cfg.ep_size * cfg.cap + 1, (FAKE, 1 << 40), compute=0)
    b.send = None
    expect(L.FS_ERR_INVALID, L.fs_moe_block_forward, d, L.FS_PHASE_BEGIN, w, FAKE, FAKE, FAKE, b,
           1000, (FAKE, 1 << 40), compute=0)
    # a comm stream needs a sync object
    b.send = FAKE
    expect(L.FS_ERR_INVALID, L.fs_moe_block_forward, d, L.FS_PHASE_ALL, w, FAKE, FAKE, FAKE, b,
           1000, (FAKE, 1 << 40), compute=0, comm=FAKE)
    # single-rank blocks need room for every routed row
    d1 = L.make_desc(CONFIGS["dsv2lite"])
    expect(L.FS_ERR_INVALID, L.fs_moe_block_forward, d1, L.FS_PHASE_ALL, w, FAKE, FAKE, FAKE, b,
           10, (FAKE, 1 << 40), compute=0)


def test_empty_batch_is_a_noop():
    d = desc(n_tokens=0)
    L.fs_router_topk(d, None, None, None, None, None, None, None, None, stream=0)
    L.fs_combine_unpack(d, None, None, None, None, None, None, stream=0)


def test_standin_link_setting():
    # process-wide link model of the stand-in copies: set, read back,
    # rejected arguments leave it unchanged, links 0 restores HBM copies
    assert L.fs_standin_link_get() == (0, 0.0, 0)
    L.fs_standin_link(7, 153e9, 64)
    assert L.fs_standin_link_get() == (7, 153e9, 64)
    for args in [(-1, 153e9, 64), (1024, 153e9, 64), (7, 5e8, 64), (7, 2e15, 64), (7, float("nan"), 64),
                 (7, 153e9, 0), (7, 153e9, 4097)]:
        with pytest.raises(L.FsError) as e:
            L.fs_standin_link(*args)
        assert e.value.status == L.FS_ERR_INVALID
        assert L.fs_standin_link_get() == (7, 153e9, 64)
    with L.standin_link(3, 50e9, 8):
        assert L.fs_standin_link_get() == (3, 50e9, 8)
    assert L.fs_standin_link_get() == (7, 153e9, 64)
    L.fs_standin_link(0, -1.0, -5)          # links 0 ignores the rest
    assert L.fs_standin_link_get() == (0, 0.0, 0)
