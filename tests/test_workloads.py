"""The seeded input generators: determinism, shapes, bf16 rounding."""

import numpy as np
import torch

from workloads import CONFIGS, make_workload, bf16_round
from workloads.generate import expert_weights, merge_shared, synthetic_topk_ids


def test_bf16_round_nearest_even():
    a = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -9], np.float32)
    got = bf16_round(a)
    want = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, want)
    # ties to even: 1 + 2^-8 is halfway between 1 and 1 + 2^-7
    assert got[1] == 0x3F80 and got[2] == 0x3F82


def test_tiny_workload_deterministic():
    cfg = CONFIGS["tiny"]
    a = make_workload(cfg, "cpu")
    b = make_workload(cfg, "cpu")
    assert torch.equal(a.x, b.x) and torch.equal(a.w_gate_up, b.w_gate_up)
    assert a.x.shape == (128, 256) and a.w_gate_up.shape == (8, 1024, 256)
    assert a.w_down.shape == (8, 256, 512) and a.w_next.shape == (256, 256)
    assert abs(a.x.float().std().item() - 1.0) < 0.05
    assert abs(a.w_router.float().std().item() - 0.02) < 0.002
    gu, dn = expert_weights(cfg, "cpu", 3)
    assert torch.equal(gu, a.w_gate_up[3]) and torch.equal(dn, a.w_down[3])


def test_merge_shared_layout():
    S, F, d = 2, 3, 4
    gu = torch.arange(S * 2 * F * d, dtype=torch.float32).reshape(S, 2 * F, d)
    dn = torch.arange(S * d * F, dtype=torch.float32).reshape(S, d, F)
    mgu, mdn = merge_shared(gu, dn)
    assert torch.equal(mgu[:F], gu[0, :F]) and torch.equal(mgu[F:2 * F], gu[1, :F])
    assert torch.equal(mgu[2 * F:3 * F], gu[0, F:]) and torch.equal(mgu[3 * F:], gu[1, F:])
    assert torch.equal(mdn[:, :F], dn[0]) and torch.equal(mdn[:, F:], dn[1])


def test_synthetic_ids_distinct():
    ids = synthetic_topk_ids(300, 16, 5, seed=3, skew=1.0)
    assert ids.shape == (300, 5) and ids.dtype == torch.int32
    for row in ids.tolist():
        assert len(set(row)) == 5 and all(0 <= e < 16 for e in row)
