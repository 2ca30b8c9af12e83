"""GPU parity of every full-attention kernel shape, not only the planner's
defaults: each (row tiles, variant) pair of the head-dim-128 table, forced
through HS2_FA_VARIANT, for the bf16 cache and (ring kernels) the E4M3 cache.
"""
from __future__ import annotations

import pytest

from paper_2609_26368_amd import workloads as W
from tests.test_gpu_parity import SMALL, parity_case

pytestmark = pytest.mark.gpu

BY_RT = {  # a reduced workload per number of 16-row query tiles per KV head
    1: SMALL[0],                                                                  # 16q/2kv, C = 1: 8 rows
    2: W.Workload("rt2_16q1kv_C2", 2, 3000, 2, 16, 1, 128, 200, 48, 1, ctx_min=1500),  # 32 rows
    4: SMALL[3],                                                                  # 32q/4kv, C = 8: 64 rows
    8: W.Workload("rt8_32q1kv_C4", 2, 2500, 4, 32, 1, 128, 200, 48, 1, ctx_min=1200),  # 128 rows
}
# (row tiles, variant) pairs of the head-dim-128 table: ring kernels 0, 2, 3,
# 5 (RT 1, 2, 4) and 7 (RT 2, 4, 8); the workgroup kernel 1 (bf16 only)
SHAPES = [(rt, v) for rt in (1, 2, 4) for v in (0, 1, 2, 3, 5, 7) if not (v == 7 and rt == 1)] + [(8, 1), (8, 7)]


@pytest.mark.parametrize("rt,variant", SHAPES, ids=[f"rt{rt}-v{v}" for rt, v in SHAPES])
@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_every_fa_kernel_shape(rt, variant, kv, monkeypatch):
    if kv == "fp8" and variant == 1:
        pytest.skip("the workgroup kernel reads bf16 caches only")
    monkeypatch.setenv("HS2_FA_VARIANT", str(variant))
    parity_case(BY_RT[rt], seed=41, kv=kv)
