"""GPU: the cache policies of the full-attention and score-pass loads change
no result.

The policies only set the non-temporal hint on loads (which rows the caches
keep), so every policy built for a row-tile count, forced through
HS2_FA_CACHE_POLICY / HS2_FA_K_KEEP, must give results bit-identical to the
default policy's on the same inputs: full-attention out, (M, Z), pooled
scores, index rows and the sparse layers.  One streaming policy per row-tile
count is also checked against the oracle.
"""
from __future__ import annotations

import numpy as np
import pytest

from tests.test_gpu_parity import SMALL, note, parity_case, run_gpu
from paper_2609_26368_amd import workloads as W

pytestmark = pytest.mark.gpu

RT1 = SMALL[0]  # 16q/2kv, one query: 8 rows per KV head (stored-logits score pass)
RT4 = SMALL[3]  # 32q/4kv, 8-query chunk: 64 rows per KV head (score pass over K)
# 16q/2kv, 4-query chunk: 32 rows per KV head, two row tiles (ring kernel with
# two token groups of 16-token tiles, score pass over K)
RT2 = W.Workload("rt2_c4_16q2kv", 2, 4000, 4, 16, 2, 128, 512, 64, 1, ctx_min=3000)

# (workload, extra environment, policies with their K-keep shares).  At these
# sizes a split is 256 tokens: each of a ring kernel's two token groups
# streams 128 of them (RT4: four 32-token tiles, RT2: eight 16-token tiles),
# so keep 75 and 40 switch from non-temporal to cacheable K rows inside a
# group, 0 streams all of a group's K rows and 100 none.
CASES = [
    ("rt1", RT1, {}, [("1", None), ("2", None)]),
    ("rt1-pool-from-K", RT1, {"HS2_POOL_FROM_K": "1"}, [("1", None), ("2", None)]),
    ("rt2", RT2, {}, [("3", "0"), ("3", "40"), ("3", "75"), ("3", "100")]),
    ("rt4", RT4, {}, [("3", "0"), ("3", "40"), ("3", "75"), ("3", "100")]),
]


def _same(a, b, what):
    if isinstance(a, list):
        for i, (x, y) in enumerate(zip(a, b)):
            _same(x, y, f"{what}[{i}]")
        return
    assert np.array_equal(a, b, equal_nan=True), f"{what} differs under a cache policy"


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
@pytest.mark.parametrize("name,w,env,policies", CASES, ids=[c[0] for c in CASES])
def test_cache_policies_bit_identical(name, w, env, policies, kv, monkeypatch):
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    inp = W.make_inputs(w, seed=77, kv=kv)
    monkeypatch.delenv("HS2_FA_CACHE_POLICY", raising=False)
    monkeypatch.delenv("HS2_FA_K_KEEP", raising=False)
    base = run_gpu(inp)
    for pol, keep in policies:
        note(f"[cache policy] {name} kv={kv} policy={pol} keep={keep}")
        monkeypatch.setenv("HS2_FA_CACHE_POLICY", pol)
        if keep is None:
            monkeypatch.delenv("HS2_FA_K_KEEP", raising=False)
        else:
            monkeypatch.setenv("HS2_FA_K_KEEP", keep)
        got = run_gpu(inp)
        for key in base:
            _same(got[key], base[key], f"{name} policy {pol} keep {keep}: {key}")


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
@pytest.mark.parametrize("w,pol", [(RT1, "2"), (RT2, "3"), (RT4, "3")], ids=["rt1-policy2", "rt2-policy3", "rt4-policy3"])
def test_streaming_policy_parity(w, pol, kv, monkeypatch):
    monkeypatch.setenv("HS2_FA_CACHE_POLICY", pol)
    parity_case(w, seed=78, kv=kv)
