"""GPU parity on seeded random shapes: batch, query chunk, group size (also
not a power of two), KV heads, head dim, ragged lengths, budget and window
drawn from a fixed generator (the same 24 shapes every run), each in both
cache formats and every other one with K and V interleaved per token, held
to the oracle's bar like the hand-picked cases.  Sizes
stay small (at most ~3000 tokens per sequence) so that the oracle keeps up."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2609_26368_amd import workloads as W
from tests.test_gpu_parity import parity_case

pytestmark = pytest.mark.gpu

MAX_ROWS = 128  # C * pow2(G) per KV head, the library's limit


def _pow2(x: int) -> int:
    return 1 << (x - 1).bit_length()


def random_shapes(n: int = 24, seed: int = 2609) -> list[W.Workload]:
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < n:
        G = int(rng.choice([1, 2, 3, 4, 5, 6, 8, 12, 16, 24, 32, 64]))
        C = int(rng.integers(1, 17))
        if C * _pow2(G) > MAX_ROWS:
            continue
        Hkv = int(rng.choice([1, 2, 4]))
        D = int(rng.choice([128, 256]))
        B = int(rng.integers(1, 4))
        ctx = int(rng.integers(max(C, 16), 3001))
        ctx_min = int(rng.integers(C, ctx + 1)) if rng.random() < 0.5 else 0
        window = int(rng.choice([0, 1, 7, 64, 200]))
        k = int(rng.integers(0 if window else 1, 700))
        i = len(out)
        out.append(W.Workload(f"rand{i:02d}_b{B}c{C}g{G}kv{Hkv}d{D}_{ctx}_{k}+{window}", B, ctx, C, G * Hkv, Hkv, D,
                              k, window, 1, ctx_min=ctx_min))
    return out


SHAPES = random_shapes()


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
@pytest.mark.parametrize("i", range(len(SHAPES)), ids=[w.name for w in SHAPES])
def test_random_shape_parity(i, kv):
    # every other shape with K and V interleaved in one record per token
    parity_case(SHAPES[i], seed=31, kv=kv, interleaved=i % 2 == 1)
