"""GPU parity at head dim 256, the paper's head layout (MQA, 64 query heads on
one KV head, head dim 256 for queries, keys and values).

Same bar and the same oracle as the head-dim-128 cases; the shapes cover one,
two and four row tiles per KV head (the three head-dim-256 full-attention
kernels), the pooled scores from stored logits and from re-reading K, both
cache formats, sinks and gates, a strided cache and the edge cases.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import hs2_oracle as O
from paper_2609_26368_amd import workloads as W
from tests import checker as CK
from tests.test_gpu_parity import dev_bf16, host_bits, note, parity_case

pytestmark = pytest.mark.gpu

PAPER = W.WORKLOADS["paper_mqa64_d256_128k_b8"]
SMALL = [
    W.shrink(PAPER, 3000, ctx_min=1800, k=300, window=64, batch=2, name="mqa64_d256@1.8k-3k"),
    W.Workload("d256_16q1kv", 2, 2500, 1, 16, 1, 256, 200, 48, 2, ctx_min=900),
    W.Workload("d256_32q2kv_C2", 1, 2200, 2, 32, 2, 256, 150, 40, 1),
    W.Workload("d256_8q2kv_C3", 2, 1700, 3, 8, 2, 256, 120, 32, 1, ctx_min=700),
    W.Workload("d256_12q4kv_C5", 1, 1400, 5, 12, 4, 256, 100, 24, 1),
    # the paper's MQA 64/1 with a 2-token verify chunk: 128 query rows per KV head
    W.Workload("mqa64_d256_C2", 2, 2200, 2, 64, 1, 256, 200, 48, 1, ctx_min=1100),
]


@pytest.mark.parametrize("w", SMALL, ids=[w.name for w in SMALL])
def test_d256_parity(w):
    parity_case(w, seed=21)


FP8 = [SMALL[0], SMALL[1], SMALL[5]]


@pytest.mark.parametrize("w", FP8, ids=[w.name for w in FP8])
def test_d256_parity_fp8(w):
    parity_case(w, seed=22, kv="fp8")


def test_d256_scores_from_k(monkeypatch):
    """One row tile with the scores recomputed from K instead of the stored logits."""
    monkeypatch.setenv("HS2_POOL_FROM_K", "1")
    parity_case(SMALL[1], seed=23)


EDGES = [
    # (name, batch, ctx, ctx_min, C, k, window)
    ("single_token", 1, 1, 0, 1, 5, 3),
    ("one_tile_plus_one", 1, 17, 0, 1, 10, 5),
    ("k_exceeds_candidates", 2, 300, 150, 2, 400, 16),
    ("window_only", 1, 900, 0, 1, 0, 50),
]


@pytest.mark.parametrize("name,B,ctx,ctx_min,C,k,win", EDGES, ids=[e[0] for e in EDGES])
def test_d256_edges(name, B, ctx, ctx_min, C, k, win):
    w = W.Workload("d256_" + name, B, ctx, C, 32, 1, 256, k, win, 1, ctx_min=ctx_min)
    parity_case(w, seed=24)


def test_d256_sparse_sink_and_gate():
    from paper_2609_26368_amd import hs2
    w = SMALL[0]
    inp = W.make_inputs(w, seed=25)
    B, C, Hq, D = w.batch, w.n_queries, w.n_q_heads, w.head_dim
    note(f"[d256 sink-gate] {w.name} lens={inp.lens.tolist()}")
    ref = O.full_attn_score_select(inp.q_fa, inp.K, inp.V, inp.lens, w.k, w.window)
    rng = np.random.default_rng(5)
    sink = (rng.standard_normal(Hq) * 3.0).astype(np.float32)
    gate = W.f32_to_bf16_bits((rng.standard_normal((B, C, Hq, D)) * 2.0).astype(np.float32))
    blk = hs2.HybridBlock(B, C, Hq, w.n_kv_heads, D, inp.K.shape[2], w.k, w.window)
    K, V = dev_bf16(inp.K), dev_bf16(inp.V)
    lens = torch.from_numpy(inp.lens.astype(np.int32)).cuda()
    got = blk.sparse(dev_bf16(inp.q_sa[0]), K, V, lens, torch.from_numpy(ref["idx"]).cuda(),
                     sink=torch.from_numpy(sink).cuda(), gate=dev_bf16(gate))
    torch.cuda.synchronize()
    want = O.sparse_attention(inp.q_sa[0], inp.K, inp.V, ref["idx"], sink=sink, gate=gate)
    CK.check_out(CK.bf16_bits_to_f64(host_bits(got)), want, "head dim 256 sparse layer with sink and gate")


def test_d256_strided_cache_layout():
    """A [B, Lmax, Hkv, D] cache passed through strides gives the same results."""
    from paper_2609_26368_amd import hs2
    w = W.Workload("d256_strided", 2, 900, 2, 16, 2, 256, 64, 32, 1, ctx_min=500)
    inp = W.make_inputs(w, seed=26)
    B, C, Hq, Hkv, D, L = w.batch, w.n_queries, w.n_q_heads, w.n_kv_heads, w.head_dim, inp.K.shape[2]
    Kt = np.ascontiguousarray(inp.K.transpose(0, 2, 1, 3))
    Vt = np.ascontiguousarray(inp.V.transpose(0, 2, 1, 3))
    blk = hs2.HybridBlock(B, C, Hq, Hkv, D, L, w.k, w.window, kv_strides=(L * Hkv * D, D, Hkv * D))
    K, V = dev_bf16(Kt), dev_bf16(Vt)
    lens = torch.from_numpy(inp.lens).cuda()
    out, idx = blk.full(dev_bf16(inp.q_fa), K, V, lens)
    ref = O.full_attn_score_select(inp.q_fa, inp.K, inp.V, inp.lens, w.k, w.window)
    ridx = torch.from_numpy(ref["idx"]).cuda()
    sa = blk.sparse(dev_bf16(inp.q_sa[0]), K, V, lens, ridx)
    torch.cuda.synchronize()
    CK.check_out(CK.bf16_bits_to_f64(host_bits(out)), ref["out"])
    CK.check_idx(idx.cpu().numpy(), ref["idx"], ref["P"], inp.lens, C, w.window)
    CK.check_out(CK.bf16_bits_to_f64(host_bits(sa)), O.sparse_attention(inp.q_sa[0], inp.K, inp.V, ref["idx"]))


@pytest.mark.parametrize("variant", [6, 8])
@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_d256_both_kernel_shapes(variant, kv, monkeypatch):
    """Four row tiles: the 16-token / 3-stage and the 32-token / 2-stage kernels."""
    monkeypatch.setenv("HS2_FA_VARIANT", str(variant))
    parity_case(SMALL[0], seed=27, kv=kv)
