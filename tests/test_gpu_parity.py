"""GPU parity: libhs2.so (through its C ABI) against the CPU oracle.

Every case draws seeded bf16 inputs, runs the hybrid block on the GPU and the
oracle on the same bits, and checks out / stats / pooled scores / index rows
/ sparse-layer outputs to the bar in tests/checker.py.  The sparse layers are
checked twice: chained on the GPU's own selection (when it equals the
oracle's) and fed the oracle's selection (always).
"""
from __future__ import annotations

import sys
import zlib

import numpy as np
import pytest
import torch

from oracle import hs2_oracle as O
from paper_2609_26368_amd import workloads as W
from tests import checker as CK

pytestmark = pytest.mark.gpu


def _hs2():
    from paper_2609_26368_amd import hs2
    return hs2


def dev_bf16(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda").view(torch.bfloat16)


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def note(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def dev_cache(inp):
    """K, V on the device and the scales of an E4M3 cache (None for bf16)."""
    if inp.k_scale is None:
        return dev_bf16(inp.K), dev_bf16(inp.V), None
    return (torch.from_numpy(inp.K).cuda(), torch.from_numpy(inp.V).cuda(),
            (torch.from_numpy(inp.k_scale).cuda(), torch.from_numpy(inp.v_scale).cuda()))


def run_gpu(inp, oracle_idx=None, interleaved=False):
    """Hybrid block on the GPU; returns host copies of every result.  With
    interleaved, K and V of a token share one 2 D record: one [B, Hkv, Lmax,
    2 D] tensor passed as two strided views."""
    hs2 = _hs2()
    w = inp.w
    B, C, Hq, Hkv, D = w.batch, w.n_queries, w.n_q_heads, w.n_kv_heads, w.head_dim
    Lmax = inp.K.shape[2]
    strides = (Hkv * Lmax * 2 * D, Lmax * 2 * D, 2 * D) if interleaved else None
    blk = hs2.HybridBlock(B, C, Hq, Hkv, D, Lmax, w.k, w.window, kv_strides=strides)
    K, V, sc = dev_cache(inp)
    if interleaved:
        KV = torch.cat([K, V], dim=-1).contiguous()
        K, V = KV[..., :D], KV[..., D:]
    lens = torch.from_numpy(inp.lens.astype(np.int32)).cuda()
    stats = torch.empty((B, C, Hq, 2), dtype=torch.float32, device="cuda")
    scores = torch.zeros((B, Hkv, C, Lmax), dtype=torch.float32, device="cuda")
    q_fa = dev_bf16(inp.q_fa)
    # with the scores and statistics requested, then the plain call (scores in the workspace)
    out_s, idx_s = blk.full(q_fa, K, V, lens, stats=stats, scores=scores, kv_scales=sc)
    out, idx = blk.full(q_fa, K, V, lens, kv_scales=sc)
    sa = [blk.sparse(dev_bf16(qs), K, V, lens, idx, kv_scales=sc) for qs in inp.q_sa]
    sa_ref_idx = None
    if oracle_idx is not None:
        ridx = torch.from_numpy(oracle_idx).cuda()
        sa_ref_idx = [blk.sparse(dev_bf16(qs), K, V, lens, ridx, kv_scales=sc) for qs in inp.q_sa]
    torch.cuda.synchronize()
    res = {"out": CK.bf16_bits_to_f64(host_bits(out)), "idx": idx.cpu().numpy(), "stats": stats.cpu().numpy(),
           "scores": scores.cpu().numpy(), "sa": [CK.bf16_bits_to_f64(host_bits(t)) for t in sa],
           "out_with_scores": CK.bf16_bits_to_f64(host_bits(out_s)), "idx_with_scores": idx_s.cpu().numpy()}
    if sa_ref_idx is not None:
        res["sa_ref_idx"] = [CK.bf16_bits_to_f64(host_bits(t)) for t in sa_ref_idx]
    return res


def _v_absmax(inp) -> np.ndarray:
    """max_t |V[b, g, t, d]| over each sequence's tokens, [B, Hkv, D] float64."""
    w = inp.w
    out = np.zeros((w.batch, w.n_kv_heads, w.head_dim))
    for b in range(w.batch):
        for g in range(w.n_kv_heads):
            L = int(inp.lens[b])
            if L > 0:
                out[b, g] = np.abs(O.cache_rows(inp.V, b, g, slice(0, L), inp.v_scale)).max(axis=0)
    return out


def _check_out_hull(inp, vmax, out, what):
    assert np.isfinite(out).all(), f"{what}: non-finite output"
    assert (np.abs(out) <= vmax * (1 + 2 ** -8) + 1e-30).all(), f"{what}: output outside the hull of its V rows"


def compare(inp, ref, gpu, groups=None):
    w = inp.w
    G = w.group
    rows = None
    if groups is not None:
        rows = np.zeros((w.batch, w.n_queries, w.n_q_heads), dtype=bool)
        for b, g in groups:
            rows[b, :, g * G:(g + 1) * G] = True
    # every row, sampled or not: oracle-free structure of the selection, and
    # outputs finite and inside the hull of their value rows (an attention
    # output is a convex combination of V rows: |out[d]| <= max_t |V[t, d]|)
    r_struct = CK.check_idx_structure(gpu["idx"], inp.lens, w.n_queries, w.k, w.window)
    vmax = np.repeat(_v_absmax(inp), w.group, axis=1)[:, None]  # [B, 1, Hq, D]
    _check_out_hull(inp, vmax, gpu["out"], "full-attention out")
    for li in range(len(inp.q_sa)):
        _check_out_hull(inp, vmax, gpu["sa"][li], f"sparse layer {li}")
    r_out = CK.check_out(gpu["out"], ref["out"], "full-attention out", rows)
    # stats: M natural-log units, Z
    M, Z = gpu["stats"][..., 0], gpu["stats"][..., 1]
    sel = rows if rows is not None else np.ones(M.shape, dtype=bool)
    assert np.allclose(M[sel], ref["M"][sel], rtol=1e-5, atol=1e-5), "stats M"
    assert np.allclose(Z[sel], ref["Z"][sel], rtol=1e-4), "stats Z"
    r_sc = CK.check_scores(gpu["scores"], ref["P"], inp.lens, w.n_queries, w.window, groups)
    r_idx = CK.check_idx(gpu["idx"], ref["idx"], ref["P"], inp.lens, w.n_queries, w.window, groups)
    assert np.array_equal(gpu["idx_with_scores"], gpu["idx"]), "selection depends on where the scores are kept"
    assert np.array_equal(gpu["out_with_scores"], gpu["out"]), "full-attention output depends on the score request"
    for li, qs in enumerate(inp.q_sa):
        ref_sa = O.sparse_attention(qs, inp.K, inp.V, ref["idx"], groups=groups, k_scale=inp.k_scale,
                                    v_scale=inp.v_scale)
        CK.check_out(gpu["sa_ref_idx"][li], ref_sa, f"sparse layer {li} (oracle selection)", rows)
        if r_idx["swaps"] == 0:
            CK.check_out(gpu["sa"][li], ref_sa, f"sparse layer {li} (own selection)", rows)
    return {**r_out, **r_sc, **r_idx, **r_struct}


def parity_case(w, seed=W.BASE_SEED, lmax=None, groups=None, kv="bf16", interleaved=False):
    inp = W.make_inputs(w, seed=seed, lmax=lmax, kv=kv)
    note(f"[parity] {w.name} kv={kv} seed={seed} lens={inp.lens.tolist()} C={w.n_queries} Hq={w.n_q_heads} "
         f"Hkv={w.n_kv_heads} k={w.k} W={w.window}" + (" interleaved K|V" if interleaved else ""))
    ref = O.full_attn_score_select(inp.q_fa, inp.K, inp.V, inp.lens, w.k, w.window, groups=groups,
                                   k_scale=inp.k_scale, v_scale=inp.v_scale)
    gpu = run_gpu(inp, oracle_idx=ref["idx"], interleaved=interleaved)
    r = compare(inp, ref, gpu, groups)
    note(f"[parity] {w.name}: {r}")
    return inp, ref, gpu


WL = W.WORKLOADS
SMALL = [
    WL["decode_4k_16q2kv"],
    W.shrink(WL["block_32k_32q4kv"], 6173, name="block_32q4kv@6173"),
    W.shrink(WL["ragged_16k_128k_b8_needles"], 9000, ctx_min=1500, k=512, name="ragged_b8_needles@1.5k-9k"),
    W.shrink(WL["chunk8_128k_b4"], 5000, k=1024, batch=2, name="chunk8_b2@5000"),
    W.shrink(WL["stress_512k_b2_64q8kv"], 6001, k=1024, batch=1, name="64q8kv@6001"),
]


@pytest.mark.parametrize("w", SMALL, ids=[w.name for w in SMALL])
def test_parity_small(w):
    inp, ref, gpu = parity_case(w)
    if w.needles:
        for b in range(w.batch):
            for g in range(w.n_kv_heads):
                assert set(inp.needles[b].tolist()) <= set(gpu["idx"][b, g, 0].tolist())


HEADS = [  # (Hq, Hkv, C): group sizes incl. non-powers of two and the 128-row maximum
    (12, 4, 1), (8, 8, 3), (16, 1, 2), (32, 1, 4), (64, 1, 2), (8, 1, 16), (6, 2, 5),
]


@pytest.mark.parametrize("Hq,Hkv,C", HEADS, ids=[f"{a}q{b}kv_C{c}" for a, b, c in HEADS])
def test_parity_head_layouts(Hq, Hkv, C):
    w = W.Workload(f"heads_{Hq}_{Hkv}_{C}", 2, 1500, C, Hq, Hkv, 128, 200, 48, 2, ctx_min=700)
    parity_case(w, seed=5)


EDGES = [
    # (name, batch, ctx, ctx_min, C, k, window)
    ("window_covers_all", 2, 100, 40, 1, 64, 128),
    ("len_equals_chunk", 1, 4, 0, 4, 8, 2),
    ("single_token", 1, 1, 0, 1, 5, 3),
    ("no_window", 1, 777, 0, 2, 100, 0),
    ("window_only", 1, 900, 0, 3, 0, 50),
    ("k_exceeds_candidates", 2, 300, 150, 2, 400, 16),
    ("one_tile_plus_one", 1, 65, 0, 1, 10, 5),
]


@pytest.mark.parametrize("name,B,ctx,ctx_min,C,k,win", EDGES, ids=[e[0] for e in EDGES])
def test_parity_edges(name, B, ctx, ctx_min, C, k, win):
    w = W.Workload(name, B, ctx, C, 16, 2, 128, k, win, 1, ctx_min=ctx_min)
    parity_case(w, seed=7)


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
def test_parity_len_below_chunk(kv):
    """Outside the precondition len >= C: queries at negative positions get an
    all -1 row, a zero output and (M, Z) = (-inf, 0); len = 0 sequences too."""
    w = W.Workload("len_below_chunk", 3, 300, 4, 16, 2, 128, 16, 8, 1, ctx_min=100)
    inp = W.make_inputs(w, seed=13, kv=kv)
    inp.lens[:] = [2, 0, 300]
    note(f"[parity] len_below_chunk kv={kv} lens={inp.lens.tolist()}")
    ref = O.full_attn_score_select(inp.q_fa, inp.K, inp.V, inp.lens, w.k, w.window, k_scale=inp.k_scale,
                                   v_scale=inp.v_scale)
    gpu = run_gpu(inp, oracle_idx=ref["idx"])
    compare(inp, ref, gpu)
    assert (gpu["idx"][1] == -1).all() and (gpu["out"][1] == 0).all()
    assert (gpu["idx"][0, :, :2] == -1).all() and (gpu["out"][0, :2] == 0).all()


def test_parity_padded_capacity():
    """Cache capacity larger than every length (rows past len are never read)."""
    w = W.Workload("capacity", 3, 1000, 2, 16, 4, 128, 96, 32, 1, ctx_min=300)
    parity_case(w, seed=9, lmax=1531)


def test_strided_cache_layout():
    """A [B, Lmax, Hkv, D] cache passed through strides gives the same results."""
    hs2 = _hs2()
    w = W.Workload("strided", 2, 800, 2, 16, 4, 128, 64, 32, 1, ctx_min=500)
    inp = W.make_inputs(w, seed=3)
    B, C, Hq, Hkv, D, L = w.batch, w.n_queries, w.n_q_heads, w.n_kv_heads, w.head_dim, inp.K.shape[2]
    Kt = np.ascontiguousarray(inp.K.transpose(0, 2, 1, 3))
    Vt = np.ascontiguousarray(inp.V.transpose(0, 2, 1, 3))
    strides = (L * Hkv * D, D, Hkv * D)
    blk = hs2.HybridBlock(B, C, Hq, Hkv, D, L, w.k, w.window, kv_strides=strides)
    K, V = dev_bf16(Kt), dev_bf16(Vt)
    lens = torch.from_numpy(inp.lens).cuda()
    out, idx = blk.full(dev_bf16(inp.q_fa), K, V, lens)
    sa = blk.sparse(dev_bf16(inp.q_sa[0]), K, V, lens, idx)
    torch.cuda.synchronize()
    ref = O.full_attn_score_select(inp.q_fa, inp.K, inp.V, inp.lens, w.k, w.window)
    CK.check_out(CK.bf16_bits_to_f64(host_bits(out)), ref["out"])
    CK.check_idx(idx.cpu().numpy(), ref["idx"], ref["P"], inp.lens, C, w.window)
    if (idx.cpu().numpy() == ref["idx"]).all():
        CK.check_out(CK.bf16_bits_to_f64(host_bits(sa)), O.sparse_attention(inp.q_sa[0], inp.K, inp.V, ref["idx"]))


@pytest.mark.parametrize("kv", ["bf16", "fp8"])
@pytest.mark.parametrize("w", [SMALL[2], SMALL[3]], ids=[SMALL[2].name, SMALL[3].name])
def test_interleaved_cache_layout(w, kv):
    """K and V of a token in one 2 D record (the benchmark's layout): the
    oracle's bar, and bit for bit the results of two separate tensors."""
    inp, ref, gpu = parity_case(w, seed=13, kv=kv, interleaved=True)
    split = run_gpu(inp, oracle_idx=ref["idx"])
    for key in ("out", "idx", "stats", "scores", "out_with_scores", "idx_with_scores"):
        np.testing.assert_array_equal(gpu[key], split[key], err_msg=key)
    for a, b in zip(gpu["sa"] + gpu["sa_ref_idx"], split["sa"] + split["sa_ref_idx"]):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("w", [SMALL[0], SMALL[2]], ids=[SMALL[0].name, SMALL[2].name])
def test_parity_scores_from_k(w, monkeypatch):
    """Single row tile with the scores recomputed from K instead of the stored logits."""
    monkeypatch.setenv("HS2_POOL_FROM_K", "1")
    parity_case(w, seed=7)


SINK_GATE = [SMALL[1], SMALL[3], SMALL[4]]


@pytest.mark.parametrize("w", SINK_GATE, ids=[w.name for w in SINK_GATE])
def test_sparse_sink_and_gate(w):
    """Sparse layers with per-head sink logits and sigmoid output gates, on the oracle's selection."""
    hs2 = _hs2()
    inp = W.make_inputs(w, seed=11)
    B, C, Hq, D = w.batch, w.n_queries, w.n_q_heads, w.head_dim
    note(f"[sink-gate] {w.name} lens={inp.lens.tolist()}")
    ref = O.full_attn_score_select(inp.q_fa, inp.K, inp.V, inp.lens, w.k, w.window)
    rng = np.random.default_rng(5)
    sink = (rng.standard_normal(Hq) * 3.0).astype(np.float32)  # some heads' sinks dominate their logits
    gate = W.f32_to_bf16_bits((rng.standard_normal((B, C, Hq, D)) * 2.0).astype(np.float32))
    blk = hs2.HybridBlock(B, C, Hq, w.n_kv_heads, D, inp.K.shape[2], w.k, w.window)
    K, V = dev_bf16(inp.K), dev_bf16(inp.V)
    lens = torch.from_numpy(inp.lens.astype(np.int32)).cuda()
    ridx = torch.from_numpy(ref["idx"]).cuda()
    q = dev_bf16(inp.q_sa[0])
    for s_, g_ in [(sink, None), (None, gate), (sink, gate)]:
        got = blk.sparse(q, K, V, lens, ridx, sink=None if s_ is None else torch.from_numpy(s_).cuda(),
                         gate=None if g_ is None else dev_bf16(g_))
        torch.cuda.synchronize()
        want = O.sparse_attention(inp.q_sa[0], inp.K, inp.V, ref["idx"], sink=s_, gate=g_)
        CK.check_out(CK.bf16_bits_to_f64(host_bits(got)), want,
                     f"sparse layer, sink={s_ is not None}, gate={g_ is not None}")


# ---------------------------------------------------------------- selection alone: bit-exact
def _select_case(B, Hkv, C, Lmax, lens, k, win, scores):
    hs2 = _hs2()
    dims = hs2.make_dims(B, C, 8 * Hkv, Hkv, 128, Lmax)
    ws = torch.empty(hs2.hs2_workspace_bytes(dims, k, win), dtype=torch.uint8, device="cuda")
    idx = torch.empty((B, Hkv, C, k + win), dtype=torch.int32, device="cuda")
    hs2.hs2_select_from_scores(dims, torch.from_numpy(scores).cuda(), torch.from_numpy(lens).cuda(), k, win, idx, ws)
    torch.cuda.synchronize()
    got = idx.cpu().numpy()
    for b in range(B):
        for g in range(Hkv):
            for c in range(C):
                pos = int(lens[b]) - C + c
                want = O.select_row(scores[b, g, c], pos, k, win)
                assert np.array_equal(got[b, g, c], want), (b, g, c, got[b, g, c][:20], want[:20])


SEL = [
    # (name, B, Hkv, C, Lmax, k, window, score kind)
    ("random", 2, 3, 2, 5000, 300, 40, "uniform"),
    ("heavy_ties", 2, 2, 1, 7000, 500, 16, "ties"),
    ("all_equal", 1, 2, 1, 3000, 700, 8, "const"),
    # every chunk overflows the filter's LDS candidate buffer; the row's
    # candidates exceed the resolver's LDS capacity
    ("all_equal_long", 1, 1, 2, 20000, 5000, 64, "const"),
    # one-workgroup rows (at most 16384 tokens): candidates past the
    # resolver's LDS capacity, and a row of exactly the limit
    ("all_equal_one_chunk", 1, 1, 1, 16000, 3000, 32, "const"),
    ("lognormal_16384", 2, 1, 1, 16384, 1024, 64, "lognormal"),
    ("denormals_and_zeros", 1, 1, 3, 2000, 100, 10, "tiny"),
    ("lognormal_long", 1, 2, 1, 200000, 4096, 256, "lognormal"),
    ("k_equals_N", 1, 1, 1, 1000, 990, 10, "uniform"),
    ("k_zero", 1, 1, 2, 1000, 0, 10, "uniform"),
    # scores on both sides of first-level bin edges (and -0.0): the filter
    # tests raw bits against per-row bounds; two-kernel and one-workgroup rows
    ("bin_edges", 2, 2, 2, 40000, 3000, 32, "edges"),
    ("bin_edges_one_chunk", 1, 2, 1, 12000, 800, 16, "edges"),
    # threshold in the top clamped bin, and in the bottom bin
    ("top_clamp_bin", 1, 2, 1, 30000, 300, 16, "top"),
    ("bottom_bin", 1, 1, 2, 30000, 2000, 16, "bottom"),
]

# First-level bin edges of the selection's histogram: bin d >= 1 starts at
# the float whose bits are (d + 1120) << 19 (an 8-exponent-bit, 4-mantissa-bit
# prefix; bins 0 and 1023 are clamped).
_EDGE_BITS = [((d + 1120) << 19) + o for d in (1, 2, 300, 917, 1000, 1022, 1023) for o in (-1, 0, 1)]
_EDGES = np.concatenate([np.array(_EDGE_BITS, dtype=np.uint32).view(np.float32),
                         np.array([0.0, -0.0, 1e-30, 3e-39], dtype=np.float32)])


@pytest.mark.parametrize("name,B,Hkv,C,Lmax,k,win,kind", SEL, ids=[s[0] for s in SEL])
def test_select_from_scores_exact(name, B, Hkv, C, Lmax, k, win, kind):
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    shape = (B, Hkv, C, Lmax)
    if kind == "uniform":
        s = rng.random(shape, dtype=np.float32)
    elif kind == "ties":
        s = (rng.integers(0, 50, size=shape) / 64.0).astype(np.float32)
    elif kind == "const":
        s = np.full(shape, 0.25, dtype=np.float32)
    elif kind == "tiny":
        s = rng.choice(np.array([0.0, 1e-40, 3e-39, 1e-38, 2e-38, 1.0], dtype=np.float32), size=shape)
    elif kind == "edges":
        s = rng.choice(_EDGES, size=shape)
    elif kind == "top":  # most scores at or above 124 (the top clamped bin)
        s = np.where(rng.random(shape) < 0.3, rng.random(shape), 124.0 + 1e4 * rng.random(shape)).astype(np.float32)
    elif kind == "bottom":  # most scores below 7e-18 (bin 0), a few above
        tiny = rng.choice(np.array([0.0, -0.0, 1e-38, 1e-30, 1e-20, 6e-18], dtype=np.float32), size=shape)
        s = np.where(rng.random(shape) < 0.02, rng.random(shape).astype(np.float32), tiny).astype(np.float32)
    else:
        s = (np.exp(rng.standard_normal(shape)) / Lmax).astype(np.float32)
    lens = np.array([Lmax - 17 * b for b in range(B)], dtype=np.int32)
    note(f"[select] {name} shape={shape} k={k} W={win}")
    _select_case(B, Hkv, C, Lmax, lens, k, win, s)
