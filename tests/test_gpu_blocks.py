"""GPU parity of block-level selection (the HySparse granularity the paper
compares token-level selection against).

Selection alone is checked bit for bit against the oracle on scores whose
block sums are exact in fp32 in any order (small multiples of 2^-12), so the
GPU's summation order cannot matter: ties, zeros, scores below FLT_MIN,
every supported block size, a row at the 16384-block capacity.  The whole
layer is then checked like the token-level path, with the index rows held
to the block-aware bar of tests/checker.py, and the sparse layers run on
the GPU's block rows.
"""
from __future__ import annotations

import zlib

import numpy as np
import pytest
import torch

from oracle import hs2_oracle as O
from paper_2609_26368_amd import workloads as W
from tests import checker as CK
from tests.test_gpu_parity import SMALL, dev_bf16, host_bits, note

pytestmark = pytest.mark.gpu


def _select_blocks_case(B, Hkv, C, Lmax, lens, k, win, block, scores):
    from paper_2609_26368_amd import hs2
    dims = hs2.make_dims(B, C, 8 * Hkv, Hkv, 128, Lmax)
    ws = torch.empty(hs2.hs2_workspace_bytes(dims, k, win), dtype=torch.uint8, device="cuda")
    idx = torch.empty((B, Hkv, C, k + win), dtype=torch.int32, device="cuda")
    hs2.hs2_select_blocks_from_scores(dims, torch.from_numpy(scores).cuda(), torch.from_numpy(lens).cuda(), k, win,
                                      block, idx, ws)
    torch.cuda.synchronize()
    got = idx.cpu().numpy()
    for b in range(B):
        for g in range(Hkv):
            for c in range(C):
                pos = int(lens[b]) - C + c
                want = O.select_row_blocks(scores[b, g, c], pos, k, win, block)
                assert np.array_equal(got[b, g, c], want), (b, g, c, got[b, g, c][:20], want[:20])


SEL = [
    # (name, B, Hkv, C, Lmax, k, window, block, score kind)
    ("random_b64", 2, 3, 2, 9000, 1024, 128, 64, "grid"),
    ("ties_b16", 1, 2, 3, 5000, 256, 16, 16, "ties"),
    ("all_equal_b32", 1, 1, 1, 4000, 320, 8, 32, "const"),
    ("tiny_and_zero_b64", 1, 2, 1, 6000, 512, 64, 64, "tiny"),
    ("b128", 2, 1, 1, 20000, 1024, 100, 128, "grid"),
    ("b256_partial_edge", 1, 1, 4, 3001, 512, 37, 256, "grid"),
    ("k_covers_all_blocks", 1, 1, 1, 900, 1024, 40, 64, "grid"),
    ("window_only", 1, 1, 1, 900, 0, 40, 64, "grid"),
    ("capacity_16384_blocks", 1, 1, 1, 16384 * 16, 2048, 128, 16, "grid"),
]


@pytest.mark.parametrize("name,B,Hkv,C,Lmax,k,win,block,kind", SEL, ids=[s[0] for s in SEL])
def test_select_blocks_exact(name, B, Hkv, C, Lmax, k, win, block, kind):
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    shape = (B, Hkv, C, Lmax)
    if kind == "grid":  # multiples of 2^-12: block sums exact in any order
        s = (rng.integers(0, 16, size=shape) / 4096.0).astype(np.float32)
    elif kind == "ties":
        s = (rng.integers(0, 2, size=shape) / 4096.0).astype(np.float32)
    elif kind == "const":
        s = np.full(shape, 1.0 / 64, dtype=np.float32)
    else:  # zeros, values below FLT_MIN (count as zero) and a few grid values
        s = np.zeros(shape, dtype=np.float32)
        s[rng.random(shape) < 0.3] = np.float32(1e-39)
        m = rng.random(shape) < 0.01
        s[m] = (rng.integers(1, 16, size=int(m.sum())) / 4096.0).astype(np.float32)
    lens = rng.integers(max(C, Lmax // 2), Lmax + 1, size=B).astype(np.int32)
    lens[0] = Lmax
    note(f"[block select] {name} lens={lens.tolist()} k={k} W={win} block={block}")
    _select_blocks_case(B, Hkv, C, Lmax, lens, k, win, block, s)


BLOCK_CASES = [SMALL[0], SMALL[1], SMALL[2], SMALL[3], SMALL[4]]


@pytest.mark.parametrize("w", BLOCK_CASES, ids=[w.name for w in BLOCK_CASES])
def test_block_selection_parity(w):
    from paper_2609_26368_amd import hs2
    block = 64
    k = max(block, w.k // block * block)
    inp = W.make_inputs(w, seed=31)
    B, C, Hq, Hkv, D, L = w.batch, w.n_queries, w.n_q_heads, w.n_kv_heads, w.head_dim, inp.K.shape[2]
    note(f"[block parity] {w.name} lens={inp.lens.tolist()} k={k} W={w.window}")
    ref = O.full_attn_score_select(inp.q_fa, inp.K, inp.V, inp.lens, k, w.window, block=block)
    blk = hs2.HybridBlock(B, C, Hq, Hkv, D, L, k, w.window)
    K, V = dev_bf16(inp.K), dev_bf16(inp.V)
    lens = torch.from_numpy(inp.lens.astype(np.int32)).cuda()
    stats = torch.empty((B, C, Hq, 2), dtype=torch.float32, device="cuda")
    out, idx = blk.full(dev_bf16(inp.q_fa), K, V, lens, stats=stats, block=block)
    gidx = idx.clone()
    sa = blk.sparse(dev_bf16(inp.q_sa[0]), K, V, lens, gidx)
    torch.cuda.synchronize()
    CK.check_out(CK.bf16_bits_to_f64(host_bits(out)), ref["out"], "full-attention out")
    assert np.allclose(stats.cpu().numpy()[..., 0], ref["M"], rtol=1e-5, atol=1e-5)
    r = CK.check_block_idx(gidx.cpu().numpy(), ref["idx"], ref["P"], inp.lens, C, w.window, block)
    # the sparse layer over the GPU's block rows (contiguous 64-token runs)
    want = O.sparse_attention(inp.q_sa[0], inp.K, inp.V, gidx.cpu().numpy())
    CK.check_out(CK.bf16_bits_to_f64(host_bits(sa)), want, "sparse layer on block rows")
    note(f"[block parity] {w.name}: {r}")
