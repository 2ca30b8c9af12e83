"""GPU: the allocation-free sparse layer (hs2_sparse_attn_noalloc, static
per-GPU scratch) against hs2_sparse_attn (caller's workspace) through the C
ABI: two calls in a row, the second with a smaller input, each bit-identical
to the workspace entry point's output and within the parity bar of the
oracle's sparse attention over the same selection."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import hs2_oracle as O
from paper_2609_26368_amd import workloads as W
from tests import checker as CK

pytestmark = pytest.mark.gpu

CASES = [  # the larger call first, then a smaller one (the array keeps the first call's contents)
    W.Workload("noalloc_chunk8_b2", 2, 5000, 8, 32, 4, 128, 1024, 256, 1, ctx_min=4200),
    W.Workload("noalloc_decode", 1, 3000, 1, 16, 2, 128, 256, 64, 1),
]


def _dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def _f64(t):
    return CK.bf16_bits_to_f64(t.view(torch.int16).cpu().numpy().view(np.uint16))


def test_noalloc_sparse_matches_workspace_entry_point():
    from paper_2609_26368_amd import hs2
    for i, w in enumerate(CASES):
        inp = W.make_inputs(w, seed=31 + i)
        print(f"[noalloc] call {i}: {w.name} lens={inp.lens.tolist()} C={w.n_queries} slots={w.slots}", flush=True)
        ref = O.full_attn_score_select(inp.q_fa, inp.K, inp.V, inp.lens, w.k, w.window)
        B, C, Hq, Hkv, D = w.batch, w.n_queries, w.n_q_heads, w.n_kv_heads, w.head_dim
        dims = hs2.make_dims(B, C, Hq, Hkv, D, inp.K.shape[2])
        K, V, q = _dev(inp.K), _dev(inp.V), _dev(inp.q_sa[0])
        lens = torch.from_numpy(inp.lens.astype(np.int32)).cuda()
        idx = torch.from_numpy(ref["idx"]).cuda()
        ws = torch.empty(hs2.hs2_workspace_bytes(dims, w.k, w.window), dtype=torch.uint8, device="cuda")
        out_ws = torch.empty((B, C, Hq, D), dtype=torch.bfloat16, device="cuda")
        out_na = torch.full((B, C, Hq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        hs2.hs2_sparse_attn(dims, q, K, V, lens, idx, w.slots, out_ws, ws)
        hs2.hs2_sparse_attn_noalloc(dims, q, K, V, lens, idx, w.slots, out_na)
        torch.cuda.synchronize()
        assert torch.equal(out_na.view(torch.int16), out_ws.view(torch.int16)), f"{w.name}: outputs differ"
        want = O.sparse_attention(inp.q_sa[0], inp.K, inp.V, ref["idx"])
        CK.check_out(_f64(out_na), want, f"{w.name}: allocation-free sparse layer")
