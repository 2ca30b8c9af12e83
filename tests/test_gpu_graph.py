"""A whole hybrid-block step captured into a HIP graph and replayed.

The library launches kernels only (no memset nodes: counters and histograms
are cleared by kernels), so one decode step (the full-attention call and the
sparse layers) can be captured once and replayed.  Each replay is checked
bit for bit against the eager results, with the program's own eager work and
a synchronisation between replays, and with inputs changed in place between
replays (a replay must read the current inputs).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2609_26368_amd import workloads as W
from tests.test_gpu_parity import dev_bf16, note

pytestmark = pytest.mark.gpu

CASES = [
    (W.Workload("graph_chunk4", 2, 3000, 4, 32, 4, 128, 256, 64, 3, ctx_min=1500), "bf16"),
    (W.Workload("graph_chunk4_fp8", 2, 3000, 4, 32, 4, 128, 256, 64, 3, ctx_min=1500), "fp8"),
    (W.Workload("graph_mqa64_d256", 2, 2500, 1, 64, 1, 256, 256, 64, 3, ctx_min=1200), "bf16"),
]


@pytest.mark.parametrize("w,kv", CASES, ids=[c[0].name for c in CASES])
def test_block_step_in_a_graph(w, kv):
    from paper_2609_26368_amd import hs2
    inp = W.make_inputs(w, seed=51, kv=kv)
    B, C, Hq, Hkv, D, L = w.batch, w.n_queries, w.n_q_heads, w.n_kv_heads, w.head_dim, inp.K.shape[2]
    note(f"[graph] {w.name} kv={kv} lens={inp.lens.tolist()}")
    blk = hs2.HybridBlock(B, C, Hq, Hkv, D, L, w.k, w.window)
    if kv == "fp8":
        K, V = torch.from_numpy(inp.K).cuda(), torch.from_numpy(inp.V).cuda()
        sc = (torch.from_numpy(inp.k_scale).cuda(), torch.from_numpy(inp.v_scale).cuda())
    else:
        K, V, sc = dev_bf16(inp.K), dev_bf16(inp.V), None
    lens = torch.from_numpy(inp.lens.astype(np.int32)).cuda()
    q_fa = dev_bf16(inp.q_fa)
    q_sa = [dev_bf16(x) for x in inp.q_sa]
    out = torch.empty((B, C, Hq, D), dtype=torch.bfloat16, device="cuda")
    idx = torch.empty((B, Hkv, C, w.k + w.window), dtype=torch.int32, device="cuda")
    sa = [torch.empty_like(out) for _ in q_sa]

    def step(stream=None):
        blk.full(q_fa, K, V, lens, out=out, idx=idx, kv_scales=sc, stream=stream)
        for qs, o in zip(q_sa, sa):
            blk.sparse(qs, K, V, lens, idx, out=o, kv_scales=sc, stream=stream)

    def snapshot():
        torch.cuda.synchronize()
        return [out.clone(), idx.clone()] + [o.clone() for o in sa]

    step()  # eager; also the library's one-time set-up, outside the capture
    want = snapshot()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step(stream=s)  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=s):
        step(stream=s)
    for rep in range(3):
        for t in [out, *sa]:
            t.zero_()
        idx.fill_(-7)
        g.replay()
        got = snapshot()
        for a, b in zip(got, want):
            assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                               b.view(torch.int16) if b.dtype == torch.bfloat16 else b), f"replay {rep}"
        step()  # eager work between replays
        torch.cuda.synchronize()
    # a replay reads the current inputs: new queries in place -> the eager results for them
    q_fa.copy_(q_sa[0])
    step()
    want2 = snapshot()
    g.replay()
    got2 = snapshot()
    for a, b in zip(got2, want2):
        assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                           b.view(torch.int16) if b.dtype == torch.bfloat16 else b), "replay after new inputs"
