"""Pins of the CPU oracle against things other than itself.

Each ``pin_*`` takes the oracle module and raises AssertionError when the
module disagrees with a closed form, a library routine (torch's CPU attention
in float64), a brute-force enumeration or an invariant the method fixes.
test_oracle_pins.py runs them on the oracle (all must pass) and on copies of
the oracle with planted mistakes (each copy must fail at least one).
"""
from __future__ import annotations

import itertools
import math
import os

import numpy as np
import torch

from paper_2609_26368_amd.workloads import f32_to_bf16_bits, Workload, make_inputs

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _bits(rng, shape, scale=1.0):
    return f32_to_bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))


def _f64(bits):
    # independent decode for the checks: via torch's own bfloat16 dtype
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    return t.to(torch.float64).numpy()


def _sdpa(q, K, V, scale, mask=None):
    """torch CPU float64 attention: q [Hq, 1, D] over K/V [Hq, n, D]."""
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(K), torch.from_numpy(V),
        attn_mask=None if mask is None else torch.from_numpy(mask), scale=scale).numpy()


# ---------------------------------------------------------------- decoding
def pin_bf16_decode(O):
    bits = np.array([0x3F80, 0xC000, 0x3F00, 0x4049, 0x0000, 0x8000, 0x3C00, 0x7F7F], dtype=np.uint16)
    want = [1.0, -2.0, 0.5, 3.140625, 0.0, -0.0, 2.0 ** -7, 3.3895313892515355e38]
    got = O.bf16_to_f64(bits)
    assert np.array_equal(got, np.array(want)), got
    rng = np.random.default_rng(1)
    b = _bits(rng, 1000, 7.0)
    assert np.array_equal(O.bf16_to_f64(b), _f64(b))


# ---------------------------------------------------------------- attention
def pin_attend_vs_library(O):
    rng = np.random.default_rng(2)
    for n, D, scale in [(1, 8, 0.3), (37, 16, 0.25), (300, 128, 1 / math.sqrt(128)), (5, 4, 2.0),
                        (90, 256, 1 / math.sqrt(256))]:
        q = _f64(_bits(rng, D))
        K = _f64(_bits(rng, (n, D), 2.0))
        V = _f64(_bits(rng, (n, D)))
        out, M, Z, p = O.attend(q, K, V, scale)
        ref = _sdpa(q[None, None], K[None], V[None], scale)[0, 0]
        assert np.allclose(out, ref, rtol=1e-12, atol=1e-13), (n, np.abs(out - ref).max())
        s = torch.from_numpy(K) @ torch.from_numpy(q) * scale
        assert np.allclose(p, torch.softmax(s, 0).numpy(), rtol=1e-12, atol=1e-15)
        assert abs((M + math.log(Z)) - torch.logsumexp(s, 0).item()) < 1e-12
        assert abs(M - s.max().item()) < 1e-12


def pin_attend_special_cases(O):
    rng = np.random.default_rng(3)
    D = 16
    q = _f64(_bits(rng, D))
    V = _f64(_bits(rng, (9, D)))
    K = _f64(_bits(rng, (9, D)))
    # one token: the output is that token's value, Z = 1
    out, M, Z, p = O.attend(q, K[:1], V[:1], 0.5)
    assert np.array_equal(out, V[0]) and Z == 1.0 and p[0] == 1.0
    assert abs(M - 0.5 * float(q @ K[0])) < 1e-12
    # identical keys: uniform weights, output = mean of values
    Kid = np.repeat(K[:1], 9, axis=0)
    out, M, Z, p = O.attend(q, Kid, V, 0.5)
    assert np.allclose(p, 1 / 9, rtol=1e-14) and abs(Z - 9) < 1e-12
    assert np.allclose(out, V.mean(axis=0), rtol=1e-12, atol=1e-14)
    # two tokens: p0 = 1 / (1 + exp(s1 - s0))
    K2 = np.zeros((2, D)); K2[0, 0] = 1.0; K2[1, 0] = -1.0
    q2 = np.zeros(D); q2[0] = 1.5
    out, M, Z, p = O.attend(q2, K2, V[:2], 1.0)
    assert abs(p[0] - 1 / (1 + math.exp(-3.0))) < 1e-15
    assert np.allclose(out, p[0] * V[0] + p[1] * V[1], rtol=1e-14)
    # a dominant key takes (almost) all the weight
    Kn = K.copy(); Kn[4] = 60.0 * q / np.linalg.norm(q)
    out, M, Z, p = O.attend(q, Kn, V, 1.0)
    assert p.argmax() == 4 and np.allclose(out, V[4], atol=1e-12)
    # empty row set
    out, M, Z, p = O.attend(q, K[:0], V[:0], 1.0)
    assert not out.any() and Z == 0.0 and p.size == 0


# ---------------------------------------------------------------- full-attention group + pooling
def _chunk_reference(qg, K, V, L, scale):
    """Causal chunk attention with torch (library), per head; probabilities too."""
    C, G, D = qg.shape
    pos = np.arange(C) + L - C
    mask = np.where(np.arange(L)[None, :] <= pos[:, None], 0.0, -np.inf)  # [C, L]
    outs = np.zeros((C, G, D))
    probs = np.zeros((C, G, L))
    for h in range(G):
        outs[:, h] = _sdpa(qg[:, h][None], K[:L][None], V[:L][None], scale, mask[None])[0]
        s = torch.from_numpy(qg[:, h]) @ torch.from_numpy(K[:L]).T * scale + torch.from_numpy(mask)
        probs[:, h] = torch.softmax(s, -1).numpy()
    return outs, probs


def pin_full_group(O):
    rng = np.random.default_rng(4)
    for C, G, L, D in [(1, 1, 50, 16), (3, 4, 41, 32), (8, 2, 64, 8), (2, 8, 9, 16), (1, 64, 40, 256)]:
        qg = _f64(_bits(rng, (C, G, D)))
        K = _f64(_bits(rng, (L + 5, D)))
        V = _f64(_bits(rng, (L + 5, D)))
        scale = 1 / math.sqrt(D)
        out, M, Z, P = O.full_attention_group(qg, K, V, L, scale)
        ref_out, ref_p = _chunk_reference(qg, K, V, L, scale)
        assert np.allclose(out, ref_out, rtol=1e-11, atol=1e-13), (C, G, L)
        ref_P = ref_p.sum(axis=1)  # sum of the G heads' probabilities
        assert np.allclose(P, ref_P, rtol=2e-7, atol=1e-30), (C, G, L)
        assert P.dtype == np.float32
        # each query's pooled scores sum to G over its causal range; zero beyond it
        pos = np.arange(C) + L - C
        for c in range(C):
            assert abs(float(P[c].astype(np.float64).sum()) - G) < 1e-5 * G
            assert not P[c, pos[c] + 1:].any()
        # rows beyond L (and beyond each query's position) never matter
        K2, V2 = K.copy(), V.copy()
        K2[L - C + 1:] += 3.0; V2[L - C + 1:] -= 2.0
        o2, _, _, P2 = O.full_attention_group(qg, K2, V2, L, scale)
        assert np.array_equal(o2[0], out[0]) and np.array_equal(P2[0], P[0])
    # G = 1: pooled score is the probability itself, ranked like the logits
    qg = _f64(_bits(rng, (1, 1, 16)))
    K = _f64(_bits(rng, (30, 16)))
    _, _, _, P = O.full_attention_group(qg, K, K, 30, 0.25)
    logits = K @ qg[0, 0]
    assert np.array_equal(np.argsort(-P[0], kind="stable"), np.argsort(-logits, kind="stable"))
    # identical heads: pooled = G x the single-head probability
    q1 = np.repeat(qg, 4, axis=1)
    _, _, _, P4 = O.full_attention_group(q1, K, K, 30, 0.25)
    assert np.allclose(P4[0], 4 * P[0].astype(np.float64), rtol=1e-6)


def pin_head_mapping(O):
    """Query head h reads KV head h // G; KV head g pools heads g*G .. g*G+G-1."""
    rng = np.random.default_rng(5)
    B, C, Hq, Hkv, D, L = 2, 2, 6, 2, 16, 23
    G = Hq // Hkv
    q = _bits(rng, (B, C, Hq, D))
    K = _bits(rng, (B, Hkv, L, D), 1.5)
    V = _bits(rng, (B, Hkv, L, D))
    lens = np.array([L, L - 4])
    res = O.full_attn_score_select(q, K, V, lens, k=4, window=3)
    scale = 1 / math.sqrt(D)
    for b in range(B):
        Lb = int(lens[b])
        for g in range(Hkv):
            qg = _f64(q[b, :, g * G:(g + 1) * G])
            ro, rp = _chunk_reference(qg, _f64(K[b, g]), _f64(V[b, g]), Lb, scale)
            assert np.allclose(res["out"][b, :, g * G:(g + 1) * G], ro, rtol=1e-11, atol=1e-13)
            assert np.allclose(res["P"][b, g, :, :Lb], rp.sum(axis=1), rtol=2e-7)


# ---------------------------------------------------------------- selection
def _brute_force_select(scores, pos, k, window):
    """Enumerate every k-subset of the candidates; keep the largest sum, then
    the lexicographically smallest ascending index tuple."""
    N = max(0, pos - window + 1)
    kk = min(k, N)
    best = None
    for sub in itertools.combinations(range(N), kk):
        key = (-sum(scores[t] for t in sub), sub)
        if best is None or key < best:
            best = key
    chosen = list(best[1]) if best else []
    win = list(range(max(0, pos - window + 1), pos + 1))
    row = sorted(chosen + win)
    return row + [-1] * (k + window - len(row))


def pin_select_bruteforce(O):
    rng = np.random.default_rng(6)
    for _ in range(60):
        n = int(rng.integers(1, 12))
        pos = n - 1
        k = int(rng.integers(0, 6))
        window = int(rng.integers(0, 5))
        if k + window == 0:
            continue
        scores = rng.integers(0, 4, size=n).astype(np.float32) / np.float32(4)  # exact sums, many ties
        got = O.select_row(scores, pos, k, window)
        want = _brute_force_select([float(x) for x in scores], pos, k, window)
        assert list(got) == want, (scores, pos, k, window, got, want)


def pin_select_golden(O):
    with open(os.path.join(GOLDEN, "selection_hand.txt")) as f:
        rows = [ln for ln in f if ln.strip() and not ln.startswith("#")]
    assert len(rows) >= 8
    for ln in rows:
        head, sc, exp = ln.split("|")
        pos, k, window = (int(x) for x in head.split())
        scores = np.array([float(x) for x in sc.split()], dtype=np.float32)
        want = [int(x) for x in exp.split()]
        got = O.select_row(scores, pos, k, window)
        assert list(got) == want, (ln, list(got))


def pin_select_invariants(O):
    rng = np.random.default_rng(7)
    for _ in range(40):
        n = int(rng.integers(1, 400))
        pos = n - 1
        k = int(rng.integers(0, 80))
        window = int(rng.integers(0, 40))
        if k + window == 0:
            continue
        scores = rng.random(n).astype(np.float32)
        row = np.asarray(O.select_row(scores, pos, k, window))
        assert row.size == k + window
        cnt = int((row >= 0).sum())
        assert cnt == min(pos + 1, k + window)
        assert (row[cnt:] == -1).all() and (row[:cnt] >= 0).all()
        sel = row[:cnt]
        assert (np.diff(sel) > 0).all() and sel.max() <= pos
        win = set(range(max(0, pos - window + 1), pos + 1))
        assert win <= set(sel.tolist())
        top = [t for t in sel.tolist() if t not in win]
        rest = [t for t in range(max(0, pos - window + 1)) if t not in set(top)]
        if top and rest:
            assert min(scores[top]) >= max(scores[rest])


# ---------------------------------------------------------------- block-level selection
def _brute_force_select_blocks(scores, pos, k, window, block):
    """Enumerate every (k // block)-subset of the candidate blocks; keep the
    largest sum of block scores, then the lexicographically smallest block
    tuple.  Block scores: numpy's segment sums of the candidates' ranking
    values, rounded to float32."""
    N = max(0, pos - window + 1)
    nb = -(-N // block)
    vals = np.array([0.0 if s < np.finfo(np.float32).tiny else float(s) for s in scores[:N]])
    sums = [float(np.float32(x)) for x in np.add.reduceat(vals, np.arange(0, N, block))] if N else []
    best = None
    for sub in itertools.combinations(range(nb), min(k // block, nb)):
        key = (-sum(sums[j] for j in sub), sub)
        if best is None or key < best:
            best = key
    chosen = [t for j in (best[1] if best else ()) for t in range(j * block, min((j + 1) * block, N))]
    win = list(range(max(0, pos - window + 1), pos + 1))
    row = sorted(chosen + win)
    return row + [-1] * (k + window - len(row))


def pin_select_blocks(O):
    """Block-level selection: brute force, the token rule at block 1, a
    hand-worked fixture and invariants."""
    rng = np.random.default_rng(16)
    for _ in range(80):
        n = int(rng.integers(1, 15))
        pos = n - 1
        block = int(rng.integers(1, 5))
        k = int(rng.integers(0, 9))
        window = int(rng.integers(0, 5))
        if k + window == 0:
            continue
        scores = rng.integers(0, 4, size=n).astype(np.float32) / np.float32(4)  # exact sums, many ties
        got = O.select_row_blocks(scores, pos, k, window, block)
        want = _brute_force_select_blocks([float(x) for x in scores], pos, k, window, block)
        assert list(got) == want, (scores, pos, k, window, block, got, want)
    for _ in range(30):  # blocks of one token: the token-level rule
        n = int(rng.integers(1, 300))
        k, window = int(rng.integers(0, 60)), int(rng.integers(0, 30))
        if k + window == 0:
            continue
        scores = (rng.integers(0, 20, size=n) / 16).astype(np.float32)
        assert np.array_equal(O.select_row_blocks(scores, n - 1, k, window, 1), O.select_row(scores, n - 1, k, window))
    with open(os.path.join(GOLDEN, "selection_blocks_hand.txt")) as f:
        rows = [ln for ln in f if ln.strip() and not ln.startswith("#")]
    assert len(rows) >= 8
    for ln in rows:
        head, sc, exp = ln.split("|")
        pos, k, window, block = (int(x) for x in head.split())
        scores = np.array([float(x) for x in sc.split()], dtype=np.float32)
        got = O.select_row_blocks(scores, pos, k, window, block)
        assert list(got) == [int(x) for x in exp.split()], (ln, list(got))
    for _ in range(40):  # invariants at larger sizes
        n = int(rng.integers(1, 3000))
        pos = n - 1
        block = int(2 ** rng.integers(4, 8))
        k = block * int(rng.integers(0, 12))
        window = int(rng.integers(0, 200))
        if k + window == 0:
            continue
        scores = rng.random(n).astype(np.float32)
        row = np.asarray(O.select_row_blocks(scores, pos, k, window, block))
        N = max(0, pos - window + 1)
        nb = -(-N // block)
        assert row.size == k + window
        cnt = int((row >= 0).sum())
        sel = row[:cnt]
        assert (row[cnt:] == -1).all() and (np.diff(sel) > 0).all() and (sel <= pos).all()
        win = set(range(max(0, pos - window + 1), pos + 1))
        assert win <= set(sel.tolist())
        picked = sorted({t // block for t in sel.tolist() if t < N})
        assert len(picked) == min(k // block, nb)
        for j in picked:  # whole blocks, cut only at N
            assert set(range(j * block, min((j + 1) * block, N))) <= set(sel.tolist())
        assert cnt == sum(min(block, N - j * block) for j in picked) + len(win)
        sums = np.add.reduceat(scores[:N].astype(np.float64), np.arange(0, N, block)) if N else np.zeros(0)
        rest = [j for j in range(nb) if j not in picked]
        if picked and rest:
            assert min(sums[picked]) >= max(sums[rest]) * (1 - 1e-6)


# ---------------------------------------------------------------- sparse attention
def pin_sparse(O):
    rng = np.random.default_rng(8)
    B, C, Hq, Hkv, D, L = 1, 3, 4, 2, 16, 29
    G = Hq // Hkv
    q = _bits(rng, (B, C, Hq, D))
    K = _bits(rng, (B, Hkv, L, D))
    V = _bits(rng, (B, Hkv, L, D))
    lens = np.array([L])
    # budget covering every token: sparse attention == full attention
    full = O.full_attn_score_select(q, K, V, lens, k=L, window=4)
    sa = O.sparse_attention(q, K, V, full["idx"])
    assert np.allclose(sa, full["out"], rtol=1e-13, atol=1e-15)
    # budget short of the cache: differs from full attention, equals attention
    # over exactly the selected rows
    part = O.full_attn_score_select(q, K, V, lens, k=5, window=3)
    sa = O.sparse_attention(q, K, V, part["idx"])
    assert not np.allclose(sa, part["out"], rtol=1e-3)
    scale = 1 / math.sqrt(D)
    for g in range(Hkv):
        for c in range(C):
            sel = part["idx"][0, g, c]
            sel = sel[sel >= 0]
            assert sel.size == 8
            for h in range(G):
                ref = _sdpa(_f64(q[0, c, g * G + h])[None, None], _f64(K[0, g, sel])[None],
                            _f64(V[0, g, sel])[None], scale)[0, 0]
                assert np.allclose(sa[0, c, g * G + h], ref, rtol=1e-12, atol=1e-14)
    # order of the index row and -1 slots do not matter
    perm = part["idx"].copy()
    perm[..., :8] = perm[..., :8][..., ::-1]
    assert np.allclose(O.sparse_attention(q, K, V, perm), sa, rtol=1e-12, atol=1e-14)
    # a single selected token: output is its value row
    one = np.full_like(part["idx"], -1)
    one[..., 0] = 7
    so = O.sparse_attention(q, K, V, one)
    for h in range(Hq):
        assert np.array_equal(so[0, :, h], np.repeat(_f64(V[0, h // G, 7])[None], C, axis=0))


def pin_sparse_sink_gate(O):
    """Sinks and output gates of the sparse layers against torch and closed forms."""
    rng = np.random.default_rng(12)
    B, C, Hq, Hkv, D, L = 1, 2, 4, 2, 16, 23
    G = Hq // Hkv
    q = _bits(rng, (B, C, Hq, D))
    K = _bits(rng, (B, Hkv, L, D))
    V = _bits(rng, (B, Hkv, L, D))
    lens = np.array([L])
    scale = 1 / math.sqrt(D)
    sink = np.array([-1.5, 0.25, 2.0, 0.7])  # a different logit per head
    part = O.full_attn_score_select(q, K, V, lens, k=5, window=3)
    sa = O.sparse_attention(q, K, V, part["idx"], sink=sink)
    for g in range(Hkv):
        for c in range(C):
            sel = part["idx"][0, g, c]
            sel = sel[sel >= 0]
            for h in range(G):
                hq = g * G + h
                # library route: one extra key with zero key and value rows whose
                # additive mask is the sink makes softmax's extra logit the sink
                Ka = np.concatenate([_f64(K[0, g, sel]), np.zeros((1, D))])[None]
                Va = np.concatenate([_f64(V[0, g, sel]), np.zeros((1, D))])[None]
                mask = np.zeros((1, 1, sel.size + 1))
                mask[0, 0, -1] = sink[hq]
                ref = _sdpa(_f64(q[0, c, hq])[None, None], Ka, Va, scale, mask)[0, 0]
                assert np.allclose(sa[0, c, hq], ref, rtol=1e-12, atol=1e-14), (g, c, h)
    # closed form, one selected token t: out = v_t * sigmoid(s_t - sink)
    one = np.full_like(part["idx"], -1)
    one[..., 0] = 5
    so = O.sparse_attention(q, K, V, one, sink=sink)
    for c in range(C):
        for hq in range(Hq):
            s_t = scale * float(_f64(q[0, c, hq]) @ _f64(K[0, hq // G, 5]))
            want = _f64(V[0, hq // G, 5]) / (1.0 + math.exp(sink[hq] - s_t))
            assert np.allclose(so[0, c, hq], want, rtol=1e-13, atol=1e-15)
    # a sink at -inf is no sink; a huge sink takes all the mass
    assert np.allclose(O.sparse_attention(q, K, V, part["idx"], sink=np.full(Hq, -np.inf)),
                       O.sparse_attention(q, K, V, part["idx"]), rtol=1e-14, atol=1e-16)
    assert np.abs(O.sparse_attention(q, K, V, part["idx"], sink=np.full(Hq, 800.0))).max() < 1e-300
    # gates: the ungated output times torch's sigmoid of the gate logits
    gate = _bits(rng, (B, C, Hq, D), 3.0)
    plain = O.sparse_attention(q, K, V, part["idx"], sink=sink)
    gated = O.sparse_attention(q, K, V, part["idx"], sink=sink, gate=gate)
    assert np.allclose(gated, plain * torch.sigmoid(torch.from_numpy(_f64(gate))).numpy(), rtol=1e-14, atol=1e-16)
    zero = np.zeros_like(gate)  # bf16 +0: sigmoid(0) = 1/2
    assert np.array_equal(O.sparse_attention(q, K, V, part["idx"], gate=zero), O.sparse_attention(q, K, V, part["idx"]) / 2)
    # a budget covering every token: sparse attention with a sink equals full
    # attention over the whole causal range with the same sink
    full = O.full_attn_score_select(q, K, V, lens, k=L, window=4)
    sf = O.sparse_attention(q, K, V, full["idx"], sink=sink)
    for c in range(C):
        pos = L - C + c
        for hq in range(Hq):
            g = hq // G
            Ka = np.concatenate([_f64(K[0, g, :pos + 1]), np.zeros((1, D))])[None]
            Va = np.concatenate([_f64(V[0, g, :pos + 1]), np.zeros((1, D))])[None]
            mask = np.zeros((1, 1, pos + 2))
            mask[0, 0, -1] = sink[hq]
            ref = _sdpa(_f64(q[0, c, hq])[None, None], Ka, Va, scale, mask)[0, 0]
            assert np.allclose(sf[0, c, hq], ref, rtol=1e-12, atol=1e-14)


def pin_fp8_cache(O):
    """E4M3 cache: decoding against torch, and the whole layer against the bf16 path and torch."""
    allb = np.arange(256, dtype=np.uint8)
    d = O.e4m3_to_f64(allb)
    ref = torch.from_numpy(allb).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(np.isnan(d), np.isnan(ref)) and np.array_equal(d[~np.isnan(d)], ref[~np.isnan(ref)])
    spot = {0x38: 1.0, 0x7E: 448.0, 0x01: 2.0 ** -9, 0x08: 2.0 ** -6, 0xB8: -1.0, 0x3C: 1.5, 0x47: 3.75}
    for bt, v in spot.items():
        assert O.e4m3_to_f64(np.array([bt], dtype=np.uint8))[0] == v, hex(bt)
    assert np.isnan(O.e4m3_to_f64(np.array([0x7F, 0xFF], dtype=np.uint8))).all()
    rng = np.random.default_rng(14)
    B, C, Hq, Hkv, D, L = 1, 2, 4, 2, 16, 37
    G = Hq // Hkv
    q = _bits(rng, (B, C, Hq, D))
    finite = np.array([b for b in range(256) if b not in (0x7F, 0xFF)], dtype=np.uint8)
    K8 = rng.choice(finite, size=(B, Hkv, L, D))
    V8 = rng.choice(finite, size=(B, Hkv, L, D))
    lens = np.array([L])
    # power-of-two scales: every cache value is a bf16 value too, so the E4M3
    # cache and the bf16 cache holding the same numbers give identical results
    ks, vs = np.array([2.0 ** -6, 2.0 ** -5]), np.array([2.0 ** -4, 2.0 ** -7])
    Kf = O.e4m3_to_f64(K8) * ks[None, :, None, None]
    Vf = O.e4m3_to_f64(V8) * vs[None, :, None, None]
    Kb = f32_to_bf16_bits(Kf.astype(np.float32))
    Vb = f32_to_bf16_bits(Vf.astype(np.float32))
    assert np.array_equal(_f64(Kb), Kf) and np.array_equal(_f64(Vb), Vf)
    r8 = O.hybrid_block(q, [q], K8, V8, lens, 6, 4, k_scale=ks, v_scale=vs)
    rb = O.hybrid_block(q, [q], Kb, Vb, lens, 6, 4)
    for key in ("out", "M", "Z", "P", "idx"):
        assert np.array_equal(r8[key], rb[key]), key
    assert np.array_equal(r8["sa_out"][0], rb["sa_out"][0])
    # arbitrary per-head scales, different for K and V: torch attention on the
    # dequantised cache
    ks, vs = np.array([0.0123, 0.031]), np.array([0.27, 0.0052])
    res = O.full_attn_score_select(q, K8, V8, lens, 6, 4, k_scale=ks, v_scale=vs)
    scale = 1 / math.sqrt(D)
    for c in range(C):
        pos = L - C + c
        for hq in range(Hq):
            g = hq // G
            Kd = (O.e4m3_to_f64(K8[0, g, :pos + 1]) * ks[g])[None]
            Vd = (O.e4m3_to_f64(V8[0, g, :pos + 1]) * vs[g])[None]
            want = _sdpa(_f64(q[0, c, hq])[None, None], Kd, Vd, scale)[0, 0]
            assert np.allclose(res["out"][0, c, hq], want, rtol=1e-12, atol=1e-15), (c, hq)


def pin_needles(O):
    """Planted keys aligned with a group's queries must all be selected."""
    w = Workload("needle_pin", 2, 700, 1, 8, 2, 32, 24, 16, 1, ctx_min=500, needles=6)
    inp = make_inputs(w, seed=11)
    res = O.full_attn_score_select(inp.q_fa, inp.K, inp.V, inp.lens, w.k, w.window)
    for b in range(w.batch):
        for g in range(w.n_kv_heads):
            sel = set(res["idx"][b, g, 0].tolist())
            assert set(inp.needles[b].tolist()) <= sel, (b, g)


ALL_PINS = [pin_bf16_decode, pin_attend_vs_library, pin_attend_special_cases, pin_full_group,
            pin_head_mapping, pin_select_bruteforce, pin_select_golden, pin_select_invariants,
            pin_select_blocks, pin_sparse, pin_sparse_sink_gate, pin_fp8_cache, pin_needles]
