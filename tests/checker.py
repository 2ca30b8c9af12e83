"""Comparison of GPU results with the oracle's, to the parity bar of the path.

* attention outputs (bf16 on the GPU, float64 in the oracle): elementwise
  |gpu - ref| <= 2e-2 + 1e-2 |ref|, and per (sequence, query, head) row a
  normwise relative error ||gpu - ref|| / ||ref|| <= 1e-2.  The normwise guard
  matters: with N(0, 1) data the outputs are O(1/sqrt(L)) small, so the
  elementwise bound alone would accept an all-zero output.
* index rows: the valid prefix must be strictly ascending, followed by -1, and
  the counts equal; the sets may differ only by swaps of candidates whose
  oracle float32 scores differ by less than 1e-6 relative.
* pooled scores: |gpu - ref| <= SCORE_RTOL * ref + SCORE_ATOL (the bound
  covers fp32 logits from exact bf16 products, one rounding each for the
  scaled logit, the row factor and a G-term fp32 sum).
* index rows without an oracle (check_idx_structure): for query position pos
  the row holds min(pos + 1, k + window) tokens, strictly ascending, all in
  [0, pos], the whole window [max(0, pos - window + 1), pos] among them and
  -1 after them; this needs no scores, so it runs on every row of a
  full-size result.
"""
from __future__ import annotations

import numpy as np

OUT_ATOL = 2e-2
OUT_RTOL = 1e-2
OUT_NORMWISE = 1e-2
TIE_RTOL = 1e-6
SCORE_RTOL = 2e-5
SCORE_ATOL = 1e-12


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits).astype(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def check_out(gpu: np.ndarray, ref: np.ndarray, what: str = "out", rows=None) -> dict:
    """gpu, ref: float arrays [..., D]; rows: optional boolean mask over [...]."""
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if rows is not None:
        gpu, ref = gpu[rows], ref[rows]
    d = np.abs(gpu - ref)
    bad = d > OUT_ATOL + OUT_RTOL * np.abs(ref)
    assert not bad.any(), f"{what}: {int(bad.sum())} elements outside 2e-2 + 1e-2|ref| (max diff {d.max():.3g})"
    nr = np.linalg.norm(ref, axis=-1)
    nd = np.linalg.norm(gpu - ref, axis=-1)
    zero = nr == 0
    assert not (nd[zero] > 0).any(), f"{what}: nonzero output where the reference is zero"
    rel = nd[~zero] / nr[~zero]
    worst = float(rel.max()) if rel.size else 0.0
    assert worst <= OUT_NORMWISE, f"{what}: normwise relative error {worst:.3g} > {OUT_NORMWISE}"
    return {"max_abs": float(d.max()) if d.size else 0.0, "max_normwise": worst}


def check_idx_row(gpu_row, ref_row, ref_scores, window_lo: int) -> int:
    """Check one selection row; returns the number of tolerated swaps."""
    gpu_row = np.asarray(gpu_row)
    ref_row = np.asarray(ref_row)
    n_ref = int((ref_row >= 0).sum())
    n_gpu = int((gpu_row >= 0).sum())
    assert (gpu_row[n_gpu:] == -1).all(), "gpu row: -1 padding not contiguous"
    assert n_gpu == n_ref, f"gpu selects {n_gpu} tokens, oracle {n_ref}"
    g = gpu_row[:n_gpu].astype(np.int64)
    assert (g >= 0).all() and (np.diff(g) > 0).all(), "gpu row not strictly ascending"
    gs, rs = set(g.tolist()), set(ref_row[:n_ref].tolist())
    only_g, only_r = sorted(gs - rs), sorted(rs - gs)
    assert len(only_g) == len(only_r)
    if not only_g:
        return 0
    assert all(t < window_lo for t in only_g + only_r), "a window token differs"
    pg = ref_scores[only_g].astype(np.float64)
    pr = ref_scores[only_r].astype(np.float64)
    gap = np.abs(pr[:, None] - pg[None, :]) / np.maximum(np.maximum(pr[:, None], pg[None, :]), 1e-300)
    assert gap.max() < TIE_RTOL, f"swap of tokens whose oracle scores differ by {gap.max():.3g} relative"
    return len(only_g)


def check_idx_structure(gpu_idx, lens, C: int, k: int, window: int) -> dict:
    """Oracle-free checks of every selection row of gpu_idx [B, Hkv, C, S]
    (S = k + window): count, order, range, window membership, padding.
    A query at a negative position (len < C) must have an all -1 row."""
    gpu_idx = np.asarray(gpu_idx)
    B, Hkv, Cq, S = gpu_idx.shape
    assert Cq == C and S == k + window, f"idx shape {gpu_idx.shape} for C={C}, k + window={k + window}"
    rows = 0
    for b in range(B):
        L = int(lens[b])
        for c in range(C):
            pos = L - C + c
            want = 0 if pos < 0 else min(pos + 1, k + window)
            wlo = max(0, pos - window + 1)
            for g in range(Hkv):
                r = gpu_idx[b, g, c].astype(np.int64)
                n = int((r >= 0).sum())
                where = f"(b={b}, g={g}, c={c}, pos={pos})"
                assert n == want, f"row {where}: {n} tokens, expected min(pos + 1, k + window) = {want}"
                assert (r[n:] == -1).all(), f"row {where}: -1 padding not contiguous or other negative values"
                v = r[:n]
                if n == 0:
                    continue
                assert (np.diff(v) > 0).all(), f"row {where}: not strictly ascending"
                assert v[0] >= 0 and v[-1] <= pos, f"row {where}: index outside [0, pos]"
                nwin = pos - wlo + 1
                assert n >= nwin and np.array_equal(v[n - nwin:], np.arange(wlo, pos + 1)), \
                    f"row {where}: window [{wlo}, {pos}] not all selected"
                rows += 1
    return {"rows_checked": rows}


def check_idx(gpu_idx, ref_idx, ref_P, lens, C: int, window: int, groups=None) -> dict:
    """gpu_idx, ref_idx [B, Hkv, C, S]; ref_P [B, Hkv, C, Lmax] float32."""
    B, Hkv = ref_idx.shape[:2]
    todo = groups if groups is not None else [(b, g) for b in range(B) for g in range(Hkv)]
    swaps = 0
    for b, g in todo:
        L = int(lens[b])
        for c in range(C):
            pos = L - C + c
            swaps += check_idx_row(gpu_idx[b, g, c], ref_idx[b, g, c], ref_P[b, g, c], max(0, pos - window + 1))
    return {"swaps": swaps}


def check_scores(gpu_P, ref_P, lens, C: int, window: int, groups=None) -> dict:
    """Candidate scores [0, N) of every row; returns the worst relative error."""
    B, Hkv = ref_P.shape[:2]
    todo = groups if groups is not None else [(b, g) for b in range(B) for g in range(Hkv)]
    worst = 0.0
    for b, g in todo:
        L = int(lens[b])
        for c in range(C):
            N = max(0, L - C + c - window + 1)
            if N == 0:
                continue
            r = ref_P[b, g, c, :N].astype(np.float64)
            x = gpu_P[b, g, c, :N].astype(np.float64)
            err = np.abs(x - r)
            bad = err > SCORE_RTOL * r + SCORE_ATOL
            assert not bad.any(), f"scores (b={b}, g={g}, c={c}): {int(bad.sum())} outside tolerance, " \
                                  f"max rel {float((err / np.maximum(r, 1e-30)).max()):.3g}"
            worst = max(worst, float((err / np.maximum(r, 1e-30)).max()))
    return {"score_max_rel": worst}


def boundary_gap(ref_P_row, pos: int, k: int, window: int) -> float:
    """Relative gap between the k-th and (k+1)-th candidate scores (diagnostic)."""
    N = max(0, pos - window + 1)
    if N <= k or k == 0:
        return float("inf")
    s = np.sort(ref_P_row[:N].astype(np.float64))[::-1]
    return float((s[k - 1] - s[k]) / max(s[k - 1], 1e-300))


# block-level selection: the GPU sums a block's fp32 scores in its own order
# from its own scores (each within ~2e-7 of the oracle's): up to 256 terms
BLOCK_TIE_RTOL = 1e-5


def check_block_idx(gpu_idx, ref_idx, ref_P, lens, C: int, window: int, block: int) -> dict:
    """Block-level selection rows [B, Hkv, C, S]: the window part exact, the
    selected blocks whole (cut only at the window) and equal to the oracle's
    except swaps of blocks whose oracle block scores differ by less than
    BLOCK_TIE_RTOL relative."""
    B, Hkv = ref_idx.shape[:2]
    swaps = 0
    for b in range(B):
        L = int(lens[b])
        for g in range(Hkv):
            for c in range(C):
                pos = L - C + c
                N = max(0, pos - window + 1)
                gr, rr = np.asarray(gpu_idx[b, g, c]), np.asarray(ref_idx[b, g, c])
                ng, nr = int((gr >= 0).sum()), int((rr >= 0).sum())
                assert (gr[ng:] == -1).all(), "gpu row: -1 padding not contiguous"
                gs, rs = gr[:ng].astype(np.int64), rr[:nr].astype(np.int64)
                assert (np.diff(gs) > 0).all(), "gpu row not strictly ascending"
                assert np.array_equal(gs[gs >= N], rs[rs >= N]), "window part differs"
                gb = sorted(set((gs[gs < N] // block).tolist()))
                rb = sorted(set((rs[rs < N] // block).tolist()))
                assert len(gb) == len(rb), f"gpu selects {len(gb)} blocks, oracle {len(rb)}"
                whole = [np.arange(j * block, min((j + 1) * block, N)) for j in gb]
                assert np.array_equal(gs[gs < N], np.concatenate(whole) if whole else gs[:0]), "partial block"
                only_g, only_r = sorted(set(gb) - set(rb)), sorted(set(rb) - set(gb))
                if not only_g:
                    continue
                P = np.asarray(ref_P[b, g, c, :N], dtype=np.float32)
                P = np.where(P < np.finfo(np.float32).tiny, 0.0, P.astype(np.float64))
                sums = np.add.reduceat(P, np.arange(0, N, block))
                pg, pr = sums[only_g], sums[only_r]
                gap = np.abs(pr[:, None] - pg[None, :]) / np.maximum(np.maximum(pr[:, None], pg[None, :]), 1e-300)
                assert gap.max() < BLOCK_TIE_RTOL, f"swap of blocks whose oracle scores differ by {gap.max():.3g}"
                swaps += len(only_g)
    return {"block_swaps": swaps}
