"""Plain CPU oracle for the decode-time attention of one HySparse2 hybrid block.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the test suite, the smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code with the HIP path; inputs reach it
as raw bf16 bit patterns from the seeded generators and it decodes them itself.

What is computed (HySparse2, Sec. "Cross-Layer KV Reuse" and "The Role of Full
Attention"; model setup in Sec. "Experimental Setup"):

  1. full attention of each decode query over the whole KV cache of its
     sequence (NoPE, so no positional transform of q or k);
  2. token importance scores taken from that layer's exact softmax
     probabilities, pooled over the query heads that share one KV head;
  3. per query, the most recent ``window`` tokens are always selected, and
     the ``k`` highest-scoring tokens *outside* that window are added;
  4. each following sparse-attention layer attends, with its own query, only
     over the selected tokens of the same KV cache (KV Reuse).

Arithmetic is float64 throughout; bf16 inputs are decoded exactly.  Attention
outputs are returned in float64.  Pooled scores are rounded once to float32:
the selection ranks those float32 values, descending, with the lower token
index first among equal values.

Readings taken where the paper is silent (each is listed in the design doc):
  * pooling = sum over the G query heads of a KV head of their softmax
    probabilities (each head normalised over its own causal range);
  * top-k is drawn only from tokens outside the forced window, so window and
    top-k are disjoint and |selection| = min(pos + 1, k + window);
  * the cache holds tokens [0, L) including the decode token(s); query c of a
    C-token chunk sits at pos = L - C + c and sees tokens [0, pos];
  * the window of query c is [max(0, pos - window + 1), pos];
  * softmax scale 1/sqrt(head_dim) unless given;
  * pooled scores below FLT_MIN count as +0 when ranking;
  * index rows are ascending and padded with -1 to k + window slots;
  * sparse layers use a plain renormalised softmax over the selected tokens
    (no sink term);
  * block-level selection (the comparison granularity): a block's score is
    the sum of its candidate tokens' pooled scores; the k / block best
    blocks before the window are taken, the last one cut short by it.

Every function here is pinned in tests/test_oracle_pins.py against closed
forms, a library attention routine, brute-force subset enumeration and
invariants of the method.
"""
from __future__ import annotations

import numpy as np

FLT_MIN = np.float32(np.finfo(np.float32).tiny)


# --------------------------------------------------------------------------
# input decoding
# --------------------------------------------------------------------------
def e4m3_to_f64(bits: np.ndarray) -> np.ndarray:
    """Decode OCP FP8 E4M3 bits: sign, 4 exponent bits (bias 7), 3 mantissa
    bits; exponent 0 holds the subnormals m/8 * 2^-6; exponent 15 with
    mantissa 7 is NaN (the format has no infinities)."""
    b = np.asarray(bits, dtype=np.uint8).astype(np.int64)
    sign = np.where(b >> 7, -1.0, 1.0)
    e = (b >> 3) & 15
    m = (b & 7).astype(np.float64)
    mag = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    return np.where((e == 15) & (m == 7), np.nan, sign * mag)


def cache_rows(X: np.ndarray, b: int, g: int, rows, scale) -> np.ndarray:
    """Rows of one (sequence, KV head) of a cache as float64: bf16 bits, or
    E4M3 bits times that KV head's scale (the paper quotes its costs with an
    FP8 KV cache, Sec. "Prefill computation and KV-cache storage")."""
    if X.dtype == np.uint8:
        return e4m3_to_f64(X[b, g, rows]) * float(scale[g])
    return bf16_to_f64(X[b, g, rows])


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns (uint16) as float64.

    A bf16 number is the upper half of an IEEE binary32 word, so shifting the
    16 bits into the top of a 32-bit word gives the same value exactly.
    """
    bits = np.asarray(bits)
    if bits.dtype != np.uint16:
        raise TypeError("bf16 inputs are passed as uint16 bit patterns")
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def query_positions(L: int, C: int) -> np.ndarray:
    """Cache positions of the C queries of a decode chunk over a cache of L tokens.

    The cache already holds the chunk's own tokens (reading of the speculative
    verification setting, Sec. "Inference Architecture"): query c sits at
    L - C + c and attends causally to [0, L - C + c].
    """
    return np.arange(C, dtype=np.int64) + (int(L) - int(C))


def default_scale(D: int) -> float:
    return 1.0 / np.sqrt(float(D))


# --------------------------------------------------------------------------
# softmax attention of one query head over a set of cached tokens
# --------------------------------------------------------------------------
def attend(q: np.ndarray, Krows: np.ndarray, Vrows: np.ndarray, scale: float):
    """Exact softmax attention of one query over the given K/V rows.

    Full-attention and sparse-attention layers both compute this (NoPE, Sec.
    "Experimental Setup"); a sparse layer merely restricts the rows to the
    selected tokens (Sec. "Cross-Layer KV Reuse").

    Returns (out[D], M, Z, p[n]) with logits s = scale * <q, k_t>,
    M = max_t s_t, Z = sum_t exp(s_t - M), p_t = exp(s_t - M) / Z and
    out = sum_t p_t v_t.  An empty row set returns out = 0, M = -inf, Z = 0.
    """
    n = Krows.shape[0]
    if n == 0:
        return np.zeros(Vrows.shape[1]), -np.inf, 0.0, np.zeros(0)
    s = scale * (Krows @ q)
    M = s.max()
    e = np.exp(s - M)
    Z = e.sum()
    p = e / Z
    out = p @ Vrows
    return out, M, Z, p


# --------------------------------------------------------------------------
# full-attention layer of one (sequence, KV head) group, with pooled scores
# --------------------------------------------------------------------------
def full_attention_group(qg: np.ndarray, Kg: np.ndarray, Vg: np.ndarray, L: int, scale: float):
    """Full attention + pooled token scores for one sequence and one KV head.

    qg: float64 [C, G, D] -- the G query heads sharing this KV head, for each
        of the C chunk queries; Kg, Vg: float64 [>=L, D] cache rows.

    Full attention (Sec. "HySparse2 Overview": FA layers attend over the whole
    cache) gives per head out/M/Z.  Its exact probabilities double as token
    scores (Sec. "The Role of Full Attention"): the pooled score of token t for
    query c is the sum over the G heads of that head's probability of t.
    Tokens beyond the query's causal position get probability 0.

    Returns out [C, G, D] float64, M [C, G], Z [C, G], P [C, L] float32.
    """
    C, G, D = qg.shape
    pos = query_positions(L, C)
    out = np.zeros((C, G, D))
    M = np.full((C, G), -np.inf)
    Z = np.zeros((C, G))
    P = np.zeros((C, L), dtype=np.float32)
    for c in range(C):
        n = int(pos[c]) + 1
        if n <= 0:
            continue
        pooled = np.zeros(n)
        for h in range(G):
            o, m, z, p = attend(qg[c, h], Kg[:n], Vg[:n], scale)
            out[c, h], M[c, h], Z[c, h] = o, m, z
            pooled += p
        P[c, :n] = pooled.astype(np.float32)
    return out, M, Z, P


# --------------------------------------------------------------------------
# selection: forced window + top-k outside it
# --------------------------------------------------------------------------
def rank_key(P: np.ndarray) -> np.ndarray:
    """Ranking value of float32 pooled scores: values below FLT_MIN count as +0."""
    P = np.asarray(P, dtype=np.float32)
    return np.where(P < FLT_MIN, np.float32(0.0), P)


def topk_outside_window(P_row: np.ndarray, pos: int, k: int, window: int) -> np.ndarray:
    """Top-k token indices among the candidates outside the forced window.

    Candidates are tokens [0, pos - window] (Sec. "Cross-Layer KV Reuse": the
    highest-scoring tokens outside the recent window are taken after it).
    Order: pooled float32 score descending, then token index ascending.
    Returns the chosen indices in rank order.
    """
    N = max(0, int(pos) - int(window) + 1)
    if N == 0 or k <= 0:
        return np.zeros(0, dtype=np.int64)
    key = rank_key(P_row[:N]).astype(np.float64)
    t = np.arange(N)
    order = np.lexsort((t, -key))  # last key is primary: -score, then index
    return order[: min(int(k), N)].astype(np.int64)


def forced_window(pos: int, window: int) -> np.ndarray:
    """The most recent ``window`` tokens up to and including ``pos``."""
    lo = max(0, int(pos) - int(window) + 1)
    return np.arange(lo, int(pos) + 1, dtype=np.int64)


def select_row(P_row: np.ndarray, pos: int, k: int, window: int) -> np.ndarray:
    """Selection index row: window union top-k, ascending, -1 padded to k + window."""
    S = int(k) + int(window)
    sel = np.concatenate([topk_outside_window(P_row, pos, k, window), forced_window(pos, window)]) if pos >= 0 \
        else np.zeros(0, dtype=np.int64)
    sel = np.sort(sel)
    row = np.full(S, -1, dtype=np.int32)
    row[: sel.size] = sel
    return row


# --------------------------------------------------------------------------
# block-level selection: the granularity of the predecessor HySparse, which
# the paper compares against (Sec. "Ablation 1: Token-Level versus
# Block-Level Sparsity": blocks of 64 tokens, the same 1,024-token global
# budget, the same local window).  How a block is scored is not restated
# there; reading: a block's score is its share of the attention mass, the
# sum of the pooled scores of its candidate tokens.
# --------------------------------------------------------------------------
def block_scores(P_row: np.ndarray, N: int, block: int) -> np.ndarray:
    """float32 score of each block [j*block, (j+1)*block) clipped to the N
    candidates: the float64 sum of its tokens' ranking values, rounded once."""
    nb = -(-int(N) // int(block))
    vals = rank_key(P_row[:N]).astype(np.float64)
    out = np.zeros(nb, dtype=np.float32)
    for j in range(nb):
        out[j] = np.float32(vals[j * block: min((j + 1) * block, N)].sum())
    return out


def topk_blocks_outside_window(P_row: np.ndarray, pos: int, k: int, window: int, block: int) -> np.ndarray:
    """The k / block best candidate blocks (score descending, then block index
    ascending), in rank order.  Candidates are the tokens before the window;
    the last block may be cut short by the window."""
    N = max(0, int(pos) - int(window) + 1)
    kb = int(k) // int(block)
    if N == 0 or kb <= 0:
        return np.zeros(0, dtype=np.int64)
    key = rank_key(block_scores(P_row, N, block)).astype(np.float64)
    j = np.arange(key.size)
    order = np.lexsort((j, -key))
    return order[: min(kb, key.size)].astype(np.int64)


def select_row_blocks(P_row: np.ndarray, pos: int, k: int, window: int, block: int) -> np.ndarray:
    """Block-level selection row: the tokens (before the window) of the best
    k / block blocks, union the window; ascending, -1 padded to k + window."""
    S = int(k) + int(window)
    if pos < 0:
        return np.full(S, -1, dtype=np.int32)
    N = max(0, int(pos) - int(window) + 1)
    parts = [np.arange(j * block, min((j + 1) * block, N), dtype=np.int64)
             for j in topk_blocks_outside_window(P_row, pos, k, window, block)]
    sel = np.sort(np.concatenate(parts + [forced_window(pos, window)]))
    row = np.full(S, -1, dtype=np.int32)
    row[: sel.size] = sel
    return row


# --------------------------------------------------------------------------
# whole-batch steps
# --------------------------------------------------------------------------
def _group_q(q: np.ndarray, b: int, g: int, G: int) -> np.ndarray:
    """float64 [C, G, D] slice of the queries of KV head g (heads g*G .. g*G+G-1)."""
    return bf16_to_f64(q[b, :, g * G:(g + 1) * G, :])


def full_attn_score_select(q, K, V, lens, k, window, scale=None, groups=None, k_scale=None, v_scale=None,
                           block=None):
    """Full-attention layer, pooled scores and selection for a whole batch.
    ``block``: block-level selection with blocks of that many tokens (k a
    multiple of it) instead of token-level.

    q: uint16 [B, C, Hq, D]; K, V: uint16 bf16 bits [B, Hkv, Lmax, D], or
    uint8 E4M3 bits with float [Hkv] scales k_scale / v_scale; lens: int [B].
    ``groups`` optionally restricts the work to a list of (b, g) pairs; other
    entries of the results are left at zero / -1.

    Returns dict with out [B, C, Hq, D] float64, M, Z [B, C, Hq] float64,
    P [B, Hkv, C, Lmax] float32 (candidates and window alike, zero beyond the
    causal range) and idx [B, Hkv, C, k + window] int32.
    """
    B, C, Hq, D = q.shape
    Hkv, Lmax = K.shape[1], K.shape[2]
    if Hq % Hkv:
        raise ValueError("query heads must be a multiple of KV heads")
    G = Hq // Hkv
    scale = default_scale(D) if scale is None else float(scale)
    out = np.zeros((B, C, Hq, D))
    M = np.full((B, C, Hq), -np.inf)
    Z = np.zeros((B, C, Hq))
    P = np.zeros((B, Hkv, C, Lmax), dtype=np.float32)
    idx = np.full((B, Hkv, C, int(k) + int(window)), -1, dtype=np.int32)
    todo = groups if groups is not None else [(b, g) for b in range(B) for g in range(Hkv)]
    for b, g in todo:
        L = int(lens[b])
        Kg = cache_rows(K, b, g, slice(0, L), k_scale)
        Vg = cache_rows(V, b, g, slice(0, L), v_scale)
        o, m, z, p = full_attention_group(_group_q(q, b, g, G), Kg, Vg, L, scale)
        out[b, :, g * G:(g + 1) * G] = o
        M[b, :, g * G:(g + 1) * G] = m
        Z[b, :, g * G:(g + 1) * G] = z
        P[b, g, :, :L] = p
        pos = query_positions(L, C)
        for c in range(C):
            if block:
                idx[b, g, c] = select_row_blocks(P[b, g, c], int(pos[c]), k, window, block)
            else:
                idx[b, g, c] = select_row(P[b, g, c], int(pos[c]), k, window)
    return {"out": out, "M": M, "Z": Z, "P": P, "idx": idx}


def attend_with_sink(q: np.ndarray, Krows: np.ndarray, Vrows: np.ndarray, scale: float, sink: float):
    """Softmax attention whose normaliser also holds a per-head sink logit.

    Sec. "Experimental Setup": the sparse layers carry learnable per-head sink
    biases (the cited gpt-oss design): one extra logit `sink`, in the units of
    the scaled logits s_t = scale * <q, k_t>, joins the softmax normaliser and
    contributes no value row:
        out = sum_t exp(s_t - M) v_t / (exp(sink - M) + sum_t exp(s_t - M)),
    M = max(sink, max_t s_t).  With no rows the output is 0.
    """
    n = Krows.shape[0]
    if n == 0:
        return np.zeros(Vrows.shape[1])
    s = scale * (Krows @ q)
    M = max(float(s.max()), float(sink))
    e = np.exp(s - M)
    return (e @ Vrows) / (np.exp(sink - M) + e.sum())


def sigmoid(x):
    """Logistic function 1 / (1 + exp(-x)), evaluated without overflow."""
    x = np.asarray(x, dtype=np.float64)
    ex = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + ex), ex / (1.0 + ex))


def sparse_attention(q, K, V, idx, scale=None, groups=None, sink=None, gate=None, k_scale=None, v_scale=None):
    """Sparse-attention layer reusing the full-attention layer's cache and indices.

    Sec. "Cross-Layer KV Reuse": the sparse layer reads the KV entries of the
    selected tokens from the full-attention layer's cache, and every query head
    of KV head g uses the selection of (b, g, c).  Slots holding -1 are unused.
    The selected tokens are visited in the order the index row lists them.

    Optional parts of the paper's sparse layers (Sec. "Experimental Setup"):
    sink: float [Hq], per-head sink logits (see attend_with_sink);
    gate: uint16 bf16 bits [B, C, Hq, D], output gate logits: the layer
    output is multiplied elementwise by sigmoid(gate) (the cited
    gated-attention design; the gate logits come from a trained projection
    of the layer input, so they are an input here).

    q: uint16 [B, C, Hq, D]; idx: int32 [B, Hkv, C, S]; K, V and their scales
    as for full_attn_score_select.  Returns float64 out.
    """
    B, C, Hq, D = q.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    scale = default_scale(D) if scale is None else float(scale)
    out = np.zeros((B, C, Hq, D))
    todo = groups if groups is not None else [(b, g) for b in range(B) for g in range(Hkv)]
    for b, g in todo:
        qg = _group_q(q, b, g, G)
        for c in range(C):
            sel = idx[b, g, c]
            sel = sel[sel >= 0].astype(np.int64)
            Ks = cache_rows(K, b, g, sel, k_scale)
            Vs = cache_rows(V, b, g, sel, v_scale)
            for h in range(G):
                hq = g * G + h
                if sink is None:
                    out[b, c, hq] = attend(qg[c, h], Ks, Vs, scale)[0]
                else:
                    out[b, c, hq] = attend_with_sink(qg[c, h], Ks, Vs, scale, float(sink[hq]))
                if gate is not None:
                    out[b, c, hq] *= sigmoid(bf16_to_f64(gate[b, c, hq]))
    return out


def hybrid_block(q_fa, q_sa, K, V, lens, k, window, scale=None, groups=None, k_scale=None, v_scale=None):
    """One hybrid block: a full-attention layer then len(q_sa) sparse layers.

    Sec. "HySparse2 Overview" / "Cross-Layer KV Reuse": the sparse layers that
    follow the full-attention layer reuse its KV cache and its selection.
    Returns the full-attention result dict with an extra key "sa_out", the
    list of sparse-layer outputs.
    """
    res = full_attn_score_select(q_fa, K, V, lens, k, window, scale, groups, k_scale, v_scale)
    res["sa_out"] = [sparse_attention(qs, K, V, res["idx"], scale, groups, k_scale=k_scale, v_scale=v_scale)
                     for qs in q_sa]
    return res
