"""Seeded synthetic inputs for the hybrid-block decode path.

This module holds no arithmetic of the method: it only draws numbers and
rounds them to bf16 bit patterns.  Both the HIP path and the CPU oracle take
their inputs from here, as raw uint16 bf16 bits, so both see identical values.

Shapes follow the decode workloads of a long-context agentic model (the paper
measures on long-context retrieval and agentic suites; none of their data is
used -- these tensors stand in for them):

  q     [B, C, Hq, D]      one query per decode token (C > 1: a verify chunk)
  K, V  [B, Hkv, Lmax, D]  the full-attention layer's cache, shared by the
                           sparse layers of the block
  lens  [B]                tokens in each sequence's cache (incl. the chunk)

Values are N(0, 1) float32 rounded to bf16 (round to nearest even).  Every
tensor chunk has its own stream, seeded by (base seed, tensor id, layer,
sequence, KV head), so a single (sequence, KV head) slice can be regenerated
without drawing the rest.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace
import os
import numpy as np

BASE_SEED = 2609

# tensor ids for the seed sequence
_T_Q_FA, _T_Q_SA, _T_K, _T_V, _T_LEN, _T_NEEDLE = 1, 2, 3, 4, 5, 6


@dataclass(frozen=True)
class Workload:
    """Shape of one decode step of a hybrid block (1 full + n_sparse layers)."""
    name: str
    batch: int
    ctx: int                      # context length (upper bound when ragged)
    n_queries: int                # C: decode tokens per sequence
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    k: int                        # top-k budget outside the window
    window: int                   # forced recent window
    n_sparse: int                 # sparse layers following the full layer
    ctx_min: int = 0              # > 0: ragged lengths drawn from [ctx_min, ctx]
    needles: int = 0              # planted high-similarity keys per sequence
    extra: dict = field(default_factory=dict)

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def slots(self) -> int:
        return self.k + self.window


WORKLOADS = {
    # small single decode step, one sparse layer
    "decode_4k_16q2kv": Workload("decode_4k_16q2kv", 1, 4096, 1, 16, 2, 128, 256, 64, 1),
    # 1 full + 3 sparse layers at 32K
    "block_32k_32q4kv": Workload("block_32k_32q4kv", 1, 32768, 1, 32, 4, 128, 2048, 128, 3),
    # batch 8, ragged 16K..128K contexts, 16 planted needles per sequence
    "ragged_16k_128k_b8_needles": Workload("ragged_16k_128k_b8_needles", 8, 131072, 1, 32, 4, 128, 2048, 128, 3,
                                           ctx_min=16384, needles=16),
    # 8-query verify chunk per sequence at 128K, batch 4
    "chunk8_128k_b4": Workload("chunk8_128k_b4", 4, 131072, 8, 32, 4, 128, 4096, 256, 3),
    # long-context stress at 512K, batch 2, 64 query / 8 KV heads
    "stress_512k_b2_64q8kv": Workload("stress_512k_b2_64q8kv", 2, 524288, 1, 64, 8, 128, 8192, 512, 3),
    # the paper's own head layout at 128K, batch 8: MQA with 64 query heads on
    # one KV head and head dim 256 (Sec. "Experimental Setup", table of the
    # attention configurations), 1024 global + 128 local tokens (same section)
    "paper_mqa64_d256_128k_b8": Workload("paper_mqa64_d256_128k_b8", 8, 131072, 1, 64, 1, 256, 1024, 128, 3),
    # the same with a 2-token verify chunk per sequence (128 query rows on the KV head), batch 4
    "paper_mqa64_d256_128k_b4_chunk2": Workload("paper_mqa64_d256_128k_b4_chunk2", 4, 131072, 2, 64, 1, 256, 1024, 128,
                                                3),
}


def shrink(w: Workload, ctx: int, ctx_min: int | None = None, k: int | None = None, window: int | None = None,
           batch: int | None = None, name: str | None = None) -> Workload:
    """Same head layout at a smaller context (for oracle-speed parity cases)."""
    return replace(w, name=name or f"{w.name}@{ctx}", ctx=ctx,
                   ctx_min=(ctx_min if ctx_min is not None else (min(w.ctx_min, ctx) if w.ctx_min else 0)),
                   k=w.k if k is None else k, window=w.window if window is None else window,
                   batch=w.batch if batch is None else batch)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rnd = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + rnd) >> 16).astype(np.uint16)


E4M3_MAX = 448.0  # largest finite OCP FP8 E4M3 value


def f32_to_e4m3_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to OCP FP8 E4M3 (nearest, ties to even), saturating
    at +-448; returns uint8 bits.  (torch's cast does the rounding.)"""
    import torch
    t = torch.from_numpy(np.clip(np.ascontiguousarray(x, dtype=np.float32), -E4M3_MAX, E4M3_MAX))
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def quantize_kv_e4m3(X: np.ndarray):
    """bf16 cache bits [B, Hkv, L, D] -> (uint8 E4M3 bits, float32 scale [Hkv]):
    one scale per KV head, max |x| / 448, so the head's largest value maps to
    the largest finite E4M3 value (x ~ bits * scale)."""
    B, Hkv = X.shape[:2]
    out = np.empty(X.shape, dtype=np.uint8)
    scale = np.ones(Hkv, dtype=np.float32)
    for g in range(Hkv):
        f = (X[:, g].astype(np.uint32) << 16).view(np.float32)
        m = float(np.abs(f).max())
        if m > 0:
            scale[g] = np.float32(m / E4M3_MAX)
        out[:, g] = f32_to_e4m3_bits(f / scale[g])
    return out, scale


def _rng(seed: int, *ids: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, *ids]))


def normal_bf16(shape, seed: int, *ids: int) -> np.ndarray:
    return f32_to_bf16_bits(_rng(seed, *ids).standard_normal(shape, dtype=np.float32))


def _fill_normal_bf16(dst: np.ndarray, seed: int, ids: tuple, tmp: np.ndarray) -> None:
    """Same values as normal_bf16(dst.shape, seed, *ids), written into dst in place.

    ``tmp`` is a float32 scratch of at least dst.size elements (reused across
    calls to avoid touching fresh memory for every chunk)."""
    n = dst.size
    f = tmp[:n].reshape(dst.shape)
    _rng(seed, *ids).standard_normal(out=f, dtype=np.float32)
    u = f.view(np.uint32)
    r = (u >> 16) & 1
    r += np.uint32(0x7FFF)
    r += u
    r >>= 16
    dst[...] = r


def draw_lengths(w: Workload, seed: int = BASE_SEED) -> np.ndarray:
    if w.ctx_min:
        return _rng(seed, _T_LEN).integers(w.ctx_min, w.ctx, size=w.batch, endpoint=True).astype(np.int32)
    return np.full(w.batch, w.ctx, dtype=np.int32)


def queries(w: Workload, layer: int, seed: int = BASE_SEED) -> np.ndarray:
    """bf16 bits [B, C, Hq, D]; layer 0 is the full-attention layer, 1.. sparse."""
    tid = _T_Q_FA if layer == 0 else _T_Q_SA
    return np.stack([normal_bf16((w.n_queries, w.n_q_heads, w.head_dim), seed, tid, layer, b)
                     for b in range(w.batch)])


def kv_slice(w: Workload, which: str, b: int, g: int, rows: int, seed: int = BASE_SEED) -> np.ndarray:
    """bf16 bits [rows, D] of K or V for sequence b, KV head g (before needles)."""
    tid = _T_K if which == "K" else _T_V
    return normal_bf16((rows, w.head_dim), seed, tid, 0, b, g)


def needle_positions(w: Workload, L: int, b: int, seed: int = BASE_SEED) -> np.ndarray:
    """Distinct positions in [0, L - window) that receive a planted key."""
    hi = max(1, L - w.window)
    n = min(w.needles, hi)
    return np.sort(_rng(seed, _T_NEEDLE, b).choice(hi, size=n, replace=False)).astype(np.int64)


def needle_key(w: Workload, q_fa: np.ndarray, b: int, g: int) -> np.ndarray:
    """Planted key for (b, g): 4*sqrt(D) times the unit mean of group g's queries.

    Its dot product with the group's queries is about four times that of a
    typical key aligned with them, so these tokens must win the selection.
    """
    G = w.group
    qf = (q_fa[b, :, g * G:(g + 1) * G, :].astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    mean = qf.reshape(-1, w.head_dim).mean(axis=0)
    unit = mean / max(np.linalg.norm(mean), 1e-30)
    return f32_to_bf16_bits((4.0 * np.sqrt(w.head_dim) * unit).astype(np.float32))


@dataclass
class Inputs:
    w: Workload
    q_fa: np.ndarray            # uint16 [B, C, Hq, D]
    q_sa: list                  # n_sparse x uint16 [B, C, Hq, D]
    K: np.ndarray               # uint16 bf16 bits [B, Hkv, Lmax, D], or uint8 E4M3 bits
    V: np.ndarray
    lens: np.ndarray            # int32 [B]
    needles: dict               # b -> positions
    k_scale: np.ndarray | None = None  # float32 [Hkv] for an E4M3 cache (value = bits * scale)
    v_scale: np.ndarray | None = None


def make_inputs(w: Workload, seed: int = BASE_SEED, lmax: int | None = None, kv: str = "bf16") -> Inputs:
    """Materialise every tensor of one decode step on the host.  kv="fp8"
    stores the cache as OCP E4M3 with one scale per KV head for K and for V
    (quantised from the same bf16 values)."""
    lens = draw_lengths(w, seed)
    Lmax = int(lmax if lmax is not None else w.ctx)
    if lens.max() > Lmax:
        raise ValueError("lmax smaller than a drawn length")
    q_fa = queries(w, 0, seed)
    q_sa = [queries(w, l, seed) for l in range(1, w.n_sparse + 1)]
    K = np.zeros((w.batch, w.n_kv_heads, Lmax, w.head_dim), dtype=np.uint16)
    V = np.zeros_like(K)
    jobs = [(which, b, g) for b in range(w.batch) for g in range(w.n_kv_heads) for which in ("K", "V")]
    nthreads = max(1, min(len(jobs), os.cpu_count() or 1, 16))
    chunk = int(lens.max()) * w.head_dim

    def work(part):
        tmp = np.empty(chunk, dtype=np.float32)
        for which, b, g in part:
            dst = (K if which == "K" else V)[b, g, :int(lens[b])]
            _fill_normal_bf16(dst, seed, (_T_K if which == "K" else _T_V, 0, b, g), tmp)

    with ThreadPoolExecutor(nthreads) as ex:
        list(ex.map(work, [jobs[i::nthreads] for i in range(nthreads)]))
    needles = {}
    for b in range(w.batch):
        L = int(lens[b])
        if w.needles:
            pos = needle_positions(w, L, b, seed)
            needles[b] = pos
            for g in range(w.n_kv_heads):
                K[b, g, pos] = needle_key(w, q_fa, b, g)
    if kv == "fp8":
        K8, ks = quantize_kv_e4m3(K)
        V8, vs = quantize_kv_e4m3(V)
        return Inputs(w, q_fa, q_sa, K8, V8, lens, needles, ks, vs)
    if kv != "bf16":
        raise ValueError(f"unknown cache format {kv}")
    return Inputs(w, q_fa, q_sa, K, V, lens, needles)
