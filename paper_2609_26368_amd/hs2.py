"""ctypes binding of libhs2.so (include/hs2.h), same names as the C ABI.

Argument marshalling only: tensors are torch tensors on the current HIP
device; their data pointers and torch's current stream go to the library,
which does all the work in its kernels.  Shapes are checked here against the
dims before any call, because the C ABI cannot see buffer sizes.

The library must have been built (``__graft_entry__.build()`` or
``python paper_2609_26368_amd/_build.py``); loading fails loudly otherwise.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhs2.so")

HS2_OK = 0
HS2_ERR_NULL = -1
HS2_ERR_SHAPE = -2
HS2_ERR_UNSUPPORTED = -3
HS2_ERR_WORKSPACE = -4
HS2_ERR_ALIGN = -5
HS2_ERR_HIP = -6

EXPORTED = ["hs2_workspace_bytes", "hs2_full_attn_score_select", "hs2_sparse_attn", "hs2_sparse_attn_ex",
            "hs2_full_attn_score_select_fp8", "hs2_sparse_attn_fp8", "hs2_full_attn_score_select_blocks",
            "hs2_select_from_scores", "hs2_select_blocks_from_scores",
            "hs2_sparse_attn_noalloc", "hs2_stream_read_probe", "hs2_status_string", "hs2_last_error", "hs2_timing_enable",
            "hs2_timing_reset", "hs2_timing_read"]


class hs2_dims(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_queries", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("max_len", ctypes.c_int32),
                ("kv_stride_b", ctypes.c_int64), ("kv_stride_h", ctypes.c_int64), ("kv_stride_t", ctypes.c_int64),
                ("scale", ctypes.c_float)]


class HS2Error(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"hs2 status {status}: {msg}")
        self.status = status


_lib = None


def load() -> ctypes.CDLL:
    """Open libhs2.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    D = ctypes.POINTER(hs2_dims)
    lib.hs2_workspace_bytes.argtypes = [D, I32, I32]
    lib.hs2_workspace_bytes.restype = SZ
    lib.hs2_full_attn_score_select.argtypes = [D, P, P, P, P, I32, I32, P, P, P, P, P, SZ, P]
    lib.hs2_full_attn_score_select.restype = I32
    lib.hs2_sparse_attn.argtypes = [D, P, P, P, P, P, I32, P, P, SZ, P]
    lib.hs2_sparse_attn.restype = I32
    lib.hs2_sparse_attn_ex.argtypes = [D, P, P, P, P, P, I32, P, P, P, P, SZ, P]
    lib.hs2_sparse_attn_ex.restype = I32
    lib.hs2_full_attn_score_select_fp8.argtypes = [D, P, P, P, P, P, P, I32, I32, P, P, P, P, P, SZ, P]
    lib.hs2_full_attn_score_select_fp8.restype = I32
    lib.hs2_sparse_attn_fp8.argtypes = [D, P, P, P, P, P, P, P, I32, P, P, P, P, SZ, P]
    lib.hs2_sparse_attn_fp8.restype = I32
    lib.hs2_full_attn_score_select_blocks.argtypes = [D, P, P, P, P, I32, I32, I32, P, P, P, P, P, SZ, P]
    lib.hs2_full_attn_score_select_blocks.restype = I32
    lib.hs2_select_blocks_from_scores.argtypes = [D, P, P, I32, I32, I32, P, P, SZ, P]
    lib.hs2_select_blocks_from_scores.restype = I32
    lib.hs2_select_from_scores.argtypes = [D, P, P, I32, I32, P, P, SZ, P]
    lib.hs2_select_from_scores.restype = I32
    lib.hs2_sparse_attn_noalloc.argtypes = [D, P, P, P, P, P, I32, P, P]
    lib.hs2_sparse_attn_noalloc.restype = I32
    lib.hs2_stream_read_probe.argtypes = [P, SZ, I32, P, P]
    lib.hs2_stream_read_probe.restype = I32
    lib.hs2_status_string.argtypes = [I32]
    lib.hs2_status_string.restype = ctypes.c_char_p
    lib.hs2_last_error.argtypes = []
    lib.hs2_last_error.restype = ctypes.c_char_p
    lib.hs2_timing_enable.argtypes = [I32]
    lib.hs2_timing_enable.restype = I32
    lib.hs2_timing_reset.argtypes = []
    lib.hs2_timing_reset.restype = None
    lib.hs2_timing_read.argtypes = [ctypes.c_char_p, SZ, ctypes.POINTER(I32), ctypes.POINTER(ctypes.c_double), I32]
    lib.hs2_timing_read.restype = I32
    _lib = lib
    return lib


def make_dims(batch, n_queries, n_q_heads, n_kv_heads, head_dim, max_len, kv_strides=None, scale=0.0) -> hs2_dims:
    """Dims of a contiguous [B, Hkv, Lmax, D] cache unless strides are given."""
    if kv_strides is None:
        kv_strides = (n_kv_heads * max_len * head_dim, max_len * head_dim, head_dim)
    return hs2_dims(batch, n_queries, n_q_heads, n_kv_heads, head_dim, max_len, *kv_strides, scale)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _check(status: int):
    if status != HS2_OK:
        lib = load()
        raise HS2Error(status, f"{lib.hs2_status_string(status).decode()}: {lib.hs2_last_error().decode()}")


def _expect(t, name, shape, dtypes, device):
    if t is None:
        raise ValueError(f"{name} is required")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.dtype not in dtypes:
        raise ValueError(f"{name}: dtype {t.dtype}, expected one of {dtypes}")
    if t.device != device:
        raise ValueError(f"{name}: on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


_BF16 = (torch.bfloat16, torch.int16, torch.uint16)


_FP8 = (torch.uint8, torch.float8_e4m3fn)


def _check_kv(dims, K, V, device, fp8=False):
    dtypes, what = (_FP8, "E4M3 (uint8)") if fp8 else (_BF16, "bf16")
    for name, t in (("K", K), ("V", V)):
        if t.dtype not in dtypes or t.device != device:
            raise ValueError(f"{name}: {what} tensor on {device} expected")
        # largest element offset the kernels may touch must lie inside the tensor's storage
        last = ((dims.batch - 1) * dims.kv_stride_b + (dims.n_kv_heads - 1) * dims.kv_stride_h
                + (dims.max_len - 1) * dims.kv_stride_t + dims.head_dim)
        avail = t.untyped_storage().nbytes() // t.element_size() - t.storage_offset()
        if last > avail:
            raise ValueError(f"{name}: strides address {last} elements, storage holds {avail}")


def _check_scales(dims, k_scale, v_scale, device):
    for name, t in (("k_scale", k_scale), ("v_scale", v_scale)):
        _expect(t, name, (dims.n_kv_heads,), (torch.float32,), device)


def hs2_workspace_bytes(dims: hs2_dims, k: int, window: int) -> int:
    return int(load().hs2_workspace_bytes(ctypes.byref(dims), int(k), int(window)))


def hs2_full_attn_score_select(dims, q, K, V, len, k, window, out, idx, stats=None, scores=None, workspace=None,
                               stream=None):
    """Full-attention layer + pooled scores + selection; fills out, idx (and stats/scores)."""
    dev = q.device
    B, C, Hq, Hkv, D, L = dims.batch, dims.n_queries, dims.n_q_heads, dims.n_kv_heads, dims.head_dim, dims.max_len
    _expect(q, "q", (B, C, Hq, D), _BF16, dev)
    _check_kv(dims, K, V, dev)
    _expect(len, "len", (B,), (torch.int32,), dev)
    _expect(out, "out", (B, C, Hq, D), _BF16, dev)
    _expect(idx, "idx", (B, Hkv, C, k + window), (torch.int32,), dev)
    if stats is not None:
        _expect(stats, "stats", (B, C, Hq, 2), (torch.float32,), dev)
    if scores is not None:
        _expect(scores, "scores", (B, Hkv, C, L), (torch.float32,), dev)
    need = hs2_workspace_bytes(dims, k, window)
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace of {need} bytes required")
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(load().hs2_full_attn_score_select(ctypes.byref(dims), _ptr(q), _ptr(K), _ptr(V), _ptr(len), int(k),
                                             int(window), _ptr(out), _ptr(idx), _ptr(stats), _ptr(scores),
                                             _ptr(workspace), ws_bytes, _stream(stream)))


def hs2_sparse_attn(dims, q, K, V, len, idx, n_slots, out, workspace, stream=None):
    """Sparse-attention layer over the selected rows of the same cache."""
    dev = q.device
    B, C, Hq, Hkv, D = dims.batch, dims.n_queries, dims.n_q_heads, dims.n_kv_heads, dims.head_dim
    _expect(q, "q", (B, C, Hq, D), _BF16, dev)
    _check_kv(dims, K, V, dev)
    _expect(len, "len", (B,), (torch.int32,), dev)
    _expect(idx, "idx", (B, Hkv, C, n_slots), (torch.int32,), dev)
    _expect(out, "out", (B, C, Hq, D), _BF16, dev)
    _check(load().hs2_sparse_attn(ctypes.byref(dims), _ptr(q), _ptr(K), _ptr(V), _ptr(len), _ptr(idx), int(n_slots),
                                  _ptr(out), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                  _stream(stream)))


def hs2_sparse_attn_noalloc(dims, q, K, V, len, idx, n_slots, out, stream=None):
    """hs2_sparse_attn with the library's static per-GPU scratch instead of a
    workspace (no allocation in the call; calls on one GPU must not overlap)."""
    dev = q.device
    B, C, Hq, Hkv, D = dims.batch, dims.n_queries, dims.n_q_heads, dims.n_kv_heads, dims.head_dim
    _expect(q, "q", (B, C, Hq, D), _BF16, dev)
    _check_kv(dims, K, V, dev)
    _expect(len, "len", (B,), (torch.int32,), dev)
    _expect(idx, "idx", (B, Hkv, C, n_slots), (torch.int32,), dev)
    _expect(out, "out", (B, C, Hq, D), _BF16, dev)
    _check(load().hs2_sparse_attn_noalloc(ctypes.byref(dims), _ptr(q), _ptr(K), _ptr(V), _ptr(len), _ptr(idx),
                                          int(n_slots), _ptr(out), _stream(stream)))


def hs2_sparse_attn_ex(dims, q, K, V, len, idx, n_slots, sink, gate, out, workspace, stream=None):
    """Sparse-attention layer with per-head sink logits [Hq] float32 and/or
    output gate logits [B, C, Hq, D] bf16 (either may be None)."""
    dev = q.device
    B, C, Hq, Hkv, D = dims.batch, dims.n_queries, dims.n_q_heads, dims.n_kv_heads, dims.head_dim
    _expect(q, "q", (B, C, Hq, D), _BF16, dev)
    _check_kv(dims, K, V, dev)
    _expect(len, "len", (B,), (torch.int32,), dev)
    _expect(idx, "idx", (B, Hkv, C, n_slots), (torch.int32,), dev)
    _expect(out, "out", (B, C, Hq, D), _BF16, dev)
    if sink is not None:
        _expect(sink, "sink", (Hq,), (torch.float32,), dev)
    if gate is not None:
        _expect(gate, "gate", (B, C, Hq, D), _BF16, dev)
    _check(load().hs2_sparse_attn_ex(ctypes.byref(dims), _ptr(q), _ptr(K), _ptr(V), _ptr(len), _ptr(idx),
                                     int(n_slots), _ptr(sink), _ptr(gate), _ptr(out), _ptr(workspace),
                                     workspace.numel() * workspace.element_size(), _stream(stream)))


def hs2_full_attn_score_select_fp8(dims, q, K8, V8, k_scale, v_scale, len, k, window, out, idx, stats=None,
                                   scores=None, workspace=None, stream=None):
    """hs2_full_attn_score_select over an E4M3 cache (uint8 K8/V8, fp32 scales [Hkv])."""
    dev = q.device
    B, C, Hq, Hkv, D, L = dims.batch, dims.n_queries, dims.n_q_heads, dims.n_kv_heads, dims.head_dim, dims.max_len
    _expect(q, "q", (B, C, Hq, D), _BF16, dev)
    _check_kv(dims, K8, V8, dev, fp8=True)
    _check_scales(dims, k_scale, v_scale, dev)
    _expect(len, "len", (B,), (torch.int32,), dev)
    _expect(out, "out", (B, C, Hq, D), _BF16, dev)
    _expect(idx, "idx", (B, Hkv, C, k + window), (torch.int32,), dev)
    if stats is not None:
        _expect(stats, "stats", (B, C, Hq, 2), (torch.float32,), dev)
    if scores is not None:
        _expect(scores, "scores", (B, Hkv, C, L), (torch.float32,), dev)
    need = hs2_workspace_bytes(dims, k, window)
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace of {need} bytes required")
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(load().hs2_full_attn_score_select_fp8(ctypes.byref(dims), _ptr(q), _ptr(K8), _ptr(V8), _ptr(k_scale),
                                                 _ptr(v_scale), _ptr(len), int(k), int(window), _ptr(out), _ptr(idx),
                                                 _ptr(stats), _ptr(scores), _ptr(workspace), ws_bytes,
                                                 _stream(stream)))


def hs2_sparse_attn_fp8(dims, q, K8, V8, k_scale, v_scale, len, idx, n_slots, sink, gate, out, workspace,
                        stream=None):
    """hs2_sparse_attn_ex over an E4M3 cache (sink and gate may be None)."""
    dev = q.device
    B, C, Hq, Hkv, D = dims.batch, dims.n_queries, dims.n_q_heads, dims.n_kv_heads, dims.head_dim
    _expect(q, "q", (B, C, Hq, D), _BF16, dev)
    _check_kv(dims, K8, V8, dev, fp8=True)
    _check_scales(dims, k_scale, v_scale, dev)
    _expect(len, "len", (B,), (torch.int32,), dev)
    _expect(idx, "idx", (B, Hkv, C, n_slots), (torch.int32,), dev)
    _expect(out, "out", (B, C, Hq, D), _BF16, dev)
    if sink is not None:
        _expect(sink, "sink", (Hq,), (torch.float32,), dev)
    if gate is not None:
        _expect(gate, "gate", (B, C, Hq, D), _BF16, dev)
    _check(load().hs2_sparse_attn_fp8(ctypes.byref(dims), _ptr(q), _ptr(K8), _ptr(V8), _ptr(k_scale), _ptr(v_scale),
                                      _ptr(len), _ptr(idx), int(n_slots), _ptr(sink), _ptr(gate), _ptr(out),
                                      _ptr(workspace), workspace.numel() * workspace.element_size(),
                                      _stream(stream)))


def hs2_full_attn_score_select_blocks(dims, q, K, V, len, k, window, block, out, idx, stats=None, scores=None,
                                      workspace=None, stream=None):
    """hs2_full_attn_score_select with block-level selection (blocks of `block` tokens)."""
    dev = q.device
    B, C, Hq, Hkv, D, L = dims.batch, dims.n_queries, dims.n_q_heads, dims.n_kv_heads, dims.head_dim, dims.max_len
    _expect(q, "q", (B, C, Hq, D), _BF16, dev)
    _check_kv(dims, K, V, dev)
    _expect(len, "len", (B,), (torch.int32,), dev)
    _expect(out, "out", (B, C, Hq, D), _BF16, dev)
    _expect(idx, "idx", (B, Hkv, C, k + window), (torch.int32,), dev)
    if stats is not None:
        _expect(stats, "stats", (B, C, Hq, 2), (torch.float32,), dev)
    if scores is not None:
        _expect(scores, "scores", (B, Hkv, C, L), (torch.float32,), dev)
    need = hs2_workspace_bytes(dims, k, window)
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace of {need} bytes required")
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(load().hs2_full_attn_score_select_blocks(ctypes.byref(dims), _ptr(q), _ptr(K), _ptr(V), _ptr(len), int(k),
                                                    int(window), int(block), _ptr(out), _ptr(idx), _ptr(stats),
                                                    _ptr(scores), _ptr(workspace), ws_bytes, _stream(stream)))


def hs2_select_blocks_from_scores(dims, scores, len, k, window, block, idx, workspace, stream=None):
    """Block-level selection alone from given pooled scores [B, Hkv, C, max_len] float32."""
    dev = scores.device
    B, C, Hkv, L = dims.batch, dims.n_queries, dims.n_kv_heads, dims.max_len
    _expect(scores, "scores", (B, Hkv, C, L), (torch.float32,), dev)
    _expect(len, "len", (B,), (torch.int32,), dev)
    _expect(idx, "idx", (B, Hkv, C, k + window), (torch.int32,), dev)
    need = hs2_workspace_bytes(dims, k, window)
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace of {need} bytes required")
    _check(load().hs2_select_blocks_from_scores(ctypes.byref(dims), _ptr(scores), _ptr(len), int(k), int(window),
                                                int(block), _ptr(idx), _ptr(workspace),
                                                workspace.numel() * workspace.element_size(), _stream(stream)))


def hs2_select_from_scores(dims, scores, len, k, window, idx, workspace, stream=None):
    """Selection alone from given pooled scores [B, Hkv, C, max_len] float32."""
    dev = scores.device
    B, C, Hkv, L = dims.batch, dims.n_queries, dims.n_kv_heads, dims.max_len
    _expect(scores, "scores", (B, Hkv, C, L), (torch.float32,), dev)
    _expect(len, "len", (B,), (torch.int32,), dev)
    _expect(idx, "idx", (B, Hkv, C, k + window), (torch.int32,), dev)
    need = hs2_workspace_bytes(dims, k, window)
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace of {need} bytes required")
    _check(load().hs2_select_from_scores(ctypes.byref(dims), _ptr(scores), _ptr(len), int(k), int(window), _ptr(idx),
                                         _ptr(workspace), workspace.numel() * workspace.element_size(),
                                         _stream(stream)))


STREAM_PROBE_SINK_WORDS = 4096


def hs2_stream_read_probe(src, mode, sink, stream=None):
    """Streaming read of the whole of tensor src (device, contiguous) in the
    given load mode; sink (STREAM_PROBE_SINK_WORDS int32 / uint32 elements)
    receives one fold per workgroup, whose xor is the xor of src's words."""
    if not src.is_contiguous():
        raise ValueError("src must be contiguous")
    if (sink.numel() < STREAM_PROBE_SINK_WORDS or sink.element_size() != 4 or sink.device != src.device
            or not sink.is_contiguous()):
        raise ValueError(f"sink: {STREAM_PROBE_SINK_WORDS} contiguous 4-byte elements on the device of src")
    _check(load().hs2_stream_read_probe(_ptr(src), src.numel() * src.element_size(), int(mode), _ptr(sink),
                                        _stream(stream)))


def hs2_status_string(status: int) -> str:
    return load().hs2_status_string(int(status)).decode()


def hs2_last_error() -> str:
    return load().hs2_last_error().decode()


def hs2_timing_enable(on: bool) -> None:
    _check(load().hs2_timing_enable(1 if on else 0))


def hs2_timing_reset() -> None:
    load().hs2_timing_reset()


def hs2_timing_read() -> dict:
    """{kernel name: (launches, total ms)} of the launches recorded so far."""
    lib = load()
    n_max = 32
    names = ctypes.create_string_buffer(4096)
    counts = (ctypes.c_int32 * n_max)()
    tot = (ctypes.c_double * n_max)()
    n = lib.hs2_timing_read(names, 4096, counts, tot, n_max)
    if n < 0:
        _check(n)
    keys = names.raw.split(b"\0")[:n]
    return {keys[i].decode(): (int(counts[i]), float(tot[i])) for i in range(n)}


class HybridBlock:
    """Convenience wrapper: one workspace and the dims of a block's calls.

    ``full(q, K, V, lens)`` runs the full-attention layer and selection and
    returns (out, idx); ``sparse(q, K, V, lens, idx)`` runs one sparse layer.
    With ``kv_scales=(k_scale, v_scale)`` K and V are an E4M3 (uint8) cache;
    ``full(..., block=64)`` selects blocks of 64 tokens instead of tokens.
    """

    def __init__(self, batch, n_queries, n_q_heads, n_kv_heads, head_dim, max_len, k, window, device="cuda",
                 kv_strides=None, scale=0.0):
        self.dims = make_dims(batch, n_queries, n_q_heads, n_kv_heads, head_dim, max_len, kv_strides, scale)
        self.k, self.window = int(k), int(window)
        need = hs2_workspace_bytes(self.dims, self.k, self.window)
        if need == 0:
            raise HS2Error(HS2_ERR_SHAPE, hs2_last_error())
        self.workspace = torch.empty(need, dtype=torch.uint8, device=device)
        self.device = torch.device(device)

    def full(self, q, K, V, lens, stats=None, scores=None, out=None, idx=None, stream=None, kv_scales=None,
             block=None):
        d = self.dims
        if out is None:
            out = torch.empty((d.batch, d.n_queries, d.n_q_heads, d.head_dim), dtype=torch.bfloat16, device=q.device)
        if idx is None:
            idx = torch.empty((d.batch, d.n_kv_heads, d.n_queries, self.k + self.window), dtype=torch.int32,
                              device=q.device)
        if block:
            if kv_scales is not None:
                raise ValueError("block-level selection is served for bf16 caches")
            hs2_full_attn_score_select_blocks(d, q, K, V, lens, self.k, self.window, block, out, idx, stats, scores,
                                              self.workspace, stream)
        elif kv_scales is None:
            hs2_full_attn_score_select(d, q, K, V, lens, self.k, self.window, out, idx, stats, scores,
                                       self.workspace, stream)
        else:
            hs2_full_attn_score_select_fp8(d, q, K, V, kv_scales[0], kv_scales[1], lens, self.k, self.window, out,
                                           idx, stats, scores, self.workspace, stream)
        return out, idx

    def sparse(self, q, K, V, lens, idx, out=None, stream=None, sink=None, gate=None, kv_scales=None):
        """One sparse layer; sink [Hq] float32 and gate [B, C, Hq, D] bf16 are optional."""
        d = self.dims
        if out is None:
            out = torch.empty((d.batch, d.n_queries, d.n_q_heads, d.head_dim), dtype=torch.bfloat16, device=q.device)
        if kv_scales is not None:
            hs2_sparse_attn_fp8(d, q, K, V, kv_scales[0], kv_scales[1], lens, idx, idx.shape[-1], sink, gate, out,
                                self.workspace, stream)
        elif sink is None and gate is None:
            hs2_sparse_attn(d, q, K, V, lens, idx, idx.shape[-1], out, self.workspace, stream)
        else:
            hs2_sparse_attn_ex(d, q, K, V, lens, idx, idx.shape[-1], sink, gate, out, self.workspace, stream)
        return out
