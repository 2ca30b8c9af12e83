"""The C ABI without a GPU: the library loads, exports what include/hs2.h
declares, sizes workspaces and rejects invalid calls before launching."""
import ctypes
import os
import re

import pytest

from paper_2609_26368_amd import hs2

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hs2.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(hs2.LIB_PATH):
        from paper_2609_26368_amd import _build
        _build.build()
    return hs2.load()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(hs2_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_the_binding_names():
    assert declared_functions() == sorted(hs2.EXPORTED)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def dims(**kw):
    base = dict(batch=2, n_queries=1, n_q_heads=32, n_kv_heads=4, head_dim=128, max_len=4096)
    base.update(kw)
    strides = kw.pop("kv_strides", None)
    d = hs2.make_dims(base["batch"], base["n_queries"], base["n_q_heads"], base["n_kv_heads"], base["head_dim"],
                      base["max_len"], strides)
    return d


def test_workspace_bytes(lib):
    d = dims()
    n = hs2.hs2_workspace_bytes(d, 256, 64)
    assert n > 0 and n % 256 == 0
    # grows with the cache capacity and the chunk
    assert hs2.hs2_workspace_bytes(dims(max_len=8192), 256, 64) > n
    assert hs2.hs2_workspace_bytes(dims(n_queries=8), 256, 64) > n
    # invalid requests size to 0
    assert hs2.hs2_workspace_bytes(dims(n_q_heads=30), 256, 64) == 0
    assert hs2.hs2_workspace_bytes(d, 0, 0) == 0
    assert hs2.hs2_workspace_bytes(d, -1, 5) == 0
    assert hs2.hs2_workspace_bytes(dims(head_dim=64), 8, 8) == 0
    # head dim 256: partials twice as wide; at most 64 query rows per KV head
    assert hs2.hs2_workspace_bytes(dims(head_dim=256), 256, 64) > n
    assert hs2.hs2_workspace_bytes(dims(head_dim=256, n_q_heads=64, n_kv_heads=1), 1024, 128) > 0
    assert hs2.hs2_workspace_bytes(dims(head_dim=256, n_queries=2, n_q_heads=64, n_kv_heads=1), 16, 8) > 0
    assert hs2.hs2_workspace_bytes(dims(head_dim=256, n_queries=4, n_q_heads=64, n_kv_heads=1), 16, 8) == 0
    # token stride at most 2^24 elements (tiles of 64 rows use 32-bit offsets)
    assert hs2.hs2_workspace_bytes(dims(kv_strides=(0, 0, 1 << 24)), 8, 8) > 0
    assert hs2.hs2_workspace_bytes(dims(kv_strides=(0, 0, (1 << 24) + 8)), 8, 8) == 0
    # one grid row per (b, g, c) selection row: at most 65535 of them
    assert hs2.hs2_workspace_bytes(dims(batch=4095, n_queries=4, n_q_heads=16, n_kv_heads=4, max_len=64), 8, 8) > 0
    assert hs2.hs2_workspace_bytes(dims(batch=4096, n_queries=4, n_q_heads=16, n_kv_heads=4, max_len=64), 8, 8) == 0


FAKE = 1 << 20  # a 256-byte aligned non-null address; never dereferenced on the error paths


def call_full(lib, d, k=16, w=8, ptrs=None, ws_bytes=1 << 40):
    p = dict(q=FAKE, K=FAKE, V=FAKE, len=FAKE, out=FAKE, idx=FAKE, stats=None, scores=None, ws=FAKE)
    p.update(ptrs or {})
    vp = ctypes.c_void_p
    return lib.hs2_full_attn_score_select(ctypes.byref(d) if d is not None else None, vp(p["q"]), vp(p["K"]),
                                          vp(p["V"]), vp(p["len"]), k, w, vp(p["out"]), vp(p["idx"]),
                                          vp(p["stats"]), vp(p["scores"]), vp(p["ws"]), ws_bytes, None)


def test_full_attn_rejects_before_launch(lib):
    d = dims()
    assert call_full(lib, None) == hs2.HS2_ERR_NULL
    assert call_full(lib, dims(n_q_heads=30)) == hs2.HS2_ERR_SHAPE
    assert call_full(lib, dims(n_queries=0)) == hs2.HS2_ERR_SHAPE
    assert call_full(lib, dims(n_queries=17)) == hs2.HS2_ERR_SHAPE
    assert call_full(lib, dims(head_dim=64)) == hs2.HS2_ERR_UNSUPPORTED
    assert call_full(lib, dims(head_dim=192)) == hs2.HS2_ERR_UNSUPPORTED
    assert call_full(lib, dims(head_dim=256, n_queries=4, n_q_heads=64, n_kv_heads=1)) == hs2.HS2_ERR_UNSUPPORTED
    assert "256" in hs2.hs2_last_error()  # 4 * 64 query rows
    # kv_stride_t must cover the head dim
    assert call_full(lib, dims(head_dim=256, kv_strides=(4096 * 128 * 4, 4096 * 128, 128))) == hs2.HS2_ERR_ALIGN
    assert call_full(lib, dims(n_q_heads=128, n_kv_heads=1)) == hs2.HS2_ERR_UNSUPPORTED  # G = 128
    assert call_full(lib, dims(n_q_heads=64, n_kv_heads=2, n_queries=8)) == hs2.HS2_ERR_UNSUPPORTED  # 256 rows
    assert call_full(lib, dims(max_len=0)) == hs2.HS2_ERR_SHAPE
    assert call_full(lib, d, k=0, w=0) == hs2.HS2_ERR_SHAPE
    assert call_full(lib, d, k=-3, w=8) == hs2.HS2_ERR_SHAPE
    assert call_full(lib, d, ptrs={"q": None}) == hs2.HS2_ERR_NULL
    assert call_full(lib, d, ptrs={"idx": None}) == hs2.HS2_ERR_NULL
    assert call_full(lib, d, ptrs={"ws": None}) == hs2.HS2_ERR_NULL
    assert call_full(lib, d, ptrs={"K": FAKE + 2}) == hs2.HS2_ERR_ALIGN
    assert call_full(lib, d, ptrs={"ws": FAKE + 16}) == hs2.HS2_ERR_ALIGN
    assert call_full(lib, dims(kv_strides=(4096 * 128 * 4, 4096 * 128, 130))) == hs2.HS2_ERR_ALIGN
    need = hs2.hs2_workspace_bytes(d, 16, 8)
    assert call_full(lib, d, ws_bytes=need - 256) == hs2.HS2_ERR_WORKSPACE
    assert "workspace" in hs2.hs2_last_error()


def test_sparse_and_select_reject_before_launch(lib):
    d = dims()
    vp = ctypes.c_void_p
    st = lib.hs2_sparse_attn(ctypes.byref(d), vp(FAKE), vp(FAKE), vp(FAKE), vp(FAKE), vp(FAKE), 0, vp(FAKE),
                             vp(FAKE), 1 << 40, None)
    assert st == hs2.HS2_ERR_SHAPE
    st = lib.hs2_sparse_attn(ctypes.byref(d), vp(FAKE), vp(FAKE), vp(FAKE), vp(FAKE), None, 64, vp(FAKE),
                             vp(FAKE), 1 << 40, None)
    assert st == hs2.HS2_ERR_NULL
    st = lib.hs2_sparse_attn(ctypes.byref(d), vp(FAKE), vp(FAKE), vp(FAKE), vp(FAKE), vp(FAKE), 64, vp(FAKE),
                             vp(FAKE), 16, None)
    assert st == hs2.HS2_ERR_WORKSPACE
    st = lib.hs2_select_from_scores(ctypes.byref(d), None, vp(FAKE), 8, 8, vp(FAKE), vp(FAKE), 1 << 40, None)
    assert st == hs2.HS2_ERR_NULL
    st = lib.hs2_select_from_scores(ctypes.byref(d), vp(FAKE + 2), vp(FAKE), 8, 8, vp(FAKE), vp(FAKE), 1 << 40,
                                    None)
    assert st == hs2.HS2_ERR_ALIGN


def test_sparse_ex_rejects_before_launch(lib):
    d = dims()
    vp = ctypes.c_void_p

    def call(sink=None, gate=None, n_slots=24, ws_bytes=1 << 40):
        return lib.hs2_sparse_attn_ex(ctypes.byref(d), vp(FAKE), vp(FAKE), vp(FAKE), vp(FAKE), vp(FAKE), n_slots,
                                      None if sink is None else vp(sink), None if gate is None else vp(gate),
                                      vp(FAKE), vp(FAKE), ws_bytes, None)

    assert call(n_slots=0) == hs2.HS2_ERR_SHAPE
    assert call(sink=FAKE + 2) == hs2.HS2_ERR_ALIGN
    assert call(gate=FAKE + 4) == hs2.HS2_ERR_ALIGN
    assert "gate" in hs2.hs2_last_error()
    assert call(sink=FAKE, gate=FAKE, ws_bytes=256) == hs2.HS2_ERR_WORKSPACE


def test_fp8_entry_points_reject_before_launch(lib):
    vp = ctypes.c_void_p

    def full(d, ks=FAKE, vs=FAKE, K=FAKE, ws_bytes=1 << 40):
        return lib.hs2_full_attn_score_select_fp8(ctypes.byref(d), vp(FAKE), vp(K), vp(FAKE),
                                                  None if ks is None else vp(ks), None if vs is None else vp(vs),
                                                  vp(FAKE), 16, 8, vp(FAKE), vp(FAKE), None, None, vp(FAKE),
                                                  ws_bytes, None)

    def sparse(d, ks=FAKE, vs=FAKE, n_slots=24):
        return lib.hs2_sparse_attn_fp8(ctypes.byref(d), vp(FAKE), vp(FAKE), vp(FAKE),
                                       None if ks is None else vp(ks), None if vs is None else vp(vs), vp(FAKE),
                                       vp(FAKE), n_slots, None, None, vp(FAKE), vp(FAKE), 1 << 40, None)

    d = dims()
    for call in (full, sparse):
        assert call(d, ks=None) == hs2.HS2_ERR_NULL
        assert call(d, vs=None) == hs2.HS2_ERR_NULL
        assert "scale" in hs2.hs2_last_error()
        assert call(d, ks=FAKE + 2) == hs2.HS2_ERR_ALIGN
        # one byte per element: strides must keep 16-byte loads aligned
        assert call(dims(kv_strides=(4096 * 136 * 4, 4096 * 136, 136))) == hs2.HS2_ERR_ALIGN
        # at most 128 query rows per KV head (C * pow2(G))
        assert call(dims(n_queries=8, n_q_heads=32, n_kv_heads=1)) == hs2.HS2_ERR_UNSUPPORTED
        assert call(dims(head_dim=64)) == hs2.HS2_ERR_UNSUPPORTED
    assert full(d, K=FAKE + 8) == hs2.HS2_ERR_ALIGN
    assert sparse(d, n_slots=0) == hs2.HS2_ERR_SHAPE
    need = hs2.hs2_workspace_bytes(d, 16, 8)
    assert full(d, ws_bytes=need - 256) == hs2.HS2_ERR_WORKSPACE


def test_fp8_binding_checks_dtypes_before_calling():
    import torch
    d = dims(batch=1, max_len=64)
    q = torch.zeros((1, 1, 32, 128), dtype=torch.bfloat16)
    K8 = torch.zeros((1, 4, 64, 128), dtype=torch.uint8)
    Kb = torch.zeros((1, 4, 64, 128), dtype=torch.bfloat16)
    sc = torch.ones(4, dtype=torch.float32)
    lens = torch.full((1,), 64, dtype=torch.int32)
    out = torch.zeros((1, 1, 32, 128), dtype=torch.bfloat16)
    idx = torch.zeros((1, 4, 1, 8), dtype=torch.int32)
    ws = torch.zeros(1 << 20, dtype=torch.uint8)
    with pytest.raises(ValueError, match="E4M3"):  # a bf16 cache passed as FP8
        hs2.hs2_full_attn_score_select_fp8(d, q, Kb, Kb, sc, sc, lens, 4, 4, out, idx, workspace=ws)
    with pytest.raises(ValueError, match="k_scale"):
        hs2.hs2_full_attn_score_select_fp8(d, q, K8, K8, torch.ones(3), sc, lens, 4, 4, out, idx, workspace=ws)
    with pytest.raises(ValueError, match="v_scale"):
        hs2.hs2_sparse_attn_fp8(d, q, K8, K8, sc, None, lens, idx, 8, None, None, out, ws)
    with pytest.raises(ValueError, match="bf16"):  # an FP8 cache passed to the bf16 entry point
        hs2.hs2_sparse_attn(d, q, K8, K8, lens, idx, 8, out, ws)


def test_block_selection_rejects_before_launch(lib):
    vp = ctypes.c_void_p

    def full(d, k=128, w=16, block=64, ws_bytes=1 << 40):
        return lib.hs2_full_attn_score_select_blocks(ctypes.byref(d), vp(FAKE), vp(FAKE), vp(FAKE), vp(FAKE), k, w,
                                                     block, vp(FAKE), vp(FAKE), None, None, vp(FAKE), ws_bytes, None)

    def sel(d, k=128, w=16, block=64, scores=FAKE, ws_bytes=1 << 40):
        return lib.hs2_select_blocks_from_scores(ctypes.byref(d), vp(scores), vp(FAKE), k, w, block, vp(FAKE),
                                                 vp(FAKE), ws_bytes, None)

    d = dims()
    for call in (full, sel):
        assert call(d, block=0) == hs2.HS2_ERR_SHAPE
        assert call(d, block=48) == hs2.HS2_ERR_SHAPE      # not a power of two
        assert call(d, block=8) == hs2.HS2_ERR_SHAPE       # below 16
        assert call(d, block=512) == hs2.HS2_ERR_SHAPE     # above 256
        assert call(d, k=100) == hs2.HS2_ERR_SHAPE         # k not a whole number of blocks
        assert "multiple" in hs2.hs2_last_error()
        # more than 16384 blocks per row
        assert call(dims(max_len=16384 * 16 + 1), block=16) == hs2.HS2_ERR_UNSUPPORTED
    assert sel(d, scores=FAKE + 2) == hs2.HS2_ERR_ALIGN
    assert sel(d, scores=None) == hs2.HS2_ERR_NULL
    need = hs2.hs2_workspace_bytes(d, 128, 16)
    assert full(d, ws_bytes=need - 256) == hs2.HS2_ERR_WORKSPACE
    assert sel(d, ws_bytes=need - 256) == hs2.HS2_ERR_WORKSPACE


def test_status_strings(lib):
    for code in (hs2.HS2_OK, hs2.HS2_ERR_NULL, hs2.HS2_ERR_SHAPE, hs2.HS2_ERR_UNSUPPORTED, hs2.HS2_ERR_WORKSPACE,
                 hs2.HS2_ERR_ALIGN, hs2.HS2_ERR_HIP):
        s = hs2.hs2_status_string(code)
        assert s and s != "unknown status"
    assert hs2.hs2_status_string(-99) == "unknown status"


def test_binding_checks_shapes_before_calling():
    import torch
    d = dims(batch=1, max_len=64)
    q = torch.zeros((1, 1, 32, 128), dtype=torch.bfloat16)
    K = torch.zeros((1, 4, 64, 128), dtype=torch.bfloat16)
    lens = torch.full((1,), 64, dtype=torch.int32)
    out = torch.zeros((1, 1, 32, 128), dtype=torch.bfloat16)
    idx_bad = torch.zeros((1, 4, 1, 7), dtype=torch.int32)
    with pytest.raises(ValueError):
        hs2.hs2_full_attn_score_select(d, q, K, K, lens, 4, 4, out, idx_bad, workspace=torch.zeros(16))
    K_short = torch.zeros((1, 4, 32, 128), dtype=torch.bfloat16)
    idx = torch.zeros((1, 4, 1, 8), dtype=torch.int32)
    with pytest.raises(ValueError):
        hs2.hs2_full_attn_score_select(d, q, K_short, K_short, lens, 4, 4, out, idx, workspace=torch.zeros(16))


def test_stream_probe_rejects_before_launch(lib):
    vp = ctypes.c_void_p
    assert lib.hs2_stream_read_probe(None, 1024, 0, vp(FAKE), None) == hs2.HS2_ERR_NULL
    assert lib.hs2_stream_read_probe(vp(FAKE), 1024, 0, None, None) == hs2.HS2_ERR_NULL
    assert lib.hs2_stream_read_probe(vp(FAKE), 1024, 6, vp(FAKE), None) == hs2.HS2_ERR_SHAPE
    # the gather modes read 512- (mode 4) or 256-byte records (mode 5), a power of two of them
    assert lib.hs2_stream_read_probe(vp(FAKE), 3 * 512, 4, vp(FAKE), None) == hs2.HS2_ERR_SHAPE
    assert lib.hs2_stream_read_probe(vp(FAKE), 1024 + 16, 4, vp(FAKE), None) == hs2.HS2_ERR_SHAPE
    assert lib.hs2_stream_read_probe(vp(FAKE), 256, 4, vp(FAKE), None) == hs2.HS2_ERR_SHAPE
    assert lib.hs2_stream_read_probe(vp(FAKE), 3 * 256, 5, vp(FAKE), None) == hs2.HS2_ERR_SHAPE
    assert lib.hs2_stream_read_probe(vp(FAKE), 1024, -1, vp(FAKE), None) == hs2.HS2_ERR_SHAPE
    assert lib.hs2_stream_read_probe(vp(FAKE), 0, 0, vp(FAKE), None) == hs2.HS2_ERR_SHAPE
    assert lib.hs2_stream_read_probe(vp(FAKE + 8), 1024, 0, vp(FAKE), None) == hs2.HS2_ERR_ALIGN
    assert lib.hs2_stream_read_probe(vp(FAKE), 1000, 0, vp(FAKE), None) == hs2.HS2_ERR_ALIGN


def test_noalloc_sparse_rejects_before_launch(lib):
    vp = ctypes.c_void_p
    d = dims()
    st = lib.hs2_sparse_attn_noalloc(ctypes.byref(d), vp(FAKE), vp(FAKE), vp(FAKE), vp(FAKE), vp(FAKE), 0, vp(FAKE),
                                     None)
    assert st == hs2.HS2_ERR_SHAPE
    # more scratch than the static array holds: 8192 selection rows of 8192 slots
    big = dims(batch=64, n_queries=16, n_q_heads=64, n_kv_heads=8)
    st = lib.hs2_sparse_attn_noalloc(ctypes.byref(big), vp(FAKE), vp(FAKE), vp(FAKE), vp(FAKE), vp(FAKE), 8192,
                                     vp(FAKE), None)
    assert st == hs2.HS2_ERR_WORKSPACE
    assert "static scratch" in hs2.hs2_last_error()
