"""GPU: the streaming-read probe reads every 32-bit word of its buffer exactly
once in each load mode (the xor of its per-workgroup folds equals the
host's xor of the buffer), including a buffer
whose size leaves partial pieces and empty workgroup slices; the gather
modes (512- and 256-byte records) over record counts that give whole
pieces, partial pieces per slice, and empty slices."""
from __future__ import annotations

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("words16", [1 << 20, (1 << 20) + 3, 4096 * 64 + 17, 5])
@pytest.mark.parametrize("mode", [0, 1, 2, 3])
def test_stream_probe_reads_every_word_once(words16, mode):
    from paper_2609_26368_amd import hs2
    rng = np.random.default_rng(words16 + mode)
    host = rng.integers(0, 2 ** 32, size=4 * words16, dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.zeros(hs2.STREAM_PROBE_SINK_WORDS, dtype=torch.int32, device="cuda")
    print(f"[probe] mode={mode} words16={words16}", flush=True)
    hs2.hs2_stream_read_probe(buf, mode, sink)
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(host)
    assert int(np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))) == int(want)


@pytest.mark.parametrize("records", [1 << 15, 1 << 13, 1 << 12, 1 << 11, 1 << 10, 1])
@pytest.mark.parametrize("mode,record_bytes", [(4, 512), (5, 256)])
def test_stream_probe_gather_reads_every_word_once(mode, record_bytes, records):
    from paper_2609_26368_amd import hs2
    rng = np.random.default_rng(records + mode)
    host = rng.integers(0, 2 ** 32, size=record_bytes // 4 * records, dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).cuda()
    sink = torch.zeros(hs2.STREAM_PROBE_SINK_WORDS, dtype=torch.int32, device="cuda")
    print(f"[probe] mode={mode} records={records}", flush=True)
    hs2.hs2_stream_read_probe(buf, mode, sink)
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(host)
    assert int(np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))) == int(want)
