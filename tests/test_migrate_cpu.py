"""Host logic of migration by recomputation (no GPU): the chunk plan that
recompute_kv issues and the KV-transfer sizes it is compared with."""

from __future__ import annotations

import torch

from paper_2606_18600_amd import synth
from paper_2606_18600_amd.migrate import migration_points, recompute_kv, transfer_bytes


class _RecordingStage:
    def __init__(self):
        self.calls = []

    def prefill(self, q_lens, ctx_lens, bt, hin, hout, stream=0):
        self.calls.append((list(q_lens), list(ctx_lens), hin.data_ptr(), hout.data_ptr(),
                           hin.shape[0], stream))
        return hout


def test_recompute_chunks_cover_every_position_in_order():
    H = 8
    for L, chunk in ((1, 2048), (2048, 2048), (2049, 2048), (5000, 2048), (37, 5)):
        st = _RecordingStage()
        hidden = torch.zeros((L, H))
        out = torch.zeros((L, H))
        recompute_kv(st, hidden, torch.zeros((1, 1), dtype=torch.int32), chunk=chunk, out=out,
                     stream=7)
        pos = 0
        for q, c, pin, pout, rows, s in st.calls:
            assert q == [rows] and c == [pos] and 1 <= rows <= chunk and s == 7
            # each chunk reads and writes its own rows of the full-length buffers
            assert pin == hidden.data_ptr() + pos * H * 4
            assert pout == out.data_ptr() + pos * H * 4
            pos += rows
        assert pos == L and len(st.calls) == -(-L // chunk)


def test_transfer_bytes_llama70b():
    # Llama-3-70B: 80 layers x 8 kv heads x 128 dims x (K, V) x 2 bytes
    # = 327,680 bytes of KV per token; 64K tokens are 20 GiB
    sh = synth.LLAMA70B
    assert transfer_bytes(sh, 1, 1) == 4096
    assert transfer_bytes(sh, 80, 1) == 327_680
    assert transfer_bytes(sh, 80, 65536) == 20 * 2**30
    rows = migration_points(sh, 20, [1024], [100.0], {"x": 1.0})
    L, b, ms, link = rows[0]
    assert (L, b, ms) == (1024, 1024 * 20 * 4096, 100.0)
    assert abs(link["x"] - b / 1e9 * 1e3) < 1e-9
