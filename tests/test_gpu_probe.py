"""Streaming-read reference (stride_probe_read): bit-exact against a host XOR of the same words.

Each sink entry is the XOR of every 32-bit word in the first read_bytes of its row; with two
matrices, entries alternate a-row, b-row.  This is integer work, so the bar is equality.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n,ld,vocab,two", [(37, 1008, 1000, True), (5, 151936, 151936, False),
                                           (1, 8, 8, True), (0, 64, 64, True)])
def test_probe_read_xor(n, ld, vocab, two):
    import torch
    import paper_2609_14636_amd as P
    g = torch.Generator().manual_seed(n + ld)
    a = torch.randint(-2**15, 2**15, (n, ld), dtype=torch.int16, generator=g)
    b = torch.randint(-2**15, 2**15, (n, ld), dtype=torch.int16, generator=g)
    read_bytes = vocab * 2 // 16 * 16
    da, db = a.view(torch.bfloat16).cuda(), b.view(torch.bfloat16).cuda()
    sink = torch.full((max(2 * n, 1),), -1, dtype=torch.int32, device="cuda")
    P.stride_probe_read(da, db if two else None, read_bytes, sink)
    torch.cuda.synchronize()

    def xor_rows(m):
        w = m.numpy().view(np.uint32)[:, :read_bytes // 4] if n else np.zeros((0, 1), np.uint32)
        return np.bitwise_xor.reduce(w, axis=1) if n else np.zeros(0, np.uint32)
    want = np.stack([xor_rows(a), xor_rows(b)], 1).reshape(-1) if two else xor_rows(a)
    got = sink.cpu().numpy().view(np.uint32)[:want.size]
    assert np.array_equal(got, want)
