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


@pytest.mark.parametrize("n_words,two,sink_len", [(4, False, 4), (1000003 * 4, True, 8192),
                                                  (64 * 1024, True, 5)])
def test_probe_read_flat_xor(n_words, two, sink_len):
    """stride_probe_read_flat: the XOR of every sink word equals the XOR of every 32-bit word
    of the ranges read (the sink words past the launched waves stay as they were)."""
    import torch
    import paper_2609_14636_amd as P
    g = torch.Generator().manual_seed(n_words)
    a = torch.randint(-2**31, 2**31 - 1, (n_words + 8,), dtype=torch.int32, generator=g)
    b = torch.randint(-2**31, 2**31 - 1, (n_words + 8,), dtype=torch.int32, generator=g)
    sink = torch.zeros(sink_len, dtype=torch.int32, device="cuda")
    P.stride_probe_read_flat(a.cuda(), b.cuda() if two else None, n_words * 4, sink)
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(a.numpy()[:n_words].view(np.uint32))
    if two:
        want ^= np.bitwise_xor.reduce(b.numpy()[:n_words].view(np.uint32))
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == want


@pytest.mark.parametrize("n,ld,cols,masked", [(37, 1008, 1000, True), (3, 151936, 151936, False),
                                              (9, 24, 8, True)])
def test_probe_copy_rows(n, ld, cols, masked):
    """stride_probe_copy: rows with mask 1 copied (first copy_bytes only), rows with mask 0
    zero-filled up to copy_bytes, the rest of every row untouched.  Integer work: equality."""
    import torch
    import paper_2609_14636_amd as P
    g = torch.Generator().manual_seed(n * ld)
    src = torch.randint(-2**15, 2**15, (n, ld), dtype=torch.int16, generator=g)
    dst0 = torch.randint(-2**15, 2**15, (n, ld), dtype=torch.int16, generator=g)
    mask = (torch.rand(n, generator=g) < 0.6).to(torch.uint8) if masked else None
    copy_bytes = cols * 2 // 16 * 16
    dst = dst0.view(torch.bfloat16).cuda()
    P.stride_probe_copy(src.view(torch.bfloat16).cuda(), dst, None if mask is None else mask.cuda(),
                        copy_bytes)
    torch.cuda.synchronize()
    got = dst.cpu().view(torch.int16).numpy()
    want = dst0.numpy().copy()
    k = copy_bytes // 2
    m = np.ones(n, bool) if mask is None else mask.numpy().astype(bool)
    want[m, :k] = src.numpy()[m, :k]
    want[~m, :k] = 0
    assert np.array_equal(got, want)
