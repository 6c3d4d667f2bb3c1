"""The measurement probes of include/delta_probe.h read what they claim to read.

The benchmark compares the attention kernels with two floors measured by these probes (a
streaming read of a buffer, and a gather of 4 KB chunks of it): the floors mean something only
if every byte they are timed on is actually loaded.  Both probes fold the words they load with
XOR into their sink words, so the sink is recomputed here on the CPU from the same bytes: the
read probe's word per workgroup is the XOR of every 32-bit word of the workgroup's share of the
buffer, the gather probe's word per (workgroup, thread) the XOR of the thread's 16 bytes of every
chunk in the workgroup's part of the list.  Ragged shares (a buffer that is no multiple of the
per-step bytes, a list that does not divide evenly over the workgroups, repeated chunks) are
included.  Random 32-bit contents make a skipped or misplaced load show up with probability
1 - 2^-32 per word.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import D, log

pytestmark = pytest.mark.gpu


def _xor_words(a: np.ndarray, axis) -> np.ndarray:
    return np.bitwise_xor.reduce(a, axis=axis)


@pytest.mark.parametrize("unroll", [1, 2, 4, 8])
@pytest.mark.parametrize("n_wg,extra", [(13, 48), (256, 0), (1, 16)])
def test_read_probe_loads_every_word_of_its_share(unroll, n_wg, extra):
    d = D()
    g = torch.Generator().manual_seed(1000 + unroll * 7 + n_wg)
    nbytes = (16 << 20) + extra                      # a multiple of 16, not of the per-step bytes
    host = torch.randint(-2**31, 2**31 - 1, (nbytes // 4,), generator=g, dtype=torch.int32)
    buf = host.cuda()
    sink = torch.zeros(n_wg, dtype=torch.int32, device="cuda")
    log(f"read probe: {nbytes} bytes, {n_wg} workgroups, unroll {unroll}")
    d.delta_hbm_read_probe(buf, sink, n_wg, unroll)
    torch.cuda.synchronize()
    words = host.numpy().view(np.uint32).reshape(-1, 4)   # one row per 16-byte load
    n = words.shape[0]
    per = n // n_wg
    expect = np.empty(n_wg, dtype=np.uint32)
    for w in range(n_wg):
        lo = w * per
        hi = n if w == n_wg - 1 else lo + per
        expect[w] = _xor_words(words[lo:hi].reshape(-1), 0)
    got = sink.cpu().numpy().view(np.uint32)
    assert np.array_equal(got, expect)


@pytest.mark.parametrize("n_chunks,n_wg", [(3001, 7), (4096, 256), (5, 8), (1, 1)])
def test_gather_probe_loads_every_listed_chunk(n_chunks, n_wg):
    d = D()
    g = torch.Generator().manual_seed(2000 + n_chunks + n_wg)
    total_chunks = 4096                              # a 16 MiB buffer
    host = torch.randint(-2**31, 2**31 - 1, (total_chunks * 1024,), generator=g, dtype=torch.int32)
    chunks = torch.randint(0, total_chunks, (n_chunks,), generator=g, dtype=torch.int64)
    if n_chunks > 4:
        chunks[3] = chunks[2]                        # a repeated chunk counts twice
    buf = host.cuda()
    sink = torch.zeros(n_wg * 256, dtype=torch.int32, device="cuda")
    log(f"gather probe: {n_chunks} chunks, {n_wg} workgroups")
    d.delta_hbm_gather_probe(buf, chunks.cuda(), sink, n_wg)
    torch.cuda.synchronize()
    words = host.numpy().view(np.uint32).reshape(total_chunks, 256, 4)   # [chunk][thread][word]
    ch = chunks.numpy()
    expect = np.zeros((n_wg, 256), dtype=np.uint32)
    for w in range(n_wg):
        c0, c1 = n_chunks * w // n_wg, n_chunks * (w + 1) // n_wg
        if c1 > c0:
            expect[w] = _xor_words(_xor_words(words[ch[c0:c1]], 0), 1)
    got = sink.cpu().numpy().view(np.uint32).reshape(n_wg, 256)
    assert np.array_equal(got, expect)
