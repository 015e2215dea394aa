"""The ceiling probes (libf2probe.so, include/f2probe.h) through their C ABI: the copy
moves every word, and the bitwise-issue kernel computes what its definition says
(checked against a plain numpy model of the same instruction sequence)."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


def _bitops_model(threads, iters, op):
    t = np.arange(threads, dtype=np.uint64)
    v = [((t * 0x9E3779B9 + k * 0x85EBCA6B) & 0xFFFFFFFF).astype(np.uint32) for k in range(16)]
    for _ in range(iters):
        for k in range(16):
            if op == 0:
                v[k] = v[k] ^ v[(k + 1) & 15]
            else:
                v[k] = v[k] ^ v[(k + 1) & 15] ^ v[(k + 5) & 15]
    r = np.zeros(threads, np.uint64)
    for k in range(16):
        r += v[k]
    return (r & 0xFFFFFFFF).astype(np.uint32)


def test_copy_and_bitops(require_gpu):
    import torch
    from paper_2608_20532_amd import f2probe
    stream = torch.cuda.current_stream().cuda_stream
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    for words in (2, 1 << 20, (1 << 22) + 6):
        print(f"probe copy: {words} words", flush=True)
        src = torch.randint(-2 ** 63, 2 ** 63 - 1, (words,), generator=g, device="cuda", dtype=torch.int64)
        dst = torch.zeros_like(src)
        assert f2probe.f2probe_copy(src, dst, words, stream) == 0
        torch.cuda.synchronize()
        assert torch.equal(src, dst)
    out = torch.zeros(3 * 256, dtype=torch.int32, device="cuda")
    assert f2probe.f2probe_copy(out, out, 3, stream) == -1          # odd word count
    assert f2probe.f2probe_bitops(out, 0, 1, 0, stream) == -1       # no workgroups
    for op in (0, 1):
        print(f"probe bitops: op {op}", flush=True)
        assert f2probe.f2probe_bitops(out, 3, 5, op, stream) == 0
        torch.cuda.synchronize()
        got = out.cpu().numpy().view(np.uint32)
        assert np.array_equal(got, _bitops_model(3 * 256, 5, op))
