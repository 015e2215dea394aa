"""The ceiling probes (libf2probe.so, include/f2probe.h) through their C ABI: the copy
moves every word, the bitwise-issue kernel computes what its definition says
(checked against a plain numpy model of the same instruction sequence), and the
scattered-access kernel reads and writes exactly the slots its hash names."""
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


def _mix64(z):
    with np.errstate(over="ignore"):
        z = z + np.uint64(0x9E3779B97F4A7C15)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


def test_scatter_probe(require_gpu):
    import torch
    from paper_2608_20532_amd import f2probe
    stream = torch.cuda.current_stream().cuda_stream
    nbytes, blocks, per = 1 << 16, 3, 5
    threads = 256 * blocks
    t = np.repeat(np.arange(threads, dtype=np.uint64), per)
    r = np.tile(np.arange(per, dtype=np.uint64), threads)
    h = _mix64(t * np.uint64(64) + r)
    g = torch.Generator(device="cuda")
    g.manual_seed(9)
    buf = torch.randint(-2 ** 63, 2 ** 63 - 1, (nbytes // 8,), generator=g, device="cuda", dtype=torch.int64)
    host = buf.cpu().numpy().view(np.uint64).copy()
    out = torch.zeros(threads, dtype=torch.int64, device="cuda")
    print("probe scatter: reads", flush=True)
    assert f2probe.f2probe_scatter(buf, nbytes, blocks, per, 0, out, stream) == 0
    torch.cuda.synchronize()
    sl = (h % np.uint64(nbytes // 32)).astype(np.int64)
    w = host.view(np.uint32).reshape(-1, 8)[sl]              # the 32-byte slot as eight 32-bit words
    v = ((w[:, 0] ^ w[:, 4]).astype(np.uint64) << np.uint64(32)) | (w[:, 1] ^ w[:, 2] ^ w[:, 3] ^ w[:, 5] ^ w[:, 6] ^ w[:, 7]).astype(np.uint64)
    want = np.bitwise_xor.reduce(v.reshape(threads, per), axis=1)
    assert np.array_equal(out.cpu().numpy().view(np.uint64), want)
    print("probe scatter: writes", flush=True)
    assert f2probe.f2probe_scatter(buf, nbytes, blocks, per, 1, None, stream) == 0
    torch.cuda.synchronize()
    got = buf.cpu().numpy().view(np.uint64).reshape(-1, 2)
    sl = (h % np.uint64(nbytes // 16)).astype(np.int64)
    hit = np.zeros(nbytes // 16, bool)
    hit[sl] = True
    assert np.array_equal(got[~hit], host.reshape(-1, 2)[~hit])   # untouched slots keep their words
    writers = {}                                                  # every written slot holds one of its writers
    for k in range(len(sl)):
        writers.setdefault(int(sl[k]), set()).add((int(t[k]) & 0xFFFFFFFF) | (int(r[k]) << 32))
    for s_, ws in writers.items():
        assert int(got[s_, 0]) in ws and int(got[s_, 1]) == 0
