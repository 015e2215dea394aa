#!/usr/bin/env python3
"""Benchmark of the GF(2) fit + encode hot path on one MI355X.

A step is one pass of the whole path over one batch of synthetic input that is
already resident in HBM: f2_fit_batch over every context (plan, reduce,
classify, insert, finalize) followed by f2_encode_batch over the query batch
against the model just fitted.  Default workload ("step"): the 80,000-context
fit (widths 8..256, lognormal row counts, 7.24M rows, 1% contradictory), then
100M Zipf(1.1) queries (stride 4 words, 1% outside the span) encoded against the
80,000 maps just fitted.  The other configurations (the 64 wide contexts of
width 4,095, the 4,096-context batch with 1M queries, the single context) are
timed the same way and reported under "other_configs" of the same line.

Prints one JSON line.  `value` is fit rows/s over the fit phase of the timed
steps; encode words/s and per-phase figures are reported beside it.  Each phase
is one library call, timed with HIP events on the stream it is enqueued on.
The roofline object describes the phase that takes longer: its algorithmic HBM
bytes per call over its average duration, against the 8 TB/s HBM peak (the
wide-context fit: algorithmic 32-bit operations against the integer issue
peak), with the rate a streaming copy or an XOR issue probe reaches on the same
GPU beside it, and the measured HBM traffic of its kernels from the committed
rocprofv3 counter summary when that summary was taken on the current kernel
source.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# integer VALU peak: the fp32 vector rate (157.3 TFLOP/s = 256 compute units x 2.4 GHz x 256
# flops) counts an FMA as two flops, so a compute unit retires 128 32-bit lane operations per
# clock; bitwise ops issue at that rate (the probe's v_xor_b32 run reaches 54.8 T/s, above the
# 39.3 T/s that 64 lanes per clock would allow)
INT_PEAK_TOPS = 256 * 128 * 2.4e9 / 1e12
KERNEL_SOURCE = os.path.join(ROOT, "paper_2608_20532_amd", "csrc", "f2gpu.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.txt")

WORKLOADS = {
    # name: (fit recipe, contexts, queries, stride, out-of-span fraction, zipf exponent, description)
    "step": (3, 80000, 100_000_000, 4, 0.01, 1.1,
             "fit 80000 contexts, n in [8,256] geometric (mean 40), lognormal rows (median 30, max 4000), "
             "x in a random 0.7n-dim subspace, 1% contradictory (7.24M rows); then encode 100M Zipf(1.1) "
             "queries, stride 4, 1% out of span, against the 80000 maps just fitted"),
    "recipe2": (2, 4096, 1_000_000, 2, 0.02, 0.0,
                "fit 4096 contexts, n in [17,97] (16-96 uniform bits + 1 reserved), 2(n+1) rows, 5% contradictory; "
                "encode 1M uniform queries, stride 2, 2% out of span"),
    "recipe1": (1, 1, 1000, 1, 0.10, 0.0,
                "fit 1 context, n=33 (32 uniform bits + 1 reserved), 200 rows; encode 1000 queries, 10% out of span"),
    "recipe3": (3, 80000, 1_000_000, 4, 0.01, 1.1,
                "fit 80000 contexts, n in [8,256] geometric (mean 40), lognormal rows (median 30, max 4000), "
                "x in a random 0.7n-dim subspace, 1% contradictory; encode 1M Zipf(1.1) queries, stride 4"),
    "recipe4": (4, 64, 0, 1, 0.0, 0.0, "fit 64 contexts, n=4095, 8192 uniform rows each (full rank)"),
    "recipe5": (5, 80000, 100_000_000, 4, 0.01, 1.1,
                "encode only: the 80000 maps of the n-in-[8,256] workload, 100M Zipf(1.1) queries, stride 4, "
                "1% out of span"),
}

# streaming kernels outside the fit/encode step: (rows or words, k values per row, description)
STREAM_WORKLOADS = {
    "vectorize": (7_240_070, 5, "Eq. 1 rows from k=5 parsed 64-bit values (d=321) plus 128-bit outputs, "
                                "7,240,070 rows (the row count of the n-in-[8,256] fit workload)"),
    "merge": (100_000_000, 0, "100M encoded words: a 17-bit field XORed in at bit 105, opaque bits 122 and 124 "
                              "restored from recorded state"),
    "pool": (80_000, 3, "pool the bases of 240,000 shard contexts (each n-in-[8,256] context's rows split in 3, "
                        "fitted apart) back into 80,000 contexts"),
    "group": (7_240_070, 0, "group the 7,240,070 rows of the n-in-[8,256] fit workload, interleaved at random "
                            "(each context's order kept, stride 7 words), back by context for the fit"),
}


def fit_bytes(wl, rank):
    """Algorithmic HBM bytes of one fit: rows, offsets and widths in; basis rows, pivots, maps and scalars out."""
    import numpy as np
    n = wl.n_bits.astype(np.int64)
    W = (n + 64) // 64 + 2
    rows_in = int(wl.rows.nbytes) + 8 * (wl.num_ctx + 1) + 4 * wl.num_ctx
    out = int((rank.astype(np.int64) * W * 8).sum() + 4 * rank.sum() + (16 * (n + 1)).sum()) + 20 * wl.num_ctx
    return rows_in + out


def fit_int_ops(wl, rank):
    """Classical Gauss-Jordan word operations of the streaming method (32-bit lane ops): the i-th
    retained row is reduced by half of the i rows before it and cleared from half of them, 2(fw+2)
    words each; every row after the rank reaches d costs the output words (4) of half the columns."""
    import numpy as np
    n = wl.n_bits.astype(np.int64)
    d = n + 1
    w32 = 2 * ((n + 64) // 64 + 2)
    r = rank.astype(np.int64)
    later = np.where(r == d, np.maximum(wl.m_rows.astype(np.int64) - d, 0), 0)
    return int((w32 * r * (r - 1) // 2).sum() + (later * (d // 2) * 4).sum())


def encode_bytes(wl, nq, stride):
    """Per query: context id, x words, 128-bit word, flag byte; plus every context's map read once."""
    import numpy as np
    return nq * (4 + 8 * stride + 16 + 1) + int((16 * (wl.n_bits.astype(np.int64) + 1)).sum())


def source_hash():
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def load_traffic(workload):
    """Measured HBM bytes per call of each phase, if the counter summary matches the current source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None, "no counter summary"
    meta, phases = {}, {}
    with open(TRAFFIC_FILE) as f:
        for line in f:
            parts = line.split()
            if not parts or parts[0].startswith("#"):
                continue
            if parts[0] == "phase" and len(parts) >= 5 and parts[1] == workload:
                phases[parts[2]] = {"bytes": float(parts[3]), "kernels": parts[4].split(",")}
            elif len(parts) == 2:
                meta[parts[0]] = parts[1]
    if meta.get("source_sha256") != source_hash():
        return None, "kernel source changed since the counters were taken"
    return phases, None


def measured_traffic(workload, phase, roof):
    """Add the measured HBM bytes per call of a phase (or why there are none) to a roofline object."""
    traffic, why = load_traffic(workload)
    tr = traffic.get(phase) if traffic else None
    roof["traffic"] = tr["bytes"] if tr else None
    if tr:
        roof["kernels"] = tr["kernels"]
    else:
        roof["traffic_note"] = why or f"no counters for the {phase} phase of this workload"
    return roof


def sub_workload(wl, c0, c1):
    """Contexts [c0, c1) of a workload as (rows, row_off, n_bits) with rebased offsets."""
    off = wl.row_off[c0:c1 + 1]
    return wl.rows[off[0]:off[-1]], off - off[0], wl.n_bits[c0:c1]


def oracle_fit_parallel(wl, k, seconds=5.0):
    """The same oracle fit run as independent context chunks on every usable host core at
    once (one thread each; the C calls release the interpreter lock): "oracle x N cores"."""
    import threading
    import oracle
    C = wl.num_ctx
    chunks = [(c0, min(C, c0 + k)) for c0 in range(0, C, k)]
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    done = [0] * n
    t0 = time.perf_counter()

    def work(tid):
        j = tid
        while time.perf_counter() - t0 < seconds:
            c0, c1 = chunks[j % len(chunks)]
            rows, off, nb = sub_workload(wl, c0, c1)
            oracle.fit_batch(rows, off, nb)
            done[tid] += int(wl.m_rows[c0:c1].sum())
            j += n

    threads = [threading.Thread(target=work, args=(t,)) for t in range(n)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    wall = time.perf_counter() - t0
    return {"value": sum(done) / wall, "unit": "rows/s", "cores": n, "kind": "oracle x N cores",
            "sample": f"{sum(done)} rows in {wall:.1f} s, chunks of {k} contexts, one thread per core"}


def cpu_baseline(wl, ctx, x, stride, nq, do_fit):
    """The oracle (single-threaded C) on a bounded sample of the same workload: context chunks
    in order, repeated, for about ten seconds of fitting; then about five seconds of encoding the
    queries that fall into the first chunk of contexts."""
    import numpy as np
    import oracle
    C = wl.num_ctx
    k = max(1, C // 32)
    t_fit, rows_fit, c0, first = 0.0, 0, 0, None
    while t_fit < (10.0 if do_fit else 0.0) or first is None:
        c1 = min(C, c0 + k)
        rows, off, nb = sub_workload(wl, c0, c1)
        t = time.perf_counter()
        ref = oracle.fit_batch(rows, off, nb)
        t_fit += time.perf_counter() - t
        rows_fit += int(wl.m_rows[c0:c1].sum())
        if first is None:
            first = (ref, c1)
        c0 = c1 % C
    out = {"cores": 1, "kind": "oracle"}
    if do_fit:
        out.update(value=rows_fit / t_fit, unit="rows/s",
                   sample=f"oracle fit of {rows_fit} rows: chunks of {k} consecutive contexts of the workload "
                          f"({C} contexts, {wl.total_rows} rows), {t_fit:.1f} s")
        out["parallel"] = oracle_fit_parallel(wl, k)
    if nq:
        ref, cn = first
        sel = np.nonzero(ctx < cn)[0][:200_000]
        xs = x.reshape(nq, stride)[sel].reshape(-1)
        t0, reps = time.perf_counter(), 0
        while True:
            oracle.encode_batch(ref, ctx[sel], xs, stride)
            reps += 1
            if time.perf_counter() - t0 > 5.0:
                break
        wps = len(sel) * reps / (time.perf_counter() - t0)
        enc_sample = f"oracle encode of {len(sel)} queries of the workload (those on contexts 0..{cn - 1}), {reps} repetitions"
        if do_fit:
            out["encode_words_per_s"] = wps
            out["sample"] += "; " + enc_sample
        else:
            out.update(value=wps, unit="words/s", sample=enc_sample)
    return out


def bench_stream(args):
    """Time the Eq. 1 row builder or the word merge alone on seeded data already in HBM."""
    import numpy as np
    import torch
    from paper_2608_20532_amd import f2gpu
    count, k, desc = STREAM_WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(0)
    g = torch.Generator(device=dev)
    g.manual_seed(0xF2A50010)
    rnd = lambda n: torch.randint(-2 ** 63, 2 ** 63 - 1, (n,), generator=g, device=dev, dtype=torch.int64)
    stream = torch.cuda.current_stream()
    ALL = 2 ** 64 - 1
    mask = (0, (1 << 58) | (1 << 60))
    if args.workload == "vectorize":
        vals, y = rnd(count * k), rnd(2 * count)
        out = torch.empty(count * (k + 3), dtype=torch.int64, device=dev)
        keep = (ALL, ALL & ~mask[1])
        call = lambda: f2gpu.f2_vectorize_rows(vals, y, count, k, keep, out, stream.cuda_stream)
        nbytes = count * (8 * k + 16 + 8 * (k + 3))
        unit, kernel = "rows/s", "f2_vectorize_rows"
    else:
        words, field, state = rnd(2 * count), rnd(count) & ((1 << 17) - 1), rnd(2 * count)
        out = torch.empty(2 * count, dtype=torch.int64, device=dev)
        call = lambda: f2gpu.f2_merge_words(words, field, 105, 17, mask, state, count, out, stream.cuda_stream)
        nbytes = count * (16 + 8 + 16 + 16)
        unit, kernel = "words/s", "f2_merge_words"
    for _ in range(args.warmup):
        assert call() == 0
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    w0 = time.perf_counter()
    for e in ev:
        e[0].record(stream)
        assert call() == 0
        e[1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    gbps = nbytes / (ms * 1e-3) / 1e9
    cpu = None
    if not args.no_cpu_baseline:
        from oracle import words as W
        rngc = np.random.default_rng(0)
        t0, done = time.perf_counter(), 0
        while time.perf_counter() - t0 < 10.0:
            if args.workload == "vectorize":
                v = rngc.integers(0, 2 ** 63, size=1000 * k, dtype=np.uint64)
                yy = rngc.integers(0, 2 ** 63, size=2000, dtype=np.uint64)
                W.vectorize_rows(v, k, yy, (ALL, ALL & ~mask[1]))
                done += 1000
            else:
                ww = rngc.integers(0, 2 ** 63, size=20000, dtype=np.uint64)
                ff = rngc.integers(0, 2 ** 17, size=10000, dtype=np.uint64)
                W.merge_words(ww, ff, 105, 17, mask, rngc.integers(0, 2 ** 63, size=20000, dtype=np.uint64))
                done += 10000
        cpu = {"value": done / (time.perf_counter() - t0), "unit": unit, "cores": 1, "kind": "oracle",
               "sample": f"oracle ({'rows' if k else 'words'} one at a time in Python integers) on {done} seeded "
                         f"items of the same shape, about 10 s"}
    print(json.dumps({
        "metric": "GF(2) fit rows/sec and encoded words/sec on 1 MI355X; % of HBM/int-op roofline",
        "value": count / (ms * 1e-3), "unit": unit, "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": 1e3 * wall / args.steps, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "u64", "data": "synthetic",
        "config": {"workload": desc, "name": args.workload, "items": count},
        "roofline": measured_traffic(args.workload, args.workload,
                                     {"bound": "hbm", "kernel": kernel, "achieved": gbps, "peak": HBM_PEAK_GBS,
                                      "unit": "GB/s", "frac": gbps / HBM_PEAK_GBS, "algorithmic_bytes": nbytes,
                                      "avg_ms": ms}),
        "cpu_baseline": cpu,
    }), flush=True)


def bench_pool(args):
    """Time f2_pool_bases: shard bases of every context pooled back into one context each."""
    import numpy as np
    import torch
    import synth
    from paper_2608_20532_amd import f2gpu
    C0, parts, desc = STREAM_WORKLOADS["pool"]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(0)
    wl0 = synth.fit_workload(3, num_ctx=C0)
    n_bits, rows_list = [], []
    for c in range(C0):
        n = int(wl0.n_bits[c])
        W = (n + 64) // 64 + 2
        for part in np.array_split(wl0.rows[wl0.row_off[c]:wl0.row_off[c + 1]].reshape(-1, W), parts):
            n_bits.append(n)
            rows_list.append(part)
    wl = synth.custom_workload(n_bits, [len(r) for r in rows_list], rows_list)
    to_dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int64) if a.dtype == np.uint64 else a).to(dev)
    members_model = f2gpu.fit(to_dev(wl.rows), to_dev(wl.row_off), wl.n_bits)
    pool_off = to_dev(np.arange(0, parts * C0 + 1, parts, dtype=np.int64))
    members = to_dev(np.arange(parts * C0, dtype=np.int32))
    pooled = f2gpu.Model(wl0.n_bits, device=dev)
    flags = torch.zeros(C0, dtype=torch.int32, device=dev)
    nb = f2gpu.f2_pool_workspace_bytes(members_model, C0)
    ws = f2gpu.workspace(nb, dev)
    stream = torch.cuda.current_stream()
    call = lambda: f2gpu.f2_pool_bases(members_model, None, pool_off, members, parts * C0, pooled, flags, ws, nb,
                                       stream.cuda_stream)
    for _ in range(args.warmup):
        assert call() == 0
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    w0 = time.perf_counter()
    for e in ev:
        e[0].record(stream)
        assert call() == 0
        e[1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    mrank = members_model.rank.cpu().numpy()[:parts * C0].astype(np.int64)
    prank = pooled.rank.cpu().numpy()[:C0].astype(np.int64)
    Wm = (np.asarray(n_bits, np.int64) + 64) // 64 + 2
    Wp = (wl0.n_bits.astype(np.int64) + 64) // 64 + 2
    rows_in = int(mrank.sum())
    nbytes = int((mrank * Wm * 8).sum() + (prank * Wp * 8).sum() + 4 * prank.sum() +
                 (16 * (wl0.n_bits.astype(np.int64) + 1)).sum() + 20 * C0 + 4 * parts * C0 + 8 * (C0 + 1))
    gbps = nbytes / (ms * 1e-3) / 1e9
    shared = int((flags.cpu().numpy()[:C0] == f2gpu.POOL_SHARED).sum())
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        from oracle import pool as PL
        ref = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
        t0, done, k = time.perf_counter(), 0, 0
        while time.perf_counter() - t0 < 10.0 and k < C0:
            k1 = min(C0, k + 2000)
            mem = np.arange(parts * k, parts * k1)
            PL.pool_bases(ref, np.concatenate([[0], np.cumsum(np.full(k1 - k, parts))]), mem, wl0.n_bits[k:k1])
            done += int(mrank[parts * k:parts * k1].sum())
            k = k1
        cpu = {"value": done / (time.perf_counter() - t0), "unit": "basis rows/s", "cores": 1, "kind": "oracle",
               "sample": f"oracle pooling of the first {k} pools ({done} member basis rows), about 10 s"}
    print(json.dumps({
        "metric": "GF(2) fit rows/sec and encoded words/sec on 1 MI355X; % of HBM/int-op roofline",
        "value": rows_in / (ms * 1e-3), "unit": "basis rows/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": 1e3 * wall / args.steps, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": {"workload": desc, "name": "pool", "pools": C0, "member_contexts": parts * C0,
                   "member_basis_rows": rows_in, "shared_pools": shared},
        "roofline": measured_traffic("pool", "pool",
                                     {"bound": "hbm", "kernel": "f2_pool_bases", "achieved": gbps, "peak": HBM_PEAK_GBS,
                                      "unit": "GB/s", "frac": gbps / HBM_PEAK_GBS, "algorithmic_bytes": nbytes,
                                      "avg_ms": ms}),
        "cpu_baseline": cpu,
    }), flush=True)


def bench_group(args):
    """Time f2_group_rows: the rows of the 80,000-context fit workload interleaved at
    random (each context's order kept), grouped back by context."""
    import numpy as np
    import torch
    import synth
    from paper_2608_20532_amd import f2gpu
    _, _, desc = STREAM_WORKLOADS["group"]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(0)
    wl = synth.fit_workload(3)
    W = (wl.n_bits.astype(np.int64) + 64) // 64 + 2
    S = int(W.max())
    rng = np.random.default_rng(0xF2A50006)
    ids = np.repeat(np.arange(wl.num_ctx, dtype=np.int32), wl.m_rows)
    ids = ids[rng.permutation(len(ids))]
    start = np.concatenate([[0], np.cumsum(wl.m_rows)[:-1]])
    order = np.argsort(ids, kind="stable")
    rank = np.empty(len(ids), np.int64)
    rank[order] = np.arange(len(ids)) - start[ids[order]]
    rows = np.zeros((len(ids), S), np.uint64)
    src = wl.row_off[ids] + rank * W[ids]
    for w in range(S):
        ok = w < W[ids]
        rows[ok, w] = wl.rows[src[ok] + w]
    R, C = len(ids), wl.num_ctx
    to_dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int64) if a.dtype == np.uint64 else a).to(dev)
    ids_d, rows_d, nb_d = to_dev(ids), to_dev(rows.reshape(-1)), to_dev(wl.n_bits.astype(np.int32))
    out = torch.empty(R * S, dtype=torch.int64, device=dev)
    off = torch.empty(C + 1, dtype=torch.int64, device=dev)
    drop = torch.empty(1, dtype=torch.int64, device=dev)
    nb = f2gpu.f2_group_workspace_bytes(C, R)
    ws = f2gpu.workspace(nb, dev)
    stream = torch.cuda.current_stream()
    call = lambda: f2gpu.f2_group_rows(ids_d, rows_d, S, R, nb_d, C, out, R * S, off, drop, ws, nb,
                                       stream.cuda_stream)
    for _ in range(args.warmup):
        assert call() == 0
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]
    w0 = time.perf_counter()
    for e in ev:
        e[0].record(stream)
        assert call() == 0
        e[1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    assert np.array_equal(off.cpu().numpy(), wl.row_off)
    # algorithmic bytes: each row's id and its fw + 2 words read, the words written, the offsets
    nbytes = int(4 * R + 16 * int((W * wl.m_rows).sum()) + 8 * (C + 1))
    gbps = nbytes / (ms * 1e-3) / 1e9
    cpu = None
    if not args.no_cpu_baseline:
        from oracle import group as G
        k = min(R, 400_000)
        t0 = time.perf_counter()
        G.group_rows(ids[:k], rows[:k], S, wl.n_bits)
        cpu = {"value": k / (time.perf_counter() - t0), "unit": "rows/s", "cores": 1, "kind": "oracle",
               "sample": f"oracle grouping of the first {k} rows of the stream"}
    print(json.dumps({
        "metric": "GF(2) fit rows/sec and encoded words/sec on 1 MI355X; % of HBM/int-op roofline",
        "value": R / (ms * 1e-3), "unit": "rows/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": 1e3 * wall / args.steps, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u64", "data": "synthetic",
        "config": {"workload": desc, "name": "group", "rows": R, "contexts": C, "stride_words": S},
        "roofline": measured_traffic("group", "group",
                                     {"bound": "hbm", "kernel": "f2_group_rows", "achieved": gbps, "peak": HBM_PEAK_GBS,
                                      "unit": "GB/s", "frac": gbps / HBM_PEAK_GBS, "algorithmic_bytes": nbytes,
                                      "avg_ms": ms}),
        "cpu_baseline": cpu,
    }), flush=True)


def host_cpu():
    """CPU model and core counts of the host the oracle baseline runs on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return {"cpu_model": model, "nproc": usable, "cpu_count": os.cpu_count()}


def measured_ceilings(stream):
    """Achievable rates from the probe library: a streaming copy (GB/s, bytes read plus
    written), a run of independent 32-bit bitwise VALU instructions (T lane ops/s), and
    scattered 32-byte reads and 16-byte writes (G accesses/s)."""
    import numpy as np
    import torch
    from paper_2608_20532_amd import f2probe
    dev = torch.device("cuda:0")
    words = (1 << 31) // 8  # 2 GiB each way
    src = torch.ones(words, dtype=torch.int64, device=dev)
    dst = torch.empty_like(src)
    out = torch.empty(256 * 256 * 8, dtype=torch.int32, device=dev)
    sp = stream.cuda_stream

    def timed(call, reps):
        for _ in range(2):
            assert call() == 0
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ms = []
        for _ in range(reps):
            ev[0].record(stream)
            assert call() == 0
            ev[1].record(stream)
            torch.cuda.synchronize()
            ms.append(ev[0].elapsed_time(ev[1]))
        return float(np.median(ms))

    copy_ms = timed(lambda: f2probe.f2probe_copy(src, dst, words, sp), 10)
    assert bool(torch.equal(src[:1024], dst[:1024]))
    blocks, iters = 256 * 8 * 4, 4096
    res = {"copy_GBps": 2 * 8 * words / (copy_ms * 1e-3) / 1e9, "copy_bytes": 2 * 8 * words}
    for op, name in ((0, "xor_Tops"), (1, "bitop3_Tops")):
        ms = timed(lambda: f2probe.f2probe_bitops(out, blocks, iters, op, sp), 5)
        res[name] = blocks * 256 * iters * 16 / (ms * 1e-3) / 1e12
    # scattered accesses: 32-byte reads over 2 GiB, 16-byte writes over 128 MiB (inside
    # the last-level cache) and over 2 GiB; G accesses/s
    sblocks, per = 8192, 16
    acc = sblocks * 256 * per
    sout = torch.empty(sblocks * 256, dtype=torch.int64, device=dev)
    for name, buf, nb, op in (("scatter_read_Gps", src, 8 * words, 0), ("scatter_write_128MiB_Gps", dst, 1 << 27, 1),
                              ("scatter_write_Gps", dst, 8 * words, 1)):
        ms = timed(lambda: f2probe.f2probe_scatter(buf, nb, sblocks, per, op, sout, sp), 5)
        res[name] = acc / (ms * 1e-3) / 1e9
    del src, dst, out, sout
    torch.cuda.empty_cache()
    return res


def time_fit_encode(f2gpu, wl, ctx, x, stride, nq, do_fit, steps, warmup, stream):
    """Upload a workload, then W untimed and K timed steps (fit then encode); returns the
    per-phase averages of HIP events recorded on the stream the library enqueues on."""
    import numpy as np
    import torch
    dev = torch.device("cuda:0")
    to_dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int64) if a.dtype == np.uint64 else a).to(dev)
    rows_d, off_d = to_dev(wl.rows), to_dev(wl.row_off)
    model = f2gpu.Model(wl.n_bits, device=dev)
    fws = f2gpu.f2_fit_workspace_bytes(model.num_ctx)
    fit_ws = f2gpu.workspace(fws, dev)
    if nq:
        ctx_d, x_d = to_dev(ctx), to_dev(x)
        words = torch.empty((nq, 2), dtype=torch.int64, device=dev)
        qf = torch.empty(nq, dtype=torch.uint8, device=dev)
        ews = f2gpu.f2_encode_workspace_bytes(model, nq)
        enc_ws = f2gpu.workspace(ews, dev)
    sptr = stream.cuda_stream

    def check(st, what):
        if st != 0:
            raise RuntimeError(f"{what}: {f2gpu.f2_status_string(st)}")

    def fit():
        check(f2gpu.f2_fit_batch(rows_d, wl.rows.size, off_d, model, fit_ws, fws, sptr), "fit")

    def encode():
        check(f2gpu.f2_encode_batch(model, ctx_d, x_d, stride, nq, words, qf, enc_ws, ews, sptr), "encode")

    if not do_fit:
        fit()
    for _ in range(warmup):
        if do_fit:
            fit()
        if nq:
            encode()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for k in range(steps):
        ev[k][0].record(stream)
        if do_fit:
            fit()
        ev[k][1].record(stream)
        if nq:
            encode()
        ev[k][2].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    fit_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev])) if do_fit else 0.0
    enc_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev])) if nq else 0.0
    rank = model.rank.cpu().numpy()[:wl.num_ctx]
    del rows_d, off_d, model, fit_ws
    if nq:
        del ctx_d, x_d, words, qf, enc_ws
    torch.cuda.empty_cache()
    return fit_ms, enc_ms, 1e3 * wall / steps, rank


def phases_and_roofline(name, wl, nq, stride, do_fit, fit_ms, enc_ms, rank, ceil):
    """Per-phase algorithmic rates and the roofline object of the phase (library call) that
    takes longer: wide-context fits against the integer issue rate, the rest against HBM."""
    phases = {}
    if do_fit:
        fb = fit_bytes(wl, rank)
        phases["fit"] = {"call": "f2_fit_batch", "ms": fit_ms, "bytes": fb, "GBps": fb / (fit_ms * 1e-3) / 1e9}
    if nq:
        eb = encode_bytes(wl, nq, stride)
        phases["encode"] = {"call": "f2_encode_batch", "ms": enc_ms, "bytes": eb,
                            "GBps": eb / (enc_ms * 1e-3) / 1e9}
    dom = max(phases, key=lambda k: phases[k]["ms"])
    traffic, why = load_traffic(name)
    tr = traffic.get(dom) if traffic else None
    if name == "recipe4":
        # wide contexts: the blocked elimination is bound by integer VALU work, not by HBM
        ops = fit_int_ops(wl, rank)
        tops = ops / (fit_ms * 1e-3) / 1e12
        phases["fit"]["int_ops"] = ops
        roof = {"bound": "alu", "kernel": phases[dom]["call"], "achieved": tops, "peak": INT_PEAK_TOPS,
                "unit": "Tops/s (32-bit integer lane ops)", "frac": tops / INT_PEAK_TOPS,
                "traffic": tr["bytes"] if tr else None, "algorithmic_ops": ops,
                "algorithmic_bytes": phases[dom]["bytes"], "avg_ms": phases[dom]["ms"]}
        if ceil:
            roof["measured_peak"] = ceil["xor_Tops"]
            roof["measured_peak_unit"] = "Tops/s, v_xor_b32 issue (probe)"
            roof["frac_of_measured_peak"] = tops / ceil["xor_Tops"]
    else:
        roof = {"bound": "hbm", "kernel": phases[dom]["call"], "achieved": phases[dom]["GBps"], "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": phases[dom]["GBps"] / HBM_PEAK_GBS,
                "traffic": tr["bytes"] if tr else None,
                "algorithmic_bytes": phases[dom]["bytes"], "avg_ms": phases[dom]["ms"]}
        if ceil:
            roof["measured_peak"] = ceil["copy_GBps"]
            roof["measured_peak_unit"] = "GB/s, streaming copy (probe)"
            roof["frac_of_measured_peak"] = phases[dom]["GBps"] / ceil["copy_GBps"]
            if dom == "encode" and nq >= (1 << 22):
                # a context-grouped encode reads each query's x at a scattered position and
                # writes its word at one: one 32-byte read and one 16-byte write per query
                # at the probes' rates (writes inside the last-level cache: the sort windows)
                floor_ms = 1e3 * nq * (1.0 / (ceil["scatter_read_Gps"] * 1e9) +
                                       1.0 / (ceil["scatter_write_128MiB_Gps"] * 1e9))
                roof["scattered_floor"] = {"ms": floor_ms, "frac": floor_ms / phases[dom]["ms"],
                                           "per_query": "one scattered 32-byte read, one scattered 16-byte write"}
    if tr:
        roof["kernels"] = tr["kernels"]
        # the bytes the counters saw crossing to the fabric, at the call's measured time
        roof["traffic_GBps"] = tr["bytes"] / (phases[dom]["ms"] * 1e-3) / 1e9
        roof["traffic_over_algorithmic"] = tr["bytes"] / phases[dom]["bytes"]
        if ceil:
            roof["traffic_frac_of_measured_peak"] = roof["traffic_GBps"] / ceil["copy_GBps"]
    else:
        roof["traffic_note"] = why or f"no counters for the {dom} phase of this workload"
    return phases, roof


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="step", choices=sorted(WORKLOADS) + sorted(STREAM_WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="default step only: skip the other configurations reported beside it")
    ap.add_argument("--no-ceilings", action="store_true", help="skip the copy and integer-issue probes")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs and reports one GPU only (contexts are independent and would shard across "
              "GPUs with no exchange); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.copy_calibration_mb:
        # a plain copy of known size: its FETCH_SIZE / WRITE_SIZE readings give the
        # counter-to-bytes factors used for the roofline traffic figure
        nbytes = args.copy_calibration_mb << 20
        src = torch.ones(nbytes // 8, dtype=torch.int64, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": nbytes, "copies": 3}), flush=True)
        return

    if args.workload == "group":
        bench_group(args)
        return
    if args.workload == "pool":
        bench_pool(args)
        return
    if args.workload in STREAM_WORKLOADS:
        bench_stream(args)
        return

    import synth
    from paper_2608_20532_amd import f2gpu

    recipe, num_ctx, nq, stride, frac, zipf, desc = WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()  # the library enqueues every kernel on this stream
    t0 = time.time()
    wl = synth.fit_workload(recipe, num_ctx=num_ctx)
    ctx = x = None
    if nq:
        ctx, x, _ = synth.queries(wl, nq, stride, frac, zipf)
    print(f"[bench] generated {args.workload}: {wl.num_ctx} contexts, {wl.total_rows} rows, {nq} queries "
          f"in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
    do_fit = args.workload != "recipe5"
    fit_ms, enc_ms, step_ms, rank = time_fit_encode(f2gpu, wl, ctx, x, stride, nq, do_fit, args.steps, args.warmup,
                                                    stream)
    print(f"[bench] timed {args.steps} steps: fit {fit_ms:.4f} ms, encode {enc_ms:.4f} ms, wall/step {step_ms:.4f} ms",
          file=sys.stderr, flush=True)
    ceil = None
    if not args.no_ceilings:
        ceil = measured_ceilings(stream)
        print(f"[bench] ceilings: copy {ceil['copy_GBps']:.0f} GB/s, xor {ceil['xor_Tops']:.1f} T/s, "
              f"bitop3 {ceil['bitop3_Tops']:.1f} T/s, scattered 32-byte reads {ceil['scatter_read_Gps']:.1f} G/s, "
              f"16-byte writes {ceil['scatter_write_128MiB_Gps']:.1f} G/s over 128 MiB and "
              f"{ceil['scatter_write_Gps']:.1f} G/s over 2 GiB", file=sys.stderr, flush=True)
    phases, roof = phases_and_roofline(args.workload, wl, nq, stride, do_fit, fit_ms, enc_ms, rank, ceil)

    extras = {}
    if args.workload == "step" and not args.no_extras:
        # the other configurations, timed the same way (no oracle baseline): the wide-context
        # fit against the integer issue rate, the small ones against HBM
        for name in ("recipe4", "recipe2", "recipe1"):
            r2, c2, nq2, s2, f2_, z2, d2 = WORKLOADS[name]
            wl2 = synth.fit_workload(r2, num_ctx=c2)
            cx2 = xx2 = None
            if nq2:
                cx2, xx2, _ = synth.queries(wl2, nq2, s2, f2_, z2)
            fm, em, sm, rk = time_fit_encode(f2gpu, wl2, cx2, xx2, s2, nq2, True, args.steps, args.warmup, stream)
            ph2, rf2 = phases_and_roofline(name, wl2, nq2, s2, True, fm, em, rk, ceil)
            extras[name] = {"workload": d2, "fit_rows_per_s": wl2.total_rows / (fm * 1e-3),
                            "encode_words_per_s": nq2 / (em * 1e-3) if nq2 else None, "ms_per_step": sm,
                            "phases": ph2, "roofline": rf2}
            print(f"[bench] {name}: fit {fm:.4f} ms, encode {em:.4f} ms", file=sys.stderr, flush=True)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, ctx, x, stride, nq, do_fit)
        cpu.update(host_cpu())
    rows_per_s = wl.total_rows / (fit_ms * 1e-3) if do_fit else None
    words_per_s = nq / (enc_ms * 1e-3) if nq else None
    out = {
        "metric": "GF(2) fit rows/sec and encoded words/sec on 1 MI355X; % of HBM/int-op roofline",
        "value": rows_per_s if do_fit else words_per_s,
        "unit": "rows/s" if do_fit else "words/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": desc, "name": args.workload, "contexts": wl.num_ctx, "rows": wl.total_rows,
                   "queries": nq, "query_stride_words": stride, "fit_in_step": do_fit},
        "fit_rows_per_s": rows_per_s,
        "encode_words_per_s": words_per_s,
        "phases": phases,
        "roofline": roof,
        "measured_ceilings": ceil,
        "cpu_baseline": cpu,
    }
    if extras:
        out["other_configs"] = extras
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
