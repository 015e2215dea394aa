#!/usr/bin/env python3
"""Benchmark of the GF(2) fit + encode hot path on one MI355X.

A step is one pass of the whole path over one batch of synthetic input that is
already resident in HBM: f2_fit_batch over every context (reduce, classify,
insert, finalize) followed by f2_encode_batch over the query batch against the
model just fitted.  Default workload: 4,096 contexts of widths 16..96 (+1
reserved bit), 2(n+1) rows each (468,656 rows, 13.5 MB), 5% contradictory,
then 1M queries (stride 2 words) with 2% outside the span.

Prints one JSON line.  `value` is fit rows/s over the fit phase of the timed
steps; encode words/s and per-phase figures are reported beside it.  The
roofline object describes the phase that takes longer.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0

WORKLOADS = {
    # name: (fit recipe, num contexts, queries, stride, out-of-span fraction, zipf exponent)
    "recipe2": (2, 4096, 1_000_000, 2, 0.02, 0.0),
    "recipe1": (1, 1, 1000, 1, 0.10, 0.0),
    "recipe3": (3, 80000, 1_000_000, 4, 0.01, 1.1),
    "recipe4": (4, 64, 0, 1, 0.0, 0.0),
    "recipe5": (5, 80000, 100_000_000, 4, 0.01, 1.1),
}


def fit_bytes(wl, rank, W):
    """Algorithmic HBM bytes of one fit: rows, offsets and widths in; basis rows, pivots, maps and scalars out."""
    import numpy as np
    n = wl.n_bits.astype(np.int64)
    rows_in = int(wl.rows.nbytes) + 8 * (wl.num_ctx + 1) + 4 * wl.num_ctx
    out = int((rank.astype(np.int64) * W * 8).sum() + 4 * rank.sum() + (16 * (n + 1)).sum()) + 20 * wl.num_ctx
    return rows_in + out


def encode_bytes(nq, stride, table_bytes):
    """Per query: context id, x words, 128-bit word, flag byte; plus the one-time table build."""
    return nq * (4 + 8 * stride + 16 + 1) + table_bytes


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="recipe2", choices=sorted(WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build measures one GPU only; run with --gpus 1 "
              "(contexts shard across GPUs with no exchange, see the design notes)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_2608_20532_amd import f2gpu

    if args.copy_calibration_mb:
        # plain copy of a known size: its FETCH_SIZE / WRITE_SIZE readings give the
        # counter-to-bytes factor used for the roofline traffic figure
        nbytes = args.copy_calibration_mb << 20
        src = torch.ones(nbytes // 8, dtype=torch.int64, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": nbytes, "copies": 3}), flush=True)
        return

    recipe, num_ctx, nq, stride, frac, zipf = WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    t0 = time.time()
    wl = synth.fit_workload(recipe, num_ctx=num_ctx)
    if nq:
        ctx, x, _ = synth.queries(wl, nq, stride, frac, zipf)
    print(f"[bench] generated {args.workload}: {wl.num_ctx} contexts, {wl.total_rows} rows, {nq} queries "
          f"in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

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
    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream
    do_fit = args.workload != "recipe5"

    def check(st, what):
        if st != 0:
            raise RuntimeError(f"{what}: {f2gpu.f2_status_string(st)}")

    def fit():
        check(f2gpu.f2_fit_batch(rows_d, wl.rows.size, off_d, model, fit_ws, fws, sptr), "fit")

    def encode():
        check(f2gpu.f2_encode_batch(model, ctx_d, x_d, stride, nq, words, qf, enc_ws, ews, sptr), "encode")

    if not do_fit:
        fit()
    for _ in range(args.warmup):
        if do_fit:
            fit()
        if nq:
            encode()
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for k in range(args.steps):
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
    step_ms = 1e3 * wall / args.steps
    print(f"[bench] timed {args.steps} steps: fit {fit_ms:.4f} ms, encode {enc_ms:.4f} ms, wall/step {step_ms:.4f} ms",
          file=sys.stderr, flush=True)

    rank = model.rank.cpu().numpy()[:wl.num_ctx]
    W = (wl.n_bits.astype(np.int64) + 64) // 64 + 2
    fb = fit_bytes(wl, rank, W)
    n = wl.n_bits.astype(np.int64)
    hw = ((n + 1 - rank) + 63) // 64
    table_bytes = int(((n + 1) * (2 + hw) * 8).sum() + (rank * W * 8).sum())
    eb = encode_bytes(nq, stride, table_bytes) if nq else 0
    rows_per_s = wl.total_rows / (fit_ms * 1e-3) if do_fit else None
    words_per_s = nq / (enc_ms * 1e-3) if nq else None
    phases = {}
    if do_fit:
        phases["fit"] = {"ms": fit_ms, "bytes": fb, "GBps": fb / (fit_ms * 1e-3) / 1e9}
    if nq:
        phases["encode"] = {"ms": enc_ms, "bytes": eb, "GBps": eb / (enc_ms * 1e-3) / 1e9}
    dom = max(phases, key=lambda k: phases[k]["ms"])
    ach = phases[dom]["GBps"]

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        # bounded sample: the oracle on the same workload (whole fit for small recipes, else a prefix)
        t = time.perf_counter()
        if do_fit:
            nsub = wl.num_ctx if wl.total_rows <= 2_000_000 else 4000
            sub = wl if nsub == wl.num_ctx else synth.fit_workload(recipe, num_ctx=nsub)
            ref = oracle.fit_batch(sub.rows, sub.row_off, sub.n_bits)
            fit_s = time.perf_counter() - t
            cpu_rows = sub.total_rows / fit_s
            sample = f"oracle fit of {sub.num_ctx} contexts ({sub.total_rows} rows) of the same workload"
            cpu = {"value": cpu_rows, "unit": "rows/s", "cores": 1, "kind": "oracle", "sample": sample}
            if nq:
                qs = min(nq, 200_000)
                ref_full = ref if nsub == wl.num_ctx else oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
                t = time.perf_counter()
                oracle.encode_batch(ref_full, ctx[:qs], x[:qs * stride], stride)
                cpu["encode_words_per_s"] = qs / (time.perf_counter() - t)
                cpu["sample"] += f"; oracle encode of the first {qs} queries"
        else:
            ref = oracle.fit_batch(wl.rows, wl.row_off, wl.n_bits)
            qs = 1_000_000
            t = time.perf_counter()
            oracle.encode_batch(ref, ctx[:qs], x[:qs * stride], stride)
            cpu = {"value": qs / (time.perf_counter() - t), "unit": "words/s", "cores": 1, "kind": "oracle",
                   "sample": f"oracle encode of the first {qs} queries"}

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
        "config": {"workload": args.workload, "contexts": wl.num_ctx, "rows": wl.total_rows, "queries": nq,
                   "query_stride_words": stride, "fit_in_step": do_fit},
        "fit_rows_per_s": rows_per_s,
        "encode_words_per_s": words_per_s,
        "phases": phases,
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": ach / HBM_PEAK_GBS, "traffic": None},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
