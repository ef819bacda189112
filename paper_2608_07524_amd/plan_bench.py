"""Host latency of dcp_plan on the text-LM workload: 1,000 packed batches
(log-normal lengths, median 2048, sigma 1, packed to <= 262,144 tokens)
planned in calls of 8 and of 32 batches, each call timed on its own.

    python -m paper_2608_07524_amd.plan_bench [--reps 20]

The cost table is analytic (the planner's work does not depend on the
measured values): one row per power of two 128 .. 131072, attention-like
quadratic times plus a linear term, the Transformer-1D shape (42 layers,
hidden 3072, 48 heads), 288 GiB.  Arguments are marshalled before the clock
starts; times include the ctypes call itself (a no-op library call is timed
alongside for scale).  Needs no GPU.
"""

from __future__ import annotations

import argparse
import json
import sys
import time

import numpy as np

from . import _native as N
from . import inputs as I


def table_rows():
    rows = []
    for e in range(7, 18):
        s = 1 << e
        t_f = 20_000 + 180 * s + (s * s) // 4000
        rows.append((s, t_f, int(2.5 * t_f), 34 * 3072 * s, 2 * 3072 * s))
    return rows


def _prepared(lib, seqs, offs, rows, mode):
    """dcp_plan with every argument marshalled up front: the returned
    closure makes only the native call."""
    import ctypes as C
    o, keep = N._plan_opts(lib, dict(n_heads=48, hidden=3072, mode=mode))
    table, crow = N._cost_table(rows, 42, 0, 22 << 30)
    lens, offs_a, nb = N._batches(seqs, offs, None)
    i32 = lambda: (C.c_int32 * nb)()
    bufs = [i32(), i32(), i32(), i32(), (C.c_uint8 * (nb * 42))(), (C.c_int64 * nb)(), (C.c_int64 * nb)()]
    out = N.PlanOutC(*bufs, 0, 0)
    args = (lens.ctypes.data_as(C.POINTER(C.c_int64)), int(lens.size), offs_a.ctypes.data_as(C.POINTER(C.c_int32)),
            nb, C.byref(table), 288 << 30, C.byref(o), C.byref(out))

    def call():
        _alive = (keep, crow, lens, offs_a, bufs)  # noqa: F841 (buffers the pointers refer to)
        return lib.dcp_plan(*args)
    return call


def main(argv=None):
    ap = argparse.ArgumentParser(description="dcp_plan host latency")
    ap.add_argument("--reps", type=int, default=20)
    args = ap.parse_args(argv)
    lib = N.load()
    rows = table_rows()
    packs = I.text_packs(np.random.default_rng(0), 1000)
    out = {}
    for mode_name, mode in (("DCP-intra", N.PLAN_INTRA), ("DCP-inter", N.PLAN_INTER)):
        for group in (8, 32):
            times = []
            for _ in range(args.reps):
                for g0 in range(0, 1000, group):
                    batch = packs[g0:g0 + group]
                    seqs = [s for p in batch for s in p.lengths]
                    offs = np.concatenate([[0], np.cumsum([len(p.lengths) for p in batch])]).tolist()
                    call = _prepared(lib, seqs, offs, rows, mode)
                    t0 = time.perf_counter_ns()
                    st = call()
                    times.append(time.perf_counter_ns() - t0)
                    if st != N.DCP_OK:
                        raise N.DCPError(st, N.last_error())
            t = np.array(times) / 1e3
            out[f"{mode_name}, {group} batches per call"] = {
                "calls": int(t.size), "p50_us": float(np.percentile(t, 50)), "p99_us": float(np.percentile(t, 99)),
                "max_us": float(t.max())}
    noop = []
    for _ in range(2000):
        t0 = time.perf_counter_ns()
        lib.dcp_version()
        noop.append(time.perf_counter_ns() - t0)
    out["no-op library call (ctypes)"] = {"p50_us": float(np.percentile(np.array(noop) / 1e3, 50))}
    print(json.dumps(out, indent=1))
    return out


if __name__ == "__main__":
    main(sys.argv[1:])
