"""Measured per-length cost table (dcp_profile_cost, Sec. 3.5) as a
markdown table, with the attention throughput each row implies.

    python -m paper_2608_07524_amd.cost_table --heads 2 --head-dim 128 --min 1024 --max 262144 [--causal]

One sequence of each power-of-two length in [min, max]; t_f and t_b are the
median forward and backward times of the library's attention over it (no
per-token terms).  TFLOP/s counts 4 * pairs * H * D forward and 10 * pairs
* H * D backward over the valid (query, key) pairs.
"""

from __future__ import annotations

import argparse
import json
import sys

from . import _native as N


def main(argv=None):
    ap = argparse.ArgumentParser(description="measured per-length attention cost rows")
    ap.add_argument("--heads", type=int, required=True)
    ap.add_argument("--head-dim", type=int, required=True)
    ap.add_argument("--min", type=int, default=1024)
    ap.add_argument("--max", type=int, default=262144)
    ap.add_argument("--causal", action="store_true")
    ap.add_argument("--reps", type=int, default=5)
    ap.add_argument("--md", default=None)
    args = ap.parse_args(argv)
    import torch
    if not torch.cuda.is_available():  # (initialises the device before the library's first call)
        raise SystemExit("needs a GPU")
    N.load()
    lengths = []
    s = args.min
    while s <= args.max:
        lengths.append(s)
        s *= 2
    rows = N.profile_cost(lengths, args.heads, args.head_dim, causal=args.causal, warmup=2, reps=args.reps)
    HD = args.heads * args.head_dim
    lines = ["| length | t_f (ms) | t_b (ms) | forward TFLOP/s | backward TFLOP/s |", "|---|---|---|---|---|"]
    out = []
    for r in rows:
        s = r.seq_len
        pairs = s * (s + 1) // 2 if args.causal else s * s
        tf, tb = r.t_f_ns / 1e6, r.t_b_ns / 1e6
        ff, fb = 4 * pairs * HD / (r.t_f_ns * 1e-9) / 1e12, 10 * pairs * HD / (r.t_b_ns * 1e-9) / 1e12
        out.append({"seq_len": s, "t_f_ns": r.t_f_ns, "t_b_ns": r.t_b_ns, "fwd_tflops": ff, "bwd_tflops": fb})
        lines.append(f"| {s} | {tf:.3f} | {tb:.3f} | {ff:.0f} | {fb:.0f} |")
    print(json.dumps(out), flush=True)
    if args.md:
        with open(args.md, "w") as f:
            f.write("\n".join(lines) + "\n")
    return out


if __name__ == "__main__":
    main(sys.argv[1:])
