"""Benchmark of the DCP hot path on one MI355X: packed varlen attention
forward + backward over a synthetic video-DiT short-mix batch.

    python bench.py [--steps K] [--warmup W] [--workload NAME]

A step is one forward and one backward pass of the whole packed batch
(inputs already resident in HBM).  Prints ONE JSON line with the throughput
in TFLOP/s counted over valid block-diagonal (query, key) pairs
(fwd 4*pairs*H*D + bwd 10*pairs*H*D), the roofline of the dominant kernel
timed live with HIP events, the padded-bucket baseline (same kernels, every
sequence zero-padded to the batch maximum, still credited with the unpadded
pairs) and the float64 oracle timed on a bounded sample on the host cores.
"""

from __future__ import annotations

import argparse
import ctypes
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix-core peak
HBM_PEAK_GBS = 8000.0

# HBM bytes per launch of the dK/dV kernel from two rocprofv3 --pmc passes
# (FETCH_SIZE x 2.000 and WRITE_SIZE x 1.000, the scales a plain device copy
# of known size reads), per workload; valid only for the kernel sources
# whose hash is recorded with them.
MEASURED_TRAFFIC = {
    "video_short": {"sources_sha256_16": "ee662c9eea106fa5", "bytes": (1127681.9 * 2.0 + 691200.5 * 1.0) * 1024},
    "video2d_temporal": {"sources_sha256_16": "ee662c9eea106fa5",
                         "bytes": (1069822.7 * 2.0 + 986398.7 * 1.0) * 1024},
}
KERNEL_SOURCES = ("attn_bwd.hip", "attn_common.h", "attn_launch.h")


def kernel_sources_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_07524_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload_name: str):
    m = MEASURED_TRAFFIC.get(workload_name)
    if m is None or m["sources_sha256_16"] != kernel_sources_hash():
        return None
    return m["bytes"]


def workload(name: str, seed: int = 0):
    from paper_2608_07524_amd import inputs as I
    rng = np.random.default_rng(seed)
    if name == "video_short":
        return I.video_short_mix(rng), rng
    if name == "tiny":
        return I.tiny(), rng
    if name == "video_long":
        return I.video_long_tail_packs(rng, n_packs=1)[0], rng
    if name == "ulysses128k":
        return I.ulysses_shard(131072), rng
    if name == "ulysses256k":
        return I.ulysses_shard(262144), rng
    if name == "text":
        return I.text_packs(rng, 1)[0], rng
    if name in ("video2d_spatial", "video2d_temporal"):
        return I.video_2d_pack(rng, name.split("_")[1]), rng
    raise SystemExit(f"unknown workload {name}")


def pairs_of(lengths, causal):
    s = np.asarray(lengths, dtype=np.int64)
    return int(np.sum(s * (s + 1) // 2)) if causal else int(np.sum(s * s))


def device_tensors(torch, rng, T, H, D):
    """q, k, v, dO: bf16 N(0,1) drawn on the host from the seeded stream."""
    from paper_2608_07524_amd import inputs as I
    out = []
    for b in I.tensors(rng, T, H, D):
        out.append(torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).cuda())
    return out


class HipEvents:
    """Raw hipEvent_t handles (the library records them on the stream the
    kernels run on)."""

    def __init__(self, n):
        self.hip = ctypes.CDLL(self._loaded_runtime())
        self.ev = []
        for _ in range(n):
            e = ctypes.c_void_p()
            if self.hip.hipEventCreate(ctypes.byref(e)) != 0:
                raise RuntimeError("hipEventCreate failed")
            self.ev.append(e.value)

    @staticmethod
    def _loaded_runtime():
        # the HIP runtime this process already uses (torch's copy), so the
        # handles belong to the same runtime as the library's streams
        with open("/proc/self/maps") as f:
            for line in f:
                if "libamdhip64.so" in line:
                    return line.split()[-1]
        return "libamdhip64.so"

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        if self.hip.hipEventElapsedTime(ctypes.byref(ms), ctypes.c_void_p(self.ev[a]), ctypes.c_void_p(self.ev[b])):
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def close(self):
        for e in self.ev:
            self.hip.hipEventDestroy(ctypes.c_void_p(e))


def time_steps(torch, P, call, steps, warmup):
    """Average ms per step plus the live-event averages of the main forward
    and backward kernels over the timed steps."""
    for _ in range(warmup):
        call.step()
    torch.cuda.synchronize()
    ev = HipEvents(4 * steps)
    t0 = time.perf_counter()
    for i in range(steps):
        P.set_kernel_events(ev.ev[4 * i], ev.ev[4 * i + 1])
        call.fwd()
        P.set_kernel_events(ev.ev[4 * i + 2], ev.ev[4 * i + 3])
        call.bwd()
    P.set_kernel_events(None, None)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps * 1e3
    fwd_ms = sum(ev.elapsed_ms(4 * i, 4 * i + 1) for i in range(steps)) / steps
    bwd_ms = sum(ev.elapsed_ms(4 * i + 2, 4 * i + 3) for i in range(steps)) / steps
    ev.close()
    return wall, fwd_ms, bwd_ms


def cpu_baseline(w, rng_seed: int, budget_s: float = 12.0):
    """float64 oracle (forward + backward) on whole sequences of the same
    batch, taken in order until the time budget is spent."""
    from oracle import attention as A
    from paper_2608_07524_amd import inputs as I
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    rng = np.random.default_rng(rng_seed + 1)
    done_pairs = 0
    done = []
    t_total = 0.0
    for s in w.lengths:
        if t_total > budget_s:
            break
        q, k, v, do = (I.bf16_to_f64(b) for b in I.tensors(rng, s, w.n_heads, w.head_dim))
        cu = [0, s]
        t0 = time.perf_counter()
        A.attention_forward(q, k, v, cu, w.scale, w.causal)
        A.attention_backward(do, q, k, v, cu, w.scale, w.causal)
        t_total += time.perf_counter() - t0
        done_pairs += pairs_of([s], w.causal)
        done.append(s)
    flops = 14.0 * done_pairs * w.n_heads * w.head_dim
    return {"value": flops / t_total / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"float64 fwd+bwd of {len(done)} whole sequences {done} of the same batch "
                      f"({w.n_heads} heads, D={w.head_dim}) in {t_total:.1f} s"}


def dkdv_bytes(cu, H: int, D: int) -> float:
    """Algorithmic HBM bytes of the dK/dV pass: Q, K, V, dO read and dK, dV
    written once (bf16), LSE and Delta read once (fp32), over the rows of
    the sequences."""
    rows = int(cu[-1])
    return 6.0 * rows * H * D * 2 + 2.0 * rows * H * 4


def window_dq_part(P, cu, H: int, D: int, causal: bool):
    """(rows, pairs) of the sequences the dK/dV pass runs as packed windows
    when that launch also computes their dQ (the library does so up to head
    width 96): their dQ rows are written, and their dQ products run, inside
    the dK/dV pass."""
    if D > 96:
        return 0, 0
    units, n_tiles, _ = P.work_list(cu, H, D, causal, 1)
    win = units[n_tiles:]
    win = win[(win[:, 4] == 0) & (win[:, 3] > 0)]
    cu = np.asarray(cu, dtype=np.int64)
    starts, lens = cu[:-1], np.diff(cu)
    first = np.searchsorted(starts, win[:, 0], side="left")
    last = np.searchsorted(starts, win[:, 0] + win[:, 3], side="left")
    inside = np.zeros(lens.size, dtype=bool)
    for a, b in zip(first, last):
        inside[a:b] = True
    inside &= lens > 0
    return int(lens[inside].sum()), pairs_of(lens[inside].tolist(), causal)


def roofline(flop: float, nbytes: float, ms: float, traffic) -> dict:
    """Roofline of the dK/dV pass: matrix-bound when its arithmetic
    intensity is above the ridge point (bf16 peak / HBM peak), else
    HBM-bound (short sequences: intensity grows with the sequence length)."""
    mfma = flop / nbytes >= BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
    out = {"kernel": "attn_bwd_dkdv_kernel", "flop_per_launch": flop, "bytes_per_launch": nbytes,
           "flop_convention": "8*pairs*H*D (S, dP, dV, dK products) + 2*pairs*H*D over packed windows whose dQ "
                              "the pass computes",
           "bytes_convention": "6*rows*H*D*2 + 2*rows*H*4 (Q, K, V, dO, dK, dV; LSE, Delta) + rows*H*D*2 "
                               "(dQ of those windows)",
           "traffic": traffic,
           "traffic_unit": "bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-scaled)"}
    if mfma:
        a = flop / (ms * 1e-3) / 1e12
        out.update(bound="mfma", achieved=a, peak=BF16_PEAK_TFLOPS, unit="TFLOP/s", frac=a / BF16_PEAK_TFLOPS)
    else:
        a = nbytes / (ms * 1e-3) / 1e9
        out.update(bound="hbm", achieved=a, peak=HBM_PEAK_GBS, unit="GB/s", frac=a / HBM_PEAK_GBS)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="video_short")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-padded", action="store_true")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run one plain device copy of this many MiB (a known-traffic reference for "
                         "HBM byte counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures the single-GPU hot path only: run it with --gpus 1 (one process, one GPU).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_07524_amd as P
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    P.load()

    if args.copy_probe_mib:
        src = torch.empty(args.copy_probe_mib << 20, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    w, rng = workload(args.workload, args.seed)
    H, D, causal = w.n_heads, w.head_dim, w.causal
    T = w.total_tokens
    cu = w.cu_seqlens
    pairs = pairs_of(w.lengths, causal)
    flop_fwd = 4.0 * pairs * H * D
    flop_bwd = 10.0 * pairs * H * D
    q, k, v, do = device_tensors(torch, rng, T, H, D)
    call = P.PreparedAttention(q, k, v, do, cu, w.scale, causal)
    ms, fwd_ms, bwd_ms = time_steps(torch, P, call, args.steps, args.warmup)
    value = (flop_fwd + flop_bwd) / (ms * 1e-3) / 1e12
    # the dK/dV pass forms S, dP, dV and dK: 4 of the 5 backward products
    flop_dkdv = 8.0 * pairs * H * D
    win_rows, win_pairs = window_dq_part(P, cu, H, D, causal)
    dkdv_tflops = flop_dkdv / (bwd_ms * 1e-3) / 1e12
    fwd_tflops = flop_fwd / (fwd_ms * 1e-3) / 1e12

    padded = None
    if not args.no_padded and len(set(w.lengths)) > 1:
        del call
        smax = max(w.lengths)
        n = len(w.lengths)
        qp, kp, vp, dop = (torch.zeros((n * smax, H, D), dtype=torch.bfloat16, device="cuda") for _ in range(4))
        off = 0
        for b, s in enumerate(w.lengths):
            for src, dst in ((q, qp), (k, kp), (v, vp), (do, dop)):
                dst[b * smax:b * smax + s] = src[off:off + s]
            off += s
        cu_p = np.arange(n + 1, dtype=np.int32) * smax
        callp = P.PreparedAttention(qp, kp, vp, dop, cu_p, w.scale, causal)
        ms_p, _, _ = time_steps(torch, P, callp, args.steps, args.warmup)
        padded = {"value": (flop_fwd + flop_bwd) / (ms_p * 1e-3) / 1e12, "ms_per_step": ms_p,
                  "padded_to": smax, "computed_pairs": pairs_of([smax] * n, causal),
                  "note": "same kernels, every sequence zero-padded to the batch maximum; credited with the "
                          "unpadded valid pairs only"}
        del callp, qp, kp, vp, dop

    line = {
        "metric": "varlen attn fwd+bwd TFLOP/s (valid pairs) + % bf16 MFMA peak, 1 MI355X",
        "value": value,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "pct_bf16_peak": 100.0 * value / BF16_PEAK_TFLOPS,
        "config": {"workload": w.name, "n_seqs": len(w.lengths), "total_tokens": T, "heads": H, "head_dim": D,
                   "causal": causal, "valid_pairs": pairs, "flop_per_step": flop_fwd + flop_bwd,
                   "flop_convention": "fwd 4*pairs*H*D + bwd 10*pairs*H*D"},
        "kernels": {"fwd_ms": fwd_ms, "fwd_tflops": fwd_tflops, "bwd_dkdv_ms": bwd_ms, "bwd_dkdv_tflops": dkdv_tflops,
                    "bwd_rest_ms": ms - fwd_ms - bwd_ms},
        "roofline": roofline(flop_dkdv + 2.0 * win_pairs * H * D, dkdv_bytes(cu, H, D) + 2.0 * win_rows * H * D,
                             bwd_ms, measured_traffic(args.workload)),
        "padded_baseline": padded,
        "cpu_baseline": None if args.no_cpu_baseline else cpu_baseline(w, args.seed),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
