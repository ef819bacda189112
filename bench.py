"""Benchmark of the DCP hot path on one MI355X: packed varlen attention
forward + backward on the long-sequence workloads the method balances.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--extras a,b]

A step is one forward and one backward pass of the whole packed batch
(inputs already resident in HBM; the batch's work lists are built and
uploaded once, before timing, through the prepared-batch calls).  Prints ONE
JSON line: the throughput in TFLOP/s counted over valid block-diagonal
(query, key) pairs (fwd 4*pairs*H*D + bwd 10*pairs*H*D) and as a fraction of
the bf16 matrix peak, for the headline workload (default: one device's
Ulysses shard of a 262,144-token sequence, 2 heads of width 128) and, as
extra keys, the causal text pack and the short video mix; the roofline of the
dominant kernel timed live with HIP events; the tile fill (valid pairs over
the pairs in the 32x32 blocks the kernels multiply) and the matrix work the
kernels execute; the padded-bucket baseline of the video mix; the float64
oracle timed on a bounded sample on the host cores; and the plan of the tiny
configuration on a cost table measured on this GPU.
"""

from __future__ import annotations

import argparse
import ctypes
import json
import math
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix-core peak
HBM_PEAK_GBS = 8000.0
METRIC = "varlen attn fwd+bwd TFLOP/s (valid pairs) + % bf16 MFMA peak, 1 MI355X"

# Per workload, from rocprofv3 --pmc passes over `bench.py --workload W`
# (profiles/): HBM bytes per launch of the dK/dV kernel (FETCH_SIZE scaled by
# what the same counter reads for a direct-to-LDS copy of known size,
# WRITE_SIZE by what it reads for that copy's stores) and the bf16 matrix
# flops of the whole step (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512).  Valid only
# for the kernel sources whose hash is recorded with them.
MEASURED = {
    "ulysses256k": {"sources_sha256_16": "80d2e41c985b0cf9", "dkdv_traffic_bytes": 9277695477.7,
                    "mfma_flop_per_step": 316663643766784.0},
    "text": {"sources_sha256_16": "80d2e41c985b0cf9", "dkdv_traffic_bytes": 16165009969.4,
             "mfma_flop_per_step": 64359992655872.0},
}
KERNEL_SOURCES = ("attn_fwd.hip", "attn_bwd.hip", "attn_common.h", "attn_launch.h", "tile_shapes.h")

WORKLOADS = {
    "ulysses256k": "Ulysses SP=8 shard, one 262,144-token sequence, H2 D128",
    "ulysses128k": "Ulysses SP=8 shard, one 131,072-token sequence, H2 D128",
    "text": "text-LM causal pack (log-normal documents to 262,144 tokens), H32 D128",
    "video_short": "video-DiT short mix, 32 clips of 1k-8k tokens, H16 D72",
    "video_long": "video-DiT long-tail pack (<= 131,072 tokens), H16 D72",
    "video2d_spatial": "Transformer-2D spatial pack, H16 D72",
    "video2d_temporal": "Transformer-2D temporal pack, H16 D72",
    "tiny": "tiny pack of 4 sequences (429 tokens), H4 D64",
}


def kernel_sources_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_07524_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured(workload_name: str, key: str):
    m = MEASURED.get(workload_name)
    if m is None or m["sources_sha256_16"] != kernel_sources_hash():
        return None
    return m.get(key)


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
    """Average ms per step (wall clock between two synchronisations) plus the
    live-event averages of the forward kernel and of the dK/dV kernel over
    the timed steps."""
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


# ---------------------------------------------------------------------------
# matrix work the kernels execute

def padded_width(D: int) -> int:
    """Width the products run over: the contraction and output widths are
    padded to 16 (D = 72 runs 16x16x32 products over 80; 64 and 128 are
    exact)."""
    return (D + 15) // 16 * 16


def computed_pairs(P, cu, H, D, causal, pass_):
    """(query, key) pairs inside the 32x32 blocks one kernel pass multiplies,
    per head: each 32-row group of a sequence tile meets the 32-row blocks of
    its own sequence (up to the diagonal when causal); each 32-row group of a
    packed window meets the blocks from its first row's sequence start to its
    last row's sequence end."""
    units, n_tiles, starts = P.work_list(cu, H, D, causal, pass_)
    total = 0
    for i, (row0, seq0, seqlen, rows, head) in enumerate(units.tolist()):
        if rows == 0 or head != 0:
            continue
        if i < n_tiles:
            nblk = (seqlen + 31) // 32
            for g0 in range(0, rows, 32):
                a = (row0 - seq0 + g0) // 32  # block index of the group's first row
                if not causal:
                    nb = nblk
                elif pass_ == 1:  # key group: query blocks at or after it
                    nb = nblk - a
                else:  # query group: key blocks up to it
                    nb = min(nblk, a + 1)
                total += nb * 1024
        else:
            mask = starts[-seqlen - 1]
            bits = [x for w in range(4) for x in range(64) if (int(mask[w]) >> x) & 1]
            seq_starts = bits + [rows]
            for g0 in range(0, rows, 32):
                g1 = min(rows, g0 + 32) - 1
                lo = max(s for s in seq_starts[:-1] if s <= g0)
                hi = min(s for s in seq_starts if s > g1)
                total += ((hi + 31) // 32 - lo // 32) * 1024
    return total


def matrix_work(P, w):
    """Tile fill per pass and the matrix flops the kernels execute against
    the algorithmic 14*pairs*H*D (products per pass: forward S and PV; dK/dV
    pass S, dP, dV, dK; dQ pass S, dP, dQ; widths padded as the products
    run).  Packed windows whose dQ the dK/dV launch forms (head widths <= 96)
    skip the dQ pass; that saving is not subtracted here, so the model
    overstates such packs' executed work."""
    H, D, causal = w.n_heads, w.head_dim, w.causal
    cu = w.cu_seqlens
    pairs = pairs_of(w.lengths, causal)
    Dp = padded_width(D)
    out = {"valid_pairs_per_head": pairs, "padded_width": Dp}
    executed = 0.0
    for pass_, name, products in ((0, "fwd", 2), (1, "dkdv", 4), (2, "dq", 3)):
        cp = computed_pairs(P, cu, H, D, causal, pass_)
        out[f"{name}_fill"] = pairs / cp if cp else None
        executed += 2.0 * products * cp * H * Dp
    out["executed_flop_per_step"] = executed
    out["algorithmic_flop_per_step"] = 14.0 * pairs * H * D
    out["executed_over_algorithmic"] = executed / out["algorithmic_flop_per_step"]
    out["note"] = ("fill = valid pairs / pairs in the 32x32 blocks a pass multiplies; executed = 2 x products x "
                   "computed pairs x H x padded width, summed over the three passes (the dQ pass recomputes S and dP: "
                   "18 products-worth per pair against the 14 of the convention)")
    return out


# ---------------------------------------------------------------------------
# baselines

def cpu_info():
    model = platform.processor() or ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas = None
    return {"model": model, "os_cpu_count": os.cpu_count(), "affinity": len(os.sched_getaffinity(0)),
            "blas_threads": blas}


def cpu_baseline(w, seed: int, budget_s: float = 20.0):
    """The float64 oracle (forward + backward), timed on the host cores over
    a bounded sample of the workload: whole sequences of the pack in order
    while they fit the time budget; a pack of one sequence too long for the
    budget (the Ulysses shard) is sampled as one sequence of the same shape
    (heads, width, mask) whose length is the largest power of two the budget
    allows.  The rate is then extrapolated, and labelled so, to the whole
    step's 14*pairs*H*D."""
    from oracle import attention as A
    from paper_2608_07524_amd import inputs as I
    info = cpu_info()
    rng = np.random.default_rng(seed + 1)

    def run(lengths):
        T = int(sum(lengths))
        q, k, v, do = (I.bf16_to_f64(b) for b in I.tensors(rng, T, w.n_heads, w.head_dim))
        cu = I.cu_from_lengths(lengths)
        t0 = time.perf_counter()
        A.attention_forward(q, k, v, cu, w.scale, w.causal)
        A.attention_backward(do, q, k, v, cu, w.scale, w.causal)
        return time.perf_counter() - t0

    done, t_total = [], 0.0
    if len(w.lengths) == 1:
        s = 2048
        t = run([s])
        done, t_total = [s], t
        while t_total + t * 4 <= budget_s and 2 * s < w.lengths[0]:
            s *= 2
            t = run([s])
            done.append(s)
            t_total += t
        sample = (f"float64 fwd+bwd of single sequences {done} at the shard's shape ({w.n_heads} heads, "
                  f"D={w.head_dim}, {'causal' if w.causal else 'non-causal'}), {t_total:.1f} s")
    else:
        for s in w.lengths:
            if t_total > budget_s:
                break
            t_total += run([s])
            done.append(s)
        sample = f"float64 fwd+bwd of the pack's first {len(done)} sequences {done[:12]}..., {t_total:.1f} s"
    flops = 14.0 * pairs_of(done, w.causal) * w.n_heads * w.head_dim
    rate = flops / t_total
    full = 14.0 * pairs_of(w.lengths, w.causal) * w.n_heads * w.head_dim
    return {"value": rate / 1e12, "unit": "TFLOP/s", "cores": info["blas_threads"] or info["affinity"],
            "kind": "oracle", "sample": sample, "cpu": info,
            "full_step_extrapolated_s": full / rate,
            "extrapolation_note": "whole-step oracle time at the sample's measured rate (not measured)"}


def padded_baseline(torch, P, w, q, k, v, do, steps, warmup, flop):
    """Same kernels on the batch zero-padded to its longest sequence,
    credited with the unpadded valid pairs."""
    smax = max(w.lengths)
    n = len(w.lengths)
    H, D = w.n_heads, w.head_dim
    qp, kp, vp, dop = (torch.zeros((n * smax, H, D), dtype=torch.bfloat16, device="cuda") for _ in range(4))
    off = 0
    for b, s in enumerate(w.lengths):
        for src, dst in ((q, qp), (k, kp), (v, vp), (do, dop)):
            dst[b * smax:b * smax + s] = src[off:off + s]
        off += s
    cu_p = np.arange(n + 1, dtype=np.int32) * smax
    callp = P.PreparedAttention(qp, kp, vp, dop, cu_p, w.scale, w.causal)
    ms_p, _, _ = time_steps(torch, P, callp, steps, warmup)
    return {"value": flop / (ms_p * 1e-3) / 1e12, "ms_per_step": ms_p, "padded_to": smax,
            "computed_pairs": pairs_of([smax] * n, w.causal),
            "note": "same kernels, every sequence zero-padded to the batch maximum; credited with the unpadded "
                    "valid pairs only"}


# ---------------------------------------------------------------------------
# roofline of the dominant kernel

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
           "traffic_unit": "HBM bytes per launch (rocprofv3 FETCH_SIZE, WRITE_SIZE; scaled by a direct-to-LDS "
                           "copy of known size)"}
    if mfma:
        a = flop / (ms * 1e-3) / 1e12
        out.update(bound="mfma", achieved=a, peak=BF16_PEAK_TFLOPS, unit="TFLOP/s", frac=a / BF16_PEAK_TFLOPS)
    else:
        a = nbytes / (ms * 1e-3) / 1e9
        out.update(bound="hbm", achieved=a, peak=HBM_PEAK_GBS, unit="GB/s", frac=a / HBM_PEAK_GBS)
    return out


def mfma_loop_tflops(torch, iters: int = 1000000):
    """The matrix-core rate of dependent bf16 32x32x16 product chains with
    nothing else running (one workgroup of 8 wavefronts per CU, two per
    SIMD, four independent chains each; the probe library's
    dcp_probe_mfma_rate), about 0.1 s of products timed with HIP events after
    one untimed launch: the practical ceiling for the kernels' product
    rates."""
    import ctypes as C
    from paper_2608_07524_amd.build import PROBE_LIB
    probe = C.CDLL(PROBE_LIB)
    probe.dcp_probe_mfma_rate.argtypes = [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_void_p, C.POINTER(C.c_double)]
    blocks = torch.cuda.get_device_properties(0).multi_processor_count
    out = torch.empty(blocks * 512, dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream()
    flops = C.c_double()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for timed in (False, True):
        if timed:
            a.record(s)
        if probe.dcp_probe_mfma_rate(out.data_ptr(), blocks, iters, 4, C.c_void_p(s.cuda_stream), C.byref(flops)) != 0:
            raise RuntimeError("matrix-core rate probe failed")
        if timed:
            b.record(s)
    torch.cuda.synchronize()
    return flops.value / (a.elapsed_time(b) * 1e-3) / 1e12


def host_us_per_call(torch, P, w, call, n: int = 5):
    """Host time of one call, averaged over n enqueued calls after one
    untimed call (the device is idle at the start and the calls do not wait
    for it): the per-call API
    (dcp_varlen_attn_fwd / _bwd build the work lists on the host and copy
    them to the device each time) against the prepared batch
    (dcp_batch_fwd / _bwd only launch)."""
    import ctypes as C
    from paper_2608_07524_amd import _native as N
    lib = P.load()
    T, H, D = w.total_tokens, w.n_heads, w.head_dim
    d = N._Desc(w.cu_seqlens, T, H, D, w.scale, w.causal)
    nf, nb = C.c_size_t(), C.c_size_t()
    lib.dcp_varlen_attn_fwd_workspace_size(d.ref, C.byref(nf))
    lib.dcp_varlen_attn_bwd_workspace_size(d.ref, C.byref(nb))
    ws_f = torch.empty(max(1, nf.value), dtype=torch.uint8, device="cuda")
    ws_b = torch.empty(max(1, nb.value), dtype=torch.uint8, device="cuda")
    s = call.stream
    a = (call.q.data_ptr(), call.k.data_ptr(), call.v.data_ptr(), call.o.data_ptr(), call.lse.data_ptr())
    g = (call.dout.data_ptr(), call.o.data_ptr(), call.lse.data_ptr(), call.q.data_ptr(), call.k.data_ptr(),
         call.v.data_ptr(), call.dq.data_ptr(), call.dk.data_ptr(), call.dv.data_ptr())
    runs = {
        "per_call_fwd": lambda: lib.dcp_varlen_attn_fwd(d.ref, *a, ws_f.data_ptr(), ws_f.numel(), s),
        "per_call_bwd": lambda: lib.dcp_varlen_attn_bwd(d.ref, *g, ws_b.data_ptr(), ws_b.numel(), s),
        "batch_fwd": lambda: lib.dcp_batch_fwd(call.batch, *a, call.ws.data_ptr(), call.ws.numel(), s),
        "batch_bwd": lambda: lib.dcp_batch_bwd(call.batch, *g, call.ws.data_ptr(), call.ws.numel(), s),
    }
    out = {}
    for key, fn in runs.items():
        if fn() != 0:
            raise RuntimeError(N.last_error())
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(n):
            if fn() != 0:
                raise RuntimeError(N.last_error())
        out[key] = (time.perf_counter() - t0) / n * 1e6
        torch.cuda.synchronize()
    return out


def measure(torch, P, name, steps, warmup, seed, padded=False, with_fill=True):
    """One workload: timing, kernels, roofline, fill, measured counters (and
    for the short video mix the padded-bucket baseline)."""
    w, rng = workload(name, seed)
    H, D, causal = w.n_heads, w.head_dim, w.causal
    T = w.total_tokens
    cu = w.cu_seqlens
    pairs = pairs_of(w.lengths, causal)
    flop_fwd = 4.0 * pairs * H * D
    flop_bwd = 10.0 * pairs * H * D
    q, k, v, do = device_tensors(torch, rng, T, H, D)
    call = P.PreparedAttention(q, k, v, do, cu, w.scale, causal)
    ms, fwd_ms, bwd_ms = time_steps(torch, P, call, steps, warmup)
    host = host_us_per_call(torch, P, w, call)
    del call
    value = (flop_fwd + flop_bwd) / (ms * 1e-3) / 1e12
    flop_dkdv = 8.0 * pairs * H * D
    win_rows, win_pairs = window_dq_part(P, cu, H, D, causal)
    res = {
        "value": value, "pct_bf16_peak": 100.0 * value / BF16_PEAK_TFLOPS, "ms_per_step": ms,
        "config": {"workload": WORKLOADS[name], "n_seqs": len(w.lengths), "total_tokens": T, "heads": H,
                   "head_dim": D, "causal": causal, "valid_pairs": pairs, "flop_per_step": flop_fwd + flop_bwd,
                   "flop_convention": "fwd 4*pairs*H*D + bwd 10*pairs*H*D"},
        "kernels": {"fwd_ms": fwd_ms, "fwd_tflops": flop_fwd / (fwd_ms * 1e-3) / 1e12, "bwd_dkdv_ms": bwd_ms,
                    "bwd_dkdv_tflops": flop_dkdv / (bwd_ms * 1e-3) / 1e12, "bwd_rest_ms": ms - fwd_ms - bwd_ms},
        "roofline": roofline(flop_dkdv + 2.0 * win_pairs * H * D, dkdv_bytes(cu, H, D) + 2.0 * win_rows * H * D,
                             bwd_ms, measured(name, "dkdv_traffic_bytes")),
        "host_us_per_call": host,
    }
    if with_fill:
        mw = matrix_work(P, w)
        counted = measured(name, "mfma_flop_per_step")
        mw["counted_flop_per_step"] = counted
        mw["counted_note"] = "SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 over one step (profiles/), null when stale"
        res["matrix_work"] = mw
    if padded and name == "video_short":
        res["padded_baseline"] = padded_baseline(torch, P, w, q, k, v, do, steps, warmup, flop_fwd + flop_bwd)
    del q, k, v, do
    torch.cuda.empty_cache()
    return w, res


def tiny_plan(P):
    """The tiny configuration's planner call on a cost table measured on
    this GPU by dcp_profile_cost (4 rows at 4 heads of width 64), next to the
    analytic table: L = 28, T_C = 100 us, M_C = 900 MiB, budget 1 GiB,
    hidden 256, p in {1, 2, 4, 8}, b <= 64, G in [1, 4], with and without
    the head-divisibility filter."""
    from paper_2608_07524_amd import inputs as I
    w = I.tiny()
    h = 256
    rows = P.profile_cost(w.lengths, w.n_heads, w.head_dim, causal=False, scale=w.scale, warmup=3, reps=10,
                          act_bytes_per_token=34 * h, inp_bytes_per_token=2 * h)
    table = [(r.seq_len, r.t_f_ns, r.t_b_ns, r.m_bytes, r.m_inp_bytes) for r in rows]
    out = {"measured_rows": table}
    for name, flags in (("head_filter", 0), ("no_head_filter", P.PLAN_FLAG_NO_HEAD_FILTER)):
        t0 = time.perf_counter()
        n_calls = 200
        for _ in range(n_calls):
            plan = P.plan(w.lengths, table, 28, 100_000, 900 << 20, 1 << 30, n_heads=w.n_heads, hidden=h,
                          flags=flags)
        us = (time.perf_counter() - t0) / n_calls * 1e6
        out[name] = {"sp_size": plan.sp_size, "micro_batch": plan.micro_batch, "grad_accum": plan.grad_accum,
                     "recompute_layers": plan.recompute_layers, "step_time_ns": plan.step_time_ns,
                     "us_per_call_incl_binding": us}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="ulysses256k", choices=sorted(WORKLOADS))
    ap.add_argument("--extras", default="text,video_short",
                    help="comma-separated workloads reported as extra keys ('' for none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-padded", action="store_true")
    ap.add_argument("--no-plan", action="store_true")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run one direct-to-LDS device copy of this many MiB (the known-size reference for "
                         "the HBM byte counters)")
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
        from paper_2608_07524_amd.build import PROBE_LIB
        probe = ctypes.CDLL(PROBE_LIB)
        probe.dcp_probe_dma_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        n = args.copy_probe_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        st = probe.dcp_probe_dma_copy(src.data_ptr(), dst.data_ptr(), n,
                                      ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        torch.cuda.synchronize()
        if st != 0 or not bool(torch.equal(src, dst)):
            raise SystemExit("direct-to-LDS copy probe failed")
        dst.copy_(src)  # a plain copy of the same size, for comparison
        torch.cuda.synchronize()
        del src, dst

    props = torch.cuda.get_device_properties(0)
    dev = P.device_info()
    # bf16 dense peak from the unit counts: a 32x32x16 product (32,768 flop)
    # every 32 clocks on each of a CU's four SIMDs
    dev_peak = dev["compute_units"] * 4 * 1024 * dev["clock_mhz"] * 1e6 / 1e12
    device = {"name": props.name, "arch": props.gcnArchName, "compute_units": dev["compute_units"],
              "clock_mhz": dev["clock_mhz"], "bf16_dense_tflops_from_units": dev_peak,
              "bf16_dense_tflops_used": BF16_PEAK_TFLOPS, "hbm_gbs_used": HBM_PEAK_GBS}
    device["mfma_loop_tflops"] = mfma_loop_tflops(torch)
    w, head = measure(torch, P, args.workload, args.steps, args.warmup, args.seed, padded=not args.no_padded)
    line = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "pct_bf16_peak": head["pct_bf16_peak"],
        "config": head["config"],
        "kernels": head["kernels"],
        "roofline": head["roofline"],
        "matrix_work": head.get("matrix_work"),
        "host_us_per_call": head.get("host_us_per_call"),
        "padded_baseline": head.get("padded_baseline"),
        "device": device,
    }
    extras = {}
    for name in [x for x in args.extras.split(",") if x and x != args.workload]:
        _, extras[name] = measure(torch, P, name, args.steps, args.warmup, args.seed, padded=not args.no_padded)
    line["also"] = extras
    line["tiny_plan"] = None if args.no_plan else tiny_plan(P)
    line["cpu_baseline"] = None if args.no_cpu_baseline else cpu_baseline(w, args.seed)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
