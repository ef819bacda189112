"""Schedule replay on measured MI355X costs: DCP (intra and inter) against
bucket parallelism on W devices, for the paper's two models (Table in
Appendix B) on synthetic length mixtures (Sec. 4.1, Appendix A shapes).

    python -m paper_2608_07524_amd.replay [--devices 32] [--md out.md]

Cost table per model, one row per length the stream uses (Transformer-1D
also a second time from the dual-layer profile of the library's whole layer,
``model.profile_rows``: attention, projections, norms and activation timed
together on the second of two layers, m = that layer's stash bytes):
* attention, measured on this GPU through the library: Transformer-1D rows
  come from dcp_profile_cost (one causal sequence of each length, all 48
  heads of width 64); Transformer-2D rows time the forward and backward of a
  clip's spatial pack (f frames of n tokens) plus its temporal pack (n
  sequences of f tokens), 16 heads of width 72;
* the rest of a layer, measured through the library: its whole layer
  (norms, projections, MLP; dcp_layer_fwd / dcp_layer_bwd) minus its
  attention, on a batch of 128 sequences of 128 tokens (attention a small
  share), gives picoseconds per token forward and backward;
* memory, analytic: 34*h bytes of stashed activations per token and layer
  with flash attention (Korthikanti et al., cited in Sec. 5) and 2*h bytes
  of layer input; model states M_C = 4 bytes per parameter (bf16 weights and
  gradients) + 12 bytes per parameter sharded over W (ZeRO-1, Sec. 4.1).
The per-iteration gradient synchronisation is modelled as a reduce-scatter
plus an all-gather of the bf16 gradients and weights over W devices at
50 GB/s per device (one 400 Gb/s NIC).

Nothing here runs on the attention hot path; the replay itself is the C++
dcp_simulate.
"""

from __future__ import annotations

import argparse
import json
import math
import sys
from typing import List

import numpy as np

from . import inputs as I

MODELS = {
    # name: (layers, hidden, heads, head_dim, params, causal)
    "Transformer-1D": (42, 3072, 48, 64, 5_000_000_000, True),
    "Transformer-2D": (28, 1152, 16, 72, 1_200_000_000, False),
}
GIB = 1 << 30


def _events(torch):
    return torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)


def layer_rest_ps_per_token(torch, P, H: int, D: int, causal: bool, n_seqs: int = 128, s: int = 128,
                            reps: int = 5):
    """Forward and backward time per token of one layer apart from its
    attention, in ps: the library's whole layer (norms, projections, MLP,
    dcp_layer_fwd / dcp_layer_bwd with a stash) minus the library's
    attention on the same packed batch, both timed on the second of two
    layers.  The batch is many short sequences (n_seqs x s tokens), so the
    attention is a small share and the difference is the per-token part."""
    from .model import profile_rows
    cu = I.cu_from_lengths([s] * n_seqs)
    T = int(cu[-1])
    layer = profile_rows([T], H, D, causal, reps=reps, cu_seqlens=cu)[0]
    af, ab = _attn_time_ns(torch, P, [s] * n_seqs, H, D, causal, reps=reps)
    return max(0, (layer.t_f_ns - af) * 1000 // T), max(0, (layer.t_b_ns - ab) * 1000 // T)


def _attn_time_ns(torch, P, lengths: List[int], H: int, D: int, causal: bool, reps: int = 5):
    """Median forward and backward time of one packed attention call."""
    cu = I.cu_from_lengths(lengths)
    T = int(cu[-1])
    q, k, v, do = (torch.randn(T, H, D, dtype=torch.bfloat16, device="cuda") for _ in range(4))
    call = P.PreparedAttention(q, k, v, do, cu, 1.0 / math.sqrt(D), causal)
    tf, tb = [], []
    for r in range(reps + 2):
        a, b = _events(torch)
        c = torch.cuda.Event(enable_timing=True)
        a.record()
        call.fwd()
        b.record()
        call.bwd()
        c.record()
        torch.cuda.synchronize()
        if r >= 2:
            tf.append(a.elapsed_time(b))
            tb.append(b.elapsed_time(c))
    del call, q, k, v, do
    return int(np.median(tf) * 1e6), int(np.median(tb) * 1e6)


def cost_rows(torch, P, model: str, lengths, clips=None):
    L, h, H, D, params, causal = MODELS[model]
    lin_f, lin_b = layer_rest_ps_per_token(torch, P, H, D, causal)
    act, inp = 34 * h, 2 * h
    rows = []
    if clips is None:
        prof = P.profile_cost(sorted(set(lengths)), H, D, causal=causal, warmup=2, reps=5,
                              lin_f_ps_per_token=lin_f, lin_b_ps_per_token=lin_b, act_bytes_per_token=act,
                              inp_bytes_per_token=inp)
        rows = [(r.seq_len, r.t_f_ns, r.t_b_ns, r.m_bytes, r.m_inp_bytes) for r in prof]
    else:
        for f, n in sorted(set(clips), key=lambda c: c[0] * c[1]):
            s = f * n
            sf, sb = _attn_time_ns(torch, P, [n] * f, H, D, False)  # spatial: within each frame
            tf, tb = _attn_time_ns(torch, P, [f] * n, H, D, False)  # temporal: along each position
            rows.append((s, sf + tf + lin_f * s // 1000, sb + tb + lin_b * s // 1000, act * s, inp * s))
    return rows, lin_f


def model_constants(model: str, W: int):
    L, h, H, D, params, causal = MODELS[model]
    M_C = 4 * params + 12 * params // W
    sync_ns = int(2 * 2 * params * (W - 1) / W / 50.0)  # bytes / (50 bytes per ns)
    return L, h, H, M_C, sync_ns


def replay(P, model: str, rows, lengths, W: int, budget: int, g_max: int = 4):
    L, h, H, M_C, sync = model_constants(model, W)
    out = {}
    for mode, name in ((P.PLAN_INTRA, "DCP-intra"), (P.PLAN_INTER, "DCP-inter")):
        d, b = P.simulate(lengths, rows, L, 0, M_C, budget, W, 0, sync, sp_cands=[1, 2, 4, 8], n_heads=H, hidden=h,
                          mode=mode, g_max=g_max, b_max=64)
        out[name] = d
        out["bucket"] = b
    return out, sync


def _summary(res, W):
    return {"tokens_per_s": res["tokens"] / res["time_ns"] * 1e9,
            "imbalance": 1.0 - res["busy_device_ns"] / (W * res["makespan_ns"]),
            "iterations": res["iterations"], "sp": res["bucket_sp"]}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--devices", type=int, default=32)
    ap.add_argument("--n-seqs", type=int, default=2000)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--md", default=None, help="also write a markdown summary here")
    args = ap.parse_args(argv)
    import torch
    import paper_2608_07524_amd as P
    if not torch.cuda.is_available():
        raise SystemExit("replay needs a GPU to measure the cost table")
    P.load()
    W = args.devices
    rng = np.random.default_rng(args.seed)
    scenarios = []
    # Transformer-1D on text: log-normal lengths, median 1k / 4k / 16k (short,
    # balanced, long stand-ins), sigma 1, clipped to [128, 131072]; the
    # table's lengths are powers of two, each sequence taking the next one up.
    grid = [128 << i for i in range(11)]
    rows_1d, lin_1d = cost_rows(torch, P, "Transformer-1D", grid)
    # and from the dual-layer profile of the library's whole layer (the
    # second of two layers timed, its stash bytes as m), Sec. 3.5
    from .model import profile_rows
    L1, h1, H1, D1, _, causal1 = MODELS["Transformer-1D"]
    rows_1d_layer = [(r.seq_len, r.t_f_ns, r.t_b_ns, r.m_bytes, r.m_inp_bytes)
                     for r in profile_rows(grid, H1, D1, causal1)]
    texts = []
    for label, med in (("short", 1024), ("balanced", 4096), ("long", 16384)):
        texts.append((med, I.text_lengths(rng, args.n_seqs, median=med).tolist()))
    for med, lens in texts:
        scenarios.append(("Transformer-1D", f"text, median {med}", rows_1d, lens, lin_1d))
    for med, lens in texts:
        scenarios.append(("Transformer-1D", f"text, median {med}, layer profile", rows_1d_layer, lens, None))
    # Transformer-2D on video: the long-tail clip mix (frames {1,16,32,51}
    # weighted .4/.3/.2/.1 x 256^2, 480x854, 720x1280), one clip per batch.
    clips = I.video_clips(rng, 64 * 1024 * args.n_seqs, cap=131072)[:args.n_seqs]  # ~30k tokens per clip
    rows_2d, lin_2d = cost_rows(torch, P, "Transformer-2D", None, clips=clips)
    scenarios.append(("Transformer-2D", "video long-tail clips", rows_2d, [f * n for f, n in clips], lin_2d))
    lines = []
    results = []
    for budget_gib in (80, 288):
        for model, data, rows, lens, lin in scenarios:
            out, sync = replay(P, model, rows, lens, W, budget_gib * GIB)
            s = {k: _summary(v, W) for k, v in out.items()}
            base = s["bucket"]["tokens_per_s"]
            rec = {"model": model, "data": data, "budget_gib": budget_gib, "devices": W, "sync_ms": sync / 1e6,
                   "layer_rest_ps_per_token_fwd": lin, "schedules": s,
                   "speedup": {k: v["tokens_per_s"] / base for k, v in s.items()}}
            results.append(rec)
            print(json.dumps(rec), flush=True)
            lines.append(f"| {model} | {data} | {budget_gib} | {s['bucket']['sp']} | "
                         f"{s['bucket']['tokens_per_s'] / 1e6:.3f} | {s['bucket']['imbalance']:.3f} | "
                         f"{s['DCP-inter']['tokens_per_s'] / 1e6:.3f} | {s['DCP-inter']['imbalance']:.3f} | "
                         f"{s['DCP-intra']['tokens_per_s'] / 1e6:.3f} | {s['DCP-intra']['imbalance']:.3f} | "
                         f"{rec['speedup']['DCP-inter']:.2f} | {rec['speedup']['DCP-intra']:.2f} |")
    if args.md:
        with open(args.md, "w") as f:
            f.write("| Model | Data | HBM budget (GiB) | bucket p | bucket Mtok/s | bucket imbalance | "
                    "DCP-inter Mtok/s | DCP-inter imbalance | DCP-intra Mtok/s | DCP-intra imbalance | "
                    "inter speedup | intra speedup |\n|---|---|---|---|---|---|---|---|---|---|---|---|\n")
            f.write("\n".join(lines) + "\n")
    return results


if __name__ == "__main__":
    main(sys.argv[1:])
