"""Layer stacks over one packed batch: the recompute executor and the
dual-layer profiling of Sec. 3.5.

* ``Stack.step(flags)``: forward through L layers, keeping the activation
  stash of layer l unless flags[l] (the planner's recompute_flags: the first
  r layers recomputed), then backward in reverse, each recomputed layer
  running its forward again first (Eqs. (4)-(6): T = L (t_f + t_b) + r t_f +
  T_C, M = (L - r) m + L m_inp + M_C).  Every layer call is the C ABI
  (dcp_layer_fwd / dcp_layer_bwd); this file only sequences them.
* ``profile_rows``: for each length, a two-layer stack without recomputation;
  the first layer warms up and the second one's forward time, backward time
  and stash bytes are the row (t_f, t_b, m), with m_inp the bytes of its bf16
  input -- the dual-layer profile of Sec. 3.5, now of the whole layer.

    python -m paper_2608_07524_amd.model [--md out.md]

measures, for the paper's Transformer-2D and Transformer-1D shapes, the
dual-layer rows and the step time of an L-layer stack for r = 0 .. L
recomputed layers against the model's prediction.
"""

from __future__ import annotations

import argparse
import json
import math
import sys
from typing import List, Optional, Sequence

import numpy as np

from . import _native as N
from . import inputs as I


class Stack:
    """L layers of one shape (random bf16 weights, fp32 gradients) over one
    packed batch with all layer buffers allocated up front."""

    def __init__(self, n_layers: int, cu_seqlens, n_heads: int, head_dim: int, causal: bool = False,
                 seed: int = 0, eps: float = 1e-6):
        import torch
        self.torch = torch
        h = n_heads * head_dim
        cu = np.asarray(cu_seqlens, dtype=np.int32)
        T = int(cu[-1])
        g = torch.Generator(device="cuda").manual_seed(seed)
        self.layers: List[N.Layer] = []
        ws = None
        for _ in range(n_layers):
            W, G = {}, {}
            for name, shape in N.layer_param_shapes(h).items():
                if name.startswith("norm"):
                    W[name] = torch.ones(shape, dtype=torch.bfloat16, device="cuda")
                else:
                    W[name] = (torch.randn(shape, generator=g, device="cuda") / math.sqrt(shape[0])).to(torch.bfloat16)
                G[name] = torch.zeros(shape, dtype=torch.float32, device="cuda")
            layer = N.Layer(W, G, cu, n_heads, head_dim, causal, None, eps, workspace=ws)
            ws = layer.ws
            self.layers.append(layer)
        L = n_layers
        self.stash = [torch.empty(self.layers[0].stash_bytes, dtype=torch.uint8, device="cuda") for _ in range(L)]
        self.xs = [torch.randn(T, h, generator=g, device="cuda").to(torch.bfloat16)]
        self.xs += [torch.empty(T, h, dtype=torch.bfloat16, device="cuda") for _ in range(L)]
        self.dys = [torch.empty(T, h, dtype=torch.bfloat16, device="cuda") for _ in range(2)]
        self.dout = torch.randn(T, h, generator=g, device="cuda").to(torch.bfloat16)
        self.T, self.h = T, h

    def forward(self, flags: Sequence[int], events=None):
        for l, layer in enumerate(self.layers):
            if events is not None:
                events[l][0].record()
            layer.fwd(self.xs[l], keep=not flags[l], out=self.xs[l + 1], stash=self.stash[l])
            if events is not None:
                events[l][1].record()

    def backward(self, flags: Sequence[int], events=None):
        dy = self.dout
        for l in range(len(self.layers) - 1, -1, -1):
            out = self.dys[l % 2]
            if events is not None:
                events[l][0].record()
            self.layers[l].bwd(self.xs[l], dy, dx=out)
            if events is not None:
                events[l][1].record()
            dy = out

    def step(self, flags: Sequence[int]):
        self.forward(flags)
        self.backward(flags)

    def time_step(self, flags: Sequence[int], reps: int = 5, warmup: int = 2) -> float:
        """Median milliseconds of one forward + backward through the stack."""
        t = self.torch
        for _ in range(warmup):
            self.step(flags)
        times = []
        for _ in range(reps):
            a, b = t.cuda.Event(enable_timing=True), t.cuda.Event(enable_timing=True)
            a.record()
            self.step(flags)
            b.record()
            t.cuda.synchronize()
            times.append(a.elapsed_time(b))
        return float(np.median(times))


def profile_rows(lengths: Sequence[int], n_heads: int, head_dim: int, causal: bool, reps: int = 5,
                 warmup: int = 2, cu_seqlens=None) -> List[N.CostRow]:
    """Dual-layer profile per length (one sequence of that length, micro-batch
    1; or, with ``cu_seqlens``, that packed batch of ``lengths[0]`` tokens):
    the second layer's median forward and backward times, its stash bytes
    and its input bytes."""
    import torch
    rows = []
    for s in lengths:
        st = Stack(2, [0, int(s)] if cu_seqlens is None else cu_seqlens, n_heads, head_dim, causal)
        ev = lambda: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(2)]
        tf, tb = [], []
        for r in range(warmup + reps):
            ef, eb = ev(), ev()
            st.forward([0, 0], ef)
            st.backward([0, 0], eb)
            torch.cuda.synchronize()
            if r >= warmup:
                tf.append(ef[1][0].elapsed_time(ef[1][1]))
                tb.append(eb[1][0].elapsed_time(eb[1][1]))
        rows.append(N.CostRow(int(s), int(np.median(tf) * 1e6), int(np.median(tb) * 1e6),
                              int(st.layers[0].stash_bytes), 2 * st.h * int(s)))
        del st
        torch.cuda.empty_cache()
    return rows


MODELS = {
    # name: (heads, head_dim, causal, layers used for the stack, tokens)
    "Transformer-2D (h 1152, 16 heads)": (16, 72, False, 8, 16384),
    "Transformer-1D (h 3072, 48 heads)": (48, 64, True, 8, 8192),
}


def main(argv=None):
    ap = argparse.ArgumentParser(description="recompute executor and dual-layer profile on this GPU")
    ap.add_argument("--md", default=None)
    ap.add_argument("--model", default=None, help="only the model whose name starts with this")
    args = ap.parse_args(argv)
    import torch
    if not torch.cuda.is_available():
        raise SystemExit("needs a GPU")
    N.load()
    md = []
    for name, (H, D, causal, L, s) in MODELS.items():
        if args.model and not name.startswith(args.model):
            continue
        row = profile_rows([s], H, D, causal)[0]
        st = Stack(L, [0, s], H, D, causal)
        curve = []
        for r in range(0, L + 1, 2):
            flags = [1 if l < r else 0 for l in range(L)]
            ms = st.time_step(flags)
            pred = (L * (row.t_f_ns + row.t_b_ns) + r * row.t_f_ns) / 1e6
            mem = ((L - r) * row.m_bytes + L * row.m_inp_bytes) / 2 ** 30
            curve.append({"r": r, "ms": ms, "predicted_ms": pred, "activation_gib": mem})
        del st
        torch.cuda.empty_cache()
        full, none = curve[-1]["ms"], curve[0]["ms"]
        rec = {"model": name, "tokens": s, "layers": L, "causal": causal,
               "dual_layer_row": {"t_f_ms": row.t_f_ns / 1e6, "t_b_ms": row.t_b_ns / 1e6,
                                  "m_mib": row.m_bytes / 2 ** 20, "m_inp_mib": row.m_inp_bytes / 2 ** 20},
               "curve": curve, "saving_no_recompute_vs_full": 1.0 - none / full}
        print(json.dumps(rec), flush=True)
        md.append(f"### {name}, one sequence of {s} tokens, {L} layers{' (causal)' if causal else ''}\n\n"
                  f"Dual-layer row (second of two layers, median of 5): t_f = {row.t_f_ns / 1e6:.3f} ms, "
                  f"t_b = {row.t_b_ns / 1e6:.3f} ms, m = {row.m_bytes / 2 ** 20:.1f} MiB stashed, "
                  f"m_inp = {row.m_inp_bytes / 2 ** 20:.1f} MiB.\n\n"
                  "| recomputed layers r | measured ms / step | L (t_f + t_b) + r t_f (ms) | activations (GiB) |\n"
                  "|---|---|---|---|\n" +
                  "\n".join(f"| {c['r']} | {c['ms']:.2f} | {c['predicted_ms']:.2f} | {c['activation_gib']:.2f} |"
                            for c in curve) +
                  f"\n\nNo recomputation against full recomputation: {100 * rec['saving_no_recompute_vs_full']:.1f} % "
                  "less time per step.\n")
    if args.md:
        with open(args.md, "w") as f:
            f.write("\n".join(md))


if __name__ == "__main__":
    main(sys.argv[1:])
