"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke check.

This module only draws random numbers, rounds them to bfloat16 and packs
sequence lengths; it holds none of the attention or planner arithmetic, so
both the CPU oracle and the GPU path can consume its output.

Recipe (all workloads): ``rng = numpy.random.default_rng(seed)``; lengths are
drawn first (when random), then q, k, v and dO in that order, each
``rng.standard_normal((T, H, D), float32)`` rounded to bfloat16 with
round-to-nearest-even.  The same bf16 bits go to the GPU and, widened
exactly to float64, to the oracle.

The workloads stand in for the paper's datasets (short / balanced / long
synthetic length mixtures, Appendix A; video clips of many resolutions and
frame counts, Sec. 2.1) whose distributions only exist as figures: they keep
the shapes of the paper's models (Table 1: Transformer-2D has 16 heads of
width 72, Transformer-1D 48 heads of width 64; a Ulysses shard holds H/p
heads of the full sequence, Sec. 6.1).
"""

from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional

import numpy as np


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bits exactly to float64."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def cu_from_lengths(lengths) -> np.ndarray:
    return np.concatenate([[0], np.cumsum(np.asarray(lengths, dtype=np.int64))]).astype(np.int32)


def greedy_pack(lengths: List[int], cap: int) -> List[List[int]]:
    """Sequential first-fit packing: start a new pack when the next length
    would overflow ``cap`` tokens."""
    packs, cur, tot = [], [], 0
    for s in lengths:
        if cur and tot + s > cap:
            packs.append(cur)
            cur, tot = [], 0
        cur.append(int(s))
        tot += int(s)
    if cur:
        packs.append(cur)
    return packs


def video_tokens_per_frame(height: int, width: int) -> int:
    """8x spatial VAE compression then 2x2 patches, each stage rounding up."""
    return math.ceil(math.ceil(height / 8) / 2) * math.ceil(math.ceil(width / 8) / 2)


@dataclass
class Workload:
    name: str
    lengths: List[int]
    n_heads: int
    head_dim: int
    causal: bool
    scale: float

    @property
    def cu_seqlens(self) -> np.ndarray:
        return cu_from_lengths(self.lengths)

    @property
    def total_tokens(self) -> int:
        return int(sum(self.lengths))


def tiny(seed: int = 0) -> Workload:
    """4 sequences {37, 64, 128, 200}, 4 heads of width 64, scale 1/8."""
    return Workload("tiny packed 4 seqs (429 tok) H4 D64", [37, 64, 128, 200], 4, 64, False, 0.125)


def video_short_mix(rng: np.random.Generator, n_seqs: int = 32) -> Workload:
    """32 clips of 1024/2048/4096/8192 tokens (uniform), 16 heads of width 72."""
    lens = rng.choice([1024, 2048, 4096, 8192], n_seqs).tolist()
    return Workload("video-DiT short mix 32 seqs {1k..8k} H16 D72", lens, 16, 72, False, 1.0 / math.sqrt(72))


VIDEO_FRAMES = (1, 16, 32, 51)
VIDEO_FRAME_WEIGHTS = (0.4, 0.3, 0.2, 0.1)
VIDEO_RESOLUTIONS = ((256, 256), (480, 854), (720, 1280))


def video_long_tail_packs(rng: np.random.Generator, n_packs: int = 8, cap: int = 131072) -> List[Workload]:
    """Clip length = frames x tokens-per-frame, frames weighted .4/.3/.2/.1,
    resolution uniform; clips above the pack cap are redrawn; sequential
    packing into <= cap tokens; the first ``n_packs`` packs."""
    lens: List[int] = []
    packs: List[List[int]] = []
    while len(packs) <= n_packs:
        f = int(rng.choice(VIDEO_FRAMES, p=VIDEO_FRAME_WEIGHTS))
        hgt, wid = VIDEO_RESOLUTIONS[int(rng.integers(0, len(VIDEO_RESOLUTIONS)))]
        s = f * video_tokens_per_frame(hgt, wid)
        if s > cap:
            continue
        lens.append(s)
        packs = greedy_pack(lens, cap)
    return [Workload(f"video-DiT long-tail pack {i} H16 D72", p, 16, 72, False, 1.0 / math.sqrt(72))
            for i, p in enumerate(packs[:n_packs])]


def video_clips(rng: np.random.Generator, n_tokens: int, cap: int = 131072) -> List[tuple]:
    """Clips (frames, tokens per frame) drawn like the long-tail mix until
    their tokens reach ``n_tokens`` (clips above ``cap`` redrawn)."""
    clips, tot = [], 0
    while tot < n_tokens:
        f = int(rng.choice(VIDEO_FRAMES, p=VIDEO_FRAME_WEIGHTS))
        hgt, wid = VIDEO_RESOLUTIONS[int(rng.integers(0, len(VIDEO_RESOLUTIONS)))]
        n = video_tokens_per_frame(hgt, wid)
        if f * n > cap:
            continue
        clips.append((f, n))
        tot += f * n
    return clips


def video_2d_pack(rng: np.random.Generator, axis: str, cap: int = 131072) -> Workload:
    """Transformer-2D attention (Sec. 4.1; Table 1: 16 heads of width 72)
    attends within one frame (spatial) or along one token position over
    the frames (temporal): a clip of f frames x n tokens per frame is f
    spatial sequences of n tokens or n temporal sequences of f tokens (a
    single-frame clip gives sequences of one token).  Clips drawn like the
    long-tail mix, sequences packed in clip order into <= cap tokens; the
    first pack."""
    lens: List[int] = []
    for f, n in video_clips(rng, cap):
        lens += [n] * f if axis == "spatial" else [f] * n
    pack = greedy_pack(lens, cap)[0]
    return Workload(f"video-DiT 2-D {axis} pack H16 D72", pack, 16, 72, False, 1.0 / math.sqrt(72))


def ulysses_shard(length: int) -> Workload:
    """One device's Ulysses shard at SP=8 of a 16-head model: all tokens of a
    single sequence, 2 local heads of width 128."""
    return Workload(f"Ulysses SP=8 shard {length} tok H2 D128", [length], 2, 128, False, 1.0 / math.sqrt(128))


def text_lengths(rng: np.random.Generator, n: int, median: int = 2048, sigma: float = 1.0,
                 lo: int = 128, hi: int = 131072) -> np.ndarray:
    """Log-normal document lengths, rounded to nearest and clipped."""
    x = np.floor(np.exp(math.log(median) + sigma * rng.standard_normal(n)) + 0.5)
    return np.clip(x, lo, hi).astype(np.int64)


def text_packs(rng: np.random.Generator, n_packs: int, cap: int = 262144) -> List[Workload]:
    """Causal text packs: log-normal lengths packed to <= cap tokens, 32 heads of width 128."""
    packs: List[List[int]] = []
    pool: List[int] = []
    while len(packs) <= n_packs:
        pool.extend(text_lengths(rng, 256).tolist())
        packs = greedy_pack(pool, cap)
    return [Workload(f"text-LM causal pack {i} H32 D128", p, 32, 128, True, 1.0 / math.sqrt(128))
            for i, p in enumerate(packs[:n_packs])]


def tensors(rng: np.random.Generator, T: int, H: int, D: int, n: int = 4) -> List[np.ndarray]:
    """``n`` bf16 tensors [T, H, D] (uint16 bits), drawn q, k, v, dO in order."""
    out = []
    for _ in range(n):
        out.append(bf16_bits(rng.standard_normal((T, H, D), dtype=np.float32)))
    return out
