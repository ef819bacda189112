"""Host work lists (no GPU): every row of every (sequence, head) is covered
exactly once, tiles never straddle two sequences, and packed windows hold
whole runs of consecutive short sequences whose start masks decode to the
true sequence bounds of every row."""

import numpy as np
import pytest

from paper_2608_07524_amd import _native as N
from paper_2608_07524_amd import inputs as I


def _tile_rows(pass_, D):
    return 256


def _window_rows(pass_, D):
    """Rows a packed window may span: the window launches' tile (the dK/dV
    pass at head width 128 launches its windows with its tile shape)."""
    return 256 if (pass_ == 1 and D > 96) else 128


def _seq_of_rows(cu):
    """Sequence index of every row of the packed batch."""
    lens = np.diff(cu)
    return np.repeat(np.arange(lens.size), lens)


def _decode(starts, x, n):
    """Bounds [lo, hi) of the sequence holding window offset x, read off the
    window's start mask bit by bit."""
    bits = [p for p in range(256) if (int(starts[p // 64]) >> (p % 64)) & 1]
    lo = max(p for p in bits if p <= x)
    after = [p for p in bits if p > x]
    return lo, (min(after) if after else n)


def _check(cu, H, D, causal, pass_):
    cu = np.asarray(cu, dtype=np.int64)
    units, n_tiles, starts = N.work_list(cu, H, D, causal, pass_)
    tile, wtile = _tile_rows(pass_, D), _window_rows(pass_, D)
    n = units.shape[0]
    assert n_tiles % 8 == 0 and (n - n_tiles) % 8 == 0
    seq_of = _seq_of_rows(cu)
    covered = np.zeros((H, int(cu[-1])), dtype=np.int32)
    windows_seen = np.zeros((starts.shape[0], H), dtype=np.int32)
    for i, (row0, seq0, seqlen, rows, head) in enumerate(units.tolist()):
        if rows == 0:
            continue
        assert 0 <= head < H and rows <= tile
        covered[head, row0:row0 + rows] += 1
        if i < n_tiles:
            # a tile of one sequence, aligned to the sequence start
            b = int(seq_of[row0])
            assert seq0 == cu[b] and seqlen == cu[b + 1] - cu[b]
            assert (row0 - seq0) % tile == 0 and rows == min(tile, seqlen - (row0 - seq0))
            continue
        assert seqlen < 0 and row0 == seq0 and rows <= wtile
        w = -seqlen - 1
        windows_seen[w, head] += 1
        # whole sequences, each shorter than a window, at least two of them
        bs = np.unique(seq_of[row0:row0 + rows])
        assert cu[bs[0]] == row0 and cu[bs[-1] + 1] == row0 + rows
        assert np.all(np.diff(cu)[bs] < wtile) and bs.size >= 2
        for x in range(rows):
            b = int(seq_of[row0 + x])
            assert _decode(starts[w], x, rows) == (cu[b] - row0, cu[b + 1] - row0)
    assert np.all(covered == 1), "a row is covered twice or not at all"
    assert np.all(windows_seen == 1)
    # no sequence of a window or more is ever packed
    long_rows = np.flatnonzero(np.diff(cu)[seq_of] >= wtile)
    for i in range(n_tiles, n):
        row0, rows = units[i, 0], units[i, 3]
        assert not np.any((long_rows >= row0) & (long_rows < row0 + rows))
    return n_tiles, n - n_tiles


@pytest.mark.parametrize("D", [64, 72, 128])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("pass_", [0, 1, 2])
def test_mixed_lengths(D, causal, pass_):
    rng = np.random.default_rng(10 * D + pass_ + causal)
    lengths = np.concatenate([rng.integers(0, 60, 200), rng.integers(100, 300, 20), [0, 0, 1, 255, 256, 257, 1000],
                              rng.integers(0, 3, 50)])
    rng.shuffle(lengths)
    tiles, windows = _check(I.cu_from_lengths(lengths.tolist()), 3, D, causal, pass_)
    assert tiles > 0 and windows > 0


@pytest.mark.parametrize("axis", ["temporal", "spatial"])
def test_transformer_2d_packs(axis):
    """The temporal pack (sequences of 1..51 tokens) runs almost entirely as
    packed windows; the spatial pack (frames of 256 tokens or more) has none."""
    w = I.video_2d_pack(np.random.default_rng(0), axis)
    tiles, windows = _check(w.cu_seqlens, 2, w.head_dim, w.causal, 0)
    if axis == "temporal":
        assert windows > 0 and tiles <= windows // 8
    else:
        assert windows == 0


def test_tiny_config_and_edges():
    _check(I.tiny().cu_seqlens, 4, 64, False, 0)  # 37 + 64 share one window; 128 and 200 run alone
    _check([0, 0, 0], 2, 72, False, 0)  # only empty sequences
    _check([0, 5], 2, 72, True, 1)  # one short sequence: a plain tile
    _check([0, 256, 512], 1, 128, False, 1)  # two sequences of exactly one dK/dV tile (D 128)
    _check(np.cumsum([0] + [1] * 600), 1, 72, False, 2)  # 600 one-token sequences


def test_window_dq_accounting():
    """The roofline's extra dQ work of packed windows (up to head width 96)
    counts exactly the sequences the dK/dV list packs into windows."""
    import bench as B
    import paper_2608_07524_amd as P
    cu = I.tiny().cu_seqlens  # 37 + 64 share a window; 128 and 200 run as tiles
    assert B.window_dq_part(P, cu, 4, 64, False) == (101, 37 * 37 + 64 * 64)
    assert B.window_dq_part(P, cu, 4, 64, True) == (101, 37 * 38 // 2 + 64 * 65 // 2)
    assert B.window_dq_part(P, cu, 4, 128, False) == (0, 0)  # two-pass windows at head width 128
    # windows {5, 0, 7} and {1, 1, 0}; 300 runs as tiles
    cu = I.cu_from_lengths([5, 0, 7, 300, 1, 1, 0])
    assert B.window_dq_part(P, cu, 2, 72, False) == (14, 25 + 49 + 1 + 1)


def test_computed_pairs_accounting():
    """The bench's tile fill counts the 32x32 blocks each pass multiplies:
    one 100-token sequence is 4 row groups x 4 blocks (16,384 pairs, 10,000
    valid); causal, groups meet 1+2+3+4 (forward, dQ) or 4+3+2+1 (dK/dV)
    blocks; a window of a 5- and a 7-token sequence is one group meeting one
    block."""
    import bench as B
    import paper_2608_07524_amd as P
    for pass_ in (0, 1, 2):
        assert B.computed_pairs(P, [0, 100], 1, 64, False, pass_) == 16 * 1024
        assert B.computed_pairs(P, [0, 100], 1, 64, True, pass_) == 10 * 1024
        assert B.computed_pairs(P, [0, 5, 12], 2, 72, False, pass_) == 1024
    w = I.Workload("t", [100], 1, 64, True, 0.125)
    mw = B.matrix_work(P, w)
    assert mw["fwd_fill"] == 5050 / 10240 and mw["dkdv_fill"] == 5050 / 10240
    assert mw["executed_flop_per_step"] == 2.0 * (2 + 4 + 3) * 10240 * 64
