"""Schedule replay (no GPU): the C++ dcp_simulate against the integer oracle,
bit for bit, plus a hand-worked example and invariants."""

import numpy as np
import pytest

import paper_2608_07524_amd as D
from oracle import planner as O
from oracle import simulate as S


def _table(rows, L, T_C=0, M_C=0):
    return O.CostTable([O.CostRow(*r) for r in rows], L, T_C, M_C)


def _both(lens, rows, L, T_C, M_C, budget, W, bucket_sp=0, sync=0, offs=None, **opts):
    got = D.simulate(lens, rows, L, T_C, M_C, budget, W, bucket_sp, sync, batch_offsets=offs, **opts)
    po = O.PlanOpts(**{k: (tuple(v) if k == "sp_cands" else v) for k, v in opts.items()})
    ref = S.simulate(lens, _table(rows, L, T_C, M_C), budget, W, bucket_sp, sync, po, batch_offsets=offs)
    return got, ref


def test_hand_worked_two_batches():
    """Two batches of 100 and 200 tokens on W = 2, one layer, full
    recomputation: T = L*(t_f + t_b) + r*t_f gives 40 ns and 160 ns.
    DCP runs them together; Eq. (3) picks C = 160 (idle 0), so g = (4, 1):
    busy = 4*40 + 160 = 320 device-ns, tokens = 4*100 + 200 = 600, no idle.
    Bucket parallelism (p = 1, b_max = 1): one step each, busy 200 of the
    2 * 160 device-ns (imbalance 3/8), 300 tokens."""
    rows = [(100, 10, 20, 0, 0), (200, 40, 80, 0, 0)]
    opts = dict(sp_cands=[1], b_max=1, g_max=4, mode=D.PLAN_INTER, n_heads=1)
    (dcp, bucket), _ = _both([100, 200], rows, 1, 0, 0, 1 << 40, 2, **opts)
    assert dcp == {"iterations": 1, "makespan_ns": 160, "time_ns": 160, "busy_device_ns": 320, "tokens": 600,
                   "bucket_sp": 0}
    assert bucket == {"iterations": 1, "makespan_ns": 160, "time_ns": 160, "busy_device_ns": 200, "tokens": 300,
                      "bucket_sp": 1}
    ref = S.simulate([100, 200], _table(rows, 1), 1 << 40, 2, 0, 0,
                     O.PlanOpts(sp_cands=(1,), b_max=1, g_max=4, mode=O.MODE_INTER, n_heads=1))
    assert (dcp, bucket) == ref
    assert S.imbalance_ratio(dcp, 2) == 0.0 and S.imbalance_ratio(bucket, 2) == 0.375
    # with b_max = 4 the bucket baseline grows the short batch to b = 4
    # (T = 40 b <= 160): 400 + 200 tokens in 320 busy device-ns
    _, bucket4 = D.simulate([100, 200], rows, 1, 0, 0, 1 << 40, 2, sp_cands=[1], b_max=4, g_max=4,
                            mode=D.PLAN_INTER, n_heads=1)
    assert (bucket4["tokens"], bucket4["busy_device_ns"]) == (600, 320)


def test_sync_and_iteration_count():
    """W = 1: every batch is an iteration of its own under both schedules;
    each iteration adds the synchronisation time once."""
    rows = [(64, 5, 9, 10, 1), (128, 11, 20, 20, 2)]
    lens = [64, 128, 64, 128, 128]
    dcp, bucket = D.simulate(lens, rows, 2, 7, 0, 1 << 40, 1, 0, 1000, sp_cands=[1], n_heads=1)
    for r in (dcp, bucket):
        assert r["iterations"] == 5
        assert r["time_ns"] == r["makespan_ns"] + 5 * 1000
        assert r["busy_device_ns"] == r["makespan_ns"]  # one device, never idle


def _random_table(rng, L):
    lens = np.unique(np.concatenate([[128], rng.integers(129, 70000, 12), [131072]]))
    rows, tf, tb, m, mi = [], 0, 0, 0, 0
    for s in lens:
        tf += int(rng.integers(1, 5000)) + int(s) // 3
        tb += int(rng.integers(1, 9000)) + int(s) // 2
        m += int(rng.integers(0, 1 << 20)) + 2000 * int(s)
        mi += int(rng.integers(0, 1 << 16)) + 300 * int(s)
        rows.append((int(s), tf, tb, m, mi))
    return rows


@pytest.mark.parametrize("seed", range(12))
def test_parity_random_streams(seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(1, 40))
    rows = _random_table(rng, L)
    n = int(rng.integers(1, 60))
    lens = np.minimum(131072, np.maximum(1, np.exp(rng.normal(7.5, 1.5, n)).astype(np.int64))).tolist()
    offs = None
    if seed % 2:
        cuts = np.sort(rng.choice(np.arange(1, n), size=min(n - 1, int(rng.integers(0, n))), replace=False)) \
            if n > 1 else np.array([], dtype=np.int64)
        offs = [0] + cuts.tolist() + [n]
    W = int(rng.choice([1, 2, 4, 8, 16, 32]))
    sp = [c for c in (1, 2, 4, 8) if c <= max(W, 1)]
    opts = dict(sp_cands=sp, b_max=int(rng.integers(1, 16)), g_max=int(rng.integers(1, 5)),
                mode=int(rng.integers(0, 2)), n_heads=16, hidden=int(rng.integers(256, 4096)))
    budget = int(rng.integers(1 << 28, 1 << 36))
    sync = int(rng.integers(0, 10 ** 6))
    T_C, M_C = int(rng.integers(0, 10 ** 5)), int(rng.integers(0, 1 << 26))
    bucket_sp = int(rng.choice([0] + sp))
    try:
        ref = S.simulate(lens, _table(rows, L, T_C, M_C), budget, W, bucket_sp, sync,
                         O.PlanOpts(**{k: (tuple(v) if k == "sp_cands" else v) for k, v in opts.items()}),
                         batch_offsets=offs)
    except O.PlanError as e:
        with pytest.raises(D.DCPError) as ei:
            D.simulate(lens, rows, L, T_C, M_C, budget, W, bucket_sp, sync, batch_offsets=offs, **opts)
        assert ei.value.code == e.code
        return
    got = D.simulate(lens, rows, L, T_C, M_C, budget, W, bucket_sp, sync, batch_offsets=offs, **opts)
    assert got == ref
    for r in got:
        assert 0 < r["busy_device_ns"] <= W * r["makespan_ns"]
        assert r["time_ns"] == r["makespan_ns"] + r["iterations"] * sync


def test_errors():
    rows = [(100, 10, 20, 0, 0)]
    # a batch whose only sequence-parallel size exceeds W
    with pytest.raises(D.DCPError) as e:
        D.simulate([100], rows, 1, 0, 0, 1 << 40, 4, sp_cands=[8], n_heads=8)
    assert e.value.code == D.DCP_ERR_INVALID
    with pytest.raises(D.DCPError) as e:
        D.simulate([100], rows, 1, 0, 0, 1 << 40, 0)
    assert e.value.code == D.DCP_ERR_INVALID
    with pytest.raises(D.DCPError) as e:
        D.simulate([100], rows, 1, 0, 0, 1 << 40, 4, bucket_sp=8, sp_cands=[1, 2, 4, 8], n_heads=8)
    assert e.value.code == D.DCP_ERR_INVALID
    with pytest.raises(D.DCPError) as e:  # beyond the table
        D.simulate([101], rows, 1, 0, 0, 1 << 40, 4)
    assert e.value.code == D.DCP_ERR_TABLE


def test_window_fill_hand_worked():
    """Iterations fill their devices from the next batches that fit.  One
    layer, no communication cost, budget 10: a 100-token batch (m_inp 20)
    needs p = 2 (ceil(20/2) = 10), a 200-token batch (m_inp 40) p = 4; step
    times T = ceil(t_f/p) + ceil(t_b/p) = 5 + 10 = 15 and 3 + 5 = 8.  Stream
    (100, 200, 100) on W = 4: the first iteration takes batches 0 and 2
    (2 + 2 devices, g = (1, 1), span 15, busy 60, 200 tokens) while batch 1
    waits; the second runs batch 1 alone (span 8, busy 32, 200 tokens).
    Filling strictly in stream order would need three iterations (38 ns)."""
    rows = [(100, 10, 20, 0, 20), (200, 10, 20, 0, 40)]
    opts = dict(sp_cands=[1, 2, 4], b_max=1, n_heads=4, hidden=0, a2a_alpha_ns=0, g_max=4, mode=D.PLAN_INTRA)
    (dcp, _), (ref, _) = _both([100, 200, 100], rows, 1, 0, 0, 10, 4, sync=7, **opts)
    assert dcp == {"iterations": 2, "makespan_ns": 23, "time_ns": 37, "busy_device_ns": 92, "tokens": 400,
                   "bucket_sp": 0}
    assert dcp == ref


def test_replay_models_follow_the_paper_table():
    """The replay's two models carry the layer counts, hidden sizes, head
    counts and parameter counts of the paper's model-settings table
    (tests/golden/model_settings.json), with head width hidden / heads."""
    import golden_cases
    from paper_2608_07524_amd import replay
    for name, m in golden_cases.load("model_settings.json")["models"].items():
        layers, hidden, heads, head_dim, params, _ = replay.MODELS[name]
        assert (layers, hidden, heads, params) == (m["layers"], m["hidden"], m["heads"], m["params"])
        assert head_dim * heads == hidden
