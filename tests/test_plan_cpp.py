"""The C++ planner behind dcp_plan against the integer oracle: bit-exact
plans and identical status codes, on fixed and random tables."""

import random
import time

import numpy as np
import pytest

import paper_2608_07524_amd as P
from oracle import planner as O

import golden_cases


def _cpp(seqs, table: O.CostTable, budget, opts: O.PlanOpts, batch_offsets=None):
    kw = dict(sp_cands=tuple(opts.sp_cands), b_max=opts.b_max, n_heads=opts.n_heads, hidden=opts.hidden,
              a2a_alpha_ns=opts.a2a_alpha_ns, link_bytes_per_ns=opts.link_bytes_per_ns, g_min=opts.g_min,
              g_max=opts.g_max, mode=opts.mode, flags=opts.flags)
    rows = [(r.seq_len, r.t_f_ns, r.t_b_ns, r.m_bytes, r.m_inp_bytes) for r in table.rows]
    return P.plan(seqs, rows, table.n_layers, table.T_C_ns, table.M_C_bytes, budget, batch_offsets=batch_offsets,
                  **kw)


def _same(seqs, table, budget, opts, batch_offsets=None):
    try:
        ref = O.plan(seqs, table, budget, opts, batch_offsets=batch_offsets)
        ref_err = None
    except O.PlanError as e:
        ref, ref_err = None, e.code
    try:
        got = _cpp(seqs, table, budget, opts, batch_offsets)
        got_err = None
    except P.DCPError as e:
        got, got_err = None, e.code
    assert ref_err == got_err, (ref_err, got_err)
    if ref is not None:
        for f in ("sp_size", "micro_batch", "grad_accum", "recompute_layers", "recompute_flags", "step_time_ns",
                  "mem_bytes", "idle_ns", "makespan_ns"):
            assert getattr(ref, f) == getattr(got, f), f
    return ref_err


def test_defaults_match():
    d = P.default_plan_opts()
    o = O.PlanOpts()
    assert d == dict(sp_cands=tuple(o.sp_cands), b_max=o.b_max, n_heads=o.n_heads, hidden=o.hidden,
                     a2a_alpha_ns=o.a2a_alpha_ns, link_bytes_per_ns=o.link_bytes_per_ns, g_min=o.g_min,
                     g_max=o.g_max, mode=o.mode, flags=o.flags)


def test_hand_example():
    t = O.CostTable([O.CostRow(100, 10, 20, 8, 2)], 4, 5, 10)
    for mode in (0, 1):
        _same([100], t, 60, O.PlanOpts(sp_cands=(1, 2), b_max=2, n_heads=2, hidden=0, a2a_alpha_ns=0,
                                       link_bytes_per_ns=1, mode=mode))


def test_comm_hand_example():
    """The C++ planner on the communication example whose step times are
    worked out by hand in tests/test_oracle_planner.py (Ulysses all-to-all
    term, p in {2, 4}, alpha > 0, hidden > 0)."""
    rows = [(500, 200000, 400000, 0, 500), (1000, 400000, 800000, 0, 1000)]
    kw = dict(sp_cands=(1, 2, 4), n_heads=4, hidden=96, a2a_alpha_ns=100, link_bytes_per_ns=7, g_min=1, g_max=4)
    out = P.plan([1000], rows, 2, 0, 0, 1500, b_max=1, **kw)
    assert (out.sp_size, out.micro_batch, out.recompute_layers, out.step_time_ns) == ([4], [1], [0], [629040])
    out = P.plan([1000], rows, 2, 0, 0, 1500, b_max=1, mode=0, **kw)
    assert (out.recompute_layers, out.step_time_ns) == ([2], [629040 + 2 * 107260])
    out = P.plan([1000], rows, 2, 0, 0, 1500, b_max=2, **kw)
    assert (out.sp_size, out.micro_batch, out.step_time_ns, out.mem_bytes) == ([4], [2], [1256464], [1000])
    assert P.plan([1000], rows, 2, 0, 0, 1500, b_max=1, **dict(kw, sp_cands=(2,))).step_time_ns == [1311328]
    out = P.plan([300, 500], rows, 2, 0, 0, 1500, batch_offsets=[0, 2], b_max=1, **kw)
    assert (out.sp_size, out.step_time_ns) == ([4], [623552])


@pytest.mark.parametrize("case", golden_cases.planner_cases(), ids=lambda c: c["name"])
def test_golden_plans(case):
    """The C++ planner on the hand-worked plans stored in
    tests/golden/planner_hand_examples.json."""
    t = case["table"]
    o = dict(case["opts"], sp_cands=tuple(case["opts"]["sp_cands"]))
    out = P.plan(case["seqs"], t["rows"], t["n_layers"], t["T_C_ns"], t["M_C_bytes"], case["budget"],
                 batch_offsets=case["batch_offsets"], **o)
    for field, want in case["expect"].items():
        assert getattr(out, field) == want, field


def _ci_table(L=28, h=256):
    # per-layer attention-like costs of the tiny packed configuration
    rows = []
    for s in (37, 64, 128, 200):
        tf = 20000 + 50 * s + s * s // 8
        rows.append(O.CostRow(s, tf, 2 * tf, 34 * s * h, 2 * s * h))
    return O.CostTable(rows, L, 100_000, 900 << 20)


@pytest.mark.parametrize("filt", [0, O.FLAG_NO_HEAD_FILTER])
@pytest.mark.parametrize("mode", [0, 1])
def test_tiny_config_plan(mode, filt):
    t = _ci_table()
    opts = O.PlanOpts(sp_cands=(1, 2, 4, 8), b_max=64, n_heads=4, hidden=256, mode=mode, flags=filt)
    assert _same([37, 64, 128, 200], t, 1 << 30, opts) is None


def test_random_tables_bit_exact():
    rng = random.Random(2024)
    n_ok = 0
    for it in range(1200):
        n_rows = rng.randint(1, 5)
        lens = sorted(rng.sample(range(1, 5000), n_rows))
        rows = [O.CostRow(s, rng.randint(0, 10 ** rng.randint(1, 9)), rng.randint(0, 10 ** rng.randint(1, 9)),
                          rng.randint(0, 10 ** rng.randint(0, 8)), rng.randint(0, 10 ** rng.randint(0, 7)))
                for s in lens]
        t = O.CostTable(rows, rng.randint(1, 48), rng.randint(0, 10 ** 6), rng.randint(0, 10 ** 8))
        opts = O.PlanOpts(sp_cands=tuple(sorted(rng.sample([1, 2, 3, 4, 6, 8, 16], rng.randint(1, 5)))),
                          b_max=rng.randint(1, 32), n_heads=rng.choice([1, 2, 4, 8, 16, 48]),
                          hidden=rng.randint(0, 4096), a2a_alpha_ns=rng.randint(0, 20000),
                          link_bytes_per_ns=rng.randint(1, 400), g_min=rng.randint(1, 8), g_max=rng.randint(1, 6),
                          mode=rng.choice([0, 1]), flags=rng.choice([0, 0, 0, 1, 2, 3]))
        n = rng.randint(1, 8)
        seqs = [rng.randint(1, lens[-1] + (50 if rng.random() < 0.05 else 0)) for _ in range(n)]
        offs = None
        if rng.random() < 0.3 and n > 1:
            cut = sorted(rng.sample(range(1, n), rng.randint(1, n - 1)))
            offs = [0] + cut + [n]
        budget = rng.randint(0, 10 ** rng.randint(3, 11))
        if _same(seqs, t, budget, opts, offs) is None:
            n_ok += 1
    assert n_ok > 300


def test_error_codes_match():
    t = O.CostTable([O.CostRow(100, 10, 20, 8, 2)], 4, 5, 10)
    cases = [
        ([0], t, 100, O.PlanOpts()),
        ([50], t, -1, O.PlanOpts()),
        ([50], t, 100, O.PlanOpts(sp_cands=(2, 2))),
        ([50], t, 100, O.PlanOpts(g_max=0)),
        ([50], t, 100, O.PlanOpts(mode=3)),
        ([101], t, 1 << 40, O.PlanOpts()),
        ([50], O.CostTable([O.CostRow(100, 1, 1, 1, 1), O.CostRow(90, 1, 1, 1, 1)], 4, 5, 10), 1 << 40, O.PlanOpts()),
        ([50], O.CostTable([O.CostRow(100, 0, 0, 0, 0)], 4, 0, 0), 1 << 40, O.PlanOpts()),
        ([50], O.CostTable([O.CostRow(100, 1 << 62, 1, 1, 1)], 4, 5, 10), 1 << 40, O.PlanOpts()),
        ([50], t, 5, O.PlanOpts()),
        ([50], t, 1 << 40, O.PlanOpts(n_heads=3, sp_cands=(2, 4))),
    ]
    codes = [_same(*c) for c in cases]
    assert codes == [O.ERR_INVALID, O.ERR_INVALID, O.ERR_INVALID, O.ERR_INVALID, O.ERR_INVALID, O.ERR_TABLE,
                     O.ERR_TABLE, O.ERR_TABLE, O.ERR_INVALID, O.ERR_INFEASIBLE, O.ERR_INFEASIBLE]


def test_replanning_adapts_to_budget():
    """Re-planning each iteration: a smaller budget forces more recompute or
    larger p, and every plan stays bit-exact with the oracle."""
    t = _ci_table()
    opts = O.PlanOpts(sp_cands=(1, 2, 4), n_heads=4, hidden=256)
    prev_r = None
    for budget in (8 << 30, 2 << 30, 1 << 30, (950 << 20)):
        if _same([200, 128], t, budget, opts) is not None:
            continue
        r = O.plan([200, 128], t, budget, opts).recompute_layers
        if prev_r is not None:
            assert sum(r) >= sum(prev_r)
        prev_r = r


def test_planner_latency():
    """32 batches per call on one core: the planner runs every iteration."""
    rng = np.random.default_rng(0)
    rows = [(2 ** e, 10 ** 5 * 2 ** e, 2 * 10 ** 5 * 2 ** e, 2 ** e * 4096, 2 ** e * 512) for e in range(7, 18)]
    seqs = rng.integers(128, 131072, 32).tolist()
    P.plan(seqs, rows, 42, 10 ** 6, 20 << 30, 288 << 30, n_heads=32, hidden=4096)
    t0 = time.perf_counter()
    for _ in range(20):
        P.plan(seqs, rows, 42, 10 ** 6, 20 << 30, 288 << 30, n_heads=32, hidden=4096)
    per_call = (time.perf_counter() - t0) / 20
    assert per_call < 0.05
