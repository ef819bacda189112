"""Pins for the integer planner oracle, on the CPU.

The planner oracle is checked against exhaustive searches written directly
from Eqs. (3)-(6) (every (p, b, r) triple, every accumulation vector), a
hand-worked example, closed-form special cases and monotonicity properties
that any correct throughput maximiser must have.
"""

import random
from fractions import Fraction

import pytest

from oracle import planner as P


def _table(rows, L=4, T_C=5, M_C=10):
    return P.CostTable([P.CostRow(*r) for r in rows], L, T_C, M_C)


# ---------------------------------------------------------------- hand example
# One profile row (s = 100): t_f = 10, t_b = 20, m = 8, m_inp = 2 per layer,
# L = 4, T_C = 5, M_C = 10, capacity M = 60, p in {1, 2}, b in {1, 2}, and no
# communication cost (alpha = 0, hidden = 0).
#
# DCP-intra, Eq. (6) gives the fewest recomputed layers r and Eqs. (4)-(5) the
# time T = 4*(t_f + t_b) + r*t_f + 5:
#   (p=1,b=1): t_f=10 t_b=20 m=8  m_inp=2  base 4*2+10=18, 4 stashed layers fit
#              (18+32=50<=60) -> r=0, T=125, throughput 1/125
#   (p=1,b=2): t_f=20 t_b=40 m=16 m_inp=4  base 26, (60-26)//16 = 2 stashed
#              -> r=2, M=58, T=4*60+2*20+5=285, throughput 2/285
#   (p=2,b=1): t_f=5  t_b=10 m=4  m_inp=1  base 14 -> r=0, T=65, 1/(2*65)
#   (p=2,b=2): t_f=10 t_b=20 m=8  m_inp=2  base 18 -> r=0, T=125, 2/(2*125)
#   best 1/125, tied by (2,2); the smaller p wins -> (p=1, b=1, r=0, T=125).
# DCP-inter keeps r = L = 4:  T = 4*(t_f+t_b) + 4*t_f + 5
#   (1,1): 165 -> 1/165; (1,2): 325 -> 2/325; (2,1): 85 -> 1/170;
#   (2,2): 165 -> 2/330.  Best (p=1, b=2, r=4, T=325).
# Accumulation (Eq. (3), Appendix C) for step times (3, 5, 4) and G_max = 4:
#   iteration length C <= 20; idle(C) = sum_i C mod T_i is 2 at C = 12, 16,
#   20 and larger elsewhere, so C = 12 and g = (4, 2, 3).  With G_min = 6 the
#   largest g (4) is below 6, so all scale by ceil(6/4) = 2 -> (8, 4, 6).

HAND_OPTS = dict(sp_cands=(1, 2), b_max=2, n_heads=2, hidden=0, a2a_alpha_ns=0, link_bytes_per_ns=1)


def test_hand_example_intra():
    t = _table([(100, 10, 20, 8, 2)])
    out = P.plan([100], t, 60, P.PlanOpts(mode=P.MODE_INTRA, **HAND_OPTS))
    assert (out.sp_size, out.micro_batch, out.recompute_layers, out.step_time_ns) == ([1], [1], [0], [125])
    assert out.mem_bytes == [50] and out.grad_accum == [1] and out.recompute_flags == [0, 0, 0, 0]


def test_hand_example_inter():
    t = _table([(100, 10, 20, 8, 2)])
    out = P.plan([100], t, 60, P.PlanOpts(mode=P.MODE_INTER, **HAND_OPTS))
    assert (out.sp_size, out.micro_batch, out.recompute_layers, out.step_time_ns) == ([1], [2], [4], [325])
    assert out.recompute_flags == [1, 1, 1, 1] and out.mem_bytes == [26]


def test_hand_example_accumulation():
    assert P.accumulation_steps([3, 5, 4], 1, 4) == ([4, 2, 3], 2, 12)
    assert P.accumulation_steps([3, 5, 4], 6, 4) == ([8, 4, 6], 4, 24)


# ------------------------------------------------------------ brute force pins

def _random_case(rng):
    n_rows = rng.randint(1, 4)
    lens = sorted(rng.sample(range(1, 400), n_rows))
    rows = [(s, rng.randint(0, 300), rng.randint(0, 600), rng.randint(0, 50), rng.randint(0, 20)) for s in lens]
    L = rng.randint(1, 6)
    table = _table(rows, L=L, T_C=rng.randint(0, 40), M_C=rng.randint(0, 100))
    opts = P.PlanOpts(sp_cands=tuple(sorted(rng.sample([1, 2, 3, 4, 8], rng.randint(1, 4)))),
                      b_max=rng.randint(1, 5), n_heads=rng.choice([1, 2, 4, 6, 8, 12]),
                      hidden=rng.randint(0, 64), a2a_alpha_ns=rng.randint(0, 50),
                      link_bytes_per_ns=rng.randint(1, 200), g_min=rng.randint(1, 6), g_max=rng.randint(1, 5),
                      mode=rng.choice([0, 1]), flags=rng.choice([0, 0, 1, 2, 3]))
    n = rng.randint(1, 4)
    seqs = [rng.randint(1, lens[-1]) for _ in range(n)]
    budget = rng.randint(0, 1500)
    return seqs, table, budget, opts


def test_config_choice_matches_brute_force():
    rng = random.Random(1234)
    checked = 0
    for _ in range(1500):
        seqs, table, budget, opts = _random_case(rng)
        try:
            out = P.plan(seqs, table, budget, opts)
        except P.PlanError as e:
            # the only legal failures here: nothing fits, or zero cost
            assert e.code in (P.ERR_INFEASIBLE, P.ERR_TABLE)
            if e.code == P.ERR_INFEASIBLE:
                assert any(P.brute_force_config(s, *(_row(table, s)), table, budget, opts) is None for s in seqs)
            continue
        for i, s in enumerate(seqs):
            bf = P.brute_force_config(s, *(_row(table, s)), table, budget, opts)
            assert bf == (out.sp_size[i], out.micro_batch[i], out.recompute_layers[i], out.step_time_ns[i])
        checked += 1
    assert checked > 500


def _row(table, s):
    r = next(r for r in table.rows if r.seq_len >= s)
    return r.t_f_ns, r.t_b_ns, r.m_bytes, r.m_inp_bytes


def test_accumulation_matches_brute_force():
    rng = random.Random(99)
    for _ in range(1500):
        n = rng.randint(1, 4)
        T = [rng.randint(1, 40) for _ in range(n)]
        g_min, g_max = rng.randint(1, 7), rng.randint(1, 4)
        assert P.accumulation_steps(T, g_min, g_max) == P.brute_force_accumulation(T, g_min, g_max)


# --------------------------------------------------------------- closed forms

def test_accumulation_special_cases():
    assert P.accumulation_steps([17], 1, 4) == ([1], 0, 17)
    assert P.accumulation_steps([17], 3, 4) == ([3], 0, 51)
    assert P.accumulation_steps([9, 9, 9], 1, 4)[0] == [1, 1, 1]
    # a batch twice as fast runs twice
    assert P.accumulation_steps([10, 20], 1, 4) == ([2, 1], 0, 20)


def test_planner_special_cases():
    t = _table([(100, 10, 20, 8, 2), (200, 40, 80, 16, 4)], L=6)
    huge = 1 << 60
    out = P.plan([100, 200, 150], t, huge, P.PlanOpts(mode=P.MODE_INTRA))
    assert out.recompute_layers == [0, 0, 0]
    out = P.plan([100, 200, 150], t, huge, P.PlanOpts(mode=P.MODE_INTER))
    assert out.recompute_layers == [6, 6, 6] and all(out.recompute_flags)
    t0 = _table([(100, 10, 20, 0, 2)], L=6)
    assert P.plan([50], t0, 10 ** 6, P.PlanOpts()).recompute_layers == [0]
    # below the constant plus input activations at b = 1 on the largest p
    with pytest.raises(P.PlanError) as e:
        P.plan([100], t, 10 + 6 * 1 - 1, P.PlanOpts(sp_cands=(1, 2), n_heads=2))
    assert e.value.code == P.ERR_INFEASIBLE
    with pytest.raises(P.PlanError) as e:
        P.plan([201], t, huge, P.PlanOpts())
    assert e.value.code == P.ERR_TABLE


def test_invalid_inputs_report_codes():
    t = _table([(100, 10, 20, 8, 2)])
    bad = [
        (dict(seq_lens=[0]), P.ERR_INVALID),
        (dict(budget=-1), P.ERR_INVALID),
        (dict(opts=P.PlanOpts(sp_cands=(2, 1))), P.ERR_INVALID),
        (dict(opts=P.PlanOpts(b_max=0)), P.ERR_INVALID),
        (dict(opts=P.PlanOpts(flags=64)), P.ERR_INVALID),
        (dict(table=_table([(100, 1, 1, 1, 1), (100, 2, 2, 2, 2)])), P.ERR_TABLE),
        (dict(table=_table([(100, -1, 1, 1, 1)])), P.ERR_TABLE),
        (dict(seq_lens=[50, 60], batch_offsets=[0, 0, 2]), P.ERR_INVALID),
        (dict(table=_table([(100, 0, 0, 0, 0)], L=2, T_C=0, M_C=0)), P.ERR_TABLE),
        (dict(table=_table([(100, 1 << 62, 1, 1, 1)])), P.ERR_INVALID),
    ]
    for kw, code in bad:
        args = dict(seq_lens=[50], table=t, budget=1 << 40, opts=P.PlanOpts(), batch_offsets=None)
        args.update(kw)
        with pytest.raises(P.PlanError) as e:
            P.plan(args["seq_lens"], args["table"], args["budget"], args["opts"], args["batch_offsets"])
        assert e.value.code == code, kw


# ------------------------------------------------------------- monotonicity

def _throughput(out, i, tokens):
    return Fraction(out.micro_batch[i] * tokens, out.sp_size[i] * out.step_time_ns[i])


def test_monotone_in_budget_comm_and_mode():
    rng = random.Random(7)
    t = _table([(1024, 2000, 4000, 900, 100), (4096, 20000, 40000, 3600, 400),
                (16384, 300000, 600000, 14400, 1600)], L=8, T_C=1000, M_C=5000)
    for _ in range(200):
        s = rng.choice([500, 1024, 3000, 16000])
        base = dict(sp_cands=(1, 2, 4, 8), b_max=8, n_heads=8, hidden=rng.randint(1, 512),
                    a2a_alpha_ns=rng.randint(0, 5000), link_bytes_per_ns=rng.randint(1, 300))
        budgets = sorted(rng.randint(20000, 400000) for _ in range(3))
        prev = None
        for M in budgets:
            try:
                out = P.plan([s], t, M, P.PlanOpts(**base))
            except P.PlanError:
                assert prev is None
                continue
            th = _throughput(out, 0, s)
            assert prev is None or th >= prev
            prev = th
            inter = P.plan([s], t, M, P.PlanOpts(mode=P.MODE_INTER, **base))
            assert th >= _throughput(inter, 0, s)
            slower = dict(base, a2a_alpha_ns=base["a2a_alpha_ns"] + 1000)
            assert _throughput(P.plan([s], t, M, P.PlanOpts(**slower)), 0, s) <= th
            narrower = dict(base, link_bytes_per_ns=max(1, base["link_bytes_per_ns"] // 2))
            assert _throughput(P.plan([s], t, M, P.PlanOpts(**narrower)), 0, s) <= th


def test_packs_sum_their_rows():
    t = _table([(100, 10, 20, 8, 2), (200, 40, 80, 16, 4)], L=3)
    a = P.plan([60, 150, 100], t, 1 << 40, P.PlanOpts(b_max=1, sp_cands=(1,)), batch_offsets=[0, 2, 3])
    # first pack: rows 100 and 200 -> t_f = 50, t_b = 100; L*(50+100) + 0 + 5
    assert a.step_time_ns[0] == 3 * 150 + 5
    assert a.step_time_ns[1] == 3 * 30 + 5
