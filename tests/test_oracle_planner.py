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

import golden_cases


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


# ------------------------------------------------ communication hand example
# The Ulysses all-to-all term of a candidate (p > 1): four all-to-alls per
# layer in the forward (Q, K, V to head shards, O back) and four in the
# backward (dO out; dQ, dK, dV back).  Each device holds b*S/p tokens of
# `hidden` bf16 values and sends a 1/p share of them to each peer, so every
# link of a fully connected node carries 2*b*S*hidden/p^2 bytes:
#     c(b, p) = 4 * (alpha + ceil(2*b*S*hidden / (p^2 * beta)))      (p > 1)
# Inputs: one row s = 1000 with t_f = 400000, t_b = 800000, m = 0,
# m_inp = 1000 per layer; L = 2, T_C = 0, M_C = 0, budget 1500;
# hidden = 96, alpha = 100 ns, beta = 7 bytes/ns, p in {1, 2, 4}, 4 heads.
# Memory (Eq. (6), r = L): M = 2*ceil(b*1000/p) -> p = 1 needs 2000 > 1500
# (infeasible), (p=2, b=1) 1000, (p=4, b=1) 500, (p=4, b=2) 1000,
# (p=2, b=2) 2000 (infeasible).  m = 0, so no layer is recomputed (r = 0).
# Per-link volume 2*b*1000*96 = 192000*b bytes:
#   (p=2, b=1): 192000/28  = 6857.14 -> 6858, c = 4*(100+6858) = 27832
#               t_f = 200000+27832 = 227832, t_b = 400000+27832 = 427832
#               T = 2*(t_f+t_b) = 1311328, p*T/b = 2622656
#   (p=4, b=1): 192000/112 = 1714.29 -> 1715, c = 4*1815 = 7260
#               t_f = 107260, t_b = 207260, T = 629040, p*T/b = 2516160
#   (p=4, b=2): 384000/112 = 3428.57 -> 3429, c = 4*3529 = 14116
#               t_f = 200000+14116 = 214116, t_b = 414116, T = 1256464,
#               p*T/b = 2512928
# Eq. (1) throughput b/(p*T): with b_max = 1, (p=4, b=1, T=629040) beats
# (p=2, T=1311328); with b_max = 2, (p=4, b=2, T=1256464) wins because the
# latency alpha is paid once for twice the tokens.  Mistakes this catches:
# p instead of p^2 gives c = 55260 at p = 2 and 27832 at p = 4, and then
# (p=2) wins (2842080 < 2845312); eight all-to-alls instead of four double
# every c; a floor instead of the ceiling gives 27828 and 7256.
# A pack of 300 + 500 tokens (both take the s = 500 row, t_f = 200000,
# t_b = 400000, m_inp = 500 each) moves S = 800 tokens, not the rows' 1000:
#   (p=2): 153600/28 = 5485.71 -> 5486, c = 22344, T = 2*(222344+422344) = 1289376
#   (p=4): 153600/112 = 1371.43 -> 1372, c = 5888, T = 2*(105888+205888) = 623552

COMM_OPTS = dict(sp_cands=(1, 2, 4), n_heads=4, hidden=96, a2a_alpha_ns=100, link_bytes_per_ns=7, g_min=1, g_max=4)
COMM_TABLE = ((500, 200000, 400000, 0, 500), (1000, 400000, 800000, 0, 1000))


@pytest.mark.parametrize("case", golden_cases.planner_cases(), ids=lambda c: c["name"])
def test_golden_plans(case):
    """The hand-worked plans above, stored with their citations in
    tests/golden/planner_hand_examples.json."""
    t = case["table"]
    table = _table(t["rows"], L=t["n_layers"], T_C=t["T_C_ns"], M_C=t["M_C_bytes"])
    o = dict(case["opts"], sp_cands=tuple(case["opts"]["sp_cands"]))
    out = P.plan(case["seqs"], table, case["budget"], P.PlanOpts(**o), batch_offsets=case["batch_offsets"])
    for field, want in case["expect"].items():
        assert getattr(out, field) == want, field


def test_golden_accumulation():
    for c in golden_cases.load("planner_hand_examples.json")["accumulation"]["cases"]:
        e = c["expect"]
        assert P.accumulation_steps(c["step_times"], c["g_min"], c["g_max"]) == (e["g"], e["idle"], e["C"])


def test_comm_hand_example():
    t = _table(COMM_TABLE, L=2, T_C=0, M_C=0)
    for mode in (P.MODE_INTRA, P.MODE_INTER):
        out = P.plan([1000], t, 1500, P.PlanOpts(b_max=1, mode=mode, **COMM_OPTS))
        r = 0 if mode == P.MODE_INTRA else 2
        # (full recomputation adds r*t_f: 2*107260)
        assert (out.sp_size, out.micro_batch, out.recompute_layers) == ([4], [1], [r])
        assert out.step_time_ns == [629040 + r * 107260] and out.mem_bytes == [500]
    out = P.plan([1000], t, 1500, P.PlanOpts(b_max=2, **COMM_OPTS))
    assert (out.sp_size, out.micro_batch, out.step_time_ns, out.mem_bytes) == ([4], [2], [1256464], [1000])
    # each p alone: the step times of the derivation above
    assert P.plan([1000], t, 1500, P.PlanOpts(b_max=1, **dict(COMM_OPTS, sp_cands=(2,)))).step_time_ns == [1311328]
    assert P.plan([1000], t, 1500, P.PlanOpts(b_max=1, **dict(COMM_OPTS, sp_cands=(4,)))).step_time_ns == [629040]
    # a pack moves its own tokens
    pk = P.plan([300, 500], t, 1500, P.PlanOpts(b_max=1, **dict(COMM_OPTS, sp_cands=(2,))), batch_offsets=[0, 2])
    assert pk.step_time_ns == [1289376]
    pk = P.plan([300, 500], t, 1500, P.PlanOpts(b_max=1, **COMM_OPTS), batch_offsets=[0, 2])
    assert (pk.sp_size, pk.step_time_ns) == ([4], [623552])


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
