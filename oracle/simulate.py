"""Integer oracle for the schedule replay: DCP against bucket parallelism
over a stream of batches on W devices.

TEST INFRASTRUCTURE ONLY.  Imported by ``tests/``; the product replay is an
independent C++ implementation behind the C ABI (``dcp_simulate``) and shares
no code with this file.  It builds on ``oracle.planner`` (the planner oracle)
for the per-batch configuration and the accumulation search.

What is replayed, from the paper and the readings taken where it is silent
-------------------------------------------------------------------------
* Eq. (1): n batches share W devices, sum_i p_i = W, per-device throughput
  b_i*s_i / (p_i*T_i).  Reading: an iteration takes, in stream order, every
  batch among the first SIM_WINDOW not yet placed whose p_i still fits its
  free devices; a batch that does not fit keeps its place for a later
  iteration; devices still left over wait out the iteration (their time
  counts as idle).  (Filling strictly in stream order, closing an iteration
  at the first batch that does not fit, left 14 % of device time idle on
  long text with DCP-intra, which gives long batches p = 8.)
* Eq. (3) / Appendix C: within an iteration the accumulation steps g_i
  minimise the idle time against the slowest batch, the iteration lasting at
  most G_max times the slowest step (the planner's rule, reused as is).
* Sec. 4.2: the imbalance ratio is the average share of time a device waits
  for the others; here 1 - busy / (W * makespan) summed over iterations,
  busy = sum_i p_i*g_i*T_i and makespan = max_i g_i*T_i.
* Sec. 4.1 / Sec. 2.4, the bucket-parallel baseline: a fixed
  sequence-parallel size for every batch, static batch sizes that equalise
  the step time -- small batches for long sequences (memory already forces
  them to 1), large ones for short sequences -- and no accumulation.
  Readings: the fixed p is the smallest candidate at which every batch fits
  at batch size 1 (or the caller's), full recomputation as in DCP-inter, the
  batch size of a batch is the largest b <= b_max whose step time stays
  within the slowest batch of the stream at b = 1 and whose memory fits, and
  floor(W / p) batches form an iteration in stream order.
* Sec. 2.4: every iteration ends with one gradient synchronisation, a
  caller-given constant added to both schedules' iteration times.
"""

from __future__ import annotations

from typing import List, Optional, Sequence

from oracle import planner as P


# batches an iteration looks at when filling its devices
SIM_WINDOW = 64


def _empty_result():
    return {"iterations": 0, "makespan_ns": 0, "time_ns": 0, "busy_device_ns": 0, "tokens": 0, "bucket_sp": 0}


def _add(res, span, sync, busy, tokens):
    res["iterations"] += 1
    res["makespan_ns"] = P._fit(res["makespan_ns"] + span)
    res["time_ns"] = P._fit(res["time_ns"] + span + sync)
    res["busy_device_ns"] = P._fit(res["busy_device_ns"] + busy)
    res["tokens"] = P._fit(res["tokens"] + tokens)


def replay_dcp(units, table: P.CostTable, budget: int, o: P.PlanOpts, W: int, sync: int):
    """DCP: planner configuration per batch; each iteration takes, in stream
    order, every batch among the first SIM_WINDOW not yet placed that still
    fits its free devices (sum p_i <= W, Eq. (1)); a batch that does not fit
    waits for a later iteration, keeping its place; accumulation per
    iteration (Eq. (3), Appendix C)."""
    cfg = []
    for i, u in enumerate(units):
        p, b, r, T, _mem = P._choose_config(u, table, budget, o, i)
        if p > W:
            raise P.PlanError(P.ERR_INVALID, f"batch {i} needs {p} devices, more than W")
        if T == 0:
            raise P.PlanError(P.ERR_TABLE, "a batch has zero step time; the cost table is empty of cost")
        cfg.append((p, b, T))
    res = _empty_result()
    pending = list(range(len(units)))  # batches not yet placed, in stream order
    while pending:
        members: List[int] = []
        rest: List[int] = []
        used = 0
        for x, k in enumerate(pending):
            if x < SIM_WINDOW and used + cfg[k][0] <= W:
                members.append(k)
                used += cfg[k][0]
            else:
                rest.append(k)
        pending = rest
        g, _idle, span = P.accumulation_steps([cfg[k][2] for k in members], o.g_min, o.g_max)
        busy = sum(cfg[k][0] * gk * cfg[k][2] for k, gk in zip(members, g))
        tokens = sum(gk * cfg[k][1] * units[k].tokens for k, gk in zip(members, g))
        _add(res, span, sync, busy, tokens)
    return res


def _full_recompute_time(u, table: P.CostTable, o: P.PlanOpts, p: int, b: int):
    """(step time with every layer recomputed, Eq. (6) memory at r = L)."""
    c = P._candidate(u, p, b, table.n_layers, table.M_C_bytes, o)
    return P._step_time(c, table.n_layers, table.n_layers, table.T_C_ns), c.M_bp


def replay_bucket(units, table: P.CostTable, budget: int, o: P.PlanOpts, W: int, sync: int, p_req: int):
    """Bucket parallelism: one p, static batch sizes equalising step time,
    floor(W/p) batches per iteration, no accumulation."""
    def fits(p):
        return all(_full_recompute_time(u, table, o, p, 1)[1] <= budget for u in units)

    if p_req == 0:
        p = None
        for c in o.sp_cands:
            if c > W:
                break
            if not (o.flags & P.FLAG_NO_HEAD_FILTER) and o.n_heads % c != 0:
                continue
            if fits(c):
                p = c
                break
        if p is None:
            raise P.PlanError(P.ERR_INFEASIBLE, "no sequence-parallel size fits every batch at micro-batch 1")
    else:
        p = p_req
        if p > W:
            raise P.PlanError(P.ERR_INVALID, "bucket sequence-parallel size exceeds W")
        if not fits(p):
            raise P.PlanError(P.ERR_INFEASIBLE, "a batch does not fit at the bucket sequence-parallel size")
    target = max(_full_recompute_time(u, table, o, p, 1)[0] for u in units)
    if target == 0:
        raise P.PlanError(P.ERR_TABLE, "a batch has zero step time; the cost table is empty of cost")
    sizes = []
    for u in units:
        # every batch size that meets both limits; the largest is taken
        ok = [b for b in range(1, o.b_max + 1)
              if _full_recompute_time(u, table, o, p, b)[0] <= target
              and _full_recompute_time(u, table, o, p, b)[1] <= budget]
        b = max(ok) if ok else 1
        sizes.append((b, _full_recompute_time(u, table, o, p, b)[0]))
    res = _empty_result()
    res["bucket_sp"] = p
    per = W // p
    for i in range(0, len(units), per):
        chunk = range(i, min(len(units), i + per))
        span = max(sizes[k][1] for k in chunk)
        busy = sum(p * sizes[k][1] for k in chunk)
        tokens = sum(sizes[k][0] * units[k].tokens for k in chunk)
        _add(res, span, sync, busy, tokens)
    return res


def simulate(seq_lens: Sequence[int], table: P.CostTable, hbm_budget: int, n_devices: int, bucket_sp: int = 0,
             iter_sync_ns: int = 0, opts: Optional[P.PlanOpts] = None,
             batch_offsets: Optional[Sequence[int]] = None, n_batches: Optional[int] = None):
    """Both schedules over the stream; returns (dcp, bucket) totals."""
    o = opts or P.PlanOpts()
    seq_lens = [int(s) for s in seq_lens]
    if n_batches is None:
        n_batches = len(seq_lens) if batch_offsets is None else len(batch_offsets) - 1
    if batch_offsets is not None:
        batch_offsets = [int(x) for x in batch_offsets]
    if n_devices < 1 or bucket_sp < 0 or iter_sync_ns < 0:
        raise P.PlanError(P.ERR_INVALID, "need n_devices >= 1, bucket_sp >= 0 and iter_sync_ns >= 0")
    P._validate(seq_lens, batch_offsets, n_batches, table, int(hbm_budget), o)
    units = P._batch_units(seq_lens, batch_offsets, n_batches, table)
    dcp = replay_dcp(units, table, int(hbm_budget), o, int(n_devices), int(iter_sync_ns))
    bucket = replay_bucket(units, table, int(hbm_budget), o, int(n_devices), int(iter_sync_ns), int(bucket_sp))
    return dcp, bucket


def imbalance_ratio(res, n_devices: int) -> float:
    """Share of device time spent waiting (Sec. 4.2)."""
    return 1.0 - res["busy_device_ns"] / (n_devices * res["makespan_ns"])


def throughput(res) -> float:
    """Tokens per second over the replay (Eq. (1) summed over devices)."""
    return res["tokens"] / res["time_ns"] * 1e9
