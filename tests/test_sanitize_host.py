"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer.

tests/sanitize/host_driver.cpp links the planner and schedule replay
(dcp_plan.cpp), the work-list builder and descriptor validation
(work_list.cpp) and the error messages (dcp_error.cpp) with the sanitizers
on, and runs them over random and edge-case inputs.  Any sanitizer report
aborts the driver (the test fails); its results are also compared with the
integer oracle (plans, replays) and with the production libdcp.so (work
lists and validation codes), so the sanitized build computes the same
thing.  No GPU is involved."""

import os
import random
import shutil
import subprocess

import numpy as np
import pytest

import paper_2608_07524_amd as P
from oracle import planner as O
from oracle import simulate as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_07524_amd", "csrc")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ is not installed")
    exe = str(tmp_path_factory.mktemp("san") / "host_driver")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "sanitize", "host_driver.cpp"), os.path.join(CSRC, "dcp_plan.cpp"),
           os.path.join(CSRC, "work_list.cpp"), os.path.join(CSRC, "dcp_error.cpp"), "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    return exe


def _run(exe, text):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    res = subprocess.run([exe], input=text, capture_output=True, text=True, env=env, timeout=600)
    assert res.returncode == 0 and "Sanitizer" not in res.stderr and "runtime error" not in res.stderr, \
        res.stderr[-4000:]
    return [list(map(int, l.split())) for l in res.stdout.splitlines()]


def _plan_case(rng):
    n_rows = rng.randint(1, 5)
    lens = sorted(rng.sample(range(1, 5000), n_rows))
    rows = [O.CostRow(s, rng.randint(0, 10 ** rng.randint(1, 9)), rng.randint(0, 10 ** rng.randint(1, 9)),
                      rng.randint(0, 10 ** rng.randint(0, 8)), rng.randint(0, 10 ** rng.randint(0, 7)))
            for s in lens]
    if rng.random() < 0.03:
        rows[0] = O.CostRow(rows[0].seq_len, 1 << 62, 1, 1, 1)  # overflow path
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
    return seqs, t, budget, opts, offs


def _plan_text(tag, seqs, t, budget, o, offs):
    nb = len(seqs) if offs is None else len(offs) - 1
    f = [tag, len(seqs), *seqs, nb, 0 if offs is None else 1, *(offs or []), len(t.rows), t.n_layers, t.T_C_ns,
         t.M_C_bytes]
    for r in t.rows:
        f += [r.seq_len, r.t_f_ns, r.t_b_ns, r.m_bytes, r.m_inp_bytes]
    f += [budget, len(o.sp_cands), *o.sp_cands, o.b_max, o.n_heads, o.hidden, o.a2a_alpha_ns, o.link_bytes_per_ns,
          o.g_min, o.g_max, o.mode, o.flags]
    return " ".join(map(str, f))


def test_planner_and_replay_under_sanitizers(driver):
    rng = random.Random(77)
    cases, lines = [], []
    for _ in range(400):
        c = _plan_case(rng)
        cases.append(("P", c))
        lines.append(_plan_text("P", *c))
    for _ in range(80):
        seqs, t, budget, o, offs = _plan_case(rng)
        W = rng.choice([1, 2, 4, 8, 32])
        extra = (W, rng.choice([0] + list(o.sp_cands)), rng.randint(0, 10 ** 5))
        cases.append(("S", (seqs, t, budget, o, offs, extra)))
        lines.append(_plan_text("S", seqs, t, budget, o, offs) + " " + " ".join(map(str, extra)))
    got = _run(driver, "\n".join(lines) + "\n")
    assert len(got) == len(cases)
    n_ok = 0
    for (tag, c), g in zip(cases, got):
        if tag == "P":
            seqs, t, budget, o, offs = c
            try:
                ref = O.plan(seqs, t, budget, o, batch_offsets=offs)
            except O.PlanError as e:
                assert g == [e.code]
                continue
            exp = [0] + ref.sp_size + ref.micro_batch + ref.grad_accum + ref.recompute_layers + \
                ref.recompute_flags + ref.step_time_ns + ref.mem_bytes + [ref.idle_ns, ref.makespan_ns]
            assert g == exp
            n_ok += 1
        else:
            seqs, t, budget, o, offs, (W, bsp, sync) = c
            try:
                a, b = S.simulate(seqs, t, budget, W, bsp, sync, o, batch_offsets=offs)
            except O.PlanError as e:
                assert g == [e.code]
                continue
            keys = ("iterations", "makespan_ns", "time_ns", "busy_device_ns", "tokens", "bucket_sp")
            assert g == [0] + [a[k] for k in keys] + [b[k] for k in keys]
    assert n_ok > 100


def _random_cu(rng):
    kind = rng.random()
    if kind < 0.3:   # thousands of short sequences (packed windows), with empties
        lens = [rng.choice([0, 1, 2, 7, 16, 31, 51, 64, 100]) for _ in range(rng.randint(1, 3000))]
    elif kind < 0.6:
        lens = [rng.randint(0, 5000) for _ in range(rng.randint(1, 40))]
    else:
        lens = [rng.choice([1, 255, 256, 257, 1024, 70000]) for _ in range(rng.randint(1, 6))]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    return cu


def test_work_lists_and_validation_under_sanitizers(driver):
    rng = random.Random(5)
    lines, cases = [], []
    for _ in range(60):
        cu = _random_cu(rng)
        T = int(cu[-1]) + rng.choice([0, 0, 3])
        H, D, causal = rng.choice([1, 2, 3, 16]), rng.choice([64, 72, 128]), rng.randint(0, 1)
        for pass_ in (0, 1, 2):
            lines.append(" ".join(map(str, ["W", len(cu) - 1, *cu.tolist(), T, H, D, causal, 125, pass_])))
            cases.append(("W", cu, T, H, D, causal, pass_))
        lines.append(" ".join(map(str, ["B", len(cu) - 1, *cu.tolist(), T, H, D, causal, 125])))
        cases.append(("B",))
    bad = [([1, 5], 5, 2, 64, 0, 125), ([0, 5, 3], 5, 2, 64, 0, 125), ([0, 9], 5, 2, 64, 0, 125),
           ([0, 5], 5, 0, 64, 0, 125), ([0, 5], 5, 65536, 64, 0, 125), ([0, 5], 5, 2, 96, 0, 125),
           ([0, 5], 5, 2, 64, 0, 0), ([0, 5], 5, 2, 64, 2, 125), ([0, 5], 1 << 31, 2, 64, 0, 125)]
    for cu, T, H, D, c, sc in bad:
        lines.append(" ".join(map(str, ["W", len(cu) - 1, *cu, T, H, D, c, sc, 0])))
        cases.append(("X", cu, T, H, D, c, sc))
    got = _run(driver, "\n".join(lines) + "\n")
    assert len(got) == len(cases)
    lib = P.load()
    from paper_2608_07524_amd import _native as N
    import ctypes as C
    for case, g in zip(cases, got):
        if case[0] == "W":
            _, cu, T, H, D, causal, pass_ = case
            units, n_tiles, starts = P.work_list(cu, H, D, bool(causal), pass_)
            assert g[:4] == [0, len(units), n_tiles, len(starts)]
            assert g[4:4 + 5 * len(units)] == units.reshape(-1).tolist()
            assert g[4 + 5 * len(units):] == starts.reshape(-1).tolist()
        elif case[0] == "B":
            assert g[0] == 0 and g[1] == 1
        else:
            _, cu, T, H, D, c, sc = case
            cu32 = np.asarray(cu, dtype=np.int32)
            d = N.AttnDesc(cu32.size - 1, cu32.ctypes.data_as(C.POINTER(C.c_int32)), T, H, D, sc / 1000.0, c)
            n = C.c_size_t()
            assert g == [lib.dcp_varlen_attn_fwd_workspace_size(C.byref(d), C.byref(n))] and g[0] < 0


def test_work_list_uploads_under_sanitizers(driver):
    """The work-list upload plan (the segments the per-call calls and the
    prepared batch copy to the device): every list and window mask lands at
    its offset, the bytes between the parts of a segment are zero, nothing
    outside the segments is written, and a per-call workspace's reserved
    space is not copied."""
    rng = random.Random(9)
    lines, kinds = [], []
    for _ in range(40):
        cu = _random_cu(rng)
        T = int(cu[-1]) + rng.choice([0, 3])
        H, D, causal = rng.choice([1, 2, 16, 32]), rng.choice([64, 72, 128]), rng.randint(0, 1)
        for kind in (0, 1, 2):
            lines.append(" ".join(map(str, ["U", len(cu) - 1, *cu.tolist(), T, H, D, causal, 125, kind])))
            kinds.append(kind)
    # the text-pack shape: 75 log-normal documents, 32 heads, causal
    from paper_2608_07524_amd import inputs as I
    w = I.text_packs(np.random.default_rng(0), 1)[0]
    for kind in (0, 1, 2):
        lines.append(" ".join(map(str, ["U", len(w.lengths), *w.cu_seqlens.tolist(), w.total_tokens, 32, 128, 1, 88,
                                        kind])))
        kinds.append(kind)
    got = _run(driver, "\n".join(lines) + "\n")
    assert len(got) == len(kinds)
    for kind, g in zip(kinds, got):
        status, ok, n_segs, staged, part_bytes, area = g
        assert status == 0 and ok == 1
        assert part_bytes <= staged <= part_bytes + (n_segs + 6) * (16 << 10)
    # the per-call backward of the text pack stages its lists, not the reserved space between them
    status, ok, n_segs, staged, part_bytes, area = got[-2]
    assert n_segs >= 2 and staged < area // 4
