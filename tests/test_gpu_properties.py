"""GPU properties: run-to-run bitwise determinism of every output, bitwise
invariance of a sequence's outputs to its position in the pack (sequences
that run in tiles of their own), the same within the parity bounds for
short sequences sharing a packed window, and the cost profiler feeding the
planner."""

import math

import numpy as np
import pytest

from oracle import planner as O
from paper_2608_07524_amd import inputs as I

from gpu_util import to_bits, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    t = pytest.importorskip("torch")
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_07524_amd as P
    P.load()
    return t


def _outputs(torch, bits, cu, scale, causal):
    import paper_2608_07524_amd as P
    q, k, v, do = (to_device(torch, b) for b in bits)
    o, lse = P.varlen_attn_fwd(q, k, v, cu, scale, causal)
    dq, dk, dv = P.varlen_attn_bwd(do, o, lse, q, k, v, cu, scale, causal)
    torch.cuda.synchronize()
    return [to_bits(o), lse.cpu().numpy(), to_bits(dq), to_bits(dk), to_bits(dv)]


# (the last two cases run packed windows: at head widths up to 96 their dQ
# comes from the window's dK/dV workgroup through LDS, still without atomics)
@pytest.mark.parametrize("D,causal,lengths", [(72, False, [700, 1, 2049, 300]), (128, True, [700, 1, 2049, 300]),
                                              (72, False, [5, 17, 40, 3, 700, 60, 60, 1, 0, 9, 127]),
                                              (64, True, [5, 17, 40, 3, 700, 60, 60, 1, 0, 9, 127])])
def test_bitwise_deterministic(torch, D, causal, lengths):
    rng = np.random.default_rng(7)
    cu = I.cu_from_lengths(lengths)
    bits = I.tensors(rng, int(cu[-1]), 4, D)
    a = _outputs(torch, bits, cu, 1 / math.sqrt(D), causal)
    b = _outputs(torch, bits, cu, 1 / math.sqrt(D), causal)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("D,causal,lengths", [(128, True, [700, 1, 2049, 300]),
                                              (72, False, [5, 17, 40, 3, 700, 60, 60, 1, 0, 9, 127])])
def test_prepared_batch_equals_per_call(torch, D, causal, lengths):
    """dcp_batch_fwd / _bwd (lists built and uploaded once) give the per-call
    results bit for bit, on repeated calls and after uploading again into a
    second buffer."""
    import paper_2608_07524_amd as P
    rng = np.random.default_rng(11)
    cu = I.cu_from_lengths(lengths)
    bits = I.tensors(rng, int(cu[-1]), 3, D)
    ref = _outputs(torch, bits, cu, 1 / math.sqrt(D), causal)
    q, k, v, do = (to_device(torch, b) for b in bits)
    call = P.PreparedAttention(q, k, v, do, cu, 1 / math.sqrt(D), causal)
    for rep in range(3):
        if rep == 2:  # a second buffer
            call.ws = torch.empty_like(call.ws)
            P.load().dcp_batch_upload(call.batch, call.ws.data_ptr(), call.ws.numel(), call.stream)
        for t in (call.o, call.dq, call.dk, call.dv):
            t.zero_()
        call.step()
        torch.cuda.synchronize()
        got = [to_bits(call.o), call.lse.cpu().numpy(), to_bits(call.dq), to_bits(call.dk), to_bits(call.dv)]
        for x, y in zip(ref, got):
            assert np.array_equal(x, y)


def test_per_call_queue_deeper_than_staging_ring(torch):
    """The per-call entry points stage their lists in a ring of four pinned
    host buffers per device: ten calls enqueued with no synchronisation
    (the ring wraps), with a backward whose lists pass 1 MiB halfway (the
    ring grows while earlier copies may still be in flight), give the
    prepared batch's results bit for bit."""
    import paper_2608_07524_amd as P
    torch.manual_seed(5)
    cases = {"small": ([700, 1, 2049, 300], 4, 128), "large": ([1024] * 128, 64, 64)}
    data, ref = {}, {}
    for name, (lengths, H, D) in cases.items():
        cu = I.cu_from_lengths(lengths)
        T = int(cu[-1])
        q, k, v, do = (torch.randn(T, H, D, device="cuda").to(torch.bfloat16) for _ in range(4))
        call = P.PreparedAttention(q, k, v, do, cu, 1 / math.sqrt(D), True)
        call.step()
        torch.cuda.synchronize()
        data[name] = (cu, q, k, v, do, D)
        ref[name] = [t.clone() for t in (call.o, call.lse, call.dq, call.dk, call.dv)]
        del call
    torch.cuda.synchronize()
    got = []
    for name in ["small"] * 3 + ["large"] + ["small"] * 2:
        cu, q, k, v, do, D = data[name]
        o, lse = P.varlen_attn_fwd(q, k, v, cu, 1 / math.sqrt(D), True)
        if name == "large" or len(got) < 4:
            dq, dk, dv = P.varlen_attn_bwd(do, o, lse, q, k, v, cu, 1 / math.sqrt(D), True)
            got.append((name, [o, lse, dq, dk, dv]))
        else:
            got.append((name, [o, lse]))
    torch.cuda.synchronize()
    for name, outs in got:
        for x, y in zip(outs, ref[name]):
            assert torch.equal(x, y), name


@pytest.mark.parametrize("causal", [False, True])
def test_position_in_pack_invariance(torch, causal):
    """A sequence's outputs do not depend on where it sits in the pack or
    on its neighbours (no cross-sequence reads)."""
    rng = np.random.default_rng(8)
    H, D = 2, 72
    target = I.tensors(rng, 333, H, D)
    left = I.tensors(rng, 517, H, D)
    right = I.tensors(rng, 64, H, D)
    solo = _outputs(torch, target, [0, 333], 0.1, causal)
    packed_bits = [np.concatenate([l, t, r]) for l, t, r in zip(left, target, right)]
    packed = _outputs(torch, packed_bits, [0, 517, 850, 914], 0.1, causal)
    sl = slice(517, 850)
    for i, (x, y) in enumerate(zip(solo, packed)):
        if i == 1:  # LSE is [H, T]
            assert np.array_equal(x, y[:, sl])
        else:
            assert np.array_equal(x, y[sl])


@pytest.mark.parametrize("causal", [False, True])
def test_packed_window_neighbours(torch, causal):
    """A short sequence shares a tile with its short neighbours (a packed
    window): its outputs match those it gets alone within the parity bounds,
    whatever its neighbours hold (each row is masked to its own sequence)."""
    from gpu_util import BF16_U, GRAD_TOL, LSE_TOL, O_TOL
    rng = np.random.default_rng(9)
    H, D = 2, 72
    target = I.tensors(rng, 45, H, D)
    solo = _outputs(torch, target, [0, 45], 0.1, causal)
    for left_len, right_len in [(19, 100), (70, 3), (1, 150)]:
        left = I.tensors(rng, left_len, H, D)
        right = I.tensors(rng, right_len, H, D)
        bits = [np.concatenate([l, t, r]) for l, t, r in zip(left, target, right)]
        cu = [0, left_len, left_len + 45, left_len + 45 + right_len]
        packed = _outputs(torch, bits, cu, 0.1, causal)
        sl = slice(left_len, left_len + 45)
        x = [I.bf16_to_f64(a) for a in (solo[0], packed[0][sl])]
        # each within the O bound of the exact result (bf16 store rounding added)
        assert np.max(np.abs(x[0] - x[1]) - 2 * BF16_U * np.abs(x[0])) <= 2 * O_TOL
        assert np.max(np.abs(solo[1] - packed[1][:, sl])) <= LSE_TOL
        for i in (2, 3, 4):
            a, b = I.bf16_to_f64(solo[i]), I.bf16_to_f64(packed[i][sl])
            assert np.max(np.abs(a - b)) <= GRAD_TOL * np.max(np.abs(a))


def test_profile_cost_rows(torch):
    import paper_2608_07524_amd as P
    lengths = [1024, 2048, 4096, 8192]
    rows = P.profile_cost(lengths, n_heads=2, head_dim=128, warmup=2, reps=5, lin_f_ps_per_token=1000,
                          act_bytes_per_token=34 * 256, inp_bytes_per_token=2 * 256)
    for s, r in zip(lengths, rows):
        print(f"profile s={s}: t_f {r.t_f_ns} ns t_b {r.t_b_ns} ns", flush=True)
        assert r.seq_len == s and r.t_f_ns > 0 and r.t_b_ns > 0
        assert r.m_bytes == 34 * 256 * s and r.m_inp_bytes == 2 * 256 * s
        assert r.t_f_ns >= s  # the linear term alone is 1 ns per token
    # quadratic attention cost: doubling the length at least doubles the time
    for a, b in zip(rows, rows[1:]):
        assert b.t_f_ns > 1.5 * a.t_f_ns and b.t_b_ns > 1.5 * a.t_b_ns
    # a measured table plans bit-exactly against the integer oracle
    table = O.CostTable([O.CostRow(r.seq_len, r.t_f_ns, r.t_b_ns, r.m_bytes, r.m_inp_bytes) for r in rows],
                        28, 100_000, 900 << 20)
    opts = O.PlanOpts(n_heads=16, hidden=1152)
    seqs = [1000, 8000, 3000, 2048, 5000, 700]
    ref = O.plan(seqs, table, 1 << 30, opts)
    got = P.plan(seqs, rows, 28, 100_000, 900 << 20, 1 << 30, n_heads=16, hidden=1152)
    assert (got.sp_size, got.micro_batch, got.grad_accum, got.recompute_layers) == \
        (ref.sp_size, ref.micro_batch, ref.grad_accum, ref.recompute_layers)


def test_text_lm_planning_over_1000_packs(torch):
    """The text-LM workload: profile per-length causal costs at H32, D128,
    then plan 1000 packs in groups of 8 (and 32): bit-exact with the oracle."""
    import paper_2608_07524_amd as P
    lengths = [2 ** e for e in range(7, 18)]
    rows = P.profile_cost(lengths, n_heads=32, head_dim=128, causal=True, warmup=1, reps=3,
                          act_bytes_per_token=34 * 4096, inp_bytes_per_token=2 * 4096)
    table = O.CostTable([O.CostRow(r.seq_len, r.t_f_ns, r.t_b_ns, r.m_bytes, r.m_inp_bytes) for r in rows],
                        42, 1_000_000, 20 << 30)
    packs = I.text_packs(np.random.default_rng(0), 1000)
    budget = 288 << 30
    opts = O.PlanOpts(n_heads=32, hidden=4096, b_max=1)
    for group in (8, 32):
        for g0 in range(0, 1000, group):
            batch = packs[g0:g0 + group]
            seqs = [s for p in batch for s in p.lengths]
            offs = np.concatenate([[0], np.cumsum([len(p.lengths) for p in batch])]).tolist()
            try:
                ref = O.plan(seqs, table, budget, opts, batch_offsets=offs)
            except O.PlanError as e:
                with pytest.raises(P.DCPError) as ei:
                    P.plan(seqs, rows, 42, 1_000_000, 20 << 30, budget, batch_offsets=offs, n_heads=32,
                           hidden=4096, b_max=1)
                assert ei.value.code == e.code
                continue
            got = P.plan(seqs, rows, 42, 1_000_000, 20 << 30, budget, batch_offsets=offs, n_heads=32, hidden=4096,
                         b_max=1)
            for f in ("sp_size", "micro_batch", "grad_accum", "recompute_layers", "step_time_ns", "mem_bytes",
                      "idle_ns", "makespan_ns"):
                assert getattr(got, f) == getattr(ref, f), (g0, f)


def test_device_info(torch):
    """dcp_device_info reports the MI355X's 256 compute units and a plausible
    engine clock (the denominators bench.py states)."""
    import paper_2608_07524_amd as P
    info = P.device_info()
    assert info["compute_units"] == torch.cuda.get_device_properties(0).multi_processor_count
    assert info["compute_units"] >= 256 and 1000.0 < info["clock_mhz"] < 4000.0
