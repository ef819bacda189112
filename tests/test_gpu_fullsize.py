"""GPU parity at the benchmark's full sizes, in the launch configuration
bench.py times.

Every output the oracle can evaluate one row at a time is checked on a
seeded sample: O, LSE and dQ rows (the first and last rows of sequences
always included).  dK and dV rows need the whole softmax column of a key,
so they are checked on sampled keys of sampled (sequence, head) pairs, plus,
for every (sequence, head), the exact identities sum_j dV_j = sum_i dO_i and
sum_j dK_j = 0.  The longest sequences of the long-sequence workloads get
dense checks: at least 512 query rows (O, LSE, dQ) and 512 key rows (dK, dV)
per checked (sequence, head), always including its first and last 64.  Key
columns of sequences up to 32k tokens come from the full-row oracle; beyond
that (the 128k and 256k Ulysses shards) from the column oracle given each
query's LSE and Delta, taken from the GPU's own LSE and O after those have
passed their row checks against the full-row oracle (a bound of 5e-3 on
LSE moves the reference gradients by at most 0.5 %, inside the 2e-2 bound).
"""

import math

import numpy as np
import pytest

from oracle import attention as A
from paper_2608_07524_amd import inputs as I

from gpu_util import BF16_U, GRAD_TOL, LSE_TOL, O_TOL, to_bits, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    t = pytest.importorskip("torch")
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2608_07524_amd as P
    P.load()
    return t


def _run(torch, w, rng):
    import paper_2608_07524_amd as P
    T, H, D = w.total_tokens, w.n_heads, w.head_dim
    bits = I.tensors(rng, T, H, D)
    q, k, v, do = (to_device(torch, b) for b in bits)
    call = P.PreparedAttention(q, k, v, do, w.cu_seqlens, w.scale, w.causal)
    call.fwd()
    call.bwd()
    torch.cuda.synchronize()
    out = dict(o=to_bits(call.o), lse=call.lse.cpu().numpy(), dq=to_bits(call.dq), dk=to_bits(call.dk),
               dv=to_bits(call.dv))
    del call, q, k, v, do
    torch.cuda.empty_cache()
    return bits, out


def _sample_rows(rng, cu, H, n_random):
    rows, heads = [], []
    for b in range(len(cu) - 1):
        if cu[b + 1] > cu[b]:
            rows += [int(cu[b]), int(cu[b + 1]) - 1]
            heads += [int(rng.integers(H)), int(rng.integers(H))]
    r = rng.integers(0, int(cu[-1]), n_random)
    rows += r.tolist()
    heads += rng.integers(0, H, n_random).tolist()
    return np.array(rows), np.array(heads)


def _check_rows(bits, out, w, rng, n_random, label):
    cu = w.cu_seqlens
    rows, heads = _sample_rows(rng, cu, w.n_heads, n_random)
    # float32 holds bf16 exactly; the oracle widens every slice it uses to float64
    q, k, v, do = (I.bf16_to_f32(b) for b in bits)
    ro, rl = A.attention_rows(q, k, v, cu, w.scale, w.causal, rows, heads)
    rdq = A.attention_dq_rows(do, q, k, v, cu, w.scale, w.causal, rows, heads)
    go = I.bf16_to_f64(out["o"][rows, heads])
    gl = out["lse"][heads, rows]
    gdq = I.bf16_to_f64(out["dq"][rows, heads])
    eo = float(np.max(np.abs(go - ro)))
    xo = float(np.max(np.abs(go - ro) - BF16_U * np.abs(ro)))  # beyond the bf16 store rounding
    el = float(np.max(np.abs(gl - rl)))
    # dQ relative to the largest reference magnitude over the sampled rows
    edq = float(np.max(np.abs(gdq - rdq)) / np.max(np.abs(rdq)))
    print(f"{label}: {rows.size} sampled rows: O {eo:.2e} LSE {el:.2e} dQ {edq:.2e}", flush=True)
    assert xo <= O_TOL and el <= LSE_TOL and edq <= GRAD_TOL
    return q, k, v, do


def _check_keys(q, k, v, do, out, w, rng, max_len, n_pairs, label):
    cu = w.cu_seqlens
    lens = np.diff(cu)
    # one-token sequences have dK identically zero: see _check_single_tokens
    cand = [b for b in range(len(lens)) if 1 < lens[b] <= max_len]
    if not cand:
        return
    for b in rng.choice(cand, size=min(n_pairs, len(cand)), replace=False):
        h = int(rng.integers(w.n_heads))
        s0, s1 = int(cu[b]), int(cu[b + 1])
        keys = np.unique(np.concatenate([[s0, s1 - 1], rng.integers(s0, s1, 62)]))
        heads = np.full(keys.size, h)
        rdk, rdv = A.attention_dkdv_rows(do, q, k, v, cu, w.scale, w.causal, keys, heads)
        # scale: the largest gradient magnitude in this (sequence, head)
        full_dk = I.bf16_to_f64(out["dk"][s0:s1, h])  # (sequence, head) slice only
        full_dv = I.bf16_to_f64(out["dv"][s0:s1, h])
        ek = float(np.max(np.abs(full_dk[keys - s0] - rdk)) / max(np.max(np.abs(rdk)), np.max(np.abs(full_dk))))
        ev = float(np.max(np.abs(full_dv[keys - s0] - rdv)) / max(np.max(np.abs(rdv)), np.max(np.abs(full_dv))))
        print(f"{label}: seq {b} (len {s1 - s0}) head {h}: dK {ek:.2e} dV {ev:.2e}", flush=True)
        assert ek <= GRAD_TOL and ev <= GRAD_TOL


def _check_identities(q, v, do, out, w, label):
    """sum_j dV_j = sum_i dO_i and sum_j dK_j = 0 per (sequence, head).

    Both hold exactly because each row of P sums to 1.  The kernels use
    bf16-rounded P (each within 2^-9) built from an LSE whose row sum was
    itself taken over bf16-rounded weights (within 2^-9), so
    |sum_j P_ij - 1| <= 2^-8, and every output is rounded to bf16 (2^-9):
      |sum dV - sum dO| <= 2^-8 (sum_j |dV_j| + sum_i |dO_i|);
      |sum dK|          <= 2^-8 sum_j |dK_j| + 2^-8 scale sum_i |q_i|
                           (sum_d |dO_id O_id| + |dO_i| max_j |v_j|),
    the last term covering sum_j dS_ij = Delta_i (sum_j P_ij - 1) with
    Delta = dO . bf16(O), and the rounding of each dS_ij
    (sum_j |dS_ij| <= 2 |dO_i| max_j |v_j|, Cauchy-Schwarz)."""
    cu = w.cu_seqlens
    worst_v = worst_k = 0.0
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        if s1 - s0 < 2:  # empty, or one token (_check_single_tokens)
            continue
        dk = I.bf16_to_f64(out["dk"][s0:s1])
        dv = I.bf16_to_f64(out["dv"][s0:s1])
        o = I.bf16_to_f64(out["o"][s0:s1])
        dob = np.asarray(do[s0:s1], dtype=np.float64)
        qb = np.asarray(q[s0:s1], dtype=np.float64)
        vb = np.asarray(v[s0:s1], dtype=np.float64)
        bound_v = 2.0 ** -8 * (np.abs(dv).sum(0) + np.abs(dob).sum(0)) + 1e-30
        vmax = np.sqrt((vb * vb).sum(-1)).max(0)                       # [H]
        row = np.abs(dob * o).sum(-1) + np.sqrt((dob * dob).sum(-1)) * vmax   # [rows, H]
        bound_k = 2.0 ** -8 * (np.abs(dk).sum(0) + w.scale * (np.abs(qb) * row[:, :, None]).sum(0)) + 1e-30
        ev = np.abs(dv.sum(0) - dob.sum(0)) / bound_v
        ek = np.abs(dk.sum(0)) / bound_k
        worst_v, worst_k = max(worst_v, float(ev.max())), max(worst_k, float(ek.max()))
    print(f"{label}: identity residual / rounding bound: dV {worst_v:.3f} dK {worst_k:.3f}", flush=True)
    assert worst_v <= 1.0 and worst_k <= 1.0


def _dense_rows(rng, s0, s1, n=512, edge=64):
    """At least n rows of [s0, s1) (all of them when shorter), always
    including the first and last `edge`."""
    if s1 - s0 <= n:
        return np.arange(s0, s1)
    fixed = np.concatenate([np.arange(s0, s0 + edge), np.arange(s1 - edge, s1)])
    rest = np.setdiff1d(np.arange(s0 + edge, s1 - edge), fixed)
    return np.sort(np.concatenate([fixed, rng.choice(rest, n - 2 * edge, replace=False)]))


def _rel(got, ref, scale):
    return float(np.max(np.abs(got - ref)) / max(scale, 1e-30))


def _check_dense(q, k, v, do, out, w, rng, seq_heads, label, exact_max=32768):
    """Dense checks of whole (sequence, head) pairs: >= 512 query rows (O,
    LSE, dQ) and >= 512 key rows (dK, dV).  Gradient errors are taken
    relative to the largest magnitude of the reference or of the GPU's
    (sequence, head) slice."""
    cu = w.cu_seqlens
    for b, h in seq_heads:
        s0, s1 = int(cu[b]), int(cu[b + 1])
        rows = _dense_rows(rng, s0, s1)
        heads = np.full(rows.size, h)
        ro, rl = A.attention_rows(q, k, v, cu, w.scale, w.causal, rows, heads)
        rdq = A.attention_dq_rows(do, q, k, v, cu, w.scale, w.causal, rows, heads)
        go = I.bf16_to_f64(out["o"][rows, h])
        xo = float(np.max(np.abs(go - ro) - BF16_U * np.abs(ro)))
        el = float(np.max(np.abs(out["lse"][h, rows] - rl)))
        full_dq = I.bf16_to_f64(out["dq"][s0:s1, h])
        edq = _rel(full_dq[rows - s0], rdq, max(np.max(np.abs(rdq)), np.max(np.abs(full_dq))))
        keys = _dense_rows(rng, s0, s1)
        kh = np.full(keys.size, h)
        if s1 - s0 <= exact_max:
            rdk, rdv = A.attention_dkdv_rows(do, q, k, v, cu, w.scale, w.causal, keys, kh)
            how = "full-row oracle"
        else:
            # normalisers of every query of the sequence from the GPU (LSE
            # checked above on this pair's rows; Delta = dO . O in float64)
            lse = np.zeros((w.n_heads, int(cu[-1])))
            lse[h, s0:s1] = out["lse"][h, s0:s1]
            delta = np.zeros_like(lse)
            delta[h, s0:s1] = np.einsum("td,td->t", np.asarray(do[s0:s1, h], dtype=np.float64),
                                        I.bf16_to_f64(out["o"][s0:s1, h]))
            rdk, rdv = A.attention_dkdv_cols_given(do, q, k, v, cu, w.scale, w.causal, keys, kh, lse, delta)
            how = "column oracle given the checked LSE and Delta"
        full_dk = I.bf16_to_f64(out["dk"][s0:s1, h])
        full_dv = I.bf16_to_f64(out["dv"][s0:s1, h])
        ek = _rel(full_dk[keys - s0], rdk, max(np.max(np.abs(rdk)), np.max(np.abs(full_dk))))
        ev = _rel(full_dv[keys - s0], rdv, max(np.max(np.abs(rdv)), np.max(np.abs(full_dv))))
        print(f"{label}: seq {b} (len {s1 - s0}) head {h}: {rows.size} query rows O {xo:.2e} LSE {el:.2e} "
              f"dQ {edq:.2e}; {keys.size} key rows ({how}) dK {ek:.2e} dV {ev:.2e}", flush=True)
        assert xo <= O_TOL and el <= LSE_TOL and edq <= GRAD_TOL and ek <= GRAD_TOL and ev <= GRAD_TOL


def test_video_short_mix_bench_batch(torch):
    """32 clips of 1k..8k tokens, H16, D72: the exact batch bench.py times."""
    rng = np.random.default_rng(0)
    w = I.video_short_mix(rng)
    bits, out = _run(torch, w, rng)
    srng = np.random.default_rng(100)
    q, k, v, do = _check_rows(bits, out, w, srng, 2048, "video short")
    _check_keys(q, k, v, do, out, w, srng, 8192, 4, "video short")
    _check_identities(q, v, do, out, w, "video short")


def test_video_long_tail_pack(torch):
    rng = np.random.default_rng(0)
    w = I.video_long_tail_packs(rng, n_packs=1)[0]
    bits, out = _run(torch, w, rng)
    srng = np.random.default_rng(101)
    q, k, v, do = _check_rows(bits, out, w, srng, 1024, "video long-tail")
    _check_keys(q, k, v, do, out, w, srng, 8192, 3, "video long-tail")
    _check_identities(q, v, do, out, w, "video long-tail")


@pytest.mark.parametrize("length", [131072, 262144])
def test_ulysses_shard(torch, length):
    """One device's Ulysses shard: a single sequence, 2 heads, D128."""
    rng = np.random.default_rng(0)
    w = I.ulysses_shard(length)
    bits, out = _run(torch, w, rng)
    srng = np.random.default_rng(102)
    q, k, v, do = _check_rows(bits, out, w, srng, 384, f"ulysses {length}")
    _check_identities(q, v, do, out, w, f"ulysses {length}")
    _check_dense(q, k, v, do, out, w, srng, [(0, 0), (0, 1)], f"ulysses {length}")


def test_ulysses_shape_keys_at_16k(torch):
    """Same launch configuration as the Ulysses shard (H2, D128, one
    sequence) at a length whose key columns the oracle evaluates quickly."""
    rng = np.random.default_rng(3)
    w = I.Workload("ulysses-shaped 16k", [16384], 2, 128, False, 1 / math.sqrt(128))
    bits, out = _run(torch, w, rng)
    srng = np.random.default_rng(103)
    q, k, v, do = _check_rows(bits, out, w, srng, 256, "16k")
    _check_keys(q, k, v, do, out, w, srng, 16384, 1, "16k")


def test_text_causal_pack(torch):
    """Log-normal documents packed to 256k tokens, causal, H32, D128."""
    rng = np.random.default_rng(0)
    w = I.text_packs(rng, 1)[0]
    bits, out = _run(torch, w, rng)
    srng = np.random.default_rng(104)
    q, k, v, do = _check_rows(bits, out, w, srng, 256, "text causal")
    _check_keys(q, k, v, do, out, w, srng, 4096, 3, "text causal")
    _check_identities(q, v, do, out, w, "text causal")
    # the three longest documents, one head each, densely
    lens = np.diff(w.cu_seqlens)
    longest = np.argsort(lens)[::-1][:3]
    assert lens[longest[-1]] > 4096
    _check_dense(q, k, v, do, out, w, srng, [(int(b), int(srng.integers(w.n_heads))) for b in longest],
                 "text causal")


def test_text_causal_pack_over_2gib(torch):
    """A causal text pack of 327,680 tokens (H32, D128): every [T, H, D]
    tensor holds 2.68e9 bytes, beyond 2^31, so rows past token 262,144 sit
    at byte offsets no 32-bit offset reaches.  Dense checks on the last
    document (entirely past that token) and on the longest one."""
    rng = np.random.default_rng(7)
    w = I.text_packs(rng, 1, cap=327680)[0]
    T = w.total_tokens
    assert T * w.n_heads * w.head_dim * 2 > 2 ** 31
    cu = w.cu_seqlens
    last = len(w.lengths) - 1
    assert int(cu[last]) * w.n_heads * w.head_dim * 2 >= 2 ** 31, "the last document should start beyond 2^31 bytes"
    bits, out = _run(torch, w, rng)
    srng = np.random.default_rng(107)
    q, k, v, do = _check_rows(bits, out, w, srng, 256, "text > 2 GiB")
    longest = int(np.argmax(np.diff(cu)))
    _check_dense(q, k, v, do, out, w, srng, [(last, int(srng.integers(w.n_heads))),
                                            (longest, int(srng.integers(w.n_heads)))], "text > 2 GiB")
    _check_identities(q, v, do, out, w, "text > 2 GiB")


def test_transformer_1d_causal_pack(torch):
    """The Transformer-1D layer's attention shape (Sec. 4.1: hidden 3072 as
    48 heads of width 64, causal) over log-normal documents (median 128,
    sigma 1.5, 8 to 18,705 tokens) packed to 64k tokens: long sequences,
    short ones and 16 causal packed windows in one call."""
    import paper_2608_07524_amd as P
    rng = np.random.default_rng(3)
    pool = I.text_lengths(rng, 4096, median=128, sigma=1.5, lo=8).tolist()
    lengths = I.greedy_pack(pool, 65536)[0]
    w = I.Workload("Transformer-1D causal pack H48 D64", lengths, 48, 64, True, 1.0 / 8.0)
    units, n_tiles, _ = P.work_list(w.cu_seqlens, 48, 64, True, 1)
    assert len(units) > n_tiles, "the pack should hold packed windows"
    bits, out = _run(torch, w, rng)
    srng = np.random.default_rng(106)
    q, k, v, do = _check_rows(bits, out, w, srng, 256, "T-1D causal")
    _check_keys(q, k, v, do, out, w, srng, 4096, 3, "T-1D causal")
    _check_identities(q, v, do, out, w, "T-1D causal")


def _check_single_tokens(bits, out, w, label):
    """A one-token sequence attends to itself only: P = 1, so O = V and
    dV = dO exactly, and dS = dP - Delta = 0, so dK (and dQ) vanish in exact
    arithmetic; the GPU's dK there is fp32 rounding of dP - Delta, checked to
    be negligible next to the tensor's gradients."""
    cu = w.cu_seqlens
    rows = np.array([int(cu[b]) for b in range(len(cu) - 1) if cu[b + 1] - cu[b] == 1], dtype=np.int64)
    if rows.size == 0:
        return
    assert np.array_equal(out["o"][rows], bits[2][rows]), "O != V on one-token sequences"
    assert np.array_equal(out["dv"][rows], bits[3][rows]), "dV != dO on one-token sequences"
    dk_all = np.abs(I.bf16_to_f64(out["dk"]))
    ratio = float(dk_all[rows].max() / dk_all.max())
    print(f"{label}: {rows.size} one-token sequences: O = V, dV = dO bitwise; max|dK| / tensor max {ratio:.1e}",
          flush=True)
    assert ratio <= 1e-3


@pytest.mark.parametrize("axis", ["spatial", "temporal"])
def test_video_2d_packs(torch, axis):
    """Transformer-2D packs: frames of up to 3,600 tokens (spatial) or
    thousands of sequences of 1..51 tokens (temporal), H16, D72."""
    rng = np.random.default_rng(0)
    w = I.video_2d_pack(rng, axis)
    bits, out = _run(torch, w, rng)
    srng = np.random.default_rng(105)
    q, k, v, do = _check_rows(bits, out, w, srng, 1024, f"2-D {axis}")
    _check_keys(q, k, v, do, out, w, srng, 4096, 4, f"2-D {axis}")
    _check_identities(q, v, do, out, w, f"2-D {axis}")
    _check_single_tokens(bits, out, w, f"2-D {axis}")
