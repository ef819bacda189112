"""Pins for the float64 attention oracle, on the CPU.

The oracle must be trusted before anything is compared with it, so each
test checks it against something other than itself: scalar brute force,
finite differences, closed forms, structural invariants of softmax
attention, and an independent library routine.
"""

import math

import numpy as np
import pytest

from oracle import attention as A


def _rand(rng, T, H, D):
    return rng.standard_normal((T, H, D))


def _brute_forward(q, k, v, cu, scale, causal):
    """Scalar loops with math.exp; no numpy arithmetic."""
    T, H, D = q.shape
    o = [[[0.0] * D for _ in range(H)] for _ in range(T)]
    lse = [[float("nan")] * T for _ in range(H)]
    for b in range(len(cu) - 1):
        s0, s1 = cu[b], cu[b + 1]
        for h in range(H):
            for i in range(s0, s1):
                keys = [j for j in range(s0, s1) if not (causal and j > i)]
                sc = []
                for j in keys:
                    acc = 0.0
                    for d in range(D):
                        acc += float(q[i, h, d]) * float(k[j, h, d])
                    sc.append(scale * acc)
                m = max(sc)
                z = sum(math.exp(x - m) for x in sc)
                l = m + math.log(z)
                lse[h][i] = l
                for d in range(D):
                    o[i][h][d] = sum(math.exp(s - l) * float(v[j, h, d]) for s, j in zip(sc, keys))
    return np.array(o), np.array(lse)


@pytest.mark.parametrize("causal", [False, True])
def test_forward_matches_scalar_brute_force(causal):
    rng = np.random.default_rng(11)
    cu = [0, 1, 6, 6, 19, 32]  # includes an empty sequence and a length-1 one
    q, k, v = (_rand(rng, 32, 2, 8) for _ in range(3))
    o, lse = A.attention_forward(q, k, v, cu, 0.37, causal)
    ob, lseb = _brute_forward(q, k, v, cu, 0.37, causal)
    assert np.max(np.abs(o - ob)) < 1e-12
    assert np.nanmax(np.abs(lse - lseb)) < 1e-12


def test_forward_row_blocking_is_exact():
    rng = np.random.default_rng(3)
    cu = [0, 70, 71, 200]
    q, k, v = (_rand(rng, 200, 3, 5) for _ in range(3))
    for causal in (False, True):
        o1, l1 = A.attention_forward(q, k, v, cu, 0.5, causal, row_block=7)
        o2, l2 = A.attention_forward(q, k, v, cu, 0.5, causal, row_block=4096)
        assert np.max(np.abs(o1 - o2)) < 1e-13
        assert np.max(np.abs(l1 - l2)) < 1e-13
        g1 = A.attention_backward(q, q, k, v, cu, 0.5, causal, row_block=9)
        g2 = A.attention_backward(q, q, k, v, cu, 0.5, causal, row_block=4096)
        for a, b in zip(g1, g2):
            assert np.max(np.abs(a - b)) < 1e-12


@pytest.mark.parametrize("causal", [False, True])
def test_backward_matches_finite_differences(causal):
    rng = np.random.default_rng(5)
    cu = [0, 3, 4, 11, 24]
    T, H, D = 24, 2, 4
    q, k, v, do = (_rand(rng, T, H, D) for _ in range(4))
    scale = 0.8
    dq, dk, dv = A.attention_backward(do, q, k, v, cu, scale, causal)

    def loss(qq, kk, vv):
        o, _ = A.attention_forward(qq, kk, vv, cu, scale, causal)
        return float(np.sum(o * do))

    eps = 1e-6
    for which, grad in ((0, dq), (1, dk), (2, dv)):
        for idx in np.ndindex(T, H, D):
            args = [q.copy(), k.copy(), v.copy()]
            args[which][idx] += eps
            up = loss(*args)
            args[which][idx] -= 2 * eps
            dn = loss(*args)
            fd = (up - dn) / (2 * eps)
            assert abs(fd - grad[idx]) <= 1e-7 + 1e-5 * abs(grad[idx]), (which, idx, fd, grad[idx])


def test_rows_of_p_sum_to_one_and_packing_is_per_sequence():
    rng = np.random.default_rng(8)
    lens = [5, 17, 1, 9]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T, H, D = int(cu[-1]), 2, 6
    q, k, do = (_rand(rng, T, H, D) for _ in range(3))
    # P rows sum to one <=> attending over all-ones values returns ones
    for causal in (False, True):
        o, _ = A.attention_forward(q, k, np.ones((T, H, D)), cu, 0.3, causal)
        assert np.max(np.abs(o - 1.0)) < 1e-12
    v = _rand(rng, T, H, D)
    for causal in (False, True):
        o, lse = A.attention_forward(q, k, v, cu, 0.3, causal)
        grads = A.attention_backward(do, q, k, v, cu, 0.3, causal)
        for b in range(len(lens)):
            s0, s1 = cu[b], cu[b + 1]
            sl = slice(s0, s1)
            ob, lb = A.attention_forward(q[sl], k[sl], v[sl], [0, s1 - s0], 0.3, causal)
            assert np.array_equal(ob, o[sl]) and np.array_equal(lb, lse[:, sl])
            gb = A.attention_backward(do[sl], q[sl], k[sl], v[sl], [0, s1 - s0], 0.3, causal)
            for full, part in zip(grads, gb):
                assert np.array_equal(full[sl], part)


def test_permuting_sequences_permutes_outputs():
    rng = np.random.default_rng(9)
    lens = [4, 11, 7]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T, H, D = int(cu[-1]), 1, 3
    q, k, v, do = (_rand(rng, T, H, D) for _ in range(4))
    perm = [2, 0, 1]
    idx = np.concatenate([np.arange(cu[p], cu[p + 1]) for p in perm])
    cu2 = np.concatenate([[0], np.cumsum([lens[p] for p in perm])])
    o, lse = A.attention_forward(q, k, v, cu, 1.1, True)
    o2, lse2 = A.attention_forward(q[idx], k[idx], v[idx], cu2, 1.1, True)
    assert np.max(np.abs(o[idx] - o2)) < 1e-14
    assert np.max(np.abs(lse[:, idx] - lse2)) < 1e-14
    g = A.attention_backward(do, q, k, v, cu, 1.1, True)
    g2 = A.attention_backward(do[idx], q[idx], k[idx], v[idx], cu2, 1.1, True)
    for a, b in zip(g, g2):
        assert np.max(np.abs(a[idx] - b)) < 1e-13


@pytest.mark.parametrize("causal", [False, True])
def test_gradient_sum_invariants(causal):
    """Per (sequence, head): sum_j dV_j = sum_i dO_i (rows of P sum to one)
    and sum_j dK_j = 0 (softmax is invariant to shifting a row's scores)."""
    rng = np.random.default_rng(12)
    lens = [1, 6, 30]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T, H, D = int(cu[-1]), 3, 5
    q, k, v, do = (_rand(rng, T, H, D) for _ in range(4))
    dq, dk, dv = A.attention_backward(do, q, k, v, cu, 0.6, causal)
    for b in range(len(lens)):
        sl = slice(cu[b], cu[b + 1])
        assert np.max(np.abs(dv[sl].sum(0) - do[sl].sum(0))) < 1e-12
        assert np.max(np.abs(dk[sl].sum(0))) < 1e-12


def test_closed_forms():
    rng = np.random.default_rng(13)
    H, D = 2, 4
    # a sequence of length one attends to itself only
    q, k, v, do = (_rand(rng, 1, H, D) for _ in range(4))
    o, lse = A.attention_forward(q, k, v, [0, 1], 0.25, False)
    assert np.array_equal(o, v)
    assert np.max(np.abs(lse[:, 0] - 0.25 * np.sum(q[0] * k[0], axis=1))) < 1e-15
    dq, dk, dv = A.attention_backward(do, q, k, v, [0, 1], 0.25, False)
    assert np.all(dq == 0) and np.all(dk == 0) and np.array_equal(dv, do)
    # zero queries: uniform attention over the visible keys
    T = 9
    k, v = _rand(rng, T, H, D), _rand(rng, T, H, D)
    z = np.zeros((T, H, D))
    o, lse = A.attention_forward(z, k, v, [0, T], 0.7, False)
    assert np.max(np.abs(o - v.mean(axis=0, keepdims=True))) < 1e-14
    assert np.max(np.abs(lse - math.log(T))) < 1e-14
    o, lse = A.attention_forward(z, k, v, [0, T], 0.7, True)
    for i in range(T):
        assert np.max(np.abs(o[i] - v[: i + 1].mean(axis=0))) < 1e-14
        assert np.max(np.abs(lse[:, i] - math.log(i + 1))) < 1e-14
    # causal first row sees only its own key
    q = _rand(rng, T, H, D)
    o, _ = A.attention_forward(q, k, v, [0, T], 0.7, True)
    assert np.array_equal(o[0], v[0])


@pytest.mark.parametrize("causal", [False, True])
def test_matches_torch_sdpa_and_autograd(causal):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(21)
    lens = [13, 1, 40]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T, H, D = int(cu[-1]), 2, 8
    q, k, v, do = (_rand(rng, T, H, D) for _ in range(4))
    scale = 0.41
    o, lse = A.attention_forward(q, k, v, cu, scale, causal)
    dq, dk, dv = A.attention_backward(do, q, k, v, cu, scale, causal)
    for b in range(len(lens)):
        sl = slice(cu[b], cu[b + 1])
        tq, tk, tv = (torch.tensor(x[sl].transpose(1, 0, 2), dtype=torch.float64, requires_grad=True)
                      for x in (q, k, v))
        to = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=causal, scale=scale)
        to.backward(torch.tensor(do[sl].transpose(1, 0, 2), dtype=torch.float64))
        assert np.max(np.abs(to.detach().numpy().transpose(1, 0, 2) - o[sl])) < 1e-12
        for mine, t in ((dq, tq), (dk, tk), (dv, tv)):
            assert np.max(np.abs(t.grad.numpy().transpose(1, 0, 2) - mine[sl])) < 1e-12
        ref_lse = torch.logsumexp(scale * tq.detach() @ tk.detach().transpose(1, 2)
                                  + (torch.triu(torch.full((lens[b], lens[b]), -math.inf,
                                                           dtype=torch.float64), 1) if causal else 0),
                                  dim=-1)
        assert np.max(np.abs(ref_lse.numpy() - lse[:, sl])) < 1e-12


def test_sampled_rows_match_full_outputs():
    rng = np.random.default_rng(31)
    lens = [50, 3, 77]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T, H, D = int(cu[-1]), 2, 6
    q, k, v, do = (_rand(rng, T, H, D) for _ in range(4))
    for causal in (False, True):
        o, lse = A.attention_forward(q, k, v, cu, 0.5, causal)
        dq, dk, dv = A.attention_backward(do, q, k, v, cu, 0.5, causal)
        rows = np.array([0, 49, 50, 52, 53, 100, 129])
        heads = np.array([1, 0, 1, 0, 1, 0, 1])
        o_r, l_r = A.attention_rows(q, k, v, cu, 0.5, causal, rows, heads)
        assert np.max(np.abs(o_r - o[rows, heads])) < 1e-13
        assert np.max(np.abs(l_r - lse[heads, rows])) < 1e-13
        dq_r = A.attention_dq_rows(do, q, k, v, cu, 0.5, causal, rows, heads)
        assert np.max(np.abs(dq_r - dq[rows, heads])) < 1e-12
        dk_r, dv_r = A.attention_dkdv_rows(do, q, k, v, cu, 0.5, causal, rows, heads, row_block=16)
        assert np.max(np.abs(dk_r - dk[rows, heads])) < 1e-12
        assert np.max(np.abs(dv_r - dv[rows, heads])) < 1e-12


def test_grouped_rows_and_given_normalisers():
    """Rows of one (sequence, head) evaluated in blocks give the full
    outputs; key columns from the supplied LSE and Delta = rowsum(dO o O)
    equal the full backward, and shifting every LSE by e (Delta kept)
    scales P, hence dV and dS and dK, by exp(-e)."""
    rng = np.random.default_rng(32)
    lens = [40, 1, 70, 0, 33]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T, H, D = int(cu[-1]), 3, 5
    q, k, v, do = (_rand(rng, T, H, D) for _ in range(4))
    for causal in (False, True):
        o, lse = A.attention_forward(q, k, v, cu, 0.4, causal)
        dq, dk, dv = A.attention_backward(do, q, k, v, cu, 0.4, causal)
        rows = rng.integers(0, T, 60)
        heads = rng.integers(0, H, 60)
        o_r, l_r = A.attention_rows(q, k, v, cu, 0.4, causal, rows, heads, row_block=3)
        assert np.max(np.abs(o_r - o[rows, heads])) < 1e-13 and np.max(np.abs(l_r - lse[heads, rows])) < 1e-13
        dq_r = A.attention_dq_rows(do, q, k, v, cu, 0.4, causal, rows, heads, row_block=5)
        assert np.max(np.abs(dq_r - dq[rows, heads])) < 1e-12
        delta = np.einsum("thd,thd->ht", do, o)
        dk_c, dv_c = A.attention_dkdv_cols_given(do, q, k, v, cu, 0.4, causal, rows, heads, lse, delta, row_block=7)
        assert np.max(np.abs(dk_c - dk[rows, heads])) < 1e-12
        assert np.max(np.abs(dv_c - dv[rows, heads])) < 1e-12
        e = 0.01
        dk_s, dv_s = A.attention_dkdv_cols_given(do, q, k, v, cu, 0.4, causal, rows, heads, lse + e, delta,
                                                 row_block=7)
        assert np.max(np.abs(dv_s - np.exp(-e) * dv[rows, heads])) < 1e-12
        assert np.max(np.abs(dk_s - np.exp(-e) * dk[rows, heads])) < 1e-12


def test_valid_pairs():
    assert A.valid_pairs([0, 37, 101, 229, 429]) == 37 ** 2 + 64 ** 2 + 128 ** 2 + 200 ** 2
    assert A.valid_pairs([0, 3, 3, 5], causal=True) == 6 + 0 + 3
