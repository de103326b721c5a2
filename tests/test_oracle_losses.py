"""Pins of the oracle's balance term (Eq. 3), specification loss (Eq. 2) and
AggregateSpec against closed forms, special cases that reduce to other
definitions, inequalities and finite differences."""
import numpy as np
import pytest

import oracle as O


# -- Eq. 3 balance term ----------------------------------------------------------
def test_balance_uniform_routing_is_lambda():
    # T_i = G_i = 1/n for every expert: B = lam * n * n * (1/n)^2 = lam
    T, E, k, lam = 24, 4, 2, 0.01
    logits = np.zeros((T, E))
    counts = np.full(E, T * k // E)
    B, c = O.balance_term(logits, counts, k, lam)
    assert B == pytest.approx(lam, rel=1e-15)
    np.testing.assert_allclose(c, np.float32(lam * E * (1 / E) / T), rtol=0)


def test_balance_collapse_to_one_expert_is_lambda_n():
    # every token on expert 0 with all of the probability: T_0 = G_0 = 1
    T, E, lam = 16, 8, 0.5
    logits = np.zeros((T, E))
    logits[:, 0] = 60.0
    counts = np.zeros(E, dtype=np.int64)
    counts[0] = T
    B, c = O.balance_term(logits, counts, 1, lam)
    assert B == pytest.approx(lam * E, rel=1e-12)
    assert c[0] == np.float32(lam * E / T) and (c[1:] == 0).all()


@pytest.mark.parametrize("counts,expect", [([2, 0], 0.75), ([0, 2], 1.25), ([1, 1], 1.0)])
def test_balance_hand_worked(counts, expect):
    # p = [[1/4, 3/4], [1/2, 1/2]]: G = [3/8, 5/8]; n = 2, k = 1, T = 2
    logits = np.array([[0.0, np.log(3.0)], [0.0, 0.0]])
    B, _ = O.balance_term(logits, np.array(counts), 1, 1.0)
    assert B == pytest.approx(expect, rel=1e-14)


def test_balance_expert_permutation_invariant():
    rng = np.random.default_rng(3)
    T, E, k = 50, 6, 2
    logits = rng.standard_normal((T, E)).astype(np.float32).astype(np.float64)
    counts = rng.integers(0, 30, E)
    perm = rng.permutation(E)
    B1, c1 = O.balance_term(logits, counts, k, 0.1)
    B2, c2 = O.balance_term(logits[:, perm], counts[perm], k, 0.1)
    assert B1 == pytest.approx(B2, rel=1e-14)
    np.testing.assert_array_equal(c1[perm], c2)


def test_balance_gradient_through_gate_bwd_matches_finite_differences():
    # dB/dl through the softmax, with the assignment counts held fixed
    rng = np.random.default_rng(4)
    T, E, k, lam, d = 5, 4, 2, 0.7, 3
    logits = rng.standard_normal((T, E))
    ids = O.topk(logits, k)
    counts = O.count_assignments(ids, E)
    _, c = O.balance_term(logits, counts, k, lam)
    x = rng.standard_normal((T, d))
    dl, dwg = O.gate_bwd(logits, ids, np.zeros((T, k)), 1, x, dprob_coef=c)
    h = 1e-6
    fd = np.zeros((T, E))
    for t in range(T):
        for e in range(E):
            lp, lm = logits.copy(), logits.copy()
            lp[t, e] += h
            lm[t, e] -= h
            fd[t, e] = (O.balance_term(lp, counts, k, lam)[0] -
                        O.balance_term(lm, counts, k, lam)[0]) / (2 * h)
    np.testing.assert_allclose(dl, fd, rtol=2e-5, atol=1e-9)
    np.testing.assert_allclose(dwg, (fd.T @ x), rtol=1e-4, atol=1e-8)


def test_gate_bwd_coefficient_adds_linearly():
    rng = np.random.default_rng(5)
    T, E, k, d = 30, 5, 2, 4
    logits = rng.standard_normal((T, E))
    ids = O.topk(logits, k)
    dw = rng.standard_normal((T, k))
    x = rng.standard_normal((T, d))
    c = rng.standard_normal(E) * 1e-2
    dl0, _ = O.gate_bwd(logits, ids, dw, 1, x)
    dlc, _ = O.gate_bwd(logits, ids, np.zeros((T, k)), 1, x, dprob_coef=c)
    dl, _ = O.gate_bwd(logits, ids, dw, 1, x, dprob_coef=c)
    np.testing.assert_allclose(dl, dl0 + dlc, rtol=1e-6, atol=1e-9)
    # a coefficient equal for every expert is absorbed by the softmax
    dl1, _ = O.gate_bwd(logits, ids, dw, 1, x, dprob_coef=np.full(E, 3.0))
    np.testing.assert_allclose(dl1, dl0, rtol=1e-6, atol=1e-7)


# -- AggregateSpec and Eq. 2 specification loss ------------------------------------
def _routing(rng, T, E, k, cap_div=None):
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    counts = O.count_assignments(ids, E)
    cap = counts if cap_div is None else counts // cap_div
    off = O.exclusive_offsets(cap)
    s = O.assign_slots(ids, E, cap, off, int(off[-1]))
    return ids, s["dest_row"], int(off[-1])


def test_aggregate_spec_rows_and_weighted_sum_is_combine():
    rng = np.random.default_rng(6)
    T, E, k, d = 40, 5, 3, 7
    ids, dest, R = _routing(rng, T, E, k, cap_div=2)
    assert (dest < 0).any()
    Y = rng.standard_normal((R, d))
    w = rng.random((T, k))
    A = O.aggregate_spec(Y, dest)
    assert A.shape == (T * k, d)
    for t in range(T):
        for j in range(k):
            r = dest[t, j]
            np.testing.assert_array_equal(A[t * k + j], Y[r] if r >= 0 else 0.0)
    mix = (w[:, :, None] * A.reshape(T, k, d)).sum(axis=1)
    np.testing.assert_allclose(mix, O.combine(Y, dest, w, "f32"), rtol=1e-14, atol=1e-15)


def test_spec_loss_single_expert_is_cooperation_loss():
    # k = 1 and weight 1: Eq. 2 and Eq. 1 are the same loss
    rng = np.random.default_rng(7)
    T, E, d = 60, 4, 9
    ids, dest, R = _routing(rng, T, E, 1)
    Y = rng.standard_normal((R, d))
    tgt = rng.standard_normal((T, d))
    w = np.ones((T, 1))
    loss, _, _ = O.spec_loss(Y, dest, w, tgt, "f32")
    y = O.combine(Y, dest, w, "f32")
    assert loss == pytest.approx(np.mean((y - tgt) ** 2), rel=1e-13)


def test_spec_loss_bounds_cooperation_loss_from_above():
    # convex task loss and weights summing to 1: sum_i g_i L(O_i) >= L(sum_i g_i O_i)
    rng = np.random.default_rng(8)
    T, E, k, d = 80, 6, 3, 5
    ids, dest, R = _routing(rng, T, E, k)
    Y = rng.standard_normal((R, d))
    tgt = rng.standard_normal((T, d))
    w = rng.random((T, k))
    w /= w.sum(axis=1, keepdims=True)
    loss, _, _ = O.spec_loss(Y, dest, w, tgt, "f32")
    coop = np.mean((O.combine(Y, dest, w, "f32") - tgt) ** 2)
    assert loss >= coop
    # equal predictions of the k experts: both losses coincide
    Yeq = np.repeat(rng.standard_normal((T, d)), k, axis=0)
    dest_eq = np.arange(T * k).reshape(T, k)
    l2, _, _ = O.spec_loss(Yeq, dest_eq, w, tgt, "f32")
    c2 = np.mean((O.combine(Yeq, dest_eq, w, "f32") - tgt) ** 2)
    assert l2 == pytest.approx(c2, rel=1e-12)


def test_spec_loss_gradients_match_finite_differences():
    rng = np.random.default_rng(9)
    T, E, k, d = 6, 4, 2, 3
    ids, dest, R = _routing(rng, T, E, k, cap_div=2)
    Y = rng.standard_normal((R, d))
    tgt = rng.standard_normal((T, d))
    w = rng.random((T, k))
    _, dw, dY = O.spec_loss(Y, dest, w, tgt, "f32")
    h = 1e-6
    kept_rows = np.unique(dest[dest >= 0])
    for r in kept_rows:
        for c in range(d):
            Yp, Ym = Y.copy(), Y.copy()
            Yp[r, c] += h
            Ym[r, c] -= h
            fd = (O.spec_loss(Yp, dest, w, tgt, "f32")[0] - O.spec_loss(Ym, dest, w, tgt, "f32")[0]) / (2 * h)
            assert dY[r, c] == pytest.approx(fd, rel=1e-6, abs=1e-10)
    for t in range(T):
        for j in range(k):
            wp, wm = w.copy(), w.copy()
            wp[t, j] += h
            wm[t, j] -= h
            fd = (O.spec_loss(Y, dest, wp, tgt, "f32")[0] - O.spec_loss(Y, dest, wm, tgt, "f32")[0]) / (2 * h)
            assert dw[t, j] == pytest.approx(fd, rel=1e-6, abs=1e-10)
            if dest[t, j] < 0:
                assert dw[t, j] == 0.0
