"""Pins of the oracle's number formats, gate, top-k, softmax and weights
(Algorithm 1, score / argmax_k / normalize) against brute force, closed forms
and library routines."""
import itertools
from fractions import Fraction

import numpy as np
import pytest
import scipy.special
import torch

import oracle as O


# -- number formats ----------------------------------------------------------
def test_round_bf16_matches_torch_rne():
    rng = np.random.default_rng(1)
    v = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(2000) * 1e-30).astype(np.float32),
        (rng.standard_normal(2000) * 1e30).astype(np.float32),
        # exact halfway cases: 1 + 2^-8 (-> 1), 1 + 3*2^-8 (-> 1 + 2^-6)
        np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 0.0, -0.0], np.float32),
    ])
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.round_bf16(v.astype(np.float64))
    np.testing.assert_array_equal(got, ref)
    assert O.round_bf16(np.array([1 + 2 ** -8]))[0] == 1.0
    assert O.round_bf16(np.array([1 + 3 * 2 ** -8]))[0] == 1 + 2 ** -6


def test_bf16_bits_decode_matches_torch():
    bits = np.arange(0, 1 << 16, 7, dtype=np.uint16)
    bits = bits[(bits & 0x7F80) != 0x7F80]           # drop inf/nan patterns
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(O.bf16_to_f64(bits), ref)


@pytest.mark.parametrize("act,fn", [
    ("relu", torch.relu),
    ("gelu_tanh", lambda t: torch.nn.functional.gelu(t, approximate="tanh")),
    ("silu", torch.nn.functional.silu),
])
def test_activations_and_grads_match_torch(act, fn):
    h = np.linspace(-6, 6, 2001)
    h = h[np.abs(h) > 1e-9]                          # away from relu's kink
    th = torch.tensor(h, dtype=torch.float64, requires_grad=True)
    y = fn(th)
    y.sum().backward()
    np.testing.assert_allclose(O.act_fwd(h, act), y.detach().numpy(), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(O.act_grad(h, act), th.grad.numpy(), rtol=1e-12, atol=1e-14)
    if act == "relu":
        assert O.act_grad(np.array([0.0]), "relu")[0] == 0.0


# -- gate logits ---------------------------------------------------------------
def test_gate_logits_exact_on_integer_inputs():
    """Integer-valued x and w_g: every partial sum is exact, so the logits
    equal the integer dot products computed with Python ints."""
    rng = np.random.default_rng(2)
    x = rng.integers(-3, 4, size=(17, 40))
    w = rng.integers(-3, 4, size=(5, 40))
    b = rng.integers(-2, 3, size=5)
    got = O.gate_logits(x.astype(np.float64), w.astype(np.float64), b.astype(np.float32))
    for t in range(17):
        for e in range(5):
            exact = sum(int(x[t, i]) * int(w[e, i]) for i in range(40)) + int(b[e])
            assert got[t, e] == np.float32(exact)


def test_gate_logits_one_hot_rows_select_gate_columns():
    w = np.random.default_rng(3).standard_normal((6, 9))
    b = np.arange(6, dtype=np.float32)
    x = np.eye(9)
    np.testing.assert_array_equal(O.gate_logits(x, w, b), (w.T + b).astype(np.float32))


# -- top-k ---------------------------------------------------------------------
def _brute_topk(l, k):
    """The k experts S such that every e in S beats every e' outside S,
    where 'beats' = larger logit, or equal logit and lower index; listed in
    that order."""
    E = len(l)
    beats = lambda a, b: l[a] > l[b] or (l[a] == l[b] and a < b)
    for S in itertools.permutations(range(E), k):
        if all(beats(S[i], S[i + 1]) for i in range(k - 1)) and \
           all(beats(s, o) for s in S for o in range(E) if o not in S):
            return list(S)
    raise AssertionError("no top-k set")


@pytest.mark.parametrize("E", [1, 2, 3, 4, 5])
def test_topk_exhaustive_ties(E):
    vals = [-1.0, 0.0, 1.0]
    grid = np.array(list(itertools.product(vals, repeat=E)), dtype=np.float32)
    for k in range(1, min(E, 3) + 1):
        got = O.topk(grid, k)
        lib = np.argsort(-grid.astype(np.float64), axis=1, kind="stable")[:, :k]
        np.testing.assert_array_equal(got, lib)
        for row, g in zip(grid, got):
            assert list(g) == _brute_topk(list(row), k)


def test_topk_random_vs_brute_and_signed_zero_and_inf():
    rng = np.random.default_rng(4)
    l = rng.integers(-2, 3, size=(300, 6)).astype(np.float32)
    l[0] = [-0.0, 0.0, -0.0, 0.0, -1, -1]            # +0 == -0: lower index wins
    l[1] = [-np.inf] * 6
    got = O.topk(l, 3)
    for row, g in zip(l, got):
        assert list(g) == _brute_topk(list(row), 3)
    assert list(got[0]) == [0, 1, 2]
    assert list(got[1]) == [0, 1, 2]
    with pytest.raises(ValueError):
        O.topk(np.array([[np.nan, 1.0]], np.float32), 1)


# -- softmax and weights -------------------------------------------------------
def test_softmax_closed_forms():
    rng = np.random.default_rng(5)
    l = (rng.standard_normal((64, 7)) * 4).astype(np.float32)
    p = O.softmax(l)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-15)
    np.testing.assert_allclose(p, scipy.special.softmax(l.astype(np.float64), axis=1),
                               rtol=1e-13)
    np.testing.assert_allclose(O.softmax(l.astype(np.float64) + 100.0), p, rtol=1e-12)   # shift invariance
    assert O.softmax(np.array([[3.5]], np.float32))[0, 0] == 1.0      # E = 1
    two = O.softmax(np.array([[0.0, np.log(3.0)]]))                   # 1:3 odds
    np.testing.assert_allclose(two[0], [0.25, 0.75], rtol=1e-15)


def test_gate_weights_raw_renorm_and_soft_mixture():
    rng = np.random.default_rng(6)
    l = rng.standard_normal((50, 8)).astype(np.float32)
    p = O.softmax(l)
    ids = O.topk(l, 1)
    w1 = O.gate_weights(p, ids, renorm=0)
    np.testing.assert_array_equal(w1[:, 0], p.max(axis=1).astype(np.float32))
    ids3 = O.topk(l, 3)
    w3 = O.gate_weights(p, ids3, renorm=1)
    np.testing.assert_allclose(w3.sum(axis=1), 1.0, rtol=0, atol=3e-7)
    sel = np.take_along_axis(p, ids3.astype(np.int64), 1)
    for t in range(5):
        S = sum(Fraction(float(s)) for s in sel[t])
        for j in range(3):
            assert abs(float(Fraction(float(sel[t, j])) / S) - float(w3[t, j])) <= 6e-8
    idsE = O.topk(l, 8)                    # k = E with renorm: weights = p
    wE = O.gate_weights(p, idsE, renorm=1)
    np.testing.assert_allclose(np.take_along_axis(p, idsE.astype(np.int64), 1), wE,
                               rtol=2e-7)


@pytest.mark.parametrize("renorm", [0, 1])
def test_invalid_cached_id_is_no_pick(renorm):
    """An id outside [0, E) in cached picks is not a pick (weight 0, out of the
    normalisation): each row's weights and gate gradients equal those of the
    same row with that column removed, computed with k - 1 picks."""
    rng = np.random.default_rng(17)
    T, E, k, d = 40, 6, 3, 5
    logits = rng.standard_normal((T, E)) * 2
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    bad_j = rng.integers(0, k, T)
    bad = ids.copy()
    bad[np.arange(T), bad_j] = np.where(np.arange(T) % 2 == 0, E + 3, -1)
    dw = rng.standard_normal((T, k))
    dw[np.arange(T), bad_j] = 0.0                  # a dropped assignment's dweight
    x = rng.standard_normal((T, d))
    p = O.softmax(logits)
    w_bad = O.gate_weights(p, bad, renorm)
    dl_bad, _ = O.gate_bwd(logits, bad, dw, renorm, x)
    for t in range(T):
        keep = [j for j in range(k) if j != bad_j[t]]
        w_ref = O.gate_weights(p[t:t + 1], ids[t:t + 1, keep], renorm)
        np.testing.assert_array_equal(w_bad[t, keep], w_ref[0])
        assert w_bad[t, bad_j[t]] == 0.0
        dl_ref, _ = O.gate_bwd(logits[t:t + 1], ids[t:t + 1, keep], dw[t:t + 1, keep], renorm,
                               x[t:t + 1])
        np.testing.assert_allclose(dl_bad[t], dl_ref[0], rtol=0, atol=1e-15)
    # the k - 1 computation is itself the full backward: rows sum to 0
    np.testing.assert_allclose(dl_bad.sum(axis=1), 0.0, atol=1e-6)
