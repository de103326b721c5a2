"""Pins of the oracle's capacity rule (Eq. 4, dynamic capacity factors) and
slot assignment / drop rule (Section 4.1) against exact rationals, the
quadratic brute-force definition and invariants."""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
import workloads as W


# -- capacity -----------------------------------------------------------------
@pytest.mark.parametrize("name,expect", [("c1", 80), ("c2", 1024), ("c3", 512)])
def test_static_capacity_worked_values(name, expect):
    """ceil(alpha * T * k / E) for the static runs of the named workloads."""
    wl = W.config(name)
    kind, num, den = wl.capacity[0]
    assert kind == "static"
    cap = O.capacity_static(wl.T, wl.k, wl.E, num, den)
    assert (cap == expect).all()
    assert expect == math.ceil(Fraction(num, den) * wl.T * wl.k / wl.E)


def test_static_capacity_half_and_clamps():
    assert O.capacity_static(256, 1, 4, 1, 2)[0] == 32
    assert O.capacity_static(10, 2, 1, 7, 1)[0] == 10          # clamp to T
    assert O.capacity_static(10, 1, 8, 1, 100, cap_min=3)[0] == 3


def test_dynamic_capacity_exact_rational():
    counts = np.arange(0, 200001)
    for num, den in [(11, 10), (21, 20), (1, 1), (5, 4)]:
        got = O.capacity_dynamic(counts, T=10 ** 9, num=num, den=den)
        ref = np.array([math.ceil(Fraction(num * int(c), den)) for c in counts[::997]])
        np.testing.assert_array_equal(got[::997], ref)
        # spot the cases a float64 ceil gets wrong (e.g. 1.1 * 50 -> 56)
        for c in (50, 90, 100, 1000):
            assert got[c] == math.ceil(Fraction(num * c, den))
    assert math.ceil(1.1 * 50) == 56 and O.capacity_dynamic([50], 10 ** 6, 11, 10)[0] == 55
    np.testing.assert_array_equal(O.capacity_dynamic([0, 5, 9], T=6, num=11, den=10, cap_min=2),
                                  [2, 6, 6])


def test_offsets():
    np.testing.assert_array_equal(O.exclusive_offsets([3, 0, 5]), [0, 3, 3, 8])
    # aligned layout, worked by hand: regions rounded up to multiples of align
    np.testing.assert_array_equal(O.exclusive_offsets([3, 0, 5], 4), [0, 4, 4, 12])
    np.testing.assert_array_equal(O.exclusive_offsets([300, 0, 256, 1], 256),
                                  [0, 512, 512, 768, 1024])


def test_aligned_layout_keeps_the_same_assignments():
    """Region alignment moves rows, never changes which assignments are kept:
    every region starts on a multiple of the alignment, regions do not
    overlap, the layout takes at most sum C + E (align - 1) rows, and counts,
    fill, the kept mask and each assignment's position inside its expert's
    region equal those of the packed layout."""
    rng = np.random.default_rng(31)
    for E, k, align in [(8, 2, 256), (64, 1, 256), (5, 3, 7), (16, 2, 1)]:
        T = 900
        ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
        counts = O.count_assignments(ids, E)
        cap = O.capacity_dynamic(counts * 9 // 10, T, 11, 10)        # lagged: some drops
        p_off = O.exclusive_offsets(cap)
        a_off = O.exclusive_offsets(cap, align)
        assert (a_off[:-1] % align == 0).all()
        assert (a_off[1:] - a_off[:-1] >= cap).all()
        assert a_off[-1] <= cap.sum() + E * (align - 1)
        ps = O.assign_slots(ids, E, cap, p_off, int(p_off[-1]))
        ak = O.assign_slots(ids, E, cap, a_off, int(a_off[-1]))
        for key in ("counts", "fill", "status"):
            np.testing.assert_array_equal(ps[key], ak[key])
        np.testing.assert_array_equal(ps["dest_row"] >= 0, ak["dest_row"] >= 0)
        kept = ps["dest_row"] >= 0
        np.testing.assert_array_equal((ps["dest_row"] - p_off[ids])[kept],
                                      (ak["dest_row"] - a_off[ids])[kept])


# -- slots ---------------------------------------------------------------------
def _brute_slots(ids, E, cap, off, rows_alloc):
    """pos(t,j) = number of live assignments to the same expert that come
    earlier in priority order (all j=0 in token order, then j=1, ...)."""
    T, k = ids.shape
    live, status = O.validate_assignments(ids, E)
    order = [(t, j) for j in range(k) for t in range(T)]
    dest = -np.ones((T, k), dtype=np.int64)
    for n, (t, j) in enumerate(order):
        if not live[t, j]:
            continue
        e = ids[t, j]
        pos = sum(1 for (t2, j2) in order[:n] if live[t2, j2] and ids[t2, j2] == e)
        room = max(0, min(cap[e], off[e + 1] - off[e], rows_alloc - off[e])) if off[e] >= 0 else 0
        if pos < room:
            dest[t, j] = off[e] + pos
    return dest


@pytest.mark.parametrize("seed", range(12))
def test_slots_match_quadratic_definition(seed):
    rng = np.random.default_rng(100 + seed)
    T = int(rng.integers(1, 9))
    E = int(rng.integers(1, 6))
    k = int(rng.integers(1, min(E, 3) + 1))
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    if seed % 3 == 0:                                      # cached-id faults
        ids[0, 0] = E + 2
        if k > 1:
            ids[-1, 1] = ids[-1, 0]
    cap = rng.integers(0, T + 1, size=E)
    off = O.exclusive_offsets(cap)
    rows_alloc = int(off[-1])
    if seed % 4 == 1:
        rows_alloc = max(0, rows_alloc - 2)                # region overflow
    s = O.assign_slots(ids, E, cap, off, rows_alloc)
    np.testing.assert_array_equal(s["dest_row"], _brute_slots(ids, E, cap, off, rows_alloc))


def _check_invariants(ids, E, cap, off, rows_alloc, s):
    T, k = ids.shape
    live, _ = O.validate_assignments(ids, E)
    dest, counts, fill = s["dest_row"], s["counts"], s["fill"]
    assert counts.sum() == live.sum()
    assert fill.sum() == (dest >= 0).sum()
    assert (fill <= np.maximum(cap, 0)).all()
    kept = dest[dest >= 0]
    assert len(np.unique(kept)) == len(kept)
    for e in range(E):
        rows = sorted(dest[(ids == e) & (dest >= 0)] - off[e])
        assert rows == list(range(fill[e]))                # first entries are used
    src = s["src"]
    for t in range(T):
        for j in range(k):
            if dest[t, j] >= 0:
                assert src[dest[t, j]] == t * k + j
    assert (src >= 0).sum() == len(kept)


def test_slot_invariants_and_monotonicity():
    rng = np.random.default_rng(7)
    T, E, k = 400, 6, 2
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    counts = O.count_assignments(ids, E)
    assert counts.sum() == T * k
    for cap in [np.zeros(E, np.int64), rng.integers(0, 200, E), counts, counts + 3,
                np.full(E, T)]:
        off = O.exclusive_offsets(cap)
        s = O.assign_slots(ids, E, cap, off, int(off[-1]))
        _check_invariants(ids, E, cap, off, int(off[-1]), s)
        np.testing.assert_array_equal(s["counts"], counts)
        if (cap >= counts).all():
            assert (s["dest_row"] >= 0).all()             # enough room: no drops
        # raising any capacity never un-keeps an assignment
        cap2 = cap + rng.integers(0, 5, E)
        off2 = O.exclusive_offsets(cap2)
        s2 = O.assign_slots(ids, E, cap2, off2, int(off2[-1]))
        assert ((s["dest_row"] >= 0) <= (s2["dest_row"] >= 0)).all()


def test_priority_first_choices_before_second():
    # expert 0 has capacity 2: token 2's first choice beats token 0's second
    ids = np.array([[1, 0], [0, 1], [0, 2]], dtype=np.int32)
    cap = np.array([2, 5, 5])
    s = O.assign_slots(ids, 3, cap, O.exclusive_offsets(cap), 12)
    np.testing.assert_array_equal(s["dest_row"], [[2, -1], [0, 3], [1, 7]])
    np.testing.assert_array_equal(s["fill"], [2, 2, 1])
    np.testing.assert_array_equal(s["counts"], [3, 2, 1])


def test_status_bits_and_all_to_one_expert():
    ids = np.array([[0, 0], [5, 1], [-1, 1]], dtype=np.int32)
    cap = np.array([4, 4])
    s = O.assign_slots(ids, 2, cap, O.exclusive_offsets(cap), 8)
    assert s["status"] == O.STATUS_BAD_ID | O.STATUS_DUP_ID
    np.testing.assert_array_equal(s["dest_row"], [[0, -1], [-1, 4], [-1, 5]])
    np.testing.assert_array_equal(s["counts"], [1, 2])
    s = O.assign_slots(np.array([[0], [0]], np.int32), 1, np.array([3]), np.array([0, 3]), 1)
    assert s["status"] == O.STATUS_REGION and list(s["dest_row"][:, 0]) == [0, -1]
    ids = np.zeros((50, 1), np.int32)                       # all tokens to one expert
    cap = np.array([20, 20, 20])
    s = O.assign_slots(ids, 3, cap, O.exclusive_offsets(cap), 60)
    assert list(s["fill"]) == [20, 0, 0] and (s["dest_row"][:20, 0] == np.arange(20)).all()
    assert (s["dest_row"][20:] == -1).all()


def test_dispatch_is_exact_copy():
    rng = np.random.default_rng(8)
    x = rng.standard_normal((30, 5))
    ids = np.stack([rng.permutation(4)[:2] for _ in range(30)]).astype(np.int32)
    cap = np.array([9, 20, 3, 40])
    off = O.exclusive_offsets(cap)
    s = O.assign_slots(ids, 4, cap, off, int(off[-1]))
    xd = O.dispatch_rows(x, s["dest_row"], int(off[-1]))
    for t in range(30):
        for j in range(2):
            r = s["dest_row"][t, j]
            if r >= 0:
                assert (xd[r] == x[t]).all()
    assert np.isnan(xd[s["src"] < 0]).all()


def test_hand_worked_example():
    """A six-token, three-expert, top-2 batch worked out by hand from Eq. 4 and
    the Section 4.1 rule (first entries of each expert tensor kept; priority:
    first choices in token order, then second choices).

    ids: t0 (0,1) t1 (0,2) t2 (1,0) t3 (0,1) t4 (2,0) t5 (0,2)
    counts: e0 = 6, e1 = 3, e2 = 3.
    Static alpha = 1: C = ceil(6*2/3) = 4 for every expert, offsets 0,4,8,12.
      first choices: t0->e0 pos 0, t1->e0 1, t2->e1 0, t3->e0 2, t4->e2 0, t5->e0 3
      second:        t0->e1 1, t1->e2 1, t2->e0 4 (drop), t3->e1 2, t4->e0 5 (drop),
                     t5->e2 2
    Dynamic 11/10: C = ceil(6.6), ceil(3.3), ceil(3.3) = 7, 4, 4, clamped to
    T = 6 -> 6, 4, 4; offsets 0,6,10,14; nothing dropped.
    Combine with Y_disp[r] = r + 1 (d = 1) under the static capacities:
      y0 = .75*1 + .25*6 = 2.25   y1 = .5*2 + .5*10 = 6   y2 = .6*5 = 3
      y3 = 1*3 + 0*7 = 3          y4 = .3*9 = 2.7         y5 = .2*4 + .8*11 = 9.6
    """
    ids = np.array([[0, 1], [0, 2], [1, 0], [0, 1], [2, 0], [0, 2]], dtype=np.int32)
    counts = O.count_assignments(ids, 3)
    assert list(counts) == [6, 3, 3]

    cap = O.capacity_static(6, 2, 3, 1, 1)
    assert list(cap) == [4, 4, 4]
    off = O.exclusive_offsets(cap)
    assert list(off) == [0, 4, 8, 12]
    s = O.assign_slots(ids, 3, cap, off, 12)
    assert s["dest_row"].tolist() == [[0, 5], [1, 9], [4, -1], [2, 6], [8, -1], [3, 10]]
    assert list(s["fill"]) == [4, 3, 3]
    assert list(s["src"]) == [0, 2, 6, 10, 4, 1, 7, -1, 8, 3, 11, -1]

    w = np.array([[.75, .25], [.5, .5], [.6, .4], [1., 0.], [.3, .7], [.2, .8]])
    Y = (np.arange(12, dtype=np.float64) + 1)[:, None]
    y = O.combine(Y, s["dest_row"], w, "f32")
    np.testing.assert_allclose(y[:, 0], [2.25, 6, 3, 3, 2.7, 9.6], rtol=1e-15)

    capd = O.capacity_dynamic(counts, 6, 11, 10)
    assert list(capd) == [6, 4, 4]
    offd = O.exclusive_offsets(capd)
    assert list(offd) == [0, 6, 10, 14]
    sd = O.assign_slots(ids, 3, capd, offd, 14)
    assert sd["dest_row"].tolist() == [[0, 7], [1, 11], [6, 4], [2, 8], [10, 5], [3, 12]]
    assert list(sd["fill"]) == [6, 3, 3]
    assert list(sd["src"]) == [0, 2, 6, 10, 5, 9, 4, 1, 7, -1, 8, 3, 11, -1]
