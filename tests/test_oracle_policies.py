"""Pins of the oracle's cache metric (Section 4.2), caching hysteresis
(Section 5.3) and launch-frontier capacity policy (Section 4.1 with the
recompile implementation appendix): hand-worked fixtures under
tests/golden/, brute force and closed forms."""
import itertools
import json
import os

import numpy as np
import pytest

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# -- cache metric ------------------------------------------------------------------
def test_cache_unchanged_is_order_free_set_equality():
    fresh = np.array([[1, 2], [1, 2], [1, 2], [0, 3], [2, 1]])
    cached = np.array([[2, 1], [1, 2], [1, 3], [3, 1], [1, 1]])
    np.testing.assert_array_equal(O.cache_unchanged(fresh, cached),
                                  [True, True, False, False, False])


def test_cache_unchanged_brute_force_against_sorted_rows():
    # for rows of distinct ids, set equality is equality of the sorted rows
    E, k = 5, 3
    rows = [p for p in itertools.permutations(range(E), k)]
    rng = np.random.default_rng(11)
    a = np.array([rows[i] for i in rng.integers(0, len(rows), 3000)])
    b = np.array([rows[i] for i in rng.integers(0, len(rows), 3000)])
    b[::3] = a[::3][:, ::-1]                   # many exact matches, reordered
    want = (np.sort(a, axis=1) == np.sort(b, axis=1)).all(axis=1)
    np.testing.assert_array_equal(O.cache_unchanged(a, b), want)


def test_cache_update_counts_then_remembers():
    fresh = np.array([[0, 1], [2, 3], [1, 0]], dtype=np.int32)
    cache = np.array([[1, 0], [3, 1], [1, 0]], dtype=np.int32)
    n, new = O.cache_update(fresh, cache)
    assert n == 2
    np.testing.assert_array_equal(new, fresh)
    n2, _ = O.cache_update(fresh, new)
    assert n2 == 3


# -- caching hysteresis (golden) ----------------------------------------------------
def test_caching_hysteresis_golden_schedule():
    g = _load("caching_hysteresis.json")
    th = g["thresholds"]
    enabled = False
    for st in g["steps"]:
        enabled = O.caching_decision(enabled, st["unchanged"], st["samples"], st["epoch"],
                                     tuple(th["on"]), tuple(th["off"]), th["min_epoch"])
        assert enabled == st["enabled"], st


# -- capacity policy ------------------------------------------------------------------
@pytest.mark.parametrize("run", [0, 1])
def test_capacity_policy_golden_example(run):
    g = _load("capacity_policy_example.json")
    r = g["runs"][run]
    np.testing.assert_array_equal(O.capacity_static(g["T"], g["k"], g["E"], 1, 1), g["init_cap"])
    sim = O.simulate_capacity_policy(g["counts"], g["T"], g["k"], r["delta"], g["init_cap"],
                                     tuple(g["grow"]), tuple(g["shrink"]), g["cap_min"])
    np.testing.assert_array_equal(sim["caps"], r["caps"])
    np.testing.assert_array_equal(sim["recompile"], r["recompile"])
    np.testing.assert_array_equal(sim["drops"], r["drops"])
    np.testing.assert_allclose(sim["factor"], r["factor"], rtol=1e-15)


@pytest.mark.parametrize("delta", [0, 1, 3])
def test_capacity_policy_step_change_takes_effect_delta_later(delta):
    # stationary demand, then a jump at iteration m: the capacities follow it
    # exactly at iteration m + 1 + delta, and never drop samples in between
    # the two recompiles except while the jump is not yet seen
    T, k, E, m = 1000, 2, 4, 6
    a = [500, 700, 500, 300]
    b = [800, 400, 400, 400]
    seq = [a] * m + [b] * 10
    init = O.capacity_static(T, k, E, 1, 1).tolist()
    sim = O.simulate_capacity_policy(seq, T, k, delta, init, (11, 10), (13, 10))
    grow_a = [min(T, -(-11 * c // 10)) for c in a]
    grow_b = [min(T, -(-11 * c // 10)) for c in b]
    first = 1 + delta
    for i in range(len(seq)):
        if i < first:
            want = init
        elif i < m + 1 + delta:
            want = grow_a
        else:
            want = grow_b
        np.testing.assert_array_equal(sim["caps"][i], want, err_msg=f"iteration {i}")
    assert sim["recompile"].sum() == 2
    late = np.arange(len(seq))
    assert (sim["drops"][(late >= m) & (late < m + 1 + delta)] > 0).all()
    assert (sim["drops"][late >= m + 1 + delta] == 0).all()


def test_capacity_policy_rejects_grow_above_shrink():
    with pytest.raises(ValueError):
        O.capacity_policy_trigger([5, 5], [5, 5], 10, (14, 10), (13, 10), 0)


def test_capacity_policy_cap_min_does_not_oscillate():
    # an expert with no demand keeps cap_min and triggers nothing
    sim = O.simulate_capacity_policy([[10, 0]] * 6, 20, 1, 0, [10, 10], (1, 1), (3, 2), cap_min=2)
    np.testing.assert_array_equal(sim["caps"][1:], [[10, 2]] * 5)
    assert sim["recompile"].tolist() == [False, True, False, False, False, False]
