"""Host-side C functions of the library against the oracle, on the CPU (no
device work): the caching decision with hysteresis (Section 5.3) and the
capacity trigger (Section 4.1 with the recompile implementation appendix),
bit-exact on the golden fixtures and on random inputs."""
import json
import os

import numpy as np
import pytest

import oracle as O
from paper_2205_01848_amd import binding as B

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_caching_decision_golden_schedule():
    with open(os.path.join(GOLDEN, "caching_hysteresis.json")) as f:
        g = json.load(f)
    th = g["thresholds"]
    enabled = False
    for st in g["steps"]:
        enabled = B.moe_caching_decision(enabled, st["unchanged"], st["samples"], st["epoch"],
                                         tuple(th["on"]), tuple(th["off"]), th["min_epoch"])
        assert enabled == st["enabled"], st


def test_caching_decision_matches_oracle_random():
    rng = np.random.default_rng(21)
    for _ in range(3000):
        n = int(rng.integers(0, 5000))
        u = int(rng.integers(0, n + 1))
        on = (int(rng.integers(1, 100)), 100)
        off = (int(rng.integers(1, on[0] + 1)), 100)
        en = bool(rng.integers(0, 2))
        ep = int(rng.integers(0, 30))
        me = int(rng.integers(0, 20))
        assert B.moe_caching_decision(en, u, n, ep, on, off, me) == \
            O.caching_decision(en, u, n, ep, on, off, me)


def test_caching_decision_large_counts_exact():
    n = 10 ** 15
    assert B.moe_caching_decision(False, 96 * 10 ** 13, n, 10) is True
    assert B.moe_caching_decision(False, 96 * 10 ** 13 - 1, n, 10) is False
    assert B.moe_caching_decision(True, 9 * 10 ** 14, n, 10) is True
    assert B.moe_caching_decision(True, 9 * 10 ** 14 - 1, n, 10) is False


def test_capacity_trigger_golden_sequence():
    with open(os.path.join(GOLDEN, "capacity_policy_example.json")) as f:
        g = json.load(f)
    run = g["runs"][0]     # delta = 0: the trigger before i sees the counts of i - 1
    cap = list(g["init_cap"])
    for i in range(1, len(g["counts"])):
        cap, rec = B.moe_capacity_trigger(g["T"], g["counts"][i - 1], cap, tuple(g["grow"]),
                                          tuple(g["shrink"]), g["cap_min"])
        assert cap == run["caps"][i] and rec == run["recompile"][i]


@pytest.mark.parametrize("seed", range(4))
def test_capacity_trigger_matches_oracle_random(seed):
    rng = np.random.default_rng(100 + seed)
    for _ in range(2000):
        E = int(rng.integers(1, 65))
        T = int(rng.integers(0, 3000))
        counts = rng.integers(0, T + 1, E).tolist()
        cap = rng.integers(0, T + 1, E).tolist()
        gd = int(rng.integers(1, 50))
        gn = int(rng.integers(gd, 3 * gd))
        sd = int(rng.integers(1, 50))
        sn = int(rng.integers(-(-gn * sd // gd), 4 * sd + gn * sd // gd + 1))
        cm = int(rng.integers(0, 5))
        got = B.moe_capacity_trigger(T, counts, cap, (gn, gd), (sn, sd), cm)
        want = O.capacity_policy_trigger(cap, counts, T, (gn, gd), (sn, sd), cm)
        assert got == (list(want[0]), want[1])


def test_capacity_trigger_rejects_grow_above_shrink():
    with pytest.raises(B.MoEError):
        B.moe_capacity_trigger(10, [5, 5], [5, 5], (14, 10), (13, 10))
