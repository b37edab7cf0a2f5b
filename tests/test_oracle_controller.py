"""Controller twin pinned by the paper's worked example, Eq. 2's fixed point and direction,
the reset rule, and convergence on a linear mixed-iteration latency model (Eq. 1)."""
import json
import math
import os

import pytest

from oracle import controller as oc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "controller_observability.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def test_worked_example():
    g = _golden()
    got = oc.next_cap(g["cap_before"], g["target_ms"], g["observed_ms"], g["c_min"], g["c_max"],
                      g["quantum"])
    assert got == g["cap_after"]


def test_worked_example_through_state_machine():
    g = _golden()
    c = oc.Controller(g["target_ms"], g["c_initial"], g["c_min"], g["c_max"], g["quantum"])
    assert c.step(num_decoding_next=5, last_was_guarded=True, observed_ms=g["observed_ms"]) == \
        g["cap_after"]


def test_floor_not_ceil():
    # 3072*80/57.51 = 4273.3 = 33.4 quanta: ceil would give 4352, floor gives the printed 4224
    x = 3072 * 80 / 57.51
    assert 128 * math.ceil(x / 128) == 4352
    assert oc.floor_quantum(x) == 4224
    # where floor and round-to-nearest differ (x.6 quanta), Eq. 2's floor takes the lower step
    assert oc.floor_quantum(128 * 33.6) == 128 * 33


def test_fixed_point_and_direction():
    for cap in (1024, 2048, 3072, 4096, 6144):
        assert oc.next_cap(cap, 80.0, 80.0, 1024, 6144) == cap
    assert oc.next_cap(3072, 80.0, 100.0, 1024, 6144) < 3072   # too slow: shrink
    assert oc.next_cap(3072, 80.0, 60.0, 1024, 6144) > 3072    # fast: grow


def test_clamps():
    assert oc.next_cap(3072, 80.0, 1e6, 1024, 6144) == 1024
    assert oc.next_cap(3072, 80.0, 1e-3, 1024, 6144) == 6144


def test_monotone_in_observation():
    caps = [oc.next_cap(3072, 80.0, L, 32, 4096) for L in (20, 40, 60, 80, 100, 150, 300)]
    assert caps == sorted(caps, reverse=True)


def test_dead_zones_below_the_quantum():
    # c_min = 32 < 128: growth from 32 needs T/L >= 4, from 128 needs T/L >= 2
    assert oc.next_cap(32, 80.0, 20.01, 32, 4096) == 32
    assert oc.next_cap(32, 80.0, 20.0, 32, 4096) == 128
    assert oc.next_cap(128, 80.0, 40.01, 32, 4096) == 128
    assert oc.next_cap(128, 80.0, 40.0, 32, 4096) == 256
    assert oc.next_cap(200, 80.0, 1000.0, 32, 4096) == 32


def test_reset_when_no_decoder_and_guard():
    c = oc.Controller(80.0, 3072, 1024, 6144)
    assert c.step(4, True, 160.0) == 1536
    # an unguarded cycle never updates, whatever it measured
    assert c.step(4, False, 10.0) == 1536
    # no decoder next: uncapped, and the cap returns to c_initial
    assert c.step(0, True, 160.0) == oc.UNCAPPED
    assert c.cap == 3072
    assert c.step(2, False, float("nan")) == 3072


@pytest.mark.parametrize("bad", [0.0, -1.0, float("nan"), float("inf")])
def test_rejects_bad_observation(bad):
    c = oc.Controller(80.0, 3072, 1024, 6144)
    with pytest.raises(ValueError):
        c.step(3, True, bad)
    assert c.cap == 3072


def test_convergence_on_linear_latency_model():
    """L(c) = a + b*c (Eq. 1 with the decode and overhead shares in a).  c*T/L(c) is
    increasing with fixed point c* = (T - a) / b, so from above one step lands within a
    quantum below c*; from below the cap grows until the floor stalls it, which happens
    exactly when c*T/L(c) - c < 128, i.e. c* - c < 128 * (1 + a / (b c)).  The loop must
    settle on such a stalled 128-multiple, never above c*."""
    for a, b, T, c0 in [(20.0, 0.02, 80.0, 3072), (5.0, 0.05, 80.0, 3072),
                        (60.0, 0.003, 80.0, 3072), (60.0, 0.003, 80.0, 8192),
                        (20.0, 0.02, 80.0, 128)]:
        c = oc.Controller(T, c0, 128, 8192)
        cap = c.cap
        for _ in range(80):
            cap = c.step(1, True, a + b * cap)
        c_star = (T - a) / b
        assert cap % 128 == 0
        assert cap <= c_star + 1e-9, (a, b, T, cap, c_star)
        assert c_star - cap < 128 * (1 + a / (b * cap)), (a, b, T, cap, c_star)
        # and it is a true fixed point of the update
        assert oc.next_cap(cap, T, a + b * cap, 128, 8192) == cap
