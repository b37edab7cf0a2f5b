"""Replay scheduler and controller loop on the CPU with a deterministic latency model.

Replay latencies on the device are parity unpinned (they depend on the GPU);
what is pinned here is determinism given a latency trace, the guard and reset
rules, token reconciliation, and the controller's direction of travel.
"""
import dataclasses

import numpy as np
import pytest

from paper_2609_38386_amd import replay as rp


def _cfg(**kw):
    base = dict(seed=801, n_requests=24, rate_per_s=40.0, prompt_lo=256, prompt_hi=4096,
                out_len=16, layers=28)
    base.update(kw)
    return rp.ReplayConfig(**base)


def test_reconciliation_and_itl_count():
    cfg = _cfg()
    reqs = []
    r = rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), rp.linear_latency_model(),
                      requests_out=reqs)
    assert r["reconciled"]
    assert r["itl_observations"] == cfg.n_requests * (cfg.out_len - 1)
    assert r["output_tokens"] == cfg.n_requests * cfg.out_len
    # a dropped token breaks reconciliation
    reqs[3].itl_ms.pop()
    assert not rp.reconcile(reqs)


def test_deterministic_given_latency_model():
    cfg = _cfg()
    t1, t2 = [], []
    a = rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), rp.linear_latency_model(), trace=t1)
    b = rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), rp.linear_latency_model(), trace=t2)
    assert a == b and t1 == t2


def test_isolated_prefill_uncapped_and_guard():
    cfg = _cfg()
    trace = []
    pol = rp.Policy(rp.Policy.DLFP, target_ms=0.02, cfg=cfg)
    rp.run_replay(cfg, pol, rp.linear_latency_model(), trace=trace)
    for it in trace:
        if it["decoders"] == 0:
            assert it["limit"] == cfg.budget          # no decoder: prefill not capped
        else:
            assert it["limit"] <= cfg.c_max           # decoder present: capped
    assert any(it["guarded"] for it in trace)


def test_controller_shrinks_cap_under_slow_prefill():
    cfg = _cfg(n_requests=12, rate_per_s=200.0, out_len=64)
    trace = []
    # prefill is expensive relative to the target: the cap must come down from c_initial
    pol = rp.Policy(rp.Policy.DLFP, target_ms=0.03, cfg=cfg)
    rp.run_replay(cfg, pol, rp.linear_latency_model(0.01, 1e-5, 1e-4), trace=trace)
    caps = [it["limit"] for it in trace if it["decoders"] > 0 and it["p_t"] > 0]
    assert caps and min(caps) < cfg.c_initial
    # fixed point of Eq. 2 under the model: L = 0.01 + 1e-5 c (+ decoders) near T = 0.03
    assert min(caps) <= 2048


def test_dlfp_trades_ttft_for_tail_itl_when_requests_overlap():
    """Under load where prompts routinely arrive beside decoders, capping overlapped
    prefill lowers the decoders' tail latency and raises time to first token
    (the trade-off of Sec. 5.2)."""
    cfg = _cfg(n_requests=40, rate_per_s=300.0, out_len=32)
    model = rp.linear_latency_model(0.01, 2e-5, 2e-4)
    base = rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), model)
    dl = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP, target_ms=0.03, cfg=cfg), model)
    assert base["reconciled"] and dl["reconciled"]
    assert dl["itl_p99_ms"] < 0.8 * base["itl_p99_ms"]
    assert dl["ttft_p99_ms"] > base["ttft_p99_ms"]


def test_fixed_cap_policy():
    cfg = _cfg()
    trace = []
    rp.run_replay(cfg, rp.Policy(rp.Policy.FIXED, cap=1024), rp.linear_latency_model(),
                  trace=trace)
    assert all(it["p_t"] <= 1024 for it in trace if it["decoders"] > 0)


def test_paired_ci_matches_student_t():
    mean, lo, hi = rp.paired_ci([24.767, 30.053, 28.209])
    assert abs(mean - 27.68) < 0.01 and abs(lo - 21.01) < 0.02 and abs(hi - 34.34) < 0.02


def test_controlled_cycles_hold_a_reachable_target():
    """Once a feedback update has set the cap (Eq. 2), guarded cycles sit at the
    target when the smallest chunk can meet it; the first cycle of an episode
    runs at c_initial and is reported apart."""
    cfg = _cfg(n_requests=12, rate_per_s=200.0, out_len=64)
    model = rp.linear_latency_model(0.01, 1e-5, 1e-4)
    r = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP, target_ms=0.03, cfg=cfg), model)
    assert r["controlled_iterations"] > 0
    assert r["controlled_iterations"] < r["guarded_iterations"]
    assert 0.8 <= r["controlled_L_over_T_mean"] <= 1.1
    assert r["controlled_within_target"] >= 0.5
    assert r["guarded_L_over_T_mean"] >= r["controlled_L_over_T_mean"]
    assert r["controlled_within_5pct"] >= r["controlled_within_target"]
    assert r["controlled_L_over_T_p50"] <= r["controlled_L_over_T_p90"]
    base = rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), model)
    assert base["controlled_iterations"] == 0 and base["controlled_L_over_T_mean"] is None


def test_stale_completion_signal_holds_the_target_worse():
    """Eq. 2 fed each completion one iteration late (an asynchronous engine
    setting the cap of t + 1 while t runs, Sec. 6.4) under the same overlapped
    load: its first cycles after an arrival still run at the old cap, so the
    decoders' tail latency is no better and the guarded cycles sit within 5% of
    the target less often than with the completion-timed signal."""
    cfg = _cfg(n_requests=40, rate_per_s=300.0, out_len=32)
    model = rp.linear_latency_model(0.01, 2e-5, 2e-4)
    dl = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP, target_ms=0.03, cfg=cfg), model)
    lag = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP_LAG1, target_ms=0.03, cfg=cfg), model)
    assert lag["reconciled"] and lag["controlled_iterations"] > 0
    assert lag["itl_p99_ms"] >= dl["itl_p99_ms"]
    assert lag["controlled_within_5pct"] < dl["controlled_within_5pct"]


def _overlap_cfg(**kw):
    return _cfg(n_requests=40, rate_per_s=300.0, out_len=32, **kw)


def test_cadence_signal_misjudges_the_device_latency_under_async_scheduling():
    """Sec. 3.2 / Sec. 6.4: with the scheduler one iteration ahead of the device,
    the interval between scheduler calls that follows a guarded cycle is set by
    the host's own cost and by the iteration queued before it, not by the
    guarded cycle's device time.  Fed to Eq. 2, it moves the cap the wrong way
    on many updates (expanding it after a short interval while a long chunk is
    still running), and the decoders' tail latency comes back close to the
    uncapped one; the completion time, delivered when it is available (one
    iteration late under this scheduling), keeps most of the reduction."""
    cfg = _overlap_cfg(pipeline="async", host_ms=0.3)
    model = rp.linear_latency_model(0.01, 2e-5, 2e-4)
    base = rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), model)
    comp = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP_LAG1, target_ms=0.03, cfg=cfg), model)
    cad = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP_CADENCE, target_ms=0.03, cfg=cfg), model)
    assert base["reconciled"] and comp["reconciled"] and cad["reconciled"]
    assert cad["signal_rel_error_mean"] > 0.3
    assert cad["wrong_direction_updates"] > 0.3
    assert cad["itl_p99_ms"] > 1.3 * comp["itl_p99_ms"]
    assert cad["itl_p99_ms"] > 0.8 * base["itl_p99_ms"]
    assert cad["controlled_within_5pct"] < comp["controlled_within_5pct"]
    assert comp["itl_p99_ms"] < 0.7 * base["itl_p99_ms"]


def test_cadence_equals_completion_when_the_host_is_synchronous_and_free():
    """With a synchronous scheduler and no host cost, the interval between calls
    is exactly the iteration's completion time: the two signals coincide."""
    cfg = _overlap_cfg(pipeline="sync", host_ms=0.0)
    model = rp.linear_latency_model(0.01, 2e-5, 2e-4)
    t1, t2 = [], []
    a = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP, target_ms=0.03, cfg=cfg), model, trace=t1)
    b = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP_CADENCE, target_ms=0.03, cfg=cfg), model,
                      trace=t2)
    assert [x["limit"] for x in t1] == [x["limit"] for x in t2]
    assert a["itl_p99_ms"] == b["itl_p99_ms"]
    assert b["signal_rel_error_mean"] < 1e-9
    # with no host cost and no pipelining the clock is the device time alone
    plain = rp.run_replay(_overlap_cfg(), rp.Policy(rp.Policy.DLFP, target_ms=0.03,
                                                    cfg=_overlap_cfg()), model)
    assert plain["itl_p99_ms"] == pytest.approx(a["itl_p99_ms"])


def test_completion_aware_revision_bounds_each_step():
    """Sec. 6.3: the revised controller updates when the cycle's output returns
    (host time from the scheduler call, so the host's own cost is counted) and
    changes the cap by at most a factor of two per update.  Under synchronous
    scheduling it keeps the tail inter-token latency low but, with the host cost
    counted as device latency, pins the cap near its floor and multiplies the
    time to first token (it moves latency rather than removing it)."""
    cfg = _overlap_cfg(pipeline="sync", host_ms=0.3)
    model = rp.linear_latency_model(0.01, 2e-5, 2e-4)
    trace = []
    rev = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP_REVISED, target_ms=0.03, cfg=cfg), model,
                        trace=trace)
    base = rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), model)
    assert rev["reconciled"]
    caps = [x["limit"] for x in trace if x["decoders"] > 0]
    steps = [(a, b) for a, b in zip(caps, caps[1:]) if a <= cfg.c_max and b <= cfg.c_max]
    assert steps
    for a, b in steps:
        assert b <= 2 * a
        assert b >= min(a, max(cfg.c_min, (a // 2) // cfg.quantum * cfg.quantum))
    assert rev["itl_p99_ms"] < base["itl_p99_ms"]
    assert rev["ttft_p99_ms"] > 3 * base["ttft_p99_ms"]
    # the bound is a clamp of the observation to [T / 2, 2 T] before Eq. 2
    pol = rp.Policy(rp.Policy.DLFP_REVISED, target_ms=0.03, cfg=cfg)
    pol.observe(3, True, {"returned": 10.0})
    assert pol.ctrl.cap == cfg.c_initial // 2 // 128 * 128
