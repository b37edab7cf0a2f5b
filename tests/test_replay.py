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
