"""Replay on the device: the scheduler drives the real append + single attention launch
and the controller reads HIP-event completion times.  Latencies are parity unpinned
(they depend on the GPU); reconciliation, the controller's guard and every control
decision are checked: the recorded latency trace, replayed through the oracle's Eq. 2
controller, must give the same cap before every iteration."""
import pytest
import torch

from oracle import controller as oc
from paper_2609_38386_amd import replay as rp

pytestmark = pytest.mark.gpu


def expected_limits(trace, cfg, target):
    """Prefill limit of every iteration after the first, from the oracle controller fed
    the trace's guarded flags and measured latencies (C3/C4: update after a guarded
    cycle, reset when the next cycle has no decoder)."""
    ctrl = oc.Controller(target, cfg.c_initial, cfg.c_min, cfg.c_max, cfg.quantum)
    out = []
    for prev, nxt in zip(trace, trace[1:]):
        cap = ctrl.step(nxt["decoders"], prev["guarded"], prev["layer_ms"])
        budget = cfg.budget - nxt["decoders"]
        out.append(budget if cap == oc.UNCAPPED else min(cap, budget))
    return out


def test_gpu_replay_uncapped_and_dlfp():
    assert torch.cuda.is_available()
    dev = torch.device("cuda:0")
    cfg = rp.ReplayConfig(seed=802, n_requests=12, rate_per_s=400.0, prompt_hi=2048, out_len=24)
    ex = rp.GpuExecutor(cfg, dev)
    trace = []
    base = rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), ex, trace=trace)
    assert base["reconciled"]
    dec_only = sorted(it["layer_ms"] for it in trace if it["decoders"] > 0 and it["p_t"] == 0)
    assert dec_only and all(0.0 < x < 50.0 for x in dec_only)
    target = 1.2 * dec_only[len(dec_only) // 2]
    trace2 = []
    dl = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP, target_ms=target, cfg=cfg), ex,
                       trace=trace2)
    assert dl["reconciled"]
    assert all(it["limit"] == cfg.budget for it in trace2 if it["decoders"] == 0)
    assert dl["guarded_iterations"] > 0
    # every decision equals the oracle controller's on the recorded latencies
    want = expected_limits(trace2, cfg, target)
    got = [it["limit"] for it in trace2[1:]]
    assert got == want
    assert len(set(got)) > 2   # the cap moved


def test_gpu_replay_with_the_layer_proxy():
    """With the layer's projections timed beside the attention (Eq. 1's linear
    term) the iteration latency grows with the prefill chunk, and the
    completion-timed controller's decisions still match the oracle's."""
    import numpy as np
    assert torch.cuda.is_available()
    dev = torch.device("cuda:0")
    cfg = rp.ReplayConfig(seed=803, n_requests=10, rate_per_s=400.0, prompt_hi=4096, out_len=16,
                          layer_proxy=True)
    ex = rp.GpuExecutor(cfg, dev)
    trace = []
    base = rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), ex, trace=trace)
    assert base["reconciled"]
    pts = [(it["p_t"], it["layer_ms"]) for it in trace if it["p_t"] > 0]
    p = np.asarray([x[0] for x in pts], dtype=np.float64)
    ms = np.asarray([x[1] for x in pts])
    assert len(pts) >= 4 and np.corrcoef(p, ms)[0, 1] > 0.8
    dec_only = sorted(it["layer_ms"] for it in trace if it["decoders"] > 0 and it["p_t"] == 0)
    target = 1.2 * dec_only[len(dec_only) // 2]
    trace2 = []
    dl = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP, target_ms=target, cfg=cfg), ex,
                       trace=trace2)
    assert dl["reconciled"]
    assert [it["limit"] for it in trace2[1:]] == expected_limits(trace2, cfg, target)


def test_gpu_retimed_layer_leaves_the_same_state():
    """An iteration whose enqueue outlasts the stream hold is timed a second
    time; its launches are idempotent, so the pages and outputs after a replay
    in which every iteration is timed twice (a 1 us hold) equal, bit for bit,
    those of a replay timed once per iteration.  Uncapped decisions do not
    depend on the measured latencies, so both replays run the same batches."""
    assert torch.cuda.is_available()
    dev = torch.device("cuda:0")
    cfg = rp.ReplayConfig(seed=804, n_requests=5, rate_per_s=400.0, prompt_hi=1536, out_len=6,
                          layer_proxy=True)
    once, twice = rp.GpuExecutor(cfg, dev), rp.GpuExecutor(cfg, dev)
    twice.hold_us = 1
    t1, t2 = [], []
    r1 = rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), once, trace=t1)
    r2 = rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), twice, trace=t2)
    assert r1["reconciled"] and r2["reconciled"]
    assert [(x["p_t"], x["decoders"]) for x in t1] == [(x["p_t"], x["decoders"]) for x in t2]
    assert twice.retimed == len(t2)
    assert all(x["layer_ms"] > 0.0 for x in t2)
    torch.cuda.synchronize()
    rows = max(x["p_t"] + x["decoders"] for x in t1)   # rows ever written
    for a, b in ((once.pool.k, twice.pool.k), (once.pool.v, twice.pool.v),
                 (once.out[:rows], twice.out[:rows]), (once.y2[:rows], twice.y2[:rows])):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
