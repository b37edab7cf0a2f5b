"""Closed-loop continuous-batching replay driven by the completion-timed controller.

Requests arrive open-loop (independent exponential gaps, Sec. 4.2) with
prompt lengths drawn uniformly and a fixed number of output tokens.  Each
iteration the scheduler (iteration-level scheduling with chunked prefill,
Sec. 2.1) forms the batch:

* every request whose prompt is complete and that still owes tokens decodes
  one token (the set D_t);
* prompt tokens are admitted first-come-first-served up to the iteration's
  prefill limit: the controller's cap c_t when at least one request is
  decoding, otherwise only the engine's token budget -- isolated prefill is not
  capped (Sec. 3.1, Sec. 3.2);
* at most ``max_seqs`` sequences and ``budget`` tokens per iteration (the
  engine limits of Sec. 4.1).

The iteration runs on the device (KV append plus the single attention launch
for one layer); its completion time, measured with HIP events after the work
has finished, is the observation L_t fed to Eq. 2 (Sec. 3.1) -- not the
interval between scheduler calls (Sec. 3.2, Sec. 6.4).  A guarded cycle is one
with at least one decoder and a non-empty prefill.  The virtual clock advances
by ``layers`` x the measured one-layer latency per iteration and idles to the
next arrival when nothing is runnable.

Reported per run: inter-token latencies seen by decoders (one observation per
decode token: the latency of the iteration that produced it), time to first
token, end-to-end latency, guarded-iteration count and L/T on guarded
iterations, and token reconciliation.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from . import workload as wl

PAGE = 16


@dataclasses.dataclass
class Request:
    rid: int
    arrival_s: float
    prompt_len: int
    out_len: int
    prefilled: int = 0
    generated: int = 0
    pages: List[int] = dataclasses.field(default_factory=list)
    first_token_s: Optional[float] = None
    done_s: Optional[float] = None
    itl_ms: List[float] = dataclasses.field(default_factory=list)

    @property
    def kv_len(self) -> int:
        return self.prefilled + max(self.generated - 1, 0)

    @property
    def decoding(self) -> bool:
        return self.prefilled == self.prompt_len and self.generated < self.out_len


class PageAllocator:
    """Free list over a seeded random permutation of the pool."""

    def __init__(self, num_blocks: int, seed: int):
        self.free = list(wl.rng_for(seed, wl.ROLE_PAGE_PERMUTATION).permutation(num_blocks)[::-1])

    def grow(self, req: Request, tokens: int):
        need = (tokens + PAGE - 1) // PAGE
        while len(req.pages) < need:
            if not self.free:
                raise RuntimeError("KV pool exhausted")
            req.pages.append(int(self.free.pop()))

    def release(self, req: Request):
        self.free.extend(reversed(req.pages))
        req.pages = []


@dataclasses.dataclass
class ReplayConfig:
    seed: int = 801
    n_requests: int = 100
    rate_per_s: float = 2.0
    prompt_lo: int = 256
    prompt_hi: int = 4096
    out_len: int = 128
    max_seqs: int = 64
    budget: int = 8192
    layers: int = 28
    num_q_heads: int = 16
    num_kv_heads: int = 8
    # controller (Eq. 2); the target is set per run
    c_initial: int = 3072
    c_min: int = 32
    c_max: int = 4096
    quantum: int = 128

    @property
    def max_blocks(self) -> int:
        return (self.prompt_hi + self.out_len + PAGE - 1) // PAGE

    def num_blocks(self) -> int:
        return self.max_seqs * self.max_blocks + 64


class Policy:
    """Prefill limit for the next iteration."""

    UNCAPPED = "uncapped"
    FIXED = "fixed"
    DLFP = "dlfp"
    # Eq. 2 fed one iteration late: an asynchronous engine that sets the cap of
    # iteration t + 1 while iteration t still runs only has the completion time
    # of iteration t - 1 (the stale signal of Sec. 6.4).
    DLFP_LAG1 = "dlfp_lag1"

    def __init__(self, kind: str, cap: int = 0, target_ms: float = 0.0, cfg: ReplayConfig = None):
        self.kind = kind
        self.fixed_cap = cap
        self.target_ms = target_ms
        self.ctrl = None
        self.pending = None       # DLFP_LAG1: the observation not yet delivered
        if kind in (self.DLFP, self.DLFP_LAG1):
            from . import dlfp as D
            self._D = D
            self.ctrl = D.dlfp_controller_init(target_ms, cfg.c_initial, cfg.c_min, cfg.c_max,
                                               cfg.quantum)
        self.next_cap = -1 if kind != self.FIXED else cap
        # True when the next cycle's cap comes from a feedback update (Eq. 2)
        # rather than from c_initial after a reset.
        self.controlled = False

    def limit(self, n_decoding: int, budget: int) -> int:
        if n_decoding == 0 or self.kind == self.UNCAPPED:
            return budget
        if self.kind == self.FIXED:
            return min(self.fixed_cap, budget)
        cap = self.next_cap if self.next_cap > 0 else self.ctrl.cap
        return min(cap, budget)

    def observe(self, n_decoding_next: int, guarded: bool, observed_ms: float):
        if self.kind == self.DLFP_LAG1:
            # this iteration's completion is delivered one call later; the
            # previous one's arrives now (nothing before the first completion)
            prev, self.pending = self.pending, (guarded, observed_ms)
            guarded, observed_ms = prev if prev is not None else (False, observed_ms)
        if self.kind in (self.DLFP, self.DLFP_LAG1):
            if guarded:
                self.controlled = True
            elif n_decoding_next == 0:
                self.controlled = False
            self.next_cap = self._D.dlfp_controller_step(self.ctrl, n_decoding_next, guarded,
                                                         observed_ms)


Executor = Callable[[np.ndarray, np.ndarray, np.ndarray], float]


def run_replay(cfg: ReplayConfig, policy: Policy, execute: Executor,
               trace: Optional[list] = None, requests_out: Optional[list] = None) -> Dict:
    """Run the replay; ``execute(q_len, kv_len, block_table) -> one-layer ms``."""
    arrivals = wl.poisson_arrivals(cfg.seed, cfg.n_requests, cfg.rate_per_s)
    prompts = wl.prompt_lengths(cfg.seed, cfg.n_requests, cfg.prompt_lo, cfg.prompt_hi)
    reqs = [Request(i, float(arrivals[i]), int(prompts[i]), cfg.out_len)
            for i in range(cfg.n_requests)]
    if requests_out is not None:
        requests_out.extend(reqs)
    alloc = PageAllocator(cfg.num_blocks(), cfg.seed)
    clock = 0.0
    nxt = 0                      # next request to arrive
    active: List[Request] = []   # arrived and not finished, in arrival order
    iterations = guarded_n = 0
    guarded_ratio = []
    controlled_ratio = []   # guarded cycles whose cap came from a feedback update
    while nxt < len(reqs) or active:
        if not active:
            clock = max(clock, reqs[nxt].arrival_s)
        while nxt < len(reqs) and reqs[nxt].arrival_s <= clock:
            active.append(reqs[nxt])
            nxt += 1
        decoders = [r for r in active if r.decoding][:cfg.max_seqs]
        limit = policy.limit(len(decoders), cfg.budget - len(decoders))
        slices = []
        left = limit
        for r in active:
            if len(decoders) + len(slices) >= cfg.max_seqs or left <= 0:
                break
            if r.prefilled < r.prompt_len:
                take = min(r.prompt_len - r.prefilled, left)
                slices.append((r, take))
                left -= take
        p_t = sum(t for _, t in slices)
        guarded = len(decoders) > 0 and p_t > 0
        # batch: prefill slices first, then decoders; kv_len includes this step's tokens
        q_len, kv_len, rows = [], [], []
        for r, take in slices:
            alloc.grow(r, r.prefilled + take)
            q_len.append(take)
            kv_len.append(r.prefilled + take)
            rows.append(r.pages)
        for r in decoders:
            alloc.grow(r, r.kv_len + 1)
            q_len.append(1)
            kv_len.append(r.kv_len + 1)
            rows.append(r.pages)
        bt = np.full((len(rows), cfg.max_blocks), -1, dtype=np.int32)
        for i, pages in enumerate(rows):
            bt[i, :len(pages)] = pages
        controlled = policy.controlled
        ms = float(execute(np.asarray(q_len, np.int32), np.asarray(kv_len, np.int32), bt))
        iter_ms = cfg.layers * ms
        clock += iter_ms * 1e-3
        iterations += 1
        for r, take in slices:
            r.prefilled += take
            if r.prefilled == r.prompt_len:
                r.generated = 1
                r.first_token_s = clock
        for r in decoders:
            r.generated += 1
            r.itl_ms.append(iter_ms)
        for r in list(active):
            if r.generated >= r.out_len:
                r.done_s = clock
                alloc.release(r)
                active.remove(r)
        n_next = sum(1 for r in active if r.decoding)
        if guarded:
            guarded_n += 1
            if policy.target_ms:
                guarded_ratio.append(ms / policy.target_ms)
                if controlled:
                    controlled_ratio.append(ms / policy.target_ms)
        policy.observe(n_next, guarded, ms)
        if trace is not None:
            trace.append({"t": round(clock, 6), "decoders": len(decoders), "p_t": p_t,
                          "limit": limit, "layer_ms": round(ms, 5), "guarded": guarded})
    itl = np.concatenate([np.asarray(r.itl_ms) for r in reqs if r.itl_ms] or [np.zeros(0)])
    ttft = np.asarray([(r.first_token_s - r.arrival_s) * 1e3 for r in reqs])
    e2e = np.asarray([(r.done_s - r.arrival_s) * 1e3 for r in reqs])
    reconciled = reconcile(reqs)
    return {
        "iterations": iterations,
        "guarded_iterations": guarded_n,
        "itl_observations": int(itl.size),
        "itl_p50_ms": float(np.percentile(itl, 50)) if itl.size else None,
        "itl_p99_ms": float(np.percentile(itl, 99)) if itl.size else None,
        "itl_mean_ms": float(itl.mean()) if itl.size else None,
        "ttft_p50_ms": float(np.percentile(ttft, 50)),
        "ttft_p99_ms": float(np.percentile(ttft, 99)),
        "e2e_p99_ms": float(np.percentile(e2e, 99)),
        "guarded_L_over_T_mean": float(np.mean(guarded_ratio)) if guarded_ratio else None,
        "controlled_iterations": len(controlled_ratio),
        "controlled_L_over_T_mean": float(np.mean(controlled_ratio)) if controlled_ratio else None,
        "controlled_within_target": (float(np.mean(np.asarray(controlled_ratio) <= 1.0))
                                     if controlled_ratio else None),
        "controlled_within_5pct": (float(np.mean(np.asarray(controlled_ratio) <= 1.05))
                                   if controlled_ratio else None),
        "controlled_L_over_T_p50": (float(np.percentile(controlled_ratio, 50))
                                    if controlled_ratio else None),
        "controlled_L_over_T_p90": (float(np.percentile(controlled_ratio, 90))
                                    if controlled_ratio else None),
        "reconciled": reconciled,
        "prompt_tokens": int(sum(r.prompt_len for r in reqs)),
        "output_tokens": int(sum(r.generated for r in reqs)),
    }


def reconcile(reqs: Sequence[Request]) -> bool:
    """Every request fully prefilled, every output token produced, one inter-token
    observation per decode step (out_len - 1 per request)."""
    return all(r.prefilled == r.prompt_len and r.generated == r.out_len and
               len(r.itl_ms) == r.out_len - 1 and r.first_token_s is not None and
               r.done_s is not None for r in reqs)


def paired_ci(reductions: Sequence[float], confidence: float = 0.95):
    """Mean and two-sided Student-t interval over paired trial-level reductions."""
    from scipy import stats as st
    x = np.asarray(reductions, dtype=np.float64)
    n = len(x)
    mean = float(x.mean())
    if n < 2:
        return mean, None, None
    half = float(st.t.ppf(0.5 + confidence / 2, n - 1) * x.std(ddof=1) / math.sqrt(n))
    return mean, mean - half, mean + half


class GpuExecutor:
    """Runs one layer of an iteration on the device: KV append plus the attention
    launch, timed with HIP events and read after completion."""

    def __init__(self, cfg: ReplayConfig, device, seed: int = 0):
        import torch
        from . import dlfp as D
        from . import runtime as rt
        self.torch, self.D = torch, D
        self.dims = D.make_dims(cfg.num_q_heads, cfg.num_kv_heads)
        self.num_blocks = cfg.num_blocks()
        self.pool = rt.KVPool(self.num_blocks, cfg.num_kv_heads, device)
        gen = torch.Generator(device=device)
        gen.manual_seed(cfg.seed + seed)
        self.pool.k.normal_(generator=gen)
        self.pool.v.normal_(generator=gen)
        rows = cfg.budget + cfg.max_seqs
        self.q = torch.empty((rows, cfg.num_q_heads, 128), dtype=torch.bfloat16, device=device)
        self.k = torch.empty((rows, cfg.num_kv_heads, 128), dtype=torch.bfloat16, device=device)
        self.v = torch.empty_like(self.k)
        for t in (self.q, self.k, self.v):
            t.normal_(generator=gen)
        self.out = torch.empty_like(self.q)
        self.stage = rt.StagedBatch(self.dims, cfg.max_seqs + 1, rows, 65536, device)
        bt_cap = (cfg.max_seqs + 1) * cfg.max_blocks
        self.bt_host = torch.empty(bt_cap, dtype=torch.int32, pin_memory=True)
        self.bt_dev = torch.empty(bt_cap, dtype=torch.int32, device=device)
        self.ws = rt.Workspace(device, 64 << 20)
        self.timer = D.Timer()
        self.scale = 1.0 / math.sqrt(128)
        self.hold_us = 150

    def __call__(self, q_len: np.ndarray, kv_len: np.ndarray, bt: np.ndarray) -> float:
        D = self.D
        st = self.stage.build(q_len, kv_len, bt, self.num_blocks)
        n = bt.size
        self.bt_host.numpy()[:n] = bt.reshape(-1)
        d_bt = self.bt_dev[:n].view(bt.shape[0], bt.shape[1])
        d_bt.view(-1).copy_(self.bt_host[:n], non_blocking=True)
        T = st.num_tokens
        ws = self.ws.ensure(st.meta.workspace_bytes)
        # Launch marshalling happens while the stream idles, so the events bracket
        # the layer's device work and not the host's launch gaps.
        D.dlfp_stream_hold(self.hold_us)
        self.timer.start()
        D.dlfp_append_attention_mixed(self.dims, st.meta, st.d_work, d_bt, self.q[:T],
                                      self.k[:T], self.v[:T], self.pool.k, self.pool.v,
                                      self.scale, self.out[:T], ws)
        self.timer.stop()
        return self.timer.elapsed_ms()


def linear_latency_model(a_ms: float = 0.02, per_prefill_token_ms: float = 2e-5,
                         per_decoder_ms: float = 5e-4) -> Executor:
    """Deterministic stand-in for the device: L = a + b p_t + c |D_t| (Eq. 1)."""
    def execute(q_len, kv_len, bt):
        p = int(np.sum(q_len[q_len > 1]))
        d = int(np.sum(q_len == 1))
        return a_ms + per_prefill_token_ms * p + per_decoder_ms * d
    return execute
