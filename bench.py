#!/usr/bin/env python3
"""Mixed-iteration benchmark of the DLFP hot path on one MI355X.

Headline workload (Qwen3-32B attention shapes on one GPU: 64 query heads, 8
KV heads, head_dim 128, bf16, 16-token pages, one layer at a time): 256
decoders with contexts U[2048, 32768] beside one 32768-token prompt
prefilled in chunks of p_t in {512, 1024, 2048, 4096, 8192}.  One timed step
runs the whole sweep, 124 chunk iterations: for every p_t the prompt is
prefilled in 32768 / p_t mixed iterations while each decoder advances one
token per iteration.  Each iteration is the full hot path -- host metadata
build and upload, the KV append and the attention (one launch,
dlfp_append_attention_mixed; --two-launch times dlfp_kv_append followed by
dlfp_attention_mixed), then the completion-timed controller step on the
iteration's measured device latency.  The one 18 GB layer pool is far larger
than the 256 MB Infinity Cache, so every launch reads its keys and values
from HBM.

Inputs are seeded synthetic N(0,1) bf16 tensors already resident in HBM.
Every attention launch of the timed steps is bracketed with HIP events on the
stream it runs on, which gives the per-launch durations behind the roofline
figures.  Also reported in the same run: latency vs p_t, decode-only and
prefill-only shares of the same kernel against the HBM and bf16 MFMA peaks,
the Qwen3-0.6B sweep (28 layers, 28 pools) and the full Qwen3-8B sweep as
other shapes, the closed-loop replay, and the CPU oracle's time on a bounded
sample.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
METRIC = "mixed-iteration latency vs prefill chunk; decode HBM GB/s %peak; prefill MFMA %"


def parse_args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--configs", default="qwen3-0.6b,qwen3-8b",
                    help="other shapes swept after the headline (comma list, or 'none')")
    ap.add_argument("--other-steps", type=int, default=3,
                    help="timed sweeps of each other shape")
    ap.add_argument("--headline-only", action="store_true",
                    help="only the headline sweep and its shares (for profiler runs)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--replay-seeds", default="801,802,803",
                    help="seeds of the closed-loop replay (comma list, or 'none')")
    ap.add_argument("--variant-requests", type=int, default=24,
                    help="requests per workload-variant replay")
    ap.add_argument("--tuning", default=None,
                    help="work-list policy overrides for every sweep (the dlfp_tuning fields, "
                         "comma-separated; 0 = automatic)")
    ap.add_argument("--quiet", action="store_true")
    ap.add_argument("--two-launch", action="store_true",
                    help="append with dlfp_kv_append, then dlfp_attention_mixed (instead of "
                         "the one-launch dlfp_append_attention_mixed)")
    ap.add_argument("--pmc-workload", choices=["sweep-32b", "sweep-0.6b", "shares-8b",
                                               "shares-32b"], default=None,
                    help="counter-pass workloads (see pmc_workload)")
    ap.add_argument("--plot", default=None,
                    help="also write a figure of latency vs p_t for every shape of the run "
                         "to this path (PNG)")
    ap.add_argument("--plot-from", default=None,
                    help="draw the --plot figure from the last JSON line of this file and exit "
                         "(no GPU needed)")
    return ap.parse_args()


def log(args, *a):
    if not args.quiet:
        print(*a, file=sys.stderr, flush=True)


# ----------------------------------------------------------------------------- work accounting

def attn_work(hq, hkv, q_len, kv_len):
    """Algorithmic bytes and flops of one attention launch (one layer).

    Per sequence: every K/V row of the keys it sees once (4096 B per token at
    Hkv=8, d=128, bf16), its queries read and outputs written once (bf16), and
    4 d Hq flops per visible (query, key) pair.
    """
    kv_tok = hkv * 128 * 2 * 2
    dec_b = pre_b = 0
    dec_f = pre_f = 0
    for q, n in zip(q_len, kv_len):
        q, n = int(q), int(n)
        io = q * hq * 128 * 2 * 2
        if q == 1:
            dec_b += n * kv_tok + io
            dec_f += 4 * 128 * hq * n
        else:
            P = n - q
            pre_b += n * kv_tok + io
            pre_f += 4 * 128 * hq * (q * P + q * (q + 1) // 2)
    return dec_b, pre_b, dec_f, pre_f


def append_work(hkv, num_tokens):
    """Algorithmic bytes of the KV append of one layer: every new token's key and
    value rows read once and written once into their pages (1024 B per token and
    KV head at d=128, bf16)."""
    return num_tokens * hkv * 128 * 2 * 2 * 2


# ----------------------------------------------------------------------------- sweep harness

class Sweep:
    def __init__(self, cfg, dev, n_pools, layers, seed_offset=0, fused=True, tuning=None):
        import torch
        from paper_2609_38386_amd import dlfp as D
        from paper_2609_38386_amd import runtime as rt
        from paper_2609_38386_amd import workload as wl
        self.torch, self.D, self.rt, self.wl = torch, D, rt, wl
        self.cfg = cfg
        self.dev = dev
        self.layers = layers
        self.fused = fused
        sh = cfg.shape
        self.hq, self.hkv = sh.num_q_heads, sh.num_kv_heads
        self.dims = D.make_dims(self.hq, self.hkv)
        self.n = cfg.n_decoders
        self.ctx = cfg.decoder_contexts().astype(np.int64)
        pages = cfg.pages_per_seq()
        self.num_blocks = int(sum(pages))
        bt = wl.block_tables(cfg.seed, pages, self.num_blocks)
        # batch order: the prompt slice first, then the decoders
        self.bt = np.ascontiguousarray(bt[[self.n] + list(range(self.n))])
        self.bt_dec = np.ascontiguousarray(bt[:self.n])
        self.d_bt = torch.from_numpy(self.bt).to(dev)
        self.d_bt_dec = torch.from_numpy(self.bt_dec).to(dev)
        gen = torch.Generator(device=dev)
        gen.manual_seed(cfg.seed + seed_offset)
        self.pools = []
        for _ in range(n_pools):
            p = rt.KVPool(self.num_blocks, self.hkv, dev)
            p.k.normal_(generator=gen)
            p.v.normal_(generator=gen)
            self.pools.append(p)
        # per chunk size: packed new rows of every chunk iteration, [prompt chunk ; decoders]
        self.inputs = {}
        for p in cfg.chunks:
            iters = cfg.prompt_len // p
            rows = iters * (p + self.n)
            q = torch.empty((rows, self.hq, 128), dtype=torch.bfloat16, device=dev)
            k = torch.empty((rows, self.hkv, 128), dtype=torch.bfloat16, device=dev)
            v = torch.empty((rows, self.hkv, 128), dtype=torch.bfloat16, device=dev)
            for t in (q, k, v):
                t.normal_(generator=gen)
            self.inputs[p] = (q, k, v)
        max_tok = max(cfg.chunks) + self.n
        self.out = torch.empty((max_tok, self.hq, 128), dtype=torch.bfloat16, device=dev)
        # two staging slots: the next iteration's metadata is built while one runs
        self.stages = [rt.StagedBatch(self.dims, self.n + 1, max_tok, 1 << 17, dev, tuning)
                       for _ in range(2)]
        self.stage = self.stages[0]
        self.ws = rt.Workspace(dev, 64 << 20)
        self.timer = D.Timer()
        # two sets of per-layer launch events, so that one iteration's can be read
        # while the next iteration runs
        self.ev_sets = [[(torch.cuda.Event(enable_timing=True),
                          torch.cuda.Event(enable_timing=True)) for _ in range(layers)]
                        for _ in range(2)]
        self.stream = torch.cuda.current_stream()
        self.scale = 1.0 / math.sqrt(128)
        self.L = D.lib()
        import ctypes
        self.ct = ctypes
        self.dims_ref = ctypes.byref(self.dims)
        self.stream_handle = ctypes.c_void_p(int(self.stream.cuda_stream))
        self.c_scale = ctypes.c_float(self.scale)
        self.pool_ptrs = [(ctypes.c_void_p(pl.k.data_ptr()), ctypes.c_void_p(pl.v.data_ptr()))
                          for pl in self.pools]

    def prepare(self, p, c, decoders=True, prefill=True, slot=0):
        """Host side of one mixed iteration: its metadata, built into staging slot
        `slot` and copied to the device on the stream (ordered after whatever was
        enqueued before, so it can be built while the previous iteration runs)."""
        torch = self.torch
        q_len, kv_len, rows = [], [], []
        if prefill:
            q_len.append(p)
            kv_len.append((c + 1) * p)
            rows.append(0)
        if decoders:
            q_len += [1] * self.n
            kv_len += [int(x) + c for x in self.ctx]
            rows += list(range(1, self.n + 1))
        q_len = np.asarray(q_len, dtype=np.int32)
        kv_len = np.asarray(kv_len, dtype=np.int32)
        bt = self.bt if (prefill and decoders) else np.ascontiguousarray(self.bt[rows])
        d_bt = self.d_bt if (prefill and decoders) else torch.from_numpy(bt).to(self.dev)
        st = self.stages[slot].build(q_len, kv_len, bt, self.num_blocks)
        T = st.num_tokens
        qa, ka, va = self.inputs[p]
        base = c * (p + self.n)
        lo = base if prefill else base + p
        return {"q_len": q_len, "kv_len": kv_len, "bt": bt, "d_bt": d_bt, "st": st, "T": T,
                "qkv": (qa[lo:lo + T], ka[lo:lo + T], va[lo:lo + T]),
                "guarded": bool(prefill and decoders), "decoders": decoders}

    def launch(self, pr, record=True, evset=0):
        """Enqueue the layers of a prepared iteration between the completion timer's
        events; with `record`, HIP events (of set `evset`) also bracket every
        attention launch (the one-launch append + attention, or the attention alone
        with two launches)."""
        D = self.D
        st, T, bt, d_bt = pr["st"], pr["T"], pr["bt"], pr["d_bt"]
        q, k, v = pr["qkv"]
        meta = st.meta
        ws = self.ws.ensure(meta.workspace_bytes)
        ct, vp = self.ct, self.ct.c_void_p
        dims_ref, stream = self.dims_ref, self.stream_handle
        app_args = (dims_ref, T, vp(k.data_ptr()), vp(v.data_ptr()), vp(st.d_slots.data_ptr()))
        att_head = (dims_ref, ct.byref(meta.c), vp(st.d_work.data_ptr()), vp(d_bt.data_ptr()),
                    int(bt.shape[1]),
                    self.num_blocks, vp(q.data_ptr()))
        att_tail = (self.c_scale, vp(self.out.data_ptr()), 0, vp(ws.data_ptr()),
                    ct.c_size_t(ws.numel()), stream)
        kv_new = (vp(k.data_ptr()), vp(v.data_ptr()))
        L = self.L
        ev = self.ev_sets[evset]
        self.timer.start(self.stream)
        for layer in range(self.layers):
            pk, pv = self.pool_ptrs[layer % len(self.pools)]
            if self.fused:
                if record:
                    ev[layer][0].record(self.stream)
                rc = L.dlfp_append_attention_mixed(*att_head, *kv_new, pk, pv, *att_tail)
                if rc:
                    D._check(rc, "dlfp_append_attention_mixed")
            else:
                rc = L.dlfp_kv_append(*app_args, pk, pv, self.num_blocks, stream)
                if rc:
                    D._check(rc, "dlfp_kv_append")
                if record:
                    ev[layer][0].record(self.stream)
                rc = L.dlfp_attention_mixed(*att_head, pk, pv, *att_tail)
                if rc:
                    D._check(rc, "dlfp_attention_mixed")
            if record:
                ev[layer][1].record(self.stream)
        self.timer.stop(self.stream)
        pr["record"] = record
        pr["evset"] = evset

    def finish(self, pr, ctrl=None, events=True):
        """Wait for the iteration (completion timing), step the controller from the
        measured latency; returns (device ms, [attention ms per layer], q_len, kv_len).
        With `events` False the per-launch events are left to `attention_ms`."""
        ms = self.timer.elapsed_ms()
        if ctrl is not None:
            self.D.dlfp_controller_step(ctrl, self.n if pr["decoders"] else 0, pr["guarded"], ms)
        attn = self.attention_ms(pr) if events else None
        return ms, attn, pr["q_len"], pr["kv_len"]

    def attention_ms(self, pr):
        """Per-layer launch times of a finished iteration (valid until its event set
        is recorded again, two launches later)."""
        if not pr["record"]:
            return []
        return [a.elapsed_time(b) for a, b in self.ev_sets[pr["evset"]]]

    def iteration(self, p, c, ctrl=None, decoders=True, prefill=True, record=True):
        """Prepare, launch and finish one mixed iteration."""
        pr = self.prepare(p, c, decoders, prefill)
        self.launch(pr, record)
        return self.finish(pr, ctrl)

    def chunks(self, p, policy):
        iters = self.cfg.prompt_len // p
        if policy == "all":
            return list(range(iters))
        return sorted({0, iters // 2, iters - 1})


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "attention_mixed_qwen3-32b_sweep_hbm_traffic.md")
# Sources whose change can change the HBM traffic of a launch: the kernel, the
# work-list policy that shapes it, and the headers they share.
KERNEL_SOURCES = ("paper_2609_38386_amd/csrc/attention_mixed.hip",
                  "paper_2609_38386_amd/csrc/dlfp_host.cpp", "include/dlfp.h",
                  "paper_2609_38386_amd/csrc/dlfp_internal.h")


def source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def profiled_traffic():
    """HBM bytes per attention launch of the headline sweep from the committed
    FETCH_SIZE / WRITE_SIZE summary (calibrated against a device copy), or None
    when the kernel or work-list sources have changed since the counters were
    taken."""
    try:
        text = open(TRAFFIC_PROFILE).read()
        digest = source_hash()
    except OSError:
        return None
    fields = dict(line.split(": ", 1) for line in text.splitlines()
                  if line.startswith(("traffic_bytes_per_launch: ", "source_sha256: ")))
    if fields.get("source_sha256", "").strip() != digest:
        return None
    return int(fields["traffic_bytes_per_launch"])


def record_all(cfg, p, c):
    """Every launch is bracketed by HIP events (a launch lasts milliseconds)."""
    return True


def record_quarter(cfg, p, c):
    """Every fourth chunk iteration of each chunk size (chunks 3, 7, 11, ...): a
    quarter of the sweep in its own mix of chunk sizes.  Each event pair adds a
    dispatch gap of several microseconds, which matters for launches of tens of
    microseconds."""
    return c % 4 == 3


def run_sweep(cfg, dev, log_fn, n_pools, layers, steps, warmup, record, fused=True,
              tuning=None):
    """Time `steps` full chunk-size sweeps of `cfg` after `warmup` untimed ones.

    Per iteration: metadata of the next iteration built on the host while the
    current one runs, `layers` launches (one per layer, rotating over `n_pools`
    distinct pools), then the controller stepped from the iteration's completion
    time.  Returns wall time, tokens, per-p_t statistics and the roofline figures
    of the launches `record` selects."""
    import torch
    from paper_2609_38386_amd import dlfp as D
    t0 = time.time()
    sw = Sweep(cfg, dev, n_pools=n_pools, layers=layers, fused=fused, tuning=tuning)
    log_fn(f"{cfg.name}: setup {time.time() - t0:.1f}s: {n_pools} pools x {sw.num_blocks} blocks")
    # decode-only latency of the first iteration sets the controller target (1.2x)
    dec_ms = [sw.iteration(cfg.chunks[0], 0, prefill=False, record=False)[0] for _ in range(3)]
    target = 1.2 * float(np.median(dec_ms))
    ctrl = D.dlfp_controller_init(target, 2048, 32, max(4096, max(cfg.chunks)), 128)
    iters = [(p, c) for p in cfg.chunks for c in range(cfg.prompt_len // p)]

    def account(stats, p, c, pr, ms, cap):
        """The benchmark's own bookkeeping of a finished iteration (run while the
        next iteration is on the device)."""
        ql, kl = pr["q_len"], pr["kv_len"]
        s = stats.setdefault(p, {"iter_ms": [], "attn_ms": 0.0, "attn_launch_ms": [],
                                 "bytes": 0, "flops": 0, "tokens": 0, "caps": [],
                                 "recorded": 0, "by_chunk": {}})
        s["iter_ms"].append(ms)
        s["by_chunk"].setdefault(c, []).append(ms)
        s["tokens"] += int(ql.sum())
        s["caps"].append(cap)
        if pr["record"]:
            attn = sw.attention_ms(pr)
            s["recorded"] += 1
            s["attn_ms"] += sum(attn)
            s["attn_launch_ms"] += list(attn)
            db, pb, df, pf = attn_work(sw.hq, sw.hkv, ql, kl)
            ab = append_work(sw.hkv, int(ql.sum())) if sw.fused else 0
            s["bytes"] += (db + pb + ab) * layers
            s["flops"] += (df + pf) * layers

    def step(stats):
        # Per iteration: launch, account for the previous iteration while this one
        # runs, build the next iteration's metadata, then wait for completion and
        # step the controller (Eq. 2) before the next launch.
        pr = sw.prepare(*iters[0], slot=0)
        pending = None
        for i, (p, c) in enumerate(iters):
            sw.launch(pr, record=record(cfg, p, c), evset=i & 1)
            if pending is not None and stats is not None:
                account(stats, *pending)
            nxt = sw.prepare(*iters[i + 1], slot=(i + 1) & 1) if i + 1 < len(iters) else None
            ms = sw.finish(pr, ctrl, events=False)[0]
            pending = (p, c, pr, ms, ctrl.cap)
            pr = nxt
        if pending is not None and stats is not None:
            account(stats, *pending)

    for _ in range(warmup):
        step(None)
    torch.cuda.synchronize()
    stats = {}
    t_start = time.perf_counter()
    for _ in range(steps):
        step(stats)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ws_error = D.dlfp_workspace_error(sw.ws.buf)
    tokens = sum(s["tokens"] for s in stats.values())
    attn_ms = sum(s["attn_ms"] for s in stats.values())
    n_launch = sum(s["recorded"] for s in stats.values()) * layers
    bytes_all = sum(s["bytes"] for s in stats.values())
    flops_all = sum(s["flops"] for s in stats.values())
    latency = {}
    lb_all = 0.0
    for p, s in stats.items():
        it = np.asarray(s["iter_ms"])
        n_l = s["recorded"] * layers
        per_launch_ms = s["attn_ms"] / n_l
        # whole-launch bounds from the algorithmic work of one call: ideal overlap of
        # the HBM and MFMA shares (t_lb) and the two run back to back (t_sum)
        t_b = s["bytes"] / n_l / (HBM_PEAK_GBS * 1e9)
        t_f = s["flops"] / n_l / (MFMA_BF16_PEAK_TFLOPS * 1e12)
        lb_all += max(t_b, t_f) * n_l
        chunks = sorted(s["by_chunk"])
        fml = sorted({chunks[0], chunks[len(chunks) // 2], chunks[-1]})
        latency[str(p)] = {
            "iter_ms_mean": round(float(it.mean()), 4),
            "iter_ms_p50": round(float(np.median(it)), 4),
            "iter_ms_p90": round(float(np.percentile(it, 90)), 4),
            "iter_ms_first_mid_last": [round(float(np.median(s["by_chunk"][c])), 4) for c in fml],
            "attn_us_per_layer": round(per_launch_ms * 1e3, 2),
            "attn_GBps": round(s["bytes"] / (s["attn_ms"] * 1e-3) / 1e9, 1),
            "attn_TFLOPs": round(s["flops"] / (s["attn_ms"] * 1e-3) / 1e12, 1),
            "ttft_proxy_ms": round(float(it.sum()) / steps, 3),
            "iterations": len(it) // steps,
            "iterations_with_launch_events": s["recorded"] // steps,
            "controller_cap_last": s["caps"][-1],
            "t_lb_us": round(max(t_b, t_f) * 1e6, 2), "t_sum_us": round((t_b + t_f) * 1e6, 2),
            "t_lb_over_measured": round(max(t_b, t_f) / (per_launch_ms * 1e-3), 4),
        }
    avg_launch_s = attn_ms * 1e-3 / n_launch
    ach = (bytes_all / n_launch) / avg_launch_s / 1e9
    g = sw.hq // sw.hkv
    roofline = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": None,
                "kernel": (f"attention_mixed_kernel<{g}, true, true> (append + attention)"
                           if sw.fused else f"attention_mixed_kernel<{g}, false, true>"),
                "launches_timed": n_launch,
                "avg_launch_us": round(avg_launch_s * 1e6, 2),
                "algorithmic_bytes_per_launch": int(bytes_all / n_launch),
                "algorithmic_tflops": round(flops_all / (attn_ms * 1e-3) / 1e12, 1),
                "t_lb_over_measured": round(lb_all / (attn_ms * 1e-3), 4)}
    shares = measure_shares(sw, cfg)
    result = {"wall": wall, "tokens": tokens, "latency": latency, "roofline": roofline,
              "shares": shares, "target_ms": target, "decode_only_iter_ms": float(np.median(dec_ms)),
              "workspace_error": ws_error, "steps": steps, "warmup": warmup}
    del sw
    torch.cuda.empty_cache()
    return result


def other_shape(name, cfg, r, layers, pools):
    """Summary of a sweep measured beside the headline."""
    return {"shape": f"Hq{cfg.shape.num_q_heads}/Hkv{cfg.shape.num_kv_heads}/d128",
            "decoders": cfg.n_decoders, "ctx": [cfg.ctx_lo, cfg.ctx_hi],
            "prompt_len": cfg.prompt_len, "chunks": list(cfg.chunks),
            "model_layers": cfg.layers, "layers_per_iteration_timed": layers,
            "distinct_layer_pools": pools, "steps": r["steps"],
            "tokens_per_s": round(r["tokens"] / r["wall"], 1),
            "ms_per_sweep": round(r["wall"] * 1e3 / r["steps"], 3),
            "roofline": r["roofline"], "latency_vs_pt": r["latency"], "shares": r["shares"],
            "decode_only_iter_ms": round(r["decode_only_iter_ms"], 4),
            "workspace_error": r["workspace_error"]}


def shares_against_ceilings(shares, ceilings):
    """Add to a shares record the fraction of the measured ceilings: the decode
    share's rate over the random 8 KiB HBM ceiling, each prefill share's over the
    bf16 MFMA ceiling (the matrix cores at the clock they hold under sustained
    load, against which the 2.5 PFLOP/s rating is not reachable)."""
    if not ceilings:
        return shares
    shares["decode"]["frac_of_measured_hbm_ceiling"] = round(
        shares["decode"]["GBps"] / ceilings["hbm_random_8KiB_GBps"], 4)
    for v in shares["prefill_last_chunk"].values():
        v["frac_of_measured_mfma_ceiling"] = round(v["TFLOPs"] / ceilings["mfma_bf16_TFLOPs"], 4)
    return shares


def measure_shares(sw, cfg, min_launches=20):
    """Decode-only and prefill-only launches of the same kernel (rotating pools),
    at least ``min_launches`` of each, each timed with its own events.  Rates are
    the median over launches of algorithmic work / launch time; the 90th
    percentile of the launch time is reported beside the median."""
    reps = max(1, -(-min_launches // sw.layers))

    def summary(times_ms, work):
        t = np.asarray(times_ms)
        rate = np.asarray(work) / (t * 1e-3)
        return t, float(np.median(rate))

    out = {}
    times, work = [], []
    for r in range(reps):
        _, a, ql, kl = sw.iteration(cfg.chunks[0], r, prefill=False)
        db, _, _, _ = attn_work(sw.hq, sw.hkv, ql, kl)
        db += append_work(sw.hkv, int(ql.sum())) if sw.fused else 0
        times += list(a)
        work += [db] * len(a)
    t, rate = summary(times, work)
    gbs = rate / 1e9
    out["decode"] = {"GBps": round(gbs, 1), "frac_hbm": round(gbs / HBM_PEAK_GBS, 4),
                     "us_per_layer": round(float(np.median(t)) * 1e3, 2),
                     "us_p90": round(float(np.percentile(t, 90)) * 1e3, 2),
                     "launches": len(t), "bytes_per_layer": int(np.median(work))}
    pre = {}
    for p in cfg.chunks:
        c = cfg.prompt_len // p - 1
        times, fl, by = [], [], []
        for r in range(reps):
            _, a, ql, kl = sw.iteration(p, c, decoders=False)
            _, pb, _, pf = attn_work(sw.hq, sw.hkv, ql, kl)
            pb += append_work(sw.hkv, int(ql.sum())) if sw.fused else 0
            times += list(a)
            fl += [pf] * len(a)
            by += [pb] * len(a)
        t, tf = summary(times, fl)
        _, bs = summary(times, by)
        tf /= 1e12
        g = sw.hq // sw.hkv
        pre[str(p)] = {"TFLOPs": round(tf, 1), "frac_mfma": round(tf / MFMA_BF16_PEAK_TFLOPS, 4),
                       "GBps": round(bs / 1e9, 1),
                       "frac_hbm": round(bs / 1e9 / HBM_PEAK_GBS, 4),
                       "above_ridge": bool(g * p >= 315),
                       "us_per_layer": round(float(np.median(t)) * 1e3, 2),
                       "us_p90": round(float(np.percentile(t, 90)) * 1e3, 2),
                       "launches": len(t)}
    out["prefill_last_chunk"] = pre
    return out


# ----------------------------------------------------------------------------- replay

def run_replays(dev, seeds, log_fn):
    """Closed-loop replay (100 Poisson arrivals at 2 req/s, prompts U[256,4096],
    128 output tokens, one layer timed, clock x28), paired per seed: the uncapped
    baseline, fixed caps of 2048 / 3072 / 4096 tokens, and DLFP with the target at
    1.2x the median decode-only iteration latency of the seed's baseline run.
    Reductions of the P99 inter-token latency against the baseline get a paired
    Student-t interval over the seeds."""
    from paper_2609_38386_amd import replay as rp
    keys = ("itl_p50_ms", "itl_p99_ms", "ttft_p50_ms", "ttft_p99_ms", "e2e_p99_ms",
            "iterations", "guarded_iterations", "guarded_L_over_T_mean", "controlled_iterations",
            "controlled_L_over_T_mean", "controlled_within_target", "reconciled")
    policies = ["fixed_2048", "fixed_3072", "fixed_4096", "dlfp"]
    out = {"per_seed": {}}
    reductions = {k: [] for k in policies}
    for seed in seeds:
        cfg = rp.ReplayConfig(seed=seed)
        ex = rp.GpuExecutor(cfg, dev)
        trace = []
        t0 = time.time()
        runs = {"uncapped": rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), ex, trace=trace)}
        dec = [it["layer_ms"] for it in trace if it["decoders"] > 0 and it["p_t"] == 0]
        target = 1.2 * float(np.median(dec))
        for cap in (2048, 3072, 4096):
            runs[f"fixed_{cap}"] = rp.run_replay(cfg, rp.Policy(rp.Policy.FIXED, cap=cap), ex)
        runs["dlfp"] = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP, target_ms=target, cfg=cfg), ex)
        base = runs["uncapped"]
        rec = {"target_layer_ms": round(target, 5)}
        for name, r in runs.items():
            rec[name] = {k: (round(r[k], 4) if isinstance(r[k], float) else r[k]) for k in keys}
            if name in reductions:
                red = 100.0 * (base["itl_p99_ms"] - r["itl_p99_ms"]) / base["itl_p99_ms"]
                rec[name]["p99_itl_reduction_pct"] = round(red, 2)
                reductions[name].append(red)
        rec["retimed_iterations"] = ex.retimed
        out["per_seed"][str(seed)] = rec
        log_fn(f"replay seed {seed}: {time.time() - t0:.1f}s, p99 ITL uncapped "
               f"{base['itl_p99_ms']:.3f} ms, dlfp {runs['dlfp']['itl_p99_ms']:.3f} ms, "
               f"guarded {runs['dlfp']['guarded_iterations']}")
        del ex
    out["p99_itl_reduction_vs_uncapped"] = {}
    for name, reds in reductions.items():
        mean, lo, hi = rp.paired_ci(reds)
        out["p99_itl_reduction_vs_uncapped"][name] = {
            "mean_pct": round(mean, 2),
            "ci95_pct": None if lo is None else [round(lo, 2), round(hi, 2)]}
    out["note"] = ("latencies are x28 one-layer device times (attention only); at 2 req/s "
                   "requests rarely overlap, so few iterations are guarded")
    return out


def run_overlap_replay(dev, seed, rate, log_fn):
    """The same replay at a higher arrival rate, so that prompts arrive while
    others decode for most of the run: the controller's steady state (L/T on the
    guarded cycles whose cap came from a feedback update), uncapped vs DLFP, and
    DLFP fed each completion time one iteration late (what an asynchronous
    engine that sets the next cap while the current iteration runs observes)."""
    from paper_2609_38386_amd import replay as rp
    keys = ("itl_p50_ms", "itl_p99_ms", "ttft_p50_ms", "ttft_p99_ms", "iterations",
            "guarded_iterations", "controlled_iterations", "controlled_L_over_T_mean",
            "controlled_L_over_T_p50", "controlled_L_over_T_p90", "controlled_within_target",
            "controlled_within_5pct", "reconciled")
    cfg = rp.ReplayConfig(seed=seed, rate_per_s=rate)
    ex = rp.GpuExecutor(cfg, dev)
    trace = []
    t0 = time.time()
    base = rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), ex, trace=trace)
    target = 1.2 * float(np.median([it["layer_ms"] for it in trace
                                    if it["decoders"] > 0 and it["p_t"] == 0]))
    trace = []
    dl = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP, target_ms=target, cfg=cfg), ex, trace=trace)
    caps = [it["limit"] for it in trace if it["guarded"]]
    lag = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP_LAG1, target_ms=target, cfg=cfg), ex)
    out = {"seed": seed, "rate_per_s": rate, "target_layer_ms": round(target, 5),
           "guarded_cap_p50": int(np.median(caps)) if caps else None,
           "guarded_cycles_at_c_min": (round(float(np.mean(np.asarray(caps) == cfg.c_min)), 4)
                                       if caps else None)}
    for name, r in (("uncapped", base), ("dlfp", dl), ("dlfp_lag1", lag)):
        out[name] = {k: (round(r[k], 4) if isinstance(r[k], float) else r[k]) for k in keys}
    out["retimed_iterations"] = ex.retimed
    log_fn(f"overlap replay {rate} req/s: {time.time() - t0:.1f}s, controlled L/T p50 "
           f"{dl['controlled_L_over_T_p50']}, within 5% {dl['controlled_within_5pct']}")
    del ex
    return out


def run_root_cause_replays(dev, seed, rates, log_fn):
    """The paper's failure mode (Sec. 3.2, Sec. 6.3, Sec. 6.4) on the device: the
    replay with an engine pipeline whose scheduler calls cost the host time
    measured for them.  Asynchronous scheduling (the scheduler one iteration
    ahead): uncapped, Eq. 2 on the completion time as it becomes available (one
    iteration late) and Eq. 2 on the interval between scheduler calls.
    Synchronous scheduling: uncapped, Eq. 2 on the completion time, and the
    completion-aware revision (host time from the call to the returned output,
    each step bounded to a factor of two).  Reported with how far each signal was
    from the guarded cycle's device time and how often it moved the cap the
    wrong way."""
    from paper_2609_38386_amd import replay as rp
    keys = ("itl_p50_ms", "itl_p99_ms", "ttft_p50_ms", "ttft_p99_ms", "iterations",
            "guarded_iterations", "controlled_iterations", "controlled_L_over_T_p50",
            "controlled_L_over_T_p90", "controlled_within_5pct", "signal_rel_error_mean",
            "wrong_direction_updates", "reconciled")
    out = {}
    for rate in rates:
        for pipe, kinds in (("async", (rp.Policy.DLFP_LAG1, rp.Policy.DLFP_CADENCE)),
                            ("sync", (rp.Policy.DLFP, rp.Policy.DLFP_REVISED))):
            cfg = rp.ReplayConfig(seed=seed, rate_per_s=rate, pipeline=pipe)
            ex = rp.GpuExecutor(cfg, dev)
            t0 = time.time()
            trace = []
            runs = {"uncapped": rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), ex, trace=trace)}
            target = 1.2 * float(np.median([it["layer_ms"] for it in trace
                                            if it["decoders"] > 0 and it["p_t"] == 0]))
            for k in kinds:
                runs[k] = rp.run_replay(cfg, rp.Policy(k, target_ms=target, cfg=cfg), ex)
            rec = {"target_layer_ms": round(target, 5)}
            for name, r in runs.items():
                rec[name] = {k: (round(r[k], 4) if isinstance(r[k], float) else r[k])
                             for k in keys}
            rec["retimed_iterations"] = ex.retimed
            out[f"{pipe}_{rate:g}_req_s"] = rec
            log_fn(f"root-cause replay {pipe} {rate} req/s: {time.time() - t0:.1f}s, p99 ITL "
                   + ", ".join(f"{n} {r['itl_p99_ms']:.3f}" for n, r in runs.items()))
            del ex
    out["note"] = ("clock = device completion times of a pipeline whose scheduler calls cost the "
                   "host time measured for them; signals per layer (x28 layers)")
    return out


REPLAY_KEYS = ("itl_p50_ms", "itl_p99_ms", "ttft_p50_ms", "ttft_p99_ms", "e2e_p99_ms",
               "iterations", "guarded_iterations", "controlled_iterations",
               "controlled_L_over_T_p50", "controlled_L_over_T_p90", "controlled_within_target",
               "controlled_within_5pct", "reconciled")


def paired_replay(cfg, dev, log_fn, label):
    """Uncapped, then DLFP with the target at 1.2x the uncapped run's median
    decode-only latency; the guarded caps' distribution and the P99 ITL change."""
    from paper_2609_38386_amd import replay as rp
    ex = rp.GpuExecutor(cfg, dev)
    t0 = time.time()
    trace = []
    base = rp.run_replay(cfg, rp.Policy(rp.Policy.UNCAPPED), ex, trace=trace)
    dec = [it["layer_ms"] for it in trace if it["decoders"] > 0 and it["p_t"] == 0]
    target = 1.2 * float(np.median(dec))
    chunk_ms = [(it["p_t"], it["layer_ms"]) for it in trace if it["p_t"] > 0]
    trace = []
    dl = rp.run_replay(cfg, rp.Policy(rp.Policy.DLFP, target_ms=target, cfg=cfg), ex, trace=trace)
    caps = np.asarray([it["limit"] for it in trace if it["guarded"]])
    rec = {"target_layer_ms": round(target, 5),
           "decode_only_layer_ms_p50": round(float(np.median(dec)), 5)}
    if len({p for p, _ in chunk_ms}) >= 2:
        pt, ms = np.asarray(chunk_ms, dtype=np.float64).T
        slope, icpt = np.polyfit(pt, ms, 1)
        rec["layer_ms_vs_p_t_fit"] = {"intercept_ms": round(float(icpt), 5),
                                      "ms_per_1k_tokens": round(float(slope) * 1e3, 5)}
    for name, r in (("uncapped", base), ("dlfp", dl)):
        rec[name] = {k: (round(r[k], 4) if isinstance(r[k], float) else r[k]) for k in REPLAY_KEYS}
    rec["p99_itl_reduction_pct"] = round(
        100.0 * (base["itl_p99_ms"] - dl["itl_p99_ms"]) / base["itl_p99_ms"], 2)
    if len(caps):
        rec["guarded_caps"] = {"p10": int(np.percentile(caps, 10)), "p50": int(np.median(caps)),
                               "p90": int(np.percentile(caps, 90)),
                               "at_c_min": round(float(np.mean(caps == cfg.c_min)), 4)}
    rec["retimed_iterations"] = ex.retimed
    log_fn(f"{label}: {time.time() - t0:.1f}s, p99 ITL {base['itl_p99_ms']:.3f} -> "
           f"{dl['itl_p99_ms']:.3f} ms, guarded {dl['guarded_iterations']}")
    del ex
    return rec


def run_layer_proxy_replays(dev, seeds, log_fn):
    """The replay of config 2 with the full-iteration proxy (Eq. 1's linear
    term): the layer's projections timed with the attention, so the iteration
    latency grows with p_t and Eq. 2 regulates instead of clamping at c_min.
    Paired per seed at 2 req/s, plus seed 801 at 20 req/s."""
    from paper_2609_38386_amd import replay as rp
    out = {"per_seed": {}}
    reds = []
    for seed in seeds:
        cfg = rp.ReplayConfig(seed=seed, layer_proxy=True)
        rec = paired_replay(cfg, dev, log_fn, f"layer proxy seed {seed}")
        out["per_seed"][str(seed)] = rec
        reds.append(rec["p99_itl_reduction_pct"])
    mean, lo, hi = rp.paired_ci(reds)
    out["p99_itl_reduction_vs_uncapped"] = {
        "mean_pct": round(mean, 2), "ci95_pct": None if lo is None else [round(lo, 2), round(hi, 2)]}
    out["overlap_20_req_s"] = paired_replay(rp.ReplayConfig(seed=seeds[0], rate_per_s=20.0,
                                                            layer_proxy=True),
                                            dev, log_fn, "layer proxy 20 req/s")
    out["note"] = ("per layer: Q, K, V projections (hidden 1024), append + attention, output "
                   "projection, MLP gate/up and down (3072), one layer timed, clock x28")
    return out


# The paper's workload shapes (Sec. 4.2): prompt / output tokens.
VARIANTS = {"chat": (1024, 128), "rag": (8192, 256), "agent": (16384, 256),
            "decode_heavy": (256, 1024)}


def run_variant_replays(dev, seed, rate, n_requests, log_fn):
    """Each of the paper's workload shapes as a replay with the layer proxy,
    open-loop Poisson arrivals at the paper's rate, paired uncapped vs DLFP with
    the paper's cap constants (c_initial 3072, c_min 1024, c_max 6144, Sec. 3.1)."""
    from paper_2609_38386_amd import replay as rp
    out = {}
    for name, (prompt, outl) in VARIANTS.items():
        cfg = rp.ReplayConfig(seed=seed, n_requests=n_requests, rate_per_s=rate,
                              prompt_lo=prompt, prompt_hi=prompt, out_len=outl,
                              layer_proxy=True, c_initial=3072, c_min=1024, c_max=6144)
        out[name] = paired_replay(cfg, dev, log_fn, f"variant {name}")
        out[name]["prompt_tokens"], out[name]["output_tokens"] = prompt, outl
    # The long-prompt shapes again with a lower cap floor: whether the paper's
    # floor (1024 tokens), which a chunk over a long prefix cannot meet the
    # target at, is what keeps Eq. 2 from cutting their tail latency.
    for name in ("rag", "agent"):
        prompt, outl = VARIANTS[name]
        cfg = rp.ReplayConfig(seed=seed, n_requests=n_requests, rate_per_s=rate,
                              prompt_lo=prompt, prompt_hi=prompt, out_len=outl,
                              layer_proxy=True, c_initial=3072, c_min=128, c_max=6144)
        key = f"{name}_c_min_128"
        out[key] = paired_replay(cfg, dev, log_fn, f"variant {key}")
        out[key]["prompt_tokens"], out[key]["output_tokens"] = prompt, outl
    out["note"] = (f"{n_requests} requests at {rate} req/s, seed {seed}, layer proxy, "
                   "one layer timed, clock x28, caps 1024..6144 from c_initial 3072 "
                   "(the *_c_min_128 entries: caps 128..6144)")
    return out


def measure_ceilings(dev, log_fn):
    """Achievable ceilings from libdlfp_probe.so, timed with HIP events (median of
    5 launches): HBM reads of random 8 KiB pieces (a decode page pair) and of a
    contiguous stream from a 4 GiB buffer, at 1, 2 or 4 pieces in flight per
    wavefront and 8 or 16 wavefronts per CU, with default caching and with
    non-temporal loads (as the decode share reads its pages); bf16 MFMA with 4
    accumulator chains per wavefront at 8 and 16 wavefronts per CU.  The HBM
    ceilings are the best over every configuration."""
    import ctypes
    import torch
    path = os.path.join(ROOT, "paper_2609_38386_amd", "libdlfp_probe.so")
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2609_38386_amd.build`")
    L = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    L.dlfp_probe_hbm_read.argtypes = [vp, i64, vp, i32, i32, i32, i32, i32, vp, vp]
    L.dlfp_probe_mfma.argtypes = [i32, i32, vp, vp]
    stream = torch.cuda.current_stream()
    sh = ctypes.c_void_p(int(stream.cuda_stream))
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def timed(fn, reps=5):
        fn()
        out = []
        for _ in range(reps):
            ev[0].record(stream)
            fn()
            ev[1].record(stream)
            ev[1].synchronize()
            out.append(ev[0].elapsed_time(ev[1]) * 1e-3)
        return float(np.median(out))

    piece, buf_bytes = 8192, 4 << 30
    buf = torch.empty(buf_bytes, dtype=torch.uint8, device=dev).fill_(7)
    n_pieces = buf_bytes // piece
    g = torch.Generator(device=dev)
    g.manual_seed(5)
    hbm = {}
    for waves_per_cu in (8, 16):
        waves = 256 * waves_per_cu
        per_wave = (1 << 30) // piece // waves           # 1 GiB per launch
        rand = torch.randint(0, n_pieces, (waves * per_wave,), generator=g, device=dev,
                             dtype=torch.int32)
        seq = torch.arange(waves * per_wave, device=dev, dtype=torch.int32)
        sink = torch.empty(waves * 64, dtype=torch.int32, device=dev)
        for name, idx in (("random", rand), ("stream", seq)):
            for nt in (0, 1):
                for inflight in (1, 2, 4):
                    assert per_wave % inflight == 0 and int(idx.max()) < n_pieces
                    t = timed(lambda: L.dlfp_probe_hbm_read(
                        vp(buf.data_ptr()), buf_bytes, vp(idx.data_ptr()), waves, per_wave,
                        piece, inflight, nt, vp(sink.data_ptr()), sh))
                    mode = "_nt" if nt else ""
                    hbm[f"{name}_8KiB{mode}_{waves_per_cu}w_{inflight}inflight"] = round(
                        waves * per_wave * piece / t / 1e9, 1)
    del buf
    mfma = {}
    iters = 4096
    for waves_per_cu in (8, 16):
        wgs = 256 * waves_per_cu // 4
        sink = torch.empty(wgs * 256, dtype=torch.float32, device=dev)
        t = timed(lambda: L.dlfp_probe_mfma(wgs, iters, vp(sink.data_ptr()), sh))
        mfma[f"{waves_per_cu}w"] = round(wgs * 4 * iters * 4 * 32768 / t / 1e12, 1)
    torch.cuda.synchronize()
    best_rand = max(v for k, v in hbm.items() if k.startswith("random"))
    best_rand_cached = max(v for k, v in hbm.items() if k.startswith("random_8KiB_")
                           and "_nt_" not in k)
    best_stream = max(v for k, v in hbm.items() if k.startswith("stream"))
    log_fn(f"ceilings: HBM random 8 KiB {best_rand} GB/s ({best_rand_cached} with default "
           f"caching), stream {best_stream} GB/s, MFMA bf16 {max(mfma.values())} TFLOP/s")
    return {"hbm_random_8KiB_GBps": best_rand,
            "hbm_random_8KiB_default_caching_GBps": best_rand_cached,
            "hbm_stream_GBps": best_stream,
            "mfma_bf16_TFLOPs": max(mfma.values()), "hbm_GBps_by_config": hbm,
            "mfma_TFLOPs_by_waves_per_cu": mfma,
            "note": "libdlfp_probe.so, HIP events, median of 5 launches of 1 GiB (HBM)"}


# ----------------------------------------------------------------------------- CPU baseline

def cpu_baseline(dev, seconds, p=512, c=32):
    """The float64 oracle on a bounded sample of the headline workload: iteration
    (p_t, chunk c) of the Qwen3-32B sweep -- the prompt chunk, then decoders one at
    a time until `seconds` have passed -- from the paged bf16 pool to the outputs
    (the oracle's page gather, exact widening to float64, masked softmax
    attention).  The pool pages of the sampled sequences are drawn on the device
    and copied to the host before the clock starts.  The per-iteration time is the
    prompt's plus the mean decoder's times the 256 decoders."""
    import torch
    from oracle import attention as oa
    from oracle import paging as op
    from paper_2609_38386_amd import runtime as rt
    from paper_2609_38386_amd import workload as wl
    cfg = wl.qwen3_32b_config()
    hq, hkv = cfg.shape.num_q_heads, cfg.shape.num_kv_heads
    ctx = cfg.decoder_contexts()
    its = cfg.iteration(p, c)                  # prompt first, then the decoders
    n_sample = min(len(its), 65)               # prompt + up to 64 decoders staged
    pages = [wl.pages_for(kl) for _, _, kl in its[:n_sample]]
    nb = int(sum(pages))
    bt = wl.block_tables(cfg.seed, pages, nb)
    pool = rt.KVPool(nb, hkv, dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfg.seed + 7)
    pool.k.normal_(generator=gen)
    pool.v.normal_(generator=gen)
    q = torch.empty((p + n_sample - 1, hq, 128), dtype=torch.bfloat16, device=dev)
    q.normal_(generator=gen)
    k_host, v_host = pool.k.view(torch.int16).cpu(), pool.v.view(torch.int16).cpu()
    q_host = q.view(torch.int16).cpu()
    del pool, q
    torch.cuda.empty_cache()
    scale = 1.0 / math.sqrt(128)

    def one(i):
        _, ql, kl = its[i]
        k, v = op.gather_pages(k_host, v_host, bt[i], kl)
        r0 = 0 if i == 0 else p + i - 1
        qq = oa.bf16_bits_to_float64_tensor(q_host[r0:r0 + ql])
        oa.attention_rows(qq, oa.bf16_bits_to_float64_tensor(k),
                          oa.bf16_bits_to_float64_tensor(v), scale, np.arange(kl - ql, kl))

    t0 = time.perf_counter()
    one(0)
    t_prompt = time.perf_counter() - t0
    n_dec, t1 = 0, time.perf_counter()
    while n_dec < n_sample - 1 and (n_dec < 2 or time.perf_counter() - t0 < seconds):
        one(1 + n_dec)
        n_dec += 1
    t_dec = (time.perf_counter() - t1) / n_dec
    per_iter = t_prompt + t_dec * cfg.n_decoders
    tokens = p + cfg.n_decoders
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    import re
    m = re.search(r"BLAS_INFO=([^,\s]+)", torch.__config__.show())
    blas = m.group(1) if m else "unknown"
    lib = [ln.strip() for ln in torch.__config__.parallel_info().splitlines()
           if "Math Kernel Library" in ln or "OpenBLAS" in ln]
    if lib:
        blas = f"{blas} ({lib[0]})"
    return {"value": round(tokens / per_iter, 2), "unit": "tok/s",
            "cores": int(torch.get_num_threads()), "kind": "oracle",
            "sample": (f"float64 oracle (PyTorch CPU ops) on iteration p_t={p}, chunk {c} of the "
                       f"Qwen3-32B sweep: the {p}-token prompt chunk over a {c * p}-token prefix "
                       f"({t_prompt:.2f} s) and {n_dec} of the 256 decoders ({t_dec * 1e3:.0f} ms "
                       f"each), scaled to the whole iteration ({per_iter:.1f} s for {tokens} "
                       f"tokens)"),
            "seconds": round(time.perf_counter() - t0, 2),
            "prefill_s_per_iteration": round(t_prompt, 3),
            "decode_s_per_iteration": round(t_dec * cfg.n_decoders, 3),
            "cpu_model": model, "nproc": os.cpu_count(), "blas": blas}


# ----------------------------------------------------------------------------- main

def pmc_workload(dev, kind, fused=True):
    """Workloads for counter passes (no timing).
    'sweep-32b' / 'sweep-0.6b': one untimed sweep of the shape (the headline's launches;
    0.6B over its 28 pools), then a plain 1 GiB device-to-device copy whose known
    traffic calibrates the FETCH_SIZE / WRITE_SIZE counters.
    'shares-8b' / 'shares-32b': 10 decode-only launches, then 10 prefill-only
    launches of the last chunk of the largest size (two layer pools)."""
    import torch
    from paper_2609_38386_amd import workload as wl
    if kind in ("shares-8b", "shares-32b"):
        cfg = wl.CONFIGS["qwen3-8b" if kind == "shares-8b" else "qwen3-32b"]()
        sw = Sweep(cfg, dev, n_pools=2, layers=2, seed_offset=1, fused=fused)
        p = max(cfg.chunks)
        for _ in range(5):
            sw.iteration(cfg.chunks[0], 0, prefill=False, record=False)
        for _ in range(5):
            sw.iteration(p, cfg.prompt_len // p - 1, decoders=False, record=False)
        torch.cuda.synchronize()
        print(json.dumps({"decode_launches": 10, "prefill_launches": 10, "p_t": p}), flush=True)
        return
    cfg = wl.qwen3_32b_config() if kind == "sweep-32b" else wl.qwen3_0_6b_config()
    sw = Sweep(cfg, dev, n_pools=cfg.layers, layers=cfg.layers, fused=fused)
    n = 0
    for p in cfg.chunks:
        for c in sw.chunks(p, "all"):
            sw.iteration(p, c, record=False)
            n += 1
    del sw
    torch.cuda.empty_cache()
    a = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"iterations": n, "attention_launches": n * cfg.layers,
                      "copy_bytes_each_way": 1 << 30}), flush=True)


def plot_latency(line, path):
    """Latency of one mixed iteration per timed layer against the prefill chunk
    p_t, one panel per shape of a bench line: the mean over the sweep's chunk
    iterations, the first-to-last chunk spread (their medians), the decode-only
    iteration at p_t = 0, and the ideal-overlap bound t_lb of the same work."""
    import matplotlib
    matplotlib.use("Agg")
    import matplotlib.pyplot as plt
    panels = [("Qwen3-32B (headline), 1 layer", line["latency_vs_pt"],
               line["controller"]["decode_only_iter_ms"], 1)]
    for name, o in line.get("other_shapes", {}).items():
        pretty = "Qwen3-" + name.split("-", 1)[1].upper()
        panels.append((f"{pretty}, {o['layers_per_iteration_timed']} layers per iteration",
                       o["latency_vs_pt"], o["decode_only_iter_ms"],
                       o["layers_per_iteration_timed"]))
    fig, axes = plt.subplots(1, len(panels), figsize=(5.2 * len(panels), 4.2), squeeze=False)
    for ax, (title, lat, dec_ms, layers) in zip(axes[0], panels):
        ps = sorted(lat, key=int)
        x = np.arange(len(ps) + 1)
        mean = [dec_ms * 1e3 / layers] + [lat[p]["iter_ms_mean"] * 1e3 / layers for p in ps]
        lo = [mean[0]] + [min(lat[p]["iter_ms_first_mid_last"]) * 1e3 / layers for p in ps]
        hi = [mean[0]] + [max(lat[p]["iter_ms_first_mid_last"]) * 1e3 / layers for p in ps]
        ax.fill_between(x, lo, hi, alpha=0.25, label="first / last chunk (medians)")
        ax.plot(x, mean, "o-", label="mean over the sweep's chunks")
        ax.plot(x[1:], [lat[p]["t_lb_us"] for p in ps], "k--", lw=1,
                label="t_lb = max(B / 8 TB/s, F / 2.5 PF)")
        ax.set_xticks(x, ["0\n(decode\nonly)"] + ps)
        ax.set_xlabel("prefill chunk p_t (tokens)")
        ax.set_ylabel("attention latency per layer (us)")
        ax.set_ylim(bottom=0)
        ax.set_title(title, fontsize=10)
        ax.grid(alpha=0.3)
        ax.legend(fontsize=7, loc="upper left")
    fig.suptitle(f"Mixed-iteration latency vs p_t on one MI355X ({line['value'] / 1e3:.1f}k "
                 f"tokens/s headline)", fontsize=11)
    fig.tight_layout()
    fig.savefig(path, dpi=110)
    plt.close(fig)


def main():
    args = parse_args()
    if args.plot_from:
        with open(args.plot_from) as fh:
            rows = [r for r in fh.read().splitlines() if r.startswith("{")]
        plot_latency(json.loads(rows[-1]), args.plot or "latency_vs_pt.png")
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported: the library "
              "has no multi-GPU path (the hot path would shard by KV head or by sequence "
              "with no exchange inside attention)", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2609_38386_amd import dlfp as D
    from paper_2609_38386_amd import workload as wl
    D.lib()  # fail loudly without the HIP library
    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    if args.pmc_workload:
        pmc_workload(dev, args.pmc_workload, fused=not args.two_launch)
        return
    logf = lambda *a: log(args, *a)  # noqa: E731
    fused = not args.two_launch
    cfg = wl.qwen3_32b_config()
    tuning = None
    if args.tuning:
        from paper_2609_38386_amd import dlfp as D
        tuning = D.dlfp_tuning(*[int(x) for x in args.tuning.split(",")])
    r = run_sweep(cfg, dev, logf, n_pools=1, layers=1, steps=args.steps, warmup=args.warmup,
                  record=record_all, fused=fused, tuning=tuning)
    logf(f"headline done: {r['wall']:.2f}s for {args.steps} steps")
    errors = {"qwen3-32b": r["workspace_error"]}
    ceilings = None
    if not args.headline_only:
        ceilings = measure_ceilings(dev, logf)
        r["roofline"]["frac_of_measured_ceiling"] = round(
            r["roofline"]["achieved"] / ceilings["hbm_random_8KiB_GBps"], 4)
        shares_against_ceilings(r["shares"], ceilings)
    if fused:
        r["roofline"]["traffic"] = profiled_traffic()
    cpu = None
    if not args.no_cpu_baseline and not args.headline_only:
        cpu = cpu_baseline(dev, args.cpu_seconds)
        logf(f"cpu baseline done: {cpu['value']} tok/s")
    extras = {}
    names = [] if args.configs in ("", "none") or args.headline_only else args.configs.split(",")
    for name in names:
        name = name.strip()
        ocfg = wl.CONFIGS[name]()
        if name == "qwen3-0.6b":   # 28 distinct pools: one pool (154 MB) fits the 256 MB cache
            pools, layers, steps, rec = ocfg.layers, ocfg.layers, args.other_steps, record_quarter
        else:                      # each pool is far larger than the cache
            pools, layers, steps, rec = 2, 2, args.other_steps, record_all
        o = run_sweep(ocfg, dev, logf, n_pools=pools, layers=layers, steps=steps, warmup=1,
                      record=rec, fused=fused, tuning=tuning)
        shares_against_ceilings(o["shares"], ceilings)
        extras[name] = other_shape(name, ocfg, o, layers, pools)
        errors[name] = o["workspace_error"]
        logf(f"{name} done: {o['tokens'] / o['wall']:.0f} tok/s")
    replay = None
    if args.replay_seeds not in ("", "none") and not args.headline_only:
        seeds = [int(x) for x in args.replay_seeds.split(",")]
        replay = run_replays(dev, seeds, logf)
        replay["overlap_20_req_s"] = run_overlap_replay(dev, seeds[0], 20.0, logf)
        replay["root_cause"] = run_root_cause_replays(dev, seeds[0], (2.0, 20.0), logf)
        replay["layer_proxy"] = run_layer_proxy_replays(dev, seeds, logf)
        replay["variants"] = run_variant_replays(dev, seeds[0], 1.0, args.variant_requests, logf)
    if any(errors.values()):
        print(f"bench.py: the workspace error word is set after the timed launches: {errors} "
              "(1 = a block id outside the pool, 2 = a wait for the append records ran out); "
              "no result is reported", file=sys.stderr)
        sys.exit(1)
    ms_per_step = r["wall"] * 1e3 / args.steps
    value = r["tokens"] / r["wall"]
    line = {
        "metric": METRIC, "value": round(value, 1),
        "unit": "tok/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": ("qwen3-32b attention, one layer, all 64 query heads on one GPU: "
                                "256 decoders ctx U[2048,32768] + 32768-token prompt chunked at "
                                "p_t in {512..8192}, full sweep (124 chunk iterations) per step"),
                   "num_q_heads": 64, "num_kv_heads": 8, "head_dim": 128, "page": 16,
                   "decoders": cfg.n_decoders, "prompt_len": cfg.prompt_len,
                   "chunks": list(cfg.chunks), "layers": 1, "distinct_layer_pools": 1,
                   "tokens_per_step": r["tokens"] // args.steps},
        "roofline": r["roofline"],
        "cpu_baseline": cpu,
        "ceilings": ceilings,
        "latency_vs_pt": r["latency"],
        "shares": r["shares"],
        "controller": {"target_ms": round(r["target_ms"], 4),
                       "decode_only_iter_ms": round(r["decode_only_iter_ms"], 4),
                       "rule": "Eq. 2, completion-timed (HIP events), quantum 128"},
        "workspace_error": errors,
        "other_shapes": extras,
        "replay": replay,
        "paper_context": "27.7% mean P99 ITL reduction, Qwen3-0.6B BF16, 1x A100 80GB (context only)",
    }
    print(json.dumps(line), flush=True)
    if args.plot:
        plot_latency(line, args.plot)


if __name__ == "__main__":
    main()
