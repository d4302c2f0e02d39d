#!/usr/bin/env python3
"""Benchmark of the paged-KV checkpoint path on one MI355X.

Headline step (the value and the roofline): one decode step of the
Llama-3-8B-shaped workload (32 layers, 8 KV heads, head_dim 128, block 16,
bf16; 256 requests with lognormal contexts; every step checkpoints each
request's newest 1-16 tokens):

    pack(step k)    source pool -> checkpoint region k mod 20
    unpack(step k') checkpoint region k' mod 20 -> restore pool

with k' = k + 10, so the restore reads a region packed 10 steps (about
5.7 GB of traffic) earlier, never a copy still held in the 256 MB Infinity
Cache.  Each copy is one launch that plans its rows from the token ranges
itself (lumen_kv_ckpt_pack_ranges / _unpack_ranges); the same steps issued
as plan + copy (a plan kernel into a workspace before each copy) are timed
right after on the same buffers and reported as other_path.  Where a buffer lands in physical memory moves the copies by up to
15%, so the written buffers (restore pool and 20-region arena) are
allocated --placements times (default 3) over one source pool, the timed
steps rotate over those sets, and each set is then timed alone.  Inputs
(pools, block tables, ranges) are resident in HBM before timing; the device
error word is checked after the timed loop.  The value is the timed pass:
exactly --steps steps with nothing else on the stream.  Per-kernel times
come from an event pass right after it: the same steps again (at least 20),
every copy kernel carrying two HIP events that its own dispatch stamps at
its start and end, on its stream (lumen_kv_ckpt_time_next_copy).

Further legs (reported beside the headline, not part of its value):
  * tiny            the 8-request, 1.77 MB full pack and restore: launch
                    latency, back-to-back rate and host enqueue cost
  * small           decode steps of the first 8 .. 128 requests, into a
                    buffer of the step's rows and into a multi-step arena
                    (the grid follows the checkpoint buffer)
  * qwen-gqa-hnd    the same decode loop on the head-major Qwen-style cache
  * qwen-gqa-nhd-twin  the same requests and tables over a token-major cache,
                    on the same buffers (what the head-major transpose costs)
  * restore-burst   64 interrupted requests restored into a 60%-occupied
                    pool; ms per restored request
  * tp8-shard       full pack and in-place unpack of one TP=8 rank of a
                    Llama-3-70B-shaped cache, the packed rows streamed to a
                    pinned host ring on a side stream during the pack
  * host staging    decode steps checkpointed straight to pinned host memory
                    beside an HBM-bound decode stand-in (its slowdown), and
                    every restore-burst request restored from host memory
  * page tags       host-side tag generation and longest-prefix lookups
  * scheduler       host-side Eq. 1 placement and recovery events
  * draft-align     draft-state alignment of 1,024 mirror requests
  * cpu_baseline    the CPU oracle on a bounded sample of the decode workload,
                    on one thread and split over the host's threads

Bytes are algorithmic: 2 x tokens x token_row_bytes (read + write),
decimal GB; peak is MI355X's 8 TB/s.
"""
from __future__ import annotations

import argparse
import ctypes
import dataclasses
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, vendor figure
METRIC = ("KV checkpoint pack/unpack GB/s and % of HBM peak, 1×MI355X; "
          "restore ms/request")
ALL_LEGS = ("decode", "tiny", "small", "qwen", "restore", "tp8", "stage",
            "tags", "sched", "draft", "cpu")
MIN_KERNEL_SAMPLES = 20  # fewest timed launches of a per-kernel figure


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--legs", default=",".join(ALL_LEGS),
                    help="comma list of " + ",".join(ALL_LEGS))
    ap.add_argument("--placements", type=int, default=3,
                    help="independently allocated (restore pool, arena) "
                    "sets of the headline decode leg")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="budget of the CPU oracle sample")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB "
                    "(5 times), the reference for HBM byte counters")
    return ap.parse_args()


def gb(x):
    return x / 1e9


_HIP = None


def _hip_runtime():
    """The HIP runtime this process has already loaded (torch's copy, which
    the checkpoint library binds to as well), so that events and streams
    belong to one runtime."""
    global _HIP
    if _HIP is None:
        with open("/proc/self/maps") as f:
            path = next((ln.split()[-1] for ln in f
                         if "libamdhip64" in ln), None)
        if path is None:
            raise RuntimeError("the HIP runtime is not loaded")
        lib = ctypes.CDLL(path)
        vp = ctypes.c_void_p
        lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(vp),
                                                ctypes.c_uint]
        lib.hipEventRecord.argtypes = [vp, vp]
        lib.hipEventSynchronize.argtypes = [vp]
        lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float),
                                            vp, vp]
        lib.hipEventDestroy.argtypes = [vp]
        _HIP = lib
    return _HIP


class TimingEvent:
    """A HIP event for timing only, created with hipEventDisableSystemFence:
    recording it does not write back and invalidate the caches, which HIP
    documents as the precise way to time device work on AMD GPUs (measured
    here: 2 us less per bracketed decode launch than a default event, closer
    to the kernel trace).  It orders nothing and must not gate host reads
    of memory the device wrote; such waits keep torch's default events.
    Same interface as torch.cuda.Event for record / synchronize /
    elapsed_time."""
    _FLAGS = 0x20000000  # hipEventDisableSystemFence

    def __init__(self):
        import torch
        self._torch = torch
        self._hip = _hip_runtime()
        self.ev = ctypes.c_void_p()
        if self._hip.hipEventCreateWithFlags(ctypes.byref(self.ev),
                                             self._FLAGS) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self, stream=None):
        s = (stream if stream is not None
             else self._torch.cuda.current_stream()).cuda_stream
        if self._hip.hipEventRecord(self.ev, ctypes.c_void_p(s)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def synchronize(self):
        if self._hip.hipEventSynchronize(self.ev) != 0:
            raise RuntimeError("hipEventSynchronize failed")

    def elapsed_time(self, end):
        ms = ctypes.c_float()
        if self._hip.hipEventElapsedTime(ctypes.byref(ms), self.ev,
                                         end.ev) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def __del__(self):
        if getattr(self, "ev", None) and self.ev.value:
            self._hip.hipEventDestroy(self.ev)


def stamp(start, stop):
    """The next copy call's kernel carries these two events: they take its
    own start and end (hipExtLaunchKernel), with no marker commands of ours
    on the stream around it."""
    import paper_2606_17787_amd.kvckpt as kv
    kv.lumen_kv_ckpt_time_next_copy(start.ev, stop.ev)


def say(msg):
    print(msg, file=sys.stderr, flush=True)


# --------------------------------------------------------------- GPU legs

def _event_steps(steps):
    """Steps of the event pass: as many as the timed pass, and never fewer
    than MIN_KERNEL_SAMPLES."""
    return list(range(max(steps, MIN_KERNEL_SAMPLES)))


def _kernel_stats(byts, ms):
    """GB/s (summed bytes over summed time), mean / median / p10 / p90 us per
    launch, of one kernel's sampled launches."""
    byts, ms = np.asarray(byts, np.float64), np.asarray(ms, np.float64)
    return dict(GBps=gb(byts.sum()) / (ms.sum() / 1e3),
                us_mean=float(ms.mean() * 1e3),
                us_median=float(np.median(ms) * 1e3),
                us_p10_p90=[float(np.percentile(ms, q) * 1e3)
                            for q in (10, 90)],
                samples=int(ms.size), bytes_mean=float(byts.mean()))


def incremental_leg(torch, kv, w, steps, warmup, seed, keep=None,
                    placements=1, regions=None, placement_steps=24,
                    path="plan", compare=None, per_request_path=None):
    """Decode loop: step i packs step k = i mod S into its checkpoint region
    and restores step k + lag from the region packed lag steps earlier (lag =
    half the regions), so the restore never reads a copy still held in the
    256 MB Infinity Cache.  Per-kernel times from HIP events on the launch
    stream.

    placements: independently allocated sets of written buffers
    (destination pool and arena), all resident at once, over one source
    pool.  Where a buffer lands in physical memory moves the copies by up to
    15%, so the timed steps rotate over the sets, and a pass after the timed
    region times placement_steps steps on each set alone.
    regions: checkpoint regions per arena (None: one per step, laid out back
    to back); fewer regions, each sized to the largest step, keep several
    arenas within HBM.
    keep: a dict that carries the buffers from one call to the next (one
    placement only; None: allocate and free here).  Workloads of the same
    byte sizes then run on the same physical memory, so that their rates
    differ only by what the workloads do, not by where the buffers landed.
    path: how a step's copies are issued: "plan" (a plan kernel into a
    workspace before each copy) or "ranges" (each copy one launch that
    plans from the ranges itself).  compare: the other path, timed the
    same way right after on the same buffers (reported as other_path).
    per_request_path: the path of the per-request row mode (default:
    path)."""
    dev = torch.device("cuda:0")
    sh = w.shape
    S = w.num_steps
    rows = np.array([w.step_tokens(k) for k in range(S)], np.int64)
    row_elems = sh.token_row_elems
    rb = sh.token_row_bytes
    if regions is None or regions >= S:
        NR = S
        region_row = np.concatenate([[0], np.cumsum(rows)])[:S]
        arena_rows = int(rows.sum())
    else:
        if S % regions or regions % 2:
            raise ValueError("regions must be even and divide the steps")
        NR = regions
        region_row = (np.arange(S) % NR) * int(rows.max())
        arena_rows = NR * int(rows.max())
    lag = NR // 2
    P = placements
    if keep is not None and P != 1:
        raise ValueError("buffers are kept across legs for one placement")

    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    sizes = (sh.pool_elems(w.num_blocks), sh.pool_elems(w.dst_num_blocks),
             arena_rows * row_elems)
    if keep is not None and keep.get("sizes") == sizes:
        src, dst, arena = keep.pop("bufs")
        dst.zero_()
        sets = [(dst, arena)]
    else:
        if keep is not None:
            keep.clear()
            torch.cuda.empty_cache()
        src = torch.empty(sizes[0], dtype=torch.bfloat16, device=dev)
        sets = [(torch.zeros(sizes[1], dtype=torch.bfloat16, device=dev),
                 torch.empty(sizes[2], dtype=torch.bfloat16, device=dev))
                for _ in range(P)]
    src.normal_(generator=g)
    bt = torch.from_numpy(w.block_tables).to(dev)
    bt_dst = torch.from_numpy(w.dst_block_tables).to(dev)
    starts = [torch.from_numpy(a).to(dev) for a in w.starts]
    ends = [torch.from_numpy(a).to(dev) for a in w.ends]
    ws_a = kv.new_workspace(w.num_reqs, dev)
    ws_b = kv.new_workspace(w.num_reqs, dev)

    # Fill every checkpoint region of every arena once (also the first
    # correctness gate).
    for _, arena in sets:
        for k in range(S):
            kv.lumen_kv_ckpt_plan(starts[k], ends[k], ws_a, int(region_row[k]))
            kv.lumen_kv_ckpt_pack(sh, w.num_blocks, src, bt, ws_a, arena)
    st = kv.lumen_kv_ckpt_status(ws_a)
    if st != 0:
        raise RuntimeError(f"pack reported {kv.lumen_kv_ckpt_strerror(st)}")

    status = torch.zeros(1, dtype=torch.int32, device=dev)

    def copies(how, k, k2, dst, arena, events, rrb=None):
        """Pack of step k and unpack of step k2, issued the `how` way;
        `events` (two pairs) take the copy kernels' own start and end."""
        b1 = 0 if rrb is not None else int(region_row[k])
        b2 = 0 if rrb is not None else int(region_row[k2])
        if how == "ranges":
            if events: stamp(events[0], events[1])
            kv.lumen_kv_ckpt_pack_ranges(sh, w.num_blocks, src, bt, starts[k],
                                         ends[k], arena, status, b1, rrb)
            if events: stamp(events[2], events[3])
            kv.lumen_kv_ckpt_unpack_ranges(sh, w.dst_num_blocks, dst, bt_dst,
                                           starts[k2], ends[k2], arena,
                                           status, b2, rrb)
            return
        kv.lumen_kv_ckpt_plan(starts[k], ends[k], ws_a, b1, rrb)
        if events: stamp(events[0], events[1])
        kv.lumen_kv_ckpt_pack(sh, w.num_blocks, src, bt, ws_a, arena)
        kv.lumen_kv_ckpt_plan(starts[k2], ends[k2], ws_b, b2, rrb)
        if events: stamp(events[2], events[3])
        kv.lumen_kv_ckpt_unpack(sh, w.dst_num_blocks, dst, bt_dst, ws_b,
                                arena)

    def check_status():
        st = min(kv.lumen_kv_ckpt_status(ws_a), kv.lumen_kv_ckpt_status(ws_b),
                 int(status.item()))
        status.zero_()
        if st != 0:
            raise RuntimeError(f"device error {kv.lumen_kv_ckpt_strerror(st)}")

    def step(i, events=None, p=None, how=path):
        k = i % S
        k2 = (k + lag) % S
        dst, arena = sets[i % P if p is None else p]
        copies(how, k, k2, dst, arena, events)
        return k, k2

    def sampled_stats(done, ev, idx):
        pk = _kernel_stats([2 * rows[done[i][0]] * rb for i in idx],
                           [ev[i][0].elapsed_time(ev[i][1]) for i in idx])
        up = _kernel_stats([2 * rows[done[i][1]] * rb for i in idx],
                           [ev[i][2].elapsed_time(ev[i][3]) for i in idx])
        return pk, up

    def events(n):
        return {i: [TimingEvent() for _ in range(4)] for i in n}

    def self_check(last, bufs):
        """The last timed step checked without an oracle, before a later
        pass rewrites its buffers (the passes over one placement at a time
        map steps to other regions): its pack's region equals a fresh pack
        of its step, and re-packing the tokens its unpack restored gives
        back the region that unpack read."""
        (k1, k2), (dst, arena) = last, bufs
        ok = True
        for k, pool, nb, table in ((k1, src, w.num_blocks, bt),
                                   (k2, dst, w.dst_num_blocks, bt_dst)):
            n = int(rows[k])
            out = torch.empty(n * row_elems, dtype=torch.bfloat16, device=dev)
            kv.lumen_kv_ckpt_plan(starts[k], ends[k], ws_b, 0)
            kv.lumen_kv_ckpt_pack(sh, nb, pool, table, ws_b, out)
            r0 = int(region_row[k])
            region = arena[r0 * row_elems:(r0 + n) * row_elems]
            ok = ok and bool(torch.equal(out.view(torch.int16),
                                         region.view(torch.int16)))
            assert kv.lumen_kv_ckpt_status(ws_b) == 0
        if not ok:
            say(f"[bench] {w.name}: self-check of the last timed step FAILED")
        return ok

    # The timed pass (the value): exactly `steps` steps with nothing but
    # the copies and their plans on the stream.
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    done = [step(warmup + i) for i in range(steps)]
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    check_status()
    step_b = sum(2.0 * (rows[k] + rows[k2]) * rb for k, k2 in done)
    wall_ms = (t1 - t0) * 1e3
    # The event pass (the per-kernel figures): the same steps again, from
    # the same schedule position, each copy kernel stamping its own start
    # and end on two HIP events.  They stay out of the timed pass.
    roundtrip = self_check(done[-1], sets[(warmup + steps - 1) % P])
    sampled = _event_steps(steps)
    ev = events(sampled)
    done_ev = [step(warmup + i, ev[i]) for i in sampled]
    torch.cuda.synchronize()
    check_status()
    pack, unpack = sampled_stats(done_ev, ev, sampled)

    # The other path, timed the same way on the same buffers.
    other = None
    if compare is not None:
        for i in range(warmup):
            step(i, how=compare)
        torch.cuda.synchronize()
        t4 = time.perf_counter()
        done_o = [step(warmup + i, how=compare) for i in range(steps)]
        torch.cuda.synchronize()
        t5 = time.perf_counter()
        check_status()
        ev_o = events(sampled)
        done_oev = [step(warmup + i, ev_o[i], how=compare) for i in sampled]
        torch.cuda.synchronize()
        check_status()
        pk_o, up_o = sampled_stats(done_oev, ev_o, sampled)
        other = dict(
            path=compare, ms_per_step=(t5 - t4) * 1e3 / steps,
            step_GBps=gb(sum(2.0 * (rows[k] + rows[k2]) * rb
                             for k, k2 in done_o)) / (t5 - t4),
            pack_GBps=pk_o["GBps"], unpack_GBps=up_o["GBps"],
            pack_us_median=pk_o["us_median"],
            unpack_us_median=up_o["us_median"])

    # Each placement alone, after the timed region.
    per_placement = []
    if P > 1:
        for p in range(P):
            evp = events(range(placement_steps))
            for i in range(4):
                step(i, p=p)
            dn = [step(i, evp[i], p=p) for i in range(placement_steps)]
            torch.cuda.synchronize()
            check_status()
            pk, up = sampled_stats(dn, evp, range(placement_steps))
            per_placement.append(dict(
                pack_GBps=pk["GBps"], unpack_GBps=up["GBps"],
                pack_us_median=pk["us_median"],
                unpack_us_median=up["us_median"],
                pack_us_p10_p90=pk["us_p10_p90"],
                unpack_us_p10_p90=up["us_p10_p90"], samples=pk["samples"]))

    # The per-request row mode: one checkpoint per request (Sec. 4.2), the
    # increments of request r appending to its own region of the arena, so a
    # step's rows land in up to R places instead of one run.  Steps
    # 0 .. NR-1 fill an arena exactly; the steps rotate over the placements
    # as in the timed pass.
    inc = w.ends[NR - 1].astype(np.int64) - w.starts[0].astype(np.int64)
    assert int(inc.sum()) == int(rows[:NR].sum()) <= arena_rows
    region0 = np.concatenate([[0], np.cumsum(inc)[:-1]])
    rrb_h = region0 - w.starts[0].astype(np.int64)  # row of token t: rrb + t
    rrb = torch.from_numpy(rrb_h).to(dev)
    for _, arena in sets:
        for k in range(NR):
            kv.lumen_kv_ckpt_plan(starts[k], ends[k], ws_a, 0, rrb)
            kv.lumen_kv_ckpt_pack(sh, w.num_blocks, src, bt, ws_a, arena)
    assert kv.lumen_kv_ckpt_status(ws_a) == 0
    pr_steps = max(steps // 2, MIN_KERNEL_SAMPLES)

    pr_path = per_request_path or path

    def step_pr(i, events=None):
        k = i % NR
        k2 = (k + lag) % NR
        dst, arena = sets[i % P]
        copies(pr_path, k, k2, dst, arena, events, rrb)
        return k, k2

    for i in range(warmup):
        step_pr(i)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    pr_done = [step_pr(warmup + i) for i in range(pr_steps)]
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    pr_sampled = _event_steps(pr_steps)
    pr_ev = events(pr_sampled)
    pr_done_ev = [step_pr(warmup + i, pr_ev[i]) for i in pr_sampled]
    torch.cuda.synchronize()
    check_status()
    pr_pack, pr_unpack = sampled_stats(pr_done_ev, pr_ev, pr_sampled)
    pr_step_b = sum(2.0 * (rows[k] + rows[k2]) * rb for k, k2 in pr_done)
    # self-check: one step's rows, gathered from the request regions, equal
    # the same step packed contiguously (every arena holds every step's
    # rows in its regions)
    k = pr_done[-1][0]
    arena = sets[(warmup + pr_steps - 1) % P][1]
    kv.lumen_kv_ckpt_plan(starts[k], ends[k], ws_a, 0)
    back = torch.empty(int(rows[k]) * row_elems, dtype=torch.bfloat16,
                       device=dev)
    kv.lumen_kv_ckpt_pack(sh, w.num_blocks, src, bt, ws_a, back)
    idx = np.concatenate([np.arange(rrb_h[r] + w.starts[k][r],
                                    rrb_h[r] + w.ends[k][r])
                          for r in range(w.num_reqs)]).astype(np.int64)
    gathered = arena.view(-1, row_elems).index_select(
        0, torch.from_numpy(idx).to(dev))
    pr_ok = bool(torch.equal(gathered.view(torch.int16).reshape(-1),
                             back.view(torch.int16)))
    assert kv.lumen_kv_ckpt_status(ws_a) == 0
    per_request_mode = dict(
        path=pr_path, steps=pr_steps, placements=P,
        ms_per_step=(t3 - t2) * 1e3 / pr_steps,
        step_GBps=gb(pr_step_b) / (t3 - t2),
        pack_GBps=pr_pack["GBps"], unpack_GBps=pr_unpack["GBps"],
        pack_us_median=pr_pack["us_median"],
        unpack_us_median=pr_unpack["us_median"],
        samples=pr_pack["samples"], check_ok=pr_ok)
    if keep is not None:
        keep["sizes"], keep["bufs"] = sizes, (src, sets[0][0], sets[0][1])
    del src, sets, arena, back, gathered
    if keep is None:
        torch.cuda.empty_cache()

    out = dict(
        workload=w.name, fingerprint=w.fingerprint(), path=path, steps=steps,
        warmup=warmup, wall_ms=wall_ms, ms_per_step=wall_ms / steps,
        step_GBps=gb(step_b) / (wall_ms / 1e3), sampled_steps=len(sampled),
        placements=P, regions=NR,
        pack_GBps=pack["GBps"], unpack_GBps=unpack["GBps"],
        pack_pct_peak=100 * pack["GBps"] / HBM_PEAK_GBPS,
        unpack_pct_peak=100 * unpack["GBps"] / HBM_PEAK_GBPS,
        pack_us_mean=pack["us_mean"], unpack_us_mean=unpack["us_mean"],
        pack_us_median=pack["us_median"],
        unpack_us_median=unpack["us_median"],
        pack_us_p10_p90=pack["us_p10_p90"],
        unpack_us_p10_p90=unpack["us_p10_p90"],
        pack_bytes_mean=pack["bytes_mean"],
        unpack_bytes_mean=unpack["bytes_mean"],
        tokens_per_step_mean=float(rows.mean()),
        roundtrip_ok=roundtrip,
        per_request_mode=per_request_mode,
    )
    if other is not None:
        out["other_path"] = other
    if per_placement:
        out["per_placement"] = per_placement
        for op in ("pack", "unpack"):
            v = sorted(x[f"{op}_GBps"] for x in per_placement)
            out[f"{op}_placement_worst_GBps"] = v[0]
            out[f"{op}_placement_median_GBps"] = float(np.median(v))
            out[f"{op}_placement_worst_pct_peak"] = \
                100 * v[0] / HBM_PEAK_GBPS
    return out


def restore_leg(torch, kv, W):
    """Failure-restore burst: 64 interrupted requests of 4K-32K tokens
    restored from contiguous checkpoints into a 60%-occupied pool, in waves
    that fit the free list.  Reports device ms per restored request."""
    dev = torch.device("cuda:0")
    w = W.c3_restore()
    sh = w.shape
    waves = W.restore_waves(w)
    ctx = w.ends[0].astype(np.int64)
    max_rows = max(int(ctx[wv].sum()) for wv in waves)
    row_elems = sh.token_row_elems
    g = torch.Generator(device=dev)
    g.manual_seed(3)
    pool = torch.zeros(sh.pool_elems(w.dst_num_blocks), dtype=torch.bfloat16,
                       device=dev)
    ck = torch.empty(max_rows * row_elems, dtype=torch.bfloat16, device=dev)
    ck.normal_(generator=g)
    per_req_ms, wave_stats = [], []
    for wv in waves:
        s = torch.from_numpy(w.starts[0][wv]).to(dev)
        e = torch.from_numpy(w.ends[0][wv]).to(dev)
        bt = torch.from_numpy(w.dst_block_tables[wv]).to(dev)
        ws = kv.new_workspace(len(wv), dev)
        nrows = int(ctx[wv].sum())
        view = ck[:nrows * row_elems]
        kv.lumen_kv_ckpt_plan(s, e, ws)
        kv.lumen_kv_ckpt_unpack(sh, w.dst_num_blocks, pool, bt, ws, view)
        torch.cuda.synchronize()
        reps = []
        for _ in range(3):
            a = TimingEvent()
            b = TimingEvent()
            kv.lumen_kv_ckpt_plan(s, e, ws)
            stamp(a, b)
            kv.lumen_kv_ckpt_unpack(sh, w.dst_num_blocks, pool, bt, ws, view)
            b.synchronize()
            reps.append(a.elapsed_time(b))
        assert kv.lumen_kv_ckpt_status(ws) == 0
        t = float(np.median(reps))
        byts = 2.0 * nrows * sh.token_row_bytes
        wave_stats.append(dict(requests=len(wv), tokens=nrows, ms=round(t, 3),
                               GBps=round(gb(byts) / (t / 1e3), 1)))
        per_req_ms += [t * float(ctx[r]) / nrows for r in wv]
    # per-request launches: each request of the last wave restored by its
    # own plan + unpack (median over the wave)
    wv = waves[-1]
    bt = torch.from_numpy(w.dst_block_tables[wv]).to(dev)
    s_w = torch.from_numpy(w.starts[0][wv]).to(dev)
    e_w = torch.from_numpy(w.ends[0][wv]).to(dev)
    ws1 = kv.new_workspace(1, dev)
    single_ms = []
    for i in range(len(wv)):
        a = TimingEvent()
        b = TimingEvent()
        a.record()
        kv.lumen_kv_ckpt_plan(s_w[i:i + 1], e_w[i:i + 1], ws1)
        kv.lumen_kv_ckpt_unpack(sh, w.dst_num_blocks, pool, bt[i:i + 1], ws1,
                                ck[:int(ctx[wv[i]]) * row_elems])
        b.record()
        b.synchronize()
        single_ms.append(a.elapsed_time(b))
    assert kv.lumen_kv_ckpt_status(ws1) == 0
    del pool, ck
    torch.cuda.empty_cache()
    tot_ms = sum(x["ms"] for x in wave_stats)
    tot_b = sum(2.0 * x["tokens"] * sh.token_row_bytes for x in wave_stats)
    return dict(workload=w.name, requests=w.num_reqs,
                restore_ms_per_request=tot_ms / w.num_reqs,
                restore_ms_per_request_median=float(np.median(per_req_ms)),
                single_request_launch_ms_median=float(np.median(single_ms)),
                single_request_launches=len(single_ms),
                unpack_GBps=gb(tot_b) / (tot_ms / 1e3),
                mean_request_GB=gb(float(ctx.mean()) * sh.token_row_bytes),
                waves=wave_stats)


def tp8_leg(torch, kv, W, chunks=8, slot_bytes=2 << 30, ring=4):
    """One TP=8 rank's shard of a Llama-3-70B-shaped cache: the full pack as
    one launch; the same pack in request chunks, alone and with each chunk's
    rows streamed to a ring of pinned host buffers on a side stream as soon
    as the chunk is packed (the chunked pack's slowdown under the concurrent
    D2H); the whole checkpoint packed straight into that pinned ring with no
    device arena (direct mode); then an in-place unpack under a fresh
    permutation."""
    dev = torch.device("cuda:0")
    w = W.c4_llama70b_tp8()
    sh = w.shape
    R = w.num_reqs
    s_all, e_all = w.starts[0], w.ends[0]
    n_rows = w.step_tokens(0)
    rb = sh.token_row_bytes
    g = torch.Generator(device=dev)
    g.manual_seed(4)
    pool = torch.empty(sh.pool_elems(w.num_blocks), dtype=torch.bfloat16,
                       device=dev)
    pool.normal_(generator=g)
    arena = torch.empty(n_rows * sh.token_row_elems, dtype=torch.bfloat16,
                        device=dev)
    bt = torch.from_numpy(w.block_tables).to(dev)
    bounds = np.linspace(0, R, chunks + 1).astype(int)
    row_first = np.concatenate([[0], np.cumsum(e_all.astype(np.int64)
                                              - s_all)])
    wss, plans = [], []
    for c in range(chunks):
        r0, r1 = bounds[c], bounds[c + 1]
        wss.append(kv.new_workspace(r1 - r0, dev))
        plans.append((torch.from_numpy(s_all[r0:r1]).to(dev),
                      torch.from_numpy(e_all[r0:r1]).to(dev),
                      bt[r0:r1].contiguous(), int(row_first[r0])))
    side = torch.cuda.Stream()
    host = [torch.empty(slot_bytes // 2, dtype=torch.int16, pin_memory=True)
            for _ in range(ring)]
    slot_free = [None] * ring

    def pack_all(events):
        done = []
        events[0].record()
        for c, (s, e, btc, base) in enumerate(plans):
            kv.lumen_kv_ckpt_plan(s, e, wss[c], base)
            kv.lumen_kv_ckpt_pack(sh, w.num_blocks, pool, btc, wss[c], arena)
            ev = torch.cuda.Event()
            ev.record()
            done.append(ev)
        events[1].record()
        return done

    # The full checkpoint of the shard: one plan, one pack (after an
    # untimed pass that first touches the arena).
    ws_all = kv.new_workspace(R, dev)
    s_dev = torch.from_numpy(s_all).to(dev)
    e_dev = torch.from_numpy(e_all).to(dev)
    t_one = []
    for rep in range(3):
        a = TimingEvent()
        b = TimingEvent()
        kv.lumen_kv_ckpt_plan(s_dev, e_dev, ws_all)
        stamp(a, b)
        kv.lumen_kv_ckpt_pack(sh, w.num_blocks, pool, bt, ws_all, arena)
        b.synchronize()
        if rep:
            t_one.append(a.elapsed_time(b))
    assert kv.lumen_kv_ckpt_status(ws_all) == 0
    # The same pack in request chunks, alone, then with each chunk's rows
    # streamed to the pinned ring as soon as it is packed.
    t_alone = [TimingEvent() for _ in range(2)]
    pack_all(t_alone)
    torch.cuda.synchronize()
    for ws in wss:
        assert kv.lumen_kv_ckpt_status(ws) == 0
    t_pack = [TimingEvent() for _ in range(2)]
    d2h = [TimingEvent() for _ in range(2)]
    done = pack_all(t_pack)
    arena16 = arena.view(torch.int16)
    piece = slot_bytes // 2
    side.wait_event(done[0])
    d2h[0].record(side)
    nslot, checked = 0, []
    for c in range(chunks):
        lo = int(row_first[bounds[c]]) * rb // 2
        hi = int(row_first[bounds[c + 1]]) * rb // 2
        side.wait_event(done[c])
        for off in range(lo, hi, piece):
            j = nslot % ring
            if slot_free[j] is not None:
                slot_free[j].synchronize()  # the host drains the slot
            n = min(piece, hi - off)
            kv.lumen_kv_ckpt_offload(arena16[off:off + n], host[j],
                                     nbytes=2 * n, producer=side, side=side)
            ev = torch.cuda.Event()
            ev.record(side)
            slot_free[j] = ev
            checked.append((off, n, j))
            nslot += 1
    d2h[1].record(side)
    side.synchronize()
    torch.cuda.synchronize()
    ok = True  # the last copy into each slot, against the device bytes
    for off, n, j in checked[-ring:]:
        k = min(n, 1 << 20)
        ok &= bool(torch.equal(host[j][:k], arena16[off:off + k].cpu()))
    for ws in wss:
        assert kv.lumen_kv_ckpt_status(ws) == 0
    # The whole checkpoint straight from the paged cache into the pinned
    # ring, window by window, with no device arena: the gather writes host
    # memory itself (one plan, one direct pack per 2 GiB slot).
    slot_rows = slot_bytes // rb
    views = [h[:slot_rows * rb // 2] for h in host]
    slot_free = [None] * ring
    t_dir = [TimingEvent() for _ in range(2)]
    kv.lumen_kv_ckpt_plan(s_dev, e_dev, ws_all)
    t_dir[0].record()
    last = None
    for c, lo in enumerate(range(0, n_rows, slot_rows)):
        j = c % ring
        if slot_free[j] is not None:
            slot_free[j].synchronize()  # the host drains the slot
        kv.lumen_kv_ckpt_pack_to_host_direct(
            sh, w.num_blocks, pool, bt, ws_all, views[j], row_begin=lo,
            row_end=lo + slot_rows, ckpt_first_row=lo)
        ev = torch.cuda.Event()
        ev.record()
        slot_free[j] = ev
        last = (lo, j)
    t_dir[1].record()
    torch.cuda.synchronize()
    assert kv.lumen_kv_ckpt_status(ws_all) == 0
    lo, j = last
    k = min(n_rows - lo, 64) * rb // 2
    direct_ok = bool(torch.equal(host[j][:k],
                                 arena16[lo * rb // 2:lo * rb // 2 + k].cpu()))
    direct_ms = t_dir[0].elapsed_time(t_dir[1])
    ws = kv.new_workspace(R, dev)
    kv.lumen_kv_ckpt_plan(torch.from_numpy(s_all).to(dev),
                          torch.from_numpy(e_all).to(dev), ws)
    bt_new = torch.from_numpy(w.dst_block_tables).to(dev)
    # validate mode on the restore table before the unpack (timed apart)
    marks = kv.new_marks(w.num_blocks, dev)
    t_val = [TimingEvent() for _ in range(2)]
    t_val[0].record()
    kv.lumen_kv_ckpt_validate_targets(sh, w.num_blocks, bt_new, ws, marks)
    t_val[1].record()
    torch.cuda.synchronize()
    assert kv.lumen_kv_ckpt_status(ws) == 0
    t_un = [TimingEvent() for _ in range(2)]
    stamp(t_un[0], t_un[1])
    kv.lumen_kv_ckpt_unpack(sh, w.num_blocks, pool, bt_new, ws, arena)
    torch.cuda.synchronize()
    assert kv.lumen_kv_ckpt_status(ws) == 0
    byts = 2.0 * n_rows * rb
    alone_ms = t_alone[0].elapsed_time(t_alone[1])
    with_ms = t_pack[0].elapsed_time(t_pack[1])
    un_ms = t_un[0].elapsed_time(t_un[1])
    d2h_ms = d2h[0].elapsed_time(d2h[1])
    del pool, arena, host
    torch.cuda.empty_cache()
    one_ms = float(np.median(t_one))
    return dict(workload=w.name, requests=R, tokens=n_rows,
                pack_GBps=gb(byts) / (one_ms / 1e3), pack_ms=one_ms,
                pack_chunks=chunks,
                pack_chunked_GBps=gb(byts) / (alone_ms / 1e3),
                pack_with_d2h_GBps=gb(byts) / (with_ms / 1e3),
                pack_slowdown_with_d2h=with_ms / alone_ms,
                unpack_in_place_GBps=gb(byts) / (un_ms / 1e3),
                unpack_ms=un_ms,
                validate_us=t_val[0].elapsed_time(t_val[1]) * 1e3,
                validate_pages=int(sum(-(-int(x) // sh.block_size)
                                       for x in e_all)),
                d2h_GBps=gb(n_rows * rb) / (d2h_ms / 1e3), d2h_ms=d2h_ms,
                d2h_bytes=n_rows * rb, d2h_spot_check_ok=ok,
                pinned_ring=f"{ring} x {slot_bytes >> 30} GiB",
                checkpoint_direct_to_host_GBps=gb(n_rows * rb)
                / (direct_ms / 1e3),
                checkpoint_direct_to_host_ms=direct_ms,
                checkpoint_direct_spot_check_ok=direct_ok)


def host_link_rates(torch, host, dev_buf, reps=3):
    """Plain copies between a pinned host buffer and device memory (the
    ceiling of the staging pipelines), GB/s each way."""
    n = min(host.numel(), dev_buf.numel())
    h, d = host[:n], dev_buf[:n]
    res = {}
    for name, (dst, src) in (("h2d", (d, h)), ("d2h", (h, d))):
        dst.copy_(src, non_blocking=True)
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            dst.copy_(src, non_blocking=True)
        b.record()
        b.synchronize()
        res[name] = gb(n * reps) / (a.elapsed_time(b) / 1e3)
    return res


def staging_leg(torch, kv, W, decode_steps=40, ring_slots=2, slot_rows=1024,
                host_slots=4):
    """Host staging both ways.

    Decode side: every step, a stand-in for the decode kernels reads the KV
    the batch attends to (one HBM-bound pass over sum(ctx) token rows of the
    source pool) on the serving stream, while that step's new tokens are
    packed through a small device ring and copied to pinned host memory on
    two other streams (lumen_kv_ckpt_pack_to_host).  Reported: the decode
    stand-in's time alone and with checkpointing, and the sustained D2H.

    Restore side: each of the 64 restore-burst requests is restored from a
    pinned host copy of its checkpoint through the staging ring
    (lumen_kv_ckpt_unpack_from_host): ms per request including the host
    link, against the 26 GB/s GPU-to-CPU figure of the paper's simulator."""
    dev = torch.device("cuda:0")
    out = {}
    # ---------------------------------------------------------- decode side
    w = W.c2_llama8b()
    sh = w.shape
    S = w.num_steps
    rb = sh.token_row_bytes
    rows = np.array([w.step_tokens(k) for k in range(S)], np.int64)
    g = torch.Generator(device=dev)
    g.manual_seed(2)
    src = torch.empty(sh.pool_elems(w.num_blocks), dtype=torch.bfloat16,
                      device=dev)
    src.normal_(generator=g)
    bt = torch.from_numpy(w.block_tables).to(dev)
    starts = [torch.from_numpy(a).to(dev) for a in w.starts]
    ends = [torch.from_numpy(a).to(dev) for a in w.ends]
    attend = int(w.starts[0].astype(np.int64).sum()) * sh.token_row_elems
    attend = min(attend, src.numel())
    kv_view = src[:attend]
    staging = torch.empty(ring_slots * slot_rows * rb, dtype=torch.uint8,
                          device=dev)
    hosts = [torch.empty(int(rows.max()) * rb, dtype=torch.uint8,
                         pin_memory=True) for _ in range(host_slots)]
    wss = [kv.new_workspace(w.num_reqs, dev) for _ in range(host_slots)]
    pack_s, copy_s = torch.cuda.Stream(), torch.cuda.Stream()
    sink = torch.empty((), dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    link = host_link_rates(torch, hosts[0], staging)
    for h in hosts[1:]:  # first touch of every pinned slot, untimed
        n = min(h.numel(), staging.numel())
        h[:n].copy_(staging[:n])
    torch.cuda.synchronize()

    def decode_loop(ckpt):
        """ckpt: None (decode alone), "ring" (pack_to_host through the
        staging ring and the copy engine) or "direct" (the gather writes
        pinned host memory itself)."""
        evs = [(torch.cuda.Event(enable_timing=True),
                torch.cuda.Event(enable_timing=True))
               for _ in range(decode_steps)]
        done = [None] * host_slots
        lat = []  # (issue, host copy complete) per checkpointed step
        c0, c1 = (torch.cuda.Event(enable_timing=True),
                  torch.cuda.Event(enable_timing=True))
        t0 = time.perf_counter()
        for i in range(decode_steps):
            evs[i][0].record()
            torch.sum(kv_view, dim=0, dtype=torch.float32, out=sink)
            evs[i][1].record()
            if ckpt:
                k, j = i % S, i % host_slots
                if done[j] is not None:
                    done[j].synchronize()  # the host drains slot j
                last = copy_s if ckpt == "ring" else pack_s
                if i == 0:
                    c0.record(last)
                issued = torch.cuda.Event(enable_timing=True)
                issued.record(pack_s)
                kv.lumen_kv_ckpt_plan(starts[k], ends[k], wss[j],
                                      stream=pack_s)
                if ckpt == "ring":
                    kv.lumen_kv_ckpt_pack_to_host(
                        sh, w.num_blocks, src, bt, wss[j], int(rows[k]),
                        staging, ring_slots, hosts[j], pack_stream=pack_s,
                        copy_stream=copy_s)
                else:
                    kv.lumen_kv_ckpt_pack_to_host_direct(
                        sh, w.num_blocks, src, bt, wss[j], hosts[j],
                        stream=pack_s)
                ev = torch.cuda.Event(enable_timing=True)
                ev.record(last)
                done[j] = ev
                lat.append((issued, ev, int(rows[k])))
        t_issue = time.perf_counter() - t0
        if ckpt:
            c1.record(copy_s if ckpt == "ring" else pack_s)
        torch.cuda.synchronize()
        t_all = time.perf_counter() - t0
        ms = np.array([a.elapsed_time(b) for a, b in evs])
        res = {"decode_ms_mean": float(ms.mean()),
               "decode_ms_median": float(np.median(ms)),
               "wall_ms": t_all * 1e3, "issue_ms": t_issue * 1e3}
        if ckpt:
            for ws in wss:
                assert kv.lumen_kv_ckpt_status(ws, stream=pack_s) == 0
            res["ckpt_span_ms"] = c0.elapsed_time(c1)
            res["ckpt_bytes"] = float(sum(rows[i % S] for i in
                                          range(decode_steps)) * rb)
            res["ckpt_latency_ms"] = np.array([a.elapsed_time(b)
                                               for a, b, _ in lat])
            res["ckpt_step_bytes"] = np.array([n * rb for _, _, n in lat],
                                              np.float64)
        return res

    def last_step_ok():
        """The last step's host copy against the device rows of that step."""
        k = (decode_steps - 1) % S
        j = (decode_steps - 1) % host_slots
        ws = kv.new_workspace(w.num_reqs, dev)
        kv.lumen_kv_ckpt_plan(starts[k], ends[k], ws)
        back = torch.empty(int(rows[k]) * rb, dtype=torch.uint8, device=dev)
        kv.lumen_kv_ckpt_pack(sh, w.num_blocks, src, bt, ws,
                              back.view(torch.bfloat16))
        ok = bool(torch.equal(back.cpu(), hosts[j][:back.numel()]))
        assert kv.lumen_kv_ckpt_status(ws) == 0
        for h in hosts:
            h.zero_()
        return ok

    decode_loop(None)  # warm-up
    alone = decode_loop(None)
    decode_GBps = gb(kv_view.numel() * 2) / (alone["decode_ms_mean"] / 1e3)
    for mode in ("ring", "direct"):
        withc = decode_loop(mode)
        ok = last_step_ok()
        key = ("decode_with_checkpoint" if mode == "ring"
               else "decode_with_checkpoint_direct")
        out[key] = {
            "workload": w.name, "decode_steps": decode_steps,
            "decode_standin": "one HBM-bound pass over the KV of the batch "
                              f"({gb(kv_view.numel() * 2):.1f} GB) per step",
            "decode_standin_GBps": decode_GBps,
            "decode_ms_alone": alone["decode_ms_mean"],
            "decode_ms_with_checkpoint": withc["decode_ms_mean"],
            "decode_slowdown": withc["decode_ms_mean"]
            / alone["decode_ms_mean"],
            "wall_ms_alone": alone["wall_ms"],
            "wall_ms_with_checkpoint": withc["wall_ms"],
            "checkpoint_GB": gb(withc["ckpt_bytes"]),
            "checkpoint_latency_ms_mean":
                float(withc["ckpt_latency_ms"].mean()),
            "checkpoint_latency_ms_max":
                float(withc["ckpt_latency_ms"].max()),
            "checkpoint_step_GBps": gb(withc["ckpt_step_bytes"].sum())
            / (withc["ckpt_latency_ms"].sum() / 1e3),
            "d2h_link_GBps": link["d2h"],
            "path": (f"staging ring {ring_slots} x {slot_rows} rows "
                     f"({ring_slots * slot_rows * rb / 2**20:.0f} MiB) "
                     "+ copy engine" if mode == "ring" else
                     "gather writes pinned host memory (64 workgroups)"),
            "host_copy_ok": ok}
    del src, kv_view, staging, hosts
    torch.cuda.empty_cache()
    # --------------------------------------------------------- restore side
    w = W.c3_restore()
    sh = w.shape
    rb = sh.token_row_bytes
    ctx = w.ends[0].astype(np.int64)
    waves = W.restore_waves(w)
    pool = torch.zeros(sh.pool_elems(w.dst_num_blocks), dtype=torch.bfloat16,
                       device=dev)
    big = int(ctx.max())
    host = torch.empty(big * rb, dtype=torch.uint8, pin_memory=True)
    fill = torch.empty(big * sh.token_row_elems, dtype=torch.bfloat16,
                       device=dev)
    fill.normal_(generator=g)
    host.copy_(fill.view(torch.uint8))
    del fill
    staging = torch.empty(ring_slots * slot_rows * rb, dtype=torch.uint8,
                          device=dev)
    cs, us = torch.cuda.Stream(), torch.cuda.Stream()
    ws = kv.new_workspace(1, dev)
    torch.cuda.synchronize()
    # plain copies first: the link's rate, and the first touch of the
    # freshly pinned buffer stays out of the timed restores
    link = host_link_rates(torch, host, staging)

    def restores(mode):
        """Every request restored from `host`, one call each, through the
        staging ring ("ring") or with the scatter reading host memory
        ("direct"); ms per request."""
        per_ms = []
        pool.zero_()
        for wv in waves:
            bt = torch.from_numpy(w.dst_block_tables[wv]).to(dev)
            s_w = torch.from_numpy(w.starts[0][wv]).to(dev)
            e_w = torch.from_numpy(w.ends[0][wv]).to(dev)
            torch.cuda.synchronize()
            for i, r in enumerate(wv):
                a = torch.cuda.Event(enable_timing=True)
                b = torch.cuda.Event(enable_timing=True)
                bt_r = bt[i:i + 1]  # a view: nothing for side streams to outlive
                kv.lumen_kv_ckpt_plan(s_w[i:i + 1], e_w[i:i + 1], ws,
                                      stream=us)
                a.record(us)
                if mode == "ring":
                    cs.wait_stream(us)
                    kv.lumen_kv_ckpt_unpack_from_host(
                        sh, w.dst_num_blocks, pool, bt_r, ws, int(ctx[r]),
                        host, staging, ring_slots, copy_stream=cs,
                        unpack_stream=us)
                else:
                    kv.lumen_kv_ckpt_unpack_from_host_direct(
                        sh, w.dst_num_blocks, pool, bt_r, ws, host,
                        row_end=int(ctx[r]), stream=us)
                b.record(us)
                b.synchronize()
                per_ms.append(a.elapsed_time(b))
                assert kv.lumen_kv_ckpt_status(ws, stream=us) == 0
        # the last request, packed back from the pool, against the host bytes
        r = int(waves[-1][-1])
        ws2 = kv.new_workspace(1, dev)
        kv.lumen_kv_ckpt_plan(torch.from_numpy(w.starts[0][[r]]).to(dev),
                              torch.from_numpy(w.ends[0][[r]]).to(dev), ws2)
        n = min(int(ctx[r]), 512)
        back = torch.empty(int(ctx[r]) * rb, dtype=torch.uint8, device=dev)
        kv.lumen_kv_ckpt_pack(sh, w.dst_num_blocks, pool,
                              torch.from_numpy(w.dst_block_tables[[r]]).to(dev),
                              ws2, back.view(torch.bfloat16))
        ok = bool(torch.equal(back[:n * rb].cpu(), host[:n * rb]))
        assert kv.lumen_kv_ckpt_status(ws2) == 0
        return np.array(per_ms), ok

    req_b = ctx * rb
    for mode in ("ring", "direct"):
        per_ms, ok = restores(mode)
        key = "restore_from_host" if mode == "ring" else \
            "restore_from_host_direct"
        out[key] = {
            "workload": w.name, "requests": int(len(per_ms)),
            "h2d_link_GBps": link["h2d"],
            "restore_ms_per_request": float(per_ms.mean()),
            "restore_ms_per_request_median": float(np.median(per_ms)),
            "h2d_GBps": gb(float(req_b.sum())) / (per_ms.sum() / 1e3),
            "model_ms_per_request_at_26GBps":
                float(gb(req_b.mean()) / 26 * 1e3),
            "path": (f"staging ring {ring_slots} x {slot_rows} rows "
                     f"({ring_slots * slot_rows * rb / 2**20:.0f} MiB) "
                     "+ copy engine" if mode == "ring" else
                     "scatter reads pinned host memory (64 workgroups)"),
            "spot_check_ok": ok}
    del pool, host, staging
    torch.cuda.empty_cache()
    return out


def tags_leg(W):
    """Host side of recovery (no GPU): tags of every complete page of the
    decode workload's contexts, and longest-prefix lookups for the 64
    restore-burst requests against a store holding all their pages."""
    from paper_2606_17787_amd import tags as T
    rng = np.random.default_rng(11)
    w = W.c2_llama8b()
    bs = w.shape.block_size
    hists = [rng.integers(0, 128256, int(n)).astype(np.int32)
             for n in w.starts[0]]
    pages = sum(len(h) // bs for h in hists)
    t0 = time.perf_counter()
    for h in hists:
        T.lumen_page_tags(h, bs)
    t_tags = time.perf_counter() - t0
    out = {"tags_pages": pages, "tags_ms": t_tags * 1e3,
           "tags_Mpages_per_s": pages / t_tags / 1e6}
    w = W.c3_restore()
    bs = w.shape.block_size
    store = T.TagStore(bs)
    hists = [rng.integers(0, 128256, int(n)).astype(np.int32)
             for n in w.ends[0]]
    for r, h in enumerate(hists):
        store.publish_pages(r, h, 0, len(h) // bs)
    t0 = time.perf_counter()
    got = [store.longest_prefix(r, h) for r, h in enumerate(hists)]
    t_look = time.perf_counter() - t0
    store.close()
    assert got == [(len(h) // bs) * bs for h in hists]
    out.update(lookup_requests=len(hists),
               lookup_pages=sum(len(h) // bs for h in hists),
               lookup_ms_per_request=t_look * 1e3 / len(hists))
    return out


def sched_leg():
    """Host side of placement and recovery (no GPU): Eq. 1 placement of
    100,000 requests (4,000 active at a time, reserved footprints of
    2K-16K Llama-3-8B-shaped tokens) over 64 workers with 80 GB checkpoint
    budgets, then a recovery event that fails one worker and one that
    fails four."""
    from paper_2606_17787_amd.sched import Scheduler
    rng = np.random.default_rng(12)
    nw, nreq = 64, 100_000
    row = 131072  # Llama-3-8B-shaped token row, bytes
    s = Scheduler([80 * 10**9] * nw, 26e9, 1.0)
    for w in range(nw):
        s.set_worker(w, float(rng.random() * 0.5), int(rng.integers(0, 8)),
                     int(rng.integers(16, 64)))
    serving = rng.integers(0, nw, nreq)
    foot = rng.integers(2048, 16385, nreq) * row  # from max context
    t0 = time.perf_counter()
    live, protected = [], 0
    for r in range(nreq):
        protected += s.place(r, int(serving[r]), int(foot[r])) >= 0
        live.append(r)
        if len(live) > 4000:  # requests complete: keep 4000 active
            s.release(live.pop(0))
    t_place = time.perf_counter() - t0
    for r in live:
        s.set_persisted(r, int(rng.integers(0, foot[r])))
    t0 = time.perf_counter()
    one = s.recover([5])
    t_one = time.perf_counter() - t0
    t0 = time.perf_counter()
    four = s.recover([9, 17, 33, 60])
    t_four = time.perf_counter() - t0
    s.close()
    return {"workers": nw, "placements": nreq, "active_requests": 4000,
            "placed_with_holder": int(protected),
            "place_us": t_place / nreq * 1e6,
            "recover_1_failure_interrupted": len(one),
            "recover_1_failure_ms": t_one * 1e3,
            "recover_1_failure_reuse": sum(1 for x in one if x[2]),
            "recover_4_failures_interrupted": len(four),
            "recover_4_failures_ms": t_four * 1e3}


def draft_leg(torch, kv, reps=50):
    """Draft-state alignment for a paired worker's batch: 1,024 mirror
    requests with 1-4K-token histories and K = 4 draft tokens each, of
    which a random number (0-4) were accepted before the correction; block
    size 16.  Times lumen_kv_draft_align with HIP events."""
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(13)
    R, K, bs = 1024, 4, 16
    hist = rng.integers(1024, 4097, R)
    cols = int(hist.max()) + K + 1
    base = rng.integers(0, 128256, (R, cols)).astype(np.int32)
    draft = base.copy()
    committed = base.copy()
    acc = rng.integers(0, K + 1, R)
    for r in range(R):  # committed: history + accepted drafts + correction
        committed[r, hist[r] + acc[r]] = -1 - int(rng.integers(0, 1000))
    dl = (hist + K).astype(np.int32)
    cl = (hist + acc + 1).astype(np.int32)
    btc = -(-cols // bs)
    bt = np.arange(R * btc, dtype=np.int32).reshape(R, btc)
    d = {k: torch.from_numpy(v).to(dev) for k, v in dict(
        draft=draft, committed=committed, dl=dl, cl=cl, bt=bt).items()}
    kl0 = torch.from_numpy(dl.copy()).to(dev)
    kl = kl0.clone()
    tab = d["bt"].clone()
    replay = torch.empty(R, dtype=torch.int32, device=dev)
    freed = torch.empty(R * 2, dtype=torch.int32, device=dev)
    cnt = torch.empty(1, dtype=torch.int64, device=dev)
    ws = kv.new_workspace(R, dev)
    ts = []
    for i in range(reps + 5):
        kl.copy_(kl0)
        tab.copy_(d["bt"])
        a = TimingEvent()
        b = TimingEvent()
        a.record()
        kv.lumen_kv_draft_align(d["draft"], d["dl"], d["committed"], d["cl"],
                                kl, tab, bs, replay, freed, cnt, ws)
        b.record()
        b.synchronize()
        if i >= 5:
            ts.append(a.elapsed_time(b))
    assert kv.lumen_kv_ckpt_status(ws) == 0
    ok = bool((kl.cpu().numpy() == hist + acc).all()
              and (replay.cpu().numpy() == 1).all())
    return {"requests": R, "draft_depth": K, "block_size": bs,
            "history_tokens_mean": float(hist.mean()),
            "align_us_mean": float(np.mean(ts) * 1e3),
            "align_us_median": float(np.median(ts) * 1e3),
            "freed_blocks": int(cnt.item()), "check_ok": ok}


def small_steps_leg(torch, kv, W, sizes=(8, 32, 64, 128), steps=20):
    """Decode steps of the first R requests of the Llama-3-8B-shaped
    workload (R = 8 .. 128), as one-launch range copies.  A copy's grid is
    sized by its checkpoint buffer's rows, so each step runs twice: into a
    buffer of exactly its rows (what a caller that knows its step's token
    count passes), and into the whole 20-region arena at the region's row
    (as the headline loop does).  Median us per pack and unpack from
    stamped events; the two placements of each step's rows are checked to
    hold the same bytes."""
    dev = torch.device("cuda:0")
    w = W.c2_llama8b()
    sh = w.shape
    NR, lag = 20, 10
    re_ = sh.token_row_elems
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    src = torch.empty(sh.pool_elems(w.num_blocks), dtype=torch.bfloat16,
                      device=dev)
    src.normal_(generator=g)
    dst = torch.zeros(sh.pool_elems(w.dst_num_blocks), dtype=torch.bfloat16,
                      device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    out = {}
    for R in sizes:
        st = [torch.from_numpy(np.ascontiguousarray(a[:R])).to(dev)
              for a in w.starts[:NR]]
        en = [torch.from_numpy(np.ascontiguousarray(a[:R])).to(dev)
              for a in w.ends[:NR]]
        bt = torch.from_numpy(np.ascontiguousarray(w.block_tables[:R])).to(dev)
        bt2 = torch.from_numpy(
            np.ascontiguousarray(w.dst_block_tables[:R])).to(dev)
        rows = [int((w.ends[k][:R].astype(np.int64) - w.starts[k][:R]).sum())
                for k in range(NR)]
        stride = max(rows)
        arena = torch.empty(NR * stride * re_, dtype=torch.bfloat16,
                            device=dev)
        for k in range(NR):
            kv.lumen_kv_ckpt_pack_ranges(sh, w.num_blocks, src, bt, st[k],
                                         en[k], arena, status, k * stride)

        def region(k):
            return arena[k * stride * re_:(k * stride + rows[k]) * re_]

        def step(i, tight, ev):
            k, k2 = i % NR, (i + lag) % NR
            stamp(ev[0], ev[1])
            if tight:
                kv.lumen_kv_ckpt_pack_ranges(sh, w.num_blocks, src, bt, st[k],
                                             en[k], region(k), status)
            else:
                kv.lumen_kv_ckpt_pack_ranges(sh, w.num_blocks, src, bt, st[k],
                                             en[k], arena, status, k * stride)
            stamp(ev[2], ev[3])
            if tight:
                kv.lumen_kv_ckpt_unpack_ranges(sh, w.dst_num_blocks, dst, bt2,
                                               st[k2], en[k2], region(k2),
                                               status)
            else:
                kv.lumen_kv_ckpt_unpack_ranges(sh, w.dst_num_blocks, dst, bt2,
                                               st[k2], en[k2], arena, status,
                                               k2 * stride)
            return k, k2

        res = {}
        for tight in (True, False):
            for i in range(4):
                step(i, tight, [TimingEvent() for _ in range(4)])
            evs = [[TimingEvent() for _ in range(4)] for _ in range(steps)]
            done = [step(i, tight, evs[i]) for i in range(steps)]
            torch.cuda.synchronize()
            pk = [e[0].elapsed_time(e[1]) * 1e3 for e in evs]
            up = [e[2].elapsed_time(e[3]) * 1e3 for e in evs]
            byts = 2.0 * np.mean([rows[k] for k, _ in done]) * sh.token_row_bytes
            res["buffer_of_step_rows" if tight else "whole_arena"] = dict(
                pack_us_median=float(np.median(pk)),
                unpack_us_median=float(np.median(up)),
                pack_GBps=gb(byts) / (float(np.median(pk)) / 1e6))
        if int(status.item()) != 0:
            raise RuntimeError("small steps reported "
                               f"{kv.lumen_kv_ckpt_strerror(int(status.item()))}")
        # both buffers receive the same rows: pack step 0 both ways
        kv.lumen_kv_ckpt_pack_ranges(sh, w.num_blocks, src, bt, st[0], en[0],
                                     arena, status, 0)
        a = region(0).clone()
        region(0).zero_()
        kv.lumen_kv_ckpt_pack_ranges(sh, w.num_blocks, src, bt, st[0], en[0],
                                     region(0), status)
        res["same_rows"] = bool(torch.equal(a.view(torch.int16),
                                            region(0).view(torch.int16)))
        res["rows_per_step_mean"] = float(np.mean(rows))
        out[str(R)] = res
        del arena, a
    torch.cuda.empty_cache()
    return out


def tiny_leg(torch, kv, W, reps=200):
    """The tiny full-pack workload (2 layers, 2 KV heads, head_dim 64,
    block 16; 8 requests, 1,729 tokens, 1.77 MB each way) is launch-bound,
    so it reports latency: device us of plan + pack and of plan + unpack
    from HIP events around each pair with the stream drained in between,
    the same pairs back to back, and the host cost of enqueueing one call
    through the binding, also with the calls prepared once (PreparedCall),
    and the one-launch range copies prepared the same way, alone and as a
    round trip, issued eagerly or replayed from a HIP graph.  Self-check:
    the restored tokens, packed again from the destination pool, equal the
    checkpoint (also after one graph replay)."""
    dev = torch.device("cuda:0")
    w = W.c1_tiny()
    sh = w.shape
    rows = w.step_tokens(0)
    src = torch.from_numpy(W.random_bits(np.random.default_rng(1),
                                         sh.pool_elems(w.num_blocks))
                           .view(np.int16)).to(dev)
    dst = torch.zeros(sh.pool_elems(w.dst_num_blocks), dtype=torch.int16,
                      device=dev)
    ck = torch.empty(rows * sh.token_row_elems, dtype=torch.int16, device=dev)
    back = torch.empty_like(ck)
    bt = torch.from_numpy(w.block_tables).to(dev)
    bt2 = torch.from_numpy(w.dst_block_tables).to(dev)
    s = torch.from_numpy(w.starts[0]).to(dev)
    e = torch.from_numpy(w.ends[0]).to(dev)
    ws = kv.new_workspace(w.num_reqs, dev)

    def pack():
        kv.lumen_kv_ckpt_plan(s, e, ws)
        kv.lumen_kv_ckpt_pack(sh, w.num_blocks, src, bt, ws, ck)

    def unpack():
        kv.lumen_kv_ckpt_plan(s, e, ws)
        kv.lumen_kv_ckpt_unpack(sh, w.dst_num_blocks, dst, bt2, ws, ck)

    def pair_us(fn):
        out = []
        for i in range(reps + 20):
            a = TimingEvent()
            b = TimingEvent()
            a.record()
            fn()
            b.record()
            b.synchronize()
            if i >= 20:
                out.append(a.elapsed_time(b) * 1e3)
        return out

    pk, up = pair_us(pack), pair_us(unpack)
    # the same calls prepared once: checks and marshalling outside the loop
    p_plan = kv.prepare_plan(s, e, ws)
    p_pack = kv.prepare_pack(sh, w.num_blocks, src, bt, ws, ck)
    p_unpack = kv.prepare_unpack(sh, w.dst_num_blocks, dst, bt2, ws, ck)

    def pack_prepared():
        p_plan()
        p_pack()

    def unpack_prepared():
        p_plan()
        p_unpack()

    pk_p, up_p = pair_us(pack_prepared), pair_us(unpack_prepared)
    # one launch per copy, planning from the ranges (prepared the same way)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    p_rpack = kv.prepare_pack_ranges(sh, w.num_blocks, src, bt, s, e, ck,
                                     status)
    p_runpack = kv.prepare_unpack_ranges(sh, w.dst_num_blocks, dst, bt2, s,
                                         e, ck, status)
    pk_r, up_r = pair_us(p_rpack), pair_us(p_runpack)

    # the round trip (pack, then unpack, one launch each) eagerly, and
    # captured once in a HIP graph and replayed: one host call per trip
    def roundtrip_ranges():
        p_rpack()
        p_runpack()

    rt_eager = pair_us(roundtrip_ranges)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        roundtrip_ranges()
    torch.cuda.synchronize()
    rt_graph = pair_us(graph.replay)
    # the replay's own result: a cleared checkpoint and pool, one replay,
    # then the restored tokens packed again must equal the checkpoint
    ck.zero_()
    dst.zero_()
    torch.cuda.synchronize()
    graph.replay()
    torch.cuda.synchronize()
    kv.lumen_kv_ckpt_plan(s, e, ws)
    kv.lumen_kv_ckpt_pack(sh, w.dst_num_blocks, dst, bt2, ws, back)
    graph_ok = bool(torch.equal(back, ck)) and bool(ck.any())
    assert kv.lumen_kv_ckpt_status(ws) == 0
    del graph
    if int(status.item()) != 0:
        raise RuntimeError("range copies reported "
                           f"{kv.lumen_kv_ckpt_strerror(int(status.item()))}")
    torch.cuda.synchronize()
    a = TimingEvent()
    b = TimingEvent()
    a.record()
    for _ in range(reps):
        pack()
        unpack()
    b.record()
    b.synchronize()
    rt_us = a.elapsed_time(b) * 1e3 / reps
    # host cost of one enqueue (binding + C ABI), the stream left to run
    t0 = time.perf_counter()
    for _ in range(reps):
        kv.lumen_kv_ckpt_pack(sh, w.num_blocks, src, bt, ws, ck)
    host_us = (time.perf_counter() - t0) * 1e6 / reps
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        p_pack()
    host_p_us = (time.perf_counter() - t0) * 1e6 / reps
    torch.cuda.synchronize()
    assert kv.lumen_kv_ckpt_status(ws) == 0
    kv.lumen_kv_ckpt_plan(s, e, ws)
    kv.lumen_kv_ckpt_pack(sh, w.dst_num_blocks, dst, bt2, ws, back)
    ok = bool(torch.equal(back, ck))
    assert kv.lumen_kv_ckpt_status(ws) == 0
    byts = 2.0 * rows * sh.token_row_bytes
    return {"workload": w.name, "requests": w.num_reqs, "tokens": rows,
            "bytes_each_way": rows * sh.token_row_bytes,
            "plan_pack_us_median": float(np.median(pk)),
            "plan_unpack_us_median": float(np.median(up)),
            "plan_pack_us_p10_p90": [float(np.percentile(pk, q))
                                     for q in (10, 90)],
            "back_to_back_roundtrip_us": rt_us,
            "back_to_back_GBps": gb(2 * byts) / (rt_us / 1e6),
            "host_enqueue_us_per_call": host_us,
            "prepared_plan_pack_us_median": float(np.median(pk_p)),
            "prepared_plan_unpack_us_median": float(np.median(up_p)),
            "prepared_host_enqueue_us_per_call": host_p_us,
            "prepared_ranges_pack_us_median": float(np.median(pk_r)),
            "prepared_ranges_unpack_us_median": float(np.median(up_r)),
            "ranges_roundtrip_us_median": float(np.median(rt_eager)),
            "graph_ranges_roundtrip_us_median": float(np.median(rt_graph)),
            "graph_roundtrip_ok": graph_ok,
            "roundtrip_ok": ok}


def calibrate_copy(torch, mib):
    """A plain device-to-device copy of known size: read + write bytes are
    exactly 2 * mib MiB per launch, the scale for the FETCH_SIZE/WRITE_SIZE
    counters of the checkpoint kernels."""
    n = mib << 20
    a = torch.empty(n // 2, dtype=torch.int16, device="cuda")
    a.fill_(1)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / 5
    print(json.dumps({"calibration_copy_bytes": n,
                      "copy_GBps": round(2 * n / dt / 1e9, 1)}), flush=True)


# ------------------------------------------------------------ CPU baseline

def cpu_threads():
    """Host threads the oracle may use: the process's CPU affinity, capped
    by OMP_NUM_THREADS when the environment sets it (the GPU machine's share)."""
    n = len(os.sched_getaffinity(0))
    cap = os.environ.get("OMP_NUM_THREADS")
    return max(1, min(n, int(cap))) if cap and cap.isdigit() else n


def cpu_baseline(W, seconds):
    """The CPU oracle (plain loops) on a bounded sample of the same decode
    workload: whole steps packed from a host pool holding only the blocks
    those steps read, until the time budget is spent.  First on one thread,
    then with the requests of each step split over the host's threads (the
    oracle's C code runs outside the interpreter lock); the threaded figure
    is the baseline."""
    import oracle
    from concurrent.futures import ThreadPoolExecutor
    w = W.c2_llama8b()
    sh = w.shape
    bs = sh.block_size
    tables = []
    for k in range(w.num_steps):
        s, e = w.starts[k], w.ends[k]
        pages = []
        for r in range(w.num_reqs):
            pages += [int(w.block_tables[r, j]) for j in
                      range(int(s[r]) // bs, (int(e[r]) - 1) // bs + 1)]
        remap = {b: i for i, b in enumerate(pages)}
        bt = np.full_like(w.block_tables, -1)
        for r in range(w.num_reqs):
            for j in range(int(s[r]) // bs, (int(e[r]) - 1) // bs + 1):
                bt[r, j] = remap[int(w.block_tables[r, j])]
        tables.append((len(pages), bt))
    nb = max(n for n, _ in tables)
    pool = W.random_bits(np.random.default_rng(0), sh.pool_elems(nb))
    lib = oracle.load()

    def run(threads, budget):
        bounds = np.linspace(0, w.num_reqs, threads + 1).astype(int)
        done_b, done_t, n_steps = 0.0, 0.0, 0
        with ThreadPoolExecutor(threads) as ex:
            for k, (n, bt) in enumerate(tables):
                s, e = w.starts[k], w.ends[k]
                lens = (e.astype(np.int64) - s)
                first = np.concatenate([[0], np.cumsum(lens)])
                ck = np.empty((int(first[-1]), sh.token_row_elems), np.uint16)

                def part(i):
                    r0, r1 = bounds[i], bounds[i + 1]
                    return oracle.pack(sh, nb, pool, bt[r0:r1], s[r0:r1],
                                       e[r0:r1], row_base=int(first[r0]),
                                       ckpt=ck, lib=lib)[0]
                t0 = time.perf_counter()
                sts = list(ex.map(part, range(threads)))
                done_t += time.perf_counter() - t0
                assert all(x == 0 for x in sts)
                done_b += 2.0 * w.step_tokens(k) * sh.token_row_bytes
                n_steps += 1
                if done_t > budget:
                    break
        return gb(done_b) / done_t, n_steps, done_b

    one, n1, b1 = run(1, seconds / 2)
    threads = cpu_threads()
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    many, n2, b2 = run(threads, seconds / 2)
    return {"value": round(many, 4), "unit": "GB/s", "cores": threads,
            "kind": "oracle",
            "sample": f"pack of decode steps 0..{n2 - 1} of the "
                      f"Llama-3-8B-shaped workload ({gb(b2):.2f} GB read+"
                      "written) from a compact host pool of the blocks those "
                      f"steps read, requests split over {threads} threads",
            "cpu_model": model,
            "single_thread_value": round(one, 4),
            "single_thread_sample": f"decode steps 0..{n1 - 1} "
                                    f"({gb(b1):.2f} GB)"}


# -------------------------------------------------------------------- main

TRAFFIC_FILE = os.path.join(ROOT, "profiles",
                            "copy_rows_kernel_llama3-8b-decode_hbm_traffic.txt")
KERNEL_SRC = os.path.join(ROOT, "paper_2606_17787_amd", "csrc",
                          "lumen_kv_ckpt.hip")


def device_code_sha256(path=KERNEL_SRC):
    """sha256 of the device code of the library source: the text from the
    opening of its anonymous namespace up to the marker line that starts
    the host side (kernels, their helpers and tuning constants), with
    comments removed and runs of whitespace folded to one space, so that
    editing a comment does not count as changing the code."""
    import hashlib
    import re
    text = open(path, "rb").read()
    a = text.index(b"namespace {")
    b = text.index(b"// " + b"-" * 61 + b" host side")
    code = text[a:b].decode()
    code = re.sub(r"/\*.*?\*/", " ", code, flags=re.S)
    code = re.sub(r"//[^\n]*", " ", code)
    code = " ".join(code.split())
    return hashlib.sha256(code.encode()).hexdigest()


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed FETCH_SIZE /
    WRITE_SIZE counter runs, or None once the device code has changed since
    those counters were taken."""
    try:
        text = open(TRAFFIC_FILE).read()
        data = json.loads(text[text.index("{", text.index("Machine-readable")):])
        sha = device_code_sha256()
    except (OSError, ValueError):
        return None
    if data.get("device_code_sha256") != sha:
        return None
    return data["llama3-8b-decode"][kernel]["traffic_bytes"]


def rounded(d):
    def r(v):
        if isinstance(v, float):
            return round(v, 4)
        if isinstance(v, list):
            return [r(x) for x in v]
        if isinstance(v, dict):
            return {k: r(x) for k, x in v.items()}
        return v
    return {k: r(v) for k, v in d.items()}


def environment(torch):
    """GPU, runtime and library versions of the run."""
    props = torch.cuda.get_device_properties(0)
    rocm = None
    try:
        with open("/opt/rocm/.info/version") as f:
            rocm = f.read().strip()
    except OSError:
        pass
    return {"gpu": torch.cuda.get_device_name(0),
            "arch": getattr(props, "gcnArchName", None),
            "cus": props.multi_processor_count,
            "hbm_GiB": round(props.total_memory / 2**30, 1),
            "rocm": rocm, "hip": torch.version.hip,
            "torch": torch.__version__, "numpy": np.__version__}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the "
              "checkpoint path has no cross-GPU exchange; run it with "
              "--gpus 1", file=sys.stderr)
        sys.exit(2)
    legs = set(args.legs.split(","))
    import torch
    import paper_2606_17787_amd.kvckpt as kv
    from paper_2606_17787_amd import workloads as W
    torch.cuda.set_device(0)
    if args.calibrate_copy_mib:
        calibrate_copy(torch, args.calibrate_copy_mib)
        return
    kv.load_library()

    say("[bench] decode leg (llama3-8b-decode)")
    w = W.c2_llama8b()
    dec = incremental_leg(torch, kv, w, args.steps, args.warmup, seed=2,
                          placements=args.placements, regions=20,
                          path="ranges", compare="plan",
                          per_request_path="plan")
    dominant = ("pack" if dec["pack_us_mean"] >= dec["unpack_us_mean"]
                else "unpack")
    achieved = dec[f"{dominant}_GBps"]
    out = {
        "metric": METRIC, "value": round(dec["step_GBps"], 1), "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(dec["ms_per_step"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "layers": w.shape.num_layers,
                   "kv_heads": w.shape.num_kv_heads,
                   "head_dim": w.shape.head_dim,
                   "block_size": w.shape.block_size,
                   "cache_layout": w.shape.order, "requests": w.num_reqs,
                   "tokens_per_step_mean": dec["tokens_per_step_mean"],
                   "step": "pack of step k, unpack of step k+10 (20 "
                           "checkpoint regions per arena), each one launch "
                           "that plans from the token ranges itself",
                   "placements": dec["placements"],
                   "fingerprint": dec["fingerprint"],
                   "parallelism": "none (1 GPU)"},
        "env": environment(torch),
        "pack_GBps": round(dec["pack_GBps"], 1),
        "unpack_GBps": round(dec["unpack_GBps"], 1),
        "pack_pct_peak": round(dec["pack_pct_peak"], 2),
        "unpack_pct_peak": round(dec["unpack_pct_peak"], 2),
        "pack_us_mean": round(dec["pack_us_mean"], 2),
        "unpack_us_mean": round(dec["unpack_us_mean"], 2),
        "pack_us_median": round(dec["pack_us_median"], 2),
        "unpack_us_median": round(dec["unpack_us_median"], 2),
        "pack_us_p10_p90": [round(x, 2) for x in dec["pack_us_p10_p90"]],
        "unpack_us_p10_p90": [round(x, 2) for x in dec["unpack_us_p10_p90"]],
        "kernel_samples": dec["sampled_steps"],
        "placement": rounded({k: dec[k] for k in (
            "pack_placement_worst_GBps", "pack_placement_median_GBps",
            "pack_placement_worst_pct_peak", "unpack_placement_worst_GBps",
            "unpack_placement_median_GBps", "unpack_placement_worst_pct_peak",
            "per_placement") if k in dec}),
        "roundtrip_ok": dec["roundtrip_ok"],
        "per_request_mode": rounded(dec["per_request_mode"]),
        "other_path": rounded(dec["other_path"]),
        "roofline": {"bound": "hbm",
                     "kernel": "copy_rows_kernel<%s, false, RangeWalk> (%s)"
                               % ("true" if dominant == "pack" else "false",
                                  dominant),
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "bytes_per_launch": dec[f"{dominant}_bytes_mean"],
                     "us_per_launch": round(dec[f"{dominant}_us_mean"], 2),
                     "traffic": measured_traffic(dominant)},
        "workloads": {},
    }
    if "tiny" in legs:
        say("[bench] tiny leg (latency)")
        out["workloads"]["tiny"] = rounded(tiny_leg(torch, kv, W))
    if "small" in legs:
        say("[bench] small decode steps leg")
        out["workloads"]["small-decode-steps"] = rounded(
            small_steps_leg(torch, kv, W))
    if "qwen" in legs:
        say("[bench] decode leg (qwen-gqa-hnd)")
        q = W.c5_qwen_hnd()
        keep = {}
        out["workloads"]["qwen-gqa-hnd"] = rounded(incremental_leg(
            torch, kv, q, 64, 8, seed=5, keep=keep))
        # the same requests and tables over a token-major cache, on the same
        # buffers: the difference is what the head-major transpose costs
        twin = dataclasses.replace(
            q, name="qwen-gqa-nhd-twin",
            shape=dataclasses.replace(q.shape, order="NHD"))
        say("[bench] decode leg (qwen-gqa-nhd-twin)")
        out["workloads"]["qwen-gqa-nhd-twin"] = rounded(incremental_leg(
            torch, kv, twin, 64, 8, seed=5, keep=keep))
        keep.clear()
        torch.cuda.empty_cache()
    if "restore" in legs:
        say("[bench] restore leg")
        res = restore_leg(torch, kv, W)
        out["restore_ms_per_request"] = round(res["restore_ms_per_request"], 4)
        out["workloads"]["restore-burst"] = rounded(res)
    if "tp8" in legs:
        say("[bench] tp8-shard leg")
        out["workloads"]["llama3-70b-tp8-shard"] = rounded(
            tp8_leg(torch, kv, W))
    if "stage" in legs:
        say("[bench] host staging leg")
        for k2, v2 in staging_leg(torch, kv, W).items():
            out["workloads"][k2] = rounded(v2)
    if "tags" in legs:
        say("[bench] page tags (host)")
        out["workloads"]["page-tags"] = rounded(tags_leg(W))
    if "sched" in legs:
        say("[bench] placement and recovery scheduling (host)")
        out["workloads"]["scheduler"] = rounded(sched_leg())
    if "draft" in legs:
        say("[bench] draft-state alignment")
        out["workloads"]["draft-align"] = rounded(draft_leg(torch, kv))
    if "cpu" in legs:
        say("[bench] cpu baseline")
        out["cpu_baseline"] = cpu_baseline(W, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
