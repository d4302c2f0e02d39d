#!/usr/bin/env python3
"""Benchmark of the paged-KV checkpoint path on one MI355X.

One step = the hot path over one decode step of the Llama-3-8B-shaped
workload (32 layers, 8 KV heads, head_dim 128, block 16, bf16; 256 requests
with lognormal contexts; each step checkpoints every request's newest 1-16
tokens):

    plan(step k)   -> pack(step k)   source pool -> checkpoint region k
    plan(step k')  -> unpack(step k') checkpoint region k' -> restore pool

with k' = k + 50 (mod 100), so the restore reads a region written 50 steps
(about 28 GB of traffic) earlier and cannot be served from the 256 MB
Infinity Cache.  Inputs (pools, block tables, ranges) are resident in HBM
before timing; the device error word is checked after the timed loop.

Printed: one JSON line with the whole-step throughput (pack + unpack bytes
read + written / wall time), per-kernel GB/s from HIP events on the launch
stream, the roofline fraction of the dominant kernel, the restore-burst leg
(ms per restored request), a device->pinned-host leg, and the CPU oracle
timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
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


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-restore", action="store_true",
                    help="skip the restore-burst leg")
    ap.add_argument("--no-offload", action="store_true",
                    help="skip the device->pinned-host leg")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="budget of the CPU oracle sample")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB "
                    "(5 times), the reference for HBM byte counters")
    return ap.parse_args()


def gb(x):
    return x / 1e9


# --------------------------------------------------------------- GPU legs

def decode_leg(torch, kv, W, steps, warmup):
    dev = torch.device("cuda:0")
    w = W.c2_llama8b()
    sh = w.shape
    S = w.num_steps
    rows = np.array([w.step_tokens(k) for k in range(S)], np.int64)
    row_off = np.concatenate([[0], np.cumsum(rows)])
    row_elems = sh.token_row_elems

    g = torch.Generator(device=dev)
    g.manual_seed(2)
    src = torch.empty(sh.pool_elems(w.num_blocks), dtype=torch.bfloat16,
                      device=dev)
    src.normal_(generator=g)
    dst = torch.zeros(sh.pool_elems(w.dst_num_blocks), dtype=torch.bfloat16,
                      device=dev)
    arena = torch.empty(int(row_off[-1]) * row_elems, dtype=torch.bfloat16,
                        device=dev)
    bt = torch.from_numpy(w.block_tables).to(dev)
    bt_dst = torch.from_numpy(w.dst_block_tables).to(dev)
    starts = [torch.from_numpy(a).to(dev) for a in w.starts]
    ends = [torch.from_numpy(a).to(dev) for a in w.ends]
    ws_a = kv.new_workspace(w.num_reqs, dev)
    ws_b = kv.new_workspace(w.num_reqs, dev)

    # Fill every checkpoint region once (also the first correctness gate).
    for k in range(S):
        kv.lumen_kv_ckpt_plan(starts[k], ends[k], ws_a, int(row_off[k]))
        kv.lumen_kv_ckpt_pack(sh, w.num_blocks, src, bt, ws_a, arena)
    st = kv.lumen_kv_ckpt_status(ws_a)
    if st != 0:
        raise RuntimeError(f"pack reported {kv.lumen_kv_ckpt_strerror(st)}")

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)]
          for _ in range(steps)]

    def step(i, events=None):
        k = i % S
        k2 = (k + S // 2) % S
        kv.lumen_kv_ckpt_plan(starts[k], ends[k], ws_a, int(row_off[k]))
        if events: events[0].record()
        kv.lumen_kv_ckpt_pack(sh, w.num_blocks, src, bt, ws_a, arena)
        if events: events[1].record()
        kv.lumen_kv_ckpt_plan(starts[k2], ends[k2], ws_b, int(row_off[k2]))
        if events: events[2].record()
        kv.lumen_kv_ckpt_unpack(sh, w.dst_num_blocks, dst, bt_dst, ws_b, arena)
        if events: events[3].record()
        return k, k2

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    done = [step(warmup + i, ev[i]) for i in range(steps)]
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    st = min(kv.lumen_kv_ckpt_status(ws_a), kv.lumen_kv_ckpt_status(ws_b))
    if st != 0:
        raise RuntimeError(f"device error {kv.lumen_kv_ckpt_strerror(st)}")

    rb = sh.token_row_bytes
    pack_b = np.array([2 * rows[k] * rb for k, _ in done], np.float64)
    unpack_b = np.array([2 * rows[k2] * rb for _, k2 in done], np.float64)
    pack_ms = np.array([e[0].elapsed_time(e[1]) for e in ev])
    unpack_ms = np.array([e[2].elapsed_time(e[3]) for e in ev])
    wall_ms = (t1 - t0) * 1e3

    # Round trip as a self-check (no oracle here): re-pack the restored
    # tokens of one step from the restore pool and compare with its region.
    k = done[-1][1]
    kv.lumen_kv_ckpt_plan(starts[k], ends[k], ws_b, 0)
    back = torch.empty(int(rows[k]) * row_elems, dtype=torch.bfloat16,
                       device=dev)
    kv.lumen_kv_ckpt_pack(sh, w.dst_num_blocks, dst, bt_dst, ws_b, back)
    region = arena[int(row_off[k]) * row_elems:int(row_off[k + 1]) * row_elems]
    roundtrip = bool(torch.equal(back.view(torch.int16),
                                 region.view(torch.int16)))
    assert kv.lumen_kv_ckpt_status(ws_b) == 0

    res = dict(
        workload=w, wall_ms=wall_ms, steps=steps,
        bytes_total=float(pack_b.sum() + unpack_b.sum()),
        pack_GBps=gb(pack_b.sum()) / (pack_ms.sum() / 1e3),
        unpack_GBps=gb(unpack_b.sum()) / (unpack_ms.sum() / 1e3),
        pack_us_median=float(np.median(pack_ms) * 1e3),
        unpack_us_median=float(np.median(unpack_ms) * 1e3),
        pack_us_mean=float(pack_ms.mean() * 1e3),
        unpack_us_mean=float(unpack_ms.mean() * 1e3),
        pack_bytes_mean=float(pack_b.mean()),
        unpack_bytes_mean=float(unpack_b.mean()),
        tokens_per_step_mean=float(rows.mean()),
        roundtrip_ok=roundtrip,
    )
    del src, dst, arena
    torch.cuda.empty_cache()
    return res


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
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            kv.lumen_kv_ckpt_plan(s, e, ws)
            a.record()
            kv.lumen_kv_ckpt_unpack(sh, w.dst_num_blocks, pool, bt, ws, view)
            b.record()
            b.synchronize()
            reps.append(a.elapsed_time(b))
        assert kv.lumen_kv_ckpt_status(ws) == 0
        t = float(np.median(reps))
        byts = 2.0 * nrows * sh.token_row_bytes
        wave_stats.append(dict(requests=len(wv), tokens=nrows, ms=t,
                               GBps=gb(byts) / (t / 1e3)))
        per_req_ms += [t * float(ctx[r]) / nrows for r in wv]
    del pool, ck
    torch.cuda.empty_cache()
    tot_ms = sum(x["ms"] for x in wave_stats)
    tot_b = sum(2.0 * x["tokens"] * sh.token_row_bytes for x in wave_stats)
    return dict(restore_ms_per_request=tot_ms / w.num_reqs,
                restore_ms_per_request_median=float(np.median(per_req_ms)),
                restore_GBps=gb(tot_b) / (tot_ms / 1e3),
                waves=wave_stats, requests=w.num_reqs,
                mean_request_GB=gb(float(ctx.mean()) * sh.token_row_bytes))


def offload_leg(torch, kv):
    """Device -> pinned host over the side stream (2 GiB), the first stage of
    shipping a checkpoint off the GPU."""
    dev = torch.device("cuda:0")
    n = 2 << 30
    d = torch.empty(n // 2, dtype=torch.int16, device=dev)
    d.fill_(3)
    h = torch.empty(n // 2, dtype=torch.int16, pin_memory=True)
    side = torch.cuda.Stream()
    kv.lumen_kv_ckpt_offload(d, h, side=side)
    side.synchronize()
    t0 = time.perf_counter()
    for _ in range(3):
        kv.lumen_kv_ckpt_offload(d, h, side=side)
    side.synchronize()
    dt = (time.perf_counter() - t0) / 3
    ok = bool(h[:1024].eq(3).all())
    return dict(d2h_GBps=gb(n) / dt, bytes=n, ok=ok)


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

def cpu_baseline(W, seconds):
    """The CPU oracle (plain loops, one thread) on a bounded sample of the
    same decode workload: whole steps packed from a host pool holding only
    the blocks those steps read, until the time budget is spent."""
    import oracle
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
    done_b, done_t, n_steps = 0.0, 0.0, 0
    for k, (n, bt) in enumerate(tables):
        t0 = time.perf_counter()
        st, _ = oracle.pack(sh, nb, pool, bt, w.starts[k], w.ends[k])
        done_t += time.perf_counter() - t0
        assert st == 0
        done_b += 2.0 * w.step_tokens(k) * sh.token_row_bytes
        n_steps += 1
        if done_t > seconds:
            break
    return {"value": round(gb(done_b) / done_t, 4), "unit": "GB/s",
            "cores": 1, "kind": "oracle",
            "sample": f"pack of decode steps 0..{n_steps - 1} of the "
                      f"Llama-3-8B-shaped workload ({gb(done_b):.2f} GB read+"
                      "written) from a compact host pool of the blocks those "
                      "steps read"}


# -------------------------------------------------------------------- main

def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the "
              "checkpoint path has no cross-GPU exchange to measure",
              file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2606_17787_amd.kvckpt as kv
    from paper_2606_17787_amd import workloads as W
    torch.cuda.set_device(0)
    if args.calibrate_copy_mib:
        calibrate_copy(torch, args.calibrate_copy_mib)
        return
    kv.load_library()

    dec = decode_leg(torch, kv, W, args.steps, args.warmup)
    w = dec.pop("workload")
    ms_per_step = dec["wall_ms"] / dec["steps"]
    value = gb(dec["bytes_total"]) / (dec["wall_ms"] / 1e3)
    dominant = "pack" if dec["pack_us_mean"] >= dec["unpack_us_mean"] else "unpack"
    achieved = dec[f"{dominant}_GBps"]
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "layers": w.shape.num_layers,
                   "kv_heads": w.shape.num_kv_heads,
                   "head_dim": w.shape.head_dim,
                   "block_size": w.shape.block_size,
                   "cache_layout": w.shape.order, "requests": w.num_reqs,
                   "tokens_per_step_mean": dec["tokens_per_step_mean"],
                   "step": "plan+pack of step k, plan+unpack of step k+50",
                   "parallelism": "none (1 GPU)"},
        "pack_GBps": round(dec["pack_GBps"], 1),
        "unpack_GBps": round(dec["unpack_GBps"], 1),
        "pack_pct_peak": round(100 * dec["pack_GBps"] / HBM_PEAK_GBPS, 2),
        "unpack_pct_peak": round(100 * dec["unpack_GBps"] / HBM_PEAK_GBPS, 2),
        "pack_us_median": round(dec["pack_us_median"], 2),
        "unpack_us_median": round(dec["unpack_us_median"], 2),
        "roundtrip_ok": dec["roundtrip_ok"],
        "roofline": {"bound": "hbm", "kernel": f"{dominant} (copy_rows_kernel)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "bytes_per_launch": dec[f"{dominant}_bytes_mean"],
                     "traffic": None},
    }
    if not args.no_restore:
        out["restore"] = restore_leg(torch, kv, W)
        out["restore_ms_per_request"] = round(
            out["restore"]["restore_ms_per_request"], 4)
    if not args.no_offload:
        out["offload"] = offload_leg(torch, kv)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(W, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
