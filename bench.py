"""Decode throughput of the page-based RaaS path on one MI355X.

A step is one raas_decode_step of one layer for the whole batch: append,
attention over every resident page, split merge, page scoring, top-r
timestamp refresh and eviction. The default workload is the batch-32
Llama-3.1-8B-shaped layer at budget L = 2048 (page 16, prefill 1024).

Setup (untimed): pool creation, prefill, and enough decode steps to fill the
budget, so the timed steps run in steady state (resident = L). Inputs are a
ring of seeded synthetic steps staged in HBM before timing; input generation
and host-to-device copies are outside the timed region. Then W warm-up steps
and K timed steps, bracketed by device synchronisation.

Prints one JSON line with the throughput (tokens/s = batch * K / time), the
attention kernel's roofline (algorithmic bytes per launch over its average
duration from HIP events recorded on the launch stream) and the CPU oracle's
throughput on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
KERNEL_ATTENTION = 1


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--workload", default=None, help="default: llama8b-b32-L2048")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--ring", type=int, default=128, help="distinct input steps staged on device")
    ap.add_argument("--splits", type=int, default=0, help="attention splits per unit (0 = automatic)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the CPU oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    return ap.parse_args()


def resident_schedule(st, ps, S, n):
    """Resident tokens per unit at each of the next n attention launches,
    from the exported state (pages fill in order; a full page is evicted
    when the tail is full and no slot is free)."""
    state, fill, tail = st["state"], st["fill"], st["tail"]
    U = state.shape[0]
    res = np.where(state != 0, fill, 0).sum(axis=1).astype(np.int64)
    free = (state == 0).sum(axis=1)
    n_ev = (state == 2).sum(axis=1)
    tf = np.where(tail >= 0, fill[np.arange(U), np.maximum(tail, 0)], ps)
    out = np.empty((n, U), np.int64)
    for i in range(n):
        new = tf == ps
        free = free - new
        n_ev = n_ev + new
        tf = np.where(new, 0, tf) + 1
        res = res + 1
        out[i] = res
        evict = (tf == ps) & (free == 0)
        tail_evicted = evict & (n_ev == 1)
        res = res - np.where(evict, ps, 0)
        free = free + evict
        n_ev = n_ev - evict
        tf = np.where(tail_evicted, ps, tf)
    return out


def step_bytes(w, resident, n_ev):
    """Algorithmic HBM bytes of one whole decode step for all units: K+V of the
    resident tokens, the representative keys of evictable pages, q read twice
    (attention and scoring) and out written, the new K/V read and stored,
    the tail page's representative keys updated, and per-slot state."""
    e = 2 if w.dtype == "bf16" else 4
    d, G, S, U = w.head_dim, w.group, w.slots, w.batch * w.n_kv_heads
    per_unit = (resident * 2 * d * e + n_ev * 2 * d * e + 3 * G * d * e + 4 * d * e + 4 * d * e + 16 * S)
    return per_unit.sum(axis=-1)


def attention_bytes(w, resident):
    """Algorithmic bytes of one attention launch: K+V of every resident token,
    q read, out written."""
    e = 2 if w.dtype == "bf16" else 4
    d, G, U = w.head_dim, w.group, w.batch * w.n_kv_heads
    return resident.sum(axis=-1) * 2 * d * e + 2 * U * G * d * e


def cpu_baseline(w, seed, ring_np, budget_s):
    """The fp64 CPU oracle on a bounded sample: a subset of units, filled to
    the budget with retention-only steps (attention skipped), then timed
    steady-state steps with attention over the same inputs."""
    import oracle
    import synth

    U = w.batch * w.n_kv_heads
    n_s = min(U, 64)
    units_idx = np.linspace(0, U - 1, n_s).astype(int)
    K, V = synth.prefill(w, seed, 0)
    ms = []
    for u in units_idx:
        b, h = divmod(int(u), w.n_kv_heads)
        m = oracle.Kvm(w.group, w.head_dim, w.page_size, w.slots, r=w.r)
        m.prefill(K[b, h].astype(np.float64), V[b, h].astype(np.float64))
        ms.append(m)
    q, k, v = ring_np
    R = q.shape[0]
    qs = q.reshape(R, U, w.group, w.head_dim)[:, units_idx]
    ks = k.reshape(R, U, w.head_dim)[:, units_idx]
    vs = v.reshape(R, U, w.head_dim)[:, units_idx]
    fill_steps = max(0, w.budget - w.prefill_len) + w.page_size
    for i in range(fill_steps):
        oracle.decode_batch(ms, qs[i % R], ks[i % R], vs[i % R], want_out=False)
    timed = 0
    t0 = time.perf_counter()
    while True:
        i = fill_steps + timed
        oracle.decode_batch(ms, qs[i % R], ks[i % R], vs[i % R], want_out=True)
        timed += 1
        el = time.perf_counter() - t0
        if el >= budget_s or timed >= 4096:
            break
    per_unit_step = el / (timed * n_s)
    tokens_per_s = w.batch / (per_unit_step * U)
    threads = min(oracle.threads(), n_s)
    return {
        "value": tokens_per_s, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
        "sample": "%d of %d units, %d steady-state decode steps with attention (%.1f s) after %d "
                  "retention-only fill steps; fp64 C oracle, OpenMP over units; scaled to the full "
                  "batch as batch / (units * seconds per unit-step)" % (n_s, U, timed, el, fill_steps),
        "host_cores_available": len(os.sched_getaffinity(0)),
    }


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU: this decode path has no multi-GPU mode "
              "(units are independent; see the design notes on sharding). Got --gpus %d." % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2502_11147_amd as raas
    import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w = synth.get_workload(args.workload or synth.workloads.HEADLINE)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    U, S = w.batch * w.n_kv_heads, w.slots

    pool = raas.Pool.for_workload(w)
    if args.splits:
        pool.set_attention_splits(args.splits)
    Kp, Vp = synth.prefill(w, args.seed, 0)
    pool.prefill(0, torch.from_numpy(Kp).to(dt).to(dev), torch.from_numpy(Vp).to(dt).to(dev))
    del Kp, Vp
    R = max(1, args.ring)
    ring_np = synth.steps(w, args.seed, 0, 0, R)
    qd, kd, vd = (torch.from_numpy(a).to(dt).to(dev) for a in ring_np)
    out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=dt, device=dev)

    prepared = [pool.prepare_step(0, qd[j], kd[j], vd[j], out) for j in range(R)]

    def run(i0, n):
        for i in range(i0, i0 + n):
            pool.decode_prepared(prepared[i % R])

    fill = max(0, w.budget - w.prefill_len) + w.page_size
    run(0, fill)
    run(fill, args.warmup)
    torch.cuda.synchronize()
    st = pool.export_state(0)
    res = resident_schedule(st, w.page_size, S, args.steps)
    n_ev0 = (st["state"] == 2).sum(axis=1)

    pool.profile(1 << KERNEL_ATTENTION)
    pool.profile_read(KERNEL_ATTENTION)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(fill + args.warmup, args.steps)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    attn_ms, attn_n = pool.profile_read(KERNEL_ATTENTION)
    pool.profile(0)
    st_end = pool.export_state(0)
    pool.close()

    ms_per_step = elapsed * 1e3 / args.steps
    tokens_per_s = w.batch * args.steps / elapsed
    attn_avg_s = attn_ms / 1e3 / max(attn_n, 1)
    attn_bytes = float(np.mean(attention_bytes(w, res)))
    achieved = attn_bytes / attn_avg_s / 1e9
    step_b = float(np.mean(step_bytes(w, res, n_ev0[None, :])))
    line = {
        "metric": "decode tokens/s per GPU at batch B, budget L; achieved HBM GB/s vs peak",
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded N(0,1) Q/K/V with planted milestone tokens; no datasets or weights)",
        "config": {
            "workload": w.name, "batch": w.batch, "layers_per_step": 1, "n_q_heads": w.n_q_heads,
            "n_kv_heads": w.n_kv_heads, "head_dim": w.head_dim, "page_size": w.page_size,
            "budget_tokens": w.budget, "prefill_len": w.prefill_len, "r": w.r,
            "resident_tokens_per_unit_avg": float(res.mean()),
            "attention_splits": args.splits or "auto",
        },
        "step_hbm_gbs_algorithmic": round(step_b / (elapsed / args.steps) / 1e9, 1),
        "roofline": {
            "kernel": "k_attn_bf16" if w.dtype == "bf16" else "k_attn_f32",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None,
            "bytes_per_launch": attn_bytes,
            "avg_launch_us": round(attn_avg_s * 1e6, 3),
            "launches_timed": attn_n,
        },
    }
    assert np.all(st_end["clock"] == w.prefill_len + fill + args.warmup + args.steps)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(w, args.seed, ring_np, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
