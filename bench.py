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
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
KERNEL_STEP, KERNEL_EPILOGUE, KERNEL_SELECT = 0, 1, 2


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--workload", default=None, help="default: llama8b-b32-L2048")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--r", type=float, default=None, help="fraction refreshed per step (default: the workload's)")
    ap.add_argument("--ring", type=int, default=128, help="distinct input steps staged on device")
    ap.add_argument("--splits", type=int, default=0, help="attention splits per unit (0 = automatic)")
    ap.add_argument("--score-aggregation", choices=("max", "softmax-sum"), default="max",
                    help="head aggregation of the page score (default: max over the heads)")
    ap.add_argument("--rank-pinned", action="store_true", help="rank the pinned prefill pages too")
    ap.add_argument("--decision-scope", choices=("kv-head", "sequence"), default="kv-head",
                    help="one page table per KV head (default) or per sequence")
    ap.add_argument("--prompt-topk", type=int, default=0,
                    help="Quest on the prompt: keep the whole prompt in a prompt region and attend to this many "
                         "prompt pages per step (0: off; the budget then counts decode tokens)")
    ap.add_argument("--deterministic", action="store_true",
                    help="bitwise-reproducible outputs: a fixed interleave of the blocks over the wavefronts")
    ap.add_argument("--no-cold", action="store_true",
                    help="skip the cold-cache row (the same layer shape, four layers stepped per token)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the CPU oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--decode-sweep", action="store_true",
                    help="per-step latency and resident tokens against decode length (prompt 128, batch 4, "
                         "decode 8192) for RaaS at L = 1024 and 2048 and for a pool holding every token")
    ap.add_argument("--sweep-window", type=int, default=256, help="decode steps per measured window")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain streaming kernel of known size (counter calibration)")
    ap.add_argument("--access-probe", action="store_true",
                    help="run only the streaming probe (libraas_probe.so): the step kernel's K/V access structure "
                         "without arithmetic, at the workloads' pool shapes, warm and cold")
    ap.add_argument("--traffic-summary", metavar="DIR", default=None,
                    help="turn rocprofv3 --pmc output under DIR/{fetch,write,copy_fetch,copy_write} "
                         "into the stored traffic profile of --workload")
    return ap.parse_args()


COPY_BYTES = 1 << 30  # bytes read (and written) by one calibration launch
PROFILES = os.path.join(ROOT, "profiles")


def traffic_profile_path(kernel, workload):
    return os.path.join(PROFILES, "traffic_%s_%s.json" % (kernel, workload))


def copy_calibration():
    """A plain streaming kernel of known size: negation of 2^30 bytes of bf16
    into a second buffer (each byte read once, written once). What FETCH_SIZE
    and WRITE_SIZE read for it scales them to bytes."""
    import torch

    assert torch.cuda.is_available(), "needs a GPU"
    n = COPY_BYTES // 2
    src = torch.ones(n, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration": "neg", "bytes_read": COPY_BYTES, "bytes_written": COPY_BYTES,
                      "launches": 5}), flush=True)


class _ProbeConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("units", "tokens", "head_dim", "layers", "waves", "nontemporal", "mode", "dynamic", "alternate",
                 "launches", "kv_interleaved")]


# (name, units, tokens per unit, waves, layers, non-temporal, mode, K and V of
# a block adjacent): the pool shapes of the workloads; layers > 1 read
# several pools in turn so that no launch finds its data in the 256 MB
# memory-side cache
PROBES = [
    ("llama8b-b32-L2048 (one layer, alternating)", 256, 2048, 8, 1, 0, 0, 0),
    ("llama8b-b32-L2048 x4 layers, cold", 256, 2048, 8, 4, 1, 0, 0),
    ("llama8b-b32-L2048 x4 layers, cold, two blocks per wavefront in LDS", 256, 2048, 4, 4, 1, 1, 0),
    ("llama8b-b32-L2048 x4 layers, cold, K and V of a block adjacent", 256, 2048, 8, 4, 1, 0, 1),
    ("llama8b-b32-L2048 x4 layers, cold, ordinary loads", 256, 2048, 8, 4, 0, 0, 0),
    ("qwen7b-28L-b64-L4096 (28 layers, cold)", 256, 4096, 8, 28, 1, 0, 0),
    ("qwen7b-28L-b64-L4096, two blocks per wavefront in LDS", 256, 4096, 4, 28, 1, 1, 0),
    ("qwen7b-28L-b64-L4096, K and V of a block adjacent", 256, 4096, 8, 28, 1, 0, 1),
    ("llama8b-b128-ps32-L8192 (4.3 GB, cold)", 1024, 8192, 4, 1, 1, 0, 0),
    ("llama8b-b128-ps32-L8192, two blocks per wavefront in LDS", 1024, 8192, 4, 1, 1, 1, 0),
    ("llama8b-b128-ps32-L8192, K and V of a block adjacent", 1024, 8192, 4, 1, 1, 0, 1),
]


def access_probe():
    """The streaming probe at the workloads' pool shapes: the rate of the
    step kernel's K/V access structure without arithmetic (a ceiling for it
    on the same data), one JSON line per shape."""
    from paper_2502_11147_amd import build as hip_build

    lib = ctypes.CDLL(hip_build.PROBE_LIB_PATH)
    lib.raas_probe_stream.argtypes = [ctypes.POINTER(_ProbeConfig), ctypes.POINTER(ctypes.c_double),
                                      ctypes.POINTER(ctypes.c_double)]
    lib.raas_probe_stream.restype = ctypes.c_int
    for name, units, tokens, waves, layers, nt, mode, kvi in PROBES:
        cfg = _ProbeConfig(units, tokens, 128, layers, waves, nt, mode, 1, 1, max(200, 4 * layers), kvi)
        us, b = ctypes.c_double(), ctypes.c_double()
        rc = lib.raas_probe_stream(ctypes.byref(cfg), ctypes.byref(us), ctypes.byref(b))
        if rc != 0:
            raise SystemExit("raas_probe_stream failed (%d) for %s" % (rc, name))
        gbs = b.value / us.value / 1e3
        print(json.dumps({"access_probe": name, "units": units, "tokens_per_unit": tokens, "waves": waves,
                          "layers": layers, "nontemporal": bool(nt), "mode": ["registers", "lds"][mode],
                          "kv_interleaved": bool(kvi),
                          "bytes_per_launch": b.value, "us_per_launch": round(us.value, 3),
                          "GB_per_s": round(gbs, 1), "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4)}), flush=True)


def _counter_rows(d, counter):
    import csv
    import glob

    files = sorted(glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True))
    if not files:
        raise SystemExit("no counter_collection.csv under %s" % d)
    rows = []
    for f in files:
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] == counter:
                    rows.append(r)
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    return rows


def traffic_summary(args):
    """Per-launch FETCH_SIZE and WRITE_SIZE of the step kernel over the last
    --steps dispatches (the timed steps of a bench run with the same flags),
    scaled by the factor that makes the same counters read the known size of
    the calibration kernel. Writes the stored traffic profile."""
    import synth
    from paper_2502_11147_amd import build as hip_build

    w = synth.get_workload(args.workload or synth.workloads.HEADLINE)
    kernel = "k_step_bf16" if w.dtype == "bf16" else "k_step_f32"
    out = {"kernel": kernel, "workload": w.name, "kernel_digest": hip_build.kernel_digest()}
    for counter, sub, csub in (("FETCH_SIZE", "fetch", "copy_fetch"), ("WRITE_SIZE", "write", "copy_write")):
        rows = [r for r in _counter_rows(os.path.join(args.traffic_summary, sub), counter)
                if kernel in r["Kernel_Name"]]
        want = args.steps * w.n_layers  # the timed steps' launches, one per layer
        rows = rows[-want:]
        if len(rows) < want:
            raise SystemExit("%s: %d %s dispatches, want %d" % (counter, len(rows), kernel, want))
        kib = float(np.mean([float(r["Counter_Value"]) for r in rows]))
        crow = [r for r in _counter_rows(os.path.join(args.traffic_summary, csub), counter)
                if "neg" in r["Kernel_Name"]]
        if not crow:
            raise SystemExit("%s: no calibration dispatches" % counter)
        ckib = float(np.median([float(r["Counter_Value"]) for r in crow]))
        factor = COPY_BYTES / (ckib * 1024.0)
        key = counter.lower()
        out[key + "_kib_per_launch"] = round(kib, 3)
        out[key + "_calibration_kib"] = round(ckib, 3)
        out[key + "_factor"] = round(factor, 5)
        out[key + "_bytes_per_launch"] = round(kib * 1024.0 * factor)
        out[key + "_launches"] = len(rows)
    out["traffic_bytes_per_launch"] = out["fetch_size_bytes_per_launch"] + out["write_size_bytes_per_launch"]
    flags = "--workload %s --steps %d --warmup %d --no-cpu-baseline --no-cold" % (w.name, args.steps, args.warmup)
    out["commands"] = [
        "timeout -s KILL 300 rocprofv3 --pmc FETCH_SIZE --output-format csv -d DIR/fetch -- python3 bench.py " + flags,
        "timeout -s KILL 300 rocprofv3 --pmc WRITE_SIZE --output-format csv -d DIR/write -- python3 bench.py " + flags,
        "timeout -s KILL 120 rocprofv3 --pmc FETCH_SIZE --output-format csv -d DIR/copy_fetch -- python3 bench.py --copy-calibration",
        "timeout -s KILL 120 rocprofv3 --pmc WRITE_SIZE --output-format csv -d DIR/copy_write -- python3 bench.py --copy-calibration",
        "python3 bench.py --traffic-summary DIR " + flags,
    ]
    os.makedirs(PROFILES, exist_ok=True)
    path = traffic_profile_path(kernel, w.name)
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out), flush=True)


def stored_traffic(kernel, workload):
    """HBM bytes per launch from the stored counter profile, or None when
    there is none or the kernels have changed since it was taken."""
    from paper_2502_11147_amd import build as hip_build

    path = traffic_profile_path(kernel, workload)
    if not os.path.exists(path):
        return None, "no stored counter profile"
    with open(path) as f:
        prof = json.load(f)
    if prof.get("kernel_digest") != hip_build.kernel_digest():
        return None, "kernel sources changed since the counters were taken"
    return float(prof["traffic_bytes_per_launch"]), os.path.relpath(path, ROOT)


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


def step_bytes(w, resident, n_ev, S=None):
    """Algorithmic HBM bytes of one whole decode step, all units: K+V of the
    resident tokens; the representative keys (per-channel min and max) of the
    n_ev scored pages (the evictable ones, plus the pinned ones when they are
    ranked); q read once, out written once; the new K and V read once
    and stored once; the tail page's min/max read and written; per slot,
    state/timestamp/id/fill read and state/timestamp written (24 B)."""
    e = 2 if w.dtype == "bf16" else 4
    d, G = w.head_dim, w.group
    S = w.slots if S is None else S
    per_unit = (resident * 2 * d * e + n_ev * 2 * d * e + 2 * G * d * e + 4 * d * e + 4 * d * e + 24 * S)
    return per_unit.sum(axis=-1)


def cpu_baseline(w, seed, ring_np, budget_s, aggregation=0, rank_pinned=False):
    """The fp64 CPU oracle on a bounded sample: a subset of units, filled to
    the budget with retention-only steps (attention skipped), then timed
    steady-state steps with attention over the same inputs."""
    import oracle
    import synth

    U = w.batch * w.n_kv_heads
    n_s = min(U, 64)
    oracle_threads_default = oracle.threads()
    units_idx = np.linspace(0, U - 1, n_s).astype(int)
    K, V = synth.prefill(w, seed, 0)
    ms = []
    for u in units_idx:
        b, h = divmod(int(u), w.n_kv_heads)
        m = oracle.Kvm(w.group, w.head_dim, w.page_size, w.slots, r=w.r, aggregation=aggregation,
                       rank_pinned=rank_pinned)
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
    tokens_per_s = w.batch / (per_unit_step * U * w.n_layers)
    threads = min(oracle.threads(), n_s)
    # the same steps on one core, a shorter sample
    oracle.set_threads(1)
    t1, timed1 = time.perf_counter(), 0
    while True:
        i = fill_steps + timed1
        oracle.decode_batch(ms, qs[i % R], ks[i % R], vs[i % R], want_out=True)
        timed1 += 1
        el1 = time.perf_counter() - t1
        if el1 >= budget_s / 3 or timed1 >= 4096:
            break
    oracle.set_threads(oracle_threads_default)
    tokens_per_s_1 = w.batch / (el1 / (timed1 * n_s) * U * w.n_layers)
    cpu_model = ""
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), "")
    except OSError:
        pass
    return {
        "value": tokens_per_s, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
        "sample": "%d of %d units, %d steady-state decode steps with attention (%.1f s) after %d "
                  "retention-only fill steps; fp64 C oracle, OpenMP over units; scaled to the full "
                  "batch%s as batch / (units * seconds per unit-step%s)"
                  % (n_s, U, timed, el, fill_steps, " and all layers" if w.n_layers > 1 else "",
                     " * layers" if w.n_layers > 1 else ""),
        "value_1core": tokens_per_s_1,
        "sample_1core": "%d steps of the same units on one thread (%.1f s)" % (timed1, el1),
        "cpu_model": cpu_model,
        "host_cores_available": len(os.sched_getaffinity(0)),
    }


def cold_row(w, args, kernel_bytes, steps=500, layers=4):
    """The step kernel on the same layer shape with `layers` layers stepped
    per token (one launch each), so that a layer's pool has left the 256 MB
    memory-side cache by the time its next step comes: per-launch duration
    from HIP events over the timed launches (the step kernel is the step's
    only kernel), against the single layer's algorithmic bytes."""
    import torch

    import paper_2502_11147_amd as raas
    import synth

    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    wl = w.replace(n_layers=layers)
    pool = raas.Pool.for_workload(wl)
    Kp, Vp = synth.prefill(w, args.seed, 0)
    Kd, Vd = torch.from_numpy(Kp).to(dt).cuda(), torch.from_numpy(Vp).to(dt).cuda()
    for layer in range(layers):
        pool.prefill(layer, Kd, Vd)
    R = 64
    qd, kd, vd = (torch.from_numpy(a).to(dt).cuda() for a in synth.steps(w, args.seed, 0, 0, R))
    out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=dt, device="cuda")
    prep = [[pool.prepare_step(layer, qd[j], kd[j], vd[j], out) for j in range(R)] for layer in range(layers)]

    def run(i0, n):
        for i in range(i0, i0 + n):
            for layer in range(layers):
                pool.decode_prepared(prep[layer][i % R])

    fill = max(0, w.budget - w.prefill_len) + w.page_size
    run(0, fill + 50)
    pool.profile(1 << KERNEL_EPILOGUE)
    run(fill + 50, 1)
    assert pool.profile_read(KERNEL_EPILOGUE)[1] == 0, "expected one fused kernel per step"
    pool.profile(0)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    run(fill + 51, steps)
    ev1.record()
    torch.cuda.synchronize()
    us = ev0.elapsed_time(ev1) * 1e3 / (steps * layers)
    pool.close()
    gbs = kernel_bytes / us / 1e3
    return {"workload": "%s, %d layers stepped per token" % (w.name, layers), "avg_launch_us": round(us, 3),
            "launches_timed": steps * layers, "achieved": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4),
            "bytes_per_launch": kernel_bytes, "pools_bytes": layers * pool_kv_bytes(w),
            "note": "each layer's pool is read once per token; the pools together exceed the memory-side "
                    "cache, so this is the rate from HBM (the runtime reads them with non-temporal loads)"}


def pool_kv_bytes(w):
    e = 2 if w.dtype == "bf16" else 4
    lcap = -(-w.slots * w.page_size // 32) * 32
    return 2 * w.batch * w.n_kv_heads * lcap * w.head_dim * e


def decode_sweep(args):
    """Decode-length sweep (the setting of the paper's Fig. 6: prompt 128,
    batch 4, decode up to 8192 tokens) on one Mistral-7B-shaped layer: per
    window of decode steps, the mean step time (HIP events on the launch
    stream) and the mean resident tokens per unit; the pool's device bytes,
    fixed at creation. One JSON line per configuration."""
    import torch

    import paper_2502_11147_amd as raas
    import synth

    assert torch.cuda.is_available(), "needs a GPU"
    dev = torch.device("cuda", 0)
    W = max(1, args.sweep_window)
    for name in ("mistral7b-b4-P128-L1024", "mistral7b-b4-P128-L2048", "mistral7b-b4-P128-dense"):
        w = synth.get_workload(name)
        pool = raas.Pool.for_workload(w)
        K, V = synth.prefill(w, args.seed, 0)
        pool.prefill(0, torch.from_numpy(K).to(torch.bfloat16).to(dev), torch.from_numpy(V).to(torch.bfloat16).to(dev))
        out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.bfloat16, device=dev)
        ends, us, resident = [], [], []
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for t0 in range(0, w.decode_steps, W):
            n = min(W, w.decode_steps - t0)
            q, k, v = (torch.from_numpy(a).to(torch.bfloat16).to(dev) for a in synth.steps(w, args.seed, 0, t0, n))
            prepared = [pool.prepare_step(0, q[i], k[i], v[i], out) for i in range(n)]
            torch.cuda.synchronize()
            ev0.record()
            for a in prepared:
                pool.decode_prepared(a)
            ev1.record()
            torch.cuda.synchronize()
            st = pool.export_state(0)
            ends.append(t0 + n)
            us.append(round(ev0.elapsed_time(ev1) * 1e3 / n, 3))
            resident.append(float(np.where(st["state"] != 0, st["fill"], 0).sum(axis=1).mean()))
        line = {"decode_sweep": name, "batch": w.batch, "prefill_len": w.prefill_len, "budget_tokens": w.budget,
                "pool_bytes": pool.pool_bytes(), "window": W, "decode_len_at_window_end": ends,
                "us_per_step": us, "resident_tokens_per_unit": resident,
                "job_ms": round(sum(u * n for u, n in zip(us, np.diff([0] + ends))) / 1e3, 3)}
        pool.close()
        print(json.dumps(line), flush=True)


def main():
    args = parse()
    if args.traffic_summary:
        traffic_summary(args)
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU: this decode path has no multi-GPU mode "
              "(units are independent; see the design notes on sharding). Got --gpus %d." % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return
    if args.access_probe:
        access_probe()
        return
    if args.decode_sweep:
        decode_sweep(args)
        return
    import torch

    import paper_2502_11147_amd as raas
    import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w = synth.get_workload(args.workload or synth.workloads.HEADLINE)
    if args.r is not None:
        w = w.replace(r=args.r)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    agg = raas.SCORE_SOFTMAX_SUM if args.score_aggregation == "softmax-sum" else raas.SCORE_MAX
    scope = raas.SCOPE_SEQUENCE if args.decision_scope == "sequence" else raas.SCOPE_KV_HEAD
    align = max(w.page_size, 32)
    prompt_tokens = -(-w.prefill_len // align) * align if args.prompt_topk > 0 else 0
    npr = prompt_tokens // w.page_size
    variant = (agg != raas.SCORE_MAX or args.rank_pinned or scope != raas.SCOPE_KV_HEAD or npr > 0
               or args.deterministic)
    t_run = time.perf_counter()
    pool = raas.Pool.for_workload(w, score_aggregation=agg, rank_pinned=args.rank_pinned, decision_scope=scope,
                                  prompt_tokens=prompt_tokens, prompt_topk=args.prompt_topk,
                                  deterministic=args.deterministic)
    U, S = w.batch * w.n_kv_heads, pool.slots
    if args.splits:
        pool.set_attention_splits(args.splits)
    # a step is one token through every layer of the workload; the layers
    # share one synthetic prompt and one ring of step inputs
    nl = w.n_layers
    Kp, Vp = synth.prefill(w, args.seed, 0)
    Kd, Vd = torch.from_numpy(Kp).to(dt).to(dev), torch.from_numpy(Vp).to(dt).to(dev)
    del Kp, Vp
    for layer in range(nl):
        pool.prefill(layer, Kd, Vd)
    del Kd, Vd
    R = max(1, args.ring)
    ring_np = synth.steps(w, args.seed, 0, 0, R)
    qd, kd, vd = (torch.from_numpy(a).to(dt).to(dev) for a in ring_np)
    out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=dt, device=dev)

    prepared = [[pool.prepare_step(layer, qd[j], kd[j], vd[j], out) for j in range(R)] for layer in range(nl)]

    def run(i0, n):
        for i in range(i0, i0 + n):
            for layer in range(nl):
                pool.decode_prepared(prepared[layer][i % R])

    fill = (w.budget if npr else max(0, w.budget - w.prefill_len)) + w.page_size
    run(0, fill)
    run(fill, args.warmup)
    torch.cuda.synchronize()

    # one kernel per step (the step kernel runs the epilogue and, with a
    # prompt region, the selection) or more?
    pool.profile((1 << KERNEL_EPILOGUE) | (1 << KERNEL_SELECT))
    run(fill + args.warmup, 1)
    fused = pool.profile_read(KERNEL_EPILOGUE)[1] == 0
    # the event span times the step kernel alone only when it is the step's
    # only launch (a separate prompt selection adds a kernel in front)
    alone = fused and pool.profile_read(KERNEL_SELECT)[1] == 0
    pool.profile(0)
    t_start = fill + args.warmup + 1
    st = pool.export_state(0)
    n_ev0 = (st["state"] == 2).sum(axis=1)
    n_pin = (st["state"] == 1).sum(axis=1) if args.rank_pinned else 0
    if npr:
        # the decode region evolves as a pool of its own; the attention reads
        # the chosen prompt pages (full ones) besides, and the selection
        # reads every kept prompt page's representative keys
        kp = (st["state"][:, :npr] == 1).sum(axis=1)
        dec = dict(state=st["state"][:, npr:], fill=st["fill"][:, npr:],
                   tail=np.where(st["tail"] >= 0, st["tail"] - npr, -1))
        res = resident_schedule(dec, w.page_size, S - npr, args.steps) + np.minimum(kp, args.prompt_topk) * w.page_size
        n_pin = kp
    else:
        res = resident_schedule(st, w.page_size, S, args.steps)

    # timed region: HIP events on the launch stream (torch's current stream)
    # around all K steps; with two kernels per step, the library also times
    # each kernel on every 16th step
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    if alone:
        run(t_start, args.steps)
    else:
        for i0 in range(0, args.steps, 16):
            pool.profile((1 << KERNEL_STEP) | (1 << KERNEL_EPILOGUE) | (1 << KERNEL_SELECT))
            run(t_start + i0, 1)
            pool.profile(0)
            run(t_start + i0 + 1, min(16, args.steps - i0) - 1)
    ev1.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    span_ms = ev0.elapsed_time(ev1)
    step_ms, step_n = pool.profile_read(KERNEL_STEP)
    epi_ms, epi_n = pool.profile_read(KERNEL_EPILOGUE)
    sel_ms, sel_n = pool.profile_read(KERNEL_SELECT)
    st_end = pool.export_state(0)
    pool.close()

    ms_per_step = elapsed * 1e3 / args.steps
    tokens_per_s = w.batch * args.steps / elapsed
    # step kernel's average duration: the event span over the K launches when
    # it is the only kernel of the step, else the sampled per-kernel events
    step_avg_s = span_ms / 1e3 / (args.steps * nl) if alone else step_ms / 1e3 / max(step_n, 1)
    step_b = float(np.mean(step_bytes(w, res, (n_ev0 + n_pin)[None, :], S)))
    # bytes of the step kernel alone: everything but what the epilogue kernel moves
    e = 2 if w.dtype == "bf16" else 4
    kernel_b = step_b if fused else step_b - U * w.group * w.head_dim * e - 24 * U * S
    achieved = kernel_b / step_avg_s / 1e9
    kname = "k_step_bf16" if w.dtype == "bf16" else ("k_step_f32_fused" if fused else "k_step_f32")
    if variant:
        traffic, traffic_src = None, "no stored counter profile for the variants"
    elif fused:
        traffic, traffic_src = stored_traffic(kname, w.name)
    else:
        traffic, traffic_src = None, "two kernels per step"
    line = {
        "metric": "decode tokens/s per GPU at batch B, budget L; achieved HBM GB/s vs peak",
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "ms_per_step_events": round(span_ms / args.steps, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded N(0,1) Q/K/V with planted milestone tokens; no datasets or weights)",
        "config": {
            "workload": w.name, "batch": w.batch, "layers_per_step": nl, "n_q_heads": w.n_q_heads,
            "n_kv_heads": w.n_kv_heads, "head_dim": w.head_dim, "page_size": w.page_size,
            "budget_tokens": w.budget, "prefill_len": w.prefill_len, "r": w.r,
            "resident_tokens_per_unit_avg": float(res.mean()),
            "attention_splits": args.splits or "auto",
            "score_aggregation": args.score_aggregation, "rank_pinned": bool(args.rank_pinned),
            "decision_scope": args.decision_scope,
            "prompt_tokens": prompt_tokens, "prompt_topk": args.prompt_topk,
            "deterministic": bool(args.deterministic),
        },
        "step_hbm_gbs_algorithmic": round(step_b * nl / (elapsed / args.steps) / 1e9, 1),
        "roofline": {
            "kernel": kname + ("" if fused else " (+k_epilogue)"),
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None if traffic is None else round(traffic),
            "traffic_source": traffic_src,
            "bytes_per_launch": kernel_b,
            "avg_launch_us": round(step_avg_s * 1e6, 3),
            "launches_timed": args.steps * nl if alone else step_n,
            "timing": "event span over the timed launches" if alone else "per-launch events, every 16th step",
            "epilogue_kernel_avg_us": round(epi_ms * 1e3 / epi_n, 3) if epi_n else None,
            "select_kernel_avg_us": round(sel_ms * 1e3 / sel_n, 3) if sel_n else None,
        },
    }
    assert np.all(st_end["clock"] == w.prefill_len + t_start + args.steps)
    if nl == 1 and fused and not variant and not args.no_cold and not args.splits:
        line["roofline_cold"] = cold_row(w, args, kernel_b)
    if not args.no_cpu_baseline:
        if scope == raas.SCOPE_KV_HEAD:
            line["cpu_baseline"] = cpu_baseline(w, args.seed, ring_np, args.cpu_seconds, agg, args.rank_pinned)
        else:
            line["cpu_baseline"] = None
            line["cpu_baseline_note"] = "not sampled for the sequence scope (its oracle step is serial)"
    line["run_wall_s"] = round(time.perf_counter() - t_run, 2)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
