"""Lockstep parity harness: the HIP decode path against the CPU oracle.

Both sides get the same seeded inputs (``synth``). Per step and checked unit:
  - page table, timestamps and evicted page must be bit-exact. The one
    allowance is a near tie: when the oracle's step has two or more ranked
    pages within NEAR_TIE of the threshold score, the two sides may rank
    them differently. A mismatch confined to those pages (and to the slots
    of a resulting different eviction) is counted, and the oracle then
    adopts the GPU's decision for that step (``Kvm.adopt_retention``) and
    goes on in lockstep, so one near tie cannot cascade. The step of a
    unit's first such re-sync is where a free-running oracle would first
    have diverged; it is reported. Any other mismatch fails.
  - attention outputs must agree within the dtype's absolute bound (the
    contract's) and within a relative L2 bound per (unit, query head),
    which stays sensitive when outputs are small (long, flat softmaxes):
    at the full-size shapes, dropping one 32-token block or one page from
    the attended set exceeds it (a CPU test checks that).

Every run's counts go to ``REPORTS``; ``conftest.py`` prints them at the end
of the session, so a quiet (-q) run still shows them.
"""
from __future__ import annotations

import dataclasses
import math
import os
import sys
import time

import numpy as np

import oracle
import synth

NEAR_TIE = 1e-6
TOL = {"bf16": 2e-2, "f32": 1e-4}       # max abs error of an output element
TOL_REL = {"bf16": 1e-2, "f32": 1e-4}   # L2 error of a head's output vector over its L2 norm

REPORTS: list = []  # (test id, tag, ParityReport) of every run in this session


@dataclasses.dataclass
class ParityReport:
    steps: int = 0
    units_checked: int = 0
    outputs_compared: int = 0
    max_abs_err: float = 0.0
    max_rel_err: float = 0.0
    flagged_steps: int = 0          # unit-steps whose threshold was a near tie
    flagged_divergences: int = 0    # of those, where the GPU decided differently (oracle re-synced)
    first_divergence: dict = dataclasses.field(default_factory=dict)  # unit -> step of its first re-sync
    evictions: int = 0
    first_eviction_step: int = -1   # earliest step at which any unit evicted (-1: none)
    invariant_checks: int = 0       # steps whose every unit was checked against the invariants
    notes: list = dataclasses.field(default_factory=list)

    def line(self, tag: str) -> str:
        fd = ""
        if self.first_divergence:
            items = sorted(self.first_divergence.items(), key=lambda kv: kv[1])[:4]
            fd = " first divergence " + ", ".join("unit %d@%d" % kv for kv in items)
        return ("%s: steps %d units %d outputs %d max_abs %.3g max_rel %.3g evictions %d "
                "flagged %d resynced %d%s" % (tag, self.steps, self.units_checked, self.outputs_compared,
                                             self.max_abs_err, self.max_rel_err, self.evictions,
                                             self.flagged_steps, self.flagged_divergences, fd))


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def record(rep: ParityReport, tag: str) -> ParityReport:
    test = os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0]
    REPORTS.append((test, tag, rep))
    say(rep.line(tag))
    return rep


def to_device(a: np.ndarray, dtype: str):
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a))
    t = t.to(torch.bfloat16) if dtype == "bf16" else t.to(torch.float32)
    return t.cuda()


def _to_device_async(a: np.ndarray, dtype: str, keep: list):
    """Host array -> device without blocking the host: staged through a new
    pinned buffer (kept alive in `keep` until the copy has run)."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a))
    t = (t.to(torch.bfloat16) if dtype == "bf16" else t.to(torch.float32)).pin_memory()
    keep.append(t)
    return t.to("cuda", non_blocking=True)


def _to_host_async(t, keep: list):
    import torch

    h = torch.empty(t.shape, dtype=t.dtype, pin_memory=True)
    h.copy_(t, non_blocking=True)
    keep.append(h)
    return h


def new_pool(w, splits=None, policy=None, aggregation=0, rank_pinned=False, scope=0, prompt_tokens=0,
             prompt_topk=0, deterministic=False):
    import paper_2502_11147_amd as raas

    kw = {"score_aggregation": aggregation, "rank_pinned": rank_pinned, "decision_scope": scope,
          "prompt_tokens": prompt_tokens, "prompt_topk": prompt_topk, "deterministic": deterministic}
    if policy is not None:
        kw["prefill_policy"] = policy
    pool = raas.Pool.for_workload(w, **kw)
    if splits is not None:
        pool.set_attention_splits(splits)
    return pool


def random_case(i: int) -> dict:
    """Seeded random configuration i: every switch of the C ABI drawn
    together (pool dtype, head_dim, group size, KV heads, batch, page size,
    budget, prompt length below and above the budget, r, the score
    aggregation, ranked pinned pages, the decision scope, Quest on the
    prompt, forced attention splits, the deterministic option). The pool is
    valid (group at most 16, budget and prompt region multiples of the page,
    the prompt region also of 32, at most 2048 slots) and small enough for
    the oracle to follow every unit for a few hundred steps, which run past
    the budget."""
    import math

    rng = np.random.default_rng(1000 + i)
    dtype = "f32" if rng.random() < 0.2 else "bf16"
    d = int(rng.choice([64, 128]))
    G = int(rng.choice([1, 2, 3, 4, 5, 7, 8, 16]))
    hkv = int(rng.choice([1, 2, 4])) if G <= 8 else 1
    batch = int(rng.integers(1, 4)) if G * hkv <= 16 else 1
    ps = int(rng.choice([8, 16, 32, 64, 128]))
    pages = int(rng.integers(2, max(2, 512 // ps) + 1))
    budget = pages * ps
    prefill = int(rng.integers(0, 2 * budget + 1))
    r = float(rng.choice([0.0, 0.25, 0.3, 0.5, 0.7, 0.9, 1.0]))
    agg = int(rng.random() < 0.2)
    scope = int(rng.random() < 0.15)
    prompt = bool(rng.random() < 0.2)
    rank = (not prompt) and bool(rng.random() < 0.15)
    prompt_tokens = prompt_topk = 0
    if prompt:
        unit = ps * 32 // math.gcd(ps, 32)
        prompt_tokens = unit * int(rng.integers(1, max(1, 512 // unit) + 1))
        prompt_topk = int(rng.integers(1, prompt_tokens // ps + 1))
    splits = None if rng.random() < 0.7 else int(rng.integers(2, 6))
    det = bool(rng.random() < 0.1)
    kept = 0 if prompt else min(prefill, budget)
    steps = int(min(800, max(120, budget - kept + 3 * ps + 40)))
    return dict(workload=dict(name="random-%02d" % i, batch=batch, n_layers=1, n_q_heads=G * hkv,
                              n_kv_heads=hkv, head_dim=d, dtype=dtype, page_size=ps, budget=budget,
                              prefill_len=prefill, decode_steps=steps, r=r, ms_period=16,
                              ms_phase_random=True, ms_wmin=8, ms_wmax=64),
                variant=dict(aggregation=agg, rank_pinned=rank, scope=scope, prompt_tokens=prompt_tokens,
                             prompt_topk=prompt_topk),
                splits=splits, deterministic=det)


def random_large_case(i: int) -> dict:
    """Seeded random configuration i with a long pool: budgets of 1024 to
    4096 tokens (up to 512 slots at page 8, past the 256 where the split
    path's refresh turns to a radix select), prompt regions up to 2048
    tokens, at most 4 units, the same switches as random_case. Outputs are
    meant to be compared on sampled steps (retention at every step)."""
    import math

    rng = np.random.default_rng(5000 + i)
    dtype = "f32" if rng.random() < 0.15 else "bf16"
    d = int(rng.choice([64, 128]))
    G = int(rng.choice([1, 2, 4, 7, 8, 16]))
    hkv = int(rng.choice([1, 2]))
    batch = int(rng.integers(1, 3))
    ps = int(rng.choice([8, 16, 32, 64]))
    budget = ps * int(rng.integers(max(2, 1024 // ps), 4096 // ps + 1))
    prefill = int(rng.integers(0, budget + 1))
    r = float(rng.choice([0.25, 0.5, 0.7, 0.9]))
    agg = int(rng.random() < 0.2)
    scope = int(rng.random() < 0.15)
    prompt = bool(rng.random() < 0.25)
    rank = (not prompt) and bool(rng.random() < 0.15)
    prompt_tokens = prompt_topk = 0
    if prompt:
        unit = ps * 32 // math.gcd(ps, 32)
        prompt_tokens = unit * int(rng.integers(1, max(1, 2048 // unit) + 1))
        prompt_topk = int(rng.integers(1, prompt_tokens // ps + 1))
    splits = None if rng.random() < 0.6 else int(rng.choice([1, 2, 5, 16, 64]))
    det = bool(rng.random() < 0.15)
    kept = 0 if prompt else min(prefill, budget)
    steps = int(budget - kept + 3 * ps + 40)
    return dict(workload=dict(name="random-large-%02d" % i, batch=batch, n_layers=1, n_q_heads=G * hkv,
                              n_kv_heads=hkv, head_dim=d, dtype=dtype, page_size=ps, budget=budget,
                              prefill_len=prefill, decode_steps=steps, r=r, ms_period=32,
                              ms_phase_random=True, ms_wmin=16, ms_wmax=256),
                variant=dict(aggregation=agg, rank_pinned=rank, scope=scope, prompt_tokens=prompt_tokens,
                             prompt_topk=prompt_topk),
                splits=splits, deterministic=det)


def random_prompt_case(i: int) -> dict:
    """Seeded random configuration i with a long prompt region at a small
    batch (at most 16 units): 128 to 1200 prompt pages at page 8, 16 or 32,
    topk up to 40, prompts that fill a quarter of the region to more than
    all of it, a decode budget of at most 240 tokens, which the run passes;
    fp32 pools every sixth case, the score aggregation, the sequence scope,
    forced splits and the deterministic option drawn as in random_case. These
    reach the plan's choices for prompt regions at small batch: the fused
    workgroup's own selection, the selection kernel with and without the
    separate interval kernel, and the fp32 selection kernel."""
    import math

    rng = np.random.default_rng(9000 + i)
    dtype = "f32" if i % 6 == 5 else "bf16"  # (every sixth: the fp32 selection kernel)
    d = int(rng.choice([64, 128]))
    G = int(rng.choice([1, 2, 4, 7, 8]))
    hkv = int(rng.choice([1, 2, 4, 8]))
    batch = int(rng.integers(1, 16 // hkv + 1))
    ps = int(rng.choice([8, 16, 32]))
    unit = ps * 32 // math.gcd(ps, 32)
    prompt_tokens = unit * int(rng.integers(128 * ps // unit, min(16384, 1200 * ps) // unit + 1))
    npr = prompt_tokens // ps
    budget = ps * int(rng.integers(4, max(4, 240 // ps) + 1))
    prefill = int(rng.integers(prompt_tokens // 4, prompt_tokens + budget + 1))
    prompt_topk = int(rng.integers(1, min(40, npr) + 1))
    r = float(rng.choice([0.25, 0.5, 0.7, 0.9]))
    agg = int(rng.random() < 0.2)
    scope = int(rng.random() < 0.1)
    splits = None if rng.random() < 0.7 else int(rng.integers(2, 6))
    det = bool(rng.random() < 0.1)
    steps = int(budget + 3 * ps + 40)
    return dict(workload=dict(name="random-prompt-%02d" % i, batch=batch, n_layers=1, n_q_heads=G * hkv,
                              n_kv_heads=hkv, head_dim=d, dtype=dtype, page_size=ps, budget=budget,
                              prefill_len=prefill, decode_steps=steps, r=r, ms_period=16,
                              ms_phase_random=True, ms_wmin=8, ms_wmax=64),
                variant=dict(aggregation=agg, rank_pinned=False, scope=scope, prompt_tokens=prompt_tokens,
                             prompt_topk=prompt_topk),
                splits=splits, deterministic=det)


def unit_index(w, seq, kvh):
    return seq * w.n_kv_heads + kvh


def compare_outputs(got, want, dtype: str, what: str, rep: ParityReport):
    """got, want: [..][G][d] outputs of the same units. Checks the absolute
    bound per element and the relative L2 bound per head."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    diff = got - want
    err = float(np.max(np.abs(diff))) if diff.size else 0.0
    rel = np.linalg.norm(diff, axis=-1) / np.maximum(np.linalg.norm(want, axis=-1), 1e-30)
    rel_max = float(np.max(rel)) if rel.size else 0.0
    rep.max_abs_err = max(rep.max_abs_err, err)
    rep.max_rel_err = max(rep.max_rel_err, rel_max)
    rep.outputs_compared += int(np.prod(got.shape[:-2])) if got.ndim > 2 else 1
    if not (err <= TOL[dtype]):
        raise AssertionError("output mismatch: %s: max abs err %.3g > %g" % (what, err, TOL[dtype]))
    if not (rel_max <= TOL_REL[dtype]):
        idx = np.unravel_index(int(np.argmax(rel)), rel.shape)
        raise AssertionError("output mismatch: %s: relative L2 error %.3g > %g at %s"
                             % (what, rel_max, TOL_REL[dtype], idx))


def _flagged_pages(scores, theta):
    """Ranked pages within NEAR_TIE of the threshold (none without a finite threshold)."""
    if theta is None or not math.isfinite(theta):
        return set()
    ok = ~np.isnan(scores)
    return set(int(s) for s in np.nonzero(ok & (np.abs(np.where(ok, scores, 0.0) - theta) <= NEAR_TIE))[0])


def _victims(pt_o, pt_g):
    """slots whose page differs only because the two sides evicted different pages"""
    return set(int(s) for s in np.nonzero(((pt_o == -1) | (pt_g == -1)) & (pt_o != pt_g))[0])


def _resync_or_fail(w, seed, layer, t, members, orc, pt_g, ts_g, ev_g, scores, theta, rep, where):
    """A retention mismatch of one decision (members: its units, rows of
    pt_g/ts_g/ev_g by unit): re-sync the oracle when it is confined to a
    near tie, else fail."""
    flagged = _flagged_pages(scores, theta)
    for u in members:
        st = orc[u].state()
        if np.array_equal(st["page_table"], pt_g[u]) and np.array_equal(st["ts"], ts_g[u]) \
                and st["evicted"] == ev_g[u]:
            continue
        bad = set(np.nonzero(st["ts"] != ts_g[u])[0]) | set(np.nonzero(st["page_table"] != pt_g[u])[0])
        if len(flagged) >= 2 and bad <= flagged | _victims(st["page_table"], pt_g[u]):
            orc[u].adopt_retention(pt_g[u], ts_g[u], ev_g[u])
            st2 = orc[u].state()
            assert np.array_equal(st2["page_table"], pt_g[u]) and np.array_equal(st2["ts"], ts_g[u]), u
            rep.flagged_divergences += 1
            rep.first_divergence.setdefault(int(u), int(t))
            rep.notes.append("unit %d step %d: near-tie divergence, oracle re-synced" % (u, t))
            continue
        raise AssertionError(
            "retention mismatch (%s): workload %s seed %d layer %d unit %d step %d\n"
            "oracle pt %s\n   gpu pt %s\noracle ts %s\n   gpu ts %s\noracle ev %d gpu ev %d\nnear-tie pages %s"
            % (where, w.name, seed, layer, u, t, st["page_table"].tolist(), pt_g[u].tolist(),
               st["ts"].tolist(), ts_g[u].tolist(), st["evicted"], ev_g[u], sorted(flagged)))


def run_parity(w, seed: int, steps: int, layer: int = 0, units=None, out_every: int = 1,
               splits=None, chunk: int = 64, pool=None, prefill_len=None, check_invariants=True,
               report: ParityReport | None = None, aggregation: int = 0,
               rank_pinned: bool = False, scope: int = 0, prompt_tokens: int = 0,
               prompt_topk: int = 0, others: str = "exact", out_units=None, inv_every: int = 1,
               progress_s: float = 20.0) -> ParityReport:
    """Runs `steps` decode steps of workload `w` on the GPU and checks the
    listed units (all when None) against the oracle, step by step.

    aggregation, rank_pinned and scope select the variants on both sides;
    with scope 1 (one page table per sequence) every KV head of a listed
    unit's sequence is checked, the oracle stepping each sequence's units
    together. prompt_tokens/prompt_topk select Quest on the prompt (a prompt
    region of that many tokens, the top prompt_topk prompt pages attended
    per step).

    others: "exact", every unit gets its own seeded inputs; "ring", only the
    checked units do, the others replay a ring of seeded steps of the same
    workload (independent units: it changes nothing for the checked ones,
    and saves generating the whole batch at every step of long runs).
    out_units: the checked units whose outputs are compared (default all),
    every out_every-th step and at the last. inv_every: every unit is
    checked against the invariants every inv_every-th step.

    The GPU runs one chunk of steps ahead of the oracle: the host copies of
    a chunk's results arrive while the next chunk computes."""
    import torch

    rep = report or ParityReport()
    B, Hq, Hkv, d, G, ps = w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.group, w.page_size
    npr = prompt_tokens // ps
    S = w.slots + npr
    U = B * Hkv
    P = w.prefill_len if prefill_len is None else prefill_len
    units = list(range(U)) if units is None else sorted(set(units))
    if scope == 1:
        units = sorted({b * Hkv + h for b in {u // Hkv for u in units} for h in range(Hkv)})
    out_units = units if out_units is None else sorted(set(out_units) & set(units))
    nu = len(units)
    pos = {u: i for i, u in enumerate(units)}
    out_pos = np.array([pos[u] for u in out_units], np.int64)
    rest_pos = np.array([pos[u] for u in units if u not in set(out_units)], np.int64)
    own_pool = pool is None
    if own_pool:
        pool = new_pool(w, splits, aggregation=aggregation, rank_pinned=rank_pinned, scope=scope,
                        prompt_tokens=prompt_tokens, prompt_topk=prompt_topk)
    if others == "exact" or P == 0:
        Kp, Vp = synth.prefill(w, seed, layer, prefill_len=P)
        Kc, Vc = Kp.reshape(U, P, d)[units], Vp.reshape(U, P, d)[units]
    else:
        # the checked units' prompts exactly; the others repeat the first one's
        Kc, Vc = synth.prefill_units(w, seed, layer, P, units)
        Kp = np.broadcast_to(Kc[:1], (U, P, d)).copy()
        Vp = np.broadcast_to(Vc[:1], (U, P, d)).copy()
        Kp[units], Vp[units] = Kc, Vc
        Kp, Vp = Kp.reshape(B, Hkv, P, d), Vp.reshape(B, Hkv, P, d)
    pool.prefill(layer, to_device(Kp, w.dtype) if P else None, to_device(Vp, w.dtype) if P else None)
    del Kp, Vp
    orc = {}
    for i, u in enumerate(units):
        m = oracle.Kvm(G, d, ps, S, r=w.r, aggregation=aggregation, rank_pinned=rank_pinned,
                       prompt_slots=npr if prompt_topk else None, prompt_topk=prompt_topk or None)
        rc = m.prefill(Kc[i].astype(np.float64), Vc[i].astype(np.float64))
        assert rc == 0, rc
        orc[u] = m
    del Kc, Vc
    ms = [orc[u] for u in units]
    ms_out = [ms[i] for i in out_pos]
    ms_rest = [ms[i] for i in rest_pos]
    groups = {}
    for u in units:
        groups.setdefault(u - u % Hkv if scope == 1 else u, []).append(u)
    rep.units_checked += nu
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    units_t = torch.tensor(units, dtype=torch.long, device="cuda")
    if others == "ring":
        R = min(64, steps)
        ring = [to_device(a, w.dtype) for a in synth.steps(w, seed + 7919, layer, 0, R)]

    def launch(t0, n):
        keep = []
        if others == "exact":
            q, k, v = synth.steps(w, seed, layer, t0, n)
            qd, kd, vd = (_to_device_async(a, w.dtype, keep) for a in (q, k, v))
            qc = q.reshape(n, U, G, d)[:, units]
            kc = k.reshape(n, U, d)[:, units]
            vc = v.reshape(n, U, d)[:, units]
        else:
            qc, kc, vc = synth.steps_units(w, seed, layer, t0, n, units)
            idx = torch.arange(t0, t0 + n, device="cuda") % R
            qd, kd, vd = (x.index_select(0, idx) for x in ring)
            qd.view(n, U, G, d)[:, units_t] = _to_device_async(qc, w.dtype, keep)
            kd.view(n, U, d)[:, units_t] = _to_device_async(kc, w.dtype, keep)
            vd.view(n, U, d)[:, units_t] = _to_device_async(vc, w.dtype, keep)
        out = torch.empty((n, B, Hq, d), dtype=dt, device="cuda")
        pt = torch.empty((n, B, Hkv, S), dtype=torch.int32, device="cuda")
        ts = torch.empty((n, B, Hkv, S), dtype=torch.int32, device="cuda")
        ev = torch.empty((n, B, Hkv), dtype=torch.int32, device="cuda")
        for i in range(n):
            pool.decode_step(layer, qd[i], kd[i], vd[i], out[i], pt[i], ts[i], ev[i])
        want = [i for i in range(n) if (t0 + i) % out_every == 0 or t0 + i == steps - 1]
        inv = [i for i in range(n) if check_invariants and (t0 + i) % inv_every == 0]
        want_t = torch.tensor(want, dtype=torch.long, device="cuda")
        inv_t = torch.tensor(inv, dtype=torch.long, device="cuda")
        h = dict(
            t0=t0, n=n, want=want, inv=inv, qc=qc, kc=kc, vc=vc,
            out=_to_host_async(out.view(n, U, G, d).index_select(0, want_t)[:, units_t], keep),
            pt=_to_host_async(pt.view(n, U, S)[:, units_t], keep),
            ts=_to_host_async(ts.view(n, U, S)[:, units_t], keep),
            ev=_to_host_async(ev.view(n, U)[:, units_t], keep),
            pt_all=_to_host_async(pt.view(n, U, S).index_select(0, inv_t), keep),
            ts_all=_to_host_async(ts.view(n, U, S).index_select(0, inv_t), keep),
            ev_all=_to_host_async(ev.view(n, U), keep),
            keep=keep, done=torch.cuda.Event())
        h["done"].record()
        return h

    def process(h):
        h["done"].synchronize()
        t0, n = h["t0"], h["n"]
        out_h = h["out"].float().numpy()
        pt_h, ts_h, ev_h = h["pt"].numpy(), h["ts"].numpy(), h["ev"].numpy()
        ev_any = np.nonzero(np.any(h["ev_all"].numpy() >= 0, axis=1))[0]
        rep.evictions += int(np.sum(h["ev_all"].numpy() >= 0))
        if len(ev_any) and rep.first_eviction_step < 0:
            rep.first_eviction_step = int(t0 + ev_any[0])
        for j, i in enumerate(h["inv"]):
            _check_invariants(h["pt_all"][j].numpy(), h["ts_all"][j].numpy(), h["ev_all"][i].numpy(),
                              P + t0 + i, P, ps, S, npr)
            rep.invariant_checks += 1
        wi = {i: j for j, i in enumerate(h["want"])}
        for i in range(n):
            t = t0 + i
            q64, k64, v64 = h["qc"][i], h["kc"][i], h["vc"][i]
            outs = None
            if scope == 1:
                outs = np.empty((nu, G, d)) if i in wi else None
                for g, members in groups.items():
                    mi = [pos[u] for u in members]
                    o = oracle.decode_group([orc[u] for u in members], q64[mi], k64[mi], v64[mi],
                                            want_out=i in wi)
                    if o is not None:
                        outs[mi] = o
            else:
                if i in wi:
                    o = oracle.decode_batch(ms_out, q64[out_pos], k64[out_pos], v64[out_pos], want_out=True)
                    if len(ms_rest):
                        oracle.decode_batch(ms_rest, q64[rest_pos], k64[rest_pos], v64[rest_pos], want_out=False)
                else:
                    oracle.decode_batch(ms, q64, k64, v64, want_out=False)
            pt_o, ts_o, ev_o = oracle.state_batch(ms)
            sc, th = oracle.scores_batch(ms)
            near = ~np.isnan(sc) & (np.abs(np.nan_to_num(sc) - th[:, None]) <= NEAR_TIE) & np.isfinite(th)[:, None]
            nflag = near.sum(axis=1) >= 2
            rep.flagged_steps += int(np.sum(nflag[[pos[g] for g in groups]]))
            same = np.all(pt_o == pt_h[i], axis=1) & np.all(ts_o == ts_h[i], axis=1) & (ev_o == ev_h[i])
            if not np.all(same):
                bad_groups = sorted({units[j] - units[j] % Hkv if scope == 1 else units[j]
                                     for j in np.nonzero(~same)[0]})
                rows = {u: pos[u] for u in units}
                for g in bad_groups:
                    members = groups[g]
                    _resync_or_fail(w, seed, layer, t, members, orc,
                                    {u: pt_h[i][rows[u]] for u in members}, {u: ts_h[i][rows[u]] for u in members},
                                    {u: int(ev_h[i][rows[u]]) for u in members}, sc[pos[g]], th[pos[g]], rep,
                                    "lockstep")
            if i in wi:
                got = out_h[wi[i]]
                if scope == 1:
                    want = outs[out_pos]
                else:
                    want = o
                compare_outputs(got[out_pos], want, w.dtype,
                                "workload %s seed %d layer %d step %d" % (w.name, seed, layer, t), rep)
        rep.steps = t0 + n

    t_start = time.time()
    t_last = t_start
    pending = None
    for t0 in range(0, steps, chunk):
        h = launch(t0, min(chunk, steps - t0))
        if pending is not None:
            process(pending)
        pending = h
        now = time.time()
        if now - t_last >= progress_s:
            say("  %s: %d/%d steps (%.0f s)" % (w.name, pending["t0"], steps, now - t_start))
            t_last = now
    if pending is not None:
        process(pending)
    if own_pool:
        pool.close()
    return rep


def _check_invariants(pt, ts, ev, clock, P, ps, S, npr=0):
    """Properties that hold for every unit at any size (Algorithm 1, Sections 3.1-3.3).
    npr: slots of a prompt region (decode pages never enter it)."""
    pinned = min(-(-P // ps), npr if npr else S - 1)
    assert np.all(pt[:, pinned:npr] == -1), "a decode page in the prompt region"
    # prefill pages stay in slots 0..pinned-1 with their own ids and no timestamp
    assert np.all(pt[:, :pinned] == np.arange(pinned)[None, :]), "pinned pages moved"
    assert np.all(ts[:, :pinned] == -1)
    # decode pages carry ids above the prefill's and timestamps no later than now
    dec = pt[:, pinned:]
    dts = ts[:, pinned:]
    assert np.all((dec == -1) | (dec >= -(-P // ps)))
    assert np.all((dec == -1) == (dts == -1))
    assert np.all(dts <= clock) and np.all((dts == -1) | (dts >= P))
    # logical ids are unique within a unit
    srt = np.sort(pt, axis=1)
    assert not np.any((srt[:, 1:] == srt[:, :-1]) & (srt[:, 1:] >= 0)), "duplicate page id"
    # an eviction leaves exactly one free slot behind
    assert np.all((ev == -1) | (ev >= -(-P // ps)))
    nfree = np.sum(pt == -1, axis=1)
    assert np.all(nfree[ev >= 0] >= 1)


def run_ragged(w, seed: int, lens, steps: int, active_p: float = 0.75, reprefill=None, splits=None,
               aggregation: int = 0, rank_pinned: bool = False, scope: int = 0, prompt_tokens: int = 0,
               prompt_topk: int = 0) -> ParityReport:
    """Ragged batch: per-sequence prompt lengths (raas_prefill_ragged), a
    seeded per-step mask of the sequences that take a token
    (raas_decode_step_masked), and prompts replaced mid-run (reprefill: step
    -> {sequence: new length}, a re-prefill of those sequences alone before
    that step). Every unit is checked against an oracle that steps only
    when its sequence is active (near ties re-synced as in run_parity);
    inactive sequences' outputs must stay untouched; at the end the whole
    exported state must agree. prompt_tokens/prompt_topk: a prompt region
    with Quest on it, as in run_parity (each sequence keeps its own number
    of prompt pages)."""
    import torch

    rep = ParityReport()
    B, Hq, Hkv, d, G, ps = w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.group, w.page_size
    npr = prompt_tokens // ps
    S = w.slots + npr
    U = B * Hkv
    reprefill = reprefill or {}
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    rng = np.random.default_rng(seed + 17)
    pool = new_pool(w, splits, aggregation=aggregation, rank_pinned=rank_pinned, scope=scope,
                    prompt_tokens=prompt_tokens, prompt_topk=prompt_topk)
    orc = {}

    def prompt(lens_now, mask, pseed):
        max_len = max([int(x) for x, m in zip(lens_now, mask) if m] + [0])
        Kp, Vp = synth.prefill(w, pseed, 0, prefill_len=max_len)
        pool.prefill_ragged(0, to_device(Kp, w.dtype) if max_len else None,
                            to_device(Vp, w.dtype) if max_len else None, lens_now, mask)
        for b in range(B):
            if not mask[b]:
                continue
            for h in range(Hkv):
                m = oracle.Kvm(G, d, ps, S, r=w.r, aggregation=aggregation, rank_pinned=rank_pinned,
                               prompt_slots=npr if prompt_topk else None, prompt_topk=prompt_topk or None)
                P = int(lens_now[b])
                assert m.prefill(Kp[b, h, :P].astype(np.float64), Vp[b, h, :P].astype(np.float64)) == 0
                orc[b * Hkv + h] = m

    lens_now = [int(x) for x in lens]
    prompt(lens_now, [1] * B, seed)
    groups = {b: [b * Hkv + h for h in range(Hkv)] for b in range(B)} if scope == 1 else {u: [u] for u in range(U)}
    rep.units_checked = U
    for t in range(steps):
        if t in reprefill:
            mask = [1 if b in reprefill[t] else 0 for b in range(B)]
            for b, P in reprefill[t].items():
                lens_now[b] = int(P)
            prompt(lens_now, mask, seed + 1000 + t)
        act = (rng.random(B) < active_p).astype(np.int32)
        q, k, v = synth.steps(w, seed, 0, t, 1)
        out = torch.full((B, Hq, d), 7.0, dtype=dt, device="cuda")
        pt = torch.full((B, Hkv, S), -7, dtype=torch.int32, device="cuda")
        ts = torch.full((B, Hkv, S), -7, dtype=torch.int32, device="cuda")
        ev = torch.full((B, Hkv), -7, dtype=torch.int32, device="cuda")
        pool.decode_prepared(pool.prepare_step(0, to_device(q[0], w.dtype), to_device(k[0], w.dtype),
                                               to_device(v[0], w.dtype), out, pt, ts, ev,
                                               active=torch.from_numpy(act).cuda()))
        torch.cuda.synchronize()
        out_h = out.float().cpu().numpy().reshape(U, G, d)
        pt_h, ts_h, ev_h = (x.cpu().numpy().reshape(U, -1) for x in (pt, ts, ev))
        q64, k64, v64 = q[0].reshape(U, G, d), k[0].reshape(U, d), v[0].reshape(U, d)
        for g, members in groups.items():
            b = members[0] // Hkv
            if not act[b]:
                for u in members:
                    assert np.all(out_h[u] == 7.0) and np.all(pt_h[u] == -7) and np.all(ts_h[u] == -7) \
                        and np.all(ev_h[u] == -7), "inactive sequence %d touched at step %d" % (b, t)
                continue
            if len(members) == 1:
                outs = {members[0]: orc[members[0]].decode(q64[members[0]], k64[members[0]], v64[members[0]])}
            else:
                o = oracle.decode_group([orc[u] for u in members], q64[members], k64[members], v64[members])
                outs = {u: o[j] for j, u in enumerate(members)}
            scores, theta = orc[members[0]].last_scores()
            if len(_flagged_pages(scores, theta)) >= 2:
                rep.flagged_steps += 1
            _resync_or_fail(w, seed, 0, t, members, orc, pt_h, ts_h, {u: int(ev_h[u, 0]) for u in members},
                            scores, theta, rep, "ragged")
            for u in members:
                rep.evictions += int(ev_h[u, 0] >= 0)
                compare_outputs(out_h[u][None], outs[u][None], w.dtype, "ragged unit %d step %d" % (u, t), rep)
        rep.steps = t + 1
    gs = pool.export_state(0)
    for u in range(U):
        st = orc[u].state()
        assert np.array_equal(np.where(gs["state"][u] == 0, -1, gs["lid"][u]), st["page_table"]), u
        assert gs["clock"][u] == st["clock"] and gs["tail"][u] == st["tail"], u
    pool.close()
    return rep
