"""Lockstep parity harness: the HIP decode path against the CPU oracle.

Both sides get the same seeded inputs (``synth``); the oracle runs free on
the units it checks and never sees anything the GPU produced. Per step and
checked unit:
  - page table, timestamps and evicted page must be bit-exact, except when
    the oracle flags the step's threshold as a near-tie (two or more
    evictable pages within NEAR_TIE of the threshold score); a mismatch
    confined to flagged pages is counted and ends the comparison of that
    unit, any other mismatch fails;
  - attention outputs must agree within the tolerance of the dtype.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

import oracle
import synth

NEAR_TIE = 1e-6
TOL = {"bf16": 2e-2, "f32": 1e-4}


@dataclasses.dataclass
class ParityReport:
    steps: int = 0
    units_checked: int = 0
    outputs_compared: int = 0
    max_abs_err: float = 0.0
    flagged_steps: int = 0
    flagged_divergences: int = 0
    evictions: int = 0
    notes: list = dataclasses.field(default_factory=list)


def to_device(a: np.ndarray, dtype: str):
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a))
    t = t.to(torch.bfloat16) if dtype == "bf16" else t.to(torch.float32)
    return t.cuda()


def new_pool(w, splits=None, policy=None, aggregation=0, rank_pinned=False, scope=0, prompt_tokens=0,
             prompt_topk=0):
    import paper_2502_11147_amd as raas

    kw = {"score_aggregation": aggregation, "rank_pinned": rank_pinned, "decision_scope": scope,
          "prompt_tokens": prompt_tokens, "prompt_topk": prompt_topk}
    if policy is not None:
        kw["prefill_policy"] = policy
    pool = raas.Pool.for_workload(w, **kw)
    if splits is not None:
        pool.set_attention_splits(splits)
    return pool


def unit_index(w, seq, kvh):
    return seq * w.n_kv_heads + kvh


def run_parity(w, seed: int, steps: int, layer: int = 0, units=None, out_every: int = 1,
               splits=None, chunk: int = 64, pool=None, prefill_len=None, check_invariants=True,
               report: ParityReport | None = None, aggregation: int = 0,
               rank_pinned: bool = False, scope: int = 0, prompt_tokens: int = 0,
               prompt_topk: int = 0) -> ParityReport:
    """Runs `steps` decode steps of workload `w` on the GPU and checks the
    listed units (all when None) against the oracle. aggregation,
    rank_pinned and scope select the variants on both sides; with scope 1
    (one page table per sequence) every KV head of a listed unit's sequence
    is checked, the oracle stepping each sequence's units together.
    prompt_tokens/prompt_topk select Quest on the prompt (a prompt region of
    that many tokens, the top prompt_topk prompt pages attended per step)."""
    import torch

    rep = report or ParityReport()
    B, Hq, Hkv, d, G, ps = w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.group, w.page_size
    npr = prompt_tokens // ps
    S = w.slots + npr
    U = B * Hkv
    P = w.prefill_len if prefill_len is None else prefill_len
    units = list(range(U)) if units is None else list(units)
    if scope == 1:
        units = sorted({b * Hkv + h for b in {u // Hkv for u in units} for h in range(Hkv)})
    tol = TOL[w.dtype]
    own_pool = pool is None
    if own_pool:
        pool = new_pool(w, splits, aggregation=aggregation, rank_pinned=rank_pinned, scope=scope,
                        prompt_tokens=prompt_tokens, prompt_topk=prompt_topk)
    Kp, Vp = synth.prefill(w, seed, layer, prefill_len=P)
    pool.prefill(layer, to_device(Kp, w.dtype) if P else None, to_device(Vp, w.dtype) if P else None)
    orc = {}
    for u in units:
        b, h = divmod(u, Hkv)
        m = oracle.Kvm(G, d, ps, S, r=w.r, aggregation=aggregation, rank_pinned=rank_pinned,
                       prompt_slots=npr if prompt_topk else None, prompt_topk=prompt_topk or None)
        rc = m.prefill(Kp[b, h].astype(np.float64), Vp[b, h].astype(np.float64))
        assert rc == 0, rc
        orc[u] = m
    # decision groups: the units deciding together, keyed by their first unit
    groups = {}
    for u in units:
        groups.setdefault(u - u % Hkv if scope == 1 else u, []).append(u)
    live = set(groups)
    rep.units_checked += len(units)
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    for t0 in range(0, steps, chunk):
        n = min(chunk, steps - t0)
        q, k, v = synth.steps(w, seed, layer, t0, n)
        qd, kd, vd = to_device(q, w.dtype), to_device(k, w.dtype), to_device(v, w.dtype)
        out = torch.empty((n, B, Hq, d), dtype=dt, device="cuda")
        pt = torch.empty((n, B, Hkv, S), dtype=torch.int32, device="cuda")
        ts = torch.empty((n, B, Hkv, S), dtype=torch.int32, device="cuda")
        ev = torch.empty((n, B, Hkv), dtype=torch.int32, device="cuda")
        for i in range(n):
            pool.decode_step(layer, qd[i], kd[i], vd[i], out[i], pt[i], ts[i], ev[i])
        torch.cuda.synchronize()
        out_h = out.float().cpu().numpy().reshape(n, U, G, d)
        pt_h = pt.cpu().numpy().reshape(n, U, S)
        ts_h = ts.cpu().numpy().reshape(n, U, S)
        ev_h = ev.cpu().numpy().reshape(n, U)
        q64 = q.reshape(n, U, G, d)
        k64 = k.reshape(n, U, d)
        v64 = v.reshape(n, U, d)
        for i in range(n):
            t = t0 + i
            clock = P + t
            want_out = (t % out_every == 0) or t == steps - 1
            rep.evictions += int(np.sum(ev_h[i] >= 0))
            if check_invariants:
                _check_invariants(pt_h[i], ts_h[i], ev_h[i], clock, P, ps, S, npr)
            for g in sorted(live):
                members = groups[g]
                if len(members) == 1:
                    u = members[0]
                    outs = {u: orc[u].decode(q64[i, u], k64[i, u], v64[i, u], want_out=want_out)}
                else:
                    o = oracle.decode_group([orc[u] for u in members], q64[i, members], k64[i, members],
                                            v64[i, members], want_out=want_out)
                    outs = {u: (None if o is None else o[j]) for j, u in enumerate(members)}
                scores, theta = orc[members[0]].last_scores()
                flagged = _flagged_pages(scores, theta)
                if len(flagged) >= 2:
                    rep.flagged_steps += 1
                for u in members:
                    st = orc[u].state()
                    same_pt = np.array_equal(st["page_table"], pt_h[i, u])
                    same_ts = np.array_equal(st["ts"], ts_h[i, u])
                    same_ev = st["evicted"] == ev_h[i, u]
                    if not (same_pt and same_ts and same_ev):
                        bad = set(np.nonzero(st["ts"] != ts_h[i, u])[0]) | set(
                            np.nonzero(st["page_table"] != pt_h[i, u])[0])
                        if len(flagged) >= 2 and bad <= flagged | _victims(st, pt_h[i, u]):
                            rep.flagged_divergences += 1
                            rep.notes.append("unit %d step %d: flagged near-tie divergence" % (u, t))
                            live.discard(g)
                            break
                        raise AssertionError(
                            "retention mismatch: workload %s seed %d layer %d unit %d step %d\n"
                            "oracle pt %s\n   gpu pt %s\noracle ts %s\n   gpu ts %s\noracle ev %d gpu ev %d"
                            % (w.name, seed, layer, u, t, st["page_table"].tolist(), pt_h[i, u].tolist(),
                               st["ts"].tolist(), ts_h[i, u].tolist(), st["evicted"], ev_h[i, u]))
                    if want_out:
                        err = float(np.max(np.abs(out_h[i, u].astype(np.float64) - outs[u])))
                        rep.max_abs_err = max(rep.max_abs_err, err)
                        rep.outputs_compared += 1
                        if not (err <= tol):
                            raise AssertionError("output mismatch: workload %s seed %d layer %d unit %d step %d: "
                                                 "max abs err %.3g > %g" % (w.name, seed, layer, u, t, err, tol))
        rep.steps = t0 + n
    if own_pool:
        pool.close()
    return rep


def _flagged_pages(scores, theta):
    if theta is None or not math.isfinite(theta):
        return set()
    ok = ~np.isnan(scores)
    return set(int(s) for s in np.nonzero(ok & (np.abs(np.where(ok, scores, 0.0) - theta) <= NEAR_TIE))[0])


def _victims(st, gpu_pt):
    """slots whose page differs only because the two sides evicted different pages"""
    return set(int(s) for s in np.nonzero((st["page_table"] == -1) | (gpu_pt == -1))[0])


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
    for row in pt:
        live = row[row >= 0]
        assert len(np.unique(live)) == len(live), "duplicate page id"
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
    when its sequence is active; inactive sequences' outputs must stay
    untouched; at the end the whole exported state must agree.
    prompt_tokens/prompt_topk: a prompt region with Quest on it, as in
    run_parity (each sequence keeps its own number of prompt pages)."""
    import torch

    rep = ParityReport()
    B, Hq, Hkv, d, G, ps = w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.group, w.page_size
    npr = prompt_tokens // ps
    S = w.slots + npr
    U = B * Hkv
    reprefill = reprefill or {}
    tol = TOL[w.dtype]
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
            for u in members:
                st = orc[u].state()
                if not (np.array_equal(st["page_table"], pt_h[u]) and np.array_equal(st["ts"], ts_h[u])
                        and st["evicted"] == ev_h[u, 0]):
                    raise AssertionError("ragged retention mismatch: unit %d step %d\noracle pt %s\n   gpu pt %s\n"
                                         "oracle ts %s\n   gpu ts %s" % (u, t, st["page_table"].tolist(),
                                                                         pt_h[u].tolist(), st["ts"].tolist(),
                                                                         ts_h[u].tolist()))
                rep.evictions += int(st["evicted"] >= 0)
                err = float(np.max(np.abs(out_h[u].astype(np.float64) - outs[u])))
                rep.max_abs_err = max(rep.max_abs_err, err)
                rep.outputs_compared += 1
                if not (err <= tol):
                    raise AssertionError("ragged output mismatch: unit %d step %d: %.3g" % (u, t, err))
        rep.steps = t + 1
    gs = pool.export_state(0)
    for u in range(U):
        st = orc[u].state()
        assert np.array_equal(np.where(gs["state"][u] == 0, -1, gs["lid"][u]), st["page_table"]), u
        assert gs["clock"][u] == st["clock"] and gs["tail"][u] == st["tail"], u
    pool.close()
    return rep
