"""Retention policies to set beside page-level RaaS -- TEST INFRASTRUCTURE ONLY.

Oracle-only references (no GPU code implements them): plain fp64 numpy
statements of the policies the paper compares with (Section 4: dense
attention, StreamingLLM's sink-plus-window, H2O's heavy hitters, Quest's
query-aware page selection) and of token-level RaaS (Section 3.2, the policy
before Section 3.3 moves it to pages). They run on the same synthetic streams
as the decode path, so that the output deviation from dense attention and the
recall of planted milestone tokens can be compared without datasets (a
dataset-free analogue of the paper's accuracy comparison, Figure 5).

Every policy sees one unit (one KV head with its G query heads). A step
attends over the tokens the policy keeps (or, for Quest, selects) plus the
new token, then stores the new token, then evicts when the cache is full
(Algorithm 1's order). Budgets are in tokens: a cache of capacity L holds at
most L-1 tokens between steps, so a step attends over at most L tokens -- the
same count as the page-level oracle with page size 1.
"""
from __future__ import annotations

import math

import numpy as np


def attention(q, K, V):
    """Scaled dot-product attention of the G query rows over K/V rows (fp64).
    Returns the outputs [G][d] and the weights [G][n]."""
    d = q.shape[-1]
    logits = (q @ K.T) / math.sqrt(d)
    logits = logits - logits.max(axis=1, keepdims=True)
    w = np.exp(logits)
    w /= w.sum(axis=1, keepdims=True)
    return w @ V, w


class _Store:
    """Token store shared by the policies: every token's K/V by position."""

    def __init__(self, K, V):
        self.K = [np.asarray(x, np.float64) for x in K]
        self.V = [np.asarray(x, np.float64) for x in V]

    def add(self, k, v):
        self.K.append(np.asarray(k, np.float64))
        self.V.append(np.asarray(v, np.float64))
        return len(self.K) - 1

    def rows(self, pos):
        return np.array([self.K[p] for p in pos]), np.array([self.V[p] for p in pos])


class Dense:
    """Every token, no budget."""

    name = "dense"

    def __init__(self, K, V):
        self.st = _Store(K, V)
        self.keep = list(range(len(self.st.K)))

    def step(self, q, k, v):
        p = self.st.add(k, v)
        att = self.keep + [p]
        out, _ = attention(q, *self.st.rows(att))
        self.keep.append(p)
        return out, att


class Sink:
    """StreamingLLM: the first n_sink tokens plus the most recent ones, L in all."""

    name = "sink"

    def __init__(self, K, V, L, n_sink=4):
        self.st = _Store(K, V)
        self.L, self.n_sink = L, n_sink
        self.keep = list(range(len(self.st.K)))
        self._trim()

    def _trim(self):
        while len(self.keep) > self.L - 1:
            del self.keep[min(self.n_sink, len(self.keep) - 1)]

    def step(self, q, k, v):
        p = self.st.add(k, v)
        att = self.keep + [p]
        out, _ = attention(q, *self.st.rows(att))
        self.keep.append(p)
        self._trim()
        return out, att


class H2O:
    """Heavy-hitter oracle (Zhang et al. 2023): the `recent` most recent
    tokens plus those with the largest attention accumulated over the steps
    so far (summed over the G heads), L in all. The prompt is not pinned."""

    name = "h2o"

    def __init__(self, K, V, L, recent=None):
        self.st = _Store(K, V)
        self.L = L
        self.recent = L // 2 if recent is None else recent
        self.keep = list(range(len(self.st.K)))
        self.acc = {p: 0.0 for p in self.keep}
        self._trim()

    def _trim(self):
        while len(self.keep) > self.L - 1:
            old = self.keep[: max(0, len(self.keep) - self.recent)]
            # the lightest token outside the recent window; the oldest when
            # the window covers every token
            victim = min(old, key=lambda p: (self.acc[p], p)) if old else self.keep[0]
            self.keep.remove(victim)

    def step(self, q, k, v):
        p = self.st.add(k, v)
        att = self.keep + [p]
        out, w = attention(q, *self.st.rows(att))
        self.acc[p] = 0.0
        for pos, a in zip(att, w.sum(axis=0)):
            self.acc[pos] += float(a)
        self.keep.append(p)
        self._trim()
        return out, att


class Quest:
    """Quest (Tang et al. 2024): every token stays (O(N) memory); each step
    attends over the pages with the largest representative bound
    (max over the heads of sum_c max(q_c kmax_c, q_c kmin_c)), L // ps pages,
    always including the page of the newest tokens."""

    name = "quest"

    def __init__(self, K, V, L, ps):
        self.st = _Store(K, V)
        self.L, self.ps = L, ps

    def step(self, q, k, v):
        p = self.st.add(k, v)
        n = len(self.st.K)
        pages = [list(range(s, min(s + self.ps, n))) for s in range(0, n, self.ps)]
        budget = max(1, self.L // self.ps)
        if len(pages) <= budget:
            chosen = pages
        else:
            last = pages[-1]
            scored = []
            for i, pg in enumerate(pages[:-1]):
                Kp = np.array([self.st.K[t] for t in pg])
                lo, hi = Kp.min(axis=0), Kp.max(axis=0)
                b = np.maximum(q * hi, q * lo).sum(axis=1).max()
                scored.append((-b, i))
            top = sorted(scored)[: budget - 1]
            chosen = [pages[i] for _, i in sorted(top, key=lambda x: x[1])] + [last]
        att = [t for pg in chosen for t in pg]
        out, _ = attention(q, *self.st.rows(att))
        return out, att


class TokenRaaS:
    """Token-level RaaS (Section 3.2, Algorithm 1 on tokens): prompt tokens
    are pinned (the first min(P, L-1)); every decode token carries a
    timestamp, set to the clock when it is stored and whenever its attention
    weight (max over the G heads) is strictly above the (n-k)-th smallest
    among the n decode tokens of the step, k = floor(r n); when the cache is
    full the decode token with the oldest timestamp is evicted (ties: the
    older token)."""

    name = "raas-token"

    def __init__(self, K, V, L, r=0.5):
        self.st = _Store(K, V)
        self.L, self.r = L, r
        P = len(self.st.K)
        self.pinned = list(range(min(P, L - 1)))
        self.dec = []  # decode tokens, by position
        self.ts = {}
        self.clock = P

    def resident(self):
        return self.pinned + self.dec

    def step(self, q, k, v):
        c = self.clock
        p = self.st.add(k, v)
        att = self.resident() + [p]
        out, w = attention(q, *self.st.rows(att))
        self.dec.append(p)
        self.ts[p] = c
        score = dict(zip(att, w.max(axis=0)))
        n = len(self.dec)
        kk = math.floor(self.r * n)
        if kk > 0:
            vals = sorted(score[t] for t in self.dec)
            theta = -math.inf if kk == n else vals[n - kk - 1]
            for t in self.dec:
                if score[t] > theta:
                    self.ts[t] = c
        if len(self.pinned) + len(self.dec) >= self.L:
            victim = min(self.dec, key=lambda t: (self.ts[t], t))
            self.dec.remove(victim)
        self.clock = c + 1
        return out, att


class PageRaaS:
    """Page-level RaaS through the C oracle (the method this repository
    builds), with the same step interface."""

    name = "raas-page"

    def __init__(self, K, V, L, ps, r=0.5, lib=None):
        self.ps, self.L, self.r, self.lib = ps, L, r, lib
        self.K0, self.V0 = np.asarray(K, np.float64), np.asarray(V, np.float64)
        self.m = None  # created at the first step, when G and d are known
        self.P = len(self.K0)  # position of the next token

    def step(self, q, k, v):
        import oracle

        if self.m is None:
            self.m = oracle.Kvm(q.shape[0], q.shape[1], self.ps, self.L // self.ps, r=self.r, lib=self.lib)
            assert self.m.prefill(self.K0, self.V0) == 0
        st = self.m.state()
        att = self._positions(st) + [self.P]
        out = self.m.decode(q, k, v)
        self.P += 1
        return out, att

    def _positions(self, st):
        """positions of the resident tokens: logical page id l holds positions
        l*ps .. (prompt pages) or the decode tokens in order"""
        pos = []
        for s in range(len(st["state"])):
            if st["state"][s] == 0:
                continue
            lid, f = int(st["page_table"][s]), int(st["fill"][s])
            pos.extend(self._lid_start(lid) + i for i in range(f))
        return sorted(pos)

    def _lid_start(self, lid):
        P0 = len(self.K0)
        prompt_pages = -(-P0 // self.ps)
        if lid < prompt_pages:
            return lid * self.ps
        return P0 + (lid - prompt_pages) * self.ps


def evaluate(w, seed, seq, kvh, steps, policies, milestones=None):
    """Runs the policies (name -> factory(K, V)) and dense attention over one
    unit's stream for `steps` decode steps. Returns name -> metrics: mean and
    95th-percentile relative L2 deviation of the output from dense, milestone
    recall (the fraction of (step, active milestone) pairs whose milestone
    token the step attends to), and the most tokens held."""
    import synth

    Kp, Vp = synth.prefill(w, seed, 0)
    K = Kp[seq, kvh].astype(np.float64)
    V = Vp[seq, kvh].astype(np.float64)
    P = len(K)
    q, k, v = synth.steps(w, seed, 0, 0, steps)
    G = w.group
    dense = Dense(K, V)
    runs = {name: make(K, V) for name, make in policies.items()}
    err = {name: [] for name in runs}
    hits = {name: 0 for name in runs}
    held = {name: 0 for name in runs}
    total = 0
    for t in range(steps):
        qt = q[t, seq, kvh * G:(kvh + 1) * G].astype(np.float64)
        kt = k[t, seq, kvh].astype(np.float64)
        vt = v[t, seq, kvh].astype(np.float64)
        ref, _ = dense.step(qt, kt, vt)
        act = [P + m for m in synth.active_milestones(w, seed, 0, seq, kvh, t)] if milestones is None \
            else milestones(t)
        total += len(act)
        for name, pol in runs.items():
            out, att = pol.step(qt, kt, vt)
            err[name].append(float(np.linalg.norm(out - ref) / np.linalg.norm(ref)))
            s = set(att)
            hits[name] += sum(1 for a in act if a in s)
            held[name] = max(held[name], len(att))
    return {name: {"err_mean": float(np.mean(err[name])), "err_p95": float(np.percentile(err[name], 95)),
                   "milestone_recall": hits[name] / total if total else float("nan"),
                   "max_attended": held[name]} for name in runs}
