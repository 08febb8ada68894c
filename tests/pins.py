"""Checks that pin the CPU oracle to what the paper and the mathematics fix.

Each check takes the path of an oracle library and raises AssertionError on
failure, so the same checks run against the committed oracle (all must pass)
and against copies of it with a planted mistake (some check must fail).
"""
from __future__ import annotations

import itertools
import math

import numpy as np

import oracle
from oracle.history import HistoryLRU


def _softmax_attention(q, K, V):
    """Textbook scaled dot-product attention (Vaswani et al. 2017), fp64."""
    d = q.shape[-1]
    logits = np.einsum("gd,td->gt", q, K) / math.sqrt(d)
    logits -= logits.max(axis=1, keepdims=True)
    w = np.exp(logits)
    w /= w.sum(axis=1, keepdims=True)
    return w @ V


def _new_slot(st, ps, base=0):
    """The slot a decode step fills with a fresh page, given the state before
    the step (the lowest free slot from `base`, the first decode slot, when
    the tail page is full or absent)."""
    if st["tail"] >= 0 and st["fill"][st["tail"]] < ps:
        return None
    return min(s for s in range(base, len(st["state"])) if st["state"][s] == oracle.FREE)


def check_dense_equivalence(lib, G=3, d=16, ps=4, S=8, P=5, T=20, seed=1):
    """Budget >= sequence length: nothing is evicted and every step is exact
    dense attention over all tokens so far (Algorithm 1 with is_full never
    true)."""
    assert S * ps > P + T
    rng = np.random.default_rng(seed)
    m = oracle.Kvm(G, d, ps, S, lib=lib)
    K = rng.standard_normal((P, d))
    V = rng.standard_normal((P, d))
    assert m.prefill(K, V) == 0
    allK, allV = list(K), list(V)
    for t in range(T):
        q = rng.standard_normal((G, d)) * 2.0
        k = rng.standard_normal(d)
        v = rng.standard_normal(d)
        out = m.decode(q, k, v)
        allK.append(k)
        allV.append(v)
        ref = _softmax_attention(q, np.array(allK), np.array(allV))
        assert np.max(np.abs(out - ref)) < 1e-12, (t, np.max(np.abs(out - ref)))
        st = m.state()
        assert st["evicted"] == -1
        assert sum(st["fill"]) == P + t + 1


def check_single_token_and_bound(lib, G=4, d=32, ps=4, S=6, P=4, T=40, seed=2):
    """Representative score (Section 3.3 takes Quest's criterion): every
    page's score bounds q_j.k_i from above for each of its keys and each
    query head; a page holding one token scores exactly max_j q_j.k; a page
    whose keys are all equal attains the bound."""
    rng = np.random.default_rng(seed)
    m = oracle.Kvm(G, d, ps, S, lib=lib)
    assert m.prefill(rng.standard_normal((P, d)), rng.standard_normal((P, d))) == 0
    seen_single = 0
    for t in range(T):
        q = rng.standard_normal((G, d))
        m.decode(q, rng.standard_normal(d), rng.standard_normal(d), want_out=False)
        st = m.state()
        sc, _ = m.last_scores()
        K, _, _, _ = m.pages()
        scored_then_evicted = 0
        for s in range(S):
            if st["state"][s] != oracle.EVICTABLE:
                if not math.isnan(sc[s]):  # the page evicted at the end of this step
                    assert st["state"][s] == oracle.FREE and st["evicted"] >= 0
                    scored_then_evicted += 1
                continue
            logits = K[s, : st["fill"][s]] @ q.T  # [tokens][G]
            assert np.isfinite(sc[s])
            assert sc[s] >= logits.max() - 1e-12
            if st["fill"][s] == 1:
                seen_single += 1
                assert abs(sc[s] - logits.max()) <= 1e-12 * (1 + abs(logits.max()))
        assert scored_then_evicted <= 1
    assert seen_single > 0
    m = oracle.Kvm(1, d, ps, 3, lib=lib)
    assert m.prefill(None, None) == 0
    q = rng.standard_normal((1, d))
    k = rng.standard_normal(d)
    for _ in range(ps):
        m.decode(q, k, k, want_out=False)
    sc, _ = m.last_scores()
    exact = float(q[0] @ k)
    assert abs(sc[0] - exact) <= 1e-12 * (1 + abs(exact))


def check_threshold_counts(lib, seed=3):
    """Top-r (Algorithm 1; r = 0.5 means above the median, Section 3.2): with
    distinct scores exactly floor(r*n) of the n evictable pages get the
    latest timestamp, and they are the highest-scoring ones."""
    rng = np.random.default_rng(seed)
    ps, S = 1, 12
    for r in (0.5, 0.25, 0.75, 1.0 / 3.0, 0.0, 1.0, 0.1):
        m = oracle.Kvm(1, 4, ps, S, r=r, lib=lib)
        assert m.prefill(np.zeros((1, 4)), np.zeros((1, 4))) == 0
        for t in range(30):
            prev = m.state()
            new = _new_slot(prev, ps)
            live = [s for s in range(S) if prev["state"][s] == oracle.EVICTABLE]
            if new is not None:
                live.append(new)
            scores = rng.permutation(S).astype(np.float64) + rng.random()
            m.decode_with_scores(scores)
            st = m.state()
            c = prev["clock"]
            n = len(live)
            k = math.floor(r * n)
            top = set(sorted(live, key=lambda s: -scores[s])[:k])
            for s in live:
                if s == new or st["page_table"][s] == -1:
                    continue  # a fresh page has ts = c anyway; an evicted one is gone
                assert (st["ts"][s] == c) == (s in top), (r, t, s, st["ts"][s], c)
            assert st["n_evictable"] == n and st["k_refreshed"] == k


def check_fifo_special_cases(lib, seed=4):
    """r = 0 (never refreshed) and r = 1 (all refreshed, all tied) both reduce
    the policy to first-in first-out over decode pages: the resident decode
    pages are always the newest ones and pages leave in creation order."""
    rng = np.random.default_rng(seed)
    for r in (0.0, 1.0):
        for ps, S, P in ((1, 5, 3), (4, 6, 9), (2, 3, 0), (3, 7, 20)):
            G, d = 2, 8
            m = oracle.Kvm(G, d, ps, S, r=r, lib=lib)
            assert m.prefill(rng.standard_normal((P, d)), rng.standard_normal((P, d))) == 0
            pinned = min(-(-P // ps), S - 1)
            first = -(-P // ps)  # logical id of the first decode page
            room = S - pinned
            evicted = []
            for t in range(60):
                m.decode(rng.standard_normal((G, d)), rng.standard_normal(d),
                         rng.standard_normal(d), want_out=False)
                st = m.state()
                if st["evicted"] >= 0:
                    evicted.append(st["evicted"])
                n_pages = t // ps + 1
                tail_full = (t + 1) % ps == 0
                keep = room - 1 if (tail_full and n_pages >= room) else min(n_pages, room)
                newest = first + n_pages - 1
                lids = sorted(x for x in st["page_table"] if x >= first)
                assert lids == list(range(newest - keep + 1, newest + 1)), (r, ps, S, P, t, lids)
            assert evicted and evicted == list(range(first, first + len(evicted)))


def _drive_both(lib, ps, S, P, r, scores_for, T, rank_pinned=False):
    """Drive the oracle and the history-replay LRU with the same page scores.

    scores_for(t, n) gives the scores of the n pages ranked during step t
    (the decode pages alive, and the pinned ones when rank_pinned), in
    increasing logical-id order."""
    m = oracle.Kvm(1, 2, ps, S, r=r, lib=lib, rank_pinned=rank_pinned)
    assert m.prefill(np.zeros((P, 2)), np.zeros((P, 2))) == 0
    h = HistoryLRU(ps, S, r, P, rank_pinned=rank_pinned)
    for t in range(T):
        st = m.state()
        ranked_states = (oracle.EVICTABLE, oracle.PINNED) if rank_pinned else (oracle.EVICTABLE,)
        slot_lid = {s: int(st["page_table"][s]) for s in range(S) if st["state"][s] in ranked_states}
        new = _new_slot(st, ps)
        if new is not None:
            slot_lid[new] = st["next_lid"]
        alive = sorted(slot_lid.values())
        score_of = dict(zip(alive, scores_for(t, len(alive))))
        slot_scores = np.zeros(S)
        for s, lid in slot_lid.items():
            slot_scores[s] = score_of[lid]
        m.decode_with_scores(slot_scores)
        ev_h = h.decode(lambda lid: score_of[lid])
        st2 = m.state()
        assert (ev_h if ev_h is not None else -1) == st2["evicted"], (t, ev_h, st2["evicted"])
        res = sorted(int(x) for x in st2["page_table"] if x >= 0)
        assert res == h.resident_lids(), (t, res, h.resident_lids())


def _weak_orders(n):
    """every weak order (ranking with ties) of n items, as rank tuples"""
    out = []
    for ranks in itertools.product(range(n), repeat=n):
        if sorted(set(ranks)) == list(range(len(set(ranks)))):
            out.append(ranks)
    return out


def check_bruteforce_eviction_order(lib, strict_steps=6, weak_steps=4):
    """Exhaustive enumeration on a tiny pool (one pinned page, three decode
    slots, one token per page so every step makes a page): every total order
    of the page scores at every step for six steps, and every weak order
    (with ties) for four; the oracle must evict exactly the page the
    history-replay LRU definition names and keep the same resident set."""
    ps, S, P = 1, 4, 1
    room = S - 1
    for orders_of, steps in ((lambda n: list(itertools.permutations(range(n))), strict_steps),
                             (_weak_orders, weak_steps)):
        per_step = [orders_of(min(t + 1, room)) for t in range(steps)]
        count = 0
        for combo in itertools.product(*per_step):
            _drive_both(lib, ps, S, P, 0.5, lambda t, n, c=combo: [float(x) for x in c[t]], steps)
            count += 1
        assert count == math.prod(len(x) for x in per_step)


def check_random_policy_vs_history(lib, seed=5, cases=80):
    """Random scores with many ties, several r, page sizes, budgets and
    prefill lengths: oracle and history-replay LRU agree at every step."""
    rng = np.random.default_rng(seed)
    for _ in range(cases):
        ps = int(rng.integers(1, 5))
        S = int(rng.integers(2, 9))
        P = int(rng.integers(0, (S - 1) * ps + 1))
        r = float(rng.choice([0.5, 0.25, 0.75, 1 / 3, 0.6, 1.0]))
        T = int(rng.integers(5, 70))
        levels = int(rng.integers(2, 6))
        _drive_both(lib, ps, S, P, r,
                    lambda t, n: [float(x) for x in rng.integers(0, levels, size=n)], T)


def check_rank_pinned_vs_history(lib, seed=8, cases=60):
    """Variant: the pinned prompt pages ranked with the decode pages (n and
    k count them; only decode pages take timestamps). Random scores with
    ties over pinned and decode pages: oracle and history-replay LRU agree at
    every step, and the step reports n = pinned + decode pages."""
    rng = np.random.default_rng(seed)
    for _ in range(cases):
        ps = int(rng.integers(1, 4))
        S = int(rng.integers(3, 9))
        P = int(rng.integers(1, (S - 1) * ps + 1))
        r = float(rng.choice([0.5, 0.25, 0.75, 1.0]))
        T = int(rng.integers(5, 50))
        levels = int(rng.integers(2, 6))
        _drive_both(lib, ps, S, P, r,
                    lambda t, n: [float(x) for x in rng.integers(0, levels, size=n)], T, rank_pinned=True)
    m = oracle.Kvm(1, 2, 2, 6, r=0.5, lib=lib, rank_pinned=True)
    assert m.prefill(np.zeros((5, 2)), np.zeros((5, 2))) == 0  # 3 pinned pages
    for t in range(7):
        m.decode_with_scores(np.arange(6, dtype=float))
        st = m.state()
        pinned = int(np.sum(st["state"] == oracle.PINNED))
        decode = int(np.sum(st["state"] == oracle.EVICTABLE)) + (st["evicted"] >= 0)
        assert pinned == 3 and st["n_evictable"] == pinned + decode, (t, st)


def check_softmax_sum_invariants(lib, seed=9):
    """Variant: a page's score is the sum over the G heads of each head's
    softmax probability over the ranked pages. Then (i) the ranked scores
    sum to G at every step; (ii) a lone ranked page scores exactly G; (iii)
    with G = 1 the score is a monotone function of the representative bound,
    so retention is identical to the max rule (R2) step for step."""
    rng = np.random.default_rng(seed)
    for G, d, ps, S, P in ((4, 16, 4, 8, 6), (7, 8, 2, 12, 3), (2, 32, 8, 5, 9)):
        for rank_pinned in (False, True):
            m = oracle.Kvm(G, d, ps, S, lib=lib, aggregation=oracle.AGG_SOFTMAX_SUM, rank_pinned=rank_pinned)
            assert m.prefill(rng.standard_normal((P, d)), rng.standard_normal((P, d))) == 0
            for t in range(40):
                m.decode(rng.standard_normal((G, d)) * 2.0, rng.standard_normal(d), rng.standard_normal(d),
                         want_out=False)
                sc, _ = m.last_scores()
                ranked = sc[~np.isnan(sc)]
                assert abs(ranked.sum() - G) < 1e-12 * G, (G, t, ranked.sum())
                if ranked.size == 1:
                    assert ranked[0] == G
    # a lone decode page: two slots, one of them pinned
    m = oracle.Kvm(3, 8, 4, 2, lib=lib, aggregation=oracle.AGG_SOFTMAX_SUM)
    assert m.prefill(rng.standard_normal((4, 8)), rng.standard_normal((4, 8))) == 0
    for t in range(9):
        m.decode(rng.standard_normal((3, 8)), rng.standard_normal(8), rng.standard_normal(8), want_out=False)
        sc, _ = m.last_scores()
        assert sc[1] == 3.0 and np.isnan(sc[0]), (t, sc)
    # G = 1: same decisions as the max rule
    for rank_pinned in (False, True):
        a = oracle.Kvm(1, 16, 2, 7, lib=lib, rank_pinned=rank_pinned)
        b = oracle.Kvm(1, 16, 2, 7, lib=lib, aggregation=oracle.AGG_SOFTMAX_SUM, rank_pinned=rank_pinned)
        K, V = rng.standard_normal((5, 16)), rng.standard_normal((5, 16))
        assert a.prefill(K, V) == 0 and b.prefill(K, V) == 0
        for t in range(60):
            q, k, v = rng.standard_normal((1, 16)), rng.standard_normal(16), rng.standard_normal(16)
            a.decode(q, k, v, want_out=False)
            b.decode(q, k, v, want_out=False)
            sa, sb = a.state(), b.state()
            for key in ("page_table", "ts"):
                assert np.array_equal(sa[key], sb[key]), (rank_pinned, t, key)


def check_softmax_sum_golden(lib):
    """Variant V1 against a hand-worked step (tests/golden/
    softmax_sum_worked_example.json): three one-token pages whose refreshed
    page is A under the scale 1/sqrt(d) of the attention logits and would be
    B under scale 1; the scores match the worked values."""
    import json
    import os

    with open(os.path.join(os.path.dirname(__file__), "golden", "softmax_sum_worked_example.json")) as f:
        g = json.load(f)
    d, G = g["head_dim"], g["group"]
    m = oracle.Kvm(G, d, g["page_size"], g["slots"], r=g["r"], lib=lib, aggregation=oracle.AGG_SOFTMAX_SUM)
    assert m.prefill(None, None) == 0
    zero_q = np.zeros((G, d))
    for name, q in (("A", zero_q), ("B", zero_q), ("C", np.array(g["queries_step2"], float))):
        m.decode(q, np.array(g["keys"][name], float), np.zeros(d), want_out=False)
    sc, _ = m.last_scores()
    for slot, name in enumerate("ABC"):
        assert abs(sc[slot] - g["scores_step2"][name]) < 2e-7, (name, sc[slot], g["scores_step2"][name])
    st = m.state()
    assert st["page_table"].tolist() == g["page_table_after"], st["page_table"]
    assert st["ts"].tolist() == g["ts_after"], st["ts"]


def check_prefill_rule(lib, seed=6):
    """Prefill pages are stored, marked non-evictable and never change
    (Algorithm 1, Section 3.1). When the prefill does not fit, the first S-1
    pages are pinned and one slot is left, so each decode page is evicted as
    soon as it is full; the ERROR policy refuses instead."""
    rng = np.random.default_rng(seed)
    G, d, ps, S = 2, 8, 4, 5
    for P in (0, 3, 4, 13, 16):
        m = oracle.Kvm(G, d, ps, S, lib=lib)
        assert m.prefill(rng.standard_normal((P, d)), rng.standard_normal((P, d))) == 0
        K0, V0, _, _ = m.pages()
        st = m.state()
        pinned = [s for s in range(S) if st["state"][s] == oracle.PINNED]
        assert pinned == list(range(-(-P // ps)))
        assert [st["fill"][s] for s in pinned] == [min(ps, P - s * ps) for s in pinned]
        for t in range(50):
            m.decode(rng.standard_normal((G, d)), rng.standard_normal(d), rng.standard_normal(d),
                     want_out=False)
            st = m.state()
            K1, V1, _, _ = m.pages()
            for s in pinned:
                assert st["state"][s] == oracle.PINNED and st["page_table"][s] == s
                assert st["ts"][s] == -1
                assert np.array_equal(K1[s], K0[s]) and np.array_equal(V1[s], V0[s])
    P = 40  # 10 pages > S - 1 = 4
    m = oracle.Kvm(G, d, ps, S, lib=lib)
    assert m.prefill(rng.standard_normal((P, d)), rng.standard_normal((P, d))) == 0
    st = m.state()
    assert st["state"].tolist() == [oracle.PINNED] * (S - 1) + [oracle.FREE]
    assert st["page_table"][: S - 1].tolist() == list(range(S - 1))
    ev = []
    for t in range(6 * ps):
        m.decode(rng.standard_normal((G, d)), rng.standard_normal(d), rng.standard_normal(d),
                 want_out=False)
        st = m.state()
        assert st["state"][: S - 1].tolist() == [oracle.PINNED] * (S - 1)
        if st["evicted"] >= 0:
            ev.append((t, st["evicted"]))
    assert ev == [(ps * (i + 1) - 1, 10 + i) for i in range(6)]
    m = oracle.Kvm(G, d, ps, S, policy=oracle.ERROR, lib=lib)
    assert m.prefill(rng.standard_normal((P, d)), rng.standard_normal((P, d))) == oracle.E_BUDGET
    assert m.prefill(rng.standard_normal((16, d)), rng.standard_normal((16, d))) == 0
    assert m.prefill(rng.standard_normal((4, d)), rng.standard_normal((4, d))) == oracle.E_STATE


def check_budget_and_attention_set(lib, seed=7):
    """Resident tokens never exceed the budget L = S*ps (O(L) memory, Section
    4.3), and a step attends to exactly the resident tokens plus the new one:
    its output is textbook attention over that set and lies in the
    per-channel hull of the values."""
    rng = np.random.default_rng(seed)
    G, d, ps, S, P = 2, 8, 3, 5, 4
    m = oracle.Kvm(G, d, ps, S, lib=lib)
    assert m.prefill(rng.standard_normal((P, d)), rng.standard_normal((P, d))) == 0
    for t in range(80):
        st = m.state()
        K, V, _, _ = m.pages()
        res = [(s, i) for s in range(S) if st["state"][s] != oracle.FREE for i in range(st["fill"][s])]
        keys = [K[s, i] for s, i in res]
        vals = [V[s, i] for s, i in res]
        q = rng.standard_normal((G, d))
        k = rng.standard_normal(d)
        v = rng.standard_normal(d)
        out = m.decode(q, k, v)
        allv = np.array(vals + [v])
        ref = _softmax_attention(q, np.array(keys + [k]), allv)
        assert np.max(np.abs(out - ref)) < 1e-12
        assert np.all(out >= allv.min(axis=0) - 1e-12) and np.all(out <= allv.max(axis=0) + 1e-12)
        st = m.state()
        assert sum(st["fill"][s] for s in range(S) if st["state"][s] != oracle.FREE) <= S * ps
    m = oracle.Kvm(G, d, ps, S, lib=lib)
    assert m.prefill(None, None) == 0
    v = rng.standard_normal(d)
    out = m.decode(rng.standard_normal((G, d)), rng.standard_normal(d), v)
    assert np.array_equal(out, np.stack([v] * G))


def _ranked_slot_lids(st, ps, rank_pinned, base=0):
    """slot -> logical id of the pages a step ranks, from the state before it"""
    states = (oracle.EVICTABLE, oracle.PINNED) if rank_pinned else (oracle.EVICTABLE,)
    out = {s: int(st["page_table"][s]) for s in range(len(st["state"])) if st["state"][s] in states}
    new = _new_slot(st, ps, base)
    if new is not None:
        out[new] = st["next_lid"]
    return out


def check_group_single_token_pages(lib, seed=10):
    """One page table per (sequence, layer), shared by n KV heads (scope
    variant of R2). With one token per page the representative bound of a
    page is the logit of its token, so a page's grouped score is exactly
    max over the n*G query heads of q.k against the head's own KV head's key
    (max rule), or the sum over those heads of the token's softmax
    probability among the ranked tokens, scale 1/sqrt(d) (softmax rule).
    Every KV head keeps the same page table, and each head's output is
    textbook attention over its own resident tokens plus the new one."""
    rng = np.random.default_rng(seed)
    n, G, d, S, P = 3, 2, 8, 6, 3
    for agg, rank_pinned in ((0, False), (1, False), (0, True), (1, True)):
        ms = [oracle.Kvm(G, d, 1, S, lib=lib, aggregation=agg, rank_pinned=rank_pinned) for _ in range(n)]
        keys = [list(rng.standard_normal((P, d))) for _ in range(n)]  # with page size 1, token = lid
        vals = [list(rng.standard_normal((P, d))) for _ in range(n)]
        for h in range(n):
            assert ms[h].prefill(np.array(keys[h]), np.array(vals[h])) == 0
        for t in range(40):
            st0 = ms[0].state()
            resident = [int(x) for x in st0["page_table"] if x >= 0]
            ranked = _ranked_slot_lids(st0, 1, rank_pinned)
            q = rng.standard_normal((n, G, d)) * 1.5
            k = rng.standard_normal((n, d))
            v = rng.standard_normal((n, d))
            out = oracle.decode_group(ms, q, k, v)
            for h in range(n):
                keys[h].append(k[h])
                vals[h].append(v[h])
                ref = _softmax_attention(q[h], np.array([keys[h][x] for x in resident] + [k[h]]),
                                         np.array([vals[h][x] for x in resident] + [v[h]]))
                assert np.max(np.abs(out[h] - ref)) < 1e-12, (agg, t, h)
            sts = [m.state() for m in ms]
            for h in range(1, n):
                for key in ("page_table", "ts", "state", "fill"):
                    assert np.array_equal(sts[h][key], sts[0][key]), (agg, t, h, key)
                assert sts[h]["evicted"] == sts[0]["evicted"]
            sc, _ = ms[0].last_scores()
            slots = sorted(ranked)
            lids = [ranked[s] for s in slots]
            logit = np.array([[[q[h, j] @ keys[h][x] for x in lids] for j in range(G)] for h in range(n)])
            if agg == 0:
                want = logit.max(axis=(0, 1))
            else:
                z = logit / math.sqrt(d)
                z = np.exp(z - z.max(axis=2, keepdims=True))
                want = (z / z.sum(axis=2, keepdims=True)).sum(axis=(0, 1))
            got = sc[slots]
            assert np.all(np.abs(got - want) <= 1e-12 * (1 + np.abs(want))), (agg, rank_pinned, t, got, want)
            assert np.all(np.isnan(np.delete(sc, slots)))


def check_group_vs_history(lib, seed=11, cases=30):
    """Given the scores a grouped step computed, its refresh and eviction
    follow the single-unit LRU rule: a history-replay LRU fed those scores
    agrees with the shared page table at every step (n = 1, 2 and 4 KV
    heads, random keys, several page sizes and r)."""
    rng = np.random.default_rng(seed)
    for _ in range(cases):
        n = int(rng.choice([1, 2, 4]))
        G = int(rng.integers(1, 4))
        ps = int(rng.integers(1, 4))
        S = int(rng.integers(3, 8))
        P = int(rng.integers(0, (S - 1) * ps + 1))
        r = float(rng.choice([0.5, 0.25, 0.75, 1.0, 0.0]))
        rank_pinned = bool(rng.integers(0, 2))
        agg = int(rng.integers(0, 2))
        d = 4
        ms = [oracle.Kvm(G, d, ps, S, r=r, lib=lib, aggregation=agg, rank_pinned=rank_pinned) for _ in range(n)]
        for m in ms:
            assert m.prefill(rng.standard_normal((P, d)), rng.standard_normal((P, d))) == 0
        hist = HistoryLRU(ps, S, r, P, rank_pinned=rank_pinned)
        for t in range(int(rng.integers(5, 40))):
            ranked = _ranked_slot_lids(ms[0].state(), ps, rank_pinned)
            oracle.decode_group(ms, rng.standard_normal((n, G, d)), rng.standard_normal((n, d)),
                                rng.standard_normal((n, d)), want_out=False)
            sc, _ = ms[0].last_scores()
            score_of = {lid: sc[s] for s, lid in ranked.items()}
            ev = hist.decode(lambda lid: score_of[lid])
            for m in ms:
                st = m.state()
                assert (ev if ev is not None else -1) == st["evicted"], (t, ev, st["evicted"])
                assert sorted(int(x) for x in st["page_table"] if x >= 0) == hist.resident_lids(), t


def check_prompt_selection(lib, seed=12):
    """Quest on the prompt pages, RaaS on the decode pages (the combination
    recommended for long prompts). With one token per page a prompt page's
    bound is its token's logit, so a step attends to exactly the k prompt
    tokens of largest max_j q_j.k (ties, from duplicated keys, to the earlier
    token), every resident decode token and the new one, and its output is
    textbook attention over that set. Prompt pages stay put; decode pages use
    only the slots after the prompt region and follow the LRU rule (history
    replay fed the step's scores)."""
    rng = np.random.default_rng(seed)
    G, d, P, npr, ndec, k = 3, 8, 20, 24, 8, 5
    for r in (0.5, 0.25):
        m = oracle.Kvm(G, d, 1, npr + ndec, r=r, lib=lib, prompt_slots=npr, prompt_topk=k)
        K = rng.standard_normal((P, d))
        K[7] = K[3]  # equal bounds: the tie goes to the earlier token
        K[11] = K[3]
        V = rng.standard_normal((P, d))
        assert m.prefill(K, V) == 0
        keys, vals = list(K), list(V)
        hist = HistoryLRU(1, ndec, r, 0)
        for t in range(60):
            st0 = m.state()
            dec = sorted(int(x) for x in st0["page_table"][npr:] if x >= 0)
            q = rng.standard_normal((G, d))
            if t % 3 == 0:
                q[0] = K[3] * 2.0  # draws the tied tokens into the top k
            kn, vn = rng.standard_normal(d), rng.standard_normal(d)
            out = m.decode(q, kn, vn)
            keys.append(kn)
            vals.append(vn)
            logit = np.array([(q @ K[i]).max() for i in range(P)])
            order = sorted(range(P), key=lambda i: (-logit[i], i))
            chosen = sorted(order[:k])
            att = m.last_attended()
            assert sorted(np.nonzero(att[:npr])[0].tolist()) == chosen, (t, chosen)
            pos = chosen + dec + [P + t]
            ref = _softmax_attention(q, np.array([keys[i] for i in pos]), np.array([vals[i] for i in pos]))
            assert np.max(np.abs(out - ref)) < 1e-12, t
            st = m.state()
            assert st["page_table"][:P].tolist() == list(range(P)) and np.all(st["page_table"][P:npr] == -1)
            sc, _ = m.last_scores()
            ranked = _ranked_slot_lids(st0, 1, False, base=npr)
            assert all(s >= npr for s in ranked)
            score_of = {lid - P: sc[s] for s, lid in ranked.items()}
            ev = hist.decode(lambda lid: score_of[lid])
            assert (P + ev if ev is not None else -1) == st["evicted"], t
            assert sorted(int(x) - P for x in st["page_table"][npr:] if x >= 0) == hist.resident_lids(), t
    # pages of 4: page 0 holds +10u and -10u (u along q), page 1 four copies
    # of 0.5u. Any upper bound puts page 0 at >= 10|q|, above page 1's exact
    # bound 0.5|q| (equal keys), so with k = 1 the step attends to page 0.
    u = rng.standard_normal(8)
    u /= np.linalg.norm(u)
    K = np.array([10 * u, -10 * u, -10 * u, 10 * u] + [0.5 * u] * 4)
    m = oracle.Kvm(1, 8, 4, 4, lib=lib, prompt_slots=2, prompt_topk=1)
    assert m.prefill(K, rng.standard_normal((8, 8))) == 0
    m.decode(u[None, :] * 3.0, rng.standard_normal(8), rng.standard_normal(8))
    assert m.last_attended()[:2].tolist() == [True, False]
    # k at least the prompt's pages: the default policy with the same slots
    a = oracle.Kvm(2, 8, 4, 9, lib=lib, prompt_slots=4, prompt_topk=4)
    b = oracle.Kvm(2, 8, 4, 9, lib=lib)
    K, V = rng.standard_normal((14, 8)), rng.standard_normal((14, 8))
    assert a.prefill(K, V) == 0 and b.prefill(K, V) == 0
    for t in range(50):
        q, kn, vn = rng.standard_normal((2, 8)), rng.standard_normal(8), rng.standard_normal(8)
        assert np.array_equal(a.decode(q, kn, vn), b.decode(q, kn, vn)), t
        sa, sb = a.state(), b.state()
        assert np.array_equal(sa["page_table"], sb["page_table"]) and np.array_equal(sa["ts"], sb["ts"]), t


ALL_CHECKS = [
    check_prompt_selection,
    check_group_single_token_pages,
    check_group_vs_history,
    check_rank_pinned_vs_history,
    check_softmax_sum_invariants,
    check_softmax_sum_golden,
    check_dense_equivalence,
    check_single_token_and_bound,
    check_threshold_counts,
    check_fifo_special_cases,
    check_bruteforce_eviction_order,
    check_random_policy_vs_history,
    check_prefill_rule,
    check_budget_and_attention_set,
]
