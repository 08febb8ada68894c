"""Pins of the oracle-only baseline policies (oracle/baselines.py).

Each policy is checked against a closed form or against an independently
written implementation: with a budget that holds every token they are dense
attention; StreamingLLM keeps the sinks and the most recent tokens; H2O with
a recent window covering the budget is pure recency; Quest with one token per
page picks the tokens of largest max_j q_j.k; token-level RaaS with one query
head makes the decisions of page-level RaaS (the C oracle) with one token per
page, and at r = 0 keeps the most recent decode tokens.
"""
from __future__ import annotations

import numpy as np
import pytest

from oracle import baselines as bl


def _stream(rng, P, T, G, d):
    K = rng.standard_normal((P, d))
    V = rng.standard_normal((P, d))
    steps = [(rng.standard_normal((G, d)) * 1.5, rng.standard_normal(d), rng.standard_normal(d)) for _ in range(T)]
    return K, V, steps


def test_every_policy_is_dense_when_everything_fits(oracle_lib):
    rng = np.random.default_rng(1)
    P, T, G, d = 7, 30, 3, 16
    K, V, steps = _stream(rng, P, T, G, d)
    L = 64  # > P + T
    dense = bl.Dense(K, V)
    pols = [bl.Sink(K, V, L), bl.H2O(K, V, L), bl.Quest(K, V, L, 4), bl.TokenRaaS(K, V, L),
            bl.PageRaaS(K, V, L, 4, lib=oracle_lib)]
    for t, (q, k, v) in enumerate(steps):
        ref, att_ref = dense.step(q, k, v)
        for pol in pols:
            out, att = pol.step(q, k, v)
            assert sorted(att) == att_ref, (pol.name, t)
            assert np.max(np.abs(out - ref)) < 1e-12, (pol.name, t)


def test_sink_keeps_sinks_and_recent_tokens():
    rng = np.random.default_rng(2)
    P, T, G, d, L = 10, 40, 2, 8, 16
    K, V, steps = _stream(rng, P, T, G, d)
    pol = bl.Sink(K, V, L, n_sink=4)
    for t, (q, k, v) in enumerate(steps):
        out, att = pol.step(q, k, v)
        n = P + t + 1  # tokens so far, the new one included
        want = list(range(min(4, n))) + list(range(max(4, n - (L - 4)), n))
        assert att == want, (t, att, want)
        Kr = np.array([K[i] if i < P else steps[i - P][1] for i in want])
        Vr = np.array([V[i] if i < P else steps[i - P][2] for i in want])
        ref, _ = bl.attention(q, Kr, Vr)
        assert np.max(np.abs(out - ref)) < 1e-12


def test_h2o_with_a_full_recent_window_is_recency():
    rng = np.random.default_rng(3)
    P, T, G, d, L = 5, 40, 2, 8, 12
    K, V, steps = _stream(rng, P, T, G, d)
    pol = bl.H2O(K, V, L, recent=L)
    for t, (q, k, v) in enumerate(steps):
        _, att = pol.step(q, k, v)
        n = P + t + 1
        assert att == list(range(max(0, n - L), n)), t


def test_h2o_keeps_the_heaviest_hitter():
    """A token that takes nearly all attention at every step stays, however
    old, while recency alone would have dropped it."""
    rng = np.random.default_rng(4)
    d, G, L = 8, 1, 8
    K = rng.standard_normal((3, d)) * 0.1
    K[0] = np.ones(d) * 3.0
    V = rng.standard_normal((3, d))
    pol = bl.H2O(K, V, L, recent=2)
    for t in range(40):
        q = np.ones((G, d))
        _, att = pol.step(q, rng.standard_normal(d) * 0.1, rng.standard_normal(d))
        assert 0 in att, t


def test_quest_with_one_token_pages_picks_the_largest_logits():
    rng = np.random.default_rng(5)
    P, T, G, d, L = 12, 30, 3, 8, 9
    K, V, steps = _stream(rng, P, T, G, d)
    pol = bl.Quest(K, V, L, 1)
    allK = list(K)
    for t, (q, k, v) in enumerate(steps):
        allK.append(k)
        _, att = pol.step(q, k, v)
        n = len(allK)
        if n <= L:
            assert att == list(range(n))
            continue
        logit = np.array([(q @ allK[i]).max() for i in range(n - 1)])
        top = sorted(np.argsort(-logit, kind="stable")[: L - 1].tolist())
        assert att == top + [n - 1], t


def test_token_raas_matches_page_raas_with_one_token_pages(oracle_lib):
    """Independent implementations (numpy here, the C oracle there): with one
    query head the attention weight orders tokens as the logit does, and a
    one-token page's representative bound is its logit, so both keep the
    same tokens at every step."""
    for seed, (P, L, r) in enumerate([(5, 12, 0.5), (0, 9, 0.25), (20, 8, 0.75), (3, 16, 1.0)]):
        rng = np.random.default_rng(10 + seed)
        K, V, steps = _stream(rng, P, 120, 1, 8)
        tok = bl.TokenRaaS(K, V, L, r=r)
        page = bl.PageRaaS(K, V, L, 1, r=r, lib=oracle_lib)
        for t, (q, k, v) in enumerate(steps):
            o1, a1 = tok.step(q, k, v)
            o2, a2 = page.step(q, k, v)
            assert sorted(a1) == sorted(a2), (seed, t, sorted(a1), sorted(a2))
            assert np.max(np.abs(o1 - o2)) < 1e-12


def test_token_raas_at_r0_keeps_the_newest_decode_tokens():
    rng = np.random.default_rng(6)
    P, L = 4, 10
    K, V, steps = _stream(rng, P, 50, 2, 8)
    pol = bl.TokenRaaS(K, V, L, r=0.0)
    for t, (q, k, v) in enumerate(steps):
        _, att = pol.step(q, k, v)
        n = P + t + 1
        room = L - P  # decode tokens attended, the new one included
        assert att == list(range(P)) + list(range(max(P, n - room), n)), t


@pytest.mark.parametrize("policy", ["sink", "h2o", "raas-token"])
def test_budget_holds(policy):
    rng = np.random.default_rng(7)
    P, L = 30, 16
    K, V, steps = _stream(rng, P, 60, 2, 8)
    pol = {"sink": lambda: bl.Sink(K, V, L), "h2o": lambda: bl.H2O(K, V, L),
           "raas-token": lambda: bl.TokenRaaS(K, V, L)}[policy]()
    for q, k, v in steps:
        _, att = pol.step(q, k, v)
        assert len(att) <= L
