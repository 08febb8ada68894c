"""The CPU oracle against what the paper and the mathematics fix (no GPU).

The checks live in ``pins.py``. They run here against the committed oracle,
and against copies of it with one planted mistake each, every one of which
must be caught by at least one check.
"""
from __future__ import annotations

import json
import os

import numpy as np
import pytest

import oracle
import pins
import synth
from oracle.history import HistoryLRU

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("check", pins.ALL_CHECKS, ids=lambda c: c.__name__)
def test_oracle_pin(check, oracle_lib):
    check(oracle_lib)


# (name, [(original text, replacement)]) -- each a plausible slip in the oracle
MUTANTS = [
    ("score_uses_min", [("acc += (a > b) ? a : b;", "acc += (a < b) ? a : b;")]),
    ("no_softmax_scale", [("const double scale = 1.0 / sqrt((double)d);\n    int n_old = 0;",
                           "const double scale = 1.0;\n    int n_old = 0;")]),
    ("refresh_ties_at_threshold", [("m->score[s] > theta) m->ts[s] = c;", "m->score[s] >= theta) m->ts[s] = c;")]),
    ("order_statistic_off_by_one", [("theta = sorted[n - k - 1];", "theta = sorted[n - k];")]),
    ("tie_break_newest", [("m->lid[s] < m->lid[v]", "m->lid[s] > m->lid[v]")]),
    ("new_page_unstamped", [("m->ts[s] = c; /* R5 */", "m->ts[s] = -1; /* R5 */")]),
    ("prefill_fills_cache", [("const int cap = m->prompt_topk >= 0 ? m->decode_base : m->S - 1;",
                              "const int cap = m->prompt_topk >= 0 ? m->decode_base : m->S;")]),
    ("pinned_not_attended", [("m->attend[s] = m->state[s] != FREE;", "m->attend[s] = m->state[s] == EVICTABLE;")]),
    ("kmax_not_widened", [("if (k[c] > m->kmax[(size_t)s * d + c]) m->kmax[(size_t)s * d + c] = k[c];", "")]),
    ("evicted_tail_kept", [("if (m->tail == v) m->tail = -1;", "")]),
    ("top_r_rounds_up", [("int k = (int)floor(m->r * (double)n);", "int k = (int)ceil(m->r * (double)n);")]),
    ("pinned_pages_scored", [("#define RANKED(st) ((st) == EVICTABLE || (m->rank_pinned && (st) == PINNED))",
                              "#define RANKED(st) ((st) == EVICTABLE || (st) == PINNED)")]),
    ("rank_pinned_ignored", [("#define RANKED(st) ((st) == EVICTABLE || (m->rank_pinned && (st) == PINNED))",
                              "#define RANKED(st) ((st) == EVICTABLE)")]),
    ("softmax_sum_unnormalised", [("m->score[s] += exp(scale * (bound[(size_t)s * H + j] - mx)) / z;",
                                   "m->score[s] += exp(scale * (bound[(size_t)s * H + j] - mx));")]),
    ("softmax_sum_scale_one", [("const double scale = 1.0 / sqrt((double)m->d);",
                                "const double scale = 1.0;")]),
    ("softmax_sum_one_head", [("        for (int j = 0; j < H; ++j) {\n            double mx = -INFINITY, z = 0.0;",
                               "        for (int j = 0; j < 1; ++j) {\n            double mx = -INFINITY, z = 0.0;")]),
    ("group_heads_overlap", [("bound[(size_t)s * H + h0 + j] = acc;", "bound[(size_t)s * H + j] = acc;")]),
    ("group_first_kv_head_refreshed", [("        refresh(ms[h], c);", "        if (h == 0) refresh(ms[h], c);")]),
    ("group_first_kv_head_scored", [("    for (int h = 0; h < n; ++h) head_bounds(ms[h], q + (size_t)h * G * d, bound, H, h * G);",
                                     "    for (int h = 0; h < n; ++h) head_bounds(ms[0], q, bound, H, h * G);")]),
    ("softmax_sign", [("double p = exp(logit[t] - mx);", "double p = exp(mx - logit[t]);")]),
    ("prompt_ties_to_later_slot", [("(b[o] == b[s] && o < s)", "(b[o] == b[s] && o > s)")]),
    ("prompt_bound_uses_min", [("acc += x > y ? x : y;", "acc += x < y ? x : y;")]),
    ("prompt_topk_one_more", [("m->attend[s] = above < m->prompt_topk;", "m->attend[s] = above <= m->prompt_topk;")]),
    ("decode_page_in_prompt_region", [("for (int i = m->decode_base; i < S; ++i)", "for (int i = 0; i < S; ++i)")]),
    ("gqa_last_head_only", [("if (bound[(size_t)s * H + j] > best) best = bound[(size_t)s * H + j];",
                             "best = bound[(size_t)s * H + j];")]),
]


@pytest.mark.parametrize("name,edits", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_is_caught(name, edits, tmp_path):
    src = open(oracle.SRC).read()
    for old, new in edits:
        assert src.count(old) == 1, (name, old)
        src = src.replace(old, new)
    path = tmp_path / ("mutant_%s.c" % name)
    path.write_text(src)
    lib = oracle.build(str(path), str(tmp_path / ("libmutant_%s.so" % name)), force=True)
    caught = []
    for check in pins.ALL_CHECKS:
        try:
            check(lib)
        except (AssertionError, oracle.OracleError, ValueError, KeyError, IndexError):
            caught.append(check.__name__)
    assert caught, "planted mistake %s went unnoticed" % name


def _golden():
    with open(os.path.join(GOLDEN, "retention_worked_example.json")) as f:
        return json.load(f)


def test_golden_worked_example_oracle(oracle_lib):
    g = _golden()
    ps, S, P = g["page_size"], g["slots"], g["prefill_len"]
    m = oracle.Kvm(1, 2, ps, S, r=g["r"], lib=oracle_lib)
    assert m.prefill(np.zeros((P, 2)), np.zeros((P, 2))) == 0
    for step in g["steps"]:
        st = m.state()
        assert st["clock"] == step["clock"]
        slot_lid = {s: int(st["page_table"][s]) for s in range(S) if st["state"][s] == oracle.EVICTABLE}
        new = pins._new_slot(st, ps)
        if new is not None:
            slot_lid[new] = st["next_lid"]
        assert sorted(slot_lid.values()) == sorted(int(x) for x in step["scores"])
        sc = np.zeros(S)
        for s, lid in slot_lid.items():
            sc[s] = step["scores"][str(lid)]
        m.decode_with_scores(sc)
        st = m.state()
        assert st["evicted"] == step["evicted"], step
        assert st["page_table"].tolist() == step["page_table"], step
        assert st["ts"].tolist() == step["ts"], step


def test_golden_worked_example_history():
    g = _golden()
    h = HistoryLRU(g["page_size"], g["slots"], g["r"], g["prefill_len"])
    for step in g["steps"]:
        ev = h.decode(lambda lid: step["scores"][str(lid)])
        assert (ev if ev is not None else -1) == step["evicted"]
        assert h.resident_lids() == sorted(x for x in step["page_table"] if x >= 0)


def test_generator_philox_known_answers(synth_lib):
    """Philox4x32-10 against the known-answer vectors published with the
    Random123 library (Salmon et al., SC 2011)."""
    kat = [
        ([0, 0, 0, 0], [0, 0], [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]),
        ([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2, [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]),
        ([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0],
         [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]),
    ]
    for ctr, key, want in kat:
        assert synth_lib.philox4x32_10(ctr, key) == want


def test_generator_statistics_and_milestones(synth_lib):
    """Shape of the synthetic inputs: N(0,1) values exactly representable in
    the dtype, and queries inside a milestone window at cos 0.8 to the
    milestone key (one active milestone)."""
    w = synth.get_workload("tiny-f32")
    q, k, v = synth.steps(w, 0, 0, 0, 200)
    assert abs(float(k.std()) - 1.0) < 0.05 and abs(float(k.mean())) < 0.05
    wb = synth.get_workload("llama8b-b1-L1024")
    qb, kb, vb = synth.steps(wb, 0, 0, 0, 4)
    bits = qb.view(np.uint32)
    assert np.all(bits & 0xFFFF == 0)  # bf16-representable
    # tiny-f32: milestones at decode steps 31, 63, ...; window 64
    assert synth.active_milestones(w, 0, 0, 0, 0, 31) == []
    assert synth.active_milestones(w, 0, 0, 0, 0, 32) == [31]
    assert synth.active_milestones(w, 0, 0, 0, 0, 95) == [31, 63]
    assert synth.active_milestones(w, 0, 0, 0, 0, 96) == [63, 95]
    # one active milestone at step 32: every query head at cos 0.8 to k_31
    q, k, _ = synth.steps(w, 0, 0, 31, 2)
    km = k[0, 0, 0].astype(np.float64)
    for j in range(w.group):
        qj = q[1, 0, j].astype(np.float64)
        cos = qj @ km / np.linalg.norm(qj) / np.linalg.norm(km)
        assert abs(cos - 0.8) < 1e-5
    assert synth.active_milestones(w, 0, 0, 0, 0, 0) == []
    # stress workload: heavy-tailed keys (excess kurtosis well above 0)
    ws = synth.get_workload("llama8b-b128-ps32-L512").replace(batch=2)
    _, ks, vs = synth.steps(ws, 0, 0, 0, 64)
    kk = ks.astype(np.float64).ravel()
    vv = vs.astype(np.float64).ravel()
    kurt_k = np.mean((kk - kk.mean()) ** 4) / np.var(kk) ** 2 - 3
    kurt_v = np.mean((vv - vv.mean()) ** 4) / np.var(vv) ** 2 - 3
    assert kurt_k > 0.5 and abs(kurt_v) < 0.3


def test_generator_random_access(synth_lib):
    """Any window of steps regenerates to the same values."""
    w = synth.get_workload("llama8b-b1-L1024")
    a = synth.steps(w, 7, 0, 100, 10)
    b = synth.steps(w, 7, 0, 105, 3)
    for x, y in zip(a, b):
        assert np.array_equal(x[5:8], y)
    c = synth.steps(w, 8, 0, 105, 3)
    assert not np.array_equal(a[0][5:8], c[0])


def test_oracle_batch_matches_single(oracle_lib):
    """The OpenMP batch entry gives the per-unit results."""
    rng = np.random.default_rng(0)
    G, d, ps, S, P, n = 2, 8, 4, 4, 6, 5
    a = [oracle.Kvm(G, d, ps, S) for _ in range(n)]
    b = [oracle.Kvm(G, d, ps, S) for _ in range(n)]
    for u in range(n):
        K = rng.standard_normal((P, d)).astype(np.float32)
        V = rng.standard_normal((P, d)).astype(np.float32)
        a[u].prefill(K, V)
        b[u].prefill(K, V)
    for t in range(30):
        q = rng.standard_normal((n, G, d)).astype(np.float32)
        k = rng.standard_normal((n, d)).astype(np.float32)
        v = rng.standard_normal((n, d)).astype(np.float32)
        out = oracle.decode_batch(a, q, k, v)
        for u in range(n):
            o1 = b[u].decode(q[u], k[u], v[u])
            assert np.array_equal(o1, out[u])
            assert a[u].state()["page_table"].tolist() == b[u].state()["page_table"].tolist()


def _drive_scores(m, scores_by_lid, ps):
    """One retention-only step with scores given per logical page id."""
    st = m.state()
    slot_lid = {s: int(st["page_table"][s]) for s in range(m.S) if st["state"][s] == oracle.EVICTABLE}
    new = pins._new_slot(st, ps)
    if new is not None:
        slot_lid[new] = st["next_lid"]
    sc = np.zeros(m.S)
    for s, lid in slot_lid.items():
        sc[s] = scores_by_lid(lid)
    m.decode_with_scores(sc)


def test_lockstep_adopt_hook(oracle_lib):
    """The parity harness's re-sync after a near tie (orc_adopt_retention):
    an oracle that decided one step differently (a refresh, and through it
    the eviction) takes the other decision and from then on evolves exactly
    as the other side; anything beyond the step's own decisions is refused
    and leaves the state unchanged."""
    ps, S, P = 2, 5, 2
    rng = np.random.default_rng(3)
    base = {lid: float(rng.standard_normal()) for lid in range(200)}
    for flip_at in range(8, 40):
        a = oracle.Kvm(1, 2, ps, S, lib=oracle_lib)
        b = oracle.Kvm(1, 2, ps, S, lib=oracle_lib)
        for m in (a, b):
            assert m.prefill(np.zeros((P, 2)), np.zeros((P, 2))) == 0
        for t in range(60):
            _drive_scores(a, lambda lid: base[(lid * 7 + t) % 200], ps)
            if t == flip_at:  # b ranks the pages in the opposite order at this step
                _drive_scores(b, lambda lid: -base[(lid * 7 + t) % 200], ps)
                sa, sb = a.state(), b.state()
                if np.array_equal(sa["ts"], sb["ts"]) and sa["evicted"] == sb["evicted"]:
                    break  # this flip changed nothing
                a.adopt_retention(sb["page_table"], sb["ts"], sb["evicted"])
            else:
                _drive_scores(b, lambda lid: base[(lid * 7 + t) % 200], ps)
            sa, sb = a.state(), b.state()
            for key in ("page_table", "ts", "fill", "tail", "next_lid", "clock", "evicted"):
                assert np.array_equal(sa[key], sb[key]), (flip_at, t, key, sa[key], sb[key])
    # refused: a pinned page changed, an unknown page, two evictions
    m = oracle.Kvm(1, 2, ps, S, lib=oracle_lib)
    assert m.prefill(np.zeros((P, 2)), np.zeros((P, 2))) == 0
    for t in range(12):
        _drive_scores(m, lambda lid: float(lid), ps)
    st = m.state()
    bad_pin = st["page_table"].copy()
    bad_pin[0] = 99
    bad_new = st["page_table"].copy()
    bad_new[int(np.argmax(st["page_table"]))] = 77
    bad_ts = st["ts"].copy()
    bad_ts[int(np.argmax(st["ts"]))] = st["clock"] + 5
    for pt, ts in ((bad_pin, st["ts"]), (bad_new, st["ts"]), (st["page_table"], bad_ts)):
        with pytest.raises(oracle.OracleError):
            m.adopt_retention(pt, ts, st["evicted"])
        st2 = m.state()
        for key in ("page_table", "ts", "fill", "tail", "evicted"):
            assert np.array_equal(st[key], st2[key])
