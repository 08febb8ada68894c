"""The GPU parity tests' output bound can see a missing block at full size
(CPU only; no kernel is involved).

At the full-size shapes the attention spreads over thousands of tokens, so
dropping one 32-token block from the attended set moves an output element by
less than the contract's absolute bound (2e-2 for bf16). The harness also
bounds the relative L2 error of every head's output vector (harness.TOL_REL).
Here the oracle runs one unit of each full-size workload to steady state;
then textbook attention over its resident tokens (checked equal to the
oracle's output) is recomputed with one block, or one page, left out, and
the relative change must exceed that bound: for nearly every block and
page at the Llama batch-32 and Qwen shapes; at the batch-128 page-32 shapes,
whose heavy-tailed keys concentrate the softmax on few tokens, for nearly
every block holding at least 2% of some head's attention (a block the
softmax ignores moves nothing that any bound above the bf16 rounding of the
output could see).
"""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle
import synth
from harness import TOL, TOL_REL


def _attention(q, K, V):
    """Textbook scaled dot-product attention (Vaswani et al. 2017), fp64."""
    logits = q @ K.T / math.sqrt(q.shape[-1])
    logits -= logits.max(axis=1, keepdims=True)
    w = np.exp(logits)
    w /= w.sum(axis=1, keepdims=True)
    return w @ V


def _rel(a, b):
    """largest relative L2 change over the heads"""
    return float(np.max(np.linalg.norm(a - b, axis=1) / np.linalg.norm(b, axis=1)))


CASES = [("llama8b-b32-L2048", True), ("qwen7b-28L-b64-L4096", True), ("llama8b-b128-ps32-L512", False),
         ("llama8b-b128-ps32-L2048", False), ("llama8b-b128-ps32-L8192", False)]


@pytest.mark.parametrize("unit", [5, 77])
@pytest.mark.parametrize("name,every", CASES, ids=[c[0] for c in CASES])
def test_relative_bound_sees_a_dropped_block(name, every, unit, oracle_lib, synth_lib):
    w = synth.get_workload(name)
    S, ps, d, G = w.slots, w.page_size, w.head_dim, w.group
    K, V = synth.prefill_units(w, 0, 0, w.prefill_len, [unit])
    m = oracle.Kvm(G, d, ps, S, r=w.r)
    assert m.prefill(K[0].astype(np.float64), V[0].astype(np.float64)) == 0
    fill = max(0, w.budget - w.prefill_len) + 2 * ps
    q, k, v = synth.steps_units(w, 0, 0, 0, fill + 8, [unit])
    for i in range(fill):
        m.decode(q[i, 0], k[i, 0], v[i, 0], want_out=False)
    checked = 0
    for i in range(fill, fill + 8):
        out = m.decode(q[i, 0], k[i, 0], v[i, 0])
        st = m.state()
        if st["evicted"] >= 0:
            continue  # the step attended a page that is gone now
        Kp, Vp, _, _ = m.pages()
        rows = [(s, t) for s in range(S) if st["state"][s] != oracle.FREE for t in range(st["fill"][s])]
        Kr = np.array([Kp[s, t] for s, t in rows])
        Vr = np.array([Vp[s, t] for s, t in rows])
        qq = q[i, 0].astype(np.float64)
        full = _attention(qq, Kr, Vr)
        assert np.max(np.abs(full - out)) < 1e-10  # the resident set is what the step attended
        row = np.array([s * ps + t for s, t in rows])
        logits = qq @ Kr.T / math.sqrt(d)
        wts = np.exp(logits - logits.max(axis=1, keepdims=True))
        wts /= wts.sum(axis=1, keepdims=True)
        for size in (32, ps):
            groups = np.unique(row // size)
            moved, even = [], []
            for g in groups:
                keep = row // size != g
                moved.append(_rel(_attention(qq, Kr[keep], Vr[keep]), full))
                even.append(np.max(wts[:, ~keep].sum(axis=1)) >= 0.02)
            moved, even = np.array(moved), np.array(even)
            seen_all = float(np.mean(moved > TOL_REL["bf16"]))
            seen_even = float(np.mean(moved[even] > TOL_REL["bf16"])) if even.any() else 1.0
            if every:
                assert seen_all >= 0.99, (name, size, seen_all)
            if even.any():
                assert seen_even >= 0.95, (name, size, seen_even, int(even.sum()))
            if name == "llama8b-b128-ps32-L8192" and size == 32:
                # the absolute bound alone misses the typical dropped block
                mid = groups[np.argsort(moved)[len(moved) // 2]]
                keep = row // 32 != mid
                assert np.max(np.abs(_attention(qq, Kr[keep], Vr[keep]) - full)) < TOL["bf16"]
        checked += 1
        if checked == 2:
            break
    assert checked == 2
