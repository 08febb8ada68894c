"""raas_decode_step_static (the step's scratch in the library's fixed device
array, for callers that cannot allocate) against raas_decode_step, through
the C ABI: two pools of one configuration take the same inputs, one through
each entry point; retention must match bit for bit at every step and outputs
within the parity bounds. Runs go from a larger step to smaller ones, so
later calls find the array holding an earlier call's contents. A step whose
scratch would not fit is refused before anything runs."""
from __future__ import annotations

import numpy as np
import pytest

import synth
from harness import ParityReport, compare_outputs, new_pool, record, say, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2502_11147_amd as raas

    raas.load_library()


def _w(**kw):
    base = dict(name="static", batch=4, n_layers=1, n_q_heads=8, n_kv_heads=2, head_dim=128, dtype="bf16",
                page_size=16, budget=256, prefill_len=100, decode_steps=200, ms_period=16,
                ms_phase_random=True, ms_wmin=8, ms_wmax=64)
    base.update(kw)
    return synth.Workload(**base)


# larger first, then smaller: (workload, splits, pool options)
RUNS = [
    (_w(batch=6), 3, {}),                                                  # split path: partials + scores
    (_w(batch=4, budget=128, prefill_len=300), 2, dict(prompt_tokens=320, prompt_topk=3)),  # + selection lists
    (_w(batch=3, dtype="f32"), None, {}),                                  # fp32 step + epilogue kernels
    (_w(batch=3, dtype="f32", head_dim=64), None, {}),                     # fp32 fused: no scratch
    (_w(batch=2, n_q_heads=16, n_kv_heads=4), None, dict(scope=1)),        # one page table per sequence
    (_w(batch=2, budget=128, prefill_len=40), 2, dict(aggregation=1)),     # per-head bounds as scratch
    (_w(batch=2), None, {}),                                               # fused: no scratch at all
]


def _step_both(a, b, w, qd, kd, vd, S, dt):
    import torch

    B, Hq, Hkv, d = w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim
    outs, states = [], []
    for pool, static in ((a, False), (b, True)):
        out = torch.full((B, Hq, d), 3.0, dtype=dt, device="cuda")
        pt = torch.full((B, Hkv, S), -9, dtype=torch.int32, device="cuda")
        ts = torch.full((B, Hkv, S), -9, dtype=torch.int32, device="cuda")
        ev = torch.full((B, Hkv), -9, dtype=torch.int32, device="cuda")
        if static:
            pool.decode_step_static(0, qd, kd, vd, out, pt, ts, ev)
        else:
            pool.decode_step(0, qd, kd, vd, out, pt, ts, ev)
        outs.append(out)
        states.append((pt, ts, ev))
    torch.cuda.synchronize()
    return outs, states


def test_static_scratch_matches_decode_step():
    import torch

    for w, splits, opts in RUNS:
        say("case static scratch batch %d dtype %s splits %s %s" % (w.batch, w.dtype, splits, opts))
        a, b = new_pool(w, splits, **opts), new_pool(w, splits, **opts)
        K, V = synth.prefill(w, 3, 0)
        for pool in (a, b):
            pool.prefill(0, to_device(K, w.dtype), to_device(V, w.dtype))
        S = a.slots
        U, G, d = w.batch * w.n_kv_heads, w.group, w.head_dim
        dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        rep = ParityReport(units_checked=U)
        q, k, v = synth.steps(w, 3, 0, 0, w.decode_steps)
        qd, kd, vd = to_device(q, w.dtype), to_device(k, w.dtype), to_device(v, w.dtype)
        for t in range(w.decode_steps):
            outs, states = _step_both(a, b, w, qd[t], kd[t], vd[t], S, dt)
            for x, y in zip(*states):
                assert torch.equal(x, y), (w.batch, opts, t)
            rep.evictions += int((states[0][2] >= 0).sum())
            compare_outputs(outs[1].float().cpu().numpy().reshape(U, G, d),
                            outs[0].float().cpu().numpy().reshape(U, G, d), w.dtype, "step %d" % t, rep)
            rep.steps = t + 1
        sa, sb = a.export_state(0), b.export_state(0)
        for key in sa:
            assert np.array_equal(sa[key], sb[key]), key
        a.close()
        b.close()
        record(rep, "static scratch batch %d %s splits %s %s" % (w.batch, w.dtype, splits, opts))
        assert rep.evictions > 0


def test_static_scratch_refuses_oversized_step():
    import torch

    import paper_2502_11147_amd as raas

    w = synth.get_workload("llama8b-b32-L2048")
    pool = new_pool(w, 64)  # 64 splits of 256 units over a nearly full pool: 34 MB of partials
    K = torch.zeros((w.batch, w.n_kv_heads, 2000, w.head_dim), dtype=torch.bfloat16, device="cuda")
    pool.prefill(0, K, K)
    q = torch.zeros((w.batch, w.n_q_heads, w.head_dim), dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros((w.batch, w.n_kv_heads, w.head_dim), dtype=torch.bfloat16, device="cuda")
    out = torch.empty_like(q)
    with pytest.raises(raas.RaasError) as e:
        pool.decode_step_static(0, q, kv, kv, out)
    assert e.value.code == raas.E_INVALID and "scratch" in str(e.value)
    st = pool.export_state(0)
    assert np.all(st["clock"] == 2000)  # nothing ran
    pool.decode_step(0, q, kv, kv, out)  # the pool's own scratch still serves it
    assert np.all(pool.export_state(0)["clock"] == 2001)
    pool.close()
