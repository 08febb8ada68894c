"""GPU parity: the HIP decode path against the CPU oracle, through the C ABI.

Small cases compare every unit at every step; the full-size workloads run
in the launch configuration the benchmark uses and compare sampled units,
plus properties every unit must satisfy.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

import synth
import oracle
from harness import TOL, ParityReport, compare_outputs, new_pool, record, run_parity, run_ragged, say, to_device

pytestmark = pytest.mark.gpu

_say = say


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2502_11147_amd as raas

    raas.load_library()  # fails loudly when the HIP library is missing


def small(**kw):
    base = dict(name="small", batch=2, n_layers=1, n_q_heads=8, n_kv_heads=2, head_dim=128, dtype="bf16",
                page_size=16, budget=128, prefill_len=40, decode_steps=300, ms_period=16,
                ms_phase_random=True, ms_wmin=8, ms_wmax=64)
    base.update(kw)
    return synth.Workload(**base)


def _report(rep: ParityReport, tag, resync_bound=0):
    """Records the run's counts (printed again in the session summary) and
    checks the re-syncs: with fp64 scores on both sides a near tie that the
    two sides decide differently needs two pages within rounding (about
    1e-13) of each other at the threshold, so none is expected."""
    record(rep, tag)
    assert rep.flagged_divergences <= resync_bound, rep.line(tag)


def test_tiny_f32_full_run():
    """The tiny fp32 workload end to end: every step, every output."""
    w = synth.get_workload("tiny-f32")
    _say("case tiny-f32 seed 0 steps %d" % w.decode_steps)
    rep = run_parity(w, seed=0, steps=w.decode_steps)
    _report(rep, "tiny-f32")
    assert rep.evictions > 0


@pytest.mark.parametrize("seed", [0, 1])
def test_small_bf16_every_step(seed):
    w = small()
    _say("case small-bf16 seed %d" % seed)
    rep = run_parity(w, seed=seed, steps=w.decode_steps)
    _report(rep, "small-bf16")
    assert rep.evictions > 0


@pytest.mark.parametrize("splits", [1, 2, 3, 5, 64])
def test_split_counts_agree(splits):
    """Split-K over pages changes only rounding, never retention."""
    w = small(budget=512, prefill_len=100, decode_steps=520)
    _say("case split-sweep splits %d" % splits)
    rep = run_parity(w, seed=3, steps=w.decode_steps, splits=splits)
    _report(rep, "splits=%d" % splits)


EDGE = [
    dict(prefill_len=0),
    dict(prefill_len=16 * 7),                     # exactly S-1 pages pinned, one decode slot
    dict(prefill_len=1000),                       # overflow: first S-1 pages pinned (PIN_HEAD)
    dict(prefill_len=3),                          # one partial pinned page
    dict(page_size=8, budget=64),
    dict(page_size=32, budget=256),
    dict(page_size=64, budget=448, prefill_len=70),
    dict(page_size=128, budget=512, prefill_len=130),
    dict(budget=80),                              # 5 pages: 80 tokens, not a multiple of 32
    dict(n_q_heads=2, n_kv_heads=2),              # G = 1
    dict(n_q_heads=28, n_kv_heads=4),             # G = 7
    dict(n_q_heads=32, n_kv_heads=2),             # G = 16
    dict(head_dim=64),
    dict(r=0.0), dict(r=1.0), dict(r=0.25), dict(r=0.75),
    # r not exact in binary: floor(r * n) at n a multiple of 10 evictable pages
    # (3 pinned + 10 or 20 decode pages) is 7 and 18, one more than a float r gives
    dict(r=0.7, budget=16 * 13), dict(r=0.9, budget=16 * 23), dict(r=0.7, budget=16 * 13, dtype="f32"),
    dict(r=0.9, page_size=8, budget=8 * 308, prefill_len=2300),   # 288 pinned + 20, the epilogue's radix select
    dict(dtype="f32", head_dim=128),
    dict(dtype="f32", n_q_heads=14, n_kv_heads=2, head_dim=64, page_size=8, budget=96),
    dict(page_size=8, budget=2400, prefill_len=2300),             # 300 slots: the epilogue's radix select
    dict(page_size=8, budget=2400, prefill_len=2300, r=0.25),
    dict(page_size=8, budget=16384, prefill_len=16000, decode_steps=80),  # 2048 slots, the most a pool has
    dict(n_q_heads=32, n_kv_heads=2, head_dim=64, page_size=128, budget=1024, prefill_len=300),  # G 16, d 64, page 128
]


@pytest.mark.parametrize("edge", EDGE, ids=[",".join("%s=%s" % kv for kv in e.items()) for e in EDGE])
def test_edge_cases(edge):
    edge = dict(edge)
    w = small(decode_steps=edge.pop("decode_steps", 200), **edge)
    _say("case edge %s" % edge)
    rep = run_parity(w, seed=5, steps=w.decode_steps)
    _report(rep, "edge")


# fp32 step kernel instances (head slots GM = 4, 8, 16 at d 64 and 128) and
# split shapes: one wavefront walking several 64-token chunks, uneven splits
F32_SHAPES = [
    dict(n_q_heads=32, n_kv_heads=2, head_dim=128),              # G 16, d 128
    dict(n_q_heads=32, n_kv_heads=2, head_dim=64),               # G 16, d 64
    dict(n_q_heads=16, n_kv_heads=2, head_dim=128),              # G 8
    dict(n_q_heads=2, n_kv_heads=2, head_dim=128),               # G 1: three idle head slots
    dict(budget=512, prefill_len=100, decode_steps=520, splits=1),   # eight chunks in one wavefront
    dict(budget=512, prefill_len=100, decode_steps=520, splits=3),   # uneven splits, ragged last chunk
    dict(budget=80, page_size=8, prefill_len=3, splits=2),       # ragged pages and chunks
    # head_dim 64: one workgroup per unit, a wavefront per split, the epilogue in the same kernel
    dict(head_dim=64, budget=256, prefill_len=40, splits=1),     # one wavefront over four chunks
    dict(head_dim=64, budget=256, prefill_len=40, splits=3),     # uneven splits
    dict(head_dim=64, budget=512, prefill_len=100, decode_steps=520, splits=8),  # eight wavefronts
    dict(head_dim=64, page_size=8, budget=80, prefill_len=3),    # ragged pages, the default plan
    dict(head_dim=64, budget=2048, prefill_len=1500, decode_steps=600),  # 32 splits: the split path
]


@pytest.mark.parametrize("shape", F32_SHAPES, ids=[",".join("%s=%s" % kv for kv in e.items()) for e in F32_SHAPES])
def test_f32_kernel_shapes(shape):
    shape = dict(shape)
    splits = shape.pop("splits", 0)
    w = small(dtype="f32", decode_steps=shape.pop("decode_steps", 200), **shape)
    _say("case f32 %s splits %d" % (shape, splits))
    rep = run_parity(w, seed=11, steps=w.decode_steps, splits=splits)
    _report(rep, "f32")
    assert rep.outputs_compared > 0


def test_multi_layer_independent():
    """Layers have their own pages and clocks; stepping one leaves the others."""
    import torch

    w = small(n_layers=3, decode_steps=150)
    pool = new_pool(w)
    _say("case multi-layer layer 2 then 0")
    rep = run_parity(w, seed=9, steps=120, layer=2, pool=pool)
    before = pool.export_state(1)
    assert np.all(before["state"] == 0) and np.all(before["lid"] == -1)
    rep = run_parity(w, seed=9, steps=w.decode_steps, layer=0, pool=pool, report=rep)
    st2 = pool.export_state(2)
    assert np.all(st2["clock"] == w.prefill_len + 120)
    st0 = pool.export_state(0)
    assert np.all(st0["clock"] == w.prefill_len + w.decode_steps)
    pool.close()
    torch.cuda.synchronize()


def test_state_errors_and_budget_policy():
    import torch

    import paper_2502_11147_amd as raas

    w = small()
    pool = new_pool(w)
    d = w.head_dim
    q = torch.zeros((w.batch, w.n_q_heads, d), dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros((w.batch, w.n_kv_heads, d), dtype=torch.bfloat16, device="cuda")
    out = torch.empty_like(q)
    with pytest.raises(raas.RaasError) as e:
        pool.decode_step(0, q, kv, kv, out)
    assert e.value.code == raas.E_STATE
    K = torch.zeros((w.batch, w.n_kv_heads, 16, d), dtype=torch.bfloat16, device="cuda")
    pool.prefill(0, K, K)
    with pytest.raises(raas.RaasError) as e:
        pool.prefill(0, K, K)
    assert e.value.code == raas.E_STATE
    with pytest.raises(raas.RaasError) as e:
        pool.decode_step(1, q, kv, kv, out)
    assert e.value.code == raas.E_INVALID
    pool.decode_step(0, q, kv, kv, out)
    st = pool.export_state(0)
    assert np.all(st["clock"] == 17)
    pool.close()
    strict = new_pool(w, policy=raas.PREFILL_ERROR)
    big = torch.zeros((w.batch, w.n_kv_heads, w.budget, d), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(raas.RaasError) as e:
        strict.prefill(0, big, big)
    assert e.value.code == raas.E_BUDGET
    st = strict.export_state(0)
    assert np.all(st["state"] == 0)  # the refused call changed nothing
    strict.close()


@pytest.mark.parametrize("splits", [None, 3], ids=["fused", "split"])
@pytest.mark.parametrize("det", [False, True], ids=["dynamic", "deterministic"])
def test_deterministic(det, splits):
    """Same inputs twice: bitwise-identical retention state. With the
    deterministic option the outputs are bitwise identical too (each
    wavefront sums a fixed interleave of the blocks). Without it they may
    differ: the wavefronts of a workgroup claim attention blocks
    dynamically, so a wavefront's running softmax maximum, under which its
    probabilities are rounded to bf16 for the PV product, depends on which
    blocks it took. Each run is within the parity bounds of the oracle, so
    the two are within twice those bounds; the test holds them to one."""
    import torch

    from harness import TOL_REL

    # 32 blocks per unit over 8 wavefronts: 16 claimed dynamically
    w = small(budget=1024, prefill_len=500, decode_steps=260)
    outs = []
    for _ in range(2):
        pool = new_pool(w, splits, deterministic=det)
        K, V = synth.prefill(w, 11, 0)
        pool.prefill(0, to_device(K, w.dtype), to_device(V, w.dtype))
        q, k, v = synth.steps(w, 11, 0, 0, w.decode_steps)
        qd, kd, vd = to_device(q, w.dtype), to_device(k, w.dtype), to_device(v, w.dtype)
        o = torch.empty((w.decode_steps, w.batch, w.n_q_heads, w.head_dim), dtype=torch.bfloat16,
                        device="cuda")
        for i in range(w.decode_steps):
            pool.decode_step(0, qd[i], kd[i], vd[i], o[i])
        st = pool.export_state(0)
        outs.append((o.float().cpu().numpy().astype(np.float64), st))
        pool.close()
    a, b = outs[0][0], outs[1][0]
    rel = np.linalg.norm(a - b, axis=-1) / np.linalg.norm(a, axis=-1)
    _say("deterministic=%d splits %s: %d of %d outputs differ; largest relative L2 difference of a head %.3g"
         % (det, splits, int(np.sum(a != b)), a.size, float(rel.max())))
    if det:
        assert np.array_equal(a, b)
    assert np.all(rel <= TOL_REL["bf16"])
    for key in ("lid", "ts", "state", "fill", "clock", "next_lid"):
        assert np.array_equal(outs[0][1][key], outs[1][1][key])


@pytest.mark.parametrize("case", [dict(), dict(splits=3),
                                  dict(prompt_tokens=128, prompt_topk=3, prefill_len=100, budget=512),
                                  dict(aggregation=1)],
                         ids=["fused", "split", "prompt-selection", "softmax-sum"])
def test_deterministic_option_parity(case):
    """The deterministic option (a fixed interleave of the blocks over the
    wavefronts) against the oracle: retention bit-exact, outputs within
    the bounds, on the fused and split plans, the in-step prompt selection
    and the softmax aggregation."""
    case = dict(case)
    splits = case.pop("splits", None)
    run_kw = {k: case.pop(k) for k in ("prompt_tokens", "prompt_topk", "aggregation") if k in case}
    w = small(budget=case.pop("budget", 1024), prefill_len=case.pop("prefill_len", 500), decode_steps=700)
    _say("case deterministic option %s splits %s" % (run_kw, splits))
    pool = new_pool(w, splits, deterministic=True, **run_kw)
    rep = run_parity(w, seed=17, steps=w.decode_steps, pool=pool, **run_kw)
    pool.close()
    _report(rep, "deterministic option")
    assert rep.evictions > 0


@pytest.mark.parametrize("splits", [None, 1], ids=["auto-split", "fused"])
@pytest.mark.parametrize("det", [False, True], ids=["dynamic", "deterministic"])
def test_long_pool_small_batch(det, splits):
    """Pools of 64 blocks and more at 4 units, whose workgroups of 8
    wavefronts issue the first score pass with the first blocks: the plan's
    own split over the CUs, and one fused workgroup per unit (the plan of
    the batch-32 workload, forced here), with every unit's outputs compared
    at every step, through the budget and 600 steps past it, with the
    dynamic claims and the deterministic option."""
    w = small(batch=2, n_kv_heads=2, n_q_heads=8, budget=2048, prefill_len=1000, decode_steps=1700)
    _say("case long pool small batch deterministic %s splits %s" % (det, splits))
    pool = new_pool(w, splits, deterministic=det)
    rep = run_parity(w, seed=19, steps=w.decode_steps, pool=pool)
    pool.close()
    _report(rep, "long pool small batch")
    assert rep.evictions > 0


@pytest.mark.parametrize("case", [dict(), dict(splits=3), dict(dtype="f32"), dict(prompt_tokens=128, prompt_topk=3)],
                         ids=["fused", "split", "f32", "prompt-selection"])
def test_checkpoint_resume(case):
    """A layer saved mid-run and loaded into a fresh pool of the same
    configuration continues exactly as the uninterrupted pool: retention
    bit for bit and (deterministic option) outputs bit for bit, through the
    budget filling and evictions; loading into a pool of another
    configuration is refused."""
    import torch

    import paper_2502_11147_amd as raas

    case = dict(case)
    splits = case.pop("splits", None)
    opts = {k: case.pop(k) for k in ("prompt_tokens", "prompt_topk") if k in case}
    w = small(budget=256, prefill_len=100, decode_steps=400, **case)
    _say("case checkpoint %s splits %s %s" % (case, splits, opts))
    a = new_pool(w, splits, deterministic=True, **opts)
    K, V = synth.prefill(w, 5, 0)
    a.prefill(0, to_device(K, w.dtype), to_device(V, w.dtype))
    q, k, v = synth.steps(w, 5, 0, 0, w.decode_steps)
    qd, kd, vd = to_device(q, w.dtype), to_device(k, w.dtype), to_device(v, w.dtype)
    B, Hq, Hkv, d, S = w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, a.slots
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32

    def step(pool, t):
        out = torch.empty((B, Hq, d), dtype=dt, device="cuda")
        pt = torch.empty((B, Hkv, S), dtype=torch.int32, device="cuda")
        ts = torch.empty((B, Hkv, S), dtype=torch.int32, device="cuda")
        ev = torch.empty((B, Hkv), dtype=torch.int32, device="cuda")
        pool.decode_step(0, qd[t], kd[t], vd[t], out, pt, ts, ev)
        return out, pt, ts, ev

    cut = 137
    for t in range(cut):
        step(a, t)
    buf = a.save_layer(0)
    b = new_pool(w, splits, deterministic=True, **opts)
    keep = b.load_layer(0, buf)
    evictions = 0
    for t in range(cut, w.decode_steps):
        ra, rb = step(a, t), step(b, t)
        for x, y in zip(ra, rb):
            assert torch.equal(x, y), t
        evictions += int((ra[3] >= 0).sum())
    torch.cuda.synchronize()
    del keep
    sa, sb = a.export_state(0), b.export_state(0)
    for key in sa:
        assert np.array_equal(sa[key], sb[key]), key
    assert evictions > 0
    other = new_pool(w.replace(r=0.25), splits, deterministic=True, **opts)  # same sizes, another rule

    def corrupt(off, value):  # header: magic, abi, bytes, 16 config fields, then the host bookkeeping
        x = buf.copy()
        x[off:off + 8] = np.frombuffer(np.int64(value).tobytes(), np.uint8)
        return x

    keep_max, steps, desc = 8 * 20, 8 * 21, 8 * 22
    for pool, data, why in ((other, buf, "configuration"), (b, np.zeros_like(buf), "checkpoint"),
                            (b, buf[:-256], "bytes"), (b, corrupt(keep_max, -1), "corrupt"),
                            (b, corrupt(keep_max, b.slots + 1), "corrupt"), (b, corrupt(steps, -5), "corrupt"),
                            (b, corrupt(desc, 2), "corrupt")):
        with pytest.raises(raas.RaasError) as e:
            pool.load_layer(0, data)
        assert e.value.code == raas.E_INVALID and why in str(e.value), str(e.value)
    for pool in (a, b, other):
        pool.close()


def test_pool_memory_is_fixed():
    """O(L) memory (Section 4.3): the pool's bytes are set at creation and
    resident tokens never exceed the budget."""
    import torch

    w = small(decode_steps=400)
    pool = new_pool(w)
    b0 = pool.pool_bytes()
    K, V = synth.prefill(w, 2, 0)
    pool.prefill(0, to_device(K, w.dtype), to_device(V, w.dtype))
    q, k, v = synth.steps(w, 2, 0, 0, w.decode_steps)
    qd, kd, vd = to_device(q, w.dtype), to_device(k, w.dtype), to_device(v, w.dtype)
    out = torch.empty((w.batch, w.n_q_heads, w.head_dim), dtype=torch.bfloat16, device="cuda")
    for i in range(w.decode_steps):
        pool.decode_step(0, qd[i], kd[i], vd[i], out)
        if i % 50 == 49:
            st = pool.export_state(0)
            resident = np.where(st["state"] != 0, st["fill"], 0).sum(axis=1)
            assert np.all(resident <= w.budget)
    assert pool.pool_bytes() == b0
    pool.close()


# ---- full-size workloads, benchmark launch configuration, sampled units ----

def _sample_units(w, n, seed=0):
    rng = np.random.default_rng(seed)
    U = w.batch * w.n_kv_heads
    picks = {0, U - 1}
    while len(picks) < min(n, U):
        picks.add(int(rng.integers(0, U)))
    return sorted(picks)


def test_llama8b_b1_full_run():
    """Batch-1 Llama-3.1-8B layer, L=1024: all 8 units, every step of the
    full 8192-step run; outputs every 16th step."""
    w = synth.get_workload("llama8b-b1-L1024")
    _say("case %s steps %d" % (w.name, w.decode_steps))
    rep = run_parity(w, seed=0, steps=w.decode_steps, out_every=16, chunk=256)
    _report(rep, w.name)
    assert rep.evictions > 0


def test_llama8b_b32_full_run():
    """Batch-32 Llama-3.1-8B layer, L=2048 (the benchmark workload), the
    whole run: all 256 units, all 16384 decode steps, in the launch
    configuration the benchmark times. The budget fills after 1024 decode
    steps; retention is compared for every unit at every step, outputs of
    every unit every 256th step."""
    w = synth.get_workload("llama8b-b32-L2048")
    steps = w.decode_steps
    _say("case %s steps %d all units" % (w.name, steps))
    rep = run_parity(w, seed=0, steps=steps, out_every=256, chunk=256)
    _report(rep, w.name)
    assert rep.evictions > 0 and rep.units_checked == 256 and rep.steps == steps


@pytest.mark.parametrize("layer", [0, 13, 27])
def test_qwen7b_28_layer_stack(layer):
    """Qwen2.5-7B-shaped stack (28 layers, 28/4 heads, batch 64, L=4096):
    the full 28-layer pool, one layer run past the budget (2048 prompt
    tokens pin 128 of the 256 pages; the rest fill after 2048 decode
    steps); 8 sampled units checked step by step."""
    w = synth.get_workload("qwen7b-28L-b64-L4096")
    steps = 2048 + 512
    _say("case %s layer %d steps %d" % (w.name, layer, steps))
    pool = new_pool(w)
    rep = run_parity(w, seed=0, steps=steps, layer=layer, units=_sample_units(w, 8, seed=layer), out_every=64,
                     chunk=256, pool=pool, others="ring", inv_every=16)
    pool.close()
    _report(rep, "%s layer %d" % (w.name, layer))
    assert rep.evictions > 0


@pytest.mark.parametrize("name,steps", [("llama8b-b128-ps32-L512", 600), ("llama8b-b128-ps32-L2048", 600),
                                        ("llama8b-b128-ps32-L8192", 4096 + 512)])
def test_stress_sweep(name, steps):
    """Batch 128, page 32, prefill 4096, heavy-tailed keys, 8 sampled units.
    At L=512 and 2048 the prefill overflows the budget: S-1 pages pinned,
    each decode page evicted once full. At L=8192 the prompt pins 128 of the
    256 pages and the decode pages fill the rest after 4096 steps: the run
    goes 512 steps past that point."""
    w = synth.get_workload(name)
    _say("case %s steps %d" % (name, steps))
    units = _sample_units(w, 8)
    rep = run_parity(w, seed=0, steps=steps, units=units, out_every=8 if steps < 1000 else 64, chunk=128,
                     others="ring", inv_every=8)
    _report(rep, name)
    assert rep.evictions > 0


@pytest.mark.parametrize("name,kw,steps", [
    ("llama8b-b128-ps32-L2048", dict(aggregation=1), 300),
    ("llama8b-b128-ps32-L512", dict(prompt_tokens=4096, prompt_topk=8, splits=2), 640),
    ("llama8b-b128-ps32-L512", dict(prompt_tokens=4096, prompt_topk=8, aggregation=1), 640),
], ids=["softmax-sum", "selection-kernel", "selection-kernel-softmax-sum"])
def test_stress_variants(name, kw, steps):
    """Variants on the batch-128 stress pools (1 GB and more, beyond the
    memory-side cache, so read with non-temporal loads): the softmax
    aggregation on the fused workgroup, and Quest on the prompt through the
    selection kernel and the list-driven step (a split plan, and the
    softmax aggregation); 4 sampled units, past the budget."""
    w = synth.get_workload(name)
    _say("case %s %s steps %d" % (name, kw, steps))
    rep = run_parity(w, seed=0, steps=steps, units=_sample_units(w, 4), out_every=16, chunk=128,
                     others="ring", inv_every=8, **kw)
    _report(rep, "%s %s" % (name, kw))
    assert rep.evictions > 0


def test_stress_dense_equivalence():
    """L = N (36864 tokens), the whole run of 32768 decode steps: the output
    is dense attention over every token (the oracle is exactly that at
    L >= N); 4 sampled units, outputs every 512th step, the last at 36864
    resident tokens. The budget is exactly full after the last token, so the
    eager eviction of Algorithm 1 frees one page of every unit at the last
    step (after its attention) and at no earlier step."""
    w = synth.get_workload("llama8b-b128-ps32-dense")
    steps = w.decode_steps
    _say("case %s steps %d" % (w.name, steps))
    rep = run_parity(w, seed=0, steps=steps, units=_sample_units(w, 4), out_every=512, chunk=64, others="ring",
                     inv_every=1024)
    _report(rep, w.name)
    assert rep.steps == steps
    assert rep.first_eviction_step == steps - 1 and rep.evictions == w.batch * w.n_kv_heads


# Score variants (raas_config.score_aggregation and rank_pinned) against the
# oracle switched the same way: (aggregation, rank_pinned), 1 = sum of
# per-head softmax.
VARIANTS = [(0, True), (1, False), (1, True)]
VARIANT_CASES = [
    dict(),                                                         # fused step kernel
    dict(budget=512, prefill_len=100, decode_steps=520, splits=3),  # split path and epilogue kernel
    dict(dtype="f32"),
    dict(n_q_heads=28, n_kv_heads=4),                               # G = 7
    dict(n_q_heads=2, n_kv_heads=2),                                # G = 1
    dict(prefill_len=1000),                                         # S-1 pinned pages, one decode slot
    dict(prefill_len=0),                                            # nothing pinned
    dict(head_dim=64, page_size=8, budget=64, prefill_len=21),
    dict(page_size=8, budget=2400, prefill_len=2300),               # 300 slots, radix select
    dict(page_size=8, budget=16384, prefill_len=16000, decode_steps=60),  # 2048 slots, 2047 of them pinned
]


@pytest.mark.parametrize("agg,rank", VARIANTS, ids=["agg%d-rank%d" % v for v in VARIANTS])
@pytest.mark.parametrize("case", VARIANT_CASES, ids=[",".join("%s=%s" % kv for kv in c.items()) or "base"
                                                     for c in VARIANT_CASES])
def test_score_variants(agg, rank, case):
    case = dict(case)
    splits = case.pop("splits", None)
    w = small(decode_steps=case.pop("decode_steps", 300), **case)
    _say("case variant agg %d rank_pinned %d %s splits %s" % (agg, rank, case, splits))
    rep = run_parity(w, seed=7, steps=w.decode_steps, splits=splits, aggregation=agg, rank_pinned=rank)
    _report(rep, "variant")


@pytest.mark.parametrize("name,steps,units,splits", [("llama8b-b32-L2048", 1024 + 320, 6, None),
                                                     ("llama8b-b1-L1024", 1024, 8, None),
                                                     ("llama8b-b1-L1024", 1024, 8, 4)])
def test_score_variants_full_size(name, steps, units, splits):
    """Both variants together at full size, in the benchmark's launch
    configuration (one fused workgroup per unit for both), and llama8b-b1
    split over 4 workgroups per unit (the epilogue kernel)."""
    w = synth.get_workload(name)
    _say("case variant agg 1 rank_pinned 1 %s steps %d splits %s" % (name, steps, splits))
    rep = run_parity(w, seed=1, steps=steps, units=_sample_units(w, units), out_every=32, chunk=128,
                     aggregation=1, rank_pinned=True, splits=splits)
    _report(rep, name + " variant")
    assert rep.evictions > 0


# One page table per (sequence, layer) shared by its KV heads (decision
# scope 1), against the oracle's grouped step; (aggregation, rank_pinned).
SCOPE_VARIANTS = [(0, False), (1, False), (0, True)]
SCOPE_CASES = [
    dict(),                                                         # 2 KV heads per sequence
    dict(n_q_heads=16, n_kv_heads=4, budget=512, prefill_len=100, decode_steps=520, splits=3),
    dict(dtype="f32"),
    dict(n_q_heads=28, n_kv_heads=4),                               # G = 7
    dict(n_q_heads=4, n_kv_heads=1),                                # one KV head: the per-head rule
    dict(prefill_len=1000),                                         # S-1 pinned pages
]


@pytest.mark.parametrize("agg,rank", SCOPE_VARIANTS, ids=["agg%d-rank%d" % v for v in SCOPE_VARIANTS])
@pytest.mark.parametrize("case", SCOPE_CASES, ids=[",".join("%s=%s" % kv for kv in c.items()) or "base"
                                                   for c in SCOPE_CASES])
def test_sequence_scope(agg, rank, case):
    case = dict(case)
    splits = case.pop("splits", None)
    w = small(decode_steps=case.pop("decode_steps", 300), **case)
    _say("case sequence-scope agg %d rank_pinned %d %s splits %s" % (agg, rank, case, splits))
    rep = run_parity(w, seed=9, steps=w.decode_steps, splits=splits, aggregation=agg, rank_pinned=rank,
                     scope=1)
    _report(rep, "sequence-scope")
    assert rep.evictions > 0


def test_sequence_scope_full_size():
    """One page table per sequence on the benchmark workload: two sampled
    sequences (16 units), in the launch configuration the benchmark times
    with this scope."""
    w = synth.get_workload("llama8b-b32-L2048")
    steps = 1024 + 320
    _say("case sequence-scope %s steps %d" % (w.name, steps))
    rep = run_parity(w, seed=2, steps=steps, units=[3 * w.n_kv_heads, 29 * w.n_kv_heads], out_every=32,
                     chunk=128, scope=1)
    _report(rep, w.name + " sequence-scope")
    assert rep.evictions > 0 and rep.units_checked == 16


RAGGED = [
    dict(),
    dict(dtype="f32"),
    dict(dtype="f32", head_dim=64),                    # the fused fp32 kernel
    dict(splits=3, budget=512),
    dict(scope=1),
    dict(scope=1, aggregation=1, rank_pinned=True),
    dict(rank_pinned=True),
    dict(prompt_tokens=128, prompt_topk=3),            # prompt selection in the step kernel
    dict(prompt_tokens=128, prompt_topk=3, splits=3),  # the selection kernel
]


@pytest.mark.parametrize("case", RAGGED, ids=[",".join("%s=%s" % kv for kv in c.items()) or "base" for c in RAGGED])
def test_ragged_batch(case):
    """Per-sequence prompt lengths (0, ragged, overflowing the budget), a
    random mask of the sequences taking each step, and two prompts replaced
    mid-run (a finished request's place reused)."""
    case = dict(case)
    wkw = {k: case.pop(k) for k in ("dtype", "budget", "head_dim") if k in case}
    w = small(batch=4, decode_steps=260, **wkw)
    lens = [0, 5, 40, 1000]
    _say("case ragged %s %s lens %s" % (wkw, case, lens))
    rep = run_ragged(w, seed=21, lens=lens, steps=w.decode_steps, reprefill={90: {1: 77}, 170: {3: 0, 0: 33}},
                     **case)
    _report(rep, "ragged")
    assert rep.evictions > 0


# 640 units in workgroups of 4 wavefronts, two per CU: 512 fit at once, so
# the hardware starts the other 128 as the first ones finish
def _many_units_workload(**kw):
    return small(batch=160, n_q_heads=16, n_kv_heads=4, budget=160, prefill_len=40, decode_steps=200, **kw)


def test_many_units_every_step():
    """More units than workgroups that fit at once: every unit, every step."""
    w = _many_units_workload()
    _say("case many units %d" % (w.batch * w.n_kv_heads))
    rep = run_parity(w, seed=13, steps=w.decode_steps)
    _report(rep, "many units")
    assert rep.units_checked == w.batch * w.n_kv_heads and rep.evictions > 0


def test_many_units_ragged():
    """The same with a mask of active sequences and prompts replaced mid-run."""
    w = _many_units_workload()
    lens = [(37 * i) % 300 for i in range(w.batch)]
    _say("case many units ragged")
    rep = run_ragged(w, seed=23, lens=lens, steps=w.decode_steps, reprefill={80: {3: 0, 77: 290}})
    _report(rep, "many units ragged")
    assert rep.evictions > 0


@pytest.mark.parametrize("name,steps,units", [("mistral7b-b4-P128-L1024", 1100, 6), ("mistral7b-b4-P128-dense", 300, 4)])
def test_decode_sweep_shapes(name, steps, units):
    """The decode-length sweep's layer (prompt 128, batch 4, split over
    several workgroups per unit): past the budget at L = 1024; dense
    attention over every token when the pool holds them all."""
    w = synth.get_workload(name)
    _say("case %s steps %d" % (name, steps))
    rep = run_parity(w, seed=4, steps=steps, units=_sample_units(w, units), out_every=16, chunk=128)
    _report(rep, name)
    if "dense" in name:
        assert rep.evictions == 0
    else:
        assert rep.evictions > 0


# Quest on the prompt pages, RaaS on the decode pages: a prompt region of
# prompt_tokens tokens, the prompt_topk prompt pages of largest bound attended
# each step (the oracle switched the same way).
PROMPT_CASES = [
    dict(prompt_tokens=128, prompt_topk=3, prefill_len=100),
    dict(prompt_tokens=128, prompt_topk=3, prefill_len=1000),                      # prompt over the region
    dict(prompt_tokens=128, prompt_topk=8, prefill_len=120),                       # every prompt page
    dict(prompt_tokens=320, prompt_topk=5, prefill_len=300, budget=512, decode_steps=520, splits=3),
    dict(prompt_tokens=256, prompt_topk=2, prefill_len=250, page_size=32, dtype="f32"),
    dict(prompt_tokens=128, prompt_topk=1, prefill_len=128, page_size=64, budget=256),
    dict(prompt_tokens=192, prompt_topk=4, prefill_len=190, n_q_heads=28, n_kv_heads=4),
    dict(prompt_tokens=128, prompt_topk=3, prefill_len=100, aggregation=1),
    dict(prompt_tokens=128, prompt_topk=3, prefill_len=100, scope=1),
    # in-step selection at more prompt pages: bound tiles over several rounds
    # per wavefront and a partial last tile (100 pages), more candidates than
    # one pass of eight pages per wavefront takes (top 40), head_dim 64, seven
    # query heads per KV head, page 32 with heavy-tailed key outliers
    dict(prompt_tokens=1600, prompt_topk=40, prefill_len=1590, decode_steps=200),
    dict(prompt_tokens=512, prompt_topk=6, prefill_len=500, head_dim=64),
    dict(prompt_tokens=1024, prompt_topk=10, prefill_len=1000, n_q_heads=28, n_kv_heads=4, decode_steps=200),
    dict(prompt_tokens=2048, prompt_topk=8, prefill_len=2048, page_size=32, budget=256, outlier_p=0.05,
         decode_steps=400),
]


@pytest.mark.parametrize("case", PROMPT_CASES, ids=[",".join("%s=%s" % kv for kv in c.items()) for c in PROMPT_CASES])
def test_prompt_selection(case):
    case = dict(case)
    run_kw = {k: case.pop(k) for k in ("prompt_tokens", "prompt_topk", "splits", "aggregation", "scope") if k in case}
    w = small(decode_steps=case.pop("decode_steps", 300), **case)
    _say("case prompt-selection %s %s" % (case, run_kw))
    rep = run_parity(w, seed=13, steps=w.decode_steps, **run_kw)
    _report(rep, "prompt-selection")
    assert rep.evictions > 0


@pytest.mark.parametrize("splits,page_size,budget", [(None, 16, 128), (2, 16, 128), (2, 8, 2400)],
                         ids=["fused", "epilogue-count", "epilogue-radix"])
def test_retention_exact_ties(splits, page_size, budget):
    """Every decode page holds the same sixteen (or eight) keys as every
    other page of its parity (two key sets, A for even pages and B for odd
    ones), so the ranked scores come in two values, equal in any summation
    order: the refresh's strict comparison with theta and the (timestamp,
    id) eviction order meet exact ties at every step. Retention must match
    the oracle bit for bit at every step (no near-tie allowance), on the
    fused workgroup's retention, the epilogue's count and its radix select
    (300 slots)."""
    import torch

    w = small(batch=2, n_kv_heads=2, n_q_heads=8, decode_steps=400, prefill_len=40, page_size=page_size,
              budget=budget)
    ps, B, Hkv, G, d, S = w.page_size, w.batch, w.n_kv_heads, w.group, w.head_dim, w.slots
    U = B * Hkv
    rng = np.random.default_rng(41)
    K = to_device(rng.standard_normal((B, Hkv, 40, d)).astype(np.float32), "bf16")
    V = to_device(rng.standard_normal((B, Hkv, 40, d)).astype(np.float32), "bf16")
    sets = to_device(rng.standard_normal((2, ps, B, Hkv, d)).astype(np.float32), "bf16")
    _say("case retention ties splits %s page %d budget %d" % (splits, ps, budget))
    pool = new_pool(w, splits)
    pool.prefill(0, K, V)
    Kr = K.float().cpu().numpy().astype(np.float64)
    Vr = V.float().cpu().numpy().astype(np.float64)
    orc = []
    for u in range(U):
        b, h = divmod(u, Hkv)
        m = oracle.Kvm(G, d, ps, S, r=w.r)
        assert m.prefill(Kr[b, h], Vr[b, h]) == 0
        orc.append(m)
    out = torch.empty((B, w.n_q_heads, d), dtype=torch.bfloat16, device="cuda")
    pt = torch.empty((B, Hkv, S), dtype=torch.int32, device="cuda")
    ts = torch.empty((B, Hkv, S), dtype=torch.int32, device="cuda")
    ev = torch.empty((B, Hkv), dtype=torch.int32, device="cuda")
    evictions = 0
    rep = ParityReport(units_checked=U)
    for t in range(w.decode_steps):
        qb = to_device(rng.standard_normal((B, w.n_q_heads, d)).astype(np.float32), "bf16")
        kb = sets[(t // ps) % 2, t % ps].contiguous()
        vb = to_device(rng.standard_normal((B, Hkv, d)).astype(np.float32), "bf16")
        pool.decode_step(0, qb, kb, vb, out, pt, ts, ev)
        torch.cuda.synchronize()
        got = out.float().cpu().numpy().reshape(U, G, d)
        pt_h, ts_h, ev_h = pt.cpu().numpy().reshape(U, S), ts.cpu().numpy().reshape(U, S), ev.cpu().numpy().reshape(U)
        q64 = qb.float().cpu().numpy().astype(np.float64).reshape(U, G, d)
        k64 = kb.float().cpu().numpy().astype(np.float64).reshape(U, d)
        v64 = vb.float().cpu().numpy().astype(np.float64).reshape(U, d)
        for u in range(U):
            want = orc[u].decode(q64[u], k64[u], v64[u])
            st = orc[u].state()
            assert np.array_equal(st["page_table"], pt_h[u]) and np.array_equal(st["ts"], ts_h[u]) \
                and st["evicted"] == ev_h[u], "unit %d step %d:\noracle pt %s ts %s ev %d\n   gpu pt %s ts %s ev %d" % (
                    u, t, st["page_table"].tolist(), st["ts"].tolist(), st["evicted"], pt_h[u].tolist(),
                    ts_h[u].tolist(), ev_h[u])
            evictions += int(st["evicted"] >= 0)
            compare_outputs(got[u][None], want[None], "bf16", "unit %d step %d" % (u, t), rep)
        rep.steps = t + 1
    pool.close()
    rep.evictions = evictions
    record(rep, "retention ties")
    assert evictions > 0 or budget > w.prefill_len + w.decode_steps


@pytest.mark.parametrize("splits", [None, 2], ids=["in-step", "selection-kernel"])
def test_prompt_selection_ties(splits):
    """Prompt pages 1, 4 and 6 copy page 2's keys (scaled up so that the four
    lead the bounds) with values of their own: their bounds are equal in any
    summation order, so with top 3 the tie rule alone keeps slot 6 out, and a
    wrong tie-break changes the outputs. Every unit, every step, against the
    oracle; the oracle's own choice is checked too."""
    import torch

    w = small(batch=2, n_kv_heads=2, n_q_heads=8, decode_steps=60, prefill_len=128)
    ps, npr, topk = w.page_size, 128 // w.page_size, 3
    B, Hkv, G, d = w.batch, w.n_kv_heads, w.group, w.head_dim
    U, S = B * Hkv, w.slots + npr
    rng = np.random.default_rng(31)
    K = rng.standard_normal((B, Hkv, 128, d)).astype(np.float32)
    V = rng.standard_normal((B, Hkv, 128, d)).astype(np.float32)
    K[:, :, 2 * ps:3 * ps] *= 3.0
    for pg in (1, 4, 6):
        K[:, :, pg * ps:(pg + 1) * ps] = K[:, :, 2 * ps:3 * ps]
    Kb = to_device(K, "bf16")
    Vb = to_device(V, "bf16")
    Kr, Vr = Kb.float().cpu().numpy().astype(np.float64), Vb.float().cpu().numpy().astype(np.float64)
    _say("case prompt-selection ties splits %s" % splits)
    pool = new_pool(w, splits, prompt_tokens=128, prompt_topk=topk)
    pool.prefill(0, Kb, Vb)
    orc = []
    for u in range(U):
        b, h = divmod(u, Hkv)
        m = oracle.Kvm(G, d, ps, S, r=w.r, prompt_slots=npr, prompt_topk=topk)
        assert m.prefill(Kr[b, h], Vr[b, h]) == 0
        orc.append(m)
    out = torch.empty((B, w.n_q_heads, d), dtype=torch.bfloat16, device="cuda")
    chosen_without_6 = 0
    rep = ParityReport(units_checked=U)
    for t in range(w.decode_steps):
        q = rng.standard_normal((B, w.n_q_heads, d)).astype(np.float32)
        kn = rng.standard_normal((B, Hkv, d)).astype(np.float32)
        vn = rng.standard_normal((B, Hkv, d)).astype(np.float32)
        qb, kb, vb = to_device(q, "bf16"), to_device(kn, "bf16"), to_device(vn, "bf16")
        pool.decode_step(0, qb, kb, vb, out)
        torch.cuda.synchronize()
        got = out.float().cpu().numpy().reshape(U, G, d)
        q64 = qb.float().cpu().numpy().astype(np.float64).reshape(U, G, d)
        k64 = kb.float().cpu().numpy().astype(np.float64).reshape(U, d)
        v64 = vb.float().cpu().numpy().astype(np.float64).reshape(U, d)
        for u in range(U):
            want = orc[u].decode(q64[u], k64[u], v64[u])
            att = orc[u].last_attended()[:npr]
            if att[1] and att[2] and att[4] and not att[6]:
                chosen_without_6 += 1
            compare_outputs(got[u][None], want[None], "bf16", "unit %d step %d" % (u, t), rep)
        rep.steps = t + 1
    pool.close()
    record(rep, "prompt-selection ties")
    assert chosen_without_6 > 0  # the tie decided the top 3 in some steps


@pytest.mark.parametrize("splits,B,P,copies", [(None, 64, 4608, (1, 4, 6)), (2, 64, 4608, (1, 4, 6)),
                                                (2, 2, 8192, (1, 600, 1000))],
                         ids=["in-step", "selection-kernel", "selection-kernel-few-units"])
def test_prompt_selection_ties_large_region(splits, B, P, copies):
    """The tie case where the selection goes by a radix select: 512 units
    with a 4608-token prompt region at page 8, 576 kept pages, more than
    twice the in-step workgroup's threads (4 wavefronts) and more than the
    selection kernel's 256. In every unit prompt pages 1, 4 and 6 copy page
    2's keys, scaled so that the four lead the bounds: with top 3 the cut
    (or theta) is the bound the four share, and the tie rule alone keeps
    slot 6 out. Few units: 16 units over 1024 prompt pages (the selection
    kernel's 8-wavefront form), the copies at pages 1, 600 and 1000, and the
    rule keeps 1000 out.
    Keys are drawn on the GPU; four sampled units against the oracle at
    every step."""
    import torch

    Hkv, Hq, d, ps, topk, budget, steps = 8, 32, 128, 8, 3, 256, 40
    w = synth.get_workload("llama8b-b128-ps32-L512").replace(
        name="prompt-ties-large-region", batch=B, page_size=ps, budget=budget, prefill_len=P)
    G, U, npr = Hq // Hkv, B * Hkv, P // ps
    S = budget // ps + npr
    gen = torch.Generator(device="cuda")
    gen.manual_seed(37)
    K = torch.randn((B, Hkv, P, d), generator=gen, device="cuda")
    V = torch.randn((B, Hkv, P, d), generator=gen, device="cuda")
    K[:, :, 2 * ps:3 * ps] *= 3.0
    for pg in copies:
        K[:, :, pg * ps:(pg + 1) * ps] = K[:, :, 2 * ps:3 * ps]
    tied = sorted((2,) + tuple(copies))
    Kb, Vb = K.to(torch.bfloat16).contiguous(), V.to(torch.bfloat16).contiguous()
    del K, V
    units = _sample_units(w, 4)
    _say("case prompt-selection ties, large region, splits %s: units %s" % (splits, units))
    pool = new_pool(w, splits, prompt_tokens=P, prompt_topk=topk)
    pool.prefill(0, Kb, Vb)
    orc = {}
    for u in units:
        b, h = divmod(u, Hkv)
        m = oracle.Kvm(G, d, ps, S, r=w.r, prompt_slots=npr, prompt_topk=topk)
        assert m.prefill(Kb[b, h].float().cpu().numpy().astype(np.float64),
                         Vb[b, h].float().cpu().numpy().astype(np.float64)) == 0
        orc[u] = m
    del Kb, Vb
    out = torch.empty((B, Hq, d), dtype=torch.bfloat16, device="cuda")
    chosen_without_last = 0
    rep = ParityReport(units_checked=len(units))
    for t in range(steps):
        qb = torch.randn((B, Hq, d), generator=gen, device="cuda").to(torch.bfloat16)
        kb = torch.randn((B, Hkv, d), generator=gen, device="cuda").to(torch.bfloat16)
        vb = torch.randn((B, Hkv, d), generator=gen, device="cuda").to(torch.bfloat16)
        pool.decode_step(0, qb, kb, vb, out)
        torch.cuda.synchronize()
        got = out.float().cpu().numpy().reshape(U, G, d)
        q64 = qb.float().cpu().numpy().astype(np.float64).reshape(U, G, d)
        k64 = kb.float().cpu().numpy().astype(np.float64).reshape(U, d)
        v64 = vb.float().cpu().numpy().astype(np.float64).reshape(U, d)
        for u in units:
            want = orc[u].decode(q64[u], k64[u], v64[u])
            att = orc[u].last_attended()[:npr]
            if all(att[pg] for pg in tied[:3]) and not att[tied[3]]:
                chosen_without_last += 1
            compare_outputs(got[u][None], want[None], "bf16", "unit %d step %d" % (u, t), rep)
        rep.steps = t + 1
    pool.close()
    record(rep, "prompt-selection ties, large region")
    assert chosen_without_last == len(units) * steps  # the four lead at every step; the tie decides


@pytest.mark.parametrize("splits", [None, 2], ids=["in-step", "selection-kernel"])
def test_prompt_selection_extreme_keys(splits):
    """Prompt pages whose bounds stress the in-step selection's intervals:
    keys scaled by 30 and by 1/30, channels of subnormal bf16 keys, an
    all-zero page, a page of negative zeros but one channel, and queries
    with subnormal channels; top 3 of 8 pages, every unit and step against
    the oracle."""
    import torch

    w = small(batch=2, n_kv_heads=2, n_q_heads=8, decode_steps=60, prefill_len=128)
    ps, npr, topk = w.page_size, 128 // w.page_size, 3
    B, Hkv, G, d = w.batch, w.n_kv_heads, w.group, w.head_dim
    U, S = B * Hkv, w.slots + npr
    rng = np.random.default_rng(37)
    K = rng.standard_normal((B, Hkv, 128, d)).astype(np.float32)
    V = rng.standard_normal((B, Hkv, 128, d)).astype(np.float32)
    K[:, :, 0:ps] *= 30.0
    K[:, :, ps:2 * ps] /= 30.0
    K[:, :, 2 * ps:3 * ps, : d // 2] = np.float32(1e-39) * np.sign(K[:, :, 2 * ps:3 * ps, : d // 2])
    K[:, :, 3 * ps:4 * ps] = 0.0
    K[:, :, 4 * ps:5 * ps] = -0.0
    K[:, :, 4 * ps:5 * ps, 7] = 1.0
    Kb = to_device(K, "bf16")
    Vb = to_device(V, "bf16")
    assert (Kb[:, :, 2 * ps:3 * ps, : d // 2].abs().float().max().item()) < 1.2e-38  # subnormal in bf16
    Kr, Vr = Kb.float().cpu().numpy().astype(np.float64), Vb.float().cpu().numpy().astype(np.float64)
    _say("case prompt-selection extreme keys splits %s" % splits)
    pool = new_pool(w, splits, prompt_tokens=128, prompt_topk=topk)
    pool.prefill(0, Kb, Vb)
    orc = []
    for u in range(U):
        b, h = divmod(u, Hkv)
        m = oracle.Kvm(G, d, ps, S, r=w.r, prompt_slots=npr, prompt_topk=topk)
        assert m.prefill(Kr[b, h], Vr[b, h]) == 0
        orc.append(m)
    out = torch.empty((B, w.n_q_heads, d), dtype=torch.bfloat16, device="cuda")
    rep = ParityReport(units_checked=U)
    chosen = np.zeros(npr, dtype=np.int64)
    for t in range(w.decode_steps):
        q = rng.standard_normal((B, w.n_q_heads, d)).astype(np.float32)
        q[:, :, : d // 4] *= np.float32(1e-39) if t % 2 else np.float32(1.0)
        kn = rng.standard_normal((B, Hkv, d)).astype(np.float32)
        vn = rng.standard_normal((B, Hkv, d)).astype(np.float32)
        qb, kb, vb = to_device(q, "bf16"), to_device(kn, "bf16"), to_device(vn, "bf16")
        pool.decode_step(0, qb, kb, vb, out)
        torch.cuda.synchronize()
        got = out.float().cpu().numpy().reshape(U, G, d)
        q64 = qb.float().cpu().numpy().astype(np.float64).reshape(U, G, d)
        k64 = kb.float().cpu().numpy().astype(np.float64).reshape(U, d)
        v64 = vb.float().cpu().numpy().astype(np.float64).reshape(U, d)
        for u in range(U):
            want = orc[u].decode(q64[u], k64[u], v64[u])
            chosen += np.asarray(orc[u].last_attended()[:npr], dtype=np.int64)
            compare_outputs(got[u][None], want[None], "bf16", "unit %d step %d" % (u, t), rep)
        rep.steps = t + 1
    pool.close()
    record(rep, "prompt-selection extreme keys")
    assert chosen.min() < U * w.decode_steps and chosen.max() > 0  # a real choice among the pages


@pytest.mark.parametrize("batch,prompt,splits", [(128, 3072, None), (64, 4608, None), (64, 4608, 2)],
                         ids=["1024-units", "512-units", "512-units-selection-kernel"])
def test_prompt_selection_large_region(batch, prompt, splits):
    """Prompt regions of more pages than twice a workgroup's threads (page 8:
    384 kept pages at batch 128, whose 1024 units run in workgroups of 2
    wavefronts, four per CU; 576 at batch 64, 512 units in workgroups of 4),
    and slots likewise (416 and 608): the in-step selection stages fills and
    slot records past the two each thread reads with its first loads, and
    finds its cut by a radix select. Split in two, the selection kernel
    chooses the pages, by its radix select beyond 256 pages. The decode
    budget (256 tokens) runs past full; sampled units."""
    w = synth.get_workload("llama8b-b128-ps32-L512").replace(
        name="prompt-region-%d" % prompt, batch=batch, page_size=8, budget=256, prefill_len=prompt)
    _say("case prompt-selection large region batch %d prompt %d" % (batch, prompt))
    rep = run_parity(w, seed=0, steps=400, units=_sample_units(w, 4), out_every=16, chunk=128, splits=splits,
                     prompt_tokens=prompt, prompt_topk=12)
    _report(rep, "prompt-selection large region")
    assert rep.evictions > 0


@pytest.mark.parametrize("ragged", [False, True, "fused"], ids=["uniform", "ragged", "fused-512-pages"])
def test_prompt_selection_few_units(ragged):
    """Fewer units than CUs over a long prompt region (page 8, 1024 prompt
    slots, 16 units, split plans): the selection kernel in its 8-wavefront
    form, bound intervals over 64 tiles, its cut by a radix select past 256
    pages, and the block list placed by a prefix count over 1024 prompt
    blocks. Ragged: prompts of 0, 40 (fewer pages than topk, nothing to
    rank), 3000 and 8192 tokens on four sequences that take steps by a
    random mask, two of them re-prefilled mid-run. Fused: 8 units over 512
    prompt pages at page 16 with the plan's own choice, one fused workgroup
    of 8 wavefronts per unit selecting in the step kernel (its count over
    512 lower ends). Every unit, every step."""
    if ragged == "fused":
        w = small(batch=2, n_q_heads=16, n_kv_heads=4, page_size=16, budget=256, prefill_len=8192,
                  decode_steps=300)
        _say("case prompt-selection few units, fused, 512 prompt pages")
        rep = run_parity(w, seed=7, steps=w.decode_steps, prompt_tokens=8192, prompt_topk=10)
    elif ragged:
        w = small(batch=4, n_q_heads=16, n_kv_heads=4, page_size=8, budget=128, decode_steps=300)
        _say("case prompt-selection few units, ragged")
        rep = run_ragged(w, seed=29, lens=[0, 40, 3000, 8192], steps=w.decode_steps,
                         reprefill={100: {1: 8000}, 200: {3: 600}}, splits=3, prompt_tokens=8192, prompt_topk=5)
    else:
        w = small(batch=2, n_q_heads=32, n_kv_heads=8, page_size=8, budget=256, prefill_len=8192,
                  decode_steps=300)
        _say("case prompt-selection few units")
        rep = run_parity(w, seed=5, steps=w.decode_steps, splits=2, prompt_tokens=8192, prompt_topk=12)
    _report(rep, "prompt-selection few units")
    assert rep.evictions > 0


@pytest.mark.parametrize("name,topk,steps,units", [("llama8b-b128-ps32-L512", 8, 640, 8),
                                                   ("llama8b-b128-ps32-L2048", 16, 2112, 4)])
def test_prompt_selection_full_size(name, topk, steps, units):
    """The long-prompt stress shapes (prompt 4096 tokens, page 32) with the
    whole prompt kept in a prompt region, topk prompt pages attended per
    step, and the decode budget run past full: sampled units."""
    w = synth.get_workload(name)
    _say("case prompt-selection %s topk %d steps %d" % (name, topk, steps))
    rep = run_parity(w, seed=0, steps=steps, units=_sample_units(w, units), out_every=16, chunk=128,
                     prompt_tokens=w.prefill_len, prompt_topk=topk)
    _report(rep, name + " prompt-selection")
    assert rep.evictions > 0
