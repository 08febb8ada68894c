"""GPU parity over seeded random configurations (harness.random_case):
every switch of the C ABI drawn together, each run past its budget against
the oracle, every unit at every step (evicting), under the same bounds as the
hand-picked cases. The draws are fixed by the case index, so a failure
names a reproducible configuration."""
from __future__ import annotations

import os

import pytest

from harness import new_pool, random_case, random_large_case, random_prompt_case, record, run_parity, say

pytestmark = pytest.mark.gpu

N_CASES = int(os.environ.get("RAAS_RANDOM_CASES", "64"))  # more for a longer sweep
N_LARGE = int(os.environ.get("RAAS_RANDOM_LARGE_CASES", "16"))
N_PROMPT = int(os.environ.get("RAAS_RANDOM_PROMPT_CASES", "24"))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2502_11147_amd as raas

    raas.load_library()  # fails loudly when the HIP library is missing


@pytest.mark.parametrize("i", range(N_CASES), ids=["rand-%02d" % i for i in range(N_CASES)])
def test_random_config_parity(i):
    import synth

    c = random_case(i)
    w = synth.Workload(**c["workload"])
    say("case %s %s splits %s deterministic %s" % (c["workload"], c["variant"], c["splits"], c["deterministic"]))
    pool = new_pool(w, c["splits"], deterministic=c["deterministic"], **c["variant"])
    try:
        rep = run_parity(w, seed=50 + i, steps=w.decode_steps, pool=pool, **c["variant"])
    finally:
        pool.close()
    record(rep, "random %02d" % i)
    assert rep.flagged_divergences == 0, rep.line("random %02d" % i)
    assert rep.evictions > 0, rep.line("random %02d" % i)  # every case runs past its budget


@pytest.mark.parametrize("i", range(N_LARGE), ids=["large-%02d" % i for i in range(N_LARGE)])
def test_random_large_config_parity(i):
    """Long pools (harness.random_large_case): retention of every unit at
    every step, outputs every 32nd step, past the budget."""
    import synth

    c = random_large_case(i)
    w = synth.Workload(**c["workload"])
    say("case %s %s splits %s deterministic %s" % (c["workload"], c["variant"], c["splits"], c["deterministic"]))
    pool = new_pool(w, c["splits"], deterministic=c["deterministic"], **c["variant"])
    try:
        rep = run_parity(w, seed=90 + i, steps=w.decode_steps, pool=pool, out_every=32, **c["variant"])
    finally:
        pool.close()
    record(rep, "random large %02d" % i)
    assert rep.flagged_divergences == 0, rep.line("random large %02d" % i)
    assert rep.evictions > 0, rep.line("random large %02d" % i)


@pytest.mark.parametrize("i", range(N_PROMPT), ids=["prompt-%02d" % i for i in range(N_PROMPT)])
def test_random_prompt_region_parity(i):
    """Long prompt regions at a small batch (harness.random_prompt_case):
    four sampled units' retention at every step and outputs every 4th,
    past the budget; the other units replay a ring of seeded steps."""
    import numpy as np

    import synth

    c = random_prompt_case(i)
    w = synth.Workload(**c["workload"])
    U = w.batch * w.n_kv_heads
    units = sorted({0, U - 1} | set(int(x) for x in np.random.default_rng(i).integers(0, U, 2)))
    say("case %s %s splits %s deterministic %s units %s" % (c["workload"], c["variant"], c["splits"],
                                                             c["deterministic"], units))
    pool = new_pool(w, c["splits"], deterministic=c["deterministic"], **c["variant"])
    try:
        rep = run_parity(w, seed=130 + i, steps=w.decode_steps, pool=pool, units=units, out_every=4,
                         others="ring", **c["variant"])
    finally:
        pool.close()
    record(rep, "random prompt %02d" % i)
    assert rep.flagged_divergences == 0, rep.line("random prompt %02d" % i)
    assert rep.evictions > 0, rep.line("random prompt %02d" % i)
