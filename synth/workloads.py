"""The five synthetic workloads of the RaaS decode path.

Shapes follow the attention layers of Llama-3.1-8B (32 query heads, 8 KV
heads, head_dim 128) and Qwen2.5-7B (28 layers, 28 query heads, 4 KV heads,
head_dim 128). Reasoning workloads have short prompts and long decodes
(Section 3.1, Limitations); the paper evaluates budgets 64..1024 with
page_size 16 and r = 0.5 (Section 4.1, Figure 5). The synthetic values stand
in for the paper's GSM8K / MATH500 / AIME runs: N(0,1) Q/K/V with planted
milestone tokens (Section 3.1), and for the stress sweep 5% heavy-tailed key
elements.
"""
from __future__ import annotations

import dataclasses


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str  # "f32" or "bf16"
    page_size: int
    budget: int  # L, tokens, includes the pinned prefill pages
    prefill_len: int
    decode_steps: int
    ms_period: int  # milestone every R-th decode step (0 = none)
    ms_phase_random: bool
    ms_wmin: int
    ms_wmax: int
    outlier_p: float = 0.0
    r: float = 0.5

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def slots(self) -> int:
        return self.budget // self.page_size

    @property
    def units_per_layer(self) -> int:
        return self.batch * self.n_kv_heads

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


_LLAMA = dict(n_q_heads=32, n_kv_heads=8, head_dim=128)

WORKLOADS = {
    # tiny, oracle-feasible: every 32nd decode token is a milestone, window 64
    "tiny-f32": Workload("tiny-f32", batch=1, n_layers=1, n_q_heads=4, n_kv_heads=1, head_dim=64,
                         dtype="f32", page_size=16, budget=256, prefill_len=64, decode_steps=1024,
                         ms_period=32, ms_phase_random=False, ms_wmin=64, ms_wmax=64),
    # one Llama-3.1-8B-shaped layer, batch 1
    "llama8b-b1-L1024": Workload("llama8b-b1-L1024", batch=1, n_layers=1, **_LLAMA, dtype="bf16",
                                 page_size=16, budget=1024, prefill_len=512, decode_steps=8192,
                                 ms_period=64, ms_phase_random=True, ms_wmin=256, ms_wmax=256),
    # the same layer at serving load: batch 32, L = 2048
    "llama8b-b32-L2048": Workload("llama8b-b32-L2048", batch=32, n_layers=1, **_LLAMA, dtype="bf16",
                                  page_size=16, budget=2048, prefill_len=1024, decode_steps=16384,
                                  ms_period=64, ms_phase_random=True, ms_wmin=64, ms_wmax=1024),
    # Qwen2.5-7B-shaped 28-layer stack, batch 64, L = 4096
    "qwen7b-28L-b64-L4096": Workload("qwen7b-28L-b64-L4096", batch=64, n_layers=28, n_q_heads=28,
                                     n_kv_heads=4, head_dim=128, dtype="bf16", page_size=16,
                                     budget=4096, prefill_len=2048, decode_steps=32768,
                                     ms_period=64, ms_phase_random=True, ms_wmin=64, ms_wmax=1024),
}

# stress sweep: batch 128, page 32, prefill 4096, heavy-tailed key outliers;
# L in {512, 2048, 8192} plus L = N (every token fits: dense equivalence)
for _L in (512, 2048, 8192, 4096 + 32768):
    _name = "llama8b-b128-ps32-L%d" % _L if _L != 36864 else "llama8b-b128-ps32-dense"
    WORKLOADS[_name] = Workload(_name, batch=128, n_layers=1, **_LLAMA, dtype="bf16", page_size=32,
                                budget=_L, prefill_len=4096, decode_steps=32768, ms_period=128,
                                ms_phase_random=True, ms_wmin=64, ms_wmax=1024, outlier_p=0.05)

# decode-length sweep (Fig. 6 setting: prompt 128, batch 4, decode up to 8k
# tokens): one Mistral-7B-shaped layer (32/8 heads, d 128), RaaS at two
# budgets, and a pool holding every token (dense attention)
for _L in (1024, 2048, 128 + 8192):
    _name = "mistral7b-b4-P128-L%d" % _L if _L != 8320 else "mistral7b-b4-P128-dense"
    WORKLOADS[_name] = Workload(_name, batch=4, n_layers=1, n_q_heads=32, n_kv_heads=8, head_dim=128,
                                dtype="bf16", page_size=16, budget=_L, prefill_len=128, decode_steps=8192,
                                ms_period=64, ms_phase_random=True, ms_wmin=64, ms_wmax=1024)

# the serving-load layer shape with four layers stepped per token: each
# layer's pool (268 MB) has left the 256 MB memory-side cache by the time its
# next step comes, so every step reads from HBM
WORKLOADS["llama8b-b32-L2048-x4"] = WORKLOADS["llama8b-b32-L2048"].replace(name="llama8b-b32-L2048-x4", n_layers=4)

HEADLINE = "llama8b-b32-L2048"


def get_workload(name: str) -> Workload:
    try:
        return WORKLOADS[name]
    except KeyError:
        raise KeyError("unknown workload %r; known: %s" % (name, ", ".join(WORKLOADS))) from None
