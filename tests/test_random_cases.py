"""The seeded random configurations of the GPU sweep (harness.random_case)
are valid pools and cover each switch both ways."""
from harness import random_case, random_large_case, random_prompt_case

from test_gpu_random import N_CASES, N_LARGE, N_PROMPT


def test_random_cases_are_valid_and_varied():
    cases = [random_case(i) for i in range(N_CASES)]

    def seen(f):
        return {f(c) for c in cases}

    assert seen(lambda c: c["workload"]["dtype"]) == {"bf16", "f32"}
    assert seen(lambda c: c["workload"]["head_dim"]) == {64, 128}
    assert seen(lambda c: c["variant"]["aggregation"]) == {0, 1}
    assert seen(lambda c: c["variant"]["scope"]) == {0, 1}
    assert seen(lambda c: c["variant"]["rank_pinned"]) == {False, True}
    assert seen(lambda c: c["variant"]["prompt_tokens"] > 0) == {False, True}
    assert seen(lambda c: c["splits"] is None) == {False, True}
    assert seen(lambda c: c["deterministic"]) == {False, True}
    assert len(seen(lambda c: c["workload"]["page_size"])) >= 4
    assert seen(lambda c: c["workload"]["prefill_len"] > c["workload"]["budget"]) == {False, True}
    for c in cases:
        w, v = c["workload"], c["variant"]
        assert w["n_q_heads"] % w["n_kv_heads"] == 0 and w["n_q_heads"] // w["n_kv_heads"] <= 16
        assert w["budget"] % w["page_size"] == 0
        assert v["prompt_tokens"] % w["page_size"] == 0 and v["prompt_tokens"] % 32 == 0
        assert 2 <= (w["budget"] + v["prompt_tokens"]) // w["page_size"] <= 2048
        assert not (v["rank_pinned"] and v["prompt_tokens"])
        assert v["prompt_topk"] <= v["prompt_tokens"] // w["page_size"]


def test_random_large_cases_are_valid():
    cases = [random_large_case(i) for i in range(max(N_LARGE, 16))]
    assert {c["variant"]["prompt_tokens"] > 0 for c in cases} == {False, True}
    assert any((c["workload"]["budget"] + c["variant"]["prompt_tokens"]) // c["workload"]["page_size"] > 256
               for c in cases)
    for c in cases:
        w, v = c["workload"], c["variant"]
        assert w["n_q_heads"] // w["n_kv_heads"] <= 16 and w["budget"] % w["page_size"] == 0
        assert v["prompt_tokens"] % w["page_size"] == 0 and v["prompt_tokens"] % 32 == 0
        assert 2 <= (w["budget"] + v["prompt_tokens"]) // w["page_size"] <= 2048
        assert not (v["rank_pinned"] and v["prompt_tokens"])
        assert v["prompt_topk"] <= v["prompt_tokens"] // w["page_size"]


def test_random_prompt_cases_are_valid():
    cases = [random_prompt_case(i) for i in range(max(N_PROMPT, 16))]
    pages = [c["variant"]["prompt_tokens"] // c["workload"]["page_size"] for c in cases]
    assert min(pages) <= 512 < max(pages) and any(p > 256 for p in pages)
    assert {c["workload"]["dtype"] for c in cases} == {"bf16", "f32"}
    for c in cases:
        w, v = c["workload"], c["variant"]
        npr = v["prompt_tokens"] // w["page_size"]
        assert w["batch"] * w["n_kv_heads"] <= 16 and w["n_q_heads"] // w["n_kv_heads"] <= 16
        assert v["prompt_tokens"] % w["page_size"] == 0 and v["prompt_tokens"] % 32 == 0
        assert 128 <= npr <= 1200 and 1 <= v["prompt_topk"] <= min(40, npr)
        assert 2 <= (w["budget"] + v["prompt_tokens"]) // w["page_size"] <= 2048
        assert w["budget"] % w["page_size"] == 0 and w["decode_steps"] > w["budget"] + w["page_size"]
        assert w["batch"] * w["n_kv_heads"] * w["prefill_len"] * w["head_dim"] <= 16 * 17000 * 128
