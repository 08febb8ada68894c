"""The C-ABI library without a GPU: it loads, exports every entry point the
header declares, and rejects bad arguments before touching the device."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "raas.h")


@pytest.fixture(scope="module")
def lib():
    import paper_2502_11147_amd as raas

    if not os.path.exists(raas.LIB_PATH):
        from paper_2502_11147_amd import build as b

        b.build()
    return raas.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(raas_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for core in ("raas_create_pool", "raas_prefill", "raas_decode_step", "raas_destroy"):
        assert core in names


def test_library_exports_every_declared_symbol(lib):
    import paper_2502_11147_amd as raas

    names = declared_functions()
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(raas.EXPORTS) == names


def test_abi_version(lib):
    text = open(HEADER).read()
    v = int(re.search(r"#define RAAS_ABI_VERSION (\d+)", text).group(1))
    assert lib.raas_abi_version() == v


def _cfg(**kw):
    import paper_2502_11147_amd as raas

    base = dict(batch=2, n_layers=1, n_q_heads=8, n_kv_heads=2, head_dim=128, page_size=16,
                budget_tokens=256, dtype=raas.BF16, r=0.5, prefill_policy=raas.PREFILL_PIN_HEAD)
    base.update(kw)
    return raas.Config(**base)


BAD = [
    dict(batch=0), dict(n_layers=0), dict(n_kv_heads=0), dict(n_q_heads=7), dict(n_q_heads=0),
    dict(n_q_heads=34, n_kv_heads=2), dict(head_dim=96), dict(head_dim=0), dict(page_size=12),
    dict(page_size=4), dict(budget_tokens=250), dict(budget_tokens=16), dict(budget_tokens=0),
    dict(budget_tokens=16 * 2049), dict(dtype=7), dict(r=-0.1), dict(r=1.5), dict(r=float("nan")),
    dict(prefill_policy=3), dict(score_aggregation=2), dict(score_aggregation=-1), dict(rank_pinned=2),
    dict(rank_pinned=-1), dict(decision_scope=2), dict(decision_scope=-1),
    dict(decision_scope=1, n_q_heads=2048, n_kv_heads=128),
    dict(prompt_tokens=48, prompt_topk=2), dict(prompt_tokens=64, prompt_topk=0), dict(prompt_tokens=-32),
    dict(prompt_topk=3), dict(prompt_tokens=64, prompt_topk=2, rank_pinned=1),
    dict(prompt_tokens=32 * 1024, prompt_topk=2), dict(deterministic=2), dict(deterministic=-1),
]


def test_config_layout_matches_header():
    """The binding's Config lists raas_config's fields in the header's order."""
    import paper_2502_11147_amd as raas

    text = open(HEADER).read()
    body = re.search(r"typedef struct \{(.*?)\} raas_config;", text, re.S).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    fields = re.findall(r"(int32_t|double)\s+(\w+);", body)
    want = [(n, ctypes.c_int32 if t == "int32_t" else ctypes.c_double) for t, n in fields]
    assert [(n, t) for n, t in raas.Config._fields_] == want


@pytest.mark.parametrize("bad", BAD, ids=[",".join("%s=%s" % kv for kv in b.items()) for b in BAD])
def test_create_pool_rejects_bad_config(lib, bad):
    import paper_2502_11147_amd as raas

    h = ctypes.c_void_p()
    rc = lib.raas_create_pool(ctypes.byref(_cfg(**bad)), None, ctypes.byref(h))
    assert rc == raas.E_INVALID
    assert not h.value
    assert lib.raas_last_error().decode() != ""


def test_null_arguments(lib):
    import paper_2502_11147_amd as raas

    assert lib.raas_create_pool(None, None, None) == raas.E_INVALID
    h = ctypes.c_void_p()
    assert lib.raas_create_pool(None, None, ctypes.byref(h)) == raas.E_INVALID
    assert "cfg" in lib.raas_last_error().decode()
    assert lib.raas_prefill(None, 0, None, None, 0, None) == raas.E_INVALID
    assert lib.raas_decode_step(None, 0, None, None, None, None, None, None, None, None) == raas.E_INVALID
    assert lib.raas_decode_step_masked(None, 0, None, None, None, None, None, None, None, None,
                                       None) == raas.E_INVALID
    lens = (ctypes.c_int32 * 2)(1, 1)
    assert lib.raas_prefill_ragged(None, 0, None, None, lens, None, 1, None) == raas.E_INVALID
    buf = (ctypes.c_int32 * 8)()
    assert lib.raas_export_state(None, 0, buf, 8, None) == raas.E_INVALID
    assert lib.raas_set_attention_splits(None, 1) == raas.E_INVALID
    assert lib.raas_profile(None, 1) == raas.E_INVALID
    ms, n = ctypes.c_double(), ctypes.c_int64()
    assert lib.raas_profile_read(None, 0, ctypes.byref(ms), ctypes.byref(n)) == raas.E_INVALID
    assert lib.raas_pool_bytes(None) == 0
    assert lib.raas_layer_checkpoint_bytes(None) == 0
    assert lib.raas_save_layer(None, 0, None, 0, None) == raas.E_INVALID
    assert lib.raas_load_layer(None, 0, None, 0, None) == raas.E_INVALID
    lib.raas_destroy(None)  # NULL-safe


def test_last_error_is_per_thread(lib):
    import threading

    h = ctypes.c_void_p()
    lib.raas_create_pool(ctypes.byref(_cfg(batch=0)), None, ctypes.byref(h))
    seen = {}

    def other():
        seen["msg"] = lib.raas_last_error().decode()

    th = threading.Thread(target=other)
    th.start()
    th.join()
    assert seen["msg"] == ""
    assert "batch" in lib.raas_last_error().decode()


def test_binding_fails_loudly_without_library(tmp_path):
    import paper_2502_11147_amd as raas

    saved = raas._lib
    raas._lib = None
    try:
        with pytest.raises(RuntimeError, match="not built"):
            raas.load_library(str(tmp_path / "missing.so"))
    finally:
        raas._lib = saved


def test_kernel_digest_follows_code_not_comments():
    """The digest that stored counter profiles are checked against covers the
    kernels' code: comments and layout leave it alone, any token changes it."""
    from paper_2502_11147_amd import build

    a = "int f(int x) { // one\n  return x + 1; /* two */ }\n"
    b = "int f(int x) {\n\n  return x + 1;   }  // reworded\n"
    c = "int f(int x) { return x + 2; }"
    assert build._code_text(a) == build._code_text(b) == "int f(int x) { return x + 1; }"
    assert build._code_text(c) != build._code_text(a)
    assert len(build.kernel_digest()) == 64
