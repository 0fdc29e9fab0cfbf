"""The C-ABI library loads and exports every symbol include/sara.h declares;
synchronous argument checks work without a GPU (no compute calls here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "sara.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:int|void|const char\*)\s+(\w+)\s*\(", src, flags=re.M)))


def test_header_declares_the_hot_path_calls():
    names = declared_functions()
    for n in ["sara_init", "sara_decode_step", "sara_posterior_decide", "sara_refill",
              "grpo_group_advantages", "sara_begin_step", "sara_query", "sara_destroy"]:
        assert n in names


def test_library_exports_every_declared_symbol():
    import paper_2607_26253_amd as sara
    lib = ctypes.CDLL(sara.LIB_PATH)
    for n in declared_functions():
        assert hasattr(lib, n), n
    assert set(sara.EXPORTED) == set(declared_functions())


def test_struct_layouts_match_header():
    import paper_2607_26253_amd as sara
    assert ctypes.sizeof(sara.sara_model_desc) == 11 * 4
    assert ctypes.sizeof(sara.sara_alloc_desc) == 4 * 4 + 3 * 8 + 8 + 6 * 4 + 2 * 4 + 4 + 4 + 8
    assert ctypes.sizeof(sara.sara_step_stats) == 10 * 4 + 7 * 8


def _descs(**over):
    import paper_2607_26253_amd as sara
    import workloads as W
    cfg = W.get_config("tiny_f32")
    a = dict(cfg["alloc"])
    m = dict(cfg["model"])
    for k, v in over.items():
        (a if k in a else m)[k] = v
    return sara.model_desc(m), sara.alloc_desc(a, 1)


@pytest.mark.parametrize("over", [dict(k=1), dict(n0=0), dict(n0=9), dict(commit_min=1), dict(tau_low=1.5),
                                  dict(alpha0=0.0), dict(kv_block=8), dict(top_p=0.0), dict(top_p=1.5), dict(head_dim=96),
                                  dict(n_kv_heads=3), dict(temperature=0.0), dict(n_slots=0),
                                  dict(budget_N=10 ** 6, pool_U=10 ** 4), dict(prio_quant_bits=30),
                                  dict(eos_id=512)])
def test_invalid_configurations_are_rejected(over):
    import paper_2607_26253_amd as sara
    md, ad = _descs(**over)
    h = ctypes.c_void_p()
    arr = (ctypes.c_void_p * 21)(*([1] * 21))
    rc = sara._lib.sara_init(ctypes.byref(md), ctypes.byref(ad), arr, 21, None, ctypes.byref(h))
    assert rc == sara.SARA_EINVAL
    assert len(sara._lib.sara_last_error()) > 0
    assert not h.value


def test_wrong_weight_count_and_null_pointers():
    import paper_2607_26253_amd as sara
    md, ad = _descs()
    h = ctypes.c_void_p()
    arr = (ctypes.c_void_p * 21)(*([1] * 21))
    assert sara._lib.sara_init(ctypes.byref(md), ctypes.byref(ad), arr, 20, None, ctypes.byref(h)) == sara.SARA_EINVAL
    arr[5] = None
    assert sara._lib.sara_init(ctypes.byref(md), ctypes.byref(ad), arr, 21, None, ctypes.byref(h)) == sara.SARA_EINVAL
    assert b"weight pointer 5" in sara._lib.sara_last_error()


def test_pure_entry_points_validate_arguments():
    import paper_2607_26253_amd as sara
    L = sara._lib
    assert L.sara_peff_batch(None, None, None, None, 8, -1, None, None) == sara.SARA_EINVAL
    assert L.sara_peff_batch(None, None, None, None, 8, 4, None, None) == sara.SARA_EINVAL
    fake = ctypes.c_void_p(16)
    assert L.sara_peff_batch(fake, None, fake, fake, 8, 4, fake, None) == sara.SARA_EINVAL
    assert L.sara_peff_batch(fake, fake, fake, fake, 0, 4, fake, None) == sara.SARA_EINVAL
    assert L.sara_poll(None, None) == sara.SARA_EINVAL
    assert L.grpo_group_advantages(None, None, -2, 1e-6, None, None) == sara.SARA_EINVAL
    assert L.grpo_group_advantages(None, None, 3, 1e-6, None, None) == sara.SARA_EINVAL
    assert L.sara_sample_logits(None, 4, 0, None, None, 0, 0, 1.0, 1.0, -1, 0, None, None) == sara.SARA_EINVAL
    # top_p outside (0, 1] is refused before anything is enqueued
    for bad in (0.0, -0.5, 1.01):
        assert L.sara_sample_logits(fake, 4, 512, fake, fake, 0, 0, 1.0, bad, -1, 0, fake, None) == sara.SARA_EINVAL
    assert L.sara_set_warm_start(None, None, None, None, 0) == sara.SARA_EINVAL
    assert L.sara_warm_start_update(None, 0.5) == sara.SARA_EINVAL
    assert L.sara_begin_step(None, None, None, None, None, 0) == sara.SARA_EINVAL
    assert L.sara_decode_step(None, None, None, 0) == sara.SARA_EINVAL
    assert L.sara_posterior_decide(None) == sara.SARA_EINVAL
    assert L.sara_refill(None) == sara.SARA_EINVAL
    L.sara_destroy(None)
