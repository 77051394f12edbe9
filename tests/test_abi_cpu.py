"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every entry point include/attuner.h declares, and rejects bad geometry before
touching a device."""

import ctypes as C
import os
import re

import pytest

from paper_2609_36722_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "attuner.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(attuner_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_entry_point():
    lib = _lib.lib()
    names = _declared()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), f"{n} not exported"
    assert set(names) == set(_lib.SIGNATURES), "binding and header disagree"


def test_bad_geometry_rejected_without_a_device():
    lib = _lib.lib()
    h = C.c_void_p()
    for field, val in [("head_dim", 64), ("page_tokens", 32), ("n_q_heads", 16), ("hidden", 100), ("n_layers", 0)]:
        cfg = _lib.ModelCfgC(36, 2560, 32, 8, 128, 16, 1e6, 1e-6)
        setattr(cfg, field, val)
        assert lib.attuner_create(C.byref(cfg), 16, 0, C.byref(h)) == -1
        assert field.split("_")[0] in lib.attuner_last_error().decode() or lib.attuner_last_error()
    assert lib.attuner_create(None, 16, 0, C.byref(h)) == -1


def test_null_context_is_an_error_not_a_crash():
    lib = _lib.lib()
    out = C.c_int32()
    assert lib.attuner_store_artifact(None, 4, None, None, None, C.byref(out)) == -1
    assert lib.attuner_release_artifact(None, 0) == -1
    assert lib.attuner_pool_info(None, None, None, None) == -1
    assert lib.attuner_qproj_lora(None, 1, None, None, 128, None, None, 0, 0.0, 0, None, None) == -1
    assert lib.attuner_assemble_table(None, 0, None, None, None, None, None, None, 0, None) == -1
    assert lib.attuner_gather_layers(None, None, 0, 0, 1, None, 0, None) == -1
    assert lib.attuner_embed(None, 1, None, None, 8, None, None) == -1
    assert lib.attuner_host_pool_create(None, 4) == -1
    assert lib.attuner_merge_lora(None, None, 64, 64, None, None, 0, 0.0, 0, None, None) == -1
    assert lib.attuner_store_artifact_host(None, 4, None, None, None, C.byref(out)) == -1
    assert lib.attuner_host_pool_info(None, None, None) == -1
    assert lib.attuner_assemble_segments_plan(None, 0, None, None, None, None, None) == -1
    assert lib.attuner_assemble_segments(None, 0, None, None, None, None, None, None, 0, None) == -1
    assert lib.attuner_span_attn(None, 0, 1, None, None, None, None, None, 0, None, None, 0, None, None, None, 0, None,
                                 None, None) == -1
    assert lib.attuner_decode_attn(None, 0, 1, None, None, None, None, 0, None, None, 0, None, None, None, 0, None,
                                   None) == -1
    assert lib.attuner_rms_norm(None, None, 1, 256, None, 1, None, None, None) == -1
    assert lib.attuner_linear(None, 1, None, 64, None, 64, None, None, None) == -1
    assert lib.attuner_gate_up_swiglu(None, 1, None, 64, None, 32, None, None) == -1
    assert lib.attuner_lm_head_argmax(None, 1, None, None, 64, None, None, None) == -1
    lib.attuner_destroy(None)


def test_checked_build_exports_the_same_abi():
    """libattuner_checked.so (device-side bounds tests) exports the same entry
    points and says which build it is; the ordinary build reports no
    violations without touching a device."""
    names = _declared()
    chk = _lib.load(_lib.CHECKED_LIB_PATH)
    for n in names:
        assert hasattr(chk, n), f"{n} not exported by the checked build"
    flag = C.c_int32(-1)
    assert chk.attuner_bounds_checked(C.byref(flag)) == 0 and flag.value == 1
    lib = _lib.load(os.path.join(os.path.dirname(_lib.CHECKED_LIB_PATH), _lib.VARIANTS[""]))
    assert lib.attuner_bounds_checked(C.byref(flag)) == 0 and flag.value == 0
    assert lib.attuner_bounds_checked(None) == -1
    bits = C.c_uint32(7)
    assert lib.attuner_bounds_violations(0, 1, C.byref(bits)) == 0 and bits.value == 0
    assert lib.attuner_bounds_violations(0, 1, None) == -1
    assert chk.attuner_bounds_violations(0, 1, None) == -1
