"""ctypes loader of libattuner.so (built in-tree by ``paper_2609_36722_amd.build``).

Loading fails loudly when the library is missing: there is no fallback path.
"""

from __future__ import annotations

import ctypes as C
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
# ATTUNER_LIB_VARIANT=checked loads the bounds-checked build (same ABI) instead
VARIANTS = {"": "libattuner.so", "checked": "libattuner_checked.so"}
VARIANT = os.environ.get("ATTUNER_LIB_VARIANT", "")
if VARIANT not in VARIANTS:
    raise RuntimeError(f"ATTUNER_LIB_VARIANT={VARIANT!r}: expected one of {sorted(VARIANTS)}")
LIB_PATH = os.path.join(_PKG, VARIANTS[VARIANT])
CHECKED_LIB_PATH = os.path.join(_PKG, VARIANTS["checked"])

STATUS = {0: "ATTUNER_OK", -1: "ATTUNER_EINVAL", -2: "ATTUNER_ENOMEM", -3: "ATTUNER_ENOENT",
          -4: "ATTUNER_EDEVICE", -5: "ATTUNER_ERANGE"}

MAX_REQUESTS = 64
MAX_RANK = 64
HOST_PAGE_FLAG = 1 << 30
STAGE_PAGE_FLAG = 1 << 29
NOALLOC_SCRATCH_BYTES = 24 << 20


class ModelCfgC(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("hidden", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("page_tokens", C.c_int32),
                ("rope_theta", C.c_float), ("rms_eps", C.c_float)]


class LimitsC(C.Structure):
    _fields_ = [("max_tokens", C.c_int32), ("max_position", C.c_int32), ("max_rank", C.c_int32),
                ("max_out", C.c_int32), ("max_lm_rows", C.c_int32), ("max_vocab", C.c_int32)]


class KernelTimeC(C.Structure):
    _fields_ = [("kernel", C.c_char * 48), ("launches", C.c_int64), ("total_ms", C.c_double), ("max_ms", C.c_double)]


_i32p = C.POINTER(C.c_int32)
_i64p = C.POINTER(C.c_int64)
_vp = C.c_void_p
_i32 = C.c_int32
_i64 = C.c_int64

# name -> (restype, argtypes); the exported C ABI of include/attuner.h
SIGNATURES = {
    "attuner_last_error": (C.c_char_p, []),
    "attuner_create": (C.c_int, [C.POINTER(ModelCfgC), _i64, _i32, C.POINTER(_vp)]),
    "attuner_destroy": (None, [_vp]),
    "attuner_reserve": (C.c_int, [_vp, C.POINTER(LimitsC)]),
    "attuner_pool_info": (C.c_int, [_vp, _i64p, _i64p, _i64p]),
    "attuner_store_artifact": (C.c_int, [_vp, _i32, _vp, _vp, _vp, _i32p]),
    "attuner_release_artifact": (C.c_int, [_vp, _i32]),
    "attuner_artifact_pages": (C.c_int, [_vp, _i32, _i32p, _i32, _i32p, _i32p]),
    "attuner_assemble_plan": (C.c_int, [_vp, _i32, _i32p, _i32p, _i32p, _i64p, _i64p]),
    "attuner_assemble_kv": (C.c_int, [_vp, _i32, _i32p, _i32p, _i32p, _vp, _i32p, _i32p, _vp, _i64, _vp]),
    "attuner_assemble_table": (C.c_int, [_vp, _i32, _i32p, _i32p, _i32p, _vp, _i32p, _i32p, _i64, _vp]),
    "attuner_gather_layers": (C.c_int, [_vp, _vp, _i64, _i32, _i32, _vp, _i64, _vp]),
    "attuner_qproj_lora": (C.c_int, [_vp, _i32, _vp, _vp, _i32, _vp, _vp, _i32, C.c_float, _i32, _vp, _vp]),
    "attuner_qk_norm_rope": (C.c_int, [_vp, _i32, _i32, _i32p, _i32p, _i32p, _i32p, _vp, _i64, _vp, _vp, _i64,
                                       _vp, _vp, _vp, _vp, _i64, _vp]),
    "attuner_attention": (C.c_int, [_vp, _i32, _i32, _i32p, _i32p, _i32p, _vp, _vp, _i64, _vp, _vp, _vp]),
    "attuner_suffix_attn": (C.c_int, [_vp, _i32, _i32, _i32p, _i32p, _i32p, _i32p, _vp, _i64, _vp, _vp, _i64,
                                      _vp, _vp, _vp, _i64, _vp, _vp, _vp]),
    "attuner_suffix_attn_noalloc": (C.c_int, [_vp, _i32, _i32, _i32p, _i32p, _i32p, _i32p, _vp, _i64, _vp, _vp,
                                              _i64, _vp, _vp, _vp, _i64, _vp, _vp, _vp]),
    "attuner_suffix_attn_gather": (C.c_int, [_vp, _i32, _i32, _i32p, _i32p, _i32p, _i32p, _vp, _i64, _vp, _vp,
                                             _i64, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _i64, _i32, _vp]),
    "attuner_merge_lora": (C.c_int, [_vp, _vp, _i32, _i32, _vp, _vp, _i32, C.c_float, _i32, _vp, _vp]),
    "attuner_host_pool_create": (C.c_int, [_vp, _i64]),
    "attuner_store_artifact_host": (C.c_int, [_vp, _i32, _vp, _vp, _vp, _i32p]),
    "attuner_host_pool_info": (C.c_int, [_vp, _i64p, _i64p]),
    "attuner_stage_pool_create": (C.c_int, [_vp, _i64]),
    "attuner_assemble_table_staged": (C.c_int, [_vp, _i32, _i32p, _i32p, _i32p, _vp, _i32p, _i32p, _i64, _i64p,
                                                _vp]),
    "attuner_stage_layers": (C.c_int, [_vp, _i32, _i32, _vp]),
    "attuner_stage_pool_info": (C.c_int, [_vp, _i64p, _i64p]),
    "attuner_assemble_segments_plan": (C.c_int, [_vp, _i32, _i32p, _i32p, _i64p, _i64p, _i32p]),
    "attuner_assemble_segments": (C.c_int, [_vp, _i32, _i32p, _i32p, _vp, _i32p, _i32p, _vp, _i64, _vp]),
    "attuner_span_attn": (C.c_int, [_vp, _i32, _i32, _i32p, _i32p, _i32p, _i32p, _vp, _i64, _vp, _vp, _i64, _vp, _vp,
                                    _vp, _i64, _vp, _vp, _vp]),
    "attuner_decode_attn": (C.c_int, [_vp, _i32, _i32, _i32p, _i32p, _i32p, _vp, _i64, _vp, _vp, _i64, _vp, _vp,
                                      _vp, _i64, _vp, _vp]),
    "attuner_embed": (C.c_int, [_vp, _i32, _i32p, _vp, _i32, _vp, _vp]),
    "attuner_rms_norm": (C.c_int, [_vp, _vp, _i64, _i64, _i32p, _i32, _vp, _vp, _vp]),
    "attuner_linear": (C.c_int, [_vp, _i32, _vp, _i32, _vp, _i32, _vp, _vp, _vp]),
    "attuner_gate_up_swiglu": (C.c_int, [_vp, _i32, _vp, _i32, _vp, _i32, _vp, _vp]),
    "attuner_lm_head_argmax": (C.c_int, [_vp, _i32, _vp, _vp, _i32, _vp, _vp, _vp]),
    "attuner_full_prefill": (C.c_int, [_vp, _i32, _i32, _vp, _vp, _vp, _vp, _i32, C.c_float, _vp, _vp, _vp, _vp,
                                       _vp, _vp, _vp]),
    "attuner_trace_begin": (C.c_int, [_vp]),
    "attuner_trace_end": (C.c_int, [_vp, C.POINTER(KernelTimeC), _i32, _i32p]),
    "attuner_bounds_checked": (C.c_int, [_i32p]),
    "attuner_bounds_violations": (C.c_int, [_i32, _i32, C.POINTER(C.c_uint32)]),
}

_LIB = None


def load(path: str) -> C.CDLL:
    """Load one build of the library and declare its exports."""
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run `python -m paper_2609_36722_amd.build` "
                           "(or __graft_entry__.build()) first")
    handle = C.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(handle, name)
        fn.restype = res
        fn.argtypes = args
    return handle


def lib() -> C.CDLL:
    """The library every binding call goes to (LIB_PATH), loaded once."""
    global _LIB
    if _LIB is None:
        _LIB = load(LIB_PATH)
    return _LIB
