"""ctypes view of liblitevlm.so (declared in include/litevlm.h).

Loading fails loudly when the library has not been built: there is no
fallback path of any kind.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblitevlm.so")

OK, ERR_NULL_POINTER, ERR_BAD_SHAPE, ERR_BAD_VALUE, ERR_UNSUPPORTED, ERR_MISALIGNED, \
    ERR_WORKSPACE, ERR_HIP = range(8)
F32, BF16, FP8_E4M3 = 0, 1, 2
MAX_VIEWS, MAX_VISUAL, MAX_BATCH, MAX_HEADS = 64, 16384, 256, 128
NOALLOC_SCRATCH_BYTES = 8 << 20
MAX_FUSED_VIEWS = 8

# Every symbol the header declares, with its C signature.
_vp, _i32, _f32, _f64, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_double, ctypes.c_size_t
SIGNATURES = {
    "litevlm_version": (_i32, []),
    "litevlm_status_string": (ctypes.c_char_p, [_i32]),
    "litevlm_patch_select": (_i32, [_i32, _i32, _i32, _vp, _vp, _vp, _f32, _f32, _vp, _vp, _vp, _vp]),
    "litevlm_token_score_topk_workspace": (_sz, [_i32, _i32, _i32, _i32, _i32, _i32]),
    "litevlm_token_score_topk": (_i32, [_i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp,
                                        _f32, _f32, _f32, _f32, _vp, _f64, _vp, _vp, _vp, _vp, _vp,
                                        _vp, _vp, _sz, _vp]),
    "litevlm_token_score_topk_noalloc": (_i32, [_i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp,
                                                _f32, _f32, _f32, _f32, _vp, _f64, _vp, _vp, _vp, _vp, _vp,
                                                _vp, _vp]),
    "litevlm_token_score_topk_rows_workspace": (_sz, [_i32, _i32, _i32, _i32, _i32, _i32, _i32]),
    "litevlm_token_score_topk_rows": (_i32, [_i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp,
                                             _vp, _f32, _f32, _f32, _f32, _vp, _f64, _vp, _vp, _vp,
                                             _vp, _vp, _vp, _vp, _sz, _vp]),
    "litevlm_select_score_topk": (_i32, [_i32, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _f32,
                                         _f32, _vp, _vp, _vp, _f32, _f32, _f32, _f32, _f64, _vp, _vp, _vp,
                                         _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "litevlm_prefill_attn": (_i32, [_i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _i32,
                                    _f32, _f32, _f32, _f32, _i32, _vp, _vp]),
    "litevlm_tsm_qk": (_i32, [_i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _f32, _f32,
                              _vp, _vp, _vp]),
    "litevlm_tsm_fold_gain": (_i32, [_i32, _i32, _vp, _vp, _vp, _vp]),
    "litevlm_gather_hidden": (_i32, [_i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp]),
    "litevlm_psm_param_count": (_sz, [_i32, _i32, _i32, _i32]),
    "litevlm_psm_workspace": (_sz, [_i32, _i32, _i32, _i32, _i32]),
    "litevlm_psm_forward": (_i32, [_i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _sz, _vp, _vp, _sz, _vp]),
    "litevlm_decode_attn_workspace": (_sz, [_i32, _i32, _i32, _i32, _i32, _i32]),
    "litevlm_decode_attn": (_i32, [_i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp,
                                   _i32, _f32, _f32, _f32, _f32, _vp, _vp, _sz, _vp]),
}

_LIB = None


class LiteVLMError(RuntimeError):
    def __init__(self, status: int, call: str):
        self.status = status
        msg = load().litevlm_status_string(status).decode()
        super().__init__(f"{call} failed: {msg} (status {status})")


def load() -> ctypes.CDLL:
    """The loaded library; raises if liblitevlm.so is missing."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                f"{LIB_PATH} is not built; run `python -m paper_2506_07416_amd.build` "
                "(or __graft_entry__.build()) first")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = lib
    return _LIB


def check(status: int, call: str) -> None:
    if status != OK:
        raise LiteVLMError(status, call)
