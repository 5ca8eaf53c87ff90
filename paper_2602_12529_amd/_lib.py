"""ctypes declarations of libff.so (include/ff.h, include/ff_ops.h, include/ff_loss.h).

Loading fails loudly when the library has not been built: there is no other
implementation to fall back to.
"""
from __future__ import annotations

import ctypes
import os
import threading
from ctypes import POINTER, c_char_p, c_double, c_float, c_int32, c_int64, c_size_t, c_uint32, c_uint64, c_void_p

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libff.so")

FF_OK, FF_EINVAL, FF_EDOMAIN, FF_EWORKSPACE, FF_EHIP, FF_EUNSUPPORTED = 0, -1, -2, -3, -4, -5
STATUS_NAMES = {0: "FF_OK", -1: "FF_EINVAL", -2: "FF_EDOMAIN", -3: "FF_EWORKSPACE", -4: "FF_EHIP",
                -5: "FF_EUNSUPPORTED"}


class DitConfig(ctypes.Structure):
    _fields_ = [
        ("model", c_int32), ("io_mode", c_int32), ("dtype", c_int32),
        ("n_dual", c_int32), ("n_single", c_int32), ("n_wan", c_int32),
        ("hidden", c_int32), ("heads", c_int32), ("head_dim", c_int32), ("mlp_hidden", c_int32),
        ("in_channels", c_int32), ("txt_dim", c_int32), ("pooled_dim", c_int32),
        ("norm_kind", c_int32), ("rope_axes", c_int32 * 3),
        ("rope_theta", c_double), ("norm_eps", c_double),
    ]


_SIGS = {
    "ff_last_error": (c_char_p, []),
    "ff_version": (c_char_p, []),
    "ff_sde_workspace_size": (c_int32, [c_int64, c_int64, POINTER(c_size_t)]),
    "ff_sde_step": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_int64, c_int64, c_double,
                              c_double, c_double, c_int32, c_void_p, c_size_t, c_void_p]),
    "ff_sde_step_noalloc": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_int64, c_int64, c_double,
                                      c_double, c_double, c_int32, c_void_p]),
    "ff_logprob": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_int64, c_int64, c_double, c_double,
                             c_double, c_int32, c_void_p, c_size_t, c_void_p]),
    "ff_sde_step_philox": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_int64, c_int64, c_double, c_double,
                                     c_double, c_uint64, c_uint32, c_int32, c_void_p, c_size_t, c_void_p]),
    "ff_philox_normal": (c_int32, [c_void_p, c_int64, c_int64, c_uint64, c_uint32, c_int32, c_void_p]),
    "ff_philox4x32": (c_int32, [c_void_p, c_int64, c_uint64, c_uint32, c_uint32, c_uint64, c_void_p]),
    "ff_group_advantage": (c_int32, [c_void_p, c_void_p, c_void_p, c_int64, c_int32, c_int32, c_int32, c_float,
                                     c_void_p, c_void_p, c_void_p]),
    "ff_dit_num_tensors": (c_int32, [POINTER(DitConfig), POINTER(c_int64)]),
    "ff_dit_tensor_info": (c_int32, [POINTER(DitConfig), c_int64, c_char_p, c_size_t, POINTER(c_int64),
                                     POINTER(c_int64)]),
    "ff_dit_create": (c_int32, [POINTER(DitConfig), POINTER(c_void_p), c_int64, POINTER(c_void_p)]),
    "ff_dit_destroy": (c_int32, [c_void_p]),
    "ff_dit_workspace_size": (c_int32, [c_void_p, c_int64, POINTER(c_int32), c_int64, c_int64, POINTER(c_size_t)]),
    "ff_dit_forward": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_int64, c_void_p, c_void_p,
                                 POINTER(c_int32), c_int64, c_int64, c_void_p, c_void_p, c_void_p, c_size_t,
                                 c_void_p]),
    "ff_dit_context_size": (c_int32, [c_void_p, c_int64, c_int64, POINTER(c_size_t)]),
    "ff_dit_prepare_context": (c_int32, [c_void_p, c_void_p, c_void_p, c_int64, POINTER(c_int32), c_int64, c_int64,
                                         c_void_p, c_size_t, c_void_p, c_size_t, c_void_p]),
    "ff_dit_forward_ctx": (c_int32, [c_void_p, c_void_p, c_void_p, c_size_t, c_void_p, POINTER(c_int32), c_int64,
                                     c_int64, c_void_p, c_void_p, c_size_t, c_void_p]),
    "ff_profile_enable": (c_int32, [c_int32]),
    "ff_profile_reset": (c_int32, []),
    "ff_profile_filter": (c_int32, [c_char_p]),
    "ff_profile_count": (c_int32, [POINTER(c_int32)]),
    "ff_profile_read": (c_int32, [c_int32, c_char_p, c_size_t, POINTER(c_int64), POINTER(c_double),
                                  POINTER(c_double), POINTER(c_double)]),
    "ff_linear": (c_int32, [c_void_p, c_int64, c_void_p, c_void_p, c_void_p, c_int64, c_int64, c_int64, c_int64,
                            c_int32, c_int64, c_void_p, c_int64, c_void_p, c_int64, c_int64, c_int32, c_void_p,
                            c_size_t, c_void_p]),
    "ff_linear_workspace_size": (c_int32, [POINTER(c_size_t)]),
    "ff_attention": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_int64, c_int64, c_int64, c_int64,
                               c_int64, c_int32, c_void_p]),
    "ff_norm_modulate": (c_int32, [c_void_p, c_void_p, c_int64, c_int64, c_void_p, c_void_p, c_int64, c_int64,
                                   c_int32, c_float, c_int32, c_void_p]),
    "ff_qk_norm_rope": (c_int32, [c_void_p, c_int64, c_int64, c_int64, c_int64, c_void_p, c_void_p, c_float,
                                  c_void_p, c_void_p, c_void_p, c_void_p, c_int64, c_int64, c_int32, c_void_p]),
    "ff_rope_table": (c_int32, [c_void_p, POINTER(c_int32), c_int32, POINTER(c_int32), c_double, c_void_p]),
    "ff_skinny_linear": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_int64, c_int64, c_int64, c_int32,
                                   c_int32, c_int32, c_void_p, c_void_p]),
    "ff_row_classes": (c_int32, [c_void_p, c_int64, c_int64, c_void_p, c_void_p]),
    "ff_quantize_fp8": (c_int32, [c_void_p, c_int64, c_void_p, c_int64, c_void_p, c_int64, c_int64, c_int32,
                                  c_void_p]),
    "ff_linear_fp8": (c_int32, [c_void_p, c_int64, c_void_p, c_void_p, c_int64, c_void_p, c_void_p, c_void_p,
                                c_int64, c_int64, c_int64, c_int64, c_int32, c_int64, c_void_p]),
    "ff_stream_probe": (c_int32, [c_int32, c_int32, c_void_p, c_void_p, c_int64, c_int32, c_void_p]),
    "ff_flow_noise": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_int64, c_int64, c_int32, c_void_p]),
    "ff_loss_workspace_size": (c_int32, [c_int64, c_int64, POINTER(c_size_t)]),
    "ff_awm_loss": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_int64, c_int64, c_int32, c_void_p, c_void_p,
                              c_void_p, c_size_t, c_void_p]),
    "ff_nft_loss": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_int64, c_int64, c_int32, c_void_p,
                              c_void_p, c_void_p, c_size_t, c_void_p]),
    "ff_grpo_loss": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_int64, c_int32, c_double, c_void_p,
                               c_void_p, c_void_p]),
}

_lib = None
_lock = threading.Lock()


def load() -> ctypes.CDLL:
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2602_12529_amd.build` "
                               "(there is no non-HIP implementation)")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
        return lib


class FFError(RuntimeError):
    def __init__(self, code: int, fn: str, msg: str):
        super().__init__(f"{fn} -> {STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


def check(rc: int, fn: str) -> None:
    if rc != FF_OK:
        raise FFError(rc, fn, load().ff_last_error().decode(errors="replace"))
