"""ctypes declarations of the C ABI in include/oq.h (argument marshalling only)."""
from __future__ import annotations

import ctypes as C
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liboq.so")

i32, i64, vp, fp = C.c_int32, C.c_int64, C.c_void_p, C.POINTER(C.c_float)


class oq_dit_config(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("arch", "n_blocks", "hidden", "mlp", "n_heads", "head_dim",
                                         "tokens", "prefix", "batch", "steps", "action_dim")]


class oq_qweight(C.Structure):
    _fields_ = [("wq", vp), ("w_scale", vp)]


class oq_dit_block(C.Structure):
    _fields_ = [("g1", vp), ("g2", vp), ("qkv", oq_qweight), ("o", oq_qweight),
                ("gate_up", oq_qweight), ("down", oq_qweight), ("prefix_k", vp), ("prefix_v", vp),
                ("b2", vp), ("cross_kv", oq_qweight)]


class oq_dit_weights(C.Structure):
    _fields_ = [("w_in", vp), ("b_in", vp), ("w_out", vp), ("b_out", vp), ("g_f", vp),
                ("blocks", C.POINTER(oq_dit_block)), ("mod", vp), ("s_table", fp)]


class oq_dit_intermediates(C.Structure):
    _fields_ = [(n, vp) for n in ("h1", "qkv", "attn", "h2", "gate_up", "act", "resid", "cond_kv", "codes",
                                  "x_scale")] + [("codes_tiled", i32)]


# name -> (restype, argtypes)
SIGNATURES = {
    "oq_status_string": (C.c_char_p, [i32]),
    "oq_version": (C.c_char_p, []),
    "oq_check_device": (i32, []),
    "oq_rotate_quantize_act": (i32, [vp, i64, i64, i64, i32, fp, i32, vp, vp, vp]),
    "oq_rotate_quantize_act_tiled": (i32, [vp, i64, i64, i64, i32, fp, i32, vp, vp, vp]),
    "oq_rotate_debug_f32": (i32, [vp, i64, i64, i64, i32, fp, i32, vp, vp, vp]),
    "oq_w4a4_linear": (i32, [vp, vp, i64, vp, vp, vp, i64, i64, vp, i64, i32, vp]),
    "oq_w4a4_gemm_i32": (i32, [vp, i64, vp, i64, i64, vp, i64, vp]),
    "oq_w4a4_linear_tiled": (i32, [vp, vp, i64, vp, vp, vp, i64, i64, vp, i64, i32, vp]),
    "oq_w4a4_gemm_i32_tiled": (i32, [vp, i64, vp, i64, i64, vp, i64, vp]),
    "oq_codes_to_tiled": (i32, [vp, i64, i64, vp, vp]),
    "oq_rotate_quantize_act_composite": (i32, [vp, i64, i64, i64, vp, vp, fp, i32, vp, vp, vp]),
    "oq_zigzag_permutation_host": (i32, [vp, i64, i32, vp]),
    "oq_block_rotations_host": (i32, [vp, i64, i32, vp]),
    "oq_quantize_weights_composite_host": (i32, [vp, i64, i64, i32, vp, vp, vp, vp]),
    "oq_quantize_weights": (i32, [vp, i64, i64, i64, i32, vp, vp, vp]),
    "oq_quantize_weights_host": (i32, [vp, i64, i64, i32, vp, vp]),
    "oq_rotate_act_f32": (i32, [vp, i64, i64, i64, i32, vp, vp]),
    "oq_channel_energy": (i32, [vp, i64, i64, i64, vp, vp]),
    "oq_zigzag_permutation": (i32, [vp, i64, i32, vp, vp]),
    "oq_block_svd": (i32, [vp, i64, i64, i64, vp, i32, vp, vp, vp]),
    "oq_block_rotations": (i32, [vp, i64, i32, vp, vp]),
    "oq_prepare_weights_workspace_bytes": (C.c_size_t, [i64]),
    "oq_prepare_weights_composite": (i32, [vp, i64, i64, i64, vp, vp, vp, vp, vp, C.c_size_t, vp]),
    "oq_rotate_quantize_act_i8": (i32, [vp, i64, i64, i64, i32, fp, i32, vp, vp, vp]),
    "oq_w4a8_linear": (i32, [vp, vp, i64, vp, vp, vp, i64, i64, vp, i64, i32, vp]),
    "oq_w4a8_gemm_i32": (i32, [vp, i64, vp, i64, i64, vp, i64, vp]),
    "oq_calibrate_workspace_bytes": (C.c_size_t, [i64]),
    "oq_calibrate_step_scales": (i32, [vp, i64, i64, i64, C.c_double, C.c_float, vp, vp, C.c_size_t, vp]),
    "oq_calibrate_step_scales_noalloc": (i32, [vp, i64, i64, i64, C.c_double, C.c_float, vp, vp]),
    "oq_rotate_quantize_act_static": (i32, [vp, i64, i64, i64, i32, vp, vp, vp, vp]),
    "oq_rotate_quantize_act_static_tiled": (i32, [vp, i64, i64, i64, i32, vp, vp, vp, vp]),
    "oq_quantize_weights_step_host": (i32, [vp, i64, i64, i32, vp, vp, vp]),
    "oq_dit_workspace_bytes": (i32, [C.POINTER(oq_dit_config), C.POINTER(C.c_size_t)]),
    "oq_dit_create": (i32, [C.POINTER(oq_dit_config), C.POINTER(oq_dit_weights), C.POINTER(vp)]),
    "oq_dit_set_workspace": (i32, [vp, vp, C.c_size_t]),
    "oq_dit_set_condition": (i32, [vp, vp, vp]),
    "oq_dit_step": (i32, [vp, vp, i32, vp]),
    "oq_dit_denoise": (i32, [vp, vp, i32, vp]),
    "oq_dit_run_block": (i32, [vp, i32, i32, vp, vp]),
    "oq_dit_run_block_until": (i32, [vp, i32, i32, vp, i32, vp]),
    "oq_dit_get_intermediates": (i32, [vp, C.POINTER(oq_dit_intermediates)]),
    "oq_dit_set_static_steps": (i32, [vp, vp, C.POINTER(oq_qweight)]),
    "oq_dit_in_projection": (i32, [vp, vp, vp, vp]),
    "oq_dit_final_stage": (i32, [vp, vp, vp, vp]),
    "oq_quantize_weights_step": (i32, [vp, i64, i64, i64, i32, vp, vp, vp, vp]),
    "oq_dit_destroy": (None, [vp]),
}

_lib = None


def load(path: str = LIB_PATH) -> C.CDLL:
    """Load liboq.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2605_28803_amd.build` "
                           "(or __graft_entry__.build()); this package has no non-HIP fallback")
    lib = C.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        if hasattr(lib, name):
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
    _lib = lib
    return lib


def header_symbols(header: str) -> list:
    """Names of the functions declared in include/oq.h."""
    import re
    txt = open(header).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(oq_[a-z0-9_]+)\s*\(", txt)))
