"""ctypes declarations of the C ABI in include/griffin_verify.h.

Argument marshalling only.  Importing this module loads the in-tree
libgriffin_verify.so and raises if it is missing: there is no fallback.
"""

from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_double, c_float, c_int32, c_int64, c_size_t, c_uint32, c_uint64, c_void_p, c_char_p

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "lib", "libgriffin_verify.so")

GRIFFIN_OK = 0
STATUS = {
    0: "GRIFFIN_OK", -1: "GRIFFIN_EINVAL", -2: "GRIFFIN_ESHAPE", -3: "GRIFFIN_ETREE", -4: "GRIFFIN_ETOKEN",
    -5: "GRIFFIN_ECAPACITY", -6: "GRIFFIN_EORDER", -7: "GRIFFIN_ENOMEM", -8: "GRIFFIN_EHIP",
    -9: "GRIFFIN_ENUMERIC",
}
CODES = {v: k for k, v in STATUS.items()}


class ModelDesc(ctypes.Structure):
    _fields_ = [
        ("n_layers", c_int32), ("d_model", c_int32), ("n_q_heads", c_int32), ("n_kv_heads", c_int32),
        ("head_dim", c_int32), ("d_ff", c_int32), ("vocab", c_int32), ("n_experts", c_int32),
        ("top_k", c_int32), ("rms_eps", c_float), ("rope_base", c_double), ("max_batch", c_int32),
        ("max_tree", c_int32), ("max_depth", c_int32), ("kv_capacity", c_int32),
    ]


class Weights(ctypes.Structure):
    _fields_ = [
        ("embed", c_void_p), ("lm_head", c_void_p), ("final_norm", c_void_p),
        ("attn_norm", POINTER(c_void_p)), ("w_qkv", POINTER(c_void_p)), ("w_o", POINTER(c_void_p)),
        ("mlp_norm", POINTER(c_void_p)), ("w_gate_up", POINTER(c_void_p)), ("w_down", POINTER(c_void_p)),
        ("w_router", POINTER(c_void_p)),
    ]


class DraftWeights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in (
        "w_m", "b_m", "ln_h_g", "ln_h_b", "ln_x_g", "ln_x_b", "w_u", "b_u", "w_d", "b_d", "w_p", "b_p", "w_r", "b_r",
        "attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")]


class GriffinError(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        self.name = STATUS.get(code, str(code))
        super().__init__(f"{what}: {self.name} ({code})")


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2502_11018_amd.build` "
            "(the verify path has no non-HIP fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    I32P = POINTER(c_int32)
    F32P = POINTER(c_float)
    sig = {
        "griffin_kv_cache_bytes": (c_size_t, [POINTER(ModelDesc)]),
        "griffin_verify_init": (c_int32, [POINTER(ModelDesc), POINTER(Weights), c_void_p, c_void_p, c_void_p,
                                          POINTER(c_void_p)]),
        "griffin_verify_step": (c_int32, [c_void_p, c_int32, I32P, I32P, I32P, I32P, c_void_p]),
        "griffin_accept": (c_int32, [c_void_p, I32P, I32P, I32P]),
        "griffin_read_predictions": (c_int32, [c_void_p, I32P]),
        "griffin_read_features": (c_int32, [c_void_p, c_int32, c_int32, I32P, c_void_p]),
        "griffin_read_router_logits": (c_int32, [c_void_p, F32P]),
        "griffin_read_margins": (c_int32, [c_void_p, F32P]),
        "griffin_set_activation_precision": (c_int32, [c_void_p, c_int32]),
        "griffin_verify_free": (None, [c_void_p]),
        "griffin_status_str": (c_char_p, [c_int32]),
        "griffin_last_error": (c_char_p, [c_void_p]),
        "griffin_tree_prepare": (c_int32, [c_int32, I32P, I32P, c_int32, c_int32, c_int32, c_int32, c_int32,
                                           I32P, I32P, POINTER(c_uint64)]),
        "griffin_accept_walk": (c_int32, [c_void_p, c_int32, c_int32, c_int32, c_int32, I32P, I32P, I32P, I32P,
                                          I32P, I32P, I32P]),
        "griffin_profile_enable": (c_int32, [c_void_p, c_uint32]),
        "griffin_profile_read": (c_int32, [c_void_p, POINTER(c_double), POINTER(c_int64)]),
        "griffin_set_graphs": (c_int32, [c_void_p, c_int32]),
        "griffin_commit": (c_int32, [c_void_p]),
        "griffin_accept_sampled": (c_int32, [c_void_p, c_void_p, c_void_p, F32P, F32P, c_float, I32P, I32P, I32P]),
        "griffin_accept_sampled_walk": (c_int32, [c_void_p, c_int32, c_int32, c_int32, c_int32, I32P, I32P, I32P,
                                                  c_void_p, c_void_p, F32P, F32P, c_float, I32P, I32P, I32P]),
        "griffin_accept_sampled_walk_noalloc": (c_int32, [c_void_p, c_int32, c_int32, c_int32, c_int32, I32P, I32P,
                                                          I32P, c_void_p, c_void_p, F32P, F32P, c_float, I32P, I32P,
                                                          I32P]),
        "griffin_draft_init": (c_int32, [POINTER(ModelDesc), c_int32, c_float, POINTER(DraftWeights), c_void_p,
                                         c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, POINTER(c_void_p)]),
        "griffin_draft_free": (None, [c_void_p]),
        "griffin_draft_context": (c_void_p, [c_void_p]),
        "griffin_draft_step": (c_int32, [c_void_p, c_int32, I32P, I32P, I32P, I32P, c_void_p, c_int32, I32P, F32P]),
        "griffin_draft_extend": (c_int32, [c_void_p, c_int32, I32P, I32P, I32P, c_void_p]),
        "griffin_draft_tree": (c_int32, [c_void_p, c_int32, I32P, I32P, c_void_p, c_int32, c_int32, c_int32, I32P,
                                         I32P, I32P, F32P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()
EXPORTED = ("griffin_kv_cache_bytes", "griffin_verify_init", "griffin_verify_step", "griffin_accept",
            "griffin_read_predictions", "griffin_verify_free", "griffin_status_str", "griffin_last_error",
            "griffin_tree_prepare", "griffin_accept_walk", "griffin_profile_enable", "griffin_profile_read",
            "griffin_set_graphs", "griffin_commit", "griffin_accept_sampled", "griffin_accept_sampled_walk",
            "griffin_draft_init", "griffin_draft_free", "griffin_draft_context", "griffin_draft_step",
            "griffin_draft_tree", "griffin_read_features", "griffin_draft_extend",
            "griffin_set_activation_precision", "griffin_read_router_logits", "griffin_read_margins",
            "griffin_accept_sampled_walk_noalloc")
KERNEL_CLASSES = ("qkv_gemm", "rope_kv_write", "tree_attention", "o_gemm", "residual_rmsnorm", "gate_up_gemm",
                  "down_gemm", "lm_head_gemm", "argmax_accept_route", "attn_merge")
