"""ctypes declarations of libstage.so (include/stage.h).  Marshalling only."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libstage.so")

STAGE_OK = 0
ERRORS = {
    -1: "STAGE_E_INVALID", -2: "STAGE_E_SHAPE", -3: "STAGE_E_CAPACITY", -4: "STAGE_E_OOM",
    -5: "STAGE_E_HIP", -6: "STAGE_E_STATE_MISMATCH", -7: "STAGE_E_UNSUPPORTED", -8: "STAGE_E_DEVICE",
}
DTYPE_F16 = 1
DTYPE_BF16 = 2
MAX_ROWS = 64
STATIC_SCRATCH_BYTES = 64 << 20   # STAGE_STATIC_SCRATCH_BYTES
MAX_PREFILL = 8192                # STAGE_MAX_PREFILL

# Every function that include/stage.h declares.
EXPORTS = (
    "stage_create", "stage_destroy", "kv_state_alloc", "kv_state_free", "kv_state_reset",
    "kv_append", "kv_length", "kv_read", "kv_truncate", "stage_forward",
    "stage_debug_dequant", "stage_weight_bytes", "stage_last_error",
    "stage_profile_enable", "stage_profile_read", "stage_profile_read_each", "stage_debug_phase_trace", "stage_device_status",
    "stage_debug_attn_arm", "stage_debug_attn_read",
    "kv_compact", "kv_capture_size", "kv_capture", "kv_restore", "kv_capture_noalloc",
    "stage_head_attach", "stage_head_top1", "stage_prefill", "stage_embed_attach", "stage_embed",
)
KERNEL_CLASSES = {"qkv": 0, "attn": 1, "oproj": 2, "gateup": 3, "down": 4, "persistent": 5}


class StageConfig(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32),
        ("group_size", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("act_dtype", ctypes.c_int32),
        ("kv_dtype", ctypes.c_int32), ("rope_theta", ctypes.c_double), ("max_positions", ctypes.c_int32),
        ("rope_cos_sin", ctypes.POINTER(ctypes.c_float)),
    ]


class QuantMatrix(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("scales", ctypes.c_void_p), ("n", ctypes.c_int32), ("k", ctypes.c_int32)]


class LayerWeights(ctypes.Structure):
    _fields_ = [("attn_norm", ctypes.c_void_p), ("ffn_norm", ctypes.c_void_p)] + [
        (name, QuantMatrix) for name in ("wq", "wk", "wv", "wo", "wg", "wu", "wd")
    ]


class StageRequest(ctypes.Structure):
    _fields_ = [
        ("state", ctypes.c_void_p), ("n_tokens", ctypes.c_int32), ("positions", ctypes.c_void_p),
        ("beam_idx", ctypes.c_void_p), ("attention_mask", ctypes.c_void_p), ("mask_len", ctypes.c_int32),
        ("attention_mask_rows", ctypes.c_void_p),
    ]


_lib = None


def load() -> ctypes.CDLL:
    """Load libstage.so; raises if it has not been built (no fallback path exists)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                          "(python -m paper_2608_19147_amd.build)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I, V = ctypes.POINTER, ctypes.c_int, ctypes.c_void_p
    sig = {
        "stage_create": (I, [P(StageConfig), P(LayerWeights), I, V, P(V)]),
        "stage_destroy": (I, [V]),
        "kv_state_alloc": (I, [V, I, I, P(V)]),
        "kv_state_free": (I, [V]),
        "kv_state_reset": (I, [V]),
        "kv_append": (I, [V, V, V, I, I, V]),
        "kv_length": (I, [V, P(I)]),
        "kv_read": (I, [V, I, I, I, I, V, V, I, V]),
        "kv_truncate": (I, [V, I]),
        "stage_forward": (I, [V, P(StageRequest), I, V, V, V]),
        "stage_debug_dequant": (I, [V, I, I, V]),
        "stage_weight_bytes": (ctypes.c_int64, [V]),
        "stage_last_error": (ctypes.c_char_p, []),
        "stage_profile_enable": (I, [V, I]),
        "stage_profile_read": (I, [V, P(I), P(ctypes.c_double)]),
        "stage_profile_read_each": (I, [V, V, I, P(I)]),
        "stage_debug_phase_trace": (I, [V, V, I, V]),
        "stage_device_status": (I, [V]),
        "stage_debug_attn_arm": (I, [V, I, I]),
        "stage_debug_attn_read": (I, [V, V, V, P(I), P(I)]),
        "kv_compact": (I, [V, V, V, V]),
        "kv_capture_size": (I, [V, V, P(ctypes.c_int64)]),
        "kv_capture": (I, [V, V, V, ctypes.c_int64, I, V]),
        "kv_restore": (I, [V, V, ctypes.c_int64, I, V, V]),
        "kv_capture_noalloc": (I, [V, V, V, ctypes.c_int64, V]),
        "stage_head_attach": (I, [V, V, P(QuantMatrix), I, V]),
        "stage_head_top1": (I, [V, V, I, V, V, V, V, V]),
        "stage_prefill": (I, [V, V, I, V, V, V, V, V]),
        "stage_embed_attach": (I, [V, V, I, I, V]),
        "stage_embed": (I, [V, V, I, V, V]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


class StageError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


def check(code: int) -> None:
    if code != STAGE_OK:
        raise StageError(code, load().stage_last_error().decode(errors="replace"))
