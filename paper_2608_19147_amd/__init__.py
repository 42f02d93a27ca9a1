"""MI355X-native stage forward: one pipeline stage's stateful decode/verify
forward (INT4 W4A16 Llama decoder layers, beam-indirect KV cache, mask-based
rewind) behind the C ABI of libstage.so."""
from ._lib import EXPORTS, LIB_PATH, StageError, load  # noqa: F401
from .stage import KVState, Request, Stage  # noqa: F401
