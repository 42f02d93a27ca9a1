"""Python binding of libstage: argument marshalling only.

Every step of the forward runs in the HIP kernels of libstage.so; torch is used
for device buffers (``data_ptr``) and for the current HIP stream.
"""
from __future__ import annotations

import atexit
import ctypes
import weakref
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np
import torch

from . import _lib
from ._lib import check

MATRIX_NAMES = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")
_DT = {"f16": _lib.DTYPE_F16, "bf16": _lib.DTYPE_BF16}
_TORCH = {"f16": torch.float16, "bf16": torch.bfloat16}


_LIVE_STATES: "weakref.WeakSet[KVState]" = weakref.WeakSet()
_LIVE_STAGES: "weakref.WeakSet[Stage]" = weakref.WeakSet()


def close_all() -> None:
    """Free every live KV state, then every live stage.  Registered with
    atexit, so the library's device synchronizations and frees run while the
    interpreter and the HIP runtime are both still whole, rather than from
    ``__del__`` during interpreter shutdown."""
    for kv in list(_LIVE_STATES):
        kv.free()
    for st in list(_LIVE_STAGES):
        st.close()


atexit.register(close_all)


def _stream_ptr(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


def _ptr(a) -> int:
    if isinstance(a, torch.Tensor):
        return a.data_ptr()
    return a.ctypes.data


class Stage:
    """One pipeline stage on the current GPU.

    ``shape`` provides n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn,
    group_size, rms_eps, rope_theta, act_dtype ('f16'|'bf16'), kv_dtype,
    max_positions.  ``layers[l]`` provides ``attn_norm``/``ffn_norm`` (torch
    tensors in the act dtype) and ``mats[name]`` with ``q`` (uint8 [N, K/2]),
    ``scales`` (float16 [N, K/G]), ``n``, ``k`` — host numpy arrays or device
    torch tensors (``on_device=True``).
    """

    def __init__(self, shape, layers: Sequence, on_device: bool = False, stream=None):
        self.lib = _lib.load()
        self.shape = shape
        cfg = _lib.StageConfig(
            n_layers=shape.n_layers, hidden=shape.hidden, n_q_heads=shape.n_q_heads,
            n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim, ffn=shape.ffn,
            group_size=shape.group_size, rms_eps=shape.rms_eps, act_dtype=_DT[shape.act_dtype],
            kv_dtype=_DT[shape.kv_dtype], rope_theta=shape.rope_theta,
            max_positions=shape.max_positions, rope_cos_sin=None)
        arr = (_lib.LayerWeights * shape.n_layers)()
        keep = []
        for l, lay in enumerate(layers):
            an = lay.attn_norm.contiguous()
            fn = lay.ffn_norm.contiguous()
            if not on_device:
                an, fn = an.cpu(), fn.cpu()
            keep += [an, fn]
            arr[l].attn_norm = an.data_ptr()
            arr[l].ffn_norm = fn.data_ptr()
            for name in MATRIX_NAMES:
                m = lay.mats[name]
                q, s = m.q, m.scales
                if not on_device:
                    q = np.ascontiguousarray(q, dtype=np.uint8)
                    s = np.ascontiguousarray(s).view(np.uint16)
                keep += [q, s]
                setattr(arr[l], name, _lib.QuantMatrix(q=_ptr(q), scales=_ptr(s), n=m.n, k=m.k))
        h = ctypes.c_void_p()
        check(self.lib.stage_create(ctypes.byref(cfg), arr, int(on_device), ctypes.c_void_p(_stream_ptr(stream)),
                                    ctypes.byref(h)))
        self.handle = h
        self.act_dtype = _TORCH[shape.act_dtype]
        self.kv_dtype = _TORCH[shape.kv_dtype]
        _LIVE_STAGES.add(self)

    # ------------------------------------------------------------------
    def close(self) -> None:
        """Free the stage's device memory (its KV states first)."""
        if getattr(self, "handle", None):
            for kv in list(_LIVE_STATES):
                if kv.stage is self:
                    kv.free()
            check(self.lib.stage_destroy(self.handle))
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def weight_bytes(self) -> int:
        return int(self.lib.stage_weight_bytes(self.handle))

    def profile(self, kernel_class: Optional[str]) -> None:
        """Bracket every launch of one kernel class ('qkv', 'attn', 'oproj',
        'gateup', 'down') with hipEvents on the launch stream; None stops."""
        check(self.lib.stage_profile_enable(self.handle, -1 if kernel_class is None else _lib.KERNEL_CLASSES[kernel_class]))

    def profile_read(self):
        """(launches, total_ms) recorded since profile() or the last read."""
        n = ctypes.c_int()
        ms = ctypes.c_double()
        check(self.lib.stage_profile_read(self.handle, ctypes.byref(n), ctypes.byref(ms)))
        return n.value, ms.value

    def profile_read_each(self, capacity: int = 65536) -> np.ndarray:
        """Each recorded launch's duration in ms (launch order) since profile()
        or the last read."""
        out = np.zeros(capacity, np.float32)
        n = ctypes.c_int()
        check(self.lib.stage_profile_read_each(self.handle, ctypes.c_void_p(out.ctypes.data), capacity, ctypes.byref(n)))
        return out[: min(n.value, capacity)].copy()

    def debug_attn_arm(self, layer: int, max_keys: int) -> None:
        """Record `layer`'s rotated queries and visible scores in later forwards
        (per-layer kernels); layer = -1 disarms."""
        check(self.lib.stage_debug_attn_arm(self.handle, layer, max_keys))
        if layer >= 0:
            self._dbg_cap = max(getattr(self, "_dbg_cap", 0), max_keys)   # the library's buffers only grow

    def debug_attn_read(self):
        """(q [M, Hq, D], logits [M, Hq, max_keys]) of the last armed forward;
        keys a row does not see are NaN."""
        sh = self.shape
        q = np.empty(64 * sh.n_q_heads * sh.head_dim, np.float32)
        rows, keys = ctypes.c_int(), ctypes.c_int()
        lg = np.empty(64 * sh.n_q_heads * self._dbg_cap, np.float32)
        check(self.lib.stage_debug_attn_read(self.handle, q.ctypes.data, lg.ctypes.data, ctypes.byref(rows), ctypes.byref(keys)))
        m, k = rows.value, keys.value
        return (q[: m * sh.n_q_heads * sh.head_dim].reshape(m, sh.n_q_heads, sh.head_dim),
                lg[: m * sh.n_q_heads * k].reshape(m, sh.n_q_heads, k))

    def device_status(self) -> None:
        """Wait for the device; raise StageError (STAGE_E_DEVICE) once if a
        single-launch forward of this stage gave up waiting on another
        workgroup or an embedding gather met an id outside its table."""
        check(self.lib.stage_device_status(self.handle))

    def phase_trace(self) -> np.ndarray:
        """[workgroups, layers, 40] device real-time stamps (100 MHz) and exchange
        pass counts of the last single-launch forward (needs STAGE_PS_TRACE=1 at
        creation)."""
        per = 40                                   # entries per workgroup and layer
        n = torch.cuda.get_device_properties(0).multi_processor_count * self.shape.n_layers * per
        out = np.empty(n, dtype=np.uint64)
        nwg = ctypes.c_int()
        check(self.lib.stage_debug_phase_trace(self.handle, out.ctypes.data, n, ctypes.byref(nwg)))
        return out[: nwg.value * self.shape.n_layers * per].reshape(nwg.value, self.shape.n_layers, per)

    def attach_head(self, final_norm: torch.Tensor, lm_head, on_device: bool = False, stream=None) -> None:
        """Final RMSNorm weight [H] (act dtype) and INT4 LM head (``q`` uint8
        [vocab, H/2], ``scales`` float16 [vocab, H/G], ``n``, ``k``)."""
        fn = final_norm.contiguous()
        q, s = lm_head.q, lm_head.scales
        if not on_device:
            fn = fn.cpu()
            q = np.ascontiguousarray(q, dtype=np.uint8)
            s = np.ascontiguousarray(s).view(np.uint16)
        qm = _lib.QuantMatrix(q=_ptr(q), scales=_ptr(s), n=lm_head.n, k=lm_head.k)
        check(self.lib.stage_head_attach(self.handle, ctypes.c_void_p(fn.data_ptr()), ctypes.byref(qm), int(on_device),
                                         ctypes.c_void_p(_stream_ptr(stream))))
        self.vocab = int(lm_head.n)

    def head_top1(self, hidden: torch.Tensor, with_logits: bool = False, stream=None):
        """(token int32 [M], p_max fp32 [M], max logit fp32 [M], logits fp32
        [M, vocab] or None) on the device for the rows of ``hidden``."""
        M = int(hidden.shape[0])
        tok = torch.empty(M, dtype=torch.int32, device=hidden.device)
        p = torch.empty(M, dtype=torch.float32, device=hidden.device)
        lg = torch.empty(M, dtype=torch.float32, device=hidden.device)
        full = torch.empty((M, self.vocab), dtype=torch.float32, device=hidden.device) if with_logits else None
        check(self.lib.stage_head_top1(self.handle, ctypes.c_void_p(hidden.contiguous().data_ptr()), M,
                                       ctypes.c_void_p(tok.data_ptr()), ctypes.c_void_p(p.data_ptr()),
                                       ctypes.c_void_p(lg.data_ptr()),
                                       ctypes.c_void_p(full.data_ptr() if full is not None else None),
                                       ctypes.c_void_p(_stream_ptr(stream))))
        return tok, p, lg, full

    def attach_embedding(self, table: torch.Tensor, on_device: bool = False, stream=None) -> None:
        """Token embedding table [vocab, H] in the act dtype (first-stage role)."""
        t = table.contiguous() if on_device else table.detach().cpu().contiguous()
        if t.dim() != 2 or t.shape[1] != self.shape.hidden or t.element_size() != 2:
            raise ValueError("embedding table must be [vocab, hidden] with 2-byte elements")
        check(self.lib.stage_embed_attach(self.handle, ctypes.c_void_p(t.data_ptr()), int(t.shape[0]), int(on_device),
                                          ctypes.c_void_p(_stream_ptr(stream))))
        self.embed_vocab = int(t.shape[0])

    def embed(self, ids: torch.Tensor, hidden_out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        """Hidden rows [n, H] (device, act dtype) = table[ids] for device int32 ids [n]."""
        if ids.dtype != torch.int32 or not ids.is_cuda:
            raise ValueError("ids must be a device int32 tensor")
        ids = ids.contiguous()
        n = int(ids.numel())
        if hidden_out is None:
            hidden_out = torch.empty((n, self.shape.hidden), dtype=self.act_dtype, device=ids.device)
        check(self.lib.stage_embed(self.handle, ctypes.c_void_p(ids.data_ptr()), n, ctypes.c_void_p(hidden_out.data_ptr()),
                                   ctypes.c_void_p(_stream_ptr(stream))))
        return hidden_out

    def prefill(self, state: "KVState", positions, hidden_in: torch.Tensor, past_mask=None,
                hidden_out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        """Prompt rows hidden_in [n, H] (device, act dtype) of a one-slot state;
        positions [n]; past_mask [P] or None."""
        if hidden_out is None:
            hidden_out = torch.empty_like(hidden_in)
        pos = np.ascontiguousarray(positions, dtype=np.int32).reshape(-1)
        pm = None if past_mask is None else np.ascontiguousarray(past_mask, dtype=np.uint8).reshape(-1)
        check(self.lib.stage_prefill(self.handle, state.handle, int(pos.size), ctypes.c_void_p(pos.ctypes.data),
                                     ctypes.c_void_p(pm.ctypes.data if pm is not None else None),
                                     ctypes.c_void_p(hidden_in.data_ptr()), ctypes.c_void_p(hidden_out.data_ptr()),
                                     ctypes.c_void_p(_stream_ptr(stream))))
        return hidden_out

    def new_state(self, n_slots: int, capacity: int) -> "KVState":
        return KVState(self, n_slots, capacity)

    def debug_dequant(self, layer: int, which: str, row_layout: bool = False) -> np.ndarray:
        """The matrix as the kernels decode it (tiled layout, or the row layout
        of the persistent kernel)."""
        n, k = self.shape.matrix_shapes()[which]
        out = np.empty((n, k), dtype=np.float32)
        code = MATRIX_NAMES.index(which) + (8 if row_layout else 0)
        check(self.lib.stage_debug_dequant(self.handle, layer, code, out.ctypes.data))
        return out

    def forward(self, requests: Sequence["Request"], hidden_in: torch.Tensor,
                hidden_out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        """hidden_in: device [M, H] in the act dtype, rows request-major, then slot, then token."""
        if hidden_out is None:
            hidden_out = torch.empty_like(hidden_in)
        arr = (_lib.StageRequest * len(requests))()
        keep = []
        for i, r in enumerate(requests):
            pos = np.ascontiguousarray(r.positions, dtype=np.int32)
            mask = None if r.mask is None else np.ascontiguousarray(r.mask, dtype=np.uint8)
            rows = None if r.mask_rows is None else np.ascontiguousarray(r.mask_rows, dtype=np.uint8)
            keep += [pos, mask, rows]
            beam = None
            if r.beam_idx is not None:
                beam = np.ascontiguousarray(r.beam_idx, dtype=np.int32)
                keep.append(beam)
            arr[i].state = r.state.handle
            arr[i].n_tokens = int(r.n_tokens)
            arr[i].positions = pos.ctypes.data
            arr[i].beam_idx = beam.ctypes.data if beam is not None else None
            arr[i].attention_mask = mask.ctypes.data if mask is not None else None
            arr[i].attention_mask_rows = rows.ctypes.data if rows is not None else None
            src = mask if mask is not None else rows
            arr[i].mask_len = int(src.shape[-1]) if src is not None and src.ndim else 0
        check(self.lib.stage_forward(self.handle, arr, len(requests), ctypes.c_void_p(hidden_in.data_ptr()),
                                     ctypes.c_void_p(hidden_out.data_ptr()), ctypes.c_void_p(_stream_ptr(stream))))
        return hidden_out


@dataclass
class Request:
    """One request of a forward: positions [S, n] int32, mask [S, P+n] uint8
    (nonzero = visible) or None, beam_idx [S] int32 or None, mask_rows
    [S, n, P+n] uint8 (one key mask per query row) or None."""

    state: "KVState"
    positions: np.ndarray
    mask: Optional[np.ndarray]
    beam_idx: Optional[np.ndarray] = None
    mask_rows: Optional[np.ndarray] = None

    @property
    def n_tokens(self) -> int:
        return int(np.asarray(self.positions).shape[-1])


class KVState:
    def __init__(self, stage: Stage, n_slots: int, capacity: int):
        self.stage = stage
        self.lib = stage.lib
        self.n_slots = n_slots
        self.capacity = capacity
        h = ctypes.c_void_p()
        check(self.lib.kv_state_alloc(stage.handle, n_slots, capacity, ctypes.byref(h)))
        self.handle = h
        _LIVE_STATES.add(self)

    def free(self) -> None:
        if getattr(self, "handle", None):
            check(self.lib.kv_state_free(self.handle))
            self.handle = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass

    @property
    def length(self) -> int:
        n = ctypes.c_int()
        check(self.lib.kv_length(self.handle, ctypes.byref(n)))
        return n.value

    def reset(self) -> None:
        check(self.lib.kv_state_reset(self.handle))

    def truncate(self, new_len: int) -> None:
        check(self.lib.kv_truncate(self.handle, int(new_len)))

    def append(self, k: torch.Tensor, v: torch.Tensor, stream=None) -> None:
        """k, v: [L][S][Hkv][n][D] in the KV dtype (host or device)."""
        k = k.contiguous()
        v = v.contiguous()
        on_dev = int(k.is_cuda)
        check(self.lib.kv_append(self.handle, ctypes.c_void_p(k.data_ptr()), ctypes.c_void_p(v.data_ptr()),
                                 int(k.shape[3]), on_dev, ctypes.c_void_p(_stream_ptr(stream))))

    def _keep(self, keep):
        if keep is None:
            return None, None
        keep = np.ascontiguousarray(keep, dtype=np.uint8)
        if keep.shape != (self.n_slots, self.length):
            raise ValueError(f"keep mask shape {keep.shape} != {(self.n_slots, self.length)}")
        return keep, ctypes.c_void_p(keep.ctypes.data)

    def compact(self, keep=None, stream=None) -> np.ndarray:
        """Remove the rows keep [S, P] (nonzero = keep; None = all) drops, in
        place.  Returns each slot's kept count; P becomes their maximum."""
        keep, kp = self._keep(keep)
        lens = np.zeros(self.n_slots, np.int32)
        check(self.lib.kv_compact(self.handle, kp, ctypes.c_void_p(lens.ctypes.data),
                                  ctypes.c_void_p(_stream_ptr(stream))))
        return lens

    def capture_size(self, keep=None) -> int:
        keep, kp = self._keep(keep)
        n = ctypes.c_int64()
        check(self.lib.kv_capture_size(self.handle, kp, ctypes.byref(n)))
        return n.value

    def capture(self, keep=None, on_device: bool = True, stream=None):
        """Serialized kept rows: a device uint8 tensor, or a host numpy array."""
        keep_arr, kp = self._keep(keep)
        n = self.capture_size(keep_arr)
        if on_device:
            blob = torch.empty(n, dtype=torch.uint8, device="cuda")
            ptr = blob.data_ptr()
        else:
            blob = np.empty(n, dtype=np.uint8)
            ptr = blob.ctypes.data
        check(self.lib.kv_capture(self.handle, kp, ctypes.c_void_p(ptr), n, int(on_device),
                                  ctypes.c_void_p(_stream_ptr(stream))))
        return blob

    def capture_noalloc(self, keep=None, stream=None) -> np.ndarray:
        """kv_capture into a host blob through the library's fixed device
        staging array (no device allocation)."""
        keep_arr, kp = self._keep(keep)
        blob = np.empty(self.capture_size(keep_arr), dtype=np.uint8)
        check(self.lib.kv_capture_noalloc(self.handle, kp, ctypes.c_void_p(blob.ctypes.data), blob.size,
                                          ctypes.c_void_p(_stream_ptr(stream))))
        return blob

    def restore(self, blob, stream=None) -> np.ndarray:
        """Install a captured state (device tensor or host array); returns each
        slot's captured count."""
        lens = np.zeros(self.n_slots, np.int32)
        if isinstance(blob, torch.Tensor) and blob.is_cuda:
            ptr, n, dev = blob.data_ptr(), blob.numel() * blob.element_size(), 1
        else:
            blob = np.ascontiguousarray(blob)
            ptr, n, dev = blob.ctypes.data, blob.nbytes, 0
        check(self.lib.kv_restore(self.handle, ctypes.c_void_p(ptr), int(n), dev, ctypes.c_void_p(lens.ctypes.data),
                                  ctypes.c_void_p(_stream_ptr(stream))))
        return lens

    def read(self, layer: int, slot: int, start: int, count: int, stream=None):
        """Rows [start, start+count) of one layer and slot as the slot sees them: K, V [Hkv, count, D]."""
        sh = self.stage.shape
        k = torch.empty((sh.n_kv_heads, count, sh.head_dim), dtype=self.stage.kv_dtype, device="cuda")
        v = torch.empty_like(k)
        check(self.lib.kv_read(self.handle, layer, slot, start, count, ctypes.c_void_p(k.data_ptr()),
                               ctypes.c_void_p(v.data_ptr()), 1, ctypes.c_void_p(_stream_ptr(stream))))
        return k, v
