"""Plain fp64 reference of one pipeline stage's stateful decode/verify forward.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``; never by the product path.  It
shares no code with the HIP library (its own nibble unpack, rounding, rotary
and attention) and takes every random input as an argument.

What it computes (paper, "Per-Stage Export Pipeline", "Stateful KV-Cached
Inference", "Reaching Monolithic Parity: the beam_idx Gather Injection",
"Mask-Based Rewind"): a stage is a contiguous block of Llama decoder layers
(pre-norm attention + SwiGLU FFN, residual stream) with symmetric INT4
group-128 weights, precomputed rotary angles taken at caller-supplied
position ids, and a stateful per-request KV cache.  Each forward:

1. reorders the cache along the slot axis with ``beam_idx`` as a *physical
   copy* (the Gather that the shards insert after every KV ReadValue);
2. per layer: RMSNorm, q/k/v projections, rotary on q and k, appends k and v
   at the next physical cache index, attends over the cache positions that
   the 2-D ``attention_mask`` keeps and that are causally visible, output
   projection + residual, RMSNorm, SwiGLU + residual;
3. returns the hidden states (a middle stage: no embedding, no final norm,
   no LM head) and advances the physical length by the number of new tokens.

Readings where the paper is silent (each listed in the design notes):
rotate-half rotary pairing (i, i + D/2); plain theta, no frequency scaling;
offset-binary nibbles u = q + 8 with the even k in the low nibble; the last
group of a ragged K has its own scale; q-head h reads kv-head
h // (Hq / Hkv); K is cached after rotary and V raw; new k and v are rounded
to the KV dtype before being stored and used ("state-faithful"); a mask byte
of 0 hides that key column only, combined with causality over the physical
index; a query row with no visible key is an error; attention scale
1/sqrt(D).

Every matrix product is row-independent (one matrix-vector product per
activation row, over fixed row blocks of the weight), so a row's result never
depends on its batch-mates; that is what makes the invariant checks bitwise.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence

import numpy as np

__all__ = [
    "round_rne", "to_fp16", "to_bf16", "fp16_bits_to_f64", "unpack_int4", "dequant",
    "rmsnorm", "rope_inv_freq", "apply_rope", "silu", "attention_slot",
    "OracleStage", "OracleState", "forward", "forward_batch", "trimmed_twin", "compact", "head_logits", "top1",
    "embed", "ORACLE_BLOCK_ROWS",
]

# (significand bits including the implicit one, minimum normal exponent)
_FORMATS = {"f16": (11, -14), "bf16": (8, -126)}

ORACLE_BLOCK_ROWS = 1024


# ------------------------------------------------------------------ rounding

def round_rne(x, fmt: str) -> np.ndarray:
    """Round fp64 values to the nearest value of an IEEE-style binary format
    (ties to even), returned as fp64.  Subnormals are kept, not flushed.
    ``"f64"`` keeps the values as they are: a cache stored at full precision,
    which the composition pin uses to compare with an unrounded reference."""
    x = np.asarray(x, dtype=np.float64)
    if fmt == "f64":
        return x.copy()
    sig, emin = _FORMATS[fmt]
    _, e = np.frexp(x)                      # x = m * 2**e with 0.5 <= |m| < 1
    e = np.maximum(e, emin + 1)             # below the normal range the spacing is fixed
    quantum = np.ldexp(np.ones_like(x), e - sig)
    return np.rint(x / quantum) * quantum


def to_fp16(x) -> np.ndarray:
    return round_rne(x, "f16")


def to_bf16(x) -> np.ndarray:
    return round_rne(x, "bf16")


def fp16_bits_to_f64(scales: np.ndarray) -> np.ndarray:
    """fp16 scales (numpy float16 or raw uint16 bits) as exact fp64 values."""
    a = np.asarray(scales)
    if a.dtype == np.uint16:
        a = a.view(np.float16)
    return a.astype(np.float64)


# ------------------------------------------------------------------ INT4 weights
# Paper, "Per-Stage Export Pipeline", Step 4: symmetric INT4, group size 128,
# one scale per group, no zero point.  Stored codes are offset-binary.

def unpack_int4(packed: np.ndarray, k: int) -> np.ndarray:
    """uint8 [N, ceil(K/2)] -> signed codes q in [-8, 7] as int8 [N, K]."""
    packed = np.asarray(packed, dtype=np.uint8)
    n, kb = packed.shape
    u = np.empty((n, 2 * kb), dtype=np.int8)
    u[:, 0::2] = packed & 0x0F      # even k in the low nibble
    u[:, 1::2] = packed >> 4
    return u[:, :k] - np.int8(8)


def dequant(q: np.ndarray, scales: np.ndarray, k: int, group: int) -> np.ndarray:
    """W[n, k] = q[n, k] * s[n, k // G] in fp64 (exact)."""
    codes = unpack_int4(q, k)
    s = fp16_bits_to_f64(scales)
    n = codes.shape[0]
    ng = (k + group - 1) // group
    assert s.shape == (n, ng)
    w = np.zeros((n, ng * group), dtype=np.float64)
    w[:, :k] = codes
    w = w.reshape(n, ng, group)
    w *= s[:, :, None]
    return w.reshape(n, ng * group)[:, :k]


# ------------------------------------------------------------------ layer pieces

def rmsnorm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gamma, per row."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gamma


def rope_inv_freq(head_dim: int, theta: float) -> np.ndarray:
    """theta^(-2i/D) for i < D/2 (plain rotary, no frequency scaling)."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    return theta ** (-(2.0 * i) / head_dim)


def apply_rope(x: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotate the last axis (D) of x [..., D] at the given positions (broadcast
    over the leading axes) with the rotate-half pairing (i, i + D/2)."""
    d = x.shape[-1]
    phi = np.asarray(positions, dtype=np.float64)[..., None] * rope_inv_freq(d, theta)
    c, s = np.cos(phi), np.sin(phi)
    x1, x2 = x[..., : d // 2], x[..., d // 2:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def gemv_rows(h: np.ndarray, w: np.ndarray) -> np.ndarray:
    """out[r] = W @ h[r], one matrix-vector product per row over fixed row
    blocks of W, so that each output depends only on its own input row."""
    h = np.atleast_2d(h)
    out = np.empty((h.shape[0], w.shape[0]), dtype=np.float64)
    for n0 in range(0, w.shape[0], ORACLE_BLOCK_ROWS):
        wb = w[n0:n0 + ORACLE_BLOCK_ROWS]
        for r in range(h.shape[0]):
            out[r, n0:n0 + ORACLE_BLOCK_ROWS] = wb @ h[r]
    return out


def attention_slot(q: np.ndarray, kc: np.ndarray, vc: np.ndarray, past: int,
                   mask: np.ndarray, mask_rows: Optional[np.ndarray] = None) -> np.ndarray:
    """Attention of one cache slot.

    q [n, Hq, D] (rotated), kc/vc [Hkv, >= past+n, D] (the slot's cache rows
    after the new ones were appended), mask [past+n] (nonzero = visible) and
    optionally mask_rows [n, past+n], one key mask per query (paper,
    "Continuous Batching on CPU, GPU, and NPU": the per-query 4-D mask of a
    packed window).  Query i sees key j iff j <= past + i, mask[j] != 0 and
    (with mask_rows) mask_rows[i, j] != 0; hidden keys are skipped, so they
    never enter the max or the sums.
    """
    n, hq, d = q.shape
    hkv = kc.shape[0]
    rep = hq // hkv
    out = np.empty_like(q)
    for i in range(n):
        vis = np.asarray(mask[: past + i + 1]) != 0
        if mask_rows is not None:
            vis = vis & (np.asarray(mask_rows[i, : past + i + 1]) != 0)
        keep = np.flatnonzero(vis)
        if keep.size == 0:
            raise ValueError(f"query row {i} has no visible key")
        for h in range(hq):
            g = h // rep
            kk = kc[g, keep]                              # [A, D]
            vv = vc[g, keep]
            s = (kk * q[i, h]).sum(axis=-1) / math.sqrt(d)
            e = np.exp(s - s.max())
            out[i, h] = (e[:, None] * vv).sum(axis=0) / e.sum()
    return out


# ------------------------------------------------------------------ stage and state

def _as_f64(a) -> np.ndarray:
    """Exact fp64 copy of an fp16/bf16/fp32 array (numpy or torch tensor)."""
    if hasattr(a, "double") and not isinstance(a, np.ndarray):
        return a.double().cpu().numpy()
    return np.asarray(a, dtype=np.float64)


class OracleStage:
    """Stage weights in fp64.  ``layers[l]`` has ``attn_norm`` / ``ffn_norm``
    (values in the activation dtype, any array-like) and ``mats[name]`` with
    ``q``, ``scales``, ``n``, ``k`` for name in wq wk wv wo wg wu wd.

    ``cache_weights=False`` dequantizes each layer when it is used
    (streaming mode) instead of keeping every fp64 matrix resident.
    """

    def __init__(self, shape, layers: Sequence, cache_weights: bool = True):
        self.shape = shape
        self.layers = layers
        self.cache_weights = cache_weights
        self._cache: Dict[int, Dict[str, np.ndarray]] = {}
        assert shape.n_q_heads % shape.n_kv_heads == 0

    def weights(self, l: int) -> Dict[str, np.ndarray]:
        if l in self._cache:
            return self._cache[l]
        lay = self.layers[l]
        w = {name: dequant(m.q, m.scales, m.k, self.shape.group_size) for name, m in lay.mats.items()}
        w["attn_norm"] = _as_f64(lay.attn_norm)
        w["ffn_norm"] = _as_f64(lay.ffn_norm)
        if self.cache_weights:
            self._cache[l] = w
        return w


class OracleState:
    """One request's KV state: K and V per layer, [S, Hkv, capacity, D] fp64
    holding values of the KV dtype, plus the physical length P."""

    def __init__(self, shape, n_slots: int, capacity: int):
        self.shape = shape
        self.n_slots = n_slots
        self.capacity = capacity
        dims = (n_slots, shape.n_kv_heads, capacity, shape.head_dim)
        self.K = [np.zeros(dims) for _ in range(shape.n_layers)]
        self.V = [np.zeros(dims) for _ in range(shape.n_layers)]
        self.P = 0

    def append(self, k, v) -> None:
        """Store already-rotated rows k, v [L][S][Hkv][n][D] at P..P+n-1."""
        k = np.asarray(k, dtype=np.float64)
        v = np.asarray(v, dtype=np.float64)
        n = k.shape[3]
        if self.P + n > self.capacity:
            raise ValueError("capacity exceeded")
        for l in range(self.shape.n_layers):
            self.K[l][:, :, self.P:self.P + n] = k[l]
            self.V[l][:, :, self.P:self.P + n] = v[l]
        self.P += n

    def copy(self) -> "OracleState":
        c = OracleState.__new__(OracleState)
        c.shape, c.n_slots, c.capacity, c.P = self.shape, self.n_slots, self.capacity, self.P
        c.K = [a.copy() for a in self.K]
        c.V = [a.copy() for a in self.V]
        return c

    def rows(self, layer: int, slot: int):
        """The slot's stored K and V rows [Hkv, P, D]."""
        return self.K[layer][slot, :, : self.P], self.V[layer][slot, :, : self.P]


def trimmed_twin(state: OracleState, slot: int, keep: np.ndarray) -> OracleState:
    """A one-slot state holding only the kept rows of ``slot`` (physical trim)."""
    keep_idx = np.flatnonzero(np.asarray(keep[: state.P]) != 0)
    t = OracleState(state.shape, 1, state.capacity)
    for l in range(state.shape.n_layers):
        t.K[l][0, :, : keep_idx.size] = state.K[l][slot][:, keep_idx]
        t.V[l][0, :, : keep_idx.size] = state.V[l][slot][:, keep_idx]
    t.P = int(keep_idx.size)
    return t


def compact(state: OracleState, keep=None):
    """Physical removal of dropped rows from every slot (paper, "Mask-Based
    Rewind": masked positions are compacted away when the state is
    serialized; "Prefix Caching: KV Capture and Warm-Resume": the captured
    state keeps only mask-valid positions).

    keep [S, P] (nonzero = keep; None keeps every row).  Slot b's kept rows,
    in their original order, become its rows 0..n_b-1; the new length is
    max_b n_b and a shorter slot is padded with zero rows.  Returns
    (new state with the same capacity, n_b per slot).  This is also the
    content of a capture blob."""
    S, P = state.n_slots, state.P
    keep = np.ones((S, P), dtype=np.uint8) if keep is None else np.asarray(keep)
    if keep.shape != (S, P):
        raise ValueError(f"keep shape {keep.shape} != {(S, P)}")
    idx = [np.flatnonzero(keep[b] != 0) for b in range(S)]
    lens = np.array([i.size for i in idx], dtype=np.int64)
    out = OracleState(state.shape, S, state.capacity)
    for l in range(state.shape.n_layers):
        for b in range(S):
            out.K[l][b, :, : lens[b]] = state.K[l][b][:, idx[b]]
            out.V[l][b, :, : lens[b]] = state.V[l][b][:, idx[b]]
    out.P = int(lens.max()) if S else 0
    return out, lens


def head_logits(x, final_norm, lm_q, lm_scales, vocab: int, group: int, eps: float) -> np.ndarray:
    """The last stage's logits: RMSNorm of each hidden row with the final norm
    weight, then the dequantized LM head [vocab, H] (paper, "Top-1 Logits
    Compression": the final stage computes the full logits row before
    reducing it).  x [M, H] -> [M, vocab] fp64, one matrix-vector product per row."""
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    h = rmsnorm(x, _as_f64(final_norm), eps)
    w = dequant(lm_q, lm_scales, x.shape[1], group)
    assert w.shape[0] == vocab
    return gemv_rows(h, w)


def top1(logits) -> tuple:
    """Per row: the index of the largest logit (the first one among equal
    maxima), its softmax probability 1 / sum_j exp(l_j - l_max), and the
    maximum.  This is what the paper's top-1 compression sends back instead
    of the full row."""
    logits = np.atleast_2d(np.asarray(logits, dtype=np.float64))
    idx = np.argmax(logits, axis=1)
    mx = logits[np.arange(logits.shape[0]), idx]
    p = 1.0 / np.exp(logits - mx[:, None]).sum(axis=1)
    return idx, p, mx


def embed(table, ids) -> np.ndarray:
    """The first stage's input: row ids[m] of the token embedding table
    [vocab, H] for each m (paper, "Per-Stage Export Pipeline": the first
    shard holds the embedding ahead of its layers).  A lookup, so the rows
    come back unchanged (same dtype, same bits).  An id outside [0, vocab)
    is an error."""
    table = np.asarray(table)
    ids = np.asarray(ids, dtype=np.int64).reshape(-1)
    if ids.size and (ids.min() < 0 or ids.max() >= table.shape[0]):
        raise IndexError("token id outside the embedding table")
    out = np.empty((ids.size, table.shape[1]), dtype=table.dtype)
    for m, t in enumerate(ids):
        out[m] = table[t]
    return out


def forward(stage: OracleStage, state: OracleState, x, positions, beam_idx=None, mask=None,
            mask_rows=None) -> np.ndarray:
    """One stage forward for one request.

    x [S*n, H] (rows slot-major, token-minor; activation-dtype values),
    positions [S, n] integers, beam_idx [S] or None, mask [S, P+n] (None =
    all visible), mask_rows [S, n, P+n] (one key mask per query row) or None.
    Returns hidden_out [S*n, H] fp64 and advances ``state``.
    """
    sh = stage.shape
    positions = np.asarray(positions, dtype=np.int64)
    S, n = positions.shape
    if S != state.n_slots:
        raise ValueError("positions do not match the state's slot count")
    P = state.P
    if P + n > state.capacity:
        raise ValueError("capacity exceeded")
    if mask is None:
        mask = np.ones((S, P + n), dtype=np.uint8)
    mask = np.asarray(mask)
    if mask.shape != (S, P + n):
        raise ValueError(f"mask shape {mask.shape} != {(S, P + n)}")
    if mask_rows is not None:
        mask_rows = np.asarray(mask_rows)
        if mask_rows.shape != (S, n, P + n):
            raise ValueError(f"mask_rows shape {mask_rows.shape} != {(S, n, P + n)}")
    x = np.array(x, dtype=np.float64).reshape(S * n, sh.hidden)

    # Gather(ReadValue, beam_idx, axis=0): a physical reorder of every layer's cache.
    if beam_idx is not None:
        bi = np.asarray(beam_idx, dtype=np.int64)
        if bi.shape != (S,) or bi.min() < 0 or bi.max() >= S:
            raise ValueError("beam_idx out of range")
        for l in range(sh.n_layers):
            state.K[l] = state.K[l][bi].copy()
            state.V[l] = state.V[l][bi].copy()

    D, Hq, Hkv = sh.head_dim, sh.n_q_heads, sh.n_kv_heads
    for l in range(sh.n_layers):
        w = stage.weights(l)
        h = rmsnorm(x, w["attn_norm"], sh.rms_eps)
        q = gemv_rows(h, w["wq"]).reshape(S, n, Hq, D)
        k = gemv_rows(h, w["wk"]).reshape(S, n, Hkv, D)
        v = gemv_rows(h, w["wv"]).reshape(S, n, Hkv, D)
        q = apply_rope(q, positions[:, :, None], sh.rope_theta)
        k = apply_rope(k, positions[:, :, None], sh.rope_theta)
        k = round_rne(k, sh.kv_dtype)
        v = round_rne(v, sh.kv_dtype)
        state.K[l][:, :, P:P + n] = k.transpose(0, 2, 1, 3)
        state.V[l][:, :, P:P + n] = v.transpose(0, 2, 1, 3)
        o = np.empty_like(q)
        for b in range(S):
            o[b] = attention_slot(q[b], state.K[l][b], state.V[l][b], P, mask[b],
                                  None if mask_rows is None else mask_rows[b])
        x = x + gemv_rows(o.reshape(S * n, Hq * D), w["wo"])
        h2 = rmsnorm(x, w["ffn_norm"], sh.rms_eps)
        act = silu(gemv_rows(h2, w["wg"])) * gemv_rows(h2, w["wu"])
        x = x + gemv_rows(act, w["wd"])
    state.P = P + n
    return x


def forward_batch(stage: OracleStage, requests: List[dict], hidden) -> np.ndarray:
    """Several independent requests in one forward (micro-batching, paper
    "Multi-User Throughput via Micro-Batching"): rows are request-major.
    Each request dict has ``state``, ``positions`` [S, n], ``beam_idx``, ``mask``."""
    hidden = np.asarray(hidden, dtype=np.float64)
    outs, r0 = [], 0
    for req in requests:
        S, n = np.asarray(req["positions"]).shape
        rows = hidden[r0:r0 + S * n]
        outs.append(forward(stage, req["state"], rows, req["positions"], req.get("beam_idx"), req.get("mask"),
                            req.get("mask_rows")))
        r0 += S * n
    if r0 != hidden.shape[0]:
        raise ValueError("hidden rows do not match the requests")
    return np.concatenate(outs, axis=0)
