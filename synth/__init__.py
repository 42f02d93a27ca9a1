"""Seeded synthetic inputs for the stage forward.

This module produces every input that both the HIP library and the fp64
oracle consume: quantized weights in the canonical packed layout, norm
weights, KV-cache contents, hidden states and the random draws of the
multi-step drivers (draft acceptances, beam permutations, mask holes, KV
lengths).  It holds none of the method's arithmetic; values are rounded to
fp16/bf16 with library conversions (numpy / torch) only.

Shapes follow the paper's workloads: a Llama-3.1-8B half stage (16 of 32
layers, the 16+16 two-stage split of the distributed experiments), a
Llama-3-70B quarter stage (20 layers, the 4-stage 70B deployment) and a tiny
one-layer stage.  Trained weights are not available, so weights are uniform
INT4 codes with |N(0, 0.02)|/7 fp16 group scales (synthetic stand-ins).

Streams are derived from ``numpy.random.SeedSequence([seed, config_id, a, b])``
so that every tensor is reproducible on its own.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Tuple

import numpy as np
import torch

F16 = "f16"
BF16 = "bf16"

_TORCH_DT = {F16: torch.float16, BF16: torch.bfloat16}


@dataclass(frozen=True)
class StageShape:
    """Dimensions of one pipeline stage (a contiguous block of decoder layers)."""

    name: str
    config_id: int
    n_layers: int
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    group_size: int = 128
    rms_eps: float = 1e-5
    rope_theta: float = 500000.0
    act_dtype: str = BF16
    kv_dtype: str = BF16
    max_positions: int = 16384

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def matrix_shapes(self) -> Dict[str, Tuple[int, int]]:
        """(N, K) of every linear layer: out = x @ W.T with W [N, K]."""
        H, F = self.hidden, self.ffn
        return {
            "wq": (self.q_dim, H),
            "wk": (self.kv_dim, H),
            "wv": (self.kv_dim, H),
            "wo": (H, self.q_dim),
            "wg": (F, H),
            "wu": (F, H),
            "wd": (H, F),
        }

    def weight_bytes(self) -> int:
        """Packed INT4 + fp16 scale + norm-weight bytes of the whole stage."""
        tot = 0
        for n, k in self.matrix_shapes().values():
            tot += n * ((k + 1) // 2) + n * ((k + self.group_size - 1) // self.group_size) * 2
        tot += 2 * self.hidden * 2
        return tot * self.n_layers

    def kv_bytes_per_token(self) -> int:
        """K and V bytes of one cache row across all layers and KV heads."""
        return self.n_layers * 2 * self.n_kv_heads * self.head_dim * 2


MATRICES = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")

TINY = StageShape("tiny", 0, n_layers=1, hidden=256, n_q_heads=4, n_kv_heads=2,
                  head_dim=64, ffn=688, act_dtype=F16, kv_dtype=F16, max_positions=4096)
LLAMA8B_HALF = StageShape("llama3.1-8b-half", 1, n_layers=16, hidden=4096, n_q_heads=32,
                          n_kv_heads=8, head_dim=128, ffn=14336)
LLAMA70B_QUARTER = StageShape("llama3-70b-quarter", 4, n_layers=20, hidden=8192, n_q_heads=64,
                              n_kv_heads=8, head_dim=128, ffn=28672)

SHAPES = {s.name: s for s in (TINY, LLAMA8B_HALF, LLAMA70B_QUARTER)}


def with_layers(shape: StageShape, n_layers: int) -> StageShape:
    """Same per-layer shape with a different layer count (for oracle-sized parity runs)."""
    d = dict(shape.__dict__)
    d["n_layers"] = n_layers
    d["name"] = f"{shape.name}-L{n_layers}"
    return StageShape(**d)


def rng(seed: int, config_id: int, a: int, b: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, config_id, a, b]))


def round_to(values: np.ndarray, dtype: str) -> torch.Tensor:
    """Round float values to the storage dtype with torch's conversion (RNE)."""
    return torch.from_numpy(np.ascontiguousarray(values, dtype=np.float32)).to(_TORCH_DT[dtype])


@dataclass
class QuantMatrixData:
    """One INT4 matrix in the canonical layout.

    ``q``: uint8 [N, ceil(K/2)], offset-binary nibbles u = q + 8, the low
    nibble holds the even k.  ``scales``: float16 [N, ceil(K/G)].
    """

    q: np.ndarray
    scales: np.ndarray
    n: int
    k: int


@dataclass
class LayerData:
    attn_norm: torch.Tensor
    ffn_norm: torch.Tensor
    mats: Dict[str, QuantMatrixData] = field(default_factory=dict)


def make_quant_matrix(n: int, k: int, g: int, r: np.random.Generator) -> QuantMatrixData:
    kb = (k + 1) // 2
    q = np.frombuffer(r.bytes(n * kb), dtype=np.uint8).reshape(n, kb).copy()
    ng = (k + g - 1) // g
    scales = (np.abs(r.standard_normal((n, ng), dtype=np.float32)) * np.float32(0.02 / 7)).astype(np.float16)
    return QuantMatrixData(q=q, scales=scales, n=n, k=k)


def make_layer(shape: StageShape, layer: int, seed: int = 0) -> LayerData:
    base = 1000 * layer
    r = rng(seed, shape.config_id, base + 1)
    an = round_to(r.uniform(0.8, 1.2, shape.hidden), shape.act_dtype)
    r = rng(seed, shape.config_id, base + 2)
    fn = round_to(r.uniform(0.8, 1.2, shape.hidden), shape.act_dtype)
    ld = LayerData(attn_norm=an, ffn_norm=fn)
    for t, name in enumerate(MATRICES):
        n, k = shape.matrix_shapes()[name]
        ld.mats[name] = make_quant_matrix(n, k, shape.group_size, rng(seed, shape.config_id, base + 10 + t))
    return ld


def make_weights(shape: StageShape, seed: int = 0) -> List[LayerData]:
    return [make_layer(shape, l, seed) for l in range(shape.n_layers)]


LLAMA3_VOCAB = 128256


def make_head(shape: StageShape, vocab: int, seed: int = 0) -> Tuple[torch.Tensor, QuantMatrixData]:
    """The final stage's RMSNorm weight [H] (act dtype, U(0.8, 1.2)) and INT4
    LM head [vocab, H] (same recipe as the layer matrices)."""
    r = rng(seed, shape.config_id, 900_001)
    fn = round_to(r.uniform(0.8, 1.2, shape.hidden), shape.act_dtype)
    return fn, make_quant_matrix(vocab, shape.hidden, shape.group_size, rng(seed, shape.config_id, 900_002))


def make_embedding(shape: StageShape, vocab: int, seed: int = 0) -> torch.Tensor:
    """The first stage's token embedding table [vocab, H] in the activation
    dtype, ~N(0, 0.02^2) (the usual initialisation scale of Llama tables),
    drawn in blocks of 8192 rows so a full vocabulary does not need one huge
    float32 temporary."""
    out = torch.empty((vocab, shape.hidden), dtype=_TORCH_DT[shape.act_dtype])
    for b0 in range(0, vocab, 8192):
        rows = min(8192, vocab - b0)
        r = rng(seed, shape.config_id, 900_010, b0 // 8192)
        out[b0:b0 + rows] = round_to(r.standard_normal((rows, shape.hidden), dtype=np.float32) * np.float32(0.02),
                                     shape.act_dtype)
    return out


def make_token_ids(vocab: int, n: int, seed: int = 0, step: int = 0) -> np.ndarray:
    """n token ids, uniform over [0, vocab), int32."""
    return rng(seed, 4, 900_020, step).integers(0, vocab, n, dtype=np.int32)


def make_kv(shape: StageShape, n_slots: int, n_tokens: int, seed: int = 0, stream: int = 0) -> Tuple[torch.Tensor, torch.Tensor]:
    """Already-stored cache rows ~N(0,1): K and V [L][S][Hkv][n][D] in the KV dtype."""
    dims = (shape.n_layers, n_slots, shape.n_kv_heads, n_tokens, shape.head_dim)
    r = rng(seed, shape.config_id, 500_001, stream)
    k = round_to(r.standard_normal(dims, dtype=np.float32), shape.kv_dtype)
    v = round_to(r.standard_normal(dims, dtype=np.float32), shape.kv_dtype)
    return k, v


def make_hidden(shape: StageShape, rows: int, seed: int = 0, step: int = 0) -> torch.Tensor:
    """Stage input hidden states ~N(0,1) [rows, H] in the activation dtype."""
    r = rng(seed, shape.config_id, 600_001, step)
    return round_to(r.standard_normal((rows, shape.hidden), dtype=np.float32), shape.act_dtype)


def zero_quant_like(m: QuantMatrixData) -> QuantMatrixData:
    """An all-zero matrix: every code is u = 8 (q = 0), scales arbitrary."""
    return QuantMatrixData(q=np.full_like(m.q, 0x88), scales=m.scales.copy(), n=m.n, k=m.k)


# ---------------------------------------------------------------- driver draws

def acceptance_draws(n_slots: int, k_drafts: int, p: float, seed: int, step: int, config_id: int = 2) -> np.ndarray:
    """Bernoulli(p) draft outcomes [S, K]; the caller truncates at the first failure."""
    r = rng(seed, config_id, 700_001, step)
    return r.random((n_slots, k_drafts)) < p


def beam_permutation(n_slots: int, seed: int, step: int, config_id: int = 2) -> np.ndarray:
    r = rng(seed, config_id, 700_002, step)
    return r.permutation(n_slots).astype(np.int32)


def hole_mask(length: int, frac: float, seed: int, req: int, config_id: int = 3) -> np.ndarray:
    """i.i.d. Bernoulli(frac) holes over ``length`` past positions: uint8, 1 = keep."""
    r = rng(seed, config_id, 700_003, req)
    return (r.random(length) >= frac).astype(np.uint8)


def kv_lengths(n_req: int, lo: int, hi: int, seed: int, config_id: int = 3) -> np.ndarray:
    r = rng(seed, config_id, 700_004, n_req)
    return r.integers(lo, hi + 1, size=n_req).astype(np.int64)
