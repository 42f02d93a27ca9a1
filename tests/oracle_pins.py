"""Pins of the fp64 oracle against facts fixed outside the oracle itself.

Each ``pin_*`` function raises AssertionError when the oracle disagrees with
the paper or with mathematics: library special cases (torch float64 SDPA,
rms_norm, silu; numpy/torch fp16/bf16 conversion), closed forms (rotary at
p=0, norm preservation, relative-position property, complex-number form,
single-key attention), brute force on tiny inputs (per-element INT4 decode
with a hand-written fp16 decoder, golden layout fixture) and the paper's
exactness claims (mask rewind equals a physical trim; the beam_idx Gather
with identity equals no gather; a permuted beam_idx equals a physically
permuted cache; micro-batched requests are isolated).

``test_oracle_pins.py`` runs them; ``test_oracle_mutations.py`` plants
plausible mistakes in the oracle and checks that some pin catches each one.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import torch
import torch.nn.functional as F

import oracle
import synth
from oracle_cases import f64, logical_positions, oracle_stage, oracle_state

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TINY = synth.TINY
TINY2 = synth.with_layers(synth.TINY, 2)


# ------------------------------------------------------------------ rounding

def pin_round_fp16_matches_numpy():
    r = np.random.default_rng(1)
    x = np.concatenate([
        r.standard_normal(20000).astype(np.float32),
        (r.standard_normal(5000) * 1e-6).astype(np.float32),       # fp16 subnormals
        np.clip(r.standard_normal(5000) * 1e4, -65000, 65000).astype(np.float32),
        np.float32([0.0, -0.0, 1 + 2 ** -11, 1 + 3 * 2 ** -11, 2 ** -25, 3 * 2 ** -25, 65504.0]),
    ]).astype(np.float64)
    ref = x.astype(np.float16).astype(np.float64)
    got = oracle.to_fp16(x)
    assert np.array_equal(got, ref), np.flatnonzero(got != ref)[:10]


def pin_round_bf16_matches_torch():
    r = np.random.default_rng(2)
    x = np.concatenate([
        r.standard_normal(20000).astype(np.float32),
        (r.standard_normal(2000) * 1e-39).astype(np.float32),      # bf16 subnormals
        np.float32([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 0.0]),
    ])
    ref = torch.from_numpy(x).to(torch.bfloat16).double().numpy()
    got = oracle.to_bf16(x.astype(np.float64))
    assert np.array_equal(got, ref), np.flatnonzero(got != ref)[:10]


# ------------------------------------------------------------------ INT4

def _fp16_by_hand(bits: int) -> float:
    s = -1.0 if bits >> 15 else 1.0
    e = (bits >> 10) & 0x1F
    m = bits & 0x3FF
    if e == 0:
        return s * m * 2.0 ** -24
    assert e != 31
    return s * (1.0 + m / 1024.0) * 2.0 ** (e - 15)


def pin_int4_golden_layout():
    with open(os.path.join(GOLDEN, "int4_layout.json")) as f:
        g = json.load(f)
    packed = np.array(g["packed"], dtype=np.uint8)
    scales = np.array(g["scale_bits"], dtype=np.uint16)
    codes = oracle.unpack_int4(packed, g["k"])
    assert codes.tolist() == g["codes"], codes
    w = oracle.dequant(packed, scales, g["k"], g["group"])
    assert w.tolist() == g["weights"], w


def pin_int4_bruteforce():
    """Per-element pure-Python decode (I4) on a ragged-K matrix whose scales
    include fp16 subnormals, zero and large values."""
    r = np.random.default_rng(3)
    n, k, grp = 5, 688, 128
    m = synth.make_quant_matrix(n, k, grp, r)
    bits = m.scales.view(np.uint16).copy()
    bits[0, 0] = 0x0001          # smallest subnormal
    bits[1, 5] = 0x03FF          # largest subnormal (ragged last group)
    bits[2, 2] = 0x0000
    bits[3, 3] = 0x7BFF          # 65504
    bits[4, 1] = 0x8001          # negative subnormal
    scales = bits.view(np.float16)
    got = oracle.dequant(m.q, scales, k, grp)
    assert got.shape == (n, k)
    for row in range(n):
        for col in range(k):
            byte = int(m.q[row, col // 2])
            nib = (byte >> 4) if (col % 2) else (byte & 0xF)
            want = (nib - 8) * _fp16_by_hand(int(bits[row, col // grp]))
            assert got[row, col] == want, (row, col, got[row, col], want)


# ------------------------------------------------------------------ layer pieces vs torch float64

def pin_rmsnorm_matches_torch():
    r = np.random.default_rng(4)
    x = r.standard_normal((3, 256)) * 3
    gam = r.uniform(0.8, 1.2, 256)
    ref = F.rms_norm(torch.from_numpy(x), (256,), weight=torch.from_numpy(gam), eps=1e-5).numpy()
    got = oracle.rmsnorm(x, gam, 1e-5)
    assert np.max(np.abs(got - ref)) <= 1e-12 * np.max(np.abs(ref))


def pin_silu_matches_torch():
    z = np.linspace(-30, 30, 1001)
    ref = F.silu(torch.from_numpy(z)).numpy()
    assert np.max(np.abs(oracle.silu(z) - ref)) <= 1e-14


def _sdpa_reference(q, kc, vc, allowed):
    """torch float64 SDPA with kv heads expanded by repeat_interleave.
    q [n, Hq, D], kc/vc [Hkv, T, D], allowed bool [n, T]."""
    hq, hkv = q.shape[1], kc.shape[0]
    kq = torch.from_numpy(kc).repeat_interleave(hq // hkv, dim=0)      # [Hq, T, D]
    vq = torch.from_numpy(vc).repeat_interleave(hq // hkv, dim=0)
    qt = torch.from_numpy(q).transpose(0, 1)                            # [Hq, n, D]
    m = torch.from_numpy(allowed)[None].expand(hq, -1, -1)
    o = F.scaled_dot_product_attention(qt[None], kq[None], vq[None], attn_mask=m[None])
    return o[0].transpose(0, 1).numpy()


def pin_attention_matches_torch_sdpa():
    r = np.random.default_rng(5)
    hq, hkv, d, past = 4, 2, 64, 40
    for n, holes in ((1, False), (5, False), (5, True)):
        kc = r.standard_normal((hkv, past + n, d))
        vc = r.standard_normal((hkv, past + n, d))
        q = r.standard_normal((n, hq, d))
        mask = np.ones(past + n, dtype=np.uint8)
        if holes:
            mask[r.choice(past, 12, replace=False)] = 0
            mask[past + 2] = 0
        allowed = np.zeros((n, past + n), dtype=bool)
        for i in range(n):
            allowed[i, : past + i + 1] = mask[: past + i + 1] != 0
        got = oracle.attention_slot(q, kc, vc, past, mask)
        ref = _sdpa_reference(q, kc, vc, allowed)
        assert np.max(np.abs(got - ref)) <= 1e-12, (n, holes)


# ------------------------------------------------------------------ rotary closed forms

def pin_rope_closed_forms():
    r = np.random.default_rng(6)
    d, theta = 64, 500000.0
    x = r.standard_normal((7, d))
    assert np.array_equal(oracle.apply_rope(x, np.zeros(7), theta), x)          # p = 0 is the identity
    p = r.integers(0, 8000, 7)
    y = oracle.apply_rope(x, p, theta)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)
    # complex form: (x_i + j x_{i+D/2}) * exp(j p theta^(-2i/D))
    i = np.arange(d // 2)
    z = (x[:, : d // 2] + 1j * x[:, d // 2:]) * np.exp(1j * p[:, None] * theta ** (-2.0 * i / d))
    assert np.max(np.abs(y - np.concatenate([z.real, z.imag], axis=-1))) <= 1e-9
    inv = oracle.rope_inv_freq(d, theta)
    assert inv[0] == 1.0 and abs(inv[-1] - theta ** (-(d - 2) / d)) <= 1e-18


def pin_rope_relative_position():
    """<R(p) q, R(p') k> depends only on p - p'."""
    r = np.random.default_rng(7)
    d, theta = 128, 500000.0
    q, k = r.standard_normal(d), r.standard_normal(d)
    base = np.dot(oracle.apply_rope(q, 100, theta), oracle.apply_rope(k, 37, theta))
    for c in (1, 250, 4000):
        s = np.dot(oracle.apply_rope(q, 100 + c, theta), oracle.apply_rope(k, 37 + c, theta))
        assert abs(s - base) <= 1e-9 * (1 + abs(base))


# ------------------------------------------------------------------ attention closed forms

def pin_single_key_and_own_value():
    r = np.random.default_rng(8)
    hkv, d, past = 2, 64, 10
    kc = r.standard_normal((hkv, past + 1, d))
    vc = r.standard_normal((hkv, past + 1, d))
    q = r.standard_normal((1, 4, d))
    mask = np.zeros(past + 1, dtype=np.uint8)
    mask[3] = 1
    o = oracle.attention_slot(q, kc, vc, past, mask)
    for h in range(4):
        assert np.array_equal(o[0, h], vc[h // 2, 3])
    mask0 = np.ones(1, dtype=np.uint8)                 # P = 0: a token sees only itself
    o0 = oracle.attention_slot(q, kc[:, :1], vc[:, :1], 0, mask0)
    for h in range(4):
        assert np.array_equal(o0[0, h], vc[h // 2, 0])


def pin_zero_weights_identity():
    layers = synth.make_weights(TINY2, 11)
    for lay in layers:
        for name in synth.MATRICES:
            lay.mats[name] = synth.zero_quant_like(lay.mats[name])
    st, _ = oracle_stage(TINY2, layers=layers)
    state = oracle_state(TINY2, 1, 30, 64, 11)
    x = f64(synth.make_hidden(TINY2, 3, 11))
    out = oracle.forward(st, state, x, np.array([[30, 31, 32]]))
    assert np.array_equal(out, x)


def pin_fully_masked_row_rejected():
    st, _ = oracle_stage(TINY)
    state = oracle_state(TINY, 1, 4, 16)
    mask = np.array([[0, 0, 0, 0, 0]], dtype=np.uint8)
    try:
        oracle.forward(st, state, f64(synth.make_hidden(TINY, 1)), np.array([[4]]), None, mask)
    except ValueError:
        return
    raise AssertionError("a query row with no visible key was accepted")


# ------------------------------------------------------------------ paper invariants (bitwise)

def pin_mask_equals_trim():
    """Mask-based rewind == physical trim (paper, "Mask-Based Rewind"), bitwise,
    for the masked verify itself and for the following decode."""
    shape = TINY2
    st, _ = oracle_stage(shape, 21)
    past, n = 72, 5
    r = np.random.default_rng(21)
    holes = np.ones(past, dtype=np.uint8)
    holes[r.choice(past, 9, replace=False)] = 0
    holed = oracle_state(shape, 1, past, 128, 21)
    twin = oracle.trimmed_twin(holed, 0, holes)

    x = f64(synth.make_hidden(shape, n, 21, 1))
    mask = np.concatenate([holes, np.array([1, 1, 1, 0, 0], dtype=np.uint8)])[None]
    pos = logical_positions(holes, n)
    out_m = oracle.forward(st, holed, x, pos, None, mask)
    out_t = oracle.forward(st, twin, x[:3], pos[:, :3], None, None)
    assert np.array_equal(out_m[:3], out_t), np.max(np.abs(out_m[:3] - out_t))

    # next decode: the holed state keeps the two rejected drafts, masked
    mask2 = np.concatenate([mask[0], np.array([1], dtype=np.uint8)])[None]
    pos2 = logical_positions(mask[0], 1)
    x2 = f64(synth.make_hidden(shape, 1, 21, 2))
    out_m2 = oracle.forward(st, holed, x2, pos2, None, mask2)
    out_t2 = oracle.forward(st, twin, x2, pos2, None, None)
    assert np.array_equal(out_m2, out_t2)


def pin_identity_beam_is_no_gather():
    shape = TINY2
    st, _ = oracle_stage(shape, 31)
    a = oracle_state(shape, 3, 20, 40, 31)
    b = a.copy()
    x = f64(synth.make_hidden(shape, 6, 31))
    pos = np.array([[20, 21]] * 3)
    oa = oracle.forward(st, a, x, pos, np.arange(3), None)
    ob = oracle.forward(st, b, x, pos, None, None)
    assert np.array_equal(oa, ob)


def pin_permuted_beam_is_permuted_cache():
    """beam_idx = perm on state A == identity on a state B whose slot rows were
    physically permuted; also for the following forward (the reorder persists)."""
    shape = TINY2
    st, _ = oracle_stage(shape, 41)
    a = oracle_state(shape, 3, 20, 40, 41)
    perm = np.array([2, 0, 2])                      # duplicates allowed, as in a Gather
    b = oracle.OracleState(shape, 3, 40)
    for l in range(shape.n_layers):
        for s in range(3):
            b.K[l][s] = a.K[l][perm[s]]
            b.V[l][s] = a.V[l][perm[s]]
    b.P = a.P
    x = f64(synth.make_hidden(shape, 3, 41))
    pos = np.array([[20], [20], [20]])
    assert np.array_equal(oracle.forward(st, a, x, pos, perm, None), oracle.forward(st, b, x, pos, None, None))
    x2 = f64(synth.make_hidden(shape, 3, 41, 1))
    pos2 = pos + 1
    assert np.array_equal(oracle.forward(st, a, x2, pos2, None, None), oracle.forward(st, b, x2, pos2, None, None))


def pin_verify_is_sequential_decodes():
    shape = TINY2
    st, _ = oracle_stage(shape, 51)
    a = oracle_state(shape, 1, 30, 64, 51)
    b = a.copy()
    x = f64(synth.make_hidden(shape, 4, 51))
    pos = np.arange(30, 34)[None]
    out_v = oracle.forward(st, a, x, pos)
    outs = [oracle.forward(st, b, x[i:i + 1], pos[:, i:i + 1]) for i in range(4)]
    assert np.array_equal(out_v, np.concatenate(outs, axis=0))


def pin_masked_rows_content_independent():
    shape = TINY2
    st, _ = oracle_stage(shape, 61)
    a = oracle_state(shape, 1, 50, 64, 61)
    holes = np.ones(50, dtype=np.uint8)
    holes[[0, 7, 8, 30, 49]] = 0
    b = a.copy()
    for l in range(shape.n_layers):
        idx = np.flatnonzero(holes == 0)
        b.K[l][0][:, idx] = 1e4 * np.sign(np.random.default_rng(l).standard_normal(b.K[l][0][:, idx].shape))
        b.V[l][0][:, idx] = -1e4
    mask = np.concatenate([holes, [1, 1]])[None]
    x = f64(synth.make_hidden(shape, 2, 61))
    pos = logical_positions(holes, 2)
    assert np.array_equal(oracle.forward(st, a, x, pos, None, mask), oracle.forward(st, b, x, pos, None, mask))


def _batch_reqs(shape, seed, pasts, ns):
    reqs = []
    for r_i, (past, n) in enumerate(zip(pasts, ns)):
        state = oracle_state(shape, 1, past, past + 8, seed, stream=r_i)
        holes = synth.hole_mask(past, 0.1, seed, r_i)
        holes[-1] = 1
        mask = np.concatenate([holes, np.ones(n, dtype=np.uint8)])[None]
        reqs.append(dict(state=state, positions=logical_positions(holes, n), beam_idx=None, mask=mask))
    return reqs


def _clone(reqs):
    return [dict(r, state=r["state"].copy()) for r in reqs]


def pin_batch_isolation():
    """A request's rows are the same alone or micro-batched, do not move when a
    batch-mate's input changes, and do move when its own input changes."""
    shape = TINY2
    st, _ = oracle_stage(shape, 71)
    reqs = _batch_reqs(shape, 71, [17, 40, 9], [1, 5, 2])
    rows = sum(np.asarray(r["positions"]).size for r in reqs)
    x = f64(synth.make_hidden(shape, rows, 71))
    full = oracle.forward_batch(st, _clone(reqs), x)
    alone = oracle.forward_batch(st, _clone(reqs[1:2]), x[1:6])
    assert np.array_equal(full[1:6], alone)
    x_mate = x.copy()
    x_mate[0] += 3.0
    x_mate[6:] *= -1
    assert np.array_equal(oracle.forward_batch(st, _clone(reqs), x_mate)[1:6], full[1:6])
    x_own = x.copy()
    x_own[3] += 1.0
    assert np.max(np.abs(oracle.forward_batch(st, _clone(reqs), x_own)[1:6] - full[1:6])) > 1e-3


def pin_request_permutation():
    shape = TINY2
    st, _ = oracle_stage(shape, 81)
    reqs = _batch_reqs(shape, 81, [12, 25], [2, 3])
    x = f64(synth.make_hidden(shape, 5, 81))
    full = oracle.forward_batch(st, _clone(reqs), x)
    swapped = oracle.forward_batch(st, _clone(reqs[::-1]), np.concatenate([x[2:], x[:2]]))
    assert np.array_equal(swapped, np.concatenate([full[2:], full[:2]]))


def pin_gqa_is_repeated_mha():
    """Hkv < Hq equals an MHA stage whose k/v projections and cache rows are
    repeated per q head (head h reads kv head h // (Hq/Hkv))."""
    shape = TINY
    mha = synth.StageShape(**{**shape.__dict__, "name": "tiny-mha", "n_kv_heads": shape.n_q_heads})
    layers = synth.make_weights(shape, 91)
    rep = shape.n_q_heads // shape.n_kv_heads
    d = shape.head_dim
    mha_layers = []
    for lay in layers:
        new = synth.LayerData(attn_norm=lay.attn_norm, ffn_norm=lay.ffn_norm, mats=dict(lay.mats))
        for name in ("wk", "wv"):
            m = lay.mats[name]
            rows = np.concatenate([np.arange(g * d, (g + 1) * d) for g in range(shape.n_kv_heads) for _ in range(rep)])
            new.mats[name] = synth.QuantMatrixData(q=m.q[rows].copy(), scales=m.scales[rows].copy(), n=m.n * rep, k=m.k)
        mha_layers.append(new)
    st_g, _ = oracle_stage(shape, layers=layers)
    st_m, _ = oracle_stage(mha, layers=mha_layers)
    g_state = oracle_state(shape, 1, 25, 40, 91)
    m_state = oracle.OracleState(mha, 1, 40)
    for l in range(shape.n_layers):
        m_state.K[l] = np.repeat(g_state.K[l], rep, axis=1)
        m_state.V[l] = np.repeat(g_state.V[l], rep, axis=1)
    m_state.P = g_state.P
    x = f64(synth.make_hidden(shape, 3, 91))
    pos = np.array([[25, 26, 27]])
    assert np.array_equal(oracle.forward(st_g, g_state, x, pos), oracle.forward(st_m, m_state, x, pos))


# ------------------------------------------------------------------ layer composition vs the HF Llama layer

def _hf_rope(positions, d, theta):
    """(cos, sin) [1, T, D] in float64 in the HF layout (angles repeated over
    both halves), for positions [T]."""
    inv = theta ** (-torch.arange(0, d, 2, dtype=torch.float64) / d)
    fr = torch.as_tensor(positions, dtype=torch.float64)[:, None] * inv[None]
    emb = torch.cat([fr, fr], dim=-1)
    return emb.cos()[None], emb.sin()[None]


def _hf_layers(shape, layers):
    """transformers' LlamaDecoderLayer per stage layer, in float64, holding the
    oracle's dequantized weights and the stage's norm weights."""
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaDecoderLayer

    cfg = LlamaConfig(hidden_size=shape.hidden, intermediate_size=shape.ffn, num_attention_heads=shape.n_q_heads,
                      num_key_value_heads=shape.n_kv_heads, head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps,
                      num_hidden_layers=shape.n_layers, attention_bias=False, mlp_bias=False,
                      rope_theta=shape.rope_theta)
    cfg._attn_implementation = "sdpa"
    out = []
    for l, lay in enumerate(layers):
        m = LlamaDecoderLayer(cfg, l).double()
        g = shape.group_size

        def wt(name):
            q = lay.mats[name]
            return torch.from_numpy(oracle.dequant(q.q, q.scales, q.k, g))

        with torch.no_grad():
            for mod, name in ((m.self_attn.q_proj, "wq"), (m.self_attn.k_proj, "wk"), (m.self_attn.v_proj, "wv"),
                              (m.self_attn.o_proj, "wo"), (m.mlp.gate_proj, "wg"), (m.mlp.up_proj, "wu"),
                              (m.mlp.down_proj, "wd")):
                mod.weight.copy_(wt(name))
            m.input_layernorm.weight.copy_(torch.from_numpy(f64(lay.attn_norm)))
            m.post_attention_layernorm.weight.copy_(torch.from_numpy(f64(lay.ffn_norm)))
        out.append(m)
    return out


def pin_layer_composition_matches_hf_llama():
    """Two decoder layers of the oracle against transformers' LlamaDecoderLayer
    in float64 (the Llama layer the paper's shards trace, "Per-Stage Export
    Pipeline"): a 5-token prefill at P = 0, then 3 tokens over the stored cache
    with one past column and one new-token column masked.  The KV cache keeps
    full precision here (format "f64"), so the two sides differ only by
    rounding: HF's RMSNorm computes in float32 (about 1e-8 relative), far below
    what a wiring mistake (gate/up order, which norm weight goes where, a
    residual tap) moves the output."""
    import dataclasses

    shape = dataclasses.replace(TINY2, name="tiny2-f64kv", kv_dtype="f64")
    layers = synth.make_weights(TINY2, 101)
    st, _ = oracle_stage(shape, layers=layers)
    state = oracle.OracleState(shape, 1, 16)
    x1 = f64(synth.make_hidden(TINY2, 5, 101, 1))
    x2 = f64(synth.make_hidden(TINY2, 3, 101, 2))
    out1 = oracle.forward(st, state, x1, np.arange(5)[None])
    mask2 = np.ones((1, 8), dtype=np.uint8)
    mask2[0, 2] = 0                                    # a rewound past position
    mask2[0, 6] = 0                                    # a rejected draft among the new tokens
    pos2 = logical_positions(mask2[0, :5], 3)
    out2 = oracle.forward(st, state, x2, pos2, None, mask2)

    allowed = np.tril(np.ones((8, 8), dtype=bool))
    allowed[5:] &= mask2[0] != 0
    cos, sin = _hf_rope(np.concatenate([np.arange(5), pos2[0]]), shape.head_dim, shape.rope_theta)
    h = torch.from_numpy(np.concatenate([x1, x2]))[None]
    am = torch.from_numpy(allowed)[None, None]
    with torch.no_grad():
        for m in _hf_layers(shape, layers):
            h = m(h, attention_mask=am, position_embeddings=(cos, sin))
    ref = h[0].numpy()
    got = np.concatenate([out1, out2])
    err = np.max(np.abs(got - ref)) / np.max(np.abs(ref))
    assert err <= 1e-6, err


def pin_stored_rows_closed_form():
    """The cache rows a forward appends are round_kv(rotary(W_k rmsnorm(x)))
    and round_kv(W_v rmsnorm(x)), with rotary after the projection and the
    rounding last; checked with torch's rms_norm, HF's rotate-half rotary and
    torch's fp16 / bf16 conversion, for both KV dtypes."""
    import dataclasses

    from transformers.models.llama.modeling_llama import apply_rotary_pos_emb

    for kv in (synth.F16, synth.BF16):
        shape = dataclasses.replace(TINY, name="tiny-" + kv, kv_dtype=kv)
        layers = synth.make_weights(shape, 111)
        st, _ = oracle_stage(shape, layers=layers)
        state = oracle.OracleState(shape, 1, 8)
        x = f64(synth.make_hidden(shape, 3, 111))
        pos = np.array([7, 300, 4000])
        oracle.forward(st, state, x, pos[None])
        lay = layers[0]
        g = shape.group_size
        wk = torch.from_numpy(oracle.dequant(lay.mats["wk"].q, lay.mats["wk"].scales, lay.mats["wk"].k, g))
        wv = torch.from_numpy(oracle.dequant(lay.mats["wv"].q, lay.mats["wv"].scales, lay.mats["wv"].k, g))
        hn = F.rms_norm(torch.from_numpy(x), (shape.hidden,), weight=torch.from_numpy(f64(lay.attn_norm)),
                        eps=shape.rms_eps)
        d, hkv = shape.head_dim, shape.n_kv_heads
        k = (hn @ wk.T).reshape(3, hkv, d).transpose(0, 1)[None]          # [1, Hkv, 3, D]
        v = (hn @ wv.T).reshape(3, hkv, d).transpose(0, 1)
        cos, sin = _hf_rope(pos, d, shape.rope_theta)
        _, k_rot = apply_rotary_pos_emb(k, k, cos, sin)
        tdt = torch.float16 if kv == synth.F16 else torch.bfloat16
        k_ref = k_rot[0].to(tdt).double().numpy()
        v_ref = v.to(tdt).double().numpy()
        assert np.array_equal(state.K[0][0, :, :3], k_ref), kv
        assert np.array_equal(state.V[0][0, :, :3], v_ref), kv


# ------------------------------------------------------------------ compaction and capture

def _holed_state(shape, seed, S, past, cap, n_holes):
    st = oracle_state(shape, S, past, cap, seed)
    r = np.random.default_rng(seed)
    keep = np.ones((S, past), dtype=np.uint8)
    for b in range(S):
        keep[b, r.choice(past, n_holes[b], replace=False)] = 0
    return st, keep


def pin_compact_bruteforce():
    """Compaction by per-element loops on a tiny state: slot b's kept rows, in
    order, at rows 0..n_b-1, zero rows after, length max_b n_b."""
    shape = TINY2
    st, keep = _holed_state(shape, 71, 3, 12, 16, [3, 0, 7])
    keep[2, :] = 0
    keep[2, [1, 4]] = 1                                   # slot 2 keeps two rows
    out, lens = oracle.compact(st, keep)
    counts = [int(sum(1 for j in range(12) if keep[b][j])) for b in range(3)]
    assert list(lens) == counts == [9, 12, 2] and out.P == 12 and out.capacity == 16
    for l in range(shape.n_layers):
        for b in range(3):
            for g in range(shape.n_kv_heads):
                i = 0
                for j in range(12):
                    if keep[b][j]:
                        for d in range(shape.head_dim):
                            assert out.K[l][b, g, i, d] == st.K[l][b, g, j, d]
                            assert out.V[l][b, g, i, d] == st.V[l][b, g, j, d]
                        i += 1
                for i2 in range(i, out.P):
                    for d in range(shape.head_dim):
                        assert out.K[l][b, g, i2, d] == 0.0 and out.V[l][b, g, i2, d] == 0.0


def pin_compact_keep_all_is_identity():
    shape = TINY2
    st = oracle_state(shape, 2, 9, 12, 72)
    out, lens = oracle.compact(st, None)
    assert out.P == 9 and list(lens) == [9, 9]
    for l in range(shape.n_layers):
        assert np.array_equal(out.K[l][:, :, :9], st.K[l][:, :, :9])
        assert np.array_equal(out.V[l][:, :, :9], st.V[l][:, :, :9])


def pin_compacted_forward_equals_masked_forward():
    """A forward on the compacted state (padding hidden by the mask) equals the
    forward on the holed state with its mask, bitwise (paper, "Mask-Based
    Rewind": masking is exact, compaction only removes what the mask hid), for
    a 3-token verify and the decode after it."""
    shape = TINY2
    st, _ = oracle_stage(shape, 73)
    S, past = 2, 40
    holed, keep = _holed_state(shape, 73, S, past, 64, [6, 13])
    comp, lens = oracle.compact(holed, keep)
    n = 3
    x = f64(synth.make_hidden(shape, S * n, 73, 1))
    pos = logical_positions(keep, n)
    mask_h = np.concatenate([keep, np.ones((S, n), np.uint8)], axis=1)
    mask_c = np.zeros((S, comp.P + n), np.uint8)
    for b in range(S):
        mask_c[b, : lens[b]] = 1
        mask_c[b, comp.P:] = 1
    oh = oracle.forward(st, holed, x, pos, None, mask_h)
    oc = oracle.forward(st, comp, x, pos, None, mask_c)
    assert np.array_equal(oh, oc), np.max(np.abs(oh - oc))
    x2 = f64(synth.make_hidden(shape, S, 73, 2))
    pos2 = pos[:, -1:] + 1
    oh2 = oracle.forward(st, holed, x2, pos2, None, np.concatenate([mask_h, np.ones((S, 1), np.uint8)], 1))
    oc2 = oracle.forward(st, comp, x2, pos2, None, np.concatenate([mask_c, np.ones((S, 1), np.uint8)], 1))
    assert np.array_equal(oh2, oc2)


# ------------------------------------------------------------------ final-stage epilogue

def pin_head_logits_and_top1_against_torch():
    """Logits against torch (rms_norm and a float64 matmul of the hand-decoded
    head), top-1 against torch.softmax / torch.max."""
    shape = TINY
    fn, lm = synth.make_head(shape, 300, 81)
    x = f64(synth.make_hidden(shape, 5, 81))
    got = oracle.head_logits(x, fn, lm.q, lm.scales, 300, shape.group_size, shape.rms_eps)
    codes = np.empty((300, shape.hidden), np.float64)
    codes[:, 0::2] = (lm.q & 0x0F).astype(np.float64) - 8
    codes[:, 1::2] = (lm.q >> 4).astype(np.float64) - 8
    sc = np.repeat(lm.scales.astype(np.float64), shape.group_size, axis=1)[:, : shape.hidden]
    w = torch.from_numpy(codes * sc)
    h = F.rms_norm(torch.from_numpy(x), (shape.hidden,), weight=fn.double(), eps=shape.rms_eps)
    ref = (h @ w.T).numpy()
    assert np.max(np.abs(got - ref)) <= 1e-12 * np.max(np.abs(ref))
    idx, p, mx = oracle.top1(got)
    pt = torch.softmax(torch.from_numpy(got), dim=1)
    vt, it = torch.max(torch.from_numpy(got), dim=1)
    assert np.array_equal(idx, it.numpy()) and np.array_equal(mx, vt.numpy())
    assert np.allclose(p, pt.numpy()[np.arange(5), idx], rtol=1e-13, atol=0)


def pin_top1_bruteforce_and_closed_forms():
    """Pure-Python loops on small rows; equal logits give p = 1/V at index 0;
    ties take the first index; one dominant logit gives p -> 1."""
    r = np.random.default_rng(82)
    lg = r.standard_normal((3, 17)) * 3
    lg[1, 4] = lg[1, 11] = lg[1].max() + 1.0                 # a tie: the first index wins
    idx, p, mx = oracle.top1(lg)
    for m in range(3):
        best, bi = -math.inf, -1
        for j in range(17):
            if lg[m, j] > best:
                best, bi = lg[m, j], j
        tot = 0.0
        for j in range(17):
            tot += math.exp(lg[m, j] - best)
        assert idx[m] == bi and mx[m] == best and abs(p[m] - 1.0 / tot) <= 1e-15
    assert idx[1] == 4
    i2, p2, _ = oracle.top1(np.zeros((1, 40)))
    assert i2[0] == 0 and abs(p2[0] - 1 / 40) <= 1e-16
    i3, p3, _ = oracle.top1(np.array([[0.0, 60.0, -3.0]]))
    assert i3[0] == 1 and 1 - p3[0] < 1e-25


def pin_head_zero_weights():
    """A head whose scales are all zero gives zero logits: token 0, p = 1/V."""
    shape = TINY
    fn, lm = synth.make_head(shape, 64, 83)
    lm.scales[:] = 0
    x = f64(synth.make_hidden(shape, 2, 83))
    lg = oracle.head_logits(x, fn, lm.q, lm.scales, 64, shape.group_size, shape.rms_eps)
    idx, p, mx = oracle.top1(lg)
    assert np.all(lg == 0) and np.all(idx == 0) and np.allclose(p, 1 / 64, rtol=0, atol=1e-16)


def pin_embed_against_torch_and_one_hot():
    """The first stage's lookup: torch's embedding op, and a one-hot matrix
    times the table (exact: one nonzero term per output), on ragged ids with
    repeats and both ends of the vocabulary; an id outside the table is an
    error."""
    shape = TINY
    V = 97
    table = synth.make_embedding(shape, V, 84)
    ids = np.concatenate([[0, V - 1, 5, 5], synth.make_token_ids(V, 9, 84)])
    got = oracle.embed(table.numpy(), ids)
    ref = F.embedding(torch.from_numpy(ids.astype(np.int64)), table).numpy()
    assert got.dtype == ref.dtype and np.array_equal(got.view(np.uint16), ref.view(np.uint16))
    one_hot = np.zeros((ids.size, V))
    one_hot[np.arange(ids.size), ids] = 1.0
    assert np.array_equal(one_hot @ f64(table), got.astype(np.float64))
    for bad in ([V], [-1]):
        try:
            oracle.embed(table.numpy(), bad)
        except IndexError:
            continue
        raise AssertionError(f"id {bad} accepted")


# ------------------------------------------------------------------ per-row (4-D) masks

def tree_case():
    """A draft tree of 6 nodes after one root: parent of node i (-1 = the
    cache), listed so that every node follows its parent, and the mask rows
    that let node i see the cache and its ancestors only."""
    parent = [-1, 0, 0, 1, 1, 2]
    n = len(parent)
    anc = np.zeros((n, n), np.uint8)
    for i in range(n):
        k = i
        while k >= 0:
            anc[i, k] = 1
            k = parent[k]
    depth = anc.sum(axis=1) - 1
    return parent, anc, depth


def pin_row_masks_equal_slot_mask():
    """Rows that all repeat the 2-D mask give the 2-D forward, bitwise."""
    shape = TINY2
    st, _ = oracle_stage(shape, 91)
    a = oracle_state(shape, 2, 30, 64, 91)
    b = a.copy()
    mask = np.ones((2, 34), np.uint8)
    mask[0, [3, 17]] = 0
    mask[1, 31] = 0
    rows = np.repeat(mask[:, None, :], 4, axis=1)
    x = f64(synth.make_hidden(shape, 8, 91))
    pos = np.array([[28, 29, 30, 31], [29, 30, 30, 31]])
    oa = oracle.forward(st, a, x, pos, None, mask)
    ob = oracle.forward(st, b, x, pos, None, None, rows)
    assert np.array_equal(oa, ob)


def pin_tree_verify_equals_paths():
    """A tree of drafts verified in one forward with per-row masks equals each
    root-to-leaf path verified on its own (a linear verify on a copy of the
    cache), bitwise, node by node (paper, "Negative Results": tree-shaped
    speculation needs a per-query mask)."""
    shape = TINY2
    st, _ = oracle_stage(shape, 92)
    past = 25
    base = oracle_state(shape, 1, past, 64, 92)
    parent, anc, depth = tree_case()
    n = len(parent)
    x = f64(synth.make_hidden(shape, n, 92))
    rows = np.ones((1, n, past + n), np.uint8)
    rows[0, :, past:] = anc
    pos = (past + depth)[None]
    tree = oracle.forward(st, base.copy(), x, pos, None, None, rows)
    leaves = [i for i in range(n) if i not in parent]
    for leaf in leaves:
        path = [i for i in range(n) if anc[leaf, i]]           # ancestors in order, ending at the leaf
        lin = oracle.forward(st, base.copy(), x[path], pos[:, path], None, None)
        assert np.array_equal(lin, tree[path]), (leaf, np.max(np.abs(lin - tree[path])))


def pin_packed_sequences_equal_separate():
    """Two sequences packed into one slot behind a shared prefix, each seeing
    the prefix and its own tokens (block-diagonal rows), equal the two run on
    separate copies of the prefix, bitwise (paper, "Continuous Batching on CPU,
    GPU, and NPU": packed slots share a read-only prefix region)."""
    shape = TINY2
    st, _ = oracle_stage(shape, 93)
    past, na, nb = 20, 3, 2
    base = oracle_state(shape, 1, past, 64, 93)
    n = na + nb
    x = f64(synth.make_hidden(shape, n, 93))
    rows = np.zeros((1, n, past + n), np.uint8)
    rows[0, :, :past] = 1
    for i in range(na):
        rows[0, i, past:past + i + 1] = 1
    for i in range(nb):
        rows[0, na + i, past + na:past + na + i + 1] = 1
    pos = np.concatenate([past + np.arange(na), past + np.arange(nb)])[None]
    packed = oracle.forward(st, base.copy(), x, pos, None, None, rows)
    sa = oracle.forward(st, base.copy(), x[:na], pos[:, :na], None, None)
    sb = oracle.forward(st, base.copy(), x[na:], pos[:, na:], None, None)
    assert np.array_equal(packed[:na], sa) and np.array_equal(packed[na:], sb)


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
