"""Plant plausible mistakes in the oracle (CPU only) and check that at least
one pin catches each of them: the pins are not vacuous."""
import numpy as np
import pytest

import oracle
import oracle.stage_oracle as so
import oracle_pins


def _patch(monkeypatch, name, fn):
    monkeypatch.setattr(so, name, fn)
    monkeypatch.setattr(oracle, name, fn)


def _unpack_swapped(packed, k):
    packed = np.asarray(packed, dtype=np.uint8)
    n, kb = packed.shape
    u = np.empty((n, 2 * kb), dtype=np.int64)
    u[:, 0::2] = packed >> 4
    u[:, 1::2] = packed & 0x0F
    return u[:, :k] - 8


def _rope_sign(x, positions, theta):
    d = x.shape[-1]
    phi = np.asarray(positions, dtype=np.float64)[..., None] * so.rope_inv_freq(d, theta)
    c, s = np.cos(phi), np.sin(phi)
    x1, x2 = x[..., : d // 2], x[..., d // 2:]
    return np.concatenate([x1 * c + x2 * s, x2 * c - x1 * s], axis=-1)


def _rope_interleaved(x, positions, theta):
    d = x.shape[-1]
    phi = np.asarray(positions, dtype=np.float64)[..., None] * so.rope_inv_freq(d, theta)
    c, s = np.cos(phi), np.sin(phi)
    x1, x2 = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = x1 * c - x2 * s
    out[..., 1::2] = x2 * c + x1 * s
    return out


def _rms_no_eps(x, gamma, eps):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) * gamma


def _rms_l2(x, gamma, eps):
    return x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps) * gamma


def _silu_wrong(z):
    return z / (1.0 + np.exp(z))


def _attn_factory(kind):
    orig = so.attention_slot

    def attn(q, kc, vc, past, mask, mask_rows=None):
        n, hq, d = q.shape
        hkv = kc.shape[0]
        rep = hq // hkv
        out = np.empty_like(q)
        for i in range(n):
            lim = past + n if kind == "no_causal" else past + i + 1
            vis = np.asarray(mask[:lim]) != 0
            if mask_rows is not None and kind != "rows_ignored":
                ri = n - 1 - i if kind == "rows_reversed" else i
                vis = vis & (np.asarray(mask_rows[ri, :lim]) != 0)
            keep = np.flatnonzero(vis)
            if kind == "mask_ignored":
                keep = np.arange(lim)
            if keep.size == 0:
                raise ValueError("empty")
            for h in range(hq):
                g = (h % hkv) if kind == "gqa_mod" else h // rep
                kk, vv = kc[g, keep], vc[g, keep]
                scale = 1.0 / d if kind == "scale" else 1.0 / np.sqrt(d)
                s = (kk * q[i, h]).sum(-1) * scale
                e = np.exp(s - s.max())
                out[i, h] = (e[:, None] * vv).sum(0) / e.sum()
        return out
    return attn


def _round_trunc(x, fmt):
    x = np.asarray(x, dtype=np.float64)
    if fmt == "f64":
        return x.copy()
    sig, emin = so._FORMATS[fmt]
    _, e = np.frexp(x)
    e = np.maximum(e, emin + 1)
    q = np.ldexp(np.ones_like(x), e - sig)
    return np.trunc(x / q) * q


def _forward_factory(kind):
    """A copy of the oracle's forward with one wiring mistake in the layer."""

    def fwd(stage, state, x, positions, beam_idx=None, mask=None, mask_rows=None):
        sh = stage.shape
        positions = np.asarray(positions, dtype=np.int64)
        S, n = positions.shape
        P = state.P
        if mask is None:
            mask = np.ones((S, P + n), dtype=np.uint8)
        mask = np.asarray(mask)
        x = np.array(x, dtype=np.float64).reshape(S * n, sh.hidden)
        if beam_idx is not None:
            bi = np.asarray(beam_idx, dtype=np.int64)
            for l in range(sh.n_layers):
                state.K[l] = state.K[l][bi].copy()
                state.V[l] = state.V[l][bi].copy()
        D, Hq, Hkv = sh.head_dim, sh.n_q_heads, sh.n_kv_heads
        for l in range(sh.n_layers):
            w = stage.weights(l)
            n_attn, n_ffn = ("ffn_norm", "attn_norm") if kind == "norm_swap" else ("attn_norm", "ffn_norm")
            h = so.rmsnorm(x, w[n_attn], sh.rms_eps)
            q = so.gemv_rows(h, w["wq"]).reshape(S, n, Hq, D)
            k = so.gemv_rows(h, w["wk"]).reshape(S, n, Hkv, D)
            v = so.gemv_rows(h, w["wv"]).reshape(S, n, Hkv, D)
            q = so.apply_rope(q, positions[:, :, None], sh.rope_theta)
            if kind == "round_before_rope":
                k = so.apply_rope(so.round_rne(k, sh.kv_dtype), positions[:, :, None], sh.rope_theta)
            else:
                k = so.apply_rope(k, positions[:, :, None], sh.rope_theta)
                if kind != "no_kv_round":
                    k = so.round_rne(k, sh.kv_dtype)
            if kind != "no_kv_round":
                v = so.round_rne(v, sh.kv_dtype)
            state.K[l][:, :, P:P + n] = k.transpose(0, 2, 1, 3)
            state.V[l][:, :, P:P + n] = v.transpose(0, 2, 1, 3)
            o = np.empty_like(q)
            for b in range(S):
                o[b] = so.attention_slot(q[b], state.K[l][b], state.V[l][b], P, mask[b],
                                         None if mask_rows is None else mask_rows[b])
            h_attn = x
            x = x + so.gemv_rows(o.reshape(S * n, Hq * D), w["wo"])
            h2 = so.rmsnorm(h_attn if kind == "ffn_norm_on_h" else x, w[n_ffn], sh.rms_eps)
            if kind == "gate_up_swap":
                act = so.silu(so.gemv_rows(h2, w["wu"])) * so.gemv_rows(h2, w["wg"])
            else:
                act = so.silu(so.gemv_rows(h2, w["wg"])) * so.gemv_rows(h2, w["wu"])
            x = x + so.gemv_rows(act, w["wd"])
        state.P = P + n
        return x
    return fwd


def _compact_factory(kind):
    orig = so.compact

    def comp(state, keep=None):
        S, P = state.n_slots, state.P
        keep = np.ones((S, P), np.uint8) if keep is None else np.asarray(keep)
        idx = [np.flatnonzero(keep[b] != 0) for b in range(S)]
        if kind == "reversed":
            idx = [i[::-1] for i in idx]
        lens = np.array([i.size for i in idx])
        out = so.OracleState(state.shape, S, state.capacity)
        for l in range(state.shape.n_layers):
            for b in range(S):
                out.K[l][b, :, : lens[b]] = state.K[l][b][:, idx[b]]
                out.V[l][b, :, : lens[b]] = state.V[l][b][:, idx[b]]
                if kind == "stale_padding":   # padding keeps the old rows instead of zeros
                    out.K[l][b, :, lens[b]:P] = state.K[l][b][:, lens[b]:P]
                    out.V[l][b, :, lens[b]:P] = state.V[l][b][:, lens[b]:P]
        out.P = int(lens.min() if kind == "min_length" else lens.max())
        return out, lens
    return comp


def _top1_last_tie(logits):
    logits = np.atleast_2d(np.asarray(logits, dtype=np.float64))
    idx = logits.shape[1] - 1 - np.argmax(logits[:, ::-1], axis=1)
    mx = logits[np.arange(logits.shape[0]), idx]
    return idx, 1.0 / np.exp(logits - mx[:, None]).sum(axis=1), mx


def _top1_prob_of_first(logits):
    logits = np.atleast_2d(np.asarray(logits, dtype=np.float64))
    idx = np.argmax(logits, axis=1)
    mx = logits[np.arange(logits.shape[0]), idx]
    return idx, np.exp(logits[:, 0] - mx) / np.exp(logits - mx[:, None]).sum(axis=1), mx


def _head_no_norm(x, final_norm, lm_q, lm_scales, vocab, group, eps):
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    return so.gemv_rows(x * so._as_f64(final_norm), so.dequant(lm_q, lm_scales, x.shape[1], group))


def _embed_off_by_one(table, ids):
    table = np.asarray(table)
    return table[np.clip(np.asarray(ids, dtype=np.int64) + 1, 0, table.shape[0] - 1)]


def _embed_column(table, ids):
    table = np.asarray(table)
    return table[:, np.asarray(ids, dtype=np.int64) % table.shape[1]].T


MUTANTS = {
    "embed_off_by_one": ("embed", _embed_off_by_one),
    "embed_column": ("embed", _embed_column),
    "top1_last_tie": ("top1", _top1_last_tie),
    "top1_prob_of_first": ("top1", _top1_prob_of_first),
    "head_no_norm": ("head_logits", _head_no_norm),
    "compact_reversed": ("compact", _compact_factory("reversed")),
    "compact_stale_padding": ("compact", _compact_factory("stale_padding")),
    "compact_min_length": ("compact", _compact_factory("min_length")),
    "gate_up_swap": ("forward", _forward_factory("gate_up_swap")),
    "norm_swap": ("forward", _forward_factory("norm_swap")),
    "round_before_rope": ("forward", _forward_factory("round_before_rope")),
    "no_kv_round": ("forward", _forward_factory("no_kv_round")),
    "ffn_norm_on_h": ("forward", _forward_factory("ffn_norm_on_h")),
    "nibble_order": ("unpack_int4", _unpack_swapped),
    "rope_sign": ("apply_rope", _rope_sign),
    "rope_interleaved": ("apply_rope", _rope_interleaved),
    "rms_no_eps": ("rmsnorm", _rms_no_eps),
    "rms_sum_not_mean": ("rmsnorm", _rms_l2),
    "silu_sign": ("silu", _silu_wrong),
    "attn_no_causal": ("attention_slot", _attn_factory("no_causal")),
    "attn_mask_ignored": ("attention_slot", _attn_factory("mask_ignored")),
    "attn_gqa_mod": ("attention_slot", _attn_factory("gqa_mod")),
    "attn_scale": ("attention_slot", _attn_factory("scale")),
    "attn_rows_ignored": ("attention_slot", _attn_factory("rows_ignored")),
    "attn_rows_reversed": ("attention_slot", _attn_factory("rows_reversed")),
    "round_truncates": ("round_rne", _round_trunc),
}


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_some_pin_catches(monkeypatch, mutant):
    name, fn = MUTANTS[mutant]
    _patch(monkeypatch, name, fn)
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin()
        except (AssertionError, ValueError):
            caught.append(pin.__name__)
    assert caught, f"no pin caught mutant {mutant}"
