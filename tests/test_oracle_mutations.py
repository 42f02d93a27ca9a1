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

    def attn(q, kc, vc, past, mask):
        n, hq, d = q.shape
        hkv = kc.shape[0]
        rep = hq // hkv
        out = np.empty_like(q)
        for i in range(n):
            lim = past + n if kind == "no_causal" else past + i + 1
            keep = np.flatnonzero(np.asarray(mask[:lim]) != 0)
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
    sig, emin = so._FORMATS[fmt]
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    e = np.maximum(e, emin + 1)
    q = np.ldexp(np.ones_like(x), e - sig)
    return np.trunc(x / q) * q


MUTANTS = {
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
