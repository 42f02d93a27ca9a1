"""Shared constructors for oracle-side test cases (CPU only).

Everything random comes from ``synth``; the oracle only computes.
"""
from __future__ import annotations

import numpy as np

import oracle
import synth


def f64(t) -> np.ndarray:
    """torch tensor of the activation/KV dtype -> exact fp64 numpy."""
    return t.double().numpy()


def oracle_stage(shape, seed=0, layers=None):
    layers = layers if layers is not None else synth.make_weights(shape, seed)
    return oracle.OracleStage(shape, layers), layers


def oracle_state(shape, n_slots, past, capacity, seed=0, stream=0):
    st = oracle.OracleState(shape, n_slots, capacity)
    if past:
        k, v = synth.make_kv(shape, n_slots, past, seed, stream)
        st.append(f64(k), f64(v))
    return st


def logical_positions(mask_past: np.ndarray, n: int) -> np.ndarray:
    """Position of new token i = number of visible past rows + i (the index it
    would have in a physically trimmed cache)."""
    mask_past = np.atleast_2d(mask_past)
    base = (mask_past != 0).sum(axis=1)
    return base[:, None] + np.arange(n)[None, :]
