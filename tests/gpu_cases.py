"""Shared helpers of the GPU parity tests: a HIP stage and its oracle twin
built from the same seeded synthetic inputs."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import synth
from paper_2608_19147_amd import Request, Stage

TOL_STAGE = 2e-2          # max-abs-rel of hidden_out vs the fp64 oracle, per stage forward


def rel_err(g, r) -> float:
    g = np.asarray(g, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    return float(np.max(np.abs(g - r)) / np.max(np.abs(r)))


def host(t: torch.Tensor) -> np.ndarray:
    return t.double().cpu().numpy()


class Pair:
    """GPU stage + oracle stage over identical weights."""

    def __init__(self, shape, seed=0, layers=None, cache_weights=True, with_oracle=True):
        self.shape = shape
        self.layers = layers if layers is not None else synth.make_weights(shape, seed)
        self.gpu = Stage(shape, self.layers)
        self.orc = oracle.OracleStage(shape, self.layers, cache_weights) if with_oracle else None

    def close(self) -> None:
        """Free the GPU stage (and every KV state it still holds) now."""
        self.gpu.close()

    def states(self, n_slots, past, capacity, seed=0, stream=0, with_oracle=True):
        g = self.gpu.new_state(n_slots, capacity)
        o = oracle.OracleState(self.shape, n_slots, capacity) if with_oracle else None
        if past:
            k, v = synth.make_kv(self.shape, n_slots, past, seed, stream)
            g.append(k, v)
            if o is not None:
                o.append(k.double().numpy(), v.double().numpy())
        return g, o


def full_mask(S, length):
    return np.ones((S, length), np.uint8)


def run_gpu(pair: Pair, reqs, x: torch.Tensor) -> np.ndarray:
    out = pair.gpu.forward(reqs, x.cuda())
    torch.cuda.synchronize()
    return host(out)


def req(state, positions, mask, beam=None):
    return Request(state, np.asarray(positions, np.int32), np.asarray(mask, np.uint8),
                   None if beam is None else np.asarray(beam, np.int32))
