"""Host-side bookkeeping of a speculative-decoding verify loop over one KV state.

The paper's stage never trims its cache when drafts are rejected: rejected rows
stay in place and later forwards ignore them through the attention mask
(Speculative Decoding via Mask-Based KV Rewind, "Mask-Based Rewind"), and beam
reordering gathers through beam_idx (Reaching Monolithic Parity: the beam_idx
Gather Injection).  This driver keeps, per cache slot, which physical rows are
valid, and builds each step's mask, positions and beam_idx:

* the mask covers the P physical rows plus the n new ones; new rows are
  visible (causality among them is applied by the kernels);
* a new token's position is the number of valid past rows plus its index,
  i.e. its index in the equivalent trimmed cache;
* after a step, slot b keeps its first (1 + a_b) new rows, where a_b is the
  number of leading accepted drafts; the rest become holes;
* when beam_idx reorders the slots, the per-slot valid masks are reordered the
  same way before the mask is built.

Only host metadata lives here; every step of the forward runs in the library.
"""
from __future__ import annotations

from typing import Optional

import numpy as np


class VerifyDriver:
    """Valid-row masks of ``n_slots`` cache slots that start with ``past`` valid rows."""

    def __init__(self, n_slots: int, past: int):
        self.n_slots = n_slots
        self.valid = np.ones((n_slots, past), np.uint8)

    @property
    def physical_len(self) -> int:
        return self.valid.shape[1]

    def step_inputs(self, n_new: int, beam_idx: Optional[np.ndarray] = None):
        """(positions [S, n], mask [S, P + n], beam_idx) of the next forward.
        Applies the reorder to the valid masks first (the reorder persists)."""
        if beam_idx is not None:
            beam_idx = np.asarray(beam_idx, np.int32)
            self.valid = self.valid[beam_idx]
        base = self.valid.sum(axis=1).astype(np.int32)
        positions = base[:, None] + np.arange(n_new, dtype=np.int32)[None, :]
        mask = np.concatenate([self.valid, np.ones((self.n_slots, n_new), np.uint8)], axis=1)
        return positions, mask, beam_idx

    def accept(self, drafts_ok: np.ndarray) -> np.ndarray:
        """Record the outcome of the last step: ``drafts_ok`` [S, n - 1] are the
        draft verdicts; slot b keeps the verified token plus the leading run of
        accepted drafts.  Returns the tokens kept per slot (1 + accepted)."""
        drafts_ok = np.asarray(drafts_ok, bool)
        s, k = drafts_ok.shape
        lead = np.argmin(np.concatenate([drafts_ok, np.zeros((s, 1), bool)], axis=1), axis=1)
        keep = (np.arange(k + 1)[None, :] <= lead[:, None]).astype(np.uint8)
        self.valid = np.concatenate([self.valid, keep], axis=1)
        return 1 + lead
