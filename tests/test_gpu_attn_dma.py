"""The attention whose cache rows arrive by direct-to-LDS loads (the default
for items of at most 64 query vectors per kv head) against the register-staged
form (STAGE_ATTN_DMA=0): same splits, steps and arithmetic, so the outputs and
the appended cache rows must be bitwise equal.  Cases: speculative verify on
4 slots x 5 tokens from KV 2048 with 10% masked holes, a masked last draft and
a beam permutation, then a decode step (two 8B layers); a micro-batch of
decode and verify requests of several lengths; a 15-node draft tree with one
key mask per query row; 24 and 64 rows of one slot (two and four query tiles
per wave); a 70B-shaped layer verifying 5 tokens (40 query vectors per kv
head: three tiles); and the tiny shape (head_dim 64).  The oracle checks of the default path run in the other GPU
tests."""
import os

import numpy as np
import pytest
import torch

import synth
from gpu_cases import Pair, full_mask
from paper_2608_19147_amd import Request

pytestmark = pytest.mark.gpu


def _pair(shape, layers, dma):
    keys = {"STAGE_PERSISTENT": "0", "STAGE_ATTN_DMA": "1" if dma else "0"}
    old = {k: os.environ.get(k) for k in keys}
    os.environ.update(keys)
    try:
        return Pair(shape, 0, layers=layers, with_oracle=False)
    finally:
        for k, v in old.items():
            if v is None:
                del os.environ[k]
            else:
                os.environ[k] = v


def _req(state, pos, mask, beam, rows=None):
    return Request(state, np.asarray(pos, np.int32), np.asarray(mask, np.uint8),
                   None if beam is None else np.asarray(beam, np.int32),
                   None if rows is None else np.asarray(rows, np.uint8))


def _bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().view(torch.int16).numpy()


def _run_both(shape, seed, steps):
    """Two stages over the same weights, one per attention form, run the same
    forwards on equal states: outputs and cache rows must be bitwise equal.
    steps["states"]: (slots, past, capacity) per state; steps["forwards"]:
    builders returning ([(state index, positions, mask, beam[, row masks])], rows)."""
    layers = synth.make_weights(shape, seed)
    pa, pb = _pair(shape, layers, True), _pair(shape, layers, False)
    try:
        states_a, states_b = [], []
        for r, (S, past, cap) in enumerate(steps["states"]):
            ga, _ = pa.states(S, past, cap, seed=seed, stream=r, with_oracle=False)
            gb, _ = pb.states(S, past, cap, seed=seed, stream=r, with_oracle=False)
            states_a.append(ga)
            states_b.append(gb)
        for k, fwd in enumerate(steps["forwards"]):
            specs, rows = fwd(states_a)
            x = synth.make_hidden(shape, rows, seed, 100 + k).cuda()
            ra = [_req(states_a[sp[0]], *sp[1:]) for sp in specs]
            rb = [_req(states_b[sp[0]], *sp[1:]) for sp in specs]
            oa = pa.gpu.forward(ra, x)
            ob = pb.gpu.forward(rb, x)
            torch.cuda.synchronize()
            assert np.array_equal(_bits(oa), _bits(ob)), f"forward {k}: hidden_out differs"
        for ga, gb in zip(states_a, states_b):
            assert ga.length == gb.length
            for layer in range(shape.n_layers):
                for slot in range(ga.n_slots):
                    ka, va = ga.read(layer, slot, 0, ga.length)
                    kb, vb = gb.read(layer, slot, 0, gb.length)
                    assert np.array_equal(_bits(ka), _bits(kb)) and np.array_equal(_bits(va), _bits(vb)), \
                        f"cache rows of layer {layer} slot {slot} differ"
    finally:
        pa.close()
        pb.close()


def test_8b_verify_then_decode():
    shape = synth.with_layers(synth.LLAMA8B_HALF, 2)
    S, P, n = 4, 2048, 5
    mask = np.ones((S, P + n), np.uint8)
    for b in range(S):
        mask[b, :P] = synth.hole_mask(P, 0.1, 71, b)
    mask[:, P + 3:] = 0                                     # rejected drafts stay as masked columns
    pos = np.tile(np.arange(P, P + n, dtype=np.int32), (S, 1))
    beam = synth.beam_permutation(S, 71, 1)

    def verify(st):
        return [(0, pos, mask, beam)], S * n

    def decode(st):
        m2 = np.concatenate([mask, np.ones((S, 1), np.uint8)], axis=1)
        return [(0, np.full((S, 1), P + n, np.int32), m2, None)], S

    _run_both(shape, 71, {"states": [(S, P, P + 64)], "forwards": [verify, decode]})


def test_8b_microbatch():
    shape = synth.with_layers(synth.LLAMA8B_HALF, 1)
    pasts, ns = [128, 700, 2047, 3000, 4096, 333], [1, 5, 1, 5, 1, 2]
    spec_states = [(1, P, P + 8) for P in pasts]

    def fwd(st):
        specs = []
        for r, (P, n) in enumerate(zip(pasts, ns)):
            holes = synth.hole_mask(P, 0.1, 72, r)
            holes[-1] = 1
            m = np.concatenate([holes, np.ones(n, np.uint8)])[None]
            specs.append((r, (P + np.arange(n, dtype=np.int32))[None], m, None))
        return specs, sum(ns)

    _run_both(shape, 72, {"states": spec_states, "forwards": [fwd]})


def test_8b_tree_row_masks():
    shape = synth.with_layers(synth.LLAMA8B_HALF, 1)
    P = 2048
    parent = [-1, 0, 0, 1, 1, 2, 2, 3, 3, 4, 4, 5, 5, 6, 6]
    n = len(parent)
    past = synth.hole_mask(P, 0.1, 75, 0)
    rows = np.zeros((1, n, P + n), np.uint8)
    depth = np.zeros(n, np.int32)
    for i in range(n):
        rows[0, i, :P] = past
        k = i
        while k >= 0:
            rows[0, i, P + k] = 1
            k = parent[k]
        depth[i] = 0 if parent[i] < 0 else depth[parent[i]] + 1
    slot_mask = rows.max(axis=1)

    def fwd(st):
        return [(0, (P + depth)[None], slot_mask, None, rows)], n

    _run_both(shape, 75, {"states": [(1, P, P + 32)], "forwards": [fwd]})


@pytest.mark.parametrize("n", [24, 64])
def test_8b_many_query_rows(n):
    """24 rows (96 query vectors per kv head: two tiles per wave) and 64 rows
    (256: four tiles per wave, the prefill chunk's shape), one slot from KV 700
    with holes."""
    shape = synth.with_layers(synth.LLAMA8B_HALF, 1)
    P = 700
    mask = np.ones((1, P + n), np.uint8)
    mask[0, :P] = synth.hole_mask(P, 0.1, 76, n)

    def fwd(st):
        return [(0, np.arange(P, P + n, dtype=np.int32)[None], mask, None)], n

    _run_both(shape, 76, {"states": [(1, P, P + 80)], "forwards": [fwd]})


def test_70b_layer_verify():
    shape = synth.with_layers(synth.LLAMA70B_QUARTER, 1)
    P, n = 4096, 5
    mask = full_mask(1, P + n)
    mask[0, 1000:1100] = 0

    def fwd(st):
        return [(0, np.arange(P, P + n, dtype=np.int32)[None], mask, None)], n

    _run_both(shape, 73, {"states": [(1, P, P + 16)], "forwards": [fwd]})


def test_tiny_head_dim_64():
    shape = synth.with_layers(synth.TINY, 2)
    S, P, n = 3, 150, 4
    mask = np.ones((S, P + n), np.uint8)
    for b in range(S):
        mask[b, :P] = synth.hole_mask(P, 0.2, 74, b)
    pos = np.tile(np.arange(P, P + n, dtype=np.int32), (S, 1))

    def fwd(st):
        return [(0, pos, mask, np.array([2, 0, 1], np.int32))], S * n

    _run_both(shape, 74, {"states": [(S, P, P + 8)], "forwards": [fwd]})
