"""The row limit of one forward (STAGE_MAX_ROWS = 64) against the fp64 oracle,
and the attention forms that only long verifies reach: more than 64 query
vectors of one (slot, kv head) take two query tiles per wave, and more than
128 take several passes over the split's keys.  One row beyond the limit is
rejected and leaves the state unchanged."""
import numpy as np
import pytest

import oracle
import synth
from gpu_cases import TOL_STAGE, Pair, host, rel_err, req, run_gpu
from paper_2608_19147_amd import StageError

pytestmark = pytest.mark.gpu

MAX_ROWS = 64


def _long_verify(p, P, n, seed, masked_from):
    """One slot: a cache of P rows with 10% holes, n new tokens, drafts from
    index masked_from masked."""
    g, o = p.states(1, P, P + n + 4, seed=seed)
    holes = synth.hole_mask(P, 0.1, seed, 0)
    holes[-1] = 1
    mask = np.concatenate([holes, np.ones(n, np.uint8)])[None]
    mask[0, P + masked_from:] = 0
    pos = (int(holes.sum()) + np.arange(n))[None]
    x = synth.make_hidden(p.shape, n, seed)
    out = run_gpu(p, [req(g, pos, mask)], x)
    ref = oracle.forward(p.orc, o, host(x), pos, None, mask)
    err = rel_err(out, ref)
    print(f"{p.shape.name}: {n} tokens from KV {P}: {err:.2e}")
    assert err <= TOL_STAGE
    assert g.length == P + n


def test_tiny_64_tokens_one_slot():
    """128 query vectors per kv head: two query tiles per wave."""
    p = Pair(synth.with_layers(synth.TINY, 2), 91)
    _long_verify(p, 40, MAX_ROWS, 91, masked_from=44)


def test_tiny_8_slots_x_8_tokens_beams():
    """64 rows over 8 slots, beam_idx a permutation with one duplicate."""
    shape = synth.with_layers(synth.TINY, 2)
    p = Pair(shape, 92)
    S, P, n = 8, 30, 8
    g, o = p.states(S, P, P + n + 4, seed=92)
    mask = np.ones((S, P + n), np.uint8)
    for b in range(S):
        mask[b, :P] = synth.hole_mask(P, 0.1, 92, b)
        mask[b, P - 1] = 1
    mask[:, P + 6:] = 0
    pos = mask[:, :P].sum(axis=1, keepdims=True) + np.arange(n)[None]
    beam = np.array([3, 0, 1, 2, 7, 7, 5, 4], np.int32)
    x = synth.make_hidden(shape, S * n, 92)
    out = run_gpu(p, [req(g, pos, mask, beam)], x)
    ref = oracle.forward(p.orc, o, host(x), pos, beam, mask)
    assert rel_err(out, ref) <= TOL_STAGE


def test_one_row_over_the_limit_is_rejected():
    shape = synth.TINY
    p = Pair(shape, 93)
    P = 10
    a, _ = p.states(1, P, 128, seed=93, with_oracle=False)
    b, _ = p.states(1, P, 128, seed=93, stream=1, with_oracle=False)
    n_a, n_b = MAX_ROWS, 1
    reqs = [req(a, P + np.arange(n_a)[None], np.ones((1, P + n_a), np.uint8)),
            req(b, P + np.arange(n_b)[None], np.ones((1, P + n_b), np.uint8))]
    x = synth.make_hidden(shape, n_a + n_b, 93).cuda()
    with pytest.raises(StageError, match="STAGE_E_CAPACITY"):
        p.gpu.forward(reqs, x)
    assert a.length == P and b.length == P


def test_8b_layer_64_tokens_kv2048():
    """256 query vectors per kv head: two passes over each split's keys."""
    p = Pair(synth.with_layers(synth.LLAMA8B_HALF, 1), 94)
    _long_verify(p, 2048, MAX_ROWS, 94, masked_from=50)


def test_70b_layer_64_tokens_kv1024():
    """512 query vectors per kv head: four passes over each split's keys."""
    p = Pair(synth.with_layers(synth.LLAMA70B_QUARTER, 1), 95)
    _long_verify(p, 1024, MAX_ROWS, 95, masked_from=60)
