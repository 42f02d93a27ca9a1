"""kv_capture_noalloc (host blob staged through the library's fixed device
array) gives the same bytes as kv_capture with a host blob, which stages
through an allocated buffer: several calls in a row on one stage, each later
call smaller than the one before (the array keeps the previous call's
contents), one capture that needs two layer slices, and a state whose single
layer exceeds the array (refused before any work)."""
import numpy as np
import pytest
import torch

import synth
from gpu_cases import Pair, req, run_gpu
from oracle_cases import logical_positions
from paper_2608_19147_amd import StageError, _lib

pytestmark = pytest.mark.gpu

TINY = synth.with_layers(synth.TINY, 2)


@pytest.fixture(scope="module")
def tiny():
    p = Pair(TINY, 160, with_oracle=False)
    yield p
    p.close()


def _holed_state(p, S, past, seed):
    g, _ = p.states(S, past, past + 8, seed, with_oracle=False)
    r = np.random.default_rng(seed)
    holes = (r.random((S, past)) >= 0.1).astype(np.uint8)
    holes[:, 0] = 1
    n = 2 if 3 * S > _lib.MAX_ROWS else 3
    mask = np.concatenate([holes, np.ones((S, n), np.uint8)], 1)
    mask[:, -1] = 0                                           # a rejected draft
    perm = r.permutation(S).astype(np.int32)
    x = synth.make_hidden(p.shape, S * n, seed, 1)
    run_gpu(p, [req(g, logical_positions(holes, n), mask, perm)], x)   # leaves a permuted beam table
    return g, mask


def _check(g, keep):
    ref = g.capture(keep, on_device=False)
    got = g.capture_noalloc(keep)
    assert got.size == ref.size and np.array_equal(got, ref)
    return ref.size


def test_noalloc_capture_matches_capture(tiny):
    big, kb = _holed_state(tiny, 32, 3000, 161)
    layer = 2 * 32 * TINY.n_kv_heads * int(kb.sum(axis=1).max()) * TINY.head_dim * 2   # K and V of one layer
    assert layer < _lib.STATIC_SCRATCH_BYTES < 2 * layer          # one layer fits the array, two do not: two slices
    n1 = _check(big, kb)
    mid, km = _holed_state(tiny, 3, 45, 162)
    n2 = _check(mid, km)
    small, ks = _holed_state(tiny, 1, 12, 163)
    n3 = _check(small, ks)
    n4 = _check(small, None)                                   # keep every row
    assert n1 > n2 > n3 and n4 > n3
    for s in (big, mid, small):
        s.free()


def test_noalloc_capture_refuses_oversized_layer(tiny):
    S, P = 64, 4096                                           # one layer: 2 x 64 x 2 x 4096 x 64 x 2 B = 128 MiB
    g = tiny.gpu.new_state(S, P)
    z = torch.zeros((TINY.n_layers, S, TINY.n_kv_heads, P, TINY.head_dim), dtype=torch.float16, device="cuda")
    g.append(z, z)
    with pytest.raises(StageError) as ei:
        g.capture_noalloc(None)
    assert ei.value.code == -3 and "STAGE_STATIC_SCRATCH_BYTES" in str(ei.value)
    # a smaller call afterwards still works
    small, ks = _holed_state(tiny, 2, 20, 164)
    _check(small, ks)
    g.free(); small.free()
