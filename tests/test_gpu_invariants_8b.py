"""The paper's exactness invariants at the 8B per-layer shape and KV 2048, in
the launch configurations the benchmark uses (16 attention splits per slot
and kv head on the per-layer path, 32 in the single launch), plus long-run
checks of the exchange and reduction machinery.

  * identity beam_idx == no gather, bitwise ("Reaching Monolithic Parity:
    the beam_idx Gather Injection");
  * permuted beam_idx == a physically permuted cache, bitwise, for decode
    and verify rows;
  * masked cache rows filled with +-1e4 garbage leave the output unchanged,
    bitwise ("Mask-Based Rewind": masked keys never enter the softmax), on
    the per-layer path and through the single launch;
  * a holed state equals its physically trimmed twin within the stage
    tolerance, both paths (splits fall at different rows);
  * a forward with the attention record armed gives bitwise the output of an
    unarmed one;
  * 6000 single-launch forwards on one stage (past the wrap of the 16-bit
    residual flags) and 300 multi-row forwards (1200 split-K last-arrival
    reductions per tile) each reproduce the first output bitwise."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_cases import TOL_STAGE, Pair, full_mask, host, rel_err, req, run_gpu
from oracle_cases import logical_positions

pytestmark = pytest.mark.gpu

SHAPE = synth.with_layers(synth.LLAMA8B_HALF, 1)
P = 2048


@pytest.fixture(scope="module")
def p8():
    p = Pair(SHAPE, 90)
    yield p
    p.close()


def _state_from(p, k, v, S, cap):
    g = p.gpu.new_state(S, cap)
    g.append(k, v)
    return g


def test_identity_beam_equals_no_gather_8b(p8):
    S = 4
    k, v = synth.make_kv(SHAPE, S, P, 91)
    a, b = _state_from(p8, k, v, S, P + 8), _state_from(p8, k, v, S, P + 8)
    x = synth.make_hidden(SHAPE, S * 5, 91)
    pos = np.full((S, 5), P) + np.arange(5)
    m = full_mask(S, P + 5)
    assert np.array_equal(run_gpu(p8, [req(a, pos, m, np.arange(S))], x), run_gpu(p8, [req(b, pos, m, None)], x))
    a.free(); b.free()


@pytest.mark.parametrize("n", [1, 5])
def test_permuted_beam_equals_permuted_cache_8b(p8, n):
    S = 4
    perm = np.array([3, 0, 3, 1], np.int32)                 # a duplicate and a dropped slot
    k, v = synth.make_kv(SHAPE, S, P, 92)
    a = _state_from(p8, k, v, S, P + 8)
    b = _state_from(p8, k[:, perm].contiguous(), v[:, perm].contiguous(), S, P + 8)
    x = synth.make_hidden(SHAPE, S * n, 92, n)
    pos = np.full((S, n), P) + np.arange(n)
    m = full_mask(S, P + n)
    m[:, P + n - 1:] = 0 if n > 1 else 1                    # a masked draft on the verify rows
    oa = run_gpu(p8, [req(a, pos, m, perm)], x)
    ob = run_gpu(p8, [req(b, pos, m, None)], x)
    assert np.array_equal(oa, ob)
    for s in range(S):                                       # kv_read through the table: bit-exact rows
        ka, va = a.read(0, s, 0, P)
        assert torch.equal(ka.cpu(), k[0, perm[s]]) and torch.equal(va.cpu(), v[0, perm[s]])
    a.free(); b.free()


@pytest.mark.parametrize("n", [1, 5])
def test_masked_rows_content_independent_8b(p8, n):
    """n = 1 takes the single launch (all 32 splits of the 8B shape), n = 5
    the per-layer kernels."""
    k, v = synth.make_kv(SHAPE, 1, P, 93)
    holes = synth.hole_mask(P, 0.1, 93, 0)
    holes[-1] = 1
    idx = torch.from_numpy(np.flatnonzero(holes == 0))
    k2, v2 = k.clone(), v.clone()
    k2[:, :, :, idx] = 1e4
    v2[:, :, :, idx] = -1e4
    a = _state_from(p8, k, v, 1, P + 8)
    b = _state_from(p8, k2, v2, 1, P + 8)
    mask = np.concatenate([holes, np.ones(n, np.uint8)])[None]
    pos = logical_positions(holes, n)
    x = synth.make_hidden(SHAPE, n, 93, n)
    oa = run_gpu(p8, [req(a, pos, mask)], x)
    ob = run_gpu(p8, [req(b, pos, mask)], x)
    assert np.all(np.isfinite(oa))
    assert np.array_equal(oa, ob)
    a.free(); b.free()


@pytest.mark.parametrize("n", [1, 5])
def test_mask_equals_trim_8b(p8, n):
    """A state with 10% holes and its physically trimmed twin (kept rows only,
    rebuilt through kv_append): same logical positions, outputs within the
    stage tolerance; the holed output also matches the oracle."""
    k, v = synth.make_kv(SHAPE, 1, P, 94)
    holes = synth.hole_mask(P, 0.1, 94, 0)
    holes[-1] = 1
    keep = torch.from_numpy(np.flatnonzero(holes))
    a = _state_from(p8, k, v, 1, P + 8)
    t = _state_from(p8, k[:, :, :, keep].contiguous(), v[:, :, :, keep].contiguous(), 1, P + 8)
    mask = np.concatenate([holes, np.ones(n, np.uint8)])[None]
    pos = logical_positions(holes, n)
    x = synth.make_hidden(SHAPE, n, 94, n)
    oa = run_gpu(p8, [req(a, pos, mask)], x)
    ot = run_gpu(p8, [req(t, pos, full_mask(1, len(keep) + n))], x)
    o = oracle.OracleState(SHAPE, 1, P + 8)
    o.append(k.double().numpy(), v.double().numpy())
    ref = oracle.forward(p8.orc, o, host(x), pos, None, mask)
    e_trim, e_orc = rel_err(oa, ot), rel_err(oa, ref)
    print(f"n={n}: holed vs trimmed {e_trim:.2e}, vs oracle {e_orc:.2e}", flush=True)
    assert e_trim <= TOL_STAGE and e_orc <= TOL_STAGE
    a.free(); t.free()


def test_armed_record_does_not_change_output_8b(p8):
    """Verify 4 x 5 from KV 2048 (per-layer kernels): the forward with layer 0's
    attention record armed equals the unarmed forward bitwise."""
    S, n = 4, 5
    k, v = synth.make_kv(SHAPE, S, P, 95)
    x = synth.make_hidden(SHAPE, S * n, 95)
    pos = np.full((S, n), P) + np.arange(n)
    m = full_mask(S, P + n)
    m[:, P + 3:] = 0
    beam = np.array([1, 0, 3, 2], np.int32)
    a = _state_from(p8, k, v, S, P + 8)
    o1 = run_gpu(p8, [req(a, pos, m, beam)], x)
    a.free()
    p8.gpu.debug_attn_arm(0, P + n)
    try:
        b = _state_from(p8, k, v, S, P + 8)
        o2 = run_gpu(p8, [req(b, pos, m, beam)], x)
        b.free()
    finally:
        p8.gpu.debug_attn_arm(-1, 0)
    assert np.array_equal(o1, o2)


def test_flag_wrap_long_run_single_launch():
    """6000 single-launch forwards of a 2-layer 8B-shaped stage on one Stage
    (the residual exchange keeps 16-bit flag numbers, which advance by 12 per
    launch and wrap after 5462 launches), each from the same state and input:
    every output equals the first bitwise."""
    shape = synth.with_layers(synth.LLAMA8B_HALF, 2)
    p = Pair(shape, 96, with_oracle=False)
    Pk = 512
    g, _ = p.states(1, Pk, Pk + 4, seed=96, with_oracle=False)
    x = synth.make_hidden(shape, 1, 96).cuda()
    pos, mask = np.array([[Pk]], np.int32), full_mask(1, Pk + 1)
    r = req(g, pos, mask)
    first = p.gpu.forward([r], x).clone()
    out = torch.empty_like(first)
    bad = -1
    for i in range(1, 6000):
        g.truncate(Pk)
        p.gpu.forward([r], x, out)
        if i % 500 == 0 or i == 5999:
            torch.cuda.synchronize()
            if not torch.equal(out, first):
                bad = i
                break
            print(f"  {i} launches equal", flush=True)
        elif i > 5400 and not torch.equal(out, first):     # around the wrap: check every launch
            bad = i
            break
    p.gpu.device_status()
    assert bad < 0, f"launch {bad} differs from the first"
    p.close()


def test_splitk_reduction_repeats_bitwise(p8):
    """300 multi-row forwards (verify 4 x 5 from KV 2048): every product's
    split-K partials are summed by the last workgroup to arrive; each output
    must equal the first bitwise."""
    S, n = 4, 5
    g, _ = p8.states(S, P, P + 8, seed=97, with_oracle=False)
    x = synth.make_hidden(SHAPE, S * n, 97).cuda()
    pos = np.full((S, n), P) + np.arange(n)
    r = req(g, pos, full_mask(S, P + n))
    first = p8.gpu.forward([r], x).clone()
    out = torch.empty_like(first)
    for i in range(1, 300):
        g.truncate(P)
        p8.gpu.forward([r], x, out)
        assert torch.equal(out, first), f"forward {i} differs from the first"
    g.free()
