"""Parity at the measured configurations' per-layer shapes and launch
configurations: the 8B half stage (bs=1 decode at KV 2048, speculative verify
on 4 slots x 5 tokens, micro-batches) and the 70B quarter stage (decode at KV
8192, verify at KV 4096).

These use one or two layers of the real per-layer shape, so that several
steps fit a test; the full-depth stages are compared with the oracle in
test_gpu_full_stage.py."""
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_cases import TOL_STAGE, Pair, full_mask, host, rel_err, req, run_gpu
from paper_2608_19147_amd.driver import VerifyDriver

pytestmark = pytest.mark.gpu


def _pair(shape, seed, persistent=True, cache_weights=True, layers=None):
    old = os.environ.get("STAGE_PERSISTENT")
    os.environ["STAGE_PERSISTENT"] = "1" if persistent else "0"
    try:
        return Pair(shape, seed, layers=layers, cache_weights=cache_weights)
    finally:
        if old is None:
            del os.environ["STAGE_PERSISTENT"]
        else:
            os.environ["STAGE_PERSISTENT"] = old


def test_8b_two_layer_decode_kv2048_persistent():
    """Single-launch forward in the benchmark's launch configuration (all CUs,
    KV 2048 split over the attention workgroups) vs the oracle."""
    shape = synth.with_layers(synth.LLAMA8B_HALF, 2)
    p = _pair(shape, 51, cache_weights=False)
    P = 2048
    g, o = p.states(1, P, P + 4, seed=51)
    x = synth.make_hidden(shape, 1, 51)
    pos, mask = np.array([[P]]), full_mask(1, P + 1)
    out = run_gpu(p, [req(g, pos, mask, [0])], x)
    ref = oracle.forward(p.orc, o, host(x), pos, np.array([0]), mask)
    assert rel_err(out, ref) <= TOL_STAGE


def test_8b_decode_long_kv_persistent():
    """Single launch from KV 12000 with 10% masked holes (splits of 375 rows:
    four 16-row chunks per wave in the matrix-core attention, the last one
    partial) vs the oracle; the forward is one stream-kernel launch."""
    shape = synth.with_layers(synth.LLAMA8B_HALF, 2)
    p = _pair(shape, 52, cache_weights=False)
    P = 12000
    g, o = p.states(1, P, P + 4, seed=52)
    holes = synth.hole_mask(P, 0.1, 52, 0)
    holes[-1] = 1
    mask = np.concatenate([holes, np.ones(1, np.uint8)])[None]
    pos = np.array([[int(holes.sum())]])
    x = synth.make_hidden(shape, 1, 52)
    p.gpu.profile("persistent")
    out = run_gpu(p, [req(g, pos, mask, [0])], x)
    launches, _ = p.gpu.profile_read()
    p.gpu.profile(None)
    assert launches == 1
    ref = oracle.forward(p.orc, o, host(x), pos, np.array([0]), mask)
    err = rel_err(out, ref)
    print(f"8B 2 layers, KV {P} with holes, single launch vs oracle: {err:.2e}")
    assert err <= TOL_STAGE


def _layer0_new_kv(shape, layer, x, position):
    """Oracle k and v rows (stored form: k rotated, both rounded to the KV dtype)
    that layer 0 appends for one input row."""
    g = shape.group_size
    h = oracle.rmsnorm(host(x)[0], layer.attn_norm.double().numpy(), shape.rms_eps)
    wk = layer.mats["wk"]
    wv = layer.mats["wv"]
    k = oracle.dequant(wk.q, wk.scales, wk.k, g) @ h
    v = oracle.dequant(wv.q, wv.scales, wv.k, g) @ h
    k = oracle.apply_rope(k.reshape(shape.n_kv_heads, shape.head_dim), np.array([position]), shape.rope_theta)
    rnd = oracle.to_bf16 if shape.kv_dtype == "bf16" else oracle.to_fp16
    return rnd(k), rnd(v.reshape(shape.n_kv_heads, shape.head_dim))


def test_8b_spec_verify_steps():
    """4 cache slots x 5 tokens from KV 2048: acceptances Bernoulli(0.6)
    truncated at the first rejection (the rest stay as masked holes), beam_idx
    identity then a permutation; every step vs the oracle."""
    shape = synth.with_layers(synth.LLAMA8B_HALF, 1)
    p = _pair(shape, 53)
    S, n, P0 = 4, 5, 2048
    g, o = p.states(S, P0, P0 + 3 * n, seed=53)
    drv = VerifyDriver(S, P0)
    for step in range(2):
        beam = np.arange(S, dtype=np.int32) if step % 2 == 0 else synth.beam_permutation(S, 53, step)
        pos, mask, beam = drv.step_inputs(n, beam)
        x = synth.make_hidden(shape, S * n, 53, step)
        out = run_gpu(p, [req(g, pos, mask, beam)], x)
        ref = oracle.forward(p.orc, o, host(x), pos, beam, mask)
        assert rel_err(out, ref) <= TOL_STAGE, step
        drv.accept(synth.acceptance_draws(S, n - 1, 0.6, 53, step))
    assert g.length == P0 + 2 * n


def test_8b_microbatch_mixed():
    """Four requests with KV lengths from U{128..4096} and 10% holes; two
    verify 5 tokens, two decode one; vs the oracle request by request."""
    shape = synth.with_layers(synth.LLAMA8B_HALF, 1)
    p = _pair(shape, 54)
    lens = synth.kv_lengths(4, 128, 4096, 54)
    ns = [5, 1, 5, 1]
    reqs, orq = [], []
    for r, (P, n) in enumerate(zip(lens, ns)):
        P = int(P)
        g, o = p.states(1, P, P + 8, seed=54, stream=r)
        holes = synth.hole_mask(P, 0.1, 54, r)
        holes[-1] = 1
        mask = np.concatenate([holes, np.ones(n, np.uint8)])[None]
        pos = (int(holes.sum()) + np.arange(n))[None]
        reqs.append(req(g, pos, mask))
        orq.append(dict(state=o, positions=pos, mask=mask))
    x = synth.make_hidden(shape, sum(ns), 54)
    out = run_gpu(p, reqs, x)
    ref = oracle.forward_batch(p.orc, orq, host(x))
    assert rel_err(out, ref) <= TOL_STAGE


def test_70b_layer_decode_kv8192_and_verify_kv4096():
    """One layer of the 70B quarter stage: decode at KV 8192, then a 5-token
    verify at KV 4096 whose last two drafts are masked, vs the oracle."""
    shape = synth.with_layers(synth.LLAMA70B_QUARTER, 1)
    p = _pair(shape, 55)
    P = 8192
    g, o = p.states(1, P, P + 4, seed=55)
    x = synth.make_hidden(shape, 1, 55)
    pos, mask = np.array([[P]]), full_mask(1, P + 1)
    out = run_gpu(p, [req(g, pos, mask, [0])], x)
    assert rel_err(out, oracle.forward(p.orc, o, host(x), pos, np.array([0]), mask)) <= TOL_STAGE
    g.free()
    P = 4096
    g, o = p.states(1, P, P + 8, seed=56)
    drv = VerifyDriver(1, P)
    pos, mask, _ = drv.step_inputs(5)
    mask[0, P + 3:] = 0
    x5 = synth.make_hidden(shape, 5, 55, 1)
    out = run_gpu(p, [req(g, pos, mask)], x5)
    assert rel_err(out, oracle.forward(p.orc, o, host(x5), pos, None, mask)) <= TOL_STAGE
