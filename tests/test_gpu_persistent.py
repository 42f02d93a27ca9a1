"""The persistent single-launch forward vs the multi-kernel forward and the
fp64 oracle (decode-sized row counts, where the persistent kernel is used)."""
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_cases import TOL_STAGE, Pair, full_mask, host, rel_err, req, run_gpu
from oracle_cases import logical_positions

pytestmark = pytest.mark.gpu


def _pair(shape, seed, persistent, layers=None):
    old = os.environ.get("STAGE_PERSISTENT")
    os.environ["STAGE_PERSISTENT"] = "1" if persistent else "0"
    try:
        return Pair(shape, seed, layers=layers)
    finally:
        if old is None:
            del os.environ["STAGE_PERSISTENT"]
        else:
            os.environ["STAGE_PERSISTENT"] = old


@pytest.mark.parametrize("n_layers", [1, 2])
def test_tiny_decode_persistent_vs_oracle(n_layers):
    shape = synth.with_layers(synth.TINY, n_layers)
    layers = synth.make_weights(shape, 40)
    p = _pair(shape, 40, True, layers)
    m = _pair(shape, 40, False, layers)
    P = 72
    gp, o = p.states(1, P, 128, seed=40)
    gm, _ = m.states(1, P, 128, seed=40, with_oracle=False)
    holes = np.ones(P, np.uint8)
    holes[[3, 10, 11, 70]] = 0
    mask = np.concatenate([holes, [1]])[None]
    pos = logical_positions(holes, 1)
    x = synth.make_hidden(shape, 1, 40, 1)
    out_p = run_gpu(p, [req(gp, pos, mask)], x)
    out_m = run_gpu(m, [req(gm, pos, mask)], x)
    ref = oracle.forward(p.orc, o, host(x), pos, None, mask)
    assert rel_err(out_p, ref) <= TOL_STAGE
    assert rel_err(out_p, out_m) <= TOL_STAGE
    # the appended row is identical in both paths (same rounding of the same k, v)
    for l in range(n_layers):
        kp, vp = gp.read(l, 0, P, 1)
        km, vm = gm.read(l, 0, P, 1)
        assert float((kp.float() - km.float()).abs().max()) <= 2e-2 * float(km.float().abs().max())


def test_tiny_persistent_decode_steps_with_holes():
    """Twelve single-token decodes on one slot through the single-launch path;
    each step's token is kept or rejected at random, so holes accumulate; every
    step vs the oracle, and the final decode vs the physically trimmed twin."""
    shape = synth.with_layers(synth.TINY, 2)
    p = _pair(shape, 41, True)
    r = np.random.default_rng(41)
    P0 = 30
    g, o = p.states(1, P0, 64, seed=41)
    valid = np.ones((1, P0), np.uint8)
    for step in range(12):
        mask = np.concatenate([valid, np.ones((1, 1), np.uint8)], axis=1)
        pos = logical_positions(valid, 1)
        x = synth.make_hidden(shape, 1, 41, step)
        out = run_gpu(p, [req(g, pos, mask, [0])], x)
        ref = oracle.forward(p.orc, o, host(x), pos, np.array([0]), mask)
        assert rel_err(out, ref) <= TOL_STAGE, step
        valid = np.concatenate([valid, (r.random((1, 1)) < 0.7).astype(np.uint8)], axis=1)
    # mask == trim on this path: the oracle's trimmed twin fed to a fresh GPU state
    twin = oracle.trimmed_twin(o, 0, valid[0])
    gt = p.gpu.new_state(1, 64)
    import torch
    L = shape.n_layers
    kt = torch.from_numpy(np.stack([twin.K[l][:, :, : twin.P] for l in range(L)])).to(torch.float16)
    vt = torch.from_numpy(np.stack([twin.V[l][:, :, : twin.P] for l in range(L)])).to(torch.float16)
    gt.append(kt, vt)
    mask = np.concatenate([valid, np.ones((1, 1), np.uint8)], axis=1)
    pos = logical_positions(valid, 1)
    x = synth.make_hidden(shape, 1, 41, 99)
    out_h = run_gpu(p, [req(g, pos, mask)], x)
    out_t = run_gpu(p, [req(gt, pos, full_mask(1, twin.P + 1))], x)
    assert rel_err(out_h, out_t) <= TOL_STAGE


def test_dequant_bitexact_row_layout():
    shape = synth.with_layers(synth.LLAMA8B_HALF, 1)
    layers = synth.make_weights(shape, 42)
    for m in layers[0].mats.values():
        b = m.scales.view(np.uint16)
        b[0, 0], b[1, -1], b[2, 0] = 0x0001, 0x03FF, 0x8001
    p = _pair(shape, 42, True, layers)
    for name in synth.MATRICES:
        mm = layers[0].mats[name]
        ref = oracle.dequant(mm.q, mm.scales, mm.k, shape.group_size)
        got = p.gpu.debug_dequant(0, name, row_layout=True)
        assert np.array_equal(got.astype(np.float64), ref), name


def test_8b_two_layer_decode_persistent():
    shape = synth.with_layers(synth.LLAMA8B_HALF, 2)
    p = _pair(shape, 43, True)
    P = 512
    g, o = p.states(1, P, P + 4, seed=43)
    x = synth.make_hidden(shape, 1, 43)
    pos, mask = np.array([[P]]), full_mask(1, P + 1)
    out = run_gpu(p, [req(g, pos, mask, [0])], x)
    ref = oracle.forward(p.orc, o, host(x), pos, np.array([0]), mask)
    assert rel_err(out, ref) <= TOL_STAGE


def test_exchange_give_up_is_reported():
    """Failure handling of the single launch, forced from the host: with
    STAGE_PS_SPIN_LIMIT=0 (set for this stage only) an exchange wait may poll
    once, so some wait gives up; the launch still ends (every later wait polls
    once), the stage reports STAGE_E_DEVICE once, and a stage with the default
    limit is unaffected."""
    from paper_2608_19147_amd import StageError

    shape = synth.with_layers(synth.TINY, 2)
    layers = synth.make_weights(shape, 44)
    old = os.environ.get("STAGE_PS_SPIN_LIMIT")
    os.environ["STAGE_PS_SPIN_LIMIT"] = "0"
    try:
        bad = _pair(shape, 44, True, layers)
    finally:
        if old is None:
            del os.environ["STAGE_PS_SPIN_LIMIT"]
        else:
            os.environ["STAGE_PS_SPIN_LIMIT"] = old
    good = _pair(shape, 44, True, layers)
    P = 40
    x = synth.make_hidden(shape, 1, 44)
    pos, mask = np.array([[P]]), full_mask(1, P + 1)
    gb, _ = bad.states(1, P, 64, seed=44, with_oracle=False)
    run_gpu(bad, [req(gb, pos, mask, [0])], x)
    with pytest.raises(StageError, match="STAGE_E_DEVICE"):
        bad.gpu.device_status()
    bad.gpu.device_status()                      # reported once, then clear
    gg, o = good.states(1, P, 64, seed=44)
    out = run_gpu(good, [req(gg, pos, mask, [0])], x)
    good.gpu.device_status()
    assert rel_err(out, oracle.forward(good.orc, o, host(x), pos, np.array([0]), mask)) <= TOL_STAGE


def test_cooperative_launch_matches_plain_launch():
    """STAGE_COOP=1 launches the single-launch forward cooperatively (the
    runtime checks co-residency per launch); the kernel and its arithmetic are
    the same, so the output is bitwise that of the plain launch, and both
    match the oracle (8B shape, two layers, KV 512)."""
    shape = synth.with_layers(synth.LLAMA8B_HALF, 2)
    layers = synth.make_weights(shape, 45)
    plain = _pair(shape, 45, True, layers)
    old = os.environ.get("STAGE_COOP")
    os.environ["STAGE_COOP"] = "1"
    try:
        coop = _pair(shape, 45, True, layers)
    finally:
        if old is None:
            del os.environ["STAGE_COOP"]
        else:
            os.environ["STAGE_COOP"] = old
    P = 512
    x = synth.make_hidden(shape, 1, 45)
    pos, mask = np.array([[P]]), full_mask(1, P + 1)
    gp, o = plain.states(1, P, P + 4, seed=45)
    gc, _ = coop.states(1, P, P + 4, seed=45, with_oracle=False)
    out_p = run_gpu(plain, [req(gp, pos, mask, [0])], x)
    out_c = run_gpu(coop, [req(gc, pos, mask, [0])], x)
    coop.gpu.device_status()
    assert np.array_equal(out_p, out_c)
    assert rel_err(out_c, oracle.forward(plain.orc, o, host(x), pos, np.array([0]), mask)) <= TOL_STAGE
