"""Full-depth stages at the measured configurations, in the launch
configuration the benchmark times, compared element by element with the fp64
oracle (streaming dequantization, one layer resident at a time):

  * the 16-layer 8B half stage: bs=1 decode at KV 512 and KV 2048 (the
    benchmark's single launch), speculative verify on 4 slots x 5 tokens from
    KV 2048 with a beam permutation, holes and a masked draft, and a mixed
    micro-batch;
  * the 20-layer 70B quarter stage with twenty distinct layers: decode at KV
    8192 and a 5-token verify at KV 4096 with masked drafts.

Each case also checks properties that hold at any depth: the output is
finite and bitwise identical when the same inputs run again on fresh caches;
every cache row that layer 0 appends equals the oracle's row; and, on the 8B
stage, the default kernels agree with the independent vector-unit forms
(one-row products, VALU attention).  The measured error of every comparison
is printed."""
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_cases import TOL_STAGE, host, rel_err, req
from paper_2608_19147_amd import Stage

pytestmark = pytest.mark.gpu

ALT_ENV = {"STAGE_PERSISTENT": "0", "STAGE_ATTN_VECTOR": "1", "STAGE_GEMM_MIN_ROWS": "65"}


def _stage(shape, layers, env):
    old = {k: os.environ.get(k) for k in env}
    os.environ.update(env)
    try:
        return Stage(shape, layers)
    finally:
        for k, v in old.items():
            if v is None:
                del os.environ[k]
            else:
                os.environ[k] = v


def _layer0_rows(shape, layer, x, positions):
    """Oracle k and v rows [rows, Hkv, D] that layer 0 appends, in stored form."""
    g = shape.group_size
    h = oracle.rmsnorm(x, layer.attn_norm.double().numpy(), shape.rms_eps)
    wk, wv = layer.mats["wk"], layer.mats["wv"]
    k = (oracle.dequant(wk.q, wk.scales, wk.k, g) @ h.T).T.reshape(-1, shape.n_kv_heads, shape.head_dim)
    v = (oracle.dequant(wv.q, wv.scales, wv.k, g) @ h.T).T.reshape(-1, shape.n_kv_heads, shape.head_dim)
    k = np.stack([oracle.apply_rope(k[r], np.array([positions[r]]), shape.rope_theta) for r in range(len(k))])
    rnd = oracle.to_bf16 if shape.kv_dtype == "bf16" else oracle.to_fp16
    return rnd(k), rnd(v)


class Case:
    """One request: S slots from a cache of P rows (fraction `holes` of them
    masked), n new tokens per slot, drafts from index `masked_from` masked,
    an optional beam permutation."""

    def __init__(self, shape, S, P, n, seed, stream, holes=0.0, masked_from=None, beam=None):
        self.S, self.P, self.n, self.beam = S, P, n, beam
        self.k, self.v = synth.make_kv(shape, S, P, seed, stream)
        hm = np.stack([synth.hole_mask(P, holes, seed, stream * 8 + b) for b in range(S)]) if holes \
            else np.ones((S, P), np.uint8)
        hm[:, -1] = 1
        self.mask = np.concatenate([hm, np.ones((S, n), np.uint8)], axis=1)
        if masked_from is not None:
            self.mask[:, P + masked_from:] = 0
        self.pos = (hm.sum(axis=1, keepdims=True) + np.arange(n)[None]).astype(np.int32)

    def request(self, st):
        g = st.new_state(self.S, self.P + self.n + 4)
        g.append(self.k, self.v)
        return g, req(g, self.pos, self.mask, self.beam)


def _run(st, cases, x):
    states, reqs = zip(*(c.request(st) for c in cases))
    out = host(st.forward(list(reqs), x))
    torch.cuda.synchronize()
    new = [[g.read(0, b, c.P, c.n) for b in range(c.S)] for g, c in zip(states, cases)]
    for g in states:
        g.free()
    return out, new


def _oracle(shape, layers, cases, xd):
    """The oracle's hidden_out for the whole micro-batch, request by request."""
    orc = oracle.OracleStage(shape, layers, cache_weights=False)
    reqs = []
    for c in cases:
        o = oracle.OracleState(shape, c.S, c.P + c.n)
        o.append(c.k.double().numpy(), c.v.double().numpy())
        reqs.append(dict(state=o, positions=c.pos, beam_idx=c.beam, mask=c.mask))
    return oracle.forward_batch(orc, reqs, xd)


def _check(shape, layers, cases, seed, alt=True):
    rows = sum(c.S * c.n for c in cases)
    x = synth.make_hidden(shape, rows, seed)
    xd = host(x)
    positions = np.concatenate([c.pos.reshape(-1) for c in cases])
    kr, vr = _layer0_rows(shape, layers[0], xd, positions)
    ref = _oracle(shape, layers, cases, xd)
    outs = {}
    for name, env in (("default", {}), ("vector", ALT_ENV))[: 2 if alt else 1]:
        st = _stage(shape, layers, env)
        o1, new = _run(st, cases, x.cuda())
        o2, _ = _run(st, cases, x.cuda())
        st.close()
        assert np.all(np.isfinite(o1)), name
        assert np.array_equal(o1, o2), f"{name}: not deterministic"
        m = 0
        for c, per_slot in zip(cases, new):
            for b, (kn, vn) in enumerate(per_slot):
                for i in range(c.n):
                    ek = rel_err(kn[:, i].double().cpu().numpy(), kr[m])
                    ev = rel_err(vn[:, i].double().cpu().numpy(), vr[m])
                    assert ek <= TOL_STAGE and ev <= TOL_STAGE, (name, m, ek, ev)
                    m += 1
        outs[name] = o1
        err = rel_err(o1, ref)
        print(f"{shape.name} L={shape.n_layers}: {name} kernels vs oracle {err:.2e}", flush=True)
        assert err <= TOL_STAGE, (name, err)
    if alt:
        err = rel_err(outs["default"], outs["vector"])
        print(f"{shape.name}: default vs vector forms {err:.2e}", flush=True)
        assert err <= TOL_STAGE


@pytest.fixture(scope="module")
def layers8b():
    return synth.make_weights(synth.LLAMA8B_HALF, 80)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("P", [512, 2048])
def test_8b_full_stage_decode_vs_oracle(layers8b, P):
    """16 layers, bs=1 decode at KV P through the single launch the benchmark
    times (the default for one row), against the oracle; the per-layer kernels
    and the vector-unit forms as well."""
    shape = synth.LLAMA8B_HALF
    _check(shape, layers8b, [Case(shape, 1, P, 1, 80 + P, 0)], 80 + P)


@pytest.mark.timeout(600)
def test_8b_full_stage_spec_verify_4x5(layers8b):
    """16 layers; 4 slots x 5 tokens from KV 2048, 10% holes, the last draft
    masked, beam_idx a permutation."""
    shape = synth.LLAMA8B_HALF
    beam = synth.beam_permutation(4, 81, 1).astype(np.int32)
    _check(shape, layers8b, [Case(shape, 4, 2048, 5, 81, 0, holes=0.1, masked_from=4, beam=beam)], 81)


@pytest.mark.timeout(600)
def test_8b_full_stage_microbatch_mixed(layers8b):
    """16 layers; four requests with KV lengths from U{128..4096} and 10%
    holes, two verifying 5 tokens (last two masked) and two decoding one."""
    shape = synth.LLAMA8B_HALF
    lens = synth.kv_lengths(4, 128, 4096, 82)
    cases = [Case(shape, 1, int(P), n, 82, r, holes=0.1, masked_from=3 if n > 1 else None)
             for r, (P, n) in enumerate(zip(lens, [5, 1, 5, 1]))]
    _check(shape, layers8b, cases, 82)


@pytest.fixture(scope="module")
def layers70b():
    """Twenty distinct synthetic 70B layers (about 8.8 GB of packed weights)."""
    return synth.make_weights(synth.LLAMA70B_QUARTER, 83)


@pytest.mark.timeout(900)
def test_70b_full_stage_decode_kv8192(layers70b):
    shape = synth.LLAMA70B_QUARTER
    _check(shape, layers70b, [Case(shape, 1, 8192, 1, 83, 0)], 83, alt=False)


@pytest.mark.timeout(900)
def test_70b_full_stage_verify_kv4096(layers70b):
    """5-token verify at KV 4096 with the last two drafts masked."""
    shape = synth.LLAMA70B_QUARTER
    _check(shape, layers70b, [Case(shape, 1, 4096, 5, 84, 0, masked_from=3)], 84, alt=False)
