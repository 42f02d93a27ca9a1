"""The forms of the per-layer kernels that the default configuration does not
pick, against the fp64 oracle: the VALU attention (STAGE_ATTN_VECTOR=1), the
matrix-core attention with cache rows staged through registers
(STAGE_ATTN_DMA=0), the one-row product for several rows (STAGE_GEMM_MIN_ROWS
above the row count), and a stage with 64-wide quantization groups, whose
products all take the one-row form.  Each runs a micro-batch of verify and decode requests with
holes and a 5-token verify whose last drafts are masked."""
import dataclasses
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_cases import TOL_STAGE, Pair, full_mask, host, rel_err, req, run_gpu

pytestmark = pytest.mark.gpu

TINY2 = synth.with_layers(synth.TINY, 2)
# the matrix-core products take 128-wide groups; 64-wide ones use the one-row product
TINY_G64 = dataclasses.replace(TINY2, name="tiny-g64", group_size=64)


def _pair(shape, seed, env):
    keys = dict(env, STAGE_PERSISTENT="0")
    old = {k: os.environ.get(k) for k in keys}
    os.environ.update(keys)
    try:
        return Pair(shape, seed)
    finally:
        for k, v in old.items():
            if v is None:
                del os.environ[k]
            else:
                os.environ[k] = v


def _microbatch(p, seed):
    shape = p.shape
    pasts, ns = [17, 40, 9, 63], [1, 5, 2, 5]
    reqs, orq = [], []
    for r, (P, n) in enumerate(zip(pasts, ns)):
        g, o = p.states(1, P, P + 8, seed=seed, stream=r)
        holes = synth.hole_mask(P, 0.1, seed, r)
        holes[-1] = 1
        mask = np.concatenate([holes, np.ones(n, np.uint8)])[None]
        pos = (int(holes.sum()) + np.arange(n))[None]
        reqs.append(req(g, pos, mask))
        orq.append(dict(state=o, positions=pos, mask=mask))
    x = synth.make_hidden(shape, sum(ns), seed)
    out = run_gpu(p, reqs, x)
    ref = oracle.forward_batch(p.orc, orq, host(x))
    assert rel_err(out, ref) <= TOL_STAGE


def _masked_verify(p, seed):
    P = 72
    g, o = p.states(1, P, 128, seed=seed)
    x = synth.make_hidden(p.shape, 5, seed, 1)
    mask = full_mask(1, P + 5)
    mask[0, P + 3:] = 0
    pos = np.arange(P, P + 5)[None]
    out = run_gpu(p, [req(g, pos, mask, [0])], x)
    ref = oracle.forward(p.orc, o, host(x), pos, np.array([0]), mask)
    assert rel_err(out, ref) <= TOL_STAGE


@pytest.mark.parametrize("shape,env", [
    (TINY2, {"STAGE_ATTN_VECTOR": "1"}),
    (TINY2, {"STAGE_GEMM_MIN_ROWS": "65"}),
    (TINY_G64, {}),
    (TINY2, {"STAGE_ATTN_DMA": "0"}),
], ids=["vector-attention", "one-row-products", "group-64", "register-staged-attention"])
def test_alternate_forms_vs_oracle(shape, env):
    p = _pair(shape, 61, env)
    _microbatch(p, 61)
    _masked_verify(p, 62)
