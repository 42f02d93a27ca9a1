"""Prefill against the oracle (paper, "Stateful KV-Cached Inference": the
prompt goes through the stage in one pass that fills the cache; "NPU Stages:
Static, Stateless Shards": long prompts in fixed-size chunks).

The oracle runs the whole prompt as one forward (causal over the prompt rows,
the past rows its mask keeps); stage_prefill runs it in chunks of 64 rows,
layer-major.  Checked: hidden_out, every cache row the prefill appends (every
layer), a decode after the prefill, chunk boundaries (64, 65 rows), a prompt
after existing rows with masked holes, agreement with the same prompt fed
through stage_forward chunk by chunk, an 8B-shaped layer, and the errors."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_cases import TOL_STAGE, Pair, full_mask, host, rel_err, req, run_gpu
from paper_2608_19147_amd import StageError

pytestmark = pytest.mark.gpu

TINY2 = synth.with_layers(synth.TINY, 2)


@pytest.fixture(scope="module")
def tiny():
    p = Pair(TINY2, 210)
    yield p
    p.close()


def _check_rows(g, o, shape, P0, n):
    """Rows P0 .. P0+n of every layer: the GPU's against the oracle's."""
    worst = 0.0
    for l in range(shape.n_layers):
        k, v = g.read(l, 0, P0, n)
        worst = max(worst, rel_err(host(k), o.K[l][0][:, P0:P0 + n]), rel_err(host(v), o.V[l][0][:, P0:P0 + n]))
    return worst


def _prefill_case(p, P0, n, seed, holes=0.0):
    g, o = p.states(1, P0, P0 + n + 8, seed)
    past = np.ones(P0, np.uint8)
    if holes and P0:
        past = synth.hole_mask(P0, holes, seed, 0)
        past[0] = 1
    x = synth.make_hidden(p.shape, n, seed, 1)
    pos = int(past.sum()) + np.arange(n)
    out = p.gpu.prefill(g, pos, x.cuda(), past if holes else None)
    torch.cuda.synchronize()
    mask = np.concatenate([past, np.ones(n, np.uint8)])[None]
    ref = oracle.forward(p.orc, o, host(x), pos[None], None, mask)
    assert g.length == P0 + n
    return g, o, host(out), ref, mask


@pytest.mark.parametrize("P0,n", [(0, 150), (0, 64), (0, 65), (40, 1), (40, 100)])
def test_prefill_tiny(tiny, P0, n):
    g, o, out, ref, _ = _prefill_case(tiny, P0, n, 211 + n)
    e = rel_err(out, ref)
    er = _check_rows(g, o, TINY2, P0, n)
    print(f"tiny prefill P0={P0} n={n}: hidden {e:.2e}, appended rows {er:.2e}")
    assert e <= TOL_STAGE and er <= TOL_STAGE
    g.free()


def test_prefill_with_holes_then_decode(tiny):
    P0, n = 60, 130
    g, o, out, ref, mask = _prefill_case(tiny, P0, n, 220, holes=0.15)
    e = rel_err(out, ref)
    assert e <= TOL_STAGE
    # decode after the prompt: the holes stay masked
    x = synth.make_hidden(TINY2, 1, 221)
    m2 = np.concatenate([mask[0], [1]])[None].astype(np.uint8)
    pos = np.array([[int(m2[0, :-1].sum())]])
    og = run_gpu(tiny, [req(g, pos, m2)], x)
    oo = oracle.forward(tiny.orc, o, host(x), pos, None, m2)
    e2 = rel_err(og, oo)
    print(f"prefill with holes: hidden {e:.2e}; decode after it {e2:.2e}")
    assert e2 <= TOL_STAGE
    g.free()


def test_prefill_matches_chunked_forward(tiny):
    """The same prompt through stage_forward, 64 rows per call."""
    P0, n = 20, 150
    ga, _ = tiny.states(1, P0, P0 + n + 8, 230, with_oracle=False)
    gb, _ = tiny.states(1, P0, P0 + n + 8, 230, with_oracle=False)
    x = synth.make_hidden(TINY2, n, 230, 1)
    pos = P0 + np.arange(n)
    a = host(tiny.gpu.prefill(ga, pos, x.cuda()))
    outs = []
    for r0 in range(0, n, 64):
        m = min(64, n - r0)
        outs.append(run_gpu(tiny, [req(gb, pos[None, r0:r0 + m], full_mask(1, P0 + r0 + m))], x[r0:r0 + m]))
    b = np.concatenate(outs)
    e = rel_err(a, b)
    print(f"prefill vs chunked stage_forward: {e:.2e}")
    assert e <= TOL_STAGE
    for l in range(TINY2.n_layers):
        ka, va = ga.read(l, 0, 0, P0 + n)
        kb, vb = gb.read(l, 0, 0, P0 + n)
        assert rel_err(host(ka), host(kb)) <= TOL_STAGE and rel_err(host(va), host(vb)) <= TOL_STAGE
    ga.free(); gb.free()


def test_prefill_8b_layer():
    p = Pair(synth.with_layers(synth.LLAMA8B_HALF, 1), 240)
    g, o, out, ref, _ = _prefill_case(p, 256, 70, 240)
    e = rel_err(out, ref)
    er = _check_rows(g, o, p.shape, 256, 70)
    print(f"8B layer prefill P0=256 n=70: hidden {e:.2e}, appended rows {er:.2e}")
    assert e <= TOL_STAGE and er <= TOL_STAGE
    g.free()
    p.close()


def test_prefill_errors(tiny):
    g2, _ = tiny.states(2, 4, 32, 250, with_oracle=False)
    x = synth.make_hidden(TINY2, 10, 250).cuda()
    with pytest.raises(StageError) as ei:
        tiny.gpu.prefill(g2, np.arange(10), x)              # two slots
    assert ei.value.code == -2
    g1, _ = tiny.states(1, 4, 12, 251, with_oracle=False)
    with pytest.raises(StageError) as ei:
        tiny.gpu.prefill(g1, np.arange(10), x)              # 4 + 10 > capacity 12
    assert ei.value.code == -3 and g1.length == 4
    with pytest.raises(StageError) as ei:
        tiny.gpu.prefill(g1, np.arange(8), x[:8], hidden_out=x[4:12])   # overlapping output
    assert ei.value.code == -1 and g1.length == 4
    g1.free(); g2.free()
