"""Per-query-row (4-D) attention masks against the oracle (paper, "Continuous
Batching on CPU, GPU, and NPU": a packed window whose mask rows open a shared
prefix and each sequence's own tokens; "Negative Results": tree-shaped
speculation needs a per-query mask).

  * rows that repeat the 2-D mask give bitwise the 2-D forward (tiny, and an
    8B layer at 4 slots x 5 tokens from KV 2048 with 16 splits per slot);
  * a draft tree verified in one forward matches the oracle, and each
    root-to-leaf path verified on its own within the stage tolerance;
  * two sequences packed behind a shared prefix match the oracle;
  * a request with row masks beside one without leaves the latter bitwise
    unchanged; the vector-unit attention; a single decode row with a row
    mask (the single launch) equals its 2-D form bitwise;
  * a query row that sees no key is refused."""
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_cases import TOL_STAGE, Pair, full_mask, host, rel_err, run_gpu
from oracle_pins import tree_case
from paper_2608_19147_amd import Request, StageError

pytestmark = pytest.mark.gpu

TINY2 = synth.with_layers(synth.TINY, 2)


def rq(state, pos, mask=None, rows=None, beam=None):
    return Request(state, np.asarray(pos, np.int32), None if mask is None else np.asarray(mask, np.uint8),
                   None if beam is None else np.asarray(beam, np.int32),
                   None if rows is None else np.asarray(rows, np.uint8))


@pytest.fixture(scope="module")
def tiny():
    p = Pair(TINY2, 190)
    yield p
    p.close()


def _tree_inputs(past):
    parent, anc, depth = tree_case()
    n = len(parent)
    rows = np.ones((1, n, past + n), np.uint8)
    rows[0, :, past:] = anc
    return parent, anc, (past + depth)[None], rows


def test_rows_repeating_slot_mask_are_bitwise_2d(tiny):
    S, past, n = 2, 30, 4
    ga, _ = tiny.states(S, past, 64, 191)
    gb, _ = tiny.states(S, past, 64, 191)
    mask = full_mask(S, past + n)
    mask[0, [3, 17]] = 0
    mask[1, past + 1] = 0
    pos = np.array([[28, 29, 30, 31], [29, 30, 30, 31]])
    x = synth.make_hidden(TINY2, S * n, 191)
    oa = run_gpu(tiny, [rq(ga, pos, mask)], x)
    ob = run_gpu(tiny, [rq(gb, pos, None, np.repeat(mask[:, None], n, axis=1))], x)
    assert np.array_equal(oa, ob)
    ga.free(); gb.free()


def _tree_vs_oracle_and_paths(p, past, seed, label):
    g, o = p.states(1, past, past + 16, seed)
    parent, anc, pos, rows = _tree_inputs(past)
    n = len(parent)
    x = synth.make_hidden(p.shape, n, seed)
    out = run_gpu(p, [rq(g, pos, None, rows)], x)
    ref = oracle.forward(p.orc, o, host(x), pos, None, None, rows)
    e = rel_err(out, ref)
    worst = 0.0
    for leaf in [i for i in range(n) if i not in parent]:
        path = [i for i in range(n) if anc[leaf, i]]
        gp, _ = p.states(1, past, past + 16, seed, with_oracle=False)
        lin = run_gpu(p, [rq(gp, pos[:, path], full_mask(1, past + len(path)))], x[path])
        worst = max(worst, rel_err(lin, out[path]))
        gp.free()
    print(f"{label}: tree verify vs oracle {e:.2e}; vs separate path verifies {worst:.2e}")
    assert e <= TOL_STAGE and worst <= TOL_STAGE
    g.free()


def test_tree_verify_tiny(tiny):
    _tree_vs_oracle_and_paths(tiny, 40, 192, "tiny")


def test_tree_verify_8b_layer_kv2048():
    p = Pair(synth.with_layers(synth.LLAMA8B_HALF, 1), 193)
    _tree_vs_oracle_and_paths(p, 2048, 193, "8B layer, KV 2048")
    # 4 slots x 5 tokens with holes: rows repeating the slot masks are bitwise the 2-D forward
    S, past, n = 4, 2048, 5
    k, v = synth.make_kv(p.shape, S, past, 194)
    ga, gb = p.gpu.new_state(S, past + 8), p.gpu.new_state(S, past + 8)
    ga.append(k, v)
    gb.append(k, v)
    mask = np.concatenate([np.stack([synth.hole_mask(past, 0.1, 194, b) for b in range(S)]),
                           np.ones((S, n), np.uint8)], 1)
    mask[:, -2:] = 0
    pos = mask[:, :past].sum(axis=1)[:, None] + np.arange(n)[None]
    x = synth.make_hidden(p.shape, S * n, 194)
    perm = np.array([1, 3, 0, 2])
    oa = run_gpu(p, [rq(ga, pos, mask, None, perm)], x)
    ob = run_gpu(p, [rq(gb, pos, None, np.repeat(mask[:, None], n, axis=1), perm)], x)
    assert np.array_equal(oa, ob)
    p.close()


def test_packed_sequences_shared_prefix(tiny):
    past, na, nb = 20, 3, 2
    g, o = tiny.states(1, past, 64, 195)
    n = na + nb
    rows = np.zeros((1, n, past + n), np.uint8)
    rows[0, :, :past] = 1
    for i in range(na):
        rows[0, i, past:past + i + 1] = 1
    for i in range(nb):
        rows[0, na + i, past + na:past + na + i + 1] = 1
    pos = np.concatenate([past + np.arange(na), past + np.arange(nb)])[None]
    x = synth.make_hidden(TINY2, n, 195)
    out = run_gpu(tiny, [rq(g, pos, None, rows)], x)
    ref = oracle.forward(tiny.orc, o, host(x), pos, None, None, rows)
    e = rel_err(out, ref)
    print(f"packed sequences: {e:.2e}")
    assert e <= TOL_STAGE
    g.free()


def test_row_masks_beside_plain_request(tiny):
    """A batch-mate with row masks leaves a plain request bitwise unchanged,
    and the rows' request matches the oracle."""
    ga, _ = tiny.states(1, 33, 64, 196)
    gb, ob = tiny.states(1, 40, 64, 197)
    gc, _ = tiny.states(1, 33, 64, 196)
    xa = synth.make_hidden(TINY2, 3, 196)
    parent, anc, pos_t, rows = _tree_inputs(40)
    xb = synth.make_hidden(TINY2, len(parent), 197)
    pos_a = np.array([[33, 34, 35]])
    import torch

    both = run_gpu(tiny, [rq(ga, pos_a, full_mask(1, 36)), rq(gb, pos_t, None, rows)], torch.cat([xa, xb]))
    alone = run_gpu(tiny, [rq(gc, pos_a, full_mask(1, 36))], xa)
    assert np.array_equal(both[:3], alone)
    ref = oracle.forward(tiny.orc, ob, host(xb), pos_t, None, None, rows)
    assert rel_err(both[3:], ref) <= TOL_STAGE
    for s in (ga, gb, gc):
        s.free()


def test_row_masks_vector_attention():
    old = {k: os.environ.get(k) for k in ("STAGE_ATTN_VECTOR", "STAGE_PERSISTENT")}
    os.environ.update(STAGE_ATTN_VECTOR="1", STAGE_PERSISTENT="0")
    try:
        p = Pair(TINY2, 198)
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    _tree_vs_oracle_and_paths(p, 40, 198, "tiny, vector-unit attention")
    p.close()


def test_single_row_with_row_mask(tiny):
    """M = 1 takes the single launch where the stage has one: its row mask is
    the slot mask, bitwise the 2-D form."""
    past = 50
    ga, o = tiny.states(1, past, 64, 199)
    gb, _ = tiny.states(1, past, 64, 199)
    mask = full_mask(1, past + 1)
    mask[0, [5, 6, 40]] = 0
    pos = np.array([[past - 3]])
    x = synth.make_hidden(TINY2, 1, 199)
    oa = run_gpu(tiny, [rq(ga, pos, mask)], x)
    ob = run_gpu(tiny, [rq(gb, pos, None, mask[:, None, :])], x)
    assert np.array_equal(oa, ob)
    assert rel_err(oa, oracle.forward(tiny.orc, o, host(x), pos, None, mask)) <= TOL_STAGE
    ga.free(); gb.free()


def test_row_with_no_visible_key_is_refused(tiny):
    g, _ = tiny.states(1, 10, 32, 200)
    rows = np.ones((1, 3, 13), np.uint8)
    rows[0, 1, :12] = 0                                       # row 1 sees only keys 0..11: all hidden
    x = synth.make_hidden(TINY2, 3, 200)
    with pytest.raises(StageError) as ei:
        run_gpu(tiny, [rq(g, np.array([[10, 11, 12]]), None, rows)], x)
    assert ei.value.code == -1 and g.length == 10
    g.free()
