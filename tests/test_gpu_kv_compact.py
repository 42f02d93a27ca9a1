"""KV compaction and capture/restore against the oracle (paper, "Mask-Based
Rewind": masked positions are removed when the state is serialized; "Prefix
Caching: KV Capture and Warm-Resume": a stage serializes its own layers'
state keeping only mask-valid rows and restores it all-or-nothing).

  * kv_compact leaves, in every layer, slot and kv head, exactly the rows of
    oracle.compact, bit for bit, after forwards that left a non-identity beam
    table and masked holes;
  * the next forward on the compacted state matches the oracle (which runs
    it on its own compacted state and, bitwise equal, on the holed state with
    its mask) within the stage tolerance;
  * a blob holds the oracle's compacted rows; host and device blobs are the
    same bytes; restore + forward is bitwise compact + forward;
  * edge cases: keep everything, a slot that keeps nothing, every row
    dropped, an empty state; all-or-nothing errors."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_cases import TOL_STAGE, Pair, full_mask, host, rel_err, req, run_gpu
from oracle_cases import logical_positions
from paper_2608_19147_amd import StageError

pytestmark = pytest.mark.gpu

TINY = synth.with_layers(synth.TINY, 2)


@pytest.fixture(scope="module")
def tiny():
    p = Pair(TINY, 110)
    yield p
    p.close()


def _rows_gpu(state, shape, P):
    """[L][S][Hkv][P][D] K and V as the slots see them (fp64)."""
    L, S = shape.n_layers, state.n_slots
    K = np.zeros((L, S, shape.n_kv_heads, P, shape.head_dim))
    V = np.zeros_like(K)
    if P == 0:
        return K, V
    for l in range(L):
        for b in range(S):
            k, v = state.read(l, b, 0, P)
            K[l, b], V[l, b] = host(k), host(v)
    return K, V


def _rows_oracle(ost, P):
    K = np.stack([ost.K[l][:, :, :P] for l in range(len(ost.K))])
    V = np.stack([ost.V[l][:, :, :P] for l in range(len(ost.V))])
    return K, V


def _blob_rows(blob: np.ndarray, shape, S):
    """(length, slot lengths, K, V) of a capture blob, parsed by the layout the
    header documents."""
    hdr = np.frombuffer(blob[:48].tobytes(), dtype=np.int32)
    assert int(np.frombuffer(blob[:8].tobytes(), np.uint64)[0]) == 0x31505643564B5453
    hbytes = int(hdr[3])
    L, S_, hkv, d, _, P = (int(x) for x in hdr[6:12])
    assert (L, S_, hkv, d) == (shape.n_layers, S, shape.n_kv_heads, shape.head_dim)
    lens = np.frombuffer(blob[48:48 + 4 * S].tobytes(), np.int32)
    dt = torch.float16 if shape.kv_dtype == "f16" else torch.bfloat16
    n = L * S * hkv * P * d
    raw = torch.from_numpy(np.ascontiguousarray(blob[hbytes:hbytes + 4 * n])).view(dt).double().numpy()
    return P, lens, raw[:n].reshape(L, S, hkv, P, d), raw[n:].reshape(L, S, hkv, P, d)


def _holed_pair(p, S, past, cap, seed, n_verify=5):
    """A GPU state and its oracle twin after one verify forward with a beam
    permutation and rejected drafts; returns them with the keep mask [S, P]."""
    g, o = p.states(S, past, cap, seed)
    r = np.random.default_rng(seed)
    holes = np.ones((S, past), np.uint8)
    for b in range(S):
        holes[b, r.choice(past, max(1, past // 8), replace=False)] = 0
    perm = r.permutation(S).astype(np.int32) if S > 1 else np.zeros(1, np.int32)
    holes = holes[perm]                                    # a slot's holes move with its rows
    acc = r.integers(0, n_verify, size=S)                  # accepted drafts per slot
    mask = np.concatenate([holes, np.ones((S, n_verify), np.uint8)], 1)
    pos = logical_positions(holes, n_verify)
    x = synth.make_hidden(p.shape, S * n_verify, seed, 1)
    og = run_gpu(p, [req(g, pos, mask, perm)], x)
    oo = oracle.forward(p.orc, o, host(x), pos, perm, mask)
    assert rel_err(og, oo) <= TOL_STAGE
    keep = mask.copy()
    for b in range(S):
        keep[b, past + 1 + acc[b]:] = 0                    # drafts after the first rejection
    _sync_new_rows(g, o, past)
    return g, o, keep


def _sync_new_rows(g, o, past):
    """The rows a forward appended are the GPU's own computation: check them
    against the oracle's within the stage tolerance and the cached rows
    exactly, then put the GPU's rows into the oracle state so that compaction
    is compared bit for bit on identical contents."""
    K, V = _rows_gpu(g, o.shape, o.P)
    Ko, Vo = _rows_oracle(o, o.P)
    assert np.array_equal(K[..., :past, :], Ko[..., :past, :]) and np.array_equal(V[..., :past, :], Vo[..., :past, :])
    assert rel_err(K[..., past:, :], Ko[..., past:, :]) <= TOL_STAGE
    assert rel_err(V[..., past:, :], Vo[..., past:, :]) <= TOL_STAGE
    for l in range(o.shape.n_layers):
        o.K[l][:, :, : o.P] = K[l]
        o.V[l][:, :, : o.P] = V[l]


def _next_forward(p, g, o, lens, n, seed, logical_len):
    """A forward of n tokens on compacted states (padding rows hidden)."""
    S = len(lens)
    P = g.length
    mask = np.zeros((S, P + n), np.uint8)
    for b in range(S):
        mask[b, :lens[b]] = 1
    mask[:, P:] = 1
    pos = np.asarray(logical_len)[:, None] + np.arange(n)[None]
    x = synth.make_hidden(p.shape, S * n, seed, 7)
    og = run_gpu(p, [req(g, pos, mask)], x)
    oo = oracle.forward(p.orc, o, host(x), pos, None, mask)
    return og, oo


@pytest.mark.parametrize("S,past", [(1, 72), (3, 40)])
def test_compact_rows_and_next_forward(tiny, S, past):
    g, o, keep = _holed_pair(tiny, S, past, 128, 111 + S)
    P = g.length
    lens = g.compact(keep)
    oc, olens = oracle.compact(o, keep)
    assert list(lens) == list(olens) and g.length == oc.P
    Kg, Vg = _rows_gpu(g, TINY, oc.P)
    Ko, Vo = _rows_oracle(oc, oc.P)
    assert np.array_equal(Kg, Ko) and np.array_equal(Vg, Vo)
    # next forward: GPU compacted vs oracle compacted, and the oracle's holed
    # state with its mask gives bitwise the same reference
    oh = o.copy()
    og, oo = _next_forward(tiny, g, oc, lens, 3, 113 + S, olens)
    mask_h = np.concatenate([keep, np.ones((S, 3), np.uint8)], 1)
    x = synth.make_hidden(TINY, S * 3, 113 + S, 7)
    ref_h = oracle.forward(tiny.orc, oh, host(x), olens[:, None] + np.arange(3)[None], None, mask_h)
    assert np.array_equal(oo, ref_h)
    e = rel_err(og, oo)
    print(f"S={S}: compacted forward vs oracle {e:.2e}")
    assert e <= TOL_STAGE
    # and a single decode row (the single-launch path where the stage has one)
    if S == 1:
        og1, oo1 = _next_forward(tiny, g, oc, olens + 3, 1, 114, olens + 3)   # no padding at S = 1
        assert rel_err(og1, oo1) <= TOL_STAGE
    g.free()


def test_capture_restore_roundtrip(tiny):
    S, past = 3, 40
    g, o, keep = _holed_pair(tiny, S, past, 128, 120)
    blob_d = g.capture(keep, on_device=True)
    blob_h = g.capture(keep, on_device=False)
    assert blob_d.numel() == blob_h.size == g.capture_size(keep)
    assert np.array_equal(blob_d.cpu().numpy(), blob_h)
    Pb, lens_b, Kb, Vb = _blob_rows(blob_h, TINY, S)
    oc, olens = oracle.compact(o, keep)
    assert Pb == oc.P and list(lens_b) == list(olens)
    Ko, Vo = _rows_oracle(oc, Pb)
    assert np.array_equal(Kb, Ko) and np.array_equal(Vb, Vo)
    P_before = g.length
    # capture leaves the state as it was
    assert g.length == P_before
    # restore into fresh states from both blobs; compact the original in place
    r_d = tiny.gpu.new_state(S, 128)
    r_h = tiny.gpu.new_state(S, 128)
    assert list(r_d.restore(blob_d)) == list(olens)
    assert list(r_h.restore(blob_h)) == list(olens)
    lens = g.compact(keep)
    for st in (r_d, r_h):
        assert st.length == g.length
        Kr, Vr = _rows_gpu(st, TINY, st.length)
        assert np.array_equal(Kr, Ko) and np.array_equal(Vr, Vo)
    # warm resume: restore + forward is bitwise compact + forward
    res = [_next_forward(tiny, st, oc.copy(), lens, 4, 121, olens) for st in (g, r_d, r_h)]
    assert np.array_equal(res[0][0], res[1][0]) and np.array_equal(res[0][0], res[2][0])
    assert rel_err(res[0][0], res[0][1]) <= TOL_STAGE
    for st in (g, r_d, r_h):
        st.free()


def test_compact_edge_cases(tiny):
    shape = TINY
    # keep everything: contents and length unchanged (identity beam table)
    g, o = tiny.states(2, 30, 64, 130)
    K0, V0 = _rows_gpu(g, shape, 30)
    assert list(g.compact(None)) == [30, 30] and g.length == 30
    K1, V1 = _rows_gpu(g, shape, 30)
    assert np.array_equal(K0, K1) and np.array_equal(V0, V1)
    # one slot keeps nothing, the other a few rows
    keep = np.zeros((2, 30), np.uint8)
    keep[1, [0, 5, 29]] = 1
    lens = g.compact(keep)
    oc, olens = oracle.compact(o, keep)
    assert list(lens) == [0, 3] and g.length == 3
    Kg, Vg = _rows_gpu(g, shape, 3)
    Ko, Vo = _rows_oracle(oc, 3)
    assert np.array_equal(Kg, Ko) and np.array_equal(Vg, Vo)
    # every row dropped: an empty state that takes a first token at P = 0
    assert list(g.compact(np.zeros((2, 3), np.uint8))) == [0, 0] and g.length == 0
    blob = g.capture(None, on_device=False)
    assert blob.size == g.capture_size(None)
    e = tiny.gpu.new_state(2, 8)
    assert list(e.restore(blob)) == [0, 0] and e.length == 0
    x = synth.make_hidden(shape, 2, 131)
    o0 = oracle.OracleState(shape, 2, 64)
    og = run_gpu(tiny, [req(g, np.zeros((2, 1), np.int32), full_mask(2, 1))], x)
    oo = oracle.forward(tiny.orc, o0, host(x), np.zeros((2, 1)), None, full_mask(2, 1))
    assert rel_err(og, oo) <= TOL_STAGE
    g.free(); e.free()


def test_restore_errors_leave_state_unchanged(tiny):
    shape = TINY
    g, _ = tiny.states(2, 20, 64, 140)
    blob = g.capture(None, on_device=False)
    tgt, _ = tiny.states(2, 5, 64, 141)
    K0, V0 = _rows_gpu(tgt, shape, 5)

    def expect(code, fn):
        with pytest.raises(StageError) as ei:
            fn()
        assert ei.value.code == code, ei.value
        assert tgt.length == 5
        K1, V1 = _rows_gpu(tgt, shape, 5)
        assert np.array_equal(K0, K1) and np.array_equal(V0, V1)

    bad = blob.copy()
    bad[0] ^= 1
    expect(-1, lambda: tgt.restore(bad))                      # magic
    expect(-2, lambda: tgt.restore(blob[:-2]))                # truncated rows
    small = tiny.gpu.new_state(2, 10)
    with pytest.raises(StageError) as ei:
        small.restore(blob)                                   # 20 rows > capacity 10
    assert ei.value.code == -3 and small.length == 0
    three = tiny.gpu.new_state(3, 64)
    with pytest.raises(StageError) as ei:
        three.restore(blob)                                   # slot count
    assert ei.value.code == -6
    other = Pair(shape, 142, with_oracle=False)               # another stage: other norm weights
    ost = other.gpu.new_state(2, 64)
    with pytest.raises(StageError) as ei:
        ost.restore(blob)
    assert ei.value.code == -6 and ost.length == 0
    other.close()
    # a blob buffer smaller than the capture
    from paper_2608_19147_amd import _lib
    import ctypes

    lib = _lib.load()
    short = np.zeros(g.capture_size(None) - 1, np.uint8)
    rc = lib.kv_capture(g.handle, None, ctypes.c_void_p(short.ctypes.data), short.size, 0,
                        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == -3
    for s in (g, tgt, small, three):
        s.free()


SHAPE8 = synth.with_layers(synth.LLAMA8B_HALF, 2)


def test_compact_8b_two_layers_kv2048():
    """Two 8B-shaped layers, 4 slots at KV 2048 with a beam permutation, 10%
    holes and rejected drafts: compacted rows bit-exact against oracle.compact
    of the rows the slots saw, capture == those rows, and the next verify
    on the compacted state vs the oracle."""
    p = Pair(SHAPE8, 150)
    S, past, n = 4, 2048, 5
    k, v = synth.make_kv(SHAPE8, S, past, 150)
    g = p.gpu.new_state(S, past + 16)
    g.append(k, v)
    o = oracle.OracleState(SHAPE8, S, past + 16)
    o.append(k.double().numpy(), v.double().numpy())
    del k, v
    perm = np.array([2, 0, 3, 1], np.int32)
    holes = np.stack([synth.hole_mask(past, 0.1, 150, b) for b in range(S)])
    mask = np.concatenate([holes, np.ones((S, n), np.uint8)], 1)
    mask[:, -2:] = 0                                          # last two drafts rejected
    pos = logical_positions(holes, n)
    x = synth.make_hidden(SHAPE8, S * n, 150, 1)
    og = run_gpu(p, [req(g, pos, mask, perm)], x)
    oo = oracle.forward(p.orc, o, host(x), pos, perm, mask)
    assert rel_err(og, oo) <= TOL_STAGE
    keep = mask
    _sync_new_rows(g, o, past)
    blob = g.capture(keep, on_device=True)
    lens = g.compact(keep)
    oc, olens = oracle.compact(o, keep)
    assert list(lens) == list(olens)
    Kg, Vg = _rows_gpu(g, SHAPE8, oc.P)
    Ko, Vo = _rows_oracle(oc, oc.P)
    assert np.array_equal(Kg, Ko) and np.array_equal(Vg, Vo)
    Pb, lens_b, Kb, Vb = _blob_rows(blob.cpu().numpy(), SHAPE8, S)
    assert Pb == oc.P and list(lens_b) == list(olens) and np.array_equal(Kb, Ko) and np.array_equal(Vb, Vo)
    og2, oo2 = _next_forward(p, g, oc, lens, n, 151, olens)
    e = rel_err(og2, oo2)
    print(f"8B 2 layers, 4 slots: compacted verify vs oracle {e:.2e}")
    assert e <= TOL_STAGE
    g.free()
    p.close()
