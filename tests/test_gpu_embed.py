"""First-stage embedding gather against the oracle (paper, "Per-Stage Export
Pipeline": the first shard holds the token embedding ahead of its layers).

  * rows equal oracle.embed bit for bit: tiny table (vocab 1000, fp16) at 1,
    37 and STAGE_MAX_PREFILL ids with repeats and both ends of the table, a
    table attached from device memory, an output that is not 16-byte aligned
    (the 2-byte copy), and the Llama-3 table (128256 x 4096, bf16) at 1 and
    2048 ids;
  * an id outside the table gives a zero row, leaves the other rows right and
    flags the stage once (stage_device_status);
  * a first stage end to end: ids -> embed -> stage forward against the
    oracle's forward of oracle.embed;
  * argument errors."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_cases import TOL_STAGE, Pair, full_mask, host, rel_err, req
from paper_2608_19147_amd import StageError

pytestmark = pytest.mark.gpu

MAX_PREFILL = 8192


def _bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().view(torch.int16).numpy()


def _ref_bits(table: torch.Tensor, ids) -> np.ndarray:
    return oracle.embed(table.view(torch.int16).numpy(), ids)


def _ids(vocab, n, seed):
    ids = synth.make_token_ids(vocab, n, seed, n)
    ends = np.array([0, vocab - 1, 3, 3], np.int32)[: n]
    ids[: ends.size] = ends
    return ids


@pytest.fixture(scope="module")
def tiny_embed():
    shape = synth.TINY
    p = Pair(shape, 190, with_oracle=False)
    table = synth.make_embedding(shape, 1000, 190)
    p.gpu.attach_embedding(table)
    yield p, table
    p.close()


@pytest.mark.parametrize("n", [1, 37, MAX_PREFILL])
def test_embed_tiny_bitexact(tiny_embed, n):
    p, table = tiny_embed
    ids = _ids(1000, n, 191)
    out = p.gpu.embed(torch.from_numpy(ids).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(_bits(out), _ref_bits(table, ids)), n
    p.gpu.device_status()


def test_embed_unaligned_output(tiny_embed):
    """hidden_out one element past a 16-byte boundary takes the 2-byte copy."""
    p, table = tiny_embed
    ids = _ids(1000, 9, 192)
    buf = torch.full((9 * p.shape.hidden + 1,), -1, dtype=p.gpu.act_dtype, device="cuda")
    view = buf[1:].view(9, p.shape.hidden)
    assert view.data_ptr() % 16 != 0
    p.gpu.embed(torch.from_numpy(ids).cuda(), hidden_out=view)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(view), _ref_bits(table, ids))
    assert buf[0].item() == -1                                # nothing written before the output


def test_embed_out_of_range_flags(tiny_embed):
    p, table = tiny_embed
    ids = _ids(1000, 6, 193)
    bad = ids.copy()
    bad[2], bad[4] = 1000, -7
    out = p.gpu.embed(torch.from_numpy(bad).cuda())
    torch.cuda.synchronize()
    got = _bits(out)
    good = [0, 1, 3, 5]
    assert np.array_equal(got[good], _ref_bits(table, ids[good]))
    assert not got[[2, 4]].any()
    with pytest.raises(StageError) as ei:
        p.gpu.device_status()
    assert ei.value.code == -8
    p.gpu.device_status()                                    # reported once, then cleared
    out = p.gpu.embed(torch.from_numpy(ids).cuda())            # the next gather is clean
    torch.cuda.synchronize()
    assert np.array_equal(_bits(out), _ref_bits(table, ids))
    p.gpu.device_status()


def test_embed_device_table():
    shape = synth.with_layers(synth.TINY, 1)
    p = Pair(shape, 194, with_oracle=False)
    table = synth.make_embedding(shape, 333, 194)
    p.gpu.attach_embedding(table.cuda(), on_device=True)
    ids = _ids(333, 50, 194)
    out = p.gpu.embed(torch.from_numpy(ids).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(_bits(out), _ref_bits(table, ids))
    p.close()


def test_embed_llama3_table():
    shape = synth.with_layers(synth.LLAMA8B_HALF, 1)
    p = Pair(shape, 195, with_oracle=False)
    table = synth.make_embedding(shape, synth.LLAMA3_VOCAB, 195)
    p.gpu.attach_embedding(table)
    for n in (1, 2048):
        ids = _ids(synth.LLAMA3_VOCAB, n, 196)
        out = p.gpu.embed(torch.from_numpy(ids).cuda())
        torch.cuda.synchronize()
        assert np.array_equal(_bits(out), _ref_bits(table, ids)), n
    p.gpu.device_status()
    p.close()


def test_first_stage_decode_from_ids():
    """Stage 0 of a pipeline: the token ids of a verify step go through the
    gather and two layers, against the oracle's forward of its own lookup."""
    shape = synth.with_layers(synth.TINY, 2)
    p = Pair(shape, 197)
    table = synth.make_embedding(shape, 500, 197)
    p.gpu.attach_embedding(table)
    g, o = p.states(1, 30, 64, 197)
    ids = _ids(500, 4, 198)
    pos = np.arange(30, 34)[None]
    x = p.gpu.embed(torch.from_numpy(ids).cuda())
    out = p.gpu.forward([req(g, pos, full_mask(1, 34))], x)
    torch.cuda.synchronize()
    ref = oracle.forward(p.orc, o, oracle.embed(table.numpy(), ids).astype(np.float64), pos, None, full_mask(1, 34))
    e = rel_err(host(out), ref)
    print(f"first stage (embed + 2 layers, 4 rows) vs oracle: {e:.2e}")
    assert e <= TOL_STAGE
    g.free()
    p.close()


def test_embed_errors(tiny_embed):
    p, table = tiny_embed
    ids = torch.zeros(MAX_PREFILL + 1, dtype=torch.int32, device="cuda")
    with pytest.raises(StageError) as ei:
        p.gpu.embed(ids)                                       # more than STAGE_MAX_PREFILL ids
    assert ei.value.code == -3
    out = torch.empty((1, p.shape.hidden), dtype=p.gpu.act_dtype, device="cuda")
    assert p.gpu.lib.stage_embed(p.gpu.handle, ctypes.c_void_p(ids.data_ptr()), 0, ctypes.c_void_p(out.data_ptr()),
                                 None) == -3                   # no ids
    with pytest.raises(StageError) as ei:
        p.gpu.attach_embedding(table)                          # once per stage
    assert ei.value.code == -7
    q = Pair(p.shape, 199, with_oracle=False)
    with pytest.raises(StageError) as ei:
        q.gpu.embed(ids[:1])                                   # no table attached
    assert ei.value.code == -1
    q.close()
