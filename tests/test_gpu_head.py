"""Final-stage epilogue against the oracle (paper, "Top-1 Logits
Compression": the last stage reduces its logits row to the top-1 token and
its probability on the device).

  * the full logits rows (written on request) match oracle.head_logits;
  * the fused top-1 equals the argmax / softmax probability of the GPU's own
    logits rows (the same fp32 values decide the integer);
  * the token equals the oracle's wherever the oracle's top-2 gap exceeds
    the logits tolerance, else the GPU's token is within it of the maximum;
  * p_max within 1e-3 absolute and 1e-2 relative of the oracle's;
  * tiny head with a ragged last tile at 1, 5 and 64 rows, the Llama-3 sized
    head (128256 x 4096) at 1 and 20 rows, and a stage forward chained into
    the head against the oracle's forward + head."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_cases import TOL_STAGE, Pair, full_mask, host, rel_err, req

pytestmark = pytest.mark.gpu

GAP = 1e-2        # absolute logit gap above which the top-1 token must match the oracle's


def _check(stage, shape, fn, lm, x, label):
    tok, p, mx, lg = stage.head_top1(x.cuda(), with_logits=True)
    torch.cuda.synchronize()
    tok, p, mx, lg = tok.cpu().numpy(), p.cpu().numpy().astype(np.float64), mx.cpu().numpy(), lg.cpu().numpy()
    ref = oracle.head_logits(host(x), fn, lm.q, lm.scales, lm.n, shape.group_size, shape.rms_eps)
    e = rel_err(lg, ref)
    ri, rp, rmx = oracle.top1(ref)
    # the fused reduction is the argmax / softmax of the GPU's own fp32 logits
    gi, gp, gmx = oracle.top1(lg.astype(np.float64))
    assert np.array_equal(tok, gi) and np.array_equal(mx, gmx.astype(np.float32))
    assert np.max(np.abs(p - gp) / gp) <= 1e-5
    # against the oracle
    srt = np.sort(ref, axis=1)
    gap = srt[:, -1] - srt[:, -2]
    for m in range(ref.shape[0]):
        if gap[m] > GAP:
            assert tok[m] == ri[m], (label, m, gap[m])
        else:
            assert ref[m, tok[m]] >= rmx[m] - GAP, (label, m)
    dp = np.abs(p - rp)
    print(f"{label}: logits {e:.2e}, max |dp| {dp.max():.2e} (p_max up to {rp.max():.2e}), "
          f"max rel dp {np.max(dp / rp):.2e}, tokens decided by gap > {GAP}: {int((gap > GAP).sum())}/{len(gap)}")
    assert e <= TOL_STAGE
    assert dp.max() <= 1e-3 and np.max(dp / rp) <= 1e-2
    assert np.max(np.abs(mx - rmx)) <= GAP


@pytest.fixture(scope="module")
def tiny_head():
    shape = synth.TINY
    p = Pair(shape, 170)
    fn, lm = synth.make_head(shape, 1000, 170)              # 15 whole tiles + 40 rows
    p.gpu.attach_head(fn, lm)
    yield p, fn, lm
    p.close()


@pytest.mark.parametrize("M", [1, 5, 64])
def test_head_tiny(tiny_head, M):
    p, fn, lm = tiny_head
    x = synth.make_hidden(p.shape, M, 171, M)
    _check(p.gpu, p.shape, fn, lm, x, f"tiny vocab 1000 M={M}")


def test_head_sharp_rows(tiny_head):
    """Rows that differ only in sign or in scale (RMSNorm removes the scale up
    to the rounding of the scaled input)."""
    p, fn, lm = tiny_head
    x = synth.make_hidden(p.shape, 4, 172).float()
    x[1] = -x[0]
    x[2] = x[0] * 50                                         # RMSNorm removes the scale: same logits as row 0
    x = x.to(p.gpu.act_dtype)
    _check(p.gpu, p.shape, fn, lm, x, "tiny sharp rows")


def test_stage_forward_into_head(tiny_head):
    """A last stage: decode through the stage, then its top-1, vs the oracle's
    forward and head."""
    p, fn, lm = tiny_head
    g, o = p.states(1, 40, 64, 173)
    x = synth.make_hidden(p.shape, 1, 173)
    pos = np.array([[40]])
    out = p.gpu.forward([req(g, pos, full_mask(1, 41))], x.cuda())
    tok, pm, _, lg = p.gpu.head_top1(out, with_logits=True)
    ref_h = oracle.forward(p.orc, o, host(x), pos, None, full_mask(1, 41))
    # the head sees the stage output in the activation dtype, as the GPU does
    ref_h = host(torch.from_numpy(ref_h).to(p.gpu.act_dtype))
    ref = oracle.head_logits(ref_h, fn, lm.q, lm.scales, lm.n, p.shape.group_size, p.shape.rms_eps)
    e = rel_err(lg.cpu().numpy(), ref)
    print(f"stage forward + head vs oracle: logits {e:.2e}")
    assert e <= TOL_STAGE
    g.free()


def test_head_llama3_vocab():
    shape = synth.with_layers(synth.LLAMA8B_HALF, 1)
    p = Pair(shape, 180, with_oracle=False)
    fn, lm = synth.make_head(shape, synth.LLAMA3_VOCAB, 180)
    p.gpu.attach_head(fn, lm)
    for M in (1, 20):
        x = synth.make_hidden(shape, M, 181, M)
        _check(p.gpu, shape, fn, lm, x, f"8B head vocab {synth.LLAMA3_VOCAB} M={M}")
    p.close()


def test_head_errors(tiny_head):
    from paper_2608_19147_amd import StageError

    p, fn, lm = tiny_head
    x = synth.make_hidden(p.shape, 65, 174).cuda()
    with pytest.raises(StageError) as ei:
        p.gpu.head_top1(x)                                    # 65 rows > STAGE_MAX_ROWS
    assert ei.value.code == -3
    with pytest.raises(StageError) as ei:
        p.gpu.attach_head(fn, lm)                             # once per stage
    assert ei.value.code == -7
    q = Pair(p.shape, 175, with_oracle=False)
    with pytest.raises(StageError) as ei:
        q.gpu.head_top1(x[:1])                                # no head attached
    assert ei.value.code == -1
    q.close()
