#!/usr/bin/env python3
"""Stage decode throughput of the Llama-3.1-8B half stage on one MI355X.

Workload: 16 Llama decoder layers (hidden 4096, 32/8 heads, head_dim 128,
SwiGLU 14336) with INT4 group-128 weights and fp16 scales, bf16 activations
and bf16 KV cache, batch 1, single-token decode over a KV cache of 2048 rows
(also reported at 512), beam_idx = identity, all-ones mask.  A step is one
stage_forward (every layer: RMSNorm, W4A16 q/k/v, rotary + KV append,
split-KV attention, W4A16 o + residual, RMSNorm, W4A16 gate|up + SwiGLU,
W4A16 down + residual) on hidden states already resident in HBM; the KV
length is reset to the measured length after each step (metadata only).

Prints one JSON line: tokens/s, algorithmic HBM bytes per step and the
achieved fraction of the 8 TB/s HBM peak, the dominant kernel's roofline
(timed with HIP events on its launch stream), and the fp64 CPU oracle timed
on a bounded sample on the host cores.

--workload selects the other measured configurations (one JSON line per case,
same fields, no CPU baseline):
  verify8b      speculative verify on the 8B half stage: 4 cache slots x 5
                tokens, KV 2048 growing to 2368 over 64 steps, draft outcomes
                Bernoulli(0.6) truncated at the first rejection (rejected rows
                stay as masked holes), beam_idx identity on even steps and a
                seeded permutation on odd steps;
  microbatch8b  2, 4 and 8 independent requests in one forward, KV lengths
                U{128..4096} with 10% masked holes, all-decode and mixed
                (half the requests verify 5 tokens) modes;
  decode70b     Llama-3-70B quarter stage (20 layers), bs=1 decode at KV 8192;
  verify70b     the same stage, 5-token verify at KV 4096 with Bernoulli(0.6)
                rejections masked over 16 steps;
  compact8b     KV compaction and capture on the 8B half stage: 4 slots at the
                speculative-verify length 2368 with the bloat of truncated
                Bernoulli(0.6) acceptance (about 7% masked holes per slot);
                kv_compact in place (state re-installed from a full blob before
                each timed call) and kv_capture of the kept rows to a device blob;
  prefill8b     prompt prefill on the 8B half stage: 2048 prompt tokens from an empty
                cache (and 512 after 1536 cached rows), stage_prefill (passes of up
                to 2048 rows through every layer: matrix-core products over the whole
                pass, the causal attention of its 64-row chunks in one launch);
  tree8b        tree-shaped speculative verify on the 8B half stage: one slot at KV
                2048, a 15-node binary draft tree (depth 3) in one forward with a
                per-query-row mask (each node sees the cache and its ancestors);
                beside it the 5-token linear verify of one path;
  head8b        final-stage epilogue: final RMSNorm + INT4 LM head (128256 x 4096,
                group 128) + on-device top-1 (token, probability), 1 and 20 rows;
                and the first stage's embedding gather from the 128256 x 4096
                bf16 table, 1, 20 and 2048 ids;
  copycal       1 GiB device copies (calibration of HBM byte counters).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0

# HBM bytes per launch of the single-launch forward at the headline workload
# (KV 2048), from one FETCH_SIZE and one WRITE_SIZE counter run scaled by what
# the same counters read for a plain 1 GiB device copy (x2.0 and x1.0).  Keyed
# by a digest of the sources and build flags that define the kernel and its
# launch: after any change to them the figure no longer applies and ``traffic``
# is null.
MEASURED_TRAFFIC = {("d5ac1b9e5a58db0e", 2048): 2_027_096_834}
KERNEL_SOURCES = ("csrc/persistent.hip", "csrc/common.h", "csrc/device.h", "csrc/stage.hip", "build.py")


def kernel_digest() -> str:
    import hashlib

    h = hashlib.sha256()
    for name in KERNEL_SOURCES:                          # the sources and the compiler flags
        with open(os.path.join(ROOT, "paper_2608_19147_amd", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(shape, kv_len: int, n_new: int = 1) -> dict:
    """Each weight byte once (INT4 codes + fp16 scales + norm weights) plus each
    KV row the step needs once per layer (the P cached rows and the new row)."""
    w = shape.weight_bytes()
    kv = shape.kv_bytes_per_token() * (kv_len + n_new)
    return {"weights": w, "kv": kv, "total": w + kv}


def gateup_bytes(shape) -> int:
    """INT4 codes + fp16 scales of W_gate and W_up of one layer (one launch)."""
    F, H, G = shape.ffn, shape.hidden, shape.group_size
    return 2 * (F * (H // 2) + F * ((H + G - 1) // G) * 2)


def cpu_baseline(shape, kv_len: int, layers_sampled: int, seed: int, min_seconds: float = 8.0) -> dict:
    """The fp64 oracle as it stands on a bounded sample: ``layers_sampled`` of the
    stage's layers for one decode step, in its two modes, each repeated for about
    ``min_seconds``; the mean per-step time is scaled to all layers.  ``value`` is
    the steady state with the dequantized fp64 weights kept (the oracle's default,
    dequantized once before timing); ``streaming`` dequantizes each layer when it
    is used."""
    import numpy as np

    import oracle
    import synth

    try:
        from threadpoolctl import threadpool_info

        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        blas_threads = 1
    sub = synth.with_layers(shape, layers_sampled)
    layers = synth.make_weights(sub, seed)
    state = oracle.OracleState(sub, 1, kv_len + 1)
    k, v = synth.make_kv(sub, 1, kv_len, seed)
    state.append(k.double().numpy(), v.double().numpy())
    del k, v
    x = synth.make_hidden(sub, 1, seed).double().numpy()
    pos, beam, mask = np.array([[kv_len]]), np.array([0]), np.ones((1, kv_len + 1), np.uint8)
    res = {}
    for mode, cached in (("cached", True), ("streaming", False)):
        ost = oracle.OracleStage(sub, layers, cache_weights=cached)
        if cached:
            for l in range(sub.n_layers):
                ost.weights(l)                               # dequantized once, outside the timing
        dt, reps = 0.0, 0
        while reps < 1 or (dt < min_seconds and reps < 64):
            s = state.copy()
            t0 = time.perf_counter()
            oracle.forward(ost, s, x, pos, beam, mask)
            dt += time.perf_counter() - t0
            reps += 1
        res[mode] = (dt, reps, dt / reps * shape.n_layers / layers_sampled)
        del ost
    dt, reps, step_s = res["cached"]
    sdt, sreps, sstep = res["streaming"]
    scale = shape.n_layers / layers_sampled
    return {
        "value": round(1.0 / step_s, 5), "unit": "tokens/s", "cores": int(blas_threads), "kind": "oracle",
        "sample": f"{layers_sampled} of {shape.n_layers} layers of one bs=1 decode step at KV {kv_len} in fp64 with the "
                  f"dequantized weights kept (steady state), run {reps} times: {dt:.2f} s, {dt / reps:.3f} s each; "
                  f"scaled x{scale:g} to a full step; BLAS threads {blas_threads}, elementwise numpy single-threaded",
        "streaming": {"value": round(1.0 / sstep, 5), "unit": "tokens/s",
                      "sample": f"the same sample dequantizing each layer when used, run {sreps} times: {sdt:.2f} s, "
                                f"{sdt / sreps:.3f} s each; scaled x{scale:g}"},
    }


WORKLOADS = ("decode8b", "verify8b", "microbatch8b", "decode70b", "verify70b", "prefill8b", "tree8b", "compact8b", "head8b",
             "copycal")


def _line(metric, value, unit, args, steps, ms, config, bytes_per_step, roof, higher=True, **extra):
    gbps = bytes_per_step / (ms * 1e-3) / 1e9
    line = {
        "metric": metric, "value": round(value, 3), "unit": unit, "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": higher, "scaling": "weak",
        "vs_baseline": None, "dtype": "w4a16", "data": "synthetic", "config": config,
        "hbm_bytes_per_step": int(bytes_per_step), "achieved_gbps": round(gbps, 1),
        "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4), "roofline": roof,
    }
    line.update(extra)
    return line


def _gateup_roofline(shape, prof):
    """Roofline of the gate|up product of the multi-kernel path (gemm_bp_kernel:
    matrix cores, prepared input, 1..64 rows)."""
    launches, total_ms = prof
    per = total_ms / max(1, launches)
    b = gateup_bytes(shape)
    g = b / (per * 1e-3) / 1e9
    name = "gemm_bp_kernel"
    return {"bound": "hbm", "kernel": f"{name} gate|up (one launch per layer)", "achieved": round(g, 1),
            "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(g / HBM_PEAK_GBPS, 4), "traffic": None,
            "bytes_per_launch": b, "avg_launch_us": round(per * 1e3, 3), "launches_timed": launches}


def _profiled(stage, run):
    """(launches, ms) of the gate|up product over one more pass of `run`, timed
    with HIP events on the launch stream around each launch."""
    import torch

    torch.cuda.synchronize()
    stage.profile("gateup")
    run()
    torch.cuda.synchronize()
    prof = stage.profile_read()
    stage.profile(None)
    return prof


def other_workload(args) -> int:
    """The measured configurations besides the headline decode (see --workload)."""
    import numpy as np
    import torch

    import synth
    from paper_2608_19147_amd import Request, Stage
    from paper_2608_19147_amd.driver import VerifyDriver

    if args.workload == "copycal":
        # calibration for HBM byte counters: device-to-device copies of a known size
        nbytes = 1 << 30
        src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        t = time.perf_counter()
        for _ in range(max(1, args.steps)):
            dst.copy_(src)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t) * 1e3 / max(1, args.steps)
        print(json.dumps({"metric": "device copy GB/s (calibration)", "value": round(2 * nbytes / (ms * 1e-3) / 1e9, 1),
                          "unit": "GB/s", "bytes_read_per_copy": nbytes, "bytes_written_per_copy": nbytes,
                          "copies": max(1, args.steps), "ms_per_copy": round(ms, 4)}), flush=True)
        return 0
    if args.workload == "compact8b":
        return compact_workload(args)
    if args.workload == "head8b":
        return head_workload(args)
    big = args.workload.endswith("70b")
    shape = synth.LLAMA70B_QUARTER if big else synth.LLAMA8B_HALF
    t0 = time.perf_counter()
    stage = Stage(shape, synth.make_weights(shape, args.seed))
    torch.cuda.synchronize()
    print(f"# setup {time.perf_counter() - t0:.1f}s (weights {stage.weight_bytes() / 1e9:.3f} GB on device)",
          file=sys.stderr, flush=True)
    kvb = shape.kv_bytes_per_token()
    wbytes = shape.weight_bytes()
    base_cfg = {"layers": shape.n_layers, "hidden": shape.hidden, "q_heads": shape.n_q_heads,
                "kv_heads": shape.n_kv_heads, "head_dim": shape.head_dim, "ffn": shape.ffn,
                "group_size": shape.group_size, "act": shape.act_dtype, "kv_cache": shape.kv_dtype}
    lines = []

    if args.workload in ("verify8b", "verify70b"):
        S, n, K = (4, 5, 64) if not big else (1, 5, 16)
        P0 = 2048 if not big else 4096
        steps = args.steps if args.steps > 0 else K
        state = stage.new_state(S, P0 + K * n + 8)
        k, v = synth.make_kv(shape, S, P0, args.seed)
        state.append(k, v)
        del k, v
        xs = [synth.make_hidden(shape, S * n, args.seed, 200 + i).cuda() for i in range(8)]
        out = torch.empty_like(xs[0])

        def episode(n_steps, step0, timed):
            """n_steps verify steps from a fresh P0-row state; returns (seconds, emitted, bytes)."""
            state.truncate(P0)
            drv = VerifyDriver(S, P0)
            emitted, nbytes, el = 0, 0, 0.0
            torch.cuda.synchronize()
            t = time.perf_counter()
            for i in range(n_steps):
                st = step0 + i
                beam = None if S == 1 else (np.arange(S, dtype=np.int32) if st % 2 == 0
                                            else synth.beam_permutation(S, args.seed, st))
                P = drv.physical_len
                pos, mask, beam = drv.step_inputs(n, beam)
                stage.forward([Request(state, pos, mask, beam)], xs[st % len(xs)], out)
                emitted += int(drv.accept(synth.acceptance_draws(S, n - 1, 0.6, args.seed, st)).sum())
                nbytes += wbytes + S * (P + n) * kvb
            torch.cuda.synchronize()
            el = time.perf_counter() - t
            return el, emitted, nbytes

        if args.warmup:
            episode(min(args.warmup, K), 10_000, False)
        tot_s, tot_em, tot_b, done = 0.0, 0, 0, 0
        while done < steps:
            m = min(K, steps - done)
            el, em, nb = episode(m, done, True)
            tot_s, tot_em, tot_b, done = tot_s + el, tot_em + em, tot_b + nb, done + m
        # the gate|up launches are timed in a pass of their own: the events around
        # each launch would otherwise add their own gaps to the timed steps
        prof = _profiled(stage, lambda: episode(min(K, steps), 0, False))
        ms = tot_s * 1e3 / steps
        cfg = {"workload": (f"llama3.1-8b half stage speculative verify, {S} slots x {n} tokens, kv {P0} growing "
                            f"by up to {n} per step, drafts Bernoulli(0.6) truncated, beam identity/permutation "
                            f"alternating") if not big else
               f"llama3-70b quarter stage verify, 1 slot x {n} tokens, kv {P0} growing, drafts Bernoulli(0.6) truncated",
               **base_cfg, "slots": S, "tokens_per_slot": n, "kv_len_start": P0}
        lines.append(_line(f"spec-verify steps/s ({'8B half' if not big else '70B quarter'}-stage, {S}x{n} tokens)",
                           1e3 / ms, "steps/s", args, steps, ms, cfg, tot_b / steps, _gateup_roofline(shape, prof),
                           query_tokens_per_s=round(S * n * 1e3 / ms, 1),
                           emitted_tokens_per_s=round(tot_em / tot_s, 1),
                           mean_tokens_kept_per_slot_step=round(tot_em / (steps * S), 4)))

    elif args.workload == "prefill8b":
        MFMA_PEAK = 2500.0                                   # dense fp16 TFLOP/s
        for P0, n in ((0, 2048), (1536, 512)):
            state = stage.new_state(1, P0 + n + 8)
            if P0:
                k, v = synth.make_kv(shape, 1, P0, args.seed)
                state.append(k, v)
                del k, v
            x = synth.make_hidden(shape, n, args.seed, 600).cuda()
            out = torch.empty_like(x)
            pos = P0 + np.arange(n, dtype=np.int32)
            steps = max(1, args.steps // 20)
            for i in range(max(1, args.warmup // 5)):
                stage.prefill(state, pos, x, hidden_out=out)
                state.truncate(P0)
            torch.cuda.synchronize()
            t = time.perf_counter()
            for i in range(steps):
                stage.prefill(state, pos, x, hidden_out=out)
                state.truncate(P0)
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t) * 1e3 / steps

            def again():
                for i in range(steps):
                    stage.prefill(state, pos, x, hidden_out=out)
                    state.truncate(P0)

            launches, gu_ms = _profiled(stage, again)
            # gate|up: one input preparation + one product per layer and pass of at most 2048 rows
            per = gu_ms / max(1, launches)
            pass_rows = [min(2048, n - r0) for r0 in range(0, n, 2048)]
            gu_flop = 2.0 * 2 * shape.ffn * shape.hidden * (sum(pass_rows) / len(pass_rows))
            tf = gu_flop / (per * 1e-3) / 1e12
            roof = {"bound": "mfma", "kernel": "bprep_rows_kernel + gemm_pf_kernel gate|up (one pass per layer)",
                    "achieved": round(tf, 1), "peak": MFMA_PEAK, "unit": "TFLOP/s", "frac": round(tf / MFMA_PEAK, 4),
                    "traffic": None, "flop_per_launch": gu_flop, "avg_launch_us": round(per * 1e3, 3),
                    "launches_timed": launches}
            lin_flop = 2.0 * n * shape.weight_bytes() * 2 / 1.03   # ~2 int4 weights per byte (scales ~3% of bytes)
            cfg = {"workload": f"llama3.1-8b half stage prefill, {n} prompt tokens after {P0} cached rows", **base_cfg,
                   "prompt_tokens": n, "kv_len_before": P0, "pass_rows": 2048, "attention_chunk_rows": 64}
            lines.append(_line(f"prefill tokens/s (8B half-stage, {n} tokens after {P0})", n * 1e3 / ms, "tokens/s", args,
                               steps, ms, cfg, wbytes + (P0 + n) * kvb, roof,
                               linear_tflops=round(lin_flop / (ms * 1e-3) / 1e12, 1)))
            state.free()
            del x, out

    elif args.workload == "tree8b":
        P = 2048
        parent = [-1] + [(i - 1) // 2 for i in range(1, 15)]       # binary tree: 1 + 2 + 4 + 8 nodes
        n = len(parent)
        anc = np.zeros((n, n), np.uint8)
        for i in range(n):
            k = i
            while k >= 0:
                anc[i, k] = 1
                k = parent[k]
        depth = anc.sum(axis=1) - 1
        rows = np.ones((1, n, P + n), np.uint8)
        rows[0, :, P:] = anc
        state = stage.new_state(1, P + n + 8)
        k, v = synth.make_kv(shape, 1, P, args.seed)
        state.append(k, v)
        del k, v
        cases = [("tree", n, Request(state, (P + depth)[None].astype(np.int32), None, None, rows)),
                 ("linear", 5, Request(state, (P + np.arange(5))[None].astype(np.int32), np.ones((1, P + 5), np.uint8)))]
        for name, nn, req in cases:
            xs = [synth.make_hidden(shape, nn, args.seed, 500 + i).cuda() for i in range(4)]
            out = torch.empty_like(xs[0])
            for i in range(args.warmup):
                stage.forward([req], xs[i % 4], out)
                state.truncate(P)
            torch.cuda.synchronize()

            def loop():
                for i in range(args.steps):
                    stage.forward([req], xs[i % 4], out)
                    state.truncate(P)

            t = time.perf_counter()
            loop()
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t) * 1e3 / args.steps
            prof = _profiled(stage, loop)
            desc = (f"{n}-node binary draft tree (depth 3), per-query-row mask" if name == "tree"
                    else "5-token linear verify of one path")
            cfg = {"workload": f"llama3.1-8b half stage spec verify, 1 slot, kv {P}, {desc}", **base_cfg,
                   "kv_len": P, "tokens": nn}
            lines.append(_line(f"spec-verify steps/s (8B half-stage, {name}, {nn} tokens)", 1e3 / ms, "steps/s", args,
                               args.steps, ms, cfg, wbytes + (P + nn) * kvb, _gateup_roofline(shape, prof),
                               query_tokens_per_s=round(nn * 1e3 / ms, 1)))

    elif args.workload == "decode70b":
        P = 8192
        state = stage.new_state(1, P + 8)
        k, v = synth.make_kv(shape, 1, P, args.seed)
        state.append(k, v)
        del k, v
        xs = [synth.make_hidden(shape, 1, args.seed, 100 + i).cuda() for i in range(8)]
        out = torch.empty_like(xs[0])
        req = Request(state, np.array([[P]], np.int32), np.ones((1, P + 1), np.uint8), np.array([0], np.int32))
        steps = args.steps
        for i in range(args.warmup):
            stage.forward([req], xs[i % 8], out)
            state.truncate(P)
        torch.cuda.synchronize()

        def loop():
            for i in range(steps):
                stage.forward([req], xs[i % 8], out)
                state.truncate(P)

        t = time.perf_counter()
        loop()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t) * 1e3 / steps
        prof = _profiled(stage, loop)
        cfg = {"workload": f"llama3-70b quarter stage decode, bs=1, kv={P}", **base_cfg, "kv_len": P, "batch": 1}
        lines.append(_line("stage decode tokens/s (70B quarter-stage, bs=1)", 1e3 / ms, "tokens/s", args, steps, ms,
                           cfg, wbytes + (P + 1) * kvb, _gateup_roofline(shape, prof)))

    else:  # microbatch8b
        lens = {nr: synth.kv_lengths(nr, 128, 4096, args.seed) for nr in (2, 4, 8)}
        for nr in (2, 4, 8):
            for mode in ("decode", "mixed"):
                ns = [1] * nr if mode == "decode" else [5 if r % 2 == 0 else 1 for r in range(nr)]
                reqs, states, nbytes = [], [], wbytes
                for r in range(nr):
                    P = int(lens[nr][r])
                    st = stage.new_state(1, P + 8)
                    k, v = synth.make_kv(shape, 1, P, args.seed, r)
                    st.append(k, v)
                    del k, v
                    holes = synth.hole_mask(P, 0.1, args.seed, r)
                    holes[-1] = 1
                    mask = np.concatenate([holes, np.ones(ns[r], np.uint8)])[None]
                    pos = (int(holes.sum()) + np.arange(ns[r], dtype=np.int32))[None]
                    reqs.append((st, P, Request(st, pos, mask, None)))
                    nbytes += (P + ns[r]) * kvb
                rows = sum(ns)
                xs = [synth.make_hidden(shape, rows, args.seed, 300 + i).cuda() for i in range(4)]
                out = torch.empty_like(xs[0])

                def one(i):
                    stage.forward([q for _, _, q in reqs], xs[i % 4], out)
                    for st, P, _ in reqs:
                        st.truncate(P)

                for i in range(args.warmup):
                    one(i)
                torch.cuda.synchronize()
                t = time.perf_counter()
                for i in range(args.steps):
                    one(i)
                torch.cuda.synchronize()
                ms = (time.perf_counter() - t) * 1e3 / args.steps
                prof = _profiled(stage, lambda: [one(i) for i in range(args.steps)])
                cfg = {"workload": f"llama3.1-8b half stage micro-batch, {nr} requests, {mode} "
                                   f"(tokens per request {ns}), kv lengths {[int(x) for x in lens[nr]]}, 10% holes",
                       **base_cfg, "requests": nr, "mode": mode, "rows": rows}
                lines.append(_line(f"micro-batch steps/s (8B half-stage, {nr} requests, {mode})", 1e3 / ms, "steps/s",
                                   args, args.steps, ms, cfg, nbytes, _gateup_roofline(shape, prof),
                                   tokens_per_s=round(rows * 1e3 / ms, 1)))
                for st, _, _ in reqs:
                    st.free()
                del xs, out
    stage.device_status()
    stage.close()
    for ln in lines:
        print(json.dumps(ln), flush=True)
    return 0


def head_workload(args) -> int:
    """stage_head_top1 with the Llama-3 vocabulary on the 8B hidden size."""
    import torch

    import synth
    from paper_2608_19147_amd import Stage

    shape = synth.with_layers(synth.LLAMA8B_HALF, 1)     # the head needs only the stage's hidden size and dtypes
    stage = Stage(shape, synth.make_weights(shape, args.seed))
    V = synth.LLAMA3_VOCAB
    fn, lm = synth.make_head(shape, V, args.seed)
    stage.attach_head(fn, lm)
    del lm
    H, G = shape.hidden, shape.group_size
    head_bytes = V * (H // 2) + V * (H // G) * 2 + 2 * H    # codes + scales + final norm
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    steps = max(1, args.steps)
    lines = []
    for M in (1, 20):
        xs = [synth.make_hidden(shape, M, args.seed, 400 + i).cuda() for i in range(4)]
        for i in range(max(1, args.warmup)):
            stage.head_top1(xs[i % 4])
        torch.cuda.synchronize()
        ev[0].record()
        for i in range(steps):
            stage.head_top1(xs[i % 4])
        ev[1].record()
        ev[1].synchronize()
        ms = ev[0].elapsed_time(ev[1]) / steps
        nbytes = head_bytes + M * H * 2
        gbps = nbytes / (ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "kernel": "bprep_kernel + gemm_bp_kernel (top-1 epilogue) + top1_merge_kernel",
                "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4),
                "traffic": None, "bytes_per_launch": nbytes, "avg_launch_us": round(ms * 1e3, 3), "launches_timed": steps,
                "timed": "HIP events around the call on its stream (three kernels)"}
        cfg = {"workload": f"final-stage head: RMSNorm + INT4 lm_head {V} x {H} + top-1, {M} rows", "vocab": V,
               "hidden": H, "group_size": G, "rows": M, "act": shape.act_dtype}
        lines.append(_line(f"final-stage top-1 rows/s (LM head {V} x {H}, {M} rows)", M * 1e3 / ms, "rows/s", args,
                           steps, ms, cfg, nbytes, roof))
    del xs
    table = synth.make_embedding(shape, V, args.seed)
    stage.attach_embedding(table)
    del table
    for n in (1, 20, 2048):
        ids = [torch.from_numpy(synth.make_token_ids(V, n, args.seed, 500 + i)).cuda() for i in range(4)]
        out = torch.empty((n, H), dtype=stage.act_dtype, device="cuda")
        for i in range(max(1, args.warmup)):
            stage.embed(ids[i % 4], hidden_out=out)
        torch.cuda.synchronize()
        ev[0].record()
        for i in range(steps):
            stage.embed(ids[i % 4], hidden_out=out)
        ev[1].record()
        ev[1].synchronize()
        ms = ev[0].elapsed_time(ev[1]) / steps
        nbytes = n * (2 * H * 2 + 4)                                # rows read + rows written + ids
        gbps = nbytes / (ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "kernel": "embed_gather_kernel", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS,
                "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4), "traffic": None, "bytes_per_launch": nbytes,
                "avg_launch_us": round(ms * 1e3, 3), "launches_timed": steps,
                "timed": "HIP events around the call on its stream (one kernel)"}
        cfg = {"workload": f"first-stage embedding gather: {n} ids from a {V} x {H} table", "vocab": V, "hidden": H,
               "rows": n, "act": shape.act_dtype}
        lines.append(_line(f"first-stage embedding rows/s ({V} x {H} table, {n} ids)", n * 1e3 / ms, "rows/s", args,
                           steps, ms, cfg, nbytes, roof, dtype=shape.act_dtype))
    stage.device_status()
    stage.close()
    for ln in lines:
        print(json.dumps(ln), flush=True)
    return 0


def compact_workload(args) -> int:
    """kv_compact and kv_capture on a 4-slot 8B half-stage state (16 layers)."""
    import numpy as np
    import torch

    import synth
    from paper_2608_19147_amd import Stage

    shape = synth.LLAMA8B_HALF
    t0 = time.perf_counter()
    stage = Stage(shape, synth.make_weights(shape, args.seed))
    S, P = 4, 2368
    state = stage.new_state(S, P)
    k, v = synth.make_kv(shape, S, P, args.seed)
    state.append(k, v)
    del k, v
    full = state.capture(None, on_device=True)               # re-installs the holed state
    keep = np.stack([synth.hole_mask(P, 0.0724, args.seed, b, config_id=2) for b in range(S)])
    keep[:, 0] = 1
    kept = keep.sum(axis=1)
    row_b = shape.n_kv_heads * shape.head_dim * 2            # one of K, V: bytes of a row per layer
    L = shape.n_layers
    kept_bytes = 2 * int(kept.sum()) * L * row_b             # K and V rows kept
    pad_bytes = 2 * int((kept.max() - kept).sum()) * L * row_b
    nbytes = 2 * kept_bytes + pad_bytes                      # each kept row read once and written once, padding written
    torch.cuda.synchronize()
    print(f"# setup {time.perf_counter() - t0:.1f}s, kept rows per slot {kept.tolist()}", file=sys.stderr, flush=True)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    steps = max(1, args.steps)

    def time_compact(n):
        tot = 0.0
        for _ in range(n):
            state.restore(full)
            ev[0].record()
            state.compact(keep)
            ev[1].record()
            ev[1].synchronize()
            tot += ev[0].elapsed_time(ev[1])
        return tot / n

    def time_capture(n):
        ev[0].record()
        for _ in range(n):
            state.capture(keep, on_device=True)
        ev[1].record()
        ev[1].synchronize()
        return ev[0].elapsed_time(ev[1]) / n

    time_compact(max(1, args.warmup))
    ms_c = time_compact(steps)
    state.restore(full)
    time_capture(max(1, args.warmup))
    ms_cap = time_capture(steps)
    lines = []
    base = {"layers": L, "kv_heads": shape.n_kv_heads, "head_dim": shape.head_dim, "kv_cache": shape.kv_dtype,
            "slots": S, "kv_len": P, "kept_rows_per_slot": kept.tolist()}
    for name, ms, kern in (("kv_compact", ms_c, "kv_compact_kernel (in place, one workgroup per layer, kv head, K|V)"),
                           ("kv_capture", ms_cap, "kv_gather_rows_kernel (kept rows into a device blob)")):
        gbps = nbytes / (ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "kernel": kern, "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(gbps / HBM_PEAK_GBPS, 4), "traffic": None, "bytes_per_launch": nbytes,
                "avg_launch_us": round(ms * 1e3, 3), "launches_timed": steps,
                "timed": "HIP events around the call on its stream (metadata upload + kernels)"}
        cfg = {"workload": f"llama3.1-8b half stage {name}, {S} slots x kv {P}, ~7% masked holes", **base}
        lines.append(_line(f"{name} GB/s (8B half-stage KV state, {S} slots x {P})", gbps, "GB/s", args, steps, ms, cfg,
                           nbytes, roof))
    state.free()
    stage.close()
    for ln in lines:
        print(json.dumps(ln), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--kv", type=int, default=2048, help="KV length of the headline value")
    ap.add_argument("--kv-also", type=int, default=512, help="second KV length reported (0 = none)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-layers", type=int, default=3, help="layers of the oracle sample (0 = skip)")
    ap.add_argument("--workload", default="decode8b", choices=WORKLOADS)
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}): "
              "this build has no multi-GPU path.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import synth
    from paper_2608_19147_amd import Request, Stage

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.workload != "decode8b":
        return other_workload(args)
    shape = synth.LLAMA8B_HALF
    t0 = time.perf_counter()
    layers = synth.make_weights(shape, args.seed)
    stage = Stage(shape, layers)
    del layers
    kv_max = max(args.kv, args.kv_also)
    state = stage.new_state(1, kv_max + 8)
    k, v = synth.make_kv(shape, 1, kv_max, args.seed)
    state.append(k, v)
    del k, v
    n_in = 8
    xs = [synth.make_hidden(shape, 1, args.seed, 100 + i).cuda() for i in range(n_in)]
    out = torch.empty_like(xs[0])
    torch.cuda.synchronize()
    print(f"# setup {time.perf_counter() - t0:.1f}s (weights {stage.weight_bytes() / 1e9:.3f} GB on device)",
          file=sys.stderr, flush=True)

    def run(kv_len: int, profile):
        state.truncate(kv_len)
        req = Request(state, np.array([[kv_len]], np.int32), np.ones((1, kv_len + 1), np.uint8), np.array([0], np.int32))
        for i in range(args.warmup):
            stage.forward([req], xs[i % n_in], out)
            state.truncate(kv_len)
        torch.cuda.synchronize()
        if profile:
            stage.profile(profile)
        t_start = time.perf_counter()
        for i in range(args.steps):
            stage.forward([req], xs[i % n_in], out)
            state.truncate(kv_len)
        torch.cuda.synchronize()
        t_end = time.perf_counter()
        prof = None
        if profile:
            each = stage.profile_read_each()
            stage.profile(None)
            prof = (len(each), float(each.astype(np.float64).sum()), each)
        ms = (t_end - t_start) * 1e3 / args.steps
        return ms, prof

    # the dominant kernel: the single-launch forward when the stage uses it,
    # else the gate|up GEMV of the multi-kernel path (54% of the weight bytes)
    ms_main, prof = run(args.kv, "persistent")
    dominant = "persistent"
    if prof[0] == 0:
        ms_main, prof = run(args.kv, "gateup")
        dominant = "gateup"
    ms_also = run(args.kv_also, None)[0] if args.kv_also else None
    print(f"# decode kv={args.kv}: {ms_main:.4f} ms/step"
          + (f"; kv={args.kv_also}: {ms_also:.4f} ms/step" if ms_also else ""), file=sys.stderr, flush=True)

    b = algorithmic_bytes(shape, args.kv)
    gbps = b["total"] / (ms_main * 1e-3) / 1e9
    launches, prof_ms, each = prof
    per_launch_ms = prof_ms / max(1, launches)
    pct = np.percentile(each, [10, 50, 90]) * 1e3 if len(each) else [0.0, 0.0, 0.0]
    if dominant == "persistent":
        k_bytes, k_name = b["total"], "stage_stream_kernel (whole stage forward, one launch per step)"
    else:
        k_bytes, k_name = gateup_bytes(shape), "gemm_bp_kernel gate|up (one launch per layer)"
    k_gbps = k_bytes / (per_launch_ms * 1e-3) / 1e9
    line = {
        "metric": "stage decode tokens/s (8B half-stage, bs=1) + achieved HBM GB/s vs peak",
        "value": round(1e3 / ms_main, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_main, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "w4a16",
        "data": "synthetic",
        "config": {
            "workload": f"llama3.1-8b half stage decode, bs=1, kv={args.kv}",
            "layers": shape.n_layers, "hidden": shape.hidden, "q_heads": shape.n_q_heads,
            "kv_heads": shape.n_kv_heads, "head_dim": shape.head_dim, "ffn": shape.ffn,
            "group_size": shape.group_size, "kv_len": args.kv, "batch": 1, "act": "bf16", "kv_cache": "bf16",
        },
        "hbm_bytes_per_step": b["total"],
        "achieved_gbps": round(gbps, 1),
        "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4),
        "roofline": {
            "bound": "hbm", "kernel": k_name,
            "achieved": round(k_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(k_gbps / HBM_PEAK_GBPS, 4),
            "traffic": MEASURED_TRAFFIC.get((kernel_digest(), args.kv)) if dominant == "persistent" else None,
            "bytes_per_launch": k_bytes, "avg_launch_us": round(per_launch_ms * 1e3, 3), "launches_timed": launches,
            "launch_us_p10_median_p90": [round(float(x), 3) for x in pct],
        },
    }
    if ms_also:
        bb = algorithmic_bytes(shape, args.kv_also)
        g2 = bb["total"] / (ms_also * 1e-3) / 1e9
        line["also"] = {"kv_len": args.kv_also, "tokens_per_s": round(1e3 / ms_also, 3), "ms_per_step": round(ms_also, 5),
                        "hbm_bytes_per_step": bb["total"], "achieved_gbps": round(g2, 1),
                        "hbm_frac": round(g2 / HBM_PEAK_GBPS, 4)}
    stage.device_status()        # raises if a single-launch forward gave up waiting (its timing is void)
    state.free()
    stage.close()
    del xs, out
    torch.cuda.empty_cache()
    if args.cpu_layers > 0:
        print("# timing the fp64 oracle sample on the host", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(shape, args.kv, args.cpu_layers, args.seed)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
