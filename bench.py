#!/usr/bin/env python3
"""Throughput of the batched speculative-verify step on one MI355X.

Workload (default): the large-v3-shape bf16 decoder (32 layers, d 1280, 20 heads,
FFN 5120, vocab 51866), batch 32, k = 6 drafts, 1500 encoder frames per sequence,
committed KV lengths ~U{0..441}, drafts planted to agree with the target's greedy
continuation for a Geometric(0.25) number of positions.  Inputs are seeded synthetic
data (random-init N(0, 0.02) weights; no checkpoints or audio exist here).

A step is one pass of the whole hot path over the batch: embed, 32 decoder layers over
the paged self-KV cache and the encoder K/V, LM head + argmax, prefix accept, and the
KV commit.  Each timed step starts from the same committed state (the commit's length
update is undone by a 128-byte device copy after the step) so every step does the same
work.  value = emitted tokens per step (accepted drafts + the bonus token, summed over
the batch) / step time.

The same line also carries: the dominant kernel's roofline (cross-attention), the oracle
CPU baseline, the anchor readout, draft, tree and AnchorDraft-objective costs, the encoder
K/V prefill, the measured copy / read rates, the ragged batch of 64 in both row layouts,
the drift-stress decode loop end to end (tokens/s, mean accepted length, s_1..s_8) and the
tiny float32 model's step and decode round.

Prints one JSON line (N = 1 only: the step is measured on one GPU).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--config", default="large_v3_bf16",
                   choices=["large_v3_bf16", "small_bf16", "ragged_large_v3"])
    p.add_argument("--layout", default="padded", choices=["padded", "packed"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-kernel-profile", action="store_true")
    p.add_argument("--anchor-layer", type=int, default=-2,
                   help="also time the step with the verification-attention anchor readout at "
                        "this layer (-2: three quarters of the depth; -1: skip)")
    p.add_argument("--draft-steps", type=int, default=6,
                   help="also time this many audio-conditioned draft steps per round (0: skip)")
    p.add_argument("--tree", type=int, default=1,
                   help="also time a draft-tree step (the 11-node tree) with its commit")
    p.add_argument("--loss", type=int, default=1,
                   help="also time the AnchorDraft objective with its gradients at a training "
                        "batch of the draft (12 utterances x 128 positions)")
    p.add_argument("--graph", type=int, default=1,
                   help="also time the step replayed from a captured HIP graph (reported beside "
                        "the eager step, which is the headline)")
    p.add_argument("--workloads", type=int, default=1,
                   help="also measure the ragged batch (padded and packed), the drift-stress "
                        "loop and the tiny float32 model, and time the encoder K/V prefill")
    p.add_argument("--copy-calibration-mb", type=int, default=0,
                   help="after the timed steps, copy a buffer of this many MiB once (a plain "
                        "copy of known size that calibrates HBM byte counters)")
    return p.parse_args()


def gpu_greedy_continuation(sess, t0, ks):
    """The target's own greedy tokens y_1..y_k per sequence, by repeated verification:
    once d_1..d_i equal the greedy tokens, row i's argmax is the next one."""
    B = len(t0)
    drafts = [np.zeros(int(k), np.int64) for k in ks]
    for it in range(int(max(ks))):
        sess.step([np.concatenate([[t0[b]], drafts[b]]) for b in range(B)])
        g = sess.results()["greedy"]
        for b in range(B):
            if it < ks[b]:
                drafts[b][it] = g[sess.row_of(b, it)]
    return drafts


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "cross_attn_{}_traffic.json")


def measured_traffic(workload: str):
    """HBM bytes per cross-attention launch from the committed FETCH_SIZE / WRITE_SIZE
    counter runs (copy-calibrated), or None if there are none for this workload or the
    kernel's sources changed since they were taken."""
    from paper_2608_12703_amd.roofline import kernel_source_hash
    path = TRAFFIC_FILE.format(workload)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("source_sha256") != kernel_source_hash():
        log("counter traffic is stale (kernel sources changed); traffic = null")
        return None
    return rec["hbm_bytes_per_launch"]


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def host_threads() -> int:
    """CPU threads this process may use (the box's share, not the machine's count)."""
    env = os.environ.get("OMP_NUM_THREADS")
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    return min(n, int(env)) if env and env.isdigit() and int(env) > 0 else n


def cpu_baseline(cfg, params, wl, n_seq=8):
    """The oracle, untuned, on a bounded sample of the workload: the verify step of each of
    sequences 0 .. n_seq-1 (their k+1 rows each), timed with BLAS threads = the host
    threads this process may use, then sequence 0's step again with one thread.  Each
    sequence's encoder K/V projection and the greedy continuation that plants its drafts
    are computed first and not timed, as on the GPU (they take about 6 s per sequence
    at this shape, which is what bounds the sample).  The same steps are then timed
    again with one BLAS thread."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import decoder as od
    from paper_2608_12703_amd import synth
    model = od.Model(cfg, params)
    threads = host_threads()
    states = []
    t0 = time.perf_counter()
    with threadpool_limits(limits=threads):
        used = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        for b in range(n_seq):
            cross = od.cross_kv(model, synth.make_encoder(cfg, b, int(wl.T[b])))
            st = od.new_state(model, cross, int(wl.t0[b]), synth.make_prefix_kv(cfg, b, int(wl.n[b])))
            y, _, _ = od.ar_decode(model, st, int(wl.k[b]))
            states.append((st, synth.plant_drafts(np.array(y), int(wl.G[b]), wl.fill_ne[b], wl.fill_any[b])))
        setup = time.perf_counter() - t0
        tokens, rows = 0, 0
        t1 = time.perf_counter()
        for st, d in states:
            r = od.verify(model, st, d)
            tokens += r.accepted + 1
            rows += len(d) + 1
        timed = time.perf_counter() - t1
    with threadpool_limits(limits=1):
        t2 = time.perf_counter()
        for st, d in states:
            od.verify(model, st, d)
        one = time.perf_counter() - t2
    return {"value": tokens / timed, "unit": "accepted tokens/s", "cores": int(used), "kind": "oracle",
            "cpu_model": cpu_model(),
            "one_thread": {"value": tokens / one, "seconds": round(one, 2), "sample": "the same steps"},
            "sample": f"the verify steps of sequences 0..{n_seq - 1} of the {wl.batch} (a quarter of the "
                      f"batch; {rows} rows, {tokens} tokens) in {timed:.1f} s with {used} BLAS threads "
                      f"(encoder K/V projection and draft planting, {setup:.1f} s, not timed)"}


def copy_peaks(mib=1024, reps=5):
    """Measured HBM rate on this GPU: a device copy of `mib` MiB (read + write bytes per
    second), the best of `reps`."""
    import torch
    n = (mib << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    best_c = 1e9
    for _ in range(reps):
        ev0.record()
        dst.copy_(src)
        ev1.record()
        torch.cuda.synchronize()
        best_c = min(best_c, ev0.elapsed_time(ev1))
    nbytes = n * 4
    del src, dst
    return {"copy_GBps": round(2 * nbytes / (best_c / 1e3) / 1e9, 1),
            "what": f"best of {reps}: device copy of {mib} MiB, read + write bytes"}


def time_prefill(sess, encs, reps=3):
    """The encoder K/V projection of the whole batch (setup, once per utterance): ms per
    call and the matrix-core rate against the dense bf16 peak (2 frames_cap 2d d flop per
    layer; padded frame slots are computed too)."""
    import torch

    from paper_2608_12703_amd import ad, roofline
    enc = sess.upload_encoder(encs)
    ad.cross_kv_prefill(sess.model, enc, sess.cross_struct())
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(reps):
        ad.cross_kv_prefill(sess.model, enc, sess.cross_struct())
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / reps
    cfg = sess.cfg
    flops = 2.0 * sess.frames_cap * 2 * cfg.d_model * cfg.d_model * cfg.n_layers
    del enc
    return {"ms_per_batch": round(ms, 3), "utterances": sess.B, "frames_cap": sess.frames_cap,
            "tflops": round(flops / (ms / 1e3) / 1e12, 1),
            "mfma_frac": round(flops / (ms / 1e3) / roofline.BF16_MFMA_PEAK, 4)}


def planted_session(cfg, params, wl, layout):
    """A session over workload wl with drafts planted on the GPU's own greedy
    continuation (Geometric agreement), prepared and ready to step."""
    from paper_2608_12703_amd import ad, synth
    from paper_2608_12703_amd.harness import Session
    sess = Session(cfg, params, wl.batch, int(wl.k.max()), wl.T, layout=layout,
                   packed_encoder=layout == ad.AD_PACKED)
    sess.prefill_encoder([synth.make_encoder(cfg, b, int(wl.T[b])) for b in range(wl.batch)])
    for b in range(wl.batch):
        sess.import_prefix(b, synth.make_prefix_kv(cfg, b, int(wl.n[b])))
    sess.set_kv_len(wl.n)
    y = gpu_greedy_continuation(sess, wl.t0, wl.k)
    blocks = [np.concatenate([[wl.t0[b]],
                              synth.plant_drafts(y[b], int(wl.G[b]), wl.fill_ne[b], wl.fill_any[b])])
              for b in range(wl.batch)]
    sess.prepare(blocks)
    return sess, blocks, y


def time_steps(sess, steps, warmup):
    """ms per step of the prepared block (verify + commit, each from the same committed
    state) with HIP events; the accept lengths of the last step."""
    import torch
    kv0 = sess.kv_len.clone()

    def one():
        sess.run()
        sess.commit()
        sess.kv_len.copy_(kv0)

    for _ in range(warmup):
        one()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(steps):
        one()
    ev1.record()
    torch.cuda.synchronize()
    res = sess.results()
    assert res["err"] == 0, f"device error flag {res['err']}"
    return ev0.elapsed_time(ev1) / steps, res


def measure_ragged(params_dev, steps, warmup):
    """The ragged large-v3 batch (64 sequences, k 2..8, 200..1500 frames, committed
    lengths 0..447-k) in both row layouts; both are charged the same algorithmic bytes."""
    import torch

    from paper_2608_12703_amd import ad, roofline, synth
    from paper_2608_12703_amd.configs import CONFIGS
    cfg = CONFIGS["ragged_large_v3"]
    wl = synth.make_step_workload(cfg)
    sb = roofline.step_bytes(cfg, wl.n, wl.T, wl.k)
    out = {"batch": wl.batch, "k": [int(wl.k.min()), int(wl.k.max())],
           "frames": [int(wl.T.min()), int(wl.T.max())], "step_hbm_bytes": sb["total"]}
    accepts = []
    for name, layout in (("padded", ad.AD_PADDED), ("packed", ad.AD_PACKED)):
        sess, _, _ = planted_session(cfg, params_dev, wl, layout)
        ms, res = time_steps(sess, steps, warmup)
        tokens = int(np.sum(res["accept_len"] + 1))
        accepts.append(res["accept_len"])
        out[name] = {"ms_per_step": round(ms, 4), "value": round(tokens / (ms / 1e3), 1),
                     "rows": sess.rows, "tokens_per_step": tokens,
                     "step_hbm_frac": round(sb["total"] / (ms / 1e3) / roofline.HBM_PEAK, 4)}
        log(f"ragged {name}: {ms:.3f} ms/step, {sess.rows} rows, {tokens} tokens/step")
        del sess
        torch.cuda.empty_cache()
    assert np.array_equal(accepts[0], accepts[1]), "padded and packed layouts disagree"
    return out


def measure_drift(params_dev):
    """The drift-stress loop (batch 32, k 8, 1500 frames): every sequence decodes from the
    start token to the last position (447 tokens) with drafts planted on the target's own
    greedy continuation and misaligned by +-1 token after Poisson(40)-spaced anchors.
    Timed end to end: the host plants each round's drafts, the step verifies, commits and
    returns the accept lengths (one host round trip per round).  The greedy continuation
    itself comes from an untimed autoregressive pass first."""
    import torch

    from paper_2608_12703_amd import decode, synth
    from paper_2608_12703_amd.configs import CONFIGS, MAX_POS, SOT_TOKEN
    from paper_2608_12703_amd.harness import Session
    cfg = CONFIGS["drift_stress"]
    B, K, T = cfg.batch, cfg.k, cfg.frames
    sess = Session(cfg, params_dev, B, K, [T] * B)
    sess.prefill_encoder([synth.make_encoder(cfg, b, T) for b in range(B)])
    sess.set_kv_len(np.zeros(B, np.int64))
    n_tok = MAX_POS - 1
    ys = np.full((B, n_tok + 1), SOT_TOKEN, np.int64)
    pend = [SOT_TOKEN] * B
    for p in range(1, n_tok + 1):
        sess.step([np.array([t], np.int64) for t in pend], commit=True)
        out = sess.out_tokens[:, 0].cpu().numpy()
        ys[:, p] = out
        pend = [int(t) for t in out]
    plans = [synth.make_drift_plan(cfg, b) for b in range(B)]
    ks = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    toks, acc, rounds = decode.decode_with_drift(sess, list(ys), plans, K, n_tok, ks_out=ks)
    wall = time.perf_counter() - t0
    assert all(list(t) == list(ys[b, 1:len(t) + 1]) for b, t in enumerate(toks)), "loop not lossless"
    a, k = np.array(acc), np.array(ks)
    live = k >= 0
    full = k == K
    s = [float(np.mean(a[full] >= j)) for j in range(1, K + 1)]
    emitted = sum(len(t) for t in toks)
    log(f"drift stress: {rounds} rounds, {emitted} tokens in {wall:.2f} s")
    del sess
    torch.cuda.empty_cache()
    return {"batch": B, "k": K, "tokens": emitted, "rounds": rounds, "seconds": round(wall, 3),
            "value": round(emitted / wall, 1), "unit": "accepted tokens/s",
            "ms_per_round": round(1e3 * wall / rounds, 3),
            "mean_accepted_length": round(float(np.mean(a[live])), 4),
            "tokens_per_round": round(float(np.mean(a[live] + 1)), 4),
            "s_k": [round(x, 4) for x in s], "L": round(sum(s), 4),
            "rounds_with_full_block": int(np.sum(full))}


def measure_tiny(steps):
    """The tiny float32 model (4 layers, d 384, vocab 51865), batch 1: the 64-token greedy
    decode with 4 linear draft heads (rounds of verify, commit and ad_draft_heads), and
    one verify step of a 5-row block alone."""
    import torch

    from paper_2608_12703_amd import ad, decode, synth
    from paper_2608_12703_amd.configs import CONFIGS, SOT_TOKEN
    from paper_2608_12703_amd.harness import Session, upload
    cfg = CONFIGS["tiny_fp32"]
    params = synth.make_params(cfg)
    heads = upload(synth.make_draft_heads(cfg), torch.float32)
    wl = synth.make_step_workload(cfg)
    T = int(wl.T[0])
    sess = Session(cfg, params, 1, cfg.draft_heads, [T])
    sess.prefill_encoder([synth.make_encoder(cfg, 0, T)])
    sess.set_kv_len([0])
    decode.decode_with_heads(sess, heads, [SOT_TOKEN], cfg.decode_tokens)   # warm
    sess.set_kv_len([0])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    toks, acc, _, rounds = decode.decode_with_heads(sess, heads, [SOT_TOKEN], cfg.decode_tokens)
    wall = time.perf_counter() - t0
    sess.set_kv_len([0])
    sess.prepare([np.array([SOT_TOKEN] + [int(x) for x in wl.fill_any[0]], np.int64)])
    ms, _ = time_steps(sess, steps, 3)
    return {"us_per_step": round(ms * 1e3, 2), "rows": sess.rows,
            "decode_tokens": cfg.decode_tokens, "rounds": rounds,
            "us_per_round_end_to_end": round(1e6 * wall / rounds, 1),
            "accepted_per_round": round(float(np.mean([int(a[0]) for a in acc[1:]])), 4)}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the verify step is measured on one GPU; --gpus must be 1 "
                                   "(sequences are independent: several GPUs would each run their "
                                   "own sequences with a weight replica and no exchange)"}))
        sys.exit(2)
    import torch

    from paper_2608_12703_amd import ad, roofline, synth
    from paper_2608_12703_amd.configs import CONFIGS
    from paper_2608_12703_amd.harness import Session

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    cfg = CONFIGS[args.config]
    layout = ad.AD_PADDED if args.layout == "padded" else ad.AD_PACKED
    t_setup = time.perf_counter()
    log(f"generating {cfg.name} inputs")
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    sess = Session(cfg, params, wl.batch, int(wl.k.max()), wl.T, layout=layout,
                   packed_encoder=layout == ad.AD_PACKED)
    params_dev = sess.params          # device parameters, shared by the later sessions
    log("encoder K/V prefill")
    encs = [synth.make_encoder(cfg, b, int(wl.T[b])) for b in range(wl.batch)]
    sess.prefill_encoder(encs)
    for b in range(wl.batch):
        sess.import_prefix(b, synth.make_prefix_kv(cfg, b, int(wl.n[b])))
    sess.set_kv_len(wl.n)
    torch.cuda.synchronize()
    log("planting drafts on the target's greedy continuation")
    y = gpu_greedy_continuation(sess, wl.t0, wl.k)
    blocks = [np.concatenate([[wl.t0[b]],
                              synth.plant_drafts(y[b], int(wl.G[b]), wl.fill_ne[b], wl.fill_any[b])])
              for b in range(wl.batch)]
    sess.prepare(blocks)
    kv0 = sess.kv_len.clone()
    torch.cuda.synchronize()
    log(f"setup {time.perf_counter() - t_setup:.1f} s; warmup {args.warmup}, timed {args.steps}")

    def one_step():
        sess.run()
        sess.commit()
        sess.kv_len.copy_(kv0)

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    res = sess.results()
    assert res["err"] == 0, f"device error flag {res['err']}"
    tokens = int(np.sum(res["accept_len"] + 1))
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        one_step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = ev0.elapsed_time(ev1) / args.steps
    res2 = sess.results()
    assert np.array_equal(res2["accept_len"], res["accept_len"]), "steps were not repeatable"
    log(f"{ms:.3f} ms/step (wall {1e3 * wall / args.steps:.3f}), {tokens} tokens/step")
    ms_eager, ms_graph = ms, None
    if args.graph:
        # The same step (verify, commit, length reset) captured once into a HIP graph and
        # replayed: the same kernels with the same arguments, launched by the graph
        # instead of one host call each.  Every replay's accept lengths, tokens and hidden
        # rows must equal the eager step's.
        ref_hidden = res2["hidden"].copy()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            one_step()
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(args.steps):
            graph.replay()
        ev1.record(stream)
        torch.cuda.synchronize()
        ms_graph = ev0.elapsed_time(ev1) / args.steps
        res3 = sess.results()
        assert np.array_equal(res3["accept_len"], res["accept_len"])
        assert np.array_equal(res3["out_tokens"], res2["out_tokens"])
        assert np.array_equal(res3["hidden"].view(np.uint32), ref_hidden.view(np.uint32))
        log(f"graph-launched: {ms_graph:.3f} ms/step (eager {ms_eager:.3f})")
        del graph

    sb = roofline.step_bytes(cfg, wl.n, wl.T, wl.k)
    rows = sess.rows
    roof = None
    if not args.no_kernel_profile:
        # The dominant kernel, timed with HIP events on the step's stream over the same
        # steps.  An event between two kernels delays the next kernel's start by the
        # launch latency the stream otherwise hides, so events around the kernel alone
        # overstate it; two passes bracket the kernel before it (the cross-attention
        # query projection) with and without the cross-attention kernel, and the
        # difference of the means is the kernel by itself.
        means = {}
        for kind in (ad.PROF_XQ_CROSS, ad.PROF_XQ):
            ad.profile_enable(sess.model, kind, cfg.n_layers * args.steps)
            for _ in range(args.steps):
                one_step()
            tot, n_launch = ad.profile_read(sess.model)
            means[kind] = tot / n_launch
        ad.profile_enable(sess.model, ad.PROF_XQ, 0)
        per_launch_s = (means[ad.PROF_XQ_CROSS] - means[ad.PROF_XQ]) / 1e3
        lb = roofline.cross_attn_launch_bytes(cfg, wl.T, rows)
        achieved = lb / per_launch_s / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": 8000.0, "unit": "GB/s",
                "frac": round(achieved / 8000.0, 4), "traffic": measured_traffic(cfg.name),
                "kernel": "cross_attn", "launch_bytes": lb,
                "launch_us": round(per_launch_s * 1e6, 2), "launches_timed": n_launch}
        log(f"cross-attention: {per_launch_s * 1e6:.1f} us/launch, {achieved:.0f} GB/s")

    anchor = None
    if args.anchor_layer != -1:
        # The same steps with the anchor readout after the accept scan: its two kernels
        # timed with an event pair, and the step-time difference.
        layer = 3 * cfg.n_layers // 4 if args.anchor_layer < -1 else args.anchor_layer
        sess.anchor_layer = layer
        sess.prepare(blocks)
        for _ in range(args.warmup):
            one_step()
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(args.steps):
            one_step()
        ev1.record(stream)
        torch.cuda.synchronize()
        ms_a = ev0.elapsed_time(ev1) / args.steps
        ad.profile_enable(sess.model, ad.PROF_ANCHOR, args.steps)
        for _ in range(args.steps):
            one_step()
        tot, n_launch = ad.profile_read(sess.model)
        ad.profile_enable(sess.model, ad.PROF_ANCHOR, 0)
        ra = sess.results()
        assert np.array_equal(ra["accept_len"], res["accept_len"]) and np.all(ra["anchor"] >= 0)
        key_bytes = int(np.sum(wl.T)) * cfg.d_model * roofline.elem_bytes(cfg)
        us = tot / n_launch * 1e3
        anchor = {"layer": layer, "us_per_step_events": round(us, 2),
                  "us_per_step_delta": round((ms_a - ms) * 1e3, 2), "key_bytes": key_bytes,
                  "achieved_GBps": round(key_bytes / (us * 1e-6) / 1e9, 1)}
        log(f"anchor readout at layer {layer}: {us:.1f} us/step (events), "
            f"{(ms_a - ms) * 1e3:.1f} us/step (step difference)")
        sess.anchor_layer = -1
        sess.prepare(blocks)

    draft = None
    if args.draft_steps > 0:
        # The audio-conditioned draft block (random-init, one layer, d_ffn = 2 d) after a
        # target step that also reads the anchor and the draft's taps; rho = one draft
        # step's time over one verify step's time.
        from paper_2608_12703_amd import decode
        K = args.draft_steps
        L = cfg.n_layers
        sess.anchor_layer = 3 * L // 4
        sess.tap_layers = tuple(max(0, L * i // 4 - 1) for i in (1, 2, 3))
        sess.out_taps = torch.empty(3, sess.max_rows, cfg.d_model, dtype=torch.float32, device="cuda")
        sess.prepare(blocks)
        one_step()
        runner = decode.DraftRunner(sess, synth.make_draft_params(cfg))
        runner.prefill_encoder([synth.make_encoder(cfg, b, int(wl.T[b])) for b in range(wl.batch)])
        for _ in range(2):
            runner.round(K)
        torch.cuda.synchronize()
        rounds = max(1, args.steps // 2)
        ev0.record(stream)
        for _ in range(rounds):
            runner.round(K)
        ev1.record(stream)
        torch.cuda.synchronize()
        us = ev0.elapsed_time(ev1) / (rounds * K) * 1e3
        draft = {"draft_steps_per_round": K, "us_per_draft_step": round(us, 2),
                 "rho": round(us / (ms * 1e3), 4), "layers": 1, "d_ffn": 2 * cfg.d_model,
                 "cross_window_frames": 2 * decode.HALF_WINDOW + 1}
        log(f"draft step: {us:.1f} us (rho = {us / (ms * 1e3):.4f})")
        sess.anchor_layer, sess.tap_layers, sess.out_taps = -1, (-1, -1, -1), None
        sess.prepare(blocks)
        del runner

    tree = None
    if args.tree:
        # Draft-tree verification of an 11-node tree per sequence (root 0 -> 1, 2, 3;
        # 1 -> 4, 5; 2 -> 6; 4 -> 7, 8; 6 -> 9; 7 -> 10) with its commit (the accepted
        # path's keys / values moved to consecutive slots).  The greedy continuation is
        # planted along the deepest path 0-1-4-7-10 to the same depth as the chain
        # workload's planted acceptance, so both emit the same tokens per step.
        parents = [-1, 0, 0, 0, 1, 1, 2, 4, 4, 6, 7]
        deep = [1, 4, 7, 10]
        del sess
        torch.cuda.empty_cache()
        ts = Session(cfg, params, wl.batch, len(parents) - 1, wl.T, layout=layout,
                     packed_encoder=layout == ad.AD_PACKED)
        ts.prefill_encoder([synth.make_encoder(cfg, b, int(wl.T[b])) for b in range(wl.batch)])
        for b in range(wl.batch):
            ts.import_prefix(b, synth.make_prefix_kv(cfg, b, int(wl.n[b])))
        ts.set_kv_len(wl.n)
        tblocks = []
        for b in range(wl.batch):
            tok = np.array([wl.t0[b]] + [wl.fill_any[b][i % len(wl.fill_any[b])] if len(wl.fill_any[b])
                                         else 0 for i in range(len(parents) - 1)], np.int64)
            acc_b = int(res["accept_len"][b])
            for j, u in enumerate(deep[: min(acc_b, len(deep))]):
                tok[u] = y[b][j]
            tblocks.append(tok)
        ts.prepare(tblocks, parents=[parents] * wl.batch)
        kt0 = ts.kv_len.clone()

        def tree_step():
            ts.run()
            ts.commit()
            ts.kv_len.copy_(kt0)

        for _ in range(args.warmup):
            tree_step()
        torch.cuda.synchronize()
        rt = ts.results()
        assert rt["err"] == 0, f"device error flag {rt['err']}"
        ev0.record(stream)
        for _ in range(args.steps):
            tree_step()
        ev1.record(stream)
        torch.cuda.synchronize()
        ms_t = ev0.elapsed_time(ev1) / args.steps
        t_tokens = int(np.sum(rt["accept_len"] + 1))
        tree = {"nodes": len(parents), "depth": 4, "ms_per_step": round(ms_t, 4),
                "tokens_per_step": t_tokens, "value": round(t_tokens / (ms_t / 1e3), 1),
                "step_ratio_vs_chain": round(ms_t / ms, 4), "rows": ts.rows}
        log(f"tree step ({len(parents)} nodes): {ms_t:.3f} ms, {t_tokens} tokens/step")
        del ts

    loss = None
    if args.loss:
        # The AnchorDraft objective (token cross-entropy + 0.5 smooth-L1 feature term +
        # lambda x alignment cross-entropy) and its gradients for the logits, the features
        # and the first draft layer's query rows, over a training batch of 12 utterances
        # (the paper's batch size) x 128 positions of the large-v3-shape draft block.
        # Inputs are synthetic: query rows, centres (about 10% unaligned), next tokens,
        # logits and features; the draft's cross keys come from its own prefill.
        LB, LR = 12, 128
        dcfg = synth.draft_config(cfg)
        dparams = synth.make_draft_params(cfg)
        dp = {n: dparams[n] for n, _ in synth.param_specs(dcfg) if n not in ("tok_emb", "pos_emb")}
        dp["tok_emb"], dp["pos_emb"] = params["tok_emb"], params["pos_emb"]
        Ts = [int(t) for t in wl.T[:LB]]
        ls = Session(dcfg, dp, LB, 0, Ts)
        ls.prefill_encoder([synth.make_encoder(cfg, b, Ts[b]) for b in range(LB)])
        g = np.random.default_rng(17)
        LM, d, V = LB * LR, dcfg.d_model, dcfg.vocab
        dev = "cuda"
        f32 = dict(dtype=torch.float32, device=dev)
        xq = torch.randn(LM, d, generator=torch.Generator(device=dev).manual_seed(1), **f32) * 8
        cen = np.concatenate([g.integers(0, T, LR) for T in Ts])
        cen[g.random(LM) < 0.1] = -1
        center = torch.tensor(cen, dtype=torch.int32, device=dev)
        targets = torch.tensor(g.integers(0, V, LM), dtype=torch.int32, device=dev)
        logits = torch.randn(LM, V, generator=torch.Generator(device=dev).manual_seed(2), **f32) * 3
        feat = torch.randn(LM, d, generator=torch.Generator(device=dev).manual_seed(3), **f32)
        feat_t = torch.randn(LM, d, generator=torch.Generator(device=dev).manual_seed(4), **f32)
        terms, row = torch.zeros(4, **f32), torch.zeros(LM, **f32)
        dxq, dlog, dfeat = torch.empty_like(xq), torch.empty_like(logits), torch.empty_like(feat)
        lerr = torch.zeros(1, dtype=torch.int32, device=dev)
        lws = torch.empty(ad.anchordraft_loss_workspace_size(ls.model, LB, LR), dtype=torch.uint8,
                          device=dev)

        def loss_call():
            ad.anchordraft_loss(ls.model, ls.cross_struct(), 0, LB, LR, xq, center, 5.0, 0.1, logits,
                                targets, feat, feat_t, terms, row, dxq, dlog, dfeat, lerr, lws)

        for _ in range(args.warmup):
            loss_call()
        torch.cuda.synchronize()
        assert int(lerr.item()) == 0 and bool(torch.isfinite(terms).all())
        ev0.record(stream)
        for _ in range(args.steps):
            loss_call()
        ev1.record(stream)
        torch.cuda.synchronize()
        us_l = ev0.elapsed_time(ev1) / args.steps * 1e3
        key_bytes = sum(Ts) * dcfg.n_heads * 64 * 2
        lbytes = (2 * LM * V * 4 + key_bytes + 2 * LM * d * 4 + 3 * LM * d * 4 + LM * 12)
        loss = {"batch": LB, "positions": LR, "frames": Ts, "us_per_call": round(us_l, 2),
                "algorithmic_bytes": lbytes, "achieved_GBps": round(lbytes / (us_l * 1e-6) / 1e9, 1),
                "terms": [round(float(x), 5) for x in terms.tolist()]}
        log(f"AnchorDraft objective + gradients: {us_l:.1f} us ({lbytes / (us_l * 1e-6) / 1e9:.0f} GB/s)")
        del ls, xq, logits, dlog

    prefill = ragged = drift = tiny = peaks = None
    if args.workloads and cfg.name == "large_v3_bf16":   # the other workloads share its weights
        torch.cuda.empty_cache()
        ps = Session(cfg, params_dev, wl.batch, int(wl.k.max()), wl.T, layout=layout,
                     packed_encoder=layout == ad.AD_PACKED)
        prefill = time_prefill(ps, encs)
        log(f"encoder K/V prefill: {prefill['ms_per_batch']:.2f} ms per batch of {wl.batch} "
            f"({prefill['tflops']:.0f} TFLOP/s)")
        del ps
        torch.cuda.empty_cache()
        ragged = measure_ragged(params_dev, args.steps, args.warmup)
        drift = measure_drift(params_dev)
        tiny = measure_tiny(max(args.steps, 50))
        log(f"tiny float32: {tiny['us_per_step']:.1f} us per verify step, "
            f"{tiny['us_per_round_end_to_end']:.1f} us per decode round")
        peaks = copy_peaks()
        log(f"device copy {peaks['copy_GBps']:.0f} GB/s")
    del encs

    if args.copy_calibration_mb:
        n = args.copy_calibration_mb << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copied {args.copy_calibration_mb} MiB (counter calibration)")
        del src, dst

    cpu = None
    if not args.no_cpu_baseline:
        log("oracle CPU baseline (eight sequences' verify steps after their setup, about a minute)")
        cpu = cpu_baseline(cfg, params, wl)
        log(f"oracle: {cpu['value']:.3f} tokens/s")

    # The paper's break-even rule for the runtime correction (section "Correction and
    # Cost"): a round of K draft steps costs about 1 + K rho verify steps; reading the
    # anchor adds Delta C_corr, which pays when the accepted length grows by at least
    # Delta L / (1 + L) >= Delta C_corr / (1 + K rho).
    break_even = None
    if anchor is not None and draft is not None:
        dc = max(anchor["us_per_step_delta"], 0.0) / (ms * 1e3)
        K = draft["draft_steps_per_round"]
        break_even = {"K": K, "rho": draft["rho"], "delta_c_corr": round(dc, 5),
                      "min_relative_length_gain": round(dc / (1 + K * draft["rho"]), 5)}

    out = {
        "metric": "accepted tokens/s, large-v3-shape spec-verify step (bf16); % of HBM roofline",
        "value": round(tokens / (ms / 1e3), 1),
        "unit": "accepted tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "graph_ms_per_step": None if ms_graph is None else round(ms_graph, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": cfg.name, "batch": wl.batch, "k": int(wl.k.max()),
                   "frames": int(np.max(wl.T)), "layers": cfg.n_layers, "d_model": cfg.d_model,
                   "layout": args.layout, "tokens_per_step": tokens, "rows": rows},
        "step_hbm_bytes": sb["total"],
        "step_hbm_frac": round(sb["total"] / (ms / 1e3) / roofline.HBM_PEAK, 4),
        "roofline": roof,
        "cpu_baseline": cpu,
        "hbm_measured": peaks,
        "prefill": prefill,
        "ragged": ragged,
        "drift_stress": drift,
        "tiny_fp32": tiny,
        "anchor_readout": anchor,
        "draft_step": draft,
        "tree_step": tree,
        "anchordraft_loss": loss,
        "break_even": break_even,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
