"""Latency versus concurrency (the shape of the paper's Section 3
experiment, Figure 2): C users each submit one recording at a random moment
of the first second; a recording of 15-120 s is cut into 3-30 s segments
(synth.recording). The same engine then serves the round two ways:

* sequential: recordings one after another in submission order, each as one
  batch (whisper_batch_transcribe of its segments), a recording starting when
  both it has arrived and the previous one has finished;
* multiplexed: every user's segments in the central queue, continuous
  batching with real-time admission (whisper_batch_serve), the paper's
  method.

A recording's latency is the completion of its last segment minus its
submission. Reports p90 latency per (concurrency, duration bucket) for both
ways, and checks that both produce identical tokens for every segment.

    python -m paper_2507_01021_amd.replay [--model large-v3] [--rounds 2]

With --policies it instead serves the turbo-u64-q512 queue (64 users,
Poisson arrivals, 512 segments of 16-224 tokens, 128 slots) in real time,
its arrival times compressed by several factors to load the GPU from light
to beyond capacity, once with continuous batching (arrival order, refill
threshold 16) and with the dynamic policy (shorter segments first with
aging; refills held back, for at most a wait bound, until 16 segments are
queued) at two wait bounds, reporting segment latency percentiles, the
makespan and the engine's pass and step counts, and checking that every
policy gives identical tokens.
"""
from __future__ import annotations

import argparse
import json
import sys
import time

import numpy as np

from . import binding, synth

BUCKETS = [(15, 30), (30, 45), (45, 60), (60, 75), (75, 90), (90, 105), (105, 120)]
MODELS = {"large-v3": synth.LARGE_V3, "turbo": synth.TURBO, "small": synth.SMALL, "base": synth.BASE}


def make_round(shape, rng, C, lo, hi, first_id):
    recs = []
    for u in range(C):
        t_us = int(rng.uniform(0.0, 1e6))
        segs = synth.recording(shape, rng, float(rng.uniform(lo, hi)), u, first_id, arrival_us=t_us)
        first_id += len(segs)
        recs.append((t_us, segs))
    return recs, first_id


def run_sequential(ctx, recs, dev):
    """Recordings in submission order, each alone; returns per-recording
    latency (s) and tokens per segment id."""
    import torch
    order = sorted(range(len(recs)), key=lambda k: (recs[k][0], k))
    t_free = 0.0
    lat = [0.0] * len(recs)
    toks = {}
    for k in order:
        arrive = recs[k][0] / 1e6
        segs = recs[k][1]
        ptrs = [dev[s.segment_id].data_ptr() for s in segs]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        res = ctx.transcribe(segs, device_audio=ptrs)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        start = max(arrive, t_free)
        t_free = start + dt
        lat[k] = t_free - arrive
        for s, r in zip(segs, res):
            toks[s.segment_id] = r["tokens"]
    return lat, toks


def run_multiplexed(ctx, recs, dev):
    import torch
    segs = [s for _, ss in recs for s in ss]
    ptrs = [dev[s.segment_id].data_ptr() for s in segs]
    torch.cuda.synchronize()
    res = ctx.transcribe(segs, device_audio=ptrs, realtime=True)
    fin = {s.segment_id: r["finish_us"] / 1e6 for s, r in zip(segs, res)}
    toks = {s.segment_id: r["tokens"] for s, r in zip(segs, res)}
    lat = [max(fin[s.segment_id] for s in ss) - t / 1e6 for t, ss in recs]
    return lat, toks


def policies(step_cost_us=1500, factors=(8, 16, 32), waits_ms=(50, 150)):
    import copy
    import torch

    shape, segs0, slots = synth.workload("turbo-u64-q512")
    blob = synth.pack_blob(synth.make_weights(shape, 0))
    ctxs = {"continuous": binding.Context(blob, max_slots=slots, max_encode_batch=32)}
    for w in waits_ms:
        ctxs[f"dynamic-wait{w}ms"] = binding.Context(blob, max_slots=slots, max_encode_batch=32, batch_policy=1,
                                                     step_cost_us=step_cost_us, max_wait_ms=w)
    del blob
    dev = [torch.from_numpy(s.audio).to("cuda:0") for s in segs0]
    ptrs = [t.data_ptr() for t in dev]
    audio_s = sum(s.seconds for s in segs0)
    for ctx in ctxs.values():   # warm-up (graph capture per row count)
        ctx.transcribe(segs0, device_audio=ptrs)
    rows = []
    for f in factors:
        segs = [copy.copy(s) for s in segs0]
        for s in segs:
            s.arrival_us = s.arrival_us // f
        span = max(s.arrival_us for s in segs) / 1e6
        toks = {}
        for name, ctx in ctxs.items():
            for _ in range(2):  # the first pass also captures graphs for row counts not seen before
                torch.cuda.synchronize()
                ctx.stats(reset=True)
                res = ctx.transcribe(segs, device_audio=ptrs, realtime=True)
            st = ctx.stats()
            lat = np.array([(r["finish_us"] - s.arrival_us) / 1e6 for s, r in zip(segs, res)])
            toks[name] = [r["tokens"] for r in res]
            row = {"arrivals_over_s": round(span, 2), "offered_audio_s_per_s": round(audio_s / span, 1),
                   "policy": name, "latency_mean_s": round(float(lat.mean()), 3),
                   "latency_p50_s": round(float(np.percentile(lat, 50)), 3),
                   "latency_p90_s": round(float(np.percentile(lat, 90)), 3),
                   "latency_p99_s": round(float(np.percentile(lat, 99)), 3),
                   "makespan_s": round(max(r["finish_us"] for r in res) / 1e6, 3),
                   "encode_passes": st["encode_passes"], "decode_steps": st["decode_steps"],
                   "mean_active": round(st["rows_decoded"] / max(1, st["decode_steps"]), 1)}
            rows.append(row)
            print(json.dumps(row), flush=True)
        for name in toks:
            for a, b in zip(toks["continuous"], toks[name]):
                if not np.array_equal(a, b):
                    raise AssertionError(f"{name} produced other tokens than continuous batching")
    for ctx in ctxs.values():
        ctx.close()
    return rows


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--model", default="large-v3", choices=sorted(MODELS))
    ap.add_argument("--rounds", type=int, default=2)
    ap.add_argument("--concurrency", default="5,10,20")
    ap.add_argument("--slots", type=int, default=64)
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--policies", action="store_true", help="compare the queue policies on turbo-u64-q512")
    a = ap.parse_args(argv)
    if a.policies:
        return policies()
    import torch

    shape = MODELS[a.model]
    W = synth.make_weights(shape, 0)
    ctx = binding.Context(synth.pack_blob(W), max_slots=a.slots, max_encode_batch=min(a.slots, 32))
    del W
    rng = np.random.Generator(np.random.PCG64(a.seed))
    # warm-up: one small round through both paths (graph capture, first launches)
    recs, _ = make_round(shape, rng, 2, 15, 30, 10 ** 6)
    dev = {s.segment_id: torch.from_numpy(s.audio).to("cuda:0") for _, ss in recs for s in ss}
    run_sequential(ctx, recs, dev)
    run_multiplexed(ctx, recs, dev)
    rows = []
    first_id = 0
    for C in [int(c) for c in a.concurrency.split(",")]:
        for lo, hi in BUCKETS:
            seq, mux = [], []
            for _ in range(a.rounds):
                recs, first_id = make_round(shape, rng, C, lo, hi, first_id)
                dev = {s.segment_id: torch.from_numpy(s.audio).to("cuda:0") for _, ss in recs for s in ss}
                ls, ts = run_sequential(ctx, recs, dev)
                lm, tm = run_multiplexed(ctx, recs, dev)
                for sid in ts:
                    if not np.array_equal(ts[sid], tm[sid]):
                        raise AssertionError(f"segment {sid}: sequential and multiplexed tokens differ")
                seq += ls
                mux += lm
                del dev
            row = {"concurrency": C, "duration_s": f"{lo}-{hi}", "recordings": len(seq),
                   "p90_sequential_s": round(float(np.percentile(seq, 90)), 3),
                   "p90_multiplexed_s": round(float(np.percentile(mux, 90)), 3)}
            row["improvement"] = round(1.0 - row["p90_multiplexed_s"] / row["p90_sequential_s"], 3)
            rows.append(row)
            print(json.dumps(row), flush=True)
    ctx.close()
    return rows


if __name__ == "__main__":
    main(sys.argv[1:])
