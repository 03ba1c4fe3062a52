"""Benchmark: batched Whisper transcription on one MI355X.

One step = one whisper_batch_transcribe call over the whole workload (log-mel
front end, conv stem, encoder, cross-attention caches, greedy decoding with
self/cross caches, argmax, slot retirement and id mapping). Audio is resident
in HBM before the timed region (device pointers); weights are seeded N(0,
0.02) of the named shape; segments are synthetic (three sinusoids plus
noise, lengths uniform on 3-30 s).

Prints one JSON line: RTFx (audio seconds transcribed per second), the
roofline of the dominant kernel (decode-step cross-attention, HBM-bound)
measured with HIP events on the library's stream, encoder MFMA and decode
HBM fractions, and the CPU oracle timed on a bounded sample on the host.
After the headline workload, each `--secondary` workload (by default the
128-slot refill queue and the 64-slot ragged batch) gets one timed call with
the same encoder and decode accounting, under "secondary".

    python bench.py [--steps K] [--warmup W] [--workload large-v3-b32]
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

PEAK_BF16 = 2.5e15     # dense bf16 MFMA, FLOP/s
PEAK_F32 = 157.3e12    # fp32 vector, FLOP/s
PEAK_HBM = 8.0e12      # bytes/s


def encoder_flops(shape):
    """Algorithmic encoder + cross-KV flops per segment (dense contractions
    only: conv stem, projections, MLP, QK^T and PV at 1500 x 1500)."""
    d, T = shape.d, 1500
    f = 2 * 3000 * d * 3 * shape.n_mels + 2 * T * d * 3 * d
    f += shape.n_enc * (2 * T * 12 * d * d + 4 * T * T * d)
    f += 2 * T * d * 2 * d * shape.n_dec
    if shape.n_dec == 0:  # encoder-only CTC model: the head over every frame
        f += 2 * T * d * shape.n_vocab
    return float(f)


def decode_bytes(shape, st):
    """Algorithmic HBM bytes of the decode steps counted in the library's work
    counters `st`: every weight once per step (plus the output head), and for
    each stepped slot the cross K/V over 1500 positions plus the self K/V over
    its positions so far, in every layer."""
    d, L, esz = shape.d, shape.n_dec, 2 if shape.dtype == "bf16" else 4
    w = (14 * L * d * d + shape.n_vocab * d) * esz
    return (w * st["decode_steps"] + 2 * L * d * esz * 1500 * st["rows_decoded"]
            + 2 * L * d * esz * st["positions_attended"])


def copy_ceiling_gbps(torch, mib=1024):
    """Measured device copy bandwidth (read + write bytes per second) of a
    plain torch copy of `mib` MiB: a practical HBM ceiling next to the
    published peak."""
    x = torch.ones(mib * (1 << 20) // 4, dtype=torch.float32, device="cuda:0")
    y = torch.empty_like(x)
    y.copy_(x)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(5):
        y.copy_(x)
    b.record()
    b.synchronize()
    gbps = 5 * 2 * x.numel() * 4 / (a.elapsed_time(b) / 1e3) / 1e9
    del x, y
    return round(gbps, 1)


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def counter_traffic(workload):
    """HBM bytes per launch of the cross-attention kernel from the committed
    rocprofv3 FETCH_SIZE/WRITE_SIZE summary (scaled by the copy-kernel
    calibration), or None when the kernel's source has changed since the
    counters were taken or no summary exists for this workload."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"cross_attn_{workload}.md")
    if not os.path.exists(path):
        return None
    fields = dict(l.split(": ", 1) for l in open(path).read().splitlines() if ": " in l and " " not in l.split(": ")[0])
    src = open(os.path.join(ROOT, "paper_2507_01021_amd", "csrc", "kernels.h")).read()
    i = src.find("__global__ __launch_bounds__(64 * CW) void cross_attn_kernel(DecAttnArgs a) {")
    if i < 0:
        return None
    j = src.index("\n}\n", i)
    if hashlib.sha256(src[i:j].encode()).hexdigest()[:16] != fields.get("kernel_source_sha256_16", "").strip():
        return None
    return float(fields["traffic_bytes_per_launch"])


def cpu_baseline(shape, W, segs):
    """The oracle, as is, on a bounded sample (about 11 s of CPU work on
    large-v3 shapes on a 16-thread host): one segment's front end, conv stem, NL encoder layers,
    NL layers of cross-attention keys/values and three decode steps of an
    NL-layer decoder (plus the output head alone), extrapolated per layer to
    the full model and the workload's token count."""
    import oracle
    from oracle import model as M

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    s0 = segs[0]
    t = time.perf_counter()
    mel = oracle.log_mel_segment(s0.audio, shape.n_mels)
    t_fe = time.perf_counter() - t
    t = time.perf_counter()
    x = M.conv_stem(W, mel[None]) + M.sinusoid_pe(1500, shape.d)[None]
    t_stem = time.perf_counter() - t
    NL = min(20, shape.n_enc, shape.n_dec)
    shl = shape.with_(n_enc=NL, n_dec=NL)
    t = time.perf_counter()
    E = M.encoder(W, shl, mel[None])
    t_encl = time.perf_counter() - t
    t_layer = max(t_encl - t_stem, 1e-9) / NL
    t = time.perf_counter()
    ckv = M._seg_ckv(M.cross_kv(W, shl, E), 0)
    t_ckv = (time.perf_counter() - t) / NL
    cache = M.DecoderCache(shl)
    t = time.perf_counter()
    for tok in s0.prompt[:3]:
        M.decoder_step(W, shl, tok, cache, ckv)
    t_stepl = (time.perf_counter() - t) / 3
    z = np.zeros((1, shape.d))
    t = time.perf_counter()
    _ = M.layer_norm(z, M._w(W, "dec.ln.g"), M._w(W, "dec.ln.b")) @ M._w(W, "dec.tok_emb").T
    t_head = time.perf_counter() - t
    t_step = t_head + (t_stepl - t_head) / NL * shape.n_dec
    per_seg = []
    for s in segs:
        per_seg.append(t_fe + t_stem + shape.n_enc * t_layer + shape.n_dec * t_ckv
                       + (len(s.prompt) - 1 + s.max_new_tokens) * t_step)
    audio = sum(s.seconds for s in segs)
    sample_s = t_fe + t_encl + NL * t_ckv + 3 * t_stepl + t_head
    return {
        "value": audio / sum(per_seg), "unit": "audio-s/s", "cores": int(threads), "kind": "oracle",
        "cpu": cpu_model(), "host_cpus": os.cpu_count(),
        "sample": (f"1 segment: front end, conv stem, {NL} of {shape.n_enc} encoder layers, {NL} of "
                   f"{shape.n_dec} cross-KV layers, 3 decode steps of a {NL}-layer decoder + output head; "
                   f"extrapolated per layer and per token to the workload ({sample_s:.1f} s of CPU work)"),
    }


def cpu_baseline_ctc(shape, W, segs):
    """The CTC oracle, as is, on one segment (front end, stem, every encoder
    layer, head, best path and collapse), extrapolated to the workload."""
    from oracle import ctc as OC
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    t = time.perf_counter()
    done = 0
    while done < min(len(segs), 32) and time.perf_counter() - t < 10.0:  # about 10 s of CPU work
        OC.transcribe_ctc(W, shape, [segs[done]])
        done += 1
    spent = time.perf_counter() - t
    audio = sum(s.seconds for s in segs[:done])
    return {"value": audio / spent, "unit": "audio-s/s", "cores": int(threads), "kind": "oracle",
            "cpu": cpu_model(), "host_cpus": os.cpu_count(),
            "sample": f"the first {done} segments, each through the whole CTC oracle ({spent:.1f} s of CPU work)"}


def run_decoder_workload(binding, torch, name, steps, warmup, pad_mode=0, encode_batch=0, prefill=0, max_new=0,
                         per_kernel=True):
    """Times `steps` whisper_batch_transcribe calls over the workload (after
    `warmup` calls), with HIP events around every encode pass in the same
    calls; the decode steps are the rest of the calls' wall time. Returns
    (result dict, context, model shape, weights, segments, slots, device
    audio pointers, audio seconds)."""
    from paper_2507_01021_amd import synth

    shape, segs, slots = synth.workload(name)
    if max_new:
        for s in segs:
            s.max_new_tokens = max_new
    W = synth.make_weights(shape, 0)
    blob = synth.pack_blob(W)
    dev_audio = [torch.from_numpy(s.audio).to("cuda:0") for s in segs]
    ptrs = [t.data_ptr() for t in dev_audio]
    eb = encode_batch or min(slots, 32)
    ctx = binding.Context(blob, max_slots=slots, max_encode_batch=eb, pad_mode=pad_mode,
                          prefill=prefill if shape.n_dec else 0)
    del blob
    ctx._keep = dev_audio
    audio_s = sum(s.seconds for s in segs)
    torch.cuda.synchronize()
    for _ in range(warmup):
        ctx.transcribe(segs, device_audio=ptrs)
    torch.cuda.synchronize()
    ctx.stats(reset=True)
    ctx.profile_enable(binding.K_ENC_PASS, True)        # events around each encode pass, decode steps unchanged
    t0 = time.perf_counter()
    for _ in range(steps):
        res = ctx.transcribe(segs, device_audio=ptrs)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    st = ctx.stats(reset=True)
    enc_ms, enc_n = ctx.profile_read(binding.K_ENC_PASS)
    ctx.profile_enable(binding.K_ENC_PASS, False)
    assert enc_n == st["encode_passes"]
    assert all(r["status"] == 0 and r["tokens"].size == s.max_new_tokens for r, s in zip(res, segs))
    fl = encoder_flops(shape) * len(segs) * steps
    peak_f = PEAK_BF16 if shape.dtype == "bf16" else PEAK_F32
    enc = {"ms_per_pass": round(enc_ms / max(enc_n, 1), 3), "passes": enc_n,
           "tflops": round(fl / (enc_ms / 1e3) / 1e12, 1), "mfma_frac": round(fl / (enc_ms / 1e3) / peak_f, 4)}
    # decode: the timed calls' wall time minus their encode passes (same calls)
    dec_wall_ms = wall * 1e3 - enc_ms
    db = decode_bytes(shape, st)
    dec = {"ms_per_step": round(dec_wall_ms / max(st["decode_steps"], 1), 3), "steps": st["decode_steps"],
           "gbps": round(db / (dec_wall_ms / 1e3) / 1e9, 1), "hbm_frac": round(db / (dec_wall_ms / 1e3) / PEAK_HBM, 4),
           "bytes_per_step": round(db / max(st["decode_steps"], 1)),
           "avg_active_slots": round(st["rows_decoded"] / max(st["decode_steps"], 1), 2)}
    batcher = {"refill_batches_per_call": st["refill_batches"] // steps,
               "host_ms_per_refill": round(st["batcher_host_ms"] / max(st["refill_batches"], 1), 4),
               "host_ms_per_call": round(st["batcher_host_ms"] / steps, 3),
               "engine_host_ms_per_call": round(st["engine_host_ms"] / steps, 2)}
    out = {"value": round(audio_s * steps / wall, 2), "ms_per_call": round(wall / steps * 1e3, 2),
           "encoder": enc, "decode": dec, "batcher": batcher,
           "padded_rtfx": round(30.0 * len(segs) * steps / wall, 2)}
    if per_kernel:
        # Per-kernel timing: the same calls again with HIP events around every
        # launch of the named kernels (decode steps then run as individual
        # launches, unsplit, instead of captured graphs)
        kinds = (binding.K_DEC_STEP, binding.K_ENC_GEMM, binding.K_FRONT_END)
        for k in kinds:
            ctx.profile_enable(k, True)
        t1 = time.perf_counter()
        for _ in range(steps):
            ctx.transcribe(segs, device_audio=ptrs)
        torch.cuda.synchronize()
        wall_timed = time.perf_counter() - t1
        prof = {k: ctx.profile_read(k) for k in kinds}
        for k in kinds:
            ctx.profile_enable(k, False)
        fe_ms, fe_n = prof[binding.K_FRONT_END]
        enc["front_end_ms_per_pass"] = round(fe_ms / max(fe_n, 1), 3)
        g_ms, g_n = prof[binding.K_ENC_GEMM]
        fc1_flops = 2 * 1500 * shape.d * 4 * shape.d * len(segs) * shape.n_enc * steps
        enc["fc1_gemm_tflops"] = round(fc1_flops / (g_ms / 1e3) / 1e12, 1) if g_ms > 0 else None
        d_ms, d_n = prof[binding.K_DEC_STEP]
        dec["ms_per_step_kernel_timed"] = round(d_ms / max(d_n, 1), 3)
        dec["ms_per_call_kernel_timed"] = round(wall_timed / steps * 1e3, 2)
        # the cross-attention as the plain steps run it (captured graphs, slots
        # split into concurrent chains): one more call with each launch's span
        # stamped by the kernel itself
        ctx.stats(reset=True)
        ctx.profile_enable(binding.K_CROSS_ATTN_STEP, True)
        ctx.transcribe(segs, device_audio=ptrs)
        torch.cuda.synchronize()
        s_ms, s_n = ctx.profile_read(binding.K_CROSS_ATTN_STEP)
        ctx.profile_enable(binding.K_CROSS_ATTN_STEP, False)
        st_s = ctx.stats(reset=True)
        esz = 2 if shape.dtype == "bf16" else 4
        s_bytes = st_s["rows_decoded"] * shape.n_dec * shape.d * 1500 * 2 * esz
        out["cross_attn_in_step"] = {
            "launches": s_n, "avg_launch_us": round(s_ms * 1e3 / max(s_n, 1), 2),
            "rows_per_launch": round(st_s["rows_decoded"] * shape.n_dec / max(s_n, 1), 2),
            "achieved": round(s_bytes / (s_ms / 1e3) / 1e9, 1) if s_ms > 0 else None,
            "frac": round(s_bytes / (s_ms / 1e3) / PEAK_HBM, 4) if s_ms > 0 else None,
            "unit": "GB/s", "timing": "device real-time counter, first workgroup start to last workgroup end"}
    return out, ctx, shape, W, segs, slots, ptrs, audio_s


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="large-v3-b32")
    ap.add_argument("--secondary", default="turbo-u64-q512,small-u8-b64",
                    help="comma-separated decoder workloads (continuous batching with refill, ragged "
                         "retirement) measured after the headline one in the same run ('' to skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one device copy of this many MiB (counter calibration)")
    ap.add_argument("--pad-mode", type=int, default=0, choices=(0, 1),
                    help="0: pad the audio to 30 s, then the front end (default); 1: front end on the "
                         "segment alone, features padded to 3000 frames")
    ap.add_argument("--encode-batch", type=int, default=0,
                    help="segments per encoder pass (0: min(slots, 32))")
    ap.add_argument("--prefill", type=int, default=0, choices=(0, 1),
                    help="decoder workloads: 1 runs each segment's prompt through the decoder in one pass at "
                         "encode time instead of one position per decode step")
    ap.add_argument("--ctc-beam", type=int, default=0,
                    help="CTC workloads: 0 greedy best path, 2..16 prefix beam search with that beam")
    ap.add_argument("--max-new", type=int, default=0,
                    help="profiling runs only: decode this many tokens per segment instead of the workload's")
    a = ap.parse_args()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {a.gpus}): segments are independent, "
              "so more GPUs would each run this same single-GPU engine on their share", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2507_01021_amd import binding, synth

    if synth.workload(a.workload)[0].n_dec == 0:
        return bench_ctc(a, binding, torch)
    r, ctx, shape, W, segs, slots, ptrs, audio_s = run_decoder_workload(
        binding, torch, a.workload, a.steps, a.warmup, a.pad_mode, a.encode_batch, a.prefill, a.max_new)
    copy_gbps = copy_ceiling_gbps(torch)

    if a.calib_copy_mib:
        x = torch.ones(a.calib_copy_mib * (1 << 20) // 4, dtype=torch.float32, device="cuda:0")
        y = torch.empty_like(x)
        torch.cuda.synchronize()
        y.copy_(x)
        torch.cuda.synchronize()

    # dominant kernel: decode-step cross-attention (HBM-bound), timed as
    # back-to-back launches over all of the workload's slots (their caches
    # hold the last pass's encoder output), two events on the library's
    # stream around 4 launches per decoder layer
    ca_rows, ca_n = slots, 4 * shape.n_dec
    ca_avg_s = ctx.time_kernel(binding.K_CROSS_ATTN, ca_rows, ca_n) / 1e6
    ca_bytes = ca_rows * shape.d * 1500 * 2 * (2 if shape.dtype == "bf16" else 4)
    achieved = ca_bytes / ca_avg_s / 1e9
    roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM / 1e9, "unit": "GB/s",
            "frac": round(achieved / (PEAK_HBM / 1e9), 4), "traffic": counter_traffic(a.workload),
            "kernel": "cross_attn_kernel<bf16> (decode-step cross-attention over the 1500 cached positions)",
            "bytes_per_launch": ca_bytes, "avg_launch_us": round(ca_avg_s * 1e6, 2), "launches": ca_n,
            "rows_per_launch": ca_rows,
            "measured_copy_gbps": copy_gbps,
            # the same kernel inside the timed steps' graphs (concurrent chains)
            "in_step": r.get("cross_attn_in_step")}
    ctx.close()

    out = {
        "metric": "audio-sec transcribed/sec (RTFx) at batch B; encoder MFMA util; decode HBM GB/s",
        "value": r["value"], "unit": "audio-s/s", "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": r["ms_per_call"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": shape.dtype, "data": "synthetic",
        "config": {"workload": a.workload, "segments": len(segs), "slots": slots,
                   "new_tokens": [int(min(s.max_new_tokens for s in segs)), int(max(s.max_new_tokens for s in segs))],
                   "audio_s": round(audio_s, 2), "weights_seed": 0, "workload_seed": 1,
                   "pad_mode": a.pad_mode, "prefill": a.prefill, "encode_batch": a.encode_batch or min(slots, 32)},
        "roofline": roof, "encoder": r["encoder"], "decode": r["decode"], "batcher": r["batcher"],
        # every segment is encoded as a full 30 s window: RTFx over padded seconds
        "padded_rtfx": r["padded_rtfx"],
    }
    more = [w for w in a.secondary.split(",") if w and w != a.workload] if not a.max_new else []
    if more:
        # the refill / ragged workloads, each one timed call after one
        # warm-up call, same accounting
        out["secondary"] = []
        for w in more:
            r2, ctx2, shape2, _, segs2, slots2, _, audio2 = run_decoder_workload(
                binding, torch, w, 1, 1, a.pad_mode, 0, a.prefill, 0, per_kernel=False)
            ctx2.close()
            out["secondary"].append({"workload": w, "segments": len(segs2), "slots": slots2,
                                     "audio_s": round(audio2, 2), "value": r2["value"], "unit": "audio-s/s",
                                     "ms_per_call": r2["ms_per_call"], "encoder": r2["encoder"],
                                     "decode": r2["decode"]})
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(shape, W, segs)
    print(json.dumps(out), flush=True)


def bench_ctc(a, binding, torch):
    """Encoder-only CTC workload: the queue in encoder passes; its roofline is
    the encoder's fc1 GEMM (MFMA-bound), timed with HIP events around every
    launch in a second run of the same calls."""
    from paper_2507_01021_amd import synth

    shape, segs, slots = synth.workload(a.workload)
    W = synth.make_weights(shape, 0)
    blob = synth.pack_blob(W)
    dev_audio = [torch.from_numpy(s.audio).to("cuda:0") for s in segs]
    ptrs = [t.data_ptr() for t in dev_audio]
    ctx = binding.Context(blob, max_slots=slots, max_encode_batch=a.encode_batch or min(slots, 32),
                          pad_mode=a.pad_mode, ctc_beam=a.ctc_beam)
    del blob
    audio_s = sum(s.seconds for s in segs)
    torch.cuda.synchronize()
    for _ in range(a.warmup):
        ctx.transcribe(segs, device_audio=ptrs)
    torch.cuda.synchronize()
    ctx.stats(reset=True)
    t0 = time.perf_counter()
    for _ in range(a.steps):
        res = ctx.transcribe(segs, device_audio=ptrs)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    st_timed = ctx.stats(reset=True)
    assert all(r["status"] == 0 and r["tokens"].size <= s.max_new_tokens for r, s in zip(res, segs))
    kinds = (binding.K_ENC_PASS, binding.K_ENC_GEMM, binding.K_FRONT_END)
    for k in kinds:
        ctx.profile_enable(k, True)
    for _ in range(a.steps):
        ctx.transcribe(segs, device_audio=ptrs)
    torch.cuda.synchronize()
    prof = {k: ctx.profile_read(k) for k in kinds}
    peak_f = PEAK_BF16 if shape.dtype == "bf16" else PEAK_F32
    enc_ms, enc_n = prof[binding.K_ENC_PASS]
    fl = encoder_flops(shape) * len(segs) * a.steps
    g_ms, g_n = prof[binding.K_ENC_GEMM]
    fc1_flops = 2 * 1500 * shape.d * 4 * shape.d * len(segs) * shape.n_enc * a.steps
    fc1_tf = fc1_flops / (g_ms / 1e3) / 1e12
    roof = {"bound": "mfma", "achieved": round(fc1_tf, 1), "peak": peak_f / 1e12, "unit": "TFLOP/s",
            "frac": round(fc1_tf * 1e12 / peak_f, 4), "traffic": None,
            "kernel": ("gemm_bf16_h_kernel" if shape.d <= 1024 else "gemm_bf16_kernel")
                      + "<EpiGelu> (encoder fc1 + GELU)",
            "flops_per_launch": fc1_flops / max(g_n, 1), "avg_launch_us": round(g_ms * 1e3 / max(g_n, 1), 2),
            "launches": g_n}
    fe_ms, fe_n = prof[binding.K_FRONT_END]
    enc = {"ms_per_pass": round(enc_ms / max(enc_n, 1), 3), "passes": enc_n,
           "tflops": round(fl / (enc_ms / 1e3) / 1e12, 1), "mfma_frac": round(fl / (enc_ms / 1e3) / peak_f, 4),
           "front_end_ms_per_pass": round(fe_ms / max(fe_n, 1), 3), "fc1_gemm_tflops": round(fc1_tf, 1)}
    batcher = {"passes_per_call": st_timed["encode_passes"] // a.steps,
               "host_ms_per_call": round(st_timed["batcher_host_ms"] / a.steps, 3),
               "engine_host_ms_per_call": round(st_timed["engine_host_ms"] / a.steps, 2)}
    value = audio_s * a.steps / wall
    out = {
        "metric": "audio-sec transcribed/sec (RTFx) at batch B; encoder MFMA util; decode HBM GB/s",
        "value": round(value, 2), "unit": "audio-s/s", "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": round(wall / a.steps * 1e3, 2), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": shape.dtype, "data": "synthetic",
        "config": {"workload": a.workload, "segments": len(segs), "encode_batch": a.encode_batch or min(slots, 32),
                   "audio_s": round(audio_s, 2), "weights_seed": 0, "workload_seed": 1, "pad_mode": a.pad_mode,
                   "decoding": "CTC best path" if a.ctc_beam < 2 else f"CTC prefix beam search, beam {a.ctc_beam}"},
        "roofline": roof, "encoder": enc, "batcher": batcher,
        "padded_rtfx": round(30.0 * len(segs) * a.steps / wall, 2),
    }
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline_ctc(shape, W, segs)
    ctx.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
