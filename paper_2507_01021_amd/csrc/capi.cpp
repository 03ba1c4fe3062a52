// C ABI (include/whisper_mi355x.h): argument validation, slot bookkeeping,
// error codes and messages, and the continuous-batching driver that ties the
// batcher to the engine. Every check runs before any device work.
#include <string.h>

#include <chrono>
#include <memory>
#include <thread>
#include <new>
#include <set>
#include <string>
#include <vector>

#include "batcher.h"
#include "common.h"
#include "engine.h"

namespace {

thread_local std::string g_create_error;

struct SlotState {
    bool active = false;
    int n_prompt = 0, max_new = 0, steps = 0, generated = 0;
};

}  // namespace

struct whisper_ctx {
    whisper_params p;
    std::unique_ptr<wmi::Engine> eng;
    std::string err;
    std::vector<SlotState> slots;
    whisper_stats stats{};
    int eot = -1;  // end-of-text token of whisper_batch_transcribe / _serve, -1: none
    bool broken = false;
};

namespace {

whisper_status fail(whisper_ctx* c, whisper_status code, const std::string& msg) {
    if (c) {
        c->err = msg;
        if (code == WHISPER_E_DEVICE) c->broken = true;
    } else {
        g_create_error = msg;
    }
    return code;
}

template <class F>
whisper_status guarded(whisper_ctx* c, F&& f) {
    try {
        return f();
    } catch (const wmi::ArgError& e) {
        return fail(c, e.code, e.what());
    } catch (const wmi::DeviceError& e) {
        return fail(c, WHISPER_E_DEVICE, e.what());
    } catch (const std::bad_alloc&) {
        return fail(c, WHISPER_E_NOMEM, "host allocation failed");
    } catch (const std::exception& e) {
        return fail(c, WHISPER_E_DEVICE, e.what());
    }
}

std::string check_segment(const whisper_params& p, const whisper_segment& s, int i) {
    const std::string at = "segment " + std::to_string(i) + ": ";
    if (!s.audio) return at + "audio is NULL";
    if (s.n_samples < 1 || s.n_samples > 480000) return at + "n_samples must be in 1..480000";
    if (s.audio_on_device != 0 && s.audio_on_device != 1) return at + "audio_on_device must be 0 or 1";
    if (p.n_text_layer == 0) {  // CTC model: no prompt, max_new_tokens is the output capacity
        if (s.max_new_tokens < 1 || s.max_new_tokens > 1500) return at + "max_new_tokens must be in 1..1500";
        return "";
    }
    if (s.n_prompt < 1 || !s.prompt) return at + "needs a prompt of at least one token";
    if (s.max_new_tokens < 1) return at + "max_new_tokens must be >= 1";
    if ((int64_t)s.n_prompt + s.max_new_tokens > p.n_text_ctx)
        return at + "n_prompt + max_new_tokens exceeds the text context (" + std::to_string(p.n_text_ctx) + ")";
    for (int k = 0; k < s.n_prompt; ++k)
        if (s.prompt[k] < 0 || s.prompt[k] >= p.n_vocab) return at + "prompt token out of range";
    return "";
}

std::string check_params(const whisper_params& p, const whisper_params& blob) {
    if (p.n_mels != blob.n_mels || p.n_audio_ctx != blob.n_audio_ctx || p.n_audio_state != blob.n_audio_state ||
        p.n_audio_head != blob.n_audio_head || p.n_audio_layer != blob.n_audio_layer || p.n_vocab != blob.n_vocab ||
        p.n_text_ctx != blob.n_text_ctx || p.n_text_state != blob.n_text_state ||
        p.n_text_head != blob.n_text_head || p.n_text_layer != blob.n_text_layer || p.dtype != blob.dtype)
        return "params do not match the weight blob header";
    if (p.dtype != WHISPER_DTYPE_F32 && p.dtype != WHISPER_DTYPE_BF16) return "dtype must be 0 (fp32) or 1 (bf16)";
    if (p.n_audio_ctx != 1500) return "n_audio_ctx must be 1500";
    if (p.n_text_ctx != 448) return "n_text_ctx must be 448";
    if (p.n_audio_state != p.n_text_state || p.n_audio_head != p.n_text_head)
        return "encoder and decoder widths and head counts must match";
    if (p.n_audio_head < 1 || p.n_audio_state != 64 * p.n_audio_head) return "head size must be 64";
    if (p.n_audio_state > 2048) return "width above 2048 is not supported";
    if (p.n_mels < 4 || p.n_mels > 128 || p.n_mels % 4) return "n_mels must be a multiple of 4 in 4..128";
    if (p.n_audio_layer < 1 || p.n_text_layer < 0 || p.n_text_layer > 256 ||
        p.n_vocab < (p.n_text_layer == 0 ? 2 : 1))
        return "encoder layers >= 1, decoder layers in 0..256 (0: CTC model), vocabulary >= 1 (CTC: >= 2)";
    if (p.max_slots < 1 || p.max_slots > 128) return "max_slots must be in 1..128";
    if (p.max_encode_batch < 0 || p.max_encode_batch > p.max_slots) return "max_encode_batch must be in 0..max_slots";
    if (p.pad_mode != 0 && p.pad_mode != 1) return "pad_mode must be 0 or 1";
    if (p.refill_min < 0) return "refill_min must be >= 0";
    if (p.batch_policy < 0 || p.batch_policy > 1) return "batch_policy must be 0 or 1";
    if (p.step_cost_us < 0 || p.max_wait_ms < 0) return "step_cost_us and max_wait_ms must be >= 0";
    if (p.ctc_beam < 0 || p.ctc_beam > 16) return "ctc_beam must be in 0..16";
    if (p.prefill != 0 && p.prefill != 1) return "prefill must be 0 or 1";
    if (p.prefill != 0 && p.n_text_layer == 0) return "prefill needs a decoder model";
    if (p.ctc_beam > 1 && (p.n_text_layer != 0 || p.n_vocab > 4096))
        return "ctc_beam >= 2 needs a CTC model with n_vocab <= 4096";
    return "";
}

// Batch backend on a real context.
// Engine calls of the batcher, with the work counters and the host time
// spent inside them (the rest of the batcher's time is its own logic).
struct EngineBackend : wmi::BatchBackend {
    using clock = std::chrono::steady_clock;
    whisper_ctx* c;
    const whisper_segment* segs;
    bool realtime = false;
    clock::time_point t0 = clock::now();
    std::vector<wmi::SegmentDesc> descs;
    std::vector<int> steps;    // decode steps taken by each slot's current segment
    std::vector<int> mark_of;  // completion mark of each retired segment
    int step_mark = -1;        // mark after the latest step, once a segment retired with it
    bool eot_stop = false;     // retire segments at their end-of-text token
    std::vector<int32_t> stop_of;  // each retired segment's end-of-text position (-1: none)
    int64_t n_steps = 0;
    double engine_ms = 0.0;
    struct Timer {
        double& acc;
        clock::time_point t0 = clock::now();
        ~Timer() { acc += std::chrono::duration<double, std::milli>(clock::now() - t0).count(); }
    };
    void encode(const int* idx, int n, const int* slots) override {
        Timer t{engine_ms};
        descs.resize(n);
        for (int k = 0; k < n; ++k) {
            const whisper_segment& s = segs[idx[k]];
            descs[k] = wmi::SegmentDesc{s.audio, s.n_samples, s.audio_on_device == 1, s.prompt, s.n_prompt};
            steps[slots[k]] = c->p.prefill ? s.n_prompt - 1 : 0;  // prefilled prompt positions
        }
        c->eng->encode(descs.data(), n, slots, realtime);
        c->stats.encode_passes += (n + c->p.max_encode_batch - 1) / c->p.max_encode_batch;
        c->stats.segments_encoded += n;
        c->stats.refill_batches += 1;
    }
    void step(const int* slots, int n) override {
        Timer t{engine_ms};
        c->eng->decode_step(slots, n, nullptr, nullptr, nullptr, realtime);
        if (eot_stop) c->eng->stop_snapshot();
        ++n_steps;
        step_mark = -1;
        c->stats.decode_steps += 1;
        c->stats.rows_decoded += n;
        for (int k = 0; k < n; ++k) c->stats.positions_attended += ++steps[slots[k]];
    }
    void retire(int slot, int idx, int count, int32_t* dst) override {
        Timer t{engine_ms};
        if (step_mark < 0) step_mark = c->eng->mark();
        mark_of[idx] = step_mark;
        c->eng->read_tokens_async(slot, count, dst);
        if (eot_stop) c->eng->read_stop_async(slot, &stop_of[idx]);
    }
    bool stops(std::vector<int>& out, int64_t& as_of) override {
        if (!eot_stop) return false;
        Timer t{engine_ms};
        const int* p = c->eng->stop_poll();
        if (!p) return false;
        for (int s = 0; s < c->p.max_slots; ++s)
            if (p[s] >= 0) out.push_back(s);
        as_of = n_steps - 2;
        return true;
    }
    void finish() override {
        Timer t{engine_ms};
        c->eng->finish_reads();
    }
    int64_t now_us() override {
        return std::chrono::duration_cast<std::chrono::microseconds>(clock::now() - t0).count();
    }
    void wait_until(int64_t t) override {
        const int64_t dt = t - now_us();
        if (dt > 0) std::this_thread::sleep_for(std::chrono::microseconds(dt));
    }
};

// Batch backend of the host-only scheduler check.
struct FakeBackend : wmi::BatchBackend {
    const int64_t* seg_ids;
    std::vector<int32_t>* events;
    std::vector<int64_t>* finish_at;
    std::vector<int32_t>* stop_of;
    int64_t clock_us = 0, encode_us = 0, step_us = 0;
    int eot = -1;
    // per slot: segment, tokens generated, end-of-text position; snapshots after each step
    std::vector<int> seg, gen, stop_at;
    std::vector<std::vector<int>> snaps;
    static int32_t token(int64_t seg_id, int j) { return (int32_t)((uint64_t)(seg_id * 7919 + (int64_t)j * 104729) % 50000); }
    void encode(const int* idx, int n, const int* slots) override {
        for (int k = 0; k < n; ++k) {
            events->insert(events->end(), {0, slots[k], idx[k]});
            seg[slots[k]] = idx[k];
            gen[slots[k]] = 0;
            stop_at[slots[k]] = -1;
        }
        clock_us += encode_us * n;
    }
    void step(const int* slots, int n) override {
        events->insert(events->end(), {1, n, 0});
        clock_us += step_us;
        for (int k = 0; k < n; ++k) {
            const int s = slots[k], g = gen[s]++;
            if (eot >= 0 && stop_at[s] < 0 && token(seg_ids[seg[s]], g) == eot) stop_at[s] = g;
        }
        snaps.push_back(stop_at);
    }
    void retire(int slot, int idx, int count, int32_t* dst) override {
        for (int j = 0; j < count; ++j) dst[j] = token(seg_ids[idx], j);
        (*finish_at)[idx] = clock_us;
        (*stop_of)[idx] = stop_at[slot];
    }
    bool stops(std::vector<int>& out, int64_t& as_of) override {
        if (eot < 0 || snaps.size() < 2) return false;
        const std::vector<int>& p = snaps[snaps.size() - 2];
        for (size_t s = 0; s < p.size(); ++s)
            if (p[s] >= 0) out.push_back((int)s);
        as_of = (int64_t)snaps.size() - 2;
        return true;
    }
    void finish() override {}
    int64_t now_us() override { return clock_us; }
    void wait_until(int64_t t) override { clock_us = t > clock_us ? t : clock_us; }
};

std::vector<int64_t> offsets_of(const std::vector<wmi::QueuedSegment>& q, int64_t* total) {
    std::vector<int64_t> off(q.size());
    int64_t t = 0;
    for (size_t i = 0; i < q.size(); ++i) { off[i] = t; t += q[i].max_new_tokens; }
    *total = t;
    return off;
}

// Batch backend of encoder-only CTC models: each pass computes and delivers
// its segments' labels (truncated to max_new_tokens) and completion mark.
struct CtcBackend : wmi::BatchBackend {
    using clock = std::chrono::steady_clock;
    whisper_ctx* c = nullptr;
    const whisper_segment* segs = nullptr;
    const std::vector<int64_t>* off = nullptr;
    int32_t* token_buf = nullptr;
    whisper_result* results = nullptr;
    clock::time_point t0 = clock::now();
    std::vector<int> mark_of;
    std::vector<int32_t> tok, cnt;
    double engine_ms = 0.0;
    struct Pending {
        int ticket = -1, mark = -1;
        std::vector<int> idx;
    } pending;  // the batch encoded last, read once the next one is queued
    void encode(const int* idx, int n, const int*) override {
        const clock::time_point t = clock::now();
        std::vector<wmi::SegmentDesc> d(n);
        for (int k = 0; k < n; ++k) {
            const whisper_segment& s = segs[idx[k]];
            d[k] = wmi::SegmentDesc{s.audio, s.n_samples, s.audio_on_device == 1, nullptr, 0};
        }
        int mark = -1;
        const int ticket = c->eng->encode_ctc(d.data(), n, &mark);
        deliver();
        pending.ticket = ticket;
        pending.mark = mark;
        pending.idx.assign(idx, idx + n);
        c->stats.encode_passes += 1;
        c->stats.segments_encoded += n;
        c->stats.refill_batches += 1;
        engine_ms += std::chrono::duration<double, std::milli>(clock::now() - t).count();
    }
    // Reads the pending batch's labels (truncated to max_new_tokens, the rest
    // of each segment's region set to -1) into token_buf.
    void deliver() {
        if (pending.ticket < 0) return;
        const int n = (int)pending.idx.size();
        tok.resize((size_t)n * 1500);
        cnt.resize(n);
        c->eng->read_ctc(pending.ticket, n, tok.data(), cnt.data());
        for (int k = 0; k < n; ++k) {
            const int i = pending.idx[k];
            const int32_t k_tok = std::min(cnt[k], segs[i].max_new_tokens);
            int32_t* dst = token_buf + (*off)[i];
            std::copy(tok.begin() + (size_t)k * 1500, tok.begin() + (size_t)k * 1500 + k_tok, dst);
            std::fill(dst + k_tok, dst + segs[i].max_new_tokens, -1);
            results[i].n_tokens = k_tok;
            mark_of[i] = pending.mark;
        }
        pending.ticket = -1;
    }
    void step(const int*, int) override {}
    void retire(int, int, int, int32_t*) override {}
    void finish() override {
        const clock::time_point t = clock::now();
        deliver();
        engine_ms += std::chrono::duration<double, std::milli>(clock::now() - t).count();
    }
    int64_t now_us() override {
        return std::chrono::duration_cast<std::chrono::microseconds>(clock::now() - t0).count();
    }
    void wait_until(int64_t t) override {
        const int64_t dt = t - now_us();
        if (dt > 0) std::this_thread::sleep_for(std::chrono::microseconds(dt));
    }
};

whisper_status serve_ctc(whisper_ctx* ctx, const whisper_segment* segs, int n, const std::vector<wmi::QueuedSegment>& q,
                         const std::vector<int64_t>& off, int32_t* token_buf, whisper_result* results, bool realtime) {
    const whisper_status r = guarded(ctx, [&]() -> whisper_status {
        CtcBackend be;
        be.c = ctx;
        be.segs = segs;
        be.off = &off;
        be.token_buf = token_buf;
        be.results = results;
        be.mark_of.assign(n, -1);
        ctx->eng->mark_reset();
        be.t0 = CtcBackend::clock::now();
        wmi::BatchPolicy pol;
        pol.dynamic = ctx->p.batch_policy == 1;
        pol.max_wait_us = 1000LL * ctx->p.max_wait_ms;
        wmi::run_queue_passes(q, ctx->p.max_encode_batch, be, realtime, pol);
        const double total_ms = std::chrono::duration<double, std::milli>(CtcBackend::clock::now() - be.t0).count();
        ctx->stats.engine_host_ms += be.engine_ms;
        ctx->stats.batcher_host_ms += total_ms - be.engine_ms;
        const std::vector<double> t = ctx->eng->mark_times_us();
        for (int i = 0; i < n; ++i)
            if (be.mark_of[i] >= 0) results[i].finish_us = (int64_t)t[be.mark_of[i]];
        return WHISPER_OK;
    });
    if (r != WHISPER_OK)
        for (int i = 0; i < n; ++i) { results[i].status = r; results[i].n_tokens = 0; }
    return r;
}

}  // namespace

extern "C" {

whisper_status whisper_params_from_blob(const void* blob, size_t blob_bytes, whisper_params* out) {
    if (!out) return fail(nullptr, WHISPER_E_INVAL, "out is NULL");
    const char* why = "";
    const int st = wmi::parse_blob_header(blob, blob_bytes, out, &why);
    if (st != WHISPER_OK) return fail(nullptr, st, why);
    return WHISPER_OK;
}

whisper_status whisper_ctx_create(const whisper_params* params, const void* weights, size_t weights_bytes, int device,
                                  whisper_ctx** out) {
    if (!params || !weights || !out) return fail(nullptr, WHISPER_E_INVAL, "params, weights and out must not be NULL");
    whisper_params blob;
    const char* why = "";
    const int st = wmi::parse_blob_header(weights, weights_bytes, &blob, &why);
    if (st != WHISPER_OK) return fail(nullptr, st, why);
    const std::string bad = check_params(*params, blob);
    if (!bad.empty()) return fail(nullptr, bad.find("header") != std::string::npos ? WHISPER_E_FORMAT : WHISPER_E_INVAL, bad);
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || device < 0 || device >= ndev)
        return fail(nullptr, WHISPER_E_DEVICE, "no HIP device " + std::to_string(device));
    whisper_params p = *params;
    if (p.max_encode_batch == 0) p.max_encode_batch = p.max_slots < 32 ? p.max_slots : 32;
    if (p.refill_min == 0) p.refill_min = 16;
    if (p.step_cost_us == 0) p.step_cost_us = 2000;
    std::unique_ptr<whisper_ctx> c(new (std::nothrow) whisper_ctx());
    if (!c) return fail(nullptr, WHISPER_E_NOMEM, "host allocation failed");
    c->p = p;
    c->slots.resize(p.max_slots);
    const whisper_status r = guarded(nullptr, [&]() -> whisper_status {
        c->eng = wmi::make_engine(p, weights, weights_bytes, device);
        return WHISPER_OK;
    });
    if (r != WHISPER_OK) return r;
    *out = c.release();
    return WHISPER_OK;
}

void whisper_ctx_destroy(whisper_ctx* ctx) { delete ctx; }

const char* whisper_last_error(const whisper_ctx* ctx) {
    return ctx ? ctx->err.c_str() : g_create_error.c_str();
}

whisper_status whisper_ctx_set_stream(whisper_ctx* ctx, void* hip_stream) {
    if (!ctx) return fail(nullptr, WHISPER_E_INVAL, "ctx is NULL");
    if (ctx->broken) return fail(ctx, WHISPER_E_DEVICE, "context unusable after a device error");
    return guarded(ctx, [&]() -> whisper_status {
        ctx->eng->set_stream(hip_stream);
        return WHISPER_OK;
    });
}

whisper_status whisper_batch_encode(whisper_ctx* ctx, const whisper_segment* segs, int32_t n, const int32_t* slots) {
    if (!ctx) return fail(nullptr, WHISPER_E_INVAL, "ctx is NULL");
    if (ctx->broken) return fail(ctx, WHISPER_E_DEVICE, "context unusable after a device error");
    if (n < 0) return fail(ctx, WHISPER_E_INVAL, "n must be >= 0");
    if (n == 0) return WHISPER_OK;
    if (ctx->p.n_text_layer == 0) {  // CTC model: one pass of n segments, slots ignored
        if (!segs) return fail(ctx, WHISPER_E_INVAL, "segs must not be NULL");
        if (n > ctx->p.max_encode_batch) return fail(ctx, WHISPER_E_CAPACITY, "a CTC encode takes at most max_encode_batch segments");
        for (int i = 0; i < n; ++i) {
            const std::string bad = check_segment(ctx->p, segs[i], i);
            if (!bad.empty()) return fail(ctx, WHISPER_E_INVAL, bad);
        }
        return guarded(ctx, [&]() -> whisper_status {
            std::vector<wmi::SegmentDesc> d(n);
            for (int i = 0; i < n; ++i)
                d[i] = wmi::SegmentDesc{segs[i].audio, segs[i].n_samples, segs[i].audio_on_device == 1, nullptr, 0};
            ctx->eng->encode_ctc(d.data(), n, nullptr);
            ctx->eng->sync();
            ctx->stats.encode_passes += 1;
            ctx->stats.segments_encoded += n;
            return WHISPER_OK;
        });
    }
    if (!segs || !slots) return fail(ctx, WHISPER_E_INVAL, "segs and slots must not be NULL");
    std::set<int> seen;
    for (int i = 0; i < n; ++i) {
        const std::string bad = check_segment(ctx->p, segs[i], i);
        if (!bad.empty()) return fail(ctx, WHISPER_E_INVAL, bad);
        if (slots[i] < 0 || slots[i] >= ctx->p.max_slots)
            return fail(ctx, WHISPER_E_CAPACITY, "slot " + std::to_string(slots[i]) + " outside 0..max_slots-1");
        if (!seen.insert(slots[i]).second) return fail(ctx, WHISPER_E_INVAL, "slots must be distinct");
        if (ctx->slots[slots[i]].active)
            return fail(ctx, WHISPER_E_STATE, "slot " + std::to_string(slots[i]) + " is active");
    }
    return guarded(ctx, [&]() -> whisper_status {
        std::vector<wmi::SegmentDesc> d(n);
        for (int i = 0; i < n; ++i)
            d[i] = wmi::SegmentDesc{segs[i].audio, segs[i].n_samples, segs[i].audio_on_device == 1, segs[i].prompt,
                                    segs[i].n_prompt};
        ctx->eng->encode(d.data(), n, slots, true);
        ctx->stats.encode_passes += (n + ctx->p.max_encode_batch - 1) / ctx->p.max_encode_batch;
        ctx->stats.segments_encoded += n;
        for (int i = 0; i < n; ++i) {
            SlotState& s = ctx->slots[slots[i]];
            s.active = true;
            s.n_prompt = segs[i].n_prompt;
            s.max_new = segs[i].max_new_tokens;
            s.steps = ctx->p.prefill ? segs[i].n_prompt - 1 : 0;  // prefilled prompt positions
            s.generated = 0;
        }
        return WHISPER_OK;
    });
}

whisper_status whisper_batch_decode_step(whisper_ctx* ctx, const int32_t* slots, int32_t n, const int32_t* forced,
                                         int32_t* out_tokens, float* out_logits) {
    if (!ctx) return fail(nullptr, WHISPER_E_INVAL, "ctx is NULL");
    if (ctx->broken) return fail(ctx, WHISPER_E_DEVICE, "context unusable after a device error");
    if (ctx->p.n_text_layer == 0) return fail(ctx, WHISPER_E_STATE, "not available for an encoder-only CTC model");
    if (n < 0 || n > ctx->p.max_slots) return fail(ctx, WHISPER_E_INVAL, "n must be in 0..max_slots");
    if (n == 0) return WHISPER_OK;
    if (!slots) return fail(ctx, WHISPER_E_INVAL, "slots must not be NULL");
    std::set<int> seen;
    for (int i = 0; i < n; ++i) {
        if (slots[i] < 0 || slots[i] >= ctx->p.max_slots)
            return fail(ctx, WHISPER_E_CAPACITY, "slot " + std::to_string(slots[i]) + " outside 0..max_slots-1");
        if (!seen.insert(slots[i]).second) return fail(ctx, WHISPER_E_INVAL, "slots must be distinct");
        if (!ctx->slots[slots[i]].active)
            return fail(ctx, WHISPER_E_STATE, "slot " + std::to_string(slots[i]) + " is idle");
        if (forced && (forced[i] < 0 || forced[i] >= ctx->p.n_vocab))
            return fail(ctx, WHISPER_E_INVAL, "forced token out of range");
    }
    return guarded(ctx, [&]() -> whisper_status {
        ctx->eng->decode_step(slots, n, forced, out_tokens, out_logits, true);
        ctx->stats.decode_steps += 1;
        ctx->stats.rows_decoded += n;
        for (int i = 0; i < n; ++i) {
            SlotState& s = ctx->slots[slots[i]];
            ctx->stats.positions_attended += s.steps + 1;
            if (s.steps >= s.n_prompt - 1) s.generated++;
            s.steps++;
            if (s.generated == s.max_new) s.active = false;
        }
        return WHISPER_OK;
    });
}

whisper_status whisper_batch_decode_step_noalloc(whisper_ctx* ctx, const int32_t* slots, int32_t n,
                                                 int32_t* out_tokens_dev) {
    if (!ctx) return fail(nullptr, WHISPER_E_INVAL, "ctx is NULL");
    if (ctx->broken) return fail(ctx, WHISPER_E_DEVICE, "context unusable after a device error");
    if (ctx->p.n_text_layer == 0) return fail(ctx, WHISPER_E_STATE, "not available for an encoder-only CTC model");
    if (n < 1 || n > WHISPER_NOALLOC_MAX_ROWS || n > ctx->p.max_slots)
        return fail(ctx, WHISPER_E_CAPACITY, "n must be in 1.." + std::to_string(WHISPER_NOALLOC_MAX_ROWS) +
                                                 " and at most max_slots");
    if (!slots) return fail(ctx, WHISPER_E_INVAL, "slots must not be NULL");
    bool seen[128] = {};
    for (int i = 0; i < n; ++i) {
        if (slots[i] < 0 || slots[i] >= ctx->p.max_slots)
            return fail(ctx, WHISPER_E_CAPACITY, "slot " + std::to_string(slots[i]) + " outside 0..max_slots-1");
        if (seen[slots[i]]) return fail(ctx, WHISPER_E_INVAL, "slots must be distinct");
        seen[slots[i]] = true;
        if (!ctx->slots[slots[i]].active)
            return fail(ctx, WHISPER_E_STATE, "slot " + std::to_string(slots[i]) + " is idle");
    }
    return guarded(ctx, [&]() -> whisper_status {
        ctx->eng->decode_step_noalloc(slots, n, out_tokens_dev);
        ctx->stats.decode_steps += 1;
        ctx->stats.rows_decoded += n;
        for (int i = 0; i < n; ++i) {
            SlotState& s = ctx->slots[slots[i]];
            ctx->stats.positions_attended += s.steps + 1;
            if (s.steps >= s.n_prompt - 1) s.generated++;
            s.steps++;
            if (s.generated == s.max_new) s.active = false;
        }
        return WHISPER_OK;
    });
}

whisper_status whisper_slot_tokens(whisper_ctx* ctx, int32_t slot, int32_t* dst, int32_t cap, int32_t* n_out) {
    if (!ctx) return fail(nullptr, WHISPER_E_INVAL, "ctx is NULL");
    if (ctx->broken) return fail(ctx, WHISPER_E_DEVICE, "context unusable after a device error");
    if (ctx->p.n_text_layer == 0) return fail(ctx, WHISPER_E_STATE, "not available for an encoder-only CTC model");
    if (slot < 0 || slot >= ctx->p.max_slots) return fail(ctx, WHISPER_E_CAPACITY, "slot outside 0..max_slots-1");
    if (!n_out || (cap > 0 && !dst) || cap < 0) return fail(ctx, WHISPER_E_INVAL, "bad output buffer");
    const int g = ctx->slots[slot].generated;
    const int k = g < cap ? g : cap;
    return guarded(ctx, [&]() -> whisper_status {
        ctx->eng->read_tokens(slot, k, dst);
        *n_out = g;
        return WHISPER_OK;
    });
}

// End-of-text results: a segment that produced its end-of-text token keeps
// the tokens before it (n_tokens); the rest of its token_buf range is -1.
static void finish_stops(const std::vector<int32_t>& stop_of, whisper_result* results, int32_t* token_buf, int n) {
    for (int i = 0; i < n; ++i) {
        const int32_t k = stop_of[i];
        if (k < 0 || k >= results[i].n_tokens) continue;
        for (int32_t j = k; j < results[i].n_tokens; ++j) token_buf[results[i].token_offset + j] = -1;
        results[i].n_tokens = k;
    }
}

whisper_status whisper_set_decoding(whisper_ctx* ctx, int32_t eot, const int32_t* suppress, int32_t n_suppress,
                                    const int32_t* suppress_first, int32_t n_first) {
    if (!ctx) return fail(nullptr, WHISPER_E_INVAL, "ctx is NULL");
    if (ctx->broken) return fail(ctx, WHISPER_E_DEVICE, "context unusable after a device error");
    if (ctx->p.n_text_layer == 0) return fail(ctx, WHISPER_E_STATE, "not available for an encoder-only CTC model");
    const int V = ctx->p.n_vocab;
    if (eot < -1 || eot >= V) return fail(ctx, WHISPER_E_INVAL, "eot must be -1 or a token id");
    if (n_suppress < 0 || n_first < 0 || (n_suppress > 0 && !suppress) || (n_first > 0 && !suppress_first))
        return fail(ctx, WHISPER_E_INVAL, "bad suppress list");
    std::set<int> never, first;
    for (int i = 0; i < n_suppress; ++i) {
        if (suppress[i] < 0 || suppress[i] >= V) return fail(ctx, WHISPER_E_INVAL, "suppressed id out of range");
        never.insert(suppress[i]);
    }
    for (int i = 0; i < n_first; ++i) {
        if (suppress_first[i] < 0 || suppress_first[i] >= V)
            return fail(ctx, WHISPER_E_INVAL, "suppressed id out of range");
        first.insert(suppress_first[i]);
    }
    std::set<int> both = never;
    both.insert(first.begin(), first.end());
    if ((int)both.size() >= V) return fail(ctx, WHISPER_E_INVAL, "the filters would suppress every token");
    for (auto& s : ctx->slots)
        if (s.active) return fail(ctx, WHISPER_E_STATE, "decoding options change with every slot idle");
    return guarded(ctx, [&]() -> whisper_status {
        const std::vector<int> a(never.begin(), never.end()), b(first.begin(), first.end());
        ctx->eng->set_decoding(eot, a.data(), (int)a.size(), b.data(), (int)b.size());
        ctx->eot = eot;
        return WHISPER_OK;
    });
}

whisper_status whisper_batch_serve(whisper_ctx* ctx, const whisper_segment* segs, int32_t n, int32_t* token_buf,
                                   int64_t token_buf_cap, whisper_result* results, int32_t realtime) {
    if (!ctx) return fail(nullptr, WHISPER_E_INVAL, "ctx is NULL");
    if (ctx->broken) return fail(ctx, WHISPER_E_DEVICE, "context unusable after a device error");
    if (n < 0) return fail(ctx, WHISPER_E_INVAL, "n must be >= 0");
    if (n == 0) return WHISPER_OK;
    if (!segs || !results) return fail(ctx, WHISPER_E_INVAL, "segs and results must not be NULL");
    for (auto& s : ctx->slots)
        if (s.active) return fail(ctx, WHISPER_E_STATE, "transcribe needs every slot idle");
    std::vector<wmi::QueuedSegment> q(n);
    for (int i = 0; i < n; ++i) {
        const std::string bad = check_segment(ctx->p, segs[i], i);
        if (!bad.empty()) return fail(ctx, WHISPER_E_INVAL, bad);
        if (realtime && segs[i].arrival_us < 0)
            return fail(ctx, WHISPER_E_INVAL, "segment " + std::to_string(i) + ": arrival_us must be >= 0");
        // with prefill, a segment's decode steps are its max_new_tokens alone
        q[i] = wmi::QueuedSegment{segs[i].arrival_us, segs[i].user_id, segs[i].segment_id,
                                  ctx->p.prefill ? 1 : segs[i].n_prompt, segs[i].max_new_tokens};
    }
    int64_t total = 0;
    const std::vector<int64_t> off = offsets_of(q, &total);
    if (!token_buf || token_buf_cap < total)
        return fail(ctx, WHISPER_E_BUFFER, "token_buf needs " + std::to_string(total) + " entries");
    for (int i = 0; i < n; ++i)
        results[i] = whisper_result{segs[i].segment_id, off[i], 0, segs[i].user_id, WHISPER_OK,
                                    segs[i].max_new_tokens, 0};
    if (ctx->p.n_text_layer == 0) return serve_ctc(ctx, segs, n, q, off, token_buf, results, realtime != 0);
    const whisper_status r = guarded(ctx, [&]() -> whisper_status {
        EngineBackend be;
        be.c = ctx;
        be.segs = segs;
        be.realtime = realtime != 0;
        be.eot_stop = ctx->eot >= 0;
        be.steps.assign(ctx->p.max_slots, 0);
        be.mark_of.assign(n, -1);
        be.stop_of.assign(n, -1);
        ctx->eng->mark_reset();
        ctx->eng->stop_reset();
        be.t0 = EngineBackend::clock::now();
        wmi::BatchPolicy pol;
        pol.dynamic = ctx->p.batch_policy == 1;
        pol.step_cost_us = ctx->p.step_cost_us;
        pol.max_wait_us = 1000LL * ctx->p.max_wait_ms;
        wmi::run_continuous_batching(q, ctx->p.max_slots, ctx->p.max_encode_batch, ctx->p.refill_min, off, token_buf,
                                     be, be.realtime, pol);
        const double total_ms =
            std::chrono::duration<double, std::milli>(EngineBackend::clock::now() - be.t0).count();
        ctx->stats.engine_host_ms += be.engine_ms;
        ctx->stats.batcher_host_ms += total_ms - be.engine_ms;
        const std::vector<double> t = ctx->eng->mark_times_us();
        for (int i = 0; i < n; ++i)
            if (be.mark_of[i] >= 0) results[i].finish_us = (int64_t)t[be.mark_of[i]];
        finish_stops(be.stop_of, results, token_buf, n);
        return WHISPER_OK;
    });
    for (auto& s : ctx->slots) s = SlotState();
    if (r != WHISPER_OK)
        for (int i = 0; i < n; ++i) { results[i].status = r; results[i].n_tokens = 0; }
    return r;
}

whisper_status whisper_batch_transcribe(whisper_ctx* ctx, const whisper_segment* segs, int32_t n, int32_t* token_buf,
                                        int64_t token_buf_cap, whisper_result* results) {
    return whisper_batch_serve(ctx, segs, n, token_buf, token_buf_cap, results, 0);
}

whisper_status whisper_debug_copy(whisper_ctx* ctx, int32_t tensor, int32_t index, void* dst, size_t bytes) {
    if (!ctx) return fail(nullptr, WHISPER_E_INVAL, "ctx is NULL");
    if (ctx->broken) return fail(ctx, WHISPER_E_DEVICE, "context unusable after a device error");
    if (!dst) return fail(ctx, WHISPER_E_INVAL, "dst is NULL");
    return guarded(ctx, [&]() -> whisper_status {
        ctx->eng->debug_copy(tensor, index, dst, bytes);
        return WHISPER_OK;
    });
}

whisper_status whisper_profile_enable(whisper_ctx* ctx, int32_t kernel, int32_t enable) {
    if (!ctx) return fail(nullptr, WHISPER_E_INVAL, "ctx is NULL");
    if (ctx->broken) return fail(ctx, WHISPER_E_DEVICE, "context unusable after a device error");
    if (kernel < 0 || kernel >= WHISPER_K_COUNT) return fail(ctx, WHISPER_E_INVAL, "unknown kernel id");
    return guarded(ctx, [&]() -> whisper_status {
        ctx->eng->profile_enable(kernel, enable != 0);
        return WHISPER_OK;
    });
}

whisper_status whisper_profile_read(whisper_ctx* ctx, int32_t kernel, double* total_ms, int64_t* launches) {
    if (!ctx) return fail(nullptr, WHISPER_E_INVAL, "ctx is NULL");
    if (ctx->broken) return fail(ctx, WHISPER_E_DEVICE, "context unusable after a device error");
    if (kernel < 0 || kernel >= WHISPER_K_COUNT || !total_ms || !launches)
        return fail(ctx, WHISPER_E_INVAL, "unknown kernel id or NULL output");
    return guarded(ctx, [&]() -> whisper_status {
        ctx->eng->profile_read(kernel, total_ms, launches);
        return WHISPER_OK;
    });
}

whisper_status whisper_time_kernel(whisper_ctx* ctx, int32_t kernel, int32_t n_rows, int32_t reps, double* avg_us) {
    if (!ctx) return fail(nullptr, WHISPER_E_INVAL, "ctx is NULL");
    if (ctx->broken) return fail(ctx, WHISPER_E_DEVICE, "context unusable after a device error");
    if (ctx->p.n_text_layer == 0) return fail(ctx, WHISPER_E_STATE, "not available for an encoder-only CTC model");
    if (kernel != WHISPER_K_CROSS_ATTN || !avg_us) return fail(ctx, WHISPER_E_INVAL, "only WHISPER_K_CROSS_ATTN; avg_us not NULL");
    if (n_rows < 1 || n_rows > ctx->p.max_slots || reps < 1)
        return fail(ctx, WHISPER_E_INVAL, "n_rows in 1..max_slots and reps >= 1");
    return guarded(ctx, [&]() -> whisper_status {
        *avg_us = ctx->eng->time_cross_attn(n_rows, reps);
        return WHISPER_OK;
    });
}

whisper_status whisper_stats_read(whisper_ctx* ctx, whisper_stats* out, int32_t reset) {
    if (!ctx) return fail(nullptr, WHISPER_E_INVAL, "ctx is NULL");
    if (!out) return fail(ctx, WHISPER_E_INVAL, "out is NULL");
    *out = ctx->stats;
    if (reset) ctx->stats = whisper_stats{};
    return WHISPER_OK;
}

whisper_status whisper_test_batcher(int32_t n, const int64_t* arrival_us, const int32_t* user_id,
                                    const int64_t* segment_id, const int32_t* max_new_tokens, int32_t slots,
                                    int32_t encode_batch, int32_t refill_min, int32_t* token_buf,
                                    int64_t token_buf_cap, whisper_result* results, int32_t* events,
                                    int32_t events_cap, int32_t* n_events, int32_t realtime, int64_t encode_us,
                                    int64_t step_us, int32_t eot, int32_t batch_policy, int64_t step_cost_us,
                                    int64_t max_wait_us) {
    if (n < 0 || (n > 0 && (!arrival_us || !user_id || !segment_id || !max_new_tokens || !results)))
        return fail(nullptr, WHISPER_E_INVAL, "bad arguments");
    if (slots < 1 || encode_batch < 1 || refill_min < 1)
        return fail(nullptr, WHISPER_E_INVAL, "slots, encode_batch and refill_min must be >= 1");
    if (encode_us < 0 || step_us < 0) return fail(nullptr, WHISPER_E_INVAL, "clock steps must be >= 0");
    if (batch_policy < 0 || batch_policy > 1 || step_cost_us < 0 || max_wait_us < 0)
        return fail(nullptr, WHISPER_E_INVAL, "bad batch policy");
    std::vector<wmi::QueuedSegment> q(n);
    for (int i = 0; i < n; ++i) {
        if (max_new_tokens[i] < 1) return fail(nullptr, WHISPER_E_INVAL, "max_new_tokens must be >= 1");
        q[i] = wmi::QueuedSegment{arrival_us[i], user_id[i], segment_id[i], 1, max_new_tokens[i]};
    }
    int64_t total = 0;
    const std::vector<int64_t> off = offsets_of(q, &total);
    if ((total > 0 && !token_buf) || token_buf_cap < total)
        return fail(nullptr, WHISPER_E_BUFFER, "token_buf needs " + std::to_string(total) + " entries");
    std::vector<int32_t> ev;
    std::vector<int64_t> fin(n, 0);
    std::vector<int32_t> stop_of(n, -1);
    FakeBackend be;
    be.seg_ids = segment_id;
    be.events = &ev;
    be.finish_at = &fin;
    be.stop_of = &stop_of;
    be.encode_us = encode_us;
    be.step_us = step_us;
    be.eot = eot < 0 ? -1 : eot;
    be.seg.assign(slots, -1);
    be.gen.assign(slots, 0);
    be.stop_at.assign(slots, -1);
    try {
        wmi::BatchPolicy pol;
        pol.dynamic = batch_policy == 1;
        pol.step_cost_us = step_cost_us;
        pol.max_wait_us = max_wait_us;
        wmi::run_continuous_batching(q, slots, encode_batch, refill_min, off, token_buf, be, realtime != 0, pol);
    } catch (const std::exception& e) {
        return fail(nullptr, WHISPER_E_INVAL, e.what());
    }
    for (int i = 0; i < n; ++i)
        results[i] = whisper_result{segment_id[i], off[i], fin[i], user_id[i], WHISPER_OK, max_new_tokens[i], 0};
    finish_stops(stop_of, results, token_buf, n);
    if (n_events) *n_events = (int32_t)(ev.size() / 3);
    if (events) {
        const size_t k = ev.size() < (size_t)events_cap * 3 ? ev.size() : (size_t)events_cap * 3;
        memcpy(events, ev.data(), k * sizeof(int32_t));
    }
    return WHISPER_OK;
}

whisper_status whisper_test_greedy_keys(const float* logits, int32_t rows, int32_t n_vocab,
                                        const uint32_t* excluded, int32_t* tokens, int32_t* no_token) {
    if (rows < 0 || n_vocab < 1 || (rows > 0 && (!logits || !tokens || !no_token)))
        return fail(nullptr, WHISPER_E_INVAL, "bad arguments");
    wmi::greedy_keys_host(logits, rows, n_vocab, excluded, tokens, no_token);
    return WHISPER_OK;
}

}  // extern "C"
