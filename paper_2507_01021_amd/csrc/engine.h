// Engine interface (host side, no HIP types): owns the device weights, the
// per-slot decoder caches and state, and the encoder workspace of one
// context, and runs encode passes and decode steps on the context's stream.
// Argument validation happens in the C ABI layer before anything here runs.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <memory>
#include <vector>

#include "../../include/whisper_mi355x.h"

namespace wmi {

struct SegmentDesc {
    const float* audio;
    int n_samples;
    bool on_device;
    const int32_t* prompt;
    int n_prompt;
};

class Engine {
   public:
    virtual ~Engine() {}
    virtual void set_stream(void* hip_stream) = 0;
    // Encodes n segments into the given slots (seating prompts). sync = false
    // leaves the work queued on the stream.
    virtual void encode(const SegmentDesc* segs, int n, const int* slots, bool sync) = 0;
    // One decode step for n slots; optional teacher forcing / outputs (host).
    // sync = false leaves the work queued (outputs must then be null).
    virtual void decode_step(const int* slots, int n, const int* forced, int* out_tok, float* out_logits,
                             bool sync) = 0;
    // One greedy step (no teacher forcing, no logits) that allocates nothing:
    // its per-step temporaries live in the library's static scratch array of
    // this device; only kernels are enqueued on the context's stream and the
    // call does not wait for them. out_tok_dev: device int32[n] or null.
    virtual void decode_step_noalloc(const int* slots, int n, int* out_tok_dev) = 0;
    // Copies gen[slot][0..count) to host dst (synchronous).
    virtual void read_tokens(int slot, int count, int32_t* dst) = 0;
    // Queues a copy of gen[slot][0..count) into host memory owned by the
    // engine; finish_reads() waits and delivers every queued copy to dst.
    virtual void read_tokens_async(int slot, int count, int32_t* dst) = 0;
    // Queues a copy of the slot's end-of-text position (tokens generated
    // before its first end-of-text token, -1 if none), delivered like tokens.
    virtual void read_stop_async(int slot, int32_t* dst) = 0;
    virtual void finish_reads() = 0;
    virtual void sync() = 0;
    virtual void debug_copy(int tensor, int index, void* dst, size_t bytes) = 0;
    virtual void profile_enable(int kernel, bool on) = 0;
    virtual void profile_read(int kernel, double* ms, int64_t* launches) = 0;
    // Average microseconds of `reps` back-to-back launches of the decode
    // cross-attention kernel over slots 0..n-1 (launch i reads layer i mod
    // the decoder depth), between two events on the stream. The slots'
    // caches are read as they are; the attention output buffer is written.
    virtual double time_cross_attn(int n, int reps) = 0;
    // Encoder-only CTC models: enqueues the front end, encoder, head and
    // decoding of n (1..max_encode_batch) segments and returns the batch's
    // ticket (with mark_out: its completion mark). Beam search runs on a
    // second stream, beside the next batch's encoder. read_ctc(ticket)
    // waits for that batch and copies each entry's labels (tokens [n][1500])
    // and their counts; a batch's buffers are reused two batches later, so
    // read each ticket before encoding the batch after next.
    virtual int encode_ctc(const SegmentDesc* segs, int n, int* mark_out) = 0;
    virtual void read_ctc(int ticket, int n, int32_t* tokens, int32_t* counts) = 0;
    // Completion-time marks: mark_reset() starts the clock on the stream,
    // mark() records a point after the work queued so far and returns its
    // index, mark_times_us() waits for the stream and returns every mark's
    // time in microseconds since the reset.
    virtual void mark_reset() = 0;
    // Decoding options for the following steps: end-of-text token (-1: none)
    // and logit filters (ids never chosen / not chosen first), ids < n_vocab.
    virtual void set_decoding(int eot, const int* never, int n_never, const int* first, int n_first) = 0;
    // End-of-text polling: stop_snapshot() queues a copy of every slot's
    // end-of-text position; stop_poll() returns the snapshot before the
    // latest (host memory, max_slots entries) or null; stop_reset() forgets them.
    virtual void stop_snapshot() = 0;
    virtual const int* stop_poll() = 0;
    virtual void stop_reset() = 0;
    virtual int mark() = 0;
    virtual std::vector<double> mark_times_us() = 0;
};

// Throws ArgError (code = whisper_status) or DeviceError.
std::unique_ptr<Engine> make_engine(const whisper_params& p, const void* blob, size_t bytes, int device);

// Host run of the device's greedy-choice keys (largest logit, lowest id on
// ties, excluded ids skipped, token 0 and bad[r] = 1 for a row with none).
void greedy_keys_host(const float* logits, int rows, int V, const unsigned* excluded, int* tokens, int* bad);

// Blob header check; fills the model fields of *out. Returns a whisper_status.
int parse_blob_header(const void* blob, size_t bytes, whisper_params* out, const char** why);

}  // namespace wmi
