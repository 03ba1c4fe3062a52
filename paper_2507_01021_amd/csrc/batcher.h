// Continuous batcher: the central priority queue over every user's segments
// feeding a fixed set of decode slots (Section 2.2: a central queue batches
// segments from all active users into one shared inference pipeline, with
// continuous batching to keep the batch full).
//
// Policy: segments are served in (arrival_us, user_id, segment_id, input
// index) order. Whenever at least `refill_min` slots are free, or fewer than
// `refill_min` are active, every free slot (lowest index first) is filled
// from the queue, in encode passes of at most `encode_batch` segments. Every
// active slot then advances one decode step; a slot retires after exactly
// n_prompt + max_new_tokens - 1 steps and its tokens are copied to the
// caller's buffer at the segment's input-order offset. Results do not depend
// on the policy's parameters, because each segment is an independent unit.
//
// Real-time admission (optional): a segment joins the queue only once the
// backend's clock has reached its arrival_us; with nothing to run, the
// batcher waits for the next arrival. Without it every segment is queued at
// the start (arrival_us is then only the priority key).
//
// Dynamic policy (optional, Section 2.2's dynamic batching by segment length
// and wait time): the queue is ordered by arrival_us + step_cost_us x the
// segment's decode steps (n_prompt + max_new_tokens - 1), so a shorter
// segment goes ahead of longer ones that arrived less than the difference in
// their service times earlier (shortest-first with aging); and refills are
// formed for encoder efficiency (an encoder pass costs a large fixed part
// plus a part per segment): free slots are refilled once they can take
// min(queued, refill_min) segments and either refill_min are queued, no
// segment is still to arrive, or the oldest queued one has waited
// max_wait_us; and, as in continuous batching, whenever fewer than
// refill_min slots are active.
//
// End-of-text stop (optional): the backend may report slots whose segment
// has produced its end-of-text token as of some earlier step; such a slot
// retires at once (its tokens up to end of text are the result), freeing it
// for the queue. A slot may run a step or two past its end of text before
// this is known; those tokens are never delivered.
#pragma once

#include <stdint.h>

#include <vector>

namespace wmi {

struct QueuedSegment {
    int64_t arrival_us;
    int32_t user_id;
    int64_t segment_id;
    int32_t n_prompt;
    int32_t max_new_tokens;
};

class BatchBackend {
   public:
    virtual ~BatchBackend() {}
    // Encode segments idx[0..n) into slots[0..n).
    virtual void encode(const int* idx, int n, const int* slots) = 0;
    // One decode step over the listed slots (ascending).
    virtual void step(const int* slots, int n) = 0;
    // Slot finished segment idx with the step just run: deliver its `count`
    // tokens to dst (may be deferred until finish()) and note its finish time.
    virtual void retire(int slot, int idx, int count, int32_t* dst) = 0;
    virtual void finish() = 0;
    // Real-time admission only: microseconds since the run started (work
    // already submitted has completed), and waiting until that clock reaches t.
    virtual int64_t now_us() { return 0; }
    virtual void wait_until(int64_t) {}
    // End-of-text stop only, called after every step: slots known to have
    // reached end of text as of step `as_of` (steps count from 0); false if
    // nothing is known yet.
    virtual bool stops(std::vector<int>& slots, int64_t& as_of) { return false; }
};

struct BatchPolicy {
    bool dynamic = false;
    int64_t step_cost_us = 2000;  // dynamic: estimated microseconds per decode step
    int64_t max_wait_us = 0;      // dynamic + real time: longest wait for a fuller refill
};

// Runs the whole queue; offsets[i] is segment i's first token in token_buf.
void run_continuous_batching(const std::vector<QueuedSegment>& segs, int n_slots, int encode_batch, int refill_min,
                             const std::vector<int64_t>& offsets, int32_t* token_buf, BatchBackend& be,
                             bool realtime = false, const BatchPolicy& policy = BatchPolicy());

// Encoder-only models (CTC): the same queue (arrival order, real-time
// admission) served in passes of up to encode_batch segments, with no slots
// or decode steps; be.encode(idx, n, nullptr) computes and delivers the
// segments' results. With the dynamic policy and real-time admission, a
// pass is held back (while more segments are still to arrive) until
// encode_batch are queued or the oldest queued one has waited max_wait_us.
void run_queue_passes(const std::vector<QueuedSegment>& segs, int encode_batch, BatchBackend& be,
                      bool realtime = false, const BatchPolicy& policy = BatchPolicy());

}  // namespace wmi
