#include "batcher.h"

#include <stdint.h>

#include <algorithm>
#include <deque>
#include <set>
#include <stdexcept>
#include <tuple>

namespace wmi {

void run_continuous_batching(const std::vector<QueuedSegment>& segs, int n_slots, int encode_batch, int refill_min,
                             const std::vector<int64_t>& offsets, int32_t* token_buf, BatchBackend& be,
                             bool realtime, const BatchPolicy& policy) {
    if (n_slots < 1 || encode_batch < 1 || refill_min < 1) throw std::invalid_argument("batcher: bad parameters");
    const int n = (int)segs.size();
    std::vector<int> order(n);
    for (int i = 0; i < n; ++i) order[i] = i;
    std::sort(order.begin(), order.end(), [&](int a, int b) {
        return std::make_tuple(segs[a].arrival_us, segs[a].user_id, segs[a].segment_id, a) <
               std::make_tuple(segs[b].arrival_us, segs[b].user_id, segs[b].segment_id, b);
    });
    // Not yet arrived (real-time admission), in arrival order.
    std::deque<int> pending(order.begin(), order.end());
    // Queued, in serving order: (key, user, segment id, input index).
    auto key_of = [&](int i) {
        int64_t k = segs[i].arrival_us;
        if (policy.dynamic)
            k += policy.step_cost_us * (int64_t)(segs[i].n_prompt + segs[i].max_new_tokens - 1);
        return std::make_tuple(k, segs[i].user_id, segs[i].segment_id, i);
    };
    std::set<std::tuple<int64_t, int32_t, int64_t, int>> queue;
    int64_t now = 0;
    auto oldest_wait = [&]() {  // the longest wait among queued segments
        int64_t first = INT64_MAX;
        for (const auto& e : queue) first = std::min(first, segs[std::get<3>(e)].arrival_us);
        return now - first;
    };
    auto admit = [&]() {
        now = realtime ? be.now_us() : 0;
        while (!pending.empty() && (!realtime || segs[pending.front()].arrival_us <= now)) {
            queue.insert(key_of(pending.front()));
            pending.pop_front();
        }
    };

    std::set<int> free_slots;
    for (int s = 0; s < n_slots; ++s) free_slots.insert(s);
    std::vector<int> seg_of(n_slots, -1), steps_left(n_slots, 0);
    std::vector<int64_t> first_step(n_slots, 0);  // index of the first step each slot's segment ran in
    int64_t steps = 0;
    int active = 0;
    std::vector<int> idx, slots, list, stopped;
    auto retire = [&](int s) {
        const int i = seg_of[s];
        be.retire(s, i, segs[i].max_new_tokens, token_buf + offsets[i]);
        seg_of[s] = -1;
        free_slots.insert(s);
        --active;
    };
    for (;;) {
        admit();
        const int nfree = n_slots - active;
        bool go = !queue.empty() && nfree > 0;
        if (go && policy.dynamic) {
            // A pass of min(queued, refill_min) segments; while fewer than
            // refill_min are queued, wait (bounded) for more to arrive.
            const int q = (int)queue.size();
            go = active < refill_min ||
                 (nfree >= std::min(q, refill_min) &&
                  (q >= refill_min || pending.empty() || oldest_wait() >= policy.max_wait_us));
        } else if (go) {
            go = nfree >= refill_min || active < refill_min;
        }
        if (go) {
            while (!queue.empty() && !free_slots.empty()) {
                idx.clear();
                slots.clear();
                while (!queue.empty() && !free_slots.empty() && (int)idx.size() < encode_batch) {
                    const int i = std::get<3>(*queue.begin());
                    queue.erase(queue.begin());
                    const int s = *free_slots.begin();
                    free_slots.erase(free_slots.begin());
                    idx.push_back(i);
                    slots.push_back(s);
                    seg_of[s] = i;
                    steps_left[s] = segs[i].n_prompt + segs[i].max_new_tokens - 1;
                    first_step[s] = steps;
                }
                be.encode(idx.data(), (int)idx.size(), slots.data());
                active += (int)idx.size();
            }
        }
        if (active == 0) {
            if (pending.empty()) break;  // nothing active, queued or still to arrive
            be.wait_until(segs[pending.front()].arrival_us);
            continue;
        }
        list.clear();
        for (int s = 0; s < n_slots; ++s)
            if (seg_of[s] >= 0) list.push_back(s);
        be.step(list.data(), (int)list.size());
        for (int s : list)
            if (--steps_left[s] == 0) retire(s);
        int64_t as_of = -1;
        stopped.clear();
        if (be.stops(stopped, as_of))
            for (int s : stopped)  // only the segment that was in the slot at step as_of
                if (seg_of[s] >= 0 && first_step[s] <= as_of) retire(s);
        ++steps;
    }
    be.finish();
}

void run_queue_passes(const std::vector<QueuedSegment>& segs, int encode_batch, BatchBackend& be, bool realtime,
                      const BatchPolicy& policy) {
    if (encode_batch < 1) throw std::invalid_argument("batcher: bad parameters");
    const int n = (int)segs.size();
    std::vector<int> order(n);
    for (int i = 0; i < n; ++i) order[i] = i;
    std::sort(order.begin(), order.end(), [&](int a, int b) {
        return std::make_tuple(segs[a].arrival_us, segs[a].user_id, segs[a].segment_id, a) <
               std::make_tuple(segs[b].arrival_us, segs[b].user_id, segs[b].segment_id, b);
    });
    size_t next = 0, head = 0;  // order[head, next): queued; order[next, n): still to arrive
    std::vector<int> idx;
    while (head < (size_t)n) {
        const int64_t now = realtime ? be.now_us() : 0;
        while (next < (size_t)n && (!realtime || segs[order[next]].arrival_us <= now)) ++next;
        if (head == next) {  // nothing queued: wait for the next arrival
            be.wait_until(segs[order[next]].arrival_us);
            continue;
        }
        if (realtime && policy.dynamic && (int)(next - head) < encode_batch && next < (size_t)n) {
            const int64_t deadline = segs[order[head]].arrival_us + policy.max_wait_us;
            if (now < deadline) {
                be.wait_until(std::min(deadline, segs[order[next]].arrival_us));
                continue;
            }
        }
        idx.clear();
        while (head < next && (int)idx.size() < encode_batch) idx.push_back(order[head++]);
        be.encode(idx.data(), (int)idx.size(), nullptr);
    }
    be.finish();
}

}  // namespace wmi
