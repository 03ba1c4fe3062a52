"""The continuous batcher (central priority queue + slot refill, Section
2.2), run inside the library against its host-only fake engine and checked
against a brute-force simulation of the same policy."""
import os

import numpy as np
import pytest

from paper_2507_01021_amd import binding, synth


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("library not built")
    return binding.load()


def fake_tokens(seg_id, n):
    return [(seg_id * 7919 + j * 104729) % 50000 for j in range(n)]


def simulate(arrival, user, seg, new, slots, eb, R):
    """Brute force: every engine call the policy makes, in order."""
    n = len(arrival)
    queue = sorted(range(n), key=lambda i: (arrival[i], user[i], seg[i], i))
    free = list(range(slots))
    seg_of = [-1] * slots
    left = [0] * slots
    events = []
    while True:
        active = slots - len(free)
        if queue and free and (len(free) >= R or active < R):
            while queue and free:
                k = 0
                while queue and free and k < eb:
                    i = queue.pop(0)
                    s = min(free)
                    free.remove(s)
                    seg_of[s], left[s] = i, 1 + new[i] - 1
                    events.append((0, s, i))
                    k += 1
        active = slots - len(free)
        if active == 0:
            break
        lst = [s for s in range(slots) if seg_of[s] >= 0]
        events.append((1, len(lst), 0))
        for s in lst:
            left[s] -= 1
            if left[s] == 0:
                seg_of[s] = -1
                free.append(s)
    return events


def workload(n, users, seed):
    segs = synth.poisson_users(synth.TINY, users, n, 5.0, 1, 9, seed=seed) if n else []
    return ([s.arrival_us for s in segs], [s.user_id for s in segs], [s.segment_id for s in segs],
            [s.max_new_tokens for s in segs])


@pytest.mark.parametrize("n,users,slots,eb,R", [(1, 1, 1, 1, 1), (7, 2, 3, 2, 1), (40, 8, 8, 3, 4),
                                               (64, 8, 16, 16, 16), (30, 5, 40, 7, 16)])
def test_schedule_matches_bruteforce(lib, n, users, slots, eb, R):
    a, u, s, m = workload(n, users, seed=n)
    toks, res, ev = binding.test_batcher(a, u, s, m, slots, eb, R)
    assert [tuple(e) for e in ev] == simulate(a, u, s, m, slots, eb, R)
    off = np.concatenate([[0], np.cumsum(m)[:-1]])
    for i in range(n):
        assert res[i] == (s[i], off[i], u[i], 0, m[i])
        assert list(toks[off[i]: off[i] + m[i]]) == fake_tokens(s[i], m[i])


def test_every_segment_served_once_and_results_independent_of_policy(lib):
    a, u, s, m = workload(50, 6, seed=3)
    ref = None
    for slots, eb, R in [(1, 1, 1), (4, 2, 2), (16, 16, 16), (50, 5, 3), (7, 7, 100)]:
        toks, res, ev = binding.test_batcher(a, u, s, m, slots, eb, R)
        enc = [e for e in ev if e[0] == 0]
        assert sorted(e[2] for e in enc) == list(range(50))      # each segment encoded exactly once
        assert max(e[1] for e in enc) < slots
        # steps = longest chain of per-slot work; every active slot advances each step
        assert sum(e[1] for e in ev if e[0] == 1) == sum(m)       # n_prompt = 1 -> m steps each
        if ref is None:
            ref = (toks.copy(), res)
        else:
            assert np.array_equal(toks, ref[0]) and res == ref[1]


def test_queue_order_is_arrival_then_user_then_id(lib):
    a = [5, 5, 1, 5, 0]
    u = [2, 1, 9, 1, 3]
    s = [10, 11, 12, 9, 13]
    m = [1, 1, 1, 1, 1]
    _, _, ev = binding.test_batcher(a, u, s, m, 1, 1, 1)
    assert [e[2] for e in ev if e[0] == 0] == [4, 2, 3, 1, 0]


def test_bad_arguments(lib):
    with pytest.raises(binding.WhisperError):
        binding.test_batcher([0], [0], [0], [0], 1, 1, 1)
    with pytest.raises(binding.WhisperError):
        binding.test_batcher([0], [0], [0], [1], 0, 1, 1)
    toks, res, ev = binding.test_batcher([], [], [], [], 2, 1, 1)
    assert len(res) == 0 and len(ev) == 0


def simulate_realtime(arrival, user, seg, new, slots, eb, R, enc_us, step_us):
    """Brute force of real-time admission on the fake engine's clock: a
    segment is queued once the clock has reached its arrival; encoding costs
    enc_us per segment, a step step_us; an idle batcher jumps to the next
    arrival. Returns the engine calls and every segment's finish time."""
    n = len(arrival)
    pending = sorted(range(n), key=lambda i: (arrival[i], user[i], seg[i], i))
    queue, free = [], list(range(slots))
    seg_of, left = [-1] * slots, [0] * slots
    events, finish, clock = [], [0] * n, 0
    while True:
        while pending and arrival[pending[0]] <= clock:
            queue.append(pending.pop(0))
        active = slots - len(free)
        if queue and free and (len(free) >= R or active < R):
            while queue and free:
                k = 0
                while queue and free and k < eb:
                    i = queue.pop(0)
                    s = min(free)
                    free.remove(s)
                    seg_of[s], left[s] = i, new[i]
                    events.append((0, s, i))
                    k += 1
                clock += enc_us * k
        if slots - len(free) == 0:
            if not pending:
                break
            clock = max(clock, arrival[pending[0]])
            continue
        lst = [s for s in range(slots) if seg_of[s] >= 0]
        events.append((1, len(lst), 0))
        clock += step_us
        for s in lst:
            left[s] -= 1
            if left[s] == 0:
                finish[seg_of[s]] = clock
                seg_of[s] = -1
                free.append(s)
    return events, finish


@pytest.mark.parametrize("n,users,slots,eb,R,enc,step", [(1, 1, 1, 1, 1, 100, 1000), (12, 3, 4, 2, 1, 50_000, 400_000),
                                                         (40, 8, 8, 3, 4, 20_000, 150_000),
                                                         (64, 8, 16, 16, 16, 5_000, 30_000),
                                                         (30, 5, 40, 7, 16, 0, 1)])
def test_realtime_admission_matches_bruteforce(lib, n, users, slots, eb, R, enc, step):
    """Segments are served only once they have arrived; with nothing to run
    the batcher waits for the next arrival (simulated clock)."""
    a, u, s, m = workload(n, users, seed=n + 7)
    toks, res, ev, fin = binding.test_batcher(a, u, s, m, slots, eb, R, realtime=True, encode_us=enc, step_us=step)
    want_ev, want_fin = simulate_realtime(a, u, s, m, slots, eb, R, enc, step)
    assert [tuple(e) for e in ev] == want_ev
    assert fin == want_fin
    assert all(f >= t for f, t in zip(fin, a))
    off = np.concatenate([[0], np.cumsum(m)[:-1]])
    for i in range(n):
        assert list(toks[off[i]: off[i] + m[i]]) == fake_tokens(s[i], m[i])


def simulate_eot(arrival, user, seg, new, slots, eb, R, eot):
    """Brute force of end-of-text stop with the fake engine: a slot's stop is
    known one step after it happened (the snapshot before the latest); a
    segment's result is its tokens before end of text."""
    n = len(arrival)
    queue = sorted(range(n), key=lambda i: (arrival[i], user[i], seg[i], i))
    free = list(range(slots))
    seg_of, left, first = [-1] * slots, [0] * slots, [0] * slots
    gen, stop_at = [0] * slots, [-1] * slots
    snaps, events, n_tok, steps = [], [], list(new), 0

    def retire(s):
        i = seg_of[s]
        if 0 <= stop_at[s] < new[i]:
            n_tok[i] = stop_at[s]
        seg_of[s] = -1
        free.append(s)

    while True:
        active = slots - len(free)
        if queue and free and (len(free) >= R or active < R):
            while queue and free:
                k = 0
                while queue and free and k < eb:
                    i = queue.pop(0)
                    s = min(free)
                    free.remove(s)
                    seg_of[s], left[s], first[s], gen[s], stop_at[s] = i, new[i], steps, 0, -1
                    events.append((0, s, i))
                    k += 1
        if slots - len(free) == 0:
            break
        lst = [s for s in range(slots) if seg_of[s] >= 0]
        events.append((1, len(lst), 0))
        for s in lst:
            g = gen[s]
            gen[s] += 1
            if stop_at[s] < 0 and fake_tokens(seg[seg_of[s]], g + 1)[g] == eot:
                stop_at[s] = g
        snaps.append(list(stop_at))
        for s in lst:
            left[s] -= 1
            if left[s] == 0:
                retire(s)
        if len(snaps) >= 2:
            p, as_of = snaps[-2], len(snaps) - 2
            for s in range(slots):
                if p[s] >= 0 and seg_of[s] >= 0 and first[s] <= as_of:
                    retire(s)
        steps += 1
    return events, n_tok


@pytest.mark.parametrize("n,users,slots,eb,R", [(12, 3, 4, 2, 1), (40, 8, 8, 3, 4), (64, 8, 16, 16, 16)])
def test_end_of_text_stop_matches_bruteforce(lib, n, users, slots, eb, R):
    a, u, s, m = workload(n, users, seed=n + 11)
    long_ones = [i for i in range(n) if m[i] >= 4][:3]
    for i in long_ones:
        eot = fake_tokens(s[i], 3)[2]          # segment i stops after 2 tokens
        toks, res, ev = binding.test_batcher(a, u, s, m, slots, eb, R, eot=eot)
        want_ev, want_n = simulate_eot(a, u, s, m, slots, eb, R, eot)
        assert [tuple(e) for e in ev] == want_ev
        assert [r[4] for r in res] == want_n
        assert want_n[i] == 2
        off = np.concatenate([[0], np.cumsum(m)[:-1]])
        for j in range(n):
            got = list(toks[off[j]: off[j] + m[j]])
            assert got[:want_n[j]] == fake_tokens(s[j], want_n[j])
            assert got[want_n[j]:] == [-1] * (m[j] - want_n[j])
            assert eot not in got[:want_n[j]]


def simulate_dynamic(arrival, user, seg, new, slots, eb, R, enc_us, step_us, cost_us, wait_us):
    """Brute force of the dynamic policy with real-time admission on the
    fake clock: queue ordered by arrival + cost_us x steps (then user,
    segment, index); refill when fewer than R slots are active, or when
    min(queued, R) slots are free and R are queued, or all have arrived, or
    the oldest queued segment has waited wait_us."""
    n = len(arrival)
    pending = sorted(range(n), key=lambda i: (arrival[i], user[i], seg[i], i))
    key = lambda i: (arrival[i] + cost_us * new[i], user[i], seg[i], i)
    queue, free = [], list(range(slots))
    seg_of, left = [-1] * slots, [0] * slots
    events, finish, clock = [], [0] * n, 0
    while True:
        while pending and arrival[pending[0]] <= clock:
            queue.append(pending.pop(0))
        queue.sort(key=key)
        active = slots - len(free)
        waited = queue and clock - min(arrival[i] for i in queue) >= wait_us
        arrived_all = all(arrival[i] <= clock for i in range(len(arrival)))
        if queue and free and (active < R or (len(free) >= min(R, len(queue)) and
                                              (len(queue) >= R or arrived_all or waited))):
            while queue and free:
                k = 0
                while queue and free and k < eb:
                    i = queue.pop(0)
                    s = min(free)
                    free.remove(s)
                    seg_of[s], left[s] = i, new[i]
                    events.append((0, s, i))
                    k += 1
                clock += enc_us * k
        if slots - len(free) == 0:
            if not pending:
                break
            clock = max(clock, arrival[pending[0]])
            continue
        lst = [s for s in range(slots) if seg_of[s] >= 0]
        events.append((1, len(lst), 0))
        clock += step_us
        for s in lst:
            left[s] -= 1
            if left[s] == 0:
                finish[seg_of[s]] = clock
                seg_of[s] = -1
                free.append(s)
    return events, finish


@pytest.mark.parametrize("n,users,slots,eb,R,cost,wait", [(12, 3, 4, 2, 4, 400_000, 0),
                                                          (40, 8, 8, 3, 4, 150_000, 300_000),
                                                          (64, 8, 16, 16, 16, 30_000, 100_000),
                                                          (64, 8, 40, 16, 8, 30_000, 2_000_000),
                                                          (30, 5, 6, 7, 6, 1_000_000, 50_000)])
def test_dynamic_policy_matches_bruteforce(lib, n, users, slots, eb, R, cost, wait):
    a, u, s, m = workload(n, users, seed=n + 23)
    toks, res, ev, fin = binding.test_batcher(a, u, s, m, slots, eb, R, realtime=True, encode_us=20_000,
                                              step_us=150_000, policy=1, step_cost_us=cost, max_wait_us=wait)
    want_ev, want_fin = simulate_dynamic(a, u, s, m, slots, eb, R, 20_000, 150_000, cost, wait)
    assert [tuple(e) for e in ev] == want_ev
    assert fin == want_fin
    off = np.concatenate([[0], np.cumsum(m)[:-1]])
    for i in range(n):
        assert list(toks[off[i]: off[i] + m[i]]) == fake_tokens(s[i], m[i])


def test_dynamic_order_prefers_short_segments_with_aging(lib):
    """Arrivals 0, 1 ms, 2 ms with 9, 1, 5 steps and cost 1 ms per step:
    keys 9, 2, 7 ms -> served 1, 2, 0 (one slot)."""
    _, _, ev = binding.test_batcher([0, 1000, 2000], [0, 0, 0], [10, 11, 12], [9, 1, 5], 1, 1, 1,
                                    policy=1, step_cost_us=1000)
    assert [e[2] for e in ev if e[0] == 0] == [1, 2, 0]
