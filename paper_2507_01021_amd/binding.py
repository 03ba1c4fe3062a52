"""ctypes binding of libwhisper_mi355x.so (include/whisper_mi355x.h).

Argument marshalling only: every step of the path runs inside the HIP
library. The functions keep the C names; `Context` wraps a context for
numpy callers. Loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libwhisper_mi355x.so")

OK, E_INVAL, E_NOMEM, E_DEVICE, E_CAPACITY, E_STATE, E_BUFFER, E_FORMAT = 0, -1, -2, -3, -4, -5, -6, -7
DTYPE_F32, DTYPE_BF16 = 0, 1
T_MEL, T_ENC_OUT, T_CROSS_K, T_CROSS_V, T_CTC_LOGITS, T_CTC_IDS = 0, 1, 2, 3, 4, 5
K_CROSS_ATTN, K_ENC_GEMM, K_SELF_ATTN, K_ENC_ATTN, K_ENC_PASS, K_DEC_STEP, K_FRONT_END = 0, 1, 2, 3, 4, 5, 6
K_CROSS_ATTN_STEP = 7

EXPORTS = (
    "whisper_params_from_blob", "whisper_ctx_create", "whisper_ctx_destroy", "whisper_last_error",
    "whisper_ctx_set_stream", "whisper_batch_encode", "whisper_batch_decode_step",
    "whisper_batch_decode_step_noalloc",
    "whisper_slot_tokens", "whisper_batch_transcribe", "whisper_batch_serve", "whisper_debug_copy",
    "whisper_profile_enable", "whisper_profile_read", "whisper_time_kernel", "whisper_stats_read",
    "whisper_set_decoding", "whisper_test_batcher", "whisper_test_greedy_keys",
)


class whisper_params(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "n_mels", "n_audio_ctx", "n_audio_state", "n_audio_head", "n_audio_layer",
        "n_vocab", "n_text_ctx", "n_text_state", "n_text_head", "n_text_layer",
        "dtype", "max_slots", "max_encode_batch", "pad_mode", "refill_min", "batch_policy",
        "step_cost_us", "max_wait_ms", "ctc_beam", "prefill")]


class whisper_segment(C.Structure):
    _fields_ = [
        ("audio", C.c_void_p), ("n_samples", C.c_int32), ("audio_on_device", C.c_int32),
        ("segment_id", C.c_int64), ("prompt", C.POINTER(C.c_int32)), ("n_prompt", C.c_int32),
        ("max_new_tokens", C.c_int32), ("user_id", C.c_int32), ("reserved", C.c_int32),
        ("arrival_us", C.c_int64)]


class whisper_result(C.Structure):
    _fields_ = [("segment_id", C.c_int64), ("token_offset", C.c_int64), ("finish_us", C.c_int64),
                ("user_id", C.c_int32), ("status", C.c_int32), ("n_tokens", C.c_int32), ("reserved", C.c_int32)]


class whisper_stats(C.Structure):
    _fields_ = [(n, C.c_int64) for n in (
        "encode_passes", "segments_encoded", "decode_steps", "rows_decoded", "positions_attended",
        "refill_batches")] + [("batcher_host_ms", C.c_double), ("engine_host_ms", C.c_double)]


_lib = None


def load(path: str = LIB_PATH) -> C.CDLL:
    """Loads the library (once). Raises if it is missing: there is no
    fallback path."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2507_01021_amd.build`")
    lib = C.CDLL(path)
    i32, i64, vp, pi32 = C.c_int32, C.c_int64, C.c_void_p, C.POINTER(C.c_int32)
    sig = {
        "whisper_params_from_blob": (i32, [vp, C.c_size_t, C.POINTER(whisper_params)]),
        "whisper_ctx_create": (i32, [C.POINTER(whisper_params), vp, C.c_size_t, C.c_int, C.POINTER(vp)]),
        "whisper_ctx_destroy": (None, [vp]),
        "whisper_last_error": (C.c_char_p, [vp]),
        "whisper_ctx_set_stream": (i32, [vp, vp]),
        "whisper_batch_encode": (i32, [vp, C.POINTER(whisper_segment), i32, pi32]),
        "whisper_batch_decode_step": (i32, [vp, pi32, i32, pi32, pi32, C.POINTER(C.c_float)]),
        "whisper_batch_decode_step_noalloc": (i32, [vp, pi32, i32, vp]),
        "whisper_slot_tokens": (i32, [vp, i32, pi32, i32, pi32]),
        "whisper_batch_transcribe": (i32, [vp, C.POINTER(whisper_segment), i32, pi32, i64,
                                          C.POINTER(whisper_result)]),
        "whisper_batch_serve": (i32, [vp, C.POINTER(whisper_segment), i32, pi32, i64,
                                     C.POINTER(whisper_result), i32]),
        "whisper_debug_copy": (i32, [vp, i32, i32, vp, C.c_size_t]),
        "whisper_profile_enable": (i32, [vp, i32, i32]),
        "whisper_profile_read": (i32, [vp, i32, C.POINTER(C.c_double), C.POINTER(i64)]),
        "whisper_time_kernel": (i32, [vp, i32, i32, i32, C.POINTER(C.c_double)]),
        "whisper_stats_read": (i32, [vp, C.POINTER(whisper_stats), i32]),
        "whisper_set_decoding": (i32, [vp, i32, pi32, i32, pi32, i32]),
        "whisper_test_batcher": (i32, [i32, C.POINTER(i64), pi32, C.POINTER(i64), pi32, i32, i32, i32,
                                      pi32, i64, C.POINTER(whisper_result), pi32, i32, pi32, i32, i64, i64, i32,
                                      i32, i64, i64]),
        "whisper_test_greedy_keys": (i32, [C.POINTER(C.c_float), i32, i32, C.POINTER(C.c_uint32), pi32, pi32]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


class WhisperError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"status {status}: {msg}")
        self.status = status


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(C.POINTER(ctype))


def _check(st: int, ctx_handle=None):
    if st != OK:
        msg = load().whisper_last_error(ctx_handle)
        raise WhisperError(st, msg.decode() if msg else "")


def params_from_blob(blob: np.ndarray) -> whisper_params:
    p = whisper_params()
    _check(load().whisper_params_from_blob(blob.ctypes.data, blob.nbytes, C.byref(p)))
    return p


class _SegArray:
    """Keeps the ctypes segment array and every buffer it points to alive."""

    def __init__(self, segs, device_audio=None):
        self.keep = []
        self.arr = (whisper_segment * max(1, len(segs)))()
        for i, s in enumerate(segs):
            pr = np.ascontiguousarray(s.prompt, dtype=np.int32)
            self.keep.append(pr)
            e = self.arr[i]
            if device_audio is not None:
                e.audio = C.c_void_p(int(device_audio[i]))
                e.audio_on_device = 1
            else:
                a = np.ascontiguousarray(s.audio, dtype=np.float32)
                self.keep.append(a)
                e.audio = C.c_void_p(a.ctypes.data)
                e.audio_on_device = 0
            e.n_samples = int(s.audio.size if hasattr(s.audio, "size") else len(s.audio))
            e.segment_id = int(s.segment_id)
            e.prompt = _ptr(pr, C.c_int32)
            e.n_prompt = int(pr.size)
            e.max_new_tokens = int(s.max_new_tokens)
            e.user_id = int(s.user_id)
            e.arrival_us = int(s.arrival_us)


class Context:
    """One engine context on a HIP device."""

    def __init__(self, blob: np.ndarray, max_slots: int = 32, max_encode_batch: int = 0,
                 pad_mode: int = 0, refill_min: int = 0, device: int = 0, batch_policy: int = 0,
                 step_cost_us: int = 0, max_wait_ms: int = 0, ctc_beam: int = 0, prefill: int = 0):
        lib = load()
        p = params_from_blob(blob)
        p.max_slots, p.max_encode_batch, p.pad_mode, p.refill_min = (
            max_slots, max_encode_batch, pad_mode, refill_min)
        p.batch_policy, p.step_cost_us, p.max_wait_ms = batch_policy, step_cost_us, max_wait_ms
        p.ctc_beam, p.prefill = ctc_beam, prefill
        self.params = p
        h = C.c_void_p()
        _check(lib.whisper_ctx_create(C.byref(p), blob.ctypes.data, blob.nbytes, device, C.byref(h)))
        self.h = h
        self.n_vocab = p.n_vocab

    def close(self):
        if getattr(self, "h", None):
            load().whisper_ctx_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *a):
        self.close()

    def _check(self, st):
        _check(st, self.h)

    def set_stream(self, stream_handle: int | None):
        self._check(load().whisper_ctx_set_stream(self.h, C.c_void_p(stream_handle or 0)))

    def encode(self, segs, slots, device_audio=None):
        sa = _SegArray(segs, device_audio)
        sl = np.ascontiguousarray(slots, dtype=np.int32)
        self._check(load().whisper_batch_encode(self.h, sa.arr, len(segs), _ptr(sl, C.c_int32)))

    def decode_step(self, slots, forced=None, logits=False):
        sl = np.ascontiguousarray(slots, dtype=np.int32)
        n = sl.size
        toks = np.empty(n, dtype=np.int32)
        fo = None if forced is None else np.ascontiguousarray(forced, dtype=np.int32)
        lg = np.empty((n, self.n_vocab), dtype=np.float32) if logits else None
        self._check(load().whisper_batch_decode_step(
            self.h, _ptr(sl, C.c_int32), n, None if fo is None else _ptr(fo, C.c_int32),
            _ptr(toks, C.c_int32), None if lg is None else _ptr(lg, C.c_float)))
        return (toks, lg) if logits else toks

    def decode_step_noalloc(self, slots, out_tokens_dev: int = 0):
        """whisper_batch_decode_step_noalloc: enqueues one greedy step that
        allocates nothing; out_tokens_dev is a device address of len(slots)
        int32 (or 0). Returns without waiting for the device."""
        sl = np.ascontiguousarray(slots, dtype=np.int32)
        self._check(load().whisper_batch_decode_step_noalloc(self.h, _ptr(sl, C.c_int32), sl.size,
                                                             C.c_void_p(out_tokens_dev or None)))

    def slot_tokens(self, slot: int, cap: int = 448):
        buf = np.empty(cap, dtype=np.int32)
        n = C.c_int32()
        self._check(load().whisper_slot_tokens(self.h, slot, _ptr(buf, C.c_int32), cap, C.byref(n)))
        return buf[: min(n.value, cap)].copy()

    def transcribe(self, segs, device_audio=None, realtime: bool = False):
        """whisper_batch_transcribe, or whisper_batch_serve with real-time
        admission (segments served from their arrival_us) when realtime."""
        sa = _SegArray(segs, device_audio)
        total = sum(int(s.max_new_tokens) for s in segs)
        buf = np.zeros(max(1, total), dtype=np.int32)
        res = (whisper_result * max(1, len(segs)))()
        if realtime:
            st = load().whisper_batch_serve(self.h, sa.arr, len(segs), _ptr(buf, C.c_int32), buf.size, res, 1)
        else:
            st = load().whisper_batch_transcribe(self.h, sa.arr, len(segs), _ptr(buf, C.c_int32), buf.size, res)
        self._check(st)
        out = []
        for i in range(len(segs)):
            r = res[i]
            out.append({"user_id": r.user_id, "segment_id": r.segment_id, "status": r.status,
                        "finish_us": r.finish_us, "tokens": buf[r.token_offset: r.token_offset + r.n_tokens].copy()})
        return out

    def debug_copy(self, tensor: int, index: int, shape, dtype=np.float32):
        out = np.empty(shape, dtype=dtype)
        self._check(load().whisper_debug_copy(self.h, tensor, index, out.ctypes.data, out.nbytes))
        return out

    def profile_enable(self, kernel: int, on: bool = True):
        self._check(load().whisper_profile_enable(self.h, kernel, 1 if on else 0))

    def profile_read(self, kernel: int):
        ms, n = C.c_double(), C.c_int64()
        self._check(load().whisper_profile_read(self.h, kernel, C.byref(ms), C.byref(n)))
        return ms.value, n.value

    def time_kernel(self, kernel: int, n_rows: int, reps: int) -> float:
        """Average microseconds of reps back-to-back launches over slots 0..n_rows-1."""
        us = C.c_double()
        self._check(load().whisper_time_kernel(self.h, kernel, n_rows, reps, C.byref(us)))
        return us.value

    def set_decoding(self, eot: int = -1, suppress=(), suppress_first=()):
        a = np.ascontiguousarray(list(suppress), dtype=np.int32)
        b = np.ascontiguousarray(list(suppress_first), dtype=np.int32)
        self._check(load().whisper_set_decoding(self.h, int(eot), _ptr(a, C.c_int32), a.size, _ptr(b, C.c_int32),
                                                b.size))

    def stats(self, reset: bool = False) -> dict:
        st = whisper_stats()
        self._check(load().whisper_stats_read(self.h, C.byref(st), 1 if reset else 0))
        return {name: getattr(st, name) for name, _ in whisper_stats._fields_}


def test_batcher(arrival_us, user_id, segment_id, max_new_tokens, slots, encode_batch, refill_min,
                 events_cap=100000, realtime=False, encode_us=0, step_us=0, eot=-1, policy=0,
                 step_cost_us=2000, max_wait_us=0):
    """Runs the library's scheduler on the host with its fake engine (and,
    with realtime, real-time admission on the fake engine's simulated clock)."""
    lib = load()
    n = len(arrival_us)
    a = np.ascontiguousarray(arrival_us, dtype=np.int64)
    u = np.ascontiguousarray(user_id, dtype=np.int32)
    s = np.ascontiguousarray(segment_id, dtype=np.int64)
    m = np.ascontiguousarray(max_new_tokens, dtype=np.int32)
    total = int(m.sum())
    buf = np.zeros(max(1, total), dtype=np.int32)
    res = (whisper_result * max(1, n))()
    ev = np.zeros(3 * events_cap, dtype=np.int32)
    ne = C.c_int32()
    st = lib.whisper_test_batcher(n, _ptr(a, C.c_int64), _ptr(u, C.c_int32), _ptr(s, C.c_int64),
                                  _ptr(m, C.c_int32), slots, encode_batch, refill_min,
                                  _ptr(buf, C.c_int32), buf.size, res, _ptr(ev, C.c_int32),
                                  events_cap, C.byref(ne), 1 if realtime else 0, encode_us, step_us, eot,
                                  policy, step_cost_us, max_wait_us)
    _check(st)
    results = [(res[i].segment_id, res[i].token_offset, res[i].user_id, res[i].status, res[i].n_tokens)
               for i in range(n)]
    if realtime:
        return buf[:total], results, ev[: 3 * min(ne.value, events_cap)].reshape(-1, 3), \
            [res[i].finish_us for i in range(n)]
    return buf[:total], results, ev[: 3 * min(ne.value, events_cap)].reshape(-1, 3)


def test_greedy_keys(logits, excluded_ids=()):
    """The greedy choice of every row of `logits` [rows, n_vocab] computed on
    the host with the decode step's key arithmetic; ids in excluded_ids are
    skipped. Returns (tokens, no_token flags)."""
    lib = load()
    lg = np.ascontiguousarray(logits, dtype=np.float32)
    rows, V = lg.shape
    mask = None
    if len(excluded_ids):
        m = np.zeros(V // 32 + 1, dtype=np.uint32)
        for i in excluded_ids:
            m[i >> 5] |= np.uint32(1 << (i & 31))
        mask = m
    tok = np.zeros(max(1, rows), dtype=np.int32)
    bad = np.zeros(max(1, rows), dtype=np.int32)
    _check(lib.whisper_test_greedy_keys(_ptr(lg, C.c_float), rows, V,
                                        None if mask is None else _ptr(mask, C.c_uint32),
                                        _ptr(tok, C.c_int32), _ptr(bad, C.c_int32)))
    return tok[:rows], bad[:rows]
