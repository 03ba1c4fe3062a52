/*
 * whisper_mi355x.h -- C ABI of the MI355X (gfx950) batched Whisper engine.
 *
 * The engine transcribes a batch of independent speech segments, each with
 * its own prompt, in one multiplexed pass: the method of "Scalable Offline
 * ASR for Command-Style Dictation in Courtrooms" (Section 2.3 and Listing 1:
 * features per segment, padded to a 30 s window, stacked, encoded once,
 * then generated from prompt + no-timestamps tokens), fed by a central
 * priority queue with continuous batching over all users' segments
 * (Section 2.2). Segments are self-contained units, so every segment's
 * result equals the one it would get alone.
 *
 * Conventions for every call:
 *  - Return value: WHISPER_OK (0) or a negative whisper_status. On error,
 *    whisper_last_error(ctx) holds a message, and no slot state changed
 *    (checks run before any device work), except WHISPER_E_DEVICE, after
 *    which the context must be destroyed.
 *  - Ownership: the caller owns every pointer it passes; inputs are only read
 *    during the call, outputs only written during it. The context owns its
 *    device memory (weights, caches, workspaces) and frees it on destroy.
 *  - Host/device: pointers are host memory unless stated otherwise.
 *  - Synchronisation: every call has finished its device work when it
 *    returns. Work runs on the context's stream (see whisper_ctx_set_stream).
 *  - Threads: a context is not thread-safe; use one context per thread.
 *    Contexts are independent of each other.
 */
#ifndef WHISPER_MI355X_H
#define WHISPER_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t whisper_status;
enum {
    WHISPER_OK = 0,
    WHISPER_E_INVAL = -1,    /* bad argument (NULL, out of range, inconsistent) */
    WHISPER_E_NOMEM = -2,    /* device or host allocation failed */
    WHISPER_E_DEVICE = -3,   /* HIP runtime or kernel launch error, or non-finite
                                model output (no admissible token, no finite CTC logit) */
    WHISPER_E_CAPACITY = -4, /* slot index or batch beyond the context's capacity */
    WHISPER_E_STATE = -5,    /* slot busy (encode) or idle (decode step) */
    WHISPER_E_BUFFER = -6,   /* caller's output buffer too small */
    WHISPER_E_FORMAT = -7    /* weight blob malformed or not matching params */
};

enum { WHISPER_DTYPE_F32 = 0, WHISPER_DTYPE_BF16 = 1 };

/*
 * Model shape and runtime options. The model fields must equal the weight
 * blob's header (whisper_params_from_blob fills them from it).
 *   n_mels            80 or 128 log-mel bins
 *   n_audio_ctx       encoder positions, must be 1500 (30 s window)
 *   n_audio_state/head/layer, n_text_state/head/layer: widths, head counts
 *                     (head size must be 64) and layer counts; the two
 *                     widths and head counts must be equal; width at most
 *                     2048, at most 256 decoder layers
 *   n_vocab           vocabulary (output head rows)
 *   n_text_ctx        decoder positions, must be 448
 *   dtype             WHISPER_DTYPE_F32: fp32 storage and arithmetic;
 *                     WHISPER_DTYPE_BF16: bf16 weights and activations, bf16
 *                     MFMA with fp32 accumulation; layer norm, softmax, the
 *                     residual stream and logits in fp32
 *   max_slots         decode slots, 1..128; each holds one segment's
 *                     self- and cross-attention caches
 *   max_encode_batch  segments per encoder pass (workspace size), 1..max_slots;
 *                     0 selects min(max_slots, 32); larger encode requests are
 *                     split into passes of this size
 *   pad_mode          0: zero-pad audio to 30 s before the transform;
 *                     1: transform the segment alone (n/160 frames) and pad
 *                     the normalised features with zeros to 3000 frames
 *   refill_min        continuous batching: refill free slots from the queue
 *                     when at least this many slots are free or fewer than
 *                     this many are active (0 selects 16); results never
 *                     depend on it
 *   batch_policy      0: continuous batching, queue in arrival order;
 *                     1: dynamic: queue ordered by arrival_us + step_cost_us x
 *                     decode steps (shorter segments first, with aging), and
 *                     refills formed for encoder efficiency: free slots are
 *                     refilled once they can take min(queued, refill_min)
 *                     segments and either refill_min are queued, every
 *                     segment has arrived, or the oldest queued one has
 *                     waited max_wait_ms; and whenever fewer than refill_min
 *                     slots are active; results never depend on it
 *   step_cost_us      dynamic policy: estimated decode step time (0 selects 2000)
 *   max_wait_ms       dynamic policy: longest wait for a fuller refill
 *   ctc_beam          CTC models only (0 for others): 0 or 1 greedy best-path
 *                     decoding; 2..16 prefix beam search with that beam and as
 *                     many candidate labels per frame (the frame's most likely
 *                     non-blank ids), no language model; n_vocab <= 4096
 *   prefill           decoder models: 0 feeds the prompt one position per
 *                     decode step (a segment's first n_prompt - 1 steps
 *                     return no token); 1 runs positions 0..n_prompt-2 of
 *                     every encoded segment through the decoder in one pass
 *                     at encode time, so its first decode step returns its
 *                     first token. The tokens are the same either way.
 *                     CTC models: 0
 */
typedef struct {
    int32_t n_mels, n_audio_ctx, n_audio_state, n_audio_head, n_audio_layer;
    int32_t n_vocab, n_text_ctx, n_text_state, n_text_head, n_text_layer;
    int32_t dtype;
    int32_t max_slots;
    int32_t max_encode_batch;
    int32_t pad_mode;
    int32_t refill_min;
    int32_t batch_policy;
    int32_t step_cost_us;
    int32_t max_wait_ms;
    int32_t ctc_beam;
    int32_t prefill;
} whisper_params;

/*
 * One speech segment (a VAD-cut unit of 3-30 s, Section 2.1).
 *   audio           16 kHz mono fp32 samples; host memory, or device memory
 *                   of the context's GPU when audio_on_device is 1
 *   n_samples       1..480000
 *   user_id,
 *   segment_id      echoed verbatim in the results
 *   prompt          host array of n_prompt token ids in [0, n_vocab)
 *   n_prompt        >= 1; n_prompt + max_new_tokens <= n_text_ctx
 *   max_new_tokens  >= 1: exactly this many tokens are generated
 *   arrival_us      queue priority key (whisper_batch_transcribe / _serve); with
 *                   real-time admission also the time, in microseconds after
 *                   the call starts, from which the segment may be served
 */
typedef struct {
    const float* audio;
    int32_t n_samples;
    int32_t audio_on_device;
    int64_t segment_id;
    const int32_t* prompt;
    int32_t n_prompt;
    int32_t max_new_tokens;
    int32_t user_id;
    int32_t reserved;
    int64_t arrival_us;
} whisper_segment;

/* Result of one input segment (results[i] belongs to segs[i]). */
typedef struct {
    int64_t segment_id;
    int64_t token_offset;  /* first token in token_buf */
    int64_t finish_us;     /* when the device had computed the segment's last token,
                              in microseconds after the call started */
    int32_t user_id;
    int32_t status;        /* WHISPER_OK, or the error that stopped the batch */
    int32_t n_tokens;      /* = max_new_tokens when status is WHISPER_OK */
    int32_t reserved;
} whisper_result;

typedef struct whisper_ctx whisper_ctx;

/*
 * Weight blob (host memory): a 256-byte header, then every tensor in the
 * canonical order below, each starting at a multiple of 256 bytes,
 * row-major, fp32 or bf16 (header dtype), no other padding.
 * Header (little-endian): char magic[8] = "WHSPMI01"; int32 version = 1,
 * dtype, n_mels, n_audio_ctx, n_audio_state, n_audio_head, n_audio_layer,
 * n_vocab, n_text_ctx, n_text_state, n_text_head, n_text_layer, n_tensors,
 * reserved; zeros to byte 256.
 * n_text_layer = 0 marks an encoder-only CTC model (the paper's remark that
 * CTC-based recognisers are served the same way, Introduction and the end of
 * Section 2.3): its tensors end after enc.ln_post with ctc.w [n_vocab, d]
 * and ctc.b [n_vocab], and id 0 is the CTC blank. Such a context decodes
 * greedily by best path: over the ceil(n_samples / 320) encoder frames that
 * cover a segment's audio (at most 1500), the most likely id per frame
 * (lowest id on ties), runs of one id merged, blanks dropped. Its segments
 * need no prompt (prompt and n_prompt are ignored) and max_new_tokens
 * (1..1500) is the output capacity: n_tokens <= max_new_tokens labels.
 * A frame with no finite logit (all NaN or -inf) counts as the blank, and
 * the call that reads its batch fails with WHISPER_E_DEVICE.
 * whisper_batch_transcribe / _serve run the same queue in encoder passes
 * of up to max_encode_batch segments; whisper_batch_encode (n <=
 * max_encode_batch, slots ignored) feeds the debug tensors; the decoder
 * calls (decode step, slot tokens, decoding options, cross-attention timing)
 * return WHISPER_E_STATE.
 * Canonical order (d = state, matrices are [out, in], conv [out, in, 3]):
 *   enc.conv1.w [d, n_mels, 3], enc.conv1.b, enc.conv2.w [d, d, 3], enc.conv2.b,
 *   per encoder layer: attn_ln.{g,b}, attn.{q.w, q.b, k.w, v.w, v.b, o.w, o.b},
 *     mlp_ln.{g,b}, mlp.{fc1.w [4d, d], fc1.b, fc2.w [d, 4d], fc2.b},
 *   enc.ln_post.{g,b}, dec.tok_emb [n_vocab, d], dec.pos_emb [n_text_ctx, d],
 *   per decoder layer: attn_ln, attn (as above), cross_ln, cross (as above),
 *     mlp_ln, mlp (as above),
 *   dec.ln.{g,b}.
 */

/* Fills the model fields of *out from a blob header and sets the runtime
 * options to their defaults (max_slots 32, max_encode_batch 0, pad_mode 0,
 * refill_min 0). Returns WHISPER_E_FORMAT for a bad header. */
whisper_status whisper_params_from_blob(const void* blob, size_t blob_bytes,
                                        whisper_params* out);

/* Creates a context on HIP device `device`: copies and repacks the weights
 * (host blob, blob_bytes must match the layout exactly), allocates caches and
 * workspaces. *out is set only on success. Errors: E_INVAL, E_FORMAT,
 * E_NOMEM, E_DEVICE; whisper_last_error(NULL) then holds the message. */
whisper_status whisper_ctx_create(const whisper_params* params, const void* weights,
                                  size_t weights_bytes, int device, whisper_ctx** out);

/* Frees everything the context owns. NULL is allowed. */
void whisper_ctx_destroy(whisper_ctx* ctx);

/* Last error message of ctx (or of the calling thread's last failed create
 * when ctx is NULL); valid until the next call on the same context. */
const char* whisper_last_error(const whisper_ctx* ctx);

/* Runs the context's work on `hip_stream` (a hipStream_t of the context's
 * device, e.g. torch.cuda.current_stream().cuda_stream) from now on; NULL
 * selects the context's own stream. The stream must outlive its use. */
whisper_status whisper_ctx_set_stream(whisper_ctx* ctx, void* hip_stream);

/*
 * Encodes n segments into the given free decode slots (slots[i] receives
 * segs[i]; host array of n distinct indices in [0, max_slots)): log-mel
 * front end, conv stem, encoder, and the cross-attention keys and values of
 * every decoder layer, written into each slot's cache. The slot's
 * self-attention cache is reset and its prompt seated (prefill = 1: prompt
 * positions 0..n_prompt-2 also run through the decoder, filling the cache,
 * so the first decode step is at the last prompt position); the slot is
 * then active. n = 0 is a no-op. Errors: E_INVAL (bad segment or slot), E_STATE
 * (a slot is active), E_CAPACITY (slot >= max_slots). Section 2.3, Listing 1
 * (features, pad to 30 s, stack, encode).
 */
whisper_status whisper_batch_encode(whisper_ctx* ctx, const whisper_segment* segs, int32_t n,
                                    const int32_t* slots);

/*
 * One greedy decoder step for each of the n active slots listed (host array,
 * distinct): every slot feeds the token at its current position (prompt
 * token, or the previous step's token) and advances by one position.
 *   forced      NULL: the next input of a generating slot is this step's
 *               argmax; else forced[i] (host) replaces it (teacher forcing)
 *   out_tokens  NULL or n int32 (host): the argmax of this step (lowest id on
 *               ties), or -1 while the slot is still inside its prompt
 *               (never with prefill = 1)
 *   out_logits  NULL or n * n_vocab fp32 (host): this step's logits
 * A slot whose generated count reaches max_new_tokens becomes idle; its
 * tokens stay readable with whisper_slot_tokens until it is encoded again.
 * n = 0 is a no-op. Errors: E_INVAL, E_STATE (slot idle). Listing 1
 * (generate with prompt + no-timestamps tokens), greedy search.
 */
whisper_status whisper_batch_decode_step(whisper_ctx* ctx, const int32_t* slots, int32_t n,
                                         const int32_t* forced, int32_t* out_tokens,
                                         float* out_logits);

/* Limits of whisper_batch_decode_step_noalloc: its static scratch array per
 * GPU, and the most slots one call steps. */
#define WHISPER_NOALLOC_SCRATCH_BYTES (8u << 20)
#define WHISPER_NOALLOC_MAX_ROWS 64

/*
 * For callers that cannot allocate memory (code under HIP graph capture,
 * tight serving loops, hosts that forbid hipMalloc): the greedy step of
 * whisper_batch_decode_step (no teacher forcing, no logits) that allocates
 * nothing. Its per-step temporaries (slot list, activations, split-K
 * partial sums, greedy-choice keys) live in one static device array of
 * WHISPER_NOALLOC_SCRATCH_BYTES per GPU, held until the process ends,
 * instead of the context's workspaces; the slot list reaches the device as
 * a kernel argument. The call only enqueues kernels on the context's stream
 * (see whisper_ctx_set_stream) and returns without waiting for them; the
 * caller synchronises that stream. The slots' state (position, generated
 * tokens, retirement) advances exactly as with whisper_batch_decode_step.
 *   slots           host array of n distinct active slots,
 *                   1 <= n <= WHISPER_NOALLOC_MAX_ROWS
 *   out_tokens_dev  NULL or device memory of the context's GPU, n int32:
 *                   this step's argmax per slot (-1 inside the prompt),
 *                   written when the enqueued work runs
 * Every call on one GPU shares that GPU's array and leaves its contents
 * behind: calls whose work overlaps in time on one GPU (contexts on
 * different streams) race on it. A row without an admissible token is
 * reported by the next call that synchronises. Errors: E_INVAL, E_STATE
 * (slot idle, or kernel timing on), E_CAPACITY (n above the maximum, or the
 * model's rows need more than the array; the message states the size).
 */
whisper_status whisper_batch_decode_step_noalloc(whisper_ctx* ctx, const int32_t* slots, int32_t n,
                                                 int32_t* out_tokens_dev);

/* Copies the tokens generated so far in `slot` (at most cap) to dst (host)
 * and their count to *n_out. */
whisper_status whisper_slot_tokens(whisper_ctx* ctx, int32_t slot, int32_t* dst, int32_t cap,
                                   int32_t* n_out);

/*
 * Transcribes n segments with continuous batching: segments are queued by
 * (arrival_us, user_id, segment_id, input index); free slots are refilled
 * from the queue (encode passes of up to max_encode_batch), every active
 * slot advances one decode step per iteration, and a slot retires when it
 * has generated max_new_tokens tokens. Section 2.2 (central priority queue,
 * continuous batching) and Section 2.3.
 *   token_buf      host, token_buf_cap int32; segment i's tokens start at
 *                  results[i].token_offset = sum of max_new_tokens of
 *                  segments 0..i-1 (input order, independent of schedule)
 *   results        host, n entries, results[i] describes segs[i]
 * Errors: E_INVAL (any bad segment: nothing runs), E_BUFFER (token_buf_cap
 * below the total; nothing runs, message states the size needed).
 * Requires every slot to be idle on entry; leaves every slot idle.
 */
whisper_status whisper_batch_transcribe(whisper_ctx* ctx, const whisper_segment* segs,
                                        int32_t n, int32_t* token_buf, int64_t token_buf_cap,
                                        whisper_result* results);

/*
 * whisper_batch_transcribe with optional real-time admission (the serving
 * form of Section 2.2's central queue): with realtime != 0 a segment joins
 * the queue only once arrival_us microseconds have passed since the call
 * started; while nothing is runnable the call waits for the next arrival,
 * and every encode pass and decode step completes before the next decision.
 * realtime = 0 is exactly whisper_batch_transcribe. Tokens do not depend on
 * admission times (segments are independent); results[i].finish_us records
 * when each segment's last token was computed.
 */
whisper_status whisper_batch_serve(whisper_ctx* ctx, const whisper_segment* segs, int32_t n,
                                   int32_t* token_buf, int64_t token_buf_cap,
                                   whisper_result* results, int32_t realtime);

/*
 * Decoding options of the context (real use of the listing's generate),
 * for every later decode step; requires every slot idle.
 *   eot             end-of-text token id, or -1 (default): with an id,
 *                   whisper_batch_transcribe / _serve end a segment at its
 *                   first end-of-text token: results[i].n_tokens counts the
 *                   tokens before it (<= max_new_tokens) and the rest of its
 *                   token_buf range is -1. whisper_batch_decode_step does not
 *                   stop by itself (the caller sees the token).
 *   suppress        n_suppress ids that are never chosen (logit filter)
 *   suppress_first  n_first ids that are not chosen as a segment's first
 *                   generated token (e.g. blank and end of text)
 * The filters act on the choice only: out_logits stay unfiltered. Ids must
 * be in [0, n_vocab) and must not cover every id. Defaults: no filters.
 */
whisper_status whisper_set_decoding(whisper_ctx* ctx, int32_t eot, const int32_t* suppress,
                                    int32_t n_suppress, const int32_t* suppress_first,
                                    int32_t n_first);

/* Tensors readable with whisper_debug_copy (test use: per-stage parity). */
enum {
    WHISPER_T_MEL = 0,     /* fp32 [n_mels][3000] normalised log-mel of entry `index`
                              of the last encode pass */
    WHISPER_T_ENC_OUT = 1, /* fp32 [1500][d] encoder output of that entry */
    WHISPER_T_CROSS_K = 2, /* fp32 [n_text_layer][n_head][1500][64] of slot `index` */
    WHISPER_T_CROSS_V = 3, /* same shape, values */
    WHISPER_T_CTC_LOGITS = 4, /* CTC models: fp32 [1500][n_vocab] head output of entry `index`
                                 of the last encode pass */
    WHISPER_T_CTC_IDS = 5     /* CTC models: int32 [1500] most likely id of every frame of it */
};

/* Copies a stage's tensor to dst (host, `bytes` must equal its size). */
whisper_status whisper_debug_copy(whisper_ctx* ctx, int32_t tensor, int32_t index, void* dst,
                                  size_t bytes);

/* Kernels that can be timed live with HIP events (on the stream they are
 * launched on): every launch between enable and read is bracketed. */
enum {
    WHISPER_K_CROSS_ATTN = 0,  /* decode-step cross-attention over the cache */
    WHISPER_K_ENC_GEMM = 1,    /* encoder fc1 GEMM (bf16 MFMA) */
    WHISPER_K_SELF_ATTN = 2,   /* decode-step self-attention */
    WHISPER_K_ENC_ATTN = 3,    /* encoder attention */
    WHISPER_K_ENC_PASS = 4,    /* a whole encode pass (front end to cross-KV) */
    WHISPER_K_DEC_STEP = 5,    /* a whole decode step (embedding to argmax) */
    WHISPER_K_FRONT_END = 6,   /* log-mel front end of an encode pass (audio to normalised mel) */
    WHISPER_K_CROSS_ATTN_STEP = 7, /* decode-step cross-attention as the plain steps run it (captured
                                      graphs, slots split into concurrent chains): each launch's span
                                      from its first workgroup's start to its last one's end, stamped
                                      by the kernel with the device's real-time counter and read after
                                      each step (steps are joined and synchronised meanwhile) */
    WHISPER_K_COUNT = 8
};

/* Starts (enable = 1) or stops (0) timing of `kernel`, clearing its totals. */
whisper_status whisper_profile_enable(whisper_ctx* ctx, int32_t kernel, int32_t enable);

/* Average duration in microseconds of `reps` back-to-back launches of one
 * kernel over rows 0..n_rows-1 mapped to slots 0..n_rows-1, timed by two
 * events on the context's stream (synchronises it). Only
 * WHISPER_K_CROSS_ATTN (the decode cross-attention of Section 2.3's batched
 * decoder: each launch reads the cached encoder keys and values of n_rows
 * slots x all heads, layer i mod the decoder depth for launch i). The slots'
 * caches are read as they are (encode them first for meaningful data) and
 * the step's attention output buffer is overwritten; call it between decode
 * steps, not during a transcribe call. Errors: WHISPER_E_INVAL for another
 * kernel, n_rows outside 1..max_slots, reps < 1 or avg_us NULL. */
whisper_status whisper_time_kernel(whisper_ctx* ctx, int32_t kernel, int32_t n_rows, int32_t reps, double* avg_us);

/* Total milliseconds and launch count of `kernel` since it was enabled
 * (synchronises the stream). */
whisper_status whisper_profile_read(whisper_ctx* ctx, int32_t kernel, double* total_ms,
                                    int64_t* launches);

/*
 * Work counters of a context since creation or the last reset, for
 * throughput and roofline accounting (the decode-step byte count of the
 * method's per-segment caches follows from rows_decoded and
 * positions_attended). Counters cover whisper_batch_encode,
 * whisper_batch_decode_step and whisper_batch_transcribe alike.
 */
typedef struct {
    int64_t encode_passes;      /* encoder passes (each of up to max_encode_batch segments) */
    int64_t segments_encoded;   /* segments through the front end and encoder */
    int64_t decode_steps;       /* decode steps (one token for every listed slot) */
    int64_t rows_decoded;       /* sum over steps of the number of slots stepped */
    int64_t positions_attended; /* sum over steps and slots of self-attention lengths (position + 1) */
    int64_t refill_batches;     /* transcribe: encode calls made by the batcher (slot refills) */
    double batcher_host_ms;     /* transcribe: host time in the batcher's own logic (queue, slot
                                   choice, retirement), engine calls excluded */
    double engine_host_ms;      /* transcribe: host time inside engine calls (enqueue and waits) */
} whisper_stats;

/* Copies the counters to *out (not NULL); reset != 0 then zeroes them. */
whisper_status whisper_stats_read(whisper_ctx* ctx, whisper_stats* out, int32_t reset);

/*
 * Host-only check of the continuous batcher (no device work): runs the
 * scheduler of whisper_batch_transcribe over n fake segments given by
 * arrival_us, user_id, segment_id and max_new_tokens (n_prompt = 1) with
 * `slots` decode slots, encode passes of up to `encode_batch` and refill
 * threshold `refill_min`, against an engine whose token at generated index
 * j of a segment is (segment_id * 7919 + j * 104729) mod 50000.
 * Writes tokens (token_buf) and results as whisper_batch_transcribe would,
 * and, if events is not NULL, the schedule: one int32 triple per engine call
 * (kind 0 = encode, slot, input index) or (kind 1 = decode step, number of
 * active slots, 0), at most events_cap triples, count in *n_events.
 * realtime != 0 runs real-time admission on a simulated clock that starts at
 * 0 and advances by encode_us per encoded segment and step_us per decode
 * step, and jumps to the next arrival when idle; finish_us is that clock
 * after the segment's last step. eot >= 0 stops a segment at its first fake
 * token equal to eot (polled one step late, as the engine's backend does).
 * batch_policy, step_cost_us and max_wait_us select the queue policy as the
 * context fields of those names do (max_wait in microseconds here).
 */
whisper_status whisper_test_batcher(int32_t n, const int64_t* arrival_us, const int32_t* user_id,
                                    const int64_t* segment_id, const int32_t* max_new_tokens,
                                    int32_t slots, int32_t encode_batch, int32_t refill_min,
                                    int32_t* token_buf, int64_t token_buf_cap,
                                    whisper_result* results, int32_t* events,
                                    int32_t events_cap, int32_t* n_events, int32_t realtime,
                                    int64_t encode_us, int64_t step_us, int32_t eot,
                                    int32_t batch_policy, int64_t step_cost_us, int64_t max_wait_us);

/*
 * Host-only check of the greedy choice's arithmetic (no device work): the
 * same 64-bit keys the decode step's kernels compare (value bits mapped to
 * an order-preserving integer, then the complement of the id, so the largest
 * key is the largest logit and, among equal logits, the lowest id; Listing
 * 1's generate read as greedy search). For each of `rows` rows of n_vocab
 * fp32 logits (host, row-major), ids whose bit is set in `excluded` (host,
 * n_vocab / 32 + 1 words, or NULL) are skipped; tokens[r] receives the
 * chosen id, or 0 with no_token[r] = 1 when no id is admissible (the decode
 * step then fails with WHISPER_E_DEVICE). Errors: WHISPER_E_INVAL.
 */
whisper_status whisper_test_greedy_keys(const float* logits, int32_t rows, int32_t n_vocab,
                                        const uint32_t* excluded, int32_t* tokens, int32_t* no_token);

#ifdef __cplusplus
}
#endif

#endif /* WHISPER_MI355X_H */
