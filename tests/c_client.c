/* A plain C client of the library's C ABI (no Python, no PyTorch): reads a
 * weight blob and a file of segments, transcribes them with one
 * whisper_batch_transcribe call on GPU 0 and prints, per segment,
 *     segment_id user_id status n_tokens token...
 * in input order.
 *
 *   whisper_c_client WEIGHTS.blob SEGMENTS.bin [max_slots]
 *
 * SEGMENTS.bin (little-endian): int32 n, then per segment: int32 n_samples,
 * int32 n_prompt, int32 max_new_tokens, int32 user_id, int64 segment_id,
 * int32 prompt[n_prompt], float audio[n_samples] (16 kHz mono).
 * Exit status 0 on success; on an error the library's message goes to
 * stderr and the status is 1 (usage, input) or 2 (a library call).
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "whisper_mi355x.h"

static void* read_file(const char* path, size_t* bytes) {
    FILE* f = fopen(path, "rb");
    if (!f) return NULL;
    if (fseek(f, 0, SEEK_END) != 0) { fclose(f); return NULL; }
    const long n = ftell(f);
    if (n < 0 || fseek(f, 0, SEEK_SET) != 0) { fclose(f); return NULL; }
    void* buf = malloc(n > 0 ? (size_t)n : 1);
    if (buf && fread(buf, 1, (size_t)n, f) != (size_t)n) { free(buf); buf = NULL; }
    fclose(f);
    *bytes = (size_t)n;
    return buf;
}

/* Reads `n` bytes at *pos of the buffer into dst; 0 when the buffer ends first. */
static int take(const unsigned char* buf, size_t size, size_t* pos, void* dst, size_t n) {
    if (n > size - *pos) return 0;
    memcpy(dst, buf + *pos, n);
    *pos += n;
    return 1;
}

int main(int argc, char** argv) {
    if (argc < 3) {
        fprintf(stderr, "usage: %s WEIGHTS.blob SEGMENTS.bin [max_slots]\n", argv[0]);
        return 1;
    }
    size_t blob_bytes = 0, in_bytes = 0;
    void* blob = read_file(argv[1], &blob_bytes);
    unsigned char* in = read_file(argv[2], &in_bytes);
    if (!blob || !in) {
        fprintf(stderr, "cannot read %s\n", !blob ? argv[1] : argv[2]);
        return 1;
    }

    /* segments: prompts and audio stay in the input buffer (copied out to
     * aligned arrays, since the file packs them back to back) */
    size_t pos = 0;
    int32_t n = 0;
    if (!take(in, in_bytes, &pos, &n, 4) || n < 0 || n > 4096) {
        fprintf(stderr, "bad segment count\n");
        return 1;
    }
    whisper_segment* segs = calloc(n > 0 ? (size_t)n : 1, sizeof(whisper_segment));
    int64_t total = 0;
    for (int32_t i = 0; i < n; ++i) {
        int32_t h[4];
        int64_t id;
        if (!take(in, in_bytes, &pos, h, sizeof h) || !take(in, in_bytes, &pos, &id, 8) || h[0] < 0 || h[1] < 0) {
            fprintf(stderr, "segment %d: truncated header\n", i);
            return 1;
        }
        int32_t* prompt = malloc(h[1] > 0 ? (size_t)h[1] * 4 : 4);
        float* audio = malloc(h[0] > 0 ? (size_t)h[0] * 4 : 4);
        if (!take(in, in_bytes, &pos, prompt, (size_t)h[1] * 4) || !take(in, in_bytes, &pos, audio, (size_t)h[0] * 4)) {
            fprintf(stderr, "segment %d: truncated data\n", i);
            return 1;
        }
        segs[i].audio = audio;
        segs[i].n_samples = h[0];
        segs[i].audio_on_device = 0;
        segs[i].prompt = prompt;
        segs[i].n_prompt = h[1];
        segs[i].max_new_tokens = h[2];
        segs[i].user_id = h[3];
        segs[i].segment_id = id;
        segs[i].arrival_us = 0;
        total += h[2] > 0 ? h[2] : 0;
    }

    whisper_params p;
    if (whisper_params_from_blob(blob, blob_bytes, &p) != WHISPER_OK) {
        fprintf(stderr, "whisper_params_from_blob: %s\n", whisper_last_error(NULL));
        return 2;
    }
    p.max_slots = argc > 3 ? atoi(argv[3]) : (n > 0 && n < 32 ? n : 32);
    whisper_ctx* ctx = NULL;
    if (whisper_ctx_create(&p, blob, blob_bytes, 0, &ctx) != WHISPER_OK) {
        fprintf(stderr, "whisper_ctx_create: %s\n", whisper_last_error(NULL));
        return 2;
    }
    int32_t* tokens = malloc(total > 0 ? (size_t)total * 4 : 4);
    whisper_result* res = calloc(n > 0 ? (size_t)n : 1, sizeof(whisper_result));
    const whisper_status st = whisper_batch_transcribe(ctx, segs, n, tokens, total, res);
    if (st != WHISPER_OK) {
        fprintf(stderr, "whisper_batch_transcribe (%d): %s\n", (int)st, whisper_last_error(ctx));
        whisper_ctx_destroy(ctx);
        return 2;
    }
    for (int32_t i = 0; i < n; ++i) {
        printf("%lld %d %d %d", (long long)res[i].segment_id, res[i].user_id, res[i].status, res[i].n_tokens);
        for (int32_t k = 0; k < res[i].n_tokens; ++k) printf(" %d", tokens[res[i].token_offset + k]);
        printf("\n");
    }
    whisper_ctx_destroy(ctx);
    for (int32_t i = 0; i < n; ++i) {
        free((void*)segs[i].prompt);
        free((void*)segs[i].audio);
    }
    free(segs);
    free(tokens);
    free(res);
    free(in);
    free(blob);
    return 0;
}
