// Non-GEMM kernels of the batched Whisper path on gfx950: audio framing
// buffer, log-mel normalisation, layer norm, decoder embedding, encoder
// attention (bf16 MFMA flash attention; fp32 SIMT variant), decode-step
// attention over the KV caches, the skinny decode GEMM (bf16 MFMA streaming
// each weight once) and the greedy argmax step.
#pragma once

#include "common.h"
#include "epilogues.h"
#include "gemm.h"

namespace wmi {

constexpr float LOG2E = 1.4426950408889634f;

// ------------------------------------------------------------- front end

struct SegSrc {
    const float* audio;  // device pointer
    int n;               // samples
    int pad;
};

// xpad[z][i], i in [0, 480400): the 30 s window (zero-padded audio, or the
// segment alone for pad mode 1) with 200 reflected samples at each end.
__global__ void prep_audio_kernel(const SegSrc* __restrict__ src, float* __restrict__ xpad, int pad_mode) {
    const int z = blockIdx.y;
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= 480400) return;
    const float* a = src[z].audio;
    const int n = src[z].n;
    const int len = pad_mode == 0 ? 480000 : n;  // length of the reflected signal
    int s = i - 200;
    if (len == 1) {
        s = 0;
    } else {
        const int period = 2 * (len - 1);
        s = s < 0 ? -s : s;
        s %= period;
        if (s >= len) s = period - s;
    }
    xpad[(long long)z * 480400 + i] = s < n ? a[s] : 0.f;
}

// STFT power of the 3000 frames of each segment on the fp32 matrix cores:
// C[i][f] = sum_n basis[i][n] xpad[160 f + n] over n < 400, where basis rows
// 2k and 2k+1 are the Hann-windowed cosine and sine of bin k, then
// power[z][f][k] = C[2k][f]^2 + C[2k+1][f]^2 (row stride DFT_PS; bins
// 201 .. 207 come from the zero basis rows and are 0).
// basisT is k-major: basisT[n][i] for i < DFT_ROWS (rows 402 .. 415 zero).
// Workgroup: DFT_RH basis rows (13 tiles of 16) x 64 frames, 4 waves, wave w
// takes frames 16 w .. 16 w + 15 against all 13 row tiles with
// v_mfma_f32_16x16x4_f32. K runs in chunks of 16 through LDS (k-major
// tiles, rows padded so the two half-waves of a read hit distinct banks),
// the next chunk's loads held in registers while the current one is used.
constexpr int DFT_ROWS = 416;        // 402 basis rows padded to 26 tiles of 16
constexpr int DFT_RH = DFT_ROWS / 2; // rows per workgroup
constexpr int DFT_FB = 64;           // frames per workgroup
constexpr int DFT_BLD = DFT_FB + 16; // LDS row length of the frame tile
constexpr int DFT_PS = DFT_RH;       // power row stride: bins 0..200, then zeros to 207

typedef float mfma_f32x4_t __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void dft_power_kernel(const float* __restrict__ basisT,
                                                        const float* __restrict__ xpad,
                                                        float* __restrict__ power) {
    __shared__ float As[2][16 * DFT_RH];
    __shared__ float Bs[2][16 * DFT_BLD];
    const int f0 = blockIdx.x * DFT_FB, half = blockIdx.y, z = blockIdx.z;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int fr = lane & 15, fc = lane >> 4;
    const float* x = xpad + (long long)z * 480400;
    // staging: A chunk = 16 k x 208 rows = 832 float4; B chunk = 64 frames x
    // 16 k = 256 float4 (thread: frame tid / 4, k 4 (tid % 4) .. +3)
    const int bj = tid >> 2, bq = tid & 3;
    const float* xb = x + (long long)min(f0 + bj, 2999) * 160 + 4 * bq;
    // A chunk element e = tid + 256 q (q < 3, and q = 3 for tid < 64): k row e / 52, float4 e % 52
    int aoff[4], loff[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int e = min(tid + 256 * q, 831), kk = e / 52, c = e - kk * 52;
        aoff[q] = kk * DFT_ROWS + half * DFT_RH + 4 * c;
        loff[q] = kk * DFT_RH + 4 * c;
    }
    const bool a3 = tid + 768 < 832;
#define WMI_DFT_GLOAD(K0)                                                                               \
    do {                                                                                                \
        a0 = *reinterpret_cast<const float4*>(basisT + (long long)(K0) * DFT_ROWS + aoff[0]);           \
        a1 = *reinterpret_cast<const float4*>(basisT + (long long)(K0) * DFT_ROWS + aoff[1]);           \
        a2 = *reinterpret_cast<const float4*>(basisT + (long long)(K0) * DFT_ROWS + aoff[2]);           \
        if (a3) a3v = *reinterpret_cast<const float4*>(basisT + (long long)(K0) * DFT_ROWS + aoff[3]);  \
        bv = *reinterpret_cast<const float4*>(xb + (K0));                                               \
    } while (0)
#define WMI_DFT_LSTORE(BUF)                                                                             \
    do {                                                                                                \
        *reinterpret_cast<float4*>(&As[BUF][loff[0]]) = a0;                                             \
        *reinterpret_cast<float4*>(&As[BUF][loff[1]]) = a1;                                             \
        *reinterpret_cast<float4*>(&As[BUF][loff[2]]) = a2;                                             \
        if (a3) *reinterpret_cast<float4*>(&As[BUF][loff[3]]) = a3v;                                    \
        Bs[BUF][(4 * bq + 0) * DFT_BLD + bj] = bv.x;                                                    \
        Bs[BUF][(4 * bq + 1) * DFT_BLD + bj] = bv.y;                                                    \
        Bs[BUF][(4 * bq + 2) * DFT_BLD + bj] = bv.z;                                                    \
        Bs[BUF][(4 * bq + 3) * DFT_BLD + bj] = bv.w;                                                    \
    } while (0)
    float4 a0, a1, a2, a3v = float4{0.f, 0.f, 0.f, 0.f}, bv;
    mfma_f32x4_t acc[13];
#pragma unroll
    for (int t = 0; t < 13; ++t) acc[t] = mfma_f32x4_t{0.f, 0.f, 0.f, 0.f};
    constexpr int NCH = 400 / 16;
    WMI_DFT_GLOAD(0);
    WMI_DFT_LSTORE(0);
    __syncthreads();
    for (int ch = 0; ch < NCH; ++ch) {
        const int buf = ch & 1;
        if (ch + 1 < NCH) WMI_DFT_GLOAD((ch + 1) * 16);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const int k = 4 * kk + fc;
            const float b = Bs[buf][k * DFT_BLD + 16 * w + fr];
#pragma unroll
            for (int t = 0; t < 13; ++t)
                acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(As[buf][k * DFT_RH + 16 * t + fr], b, acc[t], 0, 0, 0);
        }
        if (ch + 1 < NCH) WMI_DFT_LSTORE(buf ^ 1);
        __syncthreads();
    }
#undef WMI_DFT_GLOAD
#undef WMI_DFT_LSTORE
    // lane: rows 16 t + 4 fc + r (bins (half * 208 + 16 t + 4 fc) / 2 + 0, 1), frame 16 w + fr
    const int f = f0 + 16 * w + fr;
    if (f >= 3000) return;
    float* prow = power + ((long long)z * 3000 + f) * DFT_PS;
#pragma unroll
    for (int t = 0; t < 13; ++t) {
        const int k = (half * DFT_RH + 16 * t + 4 * fc) >> 1;
        prow[k] = acc[t][0] * acc[t][0] + acc[t][1] * acc[t][1];
        prow[k + 1] = acc[t][2] * acc[t][2] + acc[t][3] * acc[t][3];
    }
}

// Mel projection and log on the fp32 matrix cores: logmel[f][m] =
// log10(max(sum_k fb[m][k] power[f][k], 1e-10)) over the 208 power bins of
// a frame (fb is zero beyond bin 200). fbT is k-major [208][16 MT] (mels
// padded to MT tiles of 16 with zero rows). Workgroup: 64 frames, 4 waves,
// wave w takes frames 16 w .. 16 w + 15 against every mel tile; K in LDS
// chunks of 16, the next chunk's loads held in registers.
template <int MT>
__global__ __launch_bounds__(256) void mel_log_kernel(const float* __restrict__ fbT, const float* __restrict__ power,
                                                      float* __restrict__ logmel, int frames, int n_mels) {
    constexpr int MP = 16 * MT, ALD = MP % 32 == 0 ? MP + 16 : MP, AQ = 16 * MP / 4;
    __shared__ float As[2][16 * ALD];
    __shared__ float Bs[2][16 * DFT_BLD];
    const int f0 = blockIdx.x * 64;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int fr = lane & 15, fc = lane >> 4;
    const int bj = tid >> 2, bq = tid & 3;
    const float* pb = power + (long long)min(f0 + bj, frames - 1) * DFT_PS + 4 * bq;
    float4 a0, a1 = float4{0.f, 0.f, 0.f, 0.f}, bv;
    const bool has1 = tid + 256 < AQ;
    const int e0 = tid, e1 = min(tid + 256, AQ - 1);
    const int k0r = e0 / (MP / 4), c0 = e0 - k0r * (MP / 4), k1r = e1 / (MP / 4), c1 = e1 - k1r * (MP / 4);
#define WMI_MEL_GLOAD(K0)                                                                              \
    do {                                                                                               \
        if (e0 < AQ) a0 = *reinterpret_cast<const float4*>(fbT + (long long)((K0) + k0r) * MP + 4 * c0); \
        if (has1) a1 = *reinterpret_cast<const float4*>(fbT + (long long)((K0) + k1r) * MP + 4 * c1);    \
        bv = *reinterpret_cast<const float4*>(pb + (K0));                                              \
    } while (0)
#define WMI_MEL_LSTORE(BUF)                                                                            \
    do {                                                                                               \
        if (e0 < AQ) *reinterpret_cast<float4*>(&As[BUF][k0r * ALD + 4 * c0]) = a0;                    \
        if (has1) *reinterpret_cast<float4*>(&As[BUF][k1r * ALD + 4 * c1]) = a1;                       \
        Bs[BUF][(4 * bq + 0) * DFT_BLD + bj] = bv.x;                                                   \
        Bs[BUF][(4 * bq + 1) * DFT_BLD + bj] = bv.y;                                                   \
        Bs[BUF][(4 * bq + 2) * DFT_BLD + bj] = bv.z;                                                   \
        Bs[BUF][(4 * bq + 3) * DFT_BLD + bj] = bv.w;                                                   \
    } while (0)
    mfma_f32x4_t acc[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[t] = mfma_f32x4_t{0.f, 0.f, 0.f, 0.f};
    constexpr int NCH = DFT_PS / 16;
    WMI_MEL_GLOAD(0);
    WMI_MEL_LSTORE(0);
    __syncthreads();
    for (int ch = 0; ch < NCH; ++ch) {
        const int buf = ch & 1;
        if (ch + 1 < NCH) WMI_MEL_GLOAD((ch + 1) * 16);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const int k = 4 * kk + fc;
            const float b = Bs[buf][k * DFT_BLD + 16 * w + fr];
#pragma unroll
            for (int t = 0; t < MT; ++t)
                acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(As[buf][k * ALD + 16 * t + fr], b, acc[t], 0, 0, 0);
        }
        if (ch + 1 < NCH) WMI_MEL_LSTORE(buf ^ 1);
        __syncthreads();
    }
#undef WMI_MEL_GLOAD
#undef WMI_MEL_LSTORE
    // lane: mels 16 t + 4 fc .. +3 of frame 16 w + fr
    const int f = f0 + 16 * w + fr;
    if (f >= frames) return;
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        const int m = 16 * t + 4 * fc;
        if (m < n_mels)
            *reinterpret_cast<float4*>(logmel + (long long)f * n_mels + m) =
                float4{log10f(fmaxf(acc[t][0], 1e-10f)), log10f(fmaxf(acc[t][1], 1e-10f)),
                       log10f(fmaxf(acc[t][2], 1e-10f)), log10f(fmaxf(acc[t][3], 1e-10f))};
    }
}

// Log-mel normalisation in two launches over many workgroups: the max over
// each segment's valid frames (MEL_CHUNKS partial maxima per segment, no
// atomics), then clamp to max - 8, (L + 4) / 4, zero the frames beyond the
// segment (pad mode 1). Writes fp32 in place (frame-major [3000][n_mels])
// and the conv input Ypad[z][1 + f][c] in T.
constexpr int MEL_CHUNKS = 16;

// grid (MEL_CHUNKS, segments), 256 threads: part[z][chunk] = max of chunk
__global__ __launch_bounds__(256) void mel_max_kernel(const float* __restrict__ logmel, const int* __restrict__ nvalid,
                                                      int n_mels, float* __restrict__ part) {
    const int z = blockIdx.y, ch = blockIdx.x;
    const float* L = logmel + (long long)z * 3000 * n_mels;
    const int nv = nvalid[z] * n_mels;
    const int per = (3000 * n_mels / MEL_CHUNKS + 255) / 256 * 256;
    const int e0 = ch * per, e1 = min(nv, e0 + per);
    float m = -INFINITY;
    for (int e = e0 + threadIdx.x; e < e1; e += 256) m = fmaxf(m, L[e]);
    m = wave_max(m);
    __shared__ float red[4];
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0)
        part[z * MEL_CHUNKS + ch] = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

// grid (blocks, segments), 256 threads, each thread a run of elements
template <class T>
__global__ __launch_bounds__(256) void mel_norm_kernel(float* __restrict__ logmel, T* __restrict__ ypad,
                                                       const int* __restrict__ nvalid, int n_mels,
                                                       const float* __restrict__ part) {
    const int z = blockIdx.y;
    float mx = -INFINITY;
#pragma unroll
    for (int c = 0; c < MEL_CHUNKS; ++c) mx = fmaxf(mx, part[z * MEL_CHUNKS + c]);
    const float floor_ = mx - 8.0f;
    float* L = logmel + (long long)z * 3000 * n_mels;
    const int nv = nvalid[z] * n_mels;
    T* Y = ypad + (long long)z * 3002 * CP;
    for (int e = blockIdx.x * 256 + threadIdx.x; e < 3000 * n_mels; e += gridDim.x * 256) {
        const int f = e / n_mels, c = e - f * n_mels;
        const float y = e < nv ? (fmaxf(L[e], floor_) + 4.0f) * 0.25f : 0.0f;
        L[e] = y;
        stf(Y + (long long)(f + 1) * CP + c, y);
    }
}

// ------------------------------------------------------------- layer norm
//
// One wavefront per row of width d = 64 * E: fp32 mean and biased variance
// (two passes over registers), eps 1e-5, gain and bias. E is a compile-time
// constant so every load of a row is issued before the first use.

// Layer norm of row `row` held in registers (element lane + 64 e) with
// gain/bias already loaded; DEC: y is a decoder activation (dec_off layout),
// else row-major.
template <int E, bool DEC, class T>
__device__ __forceinline__ void ln_row_apply(const float (&v)[E], int lane, int d, const float (&gg)[E],
                                             const float (&bb)[E], T* __restrict__ y, int row) {
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) s += v[e];
    const float mean = wave_sum(s) / d;
    float q = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) { const float c = v[e] - mean; q += c * c; }
    const float rstd = rsqrtf(wave_sum(q) / d + 1e-5f);
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int c = lane + 64 * e;
        stf(y + (DEC ? dec_off<T>(row, c, d) : (long long)row * d + c), (v[e] - mean) * rstd * gg[e] + bb[e]);
    }
}

template <int E, bool DEC, class T>
__device__ __forceinline__ void ln_row_store(const float (&v)[E], int lane, int d, const float* __restrict__ g,
                                             const float* __restrict__ b, T* __restrict__ y, int row) {
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) s += v[e];
    const float mean = wave_sum(s) / d;
    float q = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) { const float c = v[e] - mean; q += c * c; }
    const float rstd = rsqrtf(wave_sum(q) / d + 1e-5f);
    float gg[E], bb[E];
#pragma unroll
    for (int e = 0; e < E; ++e) { gg[e] = g[lane + 64 * e]; bb[e] = b[lane + 64 * e]; }
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int c = lane + 64 * e;
        stf(y + (DEC ? dec_off<T>(row, c, d) : (long long)row * d + c), (v[e] - mean) * rstd * gg[e] + bb[e]);
    }
}

template <class T, int E>
__global__ __launch_bounds__(256) void layer_norm_kernel(const float* __restrict__ x, T* __restrict__ y,
                                                         const float* __restrict__ g, const float* __restrict__ b,
                                                         int rows) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (row >= rows) return;
    constexpr int d = 64 * E;
    const float* xr = x + (long long)row * d;
    float v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = xr[lane + 64 * e];
    ln_row_store<E, false>(v, lane, d, g, b, y, row);
}

// Decoder input: x = token embedding + position embedding (fp32), then the
// first layer's layer norm. The token embedding (shared with the output
// head) and z use the decoder layout (dec_off); x and pos_emb are row-major.
// Row r is slot list[r] at position rowpos[r], or at the slot's current
// position pos[list[r]] when rowpos is null.
template <class T, int E>
__global__ __launch_bounds__(64) void embed_ln_kernel(const T* __restrict__ tok_emb, const T* __restrict__ pos_emb,
                                                      const int* __restrict__ list, const int* __restrict__ pos,
                                                      const int* __restrict__ rowpos, const int* __restrict__ seq,
                                                      float* __restrict__ x, T* __restrict__ z,
                                                      const float* __restrict__ g, const float* __restrict__ b) {
    constexpr int d = 64 * E;
    const int r = blockIdx.x, lane = threadIdx.x, s = list[r], p = rowpos ? rowpos[r] : pos[s];
    const int tok = seq[s * 448 + p];
    float v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int c = lane + 64 * e;
        v[e] = ldf(tok_emb + dec_off<T>(tok, c, d)) + ldf(pos_emb + (long long)p * d + c);
    }
#pragma unroll
    for (int e = 0; e < E; ++e) x[(long long)r * d + lane + 64 * e] = v[e];
    ln_row_store<E, true>(v, lane, d, g, b, z, r);
}

// Residual update from split-K partial sums, then the next layer norm:
// x[r] += sum_ks part[ks][r] + bias (partials added in ks order), z[r] = LN(x[r])
// (z in the decoder layout). One workgroup per row, thread t owns columns
// 4t..4t+3, so every load of the row is a single 16-byte access issued up
// front; mean and variance are reduced over the workgroup in a fixed order.
template <int E>
constexpr int resid_ln_threads() { return (16 * E + 63) / 64 * 64; }

template <class T, int E, int KS>
__global__ __launch_bounds__(resid_ln_threads<E>()) void resid_ln_kernel(const float* __restrict__ part, int n,
                                                                      const float* __restrict__ bias,
                                                                      float* __restrict__ x, T* __restrict__ z,
                                                                      const float* __restrict__ g,
                                                                      const float* __restrict__ b) {
    constexpr int d = 64 * E, NW = resid_ln_threads<E>() / 64;
    __shared__ float red[2][NW];
    const int r = blockIdx.x, t = threadIdx.x, lane = t & 63, w = t >> 6;
    const bool own = t < 16 * E;
    const int c = 4 * min(t, 16 * E - 1);
    const float4 xv = ld4(x + (long long)r * d + c), bs = ld4(bias + c), gg = ld4(g + c), bb = ld4(b + c);
    float4 p[KS];
#pragma unroll
    for (int k = 0; k < KS; ++k) p[k] = ld4(part + ((long long)k * n + r) * d + c);
    float4 acc = p[0];
#pragma unroll
    for (int k = 1; k < KS; ++k) { acc.x += p[k].x; acc.y += p[k].y; acc.z += p[k].z; acc.w += p[k].w; }
    const float v0 = xv.x + (acc.x + bs.x), v1 = xv.y + (acc.y + bs.y), v2 = xv.z + (acc.z + bs.z),
                v3 = xv.w + (acc.w + bs.w);
    if (own) st4(x + (long long)r * d + c, v0, v1, v2, v3);
    float s = own ? (v0 + v1) + (v2 + v3) : 0.f;
    s = wave_sum(s);
    if (lane == 0) red[0][w] = s;
    __syncthreads();
    float tot = red[0][0];
#pragma unroll
    for (int i = 1; i < NW; ++i) tot += red[0][i];
    const float mean = tot / d;
    const float e0 = v0 - mean, e1 = v1 - mean, e2 = v2 - mean, e3 = v3 - mean;
    float q = own ? (e0 * e0 + e1 * e1) + (e2 * e2 + e3 * e3) : 0.f;
    q = wave_sum(q);
    if (lane == 0) red[1][w] = q;
    __syncthreads();
    float qt = red[1][0];
#pragma unroll
    for (int i = 1; i < NW; ++i) qt += red[1][i];
    const float rstd = rsqrtf(qt / d + 1e-5f);
    if (own)
        st4(z + dec_off<T>(r, c, d), e0 * rstd * gg.x + bb.x, e1 * rstd * gg.y + bb.y, e2 * rstd * gg.z + bb.z,
            e3 * rstd * gg.w + bb.w);
}

// Dispatch on the row width d = 64 * E.
#define WMI_SWITCH_E(d, ...)                                       \
    switch ((d) >> 6) {                                            \
        case 6: { constexpr int E = 6; __VA_ARGS__; break; }       \
        case 8: { constexpr int E = 8; __VA_ARGS__; break; }       \
        case 12: { constexpr int E = 12; __VA_ARGS__; break; }     \
        case 16: { constexpr int E = 16; __VA_ARGS__; break; }     \
        case 20: { constexpr int E = 20; __VA_ARGS__; break; }     \
        case 24: { constexpr int E = 24; __VA_ARGS__; break; }     \
        case 32: { constexpr int E = 32; __VA_ARGS__; break; }     \
        default: throw ArgError(-1, "width must be 64 * {6,8,12,16,20,24,32}"); \
    }

// ------------------------------------------------------------- encoder attention (bf16 MFMA)
//
// Non-causal attention of every query over all 1500 keys, per (segment,
// head). Q, K: [BH][TQ][64] (Q scaled by 1/8), Vt: [BH][64][TQ].
// Workgroup: 4 waves x 64 queries; key tiles of 64 staged in LDS (double
// buffer). Per wave and key tile:
//   S^T[key][q] = K Q^T          (A = K rows from LDS, B = Q in registers)
//   online softmax per query      (each lane owns one query per 16-block)
//   O^T[dim][q] += V^T P^T        (A = V^T from LDS, B = P from registers)
// The P operand uses the lane's own S values directly: the MFMA's reduction
// index k is mapped to keys so that lane l's eight k's are the keys it holds
// (keys 4*(l/16)+{0..3} of two 16-key blocks); V^T is read with the same map.
// LDS tiles are [64 rows][128 bytes] with 16-byte chunks XOR-swizzled by the
// row. The V^T fragment reads are 8 bytes per lane, and the 16 lanes of one
// LDS pass read rows r..r+15 at the same key offset: with the 16-byte swizzle
// alone, rows r and r+8 would hit the same chunk half (a 2-way bank conflict
// on every pass). In the V^T tile the two 8-byte halves of each chunk are
// therefore swapped in rows whose bit 3 is set.
namespace ea {
constexpr int QW = 64;             // queries per wave
constexpr int QB = 4 * QW;         // queries per workgroup
constexpr int KT = 64;             // keys per tile
constexpr int TILE = KT * 64 * 2;  // bytes of one K or V^T tile
}  // namespace ea

__global__ __launch_bounds__(256, 2) void enc_attn_bf16_kernel(const bf16* __restrict__ Q, const bf16* __restrict__ K,
                                                               const bf16* __restrict__ Vt, bf16* __restrict__ O,
                                                               int H, int d) {
    __shared__ __align__(16) unsigned char lds[4 * ea::TILE];
    const int bh = blockIdx.y, bseg = bh / H, h = bh - bseg * H;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int q0 = blockIdx.x * ea::QB + wave * ea::QW;
    const bf16* Qb = Q + (long long)bh * TQ * 64;
    const bf16* Kb = K + (long long)bh * TQ * 64;
    const bf16* Vb = Vt + (long long)bh * 64 * TQ;
    const int fr = lane & 15, fc = lane >> 4;

    // Q fragments (B operand): query q0 + u*16 + fr, dims s*32 + fc*8 .. +7.
    mfma_bf16x8 qf[4][2];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int s = 0; s < 2; ++s)
            qf[u][s] = *reinterpret_cast<const mfma_bf16x8*>(Qb + (long long)(q0 + u * 16 + fr) * 64 + s * 32 + fc * 8);

    mfma_f32x4 o[4][4];  // [dim tile][query tile]
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int u = 0; u < 4; ++u) o[a][u] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
    // Queries arrive scaled by log2(e)/8, so scores are in log2 units. Each
    // query keeps a reference mref (a score it has seen, at most 8 below its
    // running maximum) and the score MFMAs start from -mref, so they return
    // s - mref and the weights are plain exp2 of the result, at most 2^8.
    float mref[4], lrun[4];
    mfma_f32x4 negm[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        mref[u] = 0.f;
        lrun[u] = 0.f;
        negm[u] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
    }
    // staging: thread copies 16-byte chunk (tid & 7) of rows (tid >> 3) and +32
    const int lc = tid & 7, lr = tid >> 3;
    u32x4 rk[2], rv[2];
    auto gload = [&](int k0) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            rk[s] = *reinterpret_cast<const u32x4*>(Kb + (long long)(k0 + lr + 32 * s) * 64 + lc * 8);
            rv[s] = *reinterpret_cast<const u32x4*>(Vb + (long long)(lr + 32 * s) * TQ + k0 + lc * 8);
        }
    };
    const bool vswap = (lr >> 3) & 1;  // bit 3 of this thread's rows lr and lr + 32
    auto lstore = [&](int buf) {
        unsigned char* tk = lds + buf * 2 * ea::TILE;
        unsigned char* tv = tk + ea::TILE;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            *reinterpret_cast<u32x4*>(tk + swz(lr + 32 * s, lc)) = rk[s];
            *reinterpret_cast<u32x4*>(tv + swz(lr + 32 * s, lc)) =
                vswap ? u32x4{rv[s].z, rv[s].w, rv[s].x, rv[s].y} : rv[s];
        }
    };
    const int ntiles = (N_CTX + ea::KT - 1) / ea::KT;
    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < ntiles; ++kt) {
        if (kt + 1 < ntiles) gload((kt + 1) * ea::KT);
        const unsigned char* tk = lds + (kt & 1) * 2 * ea::TILE;
        const unsigned char* tv = tk + ea::TILE;
        // K fragments (A operand of S^T = K Q^T): key a*16 + fr, dims s*32 + fc*8 .. +7
        mfma_bf16x8 kf[4][2];
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int s = 0; s < 2; ++s)
                kf[a][s] = *reinterpret_cast<const mfma_bf16x8*>(tk + swz(a * 16 + fr, 4 * s + fc));
        const int kbase = kt * ea::KT;
        const bool tail = kbase + ea::KT > N_CTX;
        // scores of query tile u relative to its mref: sc[key tile]; keys
        // beyond the window (last tile only) get -inf
        auto scores = [&](int u, mfma_f32x4 (&sc)[4]) {
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                const mfma_f32x4 t = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[a][0], qf[u][0], negm[u], 0, 0, 0);
                sc[a] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[a][1], qf[u][1], t, 0, 0, 0);
            }
            if (tail) {
#pragma unroll
                for (int a = 0; a < 4; ++a)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (kbase + a * 16 + fc * 4 + r >= N_CTX) sc[a][r] = -INFINITY;
            }
        };
        // Software pipeline over the 4 query tiles: the softmax of tile u
        // runs while the score MFMAs of tile u+1 execute, so the vector ALU
        // and the matrix cores work at the same time.
        mfma_f32x4 scur[4], snext[4];
        mfma_bf16x8 pf[4][2];
        scores(0, scur);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            float mx = -INFINITY;
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int r = 0; r < 4; ++r) mx = fmaxf(mx, scur[a][r]);
            mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
            // The first tile sets mref to its maximum; later tiles move it
            // only when their maximum is more than 8 above it, and then scale
            // the sums so far by 2^-(the move).
            if (kt == 0 || __any(mx > 8.f)) {
                const float delta = (kt == 0 || mx > 8.f) ? mx : 0.f;
#pragma unroll
                for (int a = 0; a < 4; ++a)
#pragma unroll
                    for (int r = 0; r < 4; ++r) scur[a][r] -= delta;
                mref[u] += delta;
                negm[u] = mfma_f32x4{-mref[u], -mref[u], -mref[u], -mref[u]};
                if (kt > 0) {
                    const float alpha = exp2_softmax(-delta);
                    lrun[u] *= alpha;
#pragma unroll
                    for (int a = 0; a < 4; ++a)
#pragma unroll
                        for (int r = 0; r < 4; ++r) o[a][u][r] *= alpha;
                }
            }
            if (u < 3) scores(u + 1, snext);
            float ls = 0.f;
            float pv[4][4];
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    pv[a][r] = exp2_softmax(scur[a][r]);
                    ls += pv[a][r];
                }
            ls += __shfl_xor(ls, 16, 64);
            ls += __shfl_xor(ls, 32, 64);
            lrun[u] += ls;
            // P operand for key half s: keys s*32 + fc*4 + {0..3} and s*32 + 16 + fc*4 + {0..3}
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                mfma_bf16x8 p;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    p[r] = (__bf16)pv[2 * s][r];
                    p[4 + r] = (__bf16)pv[2 * s + 1][r];
                }
                pf[u][s] = p;
            }
#pragma unroll
            for (int a = 0; a < 4; ++a) scur[a] = snext[a];
        }
        // O^T += V^T P^T
#pragma unroll
        for (int a = 0; a < 4; ++a) {
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                // V^T row (dim) a*16 + fr, keys s*32 + fc*4 .. +3 and s*32 + 16 + fc*4 .. +3
                // (bit 3 of the row is bit 3 of fr; it selects the swapped halves)
                const int row = a * 16 + fr, half = (fr >> 3) & 1;
                const int kA = s * 32 + fc * 4, kB = kA + 16;
                const u32x2 lo =
                    *reinterpret_cast<const u32x2*>(tv + swz(row, kA >> 3) + ((((kA & 7) >> 2) ^ half) << 3));
                const u32x2 hi =
                    *reinterpret_cast<const u32x2*>(tv + swz(row, kB >> 3) + ((((kB & 7) >> 2) ^ half) << 3));
                union { u32x4 u; mfma_bf16x8 v; } cvt;
                cvt.u = u32x4{lo.x, lo.y, hi.x, hi.y};
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    o[a][u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cvt.v, pf[u][s], o[a][u], 0, 0, 0);
            }
        }
        if (kt + 1 < ntiles) lstore((kt + 1) & 1);
        __syncthreads();
    }
    // lane holds O^T[dim a*16 + fc*4 + r][query q0 + u*16 + fr]
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int q = q0 + u * 16 + fr;
        if (q >= N_CTX) continue;
        const float inv = 1.0f / lrun[u];
        bf16* orow = O + ((long long)bseg * N_CTX + q) * d + h * 64;
#pragma unroll
        for (int a = 0; a < 4; ++a)
            st4(orow + a * 16 + fc * 4, o[a][u][0] * inv, o[a][u][1] * inv, o[a][u][2] * inv, o[a][u][3] * inv);
    }
}

// fp32 variant: one thread per query, key/value tiles of 64 in LDS.
__global__ __launch_bounds__(64) void enc_attn_f32_kernel(const float* __restrict__ Q, const float* __restrict__ K,
                                                          const float* __restrict__ Vt, float* __restrict__ O,
                                                          int H, int d) {
    __shared__ float ks[64][65];
    __shared__ float vs[64][65];  // vs[dim][key]
    const int bh = blockIdx.y, bseg = bh / H, h = bh - bseg * H;
    const int q = blockIdx.x * 64 + threadIdx.x;
    const float* Qb = Q + ((long long)bh * TQ + q) * 64;
    float qv[64], o[64];
#pragma unroll
    for (int j = 0; j < 64; ++j) { qv[j] = Qb[j]; o[j] = 0.f; }
    float m = -INFINITY, l = 0.f;
    for (int k0 = 0; k0 < N_CTX; k0 += 64) {
        __syncthreads();
        for (int e = threadIdx.x; e < 64 * 64; e += 64) {
            const int r = e >> 6, c = e & 63;
            ks[r][c] = K[((long long)bh * TQ + k0 + r) * 64 + c];
            vs[r][c] = Vt[((long long)bh * 64 + r) * TQ + k0 + c];
        }
        __syncthreads();
        const int nk = min(64, N_CTX - k0);
        for (int kk = 0; kk < nk; ++kk) {
            float s = 0.f;
#pragma unroll
            for (int j = 0; j < 64; ++j) s = fmaf(qv[j], ks[kk][j], s);
            const float mnew = fmaxf(m, s);
            const float alpha = exp2_softmax(m - mnew), p = exp2_softmax(s - mnew);
            l = l * alpha + p;
#pragma unroll
            for (int j = 0; j < 64; ++j) o[j] = fmaf(p, vs[j][kk], o[j] * alpha);
            m = mnew;
        }
    }
    if (q >= N_CTX) return;
    float* orow = O + ((long long)bseg * N_CTX + q) * d + h * 64;
    const float inv = 1.0f / l;
#pragma unroll
    for (int j = 0; j < 64; ++j) orow[j] = o[j] * inv;
}

// ------------------------------------------------------------- decode attention
//
// Attention of one decode position per (row, head) over the slot's caches:
// keys stored transposed (K^T [64][positions]) so a lane owns consecutive
// positions and scores need no cross-lane reduction, values row-major so
// eight lanes read one 128-byte row; softmax in fp32. self_attn_kernel and
// cross_attn_kernel below describe their work split.
// Cache reads are non-temporal: each step streams every cached byte once,
// so they should not displace the weights and activations the projections
// keep in L2 (and the stream itself runs faster that way).
template <class T>
__device__ inline void load_vec(const T* p, float* out, int n);
template <>
__device__ inline void load_vec<bf16>(const bf16* p, float* out, int n) {
    for (int i = 0; i < n; i += 4) {
        const u32x2 u = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p + i));
        out[i] = __uint_as_float(u.x << 16);
        out[i + 1] = __uint_as_float(u.x & 0xffff0000u);
        out[i + 2] = __uint_as_float(u.y << 16);
        out[i + 3] = __uint_as_float(u.y & 0xffff0000u);
    }
}
template <>
__device__ inline void load_vec<float>(const float* p, float* out, int n) {
    for (int i = 0; i < n; i += 4) {
        typedef float f32x4 __attribute__((ext_vector_type(4)));
        const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + i));
        out[i] = v.x; out[i + 1] = v.y; out[i + 2] = v.z; out[i + 3] = v.w;
    }
}

struct DecAttnArgs {
    const void* q;      // [n][d] row-major, scaled by 1/8
    const void* kt;     // cache K^T of this layer: [S][H][64][TP]
    const void* v;      // cache V of this layer:   [S][H][TP][64]
    void* out;          // [n][d], decoder layout (dec_off)
    const int* list;    // row -> slot
    const int* rowlen;  // row -> cached positions incl. this one (self-attention)
    int TP, H, d;
    // cross-attention timing (null normally): stamp[0] = earliest workgroup
    // start, stamp[1] = latest workgroup end, in ticks of the device's
    // real-time counter
    unsigned long long* stamp;
};

// Self-attention of one decode position over the slot's cached positions
// 0..len-1 (causal by construction). Workgroup = 4 waves per (row, head):
//   scores: wave w sums dims 16w..16w+15 for all positions (lane owns 8
//     consecutive positions, 16 loads in flight), partials added in LDS;
//   softmax: every wave holds all scores (fp32, wavefront reductions);
//   P V: wave w takes positions 128w..128w+127, 8 lanes per 128-byte V row,
//     partial outputs added in LDS.
// (Issuing the V loads together with the K loads measured slower: the K and
// V phases are kept apart.) The fp32 model uses this kernel; the bf16 model
// uses self_attn_bf16_kernel below.
template <class T>
__global__ __launch_bounds__(256) void self_attn_kernel(DecAttnArgs a) {
    __shared__ float qs[64];
    __shared__ float sp[4][512];
    __shared__ float op[4][64];
    const int h = blockIdx.x, r = blockIdx.y, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int slot = a.list[r];
    const int len = a.rowlen[r];
    const T* q = reinterpret_cast<const T*>(a.q) + (long long)r * a.d + h * 64;
    if (tid < 64) qs[tid] = ldf(q + tid);
    __syncthreads();
    const long long head = (long long)slot * a.H + h;
    const T* kt = reinterpret_cast<const T*>(a.kt) + head * 64 * a.TP;
    const T* vv = reinterpret_cast<const T*>(a.v) + head * a.TP * 64;
    const int p0 = lane * 8;
    float s[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) s[i] = 0.f;
    if (p0 < len) {
        float kv[16][8];
#pragma unroll
        for (int j = 0; j < 16; ++j) load_vec<T>(kt + (long long)(16 * w + j) * a.TP + p0, kv[j], 8);
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const float qj = qs[16 * w + j];
#pragma unroll
            for (int i = 0; i < 8; ++i) s[i] = fmaf(qj, kv[j][i], s[i]);
        }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) sp[w][p0 + i] = s[i];
    __syncthreads();
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float t = ((sp[0][p0 + i] + sp[1][p0 + i]) + sp[2][p0 + i]) + sp[3][p0 + i];
        s[i] = (p0 + i < len) ? t * LOG2E : -INFINITY;
        mx = fmaxf(mx, s[i]);
    }
    mx = wave_max(mx);
    float lsum = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        s[i] = (p0 + i < len) ? exp2_softmax(s[i] - mx) : 0.f;
        lsum += s[i];
    }
    lsum = wave_sum(lsum);
    __syncthreads();  // every wave has read the partial scores
    if (w == 0) {
#pragma unroll
        for (int i = 0; i < 8; ++i) sp[0][p0 + i] = s[i];
    }
    __syncthreads();
    const int dg = lane & 7, pg = lane >> 3;
    float o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = 0.f;
    const int lo = 128 * w, hi = min(len, lo + 128);
    if (lo < hi) {
#pragma unroll
        for (int b0 = 0; b0 < 128; b0 += 64) {
            float vr[8][8];
            float pw[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int pp = lo + b0 + pg + 8 * u;
                const int pc = min(pp, hi - 1);
                load_vec<T>(vv + (long long)pc * 64 + dg * 8, vr[u], 8);
                pw[u] = pp < hi ? sp[0][pc] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < 8; ++u)
#pragma unroll
                for (int i = 0; i < 8; ++i) o[i] = fmaf(pw[u], vr[u][i], o[i]);
        }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        o[i] += __shfl_xor(o[i], 8, 64);
        o[i] += __shfl_xor(o[i], 16, 64);
        o[i] += __shfl_xor(o[i], 32, 64);
    }
    if (lane < 8) {
#pragma unroll
        for (int i = 0; i < 8; ++i) op[w][dg * 8 + i] = o[i];
    }
    __syncthreads();
    if (tid < 64) {
        const float v = ((op[0][tid] + op[1][tid]) + op[2][tid]) + op[3][tid];
        stf(reinterpret_cast<T*>(a.out) + dec_off<T>(r, h * 64 + tid, a.d), v / lsum);
    }
}

// Self-attention, second work split (bf16 caches): wave w reads the 16
// query values of its dims straight from memory (no LDS round trip), sums
// dims 16w..16w+15 of every position's score as above, and the P V product
// is spread over all four waves: wave w takes the contiguous positions
// [w c, w c + c) with c = len / 4 rounded up to a multiple of 8, 8 lanes
// per 128-byte V row. The first batch of 8 V rows per lane group is issued
// before the softmax, so its latency overlaps the score reduction. The
// scores are computed as in self_attn_kernel; the P V sums are grouped by
// this split, and the waves' partial outputs are added in LDS in wave order.
__global__ __launch_bounds__(256) void self_attn_bf16_kernel(DecAttnArgs a) {
    __shared__ float sp[4][512];
    __shared__ float op[4][64];
    const int h = blockIdx.x, r = blockIdx.y, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int slot = a.list[r];
    const int len = a.rowlen[r];
    const bf16* q = reinterpret_cast<const bf16*>(a.q) + (long long)r * a.d + h * 64 + 16 * w;
    const u32x4 q0 = *reinterpret_cast<const u32x4*>(q), q1 = *reinterpret_cast<const u32x4*>(q + 8);
    const long long head = (long long)slot * a.H + h;
    const bf16* kt = reinterpret_cast<const bf16*>(a.kt) + head * 64 * a.TP;
    const bf16* vv = reinterpret_cast<const bf16*>(a.v) + head * a.TP * 64;
    const int p0 = lane * 8;
    float s[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) s[i] = 0.f;
    if (p0 < len) {
        float kv[16][8];
#pragma unroll
        for (int j = 0; j < 16; ++j) load_vec<bf16>(kt + (long long)(16 * w + j) * a.TP + p0, kv[j], 8);
        float qv[16];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            qv[2 * e] = __uint_as_float(q0[e] << 16);
            qv[2 * e + 1] = __uint_as_float(q0[e] & 0xffff0000u);
            qv[8 + 2 * e] = __uint_as_float(q1[e] << 16);
            qv[8 + 2 * e + 1] = __uint_as_float(q1[e] & 0xffff0000u);
        }
#pragma unroll
        for (int j = 0; j < 16; ++j)
#pragma unroll
            for (int i = 0; i < 8; ++i) s[i] = fmaf(qv[j], kv[j][i], s[i]);
    }
    // this wave's positions for P V, and the first batch of their V rows
    const int c = ((len + 3) / 4 + 7) & ~7;
    const int lo = min(len, w * c), hi = min(len, lo + c);
    const int dg = lane & 7, pg = lane >> 3;
    u32x4 v0[8];
    if (lo < hi) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int pc = min(lo + pg + 8 * u, hi - 1);
            v0[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vv + (long long)pc * 64 + dg * 8));
        }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) sp[w][p0 + i] = s[i];
    __syncthreads();
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float t = ((sp[0][p0 + i] + sp[1][p0 + i]) + sp[2][p0 + i]) + sp[3][p0 + i];
        s[i] = (p0 + i < len) ? t * LOG2E : -INFINITY;
        mx = fmaxf(mx, s[i]);
    }
    mx = wave_max(mx);
    float lsum = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        s[i] = (p0 + i < len) ? exp2_softmax(s[i] - mx) : 0.f;
        lsum += s[i];
    }
    lsum = wave_sum(lsum);
    __syncthreads();  // every wave has read the partial scores
    if (w == 0) {
#pragma unroll
        for (int i = 0; i < 8; ++i) sp[0][p0 + i] = s[i];
    }
    __syncthreads();
    float o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = 0.f;
    if (lo < hi) {
#pragma unroll 1
        for (int b0 = lo; b0 < hi; b0 += 64) {
            u32x4 vr[8];
            float pw[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int pp = b0 + pg + 8 * u;
                const int pc = min(pp, hi - 1);
                vr[u] = b0 == lo ? v0[u]
                                 : __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vv + (long long)pc * 64 + dg * 8));
                pw[u] = pp < hi ? sp[0][pc] : 0.f;
            }
#pragma unroll
            for (int u = 0; u < 8; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    o[2 * e] = fmaf(pw[u], __uint_as_float(vr[u][e] << 16), o[2 * e]);
                    o[2 * e + 1] = fmaf(pw[u], __uint_as_float(vr[u][e] & 0xffff0000u), o[2 * e + 1]);
                }
        }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        o[i] += __shfl_xor(o[i], 8, 64);
        o[i] += __shfl_xor(o[i], 16, 64);
        o[i] += __shfl_xor(o[i], 32, 64);
    }
    if (lane < 8) {
#pragma unroll
        for (int i = 0; i < 8; ++i) op[w][dg * 8 + i] = o[i];
    }
    __syncthreads();
    if (tid < 64) {
        const float v = ((op[0][tid] + op[1][tid]) + op[2][tid]) + op[3][tid];
        stf(reinterpret_cast<bf16*>(a.out) + dec_off<bf16>(r, h * 64 + tid, a.d), v / lsum);
    }
}

// Cross-attention of one decode position over the 1500 cached encoder
// positions. Workgroup = CW waves per (row, head), wave w takes positions
// 256w..256w+255: scores with K^T rows (lane owns 4 consecutive positions,
// 16 dims' loads in flight), softmax over the chunk, P V with V rows (8
// lanes per 128-byte row, 8 rows in flight); the chunk results (max, sum,
// 64 outputs) are merged in LDS in wave order.
constexpr int CW = (N_CTX + 255) / 256;

template <class T>
__global__ __launch_bounds__(64 * CW) void cross_attn_kernel(DecAttnArgs a) {
    __shared__ float qs[64];
    __shared__ float ps[CW][256];
    __shared__ float ml[CW][2];
    __shared__ float op[CW][64];
    const int h = blockIdx.x, r = blockIdx.y, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    if (a.stamp && tid == 0) atomicMin(a.stamp, (unsigned long long)__builtin_amdgcn_s_memrealtime());
    const int slot = a.list[r];
    const T* q = reinterpret_cast<const T*>(a.q) + (long long)r * a.d + h * 64;
    if (tid < 64) qs[tid] = ldf(q + tid);
    __syncthreads();
    const long long head = (long long)slot * a.H + h;
    const T* kt = reinterpret_cast<const T*>(a.kt) + head * 64 * a.TP;
    const T* vv = reinterpret_cast<const T*>(a.v) + head * a.TP * 64;
    const int start = 256 * w;
    const int p0 = start + lane * 4;
    float s[4] = {0.f, 0.f, 0.f, 0.f};
    if (p0 < N_CTX) {
#pragma unroll 1
        for (int j0 = 0; j0 < 64; j0 += 16) {
            float kv[16][4];
#pragma unroll
            for (int j = 0; j < 16; ++j) load_vec<T>(kt + (long long)(j0 + j) * a.TP + p0, kv[j], 4);
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const float qj = qs[j0 + j];
#pragma unroll
                for (int i = 0; i < 4; ++i) s[i] = fmaf(qj, kv[j][i], s[i]);
            }
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        s[i] = (p0 + i < N_CTX) ? s[i] * LOG2E : -INFINITY;
        mx = fmaxf(mx, s[i]);
    }
    mx = wave_max(mx);
    float lsum = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float p = (p0 + i < N_CTX) ? exp2_softmax(s[i] - mx) : 0.f;
        ps[w][lane * 4 + i] = p;
        lsum += p;
    }
    lsum = wave_sum(lsum);
    __syncthreads();
    const int dg = lane & 7, pg = lane >> 3;
    float o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = 0.f;
    const int nloc = min(256, N_CTX - start);
#pragma unroll 1
    for (int b0 = 0; b0 < 256; b0 += 64) {
        float vr[8][8];
        float pw[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int pp = b0 + pg + 8 * u;
            const int pc = min(pp, nloc - 1);
            load_vec<T>(vv + (long long)(start + pc) * 64 + dg * 8, vr[u], 8);
            pw[u] = pp < nloc ? ps[w][pc] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
            for (int i = 0; i < 8; ++i) o[i] = fmaf(pw[u], vr[u][i], o[i]);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        o[i] += __shfl_xor(o[i], 8, 64);
        o[i] += __shfl_xor(o[i], 16, 64);
        o[i] += __shfl_xor(o[i], 32, 64);
    }
    if (lane < 8) {
#pragma unroll
        for (int i = 0; i < 8; ++i) op[w][dg * 8 + i] = o[i];
    }
    if (lane == 0) { ml[w][0] = mx; ml[w][1] = lsum; }
    __syncthreads();
    if (tid < 64) {
        float M = ml[0][0];
#pragma unroll
        for (int c = 1; c < CW; ++c) M = fmaxf(M, ml[c][0]);
        float L = 0.f, acc = 0.f;
#pragma unroll
        for (int c = 0; c < CW; ++c) {
            const float wgt = exp2_softmax(ml[c][0] - M);
            L += wgt * ml[c][1];
            acc += wgt * op[c][tid];
        }
        stf(reinterpret_cast<T*>(a.out) + dec_off<T>(r, h * 64 + tid, a.d), acc / L);
    }
    if (a.stamp) {
        __syncthreads();
        if (tid == 0) atomicMax(a.stamp + 1, (unsigned long long)__builtin_amdgcn_s_memrealtime());
    }
}

// Timing slots of n launches: start = all ones (for a minimum), end = 0.
__global__ void stamp_reset_kernel(unsigned long long* __restrict__ s, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) {
        s[2 * i] = ~0ull;
        s[2 * i + 1] = 0ull;
    }
}

// ------------------------------------------------------------- skinny decode GEMM (bf16 MFMA)
//
// C[i][r] = sum_k W[i][k] X[r][k] for a few rows r (active decode slots,
// n <= 16 * NT) and many weight rows i: each weight byte is read once.
// W and X are fragment-major (frag_off), so every load below reads 1 KiB
// contiguous. Grid (row tiles, KS): workgroup (tile, ks) covers 16 * RT
// weight rows and reduction columns [ks * Kc, (ks + 1) * Kc). Its 4 waves
// take interleaved 32-wide k-steps, U steps' loads issued before their
// MFMAs; the wave partial sums are added in LDS in a fixed order, so a row's
// result never depends on which other rows are present (row tiles past n
// re-read the last valid tile and are dropped). NW waves per workgroup
// (4, or more for long reductions), red: (NW - 1) * RT * NT * 4 * 64 floats.
template <int RT, int NT, int U, int NW = 4>
__device__ __forceinline__ void skinny_core(const bf16* __restrict__ W, const bf16* __restrict__ X, int nks_tot, int n,
                                            int Kc, float* red, float (&v)[RT][NT][4]) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int s_base = blockIdx.y * (Kc >> 5);
    const bf16* wp[RT];
#pragma unroll
    for (int t = 0; t < RT; ++t) wp[t] = W + (((long long)(blockIdx.x * RT + t) * nks_tot + s_base) * 64 + lane) * 8;
    const int ulast = (n - 1) >> 4;
    const bf16* xp[NT];
#pragma unroll
    for (int u = 0; u < NT; ++u) xp[u] = X + (((long long)min(u, ulast) * nks_tot + s_base) * 64 + lane) * 8;
    mfma_f32x4 acc[RT][NT];
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int u = 0; u < NT; ++u) acc[t][u] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
    const int nks = Kc >> 5;
    // Batches of U k-steps (s, s + NW, ...): all loads of a batch are issued
    // before its MFMAs; steps past the end re-read the last step and are skipped.
    for (int s0 = wave; s0 < nks; s0 += NW * U) {
        mfma_bf16x8 a[U][RT], b[U][NT];
#pragma unroll
        for (int q = 0; q < U; ++q) {
            const int off = min(s0 + NW * q, nks - 1) * 512;
#pragma unroll
            for (int t = 0; t < RT; ++t) a[q][t] = *reinterpret_cast<const mfma_bf16x8*>(wp[t] + off);
#pragma unroll
            for (int u = 0; u < NT; ++u) b[q][u] = *reinterpret_cast<const mfma_bf16x8*>(xp[u] + off);
        }
#pragma unroll
        for (int q = 0; q < U; ++q) {
            if (s0 + NW * q < nks) {
#pragma unroll
                for (int t = 0; t < RT; ++t)
#pragma unroll
                    for (int u = 0; u < NT; ++u)
                        acc[t][u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[q][t], b[q][u], acc[t][u], 0, 0, 0);
            }
        }
    }
    constexpr int F = RT * NT * 4;
    if (wave > 0) {
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int u = 0; u < NT; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e) red[((wave - 1) * F + (t * NT + u) * 4 + e) * 64 + lane] = acc[t][u][e];
    }
    __syncthreads();
    if (wave == 0) {
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int u = 0; u < NT; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int idx = (t * NT + u) * 4 + e;
                    float sum = acc[t][u][e];
#pragma unroll
                    for (int w = 1; w < NW; ++w) sum += red[((w - 1) * F + idx) * 64 + lane];
                    v[t][u][e] = sum;
                }
    }
}

// Plain epilogue variant: wave 0 hands rows i..i+3 of column r to epi (its
// loads, pre(), are issued before the main loop). z = ks.
template <int RT, int NT, int U, class Epi, int NW = 4>
__global__ __launch_bounds__(64 * NW) void skinny_bf16_kernel(const bf16* __restrict__ W, const bf16* __restrict__ X,
                                                              int nks_tot, int MA, int n, int Kc, Epi epi) {
    __shared__ float red[(NW - 1) * RT * NT * 4 * 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int fr = lane & 15, fc = lane >> 4;
    const int i0 = blockIdx.x * 16 * RT;
    EpiPre pre[RT][NT];
    if (wave == 0) {
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int u = 0; u < NT; ++u) {
                const int i = i0 + t * 16 + fc * 4, r = u * 16 + fr;
                if (i < MA && r < n) pre[t][u] = epi.pre(i, r, blockIdx.y);
            }
    }
    float v[RT][NT][4];
    skinny_core<RT, NT, U, NW>(W, X, nks_tot, n, Kc, red, v);
    if (wave > 0) return;
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int u = 0; u < NT; ++u) {
            const int i = i0 + t * 16 + fc * 4, r = u * 16 + fr;
            if (i < MA && r < n) epi(i, r, blockIdx.y, v[t][u][0], v[t][u][1], v[t][u][2], v[t][u][3], pre[t][u]);
        }
}

// Split-K partial sums: part[ks][r][i..i+3] (row length N).
struct EpiPartial {
    float* part;
    int N, n;
    __device__ EpiPre pre(int, int, int) const { return EpiPre{}; }
    __device__ void operator()(int i, int r, int ks, float a, float b, float c, float e, const EpiPre&) const {
        st4(part + ((long long)ks * n + r) * N + i, a, b, c, e);
    }
};

// Residual update without split-K: x[r][i..i+3] += (sum + bias), where the
// workgroup owns weight rows i..i+3 for the whole reduction (x row-major,
// width d; x and the bias are loaded before the main loop).
struct EpiResidX {
    const float* bias;
    float* x;
    int d;
    __device__ EpiPre pre(int i, int r, int) const {
        EpiPre p{};
        p.a = ld4(bias + i);
        p.b = ld4(x + (long long)r * d + i);
        return p;
    }
    __device__ void operator()(int i, int r, int, float a, float b, float c, float e, const EpiPre& p) const {
        st4(x + (long long)r * d + i, p.b.x + (a + p.a.x), p.b.y + (b + p.a.y), p.b.z + (c + p.a.z),
            p.b.w + (e + p.a.w));
    }
};

// Decode projection of layer-normed rows, C[i][r] = sum_k W[i][k] LN(x[r])[k],
// for 16 activation rows per workgroup: grid (weight-row tiles of 16 * RT,
// groups of 16 rows). The workgroup normalises its own rows from the fp32
// residual stream x (row-major, width d = 64 E; fp32 mean, then biased
// variance about it, eps 1e-5, gain and bias), rounds them to bf16 and keeps
// them in LDS in the MFMA's B-operand fragment layout. Its weight loads (W
// fragment-major, one batch covering each wave's k-steps) are issued right
// after the row loads, so they are in flight during the normalisation. The NW waves take interleaved 32-wide
// k-steps and are summed in LDS in a fixed order: a row's result depends on
// that row alone. Rows past n are zero and dropped.
namespace sln {
constexpr int NW = 8;
}
template <int RT, int E, class Epi>
__global__ __launch_bounds__(64 * sln::NW) void skinny_ln_kernel(const bf16* __restrict__ W,
                                                                 const float* __restrict__ x,
                                                                 const float* __restrict__ g,
                                                                 const float* __restrict__ b, int MA, int n,
                                                                 Epi epi) {
    constexpr int NW = sln::NW, d = 64 * E, nks = d / 32, U = (nks + NW - 1) / NW;
    constexpr int NC = 8 * E, CH = (NC + 63) / 64, RPW = 16 / NW, F = RT * 4;
    __shared__ __align__(16) bf16 zs[16 * d];
    __shared__ float red[(NW - 1) * F * 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int fr = lane & 15, fc = lane >> 4;
    const int i0 = blockIdx.x * 16 * RT, r0 = blockIdx.y * 16;
    EpiPre pre[RT];
    mfma_bf16x8 a[U][RT];
    float v[RPW][CH][8], gg[CH][8], bb[CH][8];
    // Loads in the order they are needed (the vector-memory counter retires
    // them in issue order): this wave's rows (lane holds 8-column chunks
    // lane, lane + 64, ...), then gain and bias, so the normalisation starts
    // while the weights are still in flight; then the weights, then the
    // epilogue's operands.
#pragma unroll
    for (int rr = 0; rr < RPW; ++rr) {
        const int R = r0 + wave * RPW + rr;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int c8 = lane + 64 * c;
            const bool ok = R < n && c8 < NC;
            const float* xp = x + (long long)R * d + 8 * c8;
            const float4 x0 = ok ? ld4(xp) : float4{}, x1 = ok ? ld4(xp + 4) : float4{};
            v[rr][c][0] = x0.x; v[rr][c][1] = x0.y; v[rr][c][2] = x0.z; v[rr][c][3] = x0.w;
            v[rr][c][4] = x1.x; v[rr][c][5] = x1.y; v[rr][c][6] = x1.z; v[rr][c][7] = x1.w;
        }
    }
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int c8 = lane + 64 * c;
        const bool ok = c8 < NC;
        const float4 g0 = ok ? ld4(g + 8 * c8) : float4{}, g1 = ok ? ld4(g + 8 * c8 + 4) : float4{};
        const float4 b0 = ok ? ld4(b + 8 * c8) : float4{}, b1 = ok ? ld4(b + 8 * c8 + 4) : float4{};
        gg[c][0] = g0.x; gg[c][1] = g0.y; gg[c][2] = g0.z; gg[c][3] = g0.w;
        gg[c][4] = g1.x; gg[c][5] = g1.y; gg[c][6] = g1.z; gg[c][7] = g1.w;
        bb[c][0] = b0.x; bb[c][1] = b0.y; bb[c][2] = b0.z; bb[c][3] = b0.w;
        bb[c][4] = b1.x; bb[c][5] = b1.y; bb[c][6] = b1.z; bb[c][7] = b1.w;
    }
#pragma unroll
    for (int q = 0; q < U; ++q) {
        const int st = min(wave + NW * q, nks - 1);
#pragma unroll
        for (int t = 0; t < RT; ++t)
            a[q][t] = *reinterpret_cast<const mfma_bf16x8*>(
                W + (((long long)(blockIdx.x * RT + t) * nks + st) * 64 + lane) * 8);
    }
    if (wave == 0) {
#pragma unroll
        for (int t = 0; t < RT; ++t) {
            const int i = i0 + t * 16 + fc * 4, r = r0 + fr;
            if (i < MA && r < n) pre[t] = epi.pre(i, r, 0);
        }
    }
#pragma unroll
    for (int rr = 0; rr < RPW; ++rr) {
        const int row = wave * RPW + rr, R = r0 + row;
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < CH; ++c)
#pragma unroll
            for (int j = 0; j < 8; ++j) s += v[rr][c][j];
        const float mean = wave_sum(s) / d;
        float q = 0.f;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            if (lane + 64 * c < NC) {
#pragma unroll
                for (int j = 0; j < 8; ++j) { const float e = v[rr][c][j] - mean; q += e * e; }
            }
        }
        const float rstd = rsqrtf(wave_sum(q) / d + 1e-5f);
        const bool live = R < n;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int c8 = lane + 64 * c;
            if (c8 < NC) {
                uint32_t w4[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float z0 = live ? (v[rr][c][2 * j] - mean) * rstd * gg[c][2 * j] + bb[c][2 * j] : 0.f;
                    const float z1 =
                        live ? (v[rr][c][2 * j + 1] - mean) * rstd * gg[c][2 * j + 1] + bb[c][2 * j + 1] : 0.f;
                    w4[j] = pack_bf16x2(z0, z1);
                }
                *reinterpret_cast<uint4*>(zs + (((c8 >> 2) * 64 + (c8 & 3) * 16 + row) << 3)) =
                    uint4{w4[0], w4[1], w4[2], w4[3]};
            }
        }
    }
    __syncthreads();
    mfma_f32x4 acc[RT];
#pragma unroll
    for (int t = 0; t < RT; ++t) acc[t] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < U; ++q) {
        const int st = wave + NW * q;
        if (st < nks) {
            const mfma_bf16x8 bx = *reinterpret_cast<const mfma_bf16x8*>(zs + ((st * 64 + lane) << 3));
#pragma unroll
            for (int t = 0; t < RT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[q][t], bx, acc[t], 0, 0, 0);
        }
    }
    if (wave > 0) {
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int e = 0; e < 4; ++e) red[((wave - 1) * F + t * 4 + e) * 64 + lane] = acc[t][e];
    }
    __syncthreads();
    if (wave > 0) return;
#pragma unroll
    for (int t = 0; t < RT; ++t) {
        float o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float sum = acc[t][e];
#pragma unroll
            for (int w = 1; w < NW; ++w) sum += red[((w - 1) * F + t * 4 + e) * 64 + lane];
            o[e] = sum;
        }
        const int i = i0 + t * 16 + fc * 4, r = r0 + fr;
        if (i < MA && r < n) epi(i, r, 0, o[0], o[1], o[2], o[3], pre[t]);
    }
}

// U = k-steps per wave and batch for nks k-steps over 4 waves: all of a
// wave's steps in one batch, up to 10 (4 with 8 row tiles, for registers).
constexpr int skinny_u(int nks, int NT) {
    return (nks + 3) / 4 <= 1 ? 1
         : (nks + 3) / 4 <= 2 ? 2
         : (nks + 3) / 4 <= 3 ? 3
         : ((nks + 3) / 4 <= 4 || NT >= 8) ? 4
         : (nks + 3) / 4 <= 6 ? 6 : 10;
}

#define WMI_SKINNY_U(Kc, NT, LAUNCH)                                                  \
    do {                                                                             \
        const int u_ = skinny_u((Kc) / 32, NT);                                       \
        if (u_ == 1) { constexpr int U = 1; LAUNCH; }                                 \
        else if (u_ == 2) { constexpr int U = 2; LAUNCH; }                            \
        else if (u_ == 3) { constexpr int U = 3; LAUNCH; }                            \
        else if (u_ == 4) { constexpr int U = 4; LAUNCH; }                            \
        else if (u_ == 6) { constexpr int U = (NT) >= 8 ? 4 : 6; LAUNCH; }             \
        else { constexpr int U = (NT) >= 8 ? 4 : 10; LAUNCH; }                        \
    } while (0)

#define WMI_SKINNY_NT(n, ...)                                         \
    do {                                                             \
        if ((n) <= 16) { constexpr int NT = 1; __VA_ARGS__; }          \
        else if ((n) <= 32) { constexpr int NT = 2; __VA_ARGS__; }     \
        else if ((n) <= 64) { constexpr int NT = 4; __VA_ARGS__; }     \
        else { constexpr int NT = 8; __VA_ARGS__; }                    \
    } while (0)

// Waves per workgroup of a residual projection (whole reduction in one
// workgroup): twice the usual, to keep more loads in flight. The same for
// every row count, since the waves' k-step split fixes the summation order.
constexpr int RESID_NW = 8;
// k-steps per wave and batch for nks k-steps over NW waves (fewer with many
// row tiles, for registers)
constexpr int resid_u(int nks, int NW, int NT) {
    return (nks + NW - 1) / NW <= 1 ? 1
         : ((nks + NW - 1) / NW <= 2 || NT >= 8) ? 2
         : (nks + NW - 1) / NW <= 3 ? 3
         : (nks + NW - 1) / NW <= 4 ? 4
         : (nks + NW - 1) / NW <= 6 ? 6 : 10;
}
#define WMI_RESID_U(nks, NW, NT, LAUNCH)                                              \
    do {                                                                             \
        const int u_ = resid_u(nks, NW, NT);                                          \
        if (u_ == 1) { constexpr int U = 1; LAUNCH; }                                 \
        else if (u_ == 2) { constexpr int U = 2; LAUNCH; }                            \
        else if (u_ == 3) { constexpr int U = (NT) >= 8 ? 2 : 3; LAUNCH; }             \
        else if (u_ == 4) { constexpr int U = (NT) >= 8 ? 2 : 4; LAUNCH; }             \
        else if (u_ == 6) { constexpr int U = (NT) >= 8 ? 2 : 6; LAUNCH; }             \
        else { constexpr int U = (NT) >= 8 ? 2 : (NT) >= 4 ? 6 : 10; LAUNCH; }        \
    } while (0)

// x[r] += W X[r] + bias for n rows (W fragment-major [d rounded up to 32][K],
// X fragment-major [n rounded up to 16][K], x row-major fp32 [n][d]).
// More than 64 rows go in launches of 64 (a row's result does not depend on
// the other rows of its launch).
inline void skinny_resid(const bf16* W, int d, const bf16* X, int n, int K, const float* bias, float* x,
                         hipStream_t st) {
    if (K % 32 || n <= 0 || n > 128 || d % 16) throw ArgError(-1, "skinny_resid: unsupported shape");
    const int nks = K / 32;
    const dim3 grid(d / 16, 1);
    for (int r0 = 0; r0 < n; r0 += 64) {
        const int m = min(64, n - r0);
        const bf16* Xr = X + (size_t)r0 * K;
        const EpiResidX epi{bias, x + (size_t)r0 * d, d};
        auto launch = [&](auto nt) {
            constexpr int NT = decltype(nt)::value;
            WMI_RESID_U(nks, RESID_NW, NT,
                        hipLaunchKernelGGL((skinny_bf16_kernel<1, NT, U, EpiResidX, RESID_NW>), grid,
                                           dim3(64 * RESID_NW), 0, st, W, Xr, nks, d, m, K, epi));
        };
        if (m <= 16) launch(std::integral_constant<int, 1>{});
        else if (m <= 32) launch(std::integral_constant<int, 2>{});
        else launch(std::integral_constant<int, 4>{});
    }
}

// C = W LN(x) for n rows of the fp32 residual stream x (row-major, width d),
// with the layer norm's gain g and bias b; W fragment-major [MA][d], MA a
// multiple of 16. Every workgroup of a row group repeats that group's
// normalisation, which pays only where MA is small (the cross-attention
// query projection, MA = d).
template <class Epi>
inline void skinny_ln(const bf16* W, int MA, const float* x, int n, int d, const float* g, const float* b,
                      const Epi& epi, hipStream_t st) {
    if (n <= 0 || n > 128 || MA <= 0 || MA % 16) throw ArgError(-1, "skinny_ln: unsupported shape");
    const int groups = (n + 15) / 16;
    WMI_SWITCH_E(d, hipLaunchKernelGGL((skinny_ln_kernel<1, E, Epi>), dim3(MA / 16, groups), dim3(64 * sln::NW), 0,
                                       st, W, x, g, b, MA, n, epi));
}

// W: fragment-major [MA rounded up to 32][K], X: fragment-major [n rounded up
// to 16][K]; KS workgroups split K.
template <class Epi>
inline void skinny_bf16(const bf16* W, int MA, const bf16* X, int n, int K, int KS, const Epi& epi, hipStream_t st) {
    if (KS < 1 || K % (32 * KS) || n <= 0 || n > 128 || MA <= 0) throw ArgError(-1, "skinny_bf16: unsupported shape");
    const int Kc = K / KS, nks_tot = K / 32;
    if (MA >= 16384) {  // output head: 32 rows per workgroup
        const dim3 grid((MA + 31) / 32, KS);
        WMI_SKINNY_NT(n, WMI_SKINNY_U(Kc, NT, hipLaunchKernelGGL((skinny_bf16_kernel<2, NT, U, Epi>), grid, dim3(256),
                                                                0, st, W, X, nks_tot, MA, n, Kc, epi)));
    } else {
        const dim3 grid((MA + 15) / 16, KS);
        WMI_SKINNY_NT(n, WMI_SKINNY_U(Kc, NT, hipLaunchKernelGGL((skinny_bf16_kernel<1, NT, U, Epi>), grid, dim3(256),
                                                                0, st, W, X, nks_tot, MA, n, Kc, epi)));
    }
}

// ------------------------------------------------------------- CTC greedy decoding
//
// Best-path decoding of an encoder-only CTC model (blank = id 0): the most
// likely id of every frame, then each entry's frames 0..T-1 collapsed
// (runs of one id merged, blanks dropped).

// One wave per frame: argmax over the V logits of the frame, the lowest id
// among equal maxima. A frame with no finite maximum (every logit -inf or
// NaN) records the blank and raises *err, which the next read reports.
__global__ __launch_bounds__(256) void ctc_argmax_kernel(const float* __restrict__ logits, int V, int frames,
                                                         int* __restrict__ ids, int* __restrict__ err) {
    const int f = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (f >= frames) return;
    const float* row = logits + (long long)f * V;
    float best = -INFINITY;
    int bi = V;
    for (int v = lane; v < V; v += 64) {
        const float x = row[v];
        if (x > best) { best = x; bi = v; }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float ob = __shfl_xor(best, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
    }
    if (lane == 0) {
        ids[f] = bi < V ? bi : 0;   // no finite logit: the blank, and the flag the read reports
        if (bi >= V) atomicOr(err, 1);
    }
}

// One workgroup (1024 threads) per batch entry b over its 1500 frame ids:
// frame t is kept when t < T[b], its id is not the blank and differs from
// frame t-1's; kept ids are compacted in frame order (workgroup prefix sum)
// into tok[b][.], their number into cnt[b].
__global__ __launch_bounds__(1024) void ctc_collapse_kernel(const int* __restrict__ ids, const int* __restrict__ nframes,
                                                            int* __restrict__ tok, int* __restrict__ cnt) {
    __shared__ int wsum[16];
    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int T = nframes[b];
    const int* id = ids + (long long)b * N_CTX;
    const int t0 = 2 * tid, t1 = t0 + 1;
    const int i0 = t0 < T ? id[t0] : 0, i1 = t1 < T ? id[t1] : 0;
    const int prev = (t0 > 0 && t0 < T) ? id[t0 - 1] : -1;
    const int k0 = (t0 < T && i0 != 0 && i0 != prev) ? 1 : 0;
    const int k1 = (t1 < T && i1 != 0 && i1 != i0) ? 1 : 0;
    const int c = k0 + k1;
    int x = c;  // inclusive prefix over the wave
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    if (tid == 0)
        for (int i = 1; i < 16; ++i) wsum[i] += wsum[i - 1];
    __syncthreads();
    const int pos = x - c + (w > 0 ? wsum[w - 1] : 0);
    int* out = tok + (long long)b * N_CTX;
    if (k0) out[pos] = i0;
    if (k1) out[pos + k0] = i1;
    if (tid == 0) cnt[b] = wsum[15];
}

// ------------------------------------------------------------- CTC prefix beam search
//
// Decoding variant of the CTC model: prefix beam search without a language
// model, the frame's candidates pruned to its K most likely non-blank ids.
namespace cb {
constexpr int KMAX = 16;           // largest beam (and candidates per frame)
constexpr int CMAX = KMAX * (1 + KMAX);  // stays + extensions of one frame
}

// One wave per frame: log-softmax normaliser, the blank's log-probability
// and the K most likely non-blank ids with theirs (lowest id on ties),
// written to lpb[f], cid[f][0..K), clp[f][0..K).
__global__ __launch_bounds__(256) void ctc_frame_topk_kernel(const float* __restrict__ logits, int V, int frames,
                                                             int K, float* __restrict__ lpb, int* __restrict__ cid,
                                                             float* __restrict__ clp) {
    const int f = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (f >= frames) return;
    const float* row = logits + (long long)f * V;
    float mx = -INFINITY;
    for (int v = lane; v < V; v += 64) mx = fmaxf(mx, row[v]);
    mx = wave_max(mx);
    float sum = 0.f;
    for (int v = lane; v < V; v += 64) sum += expf(row[v] - mx);
    const float lse = mx + logf(wave_sum(sum));
    if (lane == 0) lpb[f] = row[0] - lse;
    uint64_t taken = 0;  // bit i: this lane's (i)-th value v = lane + 64 i was chosen (V <= 4096)
    for (int k = 0; k < K; ++k) {
        float best = -INFINITY;
        int bi = V;
        for (int i = 0, v = lane; v < V; ++i, v += 64) {
            if (v == 0 || ((taken >> i) & 1)) continue;
            const float x = row[v];
            if (x > best) { best = x; bi = v; }
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            const float ob = __shfl_xor(best, o, 64);
            const int oi = __shfl_xor(bi, o, 64);
            if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
        }
        if (bi < V && (bi & 63) == lane) taken |= 1ull << (bi >> 6);
        if (lane == 0) {
            cid[(long long)f * cb::KMAX + k] = bi < V ? bi : 0;
            clp[(long long)f * cb::KMAX + k] = bi < V ? best - lse : -INFINITY;
        }
    }
}

__device__ inline float lae_dev(float a, float b) {  // log(exp a + exp b)
    if (a == -INFINITY) return b;
    if (b == -INFINITY) return a;
    const float m = fmaxf(a, b);
    return m + log1pf(expf(-fabsf(a - b)));
}

// Prefix identity: a 64-bit hash of the label sequence, extended one label
// at a time (equal prefixes merge when their hashes are equal).
__device__ inline uint64_t prefix_hash(uint64_t h, int c) {
    uint64_t x = (h ^ (uint64_t)(c + 1)) * 0x9E3779B97F4A7C15ull;
    x ^= x >> 31;
    x *= 0xBF58476D1CE4E5B9ull;
    return x ^ (x >> 29);
}

// One wave per batch entry b over its T[b] frames. Beams: (hash, length,
// last label, pb, pnb) in LDS; the candidates of a frame are every beam's
// "stay" (in beam order) then its K extensions (beam by beam, candidate
// order); an extension equal to a kept prefix merges into that prefix's
// stay; the B most probable candidates survive (ties: earlier candidate).
// bp[b][t][j] = (parent beam << 20) | (appended label + 1, 0 for none) of
// beam j after frame t; the best final beam is traced back into tok[b][.],
// its length into cnt[b].
__global__ __launch_bounds__(64) void ctc_beam_kernel(const float* __restrict__ lpb, const int* __restrict__ cid,
                                                     const float* __restrict__ clp, const int* __restrict__ nframes,
                                                     int B, int K, int* __restrict__ bp, int* __restrict__ tok,
                                                     int* __restrict__ cnt) {
    using namespace cb;
    __shared__ uint64_t bh[2][KMAX];
    __shared__ int blen[2][KMAX], blast[2][KMAX];
    __shared__ float bpb[2][KMAX], bpnb[2][KMAX];
    __shared__ uint64_t ch[CMAX];
    __shared__ int clen[CMAX], clast[CMAX], cpar[CMAX], capp[CMAX], cmerge[CMAX];
    __shared__ float cpb[CMAX], cpnb[CMAX], cscore[CMAX];
    __shared__ int nbeam;
    __shared__ float s_lpb[64];           // the candidates of 64 frames, staged per chunk
    __shared__ int s_id[64][KMAX];
    __shared__ float s_lp[64][KMAX];
    const int b = blockIdx.x, lane = threadIdx.x;
    const int T = nframes[b];
    const long long f0 = (long long)b * N_CTX;
    int* bpe = bp + (long long)b * N_CTX * KMAX;
    if (lane == 0) {
        bh[0][0] = 0x243F6A8885A308D3ull;  // the empty prefix
        blen[0][0] = 0;
        blast[0][0] = -1;
        bpb[0][0] = 0.f;
        bpnb[0][0] = -INFINITY;
        nbeam = 1;
    }
    __syncthreads();
    int cur = 0;
    for (int t = 0; t < T; ++t) {
        if ((t & 63) == 0) {  // lane l stages frame t + l
            const int tf = t + lane;
            if (tf < T) {
                s_lpb[lane] = lpb[f0 + tf];
                for (int k = 0; k < K; ++k) {
                    s_id[lane][k] = cid[(f0 + tf) * KMAX + k];
                    s_lp[lane][k] = clp[(f0 + tf) * KMAX + k];
                }
            }
            __syncthreads();
        }
        const int nb = nbeam, nc = nb * (1 + K);
        const float lb = s_lpb[t & 63];
        const int* fid = s_id[t & 63];
        const float* flp = s_lp[t & 63];
        for (int j = lane; j < nc; j += 64) {
            if (j < nb) {  // stay j: through the blank, or repeat of the last label
                const float tot = lae_dev(bpb[cur][j], bpnb[cur][j]);
                float rep = -INFINITY;
                if (blen[cur][j] > 0)
                    for (int k = 0; k < K; ++k)
                        if (fid[k] == blast[cur][j]) rep = bpnb[cur][j] + flp[k];
                ch[j] = bh[cur][j];
                clen[j] = blen[cur][j];
                clast[j] = blast[cur][j];
                cpar[j] = j;
                capp[j] = 0;
                cpb[j] = tot + lb;
                cpnb[j] = rep;
                cmerge[j] = -1;
            } else {  // extension of beam i by candidate k
                const int i = (j - nb) / K, k = (j - nb) - i * K;
                const int c = fid[k];
                const bool again = blen[cur][i] > 0 && c == blast[cur][i];
                const float src = again ? bpb[cur][i] : lae_dev(bpb[cur][i], bpnb[cur][i]);
                const uint64_t h = prefix_hash(bh[cur][i], c);
                ch[j] = h;
                clen[j] = blen[cur][i] + 1;
                clast[j] = c;
                cpar[j] = i;
                capp[j] = c + 1;
                cpb[j] = -INFINITY;
                cpnb[j] = src + flp[k];
                int m = -1;
                for (int q = 0; q < nb; ++q)
                    if (bh[cur][q] == h && blen[cur][q] == clen[j]) m = q;
                cmerge[j] = m;
            }
        }
        __syncthreads();
        // merge: each kept prefix receives at most one extension equal to it
        for (int j = lane + nb; j < nc; j += 64) {
            const int m = cmerge[j];
            if (m >= 0) {
                cpnb[m] = lae_dev(cpnb[m], cpnb[j]);
                cpnb[j] = -INFINITY;
            }
        }
        __syncthreads();
        for (int j = lane; j < nc; j += 64)
            cscore[j] = (j >= nb && cmerge[j] >= 0) ? -INFINITY : lae_dev(cpb[j], cpnb[j]);
        __syncthreads();
        // the B best candidates, in order (ties: lower candidate index)
        const int nxt = cur ^ 1;
        if (nc <= 128) {
            // one pass: a candidate's rank is the number of candidates ahead
            // of it, and the first B ranks become the next beams
            for (int j = lane; j < nc; j += 64) {
                const float sj = cscore[j];
                int rank = 0;
#pragma unroll 8
                for (int q = 0; q < nc; ++q) {
                    const float sq = cscore[q];
                    rank += (sq > sj || (sq == sj && q < j)) ? 1 : 0;
                }
                if (sj > -INFINITY && rank < B) {
                    bh[nxt][rank] = ch[j];
                    blen[nxt][rank] = clen[j];
                    blast[nxt][rank] = clast[j];
                    bpb[nxt][rank] = cpb[j];
                    bpnb[nxt][rank] = cpnb[j];
                    bpe[(long long)t * KMAX + rank] = (cpar[j] << 20) | capp[j];
                }
            }
            int finite = 0;
            for (int j0 = 0; j0 < nc; j0 += 64) {
                const int j = j0 + lane;
                finite += __popcll(__ballot(j < nc && cscore[j] > -INFINITY));
            }
            if (lane == 0) nbeam = min(B, finite);
            __syncthreads();
        } else {
            // B rounds of a wave-wide maximum
            int kept = 0;
            for (int r = 0; r < B; ++r) {
                float best = -INFINITY;
                int bi = CMAX;
                for (int j = lane; j < nc; j += 64)
                    if (cscore[j] > best || (cscore[j] == best && j < bi && cscore[j] > -INFINITY)) {
                        best = cscore[j];
                        bi = j;
                    }
#pragma unroll
                for (int o = 32; o >= 1; o >>= 1) {
                    const float ob = __shfl_xor(best, o, 64);
                    const int oi = __shfl_xor(bi, o, 64);
                    if (ob > best || (ob == best && oi < bi)) { best = ob; bi = oi; }
                }
                if (bi >= CMAX || best == -INFINITY) break;
                if (lane == 0) {
                    bh[nxt][r] = ch[bi];
                    blen[nxt][r] = clen[bi];
                    blast[nxt][r] = clast[bi];
                    bpb[nxt][r] = cpb[bi];
                    bpnb[nxt][r] = cpnb[bi];
                    bpe[(long long)t * KMAX + r] = (cpar[bi] << 20) | capp[bi];
                    cscore[bi] = -INFINITY;
                }
                __syncthreads();
                ++kept;
            }
            if (lane == 0) nbeam = kept;
            __syncthreads();
        }
        cur = nxt;
    }
    if (lane == 0) {  // trace the best final beam back to frame 0
        int best = 0;
        float bs = lae_dev(bpb[cur][0], bpnb[cur][0]);
        for (int j = 1; j < nbeam; ++j) {
            const float sj = lae_dev(bpb[cur][j], bpnb[cur][j]);
            if (sj > bs) { bs = sj; best = j; }
        }
        const int n = blen[cur][best];
        int* out = tok + f0;
        int w = n, beam = best;
        for (int t = T - 1; t >= 0; --t) {
            const int e = bpe[(long long)t * KMAX + beam];
            if ((e & 0xFFFFF) != 0) out[--w] = (e & 0xFFFFF) - 1;
            beam = e >> 20;
        }
        cnt[b] = n;
    }
}

// ------------------------------------------------------------- greedy step
//
// The greedy choice (largest logit, lowest id on ties) in two stages. Every
// candidate id i with logit v becomes the 64-bit key (order-preserving bits
// of v << 32 | ~i): the largest key has the largest value and, among equal
// values, the lowest id, whatever order keys are compared in. (1) Partial
// maxima: in the bf16 model the output head's own kernel reduces its
// workgroup's 32 ids per row and writes one key per (row, workgroup)
// (head_argmax_kernel, below the decode projections); the fp32 model writes
// its logits and argmax_keys_kernel reduces ARGMAX_CHUNKS chunks per row.
// (2) argmax_step_kernel: one wave per row takes the largest of the row's
// keys, records the token, feeds it (or the forced token) as the next input
// once the prompt is consumed, and advances the slot's position.
// Logit filters (optional): ids whose bit is set in `never` cannot be
// chosen, ids set in `first` not as a row's first generated token (the row
// is at its first generated token when its input is the prompt's last).
// A row with no admissible key (every id filtered, which the API refuses,
// or keys lost to non-numbers) records token 0 and raises *err.
constexpr int ARGMAX_CHUNKS = 16;

struct TokenFilter {
    const unsigned* never;  // [V / 32 + 1] bit mask, or null
    const unsigned* first;  // [V / 32 + 1] bit mask, or null
    const int* list;        // row -> slot
    const int* pos;         // slot -> input position
    const int* n_prompt;    // slot -> prompt length
};

__host__ __device__ inline unsigned long long amax_key(float v, int i) {
    return ((unsigned long long)f2ord(v) << 32) | (unsigned long long)(0xffffffffu - (unsigned)i);
}
// The token of a row's largest key; a row without any key (k = 0) gets
// token 0 and sets *bad.
__host__ __device__ inline int key_token(unsigned long long k, int* bad) {
    if (k == 0ull) {
        *bad = 1;
        return 0;
    }
    return (int)(0xffffffffu - (unsigned)(k & 0xffffffffull));
}

// fp32 model: keys[r][chunk] = the largest key of chunk `chunk` of row r's logits.
__global__ __launch_bounds__(256) void argmax_keys_kernel(const float* __restrict__ logits, int V,
                                                          unsigned long long* __restrict__ keys, TokenFilter f) {
    const int r = blockIdx.y, t = threadIdx.x;
    const int per = (V + ARGMAX_CHUNKS - 1) / ARGMAX_CHUNKS;
    const int lo = blockIdx.x * per, hi = min(V, lo + per);
    const float* lg = logits + (long long)r * V;
    const unsigned* never = f.never;
    const unsigned* first = nullptr;
    if (f.first) {
        const int s = f.list[r];
        if (f.pos[s] == f.n_prompt[s] - 1) first = f.first;
    }
    unsigned long long k = 0;
    for (int i = lo + t; i < hi; i += 256 * 4) {
        float v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = (i + 256 * q < hi) ? lg[i + 256 * q] : 0.f;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int j = i + 256 * q;
            if (j >= hi) continue;
            const unsigned bit = 1u << (j & 31);
            if ((never && (never[j >> 5] & bit)) || (first && (first[j >> 5] & bit))) continue;
            const unsigned long long c = amax_key(v[q], j);
            k = c > k ? c : k;
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const unsigned long long c = __shfl_xor(k, o, 64);
        k = c > k ? c : k;
    }
    __shared__ unsigned long long sk[4];
    if ((t & 63) == 0) sk[t >> 6] = k;
    __syncthreads();
    if (t == 0) {
        unsigned long long m = sk[0];
        for (int w = 1; w < 4; ++w) m = sk[w] > m ? sk[w] : m;
        keys[(long long)r * ARGMAX_CHUNKS + blockIdx.x] = m;
    }
}

// eot >= 0: the first time a slot's generated token is eot, stop_at[slot]
// becomes the number of tokens generated before it. One wave per row over
// its nk keys.
__global__ __launch_bounds__(64) void argmax_step_kernel(const unsigned long long* __restrict__ keys, int nk,
                                                         const int* __restrict__ list, int* __restrict__ pos,
                                                         const int* __restrict__ n_prompt, int* __restrict__ seq,
                                                         int* __restrict__ gen, const int* __restrict__ forced,
                                                         int* __restrict__ out_tok, int eot,
                                                         int* __restrict__ stop_at, int* __restrict__ err) {
    const int r = blockIdx.x, lane = threadIdx.x;
    const unsigned long long* kr = keys + (long long)r * nk;
    // 16 loads in flight per lane (the keys come from other XCDs' writes);
    // the maximum of integers does not depend on the order it is taken in
    unsigned long long kk[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) kk[u] = 0;
    for (int j0 = lane; j0 < nk; j0 += 64 * 16) {
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const int j = j0 + 64 * u;
            const unsigned long long c = j < nk ? kr[j] : 0ull;
            kk[u] = c > kk[u] ? c : kk[u];
        }
    }
    unsigned long long k = kk[0];
#pragma unroll
    for (int u = 1; u < 16; ++u) k = kk[u] > k ? kk[u] : k;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const unsigned long long c = __shfl_xor(k, o, 64);
        k = c > k ? c : k;
    }
    if (lane != 0) return;
    int bad = 0;
    const int tok = key_token(k, &bad);
    if (bad) atomicOr(err, 1);
    const int s = list[r], p = pos[s], np = n_prompt[s];
    if (p >= np - 1) {
        const int g = p - (np - 1);
        if (eot >= 0 && tok == eot && stop_at[s] < 0) stop_at[s] = g;
        gen[s * 448 + g] = tok;
        seq[s * 448 + p + 1] = forced ? forced[r] : tok;
        out_tok[r] = tok;
    } else {
        out_tok[r] = -1;
    }
    pos[s] = p + 1;
}

// Output head with the first stage of the greedy choice (bf16 model): the
// decode projection of the tied token embedding (RT = 2: 32 vocabulary rows
// per workgroup), then, per activation row, the largest key (amax_key) over
// the workgroup's admissible ids, written to keys[row][blockIdx.x]; the
// logits themselves are stored only when `logits` is set (fp32, [n][V]).
// Filter bits and the rows' first-token flags are loaded before the main
// loop.
struct HeadArgs {
    float* logits;              // [n][V] or null
    unsigned long long* keys;   // [n][gridDim.x]
    int V;
    TokenFilter f;
};

template <int NT, int U>
__global__ __launch_bounds__(256) void head_argmax_kernel(const bf16* __restrict__ W, const bf16* __restrict__ X,
                                                          int nks_tot, int n, int Kc, HeadArgs h) {
    constexpr int RT = 2;
    __shared__ float red[3 * RT * NT * 4 * 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int fr = lane & 15, fc = lane >> 4;
    const int i0 = blockIdx.x * 16 * RT;
    unsigned excl[RT][NT];  // bit q: id i + q is not admissible for this row
    if (wave == 0) {
#pragma unroll
        for (int u = 0; u < NT; ++u) {
            const int r = u * 16 + fr;
            bool first = false;
            if (h.f.first && r < n) {
                const int sl = h.f.list[r];
                first = h.f.pos[sl] == h.f.n_prompt[sl] - 1;
            }
#pragma unroll
            for (int t = 0; t < RT; ++t) {
                const int i = i0 + t * 16 + fc * 4;
                unsigned m = 0;
                if (r < n && i < h.V) {
                    if (h.f.never) m |= (h.f.never[i >> 5] >> (i & 31)) & 0xfu;
                    if (first) m |= (h.f.first[i >> 5] >> (i & 31)) & 0xfu;
                }
                excl[t][u] = m;
            }
        }
    }
    float v[RT][NT][4];
    skinny_core<RT, NT, U>(W, X, nks_tot, n, Kc, red, v);
    if (wave > 0) return;
#pragma unroll
    for (int u = 0; u < NT; ++u) {
        const int r = u * 16 + fr;
        unsigned long long k = 0;
#pragma unroll
        for (int t = 0; t < RT; ++t) {
            const int i = i0 + t * 16 + fc * 4;
            if (r >= n) continue;
            if (h.logits) {
                float* p = h.logits + (long long)r * h.V + i;
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (i + q < h.V) p[q] = v[t][u][q];
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                if (i + q >= h.V || ((excl[t][u] >> q) & 1u)) continue;
                const unsigned long long c = amax_key(v[t][u][q], i + q);
                k = c > k ? c : k;
            }
        }
        // ids i0 .. i0 + 31 of row r are spread over lanes fr, fr + 16, fr + 32, fr + 48
        unsigned long long c = __shfl_xor(k, 16, 64);
        k = c > k ? c : k;
        c = __shfl_xor(k, 32, 64);
        k = c > k ? c : k;
        if (fc == 0 && r < n) h.keys[(long long)r * gridDim.x + blockIdx.x] = k;
    }
}

// Output head + per-workgroup keys for n rows (W: fragment-major [V rounded
// up to 32][K], X fragment-major [n rounded up to 16][K]); returns the number
// of keys per row.
inline int head_argmax(const bf16* W, int V, const bf16* X, int n, int K, const HeadArgs& h, hipStream_t st) {
    if (K % 32 || n <= 0 || n > 128 || V <= 0) throw ArgError(-1, "head_argmax: unsupported shape");
    const int nks = K / 32, tiles = (V + 31) / 32;
    WMI_SKINNY_NT(n, WMI_SKINNY_U(K, NT, hipLaunchKernelGGL((head_argmax_kernel<NT, U>), dim3(tiles), dim3(256), 0,
                                                             st, W, X, nks, n, K, h)));
    return tiles;
}

// Seat prompts: for entry e, slot slots[e] gets tokens prompts[e * 448 ...]
// (position 0, no end of text seen).
// prefilled = 1: positions 0 .. n_prompt - 2 are run at encode time, so the
// slot's first decode step is at its last prompt position.
__global__ void seat_kernel(const int* __restrict__ slots, const int* __restrict__ np_in,
                            const int* __restrict__ prompts, int* __restrict__ seq, int* __restrict__ pos,
                            int* __restrict__ n_prompt, int* __restrict__ stop_at, int prefilled) {
    const int e = blockIdx.x, s = slots[e];
    for (int i = threadIdx.x; i < 448; i += blockDim.x) seq[s * 448 + i] = i < np_in[e] ? prompts[e * 448 + i] : 0;
    if (threadIdx.x == 0) {
        pos[s] = prefilled ? np_in[e] - 1 : 0;
        n_prompt[s] = np_in[e];
        stop_at[s] = -1;
    }
}

}  // namespace wmi
