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

// One workgroup per segment: max over valid frames of the log-mel, clamp to
// max - 8, (L + 4) / 4, zero the frames beyond the segment in pad mode 1.
// Writes fp32 in place (frame-major [3000][n_mels]) and the conv input
// Ypad[z][1 + f][c] in T.
template <class T>
__global__ __launch_bounds__(1024) void mel_norm_kernel(float* __restrict__ logmel, T* __restrict__ ypad,
                                                        const int* __restrict__ nvalid, int n_mels) {
    const int z = blockIdx.x;
    float* L = logmel + (long long)z * 3000 * n_mels;
    const int nv = nvalid[z] * n_mels;
    float m = -INFINITY;
    for (int e = threadIdx.x; e < nv; e += blockDim.x) m = fmaxf(m, L[e]);
    m = wave_max(m);
    __shared__ float red[16];
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x < 64) {
        float v = threadIdx.x < (blockDim.x >> 6) ? red[threadIdx.x] : -INFINITY;
        v = wave_max(v);
        if (threadIdx.x == 0) red[0] = v;
    }
    __syncthreads();
    const float floor_ = red[0] - 8.0f;
    T* Y = ypad + (long long)z * 3002 * CP;
    for (int e = threadIdx.x; e < 3000 * n_mels; e += blockDim.x) {
        const int f = e / n_mels, c = e - f * n_mels;
        const float y = e < nv ? (fmaxf(L[e], floor_) + 4.0f) * 0.25f : 0.0f;
        L[e] = y;
        stf(Y + (long long)(f + 1) * CP + c, y);
    }
}

// ------------------------------------------------------------- layer norm

// One wavefront per row of width d (d % 64 == 0, d <= 2048): fp32 mean and
// biased variance, eps 1e-5, gain and bias.
template <class T>
__global__ __launch_bounds__(256) void layer_norm_kernel(const float* __restrict__ x, T* __restrict__ y,
                                                         const float* __restrict__ g, const float* __restrict__ b,
                                                         int rows, int d) {
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (row >= rows) return;
    const float* xr = x + (long long)row * d;
    const int E = d >> 6;
    float v[32];
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < 32; ++e)
        if (e < E) { v[e] = xr[lane + 64 * e]; s += v[e]; }
    const float mean = wave_sum(s) / d;
    float q = 0.f;
#pragma unroll
    for (int e = 0; e < 32; ++e)
        if (e < E) { const float c = v[e] - mean; q += c * c; }
    const float rstd = rsqrtf(wave_sum(q) / d + 1e-5f);
    T* yr = y + (long long)row * d;
#pragma unroll
    for (int e = 0; e < 32; ++e)
        if (e < E) {
            const int c = lane + 64 * e;
            stf(yr + c, (v[e] - mean) * rstd * g[c] + b[c]);
        }
}

// ------------------------------------------------------------- decoder embedding

template <class T>
__global__ __launch_bounds__(256) void embed_kernel(const T* __restrict__ tok_emb, const T* __restrict__ pos_emb,
                                                    const int* __restrict__ list, const int* __restrict__ pos,
                                                    const int* __restrict__ seq, float* __restrict__ x, int d) {
    const int r = blockIdx.x, s = list[r], p = pos[s];
    const int tok = seq[s * 448 + p];
    for (int c = threadIdx.x; c < d; c += blockDim.x)
        x[(long long)r * d + c] = ldf(tok_emb + (long long)tok * d + c) + ldf(pos_emb + (long long)p * d + c);
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
    float mrun[4], lrun[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) { mrun[u] = -INFINITY; lrun[u] = 0.f; }

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
    auto lstore = [&](int buf) {
        unsigned char* tk = lds + buf * 2 * ea::TILE;
        unsigned char* tv = tk + ea::TILE;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            *reinterpret_cast<u32x4*>(tk + swz(lr + 32 * s, lc)) = rk[s];
            *reinterpret_cast<u32x4*>(tv + swz(lr + 32 * s, lc)) = rv[s];
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
        // S^T = K Q^T : sc[key tile][query tile]
        mfma_f32x4 sc[4][4];
#pragma unroll
        for (int a = 0; a < 4; ++a) {
            const mfma_bf16x8 k0f = *reinterpret_cast<const mfma_bf16x8*>(tk + swz(a * 16 + fr, fc));
            const mfma_bf16x8 k1f = *reinterpret_cast<const mfma_bf16x8*>(tk + swz(a * 16 + fr, 4 + fc));
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                mfma_f32x4 t = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
                t = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0f, qf[u][0], t, 0, 0, 0);
                sc[a][u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1f, qf[u][1], t, 0, 0, 0);
            }
        }
        // mask keys beyond the window (last tile only)
        const int kbase = kt * ea::KT;
        if (kbase + ea::KT > N_CTX) {
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (kbase + a * 16 + fc * 4 + r >= N_CTX)
#pragma unroll
                        for (int u = 0; u < 4; ++u) sc[a][u][r] = -INFINITY;
        }
        // online softmax per query column (log2 domain)
        mfma_bf16x8 pf[4][2];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            float mx = -INFINITY;
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int r = 0; r < 4; ++r) mx = fmaxf(mx, sc[a][u][r]);
            mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
            mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
            const float mnew = fmaxf(mrun[u], mx * LOG2E);
            const float alpha = exp2f(mrun[u] - mnew);
            mrun[u] = mnew;
            float ls = 0.f;
            float pv[4][4];
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    pv[a][r] = exp2f(fmaf(sc[a][u][r], LOG2E, -mnew));
                    ls += pv[a][r];
                }
            ls += __shfl_xor(ls, 16, 64);
            ls += __shfl_xor(ls, 32, 64);
            lrun[u] = lrun[u] * alpha + ls;
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int r = 0; r < 4; ++r) o[a][u][r] *= alpha;
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
        }
        // O^T += V^T P^T
#pragma unroll
        for (int a = 0; a < 4; ++a) {
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                // V^T row (dim) a*16 + fr, keys s*32 + fc*4 .. +3 and s*32 + 16 + fc*4 .. +3
                const int row = a * 16 + fr;
                const int kA = s * 32 + fc * 4, kB = kA + 16;
                const u32x2 lo = *reinterpret_cast<const u32x2*>(tv + swz(row, kA >> 3) + (kA & 7) * 2);
                const u32x2 hi = *reinterpret_cast<const u32x2*>(tv + swz(row, kB >> 3) + (kB & 7) * 2);
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
            s *= LOG2E;
            const float mnew = fmaxf(m, s);
            const float alpha = exp2f(m - mnew), p = exp2f(s - mnew);
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
// One wavefront per (row r, head h, chunk c) over the slot's cache: scores
// with K^T rows (lane owns PPL consecutive positions), softmax in fp32 with
// wavefront reductions, then P V with V rows (8 lanes per 128-byte row, 8
// rows per load). With one chunk the normalised output is written directly;
// otherwise (m, l, o[64]) partials go to `part` for the combine kernel.
template <class T>
__device__ inline void load_vec(const T* p, float* out, int n);
template <>
__device__ inline void load_vec<bf16>(const bf16* p, float* out, int n) {
    for (int i = 0; i < n; i += 4) { const float4 v = ld4(p + i); out[i] = v.x; out[i + 1] = v.y; out[i + 2] = v.z; out[i + 3] = v.w; }
}
template <>
__device__ inline void load_vec<float>(const float* p, float* out, int n) {
    for (int i = 0; i < n; i += 4) { const float4 v = ld4(p + i); out[i] = v.x; out[i + 1] = v.y; out[i + 2] = v.z; out[i + 3] = v.w; }
}

struct DecAttnArgs {
    const void* q;      // [n][d], scaled by 1/8
    const void* kt;     // cache K^T of this layer: [S][H][64][TP]
    const void* v;      // cache V of this layer:   [S][H][TP][64]
    void* out;          // [n][d]
    float* part;        // [n][H][n_chunks][66]
    const int* list;    // row -> slot
    const int* pos;     // slot -> position (self-attention), or nullptr
    int fixed_len;      // keys when pos is nullptr
    int TP, H, d, n_chunks;
};

template <class T, int PPL>
__global__ __launch_bounds__(64) void dec_attn_kernel(DecAttnArgs a) {
    __shared__ float qs[64];
    __shared__ float ps[64 * PPL];
    const int c = blockIdx.x, h = blockIdx.y, r = blockIdx.z, lane = threadIdx.x;
    const int slot = a.list[r];
    const int len = a.pos ? a.pos[slot] + 1 : a.fixed_len;
    const int start = c * 64 * PPL;
    const T* q = reinterpret_cast<const T*>(a.q) + (long long)r * a.d + h * 64;
    qs[lane] = ldf(q + lane);
    __syncthreads();
    const long long head = (long long)slot * a.H + h;
    const T* kt = reinterpret_cast<const T*>(a.kt) + head * 64 * a.TP;
    const T* vv = reinterpret_cast<const T*>(a.v) + head * a.TP * 64;

    float s[PPL];
#pragma unroll
    for (int i = 0; i < PPL; ++i) s[i] = 0.f;
    const int p0 = start + lane * PPL;
    if (p0 < len) {
#pragma unroll 8
        for (int j = 0; j < 64; ++j) {
            float kv[PPL];
            load_vec<T>(kt + (long long)j * a.TP + p0, kv, PPL);
            const float qj = qs[j];
#pragma unroll
            for (int i = 0; i < PPL; ++i) s[i] = fmaf(qj, kv[i], s[i]);
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < PPL; ++i) {
        s[i] = (p0 + i < len) ? s[i] * LOG2E : -INFINITY;
        mx = fmaxf(mx, s[i]);
    }
    mx = wave_max(mx);
    float lsum = 0.f;
#pragma unroll
    for (int i = 0; i < PPL; ++i) {
        const float p = (p0 + i < len) ? exp2f(s[i] - mx) : 0.f;
        ps[lane * PPL + i] = p;
        lsum += p;
    }
    lsum = wave_sum(lsum);
    __syncthreads();
    // P V: lane covers dims dg*8..+7 of positions pg, pg + 8, ...
    const int dg = lane & 7, pg = lane >> 3;
    float o[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = 0.f;
    const int nloc = min(64 * PPL, len - start);
    for (int pp = pg; pp < nloc; pp += 8) {
        float vr[8];
        load_vec<T>(vv + (long long)(start + pp) * 64 + dg * 8, vr, 8);
        const float p = ps[pp];
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = fmaf(p, vr[i], o[i]);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        o[i] += __shfl_xor(o[i], 8, 64);
        o[i] += __shfl_xor(o[i], 16, 64);
        o[i] += __shfl_xor(o[i], 32, 64);
    }
    if (a.n_chunks == 1) {
        if (lane < 8) {
            const float inv = 1.0f / lsum;
            T* out = reinterpret_cast<T*>(a.out) + (long long)r * a.d + h * 64 + dg * 8;
            st4(out, o[0] * inv, o[1] * inv, o[2] * inv, o[3] * inv);
            st4(out + 4, o[4] * inv, o[5] * inv, o[6] * inv, o[7] * inv);
        }
        return;
    }
    float* pr = a.part + (((long long)r * a.H + h) * a.n_chunks + c) * 66;
    if (lane == 0) { pr[0] = mx; pr[1] = lsum; }
    if (lane < 8) {
        st4(pr + 2 + dg * 8, o[0], o[1], o[2], o[3]);
        st4(pr + 6 + dg * 8, o[4], o[5], o[6], o[7]);
    }
}

// Combine chunk partials: out = sum_c 2^(m_c - M) o_c / sum_c 2^(m_c - M) l_c.
template <class T>
__global__ __launch_bounds__(64) void dec_attn_combine_kernel(const float* __restrict__ part, T* __restrict__ out,
                                                              int H, int d, int n_chunks) {
    const int h = blockIdx.x, r = blockIdx.y, j = threadIdx.x;
    const float* pr = part + ((long long)r * H + h) * n_chunks * 66;
    float M = -INFINITY;
    for (int c = 0; c < n_chunks; ++c) M = fmaxf(M, pr[c * 66]);
    float L = 0.f, o = 0.f;
    for (int c = 0; c < n_chunks; ++c) {
        const float m = pr[c * 66];
        const float w = m == -INFINITY ? 0.f : exp2f(m - M);
        L += w * pr[c * 66 + 1];
        o += w * pr[c * 66 + 2 + j];
    }
    stf(out + (long long)r * d + h * 64 + j, o / L);
}

// ------------------------------------------------------------- skinny decode GEMM (bf16 MFMA)
//
// C[i][r] = sum_k W[i][k] X[r][k] for a few rows r (active decode slots,
// n <= 16 * NT) and many weight rows i: each weight byte is read once.
// Workgroup = 4 waves over 16 * RT weight rows; the waves split K in
// interleaved 32-wide steps and their partial sums are added in LDS in a
// fixed order (so a row's result never depends on the other rows present).
template <int RT, int NT, class Epi>
__global__ __launch_bounds__(256) void skinny_bf16_kernel(const bf16* __restrict__ W, int MA,
                                                          const bf16* __restrict__ X, int n, int K, Epi epi) {
    __shared__ float red[3][RT * NT * 4][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int fr = lane & 15, fc = lane >> 4;
    const int i0 = blockIdx.x * 16 * RT;
    const bf16* wp[RT];
#pragma unroll
    for (int t = 0; t < RT; ++t) wp[t] = W + (long long)min(i0 + t * 16 + fr, MA - 1) * K + fc * 8;
    const bf16* xp[NT];
#pragma unroll
    for (int u = 0; u < NT; ++u) xp[u] = X + (long long)min(u * 16 + fr, n - 1) * K + fc * 8;
    mfma_f32x4 acc[RT][NT];
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int u = 0; u < NT; ++u) acc[t][u] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};
    const int nks = K >> 5;
#pragma unroll 4
    for (int s = wave; s < nks; s += 4) {
        const int k = s * 32;
        mfma_bf16x8 a[RT], b[NT];
#pragma unroll
        for (int t = 0; t < RT; ++t) a[t] = *reinterpret_cast<const mfma_bf16x8*>(wp[t] + k);
#pragma unroll
        for (int u = 0; u < NT; ++u) b[u] = *reinterpret_cast<const mfma_bf16x8*>(xp[u] + k);
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int u = 0; u < NT; ++u) acc[t][u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[t], b[u], acc[t][u], 0, 0, 0);
    }
    if (wave > 0) {
#pragma unroll
        for (int t = 0; t < RT; ++t)
#pragma unroll
            for (int u = 0; u < NT; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e) red[wave - 1][(t * NT + u) * 4 + e][lane] = acc[t][u][e];
    }
    __syncthreads();
    if (wave > 0) return;
#pragma unroll
    for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int u = 0; u < NT; ++u) {
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int idx = (t * NT + u) * 4 + e;
                v[e] = ((acc[t][u][e] + red[0][idx][lane]) + red[1][idx][lane]) + red[2][idx][lane];
            }
            const int i = i0 + t * 16 + fc * 4, r = u * 16 + fr;
            if (i < MA && r < n) epi(i, r, 0, v[0], v[1], v[2], v[3]);
        }
}

template <class Epi>
inline void skinny_bf16(const bf16* W, int MA, const bf16* X, int n, int K, const Epi& epi, hipStream_t st) {
    if (K % 32 || n <= 0 || n > 128 || MA <= 0) throw ArgError(-1, "skinny_bf16: unsupported shape");
    const bool big = MA >= 16384;  // output head: 32 rows per workgroup
#define WMI_SKINNY(RT, NT)                                                                       \
    hipLaunchKernelGGL((skinny_bf16_kernel<RT, NT, Epi>), dim3((MA + 16 * RT - 1) / (16 * RT)), \
                       dim3(256), 0, st, W, MA, X, n, K, epi)
    if (big) {
        if (n <= 16) WMI_SKINNY(2, 1); else if (n <= 32) WMI_SKINNY(2, 2);
        else if (n <= 64) WMI_SKINNY(2, 4); else WMI_SKINNY(2, 8);
    } else {
        if (n <= 16) WMI_SKINNY(1, 1); else if (n <= 32) WMI_SKINNY(1, 2);
        else if (n <= 64) WMI_SKINNY(1, 4); else WMI_SKINNY(1, 8);
    }
#undef WMI_SKINNY
}

// ------------------------------------------------------------- greedy step
//
// One workgroup per row: argmax of the logits (lowest id on exact ties);
// records it, feeds it (or the forced token) as the slot's next input once
// the prompt is consumed, and advances the slot's position.
__global__ __launch_bounds__(256) void argmax_step_kernel(const float* __restrict__ logits, int V,
                                                          const int* __restrict__ list, int* __restrict__ pos,
                                                          const int* __restrict__ n_prompt, int* __restrict__ seq,
                                                          int* __restrict__ gen, const int* __restrict__ forced,
                                                          int* __restrict__ out_tok) {
    const int r = blockIdx.x, t = threadIdx.x;
    const float* lg = logits + (long long)r * V;
    float best = -INFINITY;
    int bi = 0x7fffffff;
    for (int i = t; i < V; i += 256) {
        const float v = lg[i];
        if (v > best) { best = v; bi = i; }  // i increases: first maximum kept
    }
    __shared__ float sv[256];
    __shared__ int si[256];
    sv[t] = best;
    si[t] = bi;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (t < w) {
            const float ov = sv[t + w];
            const int oi = si[t + w];
            if (ov > sv[t] || (ov == sv[t] && oi < si[t])) { sv[t] = ov; si[t] = oi; }
        }
        __syncthreads();
    }
    if (t == 0) {
        const int s = list[r], p = pos[s], np = n_prompt[s];
        const int tok = si[0];
        if (p >= np - 1) {
            gen[s * 448 + (p - (np - 1))] = tok;
            seq[s * 448 + p + 1] = forced ? forced[r] : tok;
            out_tok[r] = tok;
        } else {
            out_tok[r] = -1;
        }
        pos[s] = p + 1;
    }
}

// Seat prompts: for entry e, slot slots[e] gets tokens prompts[e * 448 ...].
__global__ void seat_kernel(const int* __restrict__ slots, const int* __restrict__ np_in,
                            const int* __restrict__ prompts, int* __restrict__ seq, int* __restrict__ pos,
                            int* __restrict__ n_prompt) {
    const int e = blockIdx.x, s = slots[e];
    for (int i = threadIdx.x; i < 448; i += blockDim.x) seq[s * 448 + i] = i < np_in[e] ? prompts[e * 448 + i] : 0;
    if (threadIdx.x == 0) { pos[s] = 0; n_prompt[s] = np_in[e]; }
}

}  // namespace wmi
