// GEMM epilogues: each receives four consecutive output rows i0..i0+3 (the
// A-operand dimension) of column j in batch z and writes them where the next
// stage reads them. All biases and norms are fp32; T is the activation
// storage type (float or bf16).
//
// Encoder buffers (nb segments, token m = z * 1500 + t):
//   Ypad  [nb][3002][128]   normalised log-mel, row 1 + frame, zero rows 0 and 3001
//   H1pad [nb][3002][d]     first conv output, row 1 + t, zero row 0
//   x     [nb * 1500][d]    fp32 residual stream
//   Qh,Kh [nb][H][TQ][64]   per-head queries (scaled by log2(e)/8) and keys
//   Vt    [nb][H][64][TQ]   per-head values, transposed
// Decoder caches (slot s, layer l, head h):
//   self  Kt [l][s][h][64][TS], V [l][s][h][TS][64]
//   cross Kt [l][s][h][64][TC], V [l][s][h][TC][64]
#pragma once

#include "common.h"

namespace wmi {

constexpr int N_CTX = 1500;  // encoder positions of a 30 s window
constexpr int TQ = 1536;     // padded encoder positions per head
constexpr int TS = 512;      // self-attention cache stride (>= 448)
constexpr int TC = 1536;     // cross-attention cache stride (>= 1500)
constexpr int CP = 128;      // padded mel channels of the conv input

// Epilogues run in two phases so a lane's loads are issued together: pre()
// loads whatever the store needs (bias, residual, table, slot) into an
// EpiPre, then operator() computes and stores. Unused fields cost nothing.
struct EpiPre {
    float4 a, b;
    int s;
};

template <class T>
struct EpiConv1 {  // i = channel, j = frame
    const float* bias;
    T* h1;  // H1pad
    int d;
    __device__ EpiPre pre(int i, int, int) const { EpiPre p{}; p.a = ld4(bias + i); return p; }
    __device__ void operator()(int i, int j, int z, float a, float b, float c, float e, const EpiPre& p) const {
        st4(h1 + ((long long)z * 3002 + j + 1) * d + i, gelu_erf(a + p.a.x), gelu_erf(b + p.a.y),
            gelu_erf(c + p.a.z), gelu_erf(e + p.a.w));
    }
};

struct EpiConv2 {  // i = channel, j = position; adds the sinusoid table
    const float* bias;
    const float* pe;  // [1500][d]
    float* x;
    int d;
    __device__ EpiPre pre(int i, int j, int) const {
        EpiPre p{};
        p.a = ld4(bias + i);
        p.b = ld4(pe + (long long)j * d + i);
        return p;
    }
    __device__ void operator()(int i, int j, int z, float a, float b, float c, float e, const EpiPre& p) const {
        st4(x + ((long long)z * N_CTX + j) * d + i, gelu_erf(a + p.a.x) + p.b.x, gelu_erf(b + p.a.y) + p.b.y,
            gelu_erf(c + p.a.z) + p.b.z, gelu_erf(e + p.a.w) + p.b.w);
    }
};

template <class T>
struct EpiQK {  // A = [Wq; Wk] (2d rows), B = tokens
    const float* bq;
    T* q;
    T* k;
    int d, H;
    __device__ EpiPre pre(int i, int, int) const {
        EpiPre p{};
        if (i < d) p.a = ld4(bq + i);
        return p;
    }
    __device__ void operator()(int i, int m, int, float a, float b, float c, float e, const EpiPre& p) const {
        const int bseg = m / N_CTX, t = m - bseg * N_CTX;
        if (i < d) {
            const int h = i >> 6, jj = i & 63;
            // 1/8 = 1/sqrt(64), and log2(e) so that attention works in base 2
            constexpr float qs = 0.125f * 1.4426950408889634f;
            st4(q + (((long long)bseg * H + h) * TQ + t) * 64 + jj, (a + p.a.x) * qs, (b + p.a.y) * qs,
                (c + p.a.z) * qs, (e + p.a.w) * qs);
        } else {
            const int f = i - d, h = f >> 6, jj = f & 63;
            st4(k + (((long long)bseg * H + h) * TQ + t) * 64 + jj, a, b, c, e);
        }
    }
};

template <class T>
struct EpiVt {  // A = tokens (4 consecutive positions), B = Wv
    const float* bv;
    T* vt;
    int H;
    __device__ EpiPre pre(int, int f, int) const { EpiPre p{}; p.a.x = bv[f]; return p; }
    __device__ void operator()(int m, int f, int, float a, float b, float c, float e, const EpiPre& p) const {
        const int bseg = m / N_CTX, t = m - bseg * N_CTX;
        const int h = f >> 6, jj = f & 63;
        const float bb = p.a.x;
        st4(vt + (((long long)bseg * H + h) * 64 + jj) * TQ + t, a + bb, b + bb, c + bb, e + bb);
    }
};

struct EpiResid {  // x[j][i..i+3] += v + bias
    const float* bias;
    float* x;
    int ld;
    __device__ EpiPre pre(int i, int j, int) const {
        EpiPre p{};
        p.a = ld4(bias + i);
        p.b = ld4(x + (long long)j * ld + i);
        return p;
    }
    __device__ void operator()(int i, int j, int, float a, float b, float c, float e, const EpiPre& p) const {
        st4(x + (long long)j * ld + i, p.b.x + a + p.a.x, p.b.y + b + p.a.y, p.b.z + c + p.a.z, p.b.w + e + p.a.w);
    }
};

// out[j][i..i+3] = gelu(v + bias); DEC: out is a decoder activation (dec_off), else row-major.
template <class T, bool DEC = false>
struct EpiGelu {
    const float* bias;
    T* out;
    int ld;
    __device__ EpiPre pre(int i, int, int) const { EpiPre p{}; p.a = ld4(bias + i); return p; }
    __device__ void operator()(int i, int j, int, float a, float b, float c, float e, const EpiPre& p) const {
        st4(out + (DEC ? dec_off<T>(j, i, ld) : (long long)j * ld + i), gelu_erf(a + p.a.x), gelu_erf(b + p.a.y),
            gelu_erf(c + p.a.z), gelu_erf(e + p.a.w));
    }
};

// Layer index n / d of a column n of the stacked per-layer weights, with
// rd = 1 / d rounded to fp32. For n < 2^20 and d <= 2^11, (n + 1/2) / d lies
// at least 1 / (2 d) >= 2^-12 from an integer, while the product's error is
// below (n / d) 2^-23 < 2^-14 (n + 1/2 is exact; rd and the product are
// each rounded once), so truncation gives the exact quotient. This replaces
// an integer division (a long instruction sequence) per output.
__device__ inline int layer_of(int n, float rd) { return (int)(__fmul_rn((float)n + 0.5f, rd)); }

template <class T>
struct EpiCrossK {  // A = encoder output (4 consecutive positions), B = [Wk of every layer]
    T* kt;               // cross K cache
    const int* slot_of;  // batch entry -> slot
    int d, H, S;
    float rd;            // 1 / d
    __device__ EpiPre pre(int m, int, int) const { EpiPre p{}; p.s = slot_of[m / N_CTX]; return p; }
    __device__ void operator()(int m, int n, int, float a, float b, float c, float e, const EpiPre& p) const {
        const int bseg = m / N_CTX, t = m - bseg * N_CTX;
        const int l = layer_of(n, rd), f = n - l * d, h = f >> 6, jj = f & 63;
        const long long base = (((long long)l * S + p.s) * H + h) * 64 + jj;
        st4(kt + base * TC + t, a, b, c, e);
    }
};

template <class T>
struct EpiCrossV {  // A = [Wv of every layer], B = encoder output
    const float* bv;  // [L * d]
    T* v;             // cross V cache
    const int* slot_of;
    int d, H, S;
    float rd;  // 1 / d
    __device__ EpiPre pre(int n, int m, int) const {
        EpiPre p{};
        p.a = ld4(bv + n);
        p.s = slot_of[m / N_CTX];
        return p;
    }
    __device__ void operator()(int n, int m, int, float a, float b, float c, float e, const EpiPre& p) const {
        const int bseg = m / N_CTX, t = m - bseg * N_CTX;
        const int l = layer_of(n, rd), f = n - l * d, h = f >> 6, jj = f & 63;
        const long long row = (((long long)l * S + p.s) * H + h) * TC + t;
        st4(v + row * 64 + jj, a + p.a.x, b + p.a.y, c + p.a.z, e + p.a.w);
    }
};

// Decoder: A = [Wq; Wk; Wv] of one layer, B = normalised rows (row r -> slot
// list[r] at position rowpos[r], or at pos[list[r]] when rowpos is null).
// Queries go to q (scaled by 1/8); this position's key and value are appended
// to the slot's self-attention cache, and rowlen[r] = position + 1 (the
// number of cached positions the row attends to).
template <class T>
struct EpiDecQKV {
    const float* bq;
    const float* bv;
    T* q;
    T* kt;  // self K cache of this layer: [S][H][64][TS]
    T* v;   // self V cache of this layer: [S][H][TS][64]
    const int* list;
    const int* pos;
    const int* rowpos;
    int* rowlen;
    int d, H;
    __device__ EpiPre pre(int i, int r, int) const {
        EpiPre p{};
        if (i < d) {
            p.a = ld4(bq + i);
        } else {
            p.s = rowpos ? rowpos[r] : pos[list[r]];
            if (i >= 2 * d) p.a = ld4(bv + (i - 2 * d));
        }
        return p;
    }
    __device__ void operator()(int i, int r, int, float a, float b, float c, float e, const EpiPre& p) const {
        if (i < d) {
            st4(q + (long long)r * d + i, (a + p.a.x) * 0.125f, (b + p.a.y) * 0.125f, (c + p.a.z) * 0.125f,
                (e + p.a.w) * 0.125f);
            return;
        }
        const int s = list[r], ps = p.s;
        if (i == d) rowlen[r] = ps + 1;
        if (i < 2 * d) {
            const int f = i - d, h = f >> 6, jj = f & 63;
            T* base = kt + (((long long)s * H + h) * 64 + jj) * TS + ps;
            stf(base, a);
            stf(base + TS, b);
            stf(base + 2 * TS, c);
            stf(base + 3 * TS, e);
        } else {
            const int f = i - 2 * d, h = f >> 6, jj = f & 63;
            st4(v + (((long long)s * H + h) * TS + ps) * 64 + jj, a + p.a.x, b + p.a.y, c + p.a.z, e + p.a.w);
        }
    }
};

template <class T>
struct EpiQ {  // cross-attention queries, scaled by 1/8
    const float* bias;
    T* q;
    int d;
    __device__ EpiPre pre(int i, int, int) const { EpiPre p{}; p.a = ld4(bias + i); return p; }
    __device__ void operator()(int i, int r, int, float a, float b, float c, float e, const EpiPre& p) const {
        st4(q + (long long)r * d + i, (a + p.a.x) * 0.125f, (b + p.a.y) * 0.125f, (c + p.a.z) * 0.125f,
            (e + p.a.w) * 0.125f);
    }
};

// CTC head: A = head weights [n_vocab][d], B = encoder output rows (frames);
// logits[frame][i..i+3] = acc + bias[i..i+3] (fp32, row-major [frames][n_vocab]).
struct EpiCTC {
    const float* bias;
    float* out;
    int V;
    __device__ EpiPre pre(int i, int, int) const { EpiPre p{}; p.a = ld4(bias + i); return p; }
    __device__ void operator()(int i, int j, int, float a, float b, float c, float e, const EpiPre& p) const {
        st4(out + (long long)j * V + i, a + p.a.x, b + p.a.y, c + p.a.z, e + p.a.w);
    }
};

struct EpiLogits {  // out[r][i..i+3] (fp32), rows beyond n_vocab dropped
    float* out;
    int V;
    __device__ EpiPre pre(int, int, int) const { return EpiPre{}; }
    __device__ void operator()(int i, int r, int, float a, float b, float c, float e, const EpiPre&) const {
        float* p = out + (long long)r * V + i;
        if (i + 3 < V) {
            p[0] = a; p[1] = b; p[2] = c; p[3] = e;
        } else {
            if (i < V) p[0] = a;
            if (i + 1 < V) p[1] = b;
            if (i + 2 < V) p[2] = c;
        }
    }
};

}  // namespace wmi
