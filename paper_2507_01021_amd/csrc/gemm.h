// GEMM kernels: C[i][j] = sum_k A[i][k] * B[j][k] with A and B both stored
// row-major with K contiguous ("A times B transposed"), optionally batched.
//
// The result never goes to memory as a plain matrix: an epilogue functor
// receives each lane's output as four consecutive i for one j,
//     epi(i0, j, z, v0, v1, v2, v3)   (rows i0..i0+3 of batch z, column j),
// and stores it in whatever layout the consumer wants (bias, GELU, residual
// add, per-head or transposed cache layouts). Call sites pick which operand
// is A so that the four consecutive i are the contiguous output dimension.
//
// gemm_bf16: bf16 inputs, v_mfma_f32_16x16x32_bf16 with fp32 accumulation,
//   256x256x64 workgroup tile, 4 waves of 128x128, LDS double buffer with an
//   XOR swizzle on 16-byte chunks, next K tile prefetched into registers.
//   Requires K % 64 == 0, MA % 4 == 0, 16-byte aligned rows (lda, ldb % 8 == 0).
// gemm_simt: fp32 (or bf16 storage) SIMT kernel for the fp32 model and the
//   front end: 64x64x16 tile, 4x4 outputs per thread, any K, any lda.
#pragma once

#include "common.h"

namespace wmi {

typedef __bf16 mfma_bf16x8 __attribute__((ext_vector_type(8)));
typedef float mfma_f32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ bf16 MFMA

namespace gb {
constexpr int BM = 256;   // A rows per workgroup
constexpr int BN = 256;   // B rows per workgroup
constexpr int BK = 64;
constexpr int THREADS = 256;
constexpr int TILE_BYTES = BM * BK * 2;  // one operand tile (32 KiB)
}  // namespace gb

// Byte offset of 16-byte chunk c (0..7) of row r inside a [rows][64] bf16 LDS tile.
__device__ inline int swz(int r, int c) { return r * 128 + ((c ^ (r & 7)) << 4); }

// Eight 16-byte staging registers (named, so they never land in scratch).
struct Stage8 {
    u32x4 v0, v1, v2, v3, v4, v5, v6, v7;
};
// Loads 16-byte chunks of rows r0, r0 + 32, ..., r0 + 224 (clamped to nrows - 1).
__device__ __forceinline__ void gload8(Stage8& g, const bf16* p, int r0, int nrows, int ld, int k0) {
#define WMI_L(S) g.v##S = *reinterpret_cast<const u32x4*>(p + (long long)min(r0 + 32 * S, nrows - 1) * ld + k0)
    WMI_L(0); WMI_L(1); WMI_L(2); WMI_L(3); WMI_L(4); WMI_L(5); WMI_L(6); WMI_L(7);
#undef WMI_L
}
__device__ __forceinline__ void lstore8(const Stage8& g, unsigned char* dst, int lr, int lc) {
#define WMI_S(S) *reinterpret_cast<u32x4*>(dst + swz(lr + 32 * S, lc)) = g.v##S
    WMI_S(0); WMI_S(1); WMI_S(2); WMI_S(3); WMI_S(4); WMI_S(5); WMI_S(6); WMI_S(7);
#undef WMI_S
}

template <class Epi>
__global__ __launch_bounds__(256, 1) void gemm_bf16_kernel(
    const bf16* __restrict__ A, int lda, long long sA, const bf16* __restrict__ B, int ldb,
    long long sB, int MA, int MB, int K, int tilesA, Epi epi) {
    extern __shared__ __align__(16) unsigned char lds[];
    const int z = blockIdx.z;
    A += (long long)z * sA;
    B += (long long)z * sB;
    // Workgroups sharing a B tile (activations) run next to each other.
    const int ta = blockIdx.x % tilesA;
    const int tb = blockIdx.x / tilesA;
    const int a0 = ta * gb::BM, b0 = tb * gb::BN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wa = (wave & 1) * 128, wb = (wave >> 1) * 128;

    // Global -> register staging: thread copies 16-byte chunk (tid & 7) of
    // rows (tid >> 3) + 32 * s, s = 0..7 (rows past the end re-read the last row).
    const int lc = tid & 7, lr = tid >> 3;
    const bf16* Ab = A + lc * 8;
    const bf16* Bb = B + lc * 8;
    Stage8 stg;

    mfma_f32x4 acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};

#define WMI_GLOAD(P, ROW0, NROWS, LD, K0) gload8(stg, (P), (ROW0) + lr, (NROWS), (LD), (K0))
#define WMI_LSTORE(DST) lstore8(stg, (DST), lr, lc)

    const int nk = K / gb::BK;
    WMI_GLOAD(Ab, a0, MA, lda, 0);
    WMI_LSTORE(lds);
    WMI_GLOAD(Bb, b0, MB, ldb, 0);
    WMI_LSTORE(lds + gb::TILE_BYTES);
    __syncthreads();
    const int fr = lane & 15, fc = lane >> 4;  // fragment row, 8-element k group
    for (int kt = 0; kt < nk; ++kt) {
        const bool more = kt + 1 < nk;
        const unsigned char* ta_ = lds + (kt & 1) * 2 * gb::TILE_BYTES;
        const unsigned char* tb_ = ta_ + gb::TILE_BYTES;
        unsigned char* na_ = lds + ((kt + 1) & 1) * 2 * gb::TILE_BYTES;
        if (more) WMI_GLOAD(Ab, a0, MA, lda, (kt + 1) * gb::BK);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            mfma_bf16x8 fa[8];
#pragma unroll
            for (int i = 0; i < 8; ++i)
                fa[i] = *reinterpret_cast<const mfma_bf16x8*>(ta_ + swz(wa + i * 16 + fr, ks * 4 + fc));
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const mfma_bf16x8 fb = *reinterpret_cast<const mfma_bf16x8*>(tb_ + swz(wb + j * 16 + fr, ks * 4 + fc));
#pragma unroll
                for (int i = 0; i < 8; ++i)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb, acc[i][j], 0, 0, 0);
            }
            if (ks == 0 && more) {
                WMI_LSTORE(na_);
                WMI_GLOAD(Bb, b0, MB, ldb, (kt + 1) * gb::BK);
            }
        }
        if (more) WMI_LSTORE(na_ + gb::TILE_BYTES);
        __syncthreads();
    }
#undef WMI_GLOAD
#undef WMI_LSTORE
    // Lane holds C[i = base + 4*(lane>>4) + r][j = base + (lane & 15)].
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int jj = b0 + wb + j * 16 + fr;
        if (jj >= MB) continue;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int ii = a0 + wa + i * 16 + fc * 4;
            if (ii < MA) epi(ii, jj, z, acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
        }
    }
}

template <class Epi>
inline void gemm_bf16(const bf16* A, int lda, long long sA, const bf16* B, int ldb, long long sB,
                      int MA, int MB, int K, int batch, const Epi& epi, hipStream_t st) {
    if (K % gb::BK || MA % 4 || lda % 8 || ldb % 8 || MA <= 0 || MB <= 0 || batch <= 0)
        throw ArgError(-1, "gemm_bf16: unsupported shape");
    const int tilesA = (MA + gb::BM - 1) / gb::BM, tilesB = (MB + gb::BN - 1) / gb::BN;
    static bool attr_set = false;  // one per epilogue instantiation
    if (!attr_set) {
        WMI_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_bf16_kernel<Epi>),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, 4 * gb::TILE_BYTES));
        attr_set = true;
    }
    dim3 grid(tilesA * tilesB, 1, batch);
    hipLaunchKernelGGL(gemm_bf16_kernel<Epi>, grid, dim3(gb::THREADS), 4 * gb::TILE_BYTES, st, A, lda,
                       sA, B, ldb, sB, MA, MB, K, tilesA, epi);
}

// ----------------------------------------------------------------- SIMT fp32

template <class TA, class TB, class Epi>
__global__ __launch_bounds__(256) void gemm_simt_kernel(const TA* __restrict__ A, int lda, long long sA,
                                                        const TB* __restrict__ B, int ldb, long long sB,
                                                        int MA, int MB, int K, Epi epi) {
    __shared__ float As[16][64 + 4];
    __shared__ float Bs[16][64 + 4];
    const int z = blockIdx.z;
    A += (long long)z * sA;
    B += (long long)z * sB;
    const int a0 = blockIdx.x * 64, b0 = blockIdx.y * 64;
    const int t = threadIdx.x;
    const int ag = t & 15, bgp = t >> 4;  // this thread's 4 A rows and 4 B rows
    float acc[4][4] = {};
    const int lr = t >> 2, lk = (t & 3) * 4;  // loader: row lr, k lk..lk+3
    const long long rowA = min(a0 + lr, MA - 1), rowB = min(b0 + lr, MB - 1);
    for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            int k = k0 + lk + q;
            As[lk + q][lr] = k < K ? ldf(A + rowA * lda + k) : 0.f;
            Bs[lk + q][lr] = k < K ? ldf(B + rowB * ldb + k) : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            float a[4], b[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) { a[q] = As[k][ag * 4 + q]; b[q] = Bs[k][bgp * 4 + q]; }
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int y = 0; y < 4; ++y) acc[x][y] = fmaf(a[x], b[y], acc[x][y]);
        }
        __syncthreads();
    }
    const int ii = a0 + ag * 4;
    if (ii >= MA) return;
#pragma unroll
    for (int y = 0; y < 4; ++y) {
        const int jj = b0 + bgp * 4 + y;
        if (jj < MB) epi(ii, jj, z, acc[0][y], acc[1][y], acc[2][y], acc[3][y]);
    }
}

template <class TA, class TB, class Epi>
inline void gemm_simt(const TA* A, int lda, long long sA, const TB* B, int ldb, long long sB, int MA,
                      int MB, int K, int batch, const Epi& epi, hipStream_t st) {
    // rows i0..i0+3 past MA reach the epilogue when MA % 4 != 0: it must drop them
    if (MA <= 0 || MB <= 0 || K <= 0 || batch <= 0) throw ArgError(-1, "gemm_simt: unsupported shape");
    dim3 grid((MA + 63) / 64, (MB + 63) / 64, batch);
    hipLaunchKernelGGL((gemm_simt_kernel<TA, TB, Epi>), grid, dim3(256), 0, st, A, lda, sA, B, ldb, sB,
                       MA, MB, K, epi);
}

}  // namespace wmi
