// GEMM kernels: C[i][j] = sum_k A[i][k] * B[j][k] with A and B both stored
// row-major with K contiguous ("A times B transposed"), optionally batched.
//
// The result never goes to memory as a plain matrix: an epilogue functor
// receives each lane's output as four consecutive i for one j,
//     p = epi.pre(i0, j, z); epi(i0, j, z, v0, v1, v2, v3, p)
// (rows i0..i0+3 of batch z, column j; pre() issues the loads first),
// and stores it in whatever layout the consumer wants (bias, GELU, residual
// add, per-head or transposed cache layouts). Call sites pick which operand
// is A so that the four consecutive i are the contiguous output dimension.
//
// gemm_bf16: bf16 inputs, v_mfma_f32_16x16x32_bf16 with fp32 accumulation,
//   K tiles of 32 streamed into an LDS ring with direct global->LDS loads
//   (no staging registers), 16-byte chunks XOR-swizzled against bank
//   conflicts. Two tilings: 256x256 tiles, 8 waves of 128x64, a 4-stage ring
//   (one workgroup per CU), for K > 1024; 256x128 tiles, 8 waves of 64x64, a
//   3-stage ring (two workgroups per CU), for K <= 1024. Tiles are mapped to
//   the XCDs so that workgroups sharing an L2 share operand tiles.
//   Requires K % 64 == 0, MA % 4 == 0, 16-byte aligned rows (lda, ldb % 8 == 0).
// gemm_simt: fp32 (or bf16 storage) SIMT kernel for the fp32 model: 64x64x16
//   tile, 4x4 outputs per thread, any K, any lda.
#pragma once

#include <atomic>

#include "common.h"

namespace wmi {

typedef __bf16 mfma_bf16x8 __attribute__((ext_vector_type(8)));
typedef float mfma_f32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ bf16 MFMA

namespace gb {
constexpr int BM = 256;   // A rows per workgroup
constexpr int BN = 256;   // B rows per workgroup
constexpr int BK = 32;    // K per LDS stage
constexpr int NS = 4;     // LDS stages
constexpr int THREADS = 512;  // 8 waves
constexpr int TILE_BYTES = BM * BK * 2;        // one operand tile of a stage (16 KiB)
constexpr int STAGE_BYTES = 2 * TILE_BYTES;    // A and B tiles (32 KiB)
constexpr int LDS_BYTES = NS * STAGE_BYTES;    // 128 KiB
}  // namespace gb

// Byte offset of 16-byte chunk c (0..3) of row r in a [rows][32] bf16 LDS tile:
// position c ^ ((r >> 1) & 3), so the 8 rows read together by a ds_read_b128
// group hit distinct banks.
__device__ inline int swz32(int r, int c) { return r * 64 + ((c ^ ((r >> 1) & 3)) << 4); }

// s_waitcnt immediate that waits until at most n vector-memory ops are outstanding.
#define WMI_VMCNT(n) ((((n) & 0xF)) | (((n) >> 4) << 14) | (0x7 << 4) | (0xF << 8))

// Byte offset of 16-byte chunk c (0..7) of row r inside a [rows][64] bf16 LDS tile.
__device__ inline int swz(int r, int c) { return r * 128 + ((c ^ (r & 7)) << 4); }

// Tile of workgroup `bid` among tilesA x tilesB tiles, arranged for the L2
// of each XCD: workgroups are handed to the 8 XCDs in turn (bid mod 8), so
// XCD x gets a contiguous run of tiles, and runs are ordered in groups of
// GA A-tiles (A-tile fastest): the ~32 workgroups an XCD holds at a time
// then cover about 4 A-tiles x 8 B-tiles, and each tile's K-slices are
// fetched into that XCD's L2 once for several workgroups.
__device__ inline void xcd_tile(int bid, int tilesA, int tilesB, int& ta, int& tb) {
    constexpr int GA = 4;
    const int T = tilesA * tilesB, per = T >> 3, rem = T & 7;
    const int x = bid & 7, j = bid >> 3;
    const int v = x * per + min(x, rem) + j;
    const int g = v / (GA * tilesB), ga = min(GA, tilesA - g * GA);
    const int w = v - g * GA * tilesB;
    tb = w / ga;
    ta = g * GA + (w - tb * ga);
}

// Epilogue of a wave's NI x 4 blocks of 16 x 16 results: lane (fr, fc) of
// block (i, j) holds rows ia + 16 i + 4 fc .. + 3 of column jb + 16 j + fr.
// For each column block, all of its loads (pre) are issued before its
// stores. A tile wholly inside the output (full, the common case) skips the
// per-element bounds tests, each a branch and an exec-mask update.
template <int NI, class Epi>
__device__ __forceinline__ void tile_epilogue(const Epi& epi, const mfma_f32x4 (&acc)[NI][4], int ia, int jb, int fr,
                                              int fc, int z, int MA, int MB, bool full) {
    if (full) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int jj = jb + j * 16 + fr;
            EpiPre pre[NI];
#pragma unroll
            for (int i = 0; i < NI; ++i) pre[i] = epi.pre(ia + i * 16 + fc * 4, jj, z);
#pragma unroll
            for (int i = 0; i < NI; ++i)
                epi(ia + i * 16 + fc * 4, jj, z, acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3], pre[i]);
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int jj = jb + j * 16 + fr;
        const bool jok = jj < MB;
        EpiPre pre[NI];
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int ii = ia + i * 16 + fc * 4;
            if (jok && ii < MA) pre[i] = epi.pre(ii, jj, z);
        }
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int ii = ia + i * 16 + fc * 4;
            if (jok && ii < MA) epi(ii, jj, z, acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3], pre[i]);
        }
    }
}

// C = A B^T for A [MA][K], B [MB][K] (bf16, row-major, batched over z):
// a 256 x 256 workgroup tile, 8 waves (2 per SIMD) of 128 x 64 each on
// 16x16x32 MFMAs, so one wave's MFMAs run while the other waits on its LDS
// reads or the stage barrier. Operands go global -> LDS directly through a
// 4-stage ring of 32-wide K tiles.
template <class Epi>
__global__ __launch_bounds__(512, 1) void gemm_bf16_kernel(
    const bf16* __restrict__ A, int lda, long long sA, const bf16* __restrict__ B, int ldb,
    long long sB, int MA, int MB, int K, int tilesA, Epi epi) {
    extern __shared__ __align__(16) unsigned char lds[];
    const int z = blockIdx.z;
    A += (long long)z * sA;
    B += (long long)z * sB;
    int ta, tb;
    xcd_tile(blockIdx.x, tilesA, (int)(gridDim.x / tilesA), ta, tb);
    const int a0 = ta * gb::BM, b0 = tb * gb::BN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wa = (wave & 1) * 128, wb = (wave >> 1) * 64;
    const int fr = lane & 15, fc = lane >> 4;

    // Direct loads: wave w fills rows 32 w .. 32 w + 31 of both operand tiles
    // with 2 + 2 instructions of 16 rows x 64 B; lane i loads row 16 s + i / 4
    // and the logical chunk stored at its physical position i % 4.
    const int dr = lane >> 2;
    const int dc = (lane & 3) ^ ((dr >> 1) & 3);
    const bf16* ga[2];
    const bf16* gp[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int r = wave * 32 + s * 16 + dr;
        ga[s] = A + (long long)min(a0 + r, MA - 1) * lda + dc * 8;
        gp[s] = B + (long long)min(b0 + r, MB - 1) * ldb + dc * 8;
    }
    const int ldsw = wave * 32 * 64;

    mfma_f32x4 acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};

#define WMI_ISSUE8(KT)                                                                                 \
    do {                                                                                               \
        const int st_ = ((KT) % gb::NS) * gb::STAGE_BYTES + ldsw;                                      \
        const int k_ = (KT) * gb::BK;                                                                  \
        _Pragma("unroll") for (int s = 0; s < 2; ++s)                                                 \
            __builtin_amdgcn_global_load_lds(ga[s] + k_, lds + st_ + s * 1024, 16, 0, 0);              \
        _Pragma("unroll") for (int s = 0; s < 2; ++s)                                                 \
            __builtin_amdgcn_global_load_lds(gp[s] + k_, lds + st_ + gb::TILE_BYTES + s * 1024, 16, 0, 0); \
    } while (0)

    const int nk = K / gb::BK;
    WMI_ISSUE8(0);
    if (nk > 1) WMI_ISSUE8(1);
    if (nk > 2) WMI_ISSUE8(2);
    for (int kt = 0; kt < nk; ++kt) {
        // tile kt has landed once only the 4-load groups of later tiles are pending
        const int later = min(nk - 1 - kt, gb::NS - 2);
        if (later >= 2) __builtin_amdgcn_s_waitcnt(WMI_VMCNT(8));
        else if (later == 1) __builtin_amdgcn_s_waitcnt(WMI_VMCNT(4));
        else __builtin_amdgcn_s_waitcnt(WMI_VMCNT(0));
        // every wave's part of tile kt is in LDS, and every wave is done with tile kt - 1
        __builtin_amdgcn_s_barrier();
        if (kt + gb::NS - 1 < nk) WMI_ISSUE8(kt + gb::NS - 1);
        const unsigned char* stage = lds + (kt % gb::NS) * gb::STAGE_BYTES;
        mfma_bf16x8 fa[8], fb[4];
#pragma unroll
        for (int i = 0; i < 8; ++i) fa[i] = *reinterpret_cast<const mfma_bf16x8*>(stage + swz32(wa + i * 16 + fr, fc));
#pragma unroll
        for (int j = 0; j < 4; ++j)
            fb[j] = *reinterpret_cast<const mfma_bf16x8*>(stage + gb::TILE_BYTES + swz32(wb + j * 16 + fr, fc));
        __builtin_amdgcn_sched_barrier(0);  // every fragment read is issued ahead of the MFMAs
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 8; ++i)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
#undef WMI_ISSUE8
    tile_epilogue(epi, acc, a0 + wa, b0 + wb, fr, fc, z, MA, MB, a0 + gb::BM <= MA && b0 + gb::BN <= MB);
}

// Two-workgroups-per-CU variant: a 256 x 128 tile, 8 waves of 64 x 64
// (64 accumulator registers), a 3-stage ring of 24 KiB stages (72 KiB), so
// two workgroups share a CU and one's prologue and epilogue overlap the
// other's main loop.
namespace gh {
constexpr int BM = 256, BN = 128, BK = 32, NS = 3, THREADS = 512;
constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;  // 16 KiB, 8 KiB
constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
constexpr int LDS_BYTES = NS * STAGE_BYTES;  // 72 KiB
}  // namespace gh

template <class Epi>
__global__ __launch_bounds__(512, 2) void gemm_bf16_h_kernel(
    const bf16* __restrict__ A, int lda, long long sA, const bf16* __restrict__ B, int ldb,
    long long sB, int MA, int MB, int K, int tilesA, Epi epi) {
    extern __shared__ __align__(16) unsigned char lds[];
    const int z = blockIdx.z;
    A += (long long)z * sA;
    B += (long long)z * sB;
    int ta, tb;
    xcd_tile(blockIdx.x, tilesA, (int)(gridDim.x / tilesA), ta, tb);
    const int a0 = ta * gh::BM, b0 = tb * gh::BN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wa = (wave & 3) * 64, wb = (wave >> 2) * 64;
    const int fr = lane & 15, fc = lane >> 4;

    // Direct loads: wave w fills A rows 32 w .. 32 w + 31 (2 instructions of
    // 16 rows x 64 B) and B rows 16 w .. 16 w + 15 (1 instruction).
    const int dr = lane >> 2;
    const int dc = (lane & 3) ^ ((dr >> 1) & 3);
    const bf16* ga[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) ga[s] = A + (long long)min(a0 + wave * 32 + s * 16 + dr, MA - 1) * lda + dc * 8;
    const bf16* gp = B + (long long)min(b0 + wave * 16 + dr, MB - 1) * ldb + dc * 8;

    mfma_f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma_f32x4{0.f, 0.f, 0.f, 0.f};

#define WMI_ISSUE3(KT)                                                                                  \
    do {                                                                                                \
        const int st_ = ((KT) % gh::NS) * gh::STAGE_BYTES;                                              \
        const int k_ = (KT) * gh::BK;                                                                   \
        _Pragma("unroll") for (int s = 0; s < 2; ++s)                                                  \
            __builtin_amdgcn_global_load_lds(ga[s] + k_, lds + st_ + wave * 2048 + s * 1024, 16, 0, 0); \
        __builtin_amdgcn_global_load_lds(gp + k_, lds + st_ + gh::A_BYTES + wave * 1024, 16, 0, 0);     \
    } while (0)

    const int nk = K / gh::BK;
    WMI_ISSUE3(0);
    if (nk > 1) WMI_ISSUE3(1);
    for (int kt = 0; kt < nk; ++kt) {
        // tile kt has landed once only the 3-load group of the next tile is pending
        if (kt + 1 < nk) __builtin_amdgcn_s_waitcnt(WMI_VMCNT(3));
        else __builtin_amdgcn_s_waitcnt(WMI_VMCNT(0));
        __builtin_amdgcn_s_barrier();
        if (kt + gh::NS - 1 < nk) WMI_ISSUE3(kt + gh::NS - 1);
        const unsigned char* stage = lds + (kt % gh::NS) * gh::STAGE_BYTES;
        mfma_bf16x8 fa[4], fb[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) fa[i] = *reinterpret_cast<const mfma_bf16x8*>(stage + swz32(wa + i * 16 + fr, fc));
#pragma unroll
        for (int j = 0; j < 4; ++j)
            fb[j] = *reinterpret_cast<const mfma_bf16x8*>(stage + gh::A_BYTES + swz32(wb + j * 16 + fr, fc));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
#undef WMI_ISSUE3
    tile_epilogue(epi, acc, a0 + wa, b0 + wb, fr, fc, z, MA, MB, a0 + gh::BM <= MA && b0 + gh::BN <= MB);
}

// Raises kernel f's dynamic LDS limit to `bytes` on the current device, once
// per device (the attribute is per device; `done` holds one bit per device).
inline void lds_limit(const void* f, int bytes, std::atomic<uint64_t>& done) {
    int dev = 0;
    WMI_HIP(hipGetDevice(&dev));
    const uint64_t bit = 1ull << (dev & 63);
    if (done.load() & bit) return;
    WMI_HIP(hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, bytes));
    done.fetch_or(bit);
}

template <class Epi>
inline void gemm_bf16(const bf16* A, int lda, long long sA, const bf16* B, int ldb, long long sB,
                      int MA, int MB, int K, int batch, const Epi& epi, hipStream_t st) {
    if (K % 64 || MA % 4 || lda % 8 || ldb % 8 || MA <= 0 || MB <= 0 || batch <= 0)
        throw ArgError(-1, "gemm_bf16: unsupported shape");
    const int tilesA = (MA + gb::BM - 1) / gb::BM, tilesB = (MB + gb::BN - 1) / gb::BN;
    // Short reductions (K <= 1024) take the 256 x 128 tiles, two workgroups
    // per CU, whose prologues and epilogues overlap; longer ones the
    // 256 x 256 tiles. WHISPER_GEMM_H=0/1 forces one.
    static const int force = [] {
        const char* g = getenv("WHISPER_GEMM_H");
        return g ? (g[0] == '1' ? 1 : 0) : -1;
    }();
    if (force == 1 || (force < 0 && K <= 1024)) {
        static std::atomic<uint64_t> done_h{0};  // one per epilogue instantiation
        lds_limit(reinterpret_cast<const void*>(&gemm_bf16_h_kernel<Epi>), gh::LDS_BYTES, done_h);
        const int tb2 = (MB + gh::BN - 1) / gh::BN;
        dim3 grid(tilesA * tb2, 1, batch);
        hipLaunchKernelGGL((gemm_bf16_h_kernel<Epi>), grid, dim3(gh::THREADS), gh::LDS_BYTES, st, A, lda, sA, B,
                           ldb, sB, MA, MB, K, tilesA, epi);
        return;
    }
    static std::atomic<uint64_t> done{0};
    lds_limit(reinterpret_cast<const void*>(&gemm_bf16_kernel<Epi>), gb::LDS_BYTES, done);
    dim3 grid(tilesA * tilesB, 1, batch);
    hipLaunchKernelGGL((gemm_bf16_kernel<Epi>), grid, dim3(gb::THREADS), gb::LDS_BYTES, st, A, lda,
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
    EpiPre pre[4];
#pragma unroll
    for (int y = 0; y < 4; ++y) {
        const int jj = b0 + bgp * 4 + y;
        if (jj < MB) pre[y] = epi.pre(ii, jj, z);
    }
#pragma unroll
    for (int y = 0; y < 4; ++y) {
        const int jj = b0 + bgp * 4 + y;
        if (jj < MB) epi(ii, jj, z, acc[0][y], acc[1][y], acc[2][y], acc[3][y], pre[y]);
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
