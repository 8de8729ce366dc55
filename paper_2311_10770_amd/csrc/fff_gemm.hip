// fff_gemm.hip -- the dense products of MASKED mode on the matrix cores:
//   C[M, N] = A[M, K] B[N, K]^T   (both operands K-contiguous, "NT"),
// bf16 inputs on v_mfma_f32_16x16x32_bf16 or fp32 inputs on
// v_mfma_f32_16x16x4_f32, fp32 accumulation, with the result stored as fp32
// (the logits), or added to a source row and stored as bf16 or fp32 (the
// layer's output).  K is consumed in steps of 128 bytes per row (64 bf16 or
// 32 fp32 elements).  The main kernel stages each step's rows of A and B into
// LDS with global_load_lds_dwordx4 (no registers in between, one step in
// flight while the previous one is multiplied), in an XOR-swizzled layout that
// keeps the fragment reads free of bank conflicts; a workgroup of four waves
// computes a 256 x 256 (128 x 128 per wave), 256 x 192 or 128 x 128 tile, and
// consecutive tiles of one row block of A run on one XCD.  Where K is not a
// whole number of steps a register-staged kernel with a padded LDS layout
// masks the tail.  Every 16x16 MFMA returns D[4(l/16)+r][l%16] to lane l,
// register r; its bf16 operands are A[l%16][8(l/16) .. +7] and
// B[8(l/16) .. +7][l%16], its fp32 operands A[l%16][q] and B[q][l%16] for the
// lane's K slot q = l/16.  Rows past M and N read the last row (clamped
// addresses) and are never stored.
#include "fff_device.hpp"
#include "fff_internal.hpp"

#include <hip/hip_runtime.h>

#include <cstdint>

namespace fff {

namespace {

// Register-staged kernel (K not a whole number of steps).  A wave computes TM x TN MFMA tiles of
// 16 x 16 (its accumulators), a workgroup WGM x WGN waves; rows padded by 16 bytes in LDS.
template <bool BF, int TM, int TN, int WGM, int WGN>
struct GemmCfg {
    static constexpr int BM = 16 * TM * WGM, BN = 16 * TN * WGN;
    static constexpr int THREADS = 64 * WGM * WGN;
    static constexpr int BK = BF ? 64 : 32;         // K elements per step
    static constexpr int EV = BF ? 8 : 4;           // elements per 16-byte vector
    static constexpr int VPR = BK / EV;             // 16-byte vectors per row of a step (8)
    static constexpr int LDS_ROW = BK * (BF ? 2 : 4) + 16;  // bytes, padded: rows start on different banks
    static constexpr int LDS_A = BM * LDS_ROW, LDS_B = BN * LDS_ROW;  // bytes per buffer
    static constexpr int LOADS_A = BM * VPR / THREADS, LOADS_B = BN * VPR / THREADS;
    static_assert(BM * VPR % THREADS == 0 && BN * VPR % THREADS == 0, "whole vectors per thread");
};

// Output forms: fp32 C; or C plus a source row (none / fp32 / bf16), stored as bf16 or fp32.
enum { GOUT_F32 = 0, GOUT_SRC_NONE = 1, GOUT_SRC_F32 = 2, GOUT_SRC_BF16 = 3 };

template <int OUT, bool DBF>
__device__ __forceinline__ void gemm_store(void* C, const void* src, int64_t ldc, int64_t m, int64_t n, float v) {
    const int64_t e = m * ldc + n;
    if constexpr (OUT == GOUT_SRC_F32) v += static_cast<const float*>(src)[e];
    if constexpr (OUT == GOUT_SRC_BF16) v += bf16_to_f32(static_cast<const uint16_t*>(src)[e]);
    if constexpr (OUT == GOUT_F32 || !DBF) static_cast<float*>(C)[e] = v;
    else static_cast<uint16_t*>(C)[e] = f32_to_bf16(v);
}

template <bool BF, int TM, int TN, int WGM, int WGN, int OUT, bool DBF>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_nt_kernel(const void* __restrict__ A,
                                                                 const void* __restrict__ B, void* C,
                                                                 const void* src, int64_t M, int64_t N, int64_t K,
                                                                 int64_t lda, int64_t ldb, int64_t ldc) {
    using G = GemmCfg<BF, TM, TN, WGM, WGN>;
    extern __shared__ __align__(16) unsigned char gsm[];  // [2 buffers][A rows, B rows][LDS_ROW]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    const int64_t m0 = int64_t(blockIdx.y) * G::BM, n0 = int64_t(blockIdx.x) * G::BN;
    const int esz = BF ? 2 : 4;

    // global -> registers: vector v = tid + THREADS i of the step's tile, row v / VPR, vector v % VPR;
    // loaded while the previous step is computed
    uint4 ra[G::LOADS_A], rb[G::LOADS_B];
    auto load_step = [&](int64_t k0) {
#pragma unroll
        for (int i = 0; i < G::LOADS_A; ++i) {
            const int v = tid + G::THREADS * i;
            const int row = v / G::VPR, kv = v % G::VPR;
            const int64_t k = k0 + int64_t(kv) * G::EV;
            const bool kin = k < K;
            const int64_t ma = m0 + row < M ? m0 + row : M - 1;
            const uint4 a = *reinterpret_cast<const uint4*>(static_cast<const char*>(A) + (ma * lda + (kin ? k : 0)) * esz);
            ra[i] = kin ? a : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < G::LOADS_B; ++i) {
            const int v = tid + G::THREADS * i;
            const int row = v / G::VPR, kv = v % G::VPR;
            const int64_t k = k0 + int64_t(kv) * G::EV;
            const bool kin = k < K;
            const int64_t nb = n0 + row < N ? n0 + row : N - 1;
            const uint4 b = *reinterpret_cast<const uint4*>(static_cast<const char*>(B) + (nb * ldb + (kin ? k : 0)) * esz);
            rb[i] = kin ? b : make_uint4(0, 0, 0, 0);
        }
    };
    auto store_step = [&](int buf) {
        unsigned char* sa = gsm + size_t(buf) * (G::LDS_A + G::LDS_B);
        unsigned char* sb = sa + G::LDS_A;
#pragma unroll
        for (int i = 0; i < G::LOADS_A; ++i) {
            const int v = tid + G::THREADS * i;
            *reinterpret_cast<uint4*>(sa + (v / G::VPR) * G::LDS_ROW + (v % G::VPR) * 16) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < G::LOADS_B; ++i) {
            const int v = tid + G::THREADS * i;
            *reinterpret_cast<uint4*>(sb + (v / G::VPR) * G::LDS_ROW + (v % G::VPR) * 16) = rb[i];
        }
    };

    tile_v4f acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = tile_v4f{0.f, 0.f, 0.f, 0.f};

    const int64_t steps = (K + G::BK - 1) / G::BK;
    load_step(0);
    store_step(0);
    __syncthreads();
    const int r16 = lane & 15, q = lane >> 4;
    for (int64_t s = 0; s < steps; ++s) {
        const int buf = int(s & 1);
        if (s + 1 < steps) load_step((s + 1) * G::BK);
        const unsigned char* sa = gsm + size_t(buf) * (G::LDS_A + G::LDS_B) + (wm * 16 * TM + r16) * G::LDS_ROW;
        const unsigned char* sb =
            gsm + size_t(buf) * (G::LDS_A + G::LDS_B) + G::LDS_A + (wn * 16 * TN + r16) * G::LDS_ROW;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {  // bf16: two K = 32 MFMA steps; fp32: two blocks of 16
            if constexpr (BF) {
                uint4 fb[TN];
#pragma unroll
                for (int j = 0; j < TN; ++j) fb[j] = *reinterpret_cast<const uint4*>(sb + j * 16 * G::LDS_ROW + kk * 64 + q * 16);
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    const uint4 fa = *reinterpret_cast<const uint4*>(sa + i * 16 * G::LDS_ROW + kk * 64 + q * 16);
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            __builtin_bit_cast(bf16x8_t, fa), __builtin_bit_cast(bf16x8_t, fb[j]), acc[i][j], 0, 0, 0);
                }
            } else {
                // lane group q holds K slots 4q .. 4q+3 of the 16-wide block; MFMA t of the block
                // takes slot 4q + t (a permutation of the block's K indices over the four MFMAs)
                float4 fb[TN];
#pragma unroll
                for (int j = 0; j < TN; ++j) fb[j] = *reinterpret_cast<const float4*>(sb + j * 16 * G::LDS_ROW + kk * 64 + q * 16);
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    const float4 fa = *reinterpret_cast<const float4*>(sa + i * 16 * G::LDS_ROW + kk * 64 + q * 16);
#pragma unroll
                    for (int t = 0; t < 4; ++t)
#pragma unroll
                        for (int j = 0; j < TN; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fword(fa, t), fword(fb[j], t), acc[i][j],
                                                                              0, 0, 0);
                }
            }
        }
        if (s + 1 < steps) store_step(buf ^ 1);
        __syncthreads();
    }

#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int64_t n = n0 + wn * 16 * TN + j * 16 + r16;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t m = m0 + wm * 16 * TM + i * 16 + 4 * q + r;
                if (m < M && n < N) gemm_store<OUT, DBF>(C, src, ldc, m, n, acc[i][j][r]);
            }
        }
}

// Direct-to-LDS staging: global_load_lds_dwordx4 writes each lane's 16 bytes straight into LDS,
// at the wave's base address (m0) plus 16 x lane, with no registers in between, so S stages can be
// in flight at once (S - 1 steps ahead of the one being multiplied).  A step holds 128 bytes of
// every row (64 bf16 or 32 fp32 elements), rows unpadded; the eight 16-byte vectors of row r are
// stored in the order c ^ swz(r), so that the sixteen rows an MFMA fragment read touches fall on
// distinct banks.  Requires K to be a whole number of steps and 16-byte aligned rows.
template <int TM, int TN, int WGM, int WGN, int S>
struct DmaCfg {
    static constexpr int BM = 16 * TM * WGM, BN = 16 * TN * WGN;
    static constexpr int WAVES = WGM * WGN, THREADS = 64 * WAVES;
    static constexpr int ROW = 128;                          // bytes of a row per step
    static constexpr int STAGE = (BM + BN) * ROW;            // bytes per stage: A rows, then B rows
    static constexpr int LA = BM / 8 / WAVES, LB = BN / 8 / WAVES;  // 8-row wave loads per step
    static constexpr int LPS = LA + LB;                      // DMA instructions per wave and step
    static constexpr size_t LDS = size_t(S) * STAGE;
    static_assert((BM / 8) % WAVES == 0 && (BN / 8) % WAVES == 0, "whole 8-row loads per wave");
    static_assert(S >= 2 && LPS * (S - 2) <= 63, "vmcnt holds 6 bits");
};

// The XOR key of row r16 (0..15).  A b128 read is served in four passes of sixteen lanes, eight
// from each half of the wave (lanes 8t..8t+7 and 32+8t..32+8t+7, which read vectors c and c ^ 2 of
// the same eight rows): the keys of rows of one parity take distinct values with bit 1 equal within
// each group of eight rows, so the sixteen lanes of a pass cover the 64 banks once.  The same keys
// also keep eight consecutive rows on distinct 16-byte bank groups of a 32-bank array.
__device__ __forceinline__ int swz(int r16) {
    const int h = (r16 >> 1) & 3;
    return (h & 1) | ((h & 2) << 1) | ((((r16 & 1) ^ (r16 >> 3)) & 1) << 1);
}

// The compiler is not told that this load writes LDS (it would otherwise wait for every
// outstanding load before each LDS read): completion is awaited by wait_vmem and a barrier.
__device__ __forceinline__ void lds_dma16(const void* g, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(g) : "memory", "m0");
}

// s_waitcnt vmcnt(N) with lgkmcnt and expcnt left alone (gfx9 encoding: vmcnt in bits 3:0 and 15:14).
template <int N>
__device__ __forceinline__ void wait_vmem() {
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}
// Wait until at most `ahead` steps of LPS loads each are outstanding.
template <int MAXA, int LPS>
__device__ __forceinline__ void wait_steps(int ahead) {
    if constexpr (MAXA == 0) {
        wait_vmem<0>();
    } else {
        if (ahead >= MAXA) wait_vmem<MAXA * LPS>();
        else wait_steps<MAXA - 1, LPS>(ahead);
    }
}

template <bool BF, int TM, int TN, int WGM, int WGN, int S, int OUT, bool DBF>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_nt_dma_kernel(const void* __restrict__ A,
                                                                     const void* __restrict__ B, void* C,
                                                                     const void* src, int64_t M, int64_t N,
                                                                     int64_t K, int64_t lda, int64_t ldb,
                                                                     int64_t ldc) {
    using G = DmaCfg<TM, TN, WGM, WGN, S>;
    extern __shared__ __align__(16) unsigned char gsm[];  // [S stages][A rows, B rows][128 bytes]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WGN, wn = wave % WGN;
    // XCD-aware tile order: workgroup h runs on XCD h % 8, so XCD x takes a contiguous range of
    // tiles, N fastest: the tiles of one row block of A run together on one XCD and share its L2
    const int64_t tiles_n = (N + G::BN - 1) / G::BN, tiles = tiles_n * ((M + G::BM - 1) / G::BM);
    const int64_t h = blockIdx.x, x = h % 8, per = tiles / 8, rem = tiles % 8;
    const int64_t t = x * per + (x < rem ? x : rem) + h / 8;
    const int64_t m0 = (t / tiles_n) * G::BM, n0 = (t % tiles_n) * G::BN;
    const int esz = BF ? 2 : 4;
    const uint32_t lds0 = uint32_t(uintptr_t((__attribute__((address_space(3))) unsigned char*)gsm));

    // this lane's source of each wave load: tile row r = 8 (load) + lane / 8, physical vector
    // lane % 8 holding logical vector (lane % 8) ^ swz(r); rows past M and N read row M-1, N-1
    const char* ga[G::LA];
    const char* gb[G::LB];
#pragma unroll
    for (int i = 0; i < G::LA; ++i) {
        const int r = (wave * G::LA + i) * 8 + (lane >> 3);
        const int64_t m = m0 + r < M ? m0 + r : M - 1;
        ga[i] = static_cast<const char*>(A) + m * lda * esz + (((lane & 7) ^ swz(r & 15)) * 16);
    }
#pragma unroll
    for (int i = 0; i < G::LB; ++i) {
        const int r = (wave * G::LB + i) * 8 + (lane >> 3);
        const int64_t n = n0 + r < N ? n0 + r : N - 1;
        gb[i] = static_cast<const char*>(B) + n * ldb * esz + (((lane & 7) ^ swz(r & 15)) * 16);
    }
    auto issue = [&](int64_t step) {
        const uint32_t st = lds0 + uint32_t(step % S) * G::STAGE;
        const int64_t kb = step * G::ROW;
#pragma unroll
        for (int i = 0; i < G::LA; ++i) lds_dma16(ga[i] + kb, st + (wave * G::LA + i) * 1024);
#pragma unroll
        for (int i = 0; i < G::LB; ++i) lds_dma16(gb[i] + kb, st + G::BM * G::ROW + (wave * G::LB + i) * 1024);
    };

    tile_v4f acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = tile_v4f{0.f, 0.f, 0.f, 0.f};

    const int r16 = lane & 15, q = lane >> 4;
    const int sw = swz(r16);
    const int64_t steps = K / (BF ? 64 : 32);
#pragma unroll
    for (int s = 0; s < S - 1; ++s)
        if (s < steps) issue(s);
    for (int64_t s = 0; s < steps; ++s) {
        const int64_t left = steps - 1 - s;
        wait_steps<S - 2, G::LPS>(int(left < S - 2 ? left : S - 2));
        __syncthreads();  // step s is in LDS for every wave; every wave is done with step s - 1
        if (s + S - 1 < steps) issue(s + S - 1);
        const unsigned char* st = gsm + size_t(s % S) * G::STAGE;
        const unsigned char* sa = st + (wm * 16 * TM + r16) * G::ROW;
        const unsigned char* sb = st + G::BM * G::ROW + (wn * 16 * TN + r16) * G::ROW;
        // all fragments of both K halves are read up front: the second half's reads complete
        // while the first half's MFMAs run (the scheduler may not sink them below)
        uint4 fa[2][TM], fb[2][TN];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const int off = ((kk * 4 + q) ^ sw) * 16;
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[kk][j] = *reinterpret_cast<const uint4*>(sb + j * 16 * G::ROW + off);
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[kk][i] = *reinterpret_cast<const uint4*>(sa + i * 16 * G::ROW + off);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            if constexpr (BF) {
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, fa[kk][i]),
                                                                            __builtin_bit_cast(bf16x8_t, fb[kk][j]),
                                                                            acc[i][j], 0, 0, 0);
            } else {
                // lane group q holds K slots 4q .. 4q+3 of the 16-wide block; MFMA t of the block
                // takes slot 4q + t (a permutation of the block's K indices over the four MFMAs)
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    const float4 a4 = __builtin_bit_cast(float4, fa[kk][i]);
#pragma unroll
                    for (int t = 0; t < 4; ++t)
#pragma unroll
                        for (int j = 0; j < TN; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                fword(a4, t), fword(__builtin_bit_cast(float4, fb[kk][j]), t), acc[i][j], 0, 0, 0);
                }
            }
        }
    }

#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int64_t n = n0 + wn * 16 * TN + j * 16 + r16;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t m = m0 + wm * 16 * TM + i * 16 + 4 * q + r;
                if (m < M && n < N) gemm_store<OUT, DBF>(C, src, ldc, m, n, acc[i][j][r]);
            }
        }
}

template <bool BF, int TM, int TN, int WGM, int WGN, int S, int OUT, bool DBF>
void launch_dma(const void* A, const void* B, void* C, const void* src, int64_t M, int64_t N, int64_t K,
                int64_t lda, int64_t ldb, int64_t ldc, hipStream_t stream) {
    using G = DmaCfg<TM, TN, WGM, WGN, S>;
    const dim3 grid(unsigned(((N + G::BN - 1) / G::BN) * ((M + G::BM - 1) / G::BM)));
    hipLaunchKernelGGL((gemm_nt_dma_kernel<BF, TM, TN, WGM, WGN, S, OUT, DBF>), grid, dim3(G::THREADS), G::LDS, stream,
                       A, B, C, src, M, N, K, lda, ldb, ldc);
}

// Tile choice, from the shapes and the CU count only.  K a whole number of steps: direct-to-LDS
// staging with 256 x 256 tiles (128 x 128 per wave, bf16) or 256 x 192 (128 x 96 per wave), one
// workgroup per CU, whichever leaves fewer tile-rounds of idle CUs (the narrower tile reads ~7% more
// LDS per MFMA; its fp32 form is the only wide one that needs no spills), or 128 x 128 tiles with
// two workgroups per CU for small products.  Otherwise the register-staged kernel, which masks
// the K tail.
template <bool BF, int OUT, bool DBF>
hipError_t launch_gemm(const void* A, const void* B, void* C, const void* src, int64_t M, int64_t N, int64_t K,
                       int64_t lda, int64_t ldb, int64_t ldc, int cu_count, hipStream_t stream) {
    auto cdiv = [](int64_t a, int64_t b) { return (a + b - 1) / b; };
    if (K % (BF ? 64 : 32) == 0) {
        const int64_t slots = cu_count > 0 ? cu_count : 256;
        const int64_t t88 = cdiv(M, 256) * cdiv(N, 256), t86 = cdiv(M, 256) * cdiv(N, 192);
        if (t88 < slots / 4) {
            launch_dma<BF, 4, 4, 2, 2, 2, OUT, DBF>(A, B, C, src, M, N, K, lda, ldb, ldc, stream);
        } else if (BF && double(cdiv(t88, slots)) * 256 * 256 <= double(cdiv(t86, slots)) * 256 * 192 * 1.07) {
            launch_dma<BF, 8, 8, 2, 2, 2, OUT, DBF>(A, B, C, src, M, N, K, lda, ldb, ldc, stream);
        } else {
            launch_dma<BF, 8, 6, 2, 2, 2, OUT, DBF>(A, B, C, src, M, N, K, lda, ldb, ldc, stream);
        }
        return hipGetLastError();
    }
    using Small = GemmCfg<BF, 4, 4, 2, 2>;
    const dim3 grid(unsigned(cdiv(N, Small::BN)), unsigned(cdiv(M, Small::BM)));
    hipLaunchKernelGGL((gemm_nt_kernel<BF, 4, 4, 2, 2, OUT, DBF>), grid, dim3(Small::THREADS),
                       size_t(2) * (Small::LDS_A + Small::LDS_B), stream, A, B, C, src, M, N, K, lda, ldb, ldc);
    return hipGetLastError();
}

}  // namespace

hipError_t gemm_nt(bool bf16, int out, bool dst_bf16, const void* A, const void* B, void* C, const void* src,
                   int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t ldc, int cu_count,
                   hipStream_t stream) {
    if (M == 0 || N == 0) return hipSuccess;
    if (bf16) {
        switch (out) {
            case GEMM_OUT_F32: return launch_gemm<true, GOUT_F32, false>(A, B, C, src, M, N, K, lda, ldb, ldc, cu_count, stream);
            case GEMM_OUT_SRC_NONE:
                return dst_bf16 ? launch_gemm<true, GOUT_SRC_NONE, true>(A, B, C, src, M, N, K, lda, ldb, ldc, cu_count, stream)
                                : launch_gemm<true, GOUT_SRC_NONE, false>(A, B, C, src, M, N, K, lda, ldb, ldc, cu_count, stream);
            case GEMM_OUT_SRC_F32:
                return dst_bf16 ? launch_gemm<true, GOUT_SRC_F32, true>(A, B, C, src, M, N, K, lda, ldb, ldc, cu_count, stream)
                                : launch_gemm<true, GOUT_SRC_F32, false>(A, B, C, src, M, N, K, lda, ldb, ldc, cu_count, stream);
            default:
                return dst_bf16 ? launch_gemm<true, GOUT_SRC_BF16, true>(A, B, C, src, M, N, K, lda, ldb, ldc, cu_count, stream)
                                : launch_gemm<true, GOUT_SRC_BF16, false>(A, B, C, src, M, N, K, lda, ldb, ldc, cu_count, stream);
        }
    }
    switch (out) {
        case GEMM_OUT_F32: return launch_gemm<false, GOUT_F32, false>(A, B, C, src, M, N, K, lda, ldb, ldc, cu_count, stream);
        case GEMM_OUT_SRC_NONE: return launch_gemm<false, GOUT_SRC_NONE, false>(A, B, C, src, M, N, K, lda, ldb, ldc, cu_count, stream);
        default: return launch_gemm<false, GOUT_SRC_F32, false>(A, B, C, src, M, N, K, lda, ldb, ldc, cu_count, stream);
    }
}

}  // namespace fff
