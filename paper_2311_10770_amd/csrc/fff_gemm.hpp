// fff_gemm.hpp -- the direct-to-LDS product loop of the matrix-core kernels
// of fff_gemm.hip: the accumulators of each wave of a WGM x WGN-wave workgroup
// = rows [m0, m0 + BM) of A times rows [n0, n0 + BN) of B, both K-contiguous.
#pragma once

#include "fff_device.hpp"

#include <hip/hip_runtime.h>

#include <cstdint>

namespace fff {

// Direct-to-LDS staging: global_load_lds_dwordx4 writes each lane's 16 bytes straight into LDS,
// at the wave's base address (m0) plus 16 x lane, with no registers in between, so S stages can be
// in flight at once (S - 1 steps ahead of the one being multiplied).  A step holds 128 bytes of
// every row (64 bf16 or 32 fp32 elements), rows unpadded; the eight 16-byte vectors of row r are
// stored in the order c ^ swz(r), so that the sixteen rows an MFMA fragment read touches fall on
// distinct banks.  Rows must be 16-byte aligned; a partial last step goes through registers.
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
// The key for 32 x 32 x 16 fragments: a pass then serves eight consecutive rows, each reading the
// adjacent vectors 2k and 2k + 1 (lane halves), so the keys of the rows of one parity must differ
// in bits 1-2; (r & 7) ^ (r >> 3) does that and keeps eight rows apart on a 32-bank array too.
__device__ __forceinline__ int swz32(int r16) { return (r16 & 7) ^ ((r16 >> 3) & 1); }
template <bool M32>
__device__ __forceinline__ int swz_key(int r16) { return M32 ? swz32(r16) : swz(r16); }

typedef float tile_v16f __attribute__((ext_vector_type(16)));  // a 32x32 MFMA result per lane

// Accumulators of one wave: TM x TN tiles of 16 x 16, or (M32) TM/2 x TN/2 tiles of 32 x 32.
template <int TM, int TN, bool M32> struct WaveAcc { tile_v4f t[TM][TN]; };
template <int TM, int TN> struct WaveAcc<TM, TN, true> { tile_v16f t[TM / 2][TN / 2]; };

// The compiler is not told that this load writes LDS (it would otherwise wait for every
// outstanding load before each LDS read): completion is awaited by wait_vmem and a barrier.
// m0 is written nowhere else in these kernels (their assembly writes it only in these sequences),
// so its clobber (which the compiler warns about, m0 being reserved) is safe.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_dma16(const void* g, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(g) : "memory", "m0");
}
#pragma clang diagnostic pop

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

// XCD-aware tile order: workgroup h runs on XCD h % 8, so XCD x takes a contiguous range of the
// tiles (numbered with the fastest index last): neighbouring tiles run together on one XCD and
// share its L2.
__device__ __forceinline__ int64_t xcd_tile(int64_t h, int64_t tiles) {
    const int64_t x = h % 8, per = tiles / 8, rem = tiles % 8;
    return x * per + (x < rem ? x : rem) + h / 8;
}

// acc = A[m0 .. m0 + BM) B[n0 .. n0 + BN)^T over K (a multiple of 8 bf16 or 4 fp32 elements) for this
// wave's 16 TM x 16 TN block (wave w: rows 16 TM (w / WGN) on, columns 16 TN (w % WGN) on), as
// 16 x 16 MFMA tiles or (M32, bf16) 32 x 32 x 16 tiles, which issue at twice the rate per flop on
// gfx950; rows past M and N read row M-1 and N-1.  gsm: G::LDS bytes of dynamic LDS; other waves
// may still read it on return (a barrier precedes any reuse).
template <bool BF, int TM, int TN, int WGM, int WGN, int S, bool M32>
__device__ __forceinline__ void dma_product(const void* __restrict__ A, const void* __restrict__ B, int64_t M,
                                            int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t m0, int64_t n0,
                                            unsigned char* gsm, WaveAcc<TM, TN, M32>& acc) {
    static_assert(!M32 || (BF && TM % 2 == 0 && TN % 2 == 0), "32 x 32 tiles: bf16, whole tiles");
    using G = DmaCfg<TM, TN, WGM, WGN, S>;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WGN, wn = wave % WGN;
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
        ga[i] = static_cast<const char*>(A) + m * lda * esz + (((lane & 7) ^ swz_key<M32>(r & 15)) * 16);
    }
#pragma unroll
    for (int i = 0; i < G::LB; ++i) {
        const int r = (wave * G::LB + i) * 8 + (lane >> 3);
        const int64_t n = n0 + r < N ? n0 + r : N - 1;
        gb[i] = static_cast<const char*>(B) + n * ldb * esz + (((lane & 7) ^ swz_key<M32>(r & 15)) * 16);
    }
    auto issue = [&](int64_t step) {
        const uint32_t st = lds0 + uint32_t(step % S) * G::STAGE;
        const int64_t kb = step * G::ROW;
#pragma unroll
        for (int i = 0; i < G::LA; ++i) lds_dma16(ga[i] + kb, st + (wave * G::LA + i) * 1024);
#pragma unroll
        for (int i = 0; i < G::LB; ++i) lds_dma16(gb[i] + kb, st + G::BM * G::ROW + (wave * G::LB + i) * 1024);
    };

    if constexpr (M32) {
#pragma unroll
        for (int i = 0; i < TM / 2; ++i)
#pragma unroll
            for (int j = 0; j < TN / 2; ++j)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc.t[i][j][e] = 0.f;
    } else {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc.t[i][j] = tile_v4f{0.f, 0.f, 0.f, 0.f};
    }

    const int r16 = lane & 15, q = lane >> 4;
    const int sw = swz(r16);
    const int64_t steps = K / (BF ? 64 : 32);
#pragma unroll
    for (int s = 0; s < S - 1; ++s)
        if (s < steps) issue(s);
    // the MFMAs of one staged step
    auto compute = [&](const unsigned char* st) {
        if constexpr (M32) {
            // lane l reads row l % 32 of each 32-row tile, vector 2 kk + l / 32 (K 16 kk + 8 (l / 32) on)
            const int r32 = lane & 31, hv = lane >> 5, sw32 = swz32(r32 & 15);
            const unsigned char* sa = st + (wm * 16 * TM + r32) * G::ROW;
            const unsigned char* sb = st + G::BM * G::ROW + (wn * 16 * TN + r32) * G::ROW;
            // fragments of K slice kk + 1 are read while slice kk's MFMAs run (two register sets)
            uint4 fa[2][TM / 2], fb[2][TN / 2];
            auto read = [&](int kk, int buf) {
                const int off = ((2 * kk + hv) ^ sw32) * 16;
#pragma unroll
                for (int j = 0; j < TN / 2; ++j)
                    fb[buf][j] = *reinterpret_cast<const uint4*>(sb + j * 32 * G::ROW + off);
#pragma unroll
                for (int i = 0; i < TM / 2; ++i)
                    fa[buf][i] = *reinterpret_cast<const uint4*>(sa + i * 32 * G::ROW + off);
            };
            read(0, 0);
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                if (kk + 1 < 4) read(kk + 1, (kk + 1) & 1);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int i = 0; i < TM / 2; ++i)
#pragma unroll
                    for (int j = 0; j < TN / 2; ++j)
                        acc.t[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            __builtin_bit_cast(bf16x8_t, fa[kk & 1][i]), __builtin_bit_cast(bf16x8_t, fb[kk & 1][j]),
                            acc.t[i][j], 0, 0, 0);
            }
        } else {
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
                            acc.t[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, fa[kk][i]),
                                                                                __builtin_bit_cast(bf16x8_t, fb[kk][j]),
                                                                                acc.t[i][j], 0, 0, 0);
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
                                acc.t[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                    fword(a4, t), fword(__builtin_bit_cast(float4, fb[kk][j]), t), acc.t[i][j], 0, 0, 0);
                    }
                }
            }
        }
    };
    // one loop over every step, so the MFMAs have one call site; the partial last step (K not a
    // whole number of steps) is loaded through registers with zeros past K, stored where the DMA
    // would have put it (every earlier reader of its stage passed the last barrier)
    const int64_t total = steps + (K % (BF ? 64 : 32) != 0 ? 1 : 0);
    for (int64_t s = 0; s < total; ++s) {
        unsigned char* st = gsm + size_t(s % S) * G::STAGE;
        if (s < steps) {
            const int64_t left = steps - 1 - s;
            wait_steps<S - 2, G::LPS>(int(left < S - 2 ? left : S - 2));
            __syncthreads();  // step s is in LDS for every wave; every wave is done with step s - 1
            if (s + S - 1 < steps) issue(s + S - 1);
        } else {
            const int64_t kb = s * G::ROW, k0 = s * (BF ? 64 : 32);
#pragma unroll
            for (int i = 0; i < G::LA; ++i) {
                const int r = (wave * G::LA + i) * 8 + (lane >> 3);
                const bool in = k0 + (((lane & 7) ^ swz_key<M32>(r & 15)) * (BF ? 8 : 4)) < K;
                const uint4 v = in ? *reinterpret_cast<const uint4*>(ga[i] + kb) : make_uint4(0, 0, 0, 0);
                *reinterpret_cast<uint4*>(st + (wave * G::LA + i) * 1024 + lane * 16) = v;
            }
#pragma unroll
            for (int i = 0; i < G::LB; ++i) {
                const int r = (wave * G::LB + i) * 8 + (lane >> 3);
                const bool in = k0 + (((lane & 7) ^ swz_key<M32>(r & 15)) * (BF ? 8 : 4)) < K;
                const uint4 v = in ? *reinterpret_cast<const uint4*>(gb[i] + kb) : make_uint4(0, 0, 0, 0);
                *reinterpret_cast<uint4*>(st + G::BM * G::ROW + (wave * G::LB + i) * 1024 + lane * 16) = v;
            }
            __syncthreads();
        }
        compute(st);
    }
}

}  // namespace fff
