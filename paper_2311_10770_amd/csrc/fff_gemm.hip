// fff_gemm.hip -- the dense products of MASKED mode on the matrix cores:
//   C[M, N] = A[M, K] B[N, K]^T   (both operands K-contiguous, "NT"),
// bf16 inputs on v_mfma_f32_16x16x32_bf16 or fp32 inputs on
// v_mfma_f32_16x16x4_f32, fp32 accumulation, with the result stored as fp32
// (the logits), or added to a source row and stored as bf16 or fp32 (the
// layer's output).  K is consumed in steps of 128 bytes per row (64 bf16 or
// 32 fp32 elements).  The main kernel stages each step's rows of A and B into
// LDS with global_load_lds_dwordx4 (no registers in between, one step in
// flight while the previous one is multiplied), in an XOR-swizzled layout that
// keeps the fragment reads free of bank conflicts (fff_gemm.hpp); a workgroup of
// four waves computes a 256 x 256 (128 x 128 per wave), 256 x 192 or 128 x 128
// tile, and consecutive tiles of one row block of A run on one XCD.  A partial
// last step of K is loaded through registers with zeros past K.  Every 16x16
// MFMA returns D[4(l/16)+r][l%16] to lane l, register r; its bf16 operands are
// A[l%16][8(l/16) .. +7] and
// B[8(l/16) .. +7][l%16], its fp32 operands A[l%16][q] and B[q][l%16] for the
// lane's K slot q = l/16.  Rows past M and N read the last row (clamped
// addresses) and are never stored.
#include "fff_device.hpp"
#include "fff_gemm.hpp"
#include "fff_internal.hpp"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

namespace fff {

namespace {

// Output forms: fp32 C; or C plus a source row (none / fp32 / bf16), stored as bf16 or fp32; or
// the activation a of C (act), stored whole as fp32 or as two bf16 parts hi = bf16(a) and
// mid = bf16(a - hi) at part stride ldc in rows of 2 ldc elements, over the whole padded row:
// columns N .. ldc - 1 get zeros.
enum { GOUT_F32 = 0, GOUT_SRC_NONE = 1, GOUT_SRC_F32 = 2, GOUT_SRC_BF16 = 3, GOUT_ACT_F32 = 4, GOUT_ACT_P2 = 5 };

// Columns a store covers: N, or the whole padded row for the activation forms.
template <int OUT>
__device__ __forceinline__ int64_t gemm_store_cols(int64_t N, int64_t ldc) {
    return OUT >= GOUT_ACT_F32 ? ldc : N;
}

template <int OUT, bool DBF>
__device__ __forceinline__ void gemm_store(void* C, const void* src, int64_t ldc, int64_t m, int64_t n, float v,
                                           int64_t N, int act) {
    if constexpr (OUT >= GOUT_ACT_F32) {
        const float a = n < N ? activation(v, act) : 0.0f;
        if constexpr (OUT == GOUT_ACT_F32) {
            static_cast<float*>(C)[m * ldc + n] = a;
        } else {
            uint16_t* e = static_cast<uint16_t*>(C) + 2 * m * ldc + n;
            const uint16_t hi = f32_to_bf16(a);
            e[0] = hi;
            e[ldc] = f32_to_bf16(a - bf16_to_f32(hi));
        }
    } else {
        const int64_t e = m * ldc + n;
        if constexpr (OUT == GOUT_SRC_F32) v += static_cast<const float*>(src)[e];
        if constexpr (OUT == GOUT_SRC_BF16) v += bf16_to_f32(static_cast<const uint16_t*>(src)[e]);
        if constexpr (OUT == GOUT_F32 || !DBF) static_cast<float*>(C)[e] = v;
        else static_cast<uint16_t*>(C)[e] = f32_to_bf16(v);
    }
}

// Workgroup (blockIdx.x, blockIdx.y): tile xcd_tile(blockIdx.x) of C over K elements
// [blockIdx.y kchunk, +kchunk) (kchunk a whole number of steps; one chunk unless K is split, when C
// is the partial sums [gridDim.y][M][ldc] and OUT is GOUT_F32).
template <bool BF, int TM, int TN, int WGM, int WGN, int S, bool M32, int OUT, bool DBF>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_nt_dma_kernel(const void* __restrict__ A,
                                                                     const void* __restrict__ B, void* C,
                                                                     const void* src, int64_t M, int64_t N,
                                                                     int64_t K, int64_t lda, int64_t ldb,
                                                                     int64_t ldc, int64_t kchunk, int act) {
    using G = DmaCfg<TM, TN, WGM, WGN, S>;
    extern __shared__ __align__(16) unsigned char gsm[];  // [S stages][A rows, B rows][128 bytes]
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    const int r16 = lane & 15, q = lane >> 4;
    const int64_t tiles_n = (N + G::BN - 1) / G::BN;
    const int64_t t = xcd_tile(blockIdx.x, tiles_n * ((M + G::BM - 1) / G::BM));
    const int64_t m0 = (t / tiles_n) * G::BM, n0 = (t % tiles_n) * G::BN;
    const int64_t kb = int64_t(blockIdx.y) * kchunk, kl = K - kb < kchunk ? K - kb : kchunk;
    const int esz = BF ? 2 : 4;
    const int64_t nc = gemm_store_cols<OUT>(N, ldc);
    if (gridDim.y > 1) C = static_cast<float*>(C) + int64_t(blockIdx.y) * M * ldc;
    WaveAcc<TM, TN, M32> acc;
    dma_product<BF, TM, TN, WGM, WGN, S, M32>(static_cast<const char*>(A) + kb * esz,
                                              static_cast<const char*>(B) + kb * esz, M, N, kl, lda, ldb, m0, n0, gsm,
                                              acc);
    if constexpr (M32) {
        // 32 x 32 result: lane l, register r holds row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32
        const int r32 = lane & 31, hv = lane >> 5;
#pragma unroll
        for (int i = 0; i < TM / 2; ++i)
#pragma unroll
            for (int j = 0; j < TN / 2; ++j) {
                const int64_t n = n0 + wn * 16 * TN + j * 32 + r32;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int64_t m = m0 + wm * 16 * TM + i * 32 + 8 * (r / 4) + 4 * hv + (r % 4);
                    if (m < M && n < nc) gemm_store<OUT, DBF>(C, src, ldc, m, n, acc.t[i][j][r], N, act);
                }
            }
    } else {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int64_t n = n0 + wn * 16 * TN + j * 16 + r16;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int64_t m = m0 + wm * 16 * TM + i * 16 + 4 * q + r;
                    if (m < M && n < nc) gemm_store<OUT, DBF>(C, src, ldc, m, n, acc.t[i][j][r], N, act);
                }
            }
    }
}

// C = sum over the splits of the partial sums, in split order, through the product's store.
// ldc is a multiple of 4, so each thread reads four columns of every split as one 16-byte load
// (within the row of ldc columns; columns past N are never used).
template <int OUT, bool DBF>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, int splits, void* C,
                                                            const void* src, int64_t M, int64_t N, int64_t ldc,
                                                            int act) {
    const int64_t nc = gemm_store_cols<OUT>(N, ldc), nq = (nc + 3) / 4;
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < M * nq; i += int64_t(gridDim.x) * 256) {
        const int64_t m = i / nq, n = (i - m * nq) * 4;
        float4 v = *reinterpret_cast<const float4*>(part + m * ldc + n);
        for (int sp = 1; sp < splits; ++sp) {
            const float4 w = *reinterpret_cast<const float4*>(part + (int64_t(sp) * M + m) * ldc + n);
            v.x += w.x;
            v.y += w.y;
            v.z += w.z;
            v.w += w.w;
        }
        const float vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (n + k < nc) gemm_store<OUT, DBF>(C, src, ldc, m, n + k, vv[k], N, act);
    }
}

template <bool BF, int TM, int TN, int WGM, int WGN, int S, int OUT, bool DBF>
void launch_dma(const void* A, const void* B, void* C, const void* src, int64_t M, int64_t N, int64_t K,
                int64_t lda, int64_t ldb, int64_t ldc, int act, hipStream_t stream, int splits = 1, int64_t kchunk = 0) {
    using G = DmaCfg<TM, TN, WGM, WGN, S>;
    const dim3 grid(unsigned(((N + G::BN - 1) / G::BN) * ((M + G::BM - 1) / G::BM)), unsigned(splits));
    // bf16 on 32 x 32 x 16 MFMA tiles (twice the 16 x 16 x 32 rate per flop); fp32 on 16 x 16 x 4
    hipLaunchKernelGGL((gemm_nt_dma_kernel<BF, TM, TN, WGM, WGN, S, BF, OUT, DBF>), grid, dim3(G::THREADS), G::LDS, stream,
                       A, B, C, src, M, N, K, lda, ldb, ldc, splits > 1 ? kchunk : K, act);
}

// Tile choice, from the shapes and the CU count only: 256 x 256 tiles (128 x 128 per wave, bf16)
// or 256 x 192 (128 x 96 per wave), one workgroup per CU, whichever leaves fewer tile-rounds of
// idle CUs (the narrower tile reads ~7% more LDS per MFMA; its fp32 form is the only wide one
// that needs no spills), or 128 x 128 tiles with two workgroups per CU for small products and
// for the activation forms, whose epilogue evaluates the activation of every value it stores:
// at one workgroup per CU that chain of dependent instructions has nothing to hide under.  A
// small product with too few tiles for the CUs and a long K is split along K into chunks of
// whole steps (at least four each), up to two workgroups per CU and the partial sums' buffer,
// and reduced in split order: the split depends on the shapes, the CU count and split_bytes only.
template <bool BF, int OUT, bool DBF>
hipError_t launch_gemm(const void* A, const void* B, void* C, const void* src, int64_t M, int64_t N, int64_t K,
                       int64_t lda, int64_t ldb, int64_t ldc, int cu_count, void* split_ws, size_t split_bytes,
                       int act, hipStream_t stream) {
    auto cdiv = [](int64_t a, int64_t b) { return (a + b - 1) / b; };
    const int64_t slots = cu_count > 0 ? cu_count : 256;
    const int64_t t88 = cdiv(M, 256) * cdiv(N, 256), t86 = cdiv(M, 256) * cdiv(N, 192);
    if (OUT >= GOUT_ACT_F32 || t88 < slots / 4) {
        const int64_t t44 = cdiv(M, 128) * cdiv(N, 128), bk = BF ? 64 : 32, steps = cdiv(K, bk);
        int64_t splits = 1;
        if (split_ws && ldc % 4 == 0 && t44 < slots) {
            splits = std::min<int64_t>({cdiv(2 * slots, t44), steps / 4, int64_t(split_bytes / (size_t(M) * ldc * 4))});
        }
        if (splits >= 2) {
            const int64_t kchunk = cdiv(steps, splits) * bk;
            splits = cdiv(K, kchunk);
            launch_dma<BF, 4, 4, 2, 2, 2, GOUT_F32, false>(A, B, split_ws, nullptr, M, N, K, lda, ldb, ldc, 0, stream,
                                                           int(splits), kchunk);
            const int64_t work = M * cdiv(N, 4);
            const unsigned blocks = unsigned(std::min<int64_t>(cdiv(work, 256), 4 * slots));
            hipLaunchKernelGGL((splitk_reduce_kernel<OUT, DBF>), dim3(blocks), dim3(256), 0, stream,
                               static_cast<const float*>(split_ws), int(splits), C, src, M, N, ldc, act);
            return hipGetLastError();
        }
        launch_dma<BF, 4, 4, 2, 2, 2, OUT, DBF>(A, B, C, src, M, N, K, lda, ldb, ldc, act, stream);
        return hipGetLastError();
    }
    if constexpr (OUT < GOUT_ACT_F32) {
        if constexpr (BF) {
            if (double(cdiv(t88, slots)) * 256 * 256 <= double(cdiv(t86, slots)) * 256 * 192 * 1.07) {
                launch_dma<BF, 8, 8, 2, 2, 2, OUT, DBF>(A, B, C, src, M, N, K, lda, ldb, ldc, act, stream);
                return hipGetLastError();
            }
        }
        launch_dma<BF, 8, 6, 2, 2, 2, OUT, DBF>(A, B, C, src, M, N, K, lda, ldb, ldc, act, stream);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t gemm_nt(bool bf16, int out, bool dst_bf16, const void* A, const void* B, void* C, const void* src,
                   int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t ldc, int cu_count,
                   void* split_ws, size_t split_bytes, int act, hipStream_t stream) {
    if (M == 0 || N == 0) return hipSuccess;
    // the activation forms fill rows of ldc columns, within the 128-column tiles they run on
    if (out >= GEMM_OUT_ACT_F32 && (ldc % 4 != 0 || ldc < N || ldc > (N + 127) / 128 * 128)) return hipErrorInvalidValue;
#define FFF_GEMM(BF, OUT, DBF) \
    launch_gemm<BF, OUT, DBF>(A, B, C, src, M, N, K, lda, ldb, ldc, cu_count, split_ws, split_bytes, act, stream)
    if (bf16) {
        switch (out) {
            case GEMM_OUT_F32: return FFF_GEMM(true, GOUT_F32, false);
            case GEMM_OUT_SRC_NONE: return dst_bf16 ? FFF_GEMM(true, GOUT_SRC_NONE, true) : FFF_GEMM(true, GOUT_SRC_NONE, false);
            case GEMM_OUT_SRC_F32: return dst_bf16 ? FFF_GEMM(true, GOUT_SRC_F32, true) : FFF_GEMM(true, GOUT_SRC_F32, false);
            case GEMM_OUT_SRC_BF16: return dst_bf16 ? FFF_GEMM(true, GOUT_SRC_BF16, true) : FFF_GEMM(true, GOUT_SRC_BF16, false);
            case GEMM_OUT_ACT_P2: return FFF_GEMM(true, GOUT_ACT_P2, false);
            default: return hipErrorInvalidValue;
        }
    }
    switch (out) {
        case GEMM_OUT_F32: return FFF_GEMM(false, GOUT_F32, false);
        case GEMM_OUT_SRC_NONE: return FFF_GEMM(false, GOUT_SRC_NONE, false);
        case GEMM_OUT_SRC_F32: return FFF_GEMM(false, GOUT_SRC_F32, false);
        case GEMM_OUT_ACT_F32: return FFF_GEMM(false, GOUT_ACT_F32, false);
        default: return hipErrorInvalidValue;
    }
#undef FFF_GEMM
}

}  // namespace fff
