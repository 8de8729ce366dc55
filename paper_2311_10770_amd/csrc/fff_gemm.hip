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

#include <cstdint>

namespace fff {

namespace {

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

template <bool BF, int TM, int TN, int WGM, int WGN, int S, int OUT, bool DBF>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_nt_dma_kernel(const void* __restrict__ A,
                                                                     const void* __restrict__ B, void* C,
                                                                     const void* src, int64_t M, int64_t N,
                                                                     int64_t K, int64_t lda, int64_t ldb,
                                                                     int64_t ldc) {
    using G = DmaCfg<TM, TN, WGM, WGN, S>;
    extern __shared__ __align__(16) unsigned char gsm[];  // [S stages][A rows, B rows][128 bytes]
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave / WGN, wn = wave % WGN;
    const int r16 = lane & 15, q = lane >> 4;
    const int64_t tiles_n = (N + G::BN - 1) / G::BN;
    const int64_t t = xcd_tile(blockIdx.x, tiles_n * ((M + G::BM - 1) / G::BM));
    const int64_t m0 = (t / tiles_n) * G::BM, n0 = (t % tiles_n) * G::BN;
    tile_v4f acc[TM][TN];
    dma_product<BF, TM, TN, WGM, WGN, S>(A, B, M, N, K, lda, ldb, m0, n0, gsm, acc);
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

// Tile choice, from the shapes and the CU count only: 256 x 256 tiles (128 x 128 per wave, bf16)
// or 256 x 192 (128 x 96 per wave), one workgroup per CU, whichever leaves fewer tile-rounds of
// idle CUs (the narrower tile reads ~7% more LDS per MFMA; its fp32 form is the only wide one
// that needs no spills), or 128 x 128 tiles with two workgroups per CU for small products.
template <bool BF, int OUT, bool DBF>
hipError_t launch_gemm(const void* A, const void* B, void* C, const void* src, int64_t M, int64_t N, int64_t K,
                       int64_t lda, int64_t ldb, int64_t ldc, int cu_count, hipStream_t stream) {
    auto cdiv = [](int64_t a, int64_t b) { return (a + b - 1) / b; };
    const int64_t slots = cu_count > 0 ? cu_count : 256;
    const int64_t t88 = cdiv(M, 256) * cdiv(N, 256), t86 = cdiv(M, 256) * cdiv(N, 192);
    if (t88 < slots / 4) {
        launch_dma<BF, 4, 4, 2, 2, 2, OUT, DBF>(A, B, C, src, M, N, K, lda, ldb, ldc, stream);
        return hipGetLastError();
    }
    if constexpr (BF) {
        if (double(cdiv(t88, slots)) * 256 * 256 <= double(cdiv(t86, slots)) * 256 * 192 * 1.07) {
            launch_dma<BF, 8, 8, 2, 2, 2, OUT, DBF>(A, B, C, src, M, N, K, lda, ldb, ldc, stream);
            return hipGetLastError();
        }
    }
    launch_dma<BF, 8, 6, 2, 2, 2, OUT, DBF>(A, B, C, src, M, N, K, lda, ldb, ldc, stream);
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
