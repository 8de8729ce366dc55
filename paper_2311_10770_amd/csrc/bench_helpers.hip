// bench_helpers.hip -- benchmark-only helpers (libfffbench.so), not part of
// the FFF library:
//   * a dense feedforward y = GELU(x W1^T) W2^T on hipBLASLt (bf16 in/out with
//     fp32 accumulation, or fp32 throughout; MFMA), GELU fused into the first
//     GEMM's epilogue, the fastest of the heuristic's candidate algorithms
//     picked by timing -- the dense layer the FFF is compared against;
//   * a plain vectorised copy kernel whose HBM counter readings calibrate the
//     traffic measured for the FFF kernels.
#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <vector>

#define FFFB_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

struct Gemm {
    hipblasLtMatmulDesc_t desc = nullptr;
    hipblasLtMatrixLayout_t a = nullptr, b = nullptr, d = nullptr;
    hipblasLtMatmulAlgo_t algo{};
    bool have_algo = false;
};

struct DenseFF {
    hipblasLtHandle_t lt = nullptr;
    Gemm g1, g2;
    void* ws = nullptr;
    size_t ws_bytes = 0;
    int64_t tokens = 0;
    int hidden = 0, width = 0;
    hipDataType dt = HIP_R_16BF;
    char info[256] = {0};
};

constexpr size_t kWorkspace = 64u << 20;

bool lt_ok(hipblasStatus_t s) { return s == HIPBLAS_STATUS_SUCCESS; }

// Column-major view of row-major tensors: D[m x n] = op(A) * B with
// A stored as a row-major [m, k] matrix (transposed col-major k x m).
bool make_gemm(DenseFF* ff, Gemm* g, uint64_t m, uint64_t n, uint64_t k, bool gelu) {
    if (!lt_ok(hipblasLtMatmulDescCreate(&g->desc, HIPBLAS_COMPUTE_32F, HIP_R_32F))) return false;
    hipblasOperation_t ta = HIPBLAS_OP_T, tb = HIPBLAS_OP_N;
    hipblasLtMatmulDescSetAttribute(g->desc, HIPBLASLT_MATMUL_DESC_TRANSA, &ta, sizeof ta);
    hipblasLtMatmulDescSetAttribute(g->desc, HIPBLASLT_MATMUL_DESC_TRANSB, &tb, sizeof tb);
    if (gelu) {
        hipblasLtEpilogue_t ep = HIPBLASLT_EPILOGUE_GELU;
        if (!lt_ok(hipblasLtMatmulDescSetAttribute(g->desc, HIPBLASLT_MATMUL_DESC_EPILOGUE, &ep, sizeof ep)))
            return false;
    }
    if (!lt_ok(hipblasLtMatrixLayoutCreate(&g->a, ff->dt, k, m, k))) return false;
    if (!lt_ok(hipblasLtMatrixLayoutCreate(&g->b, ff->dt, k, n, k))) return false;
    if (!lt_ok(hipblasLtMatrixLayoutCreate(&g->d, ff->dt, m, n, m))) return false;
    return true;
}

hipblasStatus_t run_gemm(DenseFF* ff, Gemm* g, const void* A, const void* B, void* D, hipStream_t s,
                         const hipblasLtMatmulAlgo_t* algo) {
    const float alpha = 1.0f, beta = 0.0f;
    return hipblasLtMatmul(ff->lt, g->desc, &alpha, A, g->a, B, g->b, &beta, D, g->d, D, g->d, algo, ff->ws,
                           ff->ws_bytes, s);
}

// Time every heuristic candidate on the real buffers and keep the fastest.
bool tune(DenseFF* ff, Gemm* g, const void* A, const void* B, void* D, hipStream_t s, float* best_ms) {
    hipblasLtMatmulPreference_t pref;
    if (!lt_ok(hipblasLtMatmulPreferenceCreate(&pref))) return false;
    uint64_t ws = ff->ws_bytes;
    hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &ws, sizeof ws);
    hipblasLtMatmulHeuristicResult_t res[16];
    int n = 0;
    hipblasStatus_t st = hipblasLtMatmulAlgoGetHeuristic(ff->lt, g->desc, g->a, g->b, g->d, g->d, pref, 16, res, &n);
    hipblasLtMatmulPreferenceDestroy(pref);
    if (!lt_ok(st) || n < 1) return false;
    hipEvent_t e0, e1;
    hipEventCreate(&e0);
    hipEventCreate(&e1);
    float best = 1e30f;
    for (int i = 0; i < n; ++i) {
        if (res[i].state != HIPBLAS_STATUS_SUCCESS || res[i].workspaceSize > ff->ws_bytes) continue;
        if (!lt_ok(run_gemm(ff, g, A, B, D, s, &res[i].algo))) continue;
        hipEventRecord(e0, s);
        for (int r = 0; r < 10; ++r) run_gemm(ff, g, A, B, D, s, &res[i].algo);
        hipEventRecord(e1, s);
        hipEventSynchronize(e1);
        float ms = 0.f;
        hipEventElapsedTime(&ms, e0, e1);
        if (ms < best) {
            best = ms;
            g->algo = res[i].algo;
            g->have_algo = true;
        }
    }
    hipEventDestroy(e0);
    hipEventDestroy(e1);
    *best_ms = best / 10.0f;
    return g->have_algo;
}

__global__ void copy_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t n) {
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += int64_t(gridDim.x) * blockDim.x)
        dst[i] = src[i];
}

// Microbenchmarks of the memory hierarchy (the rooflines the FFF kernels run against).
// mb_read: every thread streams 16-byte vectors from a footprint of (mask + 1)
// vectors, `total` vectors in all (wrapping), so the footprint decides whether
// L2, MALL or HBM serves them.
__global__ void mb_read_kernel(const uint4* __restrict__ buf, int64_t mask, int64_t total, uint32_t* out) {
    uint32_t acc = 0;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < total; i += int64_t(gridDim.x) * blockDim.x) {
        const uint4 v = buf[i & mask];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x9e3779b9u) out[0] = acc;  // keeps the loads alive; practically never stores
}

// mb_write: every thread streams 16-byte vector stores over a footprint of (mask + 1) vectors,
// `total` vectors in all (wrapping), like mb_read.
__global__ void mb_write_kernel(uint4* __restrict__ buf, int64_t mask, int64_t total, uint32_t seed) {
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < total; i += int64_t(gridDim.x) * blockDim.x)
        buf[i & mask] = make_uint4(seed, seed ^ uint32_t(i), seed, seed);
}

// mb_gather: groups of 16 lanes gather whole rows (`row_vecs` 16-byte vectors)
// from a table of `rows` rows; `steps` rows per group.  dependent = 0: row ids
// come from a hash (independent loads); dependent = 1: each row id is derived
// from the previous row's data, a serial chain like a tree walk.
__global__ void mb_gather_kernel(const uint4* __restrict__ table, int64_t rows, int row_vecs, int steps, int dependent,
                                 uint32_t* out) {
    const int lane = threadIdx.x & 15;
    const int64_t group = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) >> 4;
    uint32_t h = uint32_t(group) * 2654435761u + 12345u;
    uint32_t acc = 0;
    for (int s = 0; s < steps; ++s) {
        const uint32_t key = dependent ? (h ^ acc) : h;
        const int64_t row = int64_t((key * 2246822519u) >> 7) % rows;
        const uint4* r = table + row * row_vecs;
        uint32_t part = 0;
        for (int c = lane; c < row_vecs; c += 16) {
            const uint4 v = r[c];
            part ^= v.x ^ v.y ^ v.z ^ v.w;
        }
        // fold the group's lanes so every lane sees the same value (a stand-in for the dot product reduction)
        part ^= __shfl_xor(part, 8, 16);
        part ^= __shfl_xor(part, 4, 16);
        part ^= __shfl_xor(part, 2, 16);
        part ^= __shfl_xor(part, 1, 16);
        acc += part & 1u;
        h = h * 1664525u + 1013904223u;
    }
    if (acc == 0x7fffffffu) out[0] = acc;
}

// mb_mfma: the matrix cores' issue rate.  Every wave runs `iters` rounds of NACC independent MFMAs
// on register operands (no memory traffic); launched with 1, 2 or 4 waves per SIMD.
typedef __bf16 mb_bf16x8 __attribute__((ext_vector_type(8)));
typedef float mb_v4f __attribute__((ext_vector_type(4)));
typedef float mb_v16f __attribute__((ext_vector_type(16)));

template <int SHAPE, int NACC>
__global__ __launch_bounds__(256) void mb_mfma_kernel(int iters, float seed, float* out) {
    mb_bf16x8 a, b;
    for (int i = 0; i < 8; ++i) {
        a[i] = (__bf16)(seed * float(threadIdx.x + i));
        b[i] = (__bf16)(seed - float(i));
    }
    const float af = seed * float(threadIdx.x), bf = seed - 1.0f;
    float s = 0.0f;
    if constexpr (SHAPE == 0 || SHAPE == 2) {
        mb_v4f acc[NACC];
        for (int j = 0; j < NACC; ++j) acc[j] = mb_v4f{0.f, 0.f, 0.f, 0.f};
        for (int it = 0; it < iters; ++it)
#pragma unroll
            for (int j = 0; j < NACC; ++j) {
                if constexpr (SHAPE == 0) acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[j], 0, 0, 0);
                else acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af, bf, acc[j], 0, 0, 0);
            }
        for (int j = 0; j < NACC; ++j) s += acc[j][0];
    } else {
        mb_v16f acc[NACC];
        for (int j = 0; j < NACC; ++j)
            for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;
        for (int it = 0; it < iters; ++it)
#pragma unroll
            for (int j = 0; j < NACC; ++j) {
                if constexpr (SHAPE == 1) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
                else acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af, bf, acc[j], 0, 0, 0);
            }
        for (int j = 0; j < NACC; ++j) s += acc[j][0];
    }
    out[int64_t(blockIdx.x) * blockDim.x + threadIdx.x] = s;
}

}  // namespace

FFFB_EXPORT int fffb_mb_read(const void* buf, int64_t footprint_bytes, int64_t total_bytes, void* out, int grid,
                             void* stream) {
    const int64_t nvec = footprint_bytes / 16;
    if (nvec < 1 || (nvec & (nvec - 1)) || total_bytes < 16 || grid < 1) return -1;
    hipLaunchKernelGGL(mb_read_kernel, dim3(grid), dim3(256), 0, reinterpret_cast<hipStream_t>(stream),
                       reinterpret_cast<const uint4*>(buf), nvec - 1, total_bytes / 16, reinterpret_cast<uint32_t*>(out));
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

FFFB_EXPORT int fffb_mb_write(void* buf, int64_t footprint_bytes, int64_t total_bytes, int grid, void* stream) {
    const int64_t nvec = footprint_bytes / 16;
    if (nvec < 1 || (nvec & (nvec - 1)) || total_bytes < 16 || grid < 1) return -1;
    hipLaunchKernelGGL(mb_write_kernel, dim3(grid), dim3(256), 0, reinterpret_cast<hipStream_t>(stream),
                       reinterpret_cast<uint4*>(buf), nvec - 1, total_bytes / 16, 0x5bd1e995u);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

FFFB_EXPORT int fffb_mb_gather(const void* table, int64_t rows, int row_bytes, int groups, int steps, int dependent,
                               void* out, void* stream) {
    if (rows < 1 || row_bytes < 16 || (row_bytes & 15) || groups < 16 || (groups % 16) || steps < 1) return -1;
    const int threads = groups * 16;
    hipLaunchKernelGGL(mb_gather_kernel, dim3(threads / 256), dim3(256), 0, reinterpret_cast<hipStream_t>(stream),
                       reinterpret_cast<const uint4*>(table), rows, row_bytes / 16, steps, dependent,
                       reinterpret_cast<uint32_t*>(out));
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

FFFB_EXPORT void fffb_dense_ff_destroy(void* handle) {
    DenseFF* ff = static_cast<DenseFF*>(handle);
    if (!ff) return;
    for (Gemm* g : {&ff->g1, &ff->g2}) {
        if (g->a) hipblasLtMatrixLayoutDestroy(g->a);
        if (g->b) hipblasLtMatrixLayoutDestroy(g->b);
        if (g->d) hipblasLtMatrixLayoutDestroy(g->d);
        if (g->desc) hipblasLtMatmulDescDestroy(g->desc);
    }
    if (ff->ws) hipFree(ff->ws);
    if (ff->lt) hipblasLtDestroy(ff->lt);
    delete ff;
}

// Create a tuned dense FF for [tokens, hidden] -> [tokens, width] -> [tokens, hidden]; every
// tensor bf16 (f32 = 0) or fp32 (f32 = 1), fp32 accumulation.  Buffers are used for tuning only
// (contents are overwritten).  Returns NULL on failure.
FFFB_EXPORT void* fffb_dense_ff_create(int64_t tokens, int32_t hidden, int32_t width, int32_t f32, const void* x,
                                       const void* w1, const void* w2, void* h, void* y, void* stream) {
    DenseFF* ff = new DenseFF();
    ff->dt = f32 ? HIP_R_32F : HIP_R_16BF;
    ff->tokens = tokens;
    ff->hidden = hidden;
    ff->width = width;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    bool ok = lt_ok(hipblasLtCreate(&ff->lt)) && hipMalloc(&ff->ws, kWorkspace) == hipSuccess;
    ff->ws_bytes = ok ? kWorkspace : 0;
    ok = ok && make_gemm(ff, &ff->g1, width, tokens, hidden, true) && make_gemm(ff, &ff->g2, hidden, tokens, width, false);
    float t1 = 0, t2 = 0;
    ok = ok && tune(ff, &ff->g1, w1, x, h, s, &t1) && tune(ff, &ff->g2, w2, h, y, s, &t2);
    if (!ok) {
        std::fprintf(stderr, "fffb_dense_ff_create: hipBLASLt setup failed\n");
        fffb_dense_ff_destroy(ff);
        return nullptr;
    }
    std::snprintf(ff->info, sizeof ff->info, "hipBLASLt %s, GELU epilogue; tuned gemm1 %.1f us, gemm2 %.1f us",
                  f32 ? "fp32" : "bf16", t1 * 1e3f, t2 * 1e3f);
    return ff;
}

FFFB_EXPORT const char* fffb_dense_ff_info(void* handle) {
    return handle ? static_cast<DenseFF*>(handle)->info : "";
}

// h = GELU(x W1^T); y = h W2^T.  Returns 0 or the failing hipblasStatus_t.
FFFB_EXPORT int fffb_dense_ff_run(void* handle, const void* x, const void* w1, const void* w2, void* h, void* y,
                                  void* stream) {
    DenseFF* ff = static_cast<DenseFF*>(handle);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipblasStatus_t st = run_gemm(ff, &ff->g1, w1, x, h, s, &ff->g1.algo);
    if (!lt_ok(st)) return int(st);
    st = run_gemm(ff, &ff->g2, w2, h, y, s, &ff->g2.algo);
    return lt_ok(st) ? 0 : int(st);
}

// dst = src, bytes a multiple of 16, both 16-byte aligned.
FFFB_EXPORT int fffb_copy(const void* src, void* dst, int64_t bytes, void* stream) {
    if ((bytes & 15) || (reinterpret_cast<uintptr_t>(src) & 15) || (reinterpret_cast<uintptr_t>(dst) & 15)) return -1;
    const int64_t n = bytes / 16;
    if (n == 0) return 0;
    const int block = 256;
    const int64_t grid = std::min<int64_t>((n + block - 1) / block, 256 * 16);
    hipLaunchKernelGGL(copy_kernel, dim3(unsigned(grid)), dim3(block), 0, reinterpret_cast<hipStream_t>(stream),
                       reinterpret_cast<const uint4*>(src), reinterpret_cast<uint4*>(dst), n);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

// shape: 0 = 16x16x32 bf16, 1 = 32x32x16 bf16, 2 = 16x16x4 fp32, 3 = 32x32x2 fp32 (16 or 8 independent
// accumulators per wave); blocks of four waves, waves_per_simd blocks per CU; out: blocks x 256 floats.
// Returns the flops one launch performs, or a negative value.
FFFB_EXPORT double fffb_mb_mfma(int shape, int cus, int waves_per_simd, int iters, void* out, void* stream) {
    if (cus < 1 || waves_per_simd < 1 || iters < 1 || shape < 0 || shape > 3) return -1.0;
    const int blocks = cus * waves_per_simd;
    const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    float* o = reinterpret_cast<float*>(out);
    const double waves = double(blocks) * 4, per_mfma[4] = {16.0 * 16 * 32 * 2, 32.0 * 32 * 16 * 2, 16.0 * 16 * 4 * 2,
                                                              32.0 * 32 * 2 * 2};
    const int nacc = shape == 0 || shape == 2 ? 16 : 8;
    switch (shape) {
        case 0: hipLaunchKernelGGL((mb_mfma_kernel<0, 16>), dim3(blocks), dim3(256), 0, st, iters, 0.5f, o); break;
        case 1: hipLaunchKernelGGL((mb_mfma_kernel<1, 8>), dim3(blocks), dim3(256), 0, st, iters, 0.5f, o); break;
        case 2: hipLaunchKernelGGL((mb_mfma_kernel<2, 16>), dim3(blocks), dim3(256), 0, st, iters, 0.5f, o); break;
        default: hipLaunchKernelGGL((mb_mfma_kernel<3, 8>), dim3(blocks), dim3(256), 0, st, iters, 0.5f, o); break;
    }
    if (hipGetLastError() != hipSuccess) return -2.0;
    return waves * iters * nacc * per_mfma[shape];
}
