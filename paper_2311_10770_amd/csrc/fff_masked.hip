// fff_masked.hip -- MASKED mode: the FFF layer as two dense products with the
// conditional walk between them, for shallow trees.  With K trees of depth D a
// token uses N_I = K (D+1) of the N_T = K (2^(D+1) - 1) neurons (Section 2.1,
// Table 1); at depth 0 the layer is the dense feedforward, and for small D a
// large share of each row is used, so the layer runs best as dense MFMA work:
//   G1 (hipBLASLt, bf16 MFMA, fp32 accumulate): L[B, N_T] = x W_in^T, the logit
//      of every node of every tree;
//   select_kernel: per (token, tree) the walk of Algorithm 1 over those logits
//      (left on a logit <= 0, as in the other modes), the activation of every
//      visited node split into bf16 parts (P = 2 for a bf16 y, else 3: hi, mid,
//      lo, each the rounding of what the earlier parts leave), zeros for the
//      other nodes: A[B, P N_T], part p of node j at column p N_T + j;
//   G2: y = A [W_out; ...; W_out] (W_out repeated P times in the workspace), so
//      every product is exact and y is rounded once; accumulation and the
//      residual come in through the C operand (beta = 1).
// With fp32 x, W and y both products are fp32 GEMMs (full fp32 compute) and A
// holds the activations whole.  The workspace holds L, A, the repeated W_out and
// hipBLASLt's scratch.
#include "fff_common.hpp"
#include "fff_device.hpp"
#include "fff_internal.hpp"

#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>

#include <cstdint>
#include <map>
#include <mutex>
#include <tuple>

namespace fff {

namespace {

constexpr int SELECT_BLOCK = 256;
constexpr size_t LT_WORKSPACE = size_t(32) << 20;

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

int masked_parts(bool y_bf16) { return y_bf16 ? 2 : 3; }

// One workgroup per token: first every tree's path (thread per tree, records
// into LDS), then the token's row of A, thread per column.
template <bool F32>
__global__ __launch_bounds__(SELECT_BLOCK) void select_kernel(Params p, const float* __restrict__ L,
                                                              void* __restrict__ Aout, int parts) {
    extern __shared__ float s_path[];  // [T][D+1] activation, then [T][D+1] node (as int bits)
    const int T = p.n_trees, D = p.depth;
    const int64_t Nt = p.n_nodes, NT = Nt * T;
    const int64_t b = blockIdx.x;
    float* s_act = s_path;
    int32_t* s_node = reinterpret_cast<int32_t*>(s_path + int64_t(T) * (D + 1));
    const float* lrow = L + b * NT;
    for (int t = threadIdx.x; t < T; t += SELECT_BLOCK) {
        int64_t n = 0;
        for (int l = 0; l <= D; ++l) {
            const float logit = lrow[int64_t(t) * Nt + n];
            s_act[t * (D + 1) + l] = activation(logit, p.act);
            s_node[t * (D + 1) + l] = int32_t(n);
            const int64_t rec = (b * T + t) * (D + 1) + l;
            if (p.nodes_out) p.nodes_out[rec] = int32_t(n);
            if (p.logits_out) p.logits_out[rec] = logit;
            if (l < D) n = 2 * n + 1 + (logit > 0.0f ? 1 : 0);
        }
    }
    __syncthreads();
    for (int64_t j = threadIdx.x; j < NT; j += SELECT_BLOCK) {
        const int t = int(j / Nt);
        const int i = int(j - int64_t(t) * Nt);
        const int l = 31 - __builtin_clz(uint32_t(i + 1));  // level of heap node i
        const float v = s_node[t * (D + 1) + l] == i ? s_act[t * (D + 1) + l] : 0.0f;
        if constexpr (F32) {
            static_cast<float*>(Aout)[b * NT + j] = v;
        } else {
            uint16_t* arow = static_cast<uint16_t*>(Aout) + b * parts * NT;
            const uint16_t hi = f32_to_bf16(v);
            const float r = v - bf16_to_f32(hi);
            const uint16_t mid = f32_to_bf16(r);
            arow[j] = hi;
            arow[NT + j] = mid;
            if (parts == 3) arow[2 * NT + j] = f32_to_bf16(r - bf16_to_f32(mid));
        }
    }
}

// dst[r * n + i] = src[i] for r < reps (16-byte vectors)
__global__ __launch_bounds__(256) void repeat_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t n,
                                                     int reps) {
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) {
        const uint4 v = src[i];
        for (int r = 0; r < reps; ++r) dst[int64_t(r) * n + i] = v;
    }
}

// ---------------------------------------------------------------- hipBLASLt

struct GemmEntry {
    hipblasLtMatmulDesc_t desc = nullptr;
    hipblasLtMatrixLayout_t a = nullptr, b = nullptr, c = nullptr;
    hipblasLtMatmulAlgo_t algo{};
    bool ok = false;
};

struct LtState {
    hipblasLtHandle_t handle = nullptr;
    // (m, n, k, transa, input type, d type) -> descriptors and the heuristic's first algorithm
    std::map<std::tuple<int64_t, int64_t, int64_t, int, int, int>, GemmEntry> gemms;
};

std::mutex g_lt_mutex;
std::map<int, LtState> g_lt;  // per device

bool lt_ok(hipblasStatus_t s) { return s == HIPBLAS_STATUS_SUCCESS; }

// Column-major D[m, n] = op(A) B with A stored [k, m] (transa) or [m, k], B [k, n], inputs of type
// itype (bf16, or fp32 computed in full fp32), fp32 accumulation, D (and C) of type dtype.
GemmEntry* get_gemm(LtState& st, int64_t m, int64_t n, int64_t k, bool transa, hipDataType itype, hipDataType dtype) {
    const auto key = std::make_tuple(m, n, k, int(transa), int(itype), int(dtype));
    auto it = st.gemms.find(key);
    if (it != st.gemms.end()) return it->second.ok ? &it->second : nullptr;
    GemmEntry& g = st.gemms[key];
    if (!lt_ok(hipblasLtMatmulDescCreate(&g.desc, HIPBLAS_COMPUTE_32F, HIP_R_32F))) return nullptr;
    const hipblasOperation_t ta = transa ? HIPBLAS_OP_T : HIPBLAS_OP_N, tb = HIPBLAS_OP_N;
    hipblasLtMatmulDescSetAttribute(g.desc, HIPBLASLT_MATMUL_DESC_TRANSA, &ta, sizeof ta);
    hipblasLtMatmulDescSetAttribute(g.desc, HIPBLASLT_MATMUL_DESC_TRANSB, &tb, sizeof tb);
    if (!lt_ok(transa ? hipblasLtMatrixLayoutCreate(&g.a, itype, k, m, k) : hipblasLtMatrixLayoutCreate(&g.a, itype, m, k, m)))
        return nullptr;
    if (!lt_ok(hipblasLtMatrixLayoutCreate(&g.b, itype, k, n, k))) return nullptr;
    if (!lt_ok(hipblasLtMatrixLayoutCreate(&g.c, dtype, m, n, m))) return nullptr;
    hipblasLtMatmulPreference_t pref;
    if (!lt_ok(hipblasLtMatmulPreferenceCreate(&pref))) return nullptr;
    uint64_t ws = LT_WORKSPACE;
    hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &ws, sizeof ws);
    hipblasLtMatmulHeuristicResult_t res[1];
    int found = 0;
    const hipblasStatus_t s = hipblasLtMatmulAlgoGetHeuristic(st.handle, g.desc, g.a, g.b, g.c, g.c, pref, 1, res, &found);
    hipblasLtMatmulPreferenceDestroy(pref);
    if (!lt_ok(s) || found < 1 || res[0].state != HIPBLAS_STATUS_SUCCESS || res[0].workspaceSize > LT_WORKSPACE)
        return nullptr;
    g.algo = res[0].algo;
    g.ok = true;
    return &g;
}

}  // namespace

bool masked_shape(const Params& p) {
    // bf16 x and W (the products' operands), or fp32 x, W and y (fp32 products, the activations
    // whole); depth <= MASKED_MAX_DEPTH, no LayerNorm prologue; the residual needs y of x's type
    // (C and D share one layout)
    // (and the paths of a token's trees fit the selection kernel's LDS)
    const bool types = (p.x_bf16 && p.w_bf16) || (!p.x_bf16 && !p.w_bf16 && !p.y_bf16);
    return types && p.depth <= MASKED_MAX_DEPTH && !p.norm && p.hidden % 8 == 0 &&
           int64_t(p.n_trees) * (p.depth + 1) <= 8192 && (p.out_mode != OUT_RESIDUAL || p.x_bf16 == p.y_bf16);
}

size_t masked_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t hidden) {
    if (depth > MASKED_MAX_DEPTH) return 0;
    const size_t NT = ((size_t(1) << (depth + 1)) - 1) * size_t(n_trees);
    const int P = 3;  // the larger part count (fp32 y)
    return align256(size_t(n_tokens) * NT * sizeof(float)) + align256(size_t(n_tokens) * P * NT * sizeof(uint16_t)) +
           align256(size_t(P) * NT * size_t(hidden) * sizeof(uint16_t)) + LT_WORKSPACE;
}

hipError_t run_masked(const Params& p, void* workspace, hipStream_t stream) {
    const int64_t B = p.n_tokens, H = p.hidden, NT = p.n_nodes * p.n_trees;
    const bool f32 = !p.w_bf16;          // fp32 x, W and y: fp32 products, activations whole
    const int P = f32 ? 1 : masked_parts(p.y_bf16);
    char* ws = static_cast<char*>(workspace);
    float* L = reinterpret_cast<float*>(ws);
    ws += align256(size_t(B) * NT * sizeof(float));
    void* A = ws;                        // bf16 [B, P N_T] or fp32 [B, N_T]
    ws += align256(size_t(B) * 3 * NT * sizeof(uint16_t));
    uint16_t* Wrep = reinterpret_cast<uint16_t*>(ws);
    ws += align256(size_t(3) * NT * H * sizeof(uint16_t));
    void* lt_ws = ws;

    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(g_lt_mutex);
    LtState& st = g_lt[dev];
    if (!st.handle && !lt_ok(hipblasLtCreate(&st.handle))) return hipErrorNotSupported;
    const hipDataType itype = f32 ? HIP_R_32F : HIP_R_16BF;
    const hipDataType ydt = p.y_bf16 ? HIP_R_16BF : HIP_R_32F;
    const bool beta_on = p.out_mode != OUT_STORE;
    GemmEntry* g1 = get_gemm(st, NT, B, H, true, itype, HIP_R_32F);
    GemmEntry* g2 = get_gemm(st, H, B, int64_t(P) * NT, false, itype, ydt);
    if (!g1 || !g2) return hipErrorNotSupported;  // no hipBLASLt algorithm for a product
    const float one = 1.0f, zero = 0.0f;
    // G1: L^T (column-major [N_T, B]) = W_in (row-major [N_T, H]) x^T
    if (!lt_ok(hipblasLtMatmul(st.handle, g1->desc, &one, p.w_in, g1->a, p.x, g1->b, &zero, L, g1->c, L, g1->c,
                               &g1->algo, lt_ws, LT_WORKSPACE, stream)))
        return hipErrorLaunchFailure;
    // the repeated W_out (bf16 parts) and the selection
    if (!f32) {
        const int64_t nvec = NT * H * 2 / 16;
        const int grid = int(std::min<int64_t>((nvec + 255) / 256, 2048));
        hipLaunchKernelGGL(repeat_kernel, dim3(grid), dim3(256), 0, stream, reinterpret_cast<const uint4*>(p.w_out),
                           reinterpret_cast<uint4*>(Wrep), nvec, P);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const size_t lds = size_t(p.n_trees) * (p.depth + 1) * 8;
    if (f32) hipLaunchKernelGGL(select_kernel<true>, dim3(unsigned(B)), dim3(SELECT_BLOCK), lds, stream, p, L, A, 1);
    else hipLaunchKernelGGL(select_kernel<false>, dim3(unsigned(B)), dim3(SELECT_BLOCK), lds, stream, p, L, A, P);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    // G2: y^T (column-major [H, B]) = Wrep^T (column-major [H, P N_T]) A^T, plus C (y or x)
    const void* C = p.out_mode == OUT_RESIDUAL ? p.x : p.y;
    const void* W2 = f32 ? p.w_out : static_cast<const void*>(Wrep);
    if (!lt_ok(hipblasLtMatmul(st.handle, g2->desc, &one, W2, g2->a, A, g2->b, beta_on ? &one : &zero, C, g2->c, p.y,
                               g2->c, &g2->algo, lt_ws, LT_WORKSPACE, stream)))
        return hipErrorLaunchFailure;
    return hipSuccess;
}

}  // namespace fff
