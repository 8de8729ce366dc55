// fff_masked.hip -- MASKED mode: the FFF layer as two dense products with the
// conditional walk between them, for shallow trees.  With K trees of depth D a
// token uses N_I = K (D+1) of the N_T = K (2^(D+1) - 1) neurons (Section 2.1,
// Table 1); at depth 0 the layer is the dense feedforward, and for small D a
// large share of each row is used, so the layer runs best as dense MFMA work:
//   G1 (hipBLASLt, bf16 MFMA, fp32 accumulate): L[B, N_T] = x W_in^T, the logit
//      of every node of every tree;
//   selection: per (token, tree) the walk of Algorithm 1 over those logits
//      (left on a logit <= 0, as in the other modes), the activation of every
//      visited node split into bf16 parts (P = 2 for a bf16 y, else 3: hi, mid,
//      lo, each the rounding of what the earlier parts leave), zeros for the
//      other nodes: A[B, P, N_T'], part p of node j at column p N_T' + j, with
//      N_T' = N_T rounded up to 8 (zero padding) for 16-byte rows;
//   G2: y = A [W_out; ...; W_out] (W_out repeated P times in the workspace,
//      zero rows in the padding), so
//      every product is exact and y is rounded once; accumulation and the
//      residual come in through the C operand (beta = 1).
// With fp32 x, W and y both products are fp32 GEMMs (full fp32 compute) and A
// holds the activations whole.  The workspace holds L, A, the repeated W_out and
// hipBLASLt's scratch.  Each product runs the heuristic's first algorithm for
// its shape: a fixed choice, so the call only enqueues work and its results do
// not depend on timing.
#include "fff_common.hpp"
#include "fff_device.hpp"
#include "fff_internal.hpp"

#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>

#include <algorithm>
#include <cstdint>
#include <map>
#include <mutex>
#include <tuple>

namespace fff {

namespace {

constexpr int SELECT_BLOCK = 256;
constexpr int SELECT_LDS_COLS = 8192;  // widest logit row the staged selection keeps in LDS
constexpr size_t LT_WORKSPACE = size_t(32) << 20;

typedef uint2 __attribute__((may_alias)) lds_u2a;

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

int masked_parts(bool y_bf16) { return y_bf16 ? 2 : 3; }

// Columns of a row of L and of each part of A: N_T rounded up to 8, so that rows
// and parts start on 32-byte boundaries (the padding columns of A are zeros).
int64_t padded_cols(int64_t nt) { return (nt + 7) & ~int64_t(7); }

// Writes the values of columns [8 v, 8 v + 8) of token b's row of A: fp32 whole,
// or bf16 parts (hi, mid[, lo]) at part stride ntq.
template <bool F32>
__device__ __forceinline__ void emit8(void* __restrict__ Aout, int64_t b, int v, int ntq, int parts, const float (&val)[8]) {
    if constexpr (F32) {
        float4* row = reinterpret_cast<float4*>(static_cast<float*>(Aout) + b * ntq) + 2 * v;
        row[0] = make_float4(val[0], val[1], val[2], val[3]);
        row[1] = make_float4(val[4], val[5], val[6], val[7]);
    } else {
        uint16_t hi[8], mid[8], lo[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            hi[k] = f32_to_bf16(val[k]);
            const float r = val[k] - bf16_to_f32(hi[k]);
            mid[k] = f32_to_bf16(r);
            lo[k] = f32_to_bf16(r - bf16_to_f32(mid[k]));
        }
        auto pack = [](const uint16_t (&h)[8]) {
            return make_uint4(uint32_t(h[0]) | uint32_t(h[1]) << 16, uint32_t(h[2]) | uint32_t(h[3]) << 16,
                              uint32_t(h[4]) | uint32_t(h[5]) << 16, uint32_t(h[6]) | uint32_t(h[7]) << 16);
        };
        uint4* row = reinterpret_cast<uint4*>(static_cast<uint16_t*>(Aout) + b * parts * ntq);
        const int pv = ntq / 8;  // vectors per part
        row[v] = pack(hi);
        row[pv + v] = pack(mid);
        if (parts == 3) row[2 * pv + v] = pack(lo);
    }
}

// Records the visit of node n of tree t at level l (optional outputs).
__device__ __forceinline__ void record(const Params& p, int64_t b, int t, int l, int n, float logit) {
    const int64_t rec = (b * p.n_trees + t) * (p.depth + 1) + l;
    if (p.nodes_out) p.nodes_out[rec] = n;
    if (p.logits_out) p.logits_out[rec] = logit;
}

// One workgroup per token, its row of logits (ntq <= SELECT_LDS_COLS) staged in
// LDS with 16-byte loads: a thread per tree walks its tree there, replacing each
// visited node's logit by its activation and flagging it; then the row of A is
// written 8 columns (16 bytes per part) per thread.
template <bool F32>
__global__ __launch_bounds__(SELECT_BLOCK) void select_staged_kernel(Params p, const float* __restrict__ L,
                                                                     void* __restrict__ Aout, int parts, int ntq) {
    extern __shared__ float s_l[];                                 // [ntq] logits, then activations
    uint8_t* s_f = reinterpret_cast<uint8_t*>(s_l + ntq);          // [ntq] visited flags
    const int T = p.n_trees, D = p.depth, Nt = int(p.n_nodes);
    const int64_t b = blockIdx.x;
    const float4* lrow = reinterpret_cast<const float4*>(L + b * ntq);
    for (int v = threadIdx.x; v < ntq / 4; v += SELECT_BLOCK) {
        reinterpret_cast<float4*>(s_l)[v] = lrow[v];
        reinterpret_cast<uint32_t*>(s_f)[v] = 0;
    }
    __syncthreads();
    for (int t = threadIdx.x; t < T; t += SELECT_BLOCK) {
        float* tree = s_l + t * Nt;
        int n = 0;
        for (int l = 0; l <= D; ++l) {
            const float logit = tree[n];
            tree[n] = activation(logit, p.act);
            s_f[t * Nt + n] = 1;
            record(p, b, t, l, n, logit);
            if (l < D) n = 2 * n + 1 + (logit > 0.0f ? 1 : 0);
        }
    }
    __syncthreads();
    for (int v = threadIdx.x; v < ntq / 8; v += SELECT_BLOCK) {
        const float4 a0 = reinterpret_cast<const float4*>(s_l)[2 * v];
        const float4 a1 = reinterpret_cast<const float4*>(s_l)[2 * v + 1];
        const uint2 f = *reinterpret_cast<const lds_u2a*>(s_f + 8 * v);
        const float a[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
        float val[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) val[k] = (((k < 4 ? f.x : f.y) >> (8 * (k & 3))) & 0xff) ? a[k] : 0.0f;
        emit8<F32>(Aout, b, v, ntq, parts, val);
    }
}

// Rows wider than SELECT_LDS_COLS: one workgroup per token; first every tree's
// path (thread per tree, read from L, kept in LDS), then the row of A, 8 columns
// per thread.
template <bool F32>
__global__ __launch_bounds__(SELECT_BLOCK) void select_paths_kernel(Params p, const float* __restrict__ L,
                                                                    void* __restrict__ Aout, int parts, int ntq) {
    extern __shared__ float s_path[];  // [T][D+1] activation, then [T][D+1] node
    const int T = p.n_trees, D = p.depth, Nt = int(p.n_nodes);
    const int64_t b = blockIdx.x;
    float* s_act = s_path;
    int32_t* s_node = reinterpret_cast<int32_t*>(s_path + T * (D + 1));
    const float* lrow = L + b * ntq;
    for (int t = threadIdx.x; t < T; t += SELECT_BLOCK) {
        int n = 0;
        for (int l = 0; l <= D; ++l) {
            const float logit = lrow[t * Nt + n];
            s_act[t * (D + 1) + l] = activation(logit, p.act);
            s_node[t * (D + 1) + l] = n;
            record(p, b, t, l, n, logit);
            if (l < D) n = 2 * n + 1 + (logit > 0.0f ? 1 : 0);
        }
    }
    __syncthreads();
    for (int v = threadIdx.x; v < ntq / 8; v += SELECT_BLOCK) {
        int t = (8 * v) / Nt;
        int i = 8 * v - t * Nt;
        float val[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            float x = 0.0f;
            if (t < T) {
                const int l = 31 - __builtin_clz(uint32_t(i + 1));  // level of heap node i
                if (s_node[t * (D + 1) + l] == i) x = s_act[t * (D + 1) + l];
            }
            val[k] = x;
            if (++i == Nt) { i = 0; ++t; }
        }
        emit8<F32>(Aout, b, v, ntq, parts, val);
    }
}

// W_out [N_T, H] repeated: dst [reps][ntq][H], rows N_T..ntq-1 of each copy zero (16-byte vectors;
// n = N_T H / 8 vectors of the source, np = ntq H / 8 per copy).
__global__ __launch_bounds__(256) void repeat_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t n,
                                                     int64_t np, int reps) {
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < np; i += int64_t(gridDim.x) * 256) {
        const uint4 v = i < n ? src[i] : make_uint4(0, 0, 0, 0);
        for (int r = 0; r < reps; ++r) dst[int64_t(r) * np + i] = v;
    }
}

// ---------------------------------------------------------------- hipBLASLt

constexpr int LT_CANDIDATES = 8;  // heuristic candidates asked for; the first usable one runs

struct GemmEntry {
    hipblasLtMatmulDesc_t desc = nullptr;
    hipblasLtMatrixLayout_t a = nullptr, b = nullptr, c = nullptr;
    hipblasLtMatmulAlgo_t algo{};            // the heuristic's first usable algorithm
    bool ok = false;
};

struct LtState {
    hipblasLtHandle_t handle = nullptr;
    // (m, n, k, transa, input type, d type, ldb, ldc) -> descriptors and the heuristic's first algorithm
    std::map<std::tuple<int64_t, int64_t, int64_t, int, int, int, int64_t, int64_t>, GemmEntry> gemms;
};

std::mutex g_lt_mutex;
std::map<int, LtState> g_lt;  // per device

bool lt_ok(hipblasStatus_t s) { return s == HIPBLAS_STATUS_SUCCESS; }

// Column-major D[m, n] = op(A) B with A stored [k, m] (transa) or [m, k] (packed), B [k, n] with
// leading dimension ldb, D (and C) with leading dimension ldc; inputs of type itype (bf16, or fp32
// computed in full fp32), fp32 accumulation, D (and C) of type dtype.
GemmEntry* get_gemm(LtState& st, int64_t m, int64_t n, int64_t k, bool transa, hipDataType itype, hipDataType dtype,
                    int64_t ldb, int64_t ldc) {
    const auto key = std::make_tuple(m, n, k, int(transa), int(itype), int(dtype), ldb, ldc);
    auto it = st.gemms.find(key);
    if (it != st.gemms.end()) return it->second.ok ? &it->second : nullptr;
    GemmEntry& g = st.gemms[key];
    if (!lt_ok(hipblasLtMatmulDescCreate(&g.desc, HIPBLAS_COMPUTE_32F, HIP_R_32F))) return nullptr;
    const hipblasOperation_t ta = transa ? HIPBLAS_OP_T : HIPBLAS_OP_N, tb = HIPBLAS_OP_N;
    hipblasLtMatmulDescSetAttribute(g.desc, HIPBLASLT_MATMUL_DESC_TRANSA, &ta, sizeof ta);
    hipblasLtMatmulDescSetAttribute(g.desc, HIPBLASLT_MATMUL_DESC_TRANSB, &tb, sizeof tb);
    if (!lt_ok(transa ? hipblasLtMatrixLayoutCreate(&g.a, itype, k, m, k) : hipblasLtMatrixLayoutCreate(&g.a, itype, m, k, m)))
        return nullptr;
    if (!lt_ok(hipblasLtMatrixLayoutCreate(&g.b, itype, k, n, ldb))) return nullptr;
    if (!lt_ok(hipblasLtMatrixLayoutCreate(&g.c, dtype, m, n, ldc))) return nullptr;
    hipblasLtMatmulPreference_t pref;
    if (!lt_ok(hipblasLtMatmulPreferenceCreate(&pref))) return nullptr;
    uint64_t ws = LT_WORKSPACE;
    hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &ws, sizeof ws);
    hipblasLtMatmulHeuristicResult_t res[LT_CANDIDATES];
    int found = 0;
    const hipblasStatus_t s =
        hipblasLtMatmulAlgoGetHeuristic(st.handle, g.desc, g.a, g.b, g.c, g.c, pref, LT_CANDIDATES, res, &found);
    hipblasLtMatmulPreferenceDestroy(pref);
    if (!lt_ok(s)) return nullptr;
    for (int i = 0; i < found && i < LT_CANDIDATES && !g.ok; ++i)
        if (res[i].state == HIPBLAS_STATUS_SUCCESS && res[i].workspaceSize <= LT_WORKSPACE) {
            g.algo = res[i].algo;
            g.ok = true;
        }
    return g.ok ? &g : nullptr;
}

}  // namespace

bool masked_shape(const Params& p) {
    // bf16 x and W (the products' operands), or fp32 x, W and y (fp32 products, the activations
    // whole); depth <= MASKED_MAX_DEPTH, no LayerNorm prologue; the residual needs y of x's type
    // (C and D share one layout)
    // (and the paths of a token's trees fit the LDS of the selection for wide rows)
    const bool types = (p.x_bf16 && p.w_bf16) || (!p.x_bf16 && !p.w_bf16 && !p.y_bf16);
    return types && p.depth <= MASKED_MAX_DEPTH && !p.norm && p.hidden % 8 == 0 &&
           int64_t(p.n_trees) * (p.depth + 1) <= 8192 && (p.out_mode != OUT_RESIDUAL || p.x_bf16 == p.y_bf16);
}

size_t masked_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t hidden) {
    if (depth > MASKED_MAX_DEPTH) return 0;
    const size_t ntq = size_t(padded_cols(((int64_t(1) << (depth + 1)) - 1) * n_trees));
    const int P = 3;  // the larger part count (fp32 y); three bf16 parts also cover one fp32 row
    return align256(size_t(n_tokens) * ntq * sizeof(float)) + align256(size_t(n_tokens) * P * ntq * sizeof(uint16_t)) +
           align256(size_t(P) * ntq * size_t(hidden) * sizeof(uint16_t)) + LT_WORKSPACE;
}

hipError_t run_masked(const Params& p, void* workspace, hipStream_t stream) {
    const int64_t B = p.n_tokens, H = p.hidden, NT = p.n_nodes * p.n_trees, ntq = padded_cols(NT);
    const bool f32 = !p.w_bf16;          // fp32 x, W and y: fp32 products, activations whole
    const int P = f32 ? 1 : masked_parts(p.y_bf16);
    char* ws = static_cast<char*>(workspace);
    float* L = reinterpret_cast<float*>(ws);  // [B, ntq]
    ws += align256(size_t(B) * ntq * sizeof(float));
    void* A = ws;                             // bf16 [B, P, ntq] or fp32 [B, ntq]
    ws += align256(size_t(B) * 3 * ntq * sizeof(uint16_t));
    uint16_t* Wrep = reinterpret_cast<uint16_t*>(ws);  // bf16 [P, ntq, H]
    ws += align256(size_t(3) * ntq * H * sizeof(uint16_t));
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
    // G2's reduction: fp32 over the N_T real columns of A (row stride ntq); bf16 over all P ntq
    // columns against the zero-padded copies of W_out
    const int64_t k2 = f32 ? NT : P * ntq;
    GemmEntry* g1 = get_gemm(st, NT, B, H, true, itype, HIP_R_32F, H, ntq);
    GemmEntry* g2 = get_gemm(st, H, B, k2, false, itype, ydt, f32 ? ntq : k2, H);
    if (!g1 || !g2) return hipErrorNotSupported;  // no hipBLASLt algorithm for a product
    const float one = 1.0f, zero = 0.0f;
    // G1: L^T (column-major [N_T, B], leading dimension ntq) = W_in (row-major [N_T, H]) x^T
    auto run_g1 = [&](const hipblasLtMatmulAlgo_t& algo) {
        return lt_ok(hipblasLtMatmul(st.handle, g1->desc, &one, p.w_in, g1->a, p.x, g1->b, &zero, L, g1->c, L,
                                     g1->c, &algo, lt_ws, LT_WORKSPACE, stream));
    };
    if (!run_g1(g1->algo)) return hipErrorLaunchFailure;
    if (!f32) {
        const int64_t n = NT * H / 8, np = ntq * H / 8;
        const int grid = int(std::min<int64_t>((np + 255) / 256, 2048));
        hipLaunchKernelGGL(repeat_kernel, dim3(grid), dim3(256), 0, stream, reinterpret_cast<const uint4*>(p.w_out),
                           reinterpret_cast<uint4*>(Wrep), n, np, P);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int nq = int(ntq);
    if (ntq <= SELECT_LDS_COLS) {
        const size_t lds = size_t(ntq) * (sizeof(float) + 1);
        if (f32)
            hipLaunchKernelGGL(select_staged_kernel<true>, dim3(unsigned(B)), dim3(SELECT_BLOCK), lds, stream, p, L, A,
                               1, nq);
        else
            hipLaunchKernelGGL(select_staged_kernel<false>, dim3(unsigned(B)), dim3(SELECT_BLOCK), lds, stream, p, L,
                               A, P, nq);
    } else {
        const size_t lds = size_t(p.n_trees) * (p.depth + 1) * 8;
        if (f32)
            hipLaunchKernelGGL(select_paths_kernel<true>, dim3(unsigned(B)), dim3(SELECT_BLOCK), lds, stream, p, L, A,
                               1, nq);
        else
            hipLaunchKernelGGL(select_paths_kernel<false>, dim3(unsigned(B)), dim3(SELECT_BLOCK), lds, stream, p, L, A,
                               P, nq);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    // G2: y^T (column-major [H, B]) = Wrep^T (column-major [H, k2]) A^T, plus C (y or x)
    const void* C = p.out_mode == OUT_RESIDUAL ? p.x : p.y;
    const void* W2 = f32 ? p.w_out : static_cast<const void*>(Wrep);
    if (!lt_ok(hipblasLtMatmul(st.handle, g2->desc, &one, W2, g2->a, A, g2->b, beta_on ? &one : &zero, C, g2->c, p.y,
                               g2->c, &g2->algo, lt_ws, LT_WORKSPACE, stream)))
        return hipErrorLaunchFailure;
    return hipSuccess;
}

}  // namespace fff
