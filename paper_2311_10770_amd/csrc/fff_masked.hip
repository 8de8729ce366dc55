// fff_masked.hip -- MASKED mode: the FFF layer as two dense products with the
// conditional walk between them, for shallow trees.  With K trees of depth D a
// token uses N_I = K (D+1) of the N_T = K (2^(D+1) - 1) neurons (Section 2.1,
// Table 1); at depth 0 the layer is the dense feedforward, and for small D a
// large share of each row is used, so the layer runs best as dense MFMA work:
//   G1 (fff_gemm.hip, bf16 MFMA, fp32 accumulate): L[B, N_T] = x W_in^T, the
//      logit of every node of every tree;
//   selection: per (token, tree) the walk of Algorithm 1 over those logits
//      (left on a logit <= 0, as in the other modes), the activation of every
//      visited node split into bf16 parts (P = 2 for a bf16 y, else 3: hi, mid,
//      lo, each the rounding of what the earlier parts leave), zeros for the
//      other nodes: A[B, P, N_T'], part p of node j at column p N_T' + j, with
//      N_T' = N_T rounded up to 8 (zero padding) for 16-byte rows;
//   G2: y = A [W_out; ...; W_out] against W_out transposed and repeated P times
//      in the workspace (zero columns in the padding), so every product is
//      exact and y is rounded once; accumulation and the residual are added in
//      the product's store.
// With fp32 x, W and y both products are fp32 (fp32 MFMA) and A holds the
// activations whole.  The workspace holds L, A, the transposed W_out and the partial sums of a
// product split along K (few tokens, long K).
#include "fff_common.hpp"
#include "fff_device.hpp"
#include "fff_internal.hpp"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <type_traits>

namespace fff {

namespace {

constexpr int SELECT_BLOCK = 256;
constexpr int SELECT_LDS_COLS = 8192;  // widest logit row the staged selection keeps in LDS

typedef uint2 __attribute__((may_alias)) lds_u2a;

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

int masked_parts(bool y_bf16) { return y_bf16 ? 2 : 3; }

// Columns of a row of L and of each part of A: N_T rounded up to 64, so that each
// part is a whole number of the second product's K steps (64 bf16 or 32 fp32
// elements) and rows and parts start on 128-byte boundaries (the padding columns
// of A are zeros).
int64_t padded_cols(int64_t nt) { return (nt + 63) & ~int64_t(63); }

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

// Depth 0: every node is its tree's root and is visited, so the selection is elementwise: each
// thread takes eight columns of one token's row (the padding columns, past N_T, give zeros),
// with no LDS and no barrier.
template <bool F32>
__global__ __launch_bounds__(SELECT_BLOCK) void select_depth0_kernel(Params p, const float* __restrict__ L,
                                                                     void* __restrict__ Aout, int parts, int ntq) {
    const int64_t nv = ntq / 8, nt = int64_t(p.n_trees);
    const bool rec = p.nodes_out || p.logits_out;
    for (int64_t i = int64_t(blockIdx.x) * SELECT_BLOCK + threadIdx.x; i < p.n_tokens * nv;
         i += int64_t(gridDim.x) * SELECT_BLOCK) {
        const int64_t b = i / nv;
        const int v = int(i - b * nv);
        const float4* lrow = reinterpret_cast<const float4*>(L + b * ntq) + 2 * v;
        const float4 l0 = lrow[0], l1 = lrow[1];
        const float lg[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
        float val[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int t = 8 * v + k;
            val[k] = t < nt ? activation(lg[k], p.act) : 0.0f;
            if (rec && t < nt) record(p, b, t, 0, 0, lg[k]);
        }
        emit8<F32>(Aout, b, v, ntq, parts, val);
    }
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

// W_out [N_T, H] transposed and repeated: dst [H][reps * ntq] with dst[n][r ntq + j] = W_out[j][n]
// for j < N_T and 0 on the padding columns; bf16 (BF) or fp32 elements.  64 x 64 tiles through LDS
// so that both the reads (along H) and the writes (along N_T) are contiguous.
template <bool BF>
__global__ __launch_bounds__(256) void transpose_repeat_kernel(const void* __restrict__ src, void* __restrict__ dst,
                                                               int64_t nt, int64_t ntq, int64_t H, int reps) {
    typedef typename std::conditional<BF, uint16_t, float>::type E;
    __shared__ E tile[64][65];
    const int64_t j0 = int64_t(blockIdx.x) * 64, n0 = int64_t(blockIdx.y) * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    const E* s = static_cast<const E*>(src);
    E* d = static_cast<E*>(dst);
    for (int r = ty; r < 64; r += 4) {  // tile[j][n] = W_out[j0 + j][n0 + n]
        const int64_t j = j0 + r, n = n0 + tx;
        tile[r][tx] = j < nt && n < H ? s[j * H + n] : E(0);
    }
    __syncthreads();
    for (int r = ty; r < 64; r += 4) {  // dst[n0 + r][rep ntq + j0 + tx] = tile[tx][r]
        const int64_t n = n0 + r, j = j0 + tx;
        if (n < H && j < ntq) {
            const E v = tile[tx][r];
            for (int rep = 0; rep < reps; ++rep) d[n * (int64_t(reps) * ntq) + int64_t(rep) * ntq + j] = v;
        }
    }
}

// The selection: A from the logits L (depth 0 elementwise; else staged in LDS or by paths).
void launch_select(const Params& p, const float* L, void* A, bool f32, int P, int64_t ntq, int cu_count,
                   hipStream_t stream) {
    const int64_t B = p.n_tokens;
    const int nq = int(ntq);
    if (p.depth == 0) {
        const int64_t work = B * (ntq / 8);
        const unsigned blocks = unsigned(std::min<int64_t>((work + SELECT_BLOCK - 1) / SELECT_BLOCK, int64_t(cu_count > 0 ? cu_count : 256) * 16));
        if (f32)
            hipLaunchKernelGGL(select_depth0_kernel<true>, dim3(blocks), dim3(SELECT_BLOCK), 0, stream, p, L, A, 1, nq);
        else
            hipLaunchKernelGGL(select_depth0_kernel<false>, dim3(blocks), dim3(SELECT_BLOCK), 0, stream, p, L, A, P, nq);
    } else if (ntq <= SELECT_LDS_COLS) {
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
           align256(size_t(P) * ntq * size_t(hidden) * sizeof(uint16_t)) + GEMM_SPLIT_BYTES;
}

hipError_t run_masked(const Params& p, void* workspace, int cu_count, hipStream_t stream) {
    const int64_t B = p.n_tokens, H = p.hidden, NT = p.n_nodes * p.n_trees, ntq = padded_cols(NT);
    const bool f32 = !p.w_bf16;          // fp32 x, W and y: fp32 products, activations whole
    const int P = f32 ? 1 : masked_parts(p.y_bf16);
    char* ws = static_cast<char*>(workspace);
    float* L = reinterpret_cast<float*>(ws);  // [B, ntq]
    ws += align256(size_t(B) * ntq * sizeof(float));
    void* A = ws;                             // bf16 [B, P, ntq] or fp32 [B, ntq]
    ws += align256(size_t(B) * 3 * ntq * sizeof(uint16_t));
    void* WT = ws;                            // bf16 [H, P ntq] or fp32 [H, ntq]: W_out transposed
    ws += align256(size_t(3) * ntq * size_t(H) * sizeof(uint16_t));
    void* SP = ws;                            // partial sums of a product split along K

    // Depth 0 with no records: every node is visited, so A is the activation of every logit, and
    // the first product writes it itself (the same activation and part split as the selection),
    // whole or as two parts.  Three parts (fp32 y from bf16 operands) keep the selection pass:
    // the third part's stores made the fused product slower than the two kernels (3072x0 at
    // 16384 tokens: 537 against 530 us per forward, while two parts take 404 against 432 us).
    const bool fused = p.depth == 0 && !p.nodes_out && !p.logits_out && P <= 2;
    // G1: L = x W_in^T (logits of every node; the padding columns are not written), or A itself
    hipError_t e;
    if (fused) {
        const int out = f32 ? GEMM_OUT_ACT_F32 : GEMM_OUT_ACT_P2;
        e = gemm_nt(!f32, out, false, p.x, p.w_in, A, nullptr, B, NT, H, H, H, ntq, cu_count, SP, GEMM_SPLIT_BYTES,
                    p.act, stream);
    } else {
        e = gemm_nt(!f32, GEMM_OUT_F32, false, p.x, p.w_in, L, nullptr, B, NT, H, H, H, ntq, cu_count, SP,
                    GEMM_SPLIT_BYTES, 0, stream);
    }
    if (e != hipSuccess) return e;
    {
        const dim3 grid(unsigned((ntq + 63) / 64), unsigned((H + 63) / 64));
        if (f32)
            hipLaunchKernelGGL(transpose_repeat_kernel<false>, grid, dim3(256), 0, stream, p.w_out, WT, NT, ntq, H, 1);
        else
            hipLaunchKernelGGL(transpose_repeat_kernel<true>, grid, dim3(256), 0, stream, p.w_out, WT, NT, ntq, H, P);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (!fused) {
        launch_select(p, L, A, f32, P, ntq, cu_count, stream);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    // G2: y = A WT^T plus the layer's source (x for the residual, y for accumulation)
    const int64_t k2 = int64_t(P) * ntq;
    int out = GEMM_OUT_SRC_NONE;
    const void* src = nullptr;
    if (p.out_mode == OUT_RESIDUAL) {
        src = p.x;
        out = p.x_bf16 ? GEMM_OUT_SRC_BF16 : GEMM_OUT_SRC_F32;
    } else if (p.out_mode == OUT_ACCUMULATE) {
        src = p.y;
        out = p.y_bf16 ? GEMM_OUT_SRC_BF16 : GEMM_OUT_SRC_F32;
    }
    return gemm_nt(!f32, out, p.y_bf16, A, WT, p.y, src, B, H, k2, k2, k2, H, cu_count, SP, GEMM_SPLIT_BYTES, 0,
                   stream);
}

}  // namespace fff
