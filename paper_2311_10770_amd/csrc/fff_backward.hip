// fff_backward.hip -- gfx950 kernels for the backward of the FFF layer with
// the routing held fixed (hard routing): gradients flow only through the
// D+1 nodes each token visits in each tree (Section 2.1's layer; the branch
// decisions themselves carry no gradient).
//
// Per (token b, tree t, level l) with visited node n, saved logit l and
// a = act(l):
//     dW_out[t,n] += a * dy_b,   dl = <dy_b, W_out[t,n]> act'(l),
//     dW_in[t,n]  += dl * x_b,   dx_b += dl * W_in[t,n].
//
// 1. bwd_token_kernel (or bwd_generic_token_kernel): a group of lanes per
//    token, dy in registers; per level the two rows of the known path are
//    gathered, da is reduced across the group, dx accumulates in registers;
//    the pair (a, dl) of every visit is saved and the leaves are counted.
// 2. bwd_scan_kernel + bwd_scatter_kernel: counting sort of the tokens by
//    leaf.  Sorted by leaf, the tokens through any node form one contiguous
//    run at every level (a node's leaves are a contiguous range).
// 3. bwd_weight_kernel: each wave walks a stretch of sorted tokens for one
//    256-column slice, sums a*dy and dl*x per level in registers while the
//    node stays the same, and adds each finished run to dW with one fp32
//    atomic per element -- a handful of atomics per row and stretch instead
//    of one per token.
#include "fff_common.hpp"
#include "fff_device.hpp"
#include "fff_internal.hpp"

#include <hip/hip_runtime.h>

#include <algorithm>

namespace fff {

namespace {

enum { ST_OK_ = 0, ST_UNSUPPORTED_ = -2 };

constexpr int BWD_BLOCK = 256;
constexpr int SCAN_BLOCK = 1024;
constexpr int SLICE = 256;       // columns per wave in the weight kernel (64 lanes x 4)
constexpr int LV = 12;           // levels handled per pass of the weight kernel

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

__device__ __forceinline__ bool leaf_ok(int32_t leaf, int D) {
    const int64_t first = (int64_t(1) << D) - 1;
    return int64_t(leaf) >= first && int64_t(leaf) - first < (int64_t(1) << D);
}

// Output slice store for dx through the forward's store routine (y = dx).
template <int LANES, int NV, bool WBF, class XR>
__device__ __forceinline__ void store_dx(const BwdParams& p, const XR& any, float* acc, int64_t tok, int sl) {
    Params sp{};
    sp.y = p.dx;
    sp.y_bf16 = p.dx_bf16;
    sp.out_mode = p.accumulate ? OUT_ACCUMULATE : OUT_STORE;
    store_output<LANES, NV, WBF>(sp, any, acc, tok, sl);
}

// ---------------------------------------------------------------------------
// 1. token kernel
// ---------------------------------------------------------------------------

template <int LANES, int NV, bool WBF, int BLOCK>
__global__ __launch_bounds__(BLOCK) void bwd_token_kernel(BwdParams p) {
    using S = Shape<LANES, NV, false, WBF>;
    constexpr int WAVES = BLOCK / 64;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int sl = lane % LANES;
    const int sub = lane / LANES;
    const int T = p.n_trees, D = p.depth;
    const int64_t N = p.n_nodes;
    const int64_t L = int64_t(1) << D;
    const int64_t n_groups = (p.n_tokens + S::TPW - 1) / S::TPW;
    for (int64_t g = int64_t(blockIdx.x) * WAVES + wave; g < n_groups; g += int64_t(gridDim.x) * WAVES) {
        const int64_t slot_raw = g * S::TPW + sub;
        const bool valid = slot_raw < p.n_tokens;
        const int64_t tok = valid ? slot_raw : p.n_tokens - 1;
        XRegs<LANES, NV, false, WBF> gy;  // dy in the row layout
        gy.load_widen(p.dy, p.dy_bf16, tok, sl);
        float acc[S::E];
#pragma unroll
        for (int e = 0; e < S::E; ++e) acc[e] = 0.0f;
        for (int t = 0; t < T; ++t) {
            // An out-of-range leaf is replaced by the first leaf with zero weights, so the
            // wave stays convergent; nothing of it is stored.
            const int32_t leaf = p.leaves[tok * T + t];
            const bool ok = valid && leaf_ok(leaf, D);
            const uint32_t leaf1 = uint32_t(ok ? leaf : int32_t(L - 1)) + 1;
            if (sl == 0) {
                if (ok && p.need_dw) atomicAdd(&p.counts[t * L + (int64_t(leaf1) - L)], 1);
                if (valid && !ok && p.bad) atomicAdd(p.bad, 1);
            }
            const uint4* win = reinterpret_cast<const uint4*>(p.w_in) + int64_t(t) * N * S::ROWV + sl;
            const uint4* wout = reinterpret_cast<const uint4*>(p.w_out) + int64_t(t) * N * S::ROWV + sl;
            const int64_t rec0 = (tok * T + t) * (D + 1);
            for (int l = 0; l <= D; ++l) {
                const int64_t node = int64_t(leaf1 >> (D - l)) - 1;
                uint4 ro[NV], ri[NV];
#pragma unroll
                for (int c = 0; c < NV; ++c) ro[c] = wout[node * S::ROWV + c * LANES];
#pragma unroll
                for (int c = 0; c < NV; ++c) ri[c] = win[node * S::ROWV + c * LANES];
                const float logit = ok ? p.logits[rec0 + l] : 0.0f;
                const float da = group_sum<LANES>(gy.dot(ro));
                const float dl = ok ? da * activation_grad(logit, p.act) : 0.0f;
                axpy<NV, WBF>(acc, dl, ri);
                if (ok && sl == 0 && p.need_dw) p.coef[rec0 + l] = make_float2(activation(logit, p.act), dl);
            }
        }
        if (valid && p.dx) store_dx<LANES, NV, WBF>(p, gy, acc, tok, sl);
    }
}

template <bool BF>
__device__ __forceinline__ float load1(const void* base, int64_t i) {
    if constexpr (BF) return bf16_to_f32(reinterpret_cast<const uint16_t*>(base)[i]);
    else return reinterpret_cast<const float*>(base)[i];
}

__device__ __forceinline__ float load1r(const void* base, bool bf, int64_t i) {
    return bf ? load1<true>(base, i) : load1<false>(base, i);
}

// Any hidden size: one wave per token; first the pairs of every visit (kept
// in LDS), then dx one 64-column block at a time.
constexpr int BWD_GENERIC_MAX_PAIRS = 2048;

template <bool WBF>
__global__ __launch_bounds__(BWD_BLOCK) void bwd_generic_token_kernel(BwdParams p) {
    constexpr int WAVES = BWD_BLOCK / 64;
    extern __shared__ float bwd_generic_lds[];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int T = p.n_trees, D = p.depth, H = p.hidden;
    const int P = T * (D + 1);
    const int64_t N = p.n_nodes;
    const int64_t L = int64_t(1) << D;
    float* s_dl = bwd_generic_lds + wave * P;
    for (int64_t tok = int64_t(blockIdx.x) * WAVES + wave; tok < p.n_tokens; tok += int64_t(gridDim.x) * WAVES) {
        for (int t = 0; t < T; ++t) {
            const int32_t leaf = p.leaves[tok * T + t];
            const bool ok = leaf_ok(leaf, D);
            const uint32_t leaf1 = uint32_t(ok ? leaf : int32_t(L - 1)) + 1;
            if (lane == 0) {
                if (ok && p.need_dw) atomicAdd(&p.counts[t * L + (int64_t(leaf1) - L)], 1);
                if (!ok && p.bad) atomicAdd(p.bad, 1);
            }
            const int64_t rec0 = (tok * T + t) * (D + 1);
            for (int l = 0; l <= D; ++l) {
                const int64_t row = (int64_t(t) * N + (int64_t(leaf1 >> (D - l)) - 1)) * H;
                float part = 0.0f;
                for (int h = lane; h < H; h += 64)
                    part = __builtin_fmaf(load1r(p.dy, p.dy_bf16, tok * H + h), load1<WBF>(p.w_out, row + h), part);
                const float da = group_sum<64>(part);
                const float logit = ok ? p.logits[rec0 + l] : 0.0f;
                const float dl = ok ? da * activation_grad(logit, p.act) : 0.0f;
                if (lane == 0) {
                    s_dl[t * (D + 1) + l] = dl;
                    if (ok && p.need_dw) p.coef[rec0 + l] = make_float2(activation(logit, p.act), dl);
                }
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (p.dx) {
            for (int h0 = 0; h0 < H; h0 += 64) {
                const int h = h0 + lane;
                if (h >= H) continue;
                float acc = 0.0f;
                for (int t = 0; t < T; ++t) {
                    const int32_t leaf = p.leaves[tok * T + t];
                    const uint32_t leaf1 = uint32_t(leaf_ok(leaf, D) ? leaf : int32_t(L - 1)) + 1;
                    for (int l = 0; l <= D; ++l) {
                        const int64_t row = (int64_t(t) * N + (int64_t(leaf1 >> (D - l)) - 1)) * H;
                        acc = __builtin_fmaf(s_dl[t * (D + 1) + l], load1<WBF>(p.w_in, row + h), acc);
                    }
                }
                const int64_t i = tok * H + h;
                if (p.dx_bf16) {
                    uint16_t* d = reinterpret_cast<uint16_t*>(p.dx) + i;
                    if (p.accumulate) acc += bf16_to_f32(*d);
                    *d = f32_to_bf16(acc);
                } else {
                    float* d = reinterpret_cast<float*>(p.dx) + i;
                    if (p.accumulate) acc += *d;
                    *d = acc;
                }
            }
        }
        __builtin_amdgcn_wave_barrier();  // s_dl is rewritten by the next token
    }
}

// ---------------------------------------------------------------------------
// 2. counting sort by leaf
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(BWD_BLOCK) void bwd_fill_kernel(float* a, int64_t n4, int32_t* b, int64_t nb) {
    const int64_t stride = int64_t(gridDim.x) * BWD_BLOCK;
    float4* a4 = reinterpret_cast<float4*>(a);
    for (int64_t i = int64_t(blockIdx.x) * BWD_BLOCK + threadIdx.x; i < n4; i += stride)
        a4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int64_t i = int64_t(blockIdx.x) * BWD_BLOCK + threadIdx.x; i < nb; i += stride) b[i] = 0;
}

// Exclusive prefix sums of one tree's leaf counts (block t), and the tree's total.
__global__ __launch_bounds__(SCAN_BLOCK) void bwd_scan_kernel(BwdParams p) {
    constexpr int PER = 4;
    constexpr int WAVES = SCAN_BLOCK / 64;
    __shared__ int32_t wave_tot[WAVES];
    __shared__ int32_t carry_s;
    const int t = blockIdx.x;
    const int64_t L = int64_t(1) << p.depth;
    const int32_t* c = p.counts + t * L;
    int32_t* o = p.offs + t * L;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    if (tid == 0) carry_s = 0;
    __syncthreads();
    for (int64_t base = 0; base < L; base += int64_t(SCAN_BLOCK) * PER) {
        int32_t v[PER];
        int32_t s = 0;
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int64_t i = base + int64_t(tid) * PER + j;
            v[j] = i < L ? c[i] : 0;
            s += v[j];
        }
        // inclusive scan of s over the wave
        int32_t inc = s;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int32_t u = __shfl_up(inc, d, 64);
            if (lane >= d) inc += u;
        }
        if (lane == 63) wave_tot[wave] = inc;
        __syncthreads();
        int32_t before = carry_s;
        for (int w = 0; w < wave; ++w) before += wave_tot[w];
        int32_t run = before + inc - s;  // exclusive prefix of this thread's first element
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int64_t i = base + int64_t(tid) * PER + j;
            if (i < L) o[i] = run;
            run += v[j];
        }
        __syncthreads();  // everyone has read carry_s and wave_tot
        if (tid == SCAN_BLOCK - 1) carry_s = run;
        __syncthreads();
    }
    if (tid == 0) p.total[t] = carry_s;
}

// Sorted position of every valid (token, tree): perm[t][offs[leaf]++] = token.
__global__ __launch_bounds__(BWD_BLOCK) void bwd_scatter_kernel(BwdParams p) {
    const int T = p.n_trees, D = p.depth;
    const int64_t L = int64_t(1) << D;
    const int64_t n = p.n_tokens * T;
    for (int64_t i = int64_t(blockIdx.x) * BWD_BLOCK + threadIdx.x; i < n; i += int64_t(gridDim.x) * BWD_BLOCK) {
        const int64_t b = i / T;
        const int t = int(i % T);
        const int32_t leaf = p.leaves[i];
        if (!leaf_ok(leaf, D)) continue;
        const int64_t bin = int64_t(leaf) - (L - 1);
        const int32_t pos = atomicAdd(&p.offs[t * L + bin], 1);
        p.perm[int64_t(t) * p.n_tokens + pos] = int32_t(b);
    }
}

// ---------------------------------------------------------------------------
// 3. weight kernel
// ---------------------------------------------------------------------------

__device__ __forceinline__ float4 load4(const void* base, bool bf, int64_t i) {
    if (bf) {
        const uint2 u = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint16_t*>(base) + i);
        return make_float4(bf16_lo(u.x), bf16_hi(u.x), bf16_lo(u.y), bf16_hi(u.y));
    }
    return *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(base) + i);
}

__device__ __forceinline__ void flush_row(float* dw, int64_t row, int col, bool active, const float* v) {
    if (!dw || !active) return;
#pragma unroll
    for (int k = 0; k < 4; ++k) unsafeAtomicAdd(dw + row + col + k, v[k]);
}

__global__ __launch_bounds__(BWD_BLOCK) void bwd_weight_kernel(BwdParams p) {
    const int lane = threadIdx.x & 63;
    const int64_t wid = int64_t(blockIdx.x) * (BWD_BLOCK / 64) + (threadIdx.x >> 6);
    const int T = p.n_trees, D = p.depth, H = p.hidden;
    const int64_t N = p.n_nodes;
    const int slices = (H + SLICE - 1) / SLICE;
    const int64_t chunks = (p.n_tokens + p.chunk - 1) / p.chunk;
    const int64_t per_tree = chunks * slices;
    if (wid >= per_tree * T) return;  // whole wave
    const int t = int(wid / per_tree);
    const int64_t r = wid % per_tree;
    const int s = int(r % slices);
    const int64_t c = r / slices;
    const int64_t total = p.total[t];
    const int64_t p0 = c * p.chunk;
    const int64_t p1 = std::min<int64_t>(p0 + p.chunk, total);
    if (p0 >= p1) return;
    const int col = s * SLICE + lane * 4;
    const bool active = col < H;  // H is a multiple of 4
    const int32_t* perm = p.perm + int64_t(t) * p.n_tokens;
    for (int l0 = 0; l0 <= D; l0 += LV) {
        int64_t cur[LV];
        float ao[LV][4], ai[LV][4];
#pragma unroll
        for (int j = 0; j < LV; ++j) {
            cur[j] = -1;
#pragma unroll
            for (int k = 0; k < 4; ++k) ao[j][k] = ai[j][k] = 0.0f;
        }
        for (int64_t q = p0; q < p1; ++q) {
            const int64_t b = perm[q];
            const uint32_t leaf1 = uint32_t(p.leaves[b * T + t]) + 1;
            float4 gy = make_float4(0.f, 0.f, 0.f, 0.f), xv = gy;
            if (active) {
                gy = load4(p.dy, p.dy_bf16, b * H + col);
                xv = load4(p.x, p.x_bf16, b * H + col);
            }
            const float2* cf = p.coef + (b * T + t) * (D + 1);
#pragma unroll
            for (int j = 0; j < LV; ++j) {
                const int l = l0 + j;
                if (l > D) break;
                const int64_t node = int64_t(leaf1 >> (D - l)) - 1;
                if (node != cur[j]) {  // a run ends (wave-uniform)
                    if (cur[j] >= 0) {
                        const int64_t row = (int64_t(t) * N + cur[j]) * H;
                        flush_row(p.dw_out, row, col, active, ao[j]);
                        flush_row(p.dw_in, row, col, active, ai[j]);
                    }
                    cur[j] = node;
#pragma unroll
                    for (int k = 0; k < 4; ++k) ao[j][k] = ai[j][k] = 0.0f;
                }
                const float2 cc = cf[l];
                ao[j][0] = __builtin_fmaf(cc.x, gy.x, ao[j][0]);
                ao[j][1] = __builtin_fmaf(cc.x, gy.y, ao[j][1]);
                ao[j][2] = __builtin_fmaf(cc.x, gy.z, ao[j][2]);
                ao[j][3] = __builtin_fmaf(cc.x, gy.w, ao[j][3]);
                ai[j][0] = __builtin_fmaf(cc.y, xv.x, ai[j][0]);
                ai[j][1] = __builtin_fmaf(cc.y, xv.y, ai[j][1]);
                ai[j][2] = __builtin_fmaf(cc.y, xv.z, ai[j][2]);
                ai[j][3] = __builtin_fmaf(cc.y, xv.w, ai[j][3]);
            }
        }
#pragma unroll
        for (int j = 0; j < LV; ++j) {
            if (l0 + j > D) break;
            if (cur[j] >= 0) {
                const int64_t row = (int64_t(t) * N + cur[j]) * H;
                flush_row(p.dw_out, row, col, active, ao[j]);
                flush_row(p.dw_in, row, col, active, ai[j]);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// planning
// ---------------------------------------------------------------------------

struct BwdVariant {
    int hidden;
    bool wbf;
    int lanes;
    const void* token;
};

#define FFF_BWD(H, WB, L, NV) \
    BwdVariant { H, WB, L, reinterpret_cast<const void*>(&bwd_token_kernel<L, NV, WB, BWD_BLOCK>) }

const BwdVariant kBwdVariants[] = {
    FFF_BWD(768, true, 16, 6),  FFF_BWD(768, false, 32, 6),  FFF_BWD(1024, true, 16, 8),
    FFF_BWD(1024, false, 32, 8), FFF_BWD(4096, true, 64, 8), FFF_BWD(4096, false, 64, 16),
};

int resident_blocks(const void* kernel, size_t lds) {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, BWD_BLOCK, lds) != hipSuccess || n < 1) n = 1;
    return n;
}

}  // namespace

size_t bwd_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees) {
    const size_t recs = size_t(n_tokens) * size_t(n_trees);
    const size_t bins = (size_t(1) << depth) * size_t(n_trees);
    return align256(recs * size_t(depth + 1) * sizeof(float2)) + 2 * align256(bins * sizeof(int32_t)) +
           align256(recs * sizeof(int32_t)) + align256(size_t(n_trees) * sizeof(int32_t));
}

void bwd_workspace_views(BwdParams& p, void* workspace) {
    char* w = static_cast<char*>(workspace);
    const size_t recs = size_t(p.n_tokens) * size_t(p.n_trees);
    const size_t bins = (size_t(1) << p.depth) * size_t(p.n_trees);
    p.coef = reinterpret_cast<float2*>(w);
    w += align256(recs * size_t(p.depth + 1) * sizeof(float2));
    p.counts = reinterpret_cast<int32_t*>(w);
    w += align256(bins * sizeof(int32_t));
    p.offs = reinterpret_cast<int32_t*>(w);
    w += align256(bins * sizeof(int32_t));
    p.perm = reinterpret_cast<int32_t*>(w);
    w += align256(recs * sizeof(int32_t));
    p.total = reinterpret_cast<int32_t*>(w);
}

hipError_t run_backward(BwdParams p, const DeviceInfo& dev, hipStream_t stream, int* status) {
    *status = ST_OK_;
    const BwdVariant* v = nullptr;
    for (const auto& c : kBwdVariants)
        if (c.hidden == p.hidden && c.wbf == bool(p.w_bf16)) v = &c;
    const int pairs = p.n_trees * (p.depth + 1);
    if (!v && pairs > BWD_GENERIC_MAX_PAIRS) {
        *status = ST_UNSUPPORTED_;
        return hipSuccess;
    }
    void* args[] = {&p};
    const int64_t bins = (int64_t(1) << p.depth) * p.n_trees;
    const int64_t dw4 = p.n_trees * p.n_nodes * p.hidden / 4;
    // zero the leaf counts, and dW unless accumulating (a fill kernel: no memset nodes)
    {
        const int64_t n4 = p.accumulate ? 0 : dw4;
        const int64_t work = std::max<int64_t>(n4, p.need_dw ? bins : 0);
        if (work > 0) {
            const int grid = int(std::min<int64_t>((work + BWD_BLOCK - 1) / BWD_BLOCK, int64_t(dev.cu_count) * 8));
            for (float* dw : {p.dw_in, p.dw_out}) {
                if (!dw || p.accumulate) continue;
                float* a = dw;
                int64_t na = dw4;
                int32_t* b = nullptr;
                int64_t nb = 0;
                void* fa[] = {&a, &na, &b, &nb};
                const hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_fill_kernel), dim3(grid),
                                                     dim3(BWD_BLOCK), fa, 0, stream);
                if (e != hipSuccess) return e;
            }
            if (p.need_dw) {
                float* a = nullptr;
                int64_t na = 0;
                int32_t* b = p.counts;
                int64_t nb = bins;
                void* fa[] = {&a, &na, &b, &nb};
                const hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_fill_kernel), dim3(grid),
                                                     dim3(BWD_BLOCK), fa, 0, stream);
                if (e != hipSuccess) return e;
            }
        }
    }
    // token kernel
    {
        const void* k;
        size_t lds = 0;
        int64_t want;
        if (v) {
            k = v->token;
            const int64_t groups = (p.n_tokens + 64 / v->lanes - 1) / (64 / v->lanes);
            want = (groups + BWD_BLOCK / 64 - 1) / (BWD_BLOCK / 64);
        } else {
            k = p.w_bf16 ? reinterpret_cast<const void*>(&bwd_generic_token_kernel<true>)
                         : reinterpret_cast<const void*>(&bwd_generic_token_kernel<false>);
            lds = size_t(BWD_BLOCK / 64) * size_t(pairs) * sizeof(float);
            want = (p.n_tokens + BWD_BLOCK / 64 - 1) / (BWD_BLOCK / 64);
        }
        const int64_t resident = int64_t(dev.cu_count) * resident_blocks(k, lds);
        const int grid = int(std::max<int64_t>(1, std::min(want, resident)));
        const hipError_t e = hipLaunchKernel(k, dim3(grid), dim3(BWD_BLOCK), args, lds, stream);
        if (e != hipSuccess) return e;
    }
    if (!p.need_dw) return hipSuccess;
    hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_scan_kernel), dim3(p.n_trees), dim3(SCAN_BLOCK),
                                   args, 0, stream);
    if (e != hipSuccess) return e;
    {
        const int64_t n = p.n_tokens * p.n_trees;
        const int grid = int(std::min<int64_t>((n + BWD_BLOCK - 1) / BWD_BLOCK, int64_t(dev.cu_count) * 8));
        e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_scatter_kernel), dim3(grid), dim3(BWD_BLOCK), args, 0,
                            stream);
        if (e != hipSuccess) return e;
    }
    {
        // about four waves per SIMD over all slices and trees
        const int slices = (p.hidden + SLICE - 1) / SLICE;
        const int64_t target = int64_t(dev.cu_count) * 16;
        const int64_t chunks = std::max<int64_t>(1, target / (int64_t(slices) * p.n_trees));
        p.chunk = int32_t(std::max<int64_t>(16, (p.n_tokens + chunks - 1) / chunks));
        const int64_t waves = ((p.n_tokens + p.chunk - 1) / p.chunk) * slices * p.n_trees;
        const int64_t grid = (waves + BWD_BLOCK / 64 - 1) / (BWD_BLOCK / 64);
        void* wargs[] = {&p};
        e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_weight_kernel), dim3(unsigned(grid)), dim3(BWD_BLOCK),
                            wargs, 0, stream);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace fff
