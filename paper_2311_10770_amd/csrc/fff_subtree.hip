// fff_subtree.hip -- SUBTREE mode: the FFF forward for a handful of tokens,
// where the time is the chain of D+1 dependent row gathers of Algorithm 1
// (each level's row is known only once the previous logit's sign is).
//
// One workgroup of 16 (or 8) waves per token.  Each lane group (LANES lanes, the
// layout of the other modes) computes one node's logit per step, so a step
// evaluates every node of the SPAN-level subtree below the current node at once
// (2^SPAN - 1 <= waves * 64 / LANES dot products, all rows loaded together); the
// token then descends SPAN levels through those logits in LDS.  The walk thus
// costs ceil((D+1) / SPAN) memory round trips instead of D+1, at the price of
// reading (2^SPAN - 1) / SPAN times the W_in rows -- which only a small batch
// can afford.  The path's W_out rows are then independent: every thread owns
// one 16-byte column vector and loads its slice of all D+1 rows together.
// The logits are the same dot products, in the same order and reduction, as in
// the other modes, so the branches, records and outputs agree with them.
#include "fff_common.hpp"
#include "fff_device.hpp"
#include "fff_internal.hpp"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

namespace fff {

namespace {

constexpr int SUB_MAX_LEVELS = 25;  // depth <= 24

// Waves per token: 16, or 8 where fp32 x against bf16 W (x alone takes 64 registers) would not fit
// the 128 registers a lane has at 16 waves per workgroup.
constexpr int sub_waves(int nv, bool xbf, bool wbf) { return (!xbf && wbf && nv >= 8) ? 8 : 16; }

constexpr int span_for(int groups) {
    int s = 0;
    while ((2 << s) - 1 <= groups) ++s;  // largest s with 2^s - 1 <= groups
    return s;
}

// y columns [c0, c0 + EV) of token tok from the fp32 sums (residual / accumulate applied).
template <int EV, bool XBF>
__device__ __forceinline__ void store_cols(const Params& p, float* v, int64_t tok, int64_t c0) {
    const int64_t e0 = tok * p.hidden + c0;
    if (p.out_mode == OUT_RESIDUAL) {
        if constexpr (XBF) {
            const uint16_t* xs = static_cast<const uint16_t*>(p.x) + e0;
            if constexpr (EV == 8) {
                const uint4 u = *reinterpret_cast<const uint4*>(xs);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    v[2 * j] += bf16_lo(word(u, j));
                    v[2 * j + 1] += bf16_hi(word(u, j));
                }
            } else {
                const uint2 u = *reinterpret_cast<const uint2*>(xs);
                v[0] += bf16_lo(u.x); v[1] += bf16_hi(u.x); v[2] += bf16_lo(u.y); v[3] += bf16_hi(u.y);
            }
        } else {
            const float4* xs = reinterpret_cast<const float4*>(static_cast<const float*>(p.x) + e0);
#pragma unroll
            for (int q = 0; q < EV / 4; ++q) {
                const float4 a = xs[q];
                v[4 * q] += a.x; v[4 * q + 1] += a.y; v[4 * q + 2] += a.z; v[4 * q + 3] += a.w;
            }
        }
    }
    if (p.y_bf16) {
        uint16_t* ys = static_cast<uint16_t*>(p.y) + e0;
        if constexpr (EV == 8) {
            uint4* d = reinterpret_cast<uint4*>(ys);
            if (p.out_mode == OUT_ACCUMULATE) {
                const uint4 o = *d;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    v[2 * j] += bf16_lo(word(o, j));
                    v[2 * j + 1] += bf16_hi(word(o, j));
                }
            }
            *d = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                            pack_bf16x2(v[6], v[7]));
        } else {
            uint2* d = reinterpret_cast<uint2*>(ys);
            if (p.out_mode == OUT_ACCUMULATE) {
                const uint2 o = *d;
                v[0] += bf16_lo(o.x); v[1] += bf16_hi(o.x); v[2] += bf16_lo(o.y); v[3] += bf16_hi(o.y);
            }
            *d = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
        }
    } else {
        float4* d = reinterpret_cast<float4*>(static_cast<float*>(p.y) + e0);
#pragma unroll
        for (int q = 0; q < EV / 4; ++q) {
            float4 a = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
            if (p.out_mode == OUT_ACCUMULATE) {
                const float4 o = d[q];
                a.x += o.x; a.y += o.y; a.z += o.z; a.w += o.w;
            }
            d[q] = a;
        }
    }
}

template <int LANES, int NV, bool XBF, bool WBF, int BLOCK>
__global__ __launch_bounds__(BLOCK) void subtree_kernel(Params p) {
    using S = Shape<LANES, NV, XBF, WBF>;
    constexpr int GROUPS = BLOCK / 64 * S::TPW;  // node logits per step
    constexpr int SPAN = span_for(GROUPS);       // levels per step
    static_assert(S::ROWV <= BLOCK, "one 16-byte column vector per thread");
    __shared__ float s_logit[2][GROUPS];
    __shared__ int32_t s_node[SUB_MAX_LEVELS];
    __shared__ float s_val[SUB_MAX_LEVELS];  // logit, then activation, of each level

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int sl = lane % LANES;
    const int g = (tid >> 6) * S::TPW + lane / LANES;  // this group's node slot
    const int T = p.n_trees, D = p.depth;
    const int64_t N = p.n_nodes;
    int buf = 0;
    for (int64_t tok = blockIdx.x; tok < p.n_tokens; tok += gridDim.x) {
        XRegs<LANES, NV, XBF, WBF> xr;
        xr.load(p.x, tok, sl);
        float acc[S::EV];
#pragma unroll
        for (int e = 0; e < S::EV; ++e) acc[e] = 0.0f;
        for (int t = 0; t < T; ++t) {
            const uint4* win = reinterpret_cast<const uint4*>(p.w_in) + int64_t(t) * N * S::ROWV + sl;
            uint32_t n = 0;  // current node, the same in every thread
            for (int l = 0; l <= D; l += SPAN) {
                const int s = min(SPAN, D + 1 - l);
                const int m = (1 << s) - 1;
                // slot g holds the subtree node of relative heap index r (level k below n, offset j);
                // idle slots recompute the subtree root so that every group loads
                const int r = g < m ? g : 0;
                const int k = 31 - __builtin_clz(uint32_t(r + 1));
                const uint32_t node = ((n + 1) << k) - 1 + uint32_t(r - ((1 << k) - 1));
                const uint4* row = win + int64_t(node) * S::ROWV;
                uint4 w[NV];
#pragma unroll
                for (int c = 0; c < NV; ++c) w[c] = row[c * LANES];
                const float logit = group_sum<LANES>(xr.dot(w));
                if (g < m && sl == 0) s_logit[buf][g] = logit;
                __syncthreads();
                // descend s levels through the subtree's logits
                int rel = 0;
                for (int q = 0; q < s; ++q) {
                    const float lg = s_logit[buf][rel];
                    if (tid == 0) {
                        s_node[l + q] = int32_t(n);
                        s_val[l + q] = lg;
                    }
                    const uint32_t bit = lg > 0.0f ? 1u : 0u;
                    if (l + q < D) n = 2 * n + 1 + bit;
                    rel = 2 * rel + 1 + int(bit);
                }
                buf ^= 1;
            }
            __syncthreads();
            if (tid <= D) {
                const float lg = s_val[tid];
                const int64_t rec = (tok * T + t) * (D + 1) + tid;
                if (p.nodes_out) p.nodes_out[rec] = s_node[tid];
                if (p.logits_out) p.logits_out[rec] = lg;
                s_val[tid] = activation(lg, p.act);
            }
            __syncthreads();
            // the path's W_out rows, this thread's 16-byte column vector of each, eight loads in flight
            constexpr int EB = 8;
            if (tid < S::ROWV) {
                const uint4* wo = reinterpret_cast<const uint4*>(p.w_out) + int64_t(t) * N * S::ROWV + tid;
                for (int l0 = 0; l0 <= D; l0 += EB) {
                    uint4 wv[EB];
#pragma unroll
                    for (int j = 0; j < EB; ++j) wv[j] = wo[int64_t(s_node[min(l0 + j, D)]) * S::ROWV];
#pragma unroll
                    for (int j = 0; j < EB; ++j)
                        if (l0 + j <= D) axpy<1, WBF>(acc, s_val[l0 + j], &wv[j]);
                }
            }
        }
        if (tid < S::ROWV) store_cols<S::EV, XBF>(p, acc, tok, int64_t(tid) * S::EV);
    }
}

struct SubtreeVariant {
    int hidden;
    bool xbf, wbf;
    const void* kernel;
    int block;
    int span;
    const char* name;
};

#define FFF_SUB(H, XB, WB, L, NV)                                                                             \
    SubtreeVariant {                                                                                          \
        H, XB, WB, reinterpret_cast<const void*>(&subtree_kernel<L, NV, XB, WB, 64 * sub_waves(NV, XB, WB)>), \
            64 * sub_waves(NV, XB, WB), span_for(sub_waves(NV, XB, WB) * 64 / L),                             \
            "lanes=" #L ",nv=" #NV ",x_bf16=" #XB ",w_bf16=" #WB                                              \
    }

// the lane layouts of the other modes' instantiations
const SubtreeVariant kSubtree[] = {
    FFF_SUB(768, true, true, 16, 6),    FFF_SUB(768, false, true, 16, 6),   FFF_SUB(768, false, false, 32, 6),
    FFF_SUB(768, true, false, 32, 6),   FFF_SUB(1024, true, true, 16, 8),   FFF_SUB(1024, false, true, 16, 8),
    FFF_SUB(1024, false, false, 32, 8), FFF_SUB(1024, true, false, 32, 8),  FFF_SUB(4096, true, true, 64, 8),
    FFF_SUB(4096, false, true, 64, 8),  FFF_SUB(4096, false, false, 64, 16), FFF_SUB(4096, true, false, 64, 16),
};

const SubtreeVariant* find_subtree(const Params& p) {
    for (const auto& v : kSubtree)
        if (v.hidden == p.hidden && v.xbf == bool(p.x_bf16) && v.wbf == bool(p.w_bf16)) return &v;
    return nullptr;
}

}  // namespace

bool subtree_shape(const Params& p) { return !p.norm && p.depth < SUB_MAX_LEVELS && find_subtree(p) != nullptr; }

int subtree_span(const Params& p) {
    const SubtreeVariant* v = find_subtree(p);
    return v ? v->span : 0;
}

const char* subtree_name(const Params& p) {
    const SubtreeVariant* v = find_subtree(p);
    return v ? v->name : "";
}

bool subtree_auto(const Params& p) {
    if (!subtree_shape(p) || p.depth < SUBTREE_AUTO_DEPTH || p.n_trees > SUBTREE_AUTO_TREES) return false;
    const int64_t pairs = p.hidden > 1024                           ? SUBTREE_AUTO_PAIRS_WIDE
                          : !p.w_bf16 && p.depth >= SUBTREE_DEEP_F32 ? SUBTREE_AUTO_PAIRS_DEEP_F32
                                                                     : SUBTREE_AUTO_PAIRS;
    return p.n_tokens * p.n_trees <= pairs;
}

int subtree_block(const Params& p) {
    const SubtreeVariant* v = find_subtree(p);
    return v ? v->block : 0;
}

int subtree_grid(const Params& p, int cu_count) {
    return int(std::max<int64_t>(1, std::min<int64_t>(p.n_tokens, int64_t(cu_count) * 4)));
}

hipError_t run_subtree(const Params& p, int grid, hipStream_t stream) {
    const SubtreeVariant* v = find_subtree(p);
    if (!v) return hipErrorNotSupported;
    void* args[] = {const_cast<Params*>(&p)};
    return hipLaunchKernel(v->kernel, dim3(unsigned(grid)), dim3(unsigned(v->block)), args, 0, stream);
}

}  // namespace fff
