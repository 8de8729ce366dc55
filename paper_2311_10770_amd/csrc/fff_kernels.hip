// fff_kernels.hip -- gfx950 kernels for FFF inference (conditional matrix
// multiplication, Algorithm 1 of the paper, with the Section 2.1 model:
// activation and output row at every visited node, trees summed).
//
// descent_kernel: a group of LANES lanes (16, 32 or 64) owns one token.  The
//   token's x slice and its fp32 output accumulators stay in registers for the
//   whole walk; each level gathers one W_in row and one W_out row (16-byte
//   vector loads, LANES*16 contiguous bytes per instruction), reduces the dot
//   product across the group with DPP / permlane swaps, and picks the child.
//   The top lds_levels levels of every tree are staged once per workgroup into
//   LDS (the paper's advice to preload the weights of the sub-trees a token
//   will need, Section 3.2).  Grid-stride over token groups.
// generic_kernel: any hidden size; one wave per token; logits first, with the
//   visited (node, activation) pairs kept in LDS, then the output rows summed
//   one 64-element column block at a time.
#include "fff_device.hpp"
#include "fff_internal.hpp"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <tuple>

namespace fff {

enum { OUT_STORE = 0, OUT_ACCUMULATE = 1, OUT_RESIDUAL = 2 };
enum { MODE_AUTO = 0, MODE_DESCENT = 1, MODE_GROUPED = 2, MODE_GENERIC = 3 };
// status values mirrored from fff.h
enum { ST_OK = 0, ST_INVALID = -1, ST_UNSUPPORTED = -2, ST_WORKSPACE = -3 };

// ----------------------------------------------------------------------------
// descent kernel
// ----------------------------------------------------------------------------

template <int LANES, int NV, bool XBF, bool WBF>
struct Shape {
    static constexpr int EV = WBF ? 8 : 4;  // W elements per 16-byte vector
    static constexpr int E = NV * EV;       // elements a lane owns
    static constexpr int H = LANES * E;     // hidden size
    static constexpr int TPW = 64 / LANES;  // tokens per wave
    static constexpr int ROWV = LANES * NV; // 16-byte vectors per W row
};

// Lane sl of a group owns, for c = 0..NV-1, the EV consecutive elements
// starting at element (c*LANES + sl)*EV: every load instruction covers one
// contiguous LANES*16-byte span of the row.
template <int LANES, int NV, bool XBF, bool WBF>
struct XRegs;

template <int LANES, int NV>
struct XRegs<LANES, NV, true, true> {  // bf16 x with bf16 W: keep packed pairs for dot2
    uint4 v[NV];
    __device__ void load(const void* x, int64_t tok, int sl) {
        const uint4* row = reinterpret_cast<const uint4*>(x) + tok * (LANES * NV);
#pragma unroll
        for (int c = 0; c < NV; ++c) v[c] = row[c * LANES + sl];
    }
    __device__ float dot(const uint4* w) const {
        float s = 0.0f;
#pragma unroll
        for (int c = 0; c < NV; ++c) {
            s = dot2_bf16(v[c].x, w[c].x, s);
            s = dot2_bf16(v[c].y, w[c].y, s);
            s = dot2_bf16(v[c].z, w[c].z, s);
            s = dot2_bf16(v[c].w, w[c].w, s);
        }
        return s;
    }
    __device__ float elem(int c, int e) const {
        const uint32_t u = word(v[c], e >> 1);
        return (e & 1) ? bf16_hi(u) : bf16_lo(u);
    }
};

template <int LANES, int NV>
struct XRegs<LANES, NV, false, true> {  // fp32 x with bf16 W
    float f[NV * 8];
    __device__ void load(const void* x, int64_t tok, int sl) {
        const float4* row = reinterpret_cast<const float4*>(x) + tok * (LANES * NV * 2);
#pragma unroll
        for (int c = 0; c < NV; ++c) {
            const float4 a = row[(c * LANES + sl) * 2], b = row[(c * LANES + sl) * 2 + 1];
            f[c * 8 + 0] = a.x; f[c * 8 + 1] = a.y; f[c * 8 + 2] = a.z; f[c * 8 + 3] = a.w;
            f[c * 8 + 4] = b.x; f[c * 8 + 5] = b.y; f[c * 8 + 6] = b.z; f[c * 8 + 7] = b.w;
        }
    }
    __device__ float dot(const uint4* w) const {
        float s = 0.0f;
#pragma unroll
        for (int c = 0; c < NV; ++c)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t u = word(w[c], j);
                s = __builtin_fmaf(f[c * 8 + 2 * j], bf16_lo(u), s);
                s = __builtin_fmaf(f[c * 8 + 2 * j + 1], bf16_hi(u), s);
            }
        return s;
    }
    __device__ float elem(int c, int e) const { return f[c * 8 + e]; }
};

template <int LANES, int NV, bool XBF>
struct XRegsF32W {  // fp32 W: x held as fp32 (bf16 x widened once)
    float f[NV * 4];
    __device__ void load(const void* x, int64_t tok, int sl) {
        if constexpr (XBF) {
            const uint2* row = reinterpret_cast<const uint2*>(x) + tok * (LANES * NV);
#pragma unroll
            for (int c = 0; c < NV; ++c) {
                const uint2 a = row[c * LANES + sl];
                f[c * 4 + 0] = bf16_lo(a.x); f[c * 4 + 1] = bf16_hi(a.x);
                f[c * 4 + 2] = bf16_lo(a.y); f[c * 4 + 3] = bf16_hi(a.y);
            }
        } else {
            const float4* row = reinterpret_cast<const float4*>(x) + tok * (LANES * NV);
#pragma unroll
            for (int c = 0; c < NV; ++c) {
                const float4 a = row[c * LANES + sl];
                f[c * 4 + 0] = a.x; f[c * 4 + 1] = a.y; f[c * 4 + 2] = a.z; f[c * 4 + 3] = a.w;
            }
        }
    }
    __device__ float dot(const uint4* w) const {
        float s = 0.0f;
#pragma unroll
        for (int c = 0; c < NV; ++c)
#pragma unroll
            for (int j = 0; j < 4; ++j) s = __builtin_fmaf(f[c * 4 + j], __uint_as_float(word(w[c], j)), s);
        return s;
    }
    __device__ float elem(int c, int e) const { return f[c * 4 + e]; }
};
template <int LANES, int NV>
struct XRegs<LANES, NV, false, false> : XRegsF32W<LANES, NV, false> {};
template <int LANES, int NV>
struct XRegs<LANES, NV, true, false> : XRegsF32W<LANES, NV, true> {};

template <int NV, bool WBF>
__device__ __forceinline__ void axpy(float* acc, float a, const uint4* w) {
#pragma unroll
    for (int c = 0; c < NV; ++c) {
        if constexpr (WBF) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t u = word(w[c], j);
                acc[c * 8 + 2 * j] = __builtin_fmaf(a, bf16_lo(u), acc[c * 8 + 2 * j]);
                acc[c * 8 + 2 * j + 1] = __builtin_fmaf(a, bf16_hi(u), acc[c * 8 + 2 * j + 1]);
            }
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[c * 4 + j] = __builtin_fmaf(a, __uint_as_float(word(w[c], j)), acc[c * 4 + j]);
        }
    }
}

// Final combine and store of one token's output slice.
template <int LANES, int NV, bool XBF, bool WBF>
__device__ __forceinline__ void store_output(const Params& p, const XRegs<LANES, NV, XBF, WBF>& xr, float* acc,
                                             int64_t tok, int sl) {
    using S = Shape<LANES, NV, XBF, WBF>;
    constexpr int EV = S::EV;
    if (p.out_mode == OUT_RESIDUAL) {
#pragma unroll
        for (int c = 0; c < NV; ++c)
#pragma unroll
            for (int e = 0; e < EV; ++e) acc[c * EV + e] += xr.elem(c, e);
    }
    if (p.y_bf16) {
        uint16_t* yrow = reinterpret_cast<uint16_t*>(p.y) + tok * S::H;
#pragma unroll
        for (int c = 0; c < NV; ++c) {
            uint16_t* dst = yrow + (c * LANES + sl) * EV;
            if constexpr (EV == 8) {
                uint4* d = reinterpret_cast<uint4*>(dst);
                if (p.out_mode == OUT_ACCUMULATE) {
                    const uint4 o = *d;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const uint32_t u = word(o, j);
                        acc[c * 8 + 2 * j] += bf16_lo(u);
                        acc[c * 8 + 2 * j + 1] += bf16_hi(u);
                    }
                }
                *d = make_uint4(pack_bf16x2(acc[c * 8 + 0], acc[c * 8 + 1]), pack_bf16x2(acc[c * 8 + 2], acc[c * 8 + 3]),
                                pack_bf16x2(acc[c * 8 + 4], acc[c * 8 + 5]), pack_bf16x2(acc[c * 8 + 6], acc[c * 8 + 7]));
            } else {
                uint2* d = reinterpret_cast<uint2*>(dst);
                if (p.out_mode == OUT_ACCUMULATE) {
                    const uint2 o = *d;
                    acc[c * 4 + 0] += bf16_lo(o.x); acc[c * 4 + 1] += bf16_hi(o.x);
                    acc[c * 4 + 2] += bf16_lo(o.y); acc[c * 4 + 3] += bf16_hi(o.y);
                }
                *d = make_uint2(pack_bf16x2(acc[c * 4 + 0], acc[c * 4 + 1]), pack_bf16x2(acc[c * 4 + 2], acc[c * 4 + 3]));
            }
        }
    } else {
        float* yrow = reinterpret_cast<float*>(p.y) + tok * S::H;
#pragma unroll
        for (int c = 0; c < NV; ++c) {
            float4* d = reinterpret_cast<float4*>(yrow + (c * LANES + sl) * EV);
#pragma unroll
            for (int q = 0; q < EV / 4; ++q) {
                float4 v = make_float4(acc[c * EV + 4 * q], acc[c * EV + 4 * q + 1], acc[c * EV + 4 * q + 2],
                                       acc[c * EV + 4 * q + 3]);
                if (p.out_mode == OUT_ACCUMULATE) {
                    const float4 o = d[q];
                    v.x += o.x; v.y += o.y; v.z += o.z; v.w += o.w;
                }
                d[q] = v;
            }
        }
    }
}

template <int LANES, int NV, bool XBF, bool WBF, int BLOCK>
__global__ __launch_bounds__(BLOCK) void descent_kernel(Params p) {
    using S = Shape<LANES, NV, XBF, WBF>;
    constexpr int WAVES = BLOCK / 64;
    extern __shared__ uint4 lds_rows[];  // [T][Nk][2][ROWV]: W_in row then W_out row

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int sl = lane % LANES;
    const int sub = lane / LANES;
    const int T = p.n_trees;
    const int D = p.depth;
    const int K = p.lds_levels;
    const int64_t N = p.n_nodes;
    const int64_t Nk = (int64_t(1) << K) - 1;

    if (K > 0) {
        const int64_t total = int64_t(T) * Nk * 2 * S::ROWV;
        const uint4* win = reinterpret_cast<const uint4*>(p.w_in);
        const uint4* wout = reinterpret_cast<const uint4*>(p.w_out);
        for (int64_t i = tid; i < total; i += BLOCK) {
            const int64_t v = i % S::ROWV;
            const int64_t r = i / S::ROWV;  // (t*Nk + node)*2 + mat
            const int64_t tn = r >> 1;
            const int64_t t = tn / Nk, node = tn % Nk;
            const uint4* src = (r & 1) ? wout : win;
            lds_rows[i] = src[(t * N + node) * S::ROWV + v];
        }
        __syncthreads();
    }

    const uint4* win = reinterpret_cast<const uint4*>(p.w_in);
    const uint4* wout = reinterpret_cast<const uint4*>(p.w_out);
    const int64_t n_groups = (p.n_tokens + S::TPW - 1) / S::TPW;
    for (int64_t g = int64_t(blockIdx.x) * WAVES + wave; g < n_groups; g += int64_t(gridDim.x) * WAVES) {
        const int64_t slot_raw = g * S::TPW + sub;
        const bool valid = slot_raw < p.n_tokens;
        const int64_t slot = valid ? slot_raw : p.n_tokens - 1;  // idle groups redo the last token, store nothing
        const int64_t tok = p.perm ? int64_t(p.perm[slot]) : slot;

        XRegs<LANES, NV, XBF, WBF> xr;
        xr.load(p.x, tok, sl);
        float acc[S::E];
#pragma unroll
        for (int e = 0; e < S::E; ++e) acc[e] = 0.0f;

        for (int t = 0; t < T; ++t) {
            int64_t n = 0;
            for (int l = 0; l <= D; ++l) {
                uint4 wi[NV], wo[NV];
                if (l < K) {
                    const uint4* rows = lds_rows + ((int64_t(t) * Nk + n) * 2) * S::ROWV;
#pragma unroll
                    for (int c = 0; c < NV; ++c) wi[c] = rows[c * LANES + sl];
#pragma unroll
                    for (int c = 0; c < NV; ++c) wo[c] = rows[S::ROWV + c * LANES + sl];
                } else {
                    const int64_t base = (int64_t(t) * N + n) * S::ROWV + sl;
#pragma unroll
                    for (int c = 0; c < NV; ++c) wi[c] = win[base + c * LANES];
#pragma unroll
                    for (int c = 0; c < NV; ++c) wo[c] = wout[base + c * LANES];
                }
                const float logit = group_sum<LANES>(xr.dot(wi));
                const float a = activation(logit, p.act);
                if (sl == 0 && valid) {
                    const int64_t rec = (tok * T + t) * (D + 1) + l;
                    if (p.nodes_out) p.nodes_out[rec] = int32_t(n);
                    if (p.logits_out) p.logits_out[rec] = logit;
                }
                axpy<NV, WBF>(acc, a, wo);
                n = 2 * n + 1 + (logit > 0.0f ? 1 : 0);
            }
        }
        if (valid) store_output<LANES, NV, XBF, WBF>(p, xr, acc, tok, sl);
    }
}

// ----------------------------------------------------------------------------
// generic kernel (any hidden size)
// ----------------------------------------------------------------------------

template <bool BF>
__device__ __forceinline__ float load_elem(const void* base, int64_t i) {
    if constexpr (BF) return bf16_to_f32(reinterpret_cast<const uint16_t*>(base)[i]);
    else return reinterpret_cast<const float*>(base)[i];
}

constexpr int GENERIC_BLOCK = 256;

template <bool XBF, bool WBF>
__global__ __launch_bounds__(GENERIC_BLOCK) void generic_kernel(Params p) {
    constexpr int WAVES = GENERIC_BLOCK / 64;
    extern __shared__ int32_t generic_lds[];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int T = p.n_trees, D = p.depth, H = p.hidden;
    const int P = T * (D + 1);
    const int64_t N = p.n_nodes;
    int32_t* s_node = generic_lds + wave * 2 * P;
    float* s_act = reinterpret_cast<float*>(s_node + P);

    for (int64_t slot = int64_t(blockIdx.x) * WAVES + wave; slot < p.n_tokens; slot += int64_t(gridDim.x) * WAVES) {
        const int64_t tok = p.perm ? int64_t(p.perm[slot]) : slot;
        const int64_t xoff = tok * H;
        for (int t = 0; t < T; ++t) {
            int64_t n = 0;
            for (int l = 0; l <= D; ++l) {
                const int64_t woff = (int64_t(t) * N + n) * H;
                float part = 0.0f;
                for (int h = lane; h < H; h += 64)
                    part = __builtin_fmaf(load_elem<XBF>(p.x, xoff + h), load_elem<WBF>(p.w_in, woff + h), part);
                const float logit = group_sum<64>(part);
                const float a = activation(logit, p.act);
                const int idx = t * (D + 1) + l;
                if (lane == 0) {
                    s_node[idx] = int32_t(n);
                    s_act[idx] = a;
                    const int64_t rec = tok * P + idx;
                    if (p.nodes_out) p.nodes_out[rec] = int32_t(n);
                    if (p.logits_out) p.logits_out[rec] = logit;
                }
                n = 2 * n + 1 + (logit > 0.0f ? 1 : 0);
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        for (int h0 = 0; h0 < H; h0 += 64) {
            const int h = h0 + lane;
            if (h < H) {
                float acc = 0.0f;
                for (int idx = 0; idx < P; ++idx) {
                    const int t = idx / (D + 1);
                    const int64_t row = int64_t(t) * N + s_node[idx];
                    acc = __builtin_fmaf(s_act[idx], load_elem<WBF>(p.w_out, row * H + h), acc);
                }
                if (p.out_mode == OUT_RESIDUAL) acc += load_elem<XBF>(p.x, xoff + h);
                if (p.y_bf16) {
                    uint16_t* y = reinterpret_cast<uint16_t*>(p.y) + tok * H + h;
                    if (p.out_mode == OUT_ACCUMULATE) acc += bf16_to_f32(*y);
                    *y = f32_to_bf16(acc);
                } else {
                    float* y = reinterpret_cast<float*>(p.y) + tok * H + h;
                    if (p.out_mode == OUT_ACCUMULATE) acc += *y;
                    *y = acc;
                }
            }
        }
        __builtin_amdgcn_wave_barrier();  // s_node/s_act are rewritten by the next token
    }
}

// ----------------------------------------------------------------------------
// planning
// ----------------------------------------------------------------------------

constexpr int DESCENT_BLOCK = 256;
constexpr size_t DEFAULT_LDS_BUDGET = 32 * 1024;  // per 256-thread block: keeps 4-5 blocks per CU
constexpr int GENERIC_MAX_PAIRS = 2048;

struct DescentVariant {
    int hidden;
    bool xbf, wbf;
    int lanes;
    const void* kernel;
    const char* name;
};

#define FFF_DESCENT(H, XB, WB, L, NV)                                                                  \
    DescentVariant {                                                                                   \
        H, XB, WB, L, reinterpret_cast<const void*>(&descent_kernel<L, NV, XB, WB, DESCENT_BLOCK>),    \
            "descent<lanes=" #L ",nv=" #NV ",x=" #XB ",w=" #WB ">"                                     \
    }

static const DescentVariant kDescent[] = {
    // H = 768 (BERT-base width)
    FFF_DESCENT(768, true, true, 16, 6),
    FFF_DESCENT(768, false, true, 16, 6),
    FFF_DESCENT(768, false, false, 32, 6),
    FFF_DESCENT(768, true, false, 32, 6),
    // H = 1024
    FFF_DESCENT(1024, true, true, 16, 8),
    FFF_DESCENT(1024, false, true, 16, 8),
    FFF_DESCENT(1024, false, false, 32, 8),
    FFF_DESCENT(1024, true, false, 32, 8),
    // H = 4096 (LLM width)
    FFF_DESCENT(4096, true, true, 64, 8),
    FFF_DESCENT(4096, false, true, 64, 8),
    FFF_DESCENT(4096, false, false, 64, 16),
    FFF_DESCENT(4096, true, false, 64, 16),
};

static const void* generic_kernel_for(bool xbf, bool wbf) {
    if (xbf && wbf) return reinterpret_cast<const void*>(&generic_kernel<true, true>);
    if (xbf) return reinterpret_cast<const void*>(&generic_kernel<true, false>);
    if (wbf) return reinterpret_cast<const void*>(&generic_kernel<false, true>);
    return reinterpret_cast<const void*>(&generic_kernel<false, false>);
}

// Resident blocks per CU for (kernel, block, dynamic LDS), cached per device.
static int blocks_per_cu(int device, const void* kernel, int block, size_t lds) {
    static std::mutex mu;
    static std::map<std::tuple<int, const void*, int, size_t>, int> cache;
    const auto key = std::make_tuple(device, kernel, block, lds);
    {
        std::lock_guard<std::mutex> g(mu);
        auto it = cache.find(key);
        if (it != cache.end()) return it->second;
    }
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, block, lds) != hipSuccess || n < 1) n = 1;
    std::lock_guard<std::mutex> g(mu);
    cache[key] = n;
    return n;
}

static size_t descent_lds_bytes(const Params& p, int levels) {
    if (levels <= 0) return 0;
    const size_t row_bytes = size_t(p.hidden) * (p.w_bf16 ? 2 : 4);
    return size_t(p.n_trees) * ((size_t(1) << levels) - 1) * 2 * row_bytes;
}

int plan_forward(const Params& p, int mode, int lds_levels_req, int split_level_req, const DeviceInfo& dev,
                 Plan* plan) {
    (void)split_level_req;
    *plan = Plan{};
    const DescentVariant* dv = nullptr;
    for (const auto& v : kDescent)
        if (v.hidden == p.hidden && v.xbf == bool(p.x_bf16) && v.wbf == bool(p.w_bf16)) dv = &v;

    if (mode == MODE_GROUPED) return ST_UNSUPPORTED;
    if (mode == MODE_DESCENT && !dv) return ST_UNSUPPORTED;

    if (dv && mode != MODE_GENERIC) {
        int levels;
        if (lds_levels_req < 0) {
            levels = 0;
        } else if (lds_levels_req > 0) {
            levels = lds_levels_req;
            if (levels > p.depth + 1 || descent_lds_bytes(p, levels) > dev.lds_per_block) return ST_UNSUPPORTED;
        } else {
            levels = 0;
            while (levels < p.depth + 1 && levels < 20 && descent_lds_bytes(p, levels + 1) <= DEFAULT_LDS_BUDGET)
                ++levels;
        }
        plan->kind = KIND_DESCENT;
        plan->kernel = dv->kernel;
        plan->lanes = dv->lanes;
        plan->block = DESCENT_BLOCK;
        plan->lds_levels = levels;
        plan->lds_bytes = descent_lds_bytes(p, levels);
        plan->name = dv->name;
        const int tpw = 64 / dv->lanes;
        const int64_t groups = (p.n_tokens + tpw - 1) / tpw;
        const int64_t want = (groups + DESCENT_BLOCK / 64 - 1) / (DESCENT_BLOCK / 64);
        const int64_t resident =
            int64_t(dev.cu_count) * blocks_per_cu(dev.device, dv->kernel, DESCENT_BLOCK, plan->lds_bytes);
        plan->grid = int(std::max<int64_t>(1, std::min(want, resident)));
        return ST_OK;
    }

    const int pairs = p.n_trees * (p.depth + 1);
    if (pairs > GENERIC_MAX_PAIRS) return ST_UNSUPPORTED;
    plan->kind = KIND_GENERIC;
    plan->kernel = generic_kernel_for(p.x_bf16, p.w_bf16);
    plan->lanes = 64;
    plan->block = GENERIC_BLOCK;
    plan->lds_bytes = size_t(GENERIC_BLOCK / 64) * 2 * size_t(pairs) * 4;
    plan->name = "generic<wave per token>";
    const int64_t want = (p.n_tokens + GENERIC_BLOCK / 64 - 1) / (GENERIC_BLOCK / 64);
    const int64_t resident =
        int64_t(dev.cu_count) * blocks_per_cu(dev.device, plan->kernel, GENERIC_BLOCK, plan->lds_bytes);
    plan->grid = int(std::max<int64_t>(1, std::min(want, resident)));
    return ST_OK;
}

hipError_t run_forward(const Params& p, const Plan& plan, void* workspace, size_t workspace_bytes,
                       hipStream_t stream) {
    (void)workspace;
    (void)workspace_bytes;
    Params q = p;
    q.lds_levels = plan.lds_levels;
    void* args[] = {&q};
    return hipLaunchKernel(plan.kernel, dim3(plan.grid), dim3(plan.block), args, plan.lds_bytes, stream);
}

size_t grouped_workspace_bytes(int64_t, int32_t, int32_t, int32_t) { return 0; }

}  // namespace fff
