// fff_common.hpp -- register-level building blocks shared by the FFF kernels:
// the per-token lane layout, x held in registers, the dot product, the
// output-row FMA, the group broadcast and the final combine-and-store.
#pragma once

#include "fff_device.hpp"
#include "fff_internal.hpp"

namespace fff {

enum { OUT_STORE = 0, OUT_ACCUMULATE = 1, OUT_RESIDUAL = 2 };

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
    // Replace x by the bf16 rounding of vals (laid out like an output slice).
    __device__ void set_from(const float* vals, bool /*to_bf16: always*/) {
#pragma unroll
        for (int c = 0; c < NV; ++c)
            v[c] = make_uint4(pack_bf16x2(vals[c * 8 + 0], vals[c * 8 + 1]), pack_bf16x2(vals[c * 8 + 2], vals[c * 8 + 3]),
                              pack_bf16x2(vals[c * 8 + 4], vals[c * 8 + 5]), pack_bf16x2(vals[c * 8 + 6], vals[c * 8 + 7]));
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
    // x stored as bf16 (xbf) or fp32, widened into this fp32 layout.
    __device__ void load_widen(const void* x, bool xbf, int64_t tok, int sl) {
        if (!xbf) {
            load(x, tok, sl);
            return;
        }
        const uint4* row = reinterpret_cast<const uint4*>(x) + tok * (LANES * NV);
#pragma unroll
        for (int c = 0; c < NV; ++c) {
            const uint4 a = row[c * LANES + sl];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                f[c * 8 + 2 * j] = bf16_lo(word(a, j));
                f[c * 8 + 2 * j + 1] = bf16_hi(word(a, j));
            }
        }
    }
    __device__ void set_from(const float* vals, bool to_bf16) {
#pragma unroll
        for (int i = 0; i < NV * 8; ++i) f[i] = to_bf16 ? bf16_to_f32(f32_to_bf16(vals[i])) : vals[i];
    }
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
    __device__ void load_widen(const void* x, bool xbf, int64_t tok, int sl) {
        if (xbf) {
            XRegsF32W<LANES, NV, true> t;
            t.load(x, tok, sl);
#pragma unroll
            for (int i = 0; i < NV * 4; ++i) f[i] = t.f[i];
        } else {
            XRegsF32W<LANES, NV, false> t;
            t.load(x, tok, sl);
#pragma unroll
            for (int i = 0; i < NV * 4; ++i) f[i] = t.f[i];
        }
    }
    __device__ void set_from(const float* vals, bool to_bf16) {
#pragma unroll
        for (int i = 0; i < NV * 4; ++i) f[i] = to_bf16 ? bf16_to_f32(f32_to_bf16(vals[i])) : vals[i];
    }
};
template <int LANES, int NV>
struct XRegs<LANES, NV, false, false> : XRegsF32W<LANES, NV, false> {};
template <int LANES, int NV>
struct XRegs<LANES, NV, true, false> : XRegsF32W<LANES, NV, true> {};

// Zeros standing in for an absent LayerNorm gain or shift in the register
// kernels (hidden <= 4096), so that those loads need no branch.
constexpr int NORM_TABLE = 4096;
static __device__ float g_norm_zeros[NORM_TABLE];

// LayerNorm of one token held in fp32 registers (f in the layout above, EV
// elements per vector): mean and biased variance over all H elements, summed
// per lane then across the group (every lane gets the same bits), then
// f = (f - mean) / sqrt(var + eps) * gamma + beta.  gamma / beta may be null.
template <int LANES, int NV, bool WBF>
__device__ __forceinline__ void layer_norm_regs(float* f, const float* gamma, const float* beta, float eps,
                                                int sl) {
    constexpr int EV = WBF ? 8 : 4;
    constexpr int E = NV * EV;
    constexpr float H = float(LANES * E);
    static_assert(LANES * E <= NORM_TABLE, "zero table too short");
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < E; ++i) s += f[i];
    const float mean = group_sum<LANES>(s) / H;
    float q = 0.0f;
#pragma unroll
    for (int i = 0; i < E; ++i) {
        f[i] -= mean;  // centred in place: x and x - mean are never both live
        q = __builtin_fmaf(f[i], f[i], q);
    }
    const float var = group_sum<LANES>(q) / H;
    const float rstd = 1.0f / sqrtf(var + eps);
    const bool has_gamma = gamma != nullptr;
    const float* gp = has_gamma ? gamma : g_norm_zeros;
    const float* bp = beta ? beta : g_norm_zeros;
    // One vector of gain and shift at a time: hoisting all of them above the
    // statistics would hold 2*E extra registers at the kernel's peak.  The
    // empty asm statements pin the order (loads of chunk c, then its FMAs, then
    // chunk c+1); they emit no instructions.
#pragma unroll
    for (int c = 0; c < NV; ++c) {
        asm volatile("" ::: "memory");
#pragma unroll
        for (int q4 = 0; q4 < EV / 4; ++q4) {
            const int col = (c * LANES + sl) * EV + 4 * q4;
            const float4 g = *reinterpret_cast<const float4*>(gp + col);
            const float4 b = *reinterpret_cast<const float4*>(bp + col);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                float& v = f[c * EV + 4 * q4 + j];
                v = __builtin_fmaf(v * rstd, has_gamma ? fword(g, j) : 1.0f, fword(b, j));
                asm volatile("" : "+v"(v));
            }
        }
    }
}

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

// Final combine and store of one token's output slice; xr (anything with
// elem(c, e) in the lane layout) supplies x for the residual.
template <int LANES, int NV, bool WBF, class XR>
__device__ __forceinline__ void store_output(const Params& p, const XR& xr, float* acc, int64_t tok, int sl) {
    using S = Shape<LANES, NV, false, WBF>;
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

// Value of lane `src` of this lane's LANES-wide group.
template <int LANES>
__device__ __forceinline__ float group_bcast(float v, int lane, int src) {
    if constexpr (LANES == 64) {
        return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), src));
    } else {
        const int idx = ((lane & ~(LANES - 1)) + src) << 2;
        return __int_as_float(__builtin_amdgcn_ds_bpermute(idx, __float_as_int(v)));
    }
}

// Logits of the levels of one tree, parked one per lane: level l lives in
// lane l % LANES of register l / LANES.  Depth is at most 24.
template <int LANES>
struct LevelRegs {
    static constexpr int NR = (25 + LANES - 1) / LANES;
    float v[NR];
    __device__ void clear() {
#pragma unroll
        for (int r = 0; r < NR; ++r) v[r] = 0.0f;
    }
    __device__ void park(int l, int sl, float x) {
#pragma unroll
        for (int r = 0; r < NR; ++r) v[r] = (l == r * LANES + sl) ? x : v[r];
    }
    // value of level l, broadcast to the whole group (l is uniform: no branches)
    __device__ float get(int l, int lane) const {
        float sel = v[0];
#pragma unroll
        for (int r = 1; r < NR; ++r) sel = l >= r * LANES ? v[r] : sel;
        return group_bcast<LANES>(sel, lane, l & (LANES - 1));
    }
};

// Phase 1 of one tree: the CMM walk from the root, reading only W_in rows.
// Levels below KD come from LDS rows (lrows + node*lstride, already offset by
// the lane), the rest from global rows (win + node*ROWV).  Level logits are
// parked in lv; returns leaf + 1 (the ancestor at level l is
// ((leaf + 1) >> (D - l)) - 1).
template <int LANES, int NV, bool XBF, bool WBF>
__device__ __forceinline__ uint32_t walk_tree(const XRegs<LANES, NV, XBF, WBF>& xr, const uint4* lrows,
                                              int64_t lstride, const uint4* win, int KD, int D, int sl,
                                              LevelRegs<LANES>& lv) {
    using S = Shape<LANES, NV, XBF, WBF>;
    lv.clear();
    uint32_t n = 0;
    for (int l = 0; l < KD; ++l) {
        uint4 w[NV];
        const uint4* row = lrows + int64_t(n) * lstride;
#pragma unroll
        for (int c = 0; c < NV; ++c) w[c] = row[c * LANES];
        const float logit = group_sum<LANES>(xr.dot(w));
        lv.park(l, sl, logit);
        if (l < D) n = 2 * n + 1 + (logit > 0.0f ? 1u : 0u);
    }
    for (int l = KD; l <= D; ++l) {
        uint4 w[NV];
        const uint4* row = win + int64_t(n) * S::ROWV;
#pragma unroll
        for (int c = 0; c < NV; ++c) w[c] = row[c * LANES];
        const float logit = group_sum<LANES>(xr.dot(w));
        lv.park(l, sl, logit);
        if (l < D) n = 2 * n + 1 + (logit > 0.0f ? 1u : 0u);
    }
    return n + 1;
}

// Phase 3 of one tree: acc += sum_l a_l * W_out[ancestor_l].  `lds_row(l)` and
// `global_row(l)` give the lane's first vector of level l's row (LDS below KD,
// global memory from KD on; kept apart so every load has a known address
// space), `act(l)` its activation.  The global levels keep one row in flight
// ahead of the FMAs.  The prefetch is unconditional -- past the last level it
// re-reads the last row, which is already cached -- so the compiler sees a
// plain two-buffer pipeline.
template <int LANES, int NV, bool WBF, class LdsRowFn, class GlobalRowFn, class ActFn>
__device__ __forceinline__ void emit_levels(float* acc, int KD, int D, LdsRowFn lds_row, GlobalRowFn global_row,
                                            ActFn act) {
    uint4 cur[NV], nxt[NV];
    float a_cur, a_nxt;
    auto load = [&](uint4* dst, float& a, int l) {
        const uint4* r = global_row(l);
#pragma unroll
        for (int c = 0; c < NV; ++c) dst[c] = r[c * LANES];
        a = act(l);
    };
    // The first global row is in flight while the LDS levels are accumulated;
    // sched_barrier keeps each prefetch above the FMAs it is meant to overlap
    // (the scheduler would otherwise sink it to its use to save registers).
    const bool global = KD <= D;
    if (global) load(cur, a_cur, KD);
    __builtin_amdgcn_sched_barrier(0);
    for (int l = 0; l < KD; ++l) {
        const uint4* r = lds_row(l);
        uint4 w[NV];
#pragma unroll
        for (int c = 0; c < NV; ++c) w[c] = r[c * LANES];
        axpy<NV, WBF>(acc, act(l), w);
    }
    if (!global) return;
    for (int l = KD;; l += 2) {
        load(nxt, a_nxt, l + 1 <= D ? l + 1 : D);
        __builtin_amdgcn_sched_barrier(0);
        axpy<NV, WBF>(acc, a_cur, cur);
        if (l + 1 > D) break;
        load(cur, a_cur, l + 2 <= D ? l + 2 : D);
        __builtin_amdgcn_sched_barrier(0);
        axpy<NV, WBF>(acc, a_nxt, nxt);
        if (l + 2 > D) break;
    }
}

}  // namespace fff
