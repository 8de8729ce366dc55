// fff_kernels.hip -- gfx950 kernels for FFF inference: conditional matrix
// multiplication (Algorithm 1 of the paper) followed by the output
// accumulation, with the Section 2.1 model (activation and output row at every
// visited node, no biases, trees summed).
//
// Every kernel gives one token to a group of LANES lanes (16, 32 or 64) that
// keeps the token's x slice in registers; per level it gathers whole weight
// rows with 16-byte loads, reduces the dot product across the group with DPP
// row rotations and permlane swaps, and branches on the sign.  Per tree the
// work runs in three phases (fff_common.hpp): walk (W_in only, level logits
// parked one per lane), one activation evaluation for all levels, then the
// W_out rows of the now-known path accumulated into fp32 registers.
//
// DESCENT (descent_kernel): all three phases in one kernel; the top tree
//   levels of W_in and W_out are staged once per workgroup into LDS (the
//   paper's advice to preload the weights of the sub-trees a token needs,
//   Section 3.2).
// GROUPED (walk_kernel + emit_kernel): the walk -- the CMM of Algorithm 1 --
//   writes each token's leaf and activations to the workspace; the emit
//   kernel then accumulates the output rows.  With a split level k, tokens are
//   grouped by their tree-0 node at level k and every subtree is emitted by
//   workgroups of one XCD (blockIdx % 8), so the subtree's W_out rows stay in
//   that XCD's L2 instead of being fetched by all eight.
// GENERIC (generic_kernel): any hidden size, one wave per token.
#include "fff_common.hpp"
#include "fff_device.hpp"
#include "fff_internal.hpp"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <tuple>
#include <type_traits>

namespace fff {

enum { MODE_AUTO = 0, MODE_DESCENT = 1, MODE_GROUPED = 2, MODE_GENERIC = 3, MODE_TILED = 4, MODE_MASKED = 5,
       MODE_SUBTREE = 6 };
// status values mirrored from fff.h
enum { ST_OK = 0, ST_INVALID = -1, ST_UNSUPPORTED = -2, ST_WORKSPACE = -3 };

// Copy rows [0, Nk) of every tree's matrix into LDS, [T][Nk][stride] vectors,
// at vector offset `off` within each stride (W_in and W_out interleave in the
// descent kernel: stride 2*ROWV, offsets 0 and ROWV).
template <int ROWV, int BLOCK>
__device__ __forceinline__ void stage_rows(uint4* lds, const void* w, int T, int64_t N, int Nk, int stride,
                                           int off) {
    const uint4* src = reinterpret_cast<const uint4*>(w);
    const int64_t total = int64_t(T) * Nk * ROWV;
    for (int64_t i = threadIdx.x; i < total; i += BLOCK) {
        const int64_t v = i % ROWV;
        const int64_t tn = i / ROWV;
        const int64_t t = tn / Nk, node = tn % Nk;
        lds[tn * stride + off + v] = src[(t * N + node) * ROWV + v];
    }
}

// Per-visit records (optional outputs): node and logit of every level.
template <int LANES>
__device__ __forceinline__ void write_records(int32_t* nodes, float* logits, const Params& p,
                                              const LevelRegs<LANES>& lv, uint32_t leaf1, int64_t tok, int t, int sl) {
    const int D = p.depth;
#pragma unroll
    for (int r = 0; r < LevelRegs<LANES>::NR; ++r) {
        const int l = r * LANES + sl;
        if (l <= D) {
            const int64_t rec = (tok * p.n_trees + t) * (D + 1) + l;
            if (nodes) nodes[rec] = int32_t((leaf1 >> (D - l)) - 1);
            if (logits) logits[rec] = lv.v[r];
        }
    }
}

// The FFF input of one token in registers: x itself in its stored layout, or
// (NORM) x widened to fp32 and layer-normalised.
template <int LANES, int NV, bool XBF, bool WBF, bool NORM>
using XIn = XRegs<LANES, NV, NORM ? false : XBF, WBF>;

template <int LANES, int NV, bool XBF, bool WBF, bool NORM>
__device__ __forceinline__ void load_input(XIn<LANES, NV, XBF, WBF, NORM>& xr, const Params& p, int64_t tok,
                                           int sl) {
    if constexpr (NORM) {
        xr.load_widen(p.x, p.x_bf16, tok, sl);
        layer_norm_regs<LANES, NV, WBF>(xr.f, p.gamma, p.beta, p.norm_eps, sl);
    } else {
        xr.load(p.x, tok, sl);
    }
}

// Combine and store; with NORM the residual adds the raw x, reloaded.
template <int LANES, int NV, bool XBF, bool WBF, bool NORM>
__device__ __forceinline__ void finish_token(const Params& p, const XIn<LANES, NV, XBF, WBF, NORM>& xr, float* acc,
                                             int64_t tok, int sl) {
    if (NORM && p.out_mode == OUT_RESIDUAL) {
        XRegs<LANES, NV, false, WBF> raw;
        raw.load_widen(p.x, p.x_bf16, tok, sl);
        store_output<LANES, NV, WBF>(p, raw, acc, tok, sl);
    } else {
        store_output<LANES, NV, WBF>(p, xr, acc, tok, sl);
    }
}

// ----------------------------------------------------------------------------
// DESCENT: one fused kernel
// ----------------------------------------------------------------------------

template <int LANES, int NV, bool XBF, bool WBF, int BLOCK, bool NORM>
__global__ __launch_bounds__(BLOCK) void descent_kernel(Params p) {
    static_assert(!(NORM && XBF), "normalised inputs are held in fp32");
    using S = Shape<LANES, NV, XBF, WBF>;
    constexpr bool XR_BF = NORM ? false : XBF;
    constexpr int WAVES = BLOCK / 64;
    extern __shared__ uint4 lds_rows[];  // [T][Nk][2][ROWV]: W_in row then W_out row

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int sl = lane % LANES;
    const int sub = lane / LANES;
    const int T = p.n_trees, D = p.depth, K = p.lds_levels;
    const int64_t N = p.n_nodes;
    const int Nk = (1 << K) - 1;
    if (K > 0) {
        stage_rows<S::ROWV, BLOCK>(lds_rows, p.w_in, T, N, Nk, 2 * S::ROWV, 0);
        stage_rows<S::ROWV, BLOCK>(lds_rows, p.w_out, T, N, Nk, 2 * S::ROWV, S::ROWV);
        __syncthreads();
    }
    const int KD = K < D + 1 ? K : D + 1;
    const int64_t n_groups = (p.n_tokens + S::TPW - 1) / S::TPW;
    for (int64_t g = int64_t(blockIdx.x) * WAVES + wave; g < n_groups; g += int64_t(gridDim.x) * WAVES) {
        const int64_t slot_raw = g * S::TPW + sub;
        const bool valid = slot_raw < p.n_tokens;
        const int64_t tok = valid ? slot_raw : p.n_tokens - 1;  // idle groups redo the last token, store nothing
        XIn<LANES, NV, XBF, WBF, NORM> xr;
        load_input<LANES, NV, XBF, WBF, NORM>(xr, p, tok, sl);
        float acc[S::E];
#pragma unroll
        for (int e = 0; e < S::E; ++e) acc[e] = 0.0f;
        for (int t = 0; t < T; ++t) {
            const uint4* win = reinterpret_cast<const uint4*>(p.w_in) + int64_t(t) * N * S::ROWV + sl;
            const uint4* wout = reinterpret_cast<const uint4*>(p.w_out) + int64_t(t) * N * S::ROWV + sl;
            const uint4* lrows = lds_rows + int64_t(t) * Nk * 2 * S::ROWV + sl;
            LevelRegs<LANES> lv;
            const uint32_t leaf1 = walk_tree<LANES, NV, XR_BF, WBF>(xr, lrows, 2 * S::ROWV, win, KD, D, sl, lv);
            LevelRegs<LANES> av;
#pragma unroll
            for (int r = 0; r < LevelRegs<LANES>::NR; ++r) av.v[r] = activation(lv.v[r], p.act);
            if ((p.nodes_out || p.logits_out) && valid)
                write_records<LANES>(p.nodes_out, p.logits_out, p, lv, leaf1, tok, t, sl);
            const uint4* lout = lrows + S::ROWV;
            emit_levels<LANES, NV, WBF>(
                acc, KD, D, [&](int l) { return lout + int64_t((leaf1 >> (D - l)) - 1) * 2 * S::ROWV; },
                [&](int l) { return wout + int64_t((leaf1 >> (D - l)) - 1) * S::ROWV; },
                [&](int l) { return av.get(l, lane); });
        }
        if (valid) finish_token<LANES, NV, XBF, WBF, NORM>(p, xr, acc, tok, sl);
    }
}

// ----------------------------------------------------------------------------
// GROUPED: walk kernel (CMM) then emit kernel
// ----------------------------------------------------------------------------

template <int LANES, int NV, bool XBF, bool WBF, int BLOCK, bool NORM>
__global__ __launch_bounds__(BLOCK) void walk_kernel(Params p) {
    static_assert(!(NORM && XBF), "normalised inputs are held in fp32");
    using S = Shape<LANES, NV, XBF, WBF>;
    constexpr bool XR_BF = NORM ? false : XBF;
    constexpr int WAVES = BLOCK / 64;
    extern __shared__ uint4 lds_in[];  // [T][Nk][ROWV] W_in rows of the top levels

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int sl = lane % LANES;
    const int sub = lane / LANES;
    const int T = p.n_trees, D = p.depth, K = p.lds_levels;
    const int64_t N = p.n_nodes;
    const int Nk = (1 << K) - 1;
    // Tree-affine walk (T divides the XCD count): the workgroups of XCD x walk tree x mod T for
    // all tokens, so each XCD's L2 holds one tree's rows and LDS that tree's top levels; x is
    // read once per tree.  Otherwise every workgroup walks all trees of its tokens.
    const bool affine = p.walk_affine;
    const int t_first = affine ? int(blockIdx.x % XCDS) % T : 0;
    const int t_end = affine ? t_first + 1 : T;
    const int64_t n_blk = affine ? int64_t(gridDim.x) / T : int64_t(gridDim.x);
    const int64_t blk = affine ? int64_t(blockIdx.x / XCDS) * (XCDS / T) + (blockIdx.x % XCDS) / T : int64_t(blockIdx.x);
    if (K > 0) {
        const void* src = static_cast<const char*>(p.w_in) + int64_t(t_first) * N * S::ROWV * 16;
        stage_rows<S::ROWV, BLOCK>(lds_in, src, t_end - t_first, N, Nk, S::ROWV, 0);
        __syncthreads();
    }
    const int KD = K < D + 1 ? K : D + 1;
    const int64_t n_groups = (p.n_tokens + S::TPW - 1) / S::TPW;
    for (int64_t g = blk * WAVES + wave; g < n_groups; g += n_blk * WAVES) {
        const int64_t slot_raw = g * S::TPW + sub;
        const bool valid = slot_raw < p.n_tokens;
        const int64_t tok = valid ? slot_raw : p.n_tokens - 1;
        XIn<LANES, NV, XBF, WBF, NORM> xr;
        load_input<LANES, NV, XBF, WBF, NORM>(xr, p, tok, sl);
        for (int t = t_first; t < t_end; ++t) {
            const uint4* win = reinterpret_cast<const uint4*>(p.w_in) + int64_t(t) * N * S::ROWV + sl;
            const uint4* lrows = lds_in + int64_t(t - t_first) * Nk * S::ROWV + sl;
            LevelRegs<LANES> lv;
            const uint32_t leaf1 = walk_tree<LANES, NV, XR_BF, WBF>(xr, lrows, S::ROWV, win, KD, D, sl, lv);
            float* rec = p.ws_act + (tok * T + t) * (D + 1);
            if (p.bk_count) {
                // tiled mode: take the next slot of the bucket of this tree's leaf; the
                // activations go to the slot, or to the token's record once the bucket is full
                const int64_t bin = int64_t(t) * (int64_t(1) << D) + int64_t(leaf1) - (int64_t(1) << D);
                int32_t pos = 0;
                if (valid && sl == 0) pos = atomicAdd(&p.bk_count[bin], 1);
                pos = __float_as_int(group_bcast<LANES>(__int_as_float(pos), lane, 0));
                if (valid && pos < p.bk_cap) {
                    rec = p.bk_act + (bin * p.bk_cap + pos) * TILE_REC;
                    if (sl == 0) p.bk_tok[bin * p.bk_cap + pos] = int32_t(tok);
                } else if (valid && sl == 0) {
                    p.bk_spill[int64_t(t) * p.n_tokens + atomicAdd(&p.bk_nspill[t], 1)] = int32_t(tok);
                }
            }
            if (valid) {
#pragma unroll
                for (int r = 0; r < LevelRegs<LANES>::NR; ++r) {
                    const int l = r * LANES + sl;
                    if (l <= D) rec[l] = activation(lv.v[r], p.act);
                }
                if (sl == 0) p.ws_leaf[tok * T + t] = int32_t(leaf1 - 1);
                if (p.nodes_out || p.logits_out)
                    write_records<LANES>(p.nodes_out, p.logits_out, p, lv, leaf1, tok, t, sl);
            }
        }
    }
}

constexpr int EMIT_SCAN_PER_THREAD = 4;

// XCD owning the subtree of a token whose tree-0 leaf is `leaf`: its node at
// the split level k, counted within the level, modulo the XCD count.
__device__ __forceinline__ int owner_xcd(const Params& p, int32_t leaf) {
    const int k = p.split_level, D = p.depth;
    const uint32_t leaf1 = uint32_t(leaf) + 1;
    const uint32_t bucket = (leaf1 >> (D - k)) - (1u << k);
    return int(bucket % XCDS);
}

template <int LANES, int NV, bool XBF, bool WBF, int BLOCK>
__global__ __launch_bounds__(BLOCK) void emit_kernel(Params p) {
    using S = Shape<LANES, NV, XBF, WBF>;
    constexpr int WAVES = BLOCK / 64;
    constexpr int SCAN = BLOCK * EMIT_SCAN_PER_THREAD;
    extern __shared__ uint4 lds_out[];  // [T][Nk][ROWV] W_out rows of the top levels
    __shared__ int32_t queue[SCAN];       // token
    __shared__ int32_t queue_leaf[SCAN];  // its tree-0 leaf
    __shared__ int32_t queue_len;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int sl = lane % LANES;
    const int sub = lane / LANES;
    const int T = p.n_trees, D = p.depth, K = p.lds_levels;
    const int64_t N = p.n_nodes;
    const int Nk = (1 << K) - 1;
    if (K > 0) stage_rows<S::ROWV, BLOCK>(lds_out, p.w_out, T, N, Nk, S::ROWV, 0);
    const int KD = K < D + 1 ? K : D + 1;

    // Token range of this workgroup.  Grouped by subtree: the workgroups of XCD
    // x (blockIdx % 8 == x) split the whole batch between them and each keeps
    // only the tokens whose subtree x owns.
    const bool affine = p.split_level > 0;
    const int xcd = affine ? int(blockIdx.x % XCDS) : 0;
    const int64_t nloc = affine ? gridDim.x / XCDS : gridDim.x;
    const int64_t local = affine ? blockIdx.x / XCDS : blockIdx.x;
    const int64_t chunk = (p.n_tokens + nloc - 1) / nloc;
    const int64_t b0 = local * chunk;
    const int64_t b1 = b0 + chunk < p.n_tokens ? b0 + chunk : p.n_tokens;

    // What a token group needs before its first row: the token, its tree-0 leaf and
    // tree-0 activations (one level per lane, broadcast when used).  Fetched one
    // group ahead so that these loads are off the critical path.
    struct GroupIn {
        int64_t tok;
        uint32_t leaf1;
        bool valid;
        LevelRegs<LANES> av;
    };

    for (int64_t base = b0; base < b1; base += SCAN) {
        int count;
        if (affine) {
            if (tid == 0) queue_len = 0;
            __syncthreads();  // also orders the LDS staging before first use
#pragma unroll
            for (int i = 0; i < EMIT_SCAN_PER_THREAD; ++i) {
                const int64_t b = base + int64_t(i) * BLOCK + tid;
                const int32_t leaf = b < b1 ? p.ws_leaf[b * T] : 0;
                const bool take = b < b1 && owner_xcd(p, leaf) == xcd;
                const uint64_t mask = __ballot(take);
                const int before = __builtin_amdgcn_mbcnt_hi(uint32_t(mask >> 32),
                                                              __builtin_amdgcn_mbcnt_lo(uint32_t(mask), 0));
                int wbase = 0;
                if (lane == 0 && mask) wbase = atomicAdd(&queue_len, __popcll(mask));
                wbase = __builtin_amdgcn_readfirstlane(wbase);
                if (take) {
                    queue[wbase + before] = int32_t(b);
                    queue_leaf[wbase + before] = leaf;
                }
            }
            __syncthreads();
            count = queue_len;
        } else {
            if (base == b0) __syncthreads();  // LDS staging
            count = int(b1 - base < SCAN ? b1 - base : SCAN);
        }
        const int groups = (count + S::TPW - 1) / S::TPW;
        auto fetch = [&](int g) {
            GroupIn in;
            const int idx_raw = g * S::TPW + sub;
            in.valid = idx_raw < count;
            const int idx = in.valid ? idx_raw : count - 1;
            in.tok = affine ? int64_t(queue[idx]) : base + idx;
            in.leaf1 = uint32_t(affine ? queue_leaf[idx] : p.ws_leaf[in.tok * T]) + 1;
            const float* arec = p.ws_act + in.tok * T * (D + 1);
#pragma unroll
            for (int r = 0; r < LevelRegs<LANES>::NR; ++r) {
                const int l = r * LANES + sl;
                in.av.v[r] = l <= D ? arec[l] : 0.0f;
            }
            return in;
        };
        if (wave < groups) {  // wave-uniform
            GroupIn cur = fetch(wave);
            for (int g = wave; g < groups; g += WAVES) {
                GroupIn nxt = cur;
                if (g + WAVES < groups) nxt = fetch(g + WAVES);
                const int64_t tok = cur.tok;
                float acc[S::E];
#pragma unroll
                for (int e = 0; e < S::E; ++e) acc[e] = 0.0f;
                {
                    const uint32_t leaf1 = cur.leaf1;
                    const uint4* wout = reinterpret_cast<const uint4*>(p.w_out) + sl;
                    const uint4* lrows = lds_out + sl;
                    emit_levels<LANES, NV, WBF>(
                        acc, KD, D, [&](int l) { return lrows + int64_t((leaf1 >> (D - l)) - 1) * S::ROWV; },
                        [&](int l) { return wout + int64_t((leaf1 >> (D - l)) - 1) * S::ROWV; },
                        [&](int l) { return cur.av.get(l, lane); });
                }
                for (int t = 1; t < T; ++t) {
                    const uint32_t leaf1 = uint32_t(p.ws_leaf[tok * T + t]) + 1;
                    const float* arec = p.ws_act + (tok * T + t) * (D + 1);  // one address per group
                    const uint4* wout = reinterpret_cast<const uint4*>(p.w_out) + int64_t(t) * N * S::ROWV + sl;
                    const uint4* lrows = lds_out + int64_t(t) * Nk * S::ROWV + sl;
                    emit_levels<LANES, NV, WBF>(
                        acc, KD, D, [&](int l) { return lrows + int64_t((leaf1 >> (D - l)) - 1) * S::ROWV; },
                        [&](int l) { return wout + int64_t((leaf1 >> (D - l)) - 1) * S::ROWV; },
                        [&](int l) { return arec[l]; });
                }
                XRegs<LANES, NV, XBF, WBF> xr;
                if (p.out_mode == OUT_RESIDUAL) xr.load(p.x, tok, sl);
                if (cur.valid) store_output<LANES, NV, WBF>(p, xr, acc, tok, sl);
                cur = nxt;
            }
        }
        if (affine) __syncthreads();  // the queue is refilled next round
    }
}

// ----------------------------------------------------------------------------
// TILED: the output accumulation of tokens that share a leaf on MFMA
// ----------------------------------------------------------------------------
//
// Tokens that reach the same leaf visit the same D+1 nodes, so for a tile of
// up to 16 of them the output is a dense product
//     Y[16 tokens, H] = A[16 tokens, D+1 levels] x W_out[path rows, H],
// with A the tokens' activations.  One workgroup takes one leaf; its wave w
// takes the 128-column groups g = w, w + waves, ...  Every 16x16 MFMA used here
// returns D[4(l/16)+r][l%16] to lane l, register r.  In group g, MFMA column n
// of block j is output column 128 g + 8 n + j when y is bf16, so a lane holds
// eight consecutive output columns of four tokens and sixteen lanes write 256
// contiguous bytes of a token's row; when y is fp32 it is output column
// 128 g + 64 (j/4) + 4 n + j%4, and the two halves (blocks 0..3, then 4..7) are
// computed and stored in turn, sixteen lanes writing 256 contiguous bytes per
// half, so four accumulators are live at a time instead of eight.
//
// bf16 weights: v_mfma_f32_16x16x32_bf16 takes 32 (level, part) products per
// lane group.  Lane group q = l/16 covers levels 8(q%2) .. 8(q%2)+7; each
// activation (fp32) is split into bf16 parts a = hi + mid + lo (each part the
// rounded remainder of the previous ones, exact to fp32 working accuracy), and
// group q supplies part q/2 in the first MFMA and part q/2 + 2 (lo, or zero)
// in the second.  Two parts (hi + mid, relative error about 2^-17) are used
// when y is stored in bf16, whose own rounding is 2^-9.  The B operand of
// lane (n, q) for block j is that block's column of its eight path rows: eight
// 16-byte row loads (sixteen of 8 bytes for an fp32 y), transposed in registers
// once per leaf.  Products of bf16 values are exact; the MFMA accumulates in fp32.
//
// fp32 weights: v_mfma_f32_16x16x4_f32, four levels per step: lane l supplies
// A[l%16][l/16] (token l%16, level 4s + l/16) and the weights of its level's
// row for blocks j = 0..7 from two 16-byte loads, one per half.
//
// Activation records of bucketed tokens are TILE_REC floats apart (depth at
// most 15).  Tokens whose bucket was full (more than bk_cap reached one leaf)
// are handled by extra workgroups with the per-token emit.

constexpr int TILE_MAX_STEPS = 4;  // fp32 weights: depth <= 15, at most 16 levels, four steps of four
// fp32 weights up to depth 11 take three steps: the B operands of the fourth step would hold eight
// more VGPRs per lane (94 against 106: five waves per SIMD instead of four)
constexpr int TILE_STEPS_SHALLOW = 3;

// Waves per tiled workgroup for hidden size h: one per 128-column group, at most 8
// (larger workgroups would cap the registers of the spill path below 128).
constexpr int tile_waves(int h) { return h / 128 < 8 ? h / 128 : 8; }

// Output forms of the tile kernel, fixed at compile time: the tile's result is
// added to a source row (none; fp32; bf16) and written to a destination row
// (fp32 or bf16).  One tree: the source is x (residual), y (accumulate) or
// none, the destination y.  Several trees: the trees' tile launches run in tree
// order, tree t adding its contribution to the running sum S left by tree t-1
// (S is y itself when y is fp32, else an fp32 workspace), the last writing y,
// so the sum over trees has a fixed order.  With the form fixed, every path
// through a tile issues the same memory operations, so the compiler can wait
// for the prefetched operands without draining the stores.
enum { TSRC_NONE = 0, TSRC_F32 = 1, TSRC_BF16 = 2 };

// The tile kernel's stores and source loads go through buffer resources over the
// [B, H] row blocks with 32-bit byte offsets; a forward whose fp32 rows would
// reach 2^31 bytes runs in chunks of this many tokens (the offset TILE_NO_ROW of
// empty rows then lies past every block).
static int64_t tile_chunk_tokens(int64_t hidden) { return ((int64_t(1) << 31) - 1) / (4 * hidden); }

// Eight consecutive output columns of one token: add the source and store,
// through buffer resources over the source and destination rows.  An offset
// past the resource's size (TILE_NO_ROW) makes the hardware drop the store and
// read zeros, without a memory access.
typedef uint32_t tile_u4 __attribute__((ext_vector_type(4)));
typedef uint32_t tile_u2 __attribute__((ext_vector_type(2)));
constexpr uint32_t TILE_NO_ROW = 0x80000000u;

template <int SRC, bool DBF>
__device__ __forceinline__ void tile_store8_buf(__amdgpu_buffer_rsrc_t rs, uint32_t os, __amdgpu_buffer_rsrc_t rd,
                                                uint32_t od, const float* v8) {
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = v8[i];
    if constexpr (SRC == TSRC_F32) {
        const tile_u4 a = __builtin_amdgcn_raw_buffer_load_b128(rs, int(os), 0, 0);
        const tile_u4 b = __builtin_amdgcn_raw_buffer_load_b128(rs, int(os + 16), 0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t ai = a[i], bi = b[i];  // scalar copies: this compiler bit-casts a vector element as element 0
            v[i] += __builtin_bit_cast(float, ai);
            v[4 + i] += __builtin_bit_cast(float, bi);
        }
    } else if constexpr (SRC == TSRC_BF16) {
        const tile_u4 a = __builtin_amdgcn_raw_buffer_load_b128(rs, int(os), 0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] += bf16_lo(a[i]);
            v[2 * i + 1] += bf16_hi(a[i]);
        }
    }
    if constexpr (DBF) {
        const tile_u4 d = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                           pack_bf16x2(v[6], v[7])};
        __builtin_amdgcn_raw_buffer_store_b128(d, rd, int(od), 0, 0);
    } else {
        const tile_u4 d0 = {__builtin_bit_cast(uint32_t, v[0]), __builtin_bit_cast(uint32_t, v[1]),
                            __builtin_bit_cast(uint32_t, v[2]), __builtin_bit_cast(uint32_t, v[3])};
        const tile_u4 d1 = {__builtin_bit_cast(uint32_t, v[4]), __builtin_bit_cast(uint32_t, v[5]),
                            __builtin_bit_cast(uint32_t, v[6]), __builtin_bit_cast(uint32_t, v[7])};
        __builtin_amdgcn_raw_buffer_store_b128(d0, rd, int(od), 0, 0);
        __builtin_amdgcn_raw_buffer_store_b128(d1, rd, int(od + 16), 0, 0);
    }
}

// The same for four consecutive columns.
template <int SRC, bool DBF>
__device__ __forceinline__ void tile_store4_buf(__amdgpu_buffer_rsrc_t rs, uint32_t os, __amdgpu_buffer_rsrc_t rd,
                                                uint32_t od, const float* v4) {
    float v[4] = {v4[0], v4[1], v4[2], v4[3]};
    if constexpr (SRC == TSRC_F32) {
        const tile_u4 a = __builtin_amdgcn_raw_buffer_load_b128(rs, int(os), 0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t ai = a[i];  // a scalar copy: this compiler bit-casts a vector element as element 0
            v[i] += __builtin_bit_cast(float, ai);
        }
    } else if constexpr (SRC == TSRC_BF16) {
        const tile_u2 a = __builtin_amdgcn_raw_buffer_load_b64(rs, int(os), 0, 0);
        v[0] += bf16_lo(a[0]);
        v[1] += bf16_hi(a[0]);
        v[2] += bf16_lo(a[1]);
        v[3] += bf16_hi(a[1]);
    }
    if constexpr (DBF) {
        const tile_u2 d = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
        __builtin_amdgcn_raw_buffer_store_b64(d, rd, int(od), 0, 0);
    } else {
        const tile_u4 d = {__builtin_bit_cast(uint32_t, v[0]), __builtin_bit_cast(uint32_t, v[1]),
                           __builtin_bit_cast(uint32_t, v[2]), __builtin_bit_cast(uint32_t, v[3])};
        __builtin_amdgcn_raw_buffer_store_b128(d, rd, int(od), 0, 0);
    }
}

// Final combine and store of one token's output slice in the per-token emit
// layout (LANES lanes, NV vectors of EV elements): acc + source row, written to
// the destination row.
template <int LANES, int NV, bool WBF, int SRC, bool DBF>
__device__ __forceinline__ void store_token_sd(const void* src, void* dst, float* acc, int64_t tok, int sl) {
    constexpr int EV = WBF ? 8 : 4;
    constexpr int H = LANES * NV * EV;
#pragma unroll
    for (int c = 0; c < NV; ++c) {
        const int64_t e = tok * H + int64_t(c * LANES + sl) * EV;
#pragma unroll
        for (int q = 0; q < EV / 4; ++q) {
            float v[4] = {acc[c * EV + 4 * q], acc[c * EV + 4 * q + 1], acc[c * EV + 4 * q + 2],
                          acc[c * EV + 4 * q + 3]};
            if constexpr (SRC == TSRC_F32) {
                const float4 b = *reinterpret_cast<const float4*>(static_cast<const float*>(src) + e + 4 * q);
                v[0] += b.x; v[1] += b.y; v[2] += b.z; v[3] += b.w;
            } else if constexpr (SRC == TSRC_BF16) {
                const uint2 b = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(src) + e + 4 * q);
                v[0] += bf16_lo(b.x); v[1] += bf16_hi(b.x); v[2] += bf16_lo(b.y); v[3] += bf16_hi(b.y);
            }
            if constexpr (DBF)
                *reinterpret_cast<uint2*>(static_cast<uint16_t*>(dst) + e + 4 * q) =
                    make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
            else
                *reinterpret_cast<float4*>(static_cast<float*>(dst) + e + 4 * q) = make_float4(v[0], v[1], v[2], v[3]);
        }
    }
}

// Tree p.tile_tree of the layer: grid of one workgroup per leaf (XCD-affine by
// the subtree at the split level), then spill workgroups.  ELANES/ENV: the
// per-token emit layout for tokens of overflowing leaves; SRC/DBF: the output
// form (p.tile_src, p.tile_dst); P2: two bf16 parts of each activation (the
// layer's output is bf16) instead of three.  FSTEPS: MFMA steps of four levels
// with fp32 weights (at least (D + 4) / 4; unused with bf16 weights).  PAIR (fp32
// a workgroup per pair of sibling leaves, whose tokens share one list of tiles: the
// rows of levels 0 .. D-1 are common, and two virtual levels D and D+1 hold the left
// and the right leaf's row, each token's leaf activation going to its own leaf's
// level and a zero to the other (D + 2 <= 16 levels; with fp32 weights at least
// (D + 5) / 4 steps).
template <int CB, bool XBF, bool WBF, int ELANES, int ENV, int SRC, bool DBF, bool P2, int FSTEPS, bool PAIR = false>
__global__ __launch_bounds__(64 * tile_waves(16 * CB)) void tile_kernel(Params p, int leaf_blocks) {
    constexpr int H = 16 * CB;
    static_assert(H % 128 == 0, "128-column groups");
    constexpr int GROUPS = H / 128;
    constexpr int WAVES = tile_waves(H);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int D = p.depth, T = p.n_trees, tree = p.tile_tree;
    const int64_t L = int64_t(1) << D;
    const int64_t N = p.n_nodes;
    const void* const w_out = static_cast<const char*>(p.w_out) + int64_t(tree) * N * H * (WBF ? 2 : 4);

    // The per-token emit (all levels from global memory) of `count` tokens: token i is tok_of(i),
    // its activations at rec_of(i); groups g = first, first + stride, ... of this wave.
    auto emit_per_token = [&](int64_t count, int64_t first, int64_t stride, auto tok_of, auto rec_of) {
        using S = Shape<ELANES, ENV, XBF, WBF>;
        const int sl = lane % ELANES, sub = lane / ELANES;
        const int64_t groups = (count + S::TPW - 1) / S::TPW;
        for (int64_t g = first; g < groups; g += stride) {
            const int64_t idx_raw = g * S::TPW + sub;
            const bool valid = idx_raw < count;
            const int64_t idx = valid ? idx_raw : count - 1;
            const int64_t tok = tok_of(idx);
            const uint32_t leaf1 = uint32_t(p.ws_leaf[tok * T + tree]) + 1;
            const float* arec = rec_of(idx);
            const uint4* wout = reinterpret_cast<const uint4*>(w_out) + sl;
            float acc[S::E];
#pragma unroll
            for (int e = 0; e < S::E; ++e) acc[e] = 0.0f;
            emit_levels<ELANES, ENV, WBF>(
                acc, 0, D, [&](int l) { return wout + int64_t((leaf1 >> (D - l)) - 1) * S::ROWV; },
                [&](int l) { return wout + int64_t((leaf1 >> (D - l)) - 1) * S::ROWV; },
                [&](int l) { return arec[l]; });
            if (valid) store_token_sd<ELANES, ENV, WBF, SRC, DBF>(p.tile_src, p.tile_dst, acc, tok, sl);
        }
    };

    if (int(blockIdx.x) >= leaf_blocks) {
        // spilled tokens (their leaf overflowed): the per-token emit from their own records
        const int32_t* spill = p.bk_spill + int64_t(tree) * p.n_tokens;
        emit_per_token(int64_t(p.bk_nspill[tree]), int64_t(blockIdx.x - leaf_blocks) * WAVES + wave,
                       int64_t(gridDim.x - leaf_blocks) * WAVES, [&](int64_t i) { return int64_t(spill[i]); },
                       [&](int64_t i) { return p.ws_act + (int64_t(spill[i]) * T + tree) * (D + 1); });
        return;
    }

    // this workgroup's leaf (or pair of sibling leaves): XCD x (blockIdx % 8) takes the subtrees at
    // the split level that are x mod 8
    constexpr int LPW = PAIR ? 2 : 1;  // leaves per workgroup
    int64_t unit = blockIdx.x;
    if (p.split_level > 0) {
        const int64_t per = (int64_t(1) << (D - p.split_level)) / LPW;  // workgroups per subtree
        const int64_t x = blockIdx.x % XCDS, lb = blockIdx.x / XCDS;
        unit = (x + XCDS * (lb / per)) * per + lb % per;
    }
    const int64_t leaf = unit * LPW;  // the (left) leaf
    const int64_t bin = int64_t(tree) * L + leaf;
    const int32_t cnt_all = p.bk_count[bin];
    const int32_t cnt_r = PAIR ? p.bk_count[bin + 1] : 0;  // the right sibling's
    if (cnt_all == 0 && cnt_r == 0) return;  // workgroup-uniform
    const int cap = p.bk_cap;
    const int32_t* bucket = p.bk_tok + bin * cap;
    const float* act = p.bk_act + bin * int64_t(cap) * TILE_REC;
    if (cnt_all > cap || cnt_r > cap) {
        // An overflowing leaf: which of its tokens found a slot depends on the order of the walk's
        // atomics, so all of them take the per-token emit (these from their slots, the rest in the
        // spill workgroups) and every token's output is the same bits on every run.  A pair takes
        // it for both leaves (the counts, and so this choice, do not depend on that order).
        emit_per_token(int64_t(cnt_all < cap ? cnt_all : cap), wave, WAVES,
                       [&](int64_t i) { return int64_t(bucket[i]); }, [&](int64_t i) { return act + i * TILE_REC; });
        if constexpr (PAIR)
            emit_per_token(int64_t(cnt_r < cap ? cnt_r : cap), wave, WAVES,
                           [&](int64_t i) { return int64_t(bucket[cap + i]); },
                           [&](int64_t i) { return act + (cap + i) * TILE_REC; });
        return;
    }
    const int cnt = cnt_all + cnt_r;
    const uint32_t leaf1 = uint32_t(leaf + L);
    const int n = lane & 15, kq = lane >> 4;
    constexpr int SSZ = SRC == TSRC_BF16 ? 2 : 4;
    constexpr int DSZ = DBF ? 2 : 4;
    // Stores and source loads through buffer resources over the row blocks (the
    // host keeps B H 4 below 2^31): rows of empty slots are dropped by the hardware.
    const int row_elems = int(p.n_tokens * H);
    const __amdgpu_buffer_rsrc_t rdst = __builtin_amdgcn_make_buffer_rsrc(p.tile_dst, 0, row_elems * DSZ, 0x00020000);
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void*>(SRC != TSRC_NONE ? p.tile_src : p.tile_dst), 0, row_elems * SSZ, 0x00020000);
    // Every load below is in bounds and unconditional (slots and levels are
    // clamped; values past the count or past D are replaced by 0 where used), so
    // each path through a tile issues the same memory operations.

    // stores of one tile's outputs: lane (n, kq) holds tokens 4 kq + r of the
    // tile, whose ids come from the lanes that loaded them
    // Column layout in a 128-column group g.  With an fp32 destination (HALVES) MFMA column n of
    // block j is output column 128 g + 64 (j/4) + 4n + j%4, and the two halves (blocks 0..3, then
    // 4..7) are computed and stored in turn, so only four accumulators are live (fp32 weights: 74
    // VGPRs, six waves per SIMD); with a bf16 destination column 128 g + 8n + j, all eight blocks
    // at once, one 16-byte store per row (measured faster there).
    constexpr bool HALVES = !DBF;
    constexpr int NB = HALVES ? 4 : 8;  // blocks per store
    auto store_tile = [&](int32_t tok_a, const tile_v4f* acc, int64_t col) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int32_t tok = __shfl(tok_a, 4 * kq + r, 64);
            const int64_t e = int64_t(tok) * H + col;
            float v[NB];
#pragma unroll
            for (int j = 0; j < NB; ++j) v[j] = acc[j][r];
            const uint32_t od = tok >= 0 ? uint32_t(e * DSZ) : TILE_NO_ROW;
            const uint32_t os = tok >= 0 ? uint32_t(e * SSZ) : TILE_NO_ROW;
            if constexpr (HALVES)
                tile_store4_buf<SRC, DBF>(rsrc, os, rdst, od, v);
            else
                tile_store8_buf<SRC, DBF>(rsrc, os, rdst, od, v);
        }
    };

    constexpr int VL = PAIR ? 1 : 0;  // virtual levels past D (the right leaf's row)
    // PAIR: the leaf activation at its own leaf's (virtual) level, zero at the other's
    auto pick = [&](int v, float a, bool right, float aleaf) {
        if constexpr (PAIR) return v < D ? a : v == D ? (right ? 0.0f : a) : v == D + 1 && right ? aleaf : 0.0f;
        else return v <= D ? a : 0.0f;
    };
    // node of (virtual) level v <= D + VL: the ancestor of the leaf, or the right leaf
    auto row_node = [&](int v) { return v <= D ? int64_t(leaf1 >> (D - v)) - 1 : int64_t(leaf1); };
    if constexpr (WBF) {
        constexpr int PARTS = P2 ? 2 : 3;
        const int h = kq & 1, part = kq >> 1;
        struct Raw {
            int32_t tok;
            float4 a0, a1;  // activations of levels 8h .. 8h+7
            bool right;     // PAIR: the token is in the right leaf
            float aleaf;    // PAIR: its leaf activation
        };
        // token id of list entry t0 + n (PAIR: the left leaf's slots, then the right leaf's)
        auto load_tile = [&](int t0, Raw& r) {
            const int i = t0 + n;
            r.right = PAIR && i >= cnt_all;
            const int j = r.right ? i - cnt_all : i;
            const int slot = (j < cap ? j : cap - 1) + (r.right ? cap : 0);
            r.tok = bucket[slot];
            const float* recp = act + int64_t(slot) * TILE_REC;
            const float4* rec = reinterpret_cast<const float4*>(recp + 8 * h);
            r.a0 = rec[0];
            r.a1 = rec[1];
            r.aleaf = PAIR ? recp[D] : 0.0f;
        };
        for (int g = wave; g < GROUPS; g += WAVES) {
            const int64_t col = int64_t(g) * 128 + (HALVES ? 4 : 8) * n;
            // B operands: bj[j] holds the column of block j (see the layout above) of the rows of
            // levels 8h .. 8h+7 (levels past D repeat the leaf row: their activations are 0)
            uint4 bj[8];
            if constexpr (HALVES) {
                uint2 row[2][8];
#pragma unroll
                for (int c = 0; c < 2; ++c)
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        const int lvl = 8 * h + i <= D + VL ? 8 * h + i : D + VL;
                        row[c][i] = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(w_out) +
                                                                    row_node(lvl) * H + col + 64 * c);
                    }
#pragma unroll
                for (int c = 0; c < 2; ++c)
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        uint32_t w4[4];
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const uint32_t lo = j / 2 ? row[c][2 * q].y : row[c][2 * q].x;
                            const uint32_t hi = j / 2 ? row[c][2 * q + 1].y : row[c][2 * q + 1].x;
                            w4[q] = (j & 1) ? (lo >> 16) | (hi & 0xffff0000u) : (lo & 0xffffu) | (hi << 16);
                        }
                        bj[4 * c + j] = make_uint4(w4[0], w4[1], w4[2], w4[3]);
                    }
            } else {
                uint4 row[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int lvl = 8 * h + i <= D + VL ? 8 * h + i : D + VL;
                    row[i] = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(w_out) + row_node(lvl) * H + col);
                }
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    uint32_t w4[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const uint32_t lo = word(row[2 * q], j / 2), hi = word(row[2 * q + 1], j / 2);
                        w4[q] = (j & 1) ? (lo >> 16) | (hi & 0xffff0000u) : (lo & 0xffffu) | (hi << 16);
                    }
                    bj[j] = make_uint4(w4[0], w4[1], w4[2], w4[3]);
                }
            }
            auto tile = [&](int t0, const Raw& cur) {
                const bool in = t0 + n < cnt;
                const int32_t tok_a = in ? cur.tok : -1;
                // this lane's parts of its eight activations
                float av[8] = {cur.a0.x, cur.a0.y, cur.a0.z, cur.a0.w, cur.a1.x, cur.a1.y, cur.a1.z, cur.a1.w};
                uint32_t p0[4], p1[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float x0 = in ? pick(8 * h + 2 * q, av[2 * q], cur.right, cur.aleaf) : 0.0f;
                    const float x1 = in ? pick(8 * h + 2 * q + 1, av[2 * q + 1], cur.right, cur.aleaf) : 0.0f;
                    const uint32_t hi = pack_bf16x2(x0, x1);
                    const float r0 = x0 - bf16_lo(hi), r1 = x1 - bf16_hi(hi);
                    const uint32_t mid = pack_bf16x2(r0, r1);
                    if constexpr (PARTS == 3) {
                        const uint32_t lo = pack_bf16x2(r0 - bf16_lo(mid), r1 - bf16_hi(mid));
                        p0[q] = part == 0 ? hi : mid;
                        p1[q] = part == 0 ? lo : 0u;
                    } else {
                        p0[q] = part == 0 ? hi : mid;
                    }
                }
                const bf16x8_t a0 = __builtin_bit_cast(bf16x8_t, make_uint4(p0[0], p0[1], p0[2], p0[3]));
                // the halves in turn (HALVES) or all eight blocks at once
#pragma unroll
                for (int c = 0; c < 8 / NB; ++c) {
                    tile_v4f acc[NB];
#pragma unroll
                    for (int j = 0; j < NB; ++j) {
                        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            a0, __builtin_bit_cast(bf16x8_t, bj[NB * c + j]), tile_v4f{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                    }
                    if constexpr (PARTS == 3) {
                        const bf16x8_t a1 = __builtin_bit_cast(bf16x8_t, make_uint4(p1[0], p1[1], p1[2], p1[3]));
#pragma unroll
                        for (int j = 0; j < NB; ++j)
                            acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                a1, __builtin_bit_cast(bf16x8_t, bj[NB * c + j]), acc[j], 0, 0, 0);
                    }
                    store_tile(tok_a, acc, col + 64 * c);
                }
            };
            // two operand sets in turn: the next tile's loads are in flight while
            // this one runs, and no register copy makes the wait early
            Raw r0, r1;
            load_tile(0, r0);
            for (int t0 = 0;;) {
                load_tile(t0 + 16, r1);
                tile(t0, r0);
                if ((t0 += 16) >= cnt) break;
                load_tile(t0 + 16, r0);
                tile(t0, r1);
                if ((t0 += 16) >= cnt) break;
            }
        }
    } else {
        const int steps = (D + 4 + VL) / 4;
        // (virtual) level of step s for this lane, clamped to D + VL
        int lvl_c[FSTEPS];
#pragma unroll
        for (int s = 0; s < FSTEPS; ++s) lvl_c[s] = 4 * s + kq <= D + VL ? 4 * s + kq : D + VL;
        struct Raw {
            int32_t tok;
            float a[FSTEPS];
            bool right;  // PAIR: the token is in the right leaf
        };
        // token id of list entry t0 + n (PAIR: the left leaf's slots, then the right leaf's) and
        // its activations at levels 4s + kq (the leaf's at the virtual level)
        auto load_tile = [&](int t0, Raw& r) {
            const int i = t0 + n;
            r.right = PAIR && i >= cnt_all;
            const int j = r.right ? i - cnt_all : i;
            const int slot = (j < cap ? j : cap - 1) + (r.right ? cap : 0);
            r.tok = bucket[slot];
            const float* rec = act + int64_t(slot) * TILE_REC;
#pragma unroll
            for (int s = 0; s < FSTEPS; ++s) r.a[s] = rec[lvl_c[s] <= D ? lvl_c[s] : D];
        };
        for (int g = wave; g < GROUPS; g += WAVES) {
            const int64_t col = int64_t(g) * 128 + (HALVES ? 4 : 8) * n;
            // B operand: this lane's weights of the row at level 4s + kq for its eight blocks (see
            // the layout above), kept as loaded for all of the leaf's tiles
            float4 w[FSTEPS][2];
#pragma unroll
            for (int s = 0; s < FSTEPS; ++s) {
                const int64_t at = row_node(lvl_c[s]) * H + col;
                w[s][0] = *reinterpret_cast<const float4*>(static_cast<const float*>(w_out) + at);
                w[s][1] = *reinterpret_cast<const float4*>(static_cast<const float*>(w_out) + at + (HALVES ? 64 : 4));
            }
            auto tile = [&](int t0, const Raw& cur) {
                const bool in = t0 + n < cnt;
                const int32_t tok_a = in ? cur.tok : -1;
                // the halves in turn (HALVES) or all eight blocks at once
#pragma unroll
                for (int c = 0; c < 8 / NB; ++c) {
                    tile_v4f acc[NB];
#pragma unroll
                    for (int j = 0; j < NB; ++j) acc[j] = tile_v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int s = 0; s < FSTEPS; ++s) {
                        if (s < steps) {
                            const float a = in ? pick(4 * s + kq, cur.a[s], cur.right, cur.a[s]) : 0.0f;
#pragma unroll
                            for (int j = 0; j < NB; ++j)
                                acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                    a, fword(w[s][(NB * c + j) / 4], (NB * c + j) % 4), acc[j], 0, 0, 0);
                        }
                    }
                    store_tile(tok_a, acc, col + 64 * c);
                }
            };
            Raw r0, r1;
            load_tile(0, r0);
            for (int t0 = 0;;) {
                load_tile(t0 + 16, r1);
                tile(t0, r0);
                if ((t0 += 16) >= cnt) break;
                load_tile(t0 + 16, r0);
                tile(t0, r1);
                if ((t0 += 16) >= cnt) break;
            }
        }
    }
}

__global__ __launch_bounds__(256) void fill_i32_kernel(int32_t* a, int64_t n) {
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) a[i] = 0;
}

// ----------------------------------------------------------------------------
// STACK: several layers x <- x + FFF_i(norm_i(x)) in one persistent kernel
// ----------------------------------------------------------------------------
//
// Tokens are independent through the whole stack, so a group keeps its token's
// x in registers from the first layer to the last: x is read once and y
// written once.  Each workgroup takes chunks of WAVES token groups and runs
// every layer on the chunk; the top levels of the current layer are staged
// into LDS between two barriers, so all waves of a block move through the
// layers together.  Per layer the arithmetic is exactly the descent kernel's
// (same loads, same reduction and accumulation order, the residual sum rounded
// to the storage type), so the stack equals chained single-layer calls bit for
// bit.  NORM: x is held as fp32 values of the storage type (p.x_bf16 says
// which) and each layer normalises a copy.
template <int LANES, int NV, bool XBF, bool WBF, int BLOCK, bool NORM>
__global__ __launch_bounds__(BLOCK) void stack_kernel(StackParams sp) {
    static_assert(!(NORM && XBF), "normalised inputs are held in fp32");
    using S = Shape<LANES, NV, XBF, WBF>;
    using XS = XRegs<LANES, NV, XBF, WBF>;
    constexpr int WAVES = BLOCK / 64;
    extern __shared__ uint4 lds_rows[];  // [T][Nk][2][ROWV] of the current layer

    const Params& p = sp.p;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int sl = lane % LANES;
    const int sub = lane / LANES;
    const int T = p.n_trees, D = p.depth, K = p.lds_levels;
    const int64_t N = p.n_nodes;
    const int Nk = (1 << K) - 1;
    const int KD = K < D + 1 ? K : D + 1;
    const bool to_bf16 = p.y_bf16;
    const int64_t n_groups = (p.n_tokens + S::TPW - 1) / S::TPW;
    const int64_t n_chunks = (n_groups + WAVES - 1) / WAVES;
    // The chunk loop and the layer loop have the same trip counts in every wave
    // of the block, so every wave reaches every barrier.
    for (int64_t ch = blockIdx.x; ch < n_chunks; ch += gridDim.x) {
        const int64_t g = ch * WAVES + wave;
        const bool active = g < n_groups;  // wave-uniform
        const int64_t slot_raw = g * S::TPW + sub;
        const bool valid = slot_raw < p.n_tokens;
        const int64_t tok = valid ? slot_raw : p.n_tokens - 1;
        XS xs;
        if (active) {
            if constexpr (NORM) xs.load_widen(p.x, p.x_bf16, tok, sl);
            else xs.load(p.x, tok, sl);
        }
        for (int li = 0; li < sp.n_layers; ++li) {
            const LayerPtrs L = sp.layer[li];
            if (K > 0) {
                __syncthreads();  // the previous layer's rows are no longer read
                stage_rows<S::ROWV, BLOCK>(lds_rows, L.w_in, T, N, Nk, 2 * S::ROWV, 0);
                stage_rows<S::ROWV, BLOCK>(lds_rows, L.w_out, T, N, Nk, 2 * S::ROWV, S::ROWV);
                __syncthreads();
            }
            if (!active) continue;
            float acc[S::E];
#pragma unroll
            for (int e = 0; e < S::E; ++e) acc[e] = 0.0f;
            XS u = xs;
            if constexpr (NORM) layer_norm_regs<LANES, NV, WBF>(u.f, L.gamma, L.beta, p.norm_eps, sl);
            int32_t* nodes = p.nodes_out ? p.nodes_out + li * sp.rec_stride : nullptr;
            float* logits = p.logits_out ? p.logits_out + li * sp.rec_stride : nullptr;
            for (int t = 0; t < T; ++t) {
                const uint4* win = reinterpret_cast<const uint4*>(L.w_in) + int64_t(t) * N * S::ROWV + sl;
                const uint4* wout = reinterpret_cast<const uint4*>(L.w_out) + int64_t(t) * N * S::ROWV + sl;
                const uint4* lrows = lds_rows + int64_t(t) * Nk * 2 * S::ROWV + sl;
                LevelRegs<LANES> lv;
                const uint32_t leaf1 = walk_tree<LANES, NV, XBF, WBF>(u, lrows, 2 * S::ROWV, win, KD, D, sl, lv);
                LevelRegs<LANES> av;
#pragma unroll
                for (int r = 0; r < LevelRegs<LANES>::NR; ++r) av.v[r] = activation(lv.v[r], p.act);
                if ((nodes || logits) && valid) write_records<LANES>(nodes, logits, p, lv, leaf1, tok, t, sl);
                const uint4* lout = lrows + S::ROWV;
                emit_levels<LANES, NV, WBF>(
                    acc, KD, D, [&](int l) { return lout + int64_t((leaf1 >> (D - l)) - 1) * 2 * S::ROWV; },
                    [&](int l) { return wout + int64_t((leaf1 >> (D - l)) - 1) * S::ROWV; },
                    [&](int l) { return av.get(l, lane); });
            }
            if (li + 1 < sp.n_layers) {
                // x_{i+1} = storage rounding of x_i + FFF_i, as a stored-and-reloaded residual would be
#pragma unroll
                for (int c = 0; c < NV; ++c)
#pragma unroll
                    for (int e = 0; e < S::EV; ++e) acc[c * S::EV + e] += xs.elem(c, e);
                xs.set_from(acc, to_bf16);
            } else if (valid) {
                store_output<LANES, NV, WBF>(p, xs, acc, tok, sl);  // out_mode is RESIDUAL
            }
        }
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
        const int64_t tok = slot;
        const int64_t xoff = tok * H;
        // LayerNorm statistics of the token (norm = 1); u_h is formed on the fly below
        float mean = 0.0f, rstd = 1.0f;
        if (p.norm) {
            float s = 0.0f;
            for (int h = lane; h < H; h += 64) s += load_elem<XBF>(p.x, xoff + h);
            mean = group_sum<64>(s) / float(H);
            float q = 0.0f;
            for (int h = lane; h < H; h += 64) {
                const float d = load_elem<XBF>(p.x, xoff + h) - mean;
                q = __builtin_fmaf(d, d, q);
            }
            rstd = 1.0f / sqrtf(group_sum<64>(q) / float(H) + p.norm_eps);
        }
        auto input = [&](int h) {
            const float v = load_elem<XBF>(p.x, xoff + h);
            if (!p.norm) return v;
            return __builtin_fmaf((v - mean) * rstd, p.gamma ? p.gamma[h] : 1.0f, p.beta ? p.beta[h] : 0.0f);
        };
        for (int t = 0; t < T; ++t) {
            int64_t n = 0;
            for (int l = 0; l <= D; ++l) {
                const int64_t woff = (int64_t(t) * N + n) * H;
                float part = 0.0f;
                for (int h = lane; h < H; h += 64)
                    part = __builtin_fmaf(input(h), load_elem<WBF>(p.w_in, woff + h), part);
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
// the scratch of the entry point that allocates nothing
// ----------------------------------------------------------------------------

// One copy per GPU, zero at load and afterwards holding whatever the last call
// left; the kernels clear what must start at zero (the bucket counts) on every
// call.  In host code `scratch` names a host-side stand-in: only the address
// from hipGetSymbolAddress may be handed to kernels.
static __device__ __align__(256) unsigned char scratch[STATIC_SCRATCH_BYTES];

namespace {
constexpr int kScratchDevices = 64;
std::once_flag g_scratch_once[kScratchDevices];
void* g_scratch_ptr[kScratchDevices];
hipError_t g_scratch_err[kScratchDevices];
}  // namespace

hipError_t static_scratch(int device, void** ptr) {
    if (device < 0 || device >= kScratchDevices) return hipErrorInvalidDevice;
    std::call_once(g_scratch_once[device], [&] {
        void* p = nullptr;
        g_scratch_err[device] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_scratch_ptr[device] = g_scratch_err[device] == hipSuccess ? p : nullptr;
    });
    *ptr = g_scratch_ptr[device];
    return g_scratch_err[device];
}

// ----------------------------------------------------------------------------
// planning
// ----------------------------------------------------------------------------

constexpr int BLOCK = 256;
constexpr size_t DESCENT_LDS_BUDGET = 32 * 1024;  // per 256-thread block: keeps 4-5 blocks per CU
constexpr int WALK_BLOCK = 512;                     // walk workgroups: twice the rows in LDS per wave
constexpr size_t WALK_LDS_BUDGET = 48 * 1024;     // per 512-thread walk block: three blocks per CU
// Walk workgroups larger than WALK_BLOCK, where measured faster: at four waves per SIMD (16-lane
// walks of fp32 x or fp32 weights at hidden 768, LayerNorm walks of bf16 weights) one 1024-thread
// block per CU; at five (fp32 weights at hidden 1024) two of 640 threads.  Fewer, larger blocks at
// the same waves per CU hold one more level of rows in LDS.  (Two 640-thread blocks for the bf16
// walks of hidden 1024 and 4096 were slower: grouped at hidden 1024, depth 11, 32768 tokens
// 80.9 -> 87.8 us.)
constexpr int WALK_BLOCK_WIDE = 1024;
constexpr int WALK_BLOCK_5 = 640;
static size_t walk_lds_budget(int block) {
    return block == WALK_BLOCK ? WALK_LDS_BUDGET : block == WALK_BLOCK_5 ? size_t(78) << 10 : size_t(96) << 10;
}
constexpr size_t EMIT_LDS_BUDGET = 32 * 1024;
constexpr int GENERIC_MAX_PAIRS = 2048;

struct Variant {
    int hidden;
    bool xbf, wbf;
    int lanes;
    int walk_lanes;  // the walk kernel's lanes per token (its own registers: x and one row, no output)
    int walk_block;  // its workgroup size (WALK_BLOCK, or WALK_BLOCK_WIDE for walks of four waves per SIMD)
    int walk_norm_block;  // the same for the LayerNorm walk (x widened to fp32)
    int emit_lanes;  // the emit has no cross-lane reduction: wider groups hold fewer registers per lane
    const void* descent;
    const void* walk;
    const void* emit;
    const void* tile[3][3];  // [source TSRC_*][form: fp32 dst 3 parts, fp32 dst 2 parts, bf16 dst 2 parts]
    const void* tile_deep[3][3];  // the same for fp32 weights deeper than TILE_STEPS_SHALLOW steps
    const void* tile_pair[3][3];  // a workgroup per pair of sibling leaves
    const void* stack;
    // LayerNorm prologue: x widened to fp32 whatever its storage type
    const void* descent_norm;
    const void* walk_norm;
    const void* stack_norm;
    const char* name;
};

#define FFF_K(...) reinterpret_cast<const void*>(&__VA_ARGS__)
#define FFF_TILES(H, XB, WB, EL, ENV, SRC, FS)                                                                \
    {FFF_K(tile_kernel<H / 16, XB, WB, EL, ENV, SRC, false, false, FS>),                                   \
     FFF_K(tile_kernel<H / 16, XB, WB, EL, ENV, SRC, false, true, FS>),                                    \
     FFF_K(tile_kernel<H / 16, XB, WB, EL, ENV, SRC, true, true, FS>)}
// leaf pairs
#define FFF_TILES_PAIR(H, XB, WB, EL, ENV, SRC)                                                              \
    {FFF_K(tile_kernel<H / 16, XB, WB, EL, ENV, SRC, false, false, TILE_MAX_STEPS, true>),                 \
     FFF_K(tile_kernel<H / 16, XB, WB, EL, ENV, SRC, false, true, TILE_MAX_STEPS, true>),                  \
     FFF_K(tile_kernel<H / 16, XB, WB, EL, ENV, SRC, true, true, TILE_MAX_STEPS, true>)}
// bf16 weights take one instantiation for both arrays
#define FFF_TILE_STEPS(WB) ((WB) ? TILE_MAX_STEPS : TILE_STEPS_SHALLOW)
#define FFF_VARIANT(H, XB, WB, L, NV, WL, WNV, WBLK, WNBLK, EL, ENV)                                         \
    Variant {                                                                                                 \
        H, XB, WB, L, WL, WBLK, WNBLK, EL, FFF_K(descent_kernel<L, NV, XB, WB, BLOCK, false>),                \
            FFF_K(walk_kernel<WL, WNV, XB, WB, WBLK, false>), FFF_K(emit_kernel<EL, ENV, XB, WB, BLOCK>),        \
            {FFF_TILES(H, XB, WB, EL, ENV, TSRC_NONE, FFF_TILE_STEPS(WB)),                                    \
             FFF_TILES(H, XB, WB, EL, ENV, TSRC_F32, FFF_TILE_STEPS(WB)),                                     \
             FFF_TILES(H, XB, WB, EL, ENV, TSRC_BF16, FFF_TILE_STEPS(WB))},                                   \
            {FFF_TILES(H, XB, WB, EL, ENV, TSRC_NONE, TILE_MAX_STEPS),                                        \
             FFF_TILES(H, XB, WB, EL, ENV, TSRC_F32, TILE_MAX_STEPS),                                         \
             FFF_TILES(H, XB, WB, EL, ENV, TSRC_BF16, TILE_MAX_STEPS)},                                       \
            {FFF_TILES_PAIR(H, XB, WB, EL, ENV, TSRC_NONE), FFF_TILES_PAIR(H, XB, WB, EL, ENV, TSRC_F32),      \
             FFF_TILES_PAIR(H, XB, WB, EL, ENV, TSRC_BF16)},                                                  \
            FFF_K(stack_kernel<L, NV, XB, WB, BLOCK, false>), FFF_K(descent_kernel<L, NV, false, WB, BLOCK, true>), \
            FFF_K(walk_kernel<WL, WNV, false, WB, WNBLK, true>), FFF_K(stack_kernel<L, NV, false, WB, BLOCK, true>), \
            "lanes=" #L ",nv=" #NV ",x_bf16=" #XB ",w_bf16=" #WB                                              \
    }

static const Variant kVariants[] = {
    // H = 768 (BERT-base width); the emit takes 32 (bf16 W) or 64 (fp32 W) lanes per token, the
    // walk 16 (with fp32 W: 124 VGPRs and four waves per SIMD, 64 tokens in flight per CU against
    // 48 with 32 lanes; the fused kernel keeps 32, its output accumulators need the registers)
    FFF_VARIANT(768, true, true, 16, 6, 16, 6, WALK_BLOCK, WALK_BLOCK_WIDE, 32, 3),
    FFF_VARIANT(768, false, true, 16, 6, 16, 6, WALK_BLOCK_WIDE, WALK_BLOCK_WIDE, 32, 3),
    FFF_VARIANT(768, false, false, 32, 6, 16, 12, WALK_BLOCK_WIDE, WALK_BLOCK_WIDE, 64, 3),
    FFF_VARIANT(768, true, false, 32, 6, 16, 12, WALK_BLOCK_WIDE, WALK_BLOCK_WIDE, 64, 3),
    // H = 1024
    FFF_VARIANT(1024, true, true, 16, 8, 16, 8, WALK_BLOCK, WALK_BLOCK, 32, 4),
    FFF_VARIANT(1024, false, true, 16, 8, 16, 8, WALK_BLOCK, WALK_BLOCK, 32, 4),
    FFF_VARIANT(1024, false, false, 32, 8, 32, 8, WALK_BLOCK_5, WALK_BLOCK_5, 64, 4),
    FFF_VARIANT(1024, true, false, 32, 8, 32, 8, WALK_BLOCK_5, WALK_BLOCK_5, 64, 4),
    // H = 4096 (LLM width)
    FFF_VARIANT(4096, true, true, 64, 8, 64, 8, WALK_BLOCK, WALK_BLOCK, 64, 8),
    FFF_VARIANT(4096, false, true, 64, 8, 64, 8, WALK_BLOCK, WALK_BLOCK, 64, 8),
    FFF_VARIANT(4096, false, false, 64, 16, 64, 16, WALK_BLOCK, WALK_BLOCK, 64, 16),
    FFF_VARIANT(4096, true, false, 64, 16, 64, 16, WALK_BLOCK, WALK_BLOCK, 64, 16),
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

static size_t rows_lds_bytes(const Params& p, int levels, int matrices) {
    if (levels <= 0) return 0;
    const size_t row_bytes = size_t(p.hidden) * (p.w_bf16 ? 2 : 4);
    return size_t(p.n_trees) * ((size_t(1) << levels) - 1) * matrices * row_bytes;
}

// Levels to stage: the caller's explicit k (checked), none (-1), or the most that fit the budget.
static int pick_levels(const Params& p, int req, int matrices, size_t budget, size_t limit, bool* ok) {
    *ok = true;
    if (req < 0) return 0;
    if (req > 0) {
        if (req > p.depth + 1 || rows_lds_bytes(p, req, matrices) > limit) *ok = false;
        return req;
    }
    int k = 0;
    while (k < p.depth + 1 && k < 20 && rows_lds_bytes(p, k + 1, matrices) <= budget) ++k;
    return k;
}

static int resident_grid(const DeviceInfo& dev, const void* kernel, size_t lds, int64_t want, int block = BLOCK) {
    const int64_t resident = int64_t(dev.cu_count) * blocks_per_cu(dev.device, kernel, block, lds);
    return int(std::max<int64_t>(1, std::min(want, resident)));
}

int default_split_level(int32_t depth, int32_t n_trees) {
    // Tokens are grouped by tree 0 only; with several trees the other trees' rows are not
    // XCD-local and the grouping costs more than it saves (measured), so keep token order.
    return depth >= 3 && n_trees == 1 ? std::min(depth, 5) : 0;
}

static size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

size_t grouped_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t /*split_level*/) {
    const size_t recs = size_t(n_tokens) * size_t(n_trees);
    return align256(recs * size_t(depth + 1) * sizeof(float)) + align256(recs * sizeof(int32_t));
}

// Tiled mode: up to TILE_MAX_TREES trees, depth 5..15 (records of TILE_REC levels), hidden a
// multiple of 128.
constexpr int TILE_MAX_TREES = 16;
static bool tiled_shape(int32_t depth, int32_t n_trees, int32_t hidden) {
    return n_trees >= 1 && n_trees <= TILE_MAX_TREES && depth >= 5 && depth < TILE_REC && hidden % 128 == 0;
}

// Bucket capacity: four times the mean tokens per leaf, at least one tile of 16, a multiple of 16.
static int32_t tile_cap(int64_t n_tokens, int32_t depth) {
    const int64_t leaves = int64_t(1) << depth;
    const int64_t mean = (n_tokens + leaves - 1) / leaves;
    return int32_t(std::max<int64_t>(16, (4 * mean + 15) / 16 * 16));
}

// Tiled workspace, in order: token records and leaves (as grouped; the records
// are used by spilled tokens only), bucket counts + spill counts, bucket token
// ids, spill lists, bucket activation records, and with several trees an fp32
// [B, H] running sum (used when y is bf16); B is at most one chunk of tokens.
size_t tiled_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t hidden) {
    if (!tiled_shape(depth, n_trees, hidden)) return 0;
    n_tokens = std::min(n_tokens, tile_chunk_tokens(hidden));
    const size_t T = size_t(n_trees);
    const size_t leaves = size_t(1) << depth;
    const size_t cap = size_t(tile_cap(n_tokens, depth));
    return grouped_workspace_bytes(n_tokens, depth, n_trees, 0) + align256(T * (leaves + 1) * sizeof(int32_t)) +
           align256(T * leaves * cap * sizeof(int32_t)) + align256(T * size_t(n_tokens) * sizeof(int32_t)) +
           align256(T * leaves * cap * size_t(TILE_REC) * sizeof(float)) +
           (T > 1 ? align256(size_t(n_tokens) * size_t(hidden) * sizeof(float)) : 0);
}

static const Variant* find_variant(const Params& p) {
    for (const auto& c : kVariants)
        if (c.hidden == p.hidden && c.xbf == bool(p.x_bf16) && c.wbf == bool(p.w_bf16)) return &c;
    return nullptr;
}

static int64_t token_groups(const Params& p, int lanes) { return (p.n_tokens + 64 / lanes - 1) / (64 / lanes); }

// What the layer adds its result to (see TSRC_*): x (residual), y (accumulate) or nothing.
static int out_src_kind(const Params& p) {
    if (p.out_mode == OUT_RESIDUAL) return p.x_bf16 ? TSRC_BF16 : TSRC_F32;
    if (p.out_mode == OUT_ACCUMULATE) return p.y_bf16 ? TSRC_BF16 : TSRC_F32;
    return TSRC_NONE;
}

// Output form of tree t's tile launch: the first tree adds the layer's source; later trees add
// the fp32 running sum; the last writes y, the others the running sum (fp32).  Two activation
// parts when the layer's output is bf16.
static int tile_src_kind(const Params& p, int t) { return t > 0 ? int(TSRC_F32) : out_src_kind(p); }

static const void* tile_kernel_for(const Variant& v, const Params& p, int t, bool pair) {
    const bool last = t == p.n_trees - 1;
    const int form = last && p.y_bf16 ? 2 : p.y_bf16 ? 1 : 0;
    if (pair) return v.tile_pair[tile_src_kind(p, t)][form];
    return (p.depth + 4) / 4 <= TILE_STEPS_SHALLOW ? v.tile[tile_src_kind(p, t)][form]
                                                   : v.tile_deep[tile_src_kind(p, t)][form];
}

// Leaf pairs: when a leaf holds fewer tokens than one 16-row tile on average (depth 11, 16384
// tokens: 8), and the two virtual rows still fit the MFMA steps.
static bool tile_pairs(const Params& p) {
    return p.depth >= 5 && p.depth + 2 <= 4 * TILE_MAX_STEPS && p.n_tokens < (int64_t(16) << p.depth);
}

// The walk launch of the grouped and tiled plans: with 2, 4 or 8 trees one tree per workgroup
// (by XCD), whose top levels then get the whole LDS budget; otherwise every tree per token.
static bool plan_walk(const Params& p, const Variant& v, int lds_levels_req, const DeviceInfo& dev, Plan* plan,
                      Launch& W) {
    const bool affine = p.n_trees > 1 && XCDS % p.n_trees == 0;
    Params one = p;
    if (affine) one.n_trees = 1;
    bool ok;
    const int blk = p.norm ? v.walk_norm_block : v.walk_block;
    const int kw = pick_levels(one, lds_levels_req, 1, walk_lds_budget(blk), dev.lds_per_block, &ok);
    if (!ok) return false;
    plan->lds_levels = kw;
    plan->walk_affine = affine;
    W.kernel = p.norm ? v.walk_norm : v.walk;
    W.block = blk;
    W.lds_bytes = rows_lds_bytes(one, kw, 1);
    const int64_t groups = token_groups(p, v.walk_lanes) * (affine ? p.n_trees : 1);
    int64_t want = (groups + blk / 64 - 1) / (blk / 64);
    if (affine) want = (want + XCDS - 1) / XCDS * XCDS;
    W.grid = resident_grid(dev, W.kernel, W.lds_bytes, want, blk);
    if (affine) W.grid = std::max(XCDS, W.grid / XCDS * XCDS);  // every tree gets the same XCDs' worth
    return true;
}

int plan_forward(const Params& p, int mode, int lds_levels_req, int split_level_req, size_t workspace_bytes,
                 const DeviceInfo& dev, Plan* plan, bool masked_ok) {
    *plan = Plan{};
    const Variant* v = find_variant(p);
    if (mode == MODE_AUTO) {
        // Measured on MI355X (hidden 768 / 1024 / 4096, depth 2..15, 256..128K tokens, 1..3072
        // trees, bf16 and fp32 weights):
        // * at most 4 trees of depth >= 5 and 256 token-tree pairs (32 at hidden 4096): a
        //   workgroup per token evaluating whole subtrees (depth 11, 256 tokens: 10.5 against
        //   12.3 us);
        // * shallow layers with many trees as dense products (masked; see its constants);
        // * single trees of depth 9..15 leaf-tiled on MFMA with at least 8 tokens per leaf from
        //   48M input elements, or 16 per leaf from 16M (depth 11 at 32768 tokens: 51 against
        //   60 us in bf16); at depth 9 in bf16 only from 96M (the fused kernel stays ahead below);
        //   with fp32 weights at depth >= 11 from 8 per leaf (16384 tokens: 64 against 67 us per
        //   call, 61 against 67 back to back), and from 2 per leaf where sibling leaves share a
        //   workgroup (depth <= 14) and the input has 12M elements (depth 12, 16384 tokens: 65
        //   against 75 us grouped; depth 14, 65536 tokens: 301 against 368; hidden 4096, depth 11,
        //   4096 tokens: 111 against 124 fused; one per leaf loses: depth 14, 16384 tokens, 123
        //   against 104 grouped); in bf16 at depth >= 11 from 4 per leaf when the
        //   rows are long (hidden 4096, 8192 tokens: 107 against 113 us; at hidden 768 the
        //   grouped emit is ahead at 4 per leaf, depth 13: 80 against 86 us);
        // * other single trees grouped by subtree at depth >= 11 from 48M elements, or from 16384
        //   tokens with fp32 weights (depth 11: 66 against 70 us) or 24M elements in bf16, and
        //   with fp32 weights at depth >= 5 from 65536 tokens (5-7 % ahead of the fused kernel);
        // * 2, 4 or 8 trees of depth >= 7 (the walk tree-affine: the workgroups of an XCD walk
        //   one tree, its top levels in LDS and its deep rows in that XCD's L2): with fp32 weights
        //   leaf-tiled at depth >= 11 from 8 tokens per leaf, at depth >= 10 from 16 and at
        //   depth >= 9 from 32 per leaf (eight trees of depth 11, 65536 tokens: 1481 against
        //   2556 us fused; four of depth 9: 554 against 665 at 65536 tokens, 149 against 160 at
        //   16384; four of depth 10, 16384 tokens: 174 against 200), else grouped from
        //   65536 tokens (16384 with 8 trees); with bf16 weights grouped for 8 trees, for 4 from
        //   4096 tokens at depth >= 8 (65536 at depth 7), for 2 from 65536 tokens at depth >= 8
        //   (four trees of depth 9, 65536 tokens: 272 against 306 us);
        // * eight trees at small batches grouped, its walk tree-affine (one tree per XCD: eight
        //   times the fused kernel's workgroups, each with one tree's top levels in LDS): up to
        //   2048 tokens in bf16 (4096 at depth >= 6; depth 5, 1024 tokens: 22 against 31 us),
        //   1024 with fp32 weights;
        // * else the fused descent kernel.
        const bool big = p.n_trees == 1 && p.n_tokens * int64_t(p.hidden) >= (int64_t(48) << 20);
        const int64_t tiled_ws = int64_t(tiled_workspace_bytes(p.n_tokens, p.depth, p.n_trees, p.hidden));
        const int64_t grouped_ws = int64_t(grouped_workspace_bytes(p.n_tokens, p.depth, p.n_trees, 0));
        const int64_t masked_ws = int64_t(masked_workspace_bytes(p.n_tokens, p.depth, p.n_trees, p.hidden));
        // Shallow layers: a token uses (D+1)/(2^(D+1)-1) of the nodes, at least 9.5 % at depth
        // <= 5, where bf16 MFMA products beat the walk of 16 trees or more; fp32 products (about
        // 125 TFLOP/s against the walk's 16) win down to 16 % (depth <= 4) from 32 trees.
        const int64_t elems = p.n_tokens * int64_t(p.hidden);
        const bool one = p.n_trees == 1;
        const bool affine = p.n_trees > 1 && XCDS % p.n_trees == 0;  // 2, 4 or 8 trees: tree-affine walk
        if (subtree_auto(p))
            mode = MODE_SUBTREE;
        else if (masked_ok && masked_shape(p) &&
                 (p.w_bf16 ? p.depth <= MASKED_AUTO_DEPTH &&
                                 (p.n_trees >= MASKED_AUTO_TREES ||
                                  (p.n_trees >= MASKED_AUTO_TREES * 3 / 4 && p.n_tokens >= MASKED_AUTO_TOKENS))
                           : p.depth <= MASKED_AUTO_DEPTH_F32 && p.n_trees >= MASKED_AUTO_TREES_F32) &&
                 int64_t(workspace_bytes) >= masked_ws)
            mode = MODE_MASKED;
        else if (!v) mode = MODE_GENERIC;
        else if (tiled_ws > 0 && int64_t(workspace_bytes) >= tiled_ws && p.depth >= 9 &&
                 (!p.w_bf16 || p.depth >= 10 || elems >= (int64_t(96) << 20)) &&
                 ((big && p.n_tokens >= (int64_t(8) << p.depth)) ||
                  (one && elems >= (int64_t(16) << 20) && p.n_tokens >= (int64_t(16) << p.depth)) ||
                  (one && !p.w_bf16 && p.depth >= 11 &&
                   (p.n_tokens >= (int64_t(8) << p.depth) ||
                    (tile_pairs(p) && p.n_tokens >= (int64_t(2) << p.depth) && elems >= (int64_t(12) << 20)))) ||
                  (one && p.w_bf16 && p.depth >= 11 && p.hidden >= 2048 && p.n_tokens >= (int64_t(4) << p.depth))))
            mode = MODE_TILED;
        else if (one && int64_t(workspace_bytes) >= grouped_ws &&
                 ((p.depth >= 11 && (big || (p.n_tokens >= 16384 && (!p.w_bf16 || elems >= (int64_t(24) << 20))))) ||
                  (!p.w_bf16 && p.depth >= 5 && p.n_tokens >= 65536)))
            mode = MODE_GROUPED;
        else if (affine && !p.w_bf16 && tiled_ws > 0 && int64_t(workspace_bytes) >= tiled_ws &&
                 ((p.depth >= 11 && p.n_tokens >= (int64_t(8) << p.depth)) ||
                  (p.depth >= 10 && p.n_tokens >= (int64_t(16) << p.depth)) ||
                  (p.depth >= 9 && p.n_tokens >= (int64_t(32) << p.depth))))
            mode = MODE_TILED;
        else if (affine && int64_t(workspace_bytes) >= grouped_ws && p.depth >= 7 &&
                 (p.w_bf16 ? p.n_trees == XCDS || (p.n_trees == 4 && p.n_tokens >= (p.depth >= 8 ? 4096 : 65536)) ||
                                 (p.depth >= 8 && p.n_tokens >= 65536)
                           : p.n_tokens >= 65536 || (p.n_trees == XCDS && p.n_tokens >= 16384)))
            mode = MODE_GROUPED;
        else if (p.n_trees == XCDS && int64_t(workspace_bytes) >= grouped_ws &&
                 (p.w_bf16 ? p.n_tokens <= 2048 || (p.depth >= 6 && p.n_tokens <= 4096) : p.n_tokens <= 1024))
            mode = MODE_GROUPED;
        else mode = MODE_DESCENT;
    }
    if (mode == MODE_SUBTREE) {
        if (!subtree_shape(p)) return ST_UNSUPPORTED;
        plan->kind = KIND_SUBTREE;
        plan->name = subtree_name(p);
        plan->lanes = subtree_block(p);  // a workgroup per token
        plan->split_level = subtree_span(p);
        Launch& L = plan->launch[plan->n_launch++];
        L.block = subtree_block(p);
        L.grid = subtree_grid(p, dev.cu_count);
        return ST_OK;
    }
    if (mode == MODE_MASKED) {
        if (!masked_ok || !masked_shape(p)) return ST_UNSUPPORTED;
        plan->kind = KIND_MASKED;
        plan->cu_count = dev.cu_count;
        plan->name = !p.w_bf16 ? "fp32 GEMMs"
                     : p.y_bf16 ? "bf16 GEMMs, activations in 2 parts" : "bf16 GEMMs, activations in 3 parts";
        return ST_OK;
    }
    if ((mode == MODE_DESCENT || mode == MODE_GROUPED || mode == MODE_TILED) && !v) return ST_UNSUPPORTED;
    if (mode == MODE_TILED) {
        if (!tiled_shape(p.depth, p.n_trees, p.hidden)) return ST_UNSUPPORTED;
        plan->kind = KIND_TILED;
        plan->lanes = v->walk_lanes;
        plan->emit_lanes = v->emit_lanes;
        plan->split_level = std::min<int>(p.depth - 2, 5);  // subtrees of at least four leaves
        plan->name = v->name;
        const int64_t leaves = int64_t(1) << p.depth;
        Launch& F = plan->launch[plan->n_launch++];
        F.kernel = reinterpret_cast<const void*>(&fill_i32_kernel);
        F.block = 256;
        F.grid = int(std::min<int64_t>((p.n_trees * (leaves + 1) + 255) / 256, int64_t(dev.cu_count) * 4));
        Launch& W = plan->launch[plan->n_launch++];
        if (!plan_walk(p, *v, lds_levels_req, dev, plan, W)) return ST_UNSUPPORTED;
        Launch& E = plan->launch[plan->n_launch++];
        plan->tile_pair = tile_pairs(p) ? 1 : 0;
        E.kernel = tile_kernel_for(*v, p, 0, plan->tile_pair);  // the first tree's; run_forward picks each tree's form
        E.block = 64 * tile_waves(p.hidden);
        // per tree: one workgroup per leaf or pair of leaves (a multiple of eight: leaves >= 32), then
        // spill workgroups
        E.grid = int(leaves >> plan->tile_pair) + dev.cu_count;
        return ST_OK;
    }

    if (mode == MODE_DESCENT) {
        bool ok;
        const int k = pick_levels(p, lds_levels_req, 2, DESCENT_LDS_BUDGET, dev.lds_per_block, &ok);
        if (!ok) return ST_UNSUPPORTED;
        plan->kind = KIND_DESCENT;
        plan->lanes = v->lanes;
        plan->lds_levels = k;
        plan->name = v->name;
        Launch& L = plan->launch[plan->n_launch++];
        L.kernel = p.norm ? v->descent_norm : v->descent;
        L.block = BLOCK;
        L.lds_bytes = rows_lds_bytes(p, k, 2);
        const int64_t groups = token_groups(p, v->lanes);
        L.grid = resident_grid(dev, L.kernel, L.lds_bytes, (groups + BLOCK / 64 - 1) / (BLOCK / 64));
        return ST_OK;
    }

    if (mode == MODE_GROUPED) {
        int split = split_level_req == 0 ? default_split_level(p.depth, p.n_trees) : split_level_req;
        if (split < 0) split = 0;
        if (split != 0 && (split < 3 || split > p.depth)) return ST_UNSUPPORTED;  // at least one subtree per XCD
        bool ok_e;
        const int ke = pick_levels(p, lds_levels_req, 1, EMIT_LDS_BUDGET, dev.lds_per_block, &ok_e);
        if (!ok_e) return ST_UNSUPPORTED;
        plan->kind = KIND_GROUPED;
        plan->lanes = v->walk_lanes;
        plan->split_level = split;
        plan->name = v->name;
        Launch& W = plan->launch[plan->n_launch++];
        if (!plan_walk(p, *v, lds_levels_req, dev, plan, W)) return ST_UNSUPPORTED;
        Launch& E = plan->launch[plan->n_launch++];
        E.kernel = v->emit;
        E.block = BLOCK;
        E.lds_bytes = rows_lds_bytes(p, ke, 1);
        const int64_t egroups = token_groups(p, v->emit_lanes);
        plan->emit_lanes = v->emit_lanes;
        int eg = resident_grid(dev, E.kernel, E.lds_bytes, (egroups + BLOCK / 64 - 1) / (BLOCK / 64));
        if (split) eg = std::max(XCDS, eg / XCDS * XCDS);  // every XCD gets the same number of workgroups
        E.grid = eg;
        plan->emit_lds_levels = ke;
        return ST_OK;
    }

    const int pairs = p.n_trees * (p.depth + 1);
    if (pairs > GENERIC_MAX_PAIRS) return ST_UNSUPPORTED;
    plan->kind = KIND_GENERIC;
    plan->lanes = 64;
    plan->name = "wave per token";
    Launch& L = plan->launch[plan->n_launch++];
    L.kernel = generic_kernel_for(p.x_bf16, p.w_bf16);
    L.block = GENERIC_BLOCK;
    L.lds_bytes = size_t(GENERIC_BLOCK / 64) * 2 * size_t(pairs) * 4;
    L.grid = resident_grid(dev, L.kernel, L.lds_bytes, (p.n_tokens + GENERIC_BLOCK / 64 - 1) / (GENERIC_BLOCK / 64));
    return ST_OK;
}

int plan_stack(const Params& p, int lds_levels_req, const DeviceInfo& dev, Plan* plan) {
    *plan = Plan{};
    const Variant* v = find_variant(p);
    if (!v) return ST_UNSUPPORTED;
    bool ok;
    const int k = pick_levels(p, lds_levels_req, 2, DESCENT_LDS_BUDGET, dev.lds_per_block, &ok);
    if (!ok) return ST_UNSUPPORTED;
    plan->kind = KIND_STACK;
    plan->lanes = v->lanes;
    plan->lds_levels = k;
    plan->name = v->name;
    Launch& L = plan->launch[plan->n_launch++];
    L.kernel = p.norm ? v->stack_norm : v->stack;
    L.block = BLOCK;
    L.lds_bytes = rows_lds_bytes(p, k, 2);
    L.grid = resident_grid(dev, L.kernel, L.lds_bytes, (token_groups(p, v->lanes) + BLOCK / 64 - 1) / (BLOCK / 64));
    return ST_OK;
}

hipError_t run_stack(const StackParams& sp, const Plan& plan, hipStream_t stream) {
    StackParams q = sp;
    q.p.lds_levels = plan.lds_levels;
    const Launch& L = plan.launch[0];
    void* args[] = {&q};
    return hipLaunchKernel(L.kernel, dim3(L.grid), dim3(L.block), args, L.lds_bytes, stream);
}

// One tiled forward (fill, walk, one tile launch per tree) over the tokens of p.
static hipError_t run_tiled(const Params& p, const Plan& plan, void* workspace, hipStream_t stream) {
    const size_t T = size_t(p.n_trees);
    const size_t recs = size_t(p.n_tokens) * T;
    const int64_t leaves = int64_t(1) << p.depth;
    char* ws = static_cast<char*>(workspace);
    Params q = p;
    q.lds_levels = plan.lds_levels;
    q.walk_affine = plan.walk_affine;
    q.ws_act = reinterpret_cast<float*>(ws);
    ws += align256(recs * size_t(p.depth + 1) * sizeof(float));
    q.ws_leaf = reinterpret_cast<int32_t*>(ws);
    ws += align256(recs * sizeof(int32_t));
    q.bk_count = reinterpret_cast<int32_t*>(ws);
    q.bk_nspill = q.bk_count + T * leaves;
    ws += align256(T * (size_t(leaves) + 1) * sizeof(int32_t));
    q.bk_cap = tile_cap(p.n_tokens, p.depth);
    q.bk_tok = reinterpret_cast<int32_t*>(ws);
    ws += align256(T * size_t(leaves) * size_t(q.bk_cap) * sizeof(int32_t));
    q.bk_spill = reinterpret_cast<int32_t*>(ws);
    ws += align256(T * size_t(p.n_tokens) * sizeof(int32_t));
    q.bk_act = reinterpret_cast<float*>(ws);
    ws += align256(T * size_t(leaves) * size_t(q.bk_cap) * size_t(TILE_REC) * sizeof(float));
    void* sum = p.y_bf16 && T > 1 ? static_cast<void*>(ws) : p.y;  // fp32 running sum over trees
    q.split_level = plan.split_level;
    int32_t* fa = q.bk_count;
    int64_t fn = int64_t(T) * (leaves + 1);
    void* fargs[] = {&fa, &fn};
    const Launch& F = plan.launch[0];
    hipError_t e = hipLaunchKernel(F.kernel, dim3(F.grid), dim3(F.block), fargs, 0, stream);
    if (e != hipSuccess) return e;
    void* wargs[] = {&q};
    const Launch& W = plan.launch[1];
    e = hipLaunchKernel(W.kernel, dim3(W.grid), dim3(W.block), wargs, W.lds_bytes, stream);
    if (e != hipSuccess) return e;
    const Variant* v = find_variant(p);
    const Launch& E = plan.launch[2];
    int leaf_blocks = int(leaves >> plan.tile_pair);
    const void* src0 = out_src_kind(p) == TSRC_NONE ? nullptr : p.out_mode == OUT_RESIDUAL ? p.x : p.y;
    // trees in order: tree t adds its contribution to the running sum of trees 0..t-1 (a fixed
    // order of the sum over trees, so the output bits do not depend on scheduling)
    for (int t = 0; t < int(T); ++t) {
        Params qt = q;
        qt.tile_tree = t;
        qt.tile_src = t > 0 ? sum : src0;
        qt.tile_dst = t == int(T) - 1 ? p.y : sum;
        void* targs[] = {&qt, &leaf_blocks};
        e = hipLaunchKernel(tile_kernel_for(*v, p, t, plan.tile_pair), dim3(E.grid), dim3(E.block), targs, 0, stream);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t run_forward(const Params& p, const Plan& plan, void* workspace, size_t workspace_bytes,
                       hipStream_t stream) {
    if (plan.kind == KIND_MASKED) return run_masked(p, workspace, plan.cu_count, stream);
    if (plan.kind == KIND_SUBTREE) return run_subtree(p, plan.launch[0].grid, stream);
    Params q = p;
    q.lds_levels = plan.lds_levels;
    q.walk_affine = plan.walk_affine;
    if (plan.kind == KIND_GROUPED) {
        const size_t recs = size_t(p.n_tokens) * size_t(p.n_trees);
        char* ws = static_cast<char*>(workspace);
        q.ws_act = reinterpret_cast<float*>(ws);
        q.ws_leaf = reinterpret_cast<int32_t*>(ws + align256(recs * size_t(p.depth + 1) * sizeof(float)));
        q.split_level = plan.split_level;
        (void)workspace_bytes;
    }
    if (plan.kind == KIND_TILED) {
        // The tile kernel addresses [B, H] row blocks with 32-bit offsets, so a call whose fp32
        // rows would not fit them runs as consecutive token chunks, each a complete tiled forward
        // in the same workspace (sized for one chunk).
        const int64_t chunk = tile_chunk_tokens(p.hidden);
        const int64_t H = p.hidden, R = int64_t(p.n_trees) * (p.depth + 1);
        for (int64_t c0 = 0; c0 < p.n_tokens; c0 += chunk) {
            Params c = p;
            c.n_tokens = std::min(chunk, p.n_tokens - c0);
            c.x = static_cast<const char*>(p.x) + c0 * H * (p.x_bf16 ? 2 : 4);
            c.y = static_cast<char*>(p.y) + c0 * H * (p.y_bf16 ? 2 : 4);
            if (p.nodes_out) c.nodes_out = p.nodes_out + c0 * R;
            if (p.logits_out) c.logits_out = p.logits_out + c0 * R;
            const hipError_t e = run_tiled(c, plan, workspace, stream);
            if (e != hipSuccess) return e;
        }
        return hipSuccess;
    }
    for (int i = 0; i < plan.n_launch; ++i) {
        const Launch& L = plan.launch[i];
        if (plan.kind == KIND_GROUPED && i == 1) q.lds_levels = plan.emit_lds_levels;
        void* args[] = {&q};
        const hipError_t e = hipLaunchKernel(L.kernel, dim3(L.grid), dim3(L.block), args, L.lds_bytes, stream);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace fff
