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
// 2. bwd_scan_kernel + bwd_rank/base/place_kernel: stable counting sort of the tokens by
//    leaf.  Sorted by leaf, the tokens through any node form one contiguous
//    run at every level (a node's leaves are a contiguous range).
// 3. bwd_piece_kernel: the sorted order is cut into pieces of P positions;
//    a wave walks one piece for one 256-column slice and sums a*dy and dl*x
//    per level in registers while the node stays the same.  A run that starts
//    and ends inside the piece has no other contributor: its dW row is stored
//    directly.  A run that crosses a piece boundary leaves its piece sum in
//    the workspace (slot 0: the run began before the piece; slot 1: it began
//    in the piece and goes on).
// 4. bwd_fixup_kernel: one task per node adds the piece sums of a crossing
//    run in piece order and stores the row, and stores zero rows for nodes no
//    token visits.  No atomics: every dW element has exactly one writer, and
//    the results do not depend on scheduling.  (Device-scope fp32 atomics
//    were measured at about 26 G/s on MI355X, where the L2 is per XCD; the
//    root rows alone took over a thousand of them per element.)
#include "fff_common.hpp"
#include "fff_device.hpp"
#include "fff_internal.hpp"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

namespace fff {

namespace {

enum { ST_OK_ = 0, ST_UNSUPPORTED_ = -2 };

constexpr int BWD_BLOCK = 256;
constexpr int SCAN_BLOCK = 1024;
constexpr int RANK_BLOCK = 256;   // threads of the rank kernel; a chunk is 1..16 tokens per thread
constexpr int SLICE = 256;       // columns per wave in the weight kernel (64 lanes x 4)
constexpr int LV = 6;            // levels handled per pass of the piece kernel

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

// Stable placement of every valid (token, tree) in leaf order: within a leaf
// the tokens keep their index order, so the sorted order, and every sum taken
// along it, is the same on every run.  Tokens are cut into chunks of
// RANK_BLOCK; a token's position is its leaf's start + the tokens of that leaf
// in earlier chunks + its rank among the leaf's tokens earlier in its chunk.
//
// bwd_rank_kernel (block = one chunk of one tree): each token's rank within its
// chunk and the chunk's count per leaf (hist[t][chunk][leaf], zero for absent
// leaves).  The chunk's leaves sit in LDS; every token compares itself with all
// of them.
__global__ __launch_bounds__(RANK_BLOCK) void bwd_rank_kernel(BwdParams p) {
    extern __shared__ int32_t bins[];  // [p.chunk]
    const int t = blockIdx.y, T = p.n_trees, D = p.depth;
    const int64_t L = int64_t(1) << D;
    const int64_t chunk = blockIdx.x;
    const int C = p.chunk;
    const int tid = threadIdx.x;
    for (int i = tid; i < C; i += RANK_BLOCK) {
        const int64_t b = chunk * C + i;
        int32_t bin = -1;
        if (b < p.n_tokens) {
            const int32_t leaf = p.leaves[b * T + t];
            if (leaf_ok(leaf, D)) bin = int32_t(int64_t(leaf) - (L - 1));
        }
        bins[i] = bin;
    }
    int32_t* h = p.hist + (int64_t(t) * p.chunks + chunk) * L;
    for (int64_t i = tid; i < L; i += RANK_BLOCK) h[i] = 0;
    __syncthreads();
    for (int i = tid; i < C; i += RANK_BLOCK) {
        const int64_t b = chunk * C + i;
        const int32_t bin = bins[i];
        int32_t rank = 0;
        bool last = true;
        for (int j = 0; j < C; ++j) {
            const bool same = bins[j] == bin;
            rank += same && j < i ? 1 : 0;
            last = last && !(same && j > i);
        }
        if (b < p.n_tokens) p.rank[int64_t(t) * p.n_tokens + b] = rank;
        if (bin >= 0 && last) h[bin] = rank + 1;
    }
}

// bwd_rank_wave_kernel: the same outputs for chunks of RANKW_BLOCK tokens, one
// per thread, when the chunk's leaf counters fit in LDS (depth <=
// RANKW_MAX_DEPTH).  A wave finds the lanes holding its leaf with depth + 1
// ballots (one per bit of the leaf, one for validity); a token's rank is the
// count of its leaf in the chunk's earlier waves plus its matching lanes below
// it.  The waves take their turn in order: a wave reads its leaves' counters,
// then the last lane of each leaf group adds the group's size.
constexpr int RANKW_BLOCK = 1024;
constexpr int RANKW_MAX_DEPTH = 14;  // 16384 counters: 64 KB of LDS

__global__ __launch_bounds__(RANKW_BLOCK) void bwd_rank_wave_kernel(BwdParams p) {
    extern __shared__ int32_t cnt_l[];  // [2^depth]
    const int t = blockIdx.y, T = p.n_trees, D = p.depth;
    const int64_t L = int64_t(1) << D;
    const int64_t chunk = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int64_t i = tid; i < L; i += RANKW_BLOCK) cnt_l[i] = 0;
    const int64_t b = chunk * RANKW_BLOCK + tid;
    int32_t bin = -1;
    if (b < p.n_tokens) {
        const int32_t leaf = p.leaves[b * T + t];
        if (leaf_ok(leaf, D)) bin = int32_t(int64_t(leaf) - (L - 1));
    }
    // key: the bin, or L for no bin; lanes with equal keys
    const uint32_t key = bin >= 0 ? uint32_t(bin) : uint32_t(L);
    uint64_t same = ~uint64_t(0);
    for (int i = 0; i <= D; ++i) {
        const bool bit = (key >> i) & 1u;
        const uint64_t m = __ballot(bit);
        same &= bit ? m : ~m;
    }
    const int below = __popcll(same & ((uint64_t(1) << lane) - 1));
    const bool leader = lane == 63 || (same >> (lane + 1)) == 0;  // last lane of its group
    int32_t rank = 0;
    __syncthreads();  // counters zeroed
    for (int w = 0; w < RANKW_BLOCK / 64; ++w) {
        if (wave == w && bin >= 0) {
            const int32_t base = cnt_l[bin];
            rank = base + below;
            if (leader) cnt_l[bin] = base + __popcll(same);
        }
        __syncthreads();
    }
    if (b < p.n_tokens) p.rank[int64_t(t) * p.n_tokens + b] = rank;
    int32_t* h = p.hist + (int64_t(t) * p.chunks + chunk) * L;
    for (int64_t i = tid; i < L; i += RANKW_BLOCK) h[i] = cnt_l[i];
}

// bwd_base_kernel (one wave per (tree, leaf)): turns the chunk counts into the
// first sorted position of the leaf's tokens in each chunk (an exclusive scan
// over the chunks, 64 at a time), and leaves offs at one past the leaf's last
// position.  The leaf's first position comes from offs (bwd_scan_kernel), or
// with self_scan (one tree, at most BASE_SELF_SCAN_LEAVES leaves) from the
// block itself: the sum of the counts of all earlier leaves (integer sums, so
// any order gives the same value), which saves the scan kernel's launch.
constexpr int BASE_SELF_SCAN_LEAVES = 4096;

__global__ __launch_bounds__(BWD_BLOCK) void bwd_base_kernel(BwdParams p, int self_scan) {
    const int64_t L = int64_t(1) << p.depth;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t i0 = int64_t(blockIdx.x) * (BWD_BLOCK / 64);
    const int64_t i = i0 + wave;
    int32_t run = 0;
    if (self_scan) {  // block-uniform
        __shared__ int32_t part[BWD_BLOCK / 64];
        int32_t sum = 0;
        for (int64_t j = threadIdx.x; j < i0 && j < L; j += BWD_BLOCK) sum += p.counts[j];
#pragma unroll
        for (int d = 32; d > 0; d >>= 1) sum += __shfl_xor(sum, d, 64);
        if (lane == 0) part[wave] = sum;
        __syncthreads();
        for (int w = 0; w < BWD_BLOCK / 64; ++w) run += part[w];
        for (int w = 0; w < wave; ++w) run += i0 + w < L ? p.counts[i0 + w] : 0;
    }
    if (i >= L * p.n_trees) return;  // wave-uniform
    const int64_t t = i / L, leaf = i - t * L;
    if (!self_scan) run = p.offs[i];
    int32_t* h = p.hist + t * p.chunks * L + leaf;
    for (int64_t c0 = 0; c0 < p.chunks; c0 += 64) {
        const int64_t c = c0 + lane;
        const int32_t n = c < p.chunks ? h[c * L] : 0;
        int32_t inc = n;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int32_t u = __shfl_up(inc, d, 64);
            if (lane >= d) inc += u;
        }
        if (c < p.chunks) h[c * L] = run + inc - n;
        run += __shfl(inc, 63, 64);
    }
    if (lane == 0) p.offs[i] = run;
}

// bwd_leafsum_kernel (one wave per (tree, leaf)): the leaf's token count, the
// sum of its chunk counts (the fused path counts leaves here, not in a token
// kernel).
__global__ __launch_bounds__(BWD_BLOCK) void bwd_leafsum_kernel(BwdParams p) {
    const int64_t L = int64_t(1) << p.depth;
    const int lane = threadIdx.x & 63;
    const int64_t i = int64_t(blockIdx.x) * (BWD_BLOCK / 64) + (threadIdx.x >> 6);
    if (i >= L * p.n_trees) return;  // wave-uniform
    const int64_t t = i / L, leaf = i - t * L;
    const int32_t* h = p.hist + t * p.chunks * L + leaf;
    int32_t sum = 0;
    for (int64_t c = lane; c < p.chunks; c += 64) sum += h[c * L];
#pragma unroll
    for (int d = 32; d > 0; d >>= 1) sum += __shfl_xor(sum, d, 64);
    if (lane == 0) p.counts[i] = sum;
}

// bwd_place_kernel: perm[t][position] = token.
__global__ __launch_bounds__(BWD_BLOCK) void bwd_place_kernel(BwdParams p) {
    const int T = p.n_trees, D = p.depth;
    const int64_t L = int64_t(1) << D;
    const int64_t n = p.n_tokens * T;
    for (int64_t i = int64_t(blockIdx.x) * BWD_BLOCK + threadIdx.x; i < n; i += int64_t(gridDim.x) * BWD_BLOCK) {
        const int64_t b = i / T;
        const int t = int(i % T);
        const int32_t leaf = p.leaves[i];
        if (!leaf_ok(leaf, D)) {
            if (p.fused) {  // no token kernel ran: count the pair and give the token a zero dx row
                if (p.bad) atomicAdd(p.bad, 1);
                if (p.dx && !p.accumulate) {
                    for (int64_t c = 0; c < p.hidden; ++c) {
                        if (p.dx_bf16) reinterpret_cast<uint16_t*>(p.dx)[b * p.hidden + c] = 0;
                        else reinterpret_cast<float*>(p.dx)[b * p.hidden + c] = 0.0f;
                    }
                }
            }
            continue;
        }
        const int64_t bin = int64_t(leaf) - (L - 1);
        const int64_t pos = p.hist[(int64_t(t) * p.chunks + b / p.chunk) * L + bin] + p.rank[int64_t(t) * p.n_tokens + b];
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

// dW row slice: stored, or added to (accumulate); one writer per element.
__device__ __forceinline__ void put_row(float* dw, int64_t at, bool active, bool accumulate, const float* v) {
    if (!dw || !active) return;
    float4* d = reinterpret_cast<float4*>(dw + at);
    float4 o = make_float4(v[0], v[1], v[2], v[3]);
    if (accumulate) {
        const float4 q = *d;
        o.x += q.x; o.y += q.y; o.z += q.z; o.w += q.w;
    }
    *d = o;
}

// Piece sum slot of (tree t, piece k, level l, slot, matrix m): H floats.
__device__ __forceinline__ int64_t part_at(const BwdParams& p, int t, int64_t k, int l, int slot, int m) {
    return ((((int64_t(t) * p.pieces + k) * (p.depth + 1) + l) * 2 + slot) * 2 + m) * p.hidden;
}

// Piece sums of both matrices into the workspace (a matrix not requested is skipped).
__device__ __forceinline__ void put_part(const BwdParams& p, int t, int64_t k, int l, int slot, int col, bool active,
                                         const float* o, const float* in) {
    if (p.dw_out) put_row(p.part, part_at(p, t, k, l, slot, 0) + col, active, false, o);
    if (p.dw_in) put_row(p.part, part_at(p, t, k, l, slot, 1) + col, active, false, in);
}

// One sorted token's inputs for the piece kernel.
struct WTok {
    uint32_t leaf1;
    float4 gy, xv;
    const float2* cf;
};

__global__ __launch_bounds__(BWD_BLOCK) void bwd_piece_kernel(BwdParams p) {
    const int lane = threadIdx.x & 63;
    const int64_t wid = int64_t(blockIdx.x) * (BWD_BLOCK / 64) + (threadIdx.x >> 6);
    const int T = p.n_trees, D = p.depth, H = p.hidden;
    const int64_t N = p.n_nodes;
    const int slices = (H + SLICE - 1) / SLICE;
    const int64_t per_tree = int64_t(p.pieces) * slices;
    if (wid >= per_tree * T) return;  // whole wave
    const int t = int(wid / per_tree);
    const int64_t r = wid % per_tree;
    const int s = int(r % slices);
    const int64_t k = r / slices;
    const int64_t total = p.total[t];
    const int64_t p0 = k * p.piece;
    const int64_t p1 = std::min<int64_t>(p0 + p.piece, total);
    if (p0 >= p1) return;
    const int col = s * SLICE + lane * 4;
    const bool active = col < H;  // H is a multiple of 4
    const int32_t* perm = p.perm + int64_t(t) * p.n_tokens;
    // the tokens just before and just after the piece decide which runs cross its ends
    const uint32_t prev1 = p0 > 0 ? uint32_t(p.leaves[int64_t(perm[p0 - 1]) * T + t]) + 1 : 0u;
    const uint32_t next1 = p1 < total ? uint32_t(p.leaves[int64_t(perm[p1]) * T + t]) + 1 : 0u;

    auto fetch = [&](int32_t b) {
        WTok w;
        w.leaf1 = uint32_t(p.leaves[int64_t(b) * T + t]) + 1;
        w.gy = make_float4(0.f, 0.f, 0.f, 0.f);
        w.xv = w.gy;
        if (active) {
            w.gy = load4(p.dy, p.dy_bf16, int64_t(b) * H + col);
            w.xv = load4(p.x, p.x_bf16, int64_t(b) * H + col);
        }
        w.cf = p.coef + (int64_t(b) * T + t) * (D + 1);
        return w;
    };

    for (int l0 = 0; l0 <= D; l0 += LV) {
        int32_t cur[LV];    // node of the current run per level (wave-uniform)
        uint32_t head = 0;  // bit j: the current run of level l0+j began before this piece
        float ao[LV][4], ai[LV][4];
#pragma unroll
        for (int j = 0; j < LV; ++j) {
            cur[j] = -1;
#pragma unroll
            for (int q = 0; q < 4; ++q) ao[j][q] = ai[j][q] = 0.0f;
        }
        // a run ends inside the piece: complete (store) or the tail of a crossing run (slot 0)
        auto end_run = [&](int j, int l) {
            if (head & (1u << j)) {
                put_part(p, t, k, l, 0, col, active, ao[j], ai[j]);
            } else {
                const int64_t row = (int64_t(t) * N + cur[j]) * H + col;
                put_row(p.dw_out, row, active, p.accumulate, ao[j]);
                put_row(p.dw_in, row, active, p.accumulate, ai[j]);
            }
        };
        auto consume = [&](const WTok& w) {
#pragma unroll
            for (int j = 0; j < LV; ++j) {
                const int l = l0 + j;
                if (l > D) break;
                const int32_t node = int32_t(w.leaf1 >> (D - l)) - 1;
                if (node != cur[j]) {  // a run starts (wave-uniform)
                    if (cur[j] >= 0) {
                        end_run(j, l);
                        head &= ~(1u << j);
                    } else if (prev1 != 0 && int32_t(prev1 >> (D - l)) - 1 == node) {
                        head |= 1u << j;
                    }
                    cur[j] = node;
#pragma unroll
                    for (int q = 0; q < 4; ++q) ao[j][q] = ai[j][q] = 0.0f;
                }
                const float2 cc = w.cf[l];
                ao[j][0] = __builtin_fmaf(cc.x, w.gy.x, ao[j][0]);
                ao[j][1] = __builtin_fmaf(cc.x, w.gy.y, ao[j][1]);
                ao[j][2] = __builtin_fmaf(cc.x, w.gy.z, ao[j][2]);
                ao[j][3] = __builtin_fmaf(cc.x, w.gy.w, ao[j][3]);
                ai[j][0] = __builtin_fmaf(cc.y, w.xv.x, ai[j][0]);
                ai[j][1] = __builtin_fmaf(cc.y, w.xv.y, ai[j][1]);
                ai[j][2] = __builtin_fmaf(cc.y, w.xv.z, ai[j][2]);
                ai[j][3] = __builtin_fmaf(cc.y, w.xv.w, ai[j][3]);
            }
        };
        // Sorted token indices 64 at a time (one per lane), then one token per step with the
        // next one's loads in flight.
        for (int64_t q0 = p0; q0 < p1; q0 += 64) {
            const int nb = int(std::min<int64_t>(64, p1 - q0));
            const int32_t mine = lane < nb ? perm[q0 + lane] : 0;
            WTok a = fetch(__builtin_amdgcn_readlane(mine, 0));
            int i = 0;
            for (; i + 2 <= nb; i += 2) {
                const WTok b = fetch(__builtin_amdgcn_readlane(mine, i + 1));
                consume(a);
                if (i + 2 < nb) a = fetch(__builtin_amdgcn_readlane(mine, i + 2));
                consume(b);
            }
            if (i < nb) consume(a);
        }
        // the last run of every level: complete, or it goes on into the next piece
#pragma unroll
        for (int j = 0; j < LV; ++j) {
            const int l = l0 + j;
            if (l > D) break;
            const bool goes_on = next1 != 0 && int32_t(next1 >> (D - l)) - 1 == cur[j];
            if (goes_on) {
                put_part(p, t, k, l, (head >> j) & 1u ? 0 : 1, col, active, ao[j], ai[j]);
            } else {
                end_run(j, l);
            }
        }
    }
}

// Run bounds of node n of tree t in the sorted order: [S, E).
__device__ __forceinline__ void node_run(const BwdParams& p, int t, int64_t n, int l, int64_t* S, int64_t* E) {
    const int D = p.depth;
    const int64_t L = int64_t(1) << D;
    const int64_t first = ((n + 1) << (D - l)) - L;  // its leaves, as bins of the level-D order
    const int64_t last = ((n + 2) << (D - l)) - L - 1;
    const int32_t* cnt = p.counts + t * L;
    const int32_t* end = p.offs + t * L;  // after the scatter: one past each leaf's last position
    *S = int64_t(end[first]) - cnt[first];
    *E = end[last];
}

__device__ __forceinline__ int level_of(int64_t n) { return 63 - __builtin_clzll(uint64_t(n + 1)); }

// Levels 0..top_levels-1 of every tree: one 1024-thread block per (tree, node,
// slice); the 16 waves take every 16th piece sum (eight loads in flight) and
// the wave sums are added in wave order through LDS.
constexpr int FIX_BLOCK = 1024;

__global__ __launch_bounds__(FIX_BLOCK) void bwd_fixup_top_kernel(BwdParams p, int top_levels) {
    constexpr int WAVES = FIX_BLOCK / 64;
    __shared__ float4 red[2][WAVES][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int H = p.hidden;
    const int slices = (H + SLICE - 1) / SLICE;
    const int64_t ntop = (int64_t(1) << top_levels) - 1;
    const int64_t task = blockIdx.x;
    const int s = int(task % slices);
    const int64_t n = (task / slices) % ntop;
    const int t = int(task / (slices * ntop));
    const int l = level_of(n);
    int64_t S, E;
    node_run(p, t, n, l, &S, &E);
    const int col = s * SLICE + lane * 4;
    const bool active = col < H;
    const int64_t row = (int64_t(t) * p.n_nodes + n) * H + col;
    const float zero[4] = {0.f, 0.f, 0.f, 0.f};
    if (S == E) {  // block-uniform
        if (!p.accumulate && wave == 0) {
            put_row(p.dw_out, row, active, false, zero);
            put_row(p.dw_in, row, active, false, zero);
        }
        return;
    }
    const int64_t kS = S / p.piece, kE = (E - 1) / p.piece;
    if (kS == kE) return;  // inside one piece: stored by the piece kernel
    float4 so = make_float4(0.f, 0.f, 0.f, 0.f), si = so;
    if (active) {
        constexpr int U = 8;
        for (int64_t k0 = kS + wave; k0 <= kE; k0 += int64_t(WAVES) * U) {
            float4 vo[U], vi[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t k = k0 + int64_t(u) * WAVES;
                vo[u] = vi[u] = make_float4(0.f, 0.f, 0.f, 0.f);
                if (k <= kE) {
                    const int slot = k == kS ? 1 : 0;
                    if (p.dw_out) vo[u] = *reinterpret_cast<const float4*>(p.part + part_at(p, t, k, l, slot, 0) + col);
                    if (p.dw_in) vi[u] = *reinterpret_cast<const float4*>(p.part + part_at(p, t, k, l, slot, 1) + col);
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                so.x += vo[u].x; so.y += vo[u].y; so.z += vo[u].z; so.w += vo[u].w;
                si.x += vi[u].x; si.y += vi[u].y; si.z += vi[u].z; si.w += vi[u].w;
            }
        }
    }
    red[0][wave][lane] = so;
    red[1][wave][lane] = si;
    __syncthreads();
    if (wave == 0) {
        float o[4] = {0.f, 0.f, 0.f, 0.f}, in[4] = {0.f, 0.f, 0.f, 0.f};
        for (int w = 0; w < WAVES; ++w) {
            const float4 a = red[0][w][lane], b = red[1][w][lane];
            o[0] += a.x; o[1] += a.y; o[2] += a.z; o[3] += a.w;
            in[0] += b.x; in[1] += b.y; in[2] += b.z; in[3] += b.w;
        }
        put_row(p.dw_out, row, active, p.accumulate, o);
        put_row(p.dw_in, row, active, p.accumulate, in);
    }
}

// Levels top_levels..D: one wave per (tree, node, slice), grid-stride; these
// runs usually span one or two pieces.
__global__ __launch_bounds__(BWD_BLOCK) void bwd_fixup_kernel(BwdParams p, int top_levels) {
    const int lane = threadIdx.x & 63;
    const int T = p.n_trees, H = p.hidden;
    const int64_t N = p.n_nodes;
    const int64_t n0 = (int64_t(1) << top_levels) - 1;  // first node handled here
    const int64_t nn = N - n0;
    const int slices = (H + SLICE - 1) / SLICE;
    const int64_t tasks = int64_t(T) * nn * slices;
    const int64_t waves = int64_t(gridDim.x) * (BWD_BLOCK / 64);
    for (int64_t w = int64_t(blockIdx.x) * (BWD_BLOCK / 64) + (threadIdx.x >> 6); w < tasks; w += waves) {
        const int s = int(w % slices);
        const int64_t n = n0 + (w / slices) % nn;
        const int t = int(w / (slices * nn));
        const int l = level_of(n);
        int64_t S, E;
        node_run(p, t, n, l, &S, &E);
        const int col = s * SLICE + lane * 4;
        const bool active = col < H;
        const int64_t row = (int64_t(t) * N + n) * H + col;
        float o[4] = {0.f, 0.f, 0.f, 0.f}, in[4] = {0.f, 0.f, 0.f, 0.f};
        if (S == E) {  // no token visits this node
            if (!p.accumulate) {
                put_row(p.dw_out, row, active, false, o);
                put_row(p.dw_in, row, active, false, in);
            }
            continue;
        }
        const int64_t kS = S / p.piece, kE = (E - 1) / p.piece;
        if (kS == kE) continue;  // inside one piece: stored by the piece kernel
        for (int64_t k = kS; k <= kE && active; ++k) {
            const int slot = k == kS ? 1 : 0;
            if (p.dw_out) {
                const float4 v = *reinterpret_cast<const float4*>(p.part + part_at(p, t, k, l, slot, 0) + col);
                o[0] += v.x; o[1] += v.y; o[2] += v.z; o[3] += v.w;
            }
            if (p.dw_in) {
                const float4 v = *reinterpret_cast<const float4*>(p.part + part_at(p, t, k, l, slot, 1) + col);
                in[0] += v.x; in[1] += v.y; in[2] += v.z; in[3] += v.w;
            }
        }
        put_row(p.dw_out, row, active, p.accumulate, o);
        put_row(p.dw_in, row, active, p.accumulate, in);
    }
}

// ---------------------------------------------------------------------------
// planning
// ---------------------------------------------------------------------------

// ---------------------------------------------------------------------------
// 3'. leaf-tiled weight kernel on MFMA (depth <= 15, hidden a multiple of 128)
// ---------------------------------------------------------------------------
//
// One workgroup per subtree of 2^sub leaves (the subtree's root at level
// k = D - sub), one wave per 128-column group g.  The subtree's tokens are taken
// in sorted order, leaf by leaf, four per step of v_mfma_f32_16x16x4_f32: rows
// are levels, the K dimension is the four tokens, and lane l supplies the pair
// (a, dl) of token 4s + l/16 at level l%16 and that token's eight dy (x) values
// at columns 128g + 8(l%16) .. +7 for the eight column blocks.  The
// accumulators hold the sums for all D+1 nodes of the current path, lane l
// receiving levels 4(l/16) .. +3 of its eight columns.  When a leaf is done the
// rows of the nodes it completes (levels from the leaf up to the subtree root
// whose last leaf it is) are stored and cleared; a node no token reached gets
// a zero row.  The levels above the subtree root leave this subtree's sums in
// part[] and are added in a fixed order by bwd_wsum_kernel.  Every dW element
// has one writer and the order of every sum is fixed.
constexpr int WT_WAVES_MAX = 8;
constexpr int WT_TOP_LEVELS = 9;   // subtrees hang at level min(D, 9)
constexpr int WT_MAX_SUB = 6;      // depth <= 15: at most 2^6 leaves per subtree
constexpr int WT_LDS_TOK = 4096;   // token ids of a subtree staged in LDS when they fit

__device__ __forceinline__ void load8f(const void* base, bool bf, int64_t at, float* v) {
    if (bf) {
        const uint4 u = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(base) + at);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[2 * j] = bf16_lo(word(u, j));
            v[2 * j + 1] = bf16_hi(word(u, j));
        }
    } else {
        const float4 a = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(base) + at);
        const float4 b = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(base) + at + 4);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
}

// Eight consecutive elements of a bf16 (one 16-byte word) or fp32 (two words)
// row, loaded raw so that a caller can issue every load of a tile at once and
// convert at the point of use; to8f gives the same floats as load8f.
template <bool BF>
struct Raw8 {
    uint4 w[BF ? 1 : 2];
};
template <bool BF>
__device__ __forceinline__ Raw8<BF> raw8(const void* base, int64_t at) {
    Raw8<BF> r;
    if constexpr (BF) {
        r.w[0] = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(base) + at);
    } else {
        r.w[0] = *reinterpret_cast<const uint4*>(reinterpret_cast<const float*>(base) + at);
        r.w[1] = *reinterpret_cast<const uint4*>(reinterpret_cast<const float*>(base) + at + 4);
    }
    return r;
}
template <bool BF>
__device__ __forceinline__ void to8f(const Raw8<BF>& r, float* v) {
    if constexpr (BF) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[2 * j] = bf16_lo(word(r.w[0], j));
            v[2 * j + 1] = bf16_hi(word(r.w[0], j));
        }
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[j] = __uint_as_float(word(r.w[0], j));
            v[4 + j] = __uint_as_float(word(r.w[1], j));
        }
    }
}

// Eight fp32 values of a dW row: stored, or added to what is there.
__device__ __forceinline__ void put8(float* dst, bool add, const float* v) {
    float4* d = reinterpret_cast<float4*>(dst);
    float4 a = make_float4(v[0], v[1], v[2], v[3]), b = make_float4(v[4], v[5], v[6], v[7]);
    if (add) {
        const float4 o0 = d[0], o1 = d[1];
        a.x += o0.x; a.y += o0.y; a.z += o0.z; a.w += o0.w;
        b.x += o1.x; b.y += o1.y; b.z += o1.z; b.w += o1.w;
    }
    d[0] = a;
    d[1] = b;
}

template <bool XBF, bool DYBF>
__global__ __launch_bounds__(64 * WT_WAVES_MAX) void bwd_wtile_kernel(BwdParams p, int sub) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, waves = blockDim.x >> 6;
    const int n = lane & 15, q = lane >> 4;
    const int t = blockIdx.y, T = p.n_trees, D = p.depth;
    const int64_t L = int64_t(1) << D, H = p.hidden, N = p.n_nodes;
    const int k = D - sub;
    const int64_t st = blockIdx.x;
    const int64_t leaf0 = st << sub;
    const int32_t* cnt = p.counts + t * L;
    const int32_t* end = p.offs + t * L;  // after the placement: one past each leaf's last position
    const int32_t* perm = p.perm + int64_t(t) * p.n_tokens;
    float* dwo = p.dw_out ? p.dw_out + int64_t(t) * N * H : nullptr;
    float* dwi = p.dw_in ? p.dw_in + int64_t(t) * N * H : nullptr;
    const bool add = p.accumulate != 0;
    const int lvl_a = n <= D ? n : D;  // this lane's level as A supplier (clamped; A is 0 past D)
    // The subtree's tokens are one contiguous range of the sorted order: its
    // leaves' counts and, when the range fits, its token ids are staged in LDS
    // once for all waves.
    __shared__ int32_t s_cnt[1 << WT_MAX_SUB];
    __shared__ int32_t s_tok[WT_LDS_TOK];
    const int nleaf = 1 << sub;
    for (int i = threadIdx.x; i < nleaf; i += blockDim.x) s_cnt[i] = cnt[leaf0 + i];
    const int64_t first = int64_t(end[leaf0]) - cnt[leaf0];
    const int64_t range = int64_t(end[leaf0 + nleaf - 1]) - first;
    const bool staged = range <= WT_LDS_TOK;  // workgroup-uniform
    if (staged)
        for (int64_t i = threadIdx.x; i < range; i += blockDim.x) s_tok[i] = perm[first + i];
    __syncthreads();
    for (int64_t g = wave; g < H / 128; g += waves) {
        const int64_t col = g * 128 + 8 * n;
        tile_v4f ao[8], ai[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) ao[j] = ai[j] = tile_v4f{0.f, 0.f, 0.f, 0.f};
        int64_t pos0 = first;  // sorted position of the current leaf's first token
        for (int jl = 0; jl < nleaf; ++jl) {
            const int64_t leaf = leaf0 + jl;
            const int32_t c = s_cnt[jl];
            {
                const int32_t m = c;
                // operands of step s0 for this lane: (a, dl) of token s0 + q at its level,
                // and that token's eight dy and x values as stored (token clamped into the leaf)
                struct Ops {
                    float2 cf;
                    typename std::conditional<DYBF, uint4, float4[2]>::type dy;
                    typename std::conditional<XBF, uint4, float4[2]>::type x;
                };
                auto load_ops = [&](int32_t s0, Ops& o) {
                    const int64_t pos = pos0 + (s0 + q < m ? s0 + q : 0);
                    const int32_t tok = staged ? s_tok[pos - first] : perm[pos];
                    o.cf = p.coef[(int64_t(tok) * T + t) * (D + 1) + lvl_a];
                    const int64_t at = int64_t(tok) * H + col;
                    if constexpr (DYBF) {
                        o.dy = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(p.dy) + at);
                    } else {
                        o.dy[0] = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(p.dy) + at);
                        o.dy[1] = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(p.dy) + at + 4);
                    }
                    if constexpr (XBF) {
                        o.x = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(p.x) + at);
                    } else {
                        o.x[0] = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(p.x) + at);
                        o.x[1] = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(p.x) + at + 4);
                    }
                };
                auto val = [](const auto& v, int j) -> float {
                    if constexpr (std::is_same<typename std::decay<decltype(v)>::type, uint4>::value)
                        return (j & 1) ? bf16_hi(word(v, j >> 1)) : bf16_lo(word(v, j >> 1));
                    else
                        return fword(v[j >> 2], j & 3);
                };
                auto step = [&](int32_t s0, const Ops& o) {
                    const bool in = s0 + q < m && n <= D;
                    const float a = in ? o.cf.x : 0.0f, dl = in ? o.cf.y : 0.0f;
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        ao[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, val(o.dy, j), ao[j], 0, 0, 0);
                        ai[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(dl, val(o.x, j), ai[j], 0, 0, 0);
                    }
                };
                if (m > 0) {
                    // three operand sets in turn: two steps are in flight while one runs;
                    // sched_barrier keeps each prefetch above the MFMAs it overlaps (the
                    // scheduler would otherwise sink the loads to their use)
                    Ops o0, o1, o2;
                    load_ops(0, o0);
                    load_ops(4, o1);
                    for (int32_t s0 = 0;;) {
                        load_ops(s0 + 8, o2);
                        __builtin_amdgcn_sched_barrier(0);
                        step(s0, o0);
                        if ((s0 += 4) >= m) break;
                        load_ops(s0 + 8, o0);
                        __builtin_amdgcn_sched_barrier(0);
                        step(s0, o1);
                        if ((s0 += 4) >= m) break;
                        load_ops(s0 + 8, o1);
                        __builtin_amdgcn_sched_barrier(0);
                        step(s0, o2);
                        if ((s0 += 4) >= m) break;
                    }
                }
            }
            pos0 += c;
            // rows this leaf completes: levels lv >= k whose node's last leaf this is
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int lv = 4 * q + r;
                if (lv <= D && lv >= k && ((leaf + 1) & ((int64_t(1) << (D - lv)) - 1)) == 0) {
                    const int64_t node = ((leaf + L) >> (D - lv)) - 1;
                    float v[8];
                    if (dwo) {
#pragma unroll
                        for (int j = 0; j < 8; ++j) v[j] = ao[j][r];
                        put8(dwo + node * H + col, add, v);
                    }
                    if (dwi) {
#pragma unroll
                        for (int j = 0; j < 8; ++j) v[j] = ai[j][r];
                        put8(dwi + node * H + col, add, v);
                    }
#pragma unroll
                    for (int j = 0; j < 8; ++j) ao[j][r] = ai[j][r] = 0.0f;
                }
            }
        }
        // levels above the subtree root: this subtree's sums for the fix-up
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int lv = 4 * q + r;
            if (lv < k) {
                float* dst = p.part + (((int64_t(t) << k) + st) * k + lv) * 2 * H + col;
                float v[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) v[j] = ao[j][r];
                put8(dst, false, v);
#pragma unroll
                for (int j = 0; j < 8; ++j) v[j] = ai[j][r];
                put8(dst + H, false, v);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// 1'. fused leaf-tiled backward (bf16 W, one tree, depth <= 15, hidden 128..1024)
// ---------------------------------------------------------------------------
//
// The tokens of a leaf share all D+1 rows, so after the stable sort the whole
// backward of a tile of sixteen tokens is dense algebra over one path:
//     da[16, D+1]  = dY[16, H] W_out[path]^T   (bf16 MFMA 16x16x32, K = columns)
//     a, dl        = act(l), da act'(l)         (the forward's logits)
//     dx[16, H]    = dL[16, D+1] W_in[path]     (bf16 MFMA on dl split into bf16 parts)
//     dW_out[path] += a^T dY,  dW_in[path] += dL^T X   (fp32 MFMA 16x16x4, K = four tokens)
// One workgroup per subtree as in bwd_wtile_kernel, one wave per 128-column
// group.  Each wave's da is a partial sum over its columns; the partials are
// added in wave order through LDS.  dy (as two operand layouts) and x are read
// in leaf order, once per token; dx is written once.  The dW rows are stored
// and the fix-up run exactly as in bwd_wtile_kernel.
constexpr int FUSED_WAVES_MAX = 8;
// Stores of dx rows past a tile's count (or with no dx requested) go to a junk area, 32 bytes per
// lane, so that every path through a tile issues the same vector memory operations and the
// compiler's waits for earlier loads count exactly the operations after them.
constexpr size_t BWD_JUNK_BYTES = 64 * 32;
// 16 bytes of an LDS table written as uint16_t, read through a may_alias type
typedef uint32_t lds_u32x4_base __attribute__((ext_vector_type(4)));
typedef lds_u32x4_base __attribute__((may_alias)) lds_u32x4;
__device__ __forceinline__ uint4 lds_u4(const uint16_t* p) {
    const lds_u32x4 v = *reinterpret_cast<const lds_u32x4*>(p);
    return make_uint4(v.x, v.y, v.z, v.w);
}
// v = hi + mid + lo with bf16 parts, each the round-to-nearest of what the parts before leave
__device__ __forceinline__ void split3(float v, uint16_t* out) {
    const uint16_t hi = f32_to_bf16(v);
    const float r = v - bf16_to_f32(hi);
    const uint16_t mid = f32_to_bf16(r);
    out[0] = hi;
    out[1] = mid;
    out[2] = f32_to_bf16(r - bf16_to_f32(mid));
}

template <bool XBF, bool DYBF>
__global__ __launch_bounds__(64 * FUSED_WAVES_MAX) void bwd_fused_kernel(BwdParams p, int sub) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, waves = blockDim.x >> 6;
    const int n = lane & 15, q = lane >> 4, h = q & 1, part = q >> 1;
    const int D = p.depth;
    const int64_t L = int64_t(1) << D, H = p.hidden;
    const int k = D - sub;
    const int64_t st = blockIdx.x;
    const int64_t leaf0 = st << sub;
    const int nleaf = 1 << sub;
    const int32_t* cnt = p.counts;
    const int32_t* end = p.offs;  // after the placement: one past each leaf's last position
    const int32_t* perm = p.perm;
    const bool add = p.accumulate != 0;
    const int64_t col = int64_t(wave) * 128;  // this wave's column group (hidden / 128 == waves)
    __shared__ int32_t s_cnt[1 << WT_MAX_SUB];
    __shared__ int32_t s_tok[WT_LDS_TOK];
    // Tables of one tile, in two buffers by tile parity: a wave may enter the next tile while others
    // finish this one (it cannot get two tiles ahead: the next tile's first barrier needs everyone).
    __shared__ float red[2][FUSED_WAVES_MAX][16][17];  // per-wave partial da [token][level]
    // bf16 x and dy: the dW sums on bf16 MFMA (K = tokens), with a and dl level-major; otherwise
    // on fp32 MFMA, with a token-major.  dl token-major for dx in both.
    constexpr bool BF4 = XBF && DYBF;
    __shared__ float s_a[2][BF4 ? 1 : 16][17], s_dl[2][BF4 ? 1 : 16][17];
    // a and dl as three bf16 parts (hi, mid, lo; hi + mid + lo = the fp32 value to fp32 precision):
    // dl token-major for dx ([part][token][level]); BF4: a and dl level-major for the dW sums
    __shared__ __align__(16) uint16_t s_dlQ[2][3][16][16];
    __shared__ __align__(16) uint16_t s_aP[2][BF4 ? 3 : 1][16][16], s_dlP[2][BF4 ? 3 : 1][16][16];
    // the tile's (token, level) entries go to the waves that have a SIMD to themselves when the
    // workgroup has 5..7 waves (waves w and w + 4 share one), else to all waves
    const bool shared_simd = waves > 4 && waves < 8;
    const int aw0 = shared_simd ? waves - 4 : 0;
    const int a_threads = ((shared_simd ? 4 : waves) - aw0) * 64;
    const int a_tid = int(threadIdx.x) - aw0 * 64;  // takes entries a_tid + e a_threads if in [0, a_threads)
    const bool a_live = a_tid >= 0 && a_tid < a_threads;
    // Each wave's dy tile (and, with BF4, x tile) read back in another layout: a transpose without
    // a second read.  BF4: dy then x, each [column slot][16 tokens] bf16, column c of the wave at
    // slot (c % 8) * 16 + c / 8, so that a 16-column MFMA tile is 16 consecutive slots.
    // Otherwise dy [token][column] with one padding word per row.
    constexpr int DW = DYBF ? 1 : 2;  // 16-byte words per 8 columns of dy
    constexpr int DY_WORDS = BF4 ? 2 * 128 * 16 * 2 / 16 : 16 * (16 * DW + 1);
    __shared__ uint4 s_dy[FUSED_WAVES_MAX][DY_WORDS];
    uint16_t* const t16 = reinterpret_cast<uint16_t*>(&s_dy[wave][0]);  // BF4: dy^T, then x^T at 2048
    // BF4: a row tile (token n of the tile, columns col + 32s + 8q .. +7) into a transposed table
    auto put_t = [&](int base, const uint4& v, int s, bool keep) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const uint32_t u = keep ? word(v, w) : 0u;
            t16[base + ((2 * w) * 16 + 4 * s + q) * 16 + n] = uint16_t(u & 0xffffu);
            t16[base + ((2 * w + 1) * 16 + 4 * s + q) * 16 + n] = uint16_t(u >> 16);
        }
    };
    for (int i = threadIdx.x; i < nleaf; i += blockDim.x) s_cnt[i] = cnt[leaf0 + i];
    const int64_t first = int64_t(end[leaf0]) - cnt[leaf0];
    const int64_t last = end[leaf0 + nleaf - 1];
    // s_tok holds the sorted token ids of positions win0 .. win0 + WT_LDS_TOK - 1 (clipped to the
    // subtree); a tile past the window moves it (rare: a subtree with that many tokens)
    int64_t win0 = first;
    auto stage = [&]() {
        for (int64_t i = threadIdx.x; i < WT_LDS_TOK && win0 + i < last; i += blockDim.x) s_tok[i] = perm[win0 + i];
    };
    stage();
    __syncthreads();

    const uint16_t* wout16 = reinterpret_cast<const uint16_t*>(p.w_out);
    const uint16_t* win16 = reinterpret_cast<const uint16_t*>(p.w_in);
    tile_v4f ao[8], ai[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) ao[j] = ai[j] = tile_v4f{0.f, 0.f, 0.f, 0.f};
    int par = 0;  // buffer of the current tile's tables
    // Software pipeline over the subtree's tiles (16 sorted positions of one leaf each): during a
    // tile, the token ids, dy rows (da operand layout) and logits of the positions that follow it
    // are fetched.  The next tile's positions are contiguous with this one (empty leaves have
    // none); rows past its count belong to a later leaf, are fetched all the same and are masked
    // where used.  Every load is unconditional (clamped ids and levels) and every dx store has a
    // target (junk for absent rows), so the waits for these loads do not wait for later stores.
    constexpr int LG = 256 / 64;  // (token, level) entries per thread at one wave
    int32_t tvN = -1;
    Raw8<DYBF> dyN[4];
    float lgN[LG];
    auto prefetch = [&](int64_t P) {  // P < last, workgroup-uniform; s_tok covers P .. min(P + 15, last - 1)
        tvN = P + n < last ? s_tok[P + n - win0] : -1;
        const int32_t t0n = __shfl(tvN, 0, 64);
        const int64_t ra = int64_t(tvN >= 0 ? tvN : t0n) * H + col + 8 * q;
#pragma unroll
        for (int s = 0; s < 4; ++s) dyN[s] = raw8<DYBF>(p.dy, ra + 32 * s);
#pragma unroll
        for (int e = 0; e < LG; ++e) {
            const int i = a_tid + e * a_threads;
            const int32_t tok = __shfl(tvN, (i >> 4) & 15, 64);
            const int lv = (i & 15) <= D ? (i & 15) : D;
            lgN[e] = p.logits[int64_t(tok >= 0 ? tok : t0n) * (D + 1) + lv];
        }
    };
    // bf16 x and dy: fetched one tile ahead; otherwise (more registers per row) at the tile's start
    constexpr bool PIPE = BF4;
    if (PIPE && first < last) prefetch(first);
    int64_t pos0 = first;
    for (int jl = 0; jl < nleaf; ++jl) {
        const int64_t leaf = leaf0 + jl;
        const uint32_t leaf1 = uint32_t(leaf + L);
        const int32_t c = s_cnt[jl];
        if (c > 0) {  // workgroup-uniform
            // da B operand: lane (level n, q) holds W_out[node(n)][col + 32 s + 8 q .. +7]
            uint4 wo[4];
            {
                const int lv = n <= D ? n : D;  // levels past D: any row (their da is not used)
                const int64_t node = int64_t(leaf1 >> (D - lv)) - 1;
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    wo[s] = *reinterpret_cast<const uint4*>(wout16 + node * H + col + 32 * s + 8 * q);
            }
            // dx B operand: bj[j] = column col + 8n + j of the W_in rows of levels 8h .. 8h+7
            uint4 bj[8];
            {
                uint4 row[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int lvl = 8 * h + i <= D ? 8 * h + i : D;
                    row[i] = *reinterpret_cast<const uint4*>(win16 + (int64_t(leaf1 >> (D - lvl)) - 1) * H + col + 8 * n);
                }
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    uint32_t w4[4];
#pragma unroll
                    for (int qq = 0; qq < 4; ++qq) {
                        const uint32_t lo = word(row[2 * qq], j / 2), hi = word(row[2 * qq + 1], j / 2);
                        w4[qq] = (j & 1) ? (lo >> 16) | (hi & 0xffff0000u) : (lo & 0xffffu) | (hi << 16);
                    }
                    bj[j] = make_uint4(w4[0], w4[1], w4[2], w4[3]);
                }
            }
            for (int32_t t0 = 0; t0 < c; t0 += 16, par ^= 1) {
                const int32_t m_cnt = c - t0 < 16 ? c - t0 : 16;
                // the window of staged ids covers this tile and the next one
                if (pos0 + t0 + 32 > win0 + WT_LDS_TOK) {  // workgroup-uniform
                    // every wave has read the ids of the tiles before: it passed their barriers
                    win0 = pos0 + t0;
                    stage();
                    __syncthreads();
                }
                // token of tile row r (r < 16), -1 past the leaf's count: row n in lane (n, q), the
                // others by cross-lane reads; row 0 stands in for absent rows where a load needs an address
                if constexpr (!PIPE) prefetch(pos0 + t0);
                const int32_t tv = n < m_cnt ? tvN : -1;
                Raw8<DYBF> dyA[4];
#pragma unroll
                for (int s = 0; s < 4; ++s) dyA[s] = dyN[s];
                float lg[LG];
#pragma unroll
                for (int e = 0; e < LG; ++e) lg[e] = lgN[e];
                auto row_tok = [&](int r) -> int32_t { return __shfl(tv, r, 64); };
                const int32_t tk0 = row_tok(0);
                auto valid = [&](int32_t t) -> int32_t { return t >= 0 ? t : tk0; };
                int32_t t4[4];
#pragma unroll
                for (int s = 0; s < 4; ++s) t4[s] = row_tok(4 * s + q);  // dW rows: token 4s + q
                Raw8<XBF> xB[4];  // BF4: the da operand layout; otherwise the dW one
                constexpr bool EARLY_X = XBF && DYBF;
                auto load_x = [&]() {
#pragma unroll
                    for (int s = 0; s < 4; ++s)
                        xB[s] = BF4 ? raw8<XBF>(p.x, int64_t(valid(tv)) * H + col + 8 * q + 32 * s)
                                    : raw8<XBF>(p.x, int64_t(valid(t4[s])) * H + col + 8 * n);
                };
                // 1. partial da over this wave's columns: A = dy of token n (lane (n, q))
                {
                    tile_v4f da = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int s = 0; s < 4; ++s) {
                        const bf16x8_t b = __builtin_bit_cast(bf16x8_t, wo[s]);
                        if constexpr (DYBF) {
                            da = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, dyA[s].w[0]), b, da,
                                                                         0, 0, 0);
                        } else {
                            // fp32 dy: three bf16 parts (hi, mid, lo), each product exact
                            float v[8];
                            to8f<DYBF>(dyA[s], v);
                            uint32_t ph[4], pm[4], pl[4];
#pragma unroll
                            for (int qq = 0; qq < 4; ++qq) {
                                const float x0 = v[2 * qq], x1 = v[2 * qq + 1];
                                ph[qq] = pack_bf16x2(x0, x1);
                                const float r0 = x0 - bf16_lo(ph[qq]), r1 = x1 - bf16_hi(ph[qq]);
                                pm[qq] = pack_bf16x2(r0, r1);
                                pl[qq] = pack_bf16x2(r0 - bf16_lo(pm[qq]), r1 - bf16_hi(pm[qq]));
                            }
                            da = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                __builtin_bit_cast(bf16x8_t, make_uint4(ph[0], ph[1], ph[2], ph[3])), b, da, 0, 0, 0);
                            da = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                __builtin_bit_cast(bf16x8_t, make_uint4(pm[0], pm[1], pm[2], pm[3])), b, da, 0, 0, 0);
                            da = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                __builtin_bit_cast(bf16x8_t, make_uint4(pl[0], pl[1], pl[2], pl[3])), b, da, 0, 0, 0);
                        }
                    }
                    // x rows of the dW sums (bf16 x and dy: in flight during the reduction and dx; otherwise
                    // after dx, for registers); dy to the transpose
                    if constexpr (EARLY_X) load_x();
                    if constexpr (PIPE) {
                        // after the subtree's last tile: the last position again (unused), so that the
                        // number of loads issued here does not depend on the path
                        const int64_t nxt = pos0 + (t0 + 16 < c ? t0 + 16 : c);
                        prefetch(nxt < last ? nxt : last - 1);
                    }
                    if constexpr (BF4) {
#pragma unroll
                        for (int s = 0; s < 4; ++s) put_t(0, dyA[s].w[0], s, n < m_cnt);
                    } else {
#pragma unroll
                        for (int s = 0; s < 4; ++s)
#pragma unroll
                            for (int w = 0; w < DW; ++w)
                                s_dy[wave][n * (16 * DW + 1) + (4 * s + q) * DW + w] =
                                    n < m_cnt ? dyA[s].w[w] : make_uint4(0u, 0u, 0u, 0u);
                    }
                    // lane (level n, q) holds tokens 4q + r
#pragma unroll
                    for (int r = 0; r < 4; ++r) red[par][wave][4 * q + r][n] = da[r];
                }
                __syncthreads();
                // 2. a and dl of the tile's (token, level) pairs, the partials added in wave order
#pragma unroll
                for (int e = 0; e < LG; ++e) {
                    const int i = a_tid + e * a_threads;
                    if (a_live && i < 256) {
                        const int tt = i >> 4, lv = i & 15;
                        float da = 0.0f;
                        for (int w = 0; w < waves; ++w) da += red[par][w][tt][lv];
                        float a = 0.0f, dl = 0.0f;
                        if (tt < m_cnt && lv <= D) {
                            a = activation(lg[e], p.act);
                            dl = da * activation_grad(lg[e], p.act);
                        }
                        uint16_t dp[3];
                        split3(dl, dp);
#pragma unroll
                        for (int r = 0; r < 3; ++r) s_dlQ[par][r][tt][lv] = dp[r];
                        if constexpr (BF4) {
                            uint16_t ap[3];
                            split3(a, ap);
#pragma unroll
                            for (int r = 0; r < 3; ++r) {
                                s_aP[par][r][lv][tt] = ap[r];
                                s_dlP[par][r][lv][tt] = dp[r];
                            }
                        } else {
                            s_a[par][tt][lv] = a;
                            s_dl[par][tt][lv] = dl;
                        }
                    }
                }
                __syncthreads();
                // BF4: x of the tile to its transposed table now, before the dx stores: a wait for the x
                // loads after the stores would wait for the stores too (the vector memory counter
                // retires in order)
                if constexpr (BF4) {
#pragma unroll
                    for (int s = 0; s < 4; ++s) put_t(2048, xB[s].w[0], s, n < m_cnt);
                }
                // 3. dx rows of the tile: A = parts of dl (token n, levels 8h .. 8h+7), B = bj
                {
                    // lane (token n, q): part (q / 2 ? mid : hi) of dl at levels 8h .. 8h+7, then lo or zero
                    const bf16x8_t a0 = __builtin_bit_cast(bf16x8_t, lds_u4(&s_dlQ[par][part][n][8 * h]));
                    const bf16x8_t a1 = __builtin_bit_cast(
                        bf16x8_t, part == 0 ? lds_u4(&s_dlQ[par][2][n][8 * h]) : make_uint4(0u, 0u, 0u, 0u));
                    tile_v4f acc[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, __builtin_bit_cast(bf16x8_t, bj[j]),
                                                                         tile_v4f{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, __builtin_bit_cast(bf16x8_t, bj[j]), acc[j],
                                                                         0, 0, 0);
                    }
                    // lane (n, q) holds tokens 4q + r, columns col + 8n + j
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int32_t tok = row_tok(4 * q + r);  // dx rows: token 4q + r
                        const bool real = tok >= 0 && p.dx != nullptr;
                        float v[8];
#pragma unroll
                        for (int j = 0; j < 8; ++j) v[j] = acc[j][r];
                        const int64_t at = int64_t(real ? tok : 0) * H + col + 8 * n;
                        char* const jk = p.junk + lane * 32;
                        if (p.dx_bf16) {
                            uint4* d = real ? reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(p.dx) + at)
                                            : reinterpret_cast<uint4*>(jk);
                            if (add) {
                                const uint4 o = *d;
#pragma unroll
                                for (int jj = 0; jj < 4; ++jj) {
                                    v[2 * jj] += bf16_lo(word(o, jj));
                                    v[2 * jj + 1] += bf16_hi(word(o, jj));
                                }
                            }
                            *d = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                                            pack_bf16x2(v[6], v[7]));
                        } else {
                            put8(real ? reinterpret_cast<float*>(p.dx) + at : reinterpret_cast<float*>(jk), add, v);
                        }
                    }
                }
                if constexpr (BF4) {
                    // 4. dW sums on bf16 MFMA: K-slots 2i, 2i+1 of lane group q hold token 4q + i, A = the
                    //    hi and mid bf16 parts of a (dl) in one product and the lo part and zero in a
                    //    second, B = dy (x) of the token in both slots; every product is exact.  Output
                    //    tile j, lane (n, q): levels 4q + r, column col + 8n + j.
                    // A, lane (level n, q): part (q / 2 ? mid : hi) of a (dl) for tokens 8(q % 2) .. +7, then
                    // their lo part (q < 2) or zero; B: dy (x) of the same tokens at the tile's column
                    const int half = q & 1;
                    const uint4 z4 = make_uint4(0u, 0u, 0u, 0u);
                    const bf16x8_t aa1 = __builtin_bit_cast(bf16x8_t, lds_u4(&s_aP[par][part][n][8 * half]));
                    const bf16x8_t aa2 = __builtin_bit_cast(bf16x8_t, part == 0 ? lds_u4(&s_aP[par][2][n][8 * half]) : z4);
                    const bf16x8_t ad1 = __builtin_bit_cast(bf16x8_t, lds_u4(&s_dlP[par][part][n][8 * half]));
                    const bf16x8_t ad2 = __builtin_bit_cast(bf16x8_t, part == 0 ? lds_u4(&s_dlP[par][2][n][8 * half]) : z4);
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const int at = (16 * j + n) * 16 + 8 * half;
                        const bf16x8_t bd = __builtin_bit_cast(bf16x8_t, lds_u4(t16 + at));
                        const bf16x8_t bx = __builtin_bit_cast(bf16x8_t, lds_u4(t16 + 2048 + at));
                        ao[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aa1, bd, ao[j], 0, 0, 0);
                        ao[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aa2, bd, ao[j], 0, 0, 0);
                        ai[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ad1, bx, ai[j], 0, 0, 0);
                        ai[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ad2, bx, ai[j], 0, 0, 0);
                    }
                } else {
                    // 4. dW sums on fp32 MFMA, four tokens per step: A = a (dl) of token 4s + q at level n,
                    //    B = dy (x) of that token at columns col + 8n .. +7 (absent tokens have a = dl = 0)
                    if constexpr (!EARLY_X) load_x();
#pragma unroll
                    for (int s = 0; s < 4; ++s) {
                        const float av = s_a[par][4 * s + q][n], dlv = s_dl[par][4 * s + q][n];
                        Raw8<DYBF> dyB;
#pragma unroll
                        for (int w = 0; w < DW; ++w) dyB.w[w] = s_dy[wave][(4 * s + q) * (16 * DW + 1) + n * DW + w];
                        float dy8[8], x8[8];
                        to8f<DYBF>(dyB, dy8);
                        to8f<XBF>(xB[s], x8);
#pragma unroll
                        for (int j = 0; j < 8; ++j) {
                            ao[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, dy8[j], ao[j], 0, 0, 0);
                            ai[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(dlv, x8[j], ai[j], 0, 0, 0);
                        }
                    }
                }
            }
        }
        pos0 += c;
        // rows this leaf completes (levels lv >= k whose node's last leaf this is)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int lv = 4 * q + r;
            if (lv <= D && lv >= k && ((leaf + 1) & ((int64_t(1) << (D - lv)) - 1)) == 0) {
                const int64_t node = ((leaf + L) >> (D - lv)) - 1;
                float v[8];
                if (p.dw_out) {
#pragma unroll
                    for (int j = 0; j < 8; ++j) v[j] = ao[j][r];
                    put8(p.dw_out + node * H + col + 8 * n, add, v);
                }
                if (p.dw_in) {
#pragma unroll
                    for (int j = 0; j < 8; ++j) v[j] = ai[j][r];
                    put8(p.dw_in + node * H + col + 8 * n, add, v);
                }
#pragma unroll
                for (int j = 0; j < 8; ++j) ao[j][r] = ai[j][r] = 0.0f;
            }
        }
    }
    // levels above the subtree root: this subtree's sums for the fix-up
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int lv = 4 * q + r;
        if (lv < k) {
            float* dst = p.part + ((st * k + lv) * 2) * H + col + 8 * n;
            float v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = ao[j][r];
            put8(dst, false, v);
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = ai[j][r];
            put8(dst + H, false, v);
        }
    }
}

// Rows of the levels above the subtrees (lv < k): node u at level lv sums the
// part[] of its 2^(k-lv) subtrees.  One block per (tree, level, matrix,
// 64-column slice); thread (column quad c, group g) owns four columns and
// subtrees g*per .. g*per + per - 1 (G = min(64, 2^k) groups of per = 2^k / G
// <= 8 subtrees) and loads them at once, 16 bytes per subtree.  A node inside
// one group is summed there in subtree order; a node spanning several groups
// adds its groups' sums in group order through LDS.  The order is fixed, so
// the rows are the same on every run.
constexpr int WSUM_GROUPS = 64;
constexpr int WSUM_QUADS = 16;  // column quads per block: 64 columns
constexpr int WSUM_BLOCK = WSUM_QUADS * WSUM_GROUPS;
static_assert((1 << WT_TOP_LEVELS) <= 8 * WSUM_GROUPS, "a group holds at most eight subtrees");

__device__ __forceinline__ float4 add4(float4 a, const float4& b) {
    a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
    return a;
}

__global__ __launch_bounds__(WSUM_BLOCK) void bwd_wsum_kernel(BwdParams p, int k) {
    __shared__ float4 red[WSUM_GROUPS][WSUM_QUADS + 1];
    const int c = threadIdx.x % WSUM_QUADS, g = threadIdx.x / WSUM_QUADS;
    const int64_t H = p.hidden, slices = H / (4 * WSUM_QUADS);
    const int64_t slice = blockIdx.x % slices;
    const int mat = int((blockIdx.x / slices) % 2);
    const int lv = int(blockIdx.x / (2 * slices));  // < k
    const int64_t col = (slice * WSUM_QUADS + c) * 4;
    const int t = blockIdx.y;
    const int64_t S = int64_t(1) << k;
    const int G = S < WSUM_GROUPS ? int(S) : WSUM_GROUPS;
    const int per = int(S / G);
    const int span = 1 << (k - lv);  // subtrees under a node of this level
    float* dw = mat == 0 ? p.dw_out : p.dw_in;
    auto store = [&](int64_t u, float4 v) {  // node u of the level
        if (!dw) return;
        float4* d = reinterpret_cast<float4*>(dw + (int64_t(t) * p.n_nodes + ((int64_t(1) << lv) - 1) + u) * H + col);
        *d = p.accumulate ? add4(v, *d) : v;
    };
    float4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int64_t st = int64_t(g) * per + j;
        v[j] = g < G && j < per
                   ? *reinterpret_cast<const float4*>(p.part + ((((int64_t(t) << k) + st) * k + lv) * 2 + mat) * H + col)
                   : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    if (span <= per) {  // block-uniform
        if (g < G)
            for (int j0 = 0; j0 < per; j0 += span) {
                float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (j >= j0 && j < j0 + span) sum = add4(sum, v[j]);
                store((int64_t(g) * per + j0) >> (k - lv), sum);
            }
        return;
    }
    float4 sum = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int j = 0; j < 8; ++j)
        if (j < per) sum = add4(sum, v[j]);
    red[g][c] = sum;
    __syncthreads();
    const int ng = span / per;  // groups per node
    if (g < G && g % ng == 0) {
        float4 tot = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int i = 0; i < ng; ++i) tot = add4(tot, red[g + i][c]);
        store((int64_t(g) * per) >> (k - lv), tot);
    }
}

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

int32_t bwd_piece(int64_t n_tokens, int32_t n_trees) {
    // about 1024 pieces over all trees (x 3 column slices at hidden 768: three
    // waves per SIMD), at least 64 positions (one perm load per lane)
    const int64_t want = (n_tokens * n_trees + 1023) / 1024;
    return int32_t(std::max<int64_t>(64, (want + 63) / 64 * 64));
}

static int64_t bwd_pieces(int64_t n_tokens, int32_t piece) { return std::max<int64_t>(1, (n_tokens + piece - 1) / piece); }

// Tokens per chunk of the stable placement: one per rank-kernel thread, more (up to 16) once the
// batch would need over 512 chunks, which bounds the [chunks, leaves] table.
// Tokens per chunk of the stable sort: RANKW_BLOCK with the ballot rank kernel (its leaf
// counters in LDS), else RANK_BLOCK x 1..16 for the compare-all rank kernel.
static int32_t bwd_chunk(int64_t n_tokens, int32_t depth) {
    if (depth <= RANKW_MAX_DEPTH) return RANKW_BLOCK;
    const int64_t per = std::min<int64_t>(16, std::max<int64_t>(1, (n_tokens + RANK_BLOCK * 512 - 1) / (RANK_BLOCK * 512)));
    return int32_t(RANK_BLOCK * per);
}
static int64_t bwd_chunks(int64_t n_tokens, int32_t depth) {
    const int64_t c = bwd_chunk(n_tokens, depth);
    return std::max<int64_t>(1, (n_tokens + c - 1) / c);
}

// The leaf-tiled weight kernel takes depth <= 15 (levels are the rows of a 16x16 MFMA) and
// hidden a multiple of 128; it hangs its subtrees at level min(depth, WT_TOP_LEVELS).
static bool wtile_shape(int32_t depth, int32_t hidden) { return depth <= 15 && hidden % 128 == 0; }
static int wtile_k(int32_t depth) { return std::min<int32_t>(depth, WT_TOP_LEVELS); }

size_t bwd_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t hidden) {
    const size_t recs = size_t(n_tokens) * size_t(n_trees);
    const size_t bins = (size_t(1) << depth) * size_t(n_trees);
    size_t parts;
    if (wtile_shape(depth, hidden)) {
        const int k = wtile_k(depth);
        parts = size_t(n_trees) * (size_t(1) << k) * size_t(k) * 2 * size_t(hidden);
    } else {
        parts = size_t(n_trees) * size_t(bwd_pieces(n_tokens, bwd_piece(n_tokens, n_trees))) * size_t(depth + 1) *
                4 * size_t(hidden);
    }
    return align256(recs * size_t(depth + 1) * sizeof(float2)) + 2 * align256(bins * sizeof(int32_t)) +
           align256(recs * sizeof(int32_t)) + align256(size_t(n_trees) * sizeof(int32_t)) +
           align256(recs * sizeof(int32_t)) + align256(bins * size_t(bwd_chunks(n_tokens, depth)) * sizeof(int32_t)) +
           align256(BWD_JUNK_BYTES) + align256(parts * sizeof(float));
}

void bwd_workspace_views(BwdParams& p, void* workspace) {
    char* w = static_cast<char*>(workspace);
    const size_t recs = size_t(p.n_tokens) * size_t(p.n_trees);
    const size_t bins = (size_t(1) << p.depth) * size_t(p.n_trees);
    p.piece = bwd_piece(p.n_tokens, p.n_trees);
    p.pieces = int32_t(bwd_pieces(p.n_tokens, p.piece));
    p.coef = reinterpret_cast<float2*>(w);
    w += align256(recs * size_t(p.depth + 1) * sizeof(float2));
    p.counts = reinterpret_cast<int32_t*>(w);
    w += align256(bins * sizeof(int32_t));
    p.offs = reinterpret_cast<int32_t*>(w);
    w += align256(bins * sizeof(int32_t));
    p.perm = reinterpret_cast<int32_t*>(w);
    w += align256(recs * sizeof(int32_t));
    p.total = reinterpret_cast<int32_t*>(w);
    w += align256(size_t(p.n_trees) * sizeof(int32_t));
    p.chunk = bwd_chunk(p.n_tokens, p.depth);
    p.chunks = bwd_chunks(p.n_tokens, p.depth);
    p.rank = reinterpret_cast<int32_t*>(w);
    w += align256(recs * sizeof(int32_t));
    p.hist = reinterpret_cast<int32_t*>(w);
    w += align256(bins * size_t(p.chunks) * sizeof(int32_t));
    p.junk = w;
    w += align256(BWD_JUNK_BYTES);
    p.part = reinterpret_cast<float*>(w);
}

// The fix-up of the rows above the subtrees (levels 0 .. k-1) after bwd_wtile_kernel or
// bwd_fused_kernel.
static hipError_t launch_wsum(BwdParams& p, int k, hipStream_t stream) {
    if (k <= 0) return hipSuccess;
    int kk = k;
    void* fargs[] = {&p, &kk};
    return hipLaunchKernel(reinterpret_cast<const void*>(&bwd_wsum_kernel),
                           dim3(unsigned(int64_t(k) * 2 * (p.hidden / (4 * WSUM_QUADS))), unsigned(p.n_trees)),
                           dim3(WSUM_BLOCK), fargs, 0, stream);
}

// The stable placement in leaf order (rank, [leaf sums], scan, base, place).
static hipError_t launch_sort(BwdParams& p, bool count_leaves, const int64_t cap, hipStream_t stream) {
    void* args[] = {&p};
    const int64_t bins = (int64_t(1) << p.depth) * p.n_trees;
    hipError_t e =
        p.depth <= RANKW_MAX_DEPTH
            ? hipLaunchKernel(reinterpret_cast<const void*>(&bwd_rank_wave_kernel), dim3(unsigned(p.chunks), p.n_trees),
                              dim3(RANKW_BLOCK), args, size_t(bins / p.n_trees) * sizeof(int32_t), stream)
            : hipLaunchKernel(reinterpret_cast<const void*>(&bwd_rank_kernel), dim3(unsigned(p.chunks), p.n_trees),
                              dim3(RANK_BLOCK), args, size_t(p.chunk) * sizeof(int32_t), stream);
    if (e != hipSuccess) return e;
    if (count_leaves) {
        e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_leafsum_kernel),
                            dim3(unsigned((bins + BWD_BLOCK / 64 - 1) / (BWD_BLOCK / 64))), dim3(BWD_BLOCK), args, 0,
                            stream);
        if (e != hipSuccess) return e;
    }
    // the fused path (leaf counts from bwd_leafsum_kernel, one tree) with few leaves: the base
    // kernel finds each leaf's start itself; otherwise the scan kernel (which also gives the total)
    int self_scan = count_leaves && p.n_trees == 1 && bins <= BASE_SELF_SCAN_LEAVES;
    if (!self_scan) {
        e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_scan_kernel), dim3(p.n_trees), dim3(SCAN_BLOCK), args,
                            0, stream);
        if (e != hipSuccess) return e;
    }
    void* bargs[] = {&p, &self_scan};
    e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_base_kernel),
                        dim3(unsigned((bins + BWD_BLOCK / 64 - 1) / (BWD_BLOCK / 64))), dim3(BWD_BLOCK), bargs, 0, stream);
    if (e != hipSuccess) return e;
    const int64_t n = p.n_tokens * p.n_trees;
    const int grid = int(std::max<int64_t>(1, std::min<int64_t>((n + BWD_BLOCK - 1) / BWD_BLOCK, cap)));
    return hipLaunchKernel(reinterpret_cast<const void*>(&bwd_place_kernel), dim3(grid), dim3(BWD_BLOCK), args, 0,
                           stream);
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
    const int64_t cap = int64_t(dev.cu_count) * 8;
    // bf16 weights, one tree, depth <= 15, hidden 128..1024: the fused leaf-tiled backward
    p.fused = p.need_dw && p.w_bf16 && p.n_trees == 1 && wtile_shape(p.depth, p.hidden) && p.hidden <= 1024;
    if (p.fused) {
        hipError_t e = launch_sort(p, true, cap, stream);
        if (e != hipSuccess) return e;
        const int k = wtile_k(p.depth);
        int sub = p.depth - k;
        const void* kern = p.x_bf16 ? (p.dy_bf16 ? reinterpret_cast<const void*>(&bwd_fused_kernel<true, true>)
                                                 : reinterpret_cast<const void*>(&bwd_fused_kernel<true, false>))
                                    : (p.dy_bf16 ? reinterpret_cast<const void*>(&bwd_fused_kernel<false, true>)
                                                 : reinterpret_cast<const void*>(&bwd_fused_kernel<false, false>));
        void* fargs[] = {&p, &sub};
        e = hipLaunchKernel(kern, dim3(unsigned(int64_t(1) << k)), dim3(64 * (p.hidden / 128)), fargs, 0, stream);
        if (e != hipSuccess) return e;
        return launch_wsum(p, k, stream);
    }
    void* args[] = {&p};
    if (p.need_dw) {  // zero the leaf counts (a fill kernel: no memset nodes)
        const int64_t bins = (int64_t(1) << p.depth) * p.n_trees;
        float* a = nullptr;
        int64_t na = 0;
        int32_t* b = p.counts;
        int64_t nb = bins;
        void* fa[] = {&a, &na, &b, &nb};
        const int grid = int(std::min<int64_t>((bins + BWD_BLOCK - 1) / BWD_BLOCK, cap));
        const hipError_t e =
            hipLaunchKernel(reinterpret_cast<const void*>(&bwd_fill_kernel), dim3(grid), dim3(BWD_BLOCK), fa, 0, stream);
        if (e != hipSuccess) return e;
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
    hipError_t e = launch_sort(p, false, cap, stream);
    if (e != hipSuccess) return e;
    if (wtile_shape(p.depth, p.hidden)) {  // weight sums on MFMA, leaf by leaf
        const int k = wtile_k(p.depth);
        int sub = p.depth - k;
        const void* kern = p.x_bf16 ? (p.dy_bf16 ? reinterpret_cast<const void*>(&bwd_wtile_kernel<true, true>)
                                                 : reinterpret_cast<const void*>(&bwd_wtile_kernel<true, false>))
                                    : (p.dy_bf16 ? reinterpret_cast<const void*>(&bwd_wtile_kernel<false, true>)
                                                 : reinterpret_cast<const void*>(&bwd_wtile_kernel<false, false>));
        const int waves = std::min(p.hidden / 128, WT_WAVES_MAX);
        void* wargs[] = {&p, &sub};
        e = hipLaunchKernel(kern, dim3(unsigned(int64_t(1) << k), p.n_trees), dim3(64 * waves), wargs, 0, stream);
        if (e != hipSuccess) return e;
        return launch_wsum(p, k, stream);
    }
    const int slices = (p.hidden + SLICE - 1) / SLICE;
    {
        const int64_t waves = int64_t(p.pieces) * slices * p.n_trees;
        const int64_t grid = (waves + BWD_BLOCK / 64 - 1) / (BWD_BLOCK / 64);
        e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_piece_kernel), dim3(unsigned(grid)), dim3(BWD_BLOCK),
                            args, 0, stream);
        if (e != hipSuccess) return e;
    }
    {
        // Levels whose runs span about eight pieces or more under uniform routing get a block
        // per node; any routing is handled correctly by either kernel.
        int top = 0;
        while (top < p.depth + 1 && (int64_t(p.pieces) >> top) >= 8) ++top;
        if (top > 0) {
            const int64_t blocks = int64_t(p.n_trees) * ((int64_t(1) << top) - 1) * slices;
            void* targs[] = {&p, &top};
            e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_fixup_top_kernel), dim3(unsigned(blocks)),
                                dim3(FIX_BLOCK), targs, 0, stream);
            if (e != hipSuccess) return e;
        }
        const int64_t tasks = int64_t(p.n_trees) * (p.n_nodes - ((int64_t(1) << top) - 1)) * slices;
        if (tasks > 0) {
            const int64_t grid = std::min<int64_t>((tasks + BWD_BLOCK / 64 - 1) / (BWD_BLOCK / 64), cap * 4);
            void* fargs[] = {&p, &top};
            e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_fixup_kernel), dim3(unsigned(grid)),
                                dim3(BWD_BLOCK), fargs, 0, stream);
            if (e != hipSuccess) return e;
        }
    }
    return hipSuccess;
}

}  // namespace fff
