// fff_internal.hpp -- what the C-ABI front end (fff_api.cpp) and the kernel
// translation unit (fff_kernels.hip) share: the kernel parameter block, the
// launch plan and the planning/launch entry points.  Not part of the ABI.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstddef>
#include <cstdint>

namespace fff {

// Kernel argument block, passed by value.
struct Params {
    const void* x;
    const void* w_in;
    const void* w_out;
    void* y;
    int32_t* nodes_out;   // optional [B, T, D+1]
    float* logits_out;    // optional [B, T, D+1]
    int64_t n_tokens;
    int64_t n_nodes;      // per tree: 2^(D+1) - 1
    int32_t hidden;
    int32_t depth;
    int32_t n_trees;
    int32_t x_bf16, w_bf16, y_bf16;
    int32_t act;
    int32_t out_mode;
    int32_t lds_levels;   // levels staged in LDS
    int32_t walk_affine;  // walk kernel: each workgroup walks one tree, chosen by its XCD (T divides 8)
    // grouped mode: views into the caller's workspace
    float* ws_act;        // [B, T, D+1] activation of every visited node
    int32_t* ws_leaf;     // [B, T] leaf reached in each tree
    int32_t split_level;  // group tokens by their tree-0 node at this level; 0 = keep token order
    // tiled mode: tokens bucketed by their leaf in every tree during the walk
    int32_t* bk_count;    // [T, 2^D] tokens that reached each leaf
    int32_t* bk_tok;      // [T, 2^D, bk_cap] the first bk_cap of them, in arrival order
    int32_t* bk_spill;    // [T, B] tokens that found their bucket full
    int32_t* bk_nspill;   // [T] how many
    float* bk_act;        // [T, 2^D, bk_cap, TILE_REC] activations of the bucketed tokens, by slot
    int32_t bk_cap;
    int32_t tile_tree;    // the tree a tile launch accumulates
    const void* tile_src; // [B, H] row the tile launch adds its result to (or null)
    void* tile_dst;       // [B, H] row it writes
    // LayerNorm prologue (norm = 1): u = (x - mean) / sqrt(var + eps) * gamma + beta
    int32_t norm;
    float norm_eps;
    const float* gamma;   // [H] or null (ones)
    const float* beta;    // [H] or null (zeros)
};

// One layer of a stack: its weights and LayerNorm parameters.
struct LayerPtrs {
    const void* w_in;
    const void* w_out;
    const float* gamma;
    const float* beta;
};

// Layers handled by one launch of the stack kernel (the table travels in the
// kernel arguments); longer stacks take several launches, in place on y.
constexpr int STACK_MAX_LAYERS = 32;

struct StackParams {
    Params p;             // x, y, shapes, dtypes, norm, records base; w_in/w_out unused
    int32_t n_layers;
    int64_t rec_stride;   // elements between consecutive layers' records
    LayerPtrs layer[STACK_MAX_LAYERS];
};

// Backward (hard routing) argument block, passed by value.
struct BwdParams {
    const void* x;
    const void* w_in;
    const void* w_out;
    const void* dy;
    const int32_t* leaves;   // [B, T]
    const float* logits;     // [B, T, D+1]
    void* dx;                // [B, H] or null
    float* dw_in;            // [T, N, H] or null
    float* dw_out;           // [T, N, H] or null
    int32_t* bad;            // optional counter of skipped (token, tree) pairs
    int64_t n_tokens;
    int64_t n_nodes;
    int32_t hidden, depth, n_trees;
    int32_t x_bf16, w_bf16, dy_bf16, dx_bf16;
    int32_t act, accumulate;
    // workspace views
    float2* coef;            // [B, T, D+1]: (act(l), dLoss/dl) of every visit
    int32_t* counts;         // [T, 2^D] tokens per leaf
    int32_t* offs;           // [T, 2^D] first sorted position of each leaf, then the scatter cursor
    int32_t* perm;           // [T, B] token indices sorted by leaf
    int32_t* total;          // [T] valid (token, tree) pairs per tree
    int32_t* rank;           // [T, B] rank of each token among its leaf's tokens earlier in its chunk
    int32_t* hist;           // [T, chunks, 2^D] tokens per (chunk, leaf), then their first sorted position
    int64_t chunks;          // token chunks of the stable placement
    int32_t chunk;           // tokens per chunk
    int32_t fused;           // the fused leaf-tiled path runs (no token kernel)
    float* part;             // [T, pieces, D+1, 2 slots, 2 matrices, H] run sums that cross pieces
    char* junk;              // BWD_JUNK_BYTES the fused kernel sends the stores of absent dx rows to
    int32_t piece;           // sorted positions per piece of the weight kernel
    int32_t pieces;          // pieces per tree
    int32_t need_dw;         // dW_in or dW_out requested
};

// Sorted positions per piece of the backward's weight kernel (a multiple of 64).
int32_t bwd_piece(int64_t n_tokens, int32_t n_trees);
// Workspace of the backward; the views are carved by bwd_workspace_views.
size_t bwd_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t hidden);
void bwd_workspace_views(BwdParams& p, void* workspace);

constexpr int XCDS = 8;  // MI355X: 8 XCDs, workgroups dealt to them round-robin
constexpr int TILE_REC = 16;  // floats per activation record of a bucketed token (tiled mode)

struct DeviceInfo {
    int device = -1;
    int cu_count = 0;
    size_t lds_per_block = 0;  // bytes
    size_t lds_per_cu = 0;     // bytes
};

enum KernelKind {
    KIND_NONE = 0, KIND_DESCENT = 1, KIND_GENERIC = 2, KIND_GROUPED = 3, KIND_STACK = 4, KIND_TILED = 5, KIND_MASKED = 6,
    KIND_SUBTREE = 7
};

struct Launch {
    const void* kernel = nullptr;  // __global__ function handle
    int grid = 0;                  // blocks
    int block = 0;                 // threads per block
    size_t lds_bytes = 0;          // dynamic LDS per block
};

struct Plan {
    int kind = KIND_NONE;
    Launch launch[3];              // descent/generic: [0]; grouped: walk, emit; tiled: fill, walk, tiles (one per tree)
    int n_launch = 0;
    int lanes = 0;                 // lanes per token
    int emit_lanes = 0;            // lanes per token of the grouped emit
    int lds_levels = 0;            // descent, generic, grouped walk
    int emit_lds_levels = 0;       // grouped emit
    int split_level = 0;           // grouped mode
    int walk_affine = 0;           // grouped / tiled: one tree per walk workgroup, by XCD
    int tile_pair = 0;             // tiled: a tile workgroup per pair of sibling leaves
    int cu_count = 0;              // masked: compute units, for the products' tile choice
    const char* name = "";
};

// Fills *plan for a validated request; returns an fff_status value.
// workspace_bytes: size of the 256-byte aligned workspace the caller passed (0
// if none); AUTO picks the grouped or tiled path only when it covers that
// path's scratch.
// masked_ok: whether MASKED may be planned (the entry point that allocates nothing excludes it: its
// workspace is far larger than that entry point's scratch).
int plan_forward(const Params& p, int mode, int lds_levels_req, int split_level_req, size_t workspace_bytes,
                 const DeviceInfo& dev, Plan* plan, bool masked_ok = true);

// Scratch of the entry point that allocates nothing (fff_forward_static): a file-scope device
// array of STATIC_SCRATCH_BYTES, one per GPU, held until the process ends.  Its device address
// on `device` (the current device), looked up once per device.
constexpr size_t STATIC_SCRATCH_BYTES = size_t(64) << 20;
hipError_t static_scratch(int device, void** ptr);

// Enqueues the planned work on stream; returns the first failing HIP error.
hipError_t run_forward(const Params& p, const Plan& plan, void* workspace, size_t workspace_bytes,
                       hipStream_t stream);

// Enqueues the backward on stream.  *status is ST_OK, or FFF_ERR_UNSUPPORTED's
// value when no kernel fits (nothing enqueued); returns the first HIP error.
hipError_t run_backward(BwdParams p, const DeviceInfo& dev, hipStream_t stream, int* status);

// Stack of layers in one persistent kernel: fills *plan (KIND_STACK) when a
// kernel is instantiated for the shape and types, else returns ST_UNSUPPORTED.
int plan_stack(const Params& p, int lds_levels_req, const DeviceInfo& dev, Plan* plan);

// Enqueues the stack kernel for layers [0, n) of sp (n <= STACK_MAX_LAYERS).
hipError_t run_stack(const StackParams& sp, const Plan& plan, hipStream_t stream);

// Grouped mode scratch size for a resolved split level (0 = no bucketing).
size_t grouped_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t split_level);
// Tiled mode scratch (grouped scratch plus the leaf buckets); 0 when the shape has no tiled mode.
size_t tiled_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t hidden);
// Split level used when the caller asks for the default (0 in fff_args).
int default_split_level(int32_t depth, int32_t n_trees);

// Masked mode (two dense products around the walk, fff_masked.hip): the deepest tree it takes,
// and where AUTO picks it: bf16 x and W at depth at most MASKED_AUTO_DEPTH with at least
// MASKED_AUTO_TREES trees, or three quarters as many and MASKED_AUTO_TOKENS tokens; fp32 x, W and
// y at depth at most MASKED_AUTO_DEPTH_F32 with at least MASKED_AUTO_TREES_F32 trees (its
// products and selection cost 30-55 us even at a few hundred tokens, which fewer trees do not
// win back; measured against every mode at 4..64 trees, 1024 and 16384 tokens).
constexpr int MASKED_MAX_DEPTH = 7;
constexpr int MASKED_AUTO_DEPTH = 5;
constexpr int MASKED_AUTO_DEPTH_F32 = 4;
constexpr int MASKED_AUTO_TREES = 16;
constexpr int MASKED_AUTO_TREES_F32 = 32;
constexpr int64_t MASKED_AUTO_TOKENS = 16384;
// Whether a validated request can run masked (types, depth, no LayerNorm, residual types).
bool masked_shape(const Params& p);
// Masked mode scratch (logits, split activations, transposed and repeated W_out); 0 past
// MASKED_MAX_DEPTH.
size_t masked_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t hidden);
// Enqueues the masked forward on stream.
hipError_t run_masked(const Params& p, void* workspace, int cu_count, hipStream_t stream);

// Dense products of MASKED mode on the matrix cores (fff_gemm.hip): C = A B^T with A [M, K] and
// B [N, K] row-major (K-contiguous, leading dimensions lda / ldb in elements, 16-byte aligned rows,
// K a multiple of 8 for bf16 or 4 for fp32), bf16 (bf16 = true) or fp32 inputs, fp32 accumulation.
// out: GEMM_OUT_F32 stores C as fp32; GEMM_OUT_SRC_* add a source matrix (none, fp32, bf16; leading
// dimension ldc like C, may be C itself) and store as bf16 (dst_bf16) or fp32.  fp32 inputs take
// fp32 sources and destinations only.  GEMM_OUT_ACT_* store the activation a = act(C) over whole
// rows of ldc >= N columns (zeros past N, ldc a multiple of 4): GEMM_OUT_ACT_F32 (fp32 inputs)
// as fp32, GEMM_OUT_ACT_P2 (bf16 inputs) as hi = bf16(a) at element 2 m ldc + n and
// bf16(a - hi) at ldc past it.  Any other combination returns hipErrorInvalidValue.  cu_count:
// compute units of the device (tile choice).
// split_ws / split_bytes: device scratch for the partial sums of a product split along K (a small
// product with a long K; none when null), fully overwritten before it is read.  The kernels, tile
// shape and split depend on the shapes, cu_count and split_bytes only, so the result bits do too.
enum {
    GEMM_OUT_F32 = 0,
    GEMM_OUT_SRC_NONE = 1,
    GEMM_OUT_SRC_F32 = 2,
    GEMM_OUT_SRC_BF16 = 3,
    GEMM_OUT_ACT_F32 = 4,
    GEMM_OUT_ACT_P2 = 5
};
constexpr size_t GEMM_SPLIT_BYTES = size_t(32) << 20;  // masked mode's partial-sum scratch
hipError_t gemm_nt(bool bf16, int out, bool dst_bf16, const void* A, const void* B, void* C, const void* src,
                   int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t ldc, int cu_count,
                   void* split_ws, size_t split_bytes, int act, hipStream_t stream);

// Subtree mode (fff_subtree.hip): a workgroup per token evaluates whole subtrees of logits per
// step.  AUTO takes it for at most SUBTREE_AUTO_TREES trees of depth at least SUBTREE_AUTO_DEPTH
// while tokens x trees stay within SUBTREE_AUTO_PAIRS (SUBTREE_AUTO_PAIRS_WIDE at hidden sizes
// above 1024, where a step's rows are four times longer; SUBTREE_AUTO_PAIRS_DEEP_F32 for fp32
// weights at depth >= SUBTREE_DEEP_F32, whose five-level steps read 31 rows of 3 KB per level
// walked: at 256 tokens the fused kernel is ahead, 11.6 against 12.1 us at depth 11 and 12.2
// against 13.3 at depth 13).
constexpr int SUBTREE_AUTO_DEPTH = 5;
constexpr int SUBTREE_AUTO_TREES = 4;
constexpr int64_t SUBTREE_AUTO_PAIRS = 256;
constexpr int64_t SUBTREE_AUTO_PAIRS_WIDE = 32;
constexpr int SUBTREE_DEEP_F32 = 11;
constexpr int64_t SUBTREE_AUTO_PAIRS_DEEP_F32 = 128;
bool subtree_auto(const Params& p);
// Whether a validated request has a subtree kernel (hidden size and types; no LayerNorm).
bool subtree_shape(const Params& p);
int subtree_span(const Params& p);          // levels per step
const char* subtree_name(const Params& p);
int subtree_block(const Params& p);          // threads per workgroup
int subtree_grid(const Params& p, int cu_count);
hipError_t run_subtree(const Params& p, int grid, hipStream_t stream);

}  // namespace fff
