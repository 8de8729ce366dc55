/*
 * fff.h -- C ABI of libfff.so: fast-feedforward (FFF) inference on AMD
 * Instinct MI355X (gfx950).
 *
 * The operation is the FFF forward pass of "Exponentially Faster Language
 * Modeling" (Belcak and Wattenhofer, 2023): conditional matrix multiplication
 * (CMM, Algorithm 1) followed by the output accumulation, with the model
 * changes of Section 2.1 (the same activation at every node, output weights
 * on every node, no biases, leaf size 1, several trees summed).  For every
 * token b and tree t, starting at the root n = 0, at each level l = 0..D:
 *
 *     logit  = <x[b,:], W_in[t,n,:]>
 *     y[b,:] += act(logit) * W_out[t,n,:]
 *     n      = 2n + 1 + (logit > 0)          (if l < D; a zero logit goes left)
 *
 * so each token visits D+1 of the N = 2^(D+1) - 1 nodes of each tree.
 *
 * Conventions shared by every entry point:
 *   - depth D counts edges on a root-to-leaf path (UltraFastBERT-KxD naming,
 *     Table 1): depth 11 is the 4095-node tree of UltraFastBERT-1x11.
 *   - layouts (all row-major, contiguous, no strides):
 *       x      [n_tokens, hidden]
 *       y      [n_tokens, hidden]
 *       W_in   [n_trees, N, hidden], node rows in heap order (children of n
 *       W_out  [n_trees, N, hidden]  are 2n+1 and 2n+2); row n of tree t
 *                                    starts at element (t*N + n)*hidden.
 *   - every data pointer is a DEVICE pointer owned by the caller; the library
 *     never frees or retains them.  Base pointers must be 16-byte aligned.
 *   - y may be the very buffer x (in place) when x_dtype == y_dtype; any other
 *     overlap of an output with an input is rejected.
 *   - arithmetic is fp32 (bf16 inputs are widened exactly); bf16 outputs are
 *     rounded to nearest even.
 *   - work is enqueued on hip_stream (NULL = the null stream) and the call
 *     returns without waiting; device faults surface at the caller's next
 *     synchronisation.
 *   - every argument check runs before any HIP call; on a non-zero return no
 *     device work has been enqueued, except FFF_ERR_HIP, which reports a
 *     failed HIP call (see fff_last_hip_error).
 *   - the library is reentrant.  Its global state: a per-device property
 *     cache, a cache of occupancy queries per kernel, the thread-local last
 *     HIP error, and the device address of fff_forward_static's scratch per
 *     device.  No call waits on the device.
 */
#ifndef FFF_H_
#define FFF_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FFF_VERSION 101 /* major * 100 + minor */

typedef enum {
    FFF_OK = 0,
    FFF_ERR_INVALID_ARG = -1, /* a null pointer, bad size, bad enum, misalignment or x/y overlap */
    FFF_ERR_UNSUPPORTED = -2, /* valid request the library has no kernel for */
    FFF_ERR_WORKSPACE = -3,   /* grouped mode without enough workspace */
    FFF_ERR_HIP = -4          /* a HIP runtime call failed */
} fff_status;

typedef enum { FFF_F32 = 0, FFF_BF16 = 1 } fff_dtype;

/* GELU in its exact form z*Phi(z) (the paper's activation, Section 2.1), its
 * tanh approximation, or the identity (for exact integer tests). */
typedef enum { FFF_ACT_GELU_ERF = 0, FFF_ACT_GELU_TANH = 1, FFF_ACT_IDENTITY = 2 } fff_act;

/* DESCENT: one kernel; a 16/32/64-lane group per token walks each tree and
 * accumulates the output, the top levels served from LDS.
 * GROUPED: two kernels; the walk (the CMM proper) stores every token's leaf
 * and activations in the workspace, then the output rows are accumulated with
 * tokens grouped by their tree-0 node at a split level, each group's subtree
 * handled by the workgroups of one XCD so that its rows stay in that XCD's L2.
 * With 2, 4 or 8 trees (GROUPED and TILED) each walk workgroup walks the tree
 * of its XCD, with that tree's top levels in LDS.
 * GENERIC: any hidden size, one wave per token.
 * TILED: 1..16 trees, depth 5..15, hidden a multiple of 128: the walk drops
 * each token into a bucket of its leaf in every tree, and the output rows of up
 * to 16 tokens that share a leaf (hence all D+1 nodes) are accumulated as one
 * dense product on MFMA, one launch per tree in tree order, each adding its
 * tree to the running sum (fp32 y in place; for a bf16 y an fp32 row of the
 * workspace, rounded once by the last tree): fp32 MFMA for fp32 weights; for bf16 weights bf16 MFMA on the
 * activations split into bf16 parts (three parts: fp32 working accuracy; two,
 * relative error about 2^-17, when y is bf16 and either stored or the residual
 * of bf16 x).  Below 16 tokens per leaf on average (depth <= 14) one
 * workgroup takes a pair of sibling leaves: their tokens share the rows of
 * levels 0..D-1 and fill one list of tiles, with the two leaves' rows as two
 * extra rows of the product (each token's leaf activation on its own leaf's
 * row, zero on the other).  When more tokens reach a leaf than its bucket
 * holds, all of that leaf's tokens (with pairs, both leaves') take the
 * per-token emit instead, so the output bits do not depend on the order in
 * which the walk filled the bucket's slots.  A call
 * with more than (2^31 - 1) / (4 hidden) tokens (699050 at hidden 768) runs as
 * consecutive chunks of that many tokens, each a complete tiled forward (the
 * output stores use 32-bit offsets).  Needs the workspace of
 * fff_workspace_bytes.
 * MASKED: bf16 x and W, or fp32 x, W and y; depth <= 7, no LayerNorm (a
 * residual needs y of x's type): the layer as two dense products around the
 * walk, for shallow trees
 * where a token uses a large share of the nodes (at depth 0 the layer is the
 * dense feedforward): the logits of all nodes as one bf16 GEMM with fp32
 * accumulation (the library's own MFMA kernel), the walk of Algorithm 1 over
 * them per (token, tree) with the visited nodes' activations split into bf16
 * parts (two when y is bf16, three otherwise) and zeros elsewhere, then the
 * output as a second GEMM against W_out transposed and repeated once per
 * part.  With fp32 x, W and y both GEMMs are fp32 (fp32 MFMA) and the
 * activations go in whole.  At depth 0 with no records, where every node is
 * visited, the first product stores the activations itself (fp32, or two
 * bf16 parts when y is bf16), with the same bits.  The products' kernel and tile shapes depend on
 * the shapes and the device's CU count only, so the result bits do too.
 * Needs the workspace of fff_workspace_bytes (logits, parts, the transposed
 * W_out).
 * SUBTREE: hidden 768, 1024 or 4096 (any supported types), no LayerNorm; for
 * a few tokens, where the walk's D+1 dependent row loads are the time: one
 * workgroup of 1024 threads (512 for fp32 x with bf16 W at hidden >= 1024)
 * per token computes the logits of every node of a 3- to 6-level subtree
 * (64, 32 or 16 lanes per dot product) in one step and descends through
 * them in LDS, then loads the path's W_out rows together.  Reads up to 63/6
 * times the W_in rows of a walk.
 * AUTO (from measurements on MI355X): SUBTREE for at most 4 trees of depth
 * >= 5 and 256 token-tree pairs (32 at hidden 4096, 128 with fp32 W at depth
 * 11 or more); MASKED at depth <= 5
 * for 16 bf16 trees or more (12 from 16384 tokens), or at depth <= 4 for 32
 * fp32 trees or more, when the workspace covers it; for single-tree layers whose
 * workspace is large enough, TILED at depth 9..15 with at least 8 tokens per
 * leaf and 48M input elements (tokens x hidden), or 16 tokens per leaf and
 * 16M elements (bf16 W at depth 9: from 96M elements), and at depth 11 or
 * more with 8 tokens per leaf (fp32 W; from 2 per leaf at depth <= 14 with
 * 12M elements) or 4 per leaf at hidden 2048 or more (bf16 W); else GROUPED
 * at depth
 * 11 or more from 48M elements, or from 16384 tokens with fp32 W or 24M
 * elements, and with fp32 W at depth 5 or more from 65536 tokens; for 2, 4
 * or 8 trees of depth 7 or more (the walk tree-affine), with fp32 W TILED at
 * depth 11 or more from 8 tokens per leaf, at depth 10 from 16 or at depth 9
 * or more from 32 tokens per leaf, else GROUPED from 65536 tokens (16384 with 8
 * trees), and with bf16 W GROUPED for 8 trees, for 4 from 4096 tokens at
 * depth 8 or more (65536 at depth 7) and for 2 from 65536 tokens at depth 8
 * or more; GROUPED for 8 trees up to 2048 tokens with bf16 W (4096 at depth
 * 6 or more) or 1024 with fp32 W (the workspace covering it); otherwise
 * DESCENT when a
 * kernel is compiled for the hidden size and types, else GENERIC. */
typedef enum {
    FFF_MODE_AUTO = 0,
    FFF_MODE_DESCENT = 1,
    FFF_MODE_GROUPED = 2,
    FFF_MODE_GENERIC = 3,
    FFF_MODE_TILED = 4,
    FFF_MODE_MASKED = 5,
    FFF_MODE_SUBTREE = 6
} fff_mode;

/* What is written to y: FFF(u); y + FFF(u); or x + FFF(u) (the residual of a
 * transformer block), where u is x or its LayerNorm (fff_norm). */
typedef enum { FFF_OUT_STORE = 0, FFF_OUT_ACCUMULATE = 1, FFF_OUT_RESIDUAL = 2 } fff_out;

/* Normalisation applied to x before the tree walk.  The paper's layer replaces
 * the feedforward network inside crammedBERT's pre-norm intermediate layers
 * (Section 2.1), whose input is the LayerNorm of the residual stream:
 *   u_i = (x_i - mean(x)) / sqrt(var(x) + eps) * gamma_i + beta_i,
 * mean and biased variance over the hidden dimension, computed in fp32 per
 * token inside the kernels; the residual (FFF_OUT_RESIDUAL) adds the raw x. */
typedef enum { FFF_NORM_NONE = 0, FFF_NORM_LAYERNORM = 1 } fff_norm;

/*
 * fff_forward -- y = FFF(x) with the exact GELU, the paper's layer
 * (Algorithm 1 with the Section 2.1 changes).
 *
 *   x, W_in, W_out, y : device pointers, layouts above; y is x itself (same dtype)
 *                       or disjoint from it (W_in and W_out may alias).
 *   depth             : 0..24.       n_trees : >= 1.
 *   n_tokens          : >= 0 (0 is a no-op returning FFF_OK).
 *   hidden            : >= 1.
 *   x_dtype, w_dtype, y_dtype : FFF_F32 or FFF_BF16, independently.
 *   hip_stream        : a hipStream_t, or NULL.
 * Returns an fff_status.
 */
int fff_forward(const void* x, const void* W_in, const void* W_out, int32_t depth, int32_t n_trees,
                void* y, int64_t n_tokens, int32_t hidden, int32_t x_dtype, int32_t w_dtype,
                int32_t y_dtype, void* hip_stream);

/* Full form.  Zero-initialise, then set the fields; a zeroed struct with the
 * pointers and sizes filled in is the fff_forward call. */
typedef struct {
    const void* x;
    const void* W_in;
    const void* W_out;
    void* y;
    int64_t n_tokens;
    int32_t hidden;
    int32_t depth;
    int32_t n_trees;
    int32_t x_dtype, w_dtype, y_dtype; /* fff_dtype */
    int32_t act;                       /* fff_act */
    int32_t mode;                      /* fff_mode */
    int32_t out_mode;                  /* fff_out */
    int32_t lds_levels;   /* top tree levels cached in LDS (DESCENT); 0 = default choice,
                             -1 = none, k > 0 = exactly k (FFF_ERR_UNSUPPORTED if too big) */
    int32_t split_level;  /* GROUPED: group tokens by their tree-0 node at this level (3..depth);
                             0 = default (min(depth, 5) for one tree, else none);
                             -1 = keep token order */
    int32_t* nodes_out;   /* optional device [n_tokens, n_trees, depth+1]: node visited per level */
    float* logits_out;    /* optional device [n_tokens, n_trees, depth+1]: fp32 logit per level */
    void* workspace;      /* GROUPED: device scratch of at least fff_workspace_bytes() bytes,
                             256-byte aligned, disjoint from every other buffer; its contents
                             are overwritten (FFF_ERR_WORKSPACE if missing or too small) */
    size_t workspace_bytes;
    void* hip_stream;
    int32_t norm;              /* fff_norm */
    float norm_eps;            /* LayerNorm: >= 0 and finite (BERT uses 1e-12) */
    const float* norm_gamma;   /* LayerNorm: device fp32 [hidden] gain, or NULL for ones */
    const float* norm_beta;    /* LayerNorm: device fp32 [hidden] shift, or NULL for zeros */
} fff_args;

int fff_forward_ex(const fff_args* a);

/*
 * fff_forward_static -- fff_forward_ex that allocates nothing, for callers that
 * cannot allocate device memory during the call: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  The scratch of the
 * GROUPED and TILED plans is the library's own file-scope device array of
 * FFF_STATIC_SCRATCH_BYTES (64 MiB; one per GPU, held until the process ends),
 * looked up once per device; the call makes no hipMalloc, hipFree or other
 * allocating call.  Rules beyond fff_forward_ex's:
 *   - workspace must be NULL and workspace_bytes 0 (FFF_ERR_INVALID_ARG);
 *   - MASKED is not available (FFF_ERR_UNSUPPORTED; AUTO never picks it here:
 *     its workspace is far larger than the array);
 *   - AUTO picks GROUPED or TILED only when its scratch fits the array; an
 *     explicit GROUPED or TILED whose scratch (fff_workspace_bytes for that
 *     plan) exceeds FFF_STATIC_SCRATCH_BYTES returns FFF_ERR_WORKSPACE;
 *   - every call on one GPU shares that GPU's array, which keeps the last
 *     call's contents (the kernels clear what must start at zero): calls that
 *     overlap on one GPU -- concurrent streams or threads -- race and must be
 *     serialised by the caller.
 * At depth 11 (one tree) the tiled scratch fits up to 196608 tokens, three
 * times the 65536-token batch.
 */
#define FFF_STATIC_SCRATCH_BYTES ((size_t)64 << 20)
int fff_forward_static(const fff_args* a);

/* Device scratch bytes GROUPED, TILED and MASKED mode need for n_tokens
 * tokens: one fp32 activation per visited node and one int32 leaf per (token,
 * tree), plus for TILED the leaf buckets (int32 counts; token slots, a few
 * times the mean tokens per leaf, each with its D+1 fp32 activations; a spill
 * list; for one chunk of tokens at most), and at depth <= 7 MASKED's logits of every node (fp32), their bf16
 * parts, W_out transposed and repeated three times and 32 MiB for the
 * partial sums of a product split along K (few tokens).  The result
 * covers every mode; the split level (-1..depth) does not change it.
 * Returns 0 for invalid shapes. */
size_t fff_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t hidden,
                           int32_t split_level);

/* Short human-readable description of the kernel and launch fff_forward_ex
 * would use for these arguments (after validation), written into buf
 * (NUL-terminated, truncated to len).  Makes no HIP call other than the
 * cached device-property query.  Returns an fff_status. */
int fff_describe(const fff_args* a, char* buf, size_t len);

/* One layer of a stack: device pointers to its weights ([n_trees, N, hidden]
 * each, the same layout as fff_args) and, with FFF_NORM_LAYERNORM, its
 * LayerNorm gain and shift (fp32 [hidden], NULL for ones / zeros). */
typedef struct {
    const void* W_in;
    const void* W_out;
    const float* norm_gamma;
    const float* norm_beta;
} fff_layer;

/*
 * fff_forward_stack -- n_layers intermediate layers applied in sequence:
 *     x_0 = x,   x_{i+1} = x_i + FFF_i(norm_i(x_i)),   y = x_{n_layers},
 * each x_{i+1} rounded to the storage type (y_dtype) exactly as n_layers
 * chained fff_forward_ex calls with FFF_OUT_RESIDUAL would store it (a
 * stack of the Section 2.1 layers; tokens are independent, so the whole stack
 * can run per token).  With mode DESCENT one persistent kernel keeps each
 * token's x_i in registers through all layers (x read once, y written once;
 * the result equals the chained calls bit for bit); AUTO, GROUPED and GENERIC
 * run the layers as separate launches of that mode's single-layer plan, in
 * place on y (AUTO: measured faster for most stacks on MI355X).
 *
 *   a        : shapes, dtypes, act, mode, norm, norm_eps, records, workspace
 *              and stream as for fff_forward_ex, with these rules:
 *              out_mode must be FFF_OUT_RESIDUAL; x_dtype == y_dtype; x and y
 *              are the same buffer or disjoint; W_in, W_out, norm_gamma and
 *              norm_beta must be NULL (they come from layers[]); nodes_out and
 *              logits_out, when set, are [n_layers, n_tokens, n_trees, depth+1].
 *   layers   : HOST array of n_layers descriptors (read during the call only).
 *   n_layers : >= 1.
 * Returns an fff_status.  On FFF_ERR_HIP some layers may have been enqueued.
 */
int fff_forward_stack(const fff_args* a, const fff_layer* layers, int32_t n_layers);

/*
 * fff_backward -- gradients of one layer with the routing held fixed (hard
 * routing: the branch decisions are not differentiable, so gradients flow
 * through the D+1 visited nodes of every (token, tree) only; the training
 * method that learns the routing is the original FFF paper's, cited in
 * Section 2).  With the forward's leaves (path) and logits l, a = act(l),
 * and dy = dLoss/dFFF(x):
 *     dW_out[t,n] += a  * dy_b          for every visited node n
 *     dl           = <dy_b, W_out[t,n]> * act'(l)
 *     dW_in[t,n]  += dl * x_b
 *     dx_b        += dl * W_in[t,n]
 * (x is the FFF input; a residual or a LayerNorm around the layer is the
 * caller's to differentiate).
 *
 * Work: a stable counting sort of the tokens by leaf (every node's tokens
 * form one run at every level, in token order within a leaf).  With bf16
 * weights, one tree, depth <= 15 and hidden 128..1024, one fused kernel then
 * takes each leaf's tokens sixteen at a time through the whole backward on
 * MFMA (da, a and dl, dx, the dW sums of the leaf's path), followed by a
 * fix-up of the rows above its subtrees.  Otherwise a token kernel forms dx
 * and the per-visit pairs (a, dl) first, and the weight sums run along the
 * sorted order: for depth <= 15 and hidden a multiple of 128 on MFMA, one workgroup
 * per subtree accumulating the rows of its tokens' paths, with the rows above
 * the subtrees added in subtree order by a fix-up; otherwise by fixed pieces
 * of the sorted order summed in registers and a fix-up of the runs crossing
 * pieces.  No atomics on dx or dW and every sum in a fixed order: the results
 * are the same bits on every run.
 */
typedef struct {
    const void* x;          /* [n_tokens, hidden] the layer's FFF input (x_dtype) */
    const void* W_in;       /* [n_trees, N, hidden] (w_dtype) */
    const void* W_out;
    const void* dy;         /* [n_tokens, hidden] upstream gradient (dy_dtype) */
    const int32_t* leaves;  /* [n_tokens, n_trees] leaf node reached: the forward's nodes_out[..., depth] */
    const float* logits;    /* [n_tokens, n_trees, depth+1] the forward's logits_out */
    void* dx;               /* [n_tokens, hidden] (dx_dtype), or NULL to skip */
    float* dW_in;           /* [n_trees, N, hidden] fp32, or NULL to skip */
    float* dW_out;          /* [n_trees, N, hidden] fp32, or NULL to skip */
    int64_t n_tokens;
    int32_t hidden;         /* a multiple of 4 */
    int32_t depth;
    int32_t n_trees;
    int32_t x_dtype, w_dtype, dy_dtype, dx_dtype; /* fff_dtype */
    int32_t act;            /* fff_act of the forward */
    int32_t accumulate;     /* 0: dx, dW_in, dW_out overwritten (untouched dW rows become 0); 1: added to */
    int32_t* bad_leaves;    /* optional device int32: incremented once per (token, tree) whose leaf is
                               outside [2^depth - 1, 2^(depth+1) - 2]; such pairs contribute nothing */
    void* workspace;        /* device scratch of fff_backward_workspace_bytes(), 256-byte aligned,
                               disjoint from every other buffer */
    size_t workspace_bytes;
    void* hip_stream;
} fff_backward_args;

/* Every pointer is a caller-owned device pointer, 16-byte aligned (leaves,
 * logits and bad_leaves 4-byte aligned); outputs overlap no input and no other
 * output.  Validation runs before any HIP call; FFF_ERR_WORKSPACE when the
 * workspace is missing or small.  Returns an fff_status. */
int fff_backward(const fff_backward_args* a);

/* Workspace fff_backward needs: per-visit pairs (8 bytes each), two int32
 * arrays of 2^depth leaf bins per tree, one int32 token index per (token,
 * tree), per-tree totals, and fp32 run sums (two slots of both matrices'
 * rows per level and piece).  0 for invalid shapes. */
size_t fff_backward_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t hidden);

/* fff_describe for a stack. */
int fff_describe_stack(const fff_args* a, const fff_layer* layers, int32_t n_layers, char* buf, size_t len);

const char* fff_status_str(int status);
int fff_last_hip_error(void); /* raw hipError_t behind the calling thread's last FFF_ERR_HIP */
int fff_version(void);

#ifdef __cplusplus
}
#endif

#endif /* FFF_H_ */
