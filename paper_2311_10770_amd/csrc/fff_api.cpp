// fff_api.cpp -- the C ABI declared in include/fff.h: argument validation
// (entirely on the host, before any HIP call), a per-device property cache,
// and dispatch to the kernels planned in fff_kernels.hip.
#include "fff.h"

#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "fff_internal.hpp"

#define FFF_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

thread_local int g_last_hip_error = 0;

constexpr int kMaxDepth = 24;
constexpr int kMaxDevices = 64;

int hip_fail(hipError_t e) {
    g_last_hip_error = int(e);
    return FFF_ERR_HIP;
}

struct DeviceCache {
    std::once_flag once[kMaxDevices];
    fff::DeviceInfo info[kMaxDevices];
    hipError_t err[kMaxDevices] = {};
};

DeviceCache& device_cache() {
    static DeviceCache c;
    return c;
}

// Properties of the current device, queried once per device.
int current_device_info(fff::DeviceInfo* out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e);
    if (dev < 0 || dev >= kMaxDevices) return FFF_ERR_UNSUPPORTED;
    DeviceCache& c = device_cache();
    std::call_once(c.once[dev], [&] {
        hipDeviceProp_t prop;
        hipError_t pe = hipGetDeviceProperties(&prop, dev);
        if (pe != hipSuccess) {
            c.err[dev] = pe;
            return;
        }
        fff::DeviceInfo& d = c.info[dev];
        d.device = dev;
        d.cu_count = prop.multiProcessorCount;
        d.lds_per_block = prop.sharedMemPerBlock;
        d.lds_per_cu = prop.maxSharedMemoryPerMultiProcessor;
    });
    if (c.err[dev] != hipSuccess) return hip_fail(c.err[dev]);
    *out = c.info[dev];
    return FFF_OK;
}

bool mul_ok(int64_t a, int64_t b, int64_t* out) {
    if (a < 0 || b < 0) return false;
    if (a != 0 && b > INT64_MAX / a) return false;
    *out = a * b;
    return true;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool overlap(const void* a, int64_t abytes, const void* b, int64_t bbytes) {
    if (!a || !b) return false;
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + uintptr_t(bbytes) && b0 < a0 + uintptr_t(abytes);
}

struct Span {
    const void* ptr;
    int64_t bytes;
};

// Everything a call reads and writes, for the overlap rules.
struct Buffers {
    Span x, y, nodes, logits;
    Span weights[2 * fff::STACK_MAX_LAYERS * 4];  // W_in, W_out, gamma, beta of every layer (read only)
    int n_weights = 0;
};

// Outputs must not overlap each other nor any input, except that y may be x
// itself (in place, same dtype).
bool overlaps_ok(const Buffers& b, bool same_dtype) {
    const Span outs[] = {b.y, b.nodes, b.logits};
    for (int i = 0; i < 3; ++i) {
        const Span& o = outs[i];
        if (!o.ptr) continue;
        for (int j = i + 1; j < 3; ++j)
            if (overlap(o.ptr, o.bytes, outs[j].ptr, outs[j].bytes)) return false;
        const bool in_place = i == 0 && o.ptr == b.x.ptr && same_dtype;
        if (!in_place && overlap(o.ptr, o.bytes, b.x.ptr, b.x.bytes)) return false;
        for (int k = 0; k < b.n_weights; ++k)
            if (overlap(o.ptr, o.bytes, b.weights[k].ptr, b.weights[k].bytes)) return false;
    }
    return true;
}

// Checks shared by the single-layer and stack entry points: sizes, enums and
// the norm fields.  Fills the kernel parameter block (without weights).  No
// HIP calls.
int validate_shapes(const fff_args* a, int64_t rec_layers, fff::Params* p, int64_t* rec_bytes) {
    if (!a) return FFF_ERR_INVALID_ARG;
    if (a->n_tokens < 0 || a->hidden < 1 || a->depth < 0 || a->depth > kMaxDepth || a->n_trees < 1)
        return FFF_ERR_INVALID_ARG;
    for (int dt : {a->x_dtype, a->w_dtype, a->y_dtype})
        if (dt != FFF_F32 && dt != FFF_BF16) return FFF_ERR_INVALID_ARG;
    if (a->act < FFF_ACT_GELU_ERF || a->act > FFF_ACT_IDENTITY) return FFF_ERR_INVALID_ARG;
    if (a->mode < FFF_MODE_AUTO || a->mode > FFF_MODE_SUBTREE) return FFF_ERR_INVALID_ARG;
    if (a->out_mode < FFF_OUT_STORE || a->out_mode > FFF_OUT_RESIDUAL) return FFF_ERR_INVALID_ARG;
    if (a->lds_levels < -1 || a->lds_levels > kMaxDepth + 1) return FFF_ERR_INVALID_ARG;
    if (a->split_level < -1 || a->split_level > a->depth) return FFF_ERR_INVALID_ARG;
    if (a->norm != FFF_NORM_NONE && a->norm != FFF_NORM_LAYERNORM) return FFF_ERR_INVALID_ARG;
    if (a->norm == FFF_NORM_LAYERNORM && !(a->norm_eps >= 0.0f && a->norm_eps <= 3.0e38f)) return FFF_ERR_INVALID_ARG;

    const int64_t nodes = (int64_t(1) << (a->depth + 1)) - 1;
    int64_t act_elems = 0, w_rows = 0, w_elems = 0, rec = 0, tmp = 0;
    if (!mul_ok(a->n_tokens, a->hidden, &act_elems) || !mul_ok(act_elems, 4, &tmp)) return FFF_ERR_INVALID_ARG;
    if (!mul_ok(nodes, a->n_trees, &w_rows) || !mul_ok(w_rows, a->hidden, &w_elems) || !mul_ok(w_elems, 4, &tmp))
        return FFF_ERR_INVALID_ARG;
    if (!mul_ok(a->n_tokens, int64_t(a->n_trees) * (a->depth + 1), &rec) || !mul_ok(rec, 4 * rec_layers, &tmp))
        return FFF_ERR_INVALID_ARG;
    if (w_rows > INT32_MAX) return FFF_ERR_INVALID_ARG;
    *rec_bytes = tmp;

    *p = fff::Params{};
    p->x = a->x;
    p->y = a->y;
    p->nodes_out = a->nodes_out;
    p->logits_out = a->logits_out;
    p->n_tokens = a->n_tokens;
    p->n_nodes = nodes;
    p->hidden = a->hidden;
    p->depth = a->depth;
    p->n_trees = a->n_trees;
    p->x_bf16 = a->x_dtype == FFF_BF16;
    p->w_bf16 = a->w_dtype == FFF_BF16;
    p->y_bf16 = a->y_dtype == FFF_BF16;
    p->act = a->act;
    p->out_mode = a->out_mode;
    p->lds_levels = 0;
    p->norm = a->norm;
    p->norm_eps = a->norm_eps;
    return FFF_OK;
}

// Pointer rules for one call: present, aligned, and the overlap rules over the
// given layers' weights.  Only when n_tokens > 0.
int validate_pointers(const fff_args* a, const fff_layer* layers, int n_layers, int64_t rec_bytes) {
    if (a->n_tokens == 0) return FFF_OK;
    const int64_t act = a->n_tokens * a->hidden;
    const int64_t wbytes =
        ((int64_t(1) << (a->depth + 1)) - 1) * a->n_trees * a->hidden * (a->w_dtype == FFF_BF16 ? 2 : 4);
    const int64_t nbytes = int64_t(a->hidden) * 4;
    if (!a->x || !a->y || !aligned16(a->x) || !aligned16(a->y)) return FFF_ERR_INVALID_ARG;
    if (a->nodes_out && !aligned16(a->nodes_out)) return FFF_ERR_INVALID_ARG;
    if (a->logits_out && !aligned16(a->logits_out)) return FFF_ERR_INVALID_ARG;
    Buffers b;
    b.x = {a->x, act * (a->x_dtype == FFF_BF16 ? 2 : 4)};
    b.y = {a->y, act * (a->y_dtype == FFF_BF16 ? 2 : 4)};
    b.nodes = {a->nodes_out, rec_bytes};
    b.logits = {a->logits_out, rec_bytes};
    for (int i = 0; i < n_layers; ++i) {
        const fff_layer& L = layers[i];
        if (!L.W_in || !L.W_out || !aligned16(L.W_in) || !aligned16(L.W_out)) return FFF_ERR_INVALID_ARG;
        const bool norm = a->norm == FFF_NORM_LAYERNORM;
        if (norm && ((L.norm_gamma && !aligned16(L.norm_gamma)) || (L.norm_beta && !aligned16(L.norm_beta))))
            return FFF_ERR_INVALID_ARG;
        if (b.n_weights + 4 > int(sizeof b.weights / sizeof b.weights[0])) return FFF_ERR_INVALID_ARG;
        b.weights[b.n_weights++] = {L.W_in, wbytes};
        b.weights[b.n_weights++] = {L.W_out, wbytes};
        if (norm) {
            b.weights[b.n_weights++] = {L.norm_gamma, nbytes};
            b.weights[b.n_weights++] = {L.norm_beta, nbytes};
        }
    }
    if (!overlaps_ok(b, a->x_dtype == a->y_dtype)) return FFF_ERR_INVALID_ARG;
    return FFF_OK;
}

// Full validation of a single-layer call; fills the kernel parameter block.
int validate(const fff_args* a, fff::Params* p) {
    int64_t rec_bytes = 0;
    int rc = validate_shapes(a, 1, p, &rec_bytes);
    if (rc != FFF_OK) return rc;
    const fff_layer L = {a->W_in, a->W_out, a->norm_gamma, a->norm_beta};
    rc = validate_pointers(a, &L, 1, rec_bytes);
    if (rc != FFF_OK) return rc;
    p->w_in = a->W_in;
    p->w_out = a->W_out;
    if (a->norm == FFF_NORM_LAYERNORM) {
        p->gamma = a->norm_gamma;
        p->beta = a->norm_beta;
    }
    return FFF_OK;
}

// Workspace checks for a grouped plan: present, big enough, 256-byte aligned,
// and disjoint from every tensor the kernels read or write.
int check_workspace(const fff_args* a, int kind) {
    const size_t need = kind == fff::KIND_TILED  ? fff::tiled_workspace_bytes(a->n_tokens, a->depth, a->n_trees, a->hidden)
                        : kind == fff::KIND_MASKED ? fff::masked_workspace_bytes(a->n_tokens, a->depth, a->n_trees, a->hidden)
                                                   : fff::grouped_workspace_bytes(a->n_tokens, a->depth, a->n_trees, 0);
    if (!a->workspace || a->workspace_bytes < need || (reinterpret_cast<uintptr_t>(a->workspace) & 255u))
        return FFF_ERR_WORKSPACE;
    const int64_t wsb = int64_t(need);
    const int64_t act = a->n_tokens * a->hidden;
    const int64_t rec = a->n_tokens * a->n_trees * (a->depth + 1) * 4;
    const int64_t wbytes = ((int64_t(1) << (a->depth + 1)) - 1) * a->n_trees * a->hidden * (a->w_dtype ? 2 : 4);
    const int64_t nbytes = int64_t(a->hidden) * 4;
    if (overlap(a->workspace, wsb, a->x, act * (a->x_dtype ? 2 : 4)) ||
        overlap(a->workspace, wsb, a->y, act * (a->y_dtype ? 2 : 4)) ||
        overlap(a->workspace, wsb, a->W_in, wbytes) || overlap(a->workspace, wsb, a->W_out, wbytes) ||
        overlap(a->workspace, wsb, a->nodes_out, rec) || overlap(a->workspace, wsb, a->logits_out, rec) ||
        (a->norm && (overlap(a->workspace, wsb, a->norm_gamma, nbytes) ||
                     overlap(a->workspace, wsb, a->norm_beta, nbytes))))
        return FFF_ERR_INVALID_ARG;
    return FFF_OK;
}

int plan_for(const fff_args* a, fff::Params* p, fff::Plan* plan) {
    int rc = validate(a, p);
    if (rc != FFF_OK) return rc;
    fff::DeviceInfo dev;
    rc = current_device_info(&dev);
    if (rc != FFF_OK) return rc;
    const size_t ws = a->workspace && (reinterpret_cast<uintptr_t>(a->workspace) & 255u) == 0 ? a->workspace_bytes : 0;
    rc = fff::plan_forward(*p, a->mode, a->lds_levels, a->split_level, ws, dev, plan);
    if (rc != FFF_OK) return rc;
    if ((plan->kind == fff::KIND_GROUPED || plan->kind == fff::KIND_TILED || plan->kind == fff::KIND_MASKED) &&
        a->n_tokens > 0)
        return check_workspace(a, plan->kind);
    return FFF_OK;
}

// The entry point that allocates nothing: the plan's scratch is the library's
// static device array.  No MASKED plan (its workspace is far larger than the array);
// AUTO picks a scratch-using mode only when the array covers it.
int forward_static(const fff_args* a) {
    fff::Params p;
    int rc = validate(a, &p);
    if (rc != FFF_OK) return rc;
    if (a->workspace || a->workspace_bytes) return FFF_ERR_INVALID_ARG;
    if (a->n_tokens == 0) return FFF_OK;
    fff::DeviceInfo dev;
    rc = current_device_info(&dev);
    if (rc != FFF_OK) return rc;
    fff::Plan plan;
    rc = fff::plan_forward(p, a->mode, a->lds_levels, a->split_level, fff::STATIC_SCRATCH_BYTES, dev, &plan, false);
    if (rc != FFF_OK) return rc;
    size_t need = 0;
    if (plan.kind == fff::KIND_TILED) need = fff::tiled_workspace_bytes(a->n_tokens, a->depth, a->n_trees, a->hidden);
    else if (plan.kind == fff::KIND_GROUPED) need = fff::grouped_workspace_bytes(a->n_tokens, a->depth, a->n_trees, 0);
    if (need > fff::STATIC_SCRATCH_BYTES) return FFF_ERR_WORKSPACE;
    void* ws = nullptr;
    if (need) {
        const hipError_t e = fff::static_scratch(dev.device, &ws);
        if (e != hipSuccess) return hip_fail(e);
    }
    const hipError_t e =
        fff::run_forward(p, plan, ws, fff::STATIC_SCRATCH_BYTES, reinterpret_cast<hipStream_t>(a->hip_stream));
    if (e != hipSuccess) return hip_fail(e);
    return FFF_OK;
}

int forward_one(const fff_args* a) {
    fff::Params p;
    {
        const int rc = validate(a, &p);
        if (rc != FFF_OK) return rc;
    }
    if (a->n_tokens == 0) return FFF_OK;
    fff::Plan plan;
    const int rc = plan_for(a, &p, &plan);
    if (rc != FFF_OK) return rc;
    const hipError_t e =
        fff::run_forward(p, plan, a->workspace, a->workspace_bytes, reinterpret_cast<hipStream_t>(a->hip_stream));
    if (e != hipSuccess) return hip_fail(e);
    return FFF_OK;
}

// ------------------------------------------------------------------ stacks

constexpr int kMaxStackLayers = 4096;

int validate_stack(const fff_args* a, const fff_layer* layers, int32_t n_layers, fff::Params* p) {
    if (!a || n_layers < 1 || n_layers > kMaxStackLayers || !layers) return FFF_ERR_INVALID_ARG;
    if (a->W_in || a->W_out || a->norm_gamma || a->norm_beta) return FFF_ERR_INVALID_ARG;
    if (a->out_mode != FFF_OUT_RESIDUAL || a->x_dtype != a->y_dtype) return FFF_ERR_INVALID_ARG;
    int64_t rec_bytes = 0;
    int rc = validate_shapes(a, n_layers, p, &rec_bytes);
    if (rc != FFF_OK) return rc;
    // overlap rules in windows of layers (the buffer table is bounded); every
    // window is checked against x, y and the records
    constexpr int kWindow = fff::STACK_MAX_LAYERS;
    for (int i0 = 0; i0 < n_layers; i0 += kWindow) {
        rc = validate_pointers(a, layers + i0, std::min(kWindow, n_layers - i0), rec_bytes);
        if (rc != FFF_OK) return rc;
    }
    return FFF_OK;
}

// DESCENT runs the stack in the persistent stack kernel; the other modes run
// one launch per layer.  AUTO takes the per-layer launches: measured on
// MI355X, the persistent kernel saves the re-reads of x but loses L2
// locality (its workgroups drift apart across layers, so several layers'
// rows compete for each XCD's L2), and it was slower for most stacks.
int plan_stack_for(const fff_args* a, const fff::Params& p, fff::Plan* plan, bool* use_kernel) {
    *use_kernel = false;
    if (a->mode != FFF_MODE_DESCENT) return FFF_OK;
    fff::DeviceInfo dev;
    int rc = current_device_info(&dev);
    if (rc != FFF_OK) return rc;
    rc = fff::plan_stack(p, a->lds_levels, dev, plan);
    if (rc == FFF_OK) *use_kernel = true;
    return rc;
}

// Single-layer arguments for layer i of a stack run as separate launches.
fff_args layer_args(const fff_args* a, const fff_layer* layers, int i) {
    fff_args b = *a;
    const int64_t rec = a->n_tokens * a->n_trees * (a->depth + 1);
    b.x = i == 0 ? a->x : a->y;
    b.W_in = layers[i].W_in;
    b.W_out = layers[i].W_out;
    b.norm_gamma = layers[i].norm_gamma;
    b.norm_beta = layers[i].norm_beta;
    b.nodes_out = a->nodes_out ? a->nodes_out + i * rec : nullptr;
    b.logits_out = a->logits_out ? a->logits_out + i * rec : nullptr;
    return b;
}

// ---------------------------------------------------------------- backward

bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

int validate_backward(const fff_backward_args* a, fff::BwdParams* p) {
    if (!a) return FFF_ERR_INVALID_ARG;
    if (a->n_tokens < 0 || a->hidden < 1 || a->hidden % 4 || a->depth < 0 || a->depth > kMaxDepth ||
        a->n_trees < 1)
        return FFF_ERR_INVALID_ARG;
    for (int dt : {a->x_dtype, a->w_dtype, a->dy_dtype, a->dx_dtype})
        if (dt != FFF_F32 && dt != FFF_BF16) return FFF_ERR_INVALID_ARG;
    if (a->act < FFF_ACT_GELU_ERF || a->act > FFF_ACT_IDENTITY) return FFF_ERR_INVALID_ARG;
    if (a->accumulate != 0 && a->accumulate != 1) return FFF_ERR_INVALID_ARG;
    const int64_t nodes = (int64_t(1) << (a->depth + 1)) - 1;
    int64_t act_elems = 0, w_rows = 0, w_elems = 0, pairs = 0, rec = 0, tmp = 0;
    if (!mul_ok(a->n_tokens, a->hidden, &act_elems) || !mul_ok(act_elems, 4, &tmp)) return FFF_ERR_INVALID_ARG;
    if (!mul_ok(nodes, a->n_trees, &w_rows) || !mul_ok(w_rows, a->hidden, &w_elems) || !mul_ok(w_elems, 4, &tmp))
        return FFF_ERR_INVALID_ARG;
    if (!mul_ok(a->n_tokens, a->n_trees, &pairs) || pairs > INT32_MAX) return FFF_ERR_INVALID_ARG;
    if (!mul_ok(pairs, a->depth + 1, &rec) || !mul_ok(rec, 8, &tmp)) return FFF_ERR_INVALID_ARG;
    if (w_rows > INT32_MAX) return FFF_ERR_INVALID_ARG;

    *p = fff::BwdParams{};
    if (a->n_tokens > 0) {
        const bool need_x = a->dW_in != nullptr;
        if (!a->W_in || !a->W_out || !a->dy || !a->leaves || !a->logits || (need_x && !a->x))
            return FFF_ERR_INVALID_ARG;
        for (const void* q : {a->x, a->W_in, a->W_out, a->dy, static_cast<const void*>(a->dx),
                              static_cast<const void*>(a->dW_in), static_cast<const void*>(a->dW_out)})
            if (q && !aligned16(q)) return FFF_ERR_INVALID_ARG;
        for (const void* q : {static_cast<const void*>(a->leaves), static_cast<const void*>(a->logits),
                              static_cast<const void*>(a->bad_leaves)})
            if (q && !aligned4(q)) return FFF_ERR_INVALID_ARG;
        const int64_t wbytes = w_elems * (a->w_dtype == FFF_BF16 ? 2 : 4);
        const Span ins[] = {{a->x, act_elems * (a->x_dtype == FFF_BF16 ? 2 : 4)},
                            {a->W_in, wbytes},
                            {a->W_out, wbytes},
                            {a->dy, act_elems * (a->dy_dtype == FFF_BF16 ? 2 : 4)},
                            {a->leaves, pairs * 4},
                            {a->logits, rec * 4}};
        const Span outs[] = {{a->dx, act_elems * (a->dx_dtype == FFF_BF16 ? 2 : 4)},
                             {a->dW_in, w_elems * 4},
                             {a->dW_out, w_elems * 4},
                             {a->bad_leaves, 4}};
        for (int i = 0; i < 4; ++i) {
            if (!outs[i].ptr) continue;
            for (const Span& in : ins)
                if (overlap(outs[i].ptr, outs[i].bytes, in.ptr, in.bytes)) return FFF_ERR_INVALID_ARG;
            for (int j = i + 1; j < 4; ++j)
                if (overlap(outs[i].ptr, outs[i].bytes, outs[j].ptr, outs[j].bytes)) return FFF_ERR_INVALID_ARG;
        }
        if (a->dW_in || a->dW_out) {
            const size_t need = fff::bwd_workspace_bytes(a->n_tokens, a->depth, a->n_trees, a->hidden);
            if (!a->workspace || a->workspace_bytes < need || (reinterpret_cast<uintptr_t>(a->workspace) & 255u))
                return FFF_ERR_WORKSPACE;
            for (const Span& q : ins)
                if (overlap(a->workspace, int64_t(need), q.ptr, q.bytes)) return FFF_ERR_INVALID_ARG;
            for (const Span& q : outs)
                if (overlap(a->workspace, int64_t(need), q.ptr, q.bytes)) return FFF_ERR_INVALID_ARG;
        }
    }
    p->x = a->x;
    p->w_in = a->W_in;
    p->w_out = a->W_out;
    p->dy = a->dy;
    p->leaves = a->leaves;
    p->logits = a->logits;
    p->dx = a->dx;
    p->dw_in = a->dW_in;
    p->dw_out = a->dW_out;
    p->bad = a->bad_leaves;
    p->n_tokens = a->n_tokens;
    p->n_nodes = nodes;
    p->hidden = a->hidden;
    p->depth = a->depth;
    p->n_trees = a->n_trees;
    p->x_bf16 = a->x_dtype == FFF_BF16;
    p->w_bf16 = a->w_dtype == FFF_BF16;
    p->dy_bf16 = a->dy_dtype == FFF_BF16;
    p->dx_bf16 = a->dx_dtype == FFF_BF16;
    p->act = a->act;
    p->accumulate = a->accumulate;
    p->need_dw = (a->dW_in || a->dW_out) ? 1 : 0;
    return FFF_OK;
}

}  // namespace

FFF_EXPORT int fff_forward_ex(const fff_args* a) { return forward_one(a); }

FFF_EXPORT int fff_forward_static(const fff_args* a) { return forward_static(a); }

FFF_EXPORT int fff_backward(const fff_backward_args* a) {
    fff::BwdParams p;
    int rc = validate_backward(a, &p);
    if (rc != FFF_OK) return rc;
    if (a->n_tokens == 0 || (!a->dx && !a->dW_in && !a->dW_out)) return FFF_OK;
    fff::DeviceInfo dev;
    rc = current_device_info(&dev);
    if (rc != FFF_OK) return rc;
    if (p.need_dw) fff::bwd_workspace_views(p, a->workspace);
    int status = FFF_OK;
    const hipError_t e = fff::run_backward(p, dev, reinterpret_cast<hipStream_t>(a->hip_stream), &status);
    if (status != FFF_OK) return status;
    if (e != hipSuccess) return hip_fail(e);
    return FFF_OK;
}

FFF_EXPORT size_t fff_backward_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t hidden) {
    if (n_tokens < 0 || depth < 0 || depth > kMaxDepth || n_trees < 1 || hidden < 1) return 0;
    return fff::bwd_workspace_bytes(n_tokens, depth, n_trees, hidden);
}

FFF_EXPORT int fff_forward_stack(const fff_args* a, const fff_layer* layers, int32_t n_layers) {
    fff::Params p;
    int rc = validate_stack(a, layers, n_layers, &p);
    if (rc != FFF_OK) return rc;
    if (a->n_tokens == 0) return FFF_OK;
    fff::Plan plan;
    bool use_kernel = false;
    rc = plan_stack_for(a, p, &plan, &use_kernel);
    if (rc != FFF_OK) return rc;
    if (!use_kernel) {
        for (int i = 0; i < n_layers; ++i) {
            const fff_args b = layer_args(a, layers, i);
            rc = forward_one(&b);
            if (rc != FFF_OK) return rc;
        }
        return FFF_OK;
    }
    const int64_t rec = a->n_tokens * a->n_trees * (a->depth + 1);
    fff::StackParams sp;
    std::memset(&sp, 0, sizeof sp);
    sp.rec_stride = rec;
    for (int i0 = 0; i0 < n_layers; i0 += fff::STACK_MAX_LAYERS) {
        sp.p = p;
        sp.p.x = i0 == 0 ? a->x : a->y;
        sp.p.nodes_out = a->nodes_out ? a->nodes_out + i0 * rec : nullptr;
        sp.p.logits_out = a->logits_out ? a->logits_out + i0 * rec : nullptr;
        sp.n_layers = std::min(fff::STACK_MAX_LAYERS, n_layers - i0);
        for (int j = 0; j < sp.n_layers; ++j) {
            const fff_layer& L = layers[i0 + j];
            const bool norm = a->norm == FFF_NORM_LAYERNORM;
            sp.layer[j] = {L.W_in, L.W_out, norm ? L.norm_gamma : nullptr, norm ? L.norm_beta : nullptr};
        }
        const hipError_t e = fff::run_stack(sp, plan, reinterpret_cast<hipStream_t>(a->hip_stream));
        if (e != hipSuccess) return hip_fail(e);
    }
    return FFF_OK;
}

FFF_EXPORT int fff_forward(const void* x, const void* W_in, const void* W_out, int32_t depth, int32_t n_trees,
                           void* y, int64_t n_tokens, int32_t hidden, int32_t x_dtype, int32_t w_dtype,
                           int32_t y_dtype, void* hip_stream) {
    fff_args a;
    std::memset(&a, 0, sizeof a);
    a.x = x;
    a.W_in = W_in;
    a.W_out = W_out;
    a.y = y;
    a.depth = depth;
    a.n_trees = n_trees;
    a.n_tokens = n_tokens;
    a.hidden = hidden;
    a.x_dtype = x_dtype;
    a.w_dtype = w_dtype;
    a.y_dtype = y_dtype;
    a.hip_stream = hip_stream;
    return fff_forward_ex(&a);
}

FFF_EXPORT size_t fff_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t hidden,
                                      int32_t split_level) {
    if (n_tokens < 0 || depth < 0 || depth > kMaxDepth || n_trees < 1 || hidden < 1 || split_level < -1 ||
        split_level > depth)
        return 0;
    return std::max({fff::grouped_workspace_bytes(n_tokens, depth, n_trees, split_level),
                     fff::tiled_workspace_bytes(n_tokens, depth, n_trees, hidden),
                     fff::masked_workspace_bytes(n_tokens, depth, n_trees, hidden)});
}

namespace {
void format_plan(const fff::Plan& plan, const char* prefix, char* buf, size_t len) {
    if (!buf || !len) return;
    static const char* kinds[] = {"none", "descent", "generic", "grouped", "stack", "tiled", "masked", "subtree"};
    int n = std::snprintf(buf, len, "%s%s<%s> lanes_per_token=%d lds_levels=%d", prefix, kinds[plan.kind],
                          plan.name, plan.lanes, plan.lds_levels);
    if (plan.kind == fff::KIND_SUBTREE && n > 0 && size_t(n) < len)
        n += std::snprintf(buf + n, len - n, " levels_per_step=%d", plan.split_level);
    if ((plan.kind == fff::KIND_GROUPED || plan.kind == fff::KIND_TILED) && n > 0 && size_t(n) < len)
        n += std::snprintf(buf + n, len - n, " emit_lds_levels=%d split_level=%d emit_lanes=%d walk_tree_per_xcd=%d",
                           plan.emit_lds_levels, plan.split_level, plan.emit_lanes, plan.walk_affine);
    if (plan.kind == fff::KIND_TILED && n > 0 && size_t(n) < len)
        n += std::snprintf(buf + n, len - n, " leaf_pairs=%d", plan.tile_pair);
    for (int i = 0; i < plan.n_launch && n > 0 && size_t(n) < len; ++i)
        n += std::snprintf(buf + n, len - n, " | launch%d grid=%d block=%d lds_bytes=%zu", i, plan.launch[i].grid,
                           plan.launch[i].block, plan.launch[i].lds_bytes);
}
}  // namespace

FFF_EXPORT int fff_describe(const fff_args* a, char* buf, size_t len) {
    fff::Params p;
    fff::Plan plan;
    const int rc = plan_for(a, &p, &plan);
    if (rc != FFF_OK) return rc;
    format_plan(plan, "", buf, len);
    return FFF_OK;
}

FFF_EXPORT int fff_describe_stack(const fff_args* a, const fff_layer* layers, int32_t n_layers, char* buf,
                                  size_t len) {
    fff::Params p;
    int rc = validate_stack(a, layers, n_layers, &p);
    if (rc != FFF_OK) return rc;
    fff::Plan plan;
    bool use_kernel = false;
    rc = plan_stack_for(a, p, &plan, &use_kernel);
    if (rc != FFF_OK) return rc;
    if (use_kernel) {
        format_plan(plan, "", buf, len);
        return FFF_OK;
    }
    const fff_args b = layer_args(a, layers, 0);
    fff::Params pb;
    rc = plan_for(&b, &pb, &plan);
    if (rc != FFF_OK) return rc;
    format_plan(plan, "per-layer ", buf, len);
    return FFF_OK;
}

FFF_EXPORT const char* fff_status_str(int status) {
    switch (status) {
        case FFF_OK: return "FFF_OK";
        case FFF_ERR_INVALID_ARG: return "FFF_ERR_INVALID_ARG: invalid argument";
        case FFF_ERR_UNSUPPORTED: return "FFF_ERR_UNSUPPORTED: no kernel for this request";
        case FFF_ERR_WORKSPACE: return "FFF_ERR_WORKSPACE: workspace missing or too small";
        case FFF_ERR_HIP: return "FFF_ERR_HIP: a HIP runtime call failed";
        default: return "unknown fff status";
    }
}

FFF_EXPORT int fff_last_hip_error(void) { return g_last_hip_error; }

FFF_EXPORT int fff_version(void) { return FFF_VERSION; }
