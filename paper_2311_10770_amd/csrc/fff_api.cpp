// fff_api.cpp -- the C ABI declared in include/fff.h: argument validation
// (entirely on the host, before any HIP call), a per-device property cache,
// and dispatch to the kernels planned in fff_kernels.hip.
#include "fff.h"

#include <hip/hip_runtime_api.h>

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
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + uintptr_t(bbytes) && b0 < a0 + uintptr_t(abytes);
}

// Full validation; fills the kernel parameter block.  No HIP calls.
int validate(const fff_args* a, fff::Params* p) {
    if (!a) return FFF_ERR_INVALID_ARG;
    if (a->n_tokens < 0 || a->hidden < 1 || a->depth < 0 || a->depth > kMaxDepth || a->n_trees < 1)
        return FFF_ERR_INVALID_ARG;
    for (int dt : {a->x_dtype, a->w_dtype, a->y_dtype})
        if (dt != FFF_F32 && dt != FFF_BF16) return FFF_ERR_INVALID_ARG;
    if (a->act < FFF_ACT_GELU_ERF || a->act > FFF_ACT_IDENTITY) return FFF_ERR_INVALID_ARG;
    if (a->mode < FFF_MODE_AUTO || a->mode > FFF_MODE_GENERIC) return FFF_ERR_INVALID_ARG;
    if (a->out_mode < FFF_OUT_STORE || a->out_mode > FFF_OUT_RESIDUAL) return FFF_ERR_INVALID_ARG;
    if (a->lds_levels < -1 || a->lds_levels > kMaxDepth + 1) return FFF_ERR_INVALID_ARG;
    if (a->split_level < -1 || a->split_level > a->depth) return FFF_ERR_INVALID_ARG;

    const int64_t sx = a->x_dtype == FFF_BF16 ? 2 : 4;
    const int64_t sw = a->w_dtype == FFF_BF16 ? 2 : 4;
    const int64_t sy = a->y_dtype == FFF_BF16 ? 2 : 4;
    const int64_t nodes = (int64_t(1) << (a->depth + 1)) - 1;
    int64_t act_elems = 0, w_rows = 0, w_elems = 0, rec = 0, tmp = 0;
    if (!mul_ok(a->n_tokens, a->hidden, &act_elems) || !mul_ok(act_elems, 4, &tmp)) return FFF_ERR_INVALID_ARG;
    if (!mul_ok(nodes, a->n_trees, &w_rows) || !mul_ok(w_rows, a->hidden, &w_elems) || !mul_ok(w_elems, 4, &tmp))
        return FFF_ERR_INVALID_ARG;
    if (!mul_ok(a->n_tokens, int64_t(a->n_trees) * (a->depth + 1), &rec) || !mul_ok(rec, 4, &tmp))
        return FFF_ERR_INVALID_ARG;
    if (w_rows > INT32_MAX) return FFF_ERR_INVALID_ARG;

    if (a->n_tokens > 0) {
        if (!a->x || !a->W_in || !a->W_out || !a->y) return FFF_ERR_INVALID_ARG;
        if (!aligned16(a->x) || !aligned16(a->W_in) || !aligned16(a->W_out) || !aligned16(a->y))
            return FFF_ERR_INVALID_ARG;
        if (a->nodes_out && !aligned16(a->nodes_out)) return FFF_ERR_INVALID_ARG;
        if (a->logits_out && !aligned16(a->logits_out)) return FFF_ERR_INVALID_ARG;
        if (overlap(a->x, act_elems * sx, a->y, act_elems * sy)) return FFF_ERR_INVALID_ARG;
        if (a->nodes_out && overlap(a->nodes_out, rec * 4, a->y, act_elems * sy)) return FFF_ERR_INVALID_ARG;
        if (a->logits_out && overlap(a->logits_out, rec * 4, a->y, act_elems * sy)) return FFF_ERR_INVALID_ARG;
        if (a->nodes_out && a->logits_out && overlap(a->nodes_out, rec * 4, a->logits_out, rec * 4))
            return FFF_ERR_INVALID_ARG;
    }
    (void)sw;

    *p = fff::Params{};
    p->x = a->x;
    p->w_in = a->W_in;
    p->w_out = a->W_out;
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
    return FFF_OK;
}

// Workspace checks for a grouped plan: present, big enough, 256-byte aligned,
// and disjoint from every tensor the kernels read or write.
int check_workspace(const fff_args* a) {
    const size_t need = fff::grouped_workspace_bytes(a->n_tokens, a->depth, a->n_trees, 0);
    if (!a->workspace || a->workspace_bytes < need || (reinterpret_cast<uintptr_t>(a->workspace) & 255u))
        return FFF_ERR_WORKSPACE;
    const int64_t wsb = int64_t(need);
    const int64_t act = a->n_tokens * a->hidden;
    const int64_t rec = a->n_tokens * a->n_trees * (a->depth + 1) * 4;
    const int64_t wbytes = ((int64_t(1) << (a->depth + 1)) - 1) * a->n_trees * a->hidden * (a->w_dtype ? 2 : 4);
    if (overlap(a->workspace, wsb, a->x, act * (a->x_dtype ? 2 : 4)) ||
        overlap(a->workspace, wsb, a->y, act * (a->y_dtype ? 2 : 4)) ||
        overlap(a->workspace, wsb, a->W_in, wbytes) || overlap(a->workspace, wsb, a->W_out, wbytes) ||
        (a->nodes_out && overlap(a->workspace, wsb, a->nodes_out, rec)) ||
        (a->logits_out && overlap(a->workspace, wsb, a->logits_out, rec)))
        return FFF_ERR_INVALID_ARG;
    return FFF_OK;
}

int plan_for(const fff_args* a, fff::Params* p, fff::Plan* plan) {
    int rc = validate(a, p);
    if (rc != FFF_OK) return rc;
    fff::DeviceInfo dev;
    rc = current_device_info(&dev);
    if (rc != FFF_OK) return rc;
    const size_t need = fff::grouped_workspace_bytes(a->n_tokens, a->depth, a->n_trees, 0);
    const bool have_ws = a->workspace && a->workspace_bytes >= need &&
                         (reinterpret_cast<uintptr_t>(a->workspace) & 255u) == 0;
    rc = fff::plan_forward(*p, a->mode, a->lds_levels, a->split_level, have_ws, dev, plan);
    if (rc != FFF_OK) return rc;
    if (plan->kind == fff::KIND_GROUPED && a->n_tokens > 0) return check_workspace(a);
    return FFF_OK;
}

}  // namespace

FFF_EXPORT int fff_forward_ex(const fff_args* a) {
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
    return fff::grouped_workspace_bytes(n_tokens, depth, n_trees, split_level);
}

FFF_EXPORT int fff_describe(const fff_args* a, char* buf, size_t len) {
    fff::Params p;
    fff::Plan plan;
    const int rc = plan_for(a, &p, &plan);
    if (rc != FFF_OK) return rc;
    if (buf && len) {
        static const char* kinds[] = {"none", "descent", "generic", "grouped"};
        int n = std::snprintf(buf, len, "%s<%s> lanes_per_token=%d lds_levels=%d", kinds[plan.kind], plan.name,
                              plan.lanes, plan.lds_levels);
        if (plan.kind == fff::KIND_GROUPED && n > 0 && size_t(n) < len)
            n += std::snprintf(buf + n, len - n, " emit_lds_levels=%d split_level=%d", plan.emit_lds_levels,
                               plan.split_level);
        for (int i = 0; i < plan.n_launch && n > 0 && size_t(n) < len; ++i)
            n += std::snprintf(buf + n, len - n, " | launch%d grid=%d block=%d lds_bytes=%zu", i,
                               plan.launch[i].grid, plan.launch[i].block, plan.launch[i].lds_bytes);
    }
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
