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
    const int32_t* perm;  // optional token order (grouped mode); nullptr = identity
    int64_t n_tokens;
    int64_t n_nodes;      // per tree: 2^(D+1) - 1
    int32_t hidden;
    int32_t depth;
    int32_t n_trees;
    int32_t x_bf16, w_bf16, y_bf16;
    int32_t act;
    int32_t out_mode;
    int32_t lds_levels;   // levels staged in LDS (descent kernel)
};

struct DeviceInfo {
    int device = -1;
    int cu_count = 0;
    size_t lds_per_block = 0;  // bytes
    size_t lds_per_cu = 0;     // bytes
};

enum KernelKind { KIND_NONE = 0, KIND_DESCENT = 1, KIND_GENERIC = 2, KIND_GROUPED = 3 };

struct Plan {
    int kind = KIND_NONE;
    const void* kernel = nullptr;  // __global__ function handle
    int lanes = 0;                 // lanes per token
    int block = 0;                 // threads per block
    int grid = 0;                  // blocks
    int lds_levels = 0;
    size_t lds_bytes = 0;          // dynamic LDS per block
    int split_level = 0;           // grouped mode
    const char* name = "";
};

// Fills *plan for a validated request; returns an fff_status value.
int plan_forward(const Params& p, int mode, int lds_levels_req, int split_level_req, const DeviceInfo& dev,
                 Plan* plan);

// Enqueues the planned work on stream; returns the first failing HIP error.
hipError_t run_forward(const Params& p, const Plan& plan, void* workspace, size_t workspace_bytes,
                       hipStream_t stream);

// Grouped mode scratch size (0 = not applicable).
size_t grouped_workspace_bytes(int64_t n_tokens, int32_t depth, int32_t n_trees, int32_t split_level);

}  // namespace fff
