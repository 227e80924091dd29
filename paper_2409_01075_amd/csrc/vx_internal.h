// Host-side internals shared by the ABI, the selector and the generated registry.
#pragma once
#include <hip/hip_runtime_api.h>

#include "vx.h"
#include "vx_args.h"

typedef hipError_t (*vx_launch_fn)(const VxGemmArgs* args, int64_t grid, hipStream_t stream);

struct VxKernelEntry {
    vx_kernel_info info;
    vx_launch_fn launch;
};

// The generated registry (one entry per compiled workgroup-level candidate).
const VxKernelEntry* vxi_registry(int* count);

// Device description from hipDeviceProp_t plus the per-architecture table.
// Returns 0 on success.
int vxi_device_hwinfo(int device, vx_hwinfo* out);

// Shape and alignment facts of one call, as the selector sees them.
struct VxShape {
    int64_t batch, M, N, K;
    int dt;        // vx_dtype
    int vec_ok;    // operands allow 16-byte vector loads
    int c_vec;     // C allows 4-element vector stores
};

struct VxLimits {
    size_t ws_bytes;        // split-K partials capacity
    int64_t max_tickets;    // arrival counters available
};

// Cost (ns) of kernel k with split s on shape sh; < 0 if infeasible.  On
// success also returns the K extent per slice.
double vxi_cost(const vx_hwinfo& hw, const VxShape& sh, const vx_kernel_info& k, int split,
                const VxLimits& lim, int* k_per_split);

// Argmin over the registry (Equation 1).  forced_id >= 0 restricts the search
// to that kernel; forced_split > 0 to that split.  Returns VX_OK or
// VX_ERR_NO_CANDIDATE.
vx_status vxi_select(const vx_hwinfo& hw, const VxShape& sh, const VxLimits& lim, int forced_id,
                     int forced_split, vx_plan* out);

// grid-level tile order: tile rows walked together (bounded by the tile count)
int vxi_group_m(int64_t tiles_m, int64_t tiles_n);
