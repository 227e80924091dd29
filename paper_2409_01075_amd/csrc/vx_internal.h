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
// Identifies the compiled kernel set (candidates + kernel sources).
const char* vxi_registry_hash(void);

// Offline per-kernel measurements (the empirical low levels of the hybrid
// analyzer): time of one workgroup K step and fixed per-call cost, with the
// whole device busy ("full") and at light load, all in ns.
struct VxCalib {
    double step_full, fix_full, step_light, fix_light, load_light;
    double split_a, split_b;   // split-K epilogue: split_a + split_b * (slices - 1); < 0 if not measured
    // convolution kernels that gather the image through VGPRs: one K step at
    // full and at light load when every image chunk is gathered element by
    // element; < 0 if not measured
    double step_gather, step_gather_light;
};
// Calibration of a kernel, or nullptr when none is loaded / it is disabled.
const VxCalib* vxi_calib(int kernel_id);
// Dispatch constant: the calibrated launch floor when loaded, else hw.launch_ns.
double vxi_calib_launch_ns(const vx_hwinfo& hw);

// Planning epoch: changes whenever a planning input does (calibration,
// hardware override, ablation switches, workspaces).
uint64_t vxi_plan_epoch(void);
// True while the search must price every (kernel, split) pair (a test switch).
bool vxi_exhaustive_search(void);

// Device description from hipDeviceProp_t plus the per-architecture table.
// Returns 0 on success.
int vxi_device_hwinfo(int device, vx_hwinfo* out);

// Shape and alignment facts of one call, as the selector sees them.
struct VxShape {
    int64_t batch, M, N, K;
    int dt;        // vx_dtype
    int vec_ok;    // rows allow 16-byte vector loads: bit 0 A's, bit 1 B's (3: both)
    int c_vec;     // C allows 4-element vector stores
    int op = 0;    // 0: GEMM; 1: 2-D convolution as an implicit GEMM (conv kernels only)
    int64_t a_bytes = 0;   // convolution: bytes of the image (the direct-to-LDS kernels need < 2^31)
    // convolution: the share of the image's 16-byte chunks that the kernels
    // gathering the image through VGPRs load element by element (0 when the
    // channels come in whole chunks)
    double gather_frac = 0.0;
};

struct VxLimits {
    size_t ws_bytes;        // split-K partials capacity
    int64_t max_tickets;    // arrival counters available
};

// Resident workgroups per CU of kernel k (tighter of LDS and register budgets).
int vxi_occupancy(const vx_hwinfo& hw, const vx_kernel_info& k);

// Cost (ns) of kernel k with split s on shape sh; < 0 if infeasible.  s < 0
// asks for the hybrid grid (whole waves of whole tiles, the remaining tiles
// split -s ways).  On success also returns the K extent per slice and the
// number of whole tiles (0 for a plain grid).
double vxi_cost(const vx_hwinfo& hw, const VxShape& sh, const vx_kernel_info& k, int split,
                const VxLimits& lim, int* k_per_split, int64_t* dp_tiles = nullptr);

// Restrictions of the search, for tests and the hierarchy ablations.
struct VxFilter {
    int kernel_id = -1;   // >= 0: only this kernel (a fixed workgroup and wavefront strategy)
    int split = 0;        // > 0: only this split-K factor; < 0: only the hybrid grid with split -split
    int wave_m = 0, wave_n = 0, mfma_m = 0;   // > 0: only kernels with this wavefront strategy
    int backends = 3;     // bit 0: matrix-core (MFMA) kernels, bit 1: vector-ALU kernels
    bool hybrid = true;   // the hybrid grid is among the plans considered
};

// True if kernel k passes the wavefront part of the filter.
bool vxi_wave_matches(const VxFilter& f, const vx_kernel_info& k);

// Argmin over the registry (Equation 1) among the kernels and splits the
// filter admits.  Returns VX_OK or VX_ERR_NO_CANDIDATE.
vx_status vxi_select(const vx_hwinfo& hw, const VxShape& sh, const VxLimits& lim, const VxFilter& f,
                     vx_plan* out);

// grid-level tile order: tile rows walked together (bounded by the tile count)
int vxi_group_m(int64_t tiles_m, int64_t tiles_n);

// The GEMM entry's argument checks alone (no HIP call); *noop when M, N or
// batch is 0.
vx_status vxi_gemm_check(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype, const void* A,
                         int64_t sA, const void* B, int64_t sB, void* C, int64_t sC, bool* noop);
// The batched GEMM with a caller-given split-K scratch (arrival counters at
// `scratch`, ticket_bytes of them, then partial_bytes of fp32 partials):
// plans only splits that fit, allocates nothing.
vx_status vxi_gemm_scratch(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype, const void* A,
                           int64_t sA, const void* B, int64_t sB, void* C, int64_t sC, void* stream,
                           void* scratch, size_t ticket_bytes, size_t partial_bytes);
