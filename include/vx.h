/*
 * vx — runtime-shaped dense GEMM for AMD MI355X (gfx950), C ABI.
 *
 * Operation (Section 4.1 of "Vortex: Efficient Sample-Free Dynamic Tensor
 * Program Optimization via Hardware-aware Strategy Space Hierarchization"):
 * C = A x B, where M, N and K are known only at call time (Section 2.2).
 *
 *   A  M x K, row-major, leading dimension K
 *   B  K x N, row-major, leading dimension N
 *   C  M x N, row-major, leading dimension N;   C := A x B  (no alpha/beta)
 *
 * A, B and C share one element type (fp32, fp16 or bf16).  Products are
 * accumulated in fp32 and the result is rounded to nearest-even into C's type.
 * Each call is served by one of the library's precompiled micro-kernels,
 * chosen by an analytical cost model of the kernel hierarchy (Section 5.2,
 * Equations 1-4) from the call's shape and the device's hardware description;
 * no profiling run and no shape sample is involved.
 *
 * Memory: every pointer argument of the GEMM calls is a DEVICE pointer owned
 * by the caller; the library neither retains nor frees it.  A stream argument
 * is a hipStream_t passed as void* (NULL = the default stream); the call only
 * enqueues work on it and returns.  Device-side faults surface at the
 * caller's next synchronisation of that stream.
 *
 * Errors: every function returns a vx_status; nothing throws or aborts.
 * Argument checks happen before any HIP call, so they also work on a host
 * without a GPU.
 *
 * Threads: all functions may be called concurrently.  Calls that select a
 * split-K plan share a per-(device, stream) workspace; calls on one stream
 * are ordered by the stream, so they never race.
 */
#ifndef VX_H
#define VX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { VX_F32 = 0, VX_F16 = 1, VX_BF16 = 2 } vx_dtype;

typedef enum {
    VX_OK = 0,
    VX_ERR_INVALID_ARG = 1,       /* negative size/stride, NULL operand with a non-empty extent,
                                     C overlapping A or B, overlapping C batches */
    VX_ERR_UNSUPPORTED_DTYPE = 2, /* dtype not one of vx_dtype */
    VX_ERR_NO_CANDIDATE = 3,      /* no compiled kernel fits (or a forced plan does not exist) */
    VX_ERR_WORKSPACE = 4,         /* the split-K workspace could not be provided */
    VX_ERR_HIP = 5                /* a HIP runtime call failed (no device, launch failure, ...) */
} vx_status;

/* Hardware description that drives candidate feasibility and the cost model
 * (the GetHardwareInfo step of Algorithm 2).  Filled from hipDeviceProp_t and
 * a per-architecture table. */
typedef struct vx_hwinfo {
    char arch[32];                 /* e.g. "gfx950" */
    int num_cu;                    /* compute units */
    int num_xcd;                   /* chiplets; workgroups are dispatched round-robin over them */
    int simd_per_cu;
    int wave_size;
    int max_threads_per_wg;
    int lds_bytes_per_cu;
    int vgprs_per_lane;            /* unified VGPR+AGPR file per lane of a SIMD */
    int max_waves_per_simd;
    double clock_ghz;              /* peak engine clock */
    double hbm_gbps;               /* peak HBM bandwidth, GB/s */
    double l2_bytes_per_xcd;
    double mall_bytes;             /* last-level (Infinity) cache */
    double mfma_flop_clk_cu_f16;   /* dense MFMA FLOP per clock per CU, fp16/bf16 inputs */
    double mfma_flop_clk_cu_f32;   /* dense MFMA FLOP per clock per CU, fp32 inputs */
    double l2_bytes_clk_cu;        /* L2 -> CU fill rate, bytes per clock */
    double lds_bytes_clk_cu;       /* LDS read bandwidth per CU, bytes per clock */
    double mem_latency_ns;         /* global load-to-use latency (HBM) */
    double atomic_latency_ns;      /* device-scope atomic round trip */
    double launch_ns;              /* fixed cost of one kernel dispatch */
} vx_hwinfo;

/* One micro-kernel of the registry (a workgroup-level candidate). */
typedef struct vx_kernel_info {
    int id;
    vx_dtype dtype;
    int mb, nb, kb;                /* workgroup tile */
    int wm, wn;                    /* wavefront grid; wavefront tile = (mb/wm) x (nb/wn) */
    int mfma_m, mfma_n, mfma_k;    /* instruction tile (0 for the vector-ALU family) */
    int vec;                       /* 1: needs 16-byte-aligned rows of A and B; 0: not both (see align) */
    int family;                    /* 0: MFMA, loads staged through registers; 1: MFMA, direct-to-LDS
                                      DMA; 2: vector ALU (v_dot2 / v_fma), B rows straight to VGPRs,
                                      for small M (mb = the rows one workgroup covers) */
    int stages;                    /* families 0, 1: LDS ring depth (K steps in flight + 1);
                                      family 2: K groups per lane per register set */
    int threads;
    int lds_bytes;
    int vgprs, agprs, sgprs;       /* from the compiler's resource report of this build */
    int scratch_bytes;             /* per lane; 0 for every enabled kernel */
    int enabled;
    int k_max;                     /* longest K slice one workgroup takes (0: unbounded); family 2
                                      keeps its slice of A in LDS */
    int op;                        /* 0: GEMM; 1: 2-D convolution (implicit GEMM: A is the input
                                      image read through the im2col map) */
    int align;                     /* rows that must start on 16-byte boundaries: bit 0 A's, bit 1
                                      B's (family 1 moves such an operand by DMA, the other through
                                      VGPRs) */
    int schedule;                  /* family 1, level-1 DMA issue: 0 every wave issues its share of
                                      each K step; 1 ping-pong (8 waves, 2 stages): the two halves
                                      of the waves take turns issuing whole K steps while the other
                                      half starts its MFMAs */
} vx_kernel_info;

/* A concrete execution plan for one call. */
typedef struct vx_plan {
    int kernel_id;
    int split_k;                   /* K slices reduced in fp32 by the last-arriving workgroup */
    int k_per_split;               /* K extent of one slice (a multiple of kb) */
    int c_vec;                     /* 1: C's rows are 4-element aligned (informational: full
                                      4-column chunks of C are stored as one vector either way) */
    int64_t tiles_m, tiles_n;
    int64_t grid;                  /* workgroups launched */
    int64_t dp_tiles;              /* hybrid grid (> 0): this many output tiles, whole waves of the
                                      device, run whole, one workgroup each, and only the others
                                      are split split_k ways; 0: every tile is split split_k ways */
    int group_m;
    size_t workspace_bytes;        /* fp32 partials needed by split_k > 1 */
    double predicted_ns;           /* the cost model's estimate for the call */
    vx_kernel_info kernel;
} vx_plan;

/*
 * C = A x B for one M x K by K x N product.
 * M, N, K >= 0.  M == 0 or N == 0 is a no-op; K == 0 writes C := 0.
 * A, B may be NULL only when their extent (M*K, K*N) is zero; C only when M*N is 0.
 */
vx_status vx_gemm(int64_t M, int64_t N, int64_t K, vx_dtype dtype,
                  const void* A, const void* B, void* C, void* stream);

/*
 * Batched form: for b in [0, batch): C_b = A_b x B_b with
 *   A_b = A + b*strideA, B_b = B + b*strideB, C_b = C + b*strideC   (strides in elements).
 * strideB == 0 (or strideA == 0) broadcasts that operand to every batch.
 * strideC must be >= M*N when batch > 1 (output batches may not overlap).
 */
vx_status vx_gemm_batched(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype,
                          const void* A, int64_t strideA, const void* B, int64_t strideB,
                          void* C, int64_t strideC, void* stream);

/*
 * vx_gemm_batched for callers that cannot allocate device memory: code under
 * HIP graph capture, serving loops and harnesses that forbid hipMalloc.  Same
 * arguments, semantics and errors as vx_gemm_batched; the caller still passes
 * A, B and C.  The split-K scratch (arrival counters and fp32 partial tiles)
 * is a static device array of 16 MiB + 64 KiB that each GPU the library runs
 * on holds until the process ends; no call allocates or frees anything.
 * Plans are chosen among those whose partials fit that array; a plan forced
 * with vx_force_plan that needs more returns VX_ERR_WORKSPACE.  The first call
 * on a device clears the array's counters with a small kernel on `stream`
 * (which a capture records like any kernel); afterwards they reset themselves.
 * Every call on one GPU shares that GPU's array, so calls that overlap in time
 * on one GPU (concurrent streams, or graph replays beside eager calls) race
 * and must be ordered by the caller.
 */
vx_status vx_gemm_batched_noalloc(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype,
                                  const void* A, int64_t strideA, const void* B, int64_t strideB,
                                  void* C, int64_t strideC, void* stream);

/*
 * The plan vx_gemm_batched would use, without launching anything (host only).
 * base_align: the largest power of two dividing the byte addresses of A, B
 * and C (0 means 256).  Strides as for vx_gemm_batched.
 */
vx_status vx_plan_query(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype,
                        int64_t strideA, int64_t strideB, int64_t strideC,
                        uint64_t base_align, vx_plan* out);

/*
 * The cost model's estimate (ns) for running a given kernel with a given
 * split-K factor on a shape; VX_ERR_NO_CANDIDATE if the pair is infeasible.
 * It is the selector's model: like a plan query, the first call loads the
 * shipped calibration table when it matches the compiled kernel set.
 * split_k < 0 prices the hybrid grid with -split_k slices per split tile.
 * align: which operands' rows start on 16-byte boundaries (bit 0 A, bit 1 B;
 * 3 both, 0 neither); VX_ERR_INVALID_ARG outside 0..3.
 */
vx_status vx_plan_cost(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype,
                       int kernel_id, int split_k, int align, double* out_ns);

/* Equation 2: T = t_load + (trips - 1) * max(t_load, cost_lower) + cost_lower + t_store
 * (trips >= 1; trips == 0 gives t_store). */
double vx_cost_temporal(double t_load, int64_t trips, double cost_lower, double t_store);
/* Equation 3: ceil(parallel / units) for parallel >= 0, units >= 1 (else -1). */
int64_t vx_cost_parallel_factor(int64_t parallel, int64_t units);

/* Hardware description in use on the current device (or the override). */
vx_status vx_get_hwinfo(vx_hwinfo* out);
/* Replace the device description for planning (tests, what-if studies);
 * NULL restores the real device.  Does not change which kernels exist. */
vx_status vx_set_hwinfo_override(const vx_hwinfo* hw);

/*
 * Offline calibration of the kernels' low levels — the empirical part of the
 * hybrid analyzer (Section 5.2): per kernel, the measured time of one
 * workgroup K step and the fixed per-call cost, with the device fully and
 * lightly loaded, taken once per device on synthetic shapes derived from the
 * kernel's own tile and the CU count (never from application shapes).  The
 * table is written by paper_2409_01075_amd/calibrate.py and is used only if
 * it was measured on this exact kernel set (vx_registry_hash).  The library
 * tries the default file (calib_<arch>.txt next to the library) at its first
 * plan; without it the selector is purely analytical.
 *
 * vx_calibration_load: path NULL = the default file; *n_loaded = kernels read.
 * Returns VX_ERR_INVALID_ARG if the file is missing, malformed or was taken on
 * another kernel set; a failed explicit path keeps the table in use, a failed
 * default (NULL) leaves no table in use.  vx_calibration_enable(0) returns to the analytical
 * model (ablation); vx_calibration_active reports whether it is in use.
 */
vx_status vx_calibration_load(const char* path, int* n_loaded);
vx_status vx_calibration_enable(int enable);
int vx_calibration_active(void);
const char* vx_registry_hash(void);

/* Registry introspection. */
int vx_registry_count(void);
vx_status vx_registry_get(int id, vx_kernel_info* out);
/* Workgroups of a kernel resident per CU on the current device description
 * (the tighter of its LDS and register budgets). */
vx_status vx_kernel_occupancy(int kernel_id, int* wgs_per_cu);

/*
 * Pin every following call to one kernel and split-K factor (kernel_id < 0
 * restores the analytical choice; split_k == 0 lets the selector pick the
 * split and grid for the forced kernel; split_k < 0 forces the hybrid grid
 * with -split_k slices per split tile, VX_ERR_NO_CANDIDATE at calls whose
 * tiles do not exceed one wave of the device).  For tests and ablation studies; process-wide.
 * A forced kernel of the wrong dtype or alignment class makes calls return
 * VX_ERR_NO_CANDIDATE.
 */
vx_status vx_force_plan(int kernel_id, int split_k);

/*
 * Hierarchy ablation (the Static1 variant of Section 7.4): restrict every
 * following selection to kernels whose wavefront-level strategy is a
 * wave_m x wave_n wavefront tile built from mfma_m x mfma_m MFMA instructions;
 * the workgroup tile and the split stay dynamic.  (Static2, which also fixes
 * the workgroup tile, is vx_force_plan(kernel_id, 0).)  All three 0 lifts the
 * restriction.  VX_ERR_INVALID_ARG for a partly zero or negative triple,
 * VX_ERR_NO_CANDIDATE if no enabled kernel has that strategy; calls whose
 * dtype or alignment no such kernel serves return VX_ERR_NO_CANDIDATE.
 * Process-wide; for studies and tests.
 */
vx_status vx_fix_wavefront(int wave_m, int wave_n, int mfma_m);

/*
 * Hardware-adaptation ablation (Section 7.4, "Dynamic Hardware Adaptation";
 * the adaptive backend choice of Section 6.2): restrict every following
 * selection to the matrix-core kernels (mask 1: families 0 and 1), to the
 * vector-ALU kernels (mask 2: family 2), or lift the restriction (3, or 0).
 * VX_ERR_INVALID_ARG for a mask outside 0..3, VX_ERR_NO_CANDIDATE if no
 * enabled kernel is left; calls that no allowed kernel serves (dtype,
 * alignment, K beyond a kernel's k_max) return VX_ERR_NO_CANDIDATE.
 * Process-wide; for studies and tests.
 */
vx_status vx_restrict_backends(int mask);

/*
 * Grid-level ablation: with enable = 0 the selector no longer considers the
 * hybrid grid (whole waves of whole tiles plus the remaining tiles split K
 * ways, see vx_plan.dp_tiles); 1 (the default) restores it.  Forced plans
 * (vx_force_plan) are not affected.  Process-wide; for studies and tests.
 */
vx_status vx_enable_hybrid_grid(int enable);

/*
 * Workgroup-level ablation of the rotated K order.  With enable = 1 (the
 * default), a GEMM whose A and B of one batch entry together fit in one XCD's
 * L2 (vx_hwinfo.l2_bytes_per_xcd), run by a plain-ring direct-to-LDS kernel
 * (vx_kernel_info.family 1, schedule 0), starts tile (tm, tn) at step
 * (tm + tn) mod nk of its K slice and wraps around, so that the tiles sharing
 * an A or B panel do not request the same L2 lines at the same time.  Every
 * other call, and every call with enable = 0, walks K in order.  Either way
 * each output element is the fp32 sum of the same products; only the order of
 * that sum differs (fixed per tile, so repeated calls stay bit-identical).
 * Takes effect at the next launch; plans are unaffected.  Process-wide; for
 * studies and tests.
 */
vx_status vx_enable_k_rotation(int enable);

/*
 * The search of Equation 1 is exact but prices only the (kernel, split, grid)
 * triples that can win: each calibrated kernel first gets a lower bound on
 * its cost over every split and both grids, and is skipped when that bound
 * exceeds the best cost already found.  With enable = 1 every triple is
 * priced instead (the plan is the same; the switch exists so that tests can
 * check that).  0 (the default) restores the pruned search.  Retires cached
 * plans.  Process-wide; for tests.
 */
vx_status vx_selector_exhaustive(int enable);

/* Number of (kernel, split, grid) triples the calling thread's last search
 * priced (0 before its first search; a cached plan is not a search). */
int64_t vx_selector_last_evaluations(void);

/*
 * Test hook for the split-K workspace fallback: with fail != 0 the library's
 * own lazily allocated workspace is treated as unavailable, so calls on a
 * stream without a workspace plan without split-K (as they do when the
 * allocation really fails), and plan queries report such plans.  0 restores
 * normal behaviour.  Process-wide; for tests.
 */
vx_status vx_test_fail_workspace_alloc(int fail);

/*
 * Hand the library a caller-owned device buffer to use as the split-K
 * workspace of `stream` (NULL/0 bytes: return to the library's own lazily
 * allocated buffer).  The buffer must stay valid until the stream's work
 * using it has finished; the library zeroes its first 256 KiB (the arrival
 * counters) with an asynchronous memset on `stream`.  bytes must be at least
 * 256 KiB + the partials of the plans that will run.
 */
vx_status vx_set_workspace(void* ptr, size_t bytes, void* stream);

/*
 * 2-D convolution (the paper's second operator, Section 7.1 and Table 4) on
 * the same hierarchy, as an implicit GEMM: M = n*oh*ow output pixels,
 * N = c_out, K = kh*kw*c_in, the A tile gathered from the image through the
 * im2col map, the filter read as a K x c_out row-major matrix.
 *
 *   y[n][oh][ow][co] = sum_{kh, kw, ci} x[n][ih][iw][ci] * w[kh][kw][ci][co],
 *   ih = oh*stride_h - pad_h + kh*dil_h,  iw = ow*stride_w - pad_w + kw*dil_w,
 *
 * with taps outside the h x w image absent (zero padding) and
 * oh = (h + 2*pad_h - dil_h*(kh-1) - 1) / stride_h + 1 (likewise ow; no output
 * when the numerator is negative).  Layouts (dense, element-aligned pointers
 * allowed): x n x h x w x c_in, w kh x kw x c_in x c_out, y n x oh x ow x
 * c_out.  fp32 accumulation; y rounded to nearest even in `dtype`.
 * Ownership and errors as for vx_gemm: sizes < 0, kh/kw/strides/dilations
 * < 1, pads < 0, h + 2*pad_h or w + 2*pad_w of 2^30 or more, M, K, M*c_out
 * or K*c_out beyond 2^31 - 1 elements, a NULL operand with a
 * non-empty extent, or y overlapping x or w -> VX_ERR_INVALID_ARG; an empty
 * output is a no-op; c_in = 0 writes zeros.  Asynchronous on `stream`.
 */
typedef struct vx_conv2d_desc {
    int64_t n, h, w, c_in, c_out, kh, kw;
    int64_t stride_h, stride_w, pad_h, pad_w, dil_h, dil_w;
    vx_dtype dtype;
} vx_conv2d_desc;

vx_status vx_conv2d(const vx_conv2d_desc* d, const void* x, const void* w, void* y, void* stream);

/* Output extent of the convolution `d` (host only): *oh and *ow as defined
 * above (0 when the numerator is negative).  The same descriptor checks as
 * vx_conv2d (VX_ERR_INVALID_ARG, VX_ERR_UNSUPPORTED_DTYPE); NULL outputs ->
 * VX_ERR_INVALID_ARG. */
vx_status vx_conv2d_output_dims(const vx_conv2d_desc* d, int64_t* oh, int64_t* ow);

/* The plan vx_conv2d would run for `d` (host only, no launch). */
vx_status vx_conv2d_plan_query(const vx_conv2d_desc* d, vx_plan* out);

const char* vx_status_string(vx_status s);
const char* vx_version(void);

#ifdef __cplusplus
}
#endif
#endif /* VX_H */
