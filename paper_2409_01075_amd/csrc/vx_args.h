// Launch arguments shared by the host launcher and the device kernels.
#pragma once
#include <stdint.h>

// Division of a non-negative integer below 2^31 by a divisor fixed for the
// launch, as a multiply-high, an add and a shift (Granlund and Montgomery,
// "Division by invariant integers using multiplication", 1994, Section 4):
//   s = ceil(log2 d),  m = floor(2^32 (2^s - d) / d) + 1,
//   x / d = (mulhi32(x, m) + x) >> s      for 0 <= x < 2^31 (no overflow: mulhi32 < x).
// The host derives (m, s) once per launch (vx_fastdiv_make); the kernels'
// grid-level index arithmetic (fdiv in gemm_kernel.h) then costs a few scalar
// instructions instead of a full integer division sequence per quotient.
struct VxFastDiv {
    unsigned m, s;
};

static inline VxFastDiv vx_fastdiv_make(unsigned d)
{
    unsigned s = 0;
    while ((1ull << s) < (unsigned long long)d)
        ++s;
    VxFastDiv f;
    f.s = s;
    f.m = (unsigned)(((1ull << 32) * ((1ull << s) - d)) / d + 1);
    return f;
}

struct VxGemmArgs {
    const void* A;          // M x K row-major (lda = K), batch stride sA elements
    const void* B;          // K x N row-major (ldb = N), batch stride sB (0 = broadcast)
    void* C;                // M x N row-major (ldc = N), batch stride sC
    int64_t sA, sB, sC;
    int M, N, K;
    int tiles_m, tiles_n;   // ceil(M / Mb), ceil(N / Nb)
    int split;              // split-K factor s (>= 1)
    int k_per_split;        // K extent of one slice, a multiple of Kb
    int batch;
    int group_m;            // tile rows walked together by the grid-level order
    int num_xcd;            // workgroups are dispatched round-robin over this many XCDs
    int grid;               // workgroups in the launch: tiles_m * tiles_n * split * batch, or with
                            // dp_tiles > 0, dp_tiles + (tiles_m * tiles_n * batch - dp_tiles) * split
    int dp_tiles;           // > 0: hybrid grid -- the first dp_tiles tiles (whole waves of the
                            // device, a multiple of num_xcd) run whole, one workgroup each; only
                            // the remaining tiles are split `split` ways.  0: every tile is split.
    float* ws;              // split-K partial tiles (split > 1), fp32
    unsigned* tickets;      // one self-resetting arrival counter per output tile
    // 2-D convolution as an implicit GEMM (conv kernels only): A is the input
    // image x (N x H x W x Cin) read through the im2col map, M = N*OH*OW,
    // K = KH*KW*Cin, B is the filter (KH*KW*Cin x Cout), C the output.
    int cH, cW, cC, cKW, cOH, cOW;
    int csh, csw, cph, cpw, cdh, cdw;   // stride, padding, dilation (height, width)
    int krot;               // 1: each tile walks its K steps starting at step (tm + tn) mod nk
                            // (plain-ring direct-to-LDS GEMM kernels); 0: in order
    // grid-level divisors (VxFastDiv) and the XCD remap's quotients, set by the host:
    int xq, xr;             // grid (or, hybrid, the split class) / num_xcd and % num_xcd
    int xq_dp, xr_dp;       // hybrid: dp_tiles / num_xcd and % num_xcd
    VxFastDiv f_xcd;        // num_xcd
    VxFastDiv f_tiles;      // tiles_m * tiles_n
    VxFastDiv f_split;      // split
    VxFastDiv f_rt;         // hybrid: batch * tiles_m * tiles_n - dp_tiles (tiles that are split)
    VxFastDiv f_group;      // group_m * tiles_n (tiles of one group of tile rows)
    VxFastDiv f_gm;         // group_m (rows of a full group)
    VxFastDiv f_gm_last;    // rows of the last group: tiles_m - (groups - 1) * group_m
};
