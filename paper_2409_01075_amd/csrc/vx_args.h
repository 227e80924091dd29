// Launch arguments shared by the host launcher and the device kernels.
#pragma once
#include <stdint.h>

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
};
