// Vector-ALU family for small M (gfx950): the adaptive second backend of the
// hierarchy, for calls whose M is too small to fill a matrix-core tile.
//
// The same three levels as the MFMA families, with a different level 0:
//   level 2  grid       parallel loops over (batch, K slice, tile) — shared
//                       with the MFMA kernels (grid_pos, split-K protocol)
//   level 1  workgroup  temporal reduction over the K slice, KPI rows per step;
//                       B rows go straight from memory into VGPRs (16-byte,
//                       whole-line row chunks, two register sets in flight),
//                       A's slice waits in LDS transposed to [k][m]
//   level 0  lane       MT x VE outputs: per k, one 16-byte chunk of a B row
//                       times MT values of A, accumulated in fp32 with
//                       v_dot2_f32_{f16,bf16} on (k, k+1) pairs or v_fma_f32
// The MFMA operand layout needs B's k values contiguous per lane, which forces
// B through LDS (transposing reads) and caps the bytes in flight per CU at the
// ring's size; here B is consumed in its natural n-contiguous layout.
//
// Lane layout: lane = c * KL + kl.  c selects the 16-byte column chunk of the
// tile (CW chunks cover NB columns: 128 bytes of a row), kl the k group; the
// KL lanes of one chunk are reduced by shuffles inside the wave, the waves
// through LDS, always in the same order (the result is deterministic).
#pragma once
#include "gemm_kernel.h"

namespace vxk {

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

template <int DT_, int MT_, int NB_, int WAVES_, int U_, int KSMAX_>
struct VCfg {
    static constexpr int DT = DT_, MT = MT_, NB = NB_, WAVES = WAVES_, U = U_, KSMAX = KSMAX_;
    static constexpr bool H = DT != DT_F32;
    static constexpr int EB = H ? 2 : 4;               // bytes per element
    static constexpr int VE = 16 / EB;                 // elements per 16-byte chunk
    static constexpr int CW = NB / VE;                 // lanes per row (column chunks)
    static constexpr int KL = 64 / CW;                 // k groups per wave
    static constexpr int PK = H ? 2 : 1;               // k rows per group: a pair for dot2
    static constexpr int NT = WAVES * 64;
    static constexpr int KPI = WAVES * KL * PK * U;    // k rows per step (the registry's Kb)
    static constexpr int A_LDS = KSMAX * MT * EB;      // A slice, [k / PK][m] of PK-element words
    static constexpr int RED_LDS = WAVES * MT * NB * 4;
    static constexpr int LDS_BYTES = A_LDS > RED_LDS ? A_LDS : RED_LDS;
    static constexpr int OUT4 = MT * NB / 4;           // groups of 4 outputs in the tile

    static_assert(CW == 8 && KL == 8, "one 128-byte row segment per 8 lanes");
    static_assert(MT % 4 == 0 && MT <= 16, "rows in groups of 4");
    static_assert(KSMAX % KPI == 0, "slice capacity in whole steps");
    static_assert(OUT4 <= NT, "one group of 4 outputs per thread at most");
    static_assert(LDS_BYTES <= 159 * 1024, "LDS budget of one CU, less 1 KiB for the split-K flag");
};

// (B[k][j], B[k+1][j]) packed for dot2, from two 16-byte row chunks: element
// j of b0 (row k) in the low half, element j of b1 (row k+1) in the high half.
__device__ __forceinline__ unsigned pair16(const u32x4& b0, const u32x4& b1, int j)
{
    return __builtin_amdgcn_perm(b1[j >> 1], b0[j >> 1], (j & 1) ? 0x07060302u : 0x05040100u);
}

template <int DT>
__device__ __forceinline__ float dot2(unsigned a, unsigned b, float c)
{
    if constexpr (DT == DT_F16)
        return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, a), __builtin_bit_cast(f16x2, b), c, false);
    else
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

template <class C>
__device__ __forceinline__ void gemm_valu_body(const VxGemmArgs& args)
{
    const VxGemmArgs p = pin_args(args);
    __shared__ __attribute__((aligned(16))) char smem[C::LDS_BYTES];
    lds_char* lds = (lds_char*)smem;

    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    const int c = lane / C::KL, kl = lane % C::KL;
    const GridPos g = grid_pos<C::MT, C::NB, C::KPI>(p);
    const int Mrel = p.M - g.m0;
    const int ks = g.nk * C::KPI;                     // the slice rounded up to whole steps (<= KSMAX)
    const int kv = g.kend - g.kbeg;                   // valid k of the slice

    // B: buffer resource from row kbeg; rows at or past kend read as zeros
    const char* Bb = (const char*)p.B + ((int64_t)g.b * p.sB + (int64_t)g.kbeg * p.N) * C::EB;
    const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
        (void*)Bb, (short)0, kv > 0 ? (int)((unsigned)kv * (unsigned)p.N * C::EB) : 0, 0x00020000);
    const int n = g.n0 + c * C::VE;
    const bool col_ok = n < p.N;

    // registers for two steps of B chunks
    u32x4 b0[C::U][C::PK], b1[C::U][C::PK];
    auto load = [&](u32x4 (&bs)[C::U][C::PK], int it) {
#pragma unroll
        for (int u = 0; u < C::U; ++u)
#pragma unroll
            for (int r = 0; r < C::PK; ++r) {
                const int kr = (((it * C::U + u) * C::WAVES + wave) * C::KL + kl) * C::PK + r;
                const unsigned off = col_ok ? (unsigned)(kr * p.N + n) * C::EB : 0x80000000u;
                bs[u][r] = __builtin_amdgcn_raw_buffer_load_b128(rb, off, 0, 0);
            }
    };
    if (g.nk > 0)
        load(b0, 0);

    // A slice -> LDS as At[k / PK][m] (PK-element words), zeros past M and kend
    {
        const char* Ab = (const char*)p.A + ((int64_t)g.b * p.sA + (int64_t)g.m0 * p.K + g.kbeg) * C::EB;
        const int cpr = ks / C::VE;                   // 16-byte chunks per row of the slice
        for (int q = t; q < C::MT * cpr; q += C::NT) {
            const int m = q / cpr, kc = q % cpr;
            u32x4 v = {0, 0, 0, 0};
            if (m < Mrel && kc * C::VE < kv)
                v = ld_g<u32x4>(Ab + ((int64_t)m * p.K + kc * C::VE) * C::EB);
#pragma unroll
            for (int w = 0; w < 4; ++w)              // 4 words of PK elements per chunk
                *(__attribute__((address_space(3))) unsigned*)(lds + ((kc * 4 + w) * C::MT + m) * 4) = v[w];
        }
    }
    __syncthreads();

    float acc[C::MT][C::VE];
#pragma unroll
    for (int m = 0; m < C::MT; ++m)
#pragma unroll
        for (int j = 0; j < C::VE; ++j)
            acc[m][j] = 0.0f;

    auto compute = [&](const u32x4 (&bs)[C::U][C::PK], int it) {
#pragma unroll
        for (int u = 0; u < C::U; ++u) {
            const int grp = ((it * C::U + u) * C::WAVES + wave) * C::KL + kl;   // k group of this lane
            if constexpr (C::H) {
                unsigned a[C::MT];   // (A[m][k], A[m][k+1]) pairs
#pragma unroll
                for (int m4 = 0; m4 < C::MT / 4; ++m4) {
                    const u32x4 w = *(lds_u32x4*)(lds + (grp * C::MT + m4 * 4) * 4);
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        a[m4 * 4 + e] = w[e];
                }
                unsigned bp[C::VE];
#pragma unroll
                for (int j = 0; j < C::VE; ++j)
                    bp[j] = pair16(bs[u][0], bs[u][1], j);
#pragma unroll
                for (int m = 0; m < C::MT; ++m)
#pragma unroll
                    for (int j = 0; j < C::VE; ++j)
                        acc[m][j] = dot2<C::DT>(a[m], bp[j], acc[m][j]);
            } else {
                // whole-vector bit casts: element-wise casts of vector elements
                // were compiled as if every element were element 0
                const f32x4 bf = __builtin_bit_cast(f32x4, bs[u][0]);
                float af[C::MT];
#pragma unroll
                for (int m4 = 0; m4 < C::MT / 4; ++m4) {
                    const f32x4 w = __builtin_bit_cast(f32x4, *(lds_u32x4*)(lds + (grp * C::MT + m4 * 4) * 4));
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        af[m4 * 4 + e] = w[e];
                }
#pragma unroll
                for (int m = 0; m < C::MT; ++m)
#pragma unroll
                    for (int j = 0; j < C::VE; ++j)
                        acc[m][j] = __builtin_fmaf(af[m], bf[j], acc[m][j]);
            }
        }
    };

    // K loop: the next step's loads are issued before this step's arithmetic
    for (int it = 0; it < g.nk; it += 2) {
        if (it + 1 < g.nk)
            load(b1, it + 1);
        compute(b0, it);
        if (it + 1 < g.nk) {
            if (it + 2 < g.nk)
                load(b0, it + 2);
            compute(b1, it + 1);
        }
    }

    // reduce the KL k groups of each column chunk (lane bits 0..2) in the wave
#pragma unroll
    for (int m = 0; m < C::MT; ++m)
#pragma unroll
        for (int j = 0; j < C::VE; ++j) {
            float v = acc[m][j];
            v += __shfl_xor(v, 1);
            v += __shfl_xor(v, 2);
            v += __shfl_xor(v, 4);
            acc[m][j] = v;
        }
    __syncthreads();   // every wave is done with the A slice: LDS becomes the reduction area
    __attribute__((address_space(3))) float* red = (__attribute__((address_space(3))) float*)lds;
    if (kl == 0) {
#pragma unroll
        for (int m = 0; m < C::MT; ++m)
#pragma unroll
            for (int j = 0; j < C::VE; ++j)
                red[(wave * C::MT + m) * C::NB + c * C::VE + j] = acc[m][j];
    }
    __syncthreads();
    // the workgroup's tile: thread t < OUT4 holds 4 consecutive outputs of one row
    f32x4 out = {0.0f, 0.0f, 0.0f, 0.0f};
    const int m = (4 * t) / C::NB, nn = (4 * t) % C::NB;
    if (t < C::OUT4) {
#pragma unroll
        for (int w = 0; w < C::WAVES; ++w)
            out += *(__attribute__((address_space(3))) f32x4*)(red + (w * C::MT + m) * C::NB + nn);
    }
    if (g.split > 1) {
        f32x4 v[1] = {out};
        if (!split_reduce<1>(p, g, v, t, C::OUT4))
            return;
        out = v[0];
    }
    if (t < C::OUT4 && m < Mrel) {
        char* Cb = (char*)p.C + (int64_t)g.b * p.sC * C::EB;
        const int col = g.n0 + nn;
        if (col < p.N)
            store4<C::DT>(Cb, (int64_t)(g.m0 + m) * p.N + col, col, p.N, out[0], out[1], out[2], out[3]);
    }
}

}  // namespace vxk
