// Runtime-shaped dense GEMM C = A x B for gfx950 (CDNA4), row-major, fp32
// accumulation.  One template covers every registry candidate.
//
// The hierarchy follows the unified recursive abstraction (Section 4.2,
// Algorithm 1, with the GPU rows of Table 1):
//   level 2  grid       parallel loops over (batch, K slice, tile): no load/store
//   level 1  workgroup  temporal reduction loop over K in Kb steps; each step
//                       loads the A and B tiles from global memory into a
//                       2-stage LDS ring (prefetch of step k+1 overlaps the
//                       MFMAs of step k), then runs level 0
//   level 0  wavefront  LDS -> VGPR fragment loads and MFMA instructions, with
//                       the fp32 accumulators kept in registers until Store
// Every level's tile is an integer multiple of the level below (Section 5.1);
// partial tiles at the M, N and K edges are predicated, never padded.
//
// Operand order: the MFMA is issued as D = Bt * At, i.e. with the B fragment
// in the instruction's A slot and the A fragment in its B slot.  Each lane
// then owns 4 consecutive output columns of one C row, so the epilogue writes
// row-major C with 4-element vector stores.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "vx_args.h"

namespace vxk {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
// The same vectors at element alignment.  The HSA runtime runs gfx9 memory in
// unaligned mode, so these still compile to single 8/16-byte global accesses.
typedef unsigned u32x4_u __attribute__((ext_vector_type(4), aligned(2)));
typedef unsigned u32x2_u __attribute__((ext_vector_type(2), aligned(2)));
// Global memory through address-space-1 pointers.  The operand and result
// pointers arrive in a by-value argument struct, from which the compiler
// cannot infer their address space: a plain dereference would compile to a
// flat access, which also counts against the LDS wait counter, so every wait
// for an LDS read would wait for the global loads in flight as well.
template <class T>
__device__ __forceinline__ T ld_g(const void* p)
{
    return *(const __attribute__((address_space(1))) T*)p;
}
template <class T>
__device__ __forceinline__ void st_g(void* p, T v)
{
    *(__attribute__((address_space(1))) T*)p = v;
}
// LDS pointers stay in address space 3 from the __shared__ object onwards, so
// every LDS access compiles to a ds_* instruction with no generic-address
// detour.
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) u32x2 lds_u32x2;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;

enum { DT_F32 = 0, DT_F16 = 1, DT_BF16 = 2 };

// Compile-time description of one candidate: workgroup tile Mb x Nb x Kb,
// WM x WN wavefronts, MFMA instruction tile MI x MI, operands whose rows are
// 16-byte aligned (VEC) or only element aligned, and whether A is a plain
// matrix or a convolution's input image (CONV: the implicit GEMM).
template <int DT_, int MB_, int NB_, int KB_, int WM_, int WN_, int MI_, bool VEC_, bool CONV_ = false, int PF_ = 1>
struct Cfg {
    static constexpr int DT = DT_, MB = MB_, NB = NB_, KB = KB_, WM = WM_, WN = WN_, MI = MI_;
    static constexpr bool VEC = VEC_;
    static constexpr bool CONV = CONV_;                  // A is an image read through the im2col map
    // K steps whose loads are in flight in registers while one step computes
    // from LDS (PF register sets; the LDS keeps its two stages)
    static constexpr int PF = PF_;
    static constexpr bool H = DT != DT_F32;              // 16-bit inputs
    static constexpr int NT = WM * WN * 64;              // threads per workgroup
    static constexpr int MW = MB / WM, NW = NB / WN;     // wavefront tile
    static constexpr int FM = MW / MI, FN = NW / MI;     // MFMA tiles per wavefront
    static constexpr int ACC = MI == 16 ? 4 : 16;        // fp32 accumulators per lane per MFMA tile
    static constexpr int EB = H ? 2 : 4;                 // bytes per element
    static constexpr int VE = 16 / EB;                   // elements per 16-byte vector
    static constexpr int PADK = 16 / EB;                 // LDS row padding, elements
    static constexpr int LDA = KB + PADK;                // As[m][k]
    static constexpr int LDB = H ? KB + PADK : NB + 4;   // 16-bit: Bs[n][k]; fp32: Bs[k][n]
    static constexpr int A_ELEMS = MB * LDA;
    static constexpr int B_ELEMS = H ? NB * LDB : KB * LDB;
    static constexpr int STAGE_BYTES = (A_ELEMS + B_ELEMS) * EB;
    static constexpr int LDS_BYTES = 2 * STAGE_BYTES;
    // A tile: MB*KB/VE vectors along k
    static constexpr int AV = MB * KB / VE / NT;
    // B tile, 16-bit: blocks of BK k-rows x 8 columns, transposed on the way into LDS
    static constexpr int BK = !H ? 1 : ((KB / 8) * (NB / 8) % NT == 0 && (KB / 8) * (NB / 8) >= NT) ? 8
                                     : ((KB / 4) * (NB / 8) % NT == 0 && (KB / 4) * (NB / 8) >= NT) ? 4 : 2;
    static constexpr int KBB = KB / BK;                  // k-blocks per tile
    static constexpr int BBLK = H ? KBB * (NB / 8) / NT : 0;
    // B tile, fp32: KB*NB/4 vectors along n
    static constexpr int BV = H ? NB * KB / 8 / NT : KB * NB / 4 / NT;
    static constexpr int KI = H ? (MI == 16 ? 32 : 16) : (MI == 16 ? 4 : 2);   // K per MFMA
    static constexpr int KCH = H ? KI : (MI == 16 ? 16 : 8);                      // K per fragment load

    // epilogue through LDS (store_lds) when the C tile fits the idle ring
    static constexpr int LDC = NB + VE;
    static constexpr bool LDS_EPI = MB * LDC * EB <= LDS_BYTES;

    static_assert(MB % WM == 0 && NB % WN == 0, "waves must tile the workgroup tile");
    static_assert(MW % MI == 0 && NW % MI == 0, "MFMA tiles must tile the wavefront tile");
    static_assert(KB % KCH == 0, "Kb must be a multiple of the MFMA K chunk");
    static_assert(AV >= 1 && AV * VE * NT == MB * KB, "A tile must split evenly over threads");
    static_assert(BV >= 1 && (H ? BV * 8 : BV * 4) * NT == NB * KB, "B tile must split evenly over threads");
    static_assert(!H || (BBLK >= 1 && BBLK * NT * BK * 8 == KB * NB), "B blocks must split evenly");
    static_assert(LDS_BYTES <= 159 * 1024, "LDS budget of one CU, less 1 KiB for the split-K flag");
    static_assert(PF >= 1 && PF <= 4, "register sets of K steps in flight");
};

__device__ __forceinline__ unsigned lo16(unsigned w) { return w & 0xffffu; }
__device__ __forceinline__ unsigned hi16(unsigned w) { return w >> 16; }
__device__ __forceinline__ unsigned pack2(unsigned lo, unsigned hi) { return (lo & 0xffffu) | (hi << 16); }
// element j (0..7) of a vector of eight 16-bit values
__device__ __forceinline__ unsigned elem16(const u32x4& v, int j)
{
    unsigned w = v[j >> 1];
    return (j & 1) ? hi16(w) : lo16(w);
}

// A of a convolution for one K step: the chunk column held in `ca` (see
// ConvA) of AV rows, gathered from the image X through the im2col map.  Row gm
// of the implicit A is output pixel (n, oh, ow); column gk is filter tap
// (kh, kw) and input channel ci, with gk = (kh * KW + kw) * Cin + ci.  When
// Cin is a multiple of the chunk, a chunk never straddles two taps and is one
// 16-byte load (or zeros in the padding); otherwise it is gathered element by
// element, except where it stays inside one filter row (see below).  Taps in
// the padding and k at or past kend read as zeros.
template <class CA, int AV, int VE, bool H, int EB>
__device__ __forceinline__ void conv_gather(const VxGemmArgs& p, const char* __restrict__ X, const CA& ca, int kend,
                                            u32x4 (&ra)[AV])
{
    if (p.cC % VE == 0) {   // wave-uniform: a chunk is VE channels of one tap
        const int dh = ca.kh * p.cdh, dw = ca.kw * p.cdw;
        const int64_t koff = ((int64_t)dh * p.cW + dw) * p.cC + ca.ci;
        const bool kin = ca.gk < kend;
#pragma unroll
        for (int v = 0; v < AV; ++v) {
            u32x4 x = {0, 0, 0, 0};
            if (kin && (unsigned)(ca.ih0[v] + dh) < (unsigned)p.cH && (unsigned)(ca.iw0[v] + dw) < (unsigned)p.cW)
                x = ld_g<u32x4_u>(X + (ca.pix[v] + koff) * EB);
            ra[v] = x;
        }
        return;
    }
    // channels not a multiple of the chunk: the VE elements of a chunk walk
    // over channels, then filter columns, then filter rows
    int ci = ca.ci, kw = ca.kw, kh = ca.kh;
    int dhe[VE], dwe[VE];
    int64_t koff[VE];
#pragma unroll
    for (int e = 0; e < VE; ++e) {
        dhe[e] = ca.gk + e < kend ? kh * p.cdh : -(1 << 30);   // k past kend: an out-of-range row
        dwe[e] = kw * p.cdw;
        koff[e] = ((int64_t)(kh * p.cdh) * p.cW + dwe[e]) * p.cC + ci;
        if (++ci == p.cC) {
            ci = 0;
            if (++kw == p.cKW) {
                kw = 0;
                ++kh;
            }
        }
    }
    // With unit dilation along the width, the KW x Cin elements of one filter
    // row are contiguous in the NHWC image (k = kw Cin + ci maps to kw Cin + ci
    // elements past the row's first tap): a chunk that stays within one filter
    // row, below kend, whose first and last taps fall inside the image, is one
    // 16-byte (unaligned) load.  The chunk's first tap is at column ca.kw, its
    // last at kw_last (same row ca.kh).
    const int run = p.cKW * p.cC;                  // elements of one filter row
    const int j0 = ca.kw * p.cC + ca.ci;           // the chunk's first element within its row
    const bool one_row = p.cdw == 1 && j0 + VE <= run && ca.gk + VE <= kend;
    const int kw_last = (j0 + VE - 1) / p.cC;
#pragma unroll
    for (int v = 0; v < AV; ++v) {
        unsigned e16[VE];
        if (one_row && (unsigned)(ca.ih0[v] + dhe[0]) < (unsigned)p.cH && ca.iw0[v] + dwe[0] >= 0 &&
            ca.iw0[v] + kw_last < p.cW) {
            ra[v] = ld_g<u32x4_u>(X + (ca.pix[v] + koff[0]) * EB);
            continue;
        }
#pragma unroll
        for (int e = 0; e < VE; ++e) {
            unsigned val = 0u;
            if ((unsigned)(ca.ih0[v] + dhe[e]) < (unsigned)p.cH && (unsigned)(ca.iw0[v] + dwe[e]) < (unsigned)p.cW) {
                const char* src = X + (ca.pix[v] + koff[e]) * EB;
                val = H ? (unsigned)ld_g<uint16_t>(src) : ld_g<unsigned>(src);
            }
            e16[e] = val;
        }
        u32x4 x;
        if (H) {
#pragma unroll
            for (int e = 0; e < 8; e += 2)
                x[e >> 1] = pack2(e16[e], e16[e + 1]);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                x[e] = e16[e];
        }
        ra[v] = x;
    }
}

template <class C>
struct Tile {
    // ---------------------------------------------------------- Load (level 1)
    // Registers holding one K step of A and B between the global load and the
    // LDS store.
    u32x4 ra[C::AV];
    u32x4 rb[C::H ? C::BBLK * C::BK : C::BV];

    // Global -> registers for the K step starting at k0 (< kend).  Every
    // thread moves 16-byte chunks of a row (8 elements of 16-bit data, 4 of
    // fp32).  With VEC the rows are 16-byte aligned and a chunk is wholly in
    // or out of range.  Otherwise a chunk wholly in range is still one
    // (misaligned) 16-byte load, and only the chunk straddling the K or N edge
    // is gathered element by element.
    __device__ __forceinline__ void load(const char* __restrict__ Ab, const char* __restrict__ Bb,
                                         int m0, int n0, int k0, int kend, int M, int N, int K, int t)
    {
        // A: MB x KB, chunks along k (a convolution gathers A in load_a_conv)
#pragma unroll
        for (int v = 0; v < (C::CONV ? 0 : C::AV); ++v) {
            const int idx = t + v * C::NT;
            const int r = idx / (C::KB / C::VE), c = idx % (C::KB / C::VE);
            const int gm = m0 + r, gk = k0 + c * C::VE;
            const char* p = Ab + ((int64_t)gm * K + gk) * C::EB;
            if (C::VEC) {
                ra[v] = (gm < M && gk < kend) ? ld_g<u32x4>(p) : u32x4{0, 0, 0, 0};
            } else {
                u32x4 x = {0, 0, 0, 0};
                if (gm < M) {
                    if (gk + C::VE <= kend)
                        x = ld_g<u32x4_u>(p);
                    else
                        x = gather_row(p, kend - gk);
                }
                ra[v] = x;
            }
        }
        if (C::H) {
            // B: blocks of BK rows x 8 columns (16 bytes per row)
#pragma unroll
            for (int i = 0; i < C::BBLK; ++i) {
                const int idx = t + i * C::NT;
                const int kb = idx % C::KBB, nb = idx / C::KBB;
                const int gn = n0 + nb * 8;
#pragma unroll
                for (int r = 0; r < C::BK; ++r) {
                    const int gk = k0 + kb * C::BK + r;
                    const char* p = Bb + ((int64_t)gk * N + gn) * 2;
                    if (C::VEC) {
                        rb[i * C::BK + r] = (gk < kend && gn < N) ? ld_g<u32x4>(p) : u32x4{0, 0, 0, 0};
                    } else {
                        u32x4 x = {0, 0, 0, 0};
                        if (gk < kend) {
                            if (gn + 8 <= N)
                                x = ld_g<u32x4_u>(p);
                            else
                                x = gather_row(p, N - gn);
                        }
                        rb[i * C::BK + r] = x;
                    }
                }
            }
        } else {
            // fp32 B: natural layout, 4 consecutive columns per chunk
#pragma unroll
            for (int v = 0; v < C::BV; ++v) {
                const int idx = t + v * C::NT;
                const int c = idx % (C::NB / 4), kr = idx / (C::NB / 4);
                const int gn = n0 + c * 4, gk = k0 + kr;
                const char* p = Bb + ((int64_t)gk * N + gn) * 4;
                if (C::VEC) {
                    rb[v] = (gk < kend && gn < N) ? ld_g<u32x4>(p) : u32x4{0, 0, 0, 0};
                } else {
                    u32x4 x = {0, 0, 0, 0};
                    if (gk < kend) {
                        if (gn + 4 <= N)
                            x = ld_g<u32x4_u>(p);
                        else
                            x = gather_row(p, N - gn);
                    }
                    rb[v] = x;
                }
            }
        }
    }

    // A of a convolution: the K step at the chunk column held in `ca`,
    // gathered through the im2col map (conv_gather).
    template <class CA>
    __device__ __forceinline__ void load_a_conv(const VxGemmArgs& p, const char* __restrict__ X, const CA& ca,
                                                int kend)
    {
        conv_gather<CA, C::AV, C::VE, C::H, C::EB>(p, X, ca, kend, ra);
    }

    // The first `valid` (< one chunk) elements of a row chunk, zeros after.
    __device__ __forceinline__ static u32x4 gather_row(const char* p, int valid)
    {
        u32x4 x = {0, 0, 0, 0};
        if (C::H) {
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
                const unsigned lo = e < valid ? (unsigned)ld_g<uint16_t>(p + 2 * e) : 0u;
                const unsigned hi = e + 1 < valid ? (unsigned)ld_g<uint16_t>(p + 2 * (e + 1)) : 0u;
                x[e >> 1] = pack2(lo, hi);
            }
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                x[e] = e < valid ? ld_g<unsigned>(p + 4 * e) : 0u;
        }
        return x;
    }

    // Registers -> LDS stage.
    __device__ __forceinline__ void store(char* __restrict__ stage, int t)
    {
        char* As = stage;
        char* Bs = stage + C::A_ELEMS * C::EB;
#pragma unroll
        for (int v = 0; v < C::AV; ++v) {
            const int idx = t + v * C::NT;
            const int r = idx / (C::KB / C::VE), c = idx % (C::KB / C::VE);
            *(u32x4*)(As + (r * C::LDA + c * C::VE) * C::EB) = ra[v];
        }
        if (C::H) {
            // transpose each BK x 8 block into 8 k-vectors (one per column)
#pragma unroll
            for (int i = 0; i < C::BBLK; ++i) {
                const int idx = t + i * C::NT;
                const int kb = idx % C::KBB, nb = idx / C::KBB;
                const u32x4* in = &rb[i * C::BK];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    char* dst = Bs + ((nb * 8 + j) * C::LDB + kb * C::BK) * 2;
                    if (C::BK == 8) {
                        u32x4 o;
#pragma unroll
                        for (int d = 0; d < 4; ++d)
                            o[d] = pack2(elem16(in[2 * d], j), elem16(in[2 * d + 1], j));
                        *(u32x4*)dst = o;
                    } else if (C::BK == 4) {
                        u32x2 o;
#pragma unroll
                        for (int d = 0; d < 2; ++d)
                            o[d] = pack2(elem16(in[2 * d], j), elem16(in[2 * d + 1], j));
                        *(u32x2*)dst = o;
                    } else {
                        *(unsigned*)dst = pack2(elem16(in[0], j), elem16(in[1], j));
                    }
                }
            }
        } else {
#pragma unroll
            for (int v = 0; v < C::BV; ++v) {
                const int idx = t + v * C::NT;
                const int c = idx % (C::NB / 4), kr = idx / (C::NB / 4);
                *(u32x4*)(Bs + (kr * C::LDB + c * 4) * 4) = rb[v];
            }
        }
    }
};

// ------------------------------------------------------------- level 0 -----
template <int DT, int MI>
__device__ __forceinline__ void mfma16(const u32x4& a, const u32x4& b, f32x4& acc)
{
    if (DT == DT_F16)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), acc, 0, 0, 0);
    else
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}
template <int DT>
__device__ __forceinline__ void mfma32(const u32x4& a, const u32x4& b, f32x16& acc)
{
    if (DT == DT_F16)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), acc, 0, 0, 0);
    else
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}

template <class C>
struct Acc {
    typedef typename std::conditional<C::MI == 16, f32x4, f32x16>::type T;
    T v[C::FN][C::FM];
};

// One K step of the wavefront tile out of LDS stage `stage`.
template <class C>
__device__ __forceinline__ void compute_step(const char* __restrict__ stage, Acc<C>& acc, int wm0, int wn0, int lane)
{
    const char* As = stage;
    const char* Bs = stage + C::A_ELEMS * C::EB;
    const int li = lane % C::MI, lg = lane / C::MI;
    if (C::H) {
#pragma unroll
        for (int kk = 0; kk < C::KB / C::KI; ++kk) {
            u32x4 fa[C::FM], fb[C::FN];
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm)
                fa[fm] = *(const u32x4*)(As + ((wm0 + fm * C::MI + li) * C::LDA + kk * C::KI + lg * 8) * 2);
#pragma unroll
            for (int fn = 0; fn < C::FN; ++fn)
                fb[fn] = *(const u32x4*)(Bs + ((wn0 + fn * C::MI + li) * C::LDB + kk * C::KI + lg * 8) * 2);
#pragma unroll
            for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
                for (int fm = 0; fm < C::FM; ++fm) {
                    if constexpr (C::MI == 16)
                        mfma16<C::DT, 16>(fb[fn], fa[fm], acc.v[fn][fm]);
                    else
                        mfma32<C::DT>(fb[fn], fa[fm], acc.v[fn][fm]);
                }
        }
    } else {
        // fp32: a lane's 4 k values per fragment are k = chunk + 4*lg + s (s = 0..3);
        // any k order is valid as long as both operands use the same one.
#pragma unroll
        for (int kc = 0; kc < C::KB / C::KCH; ++kc) {
            f32x4 fa[C::FM];
            float fb[C::FN][4];
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm)
                fa[fm] = *(const f32x4*)(As + ((wm0 + fm * C::MI + li) * C::LDA + kc * C::KCH + lg * 4) * 4);
#pragma unroll
            for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    fb[fn][s] = *(const float*)(Bs + ((kc * C::KCH + lg * 4 + s) * C::LDB + wn0 + fn * C::MI + li) * 4);
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
                    for (int fm = 0; fm < C::FM; ++fm) {
                        if constexpr (C::MI == 16)
                            acc.v[fn][fm] = __builtin_amdgcn_mfma_f32_16x16x4f32(fb[fn][s], fa[fm][s], acc.v[fn][fm], 0, 0, 0);
                        else
                            acc.v[fn][fm] = __builtin_amdgcn_mfma_f32_32x32x2f32(fb[fn][s], fa[fm][s], acc.v[fn][fm], 0, 0, 0);
                    }
        }
    }
}

// ---------------------------------------------------------------- Store ----
// Four consecutive outputs of one C row: one 16/8-byte store when all four
// are inside the row (at any element alignment), else element stores.
template <int DT>
__device__ __forceinline__ void store4(char* __restrict__ Cb, int64_t off, int n, int N, float a0, float a1, float a2, float a3)
{
    if (DT == DT_F32) {
        float* p = (float*)Cb + off;
        if (n + 3 < N) {
            st_g<u32x4_u>(p, __builtin_bit_cast(u32x4, f32x4{a0, a1, a2, a3}));
        } else {
            if (n < N) st_g<float>(p, a0);
            if (n + 1 < N) st_g<float>(p + 1, a1);
            if (n + 2 < N) st_g<float>(p + 2, a2);
            if (n + 3 < N) st_g<float>(p + 3, a3);
        }
    } else {
        uint16_t h[4];
        if (DT == DT_F16) {
            h[0] = __builtin_bit_cast(uint16_t, (_Float16)a0);
            h[1] = __builtin_bit_cast(uint16_t, (_Float16)a1);
            h[2] = __builtin_bit_cast(uint16_t, (_Float16)a2);
            h[3] = __builtin_bit_cast(uint16_t, (_Float16)a3);
        } else {
            h[0] = __builtin_bit_cast(uint16_t, (__bf16)a0);
            h[1] = __builtin_bit_cast(uint16_t, (__bf16)a1);
            h[2] = __builtin_bit_cast(uint16_t, (__bf16)a2);
            h[3] = __builtin_bit_cast(uint16_t, (__bf16)a3);
        }
        uint16_t* p = (uint16_t*)Cb + off;
        if (n + 3 < N) {
            st_g<u32x2_u>(p, u32x2{pack2(h[0], h[1]), pack2(h[2], h[3])});
        } else {
            if (n < N) st_g<uint16_t>(p, h[0]);
            if (n + 1 < N) st_g<uint16_t>(p + 1, h[1]);
            if (n + 2 < N) st_g<uint16_t>(p + 2, h[2]);
            if (n + 3 < N) st_g<uint16_t>(p + 3, h[3]);
        }
    }
}

// Lane -> C coordinates of accumulator group g (4 consecutive columns) of one
// MFMA tile, relative to the tile's corner (operands issued as Bt * At).
template <int MI>
__device__ __forceinline__ void acc_coord(int lane, int g, int& dm, int& dn)
{
    if (MI == 16) {
        dm = lane % 16;
        dn = 4 * (lane / 16);
    } else {
        dm = lane % 32;
        dn = 8 * g + 4 * (lane / 32);
    }
}

// Kernel arguments, all in SGPRs from the first instructions on.  Left to
// itself the compiler sinks each kernarg load next to its first use and
// waits for each batch in turn; the argument block is not cached at kernel
// start, so every batch costs a memory round trip before the first operand
// load can be issued.  Pinning every field at entry issues all the loads
// together and waits once.
// KROT: the kernel also reads krot.
template <bool KROT = false>
__device__ __forceinline__ VxGemmArgs pin_args(const VxGemmArgs& in)
{
    VxGemmArgs p = in;
    if constexpr (KROT)
        asm volatile("" : "+s"(p.A), "+s"(p.B), "+s"(p.C), "+s"(p.sA), "+s"(p.sB), "+s"(p.sC), "+s"(p.M), "+s"(p.N),
                          "+s"(p.K), "+s"(p.tiles_m), "+s"(p.tiles_n), "+s"(p.split), "+s"(p.k_per_split),
                          "+s"(p.batch), "+s"(p.group_m), "+s"(p.num_xcd), "+s"(p.grid), "+s"(p.dp_tiles),
                          "+s"(p.ws), "+s"(p.tickets), "+s"(p.krot));
    else
        asm volatile("" : "+s"(p.A), "+s"(p.B), "+s"(p.C), "+s"(p.sA), "+s"(p.sB), "+s"(p.sC), "+s"(p.M), "+s"(p.N),
                          "+s"(p.K), "+s"(p.tiles_m), "+s"(p.tiles_n), "+s"(p.split), "+s"(p.k_per_split),
                          "+s"(p.batch), "+s"(p.group_m), "+s"(p.num_xcd), "+s"(p.grid), "+s"(p.dp_tiles),
                          "+s"(p.ws), "+s"(p.tickets));
    asm volatile("" : "+s"(p.xq), "+s"(p.xr), "+s"(p.xq_dp), "+s"(p.xr_dp), "+s"(p.f_xcd.m), "+s"(p.f_xcd.s),
                      "+s"(p.f_tiles.m), "+s"(p.f_tiles.s), "+s"(p.f_split.m), "+s"(p.f_split.s), "+s"(p.f_rt.m),
                      "+s"(p.f_rt.s), "+s"(p.f_group.m), "+s"(p.f_group.s), "+s"(p.f_gm.m), "+s"(p.f_gm.s),
                      "+s"(p.f_gm_last.m), "+s"(p.f_gm_last.s));
    return p;
}

// The convolution's shape arguments, pinned like the others (conv kernels).
__device__ __forceinline__ void pin_conv(VxGemmArgs& p)
{
    asm volatile("" : "+s"(p.cH), "+s"(p.cW), "+s"(p.cC), "+s"(p.cKW), "+s"(p.cOH), "+s"(p.cOW), "+s"(p.csh),
                      "+s"(p.csw), "+s"(p.cph), "+s"(p.cpw), "+s"(p.cdh), "+s"(p.cdw));
}

// ---------------------------------------------------------- level 2 -------
// Grid level: the parallel loop over (batch, K slice, tile) of one launch.
// split is the number of K slices of this workgroup's tile (1 for a whole
// tile of a hybrid grid) and rid the tile's index among the split tiles (its
// slot in the split-K workspace and arrival counters).
struct GridPos {
    int b, z, tm, tn, m0, n0, kbeg, kend, nk, tiles, split, rid;
};

// x / d for 0 <= x < 2^31, with f = vx_fastdiv_make(d) (see vx_args.h).
__device__ __forceinline__ int fdiv(int x, VxFastDiv f)
{
    return (int)((__umulhi((unsigned)x, f.m) + (unsigned)x) >> f.s);
}

template <int MB, int NB, int KB>
__device__ __forceinline__ GridPos grid_pos(const VxGemmArgs& p)
{
    // Workgroups are dispatched round-robin over the XCDs; remap the linear id
    // so that each XCD receives a contiguous range of logical tiles
    // (neighbouring tiles share A or B panels in that XCD's L2).  Every
    // quotient below divides by a launch constant through its host-made
    // multiplier (fdiv).
    const int w = blockIdx.x;
    const int nx = p.num_xcd;
    GridPos g;
    g.tiles = p.tiles_m * p.tiles_n;
    int tile;
    bool whole = false;
    if (p.dp_tiles == 0) {
        // plain grid: every tile in split slices; grid = xq * nx + xr
        const int wq = fdiv(w, p.f_xcd), xcd = w - wq * nx;
        const int wl = xcd * p.xq + (xcd < p.xr ? xcd : p.xr) + wq;
        const int bz = fdiv(wl, p.f_tiles);
        tile = wl - bz * g.tiles;
        const int b = fdiv(bz, p.f_split);
        g.z = bz - b * p.split;
        g.b = b;
        g.split = p.split;
    } else {
        // hybrid grid: its two classes of workgroups -- the whole tiles
        // [0, dp_tiles), dispatched first, and the split tiles' slices after
        // them -- are remapped each on its own; dp_tiles is a multiple of
        // num_xcd, so a workgroup's XCD is its index within the class modulo
        // num_xcd as well
        whole = w < p.dp_tiles;
        const int wc = whole ? w : w - p.dp_tiles;
        const int q = whole ? p.xq_dp : p.xq, rem = whole ? p.xr_dp : p.xr;
        const int wq = fdiv(wc, p.f_xcd), xcd = wc - wq * nx;
        const int wl = xcd * q + (xcd < rem ? xcd : rem) + wq;
        const int rt = p.batch * g.tiles - p.dp_tiles;   // tiles that are split
        const int zq = fdiv(wl, p.f_rt), rr = wl - zq * rt;
        const int T = whole ? wl : p.dp_tiles + rr;
        g.z = whole ? 0 : zq;
        g.b = fdiv(T, p.f_tiles);
        tile = T - g.b * g.tiles;
        g.split = whole ? 1 : p.split;
        g.rid = whole ? 0 : rr;
    }
    // grouped order: group_m tile rows are walked column by column
    const int per_group = p.group_m * p.tiles_n;
    const int grp = fdiv(tile, p.f_group);
    const int r = tile - grp * per_group;
    const int first_m = grp * p.group_m;
    const bool full = p.tiles_m - first_m >= p.group_m;
    const int gm = full ? p.group_m : p.tiles_m - first_m;
    const int tn = fdiv(r, full ? p.f_gm : p.f_gm_last);
    g.tm = first_m + (r - tn * gm);
    g.tn = tn;
    g.m0 = g.tm * MB;
    g.n0 = g.tn * NB;
    if (p.dp_tiles == 0)
        g.rid = g.b * g.tiles + g.tm * p.tiles_n + g.tn;
    g.kbeg = whole ? 0 : g.z * p.k_per_split;
    g.kend = whole ? p.K : min(p.K, g.kbeg + p.k_per_split);
    g.nk = g.kend > g.kbeg ? (g.kend - g.kbeg + KB - 1) / KB : 0;
    return g;
}

template <class C>
__device__ __forceinline__ void acc_zero(Acc<C>& acc)
{
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
            for (int e = 0; e < C::ACC; ++e)
                acc.v[fn][fm][e] = 0.0f;
}

// ------------------------------------------------------------ Store_Func ---
// Split-K reduction of one output tile whose fp32 values are held by the first
// `nact` threads of the workgroup, V groups of 4 per thread.  Each slice
// publishes its partial tile, then the last slice to arrive sums all slices
// in order 0..split-1.  Returns false for a slice that is not the last to
// arrive (it has nothing more to do), true for the workgroup that now holds
// the tile's full sum in v.  The result is uniform over the workgroup.
// Partials move as 16-byte device-coherent (sc1) buffer stores and loads,
// laid out [slice][group of 4][thread] so each wave instruction covers 1 KiB
// contiguously; no workgroup has to write back or invalidate a whole L2.
template <int V>
__device__ __forceinline__ bool split_reduce(const VxGemmArgs& p, const GridPos& g, f32x4 (&v)[V], int t, int nact)
{
    const unsigned SLICE_BYTES = (unsigned)V * (unsigned)nact * 16u;
    const int64_t tile_id = g.rid;
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(p.ws + tile_id * (int64_t)g.split * (V * nact * 4)), (short)0, (int)(SLICE_BYTES * g.split), 0x00020000);
    constexpr int SC1 = 16;   // cache policy: device scope
    const bool act = t < nact;
    const unsigned mine = (unsigned)g.z * SLICE_BYTES;
    if (act) {
#pragma unroll
        for (int e4 = 0; e4 < V; ++e4)
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v[e4]), rw,
                                                   mine + (unsigned)(e4 * nact + t) * 16, 0, SC1);
    }
    // every store of the partial tile has completed before the arrival is counted
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    __shared__ unsigned arrived;
    if (t == 0)
        arrived = __hip_atomic_fetch_add(&p.tickets[tile_id], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (arrived != (unsigned)(g.split - 1))
        return false;
    // Sum slices 0..split-1 in order.  The loads of SF slices are issued
    // together before any of them is added, so the reduction waits for one
    // memory round trip per SF slices rather than one per slice (the last
    // slice's own partial is read back like the others: it is complete).
    if (act) {
        constexpr int SF = V <= 2 ? 8 : V <= 4 ? 4 : V <= 8 ? 2 : 1;
        f32x4 sum[V];
        for (int zz0 = 0; zz0 < g.split; zz0 += SF) {
            f32x4 part[SF][V];
#pragma unroll
            for (int j = 0; j < SF; ++j) {
                const int zz = min(zz0 + j, g.split - 1);   // in range; surplus loads are not added
#pragma unroll
                for (int e4 = 0; e4 < V; ++e4)
                    part[j][e4] = __builtin_bit_cast(
                        f32x4, __builtin_amdgcn_raw_buffer_load_b128(rw, zz * SLICE_BYTES + (unsigned)(e4 * nact + t) * 16,
                                                                     0, SC1));
            }
#pragma unroll
            for (int j = 0; j < SF; ++j) {
                if (zz0 + j >= g.split)
                    break;
#pragma unroll
                for (int e4 = 0; e4 < V; ++e4)
                    sum[e4] = zz0 + j == 0 ? part[j][e4] : sum[e4] + part[j][e4];
            }
        }
#pragma unroll
        for (int e4 = 0; e4 < V; ++e4)
            v[e4] = sum[e4];
    }
    if (t == 0)
        __hip_atomic_store(&p.tickets[tile_id], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return true;
}

// Split-K reduction of the MFMA accumulators (every thread holds
// FN x FM x ACC values, in groups of 4 along the accumulator index).
template <class C>
__device__ __forceinline__ bool reduce_split(const VxGemmArgs& p, Acc<C>& acc, const GridPos& g, int t)
{
    constexpr int P4 = C::FN * C::FM * C::ACC / 4;
    static_assert(C::ACC % 4 == 0, "accumulators come in groups of 4");
    f32x4 v[P4];
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
            for (int gi = 0; gi < C::ACC / 4; ++gi) {
                const int e4 = (fn * C::FM + fm) * (C::ACC / 4) + gi;
                v[e4] = f32x4{acc.v[fn][fm][4 * gi], acc.v[fn][fm][4 * gi + 1], acc.v[fn][fm][4 * gi + 2],
                              acc.v[fn][fm][4 * gi + 3]};
            }
    if (!split_reduce<P4>(p, g, v, t, C::NT))
        return false;
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
            for (int gi = 0; gi < C::ACC / 4; ++gi) {
                const int e4 = (fn * C::FM + fm) * (C::ACC / 4) + gi;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    acc.v[fn][fm][4 * gi + e] = v[e4][e];
            }
    return true;
}

// The epilogue straight from the accumulators: fp32 -> output type (round to
// nearest even) -> each lane's 4 consecutive columns of one row as one store.
template <class C>
__device__ __forceinline__ void store_direct(const VxGemmArgs& p, Acc<C>& acc, const GridPos& g, int lane, int wm0,
                                             int wn0)
{
    char* Cb = (char*)p.C + (int64_t)g.b * p.sC * C::EB;
    constexpr int NG = C::ACC / 4;
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
            for (int gi = 0; gi < NG; ++gi) {
                int dm, dn;
                acc_coord<C::MI>(lane, gi, dm, dn);
                const int m = g.m0 + wm0 + fm * C::MI + dm;
                const int n = g.n0 + wn0 + fn * C::MI + dn;
                if (m < p.M)
                    store4<C::DT>(Cb, (int64_t)m * p.N + n, n, p.N,
                                  acc.v[fn][fm][4 * gi], acc.v[fn][fm][4 * gi + 1],
                                  acc.v[fn][fm][4 * gi + 2], acc.v[fn][fm][4 * gi + 3]);
            }
}

// Four fp32 values -> four 16-bit outputs (round to nearest even), packed.
template <int DT>
__device__ __forceinline__ u32x2 pack4_16(float a0, float a1, float a2, float a3)
{
    unsigned h0, h1, h2, h3;
    if (DT == DT_F16) {
        h0 = __builtin_bit_cast(uint16_t, (_Float16)a0);
        h1 = __builtin_bit_cast(uint16_t, (_Float16)a1);
        h2 = __builtin_bit_cast(uint16_t, (_Float16)a2);
        h3 = __builtin_bit_cast(uint16_t, (_Float16)a3);
    } else {
        h0 = __builtin_bit_cast(uint16_t, (__bf16)a0);
        h1 = __builtin_bit_cast(uint16_t, (__bf16)a1);
        h2 = __builtin_bit_cast(uint16_t, (__bf16)a2);
        h3 = __builtin_bit_cast(uint16_t, (__bf16)a3);
    }
    return u32x2{pack2(h0, h1), pack2(h2, h3)};
}

// The epilogue through LDS.  The finished tile is written to the idle LDS
// (converted to the output type, rows padded by 16 bytes against bank
// conflicts), then leaves as 16-byte chunks of whole rows taken by
// consecutive threads: a wave's store covers whole 128-byte lines instead of
// 8 or 16 bytes in each of 16 or 32 rows.  Only the chunk that straddles the
// N edge is stored element by element; rows of any alignment take misaligned
// 16-byte stores.  Every wave must be done reading `buf` when this starts.
template <class C>
__device__ __forceinline__ void store_lds(const VxGemmArgs& p, Acc<C>& acc, const GridPos& g, int t, int lane, int wm0,
                                          int wn0, lds_char* buf)
{
    constexpr int EB = C::EB, VE = 16 / EB, LDC = C::LDC;
    static_assert(LDC * EB % 16 == 0, "16-byte aligned LDS rows");
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
            for (int gi = 0; gi < C::ACC / 4; ++gi) {
                int dm, dn;
                acc_coord<C::MI>(lane, gi, dm, dn);
                const int r = wm0 + fm * C::MI + dm, c = wn0 + fn * C::MI + dn;
                lds_char* dst = buf + (r * LDC + c) * EB;
                const float a0 = acc.v[fn][fm][4 * gi], a1 = acc.v[fn][fm][4 * gi + 1];
                const float a2 = acc.v[fn][fm][4 * gi + 2], a3 = acc.v[fn][fm][4 * gi + 3];
                if constexpr (EB == 2)
                    *(lds_u32x2*)dst = pack4_16<C::DT>(a0, a1, a2, a3);
                else
                    *(lds_u32x4*)dst = __builtin_bit_cast(u32x4, f32x4{a0, a1, a2, a3});
            }
    __syncthreads();
    constexpr int CPR = C::NB / VE, CHUNKS = C::MB * CPR;
    char* Cb = (char*)p.C + (int64_t)g.b * p.sC * EB;
#pragma unroll
    for (int j = 0; j < (CHUNKS + C::NT - 1) / C::NT; ++j) {
        const int i = t + j * C::NT;
        if (CHUNKS % C::NT != 0 && i >= CHUNKS)
            break;
        const int r = i / CPR, c = i % CPR;
        const int m = g.m0 + r, n = g.n0 + c * VE;
        if (m >= p.M || n >= p.N)
            continue;
        const u32x4 v = *(lds_u32x4*)(buf + (r * LDC + c * VE) * EB);
        char* dst = Cb + ((int64_t)m * p.N + n) * EB;
        if (n + VE <= p.N) {
            st_g<u32x4_u>(dst, v);
        } else {
#pragma unroll
            for (int e = 0; e < VE; ++e)
                if (n + e < p.N) {
                    if constexpr (EB == 2)
                        st_g<uint16_t>(dst + 2 * e, (uint16_t)elem16(v, e));
                    else
                        st_g<unsigned>(dst + 4 * e, v[e]);
                }
        }
    }
}

// ------------------------------------------------- register-staged family --
// Level 1 with loads staged through VGPRs (any dtype; 16-bit B is transposed
// in registers on its way into LDS).
// Per-thread im2col state of a convolution's A operand (the implicit GEMM's
// M x K matrix, row m = output pixel (n, oh, ow), column k = (kh, kw, ci) of
// the KH x KW x Cin filter).  A thread loads the same chunk column c of every
// K step in AV rows; the row part of each address (image n, top-left tap
// ih0, iw0) is fixed for the whole kernel and computed once, and the column
// part (ci, kw, kh of the chunk's first k) advances by KB per step.  Rows past
// M get ih0 = -2^30, so that every tap of theirs tests out of range (the
// host keeps H + 2 pad and W + 2 pad below 2^30, hence also the filter span
// of any convolution with a non-empty output).
template <class C>
struct ConvA {
    static constexpr int CPR = C::KB / C::VE;   // chunks per row of a K step
    static_assert(!C::CONV || C::NT % CPR == 0, "a thread's chunk column is the same in each of its rows");
    int64_t pix[C::AV];                         // element offset of (n, ih0, iw0), may be negative
    int ih0[C::AV], iw0[C::AV];
    int gk, ci, kw, kh;                         // first k of the chunk, and its (ci, kw, kh)

    __device__ __forceinline__ void init(const VxGemmArgs& p, int m0, int kbeg, int t)
    {
#pragma unroll
        for (int v = 0; v < C::AV; ++v) {
            const int gm = m0 + (t + v * C::NT) / CPR;
            const int ow = gm % p.cOW, q = gm / p.cOW;
            const int oh = q % p.cOH, n = q / p.cOH;
            const bool in = gm < p.M;
            ih0[v] = in ? oh * p.csh - p.cph : -(1 << 30);
            iw0[v] = in ? ow * p.csw - p.cpw : 0;
            pix[v] = (((int64_t)n * p.cH + ih0[v]) * p.cW + iw0[v]) * p.cC;
        }
        gk = kbeg + (t % CPR) * C::VE;
        decompose(p);
    }
    __device__ __forceinline__ void decompose(const VxGemmArgs& p)
    {
        ci = gk % p.cC;
        const int khw = gk / p.cC;
        kw = khw % p.cKW;
        kh = khw / p.cKW;
    }
    // on to the next K step
    __device__ __forceinline__ void advance(const VxGemmArgs& p)
    {
        gk += C::KB;
        if (C::KB <= p.cC) {                    // wave-uniform; one wrap at most
            ci += C::KB;
            if (ci >= p.cC) {
                ci -= p.cC;
                if (++kw == p.cKW) {
                    kw = 0;
                    ++kh;
                }
            }
        } else {
            decompose(p);
        }
    }
};

template <class C>
__device__ __forceinline__ void gemm_body(const VxGemmArgs& args)
{
    VxGemmArgs p = pin_args(args);
    if constexpr (C::CONV)
        pin_conv(p);
    __shared__ __attribute__((aligned(16))) char smem[C::LDS_BYTES];

    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const GridPos g = grid_pos<C::MB, C::NB, C::KB>(p);

    const char* Ab = (const char*)p.A + ((int64_t)g.b * p.sA + (int64_t)g.m0 * p.K) * C::EB;
    const char* Bb = (const char*)p.B + (int64_t)g.b * p.sB * C::EB;
    const int Mrel = p.M - g.m0;
    const int wm0 = (wave % C::WM) * C::MW, wn0 = (wave / C::WM) * C::NW;

    Acc<C> acc;
    acc_zero<C>(acc);

    // PF register sets: set j holds K steps j, j + PF, j + 2 PF, ... on their
    // way from memory into the LDS stage; the loop is unrolled by PF so that
    // every set index is a constant
    Tile<C> tl[C::PF];
    ConvA<C> ca;
    if constexpr (C::CONV)
        ca.init(p, g.m0, g.kbeg, t);
    // one K step of A and B into register set s (for a convolution, A through
    // the im2col map; the steps are loaded in order, so its state just advances)
    auto load = [&](Tile<C>& s, int k0) {
        s.load(Ab, Bb, 0, g.n0, k0, g.kend, Mrel, p.N, p.K, t);
        if constexpr (C::CONV) {
            s.load_a_conv(p, (const char*)p.A, ca, g.kend);
            ca.advance(p);
        }
    };
#pragma unroll
    for (int j = 0; j < C::PF; ++j)
        if (j < g.nk)
            load(tl[j], g.kbeg + j * C::KB);
    if (g.nk > 0)
        tl[0].store(smem, t);
    __syncthreads();
    for (int it0 = 0; it0 < g.nk; it0 += C::PF) {
#pragma unroll
        for (int j = 0; j < C::PF; ++j) {
            const int it = it0 + j;
            if (it >= g.nk)
                break;
            char* cur = smem + (it & 1) * C::STAGE_BYTES;
            // set j held step it, already in LDS: it takes step it + PF
            if (it + C::PF < g.nk)
                load(tl[j], g.kbeg + (it + C::PF) * C::KB);
            compute_step<C>(cur, acc, wm0, wn0, lane);
            if (it + 1 < g.nk)
                tl[(j + 1) % C::PF].store(smem + ((it + 1) & 1) * C::STAGE_BYTES, t);
            __syncthreads();
        }
    }
    // the loop ends with a barrier: LDS is idle here
    if (g.split > 1 && !reduce_split<C>(p, acc, g, t))
        return;
    if constexpr (C::LDS_EPI)
        store_lds<C>(p, acc, g, t, lane, wm0, wn0, (lds_char*)smem);
    else
        store_direct<C>(p, acc, g, lane, wm0, wn0);
}

}  // namespace vxk
