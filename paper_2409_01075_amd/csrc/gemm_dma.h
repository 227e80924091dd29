// Direct-to-LDS family for fp16/bf16 (gfx950).
//
// Level 1 (workgroup) loads its A and B tiles with buffer loads that write
// LDS directly (no VGPR staging, no VALU), into a ring of STAGES LDS stages,
// so up to STAGES-1 K steps are in flight while the MFMAs consume the oldest.
// Out-of-range rows, columns and K tails are given an out-of-range buffer
// offset: the hardware returns zeros for them, which land in LDS as padding.
// Each lane moves one 16-byte chunk, so a DMA'd operand's rows must be 16-byte
// aligned (K for A, N for B a multiple of 8, aligned bases).  Mixed kernels
// (VG) move one operand whose rows are not aligned through VGPRs into the same
// LDS layout; GEMMs with neither operand aligned use the register-staged
// family (a 2-byte buffer-to-LDS load fills a whole LDS dword per lane, which
// cannot build a dense 16-bit tile).  Three level-1 schedules: the plain ring
// (every wave issues its share of each K step), ping-pong (PP: the two halves
// of the waves take turns issuing whole K steps) and mixed (VG).
//
// K order (plain ring, GEMM only; the host sets krot when one batch entry's A
// and B fit in an XCD's L2): a tile takes its slice's K steps starting at step
// (tm + tn) mod nk, wrapping around.  The tiles resident at one time on an XCD
// share A row panels and B column panels; walked in lockstep, every one of them
// asks the L2 for the same lines at the same moment.  With the operands
// resident, rotating the start spreads those requests over the panels' K
// extent.  Larger operands stream through the L2, and there the lockstep is
// what lets one tile's miss serve its neighbours, so they keep the in-order
// walk.  Only the order of the fp32 accumulation changes, and it is a fixed
// function of the tile.
//
// LDS layouts (dense, 16-byte chunks XOR-swizzled against bank conflicts):
//   As[m][k]  Mb x Kb, k contiguous   (chunk c of row m stored at c ^ swzA(m))
//   Bs[k][n]  Kb x Nb, n contiguous   (chunk c of row k stored at c ^ swzB(k);
//                                     within groups of 8 chunks in rows of 24)
// B stays in its natural n-contiguous layout; the MFMA fragments of B are
// read with the transposing LDS read: in each 16-lane group, source lane s
// points at Bs[k0 + s/4][n0 + 4*(s%4)], and output lane j receives
// Bs[k0 + e][n0 + j] for e = 0..3 — four consecutive k of column j.
#pragma once
#include "gemm_kernel.h"

namespace vxk {

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

template <int DT_, int MB_, int NB_, int KB_, int WM_, int WN_, int MI_, int ST_, bool VEC_, bool CONV_ = false,
          bool PP_ = false, int VG_ = 0, bool FITC_ = false>
struct DCfg {
    static constexpr int DT = DT_, MB = MB_, NB = NB_, KB = KB_, WM = WM_, WN = WN_, MI = MI_, STAGES = ST_;
    static constexpr bool VEC = VEC_;
    static constexpr bool CONV = CONV_;   // A is an image read through the im2col map
    // ping-pong issue: the waves [0, 4) and [4, 8) -- one per SIMD each -- take
    // turns issuing a whole K step; the other half starts its MFMAs at once
    static constexpr bool PP = PP_;
    // operand moved through VGPRs instead of DMA (its rows need not be 16-byte
    // aligned): 0 none, 1 A, 2 B
    static constexpr int VG = VG_;
    static constexpr bool DMA_A = VG != 1, DMA_B = VG != 2;
    // LDS sized for the staged C tile as well as for the ring (short-K tiles
    // whose ring alone is smaller than their C tile keep the LDS epilogue)
    static constexpr bool FIT_C = FITC_;
    static constexpr bool H = true;
    static constexpr int EB = 2;
    static constexpr int NWAVE = WM * WN, NT = NWAVE * 64;
    static constexpr int MW = MB / WM, NW = NB / WN;
    static constexpr int FM = MW / MI, FN = NW / MI;
    static constexpr int ACC = MI == 16 ? 4 : 16;
    static constexpr int KI = MI == 16 ? 32 : 16;
    static constexpr int A_BYTES = MB * KB * 2, B_BYTES = KB * NB * 2;
    static constexpr int CPA_ = KB / 8, CPB_ = NB / 8;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    static constexpr int RING_BYTES = STAGES * STAGE_BYTES;
    static constexpr int LDC = NB + 8;
    // the whole ring (with FIT_C, at least the staged C tile, MB x LDC)
    static constexpr int LDS_BYTES = FIT_C && MB * LDC * 2 > RING_BYTES ? MB * LDC * 2 : RING_BYTES;
    static constexpr int CPA = KB / 8, CPB = NB / 8;       // 16-byte chunks per row
    static constexpr int SWA = CPA < 16 ? CPA : 16;        // A swizzle period (rows)
    static constexpr int LANE_BYTES = 16;                  // bytes one lane moves per DMA instruction
    static constexpr int WAVE_BYTES = 64 * LANE_BYTES;
    static constexpr int A_IPW = DMA_A ? A_BYTES / WAVE_BYTES / NWAVE : 0;   // DMA instructions per wave per K step
    static constexpr int B_IPW = DMA_B ? B_BYTES / WAVE_BYTES / NWAVE : 0;
    // 16-byte chunks per thread of the operand moved through VGPRs
    static constexpr int VGC = VG == 1 ? MB * CPA_ / NT : VG == 2 ? KB * CPB_ / NT : 0;
    static constexpr int LPS = A_IPW + B_IPW;

    // With a ring of 3 or more stages the next K step's DMA is spread between
    // the MFMA steps (a step of slack hides its latency); a 2-stage ring needs
    // it issued whole right after the barrier, a full step before its use.
    static constexpr bool SPREAD_DMA = STAGES >= 3;
    // epilogue through LDS (store_lds) when the C tile fits the idle ring
    static constexpr bool LDS_EPI = MB * LDC * 2 <= LDS_BYTES;

    static_assert(VEC, "direct-to-LDS loads move 16-byte chunks");
    static_assert(MB % WM == 0 && NB % WN == 0 && MW % MI == 0 && NW % MI == 0, "tile hierarchy");
    static_assert(KB % KI == 0 && KB % 8 == 0 && NB % 8 == 0, "K step and chunking");
    static_assert(!DMA_A || (A_IPW >= 1 && A_IPW * WAVE_BYTES * NWAVE == A_BYTES), "A DMA must split evenly over waves");
    static_assert(!DMA_B || (B_IPW >= 1 && B_IPW * WAVE_BYTES * NWAVE == B_BYTES), "B DMA must split evenly over waves");
    static_assert(VG == 0 || (STAGES == 2 && (!CONV || VG == 1) && !PP && VGC >= 1 &&
                              VGC * NT == (VG == 1 ? MB * CPA : KB * CPB)),
                  "an operand through VGPRs: 2-stage ring, chunks split evenly over the threads (a convolution's "
                  "image only)");
    static_assert(STAGES >= 2 && STAGES <= 16, "pipeline depth");
    static_assert((STAGES - 1) * LPS <= 63, "vmcnt range: the prologue's DMA all in flight");
    static_assert(LDS_BYTES <= 159 * 1024, "LDS budget of one CU, less 1 KiB for the split-K flag");
    static_assert(!CONV || CPA == 8, "convolution: one 128-byte row segment per 8 lanes (Kb = 64)");
    static_assert(!PP || (NWAVE == 8 && STAGES == 2 && !CONV && 2 * LPS <= 63 && (A_BYTES / WAVE_BYTES) % 4 == 0 &&
                          (B_BYTES / WAVE_BYTES) % 4 == 0),
                  "ping-pong: 8 waves, a 2-stage ring, K steps split evenly over 4 issuing waves");
};

// The LDS serves 16-byte reads 16 lanes per pass and the transposing 8-byte
// reads 32 lanes per pass, each pass over a 256-byte window of banks; a
// fragment read is conflict-free when the lanes of one pass cover distinct
// 16-byte slots of that window.  The swizzles below place the chunks so.
//
// A rows hold CPA 16-byte chunks; chunk c of row m sits at c ^ swz_a(m).  An
// A fragment read takes one chunk from each of 16 consecutive rows: with
// 128-byte rows (CPA 8) two rows share a window, so the XOR runs over pairs
// of rows; with 256 bytes and more each row fills the window.  Convolution
// tiles keep a period of 8 rows, which their im2col DMA addressing assumes.
template <class C>
__device__ __forceinline__ int swz_a(int m)
{
    if constexpr (C::CONV)
        return m & 7;
    else if constexpr (C::CPA == 8)
        return (m >> 1) & 7;
    else
        return m & (C::SWA - 1);
}
// B rows hold CPB 16-byte chunks; logical chunk c of row k sits at position
// c ^ s(k) (an XOR is its own inverse), and in rows of 24 chunks (tiles 192
// wide) the XOR acts inside aligned groups of 8 chunks.  A pass of the
// transposing read covers 4 rows x 4 chunks (32 x 32 MFMA: rows k0..k0+3, 32
// columns) or 8 rows x 2 chunks (16 x 16 MFMA: rows k0..k0+3 and
// k0+8..k0+11, 16 columns); s(k) spreads those over the 16 slots of the
// window for each row width (rows 16 columns wide, 2 chunks, cannot be).
template <int CPB, int MI>
__device__ __forceinline__ int swz_b(int k)
{
    if constexpr ((CPB & (CPB - 1)) != 0)
        return swz_b<8, MI>(k);
    else if constexpr (MI == 32 && CPB >= 16)
        return 4 * (k & 3);
    else if constexpr (MI == 32 && CPB == 8)
        return 4 * ((k >> 1) & 1);
    else if constexpr (MI == 16 && CPB >= 16)
        return 2 * (k & 3) + 8 * ((k >> 3) & 1);
    else if constexpr (MI == 16 && CPB == 8)
        return 2 * ((k >> 1) & 1) + 4 * ((k >> 3) & 1);
    else if constexpr (MI == 16 && CPB == 4)
        return 2 * ((k >> 3) & 1);
    else
        return (2 * (k & 3)) & (CPB - 1);
}
template <int CPB, int MI>
__device__ __forceinline__ int b_pos(int c, int k)   // LDS position of logical chunk c of row k
{
    if constexpr ((CPB & (CPB - 1)) == 0)
        return c ^ swz_b<CPB, MI>(k);
    else
        return (c & ~7) | ((c & 7) ^ swz_b<CPB, MI>(k));
}
template <int CPB, int MI>
__device__ __forceinline__ int b_chunk(int pos, int k)   // logical chunk held at LDS position pos of row k
{
    return b_pos<CPB, MI>(pos, k);
}

// s_waitcnt vmcnt(n) for a compile-time n (expcnt and lgkmcnt left at max).
template <int N>
__device__ __forceinline__ void wait_vm()
{
    static_assert(N >= 0 && N <= 63, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Waits until at most min(r, R) K steps of LPS DMA instructions each are in
// flight (r >= 0 is wave-uniform; s_waitcnt takes only immediates).
template <int LPS, int R>
__device__ __forceinline__ void wait_steps(int r)
{
    if constexpr (R <= 0) {
        wait_vm<0>();
    } else {
        if (r >= R)
            wait_vm<R * LPS>();
        else
            wait_steps<LPS, R - 1>(r);
    }
}

constexpr unsigned kOOB = 0x80000000u;    // buffer offset beyond every resource's range

// One buffer-load-to-LDS instruction: lane i's LANE bytes from the buffer at
// byte offset voff land at LDS address dst + i*LANE (dst is wave-uniform and
// goes through M0, set in the same statement).  Issued as inline assembly so
// that the compiler does not add its own conservative waits for LDS DMA
// before every LDS read; the pipeline's explicit vmcnt waits order the DMA
// against the reads of each stage instead.  No compiler-managed value lives
// in M0 in these kernels (no LDS DMA builtins, no indirect register indexing).
// Raw buffer resource (stride 0) for a wave-uniform base address: offsets at
// or beyond num_records read as zero.  Every dword is made scalar explicitly.
__device__ __forceinline__ u32x4 buffer_rsrc(const void* base, unsigned num_records)
{
    const uint64_t a = (uint64_t)base;
    u32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane((unsigned)a);
    r[1] = __builtin_amdgcn_readfirstlane((unsigned)(a >> 32) & 0xffffu);
    r[2] = num_records;
    r[3] = 0x00020000u;
    return r;
}

template <int LANE>
__device__ __forceinline__ void dma_lds(const u32x4& r, lds_char* dst, unsigned voff)
{
    static_assert(LANE == 16, "16-byte chunks");
    const unsigned m0v = __builtin_amdgcn_readfirstlane((unsigned)(uintptr_t)dst);
    // the resource is wave-uniform; readfirstlane keeps it in SGPRs whatever
    // the compiler could prove about it (free when it is already scalar)
    const u32x4 rs = {(unsigned)__builtin_amdgcn_readfirstlane(r[0]), (unsigned)__builtin_amdgcn_readfirstlane(r[1]),
                      (unsigned)__builtin_amdgcn_readfirstlane(r[2]), (unsigned)__builtin_amdgcn_readfirstlane(r[3])};
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" ::"s"(m0v), "v"(voff), "s"(rs)
                 : "memory");
}

// Per-lane im2col state of a convolution's A for the direct-to-LDS loads.
// With Kb = 64 the A instruction I of wave w moves row (w*A_IPW + I)*8 +
// lane/8 of the tile, always at chunk column (lane%8) ^ swizzle(lane/8): the
// column part of the map (ci, kw, kh of the chunk's first k) is shared by a
// lane's A_IPW rows and advances by Kb per K step; the row part (image n,
// top-left tap ih0, iw0) is fixed.  Element offsets are kept modulo 2^32:
// every tap that is loaded lies in the image, whose element count the host
// keeps below 2^30, so the wrapped sum of the row and column parts is exact
// there.  Rows past M get ih0 = -2^30 (every tap tests out of range; the
// host keeps H + 2 pad and W + 2 pad below 2^30).
template <class C>
struct DmaConvA {
    static constexpr int NA = C::A_IPW > 0 ? C::A_IPW : 1;
    unsigned pix[NA];   // element offset of (n, ih0, iw0), mod 2^32
    int ih0[NA], iw0[NA];
    int gk, ci, kw, kh;

    __device__ __forceinline__ void init(const VxGemmArgs& p, int m0, int kbeg, int wave, int lane)
    {
#pragma unroll
        for (int i = 0; i < C::A_IPW; ++i) {
            const int gm = m0 + (wave * C::A_IPW + i) * 8 + lane / 8;
            const int ow = gm % p.cOW, q = gm / p.cOW;
            const int oh = q % p.cOH, n = q / p.cOH;
            const bool in = gm < p.M;
            ih0[i] = in ? oh * p.csh - p.cph : -(1 << 30);
            iw0[i] = in ? ow * p.csw - p.cpw : 0;
            pix[i] = (((unsigned)n * (unsigned)p.cH + (unsigned)ih0[i]) * (unsigned)p.cW + (unsigned)iw0[i]) *
                     (unsigned)p.cC;
        }
        gk = kbeg + ((lane % 8) ^ ((lane / 8) % 8)) * 8;
        decompose(p);
    }
    __device__ __forceinline__ void decompose(const VxGemmArgs& p)
    {
        ci = gk % p.cC;
        const int khw = gk / p.cC;
        kw = khw % p.cKW;
        kh = khw / p.cKW;
    }
    __device__ __forceinline__ void advance(const VxGemmArgs& p)
    {
        gk += C::KB;
        if (C::KB <= p.cC) {   // wave-uniform; one wrap at most
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

template <class C, int NI = C::NWAVE>
struct DmaTile {
    // The DMA of one K step (starting at k0) into one LDS stage, issued by NI
    // waves: LPS instructions per wave, A's A_IPW first, then B's B_IPW.  A
    // step can be issued whole (issue) or one instruction at a time (one<I>),
    // so that the main loop can spread it between the MFMAs of the step being
    // computed.
    static constexpr int A_IPW = C::DMA_A ? C::A_BYTES / C::WAVE_BYTES / NI : 0;
    static constexpr int B_IPW = C::DMA_B ? C::B_BYTES / C::WAVE_BYTES / NI : 0;
    static constexpr int LPS = A_IPW + B_IPW;
    static_assert((!C::DMA_A || A_IPW * NI * C::WAVE_BYTES == C::A_BYTES) &&
                      (!C::DMA_B || B_IPW * NI * C::WAVE_BYTES == C::B_BYTES),
                  "the step splits evenly over the issuing waves");
    lds_char* stage;
    u32x4 ra, rb;   // A resource at column k0 of the panel; B resource at row k0, column n0
    int kv, nv;     // valid columns of A from k0; valid columns of B from n0
    // convolution: the image's resource in ra, and this step's column part of
    // the im2col map (filter row and column offsets, element offset mod 2^32)
    const DmaConvA<C>* cv = nullptr;
    int dh = 0, dw = 0, cH = 0, cW = 0;
    unsigned koff = 0;
    bool kin = false;

    __device__ __forceinline__ DmaTile(lds_char* stage_, const char* Apanel, const char* Bbatch, int k0, int kend, int n0,
                                       int N)
        : stage(stage_), ra(buffer_rsrc(Apanel + (int64_t)k0 * 2, kOOB)),
          rb(buffer_rsrc(Bbatch + ((int64_t)k0 * N + n0) * 2, kOOB)), kv(kend - k0), nv(N - n0)
    {
    }

    // Convolution step: A from the image X through the map state `c` (whose
    // column part describes this step's k0).
    __device__ __forceinline__ DmaTile(lds_char* stage_, const char* X, const char* Bbatch, int k0, int kend, int n0,
                                       const VxGemmArgs& p, const DmaConvA<C>& c)
        : stage(stage_), ra(buffer_rsrc(X, kOOB)), rb(buffer_rsrc(Bbatch + ((int64_t)k0 * p.N + n0) * 2, kOOB)),
          kv(kend - k0), nv(p.N - n0), cv(&c), dh(c.kh * p.cdh), dw(c.kw * p.cdw), cH(p.cH), cW(p.cW),
          koff(((unsigned)dh * (unsigned)p.cW + (unsigned)dw) * (unsigned)p.cC + (unsigned)c.ci), kin(c.gk < kend)
    {
    }

    template <int I>
    __device__ __forceinline__ void one(int Mrel, int N, int K, int wave, int lane) const
    {
        if constexpr (I < A_IPW && C::CONV) {
            // A: the taps of this lane's output pixel I at this step's columns
            const int instr = wave * A_IPW + I;
            const bool ok = kin && (unsigned)(cv->ih0[I] + dh) < (unsigned)cH && (unsigned)(cv->iw0[I] + dw) < (unsigned)cW;
            dma_lds<C::LANE_BYTES>(ra, stage + instr * C::WAVE_BYTES, ok ? (cv->pix[I] + koff) * 2u : kOOB);
        } else if constexpr (I < A_IPW) {
            // A: rows of the workgroup's panel
            const int instr = wave * A_IPW + I;
            const int slot = instr * 64 + lane;                  // chunk index in the stage
            const int r = slot / C::CPA, c = (slot % C::CPA) ^ swz_a<C>(r);
            const bool ok = r < Mrel && c * 8 < kv;
            dma_lds<C::LANE_BYTES>(ra, stage + instr * C::WAVE_BYTES, ok ? (unsigned)((r * K + c * 8) * 2) : kOOB);
        } else {
            // B: rows k0.. of the batch's B, columns from n0
            const int instr = wave * B_IPW + (I - A_IPW);
            const int slot = instr * 64 + lane;
            const int k = slot / C::CPB, c = b_chunk<C::CPB, C::MI>(slot % C::CPB, k);
            const bool ok = k < kv && c * 8 < nv;
            dma_lds<C::LANE_BYTES>(rb, stage + C::A_BYTES + instr * C::WAVE_BYTES,
                                   ok ? (unsigned)((k * N + c * 8) * 2) : kOOB);
        }
    }

    // instructions [FIRST, LAST) of the step
    template <int FIRST, int LAST>
    __device__ __forceinline__ void range(int Mrel, int N, int K, int wave, int lane) const
    {
        if constexpr (FIRST < LAST) {
            one<FIRST>(Mrel, N, K, wave, lane);
            range<FIRST + 1, LAST>(Mrel, N, K, wave, lane);
        }
    }

    __device__ __forceinline__ void issue(int Mrel, int N, int K, int wave, int lane) const
    {
        range<0, LPS>(Mrel, N, K, wave, lane);
    }
};

// The operand of a mixed kernel whose rows need not start on 16-byte
// boundaries moves through VGPRs: 16-byte row chunks, a chunk wholly inside
// its row as one (possibly misaligned) load, the chunk that straddles the
// row's valid end gathered element by element, rows out of range as zeros;
// then written to the LDS stage at the positions the DMA of an aligned operand
// would fill, so the fragment reads are the same.
template <class C>
struct VgOperand {
    u32x4 r[C::VGC > 0 ? C::VGC : 1];

    __device__ __forceinline__ static u32x4 gather(const char* p, int valid)
    {
        u32x4 x = {0, 0, 0, 0};
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
            const unsigned lo = e < valid ? (unsigned)ld_g<uint16_t>(p + 2 * e) : 0u;
            const unsigned hi = e + 1 < valid ? (unsigned)ld_g<uint16_t>(p + 2 * (e + 1)) : 0u;
            x[e >> 1] = pack2(lo, hi);
        }
        return x;
    }

    // the K step at k0: A rows of the panel (VG 1) or B rows k0.. from column n0 (VG 2)
    __device__ __forceinline__ void load(const char* Apanel, const char* Bbatch, int k0, int kend, int Mrel, int n0,
                                         int N, int K, int t)
    {
#pragma unroll
        for (int v = 0; v < C::VGC; ++v) {
            const int idx = t + v * C::NT;
            u32x4 x = {0, 0, 0, 0};
            if constexpr (C::VG == 1) {
                const int rr = idx / C::CPA, gk = k0 + (idx % C::CPA) * 8;
                if (rr < Mrel && gk < kend) {
                    const char* p = Apanel + ((int64_t)rr * K + gk) * 2;
                    x = gk + 8 <= kend ? ld_g<u32x4_u>(p) : gather(p, kend - gk);
                }
            } else {
                const int gk = k0 + idx / C::CPB, gn = n0 + (idx % C::CPB) * 8;
                if (gk < kend && gn < N) {
                    const char* p = Bbatch + ((int64_t)gk * N + gn) * 2;
                    x = gn + 8 <= N ? ld_g<u32x4_u>(p) : gather(p, N - gn);
                }
            }
            r[v] = x;
        }
    }

    // A convolution's A (VG 1): the K step at the chunk column held in the
    // im2col map state `ca`, gathered as the register-staged kernels do; a
    // thread's VGC chunks are rows (t + v NT) / CPA at chunk column t % CPA.
    template <class CA>
    __device__ __forceinline__ void load_conv(const VxGemmArgs& p, const char* X, const CA& ca, int kend)
    {
        static_assert(C::VG == 1 && C::CONV, "the image through VGPRs");
        conv_gather<CA, C::VGC, 8, true, 2>(p, X, ca, kend, r);
    }

    __device__ __forceinline__ void store(lds_char* stage, int t) const
    {
#pragma unroll
        for (int v = 0; v < C::VGC; ++v) {
            const int idx = t + v * C::NT;
            lds_char* dst;
            if constexpr (C::VG == 1) {
                const int rr = idx / C::CPA, c = idx % C::CPA;
                dst = stage + rr * (C::KB * 2) + ((c ^ swz_a<C>(rr)) << 4);
            } else {
                const int kk = idx / C::CPB, c = idx % C::CPB;
                dst = stage + C::A_BYTES + kk * (C::NB * 2) + (b_pos<C::CPB, C::MI>(c, kk) << 4);
            }
            *(lds_u32x4*)dst = r[v];
        }
    }
};

// The im2col map state of the register-staged kernels (ConvA) over the rows
// and the chunk column that the VGPR loads of a mixed convolution tile take.
template <class D>
struct VgConvView {
    static constexpr int KB = D::KB, VE = 8, NT = D::NT, AV = D::VGC;
    static constexpr bool CONV = true;
    static_assert(D::CPA == KB / VE, "a row of the K step is CPA chunks");
};

// Level 0 over one LDS stage.  The fragments of MFMA step kk+1 are read from
// LDS while the MFMAs of step kk run (two register sets), so the LDS latency
// and transfer overlap the matrix-core work instead of preceding it.
template <class C>
__device__ __forceinline__ void dma_frags(lds_char* stage, u32x4 (&fa)[C::FM], u32x4 (&fb)[C::FN], int kk, int wm0, int wn0,
                                          int lane)
{
    lds_char* As = stage;
    lds_char* Bs = stage + C::A_BYTES;
    const int li = lane % C::MI, lg = lane / C::MI;
    const int s = lane & 15, grp = lane >> 4;
    // transposing-read coordinates of this lane (see the header comment)
    const int tr_n = (C::MI == 16 ? 0 : 16 * (grp & 1)) + 4 * (s & 3);
    const int tr_k = (C::MI == 16 ? 8 * grp : 8 * (grp >> 1)) + (s >> 2);
#pragma unroll
    for (int fm = 0; fm < C::FM; ++fm) {
        const int m = wm0 + fm * C::MI + li;
        const int c = (kk * (C::KI / 8) + lg) ^ swz_a<C>(m);
        fa[fm] = *(lds_u32x4*)(As + m * (C::KB * 2) + c * 16);
    }
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn) {
        const int n = wn0 + fn * C::MI + tr_n;
        const int k1 = kk * C::KI + tr_k, k2 = k1 + 4;
        lds_char* p1 = Bs + k1 * (C::NB * 2) + (b_pos<C::CPB, C::MI>(n >> 3, k1) << 4) + (n & 7) * 2;
        lds_char* p2 = Bs + k2 * (C::NB * 2) + (b_pos<C::CPB, C::MI>(n >> 3, k2) << 4) + (n & 7) * 2;
        const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)p1);
        const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)p2);
        const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
        fb[fn] = u32x4{l2[0], l2[1], h2[0], h2[1]};
    }
}

// The MFMAs of one LDS stage; when `on`, the DMA `next` of a later K step is
// issued too: whole before the first MFMAs (2-stage rings), or in NKK parts,
// one after the MFMAs of each MFMA step (deeper rings), so that the CU's load
// path fills the ring while the matrix cores run.
template <int NKK, int KK, class C>
__device__ __forceinline__ void dma_part(const DmaTile<C>& next, bool on, int Mrel, int N, int K, int wave, int lane)
{
    constexpr int NP = C::SPREAD_DMA ? NKK : 1;   // MFMA steps the DMA is spread over
    constexpr int PER = (C::LPS + NP - 1) / NP;
    constexpr int FIRST = KK * PER < C::LPS ? KK * PER : C::LPS;
    constexpr int LAST = (KK + 1) * PER < C::LPS ? (KK + 1) * PER : C::LPS;
    if constexpr (FIRST < LAST) {
        if (on)
            next.template range<FIRST, LAST>(Mrel, N, K, wave, lane);
    }
}

template <class C, int KK = 0>
__device__ __forceinline__ void dma_steps(lds_char* stage, Acc<C>& acc, u32x4 (&fa)[2][C::FM], u32x4 (&fb)[2][C::FN], int wm0,
                                          int wn0, int lane, const DmaTile<C>& next, bool on, int Mrel, int N, int K,
                                          int wave)
{
    constexpr int NKK = C::KB / C::KI;
    if constexpr (KK < NKK) {
        if constexpr (KK + 1 < NKK)
            dma_frags<C>(stage, fa[(KK + 1) & 1], fb[(KK + 1) & 1], KK + 1, wm0, wn0, lane);
        // keep the reads of step KK+1 ahead of the MFMAs of step KK (the
        // machine scheduler would otherwise sink each read next to its use)
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (!C::SPREAD_DMA) {
            dma_part<NKK, KK, C>(next, on, Mrel, N, K, wave, lane);
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm) {
                if constexpr (C::MI == 16)
                    mfma16<C::DT, 16>(fb[KK & 1][fn], fa[KK & 1][fm], acc.v[fn][fm]);
                else
                    mfma32<C::DT>(fb[KK & 1][fn], fa[KK & 1][fm], acc.v[fn][fm]);
            }
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (C::SPREAD_DMA) {
            dma_part<NKK, KK, C>(next, on, Mrel, N, K, wave, lane);
            __builtin_amdgcn_sched_barrier(0);
        }
        dma_steps<C, KK + 1>(stage, acc, fa, fb, wm0, wn0, lane, next, on, Mrel, N, K, wave);
    }
}

template <class C>
__device__ __forceinline__ void dma_compute(lds_char* stage, Acc<C>& acc, int wm0, int wn0, int lane, const DmaTile<C>& next,
                                            bool on, int Mrel, int N, int K, int wave)
{
    u32x4 fa[2][C::FM], fb[2][C::FN];
    dma_frags<C>(stage, fa[0], fb[0], 0, wm0, wn0, lane);
    dma_steps<C>(stage, acc, fa, fb, wm0, wn0, lane, next, on, Mrel, N, K, wave);
}

template <class C>
__device__ __forceinline__ void gemm_dma_body(const VxGemmArgs& args)
{
    constexpr bool KROT = !C::CONV && !C::PP && C::VG == 0;   // kernels that may rotate their K order
    VxGemmArgs p = pin_args<KROT>(args);
    if constexpr (C::CONV)
        pin_conv(p);
    // The ring: STAGES stages of one K step each.  Stage indices are
    // compile-time constants in the unrolled main loop below.
    constexpr int SB = C::STAGE_BYTES;
    __shared__ __attribute__((aligned(1024))) char smem[C::LDS_BYTES];
#define VX_STAGE(j) ((lds_char*)smem + (j) * SB)

    const int t = threadIdx.x;
    const int lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    const GridPos g = grid_pos<C::MB, C::NB, C::KB>(p);

    const char* Apanel = (const char*)p.A + ((int64_t)g.b * p.sA + (int64_t)g.m0 * p.K) * 2;
    const char* Bbatch = (const char*)p.B + (int64_t)g.b * p.sB * 2;
    const int Mrel = p.M - g.m0;
    const int wm0 = (wave % C::WM) * C::MW, wn0 = (wave / C::WM) * C::NW;

    Acc<C> acc;
    acc_zero<C>(acc);

    // Only the slice's own K steps are issued: a DMA instruction costs issue
    // time even when all its offsets are out of range.  While the ring is
    // full, STAGES-2 steps stay in flight behind the one waited for; in the
    // last STAGES-2 iterations (the drain) the count falls to 0.
    // prologue: the first min(STAGES-1, nk) K steps, step s into stage s
    DmaConvA<C> cv;
    if constexpr (C::CONV && C::VG == 0)
        cv.init(p, g.m0, g.kbeg, wave, lane);
    // the DMA of the K step at k0 into stage st (for a convolution, at the
    // map state's step, which then moves on: steps are made in order)
    auto tile = [&](lds_char* st, int k0) {
        if constexpr (C::CONV) {
            const DmaTile<C> d(st, (const char*)p.A, Bbatch, k0, g.kend, g.n0, p, cv);
            cv.advance(p);
            return d;
        } else {
            return DmaTile<C>(st, Apanel, Bbatch, k0, g.kend, g.n0, p.N);
        }
    };
    int rot = 0;
    if constexpr (KROT)
        rot = p.krot != 0 && g.nk > 1 ? (g.tm + g.tn) % g.nk : 0;
    // K offset of the step the tile takes s-th: in order, or rotated by rot
    // (rc is std::true_type); a step s >= nk is never issued, any offset does
    auto kstep = [&](auto rc, int s) {
        if constexpr (decltype(rc)::value) {
            const int q = s + rot;
            return g.kbeg + (q >= g.nk ? q - g.nk : q) * C::KB;
        } else {
            return g.kbeg + s * C::KB;
        }
    };
    auto prologue = [&](auto rc) {
#pragma unroll
        for (int s = 0; s < C::STAGES - 1; ++s)
            if (s < g.nk)
                tile(VX_STAGE(s), kstep(rc, s)).issue(Mrel, p.N, p.K, wave, lane);
    };
    if constexpr (C::VG != 0 || C::PP)
        prologue(std::false_type{});
    if constexpr (C::VG != 0) {
        // Mixed (2 stages): the aligned operand by DMA, the other through VGPRs.
        // The VGPR loads of step it+1 fly with its DMA while step it computes,
        // then land in the free stage before the next barrier.
        VgOperand<C> vg;
        // a convolution's image goes through the im2col map, whose state
        // advances one K step per load (the steps come in order)
        ConvA<VgConvView<C>> ca;
        if constexpr (C::CONV)
            ca.init(p, g.m0, g.kbeg, t);
        auto vg_load = [&](int k0) {
            if constexpr (C::CONV) {
                vg.load_conv(p, (const char*)p.A, ca, g.kend);
                ca.advance(p);
            } else {
                vg.load(Apanel, Bbatch, k0, g.kend, Mrel, g.n0, p.N, p.K, t);
            }
        };
        const DmaTile<C> none(VX_STAGE(0), Apanel, Bbatch, g.kbeg, g.kend, g.n0, p.N);
        if (g.nk > 0) {
            vg_load(g.kbeg);
            wait_vm<0>();
            vg.store(VX_STAGE(0), t);
        }
        for (int it0 = 0; it0 < g.nk; it0 += 2) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int it = it0 + j;
                if (it >= g.nk)
                    break;
                wait_vm<0>();        // the DMA of step it has landed
                __syncthreads();     // ... and every wave's part of it, DMA and LDS writes; stage j ^ 1 is free
                const bool more = it + 1 < g.nk;
                if (more) {
                    const int k1 = g.kbeg + (it + 1) * C::KB;
                    DmaTile<C>(VX_STAGE(j ^ 1), Apanel, Bbatch, k1, g.kend, g.n0, p.N).issue(Mrel, p.N, p.K, wave, lane);
                    vg_load(k1);
                }
                __builtin_amdgcn_sched_barrier(0);
                dma_compute<C>(VX_STAGE(j), acc, wm0, wn0, lane, none, false, Mrel, p.N, p.K, wave);
                if (more) {
                    wait_vm<0>();
                    vg.store(VX_STAGE(j ^ 1), t);
                }
            }
        }
    } else if constexpr (C::PP) {
        // Ping-pong (2 stages): step 0 came from every wave above; then at
        // step it the half (wave >> 2) == it % 2 issues step it+1 whole into
        // the other stage while the other half starts its MFMAs right after
        // the barrier.  A wave waits only for what it issued itself.
        const DmaTile<C> none(VX_STAGE(0), Apanel, Bbatch, g.kbeg, g.kend, g.n0, p.N);
        for (int it0 = 0; it0 < g.nk; it0 += 2) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int it = it0 + j;
                if (it >= g.nk)
                    break;
                wait_vm<0>();                  // step it has landed (the part this wave issued, if any)
                __builtin_amdgcn_s_barrier();  // ... and every wave's; stage j ^ 1 is free
                if (it + 1 < g.nk && (wave >> 2) == j)
                    DmaTile<C, C::NWAVE / 2>(VX_STAGE(j ^ 1), Apanel, Bbatch, g.kbeg + (it + 1) * C::KB, g.kend, g.n0,
                                             p.N)
                        .issue(Mrel, p.N, p.K, wave & 3, lane);
                __builtin_amdgcn_sched_barrier(0);
                dma_compute<C>(VX_STAGE(j), acc, wm0, wn0, lane, none, false, Mrel, p.N, p.K, wave);
            }
        }
    } else {
        // the plain ring: prologue, then the main loop, unrolled by STAGES so
        // that every stage index is a constant.  The rotated and the in-order
        // walks are separate instances, so the in-order one carries no
        // rotation arithmetic.
        auto ring = [&](auto rc) {
            prologue(rc);
            for (int it0 = 0; it0 < g.nk; it0 += C::STAGES) {
#pragma unroll
                for (int j = 0; j < C::STAGES; ++j) {
                    const int it = it0 + j;
                    if (it >= g.nk)
                        break;
                    wait_steps<C::LPS, C::STAGES - 2>(g.nk - 1 - it);   // step `it` has landed (this wave's part)
                    __builtin_amdgcn_s_barrier();                      // ... and every wave's; stage it-1 is free
                    // step it+STAGES-1 goes into the freed stage, issued between the MFMAs of step it
                    const DmaTile<C> next =
                        tile(VX_STAGE((j + C::STAGES - 1) % C::STAGES), kstep(rc, it + C::STAGES - 1));
                    dma_compute<C>(VX_STAGE(j), acc, wm0, wn0, lane, next, it + C::STAGES - 1 < g.nk, Mrel, p.N,
                                   p.K, wave);
                }
            }
        };
        if constexpr (KROT) {
            if (rot != 0)
                ring(std::true_type{});
            else
                ring(std::false_type{});
        } else {
            ring(std::false_type{});
        }
    }
    wait_vm<0>();   // nothing is in flight here; kept as a guard before LDS is released
#undef VX_STAGE
    if (g.split > 1 && !reduce_split<C>(p, acc, g, t))
        return;
    if constexpr (C::LDS_EPI) {
        __syncthreads();   // every wave has finished reading the ring
        store_lds<C>(p, acc, g, t, lane, wm0, wn0, (lds_char*)smem);
    } else {
        store_direct<C>(p, acc, g, lane, wm0, wn0);
    }
}

}  // namespace vxk
