// Runtime strategy selection (Section 5.2 and Section 6.2): an analytical cost
// model evaluated per call over the precompiled candidates, with no profiling
// and no shape samples.
//
// Cost of one candidate, bottom-up through the levels of the hierarchy:
//   level 0 (wavefront)  temporal loop over the Kb/k0 MFMA steps of one K step:
//                        T_Load  = fragment bytes read from LDS / LDS share,
//                        Cost_-1 = MFMA time of the wavefronts' tiles,
//                        no store (accumulators stay in registers)       Eq. 2
//   level 1 (workgroup)  temporal loop over the n_k K steps of one slice:
//                        T_Load  = load latency + tile bytes / L2->CU share,
//                        Cost_0  = level-0 cost, T_Store = epilogue bytes
//                        (+ split-K partial traffic and arrival counter)   Eq. 2
//                        With an LDS ring of S stages, S-1 K steps are in
//                        flight: after the first step, a new step is ready
//                        every max(transfer, T_Load / (S-1)); Eq. 2 is this
//                        with S = 2.
//   level 2 (grid)       parallel loop over tiles x slices x batch:
//                        F = ceil(workgroups / (CUs x resident WGs per CU)) Eq. 3
//                        Cost_2 = F x T_temporal(level 1)                  Eq. 4
// The call's cost adds the dispatch constant and is floored by the
// compulsory HBM traffic at peak bandwidth.  The plan is the argmin (Eq. 1).
//
// Hybrid analyzer (Section 5.2): when an offline calibration of the kernels
// is loaded, the low levels are empirical — each kernel's measured time per
// workgroup K step and fixed cost (with the device fully loaded and lightly
// loaded) replace the analytical level-0/level-1 estimate — and the grid
// level stays analytical: F - 1 full waves of workgroups plus a last, partial
// wave whose per-step time is interpolated by its load (Eq. 3, Eq. 4).
#include <math.h>

#include <alloca.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <vector>

#include "vx_internal.h"

extern "C" double vx_cost_temporal(double t_load, int64_t trips, double cost_lower, double t_store)
{
    if (trips <= 0)
        return t_store;
    return t_load + (double)(trips - 1) * std::max(t_load, cost_lower) + cost_lower + t_store;
}

extern "C" int64_t vx_cost_parallel_factor(int64_t parallel, int64_t units)
{
    if (parallel < 0 || units < 1)
        return -1;
    return (parallel + units - 1) / units;
}

static int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

int vxi_group_m(int64_t tiles_m, int64_t tiles_n)
{
    // Walk 8 tile rows together when the grid is wide enough to need it.
    (void)tiles_n;
    return (int)std::max<int64_t>(1, std::min<int64_t>(8, tiles_m));
}

// Splits considered for K (the grid-level share of the reduction loop).
static const int kSplits[] = {1, 2, 3, 4, 5, 6, 8, 10, 12, 16, 20, 24, 32};

int vxi_occupancy(const vx_hwinfo& hw, const vx_kernel_info& k)
{
    // Resident workgroups per CU: the tighter of the LDS and register budgets.
    const int waves = k.wm * k.wn;
    const int regs = ((k.vgprs + 7) / 8) * 8 + ((k.agprs + 7) / 8) * 8;
    int waves_simd = regs > 0 ? hw.vgprs_per_lane / regs : hw.max_waves_per_simd;
    waves_simd = std::max(1, std::min(waves_simd, hw.max_waves_per_simd));
    const int by_regs = std::max(1, waves_simd * hw.simd_per_cu / waves);
    const int by_lds = std::max(1, hw.lds_bytes_per_cu / std::max(1, k.lds_bytes));
    return std::min(by_regs, by_lds);
}

namespace {

// The integer side of a plan: tile and slice counts, the grid's waves.
struct PlanInts {
    int64_t tiles, kps, nk, nk_whole, slots, dp, units_s, F, F_dp, per_cu;
};

// The checks of a plan that depend on the kernel beyond its workgroup tile
// and residency: the K extent its LDS may hold, and the 32-bit buffer offsets
// of its load family.
inline bool kernel_fits(const VxShape& sh, const vx_kernel_info& k, bool hyb, int64_t kps)
{
    if (k.k_max > 0 && (hyb ? sh.K : kps) > k.k_max)   // the kernel holds a whole slice of A in LDS
        return false;
    const int eb = sh.dt == VX_F32 ? 4 : 2;
    if (k.family == 1) {
        // direct-to-LDS kernels address each K step with 32-bit buffer offsets:
        // Mb rows of A (Mb*K elements) and Kb rows of B (Kb*N elements); a
        // convolution's A offsets run over the whole image
        const double a_span = k.op == 1 ? ((k.align & 1) ? (double)sh.a_bytes : 0.0) : (double)k.mb * sh.K * eb;
        if (a_span >= 2147483648.0 || (double)k.kb * sh.N * eb >= 2147483648.0)
            return false;
    }
    if (k.family == 2) {
        // the vector-ALU kernels address a whole slice of B with 32-bit offsets
        if ((double)(hyb ? sh.K : kps) * sh.N * eb >= 2147483648.0)
            return false;
    }
    return true;
}

// Checks that tiles x `split` slices are a feasible grid for the workgroup
// tile (mb, nb, kb) with `slots` resident workgroups on the device, and fills
// in the plan's integers (tiles, nk and nk_whole are given).  The same for
// every kernel of that tile and residency.  Returns false if infeasible.
inline bool grid_ints(const vx_hwinfo& hw, const VxShape& sh, int mb, int nb, int kb, int split, bool hyb,
                      const VxLimits& lim, int64_t slots, PlanInts* pi)
{
    const int64_t tiles = pi->tiles;
    int64_t kps = 0;
    if (sh.K != 0) {
        kps = pi->nk * kb;
        if ((int64_t)(split - 1) * kps >= sh.K)   // a slice would be empty
            return false;
    }
    if (kps > INT32_MAX || tiles > INT32_MAX)
        return false;
    const int64_t dp = hyb ? tiles / slots * slots : 0;   // whole tiles, in whole waves
    const int64_t split_tiles = tiles - dp;
    if (hyb && (dp == 0 || split_tiles == 0 || slots % std::max(1, hw.num_xcd) != 0))
        return false;   // (the kernels remap each class of workgroups over the XCDs on its own)
    const int64_t units = dp + split_tiles * split;
    if (units > INT32_MAX)
        return false;
    if (split > 1) {
        if (split_tiles > lim.max_tickets)
            return false;
        if ((double)split_tiles * split * mb * nb * 4.0 > (double)lim.ws_bytes)
            return false;
    }
    // Level 2: wave quantisation over the device (Eq. 3); a hybrid grid runs
    // dp / slots full waves of whole tiles, then the split tiles' slices.
    const int64_t units_s = hyb ? split_tiles * split : units;
    pi->kps = kps;
    pi->slots = slots;
    pi->dp = dp;
    pi->units_s = units_s;
    pi->F = vx_cost_parallel_factor(units_s, slots);
    pi->per_cu = cdiv(std::min(units_s, slots), hw.num_cu);
    pi->F_dp = dp / slots;
    return true;
}

// The cost (ns) of a feasible plan: empirical low levels when the kernel is
// calibrated (cb), else the analytical levels 0 and 1; the analytical grid
// level; the dispatch constant; the compulsory-traffic floor.
double plan_cost(const vx_hwinfo& hw, const VxShape& sh, const vx_kernel_info& k, int split, bool hyb,
                 const PlanInts& pi, const VxCalib* cb, int occ, double launch_cal, double floor_ns)
{
    const int eb = sh.dt == VX_F32 ? 4 : 2;
    const int waves = k.wm * k.wn;
    const int64_t nk = pi.nk, nk_whole = pi.nk_whole, F = pi.F, F_dp = pi.F_dp, slots = pi.slots;
    const double per_cu = (double)pi.per_cu;
    auto bw_wg_at = [&](double pc) { return hw.l2_bytes_clk_cu * hw.clock_ghz / pc; };   // B/ns, L2 -> one workgroup
    // split-K epilogue: the partial tile out, the arrival counter, and the
    // last arrival's reads of the other slices
    auto t_split_at = [&](double pc) {
        const double part = (double)k.mb * k.nb * 4.0 / bw_wg_at(pc);
        return split > 1 ? part + hw.atomic_latency_ns + hw.mem_latency_ns + (double)(split - 1) * part : 0.0;
    };

    if (cb) {
        // empirical low levels, analytical grid level
        double t_split;
        if (split > 1 && cb->split_a >= 0.0 && cb->split_b >= 0.0)
            t_split = cb->split_a + cb->split_b * (double)(split - 1);      // measured
        else
            t_split = t_split_at(per_cu);                                   // ... or analytical
        const double load_last = (double)(pi.units_s - (F - 1) * slots) / (double)slots;
        auto at_load = [&](double full, double light) {
            if (load_last <= cb->load_light || cb->load_light >= 1.0)
                return light;
            return light + (full - light) * (load_last - cb->load_light) / (1.0 - cb->load_light);
        };
        // a convolution kernel that gathers the image through VGPRs pays for the
        // share of chunks it must gather element by element (measured with every
        // chunk so); the calibrated step has whole-chunk loads only
        double step_full = cb->step_full, step_light = cb->step_light;
        if (sh.op == 1 && sh.gather_frac > 0.0 && !(k.align & 1)) {
            if (cb->step_gather > cb->step_full)
                step_full += sh.gather_frac * (cb->step_gather - cb->step_full);
            if (cb->step_gather_light > cb->step_light)
                step_light += sh.gather_frac * (cb->step_gather_light - cb->step_light);
        }
        const double wave_full = cb->fix_full + (double)nk * step_full;
        const double wave_last = at_load(cb->fix_full, cb->fix_light) + (double)nk * at_load(step_full, step_light);
        const double wave_dp = cb->fix_full + (double)nk_whole * step_full;
        const double cost2 = (double)F_dp * wave_dp + (double)(F - 1) * wave_full + wave_last + t_split;
        return launch_cal + std::max(cost2, floor_ns);
    }

    // Levels 0 and 1 for a workgroup of nk_ K steps and split_ slices, with
    // pc workgroups sharing each CU.
    const bool valu = k.family == 2;
    auto t1_for = [&](int64_t nk_, bool split_epilogue, double pc) {
        // Level 0: one K step of MFMAs fed from LDS (Eq. 2 over the Kb/k0 sub-steps),
        // or of vector-ALU dot products on B chunks held in registers (family 2:
        // v_dot2 retires 4 FLOP per lane, v_fma 2, one wave instruction per SIMD
        // every 4 clocks; A comes from LDS at a few bytes per k).
        const double flop_clk = valu ? 64.0 * hw.simd_per_cu * (sh.dt == VX_F32 ? 0.5 : 1.0)
                                     : (sh.dt == VX_F32 ? hw.mfma_flop_clk_cu_f32 : hw.mfma_flop_clk_cu_f16);
        const double rate_wg = flop_clk * hw.clock_ghz *
                               std::min((double)waves / hw.simd_per_cu, 1.0 / pc);   // FLOP/ns
        const int kstep = valu ? k.kb : k.mfma_k * (sh.dt == VX_F32 ? 4 : 1);  // fp32 loads 4 MFMA steps at once
        const int64_t sub = std::max<int64_t>(1, k.kb / kstep);
        const double c_mfma = 2.0 * k.mb * k.nb * kstep / rate_wg;
        const double lds_bw = hw.lds_bytes_clk_cu * hw.clock_ghz / pc;             // B/ns
        const double t_lds = valu ? (double)k.threads * k.stages * k.mb * 4.0 / lds_bw
                                  : (double)waves * ((double)k.mb / k.wm + (double)k.nb / k.wn) * kstep * eb / lds_bw;
        const double cost0 = vx_cost_temporal(t_lds, sub, c_mfma, 0.0);

        // Level 1: the K loop of one workgroup (Eq. 2 over n_k K steps).
        // element-aligned operands: the same 16-byte loads, but misaligned ones
        // straddle an extra cache line per row segment and the ragged edge chunks
        // are gathered element by element
        const double bw_wg = bw_wg_at(pc);
        const double load_factor = k.align == 3 ? 1.0 : k.align == 0 ? 1.25 : 1.12;
        // (family 2 reads only B from memory in the loop; its A slice is loaded once)
        const double xfer = (double)(valu ? k.nb : k.mb + k.nb) * k.kb * eb * load_factor / bw_wg;
        const double t_load = hw.mem_latency_ns + xfer;
        const double t_store = (double)k.mb * k.nb * eb / bw_wg + (split_epilogue ? t_split_at(pc) : 0.0);
        const int depth = valu ? 1 : std::max(1, k.stages - 1);   // family 2: two register sets
        if (depth == 1 || nk_ <= 1)
            return vx_cost_temporal(t_load, nk_, cost0, t_store);
        const double t_issue = std::max(xfer, t_load / depth);
        return t_load + (double)(nk_ - 1) * std::max(t_issue, cost0) + cost0 + t_store;
    };

    // Level 2 (Eq. 4), dispatch constant, compulsory-traffic floor.
    double cost2 = (double)F * t1_for(nk, split > 1, per_cu);
    if (hyb)
        cost2 += (double)F_dp * t1_for(nk_whole, false, (double)occ);
    return hw.launch_ns + std::max(cost2, floor_ns);
}

double floor_of(const vx_hwinfo& hw, const VxShape& sh)
{
    const int eb = sh.dt == VX_F32 ? 4 : 2;
    const double bytes_min = (double)sh.batch * ((double)sh.M * sh.K + (double)sh.K * sh.N + (double)sh.M * sh.N) * eb;
    return bytes_min / hw.hbm_gbps;
}

// The cost of one (kernel, split) pair with the kernel's calibration (or
// nullptr), resident workgroups per CU and calibrated dispatch constant given.
// split < 0: the hybrid grid -- whole waves of whole tiles, and the remaining
// tiles split -split ways (the last, partial wave of the plain grid spread
// over more workgroups).
double cost_core(const vx_hwinfo& hw, const VxShape& sh, const vx_kernel_info& k, int split, const VxLimits& lim,
                 int* k_per_split, int64_t* dp_tiles, const VxCalib* cb, int occ, double launch_cal)
{
    const bool hyb = split < 0;
    if (hyb)
        split = -split;
    if (!k.enabled || (int)k.dtype != sh.dt || (k.align & ~sh.vec_ok) || split < 1 || k.op != sh.op)
        return -1.0;
    if (hyb && (split < 2 || sh.K == 0))
        return -1.0;
    if (sh.K == 0 && split != 1)
        return -1.0;
    const int64_t tiles_m = cdiv(sh.M, k.mb), tiles_n = cdiv(sh.N, k.nb);
    if ((double)tiles_m * (double)tiles_n * (double)sh.batch > (double)INT32_MAX)
        return -1.0;
    PlanInts pi;
    pi.tiles = tiles_m * tiles_n * sh.batch;
    pi.nk = sh.K == 0 ? 0 : cdiv(cdiv(sh.K, split), k.kb);
    pi.nk_whole = cdiv(sh.K, k.kb);
    if (!grid_ints(hw, sh, k.mb, k.nb, k.kb, split, hyb, lim, (int64_t)hw.num_cu * occ, &pi) ||
        !kernel_fits(sh, k, hyb, pi.kps))
        return -1.0;
    if (k_per_split)
        *k_per_split = (int)pi.kps;
    if (dp_tiles)
        *dp_tiles = pi.dp;
    return plan_cost(hw, sh, k, split, hyb, pi, cb, occ, launch_cal, floor_of(hw, sh));
}

}  // namespace

double vxi_cost(const vx_hwinfo& hw, const VxShape& sh, const vx_kernel_info& k, int split,
                const VxLimits& lim, int* k_per_split, int64_t* dp_tiles)
{
    return cost_core(hw, sh, k, split, lim, k_per_split, dp_tiles, vxi_calib(k.id), vxi_occupancy(hw, k),
                     vxi_calib_launch_ns(hw));
}

bool vxi_wave_matches(const VxFilter& f, const vx_kernel_info& k)
{
    if (f.wave_m <= 0)
        return true;
    return k.mb / k.wm == f.wave_m && k.nb / k.wn == f.wave_n && k.mfma_m == f.mfma_m;
}

// ---- the search (Eq. 1) ------------------------------------------------------
//
// The argmin over (kernel, split, grid) is exact -- the same plan as pricing
// every triple -- but most triples are never priced.  Per thread, the
// registry is kept per (dtype, operator) as groups of kernels that share a
// workgroup tile (Mb, Nb, Kb) and a residency (workgroups per CU), so that a
// group's tile count, K steps per slice and grid waves are computed once for
// all its kernels; each kernel keeps a copy of its calibration.  A call
//   1. bounds every group from below (a weak bound, a few multiplications);
//   2. prices first the plan this thread last took for the same operand
//      shape class with only M different (the dynamic-M case), then the
//      groups with the least bounds, so that a tight best cost is known early;
//   3. visits the other groups in registry order, skipping a group, a
//      (group, split, grid) or a kernel whose bound exceeds the best cost so
//      far (by a relative 1e-9, which covers the bounds' own rounding).
// Ties are broken as when every triple is priced in registry order: least
// cost, then fewer slices, then the lower registry index, then the plain grid.
//
// The bounds.  A plan runs F >= 1 waves of workgroups on S = CUs x resident
// slots.  The waves but the last take the full-load fixed and step times, the
// last one times between the light- and full-load values (so >= their
// minimum), a hybrid grid first runs F_dp = floor(tiles / S) waves of whole
// tiles at the full-load times, and s > 1 slices add the split-K epilogue,
// >= a + b (s - 1) when measured (>= 0 otherwise).  With nk_s K steps per
// slice and F = ceil(tiles s / S) waves (plain grid):
//   cost >= launch + max(floor, (F - 1)(fix_full + nk_s step_full)
//                                + fix_min + nk_s step_min + epilogue).
// Over all splits: the K steps one slot runs add up to X >= max(T, 1), T =
// tiles nk / S (nk = ceil(K/Kb)), the last wave runs at most nk_s of them
// (nk_s = the steps of one of s slices, never more at a larger split), so the
// steps cost >= max(0, X - nk_s) step_full + min(X, nk_s) step_min; a plan of
// s >= 2 slices also runs >= floor(tiles / S) waves before its last, each
// with the full-load fixed time; with the epilogue growing in s, a split
// whose bound is beaten ends the split loop, and so does one where
// step_min max(T, nk / s') + a + b (s' - 1), convex in a real s', is beaten
// at its least over s' >= s.  A group's bound over its plans with s >= 2:
// the steps of s_max with the epilogue of s = 2 (weak), or the greater of
// step_min max(T, nk / s) + a + b (s - 1) at the real s = sqrt(step_min nk /
// b) clamped to [2, s_max] and to at most nk / T, and the step bound above
// with nk_2 and the epilogue a + b (tight).  A group's terms are the least of
// its kernels' (each bound grows with every term).  Uncalibrated kernels are
// bounded by launch + floor only.

thread_local int64_t t_evaluations = 0;   // (kernel, split, grid) triples priced by this thread's last search

namespace {

constexpr int kNSplits = (int)(sizeof(kSplits) / sizeof(kSplits[0]));

// the bound's terms of a kernel, or of a set of kernels (each term the least
// over the set: the bound grows with every one of them; slots the largest)
struct BoundTerms {
    double fix_min = INFINITY, fix_full = INFINITY, step_min = INFINITY, step_full = INFINITY;
    double split_a = INFINITY, split_b = INFINITY;
    int64_t slots = 0;
    double inv_slots = 0.0;   // 1 / slots
    double c_split = 0.0;     // sqrt(step_min / split_b) (0 when split_b is 0)
    bool cal = true;          // calibrated (every kernel of the set)
    void add(const BoundTerms& o)
    {
        fix_min = std::min(fix_min, o.fix_min);
        fix_full = std::min(fix_full, o.fix_full);
        step_min = std::min(step_min, o.step_min);
        step_full = std::min(step_full, o.step_full);
        split_a = std::min(split_a, o.split_a);
        split_b = std::min(split_b, o.split_b);
        slots = std::max(slots, o.slots);
        cal = cal && o.cal;
    }
    // the plan's cost less launch and floor, bounded below (nk_s steps per
    // slice, F >= 1 waves of them after F_dp waves of nk whole-tile steps)
    double lo(int64_t F, double nk_s, int s, int64_t F_dp = 0, double nk = 0.0) const
    {
        double c = (double)F_dp * (fix_full + nk * step_full) + (double)(F - 1) * (fix_full + nk_s * step_full) +
                   fix_min + nk_s * step_min;
        if (s > 1)
            c += split_a + split_b * (double)(s - 1);
        return c;
    }
};
struct SelKernel {
    int idx;                  // registry index
    int occ;                  // resident workgroups per CU
    VxCalib cb;               // its calibration (a copy; meaningful when bt.cal)
    BoundTerms bt;
};
struct SelGroup {
    int mb, nb, kb, occ;
    int mi, ni, ki;           // indices of mb, nb, kb among the class's distinct extents
    int align_and;            // AND of the members' alignment classes (a member is
                              // admitted when its align & ~vec_ok == 0)
    BoundTerms bt;
    std::vector<SelKernel> ks;
};
constexpr int kMaxExtents = 64;   // distinct Mb, Nb or Kb values of one class
struct SelClass {
    std::vector<SelGroup> gs;
    int mb[kMaxExtents], nb[kMaxExtents], kb[kMaxExtents];
    int n_mb = 0, n_nb = 0, n_kb = 0;
};
struct SelTables {
    bool valid = false;
    uint64_t epoch = 0;
    uint64_t gen = 0;         // distinct for every build of the tables in the process
    vx_hwinfo hw;
    double launch_cal = 0.0;
    SelClass cls[3][2];       // dtype x operator
};

int extent_index(int* v, int* n, int x)
{
    for (int i = 0; i < *n; ++i)
        if (v[i] == x)
            return i;
    if (*n == kMaxExtents)
        return -1;
    v[*n] = x;
    return (*n)++;
}
thread_local SelTables t_sel;

const SelTables& sel_tables(const vx_hwinfo& hw)
{
    const uint64_t ep = vxi_plan_epoch();
    SelTables& T = t_sel;
    if (T.valid && T.epoch == ep && !memcmp(&T.hw, &hw, sizeof hw))
        return T;
    static std::atomic<uint64_t> builds{0};
    T = SelTables{};
    T.epoch = ep;
    T.gen = ++builds;
    T.hw = hw;
    T.launch_cal = vxi_calib_launch_ns(hw);
    int n = 0;
    const VxKernelEntry* reg = vxi_registry(&n);
    for (int i = 0; i < n; ++i) {
        const vx_kernel_info& k = reg[i].info;
        if (!k.enabled || k.dtype < 0 || k.dtype > 2 || k.op < 0 || k.op > 1)
            continue;
        SelClass& c = T.cls[k.dtype][k.op];
        const int occ = vxi_occupancy(hw, k);
        SelGroup* g = nullptr;
        for (SelGroup& x : c.gs)
            if (x.mb == k.mb && x.nb == k.nb && x.kb == k.kb && x.occ == occ)
                g = &x;
        if (!g) {
            const int mi = extent_index(c.mb, &c.n_mb, k.mb), ni = extent_index(c.nb, &c.n_nb, k.nb),
                      ki = extent_index(c.kb, &c.n_kb, k.kb);
            c.gs.push_back(SelGroup{k.mb, k.nb, k.kb, occ, mi, ni, ki, ~0, BoundTerms{}, {}});
            g = &c.gs.back();
        }
        SelKernel s;
        s.idx = i;
        s.occ = occ;
        const VxCalib* cb = vxi_calib(k.id);
        s.cb = cb ? *cb : VxCalib{};
        BoundTerms& b = s.bt;
        b.cal = cb != nullptr;
        b.slots = (int64_t)hw.num_cu * s.occ;
        b.fix_min = cb ? std::min(cb->fix_full, cb->fix_light) : 0.0;
        b.fix_full = cb ? cb->fix_full : 0.0;
        b.step_min = cb ? std::min(cb->step_full, cb->step_light) : 0.0;
        b.step_full = cb ? cb->step_full : 0.0;
        const bool measured = cb && cb->split_a >= 0.0 && cb->split_b >= 0.0;
        b.split_a = measured ? cb->split_a : 0.0;
        b.split_b = measured ? cb->split_b : 0.0;
        g->align_and &= k.align;
        g->bt.add(b);
        g->ks.push_back(s);
    }
    for (auto& dc : T.cls)
        for (SelClass& c : dc)
            for (SelGroup& g : c.gs) {
                g.bt.inv_slots = 1.0 / (double)g.bt.slots;
                g.bt.c_split = g.bt.split_b > 0.0 ? sqrt(g.bt.step_min / g.bt.split_b) : 0.0;
            }
    T.valid = true;
    return T;
}

// Lexicographic order of the search's outcome: cost, then fewer K slices (no
// split-K epilogue and no partial traffic, which bounds such as the HBM floor
// do not see), then the lower registry index, then the plain grid.
struct Best {
    double cost = INFINITY;
    int idx = -1, split = 0, kps = 0, hyb = 0;
    int gi = -1;              // the group of the kernel
    int64_t dp = 0;
    bool beaten_by(double c, int s, int i, int h) const
    {
        if (c != cost)
            return c < cost;
        if (s != split)
            return s < split;
        if (i != idx)
            return i < idx;
        return h < hyb;
    }
};

// The plan each thread last took per operand shape class (everything but M).
struct WarmKey {
    uint64_t gen;             // the tables' build (group indices are its)
    int dt, op, vec_ok;
    int64_t N, K, batch;
    bool operator==(const WarmKey& o) const
    {
        return gen == o.gen && dt == o.dt && op == o.op && vec_ok == o.vec_ok && N == o.N && K == o.K &&
               batch == o.batch;
    }
};
struct WarmSlot {
    WarmKey key;
    int group, split_j, hyb;
    bool valid;
};
constexpr int kWarmSlots = 256;   // a power of two
thread_local WarmSlot t_warm[kWarmSlots];
inline uint64_t warm_hash(const WarmKey& k)
{
    uint64_t h = 1469598103934665603ull;
    auto mix = [&h](uint64_t v) { h = (h ^ v) * 1099511628211ull; };
    mix(k.gen);
    mix((uint64_t)k.dt | ((uint64_t)k.op << 4) | ((uint64_t)k.vec_ok << 8));
    mix((uint64_t)k.N);
    mix((uint64_t)k.K);
    mix((uint64_t)k.batch);
    return h ^ (h >> 29);
}

}  // namespace

vx_status vxi_select(const vx_hwinfo& hw, const VxShape& sh, const VxLimits& lim, const VxFilter& f,
                     vx_plan* out)
{
    const int forced_id = f.kernel_id, forced_split = f.split;
    int n = 0;
    const VxKernelEntry* reg = vxi_registry(&n);
    Best best;
    int64_t evaluated = 0;
    t_evaluations = 0;
    if (sh.dt < 0 || sh.dt > 2 || sh.op < 0 || sh.op > 1)
        return VX_ERR_NO_CANDIDATE;
    const SelTables& T = sel_tables(hw);
    const SelClass& CL = T.cls[sh.dt][sh.op];
    const std::vector<SelGroup>& C = CL.gs;
    const bool prune = !vxi_exhaustive_search();
    const bool K0 = sh.K == 0;
    const double floor_ns = floor_of(hw, sh);
    const double s_max = forced_split != 0 ? (double)(forced_split < 0 ? -forced_split : forced_split)
                                           : (double)kSplits[kNSplits - 1];
    // splits in increasing order (a forced split: only the slices it yields)
    int kcut[kNSplits];   // ceil(K / s)
    for (int j = 0; j < kNSplits; ++j)
        kcut[j] = K0 ? 0 : (int)cdiv(sh.K, kSplits[j]);
    // tile and step counts per distinct extent; K steps per slice on demand
    int64_t cm[kMaxExtents], cn[kMaxExtents], ck[kMaxExtents];
    int64_t nks[kMaxExtents][kNSplits];
    for (int i = 0; i < CL.n_mb; ++i)
        cm[i] = cdiv(sh.M, CL.mb[i]);
    for (int i = 0; i < CL.n_nb; ++i)
        cn[i] = cdiv(sh.N, CL.nb[i]);
    for (int i = 0; i < CL.n_kb; ++i) {
        ck[i] = K0 ? 0 : cdiv(sh.K, CL.kb[i]);
        for (int j = 0; j < kNSplits; ++j)
            nks[i][j] = -1;
    }
    // ceil(a / b) for 0 <= a < 2^52, 1 <= b < 2^52 without an integer
    // division: the truncated, correctly rounded quotient f is within one of
    // a / b and only off where a / b is within an ulp of an integer, so
    // f + (f b < a) is the ceiling
    auto ceil_div = [](int64_t a, int64_t b) {
        const int64_t f = (int64_t)((double)a / (double)b);
        return f + (f * b < a ? 1 : 0);
    };
    // ceil(a / b) from a precomputed 1 / b (same argument as ceil_div)
    auto ceil_mul = [](int64_t a, int64_t b, double inv_b) {
        const int64_t f = (int64_t)((double)a * inv_b);
        return f + (f * b < a ? 1 : 0);
    };
    // least K steps per slice over every split the search takes, the most over
    // splits >= 2 (those of two slices), and sqrt(nk), per Kb
    int64_t nk_smax[kMaxExtents], nk_half[kMaxExtents];
    double sq_nk[kMaxExtents];
    for (int i = 0; i < CL.n_kb; ++i) {
        nk_smax[i] = std::max<int64_t>(1, ceil_div(ck[i], (int64_t)s_max));
        nk_half[i] = K0 ? 0 : cdiv(kcut[1], CL.kb[i]);
        sq_nk[i] = sqrt((double)ck[i]);
    }
    // the K steps of a slot that runs X in all, at most `last` of them in the
    // last wave (at no less than step_min), the others at step_full
    auto steps_lo = [](const BoundTerms& b, double X, double last) {
        return std::max(0.0, X - last) * b.step_full + std::min(X, last) * b.step_min;
    };
    // a group's bound over its plans with s >= 2 slices: steps per slot >=
    // max(T, nk / s), epilogue >= a + b (s - 1); as a function of a real s this
    // is convex, least at s = sqrt(step_min nk / b), clamped to [2, s_max] and
    // to <= nk / T.  Or: the slot's max(T, 1) steps but the last wave's (at
    // most those of two slices, nk2) at the full-load step, epilogue >= a + b
    auto many_tight = [&](const BoundTerms& b, int64_t tiles, int64_t nkw, double sqnk, int64_t fdp, int64_t nk2) {
        const double nk = (double)nkw, Tq = (double)tiles * nk * b.inv_slots;
        double s = b.split_b > 0.0 ? b.c_split * sqnk : s_max;
        if (Tq > 0.0 && s * Tq > nk)
            s = nk / Tq;
        s = std::min(std::max(s, 2.0), std::max(s_max, 2.0));
        const double convex = b.step_min * std::max(Tq, nk / s) + b.split_b * (s - 1.0);
        const double waves = steps_lo(b, std::max(Tq, 1.0), (double)nk2) + b.split_b;
        return b.fix_min + (double)fdp * b.fix_full + b.split_a + std::max(convex, waves);
    };

    auto lb_of = [&](double lo, bool cal) {
        return cal ? T.launch_cal + std::max(floor_ns, lo) : hw.launch_ns + floor_ns;
    };
    // (a small relative margin covers the bounds' own rounding)
    auto beaten = [&](double lb) { return prune && lb > best.cost * (1.0 + 1e-9); };
    auto admitted = [&](const vx_kernel_info& k) {
        if ((forced_id >= 0 && k.id != forced_id) || !vxi_wave_matches(f, k))
            return false;
        // The mixed im2col tiles (image through VGPRs, filter by DMA) carry one
        // K step of image gathers at a time; where a quarter or more of the
        // image's chunks are gathered element by element (first layers over a
        // few channels) they ran 1.3-1.7x slower than the register-staged
        // tiles, and the calibrated step costs (whole-chunk and fully gathered
        // steps) priced them 30-40 % low there (stem layers: 11.2-11.8 us
        // measured, 8.1-8.4 predicted).  The selector offers them only below
        // that share; a forced plan may still take them.
        if (forced_id < 0 && k.op == 1 && k.family == 1 && !(k.align & 1) && sh.gather_frac >= 0.25)
            return false;
        return (f.backends & (k.family == 2 ? 2 : 1)) && !(k.align & ~sh.vec_ok);
    };

    // prices the members of group g for `split` slices (hybrid or plain) with
    // nk K steps per slice
    auto price_members = [&](const SelGroup& g, int64_t tiles, int64_t nk, int64_t nk_whole, int split, bool hyb) {
        PlanInts pi;
        pi.tiles = tiles;
        pi.nk = nk;
        pi.nk_whole = nk_whole;
        if (!grid_ints(hw, sh, g.mb, g.nb, g.kb, split, hyb, lim, g.bt.slots, &pi))
            return;
        for (const SelKernel& s : g.ks) {
            const vx_kernel_info& k = reg[s.idx].info;
            if (!admitted(k))
                continue;
            ++evaluated;
            if (!kernel_fits(sh, k, hyb, pi.kps))
                continue;
            if (s.bt.cal && beaten(lb_of(s.bt.lo(pi.F, (double)nk, split, pi.F_dp, (double)nk_whole), true)))
                continue;
            const double c = plan_cost(hw, sh, k, split, hyb, pi, s.bt.cal ? &s.cb : nullptr, s.occ, T.launch_cal,
                                       floor_ns);
            if (best.beaten_by(c, split, s.idx, hyb)) {
                best.gi = (int)(&g - C.data());
                best.cost = c;
                best.idx = s.idx;
                best.split = split;
                best.kps = (int)pi.kps;
                best.dp = pi.dp;
                best.hyb = hyb;
            }
        }
    };

    // prices group g over its splits
    auto price_group = [&](const SelGroup& g, int64_t tiles, int64_t nk_whole) {
        const bool ext = g.ki >= 0;
        const BoundTerms& b = g.bt;
        const int64_t Fdp = tiles / b.slots;
        if (b.cal && prune && forced_split == 0 && !K0 && nk_whole >= 2) {
            // the group passed its weak bound; the tight one over every split
            const double one = b.lo(std::max<int64_t>(1, ceil_mul(tiles, b.slots, b.inv_slots)), (double)nk_whole, 1);
            const double sq = ext ? sq_nk[g.ki] : sqrt((double)nk_whole);
            const int64_t nk2 = ext ? nk_half[g.ki] : cdiv(kcut[1], g.kb);
            if (beaten(lb_of(std::min(one, many_tight(b, tiles, nk_whole, sq, Fdp, nk2)), true)))
                return;
        }
        const double Tq = (double)tiles * (double)nk_whole * b.inv_slots;   // K steps per slot, whole grid
        // a plan of s >= 2 slices runs >= floor(tiles / slots) waves before its
        // last (plain grid: ceil(s tiles / slots) - 1; hybrid: that many whole
        // waves), each at the full-load fixed time
        const double fix_waves = (double)Fdp * b.fix_full;
        if (forced_split != 0) {
            // a forced split runs as the number of non-empty slices it yields
            const int fs = forced_split < 0 ? -forced_split : forced_split;
            const int64_t kps0 = cdiv(cdiv(std::max<int64_t>(sh.K, 1), fs), g.kb) * g.kb;
            const int split = K0 ? 1 : (int)cdiv(sh.K, kps0);
            const bool hyb = forced_split < 0;
            if ((hyb && split < 2) || (hyb && K0))
                return;
            price_members(g, tiles, K0 ? 0 : cdiv(cdiv(sh.K, split), g.kb), nk_whole, split, hyb);
            return;
        }
        for (int j = 0; j < kNSplits; ++j) {
            const int split = kSplits[j];
            if (K0 && split > 1)
                break;
            if (!K0 && split > nk_whole)
                break;   // a slice would be empty, here and at every larger split
            int64_t nk = 0;
            if (!K0) {
                if (ext) {
                    int64_t& m = nks[g.ki][j];
                    if (m < 0)
                        m = cdiv(kcut[j], g.kb);
                    nk = m;
                } else {
                    nk = cdiv(kcut[j], g.kb);
                }
            }
            if (!K0 && (int64_t)(split - 1) * nk * g.kb >= sh.K)
                continue;   // a slice would be empty
            if (b.cal && prune && split > 1) {
                // every split's slots run >= max(T, 1) K steps in all, the last
                // wave at most this split's nk of them (a larger split's slices
                // are no longer), and the epilogue grows with the split: once
                // that is beaten, every larger split is
                const double X = std::max(Tq, 1.0), nkw = (double)nk_whole;
                const double steps = steps_lo(b, X, (double)nk);
                if (beaten(lb_of(b.fix_min + fix_waves + steps + b.split_a + b.split_b * (double)(split - 1), true)))
                    break;
                // ... and a slot of s' >= split slices runs >= nk_whole / s'
                // steps too: step_min max(T, nk / s') + a + b (s' - 1) is
                // convex in a real s', least over s' >= split at max(split, s*)
                if (b.split_b > 0.0) {
                    double sr = b.c_split * (ext ? sq_nk[g.ki] : sqrt(nkw));
                    if (Tq > 0.0 && sr * Tq > nkw)
                        sr = nkw / Tq;
                    sr = std::max(sr, (double)split);
                    if (beaten(lb_of(b.fix_min + fix_waves + b.step_min * std::max(Tq, nkw / sr) + b.split_a +
                                         b.split_b * (sr - 1.0), true)))
                        break;
                }
            }
            // plain grid
            const int64_t Fg = std::max<int64_t>(1, ceil_mul(tiles * split, b.slots, b.inv_slots));
            if (!(b.cal && beaten(lb_of(b.lo(Fg, (double)nk, split), true))))
                price_members(g, tiles, nk, nk_whole, split, false);
            // hybrid grid: whole waves of whole tiles, the rest split
            if (split >= 2 && f.hybrid && Fdp >= 1) {
                if (!(b.cal && beaten(lb_of(b.lo(1, (double)nk, split, Fdp, (double)nk_whole), true))))
                    price_members(g, tiles, nk, nk_whole, split, true);
            }
        }
    };

    // groups: bounds over all their plans, the kFirst least priced first
    const int ng = (int)C.size();
    double* lb = (double*)alloca(sizeof(double) * (ng > 0 ? ng : 1));
    int64_t* tl = (int64_t*)alloca(sizeof(int64_t) * 2 * (ng > 0 ? ng : 1));
    constexpr int kFirst = 6;
    int first[kFirst];
    int n_first = 0;
    for (int i = 0; i < ng; ++i) {
        const SelGroup& g = C[i];
        lb[i] = -1.0;
        if (g.align_and & ~sh.vec_ok)
            continue;   // no member admits this shape's operands
        const bool ext = g.mi >= 0 && g.ni >= 0 && g.ki >= 0;
        const int64_t tiles = (ext ? cm[g.mi] : cdiv(sh.M, g.mb)) * (ext ? cn[g.ni] : cdiv(sh.N, g.nb)) * sh.batch;
        const int64_t nkw = K0 ? 0 : ext ? ck[g.ki] : cdiv(sh.K, g.kb);
        tl[2 * i] = tiles;
        tl[2 * i + 1] = nkw;
        const BoundTerms& b = g.bt;
        // the weak bound: one slice as above; s >= 2 slices with the steps of
        // s_max and the epilogue of s = 2 (no division, no square root)
        double lo = b.lo(std::max<int64_t>(1, ceil_mul(tiles, b.slots, b.inv_slots)), (double)nkw, 1);
        if (!K0 && nkw >= 2) {
            const double Tq = (double)tiles * (double)nkw * b.inv_slots;
            lo = std::min(lo, b.fix_min + b.step_min * std::max(Tq, (double)(ext ? nk_smax[g.ki] : 1)) + b.split_a);
        }
        lb[i] = lb_of(lo, b.cal);
        int j = n_first < kFirst ? n_first++ : kFirst;
        for (; j > 0 && lb[first[j - 1]] > lb[i]; --j)
            if (j < kFirst)
                first[j] = first[j - 1];
        if (j < kFirst)
            first[j] = i;
    }
    // warm start: the plan last taken by this thread for the same operand
    // shape class with only M different, priced first at this shape (the
    // dynamic-M case), so the bounds meet a tight best cost from the start
    WarmKey wk{T.gen, sh.dt, sh.op, sh.vec_ok, sh.N, sh.K, sh.batch};
    WarmSlot& ws = t_warm[warm_hash(wk) & (kWarmSlots - 1)];
    if (prune && forced_id < 0 && forced_split == 0 && f.wave_m <= 0 && f.backends == 3 && f.hybrid &&
        ws.valid && ws.key == wk && ws.group < ng && lb[ws.group] >= 0.0) {
        const int gi = ws.group;
        const SelGroup& g = C[gi];
        const int64_t nk = K0 ? 0 : cdiv(kcut[ws.split_j], g.kb);
        if (K0 ? ws.split_j == 0 : kSplits[ws.split_j] <= tl[2 * gi + 1])
            price_members(g, tl[2 * gi], nk, tl[2 * gi + 1], kSplits[ws.split_j], ws.hyb != 0);
    }
    for (int j = 0; j < n_first; ++j) {
        if (beaten(lb[first[j]]))
            break;
        price_group(C[first[j]], tl[2 * first[j]], tl[2 * first[j] + 1]);
        lb[first[j]] = -1.0;   // priced
    }
    for (int i = 0; i < ng; ++i) {
        if (lb[i] < 0.0 || beaten(lb[i]))
            continue;
        price_group(C[i], tl[2 * i], tl[2 * i + 1]);
    }
    t_evaluations = evaluated;
    if (best.idx < 0)
        return VX_ERR_NO_CANDIDATE;
    if (best.gi >= 0) {
        ws.key = wk;
        ws.group = best.gi;
        int sj = 0;
        while (sj + 1 < kNSplits && kSplits[sj] != best.split)
            ++sj;
        ws.split_j = kSplits[sj] == best.split ? sj : 0;
        ws.hyb = best.hyb;
        ws.valid = kSplits[sj] == best.split;
    }
    const vx_kernel_info& k = reg[best.idx].info;
    vx_plan p;
    p.kernel_id = k.id;
    p.split_k = best.split;
    p.k_per_split = best.kps;
    p.c_vec = sh.c_vec;
    p.tiles_m = cdiv(sh.M, k.mb);
    p.tiles_n = cdiv(sh.N, k.nb);
    const int64_t tiles = p.tiles_m * p.tiles_n * sh.batch;
    p.dp_tiles = best.dp;
    p.grid = best.dp + (tiles - best.dp) * best.split;
    p.group_m = vxi_group_m(p.tiles_m, p.tiles_n);
    p.workspace_bytes = best.split > 1 ? (size_t)(tiles - best.dp) * best.split * k.mb * k.nb * 4 : 0;
    p.predicted_ns = best.cost;
    p.kernel = k;
    *out = p;
    return VX_OK;
}

extern "C" int64_t vx_selector_last_evaluations(void) { return t_evaluations; }
