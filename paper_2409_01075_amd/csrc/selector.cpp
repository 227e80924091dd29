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

#include <algorithm>

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

double vxi_cost(const vx_hwinfo& hw, const VxShape& sh, const vx_kernel_info& k, int split,
                const VxLimits& lim, int* k_per_split, int64_t* dp_tiles)
{
    // split < 0: the hybrid grid -- whole waves of whole tiles, and the
    // remaining tiles split -split ways (the last, partial wave of the plain
    // grid spread over more workgroups)
    const bool hyb = split < 0;
    if (hyb)
        split = -split;
    if (!k.enabled || (int)k.dtype != sh.dt || (k.align & ~sh.vec_ok) || split < 1 || k.op != sh.op)
        return -1.0;
    if (hyb && (split < 2 || sh.K == 0))
        return -1.0;
    const int eb = sh.dt == VX_F32 ? 4 : 2;
    const int64_t tiles_m = cdiv(sh.M, k.mb), tiles_n = cdiv(sh.N, k.nb);
    const int64_t tiles = tiles_m * tiles_n * sh.batch;
    int64_t kps = 0, nk = 0;
    if (sh.K == 0) {
        if (split != 1)
            return -1.0;
    } else {
        kps = cdiv(cdiv(sh.K, split), k.kb) * k.kb;
        if (cdiv(sh.K, kps) != split)       // a slice would be empty
            return -1.0;
        nk = kps / k.kb;
    }
    if (kps > INT32_MAX || tiles > INT32_MAX)
        return -1.0;
    if (k.k_max > 0 && (hyb ? sh.K : kps) > k.k_max)   // the kernel holds a whole slice of A in LDS
        return -1.0;

    const int waves = k.wm * k.wn;
    const int occ = vxi_occupancy(hw, k);
    const int64_t slots = (int64_t)hw.num_cu * occ;
    const int64_t dp = hyb ? tiles / slots * slots : 0;   // whole tiles, in whole waves
    const int64_t split_tiles = tiles - dp;
    if (hyb && (dp == 0 || split_tiles == 0 || slots % std::max(1, hw.num_xcd) != 0))
        return -1.0;   // (the kernels remap each class of workgroups over the XCDs on its own)
    const int64_t units = dp + split_tiles * split;
    if (units > INT32_MAX)
        return -1.0;
    if (split > 1) {
        if (split_tiles > lim.max_tickets)
            return -1.0;
        if ((double)split_tiles * split * k.mb * k.nb * 4.0 > (double)lim.ws_bytes)
            return -1.0;
    }
    if (k.family == 1) {
        // direct-to-LDS kernels address each K step with 32-bit buffer offsets:
        // Mb rows of A (Mb*K elements) and Kb rows of B (Kb*N elements); a
        // convolution's A offsets run over the whole image
        const double a_span = k.op == 1 ? (double)sh.a_bytes : (double)k.mb * sh.K * eb;
        if (a_span >= 2147483648.0 || (double)k.kb * sh.N * eb >= 2147483648.0)
            return -1.0;
    }
    if (k.family == 2) {
        // the vector-ALU kernels address a whole slice of B with 32-bit offsets
        if ((double)(hyb ? sh.K : kps) * sh.N * eb >= 2147483648.0)
            return -1.0;
    }
    if (k_per_split)
        *k_per_split = (int)kps;
    if (dp_tiles)
        *dp_tiles = dp;
    const int64_t nk_whole = cdiv(sh.K, k.kb);

    // Level 2: wave quantisation over the device (Eq. 3); a hybrid grid runs
    // dp / slots full waves of whole tiles, then the split tiles' slices.
    const int64_t units_s = hyb ? split_tiles * split : units;
    const int64_t F = vx_cost_parallel_factor(units_s, slots);
    const int64_t active = std::min(units_s, slots);
    const double per_cu = (double)cdiv(active, hw.num_cu);
    const int64_t F_dp = dp / slots;

    const double bytes_min = (double)sh.batch * ((double)sh.M * sh.K + (double)sh.K * sh.N + (double)sh.M * sh.N) * eb;
    const double floor_ns = bytes_min / hw.hbm_gbps;
    auto bw_wg_at = [&](double pc) { return hw.l2_bytes_clk_cu * hw.clock_ghz / pc; };   // B/ns, L2 -> one workgroup
    // split-K epilogue: the partial tile out, the arrival counter, and the
    // last arrival's reads of the other slices
    auto t_split_at = [&](double pc) {
        const double part = (double)k.mb * k.nb * 4.0 / bw_wg_at(pc);
        return split > 1 ? part + hw.atomic_latency_ns + hw.mem_latency_ns + (double)(split - 1) * part : 0.0;
    };

    const VxCalib* cb = vxi_calib(k.id);
    if (cb) {
        // empirical low levels, analytical grid level
        double t_split = t_split_at(per_cu);                                // split-K epilogue, analytical
        if (split > 1 && cb->split_a >= 0.0 && cb->split_b >= 0.0)
            t_split = cb->split_a + cb->split_b * (double)(split - 1);      // ... or measured
        const double load_last = (double)(units_s - (F - 1) * slots) / (double)slots;
        auto at_load = [&](double full, double light) {
            if (load_last <= cb->load_light || cb->load_light >= 1.0)
                return light;
            return light + (full - light) * (load_last - cb->load_light) / (1.0 - cb->load_light);
        };
        const double wave_full = cb->fix_full + (double)nk * cb->step_full;
        const double wave_last = at_load(cb->fix_full, cb->fix_light) + (double)nk * at_load(cb->step_full, cb->step_light);
        const double wave_dp = cb->fix_full + (double)nk_whole * cb->step_full;
        const double cost2 = (double)F_dp * wave_dp + (double)(F - 1) * wave_full + wave_last + t_split;
        return vxi_calib_launch_ns(hw) + std::max(cost2, floor_ns);
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

bool vxi_wave_matches(const VxFilter& f, const vx_kernel_info& k)
{
    if (f.wave_m <= 0)
        return true;
    return k.mb / k.wm == f.wave_m && k.nb / k.wn == f.wave_n && k.mfma_m == f.mfma_m;
}

vx_status vxi_select(const vx_hwinfo& hw, const VxShape& sh, const VxLimits& lim, const VxFilter& f,
                     vx_plan* out)
{
    const int forced_id = f.kernel_id, forced_split = f.split;
    int n = 0;
    const VxKernelEntry* reg = vxi_registry(&n);
    double best = INFINITY;
    int best_id = -1, best_split = 0, best_kps = 0;
    int64_t best_dp = 0;
    for (int i = 0; i < n; ++i) {
        const vx_kernel_info& k = reg[i].info;
        if ((forced_id >= 0 && k.id != forced_id) || !vxi_wave_matches(f, k))
            continue;
        if (!(f.backends & (k.family == 2 ? 2 : 1)))
            continue;
        if (!k.enabled || (int)k.dtype != sh.dt || (k.align & ~sh.vec_ok) || k.op != sh.op)
            continue;   // infeasible at every split (the same test opens vxi_cost)
        // (split, hybrid grid) pairs: each split plain, then (split >= 2) hybrid
        int pairs[2 * (int)(sizeof(kSplits) / sizeof(kSplits[0]))][2];
        int np = 0;
        if (forced_split != 0) {
            // a forced split runs as the number of non-empty slices it yields
            const int fs = forced_split < 0 ? -forced_split : forced_split;
            const int64_t kps0 = cdiv(cdiv(std::max<int64_t>(sh.K, 1), fs), k.kb) * k.kb;
            pairs[np][0] = sh.K == 0 ? 1 : (int)cdiv(sh.K, kps0);
            pairs[np++][1] = forced_split < 0;
        } else {
            for (int s : kSplits) {
                pairs[np][0] = s;
                pairs[np++][1] = 0;
                if (s >= 2 && f.hybrid) {
                    pairs[np][0] = s;
                    pairs[np++][1] = 1;
                }
            }
        }
        for (int j = 0; j < np; ++j) {
            const int split = pairs[j][0];
            int kps = 0;
            int64_t dp = 0;
            const double c = vxi_cost(hw, sh, k, pairs[j][1] ? -split : split, lim, &kps, &dp);
            if (c < 0.0)
                continue;
            // equal predicted costs (plans bounded by the same term, e.g. the
            // operands' HBM time) go to the fewer K slices: no split-K epilogue
            // and no partial-tile traffic, which the bound does not see.
            // Remaining ties keep the earlier (lower id, plain grid) candidate.
            if (c < best || (c == best && split < best_split)) {
                best = c;
                best_id = i;
                best_split = split;
                best_kps = kps;
                best_dp = dp;
            }
        }
    }
    if (best_id < 0)
        return VX_ERR_NO_CANDIDATE;
    const vx_kernel_info& k = reg[best_id].info;
    vx_plan p;
    p.kernel_id = k.id;
    p.split_k = best_split;
    p.k_per_split = best_kps;
    p.c_vec = sh.c_vec;
    p.tiles_m = cdiv(sh.M, k.mb);
    p.tiles_n = cdiv(sh.N, k.nb);
    const int64_t tiles = p.tiles_m * p.tiles_n * sh.batch;
    p.dp_tiles = best_dp;
    p.grid = best_dp + (tiles - best_dp) * best_split;
    p.group_m = vxi_group_m(p.tiles_m, p.tiles_n);
    p.workspace_bytes = best_split > 1 ? (size_t)(tiles - best_dp) * best_split * k.mb * k.nb * 4 : 0;
    p.predicted_ns = best;
    p.kernel = k;
    *out = p;
    return VX_OK;
}
