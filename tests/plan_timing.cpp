// Host-side timing of the selector (no GPU): plans a list of shapes that the
// library has not seen, with the MI355X description as a planning override,
// and prints the mean wall-clock time per vx_plan_query (std::chrono), the
// least over several passes (each pass first retires every cached plan).
// Usage: plan_timing <calibration table> <passes> then lines "batch M N K dtype" on stdin.
#include <algorithm>
#include <chrono>
#include <cstdio>
#include <cstring>
#include <vector>

#include "vx.h"

int main(int argc, char** argv)
{
    if (argc < 3)
        return 2;
    vx_hwinfo h;
    memset(&h, 0, sizeof h);
    strcpy(h.arch, "gfx950");
    h.num_cu = 256;
    h.num_xcd = 8;
    h.simd_per_cu = 4;
    h.wave_size = 64;
    h.max_threads_per_wg = 1024;
    h.lds_bytes_per_cu = 160 * 1024;
    h.vgprs_per_lane = 512;
    h.max_waves_per_simd = 8;
    h.clock_ghz = 2.4;
    h.hbm_gbps = 8000.0;
    h.l2_bytes_per_xcd = 4.0 * 1024 * 1024;
    h.mall_bytes = 256.0 * 1024 * 1024;
    h.mfma_flop_clk_cu_f16 = 4096.0;
    h.mfma_flop_clk_cu_f32 = 256.0;
    h.l2_bytes_clk_cu = 64.0;
    h.lds_bytes_clk_cu = 128.0;
    h.mem_latency_ns = 900.0;
    h.atomic_latency_ns = 1200.0;
    h.launch_ns = 2000.0;
    if (vx_set_hwinfo_override(&h) != VX_OK)
        return 3;
    int loaded = 0;
    if (vx_calibration_load(argv[1], &loaded) != VX_OK)
        return 4;
    const int passes = atoi(argv[2]);
    struct Shape {
        long long b, m, n, k;
        int dt;
    };
    std::vector<Shape> sh;
    Shape s;
    while (scanf("%lld %lld %lld %lld %d", &s.b, &s.m, &s.n, &s.k, &s.dt) == 5)
        sh.push_back(s);
    if (sh.empty())
        return 5;
    vx_plan p;
    double best = 1e300, cached = 0.0;
    long long evals = 0;
    for (int r = 0; r < passes; ++r) {
        vx_selector_exhaustive(0);   // retires the cached plans
        for (int dt = 0; dt < 3; ++dt)
            vx_plan_query(1, 3, 5, 7, (vx_dtype)dt, 21, 35, 15, 256, &p);   // per-thread tables, outside timing
        evals = 0;
        const auto t0 = std::chrono::steady_clock::now();
        for (const Shape& x : sh) {
            if (vx_plan_query(x.b, x.m, x.n, x.k, (vx_dtype)x.dt, x.m * x.k, x.k * x.n, x.m * x.n, 256, &p) != VX_OK)
                return 6;
            evals += vx_selector_last_evaluations();
        }
        const auto t1 = std::chrono::steady_clock::now();
        for (const Shape& x : sh)
            vx_plan_query(x.b, x.m, x.n, x.k, (vx_dtype)x.dt, x.m * x.k, x.k * x.n, x.m * x.n, 256, &p);
        const auto t2 = std::chrono::steady_clock::now();
        best = std::min(best, std::chrono::duration<double, std::micro>(t1 - t0).count() / sh.size());
        cached = std::chrono::duration<double, std::micro>(t2 - t1).count() / sh.size();
    }
    printf("cold_us %.4f cached_us %.4f evals %.2f\n", best, cached, (double)evals / sh.size());
    return 0;
}
