// GetHardwareInfo (Algorithm 2): the device facts the candidate feasibility
// rules and the analytical cost model (Equations 2-4) are written against.
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "vx_internal.h"

namespace {

struct ArchFacts {
    const char* arch;
    int num_xcd, simd_per_cu, vgprs_per_lane, max_waves_per_simd;
    double hbm_gbps, mall_bytes;
    double mfma_f16, mfma_f32;      // dense FLOP per clock per CU
    double l2_clk_cu, lds_clk_cu;   // bytes per clock per CU
    double mem_latency_ns, atomic_latency_ns, launch_ns;
    double peak_clock_ghz;
};

// MI355X (gfx950, CDNA4): 256 CUs in 8 XCDs, 4 SIMDs per CU, 160 KiB LDS,
// 288 GB HBM3E at 8 TB/s, 256 MB Infinity Cache, 2.4 GHz peak engine clock.
// Dense MFMA: 2.5 PFLOP/s fp16/bf16 = 256 CU x 4096 FLOP/clk x 2.4 GHz;
// 157.3 TFLOP/s fp32 = 256 CU x 256 FLOP/clk x 2.4 GHz.  The latency figures
// are the memory system's order of magnitude, not per-shape measurements.
const ArchFacts kFacts[] = {
    {"gfx950", 8, 4, 512, 8, 8000.0, 256.0 * 1024 * 1024, 4096.0, 256.0, 64.0, 128.0,
     900.0, 1200.0, 2000.0, 2.4},
};

}  // namespace

int vxi_device_hwinfo(int device, vx_hwinfo* o)
{
    hipDeviceProp_t p;
    if (hipGetDeviceProperties(&p, device) != hipSuccess)
        return -1;
    memset(o, 0, sizeof(*o));
    strncpy(o->arch, p.gcnArchName, sizeof(o->arch) - 1);
    char* colon = strchr(o->arch, ':');
    if (colon)
        *colon = 0;
    o->num_cu = p.multiProcessorCount;
    o->wave_size = p.warpSize;
    o->max_threads_per_wg = p.maxThreadsPerBlock;
    o->lds_bytes_per_cu = (int)p.maxSharedMemoryPerMultiProcessor;
    o->l2_bytes_per_xcd = (double)p.l2CacheSize;
    o->clock_ghz = p.clockRate / 1.0e6;
    const ArchFacts* f = nullptr;
    for (const ArchFacts& a : kFacts)
        if (strcmp(a.arch, o->arch) == 0)
            f = &a;
    if (f) {
        o->num_xcd = f->num_xcd;
        o->simd_per_cu = f->simd_per_cu;
        o->vgprs_per_lane = f->vgprs_per_lane;
        o->max_waves_per_simd = f->max_waves_per_simd;
        o->hbm_gbps = f->hbm_gbps;
        o->mall_bytes = f->mall_bytes;
        o->mfma_flop_clk_cu_f16 = f->mfma_f16;
        o->mfma_flop_clk_cu_f32 = f->mfma_f32;
        o->l2_bytes_clk_cu = f->l2_clk_cu;
        o->lds_bytes_clk_cu = f->lds_clk_cu;
        o->mem_latency_ns = f->mem_latency_ns;
        o->atomic_latency_ns = f->atomic_latency_ns;
        o->launch_ns = f->launch_ns;
        if (o->clock_ghz <= 0.0)
            o->clock_ghz = f->peak_clock_ghz;
        if (o->lds_bytes_per_cu <= 0)
            o->lds_bytes_per_cu = 160 * 1024;
    } else {
        // Unknown architecture: the kernels are built for gfx950 only, so
        // launches will fail; keep the description self-consistent anyway.
        o->num_xcd = 1;
        o->simd_per_cu = 4;
        o->vgprs_per_lane = 512;
        o->max_waves_per_simd = 8;
        o->hbm_gbps = 2.0 * p.memoryClockRate * 1e3 * (p.memoryBusWidth / 8.0) / 1e9;
        o->mfma_flop_clk_cu_f16 = 1024.0;
        o->mfma_flop_clk_cu_f32 = 256.0;
        o->l2_bytes_clk_cu = 64.0;
        o->lds_bytes_clk_cu = 128.0;
        o->mem_latency_ns = 1000.0;
        o->atomic_latency_ns = 1500.0;
        o->launch_ns = 3000.0;
    }
    if (o->num_xcd < 1)
        o->num_xcd = 1;
    return 0;
}
