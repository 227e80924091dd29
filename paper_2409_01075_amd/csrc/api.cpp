// C ABI of the runtime-shaped GEMM library: argument checks, hardware
// description, plan cache, split-K workspace, launch (Section 6.2: analytical
// selection at run time, then the grid is computed from the runtime shape).
#include <dlfcn.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <string>
#include <vector>
#include <map>
#include <mutex>
#include <unordered_map>

#include <hip/hip_runtime_api.h>

#include "vx_internal.h"

namespace {

constexpr size_t kTicketBytes = 256 * 1024;                 // 65536 arrival counters
constexpr size_t kDefaultPartials = 64ull * 1024 * 1024;   // fp32 split-K partials
constexpr int kMaxDevices = 64;

std::mutex g_mu;
std::mutex& g_calib_try_mu()
{
    static std::mutex m;
    return m;
}
std::atomic<bool> g_override_set{false};
vx_hwinfo g_override;
bool g_hw_valid[kMaxDevices];
vx_hwinfo g_hw[kMaxDevices];
std::atomic<int> g_force_id{-1};
std::atomic<int> g_force_split{0};
std::atomic<int> g_fix_wm{0}, g_fix_wn{0}, g_fix_mi{0};
std::atomic<int> g_backends{3};   // kernel backends the selector may use (vx_restrict_backends)
std::atomic<bool> g_hybrid{true};  // hybrid grids among the plans (vx_enable_hybrid_grid)
std::atomic<bool> g_krot{true};    // rotated K order in the direct-to-LDS GEMM kernels (vx_enable_k_rotation)
std::atomic<uint64_t> g_epoch{0};   // bumps when planning inputs change
std::atomic<bool> g_fail_ws_alloc{false};   // test hook: the lazy workspace allocation fails
std::atomic<bool> g_exhaustive{false};      // test switch: the search prices every pair

struct PlanKey {
    int64_t batch, M, N, K;
    int dt, vec_ok, c_vec, dev;
    size_t ws;
    int64_t tickets;
    uint64_t epoch;
    int op;
    int gather_pm;   // convolution: the share of image chunks gathered element by element, per mille
    bool operator==(const PlanKey& o) const
    {
        return batch == o.batch && M == o.M && N == o.N && K == o.K && dt == o.dt && vec_ok == o.vec_ok &&
               c_vec == o.c_vec && dev == o.dev && ws == o.ws && tickets == o.tickets && epoch == o.epoch &&
               op == o.op && gather_pm == o.gather_pm;
    }
};
uint64_t plan_hash(const PlanKey& k)
{
    uint64_t h = 1469598103934665603ull;
    auto mix = [&h](uint64_t v) { h = (h ^ v) * 1099511628211ull; };
    mix(k.batch); mix(k.M); mix(k.N); mix(k.K);
    mix(k.dt | (k.vec_ok << 4) | (k.c_vec << 5) | (k.op << 6) | ((uint64_t)k.dev << 8));
    mix(k.ws); mix(k.tickets); mix(k.epoch); mix((uint64_t)k.gather_pm);
    return h ^ (h >> 29);
}

// Plan cache: a fixed table in static storage (nothing is allocated when a
// shape is first seen), 4-way probed, under g_mu; plus each thread's last
// plan, which repeated calls of one shape find without taking the lock.
// Entries carry the planning epoch, so a change of the planning inputs
// (calibration, overrides, ablation switches, workspaces) retires them all.
constexpr int kPlanSlots = 4096;   // a power of two
constexpr int kPlanProbe = 4;
struct PlanSlot {
    PlanKey key;
    vx_plan plan;
    bool used;
};
PlanSlot g_slots[kPlanSlots];
unsigned g_slot_victim = 0;
struct LastPlan {
    PlanKey key;
    vx_plan plan;
    bool valid;
};
thread_local LastPlan t_last = {};

bool cache_find(const PlanKey& k, vx_plan* out)
{
    if (t_last.valid && t_last.key == k) {
        *out = t_last.plan;
        return true;
    }
    const uint64_t h = plan_hash(k);
    std::lock_guard<std::mutex> lk(g_mu);
    for (int i = 0; i < kPlanProbe; ++i) {
        const PlanSlot& e = g_slots[(h + i) & (kPlanSlots - 1)];
        if (e.used && e.key == k) {
            *out = e.plan;
            t_last.key = k;
            t_last.plan = e.plan;
            t_last.valid = true;
            return true;
        }
    }
    return false;
}

void cache_put(const PlanKey& k, const vx_plan& p)
{
    const uint64_t h = plan_hash(k);
    {
        std::lock_guard<std::mutex> lk(g_mu);
        int slot = -1;
        for (int i = 0; i < kPlanProbe && slot < 0; ++i) {
            const PlanSlot& e = g_slots[(h + i) & (kPlanSlots - 1)];
            if (!e.used || e.key.epoch != k.epoch || e.key == k)
                slot = (int)((h + i) & (kPlanSlots - 1));
        }
        if (slot < 0)
            slot = (int)((h + (g_slot_victim++ % kPlanProbe)) & (kPlanSlots - 1));
        g_slots[slot].key = k;
        g_slots[slot].plan = p;
        g_slots[slot].used = true;
    }
    t_last.key = k;
    t_last.plan = p;
    t_last.valid = true;
}

struct Workspace {
    char* base = nullptr;
    size_t bytes = 0;
    bool owned = false;
};
std::map<std::pair<int, void*>, Workspace> g_ws;

// ---- offline calibration of the kernels (empirical low levels) ------------
std::vector<VxCalib> g_calib;
std::vector<char> g_calib_ok;
double g_calib_launch_ns = 0.0;
std::atomic<bool> g_calib_loaded{false};
std::atomic<bool> g_calib_enabled{true};
std::atomic<bool> g_calib_tried{false};

std::string default_calib_path(const char* arch)
{
    Dl_info info;
    std::string dir = ".";
    if (dladdr((void*)&vx_version, &info) && info.dli_fname) {
        dir = info.dli_fname;
        size_t slash = dir.rfind('/');
        dir = slash == std::string::npos ? "." : dir.substr(0, slash);
    }
    return dir + "/calib_" + arch + ".txt";
}

// Parses a calibration table; accepts it only for this exact kernel set.
int load_calib_file(const char* path, const char* arch)
{
    FILE* f = fopen(path, "r");
    if (!f)
        return -1;
    int n = 0;
    vxi_registry(&n);
    std::vector<VxCalib> cal(n);
    std::vector<char> ok(n, 0);
    double launch = 0.0;
    bool hash_ok = false, arch_ok = arch == nullptr;
    int loaded = 0;
    char line[512];
    while (fgets(line, sizeof line, f)) {
        char key[64], val[128];
        if (line[0] == '#' || sscanf(line, "%63s", key) != 1)
            continue;
        if (!strcmp(key, "registry_hash") && sscanf(line, "%*s %127s", val) == 1)
            hash_ok = !strcmp(val, vxi_registry_hash());
        else if (!strcmp(key, "arch") && sscanf(line, "%*s %127s", val) == 1)
            arch_ok = arch == nullptr || !strcmp(val, arch);
        else if (!strcmp(key, "launch_ns"))
            sscanf(line, "%*s %lf", &launch);
        else if (!strcmp(key, "kernel")) {
            int id;
            VxCalib c;
            c.split_a = c.split_b = c.step_gather = c.step_gather_light = -1.0;
            if (sscanf(line, "%*s %d %lf %lf %lf %lf %lf %lf %lf %lf %lf", &id, &c.step_full, &c.fix_full,
                       &c.step_light, &c.fix_light, &c.load_light, &c.split_a, &c.split_b, &c.step_gather,
                       &c.step_gather_light) >= 6 &&
                id >= 0 && id < n && c.step_full > 0.0 && c.step_light > 0.0 && c.load_light > 0.0) {
                cal[id] = c;
                ok[id] = 1;
                ++loaded;
            }
        }
    }
    fclose(f);
    if (!hash_ok || !arch_ok || loaded == 0)
        return -2;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        g_calib.swap(cal);
        g_calib_ok.swap(ok);
        g_calib_launch_ns = launch;
    }
    g_calib_loaded.store(true);
    g_epoch.fetch_add(1);
    return loaded;
}

void ensure_calib(const vx_hwinfo& hw)
{
    if (g_calib_tried.load())
        return;
    std::lock_guard<std::mutex> lk(g_calib_try_mu());
    if (g_calib_tried.load())
        return;
    load_calib_file(default_calib_path(hw.arch).c_str(), hw.arch);
    g_calib_tried.store(true);
}

int elem_bytes(int dt) { return dt == VX_F32 ? 4 : 2; }

bool overlaps(const void* a, size_t abytes, const void* b, size_t bbytes)
{
    if (!abytes || !bbytes)
        return false;
    uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + bbytes && b0 < a0 + abytes;
}

// Extent in elements of `batch` matrices of `elems` elements at `stride`.
size_t extent(int64_t batch, int64_t stride, int64_t elems)
{
    if (batch <= 0 || elems <= 0)
        return 0;
    return (size_t)((batch - 1) * stride + elems);
}

vx_status hwinfo_for(int dev, vx_hwinfo* out)
{
    std::lock_guard<std::mutex> lk(g_mu);
    if (g_override_set) {
        *out = g_override;
        return VX_OK;
    }
    if (dev < 0 || dev >= kMaxDevices)
        return VX_ERR_HIP;
    if (!g_hw_valid[dev]) {
        if (vxi_device_hwinfo(dev, &g_hw[dev]) != 0)
            return VX_ERR_HIP;
        g_hw_valid[dev] = true;
    }
    *out = g_hw[dev];
    return VX_OK;
}

vx_status current_device(int* dev)
{
    {
        std::lock_guard<std::mutex> lk(g_mu);
        if (g_override_set) {
            *dev = -1;   // planning only; no device needed
            return VX_OK;
        }
    }
    if (hipGetDevice(dev) != hipSuccess)
        return VX_ERR_HIP;
    return VX_OK;
}

vx_status plan_for(int dev, const VxShape& sh, size_t ws_bytes, int64_t tickets, vx_plan* out)
{
    // the epoch is read before the filter: a setter changes the filter and
    // then bumps the epoch, so a plan made under a stale filter is filed
    // under a stale epoch and never found again
    const uint64_t epoch = g_epoch.load();
    const int forced = g_force_id.load();
    PlanKey key{sh.batch, sh.M, sh.N, sh.K, sh.dt, sh.vec_ok, sh.c_vec, dev, ws_bytes, tickets, epoch, sh.op,
                (int)(sh.gather_frac * 1000.0 + 0.5)};
    if (forced < 0 && cache_find(key, out))
        return VX_OK;
    VxFilter f;
    f.kernel_id = forced;
    f.split = g_force_split.load();
    f.wave_m = g_fix_wm.load();
    f.wave_n = g_fix_wn.load();
    f.mfma_m = g_fix_mi.load();
    f.backends = g_backends.load();
    f.hybrid = g_hybrid.load();
    vx_hwinfo hw;
    vx_status st = hwinfo_for(dev, &hw);
    if (st != VX_OK)
        return st;
    ensure_calib(hw);
    VxLimits lim;
    lim.ws_bytes = ws_bytes;
    lim.max_tickets = ws_bytes ? tickets : 0;
    st = vxi_select(hw, sh, lim, f, out);
    if (st == VX_OK && forced < 0)
        cache_put(key, *out);
    return st;
}

// ---- split-K workspace -------------------------------------------------------
// Default calls: one buffer per (device, stream), the caller's (vx_set_workspace)
// or allocated by the library at the first call that plans split-K.
// vx_gemm_batched_noalloc: the static scratch array of its device.  Either way
// the arrival counters come first, then the fp32 partials.
struct WsView {
    char* base;             // counters at base, partials at base + ticket_bytes
    size_t ticket_bytes;
    size_t partial_bytes;
};
std::atomic<uint64_t> g_ws_epoch{1};   // bumps when a (device, stream) workspace changes
struct LastWs {
    int dev;
    void* stream;
    uint64_t epoch;
    size_t capacity;
    Workspace ws;
    bool valid;
};
thread_local LastWs t_ws = {};

// Capacity for partials of (device, stream)'s workspace: the default size if
// the library will allocate it at first use (0 while the test hook says that
// allocation fails).
size_t ws_capacity(int dev, void* stream)
{
    const uint64_t ep = g_ws_epoch.load();
    if (g_fail_ws_alloc.load())
        return 0;
    if (t_ws.valid && t_ws.dev == dev && t_ws.stream == stream && t_ws.epoch == ep)
        return t_ws.capacity;
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_ws.find({dev, stream});
    if (it == g_ws.end())
        return kDefaultPartials;   // will be allocated on first use
    t_ws = LastWs{dev, stream, ep, it->second.bytes > kTicketBytes ? it->second.bytes - kTicketBytes : 0,
                  it->second, true};
    return t_ws.capacity;
}

vx_status ws_get(int dev, void* stream, Workspace* out)
{
    const uint64_t ep = g_ws_epoch.load();
    if (t_ws.valid && t_ws.dev == dev && t_ws.stream == stream && t_ws.epoch == ep) {
        *out = t_ws.ws;
        return VX_OK;
    }
    std::lock_guard<std::mutex> lk(g_mu);
    auto key = std::make_pair(dev, stream);
    auto it = g_ws.find(key);
    if (it != g_ws.end()) {
        *out = it->second;
        return VX_OK;
    }
    if (g_fail_ws_alloc.load())
        return VX_ERR_WORKSPACE;
    Workspace w;
    if (hipMalloc((void**)&w.base, kTicketBytes + kDefaultPartials) != hipSuccess) {
        (void)hipGetLastError();
        return VX_ERR_WORKSPACE;
    }
    w.bytes = kTicketBytes + kDefaultPartials;
    w.owned = true;
    if (hipMemsetAsync(w.base, 0, kTicketBytes, (hipStream_t)stream) != hipSuccess) {
        (void)hipFree(w.base);
        return VX_ERR_WORKSPACE;
    }
    g_ws[key] = w;
    g_ws_epoch.fetch_add(1);
    *out = w;
    return VX_OK;
}

// Per-device launch facts of the hardware description (constant unless the
// planning override changes, which bumps the epoch).
struct LastHw {
    int dev;
    uint64_t epoch;
    int num_xcd;
    double l2_bytes_per_xcd;
    bool valid;
};
thread_local LastHw t_hw = {};

// Plans shape `sh` on the current device and launches the chosen kernel with
// the operand fields of `a` (pointers, batch strides, convolution shape);
// the size and grid fields are filled in here.  scratch == nullptr: the
// (device, stream) workspace; otherwise the given buffer, and nothing is
// allocated.
vx_status plan_and_launch(const VxShape& sh, VxGemmArgs a, void* stream, const WsView* scratch)
{
    int dev = 0;
    vx_status st = current_device(&dev);
    if (st != VX_OK)
        return st;
    if (dev < 0)
        return VX_ERR_HIP;   // planning override without a device: nothing to launch on

    vx_plan plan;
    WsView ws = {nullptr, kTicketBytes, 0};
    if (scratch) {
        ws = *scratch;
        st = plan_for(dev, sh, ws.partial_bytes, (int64_t)(ws.ticket_bytes / 4), &plan);
        if (st == VX_ERR_NO_CANDIDATE && g_force_id.load() >= 0) {
            // a forced plan that only fails for want of scratch space
            vx_plan unused;
            if (plan_for(dev, sh, kDefaultPartials, (int64_t)(kTicketBytes / 4), &unused) == VX_OK)
                return VX_ERR_WORKSPACE;
        }
        if (st != VX_OK)
            return st;
        if (plan.split_k > 1 && plan.workspace_bytes > ws.partial_bytes)
            return VX_ERR_WORKSPACE;
    } else {
        st = plan_for(dev, sh, ws_capacity(dev, stream), (int64_t)(kTicketBytes / 4), &plan);
        if (st != VX_OK)
            return st;
        if (plan.split_k > 1) {
            Workspace w;
            if (ws_get(dev, stream, &w) != VX_OK) {
                st = plan_for(dev, sh, 0, 0, &plan);   // fall back to plans without split-K
                if (st != VX_OK)
                    return st;
            } else {
                ws.base = w.base;
            }
        }
    }
    int n = 0;
    const VxKernelEntry* reg = vxi_registry(&n);
    if (plan.kernel_id < 0 || plan.kernel_id >= n)
        return VX_ERR_NO_CANDIDATE;

    const uint64_t ep = g_epoch.load();
    if (!(t_hw.valid && t_hw.dev == dev && t_hw.epoch == ep)) {
        vx_hwinfo hw;
        st = hwinfo_for(dev, &hw);
        if (st != VX_OK)
            return st;
        t_hw = LastHw{dev, ep, hw.num_xcd, hw.l2_bytes_per_xcd, true};
    }

    a.M = (int)sh.M;
    a.N = (int)sh.N;
    a.K = (int)sh.K;
    a.tiles_m = (int)plan.tiles_m;
    a.tiles_n = (int)plan.tiles_n;
    a.split = plan.split_k;
    a.k_per_split = plan.k_per_split;
    a.batch = (int)sh.batch;
    a.group_m = plan.group_m;
    a.num_xcd = t_hw.num_xcd;
    a.grid = (int)plan.grid;
    a.dp_tiles = (int)plan.dp_tiles;
    // rotated K order where one batch entry's operands stay resident in an
    // XCD's L2 (the plain-ring direct-to-LDS kernels read it)
    a.krot = g_krot.load() && (double)(sh.M * sh.K + sh.K * sh.N) * elem_bytes(sh.dt) <= t_hw.l2_bytes_per_xcd ? 1 : 0;
    // the grid decode's divisors (grid_pos): XCD remap quotients per class of
    // workgroups and fast-division multipliers
    {
        const int nx = t_hw.num_xcd > 0 ? t_hw.num_xcd : 1;
        const int64_t tiles = plan.tiles_m * plan.tiles_n;
        const int64_t rest = plan.grid - plan.dp_tiles;   // the plain grid, or the hybrid's split class
        a.xq = (int)(rest / nx);
        a.xr = (int)(rest % nx);
        a.xq_dp = (int)(plan.dp_tiles / nx);
        a.xr_dp = (int)(plan.dp_tiles % nx);
        a.f_xcd = vx_fastdiv_make((unsigned)nx);
        a.f_tiles = vx_fastdiv_make((unsigned)tiles);
        a.f_split = vx_fastdiv_make((unsigned)plan.split_k);
        const int64_t rt = sh.batch * tiles - plan.dp_tiles;
        a.f_rt = vx_fastdiv_make((unsigned)(rt > 0 ? rt : 1));
        a.f_group = vx_fastdiv_make((unsigned)(plan.group_m * plan.tiles_n));
        a.f_gm = vx_fastdiv_make((unsigned)plan.group_m);
        const int64_t last = plan.tiles_m - (plan.tiles_m - 1) / plan.group_m * plan.group_m;
        a.f_gm_last = vx_fastdiv_make((unsigned)last);
    }
    a.ws = plan.split_k > 1 ? (float*)(ws.base + ws.ticket_bytes) : nullptr;
    a.tickets = plan.split_k > 1 ? (unsigned*)ws.base : nullptr;
    hipError_t e = reg[plan.kernel_id].launch(&a, plan.grid, (hipStream_t)stream);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return VX_ERR_HIP;
    }
    return VX_OK;
}

// Argument checks of a (batched) GEMM call, before any HIP call; fills the
// selector's view of the shape and the operand fields of the launch
// arguments.  *noop: nothing to compute (M, N or batch is 0).
vx_status gemm_prepare(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype, const void* A,
                       int64_t sA, const void* B, int64_t sB, void* C, int64_t sC, VxShape* sh, VxGemmArgs* a,
                       bool* noop)
{
    if (dtype != VX_F32 && dtype != VX_F16 && dtype != VX_BF16)
        return VX_ERR_UNSUPPORTED_DTYPE;
    if (batch < 0 || M < 0 || N < 0 || K < 0 || sA < 0 || sB < 0 || sC < 0)
        return VX_ERR_INVALID_ARG;
    if (M > INT32_MAX || N > INT32_MAX || K > INT32_MAX || batch > INT32_MAX)
        return VX_ERR_INVALID_ARG;
    const int eb = elem_bytes(dtype);
    const size_t ea = extent(batch, sA, M * K), eb_ = extent(batch, sB, K * N), ec = extent(batch, sC, M * N);
    if ((ea && !A) || (eb_ && !B) || (ec && !C))
        return VX_ERR_INVALID_ARG;
    if (batch > 1 && M * N > 0 && sC < M * N)
        return VX_ERR_INVALID_ARG;
    if (overlaps(C, ec * eb, A, ea * eb) || overlaps(C, ec * eb, B, eb_ * eb))
        return VX_ERR_INVALID_ARG;
    *noop = batch == 0 || M == 0 || N == 0;
    if (*noop)
        return VX_OK;
    sh->batch = batch;
    sh->M = M;
    sh->N = N;
    sh->K = K;
    sh->dt = dtype;
    const int ve = 16 / eb;
    // per operand: every row starts on a 16-byte boundary
    const bool a_vec = (K % ve == 0) && ((uintptr_t)A % 16 == 0) && (batch == 1 || sA % ve == 0);
    const bool b_vec = (N % ve == 0) && ((uintptr_t)B % 16 == 0) && (batch == 1 || sB % ve == 0);
    sh->vec_ok = (a_vec ? 1 : 0) | (b_vec ? 2 : 0);
    sh->c_vec = (N % 4 == 0) && ((uintptr_t)C % (4 * eb) == 0) && (batch == 1 || sC % 4 == 0);
    *a = VxGemmArgs{};
    a->A = A;
    a->B = B;
    a->C = C;
    a->sA = sA;
    a->sB = sB;
    a->sC = sC;
    return VX_OK;
}

}  // namespace

vx_status vxi_gemm_check(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype, const void* A,
                         int64_t sA, const void* B, int64_t sB, void* C, int64_t sC, bool* noop)
{
    VxShape sh;
    VxGemmArgs a;
    return gemm_prepare(batch, M, N, K, dtype, A, sA, B, sB, C, sC, &sh, &a, noop);
}

vx_status vxi_gemm_scratch(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype, const void* A,
                           int64_t sA, const void* B, int64_t sB, void* C, int64_t sC, void* stream,
                           void* scratch, size_t ticket_bytes, size_t partial_bytes)
{
    VxShape sh;
    VxGemmArgs a;
    bool noop = false;
    const vx_status st = gemm_prepare(batch, M, N, K, dtype, A, sA, B, sB, C, sC, &sh, &a, &noop);
    if (st != VX_OK || noop)
        return st;
    const WsView view = {(char*)scratch, ticket_bytes, partial_bytes};
    return plan_and_launch(sh, a, stream, &view);
}

namespace {

vx_status gemm_impl(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype, const void* A,
                    int64_t sA, const void* B, int64_t sB, void* C, int64_t sC, void* stream)
{
    VxShape sh;
    VxGemmArgs a;
    bool noop = false;
    const vx_status st = gemm_prepare(batch, M, N, K, dtype, A, sA, B, sB, C, sC, &sh, &a, &noop);
    if (st != VX_OK || noop)
        return st;
    return plan_and_launch(sh, a, stream, nullptr);
}

int64_t conv_out_dim(int64_t in, int64_t k, int64_t stride, int64_t pad, int64_t dil)
{
    const int64_t span = in + 2 * pad - dil * (k - 1) - 1;
    return span < 0 ? 0 : span / stride + 1;
}

// Checks a convolution descriptor and maps it to its implicit-GEMM shape;
// fills the convolution fields of `a`.  Sets *empty for an empty output.
vx_status conv_shape(const vx_conv2d_desc* d, VxShape* sh, VxGemmArgs* a, bool* empty)
{
    if (!d)
        return VX_ERR_INVALID_ARG;
    if (d->dtype != VX_F32 && d->dtype != VX_F16 && d->dtype != VX_BF16)
        return VX_ERR_UNSUPPORTED_DTYPE;
    if (d->n < 0 || d->h < 0 || d->w < 0 || d->c_in < 0 || d->c_out < 0 || d->kh < 1 || d->kw < 1 ||
        d->stride_h < 1 || d->stride_w < 1 || d->pad_h < 0 || d->pad_w < 0 || d->dil_h < 1 || d->dil_w < 1)
        return VX_ERR_INVALID_ARG;
    const int64_t lim = INT32_MAX, span_lim = (int64_t)1 << 30;
    if (d->h >= span_lim || d->w >= span_lim || d->pad_h >= span_lim || d->pad_w >= span_lim ||
        d->h + 2 * d->pad_h >= span_lim || d->w + 2 * d->pad_w >= span_lim || d->kh > lim || d->kw > lim ||
        d->stride_h > lim || d->stride_w > lim || d->dil_h > lim || d->dil_w > lim)
        return VX_ERR_INVALID_ARG;
    const int64_t oh = conv_out_dim(d->h, d->kh, d->stride_h, d->pad_h, d->dil_h);
    const int64_t ow = conv_out_dim(d->w, d->kw, d->stride_w, d->pad_w, d->dil_w);
    // every element index the kernels form stays within 32 bits, except the
    // image offset, which they form in 64 bits
    const double M = (double)d->n * oh * ow, K = (double)d->kh * d->kw * d->c_in;
    if (M > lim || K > lim || d->c_out > lim || M * d->c_out > lim || K * d->c_out > lim ||
        (double)d->n * d->h * d->w * d->c_in > 9.0e15)
        return VX_ERR_INVALID_ARG;
    *empty = M == 0 || d->c_out == 0;
    sh->batch = 1;
    sh->M = (int64_t)M;
    sh->N = d->c_out;
    sh->K = (int64_t)K;
    sh->dt = d->dtype;
    // 16-byte chunks of 8 channels for the direct-to-LDS kernels, whose
    // image offsets are 32-bit (operand alignment is checked by the caller
    // that has the pointers); vec_ok is part of the plan cache's key
    sh->a_bytes = (int64_t)((double)d->n * d->h * d->w * d->c_in) * elem_bytes(d->dtype);
    // bit 0: the image (16-byte chunks of 8 channels, 32-bit image offsets);
    // bit 1: the filter (rows of c_out elements)
    sh->vec_ok = (d->dtype != VX_F32 && d->c_in % 8 == 0 && sh->a_bytes < ((int64_t)1 << 31) ? 1 : 0) |
                 (d->dtype != VX_F32 && d->c_out % 8 == 0 ? 2 : 0);
    // the kernels that gather the image through VGPRs load a 16-byte chunk
    // (ve consecutive k) as one vector when the channels come in whole chunks,
    // or when, with unit width dilation, the chunk stays inside the kw * c_in
    // contiguous elements of one filter row; otherwise element by element.
    // Chunk starts fall evenly over a filter row, so (ve - 1) of every kw * c_in
    // positions cross its end (taps in the padding aside)
    {
        const int ve = 16 / elem_bytes(d->dtype);
        const double run = (double)d->kw * (double)d->c_in;
        sh->gather_frac = d->c_in % ve == 0 ? 0.0 : (d->dil_w != 1 || run < ve) ? 1.0 : std::min(1.0, (ve - 1) / run);
    }
    sh->c_vec = 0;
    sh->op = 1;
    a->cH = (int)d->h;
    a->cW = (int)d->w;
    a->cC = (int)d->c_in;
    a->cKW = (int)d->kw;
    a->cOH = (int)oh;
    a->cOW = (int)ow;
    a->csh = (int)d->stride_h;
    a->csw = (int)d->stride_w;
    a->cph = (int)d->pad_h;
    a->cpw = (int)d->pad_w;
    a->cdh = (int)d->dil_h;
    a->cdw = (int)d->dil_w;
    return VX_OK;
}

}  // namespace

uint64_t vxi_plan_epoch(void) { return g_epoch.load(); }

bool vxi_exhaustive_search(void) { return g_exhaustive.load(std::memory_order_relaxed); }

const VxCalib* vxi_calib(int kernel_id)
{
    if (!g_calib_loaded.load() || !g_calib_enabled.load())
        return nullptr;
    if (kernel_id < 0 || kernel_id >= (int)g_calib_ok.size() || !g_calib_ok[kernel_id])
        return nullptr;
    return &g_calib[kernel_id];
}

double vxi_calib_launch_ns(const vx_hwinfo& hw)
{
    if (g_calib_loaded.load() && g_calib_enabled.load() && g_calib_launch_ns > 0.0)
        return g_calib_launch_ns;
    return hw.launch_ns;
}

extern "C" {

vx_status vx_calibration_load(const char* path, int* n_loaded)
{
    vx_hwinfo hw;
    const char* arch = nullptr;
    int dev = 0;
    if (current_device(&dev) == VX_OK && hwinfo_for(dev, &hw) == VX_OK)
        arch = hw.arch;
    std::string p = path ? std::string(path) : default_calib_path(arch ? arch : "gfx950");
    g_calib_tried.store(true);
    const int n = load_calib_file(p.c_str(), path ? nullptr : arch);
    if (n <= 0 && !path) {
        // no usable default table: the selector is purely analytical
        g_calib_loaded.store(false);
        std::lock_guard<std::mutex> lk(g_mu);
        g_epoch.fetch_add(1);
    }
    if (n_loaded)
        *n_loaded = n > 0 ? n : 0;
    return n > 0 ? VX_OK : VX_ERR_INVALID_ARG;
}

vx_status vx_selector_exhaustive(int enable)
{
    g_exhaustive.store(enable != 0);
    std::lock_guard<std::mutex> lk(g_mu);
    g_epoch.fetch_add(1);
    return VX_OK;
}

vx_status vx_calibration_enable(int enable)
{
    g_calib_enabled.store(enable != 0);
    std::lock_guard<std::mutex> lk(g_mu);
    g_epoch.fetch_add(1);
    return VX_OK;
}

int vx_calibration_active(void)
{
    return (g_calib_loaded.load() && g_calib_enabled.load()) ? 1 : 0;
}

const char* vx_registry_hash(void) { return vxi_registry_hash(); }

vx_status vx_kernel_occupancy(int kernel_id, int* wgs_per_cu)
{
    int n = 0;
    const VxKernelEntry* reg = vxi_registry(&n);
    if (!wgs_per_cu || kernel_id < 0 || kernel_id >= n)
        return VX_ERR_INVALID_ARG;
    int dev = 0;
    vx_status st = current_device(&dev);
    if (st != VX_OK)
        return st;
    vx_hwinfo hw;
    st = hwinfo_for(dev, &hw);
    if (st != VX_OK)
        return st;
    *wgs_per_cu = vxi_occupancy(hw, reg[kernel_id].info);
    return VX_OK;
}


vx_status vx_gemm(int64_t M, int64_t N, int64_t K, vx_dtype dtype, const void* A, const void* B, void* C,
                  void* stream)
{
    return gemm_impl(1, M, N, K, dtype, A, M * K, B, K * N, C, M * N, stream);
}

vx_status vx_gemm_batched(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype, const void* A,
                          int64_t strideA, const void* B, int64_t strideB, void* C, int64_t strideC,
                          void* stream)
{
    return gemm_impl(batch, M, N, K, dtype, A, strideA, B, strideB, C, strideC, stream);
}

vx_status vx_plan_query(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype, int64_t strideA,
                        int64_t strideB, int64_t strideC, uint64_t base_align, vx_plan* out)
{
    if (dtype != VX_F32 && dtype != VX_F16 && dtype != VX_BF16)
        return VX_ERR_UNSUPPORTED_DTYPE;
    if (!out || batch < 1 || M < 1 || N < 1 || K < 0 || strideA < 0 || strideB < 0 || strideC < 0)
        return VX_ERR_INVALID_ARG;
    if (M > INT32_MAX || N > INT32_MAX || K > INT32_MAX || batch > INT32_MAX)
        return VX_ERR_INVALID_ARG;
    if (base_align == 0)
        base_align = 256;
    const int eb = elem_bytes(dtype), ve = 16 / eb;
    VxShape sh;
    sh.batch = batch;
    sh.M = M;
    sh.N = N;
    sh.K = K;
    sh.dt = dtype;
    const bool a_vec = (K % ve == 0) && (base_align % 16 == 0) && (batch == 1 || strideA % ve == 0);
    const bool b_vec = (N % ve == 0) && (base_align % 16 == 0) && (batch == 1 || strideB % ve == 0);
    sh.vec_ok = (a_vec ? 1 : 0) | (b_vec ? 2 : 0);
    sh.c_vec = (N % 4 == 0) && (base_align % (4 * eb) == 0) && (batch == 1 || strideC % 4 == 0);
    int dev = 0;
    vx_status st = current_device(&dev);
    if (st != VX_OK)
        return st;
    const size_t cap = g_fail_ws_alloc.load() ? 0 : dev < 0 ? kDefaultPartials : ws_capacity(dev, nullptr);
    return plan_for(dev, sh, cap, (int64_t)(kTicketBytes / 4), out);
}

vx_status vx_conv2d(const vx_conv2d_desc* d, const void* x, const void* w, void* y, void* stream)
{
    VxShape sh;
    VxGemmArgs a = {};
    bool empty = false;
    vx_status st = conv_shape(d, &sh, &a, &empty);
    if (st != VX_OK)
        return st;
    const int eb = elem_bytes(d->dtype);
    const size_t ex = (size_t)(d->n * d->h * d->w * d->c_in), ew = (size_t)(d->kh * d->kw * d->c_in * d->c_out);
    const size_t ey = (size_t)(sh.M * sh.N);
    if ((ex && !empty && sh.K && !x) || (ew && !empty && !w) || (ey && !y))
        return VX_ERR_INVALID_ARG;
    if (overlaps(y, ey * eb, x, ex * eb) || overlaps(y, ey * eb, w, ew * eb))
        return VX_ERR_INVALID_ARG;
    if (empty)
        return VX_OK;
    sh.vec_ok &= ((uintptr_t)x % 16 == 0 ? 1 : 0) | ((uintptr_t)w % 16 == 0 ? 2 : 0);
    a.A = x;
    a.B = w;
    a.C = y;
    return plan_and_launch(sh, a, stream, nullptr);
}

vx_status vx_conv2d_output_dims(const vx_conv2d_desc* d, int64_t* oh, int64_t* ow)
{
    VxShape sh;
    VxGemmArgs a = {};
    bool empty = false;
    if (!oh || !ow)
        return VX_ERR_INVALID_ARG;
    vx_status st = conv_shape(d, &sh, &a, &empty);
    if (st != VX_OK)
        return st;
    *oh = a.cOH;
    *ow = a.cOW;
    return VX_OK;
}

vx_status vx_conv2d_plan_query(const vx_conv2d_desc* d, vx_plan* out)
{
    VxShape sh;
    VxGemmArgs a = {};
    bool empty = false;
    vx_status st = conv_shape(d, &sh, &a, &empty);
    if (st != VX_OK)
        return st;
    if (!out || empty)
        return VX_ERR_INVALID_ARG;
    int dev = 0;
    st = current_device(&dev);
    if (st != VX_OK)
        return st;
    const size_t cap = g_fail_ws_alloc.load() ? 0 : dev < 0 ? kDefaultPartials : ws_capacity(dev, nullptr);
    return plan_for(dev, sh, cap, (int64_t)(kTicketBytes / 4), out);
}

vx_status vx_plan_cost(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype, int kernel_id,
                       int split_k, int align, double* out_ns)
{
    if (dtype != VX_F32 && dtype != VX_F16 && dtype != VX_BF16)
        return VX_ERR_UNSUPPORTED_DTYPE;
    if (!out_ns || batch < 1 || M < 1 || N < 1 || K < 0)
        return VX_ERR_INVALID_ARG;
    int n = 0;
    const VxKernelEntry* reg = vxi_registry(&n);
    if (kernel_id < 0 || kernel_id >= n)
        return VX_ERR_NO_CANDIDATE;
    int dev = 0;
    vx_status st = current_device(&dev);
    if (st != VX_OK)
        return st;
    vx_hwinfo hw;
    st = hwinfo_for(dev, &hw);
    if (st != VX_OK)
        return st;
    if (align < 0 || align > 3)
        return VX_ERR_INVALID_ARG;
    ensure_calib(hw);   // the same model as the selector's, from the first call on
    VxShape sh{batch, M, N, K, (int)dtype, align, 1};
    VxLimits lim{kDefaultPartials, (int64_t)(kTicketBytes / 4)};
    const double c = vxi_cost(hw, sh, reg[kernel_id].info, split_k, lim, nullptr);
    if (c < 0.0)
        return VX_ERR_NO_CANDIDATE;
    *out_ns = c;
    return VX_OK;
}

vx_status vx_get_hwinfo(vx_hwinfo* out)
{
    if (!out)
        return VX_ERR_INVALID_ARG;
    int dev = 0;
    vx_status st = current_device(&dev);
    if (st != VX_OK)
        return st;
    return hwinfo_for(dev, out);
}

vx_status vx_set_hwinfo_override(const vx_hwinfo* hw)
{
    if (hw && (hw->num_cu < 1 || hw->simd_per_cu < 1 || hw->lds_bytes_per_cu < 1 || hw->clock_ghz <= 0.0 ||
               hw->hbm_gbps <= 0.0 || hw->vgprs_per_lane < 1 || hw->max_waves_per_simd < 1 ||
               hw->mfma_flop_clk_cu_f16 <= 0.0 || hw->mfma_flop_clk_cu_f32 <= 0.0 ||
               hw->l2_bytes_clk_cu <= 0.0 || hw->lds_bytes_clk_cu <= 0.0 || hw->num_xcd < 1))
        return VX_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lk(g_mu);
    g_override_set = hw != nullptr;
    if (hw)
        g_override = *hw;
    g_epoch.fetch_add(1);
    return VX_OK;
}

int vx_registry_count(void)
{
    int n = 0;
    vxi_registry(&n);
    return n;
}

vx_status vx_registry_get(int id, vx_kernel_info* out)
{
    int n = 0;
    const VxKernelEntry* reg = vxi_registry(&n);
    if (!out || id < 0 || id >= n)
        return VX_ERR_INVALID_ARG;
    *out = reg[id].info;
    return VX_OK;
}

vx_status vx_force_plan(int kernel_id, int split_k)
{
    if (kernel_id >= vx_registry_count())
        return VX_ERR_NO_CANDIDATE;
    g_force_id.store(kernel_id < 0 ? -1 : kernel_id);
    g_force_split.store(kernel_id < 0 ? 0 : split_k);
    return VX_OK;
}

vx_status vx_restrict_backends(int mask)
{
    if (mask < 0 || mask > 3)
        return VX_ERR_INVALID_ARG;
    if (mask == 0)
        mask = 3;
    int n = 0;
    const VxKernelEntry* reg = vxi_registry(&n);
    bool any = false;
    for (int i = 0; i < n && !any; ++i)
        any = reg[i].info.enabled && (mask & (reg[i].info.family == 2 ? 2 : 1));
    if (!any)
        return VX_ERR_NO_CANDIDATE;
    std::lock_guard<std::mutex> lk(g_mu);
    g_backends.store(mask);
    g_epoch.fetch_add(1);
    return VX_OK;
}

vx_status vx_enable_hybrid_grid(int enable)
{
    std::lock_guard<std::mutex> lk(g_mu);
    g_hybrid.store(enable != 0);
    g_epoch.fetch_add(1);
    return VX_OK;
}

vx_status vx_enable_k_rotation(int enable)
{
    // launch-time only: plans do not depend on it
    g_krot.store(enable != 0);
    return VX_OK;
}

vx_status vx_fix_wavefront(int wave_m, int wave_n, int mfma_m)
{
    if (wave_m == 0 && wave_n == 0 && mfma_m == 0) {
        std::lock_guard<std::mutex> lk(g_mu);
        g_fix_wm.store(0);
        g_fix_wn.store(0);
        g_fix_mi.store(0);
        g_epoch.fetch_add(1);
        return VX_OK;
    }
    if (wave_m <= 0 || wave_n <= 0 || mfma_m <= 0)
        return VX_ERR_INVALID_ARG;
    VxFilter f;
    f.wave_m = wave_m;
    f.wave_n = wave_n;
    f.mfma_m = mfma_m;
    int n = 0;
    const VxKernelEntry* reg = vxi_registry(&n);
    bool any = false;
    for (int i = 0; i < n && !any; ++i)
        any = reg[i].info.enabled && vxi_wave_matches(f, reg[i].info);
    if (!any)
        return VX_ERR_NO_CANDIDATE;
    std::lock_guard<std::mutex> lk(g_mu);
    g_fix_wm.store(wave_m);
    g_fix_wn.store(wave_n);
    g_fix_mi.store(mfma_m);
    g_epoch.fetch_add(1);
    return VX_OK;
}

vx_status vx_test_fail_workspace_alloc(int fail)
{
    g_fail_ws_alloc.store(fail != 0);
    g_epoch.fetch_add(1);
    return VX_OK;
}

vx_status vx_set_workspace(void* ptr, size_t bytes, void* stream)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return VX_ERR_HIP;
    if (ptr && bytes < kTicketBytes)
        return VX_ERR_INVALID_ARG;
    if ((uintptr_t)ptr % 256)
        return VX_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lk(g_mu);
    auto key = std::make_pair(dev, stream);
    auto it = g_ws.find(key);
    if (it != g_ws.end()) {
        if (it->second.owned) {
            // the stream may still be using it: free after the stream's work
            if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess)
                return VX_ERR_HIP;
            (void)hipFree(it->second.base);
        }
        g_ws.erase(it);
    }
    if (ptr) {
        if (hipMemsetAsync(ptr, 0, kTicketBytes, (hipStream_t)stream) != hipSuccess)
            return VX_ERR_HIP;
        Workspace w;
        w.base = (char*)ptr;
        w.bytes = bytes;
        w.owned = false;
        g_ws[key] = w;
    }
    g_ws_epoch.fetch_add(1);
    g_epoch.fetch_add(1);
    return VX_OK;
}

const char* vx_status_string(vx_status s)
{
    switch (s) {
    case VX_OK: return "VX_OK";
    case VX_ERR_INVALID_ARG: return "VX_ERR_INVALID_ARG";
    case VX_ERR_UNSUPPORTED_DTYPE: return "VX_ERR_UNSUPPORTED_DTYPE";
    case VX_ERR_NO_CANDIDATE: return "VX_ERR_NO_CANDIDATE";
    case VX_ERR_WORKSPACE: return "VX_ERR_WORKSPACE";
    case VX_ERR_HIP: return "VX_ERR_HIP";
    }
    return "VX_ERR_UNKNOWN";
}

const char* vx_version(void) { return "vx 0.1 (gfx950)"; }

}  // extern "C"
