"""Host-side checks of the C-ABI library: it loads, exports every declared
symbol with the declared struct layouts, validates arguments before touching
the GPU, and its registry satisfies the candidate-generation invariants."""
import os
import re
import subprocess
import sys

import pytest

from paper_2409_01075_amd import vx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vx.h")


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(vx_[a-z_0-9]+)\s*\(", src)))


def test_library_loads_and_exports_every_declared_symbol():
    L = vx.lib()
    names = _declared_functions()
    assert len(names) >= 14
    missing = [n for n in names if not hasattr(L, n)]
    assert not missing, missing
    # and nm agrees that they are real dynamic exports
    out = subprocess.run(["nm", "-D", "--defined-only", vx.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (vx_[a-z_0-9]+)\b", out))
    assert set(names) <= exported, set(names) - exported


def test_shipped_calibration_matches_the_built_kernels():
    """The per-device table that ships beside the library was measured on
    exactly the kernel set that is built: a stale table would silently turn
    the hybrid analyzer back into the purely analytical one."""
    path = os.path.join(os.path.dirname(vx.LIB_PATH), "calib_gfx950.txt")
    assert os.path.exists(path)
    kv = dict(ln.split(None, 1) for ln in open(path) if ln.strip() and not ln.startswith("#") and " " in ln)
    assert kv["registry_hash"].strip() == vx.vx_registry_hash()
    st, n = vx.vx_calibration_load(path)
    try:
        assert st == 0 and n == sum(vx.vx_registry_get(i).enabled for i in range(vx.vx_registry_count()))
    finally:
        vx.vx_calibration_load(None)


def test_calibration_file_rules(tmp_path):
    """A calibration table is accepted only for this exact kernel set, and
    changes the cost model's answer; disabling it restores the analytical one."""
    assert vx.vx_set_hwinfo_override(vx.mi355x_hwinfo()) == 0
    try:
        vx.vx_calibration_enable(False)
        p_an = vx.vx_plan_query(1, 4096, 4096, 4096, 1)
        vx.vx_calibration_enable(True)
        bad = tmp_path / "bad.txt"
        bad.write_text("arch gfx950\nregistry_hash 0000\nlaunch_ns 1600\nkernel 0 100 100 100 100 0.1\n")
        st, n = vx.vx_calibration_load(str(bad))
        assert st != 0 and n == 0
        good = tmp_path / "good.txt"
        lines = ["arch gfx950", "registry_hash %s" % vx.vx_registry_hash(), "launch_ns 1600"]
        for i in range(vx.vx_registry_count()):
            k = vx.vx_registry_get(i)
            # a table that makes one kernel per dtype far cheaper than the rest
            fast = (k.mb, k.nb, k.kb, k.wm, k.wn) == (64, 64, 64, 2, 2)
            step = 10.0 if fast else 10000.0
            lines.append("kernel %d %.1f %.1f %.1f %.1f %.5f" % (i, step, 500.0, step, 500.0, 0.125))
        good.write_text("\n".join(lines) + "\n")
        st, n = vx.vx_calibration_load(str(good))
        assert st == 0 and n == vx.vx_registry_count()
        assert vx.vx_calibration_active() == 1
        p_cal = vx.vx_plan_query(1, 4096, 4096, 4096, 1)
        assert (p_cal.kernel.mb, p_cal.kernel.nb, p_cal.kernel.kb) == (64, 64, 64)
        # the argmin still holds against the model it uses
        st, c = vx.vx_plan_cost(1, 4096, 4096, 4096, 1, p_cal.kernel_id, p_cal.split_k, 3)
        assert st == 0 and c == pytest.approx(p_cal.predicted_ns)
        vx.vx_calibration_enable(False)
        assert vx.vx_calibration_active() == 0
        p_off = vx.vx_plan_query(1, 4096, 4096, 4096, 1)
        assert (p_off.kernel_id, p_off.split_k) == (p_an.kernel_id, p_an.split_k)
    finally:
        vx.vx_calibration_enable(True)
        vx.vx_calibration_load(None)   # back to the default file (if any)
        vx.vx_set_hwinfo_override(None)


def test_struct_layouts_match_header(tmp_path):
    import ctypes
    probe = tmp_path / "probe.c"
    probe.write_text("""
#include <stdio.h>
#include <stddef.h>
#include "vx.h"
int main(void) {
  printf("%zu %zu %zu %zu %zu %zu\\n", sizeof(vx_hwinfo), sizeof(vx_kernel_info), sizeof(vx_plan),
         offsetof(vx_plan, predicted_ns), offsetof(vx_plan, kernel), offsetof(vx_hwinfo, clock_ghz));
  return 0;
}
""")
    exe = tmp_path / "probe"
    subprocess.run(["gcc", "-I", os.path.dirname(HEADER), str(probe), "-o", str(exe)], check=True)
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True).stdout.split()]
    want = [ctypes.sizeof(vx.vx_hwinfo), ctypes.sizeof(vx.vx_kernel_info), ctypes.sizeof(vx.vx_plan),
            vx.vx_plan.predicted_ns.offset, vx.vx_plan.kernel.offset, vx.vx_hwinfo.clock_ghz.offset]
    assert got == want


def test_argument_errors_without_gpu():
    F16 = vx.VX_F16
    assert vx.vx_gemm(4, 4, 4, 7, 16, 1024, 4096, None) == 2          # unsupported dtype
    assert vx.vx_gemm(-1, 4, 4, F16, 16, 1024, 4096, None) == 1       # negative M
    assert vx.vx_gemm(4, -4, 4, F16, 16, 1024, 4096, None) == 1
    assert vx.vx_gemm(4, 4, -4, F16, 16, 1024, 4096, None) == 1
    assert vx.vx_gemm(4, 4, 4, F16, None, 1024, 4096, None) == 1      # NULL A with M*K > 0
    assert vx.vx_gemm(4, 4, 4, F16, 16, None, 4096, None) == 1
    assert vx.vx_gemm(4, 4, 4, F16, 16, 1024, None, None) == 1
    assert vx.vx_gemm(4, 4, 4, F16, 4096, 1024, 4100, None) == 1      # C overlaps A
    assert vx.vx_gemm(4, 4, 4, F16, 16, 4096, 4090, None) == 1        # C overlaps B
    assert vx.vx_gemm(2 ** 31, 4, 4, F16, 16, 1024, 4096, None) == 1  # beyond int32 dims
    assert vx.vx_gemm_batched(-1, 4, 4, 4, F16, 16, 16, 1024, 16, 4096, 16, None) == 1
    assert vx.vx_gemm_batched(2, 4, 4, 4, F16, 16, 16, 1024, 16, 4096, 8, None) == 1  # C batches overlap
    assert vx.vx_gemm_batched(2, 4, 4, 4, F16, 16, -16, 1024, 16, 4096, 16, None) == 1
    # empty problems are no-ops that never reach the device
    assert vx.vx_gemm(0, 4, 4, F16, None, 1024, None, None) == 0
    assert vx.vx_gemm(4, 0, 4, F16, 16, None, None, None) == 0
    assert vx.vx_gemm_batched(0, 4, 4, 4, F16, None, 16, None, 16, None, 16, None) == 0
    for s in range(6):
        assert vx.vx_status_string(s).startswith("VX_")


def test_cost_model_golden_cases():
    path = os.path.join(ROOT, "tests", "golden", "cost_model_cases.txt")
    n = 0
    for ln in open(path):
        if not ln.strip() or ln.startswith("#"):
            continue
        f = ln.split()
        if f[0] == "temporal":
            got = vx.vx_cost_temporal(float(f[1]), int(f[2]), float(f[3]), float(f[4]))
            assert got == pytest.approx(float(f[5]), abs=0, rel=1e-15), ln
        else:
            assert vx.vx_cost_parallel_factor(int(f[1]), int(f[2])) == int(f[3]), ln
        n += 1
    assert n >= 10
    assert vx.vx_cost_parallel_factor(5, 0) == -1


def test_registry_invariants():
    n = vx.vx_registry_count()
    assert n > 0
    isa = {0: {(16, 16, 4), (32, 32, 2)}, 1: {(16, 16, 32), (32, 32, 16)}, 2: {(16, 16, 32), (32, 32, 16)}}
    seen = set()
    valu = 0
    for i in range(n):
        k = vx.vx_registry_get(i)
        assert k.id == i
        if k.family == 2:
            # vector-ALU backend: one wave covers 8 column chunks of 16 bytes x 8 k groups,
            # Kb = waves x 8 groups x (2 rows per dot2 pair for 16-bit) x groups per lane
            valu += 1
            eb = 4 if k.dtype == 0 else 2
            assert (k.mfma_m, k.mfma_n, k.mfma_k) == (0, 0, 0) and k.wm == 1 and k.vec == 1
            assert k.nb == 8 * (16 // eb) and k.mb in (4, 8, 16)
            assert k.kb == k.wn * 8 * (2 if eb == 2 else 1) * k.stages
            assert k.k_max > 0 and k.k_max % k.kb == 0 and k.k_max * k.mb * eb <= k.lds_bytes <= 160 * 1024
            assert k.threads == 64 * k.wn and k.enabled == (1 if k.scratch_bytes == 0 else 0)
            continue
        assert k.k_max == 0
        assert (k.mfma_m, k.mfma_n, k.mfma_k) in isa[k.dtype]                  # L0: FilterByISA
        mw, nw = k.mb // k.wm, k.nb // k.wn
        assert k.mb == k.wm * mw and k.nb == k.wn * nw                          # L2 multiple of L1
        assert mw % k.mfma_m == 0 and nw % k.mfma_n == 0                        # L1 multiple of L0
        assert k.kb % k.mfma_k == 0
        assert k.threads == 64 * k.wm * k.wn <= 1024
        assert k.lds_bytes <= 160 * 1024
        assert k.enabled == (1 if k.scratch_bytes == 0 else 0)
        assert k.vgprs + k.agprs <= 512 and k.vgprs > 0
        assert k.vec == (1 if k.align == 3 else 0)
        if k.family == 1:
            assert k.align in (1, 2, 3)        # at least one operand moves by DMA
        seen.add((k.dtype, k.vec))
    assert seen == {(d, v) for d in (0, 1, 2) for v in (0, 1)}
    assert valu > 0
    enabled = sum(vx.vx_registry_get(i).enabled for i in range(n))
    assert enabled >= 0.9 * n


def test_candidate_generator_properties():
    sys.path.insert(0, os.path.join(ROOT, "paper_2409_01075_amd", "csrc"))
    try:
        import candidates as C
    finally:
        sys.path.pop(0)
    for dt in ("f16", "bf16", "f32"):
        l0 = C.mfma_tiles(dt)
        assert set(l0) == set(C.GFX950["mfma"][dt])
        for fam in ("reg", "dma"):
            l1 = C.wave_tiles(dt, family=fam)
            for c, below in l1.items():
                assert below and all(c[0] % p[0] == 0 and c[1] % p[1] == 0 for p in below)
                assert set(below) <= set(l0)
                assert 4 <= c[0] * c[1] // 64 <= (256 if fam == "dma" else 128)
            # every multiple of an L0 tile within the budget is present (nothing dropped)
            for mw in (16, 32, 64, 128):
                for nw in (16, 32, 64, 128):
                    if 4 <= mw * nw // 64 <= 128 and max(mw, nw) <= 4 * min(mw, nw):
                        assert (mw, nw) in l1
            if fam == "dma" and dt == "f32":
                continue
            l2 = C.workgroup_tiles(dt, family=fam)
            assert l2
            for c, links in l2.items():
                mb, nb, kb, wm, wn, mi = c
                for (w, l0c) in links:
                    assert w in l1 and mb == wm * w[0] and nb == wn * w[1]
                    assert kb % l0c[2] == 0 and l0c in l0 and l0c[0] == mi
                assert C.lds_bytes(dt, mb, nb, kb) <= C.GFX950["lds_bytes"]
    reg = C.registry()
    assert len(reg) == vx.vx_registry_count()


@pytest.fixture
def mi355x_override():
    assert vx.vx_set_hwinfo_override(vx.mi355x_hwinfo()) == 0
    yield
    assert vx.vx_set_hwinfo_override(None) == 0


def _shapes():
    import numpy as np
    g = np.random.default_rng(5)
    out = [(1, 1, 1, 1), (1, 77, 96, 80), (1, 1, 768, 768), (1, 512, 768, 768), (1, 8192, 11008, 4096),
           (192, 1000, 1000, 64), (192, 1000, 64, 1000), (1, 5, 3, 0), (3, 7, 9, 11)]
    for _ in range(60):
        out.append((int(g.integers(1, 4)), int(g.integers(1, 5000)), int(g.integers(1, 5000)),
                    int(g.integers(0, 12000))))
    return out


def test_selector_plans_cover_and_are_feasible(mi355x_override):
    for dt in (0, 1, 2):
        for (b, M, N, K) in _shapes():
            for align in (256, 2):
                p = vx.vx_plan_query(b, M, N, K, dt, base_align=align)
                k = p.kernel
                assert k.enabled and k.dtype == dt
                ve = 8 if dt else 4
                if align == 2:
                    assert k.align == 0 and k.vec == 0
                if k.align & 1:
                    assert K % ve == 0
                if k.align & 2:
                    assert N % ve == 0
                assert p.tiles_m * k.mb >= M and (p.tiles_m - 1) * k.mb < M
                assert p.tiles_n * k.nb >= N and (p.tiles_n - 1) * k.nb < N
                tiles = p.tiles_m * p.tiles_n * b
                assert 0 <= p.dp_tiles < tiles
                if p.dp_tiles:
                    # hybrid grid: whole waves of whole tiles, the rest split
                    occ = vx.vx_kernel_occupancy(p.kernel_id)
                    assert p.split_k >= 2 and p.dp_tiles % (256 * occ) == 0
                assert p.grid == p.dp_tiles + (tiles - p.dp_tiles) * p.split_k
                if K == 0:
                    assert p.split_k == 1
                else:
                    assert p.k_per_split % k.kb == 0
                    assert p.split_k * p.k_per_split >= K > (p.split_k - 1) * p.k_per_split
                if p.split_k > 1:
                    assert p.workspace_bytes == (tiles - p.dp_tiles) * p.split_k * k.mb * k.nb * 4
                    assert p.workspace_bytes <= 64 * 2 ** 20
                    assert p.tiles_m * p.tiles_n * b <= 65536
                assert p.predicted_ns > 0
                # deterministic
                q = vx.vx_plan_query(b, M, N, K, dt, base_align=align)
                assert (q.kernel_id, q.split_k, q.dp_tiles) == (p.kernel_id, p.split_k, p.dp_tiles)


def test_selector_is_the_argmin_of_the_cost_model(mi355x_override):
    """Equation 1: the chosen plan has the lowest modelled cost of every
    (kernel, split, grid) triple, found here by brute force through
    vx_plan_cost (a negative split prices the hybrid grid)."""
    n = vx.vx_registry_count()
    splits = [1, 2, 3, 4, 5, 6, 8, 10, 12, 16, 20, 24, 32]
    splits += [-s for s in splits if s > 1]
    for dt, (b, M, N, K) in [(1, (1, 1, 768, 768)), (1, (1, 300, 768, 768)), (2, (1, 8192, 4096, 4096)),
                             (2, (192, 333, 333, 64)), (2, (192, 336, 336, 64)), (0, (1, 77, 96, 80)), (2, (1, 16, 11008, 4096))]:
        p = vx.vx_plan_query(b, M, N, K, dt)
        ve = 8 if dt else 4
        vec_ok = int(K % ve == 0 and (b == 1 or M * K % ve == 0)) | 2 * int(N % ve == 0 and (b == 1 or K * N % ve == 0))
        best = min(c for i in range(n) for s in splits
                   for st, c in [vx.vx_plan_cost(b, M, N, K, dt, i, s, vec_ok)] if st == 0)
        assert p.predicted_ns == pytest.approx(best, rel=1e-12)
        st, c = vx.vx_plan_cost(b, M, N, K, dt, p.kernel_id, -p.split_k if p.dp_tiles else p.split_k, vec_ok)
        assert st == 0 and c == pytest.approx(p.predicted_ns, rel=1e-12)


def test_selector_responds_to_hardware(mi355x_override):
    """A device with a quarter of the CUs gets plans with no more workgroups
    per CU slot wasted: the model must see the smaller machine."""
    h = vx.mi355x_hwinfo()
    p_full = vx.vx_plan_query(1, 16, 4096, 4096, 2)
    h.num_cu = 64
    assert vx.vx_set_hwinfo_override(h) == 0
    p_small = vx.vx_plan_query(1, 16, 4096, 4096, 2)
    assert p_small.predicted_ns > p_full.predicted_ns
    assert p_small.grid <= p_full.grid


def test_force_plan_validation():
    assert vx.vx_force_plan(vx.vx_registry_count(), 1) == 3
    assert vx.vx_force_plan(0, 2) == 0
    assert vx.vx_force_plan(-1, 0) == 0


def test_fix_wavefront_restricts_the_argmin(mi355x_override):
    """The Static1 ablation: with a fixed wavefront strategy the selector
    returns the cheapest plan among exactly the kernels that have it, and
    lifting the restriction restores the unrestricted plan."""
    assert vx.vx_fix_wavefront(32, 0, 16) == 1
    assert vx.vx_fix_wavefront(-32, 32, 16) == 1
    assert vx.vx_fix_wavefront(24, 24, 16) == 3
    reg = [k for k in (vx.vx_registry_get(i) for i in range(vx.vx_registry_count())) if k.op == 0]

    def wave(k):
        return (k.mb // k.wm, k.nb // k.wn, k.mfma_m)

    splits = (1, 2, 3, 4, 5, 6, 8, 10, 12, 16, 20, 24, 32)
    strat = (32, 32, 16)
    try:
        for (b, M, N, K, dt) in [(1, 77, 768, 768, 1), (1, 3000, 4096, 4096, 2), (4, 100, 200, 300, 0)]:
            p0 = vx.vx_plan_query(b, M, N, K, dt)
            assert vx.vx_fix_wavefront(*strat) == 0
            p = vx.vx_plan_query(b, M, N, K, dt)
            assert wave(p.kernel) == strat
            assert p.predicted_ns >= p0.predicted_ns
            best = min(c for k in reg if k.enabled and k.dtype == dt and wave(k) == strat for s in splits
                       for st, c in [vx.vx_plan_cost(b, M, N, K, dt, k.id, s, 3)] if st == 0)
            assert p.predicted_ns == pytest.approx(best, rel=1e-12)
            assert vx.vx_fix_wavefront(0, 0, 0) == 0
            p1 = vx.vx_plan_query(b, M, N, K, dt)
            assert (p1.kernel_id, p1.split_k) == (p0.kernel_id, p0.split_k)
        # a strategy that only disabled (spilling) kernels have is refused
        # (whether the build has one depends on what the compiler spilled)
        disabled_only = {wave(k) for k in reg if not k.enabled} - {wave(k) for k in reg if k.enabled}
        if disabled_only:
            assert vx.vx_fix_wavefront(*sorted(disabled_only)[0]) == 3
        absent = (48, 48, 16)   # no compiled kernel has this wavefront tile
        assert absent not in {wave(k) for k in reg}
        assert vx.vx_fix_wavefront(*absent) == 3
    finally:
        assert vx.vx_fix_wavefront(0, 0, 0) == 0


def test_one_hip_runtime_when_the_binding_loads_first():
    """Loading the library before anything else imports torch must not bring
    a second HIP runtime into the process (torch bundles its own)."""
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_2409_01075_amd import vx\n"
            "vx.lib()\n"
            "import torch\n"
            "maps = open('/proc/self/maps').read()\n"
            "print(len({l.split()[-1] for l in maps.splitlines() if 'libamdhip64' in l}))\n" % ROOT)
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stderr[-2000:]
    assert out.stdout.strip().splitlines()[-1] == "1"


def test_backend_restriction(mi355x_override):
    """The hardware-adaptation hook: the argmin runs over the matrix-core
    kernels only, the vector-ALU kernels only, or both."""
    try:
        assert vx.vx_restrict_backends(vx.BACKEND_VALU) == 0
        p = vx.vx_plan_query(1, 3, 1024, 1024, vx.VX_BF16)
        assert p.kernel.family == 2 and p.kernel.mfma_m == 0
        assert vx.vx_restrict_backends(vx.BACKEND_MFMA) == 0
        p = vx.vx_plan_query(1, 3, 1024, 1024, vx.VX_BF16)
        assert p.kernel.family in (0, 1) and p.kernel.mfma_m > 0
        assert vx.vx_restrict_backends(4) == 1 and vx.vx_restrict_backends(-1) == 1
        # the vector-ALU kernels need 16-byte rows: element-aligned calls have no candidate
        assert vx.vx_restrict_backends(vx.BACKEND_VALU) == 0
        with pytest.raises(vx.VxError):
            vx.vx_plan_query(1, 3, 1023, 1023, vx.VX_BF16)
    finally:
        assert vx.vx_restrict_backends(0) == 0
    p = vx.vx_plan_query(1, 3, 1024, 1024, vx.VX_BF16)
    assert p.kernel_id >= 0


def test_conv2d_argument_checks_and_plan(mi355x_override):
    """Host-side checks of the convolution entry point (no device needed) and
    its plan: a convolution kernel chosen for the implicit-GEMM shape."""
    d = vx.conv_desc(2, 14, 15, 8, 16, 3, 3, vx.VX_BF16, (2, 1), (1, 1), (1, 2))
    p = vx.vx_conv2d_plan_query(d)
    assert p.kernel.op == 1
    # channels not a multiple of 8: the register-staged (element-gathering) kernels only
    d3 = vx.conv_desc(2, 14, 15, 3, 16, 3, 3, vx.VX_BF16, (2, 1), (1, 1), (1, 2))
    assert vx.vx_conv2d_plan_query(d3).kernel.vec == 0
    oh = (14 + 2 - 2 - 1) // 2 + 1
    ow = (15 + 2 - 4 - 1) // 1 + 1
    assert p.tiles_m * p.kernel.mb >= 2 * oh * ow and p.tiles_n * p.kernel.nb >= 16
    bad = [dict(kh=0), dict(stride_h=0), dict(dil_w=0), dict(pad_h=-1), dict(n=-1), dict(c_in=-2)]
    for b in bad:
        e = vx.conv_desc(2, 14, 15, 8, 16, 3, 3, vx.VX_BF16, (2, 1), (1, 1), (1, 2))
        for k, v in b.items():
            setattr(e, k, v)
        assert vx.vx_conv2d(e, 16, 4096, 1 << 20) == 1, b
    e = vx.conv_desc(2, 14, 15, 8, 16, 3, 3, 7)
    assert vx.vx_conv2d(e, 16, 4096, 1 << 20) == 2                    # unsupported dtype
    assert vx.vx_conv2d(d, None, 4096, 1 << 20) == 1                  # NULL image with a non-empty extent
    assert vx.vx_conv2d(d, 16, 4096, 20) == 1                         # y overlaps x
    empty = vx.conv_desc(2, 2, 2, 8, 16, 5, 5, vx.VX_F16)            # the filter does not fit: no output
    assert vx.vx_conv2d(empty, None, None, None) == 0


def test_conv2d_extent_limits(mi355x_override):
    """Padded image extents of 2^30 or more are rejected (the kernels keep tap
    coordinates in 32 bits with a -2^30 sentinel for rows past M)."""
    for kw in (dict(h=(1 << 30) - 2, pad_h=1), dict(w=(1 << 29), pad_w=(1 << 28)), dict(pad_w=1 << 30)):
        d = vx.conv_desc(1, 4, 4, 8, 8, 1, 1, vx.VX_F16)
        for k, v in kw.items():
            setattr(d, k, v)
        assert vx.vx_conv2d(d, 16, 1 << 40, 1 << 41) == 1, kw
    d = vx.conv_desc(1, (1 << 30) - 3, 1, 8, 1, 1, 1, vx.VX_F16, pad=(1, 0))
    assert vx.vx_conv2d_plan_query(d).kernel.op == 1


def test_conv2d_large_image_avoids_32_bit_offsets(mi355x_override):
    """An image of 2^31 bytes or more is beyond the direct-to-LDS image
    loads' 32-bit buffer offsets: the plan takes a kernel that gathers the
    image through VGPRs with 64-bit addresses (register-staged, or mixed with
    the filter by DMA); below that a direct-to-LDS kernel is planned."""
    big = vx.conv_desc(1, 1 << 15, 1 << 12, 16, 8, 1, 1, vx.VX_F16)      # 2^31 elements, 2^32 bytes
    p = vx.vx_conv2d_plan_query(big)
    assert p.kernel.op == 1 and (p.kernel.family == 0 or not p.kernel.align & 1)
    small = vx.conv_desc(8, 256, 256, 64, 128, 3, 3, vx.VX_F16, pad=(1, 1))
    p = vx.vx_conv2d_plan_query(small)
    assert p.kernel.op == 1 and p.kernel.family == 1


def test_conv_element_gathers_priced(mi355x_override):
    """Three convolutions with the same implicit GEMM (M = 1024, N = 64,
    K = 72): a 1 x 1 filter over 72 channels (whole 16-byte chunks), an 8 x 3
    filter over 3 channels (7 of every 9 chunk positions cross the end of a
    filter row and are gathered element by element), and an 8 x 9 filter over
    one channel dilated 2 along the width (every chunk gathered).  With the
    shipped calibration, a kernel that gathers the image through VGPRs is
    priced by that share: the cost grows with it, linearly (the same grid),
    and the three shapes are planned apart (the plan cache tells them
    apart)."""
    shapes = {"whole": vx.conv_desc(1, 32, 32, 72, 64, 1, 1, vx.VX_F16),
              "part": vx.conv_desc(1, 39, 34, 3, 64, 8, 3, vx.VX_F16),
              "all": vx.conv_desc(1, 39, 48, 1, 64, 8, 9, vx.VX_F16, dil=(1, 2))}
    ks = [vx.vx_registry_get(i) for i in range(vx.vx_registry_count())]
    k = next(k for k in ks if k.op == 1 and k.dtype == 1 and k.enabled and not k.align & 1)
    cost = {}
    for name, d in shapes.items():
        assert vx.vx_force_plan(k.id, 1) == 0
        try:
            p = vx.vx_conv2d_plan_query(d)
        finally:
            vx.vx_force_plan(-1, 0)
        assert p.kernel_id == k.id and (p.tiles_m, p.tiles_n) == (-(-1024 // k.mb), -(-64 // k.nb))
        cost[name] = p.predicted_ns
    assert cost["whole"] < cost["part"] < cost["all"]
    assert cost["part"] - cost["whole"] == pytest.approx(7.0 / 9.0 * (cost["all"] - cost["whole"]), rel=1e-6)


def test_hybrid_grid_plans(mi355x_override):
    """The hybrid grid: whole waves of whole tiles plus the remaining tiles
    split.  It exists only where the tiles exceed one wave of the device; it
    is priced, forced and reported consistently."""
    occ = {}
    def slots(kid):
        if kid not in occ:
            occ[kid] = vx.vx_kernel_occupancy(kid)
        return 256 * occ[kid]
    # 6976 x 768 output, K = 3072: a hybrid candidate for every tile that leaves a partial wave
    b, M, N, K, dt = 1, 6976, 768, 3072, 2
    some = 0
    for k in (vx.vx_registry_get(i) for i in range(vx.vx_registry_count())):
        if k.op or k.dtype != dt or not k.enabled:
            continue
        tiles = -(-M // k.mb) * -(-N // k.nb)
        st, c = vx.vx_plan_cost(b, M, N, K, dt, k.id, -2, 3)
        if tiles <= slots(k.id) or tiles % slots(k.id) == 0:
            assert st == 3, (k.id, tiles)
        elif st == 0:
            some += 1
            assert vx.vx_force_plan(k.id, -2) == 0
            try:
                p = vx.vx_plan_query(b, M, N, K, dt)
            finally:
                vx.vx_force_plan(-1, 0)
            assert p.kernel_id == k.id and p.split_k == 2
            assert p.dp_tiles == tiles // slots(k.id) * slots(k.id)
            assert p.grid == p.dp_tiles + (tiles - p.dp_tiles) * 2
            assert p.predicted_ns == pytest.approx(c, rel=1e-12)
    assert some > 10
    # one wave or less: no hybrid grid, forced or chosen
    k = vx.vx_plan_query(1, 128, 128, 4096, dt).kernel
    assert vx.vx_force_plan(k.id, -2) == 0
    try:
        with pytest.raises(vx.VxError):
            vx.vx_plan_query(1, 128, 128, 4096, dt)
    finally:
        vx.vx_force_plan(-1, 0)
    assert vx.vx_plan_query(1, 128, 128, 4096, dt).dp_tiles == 0


def test_hybrid_grid_ablation_switch(mi355x_override):
    """vx_enable_hybrid_grid(0) takes the hybrid grid out of the selector's
    choices (and 1 puts it back); forced plans are not affected."""
    found = None
    for (M, N, K) in ((4904, 4096, 11008), (2544, 4096, 11008), (8192, 11008, 4096), (6976, 768, 3072)):
        p = vx.vx_plan_query(1, M, N, K, 2)
        if p.dp_tiles:
            found = (M, N, K)
            break
    if found is None:
        pytest.skip("no hybrid plan among these shapes for this calibration")
    try:
        assert vx.vx_enable_hybrid_grid(0) == 0
        q = vx.vx_plan_query(1, *found, 2)
        assert q.dp_tiles == 0 and q.predicted_ns >= p.predicted_ns
        assert vx.vx_force_plan(p.kernel_id, -p.split_k) == 0
        try:
            f = vx.vx_plan_query(1, *found, 2)
        finally:
            vx.vx_force_plan(-1, 0)
        assert f.dp_tiles == p.dp_tiles and f.predicted_ns == pytest.approx(p.predicted_ns, rel=1e-12)
    finally:
        assert vx.vx_enable_hybrid_grid(1) == 0
    assert vx.vx_plan_query(1, *found, 2).dp_tiles == p.dp_tiles


def test_k_rotation_switch_leaves_plans_alone(mi355x_override):
    """vx_enable_k_rotation only changes the K order inside the kernels at
    launch: the plan (kernel, split, grid, predicted time) is the same either way."""
    shapes = ((1, 768, 768), (300, 768, 768), (512, 4096, 4096))
    before = [vx.vx_plan_query(1, M, N, K, 1) for (M, N, K) in shapes]
    try:
        assert vx.vx_enable_k_rotation(0) == 0
        after = [vx.vx_plan_query(1, M, N, K, 1) for (M, N, K) in shapes]
    finally:
        assert vx.vx_enable_k_rotation(1) == 0
    for p, q in zip(before, after):
        assert (p.kernel_id, p.split_k, p.grid, p.dp_tiles) == (q.kernel_id, q.split_k, q.grid, q.dp_tiles)
        assert p.predicted_ns == q.predicted_ns


def test_equal_costs_go_to_fewer_k_slices(mi355x_override):
    """Among the plans at the minimum predicted cost the selector takes one
    with the fewest K slices (exact ties occur where the compulsory-bytes floor
    bounds several plans, e.g. the bf16 decode GEMM (1, 11008, 4096))."""
    splits = (1, 2, 3, 4, 5, 6, 8, 10, 12, 16, 20, 24, 32)
    reg = [k for k in (vx.vx_registry_get(i) for i in range(vx.vx_registry_count())) if k.op == 0 and k.enabled]
    for (M, N, K, dt) in ((1, 11008, 4096, 2), (16, 11008, 4096, 2), (16, 4096, 11008, 2), (1, 4096, 4096, 2),
                          (300, 768, 768, 1), (77, 96, 80, 0)):
        p = vx.vx_plan_query(1, M, N, K, dt)   # first, so that the calibration is loaded
        costs = []
        for k in reg:
            if k.dtype != dt:
                continue
            for s in splits:
                for sg in ((s, -s) if s >= 2 else (s,)):
                    st, c = vx.vx_plan_cost(1, M, N, K, dt, k.id, sg, 3)
                    if st == 0:
                        costs.append((c, s))
        best = min(c for c, _ in costs)
        fewest = min(s for c, s in costs if c == best)
        assert p.predicted_ns == best and p.split_k == fewest, ((M, N, K), p.split_k, fewest)


def test_workspace_failure_hook_plans_without_split(mi355x_override):
    """With the library's workspace unavailable, planning returns plans that
    need none (the fallback a launch takes when the allocation fails)."""
    M, N, K = 16, 4096, 11008
    p = vx.vx_plan_query(1, M, N, K, 2)
    assert p.split_k > 1 and p.workspace_bytes > 0
    assert vx.vx_test_fail_workspace_alloc(1) == 0
    try:
        q = vx.vx_plan_query(1, M, N, K, 2)
        assert q.split_k == 1 and q.workspace_bytes == 0 and q.dp_tiles == 0
    finally:
        vx.vx_test_fail_workspace_alloc(0)
    r = vx.vx_plan_query(1, M, N, K, 2)
    assert (r.kernel_id, r.split_k) == (p.kernel_id, p.split_k)
