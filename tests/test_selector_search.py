"""The pruned search of Equation 1 (CPU, no GPU): it must return exactly
the plan that pricing every (kernel, split, grid) triple returns -- same
kernel, split, grid and predicted cost, bit for bit -- under every filter
the ablation switches set, while pricing a small fraction of the triples;
and a shape seen for the first time must be planned within a few
microseconds (Section 7.4, runtime overhead; Section 6.2)."""
import ctypes
import os
import sys
import subprocess
import time

import numpy as np
import pytest

from paper_2409_01075_amd import inputs as I
from paper_2409_01075_amd import vx

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.fixture
def planning():
    assert vx.vx_set_hwinfo_override(vx.mi355x_hwinfo()) == 0
    yield
    vx.vx_selector_exhaustive(0)
    vx.vx_force_plan(-1, 0)
    vx.vx_fix_wavefront(0, 0, 0)
    vx.vx_restrict_backends(0)
    vx.vx_enable_hybrid_grid(1)
    assert vx.vx_set_hwinfo_override(None) == 0


def _random_shapes(n, seed):
    g = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        dt = int(g.integers(0, 3))
        m = int(np.exp(g.uniform(0, np.log(9000))))
        nn = int(np.exp(g.uniform(0, np.log(12000))))
        k = int(np.exp(g.uniform(0, np.log(12000)))) if g.random() > 0.02 else 0
        b = 1 if g.random() < 0.7 else int(g.integers(1, 200))
        align = 2 if g.random() < 0.2 else 256
        out.append((b, m, nn, k, dt, align))
    return out


def _workload_shapes():
    out = [(1, M, 768, 768, 1, 256) for M in range(1, 513, 7)]
    out += [(1, I.encoder_shape(t), N, K, 2, 256) for t in range(16) for (K, N) in I.ENCODER_SHAPES]
    out += [(192, L, L, 64, 2, 256) for L in map(I.attention_L, range(8))]
    out += [(192, L, 64, L, 2, 256) for L in map(I.attention_L, range(8))]
    out += [(1, I.llm_M(t), N, K, 2, 256) for t in range(16) for (K, N) in I.LLM_SHAPES]
    return out


def _plans(shapes):
    out = []
    for (b, M, N, K, dt, al) in shapes:
        try:
            p = vx.vx_plan_query(b, M, N, K, dt, base_align=al)
        except vx.VxError:
            out.append(None)
            continue
        out.append((p.kernel_id, p.split_k, p.dp_tiles, p.grid, p.k_per_split, p.predicted_ns.hex(),
                    vx.vx_selector_last_evaluations()))
    return out


def _compare(shapes):
    vx.vx_selector_exhaustive(0)
    pruned = _plans(shapes)
    vx.vx_selector_exhaustive(1)
    full = _plans(shapes)
    vx.vx_selector_exhaustive(0)
    assert len(pruned) == len(full)
    n_priced = n_full = 0
    for s, a, b in zip(shapes, pruned, full):
        assert (a is None) == (b is None), s
        if a is None:
            continue
        assert a[:6] == b[:6], (s, a, b)
        n_priced += a[6]
        n_full += b[6]
    return n_priced, n_full


def test_pruned_search_returns_the_exhaustive_plan(planning):
    shapes = _workload_shapes() + _random_shapes(700, 17)
    shapes += [(1, 1, 1, 1, 1, 256), (1, 77, 96, 80, 0, 256), (1, 5, 3, 0, 2, 256), (3, 7, 9, 11, 1, 2)]
    n_priced, n_full = _compare(shapes)
    # the bounds do their work: a small fraction of the triples is priced
    assert n_priced < 0.2 * n_full, (n_priced, n_full)


def test_pruned_search_under_every_filter(planning):
    """Forced kernels and splits, a fixed wavefront strategy, one backend,
    no hybrid grid: the same plan as the exhaustive search each time."""
    shapes = _workload_shapes()[::3] + _random_shapes(120, 23)
    for setup in (lambda: vx.vx_force_plan(-1, 3), lambda: vx.vx_force_plan(-1, -2),
                  lambda: vx.vx_fix_wavefront(32, 32, 16), lambda: vx.vx_fix_wavefront(16, 64, 16),
                  lambda: vx.vx_restrict_backends(2), lambda: vx.vx_restrict_backends(1),
                  lambda: vx.vx_enable_hybrid_grid(0)):
        setup()
        _compare(shapes)
        vx.vx_force_plan(-1, 0)
        vx.vx_fix_wavefront(0, 0, 0)
        vx.vx_restrict_backends(0)
        vx.vx_enable_hybrid_grid(1)
    # a forced kernel (each dtype's first kernel of a few families)
    n = vx.vx_registry_count()
    picked = {}
    for i in range(n):
        k = vx.vx_registry_get(i)
        if k.enabled and k.op == 0:
            picked.setdefault((k.dtype, k.family, k.align), i)
    for i in picked.values():
        k = vx.vx_registry_get(i)
        vx.vx_force_plan(i, 0)
        _compare([s for s in shapes if s[4] == k.dtype])
        vx.vx_force_plan(-1, 0)


def test_pruned_search_for_convolutions(planning):
    g = np.random.default_rng(31)
    for _ in range(60):
        dt = int(g.integers(0, 3))
        c_in = int(g.choice([3, 8, 16, 64, 5]))
        d = vx.conv_desc(int(g.integers(1, 9)), int(g.integers(4, 80)), int(g.integers(4, 80)), c_in,
                         int(g.choice([8, 16, 64, 96])), 3, 3, dt, stride=(1, 1), pad=(1, 1))
        vx.vx_selector_exhaustive(0)
        a = vx.vx_conv2d_plan_query(d)
        vx.vx_selector_exhaustive(1)
        b = vx.vx_conv2d_plan_query(d)
        vx.vx_selector_exhaustive(0)
        assert (a.kernel_id, a.split_k, a.dp_tiles, a.grid, a.predicted_ns.hex()) == \
               (b.kernel_id, b.split_k, b.dp_tiles, b.grid, b.predicted_ns.hex())


def _sweep_shapes():
    return [(1, M, 768, 768, 1) for M in range(1, 513)]


_CTYPES_TIMING = """
import ctypes, sys, time
sys.path.insert(0, %r)
from paper_2409_01075_amd import vx
assert vx.vx_set_hwinfo_override(vx.mi355x_hwinfo()) == 0
L = vx.lib()
p = vx.vx_plan()
pr = ctypes.byref(p)
q = L.vx_plan_query
shapes = [(1, M, 768, 768, 1) for M in range(1, 513)]
best = float("inf")
for _ in range(9):
    vx.vx_selector_exhaustive(0)   # retires every cached plan
    for dt in (0, 1, 2):
        vx.vx_plan_query(1, 3, 5, 7, dt)
    t0 = time.perf_counter()
    for (b, M, N, K, dt) in shapes:
        q(b, M, N, K, dt, M * K, K * N, M * N, 256, pr)
    best = min(best, (time.perf_counter() - t0) / len(shapes) * 1e6)
print(best)
"""


def test_new_shape_planning_time_through_ctypes():
    """512 shapes of the dynamic-M sweep, each seen for the first time, planned
    through the C ABI from Python (ctypes, a preallocated plan): the least mean
    over 9 passes, in the least of five processes (the same process can run
    the whole pass up to 2x slower, by where it lands on the host)."""
    best = float("inf")
    for _ in range(5):
        out = subprocess.run([sys.executable, "-c", _CTYPES_TIMING % ROOT], capture_output=True, text=True, check=True)
        best = min(best, float(out.stdout.split()[-1]))
    print("new-shape plan through ctypes: %.2f us per shape" % best)
    assert best <= 12.0   # typically 4.4-5.4 on this container (noisy host: up to 10)


def test_new_shape_planning_time_in_c(tmp_path, planning):
    """The same, timed in C++ with std::chrono (tests/plan_timing.cpp): the
    selector's own cost per new shape, for the sweep and for the LLM set."""
    exe = tmp_path / "plan_timing"
    lib_dir = os.path.dirname(vx.LIB_PATH)
    subprocess.run(["g++", "-O2", "-std=c++17", "-I", os.path.join(ROOT, "include"), os.path.join(HERE, "plan_timing.cpp"),
                    "-o", str(exe), "-L", lib_dir, "-lvx", "-Wl,-rpath," + lib_dir], check=True)
    calib = os.path.join(lib_dir, "calib_gfx950.txt")
    res = {}
    sets = {"sweep": _sweep_shapes(),
            "llm": [(1, I.llm_M(t), N, K, 2) for t in range(48) for (K, N) in I.LLM_SHAPES]}
    for name, shapes in sets.items():
        text = "\n".join("%d %d %d %d %d" % s for s in shapes) + "\n"
        best = float("inf")
        for _ in range(5):   # the least of five processes: a busy host only ever slows a pass down
            out = subprocess.run([str(exe), calib, "7"], input=text, capture_output=True, text=True, check=True).stdout
            f = out.split()
            best = min(best, float(f[1]))
        res[name] = best
        print("new-shape plan in C (%s): %.2f us per shape, cached %.3f us, %.1f triples priced" %
              (name, best, float(f[3]), float(f[5])))
    assert res["sweep"] <= 8.0   # typically 2.5-3.2 on this container (noisy host: up to 6)
    assert res["llm"] <= 20.0    # typically 9-15
