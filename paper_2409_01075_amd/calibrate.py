"""Offline calibration of the kernels' low levels on the current device.

The empirical half of the hybrid analyzer (Section 5.2): the low levels of the
hierarchy (wavefront and workgroup) are measured once per device, and the grid
level stays analytical at run time.  For every compiled kernel this times the
kernel itself on synthetic shapes built from its own workgroup tile and the
device's CU count - never from application shapes:

  * "full": one wave of workgroups filling the device (CUs x resident
    workgroups per CU), with 2 and with 10 K steps per workgroup (fewer for
    a kernel whose K slice is bounded);
  * "light": 32 workgroups (or fewer if the device holds fewer), same K steps.

Each pair gives the time of one workgroup K step (difference over the extra steps) and
the fixed per-call cost (the remainder, less the launch floor).  With the
device full, the kernel also runs split-K with 2, 3, 4, 6 and 8 slices of 2 steps
each: the extra time over the unsplit 2-step call, fitted by least squares, gives the
split-K epilogue cost a + b * (slices - 1) (partial tile out, arrival counter, last
slice's reads).  A convolution kernel that gathers the image through VGPRs
is also timed (2 and 10 steps, full and light load) on a convolution whose every image
chunk must be gathered element by element (one channel, a filter dilated
along the width): the selector adds the share of such chunks a layer has.
A spin kernel ahead of each timed window lets the host queue every call before
the device starts, so the times are device times, not host enqueue times.  Operands are
cycled through device copies totalling at least 256 MiB, so steady-state
loads come from HBM.  The launch floor is a K = 0 call of the smallest kernel.

Writes calib_<arch>.txt next to libvx.so; the library reads it at its first
plan when it was taken on the same kernel set.

Usage: python -m paper_2409_01075_amd.calibrate [--out PATH] [--dtypes f16,bf16,f32]
"""
import argparse
import ctypes
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))


def _timer(stream, cycles_per_ms):
    import torch

    def run(fn, n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(int(cycles_per_ms * max(0.2, n * 0.010)))   # ~10 us of head start per call
        e0.record(stream)
        for i in range(n):
            fn(i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e6 / n      # ns per call
    return run


# K slices at which the split-K epilogue is timed; its cost over the unsplit
# call is fitted as a + b * (slices - 1) by least squares (a difference of
# two timings alone moved b by a factor of 3 between runs).
SPLITS = (2, 3, 4, 6, 8)


def _split_fit(pts):
    """Least-squares line through (slices - 1, extra ns) points; a, b >= 0."""
    n = float(len(pts))
    mx = sum(x for x, _ in pts) / n
    my = sum(y for _, y in pts) / n
    sxx = sum((x - mx) ** 2 for x, _ in pts)
    b = max(sum((x - mx) * (y - my) for x, y in pts) / sxx, 0.0) if sxx > 0 else 0.0
    a = max(my - b * mx, 0.0)
    return a, b


def calibrate(out=None, dtypes=(0, 1, 2), rot_mib=256, verbose=True):
    import numpy as np
    import torch
    from . import vx

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    L = vx.lib()
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    hw = vx.vx_get_hwinfo()
    arch = hw.arch.decode()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    torch.cuda._sleep(1000000)
    e1.record(stream)
    torch.cuda.synchronize()
    run = _timer(stream, 1e6 / max(e0.elapsed_time(e1), 1e-3))
    tdt = {0: torch.float32, 1: torch.float16, 2: torch.bfloat16}

    # launch floor: K = 0 on one small tile (only the epilogue's zero stores)
    c0 = torch.empty((16, 16), dtype=torch.float16, device=dev)
    vx.vx_force_plan(-1, 0)
    L.vx_gemm(16, 16, 0, 1, None, None, c0.data_ptr(), sp)
    launch = float(np.median([run(lambda i: L.vx_gemm(16, 16, 0, 1, None, None, c0.data_ptr(), sp), 200)
                              for _ in range(3)]))

    rows = []
    n = vx.vx_registry_count()
    t_start = time.time()
    for kid in range(n):
        k = vx.vx_registry_get(kid)
        if not k.enabled or k.dtype not in dtypes:
            continue
        occ = vx.vx_kernel_occupancy(kid)
        slots = hw.num_cu * occ
        meas = {}
        eb = 4 if k.dtype == 0 else 2

        def timed(M, N, K, split, gather=False):
            set_bytes = (M * K + K * N + M * N) * eb
            R = int(min(max(2, -(-rot_mib * 2 ** 20 // set_bytes)), 512))
            # an operand whose rows the kernel does not need aligned is timed
            # shifted by one element, so that every row access is the
            # misaligned kind the kernel exists for
            sha = 0 if k.align & 1 else 1
            shb = 0 if k.align & 2 else 1
            shc = 0 if k.vec else 1
            A = torch.randn((R * M * K + sha,), device=dev).to(tdt[k.dtype])
            B = torch.randn((R * K * N + shb,), device=dev).to(tdt[k.dtype])
            C = torch.empty((R * M * N + shc,), dtype=tdt[k.dtype], device=dev)
            a0, b0, cc = A.data_ptr() + sha * eb, B.data_ptr() + shb * eb, C.data_ptr() + shc * eb
            sa, sb, sc = M * K * eb, K * N * eb, M * N * eb
            vx.vx_force_plan(kid, split)
            # a convolution kernel runs the same implicit-GEMM shape as a 1 x 1
            # convolution of a 1 x M image with K channels into N; with `gather`,
            # as an M x 1 output of one channel under a (K / VE) x VE filter
            # dilated 2 along the width, so that every chunk of VE consecutive k
            # is gathered element by element
            desc = None
            if k.op == 1 and gather:
                ve = 16 // eb
                kh = K // ve
                desc = vx.conv_desc(1, M + kh - 1, 1 + 2 * (ve - 1), 1, N, kh, ve, k.dtype, dil=(1, 2))
            elif k.op == 1:
                desc = vx.conv_desc(1, 1, M, K, N, 1, 1, k.dtype)
            try:
                def call(i):
                    r = i % R
                    if desc is not None:
                        st = vx.vx_conv2d(desc, a0 + r * sa, b0 + r * sb, cc + r * sc, sp)
                    else:
                        st = L.vx_gemm(M, N, K, k.dtype, a0 + r * sa, b0 + r * sb, cc + r * sc, sp)
                    if st != 0:
                        raise RuntimeError("kernel %d: %s" % (kid, vx.STATUS.get(st, st)))
                call(0)
                torch.cuda.synchronize()
                calls = max(R, 16)
                return float(np.median([run(call, calls) for _ in range(5)]))
            finally:
                vx.vx_force_plan(-1, 0)

        # K steps per workgroup: 2 and 10, or as many as the kernel's longest
        # slice allows (kernels that hold their slice of A in LDS)
        nk_hi = 10 if k.k_max <= 0 else max(3, min(10, k.k_max // k.kb))
        for tag, G in (("full", slots), ("light", min(32, slots))):
            nt = min(16, G)
            mt = G // nt
            for nk in (2, nk_hi):
                meas[(tag, nk)] = timed(mt * k.mb, nt * k.nb, nk * k.kb, 1)
        for s_ in SPLITS:
            tiles = max(1, slots // s_)
            nt = min(16, tiles)
            mt = max(1, tiles // nt)
            meas[("split", s_)] = timed(mt * k.mb, nt * k.nb, s_ * 2 * k.kb, s_)
        # convolution kernels that gather the image through VGPRs: the K step
        # when every image chunk is gathered element by element
        gathers = k.op == 1 and not k.align & 1
        if gathers:
            for tag, G in (("gather", slots), ("gather_light", min(32, slots))):
                nt = min(16, G)
                mt = G // nt
                for nk in (2, nk_hi):
                    meas[(tag, nk)] = timed(mt * k.mb, nt * k.nb, nk * k.kb, 1, gather=True)
        step_full = max((meas[("full", nk_hi)] - meas[("full", 2)]) / (nk_hi - 2.0), 1.0)
        step_gather = (max((meas[("gather", nk_hi)] - meas[("gather", 2)]) / (nk_hi - 2.0), 1.0) if gathers
                       else -1.0)
        step_gather_light = (max((meas[("gather_light", nk_hi)] - meas[("gather_light", 2)]) / (nk_hi - 2.0), 1.0)
                             if gathers else -1.0)
        step_light = max((meas[("light", nk_hi)] - meas[("light", 2)]) / (nk_hi - 2.0), 1.0)
        fix_full = max(meas[("full", 2)] - 2 * step_full - launch, 0.0)
        fix_light = max(meas[("light", 2)] - 2 * step_light - launch, 0.0)
        load_light = min(32, slots) / float(slots)
        split_a, split_b = _split_fit([(s_ - 1, max(meas[("split", s_)] - meas[("full", 2)], 0.0)) for s_ in SPLITS])
        rows.append((kid, step_full, fix_full, step_light, fix_light, load_light, split_a, split_b, step_gather,
                     step_gather_light))
        if verbose:
            print("kernel %3d %-28s occ %d  step %8.1f / %8.1f ns  fixed %8.1f / %8.1f ns  split %7.1f + %7.1f"
                  " (%.0f s)" % (kid, "%dx%dx%d w%dx%d st%d f%d v%d" % (k.mb, k.nb, k.kb, k.wm, k.wn, k.stages,
                                                                     k.family, k.vec), occ, step_full,
                                step_light, fix_full, fix_light, split_a, split_b, time.time() - t_start),
                  file=sys.stderr, flush=True)
    out = out or os.path.join(HERE, "calib_%s.txt" % arch)
    with open(out, "w") as f:
        f.write("# vx kernel calibration (offline, per device): written by paper_2409_01075_amd/calibrate.py\n")
        f.write("# kernel <id> <step_full_ns> <fixed_full_ns> <step_light_ns> <fixed_light_ns> <load_light>"
                " <split_a_ns> <split_b_ns> <step_gather_full_ns> <step_gather_light_ns>\n")
        f.write("arch %s\n" % arch)
        f.write("device_cus %d\n" % hw.num_cu)
        f.write("registry_hash %s\n" % vx.vx_registry_hash())
        f.write("launch_ns %.1f\n" % launch)
        for r in rows:
            f.write("kernel %d %.1f %.1f %.1f %.1f %.5f %.1f %.1f %.1f %.1f\n" % r)
    if verbose:
        print("wrote %s (%d kernels, launch floor %.0f ns)" % (out, len(rows), launch), file=sys.stderr)
    return out


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=None)
    ap.add_argument("--dtypes", default="f32,f16,bf16")
    a = ap.parse_args()
    codes = {"f32": 0, "f16": 1, "bf16": 2}
    calibrate(a.out, tuple(codes[d] for d in a.dtypes.split(",")))
