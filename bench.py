"""Benchmark of the runtime-shaped GEMM path on one MI355X.

Default workload (the dynamic-M sweep): fp16 A (M x 768) x fp16 B (768 x 768),
fp32 accumulation, fp16 output, for every M in 1..512, inputs U[-1, 1] seeded
per M (paper_2409_01075_amd.inputs.sweep_f16), resident in HBM before timing.

One step = the sweep: for each M, a window of R_M back-to-back vx_gemm calls
on one stream, cycling through R_M distinct device copies of that M's
operands, with R_M * (operand bytes) >= 512 MiB (twice the 256 MB last-level
cache), so every call reads its operands from HBM.  Two HIP events bracket
each window on the launch stream; the per-call device time of shape M is the
window over R_M (event overhead, about 3 us, is amortised over hundreds of
calls).  ms_per_step is the sum of the per-call times over the sweep, i.e. the
device time of one call per M.  The plain pass (each M once, back to back,
two events around the whole pass) is reported beside it.

Metric: geometric mean over M of 2*M*N*K / t_M (TFLOP/s), t_M the median over
the timed steps.  The roofline object describes the kernel that takes the most
time in the sweep: its algorithmic bytes per launch (the compulsory
(M*K + K*N + M*N)*2 bytes) over its average event-timed duration, against the
8 TB/s HBM peak (every sweep shape is below the fp16 ridge point of 314.6
FLOP/byte).  cpu_baseline times the CPU oracle on a bounded subset of the
same shapes on this host's cores, then checks (untimed) sampled outputs of the
timed back-to-back pass for every M against the oracle.

Beside the sweep the same run reports: launch_floor_us, the back-to-back
device time of an empty kernel (the dispatch floor every sweep shape sits on:
their roofline times are 0.15-0.34 us) and k0_call_us, this library's
smallest launch (a K = 0 call); and "sets", a stated sample of the bf16
workload sets (encoder trials 0-3, attention trials 0-1, LLM trials 0-5),
each GEMM timed like --workload runs do, with geomean TFLOP/s and roofline
fractions split by bound (--no-sets skips it).
"""
import argparse
import ctypes
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
MFMA_PEAK_TFLOPS = {0: 157.3, 1: 2516.6, 2: 2516.6}
N_SWEEP, K_SWEEP = 768, 768


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--workload", default="sweep",
                    choices=["sweep", "sweep-sample", "encoder", "attention", "llm", "single", "mixed", "conv", "shapes"],
                    help="sweep (default, the headline metric), one of the other GEMM sets, the "
                         "dynamic-shape convolution set, or the GEMMs listed by --shapes")
    ap.add_argument("--shapes", default="",
                    help="for --workload shapes: 'M,N,K[,batch];...' (operands N(0,1) and N(0,0.02))")
    ap.add_argument("--dtype", default="bf16", choices=["f32", "f16", "bf16"],
                    help="element type for --workload shapes")
    ap.add_argument("--trials", type=int, default=None, help="trials of a GEMM set (default: the full set)")
    ap.add_argument("--conv-cin", default="models", choices=["models", "plain"],
                    help="convolution set: channel counts as CNN layers have them (3 or a multiple of 8), "
                         "or Cin drawn over the whole range 3..832")
    ap.add_argument("--adapt", action="store_true",
                    help="hardware-adaptation study (Section 7.4): fp16, N in {1024, 2048, 4096}, K = 1024, "
                         "M = 1..16, with the matrix-core kernels only, the vector-ALU kernels only, and both")
    ap.add_argument("--study", action="store_true",
                    help="selector quality study: time every feasible (kernel, split) plan of each GEMM "
                         "of the set and compare the selector's pick, and the Static1/Static2 hierarchy "
                         "ablations, with the best")
    ap.add_argument("--no-hybrid", action="store_true",
                    help="ablation: the selector does not consider the hybrid grid")
    ap.add_argument("--no-krot", action="store_true",
                    help="ablation: the direct-to-LDS GEMM kernels walk each tile's K steps in order "
                         "instead of from a per-tile rotated start")
    ap.add_argument("--no-calibration", action="store_true",
                    help="ablation: plan with the purely analytical cost model (ignore the calibration table)")
    ap.add_argument("--compare-torch", action="store_true",
                    help="also time torch.matmul (torch's conv2d, channels-last, for the convolution set) "
                         "on each shape of a set (context only)")
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--m-max", type=int, default=512, help="sweep M = 1..m_max")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sets", action="store_true",
                    help="skip the sample of the encoder, attention and LLM sets that the default sweep run "
                         "also times")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the CPU-oracle sample")
    ap.add_argument("--detail", default=None, help="write per-M results as JSON to this path")
    ap.add_argument("--rot-mib", type=int, default=512,
                    help="bytes of rotating operand copies per timing window (MiB)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="after timing, run one plain device-to-device copy of this size (MiB): a "
                         "kernel of known traffic for calibrating memory counters under a profiler")
    return ap.parse_args()


def _profiled_traffic(kernel_name):
    """HBM traffic per launch from the committed counter summary, if it was
    taken on the current kernel sources for this kernel; else None."""
    path = os.path.join(ROOT, "profiles", "sweep_f16_traffic.txt")
    try:
        kv, traffic = {}, {}
        with open(path) as f:
            for ln in f:
                if ln.strip() and not ln.startswith("#"):
                    k, _, v = ln.strip().partition(" ")
                    if k == "traffic":
                        name, _, b = v.partition(" ")
                        traffic[name] = float(b)
                    else:
                        kv[k] = v
    except OSError:
        return None
    from paper_2409_01075_amd import vx
    if kv.get("registry_hash") != vx.vx_registry_hash():
        return None
    return traffic.get(kernel_name)


def _copy_calibration(args, dev):
    """One plain device-to-device copy of --copy-mib MiB (a kernel of known
    traffic for scaling memory counters taken under a profiler)."""
    if args.copy_mib <= 0:
        return
    import torch
    n = args.copy_mib * 2 ** 20 // 2
    src = torch.empty(n, dtype=torch.float16, device=dev)
    dst = torch.empty(n, dtype=torch.float16, device=dev)
    src.fill_(1.0)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


_ABLATIONS = []   # ablation switches given on the command line


def _selector_kind():
    from paper_2409_01075_amd import vx
    kind = "hybrid (calibrated)" if vx.vx_calibration_active() else "analytical"
    return kind + ("; ablations: " + ", ".join(_ABLATIONS) if _ABLATIONS else "")


def _cpu_threads():
    """Threads for the CPU oracle: the CPUs this process may run on, at most
    16 (one GPU's share of the host's cores on the measurement machines)."""
    return max(1, min(16, _affinity_cpus()))


def _affinity_cpus():
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def _cpu_baseline(ms, budget_s, outputs=None):
    """Times the CPU oracle (as it stands) on a bounded subset of the sweep."""
    import numpy as np
    import oracle
    from paper_2409_01075_amd import inputs as I
    threads = _cpu_threads()
    done, rates = [], []
    t_all = time.perf_counter()
    # every 8th M, in order, until the time budget is used
    for M in ms[::8]:
        A, B = I.sweep_f16(M)
        t0 = time.perf_counter()
        oracle.gemm(A, B, 1, threads=threads, with_mag=False)
        dt = time.perf_counter() - t0
        rates.append(2.0 * M * N_SWEEP * K_SWEEP / dt / 1e12)
        done.append(M)
        if time.perf_counter() - t_all > budget_s:
            break
    geo = math.exp(sum(math.log(r) for r in rates) / len(rates))
    res = {"value": geo, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "affinity_cpus": _affinity_cpus(), "cpu_model": _cpu_model(),
            "sample": "fp16 sweep shapes M in %s (every 8th M from 1, %d shapes, full outputs, "
                      "fp64 accumulation, decode included), geomean over the sample; threads = the "
                      "process's CPUs, at most 16 (one GPU's share of the host)"
                      % ("{%d..%d}" % (done[0], done[-1]), len(done))}
    if outputs is not None:
        res["outputs_checked"] = _check_outputs(ms, outputs, threads)
    return res


def _check_outputs(ms, outputs, threads, n_rand=512):
    """The sweep's outputs from the timed back-to-back pass, checked (untimed)
    against the oracle's fp64 values at sampled positions of every M: the
    whole last row and last column plus n_rand seeded random entries, each a
    full-K dot product, under the fp16 bound |C - Cref| <= 4e-3 Mag + 1e-6."""
    import numpy as np
    import oracle
    from oracle import tolerance
    from paper_2409_01075_amd import inputs as I
    g = I.rng(7000)
    worst, bad, n = 0.0, None, 0
    for M in ms:
        A, B = I.sweep_f16(M, K_SWEEP, N_SWEEP)
        rows = np.concatenate([np.full(N_SWEEP, M - 1), np.arange(M), g.integers(0, M, n_rand)])
        cols = np.concatenate([np.arange(N_SWEEP), np.full(M, N_SWEEP - 1), g.integers(0, N_SWEEP, n_rand)])
        ref, mag = oracle.gemm_sampled(A, B, I.F16, M, N_SWEEP, K_SWEEP, rows, cols, threads=threads)
        n += rows.size
        try:
            worst = max(worst, tolerance.check(outputs[M][rows, cols], ref, mag, I.F16, "sweep M=%d" % M))
        except AssertionError as e:
            bad = bad or str(e)
    out = {"shapes": len(ms), "entries": n, "max_err_over_bound": worst, "within_bound": bad is None,
           "sample": "every sweep M: last row, last column and %d random entries of the timed "
                     "back-to-back pass's C, oracle fp64 dot products" % n_rand}
    if bad is not None:
        out["first_failure"] = bad
    return out


def _set_jobs(name, trials, shapes="", dtype="bf16"):
    """(label, batch, M, N, K, dtype, make) for every GEMM of a set; make(dev)
    returns seeded device operands (A, B) of the set's distributions."""
    from paper_2409_01075_amd import inputs as I
    import torch
    bf = torch.bfloat16
    jobs = []
    if name == "shapes":
        code = I.DTYPES[dtype]
        tdt = {0: torch.float32, 1: torch.float16, 2: torch.bfloat16}[code]
        for i, spec in enumerate(x for x in shapes.split(";") if x.strip()):
            v = [int(t) for t in spec.split(",")]
            if len(v) not in (3, 4) or min(v) < 1:
                raise SystemExit("--shapes: 'M,N,K[,batch];...' with positive sizes")
            M, N, K = v[:3]
            b = v[3] if len(v) == 4 else 1
            def mk(dev, i=i, b=b, M=M, N=N, K=K):
                return (I.device_normal((b * M, K), 1.0, 1000 * i, dev, tdt),
                        I.device_normal((b * K, N), 0.02, 1000 * i + 1, dev, tdt))
            jobs.append(("%s (%d,%d)x(%d,%d)%s" % (dtype, M, K, K, N, " x%d" % b if b > 1 else ""), b, M, N, K,
                         code, mk))
        return jobs
    if name == "mixed":
        # the study's whole benchmark: samples of every set, so that a static
        # strategy has to serve the full range of shapes at once
        return (_set_jobs("sweep-sample", None) + _set_jobs("llm", 6 if trials is None else trials)
                + _set_jobs("encoder", 4 if trials is None else trials)
                + _set_jobs("attention", 3 if trials is None else trials))
    if name == "sweep-sample":
        for M in (1, 4, 16, 33, 64, 100, 128, 200, 256, 320, 384, 448, 512):
            def mk(dev, M=M):
                A, B = I.sweep_f16(M)
                return (torch.from_numpy(A.view("int16")).to(dev).view(torch.float16),
                        torch.from_numpy(B.view("int16")).to(dev).view(torch.float16))
            jobs.append(("sweep M=%d" % M, 1, M, 768, 768, 1, mk))
        return jobs
    if name == "single":
        def mk(dev):
            A, B = I.single_f32(0)
            return torch.from_numpy(A).to(dev), torch.from_numpy(B).to(dev)
        return [("fp32 77x96x80", 1, 77, 96, 80, 0, mk)]
    if name in ("encoder", "llm", "attention"):
        jobs = [(label, b, M, N, K, 2, mk) for (label, b, M, N, K, mk) in I.device_set(name, trials)]
    return jobs


def _time_calls(call, R, stream, spin_cycles, reps=3):
    import numpy as np
    import torch
    n_calls = max(R, 8)
    times = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(spin_cycles)
        e0.record(stream)
        for i in range(n_calls):
            call(i % R)
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) / n_calls * 1e-3)
    return float(np.median(times))


def _study_ctx(job, dev, rot_mib, L, sp):
    """Rotating device copies of one GEMM of a set and a call(r) closure."""
    import torch
    from paper_2409_01075_amd import vx
    label, b, M, N, K, dt, mk = job
    eb = 4 if dt == 0 else 2
    A, B = mk(dev)
    set_bytes = b * (M * K + K * N + M * N) * eb
    R = int(min(max(2, -(-rot_mib * 2 ** 20 // set_bytes)), 4096))
    pa = A.reshape(1, -1).expand(R, -1).contiguous()
    pb = B.reshape(1, -1).expand(R, -1).contiguous()
    pc = torch.empty((R, b * M * N), dtype=A.dtype, device=dev)
    del A, B
    sa, sb, sc = b * M * K * eb, b * K * N * eb, b * M * N * eb
    a0, b0, c0 = pa.data_ptr(), pb.data_ptr(), pc.data_ptr()

    def call(r):
        st = L.vx_gemm_batched(b, M, N, K, dt, a0 + r * sa, M * K, b0 + r * sb, K * N, c0 + r * sc, M * N, sp)
        if st != 0:
            raise RuntimeError("%s: %s" % (label, vx.STATUS.get(st, st)))
    return call, R, (pa, pb, pc)


def _plan_key(plan):
    """(kernel, split) of a plan; the split is negative for a hybrid grid (the
    form vx_force_plan and vx_plan_cost take)."""
    return (plan.kernel_id, -plan.split_k if plan.dp_tiles else plan.split_k)


def _wave(k):
    return (k.mb // k.wm, k.nb // k.wn, k.mfma_m)


def _most_frequent(items):
    """Most frequent item; ties go to the one seen first."""
    counts, first = {}, {}
    for i, x in enumerate(items):
        counts[x] = counts.get(x, 0) + 1
        first.setdefault(x, i)
    return max(counts, key=lambda x: (counts[x], -first[x]))


def run_study(args):
    """Selector quality and the hierarchy ablations (Section 7.4).

    Pass 1, per GEMM of the set: the time of every feasible (kernel, split in
    {1, 2, 4, 8}, plain grid or hybrid grid for splits 2 and 4) plan of the
    registry, one sample each; then the selector's plan and the fastest plans,
    timed again as a median of 3, until the fastest is a re-timed one.  The
    best stands in for the per-shape profiled upper bound.
    Pass 2, per dtype and alignment class of the set: Static1 fixes the
    wavefront strategy (wavefront tile and MFMA instruction) that is most
    often optimal over the class's GEMMs and leaves the workgroup tile and the
    split to the selector; Static2 also fixes the workgroup tile, the one most
    often optimal among kernels with that wavefront strategy, and leaves only
    the split (a grid-level choice) to the selector.  Each is reported as a
    fraction of the best."""
    import numpy as np
    import torch
    from paper_2409_01075_amd import vx
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    L = vx.lib()
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    torch.cuda._sleep(1000000)
    e1.record(stream)
    torch.cuda.synchronize()
    spin = int(1e6 / max(e0.elapsed_time(e1), 1e-3) * 0.3)
    reg = [vx.vx_registry_get(i) for i in range(vx.vx_registry_count())]   # indexed by kernel id
    jobs = _set_jobs(args.workload, args.trials)
    rows, tables, dones = [], [], []
    vx.vx_force_plan(-1, 0)
    vx.vx_fix_wavefront(0, 0, 0)
    for job in jobs:
        label, b, M, N, K, dt, mk = job
        eb = 4 if dt == 0 else 2
        ve = 16 // eb
        vec_ok = (int(K % ve == 0 and (b == 1 or (M * K) % ve == 0))
                  | 2 * int(N % ve == 0 and (b == 1 or (K * N) % ve == 0)))   # rows aligned: bit 0 A, bit 1 B
        call, R, keep = _study_ctx(job, dev, args.rot_mib, L, sp)
        plan = vx.vx_plan_query(b, M, N, K, dt, M * K, K * N, M * N)
        call(0)
        table = {}
        for k in reg:
            if k.op != 0 or k.dtype != dt or not k.enabled or (k.align & ~vec_ok):
                continue
            for split in (1, 2, 4, 8, -2, -4):   # negative: the hybrid grid
                st, _ = vx.vx_plan_cost(b, M, N, K, dt, k.id, split, vec_ok)
                if st != 0:
                    continue
                vx.vx_force_plan(k.id, split)
                try:
                    call(0)
                    table[(k.id, split)] = _time_calls(call, R, stream, spin, reps=1)
                finally:
                    vx.vx_force_plan(-1, 0)
        # The pass times each plan once; its minimum would be the luckiest of
        # many noisy samples.  So the selector's pick (through the selector) and
        # then the pass's fastest plan, until the fastest is one of them, are
        # timed again like the pick (median of 3, after the pass), and those
        # times replace the single ones.
        pick = _plan_key(plan)
        done = set()

        def retime(key):
            if key != pick:
                vx.vx_force_plan(*key)
            try:
                call(0)
                table[key] = _time_calls(call, R, stream, spin)
            finally:
                vx.vx_force_plan(-1, 0)
            done.add(key)
        retime(pick)
        while True:
            bk = min(table, key=table.get)
            if bk in done:
                break
            retime(bk)
        del keep, call
        t_pick = table[pick]
        dones.append(done)
        kb = reg[bk[0]]
        row = {"label": label, "M": M, "N": N, "K": K, "batch": b, "dtype": dt, "vec_ok": vec_ok,
               "pick_us": t_pick * 1e6, "pick": list(pick), "best_us": table[bk] * 1e6, "best": list(bk),
               "best_tile": [kb.mb, kb.nb, kb.kb, kb.wm, kb.wn, kb.stages], "best_wave": list(_wave(kb)),
               "tried": len(table)}
        rows.append(row)
        tables.append(table)
        print("%-30s pick %8.1f us %s  best %8.1f us %s %s  (%d plans)"
              % (label, row["pick_us"], row["pick"], row["best_us"], row["best"], row["best_tile"], len(table)),
              file=sys.stderr, flush=True)

    # ---- pass 2: the static ablations, one fixed strategy per (dtype, alignment class)
    classes = sorted({(r["dtype"], r["vec_ok"]) for r in rows})
    fixed = {}
    for c in classes:
        idx = [i for i, r in enumerate(rows) if (r["dtype"], r["vec_ok"]) == c]
        s1 = _most_frequent([tuple(rows[i]["best_wave"]) for i in idx])
        per = []
        for i in idx:
            cand = {kp: t for kp, t in tables[i].items() if _wave(reg[kp[0]]) == s1}
            if cand:
                per.append(min(cand, key=cand.get)[0])
        fixed[c] = (s1, _most_frequent(per) if per else None)

    def timed_plan(i, plan):
        # a static plan is timed like the pick and the best (median of 3)
        key = _plan_key(plan)
        if key not in dones[i]:
            call, R, keep = _study_ctx(jobs[i], dev, args.rot_mib, L, sp)
            vx.vx_force_plan(*key)
            try:
                call(0)
                tables[i][key] = _time_calls(call, R, stream, spin)
            finally:
                vx.vx_force_plan(-1, 0)
            dones[i].add(key)
            del keep, call
        return key, tables[i][key]

    for i, r in enumerate(rows):
        label, b, M, N, K, dt, mk = jobs[i]
        s1, s2 = fixed[(dt, r["vec_ok"])]
        vx.vx_fix_wavefront(*s1)
        try:
            p1 = vx.vx_plan_query(b, M, N, K, dt, M * K, K * N, M * N)
        finally:
            vx.vx_fix_wavefront(0, 0, 0)
        k1, t1 = timed_plan(i, p1)
        k2, t2 = None, None
        if s2 is not None:
            vx.vx_force_plan(s2, 0)
            try:
                p2 = vx.vx_plan_query(b, M, N, K, dt, M * K, K * N, M * N)
            except vx.VxError:
                p2 = None
            finally:
                vx.vx_force_plan(-1, 0)
            if p2 is not None:
                k2, t2 = timed_plan(i, p2)
        best = min(tables[i].values())
        r.update({"best_us": best * 1e6, "frac_of_best": best / (r["pick_us"] * 1e-6),
                  "static1": {"wave": list(s1), "plan": list(k1), "us": t1 * 1e6, "frac_of_best": best / t1},
                  "static2": None if t2 is None else
                  {"kernel": s2, "plan": list(k2), "us": t2 * 1e6, "frac_of_best": best / t2}})
        print("%-30s selector %.1f%%  static1 %.1f%% %s  static2 %s of best"
              % (label, 100 * r["frac_of_best"], 100 * best / t1, list(k1),
                 "-" if t2 is None else "%.1f%% %s" % (100 * best / t2, list(k2))), file=sys.stderr, flush=True)

    def geo(xs):
        return float(np.exp(np.mean(np.log(xs)))) if xs else None
    f0 = [r["frac_of_best"] for r in rows]
    f1 = [r["static1"]["frac_of_best"] for r in rows]
    f2 = [r["static2"]["frac_of_best"] for r in rows if r["static2"]]
    out = {"study": args.workload, "gemms": len(rows), "selector_frac_of_best_geomean": geo(f0),
           "selector_frac_of_best_min": min(f0), "static1_frac_of_best_geomean": geo(f1),
           "static2_frac_of_best_geomean": geo(f2), "static2_gemms": len(f2),
           "fixed": {"dtype%d_vec%d" % c: {"wave": list(v[0]), "kernel": v[1]} for c, v in fixed.items()}}
    if args.detail:
        with open(args.detail, "w") as f:
            json.dump(rows, f)
    out["selector"] = _selector_kind()
    print(json.dumps(out), flush=True)


def run_adapt(args):
    """The paper's dynamic hardware adaptation experiment (Section 7.4): the
    same GEMMs planned three ways -- matrix-core kernels only, vector-ALU
    kernels only, and the adaptive default (the calibrated argmin over both) --
    each timed over rotating HBM-resident operands.  Reports every time and the
    largest gain of the adaptive setting over each fixed one."""
    import numpy as np
    import torch
    from paper_2409_01075_amd import inputs as I
    from paper_2409_01075_amd import vx
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    L = vx.lib()
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    torch.cuda._sleep(1000000)
    e1.record(stream)
    torch.cuda.synchronize()
    spin = int(1e6 / max(e0.elapsed_time(e1), 1e-3) * 0.3)
    K = 1024
    settings = (("matrix-core only", vx.BACKEND_MFMA), ("vector-ALU only", vx.BACKEND_VALU), ("adaptive", 0))
    rows = []
    try:
        for N in (1024, 2048, 4096):
            for M in range(1, 17):
                def mk(dev, M=M, N=N):
                    g = I.rng(7000 + 100 * M + N // 1024)
                    A = I.uniform(g, (M, K), 1)
                    B = I.uniform(g, (K, N), 1)
                    return (torch.from_numpy(A.view("int16")).to(dev).view(torch.float16),
                            torch.from_numpy(B.view("int16")).to(dev).view(torch.float16))
                call, R, keep = _study_ctx(("M=%d N=%d" % (M, N), 1, M, N, K, 1, mk), dev, args.rot_mib, L, sp)
                r = {"M": M, "N": N, "K": K}
                for name, mask in settings:
                    if vx.vx_restrict_backends(mask) != 0:
                        raise RuntimeError("vx_restrict_backends(%d)" % mask)
                    p = vx.vx_plan_query(1, M, N, K, vx.VX_F16)
                    call(0)
                    r[name] = _time_calls(call, R, stream, spin) * 1e6
                    r[name + " kernel"] = [p.kernel_id, p.kernel.family, p.split_k]
                del keep, call
                rows.append(r)
                print("N=%4d M=%2d  matrix-core %6.2f us  vector-ALU %6.2f us  adaptive %6.2f us (family %d)"
                      % (N, M, r["matrix-core only"], r["vector-ALU only"], r["adaptive"], r["adaptive kernel"][1]),
                      file=sys.stderr, flush=True)
    finally:
        vx.vx_restrict_backends(0)
    gain_mfma = max(r["matrix-core only"] / r["adaptive"] - 1.0 for r in rows)
    gain_valu = max(r["vector-ALU only"] / r["adaptive"] - 1.0 for r in rows)
    geo = lambda v: float(np.exp(np.mean(np.log(v))))
    out = {"study": "hardware adaptation", "dtype": "f16", "K": K, "N": [1024, 2048, 4096], "M": "1..16",
           "adaptive_max_gain_over_matrix_core_only": gain_mfma,
           "adaptive_max_gain_over_vector_alu_only": gain_valu,
           "geomean_us": {name: geo([r[name] for r in rows]) for name, _ in settings},
           "adaptive_picks_vector_alu": sum(1 for r in rows if r["adaptive kernel"][1] == 2),
           "gemms": len(rows), "selector": _selector_kind()}
    if args.detail:
        with open(args.detail, "w") as f:
            json.dump(rows, f)
    print(json.dumps(out), flush=True)


def run_conv(args):
    """Times every layer of the convolution set (fp16, NHWC image, KH x KW x Cin
    x Cout filter) over rotating HBM-resident copies: TFLOP/s (2 M N K of the
    implicit GEMM, M = N OH OW, N = Cout, K = KH KW Cin) and the fraction of
    each layer's roofline, with the compulsory bytes image + filter + output."""
    import numpy as np
    import torch
    from paper_2409_01075_amd import inputs as I
    from paper_2409_01075_amd import vx
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    L = vx.lib()
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    torch.cuda._sleep(1000000)
    e1.record(stream)
    torch.cuda.synchronize()
    cycles_per_ms = 1e6 / max(e0.elapsed_time(e1), 1e-3)
    f16 = torch.float16
    results = []
    for t in range(40 if args.trials is None else args.trials):
        Nb, H, W, Cin, Cout, F, st, pd = I.conv_trial(t, args.conv_cin)
        d = vx.conv_desc(Nb, H, W, Cin, Cout, F, F, vx.VX_F16, (st, st), (pd, pd))
        OH = (H + 2 * pd - F) // st + 1
        OW = (W + 2 * pd - F) // st + 1
        M, N, K = Nb * OH * OW, Cout, F * F * Cin
        x = I.device_normal((Nb, H, W, Cin), 1.0, 1000 * t, dev, f16)
        w = I.device_normal((F, F, Cin, Cout), 0.05, 1000 * t + 1, dev, f16)
        sx, sw, sy = x.numel() * 2, w.numel() * 2, M * N * 2
        set_bytes = sx + sw + sy
        R = int(min(max(2, -(-args.rot_mib * 2 ** 20 // set_bytes)), 4096))
        px = x.reshape(1, -1).expand(R, -1).contiguous()
        pw = w.reshape(1, -1).expand(R, -1).contiguous()
        py = torch.empty((R, M * N), dtype=f16, device=dev)
        x0, w0, y0 = px.data_ptr(), pw.data_ptr(), py.data_ptr()
        db = ctypes.byref(d)

        def call(r):
            return L.vx_conv2d(db, x0 + r * sx, w0 + r * sw, y0 + r * sy, sp)
        rc = call(0)
        if rc != 0:
            raise RuntimeError("conv trial %d: %s" % (t, vx.STATUS.get(rc, rc)))
        torch.cuda.synchronize()
        times = []
        n_calls = max(R, 8)
        for _ in range(3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(int(cycles_per_ms * 0.3))
            e0.record(stream)
            for i in range(n_calls):
                call(i % R)
            e1.record(stream)
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1) / n_calls * 1e-3)
        tm = float(np.median(times))
        plan = vx.vx_conv2d_plan_query(d)
        flops = 2.0 * M * N * K
        t_mfma = flops / (MFMA_PEAK_TFLOPS[1] * 1e12)
        t_hbm = set_bytes / (HBM_PEAK_GBPS * 1e9)
        r = {"trial": t, "layer": [Nb, H, W, Cin, Cout, F, st, pd], "M": M, "N": N, "K": K,
             "bytes": set_bytes, "us": tm * 1e6, "tflops": flops / tm / 1e12, "gbps": set_bytes / tm / 1e9,
             "bound": "mfma" if t_mfma >= t_hbm else "hbm", "roof_frac": max(t_mfma, t_hbm) / tm,
             "kernel": plan.kernel_id, "split": plan.split_k,
             "tile": [plan.kernel.mb, plan.kernel.nb, plan.kernel.kb]}
        if args.compare_torch:
            xt = x.permute(0, 3, 1, 2)                                   # NCHW view of the NHWC image
            wt = w.permute(3, 2, 0, 1).contiguous(memory_format=torch.channels_last)
            fn = torch.nn.functional.conv2d
            fn(xt, wt, None, st, pd)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(8):
                fn(xt, wt, None, st, pd)
            e1.record(stream)
            torch.cuda.synchronize()
            r["torch_us"] = e0.elapsed_time(e1) / 8 * 1e3
        results.append(r)
        print("conv t%-3d %-36s M %7d N %4d K %6d %9.1f us %7.1f TFLOP/s %6.0f GB/s %s %5.1f%% of roof "
              "kid %d split %d%s" % (t, str(r["layer"]), M, N, K, r["us"], r["tflops"], r["gbps"], r["bound"],
                                     100 * r["roof_frac"], r["kernel"], r["split"],
                                     ("  torch %.1f us" % r["torch_us"]) if "torch_us" in r else ""),
              file=sys.stderr, flush=True)
        del px, pw, py, x, w

    def geo(v):
        v = [x for x in v if x > 0]
        return float(np.exp(np.mean(np.log(v)))) if v else None
    by_kernel = {}
    for r in results:
        by_kernel.setdefault(r["kernel"], []).append(r)
    kid = max(by_kernel, key=lambda k: sum(r["us"] for r in by_kernel[k]))
    dom = by_kernel[kid]
    dom_t = sum(r["us"] for r in dom) * 1e-6
    if sum(r["us"] for r in dom if r["bound"] == "hbm") > dom_t * 5e5:
        ach = sum(r["bytes"] for r in dom) / dom_t / 1e9
        roof = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBPS}
    else:
        ach = sum(2.0 * r["M"] * r["N"] * r["K"] for r in dom) / dom_t / 1e12
        roof = {"bound": "mfma", "achieved": ach, "peak": MFMA_PEAK_TFLOPS[1], "unit": "TFLOP/s",
                "frac": ach / MFMA_PEAK_TFLOPS[1]}
    roof.update({"traffic": None, "kernel": "vxk_%d" % kid, "launches": len(dom),
                 "avg_us": dom_t / len(dom) * 1e6})
    out = {"metric": "Conv TFLOP/s geomean over a dynamic-shape CNN convolution set; % of MFMA/HBM roofline",
           "value": geo([r["tflops"] for r in results]), "unit": "TFLOP/s", "n_gpus": 1, "steps": 1,
           "warmup": 1, "ms_per_step": sum(r["us"] for r in results) / 1e3, "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f16", "data": "synthetic (seeded, on device)",
           "config": {"workload": "dynamic-shape convolution set: fp16 NHWC layers of the CNN ranges of Table 4",
                      "layers": len(results), "cin": args.conv_cin},
           "roofline": roof, "roof_frac_geomean": geo([r["roof_frac"] for r in results])}
    # Cin decides the load family: rows of 8 fp16 channels are 16-byte aligned
    # (direct-to-LDS im2col), other counts go through the register-staged path.
    out["by_cin"] = {}
    for name, sel in (("multiple_of_8", lambda c: c % 8 == 0), ("other", lambda c: c % 8 != 0)):
        grp = [r for r in results if sel(r["layer"][3])]
        out["by_cin"][name] = {"layers": len(grp), "tflops_geomean": geo([r["tflops"] for r in grp]),
                               "roof_frac_geomean": geo([r["roof_frac"] for r in grp])}
    if args.compare_torch:
        out["vs_torch_conv2d_geomean"] = geo([r["torch_us"] / r["us"] for r in results])
    if args.detail:
        with open(args.detail, "w") as f:
            json.dump(results, f)
    out["selector"] = _selector_kind()
    print(json.dumps(out), flush=True)


def _device_warmup(dev, ms=150.0):
    """About `ms` of back-to-back bf16 4096^3 GEMMs through the library before
    a set is timed: under sustained load the device takes tens of
    milliseconds to reach its loaded clock, and the first large GEMMs of a
    process otherwise run up to a fifth slower than the same calls later."""
    import torch
    from paper_2409_01075_amd import vx
    L = vx.lib()
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    n = 4096
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    a = torch.randn((n, n), generator=g, device=dev).to(torch.bfloat16)
    b = torch.randn((n, n), generator=g, device=dev).to(torch.bfloat16)
    c = torch.empty((n, n), dtype=torch.bfloat16, device=dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    st = L.vx_gemm(n, n, n, vx.VX_BF16, a.data_ptr(), b.data_ptr(), c.data_ptr(), sp)
    e1.record(stream)
    if st != 0:
        raise RuntimeError("warm-up GEMM: %s" % vx.STATUS.get(st, st))
    torch.cuda.synchronize()
    for _ in range(int(min(2000, ms / max(e0.elapsed_time(e1), 1e-3)))):
        L.vx_gemm(n, n, n, vx.VX_BF16, a.data_ptr(), b.data_ptr(), c.data_ptr(), sp)
    torch.cuda.synchronize()
    del a, b, c


def _time_jobs(jobs, rot_mib, dev, compare_torch=False, verbose=True):
    """Times every GEMM of `jobs` over rotating HBM-resident copies; per GEMM
    the median of 3 windows of back-to-back calls (a spin ahead of each window
    lets the host queue the calls first; about 1 ms of untimed calls between
    the spin and the window brings the clock to its loaded level).  Returns
    one dict per GEMM."""
    import numpy as np
    import torch
    from paper_2409_01075_amd import vx
    L = vx.lib()
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    torch.cuda._sleep(1000000)
    e1.record(stream)
    torch.cuda.synchronize()
    cycles_per_ms = 1e6 / max(e0.elapsed_time(e1), 1e-3)
    results = []
    for (label, b, M, N, K, dt, mk) in jobs:
        eb = 4 if dt == 0 else 2
        A, B = mk(dev)
        set_bytes = b * (M * K + K * N + M * N) * eb
        R = int(min(max(2, -(-rot_mib * 2 ** 20 // set_bytes)), 4096))
        pa = A.reshape(1, -1).expand(R, -1).contiguous()
        pb = B.reshape(1, -1).expand(R, -1).contiguous()
        pc = torch.empty((R, b * M * N), dtype=A.dtype, device=dev)
        sa, sb, sc = b * M * K * eb, b * K * N * eb, b * M * N * eb
        a0, b0, c0 = pa.data_ptr(), pb.data_ptr(), pc.data_ptr()

        def call(r):
            if b == 1:
                return L.vx_gemm(M, N, K, dt, a0 + r * sa, b0 + r * sb, c0 + r * sc, sp)
            return L.vx_gemm_batched(b, M, N, K, dt, a0 + r * sa, M * K, b0 + r * sb, K * N, c0 + r * sc,
                                     M * N, sp)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        st = call(0)
        e1.record(stream)
        if st != 0:
            raise RuntimeError("%s: %s" % (label, vx.STATUS.get(st, st)))
        torch.cuda.synchronize()
        # warm-up: about 1 ms of the same calls between the spin and the timed
        # window (at most 64), so that a long MFMA-bound window starts at the
        # clock it runs at in steady state rather than ramping up from idle
        n_warm = int(min(64, -(-1.0 // max(e0.elapsed_time(e1), 1e-3))))
        times = []
        n_calls = max(R, 8)
        for _ in range(3):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(int(cycles_per_ms * (0.3 + 0.006 * (n_calls + n_warm))))
            for i in range(n_warm):
                call((n_calls + i) % R)
            e0.record(stream)
            for i in range(n_calls):
                call(i % R)
            e1.record(stream)
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1) / n_calls * 1e-3)
        t = float(np.median(times))
        plan = vx.vx_plan_query(b, M, N, K, dt, M * K, K * N, M * N)
        flops = 2.0 * b * M * N * K
        bytes_min = float(set_bytes)
        t_mfma = flops / (MFMA_PEAK_TFLOPS[dt] * 1e12)
        t_hbm = bytes_min / (HBM_PEAK_GBPS * 1e9)
        r = {"label": label, "batch": b, "M": M, "N": N, "K": K, "dt": dt, "eb": eb, "us": t * 1e6,
             "tflops": flops / t / 1e12,
             "gbps": bytes_min / t / 1e9, "bound": "mfma" if t_mfma >= t_hbm else "hbm",
             "roof_frac": max(t_mfma, t_hbm) / t, "kernel": plan.kernel_id, "split": plan.split_k,
             "tile": [plan.kernel.mb, plan.kernel.nb, plan.kernel.kb, plan.kernel.stages]}
        if compare_torch:
            At = A.reshape(b, M, K) if b > 1 else A
            Bt = B.reshape(b, K, N) if b > 1 else B
            torch.matmul(At, Bt)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(8):
                torch.matmul(At, Bt)
            e1.record(stream)
            torch.cuda.synchronize()
            r["torch_us"] = e0.elapsed_time(e1) / 8 * 1e3
        results.append(r)
        if verbose:
            print("%-34s %9.1f us %8.1f TFLOP/s %7.0f GB/s  %s %5.1f%% of roof  kid %d split %d %s%s"
                  % (label, r["us"], r["tflops"], r["gbps"], r["bound"], 100 * r["roof_frac"], r["kernel"],
                     r["split"], r["tile"], ("  torch %.1f us" % r["torch_us"]) if "torch_us" in r else ""),
                  file=sys.stderr, flush=True)
        del pa, pb, pc, A, B
    return results


def _geo(v):
    import numpy as np
    v = [x for x in v if x > 0]
    return float(np.exp(np.mean(np.log(v)))) if v else None


def _set_summary(results):
    """Geomean TFLOP/s and roofline fractions of a timed set, split by bound."""
    hbm = [r for r in results if r["bound"] == "hbm"]
    mf = [r for r in results if r["bound"] == "mfma"]
    return {"gemms": len(results), "tflops_geomean": _geo([r["tflops"] for r in results]),
            "roof_frac_geomean": _geo([r["roof_frac"] for r in results]),
            "hbm_bound": {"n": len(hbm), "gbps_geomean": _geo([r["gbps"] for r in hbm]),
                          "frac_geomean": _geo([r["roof_frac"] for r in hbm])},
            "mfma_bound": {"n": len(mf), "tflops_geomean": _geo([r["tflops"] for r in mf]),
                           "frac_geomean": _geo([r["roof_frac"] for r in mf])}}


def run_set(args):
    """Times every GEMM of a set over rotating HBM-resident copies and reports
    TFLOP/s and the fraction of each shape's roofline."""
    import torch
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    jobs = _set_jobs(args.workload, args.trials, args.shapes, args.dtype)
    _device_warmup(dev)
    results = _time_jobs(jobs, args.rot_mib, dev, args.compare_torch)
    by_kernel = {}
    for r in results:
        by_kernel.setdefault(r["kernel"], []).append(r)
    kid = max(by_kernel, key=lambda k: sum(r["us"] for r in by_kernel[k]))
    dom = by_kernel[kid]
    dom_bound = max(set(r["bound"] for r in dom), key=lambda x: sum(r["us"] for r in dom if r["bound"] == x))
    dom_t = sum(r["us"] for r in dom) * 1e-6
    if dom_bound == "hbm":
        ach = sum(r["batch"] * (r["M"] * r["K"] + r["K"] * r["N"] + r["M"] * r["N"]) * r["eb"] for r in dom) / dom_t / 1e9
        roof = {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBPS}
    else:
        ach = sum(2.0 * r["batch"] * r["M"] * r["N"] * r["K"] for r in dom) / dom_t / 1e12
        peak = MFMA_PEAK_TFLOPS[dom[0]["dt"]]
        roof = {"bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s", "frac": ach / peak}
    roof.update({"traffic": None, "kernel": "vxk_%d" % kid, "launches": len(dom),
                 "avg_us": dom_t / len(dom) * 1e6})
    summ = _set_summary(results)
    out = {"metric": "GEMM TFLOP/s geomean over dynamic-M sweep; % of MFMA/HBM roofline on 1 GPU",
           "value": summ["tflops_geomean"], "unit": "TFLOP/s", "n_gpus": 1,
           "steps": 1, "warmup": 1, "ms_per_step": sum(r["us"] for r in results) / 1e3,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": ("f32" if args.workload == "single" else args.dtype if args.workload == "shapes" else "bf16"),
           "data": "synthetic (seeded, on device)",
           "config": {"workload": args.workload, "gemms": len(results)},
           "roofline": roof,
           "roof_frac_geomean": summ["roof_frac_geomean"],
           "hbm_bound": summ["hbm_bound"], "mfma_bound": summ["mfma_bound"]}
    if args.compare_torch:
        out["vs_torch_matmul_geomean"] = _geo([r["torch_us"] / r["us"] for r in results])
    _copy_calibration(args, dev)
    if args.detail:
        with open(args.detail, "w") as f:
            json.dump(results, f)
    out["selector"] = _selector_kind()
    print(json.dumps(out), flush=True)


def _launch_floor_us(stream, reps=3, n=400):
    """Back-to-back device time of an empty kernel (the dispatch floor), with
    the host queued ahead: the smallest per-call time any kernel launch on
    this stream can reach."""
    import numpy as np
    import torch
    out = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(20000000)
        e0.record(stream)
        for _ in range(n):
            torch.cuda._sleep(0)
        e1.record(stream)
        torch.cuda.synchronize()
        out.append(e0.elapsed_time(e1) * 1e3 / n)
    return float(np.median(out))


def _k0_call_us(stream, L, reps=3, n=400):
    """Back-to-back device time of this library's smallest launch: a K = 0
    call (one 16 x 16 tile of zeros)."""
    import numpy as np
    import torch
    c0 = torch.empty((16, 16), dtype=torch.float16, device="cuda")
    sp = ctypes.c_void_p(stream.cuda_stream)
    out = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(20000000)
        e0.record(stream)
        for _ in range(n):
            L.vx_gemm(16, 16, 0, 1, None, None, c0.data_ptr(), sp)
        e1.record(stream)
        torch.cuda.synchronize()
        out.append(e0.elapsed_time(e1) * 1e3 / n)
    return float(np.median(out))


SET_SAMPLE = (("encoder", 4), ("attention", 2), ("llm", 6))


def main():
    args = _parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the GEMM path is single-device; "
              "run it with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if args.no_calibration:
        from paper_2409_01075_amd import vx
        vx.vx_calibration_enable(0)
    if args.no_hybrid:
        from paper_2409_01075_amd import vx
        vx.vx_enable_hybrid_grid(0)
        _ABLATIONS.append("no-hybrid")
    if args.no_krot:
        from paper_2409_01075_amd import vx
        vx.vx_enable_k_rotation(0)
        _ABLATIONS.append("no-krot")
    if args.study:
        run_study(args)
        return
    if args.adapt:
        run_adapt(args)
        return
    if args.workload == "conv":
        run_conv(args)
        return
    if args.workload != "sweep":
        run_set(args)
        return
    import numpy as np
    import torch
    from paper_2409_01075_amd import inputs as I
    from paper_2409_01075_amd import vx

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    L = vx.lib()
    ms = list(range(1, args.m_max + 1))
    N, K = N_SWEEP, K_SWEEP

    # ---- resident inputs
    sets = []
    for M in ms:
        A, B = I.sweep_f16(M, K, N)
        At = torch.from_numpy(A.view(np.int16)).to(dev).view(torch.float16)
        Bt = torch.from_numpy(B.view(np.int16)).to(dev).view(torch.float16)
        Ct = torch.empty((M, N), dtype=torch.float16, device=dev)
        sets.append((M, At, Bt, Ct))
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    calls = [(M, At.data_ptr(), Bt.data_ptr(), Ct.data_ptr()) for (M, At, Bt, Ct) in sets]
    gemm = L.vx_gemm

    plans = {M: vx.vx_plan_query(1, M, N, K, vx.VX_F16) for M in ms}
    for M in ms:
        if plans[M].kernel.vec == 0:
            raise RuntimeError("aligned sweep shape M=%d planned with an element-aligned kernel" % M)

    def one_pass():
        for (M, a, b, c) in calls:
            st = gemm(M, N, K, 1, a, b, c, sp)
            if st != 0:
                raise RuntimeError("vx_gemm M=%d: %s" % (M, vx.STATUS.get(st, st)))

    # rotating pools: R_M copies of M's operands, R_M * set bytes >= 512 MiB
    rot_bytes = args.rot_mib * 2 ** 20
    reps = {M: max(8, -(-rot_bytes // ((M * K + K * N + M * N) * 2))) for M in ms}
    pool_a = torch.empty(max(reps[M] * M * K for M in ms), dtype=torch.float16, device=dev)
    pool_b = torch.empty(max(reps[M] * K * N for M in ms), dtype=torch.float16, device=dev)
    pool_c = torch.empty(max(reps[M] * M * N for M in ms), dtype=torch.float16, device=dev)

    def window(i):
        M, At, Bt, _ = sets[i]
        R = reps[M]
        pa = pool_a[:R * M * K].view(R, M * K)
        pb = pool_b[:R * K * N].view(R, K * N)
        pa.copy_(At.reshape(1, -1).expand(R, -1))
        pb.copy_(Bt.reshape(1, -1).expand(R, -1))
        a0, b0, c0 = pa.data_ptr(), pb.data_ptr(), pool_c.data_ptr()
        sa, sb, sc = M * K * 2, K * N * 2, M * N * 2
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(spin_cycles)
        e0.record(stream)
        for r in range(R):
            st = gemm(M, N, K, 1, a0 + r * sa, b0 + r * sb, c0 + r * sc, sp)
            if st != 0:
                raise RuntimeError("vx_gemm M=%d: %s" % (M, vx.STATUS.get(st, st)))
        e1.record(stream)
        return e0, e1, R

    def sweep():
        evs = [window(i) for i in range(len(sets))]
        torch.cuda.synchronize()
        return [e0.elapsed_time(e1) / R for (e0, e1, R) in evs]      # ms per call

    # host cost per call with cached plans (selector lookup + launch)
    one_pass()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    one_pass()
    host_us = (time.perf_counter() - t0) / len(calls) * 1e6
    torch.cuda.synchronize()
    # a short spin ahead of each window lets the host enqueue ahead of the device
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    torch.cuda._sleep(1000000)
    e1.record(stream)
    torch.cuda.synchronize()
    cycles_per_ms = 1e6 / max(e0.elapsed_time(e1), 1e-3)
    spin_cycles = int(cycles_per_ms * 0.3)

    for _ in range(args.warmup):
        sweep()
    torch.cuda.synchronize()
    per_step = []
    for s in range(args.steps):
        t = sweep()
        per_step.append(t)
        print("step %d: sweep device time %.3f ms" % (s, sum(t)), file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    step_ms = [sum(t) for t in per_step]

    # the plain pass: each M once, back to back, two events around the pass
    pass_ms = []
    for _ in range(3):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(spin_cycles * 10)
        e0.record(stream)
        one_pass()
        e1.record(stream)
        torch.cuda.synchronize()
        pass_ms.append(e0.elapsed_time(e1))

    # the outputs of the last timed pass, for the oracle's check in the CPU leg
    host_c = None if args.no_cpu_baseline else \
        {M: Ct.view(torch.int16).cpu().numpy().view(np.uint16) for (M, _, _, Ct) in sets}

    # the dispatch floor beside the sweep (every sweep shape's roofline time is below 5 us)
    launch_floor = _launch_floor_us(stream)
    k0_call = _k0_call_us(stream, L)

    # a stated sample of the three bf16 sets, timed like their own runs
    sets_out = {}
    if not args.no_sets:
        _device_warmup(dev)
        for name, trials in SET_SAMPLE:
            res = _time_jobs(_set_jobs(name, trials), args.rot_mib, dev, verbose=False)
            summ = _set_summary(res)
            summ["trials"] = "0..%d" % (trials - 1)
            sets_out[name] = summ
            print("set %s trials 0..%d: %.1f TFLOP/s geomean, roofline fraction %.3f"
                  % (name, trials - 1, summ["tflops_geomean"], summ["roof_frac_geomean"]), file=sys.stderr, flush=True)

    _copy_calibration(args, dev)

    med = np.median(np.array(per_step), axis=0)        # ms per call, per M
    flops = np.array([2.0 * M * N * K for M in ms])
    tflops = flops / (med * 1e-3) / 1e12
    geo = float(np.exp(np.mean(np.log(tflops))))

    # dominant kernel: the most device time over the sweep
    by_kernel = {}
    for i, M in enumerate(ms):
        kid = plans[M].kernel_id
        d = by_kernel.setdefault(kid, {"t": 0.0, "bytes": 0.0, "flops": 0.0, "n": 0, "ms": []})
        d["t"] += med[i] * 1e-3
        d["bytes"] += (M * K + K * N + M * N) * 2.0
        d["flops"] += flops[i]
        d["n"] += 1
        d["ms"].append(M)
    kid = max(by_kernel, key=lambda k: by_kernel[k]["t"])
    d = by_kernel[kid]
    kinfo = vx.vx_registry_get(kid)
    achieved = d["bytes"] / d["t"] / 1e9          # GB/s
    roofline = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBPS, "traffic": _profiled_traffic("vxk_%d" % kid),
                "kernel": "vxk_%d" % kid,
                "tile": [kinfo.mb, kinfo.nb, kinfo.kb, kinfo.wm, kinfo.wn, kinfo.mfma_m],
                "launches_per_step": d["n"], "avg_us": d["t"] / d["n"] * 1e6,
                "algorithmic_bytes_per_launch": d["bytes"] / d["n"]}
    # roofline fraction of the whole sweep: t_roof / t_measured per shape (geomean)
    t_roof = np.maximum(flops / (MFMA_PEAK_TFLOPS[1] * 1e12),
                        np.array([(M * K + K * N + M * N) * 2.0 for M in ms]) / (HBM_PEAK_GBPS * 1e9))
    sweep_frac = float(np.exp(np.mean(np.log(t_roof / (med * 1e-3)))))

    out = {
        "metric": "GEMM TFLOP/s geomean over dynamic-M sweep; % of MFMA/HBM roofline on 1 GPU",
        "value": geo, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": float(np.median(step_ms)), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f16", "data": "synthetic",
        "config": {"workload": "dynamic-M sweep: fp16 (M x 768) x (768 x 768), fp32 accumulate, fp16 out, "
                               "M = 1..%d, U[-1,1] seeded per M; one step = the sweep, each M timed over a "
                               "window of back-to-back calls on rotating HBM-resident copies" % args.m_max,
                   "M": "1..%d" % args.m_max, "N": N, "K": K, "calls_per_step": len(ms)},
        "roofline": roofline,
        "sweep_roofline_frac_geomean": sweep_frac,
        "host_us_per_call": host_us,
        "pass_ms_back_to_back": float(np.median(pass_ms)),
        "kernels_used": len(by_kernel),
        "launch_floor_us": launch_floor,
        "k0_call_us": k0_call,
    }
    if sets_out:
        out["sets"] = sets_out
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = _cpu_baseline(ms, args.cpu_seconds, host_c)
    if args.detail:
        with open(args.detail, "w") as f:
            json.dump({"M": ms, "ms": med.tolist(), "tflops": tflops.tolist(),
                       "kernel": [plans[M].kernel_id for M in ms], "split": [plans[M].split_k for M in ms],
                       "by_kernel": {str(k): {kk: vv for kk, vv in v.items()} for k, v in by_kernel.items()}},
                      f)
    out["selector"] = _selector_kind()
    print(json.dumps(out), flush=True)
    chk = out.get("cpu_baseline", {}).get("outputs_checked")
    if chk is not None and not chk["within_bound"]:
        print("sweep outputs outside the bound: %s" % chk.get("first_failure"), file=sys.stderr, flush=True)
        sys.exit(3)


if __name__ == "__main__":
    main()
