"""Build-time candidate generation (Section 5.1, Algorithm 2) for gfx950.

Runs once, offline, when the library is built.  Algorithm 2 builds each
level's candidates as integer multiples of the level below it and links every
upper tile to the lower tiles it is made of; here the three levels are plain
functions of the hardware table, each calling the one below:
  mfma_tiles        L0  instruction tiles (m0, n0, k0) the ISA offers per dtype.
  wave_tiles        L1  wavefront tiles (Mw, Nw), register level: multiples of
                        an L0 tile, {wave tile: [its L0 tiles]}.
  workgroup_tiles   L2  workgroup tiles (Mb, Nb, Kb) with wm x wn wavefronts,
                        LDS level: multiples of an L1 tile,
                        {workgroup tile: [(wave tile, L0 tile)]}.
The grid level has no tile of its own: it is the runtime parallel loop.  The
workgroup tiles that pass the feasibility rules become the kernel
instantiations compiled into the library; the runtime selector then chooses
among them analytically (Section 5.2).

Two level-1 load strategies exist (the Load stage of Algorithm 1 at the
workgroup level):
  * "dma": fp16/bf16 tiles loaded by 16-byte buffer-load-to-LDS instructions
    into a ring of STAGES LDS stages (no VGPR staging); B keeps its
    n-contiguous layout and is read with the transposing LDS read.  Each tile
    is offered with 2 stages, with the deepest ring of 3 or 4, and with the
    deepest of 5..16 that fits (a whole short K range in flight).
  * "reg": loads staged through VGPRs into a 2-stage LDS ring (fp32; fp16/bf16
    operands that are not 16-byte aligned; a few fp16/bf16 tiles for operands
    whose byte extents exceed 32-bit buffer offsets).

Feasible range (the paper prunes candidates whose use of a hardware level is
"extremely low or high" without giving thresholds; the thresholds below are
this library's reading):
  * L1: accumulator registers Mw*Nw/64 in [4, 128] of the 512 per lane for
    register-staged tiles (staging, fragments and addresses must fit beside
    them), [4, 256] for direct-to-LDS tiles (no staging registers); aspect <= 4.
  * L2: 4 wavefronts per workgroup (one per SIMD of the CU), 8 for tiles of
    at least 128 x 128, 1 or 2 for tiles of at most 512 outputs (16 x 16, 16 x 32, 32 x 16); LDS for a 2-stage ring <= 160 KiB; the K step reads at
    least 128 contiguous bytes per row (two 64-byte segments); aspect of the
    workgroup tile <= 8.  DMA tiles: A and B split into whole 1 KiB wave
    transfers per K step.  Register-staged tiles: every thread moves at least
    one 16-byte vector of A and of B per K step and at most 32 (<= 128 staging
    VGPRs).
  * L0 per L1 link: the 32 x 32 MFMA when both wavefront dims are multiples of
    32 and at least 64 (half the fragment loads per FLOP of the 16 x 16 shape),
    else the 16 x 16 MFMA.  The paper takes this decision by profiling L0
    offline; until such a calibration exists this fixed rule stands in.
"""
import json
import sys

GFX950 = {
    "arch": "gfx950",
    "lds_bytes": 160 * 1024,
    "vgprs_per_lane": 512,
    "max_threads": 1024,
    "wave": 64,
    # MFMA instructions with fp32 accumulation: (m, n, k) per dtype
    "mfma": {
        "f16": [(16, 16, 32), (32, 32, 16)],
        "bf16": [(16, 16, 32), (32, 32, 16)],
        "f32": [(16, 16, 4), (32, 32, 2)],
    },
}
DT_CODE = {"f32": 0, "f16": 1, "bf16": 2}
LDS_RESERVE = 1024   # the split-K arrival flag and alignment share the CU's LDS
ELEM_BYTES = {"f32": 4, "f16": 2, "bf16": 2}


WAVE_GRIDS = [(1, 1), (1, 2), (2, 1), (2, 2), (1, 4), (4, 1), (2, 4), (4, 2)]


def lds_bytes(dtype, mb, nb, kb):
    eb = ELEM_BYTES[dtype]
    pad = 16 // eb
    if eb == 2:
        stage = (mb * (kb + pad) + nb * (kb + pad)) * eb
    else:
        stage = (mb * (kb + pad) + kb * (nb + 4)) * eb
    return 2 * stage


def lds_bytes_dma(mb, nb, kb, stages):
    return stages * (mb * kb + kb * nb) * 2


DEEP_MAX = 16   # deepest ring offered (K steps in flight = stages - 1)


def dma_stage_options(mb, nb, kb, wm, wn, mi, vec, hw):
    """Pipeline depths offered for a DMA tile: 2, the deepest of 3..4, and
    the deepest of 5..DEEP_MAX, each if it fits the LDS and the 6-bit vmcnt
    of the waits.  Deep rings keep a whole short K range in flight at once:
    a latency-bound call then waits for one memory round trip instead of
    one per group of STAGES-1 K steps."""
    nwave = wm * wn
    lane = 16 if vec else 2
    wave_bytes = 64 * lane
    a_bytes, b_bytes = mb * kb * 2, kb * nb * 2
    if a_bytes % (wave_bytes * nwave) or b_bytes % (wave_bytes * nwave):
        return []
    lps = a_bytes // (wave_bytes * nwave) + b_bytes // (wave_bytes * nwave)
    def fits(st):
        return lds_bytes_dma(mb, nb, kb, st) <= hw["lds_bytes"] - LDS_RESERVE and (st - 1) * lps <= 63
    ok = [st for st in (2, 3, 4) if fits(st)]
    if not ok:
        return []
    deep = [st for st in range(5, DEEP_MAX + 1) if fits(st)]
    return sorted({ok[0], ok[-1]} | set(deep[-1:]))


def feasible_l2(dtype, mb, nb, kb, wm, wn, mi, hw, family):
    eb = ELEM_BYTES[dtype]
    nt = wm * wn * hw["wave"]
    ve = 16 // eb
    if nt > hw["max_threads"]:
        return False
    waves = wm * wn
    # one wavefront per SIMD; 8 for large tiles; 1 or 2 for small tiles, which
    # give latency-bound calls (small M, or small N) more workgroups to spread
    # over the CUs
    if not (waves == 4 or (waves == 8 and mb >= 128 and nb >= 128) or (waves <= 2 and mb * nb <= 512)):
        return False
    if max(mb, nb) > 8 * min(mb, nb) or max(mb, nb) > 256:
        return False
    if kb * eb < 128:
        return False
    # K chunk of one fragment load
    kch = (32 if mi == 16 else 16) if eb == 2 else (16 if mi == 16 else 8)
    if kb % kch:
        return False
    if family == "dma":
        # direct-to-LDS loads: a 2-stage ring of vector DMA must fit
        return eb == 2 and bool(dma_stage_options(mb, nb, kb, wm, wn, mi, 1, hw))
    # register-staged loads
    if lds_bytes(dtype, mb, nb, kb) > hw["lds_bytes"] - LDS_RESERVE:
        return False
    a_vec = mb * kb // ve
    b_vec = nb * kb // ve
    if a_vec % nt or b_vec % nt:
        return False
    if not (1 <= a_vec // nt <= 32 and 1 <= b_vec // nt <= 32):
        return False
    if a_vec // nt + b_vec // nt > 32:
        return False
    if eb == 2:
        # B is staged in blocks of BK rows x 8 columns (BK in {8, 4, 2})
        if not any((kb // bk) * (nb // 8) >= nt and (kb // bk) * (nb // 8) % nt == 0 for bk in (8, 4, 2)):
            return False
    return True


# ------------------------------------------------------------ the levels -----
def mfma_tiles(dtype, hw=GFX950):
    """Level 0: the matrix-core instruction tiles (m, n, k) with fp32
    accumulation that the ISA offers for `dtype`."""
    return list(hw["mfma"][dtype])


def wave_tiles(dtype, hw=GFX950, family="reg"):
    """Level 1: wavefront tiles (Mw, Nw) that are integer multiples of at least
    one level-0 tile, with Mw * Nw / 64 fp32 accumulators per lane within the
    family's budget (register-staged tiles keep up to 128 VGPRs for their
    staging registers; direct-to-LDS tiles stage nothing in VGPRs and may use
    256, the AGPR half of the file) and an aspect of at most 4.
    Returns {wave tile: [the level-0 tiles it is a multiple of]}."""
    acc_max = 256 if family == "dma" else 128
    out = {}
    for mw in (16, 32, 64, 128, 256):
        for nw in (16, 32, 64, 128, 256):
            acc = mw * nw // hw["wave"]
            if not (4 <= acc <= acc_max and max(mw, nw) <= 4 * min(mw, nw)):
                continue
            below = [t for t in mfma_tiles(dtype, hw) if mw % t[0] == 0 and nw % t[1] == 0]
            if below:
                out[(mw, nw)] = below
    return out


def mfma_for(mw, nw):
    """The instruction tile a wavefront tile is built from: 32 x 32 when both
    sides are multiples of 32 and at least 64 (half the fragment loads per
    FLOP of 16 x 16), else 16 x 16."""
    return 32 if (mw % 32 == 0 and nw % 32 == 0 and min(mw, nw) >= 64) else 16


def workgroup_tiles(dtype, hw=GFX950, family=None):
    """Level 2: workgroup tiles (Mb, Nb, Kb, wm, wn, mi) = (wm Mw, wn Nw, Kb) for
    every wavefront tile (Mw, Nw) and wavefront grid (wm, wn), with Kb a
    multiple of the instruction's k, that pass the feasibility rules of the
    family (feasible_l2).  Returns {workgroup tile: [(wave tile, mfma tile)]}."""
    if family is None:
        family = "dma" if ELEM_BYTES[dtype] == 2 else "reg"
    kbs = (64, 128, 256) if ELEM_BYTES[dtype] == 2 else (32, 64)
    out = {}
    for (mw, nw), below in wave_tiles(dtype, hw, family).items():
        for (wm, wn) in WAVE_GRIDS:
            for kb in kbs:
                for l0 in below:
                    if l0[0] != mfma_for(mw, nw) or kb % l0[2]:
                        continue
                    c = (wm * mw, wn * nw, kb, wm, wn, l0[0])
                    if not feasible_l2(dtype, *c, hw, family):
                        continue
                    out.setdefault(c, []).append(((mw, nw), l0))
    return out


# fp16/bf16 register-staged vector-load tiles kept for operands whose byte
# extents exceed 32-bit buffer offsets
REG_FALLBACK_16 = [(32, 32, 128, 2, 2, 16), (64, 64, 64, 2, 2, 16), (128, 128, 64, 2, 2, 32)]


# Wide tiles (direct-to-LDS, fp16/bf16): workgroup tiles with a 192 side --
# an integer multiple (3) of the 64-wide step between the power-of-two tiles,
# outside the power-of-two L1 set above -- with 8 wavefronts whose tiles
# follow the L1 rules (accumulators, aspect <= 4).  They give the grid level
# tile counts between those of the 128 and 256 tiles: a 6976 x 768 output is
# 330 tiles of 128 x 128 (1.3 per CU) but 222 of 192 x 128.
WIDE_TILES = [(192, 128), (128, 192), (192, 192), (256, 192), (192, 256)]


def dma_wide_candidates(dtype, hw=GFX950):
    out = []
    for (mb, nb) in WIDE_TILES:
        for (wm, wn) in ((2, 4), (4, 2)):
            mw, nw = mb // wm, nb // wn
            acc = mw * nw // hw["wave"]
            if mw % 16 or nw % 16 or not (4 <= acc <= 256) or max(mw, nw) > 4 * min(mw, nw):
                continue
            c = (mb, nb, 64, wm, wn, mfma_for(mw, nw))
            for st in dma_stage_options(*c, 1, hw):
                out.append(_entry(dtype, "dma", st, c, 1, hw))
    return out


def _entry(dtype, family, stages, c, vec, hw):
    mb, nb, kb, wm, wn, mi = c
    lds = lds_bytes_dma(mb, nb, kb, stages) if family == "dma" else lds_bytes(dtype, mb, nb, kb)
    return dict(dtype=dtype, dt=DT_CODE[dtype], family=family, stages=stages, mb=mb, nb=nb, kb=kb, wm=wm,
                wn=wn, mi=mi, vec=vec, threads=wm * wn * hw["wave"], lds=lds, k_max=0, op=0, schedule=0)


# ------------------------------------------------ convolution (implicit GEMM) --
# The paper's second operator on the same hierarchy: a convolution is the
# GEMM of its output pixels (M = n*oh*ow) by its filter (K = kh*kw*c_in rows,
# N = c_out columns), with the A tile gathered from the image through the
# im2col map.  The conv kernels are register-staged, element-aligned
# workgroup tiles of the GEMM candidates (the gather goes through VGPRs
# anyway): one K step of 64 (16-bit) or 32 (fp32) elements, tiles from 32 x 32
# to 128 x 128.
CONV_TILES = {(32, 32), (32, 64), (64, 32), (64, 64), (64, 128), (128, 64), (128, 128)}


# Tiles of at most 64 x 64 also come with three register sets of K steps in
# flight (stages = 4: the register sets plus the LDS stage being computed):
# a small layer with few workgroups and few K steps (a first layer over three
# channels: K = 147, three steps) otherwise waits one gather round trip per
# K step.
CONV_PF_TILES = {(32, 32), (32, 64), (64, 32), (64, 64)}


def conv_candidates(dtype, hw=GFX950, pf=False):
    kb = 64 if ELEM_BYTES[dtype] == 2 else 32
    out = []
    for c in workgroup_tiles(dtype, hw, "reg"):
        mb, nb, ckb, wm, wn, mi = c
        if ckb == kb and (mb, nb) in CONV_TILES and wm * wn == 4 and (not pf or (mb, nb) in CONV_PF_TILES):
            e = _entry(dtype, "reg", 4 if pf else 2, c, 0, hw)
            e["op"] = 1
            out.append(e)
    return out


# fp16/bf16 convolutions whose channel counts are multiples of 8 (and whose
# image fits 32-bit buffer offsets) also get direct-to-LDS tiles: each lane's
# 16-byte chunk is one tap's 8 channels, fetched with its own buffer offset,
# and a tap in the padding gets an out-of-range offset that reads as zeros.
# Kb = 64 (one 128-byte row segment per 8 lanes keeps a lane's chunk column
# fixed); 4 waves below 128 x 128, 8 from there up to 256 x 128 (256 x 256
# spills with the map state); wave tiles at most 2:1; the 2-stage ring and
# the deepest ring of at most 4 stages.
def conv_dma_candidates(dtype, hw=GFX950):
    out = []
    for c in workgroup_tiles(dtype, hw, "dma"):
        mb, nb, kb, wm, wn, mi = c
        mw, nw = mb // wm, nb // wn
        if kb != 64 or min(mb, nb) < 64 or mb * nb > 256 * 128 or wm * wn != (8 if mb * nb >= 128 * 128 else 4):
            continue
        if max(mw, nw) > 2 * min(mw, nw):
            continue
        st = dma_stage_options(*c, 1, hw)
        for s in sorted({st[0], max(x for x in st if x <= 4)}):
            e = _entry(dtype, "dma", s, c, 1, hw)
            e["op"] = 1
            out.append(e)
    return out


# fp16/bf16 convolutions whose channel count is not a multiple of 8 (the
# image's 16-byte chunks do not start on tap boundaries) but whose filter rows
# are (c_out a multiple of 8): the filter by DMA and the image through VGPRs
# with the register-staged kernels' im2col gather, into the same LDS layout
# (mixed loads, VG 1).  The 2-stage direct-to-LDS convolution tiles of at
# least 64 x 128 whose image chunks split evenly over the threads (a 64 x 64
# mixed tile ran small layers up to 1.5x slower than the register-staged
# tiles the selector would otherwise take, and won only some by up to 1.5x).
def conv_mixed_candidates(dtype, hw=GFX950):
    out = []
    for e in conv_dma_candidates(dtype, hw):
        nt = e["wm"] * e["wn"] * hw["wave"]
        chunks = e["mb"] * (e["kb"] // 8)
        if e["stages"] != 2 or chunks % nt or chunks // nt > 16 or e["mb"] * e["nb"] < 64 * 128:
            continue
        m = dict(e)
        m["vg"] = 1
        m["vec"] = 0
        m["align"] = 2
        out.append(m)
    return out


# ------------------------------------------------- vector-ALU family (L0') --
# The adaptive second backend for small M (the paper's CUDA-core path next to
# the tensor-core path): level 0 is one lane's MT x VE outputs computed with
# v_dot2 (16-bit, on pairs of k) or v_fma (fp32) instead of an MFMA tile.
# One 16-byte chunk per lane of a B row, 8 lanes per 128-byte row segment:
# NB = 8 chunks; 8 k groups per wave; U groups per lane per register set.
VALU_ROWS = (4, 8, 16)
VALU_WAVES = (4, 8)
VALU_U = (2, 4)
VALU_A_LDS = 128 * 1024     # the A slice held in LDS


def valu_candidates(dtype, hw=GFX950):
    eb = ELEM_BYTES[dtype]
    ve = 16 // eb
    nb = 8 * ve
    pk = 2 if eb == 2 else 1
    out = []
    for mt in VALU_ROWS:
        for waves in VALU_WAVES:
            for u in VALU_U:
                kpi = waves * 8 * pk * u
                kmax = min(8192, VALU_A_LDS // (mt * eb)) // kpi * kpi
                red = waves * mt * nb * 4
                lds = max(kmax * mt * eb, red)
                # accumulators mt x ve, two register sets of u x pk chunks: within 512 VGPRs per lane
                # for one wave per SIMD, 256 for two
                regs = mt * ve + 2 * u * pk * 4 + mt + ve + 24
                if regs > (512 if waves <= 4 else 256) or kmax < kpi or lds > hw["lds_bytes"] - LDS_RESERVE:
                    continue
                out.append(dict(dtype=dtype, dt=DT_CODE[dtype], family="valu", stages=u, mb=mt, nb=nb, kb=kpi, wm=1,
                                wn=waves, mi=0, vec=1, threads=waves * hw["wave"], lds=lds, k_max=kmax, op=0))
    return out


# Ping-pong DMA issue (direct-to-LDS, 8 waves, 2-stage ring): instead of every
# wave issuing its share of the next K step right after the barrier (all
# eight then wait on the CU's load path together, with the matrix cores
# idle), the two halves of the waves -- one wave per SIMD each -- take turns
# issuing whole K steps, and the other half starts its MFMAs at once.
def pingpong_candidates(base):
    out = []
    for e in base:
        if e["family"] == "dma" and e["op"] == 0 and e["stages"] == 2 and e["wm"] * e["wn"] == 8:
            a_instr = e["mb"] * e["kb"] * 2 // 1024
            b_instr = e["kb"] * e["nb"] * 2 // 1024
            if a_instr % 4 or b_instr % 4 or 2 * (a_instr + b_instr) // 8 > 63:
                continue
            p = dict(e)
            p["schedule"] = 1
            out.append(p)
    return out


# Mixed loads (fp16/bf16): one operand by DMA, the other -- whose rows need not
# start on 16-byte boundaries (an odd K for A, an odd N for B, or such a batch
# stride) -- through VGPRs into the same LDS layout.  A GEMM with one misaligned
# operand then keeps the DMA for the other instead of falling back to the
# register-staged family for both.  Kb = 64, 2-stage rings, one wave layout
# per workgroup tile (the first the generator lists).
MIXED_TILES = {(32, 64), (64, 32), (64, 64), (128, 64), (64, 128), (128, 128), (256, 64), (64, 256), (256, 128),
               (128, 256), (256, 256)}


def mixed_candidates(base, hw=GFX950):
    out, seen = [], set()
    for e in base:
        if e["family"] != "dma" or e["op"] or e["stages"] != 2 or e.get("schedule", 0) or e["kb"] != 64:
            continue
        if (e["mb"], e["nb"]) not in MIXED_TILES or (e["dtype"], e["mb"], e["nb"]) in seen:
            continue
        nt = e["wm"] * e["wn"] * hw["wave"]
        for vg in (1, 2):
            chunks = e["mb"] * (e["kb"] // 8) if vg == 1 else e["kb"] * (e["nb"] // 8)
            if chunks % nt or chunks // nt > 16:
                continue
            m = dict(e)
            m["vg"] = vg
            m["vec"] = 0
            m["align"] = 2 if vg == 1 else 1
            out.append(m)
        seen.add((e["dtype"], e["mb"], e["nb"]))
    return out


# Short-K tiles (fp16/bf16, direct-to-LDS, 2-stage rings of Kb = 32): a GEMM
# whose K is one or two steps of the usual Kb = 64 (the attention scores
# Q x K^T, K = head size 64) has nothing to overlap with its only K step's
# loads.  With Kb = 32 the second step's DMA flies while the first computes,
# and the ring alone (2 x (Mb + Nb) x 32 x 2 bytes) is smaller than the C tile
# staged for the LDS epilogue, so the LDS is sized for the staged tile
# instead.  Three tiles, each with both operands by DMA and with B through
# VGPRs (rows not 16-byte aligned, odd lengths).
SHORT_K_TILES = ((128, 128, 32, 2, 2, 32), (128, 128, 32, 4, 2, 16), (128, 256, 32, 2, 4, 32))


def short_k_candidates(dtype, hw=GFX950):
    out = []
    for (mb, nb, kb, wm, wn, mi) in SHORT_K_TILES:
        nt = wm * wn * hw["wave"]
        lds = max(lds_bytes_dma(mb, nb, kb, 2), mb * (nb + 8) * 2)
        for vg in (0, 2):
            if vg == 2 and (kb * (nb // 8)) % nt:
                continue
            e = _entry(dtype, "dma", 2, (mb, nb, kb, wm, wn, mi), 1 if vg == 0 else 0, hw)
            e["lds"] = lds
            e["fit_c"] = 1
            if vg:
                e["vg"] = vg
                e["align"] = 1
            out.append(e)
    return out


def registry(hw=GFX950):
    """All workgroup-level candidates that are compiled into the library.

    fp16/bf16: direct-to-LDS tiles with 16-byte loads (16-byte-aligned
    operands), each with a 2-stage and with its deepest ring; register-staged
    tiles for element-aligned operands (misaligned 16-byte row chunks; a
    2-byte buffer-to-LDS load fills a whole dword of LDS, so unaligned rows
    cannot be DMA'd densely); and a few register-staged 16-byte-aligned tiles
    for very large operands.
    fp32: register-staged tiles, each for 16-byte-aligned and for
    element-aligned operands."""
    out = []
    for dtype in ("f16", "bf16"):
        for c in workgroup_tiles(dtype, hw, "dma"):
            for st in dma_stage_options(*c, 1, hw):
                out.append(_entry(dtype, "dma", st, c, 1, hw))
        for c in workgroup_tiles(dtype, hw, "reg"):
            out.append(_entry(dtype, "reg", 2, c, 0, hw))
        for c in REG_FALLBACK_16:
            out.append(_entry(dtype, "reg", 2, c, 1, hw))
    for c in workgroup_tiles("f32", hw, "reg"):
        for vec in (1, 0):
            out.append(_entry("f32", "reg", 2, c, vec, hw))
    for dtype in ("f16", "bf16", "f32"):
        out += valu_candidates(dtype, hw)
    for dtype in ("f16", "bf16", "f32"):
        out += conv_candidates(dtype, hw)
    for dtype in ("f16", "bf16"):
        out += conv_dma_candidates(dtype, hw)
    for dtype in ("f16", "bf16"):
        out += dma_wide_candidates(dtype, hw)
    out += pingpong_candidates(list(out))
    out += mixed_candidates(list(out), hw)
    for dtype in ("f16", "bf16"):
        out += short_k_candidates(dtype, hw)
    for dtype in ("f16", "bf16"):
        out += conv_mixed_candidates(dtype, hw)
    for dtype in ("f16", "bf16", "f32"):
        out += conv_candidates(dtype, hw, pf=True)
    for i, e in enumerate(out):
        e["id"] = i
    return out


if __name__ == "__main__":
    reg = registry()
    for dt in ("f16", "bf16", "f32"):
        print(dt, "L0", len(mfma_tiles(dt)), "L1", len(wave_tiles(dt)), "L2", len(workgroup_tiles(dt)),
              file=sys.stderr)
    print(len(reg), file=sys.stderr)
    json.dump(reg, sys.stdout, indent=0)
