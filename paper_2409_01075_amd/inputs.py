"""Seeded synthetic inputs for the GEMM workloads.

This module only draws random numbers and rounds them to the storage type.
It holds none of the GEMM's arithmetic, so both the GPU library's tests and
the CPU oracle can read the very same stored operands.

Generator: numpy ``Generator(PCG64(seed))``.  Values are drawn in binary64,
then rounded to nearest-even into the storage type (fp32 and fp16 by numpy;
bf16 by rounding to fp32 first and then to bf16 with torch's CPU cast).
Operands are returned as numpy arrays of the stored bits: float32 for fp32,
uint16 bit patterns for fp16 and bf16.

Workloads (their shapes follow the paper's dynamic-shape GEMM families, the
Transformer rows of Table 3 and the BERT GEMM of Section 2.2, stretched to the
sizes listed below; the paper's own benchmark items are not reproduced):

* ``single_f32``  fp32 77 x 96 x 80, U[-1, 1], seed 0, A drawn before B.
* ``sweep_f16(M)``  fp16 (M x 768) x (768 x 768), U[-1, 1], seed = M.
* ``encoder_trial(t)``  bf16, seed t: L ~ U{1..512}, M = 16 L; four GEMMs
  (M,768)x(768,2304), (M,768)x(768,768), (M,768)x(768,3072),
  (M,3072)x(3072,768); activations N(0,1), weights N(0,0.02).
* ``attention_trial(t)``  bf16, seed t: L ~ U{1..1024}, batch 192;
  S = Q (L x 64) x K^T (64 x L) and O = P (L x L) x V (L x 64); Q, K, V ~ N(0,1);
  P = row softmax (binary64) of independent N(0,1) logits.
* ``llm_trial(t)``  bf16, seed t: M = clip(floor(exp(U[0, ln 8193))), 1, 8192);
  (M,4096)x(4096,4096), (M,4096)x(4096,11008), (M,11008)x(11008,4096);
  activations N(0,1), weights N(0,0.02).
* ``conv_trial(t)``  fp16, seed 5000 + t: one convolution layer drawn inside
  the ranges of the paper's CNN convolution family (Table 4: batch 1..64,
  feature map 4..768, filter 1..11, Cin 3..832, Cout 16..512).  Filter F from
  {1, 3, 5, 7, 11} with weights (.35, .45, .08, .07, .05); a 7 x 7 or 11 x 11
  filter is a stem layer (Cin = 3) half of the time; Cin = 8 round(e^U[ln 2,
  ln 104]) otherwise, Cout = 16 round(e^U[0, ln 32]); stride 2 with
  probability 1/4 (4 for an 11 x 11 stem); padding F // 2; feature map
  round(e^U[ln 4, ln 768]) and batch round(e^U[0, ln 64]), halved (batch
  first, then the map) until the layer holds at most 2^25 input and 2^25
  output elements and 4e11 flops.  Images N(0, 1), filters N(0, 0.05).
  ``conv_trial(t, "plain")`` keeps every dimension but draws
  Cin = round(e^U[ln 3, ln 832]) (seed 9000 + t): mostly not a multiple of 8.
* ``small_int`` helpers: integer-valued operands whose every partial sum is
  exact in fp32 and whose result is exact in the output type.
"""
import numpy as np

F32, F16, BF16 = 0, 1, 2
DTYPES = {"f32": F32, "f16": F16, "bf16": BF16}
ENCODER_SHAPES = [(768, 2304), (768, 768), (768, 3072), (3072, 768)]   # (K, N) per GEMM
LLM_SHAPES = [(4096, 4096), (4096, 11008), (11008, 4096)]              # (K, N) per GEMM
ATTN_BATCH = 16 * 12
ATTN_HEAD = 64


CONV_FILTERS = (1, 3, 5, 7, 11)
CONV_FILTER_P = (0.35, 0.45, 0.08, 0.07, 0.05)


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def code_of(dtype):
    return dtype if isinstance(dtype, int) else DTYPES[dtype]


def to_storage(x, dtype):
    """binary64 values -> stored values (float32 array or uint16 bit patterns)."""
    code = code_of(dtype)
    x = np.asarray(x, dtype=np.float64)
    if code == F32:
        return x.astype(np.float32)
    if code == F16:
        return x.astype(np.float16).view(np.uint16)
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x.astype(np.float32))).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def uniform(g, shape, dtype, lo=-1.0, hi=1.0):
    return to_storage(g.uniform(lo, hi, size=shape), dtype)


def normal(g, shape, dtype, std=1.0):
    return to_storage(g.normal(0.0, std, size=shape), dtype)


def single_f32(seed=0):
    g = rng(seed)
    A = uniform(g, (77, 80), F32)
    B = uniform(g, (80, 96), F32)
    return A, B


def sweep_f16(M, K=768, N=768):
    g = rng(M)
    A = uniform(g, (M, K), F16)
    B = uniform(g, (K, N), F16)
    return A, B


def encoder_shape(t):
    L = int(rng(t).integers(1, 513))
    return 16 * L


def encoder_trial(t, gemms=(0, 1, 2, 3)):
    """Returns (M, [(A, B) for each GEMM in ENCODER_SHAPES order])."""
    g = rng(t)
    L = int(g.integers(1, 513))
    M = 16 * L
    out = []
    for i, (K, N) in enumerate(ENCODER_SHAPES):
        A = normal(g, (M, K), BF16, 1.0)
        B = normal(g, (K, N), BF16, 0.02)
        if i in gemms:
            out.append((A, B))
    return M, out


def attention_L(t):
    return int(rng(t).integers(1, 1025))


def attention_trial(t, batch=ATTN_BATCH, d=ATTN_HEAD):
    """Returns (L, Q, Kt, P, V) with Q [b,L,d], Kt [b,d,L] (materialised K^T),
    P [b,L,L], V [b,L,d], all bf16 bit patterns, contiguous."""
    g = rng(t)
    L = int(g.integers(1, 1025))
    Q = normal(g, (batch, L, d), BF16)
    Kmat = g.normal(0.0, 1.0, size=(batch, L, d))
    Kt = to_storage(np.ascontiguousarray(np.swapaxes(Kmat, 1, 2)), BF16)
    del Kmat
    V = normal(g, (batch, L, d), BF16)
    P = np.empty((batch, L, L), dtype=np.uint16)
    for b in range(batch):            # one head at a time keeps host memory small
        z = g.normal(0.0, 1.0, size=(L, L))
        z -= z.max(axis=1, keepdims=True)
        e = np.exp(z)
        P[b] = to_storage(e / e.sum(axis=1, keepdims=True), BF16)
    return L, Q, Kt, P, V


def llm_M(t):
    u = rng(t).uniform(0.0, np.log(8193.0))
    return int(min(max(np.floor(np.exp(u)), 1), 8192))


def llm_trial(t, gemms=(0, 1, 2)):
    """Returns (M, [(A, B) per GEMM in LLM_SHAPES order])."""
    g = rng(t)
    u = g.uniform(0.0, np.log(8193.0))
    M = int(min(max(np.floor(np.exp(u)), 1), 8192))
    out = []
    for i, (K, N) in enumerate(LLM_SHAPES):
        A = normal(g, (M, K), BF16, 1.0)
        B = normal(g, (K, N), BF16, 0.02)
        if i in gemms:
            out.append((A, B))
    return M, out


def device_normal(shape, std, seed, device, dtype):
    """Seeded N(0, std) values drawn on the device (for timing runs at full
    workload sizes, where host generation would dominate the run time)."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    t = torch.empty(shape, dtype=torch.float32, device=device)
    t.normal_(0.0, std, generator=gen)
    return t.to(dtype)


def device_softmax_rows(shape, seed, device, dtype):
    """Seeded row softmax (binary64) of N(0, 1) logits, drawn on the device
    (timing runs and full-size parity), rounded to `dtype`."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    z = torch.empty(shape, dtype=torch.float64, device=device)
    z.normal_(0.0, 1.0, generator=gen)
    return torch.softmax(z, dim=-1).to(dtype)


def device_set(name, trials=None):
    """The GEMMs of a bf16 workload set as drawn for the device runs (timing and
    full-size parity): a list of (label, batch, M, N, K, make), where make(dev)
    returns the seeded device operands (A, B) as bf16 torch tensors -- A with
    batch * M rows of K, B with batch * K rows of N.  Shapes come from the
    set's seeded draws (encoder_shape, attention_L, llm_M); values from
    device_normal / device_softmax_rows with seed 1000 t + operand index.

    name: "encoder" (64 trials x 4 GEMMs), "attention" (32 trials x S and O,
    batch 192) or "llm" (48 trials x 3 GEMMs)."""
    import torch
    bf = torch.bfloat16
    jobs = []
    if name == "encoder":
        for t in range(64 if trials is None else trials):
            M = encoder_shape(t)
            for gi, (K, N) in enumerate(ENCODER_SHAPES):
                def mk(dev, t=t, gi=gi, M=M, K=K, N=N):
                    return (device_normal((M, K), 1.0, 1000 * t + 2 * gi, dev, bf),
                            device_normal((K, N), 0.02, 1000 * t + 2 * gi + 1, dev, bf))
                jobs.append(("t%d G%d (%d,%d)x(%d,%d)" % (t, gi + 1, M, K, K, N), 1, M, N, K, mk))
    elif name == "llm":
        for t in range(48 if trials is None else trials):
            M = llm_M(t)
            for gi, (K, N) in enumerate(LLM_SHAPES):
                def mk(dev, t=t, gi=gi, M=M, K=K, N=N):
                    return (device_normal((M, K), 1.0, 1000 * t + 2 * gi, dev, bf),
                            device_normal((K, N), 0.02, 1000 * t + 2 * gi + 1, dev, bf))
                jobs.append(("t%d H%d (%d,%d)x(%d,%d)" % (t, gi + 1, M, K, K, N), 1, M, N, K, mk))
    elif name == "attention":
        b, d = ATTN_BATCH, ATTN_HEAD
        for t in range(32 if trials is None else trials):
            L = attention_L(t)
            def mk_s(dev, t=t, L=L):
                return (device_normal((b, L, d), 1.0, 1000 * t, dev, bf),
                        device_normal((b, d, L), 1.0, 1000 * t + 1, dev, bf))
            def mk_o(dev, t=t, L=L):
                return (device_softmax_rows((b, L, L), 1000 * t + 2, dev, bf),
                        device_normal((b, L, d), 1.0, 1000 * t + 3, dev, bf))
            jobs.append(("t%d S L=%d" % (t, L), b, L, L, d, mk_s))
            jobs.append(("t%d O L=%d" % (t, L), b, L, d, L, mk_o))
    else:
        raise ValueError("unknown set %r" % name)
    return jobs


def small_int(g, shape, dtype, lo, hi):
    """Integers drawn uniformly from [lo, hi] (inclusive), stored exactly."""
    return to_storage(g.integers(lo, hi + 1, size=shape).astype(np.float64), dtype)


def exact_range(K, dtype):
    """Largest integer magnitude r such that K * r * r stays exactly representable
    in the output type (11 significand bits fp16, 8 bf16, 24 fp32), so that every
    partial sum in any order is exact and the output needs no rounding."""
    p = {F32: 24, F16: 11, BF16: 8}[code_of(dtype)]
    r = int(np.floor(np.sqrt((2.0 ** p) / max(K, 1))))
    return max(r, 0)


def conv_trial(t, cin="models"):
    """(N, H, W, Cin, Cout, F, stride, pad) of convolution trial t (fp16, square
    filter and map, dilation 1).  cin="models": channel counts as CNN layers
    have them (3 for a stem, else a multiple of 8); cin="plain": Cin drawn
    log-uniformly over the whole range 3..832 from a stream of its own (seed
    9000 + t), every other dimension as in "models"."""
    g = rng(5000 + t)
    F = int(g.choice(CONV_FILTERS, p=CONV_FILTER_P))
    stem = F >= 7 and g.random() < 0.5
    Cin = 3 if stem else 8 * int(round(np.exp(g.uniform(np.log(2), np.log(104)))))
    if cin == "plain":
        Cin = int(round(np.exp(rng(9000 + t).uniform(np.log(3), np.log(832)))))
    elif cin != "models":
        raise ValueError("cin must be 'models' or 'plain'")
    Cout = 16 * int(round(np.exp(g.uniform(0.0, np.log(32)))))
    stride = (4 if F == 11 else 2) if (stem or g.random() < 0.25) else 1
    pad = F // 2
    H = int(round(np.exp(g.uniform(np.log(4), np.log(768)))))
    N = int(round(np.exp(g.uniform(0.0, np.log(64)))))

    def size(N, H):
        OH = (H + 2 * pad - F) // stride + 1
        return N * H * H * Cin, N * OH * OH * Cout, 2.0 * N * OH * OH * Cout * F * F * Cin
    while True:
        xi, yo, fl = size(N, H)
        if xi <= 2 ** 25 and yo <= 2 ** 25 and fl <= 4e11:
            break
        if N > 1:
            N //= 2
        else:
            H = max(H // 2, F)
            if H == F:
                break
    return N, H, H, Cin, Cout, F, stride, pad
