/*
 * CPU oracle for the dense GEMM C = A x B and the 2-D convolution (test
 * infrastructure only).
 *
 * Only the test suite, the smoke check and the CPU-baseline leg of the
 * benchmark may load this file's library.  The product path never calls it.
 *
 * What it computes (Section 4.1, the GEMM definition C = A x B, with the
 * dynamic M, N, K of Section 2.2):
 *
 *     Cref[i][j] = sum_{k=0}^{K-1} double(A[i][k]) * double(B[k][j])
 *     Mag[i][j]  = sum_{k=0}^{K-1} |double(A[i][k])| * |double(B[k][j])|
 *
 * in IEEE binary64, k ascending, one rounding per addition.  All matrices are
 * dense row-major: A is M x K, B is K x N, C is M x N.  A batched call applies
 * the same definition to every batch b with A + b*sA, B + b*sB (strides in
 * elements, sB = 0 broadcasts B).
 *
 * The inputs are the stored values: fp32, IEEE binary16 (fp16) or bfloat16
 * bit patterns.  The decoders and the round-to-nearest-even encoders below
 * are written from the formats' definitions and share nothing with the GPU
 * library.  Every product of two fp16/bf16/fp32 values is exact in binary64,
 * so only the additions round.  Build with -O2 -ffp-contract=off (no FMA
 * contraction, no fast-math).  Rows are split over threads, which does not
 * change any element's arithmetic.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_F32 = 0, OR_F16 = 1, OR_BF16 = 2 };

/* ---- codecs ------------------------------------------------------------- */

/* IEEE 754 binary16: 1 sign, 5 exponent (bias 15), 10 fraction bits. */
double oracle_f16_to_f64(uint16_t h)
{
    int s = (h >> 15) & 1, e = (h >> 10) & 0x1f, f = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);                 /* zero / subnormal: f * 2^-24 */
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(f | 0x400), e - 25);    /* (1024 + f) * 2^(e-15-10) */
    return s ? -v : v;
}

/* bfloat16: the upper 16 bits of an IEEE binary32. */
double oracle_bf16_to_f64(uint16_t h)
{
    int s = (h >> 15) & 1, e = (h >> 7) & 0xff, f = h & 0x7f;
    double v;
    if (e == 0)
        v = ldexp((double)f, -133);                /* subnormal: f * 2^(-126-7) */
    else if (e == 255)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(f | 0x80), e - 134);    /* (128 + f) * 2^(e-127-7) */
    return s ? -v : v;
}

/*
 * Round a binary64 to a binary format with `p` significand bits (hidden bit
 * included), minimum normal exponent `emin` and maximum exponent `emax`, to
 * nearest, ties to even.  Returns the encoded bits for fraction width p-1 and
 * exponent width ew.  Overflow goes to infinity, as IEEE round-to-nearest does.
 */
static uint16_t encode_rne(double x, int p, int emin, int emax, int ew)
{
    uint16_t sign = signbit(x) ? 1 : 0;
    int fw = p - 1, bias = (1 << (ew - 1)) - 1;
    uint16_t sbit = (uint16_t)(sign << (fw + ew));
    if (isnan(x))
        return (uint16_t)(sbit | (((1u << ew) - 1) << fw) | (1u << (fw - 1)));
    double a = fabs(x);
    if (isinf(a))
        return (uint16_t)(sbit | (((1u << ew) - 1) << fw));
    if (a == 0.0)
        return sbit;
    int e;
    frexp(a, &e);              /* a = m * 2^e, m in [0.5, 1): unbiased exponent e-1 */
    int ue = e - 1;
    if (ue < emin)
        ue = emin;             /* subnormal range shares the quantum of emin */
    double q = ldexp(1.0, ue - fw);        /* spacing of representable values */
    double n = a / q;                      /* exact: power-of-two scaling */
    double r = floor(n);
    double d = n - r;                      /* exact */
    if (d > 0.5 || (d == 0.5 && fmod(r, 2.0) != 0.0))
        r += 1.0;
    /* r * q is the rounded magnitude; it may have carried into the next binade */
    double rv = r * q;
    if (rv == 0.0)
        return sbit;
    int e2;
    frexp(rv, &e2);
    int ue2 = e2 - 1;
    if (ue2 > emax)
        return (uint16_t)(sbit | (((1u << ew) - 1) << fw));
    if (ue2 < emin) {          /* subnormal: exponent field 0, fraction = r */
        return (uint16_t)(sbit | (uint16_t)r);
    }
    uint32_t frac = (uint32_t)(ldexp(rv, fw - ue2) - ldexp(1.0, fw));
    return (uint16_t)(sbit | ((uint32_t)(ue2 + bias) << fw) | frac);
}

uint16_t oracle_f64_to_f16(double x) { return encode_rne(x, 11, -14, 15, 5); }
uint16_t oracle_f64_to_bf16(double x) { return encode_rne(x, 8, -126, 127, 8); }

void oracle_encode(int dtype, const double *in, void *out, int64_t n)
{
    int64_t i;
    if (dtype == OR_F32) {
        float *o = (float *)out;
        for (i = 0; i < n; ++i)
            o[i] = (float)in[i];           /* C conversion: current rounding mode, RNE */
    } else if (dtype == OR_F16) {
        uint16_t *o = (uint16_t *)out;
        for (i = 0; i < n; ++i)
            o[i] = oracle_f64_to_f16(in[i]);
    } else {
        uint16_t *o = (uint16_t *)out;
        for (i = 0; i < n; ++i)
            o[i] = oracle_f64_to_bf16(in[i]);
    }
}

void oracle_decode(int dtype, const void *in, double *out, int64_t n)
{
    int64_t i;
    if (dtype == OR_F32) {
        const float *p = (const float *)in;
        for (i = 0; i < n; ++i)
            out[i] = (double)p[i];
    } else if (dtype == OR_F16) {
        const uint16_t *p = (const uint16_t *)in;
        for (i = 0; i < n; ++i)
            out[i] = oracle_f16_to_f64(p[i]);
    } else {
        const uint16_t *p = (const uint16_t *)in;
        for (i = 0; i < n; ++i)
            out[i] = oracle_bf16_to_f64(p[i]);
    }
}

static size_t elem_size(int dtype) { return dtype == OR_F32 ? 4 : 2; }

/* ---- the GEMM ----------------------------------------------------------- */

typedef struct {
    const double *A, *B;       /* decoded operands of one batch */
    double *C, *Mag;
    int64_t M, N, K;
    int64_t r0, r1;            /* rows handled by this thread */
} rows_job;

/* i-k-j order: one binary64 row accumulator, k ascending for every element. */
static void *gemm_rows(void *arg)
{
    rows_job *j = (rows_job *)arg;
    int64_t i, k, c;
    for (i = j->r0; i < j->r1; ++i) {
        double *crow = j->C + i * j->N;
        double *mrow = j->Mag ? j->Mag + i * j->N : NULL;
        for (c = 0; c < j->N; ++c)
            crow[c] = 0.0;
        if (mrow)
            for (c = 0; c < j->N; ++c)
                mrow[c] = 0.0;
        for (k = 0; k < j->K; ++k) {
            double a = j->A[i * j->K + k];
            const double *brow = j->B + k * j->N;
            for (c = 0; c < j->N; ++c)
                crow[c] += a * brow[c];
            if (mrow) {
                double aa = fabs(a);
                for (c = 0; c < j->N; ++c)
                    mrow[c] += aa * fabs(brow[c]);
            }
        }
    }
    return NULL;
}

/*
 * Batched oracle.  A, B are stored values of `dtype`; Cref and Mag (Mag may be
 * NULL) receive batch*M*N binary64 values, batch-major, row-major.
 * Returns 0 on success, -1 on bad arguments or allocation failure.
 */
int oracle_gemm(int dtype, int64_t batch, int64_t M, int64_t N, int64_t K,
                const void *A, int64_t sA, const void *B, int64_t sB,
                double *Cref, double *Mag, int threads)
{
    if (batch < 0 || M < 0 || N < 0 || K < 0 || dtype < 0 || dtype > 2)
        return -1;
    if (threads < 1)
        threads = 1;
    if (batch == 0 || M == 0 || N == 0)
        return 0;
    size_t es = elem_size(dtype);
    double *Ad = (double *)malloc(sizeof(double) * (size_t)(M * K > 0 ? M * K : 1));
    double *Bd = (double *)malloc(sizeof(double) * (size_t)(K * N > 0 ? K * N : 1));
    pthread_t *tid = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)threads);
    rows_job *jobs = (rows_job *)malloc(sizeof(rows_job) * (size_t)threads);
    if (!Ad || !Bd || !tid || !jobs) {
        free(Ad); free(Bd); free(tid); free(jobs);
        return -1;
    }
    int64_t b;
    for (b = 0; b < batch; ++b) {
        oracle_decode(dtype, (const char *)A + (size_t)(b * sA) * es, Ad, M * K);
        oracle_decode(dtype, (const char *)B + (size_t)(b * sB) * es, Bd, K * N);
        int t, nt = threads;
        if (nt > M)
            nt = (int)M;
        for (t = 0; t < nt; ++t) {
            jobs[t].A = Ad; jobs[t].B = Bd;
            jobs[t].C = Cref + b * M * N;
            jobs[t].Mag = Mag ? Mag + b * M * N : NULL;
            jobs[t].M = M; jobs[t].N = N; jobs[t].K = K;
            jobs[t].r0 = M * t / nt;
            jobs[t].r1 = M * (t + 1) / nt;
        }
        if (nt == 1) {
            gemm_rows(&jobs[0]);
        } else {
            for (t = 0; t < nt; ++t)
                pthread_create(&tid[t], NULL, gemm_rows, &jobs[t]);
            for (t = 0; t < nt; ++t)
                pthread_join(tid[t], NULL);
        }
    }
    free(Ad); free(Bd); free(tid); free(jobs);
    return 0;
}

/*
 * Sampled oracle: the same definition evaluated only at the listed output
 * positions (bat[s], row[s], col[s]), each a full-K dot product in k order.
 * Used at sizes where the full product would take too long on the host.
 */
int oracle_gemm_sampled(int dtype, int64_t M, int64_t N, int64_t K,
                        const void *A, int64_t sA, const void *B, int64_t sB,
                        int64_t nsamp, const int64_t *bat, const int64_t *row,
                        const int64_t *col, double *ref, double *mag)
{
    int64_t s, k;
    if (M < 0 || N < 0 || K < 0 || nsamp < 0 || dtype < 0 || dtype > 2)
        return -1;
    size_t es = elem_size(dtype);
    for (s = 0; s < nsamp; ++s) {
        if (row[s] < 0 || row[s] >= M || col[s] < 0 || col[s] >= N || bat[s] < 0)
            return -1;
        const char *Ab = (const char *)A + (size_t)(bat[s] * sA) * es;
        const char *Bb = (const char *)B + (size_t)(bat[s] * sB) * es;
        double acc = 0.0, m = 0.0;
        for (k = 0; k < K; ++k) {
            double a, bv;
            oracle_decode(dtype, Ab + (size_t)(row[s] * K + k) * es, &a, 1);
            oracle_decode(dtype, Bb + (size_t)(k * N + col[s]) * es, &bv, 1);
            acc += a * bv;
            m += fabs(a) * fabs(bv);
        }
        ref[s] = acc;
        if (mag)
            mag[s] = m;
    }
    return 0;
}

/*
 * The same sampled values with the samples shared over `threads` threads.
 * Each sample's sum is exactly the one above (k ascending, the same decoded
 * products); a thread only keeps the decoded column of B of its previous
 * sample when the next one reads the same (batch, column), so callers that
 * list samples grouped by column read each strided column once.
 */
typedef struct {
    int dtype;
    int64_t M, N, K, sA, sB, s0, s1;
    const char *A, *B;
    const int64_t *bat, *row, *col;
    double *ref, *mag;
    int bad;
} samp_job;

static void *samp_rows(void *arg)
{
    samp_job *j = (samp_job *)arg;
    size_t es = elem_size(j->dtype);
    double *bcol = (double *)malloc(sizeof(double) * (size_t)(j->K > 0 ? j->K : 1));
    int64_t cur_b = -1, cur_c = -1, s, k;
    if (!bcol) {
        j->bad = 1;
        return NULL;
    }
    for (s = j->s0; s < j->s1; ++s) {
        if (j->row[s] < 0 || j->row[s] >= j->M || j->col[s] < 0 || j->col[s] >= j->N || j->bat[s] < 0) {
            j->bad = 1;
            break;
        }
        if (j->bat[s] != cur_b || j->col[s] != cur_c) {
            const char *Bb = j->B + (size_t)(j->bat[s] * j->sB) * es;
            for (k = 0; k < j->K; ++k)
                oracle_decode(j->dtype, Bb + (size_t)(k * j->N + j->col[s]) * es, &bcol[k], 1);
            cur_b = j->bat[s];
            cur_c = j->col[s];
        }
        const char *Ar = j->A + (size_t)(j->bat[s] * j->sA + j->row[s] * j->K) * es;
        double acc = 0.0, m = 0.0;
        for (k = 0; k < j->K; ++k) {
            double a;
            oracle_decode(j->dtype, Ar + (size_t)k * es, &a, 1);
            acc += a * bcol[k];
            m += fabs(a) * fabs(bcol[k]);
        }
        j->ref[s] = acc;
        if (j->mag)
            j->mag[s] = m;
    }
    free(bcol);
    return NULL;
}

int oracle_gemm_sampled_mt(int dtype, int64_t M, int64_t N, int64_t K,
                           const void *A, int64_t sA, const void *B, int64_t sB,
                           int64_t nsamp, const int64_t *bat, const int64_t *row,
                           const int64_t *col, double *ref, double *mag, int threads)
{
    if (M < 0 || N < 0 || K < 0 || nsamp < 0 || dtype < 0 || dtype > 2)
        return -1;
    if (threads < 1)
        threads = 1;
    if (threads > nsamp)
        threads = nsamp > 0 ? (int)nsamp : 1;
    pthread_t *tid = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)threads);
    samp_job *jobs = (samp_job *)malloc(sizeof(samp_job) * (size_t)threads);
    if (!tid || !jobs) {
        free(tid);
        free(jobs);
        return -2;
    }
    int t, bad = 0;
    for (t = 0; t < threads; ++t) {
        samp_job j = {dtype, M, N, K, sA, sB, nsamp * t / threads, nsamp * (t + 1) / threads,
                      (const char *)A, (const char *)B, bat, row, col, ref, mag, 0};
        jobs[t] = j;
    }
    /* a thread that cannot be started leaves its samples to the caller's thread */
    char *run = (char *)calloc((size_t)threads, 1);
    for (t = 1; t < threads; ++t)
        run[t] = run != NULL && pthread_create(&tid[t], NULL, samp_rows, &jobs[t]) == 0;
    samp_rows(&jobs[0]);
    for (t = 1; t < threads; ++t) {
        if (run && run[t])
            pthread_join(tid[t], NULL);
        else
            samp_rows(&jobs[t]);
    }
    for (t = 0; t < threads; ++t)
        if (jobs[t].bad)
            bad = -1;
    free(run);
    free(tid);
    free(jobs);
    return bad;
}

/* ---- the 2-D convolution ------------------------------------------------ */

/*
 * Direct 2-D convolution (the paper's second operator, Section 7.1,
 * benchmarked in Table 4), as deep-learning layers compute it: a
 * cross-correlation with zero padding, stride and dilation.
 *
 *   out[n][oh][ow][co] = sum_{kh, kw, ci} x[n][ih][iw][ci] * w[kh][kw][ci][co],
 *   ih = oh*sh - ph + kh*dh,  iw = ow*sw - pw + kw*dw,
 *
 * where taps with (ih, iw) outside the H x W image are absent (zero padding),
 * OH = floor((H + 2*ph - dh*(KH-1) - 1) / sh) + 1 (likewise OW; 0 when the
 * numerator is negative).  Layouts: x is N x H x W x Cin, w is KH x KW x Cin
 * x Cout, out is N x OH x OW x Cout, all dense.  Binary64, summation over kh,
 * then kw, then ci ascending; Mag sums the absolute products.
 */
typedef struct {
    const double *x, *w;
    double *out, *mag;
    int64_t H, W, Cin, Cout, KH, KW, sh, sw, ph, pw, dh, dw, OH, OW;
    int64_t r0, r1;              /* output rows (n*OH + oh) handled by this thread */
} conv_job;

static void *conv_rows(void *arg)
{
    conv_job *j = (conv_job *)arg;
    int64_t row, ow, kh, kw, ci, co;
    for (row = j->r0; row < j->r1; ++row) {
        int64_t n = row / j->OH, oh = row % j->OH;
        for (ow = 0; ow < j->OW; ++ow) {
            double *o = j->out + (row * j->OW + ow) * j->Cout;
            double *m = j->mag ? j->mag + (row * j->OW + ow) * j->Cout : NULL;
            for (co = 0; co < j->Cout; ++co) {
                o[co] = 0.0;
                if (m)
                    m[co] = 0.0;
            }
            for (kh = 0; kh < j->KH; ++kh) {
                int64_t ih = oh * j->sh - j->ph + kh * j->dh;
                if (ih < 0 || ih >= j->H)
                    continue;
                for (kw = 0; kw < j->KW; ++kw) {
                    int64_t iw = ow * j->sw - j->pw + kw * j->dw;
                    if (iw < 0 || iw >= j->W)
                        continue;
                    const double *xp = j->x + ((n * j->H + ih) * j->W + iw) * j->Cin;
                    for (ci = 0; ci < j->Cin; ++ci) {
                        double a = xp[ci];
                        const double *wp = j->w + ((kh * j->KW + kw) * j->Cin + ci) * j->Cout;
                        for (co = 0; co < j->Cout; ++co)
                            o[co] += a * wp[co];
                        if (m) {
                            double aa = fabs(a);
                            for (co = 0; co < j->Cout; ++co)
                                m[co] += aa * fabs(wp[co]);
                        }
                    }
                }
            }
        }
    }
    return NULL;
}

int64_t oracle_conv_out_dim(int64_t in, int64_t k, int64_t stride, int64_t pad, int64_t dil)
{
    int64_t span = in + 2 * pad - dil * (k - 1) - 1;
    return span < 0 ? 0 : span / stride + 1;
}

int oracle_conv2d(int dtype, int64_t N, int64_t H, int64_t W, int64_t Cin, int64_t Cout, int64_t KH,
                  int64_t KW, int64_t sh, int64_t sw, int64_t ph, int64_t pw, int64_t dh, int64_t dw,
                  const void *x, const void *w, double *out, double *mag, int threads)
{
    if (dtype < 0 || dtype > 2 || N < 0 || H < 0 || W < 0 || Cin < 0 || Cout < 0 || KH < 1 || KW < 1 ||
        sh < 1 || sw < 1 || ph < 0 || pw < 0 || dh < 1 || dw < 1)
        return -1;
    int64_t OH = oracle_conv_out_dim(H, KH, sh, ph, dh), OW = oracle_conv_out_dim(W, KW, sw, pw, dw);
    if (N == 0 || OH == 0 || OW == 0 || Cout == 0)
        return 0;
    if (threads < 1)
        threads = 1;
    int64_t nx = N * H * W * Cin, nw = KH * KW * Cin * Cout;
    double *xd = (double *)malloc(sizeof(double) * (size_t)(nx > 0 ? nx : 1));
    double *wd = (double *)malloc(sizeof(double) * (size_t)(nw > 0 ? nw : 1));
    pthread_t *tid = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)threads);
    conv_job *jobs = (conv_job *)malloc(sizeof(conv_job) * (size_t)threads);
    if (!xd || !wd || !tid || !jobs) {
        free(xd); free(wd); free(tid); free(jobs);
        return -1;
    }
    oracle_decode(dtype, x, xd, nx);
    oracle_decode(dtype, w, wd, nw);
    int64_t rows = N * OH;
    int t, nt = threads;
    if (nt > rows)
        nt = (int)rows;
    for (t = 0; t < nt; ++t) {
        conv_job *j = &jobs[t];
        j->x = xd; j->w = wd; j->out = out; j->mag = mag;
        j->H = H; j->W = W; j->Cin = Cin; j->Cout = Cout; j->KH = KH; j->KW = KW;
        j->sh = sh; j->sw = sw; j->ph = ph; j->pw = pw; j->dh = dh; j->dw = dw; j->OH = OH; j->OW = OW;
        j->r0 = rows * t / nt;
        j->r1 = rows * (t + 1) / nt;
    }
    if (nt == 1) {
        conv_rows(&jobs[0]);
    } else {
        for (t = 0; t < nt; ++t)
            pthread_create(&tid[t], NULL, conv_rows, &jobs[t]);
        for (t = 0; t < nt; ++t)
            pthread_join(tid[t], NULL);
    }
    free(xd); free(wd); free(tid); free(jobs);
    return 0;
}
