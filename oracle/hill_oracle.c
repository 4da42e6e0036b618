/*
 * hill_oracle.c -- plain, slow, obviously-correct CPU oracle for one decode
 * step of HillInfer's token-importance path (arxiv 2602.18750).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file: only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark use it.  It shares no code, header, table or constant
 * with the GPU library.
 *
 * Every quantity is computed in double precision from exactly widened
 * fp16/bf16 inputs, in the order the paper's definitions state it:
 *
 *   (1) logits       l[b,h,j] = sum_i q[b,h,i] * K[b,kv(h),j,i]
 *                    (Sec. 4.4 "Algorithmic Simplification": the raw inner
 *                    product Q.K^T; Sec. 2.1 Eq. 1 for the product itself)
 *   (2) weights      ATTN: w = softmax_j(scale * l)   (Sec. 2.1 Eq. 1, the
 *                    attention weights whose column sum is the importance,
 *                    Sec. 4.1 "System Workflow")
 *                    RAW:  w = l                      (Sec. 4.4: softmax and
 *                    the 1/sqrt(d) division dropped)
 *   (3) cumulative   S[b,r,j] += sum_{h in heads(r)} w[b,h,j]
 *                    (Sec. 4.1: importance = column-wise sum of attention
 *                    weights, carried over decode steps as in H2O)
 *   (4) selection    the k largest S per row, ties to the lower token index,
 *                    emitted in ascending token order (Sec. 3.1 "top-alpha
 *                    percent"; Sec. 4.2 HIE "global top-alpha indices")
 *   (5) attention    Eq. 1 restricted to the selected set I, softmax
 *                    renormalised over I (Sec. 4.1 workflow step 6)
 *
 *   (6) asymmetric   scoring-only low-precision casts of the keys (int8 or
 *       precision    int4) and the query (int8) (Sec. 4.4 "Streaming
 *                    Execution and Asymmetric Precision": Q.K^T in INT8/INT4
 *                    for the evaluation only; attention keeps the 16-bit K,
 *                    V).  Readings where the paper is silent: one
 *                    power-of-two scale 2^e per key row (sequence, KV head,
 *                    token) and per query head, the smallest e with
 *                    max|x| * 2^-e <= qmax (127 for int8, 7 for int4); codes
 *                    rounded to nearest, ties to even, clamped to
 *                    [-qmax, qmax]; e clamped to [-128, 127] (an all-zero row
 *                    has e = -128); the score is the exact integer dot
 *                    product times 2^(e_q + e_k).
 *
 * kv(h) = floor(h / G) with G = Hq / Hkv (contiguous GQA groups).
 * Row granularity: token mode (gran 0) has one row per batch element summing
 * all Hq heads; KV-head mode (gran 1) has one row per (batch, KV head) summing
 * that head's G query heads.
 *
 * Layouts (all contiguous, row-major):
 *   q   [B, Hq, D]        16-bit patterns (fp16 or bf16)
 *   K,V [B, Hkv, n, D]    16-bit patterns
 *   l   [B, Hq, n]        double
 *   S   [B, R, n]         double, R = 1 (token) or Hkv (KV-head)
 *   idx [B, R, k]         int32, ascending
 *   out [B, Hq, D]        double
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <time.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { HOR_F16 = 0, HOR_BF16 = 1 };
enum { HOR_ATTN = 0, HOR_RAW = 1 };
enum { HOR_TOKEN = 0, HOR_KVHEAD = 1 };

/* ---- 16-bit float decoding, from the IEEE-754 binary16 and bfloat16 bit
 * layouts (sign | exponent | fraction), written arithmetically. ---- */

double hor_decode_f16(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int m = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)m, -24);                 /* subnormal: m * 2^-24 */
    else if (e == 31)
        v = m ? NAN : INFINITY;
    else
        v = ldexp((double)(m + 1024), e - 25);     /* 1.m * 2^(e-15) */
    return sign ? -v : v;
}

double hor_decode_bf16(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 7) & 0xff;
    int m = h & 0x7f;
    double v;
    if (e == 0)
        v = ldexp((double)m, -133);                /* subnormal: m * 2^-133 */
    else if (e == 255)
        v = m ? NAN : INFINITY;
    else
        v = ldexp((double)(m + 128), e - 134);     /* 1.m * 2^(e-127) */
    return sign ? -v : v;
}

void hor_decode16(const uint16_t *src, int64_t count, int dtype, double *dst)
{
    for (int64_t i = 0; i < count; ++i)
        dst[i] = dtype == HOR_BF16 ? hor_decode_bf16(src[i]) : hor_decode_f16(src[i]);
}

/* Decoding table for one dtype: every one of the 65536 patterns, filled by
 * the decoders above.  Only a speed aid for the large loops below. */
static void build_table(int dtype, double *tab)
{
    for (int p = 0; p < 65536; ++p)
        tab[p] = dtype == HOR_BF16 ? hor_decode_bf16((uint16_t)p) : hor_decode_f16((uint16_t)p);
}

int hor_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

static int check_shape(int B, int Hq, int Hkv, int D, int n)
{
    if (B < 1 || Hq < 1 || Hkv < 1 || D < 1 || n < 1) return -1;
    if (Hq % Hkv) return -1;
    return 0;
}

/* (1) logits l[b,h,j] = sum_{i<D} q[b,h,i] * K[b,kv(h),j,i], summed in i order. */
int hor_logits(int B, int Hq, int Hkv, int D, int n, int dtype,
               const uint16_t *q, const uint16_t *k, double *l)
{
    if (check_shape(B, Hq, Hkv, D, n)) return -1;
    double *tab = (double *)malloc(65536 * sizeof(double));
    if (!tab) return -2;
    build_table(dtype, tab);
    const int G = Hq / Hkv;
    const int64_t rows = (int64_t)B * Hq;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int64_t bh = 0; bh < rows; ++bh) {
        for (int j = 0; j < n; ++j) {
            int64_t b = bh / Hq;
            int h = (int)(bh % Hq);
            int g = h / G;
            const uint16_t *qr = q + bh * D;
            const uint16_t *kr = k + (((int64_t)b * Hkv + g) * n + j) * D;
            double acc = 0.0;
            for (int i = 0; i < D; ++i)
                acc += tab[qr[i]] * tab[kr[i]];
            l[bh * n + j] = acc;
        }
    }
    free(tab);
    return 0;
}

/* (6) sketch of `rows` rows of D 16-bit values with codes in [-qmax, qmax]
 * (qmax = 127: int8, 7: int4): codes[r, i] and one exponent per row, by the
 * rule in the header.  Every operation is exact (scaling by a power of two,
 * round-to-nearest-even of a value <= qmax). */
int hor_sketch(int64_t rows, int D, int dtype, int qmax, const uint16_t *x, int8_t *codes, int8_t *exps)
{
    if (rows < 0 || D < 1 || (qmax != 127 && qmax != 7)) return -1;
    const int lg = qmax == 127 ? 7 : 3;   /* qmax + 1 = 2^lg */
    double *tab = (double *)malloc(65536 * sizeof(double));
    if (!tab) return -2;
    build_table(dtype, tab);
    #pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) {
        const uint16_t *xr = x + r * D;
        double amax = 0.0;
        for (int i = 0; i < D; ++i) {
            const double a = fabs(tab[xr[i]]);
            if (a > amax) amax = a;
        }
        int e = -128;
        if (amax > 0.0) {
            int E;
            const double m = frexp(amax, &E);       /* amax = m * 2^E, m in [0.5, 1) */
            /* smallest e with amax * 2^-e <= qmax: m * 2^(E-e) <= qmax */
            e = ldexp(m, lg) <= (double)qmax ? E - lg : E - lg + 1;
            if (e < -128) e = -128;
            if (e > 127) e = 127;
        }
        exps[r] = (int8_t)e;
        for (int i = 0; i < D; ++i) {
            double c = nearbyint(ldexp(tab[xr[i]], -e));   /* default rounding: to nearest, ties to even */
            if (c > qmax) c = qmax;
            if (c < -qmax) c = -qmax;
            codes[r * D + i] = (int8_t)c;
        }
    }
    free(tab);
    return 0;
}

/* (6) sketch logits l[b,h,j] = (sum_i q8[b,h,i] * k8[b,kv(h),j,i]) * 2^(eq[b,h] + ek[b,kv(h),j]):
 * the integer dot product is exact (int64), the scaling exact in double. */
int hor_logits_i8(int B, int Hq, int Hkv, int D, int n, const int8_t *q8, const int8_t *eq,
                  const int8_t *k8, const int8_t *ek, double *l)
{
    if (check_shape(B, Hq, Hkv, D, n)) return -1;
    const int G = Hq / Hkv;
    const int64_t rows = (int64_t)B * Hq;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int64_t bh = 0; bh < rows; ++bh) {
        for (int j = 0; j < n; ++j) {
            int64_t b = bh / Hq;
            int h = (int)(bh % Hq);
            int64_t krow = ((int64_t)b * Hkv + h / G) * n + j;
            int64_t acc = 0;
            for (int i = 0; i < D; ++i) acc += (int64_t)q8[bh * D + i] * (int64_t)k8[krow * D + i];
            l[bh * n + j] = ldexp((double)acc, (int)eq[bh] + (int)ek[krow]);
        }
    }
    return 0;
}

/* (2)+(3) per-step weights and cumulative update of S.
 * ATTN: z = scale*l; w[h,j] = exp(z[h,j] - max_j z[h,.]) / sum_j exp(z[h,j] - max).
 * RAW:  w[h,j] = l[h,j].
 * S[b,r,j] = S[b,r,j] + sum_{h in heads(r)} w[b,h,j], heads in increasing h. */
int hor_update(int B, int Hq, int Hkv, int n, int mode, int gran, double scale,
               const double *l, double *S)
{
    if (check_shape(B, Hq, Hkv, 1, n)) return -1;
    if (mode != HOR_ATTN && mode != HOR_RAW) return -1;
    if (gran != HOR_TOKEN && gran != HOR_KVHEAD) return -1;
    const int G = Hq / Hkv;
    const int R = gran == HOR_TOKEN ? 1 : Hkv;
    const int64_t rows = (int64_t)B * Hq;
    double *w = (double *)malloc((size_t)rows * n * sizeof(double));
    if (!w) return -2;

    #pragma omp parallel for schedule(static)
    for (int64_t bh = 0; bh < rows; ++bh) {
        const double *lr = l + bh * n;
        double *wr = w + bh * n;
        if (mode == HOR_RAW) {
            for (int j = 0; j < n; ++j) wr[j] = lr[j];
            continue;
        }
        double m = -INFINITY;
        for (int j = 0; j < n; ++j)
            if (scale * lr[j] > m) m = scale * lr[j];
        double Z = 0.0;
        for (int j = 0; j < n; ++j) Z += exp(scale * lr[j] - m);
        for (int j = 0; j < n; ++j) wr[j] = exp(scale * lr[j] - m) / Z;
    }

    #pragma omp parallel for collapse(2) schedule(static)
    for (int64_t br = 0; br < (int64_t)B * R; ++br) {
        for (int j = 0; j < n; ++j) {
            int64_t b = br / R;
            int r = (int)(br % R);
            int h0 = gran == HOR_TOKEN ? 0 : r * G;
            int h1 = gran == HOR_TOKEN ? Hq : (r + 1) * G;
            double col = 0.0;
            for (int h = h0; h < h1; ++h)
                col += w[(b * Hq + h) * n + j];
            S[br * n + j] += col;
        }
    }
    free(w);
    return 0;
}

/* (4) top-k.  Brute force: sort every token of the row by (S descending,
 * token index ascending), NaN below everything, keep the first k, emit them
 * in ascending token order.  -0.0 and +0.0 compare equal, so they tie. */
typedef struct { double s; int32_t j; } scored_t;

static int rank_cmp(const void *pa, const void *pb)
{
    const scored_t *a = (const scored_t *)pa, *b = (const scored_t *)pb;
    int na = isnan(a->s), nb = isnan(b->s);
    if (na != nb) return na ? 1 : -1;              /* NaN ranks last */
    if (!na) {
        if (a->s > b->s) return -1;
        if (a->s < b->s) return 1;
    }
    return a->j < b->j ? -1 : (a->j > b->j ? 1 : 0);
}

static int int_cmp(const void *pa, const void *pb)
{
    int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    return a < b ? -1 : (a > b ? 1 : 0);
}

int hor_topk(int64_t rows, int n, int k, const double *S, int32_t *idx)
{
    if (rows < 1 || n < 1 || k < 1 || k > n) return -1;
    int err = 0;
    #pragma omp parallel for schedule(dynamic)
    for (int64_t r = 0; r < rows; ++r) {
        scored_t *tmp = (scored_t *)malloc((size_t)n * sizeof(scored_t));
        if (!tmp) { err = -2; continue; }
        for (int j = 0; j < n; ++j) { tmp[j].s = S[r * n + j]; tmp[j].j = j; }
        qsort(tmp, (size_t)n, sizeof(scored_t), rank_cmp);
        int32_t *out = idx + r * k;
        for (int t = 0; t < k; ++t) out[t] = tmp[t].j;
        qsort(out, (size_t)k, sizeof(int32_t), int_cmp);
        free(tmp);
    }
    return err;
}

/* (5) sparse attention over the selected set: for query head h of batch b,
 * with I the index row of r(h) (0 in token mode, kv(h) in KV-head mode):
 *   x_j = scale * q.K_j,  p_j = exp(x_j - max_{I} x),
 *   out = sum_{j in I} p_j V_j / sum_{j in I} p_j. */
int hor_sparse_attn(int B, int Hq, int Hkv, int D, int n, int dtype, int gran,
                    double scale, const uint16_t *q, const uint16_t *k,
                    const uint16_t *v, int kk, const int32_t *idx, double *out)
{
    if (check_shape(B, Hq, Hkv, D, n)) return -1;
    if (kk < 1 || kk > n) return -1;
    if (gran != HOR_TOKEN && gran != HOR_KVHEAD) return -1;
    const int G = Hq / Hkv;
    const int R = gran == HOR_TOKEN ? 1 : Hkv;
    double *tab = (double *)malloc(65536 * sizeof(double));
    if (!tab) return -2;
    build_table(dtype, tab);
    int err = 0;
    #pragma omp parallel for schedule(dynamic)
    for (int64_t bh = 0; bh < (int64_t)B * Hq; ++bh) {
        int64_t b = bh / Hq;
        int h = (int)(bh % Hq);
        int g = h / G;
        int r = gran == HOR_TOKEN ? 0 : g;
        const int32_t *I = idx + (b * R + r) * kk;
        const uint16_t *qr = q + bh * D;
        double *x = (double *)malloc((size_t)kk * sizeof(double));
        double *o = out + bh * D;
        if (!x) { err = -2; continue; }
        for (int t = 0; t < kk; ++t) {
            int j = I[t];
            if (j < 0 || j >= n) { err = -1; x[t] = 0.0; continue; }
            const uint16_t *kr = k + (((int64_t)b * Hkv + g) * n + j) * D;
            double acc = 0.0;
            for (int i = 0; i < D; ++i) acc += tab[qr[i]] * tab[kr[i]];
            x[t] = scale * acc;
        }
        double m = -INFINITY;
        for (int t = 0; t < kk; ++t) if (x[t] > m) m = x[t];
        double den = 0.0;
        for (int i = 0; i < D; ++i) o[i] = 0.0;
        for (int t = 0; t < kk; ++t) {
            int j = I[t];
            if (j < 0 || j >= n) continue;
            double p = exp(x[t] - m);
            den += p;
            const uint16_t *vr = v + (((int64_t)b * Hkv + g) * n + j) * D;
            for (int i = 0; i < D; ++i) o[i] += p * tab[vr[i]];
        }
        for (int i = 0; i < D; ++i) o[i] /= den;
        free(x);
    }
    free(tab);
    return err;
}

static double now_s(void)
{
    struct timespec ts;
    clock_gettime(CLOCK_MONOTONIC, &ts);
    return (double)ts.tv_sec + 1e-9 * (double)ts.tv_nsec;
}

/* One decode step in the paper's order (Sec. 4.1 workflow, steps 5-6):
 * score all tokens with the current query and update S, select on the
 * updated S, then attend over the selection.  `l` is caller scratch of
 * B*Hq*n doubles.  t_phase (nullable) receives seconds spent in
 * {score+update, select, attention}. */
int hor_step(int B, int Hq, int Hkv, int D, int n, int dtype, int mode, int gran,
             double scale, const uint16_t *q, const uint16_t *k, const uint16_t *v,
             double *S, double *l, int kk, int32_t *idx, double *out, double *t_phase)
{
    double t0 = now_s();
    int rc = hor_logits(B, Hq, Hkv, D, n, dtype, q, k, l);
    if (rc) return rc;
    rc = hor_update(B, Hq, Hkv, n, mode, gran, scale, l, S);
    if (rc) return rc;
    double t1 = now_s();
    const int R = gran == HOR_TOKEN ? 1 : Hkv;
    rc = hor_topk((int64_t)B * R, n, kk, S, idx);
    if (rc) return rc;
    double t2 = now_s();
    rc = hor_sparse_attn(B, Hq, Hkv, D, n, dtype, gran, scale, q, k, v, kk, idx, out);
    double t3 = now_s();
    if (t_phase) { t_phase[0] = t1 - t0; t_phase[1] = t2 - t1; t_phase[2] = t3 - t2; }
    return rc;
}
