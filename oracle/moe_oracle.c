/*
 * moe_oracle.c -- plain fp64 CPU oracle of one routed-expert MoE layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline leg do.  It shares no code with the HIP library.
 *
 * What it computes (one layer, per token t):
 *   1. router logits  l_e = sum_i x[t,i] * Wr[e,i] + b[e]            (fp64)
 *   2. selection S_t  = first K experts ordered by (l_e desc, e asc)
 *   3. gate weights   w_e = exp(l_e - m) / sum_{j in S_t} exp(l_j - m),
 *                     m = max_{e in S_t} l_e  (softmax restricted to S_t,
 *                     equal to a full softmax renormalised over S_t)
 *   4. expert FFN     y = Wd (silu(Wg x) * (Wu x)),  silu(z) = z/(1+e^-z)
 *   5. combine        out_t = y_shared + sum_{e in S_t, ascending e} w_e y_e
 *   6. layer stack    h_0 = the stack's input; layer l reads
 *                     x_l = bf16(h_l / rms(h_l)), rms(h) = sqrt(mean_i h_i^2
 *                     + 1e-6) per row, and h_{l+1} = h_l + out_l(x_l)
 *                     (attention omitted; an unweighted RMS normalisation of
 *                     each layer's input, as a transformer block applies)
 * plus the token-by-expert permutation (a stable counting sort of the T*K
 * assignments by (expert, token)).
 *
 * The paper runs the stock router and the complete gate, up and down
 * projections of every selected expert (the principal experiment, "Output-
 * Exact Execution Beyond the Full-Residency Envelope", over a 48-layer
 * model); it does not print the MoE formulas.  Steps 1-5 are the standard
 * softmax/top-k gated-SiLU MoE with an always-on shared expert; the readings
 * taken where the paper is silent (softmax then renormalise, ungated shared
 * expert, bias added before selection, lower id wins ties, fp32/bf16/int4
 * storage upcast exactly, the stack's input normalisation) are listed in the
 * design notes.
 *
 * Inputs are read in their stored formats and upcast exactly to double:
 *   dtype 0 f32, 1 bf16 (uint16 = top half of binary32), 2 q4b32 (nibbles
 *   [rows, cols/2], low nibble = even column, 4-bit two's complement, then
 *   fp16 scales [rows, cols/32]; value = scale * q), 3 k4 and 4 k6 (the
 *   256-element super-block formats of 4.5 and 6.5625 bits per weight,
 *   decoded in wmat_at below); an expert object of dtype 3 (kq) holds Wg and
 *   Wu in k4 and Wd in k6.
 * An expert object is [Wg (I x d) | Wu (I x d) | Wd (d x I)], row-major.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#ifndef MSIO_MUTANT
#define MSIO_MUTANT 0 /* tests plant single mistakes with -DMSIO_MUTANT=n */
#endif

/* matrix formats; an expert object of format KQ holds Wg, Wu in K4 and Wd in K6 */
enum { MSIO_F32 = 0, MSIO_BF16 = 1, MSIO_Q4B32 = 2, MSIO_K4 = 3, MSIO_K6 = 4 };
#define MSIO_KQ MSIO_K4

/* ---- exact upcasts of the stored formats ------------------------------- */

double msio_bf16_to_f64(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

double msio_fp16_to_f64(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int ex = (h >> 10) & 0x1F;
    int man = h & 0x3FF;
    double v;
    if (ex == 0)
        v = ldexp((double)man, -24);                 /* zero / subnormal */
    else if (ex == 31)
        v = man ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + man), ex - 25);     /* (1.man) * 2^(ex-15) */
    return sign ? -v : v;
}

/* round-to-nearest-even double -> bf16 (used only by the layer stack) */
uint16_t msio_f64_to_bf16(double v)
{
    if (v != v)
        return 0x7FC0;
    int sign = signbit(v) ? 1 : 0;
    double a = fabs(v);
    uint16_t s = (uint16_t)(sign << 15);
    if (a == 0.0)
        return s;
    if (a >= ldexp(255.0 / 128.0 + 1.0 / 256.0, 127))   /* rounds past max */
        return s | 0x7F80;
    int e;
    frexp(a, &e);                     /* a = f * 2^e, f in [0.5, 1) */
    int ex = e - 1;                   /* a = 1.m * 2^ex               */
    if (ex < -126)
        ex = -126;                    /* subnormal range: fixed quantum */
    double q = ldexp(1.0, ex - 7);    /* spacing of bf16 values here   */
    double n = a / q;                 /* exact: power-of-two scaling   */
    double fl = floor(n);
    double r = n - fl;
    if (r > 0.5 || (r == 0.5 && fmod(fl, 2.0) != 0.0))
        fl += 1.0;
    double rv = fl * q;
    float f = (float)rv;              /* exactly representable */
    uint32_t u;
    memcpy(&u, &f, 4);
    return s | (uint16_t)(u >> 16);
}

size_t msio_matrix_nbytes(int dtype, int64_t rows, int64_t cols)
{
    switch (dtype) {
    case MSIO_F32: return (size_t)(rows * cols * 4);
    case MSIO_BF16: return (size_t)(rows * cols * 2);
    case MSIO_K4: return (size_t)(rows * cols / 2 + rows * (cols / 256) * 16);
    case MSIO_K6: return (size_t)(rows * cols / 2 + rows * cols / 4 + rows * cols / 16 + rows * (cols / 256) * 2);
    default: return (size_t)(rows * cols / 2 + rows * (cols / 32) * 2);
    }
}

static double fp16_at(const uint8_t *p)
{
    uint16_t h;
    memcpy(&h, p, 2);
    return msio_fp16_to_f64(h);
}

/* 6-bit field j of a 48-bit little-endian group of 6 bytes */
static int six_bits(const uint8_t *p, int j)
{
    uint64_t w = 0;
    for (int b = 5; b >= 0; --b)
        w = (w << 8) | p[b];
    return (int)((w >> (6 * j)) & 63);
}

typedef struct {
    int dtype;
    const uint8_t *base;
    int64_t rows, cols;
} wmat;

static inline double wmat_at(const wmat *m, int64_t r, int64_t c)
{
    switch (m->dtype) {
    case MSIO_F32: {
        float f;
        memcpy(&f, m->base + 4 * (r * m->cols + c), 4);
        return (double)f;
    }
    case MSIO_BF16: {
        uint16_t b;
        memcpy(&b, m->base + 2 * (r * m->cols + c), 2);
        return msio_bf16_to_f64(b);
    }
    case MSIO_K4: {
        /* nibbles [rows, cols/2], then a 16-byte header per (row, 256-element super-block):
         * fp16 d, fp16 dmin, eight 6-bit scales, eight 6-bit mins; value = d sc_j q - dmin m_j */
        const uint8_t byte = m->base[r * (m->cols / 2) + c / 2];
        const int q = (c & 1) ? (byte >> 4) : (byte & 0x0F);
        const uint8_t *h = m->base + (size_t)(m->rows * m->cols / 2) + 16 * (size_t)(r * (m->cols / 256) + c / 256);
        const int j = (int)((c % 256) / 32);
        const double d = fp16_at(h), dmin = fp16_at(h + 2);
#if MSIO_MUTANT == 13
        return d * six_bits(h + 4, j) * q + dmin * six_bits(h + 10, j);     /* min added */
#else
        return d * six_bits(h + 4, j) * q - dmin * six_bits(h + 10, j);
#endif
    }
    case MSIO_K6: {
        /* low nibbles [rows, cols/2], high 2-bit parts [rows, cols/4], int8 scales [rows, cols/16],
         * fp16 d [rows, cols/256]; q = low | high << 4, value = d sc_j (q - 32) */
        const int64_t R = m->rows, C = m->cols;
        const uint8_t byte = m->base[r * (C / 2) + c / 2];
        const int lo = (c & 1) ? (byte >> 4) : (byte & 0x0F);
        const int hi = (m->base[R * C / 2 + r * (C / 4) + c / 4] >> (2 * (c % 4))) & 3;
#if MSIO_MUTANT == 14
        const int q = lo | (hi << 2);                                        /* high bits misplaced */
#else
        const int q = lo | (hi << 4);
#endif
        const int8_t sc = (int8_t)m->base[R * C / 2 + R * C / 4 + r * (C / 16) + c / 16];
        const double d = fp16_at(m->base + R * C / 2 + R * C / 4 + R * C / 16 + 2 * (r * (C / 256) + c / 256));
        return d * sc * (q - 32);
    }
    default: {
        uint8_t byte = m->base[r * (m->cols / 2) + c / 2];
#if MSIO_MUTANT == 8
        int q = (c & 1) ? (byte & 0x0F) : (byte >> 4);   /* nibble order swapped */
#else
        int q = (c & 1) ? (byte >> 4) : (byte & 0x0F);
#endif
        if (q >= 8)
            q -= 16;
        uint16_t s;
        memcpy(&s, m->base + (size_t)(m->rows * m->cols / 2) + 2 * (r * (m->cols / 32) + c / 32), 2);
        return msio_fp16_to_f64(s) * (double)q;
    }
    }
}

/* q4b32 dequantisation of a whole matrix (for pins and the numpy cross-check) */
void msio_dequant(int dtype, int64_t rows, int64_t cols, const void *src, double *dst)
{
    wmat m = {dtype, (const uint8_t *)src, rows, cols};
    for (int64_t r = 0; r < rows; ++r)
        for (int64_t c = 0; c < cols; ++c)
            dst[r * cols + c] = wmat_at(&m, r, c);
}

/* ---- step 1: router logits ---------------------------------------------- */

/* The stored router weight [E, d] upcast once to fp64 (exact); caller frees. */
static double *upcast_router(int64_t d, int64_t E, const wmat *wr)
{
    double *w = (double *)malloc(sizeof(double) * (size_t)(E * d));
    for (int64_t e = 0; e < E; ++e)
        for (int64_t i = 0; i < d; ++i)
            w[e * d + i] = wmat_at(wr, e, i);
    return w;
}

/* l_e = sum_i x_i Wr[e, i] (i ascending) + b_e for one token's upcast row x. */
static void logits_one(int64_t d, int64_t E, const double *x, const double *wr, const float *bias, double *L)
{
    for (int64_t e = 0; e < E; ++e) {
        double acc = 0.0;
        for (int64_t i = 0; i < d; ++i)
            acc += x[i] * wr[e * d + i];
#if MSIO_MUTANT == 1
        (void)bias;                                   /* bias dropped */
#else
        if (bias)
            acc += (double)bias[e];
#endif
        L[e] = acc;
    }
}

void msio_router_logits(int64_t T, int64_t d, int64_t E, int xdtype, const void *x,
                        const void *wr, const float *bias, double *L)
{
    wmat X = {xdtype, (const uint8_t *)x, T, d};
    wmat W = {xdtype, (const uint8_t *)wr, E, d};
    double *w = upcast_router(d, E, &W);
#pragma omp parallel
    {
        double *xt = (double *)malloc(sizeof(double) * (size_t)d);
#pragma omp for schedule(dynamic, 16)
        for (int64_t t = 0; t < T; ++t) {
            for (int64_t i = 0; i < d; ++i)
                xt[i] = wmat_at(&X, t, i);
            logits_one(d, E, xt, w, bias, L + t * E);
        }
        free(xt);
    }
    free(w);
}

/* ---- step 2: top-K selection, ties to the lower expert id ----------------- */

typedef struct {
    double v;
    int32_t id;
} vid;

static int cmp_rank(const void *a, const void *b)
{
    const vid *p = (const vid *)a, *q = (const vid *)b;
    if (p->v > q->v) return -1;
    if (p->v < q->v) return 1;
#if MSIO_MUTANT == 2
    return (p->id < q->id) ? 1 : (p->id > q->id) ? -1 : 0;  /* higher id wins */
#else
    return (p->id < q->id) ? -1 : (p->id > q->id) ? 1 : 0;
#endif
}

static int cmp_i32(const void *a, const void *b)
{
    int32_t p = *(const int32_t *)a, q = *(const int32_t *)b;
    return (p > q) - (p < q);
}

/* idx: K ids of S_t in ascending order.  gap: l_(K) - l_(K+1) (+inf if K == E). */
static void select_one(int64_t E, int64_t K, const double *L, int32_t *idx, double *gap, vid *tmp)
{
    for (int64_t e = 0; e < E; ++e) {
        tmp[e].v = L[e];
        tmp[e].id = (int32_t)e;
    }
    qsort(tmp, (size_t)E, sizeof(vid), cmp_rank);
    for (int64_t k = 0; k < K; ++k)
        idx[k] = tmp[k].id;
    qsort(idx, (size_t)K, sizeof(int32_t), cmp_i32);
    if (gap)
        *gap = (K < E) ? tmp[K - 1].v - tmp[K].v : INFINITY;
}

void msio_select_topk(int64_t T, int64_t E, int64_t K, const double *L, int32_t *idx, double *gap)
{
#pragma omp parallel
    {
        vid *tmp = (vid *)malloc(sizeof(vid) * (size_t)E);
#pragma omp for schedule(static)
        for (int64_t t = 0; t < T; ++t)
            select_one(E, K, L + t * E, idx + t * K, gap ? gap + t : NULL, tmp);
        free(tmp);
    }
}

/* ---- step 3: softmax restricted to the selected set ----------------------- */

static void weights_one(int64_t E, int64_t K, const double *L, const int32_t *idx, double *w)
{
#if MSIO_MUTANT == 3
    /* full softmax over all E, not renormalised over S_t */
    double m = L[0];
    for (int64_t e = 1; e < E; ++e) m = fmax(m, L[e]);
    double s = 0.0;
    for (int64_t e = 0; e < E; ++e) s += exp(L[e] - m);
    for (int64_t k = 0; k < K; ++k) w[k] = exp(L[idx[k]] - m) / s;
#else
    (void)E;
    double m = L[idx[0]];
    for (int64_t k = 1; k < K; ++k)
        m = fmax(m, L[idx[k]]);
    double s = 0.0;
    for (int64_t k = 0; k < K; ++k)
        s += exp(L[idx[k]] - m);
    for (int64_t k = 0; k < K; ++k)
        w[k] = exp(L[idx[k]] - m) / s;
#endif
}

void msio_gate_weights(int64_t T, int64_t E, int64_t K, const double *L, const int32_t *idx, double *w)
{
    for (int64_t t = 0; t < T; ++t)
        weights_one(E, K, L + t * E, idx + t * K, w + t * K);
}

/* ---- token-by-expert permutation: stable counting sort by (expert, token) -- */

void msio_permute(int64_t T, int64_t E, int64_t K, const int32_t *idx, int32_t *counts,
                  int32_t *offsets, int32_t *perm, int32_t *inv)
{
    for (int64_t e = 0; e < E; ++e)
        counts[e] = 0;
    for (int64_t a = 0; a < T * K; ++a)
        counts[idx[a]]++;
    offsets[0] = 0;
    for (int64_t e = 0; e < E; ++e)
        offsets[e + 1] = offsets[e] + counts[e];
    int32_t *cursor = (int32_t *)malloc(sizeof(int32_t) * (size_t)E);
    memcpy(cursor, offsets, sizeof(int32_t) * (size_t)E);
#if MSIO_MUTANT == 9
    for (int64_t t = T - 1; t >= 0; --t)              /* tokens in reverse: unstable */
#else
    for (int64_t t = 0; t < T; ++t)
#endif
        for (int64_t k = 0; k < K; ++k) {
            int32_t e = idx[t * K + k];
            int32_t row = cursor[e]++;
            perm[row] = (int32_t)t;
            inv[t * K + k] = row;
        }
    free(cursor);
}

/* ---- step 4: one expert's gated-SiLU FFN on one token --------------------- */

static inline double silu(double z)
{
#if MSIO_MUTANT == 4
    return z / (1.0 + exp(z));                        /* sign flipped */
#else
    return z / (1.0 + exp(-z));
#endif
}

void msio_expert_ffn(int64_t d, int64_t I, int wdtype, const void *obj, const double *x,
                     double *y, double *act /* [I] scratch, may be NULL */)
{
    const uint8_t *b = (const uint8_t *)obj;
    size_t nb = msio_matrix_nbytes(wdtype, I, d);
    wmat Wg = {wdtype, b, I, d};
    wmat Wu = {wdtype, b + nb, I, d};
    wmat Wd = {wdtype == MSIO_KQ ? MSIO_K6 : wdtype, b + 2 * nb, d, I};
#if MSIO_MUTANT == 5
    Wg.base = Wu.base;                                /* gate reads the up matrix */
#endif
    double *a = act ? act : (double *)malloc(sizeof(double) * (size_t)I);
    for (int64_t i = 0; i < I; ++i) {
        double g = 0.0, u = 0.0;
        for (int64_t k = 0; k < d; ++k) {
            g += wmat_at(&Wg, i, k) * x[k];
            u += wmat_at(&Wu, i, k) * x[k];
        }
        a[i] = silu(g) * u;
    }
    for (int64_t j = 0; j < d; ++j) {
        double acc = 0.0;
        for (int64_t i = 0; i < I; ++i)
            acc += wmat_at(&Wd, j, i) * a[i];
        y[j] = acc;
    }
    if (!act)
        free(a);
}

/* ---- steps 1-5 for a list of tokens --------------------------------------- */
/*
 * tokens:     n_sel token ids to evaluate (NULL = 0..n_sel-1)
 * forced_idx: [n_sel, K] ascending expert sets to use instead of step 2 (or
 *             NULL); weights are then the restricted softmax over that set
 * experts:    E host pointers to expert objects; shared: object or NULL
 * out [n_sel, d]; idx_out [n_sel, K]; w_out [n_sel, K]; gap_out [n_sel];
 * logits_out [n_sel, E] -- each output pointer may be NULL except out.
 */
void msio_moe_layer(int64_t T, int64_t d, int64_t E, int64_t K, int64_t I, int wdtype, int xdtype,
                    const void *x, const void *wr, const float *bias,
                    const void *const *experts, const void *shared,
                    int64_t n_sel, const int64_t *tokens, const int32_t *forced_idx,
                    double *out, int32_t *idx_out, double *w_out, double *gap_out,
                    double *logits_out)
{
    wmat X = {xdtype, (const uint8_t *)x, T, d};
    wmat W = {xdtype, (const uint8_t *)wr, E, d};
    double *wrd = upcast_router(d, E, &W);
#pragma omp parallel
    {
        double *L = (double *)malloc(sizeof(double) * (size_t)E);
        vid *tmp = (vid *)malloc(sizeof(vid) * (size_t)E);
        double *xt = (double *)malloc(sizeof(double) * (size_t)d);
        double *y = (double *)malloc(sizeof(double) * (size_t)d);
        double *act = (double *)malloc(sizeof(double) * (size_t)I);
        int32_t idx[64];
        double w[64];
#pragma omp for schedule(dynamic, 1)
        for (int64_t s = 0; s < n_sel; ++s) {
            int64_t t = tokens ? tokens[s] : s;
            for (int64_t i = 0; i < d; ++i)
                xt[i] = wmat_at(&X, t, i);
            logits_one(d, E, xt, wrd, bias, L);
            double gap = NAN;
            if (forced_idx)
                memcpy(idx, forced_idx + s * K, sizeof(int32_t) * (size_t)K);
            else
                select_one(E, K, L, idx, &gap, tmp);
            weights_one(E, K, L, idx, w);
            double *o = out + s * d;
            for (int64_t j = 0; j < d; ++j)
                o[j] = 0.0;
#if MSIO_MUTANT != 6
            if (shared) {
                msio_expert_ffn(d, I, wdtype, shared, xt, y, act);
                for (int64_t j = 0; j < d; ++j)
                    o[j] += y[j];
            }
#endif
            for (int64_t k = 0; k < K; ++k) {              /* ascending expert id */
                if (!experts[idx[k]]) {                    /* caller omitted this object */
                    for (int64_t j = 0; j < d; ++j)
                        o[j] = NAN;
                    break;
                }
                msio_expert_ffn(d, I, wdtype, experts[idx[k]], xt, y, act);
                for (int64_t j = 0; j < d; ++j)
                    o[j] += w[k] * y[j];
            }
            if (idx_out)
                memcpy(idx_out + s * K, idx, sizeof(int32_t) * (size_t)K);
            if (w_out)
                memcpy(w_out + s * K, w, sizeof(double) * (size_t)K);
            if (gap_out)
                gap_out[s] = gap;
            if (logits_out)
                memcpy(logits_out + s * E, L, sizeof(double) * (size_t)E);
        }
        free(L);
        free(tmp);
        free(xt);
        free(y);
        free(act);
    }
    free(wrd);
}

/* ---- step 6: the residual stream between stacked layers ------------------- */
/*
 * One row-wise step of the stack for `rows` tokens of `cols` features:
 *   h_next = h + out   (out == NULL: h_next = h, the stack's input)
 *   x_next = bf16_rne(h_next / sqrt(mean(h_next^2) + 1e-6))
 * with the mean summed in column order in fp64.  h_next may alias h.
 */
void msio_residual_step(int64_t rows, int64_t cols, const double *h, const double *out, double *h_next,
                        uint16_t *x_next)
{
    for (int64_t r = 0; r < rows; ++r) {
        const double *hr = h + r * cols;
        double *hn = h_next + r * cols;
        double ss = 0.0;
        for (int64_t c = 0; c < cols; ++c) {
#if MSIO_MUTANT == 12
            const double v = out ? out[r * cols + c] : hr[c];   /* residual dropped */
#else
            const double v = out ? hr[c] + out[r * cols + c] : hr[c];
#endif
            hn[c] = v;
            ss += v * v;
        }
#if MSIO_MUTANT == 10
        const double rms = sqrt(ss / (double)cols);              /* epsilon dropped */
#elif MSIO_MUTANT == 11
        const double rms = sqrt(ss + 1e-6);                      /* sum, not mean */
#else
        const double rms = sqrt(ss / (double)cols + 1e-6);
#endif
        for (int64_t c = 0; c < cols; ++c)
            x_next[r * cols + c] = msio_f64_to_bf16(hn[c] / rms);
    }
}

int msio_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

int msio_mutant(void) { return MSIO_MUTANT; }
