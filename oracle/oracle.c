/*
 * CPU oracle for the derived-operator path.  TEST INFRASTRUCTURE ONLY: nothing in
 * the product library links, includes or calls this file; only the tests, the
 * smoke check and the benchmark's CPU-baseline leg load it.
 *
 * Each operator is evaluated as its plain nested-summation definition, one output
 * element at a time, with double accumulation.  There is no blocking, fusion or
 * reordering: the sums run in the order the definitions state (r, then s, then c
 * for convolutions; j for the band).  The derived GEMM + eOperator form that the
 * GPU executes is NOT used here; a second, independent evaluation of that form
 * lives in derived_form.py (NumPy) and is only used to cross-check this file.
 *
 * Conventions (shared only as a written convention with the rest of the project):
 *   X   [n][h][w][c]   input, NHWC
 *   Wt  [r][s][k][c]   weight; k is the output channel (the paper's f)
 *   out [n][ho][wo][k]
 *   Q,K,V [b][l][d], O [b][l][d], S and P [b][l][2w+1]
 * Inputs are float (the exact values the GPU sees, e.g. bf16 values widened to
 * float); outputs are double.
 *
 * Parity status: every function here is pinned by tests under tests/ (library
 * routines in float64, closed forms, brute force and hand-worked examples).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int64_t n, c, h, w;      /* input  X[n][h][w][c]          */
    int64_t k, r, s;         /* weight Wt[r][s][k][c]         */
    int64_t sh, sw;          /* stride                        */
    int64_t ph, pw;          /* zero padding                  */
    int64_t dh, dw;          /* dilation                      */
    int64_t oph, opw;        /* output padding (transposed)   */
} oracle_geom;

int oracle_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Output extent of a convolution along one dimension.
 * Forward (section 4.2 expression E1 with padding, stride and dilation):
 *   the last valid output o satisfies o*stride - pad + dil*(r-1) <= in - 1 + pad,
 *   i.e. out = floor((in + 2*pad - dil*(r-1) - 1) / stride) + 1.
 * Transposed (the adjoint map, section 6.3): every input position i and tap r
 *   lands on o = i*stride - pad + r*dil; out = (in-1)*stride - 2*pad + dil*(r-1)
 *   + out_pad + 1, the extent that covers the largest such o plus out_pad. */
int64_t oracle_conv_out_size(int64_t in, int64_t r, int64_t stride, int64_t pad,
                             int64_t dil, int64_t out_pad, int transposed) {
    if (transposed)
        return (in - 1) * stride - 2 * pad + dil * (r - 1) + out_pad + 1;
    int64_t span = in + 2 * pad - dil * (r - 1) - 1;
    if (span < 0) return 0;
    return span / stride + 1;
}

/* X zero-extended outside [0,h) x [0,w): the padding rule of section 3. */
static inline double x_at(const oracle_geom* g, const float* x, int64_t n, int64_t hi,
                          int64_t wi, int64_t c) {
    if (hi < 0 || hi >= g->h || wi < 0 || wi >= g->w) return 0.0;
    return (double)x[((n * g->h + hi) * g->w + wi) * g->c + c];
}

/* conv2d, one element:
 *   out[n,ho,wo,k] = sum_{r<R} sum_{s<S} sum_{c<C} X0[n, ho*sh - ph + r*dh, wo*sw - pw + s*dw, c]
 *                                                  * Wt[r,s,k,c]
 * This is the convolution expression E1 of section 4.2 (cross-correlation, no kernel
 * flip: the input is indexed at h+r), generalised to stride, padding and dilation. */
static double conv2d_elem(const oracle_geom* g, const float* x, const float* wt,
                          int64_t n, int64_t ho, int64_t wo, int64_t k) {
    double acc = 0.0;
    for (int64_t r = 0; r < g->r; ++r) {
        for (int64_t s = 0; s < g->s; ++s) {
            int64_t hi = ho * g->sh - g->ph + r * g->dh;
            int64_t wi = wo * g->sw - g->pw + s * g->dw;
            for (int64_t c = 0; c < g->c; ++c) {
                double wv = (double)wt[((r * g->s + s) * g->k + k) * g->c + c];
                acc += x_at(g, x, n, hi, wi, c) * wv;
            }
        }
    }
    return acc;
}

/* conv_transpose2d, one element, in gather form.  The transposed convolution sends
 * input pixel (hi,wi) through tap (r,s) to output (hi*sh - ph + r*dh, wi*sw - pw + s*dw):
 *   out[n,ho,wo,k] = sum_{hi,wi,r,s,c} [ho = hi*sh - ph + r*dh][wo = wi*sw - pw + s*dw]
 *                                      X[n,hi,wi,c] * Wt[r,s,k,c]
 * For a fixed output and tap the indicator picks at most one input pixel:
 *   th = ho + ph - r*dh must be >= 0, divisible by sh, and th/sh < h.
 * The sign test comes first so that C's remainder of a negative number never
 * decides validity. */
static double convt_elem(const oracle_geom* g, const float* x, const float* wt,
                         int64_t n, int64_t ho, int64_t wo, int64_t k) {
    double acc = 0.0;
    for (int64_t r = 0; r < g->r; ++r) {
        int64_t th = ho + g->ph - r * g->dh;
        if (th < 0 || th % g->sh != 0 || th / g->sh >= g->h) continue;
        int64_t hi = th / g->sh;
        for (int64_t s = 0; s < g->s; ++s) {
            int64_t tw = wo + g->pw - s * g->dw;
            if (tw < 0 || tw % g->sw != 0 || tw / g->sw >= g->w) continue;
            int64_t wi = tw / g->sw;
            for (int64_t c = 0; c < g->c; ++c) {
                double wv = (double)wt[((r * g->s + s) * g->k + k) * g->c + c];
                acc += (double)x[((n * g->h + hi) * g->w + wi) * g->c + c] * wv;
            }
        }
    }
    return acc;
}

static void out_dims(const oracle_geom* g, int transposed, int64_t* ho, int64_t* wo) {
    *ho = oracle_conv_out_size(g->h, g->r, g->sh, g->ph, g->dh, g->oph, transposed);
    *wo = oracle_conv_out_size(g->w, g->s, g->sw, g->pw, g->dw, g->opw, transposed);
}

/* Evaluate the whole output (idx == NULL) or only the flat output indices idx[0..npts). */
static void conv_eval(const oracle_geom* g, int transposed, const float* x, const float* wt,
                      int64_t npts, const int64_t* idx, double* out) {
    int64_t ho_n, wo_n;
    out_dims(g, transposed, &ho_n, &wo_n);
    int64_t total = g->n * ho_n * wo_n * g->k;
    int64_t count = idx ? npts : total;
    #pragma omp parallel for schedule(dynamic, 64)
    for (int64_t e = 0; e < count; ++e) {
        int64_t f = idx ? idx[e] : e;
        int64_t k = f % g->k;
        int64_t t = f / g->k;
        int64_t wo = t % wo_n;
        t /= wo_n;
        int64_t ho = t % ho_n;
        int64_t n = t / ho_n;
        out[e] = transposed ? convt_elem(g, x, wt, n, ho, wo, k)
                            : conv2d_elem(g, x, wt, n, ho, wo, k);
    }
}

void oracle_conv2d(const oracle_geom* g, const float* x, const float* wt, double* out) {
    conv_eval(g, 0, x, wt, 0, 0, out);
}
void oracle_conv2d_at(const oracle_geom* g, const float* x, const float* wt, int64_t npts,
                      const int64_t* idx, double* vals) {
    conv_eval(g, 0, x, wt, npts, idx, vals);
}
void oracle_conv_transpose2d(const oracle_geom* g, const float* x, const float* wt, double* out) {
    conv_eval(g, 1, x, wt, 0, 0, out);
}
void oracle_conv_transpose2d_at(const oracle_geom* g, const float* x, const float* wt,
                                int64_t npts, const int64_t* idx, double* vals) {
    conv_eval(g, 1, x, wt, npts, idx, vals);
}

/* Banded dilated batched matmul (general-to-band matmul, G2BMM, with the iterator
 * groups of Table 2), then a row softmax and the band-times-dense product:
 *   t(i,j)   = i + (j - w) * dil,                      j in [0, 2w]
 *   S[b,i,j] = scale * sum_d Q[b,i,d] * K0[b,t,d]      K0 = K zero outside [0,l)
 *   P[b,i,:] = softmax over j of S[b,i,:]
 *   O[b,i,e] = sum_j P[b,i,j] * V0[b,t,e]             V0 = V zero outside [0,l)
 * mask == 0 (zero mode): out-of-range entries keep S = 0 and take part in the
 *   softmax, exactly as a zero-padded K would give.
 * mask != 0 (mask mode): out-of-range entries are left out of the softmax (P = 0).
 * The softmax subtracts the row maximum (over the entries that take part) before
 * exponentiating; mathematically this does not change P.
 * rows: flat row ids b*l + i to evaluate (NULL = all rows); s_out/p_out are
 * [nrows][2w+1] and o_out [nrows][d]; s_out and p_out may be NULL. */
void oracle_band(int64_t b, int64_t l, int64_t d, int64_t w, int64_t dil, double scale,
                 int mask, const float* q, const float* kk, const float* v, int64_t nrows,
                 const int64_t* rows, double* s_out, double* p_out, double* o_out) {
    int64_t nb = 2 * w + 1;
    int64_t count = rows ? nrows : b * l;
    #pragma omp parallel
    {
        double* s = (double*)malloc(sizeof(double) * (size_t)nb);
        char* live = (char*)malloc((size_t)nb);
        #pragma omp for schedule(dynamic, 16)
        for (int64_t e = 0; e < count; ++e) {
            int64_t row = rows ? rows[e] : e;
            int64_t bi = row / l, i = row % l;
            const float* qr = q + (bi * l + i) * d;
            for (int64_t j = 0; j < nb; ++j) {
                int64_t t = i + (j - w) * dil;
                int in_range = (t >= 0 && t < l);
                double acc = 0.0;
                if (in_range) {
                    const float* kr = kk + (bi * l + t) * d;
                    for (int64_t x = 0; x < d; ++x) acc += (double)qr[x] * (double)kr[x];
                }
                s[j] = scale * acc;
                live[j] = (char)(in_range || !mask);
            }
            double m = -INFINITY;
            for (int64_t j = 0; j < nb; ++j)
                if (live[j] && s[j] > m) m = s[j];
            double den = 0.0;
            for (int64_t j = 0; j < nb; ++j)
                if (live[j]) den += exp(s[j] - m);
            double* orow = o_out + e * d;
            for (int64_t x = 0; x < d; ++x) orow[x] = 0.0;
            for (int64_t j = 0; j < nb; ++j) {
                double p = live[j] ? exp(s[j] - m) / den : 0.0;
                if (s_out) s_out[e * nb + j] = s[j];
                if (p_out) p_out[e * nb + j] = p;
                int64_t t = i + (j - w) * dil;
                if (t < 0 || t >= l) continue;
                const float* vr = v + (bi * l + t) * d;
                for (int64_t x = 0; x < d; ++x) orow[x] += p * (double)vr[x];
            }
        }
        free(s);
        free(live);
    }
}
