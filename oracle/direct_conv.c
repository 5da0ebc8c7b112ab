/*
 * TEST INFRASTRUCTURE ONLY -- the CPU oracle for the forward 2-D convolution.
 *
 * Only the tests, the smoke check and the CPU-baseline leg of the benchmark
 * may load this library.  The product path (the HIP kernels behind the C ABI)
 * never calls it, shares no code, header, table or helper with it, and this
 * file includes nothing from the product.
 *
 * What it computes: Eq. 1 of the MG3MConv paper (Sec. 2.1), the direct
 * convolution written as seven nested loops,
 *
 *   OUT[b,oc,oh,ow] = sum_{ic} sum_{fh} sum_{fw} IN[b,ic,ih,iw] * FLT[oc,ic,fh,fw]
 *   ih = oh*stdH + fh - padH,   iw = ow*stdW + fw - padW,
 *
 * where taps with (ih,iw) outside the input are skipped (the "if ih,iw exist"
 * test of Alg. 2, Sec. 4.3.1), which is zero padding.  Every matrix-
 * multiplication mapping of the paper (MM_unit, Eq. 2; Alg. 1-3) reaches this
 * same value up to the order of summation, so the oracle is the definition
 * itself.  There is no filter flip: Eq. 1 is a cross-correlation.
 *
 * Precision: inputs are fp32 (the paper's storage type, Sec. 4.1.1); every
 * product and sum is taken in fp64 (the paper's kernels also compute in
 * double, Sec. 4.3).  A product of two fp32 values is exact in fp64.  The
 * result is not rounded back to fp32.  Alongside each output the oracle
 * returns mag = sum |IN*FLT| over the same taps, the scale of the parity
 * tolerance |gpu - acc| <= 1e-5 * mag.
 *
 * Output size (never printed in the paper; the floor formula that matches the
 * loop bounds of Alg. 1 and the skip rule of Alg. 2):
 *   outH = floor((inH + 2*padH - fltH) / stdH) + 1, likewise outW.
 *
 * Layouts (both are the paper's):
 *   layout 0 "HWCN", the storage order of Sec. 4.1.1:
 *       IN[inH][inW][IC][B], FLT[fltH][fltW][IC][OC], OUT[outH][outW][OC][B]
 *   layout 1 "NCHW", the index order of Eq. 1:
 *       IN[B][IC][inH][inW], FLT[OC][IC][fltH][fltW], OUT[B][OC][outH][outW]
 * acc/mag arrays are written in the output order of the chosen layout.
 *
 * Parity pins (tests/test_oracle.py): brute force against a separately
 * written im2col + naive GEMM; torch/scipy library routines; delta-filter
 * shift; linearity; 1x1 == matmul; ones-input and ones-filter closed forms;
 * stride == subsampling; pad == explicit zero padding; channel additivity;
 * batch equivariance; layout equivalence; small-integer exactness.
 */
#include <stdint.h>
#include <math.h>

#define ORACLE_HWCN 0
#define ORACLE_NCHW 1

typedef struct {
    int n, c, h, w, k, r, s;      /* B, IC, inH, inW, OC, fltH, fltW (Table 1) */
    int std_h, std_w, pad_h, pad_w;
    int out_h, out_w;
    int layout;
} oracle_shape;

/* Output size; returns 0 on success, -1 if a dimension is < 1 or the output
 * would be empty. */
int oracle_out_dims(int h, int w, int r, int s, int std_h, int std_w,
                    int pad_h, int pad_w, int *out_h, int *out_w)
{
    if (h < 1 || w < 1 || r < 1 || s < 1 || std_h < 1 || std_w < 1 ||
        pad_h < 0 || pad_w < 0)
        return -1;
    int eh = h + 2 * pad_h - r, ew = w + 2 * pad_w - s;
    if (eh < 0 || ew < 0)
        return -1;
    *out_h = eh / std_h + 1;
    *out_w = ew / std_w + 1;
    return 0;
}

static double in_at(const float *x, const oracle_shape *p, int b, int c, int ih, int iw)
{
    int64_t i;
    if (p->layout == ORACLE_HWCN)
        i = (((int64_t)ih * p->w + iw) * p->c + c) * p->n + b;
    else
        i = (((int64_t)b * p->c + c) * p->h + ih) * p->w + iw;
    return (double)x[i];
}

static double flt_at(const float *wt, const oracle_shape *p, int oc, int c, int fh, int fw)
{
    int64_t i;
    if (p->layout == ORACLE_HWCN)
        i = (((int64_t)fh * p->s + fw) * p->c + c) * p->k + oc;
    else
        i = (((int64_t)oc * p->c + c) * p->r + fh) * p->s + fw;
    return (double)wt[i];
}

static int64_t out_index(const oracle_shape *p, int b, int oc, int oh, int ow)
{
    if (p->layout == ORACLE_HWCN)
        return (((int64_t)oh * p->out_w + ow) * p->k + oc) * p->n + b;
    return (((int64_t)b * p->k + oc) * p->out_h + oh) * p->out_w + ow;
}

/* One output element of Eq. 1, summed in Eq. 1's order (ic, then fh, then fw). */
static void one_output(const float *x, const float *wt, const oracle_shape *p,
                       int b, int oc, int oh, int ow, double *acc_out, double *mag_out)
{
    double acc = 0.0, mag = 0.0;
    for (int ic = 0; ic < p->c; ++ic) {
        for (int fh = 0; fh < p->r; ++fh) {
            for (int fw = 0; fw < p->s; ++fw) {
                int ih = oh * p->std_h + fh - p->pad_h;
                int iw = ow * p->std_w + fw - p->pad_w;
                if (ih < 0 || ih >= p->h || iw < 0 || iw >= p->w)
                    continue;                        /* tap does not exist */
                double prod = in_at(x, p, b, ic, ih, iw) * flt_at(wt, p, oc, ic, fh, fw);
                acc += prod;
                mag += fabs(prod);
            }
        }
    }
    *acc_out = acc;
    *mag_out = mag;
}

static int make_shape(oracle_shape *p, int n, int c, int h, int w, int k, int r, int s,
                      int std_h, int std_w, int pad_h, int pad_w, int layout)
{
    if (n < 1 || c < 1 || k < 1 || (layout != ORACLE_HWCN && layout != ORACLE_NCHW))
        return -1;
    p->n = n; p->c = c; p->h = h; p->w = w; p->k = k; p->r = r; p->s = s;
    p->std_h = std_h; p->std_w = std_w; p->pad_h = pad_h; p->pad_w = pad_w;
    p->layout = layout;
    return oracle_out_dims(h, w, r, s, std_h, std_w, pad_h, pad_w, &p->out_h, &p->out_w);
}

/* Every output element: the seven nested loops of the direct convolution.
 * acc and mag hold n*k*out_h*out_w doubles in the layout's output order.
 * Returns 0, or -1 on an invalid shape. */
int oracle_conv2d_f64(const float *x, const float *wt, double *acc, double *mag,
                      int n, int c, int h, int w, int k, int r, int s,
                      int std_h, int std_w, int pad_h, int pad_w, int layout)
{
    oracle_shape p;
    if (make_shape(&p, n, c, h, w, k, r, s, std_h, std_w, pad_h, pad_w, layout))
        return -1;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int b = 0; b < p.n; ++b)
        for (int oc = 0; oc < p.k; ++oc)
            for (int oh = 0; oh < p.out_h; ++oh)
                for (int ow = 0; ow < p.out_w; ++ow) {
                    int64_t o = out_index(&p, b, oc, oh, ow);
                    one_output(x, wt, &p, b, oc, oh, ow, &acc[o], &mag[o]);
                }
    return 0;
}

/* Selected output elements, given as flat indices into the layout's output
 * array (used at full layer sizes, where computing every output on the CPU
 * would take too long).  Returns 0, or -1 on an invalid shape or index. */
int oracle_conv2d_points_f64(const float *x, const float *wt, const int64_t *idx, int64_t npts,
                             double *acc, double *mag,
                             int n, int c, int h, int w, int k, int r, int s,
                             int std_h, int std_w, int pad_h, int pad_w, int layout)
{
    oracle_shape p;
    if (make_shape(&p, n, c, h, w, k, r, s, std_h, std_w, pad_h, pad_w, layout))
        return -1;
    int64_t total = (int64_t)p.n * p.k * p.out_h * p.out_w;
    for (int64_t t = 0; t < npts; ++t)
        if (idx[t] < 0 || idx[t] >= total)
            return -1;
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t t = 0; t < npts; ++t) {
        int64_t q = idx[t];
        int b, oc, oh, ow;
        if (p.layout == ORACLE_HWCN) {          /* [outH][outW][OC][B] */
            b = (int)(q % p.n);     q /= p.n;
            oc = (int)(q % p.k);    q /= p.k;
            ow = (int)(q % p.out_w);
            oh = (int)(q / p.out_w);
        } else {                                /* [B][OC][outH][outW] */
            ow = (int)(q % p.out_w); q /= p.out_w;
            oh = (int)(q % p.out_h); q /= p.out_h;
            oc = (int)(q % p.k);
            b = (int)(q / p.k);
        }
        one_output(x, wt, &p, b, oc, oh, ow, &acc[t], &mag[t]);
    }
    return 0;
}
