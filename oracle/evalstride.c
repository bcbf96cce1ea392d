/*
 * Oracle for dense signal scanning -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg use
 * this file.  The GPU library never links, loads or calls it, and it shares no
 * code with the GPU library.
 *
 * What it computes is the plain definition that the fast method provably reaches
 * (Theorem "processing chain", Sect. 4.3: the transformed network equals
 * Slide_{EvalStride_L}).  For every requested window position it
 *   1. extracts the patch of receptive-field size B (subsignal extraction
 *      operator, Definition in Sect. 2.3; 2-D patches as in Sect. 6.1),
 *   2. runs the ordinary strided network on it (EvalStride, Definition
 *      "processing chain", Sect. 4.2): per layer the multi-channel convolution of
 *      Sect. 3.3 plus bias and non-linearity, and the max-pooling kernel applied
 *      in a strided fashion (Definition "strided function" and the max-pooling
 *      example, Sect. 4),
 *   3. stores the single output sample.
 * All arithmetic is double precision, in the summation order the definitions
 * are written in.  OpenMP splits the windows over threads; each window is
 * computed by one thread start to finish, so the result does not depend on the
 * thread count.
 *
 * Conventions.  Arrays are row-major.  Signals are [C][H][W]; a 1-D signal has
 * H == 1 and filters/pools of height 1.  Filter banks are given in the paper's
 * orientation: w[o][l][mu_h][mu_w] is the tap that multiplies input sample
 * (c_h + i - mu_h, c_w + j - mu_w) in 1-based indices (Sect. 3.3), i.e. a true
 * convolution.  Indices below are 0-based; the 1-based formula
 * (xi*w)_i = sum_l sum_mu w_mu,l xi_{c+i-mu},l becomes
 * out[i] = sum_l sum_{m=0}^{c-1} w[m] * in[i + c - 1 - m].
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_CONV = 0, ORC_MAXPOOL = 1 };
enum { ORC_ACT_NONE = 0, ORC_ACT_RELU = 1, ORC_ACT_TANH = 2 };

typedef struct {
    int32_t kind;           /* ORC_CONV or ORC_MAXPOOL */
    int32_t cin, cout;      /* conv: channel counts */
    int32_t fh, fw;         /* conv: filter extents c (rows, cols) */
    int32_t act;            /* conv: non-linearity after the bias */
    int32_t kh, kw;         /* pool: block extents k (rows, cols) */
    const double* w;        /* conv: [cout][cin][fh][fw], paper orientation */
    const double* b;        /* conv: [cout] or NULL */
} orc_layer;

/* Extents after applying layers [0, upto) to a (C, h, w) patch.  Returns 0 when
 * the strided evaluation is well defined (conv: extent >= c; pool: extent is a
 * multiple of k), -1 otherwise. */
static int orc_extents(const orc_layer* L, int upto, int* C, int* h, int* w) {
    for (int t = 0; t < upto; ++t) {
        if (L[t].kind == ORC_CONV) {
            if (*C != L[t].cin || *h < L[t].fh || *w < L[t].fw) return -1;
            *C = L[t].cout;
            *h = *h - L[t].fh + 1;
            *w = *w - L[t].fw + 1;
        } else {
            if (*h % L[t].kh != 0 || *w % L[t].kw != 0 || *h == 0 || *w == 0) return -1;
            *h /= L[t].kh;
            *w /= L[t].kw;
        }
    }
    return 0;
}

/* Receptive field by brute force along one axis (0 = rows, 1 = cols): the
 * smallest patch extent for which the strided evaluation is well defined and
 * ends in exactly one sample (the condition of the main theorem, Sect. 4.3).
 * Independent of any closed form: it simply tries extents 1, 2, ... .
 * Returns the extent, or -1 if none up to smax works. */
int orc_receptive_field(const orc_layer* L, int n, int axis, int smax) {
    for (int s = 1; s <= smax; ++s) {
        int ok = 1, e = s;
        for (int t = 0; t < n && ok; ++t) {
            if (L[t].kind == ORC_CONV) {
                int c = axis == 0 ? L[t].fh : L[t].fw;
                if (e < c) ok = 0; else e = e - c + 1;
            } else {
                int k = axis == 0 ? L[t].kh : L[t].kw;
                if (e % k != 0) ok = 0; else e /= k;
            }
        }
        if (ok && e == 1) return s;
    }
    return -1;
}

static double orc_act(int act, double v) {
    if (act == ORC_ACT_RELU) return v > 0.0 ? v : 0.0;
    if (act == ORC_ACT_TANH) return tanh(v);
    return v;
}

/* Multi-channel convolution (Sect. 3.3) + bias + non-linearity on one patch.
 * in [cin][h][w] -> out [cout][h-fh+1][w-fw+1]. */
static void orc_conv(const orc_layer* l, const double* in, int h, int w, double* out) {
    const int oh = h - l->fh + 1, ow = w - l->fw + 1;
    for (int o = 0; o < l->cout; ++o) {
        const double bias = l->b ? l->b[o] : 0.0;
        for (int i = 0; i < oh; ++i) {
            for (int j = 0; j < ow; ++j) {
                double s = 0.0;
                for (int c = 0; c < l->cin; ++c) {
                    for (int mh = 0; mh < l->fh; ++mh) {
                        for (int mw = 0; mw < l->fw; ++mw) {
                            const double tap = l->w[(((int64_t)o * l->cin + c) * l->fh + mh) * l->fw + mw];
                            const int yy = i + l->fh - 1 - mh;
                            const int xx = j + l->fw - 1 - mw;
                            s += tap * in[((int64_t)c * h + yy) * w + xx];
                        }
                    }
                }
                out[((int64_t)o * oh + i) * ow + j] = orc_act(l->act, s + bias);
            }
        }
    }
}

/* Max-pooling kernel applied in a strided fashion: non-overlapping k-blocks
 * starting with the first sample, channel-wise maximum.
 * in [C][h][w] -> out [C][h/kh][w/kw]. */
static void orc_pool(const orc_layer* l, const double* in, int C, int h, int w, double* out) {
    const int oh = h / l->kh, ow = w / l->kw;
    for (int c = 0; c < C; ++c) {
        for (int i = 0; i < oh; ++i) {
            for (int j = 0; j < ow; ++j) {
                double m = in[((int64_t)c * h + i * l->kh) * w + j * l->kw];
                for (int a = 0; a < l->kh; ++a)
                    for (int b = 0; b < l->kw; ++b) {
                        const double v = in[((int64_t)c * h + i * l->kh + a) * w + j * l->kw + b];
                        if (v > m) m = v;
                    }
                out[((int64_t)c * oh + i) * ow + j] = m;
            }
        }
    }
}

/* Size of the largest intermediate (C*h*w) when running layers [0, upto) on a
 * (C0, ph, pw) patch, or -1 if the chain is not well defined on it. */
static int64_t orc_max_buffer(const orc_layer* L, int upto, int C0, int ph, int pw) {
    int C = C0, h = ph, w = pw;
    int64_t m = (int64_t)C * h * w;
    for (int t = 0; t < upto; ++t) {
        if (orc_extents(L + t, 1, &C, &h, &w) != 0) return -1;
        const int64_t s = (int64_t)C * h * w;
        if (s > m) m = s;
    }
    return m;
}

/* EvalStride on a list of windows.
 *   x        [C][H][W] signal
 *   ph, pw   patch extents (the receptive field B per axis for a full network)
 *   wi, wj   nwin top-left positions (0-based); each window is x[:, i:i+ph, j:j+pw]
 *   upto     number of layer descriptors to apply (n for the full network)
 *   out      [nwin][out_elems]: the result of each window, flattened [C][h][w]
 *   counts   optional [upto] array: number of function evaluations per layer
 *            summed over the windows (conv: output samples per channel set,
 *            i.e. evaluations of f_j; pool: evaluations of g_j)
 * Returns the number of output elements per window, or -1 on a bad request. */
int64_t orc_eval_stride(const orc_layer* L, int n, int upto, const double* x, int C, int H, int W,
                        int ph, int pw, const int64_t* wi, const int64_t* wj, int64_t nwin,
                        double* out, int64_t* counts, int nthreads) {
    if (upto < 0 || upto > n) return -1;
    int Cf = C, hf = ph, wf = pw;
    if (orc_extents(L, upto, &Cf, &hf, &wf) != 0) return -1;
    const int64_t out_elems = (int64_t)Cf * hf * wf;
    const int64_t bufsz = orc_max_buffer(L, upto, C, ph, pw);
    if (bufsz < 0) return -1;
    for (int64_t q = 0; q < nwin; ++q)
        if (wi[q] < 0 || wj[q] < 0 || wi[q] + ph > H || wj[q] + pw > W) return -1;

    if (counts) {
        int Cc = C, hc = ph, wc = pw;
        for (int t = 0; t < upto; ++t) {
            orc_extents(L + t, 1, &Cc, &hc, &wc);
            counts[t] = (int64_t)hc * wc * nwin;
        }
    }

    int err = 0;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel
#endif
    {
        double* b0 = (double*)malloc(sizeof(double) * bufsz);
        double* b1 = (double*)malloc(sizeof(double) * bufsz);
        if (!b0 || !b1) {
#ifdef _OPENMP
#pragma omp atomic write
#endif
            err = 1;
        }
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
        for (int64_t q = 0; q < nwin; ++q) {
            if (!b0 || !b1) continue;
            /* 1. subsignal (patch) extraction */
            for (int c = 0; c < C; ++c)
                for (int y = 0; y < ph; ++y)
                    memcpy(b0 + ((int64_t)c * ph + y) * pw,
                           x + ((int64_t)c * H + wi[q] + y) * W + wj[q], sizeof(double) * pw);
            /* 2. the strided network, layer by layer */
            int Cc = C, hc = ph, wc = pw;
            for (int t = 0; t < upto; ++t) {
                if (L[t].kind == ORC_CONV) {
                    orc_conv(L + t, b0, hc, wc, b1);
                    Cc = L[t].cout;
                    hc = hc - L[t].fh + 1;
                    wc = wc - L[t].fw + 1;
                } else {
                    orc_pool(L + t, b0, Cc, hc, wc, b1);
                    hc /= L[t].kh;
                    wc /= L[t].kw;
                }
                double* tmp = b0; b0 = b1; b1 = tmp;
            }
            /* 3. store */
            memcpy(out + q * out_elems, b0, sizeof(double) * out_elems);
        }
        free(b0);
        free(b1);
    }
    return err ? -1 : out_elems;
}

/* Number of threads an OpenMP region would use with the given request. */
int orc_threads(int nthreads) {
#ifdef _OPENMP
    if (nthreads > 0) return nthreads;
    return omp_get_max_threads();
#else
    (void)nthreads;
    return 1;
#endif
}
