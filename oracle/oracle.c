/*
 * Plain fp64 CPU oracle of the bidirectional gated linear recurrent track-fit
 * encoder.  TEST INFRASTRUCTURE ONLY: it exists to check the GPU library.
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load or call it; the product path never does.  It shares no code, header
 * or table with the GPU library.
 *
 * Everything is computed in double precision with scalar loops, one track at a
 * time, in the order the method states it.  A track's result depends only on
 * its own hits and the weights.
 *
 * Readings of points the paper leaves open are fixed here and listed with the
 * design notes: update-gate convention of Eq. (2) (the sigmoid output is the
 * gate z_t), zero initial state in both directions, no activation on the
 * candidate, one candidate/gate pair shared by both scan directions, the
 * unused third of the input projection is skipped, pre-norm residual layers
 * with RMSNorm eps = 1e-6 inside the square root, a learned 3->d embedding of
 * min-max normalised (x, y, z), mean pooling over exactly the track's hits,
 * and a SiLU between the two head layers.
 *
 * Weight blob (float32, matrices row-major [out][in]), in this order:
 *   embed.W[d][3], embed.b[d],
 *   per layer: norm.g[d], in.W[3d][d], in.b[3d], out.W[d][2d], out.b[d],
 *   head.W1[d][d], head.b1[d], head.W2[5][d], head.b2[5].
 * With the paper's Fourier front end (n_feat = F > 0 per-hit features instead
 * of (x, y, z)), the first two entries are replaced by
 *   fe.lo[F], fe.hi[F], fe.W[d][32 F], fe.b[d]
 * (see orc_fourier_features for the column order of fe.W).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_EPS 1e-6
#define ORC_PI 3.14159265358979323846
#define ORC_NSCALE 16 /* Fourier scales (Sec. Encoder) */

/* Fixed detector bounds used for the min-max normalisation of the hit
 * coordinates (Sec. Encoder: features are min-max normalised to [0, 1]). */
#define ORC_XY_MIN (-1000.0)
#define ORC_XY_SPAN 2000.0
#define ORC_Z_MIN (-3000.0)
#define ORC_Z_SPAN 6000.0

size_t orc_blob_size(int n_layers, int d) {
    size_t dd = (size_t)d;
    size_t per_layer = dd + 3 * dd * dd + 3 * dd + dd * 2 * dd + dd;
    return 3 * dd + dd + (size_t)n_layers * per_layer + dd * dd + dd + 5 * dd + 5;
}

/* Floats of the front end: (x, y, z) embedding, or the Fourier front end of F features. */
static size_t orc_front_size(int d, int n_feat) {
    size_t dd = (size_t)d, F = (size_t)n_feat;
    return n_feat > 0 ? 2 * F + dd * 2 * ORC_NSCALE * F + dd : 4 * dd;
}

/* Blob size of the model with the Fourier front end over n_feat features. */
size_t orc_fourier_blob_size(int n_layers, int d, int n_feat) {
    if (n_feat <= 0) return 0;
    return orc_blob_size(n_layers, d) - 4 * (size_t)d + orc_front_size(d, n_feat);
}

/* Multi-scale Fourier featurisation of one hit (Sec. Encoder): each of the F
 * features is min-max normalised with its bounds, u = (x - lo) / (hi - lo),
 * in float32 (the model's number type: the subtraction, the reciprocal of
 * the span and the product are each rounded to float32), and expanded at the
 * 16 scales 2^s, s = 0..15: phi[32 f + s] = sin(pi 2^s u_f) and
 * phi[32 f + 16 + s] = cos(pi 2^s u_f).  The phase 2^s u_f is exact in
 * double and reduced modulo 2 exactly before the sine is taken. */
void orc_fourier_features(const float *feat, int n_feat, const float *lo, const float *hi, double *phi) {
    for (int f = 0; f < n_feat; ++f) {
        const float span = hi[f] - lo[f];
        const float inv = 1.0f / span;
        const float t = feat[f] - lo[f];
        const float u = t * inv;
        for (int sc = 0; sc < ORC_NSCALE; ++sc) {
            const double x = fmod(ldexp((double)u, sc), 2.0);
            phi[2 * ORC_NSCALE * f + sc] = sin(ORC_PI * x);
            phi[2 * ORC_NSCALE * f + ORC_NSCALE + sc] = cos(ORC_PI * x);
        }
    }
}

/* Logistic sigmoid, the gate nonlinearity z_t = sigma(Linear(m_t)) of Sec. Encoder. */
double orc_sigmoid(double v) { return 1.0 / (1.0 + exp(-v)); }

/* SiLU(v) = v * sigmoid(v), the activation read between the two head layers. */
double orc_silu(double v) { return v / (1.0 + exp(-v)); }

/* Affine map applied row by row: y[t][o] = b[o] + sum_i W[o][i] * x[t][i].
 * The "Linear" of Sec. Encoder.  b may be NULL (no bias). */
void orc_linear(const double *W, const double *b, const double *x, int n_rows,
                int n_in, int n_out, double *y) {
    for (int t = 0; t < n_rows; ++t) {
        for (int o = 0; o < n_out; ++o) {
            double s = b ? b[o] : 0.0;
            for (int i = 0; i < n_in; ++i) s += W[(size_t)o * n_in + i] * x[(size_t)t * n_in + i];
            y[(size_t)t * n_out + o] = s;
        }
    }
}

/* RMSNorm (Zhang & Sennrich, cited in Sec. Encoder): each row r is scaled by
 * 1/sqrt(mean(r^2) + eps) and multiplied elementwise by the gain g. */
void orc_rmsnorm(const double *r, const double *g, int n_rows, int d, double eps, double *y) {
    for (int t = 0; t < n_rows; ++t) {
        const double *row = r + (size_t)t * d;
        double ss = 0.0;
        for (int j = 0; j < d; ++j) ss += row[j] * row[j];
        double inv = 1.0 / sqrt(ss / d + eps);
        for (int j = 0; j < d; ++j) y[(size_t)t * d + j] = g[j] * row[j] * inv;
    }
}

/* Forward scan, Eq. (2): h_t = h_{t-1} + z_t (.) (n_t - h_{t-1}), h_0 = 0,
 * for t = 1..L, each channel independently.  x is n_t, a is z_t; rows [L][d]. */
void orc_scan_forward(const double *x, const double *a, int L, int d, double *f) {
    for (int j = 0; j < d; ++j) {
        double h = 0.0;
        for (int t = 0; t < L; ++t) {
            size_t k = (size_t)t * d + j;
            h = h + a[k] * (x[k] - h);
            f[k] = h;
        }
    }
}

/* Reverse scan (Sec. Encoder: a forward and a reverse scan per layer): the same
 * update run from the last hit to the first, h_{L+1} = 0. */
void orc_scan_backward(const double *x, const double *a, int L, int d, double *b) {
    for (int j = 0; j < d; ++j) {
        double h = 0.0;
        for (int t = L - 1; t >= 0; --t) {
            size_t k = (size_t)t * d + j;
            h = h + a[k] * (x[k] - h);
            b[k] = h;
        }
    }
}

/* Pointers into the blob, resolved in blob order. */
typedef struct {
    const float *eW, *eb;
    const float *g, *inW, *inb, *outW, *outb; /* layer 0; stride per layer below */
    size_t layer_stride;
    const float *W1, *b1, *W2, *b2;
} orc_params;

static void orc_resolve(const float *blob, int n_layers, int d, int n_feat, orc_params *p) {
    size_t dd = (size_t)d, o = 0;
    p->eW = blob; /* the front end's first array (embed.W, or fe.lo) */
    p->eb = blob + 3 * dd;
    o += orc_front_size(d, n_feat);
    p->g = blob + o;
    p->inW = p->g + dd;
    p->inb = p->inW + 3 * dd * dd;
    p->outW = p->inb + 3 * dd;
    p->outb = p->outW + dd * 2 * dd;
    p->layer_stride = dd + 3 * dd * dd + 3 * dd + dd * 2 * dd + dd;
    o += (size_t)n_layers * p->layer_stride;
    p->W1 = blob + o; o += dd * dd;
    p->b1 = blob + o; o += dd;
    p->W2 = blob + o; o += 5 * dd;
    p->b2 = blob + o;
}

static void to_double(const float *src, size_t n, double *dst) {
    for (size_t i = 0; i < n; ++i) dst[i] = (double)src[i];
}

/*
 * One track through the whole model.  hits: [L][3] float (x, y, z) in mm, or
 * with n_feat = F > 0 the [L][F] per-hit features of the Fourier front end.
 * out5 receives the five head outputs (d0, z0, phi, theta, q/p order).
 * pooled (length d) and resid ([L][d], the residual stream after the last
 * layer) are optional outputs for the tests.  states (length 2d, optional)
 * receives the last layer's end states read by the paper's own readout
 * (Sec. Encoder, last paragraph): the forward state at the last hit, then
 * the reverse state at the first hit.  Returns 0, or -1 if L < 1 (then out5,
 * pooled and states are NaN: the mean over zero hits is undefined).
 */
int orc_track_forward(const float *hits, int L, int n_feat, int n_layers, int d, const float *blob,
                      double *out5, double *pooled, double *resid, double *states) {
    if (L < 1) {
        for (int k = 0; k < 5; ++k) out5[k] = NAN;
        if (pooled)
            for (int j = 0; j < d; ++j) pooled[j] = NAN;
        if (states)
            for (int j = 0; j < 2 * d; ++j) states[j] = NAN;
        return -1;
    }
    orc_params P;
    orc_resolve(blob, n_layers, d, n_feat, &P);
    size_t Ld = (size_t)L * d, dd = (size_t)d;
    const size_t K = 2 * ORC_NSCALE * (size_t)(n_feat > 0 ? n_feat : 0); /* Fourier width */
    size_t wmax = 4 * dd * dd > dd * K ? 4 * dd * dd : dd * K;
    double *buf = (double *)malloc(sizeof(double) * (7 * Ld + 3 * (size_t)L + wmax + 8 * dd + K + 16));
    double *r = buf, *y = r + Ld, *x = y + Ld, *gh = x + Ld, *a = gh + Ld, *f = a + Ld, *b = f + Ld;
    double *u = b + Ld;
    double *Wd = u + 3 * (size_t)L; /* weight staging in double: out.W [d][2d] or fe.W [d][32 F] */
    double *bd = Wd + wmax;         /* bias staging, up to 3d */
    double *fb = bd + 4 * dd;       /* one [f; b] row, 2d */
    double *tmp = fb + 2 * dd;      /* d */
    double *phi = tmp + dd;         /* one hit's Fourier features, 32 F */

    if (n_feat > 0) {
        /* Steps 1-2, paper front end: Fourier features of each hit, then the
         * dense projection to the encoder width (Sec. Encoder). */
        const float *lo = blob, *hi = blob + n_feat, *fW = hi + n_feat, *fbias = fW + dd * K;
        to_double(fW, dd * K, Wd);
        to_double(fbias, dd, bd);
        for (int t = 0; t < L; ++t) {
            orc_fourier_features(hits + (size_t)t * n_feat, n_feat, lo, hi, phi);
            orc_linear(Wd, bd, phi, 1, (int)K, d, r + (size_t)t * d);
        }
    } else {
        /* Step 1: min-max normalise the coordinates to [0, 1] (Sec. Encoder). */
        for (int t = 0; t < L; ++t) {
            u[3 * t + 0] = ((double)hits[3 * t + 0] - ORC_XY_MIN) / ORC_XY_SPAN;
            u[3 * t + 1] = ((double)hits[3 * t + 1] - ORC_XY_MIN) / ORC_XY_SPAN;
            u[3 * t + 2] = ((double)hits[3 * t + 2] - ORC_Z_MIN) / ORC_Z_SPAN;
        }
        /* Step 2: dense projection to the encoder width d (Sec. Encoder). */
        to_double(P.eW, dd * 3, Wd);
        to_double(P.eb, dd, bd);
        orc_linear(Wd, bd, u, L, 3, d, r);
    }

    /* Step 3: the stacked bidirectional layers. */
    for (int l = 0; l < n_layers; ++l) {
        size_t off = (size_t)l * P.layer_stride;
        /* pre-norm */
        to_double(P.g + off, dd, tmp);
        orc_rmsnorm(r, tmp, L, d, ORC_EPS, y);
        /* candidate n_t: rows 0..d-1 of the input projection */
        to_double(P.inW + off, dd * dd, Wd);
        to_double(P.inb + off, dd, bd);
        orc_linear(Wd, bd, y, L, d, d, x);
        /* gate pre-activation: rows d..2d-1; the gate z_t = sigmoid(.) */
        to_double(P.inW + off + dd * dd, dd * dd, Wd);
        to_double(P.inb + off + dd, dd, bd);
        orc_linear(Wd, bd, y, L, d, d, gh);
        for (size_t k = 0; k < Ld; ++k) a[k] = orc_sigmoid(gh[k]);
        /* rows 2d..3d-1 are unused and not evaluated */
        /* forward and reverse scans, Eq. (2) */
        orc_scan_forward(x, a, L, d, f);
        orc_scan_backward(x, a, L, d, b);
        if (states && l == n_layers - 1) {
            memcpy(states, f + (size_t)(L - 1) * d, sizeof(double) * dd);
            memcpy(states + dd, b, sizeof(double) * dd);
        }
        /* merge the two directions: r <- r + W_out [f; b] + b_out */
        to_double(P.outW + off, dd * 2 * dd, Wd);
        to_double(P.outb + off, dd, bd);
        for (int t = 0; t < L; ++t) {
            memcpy(fb, f + (size_t)t * d, sizeof(double) * dd);
            memcpy(fb + dd, b + (size_t)t * d, sizeof(double) * dd);
            orc_linear(Wd, bd, fb, 1, 2 * d, d, tmp);
            for (int j = 0; j < d; ++j) r[(size_t)t * d + j] += tmp[j];
        }
    }
    if (resid) memcpy(resid, r, sizeof(double) * Ld);

    /* Step 4: mean over exactly the track's L hits. */
    double *p = fb; /* reuse, length d */
    for (int j = 0; j < d; ++j) {
        double s = 0.0;
        for (int t = 0; t < L; ++t) s += r[(size_t)t * d + j];
        p[j] = s / L;
    }
    if (pooled) memcpy(pooled, p, sizeof(double) * dd);

    /* Step 5: two-layer head, out = W2 SiLU(W1 p + b1) + b2. */
    to_double(P.W1, dd * dd, Wd);
    to_double(P.b1, dd, bd);
    orc_linear(Wd, bd, p, 1, d, d, tmp);
    for (int j = 0; j < d; ++j) tmp[j] = orc_silu(tmp[j]);
    to_double(P.W2, 5 * dd, Wd);
    to_double(P.b2, 5, bd);
    orc_linear(Wd, bd, tmp, 1, d, 5, out5);
    free(buf);
    return 0;
}

/*
 * Packed batch (Sec. Kernel adaptation: packed, unpadded layout): track i owns
 * hits rows offsets[i] .. offsets[i+1]-1.  out is [n_tracks][5] double.
 * n_threads <= 0 uses the OpenMP default.  Returns the number of tracks whose
 * length was below 1 (their outputs are NaN), or -1 for bad arguments.
 */
static size_t orc_model_size(int n_layers, int d, int n_feat) {
    return n_feat > 0 ? orc_fourier_blob_size(n_layers, d, n_feat) : orc_blob_size(n_layers, d);
}

long orc_fit_tracks(const float *hits, int n_feat, const int32_t *offsets, int32_t n_tracks, int n_layers,
                    int d, const float *blob, size_t n_floats, double *out, int n_threads) {
    if (n_tracks < 0 || d <= 0 || n_layers < 0 || n_feat < 0 || !blob ||
        (n_tracks > 0 && (!hits || !offsets || !out)))
        return -1;
    if (n_floats != orc_model_size(n_layers, d, n_feat)) return -1;
    const size_t stride = n_feat > 0 ? (size_t)n_feat : 3;
    long bad = 0;
#ifdef _OPENMP
    int nt = n_threads > 0 ? n_threads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 16) num_threads(nt) reduction(+ : bad)
#endif
    for (int32_t i = 0; i < n_tracks; ++i) {
        int L = offsets[i + 1] - offsets[i];
        if (orc_track_forward(hits + (size_t)offsets[i] * stride, L, n_feat, n_layers, d, blob,
                              out + (size_t)i * 5, NULL, NULL, NULL) != 0)
            bad += 1;
    }
    (void)n_threads;
    return bad;
}

/* Packed batch of the paper readout's inputs: states [n_tracks][2d] (forward
 * state at the last hit, reverse state at the first hit, of the last layer).
 * Returns the number of tracks with no hits (NaN rows), or -1 for bad
 * arguments.  With n_layers = 0 there are no states and every row is NaN. */
long orc_track_states(const float *hits, int n_feat, const int32_t *offsets, int32_t n_tracks, int n_layers,
                      int d, const float *blob, size_t n_floats, double *states, int n_threads) {
    if (n_tracks < 0 || d <= 0 || n_layers < 0 || n_feat < 0 || !blob ||
        (n_tracks > 0 && (!hits || !offsets || !states)))
        return -1;
    if (n_floats != orc_model_size(n_layers, d, n_feat)) return -1;
    const size_t stride = n_feat > 0 ? (size_t)n_feat : 3;
    long bad = 0;
#ifdef _OPENMP
    int nt = n_threads > 0 ? n_threads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 16) num_threads(nt) reduction(+ : bad)
#endif
    for (int32_t i = 0; i < n_tracks; ++i) {
        int L = offsets[i + 1] - offsets[i];
        double out5[5];
        double *st = states + (size_t)i * 2 * d;
        if (n_layers == 0)
            for (int j = 0; j < 2 * d; ++j) st[j] = NAN;
        if (orc_track_forward(hits + (size_t)offsets[i] * stride, L, n_feat, n_layers, d, blob, out5, NULL,
                              NULL, n_layers > 0 ? st : NULL) != 0)
            bad += 1;
    }
    (void)n_threads;
    return bad;
}

/* Number of threads the OpenMP runtime would use for n_threads (<= 0: default). */
int orc_threads(int n_threads) {
#ifdef _OPENMP
    return n_threads > 0 ? n_threads : omp_get_max_threads();
#else
    (void)n_threads;
    return 1;
#endif
}
