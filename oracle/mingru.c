/*
 * Plain fp64 CPU oracle of the paper's bidirectional minGRU backbone (Sec.
 * Encoder, Eq. (2)).  Every layer of the stack carries H channels per
 * direction: four linear maps of the layer's input give a candidate and a
 * gate for the left-to-right pass and another pair for the right-to-left
 * pass; each pass runs the update of Eq. (2) over the track's hits, and at
 * every hit the 2H states of the two passes, stacked, form the input of the
 * layer above.
 * TEST INFRASTRUCTURE ONLY: it exists to check the GPU library.  Only the
 * test suite, the smoke check and the benchmark's CPU-baseline leg may load
 * or call it.  It shares no code, header or table with the GPU library.
 *
 * Readings: the update of Eq. (2) in both directions, with the sigmoid's
 * output as the update gate and a zero initial state; no activation on the
 * candidate; no normalisation or residual inside the backbone (the paper
 * names the RMSNorm only before the head); the front end is the linear
 * (x, y, z) embedding or the Fourier front end of oracle.c.
 *
 * Blob (float32, matrices row-major [out][in]):
 *   front end: embed.W[d][3], embed.b[d]  (or, with n_feat = F > 0,
 *              fe.lo[F], fe.hi[F], fe.W[d][32 F], fe.b[d]),
 *   per layer l: W[4H][D_l], b[4H], with D_0 = d and D_l = 2H after that;
 *              rows 0..H-1: forward candidate, H..2H-1: forward gate
 *              pre-activation, 2H..3H-1: reverse candidate, 3H..4H-1:
 *              reverse gate pre-activation; the input of layer l >= 1 is
 *              [f; b] of layer l - 1 (forward state in columns 0..H-1).
 * Output per track: the last layer's forward state at the last hit, then its
 * reverse state at the first hit (2H values: the readout's input).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* from oracle.c (the same test-only library) */
double orc_sigmoid(double v);
void orc_linear(const double *W, const double *b, const double *x, int n_rows, int n_in, int n_out, double *y);
void orc_scan_forward(const double *x, const double *a, int L, int d, double *f);
void orc_scan_backward(const double *x, const double *a, int L, int d, double *b);
void orc_fourier_features(const float *feat, int n_feat, const float *lo, const float *hi, double *phi);

#define MG_NSCALE 16

static size_t mg_front_size(int d, int n_feat) {
    size_t dd = (size_t)d, F = (size_t)n_feat;
    return n_feat > 0 ? 2 * F + dd * 2 * MG_NSCALE * F + dd : 4 * dd;
}

size_t orc_mingru_blob_size(int n_layers, int d, int H, int n_feat) {
    if (n_layers < 1 || d <= 0 || H <= 0 || n_feat < 0) return 0;
    size_t s = mg_front_size(d, n_feat);
    for (int l = 0; l < n_layers; ++l) {
        size_t din = l == 0 ? (size_t)d : 2 * (size_t)H;
        s += 4 * (size_t)H * din + 4 * (size_t)H;
    }
    return s;
}

static void mg_to_double(const float *src, size_t n, double *dst) {
    for (size_t i = 0; i < n; ++i) dst[i] = (double)src[i];
}

/* One track: in [L][3] (x, y, z) or [L][F] features; states [2H].  Returns
 * 0, or -1 for L < 1 (states NaN). */
int orc_mingru_track(const float *in, int L, int n_feat, int n_layers, int d, int H, const float *blob,
                     double *states) {
    if (L < 1) {
        for (int j = 0; j < 2 * H; ++j) states[j] = NAN;
        return -1;
    }
    const size_t dd = (size_t)d, HH = (size_t)H, LL = (size_t)L;
    const size_t K = 2 * MG_NSCALE * (size_t)(n_feat > 0 ? n_feat : 0);
    const size_t dmax = dd > 2 * HH ? dd : 2 * HH;
    size_t wmax = 4 * HH * dmax;
    if (dd * K > wmax) wmax = dd * K;
    if (dd * 3 > wmax) wmax = dd * 3;
    double *buf = (double *)malloc(sizeof(double) * (LL * dmax + LL * 4 * HH + 4 * LL * HH + wmax + 4 * HH + K + 3 * LL));
    double *X = buf;                 /* layer input [L][D_l] */
    double *P = X + LL * dmax;       /* projection [L][4H] */
    double *xf = P + LL * 4 * HH, *af = xf + LL * HH, *xb = af + LL * HH, *ab = xb + LL * HH;
    double *Wd = ab + LL * HH;
    double *bd = Wd + wmax;
    double *phi = bd + 4 * HH;
    double *u = phi + K;

    /* front end: the layer-1 input, width d */
    if (n_feat > 0) {
        const float *lo = blob, *hi = blob + n_feat, *fW = hi + n_feat, *fB = fW + dd * K;
        mg_to_double(fW, dd * K, Wd);
        mg_to_double(fB, dd, bd);
        for (int t = 0; t < L; ++t) {
            orc_fourier_features(in + (size_t)t * n_feat, n_feat, lo, hi, phi);
            orc_linear(Wd, bd, phi, 1, (int)K, d, X + (size_t)t * d);
        }
    } else {
        for (int t = 0; t < L; ++t) {
            u[3 * t + 0] = ((double)in[3 * t + 0] + 1000.0) / 2000.0;
            u[3 * t + 1] = ((double)in[3 * t + 1] + 1000.0) / 2000.0;
            u[3 * t + 2] = ((double)in[3 * t + 2] + 3000.0) / 6000.0;
        }
        mg_to_double(blob, dd * 3, Wd);
        mg_to_double(blob + dd * 3, dd, bd);
        orc_linear(Wd, bd, u, L, 3, d, X);
    }
    const float *lw = blob + mg_front_size(d, n_feat);
    int din = d;
    for (int l = 0; l < n_layers; ++l) {
        /* projection to the forward and reverse candidates and gates */
        mg_to_double(lw, 4 * HH * (size_t)din, Wd);
        mg_to_double(lw + 4 * HH * (size_t)din, 4 * HH, bd);
        orc_linear(Wd, bd, X, L, din, 4 * H, P);
        lw += 4 * HH * (size_t)din + 4 * HH;
        for (int t = 0; t < L; ++t)
            for (int j = 0; j < H; ++j) {
                const double *p = P + (size_t)t * 4 * HH;
                xf[(size_t)t * HH + j] = p[j];
                af[(size_t)t * HH + j] = orc_sigmoid(p[HH + j]);
                xb[(size_t)t * HH + j] = p[2 * HH + j];
                ab[(size_t)t * HH + j] = orc_sigmoid(p[3 * HH + j]);
            }
        /* the two scans of Eq. (2): forward from the first hit, reverse from the last;
         * their outputs (reusing the candidate arrays' neighbours) */
        double *f = P, *b = P + LL * HH; /* P is no longer needed */
        orc_scan_forward(xf, af, L, H, f);
        orc_scan_backward(xb, ab, L, H, b);
        if (l == n_layers - 1) {
            memcpy(states, f + (LL - 1) * HH, sizeof(double) * HH);
            memcpy(states + HH, b, sizeof(double) * HH);
        }
        /* concatenated [f; b] is the next layer's input */
        for (int t = 0; t < L; ++t) {
            memcpy(X + (size_t)t * 2 * HH, f + (size_t)t * HH, sizeof(double) * HH);
            memcpy(X + (size_t)t * 2 * HH + HH, b + (size_t)t * HH, sizeof(double) * HH);
        }
        din = 2 * H;
    }
    free(buf);
    return 0;
}

/* Packed batch: states [n_tracks][2H].  Returns the number of tracks with no
 * hits (NaN rows), or -1 for bad arguments. */
long orc_mingru_states(const float *in, int n_feat, const int32_t *offsets, int32_t n_tracks, int n_layers, int d,
                       int H, const float *blob, size_t n_floats, double *states, int n_threads) {
    if (n_tracks < 0 || d <= 0 || H <= 0 || n_layers < 1 || n_feat < 0 || !blob ||
        (n_tracks > 0 && (!in || !offsets || !states)))
        return -1;
    if (n_floats != orc_mingru_blob_size(n_layers, d, H, n_feat)) return -1;
    const size_t stride = n_feat > 0 ? (size_t)n_feat : 3;
    long bad = 0;
#ifdef _OPENMP
    int nt = n_threads > 0 ? n_threads : omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 16) num_threads(nt) reduction(+ : bad)
#endif
    for (int32_t i = 0; i < n_tracks; ++i) {
        int L = offsets[i + 1] - offsets[i];
        if (orc_mingru_track(in + (size_t)offsets[i] * stride, L, n_feat, n_layers, d, H, blob,
                             states + (size_t)i * 2 * H) != 0)
            bad += 1;
    }
    (void)n_threads;
    return bad;
}
