/*
 * Plain fp64 CPU oracle of the paper's readout and decode (Sec. Encoder, last
 * paragraph; Sec. Losses; the seed-anchored output of Sec. Method).  TEST
 * INFRASTRUCTURE ONLY: it exists to check the GPU library.  Only the test
 * suite, the smoke check and the benchmark's CPU-baseline leg may load or
 * call it.  It shares no code, header or table with the GPU library.
 *
 * For one track, with z = [f_L; b_1] the last layer's forward state at the
 * last hit and reverse state at the first hit (2d values):
 *   1. y = g (.) z / sqrt(mean(z^2) + eps), eps = 1e-6 (RMSNorm, learned gain);
 *   2. h = SiLU(W1 y + b1), with its own hidden width (the paper's head has
 *      128 hidden units);
 *   3. q = W2 h + b2: 35 outputs, seven quantiles for each of the five
 *      parameters (d0, z0, phi, theta, q/p), parameter p owning q[7p .. 7p+6]
 *      at ascending quantile levels, the middle one, q[7p + 3], at level 1/2;
 *   4. the point estimate of parameter p is its median quantile, q[7p + 3]
 *      (Sec. Losses: the median quantile is the point estimate);
 *   5. decode against the seed: d0, z0 and theta add the estimate to the seed;
 *      phi adds it and wraps to [-pi, pi); q/p is scale-free,
 *      q/p = q/p_seed + estimate * (|q/p_seed| + 0.02 / GeV).
 *
 * Head blob (float32, matrices row-major [out][in]), for states of width 2d
 * and hidden width nh:
 *   norm.g[2d], W1[nh][2d], b1[nh], W2[35][nh], b2[35].
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#define ORC_RO_EPS 1e-6
#define ORC_QOP_EPS 0.02 /* 1/GeV */
#define ORC_NQ 7         /* quantiles per parameter */
#define ORC_NOUT 35
#define ORC_PI 3.14159265358979323846

size_t orc_readout_blob_size(int d, int nh) {
    if (d <= 0 || nh <= 0) return 0;
    size_t dd = (size_t)d, h = (size_t)nh;
    return 2 * dd + h * 2 * dd + h + ORC_NOUT * h + ORC_NOUT;
}

static double orc_ro_silu(double v) { return v / (1.0 + exp(-v)); }

/* Decode the five point estimates against a seed (d0, z0, phi, theta, q/p). */
void orc_decode(const double *seed, const double *est, double *out5) {
    out5[0] = seed[0] + est[0];
    out5[1] = seed[1] + est[1];
    double phi = seed[2] + est[2];
    phi = phi - 2.0 * ORC_PI * floor((phi + ORC_PI) / (2.0 * ORC_PI)); /* [-pi, pi) */
    out5[2] = phi;
    out5[3] = seed[3] + est[3];
    out5[4] = seed[4] + est[4] * (fabs(seed[4]) + ORC_QOP_EPS);
}

/* One track: z [2d], head blob of hidden width nh, seed [5] -> q35 [35]
 * (optional) and out5. */
void orc_readout_track(const double *z, int d, int nh, const float *hb, const double *seed, double *q35,
                       double *out5) {
    const size_t dd = (size_t)d, H = (size_t)nh;
    const float *g = hb, *W1 = g + 2 * dd, *b1 = W1 + H * 2 * dd, *W2 = b1 + H, *b2 = W2 + ORC_NOUT * H;
    double *y = (double *)malloc(sizeof(double) * (2 * dd + H));
    double *h = y + 2 * dd;
    double q[ORC_NOUT];
    double ss = 0.0;
    for (size_t j = 0; j < 2 * dd; ++j) ss += z[j] * z[j];
    const double inv = 1.0 / sqrt(ss / (double)(2 * dd) + ORC_RO_EPS);
    for (size_t j = 0; j < 2 * dd; ++j) y[j] = (double)g[j] * z[j] * inv;
    for (size_t u = 0; u < H; ++u) {
        double acc = (double)b1[u];
        for (size_t j = 0; j < 2 * dd; ++j) acc += (double)W1[u * 2 * dd + j] * y[j];
        h[u] = orc_ro_silu(acc);
    }
    for (int o = 0; o < ORC_NOUT; ++o) {
        double acc = (double)b2[o];
        for (size_t u = 0; u < H; ++u) acc += (double)W2[(size_t)o * H + u] * h[u];
        q[o] = acc;
    }
    double est[5];
    for (int p = 0; p < 5; ++p) est[p] = q[ORC_NQ * p + ORC_NQ / 2];
    orc_decode(seed, est, out5);
    if (q35)
        for (int o = 0; o < ORC_NOUT; ++o) q35[o] = q[o];
    free(y);
}

/* Batch: states [n][2d], seeds [n][5] -> q35 [n][35] (optional), out [n][5].
 * A track whose states or seed hold a NaN gets NaN outputs (NaN propagates).
 * Returns 0, or -1 for bad arguments. */
long orc_readout_tracks(const double *states, int32_t n, int d, int nh, const float *hb, size_t n_floats,
                        const double *seeds, double *q35, double *out) {
    if (n < 0 || d <= 0 || nh <= 0 || !hb || n_floats != orc_readout_blob_size(d, nh) ||
        (n > 0 && (!states || !seeds || !out)))
        return -1;
    for (int32_t i = 0; i < n; ++i)
        orc_readout_track(states + (size_t)i * 2 * d, d, nh, hb, seeds + (size_t)i * 5,
                          q35 ? q35 + (size_t)i * ORC_NOUT : NULL, out + (size_t)i * 5);
    return 0;
}
