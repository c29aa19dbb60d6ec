// Analytic three-hit seed and per-hit seed residual features on gfx950, in
// fp64 (Sec. Method, "Analytic seed": the seed perigee is computed in double
// precision because the transport to the beam line cancels at high momentum).
//
// One lane per track for the seed.  The circle through the track's first three hits
// (transverse plane) comes from the intersection of two perpendicular
// bisectors, written relative to the first hit; this is the same circle the
// paper's conformal map gives.  Its radius gives pT = kappa B R, its turning
// direction the charge, its closest approach to the z axis the perigee
// (d0, phi); the transverse arc lengths of the first and third hit from the
// perigee give cot(theta) and z0.  Then (one lane per hit row, so that the
// hit reads and feature writes are coalesced) every hit of the track gets its
// residual to the seed helix in the curvilinear frame there: the transverse
// component reduces to the signed radial distance from the circle, the other
// to sin(theta) times the z residual; both are asinh-compressed (argument in
// mm), with the helix path length from the perigee as third feature.
//
// Conventions: the perigee point is d0 (-sin phi, cos phi), phi the direction
// of motion there; k = +1 for counter-clockwise motion seen from +z and the
// charge is -k (field along +z).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "trackfit.h"

namespace {

constexpr double kKappa = 0.299792458;  // pT [GeV] = kappa * B [T] * R [m], unit charge
constexpr int kSeedWaves = 4;           // waves per workgroup, 64 tracks each
constexpr int kSeedBlock = 64 * kSeedWaves;

// Residual features of one hit against a circle (centre c, radius R, sense k)
// and the line z = z0 + s cot(theta) along its transverse arc s from the
// perigee (direction -C from the centre).
__device__ __forceinline__ void hit_features(const float *p, double cx, double cy, double R, double k, double z0,
                                             double cot, double st, float *f) {
    const double wx = (double)p[0] - cx, wy = (double)p[1] - cy;
    const double rho = sqrt(wx * wx + wy * wy);
    const double s = R * k * atan2(cy * wx - cx * wy, -(cx * wx + cy * wy));
    const double du = -k * (rho - R);
    const double dv = st * ((double)p[2] - (z0 + s * cot));
    // the residuals need fp64 (they are differences of values a thousand times
    // larger); their compression and the path length are stored as float32
    // and evaluated in it
    f[0] = asinhf((float)du);
    f[1] = asinhf((float)dv);
    f[2] = (float)(s / st);
}

// One wave per 64 consecutive tracks: lane i seeds track t0 + i, then the
// wave walks the hit rows of its tracks one row per lane (coalesced), each
// row finding its track in the wave's offsets by bisection in LDS.
__global__ __launch_bounds__(kSeedBlock) void tf_seed_kernel(const float *__restrict__ hits, long long n_hits,
                                                              const int *__restrict__ offsets, int n_tracks,
                                                              double b_tesla, double *__restrict__ seeds,
                                                              float *__restrict__ features, int fstride,
                                                              int *__restrict__ flags) {
    __shared__ double circ[kSeedWaves][7][64];  // cx, cy, R, k, z0, cot(theta), sin(theta) per track
    __shared__ int woff[kSeedWaves][65];        // the wave's track offsets
    __shared__ int wbits[kSeedWaves][64];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int t0 = (blockIdx.x * kSeedWaves + wv) * 64;
    if (t0 >= n_tracks) return;  // the whole wave
    const int i = t0 + lane;
    const bool active = i < n_tracks;
    const double nan = __builtin_nan("");
    const int o0 = offsets[0], oN = offsets[n_tracks];
    const int o = active ? offsets[i] : oN, e = active ? offsets[i + 1] : oN;
    int bits = 0;
    // rows must lie in [0, n_hits) for the hits and in [offsets[0],
    // offsets[n_tracks]) for the features
    if (o < 0 || e < o || (long long)e > n_hits || o < o0 || e > oN)
        bits = TF_SEED_BAD_OFFSETS;
    else if (active && e - o < 3)
        bits = TF_SEED_TOO_SHORT;
    double cx = 0, cy = 0, R = 0, k = 0, z0 = 0, cot = 0, st = 0;
    if (active && !bits) {
        const float *p = hits + (size_t)o * 3;
        const double x1 = p[0], y1 = p[1], z1 = p[2];
        const double bx = (double)p[3] - x1, by = (double)p[4] - y1;
        const double qx = (double)p[6] - x1, qy = (double)p[7] - y1, z3 = p[8];
        // centre relative to hit 1: equidistant from hits 1, 2 and 3
        const double det = 2.0 * (bx * qy - by * qx);
        if (det == 0.0) {
            bits = TF_SEED_NO_CIRCLE;
        } else {
            const double b2 = bx * bx + by * by, q2 = qx * qx + qy * qy;
            const double ux = (qy * b2 - by * q2) / det, uy = (bx * q2 - qx * b2) / det;
            cx = x1 + ux;
            cy = y1 + uy;
            R = sqrt(ux * ux + uy * uy);
            k = det > 0.0 ? 1.0 : -1.0;
            const double D = sqrt(cx * cx + cy * cy);
            // turning angle from the perigee (direction -C from the centre) to a
            // point w = P - C, positive along the motion
            auto turn = [&](double wx, double wy) { return k * atan2(cy * wx - cx * wy, -(cx * wx + cy * wy)); };
            const double s1 = R * turn(x1 - cx, y1 - cy);
            const double s3 = R * turn(x1 + qx - cx, y1 + qy - cy);
            const double theta = atan2(s3 - s1, z3 - z1);
            cot = (z3 - z1) / (s3 - s1);
            z0 = z1 - s1 * cot;
            st = sin(theta);
            double *sd = seeds + (size_t)i * 5;
            sd[0] = k * (D - R);
            sd[1] = z0;
            sd[2] = atan2(-k * cx, k * cy);
            sd[3] = theta;
            sd[4] = -k * st / (kKappa * b_tesla * R * 1e-3);
        }
    }
    if (active && bits) {
        double *sd = seeds + (size_t)i * 5;
        for (int j = 0; j < 5; ++j) sd[j] = nan;
        if (flags) atomicOr(flags, bits);
    }
    if (!features) return;
    if (__ballot(bits == TF_SEED_BAD_OFFSETS)) {
        // offsets out of order somewhere in this wave: every good track walks
        // its own rows
        if (bits == TF_SEED_BAD_OFFSETS) return;
        for (int h = o; h < e; ++h) {
            float *f = features + (size_t)(h - o0) * fstride;
            if (bits)
                f[0] = f[1] = f[2] = (float)nan;
            else
                hit_features(hits + (size_t)h * 3, cx, cy, R, k, z0, cot, st, f);
        }
        return;
    }
    circ[wv][0][lane] = cx;
    circ[wv][1][lane] = cy;
    circ[wv][2][lane] = R;
    circ[wv][3][lane] = k;
    circ[wv][4][lane] = z0;
    circ[wv][5][lane] = cot;
    circ[wv][6][lane] = st;
    wbits[wv][lane] = bits;
    woff[wv][lane] = o;
    if (lane == 63) woff[wv][64] = e;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // the wave's rows are [woff[0], woff[64]), non-decreasing offsets in between
    const int lo = woff[wv][0], hi = woff[wv][64];
    for (int r = lo + lane; r < hi; r += 64) {
        int a = 0, b = 64;  // woff[a] <= r < woff[b]
        while (b - a > 1) {
            const int m = (a + b) >> 1;
            if (woff[wv][m] <= r)
                a = m;
            else
                b = m;
        }
        float *f = features + (size_t)(r - o0) * fstride;
        if (wbits[wv][a])
            f[0] = f[1] = f[2] = (float)nan;
        else
            hit_features(hits + (size_t)r * 3, circ[wv][0][a], circ[wv][1][a], circ[wv][2][a], circ[wv][3][a],
                         circ[wv][4][a], circ[wv][5][a], circ[wv][6][a], f);
    }
}

}  // namespace

extern "C" tf_status tf_seed_tracks(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                                    double b_tesla, double *seeds, float *features, int32_t feature_stride,
                                    int32_t *flags, hipStream_t stream) {
    if (n_tracks < 0 || n_hits < 0 || !(b_tesla > 0.0)) return TF_EINVAL;
    if (feature_stride == 0) feature_stride = 3;
    if (feature_stride < 3) return TF_EINVAL;
    if (n_tracks == 0) return TF_OK;
    if (!offsets || !seeds || (!hits && n_hits > 0)) return TF_EINVAL;
    const int blocks = (n_tracks + kSeedBlock - 1) / kSeedBlock;  // one wave per 64 tracks
    hipLaunchKernelGGL(tf_seed_kernel, dim3(blocks), dim3(kSeedBlock), 0, stream, hits, (long long)n_hits, offsets,
                       (int)n_tracks, b_tesla, seeds, features, (int)feature_stride, flags);
    return hipGetLastError() == hipSuccess ? TF_OK : TF_EHIP;
}
