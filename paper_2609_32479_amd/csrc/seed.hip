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
// Reads: a wave's rows are one contiguous range.  When it spans at most
// kSeedChunks x 64 rows (and the wave's offsets are in order), the wave reads
// it once, coalesced, into registers (lane l holds rows lo + 64 c + l), takes
// each track's first three hits from those registers by cross-lane moves, and
// computes the features from the same registers.  Otherwise each track lane
// reads its first three hits itself and the row pass reads the range again.
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
constexpr int kSeedWaves = 4;           // waves per workgroup
constexpr int kSeedBlock = 64 * kSeedWaves;
constexpr int kSeedTracks = 32;         // tracks per wave (lanes 0 .. kSeedTracks - 1)
constexpr int kSeedChunks = 8;          // 64-row chunks a wave keeps in registers

// Seed of one track from its first three hits h = (x1, y1, z1, x2, y2, z2,
// x3, y3, z3): the circle (centre, radius, sense k), z0, cot(theta) and
// sin(theta) for the features, and the perigee parameters to sd[0..4].  False
// when the three hits are collinear in the transverse plane.
struct SeedCircle {
    double cx = 0, cy = 0, R = 0, k = 0, z0 = 0, cot = 0, st = 0, ist = 0;  // ist = 1 / sin(theta)
};
__device__ __forceinline__ bool seed_from_hits(const double *h, double b_tesla, double *sd, SeedCircle &c) {
    const double x1 = h[0], y1 = h[1], z1 = h[2];
    const double bx = h[3] - x1, by = h[4] - y1;
    const double qx = h[6] - x1, qy = h[7] - y1, z3 = h[8];
    // centre relative to hit 1: equidistant from hits 1, 2 and 3
    const double det = 2.0 * (bx * qy - by * qx);
    if (det == 0.0) return false;
    const double b2 = bx * bx + by * by, q2 = qx * qx + qy * qy;
    const double ux = (qy * b2 - by * q2) / det, uy = (bx * q2 - qx * b2) / det;
    c.cx = x1 + ux;
    c.cy = y1 + uy;
    c.R = sqrt(ux * ux + uy * uy);
    c.k = det > 0.0 ? 1.0 : -1.0;
    const double cx = c.cx, cy = c.cy, R = c.R, k = c.k;
    const double D = sqrt(cx * cx + cy * cy);
    // turning angle from the perigee (direction -C from the centre) to a
    // point w = P - C, positive along the motion
    auto turn = [&](double wx, double wy) { return k * atan2(cy * wx - cx * wy, -(cx * wx + cy * wy)); };
    const double s1 = R * turn(x1 - cx, y1 - cy);
    const double s3 = R * turn(x1 + qx - cx, y1 + qy - cy);
    const double theta = atan2(s3 - s1, z3 - z1);
    c.cot = (z3 - z1) / (s3 - s1);
    c.z0 = z1 - s1 * c.cot;
    c.st = sin(theta);
    c.ist = 1.0 / c.st;
    sd[0] = k * (D - R);
    sd[1] = c.z0;
    sd[2] = atan2(-k * cx, k * cy);
    sd[3] = theta;
    sd[4] = -k * c.st / (kKappa * b_tesla * R * 1e-3);
    return true;
}

// Residual features of one hit against a circle (centre c, radius R, sense k)
// and the line z = z0 + s cot(theta) along its transverse arc s from the
// perigee (direction -C from the centre).
__device__ __forceinline__ void hit_features(float px, float py, float pz, double cx, double cy, double R, double k,
                                             double z0, double cot, double st, double ist, float *f) {
    const double wx = (double)px - cx, wy = (double)py - cy;
    const double rho = sqrt(wx * wx + wy * wy);
    const double s = R * k * atan2(cy * wx - cx * wy, -(cx * wx + cy * wy));
    const double du = -k * (rho - R);
    const double dv = st * ((double)pz - (z0 + s * cot));
    // the residuals need fp64 (they are differences of values a thousand times
    // larger); their compression and the path length are stored as float32
    // and evaluated in it
    f[0] = asinhf((float)du);
    f[1] = asinhf((float)dv);
    f[2] = (float)(s * ist);  // the path length s / sin(theta)
}

// One wave per kSeedTracks consecutive tracks: lane i seeds track t0 + i,
// then the wave walks the hit rows of its tracks one row per lane (coalesced).
// (32 tracks, about 450 rows at 14 hits a track, fit the 8 register chunks:
// fewer registers than 64 tracks in 16 chunks, and four waves per SIMD.)
__global__ __launch_bounds__(kSeedBlock) void tf_seed_kernel(const float *__restrict__ hits, long long n_hits,
                                                              const int *__restrict__ offsets, int n_tracks,
                                                              double b_tesla, double *__restrict__ seeds,
                                                              float *__restrict__ features, int fstride,
                                                              int *__restrict__ flags) {
    __shared__ double circ[kSeedWaves][8][64];  // cx, cy, R, k, z0, cot(theta), sin(theta), 1 / sin per track
    __shared__ int woff[kSeedWaves][65];        // the wave's track offsets
    __shared__ int wbits[kSeedWaves][64];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int t0 = (blockIdx.x * kSeedWaves + wv) * kSeedTracks;
    if (t0 >= n_tracks) return;  // the whole wave
    const int i = t0 + lane;
    const bool active = lane < kSeedTracks && i < n_tracks;
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
    // the wave's rows: [lo, hi) when its offsets are in order
    const bool wave_bad = __ballot(bits == TF_SEED_BAD_OFFSETS) != 0;
    const int lo = __builtin_amdgcn_readlane(o, 0), hi = __builtin_amdgcn_readlane(e, kSeedTracks - 1);
    const int nch = wave_bad ? 0 : (hi - lo + 63) >> 6;
    const bool in_regs = features && !wave_bad && nch <= kSeedChunks;
    float rx[kSeedChunks], ry[kSeedChunks], rz[kSeedChunks];
    double h[9] = {0, 0, 0, 0, 0, 0, 0, 0, 0};
    if (in_regs) {
        // one coalesced read of the rows; then the first three hits of this
        // lane's track from the lanes that hold them
        // (lanes past the last row read the last row again: no lane-dependent branch)
#pragma unroll
        for (int c = 0; c < kSeedChunks; ++c) {
            if (c < nch) {
                const int r = min(lo + 64 * c + lane, hi - 1);
                const float *p = hits + (size_t)r * 3;
                rx[c] = p[0];
                ry[c] = p[1];
                rz[c] = p[2];
            } else {
                rx[c] = ry[c] = rz[c] = 0.f;
            }
        }
        const int rel = o - lo;
        float g[9] = {0, 0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int c = 0; c < kSeedChunks; ++c) {
            if (c < nch) {
#pragma unroll
                for (int hk = 0; hk < 3; ++hk) {
                    const int qr = rel + hk - 64 * c;  // the hit's row in chunk c
                    const bool here = (unsigned)qr < 64u;
                    const float vx = __shfl(rx[c], qr & 63), vy = __shfl(ry[c], qr & 63), vz = __shfl(rz[c], qr & 63);
                    g[3 * hk] = here ? vx : g[3 * hk];
                    g[3 * hk + 1] = here ? vy : g[3 * hk + 1];
                    g[3 * hk + 2] = here ? vz : g[3 * hk + 2];
                }
            }
        }
#pragma unroll
        for (int u = 0; u < 9; ++u) h[u] = g[u];
    } else if (active && !bits) {
        const float *p = hits + (size_t)o * 3;
#pragma unroll
        for (int u = 0; u < 9; ++u) h[u] = p[u];
    }
    SeedCircle sc;
    if (active && !bits) {
        if (!seed_from_hits(h, b_tesla, seeds + (size_t)i * 5, sc)) bits = TF_SEED_NO_CIRCLE;
    }
    if (active && bits) {
        double *sd = seeds + (size_t)i * 5;
        for (int j = 0; j < 5; ++j) sd[j] = nan;
        if (flags) atomicOr(flags, bits);
    }
    if (!features) return;
    if (wave_bad) {
        // offsets out of order somewhere in this wave: every good track walks
        // its own rows
        if (bits == TF_SEED_BAD_OFFSETS) return;
        for (int hr = o; hr < e; ++hr) {
            float *f = features + (size_t)(hr - o0) * fstride;
            if (bits) {
                f[0] = f[1] = f[2] = (float)nan;
            } else {
                const float *p = hits + (size_t)hr * 3;
                hit_features(p[0], p[1], p[2], sc.cx, sc.cy, sc.R, sc.k, sc.z0, sc.cot, sc.st, sc.ist, f);
            }
        }
        return;
    }
    circ[wv][0][lane] = sc.cx;
    circ[wv][1][lane] = sc.cy;
    circ[wv][2][lane] = sc.R;
    circ[wv][3][lane] = sc.k;
    circ[wv][4][lane] = sc.z0;
    circ[wv][5][lane] = sc.cot;
    circ[wv][6][lane] = sc.st;
    circ[wv][7][lane] = sc.ist;
    wbits[wv][lane] = bits;
    woff[wv][lane] = o;
    if (lane == 63) woff[wv][64] = e;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // the features of row r (of [lo, hi); non-decreasing offsets in between),
    // its track found by bisection of the wave's offsets
    auto row_features = [&](int r, float px, float py, float pz) {
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
            hit_features(px, py, pz, circ[wv][0][a], circ[wv][1][a], circ[wv][2][a], circ[wv][3][a],
                         circ[wv][4][a], circ[wv][5][a], circ[wv][6][a], circ[wv][7][a], f);
    };
    if (in_regs) {
        // One copy of the feature code: chunk c's registers picked by selects.
        // The track of each lane's row: the tracks that start in the chunk, in
        // order (their starts read from the track lanes), each taking the rows
        // from its start on; a track without hits takes none, as the next one
        // starts at the same row.
        int a = 0, tn = 0;  // the track of the row before the chunk; the next track to start
#pragma unroll 1
        for (int c = 0; c < nch; ++c) {
            float px = rx[0], py = ry[0], pz = rz[0];
#pragma unroll
            for (int u = 1; u < kSeedChunks; ++u) {
                px = c == u ? rx[u] : px;
                py = c == u ? ry[u] : py;
                pz = c == u ? rz[u] : pz;
            }
            const int base = lo + 64 * c, r = base + lane;
            a = __builtin_amdgcn_readlane(a, 63);  // the track of row base - 1
            for (; tn < kSeedTracks; ++tn) {
                const int st = __builtin_amdgcn_readlane(o, tn);
                if (st >= base + 64) break;
                a = r >= st ? tn : a;
            }
            if (r < hi) {
                float *f = features + (size_t)(r - o0) * fstride;
                if (wbits[wv][a])
                    f[0] = f[1] = f[2] = (float)nan;
                else
                    hit_features(px, py, pz, circ[wv][0][a], circ[wv][1][a], circ[wv][2][a], circ[wv][3][a],
                                 circ[wv][4][a], circ[wv][5][a], circ[wv][6][a], circ[wv][7][a], f);
            }
        }
    } else {
        for (int r = lo + lane; r < hi; r += 64) {
            const float *p = hits + (size_t)r * 3;
            row_features(r, p[0], p[1], p[2]);
        }
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
    const int per_block = kSeedWaves * kSeedTracks;
    const int blocks = (n_tracks + per_block - 1) / per_block;  // one wave per kSeedTracks tracks
    hipLaunchKernelGGL(tf_seed_kernel, dim3(blocks), dim3(kSeedBlock), 0, stream, hits, (long long)n_hits, offsets,
                       (int)n_tracks, b_tesla, seeds, features, (int)feature_stride, flags);
    return hipGetLastError() == hipSuccess ? TF_OK : TF_EHIP;
}
