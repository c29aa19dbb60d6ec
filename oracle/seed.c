/*
 * Plain fp64 CPU oracle of the analytic three-hit seed and of the per-hit
 * seed residual features (Sec. Method, "Analytic seed").  TEST INFRASTRUCTURE
 * ONLY: it exists to check the GPU library.  Only the test suite, the smoke
 * check and the benchmark's CPU-baseline leg may load or call it.  It shares
 * no code, header or table with the GPU library.
 *
 * Seed.  The circle through the first three hits (in the transverse plane) is
 * found with the conformal map of the paper: with the first hit as origin,
 * inversion w = p / |p|^2 sends circles through the origin to straight lines,
 * so the circle follows from the line through the two mapped hits.  Its
 * radius gives pT = kappa B R (B along +z), its turning direction the charge,
 * and the closest approach to the z axis the perigee (d0, phi).  The
 * transverse arc lengths of the hits from the perigee give cot(theta) (first
 * and third hit) and z0.
 *
 * Conventions (the same as the synthetic helices): the perigee point is
 * d0 * (-sin phi, cos phi), phi is the direction of motion there, the circle
 * centre is (d0 + R / k) * (-sin phi, cos phi) with k = +1 for
 * counter-clockwise motion seen from +z and k = -q.
 *
 * Features (one reading of the paper's text): for every hit, the seed helix
 * point H at the hit's turning angle (the circle point on the ray from the
 * centre through the hit), the residual hit - H expressed in the curvilinear
 * frame of the helix at H (U = z x T / |z x T|, V = T x U, T the unit
 * direction of motion), compressed as asinh(dU / 1 mm) and asinh(dV / 1 mm),
 * and the helix path length from the perigee to H in mm.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#define ORC_KAPPA 0.299792458 /* pT [GeV] = kappa * B [T] * R [m], unit charge */

/* Seed of one track from its first three hits p[0..8] = (x, y, z) x 3 in mm.
 * out = d0 [mm], z0 [mm], phi, theta, q/p [1/GeV].  Returns 0, or -1 if two
 * hits coincide in the transverse plane or the three are collinear (no
 * circle), in which case out is NaN. */
int orc_seed_from_points(const double *p, double b_tesla, double *out) {
    for (int i = 0; i < 5; ++i) out[i] = NAN;
    const double x1 = p[0], y1 = p[1], z1 = p[2];
    /* conformal map of hits 2 and 3 about hit 1 */
    double u[2], v[2];
    for (int j = 0; j < 2; ++j) {
        const double dx = p[3 * (j + 1)] - x1, dy = p[3 * (j + 1) + 1] - y1;
        const double r2 = dx * dx + dy * dy;
        if (r2 == 0.0) return -1;
        u[j] = dx / r2;
        v[j] = dy / r2;
    }
    /* circle through the origin with centre (a, b): x^2 + y^2 = 2 a x + 2 b y,
     * i.e. the line 2 a u + 2 b v = 1 through both mapped points */
    const double det = u[0] * v[1] - u[1] * v[0];
    if (det == 0.0) return -1;
    const double a = 0.5 * (v[1] - v[0]) / det;
    const double b = 0.5 * (u[0] - u[1]) / det;
    const double cx = x1 + a, cy = y1 + b;
    const double R = sqrt(a * a + b * b);
    /* turning direction from hit 1 -> 2 -> 3 */
    const double cross = (p[3] - x1) * (p[7] - p[4]) - (p[4] - y1) * (p[6] - p[3]);
    const double k = cross > 0.0 ? 1.0 : -1.0;
    /* perigee: the circle point closest to the z axis, on the line through
     * the centre and the origin */
    const double D = sqrt(cx * cx + cy * cy);
    const double d0 = k * (D - R);
    const double phi = atan2(-k * cx, k * cy);
    const double px = cx * (1.0 - R / D), py = cy * (1.0 - R / D);
    /* transverse arc length from the perigee to hits 1 and 3, in the sense
     * of motion */
    double s[2];
    for (int j = 0; j < 2; ++j) {
        const double hx = p[6 * j] - cx, hy = p[6 * j + 1] - cy;
        const double ax = px - cx, ay = py - cy;
        const double ang = atan2(ax * hy - ay * hx, ax * hx + ay * hy);
        s[j] = R * k * ang;
    }
    const double dz = p[8] - z1, ds = s[1] - s[0];
    const double theta = atan2(ds, dz);
    const double cot = dz / ds;
    const double z0 = z1 - s[0] * cot;
    const double pt = ORC_KAPPA * b_tesla * R * 1e-3;
    const double q = -k;
    out[0] = d0;
    out[1] = z0;
    out[2] = phi;
    out[3] = theta;
    out[4] = q * sin(theta) / pt;
    return 0;
}

/* Residual features of one hit (x, y, z) against a seed (d0, z0, phi, theta,
 * q/p): out = asinh(dU), asinh(dV), helix path length, per the definition in
 * the file header. */
void orc_seed_features_hit(const double *seed, double b_tesla, const double *hit, double *out) {
    const double d0 = seed[0], z0 = seed[1], phi = seed[2], theta = seed[3], qop = seed[4];
    const double st = sin(theta), ct = cos(theta);
    const double pt = fabs(st / qop);
    const double R = pt / (ORC_KAPPA * b_tesla) * 1e3;
    const double k = qop > 0.0 ? -1.0 : 1.0;
    const double nx = -sin(phi), ny = cos(phi);
    const double cx = (d0 + R / k) * nx, cy = (d0 + R / k) * ny;
    const double px = d0 * nx, py = d0 * ny;
    /* turning angle of the hit from the perigee, in the sense of motion */
    const double wx = hit[0] - cx, wy = hit[1] - cy;
    const double ax = px - cx, ay = py - cy;
    const double ang = k * atan2(ax * wy - ay * wx, ax * wx + ay * wy);
    const double s_t = R * ang;
    /* helix point H at that angle, and the unit direction of motion there */
    const double rho = sqrt(wx * wx + wy * wy);
    const double hx = cx + R * wx / rho, hy = cy + R * wy / rho;
    const double hz = z0 + s_t * ct / st;
    const double tx = k * (-(hy - cy) / R) * st, ty = k * ((hx - cx) / R) * st, tz = ct;
    /* curvilinear frame: U = z x T / |z x T|, V = T x U */
    const double zxt_x = -ty, zxt_y = tx, zxt_n = sqrt(tx * tx + ty * ty);
    const double Ux = zxt_x / zxt_n, Uy = zxt_y / zxt_n, Uz = 0.0;
    const double Vx = ty * Uz - tz * Uy, Vy = tz * Ux - tx * Uz, Vz = tx * Uy - ty * Ux;
    const double rx = hit[0] - hx, ry = hit[1] - hy, rz = hit[2] - hz;
    out[0] = asinh(rx * Ux + ry * Uy + rz * Uz);
    out[1] = asinh(rx * Vx + ry * Vy + rz * Vz);
    out[2] = s_t / st;
}

/* Packed batch: seeds [n_tracks][5]; if features is not NULL, features
 * [offsets[n_tracks] - offsets[0]][3] for the hit rows offsets[0].. (row r of
 * features belongs to hit row offsets[0] + r).  A track with fewer than three
 * hits, or no circle through its first three, gets NaN seeds and NaN
 * features.  Returns the number of such tracks, or -1 for bad arguments. */
long orc_seed_tracks(const float *hits, const int32_t *offsets, int32_t n_tracks, double b_tesla,
                     double *seeds, double *features) {
    if (n_tracks < 0 || (n_tracks > 0 && (!hits || !offsets || !seeds))) return -1;
    long bad = 0;
    const int32_t base = n_tracks > 0 ? offsets[0] : 0;
    for (int32_t i = 0; i < n_tracks; ++i) {
        const int32_t o = offsets[i], L = offsets[i + 1] - offsets[i];
        double *sd = seeds + (size_t)i * 5;
        int ok = -1;
        if (L >= 3) {
            double p[9];
            for (int j = 0; j < 9; ++j) p[j] = (double)hits[(size_t)o * 3 + j];
            ok = orc_seed_from_points(p, b_tesla, sd);
        } else {
            for (int j = 0; j < 5; ++j) sd[j] = NAN;
        }
        if (ok != 0) bad += 1;
        if (features) {
            for (int32_t h = 0; h < L; ++h) {
                double *f = features + (size_t)(o - base + h) * 3;
                if (ok != 0) {
                    f[0] = f[1] = f[2] = NAN;
                    continue;
                }
                const double hit[3] = {hits[(size_t)(o + h) * 3], hits[(size_t)(o + h) * 3 + 1],
                                       hits[(size_t)(o + h) * 3 + 2]};
                orc_seed_features_hit(sd, b_tesla, hit, f);
            }
        }
    }
    return bad;
}
