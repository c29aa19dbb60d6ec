// The paper's readout and decode on gfx950 (Sec. Encoder, last paragraph;
// Sec. Losses for the seven quantiles and their median; the seed-anchored
// output of Sec. Method).
//
// Per track, with z = [f; b] the last layer's forward state at the last hit
// and reverse state at the first hit (2d floats, from fit_tracks_states):
// y = g (.) z / rms(z); h = SiLU(W1 y + b1); q = W2 h + b2 (35 values, seven
// quantiles for each of d0, z0, phi, theta, q/p); the point estimate of each
// parameter is the median of its seven; it is added to the fp64 seed (phi
// wrapped to [-pi, pi)), q/p through the seed's scale |q/p_seed| + 0.02/GeV.
//
// One wave per 32 tracks, both layers as fp32 matrix-core products with the
// tracks on the 32 columns: hid^T = W1' z^T with W1' = W1 diag(g) (the gain
// folded in on the host), then the per-track 1/rms scales the columns;
// q^T = W2 h^T takes the layer-1 accumulators as its B operand as they lie.
// The reduction order over k is free, so the host packs both weight matrices
// in the order in which the lanes hold their operands: lane (half s, column
// t) reads its track's half row z[t][s d ..] as consecutive float4s, and in
// layer 2 supplies hidden unit 32 m + 8 (q/4) + 4 s + q%4 at k-step (m, q).
// The weights (d = 128: 160 KiB) are read by every wave and stay in L2.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <new>
#include <vector>

#include "trackfit.h"

namespace {

typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int kNq = 7;          // quantiles per parameter
constexpr int kNout = 35;       // outputs of the head
constexpr float kRoEps = 1e-6f; // RMSNorm epsilon
constexpr double kQopEps = 0.02;  // 1/GeV, scale floor of the q/p decode
constexpr double kPi = 3.14159265358979323846;
constexpr int kWaves = 4;
constexpr int kQStride = 37;    // LDS row stride of a track's 35 outputs (floats)

__device__ __forceinline__ f32x16 mma(float a, float b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// Median of seven: the value whose rank (ties broken by position) is 3; NaN if
// any of the seven is NaN.
__device__ __forceinline__ float median7(const float *v) {
    float med = 0.f;
    bool nan = false;
#pragma unroll
    for (int i = 0; i < kNq; ++i) {
        int rank = 0;
#pragma unroll
        for (int j = 0; j < kNq; ++j)
            if (j != i) rank += (v[j] < v[i] || (v[j] == v[i] && j < i)) ? 1 : 0;
        if (rank == kNq / 2) med = v[i];
        nan |= v[i] != v[i];
    }
    return nan ? __builtin_nanf("") : med;
}

template <int D>
__global__ __launch_bounds__(64 * kWaves) void tf_readout_kernel(const float *__restrict__ states, int n,
                                                                 const double *__restrict__ seeds,
                                                                 const float4 *__restrict__ A1,
                                                                 const float *__restrict__ b1,
                                                                 const float4 *__restrict__ A2,
                                                                 const float *__restrict__ b2,
                                                                 float *__restrict__ quant, double *__restrict__ out) {
    constexpr int MT = D / 32;  // 32-unit blocks of the hidden layer
    __shared__ float qs[kWaves][32][kQStride];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int t0 = (blockIdx.x * kWaves + wv) * 32;
    if (t0 >= n) return;  // the whole wave
    const int s = lane >> 5, c = lane & 31;
    const int t = t0 + c;
    const bool valid = t < n;
    // columns past the batch repeat track t0 (in bounds); their results are dropped
    const float4 *zp = reinterpret_cast<const float4 *>(states + (size_t)(valid ? t : t0) * (2 * D) + s * D);

    // ---- layer 1: acc[m] = rows 32 m .. of W1' z^T, k-step ks of this lane half
    // reading z[t][s d + ks]
    f32x16 acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[m][q] = 0.f;
    float ss = 0.f;
#pragma unroll 2
    for (int g = 0; g < D / 4; ++g) {
        const float4 z = zp[g];
        float4 a[MT];
#pragma unroll
        for (int m = 0; m < MT; ++m) a[m] = A1[(g * MT + m) * 64 + lane];
        ss = fmaf(z.x, z.x, fmaf(z.y, z.y, fmaf(z.z, z.z, fmaf(z.w, z.w, ss))));
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            acc[m] = mma(a[m].x, z.x, acc[m]);
            acc[m] = mma(a[m].y, z.y, acc[m]);
            acc[m] = mma(a[m].z, z.z, acc[m]);
            acc[m] = mma(a[m].w, z.w, acc[m]);
        }
    }
    ss += __shfl_xor(ss, 32);  // both halves of the track's row
    const float inv = 1.0f / sqrtf(ss * (1.0f / (2 * D)) + kRoEps);

    // ---- bias and SiLU: lane (s, c) holds unit 32 m + 8 (q/4) + 4 s + q%4 of track c
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const float v = fmaf(inv, acc[m][q], b1[32 * m + 8 * (q >> 2) + 4 * s + (q & 3)]);
            acc[m][q] = v / (1.0f + expf(-__builtin_amdgcn_fmed3f(v, -80.0f, 80.0f)));
        }

    // ---- layer 2: o[rb] = rows 32 rb .. of W2 h^T (rows 35 .. 63 are zero weights)
    f32x16 o[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int q = 0; q < 16; ++q) o[rb][q] = 0.f;
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int qg = 0; qg < 4; ++qg)
#pragma unroll
            for (int rb = 0; rb < 2; ++rb) {
                const float4 a = A2[((m * 4 + qg) * 2 + rb) * 64 + lane];
                o[rb] = mma(a.x, acc[m][4 * qg + 0], o[rb]);
                o[rb] = mma(a.y, acc[m][4 * qg + 1], o[rb]);
                o[rb] = mma(a.z, acc[m][4 * qg + 2], o[rb]);
                o[rb] = mma(a.w, acc[m][4 * qg + 3], o[rb]);
            }
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int row = 32 * rb + 8 * (q >> 2) + 4 * s + (q & 3);
            if (row < kNout) qs[wv][c][row] = o[rb][q] + b2[row];
        }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // ---- medians and decode: lane half 0 takes d0, z0, phi; half 1 theta, q/p
    if (valid) {
        const float *qt = qs[wv][c];
        const double *sd = seeds + (size_t)t * 5;
        double *op = out + (size_t)t * 5;
        for (int p = s ? 3 : 0; p < (s ? 5 : 3); ++p) {
            const double med = (double)median7(qt + kNq * p);
            const double seed = sd[p];
            double v;
            if (p == 2) {
                v = seed + med;
                v -= 2.0 * kPi * floor((v + kPi) / (2.0 * kPi));
            } else if (p == 4) {
                v = seed + med * (fabs(seed) + kQopEps);
            } else {
                v = seed + med;
            }
            op[p] = v;
        }
    }
    if (quant) {
        // the wave's block of rows is contiguous: consecutive lanes, consecutive floats
        const int rows = n - t0 < 32 ? n - t0 : 32;
        float *qb = quant + (size_t)t0 * kNout;
        for (int i = lane; i < rows * kNout; i += 64) qb[i] = qs[wv][i / kNout][i % kNout];
    }
}

}  // namespace

struct tf_readout {
    int d = 0;
    float *dmem = nullptr;
    const float4 *A1 = nullptr;
    const float *b1 = nullptr;
    const float4 *A2 = nullptr;
    const float *b2 = nullptr;
};

extern "C" size_t tf_readout_blob_size(int32_t d) {
    if (d <= 0) return 0;
    const size_t dd = (size_t)d;
    return 2 * dd + dd * 2 * dd + dd + kNout * dd + kNout;
}

extern "C" tf_status tf_readout_create(int32_t d, const float *host_blob, size_t n_floats, tf_readout **out) {
    if (!out) return TF_EINVAL;
    *out = nullptr;
    if (!host_blob || d <= 0 || n_floats != tf_readout_blob_size(d)) return TF_EINVAL;
    if (d != 32 && d != 64 && d != 128 && d != 256) return TF_EUNSUPPORTED;
    const size_t dd = (size_t)d;
    const int MT = d / 32;
    const float *g = host_blob, *W1 = g + 2 * dd, *b1 = W1 + dd * 2 * dd, *W2 = b1 + dd, *b2 = W2 + kNout * dd;
    // device layout: A1 [d/4][MT][64][4], b1 [d], A2 [MT][4][2][64][4], b2 [64]
    const size_t nA1 = dd * 2 * dd, nA2 = (size_t)MT * 4 * 2 * 64 * 4, total = nA1 + dd + nA2 + 64;
    std::vector<float> h;
    try {
        h.assign(total, 0.f);
    } catch (const std::bad_alloc &) {
        return TF_ENOMEM;
    }
    float *hA1 = h.data(), *hb1 = hA1 + nA1, *hA2 = hb1 + dd, *hb2 = hA2 + nA2;
    for (int grp = 0; grp < d / 4; ++grp)
        for (int m = 0; m < MT; ++m)
            for (int lane = 0; lane < 64; ++lane)
                for (int e = 0; e < 4; ++e) {
                    const size_t u = 32 * m + (lane & 31), k = (size_t)(lane >> 5) * dd + 4 * grp + e;
                    hA1[(((size_t)grp * MT + m) * 64 + lane) * 4 + e] = W1[u * 2 * dd + k] * g[k];
                }
    for (size_t u = 0; u < dd; ++u) hb1[u] = b1[u];
    for (int m = 0; m < MT; ++m)
        for (int qg = 0; qg < 4; ++qg)
            for (int rb = 0; rb < 2; ++rb)
                for (int lane = 0; lane < 64; ++lane)
                    for (int e = 0; e < 4; ++e) {
                        const int row = 32 * rb + (lane & 31);
                        const size_t u = 32 * m + 8 * qg + 4 * (lane >> 5) + e;
                        hA2[((((size_t)m * 4 + qg) * 2 + rb) * 64 + lane) * 4 + e] =
                            row < kNout ? W2[(size_t)row * dd + u] : 0.f;
                    }
    for (int r = 0; r < kNout; ++r) hb2[r] = b2[r];
    tf_readout *ro = new (std::nothrow) tf_readout;
    if (!ro) return TF_ENOMEM;
    if (hipMalloc((void **)&ro->dmem, total * sizeof(float)) != hipSuccess) {
        delete ro;
        return TF_ENOMEM;
    }
    if (hipMemcpy(ro->dmem, h.data(), total * sizeof(float), hipMemcpyHostToDevice) != hipSuccess) {
        (void)hipFree(ro->dmem);
        delete ro;
        return TF_EHIP;
    }
    ro->d = d;
    ro->A1 = reinterpret_cast<const float4 *>(ro->dmem);
    ro->b1 = ro->dmem + nA1;
    ro->A2 = reinterpret_cast<const float4 *>(ro->dmem + nA1 + dd);
    ro->b2 = ro->dmem + nA1 + dd + nA2;
    *out = ro;
    return TF_OK;
}

extern "C" void tf_readout_destroy(tf_readout *h) {
    if (!h) return;
    (void)hipDeviceSynchronize();
    (void)hipFree(h->dmem);
    delete h;
}

extern "C" tf_status tf_decode_tracks(const float *states, int32_t n_tracks, const double *seeds,
                                      const tf_readout *h, float *quantiles, double *out, hipStream_t stream) {
    if (!h || n_tracks < 0) return TF_EINVAL;
    if (n_tracks == 0) return TF_OK;
    if (!states || !seeds || !out) return TF_EINVAL;
    const int per_block = 32 * kWaves;
    const dim3 grid((unsigned)((n_tracks + per_block - 1) / per_block)), block(64 * kWaves);
    switch (h->d) {
        case 32:
            hipLaunchKernelGGL(tf_readout_kernel<32>, grid, block, 0, stream, states, (int)n_tracks, seeds, h->A1,
                               h->b1, h->A2, h->b2, quantiles, out);
            break;
        case 64:
            hipLaunchKernelGGL(tf_readout_kernel<64>, grid, block, 0, stream, states, (int)n_tracks, seeds, h->A1,
                               h->b1, h->A2, h->b2, quantiles, out);
            break;
        case 128:
            hipLaunchKernelGGL(tf_readout_kernel<128>, grid, block, 0, stream, states, (int)n_tracks, seeds, h->A1,
                               h->b1, h->A2, h->b2, quantiles, out);
            break;
        case 256:
            hipLaunchKernelGGL(tf_readout_kernel<256>, grid, block, 0, stream, states, (int)n_tracks, seeds, h->A1,
                               h->b1, h->A2, h->b2, quantiles, out);
            break;
        default: return TF_EINVAL;
    }
    return hipGetLastError() == hipSuccess ? TF_OK : TF_EHIP;
}
