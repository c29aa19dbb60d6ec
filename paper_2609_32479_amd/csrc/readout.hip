// The paper's readout and decode on gfx950 (Sec. Encoder, last paragraph;
// Sec. Losses for the seven quantiles and their median; the seed-anchored
// output of Sec. Method).
//
// Per track, with z = [f; b] the last layer's forward state at the last hit
// and reverse state at the first hit (2d floats, from fit_tracks_states):
// y = g (.) z / rms(z); h = SiLU(W1 y + b1) with NH hidden units (the paper's
// head has 128); q = W2 h + b2 (35 values, seven quantiles at ascending levels
// for each of d0, z0, phi, theta, q/p); the point estimate of each parameter
// is its median quantile, the middle output q[7p + 3]; it is added to the
// fp64 seed (phi wrapped to [-pi, pi)), q/p through the seed's scale
// |q/p_seed| + 0.02/GeV.
//
// One wave per 32 tracks, both layers as matrix-core products with the
// tracks on the 32 columns: hid^T = W1' z^T with W1' = W1 diag(g) (the gain
// folded in on the host), then the per-track 1/rms scales the columns;
// q^T = W2 h^T takes the layer-1 accumulators as its B operand as they lie.
// The reduction order over k is free, so the host packs both weight matrices
// in the order in which the lanes hold their operands: lane (half s, column
// t) reads its track's half row z[t][s d ..] as consecutive float4s, and in
// layer 2 supplies the hidden units it holds.  The weights are read by every
// wave and stay in L2.
//
// Two number types: fp32 products (32x32x2) for the fp32 model; for the
// 16-bit models bf16 weights (W1 and W2 as given, exact for bf16-valued
// weights; the gain is applied to the fp32 activations instead of being
// folded in, which would round the products to 8 bits) against fp32
// activations split into a high and a low bf16 part (32x32x16, two products
// per k-step), which keeps the activations to about 16 significant bits.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "trackfit.h"

namespace {

typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(8))) float f32x8;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;

constexpr int kNq = 7;          // quantiles per parameter
constexpr int kNout = 35;       // outputs of the head
constexpr float kRoEps = 1e-6f; // RMSNorm epsilon
constexpr double kQopEps = 0.02;  // 1/GeV, scale floor of the q/p decode
constexpr double kPi = 3.14159265358979323846;
constexpr int kWaves = 4;
constexpr int kQStride = 37;    // LDS row stride of a track's 35 outputs (floats)
constexpr int kMaxHidden = 256; // hidden units of the head, at most (a multiple of 32)

__device__ __forceinline__ f32x16 mma(float a, float b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 mma16(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// v = hi + lo + O(2^-16 |v|), both parts bf16 (round to nearest even)
__device__ __forceinline__ void split16(const f32x8 v, bf16x8 &hi, bf16x8 &lo) {
    hi = __builtin_convertvector(v, bf16x8);
    lo = __builtin_convertvector(v - __builtin_convertvector(hi, f32x8), bf16x8);
}

// Layer 1 bias and SiLU on the accumulators (lane (s, c) holds unit
// 32 m + 8 (q/4) + 4 s + q%4 of track c), in place.
template <int MT>
__device__ __forceinline__ void bias_silu(f32x16 (&acc)[MT], float inv, const float *__restrict__ b1, int s) {
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const float v = fmaf(inv, acc[m][q], b1[32 * m + 8 * (q >> 2) + 4 * s + (q & 3)]);
            acc[m][q] = v / (1.0f + expf(-__builtin_amdgcn_fmed3f(v, -80.0f, 80.0f)));
        }
}

// Outputs to LDS, then the point estimates, decode and the optional quantile rows.  o[rb]
// holds rows 32 rb + 8 (q/4) + 4 s + q%4 of track c (rows past 34 unused).
__device__ __forceinline__ void finish(const f32x16 (&o)[2], const float *__restrict__ b2, float (*qs)[kQStride],
                                       int lane, int t0, int n, const double *__restrict__ seeds,
                                       float *__restrict__ quant, double *__restrict__ out) {
    const int s = lane >> 5, c = lane & 31;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int row = 32 * rb + 8 * (q >> 2) + 4 * s + (q & 3);
            if (row < kNout) qs[c][row] = o[rb][q] + b2[row];
        }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // point estimates (each parameter's median quantile, its middle output) and
    // decode: lane half 0 takes d0, z0, phi; half 1 theta, q/p
    const int t = t0 + c;
    if (t < n) {
        const float *qt = qs[c];
        const double *sd = seeds + (size_t)t * 5;
        double *op = out + (size_t)t * 5;
        for (int p = s ? 3 : 0; p < (s ? 5 : 3); ++p) {
            const double med = (double)qt[kNq * p + kNq / 2];
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
        for (int i = lane; i < rows * kNout; i += 64) qb[i] = qs[i / kNout][i % kNout];
    }
}

// fp32 head: A1 [d/4][MT][64] float4 (4 consecutive k-steps), A2 [MT][4][2][64] float4.
// MT: 32-unit blocks of the hidden layer; D: half the state width (a multiple of 8).
template <int MT>
__global__ __launch_bounds__(64 * kWaves) void tf_readout_kernel(const float *__restrict__ states, int n, int D,
                                                                 const double *__restrict__ seeds,
                                                                 const float4 *__restrict__ A1,
                                                                 const float *__restrict__ b1,
                                                                 const float4 *__restrict__ A2,
                                                                 const float *__restrict__ b2,
                                                                 float *__restrict__ quant, double *__restrict__ out) {
    __shared__ float qs[kWaves][32][kQStride];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int t0 = (blockIdx.x * kWaves + wv) * 32;
    if (t0 >= n) return;  // the whole wave
    const int s = lane >> 5, c = lane & 31;
    const int t = t0 + c;
    // columns past the batch repeat track t0 (in bounds); their results are dropped
    const float4 *zp = reinterpret_cast<const float4 *>(states + (size_t)(t < n ? t : t0) * (2 * D) + s * D);

    // layer 1: acc[m] = rows 32 m .. of W1' z^T, k-step ks of this lane half
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
    bias_silu<MT>(acc, 1.0f / sqrtf(ss * (1.0f / (2 * D)) + kRoEps), b1, s);

    // layer 2: o[rb] = rows 32 rb .. of W2 h^T, k-step (m, q) taking the lane's unit of acc[m][q]
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
    finish(o, b2, qs[wv], lane, t0, n, seeds, quant, out);
}

// 16-bit head: A1 [d/8][MT][64] bf16x8 (lane (s, i): W1 row 32 m + i, k = s d + 8 ks + e),
// A2 [MT][2][2][64] bf16x8 (k-step (m, qh): the lane's units of acc[m][8 qh .. 8 qh + 7]),
// gain [2d] fp32.
template <int MT>
__global__ __launch_bounds__(64 * kWaves) void tf_readout16_kernel(const float *__restrict__ states, int n, int D,
                                                                   const double *__restrict__ seeds,
                                                                   const bf16x8 *__restrict__ A1,
                                                                   const float *__restrict__ gain,
                                                                   const float *__restrict__ b1,
                                                                   const bf16x8 *__restrict__ A2,
                                                                   const float *__restrict__ b2,
                                                                   float *__restrict__ quant, double *__restrict__ out) {
    __shared__ float qs[kWaves][32][kQStride];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int t0 = (blockIdx.x * kWaves + wv) * 32;
    if (t0 >= n) return;  // the whole wave
    const int s = lane >> 5, c = lane & 31;
    const int t = t0 + c;
    const float4 *zp = reinterpret_cast<const float4 *>(states + (size_t)(t < n ? t : t0) * (2 * D) + s * D);
    const float4 *gp = reinterpret_cast<const float4 *>(gain + s * D);

    f32x16 acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int q = 0; q < 16; ++q) acc[m][q] = 0.f;
    float ss = 0.f;
#pragma unroll 2
    for (int ks = 0; ks < D / 8; ++ks) {
        const float4 z0 = zp[2 * ks], z1 = zp[2 * ks + 1];
        const float4 g0 = gp[2 * ks], g1 = gp[2 * ks + 1];
        bf16x8 a[MT];
#pragma unroll
        for (int m = 0; m < MT; ++m) a[m] = A1[(ks * MT + m) * 64 + lane];
        ss = fmaf(z0.x, z0.x, fmaf(z0.y, z0.y, fmaf(z0.z, z0.z, fmaf(z0.w, z0.w, ss))));
        ss = fmaf(z1.x, z1.x, fmaf(z1.y, z1.y, fmaf(z1.z, z1.z, fmaf(z1.w, z1.w, ss))));
        bf16x8 hi, lo;  // g (.) z, split
        split16((f32x8){g0.x * z0.x, g0.y * z0.y, g0.z * z0.z, g0.w * z0.w, g1.x * z1.x, g1.y * z1.y, g1.z * z1.z,
                        g1.w * z1.w},
                hi, lo);
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            acc[m] = mma16(a[m], hi, acc[m]);
            acc[m] = mma16(a[m], lo, acc[m]);
        }
    }
    ss += __shfl_xor(ss, 32);
    bias_silu<MT>(acc, 1.0f / sqrtf(ss * (1.0f / (2 * D)) + kRoEps), b1, s);

    f32x16 o[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int q = 0; q < 16; ++q) o[rb][q] = 0.f;
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int qh = 0; qh < 2; ++qh) {
            bf16x8 hi, lo;
            split16((f32x8){acc[m][8 * qh + 0], acc[m][8 * qh + 1], acc[m][8 * qh + 2], acc[m][8 * qh + 3],
                            acc[m][8 * qh + 4], acc[m][8 * qh + 5], acc[m][8 * qh + 6], acc[m][8 * qh + 7]},
                    hi, lo);
#pragma unroll
            for (int rb = 0; rb < 2; ++rb) {
                const bf16x8 a = A2[((m * 2 + qh) * 2 + rb) * 64 + lane];
                o[rb] = mma16(a, hi, o[rb]);
                o[rb] = mma16(a, lo, o[rb]);
            }
        }
    finish(o, b2, qs[wv], lane, t0, n, seeds, quant, out);
}

}  // namespace

struct tf_readout {
    int d = 0;
    int hidden = 0;
    bool half = false;       // 16-bit head (tf_readout16_kernel)
    char *dmem = nullptr;
    const void *A1 = nullptr;
    const float *b1 = nullptr;
    const void *A2 = nullptr;
    const float *b2 = nullptr;
    const float *gain = nullptr;  // [2d], 16-bit head only
};

namespace {

// float -> bf16 bits, round to nearest even (NaN stays a quiet NaN)
uint16_t bf16_bits(float x) {
    uint32_t u;
    std::memcpy(&u, &x, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

template <int MT>
void launch_mt(const tf_readout *h, dim3 grid, dim3 block, hipStream_t stream, const float *states, int n,
               const double *seeds, float *quant, double *out) {
    if (h->half)
        hipLaunchKernelGGL(tf_readout16_kernel<MT>, grid, block, 0, stream, states, n, h->d, seeds,
                           static_cast<const bf16x8 *>(h->A1), h->gain, h->b1, static_cast<const bf16x8 *>(h->A2),
                           h->b2, quant, out);
    else
        hipLaunchKernelGGL(tf_readout_kernel<MT>, grid, block, 0, stream, states, n, h->d, seeds,
                           static_cast<const float4 *>(h->A1), h->b1, static_cast<const float4 *>(h->A2), h->b2,
                           quant, out);
}

bool valid_dims(int d, int hidden) {
    return d >= 32 && d <= 256 && d % 32 == 0 && hidden >= 32 && hidden <= kMaxHidden && hidden % 32 == 0;
}

}  // namespace

extern "C" size_t tf_readout_blob_size(int32_t d, int32_t hidden) {
    if (d <= 0 || hidden <= 0) return 0;
    const size_t dd = (size_t)d, nh = (size_t)hidden;
    return 2 * dd + nh * 2 * dd + nh + kNout * nh + kNout;
}

extern "C" tf_status tf_readout_create(int32_t d, int32_t hidden, int32_t dtype, const float *host_blob,
                                       size_t n_floats, tf_readout **out) {
    if (!out) return TF_EINVAL;
    *out = nullptr;
    if (!host_blob || d <= 0 || hidden <= 0 || n_floats != tf_readout_blob_size(d, hidden)) return TF_EINVAL;
    if (dtype != TF_FP32 && dtype != TF_BF16 && dtype != TF_BF16_F16ACT) return TF_EINVAL;
    if (!valid_dims(d, hidden)) return TF_EUNSUPPORTED;
    const bool half = dtype != TF_FP32;
    const size_t dd = (size_t)d, nh = (size_t)hidden;
    const int MT = hidden / 32;
    const float *g = host_blob, *W1 = g + 2 * dd, *b1 = W1 + nh * 2 * dd, *W2 = b1 + nh, *b2 = W2 + kNout * nh;
    // W1 as lane (s, i) holds it: row 32 m + i, column s d + kk, where kk is the k-step's
    // position in the lane's half row, with the gain folded in for the fp32 head (the
    // 16-bit head applies it to the activations); W2 as lane (s, i) holds it: row 32 rb + i,
    // the hidden unit that the lane's accumulator slot carries
    auto w1 = [&](int m, int lane, int kk) {
        const size_t u = 32 * m + (lane & 31), k = (size_t)(lane >> 5) * dd + kk;
        return half ? W1[u * 2 * dd + k] : W1[u * 2 * dd + k] * g[k];
    };
    auto w2 = [&](int rb, int lane, int m, int q) {
        const int row = 32 * rb + (lane & 31);
        const size_t u = 32 * m + 8 * (q >> 2) + 4 * (lane >> 5) + (q & 3);
        return row < kNout ? W2[(size_t)row * nh + u] : 0.f;
    };
    const size_t esz = half ? 2 : 4;
    const size_t nA1 = nh * 2 * dd, nA2 = (size_t)MT * 2 * 16 * 64;  // elements (A2: 2 row blocks x 16 slots)
    const size_t oB1 = nA1 * esz, oA2 = oB1 + nh * 4, oB2 = oA2 + nA2 * esz, oG = oB2 + 64 * 4;
    const size_t total = oG + 2 * dd * 4;
    std::vector<char> hbuf;
    try {
        hbuf.assign(total, 0);
    } catch (const std::bad_alloc &) {
        return TF_ENOMEM;
    }
    char *hp = hbuf.data();
    if (half) {
        // A1 [d/8][MT][64][8]: k-step ks covers kk = 8 ks .. 8 ks + 7
        uint16_t *A1 = reinterpret_cast<uint16_t *>(hp);
        for (int ks = 0; ks < d / 8; ++ks)
            for (int m = 0; m < MT; ++m)
                for (int lane = 0; lane < 64; ++lane)
                    for (int e = 0; e < 8; ++e)
                        A1[(((size_t)ks * MT + m) * 64 + lane) * 8 + e] = bf16_bits(w1(m, lane, 8 * ks + e));
        // A2 [MT][2][2][64][8]: k-step (m, qh) takes accumulator slots 8 qh .. 8 qh + 7
        uint16_t *A2 = reinterpret_cast<uint16_t *>(hp + oA2);
        for (int m = 0; m < MT; ++m)
            for (int qh = 0; qh < 2; ++qh)
                for (int rb = 0; rb < 2; ++rb)
                    for (int lane = 0; lane < 64; ++lane)
                        for (int e = 0; e < 8; ++e)
                            A2[((((size_t)m * 2 + qh) * 2 + rb) * 64 + lane) * 8 + e] =
                                bf16_bits(w2(rb, lane, m, 8 * qh + e));
    } else {
        // A1 [d/4][MT][64][4]: four consecutive k-steps kk = 4 grp .. 4 grp + 3
        float *A1 = reinterpret_cast<float *>(hp);
        for (int grp = 0; grp < d / 4; ++grp)
            for (int m = 0; m < MT; ++m)
                for (int lane = 0; lane < 64; ++lane)
                    for (int e = 0; e < 4; ++e)
                        A1[(((size_t)grp * MT + m) * 64 + lane) * 4 + e] = w1(m, lane, 4 * grp + e);
        // A2 [MT][4][2][64][4]: k-steps (m, 4 qg .. 4 qg + 3)
        float *A2 = reinterpret_cast<float *>(hp + oA2);
        for (int m = 0; m < MT; ++m)
            for (int qg = 0; qg < 4; ++qg)
                for (int rb = 0; rb < 2; ++rb)
                    for (int lane = 0; lane < 64; ++lane)
                        for (int e = 0; e < 4; ++e)
                            A2[((((size_t)m * 4 + qg) * 2 + rb) * 64 + lane) * 4 + e] = w2(rb, lane, m, 4 * qg + e);
    }
    std::memcpy(hp + oB1, b1, nh * 4);
    std::memcpy(hp + oB2, b2, kNout * 4);
    std::memcpy(hp + oG, g, 2 * dd * 4);
    tf_readout *ro = new (std::nothrow) tf_readout;
    if (!ro) return TF_ENOMEM;
    if (hipMalloc((void **)&ro->dmem, total) != hipSuccess) {
        delete ro;
        return TF_ENOMEM;
    }
    if (hipMemcpy(ro->dmem, hp, total, hipMemcpyHostToDevice) != hipSuccess) {
        (void)hipFree(ro->dmem);
        delete ro;
        return TF_EHIP;
    }
    ro->d = d;
    ro->hidden = hidden;
    ro->half = half;
    ro->A1 = ro->dmem;
    ro->b1 = reinterpret_cast<const float *>(ro->dmem + oB1);
    ro->A2 = ro->dmem + oA2;
    ro->b2 = reinterpret_cast<const float *>(ro->dmem + oB2);
    ro->gain = reinterpret_cast<const float *>(ro->dmem + oG);
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
    if (!valid_dims(h->d, h->hidden)) return TF_EINVAL;
    const int nt = (int)n_tracks;
    switch (h->hidden / 32) {
        case 1: launch_mt<1>(h, grid, block, stream, states, nt, seeds, quantiles, out); break;
        case 2: launch_mt<2>(h, grid, block, stream, states, nt, seeds, quantiles, out); break;
        case 3: launch_mt<3>(h, grid, block, stream, states, nt, seeds, quantiles, out); break;
        case 4: launch_mt<4>(h, grid, block, stream, states, nt, seeds, quantiles, out); break;
        case 5: launch_mt<5>(h, grid, block, stream, states, nt, seeds, quantiles, out); break;
        case 6: launch_mt<6>(h, grid, block, stream, states, nt, seeds, quantiles, out); break;
        case 7: launch_mt<7>(h, grid, block, stream, states, nt, seeds, quantiles, out); break;
        case 8: launch_mt<8>(h, grid, block, stream, states, nt, seeds, quantiles, out); break;
        default: return TF_EINVAL;
    }
    return hipGetLastError() == hipSuccess ? TF_OK : TF_EHIP;
}
