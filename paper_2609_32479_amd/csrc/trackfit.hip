// trackfit: fused gfx950 (CDNA4) kernel for batched inference of the
// bidirectional gated linear recurrent track-fit encoder, and its C ABI.
//
// What is computed (paper: Sec. Method, Sec. Encoder, Eq. (2)): per track,
// min-max normalised hits -> 3->d embedding -> n_layers x [RMSNorm -> one
// projection to candidate x_t and gate pre-activation -> z_t = sigmoid ->
// forward and reverse scans of h_t = h_{t-1} + z_t (x_t - h_{t-1}) ->
// linear merge of both directions added to the residual stream] -> mean over
// the track's hits -> W2 SiLU(W1 p + b1) + b2.
//
// How (Sec. Kernel adaptation is prior art for another GPU; this is a design
// for CDNA4):
//  * One wave64 owns a tile of whole tracks: 32 hit slots (64 when tracks may
//    be longer than 32 hits), packed greedily from the unpadded batch.  The
//    residual stream of the tile (slots x d, fp32) stays in registers for all
//    layers; nothing but hits, offsets and the five outputs touches HBM.
//  * All waves of a workgroup walk the same sequence of weight "stages" (the
//    input and output projections of a 32-channel chunk, together or apart,
//    then the head) in lockstep.  Each stage is copied once per workgroup from
//    L2 straight into a ring of LDS slots (global_load_lds, up to three stages
//    ahead), so matrix-core operands come from LDS and the copies overlap the
//    compute.  Weights are stored in the device already in per-lane fragment
//    order, so every copy and every operand read is a contiguous 1 KiB per
//    wave.
//  * Projections run on 32x32 matrix cores: v_mfma_f32_32x32x16_{bf16,f16}
//    for the 16-bit modes, v_mfma_f32_32x32x2_f32 for the fp32 model.  The
//    residual stream is held transposed (channels on MFMA rows, hits on
//    columns), which is exactly the operand layout of the input projection,
//    so the norm output feeds the matrix core without any data movement.
//  * The input projection puts hits on MFMA rows.  Hit slots are assigned to
//    rows so that each lane's 16 accumulator rows per 32-hit tile are
//    consecutive hits of one of two streams (lanes 0-31: first half of the
//    tile, lanes 32-63: second half).  Both scans therefore run serially in
//    registers, one channel per lane; the one track that may straddle the two
//    streams is finished by a second pass from the true boundary states,
//    which reproduces an unsplit scan exactly, so every track sees the same
//    operations wherever it sits in a tile.
//  * Scan outputs go through a wave-private LDS buffer once per 32-channel
//    chunk (the only transpose), and the output projection for that chunk is
//    accumulated into the residual registers (K split over chunks).
//  * Mean pooling runs per 32-channel block through wave-private LDS; the head
//    is computed transposed (hidden units on rows), so its hidden layer feeds
//    the second head GEMM straight from the accumulators.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <type_traits>
#include <vector>

#include "common.h"
#include "internal.h"
#include "trackfit.h"

namespace {

// ---------------------------------------------------------------------------
// Compile-time shape of one kernel instance.
// ---------------------------------------------------------------------------
template <int D, int OP, int HT_, bool PAIR_ = false>
struct KCfg {
    static constexpr bool HALF = OP != OP_F32;
    static constexpr int HT = HT_;               // 32-hit tiles per wave tile
    static constexpr int CAP = 32 * HT;          // hit slots per wave tile
    static constexpr int SP = 16 * HT;           // positions per stream (2 streams)
    static constexpr int MAXTR = 16 * HT;        // tracks per wave tile (of its head)
    // PAIR: two waves hold one 64-row tile of up to 32 tracks between them (see
    // tile_row); each runs the head of 16 of its tracks
    static constexpr bool PAIR = PAIR_;
    static constexpr int TCAP = PAIR ? 64 : CAP;      // rows of a tile
    static constexpr int TMAXTR = PAIR ? 32 : MAXTR;  // tracks of a tile
    static constexpr int MT = D / 32;            // 32-channel blocks
    static constexpr int NCH = D / 32;           // chunks of the scan / output projection
    static constexpr int K = HALF ? 16 : 2;      // MFMA reduction depth
    static constexpr int KL = K / 2;             // operand values per lane per k-step
    static constexpr int KS1 = D / K;            // k-steps over d
    static constexpr int KS2 = 64 / K;           // k-steps over one chunk of [f; b]
    static constexpr int RPK = 16 / KL;          // k-steps per 16 accumulator rows
    static constexpr int KPB = 32 / K;           // k-steps per 32-channel block
    static constexpr int EB = HALF ? 2 : 4;      // operand element bytes
    static constexpr int FRAG = 64 * KL * EB;    // one wave-wide operand fragment
    // waves per workgroup (three per SIMD for the 16-bit d <= 128 kernels; two
    // where the registers of two waves fit: d = 256 with fp16 activations
    // (-26 % time per launch against one wave) and the fp32 d = 128 model
    // (-10 %); one for the rest)
    static constexpr int WAVES = (HALF && HT == 1 && D <= 128)                                   ? 12
                                 : (HT == 1 && ((OP == OP_F16 && D == 256) || (!HALF && D == 128))) ? 8
                                                                                                      : 4;
    // Three waves per SIMD leave 168 registers a wave, two 256.  Under that budget the
    // kernel re-derives lane-dependent values where they are used and defines
    // its per-tile register arrays on every path, so that nothing is held (or
    // spilled) across tiles.
    static constexpr bool TIGHT = WAVES > 4;
    // wave-private LDS: [f; b] buffer, aliased by the pooling scratch
    // [f; b] buffer: fp32 slot-major with a padded row; 16-bit channel-major
    // (row k = channel k of the chunk's [f; b], CAP slots, swizzled by fb_off)
    static constexpr int FBS = HALF ? CAP : 65;  // row stride of [f; b] (elements)
    static constexpr int STS = 33;               // row stride of the pooling scratch (floats)
    static constexpr int FB_BYTES = HALF ? (64 * CAP + (HT_ == 1 ? 64 : 0)) * EB : CAP * FBS * EB;
    static constexpr int POOL_BYTES = CAP * STS * 4 + MAXTR * STS * 4;
    static constexpr int WAVE_BYTES = round_up(cmax(FB_BYTES, POOL_BYTES), 16) + 4 * TMAXTR * 4;
    static constexpr int EMB_BYTES = D * 16;
    // PAIR: per wave pair, the two scan hand-over rows (64 floats each) and their flags
    static constexpr int PX_BYTES = PAIR ? (WAVES / 2) * (2 * 64 * 4 + 16) : 0;
    static constexpr int RING_BYTES = kLdsBytesMax - EMB_BYTES - WAVES * WAVE_BYTES - 16 - PX_BYTES;  // for the stage ring
    // Weight stages, all padded to STAGE bytes.  A chunk's input and output
    // projections share one stage (one barrier per chunk) when two such stages
    // fit in the ring; otherwise each has its own.
    static constexpr int G1_FR = 2 * KS1;        // candidate + gate fragments of a chunk
    static constexpr int G2_FR = MT * KS2;       // output-projection fragments of a chunk
    static constexpr int G1_BYTES = G1_FR * FRAG + 64 * 4;  // + bx[32], bg[32]
    static constexpr int G2_BYTES = G2_FR * FRAG + D * 4;   // + bout[D]
    static constexpr int MERGED_STAGE = round_up(round_up(G1_BYTES, 16) + G2_BYTES, kCopyBytes);
    // PIPE (16-bit, d <= 128): pipelined layers, where chunk c runs its input
    // projection and then its gate interleaved with the output projection of
    // chunk c - 1; merged, those two share a stage.
    static constexpr bool PIPE = HALF && D <= 128;
    static constexpr bool MERGE = RING_BYTES / MERGED_STAGE >= 2;
    static constexpr int STAGE = MERGE ? MERGED_STAGE : round_up(cmax(G1_BYTES, G2_BYTES), kCopyBytes);
    static constexpr int G2_OFF = MERGE ? round_up(G1_BYTES, 16) : 0;  // output projection in its stage
    static constexpr int KSPS_RAW = (STAGE - D * 4) / (MT * FRAG);   // head-1 k-steps per stage
    static constexpr int KSPS = (KSPS_RAW >= KS1 ? KS1 : KSPS_RAW / KPB * KPB);
    static constexpr int NH1 = KS1 / KSPS;       // head-1 stages
    // A tile of at most 16 tracks runs the head on 16x16x32 products (16
    // track columns; the 16-bit modes), otherwise on 32x32 ones.
    static constexpr bool HEAD16 = HALF && MAXTR <= 16;
    static constexpr int UB = D / 16;            // 16-unit blocks of the head's hidden layer
    static constexpr int COPIES = STAGE / kCopyBytes;
    static constexpr int LPW = (COPIES + WAVES - 1) / WAVES;  // copies per wave per stage
    // workgroup LDS: embedding table, a ring of stage slots, wave regions.  The
    // ring is as deep as LDS allows (at most 4 slots): stages s + 1 ..
    // s + NSLOT - 1 are resident or in flight while stage s is computed.
    static constexpr int SLOT0 = EMB_BYTES;
    static constexpr int NSLOT_FIT = RING_BYTES / STAGE;
    static constexpr int NSLOT = NSLOT_FIT > 4 ? 4 : NSLOT_FIT;
    static_assert(NSLOT >= 2, "stage ring");
    static constexpr int WAVE0 = SLOT0 + NSLOT * STAGE;
    static constexpr int FLAG_OFF = WAVE0 + WAVES * WAVE_BYTES;  // the tile flag (see the kernel)
    static constexpr int PX_OFF = FLAG_OFF + 16;
    static constexpr int LDS_BYTES = PX_OFF + PX_BYTES;
    static_assert(!PAIR || (HT == 1 && PIPE && MERGE && HEAD16 && WAVES % 2 == 0), "paired tiles");
    static_assert(LDS_BYTES <= kLdsBytesMax, "LDS budget");
    static_assert(D % 32 == 0, "d must be a multiple of 32");
    static_assert(KSPS >= KPB && KS1 % KSPS == 0, "head stage split");
};

// Device-side weights.
struct DevParams {
    const float4 *emb;           // [D] (w_x, w_y, w_z, b) with the min-max map folded in; with
                                 // the Fourier front end: bias [D], lo [16], 1 / (hi - lo) [16]
    const unsigned char *stages; // n_stages x STAGE bytes, in the order the kernel walks them
    int n_layers;
    int n_stages;                // n_fstages + layer stages + NH1 + 1
    int n_feat;                  // per-hit features of the Fourier front end (0: x, y, z)
    int n_fstages;               // stages of the front end's dense projection
    int kpf;                     // k-steps of that projection per stage
};

constexpr int kMaxFeat = 16;     // per-hit features of the Fourier front end, at most
// What the encoder kernel writes: the pooled head's five outputs, the last
// layer's end states, or (with no layers) the front end's output per hit.
enum { OUT_HEAD = 0, OUT_STATES = 1, OUT_FRONT = 2 };
// Pipelined layers: bit g set = waves 4 g .. 4 g + 3 take each chunk's stage
// barrier after the chunk's scans instead of before them.
constexpr unsigned kLateWaveGroups = 1u;
// Polls of a paired wave's flag before it gives up (far beyond any real wait:
// each poll is an LDS read and the shortest sleep, which measured 0.6 %
// faster on 64-hit tracks than 64-cycle sleeps).
constexpr int kPairSpinLimit = 1 << 20;
constexpr int kUStride = 17;     // LDS row stride of a hit slot's normalised features (floats)

// The head multiplies fp32 vectors (pooled stream, hidden layer) by the
// weights: with bf16 operands each vector is split into a rounded high part
// and the rounded remainder, and both are multiplied (the weights are exact in
// the operand type), so the head keeps about 16 significant bits.  With fp16
// operands (11 significant bits, as the layers' activations) the 16x16 head
// takes each vector as one operand.
template <class F>
__device__ __forceinline__ void split_operand(const float *v, typename F::T &hi, typename F::T &lo);
// The 16x16 head's operand: fp16 alone (lo unused), else split.
template <int OP, class F>
__device__ __forceinline__ void head_operand(const float *v, typename F::T &hi, typename F::T &lo) {
    if constexpr (OP == OP_F16) {
        hi = F::pack(v);
        lo = hi;
    } else {
        split_operand<F>(v, hi, lo);
    }
}
template <class F>
__device__ __forceinline__ void split_operand(const float *v, typename F::T &hi, typename F::T &lo) {
    hi = F::pack(v);
    if constexpr (sizeof(typename F::E) == 2) {
        float r[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) r[u] = v[u] - (float)hi[u];
        lo = F::pack(r);
    } else {
        lo = hi;
    }
}

// fp32 [f; b] buffer (slot-major): positions p and p + 1 (p even) of one
// lane's scan outputs, rows = hit slots s and s + 1, column col0 + cc.
template <class C>
__device__ __forceinline__ void store_fb_pair(char *ws, int p, float v0, float v1, int col0, int hh, int cc) {
    float *fb = reinterpret_cast<float *>(ws) + col0 + cc;
    const int s = 32 * (p >> 4) + 8 * ((p >> 2) & 3) + 4 * hh + (p & 3);
    fb[s * C::FBS] = v0;
    fb[(s + 1) * C::FBS] = v1;
}

// 16-bit [f; b] buffer (channel-major): row k (channel k of the chunk's
// [f; b]) holds the CAP hit slots in 4-slot groups.  A scan lane owns one
// channel and stores four consecutive slots at once (8 bytes); the output
// projection reads its operand with the transposing LDS read, which hands each
// lane 4 channels of one slot from 4 slot-runs loaded by 4 lanes.  A store
// writes 32 rows at one slot group, a read 4 (2 for 64 slots) consecutive rows
// across a 32-slot tile; rows that share banks must then differ in the banks
// of their groups.  32 slots: row k starts 4 (k / 4) elements late (a skew,
// so a lane's rows and groups are a base plus constants); 64 slots: group g of
// row k sits at group g ^ swz(k).
template <class C> __device__ __forceinline__ int fb_row(int k) {
    return C::HT == 1 ? k * C::CAP + 4 * (k >> 2) : k * C::CAP;
}
template <class C> __device__ __forceinline__ int fb_off(int k, int grp) {
    if constexpr (C::HT == 1)
        return fb_row<C>(k) + 4 * grp;
    else
        return fb_row<C>(k) + 4 * (grp ^ ((((k >> 1) & 1) << 3) | ((k >> 2) & 7)));
}
// Positions p0 .. p0 + 3 (p0 a multiple of 4) of one lane's scan outputs,
// channel col: hit slots 4 grp .. 4 grp + 3.
template <class C, class E>
__device__ __forceinline__ void store_fb_quad(char *ws, int p0, float v0, float v1, float v2, float v3, int col,
                                              int hh) {
    typedef E e4 __attribute__((ext_vector_type(4)));
    typedef float f4 __attribute__((ext_vector_type(4)));
    const int grp = 8 * (p0 >> 4) + 2 * ((p0 >> 2) & 3) + hh;
    *reinterpret_cast<e4 *>(reinterpret_cast<E *>(ws) + fb_off<C>(col, grp)) =
        __builtin_convertvector((f4){v0, v1, v2, v3}, e4);
}
// The output projection's B operand for 32-slot tile nt and k-step kk: lane
// (hh, cc) receives channels 16 kk + 8 hh .. + 7 of slot 32 nt + cc.  As a
// loader it fetches the slot run 32 nt + 16 (cc / 16) + 4 (cc % 4) .. + 3 of
// channel 16 kk + 8 hh + 4 h + (cc / 4) % 4 for halves h = 0, 1.
template <class C, class T>
__device__ __forceinline__ T fb_tr_frag(const char *ws, int nt, int kk, int hh, int cc) {
    typedef short s4 __attribute__((ext_vector_type(4)));
    typedef short s8 __attribute__((ext_vector_type(8)));
    typedef __attribute__((address_space(3))) s4 lds_s4;
    const short *fb = reinterpret_cast<const short *>(ws);
    const int grp = 8 * nt + 4 * (cc >> 4) + (cc & 3);
    const int jj = (cc >> 2) & 3;
    int o0, o1;
    if constexpr (C::HT == 1) {
        // rows 16 kk + 8 hh + 4 h + jj all have k / 4 = 4 kk + 2 hh + h: one
        // lane base plus constants
        const int lb = (8 * hh + jj) * C::CAP + 8 * hh + 16 * (cc >> 4) + 4 * (cc & 3);
        o0 = lb + 16 * kk * C::CAP + 16 * kk + 32 * nt;
        o1 = o0 + 4 * C::CAP + 4;
    } else {
        const int k0 = 16 * kk + 8 * hh + jj;
        o0 = fb_off<C>(k0, grp);
        o1 = fb_off<C>(k0 + 4, grp);
    }
    const s4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)(fb + o0));
    const s4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4 *)(fb + o1));
    const s8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(T, v);
}

// Tile row of hit slot s (the wave's MFMA column order).  A wave tile holds
// its 32 rows in the folded order of slot_to_row.  A paired tile (64 rows)
// folds over both waves: wave 0 of the pair holds rows 0..15 (stream 0) and
// 63..48 (stream 1), wave 1 rows 16..31 and 47..32, so that each scan runs
// along a stream of wave 0, then one of wave 1, then the other stream of
// each in turn (the hand-over states pass through LDS).
template <class C> __device__ __forceinline__ int tile_row(int s, int pb) {
    if constexpr (C::PAIR) {
        const int p = 4 * ((s >> 3) & 3) + (s & 3);
        return ((s >> 2) & 1) ? (pb ? 47 : 63) - p : (pb ? 16 : 0) + p;
    } else {
        (void)pb;
        return slot_to_row<C::SP>(s);
    }
}
// A 64-bit tile-row mask as two 16-bit stream masks of wave pb of a pair, in
// register order: stream 0 rows base0 + p, stream 1 rows base1 - p.
__device__ __forceinline__ unsigned pair_s0(unsigned long long rows, int pb) {
    return unsigned(rows >> (pb ? 16 : 0)) & 0xffffu;
}
__device__ __forceinline__ unsigned pair_s1(unsigned long long rows, int pb) {
    return __builtin_bitreverse32(unsigned(rows >> (pb ? 32 : 48)) & 0xffffu) >> 16;
}

// STATES: instead of the pooled head, write each track's last-layer end states
// (the paper's own readout input): out is then [n_tracks][2d], the forward
// state at the track's last hit in columns 0..d-1 and the reverse state at its
// first hit in columns d..2d-1.  The last layer's output projection and the
// head, whose results nothing reads in this form, are skipped.
// OUT_FRONT (no layers): the front end's output per hit, as the next stage's
// matrix operand type (FE), row (hit row - offsets[0]) of out [out_rows][d],
// in channel order; rows of rejected tracks are not written.
// FOURIER: the paper's front end instead of the (x, y, z) embedding: hits holds
// n_feat features per hit, each min-max normalised in fp32 and expanded to
// sin and cos of pi 2^s u, s = 0..15, and the 32 n_feat values are projected
// to d on the matrix cores (the projection's weights stream through the stage
// ring ahead of the first layer's).  Column k of that projection is feature
// k / 32, cosine if bit 4 of k is set, scale k % 16.
template <int D, int OP, int HT_, int OUTM, bool FOURIER, bool PAIR = false>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * KCfg<D, OP, HT_, PAIR>::WAVES,
                                                      64 * KCfg<D, OP, HT_, PAIR>::WAVES),
                          amdgpu_waves_per_eu(KCfg<D, OP, HT_, PAIR>::WAVES / 4, KCfg<D, OP, HT_, PAIR>::WAVES / 4)))
void tf_encoder_kernel(const float *__restrict__ hits, long long n_hits_total, const int *__restrict__ offsets,
                       int n_tracks, DevParams P, float *__restrict__ out, long long out_rows, int *__restrict__ err) {
    constexpr bool STATES = OUTM == OUT_STATES;
    constexpr bool FRONT = OUTM == OUT_FRONT;
    using C = KCfg<D, OP, HT_, PAIR>;
    static_assert(!PAIR || OUTM == OUT_HEAD, "paired tiles: pooled head only");
    using F = Frag<OP>;
    using FT = typename F::T;
    using FE = typename F::E;
    constexpr int HT = C::HT, CAP = C::CAP, SP = C::SP, MT = C::MT, K = C::K, KL = C::KL;
    constexpr int KS1 = C::KS1, KS2 = C::KS2, RPK = C::RPK, KPB = C::KPB, NCH = C::NCH;
    constexpr int MAXTR = C::MAXTR, TMAXTR = C::TMAXTR;
    constexpr int OUTW = STATES ? 2 * D : 5;  // floats per output row (head, states)

    __shared__ __attribute__((aligned(16))) char smem[C::LDS_BYTES];
    const int lane = threadIdx.x & 63;
    const int wid = uniform(threadIdx.x >> 6);
    const float4 *emb = reinterpret_cast<const float4 *>(smem);
    char *ws = smem + C::WAVE0 + wid * C::WAVE_BYTES;
    float *stage = reinterpret_cast<float *>(ws);                           // [CAP][STS]
    float *pblk = stage + CAP * C::STS;                                     // [MAXTR][STS]
    // the tile's tracks: first tile row, length, first hit row, track index
    int *t_start = reinterpret_cast<int *>(ws + C::WAVE_BYTES - 4 * TMAXTR * 4);
    int *t_len = t_start + TMAXTR;
    int *t_off = t_len + TMAXTR;
    int *t_id = t_off + TMAXTR;
    // PAIR: the pairs are waves (w, w + 4) for w < 4, then (8, 9) and (10, 11):
    // the waves of a workgroup take the SIMDs in turn, so every SIMD holds both
    // places (a wave that waits for its partner leaves its SIMD to the partner
    // or to a wave of the other place).  pi: the pair; pb: this wave's place
    // (0 or 1); pw0: the wave in place 0.  The pair's hand-over rows (xab: place
    // 0 to 1, xba: back), their flags, and the chunk count the flags carry.
    static_assert(!C::PAIR || C::WAVES == 12, "pair layout");
    const int pi = C::PAIR ? (wid < 8 ? (wid & 3) : 4 + ((wid - 8) >> 1)) : 0;
    const int pb = C::PAIR ? (wid < 8 ? (wid >> 2) : (wid & 1)) : 0;
    const int pw0 = C::PAIR ? (wid < 8 ? (wid & 3) : (wid & ~1)) : wid;
    const int pw1 = C::PAIR ? (wid < 8 ? (wid & 3) + 4 : (wid | 1)) : wid;
    float *xab = reinterpret_cast<float *>(smem + C::PX_OFF + pi * (2 * 64 * 4 + 16));
    float *xba = xab + 64;
    int *fab = reinterpret_cast<int *>(xba + 64), *fba = fab + 1;
    int pseq = 0;

    const int hh = lane >> 5;  // lane half
    const int cc = lane & 31;  // lane column

    // embedding table to LDS; stages 0 .. NSLOT - 2 in flight
    for (int i = threadIdx.x; i < D; i += 64 * C::WAVES) reinterpret_cast<float4 *>(smem)[i] = P.emb[i];
    const int S = P.n_stages;
    auto slot_ptr = [&](int q) -> char * { return smem + C::SLOT0 + (q % C::NSLOT) * C::STAGE; };
    // LDS byte address of the slot of stage q
    const unsigned smem_lds = (unsigned)(uintptr_t)(__attribute__((address_space(3))) char *)smem;
    auto slot_lds = [&](int q) -> unsigned { return smem_lds + C::SLOT0 + (q % C::NSLOT) * C::STAGE; };
#pragma unroll
    for (int q = 0; q < C::NSLOT - 1; ++q) copy_stage<C>(P.stages, q % S, slot_lds(q), wid, lane);
    // The tile flag: at the start of its t-th tile every wave that has a tile
    // writes t, so the workgroup stops when after the barrier it does not read
    // t.  (No wave writes t + 1 before every wave has read it: each tile has
    // barriers of its own.)
    int *tile_flag = reinterpret_cast<int *>(smem + C::FLAG_OFF);
    if (threadIdx.x == 0) *tile_flag = 0;
    if constexpr (C::PAIR) {
        if (threadIdx.x < C::WAVES / 2) {
            int *f = reinterpret_cast<int *>(smem + C::PX_OFF + threadIdx.x * (2 * 64 * 4 + 16) + 2 * 64 * 4);
            f[0] = 0;
            f[1] = 0;
        }
    }
    lds_barrier();  // the flag and the embedding table are in place
    int tile_count = 0;

    // Stage q (counted across tiles; a tile iteration takes S stages) lives in
    // slot q % NSLOT.  At the end of stage q every wave waits for its share of
    // stage q + 1 (the loads of a wave complete in order, so this is a count of
    // the younger stage loads still allowed in flight), the barrier publishes
    // stage q + 1 and retires stage q, and stage q + NSLOT goes into the slot
    // of stage q.  The last stage of a tile waits for everything (its output
    // stores may complete out of order with the loads) and leaves the next
    // load to the start of the next tile, after that tile's own loads.
    int q = 0;
    int errbits = 0;
    auto advance = [&](bool last) {
        if (last)
            wait_vmcnt<0>();
        else
            wait_vmcnt<(C::NSLOT - 2) * C::LPW>();
        lds_barrier();
        if (!last) copy_stage<C>(P.stages, (q + C::NSLOT) % S, slot_lds(q + C::NSLOT), wid, lane);
        ++q;
    };
    auto slot = [&]() -> const char * { return slot_ptr(q); };
    // PAIR hand-over of scan states: a flag holds the number (pseq) of the chunk
    // whose row is in place.  A wait gives up after kPairSpinLimit polls
    // (TF_DEVERR_PAIR), and later waits are skipped, so that a fault here
    // cannot hang the GPU.
    bool pair_broken = false;
    auto pair_give = [&](float *buf, int *flag, float v) {
        buf[lane] = v;
        if (lane == 0) __hip_atomic_store(flag, pseq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    };
    auto pair_take = [&](const float *buf, int *flag) -> float {
        if (!pair_broken) {
            for (int spins = 0;; ++spins) {
                if (uniform(__hip_atomic_load(flag, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP)) == pseq) break;
                if (spins >= kPairSpinLimit) {
                    errbits |= TF_DEVERR_PAIR;
                    pair_broken = true;
                    break;
                }
                __builtin_amdgcn_s_sleep(0);
            }
        }
        return buf[lane];
    };

    // Contiguous group of tracks for this wave, balanced by hit rows.
    // (a pair shares one group)
    constexpr int GPB = C::PAIR ? C::WAVES / 2 : C::WAVES;  // groups per workgroup
    const long long gw = (long long)blockIdx.x * GPB + (C::PAIR ? pi : wid);
    const long long nw = (long long)gridDim.x * GPB;
    const int g_begin = group_begin(offsets, n_tracks, gw, nw, lane);
    const int g_end = group_begin(offsets, n_tracks, gw + 1, nw, lane);


    // Tiles are packed from a window of the wave's tracks: the first track not
    // yet fitted (t) and the WIN - 1 after it, in track order; bit i of `taken`
    // marks track t + i as fitted into an earlier tile (or refused).  The first
    // track of the window always goes in, so every tile makes progress, and a
    // track's result does not depend on the tile it lands in.
    constexpr int WIN = 32;
    int t = g_begin;
    unsigned taken = 0;
    for (;;) {
        int k = 0, n = 0;      // tracks and hit rows of the tile
        unsigned sel = 0;      // window tracks of the tile
        int off = 0, len = 0;  // lane i < WIN: first hit row and length of track t + i
        while (t < g_end) {
            // slide the window past its leading fitted tracks
            const int sh = taken == ~0u ? WIN : __builtin_ctz(~taken);
            taken = sh == WIN ? 0u : taken >> sh;
            t += sh;
            if (t >= g_end) break;
            const int idx = t + lane;
            off = 0;
            if (lane <= WIN && idx <= g_end) off = offsets[idx];
            const int nxt = __shfl_down(off, 1);
            len = nxt - off;
            const bool fresh = lane < WIN && idx < g_end && !((taken >> (lane & 31)) & 1u);
            // tracks that cannot be fitted: rows outside [0, n_hits), an end
            // before the start, no hits, or more hits than a tile holds
            const bool bad = off < 0 || nxt < off || (long long)nxt > n_hits_total;
            const bool empty = !bad && len == 0;
            const bool too_long = !bad && len > C::TCAP;
            const unsigned long long bad_m = __ballot(fresh && bad);
            const unsigned long long empty_m = __ballot(fresh && empty);
            const unsigned long long long_m = __ballot(fresh && too_long);
            if (bad_m | empty_m | long_m) {
                errbits |= (bad_m ? TF_DEVERR_BAD_OFFSETS : 0) | (empty_m ? TF_DEVERR_EMPTY_TRACK : 0) |
                           (long_m ? TF_DEVERR_TOO_LONG : 0);
                if (!FRONT && fresh && (bad || empty || too_long)) {
                    // (a NaN made here, so that the compiler does not keep one across tiles)
                    float qnan;
                    asm volatile("v_mov_b32 %0, 0x7fc00000" : "=v"(qnan));
#pragma unroll
                    for (int e = 0; e < OUTW; ++e) out[(size_t)idx * OUTW + e] = qnan;
                }
                taken |= unsigned(bad_m | empty_m | long_m);
            }
            // first-fit in window order (the pair search costs this kernel more per
            // tile than it saves)
            const unsigned cand = unsigned(__ballot(fresh && !bad && !empty && !too_long));
            if (cand) {
                sel = pack_tile<C::TCAP, TMAXTR, false>(cand, len, lane, n);
                k = __builtin_popcount(sel);
                taken |= sel;
                break;
            }
        }
        const bool work = k > 0;
        wait_vmcnt<0>();                     // stages q .. q + NSLOT - 2 are in LDS
        ++tile_count;
        if (work && lane == 0) *tile_flag = tile_count;
        lds_barrier();
        if (uniform(*tile_flag) != tile_count) break;  // every wave of the workgroup is done
        copy_stage<C>(P.stages, (q + C::NSLOT - 1) % S, slot_lds(q + C::NSLOT - 1), wid, lane);

        // ---- tile metadata: the tile's tracks in window order, on consecutive
        // tile rows; per stream, in register order (slot_to_row), the rows whose
        // coefficient the ascending pass zeroes (su0: track starts of stream 0,
        // forward; su1: track ends of stream 1, reverse) and the descending pass
        // zeroes (sd0: ends of stream 0; sd1: starts of stream 1).  The row after
        // the last hit counts as a start, so the padding never feeds a track.
        unsigned su0 = 0, su1 = 0, sd0 = 0, sd1 = 0;
        unsigned st0 = 0, st1 = 0;  // per stream, in row order: tile rows that start a track
        f32x16 r[MT][HT];  // the residual stream (a wave without a tile keeps zeros)
        if constexpr (C::TIGHT) {
#pragma unroll
            for (int m = 0; m < MT; ++m)
#pragma unroll
                for (int nt = 0; nt < HT; ++nt)
#pragma unroll
                    for (int q = 0; q < 16; ++q) r[m][nt][q] = 0.f;
        }
        if (work) {
            const int ln = C::TIGHT ? fresh_lane() : lane;
            const bool mine = ln < WIN && ((sel >> (ln & 31)) & 1u);
            const int v = mine ? len : 0;
            int incl = v;  // inclusive prefix sum of the selected lengths over lanes
#pragma unroll
            for (int d = 1; d < WIN; d <<= 1) {
                const int y = __shfl_up(incl, d);
                if (ln >= d) incl += y;
            }
            const int row0 = incl - v;
            if (mine) {
                const int j = __builtin_amdgcn_mbcnt_lo(sel, 0);  // selected tracks before this one
                t_start[j] = row0;
                t_len[j] = len;
                t_off[j] = off;
                t_id[j] = t + ln;
            }
            unsigned long long smask = 0;  // tile rows that start a track
            for (unsigned m = sel; m; m &= m - 1u) smask |= 1ull << __builtin_amdgcn_readlane(row0, __builtin_ctz(m));
            const unsigned long long valid = n >= 64 ? ~0ull : ((1ull << n) - 1);
            const unsigned long long vstart = smask | (n < 64 ? (1ull << n) : 0ull);
            const unsigned long long emask = ((smask >> 1) | (1ull << (n - 1))) & valid;
            const unsigned int spm = SP >= 32 ? 0xffffffffu : ((1u << SP) - 1);
            if constexpr (STATES || FRONT) {
                st0 = unsigned(smask) & spm;
                st1 = unsigned(smask >> SP) & spm;
            }
            if constexpr (C::PAIR) {
                su0 = pair_s0(vstart, pb);
                su1 = pair_s1(emask, pb);
                sd0 = pair_s0(emask, pb);
                sd1 = pair_s1(vstart, pb);
            } else {
                su0 = unsigned(vstart) & spm;
                su1 = stream1_bits<SP>(emask);
                sd0 = unsigned(emask) & spm;
                sd1 = stream1_bits<SP>(vstart);
            }
            wave_lds_sync();  // the track table is written

            if constexpr (!FOURIER) {
            // embedding: r[m][nt][q] = channel 32 m + 8 (q/4) + 4 hh + (q%4) of hit slot 32 nt + cc
#pragma unroll
            for (int nt = 0; nt < HT; ++nt) {
                const int th = tile_row<C>(32 * nt + ((C::TIGHT ? fresh_lane() : lane) & 31), pb);  // tile row
                float hx = 0.f, hy = 0.f, hz = 0.f;
                if (th < n) {
                    // the track holding tile row th, and the row's hit
                    const int j = __builtin_popcountll(smask & ((2ull << th) - 1ull)) - 1;
                    const float *hp = hits + ((size_t)t_off[j] + (th - t_start[j])) * 3;
                    hx = hp[0];
                    hy = hp[1];
                    hz = hp[2];
                }
#pragma unroll
                for (int m = 0; m < MT; ++m)
#pragma unroll
                    for (int q = 0; q < 16; ++q) {
                        const float4 e = emb[32 * m + 8 * (q >> 2) + 4 * hh + (q & 3)];
                        r[m][nt][q] = fmaf(e.x, hx, fmaf(e.y, hy, fmaf(e.z, hz, e.w)));
                    }
            }
            } else {
            // Fourier front end, part 1: the normalised features u = (x - lo) * (1 / (hi - lo))
            // (each step rounded to fp32) of hit slot 32 nt + cc to the wave's scratch, lane half
            // hh taking features 8 hh .. 8 hh + 7; r starts at the projection's bias
            const float *fe = reinterpret_cast<const float *>(smem);  // bias [D], lo [16], inv [16]
            float *us = stage;                                        // [CAP][kUStride]
            const int nf = P.n_feat;
#pragma unroll
            for (int nt = 0; nt < HT; ++nt) {
                const int ln = C::TIGHT ? fresh_lane() : lane;
                const int sl = 32 * nt + (ln & 31), h2 = ln >> 5;
                const int th = tile_row<C>(sl, pb);
                const float *hp = nullptr;
                if (th < n) {
                    const int j = __builtin_popcountll(smask & ((2ull << th) - 1ull)) - 1;
                    hp = hits + ((size_t)t_off[j] + (th - t_start[j])) * nf;
                }
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int f = 8 * h2 + e;
                    if (f < nf) us[sl * kUStride + f] = hp ? (hp[f] - fe[D + f]) * fe[D + kMaxFeat + f] : 0.f;
                }
#pragma unroll
                for (int m = 0; m < MT; ++m)
#pragma unroll
                    for (int q = 0; q < 16; ++q) r[m][nt][q] = fe[32 * m + 8 * (q >> 2) + 4 * h2 + (q & 3)];
            }
            wave_lds_sync();  // the features are in the scratch
            }
        }
        if constexpr (FOURIER) {
            // Fourier front end, part 2: k-step ks of the dense projection takes, for each
            // hit slot, the KL Fourier features k = ks K + hh KL + e (column k of the
            // projection), formed in registers: sin or cos of pi 2^s u_f
            const float *us = stage;
            const int kf = 32 * P.n_feat / K;  // k-steps of the projection
            FT cnext[HT];  // 16-bit: the cosines that the k-step after an even one takes
#pragma unroll
            for (int nt = 0; nt < HT; ++nt) cnext[nt] = FT{};
            for (int js = 0; js < P.n_fstages; ++js) {
                if (work) {
                    const FT *wfr = reinterpret_cast<const FT *>(slot());
                    const int k0 = js * P.kpf;
                    const int kn = kf - k0 < P.kpf ? kf - k0 : P.kpf;
                    __builtin_amdgcn_s_setprio(1);
                    for (int kl = 0; kl < kn; ++kl) {
                        const int ks = k0 + kl;
                        FT bv[HT];
#pragma unroll
                        for (int nt = 0; nt < HT; ++nt) {
                            const int sl = 32 * nt + cc;
                            float v[8];
                            if constexpr (C::HALF) {
                                // feature ks / 2, sines (even ks) or cosines (odd ks) of
                                // pi 2^s u at scales s = 8 hh + e.  The even k-step forms both:
                                // the lowest scale from the hardware functions, in revolutions
                                // (sin(pi 2^s u) = sin(2 pi frac(2^(s - 1) u)), the product by a
                                // power of two and the fraction exact), each next scale by the
                                // double-angle formulas, i.e. squaring the unit complex number
                                // c + i s.  An error doubles with each step, so the highest scale
                                // carries 2^7 times the hardware functions' error, far below the
                                // 16-bit operand's rounding.
                                if (ks & 1) {
                                    bv[nt] = cnext[nt];
                                    continue;
                                }
                                const float u = us[sl * kUStride + (ks >> 1)];
                                const float x = __builtin_amdgcn_fractf(u * (hh ? 128.0f : 0.5f));
                                float cv[8];
                                v[0] = __builtin_amdgcn_sinf(x);
                                cv[0] = __builtin_amdgcn_cosf(x);
#pragma unroll
                                for (int e = 1; e < 8; ++e) {
                                    const float sp = v[e - 1], cp = cv[e - 1];
                                    v[e] = (sp + sp) * cp;
                                    cv[e] = (cp - sp) * (cp + sp);
                                }
                                cnext[nt] = F::pack(cv);
                            } else {
                                // one feature per lane and k-step; the library's sinpi/cospi
                                // reduce the exact argument 2^s u exactly
                                const int k = ks * K + hh;
                                const float x = ldexpf(us[sl * kUStride + (k >> 5)], k & 15);
                                v[0] = ((k >> 4) & 1) ? cospif(x) : sinpif(x);
                            }
                            bv[nt] = F::pack(v);
                        }
#pragma unroll
                        for (int m = 0; m < MT; ++m) {
                            const FT a = wfr[(kl * MT + m) * 64 + lane];
#pragma unroll
                            for (int nt = 0; nt < HT; ++nt) r[m][nt] = F::mma(a, bv[nt], r[m][nt]);
                        }
                    }
                    __builtin_amdgcn_s_setprio(0);
                }
                advance(false);
            }
        }

        // ---- layers.  With STATES the last layer is a copy of its own (LAST): it
        // stops after the scans, so the residual is dead from its norm on.
        auto layer = [&](auto last_c) {
            constexpr bool LAST = decltype(last_c)::value;
            FT yf[HT][KS1];
            if constexpr (C::TIGHT) {
#pragma unroll
                for (int nt = 0; nt < HT; ++nt)
#pragma unroll
                    for (int ks = 0; ks < KS1; ++ks) yf[nt][ks] = FT{};
            }
            if (work) {
                // RMSNorm: each lane holds half the channels of hit slot 32 nt + cc
#pragma unroll
                for (int nt = 0; nt < HT; ++nt) {
                    float ss = 0.f;
#pragma unroll
                    for (int m = 0; m < MT; ++m)
#pragma unroll
                        for (int q = 0; q < 16; ++q) ss = fmaf(r[m][nt][q], r[m][nt][q], ss);
                    ss += __shfl_xor(ss, 32);
                    float rs;
                    if constexpr (C::HALF)
                        rs = rsqrtf(ss * (1.0f / D) + kRmsEps);
                    else
                        rs = 1.0f / sqrtf(ss * (1.0f / D) + kRmsEps);
#pragma unroll
                    for (int ks = 0; ks < KS1; ++ks) {
                        float v[8];
#pragma unroll
                        for (int u = 0; u < KL; ++u) v[u] = r[ks / RPK][nt][(ks % RPK) * KL + u] * rs;
                        yf[nt][ks] = F::pack(v);
                    }
                }
            }
            for (int ch = 0; ch < NCH; ++ch) {
                // ---- stage: input projection of channels 32 ch .. +31 (hits on rows),
                // gate, both scans, [f; b] to LDS
                if (work) {
                    const char *sl = slot();
                    const FT *wf = reinterpret_cast<const FT *>(sl);
                    const float *bias = reinterpret_cast<const float *>(sl + C::G1_FR * C::FRAG);
                    // candidate and gate pre-activation (zero accumulators cost no moves)
                    const float bxv = bias[cc];
                    const float bgv = bias[32 + cc];  // -log2(e) b in the 16-bit modes
                    f32x16 ax[HT], gx[HT];
#pragma unroll
                    for (int nt = 0; nt < HT; ++nt)
#pragma unroll
                        for (int q = 0; q < 16; ++q) {
                            ax[nt][q] = 0.f;
                            gx[nt][q] = 0.f;
                        }
                    // matrix-core phases run at raised wave priority, so that a wave
                    // entering one gets the SIMD's issue slots ahead of the vector work
                    // of the other waves
                    __builtin_amdgcn_s_setprio(1);
                    // gate first, so that its exponentials can overlap the candidate's products
#pragma unroll
                    for (int ks = 0; ks < KS1; ++ks) {
                        const FT bg = wf[(KS1 + ks) * 64 + lane];
#pragma unroll
                        for (int nt = 0; nt < HT; ++nt) gx[nt] = F::mma(yf[nt][ks], bg, gx[nt]);
                    }
#pragma unroll
                    for (int ks = 0; ks < KS1; ++ks) {
                        const FT bx = wf[ks * 64 + lane];
#pragma unroll
                        for (int nt = 0; nt < HT; ++nt) ax[nt] = F::mma(yf[nt][ks], bx, ax[nt]);
                    }
                    __builtin_amdgcn_s_setprio(0);
                    // gate a = sigmoid(g): the update adds a x and keeps cf = 1 - a of the state
                    float AX[HT * 16], CF[HT * 16];
#pragma unroll
                    for (int nt = 0; nt < HT; ++nt)
#pragma unroll
                        for (int q = 0; q < 16; ++q) {
                            const float g = gx[nt][q];
                            float a, cf;
                            if constexpr (C::HALF) {
                                // hardware exp2 and reciprocal; exp2 of a large argument is inf
                                // (a = 0, cf = 1) or 0 (a = 1, cf = 0)
                                const float e = __builtin_amdgcn_exp2f(fmaf(g, -kLog2e, bgv));
                                a = __builtin_amdgcn_rcpf(1.0f + e);
                                cf = 1.0f - a;
                            } else {
                                // library exp and correctly rounded division for the fp32 model
                                const float e = expf(-__builtin_amdgcn_fmed3f(g + bgv, -80.0f, 80.0f));
                                a = 1.0f / (1.0f + e);
                                cf = e * a;
                            }
                            AX[nt * 16 + q] = a * (ax[nt][q] + bxv);
                            CF[nt * 16 + q] = cf;
                        }
                    // Both scans of Eq. (2) in two passes over the lane's registers, in the
                    // folded row order (slot_to_row): the ascending pass runs stream 0
                    // forward and stream 1 in reverse, the descending pass stream 0 in
                    // reverse and stream 1 forward.  A track start (forward) or end
                    // (reverse) drops the carried state: its coefficient is zeroed in that
                    // stream's lanes.  The two passes meet at rows SP - 1 and SP: the
                    // descending pass starts from the other stream's last ascending state
                    // (one lane swap), so a track that straddles the streams is scanned in
                    // one unbroken sequence, exactly as any other.  (The asm hides the
                    // loop invariance that would otherwise keep every position's mask in
                    // scalar registers.)
                    unsigned mu0 = su0, mu1 = su1, md0 = sd0, md1 = sd1;
                    asm volatile("" : "+s"(mu0), "+s"(mu1), "+s"(md0), "+s"(md1));
                    constexpr int NP = HT * 16;  // register positions per stream
                    wave_lds_sync();  // the previous chunk's reads of the [f; b] buffer are done
                    if constexpr (!LAST) {
                        // ascending pass: stream 0 forward states to [f], stream 1 reverse
                        // states to [b]; descending pass the other way round.  Each pair of
                        // positions goes to the [f; b] buffer as soon as it is final.
                        float U[NP], Dn[NP];
                        float u = 0.f;
#pragma unroll
                        for (int i = 0; i < NP; ++i) {
                            u = fmaf(zero_lanes(CF[i], half_mask(mu0, mu1, i)), u, AX[i]);
                            U[i] = u;
                            if constexpr (C::HALF) {
                                if ((i & 3) == 3)
                                    store_fb_quad<C, FE>(ws, i - 3, U[i - 3], U[i - 2], U[i - 1], U[i], 32 * hh + cc, hh);
                            } else if (i & 1) {
                                store_fb_pair<C>(ws, i - 1, U[i - 1], U[i], 32 * hh, hh, cc);
                            }
                        }
                        const auto xs = __builtin_amdgcn_permlane32_swap(__float_as_uint(u), __float_as_uint(u),
                                                                         false, false);
                        float dn = __uint_as_float(hh ? xs[0] : xs[1]);  // the other stream's last state
#pragma unroll
                        for (int i = NP - 1; i >= 0; --i) {
                            dn = fmaf(zero_lanes(CF[i], half_mask(md0, md1, i)), dn, AX[i]);
                            Dn[i] = dn;
                            if constexpr (C::HALF) {
                                if ((i & 3) == 0)
                                    store_fb_quad<C, FE>(ws, i, Dn[i], Dn[i + 1], Dn[i + 2], Dn[i + 3], 32 - 32 * hh + cc,
                                                         hh);
                            } else if (!(i & 1)) {
                                store_fb_pair<C>(ws, i, Dn[i], Dn[i + 1], 32 - 32 * hh, hh, cc);
                            }
                        }
                    } else {
                        // Last layer, end states only, in fp32: the forward state at a
                        // track's last row goes to scratch row j (its index in the tile),
                        // the reverse state at its first row to row MAXTR + j; every other
                        // position writes a dummy row.  The track of a row is counted
                        // along each pass from the starts it crosses: per lane, cnt marks
                        // the starts in register order, put the positions to keep, jc the
                        // running track index (stepped by dj at each start before the
                        // position is stored) and base the scratch row of track 0.
                        // (The asm keeps the compiler from hoisting every position's row
                        // out of the chunk loop into registers.)
                        const unsigned s1 = stream1_bits<SP>((unsigned long long)st1 << SP);  // stream 1 starts
                        const unsigned e0 = sd0, e1 = su1;                                    // ends, per stream
                        constexpr int DUMMY = CAP * C::STS;  // first pooled row, unused here
                        auto pass = [&](float st, unsigned cnt, unsigned put, int dj, int jc, int base, bool up,
                                        unsigned m0, unsigned m1) -> float {
                            asm volatile("" : "+v"(cnt), "+v"(put), "+v"(dj), "+v"(jc), "+v"(base));
#pragma unroll
                            for (int ii = 0; ii < NP; ++ii) {
                                const int i = up ? ii : NP - 1 - ii;
                                st = fmaf(zero_lanes(CF[i], half_mask(m0, m1, i)), st, AX[i]);
                                jc += dj * int((cnt >> i) & 1u);
                                // (select written as a product, which stays branch-free)
                                stage[DUMMY + cc + int((put >> i) & 1u) * ((base + jc) * C::STS - DUMMY)] = st;
                                __builtin_amdgcn_sched_barrier(0);  // one position at a time
                            }
                            return st;
                        };
                        const int n0 = __builtin_popcount(st0);  // tracks that start in stream 0
                        // ascending: stream 0 forward (ends kept, rows j), stream 1 reverse
                        // (starts kept, rows MAXTR + j, counted down from k)
                        const float u = pass(0.f, hh ? s1 : st0, hh ? s1 : e0, hh ? -1 : 1, hh ? k : -1,
                                             hh ? MAXTR : 0, true, mu0, mu1);
                        const auto xs = __builtin_amdgcn_permlane32_swap(__float_as_uint(u), __float_as_uint(u),
                                                                         false, false);
                        // descending: stream 0 reverse (starts kept, counted down from n0),
                        // stream 1 forward (ends kept, counted up from n0 - 1)
                        (void)pass(__uint_as_float(hh ? xs[0] : xs[1]), hh ? s1 : st0, hh ? e1 : st0, hh ? 1 : -1,
                                   hh ? n0 - 1 : n0, hh ? 0 : MAXTR, false, md0, md1);
                        wave_lds_sync();
                        // rows of the tile's tracks out, f in the low lane half, b in the high
                        for (int j = 0; j < k; ++j)
                            out[(size_t)t_id[j] * OUTW + hh * D + 32 * ch + cc] = stage[(hh * MAXTR + j) * C::STS + cc];
                    }
                }
                if constexpr (!C::MERGE) advance(false);

                // ---- stage: output projection of this chunk, K split over chunks.  The
                // 16-bit modes accumulate straight into the residual registers; the
                // fp32 model sums the chunk in fresh accumulators and adds it once.
                if (work && !LAST) {
                    const char *sl = slot() + C::G2_OFF;
                    if constexpr (C::MERGE) wave_lds_sync();  // this wave's [f; b] stores are visible
                    __builtin_amdgcn_s_setprio(1);
                    const FT *wo = reinterpret_cast<const FT *>(sl);
                    f32x16 part[C::HALF ? 1 : MT][HT];
                    if constexpr (!C::HALF) {
#pragma unroll
                        for (int m = 0; m < MT; ++m)
#pragma unroll
                            for (int nt = 0; nt < HT; ++nt)
#pragma unroll
                                for (int q = 0; q < 16; ++q) part[m][nt][q] = 0.f;
                    }
#pragma unroll
                    for (int kk = 0; kk < KS2; ++kk) {
                        FT bfr[HT];
#pragma unroll
                        for (int nt = 0; nt < HT; ++nt) {
                            if constexpr (C::HALF) {
                                bfr[nt] = fb_tr_frag<C, FT>(ws, nt, kk, hh, cc);
                            } else {
                                const float *fb = reinterpret_cast<const float *>(ws);
                                bfr[nt] = fb[(32 * nt + cc) * C::FBS + kk * K + hh * KL];
                            }
                        }
#pragma unroll
                        for (int m = 0; m < MT; ++m) {
                            const FT a = wo[(m * KS2 + kk) * 64 + lane];
#pragma unroll
                            for (int nt = 0; nt < HT; ++nt) {
                                if constexpr (C::HALF)
                                    r[m][nt] = F::mma(a, bfr[nt], r[m][nt]);
                                else
                                    part[m][nt] = F::mma(a, bfr[nt], part[m][nt]);
                            }
                        }
                    }
                    if constexpr (!C::HALF) {
#pragma unroll
                        for (int m = 0; m < MT; ++m)
#pragma unroll
                            for (int nt = 0; nt < HT; ++nt) r[m][nt] += part[m][nt];
                    }
                    if (ch == NCH - 1) {
                        const float *bo = reinterpret_cast<const float *>(sl + C::G2_FR * C::FRAG);
#pragma unroll
                        for (int m = 0; m < MT; ++m)
#pragma unroll
                            for (int q = 0; q < 16; ++q) {
                                const float bv = bo[32 * m + 8 * (q >> 2) + 4 * hh + (q & 3)];
#pragma unroll
                                for (int nt = 0; nt < HT; ++nt) r[m][nt][q] += bv;
                            }
                    }
                }
                __builtin_amdgcn_s_setprio(0);
                advance(false);
            }
        };

        // ---- pipelined layers (PIPE).  Chunk ch runs its input projection, then its
        // gate interleaved with the output projection of chunk ch - 1, then its
        // scans: the output projection reads the [f; b] buffer before this chunk's
        // scans refill it, and its products go straight into the residual
        // registers.  A layer's last output projection runs at the start of the next
        // layer (before its norm) or after the last layer.  Merged, the stage of
        // IN(ch) also holds the output projection that runs with it (one barrier
        // per chunk); unmerged, the stages are IN(0), IN(1), OUT(0), IN(2), OUT(1),
        // ..., OUT(NCH - 1).
        // out_proj: r += W_out [f; b] of the chunk in the wave's buffer (fragments
        // at g2), plus b_out when the chunk is the layer's last.  The fp32 model sums
        // a chunk in fresh accumulators and adds it once (to keep within 1e-5).
        // (the lane argument: out_proj and out_bias, which run once per layer,
        // re-derive it (see KCfg::TIGHT))
        auto out_frag = [&](const char *g2, int m, int kk, int ln) -> FT {
            return reinterpret_cast<const FT *>(g2)[(m * KS2 + kk) * 64 + ln];
        };
        auto fb_frag = [&](int nt, int kk, int ln) -> FT {
            if constexpr (C::HALF) {
                return fb_tr_frag<C, FT>(ws, nt, kk, ln >> 5, ln & 31);
            } else {
                const float *fb = reinterpret_cast<const float *>(ws);
                return fb[(32 * nt + (ln & 31)) * C::FBS + kk * K + (ln >> 5) * KL];
            }
        };
        auto out_bias = [&](const char *g2) {
            const float *bo = reinterpret_cast<const float *>(g2 + C::G2_FR * C::FRAG);
            const int h2 = (C::TIGHT ? fresh_lane() : lane) >> 5;
#pragma unroll
            for (int m = 0; m < MT; ++m)
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const float bv = bo[32 * m + 8 * (q >> 2) + 4 * h2 + (q & 3)];
#pragma unroll
                    for (int nt = 0; nt < HT; ++nt) r[m][nt][q] += bv;
                }
        };
        auto out_proj = [&](const char *g2) {
            f32x16 part[C::HALF ? 1 : MT][HT];
            if constexpr (!C::HALF) {
#pragma unroll
                for (int m = 0; m < MT; ++m)
#pragma unroll
                    for (int nt = 0; nt < HT; ++nt)
#pragma unroll
                        for (int q = 0; q < 16; ++q) part[m][nt][q] = 0.f;
            }
            const int ln = C::TIGHT ? fresh_lane() : lane;
#pragma unroll
            for (int kk = 0; kk < KS2; ++kk) {
                FT bfr[HT];
#pragma unroll
                for (int nt = 0; nt < HT; ++nt) bfr[nt] = fb_frag(nt, kk, ln);
#pragma unroll
                for (int m = 0; m < MT; ++m) {
                    const FT a = out_frag(g2, m, kk, ln);
#pragma unroll
                    for (int nt = 0; nt < HT; ++nt) {
                        if constexpr (C::HALF)
                            r[m][nt] = F::mma(a, bfr[nt], r[m][nt]);
                        else
                            part[m][nt] = F::mma(a, bfr[nt], part[m][nt]);
                    }
                }
            }
            if constexpr (!C::HALF) {
#pragma unroll
                for (int m = 0; m < MT; ++m)
#pragma unroll
                    for (int nt = 0; nt < HT; ++nt) r[m][nt] += part[m][nt];
            }
        };
        auto layer_p = [&](auto last_c, bool prev_out) {
            constexpr bool LAST = decltype(last_c)::value;
            if (prev_out) {
                // the previous layer's last output projection (merged: in the stage
                // of this layer's first input projection)
                if (work) {
                    wave_lds_sync();  // this wave's [f; b] stores are visible
                    __builtin_amdgcn_s_setprio(1);
                    out_proj(slot() + C::G2_OFF);
                    __builtin_amdgcn_s_setprio(0);
                    out_bias(slot() + C::G2_OFF);
                }
                if constexpr (!C::MERGE) advance(false);
            }
            FT yf[HT][KS1];
            if constexpr (C::TIGHT) {
#pragma unroll
                for (int nt = 0; nt < HT; ++nt)
#pragma unroll
                    for (int ks = 0; ks < KS1; ++ks) yf[nt][ks] = FT{};
            }
            if (work) {
                // RMSNorm: each lane holds half the channels of hit slot 32 nt + cc
#pragma unroll
                for (int nt = 0; nt < HT; ++nt) {
                    float ss = 0.f;
#pragma unroll
                    for (int m = 0; m < MT; ++m)
#pragma unroll
                        for (int q = 0; q < 16; ++q) ss = fmaf(r[m][nt][q], r[m][nt][q], ss);
                    ss += __shfl_xor(ss, 32);
                    float rs;
                    if constexpr (C::HALF)
                        rs = rsqrtf(ss * (1.0f / D) + kRmsEps);
                    else
                        rs = 1.0f / sqrtf(ss * (1.0f / D) + kRmsEps);
#pragma unroll
                    for (int ks = 0; ks < KS1; ++ks) {
                        float v[8];
#pragma unroll
                        for (int u = 0; u < KL; ++u) v[u] = r[ks / RPK][nt][(ks % RPK) * KL + u] * rs;
                        yf[nt][ks] = F::pack(v);
                    }
                }
            }
            auto chunk = [&](auto with_out_c, int ch) {
                // chunk ch >= 1 also takes the stage of the output projection of chunk
                // ch - 1 (computed unless this is the end-states layer)
                constexpr bool HAS_OUT = decltype(with_out_c)::value;
                constexpr bool WO = HAS_OUT && !LAST;
                // candidate and gate pre-activation (zero accumulators cost no moves;
                // a wave without a tile keeps them)
                f32x16 ax[HT], gx[HT];
                float bxv = 0.f, bgv = 0.f;
#pragma unroll
                for (int nt = 0; nt < HT; ++nt)
#pragma unroll
                    for (int q = 0; q < 16; ++q) {
                        ax[nt][q] = 0.f;
                        gx[nt][q] = 0.f;
                    }
                if (work) {
                    const char *sl = slot();
                    const FT *wf = reinterpret_cast<const FT *>(sl);
                    const float *bias = reinterpret_cast<const float *>(sl + C::G1_FR * C::FRAG);
                    bxv = bias[cc];
                    bgv = bias[32 + cc];  // -log2(e) b in the 16-bit modes
                    // input projection: the gate's products first, so that the gate
                    // arithmetic can start while the candidate's are still running
                    __builtin_amdgcn_s_setprio(1);
#pragma unroll
                    for (int ks = 0; ks < KS1; ++ks) {
                        const FT bg = wf[(KS1 + ks) * 64 + lane];
#pragma unroll
                        for (int nt = 0; nt < HT; ++nt) gx[nt] = F::mma(yf[nt][ks], bg, gx[nt]);
                    }
#pragma unroll
                    for (int ks = 0; ks < KS1; ++ks) {
                        const FT bx = wf[ks * 64 + lane];
#pragma unroll
                        for (int nt = 0; nt < HT; ++nt) ax[nt] = F::mma(yf[nt][ks], bx, ax[nt]);
                    }
                    __builtin_amdgcn_s_setprio(0);
                }
                if constexpr (!C::MERGE) advance(false);  // the input projection's stage is read
                // gate a = sigmoid(g): the update adds a x and keeps cf = 1 - a of the state
                float AX[HT * 16], CF[HT * 16];
                if constexpr (C::TIGHT) {
#pragma unroll
                    for (int e = 0; e < HT * 16; ++e) AX[e] = CF[e] = 0.f;
                }
                if (work) {
                    auto gate = [&](int e) {
                        const float g = gx[e / 16][e % 16];
                        float a, cf;
                        if constexpr (C::HALF) {
                            // hardware exp2 and reciprocal; exp2 of a large argument is inf
                            // (a = 0, cf = 1) or 0 (a = 1, cf = 0)
                            const float ex = __builtin_amdgcn_exp2f(fmaf(g, -kLog2e, bgv));
                            a = __builtin_amdgcn_rcpf(1.0f + ex);
                            cf = 1.0f - a;
                        } else {
                            // library exp and correctly rounded division for the fp32 model
                            const float ex = expf(-__builtin_amdgcn_fmed3f(g + bgv, -80.0f, 80.0f));
                            a = 1.0f / (1.0f + ex);
                            cf = ex * a;
                        }
                        AX[e] = a * (ax[e / 16][e % 16] + bxv);
                        CF[e] = cf;
                    };
                    constexpr int NE = HT * 16;  // gate elements per lane
                    if constexpr (WO) {
                        // Interleaved with the previous chunk's output projection: step i
                        // issues product i (kk outer, then m, then nt) and a share of the
                        // gate elements; each step's operands are read one step ahead.  The
                        // fence after each step keeps this order (the wave issues in order,
                        // so a run of products would hold its vector work back).
                        constexpr int NMF = MT * KS2 * HT;
                        const char *g2 = slot() + C::G2_OFF;  // the output projection's fragments
                        f32x16 part[C::HALF ? 1 : MT][HT];
                        if constexpr (!C::HALF) {
#pragma unroll
                            for (int m = 0; m < MT; ++m)
#pragma unroll
                                for (int nt = 0; nt < HT; ++nt)
#pragma unroll
                                    for (int q = 0; q < 16; ++q) part[m][nt][q] = 0.f;
                        }
                        FT bcur[HT], bnxt[HT], acur, anxt;
                        if constexpr (C::MERGE) wave_lds_sync();  // this wave's [f; b] stores are visible
#pragma unroll
                        for (int nt = 0; nt < HT; ++nt) bcur[nt] = fb_frag(nt, 0, lane);
                        acur = out_frag(g2, 0, 0, lane);
#pragma unroll
                        for (int i = 0; i < NMF; ++i) {
                            const int kk = i / (MT * HT), m = (i / HT) % MT, nt = i % HT;
                            if (i + 1 < NMF) {
                                const int kk1 = (i + 1) / (MT * HT), m1 = ((i + 1) / HT) % MT;
                                anxt = out_frag(g2, m1, kk1, lane);
                                if (kk1 != kk) {
#pragma unroll
                                    for (int t = 0; t < HT; ++t) bnxt[t] = fb_frag(t, kk1, lane);
                                }
                            }
#pragma unroll
                            for (int e = i * NE / NMF; e < (i + 1) * NE / NMF; ++e) gate(e);
                            if constexpr (C::HALF)
                                r[m][nt] = F::mma(acur, bcur[nt], r[m][nt]);
                            else
                                part[m][nt] = F::mma(acur, bcur[nt], part[m][nt]);
                            __builtin_amdgcn_sched_barrier(0);
                            acur = anxt;
                            if (i + 1 < NMF && (i + 1) / (MT * HT) != kk) {
#pragma unroll
                                for (int t = 0; t < HT; ++t) bcur[t] = bnxt[t];
                            }
                        }
                        if constexpr (!C::HALF) {
#pragma unroll
                            for (int m = 0; m < MT; ++m)
#pragma unroll
                                for (int nt = 0; nt < HT; ++nt) r[m][nt] += part[m][nt];
                        }
                    } else {
#pragma unroll
                        for (int e = 0; e < NE; ++e) gate(e);
                    }
                }
                // the stage is read: the barrier comes before this chunk's scans, or
                // (late waves) after them
                const bool late = !C::PAIR && ((kLateWaveGroups >> (wid >> 2)) & 1);
                if constexpr (HAS_OUT || C::MERGE) {
                    if (!late) advance(false);
                }
                if (work) {
                    wave_lds_sync();  // the output projection's reads of the [f; b] buffer are done
                    unsigned mu0 = su0, mu1 = su1, md0 = sd0, md1 = sd1;
                    asm volatile("" : "+s"(mu0), "+s"(mu1), "+s"(md0), "+s"(md1));
                    constexpr int NP = HT * 16;  // register positions per stream
                    if constexpr (!LAST) {
                        // ascending pass: stream 0 forward states to [f], stream 1 reverse
                        // states to [b]; descending pass the other way round.  Each pair of
                        // positions goes to the [f; b] buffer as soon as it is final.
                        // PAIR: wave 1 starts from wave 0's ascending end states (the states
                        // at rows 15 and 48), and wave 0's descending pass from wave 1's
                        // descending end states (rows 16 and 47); each gives its row on.
                        float U[NP], Dn[NP];
                        float u = 0.f;
                        if constexpr (C::PAIR) {
                            ++pseq;
                            if (pb) u = pair_take(xab, fab);
                        }
#pragma unroll
                        for (int i = 0; i < NP; ++i) {
                            u = fmaf(zero_lanes(CF[i], half_mask(mu0, mu1, i)), u, AX[i]);
                            U[i] = u;
                            if constexpr (C::HALF) {
                                if ((i & 3) == 3)
                                    store_fb_quad<C, FE>(ws, i - 3, U[i - 3], U[i - 2], U[i - 1], U[i], 32 * hh + cc, hh);
                            } else if (i & 1) {
                                store_fb_pair<C>(ws, i - 1, U[i - 1], U[i], 32 * hh, hh, cc);
                            }
                        }
                        const auto xs = __builtin_amdgcn_permlane32_swap(__float_as_uint(u), __float_as_uint(u),
                                                                         false, false);
                        float dn = __uint_as_float(hh ? xs[0] : xs[1]);  // the other stream's last state
                        if constexpr (C::PAIR) {
                            if (!pb) {
                                pair_give(xab, fab, u);
                                dn = pair_take(xba, fba);
                            }
                        }
#pragma unroll
                        for (int i = NP - 1; i >= 0; --i) {
                            dn = fmaf(zero_lanes(CF[i], half_mask(md0, md1, i)), dn, AX[i]);
                            Dn[i] = dn;
                            if constexpr (C::HALF) {
                                if ((i & 3) == 0)
                                    store_fb_quad<C, FE>(ws, i, Dn[i], Dn[i + 1], Dn[i + 2], Dn[i + 3], 32 - 32 * hh + cc,
                                                         hh);
                            } else if (!(i & 1)) {
                                store_fb_pair<C>(ws, i, Dn[i], Dn[i + 1], 32 - 32 * hh, hh, cc);
                            }
                        }
                        if constexpr (C::PAIR) {
                            if (pb) pair_give(xba, fba, dn);
                        }
                    } else {
                        // Last layer, end states only, in fp32: the forward state at a
                        // track's last row goes to scratch row j (its index in the tile),
                        // the reverse state at its first row to row MAXTR + j; every other
                        // position writes a dummy row.  The track of a row is counted
                        // along each pass from the starts it crosses: per lane, cnt marks
                        // the starts in register order, put the positions to keep, jc the
                        // running track index (stepped by dj at each start before the
                        // position is stored) and base the scratch row of track 0.
                        // (The asm keeps the compiler from hoisting every position's row
                        // out of the chunk loop into registers.)
                        const unsigned s1 = stream1_bits<SP>((unsigned long long)st1 << SP);  // stream 1 starts
                        const unsigned e0 = sd0, e1 = su1;                                    // ends, per stream
                        constexpr int DUMMY = CAP * C::STS;  // first pooled row, unused here
                        auto pass = [&](float st, unsigned cnt, unsigned put, int dj, int jc, int base, bool up,
                                        unsigned m0, unsigned m1) -> float {
                            asm volatile("" : "+v"(cnt), "+v"(put), "+v"(dj), "+v"(jc), "+v"(base));
#pragma unroll
                            for (int ii = 0; ii < NP; ++ii) {
                                const int i = up ? ii : NP - 1 - ii;
                                st = fmaf(zero_lanes(CF[i], half_mask(m0, m1, i)), st, AX[i]);
                                jc += dj * int((cnt >> i) & 1u);
                                // (select written as a product, which stays branch-free)
                                stage[DUMMY + cc + int((put >> i) & 1u) * ((base + jc) * C::STS - DUMMY)] = st;
                                __builtin_amdgcn_sched_barrier(0);  // one position at a time
                            }
                            return st;
                        };
                        const int n0 = __builtin_popcount(st0);  // tracks that start in stream 0
                        // ascending: stream 0 forward (ends kept, rows j), stream 1 reverse
                        // (starts kept, rows MAXTR + j, counted down from k)
                        const float u = pass(0.f, hh ? s1 : st0, hh ? s1 : e0, hh ? -1 : 1, hh ? k : -1,
                                             hh ? MAXTR : 0, true, mu0, mu1);
                        const auto xs = __builtin_amdgcn_permlane32_swap(__float_as_uint(u), __float_as_uint(u),
                                                                         false, false);
                        // descending: stream 0 reverse (starts kept, counted down from n0),
                        // stream 1 forward (ends kept, counted up from n0 - 1)
                        (void)pass(__uint_as_float(hh ? xs[0] : xs[1]), hh ? s1 : st0, hh ? e1 : st0, hh ? 1 : -1,
                                   hh ? n0 - 1 : n0, hh ? 0 : MAXTR, false, md0, md1);
                        wave_lds_sync();
                        // rows of the tile's tracks out, f in the low lane half, b in the high
                        for (int j = 0; j < k; ++j)
                            out[(size_t)t_id[j] * OUTW + hh * D + 32 * ch + cc] = stage[(hh * MAXTR + j) * C::STS + cc];
                    }
                }
                if constexpr (HAS_OUT || C::MERGE) {
                    if (late) advance(false);
                }
            };
            chunk(std::false_type{}, 0);
            for (int ch = 1; ch < NCH; ++ch) chunk(std::true_type{}, ch);
        };

        if constexpr (STATES && C::PIPE) {
            for (int l = 0; l + 1 < P.n_layers; ++l) layer_p(std::false_type{}, l > 0);
            layer_p(std::true_type{}, P.n_layers > 1);
            advance(false);  // the last layer's last output projection, which the end states do not need
        } else if constexpr (STATES) {
            for (int l = 0; l + 1 < P.n_layers; ++l) layer(std::false_type{});
            layer(std::true_type{});
        } else if constexpr (FRONT) {
            // the front end's output of each hit: lane (hh, cc) holds channels
            // 32 m + 8 (q/4) + 4 hh + 0..3 of hit slot 32 nt + cc, four consecutive
            // channels per register quad
            if (work) {
                const int row0 = offsets[0];
                FE *xo = reinterpret_cast<FE *>(out);
#pragma unroll
                for (int nt = 0; nt < HT; ++nt) {
                    const int th = slot_to_row<SP>(32 * nt + cc);
                    if (th < n) {
                        // the track of tile row th: the number of track starts up to it, less one
                        const int j = (th < SP ? __builtin_popcount(st0 & ((2u << th) - 1u))
                                               : __builtin_popcount(st0) +
                                                     __builtin_popcount(st1 & ((2u << (th - SP)) - 1u))) - 1;
                        const long long row = (long long)t_off[j] + (th - t_start[j]) - row0;
                        if (row >= 0 && row < out_rows) {
                            FE *dst = xo + (size_t)row * D + 4 * hh;
#pragma unroll
                            for (int m = 0; m < MT; ++m)
#pragma unroll
                                for (int g = 0; g < 4; ++g) {
                                    typedef FE e4 __attribute__((ext_vector_type(4)));
                                    typedef float f4 __attribute__((ext_vector_type(4)));
                                    const f4 v = {r[m][nt][4 * g], r[m][nt][4 * g + 1], r[m][nt][4 * g + 2],
                                                  r[m][nt][4 * g + 3]};
                                    *reinterpret_cast<e4 *>(dst + 32 * m + 8 * g) = __builtin_convertvector(v, e4);
                                }
                        }
                    }
                }
            }
        } else if constexpr (C::PIPE) {
            for (int l = 0; l < P.n_layers; ++l) layer_p(std::false_type{}, l > 0);
            if (P.n_layers > 0) {
                // the last layer's last output projection
                if (work) {
                    wave_lds_sync();  // this wave's [f; b] stores are visible
                    __builtin_amdgcn_s_setprio(1);
                    out_proj(slot() + C::G2_OFF);
                    __builtin_amdgcn_s_setprio(0);
                    out_bias(slot() + C::G2_OFF);
                }
                advance(false);
            }
        } else {
            for (int l = 0; l < P.n_layers; ++l) layer(std::false_type{});
        }

        // ---- head, transposed: hid^T = W1 p^T (hidden units on rows, tracks on
        // columns), pooled 32 channels at a time through wave-private LDS
        {  // the head re-derives its lane values (see KCfg::TIGHT)
            const int lane = C::TIGHT ? fresh_lane() : int(threadIdx.x & 63);
            const int hh = lane >> 5, cc = lane & 31;
            f32x16 hid[C::HEAD16 ? 1 : MT];  // 32x32 head: units 32 m + 8 (q/4) + 4 hh + q%4 of track cc
            f32x4 hq[C::HEAD16 ? C::UB : 1];  // 16x16 head: units 16 ub + 4 hg + i of track hcol
            const int hcol = lane & 15, hg = lane >> 4;
            if constexpr (C::HEAD16) {
                // a zero made here, so that the compiler does not keep one across tiles
                float z;
                asm volatile("v_mov_b32 %0, 0" : "=v"(z));
#pragma unroll
                for (int ub = 0; ub < C::UB; ++ub)
#pragma unroll
                    for (int i = 0; i < 4; ++i) hq[ub][i] = z;
            } else {
#pragma unroll
                for (int m = 0; m < MT; ++m)
#pragma unroll
                    for (int q = 0; q < 16; ++q) hid[m][q] = 0.f;
            }
            const int prow = cc < MAXTR ? cc : MAXTR - 1;  // columns past the tile's tracks repeat the last
            const bool hw = work && OUTM == OUT_HEAD;  // rows to pool
            // this wave's head tracks: all of the tile's, or (PAIR) 16 pb .. 16 pb + 15;
            // a wave with none (the second of a pair whose tile holds at most 16
            // tracks) still stores its rows for its partner, then skips the head
            const int tr0 = C::PAIR ? 16 * pb : 0;
            const int tr1 = C::PAIR ? (k < tr0 + 16 ? k : tr0 + 16) : k;
            const bool hc = hw && tr1 > tr0;
            // unrolled, so that the residual block pooled at each step is a fixed register block
#pragma unroll
            for (int j = 0; j < C::NH1; ++j) {
                // (PAIR: a pair pools the rows of both its waves, so every wave takes
                // the workgroup barriers between writing and reading them)
                if (C::PAIR || hw) {
                    const FT *w1 = reinterpret_cast<const FT *>(slot());
#pragma unroll
                    for (int bl = 0; bl < C::KSPS / KPB; ++bl) {
                        const int m = j * (C::KSPS / KPB) + bl;  // channel block being pooled
                        // tile row th of the block goes to row th % 32 of the pooling
                        // scratch of wave th / 32 of the pair (PAIR), else of this wave
                        auto prow_of = [&](int th) -> float * {
                            if constexpr (C::PAIR)
                                return reinterpret_cast<float *>(smem + C::WAVE0 + (th < 32 ? pw0 : pw1) * C::WAVE_BYTES) +
                                       (th & 31) * C::STS;
                            else
                                return stage + th * C::STS;
                        };
                        if constexpr (C::PAIR)
                            lds_barrier();
                        else
                            wave_lds_sync();
                        if (hw) {
#pragma unroll
                            for (int nt = 0; nt < HT; ++nt) {
                                float *row = prow_of(tile_row<C>(32 * nt + cc, pb));
#pragma unroll
                                for (int q = 0; q < 16; ++q) row[8 * (q >> 2) + 4 * hh + (q & 3)] = r[m][nt][q];
                            }
                        }
                        if constexpr (C::PAIR)
                            lds_barrier();
                        else
                            wave_lds_sync();
                        if (!hc) continue;
                        for (int tr = tr0 + hh; tr < tr1; tr += 2) {
                            const int s0 = t_start[tr], len = t_len[tr];
                            // in order of u, eight independent reads at a time (rows past the
                            // track's end are read in bounds and not added)
                            float sum = 0.f;
                            for (int u0 = 0; u0 < len; u0 += 8) {
                                float v[8];
#pragma unroll
                                for (int i = 0; i < 8; ++i) v[i] = prow_of(s0 + (u0 + i < len ? u0 + i : len - 1))[cc];
#pragma unroll
                                for (int i = 0; i < 8; ++i)
                                    if (u0 + i < len) sum += v[i];
                            }
                            pblk[(tr - tr0) * C::STS + cc] = sum / (float)len;  // 0 / 0 = NaN for an empty track
                        }
                        wave_lds_sync();
                        if constexpr (C::HEAD16) {
                            // one 32-channel k-step: lane (hg, hcol) holds channels 8 hg .. + 7 of track hcol
                            float v[8];
#pragma unroll
                            for (int u = 0; u < 8; ++u) v[u] = pblk[hcol * C::STS + 8 * hg + u];
                            FT b_hi, b_lo;
                            head_operand<OP, F>(v, b_hi, b_lo);
#pragma unroll
                            for (int ub = 0; ub < C::UB; ++ub) {
                                const FT a = w1[(bl * C::UB + ub) * 64 + lane];
                                hq[ub] = F::mma16(a, b_hi, hq[ub]);
                                if constexpr (OP != OP_F16) hq[ub] = F::mma16(a, b_lo, hq[ub]);
                            }
                        } else {
#pragma unroll
                            for (int kb = 0; kb < KPB; ++kb) {
                                float v[8];
#pragma unroll
                                for (int u = 0; u < KL; ++u) v[u] = pblk[prow * C::STS + kb * K + hh * KL + u];
                                FT b_hi, b_lo;
                                split_operand<F>(v, b_hi, b_lo);
#pragma unroll
                                for (int mu = 0; mu < MT; ++mu) {
                                    const FT a = w1[((bl * KPB + kb) * MT + mu) * 64 + lane];
                                    hid[mu] = F::mma(a, b_hi, hid[mu]);
                                    if constexpr (C::HALF) hid[mu] = F::mma(a, b_lo, hid[mu]);
                                }
                            }
                        }
                    }
                    if constexpr (C::HEAD16) {
                      if (hc && j == C::NH1 - 1) {
                        // bias and SiLU: lane (hg, hcol) holds units 16 ub + 4 hg + i of track hcol
                        const float *b1 = reinterpret_cast<const float *>(slot() + C::KSPS * MT * C::FRAG);
#pragma unroll
                        for (int ub = 0; ub < C::UB; ++ub)
#pragma unroll
                            for (int i = 0; i < 4; ++i) {
                                const float v = hq[ub][i] + b1[16 * ub + 4 * hg + i];
                                hq[ub][i] = v * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(
                                                                      __builtin_amdgcn_fmed3f(-v * kLog2e, -kGateClamp, kGateClamp)));
                            }
                      }
                    } else if (hc && j == C::NH1 - 1) {
                        // bias and SiLU: lane (hh, cc) holds units 32 mu + 8 (q/4) + 4 hh + (q%4) of track cc
                        const float *b1 = reinterpret_cast<const float *>(slot() + C::KSPS * MT * C::FRAG);
#pragma unroll
                        for (int mu = 0; mu < MT; ++mu)
#pragma unroll
                            for (int q = 0; q < 16; ++q) {
                                const float v = hid[mu][q] + b1[32 * mu + 8 * (q >> 2) + 4 * hh + (q & 3)];
                                float sv;  // SiLU(v) = v / (1 + exp(-v))
                                if constexpr (C::HALF)
                                    sv = v * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(
                                                                          __builtin_amdgcn_fmed3f(-v * kLog2e, -kGateClamp, kGateClamp)));
                                else
                                    sv = v / (1.0f + expf(-__builtin_amdgcn_fmed3f(v, -80.0f, 80.0f)));
                                hid[mu][q] = sv;
                            }
                    }
                }
                advance(false);
            }
            // ---- head layer 2: out^T = W2 hid^T; the accumulators of hid^T are its B
            // operand, output row q of column cc is output q of track cc
            if constexpr (C::HEAD16) {
              if (hc) {
                // k-step kb takes the lane's units of blocks 2 kb and 2 kb + 1 (the
                // stored W2 fragments follow that order); output rows 4 hg + i
                const FT *w2 = reinterpret_cast<const FT *>(slot());
                const float *b2 = reinterpret_cast<const float *>(slot() + (D / 32) * C::FRAG);
                f32x4 o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kb = 0; kb < D / 32; ++kb) {
                    float v[8];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        v[i] = hq[2 * kb][i];
                        v[4 + i] = hq[2 * kb + 1][i];
                    }
                    FT b_hi, b_lo;
                    head_operand<OP, F>(v, b_hi, b_lo);
                    const FT a = w2[kb * 64 + lane];
                    o = F::mma16(a, b_hi, o);
                    if constexpr (OP != OP_F16) o = F::mma16(a, b_lo, o);
                }
                const int ht = (C::PAIR ? 16 * pb : 0) + hcol;  // the track of column hcol
                if (ht < k) {
                    float *op = out + (size_t)t_id[ht] * 5;
                    if (hg == 0) {
                        op[0] = o[0] + b2[0];
                        op[1] = o[1] + b2[1];
                        op[2] = o[2] + b2[2];
                        op[3] = o[3] + b2[3];
                    } else if (hg == 1) {
                        op[4] = o[0] + b2[4];
                    }
                }
              }
            } else if (hc) {
                const FT *w2 = reinterpret_cast<const FT *>(slot());
                const float *b2 = reinterpret_cast<const float *>(slot() + KS1 * C::FRAG);
                f32x16 o;
#pragma unroll
                for (int q = 0; q < 16; ++q) o[q] = 0.f;
#pragma unroll
                for (int ks = 0; ks < KS1; ++ks) {
                    float v[8];
#pragma unroll
                    for (int u = 0; u < KL; ++u) v[u] = hid[ks / RPK][(ks % RPK) * KL + u];
                    FT b_hi, b_lo;
                    split_operand<F>(v, b_hi, b_lo);
                    const FT a = w2[ks * 64 + lane];
                    o = F::mma(a, b_hi, o);
                    if constexpr (C::HALF) o = F::mma(a, b_lo, o);
                }
                if (cc < k) {
                    float *op = out + (size_t)t_id[cc] * 5;
                    if (hh == 0) {
                        op[0] = o[0] + b2[0];
                        op[1] = o[1] + b2[1];
                        op[2] = o[2] + b2[2];
                        op[3] = o[3] + b2[3];
                    } else {
                        op[4] = o[0] + b2[4];
                    }
                }
            }
        }
        advance(true);
    }
    if (errbits && lane == 0) atomicOr(err, errbits);
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

uint16_t to_bf16(double v) {
    float f = (float)v;
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return uint16_t((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

// Writer of one weight stage: operand elements in the kernel's operand type,
// biases in fp32.
struct StageWriter {
    int op;
    unsigned char *p;
    size_t o = 0;
    void elem(double v) {
        if (op == OP_BF16) {
            uint16_t b = to_bf16(v);
            std::memcpy(p + o, &b, 2);
            o += 2;
        } else if (op == OP_F16) {
            _Float16 h = (_Float16)(float)v;
            std::memcpy(p + o, &h, 2);
            o += 2;
        } else {
            f32(v);
        }
    }
    void f32(double v) {
        float f = (float)v;
        std::memcpy(p + o, &f, 4);
        o += 4;
    }
};

// Stage geometry of one instance, for the host.
struct Geom {
    int stage, ksps, nh1, merge, g2_off, head16, pipe;
};
template <int D, int OP, int HT, bool PAIR = false>
Geom geom() {
    using C = KCfg<D, OP, HT, PAIR>;
    return {C::STAGE, C::KSPS, C::NH1, C::MERGE ? 1 : 0, C::G2_OFF, C::HEAD16 ? 1 : 0, C::PIPE ? 1 : 0};
}
// 64-hit tracks: the 16-bit modes run the pooled head on paired tiles, and the
// end-states and front-end passes (which have no head) on 64-row wave tiles
// that walk the same stages.
template <int D, int OP>
constexpr bool same_stages() {
    using A = KCfg<D, OP, 2>;
    using B = KCfg<D, OP, 1, true>;
    return A::STAGE == B::STAGE && A::KSPS == B::KSPS && A::NH1 == B::NH1 && A::MERGE == B::MERGE &&
           A::G2_OFF == B::G2_OFF && A::PIPE == B::PIPE;
}
template <int D, int OP>
Geom geom_ht(int ht) {
    if constexpr (D <= 128) {
        if (ht == 2) {
            if constexpr (OP != OP_F32) {
                static_assert(same_stages<D, OP>(), "64-row and paired tiles walk the same stages");
                return geom<D, OP, 1, true>();
            } else {
                return geom<D, OP, 2>();
            }
        }
    }
    return geom<D, OP, 1>();
}
template <int OP>
Geom geom_d(int D, int ht) {
    switch (D) {
        case 32: return geom_ht<32, OP>(ht);
        case 64: return geom_ht<64, OP>(ht);
        case 128: return geom_ht<128, OP>(ht);
        default:
            if constexpr (OP != OP_F32) return geom_ht<256, OP>(ht);
            return geom_ht<128, OP>(ht);  // unreachable: fp32 d = 256 is refused
    }
}

}  // namespace

struct tf_weights {
    int n_layers = 0, d = 0, dtype = 0, max_hits = 0, device = 0, cu_count = 0, n_feat = 0;
    void *dmem = nullptr;
    int *err = nullptr;
    DevParams params{};
};

extern "C" size_t tf_blob_size(int32_t n_layers, int32_t d) {
    if (n_layers < 0 || d <= 0) return 0;
    size_t dd = (size_t)d;
    size_t per_layer = dd + 3 * dd * dd + 3 * dd + dd * 2 * dd + dd;
    return 4 * dd + (size_t)n_layers * per_layer + dd * dd + dd + 5 * dd + 5;
}

extern "C" size_t tf_fourier_blob_size(int32_t n_layers, int32_t d, int32_t n_features) {
    if (n_features <= 0 || n_features > kMaxFeat) return 0;
    const size_t base = tf_blob_size(n_layers, d);
    if (!base) return 0;
    const size_t dd = (size_t)d, F = (size_t)n_features;
    return base - 4 * dd + 2 * F + dd * 32 * F + dd;
}

extern "C" tf_status tf_weights_create(const tf_config *cfg, const float *blob, size_t n_floats,
                                       tf_weights **out) {
    if (!out) return TF_EINVAL;
    *out = nullptr;
    if (!cfg || !blob || cfg->max_hits < 0) return TF_EINVAL;
    const int L = cfg->n_layers, D = cfg->d_model;
    if (cfg->dtype != TF_FP32 && cfg->dtype != TF_BF16 && cfg->dtype != TF_BF16_F16ACT) return TF_EINVAL;
    if (L < 0 || D <= 0 || cfg->n_features < 0) return TF_EINVAL;
    if (!(D == 32 || D == 64 || D == 128 || D == 256) || L > 64) return TF_EUNSUPPORTED;
    const int NFEAT = cfg->n_features;
    if (NFEAT > kMaxFeat || (NFEAT > 0 && D != 32 && D != 128)) return TF_EUNSUPPORTED;
    if (n_floats != (NFEAT ? tf_fourier_blob_size(L, D, NFEAT) : tf_blob_size(L, D))) return TF_EINVAL;
    const int op = cfg->dtype == TF_BF16 ? OP_BF16 : cfg->dtype == TF_BF16_F16ACT ? OP_F16 : OP_F32;
    const bool half = op != OP_F32;
    if (!half && D > 128) return TF_EUNSUPPORTED;  // fp32 stages of d = 256 do not fit in LDS
    const int supported = D <= 128 ? 64 : 32;
    const int limit = cfg->max_hits == 0 ? supported : cfg->max_hits;
    if (limit > supported) return TF_EUNSUPPORTED;
    const int ht = limit <= 32 ? 1 : 2;
    const Geom G = op == OP_BF16 ? geom_d<OP_BF16>(D, ht) : op == OP_F16 ? geom_d<OP_F16>(D, ht) : geom_d<OP_F32>(D, ht);
    const int K = half ? 16 : 2, KL = K / 2, KS1 = D / K, KS2 = 64 / K, RPK = 16 / KL;
    const int MT = D / 32, NCH = D / 32;
    const double gs = half ? -1.4426950408889634 : 1.0;  // 16-bit modes evaluate exp2

    // blob views; the front end (x, y, z embedding, or the Fourier front end's
    // bounds, dense projection and bias) precedes the layers
    const size_t dd = (size_t)D;
    const float *eW = blob, *eb = blob + 3 * dd;
    const size_t KF32 = 32 * (size_t)NFEAT;  // Fourier features per hit
    const float *f_lo = blob, *f_hi = blob + NFEAT, *fW = blob + 2 * NFEAT, *fB = fW + dd * KF32;
    const size_t front = NFEAT ? 2 * (size_t)NFEAT + dd * KF32 + dd : 4 * dd;
    const size_t lstride = dd + 3 * dd * dd + 3 * dd + dd * 2 * dd + dd;
    auto g_of = [&](int l) { return blob + front + (size_t)l * lstride; };
    auto inW_of = [&](int l) { return g_of(l) + dd; };
    auto inb_of = [&](int l) { return inW_of(l) + 3 * dd * dd; };
    auto outW_of = [&](int l) { return inb_of(l) + 3 * dd; };
    auto outb_of = [&](int l) { return outW_of(l) + dd * 2 * dd; };
    const float *W1 = blob + front + (size_t)L * lstride;
    const float *b1 = W1 + dd * dd, *W2 = b1 + dd, *b2 = W2 + 5 * dd;

    // the Fourier front end's projection: KF k-steps of MT fragments, KPF per stage
    const int frag_bytes = 64 * KL * (half ? 2 : 4);
    const int KF = NFEAT ? (int)(KF32 / K) : 0;
    const int KPF = NFEAT ? std::min(KF, G.stage / (MT * frag_bytes)) : 1;
    const int NFS = NFEAT ? (KF + KPF - 1) / KPF : 0;
    // Layer stages.  Merged: a chunk's input and output projections share a
    // stage; otherwise each has a stage of its own, in chunk order.  Pipelined
    // kernels take them in the order they need them: merged, stage (l, c) holds
    // the input projection of chunk c of layer l and the output projection of the
    // chunk before it in walk order (chunk c - 1, or the previous layer's last
    // chunk), and one stage after the last layer holds that layer's last output
    // projection; unmerged, per layer IN(0), IN(1), OUT(0), IN(2), OUT(1), ...,
    // OUT(NCH - 1), the last taken at the start of the next layer.
    const int n_layer_stages =
        G.pipe ? (G.merge ? (L > 0 ? L * NCH + 1 : 0) : 2 * L * NCH) : (G.merge ? L * NCH : 2 * L * NCH);
    auto pipe_in = [&](int l, int c) {
        return G.merge ? NFS + NCH * l + c : NFS + 2 * NCH * l + (c == 0 ? 0 : 2 * c - 1);
    };
    auto pipe_out = [&](int l, int c) {
        return G.merge ? pipe_in(l, c) + 1 : NFS + 2 * NCH * l + (c < NCH - 1 ? 2 * c + 2 : 2 * NCH - 1);
    };
    const int n_stages = NFS + n_layer_stages + G.nh1 + 1;
    const size_t emb_bytes = (size_t)D * 16;
    const size_t emb_off = 0, st_off = (emb_bytes + 255) & ~size_t(255);
    const size_t err_off = st_off + (size_t)n_stages * G.stage;
    const size_t total = err_off + 256;
    std::vector<unsigned char> hb(total, 0);

    int s = 0;
    if (NFEAT) {
        // bias [D], lo [16], 1 / (hi - lo) [16] (fp32: the divisor and the quotient each
        // rounded to float32, as the kernel's normalisation takes them)
        StageWriter w{OP_F32, hb.data() + emb_off};
        for (int c = 0; c < D; ++c) w.f32(fB[c]);
        for (int f = 0; f < kMaxFeat; ++f) w.f32(f < NFEAT ? f_lo[f] : 0.0);
        for (int f = 0; f < kMaxFeat; ++f) {
            const float span = f < NFEAT ? f_hi[f] - f_lo[f] : 1.0f;
            const float inv = 1.0f / span;
            w.f32(inv);
        }
        // projection A fragments: lane (g, c) value e of k-step ks, block m holds
        // fe.W[channel 32 m + c][column ks K + g KL + e]
        for (int js = 0; js < NFS; ++js) {
            StageWriter ws{op, hb.data() + st_off + (size_t)s++ * G.stage};
            for (int kl = 0; kl < KPF && js * KPF + kl < KF; ++kl)
                for (int m = 0; m < MT; ++m)
                    for (int lane = 0; lane < 64; ++lane)
                        for (int e = 0; e < KL; ++e) {
                            const size_t col = (size_t)(js * KPF + kl) * K + (lane / 32) * KL + e;
                            ws.elem(fW[(size_t)(32 * m + lane % 32) * KF32 + col]);
                        }
        }
    } else {
        // embedding with u = (x - lo) / span folded in: r = (W/span) x + (b - W lo / span)
        StageWriter w{OP_F32, hb.data() + emb_off};
        const double lo[3] = {-1000.0, -1000.0, -3000.0}, span[3] = {2000.0, 2000.0, 6000.0};
        for (int c = 0; c < D; ++c) {
            double b = eb[c];
            for (int k = 0; k < 3; ++k) {
                w.f32(eW[c * 3 + k] / span[k]);
                b -= eW[c * 3 + k] * lo[k] / span[k];
            }
            w.f32(b);
        }
    }
    for (int l = 0; l < L; ++l) {
        const float *Wi = inW_of(l), *g = g_of(l), *bi = inb_of(l), *Wo = outW_of(l), *bo = outb_of(l);
        for (int ch = 0; ch < NCH; ++ch) {
            // input projection B fragments: lane (g, c) value u of k-step ks holds
            // W[out 32 ch + c][in 32 m + 8 i + 4 g + j] * gain[in], with
            // (m, 4 i + j) = (ks / RPK, (ks % RPK) * KL + u); then bx[32], bg[32]
            const int s_in = G.pipe ? pipe_in(l, ch) : s++;
            StageWriter w{op, hb.data() + st_off + (size_t)s_in * G.stage};
            for (int part = 0; part < 2; ++part)
                for (int ks = 0; ks < KS1; ++ks)
                    for (int lane = 0; lane < 64; ++lane)
                        for (int u = 0; u < KL; ++u) {
                            const int gg = lane / 32, c = lane % 32;
                            const int reg = (ks % RPK) * KL + u, m = ks / RPK;
                            const int in = 32 * m + 8 * (reg / 4) + 4 * gg + (reg % 4);
                            const int row = part * D + 32 * ch + c;
                            w.elem((double)Wi[(size_t)row * D + in] * g[in]);
                        }
            for (int c = 0; c < 32; ++c) w.f32(bi[32 * ch + c]);
            for (int c = 0; c < 32; ++c) w.f32(gs * bi[D + 32 * ch + c]);
            // output projection A fragments: lane (g, c) value u of k-step kk of
            // block m holds W[out 32 m + c][column of [f; b] channel
            // q = kk K + g KL + u of the chunk]; then bout[D]
            // (merged: at g2_off in the stage of the input projection)
            const int s_out = G.pipe ? pipe_out(l, ch) : G.merge ? s_in : s++;
            StageWriter w2{op, hb.data() + st_off + (size_t)s_out * G.stage + G.g2_off};
            for (int m = 0; m < MT; ++m)
                for (int kk = 0; kk < KS2; ++kk)
                    for (int lane = 0; lane < 64; ++lane)
                        for (int u = 0; u < KL; ++u) {
                            const int gg = lane / 32, c = lane % 32;
                            const int q = kk * K + gg * KL + u;
                            const int col = q < 32 ? 32 * ch + q : D + 32 * ch + (q - 32);
                            w2.elem(Wo[(size_t)(32 * m + c) * 2 * D + col]);
                        }
            for (int c = 0; c < D; ++c) w2.f32(bo[c]);
        }
    }
    if (G.pipe) s = NFS + n_layer_stages;
    if (G.head16) {
        // 16x16x32 head.  Layer 1 A fragments, KSPS / 2 32-channel blocks per
        // stage: lane value u of block bl, unit block ub holds
        // W1[unit 16 ub + lane % 16][channel 32 bl + 8 (lane / 16) + u]; then b1[D]
        const int bps = G.ksps / 2;
        for (int j = 0; j < G.nh1; ++j) {
            StageWriter w{op, hb.data() + st_off + (size_t)s++ * G.stage};
            for (int bl = 0; bl < bps; ++bl)
                for (int ub = 0; ub < D / 16; ++ub)
                    for (int lane = 0; lane < 64; ++lane)
                        for (int u = 0; u < 8; ++u) {
                            const int ch = 32 * (j * bps + bl) + 8 * (lane / 16) + u;
                            w.elem(W1[(size_t)(16 * ub + lane % 16) * D + ch]);
                        }
            for (int c = 0; c < D; ++c) w.f32(b1[c]);
        }
        // layer 2 A fragments: lane value u of k-step kb holds W2[output lane % 16]
        // [unit 16 (2 kb + u / 4) + 4 (lane / 16) + u % 4] (zero for outputs >= 5),
        // the order of the hidden accumulators; then b2[5]
        StageWriter w{op, hb.data() + st_off + (size_t)s++ * G.stage};
        for (int kb = 0; kb < D / 32; ++kb)
            for (int lane = 0; lane < 64; ++lane)
                for (int u = 0; u < 8; ++u) {
                    const int o = lane % 16;
                    const int unit = 16 * (2 * kb + u / 4) + 4 * (lane / 16) + u % 4;
                    w.elem(o < 5 ? (double)W2[(size_t)o * D + unit] : 0.0);
                }
        for (int c = 0; c < 5; ++c) w.f32(b2[c]);
    } else {
        // head layer 1 A fragments, KSPS k-steps per stage: lane (g, c) value u of
        // k-step ks, unit tile mu holds W1[unit 32 mu + c][channel ks K + g KL + u];
        // then b1[D]
        for (int j = 0; j < G.nh1; ++j) {
            StageWriter w{op, hb.data() + st_off + (size_t)s++ * G.stage};
            for (int kl = 0; kl < G.ksps; ++kl)
                for (int mu = 0; mu < MT; ++mu)
                    for (int lane = 0; lane < 64; ++lane)
                        for (int u = 0; u < KL; ++u) {
                            const int ks = j * G.ksps + kl;
                            w.elem(W1[(size_t)(32 * mu + lane % 32) * D + ks * K + (lane / 32) * KL + u]);
                        }
            for (int c = 0; c < D; ++c) w.f32(b1[c]);
        }
        // head layer 2 A fragments: lane (g, c) value u of k-step ks holds
        // W2[output c][unit 32 m + 8 i + 4 g + j] (zero for c >= 5), the same unit
        // order as the hidden accumulators; then b2[5]
        {
            StageWriter w{op, hb.data() + st_off + (size_t)s++ * G.stage};
            for (int ks = 0; ks < KS1; ++ks)
                for (int lane = 0; lane < 64; ++lane)
                    for (int u = 0; u < KL; ++u) {
                        const int gg = lane / 32, c = lane % 32;
                        const int reg = (ks % RPK) * KL + u, m = ks / RPK;
                        const int unit = 32 * m + 8 * (reg / 4) + 4 * gg + (reg % 4);
                        w.elem(c < 5 ? (double)W2[(size_t)c * D + unit] : 0.0);
                    }
            for (int c = 0; c < 5; ++c) w.f32(b2[c]);
        }
    }

    tf_weights *wt = new (std::nothrow) tf_weights();
    if (!wt) return TF_ENOMEM;
    if (hipGetDevice(&wt->device) != hipSuccess ||
        hipDeviceGetAttribute(&wt->cu_count, hipDeviceAttributeMultiprocessorCount, wt->device) != hipSuccess) {
        delete wt;
        return TF_EHIP;
    }
    if (hipMalloc(&wt->dmem, total) != hipSuccess) {
        delete wt;
        return TF_ENOMEM;
    }
    if (hipMemcpy(wt->dmem, hb.data(), total, hipMemcpyHostToDevice) != hipSuccess) {
        (void)hipFree(wt->dmem);
        delete wt;
        return TF_EHIP;
    }
    char *b = static_cast<char *>(wt->dmem);
    wt->n_layers = L;
    wt->d = D;
    wt->dtype = cfg->dtype;
    wt->max_hits = 32 * ht;
    wt->err = reinterpret_cast<int *>(b + err_off);
    wt->params.emb = reinterpret_cast<const float4 *>(b + emb_off);
    wt->params.stages = reinterpret_cast<const unsigned char *>(b + st_off);
    wt->n_feat = NFEAT;
    wt->params.n_layers = L;
    wt->params.n_stages = n_stages;
    wt->params.n_feat = NFEAT;
    wt->params.n_fstages = NFS;
    wt->params.kpf = KPF;
    (void)KS2;
    *out = wt;
    return TF_OK;
}

extern "C" void tf_weights_destroy(tf_weights *w) {
    if (!w) return;
    (void)hipDeviceSynchronize();
    (void)hipFree(w->dmem);
    delete w;
}

extern "C" int32_t tf_max_hits(const tf_weights *w) { return w ? w->max_hits : 0; }

namespace {
template <int D, int OP, int HT, int OUTM, bool FOURIER, bool PAIR = false>
hipError_t launch(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                  const tf_weights *w, float *out, long long out_rows, hipStream_t stream) {
    using C = KCfg<D, OP, HT, PAIR>;
    // one workgroup per compute unit (the LDS ring and the register file are
    // sized for it), at least 8 tracks per wave
    long long waves = (n_tracks + 7) / 8;
    long long blocks = (waves + C::WAVES - 1) / C::WAVES;
    const long long cap = (long long)w->cu_count;
    if (blocks > cap) blocks = cap;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL((tf_encoder_kernel<D, OP, HT, OUTM, FOURIER, PAIR>), dim3((unsigned)blocks), dim3(64 * C::WAVES), 0, stream,
                       hits, (long long)n_hits, offsets, (int)n_tracks, w->params, out, out_rows, w->err);
    return hipGetLastError();
}

template <int D, int OP, int OUTM, bool FOURIER>
hipError_t launch_ht(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                     const tf_weights *w, float *out, long long out_rows, hipStream_t stream) {
    if constexpr (D <= 128) {
        if (w->max_hits == 64) {
            if constexpr (OP != OP_F32 && OUTM == OUT_HEAD)
                return launch<D, OP, 1, OUTM, FOURIER, true>(hits, n_hits, offsets, n_tracks, w, out, out_rows, stream);
            return launch<D, OP, 2, OUTM, FOURIER>(hits, n_hits, offsets, n_tracks, w, out, out_rows, stream);
        }
    }
    return launch<D, OP, 1, OUTM, FOURIER>(hits, n_hits, offsets, n_tracks, w, out, out_rows, stream);
}

template <int D, int OUTM, bool FOURIER>
hipError_t launch_d(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                    const tf_weights *w, float *out, long long out_rows, hipStream_t stream) {
    switch (w->dtype) {
        case TF_BF16:
            return launch_ht<D, OP_BF16, OUTM, FOURIER>(hits, n_hits, offsets, n_tracks, w, out, out_rows, stream);
        case TF_BF16_F16ACT:
            return launch_ht<D, OP_F16, OUTM, FOURIER>(hits, n_hits, offsets, n_tracks, w, out, out_rows, stream);
        default:
            if constexpr (D <= 128)
                return launch_ht<D, OP_F32, OUTM, FOURIER>(hits, n_hits, offsets, n_tracks, w, out, out_rows,
                                                           stream);
            return hipErrorNotSupported;
    }
}

template <int OUTM>
tf_status launch_any(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                     const tf_weights *w, float *out, long long out_rows, hipStream_t stream) {
    hipError_t e;
    // the Fourier front end and the front-end-only pass are built for the paper's
    // width (128) and the small test width (32)
    if (w->n_feat > 0 || OUTM == OUT_FRONT) {
        const bool four = w->n_feat > 0;
        switch (w->d) {
            case 32:
                e = four ? launch_d<32, OUTM, true>(hits, n_hits, offsets, n_tracks, w, out, out_rows, stream)
                         : launch_d<32, OUTM, false>(hits, n_hits, offsets, n_tracks, w, out, out_rows, stream);
                break;
            case 128:
                e = four ? launch_d<128, OUTM, true>(hits, n_hits, offsets, n_tracks, w, out, out_rows, stream)
                         : launch_d<128, OUTM, false>(hits, n_hits, offsets, n_tracks, w, out, out_rows, stream);
                break;
            default: return TF_EUNSUPPORTED;
        }
        return e == hipSuccess ? TF_OK : TF_EHIP;
    }
    if constexpr (OUTM != OUT_FRONT) {
        switch (w->d) {
            case 32: e = launch_d<32, OUTM, false>(hits, n_hits, offsets, n_tracks, w, out, out_rows, stream); break;
            case 64: e = launch_d<64, OUTM, false>(hits, n_hits, offsets, n_tracks, w, out, out_rows, stream); break;
            case 128: e = launch_d<128, OUTM, false>(hits, n_hits, offsets, n_tracks, w, out, out_rows, stream); break;
            case 256: e = launch_d<256, OUTM, false>(hits, n_hits, offsets, n_tracks, w, out, out_rows, stream); break;
            default: return TF_EUNSUPPORTED;
        }
        return e == hipSuccess ? TF_OK : TF_EHIP;
    }
    return TF_EUNSUPPORTED;
}
}  // namespace

extern "C" tf_status fit_tracks(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                                const tf_weights *w, float *out, hipStream_t stream) {
    if (!w || n_tracks < 0 || n_hits < 0) return TF_EINVAL;
    if (n_tracks == 0) return TF_OK;
    if (!offsets || !out || (!hits && n_hits > 0)) return TF_EINVAL;
    return launch_any<OUT_HEAD>(hits, n_hits, offsets, n_tracks, w, out, 0, stream);
}

extern "C" tf_status fit_tracks_states(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                                       const tf_weights *w, float *states, hipStream_t stream) {
    if (!w || n_tracks < 0 || n_hits < 0) return TF_EINVAL;
    if (w->n_layers < 1) return TF_EUNSUPPORTED;  // no scan, no states
    if (n_tracks == 0) return TF_OK;
    if (!offsets || !states || (!hits && n_hits > 0)) return TF_EINVAL;
    return launch_any<OUT_STATES>(hits, n_hits, offsets, n_tracks, w, states, 0, stream);
}

tf_status tf_internal_front_end(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                                const tf_weights *w, void *x0, long long rows, hipStream_t stream) {
    if (!w || w->n_layers != 0 || n_tracks < 0 || n_hits < 0) return TF_EINVAL;
    if (n_tracks == 0) return TF_OK;
    if (!offsets || !x0 || (!hits && n_hits > 0)) return TF_EINVAL;
    return launch_any<OUT_FRONT>(hits, n_hits, offsets, n_tracks, w, static_cast<float *>(x0), rows, stream);
}

extern "C" tf_status tf_get_device_error(const tf_weights *w, hipStream_t stream, int32_t *flags, int clear) {
    if (!w || !flags) return TF_EINVAL;
    int v = 0;
    if (hipMemcpyAsync(&v, w->err, 4, hipMemcpyDeviceToHost, stream) != hipSuccess) return TF_EHIP;
    if (hipStreamSynchronize(stream) != hipSuccess) return TF_EHIP;
    *flags = v;
    if (clear) {
        if (hipMemsetAsync(w->err, 0, 4, stream) != hipSuccess) return TF_EHIP;
        if (hipStreamSynchronize(stream) != hipSuccess) return TF_EHIP;
    }
    return TF_OK;
}

extern "C" const char *tf_status_string(tf_status s) {
    switch (s) {
        case TF_OK: return "ok";
        case TF_EINVAL: return "invalid argument";
        case TF_ENOMEM: return "out of memory";
        case TF_EHIP: return "HIP runtime error";
        case TF_EUNSUPPORTED: return "unsupported configuration";
        case TF_ETOOLARGE: return "request exceeds a fixed capacity of the library";
    }
    return "unknown status";
}
