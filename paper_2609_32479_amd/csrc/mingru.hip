// The paper's bidirectional minGRU backbone on gfx950 (Sec. Encoder, Eq. (2)):
// per layer, four linear maps of the input give the left-to-right and the
// right-to-left pass a candidate and a gate each (z = sigmoid(gate)); the
// passes run the update of Eq. (2) from each track's first hit and from its
// last, and the 2H states of the two passes at a hit, stacked, feed the
// layer above.
// The last layer's forward state at a track's last hit and reverse state at
// its first hit are the readout's input.
//
// One launch per layer.  The front end (x, y, z embedding or the Fourier
// front end) runs first as the encoder kernel's front-end pass; each layer
// reads its input rows X [rows][DIN] and writes Y [rows][2H] (rows relative to
// offsets[0], in the matrix operand type), the last one the end states
// [n_tracks][2H] in fp32.
//
// A wave takes a tile of whole tracks (at most 32 hits, 16 tracks), holds the
// tile's input rows as matrix operands in registers (hits on the rows of
// 32x32 products), and for each 32-channel chunk and direction multiplies
// them with the candidate block, then the gate block, of the weights, which
// stream through an LDS ring shared by the workgroup (one stage per block).
// The accumulators hold channel cc of tile rows 16 s + q in lane (s, cc),
// register q: two streams of 16 positions per lane half, scanned in place; a
// track start (forward) or end (reverse) zeroes the carried coefficient, and
// a second pass carries the state across the two streams.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "common.h"
#include "internal.h"
#include "trackfit.h"

namespace {

constexpr int kMgCap = 32;    // hits per wave tile
constexpr int kMgMaxTr = 16;  // tracks per wave tile
constexpr int kMgSP = 16;     // positions per stream (two streams per tile)

template <int OP, int DIN>
struct MCfg {
    static constexpr bool HALF = OP != OP_F32;
    static constexpr int K = HALF ? 16 : 2;  // reduction depth of one product
    static constexpr int KL = K / 2;         // operand values per lane per k-step
    static constexpr int KIN = DIN / K;      // k-steps over the layer's input
    static constexpr int EB = HALF ? 2 : 4;
    static constexpr int FRAG = 64 * KL * EB;
    // 16-bit operands: two waves per SIMD (256 registers: the input operands
    // take DIN / 4); fp32 operands: one (DIN / 2 of the 512)
    static constexpr int WAVES = HALF ? 8 : 4;
    // one weight block: a 32-row slice of the candidate or gate rows, then its 32 biases
    static constexpr int BLOCK = round_up(KIN * FRAG + 32 * 4, 16);
    // a stage holds one block, or both blocks of a chunk and direction when two
    // slots of that size still leave room for a ring of at least three
    static constexpr bool MERGE = 3 * round_up(2 * BLOCK, kCopyBytes) + WAVES * (4 * kMgMaxTr * 4 + kMgCap * 4 + kMgCap * (32 * EB + 16)) <= kLdsBytesMax;
    static constexpr int STAGE = round_up((MERGE ? 2 : 1) * BLOCK, kCopyBytes);
    static constexpr int SPC = MERGE ? 1 : 2;  // stages per chunk and direction
    static constexpr int COPIES = STAGE / kCopyBytes;
    static constexpr int LPW = (COPIES + WAVES - 1) / WAVES;
    // wave-private LDS: track table and row map, then the output transpose tile
    // [32 rows][32 channels] (row stride padded by 16 bytes)
    static constexpr int ROWB = 32 * EB + 16;
    static constexpr int TB_OFF = 4 * kMgMaxTr * 4 + kMgCap * 4;
    static constexpr int WAVE_BYTES = TB_OFF + kMgCap * ROWB;
    static constexpr int NSLOT_FIT = (kLdsBytesMax - WAVES * WAVE_BYTES) / STAGE;
    static constexpr int NSLOT = NSLOT_FIT > 4 ? 4 : NSLOT_FIT;
    static_assert(NSLOT >= 2, "stage ring");
    static constexpr int WAVE0 = NSLOT * STAGE;
    static constexpr int LDS_BYTES = WAVE0 + WAVES * WAVE_BYTES;
    static_assert(DIN % K == 0, "input width");
};

// Lane (s, c) of an output column: rows 16 s + q.  One direction's scan over
// this lane's stream with the coefficients cf zeroed where the mask bits
// (forward: track starts, reverse: track ends) are set, then the carry from
// the other stream (forward: stream 0's last state into stream 1; reverse:
// stream 1's first state into stream 0).  Results overwrite ax.
template <bool FWD>
__device__ __forceinline__ void scan_dir(float (&ax)[kMgSP], float (&cf)[kMgSP], unsigned m0, unsigned m1, int s) {
    asm volatile("" : "+s"(m0), "+s"(m1));
    float h = 0.f;
#pragma unroll
    for (int i = 0; i < kMgSP; ++i) {
        const int p = FWD ? i : kMgSP - 1 - i;
        cf[p] = zero_lanes(cf[p], half_mask(m0, m1, p));
        h = fmaf(cf[p], h, ax[p]);
    }
    // h: this stream's last state (forward) or first state (reverse)
    const auto xs = __builtin_amdgcn_permlane32_swap(__float_as_uint(h), __float_as_uint(h), false, false);
    float c;
    if constexpr (FWD)
        c = s ? __uint_as_float(xs[0]) : 0.f;  // stream 0's last state, into stream 1
    else
        c = s ? 0.f : __uint_as_float(xs[1]);  // stream 1's first state, into stream 0
#pragma unroll
    for (int i = 0; i < kMgSP; ++i) {
        const int p = FWD ? i : kMgSP - 1 - i;
        c = fmaf(cf[p], c, ax[p]);
        ax[p] = c;
    }
}

template <int OP, int DIN, int H, bool LAST>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * MCfg<OP, DIN>::WAVES, 64 * MCfg<OP, DIN>::WAVES),
                          amdgpu_waves_per_eu(MCfg<OP, DIN>::WAVES / 4, MCfg<OP, DIN>::WAVES / 4)))
void tf_mingru_kernel(const typename Frag<OP>::E *__restrict__ X, long long x_rows, const int *__restrict__ offsets,
                      int n_tracks, const unsigned char *__restrict__ stages, typename Frag<OP>::E *__restrict__ Y,
                      float *__restrict__ states, int *__restrict__ err) {
    using C = MCfg<OP, DIN>;
    using F = Frag<OP>;
    using FT = typename F::T;
    using FE = typename F::E;
    constexpr int K = C::K, KL = C::KL, KIN = C::KIN, NCHK = H / 32, S = 2 * C::SPC * NCHK, SP = kMgSP;
    static_assert(H % 32 == 0, "hidden width");

    __shared__ __attribute__((aligned(16))) char smem[C::LDS_BYTES];
    const int lane = threadIdx.x & 63;
    const int wid = uniform(threadIdx.x >> 6);
    const int hh = lane >> 5, cc = lane & 31;
    int *t_start = reinterpret_cast<int *>(smem + C::WAVE0 + wid * C::WAVE_BYTES);
    int *t_len = t_start + kMgMaxTr, *t_off = t_len + kMgMaxTr, *t_id = t_off + kMgMaxTr;
    int *rowmap = t_id + kMgMaxTr;  // tile row -> input row (-1: none)

    const unsigned smem_lds = (unsigned)(uintptr_t)(__attribute__((address_space(3))) char *)smem;
    auto slot_lds = [&](int q) -> unsigned { return smem_lds + (q % C::NSLOT) * C::STAGE; };
#pragma unroll
    for (int q = 0; q < C::NSLOT - 1; ++q) copy_stage<C>(stages, q % S, slot_lds(q), wid, lane);
    // Stage q (counted across tiles) lives in slot q % NSLOT.  Every stage ends
    // with all of this wave's memory operations complete and a barrier, after
    // which stage q + NSLOT goes into the slot just read; the last stage of a
    // tile leaves that copy to the start of the next tile.
    int q = 0;
    auto advance = [&](bool last) {
        wait_vmcnt<0>();
        lds_barrier();
        if (!last) copy_stage<C>(stages, (q + C::NSLOT) % S, slot_lds(q + C::NSLOT), wid, lane);
        ++q;
    };
    auto slot = [&]() -> const char * { return smem + (q % C::NSLOT) * C::STAGE; };

    const long long gw = (long long)blockIdx.x * C::WAVES + wid;
    const long long nw = (long long)gridDim.x * C::WAVES;
    const int g_begin = group_begin(offsets, n_tracks, gw, nw, lane);
    const int g_end = group_begin(offsets, n_tracks, gw + 1, nw, lane);
    const int row0 = offsets[0];
    const float qnan = __builtin_nanf("");
    int errbits = 0;

    // Tiles are packed from a window of the wave's tracks: the first track not
    // yet fitted (t) and the WIN - 1 after it; bit i of `taken` marks track
    // t + i as fitted into an earlier tile (or refused).  A track that cannot be
    // fitted (rows outside the input, no hits, more than 32) is refused: NaN end
    // states and its error bit.
    constexpr int WIN = 32;
    int t = g_begin;
    unsigned taken = 0;
    for (;;) {
        int k = 0, n = 0, off = 0, len = 0;
        unsigned sel = 0;  // window tracks of the tile
        while (t < g_end) {
            const int sh = taken == ~0u ? WIN : __builtin_ctz(~taken);
            taken = sh == WIN ? 0u : taken >> sh;
            t += sh;
            if (t >= g_end) break;
            const int idx = t + lane;
            off = (lane <= WIN && idx <= g_end) ? offsets[idx] : 0;
            const int nxt = __shfl_down(off, 1);
            len = nxt - off;
            const bool fresh = lane < WIN && idx < g_end && !((taken >> (lane & 31)) & 1u);
            const bool bad_rows = (long long)off < row0 || nxt < off || (long long)nxt - row0 > x_rows;
            const bool empty = !bad_rows && len == 0;
            const bool too_long = !bad_rows && len > kMgCap;
            const unsigned bm = unsigned(__ballot(fresh && bad_rows));
            const unsigned em = unsigned(__ballot(fresh && empty));
            const unsigned lm = unsigned(__ballot(fresh && too_long));
            if (bm | em | lm) {
                errbits |= (bm ? TF_DEVERR_BAD_OFFSETS : 0) | (em ? TF_DEVERR_EMPTY_TRACK : 0) |
                           (lm ? TF_DEVERR_TOO_LONG : 0);
                if constexpr (LAST)
                    for (unsigned m = bm | em | lm; m; m &= m - 1u)
                        for (int e = lane; e < 2 * H; e += 64)
                            states[(size_t)(t + __builtin_ctz(m)) * 2 * H + e] = qnan;
                taken |= bm | em | lm;
            }
            const unsigned cand = unsigned(__ballot(fresh && !bad_rows && !empty && !too_long));
            if (cand) {
                sel = pack_tile<kMgCap, kMgMaxTr, true>(cand, len, lane, n);
                k = __builtin_popcount(sel);
                taken |= sel;
                break;
            }
        }
        const bool work = k > 0;
        wait_vmcnt<0>();
        if (!__syncthreads_or(work)) break;  // every wave of the workgroup is done
        copy_stage<C>(stages, (q + C::NSLOT - 1) % S, slot_lds(q + C::NSLOT - 1), wid, lane);

        // ---- tile metadata, row map and the input rows as matrix operands
        unsigned sb0 = 0, sb1 = 0, eb0 = 0, eb1 = 0, st0 = 0, st1 = 0;
        FT xa[KIN];
        if (work) {
            // the tile's tracks in window order, on consecutive tile rows
            const bool mine = lane < WIN && ((sel >> (lane & 31)) & 1u);
            const int v = mine ? len : 0;
            int incl = v;  // inclusive prefix sum of the selected lengths over lanes
#pragma unroll
            for (int dd = 1; dd < WIN; dd <<= 1) {
                const int y = __shfl_up(incl, dd);
                if (lane >= dd) incl += y;
            }
            const int rs = incl - v;  // first tile row of this lane's track
            if (mine) {
                const int j = __builtin_amdgcn_mbcnt_lo(sel, 0);  // selected tracks before this one
                t_start[j] = rs;
                t_len[j] = len;
                t_off[j] = off;
                t_id[j] = t + lane;
            }
            unsigned long long smask = 0;  // tile rows that start a track
            for (unsigned m = sel; m; m &= m - 1u) smask |= 1ull << __builtin_amdgcn_readlane(rs, __builtin_ctz(m));
            const unsigned long long valid = (1ull << n) - 1ull;
            const unsigned long long vstart = smask | (1ull << n);
            const unsigned long long emask = ((smask >> 1) | (1ull << (n - 1))) & valid;
            sb0 = unsigned(vstart) & 0xffffu;
            sb1 = unsigned(vstart >> SP) & 0xffffu;
            eb0 = unsigned(emask) & 0xffffu;
            eb1 = unsigned(emask >> SP) & 0xffffu;
            st0 = unsigned(smask) & 0xffffu;
            st1 = unsigned(smask >> SP) & 0xffffu;
            wave_lds_sync();  // the track table is written
            if (lane < kMgCap) {
                int r = -1;
                if (lane < n) {
                    const int j = __builtin_popcountll(smask & ((2ull << lane) - 1ull)) - 1;
                    r = t_off[j] + (lane - t_start[j]) - row0;
                }
                rowmap[lane] = r;
            }
            wave_lds_sync();
            // A operand: lane (s, i) holds input channels k-step K + s KL .. + KL - 1 of
            // tile row slot_to_hit(i), whose products land in accumulator row i
            const int xr = rowmap[slot_to_hit<SP>(cc)];
#pragma unroll
            for (int ks = 0; ks < KIN; ++ks) {
                if (xr >= 0)
                    xa[ks] = *reinterpret_cast<const FT *>(X + (size_t)xr * DIN + ks * K + hh * KL);
                else
                    xa[ks] = FT{};
            }
        }

        // Each block's outputs leave through the wave's LDS tile as 16-byte pieces
        // (one value per lane and row would be 2- or 4-byte stores), and are
        // stored only after the barrier that ends the block: the barrier first
        // waits for this wave's memory operations (the stage copies), and stores
        // still in flight would hold it up.  Layer outputs: tile row -> input row
        // (32 rows of 32 channels); end states: the tile's tracks (up to kMgMaxTr
        // rows of 32 fp32 channels).
        constexpr int VPP = LAST ? 4 : 16 / (int)sizeof(FE);  // values per 16-byte piece
        constexpr int PPR = 32 / VPP;                          // pieces per row of 32 channels
        constexpr int NPEND = (LAST ? kMgMaxTr : 32) * PPR / 64;  // pieces per lane
        static_assert(NPEND * 64 == (LAST ? kMgMaxTr : 32) * PPR, "pieces");
        u32x4 pv[NPEND];
        int prow[NPEND];  // destination row of each piece (-1: none)
        int pcol = 0;     // first channel of the pieces (uniform)
#pragma unroll
        for (int p = 0; p < NPEND; ++p) prow[p] = -1;
        auto flush = [&]() {
#pragma unroll
            for (int p = 0; p < NPEND; ++p) {
                const int g = (lane + 64 * p) % PPR;
                if (prow[p] >= 0) {
                    if constexpr (LAST)
                        *reinterpret_cast<u32x4 *>(states + (size_t)prow[p] * 2 * H + pcol + g * VPP) = pv[p];
                    else
                        *reinterpret_cast<u32x4 *>(Y + (size_t)prow[p] * 2 * H + pcol + g * VPP) = pv[p];
                }
                prow[p] = -1;
            }
        };

        // ---- chunks of 32 hidden channels, forward then reverse direction
        for (int ch = 0; ch < NCHK; ++ch) {
#pragma unroll
            for (int dir = 0; dir < 2; ++dir) {
                f32x16 ax;
                if (work) {
                    // candidate block: rows dir 2H + 32 ch + cc of the layer's weights
                    const FT *wf = reinterpret_cast<const FT *>(slot());
#pragma unroll
                    for (int i = 0; i < 16; ++i) ax[i] = 0.f;
                    __builtin_amdgcn_s_setprio(1);
#pragma unroll
                    for (int ks = 0; ks < KIN; ++ks) ax = F::mma(xa[ks], wf[ks * 64 + lane], ax);
                    __builtin_amdgcn_s_setprio(0);
                    ax += reinterpret_cast<const float *>(slot() + KIN * C::FRAG)[cc];
                }
                if constexpr (!C::MERGE) advance(false);
                flush();  // the previous block's outputs
                // the gate block: the next stage, or the second block of this one
                const char *gsl = slot() + (C::MERGE ? C::BLOCK : 0);
                if (work) {
                    // gate block: rows dir 2H + H + 32 ch + cc; bias pre-scaled by -log2(e)
                    // in the 16-bit modes (exp2 below)
                    const FT *wf = reinterpret_cast<const FT *>(gsl);
                    f32x16 gx;
#pragma unroll
                    for (int i = 0; i < 16; ++i) gx[i] = 0.f;
                    __builtin_amdgcn_s_setprio(1);
#pragma unroll
                    for (int ks = 0; ks < KIN; ++ks) gx = F::mma(xa[ks], wf[ks * 64 + lane], gx);
                    __builtin_amdgcn_s_setprio(0);
                    const float bgv = reinterpret_cast<const float *>(gsl + KIN * C::FRAG)[cc];
                    float AX[SP], CF[SP];
#pragma unroll
                    for (int i = 0; i < SP; ++i) {
                        const float g = gx[i];
                        float a, cf;
                        if constexpr (C::HALF) {
                            const float e = __builtin_amdgcn_exp2f(fmaf(g, -kLog2e, bgv));
                            a = __builtin_amdgcn_rcpf(1.0f + e);
                            cf = 1.0f - a;
                        } else {
                            const float e = expf(-__builtin_amdgcn_fmed3f(g + bgv, -80.0f, 80.0f));
                            a = 1.0f / (1.0f + e);
                            cf = e * a;
                        }
                        AX[i] = a * ax[i];
                        CF[i] = cf;
                    }
                    if (dir == 0)
                        scan_dir<true>(AX, CF, sb0, sb1, hh);
                    else
                        scan_dir<false>(AX, CF, eb0, eb1, hh);
                    pcol = dir * H + 32 * ch;
                    char *tile = smem + C::WAVE0 + wid * C::WAVE_BYTES + C::TB_OFF;
                    wave_lds_sync();  // the previous block's reads of the tile are done
                    if constexpr (LAST) {
                        // forward state at a track's last row, reverse state at its first row,
                        // to row j of the tile (the track's index in it: the number of track
                        // starts up to the row, less one)
                        constexpr int ROWF = 32 + 4;  // row stride (floats)
                        static_assert(kMgMaxTr * ROWF * 4 <= kMgCap * C::ROWB, "end-state rows in the tile");
                        float *tf = reinterpret_cast<float *>(tile);
                        const unsigned sw = hh ? st1 : st0;
                        const unsigned mw = dir == 0 ? (hh ? eb1 : eb0) : sw;
                        const int jb = hh ? __builtin_popcount(st0) - 1 : -1;
#pragma unroll
                        for (int i = 0; i < SP; ++i)
                            if ((mw >> i) & 1u) {
                                const int j = jb + __builtin_popcount(sw & ((2u << i) - 1u));
                                tf[j * ROWF + cc] = AX[i];
                            }
                        wave_lds_sync();
#pragma unroll
                        for (int p = 0; p < NPEND; ++p) {
                            const int it = lane + 64 * p, j = it / PPR, g = it % PPR;
                            prow[p] = j < k ? t_id[j] : -1;
                            pv[p] = *reinterpret_cast<const u32x4 *>(tf + j * ROWF + g * VPP);
                        }
                    } else {
                        constexpr int ROWE = C::ROWB / (int)sizeof(FE);  // tile row stride (elements)
                        FE *tb = reinterpret_cast<FE *>(tile);
#pragma unroll
                        for (int i = 0; i < SP; ++i) {
                            // the asm keeps the state's last update (rounded to fp32) and its
                            // conversion to the operand type apart: fused into one
                            // mixed-precision fma at some positions, they would round once
                            // instead of twice, and a track's outputs would depend on where
                            // in the tile it lies
                            float v = AX[i];
                            asm volatile("" : "+v"(v));
                            tb[(SP * hh + i) * ROWE + cc] = (FE)v;
                        }
                        wave_lds_sync();
#pragma unroll
                        for (int p = 0; p < NPEND; ++p) {
                            const int it = lane + 64 * p, row = it / PPR, g = it % PPR;
                            prow[p] = rowmap[row];
                            pv[p] = *reinterpret_cast<const u32x4 *>(tb + row * ROWE + g * VPP);
                        }
                    }
                }
                advance(ch == NCHK - 1 && dir == 1);
            }
        }
        flush();  // the tile's last block
    }
    if (errbits && lane == 0) atomicOr(err, errbits);
}

template <int OP, int DIN, int H, bool LAST>
hipError_t launch_layer(const void *X, long long x_rows, const int32_t *offsets, int32_t n_tracks,
                        const unsigned char *stages, void *Y, float *states, int *err, int cu_count,
                        hipStream_t stream) {
    using C = MCfg<OP, DIN>;
    long long waves = (n_tracks + 7) / 8;
    long long blocks = (waves + C::WAVES - 1) / C::WAVES;
    if (blocks > cu_count) blocks = cu_count;
    if (blocks < 1) blocks = 1;
    using FE = typename Frag<OP>::E;
    hipLaunchKernelGGL((tf_mingru_kernel<OP, DIN, H, LAST>), dim3((unsigned)blocks), dim3(64 * C::WAVES), 0, stream,
                       static_cast<const FE *>(X), x_rows, offsets, (int)n_tracks, stages, static_cast<FE *>(Y), states,
                       err);
    return hipGetLastError();
}

template <int OP, int DIN, int H>
hipError_t launch_last(bool last, const void *X, long long x_rows, const int32_t *offsets, int32_t n_tracks,
                       const unsigned char *stages, void *Y, float *states, int *err, int cu_count, hipStream_t stream) {
    return last ? launch_layer<OP, DIN, H, true>(X, x_rows, offsets, n_tracks, stages, Y, states, err, cu_count, stream)
                : launch_layer<OP, DIN, H, false>(X, x_rows, offsets, n_tracks, stages, Y, states, err, cu_count, stream);
}

// Stage geometry of a layer for the host: bytes per stage, per block, and
// whether a chunk's candidate and gate blocks share a stage.
struct MGeom {
    int stage, block, merge;
};
template <int OP, int DIN>
MGeom stage_bytes() {
    return {MCfg<OP, DIN>::STAGE, MCfg<OP, DIN>::BLOCK, MCfg<OP, DIN>::MERGE ? 1 : 0};
}

int op_of(int32_t dtype) { return dtype == TF_BF16 ? OP_BF16 : dtype == TF_BF16_F16ACT ? OP_F16 : OP_F32; }

MGeom stage_bytes_of(int op, int din) {
    switch (op) {
        case OP_BF16:
        case OP_F16:
            return din == 32 ? stage_bytes<OP_F16, 32>() : din == 128 ? stage_bytes<OP_F16, 128>()
                                                                      : stage_bytes<OP_F16, 384>();
        default:
            return din == 32 ? stage_bytes<OP_F32, 32>() : din == 128 ? stage_bytes<OP_F32, 128>()
                                                                      : stage_bytes<OP_F32, 384>();
    }
}

// float -> bf16 / fp16 bits, round to nearest even
uint16_t bits16(float x, bool bf) {
    if (bf) {
        uint32_t u;
        std::memcpy(&u, &x, 4);
        if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
        u += 0x7fffu + ((u >> 16) & 1u);
        return (uint16_t)(u >> 16);
    }
    const _Float16 h = (_Float16)x;
    uint16_t b;
    std::memcpy(&b, &h, 2);
    return b;
}

}  // namespace

struct tf_mingru {
    tf_mingru_config cfg{};
    int op = 0, cu_count = 0;
    tf_weights *front = nullptr;      // the front end (an encoder handle with no layers)
    char *dmem = nullptr;             // layer stages, error word
    std::vector<const unsigned char *> stages;  // per layer
    int *err = nullptr;
    void *scratch = nullptr;          // this device's copy of `scratch` (tf_mingru_states_noalloc)
};

// Workspace of tf_mingru_states_noalloc: a fixed array in device memory,
// one copy on every device the library runs on, held until the process ends.
// In host code `scratch` only names the symbol; its device address (one per
// device) comes from hipGetSymbolAddress, looked up once per device while
// that device is current (in tf_mingru_create) and used for every access.
static constexpr size_t kNoAllocScratchBytes = size_t(128) << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices];   // device address of `scratch` per device (null: not looked up yet)

// The current device's address of `scratch`, looked up on first use.
hipError_t scratch_of_current_device(void **out) {
    *out = nullptr;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}
}  // namespace

static size_t front_floats(int d, int nf) {
    return nf > 0 ? 2 * (size_t)nf + (size_t)d * 32 * nf + d : 4 * (size_t)d;
}

extern "C" size_t tf_mingru_blob_size(const tf_mingru_config *cfg) {
    if (!cfg || cfg->n_layers < 1 || cfg->d_model <= 0 || cfg->hidden <= 0 || cfg->n_features < 0) return 0;
    size_t s = front_floats(cfg->d_model, cfg->n_features);
    for (int l = 0; l < cfg->n_layers; ++l) {
        const size_t din = l == 0 ? (size_t)cfg->d_model : 2 * (size_t)cfg->hidden;
        s += 4 * (size_t)cfg->hidden * din + 4 * (size_t)cfg->hidden;
    }
    return s;
}

extern "C" tf_status tf_mingru_create(const tf_mingru_config *cfg, const float *blob, size_t n_floats,
                                      tf_mingru **out) {
    if (!out) return TF_EINVAL;
    *out = nullptr;
    if (!cfg || !blob) return TF_EINVAL;
    if (cfg->dtype != TF_FP32 && cfg->dtype != TF_BF16 && cfg->dtype != TF_BF16_F16ACT) return TF_EINVAL;
    if (cfg->n_layers < 1 || cfg->d_model <= 0 || cfg->hidden <= 0 || cfg->n_features < 0) return TF_EINVAL;
    const int d = cfg->d_model, H = cfg->hidden, L = cfg->n_layers, nf = cfg->n_features;
    if (!((d == 32 && H == 64) || (d == 128 && H == 192)) || L > 8 || nf > 16) return TF_EUNSUPPORTED;
    if (n_floats != tf_mingru_blob_size(cfg)) return TF_EINVAL;
    const int op = op_of(cfg->dtype);
    const bool half = op != OP_F32, bf = op == OP_BF16;
    const int K = half ? 16 : 2, KL = K / 2;

    tf_mingru *h = new (std::nothrow) tf_mingru;
    if (!h) return TF_ENOMEM;
    h->cfg = *cfg;
    h->op = op;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&h->cu_count, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
        delete h;
        return TF_EHIP;
    }
    // the front end: an encoder handle with no layers (zero head, never evaluated)
    {
        const size_t ff = front_floats(d, nf);
        tf_config fc{0, d, cfg->dtype, 32, nf};
        const size_t fn = nf > 0 ? tf_fourier_blob_size(0, d, nf) : tf_blob_size(0, d);
        std::vector<float> fb(fn, 0.f);
        std::memcpy(fb.data(), blob, ff * sizeof(float));
        const tf_status st = tf_weights_create(&fc, fb.data(), fn, &h->front);
        if (st != TF_OK) {
            delete h;
            return st;
        }
    }
    // layer stages: for each 32-channel chunk and direction, the candidate block then
    // the gate block; lane (s, c) value e of k-step ks holds W[row 32 ch + c of the
    // block][column ks K + s KL + e]; then the block's 32 biases (the gate's times
    // -log2(e) for the 16-bit modes)
    std::vector<size_t> loff(L);
    size_t total = 0;
    for (int l = 0; l < L; ++l) {
        const int din = l == 0 ? d : 2 * H;
        loff[l] = total;
        const MGeom g = stage_bytes_of(op, din);
        total += (size_t)(g.merge ? 2 : 4) * (H / 32) * g.stage;
    }
    const size_t err_off = total;
    total += 256;
    std::vector<unsigned char> hb(total, 0);
    const float *lw = blob + front_floats(d, nf);
    for (int l = 0; l < L; ++l) {
        const int din = l == 0 ? d : 2 * H, KIN = din / K;
        const MGeom g = stage_bytes_of(op, din);
        const float *W = lw, *b = lw + (size_t)4 * H * din;
        unsigned char *dst = hb.data() + loff[l];
        for (int ch = 0; ch < H / 32; ++ch)
            for (int dir = 0; dir < 2; ++dir)
                for (int part = 0; part < 2; ++part) {
                    // the candidate block starts a stage; the gate block follows it in the
                    // same stage (merged) or starts the next one
                    unsigned char *sp = dst;
                    dst += (g.merge && part == 0) ? g.block : (g.merge ? g.stage - g.block : g.stage);
                    const int rbase = dir * 2 * H + part * H + 32 * ch;
                    size_t o = 0;
                    for (int ks = 0; ks < KIN; ++ks)
                        for (int lane = 0; lane < 64; ++lane)
                            for (int e = 0; e < KL; ++e) {
                                const float v = W[(size_t)(rbase + lane % 32) * din + ks * K + (lane / 32) * KL + e];
                                if (half) {
                                    const uint16_t bb = bits16(v, bf);
                                    std::memcpy(sp + o, &bb, 2);
                                    o += 2;
                                } else {
                                    std::memcpy(sp + o, &v, 4);
                                    o += 4;
                                }
                            }
                    for (int c = 0; c < 32; ++c) {
                        float bv = b[rbase + c];
                        if (half && part == 1) bv = (float)(-1.4426950408889634 * (double)bv);
                        std::memcpy(sp + o + 4 * c, &bv, 4);
                    }
                }
        lw += (size_t)4 * H * din + (size_t)4 * H;
    }
    if (hipMalloc((void **)&h->dmem, total) != hipSuccess) {
        tf_weights_destroy(h->front);
        delete h;
        return TF_ENOMEM;
    }
    if (hipMemcpy(h->dmem, hb.data(), total, hipMemcpyHostToDevice) != hipSuccess) {
        (void)hipFree(h->dmem);
        tf_weights_destroy(h->front);
        delete h;
        return TF_EHIP;
    }
    for (int l = 0; l < L; ++l) h->stages.push_back(reinterpret_cast<const unsigned char *>(h->dmem + loff[l]));
    h->err = reinterpret_cast<int *>(h->dmem + err_off);
    if (scratch_of_current_device(&h->scratch) != hipSuccess) {
        (void)hipFree(h->dmem);
        tf_weights_destroy(h->front);
        delete h;
        return TF_EHIP;
    }
    *out = h;
    return TF_OK;
}

extern "C" void tf_mingru_destroy(tf_mingru *h) {
    if (!h) return;
    (void)hipDeviceSynchronize();
    (void)hipFree(h->dmem);
    tf_weights_destroy(h->front);
    delete h;
}

static size_t row_bytes(const tf_mingru *h) {
    const size_t eb = h->op == OP_F32 ? 4 : 2;
    const int L = h->cfg.n_layers;
    const size_t nbuf = L > 2 ? 2 : (size_t)(L - 1);
    return eb * ((size_t)h->cfg.d_model + nbuf * 2 * (size_t)h->cfg.hidden);
}

extern "C" size_t tf_mingru_workspace_size(const tf_mingru *h, int64_t n_rows) {
    if (!h || n_rows < 0) return 0;
    return row_bytes(h) * (size_t)n_rows + 256;
}

namespace {
tf_status mingru_states(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                        const tf_mingru *h, void *workspace, size_t workspace_bytes, float *states,
                        hipStream_t stream) {
    const int d = h->cfg.d_model, H = h->cfg.hidden, L = h->cfg.n_layers;
    const size_t eb = h->op == OP_F32 ? 4 : 2;
    // rows of the batch that fit the workspace: X0 [rows][d], then up to two [rows][2H]
    const long long rows = (long long)((workspace_bytes > 256 ? workspace_bytes - 256 : 0) / row_bytes(h));
    char *ws = static_cast<char *>(workspace);
    char *x0 = ws;
    char *ybuf[2] = {x0 + (size_t)rows * d * eb, x0 + (size_t)rows * d * eb + (size_t)rows * 2 * H * eb};
    tf_status st = tf_internal_front_end(hits, n_hits, offsets, n_tracks, h->front, x0, rows, stream);
    if (st != TF_OK) return st;
    const void *xin = x0;
    for (int l = 0; l < L; ++l) {
        const bool last = l == L - 1;
        void *yout = last ? nullptr : ybuf[l % 2];
        const int din = l == 0 ? d : 2 * H;
        hipError_t e = hipErrorNotSupported;
        const unsigned char *sg = h->stages[l];
        switch (h->op) {
            case OP_BF16:
                if (H == 192)
                    e = din == 128 ? launch_last<OP_BF16, 128, 192>(last, xin, rows, offsets, n_tracks, sg, yout, states, h->err, h->cu_count, stream)
                                   : launch_last<OP_BF16, 384, 192>(last, xin, rows, offsets, n_tracks, sg, yout, states, h->err, h->cu_count, stream);
                else
                    e = din == 32 ? launch_last<OP_BF16, 32, 64>(last, xin, rows, offsets, n_tracks, sg, yout, states, h->err, h->cu_count, stream)
                                  : launch_last<OP_BF16, 128, 64>(last, xin, rows, offsets, n_tracks, sg, yout, states, h->err, h->cu_count, stream);
                break;
            case OP_F16:
                if (H == 192)
                    e = din == 128 ? launch_last<OP_F16, 128, 192>(last, xin, rows, offsets, n_tracks, sg, yout, states, h->err, h->cu_count, stream)
                                   : launch_last<OP_F16, 384, 192>(last, xin, rows, offsets, n_tracks, sg, yout, states, h->err, h->cu_count, stream);
                else
                    e = din == 32 ? launch_last<OP_F16, 32, 64>(last, xin, rows, offsets, n_tracks, sg, yout, states, h->err, h->cu_count, stream)
                                  : launch_last<OP_F16, 128, 64>(last, xin, rows, offsets, n_tracks, sg, yout, states, h->err, h->cu_count, stream);
                break;
            default:
                if (H == 192)
                    e = din == 128 ? launch_last<OP_F32, 128, 192>(last, xin, rows, offsets, n_tracks, sg, yout, states, h->err, h->cu_count, stream)
                                   : launch_last<OP_F32, 384, 192>(last, xin, rows, offsets, n_tracks, sg, yout, states, h->err, h->cu_count, stream);
                else
                    e = din == 32 ? launch_last<OP_F32, 32, 64>(last, xin, rows, offsets, n_tracks, sg, yout, states, h->err, h->cu_count, stream)
                                  : launch_last<OP_F32, 128, 64>(last, xin, rows, offsets, n_tracks, sg, yout, states, h->err, h->cu_count, stream);
                break;
        }
        if (e != hipSuccess) return TF_EHIP;
        xin = yout;
    }
    return TF_OK;
}
}  // namespace

extern "C" tf_status tf_mingru_states(const float *hits, int64_t n_hits, const int32_t *offsets, int32_t n_tracks,
                                      const tf_mingru *h, void *workspace, size_t workspace_bytes, float *states,
                                      hipStream_t stream) {
    if (!h || n_tracks < 0 || n_hits < 0) return TF_EINVAL;
    if (n_tracks == 0) return TF_OK;
    if (!offsets || !states || !workspace || (!hits && n_hits > 0)) return TF_EINVAL;
    return mingru_states(hits, n_hits, offsets, n_tracks, h, workspace, workspace_bytes, states, stream);
}

extern "C" int64_t tf_mingru_noalloc_max_rows(const tf_mingru *h) {
    if (!h) return 0;
    return (int64_t)((kNoAllocScratchBytes - 256) / row_bytes(h));
}

extern "C" tf_status tf_mingru_states_noalloc(const float *hits, int64_t n_hits, const int32_t *offsets,
                                              int32_t n_tracks, const tf_mingru *h, float *states,
                                              hipStream_t stream) {
    if (!h || n_tracks < 0 || n_hits < 0) return TF_EINVAL;
    if (n_hits > tf_mingru_noalloc_max_rows(h)) return TF_ETOOLARGE;
    if (n_tracks == 0) return TF_OK;
    if (!offsets || !states || (!hits && n_hits > 0)) return TF_EINVAL;
    if (!h->scratch) return TF_EHIP;
    // every workspace row a kernel reads was written earlier in the same call, so
    // nothing left in the array by an earlier call needs clearing
    return mingru_states(hits, n_hits, offsets, n_tracks, h, h->scratch, kNoAllocScratchBytes, states, stream);
}

extern "C" tf_status tf_mingru_device_error(const tf_mingru *h, hipStream_t stream, int32_t *flags, int clear) {
    if (!h || !flags) return TF_EINVAL;
    int v = 0;
    if (hipMemcpyAsync(&v, h->err, 4, hipMemcpyDeviceToHost, stream) != hipSuccess) return TF_EHIP;
    if (hipStreamSynchronize(stream) != hipSuccess) return TF_EHIP;
    int32_t f = 0;
    tf_status st = tf_get_device_error(h->front, stream, &f, clear);
    if (st != TF_OK) return st;
    *flags = v | f;
    if (clear) {
        const int zero = 0;
        if (hipMemcpyAsync(h->err, &zero, 4, hipMemcpyHostToDevice, stream) != hipSuccess) return TF_EHIP;
        if (hipStreamSynchronize(stream) != hipSuccess) return TF_EHIP;
    }
    return TF_OK;
}
