// The paper's bidirectional minGRU backbone on gfx950 (Sec. Encoder, Eq. (2)):
// per layer, four linear maps of the input give the left-to-right and the
// right-to-left pass a candidate and a gate each (z = sigmoid(gate)); the
// passes run the update of Eq. (2) from each track's first hit and from its
// last, and the 2H states of the two passes at a hit, stacked, feed the
// layer above.
// The last layer's forward state at a track's last hit and reverse state at
// its first hit are the readout's input.
//
// Two ways to run it.  The paper's deployed configuration (16-bit modes,
// Fourier front end, d = 128, H = 192, two layers) runs as one launch of
// tf_backbone_kernel, which keeps the front end's output and the first
// layer's states on chip (below).  Otherwise, and when asked for, one launch
// per layer: the front end (x, y, z embedding or the Fourier front end) runs
// first as the encoder kernel's front-end pass; each layer reads its input
// rows X [rows][DIN] and writes Y [rows][2H] (rows relative to offsets[0], in
// the matrix operand type), the last one the end states [n_tracks][2H] in
// fp32.  Both compute the same bits.
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
#include <climits>
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

// Tiles are packed from a window of a wave's tracks: the first track not yet
// fitted (t) and the kMgWin - 1 after it; bit i of `taken` marks track t + i as
// fitted into an earlier tile (or refused).  A track that cannot be fitted
// (rows below 0 or row0, past row0 + x_rows or n_hits, no hits, more than 32)
// is refused: its error bit and, with states, NaN end states (2H of them).
// Returns the tile's window lanes (sel; wave-uniform) and their row total (n);
// off and len are each window lane's track start and length.
constexpr int kMgWin = 32;
__device__ __forceinline__ unsigned mg_select(const int *__restrict__ offsets, int g_end, int row0, long long x_rows,
                                              long long n_hits, int lane, int &t, unsigned &taken, int &errbits,
                                              float *__restrict__ states, int H, int &n, int &off, int &len) {
    n = 0;
    off = 0;
    len = 0;
    while (t < g_end) {
        const int sh = taken == ~0u ? kMgWin : __builtin_ctz(~taken);
        taken = sh == kMgWin ? 0u : taken >> sh;
        t += sh;
        if (t >= g_end) break;
        const int idx = t + lane;
        off = (lane <= kMgWin && idx <= g_end) ? offsets[idx] : 0;
        const int nxt = __shfl_down(off, 1);
        len = nxt - off;
        const bool fresh = lane < kMgWin && idx < g_end && !((taken >> (lane & 31)) & 1u);
        const bool bad_rows =
            off < 0 || off < row0 || nxt < off || (long long)nxt - row0 > x_rows || (long long)nxt > n_hits;
        const bool empty = !bad_rows && len == 0;
        const bool too_long = !bad_rows && len > kMgCap;
        const unsigned bm = unsigned(__ballot(fresh && bad_rows));
        const unsigned em = unsigned(__ballot(fresh && empty));
        const unsigned lm = unsigned(__ballot(fresh && too_long));
        if (bm | em | lm) {
            errbits |= (bm ? TF_DEVERR_BAD_OFFSETS : 0) | (em ? TF_DEVERR_EMPTY_TRACK : 0) |
                       (lm ? TF_DEVERR_TOO_LONG : 0);
            if (states) {
                const float qnan = __builtin_nanf("");
                for (unsigned m = bm | em | lm; m; m &= m - 1u)
                    for (int e = lane; e < 2 * H; e += 64) states[(size_t)(t + __builtin_ctz(m)) * 2 * H + e] = qnan;
            }
            taken |= bm | em | lm;
        }
        const unsigned cand = unsigned(__ballot(fresh && !bad_rows && !empty && !too_long));
        if (cand) {
            const unsigned sel = pack_tile<kMgCap, kMgMaxTr, true>(cand, len, lane, n);
            taken |= sel;
            return sel;
        }
    }
    return 0u;
}

// Track table and masks of a packed tile: the tile's tracks in window order on
// consecutive tile rows; t_* [kMgMaxTr] and rowmap [kMgCap] (tile row -> input
// row relative to row0, -1: none) in the wave's LDS; per stream (16 rows) the
// bits of the rows that start a track (st), of the starts plus the row after
// the last hit (sb: where a forward pass restarts) and of the track ends (eb).
__device__ __forceinline__ void mg_tile_meta(unsigned sel, int n, int off, int len, int t, int row0, int lane,
                                             int *t_start, int *t_len, int *t_off, int *t_id, int *rowmap,
                                             unsigned &sb0, unsigned &sb1, unsigned &eb0, unsigned &eb1,
                                             unsigned &st0, unsigned &st1) {
    constexpr int SP = kMgSP;
    const bool mine = lane < kMgWin && ((sel >> (lane & 31)) & 1u);
    const int v = mine ? len : 0;
    int incl = v;  // inclusive prefix sum of the selected lengths over lanes
#pragma unroll
    for (int dd = 1; dd < kMgWin; dd <<= 1) {
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
    int errbits = 0;

    int t = g_begin;
    unsigned taken = 0;
    for (;;) {
        int n = 0, off = 0, len = 0;
        const unsigned sel = mg_select(offsets, g_end, row0, x_rows, LLONG_MAX, lane, t, taken, errbits,
                                       LAST ? states : nullptr, H, n, off, len);
        const int k = __builtin_popcount(sel);
        const bool work = k > 0;
        wait_vmcnt<0>();
        if (!__syncthreads_or(work)) break;  // every wave of the workgroup is done
        copy_stage<C>(stages, (q + C::NSLOT - 1) % S, slot_lds(q + C::NSLOT - 1), wid, lane);

        // ---- tile metadata, row map and the input rows as matrix operands
        unsigned sb0 = 0, sb1 = 0, eb0 = 0, eb1 = 0, st0 = 0, st1 = 0;
        FT xa[KIN];
        if (work) {
            mg_tile_meta(sel, n, off, len, t, row0, lane, t_start, t_len, t_off, t_id, rowmap, sb0, sb1, eb0, eb1,
                         st0, st1);
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

// ---------------------------------------------------------------------------
// The paper's deployed backbone in one launch (16-bit modes): the Fourier
// front end (d = 128), a first layer of input d and a last layer of input
// 2H = 384 (H = 192).  Per hit it does the layered path's arithmetic, operation
// for operation, so its end states are the same bits; what changes is where
// the intermediate values live.  The front end's output never leaves the
// registers: its projection puts channels on the rows of the products (the
// weights as A operand, each 32-channel block's rows stored in an order that
// leaves lane half g holding channels 16 p + 8 g .. + 7), which is exactly the
// first layer's A operand once rounded.  Each block of the first layer's
// states passes through the wave's LDS tile into the second layer's operand
// registers (96 of them).  Nothing but features, offsets, weights and the
// end states touches HBM.
// Stage sequence of a tile: the front end's projection (KPF k-steps of all
// four channel blocks per stage; the first stage also holds the bias and the
// features' lo and 1 / (hi - lo)), the first layer's candidate and gate blocks
// of both directions of a chunk in one stage, then the last layer's blocks one
// to a stage.
// ---------------------------------------------------------------------------
constexpr int kBbMaxFeat = 16;  // per-hit features, at most
constexpr int kBbUStride = 17;  // LDS row stride of a hit's normalised features (floats)

template <int OP>
struct BCfg {
    static constexpr int D = 128, H = 192, NCHK = H / 32;
    static constexpr int K = 16, KL = 8, EB = 2, FRAG = 64 * KL * EB;
    static constexpr int KIN1 = D / K, KIN2 = 2 * H / K;
    static constexpr int WAVES = 8;  // two per SIMD
    static constexpr int BLOCK1 = round_up(KIN1 * FRAG + 32 * 4, 16);
    static constexpr int BLOCK2 = round_up(KIN2 * FRAG + 32 * 4, 16);
    static constexpr int PARAM_BYTES = (D + 2 * kBbMaxFeat) * 4;
    static constexpr int STAGE = round_up(cmax(BLOCK2, 4 * BLOCK1), kCopyBytes);
    static constexpr int KPF = (STAGE - PARAM_BYTES) / (4 * FRAG);  // front-end k-steps per stage
    static constexpr int PARAM_OFF = KPF * 4 * FRAG;
    static constexpr int COPIES = STAGE / kCopyBytes;
    static constexpr int LPW = (COPIES + WAVES - 1) / WAVES;
    // wave-private LDS: track table and row map, the transpose tile [32 rows][32
    // channels] (row stride padded by 16 bytes), then the first layer's A operand
    // (KIN1 fragments of 1 KiB; before it, the front end's normalised features)
    static constexpr int ROWB = 32 * EB + 16;
    static constexpr int TB_OFF = 4 * kMgMaxTr * 4 + kMgCap * 4;
    static constexpr int XA_OFF = TB_OFF + kMgCap * ROWB;
    static constexpr int WAVE_BYTES = XA_OFF + KIN1 * FRAG;
    static constexpr int FLAG_BYTES = 16;  // the tile counter of the last wave with work
    static constexpr int NSLOT_FIT = (kLdsBytesMax - FLAG_BYTES - WAVES * WAVE_BYTES) / STAGE;
    static constexpr int NSLOT = NSLOT_FIT > 5 ? 5 : NSLOT_FIT;
    static constexpr int WAVE0 = NSLOT * STAGE;
    static constexpr int FLAG_OFF = WAVE0 + WAVES * WAVE_BYTES;
    static constexpr int LDS_BYTES = FLAG_OFF + FLAG_BYTES;
    static constexpr int L1_STAGES = NCHK, L2_STAGES = 4 * NCHK;
    static_assert(NSLOT >= 2 && KPF >= 1, "stage ring");
    static_assert(kMgCap * kBbUStride * 4 <= KIN1 * FRAG, "features in the operand area");
};

// Channel of a 32-channel block that the front end's projection puts on
// product row rho: register q of lane half g (row 8 (q / 4) + 4 g + q % 4)
// receives channel 16 (q / 8) + 8 g + q % 8.
__host__ __device__ constexpr int bb_front_channel(int rho) {
    return 16 * ((4 * (rho >> 3) + (rho & 3)) >> 3) + 8 * ((rho >> 2) & 1) + ((4 * (rho >> 3) + (rho & 3)) & 7);
}
// (a permutation of the block's 32 channels)
constexpr bool bb_front_channel_is_permutation() {
    unsigned seen = 0;
    for (int rho = 0; rho < 32; ++rho) seen |= 1u << bb_front_channel(rho);
    return seen == ~0u;
}
static_assert(bb_front_channel_is_permutation(), "front-end row order");

template <int OP>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * BCfg<OP>::WAVES, 64 * BCfg<OP>::WAVES),
                          amdgpu_waves_per_eu(BCfg<OP>::WAVES / 4, BCfg<OP>::WAVES / 4)))
void tf_backbone_kernel(const float *__restrict__ feats, int nf, long long n_hits, long long x_rows,
                        const int *__restrict__ offsets, int n_tracks, const unsigned char *__restrict__ stages,
                        int n_fst, float *__restrict__ states, int *__restrict__ err) {
    using C = BCfg<OP>;
    using F = Frag<OP>;
    using FT = typename F::T;
    using FE = typename F::E;
    constexpr int SP = kMgSP, NCHK = C::NCHK, H = C::H, D = C::D, KIN1 = C::KIN1, KIN2 = C::KIN2;
    constexpr int ROWE = C::ROWB / (int)sizeof(FE);  // tile row stride (elements)
    const int S = n_fst + C::L1_STAGES + C::L2_STAGES;  // stages per tile
    const int kf = 2 * nf;                              // front-end k-steps (32 columns per feature)

    __shared__ __attribute__((aligned(16))) char smem[C::LDS_BYTES];
    const int lane = threadIdx.x & 63;
    const int wid = uniform(threadIdx.x >> 6);
    const int hh = lane >> 5, cc = lane & 31;
    char *wave_lds = smem + C::WAVE0 + wid * C::WAVE_BYTES;
    int *t_start = reinterpret_cast<int *>(wave_lds);
    int *t_len = t_start + kMgMaxTr, *t_off = t_len + kMgMaxTr, *t_id = t_off + kMgMaxTr;
    int *rowmap = t_id + kMgMaxTr;
    char *tile = wave_lds + C::TB_OFF;  // each block's states, then end states
    FT *xa1 = reinterpret_cast<FT *>(wave_lds + C::XA_OFF);  // [KIN1][64]; first the features

    const unsigned smem_lds = (unsigned)(uintptr_t)(__attribute__((address_space(3))) char *)smem;
    auto slot_lds = [&](int q) -> unsigned { return smem_lds + (q % C::NSLOT) * C::STAGE; };
#pragma unroll
    for (int q = 0; q < C::NSLOT - 1; ++q) copy_stage<C>(stages, q % S, slot_lds(q), wid, lane);
    // the stage ring as in the layer kernel: stages q .. q + NSLOT - 2 are in LDS
    // during stage q (each stage's copy has one stage's time to land), and the
    // last stage of a tile leaves its copy to the next tile
    int q = 0;
    auto advance = [&](bool last) {
        wait_vmcnt<0>();
        lds_barrier();
        if (!last) copy_stage<C>(stages, (q + C::NSLOT) % S, slot_lds(q + C::NSLOT), wid, lane);
        ++q;
    };
    auto slot = [&]() -> const char * { return smem + (q % C::NSLOT) * C::STAGE; };
    // gate a = sigmoid(g) from the pre-activation and its bias pre-scaled by
    // -log2(e); the update adds a x and keeps 1 - a of the state
    auto gate = [&](const f32x16 &ax, const f32x16 &gx, float bgv, float (&AX)[SP], float (&CF)[SP]) {
#pragma unroll
        for (int i = 0; i < SP; ++i) {
            const float e = __builtin_amdgcn_exp2f(fmaf(gx[i], -kLog2e, bgv));
            const float a = __builtin_amdgcn_rcpf(1.0f + e);
            AX[i] = a * ax[i];
            CF[i] = 1.0f - a;
        }
    };

    const long long gw = (long long)blockIdx.x * C::WAVES + wid;
    const long long nw = (long long)gridDim.x * C::WAVES;
    const int g_begin = group_begin(offsets, n_tracks, gw, nw, lane);
    const int g_end = group_begin(offsets, n_tracks, gw + 1, nw, lane);
    const int row0 = offsets[0];
    int errbits = 0;
    // a wave with a tile writes the tile's number; the workgroup stops at the
    // first tile that no wave wrote (the next write comes after later barriers)
    int *tile_flag = reinterpret_cast<int *>(smem + C::FLAG_OFF);
    if (threadIdx.x == 0) *tile_flag = 0;
    __syncthreads();
    int tile_count = 0;

    int t = g_begin;
    unsigned taken = 0;
    for (;;) {
        int n = 0, off = 0, len = 0;
        // (lane values read afresh per tile: held across the tile's layers they
        // would take registers the last layer's operands need)
        const unsigned sel =
            mg_select(offsets, g_end, row0, x_rows, n_hits, fresh_lane(), t, taken, errbits, states, H, n, off, len);
        const int k = __builtin_popcount(sel);
        const bool work = k > 0;
        wait_vmcnt<0>();
        ++tile_count;
        if (work && lane == 0) *tile_flag = tile_count;
        lds_barrier();
        if (uniform(*tile_flag) != tile_count) break;  // every wave of the workgroup is done
        copy_stage<C>(stages, (q + C::NSLOT - 1) % S, slot_lds(q + C::NSLOT - 1), wid, lane);

        unsigned sb0 = 0, sb1 = 0, eb0 = 0, eb1 = 0, st0 = 0, st1 = 0;
        if (work)
            mg_tile_meta(sel, n, off, len, t, row0, fresh_lane(), t_start, t_len, t_off, t_id, rowmap, sb0, sb1, eb0,
                         eb1, st0, st1);

        // ---- front end: r = b + W f(u) for the hit of column cc (tile row
        // slot_to_hit(cc), the first layer's operand row cc); lane half hh forms
        // the normalised features 8 hh .. 8 hh + 7 of its column
        {
            f32x16 r[4];
            float *us = reinterpret_cast<float *>(xa1);  // [32][kBbUStride]
            if (work) {
                const int ln = fresh_lane(), h2 = ln >> 5, c2 = ln & 31;
                const float *fp = reinterpret_cast<const float *>(slot() + C::PARAM_OFF);  // bias, lo, 1 / span
                const int xr = rowmap[slot_to_hit<SP>(c2)];
                const float *hp = xr >= 0 ? feats + (size_t)(xr + row0) * nf : nullptr;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int f = 8 * h2 + e;
                    if (f < nf) us[c2 * kBbUStride + f] = hp ? (hp[f] - fp[D + f]) * fp[D + kBbMaxFeat + f] : 0.f;
                }
#pragma unroll
                for (int m = 0; m < 4; ++m)
#pragma unroll
                    for (int qq = 0; qq < 16; ++qq) r[m][qq] = fp[32 * m + 16 * (qq >> 3) + 8 * h2 + (qq & 7)];
                wave_lds_sync();  // the features are in the tile
            }
            // k-step ks takes, for this lane's column, the features k = 16 ks + 8 hh + e
            // of the projection: feature ks / 2, sines (even ks) or cosines (odd ks)
            // of pi 2^s u at scales s = 8 hh + e, the lowest from the hardware
            // functions in revolutions (sin(pi 2^s u) = sin(2 pi frac(2^(s - 1) u))), each
            // next one by the double-angle formulas (the even k-step forms both)
            FT cnext = FT{};
            for (int js = 0; js < n_fst; ++js) {
                if (work) {
                    const FT *wfr = reinterpret_cast<const FT *>(slot());
                    const int k0 = js * C::KPF;
                    const int kn = kf - k0 < C::KPF ? kf - k0 : C::KPF;
                    __builtin_amdgcn_s_setprio(1);
                    for (int kl = 0; kl < kn; ++kl) {
                        const int ks = k0 + kl;
                        FT bv;
                        if (ks & 1) {
                            bv = cnext;
                        } else {
                            const float u = us[cc * kBbUStride + (ks >> 1)];
                            const float x = __builtin_amdgcn_fractf(u * (hh ? 128.0f : 0.5f));
                            float sv[8], cv[8];
                            sv[0] = __builtin_amdgcn_sinf(x);
                            cv[0] = __builtin_amdgcn_cosf(x);
#pragma unroll
                            for (int e = 1; e < 8; ++e) {
                                const float sp = sv[e - 1], cp = cv[e - 1];
                                sv[e] = (sp + sp) * cp;
                                cv[e] = (cp - sp) * (cp + sp);
                            }
                            cnext = F::pack(cv);
                            bv = F::pack(sv);
                        }
#pragma unroll
                        for (int m = 0; m < 4; ++m) r[m] = F::mma(wfr[(kl * 4 + m) * 64 + lane], bv, r[m]);
                    }
                    __builtin_amdgcn_s_setprio(0);
                }
                advance(false);
            }
            // the first layer's A operand, to LDS (the registers hold the last
            // layer's): k-step ks = 2 m + p of operand row cc holds channels
            // 32 m + 16 p + 8 hh .. + 7, registers 8 p .. 8 p + 7 of r[m]
            if (work) {
                wave_lds_sync();  // the features are read
#pragma unroll
                for (int ks = 0; ks < KIN1; ++ks) {
                    float v[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) v[e] = r[ks >> 1][8 * (ks & 1) + e];
                    xa1[ks * 64 + lane] = F::pack(v);
                }
                wave_lds_sync();
            }
        }

        // ---- first layer (input d, both blocks of a chunk and direction in one
        // stage); its states become the last layer's A operand: k-step 12 dir +
        // 2 ch + p of operand row cc holds channels dir H + 32 ch + 16 p + 8 hh .. + 7
        // of tile row slot_to_hit(cc)
        FT xa2[KIN2];
#pragma unroll
        for (int b = 0; b < 2 * NCHK; ++b) {
            const int ch = b >> 1, dir = b & 1;
            if (work) {
                const char *sl = slot() + 2 * dir * C::BLOCK1;  // both directions of a chunk per stage
                const FT *wc = reinterpret_cast<const FT *>(sl);
                const FT *wg = reinterpret_cast<const FT *>(sl + C::BLOCK1);
                f32x16 ax, gx;
#pragma unroll
                for (int i = 0; i < 16; ++i) ax[i] = gx[i] = 0.f;
                // both chains two k-steps at a time (the fences keep the weight
                // fragments in flight to four: the registers hold the second
                // layer's operands meanwhile)
                __builtin_amdgcn_s_setprio(1);
#pragma unroll
                for (int ks = 0; ks < KIN1; ks += 2) {
                    const FT x0 = xa1[ks * 64 + lane], x1 = xa1[(ks + 1) * 64 + lane];
                    ax = F::mma(x0, wc[ks * 64 + lane], ax);
                    gx = F::mma(x0, wg[ks * 64 + lane], gx);
                    ax = F::mma(x1, wc[(ks + 1) * 64 + lane], ax);
                    gx = F::mma(x1, wg[(ks + 1) * 64 + lane], gx);
                    __builtin_amdgcn_sched_barrier(0);
                }
                __builtin_amdgcn_s_setprio(0);
                ax += reinterpret_cast<const float *>(sl + KIN1 * C::FRAG)[cc];
                const float bgv = reinterpret_cast<const float *>(sl + C::BLOCK1 + KIN1 * C::FRAG)[cc];
                float AX[SP], CF[SP];
                gate(ax, gx, bgv, AX, CF);
                if (dir == 0)
                    scan_dir<true>(AX, CF, sb0, sb1, hh);
                else
                    scan_dir<false>(AX, CF, eb0, eb1, hh);
                FE *tb = reinterpret_cast<FE *>(tile);
                wave_lds_sync();  // earlier reads of the tile are done
#pragma unroll
                for (int i = 0; i < SP; ++i) {
                    // (the update and its conversion kept apart, as in the layer kernel)
                    float v = AX[i];
                    asm volatile("" : "+v"(v));
                    tb[(SP * hh + i) * ROWE + cc] = (FE)v;
                }
                wave_lds_sync();
                const FE *row = tb + slot_to_hit<SP>(cc) * ROWE + 8 * hh;
                xa2[12 * dir + 2 * ch] = *reinterpret_cast<const FT *>(row);
                xa2[12 * dir + 2 * ch + 1] = *reinterpret_cast<const FT *>(row + 16);
            }
            if (dir == 1) advance(false);
            __builtin_amdgcn_sched_barrier(0);  // blocks one after the other (registers)
        }

        // ---- last layer (input 2H, one block per stage): end states through the
        // tile, stored after the block's barrier (as in the layer kernel)
        constexpr int PPR = 8;  // 16-byte pieces per row of 32 fp32 states
        constexpr int NPEND = kMgMaxTr * PPR / 64;
        u32x4 pv[NPEND];
        int prow[NPEND];
        int pcol = 0;
#pragma unroll
        for (int p = 0; p < NPEND; ++p) prow[p] = -1;
        auto flush = [&]() {
#pragma unroll
            for (int p = 0; p < NPEND; ++p) {
                const int g = (lane + 64 * p) % PPR;
                if (prow[p] >= 0) *reinterpret_cast<u32x4 *>(states + (size_t)prow[p] * 2 * H + pcol + 4 * g) = pv[p];
                prow[p] = -1;
            }
        };
        for (int ch = 0; ch < NCHK; ++ch) {
#pragma unroll
            for (int dir = 0; dir < 2; ++dir) {
                f32x16 ax;
                if (work) {
                    const FT *wc = reinterpret_cast<const FT *>(slot());
#pragma unroll
                    for (int i = 0; i < 16; ++i) ax[i] = 0.f;
                    __builtin_amdgcn_s_setprio(1);
#pragma unroll
                    for (int ks = 0; ks < KIN2; ++ks) {
                        ax = F::mma(xa2[ks], wc[ks * 64 + lane], ax);
                        if (ks % 4 == 3) __builtin_amdgcn_sched_barrier(0);  // four fragments in flight
                    }
                    __builtin_amdgcn_s_setprio(0);
                    ax += reinterpret_cast<const float *>(slot() + KIN2 * C::FRAG)[cc];
                }
                advance(false);
                flush();  // the previous block's end states
                if (work) {
                    const FT *wg = reinterpret_cast<const FT *>(slot());
                    f32x16 gx;
#pragma unroll
                    for (int i = 0; i < 16; ++i) gx[i] = 0.f;
                    __builtin_amdgcn_s_setprio(1);
#pragma unroll
                    for (int ks = 0; ks < KIN2; ++ks) {
                        gx = F::mma(xa2[ks], wg[ks * 64 + lane], gx);
                        if (ks % 4 == 3) __builtin_amdgcn_sched_barrier(0);
                    }
                    __builtin_amdgcn_s_setprio(0);
                    const float bgv = reinterpret_cast<const float *>(slot() + KIN2 * C::FRAG)[cc];
                    float AX[SP], CF[SP];
                    gate(ax, gx, bgv, AX, CF);
                    if (dir == 0)
                        scan_dir<true>(AX, CF, sb0, sb1, hh);
                    else
                        scan_dir<false>(AX, CF, eb0, eb1, hh);
                    pcol = dir * H + 32 * ch;
                    // forward state at a track's last row, reverse state at its first row,
                    // to row j of the tile (the track's index in it)
                    constexpr int ROWF = 32 + 4;
                    float *tf = reinterpret_cast<float *>(tile);
                    const unsigned sw = hh ? st1 : st0;
                    const unsigned mw = dir == 0 ? (hh ? eb1 : eb0) : sw;
                    const int jb = hh ? __builtin_popcount(st0) - 1 : -1;
                    wave_lds_sync();  // earlier reads of the tile are done
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
                        pv[p] = *reinterpret_cast<const u32x4 *>(tf + j * ROWF + 4 * g);
                    }
                }
                advance(ch == NCHK - 1 && dir == 1);
            }
        }
        flush();  // the tile's last block
    }
    if (errbits && lane == 0) atomicOr(err, errbits);
}

template <int OP>
hipError_t launch_backbone(const float *feats, int nf, long long n_hits, long long x_rows, const int32_t *offsets,
                           int32_t n_tracks, const unsigned char *stages, int n_fst, float *states, int *err,
                           int cu_count, hipStream_t stream) {
    using C = BCfg<OP>;
    long long waves = (n_tracks + 7) / 8;
    long long blocks = (waves + C::WAVES - 1) / C::WAVES;
    if (blocks > cu_count) blocks = cu_count;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL((tf_backbone_kernel<OP>), dim3((unsigned)blocks), dim3(64 * C::WAVES), 0, stream, feats, nf,
                       n_hits, x_rows, offsets, (int)n_tracks, stages, n_fst, states, err);
    return hipGetLastError();
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
    const unsigned char *bb_stages = nullptr;  // the fused backbone's stages (null: not this model)
    int bb_nfs = 0;                   // their front-end stages
    bool fused = false;               // run the fused backbone
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
    // the fused backbone (16-bit, Fourier front end, d 128, H 192, two layers):
    // its own stage sequence, every stage BCfg::STAGE bytes
    using BC = BCfg<OP_F16>;
    static_assert(BCfg<OP_BF16>::STAGE == BC::STAGE && BCfg<OP_BF16>::KPF == BC::KPF, "fused geometry");
    const bool fusable = half && nf > 0 && d == BC::D && H == BC::H && L == 2;
    const int bb_nfs = fusable ? (2 * nf + BC::KPF - 1) / BC::KPF : 0;
    const size_t bb_off = (total + 255) & ~size_t(255);
    if (fusable) total = bb_off + (size_t)(bb_nfs + BC::L1_STAGES + BC::L2_STAGES) * BC::STAGE;
    std::vector<unsigned char> hb(total, 0);
    auto put_elem = [&](unsigned char *sp, size_t i, float v) {
        if (half) {
            const uint16_t bb = bits16(v, bf);
            std::memcpy(sp + 2 * i, &bb, 2);
        } else {
            std::memcpy(sp + 4 * i, &v, 4);
        }
    };
    // one weight block: lane (s, c) value e of k-step ks holds W[row rbase + c][column
    // ks K + s KL + e]; then the block's 32 biases (the gate's times -log2(e) for the
    // 16-bit modes)
    auto put_block = [&](unsigned char *sp, const float *W, const float *b, int din, int rbase, bool gate_part) {
        const int KIN = din / K;
        for (int ks = 0; ks < KIN; ++ks)
            for (int lane = 0; lane < 64; ++lane)
                for (int e = 0; e < KL; ++e)
                    put_elem(sp, ((size_t)ks * 64 + lane) * KL + e,
                             W[(size_t)(rbase + lane % 32) * din + ks * K + (lane / 32) * KL + e]);
        unsigned char *bp = sp + (size_t)KIN * 64 * KL * (half ? 2 : 4);
        for (int c = 0; c < 32; ++c) {
            float bv = b[rbase + c];
            if (half && gate_part) bv = (float)(-1.4426950408889634 * (double)bv);
            std::memcpy(bp + 4 * c, &bv, 4);
        }
    };
    const float *lw = blob + front_floats(d, nf);
    for (int l = 0; l < L; ++l) {
        const int din = l == 0 ? d : 2 * H;
        const MGeom g = stage_bytes_of(op, din);
        const float *W = lw, *b = lw + (size_t)4 * H * din;
        // layered: for each 32-channel chunk and direction the candidate block starts
        // a stage; the gate block follows it in the same stage (merged) or starts the
        // next one.  Fused: layer 0 merged, layer 1 one block per stage.
        unsigned char *dst = hb.data() + loff[l];
        unsigned char *fdst = fusable ? hb.data() + bb_off + (size_t)(bb_nfs + (l == 0 ? 0 : BC::L1_STAGES)) * BC::STAGE
                                      : nullptr;
        for (int ch = 0; ch < H / 32; ++ch)
            for (int dir = 0; dir < 2; ++dir)
                for (int part = 0; part < 2; ++part) {
                    const int rbase = dir * 2 * H + part * H + 32 * ch;
                    put_block(dst, W, b, din, rbase, part == 1);
                    dst += (g.merge && part == 0) ? g.block : (g.merge ? g.stage - g.block : g.stage);
                    if (fusable) {
                        put_block(fdst + (l == 0 ? (2 * dir + part) * BC::BLOCK1 : 0), W, b, din, rbase, part == 1);
                        fdst += l == 0 ? (dir == 1 && part == 1 ? BC::STAGE : 0) : BC::STAGE;
                    }
                }
        lw += (size_t)4 * H * din + (size_t)4 * H;
    }
    if (fusable) {
        // front-end stages: lane (s, c) value e of k-step ks, channel block m holds
        // fe.W[channel 32 m + bb_front_channel(c)][column 16 ks + 8 s + e] (column k:
        // feature k / 32, cosine if bit 4 of k is set, scale k % 16); the first stage
        // then holds fe.b [d], lo [16] and 1 / (hi - lo) [16] (fp32: the span and its
        // inverse each rounded to float32, as the layered front end takes them)
        const float *f_lo = blob, *f_hi = blob + nf, *fW = blob + 2 * nf, *fB = fW + (size_t)d * 32 * nf;
        const int KF32 = 32 * nf;
        for (int js = 0; js < bb_nfs; ++js) {
            unsigned char *sp = hb.data() + bb_off + (size_t)js * BC::STAGE;
            for (int kl = 0; kl < BC::KPF && js * BC::KPF + kl < 2 * nf; ++kl)
                for (int m = 0; m < 4; ++m)
                    for (int lane = 0; lane < 64; ++lane)
                        for (int e = 0; e < 8; ++e) {
                            const size_t col = (size_t)(js * BC::KPF + kl) * 16 + (lane / 32) * 8 + e;
                            put_elem(sp, ((size_t)(kl * 4 + m) * 64 + lane) * 8 + e,
                                     fW[(size_t)(32 * m + bb_front_channel(lane % 32)) * KF32 + col]);
                        }
        }
        float par[BC::D + 2 * kBbMaxFeat];
        for (int c = 0; c < BC::D; ++c) par[c] = fB[c];
        for (int f = 0; f < kBbMaxFeat; ++f) {
            par[BC::D + f] = f < nf ? f_lo[f] : 0.0f;
            const float span = f < nf ? f_hi[f] - f_lo[f] : 1.0f;
            par[BC::D + kBbMaxFeat + f] = 1.0f / span;
        }
        std::memcpy(hb.data() + bb_off + BC::PARAM_OFF, par, sizeof(par));
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
    if (fusable) {
        h->bb_stages = reinterpret_cast<const unsigned char *>(h->dmem + bb_off);
        h->bb_nfs = bb_nfs;
        h->fused = true;
    }
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
    if (h->fused) {
        // one launch; the workspace is not touched, but bounds the rows as on the layered path
        const hipError_t e =
            h->op == OP_BF16
                ? launch_backbone<OP_BF16>(hits, h->cfg.n_features, n_hits, rows, offsets, n_tracks, h->bb_stages,
                                           h->bb_nfs, states, h->err, h->cu_count, stream)
                : launch_backbone<OP_F16>(hits, h->cfg.n_features, n_hits, rows, offsets, n_tracks, h->bb_stages,
                                          h->bb_nfs, states, h->err, h->cu_count, stream);
        return e == hipSuccess ? TF_OK : TF_EHIP;
    }
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

extern "C" tf_status tf_mingru_set_fused(tf_mingru *h, int fused) {
    if (!h) return TF_EINVAL;
    if (fused && !h->bb_stages) return TF_EUNSUPPORTED;
    h->fused = fused != 0;
    return TF_OK;
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
