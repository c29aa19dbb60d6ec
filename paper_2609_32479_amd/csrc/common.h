// Device-side building blocks shared by the library's kernels (gfx950):
// operand types, matrix-core fragments, wave and workgroup synchronisation,
// lane masks of the segmented scans, the tile's hit-slot order, the packing
// of tracks into wave tiles, and the direct-to-LDS weight-stage copy.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
typedef __attribute__((ext_vector_type(8))) float f32x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

// Matrix-core operand types.  OP_F32: fp32 weights and operands
// (v_mfma_f32_32x32x2_f32).  OP_BF16: bf16 weights and bf16 activation
// operands (v_mfma_f32_32x32x16_bf16).  OP_F16: weights converted to fp16
// (exact for bf16 values in the fp16 normal range) and fp16 activation
// operands (v_mfma_f32_32x32x16_f16).
// Accumulation is fp32 in all three.
enum { OP_F32 = 0, OP_BF16 = 1, OP_F16 = 2 };

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kRmsEps = 1e-6f;
// The fp32 gate clamps |pre-activation| to 80 and the 16-bit head clamps the
// SiLU exponent to 80 log2(e), so that exp stays finite; the change in the
// result is below exp(-80).
constexpr float kGateClamp = 80.0f * kLog2e;
constexpr int kLdsBytesMax = 160 * 1024;
constexpr int kCopyBytes = 1024;  // one wave-wide 16-byte-per-lane copy

constexpr int cmax(int a, int b) { return a > b ? a : b; }
constexpr int round_up(int v, int m) { return (v + m - 1) / m * m; }

template <int OP> struct Frag;
template <> struct Frag<OP_BF16> {
    typedef bf16x8 T;
    typedef __bf16 E;
    static __device__ __forceinline__ f32x16 mma(T a, T b, f32x16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ f32x4 mma16(T a, T b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ T pack(const float *v) {
        f32x8 f = {v[0], v[1], v[2], v[3], v[4], v[5], v[6], v[7]};
        return __builtin_convertvector(f, bf16x8);
    }
};
template <> struct Frag<OP_F16> {
    typedef f16x8 T;
    typedef _Float16 E;
    static __device__ __forceinline__ f32x16 mma(T a, T b, f32x16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ f32x4 mma16(T a, T b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ T pack(const float *v) {
        f32x8 f = {v[0], v[1], v[2], v[3], v[4], v[5], v[6], v[7]};
        return __builtin_convertvector(f, f16x8);
    }
};
template <> struct Frag<OP_F32> {
    typedef float T;
    typedef float E;
    static __device__ __forceinline__ f32x16 mma(T a, T b, f32x16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ T pack(const float *v) { return v[0]; }
};

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The lane index, read afresh: values derived from it are formed where they
// are used instead of being held in registers across the whole kernel.
__device__ __forceinline__ int fresh_lane() {
    int l;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
    return l;
}
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Lane mask (wave-uniform, 64 bits) of the lanes whose stream has bit p set:
// lanes 0-31 follow b0, lanes 32-63 follow b1.
__device__ __forceinline__ unsigned long long half_mask(unsigned b0, unsigned b1, int p) {
    typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
    const u32x2 m = {(unsigned)((int)(b0 << (31 - p)) >> 31), (unsigned)((int)(b1 << (31 - p)) >> 31)};
    return __builtin_bit_cast(unsigned long long, m);
}

// v in lanes outside m, 0 in lanes of m: one v_cndmask with the mask in SGPRs.
__device__ __forceinline__ float zero_lanes(float v, unsigned long long m) {
    float r;
    asm("v_cndmask_b32_e64 %0, %1, 0, %2" : "=v"(r) : "v"(v), "s"(m));
    return r;
}

// Tile hit index held in hit slot s (0 <= s < CAP).  Slot s = 32 n + 8 i + 4 g + j
// is row 8 i + 4 g + j of hit tile n in the input projection; that row lands
// in lanes of half g at accumulator register 4 i + j, which is position
// 16 n + 4 i + j of stream g, i.e. tile hit SP * g + 16 n + 4 i + j.
template <int SP>
__device__ __forceinline__ int slot_to_hit(int s) {
    int n = s >> 5, i = (s >> 3) & 3, g = (s >> 2) & 1, j = s & 3;
    return SP * g + 16 * n + 4 * i + j;
}

// Folded slot order of the encoder: stream 0 (lanes 0-31) holds tile rows
// 0 .. SP-1 in register order, stream 1 (lanes 32-63) holds rows 2 SP-1 down to
// SP, i.e. register position p of stream 1 is row 2 SP - 1 - p.  An ascending
// pass over the registers then runs stream 0 forward and stream 1 in reverse,
// and a descending pass the other two directions; both meet at rows SP - 1 and
// SP, so one lane swap carries a track across the streams.
template <int SP>
__device__ __forceinline__ int slot_to_row(int s) {
    const int n = s >> 5, i = (s >> 3) & 3, g = (s >> 2) & 1, j = s & 3;
    const int p = 16 * n + 4 * i + j;
    return g ? 2 * SP - 1 - p : p;
}

// The SP row bits of stream 1 (rows SP .. 2 SP - 1 of a row mask) in register
// order: bit p is row 2 SP - 1 - p.
template <int SP>
__device__ __forceinline__ unsigned stream1_bits(unsigned long long rows) {
    const unsigned hi = unsigned(rows >> SP) & (SP >= 32 ? 0xffffffffu : ((1u << SP) - 1u));
    return __builtin_bitreverse32(hi) >> (32 - SP);
}

// Copy of one weight stage from global memory straight into an LDS slot:
// global_load_lds_dwordx4 moves 16 bytes per lane, 1 KiB per wave
// instruction, into LDS at M0 + 16 * lane.  Each wave copies the pieces
// w, w + WAVES, ...; waves with fewer pieces repeat the last one (same bytes to
// the same place), so every wave issues exactly LPW loads per stage and can
// wait for an older stage with a constant vmcnt.  The instruction is written
// out because the compiler, which cannot tell the ring slots apart, would
// otherwise wait for every such load before each LDS access; the kernel keeps
// the count itself (wait_vmcnt).  The LDS address is an operand bound to M0,
// so the compiler writes M0 itself and knows it is read here; the s_nop is
// the one wait state the hardware needs between that write and the load.
__device__ __forceinline__ void lds_dma16(const void *gsrc, unsigned lds_addr) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(gsrc), "{m0}"(__builtin_amdgcn_readfirstlane(lds_addr))
                 : "memory");
}

// slot_lds: LDS byte address of the slot.
template <class C>
__device__ __forceinline__ void copy_stage(const unsigned char *stages, int s, unsigned slot_lds, int wid, int lane) {
    const unsigned char *src = stages + (size_t)s * C::STAGE + lane * 16;
#pragma unroll
    for (int i = 0; i < C::LPW; ++i) {
        int piece = wid + i * C::WAVES;
        piece = piece < C::COPIES ? piece : C::COPIES - 1;
        lds_dma16(src + piece * kCopyBytes, slot_lds + piece * kCopyBytes);
    }
}

// Packing of one wave tile from a window of up to 32 tracks, one per lane
// (lanes 0..31; len: that lane's track length).  cand: the window lanes that
// may join the tile, each at most CAP long.  The tile takes the oldest
// candidate, then (PAIR) the one or two other candidates whose lengths fill
// the remaining rows best (the lowest lanes among equals), then the rest
// first-fit in window order, up to MAXTR tracks and CAP rows.  A track's result does not
// depend on the tile it lands in, so the packing only decides how full the
// tiles are (about 94 % for lengths 8..20 in 32 rows, against 90 % for plain
// first-fit).  Returns the selected lanes (wave-uniform); rows: their total
// length.  The length masks are built in scalar registers, one candidate at a
// time, so the packing issues no cross-lane traffic through LDS.  Without PAIR
// the tile is plain first-fit from the oldest candidate: cheaper per tile,
// for kernels whose tiles are short enough that the search does not pay.
template <int CAP, int MAXTR, bool PAIR>
__device__ __forceinline__ unsigned pack_tile(unsigned cand, int len, int lane, int &rows) {
    static_assert(CAP <= 64 && MAXTR >= 3, "tile shape");
    typedef unsigned long long u64;
    const int first = __builtin_ctz(cand);
    int n = __builtin_amdgcn_readlane(len, first);
    unsigned sel = 1u << first;
    const unsigned rest = cand & ~sel;
    const int room = CAP - n;
    if constexpr (PAIR) {
        // bit l - 1 of m1: a length l among the other candidates that fit beside
        // the first; of m2: one that at least two of them have
        u64 m1 = 0, m2 = 0;
        for (unsigned c = rest; c; c &= c - 1u) {
            const int li = __builtin_amdgcn_readlane(len, __builtin_ctz(c));
            if (li <= room) {
                const u64 b = 1ull << (li - 1);
                m2 |= m1 & b;
                m1 |= b;
            }
        }
        auto upto = [](int r) -> u64 { return r <= 0 ? 0ull : r >= 64 ? ~0ull : (1ull << r) - 1ull; };
        const u64 ms = m1 & upto(room);
        const int single = ms ? 64 - __builtin_clzll(ms) : 0;
        // per candidate lane: the longest other length that fits beside it
        const bool av = lane < 32 && ((rest >> (lane & 31)) & 1u) && len <= room;
        int pair = 0, partner = 0;
        if (av) {
            const int left = room - len;
            u64 m = m1 & upto(left);
            if (len <= left && !((m2 >> (len - 1)) & 1ull)) m &= ~(1ull << (len - 1));  // not itself
            if (m) {
                partner = 64 - __builtin_clzll(m);
                pair = len + partner;
            }
        }
        // the best pair sum above the best single, counted down from the room left
        int best = 0;
        unsigned long long who = 0;
        for (int sum = room; sum > single; --sum) {
            who = __ballot(av && pair == sum);
            if (who) {
                best = sum;
                break;
            }
        }
        if (best) {
            const int i = __builtin_ctzll(who);
            const int pl = __builtin_amdgcn_readlane(partner, i);
            const bool mate = lane < 32 && lane != i && ((rest >> (lane & 31)) & 1u) && len == pl;
            const int j = __builtin_ctzll(__ballot(mate));
            sel |= (1u << i) | (1u << j);
            n += best;
        } else if (single > 0) {
            sel |= 1u << __builtin_ctzll(__ballot(av && len == single));
            n += single;
        }
    }
    // first-fit over the rest, in window order.  A lane passed over once never
    // fits later (the rows only fill up), so each step takes the lowest remaining
    // lane whose track fits the rows left: one ballot per track taken.
    int k = __builtin_popcount(sel);
    unsigned left = rest & ~sel;
    while (left && k < MAXTR && n < CAP) {
        const unsigned fit = left & unsigned(__ballot(lane < 32 && len <= CAP - n));
        if (!fit) break;
        const int i = __builtin_ctz(fit);
        n += __builtin_amdgcn_readlane(len, i);
        sel |= 1u << i;
        left &= ~(1u << i);
        ++k;
    }
    rows = n;
    return sel;
}

// First track of wave group g of ng: the tracks are split into ng contiguous
// groups of about equal hit rows.  The result is the number of tracks i with
// offsets[i] < offsets[0] + R g / ng (R: the rows of all tracks), found by a
// 64-ary search that follows the leading run of true probes; that count grows
// with the target for any offsets array, so the groups of consecutive g tile
// [0, n_tracks) even when the offsets are invalid.  Without rows (R <= 0) the
// split is by track count.  Wave-uniform.
__device__ __forceinline__ int group_begin(const int *__restrict__ offsets, int n_tracks, long long g, long long ng,
                                           int lane) {
    if (g <= 0) return 0;
    if (g >= ng) return n_tracks;
    const long long o0 = offsets[0];
    const long long rows = (long long)offsets[n_tracks] - o0;
    if (rows <= 0) return int((long long)n_tracks * g / ng);
    const long long target = o0 + rows * g / ng;
    int lo = 0, hi = n_tracks;  // the count lies in [lo, hi]
    while (hi > lo) {
        const int stride = (hi - lo + 63) / 64;
        const int p = lo + (lane + 1) * stride - 1;  // probes below hi
        const bool below = p < hi && (long long)offsets[p] < target;
        const unsigned long long nb = ~__ballot(below);
        const int c = nb ? __builtin_ctzll(nb) : 64;  // leading true probes
        const int nlo = lo + c * stride;
        const int phi = lo + (c + 1) * stride - 1;  // the first false probe, if any
        hi = phi < hi ? phi : hi;
        lo = nlo < hi ? nlo : hi;
    }
    return lo;
}

// Workgroup barrier that orders LDS only (the kernel shares nothing through
// global memory within a workgroup).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// s_waitcnt vmcnt(N) with the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

}  // namespace
