// Device-side building blocks shared by the gradient-dropping kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gd {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / kWave;

// Sort key of a value: its IEEE bit pattern with the sign cleared.  Unsigned
// order of keys is the order of |x| (with -0 == +0, Inf above every finite
// value and NaN above Inf).  Every key is below 2^31.
constexpr uint32_t kNoKey = 0xFFFFFFFFu;  // above every key: "nothing qualifies"

// The 31 key bits are resolved in three radix digits, most significant
// first: 10, 8 and 13 bits.  Digit 1 is narrow because the candidates that
// share the threshold's digit 0 are many and every bin a block touches costs
// one global atomic; digit 2 is wide because few candidates share the first
// 18 bits, so its histogram stays sparse.
constexpr int kD0Shift = 21, kNB0 = 1024;  // key bits 30..21
constexpr int kD1Shift = 13, kNB1 = 256;   // key bits 20..13
constexpr int kNB2 = 8192;                 // key bits 12..0

// Histogram words per threshold segment: one histogram per digit, and digit
// 2 also in 256 coarse bins of 32 (its top 8 bits) for a two-step pick.
constexpr int kNB2c = 256, kD2cShift = 5;
// Digit 1 is counted into kH1Copies copies of its histogram, picked by block
// number, so that the many blocks of one large segment spread their adds
// over several addresses per bin; the pick of digit 1 sums the copies.
// Digit 0 and the coarse bins of digit 2 likewise under a global threshold,
// whose one segment takes every block's adds (per tensor, summing the copies
// costs more than it saves).
constexpr int kH1Copies = 8;
constexpr int kH0Copies = 4;
constexpr int kH2cCopies = 8;
constexpr int kHistH0 = 0, kHistH1 = kH0Copies * kNB0, kHistH2 = kHistH1 + kH1Copies * kNB1, kHistH2c = kHistH2 + kNB2;
constexpr int kHistWords = kH0Copies * kNB0 + kH1Copies * kNB1 + kNB2 + kH2cCopies * kNB2c;

// Sampling: units of 16 consecutive elements (one 64-byte line per array),
// at most kMaxUnits units per segment.  A sample key is the top 16 bits of
// the 31-bit key (relative resolution 2^-8), kNoKey16 marks a missing one.
constexpr int kUnit = 16;
constexpr int kMaxUnits = 4096;
constexpr int kMinSpreadUnits = 1024;
constexpr int kSampleThreads = 128;    // gather blocks: one unit per thread
constexpr int kBracketThreads = 1024;  // one block per segment
constexpr int kBracketUnits = kMaxUnits / kBracketThreads;  // units held per thread
constexpr int kSampleBlocks = kMaxUnits / kSampleThreads;

// Sample units of a segment with n16 16-element blocks: all of them when
// there are at most kMaxUnits, else about one unit per 64 blocks (one
// 16-byte group per 256 elements and input array), clamped to
// [kMinSpreadUnits, kMaxUnits].
__host__ __device__ constexpr uint32_t sample_unit_count(uint32_t n16) {
    return n16 <= (uint32_t)kMaxUnits ? n16
           : n16 / 64 < (uint32_t)kMinSpreadUnits ? (uint32_t)kMinSpreadUnits
           : n16 / 64 > (uint32_t)kMaxUnits ? (uint32_t)kMaxUnits
           : n16 / 64;
}
constexpr uint32_t kNoKey16 = 0xFFFFu;
constexpr int kK16Shift = 15;           // key16 = key >> 15
constexpr int kS0Shift = 6, kSNB1 = 64;
constexpr int kBracketWin = 4;  // coarse digits whose fine histograms one bracket pass builds
constexpr int kSHistWords = 1024 + 2;  // per segment: digit histogram of the sample, valid and zero counts  // key16 digits: bits 15..6 (= key digit 0), bits 5..0

// Sampled-threshold mode: sampler blocks of 256 threads with 4 sample
// positions each; a top digit of 11 key bits (2048 bins), counted into one of
// 8 copies of the segment histogram by block number, so that blocks adding to
// the same hot bin rarely meet; the selection block gathers up to 8192 keys
// sharing the digit into LDS, loading 8 keys per thread at a time.
constexpr int kSsThreads = 256;
constexpr int kSsCopies = 8;
constexpr int kSsPerThread = 4;
constexpr int kSsNB0 = 2048;
constexpr int kSsD0Shift = 20;
constexpr int kSsSelThreads = 1024;
constexpr int kSsList = 8192;
constexpr int kSsBatch = 8;

// Elements per unit of the dense pass (one block).
constexpr uint32_t kUnitLen = 1024;
// Units per block of the candidate-count scan.
constexpr uint32_t kScanUnits = 1024;
constexpr int kScanThreads = 256;

// Per threshold segment state, written by one kernel and read by later ones.
struct SegState {
    uint32_t lo;    // candidates: key >= lo
    uint32_t hi;    // the dense pass wrote residual = +0 where key >= hi
    uint32_t clo;   // number of candidates (key >= lo)
    uint32_t miss;  // 1 when fewer than k candidates: every element becomes one
    uint32_t d0;    // digit 0 of the threshold key (key >> 21)
    uint32_t r1;    // rank of the threshold among candidates with that digit 0
    uint32_t p18;   // key >> 13 of the threshold key
    uint32_t r2;    // rank among candidates with that prefix
    uint32_t thr;   // the threshold key T (kNoKey when nothing is kept)
    uint32_t need;  // entries with key == T to keep, lowest index first
    uint32_t zero;  // 1 when fewer than k keys are nonzero and all of them are candidates: T = 0
    uint32_t runs;  // kept between calls: 1 when the last sample's units counted like independent
                    // draws, so the next call samples one run of 16 neighbours per unit
    uint32_t pad[4];
};

__device__ __forceinline__ uint32_t key_of(float x) { return __float_as_uint(x) & 0x7FFFFFFFu; }

// A load that stays where it is written.  A relaxed atomic of wave scope is a
// plain load to the hardware, but the compiler neither sinks it past a branch
// nor drops it, so loads that do not depend on one another can all be put in
// flight at the start of a kernel instead of one round trip after another.
__device__ __forceinline__ uint32_t load_early(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// This wave's index in its block, in a scalar register: the compiler then
// knows it is the same in every lane, so values indexed by it (kernel
// arguments, table entries) are read with scalar loads.
__device__ __forceinline__ uint32_t wave_index() { return __builtin_amdgcn_readfirstlane(threadIdx.x / kWave); }

// Number of set bits of m in lanes below this one.
__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

__device__ __forceinline__ uint32_t popc64(uint64_t m) { return (uint32_t)__popcll(m); }

// Orders this wave's LDS accesses around the call (a wave runs its LDS
// operations in order; this stops the compiler moving them across).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Value of v in lane `src` of the wave (src the same in every lane).
__device__ __forceinline__ uint32_t lane_value(uint32_t v, int src) {
    return (uint32_t)__builtin_amdgcn_readlane((int)v, src);
}

// Inclusive prefix sum over the 64 lanes, in registers: DPP shifts by 1, 2, 4
// and 8 within each 16-lane row, then the last lane of row 0 (row 2) added
// to row 1 (row 3) and the last lane of row 1 to rows 2 and 3.  A lane whose
// DPP source lies outside its row, or whose row is masked off, adds the
// `old` operand, 0.  (Cross-lane shuffles would go through the LDS crossbar,
// one round trip per step.)  Every lane of the wave must be active.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);  // row_shr:1
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);  // row_shr:2
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);  // row_shr:4
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);  // row_shr:8
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);  // row_bcast:15, rows 1 and 3
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);  // row_bcast:31, rows 2 and 3
    return v;
}

// Sum over the 64 lanes, in every lane.  Every lane must be active.
__device__ __forceinline__ uint32_t wave_sum(uint32_t v) { return lane_value(wave_incl_scan(v), kWave - 1); }

// Minimum over the 64 lanes, in every lane, by the same DPP steps (`old` is
// then the identity of min).  Every lane must be active.
__device__ __forceinline__ uint32_t wave_min(uint32_t v) {
    constexpr int kId = -1;  // 0xFFFFFFFF
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(kId, (int)v, 0x111, 0xF, 0xF, false));  // row_shr:1
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(kId, (int)v, 0x112, 0xF, 0xF, false));  // row_shr:2
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(kId, (int)v, 0x114, 0xF, 0xF, false));  // row_shr:4
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(kId, (int)v, 0x118, 0xF, 0xF, false));  // row_shr:8
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(kId, (int)v, 0x142, 0xA, 0xF, false));  // row_bcast:15
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp(kId, (int)v, 0x143, 0xC, 0xF, false));  // row_bcast:31
    return lane_value(v, kWave - 1);
}

// Maximum over this lane and the lanes below it (0 for none), by the same
// DPP steps as wave_incl_scan.  Every lane must be active.
__device__ __forceinline__ uint32_t wave_incl_max(uint32_t v) {
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false));  // row_shr:1
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false));  // row_shr:2
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false));  // row_shr:4
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false));  // row_shr:8
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false));  // row_bcast:15
    v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false));  // row_bcast:31
    return v;
}

// v of the lane below (0 in lane 0): DPP wave_shr:1.  Every lane must be active.
__device__ __forceinline__ uint32_t lane_below_value(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x138, 0xF, 0xF, false);
}

// v of the DPP source lane, both halves of the double moved with control
// CTRL in the rows ROW_MASK enables; a lane with no source gets -0.0, the
// identity of floating-point addition (x + -0.0 is x for every x, zeros too).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_f64(double v) {
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, CTRL, ROW_MASK, 0xF, false);
    const uint32_t hi =
        (uint32_t)__builtin_amdgcn_update_dpp((int)0x80000000u, (int)(uint32_t)(b >> 32), CTRL, ROW_MASK, 0xF, false);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Sum over the 64 lanes, in every lane: the steps of wave_incl_scan on
// doubles (a fixed order, so the result is the same on every run), then the
// last lane's total.  Every lane must be active.
__device__ __forceinline__ double wave_sum(double v) {
    v += dpp_f64<0x111, 0xF>(v);  // row_shr:1
    v += dpp_f64<0x112, 0xF>(v);  // row_shr:2
    v += dpp_f64<0x114, 0xF>(v);  // row_shr:4
    v += dpp_f64<0x118, 0xF>(v);  // row_shr:8
    v += dpp_f64<0x142, 0xA>(v);  // row_bcast:15, rows 1 and 3
    v += dpp_f64<0x143, 0xC>(v);  // row_bcast:31, rows 2 and 3
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = lane_value((uint32_t)b, kWave - 1), hi = lane_value((uint32_t)(b >> 32), kWave - 1);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Rank query on a histogram of NB bins (bin = digit value): find the digit
// holding the r-th largest element (r >= 1) and the number of elements in
// higher digits.  Returns false when the histogram holds fewer than r
// elements.  Called by a whole wave; hist may be global or LDS memory.
template <int NB, int C = 1>
__device__ bool wave_pick(const uint32_t* hist, uint32_t r, uint32_t& digit, uint32_t& above) {
    constexpr int B = NB >= kWave ? NB / kWave : 1;
    const int lane = lane_id();
    const int top = NB - lane * B;  // this lane owns bins [top - B, top), high to low (none when top <= 0)
    uint32_t c[B];
    uint32_t sum = 0;
#pragma unroll
    for (int i = 0; i < B; ++i) {
        uint32_t x = 0;
        if (top - 1 - i >= 0)
#pragma unroll
            for (int j = 0; j < C; ++j) x += hist[j * NB + top - 1 - i];  // C copies, NB words apart
        c[i] = x;
        sum += c[i];
    }
    const uint32_t incl = wave_incl_scan(sum);
    const uint32_t excl = incl - sum;
    const bool mine = excl < r && r <= incl;
    const uint64_t m = ballot(mine);
    if (m == 0) {
        digit = 0;
        above = lane_value(incl, kWave - 1);
        return false;
    }
    const int src = __ffsll((unsigned long long)m) - 1;
    uint32_t d = 0, ab = 0;
    if (mine) {
        bool found = false;
        uint32_t acc = excl;
#pragma unroll
        for (int i = 0; i < B; ++i) {
            if (!found && acc + c[i] >= r) {
                d = (uint32_t)(top - 1 - i);
                ab = acc;
                found = true;
            }
            acc += c[i];
        }
    }
    digit = lane_value(d, src);
    above = lane_value(ab, src);
    return true;
}

// Adds 1 to h[bin] for every active lane (an LDS atomic; lanes that hit the
// same bin are serialised by the hardware, which is cheaper than combining
// them first with cross-lane operations).
__device__ __forceinline__ void lds_hist_add(uint32_t* h, uint32_t bin, bool active) {
    if (active) atomicAdd(&h[bin], 1u);
}

// The same for a histogram of 16-bit counters, two bins per word (bin 2i in
// the low half of word i); each count must stay below 2^16.
__device__ __forceinline__ void lds_hist_add16(uint32_t* h, uint32_t bin, bool active) {
    if (active) atomicAdd(&h[bin >> 1], 1u << ((bin & 1u) << 4));
}

// lds_hist_add16 for a whole wave (every lane calls it): when all active
// lanes hold one bin (many equal keys, such as exact zeros or values of a
// narrower float type), one lane adds their count, instead of 64 atomics on
// one LDS word that the LDS would serialise.
__device__ __forceinline__ void lds_hist_add16_wave(uint32_t* h, uint32_t bin, bool active) {
    const uint64_t m = ballot(active);
    if (m == 0) return;
    const int first = __ffsll((unsigned long long)m) - 1;
    const uint32_t b0 = lane_value(bin, first);
    if (ballot(active && bin == b0) == m) {
        if (lane_id() == first) atomicAdd(&h[b0 >> 1], popc64(m) << ((b0 & 1u) << 4));
    } else if (active) {
        atomicAdd(&h[bin >> 1], 1u << ((bin & 1u) << 4));
    }
}

// Exclusive prefix over a block of NT threads; *total receives the block sum.
// lds must hold NT / 64 + 1 words.  Every thread of the block must call it.
template <int NT>
__device__ uint32_t block_excl_scan(uint32_t v, uint32_t* lds, uint32_t* total) {
    constexpr int NW = NT / kWave;
    const int w = threadIdx.x / kWave, lane = lane_id();
    const uint32_t incl = wave_incl_scan(v);
    if (lane == kWave - 1) lds[w] = incl;
    __syncthreads();
    uint32_t carry = 0, sum = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        const uint32_t x = lds[i];
        carry += i < w ? x : 0u;
        sum += x;
    }
    __syncthreads();
    *total = sum;
    return incl - v + carry;
}

// Stateless 32-bit mixer for the bracket sample's positions: the published
// "lowbias32" integer hash (xor-shift / multiply rounds with the shifts and
// multipliers found by C. Wellons' hash-prospector search, 2018).  Any good
// mixer would do; the positions only have to spread over each stratum.
__device__ __forceinline__ uint32_t mix32(uint32_t x) {
    x ^= x >> 16;
    x *= 0x7feb352dU;
    x ^= x >> 15;
    x *= 0x846ca68bU;
    x ^= x >> 16;
    return x;
}

__device__ __forceinline__ uint32_t keep_of(uint32_t n, uint32_t keep_ppm) {
    return (uint32_t)(((uint64_t)n * keep_ppm) / 1000000ull);
}

}  // namespace gd
