// Server-side apply of sparse pushes to a parameter shard (Section 3: each
// server owns a shard of the parameters and receives the clients' pieces).
//
// For an index pushed by several clients the values are summed in client
// order starting from +0, and the parameter is updated once:
// p[i] -= lr * s[i].  No atomics, so the result is deterministic.
//
// Two forms, with the same results bit for bit.  The scattered form reads
// and writes only the pushed parameters; the streaming form reads the whole
// shard in order and writes back the 16-byte vectors that change, for pushes
// dense enough that most 128-byte lines of the shard hold an update.
// Quantised pushes (indices, sign bits, centre pairs; Section 5.4) are decoded
// entry by entry where their values are read.
//
// The scattered form: one block per bucket of 2^15 consecutive parameter
// indices.  The block finds where the bucket starts and ends in every
// client's (ascending) index list by a 32-way search per half-wave (four
// rounds of loads for a list of a few hundred thousand entries, instead of a
// binary search's twenty), stages those entries in LDS, marking the indices
// pushed more than once, and then gives every index to the lowest client
// holding it, which sums all clients' values for it in client order and
// writes p once.  The parameter writes of a block stay inside its bucket.

#include <algorithm>
#include <atomic>
#include <mutex>

#include "gd_kernels.h"

namespace gd {

constexpr int kApplyBucketShift = 15;
constexpr int kApplyLds = 2048;                              // entries of all clients staged per bucket
constexpr int kBucketWords = (1 << kApplyBucketShift) / 32;  // one bit per index of a bucket

// First position in list[lo, hi) whose value is >= x, found by the 32 lanes of
// one half-wave together (g: lane within the half, mask: the half's lanes).
__device__ uint32_t half_lower_bound(const uint32_t* list, uint32_t lo, uint32_t hi, uint32_t x, uint32_t g,
                                     uint64_t mask) {
    while (hi > lo) {
        const uint32_t len = hi - lo;
        if (len <= 32u) {
            const bool below = g < len && list[lo + (g < len ? g : 0u)] < x;
            return lo + popc64(ballot(below) & mask);
        }
        const uint32_t step = (len + 31u) / 32u;
        uint32_t q = lo + (g + 1u) * step - 1u;
        if (q >= hi) q = hi - 1u;
        // probes rise with g, so the lanes below x form a prefix of the half
        const uint32_t t = popc64(ballot(list[q] < x) & mask);
        const uint64_t nlo = (uint64_t)lo + (uint64_t)t * step, nhi = nlo + step;
        lo = nlo < hi ? (uint32_t)nlo : hi;
        hi = nhi < hi ? (uint32_t)nhi : hi;
    }
    return lo;
}

// First position in list[lo, hi) holding x, or hi.
__device__ __forceinline__ uint32_t find_u32(const uint32_t* list, uint32_t lo, uint32_t hi, uint32_t x) {
    uint32_t a = lo, b = hi;
    while (a < b) {
        const uint32_t mid = a + ((b - a) >> 1);
        if (list[mid] < x) a = mid + 1;
        else b = mid;
    }
    return a < hi && list[a] == x ? a : hi;
}

// Value of entry pos (index i) of push c: sent as is, or a quantised push's
// centre, chosen by the entry's sign bit from the pair of its tensor or column.
__device__ __forceinline__ float push_val(const ApplyArgs& a, uint32_t c, uint32_t pos, uint32_t i) {
    if (a.qkind == 0) return a.val[c][pos];
    uint32_t lo = 0, hi = a.T;  // tensor holding i: the last t with tensor_off[t] <= i
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (a.tensor_off[mid] <= i) lo = mid;
        else hi = mid;
    }
    const uint32_t g = a.qkind == kQuantColumnMean ? a.colbase[lo] + (i - a.tensor_off[lo]) % a.columns[lo] : lo;
    const uint32_t neg = (a.bits[c][pos >> 5] >> (pos & 31)) & 1u;
    return a.means[c][2 * g + neg];
}

__global__ __launch_bounds__(kBlock) void k_apply(ApplyArgs a) {
    __shared__ uint32_t rng[kMaxPushes][2];  // bucket's [begin, end) in each client's list
    __shared__ uint32_t base[kMaxPushes + 1];  // first staged entry of each client
    __shared__ uint32_t sidx[kApplyLds];
    __shared__ float sval[kApplyLds];
    __shared__ uint32_t seen[2][kBucketWords];  // [0]: index pushed at least once, [1]: more than once
    const int tid = threadIdx.x, w = (int)wave_index(), lane = lane_id();
    const uint32_t b = blockIdx.x;
    const uint32_t i_lo = b << kApplyBucketShift;
    const uint64_t i_hi64 = ((uint64_t)b + 1) << kApplyBucketShift;
    const uint32_t i_hi = i_hi64 < a.n ? (uint32_t)i_hi64 : a.n;
    // 1. the bucket's range in every list: one client per wave, the two bounds
    //    by the two half-waves
    const uint32_t half = (uint32_t)lane >> 5, g = (uint32_t)lane & 31u;
    const uint64_t mask = half ? 0xFFFFFFFF00000000ull : 0x00000000FFFFFFFFull;
    for (uint32_t c = w; c < a.C; c += kWavesPerBlock) {
        const uint32_t pos = half_lower_bound(a.idx[c], 0, a.nnz[c], half ? i_hi : i_lo, g, mask);
        if (g == 0) rng[c][half] = pos;
    }
    __syncthreads();
    if (tid == 0) {
        uint32_t acc = 0;
        for (uint32_t c = 0; c < a.C; ++c) {
            base[c] = acc;
            acc += rng[c][1] - rng[c][0];
        }
        base[a.C] = acc;
    }
    __syncthreads();
    const uint32_t total = base[a.C];
    if (total == 0) return;
    const bool staged = total <= (uint32_t)kApplyLds;
    // 2. stage the bucket's entries (index, value) of every client, and mark
    //    the indices pushed more than once
    if (staged) {
        for (uint32_t q = tid; q < 2u * kBucketWords; q += kBlock) (&seen[0][0])[q] = 0;
        __syncthreads();
        for (uint32_t c = 0; c < a.C; ++c) {
            const uint32_t r0 = rng[c][0], cnt = rng[c][1] - r0, o = base[c];
            for (uint32_t q = tid; q < cnt; q += kBlock) {
                const uint32_t ii = a.idx[c][r0 + q];
                const uint32_t off = ii - i_lo, bit = 1u << (off & 31);
                // an index outside the bucket (a list out of order) is skipped
                sidx[o + q] = off < i_hi - i_lo ? ii : kNoKey;
                sval[o + q] = push_val(a, c, r0 + q, ii);
                if (off < i_hi - i_lo && (atomicOr(&seen[0][off >> 5], bit) & bit)) atomicOr(&seen[1][off >> 5], bit);
            }
        }
        __syncthreads();
    }
    // 3. each entry: skip it if a lower client holds the same index, else sum
    //    every client's value for it in client order and update p once (an
    //    index pushed once needs no search).  When staged, a thread settles all
    //    its entries first and then reads all its parameters at once, so their
    //    latencies overlap instead of adding up.
    if (staged) {
        constexpr int kPer = kApplyLds / kBlock;
        uint32_t pi[kPer];
        float pstep[kPer];
        bool pv[kPer];
#pragma unroll
        for (int t = 0; t < kPer; ++t) {
            const uint32_t e = tid + t * kBlock;
            pv[t] = false;
            pi[t] = i_lo;  // a valid parameter index for the unconditional load below
            pstep[t] = 0.0f;
            if (e < total && sidx[e] != kNoKey) {
                uint32_t c = 0;
                while (base[c + 1] <= e) ++c;  // client of staged entry e
                const uint32_t i = sidx[e];
                const uint32_t off = i - i_lo;
                const bool once = (seen[1][off >> 5] & (1u << (off & 31))) == 0;
                bool owner = true;
                for (uint32_t cc = 0; cc < c && owner && !once; ++cc)
                    owner = find_u32(sidx, base[cc], base[cc + 1], i) == base[cc + 1];
                if (owner) {
                    float sum = 0.0f + sval[e];
                    for (uint32_t cc = c + 1; cc < a.C && !once; ++cc) {
                        const uint32_t hit = find_u32(sidx, base[cc], base[cc + 1], i);
                        if (hit != base[cc + 1]) sum = sum + sval[hit];
                    }
                    pv[t] = true;
                    pi[t] = i;
                    pstep[t] = a.lr * sum;
                }
            }
        }
        float pold[kPer];
#pragma unroll
        for (int t = 0; t < kPer; ++t) pold[t] = a.p[pi[t]];
#pragma unroll
        for (int t = 0; t < kPer; ++t)
            if (pv[t]) a.p[pi[t]] = pold[t] - pstep[t];
        return;
    }
    for (uint32_t e = tid; e < total; e += kBlock) {
        uint32_t c = 0;
        while (base[c + 1] <= e) ++c;  // client of staged entry e
        const uint32_t q = e - base[c];
        const uint32_t i = staged ? sidx[e] : a.idx[c][rng[c][0] + q];
        if (i - i_lo >= i_hi - i_lo) continue;  // outside the bucket: a list out of order
        bool owner = true;
        for (uint32_t cc = 0; cc < c && owner; ++cc) {
            const uint32_t hit = staged ? find_u32(sidx, base[cc], base[cc + 1], i)
                                        : find_u32(a.idx[cc], rng[cc][0], rng[cc][1], i);
            owner = staged ? hit == base[cc + 1] : hit == rng[cc][1];
        }
        if (!owner) continue;
        float s = 0.0f;
        for (uint32_t cc = 0; cc < a.C; ++cc) {
            if (cc < c) continue;
            if (cc == c) {
                s = s + (staged ? sval[e] : push_val(a, c, rng[c][0] + q, i));
                continue;
            }
            if (staged) {
                const uint32_t hit = find_u32(sidx, base[cc], base[cc + 1], i);
                if (hit != base[cc + 1]) s = s + sval[hit];
            } else {
                const uint32_t hit = find_u32(a.idx[cc], rng[cc][0], rng[cc][1], i);
                if (hit != rng[cc][1]) s = s + push_val(a, cc, hit, i);
            }
        }
        const float step = a.lr * s;
        a.p[i] = a.p[i] - step;
    }
}

// The streaming form, for pushes dense enough that most 128-byte lines of
// the shard hold an update (the scattered form above then fetches nearly every
// line anyway, one scattered word at a time).  One block per chunk of
// kStreamLen consecutive parameters reads the whole chunk in order with
// 16-byte loads and writes back only the 16-byte vectors an entry touches.
//
// How fast a chunk streams is set by the bytes a block keeps in flight over
// its lifetime, so the roles are split between waves.  The loading waves
// issue the chunk's loads first thing and hold its 64 KB in registers; the
// list waves read the chunk's range in every client's list from a bounds
// table (k_apply_bounds, one pass over the lists before this kernel) and
// stage the chunk's entries in LDS, each wave the clients it handles, marking
// the parameters pushed at least once and more than once.  The loading waves
// then copy the vectors that an entry touches (about one in seven at a few
// percent of indices pushed) into a compact LDS array and leave, so that the
// per-parameter work is done for the touched vectors only, by the list
// waves: a parameter pushed once takes p - lr * (0 + value); the sum of one
// pushed by several clients is formed in client turns between barriers,
// started from +0 by the first client's entry, and the parameter then takes
// p - lr * sum.  The list waves store the compact vectors back.  Each
// parameter is written once, by one thread, with the scattered form's
// arithmetic, so the two forms agree bit for bit.
constexpr int kStreamShift = 14;
constexpr uint32_t kStreamLen = 1u << kStreamShift;                            // parameters per block
constexpr int kStreamLoadWaves = 4, kStreamListWaves = 4;
constexpr int kStreamThreads = (kStreamLoadWaves + kStreamListWaves) * kWave;
constexpr int kStreamLoadThreads = kStreamLoadWaves * kWave;
constexpr uint32_t kListThreads = kStreamThreads - kStreamLoadThreads;
constexpr int kStreamLoadShift = 8;                                            // log2 kStreamLoadThreads
constexpr int kStreamVecs = (int)kStreamLen / 4 / kStreamLoadThreads;         // 16-byte vectors per loading thread
constexpr int kStreamCap = 1024;                                               // entries of all clients staged per chunk
constexpr int kStreamWords = (int)kStreamLen / 32;                             // bitmap words per chunk
constexpr uint16_t kStreamNoOff = 0xFFFFu;                                     // a staged entry outside the chunk
constexpr int kStreamBatch = 8;                                                // entries per lane loaded at once when staging
constexpr int kStreamPer = kStreamCap / (int)kListThreads;                     // staged entries per list thread

static_assert(kStreamLoadThreads == 1 << kStreamLoadShift, "loading threads");
static_assert(kStreamVecs == 16, "a loading thread's parameters are two bitmap words");
static_assert(kStreamVecs * 4 * kStreamLoadThreads == (int)kStreamLen, "chunk split over the loading threads");
static_assert(kStreamCap <= 0xFFFF && kStreamLen / 4 <= 0xFFFF, "staged positions and vectors fit 16 bits");

struct StreamLds {
    uint32_t rng[kMaxPushes][2];       // the chunk's [begin, end) in each client's list
    uint32_t base[kMaxPushes + 1];     // first staged entry of each client
    uint32_t total;                    // staged entries of all clients
    uint32_t ncomp;                    // touched vectors
    uint32_t seen[3 * kStreamWords];   // pushed at least once, more than once, sum started
    uint16_t sofs[kStreamCap];         // staged entry's offset in the chunk
    float sval[kStreamCap];            // staged entry's value (the running sum, in a first entry)
    uint16_t vecpos[kStreamLen / 4];   // touched vector -> its place in comp
    uint16_t compvec[kStreamCap];      // place in comp -> vector
    uint16_t cfirst[4 * kStreamCap];   // per parameter of comp: the entry holding the sum of its clients
    f4 comp[kStreamCap];               // the touched vectors
};

// The bitmaps are laid out by loading thread: the 64 parameters thread t
// holds (vectors t + kStreamLoadThreads r) are words 2t and 2t + 1, with
// parameter 4v + q at bit 4 (r mod 8) + q of word 2t + r / 8.
__device__ __forceinline__ uint32_t stream_word(uint32_t off) {
    const uint32_t v = off >> 2;
    return 2u * (v & (kStreamLoadThreads - 1)) + (v >> (kStreamLoadShift + 3));
}
__device__ __forceinline__ uint32_t stream_bit(uint32_t off) {
    return 1u << ((((off >> 2) >> kStreamLoadShift) & 7u) * 4u + (off & 3u));
}

// The loading waves' side of a chunk.  Its barriers pair one for one with
// the list waves' first four in k_apply_stream, and both sides leave at the
// same points (no entry in the chunk; more entries than LDS holds, which the
// list waves then apply alone); after the fourth the loading waves are done.
__device__ __forceinline__ void stream_params(const ApplyArgs& a, StreamLds& L, uint32_t i_lo, uint32_t len,
                                              bool whole, int tid) {
    f4 pv[kStreamVecs];
    // vector v = tid + kStreamLoadThreads r holds parameters i_lo + 4v .. + 3
    if (whole) {
#pragma unroll
        for (int r = 0; r < kStreamVecs; ++r)
            pv[r] = *reinterpret_cast<const f4*>(a.p + i_lo + 4u * ((uint32_t)tid + (uint32_t)r * kStreamLoadThreads));
    } else {
#pragma unroll
        for (int r = 0; r < kStreamVecs; ++r) {
            const uint32_t o = 4u * ((uint32_t)tid + (uint32_t)r * kStreamLoadThreads);
            pv[r] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (o + q < len) pv[r][q] = a.p[i_lo + o + q];
        }
    }
    for (int q = tid; q < 3 * kStreamWords; q += kStreamLoadThreads) L.seen[q] = 0;
    if (tid == 0) L.ncomp = 0;
    __syncthreads();  // 1: ranges read, bitmaps cleared
    __syncthreads();  // 2: staging offsets
    // (from LDS: a kernel argument read here would be waited for together
    // with the LDS clearing above, and under a full memory queue it can miss)
    const uint32_t total = L.total;
    if (total == 0 || total > (uint32_t)kStreamCap) return;  // nothing here, or the list waves apply it entry by entry
    __syncthreads();  // 3: entries staged
    // This thread's touched vectors (a nonzero nibble of its 64 bits) go to
    // consecutive places of comp, after those of the lanes below and of the
    // waves that reserved theirs earlier.
    const uint2 m = *reinterpret_cast<const uint2*>(L.seen + 2 * tid);
    const auto nonzero_nibbles = [](uint32_t x) {
        x |= x >> 1;
        x |= x >> 2;
        return (uint32_t)__popc(x & 0x11111111u);
    };
    const uint32_t cnt = nonzero_nibbles(m.x) + nonzero_nibbles(m.y);
    const uint32_t incl = wave_incl_scan(cnt);
    uint32_t wb = 0;
    if (lane_id() == kWave - 1) wb = atomicAdd(&L.ncomp, incl);
    uint32_t pos = lane_value(wb, kWave - 1) + incl - cnt;
#pragma unroll
    for (int r = 0; r < kStreamVecs; ++r) {
        const uint32_t nib = ((r < 8 ? m.x : m.y) >> ((r & 7) * 4)) & 0xFu;
        if (nib == 0) continue;
        const uint32_t v = (uint32_t)tid + (uint32_t)r * kStreamLoadThreads;
        L.comp[pos] = pv[r];
        L.vecpos[v] = (uint16_t)pos;
        L.compvec[pos] = (uint16_t)v;
        ++pos;
    }
    __syncthreads();  // 4: touched vectors in comp
}

// The bounds table of the streaming form: row c holds, for every chunk
// boundary B_b (b * kStreamLen for b < chunks, n for b = chunks), the first
// position in client c's list whose index is at least B_b.  With f(x) the
// number of boundaries at or below x, entry e starts the boundaries in
// [f(x_{e-1}), f(x_e)), the list's head [0, f(x_0)) starts at 0 and its tail
// [f(x_last), chunks] at the list's length: one pass over the entries, no
// search.  One row of blocks per client (blockIdx.y); the first chunks + 1
// threads of a row fill the head and tail, the others one entry each.  (A
// list out of order leaves some boundaries unwritten; readers clamp.)
__global__ __launch_bounds__(kBlock) void k_apply_bounds(ApplyArgs a, uint32_t chunks) {
    const uint32_t c = blockIdx.y;
    const uint32_t m = a.nnz[c];
    const uint32_t* list = a.idx[c];
    uint32_t* row = const_cast<uint32_t*>(a.tab) + (size_t)c * a.tstride;
    const uint64_t item = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
    const auto f = [&](uint32_t x) { return x < a.n ? (x >> kStreamShift) + 1u : chunks + 1u; };
    if (item <= chunks) {
        const uint32_t b = (uint32_t)item;
        if (m == 0 || b < f(list[0])) row[b] = 0;
        else if (b >= f(list[m - 1])) row[b] = m;
        return;
    }
    const uint64_t e = item - chunks;  // 1 .. m - 1
    if (e >= m) return;
    const uint32_t hi = f(list[e]);
    for (uint32_t b = f(list[e - 1]); b < hi; ++b) row[b] = (uint32_t)e;
}

__global__ __launch_bounds__(kStreamThreads) __attribute__((amdgpu_waves_per_eu(6))) void k_apply_stream(ApplyArgs a) {
    __shared__ StreamLds L;
    uint32_t* const more = L.seen + kStreamWords;
    uint32_t* const started = L.seen + 2 * kStreamWords;
    const int tid = threadIdx.x, lane = lane_id();
    const uint32_t w = wave_index();
    const uint32_t i_lo = blockIdx.x << kStreamShift;
    const uint64_t e64 = (uint64_t)i_lo + kStreamLen;
    const bool whole = e64 <= a.n;  // the same in every thread
    const uint32_t i_hi = whole ? (uint32_t)e64 : a.n;
    const uint32_t len = i_hi - i_lo;
    // Waves 0 to 3 handle the lists and the others load the chunk: the first
    // waves of a block issue first, so the bounds read is not queued behind
    // the chunk's loads.
    if (w >= (uint32_t)kStreamListWaves) {
        stream_params(a, L, i_lo, len, whole, tid - (int)kListThreads);
        return;
    }
    // The list waves.  The chunk's range in every list, from the bounds table
    // (clamped to the list, so that any table content stays inside it).
    const uint32_t lw = w, lt = (uint32_t)tid;
    for (uint32_t c = lw; c < a.C; c += kStreamListWaves) {
        if (lane < 2) {
            const uint32_t v = a.tab[(size_t)c * a.tstride + blockIdx.x + (uint32_t)lane];
            L.rng[c][lane] = v < a.nnz[c] ? v : a.nnz[c];
        }
    }
    __syncthreads();  // 1
    if (lw == 0) {
        const uint32_t c = (uint32_t)lane;
        const uint32_t r0 = c < a.C ? L.rng[c][0] : 0u, r1 = c < a.C ? L.rng[c][1] : 0u;
        const uint32_t cnt = r1 > r0 ? r1 - r0 : 0u;
        const uint32_t incl = wave_incl_scan(cnt);
        if (c < a.C) L.base[c] = incl - cnt;
        if (c == kWave - 1) L.base[a.C] = L.total = incl;
    }
    __syncthreads();  // 2
    const uint32_t total = L.total;
    if (total == 0) return;  // no entry in this chunk: nothing to write
    if (total <= (uint32_t)kStreamCap) {
        // each list wave stages the clients it handles, a batch of up to
        // kStreamBatch entries per lane loaded at once
        for (uint32_t c = lw; c < a.C; c += kStreamListWaves) {
            const uint32_t r0 = L.rng[c][0], o = L.base[c], cnt = L.base[c + 1] - o;
            for (uint32_t q0 = 0; q0 < cnt; q0 += kStreamBatch * kWave) {
                uint32_t ii[kStreamBatch];
                float vv[kStreamBatch];
#pragma unroll
                for (int j = 0; j < kStreamBatch; ++j) {
                    const uint32_t q = q0 + (uint32_t)lane + (uint32_t)j * kWave;
                    ii[j] = q < cnt ? a.idx[c][r0 + q] : i_lo;
                    if (a.qkind == 0) vv[j] = q < cnt ? a.val[c][r0 + q] : 0.0f;
                }
#pragma unroll
                for (int j = 0; j < kStreamBatch; ++j) {
                    const uint32_t q = q0 + (uint32_t)lane + (uint32_t)j * kWave;
                    if (q >= cnt) continue;
                    const uint32_t off = ii[j] - i_lo;
                    const bool in = off < len;  // an index outside the chunk (a list out of order) is skipped
                    L.sofs[o + q] = in ? (uint16_t)off : kStreamNoOff;
                    L.sval[o + q] = a.qkind == 0 ? vv[j] : push_val(a, c, r0 + q, ii[j]);
                    if (in) {
                        const uint32_t wd = stream_word(off), bit = stream_bit(off);
                        if (atomicOr(&L.seen[wd], bit) & bit) atomicOr(&more[wd], bit);
                    }
                }
            }
        }
        __syncthreads();  // 3
        // This thread's entries (entry e = lt + kListThreads k), read at once.
        uint32_t eo[kStreamPer], mw[kStreamPer];
        float ev[kStreamPer];
#pragma unroll
        for (int k = 0; k < kStreamPer; ++k) {
            const uint32_t e = lt + (uint32_t)k * kListThreads;
            eo[k] = e < total ? L.sofs[e] : kStreamNoOff;
            ev[k] = e < total ? L.sval[e] : 0.0f;
        }
#pragma unroll
        for (int k = 0; k < kStreamPer; ++k)
            mw[k] = eo[k] != kStreamNoOff ? more[stream_word(eo[k])] & stream_bit(eo[k]) : 0u;
        __syncthreads();  // 4: the loading waves have copied the touched vectors and left
        // A parameter pushed once: p - lr * (0 + value), in comp.
#pragma unroll
        for (int k = 0; k < kStreamPer; ++k) {
            if (eo[k] == kStreamNoOff || mw[k] != 0) continue;
            const uint32_t off = eo[k];
            const uint32_t pos = min((uint32_t)L.vecpos[off >> 2], (uint32_t)kStreamCap - 1u);
            const float sum = 0.0f + ev[k];
            const float step = a.lr * sum;
            L.comp[pos][off & 3u] = L.comp[pos][off & 3u] - step;
        }
        // Pushed by several clients: the sum in client turns.  The first
        // client's entry starts it from +0 in its own value and is named in
        // cfirst; each later client's entry adds its value there.
        uint32_t first = 0;  // bit k: this thread's entry k started a sum
        for (uint32_t t = 0; t < a.C; ++t) {
            if (t > 0) __syncthreads();  // the previous client's turn done
            const uint32_t b0 = L.base[t], b1 = L.base[t + 1];
#pragma unroll
            for (int k = 0; k < kStreamPer; ++k) {
                const uint32_t e = lt + (uint32_t)k * kListThreads, off = eo[k];
                if (mw[k] == 0 || e < b0 || e >= b1) continue;
                const uint32_t wd = stream_word(off), bit = stream_bit(off);
                const uint32_t cp = 4u * min((uint32_t)L.vecpos[off >> 2], (uint32_t)kStreamCap - 1u) + (off & 3u);
                if (!(atomicOr(&started[wd], bit) & bit)) {
                    L.sval[e] = 0.0f + ev[k];
                    L.cfirst[cp] = (uint16_t)e;
                    first |= 1u << k;
                } else {
                    // (a first entry not yet named can only come from a list
                    // holding an index twice; it is kept inside the staged entries)
                    const uint32_t o = min((uint32_t)L.cfirst[cp], (uint32_t)kStreamCap - 1u);
                    L.sval[o] = L.sval[o] + ev[k];
                }
            }
        }
        __syncthreads();  // every sum complete
#pragma unroll
        for (int k = 0; k < kStreamPer; ++k) {
            if (!((first >> k) & 1u)) continue;
            const uint32_t e = lt + (uint32_t)k * kListThreads, off = eo[k];
            const uint32_t pos = min((uint32_t)L.vecpos[off >> 2], (uint32_t)kStreamCap - 1u);
            const float step = a.lr * L.sval[e];
            L.comp[pos][off & 3u] = L.comp[pos][off & 3u] - step;
        }
        __syncthreads();  // comp final
        const uint32_t ncomp = min(L.ncomp, (uint32_t)kStreamCap);
        for (uint32_t pos = lt; pos < ncomp; pos += kListThreads) {
            const uint32_t o = 4u * (uint32_t)L.compvec[pos];
            const f4 v = L.comp[pos];
            if (whole) {
                *reinterpret_cast<f4*>(a.p + i_lo + o) = v;
            } else {
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (o + q < len) a.p[i_lo + o + q] = v[q];
            }
        }
        return;
    }
    // More entries than LDS holds: entry by entry from the lists, as the
    // scattered form's unstaged path (the loading waves have left).
    for (uint32_t e = lt; e < total; e += kListThreads) {
        uint32_t c = 0;
        while (L.base[c + 1] <= e) ++c;  // client of entry e
        const uint32_t q = e - L.base[c];
        const uint32_t i = a.idx[c][L.rng[c][0] + q];
        if (i - i_lo >= len) continue;  // outside the chunk: a list out of order
        bool owner = true;
        for (uint32_t cc = 0; cc < c && owner; ++cc) {
            const uint32_t end = L.rng[cc][0] + (L.base[cc + 1] - L.base[cc]);
            owner = find_u32(a.idx[cc], L.rng[cc][0], end, i) == end;
        }
        if (!owner) continue;
        float s = 0.0f + push_val(a, c, L.rng[c][0] + q, i);
        for (uint32_t cc = c + 1; cc < a.C; ++cc) {
            const uint32_t end = L.rng[cc][0] + (L.base[cc + 1] - L.base[cc]);
            const uint32_t hit = find_u32(a.idx[cc], L.rng[cc][0], end, i);
            if (hit != end) s = s + push_val(a, cc, hit, i);
        }
        const float step = a.lr * s;
        a.p[i] = a.p[i] - step;
    }
}

// Form of later applies (a test hook): 0 chosen per call, 1 scattered, 2
// streaming wherever the parameters are 16-byte aligned.
static std::atomic<int> g_apply_form{0};

// The streaming form's bounds table is allocated in stream order from a
// memory pool the library keeps per device (created on first use, keeping
// what it has reserved, so that later calls allocate without the driver).
constexpr int kMaxDevices = 64;
static std::mutex g_pool_mu;
static hipMemPool_t g_pool[kMaxDevices] = {};

static hipMemPool_t apply_pool(int dev) {
    std::lock_guard<std::mutex> lk(g_pool_mu);
    if (dev < 0 || dev >= kMaxDevices) return nullptr;
    if (!g_pool[dev]) {
        hipMemPoolProps props{};
        props.allocType = hipMemAllocationTypePinned;
        props.location.type = hipMemLocationTypeDevice;
        props.location.id = dev;
        hipMemPool_t p = nullptr;
        if (hipMemPoolCreate(&p, &props) != hipSuccess) return nullptr;
        uint64_t keep = ~0ull;
        (void)hipMemPoolSetAttribute(p, hipMemPoolAttrReleaseThreshold, &keep);
        g_pool[dev] = p;
    }
    return g_pool[dev];
}

void set_apply_form(int form) { g_apply_form.store(form); }

hipError_t launch_apply(const ApplyArgs& a, uint32_t max_nnz, hipStream_t st) {
    if (a.C == 0 || max_nnz == 0 || a.n == 0) return hipSuccess;
    uint64_t total = 0;
    for (uint32_t c = 0; c < a.C; ++c) total += a.nnz[c];
    // Streaming reads every line of the shard: it pays once the entries touch
    // most lines (one entry per 64 parameters touches about 40% of them), and
    // while a chunk's entries usually fit its LDS (at most three quarters of
    // kStreamCap on average; a fuller chunk is applied entry by entry).  Each
    // list wave stages its clients one after another, so many clients stay
    // with the scattered form.
    const int form = g_apply_form.load();
    const bool aligned = (reinterpret_cast<uintptr_t>(a.p) & 15u) == 0;
    const bool dense = total * 64u >= a.n && total * kStreamLen <= (uint64_t)a.n * (kStreamCap * 3 / 4);
    const bool stream = aligned && form != 1 && (form == 2 || (dense && a.C <= 2u * kStreamListWaves));
    if (stream) {
        const uint32_t chunks = (uint32_t)(((uint64_t)a.n + kStreamLen - 1) >> kStreamShift);
        int dev = -1;
        hipMemPool_t pool = hipGetDevice(&dev) == hipSuccess ? apply_pool(dev) : nullptr;
        void* tab = nullptr;
        const size_t bytes = (size_t)a.C * (chunks + 1u) * sizeof(uint32_t);
        if (pool && hipMallocFromPoolAsync(&tab, bytes, pool, st) == hipSuccess) {
            ApplyArgs b = a;
            b.tab = static_cast<const uint32_t*>(tab);
            b.tstride = chunks + 1u;
            uint64_t items = 0;  // head and tail, then the entries after the first
            for (uint32_t c = 0; c < a.C; ++c) items = std::max<uint64_t>(items, chunks + 1u + (a.nnz[c] ? a.nnz[c] - 1u : 0u));
            hipLaunchKernelGGL(k_apply_bounds, dim3((uint32_t)((items + kBlock - 1) / kBlock), a.C), dim3(kBlock), 0, st, b,
                               chunks);
            hipLaunchKernelGGL(k_apply_stream, dim3(chunks), dim3(kStreamThreads), 0, st, b);
            const hipError_t launched = hipGetLastError();
            const hipError_t freed = hipFreeAsync(tab, st);
            return launched != hipSuccess ? launched : freed;
        }
        (void)hipGetLastError();  // no table: the scattered form below
    }
    const uint32_t buckets = (uint32_t)(((uint64_t)a.n + (1u << kApplyBucketShift) - 1) >> kApplyBucketShift);
    hipLaunchKernelGGL(k_apply, dim3(buckets), dim3(kBlock), 0, st, a);
    return hipGetLastError();
}

}  // namespace gd
