// Server-side apply of sparse pushes to a parameter shard (Section 3: each
// server owns a shard of the parameters and receives the clients' pieces).
//
// For an index pushed by several clients the values are summed in client
// order starting from +0, and the parameter is updated once:
// p[i] -= lr * s[i].  No atomics, so the result is deterministic.
//
// One block per bucket of 2^15 consecutive parameter indices.  The block
// finds where the bucket starts and ends in every client's (ascending) index
// list by a 32-way search per half-wave (four rounds of loads for a list of a
// few hundred thousand entries, instead of a binary search's twenty), stages
// those entries in LDS, marking the indices pushed more than once, and then
// gives every index to the lowest client holding it, which sums all clients'
// values for it in client order and writes p once.  The parameter writes of a block stay inside its bucket.
// Quantised pushes (indices, sign bits, centre pairs; Section 5.4) are decoded
// entry by entry where their values are read.

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

hipError_t launch_apply(const ApplyArgs& a, uint32_t max_nnz, hipStream_t st) {
    if (a.C == 0 || max_nnz == 0 || a.n == 0) return hipSuccess;
    const uint32_t buckets = (uint32_t)(((uint64_t)a.n + (1u << kApplyBucketShift) - 1) >> kApplyBucketShift);
    hipLaunchKernelGGL(k_apply, dim3(buckets), dim3(kBlock), 0, st, a);
    return hipGetLastError();
}

}  // namespace gd
