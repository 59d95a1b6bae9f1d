// Threshold bracket from a stratified sample (gfx950, wave64).
//
// The exact threshold of Algorithm 1 (Section 4) is found later from the
// candidates alone; this step only predicts a key range [lo, hi) that very
// likely holds the k-th largest |acc| of each threshold segment, so that the
// dense pass can set aside the few candidates (key >= lo) while it streams.
// A miss costs time, never exactness: a segment with fewer than k
// candidates falls back to treating every element as a candidate.  (The
// paper itself approximates the threshold by selecting on a 0.1% sample,
// Section 4; here the sample only bounds an exact selection.)
//
//   k_sample  : many small blocks gather sample units (16 neighbours, one
//               64-byte line per input array) and store 16-bit key prefixes;
//               they also clear the per-call histograms and counters.
//   k_bracket : one block per segment holds its sample keys in registers and
//               picks lo and hi from sample ranks around the expected rank of
//               the threshold, widened by the measured spread of per-unit
//               counts (neighbouring elements can be strongly correlated).

#include "gd_kernels.h"

namespace gd {

template <bool BASE>
__device__ __forceinline__ float acc_of(float g, float b, float r) {
    // Two separate binary32 roundings when a base is given (pull deltas).
    if (BASE) {
        const float d = g - b;
        return d + r;
    }
    return g + r;
}

__device__ __forceinline__ uint32_t key16_of(uint32_t key) {
    const uint32_t k = key >> kK16Shift;
    return k < kNoKey16 ? k : kNoKey16 - 1;  // the top NaN keys share one value
}

// Units sampled from segment [seg_a, seg_b): 16-aligned blocks of 16
// elements, at most kMaxUnits of them.
__device__ __forceinline__ void sample_units(uint32_t seg_a, uint32_t seg_b, uint32_t& n16, uint32_t& U) {
    n16 = seg_b > seg_a ? ((seg_b - 1) >> 4) - (seg_a >> 4) + 1 : 0u;
    U = n16 < (uint32_t)kMaxUnits ? n16 : (uint32_t)kMaxUnits;
}

template <bool BASE>
__global__ __launch_bounds__(kSampleThreads) void k_sample(SampleArgs a) {
    const uint32_t s = blockIdx.y;
    const int tid = threadIdx.x;
    const uint32_t seg_a = a.seg_off[s], seg_b = a.seg_off[s + 1];
    __shared__ uint32_t lds[kSampleThreads / kWave + 1];

    // Clear this segment's histograms and state for the passes that follow.
    uint32_t* h = a.hist + (size_t)s * kHistWords;
    for (uint32_t i = blockIdx.x * kSampleThreads + tid; i < (uint32_t)kHistWords; i += gridDim.x * kSampleThreads)
        h[i] = 0;
    if (blockIdx.x == 0 && tid == 0) {
        a.seg[s].clo = 0;
        a.seg[s].miss = 0;
    }
    if (s == 0 && blockIdx.x == 0) {
        for (uint32_t t = tid; t < a.T; t += kSampleThreads) a.tensor_counts[t] = 0;
        // First output slot of each segment: exclusive prefix of k_s.
        uint64_t carry = 0;
        for (uint32_t b0 = 0; b0 < a.S; b0 += kSampleThreads) {
            const uint32_t ss = b0 + tid;
            const uint32_t ks = ss < a.S ? keep_of(a.seg_off[ss + 1] - a.seg_off[ss], a.keep_ppm) : 0u;
            uint32_t total;
            const uint32_t excl = block_excl_scan<kSampleThreads>(ks, lds, &total);
            if (ss < a.S) a.out_base[ss] = carry + excl;
            carry += total;
        }
    }

    uint32_t n16, U;
    sample_units(seg_a, seg_b, n16, U);
    const uint32_t j = blockIdx.x * kSampleThreads + tid;
    if (j >= U) return;
    // stratum j of the segment's 16-element blocks, one block chosen by a fixed hash
    const uint32_t lo_j = (uint32_t)(((uint64_t)j * n16) / U);
    const uint32_t hi_j = (uint32_t)(((uint64_t)(j + 1) * n16) / U);
    uint32_t pick = 0;
    if (U != n16) pick = mix32(j * 0x9E3779B9u ^ (s + 1u) * 0x85EBCA6Bu) % (hi_j - lo_j);
    const uint32_t e0 = ((seg_a >> 4) + lo_j + pick) * kUnit;
    uint32_t k16[kUnit];
    if (e0 >= seg_a && e0 + kUnit <= seg_b) {
        const f4* g4 = reinterpret_cast<const f4*>(a.grad + e0);
        const f4* r4 = reinterpret_cast<const f4*>(a.res + e0);
        const f4* b4 = reinterpret_cast<const f4*>(BASE ? a.base + e0 : a.grad + e0);
        f4 g[4], r[4], b[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            g[q] = g4[q];
            r[q] = r4[q];
            b[q] = BASE ? b4[q] : g[q];
        }
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int c = 0; c < 4; ++c) k16[4 * q + c] = key16_of(key_of(acc_of<BASE>(g[q][c], b[q][c], r[q][c])));
    } else {
#pragma unroll
        for (int q = 0; q < kUnit; ++q) {
            const uint32_t e = e0 + q;
            k16[q] = kNoKey16;
            if (e >= seg_a && e < seg_b)
                k16[q] = key16_of(key_of(acc_of<BASE>(a.grad[e], BASE ? a.base[e] : 0.0f, a.res[e])));
        }
    }
    uint4* dst = reinterpret_cast<uint4*>(a.skeys + a.skey_base[s] + (size_t)kUnit * j);
    dst[0] = make_uint4(k16[0] | (k16[1] << 16), k16[2] | (k16[3] << 16), k16[4] | (k16[5] << 16),
                        k16[6] | (k16[7] << 16));
    dst[1] = make_uint4(k16[8] | (k16[9] << 16), k16[10] | (k16[11] << 16), k16[12] | (k16[13] << 16),
                        k16[14] | (k16[15] << 16));
}

__global__ __launch_bounds__(kBracketThreads) void k_bracket(SampleArgs a) {
    const uint32_t s = blockIdx.x;
    const int tid = threadIdx.x, w = tid >> 6;
    const uint32_t seg_a = a.seg_off[s], seg_b = a.seg_off[s + 1];
    const uint32_t n = seg_b - seg_a;
    const uint32_t k = keep_of(n, a.keep_ppm);
    __shared__ uint32_t hA[kNB0];
    __shared__ uint32_t hB[2][kSNB1];
    __shared__ uint32_t par[12];
    uint32_t n16, U;
    sample_units(seg_a, seg_b, n16, U);
    uint32_t lo, hi;
    if (k == 0) {
        lo = hi = kNoKey;
    } else if (k >= n) {
        lo = hi = 0;
    } else {
        // thread u holds the 16 keys of sample unit u
        uint32_t kv[kUnit];
        if ((uint32_t)tid < U) {
            const uint4* src = reinterpret_cast<const uint4*>(a.skeys + a.skey_base[s] + (size_t)kUnit * tid);
            const uint4 x0 = src[0], x1 = src[1];
            const uint32_t wv[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                kv[2 * i] = wv[i] & 0xFFFFu;
                kv[2 * i + 1] = wv[i] >> 16;
            }
        } else {
#pragma unroll
            for (int i = 0; i < kUnit; ++i) kv[i] = kNoKey16;
        }
        for (int i = tid; i < kNB0; i += kBracketThreads) hA[i] = 0;
        if (tid < 2 * kSNB1) (&hB[0][0])[tid] = 0;
        if (tid < 12) par[tid] = 0;
        __syncthreads();
        // Pass 1: digit-0 histogram of the nonzero sample keys; zero keys
        // (most of a sparse embedding gradient) are only counted.
        uint32_t nvalid = 0, nzero = 0;
#pragma unroll
        for (int i = 0; i < kUnit; ++i) {
            const uint32_t key = kv[i];
            const bool valid = key != kNoKey16;
            lds_hist_add(hA, valid ? key >> kS0Shift : 0u, valid && key != 0);
            nvalid += valid;
            nzero += valid && key == 0;
        }
        nvalid = wave_sum(nvalid);
        nzero = wave_sum(nzero);
        if (lane_id() == 0) {
            atomicAdd(&par[0], nvalid);
            atomicAdd(&par[1], nzero);
        }
        __syncthreads();
        const uint32_t m = par[0], mnz = par[0] - par[1];
        const bool full = m >= n;  // every element sampled: exact ranks
        const double q = (double)k * (double)m / (double)n;
        if (!full && w == 0) {
            // digit-0 bin of the estimated threshold (rank q in the sample)
            const uint32_t rq = (uint32_t)fmax(1.0, floor(q + 0.5));
            uint32_t d = 0, ab;
            if (rq > mnz || !wave_pick<kNB0>(hA, rq, d, ab)) d = 0;
            if (lane_id() == 0) par[2] = d;
        }
        __syncthreads();
        if (!full) {
            // Pass 2: spread of the per-unit counts at that bin.  Units are
            // runs of 16 neighbours, which can be strongly correlated (a
            // nonzero embedding row), so the rank uncertainty of the sample is
            // measured rather than assumed binomial.
            const uint32_t dq = par[2];
            uint32_t c = 0;
#pragma unroll
            for (int i = 0; i < kUnit; ++i) c += (kv[i] != kNoKey16 && kv[i] != 0 && (kv[i] >> kS0Shift) >= dq);
            uint32_t s1 = wave_sum(c), s2 = wave_sum(c * c);
            if (lane_id() == 0) {
                atomicAdd(&par[3], s1);
                atomicAdd(&par[4], s2);
            }
        }
        __syncthreads();
        if (tid == 0) {
            uint32_t r_hi, r_lo;
            if (full) {
                r_hi = r_lo = k;
            } else {
                const double mean = (double)par[3] / U, var = (double)par[4] / U - mean * mean;
                const double sd = sqrt(fmax(q, U * fmax(var, 0.0)));
                const double fh = floor(q - 3.0 * sd - 2.0);
                const double fl = ceil(q + 5.0 * sd + 4.0);
                r_hi = fh < 1.0 ? 0u : (uint32_t)fh;
                r_lo = fl > (double)m ? kNoKey : (uint32_t)fl;
            }
            // ranks that fall among the zero keys
            if (r_hi > mnz) r_hi = 0;
            if (r_lo != kNoKey && r_lo > mnz) r_lo = kNoKey;
            par[5] = r_hi;
            par[6] = r_lo;
        }
        __syncthreads();
        const uint32_t r_hi = par[5], r_lo = par[6];
        if (w == 0 && r_hi) {
            uint32_t d, ab;
            wave_pick<kNB0>(hA, r_hi, d, ab);
            if (lane_id() == 0) {
                par[7] = d;
                par[8] = r_hi - ab;
            }
        }
        if (w == 1 && r_lo != kNoKey) {
            uint32_t d, ab;
            wave_pick<kNB0>(hA, r_lo, d, ab);
            if (lane_id() == 0) {
                par[9] = d;
                par[10] = r_lo - ab;
            }
        }
        __syncthreads();
        const uint32_t dh = r_hi ? par[7] : kNoKey, dl = r_lo != kNoKey ? par[9] : kNoKey;
#pragma unroll
        for (int i = 0; i < kUnit; ++i) {
            const uint32_t key = kv[i];
            const bool nz = key != kNoKey16 && key != 0;
            const uint32_t d0 = key >> kS0Shift, d1 = key & (kSNB1 - 1);
            lds_hist_add(hB[0], d1, nz && d0 == dh);
            lds_hist_add(hB[1], d1, nz && d0 == dl);
        }
        __syncthreads();
        if (w == 0 && r_hi) {
            uint32_t d, ab;
            wave_pick<kSNB1>(hB[0], par[8], d, ab);
            if (lane_id() == 0) par[8] = d;
        }
        if (w == 1 && r_lo != kNoKey) {
            uint32_t d, ab;
            wave_pick<kSNB1>(hB[1], par[10], d, ab);
            if (lane_id() == 0) par[10] = d;
        }
        __syncthreads();
        hi = r_hi ? ((((dh << kS0Shift) | par[8]) + 1u) << kK16Shift) : kNoKey;
        if (r_lo != kNoKey) {
            lo = ((dl << kS0Shift) | par[10]) << kK16Shift;
            if (lo == 0) lo = 1;
        } else {
            // The rank falls among zero keys: candidates are the nonzero
            // entries, unless every element was sampled and zeros are known
            // to be needed.
            lo = (full && k > mnz) ? 0u : 1u;
        }
    }
    if (a.debug_bracket == kDebugLoTooHigh && k > 0) {
        lo = 0x7FFFFFFFu;
        hi = kNoKey;
    } else if (a.debug_bracket == kDebugHiAtLo) {
        hi = lo;
    } else if (a.debug_bracket == kDebugLoZero && k > 0) {
        lo = 0;
    }
    if (tid == 0) {
        a.seg[s].lo = lo;
        a.seg[s].hi = hi;
    }
}

hipError_t launch_sample(const SampleArgs& a, bool has_base, hipStream_t st) {
    const dim3 grid(kSampleBlocks, a.S);
    if (has_base) hipLaunchKernelGGL(k_sample<true>, grid, dim3(kSampleThreads), 0, st, a);
    else hipLaunchKernelGGL(k_sample<false>, grid, dim3(kSampleThreads), 0, st, a);
    hipLaunchKernelGGL(k_bracket, dim3(a.S), dim3(kBracketThreads), 0, st, a);
    return hipGetLastError();
}

}  // namespace gd
