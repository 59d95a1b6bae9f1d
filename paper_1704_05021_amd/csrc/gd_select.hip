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
//   k_sample  : many small blocks gather sample units and store 16-bit key
//               prefixes, with the digit histogram of each segment's sample
//               (nonzero keys) and its valid and zero counts; they also clear
//               the per-call histograms and counters.  A unit is 16 elements
//               of one stratum: 16 neighbours when the whole segment is
//               sampled, else four aligned groups of 4 neighbours spread over
//               the stratum (one 16-byte load per group and input array).
//               Neighbours are strongly correlated in sparse embedding
//               gradients (a nonzero row), so spread groups carry far more
//               information per sample than one run of 16.
//   k_bracket : one block per segment holds its sample keys in registers
//               and, in one pass over them, estimates the threshold's 16-bit
//               key prefix P from the sample rank k * m / n and measures the
//               spread of the per-unit counts of keys in or above P's
//               coarse digit (neighbouring elements can be strongly
//               correlated, so the spread is not assumed binomial: its
//               dispersion index scales the binomial standard deviation).
//               hi is just above P: the dense pass zeroes the residual of
//               keys >= hi, and every key between hi and the exact threshold
//               costs one fix-up write later, so hi is a point estimate.  lo
//               lies 5 standard deviations (plus a constant) of that count
//               below the estimate, so that fewer than k candidates is rare.

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

// Dispersion index (variance over mean of the per-unit counts) below which a
// segment's sample counts as independent draws.
constexpr double kRunsMaxDispersion = 1.5;

__device__ __forceinline__ uint32_t key16_of(uint32_t key) {
    const uint32_t k = key >> kK16Shift;
    return k < kNoKey16 ? k : kNoKey16 - 1;  // the top NaN keys share one value
}

// Units sampled from segment [seg_a, seg_b): n16 is the number of
// 16-aligned blocks of 16 elements the segment touches.
__device__ __forceinline__ void sample_units(uint32_t seg_a, uint32_t seg_b, uint32_t& n16, uint32_t& U) {
    n16 = seg_b > seg_a ? ((seg_b - 1) >> 4) - (seg_a >> 4) + 1 : 0u;
    U = sample_unit_count(n16);
}

template <bool BASE>
__global__ __launch_bounds__(kSampleThreads) void k_sample(SampleArgs a) {
    // a 1-D grid of kSampleBlocks blocks per segment (no limit on segments)
    const uint32_t s = blockIdx.x / kSampleBlocks, bx = blockIdx.x % kSampleBlocks;
    const int tid = threadIdx.x;
    const uint32_t seg_a = a.seg_off[s], seg_b = a.seg_off[s + 1];
    // The previous call on this segment found its units' counts no more spread
    // than independent draws: neighbours carry independent information, so one
    // run of 16 (two lines) serves as well as four spread groups (eight lines).
    // (Loaded with the segment bounds, not after the clearing below.)
    const bool runs = load_early(&a.seg[s].runs) != 0;
    __shared__ uint32_t lds[kSampleThreads / kWave + 1];

    // Clear this segment's histograms and state for the passes that follow.
    uint32_t* h = a.hist + (size_t)s * kHistWords;
    for (uint32_t i = bx * kSampleThreads + tid; i < (uint32_t)kHistWords; i += kSampleBlocks * kSampleThreads)
        h[i] = 0;
    if (bx == 0 && tid == 0) {
        a.seg[s].clo = 0;
        a.seg[s].miss = 0;
    }
    if (s == 0 && bx == 0) {
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
    const uint32_t j = bx * kSampleThreads + tid;
    if (bx * kSampleThreads >= U) return;  // whole block idle (block-uniform)
    __shared__ uint32_t hs[kNB0];
    __shared__ uint32_t cnt[2];
    for (int i = tid; i < kNB0; i += kSampleThreads) hs[i] = 0;
    if (tid < 2) cnt[tid] = 0;
    __syncthreads();
    uint32_t k16[kUnit];
#pragma unroll
    for (int q = 0; q < kUnit; ++q) k16[q] = kNoKey16;
    const bool nores = a.res == nullptr;  // a pull from the last pulled copy has no residual
    if (j < U) {
        // stratum j: 16-element blocks [lo_j, hi_j) of the segment's aligned grid
        const uint32_t lo_j = (uint32_t)(((uint64_t)j * n16) / U);
        const uint32_t hi_j = (uint32_t)(((uint64_t)(j + 1) * n16) / U);
        const uint32_t s0 = ((seg_a >> 4) + lo_j) * kUnit;
        if (U == n16) {
            // every block sampled: its 16 neighbours
            if (s0 >= seg_a && s0 < seg_b && seg_b - s0 >= (uint32_t)kUnit) {
                const f4* g4 = reinterpret_cast<const f4*>(a.grad + s0);
                const f4* r4 = reinterpret_cast<const f4*>(nores ? a.grad + s0 : a.res + s0);
                const f4* b4 = reinterpret_cast<const f4*>(BASE ? a.base + s0 : a.grad + s0);
                f4 g[4], r[4], b[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    g[q] = g4[q];
                    r[q] = nores ? f4{0.f, 0.f, 0.f, 0.f} : r4[q];
                    b[q] = BASE ? b4[q] : g[q];
                }
#pragma unroll
                for (int q = 0; q < 4; ++q)
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        k16[4 * q + c] = key16_of(key_of(acc_of<BASE>(g[q][c], b[q][c], r[q][c])));
            } else {
#pragma unroll
                for (int q = 0; q < kUnit; ++q) {
                    const uint32_t e = s0 + q;
                    if (e >= seg_a && e < seg_b)
                        k16[q] = key16_of(key_of(acc_of<BASE>(a.grad[e], BASE ? a.base[e] : 0.0f, nores ? 0.0f : a.res[e])));
                }
            }
        } else if (runs) {
            // one aligned run of 16 neighbours (one 64-byte line per array) at a
            // fixed hash position in the stratum
            const uint32_t h = mix32(j * 0x9E3779B9u ^ (s + 1u) * 0x85EBCA6Bu);
            const uint32_t r0 = ((seg_a >> 4) + lo_j + h % (hi_j - lo_j)) * kUnit;
            if (r0 >= seg_a && r0 < seg_b && seg_b - r0 >= (uint32_t)kUnit) {
                const f4* g4 = reinterpret_cast<const f4*>(a.grad + r0);
                const f4* r4 = reinterpret_cast<const f4*>(nores ? a.grad + r0 : a.res + r0);
                const f4* b4 = reinterpret_cast<const f4*>(BASE ? a.base + r0 : a.grad + r0);
                f4 g[4], r[4], b[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    g[q] = g4[q];
                    r[q] = nores ? f4{0.f, 0.f, 0.f, 0.f} : r4[q];
                    b[q] = BASE ? b4[q] : g[q];
                }
#pragma unroll
                for (int q = 0; q < 4; ++q)
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        k16[4 * q + c] = key16_of(key_of(acc_of<BASE>(g[q][c], b[q][c], r[q][c])));
            } else {
#pragma unroll
                for (int q = 0; q < kUnit; ++q) {
                    const uint32_t e = r0 + q;
                    if (e >= seg_a && e < seg_b)
                        k16[q] = key16_of(key_of(acc_of<BASE>(a.grad[e], BASE ? a.base[e] : 0.0f, nores ? 0.0f : a.res[e])));
                }
            }
        } else {
            // one aligned group of 4 from each quarter of the stratum, by a fixed hash
            const uint32_t len = (hi_j - lo_j) * kUnit, sub = len / 4;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t h = mix32((j * 4u + q) * 0x9E3779B9u ^ (s + 1u) * 0x85EBCA6Bu);
                const uint32_t e = s0 + q * sub + (h % (sub / 4)) * 4;
                if (e >= seg_a && e < seg_b && seg_b - e >= 4u) {
                    const f4 g = *reinterpret_cast<const f4*>(a.grad + e);
                    const f4 r = nores ? f4{0.f, 0.f, 0.f, 0.f} : *reinterpret_cast<const f4*>(a.res + e);
                    const f4 b = BASE ? *reinterpret_cast<const f4*>(a.base + e) : g;
#pragma unroll
                    for (int c = 0; c < 4; ++c) k16[4 * q + c] = key16_of(key_of(acc_of<BASE>(g[c], b[c], r[c])));
                } else {
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        const uint32_t x = e + c;
                        if (x >= seg_a && x < seg_b)
                            k16[4 * q + c] =
                                key16_of(key_of(acc_of<BASE>(a.grad[x], BASE ? a.base[x] : 0.0f, nores ? 0.0f : a.res[x])));
                    }
                }
            }
        }
        uint4* dst = reinterpret_cast<uint4*>(a.skeys + a.skey_base[s] + (size_t)kUnit * j);
        dst[0] = make_uint4(k16[0] | (k16[1] << 16), k16[2] | (k16[3] << 16), k16[4] | (k16[5] << 16),
                            k16[6] | (k16[7] << 16));
        dst[1] = make_uint4(k16[8] | (k16[9] << 16), k16[10] | (k16[11] << 16), k16[12] | (k16[13] << 16),
                            k16[14] | (k16[15] << 16));
    }
    // digit histogram of the nonzero keys; valid and zero counts
    uint32_t nvalid = 0, nzero = 0;
#pragma unroll
    for (int q = 0; q < kUnit; ++q) {
        const bool valid = k16[q] != kNoKey16;
        lds_hist_add(hs, valid ? k16[q] >> kS0Shift : 0u, valid && k16[q] != 0);
        nvalid += valid;
        nzero += valid && k16[q] == 0;
    }
    nvalid = wave_sum(nvalid);
    nzero = wave_sum(nzero);
    if (lane_id() == 0) {
        atomicAdd(&cnt[0], nvalid);
        atomicAdd(&cnt[1], nzero);
    }
    __syncthreads();
    uint32_t* sh = a.shist + (size_t)s * kSHistWords;
    for (int i = tid; i < kNB0; i += kSampleThreads)
        if (hs[i]) atomicAdd(&sh[i], hs[i]);
    if (tid < 2 && cnt[tid]) atomicAdd(&sh[kNB0 + tid], cnt[tid]);
}

// 16-bit prefix of the r-th largest nonzero sample key (r >= 1, at most the
// number of nonzero keys), from the digit histogram hA: a digit pick, then a
// histogram of the low 6 bits among keys with that digit.  Called by the
// whole block; hB is cleared here.
__device__ uint32_t pick16(const uint32_t* hA, uint32_t* hB, uint32_t* par, uint32_t r,
                           const uint32_t (&kw)[kBracketUnits][kUnit / 2], uint32_t units) {
    const int tid = threadIdx.x;
    if (tid < kSNB1) hB[tid] = 0;
    if (tid < kWave) {
        uint32_t d, ab;
        wave_pick<kNB0>(hA, r, d, ab);
        if (tid == 0) {
            par[0] = d;
            par[1] = r - ab;
        }
    }
    __syncthreads();
    const uint32_t dq = par[0];
#pragma unroll
    for (int j = 0; j < kBracketUnits; ++j)
#pragma unroll
        for (int i = 0; i < kUnit; ++i) {
            if (j * kBracketThreads + (tid & ~(kWave - 1)) >= (int)units) continue;  // no unit in this wave
            const uint32_t key = (kw[j][i >> 1] >> ((i & 1) * 16)) & 0xFFFFu;
            lds_hist_add(hB, key & (kSNB1 - 1), key != kNoKey16 && key != 0 && (key >> kS0Shift) == dq);
        }
    __syncthreads();
    if (tid < kWave) {
        uint32_t d, ab;
        wave_pick<kSNB1>(hB, par[1], d, ab);
        if (tid == 0) par[2] = (dq << kS0Shift) | d;
    }
    __syncthreads();
    const uint32_t p = par[2];
    __syncthreads();
    return p;
}

__global__ __launch_bounds__(kBracketThreads) void k_bracket(SampleArgs a) {
    const uint32_t s = blockIdx.x;
    const int tid = threadIdx.x;
    const uint32_t seg_a = a.seg_off[s], seg_b = a.seg_off[s + 1];
    const uint32_t kb_all = load_early(a.skey_base + s);  // with the bounds, not after them
    const uint32_t n = seg_b - seg_a;
    const uint32_t k = keep_of(n, a.keep_ppm);
    __shared__ uint32_t hA[kNB0];
    __shared__ uint32_t hB[kSNB1];
    __shared__ uint32_t hW[kBracketWin * kSNB1];
    __shared__ uint32_t par[4];
    __shared__ uint32_t sums[4];
    uint32_t n16, U;
    sample_units(seg_a, seg_b, n16, U);
    const bool selecting = k > 0 && k < n;
    // thread tid holds sample units tid + j * kBracketThreads, 16 keys each;
    // their loads are issued first, so that they overlap the histogram's
    uint32_t kw[kBracketUnits][kUnit / 2];
    {
        const uint32_t kb = kb_all;
#pragma unroll
        for (int j = 0; j < kBracketUnits; ++j) {
            const uint32_t u = tid + j * kBracketThreads;
            if (selecting && u < U) {
                const uint4* src = reinterpret_cast<const uint4*>(a.skeys + kb + (size_t)kUnit * u);
                const uint4 x0 = src[0], x1 = src[1];
                kw[j][0] = x0.x;
                kw[j][1] = x0.y;
                kw[j][2] = x0.z;
                kw[j][3] = x0.w;
                kw[j][4] = x1.x;
                kw[j][5] = x1.y;
                kw[j][6] = x1.z;
                kw[j][7] = x1.w;
            } else {
#pragma unroll
                for (int i = 0; i < kUnit / 2; ++i) kw[j][i] = 0xFFFFFFFFu;
            }
        }
    }
    // the sample's digit histogram and counts, cleared for the next call
    {
        uint32_t* sh = a.shist + (size_t)s * kSHistWords;
        for (int i = tid; i < kNB0; i += kBracketThreads) hA[i] = sh[i];
        if (tid < 2) sums[tid] = sh[kNB0 + tid];
        if (tid >= 2 && tid < 4) sums[tid] = 0;
        __syncthreads();
        for (int i = tid; i < kSHistWords; i += kBracketThreads) sh[i] = 0;
    }
    uint32_t lo, hi;
    if (k == 0) {
        lo = hi = kNoKey;
    } else if (k >= n) {
        lo = hi = 0;
    } else {
        const uint32_t m = sums[0], mnz = sums[0] - sums[1];
        const bool full = m >= n;  // every element sampled: exact ranks
        const double q = full ? (double)k : (double)k * (double)m / (double)n;
        const uint32_t rq = (uint32_t)fmax(1.0, floor(q + 0.5));
        if (rq > mnz) {
            // the estimate falls among zero keys: candidates are the nonzero
            // entries (or, when every element was sampled and zeros are
            // known to be needed, all of them); nothing is zeroed early
            hi = kNoKey;
            lo = (full && k > mnz) ? 0u : 1u;
        } else {
            // One pass over the sample keys: the fine (low 6-bit) histograms of
            // the kBracketWin coarse digits from dq, the digit holding rank rq,
            // downwards; and per unit, the count of keys at or above dq's floor.
            if (tid < kWave) {
                uint32_t d, ab;
                wave_pick<kNB0>(hA, rq, d, ab);
                if (tid == 0) {
                    par[0] = d;
                    par[1] = rq - ab;
                }
            }
            for (int i = tid; i < kBracketWin * kSNB1; i += kBracketThreads) hW[i] = 0;
            __syncthreads();
            const uint32_t dq = par[0], rf = par[1], floor16 = dq << kS0Shift;
            // The window is digits dq - kBracketWin + 1 .. dq, key16 values
            // [wbase, floor16 + kSNB1), zero keys left out: row r of hW holds
            // digit dq - kBracketWin + 1 + r.  Each key costs a subtraction and a
            // compare for the window and for the unit count (kNoKey16, a missing
            // key, falls outside both).
            const uint32_t wbase = dq >= (uint32_t)(kBracketWin - 1) ? (dq - (kBracketWin - 1)) << kS0Shift : 0u;
            const uint32_t wlo = wbase ? wbase : 1u, wspan = floor16 + kSNB1 - wlo;
            uint32_t* const hwin = hW + (wlo - wbase);
            const uint32_t cspan = kNoKey16 - floor16;
            uint32_t s1 = 0, s2 = 0;  // this thread's units: sum of counts and of squared counts
#pragma unroll
            for (int j = 0; j < kBracketUnits; ++j) {
                if (j * kBracketThreads + (tid & ~(kWave - 1)) >= (int)U) continue;  // no unit in this wave
                uint32_t c = 0;
#pragma unroll
                for (int i = 0; i < kUnit; ++i) {
                    const uint32_t key = (kw[j][i >> 1] >> ((i & 1) * 16)) & 0xFFFFu;
                    const uint32_t t = key - wlo;
                    if (t < wspan) atomicAdd(&hwin[t], 1u);
                    c += key - floor16 < cspan;
                }
                s1 += c;
                s2 += c * c;
            }
            if (!full) {
                s1 = wave_sum(s1);
                s2 = wave_sum(s2);
                if (lane_id() == 0) {
                    atomicAdd(&sums[2], s1);
                    atomicAdd(&sums[3], s2);
                }
            }
            __syncthreads();
            // P: the fine bin of rank rf within digit dq
            if (tid < kWave) {
                uint32_t f, ab;
                wave_pick<kSNB1>(hW + (kBracketWin - 1) * kSNB1, rf, f, ab);
                if (tid == 0) par[2] = floor16 | f;
            }
            __syncthreads();
            const uint32_t P = par[2];
            hi = (P + 1u) << kK16Shift;
            if (full) {
                lo = P << kK16Shift;
            } else {
                // The spread of the per-unit counts at dq's floor, as a
                // dispersion index (variance over mean), carried over to the
                // count at the estimate: sd = sqrt(q * max(1, index)).
                const double mean = (double)sums[2] / U;
                const double var = fmax((double)sums[3] / U - mean * mean, 0.0);
                const double disp = mean > 0.0 ? var / mean : 1.0;
                // whether the next call may sample runs of neighbours: the
                // counts spread no more than independent draws (index about 1),
                // whichever way this sample was drawn
                if (tid == 0 && mean > 0.0) a.seg[s].runs = disp < kRunsMaxDispersion ? 1u : 0u;
                const double sd = sqrt(q * fmax(1.0, disp));
                const double fl = ceil(q + 5.0 * sd + 4.0);
                if (fl > (double)mnz) {
                    lo = 1u;  // the margin reaches the zero keys
                } else {
                    // rank fl lies in digit dl <= dq: within the window, or
                    // (rarely) one more pass over the keys
                    if (tid < kWave) {
                        uint32_t dl, abl, lo16 = kNoKey;
                        wave_pick<kNB0>(hA, (uint32_t)fl, dl, abl);
                        if (dq - dl < (uint32_t)kBracketWin) {
                            uint32_t f, ab;
                            wave_pick<kSNB1>(hW + (kBracketWin - 1 - (dq - dl)) * kSNB1, (uint32_t)fl - abl, f, ab);
                            lo16 = (dl << kS0Shift) | f;
                        }
                        if (tid == 0) par[3] = lo16;
                    }
                    __syncthreads();
                    uint32_t lo16 = par[3];
                    __syncthreads();
                    if (lo16 == kNoKey) lo16 = pick16(hA, hB, par, (uint32_t)fl, kw, U);
                    lo = lo16 << kK16Shift;
                    if (lo == 0) lo = 1;
                }
            }
        }
    }
    if (a.debug_bracket == kDebugLoTooHigh && k > 0) {
        lo = 0x7FFFFFFFu;
        hi = kNoKey;
    } else if (a.debug_bracket == kDebugHiAtLo) {
        hi = lo;
    } else if (a.debug_bracket == kDebugLoZero && k > 0) {
        lo = 0;
    } else if (a.debug_bracket == kDebugLoAtHi && k > 0 && k < n) {
        lo = hi;
    }
    if (tid == 0) {
        a.seg[s].lo = lo;
        a.seg[s].hi = hi;
    }
}

hipError_t launch_sample(const SampleArgs& a, bool has_base, hipStream_t st) {
    if ((uint64_t)kSampleBlocks * a.S > 0x7FFFFFFFull) return hipErrorInvalidConfiguration;
    const dim3 grid(kSampleBlocks * a.S);
    if (has_base) hipLaunchKernelGGL(k_sample<true>, grid, dim3(kSampleThreads), 0, st, a);
    else hipLaunchKernelGGL(k_sample<false>, grid, dim3(kSampleThreads), 0, st, a);
    hipLaunchKernelGGL(k_bracket, dim3(a.S), dim3(kBracketThreads), 0, st, a);
    return hipGetLastError();
}

}  // namespace gd
