// The paper's own threshold: selection on a sample (gfx950, wave64).
//
// Section 4 approximates the expensive selection by sampling 0.1% of the
// gradient and selecting on the sample; Algorithm 1 then keeps every entry
// strictly above the threshold, so the number kept depends on the data.
//
//   k_ssample : segment s of n entries draws m = ceil(n * sample_ppm / 1e6)
//               positions, one per stratum [floor(j n / m), floor((j+1) n / m)),
//               at the offset given by output 2^32 s + j of SplitMix64 seeded
//               by the caller (Steele, Lea and Flood, OOPSLA 2014), stores the
//               key of acc at each position and adds the keys' top 11 bits to
//               the segment's histogram (one of several copies by block
//               number, so few global adds meet on a bin).  It also clears the per-tensor counts and the segment's
//               candidate state.
//   k_sselect : one block per segment takes the (k_m + 1)-th largest sample key
//               T (k_m = floor(m * keep_ppm / 1e6); the largest when k_m = 0):
//               the top digit from that histogram, then the keys sharing it
//               gathered into LDS in one pass and two 10-bit digits resolved
//               there (or, when too many share it, two more passes over all
//               sample keys).  It sets the dense pass's bracket to
//               [T + 1, T + 1): every candidate is then kept and zeroed by the
//               dense pass itself, and the later passes only compact them.
//               k_m >= m keeps every entry, R = 1 none.

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

// Output number i of SplitMix64 seeded with `seed`: the state advances by the
// golden-ratio increment per output and passes through two xor-shift-multiply
// rounds and a final xor-shift.
__device__ __forceinline__ uint64_t splitmix64_at(uint64_t seed, uint64_t i) {
    uint64_t z = seed + (i + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ uint32_t sample_count(uint32_t n, uint32_t sample_ppm) {
    return (uint32_t)(((uint64_t)n * sample_ppm + 999999u) / 1000000u);
}

template <bool BASE>
__global__ __launch_bounds__(kSsThreads) void k_ssample(SampledArgs a, uint32_t bps) {
    // a 1-D grid of bps blocks per segment (no limit on segments)
    const uint32_t s = blockIdx.x / bps, bx = blockIdx.x % bps;
    const int tid = threadIdx.x;
    const uint32_t seg_a = a.seg_off[s], n = a.seg_off[s + 1] - seg_a;
    if (bx == 0) {
        if (tid == 0) {
            a.seg[s].clo = 0;
            a.seg[s].miss = 0;
        }
        // counts of the tensors this segment covers (the emit pass writes them
        // only for tensors that have candidates)
        if (a.per_tensor) {
            if (tid == 0) a.tensor_counts[s] = 0;
        } else {
            for (uint32_t t = tid; t < a.T; t += kSsThreads) a.tensor_counts[t] = 0;
        }
    }
    const uint32_t m = sample_count(n, a.sample_ppm);
    const uint32_t j0 = bx * (kSsThreads * kSsPerThread);
    if (j0 >= m) return;  // block-uniform
    __shared__ uint32_t h[kSsNB0];
    for (int i = tid; i < kSsNB0; i += kSsThreads) h[i] = 0;
    __syncthreads();
    uint32_t key[kSsPerThread];
    bool ok[kSsPerThread];
#pragma unroll
    for (int q = 0; q < kSsPerThread; ++q) {
        const uint32_t j = j0 + q * kSsThreads + tid;
        ok[q] = j < m;
        const uint32_t jj = ok[q] ? j : j0;  // unconditional loads, all in flight
        const uint64_t lo = (uint64_t)jj * n / m, hi = (uint64_t)(jj + 1) * n / m;
        const uint64_t z = splitmix64_at(a.seed, ((uint64_t)s << 32) | jj);
        const uint32_t e = seg_a + (uint32_t)(lo + z % (hi - lo));
        key[q] = key_of(acc_of<BASE>(a.grad[e], BASE ? a.base[e] : 0.0f, a.res[e]));
    }
#pragma unroll
    for (int q = 0; q < kSsPerThread; ++q) {
        if (ok[q]) a.skeys[seg_a + j0 + q * kSsThreads + tid] = key[q];
        lds_hist_add(h, key[q] >> kSsD0Shift, ok[q]);
    }
    __syncthreads();
    uint32_t* gh = a.sshist + ((size_t)s * kSsCopies + bx % kSsCopies) * kSsNB0;
    for (int i = tid; i < kSsNB0; i += kSsThreads)
        if (h[i]) atomicAdd(&gh[i], h[i]);
}

// Digit holding the r-th largest (0-based) of the counts in h[0..NB) (bins in
// ascending key order), and how many counted keys lie in higher bins.  Called
// by the whole block; par receives {digit, above}.
template <int NB>
__device__ void block_select(const uint32_t* h, uint32_t r, uint32_t* scan_lds, uint32_t* par) {
    constexpr int PER = NB / kSsSelThreads;
    static_assert(PER >= 1 && NB % kSsSelThreads == 0, "bins per thread");
    const int tid = threadIdx.x;
    // thread t owns bins [NB - PER (t + 1), NB - PER t), visited high to low
    const int top = NB - PER * tid;
    uint32_t c[PER], sum = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        c[i] = h[top - 1 - i];
        sum += c[i];
    }
    uint32_t total;
    const uint32_t excl = block_excl_scan<kSsSelThreads>(sum, scan_lds, &total);
    if (excl <= r && r < excl + sum) {
        uint32_t acc = excl;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            if (acc <= r && r < acc + c[i]) {
                par[0] = (uint32_t)(top - 1 - i);
                par[1] = acc;
            }
            acc += c[i];
        }
    }
    __syncthreads();
}

__global__ __launch_bounds__(kSsSelThreads) void k_sselect(SampledArgs a) {
    const uint32_t s = blockIdx.x;
    const int tid = threadIdx.x;
    const uint32_t seg_a = a.seg_off[s], n = a.seg_off[s + 1] - seg_a;
    const uint32_t m = sample_count(n, a.sample_ppm);
    const uint32_t km = (uint32_t)((uint64_t)m * a.keep_ppm / 1000000u);
    __shared__ uint32_t h[kSsNB0];
    __shared__ uint32_t list[kSsList];
    __shared__ uint32_t scan_lds[kSsSelThreads / kWave + 1];
    __shared__ uint32_t par[3];
    uint32_t* gh = a.sshist + (size_t)s * kSsCopies * kSsNB0;
    for (int i = tid; i < kSsNB0; i += kSsSelThreads) {
        uint32_t c[kSsCopies], sum = 0;
#pragma unroll
        for (int q = 0; q < kSsCopies; ++q) c[q] = gh[q * kSsNB0 + i];
#pragma unroll
        for (int q = 0; q < kSsCopies; ++q) {
            sum += c[q];
            gh[q * kSsNB0 + i] = 0;  // ready for the next call
        }
        h[i] = sum;
    }
    if (tid == 0) par[0] = par[1] = par[2] = 0;
    __syncthreads();
    uint32_t lo;
    if (n == 0 || a.keep_ppm == 0) {
        lo = kNoKey;  // above every key: nothing is a candidate
    } else if (km >= m) {
        lo = 0;  // every entry is kept
    } else {
        const uint32_t* keys = a.skeys + seg_a;
        // digit 0 (key bits 30..20) from the sampler's histogram
        uint32_t r = km;
        block_select<kSsNB0>(h, r, scan_lds, par);
        const uint32_t d0 = par[0];
        r -= par[1];
        const uint32_t in_bin = h[d0];
        __syncthreads();
        if (tid == 0) par[2] = 0;
        __syncthreads();
        // the keys sharing digit 0, gathered into LDS when they fit
        const bool fits = in_bin <= (uint32_t)kSsList;
        if (fits) {
            for (uint32_t i0 = 0; i0 < m; i0 += kSsSelThreads * kSsBatch) {
                uint32_t k[kSsBatch];
#pragma unroll
                for (int q = 0; q < kSsBatch; ++q) {
                    const uint32_t i = i0 + q * kSsSelThreads + tid;
                    const uint32_t v = keys[i < m ? i : 0u];  // unconditional: all in flight
                    k[q] = i < m ? v : kNoKey;
                }
#pragma unroll
                for (int q = 0; q < kSsBatch; ++q) {
                    if (k[q] != kNoKey && (k[q] >> kSsD0Shift) == d0) {
                        const uint32_t slot = atomicAdd(&par[2], 1u);
                        if (slot < (uint32_t)kSsList) list[slot] = k[q];
                    }
                }
            }
        }
        __syncthreads();
        // the list is used only when it holds every key sharing digit 0
        const uint32_t got = par[2];
        const bool use_list = fits && got <= (uint32_t)kSsList;
        // digits 1 (bits 19..10) and 2 (bits 9..0) among them
        uint32_t prefix = d0;
        for (int level = 1; level <= 2; ++level) {
            const int shift = level == 1 ? 10 : 0;
            for (int i = tid; i < 1024; i += kSsSelThreads) h[i] = 0;
            __syncthreads();
            if (use_list) {
                for (uint32_t i = tid; i < got; i += kSsSelThreads) {
                    const uint32_t k = list[i];
                    lds_hist_add(h, (k >> shift) & 1023u, (k >> (shift + 10)) == prefix);
                }
            } else {
                for (uint32_t i = tid; i < m; i += kSsSelThreads) {
                    const uint32_t k = keys[i];
                    lds_hist_add(h, (k >> shift) & 1023u, (k >> (shift + 10)) == prefix);
                }
            }
            __syncthreads();
            block_select<1024>(h, r, scan_lds, par);
            prefix = (prefix << 10) | par[0];
            r -= par[1];
            __syncthreads();
        }
        lo = prefix + 1u;  // keep key > T = prefix
    }
    if (tid == 0) {
        a.seg[s].lo = lo;
        a.seg[s].hi = lo;
        a.seg[s].thr = lo > 0 ? lo - 1u : 0u;
        a.seg[s].need = 0;
    }
}

hipError_t launch_sampled(const SampledArgs& a, bool has_base, uint32_t max_samples, hipStream_t st) {
    constexpr uint32_t per_block = kSsThreads * kSsPerThread;
    const uint32_t bps = max_samples > 0 ? (max_samples + per_block - 1) / per_block : 1u;
    if ((uint64_t)bps * a.S > 0x7FFFFFFFull) return hipErrorInvalidConfiguration;
    const dim3 grid(bps * a.S);
    if (has_base) hipLaunchKernelGGL(k_ssample<true>, grid, dim3(kSsThreads), 0, st, a, bps);
    else hipLaunchKernelGGL(k_ssample<false>, grid, dim3(kSsThreads), 0, st, a, bps);
    hipLaunchKernelGGL(k_sselect, dim3(a.S), dim3(kSsSelThreads), 0, st, a);
    return hipGetLastError();
}

}  // namespace gd
