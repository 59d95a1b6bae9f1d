// The dense pass of gradient dropping (gfx950, wave64).
//
// Algorithm 1 (Section 4): add the carried residual to the gradient, and
// (together with the later passes) keep the largest |acc|, leaving the rest
// as the new residual.  This kernel is the only one that streams the whole
// gradient: per element it reads grad (and, for a pull, the last pulled
// copy) and the residual, writes the residual back where it changes (a
// 16-byte vector whose four values keep their bits is not stored: a zero
// gradient leaves acc equal to the residual), and appends the few
// elements whose key reaches the sampled bracket (key >= lo) to per-unit
// slots in ascending index order.  Elements with key >= hi are almost
// surely kept, so their residual is written as +0 now; the emit pass fixes
// the few that end up on the other side of the exact threshold.  A pull from
// the last pulled copy has no residual: it reads params and the copy only.
//
// A unit is the 1024 elements [1024u, 1024u + 1024) of the flat gradient,
// one block of 256 threads with one 16-byte vector per thread, so every
// load is aligned and issued before any table lookup.  The streamed arrays
// are loaded as non-temporal, and the residual's changed vectors stored with
// device scope (see unit_rsrc), so that the residual does not fill the L2
// with dirty lines while the pass streams.  The block compacts
// the unit's candidates into slots [1024u, ...) and stores their count.  A unit
// that holds a tensor boundary also records, for each tensor starting inside
// it, how many of its candidates precede that start (the candidate layout
// needs it).

#include <hip/hip_ext.h>

#include "gd_kernels.h"

namespace gd {

// The residual's stores go out as buffer stores with device scope (SC1) and
// no other cache bits.  While the pass streams its reads, such stores disturb
// the read stream less than non-temporal or plain stores: with 8% of the
// residual's 2000-byte rows rewritten at scattered places, a 137M-element
// read-and-store stream measured 186 us against 198 (non-temporal) and
// 192 us (plain); the pass itself 185.5 against 187.4 us at the NMT-shaped
// layout and 36.5 against 39.0 at the 20M-element MLP.  The resource covers
// one unit's bytes, so the 32-bit offsets never wrap and a store past the
// unit would be dropped by the hardware.
constexpr int kStoreDeviceScope = 16;  // cache-policy operand: SC1
// Fourth word of the resource: data format 32 bits (field value 4 in bits
// 18..15), the setting for untyped raw buffer access on this architecture.
constexpr int kRawBufferWord3 = 0x00020000;

// A raw buffer resource over `bytes` bytes from `base` (stride 0: offsets
// are byte offsets, and the hardware drops accesses at or past `bytes`).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t unit_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, bytes, kRawBufferWord3);
}

template <bool BASE>
__device__ __forceinline__ float acc_of(float g, float b, float r) {
    // Two separate binary32 roundings when a base is given (pull deltas).
    if (BASE) {
        const float d = g - b;
        return d + r;
    }
    return g + r;
}

// Tensor holding element e: the last t with off[t] <= e (empty tensors share
// their successor's offset, so the last one is the tensor that holds e).
__device__ __forceinline__ uint32_t tensor_of(const uint32_t* off, uint32_t T, uint32_t e) {
    uint32_t lo = 0, hi = T;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (off[mid] <= e) lo = mid;
        else hi = mid;
    }
    return lo;
}

// MODE 0: acc = grad + residual; 1: (grad - base) + residual (a pull with a
// residual); 2: grad - base with no residual at all (a pull from the last
// pulled copy, which keeps the unsent difference itself).
constexpr int kDenseThreads = kUnitLen / 4;  // one 16-byte vector per lane and input array
constexpr int kDenseWaves = kDenseThreads / kWave;

template <int MODE>
__global__ __launch_bounds__(kDenseThreads) void k_dense(DenseArgs a) {
    constexpr bool BASE = MODE >= 1, NORES = MODE == 2;
    const uint32_t u = blockIdx.x;
    const int tid = threadIdx.x, w = tid >> 6, lane = lane_id();
    const uint32_t ustart = u * kUnitLen;
    // ends and vector tests without 32-bit wrap-around (N may come within a unit of 2^32)
    const uint32_t uend = a.N - ustart > kUnitLen ? ustart + kUnitLen : a.N;
    const uint32_t e0 = ustart + 4 * tid;

    f4 g = {0.f, 0.f, 0.f, 0.f}, b = g, r = g;
    const bool whole = e0 < uend && uend - e0 >= 4;  // all four elements of this lane exist
    if (whole) {
        g = __builtin_nontemporal_load(reinterpret_cast<const f4*>(a.grad) + (e0 >> 2));
        if (BASE) b = __builtin_nontemporal_load(reinterpret_cast<const f4*>(a.base) + (e0 >> 2));
        if (!NORES) r = __builtin_nontemporal_load(reinterpret_cast<const f4*>(a.res) + (e0 >> 2));
    } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (e0 + q < uend) {
                g[q] = a.grad[e0 + q];
                if (BASE) b[q] = a.base[e0 + q];
                if (!NORES) r[q] = a.res[e0 + q];
            }
        }
    }
    const uint32_t info = a.unit_info[u];
    const bool boundary = (info >> 31) != 0;
    uint32_t lo[4], hi[4];
    if (!a.per_tensor || !boundary) {
        const uint32_t s = a.per_tensor ? (info & 0x7FFFFFFFu) : 0u;
        const uint32_t l = a.seg[s].lo, h = a.seg[s].hi;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            lo[q] = l;
            hi[q] = h;
        }
    } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            lo[q] = hi[q] = kNoKey;
            if (e0 + q < uend) {
                const uint32_t s = tensor_of(a.tensor_off, a.T, e0 + q);
                lo[q] = a.seg[s].lo;
                hi[q] = a.seg[s].hi;
            }
        }
    }
    float acc[4];
    bool cand[4];
    f4 ov;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const bool valid = e0 + q < uend;
        acc[q] = NORES ? g[q] - b[q] : acc_of<BASE>(g[q], b[q], r[q]);
        const uint32_t key = key_of(acc[q]);
        cand[q] = valid && key >= lo[q];
        ov[q] = (valid && key >= hi[q]) ? 0.0f : acc[q];
    }
    if (!NORES) {
        // Only what changes is written back.  Where the gradient is zero (the
        // rows of an embedding that no word of the batch touched) acc equals
        // the residual bit for bit and nothing is stored: such rows cost
        // their 8 bytes of reads, not 12.  The test is on bit patterns, so
        // -0 and +0 count as different.
        if (whole) {
            bool same = true;
#pragma unroll
            for (int q = 0; q < 4; ++q) same = same && __float_as_uint(ov[q]) == __float_as_uint(r[q]);
            if (!same) {
                typedef unsigned u4 __attribute__((ext_vector_type(4)));
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4, ov), unit_rsrc(a.res + ustart, 4 * (uend - ustart)),
                                                       16u * tid, 0, kStoreDeviceScope);
            }
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (e0 + q < uend && __float_as_uint(ov[q]) != __float_as_uint(r[q])) a.res[e0 + q] = ov[q];
        }
    }
    // ordered compaction over the unit: waves in order, lanes in order, then
    // the four elements of a lane, into one contiguous list per unit (fewer
    // partially written cache lines than a list per wave)
    const uint64_t m0 = ballot(cand[0]), m1 = ballot(cand[1]), m2 = ballot(cand[2]), m3 = ballot(cand[3]);
    __shared__ uint32_t qc[kDenseWaves];
    if (lane == 0) qc[w] = popc64(m0) + popc64(m1) + popc64(m2) + popc64(m3);
    __syncthreads();
    uint32_t base = 0, total = 0;
#pragma unroll
    for (int i = 0; i < kDenseWaves; ++i) {
        base += i < w ? qc[i] : 0u;
        total += qc[i];
    }
    if ((m0 | m1 | m2 | m3) != 0) {
        // plain stores: gather reads the lists next, partly from the cache
        // (device-scope or non-temporal stores here cost the pass 8 us at the
        // NMT-shaped layout)
        uint32_t pos = base + lanes_below(m0) + lanes_below(m1) + lanes_below(m2) + lanes_below(m3);
        uint2* out = a.slots + ustart;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (cand[q]) {
                out[pos] = make_uint2(e0 + q, __float_as_uint(acc[q]));
                ++pos;
            }
        }
    }
    if (tid == 0) a.cnt[u] = total;
    if (boundary) {
        // candidates before each tensor start strictly inside the unit
        __shared__ uint32_t red[kDenseWaves];
        for (uint32_t t = (info & 0x7FFFFFFFu) + 1; t < a.T && a.tensor_off[t] < uend; ++t) {
            const uint32_t x = a.tensor_off[t];
            if (x <= ustart) continue;
            uint32_t c = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) c += cand[q] && e0 + q < x;
            c = wave_sum(c);
            __syncthreads();
            if (lane == 0) red[w] = c;
            __syncthreads();
            if (tid == 0) {
                uint32_t sum = 0;
#pragma unroll
                for (int i = 0; i < kDenseWaves; ++i) sum += red[i];
                a.split[t] = sum;
            }
        }
    }
}

// When t0 and t1 are given, the dispatch itself records them at its start and
// end (no separate marker packets on the stream, so the timing adds no gap).
hipError_t launch_dense(const DenseArgs& a, bool has_base, hipStream_t st, hipEvent_t t0, hipEvent_t t1) {
    if (a.num_units == 0) return hipSuccess;
    const dim3 grid(a.num_units), block(kDenseThreads);
    auto k = has_base && a.res == nullptr ? k_dense<2> : has_base ? k_dense<1> : k_dense<0>;
    if (t0 != nullptr && t1 != nullptr) hipExtLaunchKernelGGL(k, grid, block, 0, st, t0, t1, 0, a);
    else hipLaunchKernelGGL(k, grid, block, 0, st, a);
    return hipGetLastError();
}

}  // namespace gd
