// The dense pass of gradient dropping (gfx950, wave64).
//
// Algorithm 1 (Section 4): add the carried residual to the gradient, and
// (together with the later passes) keep the largest |acc|, leaving the rest
// as the new residual.  This kernel is the only one that streams the whole
// gradient: per element it reads grad (and, for a pull, the last pulled
// copy) and the residual, writes the residual back, and appends the few
// elements whose key reaches the sampled bracket (key >= lo) to per-unit
// slots in ascending index order.  Elements with key >= hi are almost
// surely kept, so their residual is written as +0 now; the emit pass fixes
// the few that end up on the other side of the exact threshold.
//
// A unit is up to 1024 consecutive elements of one tensor, processed by one
// wave: four 16-byte loads per lane per input array, all issued before use.

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

template <bool BASE>
__global__ __launch_bounds__(kBlock) void k_dense(DenseArgs a) {
    const int w = threadIdx.x >> 6, lane = lane_id();
    const uint32_t c = blockIdx.x * kWavesPerBlock + w;
    if (c >= a.num_chunks) return;

    const uint32_t start = a.chunk_start[c], len = a.chunk_len[c], end = start + len;
    const uint32_t vb = start >> 2, ve = (end + 3) >> 2;
    const f4* g4 = reinterpret_cast<const f4*>(a.grad);
    const f4* b4 = reinterpret_cast<const f4*>(BASE ? a.base : a.grad);
    f4* r4 = reinterpret_cast<f4*>(a.res);
    uint2* out = a.slots + start;
    uint32_t nc = 0;

    for (uint32_t v0 = vb; v0 < ve; v0 += 4 * kWave) {
        // Issue every load of this step before the table lookups they do not need.
        f4 g[4], b[4], r[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const uint32_t v = v0 + u * kWave + lane;
            const uint32_t e0 = 4 * v;
            const f4 z = {0.f, 0.f, 0.f, 0.f};
            g[u] = z;
            b[u] = z;
            r[u] = z;
            if (v < ve) {
                if (e0 >= start && e0 + 4 <= end) {
                    g[u] = __builtin_nontemporal_load(g4 + v);
                    if (BASE) b[u] = __builtin_nontemporal_load(b4 + v);
                    r[u] = r4[v];
                } else {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const uint32_t e = e0 + q;
                        if (e >= start && e < end) {
                            g[u][q] = a.grad[e];
                            if (BASE) b[u][q] = a.base[e];
                            r[u][q] = a.res[e];
                        }
                    }
                }
            }
        }
        const uint32_t s = a.per_tensor ? a.chunk_tensor[c] : 0u;
        const uint32_t lo = a.seg[s].lo, hi = a.seg[s].hi;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const uint32_t v = v0 + u * kWave + lane;
            const uint32_t e0 = 4 * v;
            const bool inside = v < ve;
            const bool full = inside && e0 >= start && e0 + 4 <= end;
            float acc[4];
            bool cand[4];
            f4 ov;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t e = e0 + q;
                const bool valid = inside && e >= start && e < end;
                acc[q] = acc_of<BASE>(g[u][q], b[u][q], r[u][q]);
                const uint32_t key = key_of(acc[q]);
                cand[q] = valid && key >= lo;
                ov[q] = (valid && key >= hi) ? 0.0f : acc[q];
            }
            if (full) {
                r4[v] = ov;
            } else if (inside) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const uint32_t e = e0 + q;
                    if (e >= start && e < end) a.res[e] = ov[q];
                }
            }
            const uint64_t m0 = ballot(cand[0]), m1 = ballot(cand[1]), m2 = ballot(cand[2]), m3 = ballot(cand[3]);
            if ((m0 | m1 | m2 | m3) != 0) {
                uint32_t pos = nc + lanes_below(m0) + lanes_below(m1) + lanes_below(m2) + lanes_below(m3);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (cand[q]) {
                        out[pos] = make_uint2(e0 + q, __float_as_uint(acc[q]));
                        ++pos;
                    }
                }
                nc += popc64(m0) + popc64(m1) + popc64(m2) + popc64(m3);
            }
        }
    }
    if (lane == 0) a.cnt_lo[c] = nc;
}

static inline uint32_t blocks_for_waves(uint32_t waves) { return (waves + kWavesPerBlock - 1) / kWavesPerBlock; }

hipError_t launch_dense(const DenseArgs& a, bool has_base, hipStream_t st) {
    if (a.num_chunks == 0) return hipSuccess;
    const dim3 grid(blocks_for_waves(a.num_chunks));
    if (has_base) hipLaunchKernelGGL(k_dense<true>, grid, dim3(kBlock), 0, st, a);
    else hipLaunchKernelGGL(k_dense<false>, grid, dim3(kBlock), 0, st, a);
    return hipGetLastError();
}

}  // namespace gd
