// Gradient-dropping kernels for gfx950 (wave64).
//
// One gd_compress call runs, on the caller's stream and without any host
// synchronisation:
//   k_sample   : keys of a stratified sample of acc per threshold segment,
//                then (last block of each segment) a bracket [lo, hi) that
//                very likely contains the k-th largest key.
//   k_dense    : the single pass over the dense data: acc = grad + residual,
//                residual <- (key >= hi ? +0 : acc), candidates (key >= lo)
//                appended in index order to per-chunk slots, digit-0
//                histogram of the candidates.
//   k_fb_*     : only for segments whose bracket missed (fewer than k
//                candidates): restore residual = acc and make every element a
//                candidate.  Other segments return at once.
//   k_radix1/2 : digits 1 and 2 of the exact k-th largest key, from the
//                candidates only.
//   k_count    : the threshold key T, the number of ties to keep, and per
//                group counts of keys above / equal to T.
//   k_emit     : kept (index, value) pairs in ascending index order, residual
//                fix-ups, kept counts per tensor.
//   k_means, k_quant : per-tensor sign-mean quantisation (optional).
// k_apply is the server-side sparse apply.
//
// The method: Algorithm 1 (Section 4) of Aji & Heafield, "Sparse Communication
// for Distributed Gradient Descent": add the residual, keep the entries whose
// magnitude is among the largest (1 - R), keep the rest as the residual.

#include "gd_kernels.h"

namespace gd {

// ---------------------------------------------------------------------------
// small helpers
// ---------------------------------------------------------------------------

template <bool BASE>
__device__ __forceinline__ float acc_of(float g, float b, float r) {
    // Two separate binary32 roundings when a base is given (pull deltas).
    if (BASE) {
        const float d = g - b;
        return d + r;
    }
    return g + r;
}

// Inclusive scan over a 1024-thread block (16 waves).
__device__ uint32_t block1024_incl_scan(uint32_t v, uint32_t* lds16) {
    const int w = threadIdx.x >> 6, lane = lane_id();
    const uint32_t incl = wave_incl_scan(v);
    if (lane == kWave - 1) lds16[w] = incl;
    __syncthreads();
    uint32_t carry = 0;
    for (int i = 0; i < w; ++i) carry += lds16[i];
    __syncthreads();
    return incl + carry;
}

// ---------------------------------------------------------------------------
// k_sample: stratified sample keys and the bracket per segment
// ---------------------------------------------------------------------------

template <bool BASE>
__device__ void sample_unit(const SampleArgs& a, uint32_t s, uint32_t j, uint32_t U, uint32_t n16, uint32_t seg_a,
                            uint32_t seg_b) {
    const uint32_t first = seg_a >> 4;
    const uint32_t lo_j = (uint32_t)(((uint64_t)j * n16) / U);
    const uint32_t hi_j = (uint32_t)(((uint64_t)(j + 1) * n16) / U);
    uint32_t pick = 0;
    if (U != n16) pick = mix32(j * 0x9E3779B9u ^ (s + 1u) * 0x85EBCA6Bu) % (hi_j - lo_j);
    const uint32_t e0 = (first + lo_j + pick) * kUnit;
    uint32_t* dst = a.skeys + a.skey_base[s] + (size_t)kUnit * j;
    if (e0 >= seg_a && e0 + kUnit <= seg_b) {
        const f4* g4 = reinterpret_cast<const f4*>(a.grad + e0);
        const f4* r4 = reinterpret_cast<const f4*>(a.res + e0);
        const f4* b4 = reinterpret_cast<const f4*>(BASE ? a.base + e0 : a.grad + e0);
        uint4* d4 = reinterpret_cast<uint4*>(dst);
#pragma unroll
        for (int q = 0; q < kUnit / 4; ++q) {
            const f4 g = g4[q], r = r4[q];
            f4 b = g;
            if (BASE) b = b4[q];
            uint4 k;
            k.x = key_of(acc_of<BASE>(g.x, b.x, r.x));
            k.y = key_of(acc_of<BASE>(g.y, b.y, r.y));
            k.z = key_of(acc_of<BASE>(g.z, b.z, r.z));
            k.w = key_of(acc_of<BASE>(g.w, b.w, r.w));
            d4[q] = k;
        }
    } else {
        for (int q = 0; q < kUnit; ++q) {
            const uint32_t e = e0 + q;
            uint32_t k = kNoKey;
            if (e >= seg_a && e < seg_b) k = key_of(acc_of<BASE>(a.grad[e], BASE ? a.base[e] : 0.0f, a.res[e]));
            dst[q] = k;
        }
    }
}

template <bool BASE>
__global__ __launch_bounds__(kSampleThreads) void k_sample(SampleArgs a) {
    const uint32_t s = blockIdx.y;
    const int tid = threadIdx.x;
    const uint32_t seg_a = a.seg_off[s], seg_b = a.seg_off[s + 1];
    const uint32_t n = seg_b - seg_a;
    __shared__ uint32_t lds16[16];
    __shared__ int s_last;

    // Clear this segment's histograms and counters for the passes that follow.
    uint32_t* h = a.hist + (size_t)s * kHistWords;
    for (uint32_t i = blockIdx.x * kSampleThreads + tid; i < (uint32_t)kHistWords; i += gridDim.x * kSampleThreads)
        h[i] = 0;
    if (blockIdx.x == 0 && tid == 0) {
        a.seg[s].clo = 0;
        a.seg[s].chi = 0;
    }
    if (s == 0 && blockIdx.x == 0) {
        for (uint32_t t = tid; t < a.T; t += kSampleThreads) a.tensor_counts[t] = 0;
        // First output slot of each segment: exclusive prefix of k_s.
        __shared__ uint32_t s_tot;
        uint32_t carry = 0;
        for (uint32_t b0 = 0; b0 < a.S; b0 += kSampleThreads) {
            const uint32_t ss = b0 + tid;
            const uint32_t ks = ss < a.S ? keep_of(a.seg_off[ss + 1] - a.seg_off[ss], a.keep_ppm) : 0u;
            const uint32_t incl = block1024_incl_scan(ks, lds16);
            if (ss < a.S) a.out_base[ss] = (uint64_t)carry + (incl - ks);
            if (tid == kSampleThreads - 1) s_tot = incl;
            __syncthreads();
            carry += s_tot;
            __syncthreads();
        }
    }

    const uint32_t n16 = n ? ((seg_b - 1) >> 4) - (seg_a >> 4) + 1 : 0u;
    const uint32_t U = n16 < (uint32_t)kMaxUnits ? n16 : (uint32_t)kMaxUnits;
    const uint32_t j = blockIdx.x * kSampleThreads + tid;
    if (j < U) sample_unit<BASE>(a, s, j, U, n16, seg_a, seg_b);

    // The last block of this segment to finish computes the bracket.
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = (atomicAdd(&a.seg_done[s], 1u) == gridDim.x - 1);
    __syncthreads();
    if (!s_last) return;
    __threadfence();

    __shared__ uint32_t hA[kNB0];
    __shared__ uint32_t hB[2][kNB1];
    __shared__ uint32_t par[8];
    const uint32_t k = keep_of(n, a.keep_ppm);
    uint32_t lo, hi;
    if (k == 0) {
        lo = hi = kNoKey;
    } else if (k >= n) {
        lo = hi = 0;
    } else {
        const uint32_t nkeys = kUnit * U;
        const uint32_t* keys = a.skeys + a.skey_base[s];
        for (int i = tid; i < kNB0; i += kSampleThreads) hA[i] = 0;
        for (int i = tid; i < 2 * kNB1; i += kSampleThreads) (&hB[0][0])[i] = 0;
        if (tid == 0) par[0] = 0;
        __syncthreads();
        uint32_t mine = 0;
        for (uint32_t i = tid; i < nkeys; i += kSampleThreads) {
            const uint32_t key = keys[i];
            if (key != kNoKey) {
                atomicAdd(&hA[key >> kD0Shift], 1u);
                ++mine;
            }
        }
        mine = wave_sum(mine);
        if (lane_id() == 0 && mine) atomicAdd(&par[0], mine);
        __syncthreads();
        if (tid == 0) {
            const uint32_t m = par[0];
            uint32_t r_hi, r_lo;
            if (m >= n) {  // every element sampled: the exact rank
                r_hi = r_lo = k;
            } else {
                const double q = (double)k * (double)m / (double)n;
                const double sd = sqrt(q);
                const double fh = floor(q - 3.0 * sd - 2.0);
                const double fl = ceil(q + 5.0 * sd + 4.0);
                r_hi = fh < 1.0 ? 0u : (uint32_t)fh;
                r_lo = fl > (double)m ? 0u : (uint32_t)fl;
            }
            par[1] = r_hi;
            par[2] = r_lo;
        }
        __syncthreads();
        const uint32_t r_hi = par[1], r_lo = par[2];
        const int w = tid >> 6;
        if (w == 0 && r_hi) {
            uint32_t d, ab;
            wave_pick<kNB0>(hA, r_hi, d, ab);
            if (lane_id() == 0) {
                par[3] = d;
                par[4] = r_hi - ab;
            }
        }
        if (w == 1 && r_lo) {
            uint32_t d, ab;
            wave_pick<kNB0>(hA, r_lo, d, ab);
            if (lane_id() == 0) {
                par[5] = d;
                par[6] = r_lo - ab;
            }
        }
        __syncthreads();
        const uint32_t dh = r_hi ? par[3] : kNoKey, dl = r_lo ? par[5] : kNoKey;
        for (uint32_t i = tid; i < nkeys; i += kSampleThreads) {
            const uint32_t key = keys[i];
            if (key == kNoKey) continue;
            const uint32_t d0 = key >> kD0Shift, d1 = (key >> kD1Shift) & (kNB1 - 1);
            if (d0 == dh) atomicAdd(&hB[0][d1], 1u);
            if (d0 == dl) atomicAdd(&hB[1][d1], 1u);
        }
        __syncthreads();
        if (w == 0 && r_hi) {
            uint32_t d, ab;
            wave_pick<kNB1>(hB[0], par[4], d, ab);
            if (lane_id() == 0) par[4] = d;
        }
        if (w == 1 && r_lo) {
            uint32_t d, ab;
            wave_pick<kNB1>(hB[1], par[6], d, ab);
            if (lane_id() == 0) par[6] = d;
        }
        __syncthreads();
        hi = r_hi ? ((((dh << 11) | par[4]) + 1u) << kD1Shift) : kNoKey;
        lo = r_lo ? (((dl << 11) | par[6]) << kD1Shift) : 0u;
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
        a.seg_done[s] = 0;
    }
}

// ---------------------------------------------------------------------------
// k_dense: the one pass over grad and residual
// ---------------------------------------------------------------------------

template <bool BASE>
__global__ __launch_bounds__(kBlock) void k_dense(DenseArgs a) {
    __shared__ uint32_t lh[kWavesPerBlock][kNB0];
    const int w = threadIdx.x >> 6, lane = lane_id();
    const uint32_t c = blockIdx.x * kWavesPerBlock + w;
    uint32_t* hw = lh[w];
    for (int i = lane; i < kNB0; i += kWave) hw[i] = 0;
    wave_lds_sync();
    if (c >= a.num_chunks) return;

    const uint32_t start = a.chunk_start[c], len = a.chunk_len[c], end = start + len;
    const uint32_t s = a.per_tensor ? a.chunk_tensor[c] : 0u;
    const uint32_t lo = a.seg[s].lo, hi = a.seg[s].hi;
    uint2* out = a.slots + start;
    const f4* g4 = reinterpret_cast<const f4*>(a.grad);
    const f4* b4 = reinterpret_cast<const f4*>(BASE ? a.base : a.grad);
    f4* r4 = reinterpret_cast<f4*>(a.res);
    const uint32_t vb = start >> 2, ve = (end + 3) >> 2;
    uint32_t nc = 0, nh = 0;

    for (uint32_t v0 = vb; v0 < ve; v0 += 4 * kWave) {
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
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const uint32_t v = v0 + u * kWave + lane;
            const uint32_t e0 = 4 * v;
            const bool inside = v < ve;
            const bool full = inside && e0 >= start && e0 + 4 <= end;
            float acc[4];
            uint32_t key[4];
            bool cand[4], zero[4];
            f4 ov;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t e = e0 + q;
                const bool valid = inside && e >= start && e < end;
                acc[q] = acc_of<BASE>(g[u][q], b[u][q], r[u][q]);
                key[q] = key_of(acc[q]);
                cand[q] = valid && key[q] >= lo;
                zero[q] = valid && key[q] >= hi;
                ov[q] = zero[q] ? 0.0f : acc[q];
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
            uint32_t pos = nc + lanes_below(m0) + lanes_below(m1) + lanes_below(m2) + lanes_below(m3);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                if (cand[q]) {
                    out[pos] = make_uint2(e0 + q, __float_as_uint(acc[q]));
                    atomicAdd(&hw[key[q] >> kD0Shift], 1u);
                    ++pos;
                }
            }
            nc += popc64(m0) + popc64(m1) + popc64(m2) + popc64(m3);
            nh += popc64(ballot(zero[0])) + popc64(ballot(zero[1])) + popc64(ballot(zero[2])) + popc64(ballot(zero[3]));
        }
    }
    wave_lds_sync();
    uint32_t* hg = a.hist + (size_t)s * kHistWords + kHistH0;
    for (int i = lane; i < kNB0; i += kWave) {
        const uint32_t x = hw[i];
        if (x) atomicAdd(&hg[i], x);
    }
    if (lane == 0) {
        a.cnt_lo[c] = nc;
        a.cnt_hi[c] = nh;
        atomicAdd(&a.seg[s].clo, nc);
        atomicAdd(&a.seg[s].chi, nh);
    }
}

// ---------------------------------------------------------------------------
// fallback for segments whose bracket missed
// ---------------------------------------------------------------------------

__device__ __forceinline__ bool seg_missed(const CandArgs& a, uint32_t s, uint32_t& k) {
    k = keep_of(a.seg_off[s + 1] - a.seg_off[s], a.keep_ppm);
    return k > 0 && a.seg[s].clo < k;
}

__global__ __launch_bounds__(kBlock) void k_fb_restore(CandArgs a) {
    const int w = threadIdx.x >> 6, lane = lane_id();
    const uint32_t c = blockIdx.x * kWavesPerBlock + w;
    if (c >= a.num_chunks) return;
    const uint32_t s = a.per_tensor ? a.chunk_tensor[c] : 0u;
    uint32_t k;
    if (!seg_missed(a, s, k)) return;
    const uint32_t hi = a.seg[s].hi, start = a.chunk_start[c], cnt = a.cnt_lo[c];
    for (uint32_t i = lane; i < cnt; i += kWave) {
        const uint2 e = a.slots[start + i];
        if ((e.y & 0x7FFFFFFFu) >= hi) a.res[e.x] = __uint_as_float(e.y);
    }
}

__global__ __launch_bounds__(kBlock) void k_fb_emit(CandArgs a) {
    __shared__ uint32_t lh[kWavesPerBlock][kNB0];
    const int w = threadIdx.x >> 6, lane = lane_id();
    const uint32_t c = blockIdx.x * kWavesPerBlock + w;
    if (c >= a.num_chunks) return;
    const uint32_t s = a.per_tensor ? a.chunk_tensor[c] : 0u;
    uint32_t k;
    if (!seg_missed(a, s, k)) return;
    uint32_t* hw = lh[w];
    for (int i = lane; i < kNB0; i += kWave) hw[i] = 0;
    wave_lds_sync();
    const uint32_t start = a.chunk_start[c], len = a.chunk_len[c];
    for (uint32_t i = lane; i < len; i += kWave) {
        const uint32_t bitsv = __float_as_uint(a.res[start + i]);
        a.slots[start + i] = make_uint2(start + i, bitsv);
        atomicAdd(&hw[(bitsv & 0x7FFFFFFFu) >> kD0Shift], 1u);
    }
    wave_lds_sync();
    uint32_t* hg = a.hist + (size_t)s * kHistWords + kHistH0Fb;
    for (int i = lane; i < kNB0; i += kWave) {
        const uint32_t x = hw[i];
        if (x) atomicAdd(&hg[i], x);
    }
}

// ---------------------------------------------------------------------------
// candidate passes: one wave per group of chunks
// ---------------------------------------------------------------------------

struct GroupView {
    uint32_t g, s, t, c0, nch, total, k, first_group;
    bool miss;
};

// Loads the group's per-chunk candidate counts into LDS (pre: exclusive
// prefix, nch + 1 entries; base: slot offset of each chunk).
__device__ bool group_setup(const CandArgs& a, uint32_t g, uint32_t* pre, uint32_t* base, GroupView& v) {
    const int lane = lane_id();
    if (g >= a.num_groups) return false;
    v.g = g;
    v.c0 = a.group_chunk0[g];
    v.nch = a.group_chunk0[g + 1] - v.c0;
    v.t = a.group_tensor[g];
    v.s = a.per_tensor ? v.t : 0u;
    v.first_group = a.per_tensor ? a.tensor_group0[v.t] : 0u;
    v.miss = seg_missed(a, v.s, v.k);
    uint32_t cnt = 0;
    if (lane < (int)v.nch) {
        const uint32_t c = v.c0 + lane;
        cnt = v.miss ? a.chunk_len[c] : a.cnt_lo[c];
        base[lane] = a.chunk_start[c];
    }
    const uint32_t incl = wave_incl_scan(cnt);
    if (lane < (int)v.nch) pre[lane + 1] = incl;
    if (lane == 0) pre[0] = 0;
    v.total = __shfl(incl, (int)v.nch - 1, kWave);
    wave_lds_sync();
    return true;
}

// The e-th candidate of the group (0 <= e < total), in ascending index order.
__device__ __forceinline__ uint2 group_entry(const CandArgs& a, const GroupView& v, const uint32_t* pre,
                                             const uint32_t* base, uint32_t e) {
    uint32_t lo = 0, hi = v.nch;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (pre[mid] <= e) lo = mid;
        else hi = mid;
    }
    return a.slots[base[lo] + (e - pre[lo])];
}

__device__ __forceinline__ const uint32_t* seg_hist(const CandArgs& a, uint32_t s, int which) {
    return a.hist + (size_t)s * kHistWords + which;
}

__global__ __launch_bounds__(kBlock) void k_radix1(CandArgs a) {
    __shared__ uint32_t lh[kWavesPerBlock][kNB1];
    __shared__ uint32_t pre[kWavesPerBlock][kWave + 1], base[kWavesPerBlock][kWave];
    const int w = threadIdx.x >> 6, lane = lane_id();
    GroupView v;
    if (!group_setup(a, blockIdx.x * kWavesPerBlock + w, pre[w], base[w], v) || v.k == 0) return;
    uint32_t d0, ab;
    wave_pick<kNB0>(seg_hist(a, v.s, v.miss ? kHistH0Fb : kHistH0), v.k, d0, ab);
    if (v.g == v.first_group && lane == 0) {
        a.seg[v.s].d0 = d0;
        a.seg[v.s].r1 = v.k - ab;
    }
    uint32_t* hw = lh[w];
    for (int i = lane; i < kNB1; i += kWave) hw[i] = 0;
    wave_lds_sync();
    for (uint32_t e = lane; e < v.total; e += kWave) {
        const uint32_t key = group_entry(a, v, pre[w], base[w], e).y & 0x7FFFFFFFu;
        if ((key >> kD0Shift) == d0) atomicAdd(&hw[(key >> kD1Shift) & (kNB1 - 1)], 1u);
    }
    wave_lds_sync();
    uint32_t* hg = a.hist + (size_t)v.s * kHistWords + kHistH1;
    for (int i = lane; i < kNB1; i += kWave) {
        const uint32_t x = hw[i];
        if (x) atomicAdd(&hg[i], x);
    }
}

__global__ __launch_bounds__(kBlock) void k_radix2(CandArgs a) {
    __shared__ uint32_t lh[kWavesPerBlock][kNB2];
    __shared__ uint32_t pre[kWavesPerBlock][kWave + 1], base[kWavesPerBlock][kWave];
    const int w = threadIdx.x >> 6, lane = lane_id();
    GroupView v;
    if (!group_setup(a, blockIdx.x * kWavesPerBlock + w, pre[w], base[w], v) || v.k == 0) return;
    const uint32_t d0 = a.seg[v.s].d0, r1 = a.seg[v.s].r1;
    uint32_t d1, ab;
    wave_pick<kNB1>(seg_hist(a, v.s, kHistH1), r1, d1, ab);
    const uint32_t p21 = (d0 << 11) | d1;
    if (v.g == v.first_group && lane == 0) {
        a.seg[v.s].p21 = p21;
        a.seg[v.s].r2 = r1 - ab;
    }
    uint32_t* hw = lh[w];
    for (int i = lane; i < kNB2; i += kWave) hw[i] = 0;
    wave_lds_sync();
    for (uint32_t e = lane; e < v.total; e += kWave) {
        const uint32_t key = group_entry(a, v, pre[w], base[w], e).y & 0x7FFFFFFFu;
        if ((key >> kD1Shift) == p21) atomicAdd(&hw[key & (kNB2 - 1)], 1u);
    }
    wave_lds_sync();
    uint32_t* hg = a.hist + (size_t)v.s * kHistWords + kHistH2;
    for (int i = lane; i < kNB2; i += kWave) {
        const uint32_t x = hw[i];
        if (x) atomicAdd(&hg[i], x);
    }
}

__global__ __launch_bounds__(kBlock) void k_count(CandArgs a) {
    __shared__ uint32_t pre[kWavesPerBlock][kWave + 1], base[kWavesPerBlock][kWave];
    const int w = threadIdx.x >> 6, lane = lane_id();
    GroupView v;
    if (!group_setup(a, blockIdx.x * kWavesPerBlock + w, pre[w], base[w], v)) return;
    uint32_t thr = kNoKey, need = 0;
    if (v.k > 0) {
        const uint32_t p21 = a.seg[v.s].p21, r2 = a.seg[v.s].r2;
        uint32_t d2, ab;
        wave_pick<kNB2>(seg_hist(a, v.s, kHistH2), r2, d2, ab);
        thr = (p21 << kD1Shift) | d2;
        need = r2 - ab;
    }
    if (v.g == v.first_group && lane == 0) {
        a.seg[v.s].thr = thr;
        a.seg[v.s].need = need;
    }
    uint32_t gt = 0, eq = 0;
    if (v.k > 0) {
        for (uint32_t e = lane; e < v.total; e += kWave) {
            const uint32_t key = group_entry(a, v, pre[w], base[w], e).y & 0x7FFFFFFFu;
            gt += key > thr;
            eq += key == thr;
        }
    }
    gt = wave_sum(gt);
    eq = wave_sum(eq);
    if (lane == 0) {
        a.grp_gt[v.g] = gt;
        a.grp_eq[v.g] = eq;
    }
}

template <bool QUANT>
__global__ __launch_bounds__(kBlock) void k_emit(CandArgs a, EmitArgs o) {
    __shared__ uint32_t pre[kWavesPerBlock][kWave + 1], base[kWavesPerBlock][kWave];
    const int w = threadIdx.x >> 6, lane = lane_id();
    GroupView v;
    if (!group_setup(a, blockIdx.x * kWavesPerBlock + w, pre[w], base[w], v)) return;
    const uint32_t thr = a.seg[v.s].thr, need = a.seg[v.s].need;
    const uint32_t hi = v.miss ? kNoKey : a.seg[v.s].hi;
    // Counts of earlier groups of the same segment.
    uint32_t bg = 0, be = 0;
    for (uint32_t q = v.first_group + lane; q < v.g; q += kWave) {
        bg += a.grp_gt[q];
        be += a.grp_eq[q];
    }
    bg = wave_sum(bg);
    be = wave_sum(be);
    const uint64_t ob = a.out_base[v.s];
    uint32_t kept_n = 0;
    double sp = 0.0, sn = 0.0;
    uint32_t np = 0, nn = 0;
    for (uint32_t e0 = 0; e0 < v.total; e0 += kWave) {
        const uint32_t e = e0 + lane;
        const bool valid = e < v.total;
        uint2 ent = make_uint2(0u, 0u);
        if (valid) ent = group_entry(a, v, pre[w], base[w], e);
        const uint32_t key = ent.y & 0x7FFFFFFFu;
        const bool isgt = valid && key > thr;
        const bool iseq = valid && key == thr;
        const uint64_t mg = ballot(isgt), me = ballot(iseq);
        const uint32_t G = bg + lanes_below(mg), E = be + lanes_below(me);
        const bool kept = isgt || (iseq && E < need);
        if (kept) {
            const uint64_t pos = ob + G + (E < need ? E : need);
            if (pos < o.capacity) {
                o.idx[pos] = ent.x;
                o.val[pos] = __uint_as_float(ent.y);
            }
            if (QUANT) {
                const float x = __uint_as_float(ent.y);
                if (x < 0.0f) {
                    sn += (double)x;
                    ++nn;
                } else {
                    sp += (double)x;
                    ++np;
                }
            }
        }
        const bool wz = valid && key >= hi;
        if (kept && !wz) a.res[ent.x] = 0.0f;
        if (!kept && wz) a.res[ent.x] = __uint_as_float(ent.y);
        kept_n += popc64(ballot(kept));
        bg += popc64(mg);
        be += popc64(me);
    }
    if (lane == 0 && kept_n) atomicAdd(&o.tensor_counts[v.t], kept_n);
    if (QUANT) {
        sp = wave_sum(sp);
        sn = wave_sum(sn);
        np = wave_sum(np);
        nn = wave_sum(nn);
        if (lane == 0) {
            a.grp_q[4 * (size_t)v.g + 0] = sp;
            a.grp_q[4 * (size_t)v.g + 1] = sn;
            a.grp_q[4 * (size_t)v.g + 2] = (double)np;
            a.grp_q[4 * (size_t)v.g + 3] = (double)nn;
        }
    }
}

// ---------------------------------------------------------------------------
// sign-mean quantisation (Section 5.4): per tensor centres, then sign bits
// and the quantisation error fed back into the residual
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kBlock) void k_means(QuantArgs q) {
    const int w = threadIdx.x >> 6, lane = lane_id();
    const uint32_t t = blockIdx.x * kWavesPerBlock + w;
    if (t >= q.T) return;
    const uint32_t g0 = q.tensor_group0[t], g1 = q.tensor_group0[t + 1];
    double sp = 0.0, sn = 0.0, np = 0.0, nn = 0.0;
    for (uint32_t g = g0 + lane; g < g1; g += kWave) {
        sp += q.grp_q[4 * (size_t)g + 0];
        sn += q.grp_q[4 * (size_t)g + 1];
        np += q.grp_q[4 * (size_t)g + 2];
        nn += q.grp_q[4 * (size_t)g + 3];
    }
    sp = wave_sum(sp);
    sn = wave_sum(sn);
    np = wave_sum(np);
    nn = wave_sum(nn);
    uint32_t before = 0;
    for (uint32_t u = lane; u < t; u += kWave) before += q.tensor_counts[u];
    before = wave_sum(before);
    if (lane == 0) {
        q.means[2 * t + 0] = np > 0.0 ? (float)(sp / np) : 0.0f;
        q.means[2 * t + 1] = nn > 0.0 ? (float)(sn / nn) : 0.0f;
        q.qbase[t] = before;
        if (t + 1 == q.T) q.qbase[q.T] = before + q.tensor_counts[t];
    }
}

__global__ __launch_bounds__(kBlock) void k_quant(QuantArgs q) {
    const uint64_t j = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
    const bool valid = j < q.k_total;
    bool neg = false;
    if (valid) {
        // tensor of output slot j: the last t with qbase[t] <= j
        uint32_t lo = 0, hi = q.T;
        while (hi - lo > 1) {
            const uint32_t mid = (lo + hi) >> 1;
            if (q.qbase[mid] <= j) lo = mid;
            else hi = mid;
        }
        const float x = q.val[j];
        neg = x < 0.0f;
        const float centre = neg ? q.means[2 * lo + 1] : q.means[2 * lo + 0];
        const uint32_t i = q.idx[j];
        if (i < q.N) q.res[i] = x - centre;
    }
    const uint64_t m = ballot(valid && neg);
    const uint64_t jw = j - lane_id();  // first slot of this wave, a multiple of 64
    const uint64_t words = (q.k_total + 31) / 32;
    if (lane_id() == 0 && jw / 32 < words) q.sign_bits[jw / 32] = (uint32_t)m;
    if (lane_id() == 1 && jw / 32 + 1 < words) q.sign_bits[jw / 32 + 1] = (uint32_t)(m >> 32);
}

// ---------------------------------------------------------------------------
// server-side sparse apply (Section 3)
// ---------------------------------------------------------------------------

// First position in list[lo, hi) whose value is >= x.
__device__ __forceinline__ uint32_t lower_bound_u32(const uint32_t* list, uint32_t lo, uint32_t hi, uint32_t x) {
    while (lo < hi) {
        const uint32_t mid = lo + ((hi - lo) >> 1);
        if (list[mid] < x) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// First position in list[lo, hi) whose value is > x.
__device__ __forceinline__ uint32_t upper_bound_u32(const uint32_t* list, uint32_t lo, uint32_t hi, uint32_t x) {
    while (lo < hi) {
        const uint32_t mid = lo + ((hi - lo) >> 1);
        if (list[mid] <= x) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

constexpr int kApplyWindow = 256;

__global__ __launch_bounds__(kBlock) void k_apply(ApplyArgs a) {
    __shared__ uint32_t win[kWavesPerBlock][kApplyWindow];
    const int w = threadIdx.x >> 6, lane = lane_id();
    const uint32_t c = blockIdx.y;
    const uint32_t nnz = a.nnz[c];
    const uint32_t j0 = (blockIdx.x * kWavesPerBlock + w) * kWave;
    if (j0 >= nnz) return;
    const uint32_t j = j0 + lane;
    const bool have = j < nnz;
    const uint32_t i = have ? a.idx[c][j] : 0u;
    const bool valid = have && i < a.n;
    // index range covered by this wave (lists are ascending)
    const uint32_t last_j = (j0 + kWave <= nnz ? j0 + kWave : nnz) - 1;
    const uint32_t i_first = a.idx[c][j0], i_last = a.idx[c][last_j];
    float s = 0.0f;
    bool owner = true;
    for (uint32_t cc = 0; cc < a.C; ++cc) {
        if (cc == c) {
            s = s + (valid ? a.val[c][j] : 0.0f);
            continue;
        }
        const uint32_t* list = a.idx[cc];
        const uint32_t m = a.nnz[cc];
        uint32_t wlo = 0, whi = 0;
        if (lane == 0) wlo = lower_bound_u32(list, 0, m, i_first);
        if (lane == 1) whi = upper_bound_u32(list, 0, m, i_last);
        wlo = __shfl(wlo, 0, kWave);
        whi = __shfl(whi, 1, kWave);
        const uint32_t wn = whi - wlo;
        uint32_t pos = 0;
        bool found = false;
        if (wn <= (uint32_t)kApplyWindow) {
            for (uint32_t q = lane; q < wn; q += kWave) win[w][q] = list[wlo + q];
            wave_lds_sync();
            if (valid) {
                uint32_t lo = 0, hi = wn;
                while (lo < hi) {
                    const uint32_t mid = (lo + hi) >> 1;
                    if (win[w][mid] < i) lo = mid + 1;
                    else hi = mid;
                }
                found = lo < wn && win[w][lo] == i;
                pos = wlo + lo;
            }
            wave_lds_sync();
        } else if (valid) {
            pos = lower_bound_u32(list, wlo, whi, i);
            found = pos < whi && list[pos] == i;
        }
        if (found) {
            if (cc < c) owner = false;
            else s = s + a.val[cc][pos];
        }
    }
    if (valid && owner) {
        const float step = a.lr * s;
        a.p[i] = a.p[i] - step;
    }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

static inline uint32_t blocks_for_waves(uint32_t waves) { return (waves + kWavesPerBlock - 1) / kWavesPerBlock; }

hipError_t launch_sample(const SampleArgs& a, bool has_base, hipStream_t st) {
    dim3 grid((kMaxUnits + kSampleThreads - 1) / kSampleThreads, a.S);
    if (has_base) hipLaunchKernelGGL(k_sample<true>, grid, dim3(kSampleThreads), 0, st, a);
    else hipLaunchKernelGGL(k_sample<false>, grid, dim3(kSampleThreads), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_dense(const DenseArgs& a, bool has_base, hipStream_t st) {
    if (a.num_chunks == 0) return hipSuccess;
    dim3 grid(blocks_for_waves(a.num_chunks));
    if (has_base) hipLaunchKernelGGL(k_dense<true>, grid, dim3(kBlock), 0, st, a);
    else hipLaunchKernelGGL(k_dense<false>, grid, dim3(kBlock), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_candidates(const CandArgs& a, const EmitArgs& o, bool quant, hipStream_t st) {
    if (a.num_chunks == 0) return hipSuccess;
    const dim3 gc(blocks_for_waves(a.num_chunks)), gg(blocks_for_waves(a.num_groups)), b(kBlock);
    hipLaunchKernelGGL(k_fb_restore, gc, b, 0, st, a);
    hipLaunchKernelGGL(k_fb_emit, gc, b, 0, st, a);
    hipLaunchKernelGGL(k_radix1, gg, b, 0, st, a);
    hipLaunchKernelGGL(k_radix2, gg, b, 0, st, a);
    hipLaunchKernelGGL(k_count, gg, b, 0, st, a);
    if (quant) hipLaunchKernelGGL(k_emit<true>, gg, b, 0, st, a, o);
    else hipLaunchKernelGGL(k_emit<false>, gg, b, 0, st, a, o);
    return hipGetLastError();
}

hipError_t launch_quant(const QuantArgs& q, hipStream_t st) {
    hipLaunchKernelGGL(k_means, dim3(blocks_for_waves(q.T)), dim3(kBlock), 0, st, q);
    if (q.k_total > 0) {
        const uint64_t blocks = (q.k_total + kBlock - 1) / kBlock;
        hipLaunchKernelGGL(k_quant, dim3((uint32_t)blocks), dim3(kBlock), 0, st, q);
    }
    return hipGetLastError();
}

hipError_t launch_apply(const ApplyArgs& a, uint32_t max_nnz, hipStream_t st) {
    if (a.C == 0 || max_nnz == 0) return hipSuccess;
    dim3 grid((max_nnz + kBlock - 1) / kBlock, a.C);
    hipLaunchKernelGGL(k_apply, grid, dim3(kBlock), 0, st, a);
    return hipGetLastError();
}

}  // namespace gd
