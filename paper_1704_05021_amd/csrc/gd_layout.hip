// Candidate layout after the dense pass (gfx950, wave64).
//
//   k_scan   : scan blocks of 1024 units each scan their units' candidate
//              counts; the last block to finish scans the block totals and
//              derives, per threshold segment, the candidate total and
//              whether the bracket missed (fewer than k candidates), and per
//              tensor the first compact candidate and the first tile (tiles
//              of kTile candidates never cross a tensor).  A tensor of a
//              missed segment takes every element as a candidate, read
//              straight from the restored residual.
//   k_layout : per unit, the candidate offset in dense-pass order, the tiles
//              whose first candidate it holds, and (missed segments only)
//              the residual restored to acc where the dense pass wrote +0.

#include "gd_kernels.h"

namespace gd {

// raw(u): candidates of units [0, u) in dense-pass order.
__device__ __forceinline__ uint32_t raw_off(const CandArgs& a, const uint32_t* boff, uint32_t total, uint32_t u) {
    return u < a.num_chunks ? a.loc[u] + boff[u / kScanUnits] : total;
}

constexpr uint32_t kMaxScanBlocks = 4096;  // 2^32 elements / 1024 per unit / 1024 units per block

__global__ __launch_bounds__(kScanThreads) void k_scan(CandArgs a) {
    __shared__ uint32_t lds[kScanThreads / kWave + 1];
    __shared__ uint32_t boff[kMaxScanBlocks];
    __shared__ int s_last;
    __shared__ uint32_t any_miss;
    const int tid = threadIdx.x;
    const uint32_t C = a.num_chunks;

    // 1. local scan of this block's 1024 units (4 per thread)
    const uint32_t x = blockIdx.x * kScanUnits + 4 * tid;
    uint32_t c[4] = {0, 0, 0, 0};
    if (x + 4 <= C) {
        const uint4 v = *reinterpret_cast<const uint4*>(a.cnt_lo + x);
        c[0] = v.x;
        c[1] = v.y;
        c[2] = v.z;
        c[3] = v.w;
    } else {
        for (int q = 0; q < 4; ++q)
            if (x + q < C) c[q] = a.cnt_lo[x + q];
    }
    uint32_t total;
    const uint32_t excl = block_excl_scan<kScanThreads>(c[0] + c[1] + c[2] + c[3], lds, &total);
    const uint32_t o[4] = {excl, excl + c[0], excl + c[0] + c[1], excl + c[0] + c[1] + c[2]};
    if (x + 4 <= C) {
        *reinterpret_cast<uint4*>(a.loc + x) = make_uint4(o[0], o[1], o[2], o[3]);
    } else {
        for (int q = 0; q < 4; ++q)
            if (x + q < C) a.loc[x + q] = o[q];
    }
    if (tid == 0) a.btot[blockIdx.x] = total;

    // 2. the last block to finish lays out segments and tensors
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = atomicAdd(a.scan_done, 1u) == gridDim.x - 1;
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    if (tid == 0) {
        any_miss = 0;
        *a.scan_done = 0;
    }
    uint32_t carry = 0;
    for (uint32_t b0 = 0; b0 < gridDim.x; b0 += kScanThreads) {
        const uint32_t b = b0 + tid;
        const uint32_t t = b < gridDim.x ? a.btot[b] : 0u;
        uint32_t tot;
        const uint32_t e = block_excl_scan<kScanThreads>(t, lds, &tot);
        if (b < gridDim.x) {
            boff[b] = carry + e;
            a.boff[b] = carry + e;
        }
        carry += tot;
    }
    const uint32_t grand = carry;
    __syncthreads();
    const uint32_t S = a.per_tensor ? a.T : 1u;
    for (uint32_t s = tid; s < S; s += kScanThreads) {
        const uint32_t n = a.seg_off[s + 1] - a.seg_off[s];
        const uint32_t k = keep_of(n, a.keep_ppm);
        const uint32_t c0 = a.per_tensor ? a.tensor_chunk0[s] : 0u;
        const uint32_t c1 = a.per_tensor ? a.tensor_chunk0[s + 1] : C;
        const uint32_t cnt = raw_off(a, boff, grand, c1) - raw_off(a, boff, grand, c0);
        const uint32_t miss = (k > 0 && cnt < k) ? 1u : 0u;
        a.seg[s].clo = cnt;
        a.seg[s].miss = miss;
        if (miss) atomicOr(&any_miss, 1u);
    }
    __threadfence_block();
    __syncthreads();
    uint32_t ccarry = 0, tcarry = 0;
    for (uint32_t b0 = 0; b0 < a.T; b0 += kScanThreads) {
        const uint32_t t = b0 + tid;
        uint32_t cc = 0, tiles = 0;
        if (t < a.T) {
            const uint32_t rb = raw_off(a, boff, grand, a.tensor_chunk0[t]);
            const uint32_t re = raw_off(a, boff, grand, a.tensor_chunk0[t + 1]);
            const uint32_t s = a.per_tensor ? t : 0u;
            cc = a.seg[s].miss ? a.tensor_off[t + 1] - a.tensor_off[t] : re - rb;
            tiles = (cc + kTile - 1) / kTile;
            a.raw_tbase[t] = rb;
        }
        uint32_t ctot, ttot;
        const uint32_t ce = block_excl_scan<kScanThreads>(cc, lds, &ctot);
        const uint32_t te = block_excl_scan<kScanThreads>(tiles, lds, &ttot);
        if (t < a.T) {
            a.ten_cbase[t] = ccarry + ce;
            a.tile_base[t] = tcarry + te;
        }
        ccarry += ctot;
        tcarry += ttot;
    }
    if (tid == 0) {
        a.raw_tbase[a.T] = grand;
        a.ten_cbase[a.T] = ccarry;
        a.tile_base[a.T] = tcarry;
        a.flags[0] = any_miss;
    }
}

__global__ __launch_bounds__(kBlock) void k_layout(CandArgs a) {
    const uint32_t u = blockIdx.x * kBlock + threadIdx.x;
    const bool have = u < a.num_chunks;
    uint32_t t = 0, s = 0, raw = 0, cnt = 0;
    bool miss = false;
    if (have) {
        raw = a.loc[u] + a.boff[u / kScanUnits];
        cnt = a.cnt_lo[u];
        a.cand_off[u] = raw;
        if (u + 1 == a.num_chunks) a.cand_off[u + 1] = raw + cnt;
        t = a.chunk_tensor[u];
        s = a.per_tensor ? t : 0u;
        miss = a.seg[s].miss != 0;
        if (!miss && cnt) {
            const uint32_t rt = a.raw_tbase[t], t0 = a.tile_base[t];
            for (uint32_t j = (raw - rt + kTile - 1) / kTile; rt + j * kTile < raw + cnt; ++j) a.tile_unit0[t0 + j] = u;
        }
    }
    // Missed segments: the dense pass wrote +0 where key >= hi; put acc back
    // from the unit's candidate list (one unit at a time, the whole wave).
    uint64_t todo = ballot(have && miss && cnt > 0);
    while (todo) {
        const int src = __ffsll((unsigned long long)todo) - 1;
        todo &= todo - 1;
        const uint32_t uu = __shfl(u, src, kWave), nn = __shfl(cnt, src, kWave), ss = __shfl(s, src, kWave);
        const uint32_t start = a.chunk_start[uu], hi = a.seg[ss].hi;
        for (uint32_t i = lane_id(); i < nn; i += kWave) {
            const uint2 e = a.slots[start + i];
            if ((e.y & 0x7FFFFFFFu) >= hi) a.res[e.x] = __uint_as_float(e.y);
        }
    }
}

hipError_t launch_layout(const CandArgs& a, hipStream_t st) {
    if (a.num_chunks == 0) return hipSuccess;
    const uint32_t sb = (a.num_chunks + kScanUnits - 1) / kScanUnits;
    hipLaunchKernelGGL(k_scan, dim3(sb), dim3(kScanThreads), 0, st, a);
    hipLaunchKernelGGL(k_layout, dim3((a.num_chunks + kBlock - 1) / kBlock), dim3(kBlock), 0, st, a);
    return hipGetLastError();
}

}  // namespace gd
