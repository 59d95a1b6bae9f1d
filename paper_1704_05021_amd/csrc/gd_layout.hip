// Candidate layout after the dense pass (gfx950, wave64).
//
//   k_scan   : scan blocks of 1024 units each scan their units' candidate
//              counts.
//   k_scan_final : one block scans the block totals and derives, per
//              threshold segment, the candidate total and
//              whether the bracket missed (fewer than k candidates, unless
//              the candidates are every nonzero key and nothing was zeroed
//              early: then the segment takes the zero mode; under a
//              sampled threshold, where every candidate is sent, the first
//              output slot instead), and per
//              tensor the first candidate in dense-pass order, the first
//              compact candidate and the first tile (tiles of kTile
//              candidates never cross a tensor).  A tensor of a missed
//              segment takes every element as a candidate, read straight
//              from the restored residual.
//   k_layout : per unit, the candidate offset in dense-pass order, the tiles
//              that start in it (their tensor and first unit), and, for
//              missed segments only, the residual restored to acc where the
//              dense pass wrote +0.

#include "gd_kernels.h"

namespace gd {

constexpr uint32_t kMaxScanBlocks = (uint32_t)((1ull << 32) / kUnitLen / kScanUnits);  // for 2^32 elements

// Candidates (dense-pass order) before element offset x, x a tensor start.
__device__ __forceinline__ uint32_t raw_start(const CandArgs& a, const uint32_t* boff, uint32_t grand, uint32_t t) {
    const uint32_t x = a.tensor_off[t];
    if (x >= a.N) return grand;
    const uint32_t u = x / kUnitLen;
    return a.loc[u] + boff[u / kScanUnits] + ((x % kUnitLen) ? a.split[t] : 0u);
}

__global__ __launch_bounds__(kScanThreads) void k_scan(CandArgs a) {
    __shared__ uint32_t lds[kScanThreads / kWave + 1];
    const int tid = threadIdx.x;
    const uint32_t C = a.num_units;

    // 1. local scan of this block's 1024 units (4 per thread)
    const uint32_t x = blockIdx.x * kScanUnits + 4 * tid;
    uint32_t c[4] = {0, 0, 0, 0};
    if (x + 4 <= C) {
        const uint4 v = *reinterpret_cast<const uint4*>(a.cnt + x);
        c[0] = v.x;
        c[1] = v.y;
        c[2] = v.z;
        c[3] = v.w;
    } else {
        for (int q = 0; q < 4; ++q)
            if (x + q < C) c[q] = a.cnt[x + q];
    }
    uint32_t total, ne_total;
    const uint32_t excl = block_excl_scan<kScanThreads>(c[0] + c[1] + c[2] + c[3], lds, &total);
    const uint32_t f[4] = {c[0] != 0, c[1] != 0, c[2] != 0, c[3] != 0};
    const uint32_t nexcl = block_excl_scan<kScanThreads>(f[0] + f[1] + f[2] + f[3], lds, &ne_total);
    const uint32_t o[4] = {excl, excl + c[0], excl + c[0] + c[1], excl + c[0] + c[1] + c[2]};
    const uint32_t n[4] = {nexcl, nexcl + f[0], nexcl + f[0] + f[1], nexcl + f[0] + f[1] + f[2]};
    if (x + 4 <= C) {
        *reinterpret_cast<uint4*>(a.loc + x) = make_uint4(o[0], o[1], o[2], o[3]);
        *reinterpret_cast<uint4*>(a.neloc + x) = make_uint4(n[0], n[1], n[2], n[3]);
    } else {
        for (int q = 0; q < 4; ++q)
            if (x + q < C) {
                a.loc[x + q] = o[q];
                a.neloc[x + q] = n[q];
            }
    }
    if (tid == 0) {
        a.btot[blockIdx.x] = total;
        a.betot[blockIdx.x] = ne_total;
    }
}

// One block: offsets of the scan blocks, then segments and tensors.
__global__ __launch_bounds__(kScanThreads) void k_scan_final(CandArgs a, uint32_t nblocks) {
    __shared__ uint32_t lds[kScanThreads / kWave + 1];
    __shared__ uint32_t boff[kMaxScanBlocks];
    __shared__ uint32_t any_miss, any_zero;
    const int tid = threadIdx.x;
    if (tid == 0) {
        any_miss = 0;
        any_zero = 0;
    }
    uint32_t carry = 0, necarry = 0;
    for (uint32_t b0 = 0; b0 < nblocks; b0 += kScanThreads) {
        const uint32_t b = b0 + tid;
        const uint32_t t = b < nblocks ? a.btot[b] : 0u;
        const uint32_t te = b < nblocks ? a.betot[b] : 0u;
        uint32_t tot, netot;
        const uint32_t e = block_excl_scan<kScanThreads>(t, lds, &tot);
        const uint32_t ne = block_excl_scan<kScanThreads>(te, lds, &netot);
        if (b < nblocks) {
            boff[b] = carry + e;
            a.boff[b] = carry + e;
            a.beoff[b] = necarry + ne;
        }
        carry += tot;
        necarry += netot;
    }
    const uint32_t grand = carry;
    if (tid == 0) {
        a.num_ne[0] = necarry;
        a.ne_off[necarry] = grand;
    }
    __syncthreads();
    // per tensor: first candidate in dense-pass order
    for (uint32_t t = tid; t <= a.T; t += kScanThreads) a.raw_tbase[t] = raw_start(a, boff, grand, t);
    __threadfence_block();
    __syncthreads();
    const uint32_t S = a.per_tensor ? a.T : 1u;
    for (uint32_t s = tid; s < S; s += kScanThreads) {
        const uint32_t n = a.seg_off[s + 1] - a.seg_off[s];
        const uint32_t k = keep_of(n, a.keep_ppm);
        const uint32_t cnt = a.per_tensor ? a.raw_tbase[s + 1] - a.raw_tbase[s] : grand;
        const uint32_t short_of_k = (!a.sampled && k > 0 && cnt < k) ? 1u : 0u;
        // Fewer than k nonzero keys, every one of them a candidate (lo = 1)
        // and none zeroed early (hi: no key, or a pull from the copy, whose
        // dense pass writes nothing): the threshold is key 0, and the segment
        // keeps every candidate plus its first k - cnt zeros by index (the
        // zero mode), so it needs no fallback.
        const uint32_t zero =
            (short_of_k && a.zfill && a.seg[s].lo == 1u && (a.seg[s].hi == kNoKey || a.res == nullptr)) ? 1u : 0u;
        const uint32_t miss = short_of_k && !zero;
        a.seg[s].clo = cnt;
        a.seg[s].miss = miss;
        a.seg[s].zero = zero;
        if (miss) atomicOr(&any_miss, 1u);
        if (zero) atomicOr(&any_zero, 1u);
    }
    __threadfence_block();
    __syncthreads();
    if (a.sampled) {
        // every candidate is sent: segment s starts after the candidates of
        // the segments before it
        uint64_t carry = 0;
        for (uint32_t b0 = 0; b0 < S; b0 += kScanThreads) {
            const uint32_t s = b0 + tid;
            const uint32_t c = s < S ? (a.per_tensor ? a.raw_tbase[s + 1] - a.raw_tbase[s] : grand) : 0u;
            uint32_t tot;
            const uint32_t e = block_excl_scan<kScanThreads>(c, lds, &tot);
            if (s < S) a.out_base[s] = carry + e;
            carry += tot;
        }
    }
    uint32_t ccarry = 0, tcarry = 0;
    for (uint32_t b0 = 0; b0 < a.T; b0 += kScanThreads) {
        const uint32_t t = b0 + tid;
        uint32_t cc = 0, tiles = 0;
        if (t < a.T) {
            const uint32_t s = a.per_tensor ? t : 0u;
            cc = a.seg[s].miss ? a.tensor_off[t + 1] - a.tensor_off[t] : a.raw_tbase[t + 1] - a.raw_tbase[t];
            tiles = (uint32_t)(((uint64_t)cc + kTile - 1) / kTile);
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
    // the group sums of the candidate passes start from zero
    for (uint32_t i = tid; i < tcarry / kGroupTiles + 1; i += kScanThreads) {
        a.grp_gt[i] = 0;
        a.grp_eq[i] = 0;
    }
    if (tid == 0) {
        a.ten_cbase[a.T] = ccarry;
        a.tile_base[a.T] = tcarry;
        a.flags[0] = any_miss;
        a.flags[1] = any_zero;
    }
}

// Tiles of tensor t whose first candidate lies in [p, q) (dense-pass order
// for a regular tensor, element order for a missed one): write each one's
// descriptor, so that the candidate passes find all they need about a tile
// in one load.  Words: tensor | miss << 31, the non-empty unit ne holding
// the tile's first candidate, its compact candidates [p0, p1), the
// segment's first tile, the segment's k, and the tensor's tiles [first, end),
// then the shift from a compact position to the tile's source position (its
// dense-pass position, or for a missed tensor its element index).
// t0, t1: the tensor's tiles; c0, c1: its compact candidates; miss: whether
// its segment missed; k: the segment's keep count.
__device__ __forceinline__ void mark_tiles(const CandArgs& a, uint32_t t, uint32_t base, uint32_t p, uint32_t q,
                                           uint32_t ne, uint32_t t0, uint32_t t1, uint32_t c0, uint32_t c1,
                                           bool missed, uint32_t k) {
    const uint32_t miss = missed ? 0x80000000u : 0u;
    // base is the tensor's first source position: its first element (missed)
    // or its first candidate in dense-pass order
    const uint32_t shift = base - c0;
    // (64-bit positions: a tile start past 2^32 must end the loop, not wrap)
    for (uint32_t j = p > base ? (p - base + kTile - 1) / kTile : 0u; (uint64_t)base + (uint64_t)j * kTile < q; ++j) {
        const uint32_t p0 = c0 + j * kTile, p1 = p0 + kTile < c1 ? p0 + kTile : c1;
        uint4* d = reinterpret_cast<uint4*>(a.tile_desc + (size_t)(t0 + j) * kTileDescWords);
        d[0] = make_uint4(t | miss, ne, p0, p1);
        d[1] = make_uint4(a.per_tensor ? t0 : 0u, k, t0, t1);
        d[2] = make_uint4(shift, 0u, 0u, 0u);
    }
}

// The per-unit part of the layout: the unit's offsets, its place in the list
// of non-empty units, the tiles starting in it, and for missed segments the
// residual restored.  TAB gives the per-tensor and per-segment tables: global
// memory written by k_scan_final, or the block's own copy in LDS.
template <typename TAB>
__device__ __forceinline__ void layout_unit(const CandArgs& a, const TAB& tab, uint32_t u, bool have, uint32_t raw,
                                            uint32_t cnt, uint32_t ne, uint32_t info) {
    bool restore = false;
    if (have) {
        if (cnt) {
            a.ne_unit[ne] = u;
            a.ne_off[ne] = raw;
        }
        const uint32_t ustart = u * kUnitLen, uend = a.N - ustart > kUnitLen ? ustart + kUnitLen : a.N;
        // every tensor overlapping the unit (one, unless it holds a boundary)
        for (uint32_t t = info & 0x7FFFFFFFu; t < a.T && a.tensor_off[t] < uend; ++t) {
            const uint32_t ta = a.tensor_off[t], tb = a.tensor_off[t + 1];
            if (tb <= ustart || tb == ta) continue;
            const uint32_t s = a.per_tensor ? t : 0u;
            const bool missed = tab.miss(s);
            const uint32_t k = keep_of(a.seg_off[s + 1] - a.seg_off[s], a.keep_ppm);
            const uint32_t t0 = tab.tile_base(t), t1 = tab.tile_base(t + 1);
            const uint32_t c0 = tab.ten_cbase(t), c1 = tab.ten_cbase(t + 1);
            if (missed) {
                // direct tiles start at element offsets ta + j * kTile
                const uint32_t lo_e = ta > ustart ? ta : ustart, hi_e = tb < uend ? tb : uend;
                mark_tiles(a, t, ta, lo_e, hi_e, ne, t0, t1, c0, c1, true, k);
                // nothing to restore after a pull from the copy, or where no key reached hi
                restore = restore || (cnt > 0 && a.res != nullptr && a.seg[s].hi != kNoKey);
            } else {
                const uint32_t rb = tab.raw_tbase(t), re = tab.raw_tbase(t + 1);
                const uint32_t p = raw > rb ? raw : rb, q = raw + cnt < re ? raw + cnt : re;
                if (p < q) mark_tiles(a, t, rb, p, q, ne, t0, t1, c0, c1, false, k);
            }
        }
    }
    // Missed segments: the dense pass wrote +0 where key >= hi; put acc back
    // from the unit's candidate list (one unit at a time, the whole wave).
    uint64_t todo = ballot(restore);
    while (todo) {
        const int src = __ffsll((unsigned long long)todo) - 1;
        todo &= todo - 1;
        const uint32_t uu = lane_value(u, src), nn = lane_value(cnt, src);
        for (uint32_t i = lane_id(); i < nn; i += kWave) {
            const uint2 e = a.slots[(size_t)uu * kUnitLen + i];
            uint32_t s = 0;
            if (a.per_tensor) {
                uint32_t lo = 0, hi = a.T;
                while (hi - lo > 1) {
                    const uint32_t mid = (lo + hi) >> 1;
                    if (a.tensor_off[mid] <= e.x) lo = mid;
                    else hi = mid;
                }
                s = lo;
            }
            if (tab.miss(s) && (e.y & 0x7FFFFFFFu) >= a.seg[s].hi) a.res[e.x] = __uint_as_float(e.y);
        }
    }
}

// Tables as k_scan_final wrote them.
struct GlobalTables {
    const CandArgs& a;
    __device__ bool miss(uint32_t s) const { return a.seg[s].miss != 0; }
    __device__ uint32_t tile_base(uint32_t t) const { return a.tile_base[t]; }
    __device__ uint32_t ten_cbase(uint32_t t) const { return a.ten_cbase[t]; }
    __device__ uint32_t raw_tbase(uint32_t t) const { return a.raw_tbase[t]; }
};

__global__ __launch_bounds__(kBlock) void k_layout(CandArgs a) {
    const uint32_t u = blockIdx.x * kBlock + threadIdx.x;
    const bool have = u < a.num_units;
    uint32_t raw = 0, cnt = 0, ne = 0, info = 0;
    if (have) {
        raw = a.loc[u] + a.boff[u / kScanUnits];
        cnt = a.cnt[u];
        ne = a.neloc[u] + a.beoff[u / kScanUnits];
        info = a.unit_info[u];
    }
    layout_unit(a, GlobalTables{a}, u, have, raw, cnt, ne, info);
}

// k_scan_final and k_layout in one kernel, for layouts of at most
// kFusedMaxT tensors and kFusedMaxG scan blocks.  Every block derives the
// block offsets, the per-tensor and per-segment tables from the scan blocks'
// totals (a few hundred words, read from the cache) into its LDS, and uses
// its own copy; block 0 also stores them for the passes that follow.  This
// costs each block a short prologue and saves a kernel boundary.
constexpr uint32_t kFusedMaxT = 256;
constexpr uint32_t kFusedMaxG = 1024;

struct LdsTables {
    const uint32_t* rtb;  // [T + 1]
    const uint32_t* tcb;  // [T + 1]
    const uint32_t* ttb;  // [T + 1]
    const uint32_t* smiss;  // [S]
    __device__ bool miss(uint32_t s) const { return smiss[s] != 0; }
    __device__ uint32_t tile_base(uint32_t t) const { return ttb[t]; }
    __device__ uint32_t ten_cbase(uint32_t t) const { return tcb[t]; }
    __device__ uint32_t raw_tbase(uint32_t t) const { return rtb[t]; }
};

__global__ __launch_bounds__(kBlock) void k_layout_fused(CandArgs a, uint32_t nblocks) {
    __shared__ uint32_t lds[kBlock / kWave + 1];
    __shared__ uint32_t goff[kFusedMaxG], geoff[kFusedMaxG];
    __shared__ uint32_t rtb[kFusedMaxT + 1], tcb[kFusedMaxT + 1], ttb[kFusedMaxT + 1], smiss[kFusedMaxT];
    __shared__ uint32_t any_miss, any_zero;
    const int tid = threadIdx.x;
    const bool lead = blockIdx.x == 0;  // stores the tables for the later passes
    const uint32_t S = a.per_tensor ? a.T : 1u;
    // 0. Every load that does not depend on the scan, issued first so that
    // they are in flight together: this thread's unit, the tensor starts (and
    // behind them the unit counts at those starts), the segment's bracket.
    const uint32_t u = blockIdx.x * kBlock + tid;
    const bool have = u < a.num_units;
    uint32_t uloc = 0, ucnt = 0, uneloc = 0, uinfo = 0;
    if (have) {
        uloc = load_early(a.loc + u);
        ucnt = load_early(a.cnt + u);
        uneloc = load_early(a.neloc + u);
        uinfo = load_early(a.unit_info + u);
    }
    uint32_t s_n = 0, s_lo = 0, s_hi = 0;
    if ((uint32_t)tid < S) {
        s_n = load_early(a.seg_off + tid + 1) - load_early(a.seg_off + tid);
        s_lo = load_early(&a.seg[tid].lo);
        s_hi = load_early(&a.seg[tid].hi);
    }
    // tensor t = tid + q * kBlock (T <= kFusedMaxT: t <= T needs q <= 1)
    static_assert(kFusedMaxT <= 2 * kBlock - 1, "two tensor starts per thread");
    uint32_t tx[2] = {0, 0}, tl[2] = {0, 0}, tsp[2] = {0, 0};
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const uint32_t t = tid + q * kBlock;
        if (t <= a.T) tx[q] = load_early(a.tensor_off + t);
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const uint32_t t = tid + q * kBlock;
        if (t <= a.T && tx[q] < a.N) {
            tl[q] = load_early(a.loc + tx[q] / kUnitLen);
            if (tx[q] % kUnitLen) tsp[q] = load_early(a.split + t);
        }
    }
    if (tid == 0) {
        any_miss = 0;
        any_zero = 0;
    }
    // 1. offsets of the scan blocks
    uint32_t carry = 0, necarry = 0;
    for (uint32_t b0 = 0; b0 < nblocks; b0 += kBlock) {
        const uint32_t b = b0 + tid;
        const uint32_t t = b < nblocks ? a.btot[b] : 0u;
        const uint32_t te = b < nblocks ? a.betot[b] : 0u;
        uint32_t tot, netot;
        const uint32_t e = block_excl_scan<kBlock>(t, lds, &tot);
        const uint32_t ne = block_excl_scan<kBlock>(te, lds, &netot);
        if (b < nblocks) {
            goff[b] = carry + e;
            geoff[b] = necarry + ne;
            if (lead) a.boff[b] = carry + e;
        }
        carry += tot;
        necarry += netot;
    }
    const uint32_t grand = carry;
    __syncthreads();
    // 2. first candidate of each tensor in dense-pass order
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const uint32_t t = tid + q * kBlock;
        if (t > a.T) continue;
        const uint32_t x = tx[q];
        const uint32_t r = x < a.N ? tl[q] + goff[x / kUnitLen / kScanUnits] + tsp[q] : grand;
        rtb[t] = r;
        if (lead) a.raw_tbase[t] = r;
    }
    __syncthreads();
    // 3. per segment: candidates, bracket miss, zero mode (as k_scan_final)
    if ((uint32_t)tid < S) {
        const uint32_t s = tid;
        const uint32_t k = keep_of(s_n, a.keep_ppm);
        const uint32_t cnt = a.per_tensor ? rtb[s + 1] - rtb[s] : grand;
        const uint32_t short_of_k = (!a.sampled && k > 0 && cnt < k) ? 1u : 0u;
        const uint32_t zero =
            (short_of_k && a.zfill && s_lo == 1u && (s_hi == kNoKey || a.res == nullptr)) ? 1u : 0u;
        const uint32_t miss = short_of_k && !zero;
        smiss[s] = miss;
        if (lead) {
            a.seg[s].clo = cnt;
            a.seg[s].miss = miss;
            a.seg[s].zero = zero;
        }
        if (miss) atomicOr(&any_miss, 1u);
        if (zero) atomicOr(&any_zero, 1u);
    }
    __syncthreads();
    // 4. per tensor: first compact candidate and first tile
    {
        const uint32_t t = tid;  // T <= kFusedMaxT <= kBlock: one round
        uint32_t cc = 0, tiles = 0;
        if (t < a.T) {
            const uint32_t s = a.per_tensor ? t : 0u;
            cc = smiss[s] ? a.tensor_off[t + 1] - tx[0] : rtb[t + 1] - rtb[t];
            tiles = (uint32_t)(((uint64_t)cc + kTile - 1) / kTile);
        }
        uint32_t ctot, ttot;
        const uint32_t ce = block_excl_scan<kBlock>(cc, lds, &ctot);
        const uint32_t te = block_excl_scan<kBlock>(tiles, lds, &ttot);
        if (t < a.T) {
            tcb[t] = ce;
            ttb[t] = te;
        }
        if (t == 0) {
            tcb[a.T] = ctot;
            ttb[a.T] = ttot;
        }
        if (lead) {
            if (t < a.T) {
                a.ten_cbase[t] = ce;
                a.tile_base[t] = te;
            }
            for (uint32_t i = tid; i < ttot / kGroupTiles + 1; i += kBlock) {
                a.grp_gt[i] = 0;
                a.grp_eq[i] = 0;
            }
            if (t == 0) {
                a.ten_cbase[a.T] = ctot;
                a.tile_base[a.T] = ttot;
                a.num_ne[0] = necarry;
                a.ne_off[necarry] = grand;
            }
        }
    }
    if (lead && a.sampled) {
        // every candidate is sent: segment s starts after the candidates of the segments before it
        const uint32_t s = tid;
        const uint32_t c = s < S ? (a.per_tensor ? rtb[s + 1] - rtb[s] : grand) : 0u;
        uint32_t tot;
        const uint32_t e = block_excl_scan<kBlock>(c, lds, &tot);
        if (s < S) a.out_base[s] = e;
    }
    __syncthreads();
    if (lead && tid == 0) {
        a.flags[0] = any_miss;
        a.flags[1] = any_zero;
    }
    // 5. this block's units
    uint32_t raw = 0, ne = 0;
    if (have) {
        raw = uloc + goff[u / kScanUnits];
        ne = uneloc + geoff[u / kScanUnits];
    }
    layout_unit(a, LdsTables{rtb, tcb, ttb, smiss}, u, have, raw, ucnt, ne, uinfo);
}

hipError_t launch_layout(const CandArgs& a, hipStream_t st) {
    if (a.num_units == 0) {
        // an empty layout still needs its (zero) candidate and tile bases:
        // the quantisation pass reads the tiles of every tensor
        hipLaunchKernelGGL(k_scan_final, dim3(1), dim3(kScanThreads), 0, st, a, 0u);
        return hipGetLastError();
    }
    const uint32_t sb = (a.num_units + kScanUnits - 1) / kScanUnits;
    hipLaunchKernelGGL(k_scan, dim3(sb), dim3(kScanThreads), 0, st, a);
    if (a.T <= kFusedMaxT && sb <= kFusedMaxG) {
        hipLaunchKernelGGL(k_layout_fused, dim3((a.num_units + kBlock - 1) / kBlock), dim3(kBlock), 0, st, a, sb);
    } else {
        hipLaunchKernelGGL(k_scan_final, dim3(1), dim3(kScanThreads), 0, st, a, sb);
        hipLaunchKernelGGL(k_layout, dim3((a.num_units + kBlock - 1) / kBlock), dim3(kBlock), 0, st, a);
    }
    return hipGetLastError();
}

}  // namespace gd
