// Exact selection and ordered emission from the candidates (gfx950, wave64).
//
// Candidates (every element with key >= lo, or every element of a segment
// whose bracket missed) are processed in tiles of kTile consecutive
// candidates of one tensor, one wave per tile, so the work is balanced
// however unevenly the candidates fall across the gradient.
//
//   k_gather  : compacts each tile's candidates from the per-unit slots
//               (or, for a missed segment, straight from the residual) into
//               one array in ascending flat index, with the digit-0
//               histogram.
//   k_radix1  : digit 0 of the k-th largest key from that histogram; the
//               digit-1 histogram of candidates that share it.
//   k_radix2  : digit 1; the digit-2 histogram.
//   k_count   : digit 2, i.e. the exact threshold key T and the number of
//               candidates equal to T that are kept (lowest index first);
//               per tile, the candidates above and equal to T.
//   k_emit    : kept (index, value) pairs in ascending index order, the
//               residual of every candidate whose fate differs from what the
//               dense pass assumed, kept counts per tensor (and per-tile sums
//               for quantisation).
//
// Together they realise the exact-k rule: keep the k largest |acc| of each
// segment, ties broken by lower flat index (Algorithm 1, Section 4).

#include "gd_kernels.h"

namespace gd {

struct TileView {
    uint32_t t, s, k, p0, p1, first_tile;
    bool miss;
};

__device__ __forceinline__ void tile_setup(const CandArgs& a, uint32_t tile, TileView& v) {
    uint32_t lo = 0, hi = a.T;  // last tensor whose first tile is <= tile
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (a.tile_base[mid] <= tile) lo = mid;
        else hi = mid;
    }
    v.t = lo;
    v.s = a.per_tensor ? lo : 0u;
    v.k = keep_of(a.seg_off[v.s + 1] - a.seg_off[v.s], a.keep_ppm);
    v.miss = a.seg[v.s].miss != 0;
    v.p0 = a.ten_cbase[lo] + (tile - a.tile_base[lo]) * kTile;
    const uint32_t end = a.ten_cbase[lo + 1];
    v.p1 = v.p0 + kTile < end ? v.p0 + kTile : end;
    v.first_tile = a.per_tensor ? a.tile_base[lo] : 0u;
}

// Last unit c in [lo, hi) with cand_off[c] <= p.
__device__ __forceinline__ uint32_t unit_of(const uint32_t* cand_off, uint32_t lo, uint32_t hi, uint32_t p) {
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (cand_off[mid] <= p) lo = mid;
        else hi = mid;
    }
    return lo;
}

__device__ __forceinline__ const uint32_t* seg_hist(const CandArgs& a, uint32_t s, int which) {
    return a.hist + (size_t)s * kHistWords + which;
}

__device__ __forceinline__ void flush_hist(uint32_t* hw, uint32_t* hg, int nb) {
    wave_lds_sync();
    for (int i = lane_id(); i < nb; i += kWave) {
        const uint32_t x = hw[i];
        if (x) {
            atomicAdd(&hg[i], x);
            hw[i] = 0;
        }
    }
    wave_lds_sync();
}

constexpr uint32_t kWin = 256;  // units held in a gather window
constexpr int kRows = 8;        // rows of 64 candidates whose loads are issued together
constexpr uint32_t kBatchLen = kRows * kWave;

__global__ __launch_bounds__(kBlock) void k_gather(CandArgs a) {
    __shared__ uint32_t lh[kWavesPerBlock][kNB0];
    __shared__ uint32_t woff[kWavesPerBlock][kWin + 1], wbase[kWavesPerBlock][kWin];
    const int w = threadIdx.x >> 6, lane = lane_id();
    uint32_t* hw = lh[w];
    uint32_t* wo = woff[w];
    uint32_t* wb = wbase[w];
    for (int i = lane; i < kNB0; i += kWave) hw[i] = 0;
    wave_lds_sync();
    const uint32_t ntiles = a.tile_base[a.T];
    for (uint32_t tile = blockIdx.x * kWavesPerBlock + w; tile < ntiles; tile += gridDim.x * kWavesPerBlock) {
        TileView v;
        tile_setup(a, tile, v);
        if (v.miss) {
            // every element of the tensor is a candidate; acc is in the residual
            const uint32_t e_base = a.tensor_off[v.t] - a.ten_cbase[v.t];
            for (uint32_t pb = v.p0; pb < v.p1; pb += kBatchLen) {
                float x[kRows];
#pragma unroll
                for (int r = 0; r < kRows; ++r) {
                    const uint32_t pl = pb + r * kWave + lane;
                    x[r] = pl < v.p1 ? a.res[e_base + pl] : 0.0f;
                }
#pragma unroll
                for (int r = 0; r < kRows; ++r) {
                    const uint32_t pl = pb + r * kWave + lane;
                    const bool active = pl < v.p1;
                    if (active) a.cand[pl] = make_uint2(e_base + pl, __float_as_uint(x[r]));
                    lds_hist_add(hw, (__float_as_uint(x[r]) & 0x7FFFFFFFu) >> kD0Shift, active);
                }
            }
            flush_hist(hw, a.hist + (size_t)v.s * kHistWords + kHistH0, kNB0);
            continue;
        }
        // compact position p <-> dense-pass offset p + shift
        const uint32_t shift = a.raw_tbase[v.t] - a.ten_cbase[v.t];
        const uint32_t uend = a.tensor_chunk0[v.t + 1];
        uint32_t u0 = a.tile_unit0[tile];
        uint32_t wend = 0;  // first dense-pass offset the window does not cover
        bool loaded = false;
        for (uint32_t pb = v.p0; pb < v.p1; pb += kBatchLen) {
            const uint32_t pe = pb + kBatchLen < v.p1 ? pb + kBatchLen : v.p1;
            if (!loaded || pe + shift > wend) {
                // (re)anchor the window of unit offsets at the unit holding pb
                wave_lds_sync();
                if (loaded) u0 = unit_of(a.cand_off, u0, uend, pb + shift);
                for (uint32_t j = lane; j <= kWin; j += kWave) {
                    const uint32_t u = u0 + j;
                    wo[j] = u <= a.num_chunks ? a.cand_off[u] : kNoKey;
                    if (j < kWin) wb[j] = u < a.num_chunks ? a.chunk_start[u] : 0u;
                }
                wave_lds_sync();
                wend = wo[kWin];
                loaded = true;
            }
            uint32_t src[kRows];
#pragma unroll
            for (int r = 0; r < kRows; ++r) {
                const uint32_t pl = pb + r * kWave + lane, rp = pl + shift;
                src[r] = 0;
                if (pl < v.p1) {
                    uint32_t base, off0;
                    if (rp < wend) {
                        uint32_t lo = 0, hi = kWin;
                        while (hi - lo > 1) {
                            const uint32_t mid = (lo + hi) >> 1;
                            if (wo[mid] <= rp) lo = mid;
                            else hi = mid;
                        }
                        base = wb[lo];
                        off0 = wo[lo];
                    } else {
                        const uint32_t u = unit_of(a.cand_off, u0, uend, rp);
                        base = a.chunk_start[u];
                        off0 = a.cand_off[u];
                    }
                    src[r] = base + (rp - off0);
                }
            }
            uint2 e[kRows];
#pragma unroll
            for (int r = 0; r < kRows; ++r) e[r] = pb + r * kWave + lane < v.p1 ? a.slots[src[r]] : make_uint2(0u, 0u);
#pragma unroll
            for (int r = 0; r < kRows; ++r) {
                const uint32_t pl = pb + r * kWave + lane;
                const bool active = pl < v.p1;
                if (active) a.cand[pl] = e[r];
                lds_hist_add(hw, (e[r].y & 0x7FFFFFFFu) >> kD0Shift, active);
            }
        }
        flush_hist(hw, a.hist + (size_t)v.s * kHistWords + kHistH0, kNB0);
    }
}

// Loads rows [pb, pb + kBatchLen) of the compact candidates (keys only).
__device__ __forceinline__ void load_keys(const CandArgs& a, uint32_t pb, uint32_t p1, uint32_t key[kRows]) {
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
        const uint32_t pl = pb + r * kWave + lane_id();
        key[r] = pl < p1 ? (a.cand[pl].y & 0x7FFFFFFFu) : 0u;
    }
}

__global__ __launch_bounds__(kBlock) void k_radix1(CandArgs a) {
    __shared__ uint32_t lh[kWavesPerBlock][kNB1];
    const int w = threadIdx.x >> 6, lane = lane_id();
    uint32_t* hw = lh[w];
    for (int i = lane; i < kNB1; i += kWave) hw[i] = 0;
    wave_lds_sync();
    const uint32_t ntiles = a.tile_base[a.T];
    uint32_t cached_s = kNoKey, d0 = 0, r1 = 0;
    for (uint32_t tile = blockIdx.x * kWavesPerBlock + w; tile < ntiles; tile += gridDim.x * kWavesPerBlock) {
        TileView v;
        tile_setup(a, tile, v);
        if (v.s != cached_s) {
            uint32_t ab;
            wave_pick<kNB0>(seg_hist(a, v.s, kHistH0), v.k, d0, ab);
            r1 = v.k - ab;
            cached_s = v.s;
        }
        if (tile == v.first_tile && lane == 0) {
            a.seg[v.s].d0 = d0;
            a.seg[v.s].r1 = r1;
        }
        for (uint32_t pb = v.p0; pb < v.p1; pb += kBatchLen) {
            uint32_t key[kRows];
            load_keys(a, pb, v.p1, key);
#pragma unroll
            for (int r = 0; r < kRows; ++r) {
                const bool active = pb + r * kWave + lane < v.p1;
                lds_hist_add(hw, (key[r] >> kD1Shift) & (kNB1 - 1), active && (key[r] >> kD0Shift) == d0);
            }
        }
        flush_hist(hw, a.hist + (size_t)v.s * kHistWords + kHistH1, kNB1);
    }
}

__global__ __launch_bounds__(kBlock) void k_radix2(CandArgs a) {
    __shared__ uint32_t lh[kWavesPerBlock][kNB2];
    const int w = threadIdx.x >> 6, lane = lane_id();
    uint32_t* hw = lh[w];
    for (int i = lane; i < kNB2; i += kWave) hw[i] = 0;
    wave_lds_sync();
    const uint32_t ntiles = a.tile_base[a.T];
    uint32_t cached_s = kNoKey, p21 = 0, r2 = 0;
    for (uint32_t tile = blockIdx.x * kWavesPerBlock + w; tile < ntiles; tile += gridDim.x * kWavesPerBlock) {
        TileView v;
        tile_setup(a, tile, v);
        if (v.s != cached_s) {
            const uint32_t d0 = a.seg[v.s].d0, r1 = a.seg[v.s].r1;
            uint32_t d1, ab;
            wave_pick<kNB1>(seg_hist(a, v.s, kHistH1), r1, d1, ab);
            p21 = (d0 << 11) | d1;
            r2 = r1 - ab;
            cached_s = v.s;
        }
        if (tile == v.first_tile && lane == 0) {
            a.seg[v.s].p21 = p21;
            a.seg[v.s].r2 = r2;
        }
        for (uint32_t pb = v.p0; pb < v.p1; pb += kBatchLen) {
            uint32_t key[kRows];
            load_keys(a, pb, v.p1, key);
#pragma unroll
            for (int r = 0; r < kRows; ++r) {
                const bool active = pb + r * kWave + lane < v.p1;
                lds_hist_add(hw, key[r] & (kNB2 - 1), active && (key[r] >> kD1Shift) == p21);
            }
        }
        flush_hist(hw, a.hist + (size_t)v.s * kHistWords + kHistH2, kNB2);
    }
}

__global__ __launch_bounds__(kBlock) void k_count(CandArgs a) {
    const int w = threadIdx.x >> 6, lane = lane_id();
    const uint32_t ntiles = a.tile_base[a.T];
    uint32_t cached_s = kNoKey, thr = kNoKey, need = 0;
    for (uint32_t tile = blockIdx.x * kWavesPerBlock + w; tile < ntiles; tile += gridDim.x * kWavesPerBlock) {
        TileView v;
        tile_setup(a, tile, v);
        if (v.s != cached_s) {
            const uint32_t p21 = a.seg[v.s].p21, r2 = a.seg[v.s].r2;
            uint32_t d2, ab;
            wave_pick<kNB2>(seg_hist(a, v.s, kHistH2), r2, d2, ab);
            thr = (p21 << kD1Shift) | d2;
            need = r2 - ab;
            cached_s = v.s;
        }
        if (tile == v.first_tile && lane == 0) {
            a.seg[v.s].thr = thr;
            a.seg[v.s].need = need;
        }
        uint32_t gt = 0, eq = 0;
        for (uint32_t pb = v.p0; pb < v.p1; pb += kBatchLen) {
            uint32_t key[kRows];
            load_keys(a, pb, v.p1, key);
#pragma unroll
            for (int r = 0; r < kRows; ++r) {
                const bool active = pb + r * kWave + lane < v.p1;
                gt += active && key[r] > thr;
                eq += active && key[r] == thr;
            }
        }
        gt = wave_sum(gt);
        eq = wave_sum(eq);
        if (lane == 0) {
            a.tile_gt[tile] = gt;
            a.tile_eq[tile] = eq;
        }
    }
}

template <bool QUANT>
__global__ __launch_bounds__(kBlock) void k_emit(CandArgs a, EmitArgs o) {
    const int w = threadIdx.x >> 6, lane = lane_id();
    const uint32_t ntiles = a.tile_base[a.T];
    for (uint32_t tile = blockIdx.x * kWavesPerBlock + w; tile < ntiles; tile += gridDim.x * kWavesPerBlock) {
        TileView v;
        tile_setup(a, tile, v);
        const uint32_t thr = a.seg[v.s].thr, need = a.seg[v.s].need;
        const uint32_t hi = v.miss ? kNoKey : a.seg[v.s].hi;
        // candidates above / equal to the threshold in earlier tiles of the segment
        uint32_t bg = 0, be = 0;
        for (uint32_t q0 = v.first_tile; q0 < tile; q0 += 4 * kWave) {
            uint32_t g4[4], e4[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const uint32_t q = q0 + j * kWave + lane;
                g4[j] = q < tile ? a.tile_gt[q] : 0u;
                e4[j] = q < tile ? a.tile_eq[q] : 0u;
            }
            bg += g4[0] + g4[1] + g4[2] + g4[3];
            be += e4[0] + e4[1] + e4[2] + e4[3];
        }
        bg = wave_sum(bg);
        be = wave_sum(be);
        const uint64_t ob = a.out_base[v.s];
        uint32_t kept_n = 0;
        double sp = 0.0, sn = 0.0;
        uint32_t np = 0, nn = 0;
        for (uint32_t pb = v.p0; pb < v.p1; pb += kBatchLen) {
            uint2 ent[kRows];
#pragma unroll
            for (int r = 0; r < kRows; ++r) {
                const uint32_t pl = pb + r * kWave + lane;
                ent[r] = pl < v.p1 ? a.cand[pl] : make_uint2(0u, 0u);
            }
#pragma unroll
            for (int r = 0; r < kRows; ++r) {
                const bool valid = pb + r * kWave + lane < v.p1;
                const uint32_t key = ent[r].y & 0x7FFFFFFFu;
                const bool isgt = valid && key > thr;
                const bool iseq = valid && key == thr;
                const uint64_t mg = ballot(isgt), me = ballot(iseq);
                const uint32_t G = bg + lanes_below(mg), E = be + lanes_below(me);
                const bool kept = isgt || (iseq && E < need);
                if (kept) {
                    const uint64_t pos = ob + G + (E < need ? E : need);
                    if (pos < o.capacity) {
                        o.idx[pos] = ent[r].x;
                        o.val[pos] = __uint_as_float(ent[r].y);
                    }
                    if (QUANT) {
                        const float x = __uint_as_float(ent[r].y);
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
                if (kept && !wz) a.res[ent[r].x] = 0.0f;
                if (!kept && wz) a.res[ent[r].x] = __uint_as_float(ent[r].y);
                kept_n += popc64(ballot(kept));
                bg += popc64(mg);
                be += popc64(me);
            }
        }
        if (lane == 0 && kept_n) atomicAdd(&o.tensor_counts[v.t], kept_n);
        if (QUANT) {
            sp = wave_sum(sp);
            sn = wave_sum(sn);
            np = wave_sum(np);
            nn = wave_sum(nn);
            if (lane == 0) {
                a.tile_q[4 * (size_t)tile + 0] = sp;
                a.tile_q[4 * (size_t)tile + 1] = sn;
                a.tile_q[4 * (size_t)tile + 2] = (double)np;
                a.tile_q[4 * (size_t)tile + 3] = (double)nn;
            }
        }
    }
}

static inline uint32_t blocks_for_waves(uint32_t waves) { return (waves + kWavesPerBlock - 1) / kWavesPerBlock; }

hipError_t launch_candidates(const CandArgs& a, const EmitArgs& o, bool quant, uint32_t max_tiles, hipStream_t st) {
    if (a.num_chunks == 0) return hipSuccess;
    const dim3 b(kBlock);
    uint32_t tb = blocks_for_waves(max_tiles);
    if (tb > kTileBlocks) tb = kTileBlocks;
    if (tb == 0) tb = 1;
    const dim3 gt(tb);
    hipLaunchKernelGGL(k_gather, gt, b, 0, st, a);
    hipLaunchKernelGGL(k_radix1, gt, b, 0, st, a);
    hipLaunchKernelGGL(k_radix2, gt, b, 0, st, a);
    hipLaunchKernelGGL(k_count, gt, b, 0, st, a);
    if (quant) hipLaunchKernelGGL(k_emit<true>, gt, b, 0, st, a, o);
    else hipLaunchKernelGGL(k_emit<false>, gt, b, 0, st, a, o);
    return hipGetLastError();
}

}  // namespace gd
