// Exact selection and ordered emission from the candidates (gfx950, wave64).
//
// Candidates (every element with key >= lo, or every element of a segment
// whose bracket missed) are processed in tiles of kTile consecutive
// candidates of one tensor, one wave per tile, so the work is balanced
// however unevenly the candidates fall across the gradient.  Five phases:
//
//   gather   : compacts each tile's candidates from the per-unit slots
//              (or, for a missed segment, straight from the residual) into
//              one array in ascending flat index, with the digit-0
//              histogram.
//   radix<L> : digit L-1 of the k-th largest key from the previous
//              histogram; the histogram of digit L over the candidates that
//              share the prefix found so far (L = 1, 2; digits of 10, 8 and
//              13 key bits).  Few candidates share the first 18 bits, so
//              digit 2 is counted with direct global atomics (fine and
//              coarse bins) instead of block histograms, a repeated bin
//              once per run.
//   count    : the last digit, i.e. the exact threshold key T and the number
//              of candidates equal to T to keep (lowest index first); per
//              tile, the candidates above and equal to T.  (A sampled
//              threshold sends every candidate, so emit derives these counts
//              from positions and neither radix nor count runs.)  For a
//              segment with fewer nonzero keys than k (the zero mode: T is
//              key 0, every candidate is nonzero and sent), it also sends the
//              zeros kept, the segment's lowest-index ones, and writes the
//              segment's tensor counts; radix skips such segments.
//   emit     : kept (index, value) pairs in ascending index order, the
//              residual of every candidate whose fate differs from what the
//              dense pass assumed, kept counts per tensor (and per-tile sums
//              for quantisation).
//
// Together they realise the exact-k rule: keep the k largest |acc| of each
// segment, ties broken by lower flat index (Algorithm 1, Section 4).  Each
// phase is one kernel: on this part a kernel boundary (about 1.5 us) is
// cheaper than the coherent reads a grid barrier needs for every wave to
// see the shared histograms.

// The histogram phases run in rounds of four consecutive tiles per block;
// each wave counts into its own LDS histogram and the block adds the four
// to the segment histogram once per round (waves of one segment merged), so
// the global atomics on the few hot bins are a quarter of one per tile.
// Those adds still meet on one address per bin from every block of a large
// segment, so some histograms have copies, picked by block number, that the
// next pick sums: digit 1 always, digit 0 and digit 2's coarse bins under a
// global threshold (one segment, every block).  A segment of more than
// kBigSegTiles tiles also keeps group sums of its tile counts, for emit's
// prefixes.

#include "gd_kernels.h"

namespace gd {

// A tile as its descriptor (written by the layout pass) describes it: tensor
// t and segment s, the segment's k, the compact candidates [p0, p1), the
// segment's first tile, the tensor's tiles [tfirst, tend), the non-empty
// unit ne0 holding the first candidate, and whether the bracket missed.
// Lane positions in a tile are tested as offsets, (pos - p0) < (p1 - p0), so
// that a tile near 2^32 candidate positions cannot wrap around.
struct TileView {
    uint32_t t, s, k, p0, p1, first_tile, tfirst, tend, ne0;
    bool miss;
};

// A tile descriptor as loaded: three 16-byte words.
struct TileDesc {
    uint4 d0, d1, d2;
};

// The descriptor of tile `tile`, or of tile 0 past the buffer.  The buffer
// holds a descriptor for every tile there can be, so a wave loads its next
// tile's descriptor before it knows whether that tile exists (the tile count
// is written by the layout pass): the descriptor then arrives with the
// count, or during the previous tile's work, instead of one round trip
// after it.  A descriptor past the count is stale and never used.
// The loads are relaxed atomics of wave scope (as in load_early), so that the
// compiler does not sink them past the test of the tile count.
__device__ __forceinline__ TileDesc load_desc(const CandArgs& a, uint32_t tile) {
    const uint64_t* d = reinterpret_cast<const uint64_t*>(a.tile_desc + (size_t)(tile < a.max_tiles ? tile : 0u) * kTileDescWords);
    uint64_t x[6];
#pragma unroll
    for (int i = 0; i < 6; ++i) x[i] = __hip_atomic_load(d + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WAVEFRONT);
    auto lo = [](uint64_t v) { return (uint32_t)v; };
    auto hi = [](uint64_t v) { return (uint32_t)(v >> 32); };
    return TileDesc{make_uint4(lo(x[0]), hi(x[0]), lo(x[1]), hi(x[1])), make_uint4(lo(x[2]), hi(x[2]), lo(x[3]), hi(x[3])),
                    make_uint4(lo(x[4]), hi(x[4]), lo(x[5]), hi(x[5]))};
}

__device__ __forceinline__ void tile_setup(const CandArgs& a, const TileDesc& td, TileView& v) {
    const uint4 d0 = td.d0, d1 = td.d1;
    v.t = d0.x & 0x7FFFFFFFu;
    v.miss = (d0.x >> 31) != 0;
    v.ne0 = d0.y;
    v.p0 = d0.z;
    v.p1 = d0.w;
    v.first_tile = d1.x;
    v.k = d1.y;
    v.tfirst = d1.z;
    v.tend = d1.w;
    v.s = a.per_tensor ? v.t : 0u;
}

__device__ __forceinline__ uint32_t* seg_hist(const CandArgs& a, uint32_t s, int which) {
    return a.hist + (size_t)s * kHistWords + which;
}

// Whether the tile's segment keeps group sums of its tile counts (its tiles
// are the tensor's under a per-tensor threshold, else all of them).
__device__ __forceinline__ bool seg_grouped(const CandArgs& a, const TileView& v, uint32_t ntiles) {
    return (a.per_tensor ? v.tend - v.tfirst : ntiles) > kBigSegTiles;
}

// Adds the block's four per-wave histograms (16-bit counters, two bins per
// word: a wave counts at most one tile of kTile candidates per round) to
// their segments' histograms and clears them.  lh holds the four histograms
// of NB / 2 words each; wseg[w] is wave w's segment this round (kNoKey: no
// tile); waves of one segment are summed first.  Called by the whole block.
template <int NB>
__device__ __forceinline__ void block_flush(const CandArgs& a, uint32_t* lh, const uint32_t* wseg, int which) {
    static_assert(kWavesPerBlock * kTile < 65536, "16-bit histogram counters");
    constexpr int W = NB / 2;
    __syncthreads();
    uint32_t sg[kWavesPerBlock];
    for (int i = threadIdx.x; i < W; i += kBlock) {
        uint32_t h[kWavesPerBlock];
#pragma unroll
        for (int w = 0; w < kWavesPerBlock; ++w) {
            sg[w] = wseg[w];
            h[w] = lh[w * W + i];
            lh[w * W + i] = 0;
        }
#pragma unroll
        for (int w = 0; w < kWavesPerBlock; ++w) {
            if (sg[w] == kNoKey) continue;
            uint32_t sum = h[w];
#pragma unroll
            for (int v = w + 1; v < kWavesPerBlock; ++v) {
                if (sg[v] == sg[w]) {
                    sum += h[v];
                    sg[v] = kNoKey;
                }
            }
            uint32_t* g = seg_hist(a, sg[w], which) + 2 * i;
            if (sum & 0xFFFFu) atomicAdd(g, sum & 0xFFFFu);
            if (sum >> 16) atomicAdd(g + 1, sum >> 16);
        }
    }
    __syncthreads();
}

constexpr int kRows = kTile / kWave;  // rows of 64 candidates in a tile
constexpr uint32_t kWin = kTile;      // non-empty units held in the gather window
constexpr int kWinRows = (kWin + kWave) / kWave;  // rows of 64 window entries (kWin + 1 of them)
constexpr int kWinHeadRows = 3;                   // rows loaded first

// A tile of kTile candidates lies in at most kTile consecutive non-empty
// units, so a window of kTile non-empty units starting at the unit that
// holds the tile's first candidate always covers the tile.
// LDS words of the gather phase: four digit-0 histograms, then per wave the
// window offsets and units and the tile's slot map.
constexpr int kGatherLds = kWavesPerBlock * (kNB0 / 2 + (kWin + 1) + kWin + kTile) + kWavesPerBlock;

__device__ __forceinline__ void phase_gather(const CandArgs& a, uint32_t* lds) {
    const int w = threadIdx.x >> 6, lane = lane_id();
    uint32_t* lh = lds;
    uint32_t* hw = lh + w * (kNB0 / 2);
    uint32_t* wo = lh + kWavesPerBlock * (kNB0 / 2) + w * (kWin + 1);
    uint32_t* wu = lh + kWavesPerBlock * (kNB0 / 2 + kWin + 1) + w * kWin;
    uint32_t* sm = lh + kWavesPerBlock * (kNB0 / 2 + kWin + 1 + kWin) + w * kTile;
    uint32_t* wseg = lh + kWavesPerBlock * (kNB0 / 2 + kWin + 1 + kWin + kTile);
    for (int i = lane; i < kNB0 / 2; i += kWave) hw[i] = 0;
    wave_lds_sync();
    // this block's copy of the digit-0 histogram (global threshold only)
    const int h0_at = kHistH0 + (a.per_tensor ? 0 : (int)(blockIdx.x % kH0Copies) * kNB0);
    const uint32_t stride = gridDim.x * kWavesPerBlock;
    TileDesc next = load_desc(a, blockIdx.x * kWavesPerBlock + w);
    const uint32_t ntiles = a.tile_base[a.T];
    // non-empty units, loaded with the tile count (an atomic load stays here)
    const uint32_t nne = load_early(a.num_ne);
    for (uint32_t t0 = blockIdx.x * kWavesPerBlock; t0 < ntiles; t0 += stride) {
        const uint32_t tile = t0 + w;
        const TileDesc td = next;
        if (t0 + stride < ntiles) next = load_desc(a, tile + stride);
        if (tile >= ntiles) {
            if (lane == 0) wseg[w] = kNoKey;
            if (!a.sampled) block_flush<kNB0>(a, lh, wseg, h0_at);  // block-uniform
            continue;
        }
        TileView v;
        tile_setup(a, td, v);
        // compact position -> source position (element, or dense-pass offset)
        const uint32_t shift = td.d2.x;
        uint32_t ix[kRows], vb[kRows];
        if (v.miss) {
            // every element of the tensor is a candidate; acc is in the residual
            const uint32_t e_base = shift;
#pragma unroll
            for (int r = 0; r < kRows; ++r) {
                const uint32_t pl = v.p0 + r * kWave + lane;
                ix[r] = e_base + pl;
                const uint32_t e = e_base + (pl - v.p0 < v.p1 - v.p0 ? pl : v.p0);
                // acc is the restored residual, or for a pull from the copy p - copy
                const uint32_t x = __float_as_uint(a.res ? a.res[e] : a.pull_p[e] - a.pull_copy[e]);
                vb[r] = pl - v.p0 < v.p1 - v.p0 ? x : 0u;
            }
        } else {
            // compact position p <-> dense-pass offset p + shift
            const uint32_t j0 = v.ne0;
            const uint32_t cnt = v.p1 - v.p0, r0 = v.p0 + shift, last = r0 + (cnt - 1);
            // The window runs from the unit holding the tile's first candidate
            // to the first unit that starts after its last one, W entries on
            // (W <= kWin: every unit before it holds a candidate of the tile).
            // The first kWinHead entries nearly always reach it; the others are
            // loaded only when they do not.  Window unit j >= 1 with j < W
            // starts inside the tile: it marks its first position in the slot
            // map (cleared first), which the map's max-scan then extends over
            // the unit's other positions.
            const uint32_t q0 = kRows * lane;
            {
                uint4* z = reinterpret_cast<uint4*>(sm + q0);
#pragma unroll
                for (int i = 0; i < kRows / 4; ++i) z[i] = make_uint4(0u, 0u, 0u, 0u);
                wave_lds_sync();
            }
            {
                auto load_rows = [&](int i0, int i1) {
                    uint32_t xo[kWinRows], xu[kWinRows];
#pragma unroll
                    for (int i = 0; i < kWinRows; ++i) {
                        if (i < i0 || i >= i1) continue;
                        const uint32_t j = i * kWave + lane;
                        const bool in = j < kWin && j0 + j < nne;
                        // unconditional loads at clamped positions (j0 < nne here), so
                        // that all of them are in flight together
                        const uint32_t jo = j0 + j <= nne ? j0 + j : nne, ju = in ? j0 + j : j0;
                        const uint32_t o = a.ne_off[jo], u = a.ne_unit[ju];
                        xo[i] = (j <= kWin && j0 + j <= nne) ? o : kNoKey;
                        xu[i] = in ? u : 0u;
                    }
                    uint32_t found = kNoKey;
#pragma unroll
                    for (int i = 0; i < kWinRows; ++i) {
                        if (i < i0 || i >= i1) continue;
                        const uint32_t j = i * kWave + lane;
                        if (j <= kWin) wo[j] = xo[i];
                        if (j < kWin) wu[j] = xu[i];
                        if (j >= 1 && xo[i] <= last) sm[xo[i] - r0] = j;  // 1 <= xo - r0 < cnt: see above
                        const uint64_t m = ballot(j <= kWin && xo[i] > last);
                        if (m && found == kNoKey) found = (uint32_t)(i * kWave + __ffsll((unsigned long long)m) - 1);
                    }
                    return found;
                };
                if (load_rows(0, kWinHeadRows) == kNoKey) load_rows(kWinHeadRows, kWinRows);
                wave_lds_sync();
            }
            // Lane L maps positions q0 .. q0 + kRows - 1: the window unit of a
            // position is the last mark at or before it (unit 0 when none), a
            // running maximum in the lane, then over the lanes below.  The
            // position's slot is the unit's slot base plus its offset there.
            {
                const uint4* hv = reinterpret_cast<const uint4*>(sm + q0);
                uint32_t m[kRows];
#pragma unroll
                for (int i = 0; i < kRows / 4; ++i) {
                    const uint4 h = hv[i];
                    m[4 * i + 0] = h.x;
                    m[4 * i + 1] = h.y;
                    m[4 * i + 2] = h.z;
                    m[4 * i + 3] = h.w;
                }
#pragma unroll
                for (int i = 1; i < kRows; ++i) m[i] = max(m[i], m[i - 1]);
                const uint32_t below = lane_below_value(wave_incl_max(m[kRows - 1]));
                uint32_t o[kRows];
#pragma unroll
                for (int i = 0; i < kRows; ++i) {
                    const uint32_t j = max(m[i], below);
                    o[i] = wu[j] * kUnitLen + (r0 + q0 + i - wo[j]);
                }
                uint4* dv = reinterpret_cast<uint4*>(sm + q0);
#pragma unroll
                for (int i = 0; i < kRows / 4; ++i) dv[i] = make_uint4(o[4 * i], o[4 * i + 1], o[4 * i + 2], o[4 * i + 3]);
            }
            wave_lds_sync();
            // rows: slot loads and stores are coalesced
#pragma unroll
            for (int r = 0; r < kRows; ++r) {
                const uint32_t q = r * kWave + lane;
                const uint2 e = a.slots[sm[q < cnt ? q : 0u]];  // cnt >= 1: sm[0] is a real slot
                ix[r] = e.x;
                vb[r] = e.y;
            }
        }
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
            const uint32_t pl = v.p0 + r * kWave + lane;
            const bool active = pl - v.p0 < v.p1 - v.p0;
            if (active) {
                a.cand_idx[pl] = ix[r];
                a.cand_val[pl] = vb[r];
            }
            // a missed tensor's rows can be all one key (zeros): one add per row there
            if (v.miss) lds_hist_add16_wave(hw, (vb[r] & 0x7FFFFFFFu) >> kD0Shift, active);
            else lds_hist_add16(hw, (vb[r] & 0x7FFFFFFFu) >> kD0Shift, active && !a.sampled);
        }
        if (lane == 0) wseg[w] = v.s;
        if (!a.sampled) block_flush<kNB0>(a, lh, wseg, h0_at);  // a sampled threshold needs no histogram
    }
}

// Keys of the tile's candidates, row by row.
__device__ __forceinline__ void load_keys(const CandArgs& a, const TileView& v, uint32_t key[kRows]) {
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
        const uint32_t pl = v.p0 + r * kWave + lane_id();
        const uint32_t x = a.cand_val[pl - v.p0 < v.p1 - v.p0 ? pl : v.p0];  // unconditional: all rows in flight
        key[r] = pl - v.p0 < v.p1 - v.p0 ? (x & 0x7FFFFFFFu) : 0u;
    }
}

// Level L: resolve digit L-1 from the previous histogram, then histogram
// digit L over candidates that share the prefix so far.
template <int L>
struct Level;
template <>
struct Level<1> {
    static constexpr int kPrevNB = kNB0, kPrevHist = kHistH0, kPrevCopies = 1, kNB = kNB1, kHist = kHistH1;
    static constexpr int kPrefixShift = kD0Shift, kDigitShift = kD1Shift, kPrevBits = 0;
};
template <>
struct Level<2> {
    static constexpr int kPrevNB = kNB1, kPrevHist = kHistH1, kPrevCopies = kH1Copies, kNB = kNB2, kHist = kHistH2;
    static constexpr int kPrefixShift = kD1Shift, kDigitShift = 0, kPrevBits = kD0Shift - kD1Shift;
};

template <int L>
__device__ __forceinline__ void read_level(const SegState& g, uint32_t k, uint32_t& prefix, uint32_t& rank) {
    if (L == 1) {
        prefix = 0;
        rank = k;
    } else {
        prefix = g.d0;
        rank = g.r1;
    }
}

template <int L>
__device__ __forceinline__ void write_level(SegState& g, uint32_t prefix, uint32_t rank) {
    if (L == 1) {
        g.d0 = prefix;
        g.r1 = rank;
    } else {
        g.p18 = prefix;
        g.r2 = rank;
    }
}

template <int L>
constexpr int radix_lds() {
    return L == 1 ? kWavesPerBlock * (Level<L>::kNB / 2) + kWavesPerBlock : 1;
}

// Digit 2 is counted with global atomics, since few candidates share the
// first 18 bits of the threshold.  Many equal keys (exact zeros, values of a
// narrower float type) would put thousands of atomics on one bin, so each
// wave keeps a run: the first bin it meets and how many of its candidates
// fell in it, added once when the wave moves to another segment or ends.
// Candidates in other bins are added one by one.
// This block's copy of the coarse digit-2 bins (global threshold only).
__device__ __forceinline__ int h2c_copy(const CandArgs& a) {
    return a.per_tensor ? 0 : (int)(blockIdx.x % kH2cCopies) * kNB2c;
}

__device__ __forceinline__ void run_flush(const CandArgs& a, uint32_t s, uint32_t d, uint32_t c) {
    if (c != 0 && lane_id() == 0) {
        atomicAdd(seg_hist(a, s, kHistH2) + d, c);
        atomicAdd(seg_hist(a, s, kHistH2c) + h2c_copy(a) + (d >> kD2cShift), c);
    }
}

template <int L>
__device__ __forceinline__ void phase_radix(const CandArgs& a, uint32_t* lds) {
    using Lv = Level<L>;
    constexpr bool kBlockHist = L == 1;
    const int w = threadIdx.x >> 6, lane = lane_id();
    uint32_t* lh = lds;
    uint32_t* hw = lh + w * (Lv::kNB / 2);
    uint32_t* wseg = lh + kWavesPerBlock * (Lv::kNB / 2);
    if (kBlockHist) {
        for (int i = lane; i < Lv::kNB / 2; i += kWave) hw[i] = 0;
        wave_lds_sync();
    }
    const uint32_t stride = gridDim.x * kWavesPerBlock;
    TileDesc next = load_desc(a, blockIdx.x * kWavesPerBlock + w);
    const uint32_t ntiles = a.tile_base[a.T];
    uint32_t cached_s = kNoKey, prefix = 0, rank = 0;
    uint32_t run_s = kNoKey, run_d = 0, run_c = 0;  // digit 2: this wave's run of one bin
    for (uint32_t t0 = blockIdx.x * kWavesPerBlock; t0 < ntiles; t0 += stride) {
        const uint32_t tile = t0 + w;
        const TileDesc td = next;
        if (t0 + stride < ntiles) next = load_desc(a, tile + stride);
        if (tile < ntiles) {
            TileView v;
            tile_setup(a, td, v);
            uint32_t key[kRows];
            load_keys(a, v, key);
            if (v.s != cached_s) {
                // (the zero flag is loaded beside the rest, not branched on
                // first: a dependent load would cost a round trip per segment)
                const uint32_t zero = a.seg[v.s].zero;
                uint32_t p0, r0, d, ab;
                read_level<L>(a.seg[v.s], v.k, p0, r0);
                if (L == 1 && !a.per_tensor)
                    wave_pick<Lv::kPrevNB, kH0Copies>(seg_hist(a, v.s, Lv::kPrevHist), r0, d, ab);
                else
                    wave_pick<Lv::kPrevNB, Lv::kPrevCopies>(seg_hist(a, v.s, Lv::kPrevHist), r0, d, ab);
                // the zero mode knows its threshold: no key matches, nothing counted
                prefix = zero ? kNoKey : (p0 << Lv::kPrevBits) | d;
                rank = r0 - ab;
                cached_s = v.s;
            }
            if (tile == v.first_tile && lane == 0 && prefix != kNoKey) write_level<L>(a.seg[v.s], prefix, rank);
            if (kBlockHist) {
                if (v.miss) {  // a missed tensor's rows can be all one key (zeros): one add per row
#pragma unroll
                    for (int r = 0; r < kRows; ++r)
                        lds_hist_add16_wave(hw, (key[r] >> Lv::kDigitShift) & (Lv::kNB - 1),
                                            (uint32_t)(r * kWave + lane) < v.p1 - v.p0 &&
                                                (key[r] >> Lv::kPrefixShift) == prefix);
                } else {
#pragma unroll
                    for (int r = 0; r < kRows; ++r)
                        lds_hist_add16(hw, (key[r] >> Lv::kDigitShift) & (Lv::kNB - 1),
                                       (uint32_t)(r * kWave + lane) < v.p1 - v.p0 && (key[r] >> Lv::kPrefixShift) == prefix);
                }
                if (lane == 0) wseg[w] = v.s;
            } else {
                if (v.s != run_s) {
                    run_flush(a, run_s, run_d, run_c);
                    run_s = v.s;
                    run_c = 0;
                }
                uint32_t* hf = seg_hist(a, v.s, kHistH2);
                uint32_t* hc = seg_hist(a, v.s, kHistH2c) + h2c_copy(a);
#pragma unroll
                for (int r = 0; r < kRows; ++r) {
                    const bool in = (uint32_t)(r * kWave + lane) < v.p1 - v.p0 && (key[r] >> Lv::kPrefixShift) == prefix;
                    const uint64_t m = ballot(in);
                    if (m == 0) continue;
                    const uint32_t d = key[r] & (Lv::kNB - 1);
                    if (run_c == 0) run_d = lane_value(d, __ffsll((unsigned long long)m) - 1);
                    const bool same = in && d == run_d;
                    run_c += popc64(ballot(same));
                    if (in && !same) {
                        atomicAdd(hf + d, 1u);
                        atomicAdd(hc + (d >> kD2cShift), 1u);
                    }
                }
            }
        } else if (kBlockHist && lane == 0) {
            wseg[w] = kNoKey;
        }
        if (kBlockHist) block_flush<Lv::kNB>(a, lh, wseg, Lv::kHist + (int)(blockIdx.x % kH1Copies) * Lv::kNB);
    }
    if (!kBlockHist) run_flush(a, run_s, run_d, run_c);
}

// Zero mode, elements [xs, xe) of one segment (segment start seg_a, zb of its
// zeros before xs, output slots from ob): the zeros whose rank among the
// segment's zeros is below need are kept.  Every element before such a zero
// is kept too, so it goes to slot ob + (e - seg_a); its residual becomes +0,
// or for a pull from the copy the copy takes the sent value.  acc is the
// residual here (nothing was zeroed early), or p - copy.  Whole wave.
__device__ __forceinline__ void fill_zeros(const CandArgs& a, const EmitArgs& o, uint32_t xs, uint32_t xe,
                                           uint32_t seg_a, uint32_t zb, uint32_t need, uint64_t ob) {
    for (uint32_t d0 = 0; d0 < xe - xs && zb < need; d0 += kWave) {
        const uint32_t d = d0 + lane_id();
        const bool valid = d < xe - xs;
        const uint32_t e = xs + (valid ? d : 0u);
        const float c = a.res ? 0.0f : a.pull_copy[e];
        const float x = a.res ? a.res[e] : a.pull_p[e] - c;
        const bool z = valid && (__float_as_uint(x) & 0x7FFFFFFFu) == 0u;
        const uint64_t m = ballot(z);
        if (z && zb + lanes_below(m) < need) {
            const uint64_t pos = ob + (e - seg_a);
            o.idx[pos] = e;
            o.val[pos] = x;  // +0 or -0, as acc is
            if (a.res) a.res[e] = 0.0f;
            else a.pull_copy[e] = c + x;  // as the client adds what it receives (-0 + +0 is +0)
        }
        zb += popc64(m);
    }
}

// Zero-mode segments of unit u, or with fill = false only whether one of
// them keeps zeros in the unit (any lane may call it so); with fill = true
// the whole wave fills them.
__device__ __forceinline__ bool zero_unit(const CandArgs& a, const EmitArgs& o, uint32_t u, bool fill) {
    const uint32_t ustart = u * kUnitLen, uend = a.N - ustart > kUnitLen ? ustart + kUnitLen : a.N;
    const uint32_t raw = a.loc[u] + a.boff[u / kScanUnits];  // candidates before ustart
    if (!a.per_tensor) {
        const SegState& g = a.seg[0];
        if (!g.zero) return false;
        const uint32_t need = keep_of(a.N, a.keep_ppm) - g.clo, zb = ustart - raw;
        if (fill && zb < need) fill_zeros(a, o, ustart, uend, 0u, zb, need, a.out_base[0]);
        return zb < need;
    }
    bool any = false;
    for (uint32_t t = a.unit_info[u] & 0x7FFFFFFFu; t < a.T && a.tensor_off[t] < uend; ++t) {
        const uint32_t ta = a.tensor_off[t], tb = a.tensor_off[t + 1];
        if (tb <= ustart || tb == ta || !a.seg[t].zero) continue;
        const uint32_t need = keep_of(tb - ta, a.keep_ppm) - a.seg[t].clo;
        const uint32_t zb = ta >= ustart ? 0u : (ustart - ta) - (raw - a.raw_tbase[t]);
        if (zb < need) {
            any = true;
            if (fill) fill_zeros(a, o, ta > ustart ? ta : ustart, tb < uend ? tb : uend, ta, zb, need, a.out_base[t]);
        }
    }
    return any;
}

// The zero mode's part of the count pass, after the candidate tiles: the kept
// counts of its tensors, all its candidates plus the zeros kept before each
// tensor's end less those kept before its start (per tensor: k), then the
// kept zeros.  It runs before emit, which sets the residual of sent
// candidates to +0, since it tells zeros from candidates by the residual.
// Unit u goes to wave u mod W, so the units at the start of a segment, which
// hold its kept zeros, spread over many waves.
__device__ __forceinline__ void zero_fill(const CandArgs& a, const EmitArgs& o) {
    const uint32_t W = gridDim.x * kWavesPerBlock, wid = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int lane = lane_id();
    for (uint64_t t = (uint64_t)wid * kWave + lane; t < a.T; t += (uint64_t)W * kWave) {
        const uint32_t s = a.per_tensor ? (uint32_t)t : 0u;
        if (!a.seg[s].zero) continue;
        const uint32_t seg_a = a.seg_off[s], seg_b = a.seg_off[s + 1];
        const uint32_t need = keep_of(seg_b - seg_a, a.keep_ppm) - a.seg[s].clo;
        const uint32_t raw_seg = a.per_tensor ? a.raw_tbase[t] : 0u;
        const uint32_t zs = (a.tensor_off[t] - seg_a) - (a.raw_tbase[t] - raw_seg);
        const uint32_t ze = (a.tensor_off[t + 1] - seg_a) - (a.raw_tbase[t + 1] - raw_seg);
        o.tensor_counts[t] = (a.raw_tbase[t + 1] - a.raw_tbase[t]) + (ze < need ? ze : need) - (zs < need ? zs : need);
    }
    for (uint64_t u0 = wid; u0 < a.num_units; u0 += (uint64_t)W * kWave) {
        const uint64_t u = u0 + (uint64_t)W * lane;
        const bool fill = u < a.num_units && zero_unit(a, o, (uint32_t)u, false);
        uint64_t todo = ballot(fill);
        while (todo) {
            const int src = __ffsll((unsigned long long)todo) - 1;
            todo &= todo - 1;
            zero_unit(a, o, lane_value((uint32_t)u, src), true);
        }
    }
}

__device__ __forceinline__ void phase_count(const CandArgs& a, const EmitArgs& o) {
    const int w = threadIdx.x >> 6, lane = lane_id();
    const uint32_t stride = gridDim.x * kWavesPerBlock;
    TileDesc next = load_desc(a, blockIdx.x * kWavesPerBlock + w);
    const uint32_t ntiles = a.tile_base[a.T];
    uint32_t cached_s = kNoKey, thr = kNoKey, need = 0;
    for (uint32_t tile = blockIdx.x * kWavesPerBlock + w; tile < ntiles; tile += stride) {
        const TileDesc td = next;
        if (tile + stride < ntiles) next = load_desc(a, tile + stride);
        TileView v;
        tile_setup(a, td, v);
        uint32_t key[kRows];
        load_keys(a, v, key);
        if (v.s != cached_s) {
            // digit 2 in two steps: its coarse bin, then the bin among 32
            const uint32_t zero = a.seg[v.s].zero, clo = a.seg[v.s].clo;
            const uint32_t p18 = a.seg[v.s].p18, r2 = a.seg[v.s].r2;
            uint32_t dc, abc, df, abf;
            if (a.per_tensor) wave_pick<kNB2c>(seg_hist(a, v.s, kHistH2c), r2, dc, abc);
            else wave_pick<kNB2c, kH2cCopies>(seg_hist(a, v.s, kHistH2c), r2, dc, abc);
            wave_pick<kNB2 / kNB2c>(seg_hist(a, v.s, kHistH2) + (dc << kD2cShift), r2 - abc, df, abf);
            // zero mode: T = key 0; every candidate (nonzero) is above it and
            // the first k - cnt zeros, none of them a candidate, are kept
            thr = zero ? 0u : (p18 << kD1Shift) | (dc << kD2cShift) | df;
            need = zero ? v.k - clo : r2 - abc - abf;
            cached_s = v.s;
        }
        if (tile == v.first_tile && lane == 0) {
            a.seg[v.s].thr = thr;
            a.seg[v.s].need = need;
        }
        uint32_t gt = 0, eq = 0;
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
            const bool active = (uint32_t)(r * kWave + lane) < v.p1 - v.p0;
            gt += active && key[r] > thr;
            eq += active && key[r] == thr;
        }
        gt = wave_sum(gt);
        eq = wave_sum(eq);
        if (lane == 0) {
            a.tile_gt[tile] = gt;
            a.tile_eq[tile] = eq;
            if (seg_grouped(a, v, ntiles)) {
                if (gt) atomicAdd(&a.grp_gt[tile / kGroupTiles], gt);
                if (eq) atomicAdd(&a.grp_eq[tile / kGroupTiles], eq);
            }
        }
    }
    if (a.flags[1]) zero_fill(a, o);  // some segment takes the zero mode
}

// This lane's part of the sums of x and y over [lo, hi) (wave_sum gives the
// totals).
__device__ __forceinline__ void sum_span(const uint32_t* x, const uint32_t* y, uint32_t lo, uint32_t hi, uint32_t& g,
                                         uint32_t& e) {
    for (uint32_t b0 = lo; b0 < hi; b0 += 8 * kWave) {
        uint32_t g8[8], e8[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t q = b0 + j * kWave + lane_id();
            const uint32_t qc = q < hi ? q : lo;  // unconditional loads, all in flight
            const uint32_t xv = x[qc], yv = y[qc];
            g8[j] = q < hi ? xv : 0u;
            e8[j] = q < hi ? yv : 0u;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            g += g8[j];
            e += e8[j];
        }
    }
}

// Candidates above and equal to the threshold in tiles [lo, hi) of one
// segment (this lane's part): whole groups of a grouped segment come from
// the group sums, the tiles at either end one by one.
__device__ __forceinline__ void sum_tiles(const CandArgs& a, bool grouped, uint32_t lo, uint32_t hi, uint32_t& g,
                                          uint32_t& e) {
    const uint32_t glo = (lo + kGroupTiles - 1) / kGroupTiles, ghi = hi / kGroupTiles;
    if (grouped && glo < ghi) {
        sum_span(a.tile_gt, a.tile_eq, lo, glo * kGroupTiles, g, e);
        sum_span(a.grp_gt, a.grp_eq, glo, ghi, g, e);
        sum_span(a.tile_gt, a.tile_eq, ghi * kGroupTiles, hi, g, e);
    } else {
        sum_span(a.tile_gt, a.tile_eq, lo, hi, g, e);
    }
}

template <bool QUANT>
__device__ __forceinline__ void phase_emit(const CandArgs& a, const EmitArgs& o) {
    const int w = threadIdx.x >> 6, lane = lane_id();
    const uint32_t stride = gridDim.x * kWavesPerBlock;
    TileDesc next = load_desc(a, blockIdx.x * kWavesPerBlock + w);
    const uint32_t ntiles = a.tile_base[a.T];
    for (uint32_t tile = blockIdx.x * kWavesPerBlock + w; tile < ntiles; tile += stride) {
        const TileDesc td = next;
        if (tile + stride < ntiles) next = load_desc(a, tile + stride);
        TileView v;
        tile_setup(a, td, v);
        uint32_t ix[kRows], vb[kRows];
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
            const uint32_t pl = v.p0 + r * kWave + lane;
            const uint32_t pc = pl - v.p0 < v.p1 - v.p0 ? pl : v.p0;
            const uint32_t x = a.cand_idx[pc], y = a.cand_val[pc];
            ix[r] = pl - v.p0 < v.p1 - v.p0 ? x : 0u;
            vb[r] = pl - v.p0 < v.p1 - v.p0 ? y : 0u;
        }
        const uint32_t hi = v.miss ? kNoKey : a.seg[v.s].hi;
        const uint32_t thr = a.seg[v.s].thr, need = a.seg[v.s].need;
        // zero mode: the zeros kept before a candidate (at most need) shift it
        const bool zseg = a.seg[v.s].zero != 0;
        const uint32_t seg_a = a.per_tensor ? a.tensor_off[v.t] : 0u;
        // A pull from the copy reads the copy word of every entry that may be
        // kept, to add the sent value to it; the loads are issued here, early
        // enough to overlap the prefix work.
        const bool pull = a.res == nullptr;
        float old[kRows];
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
            const uint32_t key = vb[r] & 0x7FFFFFFFu;
            const bool valid = (uint32_t)(r * kWave + lane) < v.p1 - v.p0;
            old[r] = 0.0f;
            if (pull && valid && key >= thr) old[r] = a.pull_copy[ix[r]];
        }
        // candidates above / equal to the threshold in earlier tiles of the segment
        uint32_t bg = 0, be = 0;
        if (a.sampled) {
            // every candidate is sent: the earlier tiles hold p0 minus the segment's first candidate
            bg = v.p0 - (a.per_tensor ? a.ten_cbase[v.t] : 0u);
        } else {
            sum_tiles(a, seg_grouped(a, v, ntiles), v.first_tile, tile, bg, be);
            bg = wave_sum(bg);
            be = wave_sum(be);
        }
        const uint32_t bg0 = bg, be0 = be;
        const uint64_t ob = a.out_base[v.s];
        double sp = 0.0, sn = 0.0;
        uint32_t np = 0, nn = 0;
        uint32_t kmin = kNoKey;  // sampled threshold, threshold centre: smallest key sent by this lane
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
            const bool valid = (uint32_t)(r * kWave + lane) < v.p1 - v.p0;
            const uint32_t key = vb[r] & 0x7FFFFFFFu;
            const bool isgt = valid && (a.sampled || key > thr);
            const bool iseq = valid && !a.sampled && key == thr;
            const uint64_t mg = ballot(isgt), me = ballot(iseq);
            const uint32_t G = bg + lanes_below(mg), E = be + lanes_below(me);
            const uint32_t zb = ix[r] - seg_a - G;  // zero mode: zeros of the segment before ix
            const uint64_t pos = ob + G + (zseg ? (zb < need ? zb : need) : (E < need ? E : need));
            // past the capacity (only possible under a sampled threshold) an
            // entry is not sent and keeps acc in the residual
            const bool kept = (isgt || (iseq && E < need)) && pos < o.capacity;
            if (kept) {
                o.idx[pos] = ix[r];
                o.val[pos] = __uint_as_float(vb[r]);
                if (QUANT && a.sampled && o.qkind == kQuantThreshold) kmin = key < kmin ? key : kmin;
                if (QUANT && o.qkind != kQuantColumnMean) {  // column sums come from the sent entries later
                    const float x = __uint_as_float(vb[r]);
                    if (x < 0.0f) {
                        sn += (double)x;
                        ++nn;
                    } else {
                        sp += (double)x;
                        ++np;
                    }
                }
            }
            if (pull) {
                // the client adds the sent value to what it holds; so does its copy
                if (kept) a.pull_copy[ix[r]] = old[r] + __uint_as_float(vb[r]);
            } else {
                const bool wz = valid && key >= hi;
                if (kept != wz) a.res[ix[r]] = kept ? 0.0f : __uint_as_float(vb[r]);
            }
            bg += popc64(mg);
            be += popc64(me);
        }
        if (tile == v.tfirst && !zseg) {  // (zero-mode counts: zero_fill)
            // The first tile of a tensor writes the tensor's kept count: every
            // candidate of the tensor above T, plus as many of its candidates
            // equal to T as the segment still needs at this tile (ties go to
            // the lowest index, and a tensor's tiles are consecutive).  No
            // atomics: a few hundred tiles adding to one counter serialise badly.
            uint32_t cnt;
            if (a.sampled) {
                cnt = a.ten_cbase[v.t + 1] - a.ten_cbase[v.t];  // every candidate is sent
            } else {
                uint32_t gt_t = 0, eq_t = 0;
                sum_tiles(a, seg_grouped(a, v, ntiles), tile, v.tend, gt_t, eq_t);
                gt_t = wave_sum(gt_t);
                eq_t = wave_sum(eq_t);
                const uint32_t left = need > be0 ? need - be0 : 0u;
                cnt = gt_t + (eq_t < left ? eq_t : left);
            }
            // entries past the capacity are not sent
            const uint64_t start = ob + bg0 + (be0 < need ? be0 : need);
            const uint64_t room = o.capacity > start ? o.capacity - start : 0u;
            if (lane == 0) o.tensor_counts[v.t] = (uint64_t)cnt < room ? cnt : (uint32_t)room;
        }
        if (QUANT) {
            if (a.sampled && o.qkind == kQuantThreshold) {
                // the tile's smallest sent key (kNoKey if none) in place of its positive sum
                sp = (double)wave_min(kmin);
            } else {
                sp = wave_sum(sp);
                sn = wave_sum(sn);
                np = wave_sum(np);
                nn = wave_sum(nn);
            }
            if (lane == 0) {
                a.tile_q[4 * (size_t)tile + 0] = sp;
                a.tile_q[4 * (size_t)tile + 1] = sn;
                a.tile_q[4 * (size_t)tile + 2] = (double)np;
                a.tile_q[4 * (size_t)tile + 3] = (double)nn;
            }
        }
    }
}

__global__ __launch_bounds__(kBlock) void k_gather(CandArgs a) {
    __shared__ __align__(16) uint32_t lds[kGatherLds];
    phase_gather(a, lds);
}

template <int L>
__global__ __launch_bounds__(kBlock) void k_radix(CandArgs a) {
    __shared__ uint32_t lds[radix_lds<L>()];
    phase_radix<L>(a, lds);
}

__global__ __launch_bounds__(kBlock) void k_count(CandArgs a, EmitArgs o) { phase_count(a, o); }

template <bool QUANT>
__global__ __launch_bounds__(kBlock) void k_emit(CandArgs a, EmitArgs o) {
    phase_emit<QUANT>(a, o);
}

static inline uint32_t blocks_for_waves(uint32_t waves) { return (waves + kWavesPerBlock - 1) / kWavesPerBlock; }

hipError_t launch_candidates(const CandArgs& a, const EmitArgs& o, bool quant, uint32_t max_tiles, hipStream_t st) {
    if (a.num_units == 0) return hipSuccess;
    const dim3 b(kBlock);
    const uint32_t need = blocks_for_waves(max_tiles) ? blocks_for_waves(max_tiles) : 1u;
    const dim3 gt(need < kTileBlocks ? need : kTileBlocks);
    hipLaunchKernelGGL(k_gather, gt, b, 0, st, a);
    if (!a.sampled) {  // a sampled threshold is already exact
        hipLaunchKernelGGL(k_radix<1>, gt, b, 0, st, a);
        hipLaunchKernelGGL(k_radix<2>, gt, b, 0, st, a);
    }
    if (!a.sampled) hipLaunchKernelGGL(k_count, gt, b, 0, st, a, o);  // under a sampled threshold every candidate is sent
    if (quant) hipLaunchKernelGGL(k_emit<true>, gt, b, 0, st, a, o);
    else hipLaunchKernelGGL(k_emit<false>, gt, b, 0, st, a, o);
    return hipGetLastError();
}

}  // namespace gd
