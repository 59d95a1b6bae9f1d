// Server-side apply of sparse pushes to a parameter shard (Section 3: each
// server owns a shard of the parameters and receives the clients' pieces).
//
// For an index pushed by several clients the values are summed in client
// order starting from +0, and the parameter is updated once:
// p[i] -= lr * s[i].  No atomics, so the result is deterministic.
//
// Two forms, with the same results bit for bit.  The scattered form reads
// and writes only the pushed parameters; the streaming form reads the whole
// shard in order and writes back the 16-byte vectors that change, for pushes
// dense enough that most 128-byte lines of the shard hold an update.
// Quantised pushes (indices, sign bits, centre pairs; Section 5.4) are decoded
// entry by entry where their values are read.
//
// The scattered form: one block per bucket of 2^15 consecutive parameter
// indices.  The block finds where the bucket starts and ends in every
// client's (ascending) index list by a 32-way search per half-wave (four
// rounds of loads for a list of a few hundred thousand entries, instead of a
// binary search's twenty), stages those entries in LDS, marking the indices
// pushed more than once, and then gives every index to the lowest client
// holding it, which sums all clients' values for it in client order and
// writes p once.  The parameter writes of a block stay inside its bucket.

#include <algorithm>
#include <atomic>
#include <map>
#include <mutex>
#include <thread>
#include <utility>

#include "gd_kernels.h"

namespace gd {

constexpr int kApplyBucketShift = 15;
constexpr int kApplyLds = 2048;                              // entries of all clients staged per bucket
constexpr int kBucketWords = (1 << kApplyBucketShift) / 32;  // one bit per index of a bucket

// First position in list[lo, hi) whose value is >= x, found by the 32 lanes of
// one half-wave together (g: lane within the half, mask: the half's lanes).
__device__ uint32_t half_lower_bound(const uint32_t* list, uint32_t lo, uint32_t hi, uint32_t x, uint32_t g,
                                     uint64_t mask) {
    while (hi > lo) {
        const uint32_t len = hi - lo;
        if (len <= 32u) {
            const bool below = g < len && list[lo + (g < len ? g : 0u)] < x;
            return lo + popc64(ballot(below) & mask);
        }
        const uint32_t step = (len + 31u) / 32u;
        uint32_t q = lo + (g + 1u) * step - 1u;
        if (q >= hi) q = hi - 1u;
        // probes rise with g, so the lanes below x form a prefix of the half
        const uint32_t t = popc64(ballot(list[q] < x) & mask);
        const uint64_t nlo = (uint64_t)lo + (uint64_t)t * step, nhi = nlo + step;
        lo = nlo < hi ? (uint32_t)nlo : hi;
        hi = nhi < hi ? (uint32_t)nhi : hi;
    }
    return lo;
}

// First position in list[lo, hi) holding x, or hi.
__device__ __forceinline__ uint32_t find_u32(const uint32_t* list, uint32_t lo, uint32_t hi, uint32_t x) {
    uint32_t a = lo, b = hi;
    while (a < b) {
        const uint32_t mid = a + ((b - a) >> 1);
        if (list[mid] < x) a = mid + 1;
        else b = mid;
    }
    return a < hi && list[a] == x ? a : hi;
}

// Value of entry pos (index i) of push c: sent as is, or a quantised push's
// centre, chosen by the entry's sign bit from the pair of its tensor or column.
__device__ __forceinline__ float push_val(const ApplyArgs& a, uint32_t c, uint32_t pos, uint32_t i) {
    if (a.qkind == 0) return a.val[c][pos];
    uint32_t lo = 0, hi = a.T;  // tensor holding i: the last t with tensor_off[t] <= i
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (a.tensor_off[mid] <= i) lo = mid;
        else hi = mid;
    }
    const uint32_t g = a.qkind == kQuantColumnMean ? a.colbase[lo] + (i - a.tensor_off[lo]) % a.columns[lo] : lo;
    const uint32_t neg = (a.bits[c][pos >> 5] >> (pos & 31)) & 1u;
    return a.means[c][2 * g + neg];
}

__global__ __launch_bounds__(kBlock) void k_apply(ApplyArgs a) {
    __shared__ uint32_t rng[kMaxPushes][2];  // bucket's [begin, end) in each client's list
    __shared__ uint32_t base[kMaxPushes + 1];  // first staged entry of each client
    __shared__ uint32_t sidx[kApplyLds];
    __shared__ float sval[kApplyLds];
    __shared__ uint32_t seen[2][kBucketWords];  // [0]: index pushed at least once, [1]: more than once
    const int tid = threadIdx.x, w = (int)wave_index(), lane = lane_id();
    const uint32_t b = blockIdx.x;
    const uint32_t i_lo = b << kApplyBucketShift;
    const uint64_t i_hi64 = ((uint64_t)b + 1) << kApplyBucketShift;
    const uint32_t i_hi = i_hi64 < a.n ? (uint32_t)i_hi64 : a.n;
    // 1. the bucket's range in every list: one client per wave, the two bounds
    //    by the two half-waves
    const uint32_t half = (uint32_t)lane >> 5, g = (uint32_t)lane & 31u;
    const uint64_t mask = half ? 0xFFFFFFFF00000000ull : 0x00000000FFFFFFFFull;
    for (uint32_t c = w; c < a.C; c += kWavesPerBlock) {
        const uint32_t pos = half_lower_bound(a.idx[c], 0, a.nnz[c], half ? i_hi : i_lo, g, mask);
        if (g == 0) rng[c][half] = pos;
    }
    __syncthreads();
    if (tid == 0) {
        uint32_t acc = 0;
        for (uint32_t c = 0; c < a.C; ++c) {
            base[c] = acc;
            acc += rng[c][1] - rng[c][0];
        }
        base[a.C] = acc;
    }
    __syncthreads();
    const uint32_t total = base[a.C];
    if (total == 0) return;
    const bool staged = total <= (uint32_t)kApplyLds;
    // 2. stage the bucket's entries (index, value) of every client, and mark
    //    the indices pushed more than once
    if (staged) {
        for (uint32_t q = tid; q < 2u * kBucketWords; q += kBlock) (&seen[0][0])[q] = 0;
        __syncthreads();
        for (uint32_t c = 0; c < a.C; ++c) {
            const uint32_t r0 = rng[c][0], cnt = rng[c][1] - r0, o = base[c];
            for (uint32_t q = tid; q < cnt; q += kBlock) {
                const uint32_t ii = a.idx[c][r0 + q];
                const uint32_t off = ii - i_lo, bit = 1u << (off & 31);
                // an index outside the bucket (a list out of order) is skipped
                sidx[o + q] = off < i_hi - i_lo ? ii : kNoKey;
                sval[o + q] = push_val(a, c, r0 + q, ii);
                if (off < i_hi - i_lo && (atomicOr(&seen[0][off >> 5], bit) & bit)) atomicOr(&seen[1][off >> 5], bit);
            }
        }
        __syncthreads();
    }
    // 3. each entry: skip it if a lower client holds the same index, else sum
    //    every client's value for it in client order and update p once (an
    //    index pushed once needs no search).  When staged, a thread settles all
    //    its entries first and then reads all its parameters at once, so their
    //    latencies overlap instead of adding up.
    if (staged) {
        constexpr int kPer = kApplyLds / kBlock;
        uint32_t pi[kPer];
        float pstep[kPer];
        bool pv[kPer];
#pragma unroll
        for (int t = 0; t < kPer; ++t) {
            const uint32_t e = tid + t * kBlock;
            pv[t] = false;
            pi[t] = i_lo;  // a valid parameter index for the unconditional load below
            pstep[t] = 0.0f;
            if (e < total && sidx[e] != kNoKey) {
                uint32_t c = 0;
                while (base[c + 1] <= e) ++c;  // client of staged entry e
                const uint32_t i = sidx[e];
                const uint32_t off = i - i_lo;
                const bool once = (seen[1][off >> 5] & (1u << (off & 31))) == 0;
                bool owner = true;
                for (uint32_t cc = 0; cc < c && owner && !once; ++cc)
                    owner = find_u32(sidx, base[cc], base[cc + 1], i) == base[cc + 1];
                if (owner) {
                    float sum = 0.0f + sval[e];
                    for (uint32_t cc = c + 1; cc < a.C && !once; ++cc) {
                        const uint32_t hit = find_u32(sidx, base[cc], base[cc + 1], i);
                        if (hit != base[cc + 1]) sum = sum + sval[hit];
                    }
                    pv[t] = true;
                    pi[t] = i;
                    pstep[t] = a.lr * sum;
                }
            }
        }
        float pold[kPer];
#pragma unroll
        for (int t = 0; t < kPer; ++t) pold[t] = a.p[pi[t]];
#pragma unroll
        for (int t = 0; t < kPer; ++t)
            if (pv[t]) a.p[pi[t]] = pold[t] - pstep[t];
        return;
    }
    for (uint32_t e = tid; e < total; e += kBlock) {
        uint32_t c = 0;
        while (base[c + 1] <= e) ++c;  // client of staged entry e
        const uint32_t q = e - base[c];
        const uint32_t i = staged ? sidx[e] : a.idx[c][rng[c][0] + q];
        if (i - i_lo >= i_hi - i_lo) continue;  // outside the bucket: a list out of order
        bool owner = true;
        for (uint32_t cc = 0; cc < c && owner; ++cc) {
            const uint32_t hit = staged ? find_u32(sidx, base[cc], base[cc + 1], i)
                                        : find_u32(a.idx[cc], rng[cc][0], rng[cc][1], i);
            owner = staged ? hit == base[cc + 1] : hit == rng[cc][1];
        }
        if (!owner) continue;
        float s = 0.0f;
        for (uint32_t cc = 0; cc < a.C; ++cc) {
            if (cc < c) continue;
            if (cc == c) {
                s = s + (staged ? sval[e] : push_val(a, c, rng[c][0] + q, i));
                continue;
            }
            if (staged) {
                const uint32_t hit = find_u32(sidx, base[cc], base[cc + 1], i);
                if (hit != base[cc + 1]) s = s + sval[hit];
            } else {
                const uint32_t hit = find_u32(a.idx[cc], rng[cc][0], rng[cc][1], i);
                if (hit != rng[cc][1]) s = s + push_val(a, cc, hit, i);
            }
        }
        const float step = a.lr * s;
        a.p[i] = a.p[i] - step;
    }
}

// The streaming form, for pushes dense enough that most 128-byte lines of
// the shard hold an update (the scattered form above then fetches nearly every
// line anyway, one scattered word at a time).  One block per tile of
// kApplyTileLen consecutive parameters reads the tile in order with 16-byte
// loads, forms the sum of every pushed parameter of the tile in LDS, and
// writes back only the 16-byte vectors that an entry touches.
//
// The sums start at +0 and take the clients in turn, between barriers.  No
// two entries of one client's turn share an index (a push holds an index at
// most once), so each LDS sum is formed in client order without atomics, as
// the scattered form forms it, and the parameter then takes p - lr * sum:
// the two forms agree bit for bit.  The tile's range in every client's list
// comes from a bounds table (k_apply_bounds, one pass over the lists before
// this kernel).  Each thread loads kApplyTileEntries entries of the tile at
// once, for all clients together (entry e of the tile belongs to the last
// client whose first entry in the tile is at or before e); a tile with more
// entries takes further rounds.
//
// Tiles of 4,096 parameters (four 16-byte vectors per thread, 16.9 KB of
// LDS) keep eight blocks per compute unit in flight, which streams faster on
// this part than fewer blocks holding larger chunks in registers, or
// persistent blocks that load the next tile while they settle the current
// one (both measured slower).
constexpr int kApplyTileShift = 12;
constexpr uint32_t kApplyTileLen = 1u << kApplyTileShift;                          // parameters per block
constexpr int kApplyTileThreads = 256;
constexpr int kApplyTileVecs = (int)kApplyTileLen / 4 / kApplyTileThreads;        // 16-byte vectors per thread
constexpr int kApplyTileEntries = 2;                                                // entries per thread per round
constexpr uint32_t kApplyTileRound = (uint32_t)kApplyTileEntries * kApplyTileThreads;
static_assert(kMaxPushes <= kWave, "one lane per client holds its range");

// push_val for a client index that differs between lanes: the client's sign
// bits and centres are picked by comparing it with each client in turn.
__device__ __forceinline__ float push_val_lanes(const ApplyArgs& a, uint32_t c, uint32_t pos, uint32_t i) {
    const uint32_t* bits = a.bits[0];
    const float* means = a.means[0];
    for (uint32_t cc = 1; cc < a.C; ++cc) {
        if (c == cc) {
            bits = a.bits[cc];
            means = a.means[cc];
        }
    }
    uint32_t lo = 0, hi = a.T;  // tensor holding i
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (a.tensor_off[mid] <= i) lo = mid;
        else hi = mid;
    }
    const uint32_t g = a.qkind == kQuantColumnMean ? a.colbase[lo] + (i - a.tensor_off[lo]) % a.columns[lo] : lo;
    const uint32_t neg = (bits[pos >> 5] >> (pos & 31)) & 1u;
    return means[2 * g + neg];
}

// The bounds table of the streaming form: row c holds, for every tile
// boundary B_b (b * kApplyTileLen for b < tiles, n for b = tiles), the first
// position in client c's list whose index is at least B_b.  With f(x) the
// number of boundaries at or below x, entry e starts the boundaries in
// [f(x_{e-1}), f(x_e)), the list's head [0, f(x_0)) starts at 0 and its tail
// [f(x_last), tiles] at the list's length: one pass over the entries, no
// search.  One row of blocks per client (blockIdx.y); the first tiles + 1
// threads of a row fill the head and tail, the others one entry each.  (A
// list out of order leaves some boundaries unwritten; readers clamp.)
__global__ __launch_bounds__(kBlock) void k_apply_bounds(ApplyArgs a, uint32_t tiles) {
    const uint32_t c = blockIdx.y;
    const uint32_t m = a.nnz[c];
    const uint32_t* list = a.idx[c];
    uint32_t* row = const_cast<uint32_t*>(a.tab) + (size_t)c * a.tstride;
    const uint64_t item = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
    const auto f = [&](uint32_t x) { return x < a.n ? (x >> kApplyTileShift) + 1u : tiles + 1u; };
    if (item <= tiles) {
        const uint32_t b = (uint32_t)item;
        if (m == 0 || b < f(list[0])) row[b] = 0;
        else if (b >= f(list[m - 1])) row[b] = m;
        return;
    }
    const uint64_t e = item - tiles;  // 1 .. m - 1
    if (e >= m) return;
    const uint32_t hi = f(list[e]);
    for (uint32_t b = f(list[e - 1]); b < hi; ++b) row[b] = (uint32_t)e;
}

__global__ __launch_bounds__(kApplyTileThreads) void k_apply_tile(ApplyArgs a) {
    __shared__ __align__(16) float sum[kApplyTileLen];      // per parameter of the tile
    __shared__ uint32_t touched[kApplyTileLen / 32];       // pushed at least once
    const int tid = threadIdx.x, lane = lane_id();
    const uint32_t b = blockIdx.x, C = a.C;
    const uint32_t i_lo = b << kApplyTileShift;
    const bool whole = (uint64_t)i_lo + kApplyTileLen <= a.n;  // the same in every thread
    const uint32_t len = whole ? kApplyTileLen : a.n - i_lo;
    // The tile's range in the list of client `lane` (lanes >= C: none), from
    // the bounds table and clamped to the list, so that any table content
    // stays inside it.  Every wave reads it, so no barrier is needed for it.
    uint32_t r0 = 0, r1 = 0, nz = 0;
    if ((uint32_t)lane < C) {
        const uint32_t* row = a.tab + (size_t)lane * a.tstride + b;
        r0 = row[0];
        r1 = row[1];
    }
    // The tile's parameters: vector v = tid + kApplyTileThreads r holds
    // parameters i_lo + 4v .. 4v + 3 (each row of vectors is one coalesced
    // 4 KB read).
    f4 pv[kApplyTileVecs];
    if (whole) {
#pragma unroll
        for (int r = 0; r < kApplyTileVecs; ++r)
            pv[r] = *reinterpret_cast<const f4*>(a.p + i_lo + 4u * ((uint32_t)tid + (uint32_t)r * kApplyTileThreads));
    } else {
#pragma unroll
        for (int r = 0; r < kApplyTileVecs; ++r) {
            const uint32_t o = 4u * ((uint32_t)tid + (uint32_t)r * kApplyTileThreads);
            pv[r] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (o + q < len) pv[r][q] = a.p[i_lo + o + q];
        }
    }
    for (uint32_t c = 0; c < C; ++c)
        if ((uint32_t)lane == c) nz = a.nnz[c];
    r0 = min(r0, nz);
    r1 = min(r1, nz);
    const uint32_t cnt = r1 > r0 ? r1 - r0 : 0u;
    const uint32_t incl = wave_incl_scan(cnt);
    const uint32_t base = incl - cnt;                        // the client's first entry in the tile
    const uint32_t total = lane_value(incl, kWave - 1);      // the same in every wave
#pragma unroll
    for (int r = 0; r < kApplyTileVecs; ++r)
        reinterpret_cast<f4*>(sum)[tid + r * kApplyTileThreads] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    if (tid < (int)(kApplyTileLen / 32)) touched[tid] = 0;
    if (total == 0) return;  // nothing pushed here (block-uniform): nothing is written
    for (uint32_t e0 = 0; e0 < total; e0 += kApplyTileRound) {
        // this thread's entries e = e0 + tid + kApplyTileThreads k: offset in
        // the tile, client and value, all loaded at once
        uint32_t off[kApplyTileEntries], cl[kApplyTileEntries];
        float val[kApplyTileEntries];
#pragma unroll
        for (int k = 0; k < kApplyTileEntries; ++k) {
            const uint32_t e = e0 + (uint32_t)tid + (uint32_t)k * kApplyTileThreads;
            uint32_t c = 0, first = 0, at = lane_value(r0, 0);
            const uint32_t* ip = a.idx[0];
            const float* vp = a.val[0];
            for (uint32_t cc = 1; cc < C; ++cc) {
                const uint32_t bc = lane_value(base, (int)cc);
                if (e >= bc) {
                    c = cc;
                    first = bc;
                    at = lane_value(r0, (int)cc);
                    ip = a.idx[cc];
                    vp = a.val[cc];
                }
            }
            cl[k] = kNoKey;
            off[k] = kNoKey;
            val[k] = 0.0f;
            if (e < total) {
                const uint32_t pos = at + (e - first);
                const uint32_t i = ip[pos];
                cl[k] = c;
                off[k] = i - i_lo;  // outside the tile (a list out of order): skipped below
                val[k] = a.qkind == 0 ? vp[pos] : push_val_lanes(a, c, pos, i);
            }
        }
        __syncthreads();  // sums cleared (first round), or the previous round's turns done
        for (uint32_t t = 0; t < C; ++t) {
            if (t > 0) __syncthreads();  // the previous client's turn done
#pragma unroll
            for (int k = 0; k < kApplyTileEntries; ++k) {
                if (cl[k] != t || off[k] >= len) continue;
                sum[off[k]] = sum[off[k]] + val[k];
                atomicOr(&touched[off[k] >> 5], 1u << (off[k] & 31u));
            }
        }
    }
    __syncthreads();  // every sum complete
#pragma unroll
    for (int r = 0; r < kApplyTileVecs; ++r) {
        const uint32_t v = (uint32_t)tid + (uint32_t)r * kApplyTileThreads;
        const uint32_t nib = (touched[v >> 3] >> ((v & 7u) * 4u)) & 0xFu;  // parameters 4v .. 4v + 3
        if (nib == 0) continue;
        const f4 s = reinterpret_cast<const f4*>(sum)[v];
        f4 x = pv[r];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if ((nib >> q) & 1u) {
                const float step = a.lr * s[q];
                x[q] = x[q] - step;
            }
        }
        if (whole) {
            *reinterpret_cast<f4*>(a.p + i_lo + 4u * v) = x;
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (4u * v + q < len) a.p[i_lo + 4u * v + q] = x[q];
        }
    }
}

// Form of later applies (a test hook): 0 chosen per call, 1 scattered, 2
// streaming wherever the parameters are 16-byte aligned.
static std::atomic<int> g_apply_form{0};

// The streaming form's bounds table is kept per device and stream, and reused
// by later calls on the same stream: work on one stream runs in order, so a
// call's bounds pass cannot overwrite the table while an earlier call on that
// stream still reads it, and calls on different streams use different tables.
// (A per-call allocation in stream order from a memory pool, or an event
// ordering the calls of all streams on one table, each cost about 5-6 us per
// call.)  The per-thread default stream is one stream per host thread, so
// its tables are kept per thread.  The mutex also keeps the two launches of
// one call together when host threads share a stream.  A table grows when a
// call needs more (hipFree of the old one waits for the device) and is kept
// until the process ends.
struct TableKey {
    int dev;
    uintptr_t stream;
    std::thread::id thread;
    bool operator<(const TableKey& o) const {
        if (dev != o.dev) return dev < o.dev;
        if (stream != o.stream) return stream < o.stream;
        return thread < o.thread;
    }
};
static std::mutex g_tab_mu;
static std::map<TableKey, std::pair<void*, size_t>> g_tables;

// The table of the current device and stream st, at least `bytes` long, or
// null if it cannot be allocated.  Called with g_tab_mu held.
static uint32_t* stream_table(hipStream_t st, size_t bytes) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return nullptr;
    const TableKey key{dev, reinterpret_cast<uintptr_t>(st), st == hipStreamPerThread ? std::this_thread::get_id() : std::thread::id()};
    auto& slot = g_tables[key];
    if (slot.second < bytes) {
        if (slot.first) (void)hipFree(slot.first);
        slot = {nullptr, 0};
        const size_t want = (bytes + 65535u) & ~(size_t)65535u;
        void* q = nullptr;
        if (hipMalloc(&q, want) != hipSuccess) return nullptr;
        slot = {q, want};
    }
    return static_cast<uint32_t*>(slot.first);
}

void set_apply_form(int form) { g_apply_form.store(form); }

hipError_t launch_apply(const ApplyArgs& a, uint32_t max_nnz, hipStream_t st) {
    if (a.C == 0 || max_nnz == 0 || a.n == 0) return hipSuccess;
    uint64_t total = 0;
    for (uint32_t c = 0; c < a.C; ++c) total += a.nnz[c];
    // Streaming reads every line of the shard: it pays once the entries touch
    // most lines (one entry per 64 parameters touches about 40% of them).
    // Each client adds a turn of barriers to every tile and a comparison to
    // every entry's client lookup, so many clients stay with the scattered
    // form unless the form is forced.
    const int form = g_apply_form.load();
    const bool aligned = (reinterpret_cast<uintptr_t>(a.p) & 15u) == 0;
    const bool dense = total * 64u >= a.n;
    const bool stream = aligned && form != 1 && (form == 2 || (dense && a.C <= 8u));
    if (stream) {
        const uint32_t tiles = (uint32_t)(((uint64_t)a.n + kApplyTileLen - 1) >> kApplyTileShift);
        std::lock_guard<std::mutex> lk(g_tab_mu);
        uint32_t* tab = stream_table(st, (size_t)a.C * (tiles + 1u) * sizeof(uint32_t));
        if (tab) {
            ApplyArgs b = a;
            b.tab = tab;
            b.tstride = tiles + 1u;
            uint64_t items = 0;  // head and tail, then the entries after the first
            for (uint32_t c = 0; c < a.C; ++c) items = std::max<uint64_t>(items, tiles + 1u + (a.nnz[c] ? a.nnz[c] - 1u : 0u));
            hipLaunchKernelGGL(k_apply_bounds, dim3((uint32_t)((items + kBlock - 1) / kBlock), a.C), dim3(kBlock), 0, st, b,
                               tiles);
            hipLaunchKernelGGL(k_apply_tile, dim3(tiles), dim3(kApplyTileThreads), 0, st, b);
            return hipGetLastError();
        }
        (void)hipGetLastError();  // no table: the scattered form below
    }
    const uint32_t buckets = (uint32_t)(((uint64_t)a.n + (1u << kApplyBucketShift) - 1) >> kApplyBucketShift);
    hipLaunchKernelGGL(k_apply, dim3(buckets), dim3(kBlock), 0, st, a);
    return hipGetLastError();
}

}  // namespace gd
