// 1-bit quantisation of the kept values (Section 5.4), with the
// quantisation error fed back into the residual (gfx950, wave64).
//
// After dropping, each kept value is replaced by one of two centres, chosen by
// its sign (values not below zero are positive).  Section 5.4 compares
// several ways of choosing the centres; all four are here:
//   sign mean    : per tensor, the average of its kept positive values and of
//                  its kept negative values;
//   threshold    : +-T, T the dropping threshold, i.e. the smallest kept
//                  magnitude of the threshold segment;
//   global mean  : one positive and one negative average over every kept
//                  value of the call;
//   column mean  : per column of each tensor's row-major matrix view.
// Per-tensor and global sums are taken in fp64 in a fixed order (per
// candidate tile, then tiles in order), so they are deterministic; column
// sums are fp64 atomics over the sent entries (in LDS per slice, then once
// per touched column).  The sent bits are packed LSB-first, 32 per word,
// and residual[idx] becomes acc - centre.

#include "gd_kernels.h"

namespace gd {

constexpr uint32_t kColSlice = 4096;  // sent entries per column-sum block
constexpr int kColLds = 2048;         // most columns a block sums in LDS (48 KB)

// Zeros tensor u keeps in the zero mode (every candidate kept, plus zeros):
// its kept count less its candidates; 0 outside the zero mode.
__device__ __forceinline__ uint32_t zeros_kept(const QuantArgs& q, uint32_t u) {
    return q.seg[q.per_tensor ? u : 0u].zero ? q.tensor_counts[u] - (q.ten_cbase[u + 1] - q.ten_cbase[u]) : 0u;
}

// Centres per tensor (every kind but the column mean) and the first output
// slot of each tensor.  One wave per tensor.
__global__ __launch_bounds__(kBlock) void k_means(QuantArgs q) {
    const int w = threadIdx.x >> 6, lane = lane_id();
    const uint32_t t = blockIdx.x * kWavesPerBlock + w;
    if (t >= q.T) return;
    uint32_t before = 0;
    for (uint32_t u = lane; u < t; u += kWave) before += q.tensor_counts[u];
    before = wave_sum(before);
    if (lane == 0) {
        q.qbase[t] = before;
        if (t + 1 == q.T) q.qbase[q.T] = before + q.tensor_counts[t];
    }
    if (q.qkind == kQuantColumnMean) return;
    float pos = 0.0f, neg = 0.0f;
    if (q.qkind == kQuantThreshold) {
        // the smallest kept magnitude of the segment: the exact threshold key,
        // or under a sampled threshold the smallest key sent, the minimum over
        // the segment's tiles
        const uint32_t s = q.per_tensor ? t : 0u;
        uint32_t key = kNoKey;
        if (q.sampled) {
            const uint32_t g0 = q.per_tensor ? q.tile_base[t] : 0u, g1 = q.per_tensor ? q.tile_base[t + 1] : q.tile_base[q.T];
            for (uint32_t g = g0 + lane; g < g1; g += kWave) {
                const uint32_t x = (uint32_t)q.tile_q[4 * (size_t)g + 0];
                key = x < key ? x : key;
            }
            key = wave_min(key);
        } else if (keep_of(q.seg_off[s + 1] - q.seg_off[s], q.keep_ppm) > 0) {
            key = q.seg[s].zero ? 0u : q.seg[s].thr;  // zero mode: T = 0 (the count pass may see no tile)
        }
        if (key != kNoKey) {
            pos = __uint_as_float(key);
            neg = __uint_as_float(key | 0x80000000u);
        }
    } else {
        const bool global = q.qkind == kQuantGlobalMean;
        const uint32_t g0 = global ? 0u : q.tile_base[t], g1 = global ? q.tile_base[q.T] : q.tile_base[t + 1];
        double sp = 0.0, sn = 0.0, np = 0.0, nn = 0.0;
        for (uint32_t g = g0 + lane; g < g1; g += kWave) {
            sp += q.tile_q[4 * (size_t)g + 0];
            sn += q.tile_q[4 * (size_t)g + 1];
            np += q.tile_q[4 * (size_t)g + 2];
            nn += q.tile_q[4 * (size_t)g + 3];
        }
        sp = wave_sum(sp);
        sn = wave_sum(sn);
        np = wave_sum(np);
        nn = wave_sum(nn);
        // zero mode: the kept zeros are in no tile's sums; each counts as a
        // positive value (not below zero) and adds nothing to sp
        uint32_t zk = 0;
        if (global) {
            for (uint32_t u = lane; u < q.T; u += kWave) zk += zeros_kept(q, u);
        } else if (lane == 0) {
            zk = zeros_kept(q, t);
        }
        np += (double)wave_sum(zk);
        pos = np > 0.0 ? (float)(sp / np) : 0.0f;
        neg = nn > 0.0 ? (float)(sn / nn) : 0.0f;
    }
    if (lane == 0) {
        q.means[2 * t + 0] = pos;
        q.means[2 * t + 1] = neg;
    }
}

// Column sums of the sent entries, per sign.  Each block takes a slice of
// kColSlice consecutive output slots and walks the tensors it touches; for a
// tensor of at most kColLds columns it sums the slice in LDS first (fp64 LDS
// atomics) and then adds each touched column to the global sums once, so a
// column's global atomics number its tensor's slices rather than its entries.
// Wider tensors spread their entries over many columns and add directly.
__global__ __launch_bounds__(kBlock) void k_colsum(QuantArgs q) {
    __shared__ double ls[2 * kColLds];
    __shared__ uint32_t lc[2 * kColLds];
    const int tid = threadIdx.x;
    const uint32_t total = q.qbase[q.T];
    const uint64_t j0 = (uint64_t)blockIdx.x * kColSlice;
    if (j0 >= total) return;
    const uint32_t j1 = j0 + kColSlice < total ? (uint32_t)j0 + kColSlice : total;
    uint32_t lo = 0, hi = q.T;  // tensor of slot j0: the last t with qbase[t] <= j0
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (q.qbase[mid] <= j0) lo = mid;
        else hi = mid;
    }
    uint32_t t = lo;
    for (uint32_t j = (uint32_t)j0; j < j1;) {  // block-uniform walk over the tensors of the slice
        while (q.qbase[t + 1] <= j) ++t;
        const uint32_t e = q.qbase[t + 1] < j1 ? q.qbase[t + 1] : j1;
        const uint32_t C = q.columns[t], cb = 2 * q.colbase[t], off = q.tensor_off[t];
        const bool local = C <= (uint32_t)kColLds;
        if (local) {
            for (uint32_t i = tid; i < 2 * C; i += kBlock) {
                ls[i] = 0.0;
                lc[i] = 0;
            }
            __syncthreads();
        }
        for (uint32_t x = j + tid; x < e; x += kBlock) {
            const float v = q.val[x];
            const uint32_t sl = 2 * ((q.idx[x] - off) % C) + (v < 0.0f ? 1u : 0u);
            if (local) {
                unsafeAtomicAdd(&ls[sl], (double)v);
                atomicAdd(&lc[sl], 1u);
            } else {
                unsafeAtomicAdd(&q.csum[cb + sl], (double)v);
                atomicAdd(&q.ccnt[cb + sl], 1u);
            }
        }
        if (local) {
            __syncthreads();
            for (uint32_t i = tid; i < 2 * C; i += kBlock)
                if (lc[i]) {
                    unsafeAtomicAdd(&q.csum[cb + i], ls[i]);
                    atomicAdd(&q.ccnt[cb + i], lc[i]);
                }
            __syncthreads();
        }
        j = e;
    }
}

// Column-wise centres from the column sums, which are cleared for the next call.
__global__ __launch_bounds__(kBlock) void k_colmeans(QuantArgs q) {
    const uint32_t g = blockIdx.x * kBlock + threadIdx.x;
    if (g >= q.groups) return;
    const double sp = q.csum[2 * g + 0], sn = q.csum[2 * g + 1];
    const uint32_t np = q.ccnt[2 * g + 0], nn = q.ccnt[2 * g + 1];
    q.means[2 * g + 0] = np ? (float)(sp / (double)np) : 0.0f;
    q.means[2 * g + 1] = nn ? (float)(sn / (double)nn) : 0.0f;
    q.csum[2 * g + 0] = 0.0;
    q.csum[2 * g + 1] = 0.0;
    q.ccnt[2 * g + 0] = 0;
    q.ccnt[2 * g + 1] = 0;
}

__global__ __launch_bounds__(kBlock) void k_quant(QuantArgs q) {
    const uint64_t j = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
    const uint64_t total = q.qbase[q.T];  // entries sent (the grid covers k_total >= total)
    const bool valid = j < total;
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
        const uint32_t i = q.idx[j];
        const uint32_t g = q.qkind == kQuantColumnMean ? q.colbase[lo] + (i - q.tensor_off[lo]) % q.columns[lo] : lo;
        const float centre = neg ? q.means[2 * g + 1] : q.means[2 * g + 0];
        if (i < q.N) q.res[i] = x - centre;
    }
    const uint64_t m = ballot(valid && neg);
    const uint64_t jw = j - lane_id();  // first slot of this wave, a multiple of 64
    const uint64_t words = (total + 31) / 32;
    if (lane_id() == 0 && jw / 32 < words) q.sign_bits[jw / 32] = (uint32_t)m;
    if (lane_id() == 1 && jw / 32 + 1 < words) q.sign_bits[jw / 32 + 1] = (uint32_t)(m >> 32);
}

static inline uint32_t blocks_for_waves(uint32_t waves) { return (waves + kWavesPerBlock - 1) / kWavesPerBlock; }

hipError_t launch_quant(const QuantArgs& q, hipStream_t st) {
    hipLaunchKernelGGL(k_means, dim3(blocks_for_waves(q.T)), dim3(kBlock), 0, st, q);
    if (q.qkind == kQuantColumnMean && q.groups > 0) {
        if (q.k_total > 0)
            hipLaunchKernelGGL(k_colsum, dim3((uint32_t)((q.k_total + kColSlice - 1) / kColSlice)), dim3(kBlock), 0, st,
                               q);
        hipLaunchKernelGGL(k_colmeans, dim3((q.groups + kBlock - 1) / kBlock), dim3(kBlock), 0, st, q);
    }
    if (q.k_total > 0) {
        const uint64_t blocks = (q.k_total + kBlock - 1) / kBlock;
        hipLaunchKernelGGL(k_quant, dim3((uint32_t)blocks), dim3(kBlock), 0, st, q);
    }
    return hipGetLastError();
}

}  // namespace gd
