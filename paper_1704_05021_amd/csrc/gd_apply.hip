// Server-side apply of sparse pushes to a parameter shard (Section 3: each
// server owns a shard of the parameters and receives the clients' pieces).
//
// For an index pushed by several clients the values are summed in client
// order starting from +0, and the parameter is updated once:
// p[i] -= lr * s[i].  The lowest client holding an index owns it: it finds
// the index in the later clients' (ascending) lists through a window of
// their indices staged in LDS, sums, and writes.  No atomics, so the result
// is deterministic.

#include "gd_kernels.h"

namespace gd {

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

hipError_t launch_apply(const ApplyArgs& a, uint32_t max_nnz, hipStream_t st) {
    if (a.C == 0 || max_nnz == 0) return hipSuccess;
    dim3 grid((max_nnz + kBlock - 1) / kBlock, a.C);
    hipLaunchKernelGGL(k_apply, grid, dim3(kBlock), 0, st, a);
    return hipGetLastError();
}

}  // namespace gd
