// Kernel argument blocks and launchers (host + device visible).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gd_device.hpp"

namespace gd {

// Host-forced brackets, to exercise the paths a real sample rarely takes.
constexpr uint32_t kDebugLoTooHigh = 1;  // no candidates: every segment takes the fallback
constexpr uint32_t kDebugHiAtLo = 2;     // zero every candidate in the dense pass
constexpr uint32_t kDebugLoZero = 3;     // every element is a candidate

struct SampleArgs {
    const float* grad;
    const float* base;  // nullable
    const float* res;
    const uint32_t* seg_off;    // [S + 1]
    const uint32_t* skey_base;  // [S + 1]
    uint32_t S;
    uint32_t T;
    uint32_t keep_ppm;
    uint32_t debug_bracket;  // 0, or a kDebug* override of the sampled bracket
    uint32_t* skeys;
    uint32_t* seg_done;
    SegState* seg;
    uint32_t* hist;
    uint64_t* out_base;
    uint32_t* tensor_counts;
};

struct DenseArgs {
    const float* grad;
    const float* base;  // nullable
    float* res;
    const uint32_t* chunk_start;
    const uint32_t* chunk_len;
    const uint32_t* chunk_tensor;
    uint32_t num_chunks;
    uint32_t per_tensor;
    SegState* seg;
    uint32_t* hist;
    uint2* slots;
    uint32_t* cnt_lo;
    uint32_t* cnt_hi;
};

struct CandArgs {
    float* res;
    const uint32_t* chunk_start;
    const uint32_t* chunk_len;
    const uint32_t* chunk_tensor;
    const uint32_t* group_chunk0;
    const uint32_t* group_tensor;
    const uint32_t* tensor_group0;
    const uint32_t* seg_off;
    uint32_t num_chunks;
    uint32_t num_groups;
    uint32_t per_tensor;
    uint32_t keep_ppm;
    SegState* seg;
    uint32_t* hist;
    uint2* slots;
    uint32_t* cnt_lo;
    uint32_t* grp_gt;
    uint32_t* grp_eq;
    double* grp_q;
    const uint64_t* out_base;
};

struct EmitArgs {
    uint32_t* idx;
    float* val;
    uint32_t* tensor_counts;
    uint64_t capacity;
};

struct QuantArgs {
    float* res;
    const uint32_t* idx;
    const float* val;
    uint32_t* sign_bits;
    float* means;
    const uint32_t* tensor_counts;
    const uint32_t* tensor_group0;
    const double* grp_q;
    uint32_t* qbase;
    uint32_t T;
    uint32_t N;
    uint64_t k_total;
};

constexpr uint32_t kMaxPushes = 64;

struct ApplyArgs {
    float* p;
    uint32_t n;
    uint32_t C;
    float lr;
    const uint32_t* idx[kMaxPushes];
    const float* val[kMaxPushes];
    uint32_t nnz[kMaxPushes];
};

hipError_t launch_sample(const SampleArgs& a, bool has_base, hipStream_t st);
hipError_t launch_dense(const DenseArgs& a, bool has_base, hipStream_t st);
hipError_t launch_candidates(const CandArgs& a, const EmitArgs& o, bool quant, hipStream_t st);
hipError_t launch_quant(const QuantArgs& q, hipStream_t st);
hipError_t launch_apply(const ApplyArgs& a, uint32_t max_nnz, hipStream_t st);

}  // namespace gd
