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
    const uint32_t* skey_base;  // [S + 1] first sample key of each segment
    uint32_t S;
    uint32_t T;
    uint32_t keep_ppm;
    uint32_t debug_bracket;  // 0, or a kDebug* override of the sampled bracket
    uint16_t* skeys;
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
    const SegState* seg;
    uint2* slots;
    uint32_t* cnt_lo;
};

constexpr uint32_t kTile = 2048;        // candidates per tile of the candidate passes
constexpr uint32_t kTileBlocks = 2048;  // most blocks a candidate pass launches (4 waves each)

struct CandArgs {
    float* res;
    const uint32_t* chunk_start;
    const uint32_t* chunk_len;
    const uint32_t* chunk_tensor;
    const uint32_t* tensor_chunk0;  // [T + 1]
    const uint32_t* tensor_off;     // [T + 1] element offsets
    const uint32_t* seg_off;
    uint32_t num_chunks;
    uint32_t T;
    uint32_t per_tensor;
    uint32_t keep_ppm;
    SegState* seg;
    uint32_t* hist;
    uint2* slots;
    uint32_t* cnt_lo;
    uint32_t* loc;        // [C] candidate offset of each unit inside its scan block
    uint32_t* btot;       // [scan blocks] candidates per scan block
    uint32_t* boff;       // [scan blocks] first candidate of each scan block
    uint32_t* scan_done;  // completion counter of the scan blocks
    uint32_t* cand_off;   // [C + 1] first candidate of each unit (dense-pass order)
    uint32_t* raw_tbase;  // [T + 1] cand_off of each tensor's first unit
    uint2* cand;          // [N] compact candidates, ascending flat index
    uint32_t* ten_cbase;  // [T + 1] first compact candidate of each tensor
    uint32_t* tile_base;  // [T + 1] first tile of each tensor
    uint32_t* tile_unit0; // [max tiles] unit holding each tile's first candidate
    uint32_t* tile_gt;    // [max tiles]
    uint32_t* tile_eq;
    double* tile_q;       // [max tiles * 4]
    const uint64_t* out_base;
    uint32_t* flags;      // [0]: some segment missed its bracket
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
    const uint32_t* tile_base;
    const double* tile_q;
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
hipError_t launch_layout(const CandArgs& a, hipStream_t st);
hipError_t launch_dense(const DenseArgs& a, bool has_base, hipStream_t st);
hipError_t launch_candidates(const CandArgs& a, const EmitArgs& o, bool quant, uint32_t max_tiles, hipStream_t st);
hipError_t launch_quant(const QuantArgs& q, hipStream_t st);
hipError_t launch_apply(const ApplyArgs& a, uint32_t max_nnz, hipStream_t st);

}  // namespace gd
