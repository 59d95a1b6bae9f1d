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
constexpr uint32_t kDebugLoAtHi = 4;     // candidates only above the estimate, all zeroed: most segments miss

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
    uint32_t* shist;  // [S * kSHistWords], zero on entry; k_bracket clears it again
    SegState* seg;
    uint32_t* hist;
    uint64_t* out_base;
    uint32_t* tensor_counts;
};

// Sampled-threshold mode (Section 4: selection on a sample of the gradient).
struct SampledArgs {
    const float* grad;
    const float* base;  // nullable
    const float* res;
    const uint32_t* seg_off;  // [S + 1]
    uint32_t S;
    uint32_t T;
    uint32_t per_tensor;
    uint32_t keep_ppm;
    uint32_t sample_ppm;  // 1 .. 1e6
    uint64_t seed;
    uint32_t* skeys;   // [N] sample keys of segment s at [seg_off[s], ...)
    uint32_t* sshist;  // [S * kSsCopies * kSsNB0] top-digit histograms, zero on entry; k_sselect clears them
    SegState* seg;
    uint32_t* tensor_counts;
};

struct DenseArgs {
    const float* grad;
    const float* base;  // nullable
    float* res;
    const uint32_t* unit_info;   // [C] tensor of the unit's first element | (holds a tensor start) << 31
    const uint32_t* tensor_off;  // [T + 1]
    uint32_t num_units;
    uint32_t N;
    uint32_t T;
    uint32_t per_tensor;
    const SegState* seg;
    uint2* slots;                // [C * 1024] candidates of unit u at [1024u, ...), ascending index
    uint32_t* cnt;               // [C] candidates of each unit
    uint32_t* split;             // [T] candidates of a tensor's first unit that precede the tensor
};

constexpr uint32_t kTile = 1024;        // candidates per tile of the candidate passes
constexpr uint32_t kTileDescWords = 12;  // words of a tile descriptor (three 16-byte loads)
constexpr uint32_t kTileBlocks = 512;   // most blocks a candidate pass launches (4 waves each)
// A segment of more than kBigSegTiles tiles also keeps per-group sums of its
// tiles' counts (groups of kGroupTiles consecutive tiles), so that a tile's
// prefix over the earlier tiles of its segment costs about
// tiles / kGroupTiles + kGroupTiles loads instead of one per earlier tile.
constexpr uint32_t kGroupTiles = 256;
constexpr uint32_t kBigSegTiles = 4096;

struct CandArgs {
    float* res;
    const uint32_t* unit_info;      // [C]
    const uint32_t* tensor_off;     // [T + 1] element offsets
    const uint32_t* seg_off;
    uint32_t num_units;
    uint32_t N;
    uint32_t T;
    uint32_t per_tensor;
    uint32_t keep_ppm;
    SegState* seg;
    uint32_t* hist;
    const uint2* slots;
    const uint32_t* cnt;    // [C]
    const uint32_t* split;  // [T]
    uint32_t* loc;        // [C] candidate offset of each unit inside its scan block
    uint32_t* neloc;      // [C] index of each non-empty unit inside its scan block
    uint32_t* btot;       // [scan blocks] candidates per scan block
    uint32_t* betot;      // [scan blocks] non-empty units per scan block
    uint32_t* boff;       // [scan blocks] first candidate of each scan block
    uint32_t* beoff;      // [scan blocks] first non-empty unit of each scan block
    uint32_t* ne_unit;    // [C] the non-empty units, in order
    uint32_t* ne_off;     // [C + 1] their first candidate (dense-pass order); [count] = total
    uint32_t* num_ne;     // [1] number of non-empty units
    uint32_t* raw_tbase;  // [T + 1] first candidate of each tensor (dense-pass order)
    uint32_t* cand_idx;   // [N] compact candidates, ascending flat index
    uint32_t* cand_val;   // [N] their value bits
    uint32_t* ten_cbase;  // [T + 1] first compact candidate of each tensor
    uint32_t* tile_base;  // [T + 1] first tile of each tensor
    uint32_t* tile_desc;  // [max_tiles * kTileDescWords] per tile, written by the layout pass: see TileView
    uint32_t max_tiles;   // descriptors the buffer holds (every element a candidate)
    uint32_t* tile_gt;    // [max tiles]
    uint32_t* tile_eq;
    uint32_t* grp_gt;     // [max tiles / kGroupTiles + 1] sums of tile_gt per group (segments of many tiles)
    uint32_t* grp_eq;     //   and of tile_eq; cleared by the layout pass
    double* tile_q;       // [max tiles * 4]
    uint64_t* out_base;   // [S] first output slot of each segment (the sampled mode writes it here)
    uint32_t* flags;      // [0]: some segment missed its bracket; [1]: some segment takes the zero mode
    uint32_t sampled;     // sampled threshold: every candidate is kept, no bracket can miss
    uint32_t zfill;       // 1: a segment short of nonzero keys may take the zero mode (any exact threshold)
    const float* pull_p;  // pull from the last pulled copy (res is then null): the parameters
    float* pull_copy;     //   and the copy, which takes the sent values
};

// 1-bit centres (Section 5.4): per-tensor sign means, the dropping threshold,
// one global average, or column-wise averages.
constexpr uint32_t kQuantSignMean = 1, kQuantThreshold = 2, kQuantGlobalMean = 3, kQuantColumnMean = 4;

struct EmitArgs {
    uint32_t* idx;
    float* val;
    uint32_t* tensor_counts;
    uint64_t capacity;
    uint32_t qkind;             // 0 or a kQuant* kind
};

struct QuantArgs {
    float* res;
    const uint32_t* idx;
    const float* val;
    uint32_t* sign_bits;
    float* means;
    const uint32_t* tensor_counts;
    const uint32_t* tile_base;
    const uint32_t* ten_cbase;  // [T + 1] first candidate of each tensor (zero mode: kept zeros = count - candidates)
    const double* tile_q;
    uint32_t* qbase;
    uint32_t T;
    uint32_t N;
    uint64_t k_total;
    uint32_t qkind;
    uint32_t per_tensor;
    uint32_t keep_ppm;
    const uint32_t* seg_off;    // [S + 1]
    const uint32_t* tensor_off; // [T + 1]
    const SegState* seg;
    const uint32_t* columns;
    const uint32_t* colbase;
    uint32_t sampled;           // 1 under a sampled threshold: the count is k_total at most, qbase[T] exactly
    uint32_t groups;            // column groups (column-wise centres)
    double* csum;               // [2 * groups] column sums (positive, negative), zero on entry, cleared after use
    uint32_t* ccnt;             // [2 * groups] column counts, likewise
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
    // quantised pushes (qkind 1..4): values decoded from sign bits and centre
    // pairs per tensor or per column of the layout below
    uint32_t qkind;
    const uint32_t* bits[kMaxPushes];
    const float* means[kMaxPushes];
    const uint32_t* tensor_off;  // [T + 1]
    uint32_t T;
    const uint32_t* columns;     // [T]
    const uint32_t* colbase;     // [T + 1]
    // streaming form: first position in each client's list of every tile
    // boundary (row c at tab + c * tstride)
    const uint32_t* tab;
    uint32_t tstride;
};

hipError_t launch_sample(const SampleArgs& a, bool has_base, hipStream_t st);
hipError_t launch_sampled(const SampledArgs& a, bool has_base, uint32_t max_samples, hipStream_t st);
hipError_t launch_layout(const CandArgs& a, hipStream_t st);
hipError_t launch_dense(const DenseArgs& a, bool has_base, hipStream_t st, hipEvent_t t0 = nullptr,
                        hipEvent_t t1 = nullptr);
hipError_t launch_candidates(const CandArgs& a, const EmitArgs& o, bool quant, uint32_t max_tiles, hipStream_t st);
hipError_t launch_quant(const QuantArgs& q, hipStream_t st);
hipError_t launch_apply(const ApplyArgs& a, uint32_t max_nnz, hipStream_t st);
// Form of later applies: 0 chosen per call, 1 scattered, 2 streaming wherever the parameters are 16-byte aligned.
void set_apply_form(int form);

}  // namespace gd
