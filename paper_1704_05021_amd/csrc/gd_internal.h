// Host-side state of a gd_ctx: layout tables and device scratch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "gd.h"
#include "gd_device.hpp"

namespace gd {

// Decomposition of the flat gradient, fixed at gd_create:
//  * unit u: elements [1024u, 1024u + 1024) (the last one may be shorter),
//    one block of the dense pass; its candidates go to slots[1024u ...].
//  * tile: up to kTile consecutive candidates of one tensor, one wave of the
//    candidate passes (at most `max_tiles` of them).
struct Tables {
    uint32_t* unit_info = nullptr;         // [C] tensor of the first element | holds-a-tensor-start << 31
    uint32_t* tensor_off = nullptr;        // [T + 1] element offsets (u32)
    uint32_t* global_off = nullptr;        // [2] = {0, N}
    uint32_t* skey_base_tensor = nullptr;  // [T + 1] sample-key offsets per tensor segment
    uint32_t* skey_base_global = nullptr;  // [2]
};

struct Scratch {
    uint2* slots = nullptr;          // [C * 1024] candidates (index, value bits) of unit u at [1024u, ...)
    uint32_t* cnt = nullptr;         // [C] candidates per unit
    uint32_t* split = nullptr;       // [T] candidates of a tensor's first unit before the tensor
    uint32_t* loc = nullptr;         // [C] candidate offset of each unit inside its scan block
    uint32_t* neloc = nullptr;       // [C] non-empty unit index inside its scan block
    uint32_t* btot = nullptr;        // [scan blocks]
    uint32_t* betot = nullptr;       // [scan blocks]
    uint32_t* boff = nullptr;        // [scan blocks]
    uint32_t* beoff = nullptr;       // [scan blocks]
    uint32_t* ne_unit = nullptr;     // [C] non-empty units in order
    uint32_t* ne_off = nullptr;      // [C + 1] their first candidate (dense-pass order)
    uint32_t* num_ne = nullptr;      // [1]
    uint32_t* raw_tbase = nullptr;   // [T + 1]
    uint32_t* cand_idx = nullptr;    // [max(N,1)] candidates in ascending index order
    uint32_t* cand_val = nullptr;    // [max(N,1)] their value bits
    uint32_t* ten_cbase = nullptr;   // [T + 1] first compact candidate of each tensor
    uint32_t* tile_base = nullptr;   // [T + 1] first tile of each tensor
    uint32_t* tile_desc = nullptr;   // [max_tiles * kTileDescWords]
    uint32_t* tile_gt = nullptr;     // [max_tiles]
    uint32_t* tile_eq = nullptr;     // [max_tiles]
    uint32_t* grp_gt = nullptr;      // [max_tiles / kGroupTiles + 1]
    uint32_t* grp_eq = nullptr;
    double* tile_q = nullptr;        // [max_tiles * 4] kept positive sum, negative sum, counts
    uint32_t* flags = nullptr;       // [4] device flags (0: some bracket missed)
    uint32_t* hist = nullptr;        // [S_max * kHistWords]
    SegState* seg = nullptr;         // [S_max]
    uint64_t* out_base = nullptr;    // [S_max] first output slot of each segment
    uint16_t* skeys = nullptr;       // 16-bit sample keys
    uint32_t* shist = nullptr;       // [S_max * kSHistWords] sample histograms, kept zero between calls
    uint32_t* qbase = nullptr;       // [T + 1] first output slot of each tensor
    uint32_t* sshist = nullptr;      // [S_max * kSsCopies * kSsNB0] sampled mode: top-digit histograms
};

// Column-wise centres: each tensor's matrix view and the per-column sums.
struct ColumnTables {
    uint32_t* columns = nullptr;  // [T]
    uint32_t* colbase = nullptr;  // [T + 1] first column group of each tensor
    double* csum = nullptr;       // [2 * groups] positive and negative sums
    uint32_t* ccnt = nullptr;     // [2 * groups] positive and negative counts
    uint32_t groups = 0;
};

}  // namespace gd

struct gd_ctx;

namespace gd {

// The launch sequence of one exact-threshold compression (sample, bracket,
// dense pass, candidate passes, quantisation) on the tables and scratch ctx
// points to, after the caller's argument checks; k_total is the output size.
gd_status compress_exact(gd_ctx* ctx, const float* grad, const float* base, float* residual, double drop_ratio,
                         bool per, gd_quant quant, uint64_t k_total, const gd_sparse* out, hipStream_t st);

}  // namespace gd

struct gd_ctx {
    int device = 0;
    uint32_t T = 0;
    uint64_t N = 0;
    std::vector<uint64_t> offsets;
    uint32_t num_units = 0;
    uint32_t max_tiles = 0;
    uint32_t skeys_tensor = 0;
    uint32_t skeys_global = 0;
    gd::Tables tab;
    gd::Scratch scr;
    gd::ColumnTables cols;
    std::vector<void*> allocations;
    uint32_t debug_bracket = 0;
    uint32_t profile_every = 0;  // time dense launches 0, every, 2 * every, ... (0: off)
    std::vector<hipEvent_t> events;  // pairs
    size_t events_used = 0;
    uint64_t dense_launches = 0;
};
