// Host-side declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "gd_device.hpp"

namespace gd {

// Decomposition of the flat gradient, fixed at gd_create:
//  * chunk: up to `chunk_len` consecutive elements of one tensor, processed
//    by one wave in the dense pass; candidates of chunk c are stored at
//    slots[chunk_start[c] ...].
//  * tile: up to kTile consecutive candidates of one tensor, processed by one
//    wave in the candidate passes (at most `max_tiles` of them).
struct Tables {
    uint32_t* chunk_start = nullptr;   // [C]
    uint32_t* chunk_len = nullptr;     // [C]
    uint32_t* chunk_tensor = nullptr;  // [C]
    uint32_t* tensor_chunk0 = nullptr; // [T + 1]
    uint32_t* tensor_off = nullptr;    // [T + 1] element offsets (u32)
    uint32_t* global_off = nullptr;    // [2] = {0, N}
    uint32_t* skey_base_tensor = nullptr;  // [T + 1] sample-key offsets per tensor segment
    uint32_t* skey_base_global = nullptr;  // [2]
};

struct Scratch {
    uint2* slots = nullptr;         // [max(N,1)] candidate (index, value bits)
    uint32_t* cnt_lo = nullptr;     // [C] candidates per chunk
    uint32_t* tile_unit0 = nullptr; // [max_tiles] unit holding each tile's first candidate
    uint32_t* flags = nullptr;      // [4] device flags (0: some bracket missed)
    uint2* cand = nullptr;          // [max(N,1)] candidates in ascending index order
    uint32_t* cand_off = nullptr;   // [C + 1] first compact candidate of each chunk
    uint32_t* ten_cbase = nullptr;  // [T + 1] first compact candidate of each tensor
    uint32_t* tile_base = nullptr;  // [T + 1] first tile of each tensor
    uint32_t* tile_gt = nullptr;    // [max_tiles] candidates above the threshold per tile
    uint32_t* tile_eq = nullptr;    // [max_tiles] candidates equal to the threshold per tile
    double* tile_q = nullptr;       // [max_tiles * 4] kept positive sum, negative sum, counts
    uint32_t* hist = nullptr;       // [S_max * kHistWords]
    SegState* seg = nullptr;        // [S_max]
    uint64_t* out_base = nullptr;   // [S_max] first output slot of each segment
    uint16_t* skeys = nullptr;      // 16-bit sample keys
    uint32_t* loc = nullptr;        // [C] candidate offset of each unit inside its scan block
    uint32_t* btot = nullptr;       // [scan blocks]
    uint32_t* boff = nullptr;       // [scan blocks]
    uint32_t* scan_done = nullptr;  // [1] completion counter of the scan blocks
    uint32_t* raw_tbase = nullptr;  // [T + 1]
    uint32_t* qbase = nullptr;      // [T + 1] first output slot of each tensor
};

}  // namespace gd

struct gd_ctx {
    int device = 0;
    uint32_t T = 0;
    uint64_t N = 0;
    std::vector<uint64_t> offsets;
    uint32_t chunk_len = 0;
    uint32_t num_chunks = 0;
    uint32_t max_tiles = 0;
    uint32_t skeys_tensor = 0;
    uint32_t skeys_global = 0;
    gd::Tables tab;
    gd::Scratch scr;
    std::vector<void*> allocations;
    uint32_t debug_bracket = 0;
    bool profile = false;
    std::vector<hipEvent_t> events;  // pairs
    size_t events_used = 0;
    uint64_t dense_launches = 0;
};
