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
//  * group: up to `group_chunks` consecutive chunks of one tensor, processed
//    by one wave in the candidate passes.
struct Tables {
    uint32_t* chunk_start = nullptr;   // [C]
    uint32_t* chunk_len = nullptr;     // [C]
    uint32_t* chunk_tensor = nullptr;  // [C]
    uint32_t* group_chunk0 = nullptr;  // [NG + 1]
    uint32_t* group_tensor = nullptr;  // [NG]
    uint32_t* tensor_group0 = nullptr; // [T + 1]
    uint32_t* tensor_off = nullptr;    // [T + 1] element offsets (u32)
    uint32_t* global_off = nullptr;    // [2] = {0, N}
    uint32_t* skey_base_tensor = nullptr;  // [T + 1] sample-key offsets per tensor segment
    uint32_t* skey_base_global = nullptr;  // [2]
};

struct Scratch {
    uint2* slots = nullptr;         // [max(N,1)] candidate (index, value bits)
    uint32_t* cnt_lo = nullptr;     // [C] candidates per chunk
    uint32_t* cnt_hi = nullptr;     // [C] entries with key >= hi per chunk
    uint32_t* grp_gt = nullptr;     // [NG] candidates above the threshold per group
    uint32_t* grp_eq = nullptr;     // [NG] candidates equal to the threshold per group
    double* grp_q = nullptr;        // [NG * 4] kept positive sum, negative sum, counts
    uint32_t* hist = nullptr;       // [S_max * kHistWords]
    SegState* seg = nullptr;        // [S_max]
    uint64_t* out_base = nullptr;   // [S_max] first output slot of each segment
    uint32_t* skeys = nullptr;      // sample keys
    uint32_t* seg_done = nullptr;   // [S_max] completion counters of the sample kernel
    uint32_t* qbase = nullptr;      // [T + 1] first output slot of each tensor
};

}  // namespace gd

struct gd_ctx {
    int device = 0;
    uint32_t T = 0;
    uint64_t N = 0;
    std::vector<uint64_t> offsets;
    uint32_t chunk_len = 0;
    uint32_t group_chunks = 0;
    uint32_t num_chunks = 0;
    uint32_t num_groups = 0;
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
