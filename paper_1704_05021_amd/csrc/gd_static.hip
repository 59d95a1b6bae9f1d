// gd_compress_static: the exact compressor of gd_compress for callers that
// cannot allocate device memory.  It takes the layout per call instead of a
// context, and runs the same kernels on a fixed scratch array compiled into
// the library (one copy per GPU, held until the process ends).
//
// Host code never passes the array's name to a kernel or a copy: in host code
// that name is only a stand-in for the device symbol.  The first call on each
// device looks up that device's copy with hipGetSymbolAddress, and every later
// use goes through the address kept for the device.  A small set-up kernel
// then writes the layout tables into the array and clears the state the
// passes expect to start at zero, so the array may hold anything from an
// earlier call, of any layout.  Nothing is allocated: no hipMalloc, no host
// heap, no memset node.

#include <cmath>
#include <cstring>
#include <mutex>

#include "gd.h"
#include "gd_internal.h"
#include "gd_kernels.h"

namespace gd {

constexpr uint64_t kStaticMaxN = 1ull << 21;  // elements of the layout (2,097,152)
constexpr uint32_t kStaticMaxT = 64;          // tensors of the layout
constexpr size_t kStaticBytes = 48ull << 20;  // the scratch array: 48 MiB per GPU
constexpr int kStaticMaxDevices = 64;

// Every gd_compress_static call on a device shares that device's copy.
static __device__ __align__(256) unsigned char scratch[kStaticBytes];

namespace {

std::mutex g_scratch_mu;
void* g_scratch_ptr[kStaticMaxDevices] = {};

// This device's copy of the scratch array, looked up once per device.
hipError_t scratch_for(int dev, unsigned char** out) {
    if (dev < 0 || dev >= kStaticMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = static_cast<unsigned char*>(g_scratch_ptr[dev]);
    return hipSuccess;
}

// Hands out 256-byte aligned pieces of the array.  With base == nullptr it
// only measures (the pointers are then offsets and must not be used).
struct Carver {
    unsigned char* base;
    size_t used = 0;
    template <typename T>
    T* take(size_t count) {
        used = (used + 255) & ~(size_t)255;
        T* p = reinterpret_cast<T*>(base + used);
        used += (count ? count : 1) * sizeof(T);
        return p;
    }
};

// Sample keys stored for a segment [a, b): 16 per sample unit.
uint32_t sample_keys(uint64_t a, uint64_t b) {
    if (b <= a) return 0;
    const uint64_t n16 = ((b - 1) >> 4) - (a >> 4) + 1;
    return (uint32_t)kUnit * sample_unit_count((uint32_t)n16);
}

// Points ctx's tables and scratch into the array at base; returns the bytes
// used.  The sizes follow gd_create's for the same layout, except that the
// sampled mode's histograms and the column tables are left out.
size_t carve(gd_ctx& ctx, unsigned char* base) {
    Carver c{base};
    const uint32_t C = ctx.num_units, T = ctx.T, MT = ctx.max_tiles;
    const uint32_t sb = (C + kScanUnits - 1) / kScanUnits;
    ctx.tab.unit_info = c.take<uint32_t>(C);
    ctx.tab.tensor_off = c.take<uint32_t>(T + 1);
    ctx.tab.global_off = c.take<uint32_t>(2);
    ctx.tab.skey_base_tensor = c.take<uint32_t>(T + 1);
    ctx.tab.skey_base_global = c.take<uint32_t>(2);
    ctx.scr.slots = c.take<uint2>((size_t)C * kUnitLen);
    ctx.scr.cnt = c.take<uint32_t>(C);
    ctx.scr.split = c.take<uint32_t>(T);
    ctx.scr.loc = c.take<uint32_t>(C);
    ctx.scr.neloc = c.take<uint32_t>(C);
    ctx.scr.btot = c.take<uint32_t>(sb);
    ctx.scr.betot = c.take<uint32_t>(sb);
    ctx.scr.boff = c.take<uint32_t>(sb);
    ctx.scr.beoff = c.take<uint32_t>(sb);
    ctx.scr.ne_unit = c.take<uint32_t>(C);
    ctx.scr.ne_off = c.take<uint32_t>((size_t)C + 1);
    ctx.scr.num_ne = c.take<uint32_t>(1);
    ctx.scr.raw_tbase = c.take<uint32_t>(T + 1);
    ctx.scr.cand_idx = c.take<uint32_t>(ctx.N);
    ctx.scr.cand_val = c.take<uint32_t>(ctx.N);
    ctx.scr.ten_cbase = c.take<uint32_t>(T + 1);
    ctx.scr.tile_base = c.take<uint32_t>(T + 1);
    ctx.scr.tile_desc = c.take<uint32_t>((size_t)MT * kTileDescWords);
    ctx.scr.tile_gt = c.take<uint32_t>(MT);
    ctx.scr.tile_eq = c.take<uint32_t>(MT);
    ctx.scr.grp_gt = c.take<uint32_t>(MT / kGroupTiles + 1);
    ctx.scr.grp_eq = c.take<uint32_t>(MT / kGroupTiles + 1);
    ctx.scr.tile_q = c.take<double>(4 * (size_t)MT);
    ctx.scr.flags = c.take<uint32_t>(4);
    ctx.scr.hist = c.take<uint32_t>((size_t)T * kHistWords);
    ctx.scr.seg = c.take<SegState>(T);
    ctx.scr.out_base = c.take<uint64_t>(T);
    ctx.scr.skeys = c.take<uint16_t>(ctx.skeys_tensor > ctx.skeys_global ? ctx.skeys_tensor : ctx.skeys_global);
    ctx.scr.qbase = c.take<uint32_t>(T + 1);
    ctx.scr.shist = c.take<uint32_t>((size_t)T * kSHistWords);
    ctx.scr.sshist = nullptr;
    return c.used;
}

struct SetupArgs {
    uint32_t off[kStaticMaxT + 1];
    uint32_t T, N, C;
    uint32_t* unit_info;
    uint32_t* tensor_off;
    uint32_t* global_off;
    uint32_t* skey_base_tensor;
    uint32_t* skey_base_global;
    uint32_t* seg_words;  // T * 16 words of SegState
    uint32_t* shist;      // T * kSHistWords
    uint32_t* ten_cbase;
    uint32_t* tile_base;
    uint32_t* qbase;
};

__device__ __forceinline__ uint32_t sample_keys_dev(uint32_t a, uint32_t b) {
    if (b <= a) return 0;
    return (uint32_t)kUnit * sample_unit_count(((b - 1) >> 4) - (a >> 4) + 1);
}

// The layout tables gd_create would upload, and the state that starts at
// zero.  One thread per unit or cleared word; thread 0 also scans the
// sample-key bases (at most 64 tensors).
__global__ __launch_bounds__(kBlock) void k_static_setup(SetupArgs a) {
    const uint32_t g = blockIdx.x * kBlock + threadIdx.x;
    if (g < a.C) {
        // tensor of the unit's first element (the last t with off[t] <= start),
        // and whether another tensor starts strictly inside the unit
        const uint32_t us = g * kUnitLen, ue = a.N - us > kUnitLen ? us + kUnitLen : a.N;
        uint32_t t = 0;
        while (t + 1 < a.T && a.off[t + 1] <= us) ++t;
        bool inside = false;
        for (uint32_t x = t + 1; x < a.T && a.off[x] < ue; ++x) inside = inside || a.off[x] > us;
        a.unit_info[g] = t | (inside ? 0x80000000u : 0u);
    }
    if (g <= a.T) {
        a.tensor_off[g] = a.off[g];
        a.ten_cbase[g] = 0;
        a.tile_base[g] = 0;
        a.qbase[g] = 0;
    }
    if (g < 2) a.global_off[g] = g ? a.N : 0u;
    if (g < a.T * (uint32_t)(sizeof(SegState) / 4)) a.seg_words[g] = 0;
    if (g < a.T * (uint32_t)kSHistWords) a.shist[g] = 0;
    if (g == 0) {
        uint32_t acc = 0;
        for (uint32_t t = 0; t < a.T; ++t) {
            a.skey_base_tensor[t] = acc;
            acc += sample_keys_dev(a.off[t], a.off[t + 1]);
        }
        a.skey_base_tensor[a.T] = acc;
        a.skey_base_global[0] = 0;
        a.skey_base_global[1] = sample_keys_dev(0, a.N);
    }
}

uint64_t keep_of_host(uint64_t n, double drop_ratio) {
    return n * (uint64_t)std::llround((1.0 - drop_ratio) * 1e6) / 1000000ull;
}

template <typename E>
int enum_value(const E* e) {
    static_assert(sizeof(E) == sizeof(int), "C enums are int-sized");
    int v;
    std::memcpy(&v, e, sizeof v);
    return v;
}

}  // namespace
}  // namespace gd

extern "C" gd_status gd_compress_static(const uint64_t* off, uint32_t T, const float* grad, const float* base,
                                        float* residual, double drop_ratio, gd_threshold mode, gd_quant quant,
                                        const gd_sparse* out, void* stream) {
    using namespace gd;
    const int m = enum_value(&mode), q = enum_value(&quant);
    if (m != GD_GLOBAL && m != GD_PER_TENSOR) return GD_ERR_ARG;
    if (q < GD_QUANT_NONE || q > GD_QUANT_GLOBAL_MEAN) return GD_ERR_ARG;  // no column view here
    if (!(drop_ratio >= 0.0 && drop_ratio <= 1.0)) return GD_ERR_ARG;
    if (!off || T == 0 || !out) return GD_ERR_ARG;
    if (T > kStaticMaxT || off[0] != 0) return GD_ERR_LAYOUT;
    for (uint32_t t = 0; t < T; ++t)
        if (off[t + 1] < off[t]) return GD_ERR_LAYOUT;
    const uint64_t N = off[T];
    if (N > kStaticMaxN) return GD_ERR_LAYOUT;
    if (N > 0 && (!grad || !residual)) return GD_ERR_ARG;
    if (!out->idx || !out->val || !out->tensor_counts) return GD_ERR_ARG;
    if (q != GD_QUANT_NONE && (!out->sign_bits || !out->means)) return GD_ERR_ARG;
    if (((uintptr_t)grad & 15u) || ((uintptr_t)residual & 15u) || ((uintptr_t)base & 15u)) return GD_ERR_ALIGN;
    const bool per = m == GD_PER_TENSOR;
    uint64_t k_total = 0;
    if (per) {
        for (uint32_t t = 0; t < T; ++t) k_total += keep_of_host(off[t + 1] - off[t], drop_ratio);
    } else {
        k_total = keep_of_host(N, drop_ratio);
    }
    if (out->capacity < k_total) return GD_ERR_CAPACITY;

    // the layout as gd_create describes it, without its host tables
    gd_ctx ctx;
    ctx.T = T;
    ctx.N = N;
    ctx.num_units = (uint32_t)((N + kUnitLen - 1) / kUnitLen);
    uint64_t tiles = 0;
    uint32_t sk = 0;
    for (uint32_t t = 0; t < T; ++t) {
        tiles += (off[t + 1] - off[t] + kTile - 1) / kTile;
        sk += sample_keys(off[t], off[t + 1]);
    }
    ctx.max_tiles = (uint32_t)tiles;
    ctx.skeys_tensor = sk;
    ctx.skeys_global = sample_keys(0, N);
    if (carve(ctx, nullptr) > kStaticBytes) return GD_ERR_LAYOUT;  // cannot happen within the limits above

    if (hipGetDevice(&ctx.device) != hipSuccess) return GD_ERR_HIP;
    unsigned char* mem = nullptr;
    if (scratch_for(ctx.device, &mem) != hipSuccess) return GD_ERR_HIP;
    carve(ctx, mem);

    SetupArgs sa{};
    for (uint32_t t = 0; t <= T; ++t) sa.off[t] = (uint32_t)off[t];
    sa.T = T;
    sa.N = (uint32_t)N;
    sa.C = ctx.num_units;
    sa.unit_info = ctx.tab.unit_info;
    sa.tensor_off = ctx.tab.tensor_off;
    sa.global_off = ctx.tab.global_off;
    sa.skey_base_tensor = ctx.tab.skey_base_tensor;
    sa.skey_base_global = ctx.tab.skey_base_global;
    sa.seg_words = reinterpret_cast<uint32_t*>(ctx.scr.seg);
    sa.shist = ctx.scr.shist;
    sa.ten_cbase = ctx.scr.ten_cbase;
    sa.tile_base = ctx.scr.tile_base;
    sa.qbase = ctx.scr.qbase;
    uint32_t work = sa.C;
    if (T * (uint32_t)kSHistWords > work) work = T * (uint32_t)kSHistWords;
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(k_static_setup, dim3((work + kBlock - 1) / kBlock), dim3(kBlock), 0, st, sa);
    if (hipGetLastError() != hipSuccess) return GD_ERR_HIP;
    return compress_exact(&ctx, grad, base, residual, drop_ratio, per, quant, k_total, out, st);
}
