// C ABI of the gradient-dropping compressor: argument checks, layout tables,
// scratch ownership and the launch sequence.  The operations are defined in
// include/gd.h; the kernels' launchers are declared in gd_kernels.h.

#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <vector>

#include "gd.h"
#include "gd_internal.h"
#include "gd_kernels.h"

namespace {

using gd::kMaxUnits;
using gd::kUnit;

// Restores the caller's current device on scope exit.
struct DeviceGuard {
    int prev = -1;
    bool ok = false;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) return;
        ok = prev == dev || hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

uint64_t keep_ppm_of(double drop_ratio) { return (uint64_t)std::llround((1.0 - drop_ratio) * 1e6); }

// The integer a C caller passed for an enum parameter.  A C caller may pass
// any int; in C++ reading an enum object that holds a value outside the
// enumeration is undefined, so the bytes are copied out instead and checked
// as an int.
template <typename E>
int enum_int(const E* e) {
    static_assert(sizeof(E) == sizeof(int), "C enums are int-sized");
    int v;
    std::memcpy(&v, e, sizeof v);
    return v;
}
bool valid_mode(int m) { return m == GD_GLOBAL || m == GD_PER_TENSOR; }
bool valid_quant(int q) { return q >= GD_QUANT_NONE && q <= GD_QUANT_COLUMN_MEAN; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Units of 16 elements sampled for a segment [a, b) and the number of sample keys stored.
uint32_t sample_keys_for(uint64_t a, uint64_t b) {
    if (b <= a) return 0;
    const uint64_t n16 = ((b - 1) >> 4) - (a >> 4) + 1;
    return (uint32_t)kUnit * gd::sample_unit_count((uint32_t)n16);
}

template <typename T>
bool dev_alloc(gd_ctx* ctx, T** p, size_t count) {
    void* q = nullptr;
    if (hipMalloc(&q, std::max<size_t>(count, 1) * sizeof(T)) != hipSuccess) return false;
    ctx->allocations.push_back(q);
    *p = static_cast<T*>(q);
    return true;
}

template <typename T>
bool dev_upload(gd_ctx* ctx, T** p, const std::vector<T>& v) {
    if (!dev_alloc(ctx, p, v.size())) return false;
    if (v.empty()) return true;
    return hipMemcpy(*p, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice) == hipSuccess;
}

void free_all(gd_ctx* ctx) {
    for (void* p : ctx->allocations) (void)hipFree(p);
    ctx->allocations.clear();
    for (hipEvent_t e : ctx->events) (void)hipEventDestroy(e);
    ctx->events.clear();
}

// Column layout for the column-wise centres: the tables and the zeroed
// accumulators (two sums and two counts per column).  Replaces any earlier one.
bool set_columns(gd_ctx* ctx, const std::vector<uint32_t>& columns) {
    std::vector<uint32_t> colbase(ctx->T + 1, 0);
    for (uint32_t t = 0; t < ctx->T; ++t) colbase[t + 1] = colbase[t] + columns[t];
    const uint32_t groups = colbase[ctx->T];
    gd::ColumnTables c{};
    const size_t before = ctx->allocations.size();
    bool ok = dev_upload(ctx, &c.columns, columns) && dev_upload(ctx, &c.colbase, colbase) &&
              dev_alloc(ctx, &c.csum, 2 * (size_t)groups) && dev_alloc(ctx, &c.ccnt, 2 * (size_t)groups);
    ok = ok && hipMemset(c.csum, 0, 2 * (size_t)std::max<uint32_t>(groups, 1) * sizeof(double)) == hipSuccess &&
         hipMemset(c.ccnt, 0, 2 * (size_t)std::max<uint32_t>(groups, 1) * sizeof(uint32_t)) == hipSuccess &&
         hipDeviceSynchronize() == hipSuccess;
    if (!ok) {
        for (size_t i = before; i < ctx->allocations.size(); ++i) (void)hipFree(ctx->allocations[i]);
        ctx->allocations.resize(before);
        return false;
    }
    // the previous tables are freed
    for (void* p : {(void*)ctx->cols.columns, (void*)ctx->cols.colbase, (void*)ctx->cols.csum, (void*)ctx->cols.ccnt}) {
        if (!p) continue;
        auto it = std::find(ctx->allocations.begin(), ctx->allocations.end(), p);
        if (it != ctx->allocations.end()) {
            (void)hipFree(p);
            ctx->allocations.erase(it);
        }
    }
    c.groups = groups;
    ctx->cols = c;
    return true;
}

// The passes after the threshold bracket is set: the dense stream, the
// candidate layout, exact selection or plain compaction, and quantisation.
// k_total is the host-known output size (exact threshold), or under a sampled
// threshold the capacity, a bound the device-side count stays within.
gd_status run_after_bracket(gd_ctx* ctx, const float* grad, const float* base, float* residual, bool per,
                            uint32_t ppm, bool sampled, gd_quant quant, uint64_t k_total, const gd_sparse* out,
                            hipStream_t st) {
    const uint32_t* seg_off = per ? ctx->tab.tensor_off : ctx->tab.global_off;
    gd::DenseArgs da{};
    da.grad = grad;
    da.base = base;
    da.res = residual;
    da.unit_info = ctx->tab.unit_info;
    da.tensor_off = ctx->tab.tensor_off;
    da.num_units = ctx->num_units;
    da.N = (uint32_t)ctx->N;
    da.T = ctx->T;
    da.split = ctx->scr.split;
    da.per_tensor = per;
    da.seg = ctx->scr.seg;
    da.slots = ctx->scr.slots;
    da.cnt = ctx->scr.cnt;
    const bool timed = ctx->profile_every != 0 && ctx->dense_launches % ctx->profile_every == 0 &&
                       ctx->events_used + 2 <= ctx->events.size() && ctx->num_units > 0;
    hipEvent_t t0 = timed ? ctx->events[ctx->events_used] : nullptr;
    hipEvent_t t1 = timed ? ctx->events[ctx->events_used + 1] : nullptr;
    if (gd::launch_dense(da, base != nullptr, st, t0, t1) != hipSuccess) return GD_ERR_HIP;
    if (timed) ctx->events_used += 2;
    if (ctx->num_units > 0) ++ctx->dense_launches;

    gd::CandArgs ca{};
    ca.res = residual;
    ca.unit_info = ctx->tab.unit_info;
    ca.tensor_off = ctx->tab.tensor_off;
    ca.seg_off = seg_off;
    ca.num_units = ctx->num_units;
    ca.N = (uint32_t)ctx->N;
    ca.T = ctx->T;
    ca.per_tensor = per;
    ca.keep_ppm = ppm;
    ca.seg = ctx->scr.seg;
    ca.hist = ctx->scr.hist;
    ca.slots = ctx->scr.slots;
    ca.cnt = ctx->scr.cnt;
    ca.split = ctx->scr.split;
    ca.loc = ctx->scr.loc;
    ca.neloc = ctx->scr.neloc;
    ca.btot = ctx->scr.btot;
    ca.betot = ctx->scr.betot;
    ca.boff = ctx->scr.boff;
    ca.beoff = ctx->scr.beoff;
    ca.ne_unit = ctx->scr.ne_unit;
    ca.ne_off = ctx->scr.ne_off;
    ca.num_ne = ctx->scr.num_ne;
    ca.raw_tbase = ctx->scr.raw_tbase;
    ca.cand_idx = ctx->scr.cand_idx;
    ca.cand_val = ctx->scr.cand_val;
    ca.ten_cbase = ctx->scr.ten_cbase;
    ca.tile_base = ctx->scr.tile_base;
    ca.tile_desc = ctx->scr.tile_desc;
    ca.max_tiles = ctx->max_tiles;
    ca.flags = ctx->scr.flags;
    ca.tile_gt = ctx->scr.tile_gt;
    ca.tile_eq = ctx->scr.tile_eq;
    ca.grp_gt = ctx->scr.grp_gt;
    ca.grp_eq = ctx->scr.grp_eq;
    ca.tile_q = ctx->scr.tile_q;
    ca.out_base = ctx->scr.out_base;
    ca.sampled = sampled ? 1u : 0u;
    ca.zfill = sampled ? 0u : 1u;
    if (!residual) {  // a pull from the last pulled copy (base)
        ca.pull_p = grad;
        ca.pull_copy = const_cast<float*>(base);
    }
    gd::EmitArgs ea{};
    ea.idx = out->idx;
    ea.val = out->val;
    ea.tensor_counts = out->tensor_counts;
    ea.capacity = out->capacity;
    const bool q = quant != GD_QUANT_NONE;
    ea.qkind = (uint32_t)quant;
    if (gd::launch_layout(ca, st) != hipSuccess) return GD_ERR_HIP;
    if (gd::launch_candidates(ca, ea, q, ctx->max_tiles, st) != hipSuccess) return GD_ERR_HIP;

    if (q) {
        gd::QuantArgs qa{};
        qa.res = residual;
        qa.idx = out->idx;
        qa.val = out->val;
        qa.sign_bits = out->sign_bits;
        qa.means = out->means;
        qa.tensor_counts = out->tensor_counts;
        qa.tile_base = ctx->scr.tile_base;
        qa.ten_cbase = ctx->scr.ten_cbase;
        qa.tile_q = ctx->scr.tile_q;
        qa.qbase = ctx->scr.qbase;
        qa.T = ctx->T;
        qa.N = (uint32_t)ctx->N;
        qa.k_total = k_total;
        qa.qkind = (uint32_t)quant;
        qa.per_tensor = per;
        qa.keep_ppm = ppm;
        qa.seg_off = seg_off;
        qa.tensor_off = ctx->tab.tensor_off;
        qa.seg = ctx->scr.seg;
        qa.columns = ctx->cols.columns;
        qa.colbase = ctx->cols.colbase;
        qa.sampled = sampled ? 1u : 0u;
        qa.groups = ctx->cols.groups;
        qa.csum = ctx->cols.csum;
        qa.ccnt = ctx->cols.ccnt;
        if (gd::launch_quant(qa, st) != hipSuccess) return GD_ERR_HIP;
    }
    return GD_OK;
}

}  // namespace

namespace gd {

gd_status compress_exact(gd_ctx* ctx, const float* grad, const float* base, float* residual, double drop_ratio,
                         bool per, gd_quant quant, uint64_t k_total, const gd_sparse* out, hipStream_t st) {
    const uint32_t ppm = (uint32_t)keep_ppm_of(drop_ratio);
    SampleArgs sa{};
    sa.grad = grad;
    sa.base = base;
    sa.res = residual;
    sa.seg_off = per ? ctx->tab.tensor_off : ctx->tab.global_off;
    sa.skey_base = per ? ctx->tab.skey_base_tensor : ctx->tab.skey_base_global;
    sa.S = per ? ctx->T : 1u;
    sa.T = ctx->T;
    sa.keep_ppm = ppm;
    sa.debug_bracket = ctx->debug_bracket;
    sa.skeys = ctx->scr.skeys;
    sa.seg = ctx->scr.seg;
    sa.hist = ctx->scr.hist;
    sa.shist = ctx->scr.shist;
    sa.out_base = ctx->scr.out_base;
    sa.tensor_counts = out->tensor_counts;
    if (launch_sample(sa, base != nullptr, st) != hipSuccess) return GD_ERR_HIP;
    return run_after_bracket(ctx, grad, base, residual, per, ppm, false, quant, k_total, out, st);
}

}  // namespace gd

extern "C" {

const char* gd_status_string(gd_status status) {
    switch (enum_int(&status)) {
        case GD_OK: return "ok";
        case GD_ERR_ARG: return "invalid argument";
        case GD_ERR_LAYOUT: return "invalid tensor layout";
        case GD_ERR_CAPACITY: return "output capacity below the number of kept entries";
        case GD_ERR_ALIGN: return "buffer not 16-byte aligned";
        case GD_ERR_OOM: return "device allocation failed";
        case GD_ERR_HIP: return "HIP runtime or launch failure";
    }
    return "unknown status";
}

uint64_t gd_keep_count(uint64_t n, double drop_ratio) {
    if (!(drop_ratio >= 0.0 && drop_ratio <= 1.0)) return 0;
    return n * keep_ppm_of(drop_ratio) / 1000000ull;
}

uint64_t gd_keep_total(const gd_ctx* ctx, double drop_ratio, gd_threshold mode) {
    if (!ctx) return 0;
    if (enum_int(&mode) == GD_GLOBAL) return gd_keep_count(ctx->N, drop_ratio);
    uint64_t k = 0;
    for (uint32_t t = 0; t < ctx->T; ++t) k += gd_keep_count(ctx->offsets[t + 1] - ctx->offsets[t], drop_ratio);
    return k;
}

gd_status gd_create(gd_ctx** out, const uint64_t* off, uint32_t T) {
    if (!out) return GD_ERR_ARG;
    *out = nullptr;
    if (!off || T == 0) return GD_ERR_ARG;
    if (off[0] != 0) return GD_ERR_LAYOUT;
    for (uint32_t t = 0; t < T; ++t)
        if (off[t + 1] < off[t]) return GD_ERR_LAYOUT;
    const uint64_t N = off[T];
    if (N >= 0xFFFFFFFFull) return GD_ERR_LAYOUT;

    gd_ctx* ctx = new (std::nothrow) gd_ctx();
    if (!ctx) return GD_ERR_OOM;
    if (hipGetDevice(&ctx->device) != hipSuccess) {
        delete ctx;
        return GD_ERR_HIP;
    }
    ctx->T = T;
    ctx->N = N;
    ctx->offsets.assign(off, off + T + 1);

    // Units of the dense pass: the 1024-element blocks of the flat gradient.
    const uint32_t C = (uint32_t)((N + gd::kUnitLen - 1) / gd::kUnitLen);
    ctx->num_units = C;
    std::vector<uint32_t> toff(T + 1), info(C);
    uint64_t max_tiles = 0;
    for (uint32_t t = 0; t <= T; ++t) toff[t] = (uint32_t)off[t];
    for (uint32_t t = 0; t < T; ++t) max_tiles += (off[t + 1] - off[t] + gd::kTile - 1) / gd::kTile;
    ctx->max_tiles = (uint32_t)max_tiles;
    {
        uint32_t t = 0;
        for (uint32_t u = 0; u < C; ++u) {
            const uint64_t us = (uint64_t)u * gd::kUnitLen, ue = std::min<uint64_t>(us + gd::kUnitLen, N);
            while (t + 1 < T && off[t + 1] <= us) ++t;  // last tensor starting at or before us
            bool starts_inside = false;
            for (uint32_t x = t + 1; x < T && off[x] < ue; ++x)
                if (off[x] > us) starts_inside = true;
            info[u] = t | (starts_inside ? 0x80000000u : 0u);
        }
    }

    std::vector<uint32_t> sk_t(T + 1), sk_g(2), goff = {0u, (uint32_t)N};
    uint32_t acc = 0;
    for (uint32_t t = 0; t < T; ++t) {
        sk_t[t] = acc;
        acc += sample_keys_for(off[t], off[t + 1]);
    }
    sk_t[T] = acc;
    ctx->skeys_tensor = acc;
    sk_g[0] = 0;
    sk_g[1] = ctx->skeys_global = sample_keys_for(0, N);

    const uint32_t S_max = T;
    const uint32_t scan_blocks = (C + gd::kScanUnits - 1) / gd::kScanUnits;
    bool ok = dev_upload(ctx, &ctx->tab.unit_info, info) && dev_upload(ctx, &ctx->tab.tensor_off, toff) &&
              dev_upload(ctx, &ctx->tab.global_off, goff) && dev_upload(ctx, &ctx->tab.skey_base_tensor, sk_t) &&
              dev_upload(ctx, &ctx->tab.skey_base_global, sk_g);
    const uint32_t MT = ctx->max_tiles;
    ok = ok && dev_alloc(ctx, &ctx->scr.slots, (size_t)C * gd::kUnitLen) && dev_alloc(ctx, &ctx->scr.cnt, C) &&
         dev_alloc(ctx, &ctx->scr.split, T) && dev_alloc(ctx, &ctx->scr.loc, C) &&
         dev_alloc(ctx, &ctx->scr.neloc, C) && dev_alloc(ctx, &ctx->scr.btot, scan_blocks) &&
         dev_alloc(ctx, &ctx->scr.betot, scan_blocks) && dev_alloc(ctx, &ctx->scr.boff, scan_blocks) &&
         dev_alloc(ctx, &ctx->scr.beoff, scan_blocks) && dev_alloc(ctx, &ctx->scr.ne_unit, C) &&
         dev_alloc(ctx, &ctx->scr.ne_off, C + 1) && dev_alloc(ctx, &ctx->scr.num_ne, 1) &&
         dev_alloc(ctx, &ctx->scr.raw_tbase, T + 1) && dev_alloc(ctx, &ctx->scr.cand_idx, N) &&
         dev_alloc(ctx, &ctx->scr.cand_val, N) && dev_alloc(ctx, &ctx->scr.ten_cbase, T + 1) &&
         dev_alloc(ctx, &ctx->scr.tile_base, T + 1) &&
         dev_alloc(ctx, &ctx->scr.tile_desc, (size_t)MT * gd::kTileDescWords) &&
         dev_alloc(ctx, &ctx->scr.tile_gt, MT) && dev_alloc(ctx, &ctx->scr.tile_eq, MT) &&
         dev_alloc(ctx, &ctx->scr.grp_gt, MT / gd::kGroupTiles + 1) && dev_alloc(ctx, &ctx->scr.grp_eq, MT / gd::kGroupTiles + 1) &&
         dev_alloc(ctx, &ctx->scr.tile_q, 4 * (size_t)MT) &&
         dev_alloc(ctx, &ctx->scr.flags, 4) && dev_alloc(ctx, &ctx->scr.hist, (size_t)S_max * gd::kHistWords) &&
         dev_alloc(ctx, &ctx->scr.seg, S_max) && dev_alloc(ctx, &ctx->scr.out_base, S_max) &&
         dev_alloc(ctx, &ctx->scr.skeys, std::max(ctx->skeys_tensor, ctx->skeys_global)) &&
         dev_alloc(ctx, &ctx->scr.qbase, T + 1) && dev_alloc(ctx, &ctx->scr.shist, (size_t)S_max * gd::kSHistWords) &&
         dev_alloc(ctx, &ctx->scr.sshist, (size_t)S_max * gd::kSsCopies * gd::kSsNB0);
    if (!ok) {
        free_all(ctx);
        delete ctx;
        return GD_ERR_OOM;
    }
    if (!set_columns(ctx, std::vector<uint32_t>(T, 1u))) {
        free_all(ctx);
        delete ctx;
        return GD_ERR_OOM;
    }
    if (hipMemset(ctx->scr.seg, 0, S_max * sizeof(gd::SegState)) != hipSuccess ||
        hipMemset(ctx->scr.shist, 0, (size_t)S_max * gd::kSHistWords * sizeof(uint32_t)) != hipSuccess ||
        hipMemset(ctx->scr.sshist, 0, (size_t)S_max * gd::kSsCopies * gd::kSsNB0 * sizeof(uint32_t)) != hipSuccess ||
        hipMemset(ctx->scr.ten_cbase, 0, (T + 1) * sizeof(uint32_t)) != hipSuccess ||
        hipMemset(ctx->scr.tile_base, 0, (T + 1) * sizeof(uint32_t)) != hipSuccess ||
        hipMemset(ctx->scr.qbase, 0, (T + 1) * sizeof(uint32_t)) != hipSuccess || hipDeviceSynchronize() != hipSuccess) {
        free_all(ctx);
        delete ctx;
        return GD_ERR_HIP;
    }
    *out = ctx;
    return GD_OK;
}

void gd_destroy(gd_ctx* ctx) {
    if (!ctx) return;
    DeviceGuard guard(ctx->device);
    free_all(ctx);
    delete ctx;
}

gd_status gd_compress(gd_ctx* ctx, const float* grad, const float* base, float* residual, double drop_ratio,
                      gd_threshold mode, gd_quant quant, const gd_sparse* out, void* stream) {
    if (!ctx || !out || (ctx->N > 0 && (!grad || !residual))) return GD_ERR_ARG;  // an empty layout needs no data
    if (!valid_mode(enum_int(&mode)) || !valid_quant(enum_int(&quant))) return GD_ERR_ARG;
    if (!(drop_ratio >= 0.0 && drop_ratio <= 1.0)) return GD_ERR_ARG;
    if (!out->idx || !out->val || !out->tensor_counts) return GD_ERR_ARG;
    if (quant != GD_QUANT_NONE && (!out->sign_bits || !out->means)) return GD_ERR_ARG;
    if (!aligned16(grad) || !aligned16(residual) || (base && !aligned16(base))) return GD_ERR_ALIGN;
    const uint64_t k_total = gd_keep_total(ctx, drop_ratio, mode);
    if (out->capacity < k_total) return GD_ERR_CAPACITY;

    DeviceGuard guard(ctx->device);
    if (!guard.ok) return GD_ERR_HIP;
    return gd::compress_exact(ctx, grad, base, residual, drop_ratio, mode == GD_PER_TENSOR, quant, k_total, out,
                              static_cast<hipStream_t>(stream));
}

gd_status gd_compress_pull(gd_ctx* ctx, const float* params, float* copy, double drop_ratio, gd_threshold mode,
                           const gd_sparse* out, void* stream) {
    if (!ctx || !out || (ctx->N > 0 && (!params || !copy))) return GD_ERR_ARG;  // an empty layout needs no data
    if (!valid_mode(enum_int(&mode))) return GD_ERR_ARG;
    if (!(drop_ratio >= 0.0 && drop_ratio <= 1.0)) return GD_ERR_ARG;
    if (!out->idx || !out->val || !out->tensor_counts) return GD_ERR_ARG;
    if (!aligned16(params) || !aligned16(copy)) return GD_ERR_ALIGN;
    const uint64_t k_total = gd_keep_total(ctx, drop_ratio, mode);
    if (out->capacity < k_total) return GD_ERR_CAPACITY;

    DeviceGuard guard(ctx->device);
    if (!guard.ok) return GD_ERR_HIP;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const bool per = mode == GD_PER_TENSOR;
    const uint32_t ppm = (uint32_t)keep_ppm_of(drop_ratio);
    gd::SampleArgs sa{};
    sa.grad = params;
    sa.base = copy;
    sa.res = nullptr;  // acc = params - copy
    sa.seg_off = per ? ctx->tab.tensor_off : ctx->tab.global_off;
    sa.skey_base = per ? ctx->tab.skey_base_tensor : ctx->tab.skey_base_global;
    sa.S = per ? ctx->T : 1u;
    sa.T = ctx->T;
    sa.keep_ppm = ppm;
    sa.debug_bracket = ctx->debug_bracket;
    sa.skeys = ctx->scr.skeys;
    sa.seg = ctx->scr.seg;
    sa.hist = ctx->scr.hist;
    sa.shist = ctx->scr.shist;
    sa.out_base = ctx->scr.out_base;
    sa.tensor_counts = out->tensor_counts;
    if (gd::launch_sample(sa, true, st) != hipSuccess) return GD_ERR_HIP;
    return run_after_bracket(ctx, params, copy, nullptr, per, ppm, false, GD_QUANT_NONE, k_total, out, st);
}

gd_status gd_set_columns(gd_ctx* ctx, const uint32_t* columns) {
    if (!ctx || !columns) return GD_ERR_ARG;
    std::vector<uint32_t> c(columns, columns + ctx->T);
    uint64_t total = 0;
    for (uint32_t t = 0; t < ctx->T; ++t) {
        const uint64_t n = ctx->offsets[t + 1] - ctx->offsets[t];
        if (c[t] == 0 || n % c[t] != 0) return GD_ERR_LAYOUT;
        total += c[t];
    }
    if (total >= 0x80000000ull) return GD_ERR_LAYOUT;
    DeviceGuard guard(ctx->device);
    if (!guard.ok) return GD_ERR_HIP;
    if (hipDeviceSynchronize() != hipSuccess) return GD_ERR_HIP;  // no call may still use the old tables
    return set_columns(ctx, c) ? GD_OK : GD_ERR_OOM;
}

uint64_t gd_quant_centres(const gd_ctx* ctx, gd_quant quant) {
    const int q = enum_int(&quant);
    if (!ctx || q == GD_QUANT_NONE || !valid_quant(q)) return 0;
    return q == GD_QUANT_COLUMN_MEAN ? 2 * (uint64_t)ctx->cols.groups : 2 * (uint64_t)ctx->T;
}

gd_status gd_compress_sampled(gd_ctx* ctx, const float* grad, const float* base, float* residual,
                              double drop_ratio, gd_threshold mode, uint32_t sample_ppm, uint64_t seed,
                              gd_quant quant, const gd_sparse* out, void* stream) {
    if (!ctx || !out || (ctx->N > 0 && (!grad || !residual))) return GD_ERR_ARG;  // an empty layout needs no data
    if (!valid_mode(enum_int(&mode)) || !valid_quant(enum_int(&quant))) return GD_ERR_ARG;
    if (quant != GD_QUANT_NONE && (!out->means || (out->capacity && !out->sign_bits))) return GD_ERR_ARG;
    if (!(drop_ratio >= 0.0 && drop_ratio <= 1.0)) return GD_ERR_ARG;
    if (sample_ppm == 0 || sample_ppm > 1000000u) return GD_ERR_ARG;
    if (!out->tensor_counts || (out->capacity && (!out->idx || !out->val))) return GD_ERR_ARG;
    if (!aligned16(grad) || !aligned16(residual) || (base && !aligned16(base))) return GD_ERR_ALIGN;

    DeviceGuard guard(ctx->device);
    if (!guard.ok) return GD_ERR_HIP;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const bool per = mode == GD_PER_TENSOR;
    const uint32_t ppm = (uint32_t)keep_ppm_of(drop_ratio);
    uint64_t max_n = 0;
    if (per) {
        for (uint32_t t = 0; t < ctx->T; ++t) max_n = std::max(max_n, ctx->offsets[t + 1] - ctx->offsets[t]);
    } else {
        max_n = ctx->N;
    }
    const uint64_t max_samples = (max_n * sample_ppm + 999999u) / 1000000u;

    gd::SampledArgs sa{};
    sa.grad = grad;
    sa.base = base;
    sa.res = residual;
    sa.seg_off = per ? ctx->tab.tensor_off : ctx->tab.global_off;
    sa.S = per ? ctx->T : 1u;
    sa.T = ctx->T;
    sa.per_tensor = per;
    sa.keep_ppm = ppm;
    sa.sample_ppm = sample_ppm;
    sa.seed = seed;
    sa.skeys = ctx->scr.cand_idx;  // free until the candidate passes
    sa.sshist = ctx->scr.sshist;
    sa.seg = ctx->scr.seg;
    sa.tensor_counts = out->tensor_counts;
    if (gd::launch_sampled(sa, base != nullptr, (uint32_t)max_samples, st) != hipSuccess) return GD_ERR_HIP;

    // the number sent is only known on the device: quantisation covers up to
    // the capacity, or N, since no more can be sent
    return run_after_bracket(ctx, grad, base, residual, per, ppm, true, quant, std::min<uint64_t>(out->capacity, ctx->N),
                             out, st);
}

gd_status gd_apply_sparse(float* params, uint64_t n, uint32_t num_pushes, const uint32_t* const* idx,
                          const float* const* val, const uint64_t* nnz, float lr, void* stream) {
    if (num_pushes > gd::kMaxPushes) return GD_ERR_ARG;
    if (n >= 0xFFFFFFFFull) return GD_ERR_ARG;
    if (num_pushes == 0 || n == 0) return GD_OK;
    if (!params || !idx || !val || !nnz) return GD_ERR_ARG;
    gd::ApplyArgs a{};
    a.p = params;
    a.n = (uint32_t)n;
    a.C = num_pushes;
    a.lr = lr;
    uint32_t max_nnz = 0;
    for (uint32_t c = 0; c < num_pushes; ++c) {
        if (nnz[c] >= 0xFFFFFFFFull) return GD_ERR_ARG;
        if (nnz[c] && (!idx[c] || !val[c])) return GD_ERR_ARG;
        a.idx[c] = idx[c];
        a.val[c] = val[c];
        a.nnz[c] = (uint32_t)nnz[c];
        max_nnz = std::max(max_nnz, a.nnz[c]);
    }
    if (gd::launch_apply(a, max_nnz, static_cast<hipStream_t>(stream)) != hipSuccess) return GD_ERR_HIP;
    return GD_OK;
}

gd_status gd_apply_quantised(gd_ctx* ctx, float* params, uint32_t num_pushes, const uint32_t* const* idx,
                             const uint32_t* const* sign_bits, const float* const* means, const uint64_t* nnz,
                             gd_quant quant, float lr, void* stream) {
    if (!ctx || num_pushes > gd::kMaxPushes) return GD_ERR_ARG;
    if (!valid_quant(enum_int(&quant)) || enum_int(&quant) == GD_QUANT_NONE) return GD_ERR_ARG;
    if (num_pushes == 0 || ctx->N == 0) return GD_OK;
    if (!params || !idx || !sign_bits || !means || !nnz) return GD_ERR_ARG;
    gd::ApplyArgs a{};
    a.p = params;
    a.n = (uint32_t)ctx->N;
    a.C = num_pushes;
    a.lr = lr;
    a.qkind = (uint32_t)quant;
    a.tensor_off = ctx->tab.tensor_off;
    a.T = ctx->T;
    a.columns = ctx->cols.columns;
    a.colbase = ctx->cols.colbase;
    uint32_t max_nnz = 0;
    for (uint32_t c = 0; c < num_pushes; ++c) {
        if (nnz[c] >= 0xFFFFFFFFull) return GD_ERR_ARG;
        if (nnz[c] && (!idx[c] || !sign_bits[c] || !means[c])) return GD_ERR_ARG;
        a.idx[c] = idx[c];
        a.bits[c] = sign_bits[c];
        a.means[c] = means[c];
        a.nnz[c] = (uint32_t)nnz[c];
        max_nnz = std::max(max_nnz, a.nnz[c]);
    }
    DeviceGuard guard(ctx->device);
    if (!guard.ok) return GD_ERR_HIP;
    if (gd::launch_apply(a, max_nnz, static_cast<hipStream_t>(stream)) != hipSuccess) return GD_ERR_HIP;
    return GD_OK;
}

gd_status gd_debug_apply_form(int form) {
    if (form < 0 || form > 2) return GD_ERR_ARG;
    gd::set_apply_form(form);
    return GD_OK;
}

gd_status gd_debug_force_bracket(gd_ctx* ctx, int mode) {
    if (!ctx || mode < 0 || mode > 4) return GD_ERR_ARG;
    ctx->debug_bracket = (uint32_t)mode;
    return GD_OK;
}

gd_status gd_debug_state(gd_ctx* ctx, uint32_t* seg_words, uint32_t max_segments, uint64_t* info) {
    if (!ctx || !info || (max_segments && !seg_words)) return GD_ERR_ARG;
    DeviceGuard guard(ctx->device);
    info[0] = gd::kUnitLen;
    info[1] = ctx->num_units;
    info[2] = gd::kTile;
    info[3] = ctx->max_tiles;
    const uint32_t n = std::min(max_segments, ctx->T);
    if (n == 0) return GD_OK;
    if (hipDeviceSynchronize() != hipSuccess) return GD_ERR_HIP;
    if (hipMemcpy(seg_words, ctx->scr.seg, n * sizeof(gd::SegState), hipMemcpyDeviceToHost) != hipSuccess)
        return GD_ERR_HIP;
    return GD_OK;
}

gd_status gd_profile_enable(gd_ctx* ctx, int every) {
    if (!ctx || every < 0) return GD_ERR_ARG;
    DeviceGuard guard(ctx->device);
    if (every && ctx->events.empty()) {
        ctx->events.resize(2 * 4096);
        for (auto& e : ctx->events)
            if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return GD_ERR_HIP;
    }
    ctx->profile_every = (uint32_t)every;
    ctx->events_used = 0;
    ctx->dense_launches = 0;
    return GD_OK;
}

gd_status gd_profile_read(gd_ctx* ctx, double* dense_ms, uint64_t* dense_launches) {
    if (!ctx || !dense_ms || !dense_launches) return GD_ERR_ARG;
    DeviceGuard guard(ctx->device);
    double total = 0.0;
    for (size_t i = 0; i + 1 < ctx->events_used; i += 2) {
        if (hipEventSynchronize(ctx->events[i + 1]) != hipSuccess) return GD_ERR_HIP;
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, ctx->events[i], ctx->events[i + 1]) != hipSuccess) return GD_ERR_HIP;
        total += ms;
    }
    *dense_ms = total;
    *dense_launches = ctx->events_used / 2;
    ctx->events_used = 0;
    ctx->dense_launches = 0;
    return GD_OK;
}

}  // extern "C"
