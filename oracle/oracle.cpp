// Gradient-dropping oracle: TEST INFRASTRUCTURE ONLY.
//
// A plain, single-threaded, deliberately slow CPU statement of what the
// compressor computes.  Only the test suite, the smoke check and the
// benchmark's CPU-baseline leg may load it.  It shares no code, header or
// constant with the HIP library and includes none of its files.
//
// Source: Aji & Heafield, "Sparse Communication for Distributed Gradient
// Descent" (EMNLP 2017).
//   * Section 4, Algorithm 1 (GradDrop): add the residual to the gradient,
//     pick the threshold below which R% of |gradient| lies, keep the entries
//     above it, leave the rest as the new residual, return the kept entries
//     as a sparse (offset, value) list.
//   * Section 4, last paragraph: the threshold is chosen either once over all
//     parameters (global) or once per parameter matrix (local).
//   * Section 4, paragraph on pulls: parameter pulls are sent as deltas from
//     the last pulled copy, compressed the same way.
//   * Section 5.4: 1-bit quantisation applied after dropping, with centres
//     taken as averages of the values being quantised.
//   * Section 3: a server owns a shard of the parameters and applies the
//     pushed (sparse) gradients to it.
//
// Readings where the paper is silent (each also listed in the design notes):
//   R1  k = floor(n * keep_ppm / 1e6) with keep_ppm = llround((1 - R) * 1e6).
//   R2  exactly k entries are kept: the k largest keys, key = |acc| taken as
//       the IEEE bit pattern with the sign cleared (so -0 ties +0, Inf is above
//       every finite value and NaN above Inf).  Equal keys are taken in
//       ascending flat index.  With distinct keys this is Algorithm 1 with the
//       threshold set to the (k+1)-th largest magnitude.
//   R3  the residual of a kept entry is exactly +0.0f; a dropped entry keeps
//       acc's bits (the same as acc - dropped for finite values).
//   R4  binary32 round-to-nearest-even, no fused multiply-add, denormals kept.
//   R5  sign-mean quantisation is per tensor even under a global threshold:
//       positives (acc not < 0, so zeros count as positive) and negatives are
//       averaged separately as (sum in double, ascending index) / count,
//       rounded to float; an empty group has centre 0.  The quantisation error
//       acc - centre goes back into the residual.
//   R6  server apply: s[i] = sum of the pushed values at i in client order
//       (float adds starting from +0.0f), then p[i] = p[i] - lr * s[i].
//   R7  pull delta: acc = (p_new - p_last) + residual, two float roundings.
//   R10 the other centres Section 5.4 tests, over the same kept set and with
//       the same sign bits and error feedback as R5:
//       threshold (quant 2): every survivor maps to +-T_s, T_s the smallest
//         kept |acc| of its threshold segment (0 when the segment keeps none);
//       global average (quant 3): one positive and one negative average over
//         every kept entry of the call, the same pair for every tensor;
//       column-wise average (quant 4): tensor t is a row-major matrix of
//         columns[t] columns (columns[t] divides its size); each column's kept
//         positives and negatives are averaged separately, pairs stored for
//         the columns of tensor 0, then tensor 1, ... (columns NULL: one
//         column per tensor, which is R5).
//   R11 pull with the last pulled copy (Section 4, paragraph on pulls: the
//       server stores the copy a client last pulled and sends deltas from
//       it): acc = p - copy (one float rounding, no residual buffer: what is
//       not sent stays in the difference), the same exact selection as R2,
//       (idx, acc) sent, and the copy becomes what the client holds after
//       adding the sent values: copy[kept] = copy[kept] + acc.
//   R12 quantised pushes at the server (Section 3 with Section 5.4): entry j
//       of a push decodes to the centre its sign bit (bit j%32 of word j/32)
//       selects among the pair of its group (its tensor, or its column under
//       column-wise centres), then the decoded pushes are applied as R6.
//   R9  sampled threshold (Section 4: select on a 0.1% sample of the
//       gradient, then keep what lies strictly above the threshold):
//       segment s of n entries draws m = ceil(n * sample_ppm / 1e6)
//       positions, one per stratum [floor(j n / m), floor((j+1) n / m)), at
//       offset u mod (stratum length), where u is output number
//       2^32 * s + j of SplitMix64 seeded with `seed` (Steele, Lea and Flood,
//       OOPSLA 2014).  With k_m = floor(m * keep_ppm / 1e6) the threshold T
//       is the (k_m + 1)-th largest sample key (the exact mode's relation to
//       Algorithm 1, R2; for k_m = 0 the largest) and entries with key > T
//       are kept; k_m >= m keeps everything and R = 1 (keep_ppm = 0) keeps
//       nothing.  The count is data dependent; kept entries past the output
//       capacity (in ascending index) are not sent and keep acc in the
//       residual.
//   R13 1-bit quantisation under the sampled threshold (Section 5.4 on what
//       the Section 4 dropping sends): the centres of R5 and R10 over the
//       entries actually sent, the threshold centre being the smallest sent
//       magnitude of the segment; sent entries get acc - centre.
//
// Build: g++ -O2 -ffp-contract=off -fPIC -shared (no fast-math).

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <functional>
#include <vector>

namespace {

inline uint32_t key_of(float x) {
    uint32_t b;
    std::memcpy(&b, &x, sizeof b);
#ifdef GDO_MUTANT_SIGNED_KEY
    return b;  // mutant: compares raw bits, ignoring |.|
#else
    return b & 0x7FFFFFFFu;
#endif
}

}  // namespace
extern "C" uint64_t gdo_keep_count(uint64_t n, double drop_ratio);
namespace {
uint64_t keep_count_of(uint64_t n, double drop_ratio) { return gdo_keep_count(n, drop_ratio); }

// Algorithm 1, threshold selection and the keep mask (R2): in each segment
// the k largest keys, equal keys in ascending index.
std::vector<uint8_t> exact_keep(const std::vector<float>& acc, const std::vector<std::pair<uint64_t, uint64_t>>& seg,
                                double drop_ratio) {
    const uint64_t N = acc.size();
    (void)N;
    std::vector<uint8_t> keep(acc.size(), 0);
    for (auto& s : seg) {
        const uint64_t n = s.second - s.first;
#ifdef GDO_MUTANT_GLOBAL_K_PER_TENSOR
        const uint64_t k = std::min<uint64_t>(n, keep_count_of(N, drop_ratio) / seg.size());
#else
        const uint64_t k = keep_count_of(n, drop_ratio);
#endif
        if (k == 0) continue;
        std::vector<uint32_t> keys(n);
        for (uint64_t i = 0; i < n; ++i) keys[i] = key_of(acc[s.first + i]);
        std::nth_element(keys.begin(), keys.begin() + (k - 1), keys.end(), std::greater<uint32_t>());
        const uint32_t thr = keys[k - 1];  // the k-th largest key
        uint64_t above = 0;
        for (uint64_t i = s.first; i < s.second; ++i) above += key_of(acc[i]) > thr;
        uint64_t ties_left = k - above;  // entries equal to thr still to take
#ifdef GDO_MUTANT_STRICT_ONLY
        ties_left = 0;  // mutant: Algorithm 1's strict ">" without the exact-k rule
#endif
#ifdef GDO_MUTANT_TIES_HIGH_INDEX
        for (uint64_t i = s.second; i-- > s.first;) {
#else
        for (uint64_t i = s.first; i < s.second; ++i) {
#endif
            const uint32_t kk = key_of(acc[i]);
            if (kk > thr) {
                keep[i] = 1;
            } else if (kk == thr && ties_left > 0) {
                keep[i] = 1;
                --ties_left;
            }
        }
    }

    return keep;
}

}  // namespace

// Section 5.4, 1-bit quantisation with error feedback (R5, R10, R13): each
// of the k entries sent (idx, val, in tensor order as tensor_counts gives
// them) is sent as the centre of its group and sign, and acc minus that
// centre goes back into the residual.  Centres are taken over the entries
// sent; the threshold centre is the smallest sent magnitude of the threshold
// segment (one segment, or one per tensor when per_tensor).
static void quantise_sent(const uint64_t* offsets, uint32_t T, bool per_tensor, int quant, const uint32_t* columns,
                          const uint32_t* idx, const float* val, const uint32_t* tensor_counts, uint64_t k,
                          uint32_t* sign_bits, float* means, float* residual) {
    const size_t nseg = per_tensor ? T : 1u;
    const uint64_t words = (k + 31) / 32;
    for (uint64_t w = 0; w < words; ++w) sign_bits[w] = 0;
    // group of every output slot: its tensor, or its column for quant 4
    std::vector<uint64_t> colbase(T + 1, 0);
    for (uint32_t t = 0; t < T; ++t) colbase[t + 1] = colbase[t] + (quant == 4 && columns ? columns[t] : 1);
    std::vector<uint64_t> group(k);
    {
        uint64_t q = 0;
        for (uint32_t t = 0; t < T; ++t) {
            for (uint32_t c = 0; c < tensor_counts[t] && q < k; ++c, ++q) {
                uint64_t g = t;
                if (quant == 4) {
                    const uint64_t cols = columns ? columns[t] : 1;
#ifdef GDO_MUTANT_COLUMN_IS_ROW
                    g = colbase[t] + ((idx[q] - offsets[t]) / cols) % cols;  // mutant: rows, not columns
#else
                    g = colbase[t] + (idx[q] - offsets[t]) % cols;
#endif
                }
                group[q] = g;
            }
        }
    }
    const uint64_t G = quant == 4 ? colbase[T] : T;
    std::vector<float> pos_c(G, 0.0f), neg_c(G, 0.0f);
    if (quant == 1 || quant == 4) {
        // averages per group, summed in double in ascending index
        std::vector<double> ps(G, 0.0), ns(G, 0.0);
        std::vector<uint64_t> pn(G, 0), nn(G, 0);
        for (uint64_t q = 0; q < k; ++q) {
            if (val[q] < 0.0f) {
                ns[group[q]] += (double)val[q];
                ++nn[group[q]];
            } else {
                ps[group[q]] += (double)val[q];
                ++pn[group[q]];
            }
        }
        for (uint64_t g = 0; g < G; ++g) {
            pos_c[g] = pn[g] ? (float)(ps[g] / (double)pn[g]) : 0.0f;
            neg_c[g] = nn[g] ? (float)(ns[g] / (double)nn[g]) : 0.0f;
        }
    } else if (quant == 3) {
        // one average of each sign over the whole call
        double ps = 0.0, ns = 0.0;
        uint64_t pn = 0, nn = 0;
        for (uint64_t q = 0; q < k; ++q) {
            if (val[q] < 0.0f) {
                ns += (double)val[q];
                ++nn;
            } else {
                ps += (double)val[q];
                ++pn;
            }
        }
        const float pc = pn ? (float)(ps / (double)pn) : 0.0f;
        const float nc = nn ? (float)(ns / (double)nn) : 0.0f;
        for (uint64_t g = 0; g < G; ++g) {
#ifdef GDO_MUTANT_GLOBAL_MEAN_PER_TENSOR
            (void)pc;
            (void)nc;
#else
            pos_c[g] = pc;
            neg_c[g] = nc;
#endif
        }
#ifdef GDO_MUTANT_GLOBAL_MEAN_PER_TENSOR
        // mutant: per-tensor averages instead of one over the call
        std::vector<double> ps2(G, 0.0), ns2(G, 0.0);
        std::vector<uint64_t> pn2(G, 0), nn2(G, 0);
        for (uint64_t q = 0; q < k; ++q) {
            if (val[q] < 0.0f) { ns2[group[q]] += val[q]; ++nn2[group[q]]; }
            else { ps2[group[q]] += val[q]; ++pn2[group[q]]; }
        }
        for (uint64_t g = 0; g < G; ++g) {
            pos_c[g] = pn2[g] ? (float)(ps2[g] / (double)pn2[g]) : 0.0f;
            neg_c[g] = nn2[g] ? (float)(ns2[g] / (double)nn2[g]) : 0.0f;
        }
#endif
    } else {
        // quant 2: the smallest kept magnitude of each threshold segment
        std::vector<uint32_t> seg_min(nseg, 0xFFFFFFFFu);
        std::vector<uint8_t> seg_any(nseg, 0);
        uint64_t q = 0;
        for (uint32_t t = 0; t < T; ++t) {
            const uint32_t sg = per_tensor ? t : 0u;
            for (uint32_t c = 0; c < tensor_counts[t]; ++c, ++q) {
                const uint32_t kk = key_of(val[q]);
#ifdef GDO_MUTANT_THRESHOLD_MAX
                if (!seg_any[sg] || kk > seg_min[sg]) seg_min[sg] = kk;  // mutant: the largest instead
#else
                if (!seg_any[sg] || kk < seg_min[sg]) seg_min[sg] = kk;
#endif
                seg_any[sg] = 1;
            }
        }
        for (uint32_t t = 0; t < T; ++t) {
            const uint32_t sg = per_tensor ? t : 0u;
            if (!seg_any[sg]) continue;
            float mag;
            std::memcpy(&mag, &seg_min[sg], sizeof mag);
            pos_c[t] = mag;
            neg_c[t] = -mag;
        }
    }
    for (uint64_t g = 0; g < G; ++g) {
#ifdef GDO_MUTANT_SWAP_CENTRES
        means[2 * g + 0] = neg_c[g];
        means[2 * g + 1] = pos_c[g];
#else
        means[2 * g + 0] = pos_c[g];
        means[2 * g + 1] = neg_c[g];
#endif
    }
    for (uint64_t q = 0; q < k; ++q) {
        const bool neg = val[q] < 0.0f;
#ifdef GDO_MUTANT_BITS_MSB_FIRST
        if (neg) sign_bits[q >> 5] |= 1u << (31 - (q & 31));
#else
        if (neg) sign_bits[q >> 5] |= 1u << (q & 31);
#endif
        const float sent = neg ? means[2 * group[q] + 1] : means[2 * group[q] + 0];
        residual[idx[q]] = val[q] - sent;
    }
}

extern "C" {

// R1: the keep fraction in parts per million.
uint64_t gdo_keep_ppm(double drop_ratio) {
    return (uint64_t)std::llround((1.0 - drop_ratio) * 1e6);
}

// R1: number of entries kept out of n.
uint64_t gdo_keep_count(uint64_t n, double drop_ratio) {
    uint64_t ppm = gdo_keep_ppm(drop_ratio);
#ifdef GDO_MUTANT_CEIL_K
    return (n * ppm + 999999u) / 1000000u;  // mutant: rounds k up
#else
    return n * ppm / 1000000u;
#endif
}

// Algorithm 1 over the tensors described by offsets[0..T] (offsets[T] = N).
// grad, base (nullable), residual: length N.  residual is read and rewritten.
// Outputs (caller-allocated, capacity entries): idx, val; sign_bits
// (ceil(capacity/32) words) and means (2*T, or 2 * sum of columns for quant 4)
// when quant != 0; tensor_counts (T).  quant: 0 none, 1 per-tensor sign mean
// (R5), 2 threshold, 3 global average, 4 column-wise average (R10); columns
// (T entries, nullable) describes the matrices for quant 4.
// Returns 0 on success, 1 on bad arguments, 3 when capacity is too small.
int gdo_compress(const float* grad, const float* base, float* residual, const uint64_t* offsets,
                 uint32_t T, double drop_ratio, int per_tensor, int quant, uint32_t* idx, float* val,
                 uint32_t* sign_bits, float* means, uint32_t* tensor_counts, uint64_t capacity,
                 uint64_t* out_k, const uint32_t* columns) {
    if (!grad || !residual || !offsets || T == 0 || !idx || !val || !tensor_counts) return 1;
    if (!(drop_ratio >= 0.0 && drop_ratio <= 1.0)) return 1;
    if (quant < 0 || quant > 4) return 1;
    if (quant && (!sign_bits || !means)) return 1;
    const uint64_t N = offsets[T];
    if (offsets[0] != 0 || N > 0xFFFFFFFFull) return 1;
    for (uint32_t t = 0; t < T; ++t)
        if (offsets[t + 1] < offsets[t]) return 1;
    if (quant == 4 && columns) {
        for (uint32_t t = 0; t < T; ++t)
            if (columns[t] == 0 || (offsets[t + 1] - offsets[t]) % columns[t] != 0) return 1;
    }

    // Segments over which one threshold is chosen (Section 4: global or local).
    std::vector<std::pair<uint64_t, uint64_t>> seg;
    if (per_tensor) {
        for (uint32_t t = 0; t < T; ++t) seg.push_back({offsets[t], offsets[t + 1]});
    } else {
        seg.push_back({0, N});
    }
    uint64_t k_total = 0;
    for (auto& s : seg) {
#ifdef GDO_MUTANT_GLOBAL_K_PER_TENSOR
        k_total += std::min<uint64_t>(s.second - s.first, gdo_keep_count(N, drop_ratio) / seg.size());
#else
        k_total += gdo_keep_count(s.second - s.first, drop_ratio);
#endif
    }
    if (out_k) *out_k = k_total;
    if (capacity < k_total) return 3;

    // Algorithm 1, first line: add the carried residual (pulls: delta first, R7).
    std::vector<float> acc(N);
    for (uint64_t i = 0; i < N; ++i) {
        float g = grad[i];
#ifdef GDO_MUTANT_DELTA_REVERSED
        if (base) g = base[i] - g;
#else
        if (base) g = g - base[i];
#endif
#ifdef GDO_MUTANT_NO_RESIDUAL
        acc[i] = g;
#else
        acc[i] = g + residual[i];
#endif
    }

    std::vector<uint8_t> keep = exact_keep(acc, seg, drop_ratio);

    // Algorithm 1, sparse(dropped): ascending flat indices and values.
    uint64_t j = 0;
    for (uint32_t t = 0; t < T; ++t) tensor_counts[t] = 0;
    for (uint32_t t = 0; t < T; ++t) {
        for (uint64_t i = offsets[t]; i < offsets[t + 1]; ++i) {
            if (!keep[i]) continue;
            idx[j] = (uint32_t)i;
            val[j] = acc[i];
            ++j;
            ++tensor_counts[t];
        }
    }

    // Algorithm 1, residual update (R3).
    for (uint64_t i = 0; i < N; ++i) {
#ifdef GDO_MUTANT_KEPT_RESIDUAL_KEEPS_ACC
        residual[i] = acc[i];
#else
        residual[i] = keep[i] ? 0.0f : acc[i];
#endif
    }

    if (quant) quantise_sent(offsets, T, per_tensor != 0, quant, columns, idx, val, tensor_counts, k_total, sign_bits,
                             means, residual);
    return 0;
}

// Section 4, pulls as deltas from the last pulled copy (R11).  params (N),
// copy (N, read and rewritten), outputs as gdo_compress without quantisation.
// Returns 0 on success, 1 on bad arguments, 3 when capacity is too small.
int gdo_compress_pull(const float* params, float* copy, const uint64_t* offsets, uint32_t T, double drop_ratio,
                      int per_tensor, uint32_t* idx, float* val, uint32_t* tensor_counts, uint64_t capacity,
                      uint64_t* out_k) {
    if (!params || !copy || !offsets || T == 0 || !idx || !val || !tensor_counts) return 1;
    if (!(drop_ratio >= 0.0 && drop_ratio <= 1.0)) return 1;
    const uint64_t N = offsets[T];
    if (offsets[0] != 0 || N > 0xFFFFFFFFull) return 1;
    for (uint32_t t = 0; t < T; ++t)
        if (offsets[t + 1] < offsets[t]) return 1;
    std::vector<std::pair<uint64_t, uint64_t>> seg;
    if (per_tensor) {
        for (uint32_t t = 0; t < T; ++t) seg.push_back({offsets[t], offsets[t + 1]});
    } else {
        seg.push_back({0, N});
    }
    uint64_t k_total = 0;
    for (auto& sg : seg) k_total += gdo_keep_count(sg.second - sg.first, drop_ratio);
    if (out_k) *out_k = k_total;
    if (capacity < k_total) return 3;
    // the delta from the last pulled copy
    std::vector<float> acc(N);
    for (uint64_t i = 0; i < N; ++i) {
#ifdef GDO_MUTANT_PULL_ADDS_ZERO
        acc[i] = (params[i] - copy[i]) + 0.0f;  // mutant: an added zero residual turns -0 into +0
#else
        acc[i] = params[i] - copy[i];
#endif
    }
    std::vector<uint8_t> keep = exact_keep(acc, seg, drop_ratio);
    uint64_t j = 0;
    for (uint32_t t = 0; t < T; ++t) tensor_counts[t] = 0;
    for (uint32_t t = 0; t < T; ++t) {
        for (uint64_t i = offsets[t]; i < offsets[t + 1]; ++i) {
            if (!keep[i]) continue;
            idx[j] = (uint32_t)i;
            val[j] = acc[i];
            ++j;
            ++tensor_counts[t];
#ifdef GDO_MUTANT_PULL_COPY_IS_P
            copy[i] = params[i];  // mutant: assumes the client ends up holding p exactly
#else
            copy[i] = copy[i] + acc[i];  // what the client holds after adding the sent delta
#endif
        }
    }
    return 0;
}

// Section 3 with Section 5.4: quantised pushes decoded, then applied (R12, R6).
// The shard is the whole layout offsets[0..T]; quant 1..4 as gdo_compress
// (columns only for quant 4, nullable).  Returns 0, or 1 on bad arguments.
int gdo_apply_sparse(float* params, uint64_t n, uint32_t C, const uint32_t* const* idx,
                     const float* const* val, const uint64_t* nnz, float lr);
int gdo_apply_quantised(float* params, const uint64_t* offsets, uint32_t T, const uint32_t* columns, uint32_t C,
                        const uint32_t* const* idx, const uint32_t* const* sign_bits, const float* const* means,
                        const uint64_t* nnz, int quant, float lr) {
    if (!params || !offsets || T == 0 || quant < 1 || quant > 4) return 1;
    if (C && (!idx || !sign_bits || !means || !nnz)) return 1;
    const uint64_t N = offsets[T];
    std::vector<uint64_t> colbase(T + 1, 0);
    for (uint32_t t = 0; t < T; ++t) colbase[t + 1] = colbase[t] + (quant == 4 && columns ? columns[t] : 1);
    std::vector<std::vector<float>> dec(C);
    std::vector<const float*> vp(C);
    for (uint32_t c = 0; c < C; ++c) {
        dec[c].resize(nnz[c]);
        for (uint64_t j = 0; j < nnz[c]; ++j) {
            const uint64_t i = idx[c][j];
            if (i >= N) return 1;
            // tensor holding i: the last t with offsets[t] <= i
            uint32_t t = 0;
            while (t + 1 < T && offsets[t + 1] <= i) ++t;
            uint64_t g = t;
            if (quant == 4) g = colbase[t] + (i - offsets[t]) % (columns ? columns[t] : 1);
#ifdef GDO_MUTANT_DECODE_BITS_MSB
            const bool neg = (sign_bits[c][j >> 5] >> (31 - (j & 31))) & 1u;  // mutant: bit order reversed
#else
            const bool neg = (sign_bits[c][j >> 5] >> (j & 31)) & 1u;
#endif
            dec[c][j] = means[c][2 * g + (neg ? 1 : 0)];
        }
        vp[c] = dec[c].data();
    }
    return gdo_apply_sparse(params, N, C, idx, vp.data(), nnz, lr);
}

// R9: output number i of SplitMix64 seeded with seed: the state advances by
// the golden-ratio increment once per output and is then mixed.
uint64_t gdo_splitmix64(uint64_t seed, uint64_t i) {
    uint64_t z = seed + (i + 1) * 0x9E3779B97F4A7C15ull;
#ifdef GDO_MUTANT_SPLITMIX_SHIFT
    z = (z ^ (z >> 31)) * 0xBF58476D1CE4E5B9ull;  // mutant: wrong first shift
#else
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
#endif
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// Position of sample j of segment s ([a, a+n)) among m samples (R9).
uint64_t gdo_sample_position(uint64_t seed, uint32_t s, uint64_t a, uint64_t n, uint64_t m, uint64_t j) {
    const uint64_t lo = j * n / m, hi = (j + 1) * n / m;
#ifdef GDO_MUTANT_SAMPLE_WHOLE_SEGMENT
    (void)lo;
    (void)hi;
    return a + gdo_splitmix64(seed, ((uint64_t)s << 32) | j) % n;  // mutant: ignores the strata
#else
    return a + lo + gdo_splitmix64(seed, ((uint64_t)s << 32) | j) % (hi - lo);
#endif
}

// Algorithm 1 with the threshold selected on a sample (Section 4, R9), and
// optionally the 1-bit quantisation of Section 5.4 over the entries sent
// (R13).  Arguments as gdo_compress plus sample_ppm (1..1e6) and seed;
// idx/val (and sign_bits when quant != 0) may be null when capacity is 0.
// *out_k receives the number of entries sent.  Returns 0 on success, 1 on
// bad arguments.
int gdo_compress_sampled(const float* grad, const float* base, float* residual, const uint64_t* offsets,
                         uint32_t T, double drop_ratio, int per_tensor, uint32_t sample_ppm, uint64_t seed,
                         int quant, uint32_t* idx, float* val, uint32_t* sign_bits, float* means,
                         uint32_t* tensor_counts, uint64_t capacity, uint64_t* out_k, const uint32_t* columns) {
    if (!grad || !residual || !offsets || T == 0 || !tensor_counts) return 1;
    if (capacity && (!idx || !val)) return 1;
    if (!(drop_ratio >= 0.0 && drop_ratio <= 1.0)) return 1;
    if (sample_ppm == 0 || sample_ppm > 1000000u) return 1;
    if (quant < 0 || quant > 4) return 1;
    if (quant && (!means || (capacity && !sign_bits))) return 1;
    const uint64_t N = offsets[T];
    if (offsets[0] != 0 || N > 0xFFFFFFFFull) return 1;
    for (uint32_t t = 0; t < T; ++t)
        if (offsets[t + 1] < offsets[t]) return 1;
    if (quant == 4 && columns) {
        for (uint32_t t = 0; t < T; ++t)
            if (columns[t] == 0 || (offsets[t + 1] - offsets[t]) % columns[t] != 0) return 1;
    }
    const uint64_t keep_ppm = gdo_keep_ppm(drop_ratio);

    // Algorithm 1, first line: add the carried residual (pulls: delta first, R7).
    std::vector<float> acc(N);
    for (uint64_t i = 0; i < N; ++i) {
        float g = grad[i];
        if (base) g = g - base[i];
        acc[i] = g + residual[i];
    }

    std::vector<std::pair<uint64_t, uint64_t>> seg;
    if (per_tensor) {
        for (uint32_t t = 0; t < T; ++t) seg.push_back({offsets[t], offsets[t + 1]});
    } else {
        seg.push_back({0, N});
    }

    // Section 4: the threshold from a selection on the sample; keep above it.
    std::vector<uint8_t> keep(N, 0);
    for (uint32_t s = 0; s < seg.size(); ++s) {
        const uint64_t a = seg[s].first, n = seg[s].second - seg[s].first;
        if (n == 0) continue;
        const uint64_t m = (n * sample_ppm + 999999u) / 1000000u;
        std::vector<uint32_t> skeys(m);
        for (uint64_t j = 0; j < m; ++j) skeys[j] = key_of(acc[gdo_sample_position(seed, s, a, n, m, j)]);
        const uint64_t km = m * keep_ppm / 1000000u;
        if (keep_ppm == 0) continue;
        if (km >= m) {
            for (uint64_t i = a; i < a + n; ++i) keep[i] = 1;
            continue;
        }
#ifdef GDO_MUTANT_SAMPLED_KTH
        const uint64_t r = km ? km - 1 : 0;  // mutant: threshold at the k_m-th sample key
#else
        const uint64_t r = km;  // 0-based rank of the (k_m + 1)-th largest
#endif
        std::nth_element(skeys.begin(), skeys.begin() + r, skeys.end(), std::greater<uint32_t>());
        const uint32_t thr = skeys[r];
        for (uint64_t i = a; i < a + n; ++i) {
#ifdef GDO_MUTANT_SAMPLED_GE
            keep[i] = key_of(acc[i]) >= thr;  // mutant: keeps the threshold key too
#else
            keep[i] = key_of(acc[i]) > thr;
#endif
        }
    }

    // sparse(dropped) in ascending index, up to the capacity; the rest stays
    // in the residual.
    uint64_t j = 0;
    for (uint32_t t = 0; t < T; ++t) tensor_counts[t] = 0;
    for (uint32_t t = 0; t < T; ++t) {
        for (uint64_t i = offsets[t]; i < offsets[t + 1]; ++i) {
            if (!keep[i]) continue;
#ifndef GDO_MUTANT_SAMPLED_NO_CAPACITY
            if (j >= capacity) {
                keep[i] = 0;
                continue;
            }
#endif
            if (j < capacity) {
                idx[j] = (uint32_t)i;
                val[j] = acc[i];
            }
            ++j;
            ++tensor_counts[t];
        }
    }
    if (out_k) *out_k = j;
    for (uint64_t i = 0; i < N; ++i) residual[i] = keep[i] ? 0.0f : acc[i];
    if (quant)
        quantise_sent(offsets, T, per_tensor != 0, quant, columns, idx, val, tensor_counts, std::min(j, capacity),
                      sign_bits, means, residual);
    return 0;
}

// Section 3: a server applies sparse pushes to its parameter shard (R6).
// idx[c] (ascending, unique within a client) and val[c] hold nnz[c] entries.
// Returns 0 on success, 1 on bad arguments (including an index >= n).
int gdo_apply_sparse(float* params, uint64_t n, uint32_t C, const uint32_t* const* idx,
                     const float* const* val, const uint64_t* nnz, float lr) {
    if (!params || (C && (!idx || !val || !nnz))) return 1;
    for (uint32_t c = 0; c < C; ++c)
        for (uint64_t j = 0; j < nnz[c]; ++j)
            if (idx[c][j] >= n) return 1;
    std::vector<float> s(n, 0.0f);
    std::vector<uint8_t> touched(n, 0);
#ifdef GDO_MUTANT_APPLY_REVERSE_CLIENTS
    for (uint32_t c = C; c-- > 0;) {
#else
    for (uint32_t c = 0; c < C; ++c) {
#endif
        for (uint64_t j = 0; j < nnz[c]; ++j) {
            const uint32_t i = idx[c][j];
            s[i] = s[i] + val[c][j];
            touched[i] = 1;
        }
    }
    for (uint64_t i = 0; i < n; ++i) {
        if (!touched[i]) continue;
        const float step = lr * s[i];
#ifdef GDO_MUTANT_APPLY_ADD
        params[i] = params[i] + step;
#else
        params[i] = params[i] - step;
#endif
    }
    return 0;
}

}  // extern "C"
