/*
 * gd.h - C ABI of the gradient-dropping compressor for AMD Instinct MI355X (gfx950).
 *
 * Aji & Heafield, "Sparse Communication for Distributed Gradient Descent"
 * (EMNLP 2017).  Each call of gd_compress is one application of Algorithm 1
 * (GradDrop, Section 4) to a worker's gradient: add the carried residual, pick
 * the threshold that drops R of |gradient|, send the survivors as a sparse
 * (offset, value) list and keep the rest as the next residual.  The threshold
 * is global or per tensor (Section 4, last paragraph); survivors may be 1-bit
 * quantised to per-tensor averages (Section 5.4); pulls are compressed as
 * deltas from the last pulled copy (Section 4, paragraph on pulls).
 * gd_apply_sparse is the server side of the sharded exchange (Section 3).
 *
 * Conventions shared by every entry point:
 *   - Pointers named "device" are HIP device allocations owned by the caller;
 *     pointers named "host" are ordinary host memory.  The library never
 *     frees or keeps a caller pointer beyond the call.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL means the default
 *     stream) and the call returns without waiting for it.  No entry point
 *     synchronises the host with the device.
 *   - Argument, layout, alignment and capacity errors are reported before
 *     anything is enqueued and leave every buffer untouched.  GD_ERR_HIP means
 *     a launch failed; outputs and residual are then undefined.
 *   - Floating point is IEEE binary32 with round-to-nearest-even, no fused
 *     multiply-add and denormals preserved.
 */
#ifndef GD_H
#define GD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    GD_OK = 0,
    GD_ERR_ARG = 1,      /* null pointer, drop ratio outside [0,1], bad enum */
    GD_ERR_LAYOUT = 2,   /* offsets not starting at 0, decreasing, or N > 2^32 - 2 */
    GD_ERR_CAPACITY = 3, /* output capacity below the number of kept entries */
    GD_ERR_ALIGN = 4,    /* grad, base or residual not 16-byte aligned */
    GD_ERR_OOM = 5,      /* device scratch allocation failed (gd_create only) */
    GD_ERR_HIP = 6       /* a HIP runtime call or kernel launch failed */
} gd_status;

/* Where one threshold is chosen (Section 4, last paragraph). */
typedef enum {
    GD_GLOBAL = 0,    /* one threshold over all tensors of the layout */
    GD_PER_TENSOR = 1 /* one threshold per tensor ("per parameter matrix") */
} gd_threshold;

/* What is sent for the survivors (Section 5.4: 1-bit quantisation after
 * dropping).  Every quantised form sends the indices, one sign bit per kept
 * entry (set when acc < 0) and centre pairs (positive centre, negative
 * centre); the kept entry's residual becomes acc minus the centre it is sent
 * as. */
typedef enum {
    GD_QUANT_NONE = 0,        /* (index, value) pairs */
    GD_QUANT_SIGN_MEAN = 1,   /* per tensor: average of its kept positives, of its kept negatives */
    GD_QUANT_THRESHOLD = 2,   /* +-T, T the dropping threshold (the smallest kept |acc| of the
                                 threshold segment), stored per tensor; (0, 0) when the segment
                                 keeps nothing */
    GD_QUANT_GLOBAL_MEAN = 3, /* one average of all kept positives and one of all kept negatives,
                                 stored for every tensor */
    GD_QUANT_COLUMN_MEAN = 4  /* per column of each tensor's row-major matrix view (gd_set_columns):
                                 averages of the column's kept positives and negatives */
} gd_quant;

/* Opaque handle: the tensor layout and the device scratch the kernels use.
 * It owns no caller data; the compressor's only state is the caller's
 * residual buffer. */
typedef struct gd_ctx gd_ctx;

/*
 * gd_create - describe a gradient made of T tensors laid end to end
 * (Section 4, last paragraph: the threshold is chosen either over all
 * parameters or separately for each parameter matrix, so the compressor must
 * know where each matrix starts; Algorithm 1 then runs over this layout).
 *   tensor_offsets (host, T+1 entries): tensor t occupies flat indices
 *     [tensor_offsets[t], tensor_offsets[t+1]); tensor_offsets[0] must be 0,
 *     the sequence non-decreasing (empty tensors are allowed) and
 *     N = tensor_offsets[T] at most 2^32 - 2 (indices are sent as uint32).
 *   Allocates all device scratch on the current HIP device (about 16 bytes
 *   per element plus about 135 KB per tensor for the per-tensor histograms);
 *   gd_compress never allocates.  Any number of tensors is accepted.
 *   Returns GD_ERR_LAYOUT for a bad layout, GD_ERR_OOM when allocation fails.
 */
gd_status gd_create(gd_ctx** out, const uint64_t* tensor_offsets, uint32_t num_tensors);

/* Infrastructure, no passage of the paper: frees the scratch gd_create
 * allocated.  The caller must make sure no enqueued call still uses it.  NULL
 * is accepted and ignored. */
void gd_destroy(gd_ctx* ctx);

/*
 * Number of entries kept out of n at drop ratio R (Algorithm 1, threshold
 * selection: the threshold is placed so that the fraction R of |acc| lies
 * below it).  R is taken in parts per million: keep_ppm = round((1-R)*1e6)
 * and k = floor(n * keep_ppm / 1e6).  Returns 0 for R outside [0,1].
 */
uint64_t gd_keep_count(uint64_t n, double drop_ratio);

/* Total kept entries of one gd_compress call (Algorithm 1 applied once over
 * all parameters, or once per parameter matrix as Section 4's last paragraph
 * allows): k(N) for GD_GLOBAL, the sum of k(n_t) over tensors for
 * GD_PER_TENSOR.  This is the exact output size, known on the host before
 * anything is enqueued.  Returns 0 for a NULL ctx or R outside [0,1]; any
 * mode other than GD_GLOBAL is taken as GD_PER_TENSOR. */
uint64_t gd_keep_total(const gd_ctx* ctx, double drop_ratio, gd_threshold mode);

/* Output buffers of gd_compress (all device pointers, caller-owned). */
typedef struct {
    uint32_t* idx;           /* [capacity] kept flat indices, ascending */
    float* val;              /* [capacity] kept values acc[idx] (before quantisation) */
    uint32_t* sign_bits;     /* quantised forms: [ceil(capacity/32)] words, bit j of
                                word j/32 (LSB first) set when kept value j is negative;
                                unused bits are 0.  Ignored for GD_QUANT_NONE. */
    float* means;            /* quantised forms: gd_quant_centres() floats, (positive centre,
                                negative centre) per tensor, or per column of tensor 0, then of
                                tensor 1, ... for GD_QUANT_COLUMN_MEAN.  Ignored for
                                GD_QUANT_NONE. */
    uint32_t* tensor_counts; /* [T] kept entries per tensor */
    uint64_t capacity;       /* host value: entries idx/val can hold, >= gd_keep_total() */
} gd_sparse;

/*
 * gd_compress - one application of Algorithm 1 (Section 4).
 *   grad (device, N floats): the fresh gradient.  For a pull, the server's
 *     current parameters.
 *   base (device, N floats, or NULL): for a pull, the last pulled copy; the
 *     compressed quantity is then grad - base (Section 4, paragraph on pulls).
 *   residual (device, N floats, in/out): the carried residual.  On return it
 *     holds the new residual: +0.0 at kept entries (or acc minus the sent
 *     centre under a quantised form) and acc elsewhere.
 *   With acc = (grad [- base]) + residual, exactly k entries are kept per
 *   threshold segment: the k largest |acc|, equal magnitudes taken in
 *   ascending flat index (so -0 ties +0; Inf ranks above finite values and
 *   NaN above Inf).  Outputs are written in ascending index order.
 *   grad, base and residual must be 16-byte aligned and must not overlap each
 *   other or the outputs.  One call at a time per ctx (calls on one stream are
 *   naturally ordered).
 */
gd_status gd_compress(gd_ctx* ctx, const float* grad, const float* base, float* residual,
                      double drop_ratio, gd_threshold mode, gd_quant quant, const gd_sparse* out,
                      void* stream);

/*
 * gd_compress_pull - a parameter pull sent as a delta from the client's last
 * pulled copy (Section 4, paragraph on pulls: the server stores that copy and
 * compresses the difference like any other transmission).
 *   params (device, N floats): the server's current parameters.
 *   copy (device, N floats, in/out): what the client holds, as of its last
 *     pull.  acc = params - copy (one binary32 subtraction); the k entries of
 *     largest |acc| are selected exactly as by gd_compress (ties to the lower
 *     index, global or per tensor) and sent as (index, acc); then
 *     copy[i] += acc[i] at every sent entry, so that copy again equals what
 *     the client holds after adding the sent values.  There is no residual
 *     buffer: what is not sent remains in params - copy.
 *   out: as gd_compress without quantisation (sign_bits, means ignored).
 *   params and copy must be 16-byte aligned and must not overlap each other
 *   or the outputs.  Errors as gd_compress.
 */
gd_status gd_compress_pull(gd_ctx* ctx, const float* params, float* copy, double drop_ratio, gd_threshold mode,
                           const gd_sparse* out, void* stream);

/*
 * gd_set_columns - the matrix view used by GD_QUANT_COLUMN_MEAN (Section 5.4:
 * centres per column rather than chosen globally).
 *   columns (host, T entries): tensor t is a row-major matrix of columns[t]
 *     columns; columns[t] must be at least 1 and divide the tensor's size.
 *     Entry e of tensor t is in column (e - tensor_offsets[t]) % columns[t].
 *   Until it is called every tensor is one column (the per-tensor sign mean).
 *   Waits for the device (no call may still be running on this ctx) and
 *   allocates the column tables.  GD_ERR_LAYOUT for a bad column count,
 *   GD_ERR_OOM when allocation fails (the previous columns stay in force).
 */
gd_status gd_set_columns(gd_ctx* ctx, const uint32_t* columns);

/* Number of floats gd_compress writes to out->means for `quant`: 2*T, or twice
 * the total column count for GD_QUANT_COLUMN_MEAN; 0 for GD_QUANT_NONE. */
uint64_t gd_quant_centres(const gd_ctx* ctx, gd_quant quant);

/*
 * gd_compress_sampled - Algorithm 1 with the threshold selected on a sample,
 * the paper's own selection (Section 4: sample 0.1% of the gradient and run
 * the selection on the sample; Algorithm 1 keeps entries strictly above the
 * threshold).  The number kept depends on the data.
 *   grad, base, residual, drop_ratio, mode: as gd_compress.
 *   sample_ppm (1..1000000): sample size per million entries of each threshold
 *     segment (1000 = the paper's 0.1%).  A segment of n entries draws
 *     m = ceil(n * sample_ppm / 1e6) positions, one in each stratum
 *     [a + floor(j n / m), a + floor((j+1) n / m)) at the offset
 *     u mod (stratum length), where u is output number 2^32 * s + j of
 *     SplitMix64 (Steele, Lea and Flood, OOPSLA 2014) seeded with `seed`, s the
 *     segment number and a its first index.
 *   The threshold T is the (k_m + 1)-th largest |acc| of the m sampled entries,
 *   k_m = floor(m * keep_ppm / 1e6) (the largest when k_m = 0); every entry
 *   with |acc| > T is kept (as IEEE bit patterns with the sign cleared, the
 *   order of gd_compress).  k_m >= m keeps every entry; drop_ratio 1 keeps none.
 *   out: idx/val receive the kept entries in ascending index, at most
 *     out->capacity of them (idx and val may be NULL when capacity is 0);
 *     kept entries past the capacity are not sent and keep acc in the
 *     residual.  tensor_counts[t] receives the entries of tensor t actually
 *     sent; their sum is the output length.
 *   quant: as gd_compress (Section 5.4 on what this dropping sends).  The
 *     centres are taken over the entries sent.  The threshold centre is the
 *     smallest sent magnitude of the segment, which is above the sample
 *     threshold.  Sign bits are written for the entries sent; means needs
 *     gd_quant_centres() floats, and sign_bits ceil(capacity/32) words.
 *   residual (in/out): +0.0 at sent entries (acc minus the sent centre under
 *     a quantised form), acc elsewhere.
 *   Returns GD_ERR_ARG for a bad sample_ppm, drop ratio or quant, a NULL
 *   pointer or a bad mode, GD_ERR_ALIGN as gd_compress; never
 *   GD_ERR_CAPACITY.
 */
gd_status gd_compress_sampled(gd_ctx* ctx, const float* grad, const float* base, float* residual,
                              double drop_ratio, gd_threshold mode, uint32_t sample_ppm, uint64_t seed,
                              gd_quant quant, const gd_sparse* out, void* stream);

/*
 * gd_apply_sparse - server-side apply of sparse pushes to a parameter shard
 * (Section 3: servers own a shard and receive the clients' pieces).
 *   params (device, n floats, in/out).
 *   idx, val (host arrays of num_pushes device pointers): push c holds nnz[c]
 *     (host) entries; its indices must be ascending and unique within the push
 *     and below n (entries at an index >= n are skipped).
 *   For every index i that appears in any push: s = sum of the pushed values
 *   at i, added in push order starting from +0.0; params[i] -= lr * s.
 *   num_pushes may be 0 (nothing happens); at most 64 pushes per call.
 *   Pushes dense enough that most of the shard's 128-byte lines hold an
 *   update are applied by reading the shard in order; that form first writes
 *   a table of num_pushes * (ceil(n / 4096) + 1) uint32 (145 KB for four
 *   pushes to a 37M shard).  The library keeps one such table per device and
 *   stream (per host thread for the per-thread default stream) and reuses it
 *   on later calls on that stream; it is allocated with hipMalloc on the
 *   first call that needs it (or a larger one) and kept until the process
 *   ends, so make the first call on a stream outside graph capture.  If that
 *   allocation fails the pushes are applied in the other form; the results
 *   are the same.
 *   The result is deterministic when the precondition above holds.  It is not
 *   checked on the device (that would need a host synchronisation): an index
 *   repeated inside one push is applied by two threads that race, and an
 *   unsorted push can have entries skipped; no memory outside params[0, n)
 *   is written either way.  The Python binding checks the precondition on
 *   request (apply_sparse(..., validate=True)).
 */
gd_status gd_apply_sparse(float* params, uint64_t n, uint32_t num_pushes, const uint32_t* const* idx,
                          const float* const* val, const uint64_t* nnz, float lr, void* stream);

/*
 * gd_apply_quantised - server-side apply of quantised pushes (Section 3 with
 * Section 5.4): each push is what gd_compress sent under `quant` for the
 * layout of ctx (the shard is the whole layout: N parameters).
 *   params (device, N floats, in/out).
 *   idx, sign_bits, means (host arrays of num_pushes device pointers): push c
 *     has nnz[c] (host) ascending, unique indices below N, their sign bits
 *     (bit j % 32 of word j / 32 set for a negative value) and its centre
 *     pairs (gd_quant_centres(ctx, quant) floats; column-wise centres use the
 *     columns of ctx, see gd_set_columns).
 *   Entry j decodes to the negative centre of its tensor's (or column's) pair
 *   when its bit is set, else the positive one; the decoded pushes are then
 *   applied exactly as gd_apply_sparse does (sum in push order from +0.0,
 *   params[i] -= lr * sum).  At most 64 pushes; GD_ERR_ARG for a NULL
 *   pointer or quant GD_QUANT_NONE.
 */
gd_status gd_apply_quantised(gd_ctx* ctx, float* params, uint32_t num_pushes, const uint32_t* const* idx,
                             const uint32_t* const* sign_bits, const float* const* means, const uint64_t* nnz,
                             gd_quant quant, float lr, void* stream);

/*
 * gd_compress_static - gd_compress for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  It takes the layout per call instead of a gd_ctx and
 * allocates nothing (no device or host allocation, no memset); its kernels
 * use a fixed 48 MiB scratch array compiled into the library, one copy per
 * GPU, held from the first call on that GPU until the process ends.
 *   tensor_offsets (host, num_tensors + 1 entries): as gd_create, with at
 *     most 64 tensors and N = tensor_offsets[num_tensors] <= 2,097,152
 *     elements; larger layouts return GD_ERR_LAYOUT (use gd_create).
 *   grad, base, residual, drop_ratio, mode, out, stream: as gd_compress, and
 *     the results are those of gd_compress on a context of the same layout.
 *   quant: GD_QUANT_NONE, GD_QUANT_SIGN_MEAN, GD_QUANT_THRESHOLD or
 *     GD_QUANT_GLOBAL_MEAN; GD_QUANT_COLUMN_MEAN needs a column view
 *     (gd_set_columns) and is GD_ERR_ARG here.
 *   Every call on one GPU shares that GPU's array, and a call starts by
 *   rewriting the parts it uses: calls on one stream are ordered and safe,
 *   but calls that overlap in time on one GPU (other streams, other threads)
 *   race and give wrong results.  The first call on each GPU looks up that
 *   GPU's copy of the array (GD_ERR_HIP if that fails).
 */
gd_status gd_compress_static(const uint64_t* tensor_offsets, uint32_t num_tensors, const float* grad,
                             const float* base, float* residual, double drop_ratio, gd_threshold mode,
                             gd_quant quant, const gd_sparse* out, void* stream);

/* Infrastructure, no passage of the paper: a static, NUL-terminated
 * description of a status code ("unknown status" for other values). */
const char* gd_status_string(gd_status status);

/*
 * Timing of the dense pass (the kernel that streams grad and residual).
 * gd_profile_enable(ctx, every) with every >= 1 times the dense launches
 * numbered 0, every, 2 * every, ... from this call on (every = 1: all of
 * them); every = 0 turns timing off; a negative value is GD_ERR_ARG.  A
 * timed dispatch records a HIP event pair at its own start and end
 * (hipExtLaunchKernelGGL; the events are created without the system-scope
 * fence, as they serve timing only).  Each timed launch still delays the
 * next kernel by a few microseconds, which is why a caller may time only
 * every n-th one.  Up to 4096 launches are timed between reads.
 * gd_profile_read waits for the recorded events, returns the summed
 * milliseconds and the number of timed launches, and resets both.
 */
gd_status gd_profile_enable(gd_ctx* ctx, int every);
gd_status gd_profile_read(gd_ctx* ctx, double* dense_ms, uint64_t* dense_launches);

/*
 * Test hook: override the sampled threshold bracket of later gd_compress
 * calls on this ctx, to exercise paths that real samples rarely take.  The
 * results do not change (they are exact whatever the bracket); only the
 * work done does.  mode 0: normal; 1: bracket above every key, so every
 * segment takes the exact fallback; 2: the dense pass zeroes every
 * candidate; 3: every element is a candidate; 4: only keys at or above the
 * point estimate are candidates and all of them are zeroed, so about half
 * the segments take the exact fallback after the dense pass has zeroed
 * part of their residual.  GD_ERR_ARG for other modes.
 */
gd_status gd_debug_force_bracket(gd_ctx* ctx, int mode);

/*
 * Test hook: the form of later gd_apply_sparse and gd_apply_quantised calls
 * in this process, so that tests can run both forms at any density.  The
 * results do not change; only the work done does.  form 0: chosen per call
 * (streaming, which reads the whole shard in order, when params is 16-byte
 * aligned, the pushes hold at least one entry per 64 parameters, and there
 * are at most 8 of them; else scattered, which reads only the pushed
 * parameters); 1: scattered; 2: streaming wherever params is 16-byte
 * aligned.  A process-wide setting: it applies to every device and thread.
 * GD_ERR_ARG for other forms.
 */
gd_status gd_debug_apply_form(int form);

/*
 * Test hook: waits for the device, then copies the per-segment state of the
 * last gd_compress call (16 uint32 words per threshold segment: candidate
 * bracket lo and hi, candidate count, bracket-miss flag, radix digits and
 * ranks, threshold key, ties kept, zero-mode flag: fewer nonzero keys than
 * k, so the threshold is key 0) for up to max_segments segments into
 * seg_words (host), and the decomposition into info (host, 4 entries:
 * elements per dense-pass unit, units, candidates per tile, most tiles).
 * Synchronises the host.
 */
gd_status gd_debug_state(gd_ctx* ctx, uint32_t* seg_words, uint32_t max_segments, uint64_t* info);

#ifdef __cplusplus
}
#endif

#endif /* GD_H */
