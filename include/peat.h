/*
 * peat.h -- C ABI of libpeat: error signatures of golden/test tensor pairs and
 * seeded random-bit-flip injection, as hand-written HIP kernels for AMD
 * Instinct MI355X (gfx950).
 *
 * The operations follow the PEAT paper ("PEAT: Pseudo-Error Assessment for
 * GPU Kernel Validation in DNN Training"):
 *   - Err(golden set, FI set) of Algorithms 1 and 2 with the scores of
 *     Section IV-B.3 ("FI Assessment Scores": the error is the absolute
 *     difference; max, mean, variance), the closeness test of Section III-A
 *     (torch.isclose, here with rtol = 0) and the error value histograms of
 *     Section V-D, gathered into one error signature per tensor pair;
 *   - Inject() of Algorithms 1 and 2 with the random-bit-flip error model of
 *     Section II-B ("Error Models": flips at a given bit error rate).
 *
 * Conventions for every entry point
 *   - Tensor pointers (golden, test, tensor, pair/item pointers) are DEVICE
 *     pointers to contiguous element arrays owned by the caller; the library
 *     neither frees nor keeps them after the call's work has completed.
 *   - Struct arrays passed by pointer (pairs, items, bins, thresholds) are HOST
 *     memory owned by the caller; the library copies what it needs before
 *     returning.
 *   - Synchronous calls write HOST outputs and return after the work is done.
 *     They run on the stream set with peat_set_stream (default: the null
 *     stream).  *_async calls enqueue on the given stream, write DEVICE outputs
 *     and return without waiting.
 *   - Return value 0 (PEAT_OK) or a negative PEAT_E* code; outputs are left
 *     untouched on error.  No C++ exception crosses this boundary.
 *     peat_last_error() gives a thread-local detail string for the last error.
 *   - The library keeps one lazily grown device workspace and one pinned
 *     staging ring per device.  Growing the workspace synchronises the device.
 *     Calls from several host threads are serialised by an internal mutex;
 *     work on different streams is ordered through an event on the workspace.
 *   - Element types: PEAT_F32 (IEEE binary32), PEAT_F16 (IEEE binary16),
 *     PEAT_BF16 (bfloat16), and PEAT_F64 (IEEE binary64) as the test side of a
 *     mixed-precision pair.  Values are widened exactly to binary64; all
 *     error arithmetic is IEEE binary64 round-to-nearest-even, subnormals kept.
 */
#ifndef PEAT_H
#define PEAT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PEAT_ABI_VERSION 6
#define PEAT_MAX_THRESHOLDS 8
#define PEAT_MAX_BINS 64

/* PEAT_F64 is accepted only as the test type of a mixed-precision pair. */
typedef enum { PEAT_F32 = 0, PEAT_F16 = 1, PEAT_BF16 = 2, PEAT_F64 = 3 } peat_dtype_t;

enum {
    PEAT_OK = 0,
    PEAT_EINVAL = -1,   /* bad pointer/size/bins/thresholds/count          */
    PEAT_EDTYPE = -2,   /* unknown element type                            */
    PEAT_EBITMASK = -3, /* bitmask is 0 or has bits at/above the type width */
    PEAT_ERATE = -4,    /* injection rate is NaN or negative               */
    PEAT_EHIP = -5,     /* HIP runtime error (detail in peat_last_error)   */
    PEAT_ENOMEM = -6,   /* device or pinned host allocation failed         */
    PEAT_ENODEV = -7    /* no usable gfx950 device                         */
};

/* Histogram of the absolute error a over binades: bin b covers
 * [2^(lo + b*w), 2^(lo + (b+1)*w)) with w = (hi - lo) / nbins.  Errors equal
 * to 0 go to hist_zero, 0 < a < 2^lo to hist_under, a >= 2^hi (and a = +Inf)
 * to hist_over.  Valid: -1022 <= lo_log2 < hi_log2 <= 1024,
 * 1 <= nbins <= 64, nbins divides hi - lo.  (Section V-D histograms.) */
typedef struct {
    int32_t lo_log2;
    int32_t hi_log2;
    int32_t nbins;
    int32_t reserved; /* must be 0 */
} peat_bins_t;

/* Closeness tests j < count (0 <= count <= 8), each an absolute tolerance
 * abs_tol[j] and a relative tolerance rel_tol[j], both >= 0 and not NaN
 * (+Inf allowed).  n_mismatch[j] counts the pairs that torch.isclose(test,
 * golden, rtol=rel_tol[j], atol=abs_tol[j], equal_nan=False) calls not close
 * (Section III-A): NaN pairs, and unequal pairs whose error is infinite or
 * exceeds abs_tol[j] + |rel_tol[j] * G| (product and sum rounded
 * separately).  rel_tol = 0 is the absolute test. */
typedef struct {
    int32_t count;
    int32_t reserved; /* must be 0 */
    double abs_tol[PEAT_MAX_THRESHOLDS];
    double rel_tol[PEAT_MAX_THRESHOLDS];
} peat_thresholds_t;

/* The error signature of one pair.  G_i, T_i are the values widened to
 * binary64; a pair is "valid" when neither side is NaN, "finite" when both
 * sides are finite, "rel" when finite with G_i != 0.  For a valid pair the
 * error is a_i = 0 if G_i == T_i (IEEE equality), else |RN(T_i - G_i)|; the
 * ULP distance is |key(t_i) - key(g_i)| with key = +magnitude or -magnitude
 * of the bit pattern; the relative error is r_i = RN(a_i / |G_i|).
 * Maxima use strict > over increasing i, so ties go to the lowest index.
 * With no eligible pair a maximum is NaN (ULP: 0) and its index -1. */
typedef struct {
    int64_t n, n_valid, n_finite, n_rel;
    int64_t n_nan_golden, n_nan_test, n_inf_golden, n_inf_test;
    int64_t n_nan_pairs;     /* pairs with a NaN on either side            */
    int64_t first_nan_index; /* lowest index of such a pair, or -1         */
    int64_t n_mismatch[PEAT_MAX_THRESHOLDS]; /* first thresholds.count used */
    int64_t hist_zero, hist_under, hist_over;
    int64_t hist[PEAT_MAX_BINS];             /* first bins.nbins used       */
    double max_abs;
    int64_t argmax_abs;      /* over valid pairs */
    int64_t max_ulp;
    int64_t argmax_ulp;      /* over valid pairs */
    uint64_t sum_ulp;        /* over valid pairs */
    double max_rel;
    int64_t argmax_rel;      /* over rel pairs */
    /* binary64 sums over finite pairs (sum_rel over rel pairs): sum a_i,
     * sum RN(a_i^2), sum G_i^2, sum T_i^2, sum G_i*T_i.  Summation order is a
     * fixed tree, identical for every call with the same n and dtype. */
    double sum_abs, sum_sq, sum_rel, sum_g2, sum_t2, sum_gt;
} peat_signature_t;

/* Scores derived on the host from a signature (Section IV-B.3 mean and
 * variance; the variance is the sample variance over finite pairs). */
typedef struct {
    double mean_abs, var_abs, l2_err, l2_g, l2_t, cos, mean_rel, mean_ulp;
} peat_stats_t;

/* Mean of the top errors of one pair (Section IV-B.3, "Mean of Top 10%
 * Errors", the Analyzer's main score in Section IV-C): the k largest errors
 * a_i = |T_i - G_i| (the signature's error) over the valid pairs, with
 * k = ceil(n_valid * num / den). */
typedef struct {
    int64_t n_valid;      /* pairs with no NaN on either side */
    int64_t k;            /* ceil(n_valid * num / den) */
    int64_t count_above;  /* errors strictly greater than kth_value (< k) */
    double kth_value;     /* the k-th largest error; NaN when k = 0 */
    double sum_topk;      /* sum of the k largest errors; 0 when k = 0; +Inf
                           * when one of them is infinite */
    double mean_topk;     /* sum_topk / k; NaN when k = 0 */
} peat_topk_t;

typedef struct {
    const void *golden; /* device pointer */
    const void *test;   /* device pointer */
    int64_t n;          /* elements, >= 0 */
    int32_t dtype;      /* peat_dtype_t   */
    int32_t reserved;   /* must be 0      */
} peat_pair_t;

/* A pair whose golden and test types may differ (Section III-C: an FP32
 * golden output against the same operation run in FP16, or in FP64 for the
 * FP32-FP64 "error unit").  golden_dtype is PEAT_F32, PEAT_F16 or PEAT_BF16;
 * test_dtype may also be PEAT_F64; one format must contain the other
 * (PEAT_F16 with PEAT_BF16 is PEAT_EDTYPE).  Equal types are allowed.  Each
 * pointer must be aligned to its element size (PEAT_EINVAL otherwise). */
typedef struct {
    const void *golden; /* device pointer */
    const void *test;   /* device pointer */
    int64_t n;          /* elements of each, >= 0 */
    int32_t golden_dtype;
    int32_t test_dtype;
} peat_mixed_pair_t;

/* Error models (Section II-B "Error Models"; Section III-C pseudo-errors;
 * Section V-A draws a random value from the target tensor's distribution). */
typedef enum {
    PEAT_MODEL_BITFLIP = 0, /* toggle one bit of the mask (random bit flip)      */
    PEAT_MODEL_ZERO = 1,    /* set to +0 (random zero)                            */
    PEAT_MODEL_VALUE = 2,   /* the uncorrupted tensor's value at a random index
                             * (random value from the tensor's own distribution) */
    PEAT_MODEL_NAN = 3,     /* set to the quiet NaN 0x7FC00000 / 0x7E00 / 0x7FC0 */
    PEAT_MODEL_UNIFORM = 4  /* a uniformly random bit pattern of the type
                             * (random value over the type: may be Inf or NaN)   */
} peat_model_t;

#define PEAT_MAX_POSITIONS 4096

typedef struct {
    void *tensor;     /* device pointer, modified in place, aligned to its
                       * element size (PEAT_EINVAL otherwise) */
    int64_t n;        /* elements, >= 0 */
    int32_t dtype;    /* peat_dtype_t   */
    int32_t model;    /* peat_model_t */
    uint64_t seed;
    double rate;      /* error rate per element; >= 1 chooses every element */
    uint64_t bitmask; /* BITFLIP: candidate bits, nonzero, below the type
                       * width; ignored by the other models */
} peat_inject_item_t;

/* Static text for a PEAT_E* code; never NULL. */
const char *peat_strerror(int code);

/* Thread-local detail of the last error returned on this thread ("" if none). */
const char *peat_last_error(void);

/* PEAT_ABI_VERSION of the loaded library. */
int peat_abi_version(void);

/* Optional explicit initialisation of the current device (checks that it is
 * gfx950).  Every entry point does this lazily.  Returns 0 or PEAT_ENODEV /
 * PEAT_EHIP. */
int peat_init(void);

/* Stream (a hipStream_t, NULL = null stream) used by the synchronous calls of
 * the calling host thread. */
int peat_set_stream(void *stream);

/* Error signature of one pair: the Err(golden, FI) step of Algorithms 1 and
 * 2 for one recorded tensor, with the scores of Section IV-B.3 (error =
 * absolute difference; max, mean, variance), the closeness counts of
 * Section III-A and the error histogram of Section V-D.  golden and test are
 * device arrays of n elements of dtype (any alignment; 16-byte aligned
 * pairs take the vector path); bins and thresholds as above; out is host
 * memory, written when the call returns.  n = 0 is valid and gives zero
 * counts, NaN maxima and -1 indices.  PEAT_EINVAL for NULL tensors with
 * n > 0, n < 0 or n > 2^46, bad bins or thresholds; PEAT_EDTYPE for an
 * unknown dtype. */
int peat_signature(const void *golden, const void *test, int64_t n, peat_dtype_t dtype,
                   const peat_bins_t *bins, const peat_thresholds_t *thresholds,
                   peat_signature_t *out);

/* Signatures of count >= 0 pairs in one launch sequence: Err() over the N
 * recorded tensors of Algorithm 1 (the outputs of one kernel) or of a
 * training step in Algorithm 2, each pair as in peat_signature.  pairs is a
 * host array of count descriptors, copied before the call returns; outs is
 * a host array of count records.  Each record is bit-identical to the one
 * peat_signature gives for the same pair.  Errors as peat_signature's, per
 * pair, plus PEAT_EINVAL for count < 0 or NULL arrays. */
int peat_signature_batched(const peat_pair_t *pairs, int32_t count,
                           const peat_bins_t *bins, const peat_thresholds_t *thresholds,
                           peat_signature_t *outs);

/* As peat_signature_batched (the Err step of Algorithms 1 and 2), enqueued
 * on stream (a hipStream_t; NULL is the null stream): d_outs is a device
 * array of count records written when the stream reaches the work; the call
 * returns without waiting.  The golden and test tensors must stay allocated
 * and unchanged until then. */
int peat_signature_batched_async(const peat_pair_t *pairs, int32_t count,
                                 const peat_bins_t *bins, const peat_thresholds_t *thresholds,
                                 peat_signature_t *d_outs, void *stream);

/* For callers that cannot allocate memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  The same work and
 * records (bit-identical) as peat_signature_batched_async on the same
 * arguments, but every intermediate buffer -- pair descriptors (48 bytes per
 * pair), chunk map and chunk records (612 bytes per chunk), the first two
 * parts each rounded up to 256 bytes -- lives in one static device array of
 * PEAT_NOALLOC_SCRATCH_BYTES that every GPU the library runs on holds until
 * the process ends.  A pair of n elements has ceil(n / C) chunks, C the
 * smallest power of two in [2^12, 2^18] that is at least n / 256 (n < 2^22)
 * or n / 64 (n >= 2^22).  The call makes no device, pinned or host-heap
 * allocation; the device's one-time set-up does (events, the array's
 * address), so call peat_init() on each device first when that matters.
 * pairs is host memory read before the call returns (descriptors travel as
 * kernel arguments); d_outs is a device array of count records written when
 * the stream reaches the work.  Every call on one GPU uses the same array
 * and it keeps the last call's contents (nothing in it needs clearing):
 * calls on one GPU that can run at the same time (other streams, no ordering
 * between them) race on it and give wrong records -- order them.
 * PEAT_EINVAL, before any device access, when a batch needs more than
 * PEAT_NOALLOC_SCRATCH_BYTES; other errors as peat_signature_batched_async. */
#define PEAT_NOALLOC_SCRATCH_BYTES (64u << 20)
int peat_signature_batched_noalloc(const peat_pair_t *pairs, int32_t count,
                                   const peat_bins_t *bins, const peat_thresholds_t *thresholds,
                                   peat_signature_t *d_outs, void *stream);

/* One step of the assessment in a single pass over the data: the random bit
 * flips of peat_inject (Section II-B; same generator and decisions) are
 * applied to every pair's test tensor in place, with seed seeds[k], the
 * given rate and bitmask (valid for every pair's dtype), and the signatures
 * of the pairs (golden, flipped test) are computed -- records, tensor bits
 * and counts equal to peat_inject_batched followed by
 * peat_signature_batched.  When every test tensor starts on a 128-byte
 * boundary and no 128-byte line holding test bytes holds bytes of another
 * tensor of the batch (separately allocated tensors always qualify), each
 * chunk of a test tensor is flipped (atomic bit toggles) before it is read,
 * in the same kernel; any other batch runs as the injection kernel followed
 * by the signature pass, with the same results.  seeds is a host array
 * of count seeds; d_outs a device array of count records and d_counts a
 * device int64 array of count flip counts, written when the stream reaches
 * the work.  Test tensors must not overlap one another or any golden tensor
 * (PEAT_EINVAL); PEAT_ERATE for a NaN or negative rate, PEAT_EBITMASK for a
 * bitmask that is 0 or reaches beyond a pair's type width. */
int peat_inject_signature_batched_async(const peat_pair_t *pairs, int32_t count, const uint64_t *seeds,
                                        double rate, uint64_t bitmask, const peat_bins_t *bins,
                                        const peat_thresholds_t *thresholds, peat_signature_t *d_outs,
                                        int64_t *d_counts, void *stream);

/* Signature of a mixed-precision pair (Section III-C; types as in
 * peat_mixed_pair_t).  Every field keeps its definition over the exact
 * binary64 values of both sides, except the ULP distance, which is counted
 * in the narrower format after rounding the wider value to it (nearest, ties
 * to even, Inf beyond its range).  With equal types the record equals
 * peat_signature's.  out is host memory; the call waits for it. */
int peat_signature_mixed(const void *golden, int32_t golden_dtype, const void *test,
                         int32_t test_dtype, int64_t n, const peat_bins_t *bins,
                         const peat_thresholds_t *thresholds, peat_signature_t *out);

/* peat_signature_mixed over count >= 0 pairs of any accepted type
 * combination in one launch sequence; outs is a host array of count records,
 * each bit-identical to the single call's. */
int peat_signature_mixed_batched(const peat_mixed_pair_t *pairs, int32_t count,
                                 const peat_bins_t *bins, const peat_thresholds_t *thresholds,
                                 peat_signature_t *outs);

/* As peat_signature_mixed_batched, enqueued on stream; d_outs is a device
 * array of count records written when the stream reaches the work. */
int peat_signature_mixed_batched_async(const peat_mixed_pair_t *pairs, int32_t count,
                                       const peat_bins_t *bins, const peat_thresholds_t *thresholds,
                                       peat_signature_t *d_outs, void *stream);

/* Mean of the k largest errors of one pair, k = ceil(n_valid * num / den)
 * (num = 1, den = 10: the paper's top-10% mean of Section IV-B.3, the
 * Analyzer's main score in Section IV-C); out is host memory.
 * 1 <= num <= den <= 2^20.  Exact selection: n_valid, k, count_above and
 * kth_value are exact.  sum_topk is the binary64 sum, in a fixed order, of
 * the errors above the binade of kth_value plus the exact sum of the others
 * (within 1e-12 relative of the exact sum), bit-identical between calls and
 * between the entry points below (the signature-fed ones as they state).
 * One streaming pass over golden and test in the common case: a small
 * strided sample of each pair (about 8 K elements) guesses the binade of the
 * k-th largest error, and one pass sums the errors above it, gathers its
 * errors and counts the pair's errors, which confirm the guess; a wrong
 * guess, a pair below 2^16 elements, or one whose sampled binade holds many
 * distinct errors takes a binade-histogram pass first (two passes).  A pair
 * whose binade holds too many distinct errors for the gather takes one more
 * pass (a gather of its top 13 mantissa bits), and one whose bin still does
 * not fit one pass per remaining digit.  Every route gives the same record.
 * No step waits on the host; the call waits for its result. */
int peat_topk_mean(const void *golden, const void *test, int64_t n, peat_dtype_t dtype,
                   int32_t num, int32_t den, peat_topk_t *out);

/* peat_topk_mean over count >= 0 pairs in one launch sequence; outs is a
 * host array of count records, each bit-identical to the single call's. */
int peat_topk_mean_batched(const peat_pair_t *pairs, int32_t count, int32_t num, int32_t den,
                           peat_topk_t *outs);

/* As peat_topk_mean_batched, enqueued on stream (NULL: the default stream):
 * d_outs is a device array of count records written when the stream gets
 * there; the call returns without waiting.  The tensors must stay valid and
 * unchanged until then.  (Section IV-B.3.) */
int peat_topk_mean_batched_async(const peat_pair_t *pairs, int32_t count, int32_t num, int32_t den,
                                 peat_topk_t *d_outs, void *stream);

/* peat_topk_mean_batched over mixed-precision pairs (types as in
 * peat_mixed_pair_t; the error is |T - G| of the exact binary64 values). */
int peat_topk_mean_mixed_batched(const peat_mixed_pair_t *pairs, int32_t count, int32_t num,
                                 int32_t den, peat_topk_t *outs);

/* As peat_topk_mean_mixed_batched, enqueued on stream; d_outs as in
 * peat_topk_mean_batched_async. */
int peat_topk_mean_mixed_batched_async(const peat_mixed_pair_t *pairs, int32_t count, int32_t num,
                                       int32_t den, peat_topk_t *d_outs, void *stream);

/* peat_topk_mean_batched for pairs whose error signatures the caller already
 * holds: sigs is a host array of count records that peat_signature_batched
 * (or its async form) wrote for the same pairs with these bins; thresholds do
 * not matter.  The histogram counts the same errors of the same valid pairs,
 * so it bounds the k-th largest error to one bin, and the binade histogram
 * pass skips the pair: one streaming pass does the rest.  With one-binade
 * bins (hi_log2 - lo_log2 == nbins) and the boundary in a regular bin (or,
 * with a test type other than binary64, among the zero errors) that bin is
 * the boundary's binade, and outs are bit-identical to
 * peat_topk_mean_batched's.  Otherwise (the under or over bin, or wider
 * bins) the pass gathers the bin's whole range of binades, and n_valid, k,
 * count_above and kth_value are identical while sum_topk and mean_topk are
 * formed in another order (within 1e-12 relative; equal whenever the errors
 * inside the range sum exactly in binary64).  A range with too many
 * distinct errors for the gather falls back to the binade pass (and then
 * bit-identical records).  PEAT_EINVAL when a record's n differs from its
 * pair's or its histogram total from its n_valid.  (Section IV-B.3;
 * Section V-D histograms.) */
int peat_topk_mean_from_signature_batched(const peat_pair_t *pairs, int32_t count, int32_t num,
                                          int32_t den, const peat_signature_t *sigs,
                                          const peat_bins_t *bins, peat_topk_t *outs);

/* As peat_topk_mean_from_signature_batched, enqueued on stream: d_sigs is a
 * device array of count records (as peat_signature_batched_async or
 * peat_inject_signature_batched_async leave them, possibly still being
 * written earlier on the same stream), d_outs a device array of count
 * records written when the stream gets there.  A record whose n or
 * histogram total does not match is ignored (its pair takes the binade
 * pass), so a mismatch costs time, not correctness. */
int peat_topk_mean_from_signature_batched_async(const peat_pair_t *pairs, int32_t count, int32_t num,
                                                int32_t den, const peat_signature_t *d_sigs,
                                                const peat_bins_t *bins, peat_topk_t *d_outs,
                                                void *stream);

/* peat_topk_mean_from_signature_batched over mixed-precision pairs, with the
 * records of peat_signature_mixed_batched (or its async form) for the same
 * pairs and bins; outs relate to peat_topk_mean_mixed_batched's as above. */
int peat_topk_mean_mixed_from_signature_batched(const peat_mixed_pair_t *pairs, int32_t count,
                                                int32_t num, int32_t den, const peat_signature_t *sigs,
                                                const peat_bins_t *bins, peat_topk_t *outs);

/* As peat_topk_mean_mixed_from_signature_batched with device records,
 * enqueued on stream (as peat_topk_mean_from_signature_batched_async). */
int peat_topk_mean_mixed_from_signature_batched_async(const peat_mixed_pair_t *pairs, int32_t count,
                                                      int32_t num, int32_t den,
                                                      const peat_signature_t *d_sigs,
                                                      const peat_bins_t *bins, peat_topk_t *d_outs,
                                                      void *stream);

/* Entry capacity of the top-k gathers for later calls of this process:
 * binade_entries for the gathers of a whole binade, bin_entries for the
 * gathers of one 13-bit bin (16 bytes of device workspace each).  -1 (the
 * default) sizes them per call: max(2^16, 256 x chunks) and max(2^16,
 * 64 x chunks), a chunk being one block's share of a pair.  A pair whose
 * gather does not fit takes the next, slower route; the records do not
 * change.  Each value must be -1 or in [0, 2^36]. */
int peat_topk_set_entry_capacity(int64_t binade_entries, int64_t bin_entries);

/* Random bit flip in place (Section II-B).  The draws come from
 * Philox4x32-10 keyed by (lo32(seed), hi32(seed)); "block c of stream s" is
 * its output at counter (lo32(c), hi32(c), s, 0), four 32-bit words, bytes
 * and 64-bit words (words 2h, 2h+1) numbered little-endian.  Element i flips
 * iff its 64-bit uniform U_i < floor(rate * 2^64) (every element if
 * rate >= 1).  U_i's top byte is byte (i mod 16) of block i/16 of stream 0;
 * its low 56 bits are the low 56 bits of 64-bit word (i mod 2) of block i/2
 * of stream 1.  A flipped element toggles the j-th lowest set bit of bitmask,
 * j = floor(y * popcount(bitmask) / 2^32) with y = word 0 of block i of
 * stream 2.  Returns the number of flipped elements (>= 0) or a negative
 * PEAT_E* code.  Applying the same call twice restores the tensor. */
int64_t peat_inject(void *tensor, int64_t n, peat_dtype_t dtype, uint64_t seed,
                    double rate, uint64_t bitmask);

/* peat_inject with another error model at the same rate (Section II-B):
 * the elements peat_inject would flip (same seed and rate) are set to +0
 * (PEAT_MODEL_ZERO), to the type's quiet NaN (PEAT_MODEL_NAN), bit-flipped
 * (PEAT_MODEL_BITFLIP, identical to peat_inject), to the value the tensor
 * held before the call at index floor(W * n / 2^64), W the 64-bit word 0 of
 * block i of stream 4 (PEAT_MODEL_VALUE: a value of the tensor's own
 * distribution, Section V-A; the library copies the tensor to its workspace
 * first, n * element size bytes), or to word 2 of that block cut to the
 * type's width (PEAT_MODEL_UNIFORM).  bitmask is used by BITFLIP only.
 * Returns the number of chosen elements or a negative code. */
int64_t peat_inject_model(void *tensor, int64_t n, peat_dtype_t dtype, uint64_t seed, double rate,
                          int32_t model, uint64_t bitmask);

/* The paper's num_pos corruption (Section V-A): exactly num_pos distinct
 * positions, 0 <= num_pos <= min(n, PEAT_MAX_POSITIONS).  Draw j = 0, 1, ...
 * takes block j of stream 3 (peat_inject's generator), its 64-bit words W0
 * and W1, and the index floor(W0 * n / 2^64); the positions are the first
 * num_pos distinct indices in order of appearance.  Each becomes +0, the
 * quiet NaN, a bit flip (peat_inject's bit rule for that index), the low
 * bits (the type's width) of W1 as a uniformly random bit pattern
 * (PEAT_MODEL_UNIFORM), or -- PEAT_MODEL_VALUE, a value from the tensor's
 * own distribution -- the uncorrupted tensor's value at
 * floor(W1 * n / 2^64) of the draw that chose it.  positions (host,
 * num_pos entries, may be NULL) receives the positions in order.  Returns
 * num_pos or a negative code (PEAT_EINVAL also for a tensor not aligned to
 * its element size); waits for the device. */
int64_t peat_corrupt_positions(void *tensor, int64_t n, peat_dtype_t dtype, uint64_t seed, int32_t model,
                               int64_t num_pos, uint64_t bitmask, int64_t *positions);

/* The FP16 / BF16 error of Section III-C: every element of an f32 tensor
 * (device, in place) becomes its round-to-nearest-even value in to_dtype
 * (PEAT_F16 or PEAT_BF16) widened back to f32; overflow gives +-Inf,
 * subnormals round correctly, a NaN becomes sign | 0x7FC00000.  The tensor
 * must be 4-byte aligned (PEAT_EINVAL otherwise).  Enqueued on the calling
 * thread's stream (peat_set_stream); does not wait. */
int peat_cast_round(void *tensor, int64_t n, peat_dtype_t to_dtype);

/* peat_inject over count >= 0 items in one launch sequence; counts is a host
 * array receiving each item's flip count (chosen elements for ZERO/NAN). */
int peat_inject_batched(const peat_inject_item_t *items, int32_t count, int64_t *counts);

/* As peat_inject_batched, enqueued on stream; d_counts is a device int64
 * array written when the stream reaches the work. */
int peat_inject_batched_async(const peat_inject_item_t *items, int32_t count,
                              int64_t *d_counts, void *stream);

/* Measurement aid, not a step of the method: reads `bytes` bytes of device
 * memory at `buf` (16-byte aligned, bytes a multiple of 16) with the access
 * pattern of the signature chunk pass (16-byte nontemporal loads per lane,
 * 256-thread blocks, a contiguous 2 MiB span per block) and writes the XOR of
 * the 32-bit words of span k (bytes [k 2^21, (k+1) 2^21) of buf) to
 * d_sink[k], so that no read can be dropped.  d_sink is a device array of at
 * least ceil(bytes / 2^21) uint32 words, 4-byte aligned.  Enqueued on
 * `stream` (NULL: the default stream); timed as kernel class 4.  Its byte
 * rate is the read ceiling of this access pattern on the device.  Returns
 * PEAT_EINVAL for bad sizes, alignment or NULL pointers. */
int peat_stream_read(const void *buf, int64_t bytes, uint32_t *d_sink, void *stream);

/* Analyzer statistics over a series of scores (host memory in and out):
 * count of the non-NaN entries, their mean, sample variance (divisor
 * count - 1) and standard deviation, minimum and maximum -- the (mu, sigma)
 * of one operator's scores across epochs (Section IV-C) and the Detector's
 * ranges.  Fields without enough entries are NaN. */
typedef struct {
    int64_t count;
    double mean, var, std, min, max;
} peat_series_t;
int peat_series_stats(const double *x, int64_t n, peat_series_t *out);

/* Spearman's rank correlation of the pairs (x[i], y[i]) with no NaN: the
 * Pearson correlation of average ranks (ties share the mean rank), as the
 * Analyzer correlates scores with model metrics (Section IV-C).  *rho is NaN
 * for fewer than two pairs or constant ranks.  Host memory. */
int peat_spearman(const double *x, const double *y, int64_t n, double *rho);

/* out[i] = scores[i] / units[i]: scores in units of the FP64 error's score
 * (Section V-C), IEEE division.  Host memory. */
int peat_normalize_scores(const double *scores, const double *units, int64_t n, double *out);

/* Host-side derived scores of a signature (host memory in and out). */
int peat_finalize_stats(const peat_signature_t *sig, peat_stats_t *stats);

/* Kernel timing.  When enabled, every launch of the library's kernels is
 * bracketed by HIP events on its stream.  peat_profile_read waits for those
 * events, returns the summed duration (ms) and launch count of one kernel
 * class since the last read, and clears that class.  Kernel classes:
 * 0 signature chunk pass, 1 signature finalize, 2 injection, 3 injection
 * count reduction, 4 streaming read (peat_stream_read), 5 top-k level 0
 * (state, binade histogram pass, selection), 6 top-k from the gathering pass
 * to the records, 7 chunk pass with the injection
 * (peat_inject_signature_batched_async). */
int peat_profile_enable(int on);
int peat_profile_read(int kernel_class, double *total_ms, int64_t *launches);

#ifdef __cplusplus
}
#endif

#endif /* PEAT_H */
