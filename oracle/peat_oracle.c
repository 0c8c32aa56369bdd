/*
 * PEAT oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, scalar CPU implementation of the two operations on the hot
 * path of PEAT's pseudo-error assessment:
 *
 *   oracle_signature  the Analyzer's comparison of a golden tensor with a test
 *                     tensor ("FI Assessment Scores", Section IV-B: the error is
 *                     the absolute difference of golden and fault-injected
 *                     values; max, mean and variance of it), extended to the
 *                     error signature: per-element relative error, ULP distance,
 *                     a log2-binned error histogram (Section V-D, error value
 *                     histograms), NaN/Inf counts, absolute-threshold mismatch
 *                     counts (the closeness test of Section III-A, torch.isclose
 *                     with rtol = 0), maxima with the lowest index, and the fp64
 *                     sums from which L2 norms and the cosine follow.
 *
 *   oracle_inject     the random-bit-flip error model (Section II-B, "Error
 *                     Models": parameters flip at a given bit error rate), used
 *                     by Inject() in Playback FI (Algorithm 1) and Runtime FI
 *                     (Algorithm 2).
 *
 *   oracle_inject_model, oracle_corrupt_positions, oracle_cast_round
 *                     the paper's other error models (Section II-B "Error
 *                     Models"; Section III-C pseudo-errors; Section V-A
 *                     settings): random zero, random NaN and bit flip at a
 *                     rate; random value, random zero, random NaN or bit flip
 *                     at num_pos distinct random positions; the FP16 (and
 *                     BF16) error, a round-to-nearest-even cast of an FP32
 *                     tensor.
 *
 *   oracle_series_stats, oracle_spearman, oracle_normalize
 *                     the Analyzer's statistics over score series (Section
 *                     IV-C: model-wise (mean, std) of errors across epochs,
 *                     Spearman rank correlation with model metrics; Section
 *                     V-C: scores normalised by the FP64 error's score).
 *
 *   oracle_signature_mixed, oracle_topk_mixed
 *                     the same two definitions for a golden and a test of
 *                     different precision (Section III-C: Err(FP16, FP32),
 *                     the FP32-FP64 error); the ULP distance of such a pair
 *                     is counted in the narrower format.
 *
 *   oracle_topk       the "mean of the top 10% errors" score (Section IV-B,
 *                     FI Assessment Scores; the Analyzer's main score,
 *                     Section IV-C), for any fraction num/den: the errors of
 *                     the valid pairs sorted in decreasing order, the k largest
 *                     summed, k = ceil(n_valid * num / den).
 *
 * Only the tests, the package smoke check and the benchmark's CPU-baseline leg
 * may load this file's library.  It shares no code, header, table or constant
 * generator with the GPU library; the two are independent by construction.
 *
 * Arithmetic: IEEE binary64, round-to-nearest-even, compiled without
 * contraction or fast-math.  Elements are scanned in increasing index order.
 * Floating-point sums use Neumaier's compensated summation.
 *
 * Every field has a pin in the CPU test suite (closed forms, brute force over
 * the fp16 grid with exact rational arithmetic, math.fsum, torch float64
 * library routines, the Random123 known-answer vectors and rocRAND's
 * Philox4x32-10).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_F32 0
#define ORACLE_F16 1
#define ORACLE_BF16 2
#define ORACLE_F64 3   /* test side of a mixed-precision pair only */

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)
#define ORACLE_EDTYPE (-2)
#define ORACLE_EBITMASK (-3)
#define ORACLE_ERATE (-4)
#define ORACLE_ENOMEM (-6)

typedef struct {
    int64_t n, n_valid, n_finite, n_rel;
    int64_t n_nan_golden, n_nan_test, n_inf_golden, n_inf_test, n_nan_pairs, first_nan_index;
    int64_t n_mismatch[8];
    int64_t hist_zero, hist_under, hist_over;
    int64_t hist[64];
    double max_abs;
    int64_t argmax_abs;
    int64_t max_ulp;
    int64_t argmax_ulp;
    uint64_t sum_ulp;
    double max_rel;
    int64_t argmax_rel;
    double sum_abs, sum_sq, sum_rel, sum_g2, sum_t2, sum_gt;
} oracle_sig_t;

typedef struct {
    double mean_abs, var_abs, l2_err, l2_g, l2_t, cos, mean_rel, mean_ulp;
} oracle_stats_t;

/* ------------------------------------------------------------------------- */
/* Decoding: bit pattern of element i -> its exact binary64 value.           */
/* ------------------------------------------------------------------------- */

static int dtype_width(int dtype) {
    if (dtype == ORACLE_F32) return 32;
    if (dtype == ORACLE_F16 || dtype == ORACLE_BF16) return 16;
    return 0;
}

static uint32_t element_bits(const void *base, int64_t i, int dtype) {
    if (dtype == ORACLE_F32) {
        uint32_t b;
        memcpy(&b, (const unsigned char *)base + 4 * i, 4);
        return b;
    }
    uint16_t h;
    memcpy(&h, (const unsigned char *)base + 2 * i, 2);
    return h;
}

/* IEEE binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
static double half_value(uint32_t h) {
    int sign = (h >> 15) & 1;
    int expo = (h >> 10) & 0x1F;
    int frac = h & 0x3FF;
    double v;
    if (expo == 0x1F)
        v = frac ? NAN : INFINITY;
    else if (expo == 0)
        v = ldexp((double)frac, -24);            /* subnormal: frac * 2^-24 */
    else
        v = ldexp((double)(frac | 0x400), expo - 25); /* (1.frac) * 2^(expo-15) */
    return sign ? -v : v;
}

static double element_value(uint32_t bits, int dtype) {
    if (dtype == ORACLE_F16) return half_value(bits);
    float f;
    uint32_t b = (dtype == ORACLE_BF16) ? (bits << 16) : bits; /* bf16 = top half of binary32 */
    memcpy(&f, &b, 4);
    return (double)f; /* widening binary32 -> binary64 is exact */
}

/* Distance in units in the last place: the signed-magnitude bit pattern is
 * mapped to an integer key (+magnitude or -magnitude, so +0 and -0 coincide),
 * and the ULP distance is the absolute difference of the keys. */
static int64_t ulp_key(uint32_t bits, int width) {
    uint32_t sign_bit = 1u << (width - 1);
    int64_t mag = (int64_t)(bits & (sign_bit - 1));
    return (bits & sign_bit) ? -mag : mag;
}

/* ---- mixed-precision pairs (Section III-C: an FP32 golden output against
 * the output of the same operation in FP16 or in FP64) ------------------- */

/* Value of element i of any supported type, exactly as a binary64. */
static double element_value_any(const void *base, int64_t i, int dtype) {
    if (dtype == ORACLE_F64) {
        double d;
        memcpy(&d, (const unsigned char *)base + 8 * i, 8);
        return d;
    }
    return element_value(element_bits(base, i, dtype), dtype);
}

/* Precision p (significand bits, implicit bit included) and the normal
 * exponent range [emin, emax] of each type. */
static void format_params(int dtype, int *p, int *emin, int *emax) {
    switch (dtype) {
        case ORACLE_F16: *p = 11; *emin = -14; *emax = 15; break;
        case ORACLE_BF16: *p = 8; *emin = -126; *emax = 127; break;
        case ORACLE_F64: *p = 53; *emin = -1022; *emax = 1023; break;
        default: *p = 24; *emin = -126; *emax = 127; break;
    }
}

/* Golden and test types that a signature accepts: the golden is FP32, FP16
 * or BF16 (the golden kernel is never the binary64 one); the test may also be
 * binary64; and one format must contain the other (precision and both
 * exponent limits), which excludes FP16 against BF16. */
static int pair_types_ok(int gdt, int tdt) {
    if (!dtype_width(gdt)) return 0;
    if (!dtype_width(tdt) && tdt != ORACLE_F64) return 0;
    int pg, ming, maxg, pt, mint, maxt;
    format_params(gdt, &pg, &ming, &maxg);
    format_params(tdt, &pt, &mint, &maxt);
    int g_in_t = pg <= pt && ming >= mint && maxg <= maxt;
    int t_in_g = pt <= pg && mint >= ming && maxt <= maxg;
    return g_in_t || t_in_g;
}

/* Position of a value of a format in the ordered list of that format's
 * non-negative values (0, the subnormals, the normals, then Inf), negated for
 * a negative value; v is exactly representable in the format, or infinite.
 * For a value decoded from a bit pattern this is the signed-magnitude key of
 * the pattern. */
static int64_t format_index(double v, int p, int emin, int emax) {
    double a = fabs(v);
    int64_t idx;
    if (isinf(a)) {
        idx = (int64_t)(emax - emin + 2) << (p - 1);
    } else if (a < ldexp(1.0, emin)) {
        idx = (int64_t)(a / ldexp(1.0, emin - p + 1));       /* subnormal: multiple of the quantum */
    } else {
        int e;
        frexp(a, &e);
        int E = e - 1;                                       /* a in [2^E, 2^(E+1)) */
        int64_t m = (int64_t)(a / ldexp(1.0, E - p + 1));    /* significand in [2^(p-1), 2^p) */
        idx = ((int64_t)(E - emin) << (p - 1)) + m;
    }
    return v < 0 ? -idx : idx;
}

/* ------------------------------------------------------------------------- */
/* Neumaier compensated summation.                                           */
/* ------------------------------------------------------------------------- */

typedef struct { double s, c; } csum_t;

static void csum_add(csum_t *acc, double x) {
    double t = acc->s + x;
    if (fabs(acc->s) >= fabs(x))
        acc->c += (acc->s - t) + x;
    else
        acc->c += (x - t) + acc->s;
    acc->s = t;
}

/* An infinite or NaN running sum is the IEEE value of the whole sum: the
 * compensation term only corrects rounding, and infinities turn it into NaN. */
static double csum_value(const csum_t *acc) { return isfinite(acc->s) ? acc->s + acc->c : acc->s; }

/* ------------------------------------------------------------------------- */
/* The error signature.                                                      */
/* ------------------------------------------------------------------------- */

/* Validation of the histogram and thresholds (same acceptance rules as the
 * library: -1022 <= lo < hi <= 1024, 1 <= nbins <= 64, nbins divides hi-lo;
 * 0 <= nthr <= 8 thresholds, each absolute and relative tolerance >= 0 and
 * not NaN). */
static int check_params(int lo, int hi, int nbins, int nthr, const double *thr, const double *rthr) {
    if (lo < -1022 || hi > 1024 || lo >= hi) return ORACLE_EINVAL;
    if (nbins < 1 || nbins > 64 || (hi - lo) % nbins != 0) return ORACLE_EINVAL;
    if (nthr < 0 || nthr > 8) return ORACLE_EINVAL;
    if (nthr > 0 && !thr) return ORACLE_EINVAL;
    for (int j = 0; j < nthr; ++j) {
        if (isnan(thr[j]) || thr[j] < 0) return ORACLE_EINVAL;
        if (rthr && (isnan(rthr[j]) || rthr[j] < 0)) return ORACLE_EINVAL;
    }
    return ORACLE_OK;
}

static double round_to_format(double v, int p, int emin, int emax);

int oracle_signature_mixed(const void *golden, int gdt, const void *test, int tdt, int64_t n,
                           int lo, int hi, int nbins, int nthr, const double *thr, const double *rthr,
                           oracle_sig_t *out);
int oracle_signature_rtol(const void *golden, const void *test, int64_t n, int dtype,
                          int lo, int hi, int nbins, int nthr, const double *thr, const double *rthr,
                          oracle_sig_t *out);

int oracle_signature(const void *golden, const void *test, int64_t n, int dtype,
                     int lo, int hi, int nbins, int nthr, const double *thr,
                     oracle_sig_t *out) {
    return oracle_signature_rtol(golden, test, n, dtype, lo, hi, nbins, nthr, thr, NULL, out);
}

/* The signature with the closeness test of torch.isclose(T, G, rtol, atol)
 * (Section III-A): threshold j has the absolute tolerance thr[j] and the
 * relative tolerance rthr[j] (rthr NULL: all 0). */
int oracle_signature_rtol(const void *golden, const void *test, int64_t n, int dtype,
                          int lo, int hi, int nbins, int nthr, const double *thr, const double *rthr,
                          oracle_sig_t *out) {
    if (!dtype_width(dtype)) return ORACLE_EDTYPE;
    return oracle_signature_mixed(golden, dtype, test, dtype, n, lo, hi, nbins, nthr, thr, rthr, out);
}

/* The signature of a pair whose golden and test types may differ (Section
 * III-C: Err(FP16, FP32) and the FP32-FP64 error).  Both values are taken
 * exactly as binary64 and every field keeps its definition, except the ULP
 * distance of a mixed pair, which is counted in the narrower format: the
 * wider value is first rounded to it (nearest, ties to even, Inf beyond its
 * range). */
int oracle_signature_mixed(const void *golden, int gdt, const void *test, int tdt, int64_t n,
                           int lo, int hi, int nbins, int nthr, const double *thr, const double *rthr,
                           oracle_sig_t *out) {
    if (!pair_types_ok(gdt, tdt)) return ORACLE_EDTYPE;
    int width = dtype_width(gdt);
    int mixed = gdt != tdt;
    int np_, nemin, nemax;           /* the narrower format of a mixed pair */
    {
        int pg, ming, maxg, pt, mint, maxt;
        format_params(gdt, &pg, &ming, &maxg);
        format_params(tdt, &pt, &mint, &maxt);
        if (pg <= pt) { np_ = pg; nemin = ming; nemax = maxg; }
        else { np_ = pt; nemin = mint; nemax = maxt; }
    }
    if (!out || n < 0 || (n > 0 && (!golden || !test))) return ORACLE_EINVAL;
    int rc = check_params(lo, hi, nbins, nthr, thr, rthr);
    if (rc) return rc;

    oracle_sig_t s;
    memset(&s, 0, sizeof s);
    s.n = n;
    s.first_nan_index = -1;
    s.argmax_abs = s.argmax_ulp = s.argmax_rel = -1;
    s.max_abs = NAN;
    s.max_rel = NAN;
    int have_abs = 0, have_ulp = 0, have_rel = 0;
    int binw = (hi - lo) / nbins; /* binades per bin */
    csum_t c_abs = {0, 0}, c_sq = {0, 0}, c_rel = {0, 0};
    csum_t c_g2 = {0, 0}, c_t2 = {0, 0}, c_gt = {0, 0};

    for (int64_t i = 0; i < n; ++i) {
        double G = element_value_any(golden, i, gdt);
        double T = element_value_any(test, i, tdt);

        /* Step 1: classify.  A pair with a NaN on either side is excluded
         * from everything except the NaN counts and the mismatch counts. */
        /* isinf/isnan only promise a nonzero result (glibc's isinf is -1 for
         * -Inf), so normalise them to 0/1 before counting. */
        int nan_g = isnan(G) != 0, nan_t = isnan(T) != 0;
        int inf_g = isinf(G) != 0, inf_t = isinf(T) != 0;
        s.n_nan_golden += nan_g;
        s.n_nan_test += nan_t;
        s.n_inf_golden += inf_g;
        s.n_inf_test += inf_t;
        if (nan_g || nan_t) {
            s.n_nan_pairs += 1;
            if (s.first_nan_index < 0) s.first_nan_index = i;
            continue;
        }
        s.n_valid += 1;

        /* Step 2: error = absolute difference.  Equal values (including +0 vs
         * -0 and equal infinities) have error 0; otherwise |RN(T - G)|, which
         * is +Inf when exactly one side is infinite or the infinities differ. */
        double a = (G == T) ? 0.0 : fabs(T - G);

        /* Step 3: ULP distance from the bit patterns; for a mixed pair,
         * between the positions of the two values in the narrower format. */
        int64_t ku;
        if (!mixed) {
            ku = ulp_key(element_bits(test, i, tdt), width) - ulp_key(element_bits(golden, i, gdt), width);
        } else {
            ku = format_index(round_to_format(T, np_, nemin, nemax), np_, nemin, nemax) -
                 format_index(round_to_format(G, np_, nemin, nemax), np_, nemin, nemax);
        }
        int64_t ulp = ku < 0 ? -ku : ku;
        s.sum_ulp += (uint64_t)ulp;

        /* Step 4: histogram of the error over binades [2^k, 2^(k+1)). */
        if (a == 0.0) {
            s.hist_zero += 1;
        } else if (isinf(a)) {
            s.hist_over += 1;
        } else {
            int ex;
            frexp(a, &ex);  /* a = f * 2^ex, f in [0.5, 1) => floor(log2 a) = ex - 1 */
            int k = ex - 1;
            if (k < lo)
                s.hist_under += 1;
            else if (k >= hi)
                s.hist_over += 1;
            else
                s.hist[(k - lo) / binw] += 1;
        }

        /* Step 5: mismatches = pairs that are not close under torch.isclose
         * (Section III-A): equal values are close; otherwise the pair is
         * close only if the error is finite and at most the allowed error
         * atol + |rtol * G| (product and sum rounded separately, as torch
         * forms them; a NaN allowance, from an infinite rtol times a zero
         * golden value, admits nothing). */
        for (int j = 0; j < nthr; ++j) {
            double allowed = thr[j];
            if (rthr) {
                double rel = fabs(rthr[j] * G);
                allowed = thr[j] + rel;
            }
            if (a != 0.0 && (isinf(a) || !(a <= allowed))) s.n_mismatch[j] += 1;
        }

        /* Step 6: maxima, strict > in increasing index order (lowest index
         * wins ties). */
        if (!have_abs || a > s.max_abs) {
            s.max_abs = a;
            s.argmax_abs = i;
            have_abs = 1;
        }
        if (!have_ulp || ulp > s.max_ulp) {
            s.max_ulp = ulp;
            s.argmax_ulp = i;
            have_ulp = 1;
        }

        /* Steps 7-8: sums over pairs whose two values are finite. */
        if (inf_g || inf_t) continue;
        s.n_finite += 1;
        csum_add(&c_abs, a);
        csum_add(&c_sq, a * a);
        csum_add(&c_g2, G * G);
        csum_add(&c_t2, T * T);
        csum_add(&c_gt, G * T);
        if (G != 0.0) {
            double r = a / fabs(G); /* relative error, IEEE division */
            s.n_rel += 1;
            csum_add(&c_rel, r);
            if (!have_rel || r > s.max_rel) {
                s.max_rel = r;
                s.argmax_rel = i;
                have_rel = 1;
            }
        }
    }
    /* NaN pairs count as mismatches for every threshold. */
    for (int j = 0; j < nthr; ++j) s.n_mismatch[j] += s.n_nan_pairs;

    s.sum_abs = csum_value(&c_abs);
    s.sum_sq = csum_value(&c_sq);
    s.sum_rel = csum_value(&c_rel);
    s.sum_g2 = csum_value(&c_g2);
    s.sum_t2 = csum_value(&c_t2);
    s.sum_gt = csum_value(&c_gt);
    *out = s;
    return ORACLE_OK;
}

/* Derived statistics of a signature (Section IV-B.3 scores: mean and
 * variance of the error; plus norms, cosine, mean relative error and mean ULP
 * distance).  The variance is the sample variance (divisor n_finite - 1),
 * PyTorch's default estimator. */
int oracle_stats(const oracle_sig_t *s, oracle_stats_t *st) {
    if (!s || !st) return ORACLE_EINVAL;
    double nf = (double)s->n_finite;
    st->mean_abs = s->n_finite > 0 ? s->sum_abs / nf : NAN;
    st->var_abs = s->n_finite > 1 ? (s->sum_sq - s->sum_abs * s->sum_abs / nf) / (nf - 1.0) : NAN;
    st->l2_err = sqrt(s->sum_sq);
    st->l2_g = sqrt(s->sum_g2);
    st->l2_t = sqrt(s->sum_t2);
    st->cos = (s->sum_g2 > 0 && s->sum_t2 > 0) ? s->sum_gt / sqrt(s->sum_g2 * s->sum_t2) : NAN;
    st->mean_rel = s->n_rel > 0 ? s->sum_rel / (double)s->n_rel : NAN;
    st->mean_ulp = s->n_valid > 0 ? (double)s->sum_ulp / (double)s->n_valid : NAN;
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------- */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as    */
/* easy as 1, 2, 3", SC'11): ten rounds of two 32x32->64 multiplications     */
/* with the Weyl-sequence key schedule.                                      */
/* ------------------------------------------------------------------------- */

void oracle_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t p0 = (uint64_t)M0 * c0;
        uint64_t p1 = (uint64_t)M1 * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        c0 = hi1 ^ c1 ^ k0;
        c1 = lo1;
        c2 = hi0 ^ c3 ^ k1;
        c3 = lo0;
        k0 += W0;
        k1 += W1;
    }
    out[0] = c0;
    out[1] = c1;
    out[2] = c2;
    out[3] = c3;
}

/* ------------------------------------------------------------------------- */
/* Random bit flip at a bit error rate.                                      */
/* ------------------------------------------------------------------------- */

/* Decision threshold: element i flips iff its 64-bit uniform U_i < T with
 * T = floor(rate * 2^64) (exact: ldexp scales by a power of two and the
 * conversion truncates); rate >= 1 flips every element.  Returns 0 with
 * *all = 1 in that case. */
uint64_t oracle_rate_threshold(double rate, int *all) {
    *all = 0;
    if (rate >= 1.0) {
        *all = 1;
        return 0;
    }
    if (rate <= 0.0) return 0;
    return (uint64_t)ldexp(rate, 64);
}

/* Block number c of stream s under seed: Philox4x32-10 with the key
 * (lo32(seed), hi32(seed)) at the counter (lo32(c), hi32(c), s, 0). */
static void philox_seeded(uint64_t seed, uint64_t c, uint32_t s, uint32_t out[4]) {
    uint32_t ctr[4] = {(uint32_t)c, (uint32_t)(c >> 32), s, 0};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    oracle_philox4x32_10(ctr, key, out);
}

/* The 64-bit word h (0 or 1) of a block: words 2h (low half) and 2h+1. */
static uint64_t block_word64(const uint32_t B[4], int h) {
    return (uint64_t)B[2 * h] | ((uint64_t)B[2 * h + 1] << 32);
}

/* The per-element uniform U_i.  Its top byte is byte (i mod 16) of the
 * 16-byte block A of stream 0 at block number i/16, bytes numbered
 * little-endian through words 0..3; its low 56 bits are the low 56 bits of
 * the 64-bit word (i mod 2) of the block B of stream 1 at block number i/2. */
static uint64_t uniform_of(const uint32_t A[4], const uint32_t B[4], int64_t i) {
    int byte = (int)(i & 15);
    uint64_t top = (A[byte >> 2] >> (8 * (byte & 3))) & 0xFF;
    uint64_t low = block_word64(B, (int)(i & 1)) & ((1ULL << 56) - 1);
    return (top << 56) | low;
}

/* The flipped bit of element i: y = word 0 of the block of stream 2 at block
 * number i; j = floor(y * popcount(mask) / 2^32) selects the j-th lowest set
 * bit of the mask. */
static int chosen_bit(uint64_t seed, int64_t i, uint64_t mask) {
    uint32_t C[4];
    philox_seeded(seed, (uint64_t)i, 2, C);
    uint64_t p = 0;
    for (int b = 0; b < 64; ++b) p += (mask >> b) & 1;
    uint64_t j = ((uint64_t)C[0] * p) >> 32;
    for (int b = 0; b < 64; ++b) {
        if ((mask >> b) & 1) {
            if (j == 0) return b;
            --j;
        }
    }
    return -1; /* unreachable for a nonzero mask */
}

static int check_inject(int dtype, double rate, uint64_t mask) {
    int width = dtype_width(dtype);
    if (!width) return ORACLE_EDTYPE;
    if (mask == 0 || (width < 64 && (mask >> width) != 0)) return ORACLE_EBITMASK;
    if (isnan(rate) || rate < 0) return ORACLE_ERATE;
    return ORACLE_OK;
}

/* Decide element i alone: returns 1 and the bit if it flips, else 0. */
int oracle_inject_decide(int64_t i, int dtype, uint64_t seed, double rate, uint64_t mask, int *bit) {
    int rc = check_inject(dtype, rate, mask);
    if (rc) return rc;
    int all;
    uint64_t T = oracle_rate_threshold(rate, &all);
    uint32_t A[4], B[4];
    philox_seeded(seed, (uint64_t)i >> 4, 0, A);
    philox_seeded(seed, (uint64_t)i >> 1, 1, B);
    int flip = all || uniform_of(A, B, i) < T;
    if (flip && bit) *bit = chosen_bit(seed, i, mask);
    return flip;
}

/* Flip bits of x[0..n) in place; returns the number of flipped elements or a
 * negative error code. */
int64_t oracle_inject(void *x, int64_t n, int dtype, uint64_t seed, double rate, uint64_t mask) {
    int rc = check_inject(dtype, rate, mask);
    if (rc) return rc;
    if (n < 0 || (n > 0 && !x)) return ORACLE_EINVAL;
    int all;
    uint64_t T = oracle_rate_threshold(rate, &all);
    int64_t flips = 0;
    uint32_t A[4], B[4];
    for (int64_t i = 0; i < n; ++i) {
        if ((i & 15) == 0) philox_seeded(seed, (uint64_t)i >> 4, 0, A);
        if ((i & 1) == 0) philox_seeded(seed, (uint64_t)i >> 1, 1, B);
        if (!(all || uniform_of(A, B, i) < T)) continue;
        int b = chosen_bit(seed, i, mask);
        if (dtype == ORACLE_F32) {
            uint32_t v;
            memcpy(&v, (unsigned char *)x + 4 * i, 4);
            v ^= 1u << b;
            memcpy((unsigned char *)x + 4 * i, &v, 4);
        } else {
            uint16_t v;
            memcpy(&v, (unsigned char *)x + 2 * i, 2);
            v ^= (uint16_t)(1u << b);
            memcpy((unsigned char *)x + 2 * i, &v, 2);
        }
        ++flips;
    }
    return flips;
}

int oracle_sizeof_sig(void) { return (int)sizeof(oracle_sig_t); }

/* ------------------------------------------------------------------------ */
/* Mean of the top errors (Section IV-B, "Mean of Top 10% Errors").         */
/* ------------------------------------------------------------------------ */

typedef struct {
    int64_t n_valid;      /* pairs with no NaN on either side */
    int64_t k;            /* ceil(n_valid * num / den) */
    int64_t count_above;  /* errors strictly greater than kth_value */
    double kth_value;     /* the k-th largest error (NaN when k == 0) */
    double sum_topk;      /* sum of the k largest errors (0 when k == 0) */
    double mean_topk;     /* sum_topk / k (NaN when k == 0) */
} oracle_topk_t;

static int cmp_desc(const void *x, const void *y) {
    double a = *(const double *)x, b = *(const double *)y;
    return (a < b) - (a > b);
}

int oracle_topk_mixed(const void *golden, int gdt, const void *test, int tdt, int64_t n, int num,
                      int den, oracle_topk_t *out);

int oracle_topk(const void *golden, const void *test, int64_t n, int dtype, int num, int den,
                oracle_topk_t *out) {
    if (!dtype_width(dtype)) return ORACLE_EDTYPE;
    return oracle_topk_mixed(golden, dtype, test, dtype, n, num, den, out);
}

/* The same score for a pair whose golden and test types may differ (the
 * type rules of oracle_signature_mixed). */
int oracle_topk_mixed(const void *golden, int gdt, const void *test, int tdt, int64_t n, int num,
                      int den, oracle_topk_t *out) {
    if (!pair_types_ok(gdt, tdt)) return ORACLE_EDTYPE;
    if (!out || n < 0 || (n > 0 && (!golden || !test))) return ORACLE_EINVAL;
    if (num < 1 || den < num) return ORACLE_EINVAL;

    /* The error of every valid pair, defined as in oracle_signature. */
    double *a = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    if (!a) return ORACLE_ENOMEM;
    int64_t m = 0;
    for (int64_t i = 0; i < n; ++i) {
        double G = element_value_any(golden, i, gdt);
        double T = element_value_any(test, i, tdt);
        if (isnan(G) || isnan(T)) continue;
        a[m++] = (G == T) ? 0.0 : fabs(T - G);
    }
    /* Decreasing order; the k largest are a[0..k). */
    qsort(a, (size_t)m, sizeof(double), cmp_desc);

    oracle_topk_t r;
    r.n_valid = m;
    r.k = (int64_t)(((unsigned __int128)m * (unsigned)num + (unsigned)den - 1) / (unsigned)den);
    r.count_above = 0;
    r.kth_value = NAN;
    r.sum_topk = 0.0;
    r.mean_topk = NAN;
    if (r.k > 0) {
        r.kth_value = a[r.k - 1];
        while (r.count_above < r.k && a[r.count_above] > r.kth_value) r.count_above += 1;
        if (isinf(a[0])) {
            r.sum_topk = INFINITY;  /* an infinite error among the k largest */
        } else {
            csum_t acc = {0, 0};
            for (int64_t i = 0; i < r.k; ++i) csum_add(&acc, a[i]);
            r.sum_topk = csum_value(&acc);
        }
        r.mean_topk = r.sum_topk / (double)r.k;
    }
    free(a);
    *out = r;
    return ORACLE_OK;
}

int oracle_sizeof_topk(void) { return (int)sizeof(oracle_topk_t); }

/* ------------------------------------------------------------------------ */
/* Other error models (Section II-B; Section III-C; Section V-A).            */
/* ------------------------------------------------------------------------ */

#define ORACLE_MODEL_BITFLIP 0
#define ORACLE_MODEL_ZERO 1
#define ORACLE_MODEL_VALUE 2
#define ORACLE_MODEL_NAN 3
#define ORACLE_MODEL_UNIFORM 4
#define ORACLE_MAX_POSITIONS 4096

/* The quiet NaN written by the NaN model: sign 0, exponent all ones, top
 * mantissa bit set, the rest 0. */
static uint32_t canonical_nan(int dtype) {
    return dtype == ORACLE_F32 ? 0x7FC00000u : (dtype == ORACLE_F16 ? 0x7E00u : 0x7FC0u);
}

static void store_bits(void *x, int64_t i, int dtype, uint32_t v) {
    if (dtype == ORACLE_F32) {
        memcpy((unsigned char *)x + 4 * i, &v, 4);
    } else {
        uint16_t h = (uint16_t)v;
        memcpy((unsigned char *)x + 2 * i, &h, 2);
    }
}

/* The model's new bits for element i (not for the value model). */
static uint32_t model_bits(int model, int dtype, uint32_t old, uint64_t seed, int64_t i, uint64_t mask) {
    if (model == ORACLE_MODEL_ZERO) return 0;
    if (model == ORACLE_MODEL_NAN) return canonical_nan(dtype);
    return old ^ (1u << chosen_bit(seed, i, mask));
}

/* The random draws of the value models at a rate for element i: block i of
 * stream 4.  Its 64-bit word 0, W, gives the source index floor(W n / 2^64)
 * of the tensor-distribution model; its word 2 (32 bits), cut to the type's
 * width, is the uniform model's bit pattern. */
static int64_t value_source(uint64_t seed, int64_t i, int64_t n) {
    uint32_t V[4];
    philox_seeded(seed, (uint64_t)i, 4, V);
    return (int64_t)(((unsigned __int128)block_word64(V, 0) * (uint64_t)n) >> 64);
}
static uint32_t uniform_bits(uint64_t seed, int64_t i, int dtype) {
    uint32_t V[4];
    philox_seeded(seed, (uint64_t)i, 4, V);
    return dtype == ORACLE_F32 ? V[2] : (V[2] & 0xFFFFu);
}

/* Rate mode: the elements oracle_inject would flip (U_i < T, every element
 * when rate >= 1) are set to +0 (model 1), to the canonical quiet NaN
 * (model 3), bit-flipped (model 0, identical to oracle_inject), to a
 * uniformly random bit pattern of the type (model 4), or (model 2) to the
 * value the uncorrupted tensor -- the tensor as it was before the call --
 * holds at a uniformly random index, i.e. a value drawn from the tensor's
 * own distribution.  The mask is used by the bit-flip model only.  Returns
 * the number of chosen elements or a negative error code. */
int64_t oracle_inject_model(void *x, int64_t n, int dtype, uint64_t seed, double rate, int model,
                            uint64_t mask) {
    int width = dtype_width(dtype);
    if (!width) return ORACLE_EDTYPE;
    if (model < ORACLE_MODEL_BITFLIP || model > ORACLE_MODEL_UNIFORM) return ORACLE_EINVAL;
    int rc = check_inject(dtype, rate, model == ORACLE_MODEL_BITFLIP ? mask : 1);
    if (rc) return rc;
    if (n < 0 || (n > 0 && !x)) return ORACLE_EINVAL;
    /* the value model reads its sources from a copy taken before any write */
    void *orig = NULL;
    if (model == ORACLE_MODEL_VALUE && n > 0) {
        orig = malloc((size_t)n * (size_t)(width / 8));
        if (!orig) return ORACLE_EINVAL;
        memcpy(orig, x, (size_t)n * (size_t)(width / 8));
    }
    int all;
    uint64_t T = oracle_rate_threshold(rate, &all);
    int64_t count = 0;
    uint32_t A[4], B[4];
    for (int64_t i = 0; i < n; ++i) {
        if ((i & 15) == 0) philox_seeded(seed, (uint64_t)i >> 4, 0, A);
        if ((i & 1) == 0) philox_seeded(seed, (uint64_t)i >> 1, 1, B);
        if (!(all || uniform_of(A, B, i) < T)) continue;
        uint32_t v;
        if (model == ORACLE_MODEL_VALUE)
            v = element_bits(orig, value_source(seed, i, n), dtype);
        else if (model == ORACLE_MODEL_UNIFORM)
            v = uniform_bits(seed, i, dtype);
        else
            v = model_bits(model, dtype, element_bits(x, i, dtype), seed, i, mask);
        store_bits(x, i, dtype, v);
        ++count;
    }
    free(orig);
    return count;
}

/* Position mode (the paper's num_pos).  Draw j = 0, 1, 2, ... gives the
 * block W of stream 3 at block number j, its 64-bit words W0 and W1, and the
 * index p_j = floor(W0 * n / 2^64); the positions are the first num_pos
 * distinct p_j in order of appearance.  Position m (drawn at j) becomes +0
 * (model 1), the canonical NaN (model 3), a bit flip with the rate mode's bit
 * rule (model 0), the low bits (the type's width) of W1 as a uniformly
 * random bit pattern (model 4), or (model 2, random value) the uncorrupted
 * tensor's value at index floor(W1 * n / 2^64) -- a value drawn from the
 * tensor's own distribution.  0 <= num_pos <= min(n, 4096).  positions
 * (optional) gets the positions in order.  Returns num_pos or a negative
 * error code. */
int64_t oracle_corrupt_positions(void *x, int64_t n, int dtype, uint64_t seed, int model,
                                 int64_t num_pos, uint64_t mask, int64_t *positions) {
    int width = dtype_width(dtype);
    if (!width) return ORACLE_EDTYPE;
    if (model < ORACLE_MODEL_BITFLIP || model > ORACLE_MODEL_UNIFORM) return ORACLE_EINVAL;
    if (model == ORACLE_MODEL_BITFLIP && (mask == 0 || (mask >> width) != 0)) return ORACLE_EBITMASK;
    if (n < 0 || num_pos < 0 || num_pos > n || num_pos > ORACLE_MAX_POSITIONS) return ORACLE_EINVAL;
    if (num_pos > 0 && !x) return ORACLE_EINVAL;
    int64_t pos[ORACLE_MAX_POSITIONS], src[ORACLE_MAX_POSITIONS];
    uint32_t ubits[ORACLE_MAX_POSITIONS];
    int64_t m = 0;
    for (uint64_t j = 0; m < num_pos; ++j) {
        uint32_t W[4];
        philox_seeded(seed, j, 3, W);
        int64_t p = (int64_t)(((unsigned __int128)block_word64(W, 0) * (uint64_t)n) >> 64);
        int seen = 0;
        for (int64_t q = 0; q < m; ++q) seen |= pos[q] == p;
        if (seen) continue;
        pos[m] = p;
        src[m] = (int64_t)(((unsigned __int128)block_word64(W, 1) * (uint64_t)n) >> 64);
        ubits[m] = width == 32 ? W[2] : (W[2] & 0xFFFFu);
        ++m;
    }
    /* every source is read before any position is written */
    uint32_t val[ORACLE_MAX_POSITIONS];
    for (int64_t q = 0; q < num_pos; ++q)
        val[q] = model == ORACLE_MODEL_VALUE     ? element_bits(x, src[q], dtype)
                 : model == ORACLE_MODEL_UNIFORM ? ubits[q]
                                                 : model_bits(model, dtype, element_bits(x, pos[q], dtype), seed,
                                                              pos[q], mask);
    for (int64_t q = 0; q < num_pos; ++q) {
        store_bits(x, pos[q], dtype, val[q]);
        if (positions) positions[q] = pos[q];
    }
    return num_pos;
}

/* Round-to-nearest-even of a binary64 value to a binary format with p
 * significand bits (implicit bit included) and normal exponents
 * [emin, emax]: the result as a binary64.  Magnitudes at or above the
 * midpoint between the largest finite value and 2^(emax+1) become Inf. */
static double round_to_format(double v, int p, int emin, int emax) {
    if (isnan(v) || isinf(v) || v == 0.0) return v;
    double a = fabs(v);
    double overflow = ldexp(2.0 - ldexp(1.0, -p), emax);   /* (2 - 2^-p) 2^emax */
    if (a >= overflow) return v > 0 ? INFINITY : -INFINITY;
    int e;
    frexp(a, &e);                         /* a in [2^(e-1), 2^e) */
    int exp = e - 1;
    if (exp < emin) exp = emin;           /* the subnormal range keeps the quantum of 2^emin */
    double quantum = ldexp(1.0, exp - (p - 1));
    double r = rint(a / quantum) * quantum; /* a / quantum is exact: a power-of-two scaling */
    return v > 0 ? r : -r;
}

/* FP16 / BF16 error (Section III-C): every element of an f32 tensor x[0..n)
 * is replaced by its round-to-nearest-even value in the narrower type,
 * widened back (to_dtype 1: binary16, 2: bfloat16).  A NaN becomes the f32
 * quiet NaN with its sign kept (sign | 0x7FC00000).  Returns 0 or a
 * negative error code. */
int oracle_cast_round(void *x, int64_t n, int to_dtype) {
    if (to_dtype != ORACLE_F16 && to_dtype != ORACLE_BF16) return ORACLE_EDTYPE;
    if (n < 0 || (n > 0 && !x)) return ORACLE_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        uint32_t b = element_bits(x, i, ORACLE_F32);
        float f;
        memcpy(&f, &b, 4);
        uint32_t out;
        if (isnan(f)) {
            out = (b & 0x80000000u) | 0x7FC00000u;
        } else {
            double r = to_dtype == ORACLE_F16 ? round_to_format((double)f, 11, -14, 15)
                                              : round_to_format((double)f, 8, -126, 127);
            float g = (float)r;           /* exact: r has at most 11 significant bits */
            memcpy(&out, &g, 4);
        }
        store_bits(x, i, ORACLE_F32, out);
    }
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Analyzer statistics over score series (Section IV-C; Section V-C).        */
/* ------------------------------------------------------------------------ */

typedef struct {
    int64_t count;   /* entries that are not NaN */
    double mean;     /* their mean (NaN when count = 0) */
    double var;      /* sample variance, divisor count - 1 (NaN when count < 2) */
    double std;      /* sqrt(var) */
    double min, max; /* NaN when count = 0 */
} oracle_series_t;

/* Mean, sample variance and range of the non-NaN entries of x[0..n): the
 * (mu, sigma) pair of one operator's scores across epochs (Section IV-C). */
int oracle_series_stats(const double *x, int64_t n, oracle_series_t *out) {
    if (!out || n < 0 || (n > 0 && !x)) return ORACLE_EINVAL;
    oracle_series_t r = {0, NAN, NAN, NAN, NAN, NAN};
    csum_t acc = {0, 0};
    for (int64_t i = 0; i < n; ++i) {
        if (isnan(x[i])) continue;
        if (r.count == 0 || x[i] < r.min) r.min = x[i];
        if (r.count == 0 || x[i] > r.max) r.max = x[i];
        csum_add(&acc, x[i]);
        r.count += 1;
    }
    if (r.count > 0) r.mean = csum_value(&acc) / (double)r.count;
    if (r.count > 1) {
        /* second pass about the mean */
        csum_t sq = {0, 0};
        for (int64_t i = 0; i < n; ++i) {
            if (isnan(x[i])) continue;
            double d = x[i] - r.mean;
            csum_add(&sq, d * d);
        }
        r.var = csum_value(&sq) / (double)(r.count - 1);
        r.std = sqrt(r.var);
    }
    *out = r;
    return ORACLE_OK;
}

/* out[i] = scores[i] / units[i]: a score in units of the FP64 error's score
 * (Section V-C; IEEE division, so 0/0 gives NaN). */
int oracle_normalize(const double *scores, const double *units, int64_t n, double *out) {
    if (n < 0 || (n > 0 && (!scores || !units || !out))) return ORACLE_EINVAL;
    for (int64_t i = 0; i < n; ++i) out[i] = scores[i] / units[i];
    return ORACLE_OK;
}

/* Average rank (1-based) of v among the m values w: 1 + #(w < v) plus half
 * of the other values equal to v. */
static double average_rank(const double *w, int64_t m, double v) {
    int64_t less = 0, equal = 0;
    for (int64_t j = 0; j < m; ++j) {
        less += w[j] < v;
        equal += w[j] == v;
    }
    return 1.0 + (double)less + (double)(equal - 1) / 2.0;
}

/* Spearman's rank correlation of the pairs (x[i], y[i]) with neither entry
 * NaN (Section IV-C): the Pearson correlation of their average ranks.  NaN
 * when fewer than two pairs remain or either rank vector is constant. */
int oracle_spearman(const double *x, const double *y, int64_t n, double *rho) {
    if (!rho || n < 0 || (n > 0 && (!x || !y))) return ORACLE_EINVAL;
    double *xs = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    double *ys = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    if (!xs || !ys) {
        free(xs);
        free(ys);
        return ORACLE_ENOMEM;
    }
    int64_t m = 0;
    for (int64_t i = 0; i < n; ++i) {
        if (isnan(x[i]) || isnan(y[i])) continue;
        xs[m] = x[i];
        ys[m] = y[i];
        ++m;
    }
    *rho = NAN;
    if (m >= 2) {
        double *rx = (double *)malloc(sizeof(double) * (size_t)m);
        double *ry = (double *)malloc(sizeof(double) * (size_t)m);
        if (!rx || !ry) {
            free(rx);
            free(ry);
            free(xs);
            free(ys);
            return ORACLE_ENOMEM;
        }
        for (int64_t i = 0; i < m; ++i) {
            rx[i] = average_rank(xs, m, xs[i]);
            ry[i] = average_rank(ys, m, ys[i]);
        }
        /* Pearson correlation of the ranks (both rank vectors have mean (m+1)/2) */
        double mean = (double)(m + 1) / 2.0;
        csum_t sxy = {0, 0}, sxx = {0, 0}, syy = {0, 0};
        for (int64_t i = 0; i < m; ++i) {
            double dx = rx[i] - mean, dy = ry[i] - mean;
            csum_add(&sxy, dx * dy);
            csum_add(&sxx, dx * dx);
            csum_add(&syy, dy * dy);
        }
        double vx = csum_value(&sxx), vy = csum_value(&syy);
        if (vx > 0 && vy > 0) *rho = csum_value(&sxy) / sqrt(vx * vy);
        free(rx);
        free(ry);
    }
    free(xs);
    free(ys);
    return ORACLE_OK;
}
