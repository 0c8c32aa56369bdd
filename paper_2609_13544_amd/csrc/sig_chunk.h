// Pass 1 of the error signature (sig_chunk) for gfx950, templated on the
// golden and test element types; included by the translation units that
// instantiate it (same-type pairs in signature.hip, mixed-precision pairs in
// mixed.hip).  Pass 2 (sig_finalize, in signature.hip) combines a pair's
// chunk records in a fixed order and writes the peat_signature_t.
//
// 256-thread blocks, each streaming one or two consecutive fixed-size chunks
// (a chunk lies within one pair).  Each thread streams lane vectors of golden
// and test through nontemporal buffer loads: 16 bytes of the wider side (4
// f32, 8 f16/bf16 or 2 binary64 elements) and the matching bytes of the
// other, widens them exactly to binary64 and accumulates the signature of its
// elements.  Each chunk's record (ChunkPartial) holds the binary64 partial
// sums of each of the block's four waves; maxima with their lowest index,
// integer counts and the histogram are exact and go to the record of the last
// chunk of the block's run of chunks of one pair.
//
// The definitions follow the paper's FI assessment scores (Section IV-B.3:
// error = absolute difference of golden and faulty values; max, mean,
// variance), the closeness test of Section III-A (torch.isclose with absolute
// and relative tolerances), the error histograms of Section V-D and, for
// mixed pairs, the precision comparisons of Section III-C (the ULP distance
// counted in the narrower format).
//
// Fast path.  A wave whose current vectors hold only "ordinary" pairs (both
// finite, no NaN, golden nonzero, same sign, relative error below 0.5) needs
// no classification:
//   - one comparison of the relative error per element flags every other
//     case (a sign change or a zero golden gives a relative error >= 1 or
//     NaN) together with the candidates for the maximum relative error; the
//     exact IEEE quotient is formed only for those candidates;
//   - reciprocals come from one hardware estimate per four (or two) elements
//     plus a Newton step;
//   - the maxima of |err| and of the ULP distance are wave-uniform running
//     records; a vector that raises one is resolved to its element indices
//     on the spot, while its values are in registers;
//   - counts use wave ballots; the histogram uses lane-private 16-bit LDS
//     counters addressed through a binary64-exponent -> row table.
// Any other vector is deferred: its wave-uniform vector number goes to a
// per-wave LDS list and the generic per-element path (every IEEE case)
// processes the list out of the hot loop.  Ragged tails and unaligned pairs
// use the generic path directly.
//
// Determinism: the element -> lane mapping, per-lane order and the wave
// reductions of the sums depend only on the chunk size, which depends only on
// n; everything else is exact.  Single, batched and any-grid-size launches
// give bit-identical signatures.
#pragma once

#include <atomic>

#include "elements.h"
#include "inject_span.h"

namespace peat {
namespace {


constexpr double kRelMargin = 0x1p-30;   // relative slack of the max-rel filter
// Fast-path limit on the relative error: an element above it (or NaN) sends
// its vector to the generic path (one exactly at it may take either path;
// both are exact there).  A sign change between finite golden and test
// values gives |t - g| >= |g|, i.e. a relative error of at least 1 (less the
// reciprocal's 2^-48), and a zero golden value gives Inf or NaN, so this one
// comparison also catches every case the fast path does not handle.  Up to
// the limit t lies within a factor 1.25 (plus 2^-47) of g, so:
//   - t - g is exact in the elements' own format (Sterbenz: t/g in [1/2, 2]);
//     when the difference is formed in binary32 and rounded, it is at least
//     |g|/2 in magnitude, which this limit rejects, so a fast-path error is
//     always the exact difference;
//   - the fast path sums g^2, ge and e^2 only, and the sums of t^2 and gt
//     follow from t^2 = g^2 + 2ge + e^2 and gt = g^2 + ge (identities of
//     exact arithmetic) with a condition number below 2.8.  When neither
//     side is binary64, g and e have at most 24 significant bits, so the
//     three products are exact in binary64 and only the summation rounds;
//     with a binary64 test side e can have up to 53 bits and ge, e^2 are
//     rounded products (2^-53 relative each), within the same tolerance;
//   - an f32 ULP distance is below 2^24 and an f16/bf16 one below 2^11.
constexpr double kRareRel = 0.25;
constexpr int kDeferCap = 32;            // deferred vectors per wave before a flush
// Chunks per block: one while the launch has few chunks (every chunk gets a
// block of its own); more once there are enough for at least kMinRounds
// rounds of resident blocks, up to about kGroupElems elements per block at
// the launch's average chunk size (two chunks of 2^18, eight of 2^16): block
// start-up is shared by the group while blocks stay short enough for the
// hardware to balance the load at the end of the launch.
constexpr int64_t kMaxGroup = 8;
constexpr int64_t kMinRounds = 8;
constexpr int64_t kGroupElems = int64_t(1) << 19;
// a lane's 16-bit histogram counters hold a whole run of chunks
static_assert(kMaxGroup * (int64_t(1) << kMaxChunkLog2) / kBlock < 65536, "histogram counter width");
constexpr int kHistCols = kBlock / 2;     // histogram words per slot
// the injection's candidate queues fit in the histogram's LDS
static_assert(sizeof(uint32_t) * kWaves * kQCap <= sizeof(uint32_t) * kHistSlots * kHistCols, "queue size");

__device__ __forceinline__ uint32_t hist_col(int tid) { return (uint32_t)tid & (kHistCols - 1); }
__device__ __forceinline__ uint32_t hist_inc(int tid) { return tid < kHistCols ? 1u : 0x10000u; }

// super-step unroll: lane vectors per tensor per lane
template <int DG, int DT>
constexpr int kUnroll = DG != DT ? 4 : ((DT == PEAT_F32) ? 4 : 2);

// ULP distance of two bit patterns of width W (signed-magnitude keys).
template <int W>
__device__ __forceinline__ uint32_t ulp_dist(uint32_t gb, uint32_t tb) {
    constexpr uint32_t S = 1u << (W - 1);
    constexpr uint32_t M = S - 1;
    uint32_t mg = gb & M, mt = tb & M;
    if ((gb ^ tb) & S) return mg + mt;
    return mt > mg ? mt - mg : mg - mt;
}

__device__ __forceinline__ uint32_t wave_count(bool p) {
    return (uint32_t)__popcll(__ballot(p));
}

// Binary64 reciprocal for the relative-error sum: the hardware estimate
// (relative error below 2^-24) refined by one Newton step (below 2^-48).
__device__ __forceinline__ double recip(double b) {
    const double y = __builtin_amdgcn_rcp(b);
    return __builtin_fma(y, __builtin_fma(-b, y, 1.0), y);
}

// Reciprocals of four magnitudes from one reciprocal of their product (the
// hardware reciprocal issues at a quarter of the fma rate).  The inputs are
// widened f32/f16/bf16 golden values (the golden side is never binary64), so
// the product of four stays a normal binary64 number (between 2^-600 and
// 2^512) and the pairwise products are exact; each result is within a few
// units of 2^-48 of 1/x.  A zero, Inf or NaN among the four makes all four
// results NaN or Inf.
__device__ __forceinline__ void recip4(const double *x, double *r) {
    const double p01 = x[0] * x[1], p23 = x[2] * x[3];
    const double inv = recip(p01 * p23);
    const double i01 = inv * p23, i23 = inv * p01;
    r[0] = x[1] * i01;
    r[1] = x[0] * i01;
    r[2] = x[3] * i23;
    r[3] = x[2] * i23;
}
// The same for two magnitudes (lane vectors of two elements).
__device__ __forceinline__ void recip2(const double *x, double *r) {
    const double inv = recip(x[0] * x[1]);
    r[0] = x[1] * inv;
    r[1] = x[0] * inv;
}
// Eight magnitudes of widened f16 values (in [2^-24, 2^16]) from one
// reciprocal: the product of eight stays within [2^-192, 2^128]; the pair
// and quad products are exact (at most 44 significant bits) and only the
// product of all eight rounds, so each result is within about 2^-47.8 of
// 1/x.  A zero, Inf or NaN among the eight makes all eight NaN or Inf.
__device__ __forceinline__ void recip8(const double *x, double *r) {
    const double p01 = x[0] * x[1], p23 = x[2] * x[3], p45 = x[4] * x[5], p67 = x[6] * x[7];
    const double q0 = p01 * p23, q1 = p45 * p67;
    const double inv = recip(q0 * q1);
    const double iq0 = inv * q1, iq1 = inv * q0;
    const double i01 = iq0 * p23, i23 = iq0 * p01, i45 = iq1 * p67, i67 = iq1 * p45;
    r[0] = x[1] * i01;
    r[1] = x[0] * i01;
    r[2] = x[3] * i23;
    r[3] = x[2] * i23;
    r[4] = x[5] * i45;
    r[5] = x[4] * i45;
    r[6] = x[7] * i67;
    r[7] = x[6] * i67;
}

struct Lane {
    double s_abs, s_rel;           // both paths
    double s_sq, s_g2, s_ge;       // fast path: sums of e^2, g^2 and g*e
    double gx_abs;                 // both paths: max |err| and element index
    uint32_t gi_abs;
    uint32_t gu, gi_ulp;           // both paths: max ULP and element index
    double mx_rel;                 // both paths: max rel err and its index
    double rthr;                   // fast-path filter, at most kRareRel
    uint32_t ix_rel;
    uint64_t s_ulp;
    uint32_t s_ulp32;              // fast path: ULP sum of the current super-step
    uint32_t first_nan, first_valid;
    uint32_t cnt[kCnt];                    // generic-path counts (per lane)
    uint32_t mism[PEAT_MAX_THRESHOLDS];    // generic-path mismatches (per lane)
};

// Fast-path state shared by the wave.  Vectors reach the fast path in
// increasing vector number, and every element of a later vector has a higher
// index than every element of an earlier one, so only a vector that exceeds
// the wave's running maximum can hold the (value, lowest index) maximum: an
// element equal to the running maximum in a later vector cannot.
struct Uni {
    uint32_t common;                       // ordinary vectors per lane
    uint32_t mism[PEAT_MAX_THRESHOLDS];
    uint32_t first;                        // first ordinary vector number
    double wx_abs;                         // running max |err|
    uint32_t wu;                           // running max ULP
};

struct alignas(16) Shared {
    uint8_t hrow[4096];                    // binary64 sign and exponent field -> histogram slot
    // Lane-private 16-bit counters, two per word: word [slot][t mod 128]
    // holds lane t's count in its low half when t < 128 and in its high half
    // otherwise.  The two lanes of a word are in different waves, and a lane
    // counts at most 2^18 / 256 = 1024 elements per chunk, so no half carries.
    uint32_t hist[kHistSlots * kHistCols];
    uint32_t defer[kWaves][kDeferCap];     // deferred vector numbers per wave
    // generic-path sums of a^2, g^2, t^2 and g*t, one column per lane
    double gsum[4][kBlock];
    double rd[kWaves][6];
    double rmax[kWaves][2];
    uint32_t rix[kWaves][5];               // abs, rel, ulp, first_nan, first_valid
    uint32_t rmu[kWaves];
    uint64_t rulp[kWaves];
    uint32_t rcnt[kWaves][kCnt + PEAT_MAX_THRESHOLDS];
};

// Clear the lane-private histogram counters and build the exponent table:
// slot 0 error 0, slot 1 below 2^lo, slots 2.. bins, last slot >= 2^hi; four
// exponent fields per word, the same slots for either sign.
__device__ __forceinline__ void init_tables(Shared &sh, const SigParams &P, int tid) {
    uint4 *h4 = reinterpret_cast<uint4 *>(sh.hist);
    for (int i = tid; i < kHistSlots * kHistCols / 4; i += kBlock) h4[i] = make_uint4(0u, 0u, 0u, 0u);
    const int w = (P.hi - P.lo) / P.nbins;
    uint32_t *t4 = reinterpret_cast<uint32_t *>(sh.hrow);
    for (int q = tid; q < 512; q += kBlock) {
        uint32_t word = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int E = 4 * q + j;           // biased exponent of |value|
            int slot;
            if (E == 0) {
                slot = 0;
            } else if (E == 2047) {
                slot = P.nbins + 2;            // infinite error
            } else {
                const int k = E - 1023;        // a in [2^k, 2^(k+1))
                slot = k < P.lo ? 1 : (k >= P.hi ? P.nbins + 2 : 2 + (k - P.lo) / w);
            }
            word |= (uint32_t)slot << (8 * j);
        }
        t4[q] = word;
        t4[512 + q] = word;
    }
}
static_assert((kHistSlots * kHistCols) % 4 == 0 && offsetof(Shared, hist) % 16 == 0, "16-byte histogram clears");

__device__ __forceinline__ void lane_init(Lane &L, Uni &U) {
    L.s_abs = L.s_rel = L.s_sq = L.s_g2 = L.s_ge = 0.0;
    L.gx_abs = -1.0;
    L.gi_abs = kNone;
    L.gu = 0;
    L.gi_ulp = kNone;
    L.mx_rel = -1.0;
    L.rthr = -1.0;
    L.ix_rel = kNone;
    L.s_ulp = 0;
    L.s_ulp32 = 0;
    L.first_nan = L.first_valid = kNone;
#pragma unroll
    for (int c = 0; c < kCnt; ++c) L.cnt[c] = 0;
#pragma unroll
    for (int j = 0; j < PEAT_MAX_THRESHOLDS; ++j) L.mism[j] = 0;
    U.common = 0;
    U.first = kNone;
    U.wx_abs = -1.0;
    U.wu = 0;
#pragma unroll
    for (int j = 0; j < PEAT_MAX_THRESHOLDS; ++j) U.mism[j] = 0;
}

// Generic-path sums of one lane, kept in its LDS column between generic runs.
struct GenAcc {
    double sq, g2, t2, gt;
    __device__ __forceinline__ void load(const Shared &sh, int tid) {
        sq = sh.gsum[0][tid];
        g2 = sh.gsum[1][tid];
        t2 = sh.gsum[2][tid];
        gt = sh.gsum[3][tid];
    }
    __device__ __forceinline__ void store(Shared &sh, int tid) const {
        sh.gsum[0][tid] = sq;
        sh.gsum[1][tid] = g2;
        sh.gsum[2][tid] = t2;
        sh.gsum[3][tid] = gt;
    }
};

// Byte address of lane tid's counter word of a histogram slot within
// sh.hist: slot * (kHistCols * 4) + column * 4, one shift-or given the
// column's byte offset colb (the slot comes zero-extended from the table).
__device__ __forceinline__ uint32_t hist_addr(uint32_t slot, uint32_t colb) { return (slot << 9) | colb; }
static_assert(kHistCols * 4 == 512, "hist_addr shifts the slot by 9");
__device__ __forceinline__ void hist_bump(Shared &sh, uint32_t addr, int tid) {
    atomicAdd(reinterpret_cast<uint32_t *>(reinterpret_cast<char *>(sh.hist) + addr), hist_inc(tid));
}
// Row of a binary64 value in the table: its sign and exponent field.
__device__ __forceinline__ uint32_t hist_key(double x) {
    return (uint32_t)((uint64_t)__double_as_longlong(x) >> 52);
}

__device__ __forceinline__ void hist_add(Shared &sh, double a, int tid) {
    hist_bump(sh, hist_addr(sh.hrow[hist_key(a)], hist_col(tid) * 4u), tid);
}

// Every case of one pair (NaN, Inf, zero golden, sign change, subnormals).
// Elements may arrive out of index order (deferred vectors), so the maxima
// use (value, lowest index) comparisons.
template <int DG, int DT, int NT, typename BG, typename BT>
__device__ __forceinline__ void generic_elem(Lane &L, GenAcc &ga, Shared &sh, const SigParams &P,
                                             BG gb, BT tb, uint32_t li, int tid) {
    using PT = PairTr<DG, DT>;
    const double G = widen<DG>(gb), T = widen<DT>(tb);
    const bool nan_g = G != G, nan_t = T != T;
    const bool inf_g = __builtin_isinf(G), inf_t = __builtin_isinf(T);
    L.cnt[C_NAN_G] += nan_g;
    L.cnt[C_NAN_T] += nan_t;
    L.cnt[C_INF_G] += inf_g;
    L.cnt[C_INF_T] += inf_t;
    if (nan_g || nan_t) {
        L.cnt[C_NANPAIR] += 1;
        L.first_nan = min(L.first_nan, li);
        return;
    }
    L.cnt[C_VALID] += 1;
    L.first_valid = min(L.first_valid, li);
    const double a = (G == T) ? 0.0 : __builtin_fabs(T - G);
    // ULP distance in the narrower format (the wider value rounded to it)
    uint32_t ulp;
    if constexpr (PT::SAME) {
        ulp = ulp_dist<Tr<DT>::W>(gb, tb);
    } else if constexpr (PT::GOLDEN_NARROW) {
        ulp = ulp_dist<PT::WN>((uint32_t)gb, narrow_bits<DG, DT>(T));
    } else {
        ulp = ulp_dist<PT::WN>(narrow_bits<DT, DG>(G), (uint32_t)tb);
    }
    L.s_ulp += ulp;
    if (ulp > L.gu || (ulp == L.gu && li < L.gi_ulp)) {
        L.gu = ulp;
        L.gi_ulp = li;
    }
    if constexpr (DT == PEAT_F64) {
        // a binary64 test side can give a subnormal error (exponent field 0,
        // which the row table maps to the zero slot): it lies below every bin
        if (a != 0.0 && a < 0x1p-1022)
            atomicAdd(&sh.hist[1 * kHistCols + hist_col(tid)], hist_inc(tid));
        else
            hist_add(sh, a, tid);
    } else {
        hist_add(sh, a, tid);
    }
    const bool ainf = __builtin_isinf(a);
    // not close under torch.isclose: unequal, and the error is infinite or not
    // within atol + |rtol * G| (a NaN allowance admits nothing)
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const double allowed = P.any_rtol ? __dadd_rn(P.thr[j], __builtin_fabs(__dmul_rn(P.rthr[j], G))) : P.thr[j];
        L.mism[j] += (a != 0.0) && (ainf || !(a <= allowed));
    }
    if (a > L.gx_abs || (a == L.gx_abs && li < L.gi_abs)) {
        L.gx_abs = a;
        L.gi_abs = li;
    }
    if (inf_g || inf_t) return;
    L.cnt[C_FINITE] += 1;
    L.s_abs += a;
    ga.sq = __builtin_fma(a, a, ga.sq);
    ga.g2 = __builtin_fma(G, G, ga.g2);
    ga.t2 = __builtin_fma(T, T, ga.t2);
    ga.gt = __builtin_fma(G, T, ga.gt);
    if (G != 0.0) {
        L.cnt[C_REL] += 1;
        const double r = a / __builtin_fabs(G);
        L.s_rel += r;
        if (r > L.mx_rel || (r == L.mx_rel && li < L.ix_rel)) {
            L.mx_rel = r;
            L.ix_rel = li;
            L.rthr = __builtin_fmin(r - r * kRelMargin, kRareRel);
        }
    }
}

// |a - b| of two unsigned 32-bit values (v_sad_u32 with a zero addend).
__device__ __forceinline__ uint32_t absdiff_u32(uint32_t a, uint32_t b) {
    uint32_t r;
    asm("v_sad_u32 %0, %1, %2, 0" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

// max(|a|, |b|) of two binary64 values as one v_max_f64 with absolute-value
// source modifiers (the operands are never NaN here, so no quieting is needed).
__device__ __forceinline__ double absmax_f64(double a, double b) {
    double r;
    asm("v_max_f64 %0, |%1|, |%2|" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

// Wave maximum of a binary64 value, returned as a wave-uniform scalar.
__device__ __forceinline__ double wave_max_uniform(double x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x = __builtin_fmax(x, __shfl_xor(x, o));
    const uint64_t b = (uint64_t)__double_as_longlong(x);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ __forceinline__ uint32_t wave_max_uniform_u(uint32_t x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x = max(x, (uint32_t)__shfl_xor(x, o));
    return __builtin_amdgcn_readfirstlane(x);
}

// Merge candidate (ov, oi) into the (value desc, index asc) maximum (v, ix);
// kNone marks an empty entry.
template <typename V>
__device__ __forceinline__ void lex_merge(V &v, uint32_t &ix, V ov, uint32_t oi) {
    if (oi != kNone && (ix == kNone || ov > v || (ov == v && oi < ix))) {
        v = ov;
        ix = oi;
    }
}

// ULP distance of a fast-path element (both finite, same sign, not NaN):
// the difference of the narrower format's bit patterns.
template <int DG, int DT, typename BG, typename BT>
__device__ __forceinline__ uint32_t fast_ulp(BG gb, BT tb, double G, double T) {
    using PT = PairTr<DG, DT>;
    uint32_t a, b;
    if constexpr (PT::SAME) {
        a = gb;
        b = tb;
    } else if constexpr (PT::GOLDEN_NARROW) {
        a = (uint32_t)gb;
        // a binary32 wider side is rounded from its own bits
        if constexpr (DT == PEAT_F32)
            b = narrow_f32_bits<DG>((uint32_t)tb);
        else
            b = narrow_bits<DG, DT>(T);
    } else {
        if constexpr (DG == PEAT_F32)
            a = narrow_f32_bits<DT>((uint32_t)gb);
        else
            a = narrow_bits<DT, DG>(G);
        b = (uint32_t)tb;
    }
    if constexpr (PT::WN == 32) {
        return absdiff_u32(a, b);
    } else {
        return __builtin_amdgcn_sad_u16(a, b, 0u);
    }
}

// Threshold mismatches of a fast-path vector (every element finite, golden
// nonzero): nothing to count for threshold k while the vector's largest
// |err| va is at most its absolute tolerance (the allowance atol + |rtol G|
// is never below atol; padded thresholds are +Inf), so usually no element is
// compared.
template <int VEC, int NT, bool RT>
__device__ __forceinline__ void count_mismatches(Uni &U, const SigParams &P, const double *E, const double *G,
                                                 double va) {
    if (__ballot(va > P.thr_min) == 0) return;
#pragma unroll
    for (int k = 0; k < NT; ++k) {
        if (__ballot(va > P.thr[k]) == 0) continue;
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            if constexpr (RT) {
                // torch.isclose's allowance atol + |rtol * G|, rounded step by
                // step (never NaN here: G is finite and nonzero)
                const double allowed = __dadd_rn(P.thr[k], __builtin_fabs(__dmul_rn(P.rthr[k], G[j])));
                U.mism[k] += wave_count(__builtin_fabs(E[j]) > allowed);
            } else {
                U.mism[k] += wave_count(__builtin_fabs(E[j]) > P.thr[k]);
            }
        }
    }
}

typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// vec_fast for same-type 16-bit pairs: eight elements per lane vector, two
// per 32-bit word, worked on in pairs where the hardware has packed forms:
//   - ULP distances |t - g| of the bit patterns (same sign on the fast
//     path) by packed max - min, their sum by one 2 x 16-bit dot product per
//     word and the vector's largest by packed maxima;
//   - f16 difference by one packed subtraction per word.  On the fast path
//     it is exact (Sterbenz; f16 subnormals are kept), so it equals the
//     binary32 difference; where it is not exact (t/g outside [1/2, 2], a
//     sign change, overflow) the relative error is at least 1/4 (or NaN)
//     and the vector leaves the fast path before any of it is used;
//   - binary64 reciprocals of all eight golden magnitudes from one hardware
//     reciprocal (recip8 for f16, two recip4 for bf16).
// Same decisions, records and maxima as vec_fast.
//
// Equal vectors.  When every element of the wave's lane vectors equals its
// golden bit for bit (all ULP distances 0), every error is +0: the sums of
// |e|, e^2, g e and the relative errors gain exact zeros (never a -0: those
// sums start at +0 and a nonzero sum that cancels rounds to +0), the ULP sum
// gains 0, and once the wave's running maxima and every lane's filter hold a
// value an error of 0 can raise none of them.  Both are set by the first
// vector after lane_init that is not rare: its relative errors all exceed the
// initial filter of -1, so every lane's filter becomes the wave's maximum
// (>= 0) less the margin, and max |err| becomes >= 0; later updates (here or
// in generic_elem) only store values >= 0.  That vector is also the first
// ordinary one counted since lane_init, so the test is a nonzero count (a
// scalar compare).
// With no negative absolute tolerance a zero error is close under every
// threshold (the allowance atol + |rtol g| is at least atol >= 0).  What is
// left is the sum of g^2, in the same order as below, and eight counts in the
// zero bin, so the records are bit-identical to the full path's.  A golden
// that is zero, infinite or NaN (excluded from the relative or finite
// fields) sends the vector down the full path: each half-vector's product of
// four binary32 goldens is normal only if none of them is (four f16
// magnitudes stay within [2^-96, 2^64]; a bf16 product that leaves the
// normal range just takes the full path).
// Replays of a deterministic kernel's output are bit-identical to the golden
// except where a fault struck, so this is their common case.
template <int DT, int NT, bool RT>
__device__ __forceinline__ bool vec_fast16(Lane &L, Uni &U, Shared &sh, const SigParams &P,
                                           const u32x4 &gv, const u32x4 &tv, uint32_t v, uint32_t ib, int tid) {
    constexpr int VEC = 8;
    const uint32_t gw[4] = {gv.x, gv.y, gv.z, gv.w};
    const uint32_t tw[4] = {tv.x, tv.y, tv.z, tv.w};
    float G32[VEC], E32[VEC];
    double G[VEC], E[VEC], R[VEC], AG[VEC], IG[VEC];
    uint32_t d[4], row[VEC];
    uint64_t mflag = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const u16x2 a = __builtin_bit_cast(u16x2, gw[q]), b = __builtin_bit_cast(u16x2, tw[q]);
        d[q] = __builtin_bit_cast(uint32_t, (u16x2)(__builtin_elementwise_max(a, b) - __builtin_elementwise_min(a, b)));
        if constexpr (DT == PEAT_F16) {
            const f16x2 gh = __builtin_bit_cast(f16x2, gw[q]);
            G32[2 * q] = (float)gh.x;
            G32[2 * q + 1] = (float)gh.y;
        } else {
            G32[2 * q] = __uint_as_float(gw[q] << 16);
            G32[2 * q + 1] = __uint_as_float(gw[q] & 0xFFFF0000u);
        }
    }
    const u16x2 dm = __builtin_elementwise_max(
        __builtin_elementwise_max(__builtin_bit_cast(u16x2, d[0]), __builtin_bit_cast(u16x2, d[1])),
        __builtin_elementwise_max(__builtin_bit_cast(u16x2, d[2]), __builtin_bit_cast(u16x2, d[3])));
    const uint32_t vu = max((uint32_t)dm.x, (uint32_t)dm.y);
    // (laid out as the taken branch: the full path falls through)
    if (__builtin_expect(U.common != 0 && P.thr_min >= 0.0 && __ballot(vu != 0u) == 0, 0)) {
        const float q0 = (G32[0] * G32[1]) * (G32[2] * G32[3]);
        const float q1 = (G32[4] * G32[5]) * (G32[6] * G32[7]);
        // class test: NaN, infinite, zero or subnormal (every class but normal)
        constexpr int kNotNormal = 0x3FF & ~((1 << 3) | (1 << 8));
        if ((__ballot(__builtin_amdgcn_classf(q0, kNotNormal)) | __ballot(__builtin_amdgcn_classf(q1, kNotNormal))) == 0) {
#pragma unroll
            for (int j = 0; j < VEC; ++j) {
                G[j] = (double)G32[j];
                L.s_g2 = __builtin_fma(G[j], G[j], L.s_g2);
            }
            atomicAdd(reinterpret_cast<uint32_t *>(reinterpret_cast<char *>(sh.hist) +
                                                   hist_addr(sh.hrow[hist_key(0.0)], hist_col(tid) * 4u)),
                      hist_inc(tid) * (uint32_t)VEC);
            U.common += 1;
            if (U.first == kNone) U.first = v;
            return false;
        }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        if constexpr (DT == PEAT_F16) {
            const f16x2 gh = __builtin_bit_cast(f16x2, gw[q]);
            const f16x2 eh = __builtin_bit_cast(f16x2, tw[q]) - gh;
            E32[2 * q] = (float)eh.x;
            E32[2 * q + 1] = (float)eh.y;
        } else {
            E32[2 * q] = __uint_as_float(tw[q] << 16) - G32[2 * q];
            E32[2 * q + 1] = __uint_as_float(tw[q] & 0xFFFF0000u) - G32[2 * q + 1];
        }
    }
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        G[j] = (double)G32[j];
        E[j] = (double)E32[j];
        AG[j] = __builtin_fabs(G[j]);
    }
    if constexpr (DT == PEAT_F16) {
        recip8(AG, IG);
    } else {
        recip4(AG, IG);
        recip4(AG + 4, IG + 4);
    }
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        R[j] = __builtin_fabs(E[j]) * IG[j];
        mflag |= __ballot(!(R[j] <= L.rthr));
        row[j] = hist_key(E[j]);                      // the table is read after the branch
    }
    double va = absmax_f64(E[0], E[1]);
#pragma unroll
    for (int j = 2; j < VEC; ++j) va = absmax_f64(va, E[j]);
    mflag |= __ballot(va > U.wx_abs);
    mflag |= __ballot(vu > U.wu);
    if (mflag != 0) {
        uint64_t mrare = 0, mcand = 0;
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            mrare |= __ballot(!(R[j] < kRareRel));
            mcand |= __ballot(R[j] > L.rthr);
        }
        if (mrare != 0) return true;
        const uint32_t li0 = ib + (v * kBlock + tid) * VEC;
        if (mcand != 0) {
#pragma unroll
            for (int j = 0; j < VEC; ++j) {
                if (R[j] > L.rthr) {
                    const double r = __builtin_fabs(E[j]) / __builtin_fabs(G[j]);   // IEEE quotient
                    if (r > L.mx_rel) {
                        L.mx_rel = r;
                        L.ix_rel = li0 + j;
                    }
                }
            }
            const double wm = wave_max_uniform(L.mx_rel);
            L.rthr = __builtin_fmin(wm - wm * kRelMargin, kRareRel);
        }
        if (__ballot(va > U.wx_abs) != 0) {
            U.wx_abs = wave_max_uniform(va);
            if (va == U.wx_abs) {
                uint32_t ix = kNone;
#pragma unroll
                for (int j = VEC - 1; j >= 0; --j)
                    if (__builtin_fabs(E[j]) == U.wx_abs) ix = li0 + j;
                lex_merge(L.gx_abs, L.gi_abs, U.wx_abs, ix);
            }
        }
        if (__ballot(vu > U.wu) != 0) {
            U.wu = wave_max_uniform_u(vu);
            if (vu == U.wu) {
                uint32_t ix = kNone;
#pragma unroll
                for (int j = VEC - 1; j >= 0; --j)
                    if (((d[j >> 1] >> (16 * (j & 1))) & 0xFFFFu) == U.wu) ix = li0 + j;
                lex_merge(L.gu, L.gi_ulp, U.wu, ix);
            }
        }
    }

    {
        // the slots' LDS reads first (one round trip), then the counters
        const uint32_t colb = hist_col(tid) * 4u;
        uint32_t slot[VEC];
#pragma unroll
        for (int j = 0; j < VEC; ++j) slot[j] = sh.hrow[row[j]];
#pragma unroll
        for (int j = 0; j < VEC; ++j) hist_bump(sh, hist_addr(slot[j], colb), tid);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) L.s_ulp32 = __builtin_amdgcn_udot2(__builtin_bit_cast(u16x2, d[q]), (u16x2){1, 1},
                                                                 L.s_ulp32, false);
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        L.s_abs += __builtin_fabs(E[j]);
        L.s_sq = __builtin_fma(E[j], E[j], L.s_sq);
        L.s_g2 = __builtin_fma(G[j], G[j], L.s_g2);
        L.s_ge = __builtin_fma(G[j], E[j], L.s_ge);
        L.s_rel += R[j];
    }
    count_mismatches<VEC, NT, RT>(U, P, E, G, va);
    U.common += 1;
    if (U.first == kNone) U.first = v;
    return false;
}

// One lane vector of golden and of test (vector number v of the lane's
// sequence).  Called in wave-uniform control flow with every lane active.
// Returns true (wave-uniform) when the vector must go to the generic path.
//
// Every per-element decision is one wave mask: rare elements, candidates for
// the max relative error, and a new running maximum of |err| or of the ULP
// distance all land in one rarely taken branch, so the common path only
// accumulates.  The histogram's row reads are all issued before its atomic
// adds, so they share one LDS round trip.
template <int DG, int DT, int NT, bool RT>
__device__ __forceinline__ bool vec_fast(Lane &L, Uni &U, Shared &sh, const SigParams &P,
                                         const u32x4 &gv, const u32x4 &tv, uint32_t v, uint32_t ib, int tid) {
    if constexpr (DG == DT && Tr<DT>::W == 16) return vec_fast16<DT, NT, RT>(L, U, sh, P, gv, tv, v, ib, tid);
    constexpr int VEC = PairTr<DG, DT>::VEC;
    // both sides fit binary32: the difference is formed there (exact on the
    // fast path) and widened; otherwise in binary64
    constexpr bool kDiff32 = Tr<DG>::W <= 32 && Tr<DT>::W <= 32;
    float G32[VEC];
    double G[VEC], E[VEC], R[VEC];
    uint32_t row[VEC], u[VEC];
    uint64_t mflag = 0;
    double AG[VEC], IG[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        if constexpr (kDiff32) {
            G32[j] = widen32<DG>(lane_elem<DG>(gv, j));
            G[j] = (double)G32[j];
        } else {
            G[j] = widen<DG>(lane_elem<DG>(gv, j));
        }
        AG[j] = __builtin_fabs(G[j]);
    }
    if constexpr (VEC == 2) {
        recip2(AG, IG);
    } else {
#pragma unroll
        for (int q = 0; q < VEC; q += 4) recip4(AG + q, IG + q);
    }
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        const auto gb = lane_elem<DG>(gv, j);
        const auto tb = lane_elem<DT>(tv, j);
        double Tj;                                            // test value (used by mixed ULPs)
        if constexpr (kDiff32) {
            const float T32 = widen32<DT>(tb);
            E[j] = (double)(T32 - G32[j]);                    // signed error
            Tj = (double)T32;
        } else {
            Tj = widen<DT>(tb);
            E[j] = Tj - G[j];
        }
        R[j] = __builtin_fabs(E[j]) * IG[j];
        // rare (NaN, or at least kRareRel while the filter is there), or a
        // candidate for the max relative error
        mflag |= __ballot(!(R[j] <= L.rthr));
        // same sign on the fast path: the ULP distance is |t - g| of the bit patterns
        u[j] = fast_ulp<DG, DT>(gb, tb, G[j], Tj);
        row[j] = hist_key(E[j]);                      // the table is read after the branch
    }
    double va = absmax_f64(E[0], E[1]);
#pragma unroll
    for (int j = 2; j < VEC; ++j) va = absmax_f64(va, E[j]);
    uint32_t vu = max(u[0], u[1]);
#pragma unroll
    for (int j = 2; j < VEC; ++j) vu = max(vu, u[j]);
    mflag |= __ballot(va > U.wx_abs);
    mflag |= __ballot(vu > U.wu);
    if (mflag != 0) {
        uint64_t mrare = 0, mcand = 0;
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            mrare |= __ballot(!(R[j] < kRareRel));
            mcand |= __ballot(R[j] > L.rthr);
        }
        if (mrare != 0) return true;
        const uint32_t li0 = ib + (v * kBlock + tid) * VEC;
        if (mcand != 0) {
            // The filter threshold is shared by the wave: an element whose
            // relative error is below the wave's running maximum cannot be
            // the chunk's maximum, so only a few vectors per chunk get here.
            // Ties with the maximum still pass (the margin keeps them), and
            // the lanes' (value, lowest index) maxima are merged at the end
            // of the chunk.
#pragma unroll
            for (int j = 0; j < VEC; ++j) {
                if (R[j] > L.rthr) {
                    const double r = __builtin_fabs(E[j]) / __builtin_fabs(G[j]);   // IEEE quotient
                    if (r > L.mx_rel) {
                        L.mx_rel = r;
                        L.ix_rel = li0 + j;
                    }
                }
            }
            const double wm = wave_max_uniform(L.mx_rel);
            L.rthr = __builtin_fmin(wm - wm * kRelMargin, kRareRel);
        }
        // A new running maximum: the lanes that hold it record its lowest
        // index in this vector (an equal value in a later vector has a
        // higher index).  Lane records are (value, lowest index) maxima
        // shared with the generic path.
        if (__ballot(va > U.wx_abs) != 0) {
            U.wx_abs = wave_max_uniform(va);
            if (va == U.wx_abs) {
                uint32_t ix = kNone;
#pragma unroll
                for (int j = VEC - 1; j >= 0; --j)
                    if (__builtin_fabs(E[j]) == U.wx_abs) ix = li0 + j;
                lex_merge(L.gx_abs, L.gi_abs, U.wx_abs, ix);
            }
        }
        if (__ballot(vu > U.wu) != 0) {
            U.wu = wave_max_uniform_u(vu);
            if (vu == U.wu) {
                uint32_t ix = kNone;
#pragma unroll
                for (int j = VEC - 1; j >= 0; --j)
                    if (u[j] == U.wu) ix = li0 + j;
                lex_merge(L.gu, L.gi_ulp, U.wu, ix);
            }
        }
    }

    {
        // the slots' LDS reads first (one round trip), then the counters
        const uint32_t colb = hist_col(tid) * 4u;
        uint32_t slot[VEC];
#pragma unroll
        for (int j = 0; j < VEC; ++j) slot[j] = sh.hrow[row[j]];
#pragma unroll
        for (int j = 0; j < VEC; ++j) hist_bump(sh, hist_addr(slot[j], colb), tid);
    }
#pragma unroll
    for (int j = 0; j < VEC; ++j) L.s_ulp32 += u[j];
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        L.s_abs += __builtin_fabs(E[j]);
        L.s_sq = __builtin_fma(E[j], E[j], L.s_sq);
        L.s_g2 = __builtin_fma(G[j], G[j], L.s_g2);
        L.s_ge = __builtin_fma(G[j], E[j], L.s_ge);
        L.s_rel += R[j];
    }
    count_mismatches<VEC, NT, RT>(U, P, E, G, va);
    U.common += 1;
    if (U.first == kNone) U.first = v;
    return false;
}

// ---- wave reductions by DPP (chunk records, finalize) ------------------------
// The classic six-step pattern: pairs and quads (quad_perm), half rows and
// rows (mirrors), then rows 1 and 3 take the last lane of rows 0 and 2
// (row_bcast:15) and rows 2 and 3 the last lane of row 1 (row_bcast:31), so
// lane 63 ends with the whole wave's result.  Each lane's data moves through
// the VALU's data-parallel primitives rather than the LDS crossbar, and the
// order of the operations is fixed.
constexpr int kDppXor1 = 0xB1;           // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;           // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppMirror = 0x140;
constexpr int kDppBcast15 = 0x142;
constexpr int kDppBcast31 = 0x143;

// x moved by DPP control C within the rows of mask RM; lanes of the other
// rows get old.
template <int C, int RM>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t old, uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)x, C, RM, 0xF, false);
}
template <int C, int RM>
__device__ __forceinline__ double dpp_f64(double old, double x) {
    const uint64_t o = (uint64_t)__double_as_longlong(old), v = (uint64_t)__double_as_longlong(x);
    const uint32_t lo = dpp_u32<C, RM>((uint32_t)o, (uint32_t)v);
    const uint32_t hi = dpp_u32<C, RM>((uint32_t)(o >> 32), (uint32_t)(v >> 32));
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ __forceinline__ uint32_t lane63_u32(uint32_t v) { return (uint32_t)__builtin_amdgcn_readlane((int)v, 63); }
__device__ __forceinline__ double lane63_f64(double v) {
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    return __longlong_as_double((long long)(((uint64_t)lane63_u32((uint32_t)(b >> 32)) << 32) | lane63_u32((uint32_t)b)));
}

// One step of each reduction: combine with the value DPP control C brings.
template <int C, int RM>
__device__ __forceinline__ void dsum_step(double &v) { v += dpp_f64<C, RM>(0.0, v); }
template <int C, int RM>
__device__ __forceinline__ void dsum_step(uint32_t &v) { v += dpp_u32<C, RM>(0u, v); }
template <int C, int RM>
__device__ __forceinline__ void dmin_step(uint32_t &v) { v = min(v, dpp_u32<C, RM>(v, v)); }
template <int C, int RM, typename V>
__device__ __forceinline__ void dmax_step(V &v, uint32_t &ix) {
    V ov;
    if constexpr (sizeof(V) == 8)
        ov = dpp_f64<C, RM>(v, v);
    else
        ov = dpp_u32<C, RM>(v, v);
    const uint32_t oi = dpp_u32<C, RM>(ix, ix);
    // bitwise, not short-circuit: no branch per comparison
    const bool take = (oi != kNone) & ((ix == kNone) | (ov > v) | ((ov == v) & (oi < ix)));
    v = take ? ov : v;
    ix = take ? oi : ix;
}

// Wave sum of a binary64 value (fixed order), as a scalar.
__device__ __forceinline__ double dpp_sum(double v) {
    dsum_step<kDppXor1, 0xF>(v);
    dsum_step<kDppXor2, 0xF>(v);
    dsum_step<kDppHalfMirror, 0xF>(v);
    dsum_step<kDppMirror, 0xF>(v);
    dsum_step<kDppBcast15, 0xA>(v);
    dsum_step<kDppBcast31, 0xC>(v);
    return lane63_f64(v);
}
// Wave sum of a 32-bit count (at most 2^31 in total), as a scalar; zero
// without any data movement when every lane holds zero.
__device__ __forceinline__ uint32_t dpp_sum_u32(uint32_t v) {
    if (__ballot(v != 0) == 0) return 0;
    dsum_step<kDppXor1, 0xF>(v);
    dsum_step<kDppXor2, 0xF>(v);
    dsum_step<kDppHalfMirror, 0xF>(v);
    dsum_step<kDppMirror, 0xF>(v);
    dsum_step<kDppBcast15, 0xA>(v);
    dsum_step<kDppBcast31, 0xC>(v);
    return lane63_u32(v);
}
// Wave minimum of an index (kNone when every lane holds kNone), as a scalar.
__device__ __forceinline__ uint32_t dpp_min_u32(uint32_t v) {
    if (__ballot(v != kNone) == 0) return kNone;
    dmin_step<kDppXor1, 0xF>(v);
    dmin_step<kDppXor2, 0xF>(v);
    dmin_step<kDppHalfMirror, 0xF>(v);
    dmin_step<kDppMirror, 0xF>(v);
    dmin_step<kDppBcast15, 0xA>(v);
    dmin_step<kDppBcast31, 0xC>(v);
    return lane63_u32(v);
}
// Wave (value desc, index asc) maxima over entries with index != kNone of
// |err|, the relative error and the ULP distance, as scalars; the three go
// step by step so that their data moves overlap.
template <int C, int RM>
__device__ __forceinline__ void dmax3_step(double &a, uint32_t &ia, double &r, uint32_t &ir, uint32_t &u, uint32_t &iu) {
    dmax_step<C, RM>(a, ia);
    dmax_step<C, RM>(r, ir);
    dmax_step<C, RM>(u, iu);
}
__device__ __forceinline__ void dpp_max3(double &a, uint32_t &ia, double &r, uint32_t &ir, uint32_t &u, uint32_t &iu) {
    dmax3_step<kDppXor1, 0xF>(a, ia, r, ir, u, iu);
    dmax3_step<kDppXor2, 0xF>(a, ia, r, ir, u, iu);
    dmax3_step<kDppHalfMirror, 0xF>(a, ia, r, ir, u, iu);
    dmax3_step<kDppMirror, 0xF>(a, ia, r, ir, u, iu);
    dmax3_step<kDppBcast15, 0xA>(a, ia, r, ir, u, iu);
    dmax3_step<kDppBcast31, 0xC>(a, ia, r, ir, u, iu);
    a = lane63_f64(a);
    r = lane63_f64(r);
    u = lane63_u32(u);
    ia = lane63_u32(ia);
    ir = lane63_u32(ir);
    iu = lane63_u32(iu);
}


// A 64-bit value that is the same in every lane, as a scalar.
__device__ __forceinline__ uint64_t uniform_u64(uint64_t v) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// Position of one chunk: its record, its elements and its super-steps.
// Every field is uniform over the block.
struct ChunkCtx {
    int64_t gchunk;                          // global chunk number (its record)
    int64_t off;                             // first element of the chunk in its pair
    const char *gbase, *tbase;               // first element of golden and test
    int32_t pair;
    int32_t log2;                            // chunk size of the pair
    uint32_t len;                            // elements
    uint32_t nsuper;                         // full super-steps (0 when unaligned)
};

// The block's chunks: chunk_group consecutive chunks of the launch, streamed
// back to back; blocks are scheduled by the hardware as compute units free
// up, which keeps the load balanced.  The first super-step of the next chunk
// is loaded while the last one of the current chunk is processed and while
// the chunk's sums are reduced, and the exponent -> row table is built once
// per block.
//
// Only the binary64 sums depend on how elements are grouped, so only they
// are reduced per chunk, per wave, with no block barrier: each wave writes its
// six totals into the chunk record (one store).  Everything else (counts,
// maxima with their lowest index, first indices, the ULP sum, the histogram)
// is exact and independent of grouping, so it is carried over the block's run
// of consecutive chunks of one pair (indices relative to the run) and reduced
// once, into the record of the run's last chunk, whose run-end flag is 1; the
// other records of the run carry a flag of 0 and no exact fields, and the
// finalize skips those fields.  A run has at most kMaxGroup (8) chunks of at
// most 2^18 elements, so a lane counts at most 8192 elements per histogram
// slot.
template <int DG, int DT, int NT, bool RT, bool INJ, bool GK = false>
__device__ __forceinline__ void chunk_loop(const SigParams &P, Shared &sh, const SigDesc *__restrict__ descs,
                                           const int32_t *__restrict__ chunk_pair,
                                           ChunkPartial *__restrict__ partials, const InjDesc *__restrict__ inj) {
    using PT = PairTr<DG, DT>;
    constexpr int VEC = PT::VEC;
    constexpr int U = kUnroll<DG, DT>;
    constexpr int SUPER = kBlock * VEC * U;     // elements per block super-step (2048 or 4096)
    constexpr int ESZG = Tr<DG>::W / 8, ESZT = Tr<DT>::W / 8;
    constexpr int BG = PT::BG, BT = PT::BT;     // bytes per lane vector
    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int64_t nch = P.chunk_count;
    const uint32_t lane_off_g = (uint32_t)tid * BG, lane_off_t = (uint32_t)tid * BT;

    // A pair's descriptor (scalar loads: the tables are restrict arguments,
    // never written by the kernel; the values are uniform), and a chunk's
    // position from it.  Consecutive chunks of one pair reuse the descriptor.
    struct PairS {
        const char *g, *t;
        int64_t n, first;
        int32_t pair, log2, nchunks, aligned;
    };
    auto pair_of = [&](int64_t c) {
        PairS d;
        // one uniform branch: the descriptor comes from the kernel arguments
        // or from the table, each path's fields in one batch of scalar loads
        SigDesc dm;
        if (P.single) {
            d.pair = 0;
            dm = P.one;
        } else {
            d.pair = (int32_t)__builtin_amdgcn_readfirstlane((uint32_t)chunk_pair[P.chunk_base + c]);
            dm = descs[d.pair];
        }
        d.g = reinterpret_cast<const char *>(uniform_u64(reinterpret_cast<uint64_t>(dm.g)));
        d.t = reinterpret_cast<const char *>(uniform_u64(reinterpret_cast<uint64_t>(dm.t)));
        d.n = (int64_t)uniform_u64((uint64_t)dm.n);
        d.first = (int64_t)uniform_u64((uint64_t)dm.first_chunk);
        d.log2 = (int32_t)__builtin_amdgcn_readfirstlane((uint32_t)dm.chunk_log2);
        d.nchunks = (int32_t)__builtin_amdgcn_readfirstlane((uint32_t)dm.nchunks);
        d.aligned = (int32_t)__builtin_amdgcn_readfirstlane((uint32_t)dm.aligned);
        return d;
    };
    auto ctx = [&](const PairS &d, int64_t c) {
        ChunkCtx x;
        x.gchunk = P.chunk_base + c;
        x.pair = d.pair;
        x.log2 = d.log2;
        x.off = (x.gchunk - d.first) << d.log2;
        const int64_t rest = d.n - x.off;
        x.len = (uint32_t)(rest < (int64_t(1) << d.log2) ? rest : (int64_t(1) << d.log2));
        x.gbase = d.g + x.off * ESZG;
        x.tbase = d.t + x.off * ESZT;
        x.nsuper = d.aligned != 0 ? x.len / SUPER : 0;
        return x;
    };

    Lane L;
    Uni Un;
    uint32_t ndef;                               // wave-uniform
    auto reset_sums = [&]() {
        L.s_abs = L.s_rel = L.s_sq = L.s_g2 = L.s_ge = 0.0;
        const GenAcc zero{0.0, 0.0, 0.0, 0.0};
        zero.store(sh, tid);                     // this lane's generic-path column
    };

    // Buffer loads: the chunk base lives in a scalar resource, the per-lane
    // offsets are loop-invariant registers and the super-step moves only the
    // scalar offset, so no address register is rewritten while loads that
    // read it are in flight.  The resources cover the chunk (at most 2^18
    // elements = 2 MiB of binary64); only its full super-steps are loaded
    // here (the hardware does not range-check the scalar offset), the ragged
    // rest element by element at the chunk's end.
    auto load_at = [&](u32x4 (&g)[U], u32x4 (&t)[U], const char *gb, const char *tb, uint32_t len, uint32_t s) {
        const __amdgpu_buffer_rsrc_t grs =
            __builtin_amdgcn_make_buffer_rsrc((void *)gb, (short)0, (int)(len * ESZG), kBufFlags);
        const __amdgpu_buffer_rsrc_t trs =
            __builtin_amdgcn_make_buffer_rsrc((void *)tb, (short)0, (int)(len * ESZT), kBufFlags);
        // a golden read by many pairs of the launch keeps its lines cached
        // (default policy); otherwise every byte is read once (nontemporal)
        if constexpr (GK) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                g[u] = buf_load<BG, 0>(grs, (int)lane_off_g, (int)((s * U + u) * (kBlock * BG)));
                t[u] = buf_load<BT, kLoadNT>(trs, (int)lane_off_t, (int)((s * U + u) * (kBlock * BT)));
            }
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                g[u] = buf_load<BG, kLoadNT>(grs, (int)lane_off_g, (int)((s * U + u) * (kBlock * BG)));
                t[u] = buf_load<BT, kLoadNT>(trs, (int)lane_off_t, (int)((s * U + u) * (kBlock * BT)));
            }
        }
    };
    auto load = [&](u32x4 (&g)[U], u32x4 (&t)[U], const ChunkCtx &c, uint32_t s) {
        load_at(g, t, c.gbase, c.tbase, c.len, s);
    };
    // ib: index of the chunk's first element relative to the run
    auto step = [&](const u32x4 (&g)[U], const u32x4 (&t)[U], uint32_t s, uint32_t ib) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t v = s * U + u;
            if (vec_fast<DG, DT, NT, RT>(L, Un, sh, P, g[u], t[u], v, ib, tid)) {
                sh.defer[wave][ndef] = v;      // every lane writes the same value
                ++ndef;
            }
        }
        // at most U * VEC distances below 2^24 each: no 32-bit overflow
        L.s_ulp += L.s_ulp32;
        L.s_ulp32 = 0;
    };
    // The deferred vectors of the current chunk through the generic path.
    auto flush = [&](const ChunkCtx &c, uint32_t ib) {
        if (ndef != 0) {
            GenAcc gf;
            gf.load(sh, tid);
#pragma unroll 1
            for (uint32_t k = 0; k < ndef; ++k) {
                const uint32_t v = sh.defer[wave][k];
                const u32x4 gv = load_vec<BG>(c.gbase, v * kBlock + tid);
                const u32x4 tv = load_vec<BT>(c.tbase, v * kBlock + tid);
                const uint32_t li0 = ib + (v * kBlock + tid) * VEC;
#pragma unroll 1
                for (int j = 0; j < VEC; ++j)
                    generic_elem<DG, DT, NT>(L, gf, sh, P, lane_elem<DG>(gv, j), lane_elem<DT>(tv, j), li0 + j,
                                             tid);
            }
            gf.store(sh, tid);
            ndef = 0;
            // nothing of the flush stays in flight: the hot loop then waits
            // only for its own loads
            __builtin_amdgcn_s_waitcnt(0);
        }
    };

    // End of a chunk: the ragged tail (or the whole chunk when a pointer is
    // not 16-byte aligned) and the wave's binary64 sums.  Fast-path t^2 and
    // g*t come from their exact per-element identities, then the generic
    // path's direct sums are added; a fixed order per lane.
    auto chunk_end = [&](const ChunkCtx &c, uint32_t ib, bool run_end) {
        GenAcc ga;
        ga.load(sh, tid);
#pragma unroll 1
        for (uint32_t li = c.nsuper * SUPER + tid; li < c.len; li += kBlock)
            generic_elem<DG, DT, NT>(L, ga, sh, P, load_elem<DG>(c.gbase, li), load_elem<DT>(c.tbase, li), ib + li,
                                     tid);
        // the first ordinary element of this lane in the chunk
        if (Un.first != kNone) {
            L.first_valid = min(L.first_valid, ib + (Un.first * kBlock + tid) * VEC);
            Un.first = kNone;
        }
        ChunkPartial *out = partials + c.gchunk;
        {
            const double f_t2 = (L.s_g2 + 2.0 * L.s_ge) + L.s_sq;
            const double f_gt = L.s_g2 + L.s_ge;
            const double lane_sums[6] = {L.s_abs, L.s_sq + ga.sq, L.s_rel, L.s_g2 + ga.g2, f_t2 + ga.t2, f_gt + ga.gt};
            // One store per wave: lanes 0-5 write its six totals (wave 0: lane 0
            // the run-end flag, lanes 1-6 the totals).  A chunk that does not
            // end the run writes nothing else: its record's exact fields are
            // left as they are and the finalize skips them.
            const int w0 = wave == 0 ? 1 : 0;
            uint64_t word = run_end ? 1u : 0u;
#pragma unroll
            for (int k = 0; k < 6; ++k) {
                const double v = dpp_sum(lane_sums[k]);
                if (lane == k + w0) word = (uint64_t)__double_as_longlong(v);
            }
            uint64_t *row = reinterpret_cast<uint64_t *>(out) + (w0 ? 0 : 1 + 6 * wave);
            if (lane < 6 + w0) row[lane] = word;
        }
        reset_sums();
    };

    // End of a run: counts, maxima, first indices, ULP sum and histogram of
    // the block go into the record of the run's last chunk (indices made
    // relative to the pair by run_off); then the run state starts afresh.
    auto run_end_reduce = [&](const ChunkCtx &c, int64_t run_off) {
        {
            double mxa = L.gx_abs, mxr = L.mx_rel;
            uint32_t ixa = L.gi_abs, ixr = L.ix_rel, mu = L.gu, ixu = L.gi_ulp;
            dpp_max3(mxa, ixa, mxr, ixr, mu, ixu);
            const uint32_t fnan = dpp_min_u32(L.first_nan), fval = dpp_min_u32(L.first_valid);
            // at most 2^45 per lane (8192 distances below 2^32): exact in binary64
            const uint64_t sulp = (uint64_t)dpp_sum((double)L.s_ulp);
            if (lane == 0) {
                sh.rmax[wave][0] = mxa;
                sh.rmax[wave][1] = mxr;
                sh.rix[wave][0] = ixa;
                sh.rix[wave][1] = ixr;
                sh.rix[wave][2] = ixu;
                sh.rix[wave][3] = fnan;
                sh.rix[wave][4] = fval;
                sh.rmu[wave] = mu;
                sh.rulp[wave] = sulp;
            }
        }
        {
            // fast-path counts: every element there is valid, finite, golden nonzero
            const uint32_t common = Un.common * 64u * VEC;
#pragma unroll
            for (int k = 0; k < kCnt; ++k) {
                const uint32_t v = dpp_sum_u32(L.cnt[k]) + ((k == C_VALID || k == C_FINITE || k == C_REL) ? common : 0u);
                if (lane == 0) sh.rcnt[wave][k] = v;
            }
#pragma unroll
            for (int j = 0; j < PEAT_MAX_THRESHOLDS; ++j) {
                const uint32_t v = j < NT ? dpp_sum_u32(L.mism[j]) + Un.mism[j] : 0u;
                if (lane == 0) sh.rcnt[wave][kCnt + j] = v;
            }
        }
        __syncthreads();

        ChunkPartial *out = partials + c.gchunk;
        // histogram: thread t sums slot t/4 over a quarter of the words and
        // clears them for the next run, 16 bytes at a time (the groups are
        // rotated so that eight consecutive lanes touch all 32 banks)
        {
            const int slot = tid >> 2, q = tid & 3;
            uint32_t acc = 0;
            uint4 *row = reinterpret_cast<uint4 *>(sh.hist + slot * kHistCols + q * 32);
#pragma unroll 2
            for (int k = 0; k < 8; ++k) {
                const int g = (k + slot + 2 * q) & 7;
                const uint4 w = row[g];
                row[g] = make_uint4(0u, 0u, 0u, 0u);
                acc += ((w.x & 0xFFFFu) + (w.x >> 16)) + ((w.y & 0xFFFFu) + (w.y >> 16)) +
                       ((w.z & 0xFFFFu) + (w.z >> 16)) + ((w.w & 0xFFFFu) + (w.w >> 16));
            }
            dsum_step<kDppXor1, 0xF>(acc);        // the four quarters of the slot
            dsum_step<kDppXor2, 0xF>(acc);
            if (q == 0) out->hist[slot] = acc;
            // slots 64..66 (beyond 256/4 threads): 32 threads each, four
            // words per thread, summed across the 32 lanes (one half-wave)
            static_assert(kHistSlots - 64 <= 3 && kHistCols == 4 * 32, "tail slots");
            if (tid < 32 * (kHistSlots - 64)) {
                const int s2 = 64 + (tid >> 5), k0 = (tid & 31) * 4;
                uint32_t a2 = 0;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const uint32_t w = sh.hist[s2 * kHistCols + k0 + k];
                    sh.hist[s2 * kHistCols + k0 + k] = 0;
                    a2 += (w & 0xFFFFu) + (w >> 16);
                }
#pragma unroll
                for (int o = 16; o >= 1; o >>= 1) a2 += __shfl_xor(a2, o);
                if ((tid & 31) == 0) out->hist[s2] = a2;
            }
        }
        // the waves' totals, one field per thread, waves in order
        if (tid >= 64 && tid < 64 + kCnt + PEAT_MAX_THRESHOLDS) {
            int k = tid;
            // formed here rather than kept live (and spilled) across the hot loop
            asm volatile("" : "+v"(k));
            k -= 64;
            uint32_t a = 0;
            for (int w = 0; w < kWaves; ++w) a += sh.rcnt[w][k];
            reinterpret_cast<uint32_t *>(reinterpret_cast<char *>(out) + offsetof(ChunkPartial, cnt))[k] = a;
        } else if (tid == 128) {
            double ma = -1.0;
            uint32_t ia = kNone;
            for (int w = 0; w < kWaves; ++w) lex_merge(ma, ia, sh.rmax[w][0], sh.rix[w][0]);
            out->max_abs = ma;
            out->ix_abs = ia == kNone ? -1 : run_off + ia;
        } else if (tid == 129) {
            double mr = -1.0;
            uint32_t ir = kNone;
            for (int w = 0; w < kWaves; ++w) lex_merge(mr, ir, sh.rmax[w][1], sh.rix[w][1]);
            out->max_rel = mr;
            out->ix_rel = ir == kNone ? -1 : run_off + ir;
        } else if (tid == 130) {
            uint32_t m = 0, iu = kNone, fv = kNone;
            for (int w = 0; w < kWaves; ++w) {
                lex_merge(m, iu, sh.rmu[w], sh.rix[w][2]);
                fv = min(fv, sh.rix[w][4]);
            }
            // every ULP distance in the run is 0: the first valid element is the maximum
            if (iu == kNone || m == 0) {
                m = 0;
                iu = fv;
            }
            out->max_ulp = m;
            out->ix_ulp = iu == kNone ? -1 : run_off + iu;
        } else if (tid == 192) {
            uint32_t fn = kNone, fv = kNone;
            uint64_t su = 0;
            for (int w = 0; w < kWaves; ++w) {
                fn = min(fn, sh.rix[w][3]);
                fv = min(fv, sh.rix[w][4]);
                su += sh.rulp[w];
            }
            out->first_nan = fn == kNone ? -1 : run_off + fn;
            out->first_valid = fv == kNone ? -1 : run_off + fv;
            out->sum_ulp = su;
        }
        // the per-wave records and the histogram are free again
        __syncthreads();
        lane_init(L, Un);
    };

    lane_init(L, Un);
    reset_sums();
    ndef = 0;
    // Two register sets, used in turn: the loads of the next super-step are
    // in flight while the current one is processed.  A chunk's first
    // super-step is always in (ga, ta): the last super-step of the previous
    // chunk issues it, before its processing when it comes from (gb, tb),
    // after it when it comes from (ga, ta), so the chunk's sums are reduced
    // while the next chunk's data is on its way.
    u32x4 ga[U], ta[U], gb[U], tb[U];
    bool pre = false;              // the current chunk's first super-step is loaded
    // the block's chunks c0 + i, i < cnt (at most 8; 32-bit scalar arithmetic)
    const int64_t c0 = (int64_t)blockIdx.x * P.chunk_group;
    const int cnt = (int)__builtin_amdgcn_readfirstlane(
        (uint32_t)(nch - c0 < P.chunk_group ? nch - c0 : P.chunk_group));
    int run_first = 0;             // first chunk of the current run
    int64_t run_off = 0;           // its first element in the pair
    if constexpr (INJ) {
        // Injection first: the bit flips of every chunk of the block are
        // performed in the L2 of the block's XCD (atomics) before any of
        // their elements is loaded.  Each wave waits until its atomics have
        // completed (s_waitcnt 0) and the barrier then orders them before
        // every wave's loads, which go to the same L2; no compute unit holds
        // an older copy of these lines, because the host admits only batches
        // whose test lines no other block reads.  The per-wave candidate
        // queues borrow the histogram's LDS, cleared afterwards.
        uint32_t(*queue)[kQCap] = reinterpret_cast<uint32_t(*)[kQCap]>(sh.hist);
        for (int i = 0; i < cnt; ++i) {
            const ChunkCtx x = ctx(pair_of(c0 + i), c0 + i);
            const InjDesc &d = inj[x.pair];
            const bool none = !d.all && d.T == 0;
            const uint32_t f = none ? 0u : dpp_sum_u32(inject_span<true>(d, (uint64_t)x.off, x.len, queue));
            __builtin_amdgcn_s_waitcnt(0);
            if (lane == 0) sh.rcnt[wave][0] = f;
            __syncthreads();
            if (tid == 0) {
                uint32_t t = 0;
                for (int w = 0; w < kWaves; ++w) t += sh.rcnt[w][0];
                partials[x.gchunk].flips = t;
            }
            __syncthreads();
        }
    }
    PairS dcur = pair_of(c0);
    ChunkCtx cur = ctx(dcur, c0);
    // the block's first super-step is in flight while it sets up its tables
    if (cur.nsuper > 0) {
        load(ga, ta, cur, 0);
        pre = true;
    }
    init_tables(sh, P, tid);
    __syncthreads();
    for (int i = 0; i < cnt; ++i) {
        const int64_t c = c0 + i;
        const bool more = i + 1 < cnt;
        // the next chunk: same pair unless this one is the pair's last
        PairS dnxt = dcur;
        if (more && P.chunk_base + c + 1 >= dcur.first + dcur.nchunks) dnxt = pair_of(c + 1);
        const ChunkCtx nxt = ctx(dnxt, more ? c + 1 : c);
        const bool chain = more && nxt.nsuper > 0;
        const bool run_end = !more || nxt.pair != cur.pair;
        if (i == run_first) run_off = cur.off;
        const uint32_t ib = (uint32_t)(i - run_first) << cur.log2;
        if (cur.nsuper > 0) {
            if (!pre) load(ga, ta, cur, 0);
            // Pairs of super-steps are pipelined: each half step issues one
            // set of loads (the next super-step, or the next chunk's first at
            // the end) before it works, so the waits stay partial.  An odd
            // last super-step, loaded into (ga, ta) by the last pair (or by
            // the chunk's start), is worked after the loop, and only then is
            // the next chunk's first loaded into (ga, ta).  So no load into
            // (gb, tb) is ever in flight when the chunk ends (its registers
            // are reused there), and the next chunk's loads, in (ga, ta), stay
            // in flight through the chunk's end.
            const uint32_t npair = cur.nsuper & ~1u;
            const bool odd = (cur.nsuper & 1u) != 0;
            for (uint32_t s = 0; s < npair; s += 2) {
                load(gb, tb, cur, s + 1);
                step(ga, ta, s, ib);
                const bool last = s + 2 >= npair;
                const bool hop = last && !odd && chain;
                // (ga, ta) next: super-step s + 2 (the odd last one included),
                // the next chunk's first, or a re-read when nothing follows
                load_at(ga, ta, hop ? nxt.gbase : cur.gbase, hop ? nxt.tbase : cur.tbase, hop ? nxt.len : cur.len,
                        hop ? 0u : (last && !odd ? s + 1 : s + 2));
                step(gb, tb, s + 1, ib);
                // the deferred list must hold the next two super-steps (or the
                // odd last one)
                if (ndef > kDeferCap - 2 * U) flush(cur, ib);
            }
            if (odd) {
                step(ga, ta, npair, ib);
                if (chain) load(ga, ta, nxt, 0);
            }
        }
        // a chunk without super-steps issued no load for the next one
        pre = chain && cur.nsuper > 0;
        flush(cur, ib);
        chunk_end(cur, ib, run_end);
        if (run_end) {
            run_end_reduce(cur, run_off);
            run_first = i + 1;
        }
        dcur = dnxt;
        cur = nxt;
    }
}

// Three blocks per CU (12 waves) where the registers allow it without
// spilling in the hot loop: f32 with two absolute thresholds, the common case.
template <int DG, int DT, int NT, bool RT>
constexpr int chunk_blocks_per_cu() { return (DG == DT && NT == 2 && !RT) ? 3 : 2; }

// INJ: inject the test tensors' bit flips first (inj[pair], same decisions
// as the injection kernel) and sign the flipped tensors; the chunk records
// carry the flip counts.
template <int DG, int DT, int NT, bool RT, bool INJ>
__global__ void __launch_bounds__(kBlock, (chunk_blocks_per_cu<DG, DT, NT, RT>()))
    sig_chunk(SigParams P, const SigDesc *__restrict__ descs, const int32_t *__restrict__ chunk_pair,
              ChunkPartial *__restrict__ partials, const InjDesc *__restrict__ inj) {
    __shared__ Shared sh;
    chunk_loop<DG, DT, NT, RT, INJ>(P, sh, descs, chunk_pair, partials, inj);
}

// The same pass for a same-type launch whose goldens are shared by most of
// its pairs (a replay batch: many test tensors against one golden), in the
// common form (two thresholds, no relative tolerance): golden loads keep the
// default cache policy, so the shared lines are served from the caches.  Other
// launches with shared goldens take the nontemporal kernels (the policy is a
// hint: records are the same either way).
template <int DT>
__global__ void __launch_bounds__(kBlock, (chunk_blocks_per_cu<DT, DT, 2, false>()))
    sig_chunk_keep(SigParams P, const SigDesc *__restrict__ descs, const int32_t *__restrict__ chunk_pair,
                   ChunkPartial *__restrict__ partials) {
    __shared__ Shared sh;
    chunk_loop<DT, DT, 2, false, false, true>(P, sh, descs, chunk_pair, partials, nullptr);
}

// Blocks of one chunk-pass instantiation that the current device holds at
// once: its occupancy per compute unit times the compute units, looked up
// once per device.
template <int DG, int DT, int NT, bool RT, bool INJ>
int64_t resident_blocks() {
    constexpr int kDevs = 64;
    static std::atomic<int32_t> cached[kDevs];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) dev = -1;
    if (dev >= 0 && dev < kDevs) {
        const int32_t v = cached[dev].load(std::memory_order_relaxed);
        if (v > 0) return v;
    }
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, sig_chunk<DG, DT, NT, RT, INJ>, kBlock, 0) != hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    if (dev < 0 || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 256;
    (void)hipGetLastError();        // a failed query above is not the launch's error
    const int32_t v = per_cu * cus;
    if (dev >= 0 && dev < kDevs) cached[dev].store(v, std::memory_order_relaxed);
    return v;
}


template <int DG, int DT, int NT, bool RT, bool INJ>
void launch_chunks(const SigParams &p, int64_t n, const InjDesc *inj, hipStream_t s) {
    const int64_t r = resident_blocks<DG, DT, NT, RT, INJ>();
    const int64_t avg = p.launch_elems / n;
    int64_t kmax = kGroupElems / (avg > 0 ? avg : 1);
    kmax = kmax < 2 ? 2 : (kmax > kMaxGroup ? kMaxGroup : kmax);
    int64_t k = n / (kMinRounds * r);
    k = k < 1 ? 1 : (k > kmax ? kmax : k);
    SigParams q = p;
    q.chunk_count = n;
    q.chunk_group = k;
    if constexpr (DG == DT && NT == 2 && !RT && !INJ) {
        if (p.gkeep) {
            hipLaunchKernelGGL((sig_chunk_keep<DT>), dim3((unsigned)((n + k - 1) / k)), dim3(kBlock), 0, s, q,
                               static_cast<const SigDesc *>(p.descs), static_cast<const int32_t *>(p.chunk_pair),
                               p.partials);
            return;
        }
    }
    hipLaunchKernelGGL((sig_chunk<DG, DT, NT, RT, INJ>), dim3((unsigned)((n + k - 1) / k)), dim3(kBlock), 0, s, q,
                       static_cast<const SigDesc *>(p.descs), static_cast<const int32_t *>(p.chunk_pair), p.partials,
                       inj);
}

template <int DG, int DT, bool RT, bool INJ>
hipError_t launch_kind_rt(const SigParams &p, int64_t n, const InjDesc *inj, hipStream_t s) {
    switch (p.nthr_pad) {
        case 2: launch_chunks<DG, DT, 2, RT, INJ>(p, n, inj, s); break;
        case 4: launch_chunks<DG, DT, 4, RT, INJ>(p, n, inj, s); break;
        default: launch_chunks<DG, DT, 8, RT, INJ>(p, n, inj, s); break;
    }
    return hipGetLastError();
}

// Pass 1 over n chunks of one kind, starting at p.chunk_base.
template <int DG, int DT>
hipError_t launch_kind(const SigParams &p, int64_t n, hipStream_t s) {
    return p.any_rtol ? launch_kind_rt<DG, DT, true, false>(p, n, nullptr, s)
                      : launch_kind_rt<DG, DT, false, false>(p, n, nullptr, s);
}

// Pass 1 with the injection of the test tensors (same-type kinds).
template <int DT>
hipError_t launch_kind_inject(const SigParams &p, int64_t n, const InjDesc *inj, hipStream_t s) {
    return p.any_rtol ? launch_kind_rt<DT, DT, true, true>(p, n, inj, s)
                      : launch_kind_rt<DT, DT, false, true>(p, n, inj, s);
}

}  // namespace
}  // namespace peat

