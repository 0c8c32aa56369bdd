// Internal declarations of libpeat: device-side descriptors, the per-chunk
// partial record of the signature pass, and launch entry points shared by the
// host API and the kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "peat.h"

namespace peat {

constexpr int kBlock = 256;                        // threads per block (4 wave64)
constexpr int kWaves = kBlock / 64;
constexpr int kHistSlots = PEAT_MAX_BINS + 3;      // zero | under | bins | over
constexpr uint32_t kNone = 0xFFFFFFFFu;            // "no element" local index
constexpr int kMinChunkLog2 = 12;                  // 4096 elements: 16 per thread
constexpr int kMaxChunkLog2 = 18;                  // 262144 elements: 1024 per thread
constexpr int kInjSegLog2 = 20;                    // injector segment: 2^20 elements

// Chunk size of a pair depends on n only, so that a pair's partition (and
// hence its binary64 summation tree) is the same in single and batched calls.
// Below 2^22 elements a pair gets about 256 chunks (a lone pair still spreads
// over many CUs); from 2^22 on about 64, whose longer blocks amortise the
// per-chunk set-up and epilogue (batches of 2^24-element pairs run 10-13 %
// faster than with 256); clamped to [2^12, 2^18] elements.
inline int chunk_log2_for(int64_t n) {
    const int64_t target = n >= (int64_t(1) << 22) ? 64 : 256;
    int64_t per = (n + target - 1) / target;
    int l = 0;
    while (l < 62 && (int64_t(1) << l) < per) ++l;
    if (l < kMinChunkLog2) l = kMinChunkLog2;
    if (l > kMaxChunkLog2) l = kMaxChunkLog2;
    return l;
}

// Golden/test type combinations ("kinds"), one kernel instantiation each:
// the three same-type kinds first, then the mixed-precision ones (the golden
// side is never binary64, and the two formats nest).
constexpr int kKinds = 10;
constexpr int kSameKinds = 3;
constexpr int kKindTypes[kKinds][2] = {
    {PEAT_F32, PEAT_F32},  {PEAT_F16, PEAT_F16}, {PEAT_BF16, PEAT_BF16}, {PEAT_F32, PEAT_F64},
    {PEAT_F32, PEAT_F16},  {PEAT_F32, PEAT_BF16}, {PEAT_F16, PEAT_F32}, {PEAT_BF16, PEAT_F32},
    {PEAT_F16, PEAT_F64},  {PEAT_BF16, PEAT_F64}};

// Kind of a (golden, test) type pair, or -1 when the combination is not accepted.
inline int pair_kind(int32_t g, int32_t t) {
    for (int k = 0; k < kKinds; ++k)
        if (kKindTypes[k][0] == g && kKindTypes[k][1] == t) return k;
    return -1;
}

inline int elem_bytes(int32_t dt) { return dt == PEAT_F64 ? 8 : (dt == PEAT_F32 ? 4 : 2); }

struct SigDesc {                 // one per pair (48 bytes)
    const void *g;
    const void *t;
    int64_t n;
    int64_t first_chunk;         // index of the pair's first chunk in the batch
    int32_t nchunks;
    int16_t dtype;               // golden type
    int16_t tdtype;              // test type
    int32_t chunk_log2;
    int32_t aligned;             // both pointers 16-byte aligned
};
static_assert(sizeof(SigDesc) == 48, "SigDesc layout");

enum { C_VALID, C_FINITE, C_REL, C_NAN_G, C_NAN_T, C_INF_G, C_INF_T, C_NANPAIR, kCnt };

struct alignas(16) ChunkPartial {   // one per chunk, written by the chunk pass
    // 1 when the chunk ends its block's run of chunks of one pair: only then
    // do the exact fields below (maxima to histogram) hold the run's values,
    // otherwise they are not written
    int64_t run_end;
    // binary64 sums of each wave of the block: |err|, err^2, rel, g^2, t^2, g*t
    double s[kWaves][6];
    double max_abs, max_rel;
    int64_t ix_abs, ix_rel, ix_ulp;  // element index within the pair, -1 = none
    int64_t first_nan, first_valid;  // -1 = none
    uint64_t sum_ulp;
    uint32_t max_ulp;
    uint32_t cnt[kCnt];
    uint32_t mism[PEAT_MAX_THRESHOLDS];
    uint32_t hist[kHistSlots];
    uint32_t flips;                  // bit flips injected in the chunk (fused injection)
};
// the chunk pass writes the counts followed by the mismatches as one array
static_assert(offsetof(ChunkPartial, mism) == offsetof(ChunkPartial, cnt) + kCnt * sizeof(uint32_t),
              "ChunkPartial counts");
// wave 0 writes run_end and its six sums as seven consecutive 8-byte words
static_assert(offsetof(ChunkPartial, s) == sizeof(int64_t), "ChunkPartial run_end");

struct SigParams {
    int64_t chunk_base;            // first global chunk of this launch
    int64_t chunk_count;           // chunks of this launch
    int64_t chunk_group;           // consecutive chunks per block
    const SigDesc *descs;
    const int32_t *chunk_pair;     // chunk -> pair index
    ChunkPartial *partials;        // one per chunk
    peat_signature_t *outs;        // one per pair (device)
    int64_t *inj_counts;           // flips per pair (device), fused injection only
    int32_t count;                 // pairs
    int32_t lo, hi, nbins;
    int32_t nthr;                  // real thresholds
    int32_t nthr_pad;              // 2, 4 or 8 compared per element (+Inf padding)
    double thr[PEAT_MAX_THRESHOLDS];   // absolute tolerances
    double rthr[PEAT_MAX_THRESHOLDS];  // relative tolerances
    double thr_min;                // smallest thr (+Inf when there are none)
    int32_t any_rtol;              // some relative tolerance is nonzero
    int32_t single;                // one pair, described by `one` (descs and chunk_pair unused)
    // most pairs share a few golden tensors (a replay batch): golden loads
    // keep the default cache policy so that the shared lines stay cached
    int32_t gkeep;
    SigDesc one;
    int64_t kind_elems[kKinds];    // elements of the pairs of each kind
    int64_t launch_elems;          // elements of this launch's chunks
};

struct InjDesc {                 // one per injected tensor (80 bytes)
    void *x;
    int64_t n;
    uint64_t seed;
    uint64_t T;                  // floor(rate * 2^64) when !all
    uint64_t mask;
    const void *src;             // PEAT_MODEL_VALUE: copy of x taken before the call
    int64_t first_seg;
    int32_t nsegs;
    int32_t dtype;
    int32_t all;                 // rate >= 1
    int32_t popc;                // popcount(mask)
    int32_t model;               // peat_model_t
    int32_t reserved;
};
static_assert(sizeof(InjDesc) == 80, "InjDesc layout");

struct InjParams {
    const InjDesc *descs;
    const int32_t *seg_item;     // segment -> item index
    uint32_t *seg_counts;        // flips per segment
    int64_t *counts;             // flips per item (device)
    int32_t count;
};

// ---- top-k error mean --------------------------------------------------------
// Radix selection on the binary64 bit pattern of the error (monotone for
// a >= 0): digit 0 = bits 62..52 (the binade, 2048 bins), digits 1-4 = 13
// mantissa bits each (8192 bins).  The boundary's binade D0 comes from the
// pair's signature or from a binade histogram; one pass then sums the errors
// above D0, histograms digit 1 inside it and gathers its errors as
// deduplicated (key, count) entries, on which digits 2-4 are resolved.  When
// the signature only bounds the k-th largest error to a window of binades,
// or a sample of the pair suggests one, that pass gathers the whole window
// and every level comes from the entries.
constexpr int kTopkLevels = 5;
constexpr int kTopkBins = 8192;                  // bins of digits 1-4
enum { kTopkActive = 0, kTopkDone = 1 };

struct TopkState {               // one per pair (80 bytes), device memory
    uint64_t n_valid;
    uint64_t k;
    uint64_t need;               // k minus the errors above the boundary bin (or window)
    uint64_t cand;               // errors in the boundary bin (or window)
    uint64_t key;                // bits of the boundary fixed so far
    uint64_t wlo, whi;           // window [wlo, whi) of error keys holding the k-th largest
    int32_t level;               // last resolved level; -1 before level 0, -2 window gather pending
    int32_t status;              // kTopkActive or kTopkDone
    int32_t d0;                  // binade field of the boundary
    int32_t round;               // gathering pass that serves the pair (0, or 1 after a window overflowed)
    int32_t sampled;             // the binade is a guess from a sample: pass A counts the errors to confirm it
    int32_t reserved;
};
static_assert(sizeof(TopkState) == 80, "TopkState layout");

struct TopkEntry {               // errors of one key in one chunk (16 bytes)
    uint64_t key;
    uint32_t count;
    int32_t pair;                // pair | round << 30; -1: an unused position
};
static_assert(sizeof(TopkEntry) == 16, "TopkEntry layout");

struct TopkParams {
    int64_t chunk_base;          // first global chunk of this launch
    int64_t kind_chunks;         // chunks of this launch
    const SigDesc *descs;
    const int32_t *chunk_pair;
    TopkState *state;
    uint64_t *hist;              // count x kTopkBins counters
    double *part_a;              // per chunk: binary64 sum of its errors above binade D0
    uint64_t *xsum;              // per pair and binade: exact sum (2 words) of the significands above the boundary
    uint64_t *counts;            // per pair: valid errors, errors above a guessed binade
    uint32_t *ovf;               // per pair: [0] gather of binade D0 (or window) did not fit, [1] gather of bin
                                 // (D0, D1) did not fit; then 3 words: some pair has flag 0 set, some pair has
                                 // flag 1 set, some window gather did not fit
    TopkEntry *ents;             // cap[0] entries of binade D0 gathers, then cap[1] of bin (D0, D1) gathers
    unsigned long long *fill;    // entries handed out in each of the two regions
    uint64_t cap[2];
    const peat_signature_t *sigs;    // the pairs' signatures (device), or NULL
    peat_topk_t *outs;           // one per pair (device)
    int32_t lo, hi, nbins;       // the bins of those signatures
    int32_t count;               // pairs
    int32_t num, den;
    int32_t level;               // level of a selection, tensor-pass or entry launch
    int32_t round;               // gathering-pass round of a launch
};

// Kernel launchers (defined in the .hip translation units).
// One launch per kind present: chunks of each kind form one contiguous range
// [range[kind], range[kind + 1]) of the global chunk numbering.
hipError_t launch_sig_chunks(const SigParams &p, const int64_t range[kKinds + 1], hipStream_t s);
hipError_t launch_sig_mixed_kind(const SigParams &p, int kind, int64_t nchunks, hipStream_t s);
// Pass 1 of the same-type kinds with the test tensors' bit flips injected
// first (inj: one InjDesc per pair, device); the records carry flip counts.
hipError_t launch_sig_chunks_inject(const SigParams &p, const int64_t range[kKinds + 1], const InjDesc *inj,
                                    hipStream_t s);
hipError_t launch_sig_finalize(const SigParams &p, hipStream_t s);
hipError_t launch_inject(const InjParams &p, int64_t total_segs, hipStream_t s);
hipError_t launch_inject_sum(const InjParams &p, hipStream_t s);
hipError_t launch_corrupt_positions(void *x, int64_t n, int dtype, uint64_t seed, int model, int64_t num_pos,
                                    uint64_t mask, int64_t *d_positions, hipStream_t s);
hipError_t launch_cast_round(void *x, int64_t n, int to_dtype, hipStream_t s);
hipError_t launch_stream_read(const void *buf, int64_t bytes, uint32_t *sink, hipStream_t s);
// The top-k selection of a batch, stream-ordered (no host wait): level 0
// (state, binade histogram where the signatures leave it open, selection),
// then the rest up to the records.
hipError_t launch_topk_level0(const TopkParams &p, const int64_t range[kKinds + 1], hipStream_t s);
hipError_t launch_topk_rest(const TopkParams &p, const int64_t range[kKinds + 1], hipStream_t s);

}  // namespace peat
