// Mean of the k largest errors of each pair (the "mean of the top 10%
// errors" score of Section IV-B.3, the Analyzer's main score in Section IV-C),
// by exact radix selection on the binary64 bit pattern of the error, which is
// monotone for a >= 0.  The whole selection is stream-ordered: every count,
// boundary and buffer fill stays on the device, so no step waits on the host.
//
//   init     per pair: the state of level 0 from its signature when one is
//            given: its histogram fixes the binade D0 of the k-th largest
//            error (one-binade bins, boundary in a regular bin or among the
//            zero errors) or bounds it to a window of binades (the under or
//            over bin, wider bins); otherwise level 0 is open;
//   sample   per open pair of 2^16 elements or more: a strided sample of
//            8 K elements guesses D0 (a one-binade window whose guess pass A
//            confirms by counting);
//   pass 1   histogram of digit 0 (bits 62..52, the binade) over the pairs
//            whose level 0 is still open; select D0;
//   pass A   binary64 sum of the errors above the gathered range (a fixed
//            per-lane / butterfly / wave order in each chunk) and a gather of
//            the range -- binade D0 or the window -- as (key, count) entries:
//            each block counts its distinct keys in an LDS hash table (errors
//            of checkpoint-like data are small multiples of the golden's ULP,
//            so a binade holds few distinct values) and appends one entry per
//            key; for binade D0 also the digit-1 (bits 51..39) histogram;
//   windows  level 0 of a window from its entries' binades (a signature's
//            window) or from the counts (a guess); a window that does not
//            fit, or a wrong guess, reopens level 0: pass 1 and pass A again
//            for those pairs (round 1);
//   rounds   digits 1-4 on the entries as needed: weighted histogram, select;
//            then the exact integer sums count * significand of the entries
//            above the boundary, per binade;
//   finalize sum = pass A + the exact sums (binade D0 with need copies of T,
//            and a signature's window binades above it, from the top).
//
// A pair whose binade does not fit (a block's table overflows, or the entry
// buffer is full) instead takes pass C over its tensors: the exact sum of
// its errors in D0 above bin D1 and a gather of bin (D0, D1), whose keys
// that do not fit the table become entries of count 1; the rounds then run
// on those entries.  A pair whose bin does not fit either takes one
// histogram pass over its tensors per digit (passes T2-T4) and a last pass
// for the exact sum of digit 4 (T5).  Every route sums the errors inside D0
// exactly and the others in the lanes' order, so they give bit-identical
// records; only a signature's window of several binades sums the binades
// between D0 and its top exactly instead.
//
// The k-th largest error T is the key with all five digits fixed; count_above
// is k minus the copies of T taken.
#include "elements.h"

namespace peat {
namespace {

constexpr int kBins0 = 2048;                    // digit 0: the binade field

// A binary64 built from two 32-bit halves held in vector registers, opaque to
// constant folding.  The record's NaN and +Inf go through it: as folded
// constants they became 64-bit scalar moves whose immediate lost its high
// word in the gfx950 code object (the literal was encoded as 0).
__device__ __forceinline__ double opaque_double(uint32_t hi, uint32_t lo) {
    asm volatile("" : "+v"(hi), "+v"(lo));
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
constexpr uint64_t kMant = (uint64_t(1) << 52) - 1;
constexpr int kTable = 512;                     // LDS hash table of a gather (keys per block)
constexpr int kProbes = 8;
constexpr uint64_t kEmpty = ~uint64_t(0);       // never a key: errors have the sign bit clear
constexpr int kScanGrid = 2048;                 // blocks of the fallback tensor passes
constexpr int kEntGrid = 1024;                  // blocks of the entry rounds
enum { kModeA = 0, kModeC = 1, kModeT = 2 };    // route of an active pair

__device__ __forceinline__ int digit_shift(int level) { return level == 0 ? 52 : 52 - 13 * level; }

__device__ __forceinline__ uint32_t digit_of(uint64_t key, int level) {
    if (level == 0) return (uint32_t)(key >> 52);               // sign bit is 0
    return (uint32_t)(key >> digit_shift(level)) & (kTopkBins - 1);
}

// Significand of an error of binade d0 as an integer: binade 0 (zero and
// subnormal errors) has no implicit bit and the exponent of binade 1.
__device__ __forceinline__ uint64_t signif(uint64_t key, int d0) {
    return (key & kMant) | (d0 != 0 ? (uint64_t(1) << 52) : 0);
}

// Entries carry their pair and the round of the gathering pass that wrote
// them; a pair whose window did not fit, or whose guessed binade was wrong,
// is gathered again in round 1 and ignores what round 0 left.
constexpr uint32_t kPairMask = (1u << 30) - 1;
__device__ __forceinline__ int32_t entry_tag(int pair, int round) { return (int32_t)((uint32_t)pair | ((uint32_t)round << 30)); }

// The pair's exact sum of significands of binade b (two words).
__device__ __forceinline__ uint64_t *xsum_of(const TopkParams &P, int pair, int b) {
    return P.xsum + 2 * ((size_t)pair * kBins0 + (size_t)b);
}

__device__ __forceinline__ bool is_window(const TopkState &st) { return st.whi != 0; }

__device__ __forceinline__ int pair_mode(const TopkParams &P, int pair) {
    return P.ovf[2 * pair] == 0 ? kModeA : (P.ovf[2 * pair + 1] == 0 ? kModeC : kModeT);
}

// Exact 128-bit accumulation: the carry of each low-word addition is
// recovered from the value the atomic returns.
__device__ __forceinline__ void atomic_add128(uint64_t *x, uint64_t lo, uint64_t hi) {
    if (lo) {
        const uint64_t old = atomicAdd((unsigned long long *)&x[0], (unsigned long long)lo);
        hi += (old + lo < old) ? 1u : 0u;
    }
    if (hi) atomicAdd((unsigned long long *)&x[1], (unsigned long long)hi);
}

// Error of a valid pair (no NaN on either side) and its bit pattern.
template <int DG, int DT, typename BG, typename BT>
__device__ __forceinline__ bool error_of(BG gb, BT tb, uint64_t &key, double &a) {
    const double G = widen<DG>(gb), T = widen<DT>(tb);
    if (G != G || T != T) return false;
    a = (G == T) ? 0.0 : __builtin_fabs(T - G);
    key = (uint64_t)__double_as_longlong(a);
    return true;
}

// Calls f(key, a) for every valid pair of chunk `cin` of pair d, each lane in
// a fixed order: lane vectors (16 bytes of the wider side, four per step in
// flight), then the ragged tail (or the whole chunk when a pointer is not
// 16-byte aligned).
template <int DG, int DT, typename F>
__device__ __forceinline__ void for_each_error(const SigDesc &d, int64_t cin, F &&f) {
    using PT = PairTr<DG, DT>;
    constexpr int VEC = PT::VEC;
    constexpr int ESZG = Tr<DG>::W / 8, ESZT = Tr<DT>::W / 8;
    constexpr int BG = PT::BG, BT = PT::BT;
    constexpr int U = 4;
    const int64_t off = cin << d.chunk_log2;
    const int64_t rest = d.n - off;
    const uint32_t len = (uint32_t)(rest < (int64_t(1) << d.chunk_log2) ? rest : (int64_t(1) << d.chunk_log2));
    const char *gbase = static_cast<const char *>(d.g) + off * ESZG;
    const char *tbase = static_cast<const char *>(d.t) + off * ESZT;
    const uint32_t nvec = d.aligned ? len / VEC : 0;
    if (nvec > 0) {
        const __amdgpu_buffer_rsrc_t grs =
            __builtin_amdgcn_make_buffer_rsrc((void *)gbase, (short)0, (int)(nvec * BG), kBufFlags);
        const __amdgpu_buffer_rsrc_t trs =
            __builtin_amdgcn_make_buffer_rsrc((void *)tbase, (short)0, (int)(nvec * BT), kBufFlags);
        uint32_t v = threadIdx.x;
        for (; v + (U - 1) * kBlock < nvec; v += U * kBlock) {
            u32x4 gv[U], tv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                gv[u] = buf_load<BG, kLoadNT>(grs, (int)((v + u * kBlock) * BG), 0);
                tv[u] = buf_load<BT, kLoadNT>(trs, (int)((v + u * kBlock) * BT), 0);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
#pragma unroll
                for (int j = 0; j < VEC; ++j) {
                    uint64_t key;
                    double a;
                    if (error_of<DG, DT>(lane_elem<DG>(gv[u], j), lane_elem<DT>(tv[u], j), key, a)) f(key, a);
                }
            }
        }
        for (; v < nvec; v += kBlock) {
            const u32x4 gv = buf_load<BG, kLoadNT>(grs, (int)(v * BG), 0);
            const u32x4 tv = buf_load<BT, kLoadNT>(trs, (int)(v * BT), 0);
#pragma unroll
            for (int j = 0; j < VEC; ++j) {
                uint64_t key;
                double a;
                if (error_of<DG, DT>(lane_elem<DG>(gv, j), lane_elem<DT>(tv, j), key, a)) f(key, a);
            }
        }
    }
    for (uint32_t i = nvec * VEC + threadIdx.x; i < len; i += kBlock) {
        uint64_t key;
        double a;
        if (error_of<DG, DT>(load_elem<DG>(gbase, i), load_elem<DT>(tbase, i), key, a)) f(key, a);
    }
}

// As for_each_error, one lane vector at a time: f(key, a, ok) with arrays of
// VEC elements (ok: the element exists and is a valid pair), so that work on
// the elements of a vector can be issued together.  Tail elements come one
// per call, in element 0.
template <int DG, int DT, typename F>
__device__ __forceinline__ void for_each_error_vec(const SigDesc &d, int64_t cin, F &&f) {
    using PT = PairTr<DG, DT>;
    constexpr int VEC = PT::VEC;
    constexpr int ESZG = Tr<DG>::W / 8, ESZT = Tr<DT>::W / 8;
    constexpr int BG = PT::BG, BT = PT::BT;
    constexpr int U = VEC > 4 ? 2 : 4;                        // vectors in flight per lane
    const int64_t off = cin << d.chunk_log2;
    const int64_t rest = d.n - off;
    const uint32_t len = (uint32_t)(rest < (int64_t(1) << d.chunk_log2) ? rest : (int64_t(1) << d.chunk_log2));
    const char *gbase = static_cast<const char *>(d.g) + off * ESZG;
    const char *tbase = static_cast<const char *>(d.t) + off * ESZT;
    const uint32_t nvec = d.aligned ? len / VEC : 0;
    constexpr int NB = VEC < 4 ? VEC : 4;                     // elements per call
    uint64_t key[NB];
    double a[NB];
    bool ok[NB];
    if (nvec > 0) {
        const __amdgpu_buffer_rsrc_t grs =
            __builtin_amdgcn_make_buffer_rsrc((void *)gbase, (short)0, (int)(nvec * BG), kBufFlags);
        const __amdgpu_buffer_rsrc_t trs =
            __builtin_amdgcn_make_buffer_rsrc((void *)tbase, (short)0, (int)(nvec * BT), kBufFlags);
        uint32_t v = threadIdx.x;
        for (; v + (U - 1) * kBlock < nvec; v += U * kBlock) {
            u32x4 gv[U], tv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                gv[u] = buf_load<BG, kLoadNT>(grs, (int)((v + u * kBlock) * BG), 0);
                tv[u] = buf_load<BT, kLoadNT>(trs, (int)((v + u * kBlock) * BT), 0);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
#pragma unroll
                for (int jb = 0; jb < VEC; jb += NB) {
#pragma unroll
                    for (int j = 0; j < NB; ++j)
                        ok[j] = error_of<DG, DT>(lane_elem<DG>(gv[u], jb + j), lane_elem<DT>(tv[u], jb + j), key[j], a[j]);
                    f(key, a, ok);
                }
            }
        }
        for (; v < nvec; v += kBlock) {
            const u32x4 gv = buf_load<BG, kLoadNT>(grs, (int)(v * BG), 0);
            const u32x4 tv = buf_load<BT, kLoadNT>(trs, (int)(v * BT), 0);
#pragma unroll
            for (int jb = 0; jb < VEC; jb += NB) {
#pragma unroll
                for (int j = 0; j < NB; ++j)
                    ok[j] = error_of<DG, DT>(lane_elem<DG>(gv, jb + j), lane_elem<DT>(tv, jb + j), key[j], a[j]);
                f(key, a, ok);
            }
        }
    }
#pragma unroll
    for (int j = 1; j < NB; ++j) ok[j] = false;
    for (uint32_t i = nvec * VEC + threadIdx.x; i < len; i += kBlock) {
        ok[0] = error_of<DG, DT>(load_elem<DG>(gbase, i), load_elem<DT>(tbase, i), key[0], a[0]);
        f(key, a, ok);
    }
}

// Block sum of one binary64 per thread in a fixed order (wave butterflies,
// then the waves in order); the result is valid in thread 0.
__device__ __forceinline__ double block_sum(double x, double *red) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
    __syncthreads();
    double s = 0.0;
    if (threadIdx.x == 0) {
#pragma unroll
        for (int w = 0; w < kWaves; ++w) s += red[w];
    }
    return s;
}

// Adds the block's per-thread integers (each below 2^64) into the pair's
// 128-bit exact sum: wave sums in 128 bits, one atomic pair per wave.
__device__ __forceinline__ void block_add128(uint64_t x, uint64_t *dst) {
    uint64_t lo = x, hi = 0;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const uint64_t ol = __shfl_xor(lo, o), oh = __shfl_xor(hi, o);
        const uint64_t s = lo + ol;
        hi += oh + (s < lo ? 1u : 0u);
        lo = s;
    }
    if ((threadIdx.x & 63) == 0) atomic_add128(dst, lo, hi);
}

// Adds the block's LDS histogram to the pair's device histogram.
__device__ __forceinline__ void flush_hist(const uint32_t *h, int nb, uint64_t *H) {
    __syncthreads();
    for (int b = threadIdx.x; b < nb; b += kBlock)
        if (h[b]) atomicAdd((unsigned long long *)&H[b], (unsigned long long)h[b]);
}

// ---- LDS gather table ----------------------------------------------------------
struct Table {
    uint64_t key[kTable];
    uint32_t cnt[kTable];
    uint32_t full;               // some key found no slot
    uint32_t n;                  // occupied slots (flush)
    uint32_t pos;                // entries written (flush)
    uint32_t ok;                 // the flush fits the buffer
    unsigned long long base;
};

__device__ __forceinline__ void table_init(Table &t) {
    for (int i = threadIdx.x; i < kTable; i += kBlock) {
        t.key[i] = kEmpty;
        t.cnt[i] = 0;
    }
    if (threadIdx.x == 0) {
        t.full = 0;
        t.n = 0;
        t.pos = 0;
    }
}

// Counts key in the table (open addressing, slots go from empty to one key
// only); false when its probe sequence is full of other keys.
__device__ __forceinline__ uint32_t table_slot(uint64_t key) {
    return (uint32_t)((key * 0x9E3779B97F4A7C15ull) >> 55);                 // 9 bits
}

__device__ __forceinline__ bool table_count(Table &t, uint64_t key) {
    const uint32_t h = table_slot(key);
#pragma unroll 1
    for (int p = 0; p < kProbes; ++p) {
        const uint32_t slot = (h + p) & (kTable - 1);
        uint64_t cur = __hip_atomic_load(&t.key[slot], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (cur == kEmpty)
            cur = atomicCAS((unsigned long long *)&t.key[slot], (unsigned long long)kEmpty, (unsigned long long)key);
        if (cur == kEmpty || cur == key) {
            atomicAdd(&t.cnt[slot], 1u);
            return true;
        }
    }
    return false;
}

// Writes the table's keys as entries of `pair` into region r, or marks the
// pair (flag r) when a key found no slot or the region is full; positions
// handed out past the region's end are left to later overflows, positions
// inside it that this block cannot use are marked unused.
__device__ __forceinline__ void table_flush(Table &t, const TopkParams &P, int r, int pair, int round,
                                            bool window) {
    __syncthreads();
    for (int i = threadIdx.x; i < kTable; i += kBlock)
        if (t.cnt[i]) atomicAdd(&t.n, 1u);
    __syncthreads();
    if (threadIdx.x == 0) {
        // positions are taken only for a complete table; taken positions that
        // run past the region's end are given back as unused entries
        uint32_t n = t.full ? 0u : t.n;
        unsigned long long base = 0;
        uint32_t ok = t.full == 0;
        if (n > 0) {
            base = atomicAdd(&P.fill[r], (unsigned long long)n);
            if (base + n > P.cap[r]) ok = 0;
        }
        if (!ok) {
            P.ovf[2 * pair + r] = 1;
            P.ovf[2 * P.count + (window ? 2 : r)] = 1;
        }
        t.base = base;
        t.ok = ok;
        t.n = n;
    }
    __syncthreads();
    TopkEntry *E = P.ents + (r ? P.cap[0] : 0);
    const unsigned long long base = t.base;
    if (t.ok) {
        for (int i = threadIdx.x; i < kTable; i += kBlock)
            if (t.cnt[i]) {
                const uint32_t q = atomicAdd(&t.pos, 1u);
                E[base + q] = TopkEntry{t.key[i], t.cnt[i], entry_tag(pair, round)};
            }
    } else {
        const unsigned long long end = base + t.n < P.cap[r] ? base + t.n : P.cap[r];
        for (unsigned long long q = base + threadIdx.x; q < end; q += kBlock) E[q] = TopkEntry{0, 0, -1};
    }
}

// Appends (key, 1) entries of keys that found no slot to region 1, one
// atomic per wave; a wave past the region's end marks the pair.
__device__ __forceinline__ void spill_entry(bool take, uint64_t key, const TopkParams &P, int pair, int round) {
    const uint64_t m = __ballot(take);
    if (m == 0) return;
    const int leader = __ffsll((long long)m) - 1;
    unsigned long long base = 0;
    if ((int)(threadIdx.x & 63) == leader) base = atomicAdd(&P.fill[1], (unsigned long long)__popcll(m));
    base = __shfl(base, leader);
    if (take) {
        const uint32_t rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        const unsigned long long q = base + rank;
        if (q < P.cap[1]) {
            P.ents[P.cap[0] + q] = TopkEntry{key, 1u, entry_tag(pair, round)};
        } else {
            P.ovf[2 * pair + 1] = 1;
            P.ovf[2 * P.count + 1] = 1;
        }
    }
}

// ---- level 0 ----------------------------------------------------------------
// Status after level 0 resolved to binade b: an infinite boundary fixes the
// k-th largest error already, and so does binade 0 when it holds only zero
// errors; with a binary64 test side it also holds the subnormal errors,
// which the next levels order like any other binade.
__device__ __forceinline__ void level0_status(TopkState &st, int b, int tdtype) {
    st.d0 = b;
    st.level = 0;
    const bool zero_only = b == 0 && tdtype != PEAT_F64;
    st.status = (zero_only || b == kBins0 - 1) ? kTopkDone : kTopkActive;
}

// Level 0 from the pair's signature, which counts the same errors of the same
// valid pairs.  Bin i of the record covers the error keys from that of
// 2^(lo + i w) up to that of 2^(lo + (i + 1) w); with one-binade bins (w = 1)
// a regular bin is binade field lo + i + 1023 and fixes level 0.  A wider bin,
// the under bin (keys 1 up to that of 2^lo) or the over bin (from 2^hi up,
// +Inf included) leaves a window of binades, which the gathering pass
// collects whole.  Errors below every bin are the zero errors alone when the
// test side is not binary64 (a difference of two narrower values is a
// multiple of 2^-149, far above the subnormal range): the k-th largest error
// is then 0.  Leaves the state open when the record does not match the pair.
__device__ void level0_from_sig(const peat_signature_t &g, const SigDesc &d, const TopkParams &P,
                                TopkState &st) {
    if (g.n != d.n || g.n_valid < 0) return;
    uint64_t tot = (uint64_t)g.hist_zero + (uint64_t)g.hist_under + (uint64_t)g.hist_over;
    for (int i = 0; i < P.nbins; ++i) tot += (uint64_t)g.hist[i];
    if (tot != (uint64_t)g.n_valid) return;
    const uint64_t nv = (uint64_t)g.n_valid;
    const uint64_t k = (uint64_t)(((unsigned __int128)nv * (uint32_t)P.num + (uint32_t)P.den - 1) / (uint32_t)P.den);
    st.n_valid = nv;
    st.k = k;
    if (k == 0) {
        st.level = 0;
        st.status = kTopkDone;
        st.d0 = 0;
        return;
    }
    auto key_of = [](int e) { return (uint64_t)(e + 1023) << 52; };      // key of 2^e
    uint64_t acc = 0;
    auto window = [&](uint64_t lo, uint64_t hi, uint64_t c) {
        st.need = k - acc;
        st.cand = c;
        st.wlo = lo;
        st.whi = hi;
        st.level = -2;
        st.status = kTopkActive;
    };
    const uint64_t over = (uint64_t)g.hist_over;
    if (k <= over) {
        window(key_of(P.hi), uint64_t(1) << 63, over);
        return;
    }
    acc = over;
    const int w = (P.hi - P.lo) / P.nbins;
    for (int i = P.nbins - 1; i >= 0; --i) {
        const uint64_t c = (uint64_t)g.hist[i];
        if (acc + c >= k) {
            if (w == 1) {
                st.need = k - acc;
                st.cand = c;
                st.key = key_of(P.lo + i);
                level0_status(st, P.lo + i + 1023, d.tdtype);
            } else {
                window(key_of(P.lo + i * w), key_of(P.lo + (i + 1) * w), c);
            }
            return;
        }
        acc += c;
    }
    const uint64_t under = (uint64_t)g.hist_under;
    if (k <= acc + under) {
        window(1, key_of(P.lo), under);
        return;
    }
    acc += under;
    if (d.tdtype == PEAT_F64) return;
    st.need = k - acc;
    st.cand = (uint64_t)g.hist_zero;
    st.key = 0;
    level0_status(st, 0, d.tdtype);
}

__global__ void __launch_bounds__(kBlock) topk_init(TopkParams P) {
    const int pair = blockIdx.x * kBlock + threadIdx.x;
    if (pair == 0) {
        P.fill[0] = 0;
        P.fill[1] = 0;
        P.ovf[2 * P.count] = 0;
        P.ovf[2 * P.count + 1] = 0;
        P.ovf[2 * P.count + 2] = 0;
    }
    if (pair >= P.count) return;
    P.ovf[2 * pair] = 0;
    P.ovf[2 * pair + 1] = 0;
    P.counts[2 * pair] = 0;
    P.counts[2 * pair + 1] = 0;
    TopkState st;
    st.n_valid = 0;
    st.k = 0;
    st.need = 0;
    st.cand = 0;
    st.key = 0;
    st.wlo = 0;
    st.whi = 0;
    st.level = -1;
    st.status = kTopkActive;
    st.d0 = 0;
    st.round = 0;
    st.sampled = 0;
    st.reserved = 0;
    if (P.sigs) level0_from_sig(P.sigs[pair], P.descs[pair], P, st);
    P.state[pair] = st;
}

// ---- a window from a sample ----------------------------------------------------
constexpr int kSampleRuns = 256;                // one run of consecutive elements per thread
constexpr int kSampleRun = 32;
constexpr int64_t kSampleMinN = int64_t(1) << 16;
constexpr int kSampleSet = 8192;                // LDS hash set of the sample's window keys
constexpr int kSampleMaxDistinct = 256;         // more distinct sampled keys in the binade: no guess

// One block per open pair of this kind (n >= 2^16): errors of 256 runs of 32
// consecutive elements spread over the pair, and the binade of the sample's
// k-th largest error as a guess of binade D0 -- unless it holds zero or
// infinite errors, or its sampled errors take more than 256 distinct values
// (the gathering pass would not fit them).  Pass A then gathers that binade
// and counts the pair's valid errors and those above it, which confirm the
// guess exactly; a wrong guess costs the binade pass and a second gathering
// pass over the pair.  A right guess gives the records of the binade-pass
// route.
template <int DG, int DT>
__global__ void __launch_bounds__(kBlock) topk_sample(TopkParams P) {
    const int pair = blockIdx.x;
    const SigDesc d = P.descs[pair];
    if (d.dtype != DG || d.tdtype != DT || d.n < kSampleMinN) return;
    TopkState st = P.state[pair];
    if (st.level != -1) return;
    __shared__ uint32_t h[kBins0];
    __shared__ uint64_t set[kSampleSet];
    __shared__ uint32_t nvalid, distinct;
    __shared__ int bs;
    for (int b = threadIdx.x; b < kBins0; b += kBlock) h[b] = 0;
    for (int i = threadIdx.x; i < kSampleSet; i += kBlock) set[i] = kEmpty;
    if (threadIdx.x == 0) {
        nvalid = 0;
        distinct = 0;
    }
    __syncthreads();
    constexpr int ESZG = Tr<DG>::W / 8, ESZT = Tr<DT>::W / 8;
    const char *g = static_cast<const char *>(d.g);
    const char *t = static_cast<const char *>(d.t);
    int64_t start = (int64_t)threadIdx.x * d.n / kSampleRuns;
    if (start > d.n - kSampleRun) start = d.n - kSampleRun;
    uint64_t keys[kSampleRun];
    uint32_t mine = 0;
#pragma unroll
    for (int i = 0; i < kSampleRun; ++i) {
        double a;
        const bool ok = error_of<DG, DT>(load_elem<DG>(g + start * ESZG, (uint32_t)i),
                                         load_elem<DT>(t + start * ESZT, (uint32_t)i), keys[i], a);
        if (!ok) keys[i] = kEmpty;
        else {
            ++mine;
            atomicAdd(&h[keys[i] >> 52], 1u);
        }
    }
    atomicAdd(&nvalid, mine);
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint64_t ks = ((uint64_t)nvalid * (uint32_t)P.num + (uint32_t)P.den - 1) / (uint32_t)P.den;
        int b = -1;
        uint64_t acc = 0;
        if (ks > 0)
            for (b = kBins0 - 1; b > 0 && acc + h[b] < ks; --b) acc += h[b];
        bs = b;
    }
    __syncthreads();
    const int b = bs;
    if (b < 1 || b > kBins0 - 2) return;                      // no sample boundary, or zero or infinite errors
    const uint64_t wlo = (uint64_t)b << 52, whi = (uint64_t)(b + 1) << 52;
    // distinct sampled keys inside the binade
#pragma unroll
    for (int i = 0; i < kSampleRun; ++i) {
        const uint64_t key = keys[i];
        if (key == kEmpty || key < wlo || key >= whi) continue;
        uint32_t slot = (uint32_t)((key * 0x9E3779B97F4A7C15ull) >> 51);   // 13 bits
#pragma unroll 1
        for (int p = 0; p < kSampleSet; ++p, slot = (slot + 1) & (kSampleSet - 1)) {
            const uint64_t old = atomicCAS((unsigned long long *)&set[slot], (unsigned long long)kEmpty,
                                           (unsigned long long)key);
            if (old == kEmpty) {
                atomicAdd(&distinct, 1u);
                break;
            }
            if (old == key) break;
        }
    }
    __syncthreads();
    if (threadIdx.x != 0 || distinct > kSampleMaxDistinct) return;
    st.wlo = wlo;
    st.whi = whi;
    st.level = -2;
    st.status = kTopkActive;
    st.sampled = 1;
    st.k = ~uint64_t(0);                                       // counted by pass A
    st.n_valid = 0;
    st.need = 0;
    st.cand = 0;
    P.state[pair] = st;
}

// ---- streaming passes over the tensors ----------------------------------------
enum { kPass1 = 0, kPassA = 1, kPassC = 2, kPassT = 3 };

// pass 1: binade histogram of the pairs whose level 0 is open (one chunk per block)
template <int DG, int DT>
__device__ __forceinline__ void pass1_chunk(const TopkParams &P, int64_t gchunk, uint32_t *h) {
    const int pair = P.chunk_pair[gchunk];
    if (P.state[pair].level != -1) return;
    const SigDesc d = P.descs[pair];
    for (int b = threadIdx.x; b < kBins0; b += kBlock) h[b] = 0;
    __syncthreads();
    for_each_error<DG, DT>(d, gchunk - d.first_chunk, [&](uint64_t key, double) { atomicAdd(&h[key >> 52], 1u); });
    flush_hist(h, kBins0, P.hist + (size_t)pair * kTopkBins);
}

// pass A (one chunk per block in round 0; round 1 serves the pairs whose
// window did not fit, after their binade pass).  Sums the errors above the
// gathered range and gathers the range: binade D0, or the pair's window.
// For binade D0 each error is counted once: in the gather table, or (once a
// key of this thread found no slot) in the digit-1 histogram; at the end the
// table's counts go into that histogram too (in LDS when the block
// overflowed, else straight to the pair's).  A window that does not fit is
// given up (the pair is gathered again by binade).
template <int DG, int DT>
__device__ __forceinline__ void passA_chunk(const TopkParams &P, int64_t gchunk, uint32_t *h, Table &tab, double *red) {
    const int pair = P.chunk_pair[gchunk];
    const TopkState st = P.state[pair];
    if (st.round != P.round) return;                          // served by the other round
    // nothing above an infinite boundary; nothing at all when k = 0
    if (st.k == 0 || (st.level >= 0 && st.d0 == kBins0 - 1)) {
        if (threadIdx.x == 0) P.part_a[gchunk] = 0.0;
        return;
    }
    const SigDesc d = P.descs[pair];
    const bool win = st.level == -2;
    const uint64_t glo = win ? st.wlo : (uint64_t)st.d0 << 52;           // the gathered keys [glo, ghi)
    const uint64_t ghi = win ? st.whi : (uint64_t)(st.d0 + 1) << 52;
    const bool active = st.status == kTopkActive;            // the range needs ordering
    const bool hist1 = active && !win;
    const bool samp = st.sampled != 0;                        // a guessed binade: count the valid errors and those above
    uint32_t nv = 0, na = 0;                                  // this lane's counts
    if (active) {
        if (hist1)
            for (int b = threadIdx.x; b < kTopkBins; b += kBlock) h[b] = 0;
        table_init(tab);
        __syncthreads();
    }
    double s = 0.0;
    bool spill = false;                                       // this thread's keys find no slot
    for_each_error_vec<DG, DT>(d, gchunk - d.first_chunk, [&](const auto &key, const auto &a, const auto &ok) {
        constexpr int V = sizeof(ok) / sizeof(ok[0]);
        bool in[V];
#pragma unroll
        for (int j = 0; j < V; ++j) {
            if (ok[j] && key[j] >= ghi) s += a[j];
            in[j] = ok[j] && key[j] >= glo && key[j] < ghi && active;
        }
        if (!spill) {
            // first probes of the vector's keys issued together; a key found
            // there is counted, others take the full probe sequence
            uint32_t slot[V];
            uint64_t cur[V];
#pragma unroll
            for (int j = 0; j < V; ++j) {
                slot[j] = table_slot(key[j]);
                cur[j] = in[j] ? __hip_atomic_load(&tab.key[slot[j]], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)
                               : kEmpty;
            }
#pragma unroll
            for (int j = 0; j < V; ++j) {
                if (!in[j]) continue;
                if (cur[j] == key[j]) {
                    atomicAdd(&tab.cnt[slot[j]], 1u);
                    in[j] = false;
                } else if (table_count(tab, key[j])) {
                    in[j] = false;
                } else {
                    spill = true;
                    tab.full = 1;
                }
            }
        }
        if (hist1) {
#pragma unroll
            for (int j = 0; j < V; ++j)
                if (in[j]) atomicAdd(&h[digit_of(key[j], 1)], 1u);
        }
        if (samp) {
#pragma unroll
            for (int j = 0; j < V; ++j) {
                nv += ok[j] ? 1u : 0u;
                na += (ok[j] && key[j] >= ghi) ? 1u : 0u;
            }
        }
    });
    if (samp) {
        // lane counts (at most 2^10 each) summed over the wave
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            nv += __shfl_xor(nv, o);
            na += __shfl_xor(na, o);
        }
        if ((threadIdx.x & 63) == 0) {
            atomicAdd((unsigned long long *)&P.counts[2 * pair], (unsigned long long)nv);
            atomicAdd((unsigned long long *)&P.counts[2 * pair + 1], (unsigned long long)na);
        }
    }
    const double bs = block_sum(s, red);
    if (threadIdx.x == 0) P.part_a[gchunk] = bs;
    if (!active) return;
    __syncthreads();
    if (hist1) {
        uint64_t *H = P.hist + (size_t)pair * kTopkBins;
        if (tab.full) {
            for (int i = threadIdx.x; i < kTable; i += kBlock)
                if (tab.cnt[i]) atomicAdd(&h[digit_of(tab.key[i], 1)], tab.cnt[i]);
            flush_hist(h, kTopkBins, H);
        } else {
            for (int i = threadIdx.x; i < kTable; i += kBlock)
                if (tab.cnt[i])
                    atomicAdd((unsigned long long *)&H[digit_of(tab.key[i], 1)], (unsigned long long)tab.cnt[i]);
        }
    }
    table_flush(tab, P, 0, pair, st.round, win);
    __syncthreads();
}

// pass C (pairs whose binade did not fit): exact sum of their errors in D0
// above bin D1 and gather of bin (D0, D1)
template <int DG, int DT>
__device__ __forceinline__ void passC_chunk(const TopkParams &P, int64_t gchunk, Table &tab) {
    const int pair = P.chunk_pair[gchunk];
    const TopkState st = P.state[pair];
    if (!(st.status == kTopkActive && st.level == 1 && P.ovf[2 * pair] != 0)) return;
    const SigDesc d = P.descs[pair];
    table_init(tab);
    __syncthreads();
    const uint64_t b1 = st.key >> digit_shift(1);           // binade and digit 1 of the boundary
    const int d0 = st.d0;
    uint64_t x = 0;
    for_each_error<DG, DT>(d, gchunk - d.first_chunk, [&](uint64_t key, double) {
        const uint64_t k1 = key >> digit_shift(1);
        if ((k1 >> 13) == (b1 >> 13) && k1 > b1) x += signif(key, d0);
        const bool in = k1 == b1;
        const bool counted = in && table_count(tab, key);
        spill_entry(in && !counted, key, P, pair, st.round);
    });
    block_add128(x, xsum_of(P, pair, d0));
    tab.full = 0;                                            // keys without a slot went out as entries
    table_flush(tab, P, 1, pair, st.round, false);
    __syncthreads();
}

// pass T_L (pairs whose bin (D0, D1) did not fit either): histogram of digit
// L (L <= 4) among the errors on the level L-1 prefix, and (L >= 3) the
// exact sum of the errors on the level L-2 prefix above digit D_{L-1}
template <int DG, int DT>
__device__ __forceinline__ void passT_chunk(const TopkParams &P, int64_t gchunk, uint32_t *h) {
    const int L = P.level;
    const int pair = P.chunk_pair[gchunk];
    const TopkState st = P.state[pair];
    const bool want = L <= kTopkLevels - 1 ? (st.status == kTopkActive && st.level == L - 1) : st.level == L - 1;
    if (!(want && P.ovf[2 * pair] != 0 && P.ovf[2 * pair + 1] != 0)) return;
    const SigDesc d = P.descs[pair];
    const bool hist = L <= kTopkLevels - 1;
    const bool sum = L >= 3;
    if (hist) {
        for (int b = threadIdx.x; b < kTopkBins; b += kBlock) h[b] = 0;
        __syncthreads();
    }
    const int sh = digit_shift(hist ? L - 1 : 0);
    const uint64_t ph = st.key >> sh;
    const int sx = digit_shift(sum ? L - 2 : 0);
    const uint64_t px = st.key >> sx;
    const uint32_t dl = digit_of(st.key, sum ? L - 1 : 0);
    const int d0 = st.d0;
    uint64_t x = 0;
    for_each_error<DG, DT>(d, gchunk - d.first_chunk, [&](uint64_t key, double) {
        if (hist && (key >> sh) == ph) atomicAdd(&h[digit_of(key, L)], 1u);
        if (sum && (key >> sx) == px && digit_of(key, L - 1) > dl) x += signif(key, d0);
    });
    if (sum) block_add128(x, xsum_of(P, pair, d0));
    if (hist) flush_hist(h, kTopkBins, P.hist + (size_t)pair * kTopkBins);
    __syncthreads();
}

template <int DG, int DT, int OP>
__global__ void __launch_bounds__(kBlock) topk_scan(TopkParams P) {
    __shared__ uint32_t h[kTopkBins];
    __shared__ double red[kWaves];
    if constexpr (OP == kPass1) {
        if (P.round == 0) {
            pass1_chunk<DG, DT>(P, P.chunk_base + blockIdx.x, h);
        } else {
            if (P.ovf[2 * P.count + 2] == 0) return;         // every window fitted
            for (int64_t c = blockIdx.x; c < P.kind_chunks; c += gridDim.x) {
                pass1_chunk<DG, DT>(P, P.chunk_base + c, h);
                __syncthreads();
            }
        }
    } else if constexpr (OP == kPassA) {
        __shared__ Table tab;
        if (P.round == 0) {
            passA_chunk<DG, DT>(P, P.chunk_base + blockIdx.x, h, tab, red);
        } else {
            if (P.ovf[2 * P.count + 2] == 0) return;         // every window fitted
            for (int64_t c = blockIdx.x; c < P.kind_chunks; c += gridDim.x)
                passA_chunk<DG, DT>(P, P.chunk_base + c, h, tab, red);
        }
    } else if constexpr (OP == kPassC) {
        __shared__ Table tab;
        if (P.ovf[2 * P.count] == 0) return;                 // every binade fitted
        for (int64_t c = blockIdx.x; c < P.kind_chunks; c += gridDim.x) passC_chunk<DG, DT>(P, P.chunk_base + c, tab);
    } else {
        if (P.ovf[2 * P.count + 1] == 0) return;             // every bin fitted
        for (int64_t c = blockIdx.x; c < P.kind_chunks; c += gridDim.x) passT_chunk<DG, DT>(P, P.chunk_base + c, h);
    }
}

// ---- selection -----------------------------------------------------------------
// Loads the pair's histogram (nb bins) into LDS and clears it for the next
// level; every thread of the block takes part.
__device__ __forceinline__ void take_hist(uint64_t *H, int nb, uint64_t *hs, uint64_t *ssum) {
    const int seg = nb / kBlock;
    for (int b = threadIdx.x; b < nb; b += kBlock) {
        hs[b] = H[b];
        H[b] = 0;
    }
    __syncthreads();
    const int top = nb - (int)threadIdx.x * seg;              // thread t: bins [top - seg, top)
    uint64_t x = 0;
    for (int b = top - 1; b >= top - seg; --b) x += hs[b];
    ssum[threadIdx.x] = x;
    __syncthreads();
}

// The bin holding the need-th largest counted error (thread 0): walks the
// segments, then the bins, from the top; acc receives the count above it.
__device__ __forceinline__ int walk_hist(const uint64_t *hs, const uint64_t *ssum, int nb, uint64_t need,
                                         uint64_t &acc) {
    const int seg = nb / kBlock;
    acc = 0;
    int t = 0;
    while (t < kBlock - 1 && acc + ssum[t] < need) acc += ssum[t++];
    int b = nb - t * seg - 1;
    while (b > nb - (t + 1) * seg && acc + hs[b] < need) acc += hs[b--];
    return b;
}

// One block per pair: the bin of the level-L histogram holding the need-th
// largest remaining error.
__global__ void __launch_bounds__(kBlock) topk_select(TopkParams P) {
    const int pair = blockIdx.x;
    const int L = P.level;
    TopkState st = P.state[pair];
    if (L == 0 ? st.level != -1 : !(st.status == kTopkActive && st.level == L - 1)) return;
    const int nb = L == 0 ? kBins0 : kTopkBins;
    __shared__ uint64_t hs[kTopkBins];
    __shared__ uint64_t ssum[kBlock];
    take_hist(P.hist + (size_t)pair * kTopkBins, nb, hs, ssum);
    if (threadIdx.x != 0) return;
    uint64_t need;
    if (L == 0) {
        uint64_t nv = 0;
        for (int t = 0; t < kBlock; ++t) nv += ssum[t];
        st.n_valid = nv;
        st.k = (uint64_t)(((unsigned __int128)nv * (uint32_t)P.num + (uint32_t)P.den - 1) / (uint32_t)P.den);
        st.need = st.k;
        st.cand = 0;
        st.key = 0;
        if (st.k == 0) {
            st.level = 0;
            st.status = kTopkDone;
            st.d0 = 0;
            P.state[pair] = st;
            return;
        }
        need = st.k;
    } else {
        need = st.need;
    }
    uint64_t acc;
    const int b = walk_hist(hs, ssum, nb, need, acc);
    st.need = need - acc;                     // copies of the boundary bin taken, >= 1
    st.cand = hs[b];
    st.key |= (uint64_t)b << digit_shift(L);
    if (L == 0) {
        level0_status(st, b, P.descs[pair].tdtype);
    } else {
        st.level = L;
        st.status = L == kTopkLevels - 1 ? kTopkDone : kTopkActive;
    }
    P.state[pair] = st;
}

// One block per pair whose window was gathered: level 0 from the binade
// histogram of its entries (need counts from the top of the window; for a
// guess, from pass A's counts, which also confirm it).  A window that did
// not fit, or a wrong guess, reopens level 0 for a binade pass and a second
// gathering round.
__global__ void __launch_bounds__(kBlock) topk_select_window(TopkParams P) {
    const int pair = blockIdx.x;
    TopkState st = P.state[pair];
    if (st.level != -2) return;
    if (P.ovf[2 * pair] != 0) {
        if (threadIdx.x == 0) {
            st.level = -1;
            st.round = 1;
            st.wlo = st.whi = 0;
            st.need = st.cand = 0;
            st.sampled = 0;
            P.ovf[2 * pair] = 0;
            P.state[pair] = st;
        }
        return;
    }
    __shared__ uint64_t hs[kBins0];
    __shared__ uint64_t ssum[kBlock];
    take_hist(P.hist + (size_t)pair * kTopkBins, kBins0, hs, ssum);
    if (threadIdx.x != 0) return;
    if (st.sampled) {
        // the pair's counts decide whether the guessed binade holds the
        // boundary; otherwise level 0 reopens for a binade pass (round 1)
        const uint64_t nv = P.counts[2 * pair], above = P.counts[2 * pair + 1];
        uint64_t w = 0;
        for (int t = 0; t < kBlock; ++t) w += ssum[t];
        st.n_valid = nv;
        st.k = (uint64_t)(((unsigned __int128)nv * (uint32_t)P.num + (uint32_t)P.den - 1) / (uint32_t)P.den);
        if (st.k == 0) {
            st.level = 0;
            st.status = kTopkDone;
            st.d0 = 0;
            P.state[pair] = st;
            return;
        }
        if (st.k <= above || st.k > above + w) {
            st.level = -1;
            st.round = 1;
            st.wlo = st.whi = 0;
            st.need = st.cand = 0;
            st.sampled = 0;
            P.ovf[2 * P.count + 2] = 1;
            P.state[pair] = st;
            return;
        }
        st.need = st.k - above;
    }
    uint64_t acc;
    const int b = walk_hist(hs, ssum, kBins0, st.need, acc);
    st.need -= acc;
    st.cand = hs[b];
    st.key = (uint64_t)b << 52;
    level0_status(st, b, P.descs[pair].tdtype);
    P.state[pair] = st;
}

// ---- rounds on the entries -------------------------------------------------------
// Region 0 holds the binade and window gathers of pass A, region 1 the bin
// gathers of pass C; an entry counts for its pair when the pair takes that
// route and the entry comes from the pair's gathering round.
template <typename F>
__device__ __forceinline__ void for_each_entry(const TopkParams &P, F &&f) {
    for (int r = 0; r < 2; ++r) {
        const unsigned long long fill = P.fill[r];
        const uint64_t n = fill < P.cap[r] ? fill : P.cap[r];
        const TopkEntry *E = P.ents + (r ? P.cap[0] : 0);
        for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (uint64_t)gridDim.x * kBlock) {
            const TopkEntry e = E[i];
            if (e.pair < 0) continue;
            const int pair = (int)((uint32_t)e.pair & kPairMask);
            if (pair >= P.count) continue;
            if (pair_mode(P, pair) != (r ? kModeC : kModeA)) continue;
            const TopkState &st = P.state[pair];
            if ((int)((uint32_t)e.pair >> 30) != st.round) continue;
            f(e, pair, st);
        }
    }
}

// Level L: weighted histogram of digit L over the entries on the pair's
// level L-1 prefix.  Level 0 serves the window pairs (every entry is in the
// window), level 1 the window pairs only (the others got their digit-1
// histogram from pass A), levels 2-4 every pair on entries.
__global__ void __launch_bounds__(kBlock) topk_ent_hist(TopkParams P) {
    const int L = P.level;
    for_each_entry(P, [&](const TopkEntry &e, int pair, const TopkState &st) {
        if (L == 0) {
            if (st.level != -2) return;
        } else {
            if (!(st.status == kTopkActive && st.level == L - 1)) return;
            if (L == 1 && !is_window(st)) return;
            const int sh = digit_shift(L - 1);
            if ((e.key >> sh) != (st.key >> sh)) return;
        }
        atomicAdd((unsigned long long *)&P.hist[(size_t)pair * kTopkBins + digit_of(e.key, L)],
                  (unsigned long long)e.count);
    });
}

// Exact sums of the entries above the fixed boundary, per binade.
__global__ void __launch_bounds__(kBlock) topk_ent_sum(TopkParams P) {
    for_each_entry(P, [&](const TopkEntry &e, int pair, const TopkState &st) {
        if (st.level != kTopkLevels - 1 || e.key <= st.key) return;
        const int b = (int)(e.key >> 52);
        const unsigned __int128 v = (unsigned __int128)e.count * signif(e.key, b);
        atomic_add128(xsum_of(P, pair, b), (uint64_t)v, (uint64_t)(v >> 64));
    });
}

// ---- records -------------------------------------------------------------------
// Fixed-order sum over the pair's chunk partials (thread t sums chunks t,
// t + 256, ... in order; then butterflies and waves in order).
__device__ __forceinline__ double chunk_sum(const double *part, int64_t first, int64_t n, double *red) {
    double s = 0.0;
    for (int64_t c = threadIdx.x; c < n; c += kBlock) s += part[first + c];
    const double r = block_sum(s, red);
    __syncthreads();
    return r;
}

// The binary64 value of an exact significand sum of binade b (the boundary's
// binade with need copies of T added).
__device__ __forceinline__ double binade_value(const TopkParams &P, int pair, const TopkState &st, int b) {
    const uint64_t *xp = xsum_of(P, pair, b);
    unsigned __int128 x = ((unsigned __int128)xp[1] << 64) | xp[0];
    if (b == st.d0) x += (unsigned __int128)st.need * signif(st.key, st.d0);
    if (x == 0) return 0.0;
    const double xd = (double)(uint64_t)(x >> 64) * 0x1p64 + (double)(uint64_t)x;
    return __builtin_ldexp(xd, (b != 0 ? b : 1) - 1075);
}

__global__ void __launch_bounds__(kBlock) topk_finalize(TopkParams P) {
    __shared__ double red[kWaves];
    __shared__ double xb[kBins0];
    const int pair = blockIdx.x;
    const SigDesc d = P.descs[pair];
    const TopkState st = P.state[pair];
    const double sa = chunk_sum(P.part_a, d.first_chunk, d.nchunks, red);
    // a window's binades above D0: their exact sums converted in parallel,
    // added in a fixed order (from the top) below
    const bool ordinary = st.k != 0 && st.d0 != kBins0 - 1 && !(st.d0 == 0 && st.level == 0);
    const int top = ordinary && is_window(st) ? (int)((st.whi - 1) >> 52) : st.d0;
    if (ordinary && top > st.d0) {
        for (int b = st.d0 + threadIdx.x; b <= top; b += kBlock) xb[b] = binade_value(P, pair, st, b);
        __syncthreads();
    }
    if (threadIdx.x != 0) return;
    const double qnan = opaque_double(0x7FF80000u, 0u);
    const double inf = opaque_double(0x7FF00000u, 0u);
    peat_topk_t o;
    o.n_valid = (int64_t)st.n_valid;
    o.k = (int64_t)st.k;
    if (st.k == 0) {
        o.count_above = 0;
        o.kth_value = qnan;
        o.sum_topk = 0.0;
        o.mean_topk = qnan;
    } else if (st.d0 == kBins0 - 1) {                 // the k-th largest error is infinite
        o.count_above = (int64_t)(st.k - st.need);
        o.kth_value = inf;
        o.sum_topk = inf;
        o.mean_topk = inf;
    } else if (!ordinary) {                           // the k-th largest error is 0
        o.count_above = (int64_t)(st.k - st.need);
        o.kth_value = 0.0;
        o.sum_topk = sa;
        o.mean_topk = sa / (double)st.k;
    } else {
        // exact sums: binade D0 (everything above T, then need copies of T)
        // and, for a window, each binade above it
        double sc;
        if (top > st.d0) {
            sc = 0.0;
            for (int b = top; b >= st.d0; --b) sc += xb[b];
        } else {
            sc = binade_value(P, pair, st, st.d0);
        }
        o.count_above = (int64_t)(st.k - st.need);
        o.kth_value = __longlong_as_double((long long)st.key);
        o.sum_topk = sa + sc;
        o.mean_topk = o.sum_topk / (double)st.k;
    }
    P.outs[pair] = o;
}

__global__ void __launch_bounds__(kBlock) topk_zero(uint64_t *p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlock) p[i] = 0;
}

// ---- launches ---------------------------------------------------------------------
template <int DG, int DT, int OP>
void launch_one(const TopkParams &q, hipStream_t s) {
    const int64_t n = q.kind_chunks;
    const bool full = (OP == kPass1 || OP == kPassA) && q.round == 0;   // one chunk per block
    const int64_t grid = full ? n : (n < kScanGrid ? n : kScanGrid);
    hipLaunchKernelGGL((topk_scan<DG, DT, OP>), dim3((unsigned)grid), dim3(kBlock), 0, s, q);
}

template <int OP>
hipError_t launch_scan(const TopkParams &p, const int64_t range[kKinds + 1], hipStream_t s) {
    static_assert(kKindTypes[3][1] == PEAT_F64 && kKindTypes[9][0] == PEAT_BF16, "kind table order");
    for (int kind = 0; kind < kKinds; ++kind) {
        const int64_t n = range[kind + 1] - range[kind];
        if (n <= 0) continue;
        TopkParams q = p;
        q.chunk_base = range[kind];
        q.kind_chunks = n;
        switch (kind) {
            case 0: launch_one<PEAT_F32, PEAT_F32, OP>(q, s); break;
            case 1: launch_one<PEAT_F16, PEAT_F16, OP>(q, s); break;
            case 2: launch_one<PEAT_BF16, PEAT_BF16, OP>(q, s); break;
            case 3: launch_one<PEAT_F32, PEAT_F64, OP>(q, s); break;
            case 4: launch_one<PEAT_F32, PEAT_F16, OP>(q, s); break;
            case 5: launch_one<PEAT_F32, PEAT_BF16, OP>(q, s); break;
            case 6: launch_one<PEAT_F16, PEAT_F32, OP>(q, s); break;
            case 7: launch_one<PEAT_BF16, PEAT_F32, OP>(q, s); break;
            case 8: launch_one<PEAT_F16, PEAT_F64, OP>(q, s); break;
            default: launch_one<PEAT_BF16, PEAT_F64, OP>(q, s); break;
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// The sample kernel of every kind present (one block per pair; blocks of
// other kinds' pairs return at once).
hipError_t launch_sample(const TopkParams &p, const int64_t range[kKinds + 1], hipStream_t s) {
    for (int kind = 0; kind < kKinds; ++kind) {
        if (range[kind + 1] - range[kind] <= 0) continue;
        const dim3 grid((unsigned)p.count), block(kBlock);
        switch (kind) {
            case 0: hipLaunchKernelGGL((topk_sample<PEAT_F32, PEAT_F32>), grid, block, 0, s, p); break;
            case 1: hipLaunchKernelGGL((topk_sample<PEAT_F16, PEAT_F16>), grid, block, 0, s, p); break;
            case 2: hipLaunchKernelGGL((topk_sample<PEAT_BF16, PEAT_BF16>), grid, block, 0, s, p); break;
            case 3: hipLaunchKernelGGL((topk_sample<PEAT_F32, PEAT_F64>), grid, block, 0, s, p); break;
            case 4: hipLaunchKernelGGL((topk_sample<PEAT_F32, PEAT_F16>), grid, block, 0, s, p); break;
            case 5: hipLaunchKernelGGL((topk_sample<PEAT_F32, PEAT_BF16>), grid, block, 0, s, p); break;
            case 6: hipLaunchKernelGGL((topk_sample<PEAT_F16, PEAT_F32>), grid, block, 0, s, p); break;
            case 7: hipLaunchKernelGGL((topk_sample<PEAT_BF16, PEAT_F32>), grid, block, 0, s, p); break;
            case 8: hipLaunchKernelGGL((topk_sample<PEAT_F16, PEAT_F64>), grid, block, 0, s, p); break;
            default: hipLaunchKernelGGL((topk_sample<PEAT_BF16, PEAT_F64>), grid, block, 0, s, p); break;
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_select(const TopkParams &p, int level, hipStream_t s) {
    TopkParams q = p;
    q.level = level;
    hipLaunchKernelGGL(topk_select, dim3((unsigned)p.count), dim3(kBlock), 0, s, q);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_topk_level0(const TopkParams &p, const int64_t range[kKinds + 1], hipStream_t s) {
    if (p.count <= 0) return hipSuccess;
    hipError_t e;
    auto zero = [&](uint64_t *x, int64_t n) {
        const int64_t zb = (n + kBlock - 1) / kBlock;
        hipLaunchKernelGGL(topk_zero, dim3((unsigned)(zb < 65536 ? zb : 65536)), dim3(kBlock), 0, s, x, n);
    };
    zero(p.hist, (int64_t)kTopkBins * p.count);
    zero(p.xsum, (int64_t)2 * kBins0 * p.count);
    hipLaunchKernelGGL(topk_init, dim3((unsigned)((p.count + kBlock - 1) / kBlock)), dim3(kBlock), 0, s, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_sample(p, range, s)) != hipSuccess) return e;
    TopkParams q = p;
    q.round = 0;
    if ((e = launch_scan<kPass1>(q, range, s)) != hipSuccess) return e;
    return launch_select(q, 0, s);
}

hipError_t launch_topk_rest(const TopkParams &p, const int64_t range[kKinds + 1], hipStream_t s) {
    if (p.count <= 0) return hipSuccess;
    hipError_t e;
    TopkParams q = p;
    auto ent_hist = [&](int L) {
        q.level = L;
        hipLaunchKernelGGL(topk_ent_hist, dim3(kEntGrid), dim3(kBlock), 0, s, q);
        return hipGetLastError();
    };
    // round 0: binade D0 or the window; level 0 of the windows from their entries
    q.round = 0;
    if ((e = launch_scan<kPassA>(q, range, s)) != hipSuccess) return e;
    if ((e = ent_hist(0)) != hipSuccess) return e;
    hipLaunchKernelGGL(topk_select_window, dim3((unsigned)p.count), dim3(kBlock), 0, s, q);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // round 1: windows that did not fit and wrong guesses take the binade pass and are gathered again
    q.round = 1;
    if ((e = launch_scan<kPass1>(q, range, s)) != hipSuccess) return e;
    if ((e = launch_select(q, 0, s)) != hipSuccess) return e;
    if ((e = launch_scan<kPassA>(q, range, s)) != hipSuccess) return e;
    q.round = 0;
    // level 1 (the windows from their entries), the bin gathers, levels 2-4
    if ((e = ent_hist(1)) != hipSuccess) return e;
    if ((e = launch_select(q, 1, s)) != hipSuccess) return e;
    if ((e = launch_scan<kPassC>(q, range, s)) != hipSuccess) return e;
    for (int L = 2; L <= kTopkLevels - 1; ++L) {
        if ((e = ent_hist(L)) != hipSuccess) return e;
        q.level = L;
        if ((e = launch_scan<kPassT>(q, range, s)) != hipSuccess) return e;
        if ((e = launch_select(q, L, s)) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(topk_ent_sum, dim3(kEntGrid), dim3(kBlock), 0, s, q);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    q.level = kTopkLevels;
    if ((e = launch_scan<kPassT>(q, range, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(topk_finalize, dim3((unsigned)p.count), dim3(kBlock), 0, s, q);
    return hipGetLastError();
}

}  // namespace peat
