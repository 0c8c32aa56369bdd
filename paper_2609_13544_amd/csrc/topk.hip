// Mean of the k largest errors of each pair (the "mean of the top 10%
// errors" score of Section IV-B.3, the Analyzer's main score in Section IV-C),
// by exact radix selection on the binary64 bit pattern of the error, which is
// monotone for a >= 0:
//
//   pass 1   histogram of digit 0 (bits 62..52, the binade) over the pair;
//   select   the binade D0 holding the k-th largest error;
//   pass 2   binary64 sum of the errors above binade D0; histogram of digit 1
//            (bits 51..39) of the errors inside it;
//   select   the level-1 bin D1;
//   pass 3   binary64 sum of the errors in binade D0 above bin D1; the errors
//            of bin (D0, D1) are gathered as (key, count) entries: each block
//            counts its distinct keys in an LDS hash table (errors of
//            checkpoint-like data are small multiples of the golden's ULP,
//            so the boundary bin is mostly ties) and appends one entry per
//            key; keys that do not fit the table become entries of count 1;
//   rounds   digits 2-4 (13 bits each) on the entries: weighted histogram,
//            select, exact integer sum count * significand of the entries
//            above the boundary (they share the exponent D0), copy of the
//            entries on it;
//   finalize sum = (pass 2 + pass 3) + exact candidate sums + need * T.
//
// Given the pair's error signature with one-binade histogram bins (the same
// errors over the same valid pairs), the host resolves level 0 from that
// histogram whenever the k-th largest error falls in a regular bin, and
// pass 1 and the level-0 selection skip the pair.
//
// The k-th largest error T is the key with all five digits fixed; count_above
// is k minus the copies of T taken.  Passes 2 and 3 sum in a fixed
// per-lane / butterfly / wave order over chunks whose size depends only on
// n, and the candidate sums are exact integers, so the
// result does not depend on the order in which candidates are copied.
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
constexpr int kTable = 512;                     // LDS hash table of pass 3 (keys per block)
constexpr int kProbes = 8;
constexpr uint64_t kEmpty = ~uint64_t(0);       // never a key: errors have the sign bit clear

__device__ __forceinline__ int digit_shift(int level) { return level == 0 ? 52 : 52 - 13 * level; }

__device__ __forceinline__ uint32_t digit_of(uint64_t key, int level) {
    if (level == 0) return (uint32_t)(key >> 52);               // sign bit is 0
    return (uint32_t)(key >> digit_shift(level)) & (kTopkBins - 1);
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

// Adds the block's LDS histogram to the pair's device histogram.
__device__ __forceinline__ void flush_hist(const uint32_t *h, int nb, uint64_t *H) {
    __syncthreads();
    for (int b = threadIdx.x; b < nb; b += kBlock)
        if (h[b]) atomicAdd((unsigned long long *)&H[b], (unsigned long long)h[b]);
}

// Appends the entry (key, count) to a pair's entry buffer (two words per
// entry), one atomic per wave.
__device__ __forceinline__ void append_entry(bool take, uint64_t key, uint64_t count, uint64_t *cnt,
                                             uint64_t *dst) {
    const uint64_t m = __ballot(take);
    if (m == 0) return;
    const int leader = __ffsll((long long)m) - 1;
    uint64_t base = 0;
    if ((int)(threadIdx.x & 63) == leader) base = atomicAdd((unsigned long long *)cnt, (unsigned long long)__popcll(m));
    base = __shfl(base, leader);
    if (take) {
        const uint32_t rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        dst[2 * (base + rank)] = key;
        dst[2 * (base + rank) + 1] = count;
    }
}

// Counts key in the block's LDS table (open addressing); false when its
// probe sequence is full of other keys.
__device__ __forceinline__ bool table_count(uint64_t *tkey, uint32_t *tcnt, uint64_t key) {
    const uint32_t h = (uint32_t)((key * 0x9E3779B97F4A7C15ull) >> 55);    // 9 bits
#pragma unroll 1
    for (int p = 0; p < kProbes; ++p) {
        const uint32_t slot = (h + p) & (kTable - 1);
        const uint64_t old = atomicCAS((unsigned long long *)&tkey[slot], (unsigned long long)kEmpty,
                                       (unsigned long long)key);
        if (old == kEmpty || old == key) {
            atomicAdd(&tcnt[slot], 1u);
            return true;
        }
    }
    return false;
}

template <int DG, int DT, int PASS>
__global__ void __launch_bounds__(kBlock) topk_pass(TopkParams P) {
    __shared__ uint32_t h[kTopkBins];
    __shared__ double red[kWaves];
    const int64_t gchunk = P.chunk_base + blockIdx.x;
    const int pair = P.chunk_pair[gchunk];
    const SigDesc d = P.descs[pair];
    const int64_t cin = gchunk - d.first_chunk;
    uint64_t *H = P.hist + (size_t)pair * kTopkBins;

    if constexpr (PASS == 0) {
        if (P.skip0 && P.skip0[pair]) return;                 // level 0 already resolved
        for (int b = threadIdx.x; b < kBins0; b += kBlock) h[b] = 0;
        __syncthreads();
        for_each_error<DG, DT>(d, cin, [&](uint64_t key, double) { atomicAdd(&h[key >> 52], 1u); });
        flush_hist(h, kBins0, H);
    } else if constexpr (PASS == 1) {
        const TopkState st = P.state[pair];
        // nothing above an infinite boundary; nothing at all when k = 0
        if (st.k == 0 || st.d0 == kBins0 - 1) {
            if (threadIdx.x == 0) P.part_a[gchunk] = 0.0;
            return;
        }
        const uint64_t d0 = (uint64_t)st.d0;
        const bool hist1 = st.status == kTopkActive;          // the boundary binade needs ordering
        if (hist1) {
            for (int b = threadIdx.x; b < kTopkBins; b += kBlock) h[b] = 0;
            __syncthreads();
        }
        double s = 0.0;
        for_each_error<DG, DT>(d, cin, [&](uint64_t key, double a) {
            const uint64_t e = key >> 52;
            if (e > d0) {
                s += a;
            } else if (e == d0 && hist1) {
                atomicAdd(&h[digit_of(key, 1)], 1u);
            }
        });
        const double bs = block_sum(s, red);
        if (threadIdx.x == 0) P.part_a[gchunk] = bs;
        if (hist1) flush_hist(h, kTopkBins, H);
    } else {
        __shared__ uint64_t tkey[kTable];
        __shared__ uint32_t tcnt[kTable];
        const TopkState st = P.state[pair];
        if (st.level < 1) {
            if (threadIdx.x == 0) P.part_b[gchunk] = 0.0;
            return;
        }
        for (int i = threadIdx.x; i < kTable; i += kBlock) {
            tkey[i] = kEmpty;
            tcnt[i] = 0;
        }
        __syncthreads();
        const uint64_t b1 = st.key >> digit_shift(1);        // binade and digit 1 of the boundary
        const uint64_t off = P.cand[pair].off;
        uint64_t *cnt = &P.state[pair].cnt[0];
        uint64_t *dst = P.keys[0] + 2 * off;
        double s = 0.0;
        for_each_error<DG, DT>(d, cin, [&](uint64_t key, double a) {
            const uint64_t k1 = key >> digit_shift(1);
            if ((k1 >> 13) == (b1 >> 13) && k1 > b1) s += a;
            const bool in = k1 == b1;
            const bool counted = in && table_count(tkey, tcnt, key);
            append_entry(in && !counted, key, 1, cnt, dst);
        });
        const double bs = block_sum(s, red);
        if (threadIdx.x == 0) P.part_b[gchunk] = bs;
        __syncthreads();
        for (int i0 = 0; i0 < kTable; i0 += kBlock) {
            const int i = i0 + (int)threadIdx.x;
            append_entry(tcnt[i] != 0, tkey[i], tcnt[i], cnt, dst);
        }
    }
}

// One block per pair: the bin of the level-`level` histogram holding the
// need-th largest remaining error.
__global__ void __launch_bounds__(kBlock) topk_select(TopkParams P) {
    const int pair = blockIdx.x;
    const int L = P.level;
    if (L == 0 && P.skip0 && P.skip0[pair]) return;           // state written by the host
    TopkState st = P.state[pair];
    if (L > 0 && !(st.status == kTopkActive && st.level == L - 1)) return;
    const int nb = L == 0 ? kBins0 : kTopkBins;
    const int seg = nb / kBlock;
    const uint64_t *H = P.hist + (size_t)pair * kTopkBins;
    __shared__ uint64_t ssum[kBlock];
    {
        const int top = nb - (int)threadIdx.x * seg;          // thread t: bins [top - seg, top)
        uint64_t x = 0;
        for (int b = top - 1; b >= top - seg; --b) x += H[b];
        ssum[threadIdx.x] = x;
    }
    __syncthreads();
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
        st.cnt[0] = st.cnt[1] = 0;
        st.level = 0;
        st.d0 = 0;
        if (st.k == 0) {
            st.status = kTopkDone;
            P.state[pair] = st;
            return;
        }
        need = st.k;
    } else {
        need = st.need;
    }
    // walk the segments, then the bins, from the top
    uint64_t acc = 0;
    int t = 0;
    while (t < kBlock - 1 && acc + ssum[t] < need) acc += ssum[t++];
    int b = nb - t * seg - 1;
    while (b > nb - (t + 1) * seg && acc + H[b] < need) acc += H[b--];
    st.need = need - acc;                     // copies of the boundary bin taken, >= 1
    st.cand = H[b];
    st.key |= (uint64_t)b << digit_shift(L);
    st.level = L;
    if (L == 0) {
        st.d0 = b;
        // An infinite boundary fixes the k-th largest error already, and so
        // does binade 0 when it holds only zero errors: with a binary64 test
        // side it also holds the subnormal errors, which the next levels
        // order like any other binade.
        const bool zero_only = b == 0 && P.descs[pair].tdtype != PEAT_F64;
        st.status = (zero_only || b == kBins0 - 1) ? kTopkDone : kTopkActive;
    } else {
        st.status = L == kTopkLevels - 1 ? kTopkDone : kTopkActive;
    }
    // the buffer the next copy fills starts empty
    if (L == 1) st.cnt[0] = 0;
    if (L >= 2) st.cnt[(L - 1) & 1] = 0;
    P.state[pair] = st;
}

// Candidate rounds (levels 2-4): keys[(L - 2) & 1] holds the (key, count)
// entries of the pair's current boundary bin.
__global__ void __launch_bounds__(kBlock) topk_cand_hist(TopkParams P) {
    __shared__ unsigned long long h[kTopkBins];
    const int L = P.level;
    const int pair = P.cblk_pair[blockIdx.x];
    const TopkState st = P.state[pair];
    if (!(st.status == kTopkActive && st.level == L - 1)) return;
    const int src = (L - 2) & 1;
    const uint64_t n = st.cnt[src];
    const uint64_t lo = (uint64_t)(blockIdx.x - P.cand[pair].first_blk) * kTopkCandBlock;
    if (lo >= n) return;
    const uint64_t hi = n - lo < (uint64_t)kTopkCandBlock ? n : lo + kTopkCandBlock;
    for (int b = threadIdx.x; b < kTopkBins; b += kBlock) h[b] = 0;
    __syncthreads();
    const uint64_t *e = P.keys[src] + 2 * P.cand[pair].off;
    for (uint64_t i = lo + threadIdx.x; i < hi; i += kBlock)
        atomicAdd(&h[digit_of(e[2 * i], L)], (unsigned long long)e[2 * i + 1]);
    __syncthreads();
    uint64_t *H = P.hist + (size_t)pair * kTopkBins;
    for (int b = threadIdx.x; b < kTopkBins; b += kBlock)
        if (h[b]) atomicAdd((unsigned long long *)&H[b], h[b]);
}

// Exact sum of the entries above the level-L boundary (count * significand,
// all with exponent field d0) and copy of the entries on it.  Writes the
// block's 128-bit sum for every block, zero when it has nothing to do.
__global__ void __launch_bounds__(kBlock) topk_cand_sum(TopkParams P) {
    __shared__ uint64_t red[kWaves][2];
    const int L = P.level;
    const int pair = P.cblk_pair[blockIdx.x];
    const TopkState st = P.state[pair];
    unsigned __int128 acc = 0;
    if (st.level == L) {
        const int src = (L - 2) & 1, dst = src ^ 1;
        const uint64_t n = st.cnt[src];
        const uint64_t lo = (uint64_t)(blockIdx.x - P.cand[pair].first_blk) * kTopkCandBlock;
        const uint64_t hi = lo >= n ? lo : (n - lo < (uint64_t)kTopkCandBlock ? n : lo + kTopkCandBlock);
        const uint32_t D = digit_of(st.key, L);
        const uint64_t lead = st.d0 != 0 ? (uint64_t(1) << 52) : 0;   // implicit bit
        const uint64_t *e = P.keys[src] + 2 * P.cand[pair].off;
        uint64_t *out = P.keys[dst] + 2 * P.cand[pair].off;
        uint64_t *cnt = &P.state[pair].cnt[dst];
        for (uint64_t i0 = lo; i0 < hi; i0 += kBlock) {
            const uint64_t i = i0 + threadIdx.x;
            const bool in = i < hi;
            const uint64_t key = in ? e[2 * i] : 0, c = in ? e[2 * i + 1] : 0;
            const uint32_t dg = digit_of(key, L);
            if (in && dg > D) acc += (unsigned __int128)c * ((key & kMant) | lead);
            if (L < kTopkLevels - 1) append_entry(in && dg == D, key, c, cnt, out);
        }
    }
    uint64_t lo_sum = (uint64_t)acc, hi_sum = (uint64_t)(acc >> 64);
    // 128-bit block sum (integer: any order)
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const uint64_t ol = __shfl_xor(lo_sum, o), oh = __shfl_xor(hi_sum, o);
        const uint64_t s = lo_sum + ol;
        hi_sum += oh + (s < lo_sum);
        lo_sum = s;
    }
    if ((threadIdx.x & 63) == 0) {
        red[threadIdx.x >> 6][0] = lo_sum;
        red[threadIdx.x >> 6][1] = hi_sum;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t l = 0, h = 0;
        for (int w = 0; w < kWaves; ++w) {
            const uint64_t s = l + red[w][0];
            h += red[w][1] + (s < l);
            l = s;
        }
        uint64_t *x = P.xpart + 2 * ((size_t)(L - 2) * P.ncblk + blockIdx.x);
        x[0] = l;
        x[1] = h;
    }
}

// Fixed-order sum over the pair's chunk partials (thread t sums chunks t,
// t + 256, ... in order; then butterflies and waves in order).
__device__ __forceinline__ double chunk_sum(const double *part, int64_t first, int64_t n, double *red) {
    double s = 0.0;
    for (int64_t c = threadIdx.x; c < n; c += kBlock) s += part[first + c];
    const double r = block_sum(s, red);
    __syncthreads();
    return r;
}

__global__ void __launch_bounds__(kBlock) topk_finalize(TopkParams P) {
    __shared__ double red[kWaves];
    const int pair = blockIdx.x;
    const SigDesc d = P.descs[pair];
    const TopkState st = P.state[pair];
    const double sa = chunk_sum(P.part_a, d.first_chunk, d.nchunks, red);
    const double sb = chunk_sum(P.part_b, d.first_chunk, d.nchunks, red);
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
    } else if (st.d0 == 0 && st.level == 0) {        // the k-th largest error is 0
        o.count_above = (int64_t)(st.k - st.need);
        o.kth_value = 0.0;
        o.sum_topk = sa;
        o.mean_topk = sa / (double)st.k;
    } else {
        // exact sum of the candidate parts: rounds 2-4, then need copies of T
        unsigned __int128 x = 0;
        const TopkCand c = P.cand[pair];
        for (int r = 0; r < kTopkLevels - 2; ++r)
            for (int b = 0; b < c.nblk; ++b) {
                const uint64_t *xp = P.xpart + 2 * ((size_t)r * P.ncblk + c.first_blk + b);
                x += ((unsigned __int128)xp[1] << 64) | xp[0];
            }
        // binade 0 (subnormal errors) has no implicit bit and the exponent of binade 1
        const uint64_t lead = st.d0 != 0 ? (uint64_t(1) << 52) : 0;
        x += (unsigned __int128)st.need * ((st.key & kMant) | lead);
        const double xd = (double)(uint64_t)(x >> 64) * 0x1p64 + (double)(uint64_t)x;
        const double sc = __builtin_ldexp(xd, (st.d0 != 0 ? st.d0 : 1) - 1075);
        o.count_above = (int64_t)(st.k - st.need);
        o.kth_value = __longlong_as_double((long long)st.key);
        o.sum_topk = (sa + sb) + sc;
        o.mean_topk = o.sum_topk / (double)st.k;
    }
    P.outs[pair] = o;
}

__global__ void __launch_bounds__(kBlock) topk_zero(uint64_t *p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kBlock) p[i] = 0;
}

template <int DG, int DT, int PASS>
void launch_one(const TopkParams &q, int64_t n, hipStream_t s) {
    hipLaunchKernelGGL((topk_pass<DG, DT, PASS>), dim3((unsigned)n), dim3(kBlock), 0, s, q);
}

template <int PASS>
hipError_t launch_pass_kinds(const TopkParams &p, const int64_t range[kKinds + 1], hipStream_t s) {
    static_assert(kKindTypes[3][1] == PEAT_F64 && kKindTypes[9][0] == PEAT_BF16, "kind table order");
    for (int kind = 0; kind < kKinds; ++kind) {
        const int64_t n = range[kind + 1] - range[kind];
        if (n <= 0) continue;
        TopkParams q = p;
        q.chunk_base = range[kind];
        switch (kind) {
            case 0: launch_one<PEAT_F32, PEAT_F32, PASS>(q, n, s); break;
            case 1: launch_one<PEAT_F16, PEAT_F16, PASS>(q, n, s); break;
            case 2: launch_one<PEAT_BF16, PEAT_BF16, PASS>(q, n, s); break;
            case 3: launch_one<PEAT_F32, PEAT_F64, PASS>(q, n, s); break;
            case 4: launch_one<PEAT_F32, PEAT_F16, PASS>(q, n, s); break;
            case 5: launch_one<PEAT_F32, PEAT_BF16, PASS>(q, n, s); break;
            case 6: launch_one<PEAT_F16, PEAT_F32, PASS>(q, n, s); break;
            case 7: launch_one<PEAT_BF16, PEAT_F32, PASS>(q, n, s); break;
            case 8: launch_one<PEAT_F16, PEAT_F64, PASS>(q, n, s); break;
            default: launch_one<PEAT_BF16, PEAT_F64, PASS>(q, n, s); break;
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace

hipError_t launch_topk_zero(uint64_t *p, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const int64_t blocks = (n + kBlock - 1) / kBlock;
    hipLaunchKernelGGL(topk_zero, dim3((unsigned)(blocks < 65536 ? blocks : 65536)), dim3(kBlock), 0, s, p, n);
    return hipGetLastError();
}

hipError_t launch_topk_pass(const TopkParams &p, int pass, const int64_t range[kKinds + 1], hipStream_t s) {
    if (pass == 0) return launch_pass_kinds<0>(p, range, s);
    if (pass == 1) return launch_pass_kinds<1>(p, range, s);
    return launch_pass_kinds<2>(p, range, s);
}

hipError_t launch_topk_select(const TopkParams &p, int level, hipStream_t s) {
    if (p.count <= 0) return hipSuccess;
    TopkParams q = p;
    q.level = level;
    hipLaunchKernelGGL(topk_select, dim3((unsigned)p.count), dim3(kBlock), 0, s, q);
    return hipGetLastError();
}

hipError_t launch_topk_cand_hist(const TopkParams &p, int level, hipStream_t s) {
    if (p.ncblk <= 0) return hipSuccess;
    TopkParams q = p;
    q.level = level;
    hipLaunchKernelGGL(topk_cand_hist, dim3((unsigned)p.ncblk), dim3(kBlock), 0, s, q);
    return hipGetLastError();
}

hipError_t launch_topk_cand_sum(const TopkParams &p, int level, hipStream_t s) {
    if (p.ncblk <= 0) return hipSuccess;
    TopkParams q = p;
    q.level = level;
    hipLaunchKernelGGL(topk_cand_sum, dim3((unsigned)p.ncblk), dim3(kBlock), 0, s, q);
    return hipGetLastError();
}

hipError_t launch_topk_finalize(const TopkParams &p, hipStream_t s) {
    if (p.count <= 0) return hipSuccess;
    hipLaunchKernelGGL(topk_finalize, dim3((unsigned)p.count), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

}  // namespace peat
