// Error-signature kernels for gfx950: instantiation of pass 1 for same-type
// pairs, pass 2 (sig_finalize) and the launchers.
#include "sig_chunk.h"

namespace peat {
namespace {

// ---- pass 2 ----------------------------------------------------------------
// The output record as 8-byte words in declaration order: n, the eight
// counts, first_nan_index, the mismatch counts, hist_zero, hist_under,
// hist_over, the bins, max_abs .. argmax_rel and the six sums.
constexpr int kW_n = 0, kW_cnt = 1, kW_fnan = kW_cnt + kCnt, kW_mism = kW_fnan + 1,
              kW_hzero = kW_mism + PEAT_MAX_THRESHOLDS, kW_hunder = kW_hzero + 1, kW_hover = kW_hzero + 2,
              kW_hist = kW_hzero + 3, kW_maxabs = kW_hist + PEAT_MAX_BINS, kW_ixabs = kW_maxabs + 1,
              kW_maxulp = kW_maxabs + 2, kW_ixulp = kW_maxabs + 3, kW_sumulp = kW_maxabs + 4,
              kW_maxrel = kW_maxabs + 5, kW_ixrel = kW_maxabs + 6, kW_sums = kW_maxabs + 7, kOutWords = kW_sums + 6;
static_assert(sizeof(peat_signature_t) == kOutWords * 8, "peat_signature_t words");
static_assert(offsetof(peat_signature_t, n_valid) == (kW_cnt + C_VALID) * 8 &&
                  offsetof(peat_signature_t, n_finite) == (kW_cnt + C_FINITE) * 8 &&
                  offsetof(peat_signature_t, n_rel) == (kW_cnt + C_REL) * 8 &&
                  offsetof(peat_signature_t, n_nan_golden) == (kW_cnt + C_NAN_G) * 8 &&
                  offsetof(peat_signature_t, n_nan_test) == (kW_cnt + C_NAN_T) * 8 &&
                  offsetof(peat_signature_t, n_inf_golden) == (kW_cnt + C_INF_G) * 8 &&
                  offsetof(peat_signature_t, n_inf_test) == (kW_cnt + C_INF_T) * 8 &&
                  offsetof(peat_signature_t, n_nan_pairs) == (kW_cnt + C_NANPAIR) * 8,
              "peat_signature_t counts");
static_assert(offsetof(peat_signature_t, first_nan_index) == kW_fnan * 8 &&
                  offsetof(peat_signature_t, n_mismatch) == kW_mism * 8 &&
                  offsetof(peat_signature_t, hist_zero) == kW_hzero * 8 &&
                  offsetof(peat_signature_t, hist_under) == kW_hunder * 8 &&
                  offsetof(peat_signature_t, hist_over) == kW_hover * 8 && offsetof(peat_signature_t, hist) == kW_hist * 8,
              "peat_signature_t histogram");
static_assert(offsetof(peat_signature_t, max_abs) == kW_maxabs * 8 &&
                  offsetof(peat_signature_t, argmax_abs) == kW_ixabs * 8 &&
                  offsetof(peat_signature_t, max_ulp) == kW_maxulp * 8 &&
                  offsetof(peat_signature_t, argmax_ulp) == kW_ixulp * 8 &&
                  offsetof(peat_signature_t, sum_ulp) == kW_sumulp * 8 &&
                  offsetof(peat_signature_t, max_rel) == kW_maxrel * 8 &&
                  offsetof(peat_signature_t, argmax_rel) == kW_ixrel * 8 &&
                  offsetof(peat_signature_t, sum_abs) == kW_sums * 8 && offsetof(peat_signature_t, sum_gt) == (kW_sums + 5) * 8,
              "peat_signature_t maxima and sums");
static_assert(kHistSlots == 67, "histogram tail: three slots beyond the wave's 64 lanes");

// Output word of histogram slot s (zero | under | bins | over, then unused
// slots, which are zero, onto the unused bins): a bijection of the 67 slots
// onto the words hist_zero .. hist[63].
__device__ __forceinline__ int slot_word(int s, int nb) {
    return s == 0 ? kW_hzero
                  : (s == 1 ? kW_hunder : (s == nb + 2 ? kW_hover : (s <= nb + 1 ? kW_hist + s - 2 : kW_hist + s - 3)));
}

// The fields of a chunk record that the finalize reads.
constexpr int kRecParts = (int)(sizeof(ChunkPartial) / 16);    // 16-byte parts of a record
static_assert(sizeof(ChunkPartial) % 16 == 0, "records are copied in 16-byte parts");
struct RecF {
    double s[kWaves][6];
    int64_t end, ia, ir, iu, fn;
    double ma, mr;
    uint64_t su;
    uint32_t mu, fl;
    uint32_t cn[kCnt + PEAT_MAX_THRESHOLDS];
};
__device__ __forceinline__ RecF load_rec(const ChunkPartial &p) {
    RecF r;
#pragma unroll
    for (int w = 0; w < kWaves; ++w)
#pragma unroll
        for (int k = 0; k < 6; ++k) r.s[w][k] = p.s[w][k];
    r.end = p.run_end;
    r.ma = p.max_abs;
    r.mr = p.max_rel;
    r.ia = p.ix_abs;
    r.ir = p.ix_rel;
    r.iu = p.ix_ulp;
    r.fn = p.first_nan;
    r.su = p.sum_ulp;
    r.mu = p.max_ulp;
    r.fl = p.flips;
#pragma unroll
    for (int k = 0; k < kCnt; ++k) r.cn[k] = p.cnt[k];
#pragma unroll
    for (int j = 0; j < PEAT_MAX_THRESHOLDS; ++j) r.cn[kCnt + j] = p.mism[j];
    return r;
}

// (value desc, index asc) maximum over entries with index >= 0.
template <typename V>
__device__ __forceinline__ void lex_take(V &v, int64_t &ix, V ov, int64_t oi) {
    // bitwise, not short-circuit: no branch per comparison
    const bool take = (oi >= 0) & ((ix < 0) | (ov > v) | ((ov == v) & (oi < ix)));
    v = take ? ov : v;
    ix = take ? oi : ix;
}

// A thread's share of a pair: binary64 sums over its records in order (each
// record's waves in order), the maxima, first NaN and counts of the records
// that end a run (the others carry no exact fields).
struct FinAcc {
    double s[6];
    double ma, mr;
    int64_t ia, ir, iu;
    uint64_t fn;                             // first NaN index, ~0 = none
    uint64_t mu, sulp, flips;
    uint64_t cn[kCnt + PEAT_MAX_THRESHOLDS];
};
__device__ __forceinline__ void fin_merge(FinAcc &A, const RecF &r, bool have) {
#pragma unroll
    for (int k = 0; k < 6; ++k) {
        double t = r.s[0][k];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) t += r.s[w][k];
        // the sum starts at +0 and never becomes -0, so adding +0 is exact
        A.s[k] += have ? t : 0.0;
    }
    const bool e = have && r.end != 0;
    lex_take(A.ma, A.ia, r.ma, e ? r.ia : int64_t(-1));
    lex_take(A.mr, A.ir, r.mr, e ? r.ir : int64_t(-1));
    lex_take(A.mu, A.iu, (uint64_t)r.mu, e ? r.iu : int64_t(-1));
    A.fn = (e && r.fn >= 0 && (uint64_t)r.fn < A.fn) ? (uint64_t)r.fn : A.fn;
    A.sulp += e ? r.su : 0u;
    A.flips += have ? r.fl : 0u;
#pragma unroll
    for (int k = 0; k < kCnt + PEAT_MAX_THRESHOLDS; ++k) A.cn[k] += e ? r.cn[k] : 0u;
}

template <int C, int RM>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t old, uint64_t x) {
    const uint32_t lo = dpp_u32<C, RM>((uint32_t)old, (uint32_t)x);
    const uint32_t hi = dpp_u32<C, RM>((uint32_t)(old >> 32), (uint32_t)(x >> 32));
    return ((uint64_t)hi << 32) | lo;
}
// One step of the wave reductions of the three maxima and the first NaN,
// interleaved so that their data moves overlap.  A lane that DPP does not
// write keeps its own entry, which merges with itself unchanged.
template <int C, int RM>
__device__ __forceinline__ void fin_step(FinAcc &A) {
    const double oma = dpp_f64<C, RM>(A.ma, A.ma), omr = dpp_f64<C, RM>(A.mr, A.mr);
    const uint64_t omu = dpp_u64<C, RM>(A.mu, A.mu), ofn = dpp_u64<C, RM>(A.fn, A.fn);
    const int64_t oia = (int64_t)dpp_u64<C, RM>((uint64_t)A.ia, (uint64_t)A.ia);
    const int64_t oir = (int64_t)dpp_u64<C, RM>((uint64_t)A.ir, (uint64_t)A.ir);
    const int64_t oiu = (int64_t)dpp_u64<C, RM>((uint64_t)A.iu, (uint64_t)A.iu);
    lex_take(A.ma, A.ia, oma, oia);
    lex_take(A.mr, A.ir, omr, oir);
    lex_take(A.mu, A.iu, omu, oiu);
    A.fn = ofn < A.fn ? ofn : A.fn;
}
__device__ __forceinline__ uint64_t lane63_u64(uint64_t v) {
    return ((uint64_t)lane63_u32((uint32_t)(v >> 32)) << 32) | lane63_u32((uint32_t)v);
}
// Wave total of nonnegative integers: in 32 bits when the total is known to
// stay below 2^31 (small, uniform), else exactly in binary64 (below 2^53).
// No test for an all-zero wave: without that branch the compiler interleaves
// the finalize's many totals, whose DPP steps would otherwise wait on one
// another.
__device__ __forceinline__ uint32_t dpp_sum_u32_all(uint32_t v) {
    dsum_step<kDppXor1, 0xF>(v);
    dsum_step<kDppXor2, 0xF>(v);
    dsum_step<kDppHalfMirror, 0xF>(v);
    dsum_step<kDppMirror, 0xF>(v);
    dsum_step<kDppBcast15, 0xA>(v);
    dsum_step<kDppBcast31, 0xC>(v);
    return lane63_u32(v);
}
// The wave totals of a finalize's counts (kCnt + PEAT_MAX_THRESHOLDS) and
// three tail histogram slots, all under one uniform branch.
constexpr int kTot = kCnt + PEAT_MAX_THRESHOLDS + 3;
__device__ __forceinline__ void wave_totals(const uint64_t (&v)[kTot], uint64_t (&t)[kTot], bool small) {
    if (small) {
#pragma unroll
        for (int k = 0; k < kTot; ++k) t[k] = dpp_sum_u32_all((uint32_t)v[k]);
    } else {
#pragma unroll
        for (int k = 0; k < kTot; ++k) t[k] = (uint64_t)dpp_sum((double)v[k]);
    }
}

__global__ void __launch_bounds__(kBlock) sig_finalize(SigParams P) {
    const int pair = blockIdx.x;
    // the pair's fields (uniform: scalar loads from the arguments or the table)
    int64_t n, first;
    int m;
    if (P.single) {
        n = P.one.n;
        first = P.one.first_chunk;
        m = P.one.nchunks;
    } else {
        n = P.descs[pair].n;
        first = P.descs[pair].first_chunk;
        m = P.descs[pair].nchunks;
    }
    n = (int64_t)uniform_u64((uint64_t)n);
    m = (int)__builtin_amdgcn_readfirstlane((uint32_t)m);
    const ChunkPartial *parts = P.partials + (int64_t)uniform_u64((uint64_t)first);
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int nb = P.nbins;

    __shared__ uint64_t wv[kWaves][kOutWords + 1];   // each wave's additive words (+ flips)
    __shared__ double wd[kWaves][8];                 // six sums, max_abs, max_rel
    __shared__ int64_t wi[kWaves][4];                // argmax_abs, argmax_rel, argmax_ulp, first NaN
    __shared__ uint64_t wmu[kWaves];
    // kBlock records (152 KiB of the 160 KiB of LDS of a gfx950 workgroup)
    __shared__ u32x4 stage[kBlock * kRecParts];

    FinAcc A;
#pragma unroll
    for (int k = 0; k < 6; ++k) A.s[k] = 0.0;
    A.ma = A.mr = -1.0;
    A.ia = A.ir = A.iu = -1;
    A.fn = ~uint64_t(0);
    A.mu = A.sulp = A.flips = 0;
#pragma unroll
    for (int k = 0; k < kCnt + PEAT_MAX_THRESHOLDS; ++k) A.cn[k] = 0;
    // The pair's records go to LDS kBlock at a time in one coalesced copy (a
    // thread reading its own record from memory would touch a different
    // cache line in every lane of a load, more lines than the L1 holds);
    // thread t then merges record t of the batch, and wave w sums the
    // histogram rows of records w, w + 4, ...: lane l slot l, and lane l < 63
    // the tail slot 64 + l % 3 of records l / 3 + 21 j (every record and tail
    // slot once).
    uint64_t h0 = 0, ht = 0;
    const ChunkPartial *srec = reinterpret_cast<const ChunkPartial *>(stage);
    const int tr = lane / 3, tslot = 64 + lane % 3;
    for (int base = 0; base < m; base += kBlock) {   // uniform
        const int cnt = min(m - base, kBlock);
        // all parts in flight at once: buffer loads from one scalar base; a
        // part past the batch re-reads the batch's last part, so every load
        // lies within the batch's records (the offset is the per-lane one: a
        // scalar offset is not part of the hardware's range check)
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(parts + base), (short)0, cnt * (int)sizeof(ChunkPartial), kBufFlags);
        const int lim = cnt * kRecParts - 1;
        u32x4 v[kRecParts];
#pragma unroll
        for (int k = 0; k < kRecParts; ++k)
            v[k] = __builtin_amdgcn_raw_buffer_load_b128(rs, min(tid + k * kBlock, lim) * 16, 0, 0);
        // (the scheduler would otherwise pair each load with its store and
        // wait for it, one round trip per part)
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < kRecParts; ++k) stage[tid + k * kBlock] = v[k];
        __syncthreads();
        fin_merge(A, load_rec(srec[min(tid, cnt - 1)]), tid < cnt);
        // bit u: record wave + 4u exists and ends a run (only those rows were written)
        const uint64_t em = __ballot(wave + lane * kWaves < cnt && srec[min(wave + lane * kWaves, cnt - 1)].run_end != 0);
#pragma unroll
        for (int u = 0; u < 64; ++u) {
            const uint32_t x = srec[min(wave + u * kWaves, cnt - 1)].hist[lane];
            h0 += ((em >> u) & 1u) ? x : 0u;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = tr + 21 * j;
            const uint32_t x = srec[min(wave + min(r, 63) * kWaves, cnt - 1)].hist[tslot];
            ht += (lane < 63 && r < 64 && ((em >> r) & 1u)) ? x : 0u;
        }
        __syncthreads();                            // the stage is free again
    }

    // wave totals
    // up to this bound a wave's records (at most m / 4 chunks of 2^18
    // elements) count fewer than 2^31 elements
    const bool small = m <= kBlock * 64;
#pragma unroll
    for (int k = 0; k < 6; ++k) A.s[k] = dpp_sum(A.s[k]);
    fin_step<kDppXor1, 0xF>(A);
    fin_step<kDppXor2, 0xF>(A);
    fin_step<kDppHalfMirror, 0xF>(A);
    fin_step<kDppMirror, 0xF>(A);
    fin_step<kDppBcast15, 0xA>(A);
    fin_step<kDppBcast31, 0xC>(A);
    uint64_t vals[kTot], tot[kTot];
#pragma unroll
    for (int k = 0; k < kCnt + PEAT_MAX_THRESHOLDS; ++k) vals[k] = A.cn[k];
#pragma unroll
    for (int q = 0; q < 3; ++q) vals[kCnt + PEAT_MAX_THRESHOLDS + q] = lane % 3 == q ? ht : 0u;
    wave_totals(vals, tot, small);
    const uint64_t t0 = tot[kTot - 3], t1 = tot[kTot - 2], t2 = tot[kTot - 1];
    // ULP sum in two 32-bit halves (each wave total below 2^38: exact)
    const uint64_t sulp = ((uint64_t)dpp_sum((double)(A.sulp >> 32)) << 32) +
                          (uint64_t)dpp_sum((double)(A.sulp & 0xFFFFFFFFu));
    const uint64_t flips = P.inj_counts ? (uint64_t)dpp_sum((double)A.flips) : 0u;

    // this wave's additive words by output word: lane l slot l (lanes 0-2 the
    // tail slots too), lanes 0-15 the counts, 16 the ULP sum, 17 the flips
    uint64_t *row = wv[wave];
    row[slot_word(lane, nb)] = h0;
    uint64_t v = 0;
#pragma unroll
    for (int k = 0; k < kCnt + PEAT_MAX_THRESHOLDS; ++k) v = lane == k ? tot[k] : v;
    v = lane == 16 ? sulp : (lane == 17 ? flips : v);
    const int vw = lane < kCnt ? kW_cnt + lane
                               : (lane < 16 ? kW_mism + lane - kCnt : (lane == 16 ? kW_sumulp : kOutWords));
    if (lane < 18) row[vw] = v;
    if (lane < 3) row[slot_word(64 + lane, nb)] = lane == 0 ? t0 : (lane == 1 ? t1 : t2);
    // the reductions' results, read from lane 63 by every lane: a lane read
    // inside the branch below would let the compiler move the last step's
    // selects into it, where lane 63 does not execute them
    const double wma = lane63_f64(A.ma), wmr = lane63_f64(A.mr);
    const int64_t wia = (int64_t)lane63_u64((uint64_t)A.ia), wir = (int64_t)lane63_u64((uint64_t)A.ir);
    const int64_t wiu = (int64_t)lane63_u64((uint64_t)A.iu), wfn = (int64_t)lane63_u64(A.fn);  // ~0 is -1
    const uint64_t wmuv = lane63_u64(A.mu);
    if (lane == 0) {
#pragma unroll
        for (int k = 0; k < 6; ++k) wd[wave][k] = A.s[k];
        wd[wave][6] = wma;
        wd[wave][7] = wmr;
        wi[wave][0] = wia;
        wi[wave][1] = wir;
        wi[wave][2] = wiu;
        wi[wave][3] = wfn;
        wmu[wave] = wmuv;
    }
    __syncthreads();

    // one output word per thread, the waves in order; two stores per block.
    // Every thread forms every merged value (broadcast LDS reads) and keeps
    // its own word by selects, so the waves do not diverge here.
    if (tid > kOutWords) return;
    const int t = tid;
    const int ks = min(max(t - kW_sums, 0), 5);
    uint64_t add = 0, nanp = 0, MU = 0;
    double S = 0.0, MA = -1.0, MR = -1.0;
    int64_t IA = -1, IR = -1, IU = -1;
    uint64_t FN = ~uint64_t(0);
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        add += wv[w][t];
        nanp += wv[w][kW_cnt + C_NANPAIR];
        S += wd[w][ks];
        lex_take(MA, IA, wd[w][6], wi[w][0]);
        lex_take(MR, IR, wd[w][7], wi[w][1]);
        lex_take(MU, IU, wmu[w], wi[w][2]);
        const uint64_t x = (uint64_t)wi[w][3];     // -1 (none) is the largest
        FN = x < FN ? x : FN;
    }
    const uint64_t qnan = 0x7FF8000000000000ull;
    const int j = t - kW_mism;
    uint64_t word = add;                      // counts, histogram, sum_ulp, flips
    word = t == kW_n ? (uint64_t)n : word;
    word = t == kW_fnan ? FN : word;
    word = ((j >= 0) & (j < PEAT_MAX_THRESHOLDS)) ? (j < P.nthr ? add + nanp : 0u) : word;
    word = t == kW_maxabs ? (IA >= 0 ? (uint64_t)__double_as_longlong(MA) : qnan) : word;
    word = t == kW_ixabs ? (uint64_t)IA : word;
    word = t == kW_maxulp ? (IU >= 0 ? MU : 0u) : word;
    word = t == kW_ixulp ? (uint64_t)IU : word;
    word = t == kW_maxrel ? (IR >= 0 ? (uint64_t)__double_as_longlong(MR) : qnan) : word;
    word = t == kW_ixrel ? (uint64_t)IR : word;
    word = ((t >= kW_sums) & (t < kW_sums + 6)) ? (uint64_t)__double_as_longlong(S) : word;
    if (t < kOutWords)
        reinterpret_cast<uint64_t *>(P.outs + pair)[t] = word;
    else if (P.inj_counts)
        P.inj_counts[pair] = (int64_t)word;
}

}  // namespace

hipError_t launch_sig_chunks(const SigParams &p, const int64_t range[kKinds + 1], hipStream_t s) {
    for (int kind = 0; kind < kKinds; ++kind) {
        const int64_t n = range[kind + 1] - range[kind];
        if (n <= 0) continue;
        SigParams q = p;
        q.chunk_base = range[kind];
        q.launch_elems = p.kind_elems[kind];
        hipError_t e;
        switch (kind) {
            case 0: e = launch_kind<PEAT_F32, PEAT_F32>(q, n, s); break;
            case 1: e = launch_kind<PEAT_F16, PEAT_F16>(q, n, s); break;
            case 2: e = launch_kind<PEAT_BF16, PEAT_BF16>(q, n, s); break;
            default: e = launch_sig_mixed_kind(q, kind, n, s); break;
        }
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_sig_chunks_inject(const SigParams &p, const int64_t range[kKinds + 1], const InjDesc *inj,
                                    hipStream_t s) {
    for (int kind = 0; kind < kSameKinds; ++kind) {
        const int64_t n = range[kind + 1] - range[kind];
        if (n <= 0) continue;
        SigParams q = p;
        q.chunk_base = range[kind];
        q.launch_elems = p.kind_elems[kind];
        hipError_t e;
        switch (kind) {
            case 0: e = launch_kind_inject<PEAT_F32>(q, n, inj, s); break;
            case 1: e = launch_kind_inject<PEAT_F16>(q, n, inj, s); break;
            default: e = launch_kind_inject<PEAT_BF16>(q, n, inj, s); break;
        }
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_sig_finalize(const SigParams &p, hipStream_t s) {
    if (p.count <= 0) return hipSuccess;
    hipLaunchKernelGGL(sig_finalize, dim3((unsigned)p.count), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

}  // namespace peat
