// Error-signature kernels for gfx950.
//
// Pass 1 (sig_chunk): one 256-thread block per fixed-size chunk of one pair.
// Each thread streams 16-byte vectors of golden and test (4 f32 or 8 f16/bf16
// elements), widens them exactly to binary64 and accumulates the signature of
// its elements; the chunk's record (binary64 partial sums, maxima with their
// lowest index, integer counts, histogram) goes to one ChunkPartial.
//
// Pass 2 (sig_finalize): one block per pair combines its chunk records in a
// fixed order and writes the peat_signature_t.
//
// The definitions follow the paper's FI assessment scores (Section IV-B.3:
// error = absolute difference of golden and faulty values; max, mean,
// variance), the closeness test of Section III-A (torch.isclose, rtol = 0)
// and the error histograms of Section V-D.
//
// Fast path: a wave whose current vectors hold only "ordinary" pairs (both
// finite, no NaN, golden nonzero, same sign) skips all classification: the
// relative error uses a Newton-refined reciprocal for the sum and an exact
// IEEE division only when an element may raise the lane's maximum; counts
// use wave ballots.  Any other wave (or a ragged tail / unaligned pair)
// takes the generic per-element path, which evaluates every case.
//
// Determinism: the element -> lane mapping, the per-lane order and the
// reduction trees depend only on the chunk size, which depends only on n, so
// single, batched and any-grid-size launches give bit-identical records.
#include "peat_internal.h"

namespace peat {
namespace {

constexpr double kRelMargin = 0x1p-30;   // relative slack of the max-rel filter

template <int DT> struct Tr;
template <> struct Tr<PEAT_F32>  { static constexpr int VEC = 4, W = 32, U = 4; };
template <> struct Tr<PEAT_F16>  { static constexpr int VEC = 8, W = 16, U = 2; };
template <> struct Tr<PEAT_BF16> { static constexpr int VEC = 8, W = 16, U = 2; };

template <int DT>
__device__ __forceinline__ double widen(uint32_t b) {
    if constexpr (DT == PEAT_F32) {
        return (double)__uint_as_float(b);
    } else if constexpr (DT == PEAT_BF16) {
        return (double)__uint_as_float(b << 16);
    } else {
        return (double)(float)__builtin_bit_cast(_Float16, (uint16_t)b);
    }
}

template <int DT>
__device__ __forceinline__ uint32_t lane_elem(const uint4 &v, int j) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    if constexpr (Tr<DT>::W == 32) {
        return w[j];
    } else {
        return (w[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
    }
}

template <int DT>
__device__ __forceinline__ uint32_t load_elem(const void *base, int64_t i) {
    if constexpr (Tr<DT>::W == 32) {
        return static_cast<const uint32_t *>(base)[i];
    } else {
        return static_cast<const uint16_t *>(base)[i];
    }
}

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

// Binary64 reciprocal: hardware estimate refined by two Newton steps.
__device__ __forceinline__ double recip(double b) {
    double y = __builtin_amdgcn_rcp(b);
    double e = __builtin_fma(-b, y, 1.0);
    y = __builtin_fma(y, e, y);
    e = __builtin_fma(-b, y, 1.0);
    return __builtin_fma(y, e, y);
}

struct Lane {
    double s_abs, s_sq, s_rel, s_g2, s_t2, s_gt;
    double mx_abs, mx_rel, rthr;
    uint64_t s_ulp;
    uint32_t ix_abs, ix_rel, ix_ulp, mu;
    uint32_t first_nan, first_valid;
    uint32_t cnt[kCnt];                    // generic-path counts (per lane)
    uint32_t mism[PEAT_MAX_THRESHOLDS];    // generic-path mismatches (per lane)
};

struct Uni {                               // fast-path counts (wave-uniform)
    uint32_t common;                       // ordinary elements per lane
    uint32_t zero;
    uint32_t mism[PEAT_MAX_THRESHOLDS];
};

struct Shared {
    uint32_t hist[kHistSlots * kBlock];    // lane-private counters, [slot][lane]
    uint8_t slot_of_exp[2048];             // binary64 exponent field -> slot
    double rd[kWaves][6];
    double rmax[kWaves][2];
    uint32_t rix[kWaves][5];               // abs, rel, ulp, first_nan, first_valid
    uint32_t rmu[kWaves];
    uint32_t rcnt[kWaves][kCnt + PEAT_MAX_THRESHOLDS];
};

__device__ __forceinline__ void lane_init(Lane &L, Uni &U) {
    L.s_abs = L.s_sq = L.s_rel = L.s_g2 = L.s_t2 = L.s_gt = 0.0;
    L.mx_abs = -1.0;
    L.mx_rel = -1.0;
    L.rthr = -1.0;
    L.s_ulp = 0;
    L.ix_abs = L.ix_rel = L.ix_ulp = kNone;
    L.mu = 0;
    L.first_nan = L.first_valid = kNone;
#pragma unroll
    for (int c = 0; c < kCnt; ++c) L.cnt[c] = 0;
#pragma unroll
    for (int j = 0; j < PEAT_MAX_THRESHOLDS; ++j) L.mism[j] = 0;
    U.common = 0;
    U.zero = 0;
#pragma unroll
    for (int j = 0; j < PEAT_MAX_THRESHOLDS; ++j) U.mism[j] = 0;
}

__device__ __forceinline__ void rel_candidate(Lane &L, double a, double G, uint32_t li) {
    double r = a / __builtin_fabs(G);           // IEEE division, correctly rounded
    if (r > L.mx_rel) {
        L.mx_rel = r;
        L.ix_rel = li;
        L.rthr = r - r * kRelMargin;
    }
}

// Every case of one pair (NaN, Inf, zero golden, sign change, subnormals).
template <int DT, int NT>
__device__ __forceinline__ void generic_elem(Lane &L, Shared &sh, const SigParams &P,
                                             uint32_t gb, uint32_t tb, uint32_t li, int tid) {
    double G = widen<DT>(gb), T = widen<DT>(tb);
    bool nan_g = G != G, nan_t = T != T;
    bool inf_g = __builtin_isinf(G), inf_t = __builtin_isinf(T);
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
    double a = (G == T) ? 0.0 : __builtin_fabs(T - G);
    uint32_t ulp = ulp_dist<Tr<DT>::W>(gb, tb);
    L.s_ulp += ulp;
    if (ulp > L.mu) {
        L.mu = ulp;
        L.ix_ulp = li;
    }
    uint32_t E = (uint32_t)(__double_as_longlong(a) >> 52);   // a >= 0: no sign bit
    atomicAdd(&sh.hist[(uint32_t)sh.slot_of_exp[E] * kBlock + tid], 1u);
    L.cnt[C_ZERO] += (a == 0.0);
    bool ainf = __builtin_isinf(a);
#pragma unroll
    for (int j = 0; j < NT; ++j) L.mism[j] += (a > P.thr[j]) || ainf;
    if (a > L.mx_abs) {
        L.mx_abs = a;
        L.ix_abs = li;
    }
    if (inf_g || inf_t) return;
    L.cnt[C_FINITE] += 1;
    L.s_abs += a;
    L.s_sq = __builtin_fma(a, a, L.s_sq);
    L.s_g2 = __builtin_fma(G, G, L.s_g2);
    L.s_t2 = __builtin_fma(T, T, L.s_t2);
    L.s_gt = __builtin_fma(G, T, L.s_gt);
    if (G != 0.0) {
        L.cnt[C_REL] += 1;
        double r = a / __builtin_fabs(G);
        L.s_rel += r;
        if (r > L.mx_rel) {
            L.mx_rel = r;
            L.ix_rel = li;
            L.rthr = r - r * kRelMargin;
        }
    }
}

// One 16-byte vector of golden and one of test; li0 = local index of its
// first element.  Called in wave-uniform control flow with every lane active.
template <int DT, int NT>
__device__ __forceinline__ void vec_step(Lane &L, Uni &U, Shared &sh, const SigParams &P,
                                         const uint4 &gv, const uint4 &tv, uint32_t li0, int tid) {
    constexpr int VEC = Tr<DT>::VEC;
    double G[VEC], T[VEC], A[VEC], R[VEC];
    bool rare = false;
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        G[j] = widen<DT>(lane_elem<DT>(gv, j));
        T[j] = widen<DT>(lane_elem<DT>(tv, j));
        A[j] = __builtin_fabs(T[j] - G[j]);
        R[j] = A[j] * recip(__builtin_fabs(G[j]));
        rare |= !__builtin_isfinite(R[j]);      // NaN/Inf on either side, or G == 0
    }
    uint32_t sx = (gv.x ^ tv.x) | (gv.y ^ tv.y) | (gv.z ^ tv.z) | (gv.w ^ tv.w);
    if constexpr (Tr<DT>::W == 32) {
        rare |= (sx & 0x80000000u) != 0;        // a sign change
    } else {
        rare |= (sx & 0x80008000u) != 0;
    }
    if (__ballot(rare) == 0) {
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            const double a = A[j];
            const uint32_t li = li0 + j;
            L.s_abs += a;
            L.s_sq = __builtin_fma(a, a, L.s_sq);
            L.s_g2 = __builtin_fma(G[j], G[j], L.s_g2);
            L.s_t2 = __builtin_fma(T[j], T[j], L.s_t2);
            L.s_gt = __builtin_fma(G[j], T[j], L.s_gt);
            if (a > L.mx_abs) L.ix_abs = li;
            L.mx_abs = __builtin_fmax(L.mx_abs, a);
            uint32_t gb = lane_elem<DT>(gv, j), tb = lane_elem<DT>(tv, j);
            uint32_t ulp = __sad(tb, gb, 0u);     // same sign: |t - g| of the patterns
            L.s_ulp += ulp;
            if (ulp > L.mu) L.ix_ulp = li;
            L.mu = max(L.mu, ulp);
            uint32_t E = (uint32_t)(__double_as_longlong(a) >> 52);
            atomicAdd(&sh.hist[(uint32_t)sh.slot_of_exp[E] * kBlock + tid], 1u);
            U.zero += wave_count(a == 0.0);
#pragma unroll
            for (int k = 0; k < NT; ++k) U.mism[k] += wave_count(a > P.thr[k]);
            L.s_rel += R[j];
            if (R[j] > L.rthr) rel_candidate(L, a, G[j], li);
        }
        U.common += VEC;
        L.first_valid = min(L.first_valid, li0);
    } else {
#pragma unroll
        for (int j = 0; j < VEC; ++j)
            generic_elem<DT, NT>(L, sh, P, lane_elem<DT>(gv, j), lane_elem<DT>(tv, j), li0 + j, tid);
    }
}

// ---- wave / block reductions (fixed butterfly order) ----------------------
__device__ __forceinline__ double wsum(double v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;
}
__device__ __forceinline__ uint32_t wsum_u(uint32_t v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;
}
__device__ __forceinline__ uint64_t wsum_u64(uint64_t v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
    return v;
}
__device__ __forceinline__ uint32_t wmin_u(uint32_t v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = min(v, (uint32_t)__shfl_xor(v, o));
    return v;
}
// (value desc, index asc) over entries with index != kNone
__device__ __forceinline__ void wmax_d(double &v, uint32_t &ix) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        double ov = __shfl_xor(v, o);
        uint32_t oi = __shfl_xor(ix, o);
        bool take = (oi != kNone) && (ix == kNone || ov > v || (ov == v && oi < ix));
        v = take ? ov : v;
        ix = take ? oi : ix;
    }
}
__device__ __forceinline__ void wmax_u(uint32_t &v, uint32_t &ix) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        uint32_t ov = __shfl_xor(v, o);
        uint32_t oi = __shfl_xor(ix, o);
        bool take = (oi != kNone) && (ix == kNone || ov > v || (ov == v && oi < ix));
        v = take ? ov : v;
        ix = take ? oi : ix;
    }
}

template <int DT, int NT>
__device__ void chunk_body(const SigParams &P, Shared &sh, const SigDesc &d, int64_t cin, int64_t gchunk) {
    constexpr int VEC = Tr<DT>::VEC;
    constexpr int U = Tr<DT>::U;
    constexpr int SUPER = kBlock * VEC * U;     // elements per block super-step (4096)
    const int tid = threadIdx.x;
    const int64_t off = cin << d.chunk_log2;    // first element of the chunk
    const int64_t rest = d.n - off;
    const uint32_t len = (uint32_t)(rest < (int64_t(1) << d.chunk_log2) ? rest : (int64_t(1) << d.chunk_log2));

    Lane L;
    Uni Un;
    lane_init(L, Un);

    const uint32_t nsuper = d.aligned ? len / SUPER : 0;
    constexpr int ESZ = Tr<DT>::W / 8;
    const uint4 *gp = reinterpret_cast<const uint4 *>(static_cast<const char *>(d.g) + off * ESZ);
    const uint4 *tp = reinterpret_cast<const uint4 *>(static_cast<const char *>(d.t) + off * ESZ);

    if (nsuper > 0) {
        uint4 gc[U], tc[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            gc[u] = gp[u * kBlock + tid];
            tc[u] = tp[u * kBlock + tid];
        }
        for (uint32_t s = 0; s < nsuper; ++s) {
            uint4 gn[U], tn[U];
            const bool more = s + 1 < nsuper;
            if (more) {
                const uint32_t base = (s + 1) * (U * kBlock);
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    gn[u] = gp[base + u * kBlock + tid];
                    tn[u] = tp[base + u * kBlock + tid];
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t li0 = ((s * U + u) * kBlock + tid) * VEC;
                vec_step<DT, NT>(L, Un, sh, P, gc[u], tc[u], li0, tid);
            }
            if (more) {
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    gc[u] = gn[u];
                    tc[u] = tn[u];
                }
            }
        }
    }
    // ragged tail, or the whole chunk when a pointer is not 16-byte aligned
    const void *gb = static_cast<const char *>(d.g) + off * ESZ;
    const void *tb = static_cast<const char *>(d.t) + off * ESZ;
    for (uint32_t li = nsuper * SUPER + tid; li < len; li += kBlock)
        generic_elem<DT, NT>(L, sh, P, load_elem<DT>(gb, li), load_elem<DT>(tb, li), li, tid);

    // ---- epilogue: reduce the block into the chunk record ----------------
    const int wave = tid >> 6, lane = tid & 63;
    double sums[6] = {L.s_abs, L.s_sq, L.s_rel, L.s_g2, L.s_t2, L.s_gt};
#pragma unroll
    for (int k = 0; k < 6; ++k) sums[k] = wsum(sums[k]);
    double mxa = L.mx_abs, mxr = L.mx_rel;
    uint32_t ixa = L.ix_abs, ixr = L.ix_rel, ixu = L.ix_ulp, mu = L.mu;
    wmax_d(mxa, ixa);
    wmax_d(mxr, ixr);
    wmax_u(mu, ixu);
    uint32_t fnan = wmin_u(L.first_nan), fval = wmin_u(L.first_valid);
    uint64_t sulp = wsum_u64(L.s_ulp);
    uint32_t cnts[kCnt + PEAT_MAX_THRESHOLDS];
#pragma unroll
    for (int c = 0; c < kCnt; ++c) cnts[c] = wsum_u(L.cnt[c]);
#pragma unroll
    for (int j = 0; j < PEAT_MAX_THRESHOLDS; ++j) cnts[kCnt + j] = j < NT ? wsum_u(L.mism[j]) : 0u;
    // fast-path (wave-uniform) counts: every element there is valid, finite
    // and has a nonzero golden
    const uint32_t common = Un.common * 64u;
    cnts[C_VALID] += common;
    cnts[C_FINITE] += common;
    cnts[C_REL] += common;
    cnts[C_ZERO] += Un.zero;
#pragma unroll
    for (int j = 0; j < NT; ++j) cnts[kCnt + j] += Un.mism[j];
    if (lane == 0) {
#pragma unroll
        for (int k = 0; k < 6; ++k) sh.rd[wave][k] = sums[k];
        sh.rmax[wave][0] = mxa;
        sh.rmax[wave][1] = mxr;
        sh.rix[wave][0] = ixa;
        sh.rix[wave][1] = ixr;
        sh.rix[wave][2] = ixu;
        sh.rix[wave][3] = fnan;
        sh.rix[wave][4] = fval;
        sh.rmu[wave] = mu;
#pragma unroll
        for (int c = 0; c < kCnt + PEAT_MAX_THRESHOLDS; ++c) sh.rcnt[wave][c] = cnts[c];
    }
    // the u64 ulp sum is kept per wave in the double scratch (bit copy)
    __shared__ uint64_t rulp[kWaves];
    if (lane == 0) rulp[wave] = sulp;
    __syncthreads();

    ChunkPartial *out = P.partials + gchunk;
    // histogram: thread t sums slot t/4 over a quarter of the lanes
    {
        const int slot = tid >> 2, q = tid & 3;
        uint32_t acc = 0;
        if (slot < kHistSlots) {
            const uint32_t *row = sh.hist + slot * kBlock + q * 64;
#pragma unroll 8
            for (int c = 0; c < 64; ++c) acc += row[(c + slot + 8 * q) & 63];
        }
        acc += __shfl_xor(acc, 1);
        acc += __shfl_xor(acc, 2);
        if (q == 0 && slot < kHistSlots) out->hist[slot] = acc;
        // slots 64, 65 (beyond 256/4 threads): one thread each
        if (tid < kHistSlots - 64) {
            const int s2 = 64 + tid;
            uint32_t a2 = 0;
            for (int c = 0; c < kBlock; ++c) a2 += sh.hist[s2 * kBlock + c];
            out->hist[s2] = a2;
        }
    }
    if (tid == 0) {
        double s[6] = {0, 0, 0, 0, 0, 0};
        double ma = -1.0, mr = -1.0;
        uint32_t ia = kNone, ir = kNone, iu = kNone, fn = kNone, fv = kNone, m = 0;
        uint64_t su = 0;
        uint32_t cn[kCnt + PEAT_MAX_THRESHOLDS];
        for (int c = 0; c < kCnt + PEAT_MAX_THRESHOLDS; ++c) cn[c] = 0;
        for (int w = 0; w < kWaves; ++w) {
            for (int k = 0; k < 6; ++k) s[k] += sh.rd[w][k];
            double va = sh.rmax[w][0], vr = sh.rmax[w][1];
            uint32_t xa = sh.rix[w][0], xr = sh.rix[w][1], xu = sh.rix[w][2];
            if (xa != kNone && (ia == kNone || va > ma || (va == ma && xa < ia))) { ma = va; ia = xa; }
            if (xr != kNone && (ir == kNone || vr > mr || (vr == mr && xr < ir))) { mr = vr; ir = xr; }
            uint32_t vu = sh.rmu[w];
            if (xu != kNone && (iu == kNone || vu > m || (vu == m && xu < iu))) { m = vu; iu = xu; }
            fn = min(fn, sh.rix[w][3]);
            fv = min(fv, sh.rix[w][4]);
            su += rulp[w];
            for (int c = 0; c < kCnt + PEAT_MAX_THRESHOLDS; ++c) cn[c] += sh.rcnt[w][c];
        }
        // every ULP distance in the chunk is 0: the first valid element is the maximum
        if (iu == kNone) { m = 0; iu = fv; }
        out->s_abs = s[0];
        out->s_sq = s[1];
        out->s_rel = s[2];
        out->s_g2 = s[3];
        out->s_t2 = s[4];
        out->s_gt = s[5];
        out->max_abs = ma;
        out->max_rel = mr;
        out->ix_abs = ia == kNone ? -1 : off + ia;
        out->ix_rel = ir == kNone ? -1 : off + ir;
        out->ix_ulp = iu == kNone ? -1 : off + iu;
        out->first_nan = fn == kNone ? -1 : off + fn;
        out->first_valid = fv == kNone ? -1 : off + fv;
        out->sum_ulp = su;
        out->max_ulp = m;
        for (int c = 0; c < kCnt; ++c) out->cnt[c] = cn[c];
        for (int j = 0; j < PEAT_MAX_THRESHOLDS; ++j) out->mism[j] = cn[kCnt + j];
    }
}

template <int NT>
__global__ void __launch_bounds__(kBlock, 2) sig_chunk(SigParams P) {
    __shared__ Shared sh;
    const int64_t gchunk = blockIdx.x;
    const int pair = P.chunk_pair[gchunk];
    const SigDesc d = P.descs[pair];
    const int64_t cin = gchunk - d.first_chunk;
    const int tid = threadIdx.x;
    // clear the lane-private histogram counters and build the exponent table
    for (int i = tid; i < kHistSlots * kBlock; i += kBlock) sh.hist[i] = 0;
    const int w = (P.hi - P.lo) / P.nbins;
    for (int E = tid; E < 2048; E += kBlock) {
        int slot;
        if (E == 0) {
            slot = 0;                          // error 0 (counted apart, under here)
        } else if (E == 2047) {
            slot = P.nbins + 1;                // infinite error
        } else {
            int k = E - 1023;                  // a in [2^k, 2^(k+1))
            slot = k < P.lo ? 0 : (k >= P.hi ? P.nbins + 1 : 1 + (k - P.lo) / w);
        }
        sh.slot_of_exp[E] = (uint8_t)slot;
    }
    __syncthreads();
    switch (d.dtype) {
        case PEAT_F32: chunk_body<PEAT_F32, NT>(P, sh, d, cin, gchunk); break;
        case PEAT_F16: chunk_body<PEAT_F16, NT>(P, sh, d, cin, gchunk); break;
        default: chunk_body<PEAT_BF16, NT>(P, sh, d, cin, gchunk); break;
    }
}

// ---- pass 2 ----------------------------------------------------------------
__global__ void __launch_bounds__(kBlock) sig_finalize(SigParams P) {
    const int pair = blockIdx.x;
    const SigDesc d = P.descs[pair];
    const ChunkPartial *parts = P.partials + d.first_chunk;
    const int m = d.nchunks;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;

    __shared__ double sd[kWaves][8];
    __shared__ int64_t si[kWaves][5];
    __shared__ uint64_t su[kWaves][2 + kCnt + PEAT_MAX_THRESHOLDS];
    __shared__ uint64_t sh_hist[kHistSlots];

    // fp64 sums: each thread a fixed strided subset in order, then a fixed tree
    double s[6] = {0, 0, 0, 0, 0, 0};
    double ma = -1.0, mr = -1.0;
    int64_t ia = -1, ir = -1, iu = -1, fn = -1, fv = -1;
    uint64_t mu = 0, sulp = 0;
    uint64_t cn[kCnt + PEAT_MAX_THRESHOLDS];
#pragma unroll
    for (int c = 0; c < kCnt + PEAT_MAX_THRESHOLDS; ++c) cn[c] = 0;
    for (int c = tid; c < m; c += kBlock) {
        const ChunkPartial &p = parts[c];
        s[0] += p.s_abs; s[1] += p.s_sq; s[2] += p.s_rel;
        s[3] += p.s_g2; s[4] += p.s_t2; s[5] += p.s_gt;
        if (p.ix_abs >= 0 && (ia < 0 || p.max_abs > ma || (p.max_abs == ma && p.ix_abs < ia))) { ma = p.max_abs; ia = p.ix_abs; }
        if (p.ix_rel >= 0 && (ir < 0 || p.max_rel > mr || (p.max_rel == mr && p.ix_rel < ir))) { mr = p.max_rel; ir = p.ix_rel; }
        if (p.ix_ulp >= 0 && (iu < 0 || p.max_ulp > mu || (p.max_ulp == mu && p.ix_ulp < iu))) { mu = p.max_ulp; iu = p.ix_ulp; }
        if (p.first_nan >= 0 && (fn < 0 || p.first_nan < fn)) fn = p.first_nan;
        if (p.first_valid >= 0 && (fv < 0 || p.first_valid < fv)) fv = p.first_valid;
        sulp += p.sum_ulp;
#pragma unroll
        for (int k = 0; k < kCnt; ++k) cn[k] += p.cnt[k];
#pragma unroll
        for (int j = 0; j < PEAT_MAX_THRESHOLDS; ++j) cn[kCnt + j] += p.mism[j];
    }
    // histogram: thread t < slots sums slot t over the chunks
    if (tid < kHistSlots) {
        uint64_t h = 0;
        for (int c = 0; c < m; ++c) h += parts[c].hist[tid];
        sh_hist[tid] = h;
    }
    // wave reductions (fixed butterfly), then waves in order
#pragma unroll
    for (int k = 0; k < 6; ++k) s[k] = wsum(s[k]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        double ova = __shfl_xor(ma, o), ovr = __shfl_xor(mr, o);
        int64_t oia = __shfl_xor(ia, o), oir = __shfl_xor(ir, o), oiu = __shfl_xor(iu, o);
        uint64_t omu = __shfl_xor(mu, o);
        int64_t ofn = __shfl_xor(fn, o), ofv = __shfl_xor(fv, o);
        if (oia >= 0 && (ia < 0 || ova > ma || (ova == ma && oia < ia))) { ma = ova; ia = oia; }
        if (oir >= 0 && (ir < 0 || ovr > mr || (ovr == mr && oir < ir))) { mr = ovr; ir = oir; }
        if (oiu >= 0 && (iu < 0 || omu > mu || (omu == mu && oiu < iu))) { mu = omu; iu = oiu; }
        if (ofn >= 0 && (fn < 0 || ofn < fn)) fn = ofn;
        if (ofv >= 0 && (fv < 0 || ofv < fv)) fv = ofv;
    }
    sulp = wsum_u64(sulp);
#pragma unroll
    for (int k = 0; k < kCnt + PEAT_MAX_THRESHOLDS; ++k) cn[k] = wsum_u64(cn[k]);
    if (lane == 0) {
        for (int k = 0; k < 6; ++k) sd[wave][k] = s[k];
        sd[wave][6] = ma;
        sd[wave][7] = mr;
        si[wave][0] = ia; si[wave][1] = ir; si[wave][2] = iu; si[wave][3] = fn; si[wave][4] = fv;
        su[wave][0] = mu;
        su[wave][1] = sulp;
        for (int k = 0; k < kCnt + PEAT_MAX_THRESHOLDS; ++k) su[wave][2 + k] = cn[k];
    }
    __syncthreads();
    if (tid != 0) return;
    double S[6] = {0, 0, 0, 0, 0, 0};
    double MA = -1.0, MR = -1.0;
    int64_t IA = -1, IR = -1, IU = -1, FN = -1, FV = -1;
    uint64_t MU = 0, SU = 0, CN[kCnt + PEAT_MAX_THRESHOLDS];
    for (int k = 0; k < kCnt + PEAT_MAX_THRESHOLDS; ++k) CN[k] = 0;
    for (int w = 0; w < kWaves; ++w) {
        for (int k = 0; k < 6; ++k) S[k] += sd[w][k];
        double va = sd[w][6], vr = sd[w][7];
        int64_t xa = si[w][0], xr = si[w][1], xu = si[w][2];
        if (xa >= 0 && (IA < 0 || va > MA || (va == MA && xa < IA))) { MA = va; IA = xa; }
        if (xr >= 0 && (IR < 0 || vr > MR || (vr == MR && xr < IR))) { MR = vr; IR = xr; }
        if (xu >= 0 && (IU < 0 || su[w][0] > MU || (su[w][0] == MU && xu < IU))) { MU = su[w][0]; IU = xu; }
        if (si[w][3] >= 0 && (FN < 0 || si[w][3] < FN)) FN = si[w][3];
        if (si[w][4] >= 0 && (FV < 0 || si[w][4] < FV)) FV = si[w][4];
        SU += su[w][1];
        for (int k = 0; k < kCnt + PEAT_MAX_THRESHOLDS; ++k) CN[k] += su[w][2 + k];
    }
    peat_signature_t o;
    o.n = d.n;
    o.n_valid = (int64_t)CN[C_VALID];
    o.n_finite = (int64_t)CN[C_FINITE];
    o.n_rel = (int64_t)CN[C_REL];
    o.n_nan_golden = (int64_t)CN[C_NAN_G];
    o.n_nan_test = (int64_t)CN[C_NAN_T];
    o.n_inf_golden = (int64_t)CN[C_INF_G];
    o.n_inf_test = (int64_t)CN[C_INF_T];
    o.n_nan_pairs = (int64_t)CN[C_NANPAIR];
    o.first_nan_index = FN;
    for (int j = 0; j < PEAT_MAX_THRESHOLDS; ++j)
        o.n_mismatch[j] = j < P.nthr ? (int64_t)(CN[kCnt + j] + CN[C_NANPAIR]) : 0;
    o.hist_zero = (int64_t)CN[C_ZERO];
    o.hist_under = (int64_t)sh_hist[0] - (int64_t)CN[C_ZERO];
    o.hist_over = (int64_t)sh_hist[P.nbins + 1];
    for (int b = 0; b < PEAT_MAX_BINS; ++b) o.hist[b] = b < P.nbins ? (int64_t)sh_hist[1 + b] : 0;
    const double qnan = __longlong_as_double(0x7FF8000000000000LL);
    o.max_abs = IA >= 0 ? MA : qnan;
    o.argmax_abs = IA;
    o.max_ulp = IU >= 0 ? (int64_t)MU : 0;
    o.argmax_ulp = IU;
    o.sum_ulp = SU;
    o.max_rel = IR >= 0 ? MR : qnan;
    o.argmax_rel = IR;
    o.sum_abs = S[0];
    o.sum_sq = S[1];
    o.sum_rel = S[2];
    o.sum_g2 = S[3];
    o.sum_t2 = S[4];
    o.sum_gt = S[5];
    (void)FV;
    P.outs[pair] = o;
}

}  // namespace

hipError_t launch_sig_chunks(const SigParams &p, int64_t total_chunks, hipStream_t s) {
    if (total_chunks <= 0) return hipSuccess;
    dim3 grid((unsigned)total_chunks), block(kBlock);
    switch (p.nthr_pad) {
        case 2: hipLaunchKernelGGL(sig_chunk<2>, grid, block, 0, s, p); break;
        case 4: hipLaunchKernelGGL(sig_chunk<4>, grid, block, 0, s, p); break;
        default: hipLaunchKernelGGL(sig_chunk<8>, grid, block, 0, s, p); break;
    }
    return hipGetLastError();
}

hipError_t launch_sig_finalize(const SigParams &p, hipStream_t s) {
    if (p.count <= 0) return hipSuccess;
    hipLaunchKernelGGL(sig_finalize, dim3((unsigned)p.count), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

}  // namespace peat
