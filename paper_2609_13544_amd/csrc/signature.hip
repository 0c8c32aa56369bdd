// Error-signature kernels for gfx950: instantiation of pass 1 for same-type
// pairs, pass 2 (sig_finalize) and the launchers.
#include "sig_chunk.h"

namespace peat {
namespace {

// ---- pass 2 ----------------------------------------------------------------
__global__ void __launch_bounds__(kBlock) sig_finalize(SigParams P) {
    const int pair = blockIdx.x;
    const SigDesc d = P.single ? P.one : P.descs[pair];
    const ChunkPartial *parts = P.partials + d.first_chunk;
    const int m = d.nchunks;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;

    __shared__ double sd[kWaves][8];
    __shared__ int64_t si[kWaves][5];
    __shared__ uint64_t su[kWaves][2 + kCnt + PEAT_MAX_THRESHOLDS];
    __shared__ uint64_t sh_hist[kHistSlots];
    __shared__ uint64_t sh_hwave[kWaves][kHistSlots];
    __shared__ uint64_t su_flips[kWaves];

    // binary64 sums: each thread a fixed strided subset in order, then a fixed tree
    double s[6] = {0, 0, 0, 0, 0, 0};
    double ma = -1.0, mr = -1.0;
    int64_t ia = -1, ir = -1, iu = -1, fn = -1, fv = -1;
    uint64_t mu = 0, sulp = 0, flips = 0;
    uint64_t cn[kCnt + PEAT_MAX_THRESHOLDS];
#pragma unroll
    for (int c = 0; c < kCnt + PEAT_MAX_THRESHOLDS; ++c) cn[c] = 0;
    for (int c = tid; c < m; c += kBlock) {
        const ChunkPartial &p = parts[c];
#pragma unroll
        for (int k = 0; k < 6; ++k) {
            double t = p.s[0][k];                 // the chunk: its waves in order
#pragma unroll
            for (int w = 1; w < kWaves; ++w) t += p.s[w][k];
            s[k] += t;
        }
        // every field read before any comparison, so the loads go out together
        // instead of one round trip per branch; the exact fields count only
        // in a record that ends its block's run (the others were not written)
        const int64_t pend = p.run_end;
        const double pma = p.max_abs, pmr = p.max_rel;
        const int64_t pia = p.ix_abs, pir = p.ix_rel, piu = p.ix_ulp, pfn = p.first_nan, pfv = p.first_valid;
        const uint64_t pmu = p.max_ulp, psu = p.sum_ulp;
        const uint32_t pfl = p.flips;
        uint32_t pcn[kCnt + PEAT_MAX_THRESHOLDS];
#pragma unroll
        for (int k = 0; k < kCnt; ++k) pcn[k] = p.cnt[k];
#pragma unroll
        for (int j = 0; j < PEAT_MAX_THRESHOLDS; ++j) pcn[kCnt + j] = p.mism[j];
        if (P.inj_counts) flips += pfl;
        // (no early exit: that would let the compiler load the exact fields
        // only after the flag, one more round trip per record)
        const bool e = pend != 0;
        if (e && pia >= 0 && (ia < 0 || pma > ma || (pma == ma && pia < ia))) { ma = pma; ia = pia; }
        if (e && pir >= 0 && (ir < 0 || pmr > mr || (pmr == mr && pir < ir))) { mr = pmr; ir = pir; }
        if (e && piu >= 0 && (iu < 0 || pmu > mu || (pmu == mu && piu < iu))) { mu = pmu; iu = piu; }
        if (e && pfn >= 0 && (fn < 0 || pfn < fn)) fn = pfn;
        if (e && pfv >= 0 && (fv < 0 || pfv < fv)) fv = pfv;
        sulp += e ? psu : 0u;
#pragma unroll
        for (int k = 0; k < kCnt + PEAT_MAX_THRESHOLDS; ++k) cn[k] += e ? pcn[k] : 0u;
    }
    // histogram: wave w sums chunks w, w + 4, ... (lane l: slots l and 64 + l),
    // 32 chunks' loads in flight per step (a single pair's records are read
    // in few round trips); the waves are added in order
    {
        constexpr int D = 32;
        uint64_t h0 = 0, h1 = 0;
        const bool two = lane < kHistSlots - 64;
        // every lane loads a valid slot (its value is masked afterwards): a
        // load only some lanes make becomes a branch with a full wait inside,
        // which would take the loads one round trip at a time
        const int lb = 64 + (two ? lane : 0);
        int c = wave;
        for (; c + (D - 1) * kWaves < m; c += D * kWaves) {
            uint32_t a[D], b[D];
#pragma unroll
            for (int u = 0; u < D; ++u) {
                a[u] = parts[c + u * kWaves].hist[lane];
                b[u] = parts[c + u * kWaves].hist[lb];
            }
            // the step's run-end flags, lane u reading chunk u's, issued after
            // the histogram rows so that one wait covers all of them (a wait
            // for the flags first costs a round trip per step)
            const int64_t fl = parts[c + (lane & (D - 1)) * kWaves].run_end;
            const uint64_t em = __ballot(fl != 0);
#pragma unroll
            for (int u = 0; u < D; ++u) {
                const bool e = (em >> u) & 1u;
                h0 += e ? a[u] : 0u;
                h1 += (e && two) ? b[u] : 0u;
            }
        }
        for (; c < m; c += kWaves) {
            const bool e = parts[c].run_end != 0;
            const uint32_t a = parts[c].hist[lane], b = parts[c].hist[lb];
            h0 += e ? a : 0u;
            h1 += (e && two) ? b : 0u;
        }
        sh_hwave[wave][lane] = h0;
        if (two) sh_hwave[wave][64 + lane] = h1;
    }
    __syncthreads();
    if (tid < kHistSlots) {
        uint64_t h = 0;
        for (int w = 0; w < kWaves; ++w) h += sh_hwave[w][tid];
        sh_hist[tid] = h;
    }
#pragma unroll
    for (int k = 0; k < 6; ++k) s[k] = dpp_sum(s[k]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const double ova = __shfl_xor(ma, o), ovr = __shfl_xor(mr, o);
        const int64_t oia = __shfl_xor(ia, o), oir = __shfl_xor(ir, o), oiu = __shfl_xor(iu, o);
        const uint64_t omu = __shfl_xor(mu, o);
        const int64_t ofn = __shfl_xor(fn, o), ofv = __shfl_xor(fv, o);
        if (oia >= 0 && (ia < 0 || ova > ma || (ova == ma && oia < ia))) { ma = ova; ia = oia; }
        if (oir >= 0 && (ir < 0 || ovr > mr || (ovr == mr && oir < ir))) { mr = ovr; ir = oir; }
        if (oiu >= 0 && (iu < 0 || omu > mu || (omu == mu && oiu < iu))) { mu = omu; iu = oiu; }
        if (ofn >= 0 && (fn < 0 || ofn < fn)) fn = ofn;
        if (ofv >= 0 && (fv < 0 || ofv < fv)) fv = ofv;
    }
    // integer totals by DPP in binary64, exact: a count is at most 2^46, and
    // the ULP sum goes as two halves of 32 bits (each wave total below 2^52)
    sulp = ((uint64_t)dpp_sum((double)(sulp >> 32)) << 32) + (uint64_t)dpp_sum((double)(sulp & 0xFFFFFFFFu));
    if (P.inj_counts) {
        flips = (uint64_t)dpp_sum((double)flips);
        if (lane == 0) su_flips[wave] = flips;
    }
#pragma unroll
    for (int k = 0; k < kCnt + PEAT_MAX_THRESHOLDS; ++k) cn[k] = (uint64_t)dpp_sum((double)cn[k]);
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
    if (P.inj_counts) {
        uint64_t f = 0;
        for (int w = 0; w < kWaves; ++w) f += su_flips[w];
        P.inj_counts[pair] = (int64_t)f;
    }
    double S[6] = {0, 0, 0, 0, 0, 0};
    double MA = -1.0, MR = -1.0;
    int64_t IA = -1, IR = -1, IU = -1, FN = -1;
    uint64_t MU = 0, SU = 0, CN[kCnt + PEAT_MAX_THRESHOLDS];
    for (int k = 0; k < kCnt + PEAT_MAX_THRESHOLDS; ++k) CN[k] = 0;
    for (int w = 0; w < kWaves; ++w) {
        for (int k = 0; k < 6; ++k) S[k] += sd[w][k];
        const double va = sd[w][6], vr = sd[w][7];
        const int64_t xa = si[w][0], xr = si[w][1], xu = si[w][2];
        if (xa >= 0 && (IA < 0 || va > MA || (va == MA && xa < IA))) { MA = va; IA = xa; }
        if (xr >= 0 && (IR < 0 || vr > MR || (vr == MR && xr < IR))) { MR = vr; IR = xr; }
        if (xu >= 0 && (IU < 0 || su[w][0] > MU || (su[w][0] == MU && xu < IU))) { MU = su[w][0]; IU = xu; }
        if (si[w][3] >= 0 && (FN < 0 || si[w][3] < FN)) FN = si[w][3];
        SU += su[w][1];
        for (int k = 0; k < kCnt + PEAT_MAX_THRESHOLDS; ++k) CN[k] += su[w][2 + k];
    }
    const int nb = P.nbins;
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
    o.hist_zero = (int64_t)sh_hist[0];
    o.hist_under = (int64_t)sh_hist[1];
    o.hist_over = (int64_t)sh_hist[nb + 2];
    for (int b = 0; b < PEAT_MAX_BINS; ++b) o.hist[b] = b < nb ? (int64_t)sh_hist[2 + b] : 0;
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
    P.outs[pair] = o;
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
