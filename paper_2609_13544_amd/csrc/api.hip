// Host side of libpeat: argument validation, per-device workspace and pinned
// staging, stream ordering, optional kernel timing, and the extern "C"
// entry points declared in include/peat.h.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "peat_internal.h"

using namespace peat;

namespace {

thread_local std::string t_err;
thread_local hipStream_t t_stream = nullptr;
std::mutex g_mu;   // serialises every entry point that touches device state

int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_err = buf;
    return code;
}

int fail_hip(hipError_t e, const char *what) {
    int code = (e == hipErrorOutOfMemory) ? PEAT_ENOMEM : PEAT_EHIP;
    return fail(code, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

#define HIP_OR_FAIL(expr)                                   \
    do {                                                    \
        hipError_t e_ = (expr);                             \
        if (e_ != hipSuccess) return fail_hip(e_, #expr);   \
    } while (0)

constexpr int kSlots = 4;            // pinned staging ring depth
constexpr size_t kAlign = 256;
constexpr int kMaxDevices = 64;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Slot {
    void *host = nullptr;
    size_t size = 0;
    hipEvent_t ev = nullptr;
    bool pending = false;
};

struct ProfRec {
    int cls;
    hipEvent_t a, b;
};

struct Dev {
    int state = 0;                   // 0 unchecked, 1 ok, <0 error code
    char *scratch = nullptr;         // this device's copy of `scratch` (device address)
    void *ws = nullptr;
    size_t ws_size = 0;
    hipEvent_t ws_ev = nullptr;
    bool ws_pending = false;
    Slot slot[kSlots];
    int next_slot = 0;
    bool prof = false;
    std::vector<ProfRec> log;
    std::vector<hipEvent_t> pool;
};

Dev g_dev[kMaxDevices];

// Scratch of peat_signature_batched_noalloc: pair descriptors, chunk map and
// chunk records of one call.  Each device that loads the library holds its
// own copy until the process ends; host code reaches it only through the
// address hipGetSymbolAddress returns for the current device (Dev::scratch).
static __device__ __align__(256) char scratch[PEAT_NOALLOC_SCRATCH_BYTES];

int current_dev(Dev **out) {
    int id = 0;
    HIP_OR_FAIL(hipGetDevice(&id));
    if (id < 0 || id >= kMaxDevices) return fail(PEAT_ENODEV, "device index %d out of range", id);
    Dev &d = g_dev[id];
    if (d.state == 0) {
        hipDeviceProp_t prop;
        HIP_OR_FAIL(hipGetDeviceProperties(&prop, id));
        if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0) {
            d.state = PEAT_ENODEV;
        } else {
            HIP_OR_FAIL(hipEventCreateWithFlags(&d.ws_ev, hipEventDisableTiming));
            for (int k = 0; k < kSlots; ++k)
                HIP_OR_FAIL(hipEventCreateWithFlags(&d.slot[k].ev, hipEventDisableTiming));
            // this device's copy of the static scratch array (device `id` is current)
            void *p = nullptr;
            HIP_OR_FAIL(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
            if (!p) return fail(PEAT_EHIP, "no address for the scratch array on device %d", id);
            d.scratch = static_cast<char *>(p);
            d.state = 1;
        }
    }
    if (d.state < 0) return fail(d.state, "device %d is not gfx950 (MI355X)", id);
    *out = &d;
    return PEAT_OK;
}

// Device workspace of at least `bytes`; orders `s` after the previous user.
int acquire_ws(Dev &d, size_t bytes, hipStream_t s, char **ws) {
    if (bytes > d.ws_size) {
        HIP_OR_FAIL(hipDeviceSynchronize());      // the old buffer may still be in use
        if (d.ws) HIP_OR_FAIL(hipFree(d.ws));
        d.ws = nullptr;
        d.ws_size = 0;
        size_t want = align_up(bytes + bytes / 4 + (size_t(1) << 20));
        HIP_OR_FAIL(hipMalloc(&d.ws, want));
        d.ws_size = want;
        d.ws_pending = false;
    }
    if (d.ws_pending) HIP_OR_FAIL(hipStreamWaitEvent(s, d.ws_ev, 0));
    *ws = static_cast<char *>(d.ws);
    return PEAT_OK;
}

int release_ws(Dev &d, hipStream_t s) {
    HIP_OR_FAIL(hipEventRecord(d.ws_ev, s));
    d.ws_pending = true;
    return PEAT_OK;
}

// Pinned staging buffer of at least `bytes` whose previous copies are done.
int acquire_slot(Dev &d, size_t bytes, Slot **out) {
    Slot &sl = d.slot[d.next_slot];
    d.next_slot = (d.next_slot + 1) % kSlots;
    if (sl.pending) {
        HIP_OR_FAIL(hipEventSynchronize(sl.ev));
        sl.pending = false;
    }
    if (bytes > sl.size) {
        if (sl.host) HIP_OR_FAIL(hipHostFree(sl.host));
        sl.host = nullptr;
        sl.size = 0;
        size_t want = align_up(bytes + bytes / 4 + 4096);
        HIP_OR_FAIL(hipHostMalloc(&sl.host, want, hipHostMallocDefault));
        sl.size = want;
    }
    *out = &sl;
    return PEAT_OK;
}

int release_slot(Slot &sl, hipStream_t s) {
    HIP_OR_FAIL(hipEventRecord(sl.ev, s));
    sl.pending = true;
    return PEAT_OK;
}

int prof_begin(Dev &d, hipStream_t s, hipEvent_t *a) {
    *a = nullptr;
    if (!d.prof) return PEAT_OK;
    if (d.pool.empty()) {
        hipEvent_t e;
        HIP_OR_FAIL(hipEventCreate(&e));
        d.pool.push_back(e);
    }
    *a = d.pool.back();
    d.pool.pop_back();
    HIP_OR_FAIL(hipEventRecord(*a, s));
    return PEAT_OK;
}

int prof_end(Dev &d, hipStream_t s, int cls, hipEvent_t a) {
    if (!a) return PEAT_OK;
    if (d.pool.empty()) {
        hipEvent_t e;
        HIP_OR_FAIL(hipEventCreate(&e));
        d.pool.push_back(e);
    }
    hipEvent_t b = d.pool.back();
    d.pool.pop_back();
    HIP_OR_FAIL(hipEventRecord(b, s));
    d.log.push_back({cls, a, b});
    return PEAT_OK;
}

int check_dtype(int32_t dt) {
    return (dt == PEAT_F32 || dt == PEAT_F16 || dt == PEAT_BF16) ? PEAT_OK : PEAT_EDTYPE;
}

int elem_size(int32_t dt) { return dt == PEAT_F32 ? 4 : 2; }

int check_bins(const peat_bins_t &b) {
    if (b.reserved != 0) return fail(PEAT_EINVAL, "reserved fields must be 0");
    const int lo = b.lo_log2, hi = b.hi_log2, nb = b.nbins;
    if (lo < -1022 || hi > 1024 || lo >= hi)
        return fail(PEAT_EINVAL, "bins need -1022 <= lo_log2 < hi_log2 <= 1024 (got %d, %d)", lo, hi);
    if (nb < 1 || nb > PEAT_MAX_BINS || (hi - lo) % nb != 0)
        return fail(PEAT_EINVAL, "nbins must be in [1, 64] and divide hi_log2 - lo_log2 (got %d)", nb);
    return PEAT_OK;
}

int check_bins_thr(const peat_bins_t *bins, const peat_thresholds_t *thr) {
    if (!bins || !thr) return fail(PEAT_EINVAL, "bins and thresholds must not be NULL");
    if (thr->reserved != 0) return fail(PEAT_EINVAL, "reserved fields must be 0");
    int rc = check_bins(*bins);
    if (rc) return rc;
    if (thr->count < 0 || thr->count > PEAT_MAX_THRESHOLDS)
        return fail(PEAT_EINVAL, "threshold count must be in [0, 8] (got %d)", thr->count);
    for (int j = 0; j < thr->count; ++j) {
        if (std::isnan(thr->abs_tol[j]) || thr->abs_tol[j] < 0)
            return fail(PEAT_EINVAL, "threshold %d must be >= 0 and not NaN", j);
        if (std::isnan(thr->rel_tol[j]) || thr->rel_tol[j] < 0)
            return fail(PEAT_EINVAL, "relative tolerance %d must be >= 0 and not NaN", j);
    }
    return PEAT_OK;
}

int check_pair(const peat_pair_t &p, int k) {
    if (check_dtype(p.dtype)) return fail(PEAT_EDTYPE, "pair %d: unknown dtype %d", k, p.dtype);
    if (p.n < 0) return fail(PEAT_EINVAL, "pair %d: n < 0", k);
    if (p.reserved != 0) return fail(PEAT_EINVAL, "pair %d: reserved field must be 0", k);
    if (p.n > 0 && (!p.golden || !p.test)) return fail(PEAT_EINVAL, "pair %d: NULL tensor with n > 0", k);
    if (p.n > (int64_t(1) << 46)) return fail(PEAT_EINVAL, "pair %d: n above 2^46", k);
    return PEAT_OK;
}

int check_mixed(const peat_mixed_pair_t &p, int k) {
    if (pair_kind(p.golden_dtype, p.test_dtype) < 0)
        return fail(PEAT_EDTYPE, "pair %d: golden/test types %d/%d not accepted", k, p.golden_dtype, p.test_dtype);
    if (p.n < 0) return fail(PEAT_EINVAL, "pair %d: n < 0", k);
    if (p.n > 0 && (!p.golden || !p.test)) return fail(PEAT_EINVAL, "pair %d: NULL tensor with n > 0", k);
    if (p.n > (int64_t(1) << 46)) return fail(PEAT_EINVAL, "pair %d: n above 2^46", k);
    if ((reinterpret_cast<uintptr_t>(p.golden) % elem_bytes(p.golden_dtype)) != 0 ||
        (reinterpret_cast<uintptr_t>(p.test) % elem_bytes(p.test_dtype)) != 0)
        return fail(PEAT_EINVAL, "pair %d: a tensor is not aligned to its element size", k);
    return PEAT_OK;
}

// Same-type pairs, validated, as mixed pairs of equal types.
int same_type_pairs(const peat_pair_t *pairs, int32_t count, std::vector<peat_mixed_pair_t> &out) {
    if (count < 0) return fail(PEAT_EINVAL, "count < 0");
    if (count > 0 && !pairs) return fail(PEAT_EINVAL, "pairs is NULL");
    int rc;
    for (int k = 0; k < count; ++k)
        if ((rc = check_pair(pairs[k], k))) return rc;
    out.resize((size_t)count);
    for (int k = 0; k < count; ++k)
        out[k] = peat_mixed_pair_t{pairs[k].golden, pairs[k].test, pairs[k].n, pairs[k].dtype, pairs[k].dtype};
    return PEAT_OK;
}

// Partition every pair into chunks; the chunks of each kind (golden/test
// type combination) get one contiguous range [range[kind], range[kind + 1])
// of the global numbering (one launch per kind).
int build_descs(const peat_mixed_pair_t *pairs, int32_t count, std::vector<SigDesc> &descs,
                int64_t range[kKinds + 1], int64_t *total_out) {
    descs.assign((size_t)count, SigDesc{});
    // Within a kind the pairs with the largest chunks come first, so that a
    // launch ends on its smallest chunks and its last round of blocks is
    // short (a chunk's record does not depend on where it lies in the launch
    // or on which block works it).  A stable counting sort by (kind, chunk
    // class); the pairs of a class keep their order.
    constexpr int kClasses = kMaxChunkLog2 - kMinChunkLog2 + 1;
    std::vector<int> key((size_t)count), order((size_t)count);
    int start[kKinds * kClasses + 1] = {};
    for (int k = 0; k < count; ++k) {
        key[k] = pair_kind(pairs[k].golden_dtype, pairs[k].test_dtype) * kClasses +
                 (kMaxChunkLog2 - chunk_log2_for(pairs[k].n));
        ++start[key[k] + 1];
    }
    for (int i = 0; i < kKinds * kClasses; ++i) start[i + 1] += start[i];
    for (int k = 0; k < count; ++k) order[start[key[k]]++] = k;
    int64_t total = 0;
    int pos = 0;
    for (int kind = 0; kind < kKinds; ++kind) {
        range[kind] = total;
        for (; pos < count && key[order[pos]] / kClasses == kind; ++pos) {
            const int k = order[pos];
            SigDesc &sd = descs[k];
            sd.g = pairs[k].golden;
            sd.t = pairs[k].test;
            sd.n = pairs[k].n;
            sd.dtype = (int16_t)pairs[k].golden_dtype;
            sd.tdtype = (int16_t)pairs[k].test_dtype;
            sd.chunk_log2 = chunk_log2_for(sd.n);
            const int64_t nch = (sd.n + (int64_t(1) << sd.chunk_log2) - 1) >> sd.chunk_log2;
            sd.first_chunk = total;
            sd.nchunks = (int32_t)nch;
            sd.aligned = ((reinterpret_cast<uintptr_t>(sd.g) | reinterpret_cast<uintptr_t>(sd.t)) & 15) == 0;
            total += nch;
        }
    }
    range[kKinds] = total;
    if (total > 0x7FFFFFFF) return fail(PEAT_EINVAL, "batch needs %lld chunks (max 2^31-1)", (long long)total);
    *total_out = total;
    return PEAT_OK;
}

// Elements of each kind's pairs (the chunk pass sizes its block groups by them).
void set_kind_elems(SigParams &P, const peat_mixed_pair_t *pairs, int32_t count) {
    for (int kind = 0; kind < kKinds; ++kind) P.kind_elems[kind] = 0;
    for (int k = 0; k < count; ++k) {
        const int kind = pair_kind(pairs[k].golden_dtype, pairs[k].test_dtype);
        if (kind >= 0) P.kind_elems[kind] += pairs[k].n;
    }
}

// Golden reuse: a batch in which at most half as many distinct golden
// tensors as pairs appear (a replay batch signs many test tensors against one
// golden), together at most kKeepGoldenBytes, has its goldens read with the
// default cache policy, so that the shared lines are served from the caches
// instead of HBM; otherwise every byte is read once, nontemporally.
constexpr int64_t kKeepGoldenBytes = int64_t(64) << 20;
template <typename PairT, typename DtypeFn>
int32_t golden_reuse(const PairT *pairs, int32_t count, DtypeFn golden_dtype) {
    if (count < 2) return 0;
    std::vector<std::pair<uintptr_t, int64_t>> g((size_t)count);
    for (int k = 0; k < count; ++k)
        g[k] = {reinterpret_cast<uintptr_t>(pairs[k].golden), pairs[k].n * elem_bytes(golden_dtype(pairs[k]))};
    std::sort(g.begin(), g.end());
    int64_t distinct = 0, bytes = 0;
    for (size_t i = 0; i < g.size(); ++i) {
        if (i + 1 < g.size() && g[i + 1].first == g[i].first) continue;   // the largest extent of a pointer
        ++distinct;
        bytes += g[i].second;
    }
    return (2 * distinct <= count && bytes <= kKeepGoldenBytes) ? 1 : 0;
}

// The bins and closeness tests of a signature launch.
void set_bins_thr(SigParams &P, const peat_bins_t &bins, const peat_thresholds_t &thr) {
    P.lo = bins.lo_log2;
    P.hi = bins.hi_log2;
    P.nbins = bins.nbins;
    P.nthr = thr.count;
    P.nthr_pad = thr.count <= 2 ? 2 : (thr.count <= 4 ? 4 : 8);
    P.thr_min = HUGE_VAL;
    P.any_rtol = 0;
    for (int j = 0; j < PEAT_MAX_THRESHOLDS; ++j) {
        P.thr[j] = j < thr.count ? thr.abs_tol[j] : HUGE_VAL;
        P.rthr[j] = j < thr.count ? thr.rel_tol[j] : 0.0;
        if (P.rthr[j] != 0.0) P.any_rtol = 1;
        if (P.thr[j] < P.thr_min) P.thr_min = P.thr[j];
    }
}

// Common core of every signature call.  When host_outs is set the records go
// through workspace + pinned staging and the call waits for them.  With inj
// (one InjDesc per pair, same-type pairs) the chunk pass first injects the
// test tensors' bit flips and d_counts receives the flip counts.
int signature_core(const peat_mixed_pair_t *pairs, int32_t count, const peat_bins_t *bins,
                   const peat_thresholds_t *thr, peat_signature_t *d_outs,
                   peat_signature_t *host_outs, hipStream_t s, const std::vector<InjDesc> *inj = nullptr,
                   int64_t *d_counts = nullptr) {
    if (count < 0) return fail(PEAT_EINVAL, "count < 0");
    if (count > 0 && !pairs) return fail(PEAT_EINVAL, "pairs is NULL");
    int rc = check_bins_thr(bins, thr);
    if (rc) return rc;
    for (int k = 0; k < count; ++k)
        if ((rc = check_mixed(pairs[k], k))) return rc;
    if (count == 0) return PEAT_OK;
    if (!host_outs && !d_outs) return fail(PEAT_EINVAL, "d_outs is NULL");

    std::lock_guard<std::mutex> lock(g_mu);
    Dev *dv;
    if ((rc = current_dev(&dv))) return rc;
    Dev &d = *dv;

    std::vector<SigDesc> descs;
    int64_t total = 0;
    int64_t range[kKinds + 1];
    if ((rc = build_descs(pairs, count, descs, range, &total))) return rc;

    // A lone pair without injection travels in the kernel arguments: nothing
    // to stage, and no copy ahead of the chunk pass.
    const bool single = count == 1 && !inj;
    const size_t b_desc = single ? 0 : align_up(sizeof(SigDesc) * count);
    const size_t b_inj = inj ? align_up(sizeof(InjDesc) * count) : 0;
    const size_t b_map = single ? 0 : align_up(sizeof(int32_t) * (size_t)total);
    const size_t b_part = align_up(sizeof(ChunkPartial) * (size_t)total);
    const size_t b_out = host_outs ? align_up(sizeof(peat_signature_t) * count) : 0;
    const size_t b_stage = b_desc + b_inj + b_map;

    // device workspace: descriptors | injection descriptors | chunk map |
    // chunk records; the first three are staged and copied at once.  A
    // synchronous call's records go straight to the pinned host slot behind
    // the staged part (the finalize writes them there: no copy afterwards).
    char *ws;
    if ((rc = acquire_ws(d, b_stage + b_part, s, &ws))) return rc;
    Slot *sl = nullptr;
    char *h = nullptr;
    if (b_stage + b_out > 0) {
        if ((rc = acquire_slot(d, b_stage + b_out, &sl))) return rc;
        h = static_cast<char *>(sl->host);
    }
    if (!single) {
        std::memcpy(h, descs.data(), sizeof(SigDesc) * count);
        if (inj) std::memcpy(h + b_desc, inj->data(), sizeof(InjDesc) * count);
        int32_t *hmap = reinterpret_cast<int32_t *>(h + b_desc + b_inj);
        for (int k = 0; k < count; ++k)
            for (int32_t c = 0; c < descs[k].nchunks; ++c) hmap[descs[k].first_chunk + c] = k;
        HIP_OR_FAIL(hipMemcpyAsync(ws, h, b_desc + b_inj + sizeof(int32_t) * (size_t)total, hipMemcpyHostToDevice, s));
    }

    SigParams P{};
    P.chunk_base = 0;
    P.single = single ? 1 : 0;
    P.gkeep = golden_reuse(pairs, count, [](const peat_mixed_pair_t &q) { return q.golden_dtype; });
    if (single) {
        P.one = descs[0];
    } else {
        P.descs = reinterpret_cast<const SigDesc *>(ws);
        P.chunk_pair = reinterpret_cast<const int32_t *>(ws + b_desc + b_inj);
    }
    P.partials = reinterpret_cast<ChunkPartial *>(ws + b_stage);
    P.outs = host_outs ? reinterpret_cast<peat_signature_t *>(h + b_stage) : d_outs;
    P.inj_counts = inj ? d_counts : nullptr;
    P.count = count;
    set_bins_thr(P, *bins, *thr);
    set_kind_elems(P, pairs, count);

    hipEvent_t ev;
    if ((rc = prof_begin(d, s, &ev))) return rc;
    if (inj)
        HIP_OR_FAIL(launch_sig_chunks_inject(P, range, reinterpret_cast<const InjDesc *>(ws + b_desc), s));
    else
        HIP_OR_FAIL(launch_sig_chunks(P, range, s));
    if ((rc = prof_end(d, s, inj ? 7 : 0, ev))) return rc;
    if ((rc = prof_begin(d, s, &ev))) return rc;
    HIP_OR_FAIL(launch_sig_finalize(P, s));
    if ((rc = prof_end(d, s, 1, ev))) return rc;

    char *hout = h ? h + b_stage : nullptr;
    if (sl && (rc = release_slot(*sl, s))) return rc;
    if ((rc = release_ws(d, s))) return rc;
    if (host_outs) {
        HIP_OR_FAIL(hipStreamSynchronize(s));
        std::memcpy(host_outs, hout, sizeof(peat_signature_t) * count);
    }
    return PEAT_OK;
}

int check_item(const peat_inject_item_t &it, int k) {
    if (check_dtype(it.dtype)) return fail(PEAT_EDTYPE, "item %d: unknown dtype %d", k, it.dtype);
    const int width = elem_size(it.dtype) * 8;
    if (it.model < PEAT_MODEL_BITFLIP || it.model > PEAT_MODEL_UNIFORM)
        return fail(PEAT_EINVAL, "item %d: unknown model %d", k, it.model);
    if (it.model == PEAT_MODEL_BITFLIP && (it.bitmask == 0 || (it.bitmask >> width) != 0))
        return fail(PEAT_EBITMASK, "item %d: bitmask 0x%llx is 0 or has bits at or above bit %d", k,
                    (unsigned long long)it.bitmask, width);
    if (std::isnan(it.rate) || it.rate < 0) return fail(PEAT_ERATE, "item %d: rate must be >= 0", k);
    if (it.n < 0) return fail(PEAT_EINVAL, "item %d: n < 0", k);
    if (it.n > 0 && !it.tensor) return fail(PEAT_EINVAL, "item %d: NULL tensor with n > 0", k);
    if (it.n > (int64_t(1) << 46)) return fail(PEAT_EINVAL, "item %d: n above 2^46", k);
    if (reinterpret_cast<uintptr_t>(it.tensor) % elem_size(it.dtype) != 0)
        return fail(PEAT_EINVAL, "item %d: tensor is not aligned to its element size", k);
    return PEAT_OK;
}

int inject_core(const peat_inject_item_t *items, int32_t count, int64_t *d_counts,
                int64_t *host_counts, hipStream_t s) {
    if (count < 0) return fail(PEAT_EINVAL, "count < 0");
    if (count > 0 && !items) return fail(PEAT_EINVAL, "items is NULL");
    int rc;
    for (int k = 0; k < count; ++k)
        if ((rc = check_item(items[k], k))) return rc;
    if (count == 0) return PEAT_OK;
    if (!host_counts && !d_counts) return fail(PEAT_EINVAL, "d_counts is NULL");

    std::lock_guard<std::mutex> lock(g_mu);
    Dev *dv;
    if ((rc = current_dev(&dv))) return rc;
    Dev &d = *dv;

    std::vector<InjDesc> descs((size_t)count);
    int64_t total = 0;
    for (int k = 0; k < count; ++k) {
        const peat_inject_item_t &it = items[k];
        InjDesc &q = descs[k];
        q.x = it.tensor;
        q.n = it.n;
        q.seed = it.seed;
        q.mask = it.model == PEAT_MODEL_BITFLIP ? it.bitmask : 1;
        q.dtype = it.dtype;
        q.popc = __builtin_popcountll(q.mask);
        q.model = it.model;
        q.src = nullptr;
        q.reserved = 0;
        q.all = it.rate >= 1.0;
        // T = floor(rate * 2^64): ldexp is exact and the conversion truncates
        q.T = (q.all || it.rate == 0.0) ? 0 : (uint64_t)std::ldexp(it.rate, 64);
        const bool none = !q.all && q.T == 0;
        const int64_t nseg = none ? 0 : (it.n + (int64_t(1) << kInjSegLog2) - 1) >> kInjSegLog2;
        q.first_seg = total;
        q.nsegs = (int32_t)nseg;
        total += nseg;
    }
    if (total > 0x7FFFFFFF) return fail(PEAT_EINVAL, "batch needs too many segments");

    const size_t b_desc = align_up(sizeof(InjDesc) * count);
    const size_t b_map = align_up(sizeof(int32_t) * (size_t)total);
    const size_t b_seg = align_up(sizeof(uint32_t) * (size_t)total);
    const size_t b_out = host_counts ? align_up(sizeof(int64_t) * count) : 0;
    // the random-value items read their sources from copies of their tensors
    // taken before the injection kernel writes anything
    std::vector<size_t> copy_off((size_t)count, 0);
    size_t b_copy = 0;
    for (int k = 0; k < count; ++k) {
        if (descs[k].model != PEAT_MODEL_VALUE || descs[k].nsegs == 0) continue;
        copy_off[k] = b_copy;
        b_copy += align_up((size_t)items[k].n * (size_t)elem_size(items[k].dtype));
    }
    const size_t o_copy = b_desc + b_map + b_seg + b_out;

    char *ws;
    if ((rc = acquire_ws(d, o_copy + b_copy, s, &ws))) return rc;
    for (int k = 0; k < count; ++k)
        if (descs[k].model == PEAT_MODEL_VALUE && descs[k].nsegs > 0) descs[k].src = ws + o_copy + copy_off[k];
    Slot *sl;
    if ((rc = acquire_slot(d, b_desc + b_map + b_out, &sl))) return rc;
    char *h = static_cast<char *>(sl->host);
    std::memcpy(h, descs.data(), sizeof(InjDesc) * count);
    int32_t *hmap = reinterpret_cast<int32_t *>(h + b_desc);
    for (int k = 0; k < count; ++k)
        for (int32_t c = 0; c < descs[k].nsegs; ++c) hmap[descs[k].first_seg + c] = k;
    HIP_OR_FAIL(hipMemcpyAsync(ws, h, b_desc + sizeof(int32_t) * (size_t)total, hipMemcpyHostToDevice, s));
    for (int k = 0; k < count; ++k)
        if (descs[k].model == PEAT_MODEL_VALUE && descs[k].nsegs > 0)
            HIP_OR_FAIL(hipMemcpyAsync(const_cast<void *>(descs[k].src), items[k].tensor,
                                       (size_t)items[k].n * (size_t)elem_size(items[k].dtype),
                                       hipMemcpyDeviceToDevice, s));

    InjParams P;
    P.descs = reinterpret_cast<const InjDesc *>(ws);
    P.seg_item = reinterpret_cast<const int32_t *>(ws + b_desc);
    P.seg_counts = reinterpret_cast<uint32_t *>(ws + b_desc + b_map);
    P.counts = host_counts ? reinterpret_cast<int64_t *>(ws + b_desc + b_map + b_seg) : d_counts;
    P.count = count;

    hipEvent_t ev;
    if ((rc = prof_begin(d, s, &ev))) return rc;
    HIP_OR_FAIL(launch_inject(P, total, s));
    if ((rc = prof_end(d, s, 2, ev))) return rc;
    if ((rc = prof_begin(d, s, &ev))) return rc;
    HIP_OR_FAIL(launch_inject_sum(P, s));
    if ((rc = prof_end(d, s, 3, ev))) return rc;

    char *hout = h + b_desc + b_map;
    if (host_counts)
        HIP_OR_FAIL(hipMemcpyAsync(hout, P.counts, sizeof(int64_t) * count, hipMemcpyDeviceToHost, s));
    if ((rc = release_slot(*sl, s))) return rc;
    if ((rc = release_ws(d, s))) return rc;
    if (host_counts) {
        HIP_OR_FAIL(hipStreamSynchronize(s));
        std::memcpy(host_counts, hout, sizeof(int64_t) * count);
    }
    return PEAT_OK;
}

// Whether the fused pass may inject the batch: every nonempty test tensor
// starts on a 128-byte cache line and no line that holds test bytes holds
// bytes of any other tensor of the batch.  Chunks are at least 4096 elements
// (8 KiB) long, so every chunk of such a tensor then covers whole lines that
// no other chunk, pair or block of the launch reads: the only load of a line
// that a block flips is that block's own, after its flips.  (The other
// caches' state at the start of the kernel is clean: the dispatch
// invalidates the compute units' L1 caches.)  A line shared with a chunk of
// another block could otherwise sit in the compute unit's L1 from that
// block's load, taken before the flip reached L2, and satisfy the later read
// with the old bits.
bool fused_lines_private(const peat_pair_t *pairs, int32_t count) {
    constexpr uintptr_t kLine = 128;
    struct Span { uintptr_t a, b; int test; };
    std::vector<Span> sp;
    sp.reserve(2 * (size_t)count);
    for (int k = 0; k < count; ++k) {
        if (pairs[k].n == 0) continue;
        const uintptr_t bytes = (uintptr_t)pairs[k].n * (uintptr_t)elem_size(pairs[k].dtype);
        const uintptr_t g = reinterpret_cast<uintptr_t>(pairs[k].golden);
        const uintptr_t t = reinterpret_cast<uintptr_t>(pairs[k].test);
        if (t % kLine != 0) return false;
        sp.push_back({g / kLine, (g + bytes + kLine - 1) / kLine, 0});
        sp.push_back({t / kLine, (t + bytes + kLine - 1) / kLine, 1});
    }
    std::sort(sp.begin(), sp.end(), [](const Span &x, const Span &y) { return x.a < y.a; });
    uintptr_t end_any = 0, end_test = 0;
    for (const Span &x : sp) {
        if (x.test && x.a < end_any) return false;     // a test line shared with an earlier span
        if (!x.test && x.a < end_test) return false;   // a golden line shared with an earlier test
        end_any = std::max(end_any, x.b);
        if (x.test) end_test = std::max(end_test, x.b);
    }
    return true;
}

// Injection and signature in one pass (same-type pairs, the bit-flip model):
// the records and flip counts of peat_inject_batched on the test tensors
// followed by peat_signature_batched.  Batches whose test tensors are not
// line-private (fused_lines_private) take the two launches instead.
int inject_signature_core(const peat_pair_t *pairs, int32_t count, const uint64_t *seeds, double rate,
                          uint64_t bitmask, const peat_bins_t *bins, const peat_thresholds_t *thr,
                          peat_signature_t *d_outs, int64_t *d_counts, hipStream_t s) {
    std::vector<peat_mixed_pair_t> mp;
    int rc = same_type_pairs(pairs, count, mp);
    if (rc) return rc;
    if ((rc = check_bins_thr(bins, thr))) return rc;
    if (std::isnan(rate) || rate < 0) return fail(PEAT_ERATE, "rate must be >= 0");
    if (count > 0 && !seeds) return fail(PEAT_EINVAL, "seeds is NULL");
    for (int k = 0; k < count; ++k) {
        const int width = elem_size(pairs[k].dtype) * 8;
        if (bitmask == 0 || (bitmask >> width) != 0)
            return fail(PEAT_EBITMASK, "pair %d: bitmask 0x%llx is 0 or has bits at or above bit %d", k,
                        (unsigned long long)bitmask, width);
    }
    // The flips go into the test tensors, which must not overlap one another
    // or any golden tensor of the batch (the result would depend on order).
    {
        struct Span { uintptr_t a, b; int test; int k; };
        std::vector<Span> sp;
        sp.reserve(2 * (size_t)count);
        for (int k = 0; k < count; ++k) {
            if (pairs[k].n == 0) continue;
            const uintptr_t es = (uintptr_t)elem_size(pairs[k].dtype);
            const uintptr_t g = reinterpret_cast<uintptr_t>(pairs[k].golden);
            const uintptr_t t = reinterpret_cast<uintptr_t>(pairs[k].test);
            sp.push_back({g, g + (uintptr_t)pairs[k].n * es, 0, k});
            sp.push_back({t, t + (uintptr_t)pairs[k].n * es, 1, k});
        }
        std::sort(sp.begin(), sp.end(), [](const Span &x, const Span &y) { return x.a < y.a; });
        // sweep: a test span may not intersect any other span
        uintptr_t end_any = 0, end_test = 0;
        int k_any = -1, k_test = -1;
        for (const Span &x : sp) {
            if (x.test && x.a < end_any)
                return fail(PEAT_EINVAL, "pair %d: test tensor overlaps a tensor of pair %d", x.k, k_any);
            if (!x.test && x.a < end_test)
                return fail(PEAT_EINVAL, "pair %d: test tensor overlaps the golden tensor of pair %d", k_test, x.k);
            if (x.b > end_any) { end_any = x.b; k_any = x.k; }
            if (x.test && x.b > end_test) { end_test = x.b; k_test = x.k; }
        }
    }
    if (count == 0) return PEAT_OK;
    if (!d_outs || !d_counts) return fail(PEAT_EINVAL, "d_outs or d_counts is NULL");
    if (!fused_lines_private(pairs, count)) {
        // Two launches: the injection kernel, then the signature pass; the
        // kernel boundary orders every flip before every read.
        std::vector<peat_inject_item_t> items((size_t)count);
        for (int k = 0; k < count; ++k)
            items[k] = peat_inject_item_t{const_cast<void *>(pairs[k].test), pairs[k].n, pairs[k].dtype,
                                          PEAT_MODEL_BITFLIP, seeds[k], rate, bitmask};
        if ((rc = inject_core(items.data(), count, d_counts, nullptr, s))) return rc;
        return signature_core(mp.data(), count, bins, thr, d_outs, nullptr, s);
    }
    std::vector<InjDesc> inj((size_t)count);
    for (int k = 0; k < count; ++k) {
        InjDesc &q = inj[k];
        std::memset(&q, 0, sizeof q);
        q.x = const_cast<void *>(pairs[k].test);
        q.n = pairs[k].n;
        q.seed = seeds[k];
        q.mask = bitmask;
        q.dtype = pairs[k].dtype;
        q.popc = __builtin_popcountll(bitmask);
        q.model = PEAT_MODEL_BITFLIP;
        q.all = rate >= 1.0;
        q.T = (q.all || rate == 0.0) ? 0 : (uint64_t)std::ldexp(rate, 64);
    }
    return signature_core(mp.data(), count, bins, thr, d_outs, nullptr, s, &inj, d_counts);
}

// Entries of the two top-k gather regions (binade gathers of pass A, bin
// gathers of pass C); -1: sized per call from its chunk count.
int64_t g_topk_cap[2] = {-1, -1};
constexpr int64_t kTopkCapMin = int64_t(1) << 16;
constexpr int64_t kTopkCapPerChunk[2] = {256, 64};
constexpr int kBins0Topk = 2048;         // binade field values (exact sums per binade)

// Mean of the k largest errors (see topk.hip): every step stream-ordered.
// With host_outs the records go through workspace + pinned staging and the
// call waits for them; otherwise they land in d_outs when the stream gets
// there.  host_sigs (validated here) or d_sigs (validated on the device: a
// record that does not match its pair is ignored) give level 0.
int topk_core(const peat_mixed_pair_t *pairs, int32_t count, int32_t num, int32_t den, peat_topk_t *host_outs,
              peat_topk_t *d_outs, hipStream_t s, const peat_signature_t *host_sigs = nullptr,
              const peat_signature_t *d_sigs = nullptr, const peat_bins_t *bins = nullptr) {
    if (count < 0) return fail(PEAT_EINVAL, "count < 0");
    if (count > 0 && !pairs) return fail(PEAT_EINVAL, "pairs is NULL");
    if (num < 1 || den < num || den > (1 << 20))
        return fail(PEAT_EINVAL, "need 1 <= num <= den <= 2^20 (got %d/%d)", num, den);
    int rc;
    for (int k = 0; k < count; ++k)
        if ((rc = check_mixed(pairs[k], k))) return rc;
    if (count == 0) return PEAT_OK;
    if (!host_outs && !d_outs) return fail(PEAT_EINVAL, "outs is NULL");
    if (host_sigs || d_sigs) {
        if (!bins) return fail(PEAT_EINVAL, "bins is NULL");
        if ((rc = check_bins(*bins))) return rc;
    }
    if (host_sigs) {
        for (int k = 0; k < count; ++k) {
            const peat_signature_t &g = host_sigs[k];
            int64_t tot = g.hist_zero + g.hist_under + g.hist_over;
            for (int i = 0; i < bins->nbins; ++i) tot += g.hist[i];
            if (g.n != pairs[k].n || tot != g.n_valid)
                return fail(PEAT_EINVAL, "signature %d does not match pair %d and these bins (n %lld vs %lld, "
                            "histogram total %lld vs n_valid %lld)", k, k, (long long)g.n, (long long)pairs[k].n,
                            (long long)tot, (long long)g.n_valid);
        }
    }

    std::lock_guard<std::mutex> lock(g_mu);
    Dev *dv;
    if ((rc = current_dev(&dv))) return rc;
    Dev &d = *dv;

    std::vector<SigDesc> descs;
    int64_t total = 0;
    int64_t range[kKinds + 1];
    if ((rc = build_descs(pairs, count, descs, range, &total))) return rc;

    uint64_t cap[2];
    for (int r = 0; r < 2; ++r) {
        const int64_t c = g_topk_cap[r] >= 0 ? g_topk_cap[r] : std::max(kTopkCapMin, kTopkCapPerChunk[r] * total);
        cap[r] = (uint64_t)c;
    }
    const size_t b_desc = align_up(sizeof(SigDesc) * count);
    const size_t b_map = align_up(sizeof(int32_t) * (size_t)total);
    const size_t b_sig = host_sigs ? align_up(sizeof(peat_signature_t) * count) : 0;
    const size_t b_out = host_outs ? align_up(sizeof(peat_topk_t) * count) : 0;
    const size_t b_state = align_up(sizeof(TopkState) * count);
    const size_t b_hist = align_up(sizeof(uint64_t) * kTopkBins * (size_t)count);
    const size_t b_part = align_up(sizeof(double) * (size_t)total);
    const size_t b_xsum = align_up(2 * sizeof(uint64_t) * kBins0Topk * (size_t)count);
    const size_t b_ovf = align_up(sizeof(uint32_t) * (2 * (size_t)count + 3));
    const size_t b_cnt = align_up(2 * sizeof(uint64_t) * count);
    const size_t b_fill = align_up(2 * sizeof(unsigned long long));
    const size_t b_ents = align_up(sizeof(TopkEntry) * (size_t)(cap[0] + cap[1]));
    // device workspace: descriptors | chunk map | signatures | records (the
    // first three staged and copied as they lie) | state | histograms | chunk
    // sums | exact sums | flags | counts | fills | entries
    const size_t o_map = b_desc, o_sig = o_map + b_map, o_out = o_sig + b_sig, o_state = o_out + b_out;
    const size_t o_hist = o_state + b_state, o_part = o_hist + b_hist, o_xsum = o_part + b_part;
    const size_t o_ovf = o_xsum + b_xsum, o_cnt = o_ovf + b_ovf, o_fill = o_cnt + b_cnt, o_ents = o_fill + b_fill;

    char *ws;
    if ((rc = acquire_ws(d, o_ents + b_ents, s, &ws))) return rc;
    Slot *sl;
    if ((rc = acquire_slot(d, o_state, &sl))) return rc;
    char *h = static_cast<char *>(sl->host);
    std::memcpy(h, descs.data(), sizeof(SigDesc) * count);
    int32_t *hmap = reinterpret_cast<int32_t *>(h + o_map);
    for (int k = 0; k < count; ++k)
        for (int32_t c = 0; c < descs[k].nchunks; ++c) hmap[descs[k].first_chunk + c] = k;
    if (host_sigs) std::memcpy(h + o_sig, host_sigs, sizeof(peat_signature_t) * count);
    HIP_OR_FAIL(hipMemcpyAsync(ws, h, o_out, hipMemcpyHostToDevice, s));

    TopkParams P{};
    P.descs = reinterpret_cast<const SigDesc *>(ws);
    P.chunk_pair = reinterpret_cast<const int32_t *>(ws + o_map);
    P.state = reinterpret_cast<TopkState *>(ws + o_state);
    P.hist = reinterpret_cast<uint64_t *>(ws + o_hist);
    P.part_a = reinterpret_cast<double *>(ws + o_part);
    P.xsum = reinterpret_cast<uint64_t *>(ws + o_xsum);
    P.ovf = reinterpret_cast<uint32_t *>(ws + o_ovf);
    P.counts = reinterpret_cast<uint64_t *>(ws + o_cnt);
    P.fill = reinterpret_cast<unsigned long long *>(ws + o_fill);
    P.ents = reinterpret_cast<TopkEntry *>(ws + o_ents);
    P.cap[0] = cap[0];
    P.cap[1] = cap[1];
    P.sigs = host_sigs ? reinterpret_cast<const peat_signature_t *>(ws + o_sig) : d_sigs;
    P.outs = host_outs ? reinterpret_cast<peat_topk_t *>(ws + o_out) : d_outs;
    if (bins) {
        P.lo = bins->lo_log2;
        P.hi = bins->hi_log2;
        P.nbins = bins->nbins;
    }
    P.count = count;
    P.num = num;
    P.den = den;

    hipEvent_t ev;
    if ((rc = prof_begin(d, s, &ev))) return rc;
    HIP_OR_FAIL(launch_topk_level0(P, range, s));
    if ((rc = prof_end(d, s, 5, ev))) return rc;
    if ((rc = prof_begin(d, s, &ev))) return rc;
    HIP_OR_FAIL(launch_topk_rest(P, range, s));
    if ((rc = prof_end(d, s, 6, ev))) return rc;

    char *hout = h + o_out;
    if (host_outs)
        HIP_OR_FAIL(hipMemcpyAsync(hout, P.outs, sizeof(peat_topk_t) * count, hipMemcpyDeviceToHost, s));
    if ((rc = release_slot(*sl, s))) return rc;
    if ((rc = release_ws(d, s))) return rc;
    if (host_outs) {
        HIP_OR_FAIL(hipStreamSynchronize(s));
        std::memcpy(host_outs, hout, sizeof(peat_topk_t) * count);
    }
    return PEAT_OK;
}

// ---- signatures without allocation -------------------------------------------
// Pair descriptors reach the scratch array as kernel arguments, kFillDescs per
// launch (the launch copies its arguments, so no host buffer has to outlive
// the call and nothing is staged through pinned memory); each block writes
// one descriptor and its pair's entries of the chunk map.
constexpr int kFillDescs = 32;
struct DescBatch {
    SigDesc d[kFillDescs];
    int32_t first;                   // pair index of d[0]
    int32_t count;                   // descriptors used
};

__global__ void __launch_bounds__(kBlock) noalloc_fill(DescBatch b, SigDesc *descs, int32_t *chunk_pair) {
    const int j = blockIdx.x;
    if (j >= b.count) return;
    const SigDesc &sd = b.d[j];
    if (threadIdx.x == 0) descs[b.first + j] = sd;
    for (int32_t c = threadIdx.x; c < sd.nchunks; c += kBlock) chunk_pair[sd.first_chunk + c] = b.first + j;
}

// peat_signature_batched_async with every intermediate buffer in `scratch`:
// descriptors | chunk map | chunk records.  Host work is validation, two
// scans over the pairs and the launches; no heap, pinned or device memory is
// allocated (the device's one-time set-up in current_dev aside).  The chunk
// records need no clearing: the chunk pass writes every field the finalize
// reads, so what a previous call left in the array does not matter.
int signature_noalloc_core(const peat_pair_t *pairs, int32_t count, const peat_bins_t *bins,
                           const peat_thresholds_t *thr, peat_signature_t *d_outs, hipStream_t s) {
    if (count < 0) return fail(PEAT_EINVAL, "count < 0");
    if (count > 0 && !pairs) return fail(PEAT_EINVAL, "pairs is NULL");
    int rc = check_bins_thr(bins, thr);
    if (rc) return rc;
    // scan 1: validation and the chunks of each kind and chunk class
    // (same-type kinds only; the classes ordered as build_descs orders them)
    constexpr int kClasses = kMaxChunkLog2 - kMinChunkLog2 + 1;
    int64_t per_class[kKinds * kClasses] = {};
    for (int k = 0; k < count; ++k) {
        if ((rc = check_pair(pairs[k], k))) return rc;
        const int64_t n = pairs[k].n;
        const int lg = chunk_log2_for(n);
        per_class[pair_kind(pairs[k].dtype, pairs[k].dtype) * kClasses + (kMaxChunkLog2 - lg)] +=
            (n + (int64_t(1) << lg) - 1) >> lg;
    }
    if (count == 0) return PEAT_OK;
    if (!d_outs) return fail(PEAT_EINVAL, "d_outs is NULL");
    int64_t range[kKinds + 1];
    int64_t cursor[kKinds * kClasses];
    int64_t total = 0;
    for (int kind = 0; kind < kKinds; ++kind) {
        range[kind] = total;
        for (int c = 0; c < kClasses; ++c) {
            cursor[kind * kClasses + c] = total;
            total += per_class[kind * kClasses + c];
        }
    }
    range[kKinds] = total;
    const size_t b_desc = align_up(sizeof(SigDesc) * (size_t)count);
    const size_t b_map = align_up(sizeof(int32_t) * (size_t)total);
    const size_t need = b_desc + b_map + sizeof(ChunkPartial) * (size_t)total;
    if (total > 0x7FFFFFFF || need > (size_t)PEAT_NOALLOC_SCRATCH_BYTES)
        return fail(PEAT_EINVAL, "batch needs %zu bytes of scratch (%lld chunks, %d pairs); the maximum is %zu",
                    need, (long long)total, count, (size_t)PEAT_NOALLOC_SCRATCH_BYTES);

    std::lock_guard<std::mutex> lock(g_mu);
    Dev *dv;
    if ((rc = current_dev(&dv))) return rc;
    char *ws = dv->scratch;
    SigDesc *d_desc = reinterpret_cast<SigDesc *>(ws);
    int32_t *d_map = reinterpret_cast<int32_t *>(ws + b_desc);

    // scan 2: descriptors, in pair order, numbered by kind and chunk class
    // as build_descs numbers them
    DescBatch b;
    std::memset(&b, 0, sizeof b);
    b.first = 0;
    for (int k = 0; k < count; ++k) {
        SigDesc &sd = b.d[b.count++];
        const int kind = pair_kind(pairs[k].dtype, pairs[k].dtype);
        sd.g = pairs[k].golden;
        sd.t = pairs[k].test;
        sd.n = pairs[k].n;
        sd.dtype = (int16_t)pairs[k].dtype;
        sd.tdtype = (int16_t)pairs[k].dtype;
        sd.chunk_log2 = chunk_log2_for(sd.n);
        sd.nchunks = (int32_t)((sd.n + (int64_t(1) << sd.chunk_log2) - 1) >> sd.chunk_log2);
        int64_t &cur = cursor[kind * kClasses + (kMaxChunkLog2 - sd.chunk_log2)];
        sd.first_chunk = cur;
        cur += sd.nchunks;
        sd.aligned = ((reinterpret_cast<uintptr_t>(sd.g) | reinterpret_cast<uintptr_t>(sd.t)) & 15) == 0;
        if (b.count == kFillDescs || k + 1 == count) {
            hipLaunchKernelGGL(noalloc_fill, dim3((unsigned)b.count), dim3(kBlock), 0, s, b, d_desc, d_map);
            HIP_OR_FAIL(hipGetLastError());
            std::memset(&b, 0, sizeof b);
            b.first = k + 1;
        }
    }

    SigParams P{};
    P.chunk_base = 0;
    P.chunk_count = 0;
    P.chunk_group = 1;
    P.descs = d_desc;
    P.chunk_pair = d_map;
    P.partials = reinterpret_cast<ChunkPartial *>(ws + b_desc + b_map);
    P.outs = d_outs;
    P.inj_counts = nullptr;
    P.count = count;
    P.gkeep = golden_reuse(pairs, count, [](const peat_pair_t &q) { return q.dtype; });
    set_bins_thr(P, *bins, *thr);
    for (int k = 0; k < count; ++k) P.kind_elems[pair_kind(pairs[k].dtype, pairs[k].dtype)] += pairs[k].n;
    HIP_OR_FAIL(launch_sig_chunks(P, range, s));
    HIP_OR_FAIL(launch_sig_finalize(P, s));
    return PEAT_OK;
}

}  // namespace

extern "C" {

const char *peat_strerror(int code) {
    switch (code) {
        case PEAT_OK: return "success";
        case PEAT_EINVAL: return "invalid argument";
        case PEAT_EDTYPE: return "unknown element type";
        case PEAT_EBITMASK: return "bitmask is zero or wider than the element type";
        case PEAT_ERATE: return "injection rate is NaN or negative";
        case PEAT_EHIP: return "HIP runtime error";
        case PEAT_ENOMEM: return "out of memory";
        case PEAT_ENODEV: return "no gfx950 device";
        default: return "unknown error code";
    }
}

const char *peat_last_error(void) { return t_err.c_str(); }

int peat_abi_version(void) { return PEAT_ABI_VERSION; }

int peat_init(void) {
    std::lock_guard<std::mutex> lock(g_mu);
    Dev *d;
    return current_dev(&d);
}

int peat_set_stream(void *stream) {
    t_stream = static_cast<hipStream_t>(stream);
    return PEAT_OK;
}

int peat_signature(const void *golden, const void *test, int64_t n, peat_dtype_t dtype,
                   const peat_bins_t *bins, const peat_thresholds_t *thresholds,
                   peat_signature_t *out) {
    if (!out) return fail(PEAT_EINVAL, "out is NULL");
    peat_pair_t p{golden, test, n, (int32_t)dtype, 0};
    std::vector<peat_mixed_pair_t> mp;
    int rc = same_type_pairs(&p, 1, mp);
    if (rc) return rc;
    return signature_core(mp.data(), 1, bins, thresholds, nullptr, out, t_stream);
}

int peat_signature_batched(const peat_pair_t *pairs, int32_t count, const peat_bins_t *bins,
                           const peat_thresholds_t *thresholds, peat_signature_t *outs) {
    if (count > 0 && !outs) return fail(PEAT_EINVAL, "outs is NULL");
    std::vector<peat_mixed_pair_t> mp;
    int rc = same_type_pairs(pairs, count, mp);
    if (rc) return rc;
    return signature_core(mp.data(), count, bins, thresholds, nullptr, outs, t_stream);
}

int peat_signature_batched_async(const peat_pair_t *pairs, int32_t count, const peat_bins_t *bins,
                                 const peat_thresholds_t *thresholds, peat_signature_t *d_outs,
                                 void *stream) {
    std::vector<peat_mixed_pair_t> mp;
    int rc = same_type_pairs(pairs, count, mp);
    if (rc) return rc;
    return signature_core(mp.data(), count, bins, thresholds, d_outs, nullptr,
                          static_cast<hipStream_t>(stream));
}

int peat_signature_batched_noalloc(const peat_pair_t *pairs, int32_t count, const peat_bins_t *bins,
                                   const peat_thresholds_t *thresholds, peat_signature_t *d_outs, void *stream) {
    return signature_noalloc_core(pairs, count, bins, thresholds, d_outs, static_cast<hipStream_t>(stream));
}

int peat_inject_signature_batched_async(const peat_pair_t *pairs, int32_t count, const uint64_t *seeds,
                                        double rate, uint64_t bitmask, const peat_bins_t *bins,
                                        const peat_thresholds_t *thresholds, peat_signature_t *d_outs,
                                        int64_t *d_counts, void *stream) {
    return inject_signature_core(pairs, count, seeds, rate, bitmask, bins, thresholds, d_outs, d_counts,
                                 static_cast<hipStream_t>(stream));
}

int peat_signature_mixed(const void *golden, int32_t golden_dtype, const void *test, int32_t test_dtype,
                         int64_t n, const peat_bins_t *bins, const peat_thresholds_t *thresholds,
                         peat_signature_t *out) {
    if (!out) return fail(PEAT_EINVAL, "out is NULL");
    peat_mixed_pair_t p{golden, test, n, golden_dtype, test_dtype};
    return signature_core(&p, 1, bins, thresholds, nullptr, out, t_stream);
}

int peat_signature_mixed_batched(const peat_mixed_pair_t *pairs, int32_t count, const peat_bins_t *bins,
                                 const peat_thresholds_t *thresholds, peat_signature_t *outs) {
    if (count > 0 && !outs) return fail(PEAT_EINVAL, "outs is NULL");
    return signature_core(pairs, count, bins, thresholds, nullptr, outs, t_stream);
}

int peat_signature_mixed_batched_async(const peat_mixed_pair_t *pairs, int32_t count, const peat_bins_t *bins,
                                       const peat_thresholds_t *thresholds, peat_signature_t *d_outs,
                                       void *stream) {
    return signature_core(pairs, count, bins, thresholds, d_outs, nullptr, static_cast<hipStream_t>(stream));
}

int64_t peat_inject(void *tensor, int64_t n, peat_dtype_t dtype, uint64_t seed, double rate,
                    uint64_t bitmask) {
    peat_inject_item_t it{tensor, n, (int32_t)dtype, PEAT_MODEL_BITFLIP, seed, rate, bitmask};
    int64_t c = 0;
    int rc = inject_core(&it, 1, nullptr, &c, t_stream);
    return rc ? rc : c;
}

int64_t peat_inject_model(void *tensor, int64_t n, peat_dtype_t dtype, uint64_t seed, double rate,
                          int32_t model, uint64_t bitmask) {
    peat_inject_item_t it{tensor, n, (int32_t)dtype, model, seed, rate, bitmask};
    int64_t c = 0;
    int rc = inject_core(&it, 1, nullptr, &c, t_stream);
    return rc ? rc : c;
}

int64_t peat_corrupt_positions(void *tensor, int64_t n, peat_dtype_t dtype, uint64_t seed, int32_t model,
                               int64_t num_pos, uint64_t bitmask, int64_t *positions) {
    if (check_dtype(dtype)) return fail(PEAT_EDTYPE, "unknown dtype %d", (int)dtype);
    if (model < PEAT_MODEL_BITFLIP || model > PEAT_MODEL_UNIFORM) return fail(PEAT_EINVAL, "unknown model %d", model);
    const int width = elem_size(dtype) * 8;
    if (model == PEAT_MODEL_BITFLIP && (bitmask == 0 || (bitmask >> width) != 0))
        return fail(PEAT_EBITMASK, "bitmask 0x%llx is 0 or has bits at or above bit %d",
                    (unsigned long long)bitmask, width);
    if (n < 0 || n > (int64_t(1) << 46)) return fail(PEAT_EINVAL, "n must be in [0, 2^46]");
    if (num_pos < 0 || num_pos > n || num_pos > PEAT_MAX_POSITIONS)
        return fail(PEAT_EINVAL, "num_pos must be in [0, min(n, %d)] (got %lld)", PEAT_MAX_POSITIONS,
                    (long long)num_pos);
    if (num_pos == 0) return 0;
    if (!tensor) return fail(PEAT_EINVAL, "tensor is NULL");
    if (reinterpret_cast<uintptr_t>(tensor) % elem_size(dtype) != 0)
        return fail(PEAT_EINVAL, "tensor is not aligned to its element size");
    std::lock_guard<std::mutex> lock(g_mu);
    Dev *dv;
    int rc = current_dev(&dv);
    if (rc) return rc;
    Dev &d = *dv;
    hipStream_t s = t_stream;
    char *ws;
    if ((rc = acquire_ws(d, sizeof(int64_t) * PEAT_MAX_POSITIONS, s, &ws))) return rc;
    Slot *sl;
    if ((rc = acquire_slot(d, sizeof(int64_t) * PEAT_MAX_POSITIONS, &sl))) return rc;
    int64_t *dpos = reinterpret_cast<int64_t *>(ws);
    HIP_OR_FAIL(launch_corrupt_positions(tensor, n, dtype, seed, model, num_pos, bitmask, dpos, s));
    HIP_OR_FAIL(hipMemcpyAsync(sl->host, dpos, sizeof(int64_t) * num_pos, hipMemcpyDeviceToHost, s));
    if ((rc = release_slot(*sl, s))) return rc;
    if ((rc = release_ws(d, s))) return rc;
    HIP_OR_FAIL(hipStreamSynchronize(s));
    const int64_t *hp = static_cast<const int64_t *>(sl->host);
    if (hp[0] < 0) return fail(PEAT_EHIP, "position draw limit reached before %lld distinct positions", (long long)num_pos);
    if (positions) std::memcpy(positions, hp, sizeof(int64_t) * num_pos);
    return num_pos;
}

int peat_cast_round(void *tensor, int64_t n, peat_dtype_t to_dtype) {
    if (to_dtype != PEAT_F16 && to_dtype != PEAT_BF16)
        return fail(PEAT_EDTYPE, "to_dtype must be PEAT_F16 or PEAT_BF16 (got %d)", (int)to_dtype);
    if (n < 0) return fail(PEAT_EINVAL, "n < 0");
    if (n == 0) return PEAT_OK;
    if (!tensor) return fail(PEAT_EINVAL, "tensor is NULL");
    if (reinterpret_cast<uintptr_t>(tensor) % 4 != 0) return fail(PEAT_EINVAL, "tensor is not 4-byte aligned");
    std::lock_guard<std::mutex> lock(g_mu);
    Dev *dv;
    int rc = current_dev(&dv);
    if (rc) return rc;
    HIP_OR_FAIL(launch_cast_round(tensor, n, to_dtype, t_stream));
    return PEAT_OK;
}

int peat_inject_batched(const peat_inject_item_t *items, int32_t count, int64_t *counts) {
    if (count > 0 && !counts) return fail(PEAT_EINVAL, "counts is NULL");
    return inject_core(items, count, nullptr, counts, t_stream);
}

int peat_inject_batched_async(const peat_inject_item_t *items, int32_t count, int64_t *d_counts,
                              void *stream) {
    return inject_core(items, count, d_counts, nullptr, static_cast<hipStream_t>(stream));
}

int peat_topk_mean(const void *golden, const void *test, int64_t n, peat_dtype_t dtype, int32_t num,
                   int32_t den, peat_topk_t *out) {
    if (!out) return fail(PEAT_EINVAL, "out is NULL");
    peat_pair_t p{golden, test, n, (int32_t)dtype, 0};
    std::vector<peat_mixed_pair_t> mp;
    int rc = same_type_pairs(&p, 1, mp);
    if (rc) return rc;
    return topk_core(mp.data(), 1, num, den, out, nullptr, t_stream);
}

int peat_topk_mean_batched(const peat_pair_t *pairs, int32_t count, int32_t num, int32_t den,
                           peat_topk_t *outs) {
    std::vector<peat_mixed_pair_t> mp;
    int rc = same_type_pairs(pairs, count, mp);
    if (rc) return rc;
    if (count > 0 && !outs) return fail(PEAT_EINVAL, "outs is NULL");
    return topk_core(mp.data(), count, num, den, outs, nullptr, t_stream);
}

int peat_topk_mean_batched_async(const peat_pair_t *pairs, int32_t count, int32_t num, int32_t den,
                                 peat_topk_t *d_outs, void *stream) {
    std::vector<peat_mixed_pair_t> mp;
    int rc = same_type_pairs(pairs, count, mp);
    if (rc) return rc;
    if (count > 0 && !d_outs) return fail(PEAT_EINVAL, "d_outs is NULL");
    return topk_core(mp.data(), count, num, den, nullptr, d_outs, static_cast<hipStream_t>(stream));
}

int peat_topk_mean_mixed_batched(const peat_mixed_pair_t *pairs, int32_t count, int32_t num, int32_t den,
                                 peat_topk_t *outs) {
    if (count > 0 && !outs) return fail(PEAT_EINVAL, "outs is NULL");
    return topk_core(pairs, count, num, den, outs, nullptr, t_stream);
}

int peat_topk_mean_mixed_batched_async(const peat_mixed_pair_t *pairs, int32_t count, int32_t num, int32_t den,
                                       peat_topk_t *d_outs, void *stream) {
    if (count > 0 && !d_outs) return fail(PEAT_EINVAL, "d_outs is NULL");
    return topk_core(pairs, count, num, den, nullptr, d_outs, static_cast<hipStream_t>(stream));
}

int peat_topk_mean_from_signature_batched(const peat_pair_t *pairs, int32_t count, int32_t num, int32_t den,
                                          const peat_signature_t *sigs, const peat_bins_t *bins,
                                          peat_topk_t *outs) {
    if (count > 0 && !sigs) return fail(PEAT_EINVAL, "sigs is NULL");
    std::vector<peat_mixed_pair_t> mp;
    int rc = same_type_pairs(pairs, count, mp);
    if (rc) return rc;
    if (count > 0 && !outs) return fail(PEAT_EINVAL, "outs is NULL");
    return topk_core(mp.data(), count, num, den, outs, nullptr, t_stream, sigs, nullptr, bins);
}

int peat_topk_mean_from_signature_batched_async(const peat_pair_t *pairs, int32_t count, int32_t num,
                                                int32_t den, const peat_signature_t *d_sigs,
                                                const peat_bins_t *bins, peat_topk_t *d_outs, void *stream) {
    if (count > 0 && !d_sigs) return fail(PEAT_EINVAL, "d_sigs is NULL");
    std::vector<peat_mixed_pair_t> mp;
    int rc = same_type_pairs(pairs, count, mp);
    if (rc) return rc;
    if (count > 0 && !d_outs) return fail(PEAT_EINVAL, "d_outs is NULL");
    return topk_core(mp.data(), count, num, den, nullptr, d_outs, static_cast<hipStream_t>(stream), nullptr,
                     d_sigs, bins);
}

int peat_topk_mean_mixed_from_signature_batched(const peat_mixed_pair_t *pairs, int32_t count, int32_t num,
                                                int32_t den, const peat_signature_t *sigs,
                                                const peat_bins_t *bins, peat_topk_t *outs) {
    if (count > 0 && !sigs) return fail(PEAT_EINVAL, "sigs is NULL");
    if (count > 0 && !outs) return fail(PEAT_EINVAL, "outs is NULL");
    return topk_core(pairs, count, num, den, outs, nullptr, t_stream, sigs, nullptr, bins);
}

int peat_topk_mean_mixed_from_signature_batched_async(const peat_mixed_pair_t *pairs, int32_t count,
                                                      int32_t num, int32_t den, const peat_signature_t *d_sigs,
                                                      const peat_bins_t *bins, peat_topk_t *d_outs,
                                                      void *stream) {
    if (count > 0 && !d_sigs) return fail(PEAT_EINVAL, "d_sigs is NULL");
    if (count > 0 && !d_outs) return fail(PEAT_EINVAL, "d_outs is NULL");
    return topk_core(pairs, count, num, den, nullptr, d_outs, static_cast<hipStream_t>(stream), nullptr, d_sigs,
                     bins);
}

int peat_topk_set_entry_capacity(int64_t binade_entries, int64_t bin_entries) {
    if (binade_entries < -1 || bin_entries < -1 || binade_entries > (int64_t(1) << 36) ||
        bin_entries > (int64_t(1) << 36))
        return fail(PEAT_EINVAL, "capacities must be -1 or in [0, 2^36]");
    std::lock_guard<std::mutex> lock(g_mu);
    g_topk_cap[0] = binade_entries;
    g_topk_cap[1] = bin_entries;
    return PEAT_OK;
}

int peat_stream_read(const void *buf, int64_t bytes, uint32_t *d_sink, void *stream) {
    if (bytes < 0) return fail(PEAT_EINVAL, "bytes < 0");
    if (bytes == 0) return PEAT_OK;
    if (!buf || !d_sink) return fail(PEAT_EINVAL, "NULL pointer with bytes > 0");
    if (bytes % 16 != 0 || reinterpret_cast<uintptr_t>(buf) % 16 != 0)
        return fail(PEAT_EINVAL, "buf must be 16-byte aligned and bytes a multiple of 16");
    if (reinterpret_cast<uintptr_t>(d_sink) % 4 != 0) return fail(PEAT_EINVAL, "d_sink must be 4-byte aligned");
    std::lock_guard<std::mutex> lock(g_mu);
    Dev *d;
    int rc = current_dev(&d);
    if (rc) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipEvent_t ev;
    if ((rc = prof_begin(*d, s, &ev))) return rc;
    HIP_OR_FAIL(launch_stream_read(buf, bytes, d_sink, s));
    return prof_end(*d, s, 4, ev);
}

int peat_finalize_stats(const peat_signature_t *sg, peat_stats_t *st) {
    if (!sg || !st) return fail(PEAT_EINVAL, "NULL argument");
    const double nf = (double)sg->n_finite;
    st->mean_abs = sg->n_finite > 0 ? sg->sum_abs / nf : NAN;
    // sample variance of the absolute error over finite pairs
    st->var_abs = sg->n_finite > 1 ? (sg->sum_sq - sg->sum_abs * (sg->sum_abs / nf)) / (nf - 1.0) : NAN;
    st->l2_err = std::sqrt(sg->sum_sq);
    st->l2_g = std::sqrt(sg->sum_g2);
    st->l2_t = std::sqrt(sg->sum_t2);
    st->cos = (sg->sum_g2 > 0 && sg->sum_t2 > 0) ? sg->sum_gt / std::sqrt(sg->sum_g2 * sg->sum_t2) : NAN;
    st->mean_rel = sg->n_rel > 0 ? sg->sum_rel / (double)sg->n_rel : NAN;
    st->mean_ulp = sg->n_valid > 0 ? (double)sg->sum_ulp / (double)sg->n_valid : NAN;
    return PEAT_OK;
}

int peat_profile_enable(int on) {
    std::lock_guard<std::mutex> lock(g_mu);
    Dev *d;
    int rc = current_dev(&d);
    if (rc) return rc;
    d->prof = on != 0;
    return PEAT_OK;
}

int peat_profile_read(int kernel_class, double *total_ms, int64_t *launches) {
    if (!total_ms || !launches) return fail(PEAT_EINVAL, "NULL argument");
    std::lock_guard<std::mutex> lock(g_mu);
    Dev *d;
    int rc = current_dev(&d);
    if (rc) return rc;
    double sum = 0.0;
    int64_t cnt = 0;
    std::vector<ProfRec> keep;
    for (const ProfRec &r : d->log) {
        if (r.cls != kernel_class) {
            keep.push_back(r);
            continue;
        }
        HIP_OR_FAIL(hipEventSynchronize(r.b));
        float ms = 0.f;
        HIP_OR_FAIL(hipEventElapsedTime(&ms, r.a, r.b));
        sum += ms;
        ++cnt;
        d->pool.push_back(r.a);
        d->pool.push_back(r.b);
    }
    d->log.swap(keep);
    *total_ms = sum;
    *launches = cnt;
    return PEAT_OK;
}

}  // extern "C"
