#!/usr/bin/env python3
"""Throughput of the error-signature hot path on one MI355X.

One step is one pass of the whole hot path over one batch of synthetic input
resident in HBM: the bit-flip injection into every test tensor (fresh seeds
each step) and the error signature of every (golden, test) pair.  Where every
test tensor is injected with one rate and mask (the default workload) the
step is one call, peat_inject_signature_batched_async, which injects each
chunk and then signs it in the same kernel; the same step as two calls
(injection, then signature) is timed after it for reference (--separate makes
the two calls the timed step).  The default workload is the Llama-7B-shaped
checkpoint pair (weights plus both Adam moments: 873 f32 tensors,
20,215,246,848 elements per side, 161.72 GB signed per step).

Prints ONE JSON line on stdout (everything else goes to stderr):
  value     golden+test bytes signed per second over the timed steps (GB/s)
  roofline  the dominant kernel (the chunk pass, with the injection when the
            step is fused): algorithmic bytes per launch / its average launch
            duration from HIP events on its stream, against the 8 TB/s HBM
            peak; traffic from the committed rocprofv3 counter summary when it
            was taken on the current kernel source
  cpu_baseline  the CPU oracle on a bounded sample of the same workload, in
            equal element slices over the host share of one GPU (16 cores)
  other_workloads  the other paper-shaped workloads (activations with bf16
            rounding, the GPT-1.3B checkpoint, the 1000-call f16 replay), one
            step each (their injections, then the batched signature), each
            with its chunk pass's fraction of the HBM peak

Also reported: the read ceiling of the same box (peat_stream_read over a
16 GiB buffer with the chunk pass's access pattern) and the signature chunk
pass as a fraction of it; per-step times (median, min, max); the top-10%
error mean of the workload; single-call latencies (a 1024x1024 f32 pair
warm and cold, one f16 [4096, 4096] replay call); the signature of
mixed-precision pairs (FP32 golden against FP64 and FP16 outputs).

Modes used to produce the committed profiles: --copy-calibration (a plain
device copy of known size, for scaling the HBM byte counters), --mixed-only
(the mixed-precision measurement alone).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "GB/s of golden+test tensor bytes signed (fraction of HBM peak), 1 MI355X"
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2609_13544_amd", "csrc", f)
                  for f in ("sig_chunk.h", "signature.hip", "elements.h", "peat_internal.h", "inject_span.h",
                            "philox.h")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """sha256[:16] of the chunk pass's sources with comments and blank space
    removed (a comment edit does not change the kernel)."""
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(p) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def committed_traffic(workload: str, fused: bool = False):
    """HBM bytes per launch of the chunk pass (with the injection when fused)
    from profiles/, or None when the counters were taken on a different
    kernel source."""
    kernel = "sig_chunk_inject" if fused else "sig_chunk"
    path = os.path.join(PROFILES, f"{kernel}_{workload}_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"kernel_source_sha256_16:\s*`?([0-9a-f]{16})", text)
    m_val = re.search(r"traffic_bytes_per_launch:\s*`?([0-9.eE+]+)", text)
    if not m_hash or not m_val or m_hash.group(1) != kernel_source_hash():
        return None
    return float(m_val.group(1))


# ---------------------------------------------------------------------------
# workloads
# ---------------------------------------------------------------------------
class Workload:
    name = ""
    description = ""
    roofline_note = ""

    def __init__(self, torch, P, synth):
        self.torch, self.P, self.synth = torch, P, synth
        self.pairs = []          # (G, T) device tensors
        self.items = []          # (T, base_seed, rate, mask) injected each step
        self.sample = []         # indices of pairs for the CPU baseline

    def inject_items(self, step: int):
        return [(T, (seed + (step << 40)) & (2 ** 64 - 1), rate, mask) for T, seed, rate, mask in self.items]

    def fusable(self) -> bool:
        """Every pair's test tensor is injected, in pair order, with one rate
        and mask: the step can be the fused injection + signature call."""
        return (len(self.items) == len(self.pairs) > 0
                and all(T is t for (T, *_), (_, t) in zip(self.items, self.pairs))
                and len({(r, m) for _, _, r, m in self.items}) == 1)

    def bytes_signed(self) -> int:
        return sum(G.numel() * G.element_size() * 2 for G, _ in self.pairs)

    def elements(self) -> int:
        return sum(G.numel() for G, _ in self.pairs)


class Llama7B(Workload):
    name = "llama7b_ckpt_adam"
    description = ("Llama-7B-shaped checkpoint pair: weights + Adam m + Adam v, 873 f32 tensors, "
                   "T = G*(1+1e-7 z) with 1e-8-rate exponent-bit flips")

    def __init__(self, torch, P, synth):
        super().__init__(torch, P, synth)
        names = []
        for k, (name, state, G, T) in enumerate(synth.config5_all("cuda")):
            self.pairs.append((G, T))
            self.items.append((T, synth.inject_seed(5, k), synth.CONFIG5_RATE, synth.CONFIG5_MASK))
            names.append((name, state))
            if k % 100 == 0:
                log(f"  generated {k}/873")
        self.sample = [k for k, (nm, st) in enumerate(names)
                       if nm in ("embed", "lm_head", "l0.gate", "l0.up", "l0.down")]


class GPT13B(Workload):
    name = "gpt13b_ckpt"
    description = "GPT-style 1.3B checkpoint pair: 292 f32 tensors, T = G*(1+1e-6 z), NaN at rate 1e-9"

    def __init__(self, torch, P, synth):
        super().__init__(torch, P, synth)
        for name, G, T in synth.config3_all("cuda"):
            self.pairs.append((G, T))
        self.sample = [0, 1, 4, 8, 10]


class Activations(Workload):
    name = "activations_bf16_rounding"
    description = "32 f32 [8,512,4096] activation pairs, T = bf16-rounded G"

    def __init__(self, torch, P, synth):
        super().__init__(torch, P, synth)
        self.pairs = synth.config2_all("cuda")
        self.sample = [0, 1, 2, 3]


class Replay(Workload):
    name = "rfi_replay_f16"
    description = "1000 replayed f16 [4096,4096] calls, every 10th injected at rate 1e-7"
    roofline_note = ("the 1000 calls share one 33.5 MB golden, which the last-level cache keeps, so HBM moves "
                     "less than the algorithmic bytes (the golden counted once per call) and frac can pass 1; "
                     "traffic_frac is the rate of the bytes HBM moved")

    def __init__(self, torch, P, synth):
        super().__init__(torch, P, synth)
        G = synth.config4_golden("cuda")
        for c in range(synth.CONFIG4_CALLS):
            T = G.clone()
            self.pairs.append((G, T))
            if synth.config4_injected(c):
                self.items.append((T, synth.inject_seed(4, c), synth.CONFIG4_RATE, synth.CONFIG4_MASK))
        self.sample = [9, 19, 29]


class Single(Workload):
    name = "single_f32_1024x1024"
    description = "one f32 [1024,1024] pair with 16 planted bit flips"

    def __init__(self, torch, P, synth):
        super().__init__(torch, P, synth)
        import numpy as np
        G, T = synth.config1()
        self.pairs = [(torch.from_numpy(G).cuda(), torch.from_numpy(T).cuda())]
        self.sample = [0]
        del np


WORKLOADS = {"5": Llama7B, "3": GPT13B, "2": Activations, "4": Replay, "1": Single}


# ---------------------------------------------------------------------------
def host_share() -> int:
    """CPU cores this process may use: its affinity set, capped at the 16-core
    host share that goes with one GPU."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def cpu_baseline(wl: Workload, threads: int, target_bytes: float = 12e9):
    """The oracle, as it stands, on a bounded sample of the workload: host
    copies of the sampled pairs' device bytes (about target_bytes of golden +
    test), cut into equal element slices, one per thread (ctypes releases the
    GIL), so every core works for the whole timed span.  Each slice is one
    oracle step on its own: the oracle's injection of the test slice (with its
    pair's seed, rate and mask) when the workload injects that pair, then the
    oracle's signature of the slice -- the per-element work of the real step.
    Returns GB/s of golden+test bytes signed."""
    import numpy as np
    import oracle
    from tests.parity import to_host_bits

    inj = {id(T): (seed, rate, mask) for T, seed, rate, mask in wl.inject_items(0)}
    host, nbytes = [], 0
    t0 = time.time()
    for k in wl.sample:
        if nbytes >= target_bytes:
            break
        G, T = wl.pairs[k]
        code = {wl.torch.float32: 0, wl.torch.float16: 1, wl.torch.bfloat16: 2}[G.dtype]
        host.append((k, to_host_bits(G).reshape(-1), to_host_bits(T).reshape(-1), code, inj.get(id(T))))
        nbytes += G.numel() * G.element_size() * 2
    copy_s = time.time() - t0
    # equal element slices over the sample (slices never straddle two pairs'
    # byte arrays: each slice is cut from one pair, the last one of a pair may
    # be shorter)
    elems = sum(g.size for _, g, _, _, _ in host)
    per = -(-elems // threads)
    slices = []
    for k, g, t, code, spec in host:
        for a in range(0, g.size, per):
            slices.append((g[a:a + per], t[a:a + per].copy(), code, spec))
    slices.sort(key=lambda x: -x[0].size)

    def one(g, t, code, spec):
        if spec is not None:
            oracle.inject(t, dtype=code, seed=spec[0], rate=spec[1], mask=spec[2])
        oracle.signature(g, t, dtype=code)

    # one core, one slice: the oracle's per-core rate
    g1, t1, c1, s1 = slices[-1]
    t0 = time.time()
    one(g1, t1.copy(), c1, s1)
    per_core = (g1.nbytes + t1.nbytes) / (time.time() - t0) / 1e9

    work = list(range(len(slices)))
    lock = threading.Lock()

    def worker():
        while True:
            with lock:
                if not work:
                    return
                j = work.pop(0)
            one(*slices[j])

    t0 = time.time()
    ths = [threading.Thread(target=worker) for _ in range(threads)]
    for th in ths:
        th.start()
    for th in ths:
        th.join()
    dt = time.time() - t0
    del np
    return {"value": round(nbytes / dt / 1e9, 3), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "per_core_value": round(per_core, 3), "os_cpu_count": os.cpu_count(),
            "sample": f"{len(host)} of {len(wl.pairs)} pairs ({nbytes / 1e9:.2f} GB: pairs "
                      f"{', '.join(str(h[0]) for h in host)}) cut into {len(slices)} slices of at most {per} "
                      f"elements, one oracle step per slice ({'injection + ' if any(h[4] for h in host) else ''}"
                      f"signature), {dt:.1f} s wall on {threads} threads ({threads} of os.cpu_count() = "
                      f"{os.cpu_count()}: the host share of one GPU), D2H copy {copy_s:.1f} s not counted"}


def topk_measure(torch, P, prep_pairs, nbytes: int, reps: int = 3):
    """The paper's main score, the mean of the top 10% errors, over every pair
    of the workload: peat_topk_mean_batched (a sampled guess of each pair's
    boundary binade, the gathering pass that confirms it, the binade pass
    only where a guess fails, and the rounds), and the stream-ordered
    peat_topk_mean_from_signature_batched_async fed with the device records
    of the step's signature call on the same stream (the binade pass skips
    every pair whose record bounds the k-th largest error to one bin; the
    gathering pass collects that bin's range).  Best of
    reps from the library's kernel events: level 0 (class K_TOPK_A) and the
    rest (K_TOPK_B); nothing in either waits on the host."""
    def timed(call):
        call()                                                   # warm-up
        P.profile_enable(True)
        P.profile_read(P.K_TOPK_A)
        P.profile_read(P.K_TOPK_B)
        best = None
        for _ in range(reps):
            call()
            torch.cuda.synchronize()
            a, na = P.profile_read(P.K_TOPK_A)
            b, nb = P.profile_read(P.K_TOPK_B)
            cur = (a / max(1, na), b / max(1, nb))
            best = cur if best is None or sum(cur) < sum(best) else best
        P.profile_enable(False)
        return best

    count = prep_pairs.count
    recs = []
    lvl0, rest = timed(lambda: recs.__setitem__(slice(None), P.topk_mean_batched(prep_pairs, 1, 10)))
    d_sig = torch.empty(count * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    P.signature_batched_async(prep_pairs, d_sig)
    d_top = torch.empty(count * P.TOPK_BYTES, dtype=torch.uint8, device="cuda")
    slvl0, srest = timed(lambda: P.topk_mean_from_signature_batched_async(prep_pairs, d_sig, d_top, num=1, den=10))
    recs_s = P.decode_topk(d_top, count)
    # exact fields identical; sums identical where the record fixes the
    # boundary's binade, else formed per binade (within 1e-12 relative)
    same = all(x[f] == y[f] or (x[f] != x[f] and y[f] != y[f]) for x, y in zip(recs, recs_s)
               for f in ("n_valid", "k", "count_above", "kth_value"))
    rel = max((abs(x["sum_topk"] - y["sum_topk"]) / abs(y["sum_topk"]) if y["sum_topk"] not in (0.0, float("inf"))
               and y["sum_topk"] == y["sum_topk"] else 0.0) for x, y in zip(recs_s, recs)) if recs else 0.0
    nbit = sum(1 for x, y in zip(recs, recs_s) if x["sum_topk"] != y["sum_topk"])
    ms, ms_s = lvl0 + rest, slvl0 + srest
    return {"ms": round(ms, 3), "GBps_of_bytes_signed": round(nbytes / (ms / 1e3) / 1e9, 1),
            "level0_ms": round(lvl0, 3), "rest_ms": round(rest, 3),
            "pairs": len(recs), "k_total": int(sum(r["k"] for r in recs)),
            "what": "peat_topk_mean_batched, num/den = 1/10, kernel time of the whole stream-ordered sequence",
            "from_signature": {"ms": round(ms_s, 3), "GBps_of_bytes_signed": round(nbytes / (ms_s / 1e3) / 1e9, 1),
                               "level0_ms": round(slvl0, 3), "rest_ms": round(srest, 3),
                               "exact_fields_equal": bool(same), "sum_max_rel_diff": rel,
                               "pairs_with_other_sum_bits": nbit,
                               "what": "peat_topk_mean_from_signature_batched_async with the device records of "
                                       "the pairs' signatures (bins -40..24, one binade each), kernel time"}}


def mixed_measure(torch, P, reps: int = 5, count: int = 64, shape=(4096, 4096)):
    """Signature of mixed-precision pairs (Section III-C): FP32 golden outputs
    against the same outputs in FP64 (a few FP32 ulps of rounding-error-like
    noise) and in FP16 (the FP16 cast); count pairs of the given shape.  Best
    of reps of the chunk pass, from the library's kernel events."""
    g = torch.Generator(device="cuda")
    g.manual_seed(2609)
    golden = [torch.randn(shape, device="cuda", generator=g) for _ in range(count)]
    res = {}
    for name, make in (("f32_vs_f64", lambda x: x.double() * (1 + 2.0 ** -23 * torch.randn(
                            shape, device="cuda", dtype=torch.float64, generator=g))),
                       ("f32_vs_f16", lambda x: x.half())):
        tests = [make(x) for x in golden]
        pairs = list(zip(golden, tests))
        nbytes = sum(x.numel() * x.element_size() + t.numel() * t.element_size() for x, t in pairs)
        P.signature_mixed_batched(pairs)                           # warm-up
        P.profile_enable(True)
        P.profile_read(P.K_SIG_CHUNK)
        best = None
        for _ in range(reps):
            P.signature_mixed_batched(pairs)
            ms, n = P.profile_read(P.K_SIG_CHUNK)
            best = ms / n if best is None else min(best, ms / n)
        P.profile_enable(False)
        gbps = nbytes / (best / 1e3) / 1e9
        res[name] = {"ms": round(best, 4), "bytes": nbytes, "GBps": round(gbps, 1),
                     "frac_of_hbm_peak": round(gbps / HBM_PEAK_GBS, 4),
                     "bytes_per_element": tests[0].element_size() + golden[0].element_size()}
        del tests, pairs
        torch.cuda.empty_cache()
    res["config"] = f"{count} pairs of {list(shape)} (FP32 golden, N(0,1))"
    del golden
    torch.cuda.empty_cache()
    return res


def latency_measure(torch, P, synth, stream, reps: int = 50):
    """Per-call times of single-pair signatures (async call, HIP events on the
    stream, chunk pass + finalize): the 1024x1024 f32 pair warm, with the
    queue busy when the call is enqueued (the device's share), and cold
    (after reading 1 GiB so the pair is in no cache), the host round trip of
    the synchronous call, and one f16 [4096, 4096] replay call."""
    import statistics
    G, T = synth.config1()
    g, t = torch.from_numpy(G).cuda(), torch.from_numpy(T).cuda()
    h = synth.config4_golden("cuda")
    h2 = h.clone()
    h2.view(-1)[::9973] += 1.0
    d_out = torch.empty(P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    flush = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    flush.fill_(1)
    sink = torch.zeros(-(-flush.numel() // P.STREAM_SPAN), dtype=torch.int32, device="cuda")

    def timed(prep, cold=False, busy=False):
        if cold:
            P.stream_read(flush, sink, stream=stream)
        if busy:
            # the queue is still working when the call is enqueued, so the
            # events see the kernels and their dispatch, not the host's launch
            with torch.cuda.stream(stream):
                torch.cuda._sleep(200000)
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        P.signature_batched_async(prep, d_out, synth.BINS, synth.THRESHOLDS, stream=stream)
        b.record(stream)
        b.synchronize()
        return a.elapsed_time(b) * 1e3

    p1, p4 = P.PreparedPairs([(g, t)]), P.PreparedPairs([(h, h2)])
    for _ in range(5):
        timed(p1)
        timed(p4)
    warm = statistics.median(timed(p1) for _ in range(reps))
    device = statistics.median(timed(p1, busy=True) for _ in range(reps))
    cold = statistics.median(timed(p1, cold=True) for _ in range(10))
    f16 = statistics.median(timed(p4) for _ in range(20))
    walls = []
    for _ in range(reps):
        t0 = time.perf_counter()
        P.signature(g, t, synth.BINS, synth.THRESHOLDS)
        walls.append((time.perf_counter() - t0) * 1e6)
    del flush, sink
    torch.cuda.empty_cache()
    return {"single_f32_1024x1024": {"warm_us": round(warm, 1), "device_us": round(device, 1),
                                     "cold_us": round(cold, 1),
                                     "sync_call_wall_us": round(statistics.median(walls), 1)},
            "replay_f16_4096x4096_call_us": round(f16, 1),
            "what": "async single-pair signature, HIP events around the call on its stream (chunk pass + "
                    "finalize + launch gaps); device = the same with the queue busy when the call is enqueued "
                    "(no host launch time); cold = after a 1 GiB read; sync = host round trip of peat_signature"}


def read_ceiling(torch, P, stream, gib: int = 16, reps: int = 5):
    """GB/s of peat_stream_read over a gib-GiB buffer (best of reps)."""
    buf = torch.empty(gib << 30, dtype=torch.uint8, device="cuda")
    buf.fill_(0x5A)
    sink = torch.zeros(-(-buf.numel() // P.STREAM_SPAN), dtype=torch.int32, device="cuda")
    P.stream_read(buf, sink, stream=stream)          # warm-up
    torch.cuda.synchronize()
    P.profile_enable(True)
    P.profile_read(P.K_STREAM_READ)
    best = None
    for _ in range(reps):
        P.stream_read(buf, sink, stream=stream)
        torch.cuda.synchronize()
        ms, n = P.profile_read(P.K_STREAM_READ)
        best = ms / n if best is None else min(best, ms / n)
    P.profile_enable(False)
    nbytes = buf.numel()
    del buf
    torch.cuda.empty_cache()
    return {"GBps": round(nbytes / (best / 1e3) / 1e9, 1), "bytes": nbytes, "ms": round(best, 4),
            "kernel": "peat_stream_read (16-byte nontemporal buffer loads, 2 MiB per 256-thread block)"}


def time_steps(torch, P, stream, step, first: int, warmup: int, steps: int, classes):
    """warmup untimed steps, then steps timed ones (first, first + 1, ...)
    bracketed by events on the stream: total ms, sorted step times, and per
    kernel class (ms per launch, launches) from the library's HIP events."""
    for s in range(first, first + warmup):
        step(s)
    torch.cuda.synchronize()
    P.profile_enable(True)
    for k in classes:
        P.profile_read(k)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for j, s in enumerate(range(first + warmup, first + warmup + steps)):
        step(s)
        evs[j + 1].record(stream)
    torch.cuda.synchronize()
    total = evs[0].elapsed_time(evs[-1])
    step_ms = sorted(evs[j].elapsed_time(evs[j + 1]) for j in range(steps))
    P.profile_enable(False)
    per = {}
    for k in classes:
        ms, n = P.profile_read(k)
        per[k] = (ms / max(1, n), n)
    return total, step_ms, per


def workload_leg(torch, P, synth, key: str, stream, steps: int, warmup: int):
    """One step of another workload (its injections, then the batched
    signature of every pair), timed like the main step; the chunk pass's
    roofline fraction from its own kernel events."""
    t0 = time.time()
    wl = WORKLOADS[key](torch, P, synth)
    torch.cuda.synchronize()
    gen_s = time.time() - t0
    prep = P.PreparedPairs(wl.pairs)
    d_out = torch.empty(len(wl.pairs) * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    d_counts = torch.empty(max(1, len(wl.items)), dtype=torch.int64, device="cuda")
    items = [P.PreparedItems(wl.inject_items(s)) for s in range(warmup + steps)] if wl.items else []

    def step(s):
        if wl.items:
            P.inject_batched_async(items[s], d_counts, stream=stream)
        P.signature_batched_async(prep, d_out, synth.BINS, synth.THRESHOLDS, stream=stream)

    total, step_ms, per = time_steps(torch, P, stream, step, 0, warmup, steps,
                                     (P.K_SIG_CHUNK, P.K_SIG_FINALIZE, P.K_INJECT, P.K_INJECT_SUM))
    nbytes = wl.bytes_signed()
    ms = total / steps
    chunk = per[P.K_SIG_CHUNK][0]
    traffic = committed_traffic(wl.name)
    out = {"description": wl.description, "pairs": len(wl.pairs), "bytes_signed_per_step": nbytes,
           "step": "batched injection of the injected calls + batched signature of every pair" if wl.items
           else "batched signature of every pair",
           "ms_per_step": round(ms, 4), "GBps": round(nbytes / (ms / 1e3) / 1e9, 1),
           "step_ms": {"median": round(step_ms[len(step_ms) // 2], 4), "min": round(step_ms[0], 4),
                       "max": round(step_ms[-1], 4)},
           "kernels_ms_per_step": {"sig_chunk": round(chunk, 4), "sig_finalize": round(per[P.K_SIG_FINALIZE][0], 4),
                                   "inject": round(per[P.K_INJECT][0], 4) if wl.items else 0.0,
                                   "inject_sum": round(per[P.K_INJECT_SUM][0], 4) if wl.items else 0.0},
           "roofline": {"bound": "hbm", "kernel": "sig_chunk", "achieved": round(nbytes / (chunk / 1e3) / 1e9, 1),
                        "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": round(nbytes / (chunk / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                        "traffic": traffic},
           "generated_s": round(gen_s, 1)}
    if traffic:
        # the bytes HBM actually moved per second (committed counters), as a
        # fraction of the peak
        out["roofline"]["traffic_frac"] = round(traffic / (chunk / 1e3) / 1e9 / HBM_PEAK_GBS, 4)
    if wl.roofline_note:
        out["roofline"]["note"] = wl.roofline_note
    log(f"  {wl.name}: step {ms:.3f} ms, chunk pass {chunk:.3f} ms = {out['roofline']['frac']:.3f} of HBM peak")
    del wl, prep, d_out, d_counts, items
    torch.cuda.empty_cache()
    return out


def copy_calibration(torch, gib: int, reps: int):
    """A plain device copy of known size, for scaling FETCH_SIZE/WRITE_SIZE."""
    n = gib * (1 << 30) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": n * 4, "bytes_written": n * 4, "reps": reps}))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="5", choices=sorted(WORKLOADS))
    ap.add_argument("--separate", action="store_true",
                    help="time the step as two calls (injection, then signature) instead of the fused pass")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=16, help="at most this many (and at most the host share)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="GIB")
    ap.add_argument("--no-read-ceiling", action="store_true")
    ap.add_argument("--no-topk", action="store_true")
    ap.add_argument("--no-mixed", action="store_true")
    ap.add_argument("--mixed-only", action="store_true", help="only the mixed-precision measurement")
    ap.add_argument("--no-latency", action="store_true")
    ap.add_argument("--no-others", action="store_true", help="skip the legs of workloads 2, 3 and 4")
    ap.add_argument("--other-steps", type=int, default=5, help="timed steps of each other workload")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the signature of N GPUs is "
              f"N independent shards of the pair list with no exchange on the hot path", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_13544_amd as P
    import synth

    if args.copy_calibration:
        copy_calibration(torch, args.copy_calibration, 5)
        return
    if args.mixed_only:
        torch.cuda.set_device(0)
        print(json.dumps({"mixed_precision": mixed_measure(torch, P)}), flush=True)
        return

    torch.cuda.set_device(0)
    log(f"generating workload {args.workload} ...")
    t0 = time.time()
    wl = WORKLOADS[args.workload](torch, P, synth)
    torch.cuda.synchronize()
    log(f"generated in {time.time() - t0:.1f} s: {len(wl.pairs)} pairs, {wl.bytes_signed() / 1e9:.2f} GB")

    stream = torch.cuda.current_stream()
    prep_pairs = P.PreparedPairs(wl.pairs)
    d_out = torch.empty(len(wl.pairs) * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    d_counts = torch.empty(max(1, len(wl.items)), dtype=torch.int64, device="cuda")
    nsteps_all = args.warmup + args.steps
    fused = wl.fusable() and not args.separate
    step_items = [wl.inject_items(s) for s in range(2 * nsteps_all if fused else nsteps_all)]
    prepared_items = [P.PreparedItems(it) for it in step_items]

    def step_separate(s):
        if wl.items:
            P.inject_batched_async(prepared_items[s], d_counts, stream=stream)
        P.signature_batched_async(prep_pairs, d_out, synth.BINS, synth.THRESHOLDS, stream=stream)

    def step_fused(s):
        _, _, rate, mask = step_items[s][0]
        P.inject_signature_batched_async(prep_pairs, [seed for _, seed, _, _ in step_items[s]], rate, mask,
                                         d_out, d_counts, synth.BINS, synth.THRESHOLDS, stream=stream)

    classes = (P.K_SIG_CHUNK, P.K_SIG_FINALIZE, P.K_INJECT, P.K_INJECT_SUM, P.K_SIG_INJECT)

    ms_total, step_ms, per = time_steps(torch, P, stream, step_fused if fused else step_separate, 0,
                                        args.warmup, args.steps, classes)
    ms_step = ms_total / args.steps
    nbytes = wl.bytes_signed()
    value = nbytes / (ms_step / 1e3) / 1e9
    recs = P.decode_records(d_out, len(wl.pairs), nthr=len(synth.THRESHOLDS))
    flips = int(d_counts.sum().item()) if wl.items else 0
    if fused:
        # the same injections done by the two separate calls, for reference
        # (fresh seeds: steps nsteps_all ... 2 nsteps_all - 1)
        sep_total, _, sep_per = time_steps(torch, P, stream, step_separate, nsteps_all, args.warmup, args.steps,
                                           classes)
        chunk_avg = per[P.K_SIG_INJECT][0]
        sig_chunk_avg, inj_avg, isum_avg = sep_per[P.K_SIG_CHUNK][0], sep_per[P.K_INJECT][0], sep_per[P.K_INJECT_SUM][0]
        fin_avg = per[P.K_SIG_FINALIZE][0]
        dominant = "sig_chunk with injection (peat_inject_signature_batched_async)"
    else:
        chunk_avg = sig_chunk_avg = per[P.K_SIG_CHUNK][0]
        inj_avg, isum_avg, fin_avg = per[P.K_INJECT][0], per[P.K_INJECT_SUM][0], per[P.K_SIG_FINALIZE][0]
        dominant = "sig_chunk"
    achieved = nbytes / (chunk_avg / 1e3) / 1e9
    log(f"step {ms_step:.3f} ms ({'fused' if fused else 'separate'}): chunk pass {chunk_avg:.3f} ms, "
        f"finalize {fin_avg:.3f} ms; last step {flips} flips, {sum(r['n_nan_pairs'] for r in recs)} NaN pairs")
    if fused:
        log(f"separate calls: step {sep_total / args.steps:.3f} ms = injection {inj_avg:.3f} + {isum_avg:.3f} ms "
            f"+ signature chunk pass {sig_chunk_avg:.3f} ms")

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": wl.name, "description": wl.description, "pairs": len(wl.pairs),
                   "elements_per_side": wl.elements(), "bytes_signed_per_step": nbytes,
                   "bins": list(synth.BINS), "thresholds": list(synth.THRESHOLDS),
                   "step": ("bit-flip injection + signature of every pair in one pass "
                            "(peat_inject_signature_batched_async)") if fused else
                           ("batched injection + batched signature" if wl.items else "batched signature")},
        "roofline": {"bound": "hbm", "kernel": dominant, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": committed_traffic(wl.name, fused)},
        "kernels_ms_per_step": ({"sig_chunk_inject": round(chunk_avg, 4)} if fused else {}) | {
                                "sig_chunk": round(sig_chunk_avg, 4),
                                "sig_finalize": round(fin_avg, 4),
                                "inject": round(inj_avg, 4) if wl.items else 0.0,
                                "inject_sum": round(isum_avg, 4) if wl.items else 0.0},
        "step_ms": {"median": round(step_ms[len(step_ms) // 2], 4), "min": round(step_ms[0], 4),
                    "max": round(step_ms[-1], 4)},
        "signature_only_GBps": round(nbytes / ((sig_chunk_avg + fin_avg) / 1e3) / 1e9, 1),
        "inject_Gelem_per_s": round(sum(T.numel() for T, *_ in wl.items) / (inj_avg / 1e3) / 1e9, 1)
        if wl.items else None,
    }
    if out["roofline"]["traffic"]:
        out["roofline"]["traffic_frac"] = round(out["roofline"]["traffic"] / (chunk_avg / 1e3) / 1e9 / HBM_PEAK_GBS, 4)
    if wl.roofline_note:
        out["roofline"]["note"] = wl.roofline_note
    if fused:
        out["separate_calls"] = {"ms_per_step": round(sep_total / args.steps, 4),
                                 "GBps": round(nbytes / (sep_total / args.steps / 1e3) / 1e9, 1),
                                 "what": "the same step as peat_inject_batched_async + "
                                         "peat_signature_batched_async (the kernel times above)"}
    if not args.no_topk:
        log("top-10% mean ...")
        out["topk_mean"] = topk_measure(torch, P, prep_pairs, nbytes)
    if not args.no_read_ceiling:
        log("read ceiling ...")
        del prepared_items
        rc = read_ceiling(torch, P, stream)
        rc["chunk_pass_frac_of_ceiling"] = round(achieved / rc["GBps"], 4)
        rc["sig_chunk_frac_of_ceiling"] = round(nbytes / (sig_chunk_avg / 1e3) / 1e9 / rc["GBps"], 4)
        out["read_ceiling"] = rc
    if not args.no_cpu_baseline:
        log("cpu baseline ...")
        out["cpu_baseline"] = cpu_baseline(wl, min(args.cpu_threads, host_share()))
    if not args.no_latency:
        log("single-call latency ...")
        out["latency"] = latency_measure(torch, P, synth, stream)
    # the main workload's memory is released before the other legs
    main_key = args.workload
    del wl, prep_pairs, d_out, d_counts, step_items
    prepared_items = None
    torch.cuda.empty_cache()
    if not args.no_others:
        out["other_workloads"] = {}
        for key in ("2", "3", "4"):
            if key == main_key:
                continue
            log(f"workload {key} ...")
            leg = workload_leg(torch, P, synth, key, stream, args.other_steps, 2)
            out["other_workloads"][WORKLOADS[key].name] = leg
    if not args.no_mixed:
        log("mixed-precision pairs ...")
        out["mixed_precision"] = mixed_measure(torch, P)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
