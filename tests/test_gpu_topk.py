"""GPU parity of the top-k error mean (peat_topk_mean, the paper's "mean of
the top 10% errors") against the oracle's sort: n_valid, k, count_above and
the k-th largest error bit-exact; the sum and mean within 1e-12 relative
(both are binary64 sums of k non-negative terms: the device's fixed tree plus
an exact integer sum inside the k-th largest error's binade, against the
oracle's compensated sum).  Cases span several chunks with ragged tails in
the three element types, special values, heavy ties, a zero and an infinite
k-th error, unaligned pointers, batched against single calls, every route
of the selection (binade gather, bin gather, one pass per digit) against the
others, the stream-ordered forms against the synchronous ones, and a
full-size Llama-7B-shaped tensor."""
from __future__ import annotations

import math
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_13544_amd as P
import synth
from tests.parity import special_pair, to_device

pytestmark = pytest.mark.gpu

FRACS = [(1, 10), (1, 100), (1, 1), (3, 7), (1, 1 << 20)]


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def assert_topk(got: dict, ref: dict, ctx: str = ""):
    for key in ("n_valid", "k", "count_above"):
        assert got[key] == ref[key], f"{ctx}: {key} {got[key]} != {ref[key]}"
    for key in ("kth_value", "sum_topk", "mean_topk"):
        a, b = got[key], ref[key]
        if math.isnan(b):
            assert math.isnan(a), f"{ctx}: {key} {a} != NaN"
        elif math.isinf(b) or key == "kth_value":
            assert a == b, f"{ctx}: {key} {a!r} != {b!r}"
        else:
            assert abs(a - b) <= 1e-12 * abs(b), f"{ctx}: {key} {a!r} vs {b!r}"


def close_record(a: dict, b: dict) -> bool:
    """The exact fields equal; sum and mean equal or within 1e-12 relative
    (a window gather sums its binades in another order)."""
    for key in ("n_valid", "k", "count_above", "kth_value"):
        if not (a[key] == b[key] or (math.isnan(a[key]) and math.isnan(b[key]))):
            return False
    for key in ("sum_topk", "mean_topk"):
        x, y = a[key], b[key]
        if x == y or (math.isnan(x) and math.isnan(y)):
            continue
        if math.isinf(y) or abs(x - y) > 1e-12 * abs(y):
            return False
    return True


def same_record(a: dict, b: dict) -> bool:
    """Bit-identical records (NaN fields compare equal to NaN)."""
    return all(a[k] == b[k] or (isinstance(a[k], float) and math.isnan(a[k]) and math.isnan(b[k]))
               for k in a)


def check(gb, tb, code, num=1, den=10, ctx=""):
    got = P.topk_mean(to_device(gb, code), to_device(tb, code), num, den)
    ref = oracle.topk(gb, tb, dtype=code, num=num, den=den)
    assert_topk(got, ref, ctx)
    return got


@pytest.mark.parametrize("code", [0, 1, 2])
def test_sizes_specials_and_fractions(code):
    for i, n in enumerate([0, 1, 7, 4095, 4097, 65536 + 13, 300005, (1 << 20) + 3]):
        gb, tb = special_pair(n, code, seed=4000 + 13 * i + code)
        for num, den in FRACS:
            log(f"  dtype={code} n={n} frac={num}/{den}")
            check(gb, tb, code, num, den, f"dtype={code} n={n} {num}/{den}")


@pytest.mark.parametrize("code", [0, 1, 2])
def test_ties_and_equal_errors(code):
    n = 200003
    rng = np.random.default_rng(55 + code)
    g = rng.standard_normal(n)
    # errors on a coarse grid: many equal keys in every boundary bin
    q = rng.integers(0, 6, n).astype(np.float64)
    from tests.parity import float_to_bits
    for name, t in [("grid", g + q * 0.25), ("constant", g + 0.5), ("identical", g.copy())]:
        gb, tb = float_to_bits(g, code), float_to_bits(t, code)
        for num, den in FRACS:
            log(f"  dtype={code} {name} frac={num}/{den}")
            check(gb, tb, code, num, den, f"{name} {num}/{den}")


def test_zero_and_infinite_kth():
    code = 0
    n = 100000
    rng = np.random.default_rng(9)
    g = rng.standard_normal(n).astype(np.float32)
    t = g.copy()
    t[rng.integers(0, n, 50)] += 1.0                     # 50 nonzero errors: the top 10% ends at 0
    check(g.view(np.uint32), t.view(np.uint32), code, 1, 10, "zero kth")
    t2 = g.copy()
    t2[rng.integers(0, n, 20000)] = np.inf               # ~18% infinite errors: the 10th percentile is Inf
    check(g.view(np.uint32), t2.view(np.uint32), code, 1, 10, "inf kth")
    check(g.view(np.uint32), t2.view(np.uint32), code, 1, 2, "inf above, finite kth")
    t3 = np.full(n, np.nan, np.float32)
    check(g.view(np.uint32), t3.view(np.uint32), code, 1, 10, "all NaN")


@pytest.mark.parametrize("code", [0, 1, 2])
def test_unaligned_pointers(code):
    n = 90001
    gb, tb = special_pair(n + 1, code, seed=71 + code)
    got = P.topk_mean(to_device(gb, code)[1:], to_device(tb, code)[1:], 1, 10)
    assert_topk(got, oracle.topk(gb[1:], tb[1:], dtype=code, num=1, den=10), "unaligned")


def test_batched_equals_single_and_is_deterministic():
    pairs_host = []
    for k, (n, code) in enumerate([(300000, 0), (5000, 1), (1 << 20, 2), (77, 0), (0, 1), (250000, 0)]):
        pairs_host.append((*special_pair(n, code, seed=900 + k), code))
    pairs = [(to_device(g, c), to_device(t, c)) for g, t, c in pairs_host]
    for num, den in ((1, 10), (1, 1000)):
        batched = P.topk_mean_batched(pairs, num, den)
        again = P.topk_mean_batched(pairs, num, den)
        for k, ((g, t, c), (gd, td)) in enumerate(zip(pairs_host, pairs)):
            single = P.topk_mean(gd, td, num, den)
            assert same_record(single, batched[k]) and same_record(batched[k], again[k]), f"pair {k}"
            assert_topk(batched[k], oracle.topk(g, t, dtype=c, num=num, den=den), f"pair {k}")


def test_llama7b_tensor_full_size():
    """Full-size Llama-7B-shaped tensors of the benchmark workload: the gate
    projection of layer 0 (45 M elements) as weights and as Adam second
    moment, with the workload's exponent-bit injection applied."""
    from tests.parity import to_host_bits
    states = synth.llama7b_states()
    for k, (name, shape, state) in enumerate(states):
        if name != "l0.gate" or state not in (0, 2):
            continue
        log(f"  {name} state={state} {shape}")
        G, T = synth.config5_pair(k, shape, state, "cuda")
        P.inject(T, synth.inject_seed(5, k), synth.CONFIG5_RATE, synth.CONFIG5_MASK)
        got = P.topk_mean(G, T, 1, 10)
        ref = oracle.topk(to_host_bits(G), to_host_bits(T), dtype=0, num=1, den=10)
        assert_topk(got, ref, f"{name} state={state}")
        assert got["k"] == -(-G.numel() // 10)
        del G, T
    torch.cuda.empty_cache()


def test_from_signature_equals_standalone():
    """peat_topk_mean_from_signature_batched against the standalone call and
    the oracle: bit-identical where the signature's one-binade histogram
    fixes level 0 (regular bins, zero errors), the exact fields identical
    and the sums within 1e-12 where it leaves a window of binades (k-th
    largest error in hist_over or hist_under, or bins two binades wide),
    with Inf and NaN pairs, empty pairs and unaligned views."""
    from tests.parity import float_to_bits
    rng = np.random.default_rng(2024)
    cases = []
    n = 300007
    g = rng.standard_normal(n)
    for code in (0, 1, 2):
        cases.append(("specials", *special_pair(200003, code, seed=3100 + code), code))
        cases.append(("relative 1e-3", float_to_bits(g, code), float_to_bits(g * (1 + 1e-3 * rng.standard_normal(n)), code), code))
    g32 = g.astype(np.float32)
    cases.append(("huge errors (over)", g32.view(np.uint32), (g32 * np.float32(3e8)).view(np.uint32), 0))
    cases.append(("tiny errors (under)", g32.view(np.uint32),
                  (g32 + np.float32(1e-13) * (np.arange(n) % 7 == 0)).view(np.uint32), 0))
    t_inf = g32.copy()
    t_inf[rng.integers(0, n, 40000)] = np.inf
    cases.append(("Inf errors above", g32.view(np.uint32), t_inf.view(np.uint32), 0))
    t_nan = (g32 * np.float32(1.001)).copy()
    t_nan[rng.integers(0, n, 5000)] = np.nan
    cases.append(("NaN pairs", g32.view(np.uint32), t_nan.view(np.uint32), 0))
    cases.append(("identical", g32.view(np.uint32), g32.view(np.uint32).copy(), 0))
    cases.append(("empty", np.zeros(0, np.uint32), np.zeros(0, np.uint32), 0))
    pairs = [(to_device(gb, c), to_device(tb, c)) for _, gb, tb, c in cases]
    gbu, tbu = special_pair(90001, 0, seed=77)
    pairs.append((to_device(gbu, 0)[1:], to_device(tbu, 0)[1:]))
    cases.append(("unaligned", gbu[1:], tbu[1:], 0))
    for bins in ((-40, 24, 64), (-40, 24, 32), (-20, 10, 30)):
        sigs = P.signature_batched(pairs, bins=bins)
        for num, den in ((1, 10), (1, 1000), (1, 1), (3, 7)):
            log(f"  bins={bins} frac={num}/{den}")
            ref = P.topk_mean_batched(pairs, num, den)
            got = P.topk_mean_from_signature_batched(pairs, sigs, bins, num, den)
            again = P.topk_mean_from_signature_batched(pairs, sigs, bins, num, den)
            for k, (name, gb, tb, c) in enumerate(cases):
                ctx = f"{name} bins={bins} {num}/{den}"
                assert same_record(got[k], again[k]), ctx
                if _fixes_binade(sigs[k], bins, num, den):
                    assert same_record(got[k], ref[k]), f"{ctx}: {got[k]} != {ref[k]}"
                else:
                    assert close_record(got[k], ref[k]), f"{ctx}: {got[k]} vs {ref[k]}"
                if bins == (-40, 24, 64) and (num, den) == (1, 10):
                    assert_topk(got[k], oracle.topk(gb, tb, dtype=c, num=num, den=den), name)


def _fixes_binade(sig: dict, bins, num: int, den: int) -> bool:
    """Whether a record's histogram fixes the binade of the k-th largest
    error: a regular one-binade bin, or the zero errors (no binary64 test
    side here); records that do not match are not given."""
    lo, hi, nb = bins
    nv = sig["n_valid"]
    k = -(-nv * num // den)
    if k == 0:
        return True
    acc = sig["hist_over"]
    if k <= acc:
        return False
    for i in range(nb - 1, -1, -1):
        acc += sig["hist"][i]
        if k <= acc:
            return hi - lo == nb
    return k > acc + sig["hist_under"]


def _window_cases():
    """f32 pairs whose top-10 % boundary lies below 2^-40 (the default bins'
    under bin): Adam second-moment-like values with relative noise (a few
    distinct errors per binade: the window fits the gather) and errors
    spread over about a hundred binades (the window does not fit; the pair
    is gathered again by binade), plus huge errors (the over bin)."""
    rng = np.random.default_rng(4242)
    n = 300007
    v = (rng.standard_normal(n) * 1e-3).astype(np.float32) ** 2
    t = (v * (1 + 1e-7 * rng.standard_normal(n))).astype(np.float32)
    z = np.zeros(n, np.float32)
    spread = np.ldexp(rng.integers(1, 9, n).astype(np.float64), -40 - rng.integers(3, 103, n)).astype(np.float32)
    g32 = rng.standard_normal(n).astype(np.float32)
    return [("adam v", v.view(np.uint32), t.view(np.uint32)),
            ("spread below 2^-40", z.view(np.uint32), spread.view(np.uint32)),
            ("huge errors", g32.view(np.uint32), (g32 * np.float32(3e8)).view(np.uint32))]


@pytest.mark.parametrize("caps", [(-1, -1), (0, -1), (0, 0), (16, 1 << 10)])
def test_from_signature_windows(caps):
    """Windows of binades gathered whole, given up and gathered again by
    binade, or overflowing further: every route against the standalone call
    (exact fields identical, sums within 1e-12) and the oracle."""
    cases = _window_cases()
    pairs = [(to_device(gb, 0), to_device(tb, 0)) for _, gb, tb in cases]
    try:
        P.topk_set_entry_capacity(*caps)
        for bins in ((-40, 24, 64), (-40, 24, 32)):
            sigs = P.signature_batched(pairs, bins=bins)
            for num, den in ((1, 10), (1, 3)):
                log(f"  caps={caps} bins={bins} frac={num}/{den}")
                ref = P.topk_mean_batched(pairs, num, den)
                got = P.topk_mean_from_signature_batched(pairs, sigs, bins, num, den)
                for k, (name, gb, tb) in enumerate(cases):
                    assert close_record(got[k], ref[k]), f"{name}: {got[k]} vs {ref[k]}"
                    assert_topk(got[k], oracle.topk(gb, tb, dtype=0, num=num, den=den), name)
    finally:
        P.topk_set_entry_capacity(-1, -1)


def test_from_signature_with_fused_step_records():
    """The records of the fused injection + signature call (decoded from
    device memory) serve the top-k call on the injected tensors."""
    pairs_host = [special_pair(n, 0, seed=5100 + n % 97) for n in (400009, 70001, 1 << 20)]
    pairs = [(to_device(g, 0), to_device(t, 0)) for g, t in pairs_host]
    seeds = [11, 12, 13]
    d_out = torch.zeros(len(pairs) * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    d_counts = torch.zeros(len(pairs), dtype=torch.int64, device="cuda")
    P.inject_signature_batched_async(pairs, seeds, 1e-4, 0x7F800000, d_out, d_counts)
    torch.cuda.synchronize()
    sigs = P.decode_records(d_out, len(pairs))
    for num, den in ((1, 10), (1, 100)):
        ref3 = P.topk_mean_batched(pairs, num, den)
        got = P.topk_mean_from_signature_batched(pairs, sigs, num=num, den=den)
        for k in range(len(pairs)):
            assert close_record(got[k], ref3[k]), f"pair {k} {num}/{den}: {got[k]} != {ref3[k]}"


def _route_cases():
    """Pairs whose boundary binade holds few distinct errors (checkpoint-like
    relative noise: the binade gather fits), many (independent values: the
    gather overflows its table), ties on a grid, special values, a binary64
    test side with subnormal errors, a zero k-th error, empty and unaligned
    views; each spans several chunks with a ragged tail."""
    from tests.parity import float_to_bits
    rng = np.random.default_rng(8080)
    cases = []
    n = 600007
    g = rng.standard_normal(n)
    g32 = (0.02 * g).astype(np.float32)
    t32 = (g32 * (1 + 1e-7 * rng.standard_normal(n))).astype(np.float32)
    cases.append(("checkpoint f32", g32.view(np.uint32), t32.view(np.uint32), (0, 0)))
    cases.append(("independent f32", float_to_bits(g, 0), float_to_bits(rng.standard_normal(n), 0), (0, 0)))
    for code in (1, 2):
        cases.append((f"independent dtype={code}", float_to_bits(g, code),
                      float_to_bits(g + 0.01 * rng.standard_normal(n), code), (code, code)))
        cases.append((f"specials dtype={code}", *special_pair(300001, code, seed=8100 + code), (code, code)))
    q = rng.integers(0, 6, n).astype(np.float64)
    cases.append(("grid ties", float_to_bits(g, 0), float_to_bits(g + q * 0.25, 0), (0, 0)))
    t_zero = g32.copy()
    t_zero[rng.integers(0, n, 40)] += 1.0
    cases.append(("zero kth", g32.view(np.uint32), t_zero.view(np.uint32), (0, 0)))
    # binary64 test side: 3% normal errors, the rest subnormal (the k-th
    # largest error in binade 0, ordered by the later digits), with few and
    # with many distinct values
    normal = rng.random(n) < 0.03
    gz = np.where(normal, g32, np.float32(0))
    for name, vals in (("few", rng.integers(0, 8, n) << 20), ("many", rng.integers(0, 1 << 40, n))):
        t64 = np.where(normal, gz.astype(np.float64) * (1 + 1e-3 * rng.standard_normal(n)),
                       np.ldexp(vals.astype(np.float64), -1074))
        cases.append((f"f32 vs f64 subnormal errors, {name}", gz.view(np.uint32), t64.view(np.uint64), (0, 3)))
    cases.append(("empty", np.zeros(0, np.uint32), np.zeros(0, np.uint32), (0, 0)))
    return cases


def _dev(bits, code):
    if code == 3:
        return torch.from_numpy(bits.view(np.float64).copy()).cuda()
    return to_device(bits, code)


def _mixed_device(cases):
    return [(_dev(gb, cg), _dev(tb, ct)) for _, gb, tb, (cg, ct) in cases]


@pytest.mark.parametrize("caps", [(-1, -1), (0, -1), (0, 0), (64, 1 << 12)])
def test_routes_give_identical_records(caps):
    """Every route through the selection (binade gather, bin gather, one
    histogram pass per digit, and capacities that overflow part way) gives
    records bit-identical to the default route's and within the oracle's bar."""
    cases = _route_cases()
    pairs = _mixed_device(cases)
    ref = {}
    try:
        P.topk_set_entry_capacity(-1, -1)
        for num, den in ((1, 10), (1, 1000), (3, 7)):
            ref[(num, den)] = P.topk_mean_mixed_batched(pairs, num, den)
        P.topk_set_entry_capacity(*caps)
        for num, den in ((1, 10), (1, 1000), (3, 7)):
            log(f"  caps={caps} frac={num}/{den}")
            got = P.topk_mean_mixed_batched(pairs, num, den)
            for k, (name, gb, tb, (cg, ct)) in enumerate(cases):
                assert same_record(got[k], ref[(num, den)][k]), f"{name} {num}/{den}: {got[k]} != {ref[(num, den)][k]}"
                if (num, den) == (1, 10):
                    assert_topk(got[k], oracle.topk_mixed(gb, tb, gdtype=cg, tdtype=ct, num=num, den=den), name)
    finally:
        P.topk_set_entry_capacity(-1, -1)


def test_async_entry_points_match_sync():
    """The stream-ordered forms: records in device memory equal to the
    synchronous calls', with the signature records handed over on the same
    stream (no host copy in between), and a record that does not match its
    pair ignored rather than trusted."""
    cases = _route_cases()
    same = [(gb, tb, cg) for _, gb, tb, (cg, ct) in cases if cg == ct]
    pairs = [(to_device(gb, c), to_device(tb, c)) for gb, tb, c in same]
    prep = P.PreparedPairs(pairs)
    stream = torch.cuda.Stream()
    bins = (-40, 24, 64)
    d_sig = torch.zeros(len(pairs) * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    d_out = torch.zeros(len(pairs) * P.TOPK_BYTES, dtype=torch.uint8, device="cuda")
    d_out2 = torch.zeros_like(d_out)
    with torch.cuda.stream(stream):
        P.signature_batched_async(prep, d_sig, bins, stream=stream)
        P.topk_mean_from_signature_batched_async(prep, d_sig, d_out, bins, 1, 10, stream=stream)
        P.topk_mean_batched_async(prep, d_out2, 1, 10, stream=stream)
    stream.synchronize()
    ref = P.topk_mean_batched(pairs, 1, 10)
    got = P.decode_topk(d_out, len(pairs))
    got2 = P.decode_topk(d_out2, len(pairs))
    sigs = P.decode_records(d_sig, len(pairs))
    got3 = P.topk_mean_from_signature_batched(pairs, sigs, bins, 1, 10)
    for k in range(len(pairs)):
        assert same_record(got[k], got3[k]) and same_record(got2[k], ref[k]) and close_record(got[k], ref[k]), f"pair {k}"
    # a record of another pair (n differs): ignored on the device
    if len(pairs) >= 2:
        host = d_sig.view(-1).cpu().numpy().copy()
        rec = host.reshape(len(pairs), P.SIG_BYTES)
        rec[0], rec[-1] = rec[-1].copy(), rec[0].copy()
        d_bad = torch.from_numpy(host).cuda()
        P.topk_mean_from_signature_batched_async(prep, d_bad, d_out, bins, 1, 10)
        torch.cuda.synchronize()
        got4 = P.decode_topk(d_out, len(pairs))
        for k in range(len(pairs)):
            assert close_record(got4[k], ref[k]), f"swapped records, pair {k}"
    # mixed-precision forms
    mpairs = _mixed_device(cases)
    d_msig = torch.zeros(len(mpairs) * P.SIG_BYTES, dtype=torch.uint8, device="cuda")
    d_mout = torch.zeros(len(mpairs) * P.TOPK_BYTES, dtype=torch.uint8, device="cuda")
    d_mout2 = torch.zeros_like(d_mout)
    P.signature_mixed_batched_async(mpairs, d_msig, bins)
    P.topk_mean_mixed_from_signature_batched_async(mpairs, d_msig, d_mout, bins, 1, 10)
    P.topk_mean_mixed_batched_async(mpairs, d_mout2, 1, 10)
    torch.cuda.synchronize()
    mref = P.topk_mean_mixed_batched(mpairs, 1, 10)
    for k, (a, b) in enumerate(zip(P.decode_topk(d_mout, len(mpairs)), P.decode_topk(d_mout2, len(mpairs)))):
        assert close_record(a, mref[k]) and same_record(b, mref[k]), f"mixed pair {k}"


def test_standalone_guess_misses_and_hits():
    """The standalone call guesses the boundary's binade from a strided
    sample of the pair.  Large errors placed only between the sampled runs
    (256 runs of 32 elements) make the guess wrong, which costs the binade
    pass and a second gathering pass; the records stay exact, equal for
    single and batched calls and for every entry capacity."""
    n = 1 << 20
    rng = np.random.default_rng(5150)
    g = rng.standard_normal(n).astype(np.float32)
    t = (g * (1 + 1e-6 * rng.standard_normal(n))).astype(np.float32)
    sampled = np.zeros(n, bool)
    for r in range(256):
        st = min(r * n // 256, n - 32)
        sampled[st:st + 32] = True
    hidden = np.flatnonzero(~sampled)
    big = rng.choice(hidden, size=n // 7, replace=False)
    t_miss = t.copy()
    t_miss[big] = g[big] + np.float32(2.0 ** -5) * (1 + rng.random(big.size).astype(np.float32))
    cases = [("guess right", g, t), ("guess wrong", g, t_miss)]
    pairs = [(to_device(a.view(np.uint32), 0), to_device(b.view(np.uint32), 0)) for _, a, b in cases]
    try:
        for caps in ((-1, -1), (0, -1), (0, 0)):
            P.topk_set_entry_capacity(*caps)
            batched = P.topk_mean_batched(pairs, 1, 10)
            for k, (name, a, b) in enumerate(cases):
                log(f"  {name} caps={caps}")
                single = P.topk_mean(*pairs[k], 1, 10)
                assert same_record(single, batched[k]), f"{name} caps={caps}"
                if caps == (-1, -1):
                    assert_topk(single, oracle.topk(a.view(np.uint32), b.view(np.uint32), dtype=0, num=1, den=10),
                                name)
            if caps == (-1, -1):
                refs = batched
            else:
                for k in range(len(cases)):
                    assert same_record(batched[k], refs[k]), f"{cases[k][0]} caps={caps}"
    finally:
        P.topk_set_entry_capacity(-1, -1)
