"""Pins of the CPU oracle to facts fixed outside the oracle itself.

Each test ties an oracle function to something the paper prints (Table II, scaling limits,
the 4.6 % clean-bucket rate, the 1.2533 clipped-mean constant, the bit-26 example), to a closed
form, to a library routine on a special case, or to published test vectors — chosen so that a
dropped term, a wrong sign, an off-by-one index or a transposed operand fails one of them.
"""
import math

import numpy as np
import pytest

from oracle import fpsketch_oracle as o
from paper_2609_19758_amd import workloads as wl
from conftest import load_golden

P = o.Params()


# --- hashing ---------------------------------------------------------------------------------

def test_splitmix64_published_vectors():
    for row in load_golden("splitmix64_vectors.csv"):
        got = int(o.splitmix64_stream(int(row["seed"]), np.array([int(row["index"])],
                                                                  dtype=np.uint64))[0])
        assert got == int(row["output"]), row


def test_hash_ranges_and_balance():
    n, m = 200_000, 48
    b, s = o.hash_round(7, 2, 1, n, m)
    assert b.min() >= 0 and b.max() < m
    assert set(np.unique(s)) == {-1.0, 1.0}
    counts = np.bincount(b, minlength=m)
    # multinomial: each count ~ n/m with sd sqrt(n/m); allow 6 sd.
    assert np.all(np.abs(counts - n / m) < 6 * math.sqrt(n / m))
    assert abs(s.mean()) < 6 / math.sqrt(n)


def test_hash_rounds_and_sides_independent():
    n, m = 50_000, 64
    b0, _ = o.hash_round(1, 1, 0, n, m)
    b1, _ = o.hash_round(1, 1, 1, n, m)
    b2, _ = o.hash_round(1, 2, 0, n, m)
    b3, _ = o.hash_round(2, 1, 0, n, m)
    for other in (b1, b2, b3):
        # agreement of two independent uniform hashes is ~1/m
        assert abs(np.mean(b0 == other) - 1 / m) < 6 * math.sqrt(1 / m / n)


def test_lemma2_collision_bound_monte_carlo():
    """Lemma 2: P[(i, j) not isolated] <= 2 (Delta - 1)/m + s/m^2 under the hash family."""
    m, s, delta = 32, 12, 3
    rng = np.random.Generator(np.random.PCG64(5))
    # s errors: the first at (0, 0), delta-1 more in row 0, the rest scattered (distinct rows).
    fails, trials = 0, 3000
    n1 = n3 = 4096
    rows = np.concatenate([[0] * delta, rng.choice(np.arange(1, n1), s - delta, replace=False)])
    cols = np.concatenate([np.arange(delta), rng.choice(np.arange(delta, n3), s - delta,
                                                        replace=False)])
    for seed in range(trials):
        hr = o.make_round(seed, 1, n1, n3, m)
        a0, b0 = hr.h1[rows[0]], hr.h2[cols[0]]
        others = [(hr.h1[r], hr.h2[c]) for r, c in zip(rows[1:], cols[1:])]
        fails += any(x == (a0, b0) for x in others)
    bound = 2 * (delta - 1) / m + s / m ** 2
    # bound holds with sampling slack (3 sd of a binomial at the bound)
    assert fails / trials <= bound + 3 * math.sqrt(bound / trials)
    # and the row-mates alone give about (delta - 1)/m^... (sanity: not trivially zero)
    assert fails > 0


# --- decoding --------------------------------------------------------------------------------

def test_decode_fp16_known_values_and_all_patterns():
    known = {0x3C00: 1.0, 0xC000: -2.0, 0x0001: 2.0 ** -24, 0x0400: 2.0 ** -14,
             0x7BFF: 65504.0, 0x3555: 0.333251953125, 0x8000: -0.0}
    for bits, val in known.items():
        assert o.decode_fp16(np.array([bits], dtype=np.uint16))[0] == val
    assert np.isinf(o.decode_fp16(np.array([0x7C00], dtype=np.uint16))[0])
    assert np.isnan(o.decode_fp16(np.array([0x7E00], dtype=np.uint16))[0])
    allp = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = allp.view(np.float16).astype(np.float64)
    got = o.decode_fp16(allp)
    fin = np.isfinite(ref)
    assert np.array_equal(got[fin], ref[fin])


def test_decode_bf16_known_values():
    known = {0x3F80: 1.0, 0xC040: -3.0, 0x0001: 2.0 ** -133, 0x7F7F: 3.3895313892515355e38,
             0x3E80: 0.25}
    for bits, val in known.items():
        assert o.decode_bf16(np.array([bits], dtype=np.uint16))[0] == val


def test_bf16_rounding_of_generator_is_rne():
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: ties to even -> 1.0; 1 + 3*2^-8 -> 1 + 2^-6
    x = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -1 - 2 ** -9], dtype=np.float32)
    got = o.decode_bf16(wl.f32_to_bf16_bits(x))
    assert list(got) == [1.0, 1 + 2 ** -6, -1.0]


# --- Eq. 1 and the moment sketches ---------------------------------------------------------

def _dense_h(h, v, m, w=None):
    n = h.size
    H = np.zeros((m, n))
    H[h, np.arange(n)] = v if w is None else v * w
    return H


def test_sketches_equal_factored_form_eq1():
    """The oracle's explicit-E bucket sums equal Eq. 1's factored form (H1 A)(B H2^T) - H1 C H2^T
    built from dense H matrices, and R, T equal it with W1 on the A and C rows or W2 on the
    B and C columns."""
    rng = np.random.Generator(np.random.PCG64(11))
    n1, n2, n3, m = 37, 19, 29, 6
    A = rng.standard_normal((n1, n2))
    B = rng.standard_normal((n2, n3))
    C = A @ B + rng.standard_normal((n1, n3)) * 1e-3
    C[3, 4] += 2.5
    hr = o.make_round(3, 1, n1, n3, m)
    S, R, T = o.sketches(A @ B - C, hr)
    w1 = np.arange(1, n1 + 1) / 64.0      # 2^ceil(log2 37) = 64
    w2 = np.arange(1, n3 + 1) / 32.0      # 2^ceil(log2 29) = 32
    H1, H2 = _dense_h(hr.h1, hr.v1, m), _dense_h(hr.h2, hr.v2, m)
    H1w, H2w = _dense_h(hr.h1, hr.v1, m, w1), _dense_h(hr.h2, hr.v2, m, w2)
    np.testing.assert_allclose(S, (H1 @ A) @ (B @ H2.T) - H1 @ C @ H2.T, rtol=0, atol=1e-9)
    np.testing.assert_allclose(R, (H1w @ A) @ (B @ H2.T) - H1w @ C @ H2.T, rtol=0, atol=1e-9)
    np.testing.assert_allclose(T, (H1 @ A) @ (B @ H2w.T) - H1 @ C @ H2w.T, rtol=0, atol=1e-9)


def test_single_bucket_reduces_to_bilinear_form():
    """m = 1: S = v1^T E v2 and R = (v1 * w)^T E v2, a library matrix-vector product."""
    rng = np.random.Generator(np.random.PCG64(2))
    E = rng.standard_normal((23, 41))
    hr = o.make_round(9, 0, 23, 41, 1)
    S, R, T = o.sketches(E, hr)
    assert abs(S[0, 0] - hr.v1 @ E @ hr.v2) < 1e-10
    assert abs(R[0, 0] - (hr.v1 * np.arange(1, 24) / 32) @ E @ hr.v2) < 1e-10
    assert abs(T[0, 0] - hr.v1 @ E @ (hr.v2 * np.arange(1, 42) / 64)) < 1e-10


def test_eq2_ratio_recovers_index_exactly():
    """Eq. 2: an isolated integer error gives 2^L R/S = i and 2^L' T/S = j exactly (1-based),
    including the last index of a non-power-of-two size (power-of-two weights are exact)."""
    n1, n3, m = 3000, 1500, 16
    hr = o.make_round(4, 2, n1, n3, m)
    for (i, j, d) in [(0, 0, 3.0), (n1 - 1, n3 - 1, -7.0), (1234, 777, 1.0), (2047, 1023, 5.0)]:
        E = np.zeros((n1, n3))
        E[i, j] = d
        S, R, T = o.sketches(E, hr)
        a, b = hr.h1[i], hr.h2[j]
        assert np.count_nonzero(S) == 1 and S[a, b] == hr.v1[i] * hr.v2[j] * d
        assert 4096 * R[a, b] / S[a, b] == i + 1
        assert 2048 * T[a, b] / S[a, b] == j + 1


def test_linearity():
    rng = np.random.Generator(np.random.PCG64(8))
    E1, E2 = rng.standard_normal((40, 30)), rng.standard_normal((40, 30))
    hr = o.make_round(1, 3, 40, 30, 5)
    s1, r1, t1 = o.sketches(E1, hr)
    s2, r2, t2 = o.sketches(E2, hr)
    s3, r3, t3 = o.sketches(2.5 * E1 - E2, hr)
    for x1, x2, x3 in ((s1, s2, s3), (r1, r2, r3), (t1, t2, t3)):
        np.testing.assert_allclose(x3, 2.5 * x1 - x2, rtol=0, atol=1e-12)


# --- thresholds ------------------------------------------------------------------------------

def test_clipped_mean_constant_is_sqrt_pi_over_2():
    assert abs(o.CLIP_MEAN_CONST - math.sqrt(math.pi / 2)) < 1e-4
    rng = np.random.Generator(np.random.PCG64(3))
    S = rng.standard_normal(2_000_000) * 0.37
    # clipping at 5 x mean|S| (= 4 sigma) removes ~6e-5 of the mass: sigma_hat ~ sigma
    assert abs(o.clipped_sigma(S) / 0.37 - 1) < 0.005


def test_mad_reading_matches_stated_clean_bucket_rate():
    """Sec. III-E puts the share of clean buckets above tau_c = 2 sigma_MAD near 4.6 %; only the
    MAD of the signed sketch gives that share (the two-sided Gaussian tail at 2 sigma)."""
    rng = np.random.Generator(np.random.PCG64(4))
    S = rng.standard_normal(2_000_000) * 1.7
    sig = o.mad_sigma(S)
    assert abs(sig / 1.7 - 1) < 0.005
    frac = np.mean(np.abs(S) > 2 * sig)
    assert 0.044 < frac < 0.048
    # the printed |S|-inside form would give ~0.59 sigma and ~24 %: not the stated rate
    lit = 1.4826 * o.median(np.abs(np.abs(S) - o.median(np.abs(S))))
    assert 0.55 < lit / 1.7 < 0.63 and np.mean(np.abs(S) > 2 * lit) > 0.2


def test_median_even_count():
    assert o.median(np.array([4.0, 1.0, 3.0, 2.0])) == 2.5
    assert o.median(np.array([5.0, 1.0, 3.0])) == 3.0


def test_huge_limit():
    assert o.HUGE_LIMIT == float(np.finfo(np.float32).max) / 16
    assert abs(o.HUGE_LIMIT - 2.1267647e37) < 1e30


def test_bit26_flip_example():
    """Sec. VI-A's worked example: an FP32 value of 16 with bit 26 (an exponent bit) flipped
    reads 4096, i.e. 256 times larger."""
    assert wl.flip_bit_value(16.0, wl.FP32_EXP_BIT26) == 4096.0


# --- bucket-count rules (Eq. 3-5) and plan (Sec. III-G) -----------------------------------

def test_table2_bucket_counts():
    for row in load_golden("table2_bucket_counts.csv"):
        n1, n2, n3 = int(row["n1"]), int(row["n2"]), int(row["n3"])
        assert o.m_start(n1, n2, n3, "bf16", P) == int(row["m_bf16"]), row
        assert o.m_start(n1, n2, n3, "fp16", P) == int(row["m_fp16"]), row


def test_law_sigma_over_rms_against_table2():
    """Eq. 3 (the noise law, per unit of rms(C)) pinned by Table II: at m = 1 and delta = rms(C),
    Eq. 4 is Eq. 3 times max(n1, n3) / B*, so ceil(max(n1, n3) / B* x law(m = 1)) must equal
    every printed bucket count, except where Eq. 5 raises it to m_comb = 48 (the count printed is
    then 48 and the law's value is at most 48).  The law is evaluated through
    law_sigma_over_rms alone; m_num is not used."""
    mcomb = o.m_comb(P)
    for row in load_golden("table2_bucket_counts.csv"):
        n1, n2, n3 = int(row["n1"]), int(row["n2"]), int(row["n3"])
        for fmt, key in (("bf16", "m_bf16"), ("fp16", "m_fp16")):
            printed = int(row[key])
            v = math.ceil(max(n1, n3) / P.b_star * o.law_sigma_over_rms(n1, n2, n3, 1, fmt, P))
            if printed == mcomb:
                assert v <= mcomb, (row, fmt, v)
            else:
                assert v == printed, (row, fmt, v)
    # the law falls as 1/m: sigma of an m-bucket sketch is the m = 1 value over m
    base = o.law_sigma_over_rms(8192, 4096, 4096, 1, "bf16", P)
    for m in (2, 48, 1000):
        assert abs(o.law_sigma_over_rms(8192, 4096, 4096, m, "bf16", P) * m - base) <= 1e-15 * base


def _abs_contrib_loops(a, b, c, hr):
    """Per-bucket sums of absolute contributions written out with explicit loops: for bucket
    (a, b), sum_k (sum_{i in a} w|A_ik|)(sum_{j in b} w|B_kj|) + sum_{i in a, j in b} w|C_ij|,
    with w = 1 for S, w_i = (i+1)/2^ceil(log2 n1) for R and w_j = (j+1)/2^ceil(log2 n3) for T."""
    n1, n2 = a.shape
    n3 = b.shape[1]
    m = hr.m
    L1 = 1
    while L1 < n1:
        L1 *= 2
    L3 = 1
    while L3 < n3:
        L3 *= 2
    out = {name: np.zeros((m, m)) for name in "SRT"}
    for ba in range(m):
        rows = [i for i in range(n1) if hr.h1[i] == ba]
        for bb in range(m):
            cols = [j for j in range(n3) if hr.h2[j] == bb]
            for name in "SRT":
                wi = (lambda i: (i + 1) / L1) if name == "R" else (lambda i: 1.0)
                wj = (lambda j: (j + 1) / L3) if name == "T" else (lambda j: 1.0)
                tot = 0.0
                for k in range(n2):
                    sa = sum(wi(i) * abs(a[i, k]) for i in rows)
                    sb = sum(wj(j) * abs(b[k, j]) for j in cols)
                    tot += sa * sb
                for i in rows:
                    for j in cols:
                        tot += wi(i) * wj(j) * abs(c[i, j])
                out[name][ba, bb] = tot
    return out["S"], out["R"], out["T"]


def test_abs_contributions_against_explicit_sums():
    """The float-parity scale D^S, D^R, D^T (the sum of absolute contributions of the factored
    evaluation of Eq. 1 and of the first-moment sketches) against its definition evaluated with
    plain loops, on a ragged case whose buckets are of unequal size."""
    rng = np.random.default_rng(11)
    n1, n2, n3, m = 7, 5, 9, 3
    a = rng.standard_normal((n1, n2))
    b = rng.standard_normal((n2, n3))
    c = rng.standard_normal((n1, n3))
    hr = o.make_round(5, 1, n1, n3, m)
    assert len(set(np.bincount(hr.h1, minlength=m))) > 1   # buckets of unequal size
    DS, DR, DT = o.abs_contributions(a, b, c, hr)
    eS, eR, eT = _abs_contrib_loops(a, b, c, hr)
    for got, exp in ((DS, eS), (DR, eR), (DT, eT)):
        assert np.allclose(got, exp, rtol=1e-13, atol=0.0)
    # R weights rows and T weights columns: the three scales differ
    assert not np.allclose(DR, DT) and not np.allclose(DS, DR)


def test_abs_contributions_bounds_fp32_evaluation_of_eq1():
    """What the scale is for: an FP32 evaluation of the factored form (H1 A)(B H2^T) - H1 C H2^T
    differs from the exact S by a small multiple of 2^-24 D^S per bucket (a sum of n terms in
    FP32 errs by at most about n 2^-24 times the sum of their magnitudes)."""
    rng = np.random.default_rng(3)
    n1, n2, n3, m = 64, 48, 40, 4
    a = rng.standard_normal((n1, n2)).astype(np.float32).astype(np.float64)
    b = rng.standard_normal((n2, n3)).astype(np.float32).astype(np.float64)
    c = (a @ b).astype(np.float32).astype(np.float64)
    hr = o.make_round(9, 0, n1, n3, m)
    S, _, _ = o.sketches(o.error_matrix(a, b, c), hr, moments=False)
    H1 = np.zeros((m, n1), dtype=np.float32)
    H1[hr.h1, np.arange(n1)] = hr.v1
    H2 = np.zeros((m, n3), dtype=np.float32)
    H2[hr.h2, np.arange(n3)] = hr.v2
    a32, b32, c32 = a.astype(np.float32), b.astype(np.float32), c.astype(np.float32)
    s32 = (H1 @ a32) @ (b32 @ H2.T) - H1 @ c32 @ H2.T
    DS, _, _ = o.abs_contributions(a, b, c, hr)
    err = np.abs(s32.astype(np.float64) - S)
    assert np.all(err <= (n1 + n2 + n3) * 2.0 ** -24 * DS)
    assert err.max() > 0.0        # the FP32 evaluation does round


def test_scaling_limits():
    for row in load_golden("scaling_limits.csv"):
        n1, n2, n3 = int(row["n1"]), int(row["n2"]), int(row["n3"])
        q, v = row["quantity"], float(row["value"])
        if q == "m_num_bf16":
            assert o.m_num(n1, n2, n3, "bf16", P) == v
        elif q == "m_start_bf16":
            assert o.m_start(n1, n2, n3, "bf16", P) == v
        elif q == "sketch_gib_at_m_num":
            m = o.m_num(n1, n2, n3, "bf16", P)
            assert abs(3 * m * m * 4 / 2 ** 30 - v) < 0.05
        elif q == "m_max":
            assert o.m_max(n1, n3) == v


def test_m_comb_default_budget():
    assert o.m_comb(P) == 48          # ceil(max(3*2*8, sqrt(3*2*16)))
    assert o.m_comb(o.Params(s_budget=32)) == 48
    assert o.m_comb(o.Params(delta_rc=1, s_budget=600)) == 60   # sqrt(3600) = 60


def test_m_mem_quadratic_root():
    for n2 in (256, 4096, 11008, 16384):
        # 12 m^2 + 24 n2 m - 2^31 = 0
        root = (-24 * n2 + math.sqrt((24 * n2) ** 2 + 4 * 12 * 2 ** 31)) / 24
        assert o.m_mem(n2) == math.floor(root)
    assert o.m_mem(4096) == 9894


def test_radius_rule():
    assert o.radius_rule(0.05) == 0
    assert o.radius_rule(0.0500001) == 2
    assert o.radius_rule(0.79) == 2       # ceil(1.975) = 2
    assert o.radius_rule(0.81) == 3       # ceil(2.025) = 3
    assert o.radius_rule(10.0) == 25


def test_plan_small_budget_keeps_m():
    # B = 4096 * 1e-5 / (0.02 * 64) = 0.032 <= 0.05 -> r = 0, m_loc = m
    pl = o.plan_localize(4096, 4096, 4096, "bf16", 48, 1e-5, 64.0, P)
    assert (pl.m_loc, pl.r) == (48, 0)
    # B = 4096 * 5e-5 / 1.28 = 0.16 -> r_B = 2 <= r* -> m_loc = m, r = 2
    pl = o.plan_localize(4096, 4096, 4096, "bf16", 48, 5e-5, 64.0, P)
    assert (pl.m_loc, pl.r) == (48, 2)


def test_plan_growth_and_caps():
    p = o.Params(rho_min=0.015)
    # B = 4096 * 0.004 / (0.015 * 64) = 17.0667; r_B = ceil(42.67) = 43
    # m_loc = 16 ceil(ceil(48 * 43 / 4) / 16) = 16 ceil(516/16) = 528; B' = B*48/528 = 1.5515
    # r = max(2, ceil(3.88)) = 4
    pl = o.plan_localize(4096, 4096, 4096, "bf16", 48, 0.004, 64.0, p)
    assert (pl.m_loc, pl.r) == (528, 4)
    # huge noise: m_loc capped at m_max = 1024 and r capped at r_max
    pl = o.plan_localize(4096, 11008, 4096, "bf16", 68, 0.5, 1.0, P)
    assert pl.m_loc == 1024 and pl.r == 16
    # memory cap: n2 large enough that m_mem < m_max
    pl = o.plan_localize(65536, 1 << 20, 65536, "bf16", 48, 0.5, 1.0, P)
    assert pl.m_loc == o.m_mem(1 << 20)


def test_plan_fallback_to_law():
    pl = o.plan_localize(4096, 4096, 4096, "bf16", 48, float("nan"), 64.0, P)
    assert pl.fallback
    B = 4096 * o.law_sigma_over_rms(4096, 4096, 4096, 48, "bf16", P) / P.rho_min
    assert abs(pl.B - B) < 1e-12
    assert o.plan_localize(4096, 4096, 4096, "bf16", 48, 0.0, 64.0, P).fallback
    assert o.plan_localize(4096, 4096, 4096, "bf16", 48, 1e-3, float("inf"), P).fallback


def test_recalibration_rule():
    # B1 = 4096 * 0.0075 / 64 = 0.48; m' = max(48, 16, min(ceil(48*0.48/0.3), 1024)) = 77
    m, rebuild = o.recalibrate_m(4096, 4096, 48, 0.0075, 64.0, P)
    assert (m, rebuild) == (77, True)
    # within the +-25 % band: keep m
    m, rebuild = o.recalibrate_m(4096, 4096, 48, 0.0045, 64.0, P)   # m' = 48
    assert (m, rebuild) == (48, False)
    m, rebuild = o.recalibrate_m(4096, 4096, 100, 0.0045, 64.0, P)  # m' = ceil(96)=96
    assert (m, rebuild) == (100, False)
    # never below m_comb
    m, rebuild = o.recalibrate_m(4096, 4096, 200, 1e-6, 64.0, P)
    assert (m, rebuild) == (48, True)


def test_rms_hat():
    rng = np.random.Generator(np.random.PCG64(6))
    c = (rng.standard_normal((512, 512)) * 3.0).astype(np.float32)
    assert abs(o.rms_hat(c) / 3.0 - 1) < 0.01
    c2 = c.copy()
    c2[0, 0] = np.nan            # sampled (stride 4 in row-major order), excluded
    c2[0, 4] = np.inf            # sampled, excluded
    c2[0, 8] = 1e30              # sampled, clipped at 64 x median
    r = o.rms_hat(c2)
    samp = np.abs(c.ravel()[::4].astype(np.float64))
    samp = np.delete(samp, [0, 1])
    samp[0] = 1e30
    clip = 64 * o.median(samp)
    assert abs(r - math.sqrt(np.mean(np.minimum(samp, clip) ** 2))) < 1e-9
    assert math.isnan(o.rms_hat(np.full((4, 4), np.nan, dtype=np.float32)))


def test_window_order():
    offs = o.window_offsets(1)
    assert offs[0] == (0, 0)
    assert offs[1:5] == [(-1, 0), (0, -1), (0, 1), (1, 0)]
    assert offs[5:] == [(-1, -1), (-1, 1), (1, -1), (1, 1)]
    assert len(o.window_offsets(4)) == 81


# --- additional pins (each targets a specific plausible slip) ------------------------------

def test_hash_word_reduction_on_published_outputs():
    """The hash reduces each splitmix64 output word x to bucket (x >> 32) * m >> 32 and sign -1
    iff bit 0 of x is set; the words here are the published outputs for state 1234567, which are
    the words of indices 0..4 of the stream keyed with 1234567."""
    rows = [r for r in load_golden("splitmix64_vectors.csv") if r["seed"] == "1234567"]
    words = [int(r["output"]) for r in rows]
    got_x = o.splitmix64_stream(1234567, np.arange(5, dtype=np.uint64))
    assert [int(v) for v in got_x] == words
    for m in (1, 7, 48, 1000, 65535):
        b, s = o.bucket_sign_from_word(np.array(words, dtype=np.uint64), m)
        assert list(b) == [((w >> 32) * m) >> 32 for w in words]
        assert list(s) == [-1.0 if w & 1 else 1.0 for w in words]
    # words 1234567/0 = ...05 (odd) and /1 = ...73 (odd): negative signs; /3 = ...31 (odd)
    assert words[0] % 2 == 1


def test_round_key_uses_stream_index_2t_plus_side():
    seed = 1234567
    rows = [int(r["output"]) for r in load_golden("splitmix64_vectors.csv") if r["seed"] == "1234567"]
    assert o.round_key(seed, 0, 0) == rows[0]
    assert o.round_key(seed, 0, 1) == rows[1]
    assert o.round_key(seed, 1, 0) == rows[2]
    assert o.round_key(seed, 2, 0) == rows[4]


def test_clipped_mean_clips_at_five_means():
    """Sec. III-E: sigma_hat = 1.2533 mean(min(|S|, 5 mean|S|)); with 99 unit buckets and one
    of 1000, mean|S| = 10.99, the outlier is clipped to 54.95."""
    S = np.array([1.0] * 99 + [-1000.0])
    assert abs(o.clipped_sigma(S) - 1.2533 * (99 + 54.95) / 100) < 1e-12


def test_probe_threshold_closed_form():
    """thr = min(tau, mu sqrt(2 ln m^2) sigma_hat): m = 10 gives sqrt(2 ln 100) = 3.0349."""
    S = np.ones((10, 10))
    S[0, 0] = 14.0
    # mean|S| = 1.13, all below 5.65 except 14 -> clipped: mean(min) = (99 + 5.65)/100
    sig = 1.2533 * (99 + 5.65) / 100
    pr = o.probe_from_sketch(S, 8, 1.0, 1.0, o.Params(c_valid=1e12))
    assert abs(pr.thr - 4 * math.sqrt(2 * math.log(100)) * sig) < 1e-9
    assert not pr.dirty                 # 14 <= 4 * 3.0349 * 1.3116 = 15.92
    S[0, 0] = 17.0                      # mean|S| 1.16, clip 5.8, thr = 4 * 3.0349 * 1.3135
    pr = o.probe_from_sketch(S, 8, 1.0, 1.0, o.Params(c_valid=1e12))
    assert abs(pr.thr - 4 * math.sqrt(2 * math.log(100)) * 1.2533 * 1.048) < 1e-9
    assert pr.dirty
    # the analytic tau caps the threshold
    pr2 = o.probe_from_sketch(S, 8, 1.0, 1.0, o.Params())
    assert pr2.thr == pr2.tau == 100 * 8 * 2.0 ** -23


def test_window_order_chebyshev_before_manhattan():
    """Offsets by Chebyshev then Manhattan distance: the whole 3x3 ring precedes (+-2, 0)."""
    offs = o.window_offsets(2)
    assert set(offs[:9]) == {(a, b) for a in (-1, 0, 1) for b in (-1, 0, 1)}
    assert offs[9:13] == [(-2, 0), (0, -2), (0, 2), (2, 0)]
    assert len(offs) == 25 and len(set(offs)) == 25


def test_rms_hat_stride_is_floor_of_count_over_65536():
    """n1 n3 = 131070: stride floor(131070/65536) = 1, so every entry is sampled."""
    c = np.ones((510, 257), dtype=np.float32)
    c.ravel()[1::2] = 3.0                       # odd flat positions 3, even 1
    expect = math.sqrt((65535 * 1.0 + 65535 * 9.0) / 131070)
    assert abs(o.rms_hat(c) - expect) < 1e-12


def test_recalibration_band_is_25_percent():
    # m' = ceil(100 * B1 / 0.3) with B1 = 4096 * sigma / 64: sigma = 0.006094 -> m' = 131 > 125
    m, rebuild = o.recalibrate_m(4096, 4096, 100, 0.006094, 64.0, P)
    assert (m, rebuild) == (131, True)
    m, rebuild = o.recalibrate_m(4096, 4096, 100, 0.0055, 64.0, P)   # m' = 118 in band
    assert (m, rebuild) == (100, False)


def test_candidate_cap_K():
    """K = max(64, 8 s) (Sec. III-E): s = 16 -> 128 (the cap Table VI runs into)."""
    assert o.Params().K == 128
    assert o.Params(s_budget=4).K == 64
    assert o.Params(s_budget=32).K == 256
