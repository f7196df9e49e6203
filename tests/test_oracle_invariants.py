"""Invariants of the oracle's probe and localizer (Lemma 1, Theorem 1-2, exact special cases,
brute force on tiny inputs)."""
import itertools
import math

import numpy as np
import pytest

from oracle import fpsketch_oracle as o
from paper_2609_19758_amd import workloads as wl

P = o.Params()


def _int_case(n1, n2, n3, seed, lo=-4, hi=4):
    """Small-integer operands: exact in both half formats; C = AB exactly in FP32."""
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, "bf16", ("int", lo, hi), ("int", lo, hi), seed)
    a64, b64 = o.decode_bf16(a_bits), o.decode_bf16(b_bits)
    c = (a64 @ b64).astype(np.float32)
    assert np.array_equal(c.astype(np.float64), a64 @ b64)
    return a64, b64, c


def test_exact_single_error_recovery():
    """Integer operands, C = AB, one integer fault: one nonzero bucket equal to v1 v2 delta,
    sigma_MAD = 0 so the cuts vanish, r = 0 and F = {(i, j, delta)} exactly."""
    a64, b64, c = _int_case(96, 40, 80, 1)
    i, j, fault = 37, 61, 5.0
    cf = c.copy()
    cf[i, j] += fault
    E = o.error_matrix(a64, b64, cf)
    hr = o.make_round(12, 1, 96, 80, 16)
    S, R, T = o.sketches(E, hr)
    assert np.count_nonzero(S) == 1
    assert S[hr.h1[i], hr.h2[j]] == -hr.v1[i] * hr.v2[j] * fault
    assert o.mad_sigma(S) == 0.0
    res = o.localize(a64, b64, cf, "bf16", 16, seed=12, p=P, plan=o.Plan(16, 0, 0.0, False))
    assert [(f.i, f.j, f.delta, f.absolute) for f in res.faults] == [(i, j, -fault, False)]


def test_probe_clean_and_dirty_exact():
    a64, b64, c = _int_case(64, 32, 48, 2)
    hr = o.make_round(1, 0, 64, 48, 8)
    pr = o.probe(a64, b64, c, hr, P)
    assert not pr.dirty and pr.sigma_hat == 0.0 and pr.max_abs == 0.0
    cf = c.copy()
    cf[5, 7] += 1.0
    assert o.probe(a64, b64, cf, hr, P).dirty


@pytest.mark.parametrize("bad", [np.nan, np.inf, -np.inf, 3e37])
def test_probe_nonfinite_and_huge_are_dirty(bad):
    a64, b64, c = _int_case(64, 32, 48, 3)
    cf = c.copy()
    cf[10, 20] = bad
    pr = o.probe(a64, b64, cf, o.make_round(1, 0, 64, 48, 8), P)
    assert pr.dirty


def _isolated_somewhere(faults, seed, rounds, n1, n3, m):
    """Every fault shares its bucket with no other fault in at least one round."""
    for (i, j) in faults:
        ok = False
        for t in range(1, rounds + 1):
            hr = o.make_round(seed, t, n1, n3, m)
            cell = (hr.h1[i], hr.h2[j])
            if all((hr.h1[a], hr.h2[b]) != cell for (a, b) in faults if (a, b) != (i, j)):
                ok = True
                break
        if not ok:
            return False
    return True


def test_brute_force_tiny():
    """n1, n3 <= 32, n2 <= 16, m = 8, 1-6 integer faults: F is a subset of the brute-force set
    {(i, j): |E_ij| > tau_ij} and equals it whenever every fault is isolated in some round."""
    rng = np.random.Generator(np.random.PCG64(99))
    checked_equal = 0
    for case in range(60):
        n1, n2, n3 = int(rng.integers(8, 33)), int(rng.integers(4, 17)), int(rng.integers(8, 33))
        a64, b64, c = _int_case(n1, n2, n3, 1000 + case, -3, 3)
        nf = int(rng.integers(1, 7))
        sites = wl.fault_sites(n1, n3, nf, 2000 + case)
        deltas = rng.integers(1, 9, size=nf) * np.where(rng.integers(0, 2, size=nf) == 1, -1, 1)
        cf = wl.inject_additive(c, sites, deltas)
        E = o.error_matrix(a64, b64, cf)
        truth = {(i, j) for i in range(n1) for j in range(n3)
                 if abs(E[i, j]) > o.validation_bound(a64, b64, i, j, P)}
        assert truth == {tuple(s) for s in sites.tolist()}
        seed = 3000 + case
        res = o.localize(a64, b64, cf, "bf16", 8, seed, P, plan=o.Plan(8, 0, 0.0, False))
        got = {(f.i, f.j) for f in res.faults}
        assert got <= truth
        for f in res.faults:
            assert f.delta == E[f.i, f.j]
        if _isolated_somewhere(sorted(truth), seed, P.rounds, n1, n3, 8):
            assert got == truth
            checked_equal += 1
    assert checked_equal >= 30


def test_zero_false_positives_gaussian():
    """Lemma 1: every accepted coordinate is a corrupted entry, on float products with noise."""
    n1, n2, n3 = 192, 96, 160
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, "bf16", ("normal", 1.0), ("normal", 1.0), 5)
    c = wl.cpu_gemm_f32(a_bits, b_bits, "bf16")
    a64, b64 = o.decode_bf16(a_bits), o.decode_bf16(b_bits)
    sites = wl.fault_sites(n1, n3, 6, 6)
    deltas = wl.fault_magnitudes(6, 0.5, 4.0, wl.mean_abs(c), 7)
    cf = wl.inject_additive(c, sites, deltas)
    m = 32
    pr = o.probe(a64, b64, cf, o.make_round(1, 0, n1, n3, m), P)
    assert pr.dirty
    res = o.localize(a64, b64, cf, "bf16", m, 21, P, sigma_probe=pr.sigma_hat)
    injected = {tuple(s) for s in sites.tolist()}
    E = o.error_matrix(a64, b64, cf)
    for f in res.faults:
        assert (f.i, f.j) in injected
        assert abs(E[f.i, f.j]) > o.validation_bound(a64, b64, f.i, f.j, P)
    # faults of 0.5-4 x mean|C| are far above the noise: all recovered, delta = -fault
    assert {(f.i, f.j) for f in res.faults} == injected
    for f in res.faults:
        k = [tuple(s) for s in sites.tolist()].index((f.i, f.j))
        assert abs(f.delta + (np.float64(cf[f.i, f.j]) - np.float64(c[f.i, f.j]))) <= \
            1e-3 * abs(f.delta)


def test_clean_float_product_probe_is_clean():
    n1, n2, n3 = 256, 256, 256
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, "fp16", ("uniform", -1, 1), ("uniform", -1, 1), 1)
    c = wl.cpu_gemm_f32(a_bits, b_bits, "fp16")
    a64, b64 = o.decode_fp16(a_bits), o.decode_fp16(b_bits)
    for seed in range(4):
        pr = o.probe(a64, b64, c, o.make_round(seed, 0, n1, n3, 64), P)
        assert not pr.dirty
        assert pr.thr < pr.tau


def test_nonfinite_scan_and_patch():
    """Sec. III-I: non-finite and out-of-range entries are found by the exact scan in row-major
    order, recomputed as absolute values, and do not poison the other faults' buckets."""
    a64, b64, c = _int_case(64, 24, 64, 8)
    cf = c.copy()
    cf[3, 9] = np.inf
    cf[3, 2] = np.nan
    cf[40, 1] = -5e37
    cf[20, 30] += 6.0          # a finite fault sharing no special structure
    res = o.localize(a64, b64, cf, "bf16", 16, 5, P, plan=o.Plan(16, 0, 0.0, False))
    absf = [(f.i, f.j) for f in res.faults if f.absolute]
    assert absf == [(3, 2), (3, 9), (40, 1)]
    for f in res.faults:
        if f.absolute:
            assert f.delta == float(a64[f.i] @ b64[:, f.j])
    fin = [(f.i, f.j, f.delta) for f in res.faults if not f.absolute]
    assert fin == [(20, 30, -6.0)]


def test_peeling_across_rounds_unlocks_mixture():
    """Sec. III-H: a fault confirmed in one round is subtracted from the next round's sketches,
    so a bucket that mixed two faults becomes a singleton."""
    a64, b64, c = _int_case(128, 16, 128, 9)
    # find a seed where faults x and y collide in round 1 (and x is isolated in round 1? no:
    # they share the bucket) but each is isolated in round 2 after peeling of x.
    x, y, z = (10, 20), (50, 90), (100, 5)
    seed = None
    for s in range(2000):
        h1 = o.make_round(s, 1, 128, 128, 4)
        h2 = o.make_round(s, 2, 128, 128, 4)
        col1 = (h1.h1[x[0]], h1.h2[x[1]]) == (h1.h1[y[0]], h1.h2[y[1]])
        # in round 2, y shares with z only; x is isolated
        cx = (h2.h1[x[0]], h2.h2[x[1]])
        cy = (h2.h1[y[0]], h2.h2[y[1]])
        cz = (h2.h1[z[0]], h2.h2[z[1]])
        z1 = (h1.h1[z[0]], h1.h2[z[1]])
        if col1 and z1 != (h1.h1[x[0]], h1.h2[x[1]]) and cy == cz and cx != cy:
            seed = s
            break
    assert seed is not None
    cf = c.copy()
    for (i, j), d in ((x, 3.0), (y, -4.0), (z, 2.0)):
        cf[i, j] += d
    p1 = o.Params(rounds=2)
    res = o.localize(a64, b64, cf, "bf16", 4, seed, p1, plan=o.Plan(4, 0, 0.0, False))
    got = {(f.i, f.j): f.round for f in res.faults}
    # round 1 finds z (isolated); x, y mixed.  Round 2: x isolated -> found; y+z mixed but z is
    # peeled, so y becomes a singleton -> found.
    assert got.get(z) == 1
    assert got.get(x) == 2 and got.get(y) == 2


def _noise_case(n1, n2, n3, seed, noise=1e-3):
    rng = np.random.Generator(np.random.PCG64(seed))
    a64, b64, c = _int_case(n1, n2, n3, seed)
    cn = (c.astype(np.float64) + rng.standard_normal(c.shape) * noise).astype(np.float32)
    return a64, b64, cn


def test_tau_c_clean_bucket_rate_inside_a_round():
    """Sec. III-E puts the share of clean buckets above tau_c = min(tau, 2 sigma_MAD) near
    4.6 % (two-sided Gaussian tail at 2 sigma); a round must see that share."""
    # bucket populations of ~64 x 64 entries keep S close to Gaussian
    a64, b64, cn = _noise_case(4096, 4, 4096, 31)
    E = o.error_matrix(a64, b64, cn)
    hr = o.make_round(2, 1, 4096, 4096, 64)
    tr = []
    o.localize_round(a64, b64, E, hr, 4, 1e9, [], P, 1, tr)
    frac = tr[0].n_above_tau_c / 64 ** 2
    assert 0.038 < frac < 0.056
    assert abs(tr[0].tau_c - 2 * tr[0].sigma_mad) < 1e-15


def test_tau_d_uses_larger_output_dimension():
    """tau_d = max(n1, n3) sigma_MAD / max(r, 1/2): with n1 = 64 and n3 = 2048 a fault whose
    bucket value lies between min(n1, n3) sigma / r and max(n1, n3) sigma / r is not selected."""
    a64, b64, cn = _noise_case(64, 8, 2048, 32, noise=1e-2)
    E0 = o.error_matrix(a64, b64, cn)
    hr = o.make_round(5, 1, 64, 2048, 64)
    tr = []
    o.localize_round(a64, b64, E0, hr, 4, 1e9, [], P, 1, tr)
    sig = tr[0].sigma_mad
    assert abs(tr[0].tau_d - 2048 * sig / 4) < 1e-12
    cf = cn.copy()
    i, j = 10, 700
    cf[i, j] -= np.float32(20 * 64 * sig / 4)        # |S| ~ 20 x (64 sigma / r): well above the
    E = o.error_matrix(a64, b64, cf)                   # min-form cut, below the max-form 512 x
    F = o.localize_round(a64, b64, E, hr, 4, 1e9, [], P, 1, [])
    assert (i, j) not in {(f.i, f.j) for f in F}


def test_rounding_bound_uses_absolute_products():
    """tau_ij = c eps sum_k |A_ik||B_kj| (Sec. III-D): a change below that bound at an entry
    whose products cancel (A_i,* B_*,j = 0 with sum |A||B| = 16) is not accepted."""
    n1 = n2 = n3 = 16
    a64 = np.zeros((n1, n2))
    b64 = np.zeros((n2, n3))
    a64[3, :] = np.tile([1.0, -1.0], 8)
    b64[:, 5] = 1.0
    a64[7, :] = 1.0
    b64[:, 9] = 1.0
    c = (a64 @ b64).astype(np.float32)
    bound_35 = 100 * 2.0 ** -23 * 16          # 1.9e-4
    cf = c.copy()
    cf[3, 5] = np.float32(1e-4)               # below its bound although AB_35 = 0
    E = o.error_matrix(a64, b64, cf)
    assert abs(E[3, 5]) < bound_35
    F = o.localize_round(a64, b64, E, o.make_round(1, 1, n1, n3, 4), 0, 1e9, [], P, 1, [])
    assert (3, 5) not in {(f.i, f.j) for f in F}
    cf[3, 5] = np.float32(1e-3)               # above it: accepted
    E = o.error_matrix(a64, b64, cf)
    F = o.localize_round(a64, b64, E, o.make_round(1, 1, n1, n3, 4), 0, 1e9, [], P, 1, [])
    assert (3, 5) in {(f.i, f.j) for f in F}


def test_absolute_entries_leave_no_trace_in_the_sketch():
    """Sec. III-I: while sketching, C holds the recomputed value of each absolute entry, so on
    exact inputs the only nonzero bucket of a round is the finite fault's."""
    a64, b64, c = _int_case(64, 24, 64, 8)
    cf = c.copy()
    cf[3, 9] = np.inf
    cf[40, 1] = -5e37
    cf[20, 30] += 6.0
    res = o.localize(a64, b64, cf, "bf16", 16, 5, P, plan=o.Plan(16, 0, 0.0, False))
    assert np.count_nonzero(res.trace[0].S) == 1


def test_candidate_cap_limits_one_round():
    """At most K candidates per round (Sec. III-E; Table VI's cap): 200 exact isolated faults,
    one round, K = 128 -> exactly the 128 largest are recovered."""
    n1 = n3 = 1024
    a64, b64, c = _int_case(n1, 8, n3, 41)
    m = 1024
    hr = o.make_round(77, 1, n1, n3, m)
    # 200 faults in distinct buckets with distinct magnitudes
    rng = np.random.Generator(np.random.PCG64(3))
    cells, sites = set(), []
    while len(sites) < 200:
        i, j = int(rng.integers(0, n1)), int(rng.integers(0, n3))
        cell = (hr.h1[i], hr.h2[j])
        if cell not in cells:
            cells.add(cell)
            sites.append((i, j))
    mags = np.arange(1, 201, dtype=np.float64)
    cf = c.copy()
    for (i, j), d in zip(sites, mags):
        cf[i, j] += d
    E = o.error_matrix(a64, b64, cf)
    F = o.localize_round(a64, b64, E, hr, 0, 1e9, [], P, 1, [])
    got = {(f.i, f.j) for f in F}
    assert len(got) == 128
    assert got == set(sites[72:])           # the 128 largest magnitudes


def test_search_is_offset_major():
    """The validated search visits offsets in the outer loop and buckets in the inner one
    (Sec. III-E): at offset (0, 0) bucket 2 claims (5, 6) at its own center, so bucket 1, whose
    window also holds (5, 6), passes over it and never reaches (5, 7), which lies outside its
    window.  Searching bucket by bucket instead would let bucket 1 claim (5, 6) and bucket 2 then
    claim (5, 7)."""
    n1 = n3 = 12
    P = o.Params()
    a64 = np.full((n1, 2), 0.01)
    b64 = np.full((2, n3), 0.01)            # validation bounds of about 2.4e-9
    E = np.zeros((n1, n3))
    E[5, 6] = E[5, 7] = 1.0
    F = o.search_windows([10, 20], {10: (5, 5), 20: (5, 6)}, E, a64, b64, 1, [], P, 1)
    assert [(f.i, f.j, f.round) for f in F] == [(5, 6, 1)]
    # a coordinate outside C is passed over and the bucket goes on searching
    E2 = np.zeros((n1, n3))
    E2[0, 1] = -2.0
    F2 = o.search_windows([7], {7: (0, 0)}, E2, a64, b64, 1, [], P, 2)
    assert [(f.i, f.j, f.delta) for f in F2] == [(0, 1, -2.0)]
    # an entry already found is not found again, and a bucket without a center is skipped
    F3 = o.search_windows([7, 8], {7: (0, 0)}, E2, a64, b64, 1, list(F2), P, 3)
    assert len(F3) == 1
