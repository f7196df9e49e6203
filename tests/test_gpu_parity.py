"""GPU parity of the HIP path (through the C ABI) against the CPU FP64 oracle.

Bar: bit-exact sketches, verdicts and fault sets on small-integer inputs where every step is
exact in both implementations; on float inputs, sketches within 1e-4 of the sum of absolute
contributions per bucket (and within 2^-20 of it, a bound derived from FP32 storage of the
factors), identical verdicts and fault sets, fault magnitudes within 1e-3 relative.
"""
import math

import numpy as np
import pytest

from oracle import fpsketch_oracle as o
from paper_2609_19758_amd import workloads as wl
from gpu_util import gemm_f32, int_case, to_dev_f32, to_dev_half

pytestmark = pytest.mark.gpu

P = o.Params()


@pytest.fixture(scope="module")
def fk():
    import torch
    assert torch.cuda.is_available()
    from paper_2609_19758_amd import fpsketch
    fpsketch.load()
    return fpsketch


def _dev(a_bits, b_bits, c, fmt):
    return to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt), to_dev_f32(c)


# --- sketches --------------------------------------------------------------------------------

EXACT_CASES = [
    # n1, n2, n3, m, fmt : exercises (RB, G) paths, ragged tiles, unaligned rows, size 1
    (256, 256, 256, 64, "fp16"),
    (200, 72, 136, 13, "bf16"),
    (130, 37, 131, 7, "bf16"),          # n2 % 8 != 0 and n3 % 4 != 0: element loads
    (1, 1, 1, 1, "fp16"),
    (1, 8, 300, 4, "bf16"),
    (300, 3, 1, 2, "fp16"),
    (1000, 40, 700, 300, "bf16"),       # G = 2
    (300, 520, 9000, 400, "fp16"),      # G = 2 over three B chunks, the last partial
    (600, 24, 1100, 700, "fp16"),       # RB = 4, G = 4
    (300, 1030, 700, 600, "fp16"),      # RB = 4 over 258 row blocks: XCD-grouped order, ragged
    (300, 24, 6145, 300, "bf16"),       # C tiles one per wave, element loads, last group 1 tile
    (2000, 8, 7000, 1000, "fp16"),      # C tiles one per wave, G = 4, 7 tiles per group
    (1000, 64, 2560, 100, "bf16"),      # C tiles one per wave at m <= 192: padded lists, 3 tiles
    (600, 40, 4104, 160, "fp16"),       # the same over 9 tiles (groups of 3, the last partial)
    (400, 16, 3000, 1500, "bf16"),      # RB = 2, G = 8
    (700, 8, 5000, 4096, "fp16"),       # RB = 1, G = 16, m at the limit
    (2100, 520, 1030, 48, "bf16"),      # several A/C tiles and a ragged tail
    (100, 37, 90, 13, "fp16"),          # small buckets (one wave per tile), element loads
    (300, 2100, 200, 64, "bf16"),       # small buckets over 5 tiles: waves past the last idle
    (600, 64, 8192, 64, "bf16"),        # B chunks from (row block mod 2) on: two whole chunks
    (300, 40, 12288, 100, "fp16"),      # the same over three whole chunks (every rotation)
]


@pytest.mark.parametrize("n1,n2,n3,m,fmt", EXACT_CASES)
def test_sketches_bit_exact_on_integer_inputs(fk, n1, n2, n3, m, fmt):
    a_bits, b_bits, a64, b64, c = int_case(n1, n2, n3, fmt, seed=n1 + n2 + n3)
    cf = c.copy()
    nf = min(5, n1 * n3)
    sites = wl.fault_sites(n1, n3, nf, 9)
    for k, (i, j) in enumerate(sites):
        cf[i, j] += np.float32(k + 1)
    A, B, C = _dev(a_bits, b_bits, cf, fmt)
    v = fk.Verifier(n1, n2, n3, fmt, m=m)
    for seed, rnd in ((7, 0), (11, 2)):
        S, R, T, ma, mb = v.sketch(A, B, C, seed, rnd, m, moments=True)
        hr = o.make_round(seed, rnd, n1, n3, m)
        oS, oR, oT = o.sketches(o.error_matrix(a64, b64, cf), hr)
        assert np.array_equal(S, oS)
        assert np.array_equal(R, oR)
        assert np.array_equal(T, oT)
        assert ma == np.max(np.abs(a64)) and mb == np.max(np.abs(b64))
        S2, _, _, _, _ = v.sketch(A, B, C, seed, rnd, m, moments=False)
        assert np.array_equal(S2, oS)
    v.close()


def test_sketches_float_within_contract_and_fp32_bound(fk):
    n1, n2, n3, m = 640, 1024, 768, 48
    fmt = "bf16"
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, ("normal", 1.0), ("normal", 1.0), 3)
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    C = gemm_f32(A, B)
    c = C.cpu().numpy()
    sites = wl.fault_sites(n1, n3, 4, 4)
    cf = wl.inject_additive(c, sites, wl.fault_magnitudes(4, 0.02, 0.09, wl.mean_abs(c), 5))
    Cf = to_dev_f32(cf)
    a64, b64 = o.decode(a_bits, fmt), o.decode(b_bits, fmt)
    v = fk.Verifier(n1, n2, n3, fmt, m=m)
    S, R, T, _, _ = v.sketch(A, B, Cf, 5, 1, m)
    hr = o.make_round(5, 1, n1, n3, m)
    oS, oR, oT = o.sketches(o.error_matrix(a64, b64, cf), hr)
    DS, DR, DT = o.abs_contributions(a64, b64, cf.astype(np.float64), hr)
    for g, r_, d in ((S, oS, DS), (R, oR, DR), (T, oT, DT)):
        err = np.abs(g - r_)
        assert np.all(err <= 1e-4 * d)
        assert np.all(err <= 2.0 ** -20 * d)
    # determinism: no atomics, fixed reduction orders
    S2, R2, T2, _, _ = v.sketch(A, B, Cf, 5, 1, m)
    assert np.array_equal(S, S2) and np.array_equal(R, R2) and np.array_equal(T, T2)
    v.close()


# --- probe -----------------------------------------------------------------------------------

def test_probe_verdicts_match_oracle(fk):
    import torch
    n1, n2, n3 = 512, 768, 640
    fmt = "fp16"
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, ("normal", 1.0), ("normal", 0.02), 6)
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    c = gemm_f32(A, B).cpu().numpy()
    a64, b64 = o.decode(a_bits, fmt), o.decode(b_bits, fmt)
    v = fk.Verifier(n1, n2, n3, fmt)
    m = v.m
    hr = o.make_round(v.params.seed, 0, n1, n3, m)
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    sites = wl.fault_sites(n1, n3, 3, 7)
    dirty_c = wl.inject_additive(c, sites, wl.fault_magnitudes(3, 0.5, 2.0, wl.mean_abs(c), 8))
    for cc, expect_dirty in ((c, False), (dirty_c, True)):
        flag.zero_()
        v.probe(A, B, to_dev_f32(cc), d_dirty=flag)
        st = v.probe_stats()
        ref = o.probe(a64, b64, cc, hr, P)
        assert bool(st["dirty"]) == ref.dirty == expect_dirty
        assert int(flag.item()) == int(expect_dirty)
        assert abs(st["sigma_hat"] / ref.sigma_hat - 1) < 0.05
        assert abs(st["tau"] / ref.tau - 1) < 1e-12
        # on a clean product max|S| is itself noise: compare within the FP32-storage bound
        DS, _, _ = o.abs_contributions(a64, b64, cc.astype(np.float64), hr)
        assert abs(st["max_abs"] - ref.max_abs) <= 2.0 ** -20 * DS.max()
    v.close()


@pytest.mark.parametrize("bad", [float("nan"), float("inf"), -float("inf"), 3e37])
def test_probe_nonfinite_and_huge_entries_are_dirty(fk, bad):
    import torch
    a_bits, b_bits, a64, b64, c = int_case(128, 64, 96, "bf16", 1)
    cf = c.copy()
    cf[17, 33] = bad
    A, B, C = _dev(a_bits, b_bits, cf, "bf16")
    v = fk.Verifier(128, 64, 96, "bf16", m=16)
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    v.probe(A, B, C, d_dirty=flag)
    st = v.probe_stats()
    assert st["dirty"] == 1.0 and int(flag.item()) == 1
    assert o.probe(a64, b64, cf, o.make_round(v.params.seed, 0, 128, 96, 16), P).dirty
    v.close()


def test_probe_rejects_narrowed_product(fk):
    import torch
    a_bits, b_bits, _, _, c = int_case(64, 32, 64, "bf16", 2)
    A, B, C = _dev(a_bits, b_bits, c, "bf16")
    v = fk.Verifier(64, 32, 64, "bf16", m=8)
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    Cn = C.to(torch.bfloat16)
    assert v.probe_status(A, B, Cn, d_dirty=flag) == fk.EDTYPE
    assert v.probe_status(A, B, C, d_dirty=flag, c_dtype=fk.F16) == fk.EDTYPE
    torch.cuda.synchronize()
    assert int(flag.item()) == 0
    v.close()


def test_clean_probes_accumulate_sigma_and_calibrate(fk):
    n1, n2, n3 = 1024, 512, 1024
    fmt = "bf16"
    v = fk.Verifier(n1, n2, n3, fmt, m=200)
    sig = []
    _, b_bits = wl.gen_operands(n1, n2, n3, fmt, ("normal", 1.0), ("normal", 1.0), 100)
    B = to_dev_half(b_bits, fmt)
    for call in range(4):
        a_bits, _ = wl.gen_operands(n1, n2, n3, fmt, ("normal", 1.0), ("normal", 1.0), 200 + call)
        A = to_dev_half(a_bits, fmt)
        C = gemm_f32(A, B)
        v.probe(A, B, C)
        st = v.probe_stats()
        assert st["dirty"] == 0.0
        sig.append(st["sigma_hat"])
    c_last = C.cpu().numpy()
    m_new, sbar, rebuilt = v.calibrate_noise(C)
    assert abs(sbar - np.mean(sig)) <= 1e-12 * sbar
    ref_m, ref_rb = o.recalibrate_m(n1, n3, 200, sbar, o.rms_hat(c_last), P)
    assert (m_new, rebuilt) == (ref_m, ref_rb)
    assert v.m == m_new
    v.close()


# --- recheck ---------------------------------------------------------------------------------

def test_recheck_matches_fp64_dot(fk):
    n1, n2, n3 = 300, 1000, 260
    for fmt in ("bf16", "fp16"):
        a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, ("normal", 1.0), ("normal", 1.0), 12)
        A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
        a64, b64 = o.decode(a_bits, fmt), o.decode(b_bits, fmt)
        v = fk.Verifier(n1, n2, n3, fmt, m=16)
        coords = [(0, 0), (n1 - 1, n3 - 1), (150, 7), (3, 259)] + \
                 [(int(i), int(j)) for i, j in wl.fault_sites(n1, n3, 100, 13)]
        g, ab = v.recheck(A, B, coords)
        for k, (i, j) in enumerate(coords):
            ref = o.recompute(a64, b64, i, j)
            refab = float(np.abs(a64[i]) @ np.abs(b64[:, j]))
            assert abs(g[k] - ref) <= 1e-12 * refab
            assert abs(ab[k] - refab) <= 1e-12 * refab
        with pytest.raises(fk.FpsketchError):
            v.recheck(A, B, [(n1, 0)])
        v.close()


# --- localize --------------------------------------------------------------------------------

def _oracle_localize_like_gpu(v, a64, b64, cf, fmt, seed, plan):
    return o.localize(a64, b64, cf, fmt, v.m, seed, P,
                      plan=o.Plan(plan["m_loc"], plan["r"], plan["B"], bool(plan["fallback"])))


def test_localize_exact_matches_oracle(fk):
    """Integer inputs: identical records, in the same order, as the oracle's Algorithm 1/2."""
    n1, n2, n3, fmt = 512, 64, 384, "fp16"
    a_bits, b_bits, a64, b64, c = int_case(n1, n2, n3, fmt, 21)
    cf = c.copy()
    sites = wl.fault_sites(n1, n3, 12, 22)
    for k, (i, j) in enumerate(sites):
        cf[i, j] += np.float32((k % 5 + 1) * (-1) ** k)
    cf[5, 6] = np.nan
    cf[300, 2] = np.inf
    cf[301, 100] = -4e37
    A, B, C = _dev(a_bits, b_bits, cf, fmt)
    v = fk.Verifier(n1, n2, n3, fmt, m=32)
    recs, n, st = v.localize(A, B, C, seed=77, sigma_from_probe=False)
    assert st == fk.OK
    plan = v.plan()
    # same plan from the oracle's own noise measurement
    ref = o.localize(a64, b64, cf, fmt, 32, 77, P)
    assert (ref.plan.m_loc, ref.plan.r) == (plan["m_loc"], plan["r"])
    got = [(i, j, d, a, r) for i, j, d, a, r in recs]
    exp = [(f.i, f.j, f.delta, f.absolute, f.round) for f in ref.faults]
    assert got == exp
    truth = {tuple(s) for s in sites.tolist()} | {(5, 6), (300, 2), (301, 100)}
    assert {(g[0], g[1]) for g in got} == truth
    v.close()


def test_localize_large_mloc_matches_oracle(fk):
    """m_loc above 240: the localize rounds form S on the 64 x 64 matrix-core tiles and R, T
    only at the selected buckets (with the peel of earlier rounds' faults); the records equal
    the oracle's, whose rounds form the three full sketches."""
    n1, n2, n3, fmt = 2048, 1024, 2048, "bf16"
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, ("normal", 1.0), ("normal", 0.02), 41)
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    c = gemm_f32(A, B).cpu().numpy()
    a64, b64 = o.decode(a_bits, fmt), o.decode(b_bits, fmt)
    sites = wl.fault_sites(n1, n3, 10, 42)
    cf = wl.inject_additive(c, sites, wl.fault_magnitudes(10, 0.05, 4.0, wl.mean_abs(c), 43))
    C = to_dev_f32(cf)
    v = fk.Verifier(n1, n2, n3, fmt, rho_min=0.0015)
    v.probe(A, B, C)
    assert v.probe_stats()["dirty"] == 1.0
    recs, n, st = v.localize(A, B, C, seed=6, sigma_from_probe=True)
    plan = v.plan()
    assert plan["m_loc"] > 240
    pl = o.Params(rho_min=0.0015)
    ref = o.localize(a64, b64, cf, fmt, v.m, 6, pl,
                     plan=o.Plan(plan["m_loc"], plan["r"], plan["B"], bool(plan["fallback"])))
    got = {(i, j): d for i, j, d, a, r in recs}
    exp = {(f.i, f.j): f.delta for f in ref.faults}
    assert set(got) == set(exp) == {tuple(x) for x in sites.tolist()}
    for k in got:
        assert abs(got[k] - exp[k]) <= 1e-3 * abs(exp[k])
    v.close()


def test_localize_float_matches_oracle(fk):
    import torch
    n1, n2, n3, fmt = 768, 512, 640, "bf16"
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, ("normal", 1.0), ("normal", 0.02), 31)
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    c = gemm_f32(A, B).cpu().numpy()
    a64, b64 = o.decode(a_bits, fmt), o.decode(b_bits, fmt)
    sites = wl.fault_sites(n1, n3, 6, 32)
    deltas = wl.fault_magnitudes(6, 0.05, 4.0, wl.mean_abs(c), 33)
    cf = wl.inject_additive(c, sites, deltas)
    cf[100, 200] = np.float32(wl.flip_bit_value(float(cf[100, 200]), 30))
    C = to_dev_f32(cf)
    v = fk.Verifier(n1, n2, n3, fmt)
    v.probe(A, B, C)
    assert v.probe_stats()["dirty"] == 1.0
    recs, n, st = v.localize(A, B, C, seed=5, sigma_from_probe=True)
    plan = v.plan()
    ref = _oracle_localize_like_gpu(v, a64, b64, cf, fmt, 5, plan)
    got = {(i, j): d for i, j, d, a, r in recs}
    exp = {(f.i, f.j): f.delta for f in ref.faults}
    assert set(got) == set(exp)
    truth = {tuple(s) for s in sites.tolist()} | {(100, 200)}
    assert set(got) == truth
    for k in got:
        assert abs(got[k] - exp[k]) <= 1e-3 * abs(exp[k])
    v.close()
