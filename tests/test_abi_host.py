"""CPU checks of the C ABI: the library loads and exports every symbol the header declares,
and its host logic (hash rounds, bucket-count rules, plan, recalibration, rms-hat) agrees with
the oracle.  No device work runs here."""
import ctypes
import math

import numpy as np
import pytest

from oracle import fpsketch_oracle as o
from paper_2609_19758_amd import fpsketch as fk
from conftest import load_golden

P = o.Params()


def test_library_exports_every_header_symbol():
    lib = fk.load()
    names = fk.header_symbols()
    assert len(names) >= 18
    for name in names:
        assert hasattr(lib, name), name
    # and the binding declares a signature for each of them
    assert set(names) == set(fk._SIGS)


def test_status_strings_and_defaults():
    lib = fk.load()
    for s in range(8):
        assert lib.fpsketch_status_str(s).decode()
    p = fk.default_params()
    assert (p.rounds, p.r_star, p.r_max, p.s_budget, p.delta_rc, p.k_cap) == (3, 4, 16, 16, 8, 0)
    assert (p.rho_min, p.mu, p.c_valid, p.b_star, p.c_coll) == (0.02, 4.0, 100.0, 0.3, 2.0)


@pytest.mark.parametrize("seed", range(10))
def test_hash_tables_match_oracle(seed):
    for rnd, side, n, m in [(0, 0, 4096, 48), (1, 1, 11008, 528), (3, 0, 1000, 1), (2, 1, 777, 4096)]:
        b, s = fk.hash_table(seed, rnd, side, n, m)
        ob, os_ = o.hash_round(seed, rnd, side, n, m)
        assert np.array_equal(b, ob)
        assert np.array_equal(s.astype(np.float64), os_)


def test_hash_large_seed():
    seed = 0xFFFFFFFFFFFFFFF1
    b, s = fk.hash_table(seed, 5, 1, 300, 77)
    ob, os_ = o.hash_round(seed, 5, 1, 300, 77)
    assert np.array_equal(b, ob) and np.array_equal(s.astype(np.float64), os_)


def test_m_start_matches_oracle_and_table2():
    for row in load_golden("table2_bucket_counts.csv"):
        n1, n2, n3 = int(row["n1"]), int(row["n2"]), int(row["n3"])
        assert fk.m_start(n1, n2, n3, "bf16") == int(row["m_bf16"])
        assert fk.m_start(n1, n2, n3, "fp16") == int(row["m_fp16"])
    rng = np.random.Generator(np.random.PCG64(1))
    for _ in range(200):
        n1, n2, n3 = (int(x) for x in rng.integers(1, 70000, size=3))
        for fmt in ("bf16", "fp16"):
            assert fk.m_start(n1, n2, n3, fmt) == o.m_start(n1, n2, n3, fmt, P)


def test_law_constants_are_parameters():
    """Eq. 3's constants taken from the parameters (as measured for another BLAS): the library's
    start m and fallback plan equal the oracle's under the same constants, and out-of-range
    constants are rejected."""
    rng = np.random.Generator(np.random.PCG64(11))
    for cf_b, cf_f, e in ((0.05, 0.08, 0.0), (0.31, 0.5, 0.2), (0.11, 0.11, -0.05)):
        po = o.Params(law_cf_bf16=cf_b, law_cf_fp16=cf_f, law_n2_exp=e)
        pl = fk.default_params(law_cf_bf16=cf_b, law_cf_fp16=cf_f, law_n2_exp=e)
        for _ in range(100):
            n1, n2, n3 = (int(x) for x in rng.integers(1, 70000, size=3))
            for fmt in ("bf16", "fp16"):
                assert fk.m_start(n1, n2, n3, fmt, pl) == o.m_start(n1, n2, n3, fmt, po)
        for fmt in ("bf16", "fp16"):
            ref = o.plan_localize(4096, 11008, 4096, fmt, 48, float("nan"), 2.0, po)
            got = fk.plan_host(4096, 11008, 4096, fmt, 48, float("nan"), 2.0, pl)
            assert got[:2] == (ref.m_loc, ref.r) and got[3] and ref.fallback
            assert abs(got[2] - ref.B) <= 1e-12 * abs(ref.B)
    # a smaller c_f lowers the start m; the paper's constants are the defaults
    assert fk.m_start(2048, 4096, 12288, "bf16", fk.default_params(law_cf_bf16=0.1)) < \
        fk.m_start(2048, 4096, 12288, "bf16")
    d = fk.default_params()
    assert (d.law_cf_bf16, d.law_cf_fp16, d.law_n2_exp) == (P.law_cf_bf16, P.law_cf_fp16,
                                                            P.law_n2_exp)
    out = ctypes.c_int32()
    lib = fk.load()
    for bad in ({"law_cf_bf16": 0.0}, {"law_cf_fp16": -1.0}, {"law_n2_exp": float("nan")},
                {"law_cf_bf16": float("inf")}):
        p = fk.default_params(**bad)
        assert lib.fpsketch_m_start(4096, 4096, 4096, fk.BF16, ctypes.byref(p),
                                    ctypes.byref(out)) == fk.EINVAL


def test_plan_matches_oracle():
    rng = np.random.Generator(np.random.PCG64(2))
    shapes = [(4096, 4096, 4096), (4096, 11008, 4096), (2048, 13824, 5120),
              (16384, 16384, 16384), (256, 256, 256), (16384, 8192, 8192)]
    for n1, n2, n3 in shapes:
        for fmt in ("bf16", "fp16"):
            m = o.m_start(n1, n2, n3, fmt, P)
            for _ in range(40):
                sigma = float(10 ** rng.uniform(-6, 0))
                rms = float(10 ** rng.uniform(-1, 2.5))
                for rho in (0.015, 0.02, 1.0):
                    p = o.Params(rho_min=rho)
                    ref = o.plan_localize(n1, n2, n3, fmt, m, sigma, rms, p)
                    got = fk.plan_host(n1, n2, n3, fmt, m, sigma, rms,
                                       fk.default_params(rho_min=rho))
                    assert got[:2] == (ref.m_loc, ref.r), (n1, n2, n3, fmt, sigma, rms, rho)
                    assert got[3] == ref.fallback
                    assert abs(got[2] - ref.B) <= 1e-12 * abs(ref.B)
    for bad in (float("nan"), 0.0, -1.0, float("inf")):
        ref = o.plan_localize(4096, 4096, 4096, "bf16", 48, bad, 64.0, P)
        got = fk.plan_host(4096, 4096, 4096, "bf16", 48, bad, 64.0)
        assert got[:2] == (ref.m_loc, ref.r) and got[3] and ref.fallback


def test_plan_with_huge_noise_estimate_matches_oracle():
    """A probe estimate taken on a C that holds entries near fp32max is itself of that order;
    the radius rule then asks for far more than any integer radius, and the plan must saturate
    at the largest m_loc and r_max (Sec. III-G), as the oracle's unbounded integers do."""
    for sigma in (1e9, 1e20, 1e35, 1e300):
        for (n1, n2, n3) in ((4096, 11008, 4096), (16384, 16384, 16384), (2048, 4096, 4096)):
            ref = o.plan_localize(n1, n2, n3, "bf16", 48, sigma, 2.0, P)
            got = fk.plan_host(n1, n2, n3, "bf16", 48, sigma, 2.0)
            assert got[:2] == (ref.m_loc, ref.r), (sigma, n1, n2, n3, got, ref)
            assert ref.r == P.r_max and ref.m_loc == min(o.m_max(n1, n3), o.m_mem(n2))
    ref = o.recalibrate_m(4096, 4096, 48, 1e300, 2.0, P)
    assert fk.recalibrate_host(4096, 4096, 48, 1e300, 2.0) == (ref[0], ref[1])


def test_recalibration_matches_oracle():
    rng = np.random.Generator(np.random.PCG64(3))
    for _ in range(500):
        n1, n3 = (int(x) for x in rng.integers(64, 40000, size=2))
        m = int(rng.integers(16, 3000))
        sb = float(10 ** rng.uniform(-6, -1))
        rms = float(10 ** rng.uniform(-1, 2))
        ref = o.recalibrate_m(n1, n3, m, sb, rms, P)
        got = fk.recalibrate_host(n1, n3, m, sb, rms)
        assert got == (ref[0], ref[1]), (n1, n3, m, sb, rms)


def test_rms_hat_samples_match_oracle():
    rng = np.random.Generator(np.random.PCG64(4))
    c = (rng.standard_normal((700, 900)) * 5).astype(np.float32)
    c[3, 5] = np.nan
    c[100, 0] = np.inf
    c[200, 8] = 1e33
    stride = max(1, c.size // 65536)
    samples = c.ravel()[::stride]
    assert abs(fk.rms_hat_samples(samples) - o.rms_hat(c)) <= 1e-12 * o.rms_hat(c)
    assert math.isnan(fk.rms_hat_samples(np.array([np.nan, np.inf], dtype=np.float32)))


def test_invalid_arguments_rejected_on_host():
    lib = fk.load()
    assert lib.fpsketch_hash_table(1, 0, 2, 10, 4, None, None) == fk.EINVAL
    out = ctypes.c_int32()
    assert lib.fpsketch_m_start(4096, 4096, 4096, fk.F32, None, ctypes.byref(out)) == fk.EDTYPE
    assert lib.fpsketch_m_start(0, 4096, 4096, fk.BF16, None, ctypes.byref(out)) == fk.EINVAL
    h = ctypes.c_void_p()
    assert lib.fpsketch_create(64, 64, 64, fk.F32, None, ctypes.byref(h)) == fk.EDTYPE
    assert lib.fpsketch_create(0, 64, 64, fk.BF16, None, ctypes.byref(h)) == fk.ESHAPE
    bad = fk.default_params(rounds=0)
    assert lib.fpsketch_create(64, 64, 64, fk.BF16, ctypes.byref(bad), ctypes.byref(h)) == fk.EINVAL
    assert lib.fpsketch_probe(None, None, None, None, fk.F32, None, None) == fk.EINVAL
