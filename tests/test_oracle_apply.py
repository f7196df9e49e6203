"""Pins of the oracle's apply step (Algorithm 2, last part): records written into C, then a
re-probe with a fresh hash round.  Exact special cases on integer products (C = AB exactly), the
absolute-entry case, a missing record, and the FP32 rounding of the repaired value."""
import numpy as np

from oracle import fpsketch_oracle as o
from paper_2609_19758_amd import workloads as wl

P = o.Params()


def _int_case(n1, n2, n3, seed, lo=-4, hi=4):
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, "bf16", ("int", lo, hi), ("int", lo, hi), seed)
    a64, b64 = o.decode_bf16(a_bits), o.decode_bf16(b_bits)
    c = (a64 @ b64).astype(np.float32)
    return a64, b64, c


def test_apply_restores_exact_product_and_reprobe_is_clean():
    """Integer faults localized exactly; applying the records gives back AB bit for bit, and the
    fresh-round probe of the repaired C sees S = 0 (clean)."""
    a64, b64, c = _int_case(128, 48, 96, 3)
    cf = c.copy()
    sites = [(5, 7, 3.0), (70, 40, -6.0), (127, 95, 2.0)]
    for i, j, d in sites:
        cf[i, j] += d
    res = o.localize(a64, b64, cf, "bf16", 16, seed=21, p=P, plan=o.Plan(32, 0, 0.0, False))
    assert {(f.i, f.j) for f in res.faults} == {(i, j) for i, j, _ in sites}
    c2, pr = o.apply_and_reprobe(a64, b64, cf, res.faults, seed=777, m=16, p=P)
    assert np.array_equal(c2, c)
    assert not pr.dirty and pr.max_abs == 0.0
    assert all(cf[i, j] == np.float32(c[i, j] + d) for i, j, d in sites)      # input untouched


def test_missing_record_leaves_the_reprobe_dirty():
    """With one of two records dropped the repaired C still differs from AB by that fault, whose
    bucket is the only nonzero one of the fresh round: the re-probe fires (the caller then
    recomputes)."""
    a64, b64, c = _int_case(96, 40, 80, 4)
    cf = c.copy()
    cf[10, 20] += 5.0
    cf[50, 60] -= 7.0
    F = [o.Fault(10, 20, -5.0, False, 1)]
    c2, pr = o.apply_and_reprobe(a64, b64, cf, F, seed=99, m=16, p=P)
    assert c2[10, 20] == c[10, 20] and c2[50, 60] == c[50, 60] - 7.0
    assert pr.dirty
    assert np.count_nonzero(pr.S) == 1 and pr.max_abs == 7.0


def test_absolute_record_writes_the_recomputed_value():
    """A non-finite entry comes back from the exact scan as an absolute record whose value is
    the recomputed product; applying it restores AB there."""
    a64, b64, c = _int_case(64, 32, 64, 5)
    cf = c.copy()
    cf[3, 9] = np.nan
    res = o.localize(a64, b64, cf, "bf16", 16, seed=8, p=P, plan=o.Plan(16, 0, 0.0, False))
    assert [(f.i, f.j, f.absolute) for f in res.faults] == [(3, 9, True)]
    c2, pr = o.apply_and_reprobe(a64, b64, cf, res.faults, seed=5, m=16, p=P)
    assert np.array_equal(c2, c) and not pr.dirty


def test_repaired_value_is_the_fp32_rounding_of_c_plus_delta():
    """C_ij + delta is formed in FP64 and rounded once to FP32: with delta = gamma - C_ij (FP64)
    the repaired entry is the float nearest to gamma."""
    rng = np.random.Generator(np.random.PCG64(6))
    c = rng.standard_normal((4, 4)).astype(np.float32)
    gamma = rng.standard_normal(16) * 10.0
    F = [o.Fault(k // 4, k % 4, float(gamma[k] - np.float64(c[k // 4, k % 4])), False, 1)
         for k in range(16)]
    c2 = o.apply_records(c, F)
    assert np.array_equal(c2.ravel(), gamma.astype(np.float32))
