"""GPU parity of Algorithm 2's apply step (fpsketch_apply) against the oracle: the repaired C
bit for bit (each record's FP64 sum rounded once to FP32, absolute records written as their
value), the fresh-round re-probe verdict, the dirty re-probe when a record is missing, the
full-size 4096^3 BF16 workload, and the argument checks."""
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


def _oracle_faults(recs):
    return [o.Fault(int(i), int(j), float(d), bool(a), int(r)) for i, j, d, a, r in recs]


def test_apply_integer_case_matches_oracle(fk):
    """Integer product with integer faults and non-finite / huge entries: localize, apply and
    re-probe on the GPU give the oracle's repaired C (equal to AB) and its clean verdict."""
    n1, n2, n3, fmt = 512, 64, 384, "fp16"
    a_bits, b_bits, a64, b64, c = int_case(n1, n2, n3, fmt, 41)
    cf = c.copy()
    sites = wl.fault_sites(n1, n3, 10, 42)
    for k, (i, j) in enumerate(sites):
        cf[i, j] += np.float32((k % 4 + 1) * (-1) ** k)
    cf[7, 8] = np.nan
    cf[400, 3] = -np.inf
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    C = to_dev_f32(cf)
    v = fk.Verifier(n1, n2, n3, fmt, m=32)
    recs, n, st = v.localize(A, B, C, seed=77, sigma_from_probe=False)
    assert st == fk.OK and n == len(sites) + 2
    dirty = v.apply(A, B, C, recs, seed=9001)
    c_rep, pr = o.apply_and_reprobe(a64, b64, cf, _oracle_faults(recs), 9001, v.m, P)
    got = C.cpu().numpy()
    assert np.array_equal(got, c_rep)
    assert np.array_equal(got, c)                 # every fault found: AB restored exactly
    assert dirty == pr.dirty == False
    v.close()


def test_apply_missing_record_reprobe_fires(fk):
    """Dropping one record leaves that fault in C: the re-probe fires on both sides."""
    n1, n2, n3, fmt = 256, 48, 320, "bf16"
    a_bits, b_bits, a64, b64, c = int_case(n1, n2, n3, fmt, 43)
    cf = c.copy()
    cf[10, 20] += 6.0
    cf[200, 300] -= 5.0
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    C = to_dev_f32(cf)
    v = fk.Verifier(n1, n2, n3, fmt, m=16)
    recs, n, st = v.localize(A, B, C, seed=3, sigma_from_probe=False)
    assert st == fk.OK and {(r[0], r[1]) for r in recs} == {(10, 20), (200, 300)}
    keep = [r for r in recs if (r[0], r[1]) == (10, 20)]
    dirty = v.apply(A, B, C, keep, seed=55)
    c_rep, pr = o.apply_and_reprobe(a64, b64, cf, _oracle_faults(keep), 55, v.m, P)
    assert np.array_equal(C.cpu().numpy(), c_rep)
    assert dirty and pr.dirty
    v.close()


def test_apply_float_case_matches_oracle(fk):
    """Float product (hipBLASLt C) with additive faults and one exponent flip: the repaired entries
    equal the oracle's FP32 rounding of C + delta bit for bit, nothing else changes, and both
    re-probes are clean."""
    n1, n2, n3, fmt = 768, 512, 640, "bf16"
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, ("normal", 1.0), ("normal", 0.02), 51)
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    c = gemm_f32(A, B).cpu().numpy()
    a64, b64 = o.decode(a_bits, fmt), o.decode(b_bits, fmt)
    sites = wl.fault_sites(n1, n3, 6, 52)
    deltas = wl.fault_magnitudes(6, 0.05, 4.0, wl.mean_abs(c), 53)
    cf = wl.inject_additive(c, sites, deltas)
    cf[300, 400] = np.float32(wl.flip_bit_value(float(cf[300, 400]), 30))
    C = to_dev_f32(cf)
    v = fk.Verifier(n1, n2, n3, fmt)
    v.probe(A, B, C)
    recs, n, st = v.localize(A, B, C, seed=6, sigma_from_probe=True)
    assert st == fk.OK
    assert {(r[0], r[1]) for r in recs} == {tuple(s) for s in sites.tolist()} | {(300, 400)}
    dirty = v.apply(A, B, C, recs, seed=6006)
    c_rep, pr = o.apply_and_reprobe(a64, b64, cf, _oracle_faults(recs), 6006, v.m, P)
    got = C.cpu().numpy()
    assert np.array_equal(got, c_rep)
    changed = np.argwhere(got != cf)
    assert {tuple(x) for x in changed.tolist()} <= {(r[0], r[1]) for r in recs}
    assert dirty == pr.dirty == False
    # the repaired entries carry at most the rounding a clean GEMM entry carries
    for i, j, d, a, r in recs:
        tau = o.validation_bound(a64, b64, i, j, P)
        assert abs(float(got[i, j]) - o.recompute(a64, b64, i, j)) <= tau
    v.close()


def test_apply_full_size_square4096(fk):
    """4096^3 BF16 with 8 faults of 2-9 % of mean|C|: localize and apply leave a C that the
    fresh-round probe finds clean, with every repaired entry within the validation bound of the
    exact product."""
    import torch
    w = wl.workload("square4096_bf16")
    a_bits, b_bits = wl.gen_operands(w.n1, w.n2, w.n3, w.fmt, w.dist_a, w.dist_b, 7)
    A, B = to_dev_half(a_bits, w.fmt), to_dev_half(b_bits, w.fmt)
    C = gemm_f32(A, B)
    torch.cuda.synchronize()
    unit = float(C.abs().double().mean().item())
    sites, deltas, masks = wl.call_faults(w, w.n1, w.n3, unit, 71)
    ii = torch.from_numpy(sites[:, 0].copy()).cuda()
    jj = torch.from_numpy(sites[:, 1].copy()).cuda()
    Cf = C.clone()
    Cf[ii, jj] = torch.from_numpy(wl.apply_faults(C[ii, jj].cpu().numpy(), deltas, masks)).cuda()
    v = fk.Verifier(w.n1, w.n2, w.n3, w.fmt, rho_min=w.rho_min)
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    v.probe(A, B, Cf, d_dirty=flag)
    assert int(flag.item()) == 1
    recs, n, st = v.localize(A, B, Cf, seed=72, sigma_from_probe=True)
    assert st == fk.OK and {(r[0], r[1]) for r in recs} == {tuple(s) for s in sites.tolist()}
    before = Cf.clone()
    assert v.apply(A, B, Cf, recs, seed=73) is False
    diff = (Cf != before).nonzero().cpu().numpy()
    assert {tuple(x) for x in diff.tolist()} <= {tuple(s) for s in sites.tolist()}
    for i, j in sites.tolist():
        a64 = o.decode(np.ascontiguousarray(a_bits[i:i + 1]), w.fmt)
        b64 = o.decode(np.ascontiguousarray(b_bits[:, j:j + 1]), w.fmt)
        assert abs(float(Cf[i, j].item()) - o.recompute(a64, b64, 0, 0)) <= \
            o.validation_bound(a64, b64, 0, 0, P)
    # the context's own probe statistics are untouched by the re-probe
    assert v.probe_stats()["dirty"] == 1.0
    v.close()


def test_apply_argument_checks(fk):
    import torch
    n1, n2, n3, fmt = 64, 32, 48, "fp16"
    a_bits, b_bits, a64, b64, c = int_case(n1, n2, n3, fmt, 61)
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    C = to_dev_f32(c)
    v = fk.Verifier(n1, n2, n3, fmt, m=16)
    st, _ = v.apply_status(A, B, C, [(1, 2, 1.0, False, 1), (1, 2, 2.0, False, 1)], seed=1)
    assert st == fk.EINVAL                      # a coordinate listed twice
    st, _ = v.apply_status(A, B, C, [(n1, 0, 1.0, False, 1)], seed=1)
    assert st == fk.EINVAL                      # outside C
    st, _ = v.apply_status(A, B, C.to(torch.float16), [], seed=1)
    assert st == fk.EDTYPE                      # C narrowed below FP32
    assert np.array_equal(C.cpu().numpy(), c)   # nothing written on a rejected call
    assert v.apply(A, B, C, [], seed=2) is False   # no records: a clean product re-probes clean
    v.close()
