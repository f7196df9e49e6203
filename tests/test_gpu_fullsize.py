"""Full-size parity at the square 4096^3 BF16 workload (N(0,1) operands, FP32 product from the
black-box GEMM, 8 faults of 2-9 % of mean|C|): sketch values on sampled buckets computed one by
one by the oracle, the probe verdicts, and localization checked entry by entry."""
import numpy as np
import pytest

from oracle import fpsketch_oracle as o
from paper_2609_19758_amd import workloads as wl
from gpu_util import gemm_f32, to_dev_f32, to_dev_half

pytestmark = pytest.mark.gpu

P = o.Params()


def _bucket_values(a64, b64, c, hr, a, b):
    """S, R, T and their absolute-contribution scales of one bucket, from the definition."""
    n1, n3 = c.shape
    rows = np.flatnonzero(hr.h1 == a)
    cols = np.flatnonzero(hr.h2 == b)
    E = a64[rows] @ b64[:, cols] - c[np.ix_(rows, cols)].astype(np.float64)
    v1, v2 = hr.v1[rows], hr.v2[cols]
    w1 = (rows + 1) / o.pow2_ceil(n1)
    w2 = (cols + 1) / o.pow2_ceil(n3)
    S = v1 @ E @ v2
    R = (v1 * w1) @ E @ v2
    T = v1 @ E @ (v2 * w2)
    pa = np.abs(a64[rows]).sum(axis=0)
    pb = np.abs(b64[:, cols]).sum(axis=1)
    cc = np.abs(c[np.ix_(rows, cols)].astype(np.float64))
    DS = pa @ pb + cc.sum()
    return (S, R, T), DS


def test_square4096_bf16(tmp_path):
    import torch
    from paper_2609_19758_amd import fpsketch as fk
    w = wl.workload("square4096_bf16")
    n1, n2, n3, fmt = w.n1, w.n2, w.n3, w.fmt
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, w.dist_a, w.dist_b, 1)
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    C = gemm_f32(A, B)
    torch.cuda.synchronize()
    c = C.cpu().numpy()
    a64, b64 = o.decode(a_bits, fmt), o.decode(b_bits, fmt)
    v = fk.Verifier(n1, n2, n3, fmt, rho_min=w.rho_min)
    m = v.m
    assert m == o.m_start(n1, n2, n3, fmt, P) == 48

    # clean probe
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    v.probe(A, B, C, d_dirty=flag)
    st = v.probe_stats()
    assert st["dirty"] == 0.0 and int(flag.item()) == 0
    assert st["max_a"] == np.max(np.abs(a64)) and st["max_b"] == np.max(np.abs(b64))

    # sampled buckets of S, R, T against the definition
    seed = 1234
    S, R, T, _, _ = v.sketch(A, B, C, seed, 0, m)
    hr = o.make_round(seed, 0, n1, n3, m)
    rng = np.random.Generator(np.random.PCG64(0))
    for a, b in [(0, 0), (m - 1, m - 1)] + [tuple(x) for x in rng.integers(0, m, size=(6, 2))]:
        (rs, rr, rt), D = _bucket_values(a64, b64, c, hr, int(a), int(b))
        for got, ref in ((S[a, b], rs), (R[a, b], rr), (T[a, b], rt)):
            assert abs(got - ref) <= 2.0 ** -20 * D, (a, b, got, ref, D)

    # faults of 2-9 % of mean|C|
    sites = wl.fault_sites(n1, n3, w.faults, 2)
    deltas = wl.fault_magnitudes(w.faults, w.fault_lo, w.fault_hi, wl.mean_abs(c), 3)
    cf = wl.inject_additive(c, sites, deltas)
    Cf = to_dev_f32(cf)
    flag.zero_()
    v.probe(A, B, Cf, d_dirty=flag)
    assert int(flag.item()) == 1
    recs, n, status = v.localize(A, B, Cf, seed=99, sigma_from_probe=True)
    assert status == fk.OK
    got = {(i, j): d for i, j, d, ab, r in recs}
    injected = {tuple(s) for s in sites.tolist()}
    assert set(got) == injected            # recovery 1.000, zero false positives
    for (i, j), d in got.items():
        ref = o.recompute(a64, b64, i, j) - float(cf[i, j])       # E_ij in FP64
        assert abs(d - ref) <= 1e-3 * abs(ref)
        assert abs(ref) > o.validation_bound(a64, b64, i, j, P)
    v.close()


def _noise_ratio_case(name: str, seed_ops: int, with_faults: bool):
    """The verifier's own rounding against the GEMM noise it measures: on a clean product the
    full-grid statistic std(S_gpu - S_oracle) / sigma_hat_oracle (S_oracle is the definition on
    the explicit FP64 error, sigma_hat_oracle its clipped-mean noise estimate), and on a dirty
    product every fault bucket within 1e-3 relative of the oracle's.  S_gpu comes from
    fpsketch_sketch, whose stream pass (where the verifier rounds: FP32 factors) is the probe's;
    its bucket-space product is FP64 like the probe's."""
    import torch
    from paper_2609_19758_amd import fpsketch as fk
    w = wl.workload(name)
    n1, n2, n3, fmt = w.n1, w.n2, w.n3, w.fmt
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, w.dist_a, w.dist_b, seed_ops)
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    C = gemm_f32(A, B)
    torch.cuda.synchronize()
    c = C.cpu().numpy()
    a64, b64 = o.decode(a_bits, fmt), o.decode(b_bits, fmt)
    v = fk.Verifier(n1, n2, n3, fmt, rho_min=w.rho_min)
    m, seed = v.m, 777
    hr = o.make_round(seed, 0, n1, n3, m)
    E = o.error_matrix(a64, b64, c)
    S_ref, _, _ = o.sketches(E, hr, moments=False)
    S_gpu, _, _, _, _ = v.sketch(A, B, C, seed, 0, m, moments=False)
    sigma = o.clipped_sigma(S_ref)
    ratio = float(np.std(S_gpu - S_ref) / sigma)
    print(f"\n[{name}] m {m}: sigma_hat oracle {sigma:.4g}, std(S_gpu - S_oracle) / sigma_hat "
          f"= {ratio:.4f}, max |S_gpu - S_oracle| / sigma_hat "
          f"= {float(np.max(np.abs(S_gpu - S_ref)) / sigma):.4f}", flush=True)
    res = {"ratio": ratio}
    if with_faults:
        sites = wl.fault_sites(n1, n3, w.faults, 2)
        deltas = wl.fault_magnitudes(w.faults, w.fault_lo, w.fault_hi, wl.mean_abs(c), 3)
        cf = wl.inject_additive(c, sites, deltas)
        Ef = E - (cf.astype(np.float64) - c.astype(np.float64))
        Sf_ref, _, _ = o.sketches(Ef, hr, moments=False)
        Sf_gpu, _, _, _, _ = v.sketch(A, B, to_dev_f32(cf), seed, 0, m, moments=False)
        worst = 0.0
        for i, j in sites.tolist():
            a, b = int(hr.h1[i]), int(hr.h2[j])
            worst = max(worst, abs(Sf_gpu[a, b] - Sf_ref[a, b]) / abs(Sf_ref[a, b]))
        print(f"[{name}] fault buckets: worst relative error {worst:.3g}", flush=True)
        res["fault_rel"] = worst
    v.close()
    return res


# The verifier rounds where it stores the factors P = H1 A and Q = B H2^T in FP32.  A bucket sum
# of at most about 110 half values mostly fits FP32's 24 bits exactly, so the measured ratio is
# small: 0.012 at 4096^3 BF16 and 0.009 at 2048 x 4096 x 4096 BF16 on MI355X.  The bound keeps a
# fourfold margin over that and fails once the verifier's own rounding reaches 5 % of the GEMM
# noise it measures (rounding at FP32 of every factor entry would give about 0.08).
NOISE_RATIO_BOUND = 0.05


def test_sketch_rounding_against_gemm_noise_square4096_bf16():
    res = _noise_ratio_case("square4096_bf16", 1, with_faults=True)
    assert res["ratio"] <= NOISE_RATIO_BOUND
    assert res["fault_rel"] <= 1e-3


def test_sketch_rounding_against_gemm_noise_transformer_cell():
    res = _noise_ratio_case("xfmr_4096x4096_bf16", 5, with_faults=False)
    assert res["ratio"] <= NOISE_RATIO_BOUND
