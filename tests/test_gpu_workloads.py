"""Full-size parity at the paper's other workload shapes (Table II, Fig. 3, Sec. VI):

* the MLP down projection 4096 x 11008 x 4096 BF16 with 16 single-bit flips of C entries;
* the sixteen transformer projection cells (2048 tokens, eight (k, n) shapes, BF16 and FP16)
  with 4 additive faults of 5-400 % of mean|C|;
* the 16384^3 FP16 square product (uniform operands) with 0-32 log-uniform faults per call.

Each case runs clean probes (verdict, operand maxima), the run-time calibration (the library's
m' against the oracle's rule on the same measured noise), sampled buckets of S, R and T at the
calibrated m against their definition, and localization of seeded dirty calls against the
definition of a recoverable fault: every fault above the noise floor (or non-finite / huge) is
found, nothing else is reported, and each magnitude is within 1e-3 of the FP64 error."""
import numpy as np
import pytest

from oracle import fpsketch_oracle as o
from paper_2609_19758_amd import workloads as wl
from gpu_util import (bucket_reference, gemm_f32, rms_hat_device, site_truth, to_dev_half)

pytestmark = pytest.mark.gpu

CELLS = [f"xfmr_{k}x{n}_{fmt}" for (k, n) in wl.TRANSFORMER_KN for fmt in ("bf16", "fp16")]


def _oracle_params(w) -> o.Params:
    return o.Params(rho_min=w.rho_min, s_budget=w.s_budget)


def _max_abs(bits: np.ndarray, fmt: str) -> float:
    """max |x| over half bit patterns without widening the whole matrix: for finite values the
    magnitude grows with the pattern's low 15 bits in both formats."""
    top = np.max(np.bitwise_and(bits, np.uint16(0x7FFF)))
    return float(o.decode(np.array([top], dtype=np.uint16), fmt)[0])


def _run(name: str, n_act: int, calib_calls: int, dirty_calls: int, n_buckets: int):
    import torch
    from paper_2609_19758_amd import fpsketch as fk
    w = wl.workload(name)
    n1, n2, n3, fmt = w.n1, w.n2, w.n3, w.fmt
    P = _oracle_params(w)
    print(f"\n[{name}] {n1}x{n2}x{n3} {fmt}: generating operands", flush=True)
    acts = [wl.gen_side(n1, n2, fmt, w.dist_a, 500 + s, 0xA) for s in range(n_act)]
    b_bits = wl.gen_side(n2, n3, fmt, w.dist_b, 600, 0xB)
    B = to_dev_half(b_bits, fmt)
    As = [to_dev_half(a, fmt) for a in acts]
    Cs = [gemm_f32(A, B) for A in As]
    torch.cuda.synchronize()

    v = fk.Verifier(n1, n2, n3, fmt, m=w.m_forced, rho_min=w.rho_min, s_budget=w.s_budget)
    m0 = v.m
    assert m0 == (w.m_forced or o.m_start(n1, n2, n3, fmt, P))
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")

    # clean probes on distinct activations, then the run-time calibration
    maxb = _max_abs(b_bits, fmt)
    for k in range(calib_calls):
        t = k % n_act
        v.probe(As[t], B, Cs[t], d_dirty=flag)
        st = v.probe_stats()
        assert st["dirty"] == 0.0 and st["finite"] == 1.0, (k, st)
        if k < n_act:
            assert st["max_a"] == _max_abs(acts[t], fmt)
            assert st["max_b"] == maxb
    assert int(flag.item()) == 0
    m_cal, sigma_bar, rebuilt = v.calibrate_noise(Cs[0])
    rms0 = rms_hat_device(Cs[0])
    m_ref, rb_ref = o.recalibrate_m(n1, n3, m0, sigma_bar, rms0, P)
    print(f"[{name}] m {m0} -> {m_cal} (sigma_bar {sigma_bar:.4g}, rms {rms0:.4g})", flush=True)
    assert (m_cal, rebuilt) == (m_ref, rb_ref)
    assert v.m == m_cal
    for t in range(n_act):                      # still clean at the calibrated m
        v.probe(As[t], B, Cs[t], d_dirty=flag)
    assert int(flag.item()) == 0

    # sampled buckets of S, R, T at the calibrated m against the definition
    m = v.m
    seed = 4321
    S, R, T, mxa, mxb = v.sketch(As[0], B, Cs[0], seed, 0, m)
    hr = o.make_round(seed, 0, n1, n3, m)
    rng = np.random.Generator(np.random.PCG64(7))
    picks = [(0, 0), (m - 1, m - 1)] + [tuple(int(x) for x in p)
                                        for p in rng.integers(0, m, size=(n_buckets - 2, 2))]
    for a, b in picks:
        (rs, rr, rt), D = bucket_reference(acts[0], b_bits, fmt, Cs[0], hr, a, b)
        for got, ref in ((S[a, b], rs), (R[a, b], rr), (T[a, b], rt)):
            assert abs(got - ref) <= 2.0 ** -20 * D, (name, a, b, got, ref, D)

    # dirty calls
    unit = float(Cs[0].abs().double().mean().item())
    found = must = 0
    for r in range(dirty_calls):
        t = r % n_act
        A, C = As[t], Cs[t]
        sites, deltas, masks = wl.call_faults(w, n1, n3, unit, 7000 + r)
        Cf = C.clone()
        if len(sites):
            ii = torch.from_numpy(sites[:, 0].copy()).cuda()
            jj = torch.from_numpy(sites[:, 1].copy()).cuda()
            vals = wl.apply_faults(C[ii, jj].cpu().numpy(), deltas, masks)
            Cf[ii, jj] = torch.from_numpy(vals).cuda()
        else:
            vals = np.zeros(0, dtype=np.float32)
        flag.zero_()
        v.probe(A, B, Cf, d_dirty=flag)
        recs, n, status = v.localize(A, B, Cf, seed=9000 + r, sigma_from_probe=True)
        assert status == fk.OK
        plan = v.plan()
        floor = w.rho_min * rms_hat_device(Cf)
        truth = site_truth(acts[t], b_bits, fmt, sites, vals, floor, P)
        got = {(i, j): (d, ab) for i, j, d, ab, _ in recs}
        need = {s for s, x in truth.items() if x[3]}
        print(f"[{name}] call {r}: {len(sites)} faults, {len(need)} above floor, "
              f"{len(got)} found (m_loc {plan['m_loc']}, r {plan['r']})", flush=True)
        if need:
            assert int(flag.item()) == 1
        assert need <= set(got), sorted(need - set(got))
        assert set(got) <= set(truth), sorted(set(got) - set(truth))    # zero false positives
        for s, (d, ab) in got.items():
            e, tau, absolute, _ = truth[s]
            assert ab == absolute
            assert abs(d - e) <= 1e-3 * abs(e), (s, d, e)
            if not absolute:
                assert abs(e) > tau
        found += len(need & set(got))
        must += len(need)
    v.close()
    return found, must


def test_mlp_down_bf16_bitflips():
    found, must = _run("mlp_down_bf16", n_act=2, calib_calls=16, dirty_calls=3, n_buckets=6)
    assert found == must


@pytest.mark.parametrize("name", CELLS)
def test_transformer_cell(name):
    found, must = _run(name, n_act=2, calib_calls=16, dirty_calls=2, n_buckets=4)
    assert found == must and must > 0


def test_square16384_fp16_mixed():
    found, must = _run("square16384_fp16", n_act=2, calib_calls=8, dirty_calls=3, n_buckets=4)
    assert found == must
