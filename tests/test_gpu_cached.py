"""The probe with a cached B side (fpsketch_cache_b, fpsketch_probe_cached): the same statistics
and verdict, bit for bit, as the streamed probe on the B the cache was formed from, on the block
path (m <= 64), the tile path (m > 64) and element-load shapes; rotating activations against one
cached weight; and the cache dropped by a rebuild."""
import numpy as np
import pytest

from oracle import fpsketch_oracle as o
from paper_2609_19758_amd import workloads as wl
from gpu_util import gemm_f32, int_case, to_dev_f32, to_dev_half

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fk():
    import torch
    assert torch.cuda.is_available()
    from paper_2609_19758_amd import fpsketch
    fpsketch.load()
    return fpsketch


@pytest.mark.parametrize("n1,n2,n3,m,fmt", [
    (512, 256, 384, 48, "bf16"),      # block path
    (640, 320, 512, 96, "fp16"),      # tile path
    (130, 37, 131, 7, "bf16"),        # element loads (rows not multiples of 8)
    (600, 64, 8192, 64, "bf16"),      # B chunks in rotated order (two whole chunks)
])
def test_cached_probe_equals_streamed_probe(fk, n1, n2, n3, m, fmt):
    import torch
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, ("normal", 1.0), ("normal", 0.02), 81)
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    C = gemm_f32(A, B)
    Cf = C.clone()
    Cf[n1 // 2, n3 // 3] += 1.0
    v = fk.Verifier(n1, n2, n3, fmt, m=m)
    v.cache_b(B)
    for X in (C, Cf):
        f1 = torch.zeros(1, dtype=torch.int32, device="cuda")
        f2 = torch.zeros(1, dtype=torch.int32, device="cuda")
        v.probe(A, B, X, d_dirty=f1)
        s1 = v.probe_stats()
        v.probe_cached(A, X, d_dirty=f2)
        s2 = v.probe_stats()
        assert s1 == s2
        assert int(f1.item()) == int(f2.item())
    assert int(f2.item()) == 1            # the faulted product
    v.close()


@pytest.mark.parametrize("n1,n2,n3,m,fmt", [
    (512, 1000, 640, 40, "fp16"),     # two A tiles, the second ragged
    (300, 1537, 200, 64, "bf16"),     # four A tiles, one column in the last; largest block m
])
def test_cached_block_probe_matches_oracle(fk, n1, n2, n3, m, fmt):
    """The cached probe on the block path (m <= 64) across several 512-column A tiles, the last
    ragged, against the oracle's probe: verdicts, tau and max|A|, max|B| exact, max|S|
    within the FP32-storage bound of the factors, sigma-hat within the 5 % the streamed probe's
    parity test allows (both measure noise that the FP32 factors add to)."""
    import torch
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, ("normal", 1.0), ("normal", 0.02), 83)
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    c = gemm_f32(A, B).cpu().numpy()
    a64, b64 = o.decode(a_bits, fmt), o.decode(b_bits, fmt)
    v = fk.Verifier(n1, n2, n3, fmt, m=m)
    v.cache_b(B)
    hr = o.make_round(v.params.seed, 0, n1, n3, m)
    P = o.Params()
    sites = wl.fault_sites(n1, n3, 3, 84)
    dirty_c = wl.inject_additive(c, sites, wl.fault_magnitudes(3, 0.5, 2.0, wl.mean_abs(c), 85))
    for cc, expect_dirty in ((c, False), (dirty_c, True)):
        flag = torch.zeros(1, dtype=torch.int32, device="cuda")
        v.probe_cached(A, to_dev_f32(cc), d_dirty=flag)
        st = v.probe_stats()
        ref = o.probe(a64, b64, cc, hr, P)
        assert bool(st["dirty"]) == ref.dirty == expect_dirty
        assert int(flag.item()) == int(expect_dirty)
        assert abs(st["tau"] / ref.tau - 1) < 1e-12
        assert st["max_a"] == float(np.abs(a64).max()) and st["max_b"] == float(np.abs(b64).max())
        DS, _, _ = o.abs_contributions(a64, b64, cc.astype(np.float64), hr)
        assert abs(st["max_abs"] - ref.max_abs) <= 2.0 ** -20 * DS.max()
        assert abs(st["sigma_hat"] / ref.sigma_hat - 1) < 0.05
    v.close()


def test_cached_weight_with_rotating_activations(fk):
    """One cached weight, several activation matrices: every verdict and statistic equals the
    streamed probe's, clean and dirty."""
    import torch
    w = wl.workload("xfmr_4096x4096_bf16")
    b_bits = wl.gen_side(w.n2, w.n3, w.fmt, w.dist_b, 91, 0xB)
    B = to_dev_half(b_bits, w.fmt)
    v = fk.Verifier(w.n1, w.n2, w.n3, w.fmt)
    v.cache_b(B)
    for s in range(3):
        A = to_dev_half(wl.gen_side(w.n1, w.n2, w.fmt, w.dist_a, 92 + s, 0xA), w.fmt)
        C = gemm_f32(A, B)
        if s == 2:
            C[100, 200] += 0.5 * float(C.abs().mean().item())
        v.probe(A, B, C)
        s1 = v.probe_stats()
        v.probe_cached(A, C)
        assert v.probe_stats() == s1
        assert s1["dirty"] == (1.0 if s == 2 else 0.0)
    v.close()


def test_rebuild_drops_the_cache(fk):
    """A calibration rebuild (m = 16 forced, below m_comb = 48, so m' >= 48 after clean probes
    of a float product) drops the cached B side until it is formed again at the new m."""
    n1, n2, n3, fmt = 512, 256, 384, "fp16"
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, ("uniform", -1, 1), ("uniform", -1, 1), 96)
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    C = gemm_f32(A, B)
    v = fk.Verifier(n1, n2, n3, fmt, m=16)
    assert v.probe_cached_status(A, C) == fk.EINVAL        # nothing cached yet
    v.cache_b(B)
    for _ in range(3):
        v.probe_cached(A, C)
    assert v.probe_stats()["dirty"] == 0.0
    m1, sb, rebuilt = v.calibrate_noise(C)
    assert rebuilt and v.m == m1 >= 48
    assert v.probe_cached_status(A, C) == fk.EINVAL
    v.cache_b(B)
    v.probe(A, B, C)
    s1 = v.probe_stats()
    v.probe_cached(A, C)
    assert v.probe_stats() == s1 and s1["dirty"] == 0.0
    v.close()
