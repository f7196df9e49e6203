"""The probe's decision statistics against their definition (Sec. III-E) on the library's own S
(fpsketch_sketch at the probe's round and m): sigma-hat = 1.2533 mean(min(|S|, 5 mean|S|)),
max|S|, thr = min(tau, mu sqrt(2 ln m^2) sigma-hat), on the block path (m <= 64), the tile path
with one deciding work-group's pass, and the tile path whose clipped sum is spread over one
work-group per tile (m >= 192), with buckets that do and do not reach the clip.  The sketch
call forms S with the matrix-core product; the block path's S differs from it only in FP64
summation order (relative 1e-9 here)."""
import math

import numpy as np
import pytest

from oracle import fpsketch_oracle as o
from paper_2609_19758_amd import workloads as wl
from gpu_util import gemm_f32, to_dev_f32, to_dev_half

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fk():
    import torch
    assert torch.cuda.is_available()
    from paper_2609_19758_amd import fpsketch
    fpsketch.load()
    return fpsketch


@pytest.mark.parametrize("n1,n2,n3,m,fmt", [
    (512, 768, 640, 48, "bf16"),      # block path
    (700, 520, 600, 100, "fp16"),     # tile path, one work-group's pass
    (1024, 512, 1024, 256, "bf16"),   # tile path, clipped sums per tile
    (1500, 300, 1300, 330, "fp16"),   # ragged tiles
])
def test_decision_statistics_match_definition(fk, n1, n2, n3, m, fmt):
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, ("normal", 1.0), ("normal", 0.02), 111)
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    c = gemm_f32(A, B).cpu().numpy()
    P = o.Params()
    v = fk.Verifier(n1, n2, n3, fmt, m=m)
    reached = set()
    for name, cc in (("clean", c), ("big", wl.inject_additive(
            c, wl.fault_sites(n1, n3, 3, 112), np.array([50.0, -40.0, 30.0])))):
        C = to_dev_f32(cc)
        v.probe(A, B, C)
        st = v.probe_stats()
        S, _, _, ma, mb = v.sketch(A, B, C, v.params.seed, 0, m, moments=False)
        a = np.abs(S.ravel())
        mean = a.mean()
        clip = 5.0 * mean
        reached.add(bool(a.max() > clip))
        sigma = 1.2533 * np.minimum(a, clip).mean()
        assert abs(st["max_abs"] - a.max()) <= 1e-9 * a.max(), name
        assert abs(st["sigma_hat"] - sigma) <= 1e-9 * sigma, (name, st["sigma_hat"], sigma)
        tau = o.tau_analytic(n2, ma, mb, P)
        assert abs(st["tau"] - tau) <= 1e-12 * tau
        thr = min(tau, P.mu * math.sqrt(2.0 * math.log(m * m)) * st["sigma_hat"])
        assert abs(st["thr"] - thr) <= 1e-12 * thr
        assert st["dirty"] == float(st["max_abs"] > st["thr"]), name
        assert abs(a.max() - st["thr"]) > 1e-6 * st["thr"]      # not a knife-edge verdict
    assert True in reached       # the faulted product's buckets reach the clip
    v.close()
