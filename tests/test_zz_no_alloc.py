"""fpsketch_probe_noalloc (the probe with the library's static per-GPU scratch) against
fpsketch_probe on the same context and inputs: the statistics bit for bit and the verdict in the
caller's flag, on two calls in a row, the second with a smaller product whose n2 is not a
multiple of 4 (the factors' padding columns, left over from the larger call in the shared
scratch, must read as zero)."""
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


def _stats_tuple(st):
    return tuple(np.float64(st[k]).tobytes() for k in sorted(st))


def _case(fk, n1, n2, n3, fmt, m, seed):
    import torch
    print(f"\n[noalloc] {n1}x{n2}x{n3} {fmt} m={m}", flush=True)
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, ("normal", 1.0), ("normal", 1.0), seed)
    A, B = to_dev_half(a_bits, fmt), to_dev_half(b_bits, fmt)
    C = gemm_f32(A, B)
    torch.cuda.synchronize()
    c = C.cpu().numpy()
    sites = wl.fault_sites(n1, n3, 3, seed + 1)
    cf = wl.inject_additive(c, sites, wl.fault_magnitudes(3, 0.5, 2.0, wl.mean_abs(c), seed + 2))
    Cf = to_dev_f32(cf)
    v = fk.Verifier(n1, n2, n3, fmt, m=m)
    hr = o.make_round(v.params.seed, 0, n1, n3, m)
    a64, b64 = o.decode(a_bits, fmt), o.decode(b_bits, fmt)
    for X, x, want in ((C, c, False), (Cf, cf, True)):
        f1 = torch.zeros(1, dtype=torch.int32, device="cuda")
        f2 = torch.zeros(1, dtype=torch.int32, device="cuda")
        v.probe(A, B, X, d_dirty=f1)
        s1 = v.probe_stats()
        v.probe_noalloc(A, B, X, d_dirty=f2)
        s2 = v.probe_stats()
        torch.cuda.synchronize()
        assert _stats_tuple(s1) == _stats_tuple(s2), (s1, s2)
        assert int(f1.item()) == int(f2.item()) == int(want)
        assert o.probe(a64, b64, x, hr, o.Params()).dirty == want
    v.close()


def test_noalloc_probe_matches_probe_on_two_calls(fk):
    _case(fk, 2048, 4096, 3072, "bf16", 48, 31)       # first call: the larger product
    _case(fk, 192, 510, 200, "fp16", 16, 32)          # second: smaller, n2 = 510, kact = 512


def test_noalloc_probe_rejects_the_tile_path(fk):
    import torch
    v = fk.Verifier(512, 256, 512, "bf16", m=96)
    A = torch.zeros(512, 256, dtype=torch.bfloat16, device="cuda")
    B = torch.zeros(256, 512, dtype=torch.bfloat16, device="cuda")
    C = torch.zeros(512, 512, dtype=torch.float32, device="cuda")
    assert v.probe_noalloc_status(A, B, C) == fk.ESHAPE
    v.close()
