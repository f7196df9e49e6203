"""Deferred probes (fpsketch_probe_deferred / fpsketch_probe_flush): each call's pass, the
previous call's block products and the decision of the call before run in one launch.  Every
call's verdict, the statistics and the running noise sum equal those of the same sequence of
ordinary probes bit for bit; other calls on the context flush first; shapes off the block path
run ordinary probes.  The verdicts and the last call's statistics are also checked against the
oracle's probe."""
import numpy as np
import pytest

from oracle import fpsketch_oracle as o
from paper_2609_19758_amd import workloads as wl
from gpu_util import gemm_f32, to_dev_half

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fk():
    import torch
    assert torch.cuda.is_available()
    from paper_2609_19758_amd import fpsketch
    fpsketch.load()
    return fpsketch


def _sequence(n1, n2, n3, fmt, calls, seed, bits=None):
    """(A_k, B, C_k, dirty_k): one weight, fresh activations, every third product faulted.  With
    a list `bits`, the operands' bits (a_k, b) are appended to it per call."""
    import torch
    b_bits = wl.gen_side(n2, n3, fmt, ("normal", 0.02), seed, 0xB)
    B = to_dev_half(b_bits, fmt)
    out = []
    for k in range(calls):
        a_bits = wl.gen_side(n1, n2, fmt, ("normal", 1.0), seed + 1 + k, 0xA)
        A = to_dev_half(a_bits, fmt)
        C = gemm_f32(A, B)
        dirty = k % 3 == 1
        if dirty:
            C[(7 * k) % n1, (11 * k) % n3] += 0.5 * float(C.abs().mean().item())
        out.append((A, B, C, dirty))
        if bits is not None:
            bits.append((a_bits, b_bits))
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("n1,n2,n3,m,fmt", [
    (512, 768, 640, 48, "bf16"),
    (130, 37, 131, 7, "fp16"),       # element loads
    (600, 4100, 520, 48, "bf16"),    # two block-product slices, 3 x 3 blocks
    (300, 512, 260, 64, "fp16"),     # m > 48: 3 x 3 blocks in the pipelined launch
    (640, 4100, 520, 49, "bf16"),    # m = 49, two slices
    (600, 512, 2048, 64, "bf16"),    # C tiles one per wave in both launches
    (600, 64, 8192, 64, "bf16"),     # B chunks in rotated order (two whole chunks)
])
def test_deferred_equals_ordinary(fk, n1, n2, n3, m, fmt):
    import torch
    bits = []
    seq = _sequence(n1, n2, n3, fmt, 7, 61, bits)
    vd = fk.Verifier(n1, n2, n3, fmt, m=m)
    vs = fk.Verifier(n1, n2, n3, fmt, m=m)
    fd = [torch.zeros(1, dtype=torch.int32, device="cuda") for _ in seq]
    fs = [torch.zeros(1, dtype=torch.int32, device="cuda") for _ in seq]
    stats = []
    for k, (A, B, C, dirty) in enumerate(seq):
        vd.probe_deferred(A, B, C, d_dirty=fd[k])
        vs.probe(A, B, C, d_dirty=fs[k])
        stats.append(vs.probe_stats())
    vd.probe_flush()
    torch.cuda.synchronize()
    for k, (_, _, _, dirty) in enumerate(seq):
        assert int(fd[k].item()) == int(fs[k].item()) == int(dirty), k
    assert vd.probe_stats() == stats[-1]
    # the deferred verdicts and the last call's statistics against the oracle's probe (the same
    # hash round, the definition of S in FP64; its noise estimate within 5 %, as for the
    # ordinary probe: the FP32 factors round differently from the FP64 definition)
    hr = o.make_round(vd.params.seed, 0, n1, n3, m)
    p = o.Params()
    b64 = o.decode(bits[0][1], fmt)
    for k in (0, 1, len(seq) - 1):
        ref = o.probe(o.decode(bits[k][0], fmt), b64, seq[k][2].cpu().numpy(), hr, p)
        assert ref.dirty == bool(int(fd[k].item())), k
    st = vd.probe_stats()
    assert abs(st["tau"] / ref.tau - 1) < 1e-12
    assert abs(st["sigma_hat"] / ref.sigma_hat - 1) < 0.05
    # the running noise sums agree: the same calibration outcome
    assert vd.calibrate_noise(seq[0][2]) == vs.calibrate_noise(seq[0][2])
    vd.close()
    vs.close()


def test_other_calls_flush_first(fk):
    """An ordinary probe, probe_stats and localize after deferred calls see every deferred call
    decided; a flush with nothing pending is a no-op."""
    import torch
    n1, n2, n3, m, fmt = 256, 512, 384, 32, "bf16"
    seq = _sequence(n1, n2, n3, fmt, 4, 71)
    v = fk.Verifier(n1, n2, n3, fmt, m=m)
    flags = [torch.zeros(1, dtype=torch.int32, device="cuda") for _ in seq]
    for k, (A, B, C, _) in enumerate(seq[:2]):
        v.probe_deferred(A, B, C, d_dirty=flags[k])
    st = v.probe_stats()                       # flushes: call 1 (dirty) decided last
    assert st["dirty"] == 1.0 and int(flags[1].item()) == 1 and int(flags[0].item()) == 0
    v.probe_flush()
    A, B, C, _ = seq[3]
    v.probe_deferred(*seq[2][:3], d_dirty=flags[2])
    v.probe(A, B, C, d_dirty=flags[3])         # flushes call 2 first
    torch.cuda.synchronize()
    assert int(flags[2].item()) == 0 and int(flags[3].item()) == 0
    assert v.probe_stats()["dirty"] == 0.0
    A, B, C, _ = seq[1]
    v.probe_deferred(A, B, C)
    recs, n, status = v.localize(A, B, C, seed=5, sigma_from_probe=True)
    assert status == fk.OK and n == 1
    v.close()


def test_deferred_off_the_block_path_is_an_ordinary_probe(fk):
    import torch
    n1, n2, n3, m, fmt = 384, 520, 300, 96, "fp16"
    seq = _sequence(n1, n2, n3, fmt, 3, 81)
    v = fk.Verifier(n1, n2, n3, fmt, m=m)
    for A, B, C, dirty in seq:
        f = torch.zeros(1, dtype=torch.int32, device="cuda")
        v.probe_deferred(A, B, C, d_dirty=f)
        torch.cuda.synchronize()
        assert int(f.item()) == int(dirty)      # decided within the call
    v.close()


def test_deferred_stream_mismatch_is_rejected(fk):
    import torch
    n1, n2, n3, fmt = 256, 256, 256, "bf16"
    seq = _sequence(n1, n2, n3, fmt, 2, 91)
    v = fk.Verifier(n1, n2, n3, fmt, m=16)
    other = torch.cuda.Stream()
    A, B, C, _ = seq[0]
    v.probe_deferred(A, B, C)
    status = v.lib.fpsketch_probe_deferred(v.handle, A.data_ptr(), B.data_ptr(), C.data_ptr(),
                                           fk.F32, None, other.cuda_stream)
    assert status == fk.EINVAL
    assert v.lib.fpsketch_probe_flush(v.handle, other.cuda_stream) == fk.EINVAL
    v.probe_flush()
    assert v.lib.fpsketch_probe_flush(v.handle, other.cuda_stream) == fk.OK   # nothing pending
    v.close()


def test_cached_deferred_equals_cached(fk):
    """Deferred cached probes mixed with deferred streamed ones: every verdict and the final
    statistics equal the ordinary calls'."""
    import torch
    n1, n2, n3, m, fmt = 512, 1000, 384, 40, "bf16"
    seq = _sequence(n1, n2, n3, fmt, 6, 101)
    B = seq[0][1]
    vd = fk.Verifier(n1, n2, n3, fmt, m=m)
    vs = fk.Verifier(n1, n2, n3, fmt, m=m)
    vd.cache_b(B)
    vs.cache_b(B)
    fd = [torch.zeros(1, dtype=torch.int32, device="cuda") for _ in seq]
    fs = [torch.zeros(1, dtype=torch.int32, device="cuda") for _ in seq]
    for k, (A, _, C, _) in enumerate(seq):
        if k % 2:
            vd.probe_cached_deferred(A, C, d_dirty=fd[k])
            vs.probe_cached(A, C, d_dirty=fs[k])
        else:
            vd.probe_deferred(A, B, C, d_dirty=fd[k])
            vs.probe(A, B, C, d_dirty=fs[k])
    last = vs.probe_stats()
    vd.probe_flush()
    torch.cuda.synchronize()
    for k, (_, _, _, dirty) in enumerate(seq):
        assert int(fd[k].item()) == int(fs[k].item()) == int(dirty), k
    assert vd.probe_stats() == last
    vd.close()
    vs.close()
