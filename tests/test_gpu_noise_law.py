"""The MI355X noise law (Sec. III-F, Eq. 3 measured for hipBLASLt products): a fresh measurement
lies under the fitted envelope, and a context started from it needs no rebuild at the first
calibration (Sec. III-G) on shapes where the paper's H100 law starts m far too high."""
import pytest

from paper_2609_19758_amd import noise_law as nl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fk():
    import torch
    assert torch.cuda.is_available()
    from paper_2609_19758_amd import fpsketch
    fpsketch.load()
    return fpsketch


@pytest.mark.parametrize("fmt", ["bf16", "fp16"])
def test_measurement_under_the_envelope(fk, fmt):
    law = nl.LAW_GFX950_HIPBLASLT
    x = nl.measure(2048, 3072, 2560, 48, fmt, calls=3, seed=17)
    bound = law[f"law_cf_{fmt}"] * (x.n2 / 8192) ** law["law_n2_exp"]
    print(f"\n{fmt}: normalized {x.normalized:.4f}, envelope {bound:.4f}", flush=True)
    assert 0.5 * bound <= x.normalized <= 1.1 * bound


@pytest.mark.parametrize("fmt", ["bf16", "fp16"])
def test_calibration_converges_in_one_step(fk, fmt):
    """2048 x 4096 x 12288 (a transformer's up projection): started from the measured law the
    first calibration keeps m; started from the paper's law it rebuilds to about the same m."""
    import torch
    n1, n2, n3 = 2048, 4096, 12288
    hd = torch.bfloat16 if fmt == "bf16" else torch.float16
    g = torch.Generator(device="cuda")
    g.manual_seed(23)
    B = (0.02 * torch.randn(n2, n3, device="cuda", generator=g)).to(hd)
    As = [torch.randn(n1, n2, device="cuda", generator=g).to(hd) for _ in range(4)]
    Cs = [torch.mm(A, B, out_dtype=torch.float32) for A in As]
    res = {}
    for name, law in (("measured", nl.LAW_GFX950_HIPBLASLT), ("paper", nl.LAW_PAPER)):
        p = nl.apply_law(fk.default_params(), law)
        v = fk.Verifier(n1, n2, n3, fmt, p)
        m0 = v.m
        for k in range(16):
            v.probe(As[k % 4], B, Cs[k % 4])
        m1, sigma_bar, rebuilt = v.calibrate_noise(Cs[0])
        res[name] = (m0, m1, rebuilt)
        v.close()
    print(f"\n{fmt}: {res}", flush=True)
    assert not res["measured"][2]
    assert res["paper"][2]
    assert abs(res["paper"][1] - res["measured"][0]) <= 0.25 * res["measured"][0]


def test_recalibration_beyond_the_kernels_bucket_limit_is_an_error(fk):
    """Eq. 5's m' above the kernels' 4096 buckets (possible beyond 16384 x 16384 outputs; a tiny
    index budget B* forces it here at 65536 x 64 x 8192, where m_max = 5792): the call returns
    FPSK_ESHAPE, the probe keeps its m and goes on probing."""
    import torch
    from oracle import fpsketch_oracle as o
    n1, n2, n3 = 65536, 64, 8192
    g = torch.Generator(device="cuda").manual_seed(5)
    A = torch.randn(n1, n2, device="cuda", generator=g).to(torch.bfloat16)
    B = torch.randn(n2, n3, device="cuda", generator=g).to(torch.bfloat16)
    C = torch.mm(A, B, out_dtype=torch.float32)
    v = fk.Verifier(n1, n2, n3, "bf16", m=64, b_star=0.001)
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    for _ in range(3):
        v.probe(A, B, C, d_dirty=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 0
    sb = v.probe_stats()["sigma_hat"]
    want, rebuild = o.recalibrate_m(n1, n3, 64, sb, float(C.double().pow(2).mean().sqrt()),
                                    o.Params(b_star=0.001))
    assert rebuild and want > 4096, want       # the rule itself asks for m_max
    with pytest.raises(fk.FpsketchError) as e:
        v.calibrate_noise(C)
    assert e.value.status == fk.ESHAPE and "4096" in str(e.value)
    assert v.m == 64
    v.probe(A, B, C, d_dirty=flag)
    torch.cuda.synchronize()
    assert int(flag.item()) == 0 and v.probe_stats()["dirty"] == 0.0
    v.close()
    del A, B, C
    torch.cuda.empty_cache()
