"""The noise-law fit (Sec. III-F, Eq. 3): on measurements that follow a known law exactly the
fit returns it; one kernel switch at a large n2 does not move the exponent; the envelope covers
every measurement.  The constants reach Eq. 3-5 through the context parameters."""
import math

import numpy as np

from oracle import fpsketch_oracle as o
from paper_2609_19758_amd import fpsketch as fk
from paper_2609_19758_amd import noise_law as nl


def _meas(n1, n2, n3, m, fmt, y):
    return nl.Measurement(n1, n2, n3, m, fmt, 4, float("nan"), 1.0, y)


def test_fit_recovers_an_exact_law():
    cf = {"bf16": 0.17, "fp16": 0.29}
    e = 0.07
    ms = [_meas(4096, n2, 4096, 64, f, cf[f] * (n2 / 8192) ** e)
          for f in cf for n2 in (1024, 2048, 4096, 8192, 16384, 65536)]
    law = nl.fit(ms)
    assert abs(law["law_n2_exp"] - e) < 1e-12
    assert abs(law["law_cf_bf16"] - 0.17) < 1e-12 and abs(law["law_cf_fp16"] - 0.29) < 1e-12


def test_fit_is_robust_to_one_kernel_switch_and_is_an_envelope():
    rng = np.random.Generator(np.random.PCG64(5))
    ms = []
    for f in ("bf16", "fp16"):
        for n2 in (1024, 2048, 4096, 8192, 16384):
            ms.append(_meas(2048, n2, 2048, 64, f, 0.1 * (1 + 0.03 * rng.standard_normal())))
        ms.append(_meas(2048, 32768, 2048, 64, f, 0.065))      # a different kernel
    law = nl.fit(ms)
    assert abs(law["law_n2_exp"]) < 0.02
    for x in ms:
        bound = law[f"law_cf_{x.fmt}"] * (x.n2 / 8192) ** law["law_n2_exp"]
        assert x.normalized <= bound * (1 + 1e-12)


def test_measured_law_sets_the_start_m():
    """The MI355X constants change Eq. 5 exactly as the oracle does with the same constants."""
    law = nl.LAW_GFX950_HIPBLASLT
    po = o.Params(**law)
    pl = nl.apply_law(fk.default_params(), law)
    for (n1, n2, n3) in ((2048, 4096, 12288), (2048, 5120, 13824), (4096, 11008, 4096),
                         (16384, 16384, 16384)):
        for fmt in ("bf16", "fp16"):
            assert fk.m_start(n1, n2, n3, fmt, pl) == o.m_start(n1, n2, n3, fmt, po)
            assert fk.m_start(n1, n2, n3, fmt, pl) <= fk.m_start(n1, n2, n3, fmt)
    assert math.isclose(pl.law_cf_bf16, law["law_cf_bf16"])
