"""Noise-law characterization of the probe on this GPU and BLAS (Sec. III-F, Eq. 3).

Eq. 3 bounds the noise of a clean sketch bucket by c_f 2^-24 sqrt(n1 n3 n2) (n2/8192)^e rms(C)/m.
The paper fits c_f and e on one GPU and one BLAS and notes that both belong to the library that
computed C (its blocking sets how far its summation departs from sequential order), so the law
is only the starting point of the bucket count and the noise is measured at run time.  This
module repeats that characterization for the products a caller actually verifies: it measures
the probe's noise estimate sigma-hat on clean products over sweeps of n1, n3, m and n2 in both
half formats, normalizes each by 2^-24 sqrt(n1 n3 n2) rms-hat(C) / m, fits the n2 exponent as a
robust slope and takes c_f per format as the upper envelope (no measurement exceeds the fitted
law).  The result goes into the context parameters
(law_cf_bf16, law_cf_fp16, law_n2_exp), where Eq. 3-5 read it.

Operands follow the paper's characterization: A ~ N(0, 1), B ~ N(0, 0.02), rounded to the half
format; C comes from the caller's GEMM (by default torch.mm with an FP32 result, hipBLASLt).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, asdict
from typing import Callable, Optional

import numpy as np

from . import fpsketch as fk

# The paper's envelope, fitted on an H100 with cuBLAS (Eq. 3).
LAW_PAPER = {"law_cf_bf16": 0.19, "law_cf_fp16": 0.19 * 1.76, "law_n2_exp": 0.07}

# The same characterization (default_sweep, 4 clean calls per shape, fit) on one MI355X with
# hipBLASLt products (torch.mm, FP32 result): the normalized noise is flat in n1, n3, m and n2
# up to 16384 (0.097 to 0.105 BF16, 0.102 to 0.107 FP16), and drops to 0.065 at n2 = 32768
# where the library changes kernels; the robust slope is 0.
LAW_GFX950_HIPBLASLT = {"law_cf_bf16": 0.1050, "law_cf_fp16": 0.1073, "law_n2_exp": 0.0}


@dataclass
class Measurement:
    n1: int
    n2: int
    n3: int
    m: int
    fmt: str
    calls: int
    sigma_hat: float        # mean probe sigma-hat over the clean calls
    rms: float              # rms-hat(C) of the first call's product
    normalized: float       # sigma_hat m / (2^-24 sqrt(n1 n3 n2) rms)


def default_sweep() -> list[tuple[int, int, int, int, str]]:
    """(n1, n2, n3, m, fmt): the paper's axes around a 4096^3 product (n3 from 1024 to 16384, m
    from 32 to 512, n1 from 1024 to 8192) and an n2 sweep from 1024 to 32768 at n1 = n3 = 2048,
    in both formats."""
    shapes = []
    for fmt in ("bf16", "fp16"):
        for n3 in (1024, 4096, 16384):
            shapes.append((4096, 4096, n3, 64, fmt))
        for m in (32, 128, 256, 512):
            shapes.append((4096, 4096, 4096, m, fmt))
        for n1 in (1024, 8192):
            shapes.append((n1, 4096, 4096, 64, fmt))
        for n2 in (1024, 2048, 4096, 8192, 16384, 32768):
            shapes.append((2048, n2, 2048, 64, fmt))
    return shapes


def _torch_gemm(A, B):
    import torch
    try:
        return torch.mm(A, B, out_dtype=torch.float32)
    except (TypeError, RuntimeError, NotImplementedError):
        return torch.mm(A.float(), B.float())


def rms_hat(C) -> float:
    """rms-hat(C) of a device product (Sec. III-G): the strided sample is taken on the device,
    the clipped rms by the library."""
    flat = C.reshape(-1)
    stride = max(1, flat.numel() // 65536)
    samp = np.ascontiguousarray(flat[::stride].float().cpu().numpy(), dtype=np.float32)
    return fk.rms_hat_samples(samp)


def measure(n1: int, n2: int, n3: int, m: int, fmt: str, calls: int = 4, seed: int = 0,
            gemm: Optional[Callable] = None) -> Measurement:
    """Mean probe sigma-hat over `calls` clean products (distinct activations, one weight)."""
    import torch
    gemm = gemm or _torch_gemm
    hd = torch.bfloat16 if fmt == "bf16" else torch.float16
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    B = (0.02 * torch.randn(n2, n3, device="cuda", generator=g)).to(hd)
    v = fk.Verifier(n1, n2, n3, fmt, m=m)
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    sig = []
    rms = float("nan")
    for k in range(calls):
        A = torch.randn(n1, n2, device="cuda", generator=g).to(hd)
        C = gemm(A, B)
        v.probe(A, B, C, d_dirty=flag)
        st = v.probe_stats()
        if st["dirty"] != 0.0:
            raise RuntimeError(f"clean product {n1}x{n2}x{n3} {fmt} m={m} reported dirty")
        sig.append(st["sigma_hat"])
        if k == 0:
            rms = rms_hat(C)
        del A, C
    v.close()
    s = float(np.mean(sig))
    norm = s * m / (2.0 ** -24 * math.sqrt(float(n1) * n3 * n2) * rms)
    return Measurement(n1, n2, n3, m, fmt, calls, s, rms, norm)


def fit(ms: list[Measurement]) -> dict:
    """Eq. 3 fitted to measurements.  The n2 exponent is the Theil-Sen slope of
    log(normalized) against log(n2): the median of the slopes between every two measurements of
    one format at different n2 (robust to a library that switches kernels at some n2, which a
    least-squares slope would follow).  Then c_f per format is the largest
    normalized (n2 / 8192)^-e, so that no measurement exceeds the law."""
    fmts = sorted({x.fmt for x in ms})
    slopes = []
    for f in fmts:
        xs = [x for x in ms if x.fmt == f]
        for i in range(len(xs)):
            for j in range(i + 1, len(xs)):
                if xs[i].n2 != xs[j].n2:
                    slopes.append((math.log(xs[j].normalized) - math.log(xs[i].normalized)) /
                                  (math.log(xs[j].n2) - math.log(xs[i].n2)))
    e = float(np.median(slopes)) if slopes else 0.0
    out = {"law_n2_exp": e}
    for f in fmts:
        env = max(x.normalized * (x.n2 / 8192.0) ** -e for x in ms if x.fmt == f)
        out[f"law_cf_{f}"] = float(env)
    return out


def apply_law(params: "fk.Params", law: dict) -> "fk.Params":
    """Set the law's constants in a parameter block (other fields unchanged)."""
    for k in ("law_cf_bf16", "law_cf_fp16", "law_n2_exp"):
        if k in law:
            setattr(params, k, float(law[k]))
    return params


def as_rows(ms: list[Measurement]) -> list[dict]:
    return [asdict(x) for x in ms]
