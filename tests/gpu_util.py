"""Helpers shared by the GPU tests: uploading seeded inputs and the black-box GEMM."""
import numpy as np

from oracle import fpsketch_oracle as o
from paper_2609_19758_amd import workloads as wl


def torch_mod():
    import torch
    return torch


def to_dev_half(bits: np.ndarray, fmt: str):
    torch = torch_mod()
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to("cuda")
    return t.view(torch.bfloat16 if fmt == "bf16" else torch.float16)


def to_dev_f32(c: np.ndarray):
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(c, dtype=np.float32)).to("cuda")


def gemm_f32(A, B):
    """The guarded GEMM as a black box: half operands, FP32 output (hipBLASLt)."""
    torch = torch_mod()
    try:
        return torch.mm(A, B, out_dtype=torch.float32)
    except (TypeError, RuntimeError, NotImplementedError):
        return torch.mm(A.float(), B.float())


def int_case(n1, n2, n3, fmt, seed, lo=-4, hi=4):
    """Small-integer operands (exact in both half formats) and C = AB exactly."""
    a_bits, b_bits = wl.gen_operands(n1, n2, n3, fmt, ("int", lo, hi), ("int", lo, hi), seed)
    a64, b64 = o.decode(a_bits, fmt), o.decode(b_bits, fmt)
    c = (a64 @ b64).astype(np.float32)
    return a_bits, b_bits, a64, b64, c


def bucket_reference(a_bits, b_bits, fmt, C, hr, a: int, b: int):
    """S, R, T of bucket (a, b) from the definition (the explicit E over the bucket's rows and
    columns, FP64) and D^S, the sum of absolute contributions.  C is the device product; only
    the bucket's block of it is copied to the host."""
    torch = torch_mod()
    n1, n3 = a_bits.shape[0], b_bits.shape[1]
    rows = np.flatnonzero(hr.h1 == a)
    cols = np.flatnonzero(hr.h2 == b)
    if rows.size == 0 or cols.size == 0:
        return (0.0, 0.0, 0.0), 0.0
    a64 = o.decode(np.ascontiguousarray(a_bits[rows]), fmt)
    b64 = o.decode(np.ascontiguousarray(b_bits[:, cols]), fmt)
    ri = torch.from_numpy(rows).to(C.device)
    ci = torch.from_numpy(cols).to(C.device)
    c = C.index_select(0, ri).index_select(1, ci).cpu().numpy().astype(np.float64)
    E = a64 @ b64 - c
    v1, v2 = hr.v1[rows], hr.v2[cols]
    w1 = (rows + 1) / o.pow2_ceil(n1)
    w2 = (cols + 1) / o.pow2_ceil(n3)
    S = v1 @ E @ v2
    R = (v1 * w1) @ E @ v2
    T = v1 @ E @ (v2 * w2)
    D = np.abs(a64).sum(axis=0) @ np.abs(b64).sum(axis=1) + np.abs(c).sum()
    return (float(S), float(R), float(T)), float(D)


def rms_hat_device(C) -> float:
    """The oracle's rms-hat of a device product: the oracle's strided sample (stride
    max(1, floor(n1 n3 / 65536)) over the row-major order) is taken on the device, and the
    oracle's rule applied to it; on that sample the oracle's own stride is 1, so the value is the
    oracle's on the whole C."""
    flat = C.reshape(-1)
    stride = max(1, flat.numel() // 65536)
    samp = flat[::stride].cpu().numpy()
    assert max(1, samp.size // 65536) == 1
    return o.rms_hat(samp)


def site_truth(a_bits, b_bits, fmt, sites, cvals, floor: float, p):
    """For each fault site: the FP64 error E_ij = gamma - C_ij (gamma for absolute entries), the
    validation bound tau_ij, and whether the method must recover it: C_ij non-finite or beyond
    fp32max/16 (exact scan), else |E_ij| >= floor and |E_ij| > tau_ij."""
    out = {}
    for (i, j), x in zip(np.asarray(sites).tolist(), np.asarray(cvals, dtype=np.float32)):
        a64 = o.decode(np.ascontiguousarray(a_bits[i:i + 1]), fmt)
        b64 = o.decode(np.ascontiguousarray(b_bits[:, j:j + 1]), fmt)
        gamma = o.recompute(a64, b64, 0, 0)
        tau = o.validation_bound(a64, b64, 0, 0, p)
        x = float(x)
        absolute = (not np.isfinite(x)) or abs(x) > o.HUGE_LIMIT
        e = gamma if absolute else gamma - x
        must = absolute or (abs(e) >= floor and abs(e) > tau)
        out[(i, j)] = (e, tau, absolute, must)
    return out
