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
