"""Seeded synthetic inputs for the FP-Sketch verifier.

This module is shared by the tests, ``bench.py`` and ``smoke()``.  It holds none of the
verifier's arithmetic: it draws operands, rounds them to the half formats, produces a CPU
stand-in for the guarded GEMM's FP32 output, picks fault sites and writes faults into a copy of
C.  Both the HIP path and the CPU oracle receive exactly the arrays made here.

Shapes and distributions follow the paper's workloads: Gaussian activations N(0, 1) against
weights N(0, 0.02) on transformer projection shapes (Table II, Fig. 3) and uniform or Gaussian
square products.  Output-side faults are additive deltas or IEEE-754 bit flips written into the
finished FP32 product (Sec. VI-A, "output side" faults flip bit 26 of an entry).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

FP32_EXP_BIT26 = 26

# ---------------------------------------------------------------------------------------------
# Half-format rounding (input construction only).


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round FP32 values to bfloat16 (round to nearest, ties to even) and return the bit pattern."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        r[nan] = np.uint16(0x7FC0)
    return r


def f32_to_f16_bits(x: np.ndarray) -> np.ndarray:
    """Round FP32 values to IEEE binary16 (numpy rounds to nearest even) and return the bits."""
    return np.ascontiguousarray(x, dtype=np.float32).astype(np.float16).view(np.uint16)


def half_bits_to_f32(bits: np.ndarray, fmt: str) -> np.ndarray:
    """Widen half bit patterns to FP32 (exact) for the CPU stand-in GEMM."""
    if fmt == "bf16":
        return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)
    if fmt == "fp16":
        return bits.view(np.float16).astype(np.float32)
    raise ValueError(f"unknown half format {fmt!r}")


def round_to_half(x: np.ndarray, fmt: str) -> np.ndarray:
    if fmt == "bf16":
        return f32_to_bf16_bits(x)
    if fmt == "fp16":
        return f32_to_f16_bits(x)
    raise ValueError(f"unknown half format {fmt!r}")


# ---------------------------------------------------------------------------------------------
# Operand draws.


def _draw(rng: np.random.Generator, shape, dist) -> np.ndarray:
    kind = dist[0]
    if kind == "normal":
        std = float(dist[1])
        return (rng.standard_normal(shape, dtype=np.float32) * np.float32(std)).astype(np.float32)
    if kind == "uniform":
        lo, hi = float(dist[1]), float(dist[2])
        return rng.uniform(lo, hi, size=shape).astype(np.float32)
    if kind == "int":
        lo, hi = int(dist[1]), int(dist[2])
        return rng.integers(lo, hi + 1, size=shape).astype(np.float32)
    raise ValueError(f"unknown distribution {dist!r}")


def gen_operands(n1: int, n2: int, n3: int, fmt: str, dist_a, dist_b, seed: int,
                 seed_b: int | None = None):
    """Return (A_bits, B_bits): uint16 arrays n1 x n2 and n2 x n3 in the half format ``fmt``.

    ``seed`` drives A; B uses ``seed_b`` (defaults to ``seed``), so a fixed weight matrix can be
    paired with rotating activations.
    """
    return (gen_side(n1, n2, fmt, dist_a, seed, 0xA),
            gen_side(n2, n3, fmt, dist_b, seed if seed_b is None else seed_b, 0xB))


def gen_side(rows: int, cols: int, fmt: str, dist, seed: int, side: int) -> np.ndarray:
    """One operand of ``gen_operands`` (side 0xA for A, 0xB for B) as uint16 half bits."""
    rng = np.random.Generator(np.random.PCG64([int(seed), int(side)]))
    return round_to_half(_draw(rng, (rows, cols), dist), fmt)


def cpu_gemm_f32(a_bits: np.ndarray, b_bits: np.ndarray, fmt: str) -> np.ndarray:
    """CPU stand-in for the guarded GEMM: half operands, FP32 accumulation, FP32 output."""
    a = half_bits_to_f32(a_bits, fmt)
    b = half_bits_to_f32(b_bits, fmt)
    return np.matmul(a, b, dtype=np.float32)


def mean_abs(c: np.ndarray) -> float:
    """mean |C_ij| of a clean product in FP64 (the unit fault magnitudes are quoted in)."""
    return float(np.mean(np.abs(c.astype(np.float64))))


# ---------------------------------------------------------------------------------------------
# Fault sites and injection (output side: written into a finished FP32 product).


def fault_sites(n1: int, n3: int, count: int, seed: int) -> np.ndarray:
    """``count`` distinct (i, j) coordinates, seeded, as an int64 array of shape (count, 2)."""
    total = n1 * n3
    if count > total:
        raise ValueError("more faults than entries")
    rng = np.random.Generator(np.random.PCG64([int(seed), 0xF]))
    chosen: list[int] = []
    seen: set[int] = set()
    while len(chosen) < count:
        for f in rng.integers(0, total, size=2 * (count - len(chosen)) + 4):
            f = int(f)
            if f not in seen:
                seen.add(f)
                chosen.append(f)
                if len(chosen) == count:
                    break
    flat = np.asarray(chosen, dtype=np.int64)
    return np.stack([flat // n3, flat % n3], axis=1)


def fault_magnitudes(count: int, lo: float, hi: float, unit: float, seed: int,
                     log_uniform: bool = False) -> np.ndarray:
    """Signed magnitudes ±U(lo, hi)·unit (or log-uniform between lo and hi), seeded."""
    rng = np.random.Generator(np.random.PCG64([int(seed), 0xD]))
    if log_uniform:
        mag = np.exp(rng.uniform(math.log(lo), math.log(hi), size=count))
    else:
        mag = rng.uniform(lo, hi, size=count)
    sign = np.where(rng.integers(0, 2, size=count) == 1, -1.0, 1.0)
    return sign * mag * unit


def inject_additive(c: np.ndarray, sites: np.ndarray, deltas: np.ndarray) -> np.ndarray:
    """Copy of C with C[i, j] += delta (in FP32) at each site."""
    out = np.array(c, dtype=np.float32, copy=True)
    for (i, j), d in zip(sites, deltas):
        out[i, j] = np.float32(np.float64(out[i, j]) + float(d))
    return out


def flip_bits(c: np.ndarray, sites: np.ndarray, masks) -> np.ndarray:
    """Copy of C with the FP32 bit pattern of C[i, j] XORed by ``mask`` at each site."""
    out = np.array(c, dtype=np.float32, copy=True)
    u = out.view(np.uint32)
    for (i, j), mk in zip(sites, masks):
        u[i, j] ^= np.uint32(mk)
    return out


def flip_bit_value(x: float, bit: int) -> float:
    """FP32 value with one bit of its pattern inverted (the paper's bit-26 fault is x256)."""
    u = np.array([x], dtype=np.float32).view(np.uint32)
    u ^= np.uint32(1 << bit)
    return float(u.view(np.float32)[0])


def bitflip_plan(count: int, seed: int) -> list[int]:
    """Seeded bit positions for emulated accumulator upsets: mantissa bits 13..22 and exponent
    bits 23..30, one flipped bit per fault."""
    rng = np.random.Generator(np.random.PCG64([int(seed), 0xE]))
    return [int(b) for b in rng.integers(13, 31, size=count)]


def call_faults(w: "Workload", n1: int, n3: int, unit: float, seed: int):
    """Faults of one dirty call of workload ``w``: (sites, deltas, masks).

    ``w.faults`` distinct sites (for "mixed" workloads a seeded count in 0..faults); additive and
    mixed workloads carry signed deltas of U(lo, hi)·unit (log-uniform when ``w.log_uniform``),
    bit-flip workloads one mask per site from ``bitflip_plan``.  The unused one of deltas /
    masks is None."""
    count = w.faults
    if w.fault_kind == "mixed":
        rng = np.random.Generator(np.random.PCG64([int(seed), 0xC]))
        count = int(rng.integers(0, w.faults + 1))
    sites = fault_sites(n1, n3, count, seed)
    if w.fault_kind == "bitflip":
        return sites, None, [1 << b for b in bitflip_plan(count, seed + 1)]
    deltas = fault_magnitudes(count, w.fault_lo, w.fault_hi, unit, seed + 1,
                              log_uniform=w.log_uniform)
    return sites, deltas, None


def apply_faults(values: np.ndarray, deltas, masks) -> np.ndarray:
    """FP32 values at the fault sites after the faults are written (values in site order):
    fl32(value + delta), or the bit pattern XOR mask."""
    v = np.array(values, dtype=np.float32, copy=True).ravel()
    if masks is not None:
        u = v.view(np.uint32)
        for t, mk in enumerate(masks):
            u[t] ^= np.uint32(mk)
        return v
    for t, d in enumerate(deltas):
        v[t] = np.float32(np.float64(v[t]) + float(d))
    return v


# ---------------------------------------------------------------------------------------------
# Named workloads.


@dataclass
class Workload:
    name: str
    n1: int
    n2: int
    n3: int
    fmt: str
    dist_a: tuple
    dist_b: tuple
    faults: int
    fault_lo: float = 0.0
    fault_hi: float = 0.0
    fault_kind: str = "additive"          # "additive" | "bitflip" | "mixed"
    log_uniform: bool = False
    m_forced: int = 0
    rho_min: float = 0.02
    s_budget: int = 16
    calib_calls: int = 16
    extra: dict = field(default_factory=dict)

    @property
    def bytes_abc(self) -> int:
        """Bytes one verify call must read: A and B in half precision and C in FP32."""
        return 2 * self.n1 * self.n2 + 2 * self.n2 * self.n3 + 4 * self.n1 * self.n3


TRANSFORMER_KN = [(4096, 4096), (4096, 12288), (4096, 11008), (11008, 4096),
                  (5120, 5120), (5120, 13824), (13824, 5120), (8192, 8192)]


def workload(name: str) -> Workload:
    if name == "tiny256":
        return Workload("tiny256", 256, 256, 256, "fp16", ("uniform", -1, 1), ("uniform", -1, 1),
                        faults=3, fault_lo=0.5, fault_hi=4.0, m_forced=64)
    if name == "square4096_bf16":
        return Workload("square4096_bf16", 4096, 4096, 4096, "bf16", ("normal", 1.0),
                        ("normal", 1.0), faults=8, fault_lo=0.02, fault_hi=0.09, rho_min=0.015)
    if name == "mlp_down_bf16":
        return Workload("mlp_down_bf16", 4096, 11008, 4096, "bf16", ("normal", 1.0),
                        ("normal", 0.02), faults=16, fault_kind="bitflip")
    if name.startswith("xfmr_"):
        # xfmr_<k>x<n>_<fmt>
        body, fmt = name[5:].rsplit("_", 1)
        k, n = (int(v) for v in body.split("x"))
        return Workload(name, 2048, k, n, fmt, ("normal", 1.0), ("normal", 0.02),
                        faults=4, fault_lo=0.05, fault_hi=4.0)
    if name == "square16384_fp16":
        return Workload("square16384_fp16", 16384, 16384, 16384, "fp16", ("uniform", -1, 1),
                        ("uniform", -1, 1), faults=32, fault_lo=0.02, fault_hi=10.0,
                        fault_kind="mixed", log_uniform=True, rho_min=0.015, s_budget=32,
                        calib_calls=8)
    raise KeyError(name)
