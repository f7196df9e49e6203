"""FP-Sketch oracle: a plain, slow CPU FP64 implementation of the post hoc GEMM verifier.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline``
leg of ``bench.py`` may import, call or run anything in ``oracle/``.  The HIP product path never
routes through it, and it shares no code, table or constant generator with that path.

What it computes (paper: "Sketching the Error, Not the Product", arXiv 2609.19758):

* the error E = AB - C of a half-precision GEMM delivered at FP32 is formed EXPLICITLY in FP64
  (a numpy matmul is the one library step), and every sketch is its plain definition: a hashed,
  signed, optionally index-weighted bucket sum of E (Sec. III-B, Eq. 1; the factored form the GPU
  uses is never evaluated here);
* the probe statistic, thresholds and verdict (Sec. III-C, III-E, III-I, Algorithm 2 probe part);
* the noise law and bucket-count rules (Sec. III-F, Eq. 3-5) and the localization plan and
  probe recalibration (Sec. III-G);
* one localization round (Algorithm 1) and the verify/localize pipeline (Algorithm 2), with each
  candidate validated from the FP64 error (Sec. III-D, Lemma 1).

Readings of passages the paper leaves open are fixed in the module constants and named where
used (hash family, median of an even count, MAD of the signed sketch, rounding of Eq. 2, the
window order, tie-breaks).  Nothing here is tuned for speed.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

# ---------------------------------------------------------------------------------------------
# Constants of the method.

FP32_MAX = 3.4028234663852886e38          # largest finite binary32 value
EPS32 = 2.0 ** -23                        # FP32 machine epsilon (Sec. III-D)
HUGE_LIMIT = FP32_MAX / 16.0              # out-of-range bound of the exact scan (Sec. III-I)
CLIP_MEAN_CONST = 1.2533                  # sqrt(pi/2), clipped-mean scale (Sec. III-E)
MAD_CONST = 1.4826                        # MAD-to-sigma scale (Sec. III-E)
MEM_CAP_BYTES = 2 ** 31                   # 2 GiB sketch-memory cap on m_loc (Sec. III-G)

# splitmix64 (Steele, Lea, Flood 2014; Vigna's reference mixer): golden-gamma increment and the
# two multipliers of the finalizer.
SM64_GAMMA = 0x9E3779B97F4A7C15
SM64_MUL1 = 0xBF58476D1CE4E5B9
SM64_MUL2 = 0x94D049BB133111EB


@dataclass
class Params:
    """The paper's parameters (Sec. VI-A defaults; s and Delta are the declared budget)."""
    rounds: int = 3            # k independent hash rounds (Sec. III-H)
    rho_min: float = 0.02      # smallest fault magnitude to localize, x rms(C) (Sec. III-G)
    r_star: int = 4            # target radius (Sec. III-G)
    r_max: int = 16            # largest radius (Sec. III-G)
    mu: float = 4.0            # probe margin (Sec. III-E)
    c_valid: float = 100.0     # validation constant c (Sec. III-D)
    b_star: float = 0.3        # index budget target (Sec. III-F)
    c_coll: float = 2.0        # collision constant c of m_comb (Sec. III-F)
    s_budget: int = 16         # declared error budget s
    delta_rc: int = 8          # errors per row or column, Delta
    k_cap: int = 0             # K; 0 means max(64, 8 s) (Sec. III-E)
    # Eq. 3's constants, the paper's envelope: c_f per operand format and the n2 exponent
    law_cf_bf16: float = 0.19
    law_cf_fp16: float = 0.19 * 1.76
    law_n2_exp: float = 0.07

    def law_cf(self, fmt: str) -> float:
        return self.law_cf_fp16 if fmt == "fp16" else self.law_cf_bf16

    @property
    def K(self) -> int:
        return self.k_cap if self.k_cap > 0 else max(64, 8 * self.s_budget)


# ---------------------------------------------------------------------------------------------
# Operand decoding: half bit patterns to FP64, exactly.


def decode_bf16(bits: np.ndarray) -> np.ndarray:
    """bfloat16 is the upper half of a binary32 pattern; widen and reinterpret (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(
        np.float32).astype(np.float64)


def decode_fp16(bits: np.ndarray) -> np.ndarray:
    """IEEE binary16 from its fields: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.int64)
    sign = np.where((b >> 15) & 1, -1.0, 1.0)
    e = (b >> 10) & 0x1F
    f = (b & 0x3FF).astype(np.float64)
    normal = sign * (1024.0 + f) * np.exp2(e.astype(np.float64) - 25.0)
    sub = sign * f * 2.0 ** -24
    out = np.where(e == 0, sub, normal)
    special = e == 31
    if special.any():
        out = np.where(special & (f == 0), sign * np.inf, out)
        out = np.where(special & (f != 0), np.nan, out)
    return out


def decode(bits: np.ndarray, fmt: str) -> np.ndarray:
    if fmt == "bf16":
        return decode_bf16(bits)
    if fmt == "fp16":
        return decode_fp16(bits)
    raise ValueError(fmt)


def error_matrix(a64: np.ndarray, b64: np.ndarray, c32: np.ndarray) -> np.ndarray:
    """E = AB - C in FP64, formed explicitly (Sec. III-B)."""
    return a64 @ b64 - np.asarray(c32, dtype=np.float64)


# ---------------------------------------------------------------------------------------------
# Hash rounds.  The paper asks for independent uniform hashes h1:[n1]->[m], h2:[n3]->[m] and
# Rademacher signs (Sec. III-B, Lemma 2) and names no family.  Reading used here: a splitmix64
# stream keyed per (seed, round, side); index idx takes output idx of the stream keyed with
# key = output (2*round + side) of the stream seeded with `seed`.  The bucket is Lemire's
# multiply-shift reduction of the high 32 bits, the sign is the low bit (1 -> -1).


def _u64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.uint64)


def splitmix64_mix(z: np.ndarray) -> np.ndarray:
    z = _u64(z)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(SM64_MUL1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(SM64_MUL2)
    return z ^ (z >> np.uint64(31))


def splitmix64_stream(seed: int, idx: np.ndarray) -> np.ndarray:
    """Output number idx (0-based) of the splitmix64 generator whose state starts at `seed`."""
    idx = _u64(idx)
    with np.errstate(over="ignore"):
        state = _u64(seed & 0xFFFFFFFFFFFFFFFF) + (idx + np.uint64(1)) * np.uint64(SM64_GAMMA)
    return splitmix64_mix(state)


def round_key(seed: int, rnd: int, side: int) -> int:
    return int(splitmix64_stream(seed, np.array([2 * rnd + side], dtype=np.uint64))[0])


def bucket_sign_from_word(x: np.ndarray, m: int):
    """Bucket = (high 32 bits x m) >> 32 (Lemire's multiply-shift); sign = -1 if bit 0 is set."""
    x = _u64(x)
    bucket = (((x >> np.uint64(32)) * np.uint64(m)) >> np.uint64(32)).astype(np.int64)
    sign = np.where((x & np.uint64(1)) == np.uint64(1), -1.0, 1.0)
    return bucket, sign


def hash_round(seed: int, rnd: int, side: int, n: int, m: int):
    """(bucket[n] in [0, m), sign[n] in {+1, -1}) for one side of one hash round."""
    key = round_key(seed, rnd, side)
    return bucket_sign_from_word(splitmix64_stream(key, np.arange(n, dtype=np.uint64)), m)


@dataclass
class HashRound:
    m: int
    h1: np.ndarray
    v1: np.ndarray
    h2: np.ndarray
    v2: np.ndarray


def make_round(seed: int, rnd: int, n1: int, n3: int, m: int) -> HashRound:
    h1, v1 = hash_round(seed, rnd, 0, n1, m)
    h2, v2 = hash_round(seed, rnd, 1, n3, m)
    return HashRound(m, h1, v1, h2, v2)


# ---------------------------------------------------------------------------------------------
# Sketches (Sec. III-B, Eq. 1 and the first-moment sketches).


def pow2_ceil(n: int) -> int:
    """2^ceil(log2 n) for n >= 1 (1 for n = 1)."""
    p = 1
    while p < n:
        p *= 2
    return p


def row_weights(n1: int) -> np.ndarray:
    """w_i = i / 2^ceil(log2 n1) with i counted from 1 (storage index i -> i + 1)."""
    return np.arange(1, n1 + 1, dtype=np.float64) / pow2_ceil(n1)


def col_weights(n3: int) -> np.ndarray:
    return np.arange(1, n3 + 1, dtype=np.float64) / pow2_ceil(n3)


def bucket_sum(X: np.ndarray, hr: HashRound) -> np.ndarray:
    """m x m grid: entry (a, b) = sum of X_ij over h1(i) = a, h2(j) = b."""
    m = hr.m
    idx = (hr.h1[:, None] * m + hr.h2[None, :]).ravel()
    return np.bincount(idx, weights=X.ravel(), minlength=m * m).reshape(m, m)


def sketches(E: np.ndarray, hr: HashRound, moments: bool = True):
    """S = H1 E H2^T; R and T repeat it with rows weighted by w_i and columns by w_j."""
    signed = hr.v1[:, None] * E * hr.v2[None, :]
    S = bucket_sum(signed, hr)
    if not moments:
        return S, None, None
    n1, n3 = E.shape
    R = bucket_sum(signed * row_weights(n1)[:, None], hr)
    T = bucket_sum(signed * col_weights(n3)[None, :], hr)
    return S, R, T


def abs_contributions(a64, b64, c64, hr: HashRound):
    """Sum of absolute contributions of the factored evaluation of each bucket of S, R, T:
    (|H1||A|)(|B||H2|^T) + |H1||C||H2|^T, with w_i or w_j carried by R or T.  This is the scale
    that bounds the rounding of a floating-point evaluation of Eq. 1."""
    n1, n3 = c64.shape
    aa, ab, ac = np.abs(a64), np.abs(b64), np.abs(c64)
    m = hr.m
    H1 = np.zeros((m, n1))
    H1[hr.h1, np.arange(n1)] = 1.0
    H2 = np.zeros((m, n3))
    H2[hr.h2, np.arange(n3)] = 1.0
    wr, wc = row_weights(n1), col_weights(n3)
    PA, PAw = H1 @ aa, (H1 * wr[None, :]) @ aa
    QB, QBw = ab @ H2.T, ab @ (H2 * wc[None, :]).T
    DS = PA @ QB + H1 @ ac @ H2.T
    DR = PAw @ QB + (H1 * wr[None, :]) @ ac @ H2.T
    DT = PA @ QBw + H1 @ ac @ (H2 * wc[None, :]).T
    return DS, DR, DT


# ---------------------------------------------------------------------------------------------
# Probe (Sec. III-C, III-E, III-I; Algorithm 2, probe part).


def tau_analytic(n2: int, max_a: float, max_b: float, p: Params) -> float:
    """tau = c n2 eps max|A| max|B| (Sec. III-E)."""
    return p.c_valid * n2 * EPS32 * max_a * max_b


def clipped_sigma(S: np.ndarray) -> float:
    """sigma_hat = 1.2533 mean(min(|S|, 5 mean|S|)) (Sec. III-E)."""
    a = np.abs(S).ravel()
    mean_abs = a.mean()
    return CLIP_MEAN_CONST * float(np.minimum(a, 5.0 * mean_abs).mean())


@dataclass
class ProbeResult:
    dirty: bool
    sigma_hat: float
    thr: float
    tau: float
    max_abs: float
    finite: bool
    S: np.ndarray


def probe_from_sketch(S: np.ndarray, n2: int, max_a: float, max_b: float, p: Params) -> ProbeResult:
    m = S.shape[0]
    tau = tau_analytic(n2, max_a, max_b, p)
    sigma = clipped_sigma(S)
    thr = min(tau, p.mu * math.sqrt(2.0 * math.log(m * m)) * sigma)
    finite = bool(np.all(np.isfinite(S)))
    max_abs = float(np.max(np.abs(S)))
    clean = finite and max_abs <= thr
    return ProbeResult(not clean, sigma, thr, tau, max_abs, finite, S)


def probe(a64, b64, c32, hr: HashRound, p: Params) -> ProbeResult:
    E = error_matrix(a64, b64, c32)
    S, _, _ = sketches(E, hr, moments=False)
    return probe_from_sketch(S, a64.shape[1], float(np.max(np.abs(a64))),
                             float(np.max(np.abs(b64))), p)


# ---------------------------------------------------------------------------------------------
# Noise law and bucket counts (Sec. III-F, Eq. 3-5).


def law_sigma_over_rms(n1: int, n2: int, n3: int, m: int, fmt: str, p: Params) -> float:
    """Eq. 3 divided by rms(C): c_f 2^-24 sqrt(n1 n3 n2) (n2/8192)^e / m."""
    return p.law_cf(fmt) * 2.0 ** -24 * math.sqrt(n1 * n3 * n2) * (n2 / 8192.0) ** p.law_n2_exp / m


def m_num(n1: int, n2: int, n3: int, fmt: str, p: Params) -> int:
    """Eq. 4 sized for delta = rms(C) with target B*; rms(C) cancels.  Integer: ceiling."""
    v = max(n1, n3) / p.b_star * p.law_cf(fmt) * 2.0 ** -24 * math.sqrt(n1 * n3 * n2) * \
        (n2 / 8192.0) ** p.law_n2_exp
    return int(math.ceil(v))


def m_comb(p: Params) -> int:
    """ceil(max(3 c Delta, sqrt(3 c s))) (Sec. III-F, Lemma 3)."""
    return int(math.ceil(max(3.0 * p.c_coll * p.delta_rc, math.sqrt(3.0 * p.c_coll * p.s_budget))))


def m_max(n1: int, n3: int) -> int:
    """max(16, floor(sqrt(n1 n3 / 16))): at least 16 entries per bucket on average."""
    return max(16, math.isqrt((n1 * n3) // 16))


def m_start(n1: int, n2: int, n3: int, fmt: str, p: Params) -> int:
    """Eq. 5."""
    mc = m_comb(p)
    return min(max(mc, m_num(n1, n2, n3, fmt, p), 16), max(mc, m_max(n1, n3)))


def m_mem(n2: int) -> int:
    """Largest m with 4 (3 m^2 + 6 m n2) bytes within 2 GiB (Sec. III-G)."""
    lo, hi = 0, 1
    while 4 * (3 * hi * hi + 6 * hi * n2) <= MEM_CAP_BYTES:
        hi *= 2
    while hi - lo > 1:
        mid = (lo + hi) // 2
        if 4 * (3 * mid * mid + 6 * mid * n2) <= MEM_CAP_BYTES:
            lo = mid
        else:
            hi = mid
    return lo


# ---------------------------------------------------------------------------------------------
# Calibration and the localization plan (Sec. III-G).


def median(x: np.ndarray) -> float:
    """Median; an even count takes the mean of the two middle order statistics."""
    s = np.sort(np.asarray(x, dtype=np.float64).ravel())
    n = s.size
    if n == 0:
        return float("nan")
    if n % 2:
        return float(s[n // 2])
    return 0.5 * (float(s[n // 2 - 1]) + float(s[n // 2]))


def rms_hat(c32: np.ndarray) -> float:
    """rms of the finite entries of C taken at stride max(1, floor(n1 n3 / 65536)) over the
    row-major order, magnitudes clipped at 64 x their median.  NaN if no finite sample."""
    flat = np.asarray(c32).ravel()
    stride = max(1, flat.size // 65536)
    samp = flat[::stride].astype(np.float64)
    samp = np.abs(samp[np.isfinite(samp)])
    if samp.size == 0:
        return float("nan")
    clip = 64.0 * median(samp)
    return math.sqrt(float(np.mean(np.minimum(samp, clip) ** 2)))


def radius_rule(B: float) -> int:
    """0 if B <= 0.05, else max(2, ceil(2.5 B))."""
    return 0 if B <= 0.05 else max(2, int(math.ceil(2.5 * B)))


@dataclass
class Plan:
    m_loc: int
    r: int
    B: float
    fallback: bool


def _ok(x: float) -> bool:
    return math.isfinite(x) and x > 0.0


def plan_localize(n1: int, n2: int, n3: int, fmt: str, m: int, sigma_hat: float, rms: float,
                  p: Params) -> Plan:
    """(m_loc, r) from the noise measured on this call; Eq. 3 when it is unusable."""
    mx = max(n1, n3)
    fallback = not (_ok(sigma_hat) and _ok(rms))
    if fallback:
        B = mx * law_sigma_over_rms(n1, n2, n3, m, fmt, p) / p.rho_min
    else:
        B = mx * sigma_hat / (p.rho_min * rms)
    r_b = radius_rule(B)
    if r_b <= p.r_star:
        return Plan(m, r_b, B, fallback)
    grown = 16 * math.ceil(math.ceil(m * r_b / p.r_star) / 16)
    m_loc = max(m, min(grown, m_max(n1, n3), m_mem(n2)))
    b2 = B * m / m_loc
    r = 0 if b2 <= 0.05 else min(p.r_max, max(2, int(math.ceil(2.5 * b2))))
    return Plan(m_loc, r, B, fallback)


def recalibrate_m(n1: int, n3: int, m: int, sigma_bar: float, rms: float, p: Params):
    """Probe recalibration: (m', rebuild?).  B1 = max(n1,n3) sigma_bar / rms(C),
    m' = max(m_comb, 16, min(ceil(m B1 / B*), m_max)); rebuild if m' is outside [m/1.25, 1.25 m].
    """
    if not (_ok(sigma_bar) and _ok(rms)):
        return m, False
    b1 = max(n1, n3) * sigma_bar / rms
    mp = max(m_comb(p), 16, min(int(math.ceil(m * b1 / p.b_star)), m_max(n1, n3)))
    rebuild = mp < m / 1.25 or mp > 1.25 * m
    return (mp if rebuild else m), rebuild


# ---------------------------------------------------------------------------------------------
# Localization (Algorithm 1, Algorithm 2, Sec. III-D, III-E, III-H, III-I).


@dataclass
class Fault:
    i: int
    j: int
    delta: float          # correction to add to C (or the absolute value when `absolute`)
    absolute: bool
    round: int            # 0 for the exact scan, t for hash round t


def mad_sigma(S: np.ndarray) -> float:
    """sigma_MAD = 1.4826 median(|S - median S|), the MAD of the signed sketch.  (The printed
    formula takes |S| inside; that estimate is about 0.59 sigma on clean Gaussian buckets and
    would let ~24 % of them clear tau_c, against the 4.6 % the text states, so the signed MAD,
    which gives sigma and 4.6 %, is used.)"""
    s = np.asarray(S, dtype=np.float64).ravel()
    med = median(s)
    return MAD_CONST * median(np.abs(s - med))


def window_offsets(r: int):
    """All (di, dj) with |di|, |dj| <= r, by Chebyshev then Manhattan distance, then di, dj."""
    offs = [(di, dj) for di in range(-r, r + 1) for dj in range(-r, r + 1)]
    offs.sort(key=lambda o: (max(abs(o[0]), abs(o[1])), abs(o[0]) + abs(o[1]), o[0], o[1]))
    return offs


def validation_bound(a64, b64, i: int, j: int, p: Params) -> float:
    """tau_ij = c eps sum_k |A_ik||B_kj| (Sec. III-D)."""
    return p.c_valid * EPS32 * float(np.abs(a64[i, :]) @ np.abs(b64[:, j]))


def recompute(a64, b64, i: int, j: int) -> float:
    """gamma = A_i,* B_*,j, here in FP64 (products of half values are exact)."""
    return float(a64[i, :] @ b64[:, j])


def scan_absolute(c32: np.ndarray, a64, b64, K: int):
    """Exact scan (Sec. III-I): entries of C that are non-finite or exceed fp32max/16 in
    magnitude, in row-major order, at most K; each recomputed as an absolute value."""
    c = np.asarray(c32)
    bad = ~np.isfinite(c) | (np.abs(c.astype(np.float64)) > HUGE_LIMIT)
    flat = np.flatnonzero(bad.ravel())[:K]
    n3 = c.shape[1]
    out = []
    for f in flat:
        i, j = int(f // n3), int(f % n3)
        out.append(Fault(i, j, recompute(a64, b64, i, j), True, 0))
    return out


def peel(S, R, T, hr: HashRound, faults, n1: int, n3: int):
    """Subtract v1(i) v2(j) delta (1, w_i, w_j) at (h1(i), h2(j)) for each finite fault found
    so far (Sec. III-H); absolute entries are already absent from the sketch."""
    wr_scale, wc_scale = pow2_ceil(n1), pow2_ceil(n3)
    for f in faults:
        if f.absolute:
            continue
        a, b = hr.h1[f.i], hr.h2[f.j]
        s = hr.v1[f.i] * hr.v2[f.j] * f.delta
        S[a, b] -= s
        R[a, b] -= s * (f.i + 1) / wr_scale
        T[a, b] -= s * (f.j + 1) / wc_scale


@dataclass
class RoundTrace:
    sigma_mad: float
    tau_c: float
    tau_d: float
    n_above_tau_c: int
    Q: list
    U: list
    centers: dict
    S: np.ndarray


def round_cut(S: np.ndarray, n1: int, n3: int, r: int, tau: float):
    """The round's noise and thresholds (Sec. III-E, III-G): sigma_MAD of the peeled S, the
    candidate threshold tau_c = min(tau, 2 sigma_MAD), the decodability threshold
    tau_d = max(n1, n3) sigma_MAD / max(r, 1/2), and the cut max(tau_c, tau_d) a bucket must
    exceed."""
    sig = mad_sigma(S)
    tau_c = min(tau, 2.0 * sig)
    tau_d = max(n1, n3) * sig / max(r, 0.5)
    return sig, tau_c, tau_d, max(tau_c, tau_d)


def candidate_buckets(S, R, T, cut: float, K: int):
    """Buckets above the cut (Sec. III-E): Q is the K largest |S_ab| in the order |S_ab|
    descending, then flat index a*m + b ascending; U keeps those of Q whose S is nonzero and
    whose S, R and T are finite (Eq. 2 needs all three), in Q's order."""
    absS = np.abs(S).ravel()
    Sf, Rf, Tf = S.ravel(), R.ravel(), T.ravel()
    above = np.flatnonzero(absS > cut)
    Q = sorted(above.tolist(), key=lambda f: (-absS[f], f))[:K]
    U = [f for f in Q if Sf[f] != 0.0 and all(math.isfinite(x) for x in (Sf[f], Rf[f], Tf[f]))]
    return Q, U


def bucket_centers(U, S, R, T, n1: int, n3: int) -> dict:
    """Eq. 2 for each usable bucket: the 1-based indices 2^L R/S and 2^L' T/S, rounded half to
    even and returned 0-based; a non-finite ratio or one beyond 2^40 gives no center."""
    L1, L3 = pow2_ceil(n1), pow2_ceil(n3)
    Sf, Rf, Tf = S.ravel(), R.ravel(), T.ravel()
    centers = {}
    for f in U:
        ri = L1 * Rf[f] / Sf[f]
        rj = L3 * Tf[f] / Sf[f]
        if all(math.isfinite(x) and abs(x) <= 2.0 ** 40 for x in (ri, rj)):
            centers[f] = (int(np.rint(ri)) - 1, int(np.rint(rj)) - 1)
    return centers


def search_windows(order, centers: dict, E, a64, b64, r: int, F: list, p: Params, rnd: int):
    """The validated search (Sec. III-D, Sec. III-E): the (2r+1)^2 windows around the centers
    are visited offset by offset in the canonical window order, and at each offset every bucket
    still searching, in `order`, tests its coordinate.  A coordinate outside C or already in F is
    passed over; one whose FP64 error exceeds its validation bound tau_ij is accepted (appended to
    F as round `rnd`) and ends its bucket's search."""
    n1, n3 = E.shape
    searching = [f for f in order if f in centers]
    found = {(g.i, g.j) for g in F}
    for di, dj in window_offsets(r):
        if not searching:
            break
        keep = []
        for f in searching:
            i, j = centers[f][0] + di, centers[f][1] + dj
            inside = 0 <= i < n1 and 0 <= j < n3
            if inside and (i, j) not in found and abs(float(E[i, j])) > \
                    validation_bound(a64, b64, i, j, p):
                F.append(Fault(i, j, float(E[i, j]), False, rnd))
                found.add((i, j))
            else:
                keep.append(f)
        searching = keep
    return F


def localize_round(a64, b64, E, hr: HashRound, r: int, tau: float, F: list, p: Params,
                   rnd: int, trace: list | None = None):
    """One round of localization (Algorithm 1) from the definitions above: the sketches of this
    round's hash, with the faults found so far peeled; the cut; the candidate buckets; their
    centers (Eq. 2); the validated search.  Appends accepted faults to F."""
    n1, n3 = E.shape
    S, R, T = sketches(E, hr, moments=True)
    peel(S, R, T, hr, F, n1, n3)
    sig, tau_c, tau_d, cut = round_cut(S, n1, n3, r, tau)
    Q, U = candidate_buckets(S, R, T, cut, p.K)
    centers = bucket_centers(U, S, R, T, n1, n3)
    search_windows(U, centers, E, a64, b64, r, F, p, rnd)
    if trace is not None:
        trace.append(RoundTrace(sig, tau_c, tau_d, int(np.count_nonzero(np.abs(S) > tau_c)), Q,
                                U, centers, S))
    return F


@dataclass
class LocalizeResult:
    faults: list
    plan: Plan
    sigma_hat: float
    rms: float
    tau: float
    trace: list = field(default_factory=list)


def patch_absolute(c32: np.ndarray, F_abs: list) -> np.ndarray:
    """C holding the recomputed (FP32) value of each absolute entry while sketching."""
    cp = np.array(c32, dtype=np.float32, copy=True)
    for f in F_abs:
        cp[f.i, f.j] = np.float32(f.delta)
    return cp


def localize(a64, b64, c32, fmt: str, m: int, seed: int, p: Params,
             sigma_probe: float | None = None, plan: Plan | None = None) -> LocalizeResult:
    """Algorithm 2, localize part: exact scan, plan, then k fresh hash rounds of Algorithm 1.

    Round t (t = 1..k) uses hash round t of `seed` at m_loc.  When no probe estimate is given the
    noise is the MAD estimate of a fresh S built at the probe's m with hash round 0 of `seed`
    (Sec. III-G).  C is not modified.
    """
    n1, n2 = a64.shape
    n3 = b64.shape[1]
    tau = tau_analytic(n2, float(np.max(np.abs(a64))), float(np.max(np.abs(b64))), p)
    F_abs = scan_absolute(c32, a64, b64, p.K)
    cp = patch_absolute(c32, F_abs)
    E = error_matrix(a64, b64, cp)
    rms = rms_hat(c32)
    if sigma_probe is None:
        S0, _, _ = sketches(E, make_round(seed, 0, n1, n3, m), moments=False)
        sig = mad_sigma(S0)
    else:
        sig = float(sigma_probe)
    if plan is None:
        plan = plan_localize(n1, n2, n3, fmt, m, sig, rms, p)
    F = list(F_abs)
    trace: list = []
    for t in range(1, p.rounds + 1):
        hr = make_round(seed, t, n1, n3, plan.m_loc)
        localize_round(a64, b64, E, hr, plan.r, tau, F, p, t, trace)
    return LocalizeResult(F, plan, sig, rms, tau, trace)


# ---------------------------------------------------------------------------------------------
# Apply (Algorithm 2, last part).


def apply_records(c32: np.ndarray, F) -> np.ndarray:
    """A repaired copy of C: each record written in order, C_ij := delta for an absolute entry
    (its recomputed value), else C_ij := C_ij + delta, the sum formed in FP64 and rounded to
    FP32 (C is delivered in FP32).  The input is not modified."""
    out = np.array(c32, dtype=np.float32, copy=True)
    for f in F:
        if f.absolute:
            out[f.i, f.j] = np.float32(f.delta)
        else:
            out[f.i, f.j] = np.float32(np.float64(out[f.i, f.j]) + float(f.delta))
    return out


def apply_and_reprobe(a64, b64, c32, F, seed: int, m: int, p: Params):
    """Algorithm 2's apply step: write the records, then probe the repaired C once more with a
    fresh hash round (round 0 of `seed`) at the probe's m.  Returns (repaired C, probe result);
    when the probe fires the caller recomputes C = AB at FP32 (the GEMM is the caller's)."""
    c2 = apply_records(c32, F)
    n1, n3 = c2.shape
    res = probe(a64, b64, c2, make_round(seed, 0, n1, n3, m), p)
    return c2, res
