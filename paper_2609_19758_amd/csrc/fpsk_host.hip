// Host side of the FP-Sketch verifier library: the C ABI of include/fpsketch.h.
//
// Owns the hash rounds and bucket-sorted tables (Sec. III-B), the bucket-count rules and the
// localization plan (Eq. 3-5, Sec. III-G), device workspaces, and the localization driver
// (Algorithm 2 with Algorithm 1 per round).  Every arithmetic step over A, B and C runs in the
// kernels of fpsk_kernels.hip; the host handles O(m^2) selection on the dirty path only.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <numeric>
#include <string>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "../../include/fpsketch.h"
#include "fpsk_internal.h"

using fpsk::kColTile;
using fpsk::kThreads;

namespace {

thread_local std::string g_last_error;

fpsketch_status fail(fpsketch_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

#define FPSK_HIP(call)                                                                    \
  do {                                                                                    \
    hipError_t e_ = (call);                                                               \
    if (e_ != hipSuccess) {                                                               \
      return fail(e_ == hipErrorOutOfMemory ? FPSK_ENOMEM : FPSK_EHIP,                    \
                  std::string(#call) + " failed: " + hipGetErrorString(e_));              \
    }                                                                                     \
  } while (0)

#define FPSK_TRY(expr)                      \
  do {                                      \
    fpsketch_status s_ = (expr);            \
    if (s_ != FPSK_OK) return s_;           \
  } while (0)

// ------------------------------------------------------------------------------------------
// splitmix64 (Steele, Lea and Flood 2014; Vigna's reference mixer).  Output idx of the stream
// whose state starts at `seed` is mix(seed + (idx + 1) * golden_gamma).

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

inline uint64_t sm_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

inline uint64_t sm_output(uint64_t seed, uint64_t idx) { return sm_mix(seed + (idx + 1) * kGamma); }

// Hash of one side of one round: key = output (2 round + side) of the stream at `seed`;
// index idx uses output idx of the stream at key; bucket = (x >> 32) * m >> 32; sign = bit 0.
void hash_side(uint64_t seed, int round, int side, int64_t n, int m, int32_t* bucket,
               int8_t* sign) {
  const uint64_t key = sm_output(seed, 2ull * static_cast<uint64_t>(round) + side);
  for (int64_t idx = 0; idx < n; ++idx) {
    const uint64_t x = sm_output(key, static_cast<uint64_t>(idx));
    bucket[idx] = static_cast<int32_t>(((x >> 32) * static_cast<uint64_t>(m)) >> 32);
    sign[idx] = (x & 1ull) ? -1 : 1;
  }
}

int64_t pow2_ceil(int64_t n) {
  int64_t p = 1;
  while (p < n) p *= 2;
  return p;
}

// ------------------------------------------------------------------------------------------
// Bucket-count rules (Sec. III-F, Eq. 3-5) and plan (Sec. III-G).

double law_cf(fpsketch_dtype dt, const fpsketch_params& p) {
  return dt == FPSK_F16 ? p.law_cf_fp16 : p.law_cf_bf16;
}

int32_t m_comb(const fpsketch_params& p) {
  const double a = 3.0 * p.c_coll * p.delta_rc;
  const double b = std::sqrt(3.0 * p.c_coll * p.s_budget);
  return static_cast<int32_t>(std::ceil(std::max(a, b)));
}

int64_t m_max(int64_t n1, int64_t n3) {
  const int64_t q = (n1 * n3) / 16;
  int64_t r = static_cast<int64_t>(std::sqrt(static_cast<double>(q)));
  while (r * r > q) --r;
  while ((r + 1) * (r + 1) <= q) ++r;
  return std::max<int64_t>(16, r);
}

// Eq. 3 noise over rms(C): c_f 2^-24 sqrt(n1 n3 n2) (n2/8192)^e / m.
double law_sigma_over_rms(int64_t n1, int64_t n2, int64_t n3, int64_t m, fpsketch_dtype dt,
                          const fpsketch_params& p) {
  return law_cf(dt, p) * std::ldexp(1.0, -24) *
         std::sqrt(static_cast<double>(n1) * static_cast<double>(n3) * static_cast<double>(n2)) *
         std::pow(static_cast<double>(n2) / 8192.0, p.law_n2_exp) / static_cast<double>(m);
}

int64_t m_start(int64_t n1, int64_t n2, int64_t n3, fpsketch_dtype dt, const fpsketch_params& p) {
  // Eq. 4 at delta = rms(C) with target B* (rms(C) cancels), then Eq. 5.
  const double v = static_cast<double>(std::max(n1, n3)) / p.b_star * law_cf(dt, p) *
                   std::ldexp(1.0, -24) *
                   std::sqrt(static_cast<double>(n1) * static_cast<double>(n3) *
                             static_cast<double>(n2)) *
                   std::pow(static_cast<double>(n2) / 8192.0, p.law_n2_exp);
  const int64_t mnum = static_cast<int64_t>(std::ceil(v));
  const int64_t mc = m_comb(p);
  return std::min(std::max<int64_t>({mc, mnum, 16}), std::max<int64_t>(mc, m_max(n1, n3)));
}

// Largest m with 4 (3 m^2 + 6 m n2) bytes within 2 GiB.
int64_t m_mem(int64_t n2) {
  auto fits = [n2](int64_t m) { return 4 * (3 * m * m + 6 * m * n2) <= (int64_t{1} << 31); };
  int64_t lo = 0, hi = 1;
  while (fits(hi)) hi *= 2;
  while (hi - lo > 1) {
    const int64_t mid = (lo + hi) / 2;
    (fits(mid) ? lo : hi) = mid;
  }
  return lo;
}

bool positive_finite(double x) { return std::isfinite(x) && x > 0.0; }

// ceil(x) for x >= 0 as an integer, saturated at hi (x may be huge or +inf: a probe estimate
// taken on a C with out-of-range entries can be of the order of those entries).
int64_t ceil_sat(double x, int64_t hi) {
  const double c = std::ceil(x);
  return c < static_cast<double>(hi) ? static_cast<int64_t>(c) : hi;
}

// r_B of Sec. III-G, saturated far above any radius the plan can use.
int64_t radius_rule(double B) {
  if (B <= 0.05) return 0;
  return std::max<int64_t>(2, ceil_sat(2.5 * B, int64_t{1} << 40));
}

struct PlanOut {
  int32_t m_loc, r, fallback;
  double B;
};

PlanOut plan_localize(int64_t n1, int64_t n2, int64_t n3, fpsketch_dtype dt, int32_t m,
                      double sigma, double rms, const fpsketch_params& p) {
  const double mx = static_cast<double>(std::max(n1, n3));
  PlanOut o{};
  o.fallback = !(positive_finite(sigma) && positive_finite(rms));
  o.B = o.fallback ? mx * law_sigma_over_rms(n1, n2, n3, m, dt, p) / p.rho_min
                   : mx * sigma / (p.rho_min * rms);
  const int64_t rb = radius_rule(o.B);
  if (rb <= p.r_star) {
    o.m_loc = m;
    o.r = static_cast<int32_t>(rb);
    return o;
  }
  const int64_t cap = std::min(m_max(n1, n3), m_mem(n2));
  const int64_t need = ceil_sat(static_cast<double>(m) * static_cast<double>(rb) /
                                    static_cast<double>(p.r_star), cap + 16);
  const int64_t grown = 16 * ((need + 15) / 16);
  const int64_t mloc = std::max<int64_t>(m, std::min(grown, cap));
  o.m_loc = static_cast<int32_t>(mloc);
  const double b2 = o.B * static_cast<double>(m) / static_cast<double>(mloc);
  o.r = b2 <= 0.05 ? 0
                   : static_cast<int32_t>(std::min<int64_t>(
                         p.r_max, std::max<int64_t>(2, ceil_sat(2.5 * b2, p.r_max))));
  return o;
}

void recalibrate(int64_t n1, int64_t n3, int32_t m, double sigma_bar, double rms,
                 const fpsketch_params& p, int32_t* m_new, int32_t* rebuild) {
  *m_new = m;
  *rebuild = 0;
  if (!(positive_finite(sigma_bar) && positive_finite(rms))) return;
  const double b1 = static_cast<double>(std::max(n1, n3)) * sigma_bar / rms;
  const int64_t want = ceil_sat(static_cast<double>(m) * b1 / p.b_star, m_max(n1, n3));
  const int64_t mp = std::max<int64_t>({m_comb(p), 16, std::min(want, m_max(n1, n3))});
  if (static_cast<double>(mp) < m / 1.25 || static_cast<double>(mp) > 1.25 * m) {
    *m_new = static_cast<int32_t>(mp);
    *rebuild = 1;
  }
}

// Median with the even-count convention (mean of the two middle order statistics).
double median_of(std::vector<double> v) {
  const size_t n = v.size();
  if (n == 0) return std::nan("");
  const size_t h = n / 2;
  std::nth_element(v.begin(), v.begin() + h, v.end());
  const double hi = v[h];
  if (n % 2) return hi;
  const double lo = *std::max_element(v.begin(), v.begin() + h);
  return 0.5 * (lo + hi);
}

double rms_hat_from_samples(const float* s, int64_t count) {
  std::vector<double> a;
  a.reserve(static_cast<size_t>(count));
  for (int64_t t = 0; t < count; ++t) {
    const double x = s[t];
    if (std::isfinite(x)) a.push_back(std::fabs(x));
  }
  if (a.empty()) return std::nan("");
  const double clip = 64.0 * median_of(a);
  double acc = 0.0;
  for (double x : a) {
    const double c = std::min(x, clip);
    acc += c * c;
  }
  return std::sqrt(acc / static_cast<double>(a.size()));
}

// ------------------------------------------------------------------------------------------
// Tables of one hash round at one m.

struct HostRound {
  int m = 0;
  int cap = 0;
  bool mom = false;
  std::vector<int32_t> h1, h2;
  std::vector<int8_t> v1, v2;
  std::vector<int32_t> perm, coff, boff;
  std::vector<uint16_t> ctab, btab;
  std::vector<uint8_t> bsign;
  // B passed transposed: the column lists of each bucket (j | (v2 < 0) << 31, ascending,
  // padded to cap2 with -1), natural bucket order (the C grid's column order)
  int cap2 = 0;
  std::vector<int32_t> perm2;
};

// Bucket segments are padded to a multiple of 8 for m <= 256 (the kernels then fold 8 list
// entries per step); above that the lists are unpadded, except the probe's B chunks up to
// m = 512 (the 4-row B work-groups fold whole groups of 8).
int table_pad(int m) { return m <= 256 ? 8 : 1; }
int btab_pad(int m, bool mom) { return !mom && m <= 512 ? 8 : table_pad(m); }

int64_t table_stride(int m, int64_t W, int pad) {
  const int64_t s = W + static_cast<int64_t>(pad - 1) * m;
  return (s + 7) / 8 * 8;
}

// Staged LDS slot of column offset cc in a B chunk of W columns (W: the zero sentinel slot):
// column-block major, slot (cc mod 8) (W / 8) + cc / 8, so the thread that loads columns
// 8g .. 8g + 7 stores them at one base address plus constant offsets, and the 64 lanes of a wave
// store to consecutive slots.
int64_t b_slot(int64_t cc, int64_t W) { return cc < W ? (cc & 7) * (W / 8) + (cc >> 3) : W; }

// Column tiles of width W sorted by bucket (stable in column order); segment starts per tile,
// segments padded with the sentinel W.  Entry format: 0 = offset | (v2 < 0) << 15 (C tiles),
// 1 = offset (B chunks with moments), 2 = staged slot (B chunks of the probe).
void build_col_tables(const std::vector<int32_t>& h2, const std::vector<int8_t>& v2, int m,
                      int64_t W, int format, int pad, std::vector<uint16_t>& tab,
                      std::vector<int32_t>& off) {
  const int64_t n3 = static_cast<int64_t>(h2.size());
  const int64_t T = (n3 + W - 1) / W;
  const int64_t stride = table_stride(m, W, pad);
  tab.assign(static_cast<size_t>(T * stride), static_cast<uint16_t>(W));
  off.assign(static_cast<size_t>(T * (m + 1)), 0);
  std::vector<int32_t> cnt(static_cast<size_t>(m) + 1), pos(static_cast<size_t>(m));
  for (int64_t t = 0; t < T; ++t) {
    const int64_t j0 = t * W, j1 = std::min(n3, j0 + W);
    std::fill(cnt.begin(), cnt.end(), 0);
    for (int64_t j = j0; j < j1; ++j) cnt[static_cast<size_t>(h2[j]) + 1]++;
    int32_t* o = off.data() + t * (m + 1);
    o[0] = 0;
    for (int b = 0; b < m; ++b) {
      const int32_t padded = (cnt[b + 1] + pad - 1) / pad * pad;
      o[b + 1] = o[b] + padded;
      pos[b] = o[b];
    }
    for (int64_t j = j0; j < j1; ++j) {
      const int32_t p = pos[h2[j]]++;
      const int64_t cc = j - j0;
      uint16_t e;
      if (format == 0) {
        e = static_cast<uint16_t>(cc | (v2[j] < 0 ? 0x8000 : 0));
      } else if (format == 1) {
        e = static_cast<uint16_t>(cc);
      } else {
        e = static_cast<uint16_t>(b_slot(cc, W));
      }
      tab[static_cast<size_t>(t * stride + p)] = e;
    }
  }
}

// size_order: the row lists are stored largest bucket first (list slot a holds the a-th largest
// bucket), so that the row-bucket work-groups, dispatched in list order, start with the longest.
// The sketch rows then come out in that order; only the probe, whose statistics do not depend
// on the numbering of the buckets, uses it.
void build_round(uint64_t seed, int round, int64_t n1, int64_t n3, int m, int64_t cwb, bool mom,
                 bool transb, HostRound& R, bool size_order = false) {
  R.m = m;
  R.mom = mom;
  R.h1.resize(n1);
  R.v1.resize(n1);
  R.h2.resize(n3);
  R.v2.resize(n3);
  hash_side(seed, round, 0, n1, m, R.h1.data(), R.v1.data());
  hash_side(seed, round, 1, n3, m, R.h2.data(), R.v2.data());
  // rows of each bucket, ascending, padded to the largest bucket with -1
  std::vector<int32_t> cnt(static_cast<size_t>(m), 0);
  for (int64_t i = 0; i < n1; ++i) cnt[R.h1[i]]++;
  R.cap = std::max(1, *std::max_element(cnt.begin(), cnt.end()));
  std::vector<int32_t> slot(static_cast<size_t>(m));
  for (int b = 0; b < m; ++b) slot[b] = b;
  if (size_order) {
    std::vector<int32_t> byz(static_cast<size_t>(m));
    for (int b = 0; b < m; ++b) byz[b] = b;
    std::stable_sort(byz.begin(), byz.end(), [&](int32_t x, int32_t y) { return cnt[x] > cnt[y]; });
    for (int a = 0; a < m; ++a) slot[byz[a]] = a;
  }
  R.perm.assign(static_cast<size_t>(m) * R.cap, -1);
  std::fill(cnt.begin(), cnt.end(), 0);
  for (int64_t i = 0; i < n1; ++i) {
    const int b = R.h1[i];
    R.perm[static_cast<size_t>(slot[b]) * R.cap + cnt[b]++] =
        static_cast<int32_t>(static_cast<uint32_t>(i) | (R.v1[i] < 0 ? 0x80000000u : 0u));
  }
  build_col_tables(R.h2, R.v2, m, kColTile, 0, table_pad(m), R.ctab, R.coff);
  build_col_tables(R.h2, R.v2, m, cwb, mom ? 1 : 2, btab_pad(m, mom), R.btab, R.boff);
  if (transb) {
    std::vector<int32_t> c2(static_cast<size_t>(m), 0);
    for (int64_t j = 0; j < n3; ++j) c2[R.h2[j]]++;
    R.cap2 = std::max(1, *std::max_element(c2.begin(), c2.end()));
    R.perm2.assign(static_cast<size_t>(m) * R.cap2, -1);
    std::fill(c2.begin(), c2.end(), 0);
    for (int64_t j = 0; j < n3; ++j) {
      const int b = R.h2[j];
      R.perm2[static_cast<size_t>(b) * R.cap2 + c2[b]++] =
          static_cast<int32_t>(static_cast<uint32_t>(j) | (R.v2[j] < 0 ? 0x80000000u : 0u));
    }
  } else {
    R.cap2 = 0;
    R.perm2.clear();
  }
  // column signs as bits, padded to whole B chunks
  const int64_t TB = (n3 + cwb - 1) / cwb;
  R.bsign.assign(static_cast<size_t>(TB * cwb / 8), 0);
  for (int64_t j = 0; j < n3; ++j) {
    if (R.v2[j] < 0) R.bsign[static_cast<size_t>(j / 8)] |= static_cast<uint8_t>(1u << (j % 8));
  }
}

// ------------------------------------------------------------------------------------------
// Device memory helpers.

struct DevBuf {
  void* p = nullptr;
  size_t bytes = 0;
};

fpsketch_status dev_alloc(DevBuf& b, size_t bytes) {
  if (b.p != nullptr && b.bytes >= bytes) return FPSK_OK;
  if (b.p != nullptr) {
    (void)hipFree(b.p);
    b.p = nullptr;
    b.bytes = 0;
  }
  if (bytes == 0) return FPSK_OK;
  FPSK_HIP(hipMalloc(&b.p, bytes));
  b.bytes = bytes;
  return FPSK_OK;
}

// As dev_alloc, and a new allocation is zero-filled.
fpsketch_status dev_alloc_zero(DevBuf& b, size_t bytes) {
  if (b.p != nullptr && b.bytes >= bytes) return FPSK_OK;
  FPSK_TRY(dev_alloc(b, bytes));
  if (bytes != 0) FPSK_HIP(hipMemset(b.p, 0, bytes));
  return FPSK_OK;
}

void dev_free(DevBuf& b) {
  if (b.p != nullptr) (void)hipFree(b.p);
  b.p = nullptr;
  b.bytes = 0;
}

template <typename T>
T* as(DevBuf& b) {
  return static_cast<T*>(b.p);
}

// Work decomposition of one sketch pass at bucket count m.
struct Decomp {
  int m = 0;
  int TA = 0, nA = 0;
  int rb = 8, g = 1, ng = 1, cwb = 2048, TB = 0, nB = 0;
  int TC = 0, npc = 1, tg = 1, nC = 0;
  int ctab_stride = 0, btab_stride = 0, tab_off = 0;
  int ts = 32, nt = 1, NS = 1, ksl = 0;
  bool kw = false;             // product tiles whose k-range the 4 waves split
  size_t lds_stream = 0;
  int kact = 0;                // k-range of the factors: n2 rounded up to a multiple of 4
  int ldp = 0;                 // row stride of the factors (kact padded; see decompose)
  // probe block product (nX > 0): work-groups of xb x xb outputs over xns k-slices
  int xb = 0, xnb = 0, xns = 0, nX = 0;
  int xsr = 1, xsc = 1, xnstc = 1, xslots = 0;   // supertiles of blocks (XCD-local sets)
  // B work-groups of 1 or 2 rows write Q k-major (n2 x m), then a transpose forms Q
  bool qk = false;
  bool wt_c = false;                  // C work-groups of one tile per wave
  bool wt_a = false, wt_w = false;   // row-bucket work-groups of four tiles (small buckets)
};

// pipe: the deferred probe's decomposition, whose output blocks stay at most 3 x 3 (the
// pipelined launch holds the block product within the stream pass's registers).
Decomp decompose(int64_t n1, int64_t n2, int64_t n3, int m, bool mom, bool transb,
                 bool pipe = false) {
  (void)n1;
  Decomp d;
  d.m = m;
  d.TA = static_cast<int>((n2 + kColTile - 1) / kColTile);
  // buckets of at most about 16 rows: one wave per column tile, four tiles per work-group; also
  // up to 32 rows when the one-tile work-groups would number 8192 or more, each too short for
  // its dispatch (16384^3 FP16, m = 697: 22,304 work-groups of 3.8 us; four tiles each, the
  // pass took 470 -> 445 us; at 2048 x 8192 x 8192, m = 100, with 1600 it was 0.4 us slower)
  d.wt_a = n1 <= 16 * static_cast<int64_t>(m) ||
           (n1 <= 32 * static_cast<int64_t>(m) && static_cast<int64_t>(m) * d.TA >= 8192);
  d.wt_w = transb && n3 <= 16 * static_cast<int64_t>(m);
  const int tq = (d.TA + 3) / 4;
  d.nA = m * (d.wt_a ? tq : d.TA);
  // the probe at m <= 512 (B as stored): 4-row B work-groups over whole 4096-column chunks,
  // G = 1 or 2 buckets per thread in their (and the C work-groups') per-bucket sums
  const bool probe4 = !mom && !transb && m <= 512;
  if (probe4) {
    d.rb = 4, d.g = m <= 256 ? 1 : 2, d.ng = 1;
  } else if (m <= 64) {
    d.rb = 8, d.g = 1, d.ng = 4;
  } else if (m <= 128) {
    d.rb = 8, d.g = 1, d.ng = 2;
  } else if (m <= 256) {
    d.rb = 8, d.g = 1;
  } else if (m <= 512) {
    d.rb = 8, d.g = 2;
  } else if (m <= 1024) {
    d.rb = 4, d.g = 4;
  } else if (m <= 2048) {
    d.rb = 2, d.g = 8;
  } else {
    d.rb = 1, d.g = 16;
  }
  d.cwb = fpsk::kBChunkHalfs / d.rb;
  d.TB = static_cast<int>((n3 + d.cwb - 1) / d.cwb);
  d.nB = static_cast<int>((n2 + d.rb - 1) / d.rb);
  // B passed transposed: row-bucket work-groups over the rows of W = B^T, as many as A's
  if (transb) d.nB = m * (d.wt_w ? tq : d.TA);
  d.qk = !transb && d.rb < 4;
  d.TC = static_cast<int>((n3 + kColTile - 1) / kColTile);
  int npc = static_cast<int>((1024 + m - 1) / m);
  npc = std::max(1, std::min(npc, d.TC));
  d.tg = (d.TC + npc - 1) / npc;
  d.npc = (d.TC + d.tg - 1) / d.tg;
  d.nC = m * d.npc;
  // C work-groups with one tile per wave where buckets hold few rows: the four waves of
  // the one-tile form each hold a handful of rows per tile and meet at three barriers per
  // tile (16384^3 FP16, m = 698: stream pass 445.8 -> 426.7 us; 2048 x 4096 x 12288 at
  // m = 400: 82.5 -> 59.2 us).  The 512-entry tile lists of m > 256 let one 16-byte load per
  // thread stage all four; m <= 1024 keeps the fold's segment starts (8 G) in registers.
  d.wt_c = m > 256 && m <= 1024 && n1 <= 32 * static_cast<int64_t>(m) && d.tg >= 4;
  // The same at 48 < m <= 192 for the probe with B as stored and whole 16-byte rows (the
  // instance with 4-row B work-groups; its unaligned form would spill): column groups of 4 tiles
  // instead of about 1024 / m groups, the padded 8-entry lists staged after the column sums
  // (2048 x 4096 x 12288 at m = 80: stream pass 43.3 -> 41.5 us; 2048 x 8192 x 8192 at m = 64:
  // 45.3 -> 43.8 us).
  if (!mom && !transb && m > 48 && m <= 192 && n1 <= 32 * static_cast<int64_t>(m) &&
      d.TC >= 4 && n2 % 8 == 0 && n3 % 8 == 0) {
    d.wt_c = true;
    d.npc = (d.TC + 3) / 4;
    d.tg = (d.TC + d.npc - 1) / d.npc;
    d.nC = m * d.npc;
  }
  // Bucket-space product on the matrix cores, tiles of ts x ts outputs over NS k-slices.
  // Without moments: 16 x 16 tiles whose k-range the 4 waves split, while there are fewer than
  // 256 of them (slices for about 2048 waves); else 64 x 64 tiles of four 32 x 32 wave quadrants.
  // With moments: four 16 x 16 quadrants (32 x 32 tiles) up to m = 2048 (the 64 x 64 tile's
  // three accumulator sets leave one wave per SIMD: 1.1 to 1.8x slower at m = 256 to 1024), then
  // 64 x 64 (its operand reuse wins at m = 4096).  Without the split, slices for at most 1024
  // work-groups.  A wave takes k in steps of 32 or 16; at most 32 slices.
  if (!mom) {
    const int t16 = (m + 15) / 16;
    d.kw = t16 * t16 < 256;
    d.ts = d.kw ? 16 : 64;
  } else {
    d.kw = false;
    d.ts = m <= 2048 ? 32 : 64;
  }
  d.nt = (m + d.ts - 1) / d.ts;
  const int tiles = d.nt * d.nt;
  // k per work-group slice: whole steps of the waves' k-loops (32 k per step for S alone on the
  // quadrant tiles, else 16; with the k-range split over the 4 waves, four of those)
  const int kstep = d.kw ? 64 : (mom ? 16 : 32);
  // k-slices rounded down, so that tiles x slices stays within the work-groups one round of the
  // chip holds (4 per CU for the 64 x 64 tiles): rounding up left a second round of a few
  // work-groups (m = 698: 121 tiles x 9 slices = 1089; now 8 slices, 373 -> 337 us)
  int ns = (d.kw ? 512 : 1024) / tiles;
  ns = std::max(1, std::min<int>({ns, 32, static_cast<int>((n2 + kstep - 1) / kstep)}));
  int64_t ksl = (n2 + ns - 1) / ns;
  ksl = (ksl + kstep - 1) / kstep * kstep;
  d.ksl = static_cast<int>(ksl);
  d.NS = static_cast<int>((n2 + ksl - 1) / ksl);
  // dynamic LDS of the stream kernel: a data area (A/C combine and column sums, or the staged
  // B chunk plus its zero column), then the staged sorted column list
  d.ctab_stride = static_cast<int>(table_stride(m, kColTile, table_pad(m)));
  d.btab_stride = static_cast<int>(table_stride(m, d.cwb, btab_pad(m, mom)));
  const size_t comb = (mom ? 4096 : 2048) * sizeof(double);
  const size_t cs = (mom ? 1040 : 520) * sizeof(double);
  const size_t bdata = (static_cast<size_t>(d.cwb) * d.rb + d.rb) * sizeof(uint16_t);
  // one-tile-per-wave C work-groups: four tiles' column sums (and weighted sums), and at
  // m <= 256 the four padded tile lists
  const size_t wtc =
      d.wt_c ? (mom ? 8 : 4) * 520 * sizeof(double) +
                   (m <= 256 ? 4 * static_cast<size_t>(d.ctab_stride) * sizeof(uint16_t) : 0)
             : 0;
  const size_t data = (std::max({comb + cs, bdata, wtc}) + 15) / 16 * 16;
  d.tab_off = static_cast<int>(data);
  // (the probe's B group fold, 8-row work-groups up to m = 256, stages the m + 1 segment
  // starts after the column list; at larger m they would take up to 16 KiB per work-group)
  const bool group_fold = !mom && d.rb == 8 && d.g == 1;
  d.lds_stream = data + static_cast<size_t>(std::max(d.ctab_stride, d.btab_stride)) *
                            sizeof(uint16_t) +
                 (group_fold ? (static_cast<size_t>(m) + 1) * sizeof(int32_t) : 0);
  if (probe4) {
    // the 4-row B work-groups read their sorted lists from global memory and stage only the
    // m + 1 segment starts after the data (the C tiles' lists use the same area)
    d.lds_stream = data + std::max<size_t>(static_cast<size_t>(d.ctab_stride) * sizeof(uint16_t),
                                           (static_cast<size_t>(m) + 1) * sizeof(int32_t));
  }
  if (d.wt_c) {
    // the four staged 512-entry tile lists of the one-tile-per-wave C work-groups
    d.lds_stream = std::max(d.lds_stream, data + 4 * 512 * sizeof(uint16_t));
  }
  d.kact = static_cast<int>((n2 + 3) / 4 * 4);
  // Factor rows sit 64 floats past a multiple of 1024 apart (an odd multiple of 256 bytes), so
  // that the 16 rows one matrix-core load instruction touches at the same k fall on 16
  // different L2 channels rather than one.
  d.ldp = static_cast<int>((n2 + 1023) / 1024 * 1024 + 64);
  // The probe's product for m <= 64 (at most a 16 x 16 grid of output blocks) and
  // n2 <= kMaxXSlices * kXSlice: block products over whole k-slices, then one deciding
  // work-group.
  const int xns = static_cast<int>((d.kact + fpsk::kXSlice - 1) / fpsk::kXSlice);
  if (!mom && m <= 64 && xns <= fpsk::kMaxXSlices) {
    d.xb = (m + 15) / 16;
    if (pipe && d.xb > 3) d.xb = 3;
    d.xnb = (m + d.xb - 1) / d.xb;
    d.xns = xns;
    // The 8 XCDs take launch indices round-robin, and the kernel maps index i to slot
    // (i mod 8) nX / 8 + i / 8: each XCD runs a contiguous range of slots.  Slots run over
    // supertiles of xsr x xsc output blocks within a slice, so one XCD's blocks form a compact
    // rectangle that shares factor rows in that XCD's L2.
    d.xsc = std::min(8, d.xnb);
    const int per = (d.xnb * d.xnb + 7) / 8;
    d.xsr = std::max(1, std::min(d.xnb, (per + d.xsc - 1) / d.xsc));
    d.xnstc = (d.xnb + d.xsc - 1) / d.xsc;
    d.xslots = ((d.xnb + d.xsr - 1) / d.xsr) * d.xsr * d.xnstc * d.xsc;
    d.nX = (d.xns * d.xslots + 7) / 8 * 8;
  }
  return d;
}

struct DevRound {
  int m = 0;
  int cap = 0;
  bool mom = false;
  int64_t cwb = 0;
  int cap2 = 0;
  DevBuf perm, ctab, coff, btab, boff, bsign, perm2;
};

fpsketch_status upload_round(const HostRound& R, int64_t cwb, DevRound& D, hipStream_t st) {
  D.m = R.m;
  D.cap = R.cap;
  D.mom = R.mom;
  D.cwb = cwb;
  auto up = [st](DevBuf& b, const void* src, size_t bytes) -> fpsketch_status {
    FPSK_TRY(dev_alloc(b, bytes));
    if (bytes) FPSK_HIP(hipMemcpyAsync(b.p, src, bytes, hipMemcpyHostToDevice, st));
    return FPSK_OK;
  };
  FPSK_TRY(up(D.perm, R.perm.data(), R.perm.size() * 4));
  FPSK_TRY(up(D.bsign, R.bsign.data(), R.bsign.size()));
  FPSK_TRY(up(D.ctab, R.ctab.data(), R.ctab.size() * 2));
  FPSK_TRY(up(D.coff, R.coff.data(), R.coff.size() * 4));
  FPSK_TRY(up(D.btab, R.btab.data(), R.btab.size() * 2));
  FPSK_TRY(up(D.boff, R.boff.data(), R.boff.size() * 4));
  D.cap2 = R.cap2;
  if (!R.perm2.empty()) FPSK_TRY(up(D.perm2, R.perm2.data(), R.perm2.size() * 4));
  // host vectors must outlive the asynchronous copies
  FPSK_HIP(hipStreamSynchronize(st));
  return FPSK_OK;
}

void free_round(DevRound& D) {
  dev_free(D.perm);
  dev_free(D.bsign);
  dev_free(D.ctab);
  dev_free(D.coff);
  dev_free(D.btab);
  dev_free(D.boff);
  dev_free(D.perm2);
}

struct Workspace {
  Decomp d;
  // with moments: the product decomposition of S alone (localize rounds form R and T only at
  // the selected buckets)
  Decomp ds;
  bool mom = false;
  DevBuf P, Pw, Q, Qw, partS, partR, partT, scratch, S, R, T, maxpart, tilestat;
  DevBuf xpart;                // probe block-product partials
  DevBuf Qk, Qwk;              // k-major B-side rows (qk passes), transposed into Q, Qw
};

fpsketch_status ensure_workspace(Workspace& W, int64_t n1, int64_t n2, int64_t n3, int m,
                                 bool mom, bool transb, bool pipe = false) {
  const Decomp d = decompose(n1, n2, n3, m, mom, transb, pipe);
  W.d = d;
  W.mom = mom;
  // factor rows are ldp long; the padding past n2 is never written and stays zero
  const size_t fm = static_cast<size_t>(m) * static_cast<size_t>(d.ldp) * sizeof(float);
  const size_t mm = static_cast<size_t>(m) * static_cast<size_t>(m) * sizeof(double);
  FPSK_TRY(dev_alloc_zero(W.P, fm));
  FPSK_TRY(dev_alloc_zero(W.Q, fm));
  FPSK_TRY(dev_alloc(W.partS, mm * d.npc));
  FPSK_TRY(dev_alloc(W.S, mm));
  if (mom) {
    FPSK_TRY(dev_alloc_zero(W.Pw, fm));
    FPSK_TRY(dev_alloc_zero(W.Qw, fm));
    FPSK_TRY(dev_alloc(W.partR, mm * d.npc));
    FPSK_TRY(dev_alloc(W.partT, mm * d.npc));
    FPSK_TRY(dev_alloc(W.R, mm));
    FPSK_TRY(dev_alloc(W.T, mm));
  }
  W.ds = mom ? decompose(n1, n2, n3, m, false, transb) : d;
  const int tiles = std::max(d.nt * d.nt, W.ds.nt * W.ds.nt);
  // slice partials (also used with a single slice when the probe's decision is fused)
  const size_t sc = std::max(
      static_cast<size_t>(d.NS) * d.nt * d.nt * d.ts * d.ts * (mom ? 3 : 1),
      static_cast<size_t>(W.ds.NS) * W.ds.nt * W.ds.nt * W.ds.ts * W.ds.ts) * sizeof(double);
  FPSK_TRY(dev_alloc(W.scratch, sc));
  FPSK_TRY(dev_alloc(W.maxpart, static_cast<size_t>(d.nA + d.nB) * sizeof(float)));
  FPSK_TRY(dev_alloc(W.tilestat, static_cast<size_t>(tiles) * 4 * sizeof(double)));
  if (d.nX > 0) FPSK_TRY(dev_alloc(W.xpart, static_cast<size_t>(d.xns) * mm));
  if (d.qk) {
    const size_t qk = static_cast<size_t>(n2) * static_cast<size_t>(m) * sizeof(float);
    FPSK_TRY(dev_alloc(W.Qk, qk));
    if (mom) FPSK_TRY(dev_alloc(W.Qwk, qk));
  }
  return FPSK_OK;
}

void free_workspace(Workspace& W) {
  for (DevBuf* b : {&W.P, &W.Pw, &W.Q, &W.Qw, &W.partS, &W.partR, &W.partT, &W.scratch, &W.S,
                    &W.R, &W.T, &W.maxpart, &W.tilestat, &W.xpart, &W.Qk, &W.Qwk}) {
    dev_free(*b);
  }
}

}  // namespace

// ------------------------------------------------------------------------------------------
// Scratch of fpsketch_probe_noalloc: one array per GPU that runs the library, held until the
// process ends.  In host code `scratch` names a host-side stand-in, not device memory: kernels
// and copies take the device address that hipGetSymbolAddress gives on each device, resolved
// once per device (with that device current) when the first context on it is created.

namespace {

constexpr size_t kScratchBytes = size_t{16} << 20;    // 16 MiB
__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
std::unordered_map<int, unsigned char*> g_scratch_addr;   // device -> address of its scratch

fpsketch_status scratch_address(int dev, unsigned char** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  auto it = g_scratch_addr.find(dev);
  if (it == g_scratch_addr.end()) {
    void* p = nullptr;
    FPSK_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    it = g_scratch_addr.emplace(dev, static_cast<unsigned char*>(p)).first;
  }
  *out = it->second;
  return FPSK_OK;
}

}  // namespace

// ------------------------------------------------------------------------------------------
// Context.

struct fpsketch_ctx {
  int64_t n1 = 0, n2 = 0, n3 = 0;
  fpsketch_dtype dt = FPSK_BF16;
  bool transb = false;        // B passed as W = B^T (p.b_layout == 1)
  fpsketch_params p{};
  int device = 0;
  int m = 0;
  double inv_l1 = 1.0, inv_l3 = 1.0;
  int64_t L1 = 1, L3 = 1;
  // probe: hash round 0 of the context seed at m
  DevRound probe_round;
  Workspace probe_ws;
  DevBuf stats;       // 8 doubles
  DevBuf zero;        // 64 bytes of zeros
  DevBuf sigma_acc;   // 2 doubles
  // localize / diagnostic workspaces
  DevRound aux_round;
  Workspace aux_ws;
  DevBuf scan_counts, scan_rows, scan_base, scan_out, samples, patch_rowptr, patch_col,
      patch_val, rc_coords, rc_gamma, rc_abs, rc_c;
  // localize rounds on the device: selection state and histogram, peel list, candidates
  DevBuf sel_state, sel_hist, peel_list, cands, cand_count;
  // the selected buckets of a round and their moment sketches (R then T)
  DevBuf mo_list, mo_rt;
  // apply step: the record list and the re-probe's statistics and scratch noise sum
  DevBuf apply_list, reprobe_stats, reprobe_acc;
  // the B-side cache of the probe: Q = (B H2^T)^T for the probe's round at m = qcache_m
  // (0: nothing cached) and the per-work-group max |B|
  DevBuf qcache, maxb_cache;
  int qcache_m = 0;
  // deferred probes (m <= 64): three workspace sets in rotation; the previous call, whose block
  // products are still to run, and the one before it, whose decision is; the stream their
  // launches go to
  Workspace pipe_ws[3];
  int pipe_next = 0;
  bool pipe_has_prod = false, pipe_has_dec = false;
  fpsk::ProductArgs pipe_prod{}, pipe_dec{};
  int pipe_nprod = 0, pipe_xb = 1;
  hipStream_t pipe_stream = nullptr;
  fpsketch_plan_info last_plan{};
  unsigned char* scratch_dev = nullptr;   // this device's scratch (fpsketch_probe_noalloc)

  // optional per-probe events: start and end of the stream kernel, of the product dispatches
  bool timing = false;
  std::vector<hipEvent_t> events;
  size_t events_used = 0;
};

namespace {

bool valid_half(fpsketch_dtype d) { return d == FPSK_F16 || d == FPSK_BF16; }

fpsketch_status check_params(const fpsketch_params& p) {
  if (p.m < 0 || p.rounds < 1 || p.r_star < 0 || p.r_max < 0 || p.s_budget < 1 ||
      p.delta_rc < 1 || p.k_cap < 0 || !(p.rho_min > 0) || !(p.mu > 0) || !(p.c_valid > 0) ||
      !(p.b_star > 0) || !(p.c_coll > 0) || (p.b_layout != 0 && p.b_layout != 1) ||
      !(std::isfinite(p.law_cf_bf16) && p.law_cf_bf16 > 0) ||
      !(std::isfinite(p.law_cf_fp16) && p.law_cf_fp16 > 0) || !std::isfinite(p.law_n2_exp)) {
    return fail(FPSK_EINVAL, "parameter out of range");
  }
  return FPSK_OK;
}

int32_t cap_K(const fpsketch_params& p) {
  return p.k_cap > 0 ? p.k_cap : std::max(64, 8 * p.s_budget);
}

fpsketch_status set_device(const fpsketch_ctx* c) {
  FPSK_HIP(hipSetDevice(c->device));
  return FPSK_OK;
}

// How a pass treats the B side: streamed, only filled into the context's cache (no product),
// or taken from that cache (A and C streamed).
enum class BSide { kStream, kFillCache, kUseCache };

// Arguments of one sketch pass (stream + product) over workspace W.
fpsketch_status pass_args(fpsketch_ctx* c, const DevRound& R, Workspace& W, const void* A,
                          const void* B, const float* Cm, bool mom, int mode, int32_t* d_dirty,
                          const int32_t* prow, const int32_t* pcol, const float* pval,
                          double* stats_out, double* sigma_acc_out, BSide bside,
                          fpsk::StreamArgs& s, fpsk::ProductArgs& a) {
  const Decomp& d = W.d;
  s = fpsk::StreamArgs{};
  s.A = static_cast<const uint16_t*>(A);
  s.B = static_cast<const uint16_t*>(B);
  s.C = Cm;
  s.n1 = c->n1;
  s.n2 = c->n2;
  s.n3 = c->n3;
  s.m = d.m;
  s.perm = static_cast<const int32_t*>(R.perm.p);
  s.cap = R.cap;
  s.transb = c->transb ? 1 : 0;
  s.perm2 = static_cast<const int32_t*>(R.perm2.p);
  s.cap2 = R.cap2;
  s.bsign = static_cast<const uint8_t*>(R.bsign.p);
  s.ctab = static_cast<const uint16_t*>(R.ctab.p);
  s.coff = static_cast<const int32_t*>(R.coff.p);
  s.btab = static_cast<const uint16_t*>(R.btab.p);
  s.boff = static_cast<const int32_t*>(R.boff.p);
  s.cwb = d.cwb;
  s.ctab_stride = d.ctab_stride;
  s.btab_stride = d.btab_stride;
  s.tab_off = d.tab_off;
  s.P = as<float>(W.P);
  s.Pw = mom ? as<float>(W.Pw) : nullptr;
  s.Q = as<float>(W.Q);
  s.Qw = mom ? as<float>(W.Qw) : nullptr;
  s.partS = as<double>(W.partS);
  s.partR = mom ? as<double>(W.partR) : nullptr;
  s.partT = mom ? as<double>(W.partT) : nullptr;
  s.maxpart = as<float>(W.maxpart);
  s.patch_rowptr = prow;
  s.patch_col = pcol;
  s.patch_val = pval;
  s.nA = d.nA;
  s.nB = d.nB;
  s.nC = d.nC;
  {
    const double half_bytes = 2.0 * static_cast<double>(c->n2);
    const double a_wg = half_bytes * static_cast<double>(c->n1) / std::max(1, d.nA);
    const double b_wg = half_bytes * static_cast<double>(c->n3) / std::max(1, d.nB);
    s.a_first = a_wg >= b_wg ? 1 : 0;
  }
  s.TA = d.TA;
  s.TC = d.TC;
  s.TB = d.TB;
  s.npc = d.npc;
  s.tg = d.tg;
  s.wt_a = d.wt_a ? 1 : 0;
  s.wt_c = d.wt_c ? 1 : 0;
  // (2048 x 8192 x 8192 at m = 64, two whole chunks: stream pass 43.8 -> 42.2 us;
  // 2048 x 4096 x 12288 unchanged; shapes with a partial last chunk measured mixed, within
  // +-0.35 us, so whole chunks only)
  s.rot_b = (c->n3 % d.cwb == 0 && d.TB > 1) ? 1 : 0;
  s.wt_w = d.wt_w ? 1 : 0;
  s.inv_l1 = c->inv_l1;
  s.inv_l3 = c->inv_l3;
  auto aligned16 = [](const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; };
  s.vec_a = (c->n2 % 8 == 0) && aligned16(A);
  // B as stored: rows of n3; transposed: rows of W, n2 long
  s.vec_b = ((c->transb ? c->n2 : c->n3) % 8 == 0) && aligned16(B);
  s.vec_c = (c->n3 % 4 == 0) && aligned16(Cm);
  // the vector path loads whole 8-element groups: every row length must be a multiple of 8
  if (c->n2 % 8 != 0 || c->n3 % 8 != 0) s.vec_a = s.vec_b = s.vec_c = 0;
  s.zero = c->zero.p;
  if (R.cwb != d.cwb || R.m != d.m || R.mom != mom || (c->transb && R.perm2.p == nullptr)) {
    return fail(FPSK_EINVAL, "internal: tables do not match the pass");
  }
  s.ldp = d.ldp;
  if (d.qk) {
    s.Qk = as<float>(W.Qk);
    s.Qwk = mom ? as<float>(W.Qwk) : nullptr;
    s.mq = d.m;
  }
  if (bside == BSide::kFillCache) {
    // B work-groups only, into the cache (Q and the per-work-group max |B|)
    s.nA = 0;
    s.nC = 0;
    s.Q = as<float>(c->qcache);
    s.maxpart = as<float>(c->maxb_cache);
  }
  if (bside == BSide::kUseCache) s.nB = 0;

  a = fpsk::ProductArgs{};
  a.P = s.P;
  a.Pw = s.Pw;
  a.Q = s.Q;
  a.Qw = s.Qw;
  a.partS = s.partS;
  a.partR = s.partR;
  a.partT = s.partT;
  a.S = as<double>(W.S);
  a.R = mom ? as<double>(W.R) : nullptr;
  a.T = mom ? as<double>(W.T) : nullptr;
  a.scratch = as<double>(W.scratch);
  a.tilestat = as<double>(W.tilestat);
  a.m = d.m;
  a.n2 = static_cast<int>(c->n2);
  a.ldp = d.ldp;
  a.kact = d.kact;
  a.nt = d.nt;
  a.ts = d.ts;
  // large m: the clipped sum of the decision spread over one work-group per tile
  a.clip_tiles = (mode == 1 && !mom && d.nX == 0 && d.m >= 192) ? 1 : 0;
  a.NS = d.NS;
  a.ksl = d.ksl;
  a.npc = d.npc;
  a.mode = mode;
  a.maxpart = s.maxpart;
  a.nA = d.nA;
  a.nB = d.nB;
  if (bside == BSide::kUseCache) {
    a.Q = as<float>(c->qcache);
    a.maxpart_b = as<float>(c->maxb_cache);
  }
  // the decision's outputs: the context's probe statistics and noise average unless redirected
  a.stats = stats_out != nullptr ? stats_out : as<double>(c->stats);
  a.d_dirty = d_dirty;
  a.sigma_acc = sigma_acc_out != nullptr ? sigma_acc_out : as<double>(c->sigma_acc);
  a.mu = c->p.mu;
  a.c_valid = c->p.c_valid;
  const double mmd = static_cast<double>(d.m) * d.m;
  a.lim_factor = c->p.mu * std::sqrt(2.0 * std::log(mmd));

  if (mode == 1 && !mom && d.nX > 0) {
    a.nX = d.nX;
    a.xb = d.xb;
    a.xnb = d.xnb;
    a.xns = d.xns;
    a.xsr = d.xsr;
    a.xsc = d.xsc;
    a.xnstc = d.xnstc;
    a.xslots = d.xslots;
    a.xpart = as<double>(W.xpart);
  }
  return FPSK_OK;
}

// One sketch pass (stream + product) on `st`.
fpsketch_status run_pass(fpsketch_ctx* c, const DevRound& R, Workspace& W, const void* A,
                         const void* B, const float* Cm, bool mom, int mode, int32_t* d_dirty,
                         const int32_t* prow, const int32_t* pcol, const float* pval,
                         hipStream_t st, hipEvent_t* ev = nullptr,
                         double* stats_out = nullptr, double* sigma_acc_out = nullptr,
                         BSide bside = BSide::kStream, bool prod_mom = true) {
  const Decomp& d = W.d;
  fpsk::StreamArgs s;
  fpsk::ProductArgs a;
  FPSK_TRY(pass_args(c, R, W, A, B, Cm, mom, mode, d_dirty, prow, pcol, pval, stats_out,
                     sigma_acc_out, bside, s, a));
  if (bside == BSide::kFillCache) {
    FPSK_HIP(fpsk::launch_stream(s, c->dt == FPSK_BF16 ? 1 : 0, false, d.rb, d.g, d.ng,
                                 d.lds_stream, st));
    if (d.qk) {
      FPSK_HIP(fpsk::launch_transpose_q(s.Qk, s.Q, d.m, c->n2, s.mq, d.ldp, st));
    }
    return FPSK_OK;
  }
  // with ev: the dispatches themselves time-stamp ev[0..1] (stream kernel) and ev[2..3]
  // (first product dispatch start to last dispatch end)
  FPSK_HIP(fpsk::launch_stream(s, c->dt == FPSK_BF16 ? 1 : 0, mom, d.rb, d.g, d.ng,
                               d.lds_stream, st, ev ? ev[0] : nullptr, ev ? ev[1] : nullptr));
  if (d.qk && s.nB > 0) {
    FPSK_HIP(fpsk::launch_transpose_q(s.Qk, s.Q, d.m, c->n2, s.mq, d.ldp, st));
    if (mom) FPSK_HIP(fpsk::launch_transpose_q(s.Qwk, s.Qw, d.m, c->n2, s.mq, d.ldp, st));
  }
  if (mom && !prod_mom) {
    // the moment factors stay for launch_moments_at; the product forms S alone
    const Decomp& ds = W.ds;
    a.R = nullptr;
    a.T = nullptr;
    a.nt = ds.nt;
    a.ts = ds.ts;
    a.NS = ds.NS;
    a.ksl = ds.ksl;
    FPSK_HIP(fpsk::launch_product(a, ds.ts, ds.kw, false, st, ev ? ev[2] : nullptr,
                                  ev ? ev[3] : nullptr));
    return FPSK_OK;
  }
  FPSK_HIP(fpsk::launch_product(a, d.ts, d.kw, mom, st, ev ? ev[2] : nullptr,
                                ev ? ev[3] : nullptr));
  return FPSK_OK;
}

// Enqueue what deferred probes still owe (at most two launches of block products and
// decisions) on their stream.  When the caller continues on another stream, wait for them.
fpsketch_status pipe_flush(fpsketch_ctx* c, hipStream_t next_st) {
  const bool had = c->pipe_has_prod || c->pipe_has_dec;
  while (c->pipe_has_prod || c->pipe_has_dec) {
    fpsk::StreamArgs none{};
    const size_t lds = fpsk::probe_pipe_lds(c->pipe_xb);
    FPSK_HIP(fpsk::launch_probe_pipe(none, c->pipe_prod, c->pipe_dec,
                                     c->pipe_has_prod ? c->pipe_nprod : 0,
                                     c->pipe_has_dec ? 1 : 0, c->dt == FPSK_BF16 ? 1 : 0,
                                     c->pipe_xb, lds, c->pipe_stream));
    c->pipe_dec = c->pipe_prod;
    c->pipe_has_dec = c->pipe_has_prod;
    c->pipe_has_prod = false;
  }
  if (had && next_st != c->pipe_stream) FPSK_HIP(hipStreamSynchronize(c->pipe_stream));
  return FPSK_OK;
}

fpsketch_status build_probe(fpsketch_ctx* c, int m, hipStream_t st) {
  HostRound R;
  const Decomp d = decompose(c->n1, c->n2, c->n3, m, false, c->transb);
  build_round(c->p.seed, 0, c->n1, c->n3, m, d.cwb, false, c->transb, R, true);
  FPSK_TRY(upload_round(R, d.cwb, c->probe_round, st));
  FPSK_TRY(ensure_workspace(c->probe_ws, c->n1, c->n2, c->n3, m, false, c->transb));
  c->m = m;
  c->qcache_m = 0;      // a cached B side belongs to the previous round
  return FPSK_OK;
}

fpsketch_status check_matrices(const fpsketch_ctx* c, const void* A, const void* B,
                               const void* C, fpsketch_dtype c_dtype) {
  if (c == nullptr) return fail(FPSK_EINVAL, "null context");
  if (c_dtype != FPSK_F32) {
    return fail(FPSK_EDTYPE, "C must be delivered in FP32 (a narrowed product is rejected)");
  }
  if (A == nullptr || B == nullptr || C == nullptr) return fail(FPSK_EINVAL, "null matrix");
  return FPSK_OK;
}

// rms-hat(C): strided samples on the device, statistics on the host (Sec. III-G).
fpsketch_status rms_hat_device(fpsketch_ctx* c, const float* C, hipStream_t st, double* out) {
  const int64_t total = c->n1 * c->n3;
  const int64_t stride = std::max<int64_t>(1, total / 65536);
  const int64_t count = (total + stride - 1) / stride;
  FPSK_TRY(dev_alloc(c->samples, static_cast<size_t>(count) * sizeof(float)));
  FPSK_HIP(fpsk::launch_sample(C, stride, count, as<float>(c->samples), st));
  std::vector<float> h(static_cast<size_t>(count));
  FPSK_HIP(hipMemcpyAsync(h.data(), c->samples.p, h.size() * sizeof(float),
                          hipMemcpyDeviceToHost, st));
  FPSK_HIP(hipStreamSynchronize(st));
  *out = rms_hat_from_samples(h.data(), count);
  return FPSK_OK;
}

// Recheck a list of coordinates: gamma, sum |A||B| and C_ij.
fpsketch_status recheck_coords(fpsketch_ctx* c, const void* A, const void* B, const float* C,
                               const std::vector<int64_t>& coords, std::vector<double>& gamma,
                               std::vector<double>& abssum, std::vector<float>& cval,
                               hipStream_t st) {
  const int n = static_cast<int>(coords.size() / 2);
  gamma.assign(n, 0.0);
  abssum.assign(n, 0.0);
  cval.assign(n, 0.0f);
  if (n == 0) return FPSK_OK;
  FPSK_TRY(dev_alloc(c->rc_coords, coords.size() * sizeof(int64_t)));
  FPSK_TRY(dev_alloc(c->rc_gamma, n * sizeof(double)));
  FPSK_TRY(dev_alloc(c->rc_abs, n * sizeof(double)));
  FPSK_TRY(dev_alloc(c->rc_c, n * sizeof(float)));
  FPSK_HIP(hipMemcpyAsync(c->rc_coords.p, coords.data(), coords.size() * sizeof(int64_t),
                          hipMemcpyHostToDevice, st));
  FPSK_HIP(fpsk::launch_recheck(static_cast<const uint16_t*>(A), static_cast<const uint16_t*>(B),
                                c->transb ? 1 : c->n3, c->transb ? c->n2 : 1,
                                C, c->n2, c->n3, c->dt == FPSK_BF16 ? 1 : 0,
                                as<int64_t>(c->rc_coords), n, as<double>(c->rc_gamma),
                                as<double>(c->rc_abs), as<float>(c->rc_c), st));
  FPSK_HIP(hipMemcpyAsync(gamma.data(), c->rc_gamma.p, n * sizeof(double), hipMemcpyDeviceToHost,
                          st));
  FPSK_HIP(hipMemcpyAsync(abssum.data(), c->rc_abs.p, n * sizeof(double), hipMemcpyDeviceToHost,
                          st));
  FPSK_HIP(hipMemcpyAsync(cval.data(), c->rc_c.p, n * sizeof(float), hipMemcpyDeviceToHost, st));
  FPSK_HIP(hipStreamSynchronize(st));
  return FPSK_OK;
}

// Exact scan (Sec. III-I): first K entries in row-major order that are non-finite or above
// fp32max/16 in magnitude.
fpsketch_status exact_scan(fpsketch_ctx* c, const float* C, int32_t K, hipStream_t st,
                           std::vector<int64_t>& coords) {
  coords.clear();
  FPSK_TRY(dev_alloc(c->scan_counts, static_cast<size_t>(c->n1) * sizeof(int32_t)));
  FPSK_HIP(fpsk::launch_scan_count(C, c->n1, c->n3, as<int32_t>(c->scan_counts), st));
  std::vector<int32_t> counts(static_cast<size_t>(c->n1));
  FPSK_HIP(hipMemcpyAsync(counts.data(), c->scan_counts.p, counts.size() * sizeof(int32_t),
                          hipMemcpyDeviceToHost, st));
  FPSK_HIP(hipStreamSynchronize(st));
  std::vector<int32_t> rows, base;
  int64_t total = 0;
  for (int64_t i = 0; i < c->n1 && total < K; ++i) {
    if (counts[i] > 0) {
      rows.push_back(static_cast<int32_t>(i));
      base.push_back(static_cast<int32_t>(total));
      total += counts[i];
    }
  }
  if (rows.empty()) return FPSK_OK;
  const int32_t keep = static_cast<int32_t>(std::min<int64_t>(total, K));
  FPSK_TRY(dev_alloc(c->scan_rows, rows.size() * sizeof(int32_t)));
  FPSK_TRY(dev_alloc(c->scan_base, base.size() * sizeof(int32_t)));
  FPSK_TRY(dev_alloc(c->scan_out, static_cast<size_t>(keep) * 2 * sizeof(int64_t)));
  FPSK_HIP(hipMemcpyAsync(c->scan_rows.p, rows.data(), rows.size() * sizeof(int32_t),
                          hipMemcpyHostToDevice, st));
  FPSK_HIP(hipMemcpyAsync(c->scan_base.p, base.data(), base.size() * sizeof(int32_t),
                          hipMemcpyHostToDevice, st));
  FPSK_HIP(fpsk::launch_scan_extract(C, c->n3, as<int32_t>(c->scan_rows),
                                     as<int32_t>(c->scan_base), static_cast<int>(rows.size()),
                                     keep, as<int64_t>(c->scan_out), st));
  coords.resize(static_cast<size_t>(keep) * 2);
  FPSK_HIP(hipMemcpyAsync(coords.data(), c->scan_out.p, coords.size() * sizeof(int64_t),
                          hipMemcpyDeviceToHost, st));
  FPSK_HIP(hipStreamSynchronize(st));
  return FPSK_OK;
}

// Sketches of one round into host arrays (S always; R, T with moments).
fpsketch_status sketch_round(fpsketch_ctx* c, uint64_t seed, int round, int m, bool mom,
                             const void* A, const void* B, const float* C, const int32_t* prow,
                             const int32_t* pcol, const float* pval, hipStream_t st,
                             HostRound& HR, std::vector<double>& S, std::vector<double>& Rm,
                             std::vector<double>& T, double* maxA, double* maxB) {
  const Decomp d = decompose(c->n1, c->n2, c->n3, m, mom, c->transb);
  build_round(seed, round, c->n1, c->n3, m, d.cwb, mom, c->transb, HR);
  FPSK_TRY(upload_round(HR, d.cwb, c->aux_round, st));
  FPSK_TRY(ensure_workspace(c->aux_ws, c->n1, c->n2, c->n3, m, mom, c->transb));
  FPSK_TRY(run_pass(c, c->aux_round, c->aux_ws, A, B, C, mom, 0, nullptr, prow, pcol, pval, st));
  const size_t mm = static_cast<size_t>(m) * static_cast<size_t>(m);
  S.resize(mm);
  FPSK_HIP(hipMemcpyAsync(S.data(), c->aux_ws.S.p, mm * sizeof(double), hipMemcpyDeviceToHost,
                          st));
  if (mom) {
    Rm.resize(mm);
    T.resize(mm);
    FPSK_HIP(hipMemcpyAsync(Rm.data(), c->aux_ws.R.p, mm * sizeof(double),
                            hipMemcpyDeviceToHost, st));
    FPSK_HIP(hipMemcpyAsync(T.data(), c->aux_ws.T.p, mm * sizeof(double),
                            hipMemcpyDeviceToHost, st));
  }
  std::vector<float> mp(static_cast<size_t>(d.nA + d.nB));
  FPSK_HIP(hipMemcpyAsync(mp.data(), c->aux_ws.maxpart.p, mp.size() * sizeof(float),
                          hipMemcpyDeviceToHost, st));
  FPSK_HIP(hipStreamSynchronize(st));
  float ma = 0.0f, mb = 0.0f;
  for (int i = 0; i < d.nA; ++i) ma = std::fmax(ma, mp[i]);
  for (int i = 0; i < d.nB; ++i) mb = std::fmax(mb, mp[d.nA + i]);
  if (maxA) *maxA = ma;
  if (maxB) *maxB = mb;
  return FPSK_OK;
}

// One sketch pass at m whose S stays in the auxiliary workspace, with the moment factors and
// C-grid partials when mom (R and T are then formed at selected buckets by launch_moments_at);
// max|A|, max|B| to host.
fpsketch_status sketch_round_device(fpsketch_ctx* c, uint64_t seed, int round, int m, bool mom,
                                    const void* A, const void* B, const float* C,
                                    const int32_t* prow, const int32_t* pcol, const float* pval,
                                    hipStream_t st, HostRound& HR, double* maxA, double* maxB) {
  const Decomp d = decompose(c->n1, c->n2, c->n3, m, mom, c->transb);
  build_round(seed, round, c->n1, c->n3, m, d.cwb, mom, c->transb, HR);
  FPSK_TRY(upload_round(HR, d.cwb, c->aux_round, st));
  FPSK_TRY(ensure_workspace(c->aux_ws, c->n1, c->n2, c->n3, m, mom, c->transb));
  FPSK_TRY(run_pass(c, c->aux_round, c->aux_ws, A, B, C, mom, 0, nullptr, prow, pcol, pval, st,
                    nullptr, nullptr, nullptr, BSide::kStream, false));
  std::vector<float> mp(static_cast<size_t>(d.nA + d.nB));
  FPSK_HIP(hipMemcpyAsync(mp.data(), c->aux_ws.maxpart.p, mp.size() * sizeof(float),
                          hipMemcpyDeviceToHost, st));
  FPSK_HIP(hipStreamSynchronize(st));
  float ma = 0.0f, mb = 0.0f;
  for (int i = 0; i < d.nA; ++i) ma = std::fmax(ma, mp[i]);
  for (int i = 0; i < d.nB; ++i) mb = std::fmax(mb, mp[d.nA + i]);
  *maxA = ma;
  *maxB = mb;
  return FPSK_OK;
}

// sigma_MAD = 1.4826 median(|S - median S|) of the m^2 buckets in the auxiliary workspace,
// selected exactly on the device (the host rule's values: even counts take the mean of the two
// middle order statistics).
fpsketch_status device_mad_sigma(fpsketch_ctx* c, int64_t mm, hipStream_t st, double* sigma) {
  FPSK_TRY(dev_alloc(c->sel_state, sizeof(fpsk::SelState)));
  FPSK_TRY(dev_alloc_zero(c->sel_hist, 256 * sizeof(uint32_t)));
  FPSK_HIP(fpsk::launch_median_mad(as<double>(c->aux_ws.S), mm, as<fpsk::SelState>(c->sel_state),
                                   as<uint32_t>(c->sel_hist), st));
  fpsk::SelState h{};
  FPSK_HIP(hipMemcpyAsync(&h, c->sel_state.p, sizeof(h), hipMemcpyDeviceToHost, st));
  FPSK_HIP(hipStreamSynchronize(st));
  *sigma = 1.4826 * h.mad;
  return FPSK_OK;
}

struct Found {
  int64_t i, j;
  double delta;
  int absolute;
  int round;
};

}  // namespace

// ==========================================================================================
// C ABI.

extern "C" {

void fpsketch_default_params(fpsketch_params* p) {
  if (p == nullptr) return;
  std::memset(p, 0, sizeof(*p));
  p->m = 0;
  p->rounds = 3;
  p->r_star = 4;
  p->r_max = 16;
  p->s_budget = 16;
  p->delta_rc = 8;
  p->k_cap = 0;
  p->rho_min = 0.02;
  p->mu = 4.0;
  p->c_valid = 100.0;
  p->b_star = 0.3;
  p->c_coll = 2.0;
  p->seed = 0x5EED5EEDull;
  p->law_cf_bf16 = 0.19;
  p->law_cf_fp16 = 0.19 * 1.76;
  p->law_n2_exp = 0.07;
}

const char* fpsketch_status_str(fpsketch_status s) {
  switch (s) {
    case FPSK_OK: return "ok";
    case FPSK_EINVAL: return "invalid argument";
    case FPSK_EDTYPE: return "unsupported dtype (C must be FP32; A, B FP16 or BF16)";
    case FPSK_ESHAPE: return "unsupported shape or bucket count";
    case FPSK_ENOMEM: return "device out of memory";
    case FPSK_EHIP: return "HIP runtime error";
    case FPSK_ECAPACITY: return "more fault records than capacity";
    case FPSK_ENODEV: return "no gfx950 device";
  }
  return "unknown status";
}

const char* fpsketch_last_error(void) { return g_last_error.c_str(); }

fpsketch_status fpsketch_hash_table(uint64_t seed, int32_t round, int32_t side, int64_t n,
                                    int32_t m, int32_t* bucket, int8_t* sign) {
  if (bucket == nullptr || sign == nullptr || n < 0 || m < 1 || round < 0 || side < 0 ||
      side > 1) {
    return fail(FPSK_EINVAL, "fpsketch_hash_table: bad argument");
  }
  hash_side(seed, round, side, n, m, bucket, sign);
  return FPSK_OK;
}

fpsketch_status fpsketch_m_start(int64_t n1, int64_t n2, int64_t n3, fpsketch_dtype ab_dtype,
                                 const fpsketch_params* params, int32_t* m_out) {
  fpsketch_params p;
  fpsketch_default_params(&p);
  if (params) p = *params;
  if (m_out == nullptr || n1 < 1 || n2 < 1 || n3 < 1) return fail(FPSK_EINVAL, "bad argument");
  if (!valid_half(ab_dtype)) return fail(FPSK_EDTYPE, "A, B must be FP16 or BF16");
  FPSK_TRY(check_params(p));
  *m_out = static_cast<int32_t>(m_start(n1, n2, n3, ab_dtype, p));
  return FPSK_OK;
}

fpsketch_status fpsketch_plan_host(int64_t n1, int64_t n2, int64_t n3, fpsketch_dtype ab_dtype,
                                   int32_t m, double sigma_hat, double rms,
                                   const fpsketch_params* params, int32_t* m_loc, int32_t* r,
                                   double* B, int32_t* fallback) {
  fpsketch_params p;
  fpsketch_default_params(&p);
  if (params) p = *params;
  if (m_loc == nullptr || r == nullptr || n1 < 1 || n2 < 1 || n3 < 1 || m < 1) {
    return fail(FPSK_EINVAL, "bad argument");
  }
  if (!valid_half(ab_dtype)) return fail(FPSK_EDTYPE, "A, B must be FP16 or BF16");
  FPSK_TRY(check_params(p));
  const PlanOut o = plan_localize(n1, n2, n3, ab_dtype, m, sigma_hat, rms, p);
  *m_loc = o.m_loc;
  *r = o.r;
  if (B) *B = o.B;
  if (fallback) *fallback = o.fallback;
  return FPSK_OK;
}

fpsketch_status fpsketch_recalibrate_host(int64_t n1, int64_t n3, int32_t m, double sigma_bar,
                                          double rms, const fpsketch_params* params,
                                          int32_t* m_new, int32_t* rebuild) {
  fpsketch_params p;
  fpsketch_default_params(&p);
  if (params) p = *params;
  if (m_new == nullptr || rebuild == nullptr || n1 < 1 || n3 < 1 || m < 1) {
    return fail(FPSK_EINVAL, "bad argument");
  }
  FPSK_TRY(check_params(p));
  recalibrate(n1, n3, m, sigma_bar, rms, p, m_new, rebuild);
  return FPSK_OK;
}

double fpsketch_rms_hat_samples(const float* samples, int64_t count) {
  if (samples == nullptr || count <= 0) return std::nan("");
  return rms_hat_from_samples(samples, count);
}

fpsketch_status fpsketch_create(int64_t n1, int64_t n2, int64_t n3, fpsketch_dtype ab_dtype,
                                const fpsketch_params* params, fpsketch_ctx** out) {
  if (out == nullptr) return fail(FPSK_EINVAL, "null output pointer");
  *out = nullptr;
  if (!valid_half(ab_dtype)) return fail(FPSK_EDTYPE, "A, B must be FP16 or BF16");
  const int64_t lim = int64_t{1} << 31;
  if (n1 < 1 || n2 < 1 || n3 < 1 || n1 >= lim || n2 >= lim || n3 >= lim) {
    return fail(FPSK_ESHAPE, "dimensions must be in [1, 2^31)");
  }
  fpsketch_params p;
  fpsketch_default_params(&p);
  if (params) p = *params;
  FPSK_TRY(check_params(p));
  int dev = 0;
  FPSK_HIP(hipGetDevice(&dev));
  hipDeviceProp_t prop;
  FPSK_HIP(hipGetDeviceProperties(&prop, dev));
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0) {
    return fail(FPSK_ENODEV, std::string("device is ") + prop.gcnArchName + ", not gfx950");
  }
  const int64_t m = p.m > 0 ? p.m : m_start(n1, n2, n3, ab_dtype, p);
  if (m < 1 || m > fpsk::kMaxM) return fail(FPSK_ESHAPE, "bucket count outside [1, 4096]");
  auto* c = new fpsketch_ctx();
  c->n1 = n1;
  c->n2 = n2;
  c->n3 = n3;
  c->dt = ab_dtype;
  c->transb = p.b_layout == 1;
  c->p = p;
  c->device = dev;
  c->L1 = pow2_ceil(n1);
  c->L3 = pow2_ceil(n3);
  c->inv_l1 = 1.0 / static_cast<double>(c->L1);
  c->inv_l3 = 1.0 / static_cast<double>(c->L3);
  fpsketch_status s = dev_alloc(c->stats, 8 * sizeof(double));
  if (s == FPSK_OK) s = dev_alloc(c->sigma_acc, 2 * sizeof(double));
  if (s == FPSK_OK) s = dev_alloc(c->zero, 64);
  if (s == FPSK_OK) {
    hipError_t e = hipMemset(c->stats.p, 0, 8 * sizeof(double));
    if (e == hipSuccess) e = hipMemset(c->zero.p, 0, 64);
    if (e == hipSuccess) e = hipMemset(c->sigma_acc.p, 0, 2 * sizeof(double));
    if (e != hipSuccess) s = fail(FPSK_EHIP, std::string("hipMemset: ") + hipGetErrorString(e));
  }
  if (s == FPSK_OK) s = build_probe(c, static_cast<int>(m), nullptr);
  if (s == FPSK_OK) s = scratch_address(dev, &c->scratch_dev);
  if (s != FPSK_OK) {
    fpsketch_destroy(c);
    return s;
  }
  *out = c;
  return FPSK_OK;
}

void fpsketch_destroy(fpsketch_ctx* c) {
  if (c == nullptr) return;
  (void)hipSetDevice(c->device);
  (void)pipe_flush(c, c->pipe_stream);
  (void)hipDeviceSynchronize();
  for (hipEvent_t e : c->events) (void)hipEventDestroy(e);
  free_round(c->probe_round);
  free_workspace(c->probe_ws);
  free_round(c->aux_round);
  free_workspace(c->aux_ws);
  for (Workspace& w : c->pipe_ws) free_workspace(w);
  for (DevBuf* b : {&c->stats, &c->sigma_acc, &c->zero, &c->scan_counts, &c->scan_rows, &c->scan_base,
                    &c->scan_out, &c->samples, &c->patch_rowptr, &c->patch_col, &c->patch_val,
                    &c->rc_coords, &c->rc_gamma, &c->rc_abs, &c->rc_c, &c->sel_state,
                    &c->sel_hist, &c->peel_list, &c->cands, &c->cand_count, &c->apply_list,
                    &c->mo_list, &c->mo_rt,
                    &c->reprobe_stats, &c->reprobe_acc, &c->qcache, &c->maxb_cache}) {
    dev_free(*b);
  }
  delete c;
}

fpsketch_status fpsketch_probe(fpsketch_ctx* c, const void* A, const void* B, const void* C,
                               fpsketch_dtype c_dtype, int32_t* d_dirty, void* stream) {
  FPSK_TRY(check_matrices(c, A, B, C, c_dtype));
  FPSK_TRY(set_device(c));
  const hipStream_t st = static_cast<hipStream_t>(stream);
  FPSK_TRY(pipe_flush(c, st));
  hipEvent_t* ev = nullptr;
  if (c->timing) {
    while (c->events.size() < c->events_used + 4) {
      hipEvent_t e;
      FPSK_HIP(hipEventCreate(&e));
      c->events.push_back(e);
    }
    ev = c->events.data() + c->events_used;
    c->events_used += 4;
  }
  return run_pass(c, c->probe_round, c->probe_ws, A, B, static_cast<const float*>(C), false, 1,
                  d_dirty, nullptr, nullptr, nullptr, st, ev);
}

// fpsketch_probe on the block path with its factors (P, Q), C-grid partials, block-product
// partials and per-work-group maxima carved from this device's scratch instead of the
// context's workspace.  The factors' padding columns [n2, kact) must read as zero in the
// products; the scratch keeps whatever the previous call left there, so a fill kernel clears
// them (a kernel, not a memset, so that the call stays capturable).
fpsketch_status fpsketch_probe_noalloc(fpsketch_ctx* c, const void* A, const void* B,
                                       const void* C, fpsketch_dtype c_dtype, int32_t* d_dirty,
                                       void* stream) {
  FPSK_TRY(check_matrices(c, A, B, C, c_dtype));
  const Decomp& d = c->probe_ws.d;
  if (d.nX == 0) {
    return fail(FPSK_ESHAPE, "the probe without allocation takes the block path only (m <= 64, "
                             "n2 <= 16384); this context has m = " + std::to_string(d.m));
  }
  if (c->scratch_dev == nullptr) return fail(FPSK_EINVAL, "internal: no scratch address");
  FPSK_TRY(set_device(c));
  const hipStream_t st = static_cast<hipStream_t>(stream);
  FPSK_TRY(pipe_flush(c, st));
  const size_t mm = static_cast<size_t>(d.m) * d.m;
  const size_t fm = static_cast<size_t>(d.m) * d.ldp * sizeof(float);
  size_t off = 0;
  auto take = [&off](size_t bytes) {
    const size_t o = off;
    off += (bytes + 255) / 256 * 256;
    return o;
  };
  const size_t oP = take(fm), oQ = take(fm);
  const size_t oS = take(mm * d.npc * sizeof(double));
  const size_t oX = take(mm * d.xns * sizeof(double));
  const size_t oM = take(static_cast<size_t>(d.nA + d.nB) * sizeof(float));
  if (off > kScratchBytes) {
    return fail(FPSK_ESHAPE, "the probe without allocation needs " + std::to_string(off) +
                                 " bytes of scratch, more than its " +
                                 std::to_string(kScratchBytes));
  }
  Workspace W;            // a view of the scratch: owns nothing and is never freed
  W.d = d;
  W.ds = d;
  W.P.p = c->scratch_dev + oP;
  W.Q.p = c->scratch_dev + oQ;
  W.partS.p = c->scratch_dev + oS;
  W.xpart.p = c->scratch_dev + oX;
  W.maxpart.p = c->scratch_dev + oM;
  if (d.kact > c->n2) {
    const int n2 = static_cast<int>(c->n2);
    FPSK_HIP(fpsk::launch_zero_cols(as<float>(W.P), d.m, d.ldp, n2, d.kact, st));
    FPSK_HIP(fpsk::launch_zero_cols(as<float>(W.Q), d.m, d.ldp, n2, d.kact, st));
  }
  return run_pass(c, c->probe_round, W, A, B, static_cast<const float*>(C), false, 1, d_dirty,
                  nullptr, nullptr, nullptr, st);
}

fpsketch_status fpsketch_cache_b(fpsketch_ctx* c, const void* B, void* stream) {
  if (c == nullptr || B == nullptr) return fail(FPSK_EINVAL, "null argument");
  FPSK_TRY(set_device(c));
  const hipStream_t st = static_cast<hipStream_t>(stream);
  FPSK_TRY(pipe_flush(c, st));
  const Decomp& d = c->probe_ws.d;
  const size_t fm = static_cast<size_t>(c->m) * static_cast<size_t>(d.ldp) * sizeof(float);
  FPSK_TRY(dev_alloc_zero(c->qcache, fm));
  FPSK_TRY(dev_alloc(c->maxb_cache, static_cast<size_t>(d.nB) * sizeof(float)));
  FPSK_TRY(run_pass(c, c->probe_round, c->probe_ws, c->zero.p, B, nullptr, false, 1, nullptr,
                    nullptr, nullptr, nullptr, st, nullptr, nullptr, nullptr,
                    BSide::kFillCache));
  c->qcache_m = c->m;
  return FPSK_OK;
}

fpsketch_status fpsketch_probe_cached(fpsketch_ctx* c, const void* A, const void* C,
                                      fpsketch_dtype c_dtype, int32_t* d_dirty, void* stream) {
  if (c == nullptr) return fail(FPSK_EINVAL, "null context");
  FPSK_TRY(check_matrices(c, A, c->zero.p, C, c_dtype));
  if (c->qcache_m != c->m) {
    return fail(FPSK_EINVAL, "no B side cached for the probe's current m (call fpsketch_cache_b)");
  }
  FPSK_TRY(set_device(c));
  const hipStream_t st = static_cast<hipStream_t>(stream);
  FPSK_TRY(pipe_flush(c, st));
  hipEvent_t* ev = nullptr;
  if (c->timing) {
    while (c->events.size() < c->events_used + 4) {
      hipEvent_t e;
      FPSK_HIP(hipEventCreate(&e));
      c->events.push_back(e);
    }
    ev = c->events.data() + c->events_used;
    c->events_used += 4;
  }
  return run_pass(c, c->probe_round, c->probe_ws, A, c->zero.p, static_cast<const float*>(C),
                  false, 1, d_dirty, nullptr, nullptr, nullptr, st, ev, nullptr, nullptr,
                  BSide::kUseCache);
}

// A deferred probe (streamed or cached B side) on the caller's stream.
fpsketch_status deferred_probe(fpsketch_ctx* c, const void* A, const void* B, const float* C,
                               int32_t* d_dirty, hipStream_t st, BSide bside) {
  if ((c->pipe_has_prod || c->pipe_has_dec) && st != c->pipe_stream) {
    return fail(FPSK_EINVAL, "deferred probes are pending on another stream");
  }
  if (c->probe_ws.d.nX == 0) {
    // not the block path (m > 64 or n2 > 16384): an ordinary probe, nothing left pending
    FPSK_TRY(pipe_flush(c, st));
    return run_pass(c, c->probe_round, c->probe_ws, A, B, C, false, 1, d_dirty, nullptr, nullptr,
                    nullptr, st, nullptr, nullptr, nullptr, bside);
  }
  Workspace& W = c->pipe_ws[c->pipe_next];
  FPSK_TRY(ensure_workspace(W, c->n1, c->n2, c->n3, c->m, false, c->transb, true));
  const Decomp& d = W.d;
  fpsk::StreamArgs s;
  fpsk::ProductArgs a;
  FPSK_TRY(pass_args(c, c->probe_round, W, A, B, C, false, 1, d_dirty, nullptr, nullptr, nullptr,
                     nullptr, nullptr, bside, s, a));
  const size_t lds = std::max(d.lds_stream, fpsk::probe_pipe_lds(d.xb));
  FPSK_HIP(fpsk::launch_probe_pipe(s, c->pipe_prod, c->pipe_dec,
                                   c->pipe_has_prod ? c->pipe_nprod : 0,
                                   c->pipe_has_dec ? 1 : 0, c->dt == FPSK_BF16 ? 1 : 0, d.xb,
                                   lds, st));
  c->pipe_dec = c->pipe_prod;
  c->pipe_has_dec = c->pipe_has_prod;
  c->pipe_prod = a;
  c->pipe_has_prod = true;
  c->pipe_nprod = d.nX;
  c->pipe_xb = d.xb;
  c->pipe_stream = st;
  c->pipe_next = (c->pipe_next + 1) % 3;
  return FPSK_OK;
}

fpsketch_status fpsketch_probe_deferred(fpsketch_ctx* c, const void* A, const void* B,
                                        const void* C, fpsketch_dtype c_dtype, int32_t* d_dirty,
                                        void* stream) {
  FPSK_TRY(check_matrices(c, A, B, C, c_dtype));
  FPSK_TRY(set_device(c));
  return deferred_probe(c, A, B, static_cast<const float*>(C), d_dirty,
                        static_cast<hipStream_t>(stream), BSide::kStream);
}

fpsketch_status fpsketch_probe_cached_deferred(fpsketch_ctx* c, const void* A, const void* C,
                                               fpsketch_dtype c_dtype, int32_t* d_dirty,
                                               void* stream) {
  if (c == nullptr) return fail(FPSK_EINVAL, "null context");
  FPSK_TRY(check_matrices(c, A, c->zero.p, C, c_dtype));
  if (c->qcache_m != c->m) {
    return fail(FPSK_EINVAL, "no B side cached for the probe's current m (call fpsketch_cache_b)");
  }
  FPSK_TRY(set_device(c));
  return deferred_probe(c, A, c->zero.p, static_cast<const float*>(C), d_dirty,
                        static_cast<hipStream_t>(stream), BSide::kUseCache);
}

fpsketch_status fpsketch_probe_flush(fpsketch_ctx* c, void* stream) {
  if (c == nullptr) return fail(FPSK_EINVAL, "null context");
  if (!(c->pipe_has_prod || c->pipe_has_dec)) return FPSK_OK;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  if (st != c->pipe_stream) {
    return fail(FPSK_EINVAL, "deferred probes are pending on another stream");
  }
  FPSK_TRY(set_device(c));
  return pipe_flush(c, st);
}

fpsketch_status fpsketch_timing(fpsketch_ctx* c, int32_t enable) {
  if (c == nullptr) return fail(FPSK_EINVAL, "null context");
  c->timing = enable != 0;
  c->events_used = 0;
  return FPSK_OK;
}

fpsketch_status fpsketch_timing_read(fpsketch_ctx* c, double* stream_ms, double* product_ms,
                                     int64_t* calls) {
  if (c == nullptr || stream_ms == nullptr || product_ms == nullptr || calls == nullptr) {
    return fail(FPSK_EINVAL, "null argument");
  }
  FPSK_TRY(set_device(c));
  double s1 = 0.0, s2 = 0.0;
  const size_t n = c->events_used / 4;
  if (n > 0) FPSK_HIP(hipEventSynchronize(c->events[4 * n - 1]));
  for (size_t k = 0; k < n; ++k) {
    float a = 0.0f, b = 0.0f;
    FPSK_HIP(hipEventElapsedTime(&a, c->events[4 * k], c->events[4 * k + 1]));
    FPSK_HIP(hipEventElapsedTime(&b, c->events[4 * k + 2], c->events[4 * k + 3]));
    s1 += a;
    s2 += b;
  }
  *stream_ms = s1;
  *product_ms = s2;
  *calls = static_cast<int64_t>(n);
  c->events_used = 0;
  return FPSK_OK;
}

fpsketch_status fpsketch_get_m(fpsketch_ctx* c, int32_t* m_out) {
  if (c == nullptr || m_out == nullptr) return fail(FPSK_EINVAL, "null argument");
  *m_out = c->m;
  return FPSK_OK;
}

fpsketch_status fpsketch_probe_stats(fpsketch_ctx* c, double* out, void* stream) {
  if (c == nullptr || out == nullptr) return fail(FPSK_EINVAL, "null argument");
  FPSK_TRY(set_device(c));
  const hipStream_t st = static_cast<hipStream_t>(stream);
  FPSK_TRY(pipe_flush(c, st));
  FPSK_HIP(hipMemcpyAsync(out, c->stats.p, 8 * sizeof(double), hipMemcpyDeviceToHost, st));
  FPSK_HIP(hipStreamSynchronize(st));
  return FPSK_OK;
}

fpsketch_status fpsketch_get_plan(fpsketch_ctx* c, fpsketch_plan_info* out) {
  if (c == nullptr || out == nullptr) return fail(FPSK_EINVAL, "null argument");
  *out = c->last_plan;
  return FPSK_OK;
}

fpsketch_status fpsketch_sketch(fpsketch_ctx* c, const void* A, const void* B, const void* C,
                                fpsketch_dtype c_dtype, uint64_t seed, int32_t round, int32_t m,
                                int32_t moments, double* S, double* R, double* T, double* maxab,
                                void* stream) {
  FPSK_TRY(check_matrices(c, A, B, C, c_dtype));
  if (S == nullptr || (moments && (R == nullptr || T == nullptr)) || round < 0) {
    return fail(FPSK_EINVAL, "null output or bad round");
  }
  if (m < 1 || m > fpsk::kMaxM) return fail(FPSK_ESHAPE, "bucket count outside [1, 4096]");
  FPSK_TRY(set_device(c));
  const hipStream_t st = static_cast<hipStream_t>(stream);
  FPSK_TRY(pipe_flush(c, st));
  HostRound HR;
  std::vector<double> hS, hR, hT;
  double ma = 0, mb = 0;
  FPSK_TRY(sketch_round(c, seed, round, m, moments != 0, A, B, static_cast<const float*>(C),
                        nullptr, nullptr, nullptr, st, HR, hS, hR, hT, &ma, &mb));
  std::memcpy(S, hS.data(), hS.size() * sizeof(double));
  if (moments) {
    std::memcpy(R, hR.data(), hR.size() * sizeof(double));
    std::memcpy(T, hT.data(), hT.size() * sizeof(double));
  }
  if (maxab) {
    maxab[0] = ma;
    maxab[1] = mb;
  }
  return FPSK_OK;
}

fpsketch_status fpsketch_recheck(fpsketch_ctx* c, const void* A, const void* B,
                                 const int64_t* coords, int32_t n, double* gamma, double* abssum,
                                 void* stream) {
  if (c == nullptr || A == nullptr || B == nullptr || (n > 0 && (coords == nullptr ||
                                                                 gamma == nullptr ||
                                                                 abssum == nullptr)) ||
      n < 0) {
    return fail(FPSK_EINVAL, "null argument");
  }
  for (int32_t t = 0; t < n; ++t) {
    if (coords[2 * t] < 0 || coords[2 * t] >= c->n1 || coords[2 * t + 1] < 0 ||
        coords[2 * t + 1] >= c->n3) {
      return fail(FPSK_EINVAL, "coordinate outside C");
    }
  }
  FPSK_TRY(set_device(c));
  const hipStream_t st = static_cast<hipStream_t>(stream);
  FPSK_TRY(pipe_flush(c, st));
  if (n == 0) return FPSK_OK;
  const size_t nn = static_cast<size_t>(n);
  FPSK_TRY(dev_alloc(c->rc_coords, 2 * nn * sizeof(int64_t)));
  FPSK_TRY(dev_alloc(c->rc_gamma, nn * sizeof(double)));
  FPSK_TRY(dev_alloc(c->rc_abs, nn * sizeof(double)));
  FPSK_HIP(hipMemcpyAsync(c->rc_coords.p, coords, 2 * nn * sizeof(int64_t),
                          hipMemcpyHostToDevice, st));
  // no C here: the kernel skips the C read when C is null
  FPSK_HIP(fpsk::launch_recheck(static_cast<const uint16_t*>(A), static_cast<const uint16_t*>(B),
                                c->transb ? 1 : c->n3, c->transb ? c->n2 : 1,
                                nullptr, c->n2, c->n3, c->dt == FPSK_BF16 ? 1 : 0,
                                as<int64_t>(c->rc_coords), n, as<double>(c->rc_gamma),
                                as<double>(c->rc_abs), nullptr, st));
  FPSK_HIP(hipMemcpyAsync(gamma, c->rc_gamma.p, nn * sizeof(double), hipMemcpyDeviceToHost, st));
  FPSK_HIP(hipMemcpyAsync(abssum, c->rc_abs.p, nn * sizeof(double), hipMemcpyDeviceToHost, st));
  FPSK_HIP(hipStreamSynchronize(st));
  return FPSK_OK;
}

fpsketch_status fpsketch_apply(fpsketch_ctx* c, const void* A, const void* B, void* C,
                               fpsketch_dtype c_dtype, const fpsketch_fault* recs, int32_t n,
                               uint64_t seed, int32_t* still_dirty, void* stream) {
  FPSK_TRY(check_matrices(c, A, B, C, c_dtype));
  if (still_dirty == nullptr || n < 0 || (n > 0 && recs == nullptr)) {
    return fail(FPSK_EINVAL, "null argument or negative record count");
  }
  std::vector<fpsk::ApplyEntry> list(static_cast<size_t>(n));
  std::unordered_set<int64_t> seen;
  for (int32_t t = 0; t < n; ++t) {
    const fpsketch_fault& f = recs[t];
    if (f.i < 0 || f.i >= c->n1 || f.j < 0 || f.j >= c->n3) {
      return fail(FPSK_EINVAL, "record outside C");
    }
    const int64_t o = f.i * c->n3 + f.j;
    if (!seen.insert(o).second) return fail(FPSK_EINVAL, "record coordinate listed twice");
    list[t] = {o, f.delta, f.absolute ? 1 : 0, 0};
  }
  FPSK_TRY(set_device(c));
  const hipStream_t st = static_cast<hipStream_t>(stream);
  FPSK_TRY(pipe_flush(c, st));
  float* Cm = static_cast<float*>(C);
  if (n > 0) {
    FPSK_TRY(dev_alloc(c->apply_list, list.size() * sizeof(fpsk::ApplyEntry)));
    FPSK_HIP(hipMemcpyAsync(c->apply_list.p, list.data(), list.size() * sizeof(fpsk::ApplyEntry),
                            hipMemcpyHostToDevice, st));
    FPSK_HIP(fpsk::launch_apply(Cm, as<fpsk::ApplyEntry>(c->apply_list), n, st));
  }
  // re-probe with a fresh round at the probe's m; its statistics go to buffers of their own
  const int m = c->m;
  const Decomp d = decompose(c->n1, c->n2, c->n3, m, false, c->transb);
  HostRound HR;
  build_round(seed, 0, c->n1, c->n3, m, d.cwb, false, c->transb, HR, true);
  FPSK_TRY(upload_round(HR, d.cwb, c->aux_round, st));
  FPSK_TRY(ensure_workspace(c->aux_ws, c->n1, c->n2, c->n3, m, false, c->transb));
  FPSK_TRY(dev_alloc(c->reprobe_stats, 8 * sizeof(double)));
  FPSK_TRY(dev_alloc(c->reprobe_acc, 2 * sizeof(double)));
  FPSK_TRY(run_pass(c, c->aux_round, c->aux_ws, A, B, Cm, false, 1, nullptr, nullptr, nullptr,
                    nullptr, st, nullptr, as<double>(c->reprobe_stats),
                    as<double>(c->reprobe_acc)));
  double stt[8];
  FPSK_HIP(hipMemcpyAsync(stt, c->reprobe_stats.p, sizeof(stt), hipMemcpyDeviceToHost, st));
  FPSK_HIP(hipStreamSynchronize(st));
  *still_dirty = stt[5] != 0.0 ? 1 : 0;
  return FPSK_OK;
}

fpsketch_status fpsketch_calibrate_noise(fpsketch_ctx* c, const void* C, fpsketch_dtype c_dtype,
                                         void* stream, int32_t* m_out, double* sigma_bar_out,
                                         int32_t* rebuilt_out) {
  if (c == nullptr) return fail(FPSK_EINVAL, "null context");
  if (c_dtype != FPSK_F32) return fail(FPSK_EDTYPE, "C must be delivered in FP32");
  if (C == nullptr) return fail(FPSK_EINVAL, "null C");
  FPSK_TRY(set_device(c));
  const hipStream_t st = static_cast<hipStream_t>(stream);
  FPSK_TRY(pipe_flush(c, st));
  double acc[2] = {0.0, 0.0};
  FPSK_HIP(hipMemcpyAsync(acc, c->sigma_acc.p, sizeof(acc), hipMemcpyDeviceToHost, st));
  FPSK_HIP(hipStreamSynchronize(st));
  const double sigma_bar = acc[1] > 0 ? acc[0] / acc[1] : std::nan("");
  int32_t rebuilt = 0;
  if (acc[1] > 0) {
    double rms = 0;
    FPSK_TRY(rms_hat_device(c, static_cast<const float*>(C), st, &rms));
    int32_t m_new = c->m;
    recalibrate(c->n1, c->n3, c->m, sigma_bar, rms, c->p, &m_new, &rebuilt);
    if (rebuilt && m_new > fpsk::kMaxM) {
      // the noise asks for more buckets than the kernels take: nothing changes
      if (m_out) *m_out = c->m;
      if (sigma_bar_out) *sigma_bar_out = sigma_bar;
      if (rebuilt_out) *rebuilt_out = 0;
      return fail(FPSK_ESHAPE, "recalibrated bucket count " + std::to_string(m_new) +
                                   " is beyond the kernels' 4096; the probe keeps m = " +
                                   std::to_string(c->m));
    }
    if (rebuilt) {
      FPSK_TRY(build_probe(c, m_new, st));
      const double zero[2] = {0.0, 0.0};
      FPSK_HIP(hipMemcpyAsync(c->sigma_acc.p, zero, sizeof(zero), hipMemcpyHostToDevice, st));
      FPSK_HIP(hipStreamSynchronize(st));
    }
  }
  if (m_out) *m_out = c->m;
  if (sigma_bar_out) *sigma_bar_out = sigma_bar;
  if (rebuilt_out) *rebuilt_out = rebuilt;
  return FPSK_OK;
}

fpsketch_status fpsketch_localize(fpsketch_ctx* c, const void* A, const void* B, const void* C,
                                  fpsketch_dtype c_dtype, uint64_t seed, int32_t sigma_from_probe,
                                  fpsketch_fault* out, int32_t cap, int32_t* n_out,
                                  void* stream) {
  FPSK_TRY(check_matrices(c, A, B, C, c_dtype));
  if (n_out == nullptr || cap < 0 || (cap > 0 && out == nullptr)) {
    return fail(FPSK_EINVAL, "bad output arguments");
  }
  FPSK_TRY(set_device(c));
  const hipStream_t st = static_cast<hipStream_t>(stream);
  FPSK_TRY(pipe_flush(c, st));
  const float* Cf = static_cast<const float*>(C);
  const int32_t K = cap_K(c->p);
  std::vector<Found> F;

  // 1. Exact scan and absolute recompute (Sec. III-I; Algorithm 2).
  std::vector<int64_t> abs_coords;
  FPSK_TRY(exact_scan(c, Cf, K, st, abs_coords));
  std::vector<double> g, ab;
  std::vector<float> cv;
  FPSK_TRY(recheck_coords(c, A, B, Cf, abs_coords, g, ab, cv, st));
  const size_t n_abs = abs_coords.size() / 2;
  for (size_t t = 0; t < n_abs; ++t) {
    F.push_back({abs_coords[2 * t], abs_coords[2 * t + 1], g[t], 1, 0});
  }
  // Patch list (row-major order already): C holds fl32(gamma) at these entries while sketching.
  const int32_t* prow = nullptr;
  const int32_t* pcol = nullptr;
  const float* pval = nullptr;
  if (n_abs > 0) {
    std::vector<int32_t> rowptr(static_cast<size_t>(c->n1) + 1, 0), col(n_abs);
    std::vector<float> val(n_abs);
    for (size_t t = 0; t < n_abs; ++t) {
      rowptr[static_cast<size_t>(abs_coords[2 * t]) + 1]++;
      col[t] = static_cast<int32_t>(abs_coords[2 * t + 1]);
      val[t] = static_cast<float>(g[t]);
    }
    for (int64_t i = 0; i < c->n1; ++i) rowptr[i + 1] += rowptr[i];
    FPSK_TRY(dev_alloc(c->patch_rowptr, rowptr.size() * sizeof(int32_t)));
    FPSK_TRY(dev_alloc(c->patch_col, col.size() * sizeof(int32_t)));
    FPSK_TRY(dev_alloc(c->patch_val, val.size() * sizeof(float)));
    FPSK_HIP(hipMemcpyAsync(c->patch_rowptr.p, rowptr.data(), rowptr.size() * sizeof(int32_t),
                            hipMemcpyHostToDevice, st));
    FPSK_HIP(hipMemcpyAsync(c->patch_col.p, col.data(), col.size() * sizeof(int32_t),
                            hipMemcpyHostToDevice, st));
    FPSK_HIP(hipMemcpyAsync(c->patch_val.p, val.data(), val.size() * sizeof(float),
                            hipMemcpyHostToDevice, st));
    FPSK_HIP(hipStreamSynchronize(st));
    prow = as<int32_t>(c->patch_rowptr);
    pcol = as<int32_t>(c->patch_col);
    pval = as<float>(c->patch_val);
  }

  // 2. Plan from the measured noise (Sec. III-G).
  double rms = 0.0;
  FPSK_TRY(rms_hat_device(c, Cf, st, &rms));
  double sigma = std::nan("");
  if (sigma_from_probe) {
    double stt[8];
    FPSK_HIP(hipMemcpyAsync(stt, c->stats.p, sizeof(stt), hipMemcpyDeviceToHost, st));
    FPSK_HIP(hipStreamSynchronize(st));
    sigma = stt[0];
  } else {
    HostRound HR0;
    double ma0 = 0.0, mb0 = 0.0;
    FPSK_TRY(sketch_round_device(c, seed, 0, c->m, false, A, B, Cf, prow, pcol, pval, st, HR0,
                                 &ma0, &mb0));
    FPSK_TRY(device_mad_sigma(c, static_cast<int64_t>(c->m) * c->m, st, &sigma));
  }
  const PlanOut plan = plan_localize(c->n1, c->n2, c->n3, c->dt, c->m, sigma, rms, c->p);
  if (plan.m_loc > fpsk::kMaxM) return fail(FPSK_ESHAPE, "m_loc beyond 4096");

  // 3. Rounds t = 1..k (Algorithm 1).
  std::unordered_set<int64_t> inF;
  auto key = [c](int64_t i, int64_t j) { return i * c->n3 + j; };
  for (const Found& f : F) inF.insert(key(f.i, f.j));
  const int r = plan.r;
  std::vector<std::pair<int, int>> offs;
  for (int di = -r; di <= r; ++di)
    for (int dj = -r; dj <= r; ++dj) offs.emplace_back(di, dj);
  std::sort(offs.begin(), offs.end(), [](const std::pair<int, int>& x, const std::pair<int, int>& y) {
    const int cx = std::max(std::abs(x.first), std::abs(x.second));
    const int cy = std::max(std::abs(y.first), std::abs(y.second));
    if (cx != cy) return cx < cy;
    const int mx = std::abs(x.first) + std::abs(x.second);
    const int my = std::abs(y.first) + std::abs(y.second);
    if (mx != my) return mx < my;
    return x < y;
  });
  double tau = 0.0;
  int32_t n_rechecked = 0;
  const int m = plan.m_loc;
  const double L1 = static_cast<double>(c->L1), L3 = static_cast<double>(c->L3);
  for (int t = 1; t <= c->p.rounds; ++t) {
    HostRound HR;
    double maxA = 0, maxB = 0;
    FPSK_TRY(sketch_round_device(c, seed, t, m, true, A, B, Cf, prow, pcol, pval, st, HR, &maxA,
                                 &maxB));
    tau = c->p.c_valid * static_cast<double>(c->n2) * std::ldexp(1.0, -23) * maxA * maxB;
    const int64_t mm = static_cast<int64_t>(m) * m;
    double* dS = as<double>(c->aux_ws.S);
    // peel every finite fault confirmed so far (Sec. III-H), in order, on the device (S here;
    // R and T at the selected buckets below)
    std::vector<fpsk::PeelEntry> peel;
    for (const Found& f : F) {
      if (f.absolute) continue;
      const int64_t o = static_cast<int64_t>(HR.h1[f.i]) * m + HR.h2[f.j];
      const double sv = static_cast<double>(HR.v1[f.i]) * HR.v2[f.j] * f.delta;
      peel.push_back({o, sv, sv * static_cast<double>(f.i + 1) / L1,
                      sv * static_cast<double>(f.j + 1) / L3});
    }
    if (!peel.empty()) {
      FPSK_TRY(dev_alloc(c->peel_list, peel.size() * sizeof(fpsk::PeelEntry)));
      FPSK_HIP(hipMemcpyAsync(c->peel_list.p, peel.data(), peel.size() * sizeof(fpsk::PeelEntry),
                              hipMemcpyHostToDevice, st));
      FPSK_HIP(fpsk::launch_peel(dS, nullptr, nullptr, as<fpsk::PeelEntry>(c->peel_list),
                                 static_cast<int>(peel.size()), st));
    }
    double sig = 0.0;
    FPSK_TRY(device_mad_sigma(c, mm, st, &sig));
    const double tau_c = std::min(tau, 2.0 * sig);
    const double tau_d = static_cast<double>(std::max(c->n1, c->n3)) * sig /
                         std::max(static_cast<double>(r), 0.5);
    const double cut = std::max(tau_c, tau_d);
    // buckets with |S| > cut, with their sketches; by |S| descending, then bucket index
    constexpr uint32_t kCandCap = 1u << 20;
    FPSK_TRY(dev_alloc(c->cands, static_cast<size_t>(kCandCap) * sizeof(fpsk::Cand)));
    FPSK_TRY(dev_alloc(c->cand_count, sizeof(uint32_t)));
    FPSK_HIP(hipMemsetAsync(c->cand_count.p, 0, sizeof(uint32_t), st));
    FPSK_HIP(fpsk::launch_above(dS, nullptr, nullptr, mm, cut, as<fpsk::Cand>(c->cands),
                                kCandCap, as<uint32_t>(c->cand_count), st));
    uint32_t ncand = 0;
    FPSK_HIP(hipMemcpyAsync(&ncand, c->cand_count.p, sizeof(ncand), hipMemcpyDeviceToHost, st));
    FPSK_HIP(hipStreamSynchronize(st));
    std::vector<fpsk::Cand> above;
    if (ncand <= kCandCap) {
      above.resize(ncand);
      if (ncand > 0) {
        FPSK_HIP(hipMemcpyAsync(above.data(), c->cands.p, ncand * sizeof(fpsk::Cand),
                                hipMemcpyDeviceToHost, st));
        FPSK_HIP(hipStreamSynchronize(st));
      }
    } else {
      // more candidates than the buffer holds: scan the whole grid on the host
      std::vector<double> S(mm);
      FPSK_HIP(hipMemcpyAsync(S.data(), dS, mm * sizeof(double), hipMemcpyDeviceToHost, st));
      FPSK_HIP(hipStreamSynchronize(st));
      for (int64_t o = 0; o < mm; ++o)
        if (std::fabs(S[o]) > cut) above.push_back({o, S[o], 0.0, 0.0});
    }
    std::sort(above.begin(), above.end(), [](const fpsk::Cand& x, const fpsk::Cand& y) {
      const double ax = std::fabs(x.s), ay = std::fabs(y.s);
      if (ax != ay) return ax > ay;
      return x.o < y.o;
    });
    if (static_cast<int64_t>(above.size()) > K) above.resize(K);
    // R and T (Eq. 2) at the top-K buckets only, with the peel terms
    if (!above.empty()) {
      const size_t na = above.size();
      std::vector<int64_t> ol(na);
      for (size_t q = 0; q < na; ++q) ol[q] = above[q].o;
      FPSK_TRY(dev_alloc(c->mo_list, na * sizeof(int64_t)));
      FPSK_TRY(dev_alloc(c->mo_rt, 2 * na * sizeof(double)));
      FPSK_HIP(hipMemcpyAsync(c->mo_list.p, ol.data(), na * sizeof(int64_t),
                              hipMemcpyHostToDevice, st));
      fpsk::MomentsAtArgs g{};
      g.P = as<float>(c->aux_ws.P);
      g.Pw = as<float>(c->aux_ws.Pw);
      g.Q = as<float>(c->aux_ws.Q);
      g.Qw = as<float>(c->aux_ws.Qw);
      g.partR = as<double>(c->aux_ws.partR);
      g.partT = as<double>(c->aux_ws.partT);
      g.o = as<int64_t>(c->mo_list);
      g.peel = peel.empty() ? nullptr : as<fpsk::PeelEntry>(c->peel_list);
      g.npeel = static_cast<int>(peel.size());
      g.r = as<double>(c->mo_rt);
      g.t = g.r + na;
      g.m = m;
      g.ldp = c->aux_ws.d.ldp;
      g.kact = c->aux_ws.d.kact;
      g.npc = c->aux_ws.d.npc;
      FPSK_HIP(fpsk::launch_moments_at(g, static_cast<int>(na), st));
      std::vector<double> rt(2 * na);
      FPSK_HIP(hipMemcpyAsync(rt.data(), c->mo_rt.p, 2 * na * sizeof(double),
                              hipMemcpyDeviceToHost, st));
      FPSK_HIP(hipStreamSynchronize(st));
      for (size_t q = 0; q < na; ++q) {
        above[q].r = rt[q];
        above[q].t = rt[na + q];
      }
    }
    struct Center {
      int64_t ci, cj;
    };
    std::vector<Center> live;
    for (const fpsk::Cand& cd : above) {
      const double s = cd.s, rr = cd.r, tt = cd.t;
      if (!(s != 0.0 && std::isfinite(s) && std::isfinite(rr) && std::isfinite(tt))) continue;
      const double ri = L1 * rr / s, rj = L3 * tt / s;
      if (!std::isfinite(ri) || !std::isfinite(rj) || std::fabs(ri) > 0x1p40 ||
          std::fabs(rj) > 0x1p40) {
        continue;
      }
      live.push_back({static_cast<int64_t>(std::nearbyint(ri)) - 1,
                      static_cast<int64_t>(std::nearbyint(rj)) - 1});
    }
    if (live.empty()) continue;
    // Acceptance of every window coordinate is a pure function of (i, j): recheck them all,
    // then replay Algorithm 1's offset-major loop sequentially.
    std::vector<int64_t> coords;
    std::unordered_map<int64_t, int32_t> slot;
    for (const Center& cd : live) {
      for (const auto& od : offs) {
        const int64_t i = cd.ci + od.first, j = cd.cj + od.second;
        if (i < 0 || i >= c->n1 || j < 0 || j >= c->n3) continue;
        const int64_t kk = key(i, j);
        if (inF.count(kk) || slot.count(kk)) continue;
        slot.emplace(kk, static_cast<int32_t>(coords.size() / 2));
        coords.push_back(i);
        coords.push_back(j);
      }
    }
    std::vector<double> gg, aa;
    std::vector<float> cc;
    FPSK_TRY(recheck_coords(c, A, B, Cf, coords, gg, aa, cc, st));
    n_rechecked += static_cast<int32_t>(coords.size() / 2);
    std::vector<char> alive(live.size(), 1);
    size_t nlive = live.size();
    for (const auto& od : offs) {
      if (nlive == 0) break;
      for (size_t u = 0; u < live.size(); ++u) {
        if (!alive[u]) continue;
        const int64_t i = live[u].ci + od.first, j = live[u].cj + od.second;
        if (i < 0 || i >= c->n1 || j < 0 || j >= c->n3) continue;
        const int64_t kk = key(i, j);
        if (inF.count(kk)) continue;
        const int32_t sl = slot.at(kk);
        const double diff = gg[sl] - static_cast<double>(cc[sl]);
        const double bound = c->p.c_valid * std::ldexp(1.0, -23) * aa[sl];
        if (std::fabs(diff) > bound) {
          F.push_back({i, j, diff, 0, t});
          inF.insert(kk);
          alive[u] = 0;
          --nlive;
        }
      }
    }
  }

  c->last_plan.m = c->m;
  c->last_plan.m_loc = plan.m_loc;
  c->last_plan.r = plan.r;
  c->last_plan.fallback = plan.fallback;
  c->last_plan.n_abs = static_cast<int32_t>(n_abs);
  c->last_plan.n_rechecked = n_rechecked;
  c->last_plan.sigma_hat = sigma;
  c->last_plan.rms_hat = rms;
  c->last_plan.B = plan.B;
  c->last_plan.tau = tau;

  *n_out = static_cast<int32_t>(F.size());
  const size_t nw = std::min<size_t>(F.size(), static_cast<size_t>(cap));
  for (size_t t = 0; t < nw; ++t) {
    out[t].i = F[t].i;
    out[t].j = F[t].j;
    out[t].delta = F[t].delta;
    out[t].absolute = F[t].absolute;
    out[t].round = F[t].round;
  }
  if (F.size() > static_cast<size_t>(cap)) {
    return fail(FPSK_ECAPACITY, "more fault records than capacity");
  }
  return FPSK_OK;
}

fpsketch_status fpsketch_stream_read(const void* src, int64_t bytes, uint32_t* d_out,
                                     int32_t grid, void* stream) {
  if (src == nullptr || d_out == nullptr || bytes < 0 || bytes % 16 != 0 || grid < 1 ||
      (reinterpret_cast<uintptr_t>(src) & 15u) != 0) {
    return fail(FPSK_EINVAL, "fpsketch_stream_read: bad argument");
  }
  FPSK_HIP(fpsk::launch_read(src, bytes, d_out, grid, static_cast<hipStream_t>(stream)));
  return FPSK_OK;
}

fpsketch_status fpsketch_stream_copy(const void* src, void* dst, int64_t bytes, int32_t grid,
                                     void* stream) {
  if (src == nullptr || dst == nullptr || bytes < 0 || bytes % 16 != 0 || grid < 1 ||
      ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15u) != 0) {
    return fail(FPSK_EINVAL, "fpsketch_stream_copy: bad argument");
  }
  FPSK_HIP(fpsk::launch_copy(src, dst, bytes, grid, static_cast<hipStream_t>(stream)));
  return FPSK_OK;
}

}  // extern "C"
