// gfx950 stream kernel of the FP-Sketch post hoc verifier: one pass over A, B and C forming
// the factors of Eq. 1 without forming AB: P = H1 A (row-bucket segmented reduction),
// Q = B H2^T (column-bucket fold of each row of B) and the bucket grid of C (row-bucket
// accumulation, then a column-bucket fold once per row bucket and tile); with moments, the
// weighted forms that give the first-moment sketches R and T (paper, Sec. III-B).  No atomics:
// every sum has a fixed order, so sketches are bit-reproducible.  Streaming sums accumulate in
// FP64.
#include "fpsk_block.h"

namespace fpsk {

// Work-group timeline of the stream kernel (diagnostic build only; the stamp is in
// fpsk_device.h): one record per work-group of the last stream launch, at its launch index.
#ifdef FPSK_WG_TIMELINE
static __device__ unsigned long long wg_timeline_stream[4 * kTimelineMax];
#define FPSK_WG_STAMP(type) const WgStamp wg_stamp_(wg_timeline_stream, blockIdx.x, type)
#else
#define FPSK_WG_STAMP(type)
#endif

// ----------------------------------------------------------------------------------------
// Row-bucket passes (A and C work-groups).  Wave w of a work-group takes rows w, w + 4, ... of
// the bucket's sorted row list.  The row entries of up to 64 of its rows arrive with one vector
// load and are broadcast with readlane, so a group of row loads issues back to back instead of
// waiting on an index load per row.

// Row entry (row | negative-sign bit) of this wave's r-th row in the current batch.
__device__ __forceinline__ int32_t row_entry(int32_t pe, int r) {
  return __builtin_amdgcn_readlane(pe, r);
}

// A row-bucket side: a matrix with rows of n2 halfs whose rows are hashed into buckets.  The A
// side (rows i of A, h1, v1, w_i) gives P and Pw; with B passed transposed (W = B^T, n3 x n2),
// the rows j of W with h2, v2, w_j give Q = (B H2^T)^T and Qw directly, in the same layout.
struct RowSide {
  const uint16_t* X;       // rows x n2 half bits
  const int32_t* perm;     // bucket lists (row | sign << 31), cap entries each
  int cap;
  double inv_l;            // 1 / 2^ceil(log2 rows)
  float* out;              // m x ldp
  float* outw;             // m x ldp (moments)
  float* maxslot;          // max |X| per work-group (A: maxpart, W: after the nA A entries)
};

__device__ __forceinline__ RowSide a_side(const StreamArgs& s) {
  return RowSide{s.A, s.perm, s.cap, s.inv_l1, s.P, s.Pw, s.maxpart};
}

__device__ __forceinline__ RowSide w_side(const StreamArgs& s) {
  return RowSide{s.B, s.perm2, s.cap2, s.inv_l3, s.Q, s.Qw, s.maxpart + s.nA};
}

// Row-bucket work-group: bucket a, column tile t.  out[a, tile] = sum over the bucket's rows of
// v(i) X[i, tile] (and outw with w_i).  Groups of 8 rows are summed in FP32 (their partial sums
// stay within a few units of the last place of the stored FP32 factor), groups in FP64; the 4
// waves are combined in fixed wave order.
template <int DT, bool MOM, bool VEC>
__device__ void a_unit(const StreamArgs& s, const RowSide& rs, int u, double* lds,
                       uint32_t* ldsu) {
  constexpr int U = 8;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int a = u / s.TA, t = u - a * s.TA;
  const int64_t col = static_cast<int64_t>(t) * kColTile + lane * 8;
  const bool lane_ok = col < s.n2;
  const int32_t* prow = rs.perm + static_cast<int64_t>(a) * rs.cap;
  double acc[8], accw[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    acc[k] = 0.0;
    accw[k] = 0.0;
  }
  uint32_t mx = 0;
  for (int base = w; base < rs.cap; base += 4 * 64) {
    const int32_t pe = base + 4 * lane < rs.cap ? prow[base + 4 * lane] : -1;
    const int nr = __popcll(__ballot(pe != -1));   // valid entries are a prefix of the lanes
    if (nr == 0) break;
    for (int r0 = 0; r0 < nr; r0 += U) {
      u32x4 v[U];
      float sg[U], sw[U];
#pragma unroll
      for (int q = 0; q < U; ++q) {
        const bool ok = r0 + q < nr;
        const int32_t e = row_entry(pe, ok ? r0 + q : 0);
        const int64_t row = e & 0x7fffffff;
        sg[q] = ok ? (e < 0 ? -1.0f : 1.0f) : 0.0f;
        sw[q] = MOM ? static_cast<float>(sg[q] * static_cast<double>(row + 1) * rs.inv_l) : 0.0f;
        if (VEC) {
          v[q] = load8h_sel(rs.X + row * s.n2 + col, ok && lane_ok, s.zero);
        } else {
          v[q] = ok ? load8h(rs.X + row * s.n2, col, s.n2, false) : u32x4{0u, 0u, 0u, 0u};
        }
      }
      float g32[8], gw32[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        g32[k] = 0.0f;
        gw32[k] = 0.0f;
      }
#pragma unroll
      for (int q = 0; q < U; ++q) {
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          const uint32_t wd = v[q][h];
          mx = absmax2(mx, wd);
          const float x0 = lo_half<DT>(wd), x1 = hi_half<DT>(wd);
          g32[2 * h] = fmaf(sg[q], x0, g32[2 * h]);
          g32[2 * h + 1] = fmaf(sg[q], x1, g32[2 * h + 1]);
          if (MOM) {
            gw32[2 * h] = fmaf(sw[q], x0, gw32[2 * h]);
            gw32[2 * h + 1] = fmaf(sw[q], x1, gw32[2 * h + 1]);
          }
        }
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        acc[k] += static_cast<double>(g32[k]);
        if (MOM) accw[k] += static_cast<double>(gw32[k]);
      }
    }
  }
  // Combine the 4 waves: layout [wave][k][lane].
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    lds[(w * 8 + k) * 64 + lane] = acc[k];
    if (MOM) lds[2048 + (w * 8 + k) * 64 + lane] = accw[k];
  }
  const float amax = block_absmax_half<DT>(mx, ldsu);   // contains __syncthreads
  for (int c = threadIdx.x; c < kColTile; c += kThreads) {
    const int ln = c >> 3, k = c & 7;
    const int64_t gc = static_cast<int64_t>(t) * kColTile + c;
    if (gc < s.n2) {
      double v = lds[k * 64 + ln] + lds[(8 + k) * 64 + ln];
      v += lds[(16 + k) * 64 + ln];
      v += lds[(24 + k) * 64 + ln];
      rs.out[static_cast<int64_t>(a) * s.ldp + gc] = static_cast<float>(v);
      if (MOM) {
        double vw = lds[2048 + k * 64 + ln] + lds[2048 + (8 + k) * 64 + ln];
        vw += lds[2048 + (16 + k) * 64 + ln];
        vw += lds[2048 + (24 + k) * 64 + ln];
        rs.outw[static_cast<int64_t>(a) * s.ldp + gc] = static_cast<float>(vw);
      }
    }
  }
  if (threadIdx.x == 0) rs.maxslot[u] = amax;
}

// Row-bucket work-group for small buckets (at most about 16 rows): bucket a, four column tiles,
// wave w taking tile 4 tq + w over all of the bucket's rows, so no combine across waves.  The
// same groups of 8 rows in FP32, then FP64, in list order.
template <int DT, bool MOM, bool VEC>
__device__ void a_unit_wt(const StreamArgs& s, const RowSide& rs, int u, uint32_t* ldsu) {
  constexpr int U = 8;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int tq = (s.TA + 3) / 4;
  const int a = u / tq, t = 4 * (u - a * tq) + w;
  const int64_t col = static_cast<int64_t>(t) * kColTile + lane * 8;
  const bool lane_ok = t < s.TA && col < s.n2;
  const int32_t* prow = rs.perm + static_cast<int64_t>(a) * rs.cap;
  double acc[8], accw[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    acc[k] = 0.0;
    accw[k] = 0.0;
  }
  uint32_t mx = 0;
  for (int base = 0; base < rs.cap; base += 64) {
    const int32_t pe = base + lane < rs.cap ? prow[base + lane] : -1;
    const int nr = __popcll(__ballot(pe != -1));   // valid entries are a prefix of the lanes
    if (nr == 0) break;
    for (int r0 = 0; r0 < nr; r0 += U) {
      u32x4 v[U];
      float sg[U], sw[U];
#pragma unroll
      for (int q = 0; q < U; ++q) {
        const bool ok = r0 + q < nr;
        const int32_t e = row_entry(pe, ok ? r0 + q : 0);
        const int64_t row = e & 0x7fffffff;
        sg[q] = ok ? (e < 0 ? -1.0f : 1.0f) : 0.0f;
        sw[q] = MOM ? static_cast<float>(sg[q] * static_cast<double>(row + 1) * rs.inv_l) : 0.0f;
        if (VEC) {
          v[q] = load8h_sel(rs.X + row * s.n2 + col, ok && lane_ok, s.zero);
        } else {
          v[q] = ok && lane_ok ? load8h(rs.X + row * s.n2, col, s.n2, false)
                               : u32x4{0u, 0u, 0u, 0u};
        }
      }
      float g32[8], gw32[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        g32[k] = 0.0f;
        gw32[k] = 0.0f;
      }
#pragma unroll
      for (int q = 0; q < U; ++q) {
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          const uint32_t wd = v[q][h];
          mx = absmax2(mx, wd);
          const float x0 = lo_half<DT>(wd), x1 = hi_half<DT>(wd);
          g32[2 * h] = fmaf(sg[q], x0, g32[2 * h]);
          g32[2 * h + 1] = fmaf(sg[q], x1, g32[2 * h + 1]);
          if (MOM) {
            gw32[2 * h] = fmaf(sw[q], x0, gw32[2 * h]);
            gw32[2 * h + 1] = fmaf(sw[q], x1, gw32[2 * h + 1]);
          }
        }
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        acc[k] += static_cast<double>(g32[k]);
        if (MOM) accw[k] += static_cast<double>(gw32[k]);
      }
    }
  }
  if (lane_ok) {
    float* o = rs.out + static_cast<int64_t>(a) * s.ldp + col;
    float* ow = MOM ? rs.outw + static_cast<int64_t>(a) * s.ldp + col : nullptr;
    if (col + 8 <= s.n2) {
      // the row starts on a 256-byte boundary and col is a multiple of 8
      reinterpret_cast<f32x4*>(o)[0] = f32x4{static_cast<float>(acc[0]), static_cast<float>(acc[1]),
                                             static_cast<float>(acc[2]), static_cast<float>(acc[3])};
      reinterpret_cast<f32x4*>(o)[1] = f32x4{static_cast<float>(acc[4]), static_cast<float>(acc[5]),
                                             static_cast<float>(acc[6]), static_cast<float>(acc[7])};
      if (MOM) {
        reinterpret_cast<f32x4*>(ow)[0] =
            f32x4{static_cast<float>(accw[0]), static_cast<float>(accw[1]),
                  static_cast<float>(accw[2]), static_cast<float>(accw[3])};
        reinterpret_cast<f32x4*>(ow)[1] =
            f32x4{static_cast<float>(accw[4]), static_cast<float>(accw[5]),
                  static_cast<float>(accw[6]), static_cast<float>(accw[7])};
      }
    } else {
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        if (col + k < s.n2) {
          o[k] = static_cast<float>(acc[k]);
          if (MOM) ow[k] = static_cast<float>(accw[k]);
        }
      }
    }
  }
  const float amax = block_absmax_half<DT>(mx, ldsu);   // contains __syncthreads
  if (threadIdx.x == 0) rs.maxslot[u] = amax;
}

// Row-bucket unit of either kind.
template <int DT, bool MOM, bool VEC>
__device__ __forceinline__ void row_unit(const StreamArgs& s, const RowSide& rs, bool wt, int u,
                                         double* lds, uint32_t* ldsu) {
  if (wt) {
    a_unit_wt<DT, MOM, VEC>(s, rs, u, ldsu);
  } else {
    a_unit<DT, MOM, VEC>(s, rs, u, lds, ldsu);
  }
}

// ----------------------------------------------------------------------------------------
// B work-group: RB consecutive rows of B, all columns, in chunks of CW = kBChunkHalfs / RB
// columns.  Per chunk, every thread issues its 8 x 16-byte loads of B and its share of the
// chunk's bucket-sorted column list at once; B is then staged column-major ([column][RB rows])
// in LDS and thread (row group rg, bucket b) folds the chunk's columns of bucket b for its
// RB / NG rows: Q[k, b] = sum v2(j) B[k, j].

template <int RB>
__device__ __forceinline__ uint32_t pick_half(uint32_t wa, uint32_t wb, int odd) {
  return odd ? ((wa >> 16) | (wb & 0xffff0000u)) : ((wa & 0xffffu) | (wb << 16));
}

// Write the 8 columns held by one thread (RB rows x 8 columns) column-major into LDS.  Column
// 8 g8 + e goes to slot e (W / 8) + g8 of a chunk of W = kBChunkHalfs / RB columns: one base
// address (dst = slot g8) plus the constant offset e * kBChunkHalfs / 8 halfs per column, and
// the lanes of a wave write consecutive slots.
template <int RB>
__device__ __forceinline__ void store_cols(uint16_t* dst, const u32x4* v) {
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    uint16_t* d = dst + e * (kBChunkHalfs / 8);
    if constexpr (RB == 1) {
      d[0] = static_cast<uint16_t>(v[0][e >> 1] >> (16 * (e & 1)));
    } else if constexpr (RB == 2) {
      *reinterpret_cast<uint32_t*>(d) = pick_half<RB>(v[0][e >> 1], v[1][e >> 1], e & 1);
    } else if constexpr (RB == 4) {
      u32x2 o;
      o[0] = pick_half<RB>(v[0][e >> 1], v[1][e >> 1], e & 1);
      o[1] = pick_half<RB>(v[2][e >> 1], v[3][e >> 1], e & 1);
      *reinterpret_cast<u32x2*>(d) = o;
    } else {
      u32x4 o;
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) o[rr] = pick_half<RB>(v[2 * rr][e >> 1], v[2 * rr + 1][e >> 1], e & 1);
      *reinterpret_cast<u32x4*>(d) = o;
    }
  }
}

// Staged slot of column cc of a chunk of CW columns (CW itself is the zero sentinel slot).
template <int CW>
__device__ __forceinline__ int col_slot(int cc) {
  return cc < CW ? (cc & 7) * (CW / 8) + (cc >> 3) : CW;
}

// RBG consecutive halfs of one staged column.
template <int DT, int RBG>
__device__ __forceinline__ void load_col(const uint16_t* src, float* x) {
  if constexpr (RBG == 1) {
    x[0] = half_bits_to_float<DT>(*src);
  } else if constexpr (RBG == 2) {
    const uint32_t w = *reinterpret_cast<const uint32_t*>(src);
    x[0] = lo_half<DT>(w);
    x[1] = hi_half<DT>(w);
  } else if constexpr (RBG == 4) {
    const u32x2 w = *reinterpret_cast<const u32x2*>(src);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      x[2 * h] = lo_half<DT>(w[h]);
      x[2 * h + 1] = hi_half<DT>(w[h]);
    }
  } else {
    const u32x4 w = *reinterpret_cast<const u32x4*>(src);
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      x[2 * h] = lo_half<DT>(w[h]);
      x[2 * h + 1] = hi_half<DT>(w[h]);
    }
  }
}

// Loads of one B chunk in flight: 8 x 16 bytes of B, the sign bits of the thread's columns,
// the chunk's staged column list and this thread's segment bounds.
template <int RB, int G, int NT>
struct BChunk {
  static constexpr int NV = kBChunkHalfs / 8 / kThreads;
  static constexpr int NI = NV / RB;
  u32x4 v[NV];
  u32x4 tv[NT];
  uint32_t sb[NI];
  int qb[G], qe[G];
};

// The block of B rows that B work-group u takes.  A 4-row work-group writes a 16-byte piece of
// every Q row; the 8 work-groups whose pieces fill one 128-byte line run on one XCD, one after
// another, so that the line is whole in that XCD's L2 before it is written back.  Launch index i
// runs on XCD i mod 8, so the units of one XCD are u, u + 8, u + 16, ...: unit u takes block
// 64 (u / 64) + 8 (u mod 8) + (u / 8) mod 8 (whole groups of 64 units; the rest keep theirs).
template <int RB>
__device__ __forceinline__ int b_block(int u, int nB) {
  if (RB != 4 || u >= nB / 64 * 64) return u;
  return (u & ~63) | ((u & 7) << 3) | ((u >> 3) & 7);
}

template <int DT, bool MOM, int RB, int G, int NG, bool VEC>
__device__ void b_unit(const StreamArgs& s, int u, uint16_t* L, uint16_t* tabL, uint32_t* ldsu) {
  constexpr int CW = kBChunkHalfs / RB;      // columns per chunk
  constexpr int RBG = RB / NG;               // rows per fold group
  constexpr int SLOTS = kThreads / NG;       // bucket slots per fold group
  constexpr int PADG = (RB == 8 && G == 1) ? 8 : 1; // bucket segments padded to this multiple
  constexpr int NT = PADG == 8 ? 2 : (CW / 8 / kThreads > 0 ? CW / 8 / kThreads : 1);
  // Group fold (probe, 8 rows, m <= 256): thread t sums the 8 columns of entry groups t and
  // t + 256 of the chunk's sorted list (each group lies in one bucket, as segments are padded
  // to whole groups) over all 8 rows with one 16-byte LDS read per column; thread (b, r) then
  // adds the group partials of bucket b, row r in FP64.
  constexpr bool GF = !MOM && PADG == 8;
  constexpr int GFP = 8 / NG;                // (bucket, row) pairs per thread: 8 m <= 2048 / NG
  double qacc[GF ? GFP : 1];
#pragma unroll
  for (int i = 0; i < (GF ? GFP : 1); ++i) qacc[i] = 0.0;
  using Chunk = BChunk<RB, G, NT>;
  constexpr int NI = Chunk::NI;
  static_assert(Chunk::NV == 8, "each thread stages 64 halfs of B per chunk");
  const int m = s.m;
  const int stride = s.btab_stride;
  const int rg = threadIdx.x / SLOTS, bslot = threadIdx.x - rg * SLOTS;
  const int64_t k0 = static_cast<int64_t>(b_block<RB>(u, s.nB)) * RB;
  double acc[G][RBG], accw[G][RBG];
#pragma unroll
  for (int g = 0; g < G; ++g) {
#pragma unroll
    for (int r = 0; r < RBG; ++r) {
      acc[g][r] = 0.0;
      accw[g][r] = 0.0;
    }
  }
  if (threadIdx.x < RB) L[CW * RB + threadIdx.x] = 0;   // zero sentinel column
  uint32_t mx = 0;

  // Every load of chunk c, unconditionally (a chunk past the end reads the zero buffer).
  auto issue = [&](Chunk& ch, int c) {
    const bool live = c < s.TB;
    const int64_t cbase = static_cast<int64_t>(c) * CW;
#pragma unroll
    for (int it = 0; it < NI; ++it) {
      const int g8 = threadIdx.x + kThreads * it;
      const int64_t col = cbase + static_cast<int64_t>(g8) * 8;
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        const bool ok = live && k0 + r < s.n2 && col < s.n3;
        if (VEC) {
          ch.v[it * RB + r] = load8h_sel(s.B + (k0 + r) * s.n3 + col, ok, s.zero);
        } else {
          ch.v[it * RB + r] = ok ? load8h(s.B + (k0 + r) * s.n3, col, s.n3, false)
                                 : u32x4{0u, 0u, 0u, 0u};
        }
      }
      const uint8_t* sp = live ? s.bsign + cbase / 8 + g8 : static_cast<const uint8_t*>(s.zero);
      ch.sb[it] = *sp;
    }
    const uint16_t* btab = s.btab + static_cast<int64_t>(live ? c : 0) * stride;
#pragma unroll
    for (int it = 0; it < NT; ++it) {
      const int o = (threadIdx.x + kThreads * it) * 8;
      const u32x4* tp = (live && o < stride) ? reinterpret_cast<const u32x4*>(btab + o)
                                             : static_cast<const u32x4*>(s.zero);
      ch.tv[it] = *tp;
    }
    const int32_t* boff = s.boff + static_cast<int64_t>(live ? c : 0) * (m + 1);
    if constexpr (GF) {
      // segment starts m + 1 <= 257: entries t and t + 256, staged in LDS after the list
      const int t = threadIdx.x;
      const int32_t* p0 = (live && t <= m) ? boff + t : static_cast<const int32_t*>(s.zero);
      const int32_t* p1 = (live && t + kThreads <= m) ? boff + t + kThreads
                                                      : static_cast<const int32_t*>(s.zero);
      ch.qb[0] = *p0;
      ch.qe[0] = *p1;
    } else {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const int b = bslot + SLOTS * g;
        const int32_t* bp = (live && b < m) ? boff + b : static_cast<const int32_t*>(s.zero);
        ch.qb[g] = bp[0];
        ch.qe[g] = bp[1];
      }
    }
  };

  // Stage chunk c: signs v2(j) applied to the halves, columns and the sorted list into LDS.
  auto stage = [&](Chunk& ch) {
#pragma unroll
    for (int it = 0; it < NI; ++it) {
      const int g8 = threadIdx.x + kThreads * it;
      u32x4 smask;
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        smask[h] = (((ch.sb[it] >> (2 * h)) & 1u) << 15) | (((ch.sb[it] >> (2 * h + 1)) & 1u) << 31);
      }
#pragma unroll
      for (int r = 0; r < RB; ++r) {
#pragma unroll
        for (int h = 0; h < 4; ++h) mx = absmax2(mx, ch.v[it * RB + r][h]);
        ch.v[it * RB + r] ^= smask;
      }
      store_cols<RB>(L + static_cast<int64_t>(g8) * RB, ch.v + it * RB);
    }
#pragma unroll
    for (int it = 0; it < NT; ++it) {
      const int o = (threadIdx.x + kThreads * it) * 8;
      if (o < stride) *reinterpret_cast<u32x4*>(tabL + o) = ch.tv[it];
    }
    if constexpr (GF) {
      int32_t* boffL = reinterpret_cast<int32_t*>(tabL + stride);
      const int t = threadIdx.x;
      if (t <= m) boffL[t] = ch.qb[0];
      if (t + kThreads <= m) boffL[t + kThreads] = ch.qe[0];
    }
    __syncthreads();
  };

  // Fold the staged chunk c into the bucket sums; qb, qe are this thread's segment bounds.
  auto fold = [&](int c, const int* qb, const int* qe) {
    const int64_t cbase = static_cast<int64_t>(c) * CW;
    (void)cbase;
    if constexpr (GF) {
      const int32_t* boffL = reinterpret_cast<const int32_t*>(tabL + stride);
      const int ngroups = boffL[m] >> 3;
      float part[2][8];
      // FP16: x * one + part converts and adds in one instruction (v_fma_mix_f32) without a
      // temporary; `one` is opaque so the multiply by 1 is not folded away (exact either way)
      float one = 1.0f;
      asm volatile("" : "+v"(one));
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int grp = threadIdx.x + kThreads * h;
        const bool gok = grp < ngroups;
#pragma unroll
        for (int r = 0; r < 8; ++r) part[h][r] = 0.0f;
        if (h == 1 && ngroups <= kThreads) break;   // uniform: no second groups
        // a missing group reads the zero sentinel column
        const u32x4 tw = *reinterpret_cast<const u32x4*>(tabL + 8 * (gok ? grp : 0));
#pragma unroll
        for (int z0 = 0; z0 < 8; z0 += 4) {
          u32x4 cv[4];
#pragma unroll
          for (int z = 0; z < 4; ++z) {
            const int zz = z0 + z;
            const int e = gok ? static_cast<int>((tw[zz >> 1] >> (16 * (zz & 1))) & 0xffffu) : CW;
            cv[z] = *reinterpret_cast<const u32x4*>(L + e * RB);
          }
#pragma unroll
          for (int z = 0; z < 4; ++z)
#pragma unroll
            for (int w2 = 0; w2 < 4; ++w2) {
              if constexpr (DT == 0) {
                part[h][2 * w2] = __builtin_fmaf(lo_half<DT>(cv[z][w2]), one, part[h][2 * w2]);
                part[h][2 * w2 + 1] =
                    __builtin_fmaf(hi_half<DT>(cv[z][w2]), one, part[h][2 * w2 + 1]);
              } else {
                part[h][2 * w2] += lo_half<DT>(cv[z][w2]);
                part[h][2 * w2 + 1] += hi_half<DT>(cv[z][w2]);
              }
            }
        }
      }
      __syncthreads();
      // group partials [group][row] over the staged data (the zero column lies beyond them)
      float* PL = reinterpret_cast<float*>(L);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int grp = threadIdx.x + kThreads * h;
        if (grp < ngroups) {
          *reinterpret_cast<f32x4*>(PL + grp * 8) =
              f32x4{part[h][0], part[h][1], part[h][2], part[h][3]};
          *reinterpret_cast<f32x4*>(PL + grp * 8 + 4) =
              f32x4{part[h][4], part[h][5], part[h][6], part[h][7]};
        }
      }
      __syncthreads();
#pragma unroll
      for (int i = 0; i < GFP; ++i) {
        const int p = threadIdx.x + kThreads * i;
        if (p < 8 * m) {
          const int b = p >> 3, r = p & 7;
          const int g1 = boffL[b + 1] >> 3;
          double sum = 0.0;
          for (int g = boffL[b] >> 3; g < g1; ++g) sum += static_cast<double>(PL[g * 8 + r]);
          qacc[i] += sum;
        }
      }
    }
#pragma unroll
    for (int g = 0; g < (GF ? 0 : G); ++g) {
      if constexpr (PADG == 8) {
        // segments are whole multiples of 8 entries (sentinels read the zero slot): 8 list
        // entries with one LDS read, their 8 columns summed in FP32, then added in FP64
        for (int q = qb[g]; q < qe[g]; q += 8) {
          const u32x4 tw = *reinterpret_cast<const u32x4*>(tabL + q);
          float part[RBG], partw[RBG];
#pragma unroll
          for (int r = 0; r < RBG; ++r) {
            part[r] = 0.0f;
            partw[r] = 0.0f;
          }
#pragma unroll
          for (int z = 0; z < 8; ++z) {
            const int e = static_cast<int>((tw[z >> 1] >> (16 * (z & 1))) & 0xffffu);
            float x[RBG];
            if (MOM) {
              // MOM tables hold column offsets: slot swizzle and weight w_j per column
              load_col<DT, RBG>(L + col_slot<CW>(e) * RB + rg * RBG, x);
              const float wj = static_cast<float>(static_cast<double>(cbase + e + 1) * s.inv_l3);
#pragma unroll
              for (int r = 0; r < RBG; ++r) partw[r] = fmaf(wj, x[r], partw[r]);
            } else {
              load_col<DT, RBG>(L + e * RB + rg * RBG, x);   // pre-swizzled slot
            }
#pragma unroll
            for (int r = 0; r < RBG; ++r) part[r] += x[r];
          }
#pragma unroll
          for (int r = 0; r < RBG; ++r) {
            acc[g][r] += static_cast<double>(part[r]);
            if (MOM) accw[g][r] += static_cast<double>(partw[r]);
          }
        }
      } else {
        constexpr int UN = 2;
        // Unpadded segments, two list entries per step so that their LDS reads overlap (four
        // measured no faster and spill under prefetch); an entry past the segment's end reads
        // the zero column (slot CW), which adds +0.
        for (int q = qb[g]; q < qe[g]; q += UN) {
          int e[UN];
#pragma unroll
          for (int z = 0; z < UN; ++z) e[z] = q + z < qe[g] ? static_cast<int>(tabL[q + z]) : -1;
          float x[UN][RBG];
#pragma unroll
          for (int z = 0; z < UN; ++z) {
            const int sl = e[z] < 0 ? CW : (MOM ? col_slot<CW>(e[z]) : e[z]);
            load_col<DT, RBG>(L + sl * RB + rg * RBG, x[z]);
          }
#pragma unroll
          for (int z = 0; z < UN; ++z) {
            const double wj = MOM ? static_cast<double>(cbase + e[z] + 1) * s.inv_l3 : 0.0;
#pragma unroll
            for (int r = 0; r < RBG; ++r) {
              const double d = static_cast<double>(x[z][r]);
              acc[g][r] += d;
              if (MOM) accw[g][r] = fma(d, wj, accw[g][r]);
            }
          }
        }
      }
    }
  };

  // 4-row probe work-groups (m = 513 to 1024) fold chunk c while the loads of chunk c + 1 are
  // in flight (the list bounds are copied out of the chunk registers first); their 3 resident
  // work-groups per CU leave the registers for it.  Elsewhere it would spill.
  constexpr bool PF = !GF && !MOM && RB == 4;
  if constexpr (PF) {
    Chunk ch;
    issue(ch, 0);
    for (int c = 0; c < s.TB; ++c) {
      stage(ch);
      int qb[G], qe[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        qb[g] = ch.qb[g];
        qe[g] = ch.qe[g];
      }
      if (c + 1 < s.TB) issue(ch, c + 1);
      fold(c, qb, qe);
      __syncthreads();
    }
  } else {
    for (int c = 0; c < s.TB; ++c) {
      Chunk ch;
      issue(ch, c);
      stage(ch);
      fold(c, ch.qb, ch.qe);
      __syncthreads();
    }
  }
  if constexpr (GF) {
#pragma unroll
    for (int i = 0; i < GFP; ++i) {
      const int p = threadIdx.x + kThreads * i;
      const int64_t k = k0 + (p & 7);
      if (p < 8 * m && k < s.n2) {
        s.Q[static_cast<int64_t>(p >> 3) * s.ldp + k] = static_cast<float>(qacc[i]);
      }
    }
  }
#pragma unroll
  for (int g = 0; g < (GF ? 0 : G); ++g) {
    const int b = bslot + SLOTS * g;
    const int64_t kg = k0 + rg * RBG;        // this thread's first row
    if (RBG == 4 && s.Qk == nullptr && b < m && kg + 4 <= s.n2) {
      // one 16-byte piece per Q row (kg is a multiple of 4; rows start on 256-byte boundaries)
      const int64_t o = static_cast<int64_t>(b) * s.ldp + kg;
      *reinterpret_cast<f32x4*>(s.Q + o) =
          f32x4{static_cast<float>(acc[g][0]), static_cast<float>(acc[g][1]),
                static_cast<float>(acc[g][2]), static_cast<float>(acc[g][3])};
      if (MOM) {
        *reinterpret_cast<f32x4*>(s.Qw + o) =
            f32x4{static_cast<float>(accw[g][0]), static_cast<float>(accw[g][1]),
                  static_cast<float>(accw[g][2]), static_cast<float>(accw[g][3])};
      }
    } else if (b < m) {
#pragma unroll
      for (int r = 0; r < RBG; ++r) {
        const int64_t k = k0 + rg * RBG + r;
        if (k < s.n2) {
          if (s.Qk != nullptr) {
            // k-major rows (consecutive buckets of a wave write consecutive floats)
            s.Qk[k * s.mq + b] = static_cast<float>(acc[g][r]);
            if (MOM) s.Qwk[k * s.mq + b] = static_cast<float>(accw[g][r]);
          } else {
            s.Q[static_cast<int64_t>(b) * s.ldp + k] = static_cast<float>(acc[g][r]);
            if (MOM) s.Qw[static_cast<int64_t>(b) * s.ldp + k] = static_cast<float>(accw[g][r]);
          }
        }
      }
    }
  }
  const float bmax = block_absmax_half<DT>(mx, ldsu);
  if (threadIdx.x == 0) s.maxpart[s.nA + u] = bmax;
}

// B work-group of the probe at m <= 512: 4 consecutive rows of B over all columns, in chunks
// of 4096 columns (one chunk when n3 <= 4096) whose loads are all issued at once, so a
// work-group waits for memory once per chunk.  The columns are staged column-major in LDS
// ([slot][4 rows], 8 bytes each, signs v2(j) applied).  The chunk's bucket-sorted list has its
// segments padded to whole groups of 8 (at most 4096 + 7m entries: 3 groups per thread up to
// m = 256, 4 up to m = 512) and is read from global memory, which keeps the work-group's LDS
// small; thread t sums the 8 columns of its groups t, t + 256, ... in FP32, the group partials
// replace the staged data, and thread t then adds the partials of buckets t, t + 256, ... (G of
// them) in FP64.  At the end each bucket's Q[b, k0 .. k0 + 3] is one 16-byte store.
// ROT (the instances with one-tile-per-wave C work-groups): with rot_b the chunks are taken
// from (row block mod TB) on, wrapping around, so that the work-groups in flight read
// different column ranges of their rows (2048 x 8192 x 8192 at m = 64: stream pass 43.8 ->
// 42.2 us).  The other instance, the 4096^3 one among them, is compiled without it: the index
// arithmetic cost it 0.1 us per pass with a single chunk.
template <int DT, bool VEC, int G, bool ROT>
__device__ void b_unit_probe4(const StreamArgs& s, int u, uint16_t* L, uint32_t* ldsu) {
  constexpr int RB = 4;
  constexpr int CW = kBChunkHalfs / RB;          // 4096 columns per chunk
  constexpr int NI = CW / 8 / kThreads;          // groups of 8 columns a thread loads
  constexpr int NGT = G == 1 ? 3 : 4;            // sorted-list groups a thread folds
  constexpr int NBO = G + 1;                     // segment starts a thread stages
  static_assert(CW == 4096 && NI == 2, "the slot format and the sentinel assume 4096 columns");
  static_assert(8 * NGT * kThreads >= CW + 7 * 256 * G, "the padded list fits the groups");
  static_assert(NGT * kThreads * RB * 4 <= CW * RB * 2, "the group partials fit the staging");
  const int m = s.m;
  const int stride = s.btab_stride;              // multiple of 8, at most 8 NGT kThreads
  const int t = threadIdx.x;
  const int rbk = b_block<RB>(u, s.nB);
  const int64_t k0 = static_cast<int64_t>(rbk) * RB;
  int32_t* boffL = reinterpret_cast<int32_t*>(L + CW * RB + 8);   // after the zero column
  float* PL = reinterpret_cast<float*>(L);       // group partials, over the staged data
  if (t < RB) L[CW * RB + t] = 0;                // zero sentinel column (slot CW)
  double q[G][RB];
#pragma unroll
  for (int g = 0; g < G; ++g)
#pragma unroll
    for (int r = 0; r < RB; ++r) q[g][r] = 0.0;
  uint32_t mx = 0;
  const u32x4 sent = {0x10001000u, 0x10001000u, 0x10001000u, 0x10001000u};   // 8 x slot CW
  const int rot = (ROT && s.rot_b) ? rbk % s.TB : 0;
  for (int i = 0; i < s.TB; ++i) {
    const int c = i + rot < s.TB ? i + rot : i + rot - s.TB;   // chunk (rot + i) mod TB
    const int64_t cbase = static_cast<int64_t>(c) * CW;
    u32x4 v[NI][RB];
    uint32_t sb[NI];
    u32x4 tw[NGT];
#pragma unroll
    for (int it = 0; it < NI; ++it) {
      const int g8 = t + kThreads * it;
      const int64_t col = cbase + static_cast<int64_t>(g8) * 8;
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        const bool ok = k0 + r < s.n2 && col < s.n3;
        if (VEC) {
          v[it][r] = load8h_sel(s.B + (k0 + r) * s.n3 + col, ok, s.zero);
        } else {
          v[it][r] = ok ? load8h(s.B + (k0 + r) * s.n3, col, s.n3, false)
                        : u32x4{0u, 0u, 0u, 0u};
        }
      }
      sb[it] = s.bsign[cbase / 8 + g8];          // the sign bits cover whole chunks
    }
    const uint16_t* btab = s.btab + static_cast<int64_t>(c) * stride;
#pragma unroll
    for (int h = 0; h < NGT; ++h) {
      const int o = 8 * (t + kThreads * h);
      tw[h] = o < stride ? *reinterpret_cast<const u32x4*>(btab + o) : sent;
    }
    int32_t bo[NBO];
#pragma unroll
    for (int j = 0; j < NBO; ++j) {
      const int b = t + kThreads * j;
      bo[j] = b <= m ? s.boff[static_cast<int64_t>(c) * (m + 1) + b] : 0;
    }
#pragma unroll
    for (int it = 0; it < NI; ++it) {
      const int g8 = t + kThreads * it;
      u32x4 smask;
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        smask[h] = (((sb[it] >> (2 * h)) & 1u) << 15) | (((sb[it] >> (2 * h + 1)) & 1u) << 31);
      }
#pragma unroll
      for (int r = 0; r < RB; ++r) {
#pragma unroll
        for (int h = 0; h < 4; ++h) mx = absmax2(mx, v[it][r][h]);
        v[it][r] ^= smask;
      }
      store_cols<RB>(L + static_cast<int64_t>(g8) * RB, v[it]);
    }
#pragma unroll
    for (int j = 0; j < NBO; ++j) {
      if (t + kThreads * j <= m) boffL[t + kThreads * j] = bo[j];
    }
    __syncthreads();
    float part[NGT][RB];
#pragma unroll
    for (int h = 0; h < NGT; ++h) {
#pragma unroll
      for (int r = 0; r < RB; ++r) part[h][r] = 0.0f;
#pragma unroll
      for (int z = 0; z < 8; ++z) {
        const int e = static_cast<int>((tw[h][z >> 1] >> (16 * (z & 1))) & 0xffffu);
        const u32x2 w = *reinterpret_cast<const u32x2*>(L + e * RB);
        part[h][0] += lo_half<DT>(w[0]);
        part[h][1] += hi_half<DT>(w[0]);
        part[h][2] += lo_half<DT>(w[1]);
        part[h][3] += hi_half<DT>(w[1]);
      }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < NGT; ++h) {
      const int grp = t + kThreads * h;
      if (8 * grp < stride) {
        *reinterpret_cast<f32x4*>(PL + 4 * grp) =
            f32x4{part[h][0], part[h][1], part[h][2], part[h][3]};
      }
    }
    __syncthreads();
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int b = t + kThreads * g;
      if (b < m) {
        const int g1 = boffL[b + 1] >> 3;
        for (int gg = boffL[b] >> 3; gg < g1; ++gg) {
          const f32x4 p = *reinterpret_cast<const f32x4*>(PL + 4 * gg);
#pragma unroll
          for (int r = 0; r < RB; ++r) q[g][r] += static_cast<double>(p[r]);
        }
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int b = t + kThreads * g;
    if (b < m) {
      float* qo = s.Q + static_cast<int64_t>(b) * s.ldp + k0;
      if (k0 + RB <= s.n2) {
        // k0 is a multiple of 4 and the rows start on 256-byte boundaries
        *reinterpret_cast<f32x4*>(qo) =
            f32x4{static_cast<float>(q[g][0]), static_cast<float>(q[g][1]),
                  static_cast<float>(q[g][2]), static_cast<float>(q[g][3])};
      } else {
#pragma unroll
        for (int r = 0; r < RB; ++r) {
          if (k0 + r < s.n2) qo[r] = static_cast<float>(q[g][r]);
        }
      }
    }
  }
  const float bmax = block_absmax_half<DT>(mx, ldsu);
  if (t == 0) s.maxpart[s.nA + u] = bmax;
}

// ----------------------------------------------------------------------------------------
// C work-group: row bucket a, a group of tg column tiles.  Per tile, the 4 waves accumulate
// v1(i) C[i, tile] (and w_i v1(i) C) over the bucket's rows in FP64, combine in fixed order,
// and thread b folds the tile's columns of bucket b from the tile's bucket-sorted column list
// (staged in LDS with the row loads): S_C[a, b] += sum v2(j) colsum[j] (T_C with w_j, R_C from
// the row-weighted sums).  One partial per tile group.

template <bool MOM, int G, bool VEC>
__device__ void c_unit(const StreamArgs& s, int u, double* lds, uint16_t* tabL) {
  // rows in flight per wave: 4 at m > 2048 (a few rows per bucket, and the fold's 16 buckets
  // per thread need the registers)
  constexpr int U = G >= 16 ? 4 : 8;
  constexpr int PADG = G == 1 ? 8 : 1;       // bucket segments padded to this multiple
  const int m = s.m;
  const int a = u / s.npc, gi = u - a * s.npc;
  const int t0 = gi * s.tg;
  const int t1 = (t0 + s.tg < s.TC) ? t0 + s.tg : s.TC;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int32_t* prow = s.perm + static_cast<int64_t>(a) * s.cap;
  const bool patched = s.patch_rowptr != nullptr;
  double* comb = lds;                          // [2][4][8][64]
  double* cs = lds + (MOM ? 4096 : 2048);      // column sums [513] (+ weighted at 520)
  double fS[G], fR[G], fT[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    fS[g] = 0.0;
    fR[g] = 0.0;
    fT[g] = 0.0;
  }
  for (int t = t0; t < t1; ++t) {
    const int64_t col = static_cast<int64_t>(t) * kColTile + lane * 8;
    const bool lane_ok = col < s.n3;
    // fold tables of this tile, loaded with the first rows
    const int stride = s.ctab_stride;
    const uint16_t* ctab = s.ctab + static_cast<int64_t>(t) * stride;
    u32x4 tv[2];
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int o = (threadIdx.x + kThreads * it) * 8;
      tv[it] = o < stride ? *reinterpret_cast<const u32x4*>(ctab + o) : u32x4{0u, 0u, 0u, 0u};
    }
    const int32_t* coff = s.coff + static_cast<int64_t>(t) * (m + 1);
    // (the thread index is opaque here, so the compiler does not hoist the per-thread address
    // out of the tile loop: that 64-bit pointer was the instance's only spill, and its reload
    // waited on the tile's list load before the segment starts and rows could be issued)
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    int qb[G], qe[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int b = tid + kThreads * g;
      qb[g] = b < m ? coff[b] : 0;
      qe[g] = b < m ? coff[b + 1] : 0;
    }
    double acc[8], accw[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      acc[k] = 0.0;
      accw[k] = 0.0;
    }
    for (int base = w; base < s.cap; base += 4 * 64) {
      const int32_t pe = base + 4 * lane < s.cap ? prow[base + 4 * lane] : -1;
      const int nr = __popcll(__ballot(pe != -1));
      if (nr == 0) break;
      for (int r0 = 0; r0 < nr; r0 += U) {
        f32x4 v0[U], v1[U];
        double sg[U], sw[U];
        int64_t rows[U];
#pragma unroll
        for (int q = 0; q < U; ++q) {
          const bool ok = r0 + q < nr;
          const int32_t e = row_entry(pe, ok ? r0 + q : 0);
          const int64_t row = e & 0x7fffffff;
          rows[q] = row;
          sg[q] = ok ? (e < 0 ? -1.0 : 1.0) : 0.0;
          sw[q] = MOM ? sg[q] * static_cast<double>(row + 1) * s.inv_l1 : 0.0;
          if (VEC) {
            load8f_sel(s.C + row * s.n3 + col, ok && lane_ok, s.zero, v0[q], v1[q]);
          } else if (ok) {
            load8f(s.C + row * s.n3, col, s.n3, false, v0[q], v1[q]);
          } else {
            v0[q] = f32x4{0.f, 0.f, 0.f, 0.f};
            v1[q] = f32x4{0.f, 0.f, 0.f, 0.f};
          }
        }
        if (patched) {
#pragma unroll
          for (int q = 0; q < U; ++q) {
            if (r0 + q < nr) apply_patches(s, rows[q], col, v0[q], v1[q]);
          }
        }
#pragma unroll
        for (int q = 0; q < U; ++q) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const double x = static_cast<double>(e < 4 ? v0[q][e] : v1[q][e - 4]);
            acc[e] = fma(x, sg[q], acc[e]);
            if (MOM) accw[e] = fma(x, sw[q], accw[e]);
          }
        }
      }
    }
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      const int o = (threadIdx.x + kThreads * it) * 8;
      if (o < stride) *reinterpret_cast<u32x4*>(tabL + o) = tv[it];
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      comb[(w * 8 + k) * 64 + lane] = acc[k];
      if (MOM) comb[2048 + (w * 8 + k) * 64 + lane] = accw[k];
    }
    __syncthreads();
    for (int c = threadIdx.x; c < kColTile; c += kThreads) {
      const int ln = c >> 3, k = c & 7;
      double v = comb[k * 64 + ln] + comb[(8 + k) * 64 + ln];
      v += comb[(16 + k) * 64 + ln];
      v += comb[(24 + k) * 64 + ln];
      cs[c] = v;
      if (MOM) {
        double vw = comb[2048 + k * 64 + ln] + comb[2048 + (8 + k) * 64 + ln];
        vw += comb[2048 + (16 + k) * 64 + ln];
        vw += comb[2048 + (24 + k) * 64 + ln];
        cs[520 + c] = vw;
      }
    }
    if (threadIdx.x == 0) {
      cs[kColTile] = 0.0;            // zero sentinel column
      if (MOM) cs[520 + kColTile] = 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int g = 0; g < G; ++g) {
      for (int q = qb[g]; q < qe[g]; q += PADG) {
        uint32_t ez[PADG];
        if constexpr (PADG == 8) {
          const u32x4 tw = *reinterpret_cast<const u32x4*>(tabL + q);
#pragma unroll
          for (int z = 0; z < 8; ++z) ez[z] = (tw[z >> 1] >> (16 * (z & 1))) & 0xffffu;
        } else {
          ez[0] = tabL[q];
        }
#pragma unroll
        for (int z = 0; z < PADG; ++z) {
          const int cc = ez[z] & 0x7fff;
          const double sgd = (ez[z] & 0x8000u) ? -1.0 : 1.0;
          const double x = sgd * cs[cc];
          fS[g] += x;
          if (MOM) {
            const double wj =
                static_cast<double>(static_cast<int64_t>(t) * kColTile + cc + 1) * s.inv_l3;
            fT[g] = fma(x, wj, fT[g]);
            fR[g] += sgd * cs[520 + cc];
          }
        }
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int b = threadIdx.x + kThreads * g;
    if (b < m) {
      const int64_t o = (static_cast<int64_t>(gi) * m + a) * m + b;
      s.partS[o] = fS[g];
      if (MOM) {
        s.partR[o] = fR[g];
        s.partT[o] = fT[g];
      }
    }
  }
}

// C work-group with one column tile per wave (small buckets at 256 < m <= 1024, and at
// 48 < m <= 192 for the probe): wave w sums all of bucket a's rows over tile tq + w (and, with
// moments, the row-weighted sums), four tiles at a time, so no partial sums cross waves.  The four
// tiles' column sums and lists go to LDS (the 512-entry lists of m > 256 in the list area, one
// 16-byte load per thread, loaded with the first rows; the padded lists of m <= 256 after the
// column sums, loaded once the rows are summed); thread b then folds bucket b over the four tiles
// in tile order (the same order as the one-tile form; the column sums add each tile's rows in one
// wave's order instead of four waves' interleaved order).  Two barriers per four tiles instead of
// three per tile.
template <bool MOM, int G, bool VEC>
__device__ void c_unit_wt(const StreamArgs& s, int u, double* lds, uint16_t* tabL) {
  constexpr int U = 8;
  constexpr int PADG = G == 1 ? 8 : 1;         // padded 8-entry segments at m <= 256
  static_assert(!(MOM && G == 1), "the padded lists and weighted sums exceed the data area");
  const int m = s.m;
  const int a = u / s.npc, gi = u - a * s.npc;
  const int t0 = gi * s.tg;
  const int t1 = (t0 + s.tg < s.TC) ? t0 + s.tg : s.TC;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int32_t* prow = s.perm + static_cast<int64_t>(a) * s.cap;
  const bool patched = s.patch_rowptr != nullptr;
  double* cs = lds;                    // [4][520]: the four tiles' column sums and sentinels
  double* csw = lds + 4 * 520;         // [4][520]: row-weighted column sums (moments)
  // the four tiles' lists: 512-entry lists in the list area; padded lists after the column sums
  const int stride = s.ctab_stride;
  uint16_t* lists = PADG == 8 ? reinterpret_cast<uint16_t*>(lds + 4 * 520) : tabL;
  double fS[G], fR[G], fT[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    fS[g] = 0.0;
    fR[g] = 0.0;
    fT[g] = 0.0;
  }
  for (int tq = t0; tq < t1; tq += 4) {
    const int t = tq + w;
    const bool tok = t < t1;
    const int64_t col = static_cast<int64_t>(t) * kColTile + lane * 8;
    const bool lane_ok = tok && col < s.n3;
    // this wave's tile list (512 entries, 8 per lane), loaded with the first rows
    u32x4 tv = {0u, 0u, 0u, 0u};
    if (PADG == 1 && tok) {
      tv = *reinterpret_cast<const u32x4*>(s.ctab + static_cast<int64_t>(t) * 512 + lane * 8);
    }
    double acc[8], accw[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      acc[k] = 0.0;
      accw[k] = 0.0;
    }
    if (tok) {
      for (int base = 0; base < s.cap; base += 64) {
        const int32_t pe = base + lane < s.cap ? prow[base + lane] : -1;
        const int nr = __popcll(__ballot(pe != -1));
        if (nr == 0) break;
        for (int r0 = 0; r0 < nr; r0 += U) {
          f32x4 v0[U], v1[U];
          double sg[U], sw[U];
          int64_t rows[U];
#pragma unroll
          for (int q = 0; q < U; ++q) {
            const bool ok = r0 + q < nr;
            const int32_t e = row_entry(pe, ok ? r0 + q : 0);
            const int64_t row = e & 0x7fffffff;
            rows[q] = row;
            sg[q] = ok ? (e < 0 ? -1.0 : 1.0) : 0.0;
            sw[q] = MOM ? sg[q] * static_cast<double>(row + 1) * s.inv_l1 : 0.0;
            if (VEC) {
              load8f_sel(s.C + row * s.n3 + col, ok && lane_ok, s.zero, v0[q], v1[q]);
            } else if (ok && lane_ok) {
              load8f(s.C + row * s.n3, col, s.n3, false, v0[q], v1[q]);
            } else {
              v0[q] = f32x4{0.f, 0.f, 0.f, 0.f};
              v1[q] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
          }
          if (patched) {
#pragma unroll
            for (int q = 0; q < U; ++q) {
              if (r0 + q < nr && lane_ok) apply_patches(s, rows[q], col, v0[q], v1[q]);
            }
          }
#pragma unroll
          for (int q = 0; q < U; ++q) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const double x = static_cast<double>(e < 4 ? v0[q][e] : v1[q][e - 4]);
              acc[e] = fma(x, sg[q], acc[e]);
              if (MOM) accw[e] = fma(x, sw[q], accw[e]);
            }
          }
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      cs[w * 520 + lane * 8 + e] = acc[e];
      if (MOM) csw[w * 520 + lane * 8 + e] = accw[e];
    }
    if (lane == 0) {
      cs[w * 520 + kColTile] = 0.0;
      if (MOM) csw[w * 520 + kColTile] = 0.0;
    }
    if (PADG == 1) {
      *reinterpret_cast<u32x4*>(lists + w * 512 + lane * 8) = tv;
    } else {
      // the four padded lists (at most 4 x 1856 entries at m <= 192): 8 entries per thread and
      // pass, every pass's load issued before the first store
      u32x4 x[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = (threadIdx.x + kThreads * k) * 8;
        const int ti = e / stride, off = e - ti * stride;
        const bool ok = e < 4 * stride && tq + ti < t1;
        const uint16_t* src =
            s.ctab + static_cast<int64_t>(ok ? tq + ti : 0) * stride + (ok ? off : 0);
        x[k] = ok ? *reinterpret_cast<const u32x4*>(src) : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = (threadIdx.x + kThreads * k) * 8;
        if (e < 4 * stride) *reinterpret_cast<u32x4*>(lists + e) = x[k];
      }
    }
    // segment starts of this thread's buckets in the four tiles, all loads issued at once
    int qb[G][4], qe[G][4];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int b = threadIdx.x + kThreads * g;
#pragma unroll
      for (int ti = 0; ti < 4; ++ti) {
        const bool ok = b < m && tq + ti < t1;
        const int32_t* co =
            s.coff + static_cast<int64_t>(ok ? tq + ti : 0) * (m + 1) + (ok ? b : 0);
        qb[g][ti] = ok ? co[0] : 0;
        qe[g][ti] = ok ? co[1] : 0;
      }
    }
    __syncthreads();
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int ti = 0; ti < 4; ++ti) {
        for (int q = qb[g][ti]; q < qe[g][ti]; q += PADG) {
          uint32_t ez[PADG];
          if constexpr (PADG == 8) {
            const u32x4 tw = *reinterpret_cast<const u32x4*>(lists + ti * stride + q);
#pragma unroll
            for (int z = 0; z < 8; ++z) ez[z] = (tw[z >> 1] >> (16 * (z & 1))) & 0xffffu;
          } else {
            ez[0] = lists[ti * 512 + q];
          }
#pragma unroll
          for (int z = 0; z < PADG; ++z) {
            const int cc = ez[z] & 0x7fff;
            const double sgd = (ez[z] & 0x8000u) ? -1.0 : 1.0;
            const double x = sgd * cs[ti * 520 + cc];
            fS[g] += x;
            if (MOM) {
              const double wj =
                  static_cast<double>(static_cast<int64_t>(tq + ti) * kColTile + cc + 1) * s.inv_l3;
              fT[g] = fma(x, wj, fT[g]);
              fR[g] += sgd * csw[ti * 520 + cc];
            }
          }
        }
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int b = threadIdx.x + kThreads * g;
    if (b < m) {
      const int64_t o = (static_cast<int64_t>(gi) * m + a) * m + b;
      s.partS[o] = fS[g];
      if (MOM) {
        s.partR[o] = fR[g];
        s.partT[o] = fT[g];
      }
    }
  }
}

// LDS layout of the stream kernel (dynamic): the A/C combine area or the staged B chunk first,
// then the sorted column list of the current B chunk or C tile.  The longer lists of B chunks
// with fewer rows hold the probe to 3 (2 or 4 rows) or 2 (1 row) work-groups per CU, so those
// instances may use the registers of that occupancy instead of spilling at 4's 128.
// WTC: C work-groups of one tile per wave (c_unit_wt) in place of the one-tile form, as its own
// instance so that the others keep their code and registers.
template <int DT, bool MOM, int RB, int G, int NG, bool VEC, bool WTC>
__global__ __launch_bounds__(kThreads, MOM ? 2 : ((RB == 8 || (RB == 4 && G == 1)) ? 4 : (RB >= 2 ? 3 : 2))) void stream_kernel(
    StreamArgs s) {
  extern __shared__ double lds_dyn[];
  __shared__ uint32_t ldsu[kThreads / 64];
  // the sorted column list of the current B chunk or C tile follows the data area
  uint16_t* tabL = reinterpret_cast<uint16_t*>(reinterpret_cast<char*>(lds_dyn) + s.tab_off);
  // Work-groups are dispatched in index order: the C work-groups (the largest) first, then A and
  // B, the type with the smaller work-groups last, where they fill the tail in the smallest
  // pieces.  (At 4096^3, A work-groups of about 85 KB last ran about 7 us each at the end of the
  // pass and left the chip a third busy for its last 4 us; B last: 35.7 -> 35.3 us per call.
  // Where B work-groups are the larger, as at 16384^3 or 2048 x 8192 x 8192, B last was 2 to
  // 10 us slower.)
  int u = blockIdx.x;
  if (u < s.nC) {
    FPSK_WG_STAMP(0);
    if constexpr (WTC) {
      c_unit_wt<MOM, G, VEC>(s, u, lds_dyn, tabL);
    } else {
      c_unit<MOM, G, VEC>(s, u, lds_dyn, tabL);
    }
    return;
  }
  u -= s.nC;
  if (s.a_first ? u < s.nA : u >= s.nB) {
    FPSK_WG_STAMP(1);
    row_unit<DT, MOM, VEC>(s, a_side(s), s.wt_a != 0, s.a_first ? u : u - s.nB, lds_dyn, ldsu);
    return;
  }
  if (s.a_first) u -= s.nA;
  FPSK_WG_STAMP(2);
  if (s.transb) {
    row_unit<DT, MOM, VEC>(s, w_side(s), s.wt_w != 0, u, lds_dyn, ldsu);
  } else if constexpr (RB == 4 && G <= 2 && !MOM) {
    b_unit_probe4<DT, VEC, G, WTC>(s, u, reinterpret_cast<uint16_t*>(lds_dyn), ldsu);
  } else {
    b_unit<DT, MOM, RB, G, NG, VEC>(s, u, reinterpret_cast<uint16_t*>(lds_dyn), tabL, ldsu);
  }
}

// ----------------------------------------------------------------------------------------
// Pipelined probe (m <= 64, no moments; output blocks of at most 3 x 3, as the 4 x 4 block's
// product does not fit the stream pass's 128 registers): one launch runs the decision of the call
// before the previous one, the block products of the previous call and the stream pass of this
// call.  The three read and write disjoint workspace sets, and each reads only what an earlier
// launch wrote, so they need no ordering among themselves; the product and decision
// work-groups run beside the stream's.  Grid: [decision, 7 idle, the C, A and B work-groups in
// the stream kernel's order, idle up to a multiple of 8, nprod block products]: the block
// products start at a multiple of 8 so that their XCD-local slots hold, and come last so that
// they fill the stream pass's tail.  The decision uses the kernel's 256 threads over
// kDecideThreads virtual threads: the same bits as the stand-alone decision.
template <int DT, bool VEC, int XB, bool WTC>
__global__ __launch_bounds__(kThreads, 4) void probe_pipe_kernel(StreamArgs s, ProductArgs prod,
                                                                 ProductArgs dec, int nprod,
                                                                 int has_dec) {
  extern __shared__ double lds_dyn[];
  __shared__ uint32_t ldsu[kThreads / 64];
  int u = blockIdx.x;
  if (u < 8) {
    if (u == 0 && has_dec) block_decide_body<kThreads, 1>(dec, lds_dyn);
    return;
  }
  u -= 8;
  const int pbase = (s.nC + s.nB + s.nA + 7) / 8 * 8;
  if (u >= pbase) {
    block_product_body<XB, 2, XB * XB>(prod, u - pbase, nprod, lds_dyn);
    return;
  }
  if (u >= s.nC + s.nB + s.nA) return;
  uint16_t* tabL = reinterpret_cast<uint16_t*>(reinterpret_cast<char*>(lds_dyn) + s.tab_off);
  if (u < s.nC) {
    if constexpr (WTC) {
      c_unit_wt<false, 1, VEC>(s, u, lds_dyn, tabL);
    } else {
      c_unit<false, 1, VEC>(s, u, lds_dyn, tabL);
    }
    return;
  }
  u -= s.nC;
  if (s.a_first ? u < s.nA : u >= s.nB) {
    row_unit<DT, false, VEC>(s, a_side(s), s.wt_a != 0, s.a_first ? u : u - s.nB, lds_dyn, ldsu);
    return;
  }
  if (s.a_first) u -= s.nA;
  if (s.transb) {
    row_unit<DT, false, VEC>(s, w_side(s), s.wt_w != 0, u, lds_dyn, ldsu);
  } else {
    b_unit_probe4<DT, VEC, 1, WTC>(s, u, reinterpret_cast<uint16_t*>(lds_dyn), ldsu);
  }
}

// LDS the pipelined launch needs besides the stream pass's: the block product's reductions
// and the decision's.
size_t probe_pipe_lds(int xb) {
  const size_t prod = static_cast<size_t>(xb * xb) * (kThreads + 2 * kThreads / 16 + 1);
  const size_t dec = lds_reduce_doubles<kDecideThreads, 1>();
  return (prod > dec ? prod : dec) * sizeof(double);
}

template <int DT, bool VEC, int XB, bool WTC>
static void pipe_launch(const StreamArgs& s, const ProductArgs& prod, const ProductArgs& dec,
                        int nprod, int has_dec, size_t lds, hipStream_t st, hipEvent_t e0,
                        hipEvent_t e1) {
  const dim3 grid(8 + (s.nC + s.nB + s.nA + 7) / 8 * 8 + nprod);
  launch_k(probe_pipe_kernel<DT, VEC, XB, WTC>, grid, dim3(kThreads), lds, st, e0, e1, s, prod,
           dec, nprod, has_dec);
}

template <int DT, bool VEC, bool WTC>
static hipError_t pipe_dispatch(const StreamArgs& s, const ProductArgs& prod,
                                const ProductArgs& dec, int nprod, int has_dec, int xb,
                                size_t lds, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  switch (xb) {
    case 1: pipe_launch<DT, VEC, 1, WTC>(s, prod, dec, nprod, has_dec, lds, st, e0, e1); break;
    case 2: pipe_launch<DT, VEC, 2, WTC>(s, prod, dec, nprod, has_dec, lds, st, e0, e1); break;
    case 3: pipe_launch<DT, VEC, 3, WTC>(s, prod, dec, nprod, has_dec, lds, st, e0, e1); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_probe_pipe(const StreamArgs& s, const ProductArgs& prod, const ProductArgs& dec,
                             int nprod, int has_dec, int dt, int xb, size_t lds_bytes,
                             hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  const bool vec = s.vec_a && s.vec_b && s.vec_c;
  // (one-tile-per-wave C work-groups only with whole 16-byte rows, as in the stream kernel)
  if (vec && s.wt_c) {
    return dt == 1 ? pipe_dispatch<1, true, true>(s, prod, dec, nprod, has_dec, xb, lds_bytes, st,
                                                  e0, e1)
                   : pipe_dispatch<0, true, true>(s, prod, dec, nprod, has_dec, xb, lds_bytes, st,
                                                  e0, e1);
  }
  if (dt == 1) {
    return vec ? pipe_dispatch<1, true, false>(s, prod, dec, nprod, has_dec, xb, lds_bytes, st, e0,
                                               e1)
               : pipe_dispatch<1, false, false>(s, prod, dec, nprod, has_dec, xb, lds_bytes, st,
                                                e0, e1);
  }
  return vec ? pipe_dispatch<0, true, false>(s, prod, dec, nprod, has_dec, xb, lds_bytes, st, e0,
                                             e1)
             : pipe_dispatch<0, false, false>(s, prod, dec, nprod, has_dec, xb, lds_bytes, st, e0,
                                              e1);
}

// ----------------------------------------------------------------------------------------
// Launcher.

template <int DT, bool MOM>
static hipError_t stream_dispatch(const StreamArgs& s, int rb, int g, int ng, size_t lds,
                                  hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  const int grid = s.nA + s.nB + s.nC;
  if (grid <= 0) return hipSuccess;
  const bool vec = s.vec_a && s.vec_b && s.vec_c;
  // one-tile-per-wave C work-groups: their own instances (at G = 1 only the probe's aligned one)
  const bool wtc = s.wt_c && !(g == 1 && (MOM || !vec));
#define FPSK_STREAM_LAUNCH(RB_, G_, NG_, VEC_, WTC_)                                          \
  launch_k(stream_kernel<DT, MOM, RB_, G_, NG_, VEC_, WTC_>, dim3(grid), dim3(kThreads), lds, st, \
           e0, e1, s)
#define FPSK_STREAM_CASE(RB_, G_, NG_)                                                        \
  if (rb == RB_ && g == G_ && ng == NG_) {                                                    \
    if (vec) {                                                                                \
      FPSK_STREAM_LAUNCH(RB_, G_, NG_, true, false);                                          \
    } else {                                                                                  \
      FPSK_STREAM_LAUNCH(RB_, G_, NG_, false, false);                                         \
    }                                                                                         \
    return hipGetLastError();                                                                 \
  }
#define FPSK_STREAM_WTC_CASE(RB_, G_, NG_)                                                    \
  if (wtc && rb == RB_ && g == G_ && ng == NG_) {                                             \
    if (vec) {                                                                                \
      FPSK_STREAM_LAUNCH(RB_, G_, NG_, true, true);                                           \
    } else {                                                                                  \
      FPSK_STREAM_LAUNCH(RB_, G_, NG_, false, true);                                          \
    }                                                                                         \
    return hipGetLastError();                                                                 \
  }
  if constexpr (!MOM) {
    if (wtc && rb == 4 && g == 1 && ng == 1) {
      FPSK_STREAM_LAUNCH(4, 1, 1, true, true);
      return hipGetLastError();
    }
  }
  FPSK_STREAM_WTC_CASE(4, 2, 1)
  FPSK_STREAM_WTC_CASE(8, 2, 1)
  FPSK_STREAM_WTC_CASE(4, 4, 1)
  FPSK_STREAM_CASE(8, 1, 4)
  FPSK_STREAM_CASE(8, 1, 2)
  FPSK_STREAM_CASE(8, 1, 1)
  FPSK_STREAM_CASE(8, 2, 1)
  FPSK_STREAM_CASE(4, 1, 1)
  FPSK_STREAM_CASE(4, 2, 1)
  FPSK_STREAM_CASE(4, 4, 1)
  FPSK_STREAM_CASE(2, 8, 1)
  FPSK_STREAM_CASE(1, 16, 1)
#undef FPSK_STREAM_CASE
#undef FPSK_STREAM_WTC_CASE
#undef FPSK_STREAM_LAUNCH
  return hipErrorInvalidValue;
}

hipError_t launch_stream(const StreamArgs& s, int dt, bool moments, int rb, int g, int ng,
                         size_t lds_bytes, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  if (dt == 1) {
    return moments ? stream_dispatch<1, true>(s, rb, g, ng, lds_bytes, st, e0, e1)
                   : stream_dispatch<1, false>(s, rb, g, ng, lds_bytes, st, e0, e1);
  }
  return moments ? stream_dispatch<0, true>(s, rb, g, ng, lds_bytes, st, e0, e1)
                 : stream_dispatch<0, false>(s, rb, g, ng, lds_bytes, st, e0, e1);
}

}  // namespace fpsk

#ifdef FPSK_WG_TIMELINE
// Copies the first max_records work-group records of the last stream launch (four 64-bit words
// each, as WgStamp writes them) to host memory; synchronous.  Returns 0, or -1 on a bad
// argument or a failed copy.  Exported by the diagnostic build only.
extern "C" int fpsketch_wg_timeline(unsigned long long* out, int64_t max_records) {
  if (out == nullptr || max_records < 1) return -1;
  const int64_t n = max_records < fpsk::kTimelineMax ? max_records : fpsk::kTimelineMax;
  const hipError_t e = hipMemcpyFromSymbol(out, HIP_SYMBOL(fpsk::wg_timeline_stream),
                                           static_cast<size_t>(n) * 4 * sizeof(unsigned long long),
                                           0, hipMemcpyDeviceToHost);
  return e == hipSuccess ? 0 : -1;
}
#endif
