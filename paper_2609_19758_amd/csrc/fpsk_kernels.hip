// gfx950 kernels of the FP-Sketch post hoc verifier.
//
// stream:   one pass over A, B and C forming the factors of Eq. 1 without forming AB:
//           P = H1 A (row-bucket segmented reduction), Q = B H2^T (column-bucket fold of each
//           row of B) and the bucket grid of C (row-bucket accumulation, then a column-bucket
//           fold once per row bucket and tile); with moments, the weighted forms that give the
//           first-moment sketches R and T (paper, Sec. III-B).  No atomics: every sum has a
//           fixed order, so sketches are bit-reproducible.  Streaming sums accumulate in FP64.
// product:  S = P Q - H1 C H2^T (and R, T) with split-K partials in FP64, reduced in fixed
//           slice order per output tile; in probe mode one work-group then computes the
//           clipped-mean noise, the threshold and the verdict (Sec. III-E, III-I, Algorithm 2).
// scan / sample / recheck: the exact scan for non-finite and out-of-range entries
//           (Sec. III-I), strided samples of C for rms-hat (Sec. III-G) and the validation
//           recomputation of candidates (Sec. III-D).
#include "fpsk_internal.h"

#include <hip/hip_ext.h>

namespace fpsk {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));

// ----------------------------------------------------------------------------------------
// Element helpers.  DT: 0 = FP16, 1 = BF16.

template <int DT>
__device__ __forceinline__ float lo_half(uint32_t w) {
  if constexpr (DT == 1) {
    return __uint_as_float(w << 16);
  } else {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w & 0xffffu)));
  }
}

template <int DT>
__device__ __forceinline__ float hi_half(uint32_t w) {
  if constexpr (DT == 1) {
    return __uint_as_float(w & 0xffff0000u);
  } else {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w >> 16)));
  }
}

template <int DT>
__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  return lo_half<DT>(h);
}

// Running max of |x| over both halves of a word, on the bit patterns (|x| is monotone in the
// low 15 bits for non-negative patterns).
__device__ __forceinline__ uint32_t absmax2(uint32_t mx, uint32_t w) {
  const u16x2 a = __builtin_bit_cast(u16x2, mx);
  const u16x2 b = __builtin_bit_cast(u16x2, w & 0x7fff7fffu);
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(a, b));
}

// 8 halfs of a row starting at column col (zero beyond n).
__device__ __forceinline__ u32x4 load8h(const uint16_t* row, int64_t col, int64_t n, bool vec) {
  if (vec && col + 8 <= n) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(row + col));
  }
  u32x4 r = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    if (col + e < n) {
      const uint32_t h = row[col + e];
      r[e >> 1] |= h << (16 * (e & 1));
    }
  }
  return r;
}

// Branch-free 16-byte loads for the vector path: an invalid row or lane reads the zero buffer
// instead of branching, so a group of loads issues back to back.
__device__ __forceinline__ u32x4 load8h_sel(const uint16_t* p, bool ok, const void* zero) {
  const u32x4* q = ok ? reinterpret_cast<const u32x4*>(p) : static_cast<const u32x4*>(zero);
  return __builtin_nontemporal_load(q);
}

__device__ __forceinline__ void load8f_sel(const float* p, bool ok, const void* zero, f32x4& v0,
                                           f32x4& v1) {
  const f32x4* q = ok ? reinterpret_cast<const f32x4*>(p) : static_cast<const f32x4*>(zero);
  v0 = __builtin_nontemporal_load(q);
  v1 = __builtin_nontemporal_load(q + 1);
}

// 8 floats of a row starting at column col (zero beyond n).
__device__ __forceinline__ void load8f(const float* row, int64_t col, int64_t n, bool vec,
                                       f32x4& v0, f32x4& v1) {
  if (vec && col + 8 <= n) {
    v0 = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(row + col));
    v1 = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(row + col + 4));
    return;
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v0[e] = (col + e < n) ? row[col + e] : 0.0f;
    v1[e] = (col + 4 + e < n) ? row[col + 4 + e] : 0.0f;
  }
}

// Replace loaded C values by the recomputed values of absolute entries in this row (compile-time
// element indices only, so the loaded vectors stay in registers).
__device__ __forceinline__ void apply_patches(const StreamArgs& s, int64_t row, int64_t col,
                                              f32x4& v0, f32x4& v1) {
  const int q0 = s.patch_rowptr[row];
  const int q1 = s.patch_rowptr[row + 1];
  for (int q = q0; q < q1; ++q) {
    const int64_t d = static_cast<int64_t>(s.patch_col[q]) - col;
    const float pv = s.patch_val[q];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (d == e) v0[e] = pv;
      if (d == e + 4) v1[e] = pv;
    }
  }
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t o = __shfl_xor(v, off, 64);
    v = v > o ? v : o;
  }
  return v;
}

// Block-wide max of the half-bit maxima; thread 0 returns the value as a float.
template <int DT>
__device__ float block_absmax_half(uint32_t mx, uint32_t* ldsu) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t m16 = (mx & 0xffffu) > (mx >> 16) ? (mx & 0xffffu) : (mx >> 16);
  m16 = wave_max_u32(m16);
  if (lane == 0) ldsu[w] = m16;
  __syncthreads();
  float r = 0.0f;
  if (threadIdx.x == 0) {
    uint32_t b = ldsu[0];
    for (int i = 1; i < kThreads / 64; ++i) b = ldsu[i] > b ? ldsu[i] : b;
    r = half_bits_to_float<DT>(b);
  }
  __syncthreads();
  return r;
}

// ----------------------------------------------------------------------------------------
// Row-bucket passes (A and C work-groups).  Wave w of a work-group takes rows w, w + 4, ... of
// the bucket's sorted row list.  The row entries of up to 64 of its rows arrive with one vector
// load and are broadcast with readlane, so a group of row loads issues back to back instead of
// waiting on an index load per row.

// Row entry (row | negative-sign bit) of this wave's r-th row in the current batch.
__device__ __forceinline__ int32_t row_entry(int32_t pe, int r) {
  return __builtin_amdgcn_readlane(pe, r);
}

// A work-group: bucket a, column tile t of A.  P[a, tile] = sum over the bucket's rows of
// v1(i) A[i, tile] (and Pw with w_i).  Groups of 8 rows are summed in FP32 (their partial sums
// stay within a few units of the last place of the stored FP32 factor), groups in FP64; the 4
// waves are combined in fixed wave order.
template <int DT, bool MOM, bool VEC>
__device__ void a_unit(const StreamArgs& s, int u, double* lds, uint32_t* ldsu) {
  constexpr int U = 8;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int a = u / s.TA, t = u - a * s.TA;
  const int64_t col = static_cast<int64_t>(t) * kColTile + lane * 8;
  const bool lane_ok = col < s.n2;
  const int32_t* prow = s.perm + static_cast<int64_t>(a) * s.cap;
  double acc[8], accw[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    acc[k] = 0.0;
    accw[k] = 0.0;
  }
  uint32_t mx = 0;
  for (int base = w; base < s.cap; base += 4 * 64) {
    const int32_t pe = base + 4 * lane < s.cap ? prow[base + 4 * lane] : -1;
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
        sw[q] = MOM ? static_cast<float>(sg[q] * static_cast<double>(row + 1) * s.inv_l1) : 0.0f;
        if (VEC) {
          v[q] = load8h_sel(s.A + row * s.n2 + col, ok && lane_ok, s.zero);
        } else {
          v[q] = ok ? load8h(s.A + row * s.n2, col, s.n2, false) : u32x4{0u, 0u, 0u, 0u};
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
      s.P[static_cast<int64_t>(a) * s.ldp + gc] = static_cast<float>(v);
      if (MOM) {
        double vw = lds[2048 + k * 64 + ln] + lds[2048 + (8 + k) * 64 + ln];
        vw += lds[2048 + (16 + k) * 64 + ln];
        vw += lds[2048 + (24 + k) * 64 + ln];
        s.Pw[static_cast<int64_t>(a) * s.ldp + gc] = static_cast<float>(vw);
      }
    }
  }
  if (threadIdx.x == 0) s.maxpart[u] = amax;
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
  const int64_t k0 = static_cast<int64_t>(u) * RB;
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

  // Stage chunk c (signs v2(j) applied to the halves) and fold it.
  auto process = [&](Chunk& ch, int c) {
    const int64_t cbase = static_cast<int64_t>(c) * CW;
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
        for (int q = ch.qb[g]; q < ch.qe[g]; q += 8) {
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
        for (int q = ch.qb[g]; q < ch.qe[g]; ++q) {
          const int e = tabL[q];
          float x[RBG];
          load_col<DT, RBG>(L + (MOM ? col_slot<CW>(e) : e) * RB + rg * RBG, x);
          const double wj = MOM ? static_cast<double>(cbase + e + 1) * s.inv_l3 : 0.0;
#pragma unroll
          for (int r = 0; r < RBG; ++r) {
            const double d = static_cast<double>(x[r]);
            acc[g][r] += d;
            if (MOM) accw[g][r] = fma(d, wj, accw[g][r]);
          }
        }
      }
    }
    __syncthreads();
  };

  for (int c = 0; c < s.TB; ++c) {
    Chunk ch;
    issue(ch, c);
    process(ch, c);
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
    if (b < m) {
#pragma unroll
      for (int r = 0; r < RBG; ++r) {
        const int64_t k = k0 + rg * RBG + r;
        if (k < s.n2) {
          s.Q[static_cast<int64_t>(b) * s.ldp + k] = static_cast<float>(acc[g][r]);
          if (MOM) s.Qw[static_cast<int64_t>(b) * s.ldp + k] = static_cast<float>(accw[g][r]);
        }
      }
    }
  }
  const float bmax = block_absmax_half<DT>(mx, ldsu);
  if (threadIdx.x == 0) s.maxpart[s.nA + u] = bmax;
}

// ----------------------------------------------------------------------------------------
// C work-group: row bucket a, a group of tg column tiles.  Per tile, the 4 waves accumulate
// v1(i) C[i, tile] (and w_i v1(i) C) over the bucket's rows in FP64, combine in fixed order,
// and thread b folds the tile's columns of bucket b from the tile's bucket-sorted column list
// (staged in LDS with the row loads): S_C[a, b] += sum v2(j) colsum[j] (T_C with w_j, R_C from
// the row-weighted sums).  One partial per tile group.

template <bool MOM, int G, bool VEC>
__device__ void c_unit(const StreamArgs& s, int u, double* lds, uint16_t* tabL) {
  constexpr int U = 8;
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
    int qb[G], qe[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int b = threadIdx.x + kThreads * g;
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

// ----------------------------------------------------------------------------------------
// Reductions and the probe decision shared by the fused and separate product paths.

// Fixed-order work-group reduction of NV values per thread through LDS (cross-lane shuffles
// of doubles cost tens of cycles each).  Levels of 16: at a level over N entries, thread
// g < N / 16 of value i combines entries g, g + N / 16, ..., g + 15 N / 16 (consecutive threads
// read consecutive addresses; the 16 reads are issued together), until at most 16 remain,
// which one thread per value combines in order.  Bit i of max_mask selects max instead of sum
// for value i.  buf holds NV * (2 NT / 16 + NT + 1) doubles; every thread receives the results.
template <int N, int NV>
__device__ __forceinline__ void lds_reduce_level(const double* src, double* dst,
                                                 uint32_t max_mask) {
  if constexpr (N <= 16) {
    if (static_cast<int>(threadIdx.x) < NV) {
      const int i = threadIdx.x;
      const bool mx = (max_mask >> i) & 1u;
      double e[N];
#pragma unroll
      for (int q = 0; q < N; ++q) e[q] = src[i * N + q];
      double r = e[0];
#pragma unroll
      for (int q = 1; q < N; ++q) r = mx ? fmax(r, e[q]) : r + e[q];
      dst[i] = r;
    }
    __syncthreads();
  } else {
    constexpr int GN = N / 16;
    if (static_cast<int>(threadIdx.x) < NV * GN) {
      const int i = threadIdx.x / GN, g = threadIdx.x - i * GN;
      const bool mx = (max_mask >> i) & 1u;
      const double* b = src + i * N + g;
      double e[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) e[q] = b[q * GN];
      double r = e[0];
#pragma unroll
      for (int q = 1; q < 16; ++q) r = mx ? fmax(r, e[q]) : r + e[q];
      dst[i * GN + g] = r;
    }
    __syncthreads();
    lds_reduce_level<GN, NV>(dst, dst + NV * GN, max_mask);
  }
}

template <int NT, int NV>
__device__ void lds_reduce(double (&v)[NV], double* buf, uint32_t max_mask) {
  static_assert(NT % 16 == 0 && NT <= 4096, "levels of 16");
#pragma unroll
  for (int i = 0; i < NV; ++i) buf[i * NT + threadIdx.x] = v[i];
  __syncthreads();
  double* tmp = buf + NV * NT;
  lds_reduce_level<NT, NV>(buf, tmp, max_mask);
  // the results follow the last level's inputs: locate them by replaying the level sizes
  int n = NT;
  double* res = tmp;
  while (n > 16) {
    res += NV * (n / 16);
    n /= 16;
  }
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = res[i];
  __syncthreads();
}

// The probe's decision from the reduced statistics (Sec. III-B): clipped-mean noise estimate,
// validity bound from max|A| and max|B|, threshold and verdict.
__device__ void decide_tail(const ProductArgs& pa, double sum_abs, double max_abs, double nbad,
                            double clipped, double maxA, double maxB, double acc0, double acc1) {
  const double mm = static_cast<double>(pa.m) * pa.m;
  const double sigma = 1.2533 * (clipped / mm);
  const double tau = pa.c_valid * static_cast<double>(pa.n2) * 0x1p-23 * maxA * maxB;
  const double lim = pa.lim_factor * sigma;
  const double thr = fmin(tau, lim);
  const bool finite = nbad == 0.0;
  const bool clean = finite && max_abs <= thr;
  (void)sum_abs;
  pa.stats[0] = sigma;
  pa.stats[1] = thr;
  pa.stats[2] = tau;
  pa.stats[3] = max_abs;
  pa.stats[4] = finite ? 1.0 : 0.0;
  pa.stats[5] = clean ? 0.0 : 1.0;
  pa.stats[6] = maxA;
  pa.stats[7] = maxB;
  if (clean) {
    pa.sigma_acc[0] = acc0 + sigma;
    pa.sigma_acc[1] = acc1 + 1.0;
  } else if (pa.d_dirty != nullptr) {
    *pa.d_dirty = 1;
  }
}

// LDS layout of the stream kernel (dynamic): the A/C combine area or the staged B chunk first,
// then the sorted column list of the current B chunk or C tile.
template <int DT, bool MOM, int RB, int G, int NG, bool VEC>
__global__ __launch_bounds__(kThreads, MOM ? 2 : 4) void stream_kernel(StreamArgs s) {
  extern __shared__ double lds_dyn[];
  __shared__ uint32_t ldsu[kThreads / 64];
  // the sorted column list of the current B chunk or C tile follows the data area
  uint16_t* tabL = reinterpret_cast<uint16_t*>(reinterpret_cast<char*>(lds_dyn) + s.tab_off);
  // Work-groups are dispatched in index order: the C work-groups (the largest) come first, then
  // B, then A, so the short A work-groups fill the tail.
  int u = blockIdx.x;
  if (u < s.nC) {
    c_unit<MOM, G, VEC>(s, u, lds_dyn, tabL);
    return;
  }
  u -= s.nC;
  if (u < s.nB) {
    b_unit<DT, MOM, RB, G, NG, VEC>(s, u, reinterpret_cast<uint16_t*>(lds_dyn), tabL, ldsu);
    return;
  }
  a_unit<DT, MOM, VEC>(s, u - s.nB, lds_dyn, ldsu);
}

// ----------------------------------------------------------------------------------------
// Probe product for m <= 64: block_product_kernel, then block_decide_kernel.
//   block_product_kernel (block, slice): outputs (a0 .. a0 + XB) x (b0 .. b0 + XB) over the
//     k-slice [slice * kXSlice, + kXSlice).  Thread t takes k = 4 (t + 256 j) within the slice;
//     the dot products run in FP64 on the FP32 factors (rows of P and of the transposed Q, both
//     k-contiguous, read with 16-byte loads that the work-groups of an XCD share through its L2);
//     the 4 waves are combined in fixed order.  Slice 0 subtracts the C grid (the sum of the
//     column-group partials).
//   block_decide_kernel (one work-group): S = sum of the slice partials in slice order, the
//     probe statistics and the verdict.

template <int XB>
__global__ __launch_bounds__(kThreads) void block_product_kernel(ProductArgs pa) {
  constexpr int NV = XB * XB;
  __shared__ double red[NV * (kThreads + 2 * kThreads / 16 + 1)];
  const int m = pa.m;
  const int64_t mm = static_cast<int64_t>(m) * m;
  // XCD-local slot of this launch index, then its slice and output block
  const int per = gridDim.x / 8;
  const int slot = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
  const int slice = slot / pa.xslots;
  if (slice >= pa.xns) return;
  const int q = slot - slice * pa.xslots;
  const int st = q / (pa.xsr * pa.xsc), within = q - st * (pa.xsr * pa.xsc);
  const int rbk = (st / pa.xnstc) * pa.xsr + within / pa.xsc;
  const int cbk = (st % pa.xnstc) * pa.xsc + within % pa.xsc;
  if (rbk >= pa.xnb || cbk >= pa.xnb) return;
  const int a0 = rbk * XB, b0 = cbk * XB;
  // uniform row bases (rows past m repeat row m - 1; their results are dropped)
  const float* prow[XB];
  const float* qrow[XB];
#pragma unroll
  for (int i = 0; i < XB; ++i) {
    prow[i] = pa.P + static_cast<int64_t>(a0 + i < m ? a0 + i : m - 1) * pa.ldp;
    qrow[i] = pa.Q + static_cast<int64_t>(b0 + i < m ? b0 + i : m - 1) * pa.ldp;
  }
  // every load is issued before the first is used: the slice's factor rows, then the C grid of
  // the block (slice 0; thread (v = t & 15, group t >> 4) takes every 16th column-group partial)
  const int kb = slice * kXSlice;
  // the slice in 4 / JH round trips of JH 16-byte loads per row (JH = 2 for the largest block
  // keeps the loads within the register file)
  constexpr int JH = XB <= 3 ? 4 : 2;
  double acc[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) acc[v] = 0.0;
  double c4[4];
  const int cv = threadIdx.x & 15, gs = threadIdx.x >> 4;
  const int ci = cv / XB, cj = cv - (cv / XB) * XB;
  const bool vok = slice == 0 && cv < NV && a0 + ci < m && b0 + cj < m;
  const int64_t co = vok ? static_cast<int64_t>(a0 + ci) * m + b0 + cj : 0;
#pragma unroll
  for (int h = 0; h < 4 / JH; ++h) {
  float4 pv[XB][JH], qv[XB][JH];
#pragma unroll
  for (int j = 0; j < JH; ++j) {
    const int k = kb + 4 * (static_cast<int>(threadIdx.x) + kThreads * (h * JH + j));
    const bool kok = k < pa.kact;
    const int kk = kok ? k : 0;
#pragma unroll
    for (int i = 0; i < XB; ++i) {
      const float4 p = *reinterpret_cast<const float4*>(prow[i] + kk);
      const float4 q = *reinterpret_cast<const float4*>(qrow[i] + kk);
      const float4 z = {0.f, 0.f, 0.f, 0.f};
      pv[i][j] = kok ? p : z;
      qv[i][j] = kok ? q : z;
    }
  }
  if (h == 0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int g = gs + 16 * q;
      const double c = pa.partS[static_cast<int64_t>(g < pa.npc ? g : 0) * mm + co];
      c4[q] = (vok && g < pa.npc) ? c : 0.0;
    }
  }
#pragma unroll
  for (int j = 0; j < JH; ++j)
#pragma unroll
    for (int i = 0; i < XB; ++i)
#pragma unroll
      for (int c = 0; c < XB; ++c) {
        double t = acc[i * XB + c];
        t = fma(static_cast<double>(pv[i][j].x), static_cast<double>(qv[c][j].x), t);
        t = fma(static_cast<double>(pv[i][j].y), static_cast<double>(qv[c][j].y), t);
        t = fma(static_cast<double>(pv[i][j].z), static_cast<double>(qv[c][j].z), t);
        t = fma(static_cast<double>(pv[i][j].w), static_cast<double>(qv[c][j].w), t);
        acc[i * XB + c] = t;
      }
  }
  double cp = (c4[0] + c4[1]) + (c4[2] + c4[3]);
  for (int g = gs + 64; g < pa.npc; g += 16) {   // more than 64 column groups (small m)
    cp += vok ? pa.partS[static_cast<int64_t>(g) * mm + co] : 0.0;
  }
  lds_reduce<kThreads, NV>(acc, red, 0u);
  // C grid of output v: the 16 column-group sums of threads v, 16 + v, ... in order
  red[threadIdx.x] = cp;
  __syncthreads();
  if (static_cast<int>(threadIdx.x) < NV) {
    const int v = threadIdx.x;
    const int i = v / XB, c = v - (v / XB) * XB;
    double cg = 0.0;
    for (int g = 0; g < 16; ++g) cg += red[g * 16 + v];
    if (a0 + i < m && b0 + c < m) {
      pa.xpart[slice * mm + static_cast<int64_t>(a0 + i) * m + b0 + c] = acc[v] - cg;
    }
  }
}

constexpr int kDecideThreads = 1024;

__global__ __launch_bounds__(kDecideThreads) void block_decide_kernel(ProductArgs pa) {
  constexpr int NQ = 4;                       // m <= 64: m^2 <= 4096 outputs
  __shared__ double red[5 * (kDecideThreads + 2 * kDecideThreads / 16 + 1)];
  const int m = pa.m;
  const int mm = m * m;
  // the first slice's partials and the first share of the maxima are loaded together; only
  // outputs and maxima that exist are loaded
  double v[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int o = static_cast<int>(threadIdx.x) + kDecideThreads * q;
    v[q] = o < mm ? pa.xpart[o] : 0.0;
  }
  const int t = threadIdx.x;
  // the running noise sum, read now so that the verdict does not wait on it
  double acc0 = 0.0, acc1 = 0.0;
  if (t == 0) {
    acc0 = pa.sigma_acc[0];
    acc1 = pa.sigma_acc[1];
  }
  float amax = t < pa.nA ? pa.maxpart[t] : 0.0f;
  float bmax = t < pa.nB ? pa.maxpart[pa.nA + t] : 0.0f;
  for (int sl = 1; sl < pa.xns; ++sl) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int o = t + kDecideThreads * q;
      if (o < mm) v[q] += pa.xpart[static_cast<int64_t>(sl) * mm + o];
    }
  }
  for (int i = t + kDecideThreads; i < pa.nA; i += kDecideThreads) {
    amax = fmaxf(amax, pa.maxpart[i]);
  }
  for (int i = t + kDecideThreads; i < pa.nB; i += kDecideThreads) {
    bmax = fmaxf(bmax, pa.maxpart[pa.nA + i]);
  }
  double lsum = 0.0, lmax = 0.0, lbad = 0.0;
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int o = static_cast<int>(threadIdx.x) + kDecideThreads * q;
    if (o < mm) {
      const double av = fabs(v[q]);
      if (__builtin_isfinite(v[q])) {
        lsum += av;
        lmax = fmax(lmax, av);
      } else {
        lbad += 1.0;
      }
    }
  }
  // the five first-phase reductions in one pass (sums: 0, 2; maxima: 1, 3, 4)
  double r5[5] = {lsum, lmax, lbad, static_cast<double>(amax), static_cast<double>(bmax)};
  lds_reduce<kDecideThreads, 5>(r5, red, 0x1au);
  const double sum_abs = r5[0], max_abs = r5[1], nbad = r5[2];
  const double mean_abs = nbad > 0.0 ? __builtin_nan("") : sum_abs / static_cast<double>(mm);
  const double clip = 5.0 * mean_abs;
  double c2 = 0.0;
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int o = static_cast<int>(threadIdx.x) + kDecideThreads * q;
    if (o < mm) {
      const double a = fabs(v[q]);
      c2 += a < clip ? a : clip;
    }
  }
  double r1[1] = {c2};
  lds_reduce<kDecideThreads, 1>(r1, red, 0u);
  if (threadIdx.x == 0) decide_tail(pa, sum_abs, max_abs, nbad, r1[0], r5[3], r5[4], acc0, acc1);
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int o = static_cast<int>(threadIdx.x) + kDecideThreads * q;
    if (o < mm) pa.S[o] = v[q];
  }
}

// ----------------------------------------------------------------------------------------
// Product and decision, ordered by kernel boundaries only (no cross-work-group
// synchronization inside a kernel):
//   mfma_product_kernel (tile, slice): partial P Q over one k-slab on the FP64 matrix cores;
//                   slice 0 also subtracts the C grid (the sum of its column-group partials).
//                   With a single slice it finishes the tile.
//   reduce_kernel   (tile): sums the slices in slice order, stores S (R, T) and, for the probe,
//                   the tile's sum |S|, max |S| and non-finite count;
//   tile_decide_kernel (one work-group): clipped-mean noise, threshold and verdict.

// Store S (R, T) of this thread's outputs and, in probe mode, the tile statistics.  acc holds
// the full P Q - C grid (and Pw Q - R grid, P Qw - T grid).
template <int TS, bool MOM>
__device__ void finish_tile(const ProductArgs& pa, int tile,
                            const double (&acc)[MOM ? 3 : 1][TS / 16][TS / 16], double* red) {
  constexpr int RT = TS / 16;
  const int m = pa.m;
  const int ta = tile / pa.nt, tb = tile - ta * pa.nt;
  const int ty = threadIdx.x >> 4, tx = threadIdx.x & 15;
  double lsum = 0.0, lmax = 0.0, lbad = 0.0;
#pragma unroll
  for (int i = 0; i < RT; ++i)
#pragma unroll
    for (int j = 0; j < RT; ++j) {
      const int row = ta * TS + ty + 16 * i, colb = tb * TS + tx + 16 * j;
      if (row < m && colb < m) {
        const int64_t o = static_cast<int64_t>(row) * m + colb;
        const double sv = acc[0][i][j];
        pa.S[o] = sv;
        if (MOM) {
          pa.R[o] = acc[1][i][j];
          pa.T[o] = acc[2][i][j];
        }
        const double av = fabs(sv);
        if (__builtin_isfinite(sv)) {
          lsum += av;
          lmax = fmax(lmax, av);
        } else {
          lbad += 1.0;
        }
      }
    }
  if (pa.mode != 1) return;
  double r3[3] = {lsum, lmax, lbad};
  lds_reduce<kThreads, 3>(r3, red, 0x2u);
  if (threadIdx.x == 0) {
    pa.tilestat[tile * 4 + 0] = r3[0];
    pa.tilestat[tile * 4 + 1] = r3[1];
    pa.tilestat[tile * 4 + 2] = r3[2];
  }
}

// Product on the FP64 matrix cores.  A wave owns WB x WB blocks of 16 x 16 outputs, each an
// accumulator of v_mfma_f64_16x16x4 (lane l holds rows 4 r + l / 16, column l mod 16 of a block,
// r = 0..3).  Lane l reads row (l mod 16) of the block's factor rows (P, and the transposed Q,
// both k-contiguous) 16 bytes at k + 4 (l / 16): the four elements feed four consecutive MFMA
// steps, which applies one permutation of the 16 k of a step to both operands, so each k is
// taken exactly once.  The FP32 factors are widened to FP64 (their products are exact) and
// accumulated in FP64.  KW: the 4 waves split the k-range of one (16 WB)^2 tile and are summed in
// wave order through LDS (the probe, few tiles); otherwise the 4 waves own the quadrants of a
// (32 WB)^2 tile.  The C grid (minus the column-group partials of S_C, R_C, T_C) is spread over
// the (slice, wave) pairs: each subtracts the groups assigned to it, all of a group's loads in
// one round trip.  With one slice the kernel stores S (R, T) and the probe's tile statistics;
// otherwise the tile partial goes to the scratch, row-major in the tile, for reduce_kernel.
typedef double f64x4 __attribute__((ext_vector_type(4)));

template <int WB, bool KW, bool MOM>
__global__ __launch_bounds__(kThreads) void mfma_product_kernel(ProductArgs pa) {
  static_assert(!(KW && MOM), "the k-split tile serves the probe");
  constexpr int NX = MOM ? 3 : 1;
  constexpr int NF = MOM ? 2 : 1;        // factors per side: P (Pw), Q (Qw)
  constexpr int WT = 16 * WB;            // wave tile edge
  constexpr int TS = KW ? WT : 2 * WT;   // work-group tile edge
  __shared__ f64x4 xl[KW ? 3 * WB * WB * 64 : 1];
  __shared__ double red[3 * (kThreads + 2 * kThreads / 16 + 1)];
  const int m = pa.m;
  const int64_t mm = static_cast<int64_t>(m) * m;
  const int ntiles = pa.nt * pa.nt;
  // the 8 XCDs take launch indices round-robin: launch index i runs slot (i mod 8) G / 8 + i / 8
  // of a slice-major order, so each XCD's work-groups share k-slices of the factors in its L2
  const int per = gridDim.x / 8;
  const int slot = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
  if (slot >= ntiles * pa.NS) return;
  const int slice = slot / ntiles, tile = slot - slice * ntiles;
  const int ta = tile / pa.nt, tb = tile - ta * pa.nt;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int ro = KW ? 0 : (w >> 1) * WT, co = KW ? 0 : (w & 1) * WT;   // wave origin in the tile
  // the wave's k-range: whole steps of 16 (loads at or past kact read zeros)
  const int kw = KW ? pa.ksl / 4 : pa.ksl;
  const int kbeg = slice * pa.ksl + (KW ? w * kw : 0);
  const int kend = (kbeg + kw < pa.kact) ? kbeg + kw : pa.kact;
  const int kq = 4 * (lane >> 4);
  // factor rows of this lane (rows past m repeat row m - 1; their outputs are dropped)
  const float* pr[NF][WB];
  const float* qr[NF][WB];
#pragma unroll
  for (int i = 0; i < WB; ++i) {
    const int ra = ta * TS + ro + 16 * i + (lane & 15);
    const int rb = tb * TS + co + 16 * i + (lane & 15);
    const int64_t oa = static_cast<int64_t>(ra < m ? ra : m - 1) * pa.ldp + kq;
    const int64_t ob = static_cast<int64_t>(rb < m ? rb : m - 1) * pa.ldp + kq;
    pr[0][i] = pa.P + oa;
    qr[0][i] = pa.Q + ob;
    if (MOM) {
      pr[NF - 1][i] = pa.Pw + oa;
      qr[NF - 1][i] = pa.Qw + ob;
    }
  }
  f64x4 acc[NX][WB][WB];
#pragma unroll
  for (int x = 0; x < NX; ++x)
#pragma unroll
    for (int i = 0; i < WB; ++i)
#pragma unroll
      for (int j = 0; j < WB; ++j) acc[x][i][j] = f64x4{0.0, 0.0, 0.0, 0.0};

  // every step's loads are issued one step ahead (the last step reloads itself, in bounds)
  auto load = [&](float4 (&pv)[NF][WB], float4 (&qv)[NF][WB], int k) {
    const bool ok = k + kq < pa.kact;    // kact is a multiple of 4: a float4 is in or out
    const int kk = ok ? k : -kq;         // a float4 past the row reads the row's first instead
    const float4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int i = 0; i < WB; ++i) {
        const float4 p = *reinterpret_cast<const float4*>(pr[f][i] + kk);
        const float4 q = *reinterpret_cast<const float4*>(qr[f][i] + kk);
        pv[f][i] = ok ? p : z;
        qv[f][i] = ok ? q : z;
      }
  };
  float4 pv[NF][WB], qv[NF][WB];
  if (kbeg < kend) load(pv, qv, kbeg);
  for (int k = kbeg; k < kend; k += 16) {
    float4 pn[NF][WB], qn[NF][WB];
    load(pn, qn, k + 16 < kend ? k + 16 : k);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      double a[NF][WB], b[NF][WB];
#pragma unroll
      for (int f = 0; f < NF; ++f)
#pragma unroll
        for (int i = 0; i < WB; ++i) {
          a[f][i] = static_cast<double>(pv[f][i][e]);
          b[f][i] = static_cast<double>(qv[f][i][e]);
        }
#pragma unroll
      for (int i = 0; i < WB; ++i)
#pragma unroll
        for (int j = 0; j < WB; ++j) {
          acc[0][i][j] =
              __builtin_amdgcn_mfma_f64_16x16x4f64(a[0][i], b[0][j], acc[0][i][j], 0, 0, 0);
          if (MOM) {
            acc[1][i][j] =
                __builtin_amdgcn_mfma_f64_16x16x4f64(a[1][i], b[0][j], acc[1][i][j], 0, 0, 0);
            acc[2][i][j] =
                __builtin_amdgcn_mfma_f64_16x16x4f64(a[0][i], b[1][j], acc[2][i][j], 0, 0, 0);
          }
        }
    }
#pragma unroll
    for (int f = 0; f < NF; ++f)
#pragma unroll
      for (int i = 0; i < WB; ++i) {
        pv[f][i] = pn[f][i];
        qv[f][i] = qn[f][i];
      }
  }
  // this wave's share of the C grid: groups g = g0, g0 + gs, ...
  {
    const double* part[3] = {pa.partS, pa.partR, pa.partT};
    const int g0 = KW ? slice * 4 + w : slice;
    const int gs = KW ? 4 * pa.NS : pa.NS;
    for (int g = g0; g < pa.npc; g += gs) {
      const int64_t gb = static_cast<int64_t>(g) * mm;
#pragma unroll
      for (int x = 0; x < NX; ++x)
#pragma unroll
        for (int i = 0; i < WB; ++i)
#pragma unroll
          for (int j = 0; j < WB; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int row = ta * TS + ro + 16 * i + 4 * r + (lane >> 4);
              const int col = tb * TS + co + 16 * j + (lane & 15);
              if (row < m && col < m) {
                acc[x][i][j][r] -= part[x][gb + static_cast<int64_t>(row) * m + col];
              }
            }
    }
  }
  if constexpr (KW) {
    // waves 1..3 hand their accumulators to wave 0, which adds them in wave order
    if (w > 0) {
#pragma unroll
      for (int i = 0; i < WB; ++i)
#pragma unroll
        for (int j = 0; j < WB; ++j) xl[((w - 1) * WB * WB + i * WB + j) * 64 + lane] = acc[0][i][j];
    }
    __syncthreads();
    if (w == 0) {
#pragma unroll
      for (int v = 0; v < 3; ++v)
#pragma unroll
        for (int i = 0; i < WB; ++i)
#pragma unroll
          for (int j = 0; j < WB; ++j) acc[0][i][j] += xl[(v * WB * WB + i * WB + j) * 64 + lane];
    }
  }
  const bool owner = !KW || w == 0;       // waves that hold finished tile outputs
  double* outm[3] = {pa.S, pa.R, pa.T};
  double lsum = 0.0, lmax = 0.0, lbad = 0.0;
#pragma unroll
  for (int x = 0; x < NX; ++x)
#pragma unroll
    for (int i = 0; i < WB; ++i)
#pragma unroll
      for (int j = 0; j < WB; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int rt = ro + 16 * i + 4 * r + (lane >> 4);   // row and column in the tile
          const int ct = co + 16 * j + (lane & 15);
          const int row = ta * TS + rt, col = tb * TS + ct;
          const bool valid = owner && row < m && col < m;
          const double v = acc[x][i][j][r];
          if (pa.NS > 1) {
            if (owner) {
              pa.scratch[((static_cast<int64_t>(slice) * ntiles + tile) * NX + x) * TS * TS +
                         rt * TS + ct] = v;
            }
          } else if (valid) {
            outm[x][static_cast<int64_t>(row) * m + col] = v;
            if (x == 0) {
              if (__builtin_isfinite(v)) {
                lsum += fabs(v);
                lmax = fmax(lmax, fabs(v));
              } else {
                lbad += 1.0;
              }
            }
          }
        }
  if (pa.NS > 1 || pa.mode != 1) return;
  double r3[3] = {lsum, lmax, lbad};
  lds_reduce<kThreads, 3>(r3, red, 0x2u);
  if (threadIdx.x == 0) {
    pa.tilestat[tile * 4 + 0] = r3[0];
    pa.tilestat[tile * 4 + 1] = r3[1];
    pa.tilestat[tile * 4 + 2] = r3[2];
  }
}

template <int TS, bool MOM>
__global__ __launch_bounds__(kThreads) void reduce_kernel(ProductArgs pa) {
  constexpr int RT = TS / 16;
  constexpr int NX = MOM ? 3 : 1;
  __shared__ double red[3 * (kThreads + 2 * kThreads / 16 + 1)];
  const int ntiles = pa.nt * pa.nt;
  const int tile = blockIdx.x;
  const int ty = threadIdx.x >> 4, tx = threadIdx.x & 15;
  double acc[NX][RT][RT];
#pragma unroll
  for (int x = 0; x < NX; ++x)
#pragma unroll
    for (int i = 0; i < RT; ++i)
#pragma unroll
      for (int j = 0; j < RT; ++j) {
        double v = 0.0;
#pragma unroll 8
        for (int sl = 0; sl < pa.NS; ++sl) {
          const int64_t o = ((static_cast<int64_t>(sl) * ntiles + tile) * NX + x) * TS * TS +
                            (ty + 16 * i) * TS + tx + 16 * j;
          v += pa.scratch[o];
        }
        acc[x][i][j] = v;
      }
  finish_tile<TS, MOM>(pa, tile, acc, red);
}

// The probe's decision after the tile path (one work-group of 1024): the tile statistics and
// operand maxima in one reduction, then the clipped sum over S, whose first 16 x 1024 entries
// were loaded with the statistics.
__global__ __launch_bounds__(kDecideThreads) void tile_decide_kernel(ProductArgs pa) {
  constexpr int NQ = 16;
  __shared__ double red[5 * (kDecideThreads + 2 * kDecideThreads / 16 + 1)];
  const int t = threadIdx.x;
  // the running noise sum, read now so that the verdict does not wait on it
  double acc0 = 0.0, acc1 = 0.0;
  if (t == 0) {
    acc0 = pa.sigma_acc[0];
    acc1 = pa.sigma_acc[1];
  }
  const int64_t mm = static_cast<int64_t>(pa.m) * pa.m;
  const int ntiles = pa.nt * pa.nt;
  double v[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int64_t o = t + static_cast<int64_t>(kDecideThreads) * q;
    v[q] = o < mm ? pa.S[o] : 0.0;
  }
  double lsum = 0.0, lmax = 0.0, lbad = 0.0;
  for (int i = t; i < ntiles; i += kDecideThreads) {
    lsum += pa.tilestat[i * 4 + 0];
    lmax = fmax(lmax, pa.tilestat[i * 4 + 1]);
    lbad += pa.tilestat[i * 4 + 2];
  }
  float amax = 0.0f, bmax = 0.0f;
  for (int i = t; i < pa.nA; i += kDecideThreads) amax = fmaxf(amax, pa.maxpart[i]);
  for (int i = t; i < pa.nB; i += kDecideThreads) bmax = fmaxf(bmax, pa.maxpart[pa.nA + i]);
  // sums: 0, 2; maxima: 1, 3, 4
  double r5[5] = {lsum, lmax, lbad, static_cast<double>(amax), static_cast<double>(bmax)};
  lds_reduce<kDecideThreads, 5>(r5, red, 0x1au);
  const double sum_abs = r5[0], max_abs = r5[1], nbad = r5[2];
  // mean|S| over all buckets (a non-finite bucket makes the mean non-finite)
  const double mean_abs = nbad > 0.0 ? __builtin_nan("") : sum_abs / static_cast<double>(mm);
  const double clip = 5.0 * mean_abs;
  double c2 = 0.0;
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int64_t o = t + static_cast<int64_t>(kDecideThreads) * q;
    const double a = fabs(v[q]);
    if (o < mm) c2 += a < clip ? a : clip;
  }
#pragma unroll 8
  for (int64_t o = t + static_cast<int64_t>(kDecideThreads) * NQ; o < mm; o += kDecideThreads) {
    const double a = fabs(pa.S[o]);
    c2 += a < clip ? a : clip;
  }
  double r1[1] = {c2};
  lds_reduce<kDecideThreads, 1>(r1, red, 0u);
  if (t == 0) decide_tail(pa, sum_abs, max_abs, nbad, r1[0], r5[3], r5[4], acc0, acc1);
}

// ----------------------------------------------------------------------------------------
// Exact scan (non-finite or |C| > fp32max/16), samples, recheck.

__device__ __forceinline__ bool is_absolute_entry(float x) {
  return !(fabsf(x) <= static_cast<float>(kHugeLimit));
}

__global__ __launch_bounds__(kThreads) void scan_count_kernel(const float* C, int64_t n3,
                                                              int32_t* counts) {
  __shared__ int red[kThreads];
  const int64_t row = blockIdx.x;
  int cnt = 0;
  for (int64_t j = threadIdx.x; j < n3; j += kThreads) cnt += is_absolute_entry(C[row * n3 + j]);
  red[threadIdx.x] = cnt;
  __syncthreads();
  for (int st = kThreads / 2; st > 0; st >>= 1) {
    if (threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
    __syncthreads();
  }
  if (threadIdx.x == 0) counts[row] = red[0];
}

__global__ __launch_bounds__(kThreads) void scan_extract_kernel(const float* C, int64_t n3,
                                                                const int32_t* rows,
                                                                const int32_t* base, int32_t cap,
                                                                int64_t* out) {
  __shared__ int wtot[kThreads / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t row = rows[blockIdx.x];
  int pos = base[blockIdx.x];
  for (int64_t j0 = 0; j0 < n3; j0 += kThreads) {
    const int64_t j = j0 + threadIdx.x;
    const bool f = j < n3 && is_absolute_entry(C[row * n3 + j]);
    const uint64_t bal = __ballot(f);
    const uint64_t below = lane == 0 ? 0ull : (bal & (~0ull >> (64 - lane)));
    const int pre = __popcll(below);
    if (lane == 0) wtot[w] = __popcll(bal);
    __syncthreads();
    int woff = 0, tot = 0;
    for (int i = 0; i < kThreads / 64; ++i) {
      if (i < w) woff += wtot[i];
      tot += wtot[i];
    }
    if (f) {
      const int idx = pos + woff + pre;
      if (idx < cap) {
        out[2 * idx] = row;
        out[2 * idx + 1] = j;
      }
    }
    pos += tot;
    __syncthreads();
  }
}

// ----------------------------------------------------------------------------------------
// Order statistics of the bucket grid (the MAD of Sec. III-E and the candidate scan of
// Algorithm 1) by radix selection over order-preserving 64-bit keys: eight passes of 8-bit
// digits, each a histogram of the keys that match the digits fixed so far, then one work-group
// that fixes the next digit.  Exact: the selected key is the k-th smallest.

// Key order equals the order of the doubles (-0 just below +0); NaN sorts above +inf.
__device__ __forceinline__ uint64_t order_key(double x) {
  if (__builtin_isnan(x)) return ~0ull;
  const uint64_t u = __builtin_bit_cast(uint64_t, x);
  return (u >> 63) ? ~u : (u | (1ull << 63));
}

__device__ __forceinline__ double key_value(uint64_t k) {
  const uint64_t u = (k >> 63) ? (k & ~(1ull << 63)) : ~k;
  return __builtin_bit_cast(double, u);
}

// MODE 0: keys of S; MODE 1: keys of |S - st->med|
template <int MODE>
__device__ __forceinline__ uint64_t sel_key(const double* S, int64_t i, double med) {
  const double x = MODE == 0 ? S[i] : fabs(S[i] - med);
  return order_key(x);
}

__global__ __launch_bounds__(kThreads) void sel_init_kernel(SelState* st, uint64_t k) {
  st->prefix = 0;
  st->k = k;
  st->next = ~0ull;
  st->count_eq = 0;
  st->pass = 0;
}

template <int MODE>
__global__ __launch_bounds__(kThreads) void sel_hist_kernel(const double* S, int64_t n,
                                                            const SelState* st, uint32_t* hist) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int shift = 56 - 8 * st->pass;
  const uint64_t hmask = shift == 56 ? 0ull : (~0ull << (shift + 8));
  const uint64_t pref = st->prefix;
  const double med = st->med;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kThreads) {
    const uint64_t key = sel_key<MODE>(S, i, med);
    if ((key & hmask) == pref) atomicAdd(&h[(key >> shift) & 255u], 1u);
  }
  __syncthreads();
  if (h[threadIdx.x] != 0) atomicAdd(&hist[threadIdx.x], h[threadIdx.x]);
}

// One work-group of 256: the digit whose cumulative count passes k; clears the histogram.
__global__ __launch_bounds__(kThreads) void sel_step_kernel(SelState* st, uint32_t* hist) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = hist[threadIdx.x];
  __syncthreads();
  hist[threadIdx.x] = 0;
  if (threadIdx.x == 0) {
    const int shift = 56 - 8 * st->pass;
    uint64_t below = 0;
    int b = 0;
    for (; b < 255; ++b) {
      if (st->k < below + h[b]) break;
      below += h[b];
    }
    st->prefix |= static_cast<uint64_t>(b) << shift;
    st->k -= below;
    st->count_eq = h[b];
    st->pass += 1;
  }
}

// Smallest key above the selected one (the upper middle element when it differs).
template <int MODE>
__global__ __launch_bounds__(kThreads) void sel_next_kernel(const double* S, int64_t n,
                                                            SelState* st) {
  __shared__ uint64_t red[kThreads];
  const uint64_t sel = st->prefix;
  const double med = st->med;
  uint64_t best = ~0ull;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kThreads) {
    const uint64_t key = sel_key<MODE>(S, i, med);
    if (key > sel && key < best) best = key;
  }
  red[threadIdx.x] = best;
  __syncthreads();
  for (int w = kThreads / 2; w > 0; w >>= 1) {
    if (static_cast<int>(threadIdx.x) < w && red[threadIdx.x + w] < red[threadIdx.x]) {
      red[threadIdx.x] = red[threadIdx.x + w];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0 && red[0] != ~0ull) atomicMin(reinterpret_cast<unsigned long long*>(&st->next), static_cast<unsigned long long>(red[0]));
}

// The median from the selected order statistic(s): x_(n/2) for odd n, else the mean of
// x_(n/2 - 1) (selected) and x_(n/2) (the same key while equal keys remain, else the next).
template <int MODE>
__global__ __launch_bounds__(kThreads) void sel_final_kernel(SelState* st, int64_t n) {
  const double lo = key_value(st->prefix);
  double v = lo;
  if (n % 2 == 0) {
    const double hi = (st->k + 1 < st->count_eq) ? lo : key_value(st->next);
    v = 0.5 * (lo + hi);
  }
  if (MODE == 0) {
    st->med = v;
  } else {
    st->mad = v;
  }
}

__global__ __launch_bounds__(1) void peel_kernel(double* S, double* R, double* T,
                                                 const PeelEntry* list, int n) {
  for (int q = 0; q < n; ++q) {
    const PeelEntry e = list[q];
    S[e.o] -= e.ds;
    R[e.o] -= e.dr;
    T[e.o] -= e.dt;
  }
}

__global__ __launch_bounds__(kThreads) void above_kernel(const double* S, const double* R,
                                                         const double* T, int64_t n, double cut,
                                                         Cand* out, uint32_t cap,
                                                         uint32_t* count) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * kThreads) {
    const double s = S[i];
    if (fabs(s) > cut) {
      const uint32_t p = atomicAdd(count, 1u);
      if (p < cap) out[p] = Cand{i, s, R[i], T[i]};
    }
  }
}

__global__ __launch_bounds__(kThreads) void sample_kernel(const float* C, int64_t stride,
                                                          int64_t count, float* out) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
  if (t < count) out[t] = C[t * stride];
}

// One wave per coordinate: gamma = sum_k A_ik B_kj and sum_k |A_ik B_kj|, exact products
// accumulated in FP64, reduced across lanes in fixed butterfly order.
template <int DT>
__global__ __launch_bounds__(kThreads) void recheck_kernel(const uint16_t* A, const uint16_t* B,
                                                           const float* C, int64_t n2, int64_t n3,
                                                           const int64_t* coords, int n,
                                                           double* gamma, double* abssum,
                                                           float* cval) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = blockIdx.x * (kThreads / 64) + w;
  if (c >= n) return;
  const int64_t i = coords[2 * c], j = coords[2 * c + 1];
  double g = 0.0, ab = 0.0;
  for (int64_t k = lane; k < n2; k += 64) {
    const double a = static_cast<double>(half_bits_to_float<DT>(A[i * n2 + k]));
    const double b = static_cast<double>(half_bits_to_float<DT>(B[k * n3 + j]));
    const double p = a * b;
    g += p;
    ab += fabs(p);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    g += __shfl_xor(g, off, 64);
    ab += __shfl_xor(ab, off, 64);
  }
  if (lane == 0) {
    gamma[c] = g;
    abssum[c] = ab;
    if (C != nullptr && cval != nullptr) cval[c] = C[i * n3 + j];
  }
}

// ----------------------------------------------------------------------------------------
// Reference streams of known size: a plain read (XOR-folded so no load is dropped) and a
// plain copy, 16 bytes per lane, grid-stride.

__global__ __launch_bounds__(kThreads) void read_kernel(const u32x4* src, int64_t n16,
                                                        uint32_t* out) {
  uint32_t x = 0;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n16;
       i += stride) {
    const u32x4 v = __builtin_nontemporal_load(src + i);
    x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  if (x == 0x9E3779B9u) out[0] = x;   // practically never taken; keeps the loads alive
}

__global__ __launch_bounds__(kThreads) void copy_kernel(const u32x4* src, u32x4* dst,
                                                        int64_t n16) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n16;
       i += stride) {
    dst[i] = __builtin_nontemporal_load(src + i);
  }
}

// ----------------------------------------------------------------------------------------
// Launchers.

// A launch whose dispatch packet, when e0 / e1 are given, records its own start / end time in
// them (no extra queue packets, so the events bracket exactly the kernel).
template <typename K, typename... Args>
static void launch_k(K kernel, dim3 grid, dim3 block, size_t shmem, hipStream_t st, hipEvent_t e0,
                     hipEvent_t e1, Args... args) {
  if (e0 != nullptr || e1 != nullptr) {
    hipExtLaunchKernelGGL(kernel, grid, block, static_cast<uint32_t>(shmem), st, e0, e1, 0u,
                          args...);
  } else {
    hipLaunchKernelGGL(kernel, grid, block, shmem, st, args...);
  }
}

template <int DT, bool MOM>
static hipError_t stream_dispatch(const StreamArgs& s, int rb, int g, int ng, size_t lds,
                                  hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
  const int grid = s.nA + s.nB + s.nC;
  if (grid <= 0) return hipSuccess;
  const bool vec = s.vec_a && s.vec_b && s.vec_c;
#define FPSK_STREAM_CASE(RB_, G_, NG_)                                                        \
  if (rb == RB_ && g == G_ && ng == NG_) {                                                    \
    if (vec) {                                                                                \
      launch_k(stream_kernel<DT, MOM, RB_, G_, NG_, true>, dim3(grid), dim3(kThreads), lds,   \
               st, e0, e1, s);                                                                \
    } else {                                                                                  \
      launch_k(stream_kernel<DT, MOM, RB_, G_, NG_, false>, dim3(grid), dim3(kThreads), lds,  \
               st, e0, e1, s);                                                                \
    }                                                                                         \
    return hipGetLastError();                                                                 \
  }
  FPSK_STREAM_CASE(8, 1, 4)
  FPSK_STREAM_CASE(8, 1, 2)
  FPSK_STREAM_CASE(8, 1, 1)
  FPSK_STREAM_CASE(8, 2, 1)
  FPSK_STREAM_CASE(4, 4, 1)
  FPSK_STREAM_CASE(2, 8, 1)
  FPSK_STREAM_CASE(1, 16, 1)
#undef FPSK_STREAM_CASE
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

hipError_t launch_product(const ProductArgs& a0, int ts, bool kw, bool moments, hipStream_t st,
                          hipEvent_t e0, hipEvent_t e1) {
  ProductArgs a = a0;
  if (a.mode == 1 && !moments && a.nX > 0) {
    const dim3 g(a.nX), b(kThreads);
    switch (a.xb) {
      case 1: launch_k(block_product_kernel<1>, g, b, 0, st, e0, nullptr, a); break;
      case 2: launch_k(block_product_kernel<2>, g, b, 0, st, e0, nullptr, a); break;
      case 3: launch_k(block_product_kernel<3>, g, b, 0, st, e0, nullptr, a); break;
      default: launch_k(block_product_kernel<4>, g, b, 0, st, e0, nullptr, a); break;
    }
    launch_k(block_decide_kernel, dim3(1), dim3(kDecideThreads), 0, st, nullptr, e1, a);
    return hipGetLastError();
  }
  const dim3 grid((a.nt * a.nt * a.NS + 7) / 8 * 8);     // whole rounds of the 8 XCDs
  const dim3 rgrid(a.nt * a.nt);
  const bool red = a.NS > 1, dec = a.mode == 1;
#define FPSK_PRODUCT_CASE(TS_, WB_, KW_, MOM_)                                              \
  if (ts == TS_ && kw == KW_ && moments == MOM_) {                                          \
    launch_k(mfma_product_kernel<WB_, KW_, MOM_>, grid, dim3(kThreads), 0, st, e0,          \
             (red || dec) ? nullptr : e1, a);                                               \
    if (red) {                                                                              \
      launch_k(reduce_kernel<TS_, MOM_>, rgrid, dim3(kThreads), 0, st, nullptr,             \
               dec ? nullptr : e1, a);                                                      \
    }                                                                                       \
    if (dec) launch_k(tile_decide_kernel, dim3(1), dim3(kDecideThreads), 0, st, nullptr, e1, a); \
    return hipGetLastError();                                                               \
  }
  FPSK_PRODUCT_CASE(16, 1, true, false)
  FPSK_PRODUCT_CASE(64, 2, false, false)
  FPSK_PRODUCT_CASE(32, 1, false, true)
  FPSK_PRODUCT_CASE(64, 2, false, true)
#undef FPSK_PRODUCT_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_scan_count(const float* C, int64_t n1, int64_t n3, int32_t* counts,
                             hipStream_t st) {
  hipLaunchKernelGGL(scan_count_kernel, dim3(static_cast<unsigned>(n1)), dim3(kThreads), 0, st,
                     C, n3, counts);
  return hipGetLastError();
}

hipError_t launch_scan_extract(const float* C, int64_t n3, const int32_t* rows,
                               const int32_t* base, int nrows, int32_t cap, int64_t* out,
                               hipStream_t st) {
  if (nrows <= 0) return hipSuccess;
  hipLaunchKernelGGL(scan_extract_kernel, dim3(nrows), dim3(kThreads), 0, st, C, n3, rows, base,
                     cap, out);
  return hipGetLastError();
}

hipError_t launch_sample(const float* C, int64_t stride, int64_t count, float* out,
                         hipStream_t st) {
  if (count <= 0) return hipSuccess;
  const unsigned grid = static_cast<unsigned>((count + kThreads - 1) / kThreads);
  hipLaunchKernelGGL(sample_kernel, dim3(grid), dim3(kThreads), 0, st, C, stride, count, out);
  return hipGetLastError();
}

hipError_t launch_peel(double* S, double* R, double* T, const PeelEntry* list, int n,
                       hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(peel_kernel, dim3(1), dim3(1), 0, st, S, R, T, list, n);
  return hipGetLastError();
}

namespace {
unsigned grid_for(int64_t n) {
  const int64_t g = (n + 8 * kThreads - 1) / (8 * kThreads);
  return static_cast<unsigned>(g < 1 ? 1 : (g > 1024 ? 1024 : g));
}

template <int MODE>
void select_median(const double* S, int64_t n, SelState* st, uint32_t* hist, hipStream_t s) {
  const unsigned g = grid_for(n);
  hipLaunchKernelGGL(sel_init_kernel, dim3(1), dim3(1), 0, s, st,
                     static_cast<uint64_t>(n % 2 ? n / 2 : n / 2 - 1));
  for (int p = 0; p < 8; ++p) {
    hipLaunchKernelGGL(sel_hist_kernel<MODE>, dim3(g), dim3(kThreads), 0, s, S, n, st, hist);
    hipLaunchKernelGGL(sel_step_kernel, dim3(1), dim3(kThreads), 0, s, st, hist);
  }
  if (n % 2 == 0) hipLaunchKernelGGL(sel_next_kernel<MODE>, dim3(g), dim3(kThreads), 0, s, S, n, st);
  hipLaunchKernelGGL(sel_final_kernel<MODE>, dim3(1), dim3(1), 0, s, st, n);
}
}  // namespace

hipError_t launch_median_mad(const double* S, int64_t n, SelState* st, uint32_t* hist,
                             hipStream_t s) {
  if (n <= 0) return hipErrorInvalidValue;
  select_median<0>(S, n, st, hist, s);
  select_median<1>(S, n, st, hist, s);
  return hipGetLastError();
}

hipError_t launch_above(const double* S, const double* R, const double* T, int64_t n,
                        double cut, Cand* out, uint32_t cap, uint32_t* count, hipStream_t st) {
  hipLaunchKernelGGL(above_kernel, dim3(grid_for(n)), dim3(kThreads), 0, st, S, R, T, n, cut,
                     out, cap, count);
  return hipGetLastError();
}

hipError_t launch_recheck(const uint16_t* A, const uint16_t* B, const float* C, int64_t n2,
                          int64_t n3, int dt, const int64_t* coords, int n, double* gamma,
                          double* abssum, float* cval, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const unsigned grid = static_cast<unsigned>((n + 3) / 4);
  if (dt == 1) {
    hipLaunchKernelGGL(recheck_kernel<1>, dim3(grid), dim3(kThreads), 0, st, A, B, C, n2, n3,
                       coords, n, gamma, abssum, cval);
  } else {
    hipLaunchKernelGGL(recheck_kernel<0>, dim3(grid), dim3(kThreads), 0, st, A, B, C, n2, n3,
                       coords, n, gamma, abssum, cval);
  }
  return hipGetLastError();
}

hipError_t launch_read(const void* src, int64_t bytes, uint32_t* out, int grid, hipStream_t st) {
  hipLaunchKernelGGL(read_kernel, dim3(grid), dim3(kThreads), 0, st,
                     static_cast<const u32x4*>(src), bytes / 16, out);
  return hipGetLastError();
}

hipError_t launch_copy(const void* src, void* dst, int64_t bytes, int grid, hipStream_t st) {
  hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(kThreads), 0, st,
                     static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), bytes / 16);
  return hipGetLastError();
}

}  // namespace fpsk
