// gfx950 kernels of the FP-Sketch post hoc verifier after the stream pass (the stream kernel
// itself is in fpsk_stream.hip).
//
// product:  S = P Q - H1 C H2^T (and R, T) with split-K partials in FP64, reduced in fixed
//           slice order per output tile; in probe mode one work-group then computes the
//           clipped-mean noise, the threshold and the verdict (Sec. III-E, III-I, Algorithm 2).
// scan / sample / recheck: the exact scan for non-finite and out-of-range entries
//           (Sec. III-I), strided samples of C for rms-hat (Sec. III-G) and the validation
//           recomputation of candidates (Sec. III-D).
// select:   exact order statistics, peel and candidate scan of a localize round (Algorithm 1).
#include "fpsk_block.h"

#include <algorithm>

namespace fpsk {

// ----------------------------------------------------------------------------------------
// Probe product for m <= 64 (bodies in fpsk_block.h): the block products, then one deciding
// work-group of kDecideThreads.  The diagnostic timeline build records the block products at
// their launch indices (type 3) and the decision in the last slot (type 4).

#ifdef FPSK_WG_TIMELINE
static __device__ unsigned long long wg_timeline_tail[4 * kTimelineMax];
#define FPSK_TAIL_STAMP(slot, type) const WgStamp wg_stamp_(wg_timeline_tail, slot, type)
#else
#define FPSK_TAIL_STAMP(slot, type)
#endif

template <int XB>
__global__ __launch_bounds__(kThreads) void block_product_kernel(ProductArgs pa) {
  FPSK_TAIL_STAMP(blockIdx.x, 3);
  __shared__ double red[lds_reduce_doubles<kThreads, XB * XB>()];
  block_product_body<XB, (XB <= 3 ? 4 : 2), XB * XB>(pa, blockIdx.x, gridDim.x, red);
}

__global__ __launch_bounds__(kDecideThreads) void block_decide_kernel(ProductArgs pa) {
  FPSK_TAIL_STAMP(kTimelineMax - 1, 4);
  __shared__ double red[lds_reduce_doubles<kDecideThreads, 5>()];
  block_decide_body<kDecideThreads, 4>(pa, red);
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
  // k per step: 32 for S alone on the quadrant tiles (large m), so that the 4 lanes of a factor
  // row read one whole 128-byte line (two 16-byte pieces each) per step (m = 698: 339 -> 332 us
  // for product and decision); 16 with moments (the registers of three products) and on the
  // k-split tiles of mid m, where it measured slower
  constexpr int NE = (MOM || KW) ? 1 : 2;   // 16-byte pieces per lane and operand per step
  constexpr int KS = 16 * NE;
  // the wave's k-range
  const int kw = KW ? pa.ksl / 4 : pa.ksl;
  const int kbeg = slice * pa.ksl + (KW ? w * kw : 0);
  const int kend = (kbeg + kw < pa.kact) ? kbeg + kw : pa.kact;
  const int kq = 4 * NE * (lane >> 4);
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

  // The wave's k-range in whole steps: past kend (the last slice's end at kact) the factor rows
  // hold zeros up to ldp, which is at least kact rounded up to 1024, so the loads need no
  // bounds test.  Two register sets alternate, each step's loads issued one step ahead.
  const int kstop = kbeg < kend ? kbeg + (kend - kbeg + KS - 1) / KS * KS : kbeg;
  auto load = [&](float4 (&pv)[NF][WB][NE], float4 (&qv)[NF][WB][NE], int k) {
#pragma unroll
    for (int h = 0; h < NE; ++h)
#pragma unroll
      for (int f = 0; f < NF; ++f)
#pragma unroll
        for (int i = 0; i < WB; ++i) {
          pv[f][i][h] = *reinterpret_cast<const float4*>(pr[f][i] + k + 4 * h);
          qv[f][i][h] = *reinterpret_cast<const float4*>(qr[f][i] + k + 4 * h);
        }
  };
  auto step = [&](const float4 (&pv)[NF][WB][NE], const float4 (&qv)[NF][WB][NE]) {
#pragma unroll
    for (int e = 0; e < 4 * NE; ++e) {
      double a[NF][WB], b[NF][WB];
#pragma unroll
      for (int f = 0; f < NF; ++f)
#pragma unroll
        for (int i = 0; i < WB; ++i) {
          a[f][i] = static_cast<double>(pv[f][i][e >> 2][e & 3]);
          b[f][i] = static_cast<double>(qv[f][i][e >> 2][e & 3]);
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
  };
  // (a load past the last step rereads the last step: every iteration issues the same loads,
  // so the waits for a step's operands never cover the next step's loads)
  const int nst = (kstop - kbeg) / KS;
  const int klast = kstop - KS;
  if (nst > 0) {
    float4 p0[NF][WB][NE], q0[NF][WB][NE], p1[NF][WB][NE], q1[NF][WB][NE];
    load(p0, q0, kbeg);
    int k = kbeg;
    for (int s = 0; s + 2 <= nst; s += 2, k += 2 * KS) {
      load(p1, q1, k + KS);
      step(p0, q0);
      load(p0, q0, k + 2 * KS <= klast ? k + 2 * KS : klast);
      step(p1, q1);
    }
    if (nst & 1) step(p0, q0);
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
  // each output's slices are added in slice order; SB slices' loads of all the thread's outputs
  // are in flight together
  constexpr int SB = MOM ? 1 : 4;
  double acc[NX][RT][RT];
#pragma unroll
  for (int x = 0; x < NX; ++x)
#pragma unroll
    for (int i = 0; i < RT; ++i)
#pragma unroll
      for (int j = 0; j < RT; ++j) acc[x][i][j] = 0.0;
  for (int sl0 = 0; sl0 < pa.NS; sl0 += SB) {
    double v[SB][NX][RT][RT];
#pragma unroll
    for (int s = 0; s < SB; ++s)
#pragma unroll
      for (int x = 0; x < NX; ++x)
#pragma unroll
        for (int i = 0; i < RT; ++i)
#pragma unroll
          for (int j = 0; j < RT; ++j) {
            const int sl = sl0 + s < pa.NS ? sl0 + s : sl0;
            const int64_t o = ((static_cast<int64_t>(sl) * ntiles + tile) * NX + x) * TS * TS +
                              (ty + 16 * i) * TS + tx + 16 * j;
            v[s][x][i][j] = pa.scratch[o];
          }
#pragma unroll
    for (int s = 0; s < SB; ++s) {
      if (sl0 + s < pa.NS) {
#pragma unroll
        for (int x = 0; x < NX; ++x)
#pragma unroll
          for (int i = 0; i < RT; ++i)
#pragma unroll
            for (int j = 0; j < RT; ++j) acc[x][i][j] += v[s][x][i][j];
      }
    }
  }
  finish_tile<TS, MOM>(pa, tile, acc, red);
}

// The probe's decision after the tile path (one work-group of 1024): the tile statistics and
// operand maxima in one reduction, then the clipped sum over S, whose first 16 x 1024 entries
// were loaded with the statistics.
// The tile statistics reduced as the decision reduces them (1024 virtual threads, the same
// bits on any work-group size): sum|S|, max|S|, non-finite count.
static_assert(((kMaxM + 63) / 64) * ((kMaxM + 63) / 64) <= 4 * kDecideThreads,
              "a probe's tiles (64 x 64, or 16 x 16 below 256 tiles) fit 4 per decision thread");

// Virtual thread i's tile statistics: sum|S|, max|S| and non-finite count over tiles i,
// i + kDecideThreads, ... in that order (at most 4096 tiles: the loads issued together).
__device__ __forceinline__ void tile_partials(const ProductArgs& pa, int i, double& lsum,
                                              double& lmax, double& lbad) {
  const int ntiles = pa.nt * pa.nt;
  lsum = 0.0;
  lmax = 0.0;
  lbad = 0.0;
  for (int i0 = i; i0 < ntiles; i0 += 4 * kDecideThreads) {
    double e[4][3];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int ti = i0 + j * kDecideThreads;
      const bool ok = ti < ntiles;
#pragma unroll
      for (int q = 0; q < 3; ++q) e[j][q] = ok ? pa.tilestat[(ok ? ti : 0) * 4 + q] : 0.0;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (i0 + j * kDecideThreads < ntiles) {
        lsum += e[j][0];
        lmax = fmax(lmax, e[j][1]);
        lbad += e[j][2];
      }
    }
  }
}

template <int NTR>
__device__ void tile_totals(const ProductArgs& pa, double* red, double (&out)[3]) {
  constexpr int N = kDecideThreads;
  constexpr int VT = N / NTR;
  double v[VT][3];
#pragma unroll
  for (int j = 0; j < VT; ++j) {
    tile_partials(pa, threadIdx.x + NTR * j, v[j][0], v[j][1], v[j][2]);
  }
  if constexpr (VT == 1) {
#pragma unroll
    for (int i = 0; i < 3; ++i) out[i] = v[0][i];
    lds_reduce<N, 3>(out, red, 0x2u);
  } else {
    lds_reduce_virtual_all<N, 3, NTR>(v, red, 0x2u, out);
  }
}

// Probe, large m: one work-group per tile forms the global clip 5 mean|S| from the tile
// statistics (the decision's own reduction, so the same clip) and, when some bucket reaches it,
// the tile's sum of min(|S|, clip) into tilestat[4 tile + 3] (fixed order: thread partials over
// the tile's row-major buckets, then the work-group reduction).  Replaces one work-group's pass
// over all m^2 buckets.
__global__ __launch_bounds__(kThreads) void clip_kernel(ProductArgs pa) {
  __shared__ double red[lds_reduce_doubles<kDecideThreads, 3>()];
  double tot[3];
  tile_totals<kThreads>(pa, red, tot);
  const int m = pa.m;
  const double mm = static_cast<double>(m) * m;
  const double mean_abs = tot[2] > 0.0 ? __builtin_nan("") : tot[0] / mm;
  const double clip = 5.0 * mean_abs;
  if (tot[2] == 0.0 && tot[1] <= clip) return;
  const int tile = blockIdx.x;
  const int ta = tile / pa.nt, tb = tile - ta * pa.nt;
  const int ts = pa.ts;
  double c2 = 0.0;
  for (int e0 = threadIdx.x; e0 < ts * ts; e0 += 16 * kThreads) {   // 16 loads in flight
    double a[16];
    bool ok[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int e = e0 + j * kThreads;
      const int r = ta * ts + e / ts, c = tb * ts + e % ts;
      ok[j] = e < ts * ts && r < m && c < m;
      a[j] = fabs(pa.S[ok[j] ? static_cast<int64_t>(r) * m + c : 0]);
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (ok[j]) c2 += a[j] < clip ? a[j] : clip;
    }
  }
  double r1[1] = {c2};
  lds_reduce<kThreads, 1>(r1, red, 0u);
  if (threadIdx.x == 0) pa.tilestat[tile * 4 + 3] = r1[0];
}

__global__ __launch_bounds__(kDecideThreads) void tile_decide_kernel(ProductArgs pa) {
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
  double lsum, lmax, lbad;
  tile_partials(pa, t, lsum, lmax, lbad);
  // (the same partials and tree as tile_totals, with the maxima of A and B as values 3 and 4)
  const float* mb = pa.maxpart_b != nullptr ? pa.maxpart_b : pa.maxpart + pa.nA;
  const float amax = strided_max(pa.maxpart, pa.nA, t, kDecideThreads, 0.0f);
  const float bmax = strided_max(mb, pa.nB, t, kDecideThreads, 0.0f);
  // sums: 0, 2; maxima: 1, 3, 4
  double r5[5] = {lsum, lmax, lbad, static_cast<double>(amax), static_cast<double>(bmax)};
  lds_reduce<kDecideThreads, 5>(r5, red, 0x1au);
  const double sum_abs = r5[0], max_abs = r5[1], nbad = r5[2];
  // mean|S| over all buckets (a non-finite bucket makes the mean non-finite)
  const double mean_abs = nbad > 0.0 ? __builtin_nan("") : sum_abs / static_cast<double>(mm);
  const double clip = 5.0 * mean_abs;
  // When no bucket reaches the clip (the usual clean case) the clipped sum is sum|S| itself and
  // S is not read again; otherwise a pass over S.
  double clipped = sum_abs;
  if (!(nbad == 0.0 && max_abs <= clip)) {
    double c2 = 0.0;
    if (pa.clip_tiles) {
      double e[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {       // at most 4096 tiles
        const int ti = t + j * kDecideThreads;
        e[j] = ti < ntiles ? pa.tilestat[ti * 4 + 3] : 0.0;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (t + j * kDecideThreads < ntiles) c2 += e[j];
      }
    } else {
#pragma unroll 8
      for (int64_t o = t; o < mm; o += kDecideThreads) {
        const double a = fabs(pa.S[o]);
        c2 += a < clip ? a : clip;
      }
    }
    double r1[1] = {c2};
    lds_reduce<kDecideThreads, 1>(r1, red, 0u);
    clipped = r1[0];
  }
  if (t == 0) decide_tail(pa, sum_abs, max_abs, nbad, clipped, r5[3], r5[4], acc0, acc1);
}

// ----------------------------------------------------------------------------------------
// Q from the k-major rows of the B work-groups: 64 x 64 tiles through LDS (rows padded to 65
// floats), read along the buckets and written along k, both coalesced.

__global__ __launch_bounds__(kThreads) void transpose_q_kernel(const float* src, float* dst,
                                                               int m, int64_t n2, int mq,
                                                               int ldp) {
  __shared__ float tile[64][65];
  const int64_t tk = static_cast<int64_t>(blockIdx.x) * 64;
  const int tb = blockIdx.y * 64;
  const int c = threadIdx.x & 63, r0 = threadIdx.x >> 6;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int r = r0 + 4 * j;
    const int64_t k = tk + r;
    const int b = tb + c;
    tile[r][c] = (k < n2 && b < m) ? src[k * mq + b] : 0.0f;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int r = r0 + 4 * j;
    const int b = tb + r;
    const int64_t k = tk + c;
    if (b < m && k < n2) dst[static_cast<int64_t>(b) * ldp + k] = tile[c][r];
  }
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

// One work-group of 256: the digit whose cumulative count passes k (the first bin b with
// k < count(bins 0..b), or bin 255 when none before it does); clears the histogram.  The
// cumulative counts come from an inclusive scan across the 256 threads.
__global__ __launch_bounds__(kThreads) void sel_step_kernel(SelState* st, uint32_t* hist) {
  static_assert(kThreads == 256, "one thread per digit");
  __shared__ uint32_t h[256];
  const int t = threadIdx.x;
  const uint64_t k = st->k;
  const uint32_t mine = hist[t];
  h[t] = mine;
  hist[t] = 0;
  __syncthreads();
  for (int d = 1; d < 256; d <<= 1) {
    const uint32_t add = t >= d ? h[t - d] : 0u;
    __syncthreads();
    h[t] += add;
    __syncthreads();
  }
  const uint64_t incl = h[t], excl = incl - mine;
  const bool hit = t == 255 ? excl <= k : (excl <= k && k < incl);
  if (hit) {
    const int shift = 56 - 8 * st->pass;
    st->prefix |= static_cast<uint64_t>(t) << shift;
    st->k = k - excl;
    st->count_eq = mine;
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
    if (R != nullptr) R[e.o] -= e.dr;
    if (T != nullptr) T[e.o] -= e.dt;
  }
}

// The moment sketches of Eq. 2 at the selected buckets only: for bucket o = a m + b,
// R = Pw[a] . Q[b] - R_C(a, b) and T = P[a] . Qw[b] - T_C(a, b), then the peel list's R and T
// terms at o, in list order.  One work-group per bucket: exact FP32 x FP32 products summed in
// FP64 over the factor rows (k-contiguous, zero past n2), threads combined in fixed order.
__global__ __launch_bounds__(kThreads) void moments_at_kernel(MomentsAtArgs g) {
  __shared__ double red[lds_reduce_doubles<kThreads, 2>()];
  const int q = blockIdx.x;
  const int64_t o = g.o[q];
  const int64_t a = o / g.m, b = o - (o / g.m) * g.m;
  const float* pw = g.Pw + a * g.ldp;
  const float* pp = g.P + a * g.ldp;
  const float* qq = g.Q + b * g.ldp;
  const float* qw = g.Qw + b * g.ldp;
  double v[2] = {0.0, 0.0};
  for (int k = 4 * threadIdx.x; k < g.kact; k += 4 * kThreads) {
    const f32x4 x1 = *reinterpret_cast<const f32x4*>(pw + k);
    const f32x4 y1 = *reinterpret_cast<const f32x4*>(qq + k);
    const f32x4 x2 = *reinterpret_cast<const f32x4*>(pp + k);
    const f32x4 y2 = *reinterpret_cast<const f32x4*>(qw + k);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[0] = fma(static_cast<double>(x1[e]), static_cast<double>(y1[e]), v[0]);
      v[1] = fma(static_cast<double>(x2[e]), static_cast<double>(y2[e]), v[1]);
    }
  }
  lds_reduce<kThreads, 2>(v, red, 0u);
  if (threadIdx.x != 0) return;
  const int64_t mm = static_cast<int64_t>(g.m) * g.m;
  for (int p = 0; p < g.npc; ++p) {
    v[0] -= g.partR[p * mm + o];
    v[1] -= g.partT[p * mm + o];
  }
  for (int p = 0; p < g.npeel; ++p) {
    if (g.peel[p].o == o) {
      v[0] -= g.peel[p].dr;
      v[1] -= g.peel[p].dt;
    }
  }
  g.r[q] = v[0];
  g.t[q] = v[1];
}

// Apply step of Algorithm 2: one thread per record (the coordinates are distinct).
__global__ __launch_bounds__(kThreads) void apply_kernel(float* C, const ApplyEntry* list,
                                                         int n) {
  const int t = static_cast<int>(blockIdx.x) * kThreads + static_cast<int>(threadIdx.x);
  if (t >= n) return;
  const ApplyEntry e = list[t];
  C[e.o] = e.absolute ? static_cast<float>(e.d)
                      : static_cast<float>(static_cast<double>(C[e.o]) + e.d);
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
      if (p < cap) out[p] = Cand{i, s, R != nullptr ? R[i] : 0.0, T != nullptr ? T[i] : 0.0};
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
                                                           int64_t bsk, int64_t bsj,
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
    const double b = static_cast<double>(half_bits_to_float<DT>(B[k * bsk + j * bsj]));
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
    if (dec && a.clip_tiles) {                                                              \
      launch_k(clip_kernel, rgrid, dim3(kThreads), 0, st, nullptr, nullptr, a);             \
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

// Zeroes columns [c0, c1) of `rows` rows of a row-major FP32 matrix whose rows are ld apart.
__global__ __launch_bounds__(kThreads) void zero_cols_kernel(float* base, int rows, int ld,
                                                             int c0, int c1) {
  const int64_t w = c1 - c0;
  const int64_t total = static_cast<int64_t>(rows) * w;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * kThreads) {
    const int64_t r = i / w;
    base[r * ld + c0 + (i - r * w)] = 0.0f;
  }
}

hipError_t launch_zero_cols(float* base, int rows, int ld, int c0, int c1, hipStream_t st) {
  if (rows <= 0 || c1 <= c0) return hipSuccess;
  if (c0 < 0 || c1 > ld) return hipErrorInvalidValue;
  const int64_t total = static_cast<int64_t>(rows) * (c1 - c0);
  const int grid = static_cast<int>(std::min<int64_t>(256, (total + kThreads - 1) / kThreads));
  hipLaunchKernelGGL(zero_cols_kernel, dim3(grid), dim3(kThreads), 0, st, base, rows, ld, c0, c1);
  return hipGetLastError();
}

hipError_t launch_apply(float* C, const ApplyEntry* list, int n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(apply_kernel, dim3((n + kThreads - 1) / kThreads), dim3(kThreads), 0, st, C,
                     list, n);
  return hipGetLastError();
}

hipError_t launch_above(const double* S, const double* R, const double* T, int64_t n,
                        double cut, Cand* out, uint32_t cap, uint32_t* count, hipStream_t st) {
  hipLaunchKernelGGL(above_kernel, dim3(grid_for(n)), dim3(kThreads), 0, st, S, R, T, n, cut,
                     out, cap, count);
  return hipGetLastError();
}

hipError_t launch_moments_at(const MomentsAtArgs& g, int n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(moments_at_kernel, dim3(static_cast<unsigned>(n)), dim3(kThreads), 0, st, g);
  return hipGetLastError();
}

hipError_t launch_transpose_q(const float* src, float* dst, int m, int64_t n2, int mq, int ldp,
                              hipStream_t st) {
  if (m <= 0 || n2 <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((n2 + 63) / 64), static_cast<unsigned>((m + 63) / 64));
  hipLaunchKernelGGL(transpose_q_kernel, grid, dim3(kThreads), 0, st, src, dst, m, n2, mq, ldp);
  return hipGetLastError();
}

hipError_t launch_recheck(const uint16_t* A, const uint16_t* B, int64_t bsk, int64_t bsj,
                          const float* C, int64_t n2, int64_t n3, int dt, const int64_t* coords,
                          int n, double* gamma, double* abssum, float* cval, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const unsigned grid = static_cast<unsigned>((n + 3) / 4);
  if (dt == 1) {
    hipLaunchKernelGGL(recheck_kernel<1>, dim3(grid), dim3(kThreads), 0, st, A, B, bsk, bsj, C,
                       n2, n3, coords, n, gamma, abssum, cval);
  } else {
    hipLaunchKernelGGL(recheck_kernel<0>, dim3(grid), dim3(kThreads), 0, st, A, B, bsk, bsj, C,
                       n2, n3, coords, n, gamma, abssum, cval);
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

#ifdef FPSK_WG_TIMELINE
// Copies the records of the last block-product launch (its first max_records slots) and of the
// last decision (the final slot) to host memory, out[0 .. 4 max_records) and
// out[4 max_records .. + 4); synchronous.  Returns 0, or -1 on a bad argument or a failed copy.
// Exported by the diagnostic build only.
extern "C" int fpsketch_wg_timeline_tail(unsigned long long* out, int64_t max_records) {
  if (out == nullptr || max_records < 1) return -1;
  const int64_t n = max_records < fpsk::kTimelineMax - 1 ? max_records : fpsk::kTimelineMax - 1;
  const size_t rec = 4 * sizeof(unsigned long long);
  if (hipMemcpyFromSymbol(out, HIP_SYMBOL(fpsk::wg_timeline_tail), static_cast<size_t>(n) * rec,
                          0, hipMemcpyDeviceToHost) != hipSuccess) {
    return -1;
  }
  return hipMemcpyFromSymbol(out + 4 * max_records, HIP_SYMBOL(fpsk::wg_timeline_tail), rec,
                             static_cast<size_t>(fpsk::kTimelineMax - 1) * rec,
                             hipMemcpyDeviceToHost) == hipSuccess ? 0 : -1;
}
#endif
