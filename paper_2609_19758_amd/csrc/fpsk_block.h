// The probe's decision and its block product for m <= 64 as device functions, shared by the
// stand-alone kernels (fpsk_kernels.hip) and the pipelined probe launch (fpsk_stream.hip), plus
// the fixed-order work-group reductions they use.
#pragma once

#include "fpsk_device.h"

namespace fpsk {

constexpr int kDecideThreads = 1024;

// Fixed-order work-group reduction through LDS (cross-lane shuffles of doubles cost tens of
// cycles each).  N entries per value, held by NTR real threads (N / NTR each).  Levels of 16:
// at a level over N entries, pair (value i, group g < N / 16) combines entries g, g + N / 16,
// ..., g + 15 N / 16 (consecutive threads read consecutive addresses; the 16 reads are issued
// together), until at most 16 remain, which one thread per value combines in order.  Bit i of
// max_mask selects max instead of sum for value i.  The order depends on N only, so a
// reduction over N virtual threads gives the same bits whatever NTR holds them.
template <int N, int NV, int NTR>
__device__ __forceinline__ void lds_reduce_level(const double* src, double* dst,
                                                 uint32_t max_mask) {
  if constexpr (N <= 16) {
    for (int i = threadIdx.x; i < NV; i += NTR) {
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
    for (int p = threadIdx.x; p < NV * GN; p += NTR) {
      const int i = p / GN, g = p - i * GN;
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
    lds_reduce_level<GN, NV, NTR>(dst, dst + NV * GN, max_mask);
  }
}

// Doubles of LDS that a reduction of NV values over N entries uses.
template <int N, int NV>
constexpr int lds_reduce_doubles() { return NV * (N + 2 * N / 16 + 1); }

// Where the results of a reduction over N entries land, after the level outputs.
template <int N, int NV>
__device__ __forceinline__ const double* lds_reduce_result(const double* buf) {
  const double* res = buf + NV * N;
  int n = N;
  while (n > 16) {
    res += NV * (n / 16);
    n /= 16;
  }
  return res;
}

// NT threads, NV values each; every thread receives the results in v.
template <int NT, int NV>
__device__ void lds_reduce(double (&v)[NV], double* buf, uint32_t max_mask) {
  static_assert(NT % 16 == 0 && NT <= 4096, "levels of 16");
#pragma unroll
  for (int i = 0; i < NV; ++i) buf[i * NT + threadIdx.x] = v[i];
  __syncthreads();
  lds_reduce_level<NT, NV, NT>(buf, buf + NV * NT, max_mask);
  const double* res = lds_reduce_result<NT, NV>(buf);
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = res[i];
  __syncthreads();
}

// N virtual threads held by NTR real threads (virtual thread threadIdx.x + NTR j holds v[j]),
// the values reduced one at a time in a buffer of lds_reduce_doubles<N, 1>() doubles; the
// results (in out, for every thread) equal lds_reduce<N, NV> over N real threads.
template <int N, int NV, int NTR>
__device__ void lds_reduce_virtual(const double (&v)[N / NTR][NV], double* buf,
                                   uint32_t max_mask, double (&out)[NV]) {
  static_assert(N % NTR == 0 && N % 16 == 0 && N <= 4096, "levels of 16");
  constexpr int VT = N / NTR;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
#pragma unroll
    for (int j = 0; j < VT; ++j) buf[threadIdx.x + NTR * j] = v[j][i];
    __syncthreads();
    lds_reduce_level<N, 1, NTR>(buf, buf + N, (max_mask >> i) & 1u);
    out[i] = lds_reduce_result<N, 1>(buf)[0];
    __syncthreads();
  }
}

// As lds_reduce_virtual, all NV values in one pass through a buffer of
// lds_reduce_doubles<N, NV>() doubles (fewer barriers, more LDS).
template <int N, int NV, int NTR>
__device__ void lds_reduce_virtual_all(const double (&v)[N / NTR][NV], double* buf,
                                       uint32_t max_mask, double (&out)[NV]) {
  static_assert(N % NTR == 0 && N % 16 == 0 && N <= 4096, "levels of 16");
  constexpr int VT = N / NTR;
#pragma unroll
  for (int i = 0; i < NV; ++i)
#pragma unroll
    for (int j = 0; j < VT; ++j) buf[i * N + threadIdx.x + NTR * j] = v[j][i];
  __syncthreads();
  lds_reduce_level<N, NV, NTR>(buf, buf + NV * N, max_mask);
  const double* res = lds_reduce_result<N, NV>(buf);
#pragma unroll
  for (int i = 0; i < NV; ++i) out[i] = res[i];
  __syncthreads();
}

// max of p[i] over i = t, t + stride, ... below n, with the loads issued eight at a time (a
// loop of single loads waits one round trip per entry)
__device__ __forceinline__ float strided_max(const float* p, int n, int t, int stride, float mx) {
  for (int i0 = t; i0 < n; i0 += 8 * stride) {
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int i = i0 + j * stride;
      x[j] = i < n ? p[i] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) mx = fmaxf(mx, x[j]);
  }
  return mx;
}

// The probe's decision from the reduced statistics (Sec. III-B): clipped-mean noise estimate,
// validity bound from max|A| and max|B|, threshold and verdict.
__device__ inline void decide_tail(const ProductArgs& pa, double sum_abs, double max_abs,
                                   double nbad, double clipped, double maxA, double maxB,
                                   double acc0, double acc1) {
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

// ----------------------------------------------------------------------------------------
// Probe product for m <= 64: block products, then one deciding work-group.
//   block_product_body (block, slice): outputs (a0 .. a0 + XB) x (b0 .. b0 + XB) over the
//     k-slice [slice * kXSlice, + kXSlice).  Thread t takes k = 4 (t + 256 j) within the slice;
//     the dot products run in FP64 on the FP32 factors (rows of P and of the transposed Q, both
//     k-contiguous, read with 16-byte loads that the work-groups of an XCD share through its L2);
//     the 4 waves are combined in fixed order.  Slice 0 subtracts the C grid (the sum of the
//     column-group partials).  JH loads per factor row are in flight at a time; the summation
//     order does not depend on it.
//   block_decide_body (one work-group): S = sum of the slice partials in slice order (kept
//     in registers, not stored), the probe statistics and the verdict.  Its reductions run over
//     kDecideThreads virtual threads, so any work-group size gives the same bits.

// Block i of nblk (nblk a multiple of 8; the 8 XCDs take indices round-robin, and index i maps
// to slot (i mod 8) nblk / 8 + i / 8, so each XCD runs a contiguous range of slots).  red holds
// lds_reduce_doubles<kThreads, NVP>() doubles; the XB^2 outputs are reduced NVP at a time.
template <int XB, int JHMAX, int NVP>
__device__ void block_product_body(const ProductArgs& pa, int i, int nblk, double* red) {
  constexpr int NV = XB * XB;
  static_assert(NV % NVP == 0, "whole reduction passes");
  const int m = pa.m;
  const int64_t mm = static_cast<int64_t>(m) * m;
  // XCD-local slot of this launch index, then its slice and output block
  const int per = nblk / 8;
  const int slot = (i & 7) * per + (i >> 3);
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
  for (int r = 0; r < XB; ++r) {
    prow[r] = pa.P + static_cast<int64_t>(a0 + r < m ? a0 + r : m - 1) * pa.ldp;
    qrow[r] = pa.Q + static_cast<int64_t>(b0 + r < m ? b0 + r : m - 1) * pa.ldp;
  }
  // every load of a round is issued before the first is used: the slice's factor rows, then
  // the C grid of the block (slice 0; thread (v = t & 15, group t >> 4) takes every 16th
  // column-group partial)
  const int kb = slice * kXSlice;
  constexpr int NJ = kXSlice / (4 * kThreads);
  constexpr int JH = JHMAX < NJ ? JHMAX : NJ;
  double acc[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) acc[v] = 0.0;
  double c4[4];
  const int cv = threadIdx.x & 15, gs = threadIdx.x >> 4;
  const int ci = cv / XB, cj = cv - (cv / XB) * XB;
  const bool vok = slice == 0 && cv < NV && a0 + ci < m && b0 + cj < m;
  const int64_t co = vok ? static_cast<int64_t>(a0 + ci) * m + b0 + cj : 0;
#pragma unroll
  for (int h = 0; h < NJ / JH; ++h) {
    float4 pv[XB][JH], qv[XB][JH];
#pragma unroll
    for (int j = 0; j < JH; ++j) {
      const int k = kb + 4 * (static_cast<int>(threadIdx.x) + kThreads * (h * JH + j));
      const bool kok = k < pa.kact;
      const int kk = kok ? k : 0;
#pragma unroll
      for (int r = 0; r < XB; ++r) {
        const float4 p = *reinterpret_cast<const float4*>(prow[r] + kk);
        const float4 qq = *reinterpret_cast<const float4*>(qrow[r] + kk);
        const float4 z = {0.f, 0.f, 0.f, 0.f};
        pv[r][j] = kok ? p : z;
        qv[r][j] = kok ? qq : z;
      }
    }
    if (h == 0) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int g = gs + 16 * u;
        const double c = pa.partS[static_cast<int64_t>(g < pa.npc ? g : 0) * mm + co];
        c4[u] = (vok && g < pa.npc) ? c : 0.0;
      }
    }
#pragma unroll
    for (int j = 0; j < JH; ++j)
#pragma unroll
      for (int r = 0; r < XB; ++r)
#pragma unroll
        for (int c = 0; c < XB; ++c) {
          double t = acc[r * XB + c];
          t = fma(static_cast<double>(pv[r][j].x), static_cast<double>(qv[c][j].x), t);
          t = fma(static_cast<double>(pv[r][j].y), static_cast<double>(qv[c][j].y), t);
          t = fma(static_cast<double>(pv[r][j].z), static_cast<double>(qv[c][j].z), t);
          t = fma(static_cast<double>(pv[r][j].w), static_cast<double>(qv[c][j].w), t);
          acc[r * XB + c] = t;
        }
  }
  double cp = (c4[0] + c4[1]) + (c4[2] + c4[3]);
  for (int g = gs + 64; g < pa.npc; g += 16) {   // more than 64 column groups (small m)
    cp += vok ? pa.partS[static_cast<int64_t>(g) * mm + co] : 0.0;
  }
#pragma unroll
  for (int v0 = 0; v0 < NV; v0 += NVP) {
    double part[NVP];
#pragma unroll
    for (int v = 0; v < NVP; ++v) part[v] = acc[v0 + v];
    lds_reduce<kThreads, NVP>(part, red, 0u);
#pragma unroll
    for (int v = 0; v < NVP; ++v) acc[v0 + v] = part[v];
  }
  // C grid of output v: the 16 column-group sums of threads v, 16 + v, ... in order
  red[threadIdx.x] = cp;
  __syncthreads();
  if (static_cast<int>(threadIdx.x) < NV) {
    const int v = threadIdx.x;
    const int r = v / XB, c = v - (v / XB) * XB;
    double cg = 0.0;
    for (int g = 0; g < 16; ++g) cg += red[g * 16 + v];
    if (a0 + r < m && b0 + c < m) {
      pa.xpart[slice * mm + static_cast<int64_t>(a0 + r) * m + b0 + c] = acc[v] - cg;
    }
  }
}

// NTR real threads (a multiple of 64 dividing kDecideThreads); red holds
// lds_reduce_doubles<kDecideThreads, 1>() doubles when NTR < kDecideThreads, else
// lds_reduce_doubles<kDecideThreads, 5>().  SB slices' loads are issued before their sums.
template <int NTR, int SB>
__device__ void block_decide_body(const ProductArgs& pa, double* red) {
  constexpr int N = kDecideThreads;
  constexpr int VT = N / NTR;
  constexpr int NQ = 4096 / N;                // m <= 64: m^2 <= 4096 outputs
  const int m = pa.m;
  const int mm = m * m;
  const int t = threadIdx.x;
  // virtual thread t + NTR j holds outputs o = t + NTR j + N q; the first slice's partials and
  // the first share of the maxima are loaded together; only outputs that exist are loaded
  double v[VT][NQ];
#pragma unroll
  for (int j = 0; j < VT; ++j)
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int o = t + NTR * j + N * q;
      v[j][q] = o < mm ? pa.xpart[o] : 0.0;
    }
  // the running noise sum, read now so that the verdict does not wait on it
  double acc0 = 0.0, acc1 = 0.0;
  if (t == 0) {
    acc0 = pa.sigma_acc[0];
    acc1 = pa.sigma_acc[1];
  }
  const float* mb = pa.maxpart_b != nullptr ? pa.maxpart_b : pa.maxpart + pa.nA;
  float amax = t < pa.nA ? pa.maxpart[t] : 0.0f;
  float bmax = t < pa.nB ? mb[t] : 0.0f;
  // the other slices in slice order
  for (int sl0 = 1; sl0 < pa.xns; sl0 += SB) {
    double x[SB][VT][NQ];
#pragma unroll
    for (int s = 0; s < SB; ++s)
#pragma unroll
      for (int j = 0; j < VT; ++j)
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          const int o = t + NTR * j + N * q;
          x[s][j][q] = (sl0 + s < pa.xns && o < mm)
                           ? pa.xpart[static_cast<int64_t>(sl0 + s) * mm + o] : 0.0;
        }
#pragma unroll
    for (int s = 0; s < SB; ++s) {
      if (sl0 + s < pa.xns) {
#pragma unroll
        for (int j = 0; j < VT; ++j)
#pragma unroll
          for (int q = 0; q < NQ; ++q) v[j][q] += x[s][j][q];
      }
    }
  }
  // maxima are exact whatever the grouping
  amax = strided_max(pa.maxpart, pa.nA, t + NTR, NTR, amax);
  bmax = strided_max(mb, pa.nB, t + NTR, NTR, bmax);
  double r5[VT][5];
#pragma unroll
  for (int j = 0; j < VT; ++j) {
    double lsum = 0.0, lmax = 0.0, lbad = 0.0;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int o = t + NTR * j + N * q;
      if (o < mm) {
        const double av = fabs(v[j][q]);
        if (__builtin_isfinite(v[j][q])) {
          lsum += av;
          lmax = fmax(lmax, av);
        } else {
          lbad += 1.0;
        }
      }
    }
    r5[j][0] = lsum;
    r5[j][1] = lmax;
    r5[j][2] = lbad;
    r5[j][3] = j == 0 ? static_cast<double>(amax) : 0.0;
    r5[j][4] = j == 0 ? static_cast<double>(bmax) : 0.0;
  }
  // the five first-phase reductions (sums: 0, 2; maxima: 1, 3, 4)
  double s5[5];
  if constexpr (VT == 1) {
#pragma unroll
    for (int i = 0; i < 5; ++i) s5[i] = r5[0][i];
    lds_reduce<N, 5>(s5, red, 0x1au);
  } else {
    lds_reduce_virtual<N, 5, NTR>(r5, red, 0x1au, s5);
  }
  const double sum_abs = s5[0], max_abs = s5[1], nbad = s5[2];
  const double mean_abs = nbad > 0.0 ? __builtin_nan("") : sum_abs / static_cast<double>(mm);
  const double clip = 5.0 * mean_abs;
  // When no bucket reaches the clip (the usual clean case) the clipped sum is sum|S| itself:
  // the same terms in the same order through the same reduction tree.  Otherwise a second pass.
  double clipped = sum_abs;
  if (!(nbad == 0.0 && max_abs <= clip)) {
    double c2[VT][1];
#pragma unroll
    for (int j = 0; j < VT; ++j) {
      c2[j][0] = 0.0;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int o = t + NTR * j + N * q;
        if (o < mm) {
          const double a = fabs(v[j][q]);
          c2[j][0] += a < clip ? a : clip;
        }
      }
    }
    double s1[1];
    if constexpr (VT == 1) {
      s1[0] = c2[0][0];
      lds_reduce<N, 1>(s1, red, 0u);
    } else {
      lds_reduce_virtual<N, 1, NTR>(c2, red, 0u, s1);
    }
    clipped = s1[0];
  }
  if (t == 0) decide_tail(pa, sum_abs, max_abs, nbad, clipped, s5[3], s5[4], acc0, acc1);
}

}  // namespace fpsk
