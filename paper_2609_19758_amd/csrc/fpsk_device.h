// Device-side helpers shared by the gfx950 kernels of the FP-Sketch verifier: vector types,
// half-precision element access, loads with a zero buffer in place of branches, and the
// launcher that lets dispatch packets time-stamp events.
#pragma once

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

// ----------------------------------------------------------------------------------------
// Work-group timeline, compiled only with FPSK_WG_TIMELINE (a diagnostic build of the library;
// the build the binding loads has none of it).  A work-group that holds a WgStamp leaves one
// record of four words at slot `slot` of `base`: its start and end on the 100 MHz constant
// clock, the XCD and the hardware-id word of the CU it ran on, and the launch's work-group
// count with the work-group's type.  Thread 0 stamps the end after the kernel's last block
// reduction, so the record spans the whole work-group.  Each launch overwrites the records of
// the one before.
#ifdef FPSK_WG_TIMELINE
constexpr int kTimelineMax = 1 << 16;

struct WgStamp {
  unsigned long long* rec;
  unsigned long long t0;
  int type;
  __device__ WgStamp(unsigned long long* base, unsigned slot, int ty)
      : rec(slot < static_cast<unsigned>(kTimelineMax) ? base + 4 * slot : nullptr),
        t0(__builtin_amdgcn_s_memrealtime()), type(ty) {}
  __device__ ~WgStamp() {
    if (threadIdx.x == 0 && rec != nullptr) {
      const unsigned long long t1 = __builtin_amdgcn_s_memrealtime();
      const unsigned hw = __builtin_amdgcn_s_getreg((31 << 11) | 4);     // HW_ID, 32 bits
      const unsigned xcc = __builtin_amdgcn_s_getreg((15 << 11) | 20);   // XCC_ID, 16 bits
      rec[0] = t0;
      rec[1] = t1;
      rec[2] = (static_cast<unsigned long long>(xcc & 15u) << 32) | hw;
      rec[3] = (static_cast<unsigned long long>(gridDim.x) << 8) | static_cast<unsigned>(type);
    }
  }
};
#endif

}  // namespace fpsk
