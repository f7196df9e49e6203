// Internal interface between the host library and the gfx950 kernels of the FP-Sketch verifier.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace fpsk {

constexpr int kThreads = 256;          // work-group size of every kernel (4 wave64)
constexpr int kColTile = 512;          // columns per A or C tile: 64 lanes x 8 elements
constexpr int kBChunkHalfs = 16384;    // halfs of B staged in LDS per chunk (32 KiB)
constexpr int kMaxM = 4096;            // largest bucket count the kernels accept
constexpr double kHugeLimit = 3.4028234663852886e38 / 16.0;   // fp32max / 16
// block product of the probe (m <= 64)
constexpr int kXSlice = 4096;            // k per block-product work-group
constexpr int kMaxXSlices = 4;           // n2 <= kMaxXSlices * kXSlice

// One pass over A, B and C producing the factors of Eq. 1 (and their weighted forms).
struct StreamArgs {
  const uint16_t* A;          // n1 x n2 half bits
  const uint16_t* B;          // n2 x n3 half bits, or with transb its transpose W (n3 x n2)
  const float* C;             // n1 x n3
  int64_t n1, n2, n3;
  int m;
  // row side: per bucket a, its rows at perm[a * cap + i] (ascending) as row | (v1 < 0) << 31,
  // padded to cap entries with -1
  const int32_t* perm;
  int cap;
  // transb: B is passed as W = B^T (n3 x n2 row-major) and the nB B work-groups are row-bucket
  // work-groups over W's rows (m x TA of them, like A's), with the column lists perm2 / cap2
  // (per bucket b its columns j ascending as j | (v2 < 0) << 31, natural bucket order)
  int transb;
  const int32_t* perm2;
  int cap2;
  // C column tiles of kColTile: per tile (ctab_stride entries), columns sorted by bucket as
  // (offset in tile) | (v2 < 0) << 15, with coff[t * (m + 1) + b] segment starts; for m <= 256
  // each segment is padded to a multiple of 8 with the sentinel offset kColTile (a zero column)
  const uint16_t* ctab;
  const int32_t* coff;
  // B column chunks of cwb columns: sorted lists without signs (the signs v2(j) are applied when
  // a chunk is staged, from the bit mask bsign: bit j % 8 of byte j / 8); entries are the
  // column offset with moments, else the column's staged LDS slot (sentinel cwb)
  const uint8_t* bsign;
  const uint16_t* btab;
  const int32_t* boff;
  int cwb;
  int ctab_stride, btab_stride;
  int tab_off;                // byte offset of the staged column list in dynamic LDS
  // outputs
  // factors, row stride ldp >= n2 (a multiple of 4; entries past n2 are kept at zero)
  float* P;        // m x ldp      H1 A
  float* Pw;       // m x ldp      H1 W1 A            (moments only)
  float* Q;        // m x ldp      (B H2^T)^T: row b holds column b of B H2^T
  float* Qw;       // m x ldp      (B W2 H2^T)^T      (moments only)
  int ldp;
  // B work-groups of 1 or 2 rows (m > 1024) write Q (Qw) k-major instead, n2 x mq, for a
  // transpose into Q: a bucket-major row per work-group would be an 8-byte or smaller piece per
  // bucket; null otherwise
  float* Qk;
  float* Qwk;
  int mq;
  double* partS;   // npc x m x m  partial H1 C H2^T over column-tile groups
  double* partR;   // npc x m x m  partial H1 W1 C H2^T
  double* partT;   // npc x m x m  partial H1 C W2 H2^T
  float* maxpart;  // nA + nB: max |A| per A work-group, then max |B| per B work-group
  // C entries replaced while sketching (absolute entries): CSR by row, may be null
  const int32_t* patch_rowptr;
  const int32_t* patch_col;
  const float* patch_val;
  // decomposition
  int nA, nB, nC;
  // dispatch order after the C work-groups: A then B when an A work-group reads at least as many
  // bytes as a B work-group (the smaller ones last, where they fill the tail), else B then A
  int a_first;
  int TA, TC, TB;
  int npc, tg;
  // small buckets: row-bucket work-groups of four tiles, one per wave (A side; W side with
  // transb), m x ceil(TA / 4) of them
  int wt_a, wt_w;
  // C work-groups with one column tile per wave, four tiles at a time (256 < m <= 1024,
  // buckets of at most 32 rows, at least 4 tiles per work-group)
  int wt_c;
  // the 4-row probe B work-groups of the one-tile-per-wave instances start at chunk
  // (row block mod TB) and wrap (n3 a whole number of chunks, TB > 1)
  int rot_b;
  double inv_l1, inv_l3;      // 1 / 2^ceil(log2 n1), 1 / 2^ceil(log2 n3)
  int vec_a, vec_b, vec_c;    // 16-byte vector loads allowed
  const void* zero;           // >= 64 bytes of zeros (read in place of invalid rows or lanes)
};

// Bucket-space product S = P Q - S_C (and R = Pw Q - R_C, T = P Qw - T_C), plus the probe
// decision.
struct ProductArgs {
  const float* P;
  const float* Pw;
  const float* Q;
  const float* Qw;
  const double* partS;
  const double* partR;
  const double* partT;
  double* S;
  double* R;
  double* T;
  double* scratch;      // NS x tiles x ts^2 (x 3 with moments) slice partials, row-major tiles
  double* tilestat;     // tiles x 4: sum|S|, max|S|, non-finite count, clipped sum
  int m, n2, nt, NS, ksl, npc;
  int ldp;              // row stride of the factors
  int kact;             // k-range the products cover: n2 rounded up to a multiple of 4
  int mode;             // 0: sketch only; 1: probe decision
  int ts;               // tile edge of the tile path
  int clip_tiles;       // probe, large m: clip_kernel writes each tile's clipped sum to
                        // tilestat[4 tile + 3] and the decision adds those
  const float* maxpart;
  int nA, nB;
  const float* maxpart_b; // max |B| per B work-group when the B side is cached, else null
  double* stats;        // [8] sigma_hat, thr, tau, max|S|, finite, dirty, max|A|, max|B|
  int32_t* d_dirty;     // caller's flag (may be null)
  double* sigma_acc;    // [2] running sum of clean sigma_hat, count
  double mu, c_valid;
  double lim_factor;    // mu sqrt(2 ln m^2): the noise limit in units of sigma_hat
  // probe with m <= 64 (nX > 0): nX = xnb^2 xns block-product work-groups of xb x xb outputs
  // over k-slices of kXSlice, their partials in xpart (xns x m x m, slice 0 minus the C grid)
  int nX, xb, xnb, xns;
  // launch index i -> slot (i mod 8) nX / 8 + i / 8; xslots slots per slice, in supertiles of
  // xsr x xsc blocks, xnstc supertiles per row of blocks (slots past the grid are idle)
  int xsr, xsc, xnstc, xslots;
  double* xpart;
};

// e0 / e1 (may be null): events that the first / last dispatch of the call records its
// start / end time in.
// Pipelined probe launch (m <= 64, block path): the decision of `dec` (if has_dec), the nprod
// block products of `prod` and the stream pass of `s` (which may be empty: nA = nB = nC = 0).
// lds_bytes covers the stream pass and probe_pipe_lds(xb).
size_t probe_pipe_lds(int xb);
hipError_t launch_probe_pipe(const StreamArgs& s, const ProductArgs& prod, const ProductArgs& dec,
                             int nprod, int has_dec, int dt, int xb, size_t lds_bytes,
                             hipStream_t st, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
hipError_t launch_stream(const StreamArgs& s, int dt, bool moments, int rb, int g, int ng,
                         size_t lds_bytes, hipStream_t st, hipEvent_t e0 = nullptr,
                         hipEvent_t e1 = nullptr);
// ts, kw: product tile edge and whether its k-range is split over the 4 waves
hipError_t launch_product(const ProductArgs& a, int ts, bool kw, bool moments, hipStream_t st,
                          hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
hipError_t launch_scan_count(const float* C, int64_t n1, int64_t n3, int32_t* counts,
                             hipStream_t st);
hipError_t launch_scan_extract(const float* C, int64_t n3, const int32_t* rows,
                               const int32_t* base, int nrows, int32_t cap, int64_t* out,
                               hipStream_t st);
hipError_t launch_sample(const float* C, int64_t stride, int64_t count, float* out,
                         hipStream_t st);
// B[k][j] is read at B + k * bsk + j * bsj (n3, 1 for B as stored; 1, n2 for W = B^T).
// dst (m x ldp) = transpose of src (n2 x mq), columns past m and rows past n2 left alone.
hipError_t launch_transpose_q(const float* src, float* dst, int m, int64_t n2, int mq, int ldp,
                              hipStream_t st);
hipError_t launch_recheck(const uint16_t* A, const uint16_t* B, int64_t bsk, int64_t bsj,
                          const float* C, int64_t n2, int64_t n3, int dt, const int64_t* coords,
                          int n, double* gamma, double* abssum, float* cval, hipStream_t st);

// Order statistics of a bucket grid on the device (the MAD and candidate scan of a localize
// round).  The selection state lives in device memory.
struct SelState {
  uint64_t prefix;     // key bits fixed so far
  uint64_t k;          // rank sought among the keys that match the prefix
  uint64_t next;       // smallest key above the selected one
  uint32_t count_eq;   // keys equal to the selected one (after the last digit)
  int32_t pass;        // digits fixed so far
  double med;          // median of S
  double mad;          // median of |S - med|
};
struct PeelEntry {     // S[o] -= ds, R[o] -= dr, T[o] -= dt
  int64_t o;
  double ds, dr, dt;
};
// Moment sketches R, T at a list of n buckets o (launch_moments_at): the factors (rows ldp
// apart, zero from n2 to kact), the npc C-grid partials of R and T, the peel list.
struct MomentsAtArgs {
  const float* P;
  const float* Pw;
  const float* Q;
  const float* Qw;
  const double* partR;
  const double* partT;
  const int64_t* o;
  const PeelEntry* peel;
  double* r;
  double* t;
  int m, ldp, kact, npc, npeel;
};
hipError_t launch_moments_at(const MomentsAtArgs& g, int n, hipStream_t st);
struct ApplyEntry {    // one record of the apply step: C[o] <- d, or C[o] + d
  int64_t o;
  double d;
  int32_t absolute;
  int32_t pad;
};
hipError_t launch_apply(float* C, const ApplyEntry* list, int n, hipStream_t st);
// Zeroes columns [c0, c1) of rows x ld FP32 rows (c1 <= ld).
hipError_t launch_zero_cols(float* base, int rows, int ld, int c0, int c1, hipStream_t st);
struct Cand {          // a bucket above the cut with its three sketches
  int64_t o;
  double s, r, t;
};
// Applies the peel list in order (one thread), so the result equals sequential subtraction.
hipError_t launch_peel(double* S, double* R, double* T, const PeelEntry* list, int n,
                       hipStream_t st);
// st->med = median of S[0 .. n), then st->mad = median of |S - med| (even counts: the mean of
// the two middle order statistics; NaN orders above +inf).  hist: 256 words of scratch, zero
// on entry and on return.
hipError_t launch_median_mad(const double* S, int64_t n, SelState* st, uint32_t* hist,
                             hipStream_t st_);
// Appends (o, S, R, T) of every bucket with |S[o]| > cut to out (at most cap; *count receives
// the number found, which may exceed cap); the order of the entries is unspecified.
hipError_t launch_above(const double* S, const double* R, const double* T, int64_t n,
                        double cut, Cand* out, uint32_t cap, uint32_t* count, hipStream_t st);

hipError_t launch_read(const void* src, int64_t bytes, uint32_t* out, int grid, hipStream_t st);
hipError_t launch_copy(const void* src, void* dst, int64_t bytes, int grid, hipStream_t st);

}  // namespace fpsk
