/*
 * fpsketch.h — C ABI of the FP-Sketch post hoc GEMM verifier for AMD Instinct MI355X (gfx950).
 *
 * The verifier runs after an unmodified half-precision GEMM whose output C is delivered in FP32
 * (paper: "Sketching the Error, Not the Product", arXiv 2609.19758, Sec. II-A and III).  With
 * A (n1 x n2) and B (n2 x n3) in FP16 or BF16 and C (n1 x n3) in FP32, it
 *   - probes: forms the sum sketch S = H1 E H2^T of E = AB - C without forming AB (Eq. 1) and
 *     decides clean/dirty against the probe threshold (Sec. III-C, III-E, III-I, Algorithm 2);
 *   - localizes: on a dirty product, forms first-moment sketches R, T with power-of-two scaled
 *     index weights, recovers each isolated error as a ratio (Eq. 2) and keeps a candidate
 *     entry only when recomputing its dot product afresh differs from C beyond the rounding
 *     bound (Sec. III-D, Algorithm 1), over k peeled hash rounds (Sec. III-H), after an exact
 *     scan for non-finite and out-of-range entries (Sec. III-I);
 *   - recalibrates the probe's bucket count from noise measured on clean calls (Sec. III-G).
 *
 * Conventions (all entry points):
 *   - Matrices are dense row-major with no padding: A[i*n2 + k], B[k*n3 + j], C[i*n3 + j].
 *   - Matrix arguments are DEVICE pointers on the context's device, owned by the caller; the
 *     library never frees or writes them (localize does not modify C, Sec. III-A).
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).  Work is ordered on
 *     that stream; a context is not thread-safe and calls on one context must not overlap.
 *   - Coordinates are 0-based.  Index weights use i + 1 (the paper counts from 1).
 *   - Every input is validated before any launch; errors are returned as status codes, never
 *     thrown or aborted across the ABI.  fpsketch_last_error() gives a detail string for the
 *     calling thread.
 */
#ifndef FPSKETCH_H
#define FPSKETCH_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct fpsketch_ctx fpsketch_ctx;

typedef enum {
  FPSK_OK = 0,
  FPSK_EINVAL = 1,     /* null pointer or parameter out of range */
  FPSK_EDTYPE = 2,     /* C is not FP32 (a narrowed product is rejected, Sec. II-A, Alg. 2),
                          or A/B not FP16/BF16 */
  FPSK_ESHAPE = 3,     /* a dimension or bucket count outside what the kernels support */
  FPSK_ENOMEM = 4,     /* device allocation failed */
  FPSK_EHIP = 5,       /* HIP runtime error (detail in fpsketch_last_error) */
  FPSK_ECAPACITY = 6,  /* more fault records than the caller's capacity; the first `cap`
                          records were written */
  FPSK_ENODEV = 7      /* the current device is not a gfx950 GPU */
} fpsketch_status;

typedef enum { FPSK_F16 = 0, FPSK_BF16 = 1, FPSK_F32 = 2 } fpsketch_dtype;

/* The method's parameters (Sec. VI-A defaults; fpsketch_default_params fills them). */
typedef struct {
  int32_t m;          /* probe buckets per side; 0 = start from Eq. 5 */
  int32_t rounds;     /* k independent hash rounds of localization (3, Sec. III-H) */
  int32_t r_star;     /* target search radius r* (4, Sec. III-G) */
  int32_t r_max;      /* largest radius (16, Sec. III-G) */
  int32_t s_budget;   /* declared error budget s (16) */
  int32_t delta_rc;   /* errors per row or column Delta (8) */
  int32_t k_cap;      /* candidate cap K per round; 0 = max(64, 8 s) (Sec. III-E) */
  int32_t b_layout;   /* 0: B is n2 x n3 row-major (C = A B); 1: B is passed as W = B^T,
                         n3 x n2 row-major (a linear layer's weight, C = A W^T); every call
                         of the context then takes W where it takes B */
  double rho_min;     /* smallest fault magnitude to localize, x rms(C) (0.02, Sec. III-G) */
  double mu;          /* probe margin (4, Sec. III-E) */
  double c_valid;     /* validation constant c (100, Sec. III-D) */
  double b_star;      /* index-budget target B* (0.3, Sec. III-F) */
  double c_coll;      /* collision constant c of m_comb (2, Sec. III-F) */
  uint64_t seed;      /* context seed; the probe uses hash round 0 of it */
  /* Eq. 3's noise law c_f 2^-24 sqrt(n1 n3 n2) (n2/8192)^e rms(C) / m, which starts the bucket
   * count (Eq. 4-5) and stands in for an unusable noise measurement in the plan (Sec. III-G).
   * Defaults: the paper's envelope (c_f 0.19 BF16, 0.3344 FP16, e 0.07); the constants belong
   * to the BLAS that computes C and can be measured for it (c_f > 0, e finite). */
  double law_cf_bf16;
  double law_cf_fp16;
  double law_n2_exp;
} fpsketch_params;

/* One localized fault (Algorithm 2 "emit record").  When `absolute` is 0, C_ij + delta is the
 * repaired value; when 1 (non-finite or out-of-range entry, Sec. III-I), delta IS the
 * recomputed value.  `round` is 0 for the exact scan, t for hash round t. */
typedef struct {
  int64_t i;
  int64_t j;
  double delta;
  int32_t absolute;
  int32_t round;
} fpsketch_fault;

/* Plan and noise figures of the last localize call (Sec. III-G). */
typedef struct {
  int32_t m;          /* probe bucket count */
  int32_t m_loc;      /* localization bucket count */
  int32_t r;          /* search radius */
  int32_t fallback;   /* 1 if the plan fell back to Eq. 3 */
  int32_t n_abs;      /* entries found by the exact scan */
  int32_t n_rechecked;/* coordinates recomputed in all rounds */
  double sigma_hat;   /* noise estimate the plan used */
  double rms_hat;     /* rms-hat(C) */
  double B;           /* index budget */
  double tau;         /* analytic threshold c n2 eps max|A| max|B| */
} fpsketch_plan_info;

/* ----------------------------------------------------------------------------------------- */
/* Library and context.                                                                      */

/* Fills the defaults of Sec. VI-A (k = 3, rho_min = 0.02, r* = 4, r_max = 16, mu = 4, c = 100,
 * B* = 0.3, collision c = 2, s = 16, Delta = 8, K = max(64, 8 s)). */
void fpsketch_default_params(fpsketch_params* p);

/* Static description of a status code. */
const char* fpsketch_status_str(fpsketch_status s);

/* Detail of the last error raised on the calling thread ("" if none). */
const char* fpsketch_last_error(void);

/* Creates a context for products A (n1 x n2) x B (n2 x n3) with operands in `ab_dtype`
 * (FPSK_F16 or FPSK_BF16) on the CURRENT HIP device, which must be gfx950.  The probe's
 * bucket count is params->m, or the Eq. 5 start when it is 0.  The context owns every table
 * and workspace (device memory) and the recalibration state.  `params` may be NULL (defaults).
 * Errors: FPSK_EINVAL (null out, bad params), FPSK_EDTYPE, FPSK_ESHAPE (n < 1, n >= 2^31,
 * m > 4096), FPSK_ENODEV, FPSK_ENOMEM, FPSK_EHIP. */
fpsketch_status fpsketch_create(int64_t n1, int64_t n2, int64_t n3, fpsketch_dtype ab_dtype,
                                const fpsketch_params* params, fpsketch_ctx** out);

/* Releases the context and its device memory.  NULL is ignored. */
void fpsketch_destroy(fpsketch_ctx* ctx);

/* ----------------------------------------------------------------------------------------- */
/* Hot path.                                                                                 */

/* The S-only probe (Sec. III-C; Algorithm 2, probe part).  Enqueues on `stream` and returns
 * without a host synchronization.  Reads A, B and C once; forms S at the context's m;
 * sigma_hat = 1.2533 mean(min(|S|, 5 mean|S|)), thr = min(tau, mu sqrt(2 ln m^2) sigma_hat)
 * with tau = c n2 2^-23 max|A| max|B| (Sec. III-E); the product is dirty unless every bucket
 * of S is finite and max|S| <= thr (Sec. III-I).  On a dirty product the device int32 at
 * `d_dirty` is set to 1 (it is never cleared: the caller zeroes it, then may OR many probes
 * into it and read it once per step); on a clean product sigma_hat is added to the context's
 * recalibration sum.  `c_dtype` must be FPSK_F32, otherwise FPSK_EDTYPE and nothing runs.
 * `d_dirty` may be NULL (the verdict is then only kept in the context's statistics). */
fpsketch_status fpsketch_probe(fpsketch_ctx* ctx, const void* A, const void* B, const void* C,
                               fpsketch_dtype c_dtype, int32_t* d_dirty, void* stream);

/* Localization (Algorithm 2, localize part, with Algorithm 1 per round).  Synchronous: returns
 * when the records are on the host.  Steps: exact scan of C for non-finite entries and entries
 * above fp32max/16 in magnitude, at most K in row-major order, each recomputed as an absolute
 * value (Sec. III-I); the plan (m_loc, r) from the noise estimate and rms-hat(C) (Sec. III-G);
 * then hash rounds t = 1..k of `seed` at m_loc, each forming S with C holding the recomputed
 * values at the absolute entries, peeling the finite faults found so far, selecting up to K
 * buckets above max(tau_c, tau_d), forming R and T at those buckets only (with the same peel),
 * decoding Eq. 2 and searching a (2r+1)^2 window in
 * Chebyshev-then-Manhattan order; a candidate (i, j) is accepted iff
 * |gamma - C_ij| > c 2^-23 sum_k |A_ik||B_kj| (Sec. III-D), with delta = gamma - C_ij.
 * `sigma_from_probe` = 1 uses the sigma_hat of this context's last probe (valid only if that
 * probe ran on this same C); 0 measures the MAD noise of a fresh S at the probe's m built with
 * hash round 0 of `seed`.  Writes at most `cap` records to the HOST array `out` and the number
 * found to *n_out (records beyond cap: FPSK_ECAPACITY).  C is not modified. */
fpsketch_status fpsketch_localize(fpsketch_ctx* ctx, const void* A, const void* B, const void* C,
                                  fpsketch_dtype c_dtype, uint64_t seed, int32_t sigma_from_probe,
                                  fpsketch_fault* out, int32_t cap, int32_t* n_out, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): fpsketch_probe with the same kernels, the same
 * statistics bit for bit and the same effect on d_dirty and on the context's noise average, but
 * the stream pass's factors and partials live in a scratch array of 16 MiB that the library
 * holds on each GPU it runs on until the process ends, instead of the context's workspace.  The
 * call allocates nothing (no hipMalloc, hipFree or allocating library routine; it never creates
 * timing events, so fpsketch_timing does not cover it) and enqueues only kernels on `stream`.
 * Takes the probe's block path only (m <= 64, n2 <= 16384; every such shape fits the array):
 * FPSK_ESHAPE otherwise.  Every call on one GPU shares its array, which keeps the last call's
 * contents: calls that overlap in time on one GPU (other streams, contexts or host threads)
 * race and must not be issued; calls ordered on one stream are safe.  Errors as fpsketch_probe. */
fpsketch_status fpsketch_probe_noalloc(fpsketch_ctx* ctx, const void* A, const void* B,
                                       const void* C, fpsketch_dtype c_dtype, int32_t* d_dirty,
                                       void* stream);

/* The B-side cache of the probe (Sec. III-C; Algorithm 2's probe keeps BH2^T of a weight):
 * forms Q = B H2^T for the probe's current hash round and m, and max |B|, from the device weight
 * B (n2 x n3, the context's half format, row-major) and keeps them in the context.  Enqueue only
 * on `stream`; B is not referenced afterwards.  A rebuild at a new m (fpsketch_calibrate_noise)
 * drops the cache.  FPSK_EINVAL for null arguments. */
fpsketch_status fpsketch_cache_b(fpsketch_ctx* ctx, const void* B, void* stream);

/* fpsketch_probe with the cached B side: streams A and C only and decides exactly as
 * fpsketch_probe does on the B the cache was formed from (same statistics, bit for bit).
 * Enqueue only.  FPSK_EINVAL when nothing is cached for the probe's current m; FPSK_EDTYPE
 * unless c_dtype is FPSK_F32. */
fpsketch_status fpsketch_probe_cached(fpsketch_ctx* ctx, const void* A, const void* C,
                                      fpsketch_dtype c_dtype, int32_t* d_dirty, void* stream);

/* fpsketch_probe without waiting for its own product and decision (Sec. III-C: the verdict is a
 * device flag the caller reads later).  For the probe's block path (m <= 64, n2 <= 16384) each
 * call enqueues ONE launch holding the decision of the call before the previous one, the
 * block products of the previous call and this call's pass over A, B and C; these run side by side
 * on three workspace sets in rotation, with the same arithmetic, hence the same bits, as
 * fpsketch_probe.  A call's verdict (ORed into its d_dirty), its statistics and its share of the
 * running noise sum are therefore final only after two more deferred calls or
 * fpsketch_probe_flush.  Every other call on the context flushes first (and waits for the
 * pending work when it runs on another stream).  A, B and C are read by this call's launch only:
 * the caller may reuse them as for fpsketch_probe; d_dirty must stay valid until the flush.
 * Deferred calls and the flush go to one stream (FPSK_EINVAL for another while calls are
 * pending).  Other shapes run an ordinary probe.  Errors as fpsketch_probe. */
fpsketch_status fpsketch_probe_deferred(fpsketch_ctx* ctx, const void* A, const void* B,
                                        const void* C, fpsketch_dtype c_dtype, int32_t* d_dirty,
                                        void* stream);

/* fpsketch_probe_cached, deferred as fpsketch_probe_deferred (the two may be mixed in one
 * sequence).  Errors as fpsketch_probe_cached. */
fpsketch_status fpsketch_probe_cached_deferred(fpsketch_ctx* ctx, const void* A, const void* C,
                                               fpsketch_dtype c_dtype, int32_t* d_dirty,
                                               void* stream);

/* Enqueues what deferred probes still owe (at most two launches); nothing pending: no-op. */
fpsketch_status fpsketch_probe_flush(fpsketch_ctx* ctx, void* stream);

/* Algorithm 2, apply step: writes the n records `recs` (a HOST array, as fpsketch_localize
 * returns them) into the device product C (n1 x n3 FP32, row-major), then probes the repaired
 * C once more with a fresh hash round.  Record (i, j, delta, absolute): C_ij <- delta when
 * absolute is 1 (the recomputed value of a non-finite or out-of-range entry), else
 * C_ij <- C_ij + delta, the sum formed in FP64 and rounded once to FP32.  The re-probe uses hash
 * round 0 of `seed` at the probe's m (pass a seed not used for this C before); it leaves the
 * context's probe statistics and noise average untouched.  *still_dirty = 1 when the re-probe
 * fires: the paper then recomputes C = AB at FP32, which is the caller's GEMM.  Synchronous on
 * `stream`.  C is modified.  FPSK_EINVAL for null pointers, n < 0, a coordinate outside C or a
 * coordinate listed twice; FPSK_EDTYPE unless c_dtype is FPSK_F32. */
fpsketch_status fpsketch_apply(fpsketch_ctx* ctx, const void* A, const void* B, void* C,
                               fpsketch_dtype c_dtype, const fpsketch_fault* recs, int32_t n,
                               uint64_t seed, int32_t* still_dirty, void* stream);

/* Probe recalibration (Sec. III-G).  Synchronous.  sigma_bar = mean sigma_hat over the clean
 * probes since the last rebuild; B1 = max(n1, n3) sigma_bar / rms-hat(C);
 * m' = max(m_comb, 16, min(ceil(m B1 / B*), m_max)).  If m' lies outside [m/1.25, 1.25 m] the
 * context rebuilds its probe hash, tables and workspace at m' and restarts the average.
 * Outputs (each may be NULL): the probe's m after the call, sigma_bar, and 1 if rebuilt.
 * With no clean probe recorded nothing changes.  When the rule asks for a rebuild at an m'
 * above 4096 (the kernels' largest bucket count; Eq. 5 reaches it only beyond about
 * 16384 x 16384 outputs) the context is left as it was, the outputs report the unchanged m, and
 * the call returns FPSK_ESHAPE. */
fpsketch_status fpsketch_calibrate_noise(fpsketch_ctx* ctx, const void* C, fpsketch_dtype c_dtype,
                                         void* stream, int32_t* m_out, double* sigma_bar_out,
                                         int32_t* rebuilt_out);

/* ----------------------------------------------------------------------------------------- */
/* Diagnostics used by the parity tests.                                                     */

/* Plan of the last localize call. */
fpsketch_status fpsketch_get_plan(fpsketch_ctx* ctx, fpsketch_plan_info* out);

/* The probe's current bucket count. */
fpsketch_status fpsketch_get_m(fpsketch_ctx* ctx, int32_t* m_out);

/* Statistics of the last probe, synchronously copied to the host array out[8]:
 * sigma_hat, thr, tau, max|S|, finite (1/0), dirty (1/0), max|A|, max|B|. */
fpsketch_status fpsketch_probe_stats(fpsketch_ctx* ctx, double* out, void* stream);

/* Sketches of E = AB - C at bucket count m with hash round `round` of `seed`, through the same
 * kernels as the probe and localize (Eq. 1 and the first-moment sketches; with `moments`, R and
 * T over the whole grid, which localize forms only at its selected buckets).  Synchronous.
 * Writes m*m doubles (row-major, bucket (a, b) at a*m + b) to the HOST arrays S and, when
 * `moments` is 1, R and T; maxab[0..1] receive max|A|, max|B| (maxab may be NULL). */
fpsketch_status fpsketch_sketch(fpsketch_ctx* ctx, const void* A, const void* B, const void* C,
                                fpsketch_dtype c_dtype, uint64_t seed, int32_t round, int32_t m,
                                int32_t moments, double* S, double* R, double* T, double* maxab,
                                void* stream);

/* Validation recomputation (Sec. III-D) at n coordinates given in the HOST array
 * coords[2n] = (i0, j0, i1, j1, ...): gamma = sum_k A_ik B_kj and sum_k |A_ik||B_kj|, with
 * exact half x half products accumulated in FP64.  Synchronous; writes n doubles to each HOST
 * array.  Coordinates outside C: FPSK_EINVAL. */
fpsketch_status fpsketch_recheck(fpsketch_ctx* ctx, const void* A, const void* B,
                                 const int64_t* coords, int32_t n, double* gamma, double* abssum,
                                 void* stream);

/* Probe timing.  With timing enabled, every fpsketch_probe launches its kernels with four
 * hipEvents that the dispatches time-stamp themselves (no extra queue packets): start and end
 * of the streaming kernel (A, B, C pass), and start of the first product dispatch and end of
 * the last (product and decision).  No work is skipped or reordered.  Enabling resets the
 * record.  Events are created on demand (so this mode allocates; leave it off in capture or
 * serving). */
fpsketch_status fpsketch_timing(fpsketch_ctx* ctx, int32_t enable);

/* Waits for the last recorded probe and returns the summed durations (ms) of the streaming
 * kernel and of the product/decision dispatches over the probes recorded since timing was
 * enabled or last read, and their number; then clears the record. */
fpsketch_status fpsketch_timing_read(fpsketch_ctx* ctx, double* stream_ms, double* product_ms,
                                     int64_t* calls);

/* Reference streams of known size, for the achievable-bandwidth line and for scaling HBM
 * traffic counters: a plain read of `bytes` from device memory `src` (16-byte aligned, bytes a
 * multiple of 16), folded into one word that is written to the device word `d_out` only in a
 * practically unreachable case, and a plain copy of `bytes` from `src` to `dst`.  `grid`
 * work-groups of 256 threads stride over the buffer.  Enqueue only. */
fpsketch_status fpsketch_stream_read(const void* src, int64_t bytes, uint32_t* d_out,
                                     int32_t grid, void* stream);
fpsketch_status fpsketch_stream_copy(const void* src, void* dst, int64_t bytes, int32_t grid,
                                     void* stream);

/* ----------------------------------------------------------------------------------------- */
/* Host-only helpers (no device work; usable without a GPU).                                  */

/* Hash of one side of one round (Sec. III-B; family: splitmix64 stream keyed per
 * (seed, round, side), bucket by multiply-shift of the high 32 bits, sign by bit 0):
 * bucket[idx] in [0, m), sign[idx] in {+1, -1} for idx < n.  Host arrays. */
fpsketch_status fpsketch_hash_table(uint64_t seed, int32_t round, int32_t side, int64_t n,
                                    int32_t m, int32_t* bucket, int8_t* sign);

/* Eq. 5 starting bucket count for a shape and operand format (Sec. III-F). */
fpsketch_status fpsketch_m_start(int64_t n1, int64_t n2, int64_t n3, fpsketch_dtype ab_dtype,
                                 const fpsketch_params* params, int32_t* m_out);

/* Localization plan (Sec. III-G): (m_loc, r, B, fallback) from the probe's m, a noise estimate
 * and rms-hat(C); falls back to Eq. 3 when either is not a positive finite number. */
fpsketch_status fpsketch_plan_host(int64_t n1, int64_t n2, int64_t n3, fpsketch_dtype ab_dtype,
                                   int32_t m, double sigma_hat, double rms,
                                   const fpsketch_params* params, int32_t* m_loc, int32_t* r,
                                   double* B, int32_t* fallback);

/* Probe recalibration rule (Sec. III-G): the new m and whether it triggers a rebuild. */
fpsketch_status fpsketch_recalibrate_host(int64_t n1, int64_t n3, int32_t m, double sigma_bar,
                                          double rms, const fpsketch_params* params,
                                          int32_t* m_new, int32_t* rebuild);

/* rms-hat(C) from samples already taken at the stride max(1, floor(n1 n3 / 65536)) (Sec.
 * III-G): finite samples only, magnitudes clipped at 64 x their median.  NaN if none. */
double fpsketch_rms_hat_samples(const float* samples, int64_t count);

#ifdef __cplusplus
}
#endif

#endif /* FPSKETCH_H */
