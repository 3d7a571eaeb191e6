/*
 * thin -- thinned attention on AMD Instinct MI355X (gfx950).
 *
 * C ABI of the non-causal thinning path of "Express Language Modeling":
 * for every (batch, head) slice, kernel halving (KH) under the attention
 * kernel kappa_att thins the n key/value rows to n_out coreset rows
 * (thin_compress), then every query attends over the coreset only
 * (thin_attention).
 *
 * Conventions shared by every entry point
 *   - Tensors are contiguous row-major [B, H, rows, d] (d fastest); the slice
 *     s = b*H + h owns rows [s*rows, (s+1)*rows).  K and V have n rows, Q and
 *     O have n_q rows.
 *   - Pointers marked (device) are HIP device pointers; (host) are host
 *     pointers.  The caller owns every buffer; the library allocates nothing
 *     and keeps no state between calls.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Work is enqueued
 *     asynchronously; nothing synchronises.  Calls on one stream are ordered.
 *   - Arguments are validated on the host before anything is enqueued.  On any
 *     error nothing is launched and no output is written.  THIN_EHIP reports a
 *     launch error; faults inside a kernel surface at the caller's next
 *     synchronisation.
 *   - Supported: dtype THIN_FP32 or THIN_BF16 (Q, K, V share it), d in
 *     {32, 64, 128}, B*H <= 65535 slices (THIN_EINVAL beyond).
 *   - Device status word: the first 4 bytes (int32) of every workspace
 *     (thin_compress*, the Express object's, thin_express_prefill's).  A call
 *     that runs kernel-halving decisions clears it first (an Express object:
 *     at its first step); a decision pass whose bounded wait for another
 *     wavefront's progress runs out sets it to THIN_STATUS_WAIT_EXHAUSTED
 *     and still ends normally.  Nonzero means that call's (that object's)
 *     coreset is not the one Algorithm A.1 defines; read it with
 *     thin_workspace_status after the call.
 */
#ifndef THIN_H
#define THIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  THIN_OK = 0,
  THIN_EINVAL = 1,     /* bad size, pointer, or no valid level structure   */
  THIN_EDTYPE = 2,     /* unsupported dtype / output dtype                  */
  THIN_EUNIFORMS = 3,  /* uniforms buffer shorter than the plan requires    */
  THIN_EWORKSPACE = 4, /* workspace missing or smaller than the plan's size */
  THIN_EHIP = 5        /* the HIP runtime reported an error                 */
} thin_status_t;

typedef enum { THIN_FP32 = 0, THIN_BF16 = 1 } thin_dtype_t;

/* Bits of the device status word. */
#define THIN_STATUS_WAIT_EXHAUSTED 1

/*
 * Level structure of one compress call (identical for every slice).
 *
 * Reading of the output size n_out and the oversampling parameter g
 * (Sec. 3.1; App. H, Algorithm H.2 Offline-Compress2; Alg. 1's final
 * Halve(Halve(.))): L = floor(log2(n / n_out)) halving rounds take
 * n_kept = n_out * 2^L rows to n_out.  If n_kept < n a stratified subsample
 * (one uniform draw per contiguous stratum; Alg. 3 / Algorithm H.1) keeps
 * n_kept rows first.  Round r = 0..L-1 splits the current n_kept / 2^r rows
 * of a slice into G_r = 4^max(L-g-1-r, 0) contiguous equal buckets and runs
 * KH(1/2) (App. A, Algorithm A.1) on each: the first L - min(g, L) rounds are
 * Offline-Compress2 with output size 2^g n_out, the rest halve the whole set.
 * Every bucket must hold an even number >= 2 of rows.
 */
typedef struct {
  int64_t n_kept;             /* rows entering round 0                        */
  int32_t rounds;             /* L                                            */
  int32_t compress_levels;    /* rounds with more than one bucket possible    */
  int64_t uniforms_per_slice; /* U: uniforms one slice consumes               */
  int64_t uniforms_total;     /* B * H * U                                    */
  int64_t max_bucket;         /* largest bucket (rows) of any round           */
  size_t workspace_bytes;     /* device workspace thin_compress needs         */
} thin_plan_t;

/*
 * Plan a compress call.  Host-only; touches no device.
 * Returns THIN_OK and fills *plan (host), or THIN_EINVAL when B, H, n, d,
 * n_out, g are out of range (n_out < 1, n_out > n, g < 0, d unsupported) or
 * when some bucket would hold fewer than two rows or an odd number of rows.
 */
int thin_plan(int64_t B, int64_t H, int64_t n, int64_t d, int64_t n_out, int32_t g,
              thin_plan_t* plan);

/*
 * Compress every slice's key/value rows to n_out coreset rows.
 *
 *   K, V        (device) [B,H,n,d] of `dtype`.
 *   uniforms    (device) float32 in [0,1), at least B*H*U of them, slice-major:
 *               slice s reads [s*U, (s+1)*U).  Within a slice: first the
 *               n_kept subsample draws (only when n_kept < n), then for each
 *               round r the n_r/2 pair draws (n_r = n_kept / 2^r) in bucket
 *               order, pair order within a bucket.  Pair i of a bucket swaps
 *               iff u_i < min(1, (1 - alpha_i/a_i)_+ / 2) (App. A).
 *               Values k * 2^-24 make every derived quantity exact.
 *   idx_out     (device) int32 [B,H,n_out]: kept row indices in [0,n),
 *               strictly increasing within a slice.
 *   workspace   (device) at least plan.workspace_bytes bytes, 256-byte
 *               aligned; contents on entry are irrelevant.
 *
 * kappa_att((k,v),(k',v')) = exp(<k,k'>/sqrt(d)) (<v,v'> + v_max^2) with
 * v_max = max over all n rows of ||v||_inf (Sec. 2.1, eq. katt); delta = 1/2
 * (App. I).  With n_out == n the result is 0..n-1.  The kernel values are
 * evaluated in float32 under per-pair power-of-two scales chosen from the
 * keys' norms, so no exponent overflows whatever the keys; keys whose
 * ||k||^2/sqrt(d) exceeds about 1.1e7 (kappa_att itself far beyond float64)
 * are not supported.
 * Errors: THIN_EINVAL (sizes / null pointers / no level structure),
 * THIN_EDTYPE, THIN_EUNIFORMS (n_uniforms < plan.uniforms_total),
 * THIN_EWORKSPACE, THIN_EHIP.
 */
int thin_compress(const void* K, const void* V, int32_t dtype, int64_t B, int64_t H, int64_t n,
                  int64_t d, int64_t n_out, int32_t g, const float* uniforms,
                  int64_t n_uniforms, int32_t* idx_out, void* workspace,
                  size_t workspace_bytes, void* stream);

/*
 * thin_compress for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * no workspace argument; the workspace is a static device array of
 * THIN_STATIC_SCRATCH_BYTES that every GPU the library runs on holds from
 * the time the library's code is loaded on it until the process ends.  The
 * call allocates nothing (no hipMalloc / hipFree).
 *   Arguments, layouts and results as thin_compress (KH, delta = 1/2), on
 *   the calling thread's current device (the device of `stream`).
 *   status  (device, nullable) int32: receives the call's device status word
 *           (see the conventions above), ordered after its kernels.
 * The score region takes what the other regions leave, so rounds whose
 * buckets' scores do not all fit run in several launches (same result).
 * Calls on one GPU share the array, which keeps the last call's contents:
 * calls that overlap in time on one GPU (different streams or threads) race
 * and must not be made; calls ordered on one stream are fine.
 * Errors: those of thin_compress, and THIN_EWORKSPACE when the call needs
 * more than THIN_STATIC_SCRATCH_BYTES (index lists, pair terms and row
 * scales grow with B*H*n; the long workload B=4 H=16 n=16384 and the stress
 * workload B=1 H=32 n=65536 fit).
 */
#define THIN_STATIC_SCRATCH_BYTES ((size_t)128 << 20)
int thin_compress_static(const void* K, const void* V, int32_t dtype, int64_t B, int64_t H,
                         int64_t n, int64_t d, int64_t n_out, int32_t g, const float* uniforms,
                         int64_t n_uniforms, int32_t* idx_out, int32_t* status, void* stream);

/*
 * thin_compress plus a record of every swap decision, for checking a run
 * against a reference implementation.
 *   swap_trace  (device) uint8 [B*H*U], indexed exactly like `uniforms`:
 *               1 if that pair swapped, 0 otherwise; the subsample entries
 *               are written as 0.  trace_len must be >= B*H*U (THIN_EINVAL).
 */
int thin_compress_traced(const void* K, const void* V, int32_t dtype, int64_t B, int64_t H,
                         int64_t n, int64_t d, int64_t n_out, int32_t g,
                         const float* uniforms, int64_t n_uniforms, int32_t* idx_out,
                         void* workspace, size_t workspace_bytes, uint8_t* swap_trace,
                         int64_t trace_len, void* stream);

/*
 * Halving algorithm of thin_compress_ex.
 *   THIN_HALVE_KH       kernel halving KH(delta) under kappa_att (App. A,
 *                       Algorithm A.1), as in thin_compress.
 *   THIN_HALVE_UNIFORM  every pair keeps one of its two rows with
 *                       probability 1/2: the second iff u_i < 1/2.  No kernel
 *                       is evaluated; this is the rule KH applies to a pair
 *                       whose threshold a_i is 0, and the simplest base
 *                       halving the construction accepts (Sec. 5: any halving
 *                       algorithm can be used).
 */
typedef enum { THIN_HALVE_KH = 0, THIN_HALVE_UNIFORM = 1 } thin_halve_t;

/*
 * Options of thin_compress_ex; {THIN_HALVE_KH, NULL, 0, 0, NULL} gives
 * thin_compress.
 *   halve     a thin_halve_t.
 *   delta     (host, nullable) float64 [plan.rounds]: the failure probability
 *             of every KH call of round r (its threshold carries the factor
 *             1/2 + log(2 N_r / delta[r]), App. A), each in (0, 1]; read
 *             during the call only.  NULL = 1/2 for every round (App. I).
 *             Ignored by THIN_HALVE_UNIFORM.
 *   n_sinks   rows 0..n_sinks-1 of every slice are kept exactly (attention
 *             sinks, the n_sinks setting of the experiments of App. I).
 *   n_window  rows n-n_window..n-1 of every slice are kept exactly (the
 *             recent window, n_window in App. I).
 *             The n_mid = n - n_sinks - n_window rows between them are
 *             thinned to n_out as a dataset of their own: v_max of eq. katt
 *             is taken over them, and the plan (uniforms, workspace) is
 *             thin_plan's for n_mid rows.  idx_out is then int32
 *             [B,H,n_sinks+n_out+n_window]: the sinks, the coreset (rows of
 *             the whole slice) and the window, in that order.
 *   logw_out  (device, nullable) float32 [B,H,n_sinks+n_out+n_window]: the
 *             log-weight of every output row for eq. def:att_approx, 0 for
 *             an exact row and log(n_mid/n_out) for a coreset row (which
 *             stands for n_mid/n_out rows); the weights of a slice sum to n.
 */
typedef struct {
  int32_t halve;
  const double* delta;
  int64_t n_sinks;
  int64_t n_window;
  float* logw_out;
} thin_compress_opts_t;

/*
 * thin_compress with a choice of halving algorithm, of KH's delta per round
 * and of exact sink/window rows.  Same arguments, uniforms layout (the pair
 * draws of a round are consumed the same way by either algorithm), workspace
 * and level structure as thin_compress of the thinned rows; opts (host) must
 * not be NULL.  swap_trace (device, nullable): as in thin_compress_traced,
 * with trace_len >= B*H*U when given.
 * Errors: those of thin_compress, and THIN_EINVAL for an unknown halve, a
 * delta[r] outside (0, 1], a negative n_sinks or n_window, or
 * n - n_sinks - n_window < n_out.
 */
int thin_compress_ex(const void* K, const void* V, int32_t dtype, int64_t B, int64_t H,
                     int64_t n, int64_t d, int64_t n_out, int32_t g, const float* uniforms,
                     int64_t n_uniforms, int32_t* idx_out, void* workspace,
                     size_t workspace_bytes, const thin_compress_opts_t* opts,
                     uint8_t* swap_trace, int64_t trace_len, void* stream);

/*
 * Attention of every query over its slice's coreset (Sec. 2.1 eq.
 * unmaskedatt restricted to the coreset; eq. def:att_approx with equal
 * weights, which cancel):
 *   O[s,q,:] = sum_j exp(<Q[s,q],K[s,I_j]>/sqrt d) V[s,I_j] / sum_j exp(...)
 * with I = idx[s, 0..n_out).
 *   Q           (device) [B,H,n_q,d] of `dtype`;  K, V (device) [B,H,n,d].
 *   idx         (device) int32 [B,H,n_out], every entry in [0,n) (entries
 *               outside are clamped to the nearest row; duplicates allowed).
 *   O           (device) [B,H,n_q,d] of `out_dtype` (THIN_FP32 or THIN_BF16).
 * Scores and the softmax are accumulated in float32.
 * Errors: THIN_EINVAL, THIN_EDTYPE, THIN_EHIP.
 */
int thin_attention(const void* Q, const void* K, const void* V, int32_t dtype, int64_t B,
                   int64_t H, int64_t n_q, int64_t n, int64_t d, const int32_t* idx,
                   int64_t n_out, void* O, int32_t out_dtype, void* stream);

/*
 * Weighted attention over a weighted coreset (eq. def:att_approx): key j of
 * slice s carries the weight w_j = exp(logw[s, j]),
 *   O[s,q,:] = sum_j w_j exp(<Q[s,q],K[s,I_j]>/sqrt d) V[s,I_j] / sum_j w_j exp(...).
 *   logw  (device, nullable) float32 [B,H,n_out]; -inf drops a key, NULL
 *         gives thin_attention.  Every query needs at least one key of
 *         finite log-weight (else its row of O is undefined).
 * Other arguments, layouts and errors as thin_attention; logw_out of
 * thin_compress_ex is this call's logw for its idx_out.
 */
int thin_attention_ex(const void* Q, const void* K, const void* V, int32_t dtype, int64_t B,
                      int64_t H, int64_t n_q, int64_t n, int64_t d, const int32_t* idx,
                      const float* logw, int64_t n_out, void* O, int32_t out_dtype,
                      void* stream);

/*
 * Thinformer decoding over an Express cache (Sec. 3-4: Alg. 1 Express with
 * Compress2 of Alg. 2 in its thin phase, Alg. 4 Thinformer, Alg. 5
 * WtdAttention), for all B*H slices in lockstep.  Point t (t = 0, 1, ...) of
 * every slice first attends over the weighted cache of points 0..t-1 plus
 * itself, then enters the cache.  The cache holds, per slice, the Express
 * coreset E (weight 1) and the Compress2 coresets C_0..C_mp (weight
 * 2^(i-mp)); its Halve calls are KH(delta_{m,i}) and, in the Halve phase,
 * KH(delta_m / 2) with Cor. 2's schedule for the given delta, under
 * kappa_att with v_max over the rows of each call (or uniform halving).
 * Every Halve call of N points consumes the next N/2 uniforms of each slice.
 * Above mbar, Subsample (Alg. 3) keeps the point at offset floor(u R) of each
 * stratum of R = 2^(m - mbar) points, u the stratum's draw; the draws are
 * host memory, one per stratum in order, shared by all slices (the slices
 * run in lockstep, so they keep the same positions).
 * Supported: every Compress2 group size 4 n_out / 2^mp (1 <= mp <= mbar, as
 * reached by n_max points) an even integer >= 2; 4 n_out <= 8192.
 */
typedef struct thin_express thin_express_t;

typedef struct {
  int64_t uniforms_per_slice; /* uniforms the Halve calls of n_max points consume
                                 at most (every Halve call as early as the
                                 draws allow)                                    */
  int64_t max_keys;           /* largest key list of one attention call           */
  size_t workspace_bytes;     /* device workspace of thin_express_create          */
  int64_t subsample_draws;    /* Subsample draws n_max points need                */
} thin_express_plan_t;

/* Host-only.  THIN_EINVAL for unsupported sizes (see above). */
int thin_express_plan(int64_t B, int64_t H, int64_t d, int64_t n_out, int32_t mbar,
                      int64_t n_max, thin_express_plan_t* plan);

/*
 * Create the cache state (host memory, freed by thin_express_destroy) over
 * the caller's device workspace (>= plan.workspace_bytes, 256-byte aligned),
 * which the object uses until destroyed.  halve: a thin_halve_t.  delta in
 * (0, 1) (1/2 in the paper's guarantee).  Launches nothing.
 */
int thin_express_create(int32_t dtype, int64_t B, int64_t H, int64_t d, int64_t n_out,
                        int32_t mbar, double delta, int32_t halve, int64_t n_max,
                        void* workspace, size_t workspace_bytes, thin_express_t** out);

/*
 * One decoding step for point t = the number of points seen so far:
 *   Q         (device) [B,H,d]: the point's query.
 *   K, V      (device) [B,H,n_max,d]: the key/value rows of points 0..t
 *             (row t written before the call).
 *   uniforms  (device) float32 [B*H, plan.uniforms_per_slice], n_uniforms
 *             its size (nullable when the plan needs none).
 *   draws     (host) float32 [n_draws] Subsample draws, read only at the
 *             first point of a stratum (nullable when the plan needs none).
 *   O         (device) [B,H,d] of out_dtype: the point's output.
 *   swap_trace (device, nullable) uint8 indexed like uniforms.
 * Enqueued on `stream`; calls on one object must be stream-ordered.
 * Errors: THIN_EINVAL (null arguments, t = n_max, a missing draw, or a
 * point beyond the supported levels), THIN_EDTYPE, THIN_EUNIFORMS,
 * THIN_EHIP; nothing is enqueued or changed on an error found before launch.
 */
int thin_express_step(thin_express_t* x, const void* Q, const void* K, const void* V,
                      const float* uniforms, int64_t n_uniforms, const float* draws,
                      int64_t n_draws, void* O, int32_t out_dtype, uint8_t* swap_trace,
                      void* stream);

/*
 * The current weighted cache: idx (device) int32 and logw (device) float32,
 * each [B,H,plan.max_keys], receive in their first *len entries per slice
 * the cache in the order C_0, C_1, .., C_mp, E with log-weights
 * (i - mp) log 2 and 0; *len (host) its size, *m (host, nullable) the
 * thinning factor m.  Enqueued on `stream`.
 */
int thin_express_cache(const thin_express_t* x, int32_t* idx, float* logw, int64_t* len,
                       int32_t* m, void* stream);

/* Host-only: *keys = the size of the key list the next step attends over
 * (the cache plus the point itself), *t = the next point's position. */
int thin_express_next(const thin_express_t* x, int64_t* keys, int64_t* t);

/* Free the host state (the workspace stays the caller's). */
int thin_express_destroy(thin_express_t* x);

/*
 * Masked prefill: the outputs of Thinformer decoding (thin_express_step) for
 * every point of a whole sequence at once (Alg. 4; the offline form of the
 * Express recursion, App. H, Algorithm H.3).  Point p attends over the cache
 * of points 0..p-1 plus itself, exactly as a decoding step would, with the
 * same uniforms layout (every Halve call's N/2 draws at the offset it has in
 * decoding) and the same Subsample draws (host, one per stratum).
 * The Compress2 calls of a level run batched by depth (their outputs kept),
 * the Halve phases level by level, then one attention launch.  The call plans
 * on the host (tables of Halve calls, query tiles and cache pieces), writes
 * the tables into the caller's host staging buffer and enqueues one copy of
 * it into the workspace; nothing synchronises.
 *   Q, K, V (device) [B,H,n,d] of `dtype`;  O (device) [B,H,n,d] of out_dtype.
 *   uniforms (device) [B*H, plan.uniforms_per_slice];  draws (host).
 *   host_staging (host) at least plan.host_staging_bytes: its contents must
 *               stay unchanged until the stream has executed this call (for
 *               instance until an event recorded after it has completed).
 *               Pinned memory (hipHostMalloc) keeps the copy asynchronous;
 *               with pageable memory the runtime may block the host during
 *               the copy.
 *   swap_trace (device, nullable) uint8 indexed like uniforms.
 * Sizes as for thin_express_plan with n_max = n, and n <= 2^30.
 * Errors: THIN_EINVAL, THIN_EDTYPE, THIN_EUNIFORMS, THIN_EWORKSPACE (also for
 * a missing or short host_staging), THIN_EHIP.
 */
typedef struct {
  int64_t uniforms_per_slice; /* as thin_express_plan for n points          */
  int64_t subsample_draws;    /* Subsample draws the n points need          */
  size_t workspace_bytes;     /* device workspace of thin_express_prefill   */
  int64_t attention_keys;     /* per slice: keys summed over the points
                                 (Subsample draws of 0)                     */
  int64_t staged_keys;        /* per slice: keys the attention launch
                                 gathers, summed over its 128-point tiles   */
  size_t host_staging_bytes;  /* host staging buffer of thin_express_prefill */
} thin_prefill_plan_t;

/* Host-only. */
int thin_express_prefill_plan(int64_t B, int64_t H, int64_t n, int64_t d, int64_t n_out,
                              int32_t mbar, thin_prefill_plan_t* plan);

int thin_express_prefill(int32_t dtype, int64_t B, int64_t H, int64_t n, int64_t d,
                         int64_t n_out, int32_t mbar, double delta, int32_t halve,
                         const void* Q, const void* K, const void* V, const float* uniforms,
                         int64_t n_uniforms, const float* draws, int64_t n_draws, void* O,
                         int32_t out_dtype, void* workspace, size_t workspace_bytes,
                         void* host_staging, size_t host_staging_bytes, uint8_t* swap_trace,
                         void* stream);

/*
 * Diagnostic: out[m*16 + n] = <rows[m], rows[16 + n]> for m, n < 16, computed
 * through the MFMA row-fragment path the pair-score kernel uses.
 *   rows (device) [32, d] of `dtype`;  out (device) float32 [16, 16].
 * Errors: THIN_EINVAL, THIN_EDTYPE, THIN_EHIP.
 */
int thin_selftest_gram16(int32_t dtype, int64_t d, const void* rows, float* out, void* stream);

/* Static, human-readable text for a status code. */
const char* thin_status_str(int status);

/*
 * Enqueue a copy of a workspace's device status word (see the conventions
 * above) into *status (host; pinned memory keeps the copy asynchronous) on
 * `stream`; read *status after synchronising the stream.
 * Errors: THIN_EINVAL (null pointer), THIN_EHIP.
 */
int thin_workspace_status(const void* workspace, int32_t* status, void* stream);

/*
 * Launch observer, a diagnostic for tracing and per-kernel timing (not part
 * of the compute contract; the library keeps no state between calls apart
 * from it).  While a hook is set,
 * every kernel launch made by thin_compress, thin_compress_traced,
 * thin_compress_ex, thin_attention, thin_attention_ex and thin_express_step
 * is bracketed by two calls on the
 * calling thread:
 * hook(ctx, kernel, round, 0, stream) right before the launch is enqueued and
 * hook(ctx, kernel, round, 1, stream) right after.  The hook may enqueue
 * stream-ordered work of its own (for instance record an event on `stream`),
 * so that consecutive records time one kernel.  `kernel` is a
 * thin_kernel_t, `round` the Halve round 0..L-1 of a THIN_KERNEL_SCORES,
 * THIN_KERNEL_DECIDE, THIN_KERNEL_LOCAL or per-round THIN_KERNEL_UNIFORM
 * launch and -1 otherwise (uniform halving runs every round in one launch
 * when a slice keeps at most 32768 rows, else one launch per round).  A round
 * runs either as SCORES + DECIDE launches or, when its buckets are small
 * enough for one workgroup to hold all their scores in LDS, as one LOCAL
 * launch.  The setting belongs to the calling thread (thread-local): only
 * launches made by that thread are observed, and calls on other threads are
 * unaffected.  hook = NULL turns it off (the default).  Returns THIN_OK.
 */
typedef enum {
  THIN_KERNEL_TRACE_CLEAR = 0, /* zeroing of the swap trace               */
  THIN_KERNEL_SUBSAMPLE = 1,   /* stratified subsample                    */
  THIN_KERNEL_FILL = 2,        /* index copy when no round runs           */
  THIN_KERNEL_VMAX = 3,        /* v_max scan (with its zeroing)           */
  THIN_KERNEL_SCORES = 4,      /* pair scores of one round                */
  THIN_KERNEL_DECIDE = 5,      /* decision pass of one round              */
  THIN_KERNEL_ATTENTION = 6,   /* coreset attention                       */
  THIN_KERNEL_LOCAL = 7,       /* scores and decisions of one round       */
  THIN_KERNEL_UNIFORM = 8,     /* uniform halving (all rounds, or one)    */
  THIN_KERNEL_ASSEMBLE = 9,    /* sinks + coreset + window, log-weights   */
  THIN_KERNEL_EXPRESS = 10,    /* Express cache moves, per-call v_max, keys */
  THIN_KERNEL_STATUS = 11      /* clearing of the device status word      */
} thin_kernel_t;
typedef void (*thin_launch_hook_t)(void* ctx, int32_t kernel, int32_t round, int32_t phase,
                                   void* stream);
int thin_set_launch_hook(thin_launch_hook_t hook, void* ctx);

#ifdef __cplusplus
}
#endif
#endif /* THIN_H */
