/*
 * CPU oracle for the thinning hot path -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, single-threaded, float64 implementation of what the path computes,
 * written from the paper ("Express Language Modeling"):
 *   - the attention kernel kappa_att                 (Sec. 2.1, eq. katt)
 *   - kernel halving KH(delta)                       (App. A, Algorithm A.1)
 *   - stratified subsampling                         (Alg. 3 / App. H, Algorithm H.1)
 *   - offline Compress2 and the oversampled Compress (App. H, Algorithm H.2)
 *   - softmax attention over a coreset               (Sec. 2.1 eq. unmaskedatt;
 *                                                     Sec. 2.2 eq. def:att_approx with equal weights)
 * Only tests, the smoke check and the benchmark's CPU-baseline leg may load it.
 * It shares no code, header, constant or helper with the HIP library.
 */
#ifndef THIN_ORACLE_H
#define THIN_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OR_KERNEL_KATT 0   /* kappa_att((k,v),(k',v')) = exp(<k,k'>/sqrt d) (<v,v'> + vmax^2) */
#define OR_KERNEL_LINEAR 1 /* <k,k'> + <v,v'>  (only used to pin the halving arithmetic) */

/* Level structure of one compress call (per slice). */
typedef struct {
  int64_t n_kept;         /* rows entering the first halving round */
  int32_t rounds;         /* number of halving rounds L */
  int32_t compress_levels;/* rounds that belong to Compress2 (the rest are single-bucket halvings) */
  int64_t uniforms;       /* uniforms consumed per slice */
  int32_t subsample;      /* 1 if a stratified subsample runs first */
} or_plan_t;

/* Counters filled by the halving routines (accumulated, caller zeroes). */
typedef struct {
  int64_t decisions;      /* swap decisions taken */
  int64_t swaps;          /* decisions that swapped */
  int64_t near_ties;      /* |rho| < tol: GPU bit adopted (follow mode) */
  int64_t hard_mismatch;  /* |rho| >= tol and the followed bit disagreed */
  int64_t zero_threshold; /* decisions with a == 0 (reading: swap iff u < 1/2) */
  double min_abs_rho;     /* smallest |rho| seen */
} or_stats_t;

/* Returns 0, or -1 if the arguments admit no valid level structure. */
int or_plan(int64_t n, int64_t n_out, int32_t g, or_plan_t* plan);

/* (max_{i,c} |V[i,c]|)^2 over all n rows. */
double or_vmax2(const double* V, int64_t n, int64_t d);

/* Stratified subsample of n rows down to n_kept, one draw per stratum. */
void or_subsample(int64_t n, int64_t n_kept, const float* u, int32_t* out);

/*
 * KH(delta) on one bucket: rows[0..N) index K/V (row-major, d columns).
 * u[i] drives pair i.  out[i] receives the row kept for pair i (coreset 1).
 * follow (nullable): bits of another implementation; adopted at near ties
 * (|rho| < tol) and, counted as hard mismatches, elsewhere.
 * bits/rho/alpha/thresh (nullable): per-decision trace.
 */
int or_kernel_halving(const double* K, const double* V, int64_t d, double vmax2,
                      int kernel, double delta, const int32_t* rows, int64_t N,
                      const float* u, int32_t* out, const uint8_t* follow, double tol,
                      uint8_t* bits, double* rho, double* alpha, double* thresh,
                      or_stats_t* st);

/*
 * One slice: [stratified subsample] -> Compress2 down to 2^g n_out -> g more
 * single-bucket halvings -> n_out indices (strictly increasing).
 * U holds this slice's uniforms (plan.uniforms of them).  follow/bits are
 * indexed like U (entries of the subsample part are unused).
 */
int or_compress(const double* K, const double* V, int64_t n, int64_t d,
                int64_t n_out, int32_t g, int kernel, const float* U,
                int32_t* idx_out, const uint8_t* follow, double tol,
                uint8_t* bits, double* rho, or_stats_t* st);

/* Halving algorithm of a compress call. */
#define OR_HALVE_KH 0      /* KH(delta), App. A Algorithm A.1 */
#define OR_HALVE_UNIFORM 1 /* one point of each pair, each with probability 1/2 */

/* Uniform halving of one bucket: out[i] = rows[2i + (u[i] < 1/2)]. */
int or_uniform_halving(const int32_t* rows, int64_t N, const float* u, int32_t* out,
                       uint8_t* bits, or_stats_t* st);

/*
 * or_compress with a choice of halving algorithm and, for KH, the failure
 * probability delta[r] of every call of round r (delta NULL = 1/2).  Round r
 * counts the halving rounds from 0 as in or_plan.
 */
int or_compress_ex(const double* K, const double* V, int64_t n, int64_t d,
                   int64_t n_out, int32_t g, int kernel, int halve, const double* delta,
                   const float* U, int32_t* idx_out, const uint8_t* follow, double tol,
                   uint8_t* bits, double* rho, or_stats_t* st);

/* O[q] = sum_j exp(<Q_q,K_rows[j]>/sqrt d) V_rows[j] / sum_j exp(...), j < m. */
void or_attention(const double* Q, const double* K, const double* V, int64_t n_q,
                  int64_t d, const int32_t* rows, int64_t m, double* O);

/*
 * Thinformer decoding (Alg. 4): for p = 0..n-1, O[p] = WtdAttention (Alg. 5)
 * of Q[p] over the Express cache (Alg. 1, Compress2 of Alg. 2 in its thin
 * phase) after p updates plus point p itself, then the cache is updated with
 * point p.  Halve_{m,i} = KH(delta_{m,i}) and Halve_{m,m} = KH(delta_m / 2)
 * (Cor. 2) under kappa_att with v_max over the rows of each call (halve =
 * OR_HALVE_UNIFORM: uniform halving instead).  Every Halve call of N points
 * consumes the next N/2 uniforms of U (follow/bits indexed alike).  Above
 * mbar, Subsample (Alg. 3) keeps the point at offset floor(u R) of every
 * stratum of R = 2^(m - mbar) points, u = sub_u[k] for the k-th stratum
 * (sub_u NULL: u = 0).  Returns -1 if a Compress2 group size 4 n_out / 2^mp
 * is not an even integer >= 2.  O (nullable) [n, d]; the final cache
 * (C_0..C_mp with log-weights (i - mp) log 2, then E with 0) goes to
 * cache_rows / cache_logw (capacity 8 n_out + 2), its size to cache_len and
 * the final thinning factor m to m_final.
 */
int or_express_decode(const double* Q, const double* K, const double* V, int64_t n, int64_t d,
                      int64_t n_out, int mbar, double delta, int halve, const float* U,
                      const float* sub_u, const uint8_t* follow, double tol, uint8_t* bits,
                      double* O, int32_t* cache_rows, double* cache_logw, int64_t* cache_len,
                      int* m_final, or_stats_t* st);

/* Per-point key counts of Thinformer decoding: keys[p] = size of point p's
 * weighted cache plus one (the point itself), p < n.  Returns 0. */
int or_express_keys(int64_t n, int64_t n_out, int mbar, const float* sub_u, int64_t* keys);
/* Uniforms a decode of n points consumes at most (or -1); *draws (nullable)
 * the Subsample draws it needs. */
int64_t or_express_uniforms(int64_t n, int64_t n_out, int mbar, int64_t* draws);
/* Cor. 2: delta_{m,i} (i >= 0) or delta_m / 2 (i < 0, the Halve phase). */
double or_express_delta(int m, int i, int mbar, double delta);

/* Weighted attention (eq. def:att_approx): key j weighs exp(logw[j]). */
void or_attention_weighted(const double* Q, const double* K, const double* V, int64_t n_q,
                           int64_t d, const int32_t* rows, const double* logw, int64_t m,
                           double* O);

#ifdef __cplusplus
}
#endif
#endif
