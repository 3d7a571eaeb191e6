/*
 * CPU oracle for the thinning hot path -- TEST INFRASTRUCTURE ONLY.
 * See oracle.h.  Everything is float64, single-threaded and written in the
 * order the paper states it; no blocking, no incremental reformulation.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ */
/* Level structure.                                                    */
/*                                                                     */
/* The output size n_out and the oversampling parameter g are read as  */
/* follows.  L = floor(log2(n / n_out)) halving rounds take            */
/* n_kept = n_out 2^L rows down to n_out.  If n_kept < n, a stratified */
/* subsample (one draw per contiguous stratum) first keeps n_kept rows */
/* (Sec. 3.1: Express subsamples first, then runs Compress2).  The     */
/* first m_c = L - min(g, L) rounds are Offline-Compress2 (App. H,     */
/* Algorithm H.2) with output size 2^g n_out; the remaining rounds      */
/* halve the whole set, as Express halves its coreset twice (Alg. 1).  */
/* Compress2 at level m partitions its 2^m n_out' input into 4^(m-1)    */
/* equal groups, so every group must hold an even number >= 2 of rows. */
/* ------------------------------------------------------------------ */
int or_plan(int64_t n, int64_t n_out, int32_t g, or_plan_t* plan) {
  if (n < 1 || n_out < 1 || n_out > n || g < 0 || plan == NULL) return -1;
  int32_t L = 0;
  while (n_out * ((int64_t)1 << (L + 1)) <= n) L++;
  int64_t n_kept = n_out * ((int64_t)1 << L);
  int32_t g_eff = g < L ? g : L;
  int32_t mc = L - g_eff;
  /* every Compress2 group at every level: n_in(m) / 4^(m-1), n_in(m) = 2^m 2^g_eff n_out */
  for (int32_t m = mc; m >= 1; --m) {
    int64_t n_in = n_out * ((int64_t)1 << (g_eff + m));
    int64_t groups = (int64_t)1 << (2 * (m - 1));
    if (n_in % groups != 0) return -1;
    int64_t size = n_in / groups;
    if (size < 2 || size % 2 != 0) return -1;
  }
  plan->n_kept = n_kept;
  plan->rounds = L;
  plan->compress_levels = mc;
  plan->subsample = n_kept < n ? 1 : 0;
  plan->uniforms = (plan->subsample ? n_kept : 0) + (n_kept - n_out);
  return 0;
}

/* v_max = max_i ||v_i||_inf over all n rows (Sec. 2.1, eq. katt). */
double or_vmax2(const double* V, int64_t n, int64_t d) {
  double m = 0.0;
  for (int64_t i = 0; i < n * d; ++i) {
    double a = fabs(V[i]);
    if (a > m) m = a;
  }
  return m * m;
}

/*
 * Stratified subsample (Alg. 3 / Algorithm H.1: keep one uniformly drawn
 * point per group).  Strata are the contiguous ranges
 * [floor(t n / n_kept), floor((t+1) n / n_kept)); with u = k 2^-24 the draw
 * floor(u len) is computed exactly in integers.
 */
void or_subsample(int64_t n, int64_t n_kept, const float* u, int32_t* out) {
  for (int64_t t = 0; t < n_kept; ++t) {
    int64_t start = (t * n) / n_kept;
    int64_t end = ((t + 1) * n) / n_kept;
    int64_t len = end - start;
    int64_t k = (int64_t)((double)u[t] * 16777216.0);
    int64_t pick = (k * len) >> 24;
    if (pick > len - 1) pick = len - 1;
    out[t] = (int32_t)(start + pick);
  }
}

/* ------------------------------------------------------------------ */
/* Kernels.                                                            */
/* ------------------------------------------------------------------ */
typedef struct {
  const double* K;
  const double* V;
  int64_t d;
  double vmax2;
  double inv_sqrt_d;
  int kernel;
} kctx_t;

static double dot(const double* a, const double* b, int64_t d) {
  double s = 0.0;
  for (int64_t c = 0; c < d; ++c) s += a[c] * b[c];
  return s;
}

/* Sec. 2.1, eq. katt. */
static double kap(const kctx_t* c, int32_t i, int32_t j) {
  const double* ki = c->K + (int64_t)i * c->d;
  const double* kj = c->K + (int64_t)j * c->d;
  const double* vi = c->V + (int64_t)i * c->d;
  const double* vj = c->V + (int64_t)j * c->d;
  if (c->kernel == OR_KERNEL_LINEAR) return dot(ki, kj, c->d) + dot(vi, vj, c->d);
  return exp(dot(ki, kj, c->d) * c->inv_sqrt_d) * (dot(vi, vj, c->d) + c->vmax2);
}

/*
 * KH(delta), App. A Algorithm A.1.  Pair i takes the next two points
 * (x, x') = (y_{2i-1}, y_{2i}) in input order.  Its RKHS distance b_i and the
 * running maximum b_max give the threshold a_i = b_i b_max (1/2 + log(2N/delta))
 * (natural log).  The balance score alpha_i sums f_i = k(x,.) - k(x',.) over
 * all earlier points and subtracts twice the sum over coreset 1.  The pair is
 * swapped with probability min(1, (1 - alpha_i/a_i)_+ / 2), realised as
 * "u_i < p_i"; coreset 1 then receives the first element.  When a_i = 0 the
 * ratio is undefined and p_i = 1/2 is used.
 */
int or_kernel_halving(const double* K, const double* V, int64_t d, double vmax2,
                      int kernel, double delta, const int32_t* rows, int64_t N,
                      const float* u, int32_t* out, const uint8_t* follow, double tol,
                      uint8_t* bits, double* rho, double* alpha_tr, double* thresh_tr,
                      or_stats_t* st) {
  if (N < 2 || (N % 2) != 0 || d < 1 || !(delta > 0.0)) return -1;
  kctx_t c = {K, V, d, vmax2, 1.0 / sqrt((double)d), kernel};
  int64_t half = N / 2;
  double* f = (double*)malloc(sizeof(double) * (size_t)N);
  uint8_t* sw = (uint8_t*)malloc((size_t)half);
  if (!f || !sw) {
    free(f);
    free(sw);
    return -2;
  }
  const double logterm = 0.5 + log(2.0 * (double)N / delta);
  double bmax = 0.0;
  for (int64_t i = 0; i < half; ++i) {
    int32_t x = rows[2 * i], xp = rows[2 * i + 1];
    double b2 = kap(&c, x, x) + kap(&c, xp, xp) - 2.0 * kap(&c, x, xp);
    double b = sqrt(b2 > 0.0 ? b2 : 0.0);
    if (b > bmax) bmax = b;
    double a = b * bmax * logterm;

    double alpha = 0.0;
    for (int64_t j = 0; j < 2 * i; ++j) {
      f[j] = kap(&c, rows[j], x) - kap(&c, rows[j], xp);
      alpha += f[j];
    }
    double s1 = 0.0;
    for (int64_t ip = 0; ip < i; ++ip) s1 += f[2 * ip + sw[ip]];
    alpha -= 2.0 * s1;

    double ui = (double)u[i];
    double ratio = 0.0, p;
    if (a > 0.0) {
      ratio = alpha / a;
      p = 0.5 * (1.0 - ratio);
      if (p < 0.0) p = 0.0;
      if (p > 1.0) p = 1.0;
    } else {
      p = 0.5;
      if (st) st->zero_threshold++;
    }
    int swap = ui < p;
    double r = ratio - (1.0 - 2.0 * ui);
    if (st) {
      double ar = fabs(r);
      if (st->decisions == 0 || ar < st->min_abs_rho) st->min_abs_rho = ar;
    }
    if (follow) {
      int fb = follow[i] ? 1 : 0;
      if (fabs(r) < tol) {
        if (st) st->near_ties++;
        swap = fb;
      } else if (fb != swap) {
        if (st) st->hard_mismatch++;
        swap = fb;
      }
    }
    sw[i] = (uint8_t)swap;
    out[i] = swap ? xp : x;
    if (bits) bits[i] = (uint8_t)swap;
    if (rho) rho[i] = r;
    if (alpha_tr) alpha_tr[i] = alpha;
    if (thresh_tr) thresh_tr[i] = a;
    if (st) {
      st->decisions++;
      st->swaps += swap;
    }
  }
  free(f);
  free(sw);
  return 0;
}

/*
 * Uniform halving: each pair (x, x') = (y_{2i-1}, y_{2i}) keeps one of its
 * two points with probability 1/2, the second iff u_i < 1/2.  It uses no
 * kernel: the simplest of the base halving algorithms the streaming
 * construction admits (Sec. 5, Conclusion: any halving algorithm), and the
 * rule KH(delta) applies to a pair whose threshold a_i is 0.
 */
int or_uniform_halving(const int32_t* rows, int64_t N, const float* u, int32_t* out,
                       uint8_t* bits, or_stats_t* st) {
  if (N < 2 || (N % 2) != 0) return -1;
  for (int64_t i = 0; i < N / 2; ++i) {
    int swap = u[i] < 0.5f;
    out[i] = rows[2 * i + swap];
    if (bits) bits[i] = (uint8_t)swap;
    if (st) {
      st->decisions++;
      st->swaps += swap;
    }
  }
  return 0;
}

/* ------------------------------------------------------------------ */
/* Compress.                                                           */
/* ------------------------------------------------------------------ */
typedef struct {
  const double* K;
  const double* V;
  int64_t d;
  double vmax2;
  int kernel;
  const float* U;
  int64_t upos;          /* next unread uniform of this slice */
  const uint8_t* follow; /* indexed like U */
  double tol;
  uint8_t* bits;
  double* rho;
  or_stats_t* st;
  int halve;            /* OR_HALVE_KH or OR_HALVE_UNIFORM */
  const double* delta;  /* KH failure probability per round, or NULL = 1/2 */
  int32_t round;        /* round of the calls being made */
} cctx_t;

static int halve_group(cctx_t* c, const int32_t* rows, int64_t N, int32_t* out) {
  int64_t o = c->upos;
  int rc;
  if (c->halve == OR_HALVE_UNIFORM) {
    rc = or_uniform_halving(rows, N, c->U + o, out, c->bits ? c->bits + o : NULL, c->st);
  } else {
    const double delta = c->delta ? c->delta[c->round] : 0.5;
    rc = or_kernel_halving(c->K, c->V, c->d, c->vmax2, c->kernel, delta, rows, N, c->U + o,
                           out, c->follow ? c->follow + o : NULL, c->tol,
                           c->bits ? c->bits + o : NULL, c->rho ? c->rho + o : NULL, NULL,
                           NULL, c->st);
  }
  c->upos += N / 2;
  return rc;
}

/*
 * Offline-Compress2 (App. H, Algorithm H.2): with m = 0 return the input;
 * otherwise split the 2^m n_out' input into 4^(m-1) equal contiguous groups,
 * halve every group, concatenate the halves in group order and recurse on
 * m - 1.  `rows` is consumed; the result is written to `rows` itself.
 */
static int compress2(cctx_t* c, int32_t m, int32_t* rows, int64_t n_in, int32_t* tmp) {
  if (m == 0) return 0;
  int64_t groups = (int64_t)1 << (2 * (m - 1));
  int64_t size = n_in / groups;
  for (int64_t k = 0; k < groups; ++k) {
    int rc = halve_group(c, rows + k * size, size, tmp + k * (size / 2));
    if (rc) return rc;
  }
  memcpy(rows, tmp, sizeof(int32_t) * (size_t)(n_in / 2));
  c->round++;
  return compress2(c, m - 1, rows, n_in / 2, tmp);
}

int or_compress(const double* K, const double* V, int64_t n, int64_t d, int64_t n_out,
                int32_t g, int kernel, const float* U, int32_t* idx_out,
                const uint8_t* follow, double tol, uint8_t* bits, double* rho,
                or_stats_t* st) {
  return or_compress_ex(K, V, n, d, n_out, g, kernel, OR_HALVE_KH, NULL, U, idx_out, follow,
                        tol, bits, rho, st);
}

int or_compress_ex(const double* K, const double* V, int64_t n, int64_t d, int64_t n_out,
                   int32_t g, int kernel, int halve, const double* delta, const float* U,
                   int32_t* idx_out, const uint8_t* follow, double tol, uint8_t* bits,
                   double* rho, or_stats_t* st) {
  or_plan_t plan;
  if (or_plan(n, n_out, g, &plan) != 0) return -1;
  int32_t* rows = (int32_t*)malloc(sizeof(int32_t) * (size_t)n);
  int32_t* tmp = (int32_t*)malloc(sizeof(int32_t) * (size_t)n);
  if (!rows || !tmp) {
    free(rows);
    free(tmp);
    return -2;
  }
  if (halve != OR_HALVE_KH && halve != OR_HALVE_UNIFORM) {
    free(rows);
    free(tmp);
    return -1;
  }
  cctx_t c = {K, V, d, halve == OR_HALVE_KH ? or_vmax2(V, n, d) : 0.0, kernel, U, 0, follow,
              tol, bits, rho, st, halve, delta, 0};
  int64_t cur = n;
  if (plan.subsample) {
    or_subsample(n, plan.n_kept, U, rows);
    c.upos = plan.n_kept;
    cur = plan.n_kept;
  } else {
    for (int64_t i = 0; i < n; ++i) rows[i] = (int32_t)i;
  }
  int rc = compress2(&c, plan.compress_levels, rows, cur, tmp);
  cur >>= plan.compress_levels;
  for (int32_t r = plan.compress_levels; rc == 0 && r < plan.rounds; ++r) {
    c.round = r;
    rc = halve_group(&c, rows, cur, tmp);
    memcpy(rows, tmp, sizeof(int32_t) * (size_t)(cur / 2));
    cur /= 2;
  }
  if (rc == 0) memcpy(idx_out, rows, sizeof(int32_t) * (size_t)n_out);
  free(rows);
  free(tmp);
  return rc;
}

/* ------------------------------------------------------------------ */
/* Attention over a coreset (eq. unmaskedatt; eq. def:att_approx with   */
/* equal weights, which cancel in the ratio).                          */
/* ------------------------------------------------------------------ */
void or_attention(const double* Q, const double* K, const double* V, int64_t n_q,
                  int64_t d, const int32_t* rows, int64_t m, double* O) {
  double* s = (double*)malloc(sizeof(double) * (size_t)(m > 0 ? m : 1));
  double inv = 1.0 / sqrt((double)d);
  for (int64_t q = 0; q < n_q; ++q) {
    const double* qq = Q + q * d;
    double mx = -INFINITY;
    for (int64_t j = 0; j < m; ++j) {
      s[j] = dot(qq, K + (int64_t)rows[j] * d, d) * inv;
      if (s[j] > mx) mx = s[j];
    }
    double den = 0.0;
    double* o = O + q * d;
    for (int64_t c = 0; c < d; ++c) o[c] = 0.0;
    for (int64_t j = 0; j < m; ++j) {
      double w = exp(s[j] - mx);
      den += w;
      const double* v = V + (int64_t)rows[j] * d;
      for (int64_t c = 0; c < d; ++c) o[c] += w * v[c];
    }
    for (int64_t c = 0; c < d; ++c) o[c] /= den;
  }
  free(s);
}

/*
 * Weighted attention over a weighted coreset (eq. def:att_approx): key j
 * carries weight w_j = exp(logw[j]) (logw[j] = -inf drops it),
 *   O[q] = sum_j w_j exp(<Q_q,K_rows[j]>/sqrt d) V_rows[j] / sum_j w_j exp(...).
 */
void or_attention_weighted(const double* Q, const double* K, const double* V, int64_t n_q,
                           int64_t d, const int32_t* rows, const double* logw, int64_t m,
                           double* O) {
  double* s = (double*)malloc(sizeof(double) * (size_t)(m > 0 ? m : 1));
  double inv = 1.0 / sqrt((double)d);
  for (int64_t q = 0; q < n_q; ++q) {
    const double* qq = Q + q * d;
    double mx = -INFINITY;
    for (int64_t j = 0; j < m; ++j) {
      s[j] = dot(qq, K + (int64_t)rows[j] * d, d) * inv + logw[j];
      if (s[j] > mx) mx = s[j];
    }
    double den = 0.0;
    double* o = O + q * d;
    for (int64_t c = 0; c < d; ++c) o[c] = 0.0;
    for (int64_t j = 0; j < m; ++j) {
      if (!(s[j] > -INFINITY)) continue;
      double w = exp(s[j] - mx);
      den += w;
      const double* v = V + (int64_t)rows[j] * d;
      for (int64_t c = 0; c < d; ++c) o[c] += w * v[c];
    }
    for (int64_t c = 0; c < d; ++c) o[c] /= den;
  }
  free(s);
}

/* ------------------------------------------------------------------ */
/* Express (Alg. 1) with Subsample (Alg. 3) and Compress2 (Alg. 2),  */
/* and Thinformer decoding (Alg. 4 with WtdAttention, Alg. 5).        */
/* ------------------------------------------------------------------ */
#define EX_MAXL 32

typedef struct {
  const double* K;
  const double* V;
  int64_t d, n_out;
  int mbar;
  double delta;
  int halve;
  const float* U;
  int64_t upos;
  const uint8_t* follow;
  double tol;
  uint8_t* bits;
  or_stats_t* st;
  int m;             /* thinning factor */
  int64_t n, ell;    /* points seen, points of the current thin group */
  int32_t* E;        /* Express coreset */
  int64_t nE;
  int mp;            /* m ^ mbar of the current Compress2 */
  int32_t* C[EX_MAXL + 1];
  int64_t nC[EX_MAXL + 1];
  int32_t* tmp;
  int over;          /* a Compress2 group size is not an even integer >= 2 */
  int count_only;    /* only count the uniforms the Halve calls consume */
  const float* sub_u; /* Subsample draws, one per stratum (NULL: 0 each) */
  int64_t sub_pos;   /* draws used */
  int64_t sub_n, sub_i; /* Subsample: points seen since its reset, the kept one */
} ex_t;

/* Cor. 2: delta_m, the budget of level m, and delta_{m,i}. */
double or_express_delta(int m, int i, int mbar, double delta) {
  const double dm = 0.5 * delta * (1.0 / log2(m / 2.0 + 2.0) - 1.0 / log2(m / 2.0 + 3.0));
  if (i < 0) return dm / 2.0; /* Halve_{m,m} = KH(delta_m / 2) */
  const int mp = m < mbar ? m : mbar;
  return ldexp(dm, 2 * (i + 1 - mp)) / (3.0 * mp);
}

/* One Halve call on rows[0..N): KH under kappa_att with v_max over these rows. */
static int ex_halve(ex_t* x, const int32_t* rows, int64_t N, double delta, int32_t* out) {
  const int64_t o = x->upos;
  int rc;
  if (x->count_only) {
    for (int64_t i = 0; i < N / 2; ++i) out[i] = rows[2 * i];
    rc = 0;
  } else if (x->halve == OR_HALVE_UNIFORM) {
    rc = or_uniform_halving(rows, N, x->U + o, out, x->bits ? x->bits + o : NULL, x->st);
  } else {
    double vm = 0.0;
    for (int64_t j = 0; j < N; ++j)
      for (int64_t c = 0; c < x->d; ++c) {
        const double a = fabs(x->V[(int64_t)rows[j] * x->d + c]);
        if (a > vm) vm = a;
      }
    rc = or_kernel_halving(x->K, x->V, x->d, vm * vm, OR_KERNEL_KATT, delta, rows, N, x->U + o,
                           out, x->follow ? x->follow + o : NULL, x->tol,
                           x->bits ? x->bits + o : NULL, NULL, NULL, NULL, x->st);
  }
  x->upos += N / 2;
  return rc;
}

/* Compress2(mp, 2^mp n_out).update: C_i is halved when it holds n_out 2^(i+2-mp) points. */
static int ex_compress2_update(ex_t* x, int32_t p) {
  x->C[0][x->nC[0]++] = p;
  for (int i = 0; i < x->mp; ++i) {
    const int64_t T = (x->n_out << (i + 2)) >> x->mp;
    if (x->nC[i] == T) {
      int rc = ex_halve(x, x->C[i], T, or_express_delta(x->m, i, x->mbar, x->delta),
                        x->C[i + 1] + x->nC[i + 1]);
      if (rc) return rc;
      x->nC[i + 1] += T / 2;
      x->nC[i] = 0;
    }
  }
  return 0;
}

/* Subsample(m, mbar).keep (Alg. 3): above mbar one point of each stratum of
 * 2^(m - mbar) points, at offset floor(u R) from the stratum's start. */
static int ex_keep(ex_t* x) {
  x->sub_n += 1;
  if (x->m <= x->mbar) return 1;
  const int64_t R = (int64_t)1 << (x->m - x->mbar);
  if ((x->sub_n - 1) % R == 0) {
    const double u = x->sub_u ? (double)x->sub_u[x->sub_pos] : 0.0;
    x->sub_pos += 1;
    int64_t off = (int64_t)floor(u * (double)R);
    if (off > R - 1) off = R - 1;
    x->sub_i = x->sub_n + off;
  }
  return x->sub_n == x->sub_i;
}

static void ex_reset_c(ex_t* x) {
  x->mp = x->m < x->mbar ? x->m : x->mbar;
  x->sub_n = 0;
  /* Compress2's smallest groups, 4 n_out / 2^mp points, must be even and >= 2 */
  if (x->mp >= 1 && ((4 * x->n_out) % ((int64_t)1 << x->mp) != 0 ||
                     ((4 * x->n_out) >> x->mp) < 2 || (((4 * x->n_out) >> x->mp) & 1)))
    x->over = 1;
  for (int i = 0; i <= EX_MAXL; ++i) x->nC[i] = 0;
}

/* Express.update with point p (Alg. 1). */
static int ex_update(ex_t* x, int32_t p) {
  x->n += 1;
  if (x->n <= x->n_out) {
    x->E[x->nE++] = p;
    return 0;
  }
  if (x->over) return -1;
  x->ell += 1;
  int rc = ex_keep(x) ? ex_compress2_update(x, p) : 0;
  if (rc) return rc;
  if (x->ell == (x->n_out << x->m)) {
    memcpy(x->E + x->nE, x->C[x->mp], sizeof(int32_t) * (size_t)x->nC[x->mp]);
    x->nE += x->nC[x->mp];
    x->ell = 0;
  }
  if (x->n == 4 * (x->n_out << x->m)) {
    const double dl = or_express_delta(x->m, -1, x->mbar, x->delta);
    rc = ex_halve(x, x->E, x->nE, dl, x->tmp);
    if (!rc) rc = ex_halve(x, x->tmp, x->nE / 2, dl, x->E);
    if (rc) return rc;
    x->nE /= 4;
    x->m += 2;
  }
  if (x->ell == 0) ex_reset_c(x);
  return 0;
}

/* Weighted cache (Express.wtd_cache): C_0..C_mp with weights 2^(i-mp), then E
 * with weight 1; returns its size. */
static int64_t ex_cache(const ex_t* x, int32_t* rows, double* logw) {
  int64_t k = 0;
  for (int i = 0; i <= x->mp; ++i)
    for (int64_t j = 0; j < x->nC[i]; ++j) {
      rows[k] = x->C[i][j];
      logw[k++] = (double)(i - x->mp) * log(2.0);
    }
  for (int64_t j = 0; j < x->nE; ++j) {
    rows[k] = x->E[j];
    logw[k++] = 0.0;
  }
  return k;
}

/* forward declaration: the uniforms a decode of n points consumes */
static int ex_run(ex_t* x, const double* Q, int64_t n, double* O, int32_t* rows, double* logw,
                  int64_t* keys);

int or_express_decode(const double* Q, const double* K, const double* V, int64_t n, int64_t d,
                      int64_t n_out, int mbar, double delta, int halve, const float* U,
                      const float* sub_u, const uint8_t* follow, double tol, uint8_t* bits,
                      double* O, int32_t* cache_rows, double* cache_logw, int64_t* cache_len,
                      int* m_final, or_stats_t* st) {
  if (n < 0 || n_out < 1 || d < 1 || mbar < 0 || mbar > EX_MAXL - 2) return -1;
  ex_t x;
  memset(&x, 0, sizeof(x));
  x.sub_u = sub_u;
  x.K = K; x.V = V; x.d = d; x.n_out = n_out; x.mbar = mbar; x.delta = delta;
  x.halve = halve; x.U = U; x.follow = follow; x.tol = tol; x.bits = bits; x.st = st;
  const int64_t capE = 4 * n_out, capW = 8 * n_out + 2;
  x.E = (int32_t*)malloc(sizeof(int32_t) * (size_t)capE);
  x.tmp = (int32_t*)malloc(sizeof(int32_t) * (size_t)capE);
  int32_t* rows = (int32_t*)malloc(sizeof(int32_t) * (size_t)capW);
  double* logw = (double*)malloc(sizeof(double) * (size_t)capW);
  int ok = x.E && x.tmp && rows && logw;
  for (int i = 0; i <= EX_MAXL && ok; ++i) {
    x.C[i] = (int32_t*)malloc(sizeof(int32_t) * (size_t)(4 * n_out));
    ok = x.C[i] != NULL;
  }
  int rc = ok ? ex_run(&x, Q, n, O, rows, logw, NULL) : -2;
  if (rc == 0) {
    int64_t k = ex_cache(&x, rows, logw);
    if (cache_rows) memcpy(cache_rows, rows, sizeof(int32_t) * (size_t)k);
    if (cache_logw) memcpy(cache_logw, logw, sizeof(double) * (size_t)k);
    if (cache_len) *cache_len = k;
    if (m_final) *m_final = x.m;
  }
  for (int i = 0; i <= EX_MAXL; ++i) free(x.C[i]);
  free(x.E);
  free(x.tmp);
  free(rows);
  free(logw);
  return rc;
}

static int ex_run(ex_t* x, const double* Q, int64_t n, double* O, int32_t* rows, double* logw,
                  int64_t* keys) {
  int rc = 0;
  ex_reset_c(x);
  for (int64_t p = 0; p < n && rc == 0; ++p) {
    if (keys) {
      /* the size of WtdAttention's key list for point p: the cache plus p */
      int64_t k = x->nE + 1;
      for (int i = 0; i <= x->mp; ++i) k += x->nC[i];
      keys[p] = k;
    }
    if (O) {
      /* WtdAttention: the cache plus the token itself in C_0 (weight 2^-mp) */
      int64_t k = ex_cache(x, rows, logw);
      rows[k] = (int32_t)p;
      logw[k++] = -(double)x->mp * log(2.0);
      or_attention_weighted(Q + p * x->d, x->K, x->V, 1, x->d, rows, logw, k, O + p * x->d);
    }
    rc = ex_update(x, (int32_t)p);
  }
  return rc;
}

/* Uniforms (upper bound: every stratum keeps its first point, so every Halve
 * call happens as early as it can) and Subsample draws of n points. */
int64_t or_express_uniforms(int64_t n, int64_t n_out, int mbar, int64_t* draws) {
  if (n < 0 || n_out < 1 || mbar < 0 || mbar > EX_MAXL - 2) return -1;
  ex_t x;
  memset(&x, 0, sizeof(x));
  x.n_out = n_out; x.mbar = mbar; x.delta = 0.5; x.count_only = 1;
  x.E = (int32_t*)malloc(sizeof(int32_t) * (size_t)(4 * n_out));
  x.tmp = (int32_t*)malloc(sizeof(int32_t) * (size_t)(4 * n_out));
  int ok = x.E && x.tmp;
  for (int i = 0; i <= EX_MAXL && ok; ++i) {
    x.C[i] = (int32_t*)malloc(sizeof(int32_t) * (size_t)(4 * n_out));
    ok = x.C[i] != NULL;
  }
  int rc = ok ? ex_run(&x, NULL, n, NULL, NULL, NULL, NULL) : -2;
  for (int i = 0; i <= EX_MAXL; ++i) free(x.C[i]);
  free(x.E);
  free(x.tmp);
  if (draws) *draws = x.sub_pos;
  return rc == 0 ? x.upos : -1;
}

/* keys[p] = the number of keys point p attends over in Thinformer decoding
 * (its weighted cache plus itself), p < n; sub_u as in or_express_decode.
 * The sizes do not depend on the halving decisions, so no kernel is
 * evaluated. */
int or_express_keys(int64_t n, int64_t n_out, int mbar, const float* sub_u, int64_t* keys) {
  if (n < 0 || n_out < 1 || mbar < 0 || mbar > EX_MAXL - 2 || !keys) return -1;
  ex_t x;
  memset(&x, 0, sizeof(x));
  x.n_out = n_out; x.mbar = mbar; x.delta = 0.5; x.count_only = 1; x.sub_u = sub_u;
  x.E = (int32_t*)malloc(sizeof(int32_t) * (size_t)(4 * n_out));
  x.tmp = (int32_t*)malloc(sizeof(int32_t) * (size_t)(4 * n_out));
  int ok = x.E && x.tmp;
  for (int i = 0; i <= EX_MAXL && ok; ++i) {
    x.C[i] = (int32_t*)malloc(sizeof(int32_t) * (size_t)(4 * n_out));
    ok = x.C[i] != NULL;
  }
  int rc = ok ? ex_run(&x, NULL, n, NULL, NULL, NULL, keys) : -2;
  for (int i = 0; i <= EX_MAXL; ++i) free(x.C[i]);
  free(x.E);
  free(x.tmp);
  return rc;
}
